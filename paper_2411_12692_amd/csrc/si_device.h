// Device-side building blocks shared by the SparseInfer kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace si {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;       // CDNA wavefront width
constexpr int kRowGroup = 64;   // rows interleaved together in the packed-sign layout
constexpr int kMaxD = 8192;     // largest supported model dimension
constexpr int kMaxB = 8;        // largest supported decode batch
constexpr int kTile = 512;      // columns of y handled by one down-projection block

// Header words at the start of the workspace.
enum : int {
  H_EPOCH = 0,        // call counter: every predictor or layer call advances it once
  H_ERR = 1,          // sticky device-side error bits (read together with H_EPOCH as one 64-bit word)
  H_N_INTERNAL = 2,   // kept-row count when the list lives in the workspace
  H_H3_FORM = 3,      // where the last MLP call left its per-row h3 values (kH3*)
  H_WORDS = 64
};

constexpr uint32_t kErrLookbackSpin = 1u;  // a look-back wait hit its spin limit
constexpr uint32_t kErrRow = 4u;           // kept-row index outside [0, k)

// Where the last MLP call left h3 (Eq. (1) step 3) in the workspace.
constexpr uint32_t kH3ByRow = 1u;       // h3e[row][b]: this call's tag | fp32 bits
constexpr uint32_t kH3ByPos = 2u;       // h3e[list position][b]: this call's tag | fp32 bits
constexpr uint32_t kH3PlainByRow = 3u;  // h3[row][b] fp32, valid on the kept rows

constexpr int kGateUpMaxBlocks = 2048;     // grid cap of the list-driven gate/up kernel
constexpr int kMaxLayerBlocks = 1024;      // grid cap of the single-kernel path
constexpr int kOwnPubStride = 32;          // published words per block of the row-owning kernel

// Workspace layout (byte offsets), identical on host and device.  Regions
// whose size depends on the batch come last, so every other offset is the
// same for all batch sizes a workspace serves.
struct WsLayout {
  size_t status;  // uint64 [groups] look-back words
  size_t counts;  // int32 [slots][2]: rows whose W_up / W_down^T row was read, per block
  size_t idx;     // int32 [k] kept rows (when the caller gives none)
  size_t mask;    // uint8 [k] mask (when the caller gives none)
  size_t upflag;  // uint8 [k] 1 where the W_up row was read
  size_t lmask;   // uint64 [groups][4] single-kernel kept / confident masks
  size_t zflag;   // uint64 [64] single-kernel "tile of y zeroed" flags
  size_t alive;   // uint64 [kMaxLayerBlocks] single-kernel "this block has read the call counter" words
  size_t opub;    // uint64 [kMaxLayerBlocks][kOwnPubStride] row-owning kernel: masks and count per block
  size_t h3;      // float [k][b] h3 per row (valid on kept rows)
  size_t h3e;     // uint64 [groups][64][b] single-kernel h3 exchange words
  size_t total;
};

__host__ __device__ inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

__host__ __device__ inline int row_groups(int k) { return (k + kRowGroup - 1) / kRowGroup; }

__host__ __device__ inline int count_slots(int k) {
  const int g = row_groups(k);
  return g > kGateUpMaxBlocks ? g : kGateUpMaxBlocks;
}

__host__ __device__ inline WsLayout ws_layout(int k, int b) {
  WsLayout L;
  const size_t groups = (size_t)row_groups(k);
  L.status = align256(H_WORDS * sizeof(uint32_t));
  L.counts = L.status + align256(groups * sizeof(uint64_t));
  L.idx = L.counts + align256((size_t)count_slots(k) * 2 * sizeof(int32_t));
  L.mask = L.idx + align256((size_t)k * sizeof(int32_t));
  L.upflag = L.mask + align256((size_t)k);
  L.lmask = L.upflag + align256((size_t)k);
  L.zflag = L.lmask + align256(groups * 4 * sizeof(uint64_t));
  L.alive = L.zflag + align256(64 * sizeof(uint64_t));
  L.opub = L.alive + align256(kMaxLayerBlocks * sizeof(uint64_t));
  L.h3 = L.opub + align256((size_t)kMaxLayerBlocks * kOwnPubStride * sizeof(uint64_t));
  L.h3e = L.h3 + align256((size_t)k * b * sizeof(float));
  L.total = L.h3e + align256(groups * kRowGroup * (size_t)b * sizeof(uint64_t));
  return L;
}

// Sign bits of the 8 fp16 values held in one 16-byte vector, as bits 0..7.
__device__ inline uint32_t sign_byte(u32x4 v) {
  return ((v.x >> 15) & 1u) | ((v.x >> 30) & 2u) | ((v.y >> 13) & 4u) | ((v.y >> 28) & 8u) |
         ((v.z >> 11) & 16u) | ((v.z >> 26) & 32u) | ((v.w >> 9) & 64u) | ((v.w >> 24) & 128u);
}

// Packed word of the sign bits of 32 consecutive fp16 values (bit j = element j).
__device__ inline uint32_t sign_word(const u32x4* p) {
  return sign_byte(p[0]) | (sign_byte(p[1]) << 8) | (sign_byte(p[2]) << 16) | (sign_byte(p[3]) << 24);
}

__device__ inline f16x2 as_h2(uint32_t v) { return __builtin_bit_cast(f16x2, v); }

// Two floats rounded to fp16 (to nearest even), low half first.  The
// values are pinned as they are first: the compiler would otherwise fold a
// product that feeds the conversion into a mixed-precision FMA with a +0
// addend, which turns a -0 product into +0 (the predictor reads that sign).
__device__ inline uint32_t pack_h2(float lo, float hi) {
  asm volatile("" : "+v"(lo), "+v"(hi));
  const _Float16 a = (_Float16)lo, b = (_Float16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// acc + sum of the 8 products of two 16-byte fp16 vectors (fp32 accumulation).
__device__ inline float dot8(u32x4 a, u32x4 b, float acc) {
  acc = __builtin_amdgcn_fdot2(as_h2(a.x), as_h2(b.x), acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(a.y), as_h2(b.y), acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(a.z), as_h2(b.z), acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(a.w), as_h2(b.w), acc, false);
  return acc;
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

__device__ inline int wave_sum_int(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

__device__ inline u32x4 load_nt(const u32x4* p) { return __builtin_nontemporal_load(p); }

__device__ inline uint64_t lanes_below(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Tag that marks a word as written in the call with this epoch.  The high
// bit is always set, so a zero-filled workspace never carries a valid tag.
__device__ inline uint32_t epoch_tag(uint32_t epoch) { return (epoch & 0x7fffffffu) | 0x80000000u; }

// Wait until this wave's outstanding memory operations have completed.  The
// exchange words are written with agent-scope (write-through) stores, so once
// they complete they are visible to agent-scope loads from any XCD; a
// counter bumped afterwards therefore never runs ahead of the data it
// announces.  (Consumers also check every word's tag.)
__device__ inline void wait_own_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Wait for every outstanding vector memory request of the wave, as an
// instruction the compiler's wait-count pass sees (inline assembly is opaque
// to it): afterwards it knows that no load is pending, so it inserts no
// blanket wait, which would also wait for stores issued later, where a
// register of a possibly pending load is reused.
__device__ inline void wait_all_requests() { __builtin_amdgcn_s_waitcnt(0x0F70); }

__device__ inline uint32_t ld_agent(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void st_agent(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t ld_agent64(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void st_agent64(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

constexpr int kMaxUnitsPerLane = kMaxD / 8 / kWave;  // 16-byte units of a row per lane (16)

// Dot products of one [d] fp16 row (U = d/8 16-byte units, streamed with
// non-temporal loads) with B tokens staged in LDS as xs[t][U].  Every load of
// the row is issued before the first product.  Result in every lane.
template <int B>
__device__ inline void row_dot(const u32x4* __restrict__ row, const u32x4* xs, int U, int lane, float (&out)[B]) {
  u32x4 w[kMaxUnitsPerLane];
#pragma unroll
  for (int j = 0; j < kMaxUnitsPerLane; ++j) {
    const int u = lane + kWave * j;
    if (u < U) w[j] = load_nt(row + u);
  }
  float acc[B];
#pragma unroll
  for (int t = 0; t < B; ++t) acc[t] = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxUnitsPerLane; ++j) {
    const int u = lane + kWave * j;
    if (u < U) {
#pragma unroll
      for (int t = 0; t < B; ++t) acc[t] = dot8(w[j], xs[t * U + u], acc[t]);
    }
  }
#pragma unroll
  for (int t = 0; t < B; ++t) out[t] = wave_sum(acc[t]);
}

// Gate/up of one kept row (Eq. (1) steps 1-3 with actual sparsity): returns
// through h[] the B values h3 = ReLU(W_gate,row . x) * (W_up,row . x); the
// W_up row is read only if some token has a positive gate value (or always
// with no_as).  Without W_up (wu == nullptr: the non-gated ReLU MLP of
// blocks without step 2) h3 = ReLU(W_gate,row . x).  Stores h3 per row, the
// up-read flag, and counts the work.
template <int B>
__device__ inline void gate_up_row(const u32x4* __restrict__ wg, const u32x4* __restrict__ wu, int row, int U,
                                   const u32x4* xs, int lane, bool no_as, float* __restrict__ h3row,
                                   uint8_t* __restrict__ upflag, int& n_up, int& n_down) {
  float g[B];
  row_dot<B>(wg + (size_t)row * U, xs, U, lane, g);
  bool any = false;
#pragma unroll
  for (int t = 0; t < B; ++t) {
    g[t] = fmaxf(g[t], 0.f);
    any |= g[t] > 0.f;
  }
  float h[B];
#pragma unroll
  for (int t = 0; t < B; ++t) h[t] = 0.f;
  const bool gated = wu != nullptr;
  const bool up = gated && (any || no_as);
  if (up) {
    float u[B];
    row_dot<B>(wu + (size_t)row * U, xs, U, lane, u);
#pragma unroll
    for (int t = 0; t < B; ++t) h[t] = g[t] * u[t];
  } else if (!gated) {
#pragma unroll
    for (int t = 0; t < B; ++t) h[t] = g[t];
  }
  bool nz = false;
#pragma unroll
  for (int t = 0; t < B; ++t) nz |= h[t] != 0.f;
  n_up += up ? 1 : 0;
  n_down += (nz || no_as) ? 1 : 0;
#pragma unroll
  for (int t = 0; t < B; ++t)
    if (lane == t) h3row[(size_t)row * B + t] = h[t];
  if (lane == 0) upflag[row] = up ? 1 : 0;
}

// Optional phase timeline of the single-kernel paths (compile with
// -DSI_TRACE): per block (wave 0) and per wave, the 100 MHz real-time
// counter at numbered points, held in registers and written out once at the
// end of the kernel so that no store is in flight while the kernel runs.
// Off in normal builds, where the marks compile to nothing.
constexpr int kTraceSlots = 32;
constexpr int kTraceBlockMarks = 12;
constexpr int kTraceWaveMarks = 8;
#ifdef SI_TRACE
extern __device__ uint64_t g_si_trace[];
extern __device__ uint64_t g_si_trace_wave[];
#define SI_TRACE_DECL                                                 \
  __shared__ uint64_t si_tr_[kTraceBlockMarks + 16 * kTraceWaveMarks]; \
  for (int si_i_ = threadIdx.x; si_i_ < kTraceBlockMarks + 16 * kTraceWaveMarks; si_i_ += blockDim.x) si_tr_[si_i_] = 0
#define SI_TRACE_MARK(slot)                                               \
  do {                                                                    \
    if (threadIdx.x == 0) si_tr_[(slot)] = __builtin_amdgcn_s_memrealtime(); \
  } while (0)
#define SI_TRACE_WAVE(mark)                                                                                  \
  do {                                                                                                       \
    if ((threadIdx.x & 63) == 0)                                                                             \
      si_tr_[kTraceBlockMarks + (threadIdx.x >> 6) * kTraceWaveMarks + (mark)] = __builtin_amdgcn_s_memrealtime(); \
  } while (0)
#define SI_TRACE_FLUSH                                                                                     \
  do {                                                                                                     \
    __syncthreads();                                                                                       \
    if (threadIdx.x < kTraceBlockMarks)                                                                    \
      g_si_trace[(size_t)blockIdx.x * kTraceSlots + threadIdx.x] = si_tr_[threadIdx.x];                    \
    if (threadIdx.x < 16 * kTraceWaveMarks)                                                                \
      g_si_trace_wave[(size_t)blockIdx.x * 16 * kTraceWaveMarks + threadIdx.x] =                           \
          si_tr_[kTraceBlockMarks + threadIdx.x];                                                          \
  } while (0)
#else
#define SI_TRACE_DECL \
  do {                \
  } while (0)
#define SI_TRACE_MARK(slot) \
  do {                      \
  } while (0)
#define SI_TRACE_WAVE(mark) \
  do {                      \
  } while (0)
#define SI_TRACE_FLUSH \
  do {                 \
  } while (0)
#endif

}  // namespace si
