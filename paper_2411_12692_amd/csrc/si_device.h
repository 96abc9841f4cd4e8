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
  H_PRED_TICKET = 0,  // next virtual row-group id of the predictor
  H_PRED_EPOCH = 1,   // call counter tagging the predictor's look-back words
  H_PRED_DONE = 2,    // predictor blocks finished in this call
  H_ERR = 3,          // sticky device-side error bits
  H_N_UP = 4,         // rows whose W_up row was read (this call)
  H_N_DOWN = 5,       // rows whose W_down^T row was read (this call)
  H_DOWN_DONE = 6,    // down-projection blocks finished in this call
  H_N_INTERNAL = 7,   // kept-row count when the list lives in the workspace
  H_WORDS = 64
};

constexpr uint32_t kErrLookbackSpin = 1u;  // a look-back wait hit its spin limit
constexpr uint32_t kErrTicket = 2u;        // predictor ticket out of range
constexpr uint32_t kErrRow = 4u;           // kept-row index outside [0, k)

// Workspace layout (byte offsets), identical on host and device.
struct WsLayout {
  size_t status;  // uint64 look-back word per row group
  size_t idx;     // int32 [k] kept rows (when the caller gives none)
  size_t mask;    // uint8 [k] mask (when the caller gives none)
  size_t h3;      // float [k][b] h3 of each kept position
  size_t total;
};

__host__ __device__ inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

__host__ __device__ inline WsLayout ws_layout(int k, int b) {
  WsLayout L;
  const size_t groups = (size_t)(k + kRowGroup - 1) / kRowGroup;
  L.status = align256(H_WORDS * sizeof(uint32_t));
  L.idx = L.status + align256(groups * sizeof(uint64_t));
  L.mask = L.idx + align256((size_t)k * sizeof(int32_t));
  L.h3 = L.mask + align256((size_t)k);
  L.total = L.h3 + align256((size_t)k * b * sizeof(float));
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

__device__ inline u32x4 load_nt(const u32x4* p) { return __builtin_nontemporal_load(p); }

__device__ inline uint64_t lanes_below(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

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

}  // namespace si
