// Sparse gated MLP over a kept-row list (Section III Eq. (1), Section IV-B 3)-4)).
//
// k_gate_up: list-driven gate/up (steps 1-3) for callers that pass their own
// kept list: one wavefront per kept position, W_gate row streamed with
// 16-byte non-temporal loads (1 KB per wave instruction), W_up row only where
// some token's h1 > 0 (actual sparsity); h3 stored per row.
//
// k_down: step 4, y = sum_i h3_i * W_down^T[i, :] over the kept list.  The
// columns of y are cut into 512-wide tiles and the kept positions into
// chunks; block (tile, chunk) streams the 1 KB row segments of W_down^T of
// its chunk, skipping rows whose h3 is zero for every token, accumulates in
// registers, combines its waves in LDS and adds the tile into y with fp32
// atomics (y was zeroed by the gate/up kernel).  With 8 tiles the tile is
// blockIdx % 8, i.e. the XCD, so every atomic on a y tile stays on one XCD.
// One extra block sums the per-block work counters when they are requested.
#include "si_device.h"
#include "si_launch.h"

namespace si {

constexpr uint32_t kNoAS = 1u;
constexpr int kDownChunks = 32;
constexpr int kDownWaves = 8;

template <int B>
__global__ __launch_bounds__(256) void k_gate_up(const u32x4* __restrict__ wg, const u32x4* __restrict__ wu,
                                                 int k, int d, const uint16_t* __restrict__ x,
                                                 const int32_t* __restrict__ idx,
                                                 const int32_t* __restrict__ n_ptr, float* __restrict__ h3row,
                                                 uint8_t* __restrict__ upflag, int32_t* __restrict__ counts,
                                                 uint32_t* __restrict__ hdr, float* __restrict__ y,
                                                 uint32_t flags) {
  extern __shared__ u32x4 xs[];  // [B][d/8]
  __shared__ int s_up, s_down;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int U = d >> 3;
  if (blockIdx.x == 0) {  // y is accumulated with atomics by k_down
    for (int i = tid; i < B * d; i += 256) y[i] = 0.f;
    if (tid == 0) hdr[H_H3_FORM] = kH3PlainByRow;
  }
  const int n = min(max(*n_ptr, 0), k);
  if ((int)blockIdx.x * 4 >= n) {
    if (tid == 0) {
      counts[2 * blockIdx.x] = 0;
      counts[2 * blockIdx.x + 1] = 0;
    }
    return;
  }
  for (int i = tid; i < B * U; i += 256) xs[i] = reinterpret_cast<const u32x4*>(x)[i];
  if (tid == 0) { s_up = 0; s_down = 0; }
  __syncthreads();

  int n_up = 0, n_down = 0;
  const bool no_as = (flags & kNoAS) != 0;
  for (int p = blockIdx.x * 4 + wv; p < n; p += gridDim.x * 4) {
    const int row = idx[p];
    if ((unsigned)row >= (unsigned)k) {  // never produced by the predictor
      if (lane == 0) atomicOr(&hdr[H_ERR], kErrRow);
      continue;
    }
    gate_up_row<B>(wg, wu, row, U, xs, lane, no_as, h3row, upflag, n_up, n_down);
  }
  if (lane == 0) { atomicAdd(&s_up, n_up); atomicAdd(&s_down, n_down); }
  __syncthreads();
  if (tid == 0) {
    counts[2 * blockIdx.x] = s_up;
    counts[2 * blockIdx.x + 1] = s_down;
  }
}

template <int B>
__global__ __launch_bounds__(kDownWaves * kWave) void k_down(
    const u32x4* __restrict__ wdt, int k, int d, const int32_t* __restrict__ idx,
    const int32_t* __restrict__ n_ptr, const float* __restrict__ h3row, float* __restrict__ y,
    const int32_t* __restrict__ counts, int slots, int32_t* __restrict__ counters, uint32_t flags, int tiles) {
  __shared__ float red[B][kTile];
  constexpr int NT = kDownWaves * kWave;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n = min(max(*n_ptr, 0), k);

  if ((int)blockIdx.x == tiles * kDownChunks) {  // counter block
    __shared__ int s_cnt[2];
    if (tid < 2) s_cnt[tid] = 0;
    __syncthreads();
    int a = 0, b = 0;
    for (int i = tid; i < slots; i += NT) { a += counts[2 * i]; b += counts[2 * i + 1]; }
    a = wave_sum_int(a);
    b = wave_sum_int(b);
    if (lane == 0) { atomicAdd(&s_cnt[0], a); atomicAdd(&s_cnt[1], b); }
    __syncthreads();
    if (tid == 0) {
      counters[0] = n;
      counters[1] = s_cnt[0];
      counters[2] = s_cnt[1];
    }
    return;
  }

  const int U = d >> 3;
  const int c = blockIdx.x % tiles, q = blockIdx.x / tiles;
  const int unit = c * (kTile / 8) + lane;  // 16-byte unit of the row: 8 columns
  const bool col_ok = unit < U;
  const int p0 = (int)((long long)n * q / kDownChunks);
  const int p1 = (int)((long long)n * (q + 1) / kDownChunks);
  if (p1 <= p0) return;
  for (int i = tid; i < B * kTile; i += NT) (&red[0][0])[i] = 0.f;
  __syncthreads();

  float acc[B][8];
#pragma unroll
  for (int t = 0; t < B; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[t][e] = 0.f;

  const bool no_as = (flags & kNoAS) != 0;
  constexpr int UNR = 4;
  for (int base = p0 + wv; base < p1; base += kDownWaves * UNR) {
    u32x4 w[UNR];
    float hv[UNR][B];
#pragma unroll
    for (int r = 0; r < UNR; ++r) {
      const int p = base + kDownWaves * r;
      const int row = p < p1 ? idx[p] : -1;
      const bool ok = (unsigned)row < (unsigned)k;
      bool any = false;
#pragma unroll
      for (int t = 0; t < B; ++t) {
        hv[r][t] = ok ? h3row[(size_t)row * B + t] : 0.f;
        any |= hv[r][t] != 0.f;
      }
      w[r] = u32x4{0, 0, 0, 0};
      if (ok && col_ok && (any || no_as)) w[r] = load_nt(wdt + (size_t)row * U + unit);
    }
#pragma unroll
    for (int r = 0; r < UNR; ++r) {
      const f16x2 a = as_h2(w[r].x), b2 = as_h2(w[r].y), c2 = as_h2(w[r].z), d2 = as_h2(w[r].w);
      const float f[8] = {(float)a.x, (float)a.y, (float)b2.x, (float)b2.y,
                          (float)c2.x, (float)c2.y, (float)d2.x, (float)d2.y};
#pragma unroll
      for (int t = 0; t < B; ++t)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[t][e] = fmaf(hv[r][t], f[e], acc[t][e]);
    }
  }
  if (col_ok) {
#pragma unroll
    for (int t = 0; t < B; ++t)
#pragma unroll
      for (int e = 0; e < 8; ++e) atomicAdd(&red[t][lane * 8 + e], acc[t][e]);
  }
  __syncthreads();
  for (int i = tid; i < B * kTile; i += NT) {
    const int t = i / kTile, col = c * kTile + (i - t * kTile);
    const float v = (&red[0][0])[i];
    if (col < d && v != 0.f) unsafeAtomicAdd(&y[(size_t)t * d + col], v);
  }
}

template <int B>
static hipError_t down_b(const uint16_t* w_down_t, int k, int d, const int32_t* idx, const int32_t* n_active,
                         float* y, void* ws, int slots, uint32_t flags, int32_t* counters, hipStream_t s) {
  const WsLayout L = ws_layout(k, B);
  char* base = static_cast<char*>(ws);
  const int tiles = (d + kTile - 1) / kTile;
  const int blocks = tiles * kDownChunks + (counters ? 1 : 0);
  k_down<B><<<blocks, kDownWaves * kWave, 0, s>>>(
      reinterpret_cast<const u32x4*>(w_down_t), k, d, idx, n_active, reinterpret_cast<const float*>(base + L.h3),
      y, reinterpret_cast<const int32_t*>(base + L.counts), slots, counters, flags, tiles);
  return hipGetLastError();
}

template <int B>
static hipError_t gate_up_b(const uint16_t* w_gate, const uint16_t* w_up, int k, int d, const uint16_t* x,
                            const int32_t* idx, const int32_t* n_active, float* y, void* ws, uint32_t flags,
                            int* slots, hipStream_t s) {
  const WsLayout L = ws_layout(k, B);
  char* base = static_cast<char*>(ws);
  const size_t lds = (size_t)B * d * sizeof(uint16_t);
  // the kernel's dynamic LDS limit, set once per device
  static std::atomic<int> attr_set[kMaxDevices];
  const int ok = per_device_once(attr_set, [](int) -> int {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gate_up<B>), hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)((size_t)kMaxB * kMaxD * sizeof(uint16_t))) == hipSuccess ? 1 : -1;
  });
  if (ok != 1) return hipErrorInvalidConfiguration;
  int blocks = (k + 3) / 4;
  if (blocks > kGateUpMaxBlocks) blocks = kGateUpMaxBlocks;
  *slots = blocks;
  k_gate_up<B><<<blocks, 256, lds, s>>>(
      reinterpret_cast<const u32x4*>(w_gate), reinterpret_cast<const u32x4*>(w_up), k, d, x, idx, n_active,
      reinterpret_cast<float*>(base + L.h3), reinterpret_cast<uint8_t*>(base + L.upflag),
      reinterpret_cast<int32_t*>(base + L.counts), reinterpret_cast<uint32_t*>(base), y, flags);
  return hipGetLastError();
}

#define SI_B_CASES(CALL)             \
  switch (b) {                       \
    case 1: return CALL(1);          \
    case 2: return CALL(2);          \
    case 3: return CALL(3);          \
    case 4: return CALL(4);          \
    case 5: return CALL(5);          \
    case 6: return CALL(6);          \
    case 7: return CALL(7);          \
    case 8: return CALL(8);          \
    default: return hipErrorInvalidValue; \
  }

hipError_t launch_down(const uint16_t* w_down_t, int k, int d, int b, const int32_t* idx, const int32_t* n_active,
                       float* y, void* ws, int slots, uint32_t flags, int32_t* counters, hipStream_t s) {
#define CALL(B) down_b<B>(w_down_t, k, d, idx, n_active, y, ws, slots, flags, counters, s)
  SI_B_CASES(CALL)
#undef CALL
}

hipError_t launch_sparse_mlp(const uint16_t* w_gate, const uint16_t* w_up, const uint16_t* w_down_t, int k,
                             int d, const uint16_t* x, int b, const int32_t* idx, const int32_t* n_active,
                             float* y, void* ws, uint32_t flags, int32_t* counters, hipStream_t s) {
  int slots = 0;
  hipError_t e;
  switch (b) {
#define CASE(B) \
  case B: e = gate_up_b<B>(w_gate, w_up, k, d, x, idx, n_active, y, ws, flags, &slots, s); break;
    CASE(1) CASE(2) CASE(3) CASE(4) CASE(5) CASE(6) CASE(7) CASE(8)
#undef CASE
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  return launch_down(w_down_t, k, d, b, idx, n_active, y, ws, slots, flags, counters, s);
}

#undef SI_B_CASES

}  // namespace si
