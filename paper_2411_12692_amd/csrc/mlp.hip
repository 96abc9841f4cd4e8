// Sparse gated MLP over the kept rows (Section III Eq. (1), Section IV-B 3)-4)).
//
// k_gate_up: one wavefront per kept position.  The wave streams the W_gate
// row (16-byte non-temporal loads, 1 KB per wave instruction), dots it with
// every token of x (staged once per block in LDS), reduces across lanes, and
// applies ReLU.  Only if some token's h1 is positive does it stream the W_up
// row (actual sparsity); h3 = h1 * u is written per position.
//
// k_down: y = sum_i h3_i * W_down^T[i, :].  The columns of y are cut into
// 512-wide tiles and the kept positions into Q chunks; block (tile, chunk)
// reads 1 KB row segments of W_down^T for its chunk, skipping positions whose
// h3 is zero for every token, accumulates in registers, combines its 4 waves
// in LDS and adds the tile into y with fp32 atomics.  With 8 tiles, tile ==
// blockIdx % 8 keeps every atomic on one y tile inside one XCD.
#include "si_device.h"
#include "si_launch.h"

namespace si {

constexpr uint32_t kNoAS = 1u;
constexpr int kDownChunks = 64;
constexpr int kGateUpMaxBlocks = 2048;
constexpr int kMaxUnitsPerLane = kMaxD / 8 / kWave;  // 16

// Dot products of one [d] fp16 row with the B tokens staged in LDS.
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

template <int B>
__global__ __launch_bounds__(256) void k_gate_up(const u32x4* __restrict__ wg, const u32x4* __restrict__ wu,
                                                 int k, int d, const uint16_t* __restrict__ x,
                                                 const int32_t* __restrict__ idx,
                                                 const int32_t* __restrict__ n_ptr, float* __restrict__ h3,
                                                 uint32_t* __restrict__ hdr, float* __restrict__ y,
                                                 uint32_t flags) {
  extern __shared__ u32x4 xs[];  // [B][d/8]
  __shared__ int s_up, s_down;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int U = d >> 3;
  if (blockIdx.x == 0) {  // y is accumulated with atomics by k_down
    for (int i = tid; i < B * d; i += 256) y[i] = 0.f;
  }
  const int n = min(max(*n_ptr, 0), k);
  if ((int)blockIdx.x * 4 >= n) return;
  for (int i = tid; i < B * U; i += 256) xs[i] = reinterpret_cast<const u32x4*>(x)[i];
  if (tid == 0) { s_up = 0; s_down = 0; }
  __syncthreads();

  int my_up = 0, my_down = 0;
  for (int p = blockIdx.x * 4 + wv; p < n; p += gridDim.x * 4) {
    const int row = idx[p];
    if ((unsigned)row >= (unsigned)k) {  // never produced by the predictor
      if (lane == 0) atomicOr(&hdr[H_ERR], kErrRow);
      if (lane < B) h3[(size_t)p * B + lane] = 0.f;
      continue;
    }
    float g[B];
    row_dot<B>(wg + (size_t)row * U, xs, U, lane, g);
    bool any = false;
#pragma unroll
    for (int t = 0; t < B; ++t) { g[t] = fmaxf(g[t], 0.f); any |= g[t] > 0.f; }
    float h[B];
#pragma unroll
    for (int t = 0; t < B; ++t) h[t] = 0.f;
    if (any || (flags & kNoAS)) {
      float u[B];
      row_dot<B>(wu + (size_t)row * U, xs, U, lane, u);
#pragma unroll
      for (int t = 0; t < B; ++t) h[t] = g[t] * u[t];
      ++my_up;
    }
    bool nz = false;
#pragma unroll
    for (int t = 0; t < B; ++t) nz |= h[t] != 0.f;
    my_down += (nz || (flags & kNoAS)) ? 1 : 0;
#pragma unroll
    for (int t = 0; t < B; ++t)
      if (lane == t) h3[(size_t)p * B + t] = h[t];
  }
  if (lane == 0) { atomicAdd(&s_up, my_up); atomicAdd(&s_down, my_down); }
  __syncthreads();
  if (tid == 0) {
    if (s_up) atomicAdd(&hdr[H_N_UP], (uint32_t)s_up);
    if (s_down) atomicAdd(&hdr[H_N_DOWN], (uint32_t)s_down);
  }
}

template <int B>
__global__ __launch_bounds__(256) void k_down(const u32x4* __restrict__ wdt, int k, int d,
                                              const int32_t* __restrict__ idx,
                                              const int32_t* __restrict__ n_ptr,
                                              const float* __restrict__ h3, float* __restrict__ y,
                                              uint32_t* __restrict__ hdr, int32_t* __restrict__ counters,
                                              uint32_t flags, int tiles) {
  __shared__ float red[B][kTile];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int U = d >> 3;
  const int c = blockIdx.x % tiles, q = blockIdx.x / tiles;
  const int n = min(max(*n_ptr, 0), k);
  const int unit = c * (kTile / 8) + lane;  // 16-byte unit of the row: 8 columns
  const bool col_ok = unit < U;
  const int p0 = (int)((long long)n * q / kDownChunks);
  const int p1 = (int)((long long)n * (q + 1) / kDownChunks);
  for (int i = tid; i < B * kTile; i += 256) (&red[0][0])[i] = 0.f;
  __syncthreads();

  float acc[B][8];
#pragma unroll
  for (int t = 0; t < B; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[t][e] = 0.f;

  constexpr int UNR = 4;
  for (int base = p0 + wv; base < p1; base += 4 * UNR) {
    u32x4 w[UNR];
    float hv[UNR][B];
#pragma unroll
    for (int r = 0; r < UNR; ++r) {
      const int p = base + 4 * r;
      bool any = false;
#pragma unroll
      for (int t = 0; t < B; ++t) {
        hv[r][t] = p < p1 ? h3[(size_t)p * B + t] : 0.f;
        any |= hv[r][t] != 0.f;
      }
      w[r] = u32x4{0, 0, 0, 0};
      if (p < p1 && col_ok && (any || (flags & kNoAS))) {
        const int row = idx[p];
        if ((unsigned)row < (unsigned)k) w[r] = load_nt(wdt + (size_t)row * U + unit);
      }
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
  if (col_ok && p1 > p0) {
#pragma unroll
    for (int t = 0; t < B; ++t)
#pragma unroll
      for (int e = 0; e < 8; ++e) atomicAdd(&red[t][lane * 8 + e], acc[t][e]);
  }
  __syncthreads();
  if (p1 > p0) {
    for (int i = tid; i < B * kTile; i += 256) {
      const int t = i / kTile, col = c * kTile + (i - t * kTile);
      const float v = (&red[0][0])[i];
      if (col < d && v != 0.f) unsafeAtomicAdd(&y[(size_t)t * d + col], v);
    }
  }
  if (tid == 0) {
    __threadfence();
    const uint32_t done = atomicAdd(&hdr[H_DOWN_DONE], 1u);
    if (done == gridDim.x - 1) {  // last block: publish and reset the per-call counters
      __threadfence();
      if (counters) {
        counters[0] = n;
        counters[1] = (int32_t)ld_agent(&hdr[H_N_UP]);
        counters[2] = (int32_t)ld_agent(&hdr[H_N_DOWN]);
      }
      st_agent(&hdr[H_N_UP], 0u);
      st_agent(&hdr[H_N_DOWN], 0u);
      st_agent(&hdr[H_DOWN_DONE], 0u);
    }
  }
}

template <int B>
static hipError_t sparse_mlp_b(const uint16_t* w_gate, const uint16_t* w_up, const uint16_t* w_down_t, int k,
                               int d, const uint16_t* x, const int32_t* idx, const int32_t* n_active, float* y,
                               void* ws, uint32_t flags, int32_t* counters, hipStream_t s) {
  const WsLayout L = ws_layout(k, B);
  char* base = static_cast<char*>(ws);
  uint32_t* hdr = reinterpret_cast<uint32_t*>(base);
  float* h3 = reinterpret_cast<float*>(base + L.h3);
  const size_t lds = (size_t)B * d * sizeof(uint16_t);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gate_up<B>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)((size_t)kMaxB * kMaxD * sizeof(uint16_t)));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  int blocks = (k + 3) / 4;
  if (blocks > kGateUpMaxBlocks) blocks = kGateUpMaxBlocks;
  k_gate_up<B><<<blocks, 256, lds, s>>>(reinterpret_cast<const u32x4*>(w_gate),
                                        reinterpret_cast<const u32x4*>(w_up), k, d, x, idx, n_active, h3, hdr, y,
                                        flags);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int tiles = (d + kTile - 1) / kTile;
  k_down<B><<<tiles * kDownChunks, 256, 0, s>>>(reinterpret_cast<const u32x4*>(w_down_t), k, d, idx, n_active, h3,
                                                 y, hdr, counters, flags, tiles);
  return hipGetLastError();
}

hipError_t launch_sparse_mlp(const uint16_t* w_gate, const uint16_t* w_up, const uint16_t* w_down_t, int k,
                             int d, const uint16_t* x, int b, const int32_t* idx, const int32_t* n_active,
                             float* y, void* ws, uint32_t flags, int32_t* counters, hipStream_t s) {
  switch (b) {
    case 1: return sparse_mlp_b<1>(w_gate, w_up, w_down_t, k, d, x, idx, n_active, y, ws, flags, counters, s);
    case 2: return sparse_mlp_b<2>(w_gate, w_up, w_down_t, k, d, x, idx, n_active, y, ws, flags, counters, s);
    case 3: return sparse_mlp_b<3>(w_gate, w_up, w_down_t, k, d, x, idx, n_active, y, ws, flags, counters, s);
    case 4: return sparse_mlp_b<4>(w_gate, w_up, w_down_t, k, d, x, idx, n_active, y, ws, flags, counters, s);
    case 5: return sparse_mlp_b<5>(w_gate, w_up, w_down_t, k, d, x, idx, n_active, y, ws, flags, counters, s);
    case 6: return sparse_mlp_b<6>(w_gate, w_up, w_down_t, k, d, x, idx, n_active, y, ws, flags, counters, s);
    case 7: return sparse_mlp_b<7>(w_gate, w_up, w_down_t, k, d, x, idx, n_active, y, ws, flags, counters, s);
    case 8: return sparse_mlp_b<8>(w_gate, w_up, w_down_t, k, d, x, idx, n_active, y, ws, flags, counters, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace si
