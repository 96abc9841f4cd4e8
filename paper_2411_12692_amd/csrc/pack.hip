// Load-time preprocessing: sign packing of W_gate (Section IV-B 1), the
// transpose of W_down (Section IV-B 4), and for INT8 weights their symmetric
// per-row quantization and the packing of their MSBs (Section IV-A).
//
// Packed-sign layout (private to the library).  A unit is 4 consecutive
// 32-bit words (128 elements) of one row; units are stored unit-major over
// the rows, which are padded to a multiple of 64 (kpad):
//     word (row i, w) -> [unit w/4][row i][w%4]
// so that unit q of any run of consecutive rows is one contiguous piece of
// memory, read with one 16-byte load per lane (lane = row): 1 KB for a
// 64-row group, R * 16 bytes for a block's R rows.  Bit j of word w is the
// sign of element 32*w + j.  Padding rows are all zero.
#include "si_device.h"
#include "si_launch.h"

namespace si {

__device__ inline size_t packed_index(int i, int w, int kpad) {
  return ((size_t)(w >> 2) * kpad + i) * 4 + (w & 3);
}

// One thread per (row, word): reads 32 consecutive fp16 (64 bytes; adjacent
// threads read adjacent words of a row).
__global__ __launch_bounds__(256) void k_pack_signs(const uint16_t* __restrict__ w, int k, int d,
                                                    uint32_t* __restrict__ signs) {
  const int W = d >> 5;
  const int kpad = (k + kRowGroup - 1) / kRowGroup * kRowGroup;
  const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (size_t)kpad * W) return;
  const int i = (int)(t / W), wd = (int)(t % W);
  uint32_t word = 0;
  if (i < k) word = sign_word(reinterpret_cast<const u32x4*>(w + (size_t)i * d + 32 * wd));
  signs[packed_index(i, wd, kpad)] = word;
}

// Sign word of 32 consecutive INT8 values (bit j = MSB of byte j).
__device__ inline uint32_t sign_word_i8(const u32x4* p) {
  uint32_t word = 0;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const u32x4 v = p[h];
    const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) word |= ((w4[i] >> (8 * j + 7)) & 1u) << (16 * h + 4 * i + j);
  }
  return word;
}

// The INT8 form of k_pack_signs: one thread per (row, word), 32 bytes each.
__global__ __launch_bounds__(256) void k_pack_signs_i8(const int8_t* __restrict__ w, int k, int d,
                                                       uint32_t* __restrict__ signs) {
  const int W = d >> 5;
  const int kpad = (k + kRowGroup - 1) / kRowGroup * kRowGroup;
  const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (size_t)kpad * W) return;
  const int i = (int)(t / W), wd = (int)(t % W);
  uint32_t word = 0;
  if (i < k) word = sign_word_i8(reinterpret_cast<const u32x4*>(w + (size_t)i * d + 32 * wd));
  signs[packed_index(i, wd, kpad)] = word;
}

// Symmetric per-row INT8 quantization, one block per row of n fp16 values:
// scale = max |w| / 127 and q = rint(w / scale) (ties to even, clamped to
// +-127), in float32 with correctly rounded division; a row of zeros gets
// scale 0 and q = 0.
__global__ __launch_bounds__(256) void k_quantize_rows(const uint16_t* __restrict__ w, int n,
                                                       int8_t* __restrict__ q, float* __restrict__ scale) {
  __shared__ float wmax[4];
  const size_t base = (size_t)blockIdx.x * n;
  const int tid = threadIdx.x;
  float m = 0.f;
  for (int j = tid; j < n; j += 256) m = fmaxf(m, fabsf((float)__builtin_bit_cast(_Float16, w[base + j])));
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, kWave));
  if ((tid & 63) == 0) wmax[tid >> 6] = m;
  __syncthreads();
  const float amax = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
  const float s = amax / 127.0f;
  for (int j = tid; j < n; j += 256) {
    float v = 0.f;
    if (s > 0.f) v = fminf(fmaxf(rintf((float)__builtin_bit_cast(_Float16, w[base + j]) / s), -127.f), 127.f);
    q[base + j] = (int8_t)(int)v;
  }
  if (tid == 0) scale[blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_signs_to_canonical(const uint32_t* __restrict__ signs, int k,
                                                            int d, uint32_t* __restrict__ out) {
  const int W = d >> 5;
  const int kpad = (k + kRowGroup - 1) / kRowGroup * kRowGroup;
  const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (size_t)k * W) return;
  const int i = (int)(t / W), wd = (int)(t % W);
  out[t] = signs[packed_index(i, wd, kpad)];
}

// out[c][r] = in[r][c] for a rows x cols matrix (fp16 or INT8 elements),
// 64x64 tiles through LDS.
template <typename E>
__global__ __launch_bounds__(256) void k_transpose(const E* __restrict__ in, int rows, int cols,
                                                   E* __restrict__ out) {
  __shared__ E tile[64][65];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
  for (int rr = ty; rr < 64; rr += 4) {
    const int r = r0 + rr, c = c0 + tx;
    if (r < rows && c < cols) tile[rr][tx] = in[(size_t)r * cols + c];
  }
  __syncthreads();
  for (int cc = ty; cc < 64; cc += 4) {
    const int c = c0 + cc, r = r0 + tx;
    if (c < cols && r < rows) out[(size_t)c * rows + r] = tile[tx][cc];
  }
}

hipError_t launch_pack_signs(const uint16_t* w_gate, int k, int d, uint32_t* signs, hipStream_t s) {
  const int kpad = (k + kRowGroup - 1) / kRowGroup * kRowGroup;
  const size_t threads = (size_t)kpad * (d >> 5);
  const unsigned grid = (unsigned)((threads + 255) / 256);
  k_pack_signs<<<grid, 256, 0, s>>>(w_gate, k, d, signs);
  return hipGetLastError();
}

hipError_t launch_signs_to_canonical(const uint32_t* signs, int k, int d, uint32_t* out, hipStream_t s) {
  const size_t threads = (size_t)k * (d >> 5);
  const unsigned grid = (unsigned)((threads + 255) / 256);
  k_signs_to_canonical<<<grid, 256, 0, s>>>(signs, k, d, out);
  return hipGetLastError();
}

hipError_t launch_transpose(const uint16_t* in, int rows, int cols, uint16_t* out, hipStream_t s) {
  dim3 grid((cols + 63) / 64, (rows + 63) / 64);
  k_transpose<uint16_t><<<grid, 256, 0, s>>>(in, rows, cols, out);
  return hipGetLastError();
}

hipError_t launch_transpose_i8(const int8_t* in, int rows, int cols, int8_t* out, hipStream_t s) {
  dim3 grid((cols + 63) / 64, (rows + 63) / 64);
  k_transpose<int8_t><<<grid, 256, 0, s>>>(in, rows, cols, out);
  return hipGetLastError();
}

hipError_t launch_pack_signs_i8(const int8_t* w_gate, int k, int d, uint32_t* signs, hipStream_t s) {
  const int kpad = (k + kRowGroup - 1) / kRowGroup * kRowGroup;
  const size_t threads = (size_t)kpad * (d >> 5);
  const unsigned grid = (unsigned)((threads + 255) / 256);
  k_pack_signs_i8<<<grid, 256, 0, s>>>(w_gate, k, d, signs);
  return hipGetLastError();
}

hipError_t launch_quantize_rows(const uint16_t* w, int rows, int n, int8_t* q, float* scale, hipStream_t s) {
  k_quantize_rows<<<rows, 256, 0, s>>>(w, n, q, scale);
  return hipGetLastError();
}

}  // namespace si
