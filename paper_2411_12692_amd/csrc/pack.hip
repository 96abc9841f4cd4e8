// Load-time preprocessing: sign packing of W_gate (Section IV-B 1) and the
// transpose of W_down (Section IV-B 4).
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

__global__ __launch_bounds__(256) void k_signs_to_canonical(const uint32_t* __restrict__ signs, int k,
                                                            int d, uint32_t* __restrict__ out) {
  const int W = d >> 5;
  const int kpad = (k + kRowGroup - 1) / kRowGroup * kRowGroup;
  const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (size_t)k * W) return;
  const int i = (int)(t / W), wd = (int)(t % W);
  out[t] = signs[packed_index(i, wd, kpad)];
}

// out[c][r] = in[r][c] for a rows x cols fp16 matrix, 64x64 tiles through LDS.
__global__ __launch_bounds__(256) void k_transpose(const uint16_t* __restrict__ in, int rows, int cols,
                                                   uint16_t* __restrict__ out) {
  __shared__ uint16_t tile[64][65];
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
  k_transpose<<<grid, 256, 0, s>>>(in, rows, cols, out);
  return hipGetLastError();
}

}  // namespace si
