// Host-side launchers of the SparseInfer kernels.  Arguments are validated
// by the caller (api.hip); these only enqueue work and report launch errors.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace si {

constexpr int kMaxDevices = 64;

// A value computed once per device on first use there (grid sizes, kernel
// attributes): computed into a local and published with one atomic store, so
// that concurrent first calls from several host threads each compute the same
// value and none reads a half-made one.  `compute(dev)` runs with `dev`
// current and returns -1 on a HIP error (nothing is cached, 0 is returned).
template <class F>
inline int per_device_once(std::atomic<int> (&cache)[kMaxDevices], F compute) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  const int c = cache[dev].load(std::memory_order_acquire);
  if (c != 0) return c - 1;
  const int v = compute(dev);
  if (v < 0) return 0;
  cache[dev].store(v + 1, std::memory_order_release);
  return v;
}

hipError_t launch_pack_signs(const uint16_t* w_gate, int k, int d, uint32_t* signs, hipStream_t s);
hipError_t launch_signs_to_canonical(const uint32_t* signs, int k, int d, uint32_t* out, hipStream_t s);
hipError_t launch_transpose(const uint16_t* in, int rows, int cols, uint16_t* out, hipStream_t s);
hipError_t launch_transpose_i8(const int8_t* in, int rows, int cols, int8_t* out, hipStream_t s);
hipError_t launch_pack_signs_i8(const int8_t* w_gate, int k, int d, uint32_t* signs, hipStream_t s);
hipError_t launch_quantize_rows(const uint16_t* w, int rows, int n, int8_t* q, float* scale, hipStream_t s);

// Predictor: x-sign pack, XOR/popcount, Eq. (2) via threshold T, mask and
// ordered compaction.  `ws` is the workspace base.
hipError_t launch_predict(const uint32_t* signs, int k, int d, const uint16_t* x, int b, int T,
                          uint8_t* mask, int32_t* idx, int32_t* n_out, void* ws, hipStream_t s);

// Predictor fused with the sparse gate/up GEMV of the kept rows (h3 per row
// into the workspace; y zeroed for the down-projection's atomics).
hipError_t launch_predict_gate_up(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up, int k,
                                  int d, const uint16_t* x, int b, int T, uint8_t* mask, int32_t* idx,
                                  int32_t* n_out, float* y, void* ws, uint32_t flags, hipStream_t s);

// Down-projection over the kept list; `slots` per-block work counts are
// summed into `counters` when it is not NULL.
hipError_t launch_down(const uint16_t* w_down_t, int k, int d, int b, const int32_t* idx, const int32_t* n_active,
                       float* y, void* ws, int slots, uint32_t flags, int32_t* counters, hipStream_t s);

// The path of one layer in one kernel (layer.hip).  The kept rows come from
// the packed signs (predict: signs set, mask_in and idx_in NULL), from a
// caller's mask (mask_in set) or from a caller's list (idx_in and n_in set);
// y NULL runs the predictor alone.  Only valid when layer_supported(k, d, b).
struct LayerCall {
  const uint32_t* signs = nullptr;
  const uint16_t* w_gate = nullptr;
  const uint16_t* w_up = nullptr;
  const uint16_t* w_down_t = nullptr;
  const uint16_t* x = nullptr;
  const uint8_t* mask_in = nullptr;
  const int32_t* idx_in = nullptr;
  const int32_t* n_in = nullptr;
  int k = 0, d = 0, b = 1;
  int T = 0;       // integer threshold of Eq. (2) (predict)
  int margin = 0;  // rows with N_neg < T - margin are treated as surely kept (speculative requests)
  uint32_t flags = 0;
  uint8_t* mask = nullptr;   // predict: the mask
  int32_t* idx = nullptr;    // predict and mask: the kept list
  int32_t* n_out = nullptr;  // predict and mask: its length
  float* y = nullptr;
  void* ws = nullptr;
  int32_t* counters = nullptr;
  // decoder-block mode (row-owning kernel only): x = fp16(RMSNorm(h) * norm_w)
  // is formed in the kernel (x must be NULL) and y = h + MLP(x)
  const float* h = nullptr;
  const float* norm_w = nullptr;
  float eps = 0.f;
  // INT8 form (row-owning kernel only): w_gate, w_up and w_down_t hold INT8
  // values with scales per row of W_gate / W_up and per column of y
  bool i8 = false;
  const float* s_gate = nullptr;
  const float* s_up = nullptr;
  const float* s_down = nullptr;
};
bool layer_supported(int k, int d, int b);
hipError_t launch_layer(const LayerCall& c, hipStream_t s);

// The row-owning single-launch kernel (owned.hip) for predict and mask
// calls (idx_in must be NULL); idx, mask and n_out are each written when not
// NULL.  Only valid when owned_supported(k, d, b).
bool owned_supported(int k, int d, int b);
hipError_t launch_owned(const LayerCall& c, hipStream_t s);

// Per-row h3 of the last MLP call made with workspace `ws` -> out[k][b]
// (kept rows of `mask`; 0 elsewhere; NaN where the call left no value).
hipError_t launch_read_h3(const void* ws, int k, int b, const uint8_t* mask, float* out, hipStream_t s);

// Streaming read of `bytes` (a multiple of 16) at `buf` (diagnostic).
hipError_t launch_read_probe(const void* buf, size_t bytes, uint32_t* sink, hipStream_t s);

// mask -> ascending kept list and count (single block).
hipError_t launch_compact(const uint8_t* mask, int k, int32_t* idx, int32_t* n_out, hipStream_t s);

// ascending kept list and count -> [k] mask (single block).
hipError_t launch_list_to_mask(const int32_t* idx, const int32_t* n_in, int k, uint8_t* mask, hipStream_t s);

// Sparse gate/up (+ReLU, product, actual sparsity) and sparse down.
hipError_t launch_sparse_mlp(const uint16_t* w_gate, const uint16_t* w_up, const uint16_t* w_down_t,
                             int k, int d, const uint16_t* x, int b, const int32_t* idx,
                             const int32_t* n_active, float* y, void* ws, uint32_t flags,
                             int32_t* counters, hipStream_t s);

}  // namespace si
