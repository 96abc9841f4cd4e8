// Host-side launchers of the SparseInfer kernels.  Arguments are validated
// by the caller (api.hip); these only enqueue work and report launch errors.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace si {

hipError_t launch_pack_signs(const uint16_t* w_gate, int k, int d, uint32_t* signs, hipStream_t s);
hipError_t launch_signs_to_canonical(const uint32_t* signs, int k, int d, uint32_t* out, hipStream_t s);
hipError_t launch_transpose(const uint16_t* in, int rows, int cols, uint16_t* out, hipStream_t s);

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

// The whole path of one layer in one kernel (layer.hip).  Only valid when
// layer_supported(k, d, b); `margin` gates the speculative row requests.
bool layer_supported(int k, int d, int b);
hipError_t launch_layer(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up,
                        const uint16_t* w_down_t, int k, int d, const uint16_t* x, int b, int T, int margin,
                        uint8_t* mask, int32_t* idx, int32_t* n_out, float* y, void* ws, uint32_t flags,
                        int32_t* counters, hipStream_t s);

// mask -> ascending kept list and count (single block).
hipError_t launch_compact(const uint8_t* mask, int k, int32_t* idx, int32_t* n_out, hipStream_t s);

// Sparse gate/up (+ReLU, product, actual sparsity) and sparse down.
hipError_t launch_sparse_mlp(const uint16_t* w_gate, const uint16_t* w_up, const uint16_t* w_down_t,
                             int k, int d, const uint16_t* x, int b, const int32_t* idx,
                             const int32_t* n_active, float* y, void* ws, uint32_t flags,
                             int32_t* counters, hipStream_t s);

}  // namespace si
