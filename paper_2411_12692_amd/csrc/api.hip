// C ABI of libsparseinfer: argument validation, Eq. (2) threshold, launches.
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "../../include/sparseinfer.h"
#include "si_device.h"
#include "si_launch.h"

namespace {

thread_local char g_err[512] = "";

int32_t threshold(float alpha, int d);

// Rows with N_neg < T - margin count as surely active: their W_up and
// W_down^T requests go out with the W_gate row, before the gate result.
// Products of the signs are symmetric (Section IV-A), so a row whose signs
// agree with the token's on at least half of the elements (the rows Eq. (2)
// keeps at alpha = 1: N_neg < T(1)) is more likely positive than not, and a
// row kept only because alpha > 1 is more likely zero: those wait for their
// gate value, so a larger alpha never adds speculative reads.  With 2-4
// tokens the kept rows of one token are confident only d/16 below that (a
// row kept by a fresh token sits near N_neg = d/2); with 5-8 tokens the union
// of the tokens' kept sets is nearly every row and nearly every one is active
// for some token, so every kept row is treated as confident.
int confident_margin(int d, int b, int T) {
  if (b > 4) return 0;
  const int T1 = threshold(1.0f, d);
  return (T > T1 ? T - T1 : 0) + (b == 1 ? 0 : d / 16);
}

si_status fail(si_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

si_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return SI_OK;
  return fail(SI_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQUIRE_PTR(p) \
  if (!(p)) return fail(SI_ERR_NULL, "%s is NULL", #p)
#define REQUIRE_ALIGNED(p) \
  if ((p) && !aligned16(p)) return fail(SI_ERR_ALIGN, "%s is not 16-byte aligned", #p)

si_status check_kd(int k, int d) {
  if (k < 1 || k > (1 << 24)) return fail(SI_ERR_SHAPE, "k=%d outside [1, 2^24]", k);
  if (d < 128 || d > si::kMaxD || d % 128 != 0)
    return fail(SI_ERR_SHAPE, "d=%d must be a multiple of 128 in [128, %d]", d, si::kMaxD);
  return SI_OK;
}

si_status check_b(int b) {
  if (b < 1 || b > si::kMaxB) return fail(SI_ERR_SHAPE, "b=%d outside [1, %d]", b, si::kMaxB);
  return SI_OK;
}

si_status check_ws(const void* ws, size_t bytes, int k, int b) {
  REQUIRE_PTR(ws);
  REQUIRE_ALIGNED(ws);
  const size_t need = si::ws_layout(k, b).total;
  if (bytes < need) return fail(SI_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", bytes, need);
  return SI_OK;
}

// Smallest N_neg in [0, d] for which alpha * (d - N_neg) < N_neg (Eq. (2)).
// Both sides are exact in double: alpha has 24 significant bits and d < 2^25.
int32_t threshold(float alpha, int d) {
  const double a = alpha;
  int lo = 0, hi = d;  // the predicate holds at N_neg = d (0 < d) and is monotone
  while (lo < hi) {
    const int mid = lo + (hi - lo) / 2;
    if (a * (double)(d - mid) < (double)mid)
      hi = mid;
    else
      lo = mid + 1;
  }
  return lo;
}

}  // namespace

extern "C" {

const char* si_last_error(void) { return g_err; }

const char* si_version(void) { return "sparseinfer-gfx950 0.1"; }

size_t si_signs_bytes(int k, int d) {
  if (check_kd(k, d) != SI_OK) return 0;
  const size_t kpad = (size_t)(k + si::kRowGroup - 1) / si::kRowGroup * si::kRowGroup;
  return kpad * (size_t)d / 8;
}

size_t si_workspace_bytes(int k, int d, int b) {
  if (check_kd(k, d) != SI_OK || check_b(b) != SI_OK) return 0;
  return si::ws_layout(k, b).total;
}

si_status si_device_error_status(uint32_t bits) {
  if (bits == 0) return SI_OK;
  if (bits & ~(si::kErrLookbackSpin | si::kErrRow)) return fail(SI_ERR_ARG, "unknown device error bits 0x%x", bits);
  if (bits & si::kErrLookbackSpin)
    return fail(SI_ERR_TIMEOUT, "a wait inside a kernel gave up: not every block of a single-launch call was resident");
  return fail(SI_ERR_LIST, "a caller's active_idx held a row outside [0, k)");
}

si_status si_workspace_check(void* workspace, size_t workspace_bytes, void* stream) {
  REQUIRE_PTR(workspace);
  REQUIRE_ALIGNED(workspace);
  if (workspace_bytes < si::H_WORDS * sizeof(uint32_t))
    return fail(SI_ERR_WORKSPACE, "workspace of %zu bytes is smaller than its header", workspace_bytes);
  hipStream_t st = (hipStream_t)stream;
  if (si_status s = hip_status(hipStreamSynchronize(st), "stream synchronize")) return s;
  uint32_t bits = 0;
  const uint32_t* hdr = static_cast<const uint32_t*>(workspace);
  if (si_status s = hip_status(hipMemcpy(&bits, hdr + si::H_ERR, sizeof bits, hipMemcpyDeviceToHost), "read error word"))
    return s;
  const si_status st_bits = si_device_error_status(bits);
  if (st_bits == SI_OK) return SI_OK;
  char msg[sizeof g_err];
  snprintf(msg, sizeof msg, "%s", g_err);
  if (si_status s = hip_status(hipMemsetAsync(workspace, 0, workspace_bytes, st), "workspace reset")) return s;
  if (si_status s = hip_status(hipStreamSynchronize(st), "stream synchronize")) return s;
  return fail(st_bits, "%s (the workspace has been reset)", msg);
}

si_status si_read_h3(const void* workspace, size_t workspace_bytes, int k, int d, int b, const uint8_t* mask,
                     float* h3, void* stream) {
  REQUIRE_PTR(mask);
  REQUIRE_PTR(h3);
  REQUIRE_ALIGNED(mask);
  REQUIRE_ALIGNED(h3);
  if (si_status s = check_kd(k, d)) return s;
  if (si_status s = check_b(b)) return s;
  if (si_status s = check_ws(workspace, workspace_bytes, k, b)) return s;
  return hip_status(si::launch_read_h3(workspace, k, b, mask, h3, (hipStream_t)stream), "read_h3 launch");
}

si_status si_read_bandwidth_probe(const void* buf, size_t bytes, uint32_t* sink, void* stream) {
  REQUIRE_PTR(buf);
  REQUIRE_PTR(sink);
  REQUIRE_ALIGNED(buf);
  if (bytes == 0 || bytes % 16 != 0) return fail(SI_ERR_SHAPE, "bytes=%zu must be a positive multiple of 16", bytes);
  return hip_status(si::launch_read_probe(buf, bytes, sink, (hipStream_t)stream), "read probe launch");
}

int si_single_launch(int k, int d, int b) {
  if (check_kd(k, d) != SI_OK || check_b(b) != SI_OK) return 0;
  return si::layer_supported(k, d, b) && si::owned_supported(k, d, b) ? 1 : 0;
}

int32_t si_alpha_threshold(float alpha, int d) {
  if (std::isnan(alpha) || alpha < 0.0f) return -1;
  if (d < 1 || d > (1 << 24)) return -1;
  if (std::isinf(alpha)) return d + 1;
  return threshold(alpha, d);
}

si_status si_pack_signs(const uint16_t* w_gate, int k, int d, uint32_t* signs, void* stream) {
  REQUIRE_PTR(w_gate);
  REQUIRE_PTR(signs);
  REQUIRE_ALIGNED(w_gate);
  REQUIRE_ALIGNED(signs);
  if (si_status s = check_kd(k, d)) return s;
  return hip_status(si::launch_pack_signs(w_gate, k, d, signs, (hipStream_t)stream), "pack_signs launch");
}

si_status si_signs_to_canonical(const uint32_t* signs, int k, int d, uint32_t* out, void* stream) {
  REQUIRE_PTR(signs);
  REQUIRE_PTR(out);
  REQUIRE_ALIGNED(signs);
  REQUIRE_ALIGNED(out);
  if (si_status s = check_kd(k, d)) return s;
  return hip_status(si::launch_signs_to_canonical(signs, k, d, out, (hipStream_t)stream),
                    "signs_to_canonical launch");
}

si_status si_transpose_down(const uint16_t* w_down, int d, int k, uint16_t* w_down_t, void* stream) {
  REQUIRE_PTR(w_down);
  REQUIRE_PTR(w_down_t);
  REQUIRE_ALIGNED(w_down);
  REQUIRE_ALIGNED(w_down_t);
  if (si_status s = check_kd(k, d)) return s;
  const uintptr_t a = reinterpret_cast<uintptr_t>(w_down), c = reinterpret_cast<uintptr_t>(w_down_t);
  const uintptr_t n = (uintptr_t)k * (uintptr_t)d * 2u;
  if (a < c + n && c < a + n) return fail(SI_ERR_SHAPE, "w_down and w_down_t overlap");
  return hip_status(si::launch_transpose(w_down, d, k, w_down_t, (hipStream_t)stream), "transpose launch");
}

si_status si_predict(const uint32_t* signs, int k, int d, const uint16_t* x, int b, float alpha, uint8_t* mask,
                     int32_t* active_idx, int32_t* n_active, void* workspace, size_t workspace_bytes,
                     void* stream) {
  REQUIRE_PTR(signs);
  REQUIRE_PTR(x);
  REQUIRE_PTR(mask);
  REQUIRE_ALIGNED(signs);
  REQUIRE_ALIGNED(x);
  REQUIRE_ALIGNED(mask);
  REQUIRE_ALIGNED(active_idx);
  REQUIRE_ALIGNED(n_active);
  if (si_status s = check_kd(k, d)) return s;
  if (si_status s = check_b(b)) return s;
  if (std::isnan(alpha) || alpha < 0.0f) return fail(SI_ERR_ALPHA, "alpha=%g must be >= 0 (or +inf)", (double)alpha);
  if (si_status s = check_ws(workspace, workspace_bytes, k, b)) return s;
  const int T = si_alpha_threshold(alpha, d);
  if (si::owned_supported(k, d, b)) {
    si::LayerCall c;
    c.signs = signs;
    c.x = x;
    c.k = k;
    c.d = d;
    c.b = b;
    c.T = T;
    c.mask = mask;
    c.idx = active_idx;
    c.n_out = n_active;
    c.ws = workspace;
    return hip_status(si::launch_owned(c, (hipStream_t)stream), "predict launch");
  }
  return hip_status(si::launch_predict(signs, k, d, x, b, T, mask, active_idx, n_active, workspace,
                                       (hipStream_t)stream),
                    "predict launch");
}

}  // extern "C"

namespace {

// si_sparse_mlp and si_sparse_relu_mlp (w_up == nullptr: no W_up).
si_status sparse_mlp_impl(const uint16_t* w_gate, const uint16_t* w_up, const uint16_t* w_down_t, int k, int d,
                          const uint16_t* x, int b, const uint8_t* mask, const int32_t* active_idx,
                          const int32_t* n_active, float* y, void* workspace, size_t workspace_bytes,
                          uint32_t flags, int32_t* counters, void* stream) {
  REQUIRE_PTR(w_gate);
  REQUIRE_PTR(w_down_t);
  REQUIRE_PTR(x);
  REQUIRE_PTR(y);
  REQUIRE_ALIGNED(w_gate);
  REQUIRE_ALIGNED(w_up);
  REQUIRE_ALIGNED(w_down_t);
  REQUIRE_ALIGNED(x);
  REQUIRE_ALIGNED(y);
  REQUIRE_ALIGNED(mask);
  REQUIRE_ALIGNED(active_idx);
  REQUIRE_ALIGNED(n_active);
  REQUIRE_ALIGNED(counters);
  if ((active_idx == nullptr) != (n_active == nullptr))
    return fail(SI_ERR_NULL, "active_idx and n_active must both be given or both be NULL");
  if (!active_idx && !mask) return fail(SI_ERR_NULL, "mask is NULL and no active_idx was given");
  if (flags & ~(SI_NO_AS | SI_NO_SPECULATION)) return fail(SI_ERR_FLAGS, "unknown flags 0x%x", flags);
  if (si_status s = check_kd(k, d)) return s;
  if (si_status s = check_b(b)) return s;
  if (si_status s = check_ws(workspace, workspace_bytes, k, b)) return s;
  hipStream_t st = (hipStream_t)stream;
  const si::WsLayout L = si::ws_layout(k, b);
  char* base = static_cast<char*>(workspace);
  if (active_idx && b > 4 && si::owned_supported(k, d, b)) {
    // With 5-8 tokens the list-driven kernel (16 waves per block, so at most
    // 128 registers per lane) spills; the list becomes a mask in the
    // workspace and the row-owning kernel (8 waves) runs in mask mode.
    uint8_t* wmask = reinterpret_cast<uint8_t*>(base + L.mask);
    if (si_status s = hip_status(si::launch_list_to_mask(active_idx, n_active, k, wmask, st), "list launch"))
      return s;
    mask = wmask;
    active_idx = nullptr;
    n_active = nullptr;
  }
  if (active_idx ? si::layer_supported(k, d, b) : si::owned_supported(k, d, b)) {
    si::LayerCall c;
    c.w_gate = w_gate;
    c.w_up = w_up;
    c.w_down_t = w_down_t;
    c.x = x;
    c.k = k;
    c.d = d;
    c.b = b;
    c.flags = flags;
    c.y = y;
    c.ws = workspace;
    c.counters = counters;
    if (active_idx) {
      c.idx_in = active_idx;
      c.n_in = n_active;
      return hip_status(si::launch_layer(c, st), "sparse_mlp launch");
    }
    c.mask_in = mask;
    c.n_out = reinterpret_cast<int32_t*>(base) + si::H_N_INTERNAL;  // n_gate of the counters
    return hip_status(si::launch_owned(c, st), "sparse_mlp launch");
  }
  if (!active_idx) {
    int32_t* idx = reinterpret_cast<int32_t*>(base + L.idx);
    int32_t* n = reinterpret_cast<int32_t*>(base) + si::H_N_INTERNAL;
    if (si_status s = hip_status(si::launch_compact(mask, k, idx, n, st), "compact launch")) return s;
    active_idx = idx;
    n_active = n;
  }
  return hip_status(si::launch_sparse_mlp(w_gate, w_up, w_down_t, k, d, x, b, active_idx, n_active, y, workspace,
                                          flags, counters, st),
                    "sparse_mlp launch");
}

// si_predict_sparse_mlp and si_predict_sparse_relu_mlp (w_up == nullptr).
si_status predict_sparse_mlp_impl(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up,
                                  const uint16_t* w_down_t, int k, int d, const uint16_t* x, int b, float alpha,
                                  uint8_t* mask, int32_t* active_idx, int32_t* n_active, float* y, void* workspace,
                                  size_t workspace_bytes, uint32_t flags, int32_t* counters, void* stream) {
  REQUIRE_PTR(signs);
  REQUIRE_PTR(w_gate);
  REQUIRE_PTR(w_down_t);
  REQUIRE_PTR(x);
  REQUIRE_PTR(y);
  REQUIRE_ALIGNED(signs);
  REQUIRE_ALIGNED(w_gate);
  REQUIRE_ALIGNED(w_up);
  REQUIRE_ALIGNED(w_down_t);
  REQUIRE_ALIGNED(x);
  REQUIRE_ALIGNED(y);
  REQUIRE_ALIGNED(mask);
  REQUIRE_ALIGNED(active_idx);
  REQUIRE_ALIGNED(n_active);
  REQUIRE_ALIGNED(counters);
  if (flags & ~(SI_NO_AS | SI_NO_SPECULATION)) return fail(SI_ERR_FLAGS, "unknown flags 0x%x", flags);
  if (si_status s = check_kd(k, d)) return s;
  if (si_status s = check_b(b)) return s;
  if (std::isnan(alpha) || alpha < 0.0f) return fail(SI_ERR_ALPHA, "alpha=%g must be >= 0 (or +inf)", (double)alpha);
  if (si_status s = check_ws(workspace, workspace_bytes, k, b)) return s;
  const si::WsLayout L = si::ws_layout(k, b);
  char* base = static_cast<char*>(workspace);
  if (!n_active) n_active = reinterpret_cast<int32_t*>(base) + si::H_N_INTERNAL;
  hipStream_t st = (hipStream_t)stream;
  const int T = si_alpha_threshold(alpha, d);
  if (si::owned_supported(k, d, b)) {
    si::LayerCall c;
    c.signs = signs;
    c.w_gate = w_gate;
    c.w_up = w_up;
    c.w_down_t = w_down_t;
    c.x = x;
    c.k = k;
    c.d = d;
    c.b = b;
    c.T = T;
    c.margin = confident_margin(d, b, c.T);
    c.flags = flags;
    c.mask = mask;
    c.idx = active_idx;
    c.n_out = n_active;
    c.y = y;
    c.ws = workspace;
    c.counters = counters;
    return hip_status(si::launch_owned(c, st), "layer launch");
  }
  if (!mask) mask = reinterpret_cast<uint8_t*>(base + L.mask);
  if (!active_idx) active_idx = reinterpret_cast<int32_t*>(base + L.idx);
  if (si_status s = hip_status(si::launch_predict_gate_up(signs, w_gate, w_up, k, d, x, b, T, mask, active_idx,
                                                          n_active, y, workspace, flags, st),
                               "predict/gate-up launch"))
    return s;
  return hip_status(si::launch_down(w_down_t, k, d, b, active_idx, n_active, y, workspace, si::row_groups(k), flags,
                                    counters, st),
                    "down-projection launch");
}

}  // namespace

extern "C" {

si_status si_sparse_mlp(const uint16_t* w_gate, const uint16_t* w_up, const uint16_t* w_down_t, int k, int d,
                        const uint16_t* x, int b, const uint8_t* mask, const int32_t* active_idx,
                        const int32_t* n_active, float* y, void* workspace, size_t workspace_bytes,
                        uint32_t flags, int32_t* counters, void* stream) {
  REQUIRE_PTR(w_up);
  return sparse_mlp_impl(w_gate, w_up, w_down_t, k, d, x, b, mask, active_idx, n_active, y, workspace,
                         workspace_bytes, flags, counters, stream);
}

si_status si_sparse_relu_mlp(const uint16_t* w_fc1, const uint16_t* w_down_t, int k, int d, const uint16_t* x,
                             int b, const uint8_t* mask, const int32_t* active_idx, const int32_t* n_active,
                             float* y, void* workspace, size_t workspace_bytes, uint32_t flags, int32_t* counters,
                             void* stream) {
  return sparse_mlp_impl(w_fc1, nullptr, w_down_t, k, d, x, b, mask, active_idx, n_active, y, workspace,
                         workspace_bytes, flags, counters, stream);
}

si_status si_predict_sparse_mlp(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up,
                                const uint16_t* w_down_t, int k, int d, const uint16_t* x, int b, float alpha,
                                uint8_t* mask, int32_t* active_idx, int32_t* n_active, float* y, void* workspace,
                                size_t workspace_bytes, uint32_t flags, int32_t* counters, void* stream) {
  REQUIRE_PTR(w_up);
  return predict_sparse_mlp_impl(signs, w_gate, w_up, w_down_t, k, d, x, b, alpha, mask, active_idx, n_active, y,
                                 workspace, workspace_bytes, flags, counters, stream);
}

si_status si_predict_sparse_relu_mlp(const uint32_t* signs, const uint16_t* w_fc1, const uint16_t* w_down_t, int k,
                                     int d, const uint16_t* x, int b, float alpha, uint8_t* mask,
                                     int32_t* active_idx, int32_t* n_active, float* y, void* workspace,
                                     size_t workspace_bytes, uint32_t flags, int32_t* counters, void* stream) {
  return predict_sparse_mlp_impl(signs, w_fc1, nullptr, w_down_t, k, d, x, b, alpha, mask, active_idx, n_active,
                                 y, workspace, workspace_bytes, flags, counters, stream);
}

si_status si_rmsnorm_predict_sparse_mlp(const float* h, const float* norm_w, float eps, const uint32_t* signs,
                                        const uint16_t* w_gate, const uint16_t* w_up, const uint16_t* w_down_t,
                                        int k, int d, int b, float alpha, uint8_t* mask, int32_t* active_idx,
                                        int32_t* n_active, float* y, void* workspace, size_t workspace_bytes,
                                        uint32_t flags, int32_t* counters, void* stream) {
  REQUIRE_PTR(h);
  REQUIRE_PTR(norm_w);
  REQUIRE_PTR(signs);
  REQUIRE_PTR(w_gate);
  REQUIRE_PTR(w_down_t);
  REQUIRE_PTR(y);
  REQUIRE_ALIGNED(h);
  REQUIRE_ALIGNED(norm_w);
  REQUIRE_ALIGNED(signs);
  REQUIRE_ALIGNED(w_gate);
  REQUIRE_ALIGNED(w_up);
  REQUIRE_ALIGNED(w_down_t);
  REQUIRE_ALIGNED(y);
  REQUIRE_ALIGNED(mask);
  REQUIRE_ALIGNED(active_idx);
  REQUIRE_ALIGNED(n_active);
  REQUIRE_ALIGNED(counters);
  if (flags & ~(SI_NO_AS | SI_NO_SPECULATION)) return fail(SI_ERR_FLAGS, "unknown flags 0x%x", flags);
  if (si_status s = check_kd(k, d)) return s;
  if (si_status s = check_b(b)) return s;
  if (std::isnan(alpha) || alpha < 0.0f) return fail(SI_ERR_ALPHA, "alpha=%g must be >= 0 (or +inf)", (double)alpha);
  if (!std::isfinite(eps) || eps < 0.0f) return fail(SI_ERR_ARG, "eps=%g must be finite and >= 0", (double)eps);
  const uintptr_t ha = reinterpret_cast<uintptr_t>(h), ya = reinterpret_cast<uintptr_t>(y);
  const uintptr_t nb = (uintptr_t)b * (uintptr_t)d * sizeof(float);
  if (ha < ya + nb && ya < ha + nb) return fail(SI_ERR_ARG, "h and y overlap");
  if (si_status s = check_ws(workspace, workspace_bytes, k, b)) return s;
  if (!si::owned_supported(k, d, b))
    return fail(SI_ERR_SHAPE, "k=%d d=%d b=%d: the decoder-block call needs the single-launch path", k, d, b);
  char* base = static_cast<char*>(workspace);
  si::LayerCall c;
  c.signs = signs;
  c.w_gate = w_gate;
  c.w_up = w_up;
  c.w_down_t = w_down_t;
  c.k = k;
  c.d = d;
  c.b = b;
  c.T = si_alpha_threshold(alpha, d);
  c.margin = confident_margin(d, b, c.T);
  c.flags = flags;
  c.mask = mask;
  c.idx = active_idx;
  c.n_out = n_active ? n_active : reinterpret_cast<int32_t*>(base) + si::H_N_INTERNAL;
  c.y = y;
  c.ws = workspace;
  c.counters = counters;
  c.h = h;
  c.norm_w = norm_w;
  c.eps = eps;
  return hip_status(si::launch_owned(c, (hipStream_t)stream), "decoder-block launch");
}

}  // extern "C"

// ---- INT8 weights ---------------------------------------------------------

namespace {

// si_sparse_mlp_i8 (mask given, predict == false) and si_predict_sparse_mlp_i8.
si_status int8_impl(bool predict, const uint32_t* signs, const int8_t* w_gate, const float* s_gate,
                    const int8_t* w_up, const float* s_up, const int8_t* w_down_t, const float* s_down, int k,
                    int d, const uint16_t* x, int b, float alpha, const uint8_t* mask_in, uint8_t* mask,
                    int32_t* active_idx, int32_t* n_active, float* y, void* workspace, size_t workspace_bytes,
                    uint32_t flags, int32_t* counters, void* stream) {
  if (predict) {
    REQUIRE_PTR(signs);
  } else {
    REQUIRE_PTR(mask_in);
  }
  REQUIRE_PTR(w_gate);
  REQUIRE_PTR(s_gate);
  REQUIRE_PTR(w_down_t);
  REQUIRE_PTR(s_down);
  REQUIRE_PTR(x);
  REQUIRE_PTR(y);
  if (w_up) REQUIRE_PTR(s_up);
  REQUIRE_ALIGNED(signs);
  REQUIRE_ALIGNED(w_gate);
  REQUIRE_ALIGNED(s_gate);
  REQUIRE_ALIGNED(w_up);
  REQUIRE_ALIGNED(s_up);
  REQUIRE_ALIGNED(w_down_t);
  REQUIRE_ALIGNED(s_down);
  REQUIRE_ALIGNED(x);
  REQUIRE_ALIGNED(y);
  REQUIRE_ALIGNED(mask_in);
  REQUIRE_ALIGNED(mask);
  REQUIRE_ALIGNED(active_idx);
  REQUIRE_ALIGNED(n_active);
  REQUIRE_ALIGNED(counters);
  if (flags & ~(SI_NO_AS | SI_NO_SPECULATION)) return fail(SI_ERR_FLAGS, "unknown flags 0x%x", flags);
  if (si_status s = check_kd(k, d)) return s;
  if (si_status s = check_b(b)) return s;
  if (predict && (std::isnan(alpha) || alpha < 0.0f))
    return fail(SI_ERR_ALPHA, "alpha=%g must be >= 0 (or +inf)", (double)alpha);
  if (si_status s = check_ws(workspace, workspace_bytes, k, b)) return s;
  if (!si::owned_supported(k, d, b))
    return fail(SI_ERR_SHAPE, "k=%d d=%d b=%d: INT8 weights need the single-launch path", k, d, b);
  char* base = static_cast<char*>(workspace);
  si::LayerCall c;
  c.signs = predict ? signs : nullptr;
  c.mask_in = predict ? nullptr : mask_in;
  c.w_gate = reinterpret_cast<const uint16_t*>(w_gate);
  c.w_up = reinterpret_cast<const uint16_t*>(w_up);
  c.w_down_t = reinterpret_cast<const uint16_t*>(w_down_t);
  c.i8 = true;
  c.s_gate = s_gate;
  c.s_up = w_up ? s_up : nullptr;
  c.s_down = s_down;
  c.x = x;
  c.k = k;
  c.d = d;
  c.b = b;
  if (predict) {
    c.T = si_alpha_threshold(alpha, d);
    c.margin = confident_margin(d, b, c.T);
    c.mask = mask;
    c.idx = active_idx;
  }
  c.n_out = predict && n_active ? n_active : reinterpret_cast<int32_t*>(base) + si::H_N_INTERNAL;
  c.flags = flags;
  c.y = y;
  c.ws = workspace;
  c.counters = counters;
  return hip_status(si::launch_owned(c, (hipStream_t)stream), "INT8 layer launch");
}

}  // namespace

extern "C" {

si_status si_quantize_rows_i8(const uint16_t* w, int rows, int n, int8_t* q, float* scale, void* stream) {
  REQUIRE_PTR(w);
  REQUIRE_PTR(q);
  REQUIRE_PTR(scale);
  REQUIRE_ALIGNED(w);
  REQUIRE_ALIGNED(q);
  REQUIRE_ALIGNED(scale);
  if (rows < 1 || rows > (1 << 24) || n < 1 || n > (1 << 24))
    return fail(SI_ERR_SHAPE, "rows=%d n=%d outside [1, 2^24]", rows, n);
  return hip_status(si::launch_quantize_rows(w, rows, n, q, scale, (hipStream_t)stream), "quantize launch");
}

si_status si_pack_signs_i8(const int8_t* w_gate, int k, int d, uint32_t* signs, void* stream) {
  REQUIRE_PTR(w_gate);
  REQUIRE_PTR(signs);
  REQUIRE_ALIGNED(w_gate);
  REQUIRE_ALIGNED(signs);
  if (si_status s = check_kd(k, d)) return s;
  return hip_status(si::launch_pack_signs_i8(w_gate, k, d, signs, (hipStream_t)stream), "pack_signs_i8 launch");
}

si_status si_transpose_down_i8(const int8_t* w_down, int d, int k, int8_t* w_down_t, void* stream) {
  REQUIRE_PTR(w_down);
  REQUIRE_PTR(w_down_t);
  REQUIRE_ALIGNED(w_down);
  REQUIRE_ALIGNED(w_down_t);
  if (si_status s = check_kd(k, d)) return s;
  const uintptr_t a = reinterpret_cast<uintptr_t>(w_down), c = reinterpret_cast<uintptr_t>(w_down_t);
  const uintptr_t n = (uintptr_t)k * (uintptr_t)d;
  if (a < c + n && c < a + n) return fail(SI_ERR_SHAPE, "w_down and w_down_t overlap");
  return hip_status(si::launch_transpose_i8(w_down, d, k, w_down_t, (hipStream_t)stream), "transpose_i8 launch");
}

si_status si_sparse_mlp_i8(const int8_t* w_gate, const float* s_gate, const int8_t* w_up, const float* s_up,
                           const int8_t* w_down_t, const float* s_down, int k, int d, const uint16_t* x, int b,
                           const uint8_t* mask, float* y, void* workspace, size_t workspace_bytes, uint32_t flags,
                           int32_t* counters, void* stream) {
  return int8_impl(false, nullptr, w_gate, s_gate, w_up, s_up, w_down_t, s_down, k, d, x, b, 0.0f, mask, nullptr,
                   nullptr, nullptr, y, workspace, workspace_bytes, flags, counters, stream);
}

si_status si_predict_sparse_mlp_i8(const uint32_t* signs, const int8_t* w_gate, const float* s_gate,
                                   const int8_t* w_up, const float* s_up, const int8_t* w_down_t,
                                   const float* s_down, int k, int d, const uint16_t* x, int b, float alpha,
                                   uint8_t* mask, int32_t* active_idx, int32_t* n_active, float* y,
                                   void* workspace, size_t workspace_bytes, uint32_t flags, int32_t* counters,
                                   void* stream) {
  return int8_impl(true, signs, w_gate, s_gate, w_up, s_up, w_down_t, s_down, k, d, x, b, alpha, nullptr, mask,
                   active_idx, n_active, y, workspace, workspace_bytes, flags, counters, stream);
}

}  // extern "C"

// ---- the whole path without a caller's workspace ---------------------------

namespace {

// The scratch of si_predict_sparse_mlp_noalloc: one array per device, zero at
// load (a zero-filled workspace is the state before a first call) and kept
// from one call to the next exactly like a caller's workspace.
constexpr size_t kScratchBytes = (size_t)8 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// The device address of `scratch` on each device (its host-side name is not
// a device address), looked up once per device with that device current.
std::atomic<void*> g_scratch_ptr[si::kMaxDevices];

si_status scratch_ptr(void** out) {
  int dev = 0;
  if (si_status s = hip_status(hipGetDevice(&dev), "hipGetDevice")) return s;
  if (dev < 0 || dev >= si::kMaxDevices) return fail(SI_ERR_HIP, "device %d beyond the %d supported", dev, si::kMaxDevices);
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    if (si_status s = hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"))
      return s;
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return SI_OK;
}

}  // namespace

extern "C" si_status si_predict_sparse_mlp_noalloc(const uint32_t* signs, const uint16_t* w_gate,
                                                   const uint16_t* w_up, const uint16_t* w_down_t, int k, int d,
                                                   const uint16_t* x, int b, float alpha, uint8_t* mask,
                                                   int32_t* active_idx, int32_t* n_active, float* y, uint32_t flags,
                                                   int32_t* counters, void* stream) {
  REQUIRE_PTR(signs);
  REQUIRE_PTR(w_gate);
  REQUIRE_PTR(w_up);
  REQUIRE_PTR(w_down_t);
  REQUIRE_PTR(x);
  REQUIRE_PTR(y);
  if (si_status s = check_kd(k, d)) return s;
  if (si_status s = check_b(b)) return s;
  const size_t need = si::ws_layout(k, b).total;
  if (need > kScratchBytes)
    return fail(SI_ERR_WORKSPACE, "k=%d b=%d needs %zu bytes of scratch; the no-allocation call holds %zu per device",
                k, b, need, kScratchBytes);
  void* ws = nullptr;
  if (si_status s = scratch_ptr(&ws)) return s;
  return predict_sparse_mlp_impl(signs, w_gate, w_up, w_down_t, k, d, x, b, alpha, mask, active_idx, n_active, y,
                                 ws, kScratchBytes, flags, counters, stream);
}
