/*
 * sparseinfer.h -- C ABI of the MI355X (gfx950) SparseInfer decode path.
 *
 * SparseInfer (arXiv 2411.12692) predicts which rows of a ReLU-fied gated MLP
 * produce a zero activation by comparing sign bits only (Section IV-A), then
 * runs the MLP of Eq. (1) over the remaining rows (Section IV-B).  This
 * library implements that per-token path with hand-written HIP kernels.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensors are DEVICE pointers allocated by the caller (the library never
 *   allocates or frees), row-major, 16-byte aligned.  fp16 tensors are passed
 *   as uint16_t bit patterns (IEEE binary16).
 * - Shapes: d = model dimension, k = hidden (d_ff) dimension, b = tokens in
 *   the decode batch.  Supported: 1 <= k <= 2^24, 128 <= d <= 8192 with
 *   d % 128 == 0, 1 <= b <= 8.
 * - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL means
 *   the default stream).  Calls return after enqueueing.
 * - Errors: arguments are validated on the host before anything is enqueued;
 *   on any error nothing is launched, outputs are untouched, the status code
 *   says which check failed and si_last_error() (thread-local) says why.
 *   A failed launch returns SI_ERR_HIP.  Faults inside kernels surface at the
 *   caller's next synchronisation, as for any HIP kernel.
 * - Workspace: entry points that take `workspace` need a caller-owned device
 *   buffer of at least si_workspace_bytes(k, d, b) bytes that is ZERO-FILLED
 *   before its first use.  The library keeps it consistent from one call to
 *   the next (it resets its own counters), so it must not be modified by the
 *   caller afterwards, and one workspace must not be used by two calls that
 *   can run at the same time (e.g. on two streams).
 * - Co-residency: where si_single_launch(k, d, b) is 1, a call is one kernel
 *   of one block per compute unit whose blocks hand each other data while it
 *   runs, so every block must be resident at once.  The call needs every
 *   compute unit of the device to itself: a kernel running concurrently on
 *   another stream, or a CU mask that hides compute units, can keep a block
 *   from starting.  Every wait inside the kernel is bounded (on the order of
 *   a millisecond); a wait that gives up lets the call finish with wrong
 *   results and sets a sticky error word in the workspace.  From then on the
 *   single-launch calls on that workspace compute nothing and fill y with NaN
 *   until si_workspace_check() has reported the error (SI_ERR_TIMEOUT) and
 *   reset the workspace.
 */
#ifndef SPARSEINFER_H
#define SPARSEINFER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SI_OK = 0,
  SI_ERR_NULL = 1,      /* a required pointer is NULL                      */
  SI_ERR_SHAPE = 2,     /* k, d or b outside the supported range           */
  SI_ERR_ALIGN = 3,     /* a pointer is not 16-byte aligned                */
  SI_ERR_ALPHA = 4,     /* alpha is NaN or negative                        */
  SI_ERR_WORKSPACE = 5, /* workspace smaller than si_workspace_bytes()     */
  SI_ERR_HIP = 6,       /* the HIP runtime reported an error               */
  SI_ERR_FLAGS = 7,     /* unknown bits in `flags`                         */
  SI_ERR_ARG = 8,       /* another argument out of range (eps, overlapping
                           buffers)                                        */
  SI_ERR_TIMEOUT = 9,   /* a bounded wait inside a kernel gave up (blocks of
                           a single-launch call were not all resident)     */
  SI_ERR_LIST = 10      /* a caller's active_idx held a row outside [0, k) */
} si_status;

/* Flags of si_sparse_mlp / si_predict_sparse_mlp. */
#define SI_NO_AS 1u /* ignore actual sparsity (Section IV-B 3): read the W_up
                       and W_down^T rows of every predicted-active row even
                       where h1 or h3 is zero.  Results are identical; only
                       the work differs.  Used for the paper's +-AS ablation. */
#define SI_NO_SPECULATION 2u /* read W_up / W_down^T rows strictly after the
                       values that decide whether they are needed.  By default
                       the single-kernel path requests them with the W_gate
                       row for rows that are likely active: with one token,
                       the rows Eq. (2) would keep at alpha = 1 (N_neg <=
                       d/2; rows kept only because alpha > 1 wait for their
                       gate value); with 2-4 tokens, rows d/16 inside that;
                       with 5-8 tokens, every kept row.  Results are
                       identical; only the work may differ. */

/* Human-readable reason of the last non-SI_OK status on this thread. */
const char* si_last_error(void);

/* Library version string. */
const char* si_version(void);

/*
 * Size in bytes of the packed sign buffer of one W_gate (Section IV-B 1):
 * one bit per element, rows padded to a multiple of 64.  Equals k*d/8 when
 * k % 64 == 0.  Returns 0 for unsupported shapes.
 */
size_t si_signs_bytes(int k, int d);

/*
 * Pack the sign bits (MSBs) of W_gate, once at model load (Section IV-B 1).
 *   w_gate : [k][d] fp16, read.
 *   signs  : si_signs_bytes(k, d) bytes, written.  The layout is private to
 *            the library (rows interleaved for coalesced per-row counting);
 *            si_signs_to_canonical() exports it.
 */
si_status si_pack_signs(const uint16_t* w_gate, int k, int d, uint32_t* signs, void* stream);

/*
 * Export packed signs in the canonical layout of Section IV-B 1) (each row's
 * sign bits packed 32 to a word, in element order): out[i][w] (k rows of
 * d/32 uint32, written) has bit j set iff W_gate[i][32*w + j] has its sign
 * bit set.  signs: si_signs_bytes(k, d) bytes from si_pack_signs, read.
 * For tests and inspection; the decode path never calls it.
 */
si_status si_signs_to_canonical(const uint32_t* signs, int k, int d, uint32_t* out, void* stream);

/*
 * W_down^T, once at model load (Section IV-B 4): the paper's W_down is
 * [d][k]; the down-projection kernel skips whole rows of the [k][d]
 * transpose.   w_down: [d][k] fp16, read.  w_down_t: [k][d] fp16, written.
 * The two buffers must not overlap.
 */
si_status si_transpose_down(const uint16_t* w_down, int d, int k, uint16_t* w_down_t, void* stream);

/*
 * Integer form of Eq. (2).  A row is sparse iff alpha * N_pos < N_neg with
 * N_pos = d - N_neg; this returns T = the smallest N_neg in [0, d] for which
 * the row is sparse (d + 1 if none, e.g. alpha = +inf), so a row is kept
 * iff N_neg < T.  alpha is taken as its exact float32 value; ties
 * (alpha * N_pos == N_neg) are kept.  Returns -1 for NaN or negative alpha
 * or unsupported d.  Host-only; needs no GPU.
 */
int32_t si_alpha_threshold(float alpha, int d);

/* Bytes of workspace needed by si_predict / si_sparse_mlp /
 * si_predict_sparse_mlp for these shapes (0 for unsupported shapes): the
 * scratch of the prediction's outputs handed between blocks (Section IV-B
 * 2)), of the h3 values handed from the gate/up step to the down-projection
 * (Eq. (1), steps 3 and 4; Section IV-B 3), 4)), and the call counter and
 * error bits.  Host-only. */
size_t si_workspace_bytes(int k, int d, int b);

/*
 * Errors found inside kernels, which no call can return when it is made
 * (calls only enqueue work).  Waits for `stream` (NULL: the default
 * stream), then reads the workspace's sticky error word:
 *   SI_OK          : no error since the workspace was zero-filled or last
 *                    checked;
 *   SI_ERR_TIMEOUT : a bounded wait gave up (see "Co-residency" above); the
 *                    results of that call and of the single-launch calls on
 *                    this workspace since then are wrong (y is NaN);
 *   SI_ERR_LIST    : a caller's active_idx held a row outside [0, k) (the
 *                    entry was skipped).
 * On an error the whole workspace (workspace_bytes bytes) is zero-filled,
 * which restores it to its first-use state, and later calls compute again.
 * Not for use during stream capture (it synchronizes).  SI_ERR_NULL /
 * SI_ERR_ALIGN for a bad pointer, SI_ERR_HIP if the synchronization or a
 * copy fails.
 */
si_status si_workspace_check(void* workspace, size_t workspace_bytes, void* stream);

/*
 * Host-only: the status that si_workspace_check() returns for the value
 * `bits` of the sticky error word (bit 0: a wait gave up, bit 2: a list row
 * outside [0, k); a wait that gave up takes precedence).  Unknown bits give
 * SI_ERR_ARG.  Needs no GPU.
 */
si_status si_device_error_status(uint32_t bits);

/*
 * Diagnostic read-back, for tests: the per-row values h3_i,t of Eq. (1)
 * step 3 (h3 = ReLU(W_gate,i . x_t) * (W_up,i . x_t); ReLU(W_fc1,i . x_t)
 * for the non-gated MLP; with the INT8 scales applied) that the last MLP
 * call made with this workspace computed.
 *   mask : [k] uint8, the rows that call kept (nonzero = kept), read.
 *   h3   : [k][b] float32, written: the call's value for each kept row, 0 for
 *          the other rows, NaN for a kept row for which the call left no
 *          value of its own (a row it dropped).
 *   b    : the batch of that call.
 * The MLP call must be the last call made with the workspace (a later
 * si_predict replaces what it left).  Enqueued on `stream`.
 */
si_status si_read_h3(const void* workspace, size_t workspace_bytes, int k, int d, int b, const uint8_t* mask,
                     float* h3, void* stream);

/*
 * Diagnostic, outside the path: read `bytes` bytes of device memory at `buf`
 * (16-byte aligned, bytes a positive multiple of 16) once, with 16-byte
 * non-temporal loads from a grid of 8 blocks of 256 threads per compute unit.
 * The time it takes gives the streaming-read bandwidth the device achieves,
 * which the benchmark reports beside the HBM peak.  `sink` ([1] uint32) is
 * written only if the XOR of the data equals one fixed constant (so that the
 * loads cannot be dropped).  Enqueued on `stream`.
 */
si_status si_read_bandwidth_probe(const void* buf, size_t bytes, uint32_t* sink, void* stream);

/*
 * Predict the rows of W_gate whose ReLU output will be zero (Section IV-A).
 * For every token t and row i: N_neg = popcount(sign(W_gate,i) XOR
 * sign(x_t)) over the d elements, and the row is sparse for that token iff
 * alpha * (d - N_neg) < N_neg (Eq. (2)).  A row is kept (predicted active)
 * when at least one token keeps it.
 *   signs      : from si_pack_signs(), read.
 *   x          : [b][d] fp16, read.
 *   alpha      : conservativeness, >= 0 (+inf keeps every row).
 *   mask       : [k] uint8, written; 1 = kept, 0 = predicted sparse.
 *   active_idx : [k] int32, written: the kept rows in ascending order in
 *                entries 0 .. n-1 (later entries untouched).  May be NULL.
 *   n_active   : [1] int32, written with n.  May be NULL.
 *   workspace  : see the conventions above.
 */
si_status si_predict(const uint32_t* signs, int k, int d, const uint16_t* x, int b, float alpha,
                     uint8_t* mask, int32_t* active_idx, int32_t* n_active,
                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * Gated MLP of Eq. (1) over the kept rows (Section IV-B 3)-4)), fp32
 * accumulation.  For every kept row i and token t:
 *   g = W_gate,i . x_t ;  h1 = max(g, 0) ;  u = W_up,i . x_t (read only when
 *   some token has h1 > 0) ;  h3 = h1 * u ;  y_t += h3 * W_down^T[i, :]
 *   (row read only when some token has h3 != 0).
 *   w_gate, w_up : [k][d] fp16; w_down_t : [k][d] fp16 (si_transpose_down).
 *   x            : [b][d] fp16.
 *   mask         : [k] uint8 (nonzero = kept); used only when active_idx is
 *                  NULL, in which case the kept list is built from it.
 *   active_idx, n_active : kept rows in ascending order and their count, as
 *                  written by si_predict (device memory).  Either both or
 *                  neither may be NULL.
 *   y            : [b][d] float, overwritten.
 *   flags        : 0, SI_NO_AS, SI_NO_SPECULATION or both.
 *   counters     : [3] int32 or NULL: rows whose W_gate, W_up and W_down^T
 *                  rows were read (n_gate, n_up, n_down; rows requested
 *                  speculatively count as read).
 */
si_status si_sparse_mlp(const uint16_t* w_gate, const uint16_t* w_up, const uint16_t* w_down_t,
                        int k, int d, const uint16_t* x, int b, const uint8_t* mask,
                        const int32_t* active_idx, const int32_t* n_active, float* y,
                        void* workspace, size_t workspace_bytes, uint32_t flags, int32_t* counters,
                        void* stream);

/*
 * 1 if si_predict, si_sparse_mlp and si_predict_sparse_mlp (and their
 * non-gated forms), the steps of Section IV-B for one layer, run as a
 * single kernel launch for these shapes on the
 * current device: at most 256 rows of W_gate per compute unit (k <= 65536 on
 * a 256-CU MI355X) and one block with 96-160 KB of LDS resident on every
 * compute unit; 0 if they take the multi-launch path (same results) or the
 * shapes are invalid.  Host-only query.
 */
int si_single_launch(int k, int d, int b);

/*
 * The whole per-token MLP path in one call: si_predict followed by
 * si_sparse_mlp, with the same arguments and outputs (mask, active_idx,
 * n_active and counters may each be NULL).  This is the decode hot path.
 */
si_status si_predict_sparse_mlp(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up,
                                const uint16_t* w_down_t, int k, int d, const uint16_t* x, int b,
                                float alpha, uint8_t* mask, int32_t* active_idx, int32_t* n_active,
                                float* y, void* workspace, size_t workspace_bytes, uint32_t flags,
                                int32_t* counters, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * si_predict_sparse_mlp without a workspace argument.  Its scratch is one
 * array of 8 MiB per device inside the library (a file-scope device array,
 * held on every device the library runs on until the process ends); the
 * call allocates and frees nothing.  Arguments, outputs and errors as
 * si_predict_sparse_mlp without workspace / workspace_bytes; shapes whose
 * workspace (si_workspace_bytes(k, d, b)) exceeds 8 MiB return
 * SI_ERR_WORKSPACE (every k <= 65536 fits, at any d and b).
 * Every call on one device shares that device's array: calls that can
 * overlap on one device (two streams, two host threads) race and must not
 * be made.  Nothing needs clearing between calls: the array starts
 * zero-filled, and a call reads only words it wrote itself or that carry its
 * own call tag, whatever shapes earlier calls had.  After a bounded wait has
 * given up (see "Co-residency") the later single-launch calls of this entry
 * point on that device fill y with NaN until the process ends.
 */
si_status si_predict_sparse_mlp_noalloc(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up,
                                        const uint16_t* w_down_t, int k, int d, const uint16_t* x, int b,
                                        float alpha, uint8_t* mask, int32_t* active_idx, int32_t* n_active,
                                        float* y, uint32_t flags, int32_t* counters, void* stream);

/*
 * Non-gated ReLU MLP: the MLP block of models without step 2 of Section III
 * (no W_up; e.g. OPT and Falcon after ReLUfication):
 *   MLP(X) = ReLU(X W_fc1) W_down^T.
 * For every kept row i and token t: g = W_fc1,i . x_t ; h = max(g, 0) ;
 * y_t += h * W_down^T[i, :] (row read only when some token has h != 0).
 * Arguments, outputs, flags and errors as si_sparse_mlp, with w_fc1 [k][d]
 * fp16 in place of w_gate and no w_up; counters[1] (n_up) is always 0.
 * The predictor runs on the signs of W_fc1 (si_pack_signs(w_fc1)).
 */
si_status si_sparse_relu_mlp(const uint16_t* w_fc1, const uint16_t* w_down_t, int k, int d, const uint16_t* x,
                             int b, const uint8_t* mask, const int32_t* active_idx, const int32_t* n_active,
                             float* y, void* workspace, size_t workspace_bytes, uint32_t flags, int32_t* counters,
                             void* stream);

/*
 * The whole per-token path of the non-gated ReLU MLP: si_predict on the
 * signs of W_fc1 followed by si_sparse_relu_mlp, with the arguments and
 * outputs of si_predict_sparse_mlp (no w_up).
 */
si_status si_predict_sparse_relu_mlp(const uint32_t* signs, const uint16_t* w_fc1, const uint16_t* w_down_t, int k,
                                     int d, const uint16_t* x, int b, float alpha, uint8_t* mask,
                                     int32_t* active_idx, int32_t* n_active, float* y, void* workspace,
                                     size_t workspace_bytes, uint32_t flags, int32_t* counters, void* stream);

/*
 * The MLP half of a decoder layer in one launch, with the path's neighbours
 * fused: the RMSNorm that produces the MLP input (whose sign words the
 * predictor needs, Section IV-B 1) and the residual add after the
 * down-projection.  Per token t:
 *   x_t = fp16( h_t / sqrt(mean_j(h_t,j^2) + eps) * norm_w )  (in the kernel)
 *   y_t = h_t + MLP(x_t)   with MLP as in si_predict_sparse_mlp (gated), or
 *                          si_predict_sparse_relu_mlp when w_up is NULL.
 *   h      : [b][d] float32, the residual stream, read.
 *   norm_w : [d] float32, the RMSNorm weight, read.
 *   eps    : finite, >= 0.
 *   y      : [b][d] float32, overwritten; must not overlap h.
 * Other arguments, outputs and errors as si_predict_sparse_mlp.  Runs only
 * where the single-launch path applies (si_single_launch(k, d, b) == 1);
 * other shapes return SI_ERR_SHAPE.
 */
si_status si_rmsnorm_predict_sparse_mlp(const float* h, const float* norm_w, float eps, const uint32_t* signs,
                                        const uint16_t* w_gate, const uint16_t* w_up, const uint16_t* w_down_t,
                                        int k, int d, int b, float alpha, uint8_t* mask, int32_t* active_idx,
                                        int32_t* n_active, float* y, void* workspace, size_t workspace_bytes,
                                        uint32_t flags, int32_t* counters, void* stream);

/*
 * INT8 weights.  The predictor reads only the sign bit of each weight, so it
 * applies to INT8 weights unchanged (Section IV-A, robustness to the
 * quantization scheme): the MSB of a two's-complement INT8 value is its
 * sign (0 for zero).  The paper names INT8 without a scheme; these entry
 * points use symmetric INT8 with one float32 scale per output channel, each
 * weight standing for scale * q:
 *   W_gate, W_up : [k][d] int8, scales [k] (one per row);
 *   W_down       : [d][k] int8 (the paper's layout), scales [d] (one per row,
 *                  i.e. per column of y); the kernels take its transpose
 *                  W_down^T [k][d] int8 (si_transpose_down_i8) and the
 *                  same [d] scales.
 */

/*
 * Symmetric per-row quantization, once at load: for each of `rows` rows of
 * n fp16 values, scale = max_j |w_j| / 127 and q_j = rint(w_j / scale)
 * (ties to even, clamped to [-127, 127]), computed in float32 with
 * correctly rounded division; a row of zeros gets scale 0 and q = 0.
 *   w     : [rows][n] fp16, read.       q : [rows][n] int8, written.
 *   scale : [rows] float32, written.    1 <= rows, n <= 2^24 (n need not be
 *   a multiple of anything; only the base pointers must be aligned).
 */
si_status si_quantize_rows_i8(const uint16_t* w, int rows, int n, int8_t* q, float* scale, void* stream);

/*
 * Pack the sign bits (MSBs) of INT8 W_gate (or W_fc1), once at load.
 * w_gate : [k][d] int8, read.  signs : si_signs_bytes(k, d) bytes, written,
 * in the same private layout as si_pack_signs (si_signs_to_canonical
 * exports it); si_predict accepts them as they are.
 */
si_status si_pack_signs_i8(const int8_t* w_gate, int k, int d, uint32_t* signs, void* stream);

/*
 * INT8 W_down [d][k] -> W_down^T [k][d], once at load (the buffers must not
 * overlap).
 */
si_status si_transpose_down_i8(const int8_t* w_down, int d, int k, int8_t* w_down_t, void* stream);

/*
 * Eq. (1) over the rows kept by a caller's mask with INT8 weights (the INT8
 * form of si_sparse_mlp / si_sparse_relu_mlp in mask mode).  For every kept
 * row i and token t:
 *   g = s_gate[i] * (q_gate,i . x_t) ; h1 = max(g, 0) ;
 *   u = s_up[i] * (q_up,i . x_t)  (read only when some token has h1 > 0) ;
 *   h3 = h1 * u ;  y_t[j] += s_down[j] * sum_i h3_i * q_downT[i][j]
 *   (rows read only when some token has h3 != 0).
 * w_up == NULL (s_up ignored) runs the non-gated ReLU MLP (h3 = h1).
 *   mask    : [k] uint8, nonzero = kept (required).
 *   y       : [b][d] float32, overwritten.
 * Flags, counters, workspace and errors as si_sparse_mlp.  Runs where the
 * single-launch path applies (si_single_launch(k, d, b) == 1); other shapes
 * return SI_ERR_SHAPE.
 */
si_status si_sparse_mlp_i8(const int8_t* w_gate, const float* s_gate, const int8_t* w_up, const float* s_up,
                           const int8_t* w_down_t, const float* s_down, int k, int d, const uint16_t* x, int b,
                           const uint8_t* mask, float* y, void* workspace, size_t workspace_bytes, uint32_t flags,
                           int32_t* counters, void* stream);

/*
 * The whole per-token path with INT8 weights: si_predict on the signs of
 * the INT8 W_gate (si_pack_signs_i8) followed by si_sparse_mlp_i8 over the
 * predicted rows, in one launch, with the arguments and outputs of
 * si_predict_sparse_mlp (mask, active_idx, n_active and counters may each be
 * NULL; w_up == NULL: the non-gated ReLU MLP).  Runs where the
 * single-launch path applies; other shapes return SI_ERR_SHAPE.
 */
si_status si_predict_sparse_mlp_i8(const uint32_t* signs, const int8_t* w_gate, const float* s_gate,
                                   const int8_t* w_up, const float* s_up, const int8_t* w_down_t,
                                   const float* s_down, int k, int d, const uint16_t* x, int b, float alpha,
                                   uint8_t* mask, int32_t* active_idx, int32_t* n_active, float* y,
                                   void* workspace, size_t workspace_bytes, uint32_t flags, int32_t* counters,
                                   void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPARSEINFER_H */
