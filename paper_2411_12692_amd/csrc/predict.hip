// Sign-bit activation-sparsity predictor (Section IV-A, Eq. (2)) with ordered
// compaction of the kept rows.
//
// One block of 4 wavefronts handles one group of 64 rows; lane r of every
// wave owns row 64*v + r (lane-per-row: no cross-lane reduction, and a
// wave-wide ballot gives the group's kept rows directly).  The 4 waves split
// the row's packed words and add their counts through LDS.  The sign words of
// x (one token or up to 8) are packed by the block itself into LDS.
//
// Eq. (2) is applied through the integer threshold T computed on the host:
// a row is kept for a token iff N_neg < T.
//
// The ascending kept list needs each group's offset, i.e. an exclusive
// prefix over the groups' counts.  It is obtained in the same pass with a
// decoupled look-back: blocks take their group id from a ticket counter (so
// a block only ever waits on groups owned by blocks that already run), post
// their own count, and walk back over their predecessors' posted counts.
// Posted words carry a call counter (epoch) so the workspace never needs to
// be cleared between calls; the last block of a call resets the ticket and
// advances the epoch.
#include "si_device.h"
#include "si_launch.h"

namespace si {

constexpr uint64_t kFlagAggregate = 1ull << 30;  // count of this group only
constexpr uint64_t kFlagPrefix = 2ull << 30;     // inclusive prefix up to this group
constexpr long kSpinLimit = 1l << 22;

// Returns the number of kept rows in groups 0 .. v-1.
__device__ int lookback(uint64_t* status, int v, int local, uint32_t epoch, uint32_t* hdr) {
  const uint64_t tag = (uint64_t)epoch << 32;
  if (v == 0) {
    st_agent64(&status[0], tag | kFlagPrefix | (uint64_t)local);
    return 0;
  }
  st_agent64(&status[v], tag | kFlagAggregate | (uint64_t)local);
  int excl = 0;
  int j = v - 1;
  long spins = 0;
  while (j >= 0) {
    const uint64_t s = ld_agent64(&status[j]);
    const uint64_t flag = s & (3ull << 30);
    if ((uint32_t)(s >> 32) != epoch || flag == 0) {
      if (++spins > kSpinLimit) {  // never expected: predecessors are running
        atomicOr(&hdr[H_ERR], kErrLookbackSpin);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      continue;
    }
    excl += (int)(s & 0x3fffffffu);
    if (flag == kFlagPrefix) break;
    --j;
  }
  st_agent64(&status[v], tag | kFlagPrefix | (uint64_t)(excl + local));
  return excl;
}

// Count this block as finished; the last block of the call resets the ticket
// and advances the epoch for the next call.
__device__ inline void finish_predict(uint32_t* hdr, int groups, uint32_t epoch) {
  const uint32_t done = atomicAdd(&hdr[H_PRED_DONE], 1u);
  if (done == (uint32_t)groups - 1) {  // every block has taken its ticket and finished
    st_agent(&hdr[H_PRED_TICKET], 0u);
    st_agent(&hdr[H_PRED_DONE], 0u);
    st_agent(&hdr[H_PRED_EPOCH], epoch + 1u);
  }
}

template <int B>
__global__ __launch_bounds__(256) void k_predict(const u32x4* __restrict__ signs, int k, int d,
                                                 const uint16_t* __restrict__ x, int T,
                                                 uint8_t* __restrict__ mask, int32_t* __restrict__ idx,
                                                 int32_t* __restrict__ n_out, uint64_t* __restrict__ status,
                                                 uint32_t* __restrict__ hdr) {
  __shared__ __attribute__((aligned(16))) uint32_t xw[B * (kMaxD / 32)];
  __shared__ int cnt[4][B][kWave];
  __shared__ uint32_t s_v, s_epoch;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int W = d >> 5, units = W >> 2;
  const int groups = (k + kRowGroup - 1) / kRowGroup;

  if (tid == 0) {
    s_v = atomicAdd(&hdr[H_PRED_TICKET], 1u);
    s_epoch = ld_agent(&hdr[H_PRED_EPOCH]);
  }
  // sign words of the b input tokens
  for (int t = tid; t < B * W; t += 256) {
    const int tok = t / W, w = t - tok * W;
    xw[t] = sign_word(reinterpret_cast<const u32x4*>(x + (size_t)tok * d + 32 * w));
  }
  __syncthreads();
  const int v = (int)s_v;
  const uint32_t epoch = s_epoch;
  if (v >= groups) {  // only if the workspace was not zero-filled before first use
    if (tid == 0) {
      atomicOr(&hdr[H_ERR], kErrTicket);
      finish_predict(hdr, groups, epoch);
    }
    return;
  }
  const int row = v * kRowGroup + lane;

  int c[B];
#pragma unroll
  for (int t = 0; t < B; ++t) c[t] = 0;
  const u32x4* sg = signs + (size_t)v * units * kRowGroup + lane;
#pragma unroll 4
  for (int q = wv; q < units; q += 4) {
    const u32x4 s = load_nt(sg + (size_t)q * kRowGroup);
#pragma unroll
    for (int t = 0; t < B; ++t) {
      const u32x4 xv = *reinterpret_cast<const u32x4*>(&xw[t * W + 4 * q]);
      c[t] += __popc(s.x ^ xv.x) + __popc(s.y ^ xv.y) + __popc(s.z ^ xv.z) + __popc(s.w ^ xv.w);
    }
  }
#pragma unroll
  for (int t = 0; t < B; ++t) cnt[wv][t][lane] = c[t];
  __syncthreads();
  if (wv != 0) return;

  bool keep = false;
#pragma unroll
  for (int t = 0; t < B; ++t) {
    const int n_neg = cnt[0][t][lane] + cnt[1][t][lane] + cnt[2][t][lane] + cnt[3][t][lane];
    keep |= n_neg < T;
  }
  keep = keep && row < k;
  if (row < k) mask[row] = keep ? 1 : 0;
  const uint64_t ballot = __ballot(keep);
  const int local = __popcll(ballot);
  int excl = 0;
  if (lane == 0) excl = lookback(status, v, local, epoch, hdr);
  excl = __shfl(excl, 0, kWave);
  if (keep && idx) idx[excl + __popcll(ballot & lanes_below(lane))] = row;
  if (lane == 0) {
    if (v == groups - 1 && n_out) *n_out = excl + local;
    finish_predict(hdr, groups, epoch);
  }
}

// mask -> ascending list of the nonzero positions and their count.
__global__ __launch_bounds__(1024) void k_compact(const uint8_t* __restrict__ mask, int k,
                                                  int32_t* __restrict__ idx, int32_t* __restrict__ n_out) {
  __shared__ int wsum[16];
  __shared__ int base;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (tid == 0) base = 0;
  __syncthreads();
  for (int off = 0; off < k; off += 1024) {
    const int i = off + tid;
    const bool a = i < k && mask[i] != 0;
    const uint64_t bal = __ballot(a);
    if (lane == 0) wsum[wv] = __popcll(bal);
    __syncthreads();
    int pre = base;
    for (int w = 0; w < wv; ++w) pre += wsum[w];
    if (a) idx[pre + __popcll(bal & lanes_below(lane))] = i;
    __syncthreads();
    if (tid == 0) {
      int s = 0;
      for (int w = 0; w < 16; ++w) s += wsum[w];
      base += s;
    }
    __syncthreads();
  }
  if (tid == 0) *n_out = base;
}

template <int B>
static void predict_b(const uint32_t* signs, int k, int d, const uint16_t* x, int T, uint8_t* mask,
                      int32_t* idx, int32_t* n_out, void* ws, hipStream_t s) {
  const WsLayout L = ws_layout(k, B);
  char* base = static_cast<char*>(ws);
  const int groups = (k + kRowGroup - 1) / kRowGroup;
  k_predict<B><<<groups, 256, 0, s>>>(reinterpret_cast<const u32x4*>(signs), k, d, x, T, mask, idx, n_out,
                                       reinterpret_cast<uint64_t*>(base + L.status),
                                       reinterpret_cast<uint32_t*>(base));
}

hipError_t launch_predict(const uint32_t* signs, int k, int d, const uint16_t* x, int b, int T,
                          uint8_t* mask, int32_t* idx, int32_t* n_out, void* ws, hipStream_t s) {
  switch (b) {
    case 1: predict_b<1>(signs, k, d, x, T, mask, idx, n_out, ws, s); break;
    case 2: predict_b<2>(signs, k, d, x, T, mask, idx, n_out, ws, s); break;
    case 3: predict_b<3>(signs, k, d, x, T, mask, idx, n_out, ws, s); break;
    case 4: predict_b<4>(signs, k, d, x, T, mask, idx, n_out, ws, s); break;
    case 5: predict_b<5>(signs, k, d, x, T, mask, idx, n_out, ws, s); break;
    case 6: predict_b<6>(signs, k, d, x, T, mask, idx, n_out, ws, s); break;
    case 7: predict_b<7>(signs, k, d, x, T, mask, idx, n_out, ws, s); break;
    case 8: predict_b<8>(signs, k, d, x, T, mask, idx, n_out, ws, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_compact(const uint8_t* mask, int k, int32_t* idx, int32_t* n_out, hipStream_t s) {
  k_compact<<<1, 1024, 0, s>>>(mask, k, idx, n_out);
  return hipGetLastError();
}

}  // namespace si
