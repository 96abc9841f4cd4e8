// Sign-bit activation-sparsity predictor (Section IV-A, Eq. (2)) with ordered
// compaction of the kept rows, optionally fused with the sparse gate/up GEMV
// (Section IV-B 3)-4): steps 1-3 of Eq. (1) for the kept rows).
//
// One block of 8 wavefronts owns one group of 64 rows (blockIdx = group).
//  1. x is staged in LDS and its sign words are packed there.
//  2. Lane r of every wave counts N_neg of row 64*g + r over an eighth of the
//     row's packed words (XOR + popcount, 16-byte coalesced loads from the
//     interleaved sign layout); the 8 partial counts meet in LDS.
//  3. Wave 0 applies Eq. (2) through the host-computed integer threshold T
//     (kept iff N_neg < T for some token), writes the mask, and ballots the
//     kept rows into an LDS list.
//  4. Fused variant: waves 1..7 stream the W_gate row of each kept row, and
//     the W_up row only where some token's ReLU output is positive (actual
//     sparsity), writing h3 = h1 * u per row.
//  5. Meanwhile wave 0 finds the group's offset in the ascending kept list
//     with a decoupled look-back: it posts its count, then reads up to 64
//     predecessors' posted words at once (one per lane) until it meets an
//     inclusive prefix.  It then writes its kept rows at that offset.
//
// Posted words carry a per-call counter (epoch) so the workspace is never
// cleared between calls.  The last group advances the epoch once its
// look-back completes: by then every group has posted, so every block has
// read the current epoch.  No single-address atomic counters are used (they
// serialise across the chip).
#include "si_device.h"
#include "si_launch.h"

namespace si {

constexpr uint64_t kFlagAggregate = 1ull << 30;  // count of this group only
constexpr uint64_t kFlagPrefix = 2ull << 30;     // inclusive prefix up to this group
constexpr uint64_t kFlagMask = 3ull << 30;
constexpr long kSpinLimit = 1l << 20;
constexpr int kPredWaves = 8;

// Wave-wide look-back: returns the number of kept rows in groups 0 .. v-1.
// The caller has already posted the group's aggregate.
__device__ int lookback_wave(const uint64_t* status, int v, uint32_t tag, int lane, uint32_t* hdr) {
  int excl = 0;
  int j = v - 1;
  long spins = 0;
  while (j >= 0) {
    const int jj = j - lane;  // lane 0 = nearest predecessor
    uint64_t s = 0;
    bool ready = true, prefix = true;
    if (jj >= 0) {
      s = ld_agent64(&status[jj]);
      ready = (uint32_t)(s >> 32) == tag && (s & kFlagMask) != 0;
      prefix = ready && (s & kFlagMask) == kFlagPrefix;
    }
    const uint64_t pmask = __ballot(prefix);
    const uint64_t rmask = __ballot(ready);
    const int first = pmask ? __builtin_ctzll(pmask) : kWave;
    const uint64_t need = first >= kWave - 1 ? ~0ull : ((2ull << first) - 1ull);
    if ((rmask & need) != need) {
      if (++spins > kSpinLimit) {  // never expected: every group posts right after counting
        if (lane == 0) atomicOr(&hdr[H_ERR], kErrLookbackSpin);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      continue;
    }
    const int val = (jj >= 0 && lane <= first) ? (int)(s & 0x3fffffffu) : 0;
    excl += wave_sum_int(val);
    if (first < kWave) break;
    j -= kWave;
  }
  return excl;
}

template <int B, bool FUSED>
__global__ __launch_bounds__(kPredWaves * kWave) void k_rows(
    const u32x4* __restrict__ signs, int k, int d, const uint16_t* __restrict__ x, int T,
    uint8_t* __restrict__ mask, int32_t* __restrict__ idx, int32_t* __restrict__ n_out,
    uint64_t* __restrict__ status, uint32_t* __restrict__ hdr,
    const u32x4* __restrict__ wg, const u32x4* __restrict__ wu, float* __restrict__ h3row,
    uint8_t* __restrict__ upflag, int32_t* __restrict__ counts, float* __restrict__ y, uint32_t flags) {
  extern __shared__ u32x4 xs[];  // [B][d/8] fp16 tokens
  __shared__ __attribute__((aligned(16))) uint32_t xw[B * (kMaxD / 32)];
  __shared__ int cnt[kPredWaves][B][kWave];
  __shared__ int kept[kRowGroup];
  __shared__ int s_nkept, s_up, s_down;
  constexpr int NT = kPredWaves * kWave;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int U = d >> 3, W = d >> 5, units = W >> 2;
  const int v = blockIdx.x;
  const int groups = gridDim.x;
  const int row = v * kRowGroup + lane;

  if (FUSED && v == 0) {  // y is accumulated with atomics by the down-projection kernel
    for (int i = tid; i < B * d; i += NT) y[i] = 0.f;
    if (tid == 0) hdr[H_H3_FORM] = kH3PlainByRow;
  }
  // 1. tokens -> LDS, then their packed sign words
  for (int i = tid; i < B * U; i += NT) xs[i] = reinterpret_cast<const u32x4*>(x)[i];
  __syncthreads();
  for (int i = tid; i < B * W; i += NT) {
    const int t = i / W, w = i - t * W;
    xw[i] = sign_word(&xs[t * U + 4 * w]);
  }
  __syncthreads();

  // 2. N_neg partial counts
  int c[B];
#pragma unroll
  for (int t = 0; t < B; ++t) c[t] = 0;
  const int kpad = groups * kRowGroup;  // rows of the packed layout (unit q of row i at q * kpad + i)
  const u32x4* sg = signs + (size_t)v * kRowGroup + lane;
#pragma unroll 4
  for (int q = wv; q < units; q += kPredWaves) {
    const u32x4 s = load_nt(sg + (size_t)q * kpad);
#pragma unroll
    for (int t = 0; t < B; ++t) {
      const u32x4 xv = *reinterpret_cast<const u32x4*>(&xw[t * W + 4 * q]);
      c[t] += __popc(s.x ^ xv.x) + __popc(s.y ^ xv.y) + __popc(s.z ^ xv.z) + __popc(s.w ^ xv.w);
    }
  }
#pragma unroll
  for (int t = 0; t < B; ++t) cnt[wv][t][lane] = c[t];
  __syncthreads();

  // 3. Eq. (2), mask, kept list in LDS, post this group's count
  uint64_t ballot = 0;
  uint32_t epoch = 0;
  if (wv == 0) {
    bool keep = false;
#pragma unroll
    for (int t = 0; t < B; ++t) {
      int n_neg = 0;
#pragma unroll
      for (int w = 0; w < kPredWaves; ++w) n_neg += cnt[w][t][lane];
      keep |= n_neg < T;
    }
    keep = keep && row < k;
    if (row < k) mask[row] = keep ? 1 : 0;
    ballot = __ballot(keep);
    const int local = __popcll(ballot);
    if (keep) kept[__popcll(ballot & lanes_below(lane))] = row;
    if (lane == 0) {
      s_nkept = local;
      s_up = 0;
      s_down = 0;
      epoch = ld_agent(&hdr[H_EPOCH]);
      const uint64_t tag = (uint64_t)epoch_tag(epoch) << 32;
      st_agent64(&status[v], tag | (v == 0 ? kFlagPrefix : kFlagAggregate) | (uint64_t)local);
    }
    epoch = __shfl(epoch, 0, kWave);
  }
  __syncthreads();
  const int nkept = s_nkept;

  if (wv == 0) {
    // 5. offset of this group in the ascending kept list
    const int excl = v == 0 ? 0 : lookback_wave(status, v, epoch_tag(epoch), lane, hdr);
    if (lane == 0 && v > 0)
      st_agent64(&status[v], ((uint64_t)epoch_tag(epoch) << 32) | kFlagPrefix | (uint64_t)(excl + nkept));
    if (lane < nkept && idx) idx[excl + lane] = kept[lane];
    if (lane == 0 && v == groups - 1) {
      if (n_out) *n_out = excl + nkept;
      st_agent(&hdr[H_EPOCH], epoch + 1u);  // every group has posted: all read this epoch
    }
  } else if (FUSED) {
    // 4. sparse gate/up over the kept rows of this group
    int n_up = 0, n_down = 0;
    const bool no_as = (flags & 1u) != 0;
    for (int i = wv - 1; i < nkept; i += kPredWaves - 1)
      gate_up_row<B>(wg, wu, kept[i], U, xs, lane, no_as, h3row, upflag, n_up, n_down);
    if (lane == 0 && (n_up | n_down)) {
      atomicAdd(&s_up, n_up);
      atomicAdd(&s_down, n_down);
    }
  }
  if (FUSED) {
    __syncthreads();
    if (tid == 0) {
      counts[2 * v] = s_up;
      counts[2 * v + 1] = s_down;
    }
  }
}

template <int B, bool FUSED>
static hipError_t rows_b(const uint32_t* signs, int k, int d, const uint16_t* x, int T, uint8_t* mask,
                         int32_t* idx, int32_t* n_out, void* ws, const uint16_t* w_gate, const uint16_t* w_up,
                         float* y, uint32_t flags, hipStream_t s) {
  const WsLayout L = ws_layout(k, B);
  char* base = static_cast<char*>(ws);
  const size_t lds = (size_t)B * d * sizeof(uint16_t);
  // the kernel's dynamic LDS limit, set once per device
  static std::atomic<int> attr_set[kMaxDevices];
  const int ok = per_device_once(attr_set, [](int) -> int {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&k_rows<B, FUSED>), hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)((size_t)kMaxB * kMaxD * sizeof(uint16_t))) == hipSuccess ? 1 : -1;
  });
  if (ok != 1) return hipErrorInvalidConfiguration;
  k_rows<B, FUSED><<<row_groups(k), kPredWaves * kWave, lds, s>>>(
      reinterpret_cast<const u32x4*>(signs), k, d, x, T, mask, idx, n_out,
      reinterpret_cast<uint64_t*>(base + L.status), reinterpret_cast<uint32_t*>(base),
      reinterpret_cast<const u32x4*>(w_gate), reinterpret_cast<const u32x4*>(w_up),
      reinterpret_cast<float*>(base + L.h3), reinterpret_cast<uint8_t*>(base + L.upflag),
      reinterpret_cast<int32_t*>(base + L.counts), y, flags);
  return hipGetLastError();
}

#define SI_ROWS_CASES(FUSED)                                                                              \
  switch (b) {                                                                                            \
    case 1: return rows_b<1, FUSED>(signs, k, d, x, T, mask, idx, n_out, ws, w_gate, w_up, y, flags, s); \
    case 2: return rows_b<2, FUSED>(signs, k, d, x, T, mask, idx, n_out, ws, w_gate, w_up, y, flags, s); \
    case 3: return rows_b<3, FUSED>(signs, k, d, x, T, mask, idx, n_out, ws, w_gate, w_up, y, flags, s); \
    case 4: return rows_b<4, FUSED>(signs, k, d, x, T, mask, idx, n_out, ws, w_gate, w_up, y, flags, s); \
    case 5: return rows_b<5, FUSED>(signs, k, d, x, T, mask, idx, n_out, ws, w_gate, w_up, y, flags, s); \
    case 6: return rows_b<6, FUSED>(signs, k, d, x, T, mask, idx, n_out, ws, w_gate, w_up, y, flags, s); \
    case 7: return rows_b<7, FUSED>(signs, k, d, x, T, mask, idx, n_out, ws, w_gate, w_up, y, flags, s); \
    case 8: return rows_b<8, FUSED>(signs, k, d, x, T, mask, idx, n_out, ws, w_gate, w_up, y, flags, s); \
    default: return hipErrorInvalidValue;                                                                 \
  }

hipError_t launch_predict(const uint32_t* signs, int k, int d, const uint16_t* x, int b, int T,
                          uint8_t* mask, int32_t* idx, int32_t* n_out, void* ws, hipStream_t s) {
  const uint16_t* w_gate = nullptr;
  const uint16_t* w_up = nullptr;
  float* y = nullptr;
  const uint32_t flags = 0;
  SI_ROWS_CASES(false)
}

hipError_t launch_predict_gate_up(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up, int k,
                                  int d, const uint16_t* x, int b, int T, uint8_t* mask, int32_t* idx,
                                  int32_t* n_out, float* y, void* ws, uint32_t flags, hipStream_t s) {
  SI_ROWS_CASES(true)
}

#undef SI_ROWS_CASES

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

// ascending list of n rows (n read from n_in) -> [k] mask (1 = listed): the
// block clears every byte, then sets the listed rows; entries outside
// [0, k) are ignored.
__global__ __launch_bounds__(1024) void k_list_to_mask(const int32_t* __restrict__ idx,
                                                       const int32_t* __restrict__ n_in, int k,
                                                       uint8_t* __restrict__ mask) {
  const int tid = threadIdx.x;
  for (int i = tid; i < k; i += 1024) mask[i] = 0;
  const int n = min(max(*n_in, 0), k);
  __syncthreads();
  for (int j = tid; j < n; j += 1024) {
    const int r = idx[j];
    if (r >= 0 && r < k) mask[r] = 1;
  }
}

hipError_t launch_list_to_mask(const int32_t* idx, const int32_t* n_in, int k, uint8_t* mask, hipStream_t s) {
  k_list_to_mask<<<1, 1024, 0, s>>>(idx, n_in, k, mask);
  return hipGetLastError();
}

hipError_t launch_compact(const uint8_t* mask, int k, int32_t* idx, int32_t* n_out, hipStream_t s) {
  k_compact<<<1, 1024, 0, s>>>(mask, k, idx, n_out);
  return hipGetLastError();
}

}  // namespace si
