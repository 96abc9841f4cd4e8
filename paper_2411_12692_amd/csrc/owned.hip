// The per-token MLP path of one layer in a single kernel, organised by row
// ownership: sign-bit prediction (Section IV-A, Eq. (2)) or a caller's mask,
// sparse gate/up with actual sparsity and the sparse down-projection
// (Section IV-B 3)-4)), for decode batches of up to 8 tokens.
//
// One block of 16 wavefronts per compute unit, all blocks resident at once.
// With T = 512-column tiles of y, the blocks form groups of T consecutive
// blocks; block b of the first (P / T) T owns rows [b R, (b + 1) R).
//
//  1. predict   each wave XOR/popcounts its share of the 16-byte sign units
//               of the block's rows (lane = row, 64 rows per pass); the last
//               wave applies Eq. (2) as N_neg < T(alpha), writes the mask and
//               publishes the rows' kept mask, "confident" mask (N_neg <
//               T(alpha) - margin: almost surely active) and kept count as
//               tagged words.  In mask mode the kept mask is read from the
//               caller's mask and every kept row counts as confident.
//  2. group     the block reads its group's published masks (a few dozen
//               words, while the memory system is still quiet) and lists the
//               group's kept rows in ascending order.
//  3. gate/up   member m of the group takes positions [n m / T, n (m+1) / T)
//               of the group's n kept rows (an even share, so one round of
//               8 rows almost always suffices): wave w owns (row w/2, W_gate
//               or W_up) and requests all its 16-byte units at once.  W_up
//               rows of confident rows are requested with W_gate; other rows
//               read W_up only where some token's ReLU output is positive
//               (actual sparsity).  h3 is published per row and token.
//  4. down      member m also owns the down item (tile m of y, the group's
//               kept rows): the tile's W_down^T pieces of the confident rows
//               are requested once each wave's gate/up data is in; the
//               item's h3 words are collected, the remaining rows with
//               non-zero h3 are fetched, the per-wave partial tiles are
//               folded in LDS and the tile is added into y with fp32 atomics
//               once the tile's owner has zeroed it in this call.
//
// No block waits for the whole grid: the only exchanges are inside a group.
// Block 0 adds the published kept counts (the count of the call) and, having
// seen a word of this call from every block, advances the call counter.
// When the caller asks for the ascending kept list, each block adds the
// counts of the blocks before it at the end and writes its rows' entries.
//
// Exchange words are 64-bit: this call's tag (the workspace's call counter
// with the high bit set) in the high half, the payload in the low half,
// written with agent-scope write-through stores and read with agent-scope
// loads, so no cache flush or fence is needed and the workspace is never
// cleared between calls.  Every wait is bounded: past a spin limit the block
// sets an error bit in the workspace header and goes on without the data.

#include "layer_common.h"

namespace si {

#ifdef SI_TRACE
__device__ uint64_t g_si_trace[1024 * kTraceSlots];
__device__ uint64_t g_si_trace_wave[1024 * 16 * kTraceWaveMarks];
extern "C" hipError_t si_trace_read(void* dst, size_t bytes) {
  return hipMemcpyFromSymbol(dst, HIP_SYMBOL(g_si_trace), bytes, 0, hipMemcpyDeviceToHost);
}
extern "C" hipError_t si_trace_wave_read(void* dst, size_t bytes) {
  return hipMemcpyFromSymbol(dst, HIP_SYMBOL(g_si_trace_wave), bytes, 0, hipMemcpyDeviceToHost);
}
#endif

constexpr int kMaxOwnRows = 256;                   // rows one block owns (at most)
constexpr int kMaxOwnSub = kMaxOwnRows / kWave;    // 64-row passes of one block (4)
constexpr int kCountWord = 4 * kMaxOwnSub;         // published word that holds the block's kept count
constexpr int kMaxPairs = kWave;                   // (owner block, pass) pairs of one down chunk
constexpr int kMaxChunkRows = 4096;                // rows of one down chunk (at most)
constexpr int kFin = kLWaves - 1;                  // the wave that finishes the prediction
static_assert(kCountWord < kOwnPubStride, "published words of a block");

struct OwnedArgs {
  const u32x4* signs;
  const u32x4* wg;
  const u32x4* wu;
  const u32x4* wdt;
  const uint16_t* x;
  const uint8_t* mask_in;  // mask mode (else predict mode)
  int k, d, b, T, margin;
  uint32_t flags;
  int mlp;
  int R, nsub;             // rows per block, 64-row passes per block
  int tiles, groups;       // tiles of y (= blocks per group), groups (blocks [0, groups * tiles) own rows)
  uint8_t* mask;           // written when not NULL
  int32_t* idx;            // ascending kept list, written when not NULL
  int32_t* n_out;          // kept count, written when not NULL
  uint32_t* hdr;
  uint64_t* pub;           // [blocks][kOwnPubStride]: per pass kept low/high, confident low/high; count
  uint64_t* h3e;           // [k][b] tag | fp32 bits of h3, by row and token
  uint64_t* zflag;         // [tiles] tag once the tile of y is zero
  int32_t* counts;         // [blocks][2] W_up rows read, W_down^T rows read (tile-0 items)
  float* y;
};

template <int BM, int NU>
struct OwnedLds {
  static constexpr int kUnits = NU * kWave;
  static constexpr int kFold = kLWaves / BM;
  // tokens (fp16); once the gate/up work is done, the per-wave partial tiles
  union {
    u32x4 xs[BM * kUnits];
    float dpart[kFold][BM][kTile];
  };
  uint32_t xw[BM * kUnits / 4];  // sign words of the tokens
  // per-wave N_neg partial counts during the prediction; the down chunk's
  // masks, their prefix and its ordered kept rows afterwards
  union {
    int cpart[kLWaves][BM][kWave];
    struct {
      uint32_t pm[4 * kMaxPairs];
      uint32_t dent[kMaxChunkRows];  // conf << 31 | row
    } ch;
  };
  float dots[kRoundRows][2][BM];
  float h1[kRoundRows][BM];
  uint32_t need[kRoundRows];
  uint32_t srow[kMaxOwnRows];  // conf << 31 | row of the block's kept rows, ascending
  float hs[kDownRound * BM];   // h3 of the down round's positions
  int wsum[kLWaves];
  int n_own, n_late, n_up, n_down, zok;
  uint32_t epoch;
};

template <int BM, int NU>
constexpr int owned_lds_bytes() {
  const int need = (int)((sizeof(OwnedLds<BM, NU>) + 1023) / 1024 * 1024);
  return need < kMinLds ? kMinLds : need;
}

// Poll `n` tagged words (lanes may use different addresses) until each
// carries `tag`; payloads into out[].  After the spin limit the missing
// payloads read 0 and the error bit is set.
template <int N>
__device__ inline void poll_words(const uint64_t* const (&p)[N], int n, uint32_t tag, uint32_t* hdr,
                                  uint32_t (&out)[N]) {
  uint32_t pending = 0;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    out[i] = 0;
    if (i < n) pending |= 1u << i;
  }
  long spins = 0;
  while (pending) {
    uint64_t v[N];
#pragma unroll
    for (int i = 0; i < N; ++i)
      if ((pending >> i) & 1u) v[i] = ld_agent64(p[i]);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if (((pending >> i) & 1u) && (uint32_t)(v[i] >> 32) == tag) {
        out[i] = (uint32_t)v[i];
        pending &= ~(1u << i);
      }
    }
    if (pending) {
      if (++spins > kPollLimit) {
        atomicOr(&hdr[H_ERR], kErrLookbackSpin);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
}

// Sum over the block of one int per thread (all threads call it).
template <int BM, int NU>
__device__ inline int block_sum(OwnedLds<BM, NU>& L, int v, int lane, int wv) {
  v = wave_sum_int(v);
  if (lane == 0) L.wsum[wv] = v;
  __syncthreads();
  int t = lane < kLWaves ? L.wsum[lane] : 0;
  t = wave_sum_int(t);
  __syncthreads();
  return t;
}

template <int BM, int NU>
__global__ __launch_bounds__(kLThreads) void k_owned(OwnedArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  OwnedLds<BM, NU>& L = *reinterpret_cast<OwnedLds<BM, NU>*>(lds_raw);

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d = a.d, U = d >> 3, W = d >> 5, units = d >> 7;
  const int b = a.b, k = a.k;
  const int P = gridDim.x, blk = blockIdx.x;
  const int T = a.tiles, R = a.R, nsub = a.nsub;
  const int r0 = blk * R;
  const int Rb = blk < a.groups * T ? max(0, min(R, k - r0)) : 0;  // rows this block owns
  const bool predict = a.mask_in == nullptr;
  const bool no_as = (a.flags & kNoAS) != 0;
  const bool spec_ok = (a.flags & kNoSpec) == 0;
  const bool owns_tile = a.mlp && blk < T;

  SI_TRACE_DECL;
  SI_TRACE_MARK(0);
  // ---- the sign units (or mask bytes) of the first 64 owned rows are
  // requested, then the tokens and (behind the first token requests, so that
  // the wait for it, which comes at once for an atomic load, also covers
  // them) the call counter; addresses are clamped so that the requests are
  // unconditional and go out back to back; tokens b..BM-1 are zero
  u32x4 sreg[kMaxSignUnitsPerWave];
  const int kpad = (k + kRowGroup - 1) / kRowGroup * kRowGroup;  // rows of the packed layout
  auto load_signs = [&](int s) {
    const u32x4* sg = a.signs + r0 + min(s * kWave + lane, Rb - 1);
#pragma unroll
    for (int i = 0; i < kMaxSignUnitsPerWave; ++i) {
      const int q = wv + kLWaves * i;
      if (q < units) sreg[i] = load_nt(sg + (size_t)q * kpad);
    }
  };
  uint32_t mbyte = 0;
  if (Rb > 0) {
    if (predict) load_signs(0);
    else if (wv == kFin) mbyte = a.mask_in[r0 + min(lane, Rb - 1)];
  }
  // the owner of tile blk of y zeroes it (the finishing wave, which later
  // announces it in the tile's flag)
  if (owns_tile && wv == kFin) {
    const int half_cols = min(kTile, d - blk * kTile) / 2;
    for (int t = 0; t < b; ++t) {
      uint64_t* yt = reinterpret_cast<uint64_t*>(a.y + (size_t)t * d + blk * kTile);
      for (int c = lane; c < half_cols; c += kWave) st_agent64(yt + c, 0ull);
    }
  }
  {
    const u32x4* xg = reinterpret_cast<const u32x4*>(a.x);
    const int nx = b * U;
    for (int i = tid; i < BM * U; i += kLThreads) {
      const u32x4 xv = xg[min(i, nx - 1)];
      if (i == tid && tid == 0) {
        asm volatile("" ::: "memory");
        L.epoch = ld_agent(&a.hdr[H_EPOCH]);
        L.n_up = 0;
        L.n_down = 0;
        L.zok = 0;
        L.n_late = 0;
      }
      L.xs[i] = i < nx ? xv : u32x4{0, 0, 0, 0};
    }
  }
  __syncthreads();
  const uint32_t epoch = uniform(L.epoch);
  const uint32_t tag = epoch_tag(epoch);
  // consumed here, where the wait for it is covered by the token requests (a
  // load left outstanding into the loop below would make the compiler wait
  // for every outstanding request, stores included, inside it)
  bool mkeep = mbyte != 0;
  if (predict) {
    for (int i = tid; i < b * W; i += kLThreads) {
      const int t = i / W, w = i - t * W;
      L.xw[i] = sign_word(&L.xs[t * U + 4 * w]);
    }
  }
  __syncthreads();
  SI_TRACE_MARK(1);

  // ---- 1. kept and confident masks of the owned rows, 64 rows per pass;
  // the finishing wave (the last one, which almost never has gate/up work in
  // the first round) applies the rule, lists the kept rows in order and
  // publishes, so no other wave waits for those stores
  int n_own = 0;  // finishing wave
  for (int s = 0; s < nsub; ++s) {
    const bool any_rows = s * kWave < Rb;
    if (predict && any_rows) {
      if (s > 0) load_signs(s);
      int c[BM];
#pragma unroll
      for (int t = 0; t < BM; ++t) c[t] = 0;
      bool any_unit = false;
#pragma unroll
      for (int i = 0; i < kMaxSignUnitsPerWave; ++i) {
        const int q = wv + kLWaves * i;
        if (q < units) {
          any_unit = true;
#pragma unroll
          for (int t = 0; t < BM; ++t) {
            if (t < b) {
              const u32x4 xv = *reinterpret_cast<const u32x4*>(&L.xw[t * W + 4 * q]);
              c[t] += __popc(sreg[i].x ^ xv.x) + __popc(sreg[i].y ^ xv.y) + __popc(sreg[i].z ^ xv.z) +
                      __popc(sreg[i].w ^ xv.w);
            }
          }
        }
      }
      if (any_unit) {
#pragma unroll
        for (int t = 0; t < BM; ++t)
          if (t < b) L.cpart[wv][t][lane] = c[t];
      }
      __syncthreads();
      if (s == 0) SI_TRACE_MARK(2);
    }
    if (wv == kFin) {
      const int i = s * kWave + lane;
      const int row = r0 + i;
      const bool valid = i < Rb;
      bool keep = false, conf = false;
      if (predict) {
        if (any_rows) {
          const int nw = min(units, kLWaves);  // waves that counted units
#pragma unroll
          for (int t = 0; t < BM; ++t) {
            if (t < b) {
              int n_neg = 0;
              for (int w = 0; w < nw; ++w) n_neg += L.cpart[w][t][lane];
              keep |= n_neg < a.T;
              conf |= n_neg < a.T - a.margin;
            }
          }
        }
      } else if (any_rows) {
        if (s > 0) mkeep = a.mask_in[r0 + min(i, Rb - 1)] != 0;
        keep = mkeep;
        conf = keep;
      }
      keep = keep && valid;
      if (s == 0) SI_TRACE_WAVE(5);
      const uint64_t kb = __ballot(keep);
      const uint64_t cb = __ballot(keep && conf);
      if (keep) L.srow[n_own + __popcll(kb & lanes_below(lane))] = (uint32_t)row | (conf ? 0x80000000u : 0u);
      n_own += __popcll(kb);
      if (lane < 4) {
        const uint64_t m = lane < 2 ? kb : cb;
        st_agent64(&a.pub[(size_t)blk * kOwnPubStride + 4 * s + lane],
                   tagged(tag, (uint32_t)(m >> (32 * (lane & 1)))));
      }
      if (valid && a.mask) a.mask[row] = keep ? 1 : 0;
      if (s == 0) SI_TRACE_WAVE(6);
    }
    if (predict && any_rows && s + 1 < nsub) __syncthreads();  // the partial counts are reused
  }
  if (wv == kFin) {
    SI_TRACE_MARK(4);
    if (lane == 0) {
      L.n_own = n_own;
      st_agent64(&a.pub[(size_t)blk * kOwnPubStride + kCountWord], tagged(tag, (uint32_t)n_own));
    }
  }
  if (wv == kFin) SI_TRACE_WAVE(7);
  __syncthreads();
  n_own = uniform(L.n_own);
  SI_TRACE_MARK(3);

  if (a.mlp) {
    // ---- the block's group: the T blocks [g T, g T + T) (T = tiles of y);
    // member m takes an even share of the group's kept rows for gate/up and
    // the down item (tile m, the group's rows)
    const bool in_group = blk < a.groups * T;
    const int g = in_group ? blk / T : 0, m = in_group ? blk - g * T : 0;
    const int tile = m;
    const int npairs = in_group ? T * nsub : 0;  // (owner block, pass) pairs of the group

    // the group's mask words, one per thread (waves 0..3), before any
    // gate/up request is out (a round trip behind the grid's row requests
    // would take several times as long)
    if (tid < 4 * npairs) {
      const int p = tid >> 2;
      const int o = g * T + p / nsub, sb = p - (p / nsub) * nsub;
      const uint64_t* src[1] = {&a.pub[(size_t)o * kOwnPubStride + 4 * sb + (tid & 3)]};
      uint32_t v[1];
      poll_words<1>(src, 1, tag, a.hdr, v);
      L.ch.pm[tid] = v[0];
    }
    __syncthreads();
    if (owns_tile && wv == kFin) {  // the tile's zeroing stores have landed by now
      wait_own_stores();
      if (lane == 0) st_agent64(&a.zflag[blk], tagged(tag, 1u));
    }
    // the group's kept rows in order: every wave forms the prefix of the
    // pairs' kept counts (lane = pair), then one wave per pair writes its
    // rows' entries (lane = row)
    const int cnt = lane < npairs ? __popc(L.ch.pm[4 * lane]) + __popc(L.ch.pm[4 * lane + 1]) : 0;
    const int incl = wave_incl_scan(cnt);
    const int pre = incl - cnt;
    const int n = min(uniform(__builtin_amdgcn_readlane(incl, kWave - 1)), kMaxChunkRows);
    for (int p = wv; p < npairs; p += kLWaves) {
      const uint64_t kb = (uint64_t)L.ch.pm[4 * p] | ((uint64_t)L.ch.pm[4 * p + 1] << 32);
      const uint64_t cb = (uint64_t)L.ch.pm[4 * p + 2] | ((uint64_t)L.ch.pm[4 * p + 3] << 32);
      const int q0p = __builtin_amdgcn_readlane(pre, p);
      if ((kb >> lane) & 1ull) {
        const int o = g * T + p / nsub, sb = p - (p / nsub) * nsub;
        const uint32_t row = (uint32_t)(o * R + sb * kWave + lane);
        const int q = q0p + __popcll(kb & lanes_below(lane));
        if (q < kMaxChunkRows) L.ch.dent[q] = row | (((cb >> lane) & 1ull) ? 0x80000000u : 0u);
      }
    }
    const int lo = (n * m) / T, hi = (n * (m + 1)) / T;  // this member's gate/up positions
    const int dN = n;                                     // the down item's positions
    __syncthreads();
    SI_TRACE_MARK(4);

    // down requests of a round: this wave's positions q0 + wv + 16 j
    u32x4 vd[kDN];
    uint32_t dloaded = 0;
    const int dunit = tile * kWave + lane;
    const bool dcol_ok = dunit < U;
    auto issue_down = [&](int q0) {
      dloaded = 0;
#pragma unroll
      for (int j = 0; j < kDN; ++j) {
        vd[j] = u32x4{0, 0, 0, 0};
        const int q = q0 + wv + kLWaves * j;
        if (q < dN) {
          const uint32_t e = L.ch.dent[q];
          if ((spec_ok && (e >> 31)) || no_as) {
            if (dcol_ok) vd[j] = load_nt(a.wdt + (size_t)(e & 0x7fffffffu) * U + dunit);
            dloaded |= 1u << j;
          }
        }
      }
    };

    // ---- 2. gate/up over the member's positions [lo, hi) of the group's
    // list (the first round runs also when there are none)
    const int ir = wv >> 1, imat = wv & 1;
    for (int r0r = lo, first = 1;; r0r += kRoundRows, first = 0) {
      const int mr = max(0, min(kRoundRows, hi - r0r));
      const uint32_t* srow = &L.ch.dent[r0r];
      if (!first) __syncthreads();
      const uint32_t e = ir < mr ? srow[ir] : kBadRow;
      // the row's requests and their use sit in one branch, so that no
      // request is left outstanding across rounds (the compiler then issues
      // them back to back instead of waiting before each)
      if (e != kBadRow && (imat == 0 || (spec_ok && (e >> 31)))) {
        u32x4 v[NU];
        load_row<NU>((imat ? a.wu : a.wg) + (size_t)(e & 0x7fffffffu) * U, U, lane, v);
        SI_TRACE_WAVE(0);
        float dt[BM];
        row_dots<BM, NU>(v, L.xs, U, lane, dt);
        if (lane == 0) {
#pragma unroll
          for (int t = 0; t < BM; ++t) L.dots[ir][imat][t] = dt[t];
        }
      }
      SI_TRACE_WAVE(1);
      // the item's W_down^T pieces go out once this wave's gate/up data is
      // in, so they stream behind the loads that h3 depends on (issued
      // before them, they would only delay h3: the requests of a wave
      // complete in order)
      if (first) issue_down(0);
      __syncthreads();
      if (wv == 0 && mr > 0) {  // rows of the round: one per lane (mr <= 8)
        bool any = no_as, spec = false;
        if (lane < mr) {
#pragma unroll
          for (int t = 0; t < BM; ++t) {
            const float h = fmaxf(L.dots[lane][0][t], 0.f);
            L.h1[lane][t] = h;
            any |= h > 0.f;
          }
          spec = spec_ok && (srow[lane] >> 31);
          L.need[lane] = (any && !spec) ? 1u : 0u;
        }
        const uint64_t late = __ballot(lane < mr && any && !spec);
        const uint64_t upr = __ballot(lane < mr && (any || spec));
        if (lane == 0) {
          L.n_late = __popcll(late);
          L.n_up += __popcll(upr);
        }
      }
      __syncthreads();
      if (mr > 0 && L.n_late) {  // W_up rows whose gate value asks for them
        if (imat == 1 && ir < mr && L.need[ir]) {
          u32x4 v[NU];
          load_row<NU>(a.wu + (size_t)(srow[ir] & 0x7fffffffu) * U, U, lane, v);
          float dt[BM];
          row_dots<BM, NU>(v, L.xs, U, lane, dt);
          if (lane == 0) {
#pragma unroll
            for (int t = 0; t < BM; ++t) L.dots[ir][1][t] = dt[t];
          }
        }
        __syncthreads();
      }
      for (int i = tid; i < mr * BM; i += kLThreads) {
        const int r = i / BM, t = i - r * BM;
        if (t < b) {
          const bool spec = spec_ok && (srow[r] >> 31);
          const float h = (L.need[r] || spec) ? L.h1[r][t] * L.dots[r][1][t] : 0.f;
          st_agent64(&a.h3e[(size_t)(srow[r] & 0x7fffffffu) * b + t], tagged(tag, __float_as_uint(h)));
        }
      }
      if (r0r + kRoundRows >= hi) break;
    }
    SI_TRACE_MARK(6);

    // ---- 3. down-projection of (tile, chunk)
    float acc[BM][8];
#pragma unroll
    for (int t = 0; t < BM; ++t)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[t][q] = 0.f;
    int n_down = 0;
    bool census_done = false;
    for (int q0 = 0; q0 < dN; q0 += kDownRound) {
      const int nq = min(kDownRound, dN - q0);
      if (q0 != 0) {
        __syncthreads();  // the previous round's h3 values have been used
        issue_down(q0);
      }
      // waves 0..3 collect the round's h3 words (slot = position x BM +
      // token, all requests in flight together); in the first round wave 4
      // checks the tile's zero flag and waves 8.. of block 0 take the census
      if (tid < kDownPollThreads) {
        constexpr int kPer = (kDownRound * BM + kDownPollThreads - 1) / kDownPollThreads;
        const uint64_t* src[kPer];
        int nv = 0;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
          const int j = tid + kDownPollThreads * i;
          const int q = j / BM, t = j - q * BM;
          const bool ok = q < nq && t < b;
          const int qc = ok ? q : 0;
          src[i] = a.h3e + (size_t)(L.ch.dent[q0 + qc] & 0x7fffffffu) * b + (ok ? t : 0);
          if (ok) nv = i + 1;  // slots of one thread are valid as a prefix
        }
        uint32_t hv[kPer];
        poll_words<kPer>(src, nv, tag, a.hdr, hv);
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
          const int j = tid + kDownPollThreads * i;
          if (j < kDownRound * BM) L.hs[j] = i < nv ? __uint_as_float(hv[i]) : 0.f;
        }
      } else if (q0 == 0 && wv == kDownPollThreads / kWave) {
        bool abort = false;
        poll_lane(&a.zflag[tile], lane == 0, tag, a.hdr, abort);
        if (lane == 0 && !abort) L.zok = 1;
      } else if (q0 == 0 && blk == 0 && wv >= kLWaves / 2) {
        // every block's kept count: the call's count, and proof that every
        // block has read the call counter
        int sum = 0;
        for (int o = tid - kLThreads / 2; o < P; o += kLThreads / 2) {
          const uint64_t* src[1] = {&a.pub[(size_t)o * kOwnPubStride + kCountWord]};
          uint32_t v[1];
          poll_words<1>(src, 1, tag, a.hdr, v);
          sum += (int)v[0];
        }
        sum = wave_sum_int(sum);
        if (lane == 0) L.wsum[wv] = sum;
      }
      __syncthreads();
      if (q0 == 0 && blk == 0) {
        if (tid == 0) {
          int n = 0;
          for (int w = kLWaves / 2; w < kLWaves; ++w) n += L.wsum[w];
          if (a.n_out) *a.n_out = n;
          advance_epoch(a.hdr, epoch);
        }
        census_done = true;
      }
      if (q0 == 0) SI_TRACE_WAVE(3);
#pragma unroll
      for (int j = 0; j < kDN; ++j) {
        const int q = wv + kLWaves * j;
        float hv[BM];
        bool nz = false;
#pragma unroll
        for (int t = 0; t < BM; ++t) {
          hv[t] = (q < nq && t < b) ? L.hs[q * BM + t] : 0.f;
          nz |= hv[t] != 0.f;
        }
        if (q < nq && !((dloaded >> j) & 1u) && nz) {  // late request
          const uint32_t e = L.ch.dent[q0 + q];
          if (dcol_ok) vd[j] = load_nt(a.wdt + (size_t)(e & 0x7fffffffu) * U + dunit);
          dloaded |= 1u << j;
        }
        const f16x2 p0 = as_h2(vd[j].x), p1 = as_h2(vd[j].y), p2 = as_h2(vd[j].z), p3 = as_h2(vd[j].w);
        const float f[8] = {(float)p0.x, (float)p0.y, (float)p1.x, (float)p1.y,
                            (float)p2.x, (float)p2.y, (float)p3.x, (float)p3.y};
#pragma unroll
        for (int t = 0; t < BM; ++t)
#pragma unroll
          for (int qq = 0; qq < 8; ++qq) acc[t][qq] = fmaf(hv[t], f[qq], acc[t][qq]);
      }
      n_down += __popc(dloaded);
      if (q0 == 0) SI_TRACE_WAVE(4);
    }
    // per-wave partial tiles folded in LDS (plain stores; x is no longer
    // needed): kFold waves store, the others add in turn
    constexpr int kFold = OwnedLds<BM, NU>::kFold;
    if (dN > 0) {
#pragma unroll
      for (int pass = 0; pass < kLWaves / kFold; ++pass) {
        if (wv / kFold == pass) {
          const int s = wv - pass * kFold;
#pragma unroll
          for (int t = 0; t < BM; ++t)
#pragma unroll
            for (int q = 0; q < 8; ++q) {
              float& dst = L.dpart[s][t][lane * 8 + q];
              dst = pass == 0 ? acc[t][q] : dst + acc[t][q];
            }
        }
        if (pass + 1 < kLWaves / kFold) __syncthreads();
      }
    }
    if (lane == 0 && tile == 0 && n_down) atomicAdd(&L.n_down, n_down);
    SI_TRACE_MARK(8);
    __syncthreads();

    // ---- the item's tile into y (its owner zeroed it in this call)
    if (dN > 0) {
      if (tid == 0 && !L.zok) {  // only after a timed-out poll
        long spins = 0;
        while ((uint32_t)(ld_agent64(&a.zflag[tile]) >> 32) != tag) {
          if (++spins > kPollLimit) {
            atomicOr(&a.hdr[H_ERR], kErrLookbackSpin);
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      __syncthreads();
      SI_TRACE_MARK(9);
      for (int i = tid; i < b * kTile; i += kLThreads) {
        const int t = i / kTile, c = i - t * kTile, col = tile * kTile + c;
        float v = 0.f;
#pragma unroll
        for (int s = 0; s < kFold; ++s) v += L.dpart[s][t][c];
        if (col < d && v != 0.f) unsafeAtomicAdd(&a.y[(size_t)t * d + col], v);
      }
    }
    if (blk == 0 && !census_done) {
      int sum = 0;
      for (int o = tid; o < P; o += kLThreads) {
        const uint64_t* src[1] = {&a.pub[(size_t)o * kOwnPubStride + kCountWord]};
        uint32_t v[1];
        poll_words<1>(src, 1, tag, a.hdr, v);
        sum += (int)v[0];
      }
      sum = block_sum(L, sum, lane, wv);
      if (tid == 0) {
        if (a.n_out) *a.n_out = sum;
        advance_epoch(a.hdr, epoch);
      }
    }
    if (tid == 0) {
      a.counts[2 * blk] = L.n_up;
      a.counts[2 * blk + 1] = L.n_down;
    }
  } else if (blk == 0) {  // the predictor alone: the census of block 0
    int sum = 0;
    for (int o = tid; o < P; o += kLThreads) {
      const uint64_t* src[1] = {&a.pub[(size_t)o * kOwnPubStride + kCountWord]};
      uint32_t v[1];
      poll_words<1>(src, 1, tag, a.hdr, v);
      sum += (int)v[0];
    }
    sum = block_sum(L, sum, lane, wv);
    if (tid == 0) {
      if (a.n_out) *a.n_out = sum;
      advance_epoch(a.hdr, epoch);
    }
  }

  // ---- the ascending kept list: the counts of the blocks before this one
  if (a.idx) {
    int sum = 0;
    for (int o = tid; o < blk; o += kLThreads) {
      const uint64_t* src[1] = {&a.pub[(size_t)o * kOwnPubStride + kCountWord]};
      uint32_t v[1];
      poll_words<1>(src, 1, tag, a.hdr, v);
      sum += (int)v[0];
    }
    const int before = block_sum(L, sum, lane, wv);
    for (int q = tid; q < n_own; q += kLThreads) a.idx[before + q] = (int32_t)(L.srow[q] & 0x7fffffffu);
  }
  SI_TRACE_MARK(10);
  SI_TRACE_FLUSH;
}

// Rows per block: the rows spread over the whole groups of the grid,
// rounded up to a multiple of 8 so that a block's piece of each sign unit
// (R * 16 bytes) starts and ends on a 128-byte line.
static int owned_rows_per_block(int k, int P, int tiles) {
  const int working = P / tiles * tiles;
  const int R = (k + working - 1) / working;
  return (R + 7) / 8 * 8;
}

template <int BM, int NU>
static int owned_blocks() {
  static int blocks = -1;
  if (blocks < 0) {
    blocks = 0;
    constexpr int lds = owned_lds_bytes<BM, NU>();
    if constexpr (lds <= kMaxLds) {
      int dev = 0, cus = 0, per_cu = 0;
      const void* fn = reinterpret_cast<const void*>(&k_owned<BM, NU>);
      if (hipGetDevice(&dev) != hipSuccess) return 0;
      if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
      if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess) return 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kLThreads, lds) != hipSuccess) return 0;
      if (per_cu >= 1) blocks = cus < kMaxLayerBlocks ? cus : kMaxLayerBlocks;
    }
  }
  return blocks;
}

template <int BM, int NU>
static hipError_t owned_b(const LayerCall& c, hipStream_t s) {
  if constexpr (owned_lds_bytes<BM, NU>() > kMaxLds) {
    return hipErrorInvalidConfiguration;
  } else {
    const int k = c.k, d = c.d;
    const WsLayout L = ws_layout(k, c.b);
    char* base = static_cast<char*>(c.ws);
    const int P = owned_blocks<BM, NU>();
    if (P < 1) return hipErrorInvalidConfiguration;
    OwnedArgs a;
    a.signs = reinterpret_cast<const u32x4*>(c.signs);
    a.wg = reinterpret_cast<const u32x4*>(c.w_gate);
    a.wu = reinterpret_cast<const u32x4*>(c.w_up);
    a.wdt = reinterpret_cast<const u32x4*>(c.w_down_t);
    a.x = c.x;
    a.mask_in = c.mask_in;
    a.k = k;
    a.d = d;
    a.b = c.b;
    a.T = c.T;
    a.margin = c.margin;
    a.flags = c.flags;
    a.mlp = c.y != nullptr;
    a.tiles = (d + kTile - 1) / kTile;
    a.R = owned_rows_per_block(k, P, a.tiles);
    a.groups = min(P / a.tiles, (k + a.R * a.tiles - 1) / (a.R * a.tiles));
    a.nsub = (a.R + kWave - 1) / kWave;
    a.mask = c.mask;
    a.idx = c.idx;
    a.n_out = c.n_out;
    a.hdr = reinterpret_cast<uint32_t*>(base);
    a.pub = reinterpret_cast<uint64_t*>(base + L.opub);
    a.h3e = reinterpret_cast<uint64_t*>(base + L.h3e);
    a.zflag = reinterpret_cast<uint64_t*>(base + L.zflag);
    a.counts = reinterpret_cast<int32_t*>(base + L.counts);
    a.y = c.y;
    k_owned<BM, NU><<<P, kLThreads, owned_lds_bytes<BM, NU>(), s>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !c.counters || !c.y) return e;
    return launch_sum_counts(a.counts, P, c.n_out, k, c.counters, s);
  }
}

static int owned_blocks_for(int d, int b) {
  if (b < 1 || b > kMaxB) return 0;
#define BLOCKS(BM, NU) owned_blocks<BM, NU>()
  SI_LAYER_DISPATCH(BLOCKS)
#undef BLOCKS
}

// The row-owning kernel applies when every block's rows fit its passes, a
// group's (owner block, pass) pairs fit one wave and its rows the LDS list,
// and one block per CU can be resident with the LDS that the batch and row
// width need.
bool owned_supported(int k, int d, int b) {
  const int P = owned_blocks_for(d, b);
  const int tiles = (d + kTile - 1) / kTile;
  if (P < 1 || P < tiles) return false;
  const int R = owned_rows_per_block(k, P, tiles);
  if (R > kMaxOwnRows) return false;
  const int nsub = (R + kWave - 1) / kWave;
  return tiles * nsub <= kMaxPairs && tiles * R <= kMaxChunkRows;
}

hipError_t launch_owned(const LayerCall& c, hipStream_t s) {
  const int d = c.d, b = c.b;
#define LAUNCH(BM, NU) owned_b<BM, NU>(c, s)
  SI_LAYER_DISPATCH(LAUNCH)
#undef LAUNCH
}

}  // namespace si
