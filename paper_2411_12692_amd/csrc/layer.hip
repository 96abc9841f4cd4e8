// The whole per-token MLP path of one layer in a single kernel: sign-bit
// prediction (Section IV-A, Eq. (2)), ordered compaction, sparse gate/up with
// actual sparsity and sparse down-projection (Section IV-B 3)-4)).
//
// One block of 12 wavefronts per group of 64 rows; all blocks are resident
// at once (the host takes this path only when they fit).  Groups are cut
// into chunks of consecutive groups; a down-projection work item is a
// (512-column tile of y, chunk) pair, at most one per block.
//
//  all waves    issue the group's packed-sign loads first, stage x in LDS,
//               pack its sign words and add their XOR/popcount partials.
//  wave 0       applies Eq. (2) (kept iff N_neg < T), writes the mask,
//               publishes the group's kept and "confident" masks (rows with
//               N_neg < T - margin, almost surely active), then places the
//               group in the ascending kept list with a wave-wide look-back.
//  waves 1-7    gate/up: the kept rows of the block's chunk are split evenly
//               over the chunk's blocks (balancing groups with many kept
//               rows); for each row the W_gate row is streamed and the W_up
//               row too where some token's ReLU output is positive (requested
//               together with W_gate for confident rows); h3 is published
//               per chunk position.
//  waves 8-11   down-projection of the block's item: they read the chunk's
//               masks, request the W_down^T row segments of the confident
//               rows at once (overlapping the gate/up traffic), collect h3
//               and finish the other rows, reduce in LDS and add the tile
//               into y with fp32 atomics once block `tile` has zeroed it.
//
// Blocks exchange data through epoch-tagged 64-bit words (tag = per-call
// counter with the high bit set, in the high half; payload in the low half)
// written with agent-scope write-through stores and polled one word per lane
// with agent-scope loads: a word is valid once it carries the call's tag, so
// no cache flush or fence is needed and the workspace is never cleared
// between calls.  Every poll has a spin limit that sets an error bit instead
// of hanging.
#include "si_device.h"
#include "si_launch.h"

namespace si {

#ifdef SI_TRACE
__device__ uint64_t g_si_trace[1024 * kTraceSlots];
extern "C" hipError_t si_trace_read(void* dst, size_t bytes) {
  return hipMemcpyFromSymbol(dst, HIP_SYMBOL(g_si_trace), bytes, 0, hipMemcpyDeviceToHost);
}
#endif

constexpr int kLayerWaves = 12;
constexpr int kLayerThreads = kLayerWaves * kWave;
constexpr int kLayerMaxB = 2;  // larger batches take the two-kernel path (register budget)
constexpr int kGateWaves = 7;  // waves 1..7: gate/up; wave 0: decisions and compaction
constexpr int kDownWaves = 4;  // waves 8..11: down-projection
constexpr int kMaxSignUnitsPerWave = kMaxD / 128 / kLayerWaves;  // 4
constexpr long kPollLimit = 1l << 16;
constexpr uint32_t kNoAS = 1u, kNoSpec = 2u;

constexpr uint64_t kFlagAggregate = 1ull << 30;
constexpr uint64_t kFlagPrefix = 2ull << 30;
constexpr uint64_t kFlagMask = 3ull << 30;

struct LayerArgs {
  const u32x4* signs;
  const u32x4* wg;
  const u32x4* wu;
  const u32x4* wdt;
  const uint16_t* x;
  int k, d, T, margin;
  uint32_t flags;
  uint8_t* mask;
  int32_t* idx;
  int32_t* n_out;
  uint32_t* hdr;
  uint64_t* status;  // [groups] look-back words
  uint64_t* lmask;   // [groups][4] tag | kept mask low/high half, tag | confident mask low/high half
  uint64_t* h3e;     // [groups][64][B] tag | fp32 bits, by rank in the group's kept list
  uint64_t* zflag;   // [tiles] tag once the tile of y is zero
  uint32_t* ready;   // [2 parities][2][groups]: per chunk, groups whose masks / h3 are published
  int32_t* counts;   // [groups][2] W_up rows read, W_down^T rows read (tile-0 items)
  float* y;
  int tiles, chunks, gpc;
};

__device__ inline uint64_t tagged(uint32_t tag, uint32_t payload) { return ((uint64_t)tag << 32) | payload; }

// Poll one tagged word per lane (lanes may use different addresses) until it
// carries `tag`; returns the payload.  After a timeout the wave
// stops waiting (`abort`) and the error bit is set.
__device__ inline uint32_t poll_lane(const uint64_t* p, bool active, uint32_t tag, uint32_t* hdr, bool& abort) {
  uint32_t out = 0;
  bool pending = active;
  long spins = 0;
  while (__ballot(pending) && !abort) {
    if (pending) {
      const uint64_t v = ld_agent64(p);
      if ((uint32_t)(v >> 32) == tag) {
        out = (uint32_t)v;
        pending = false;
      }
    }
    if (__ballot(pending)) {
      if (++spins > kPollLimit) {
        abort = true;
        if (pending) atomicOr(&hdr[H_ERR], kErrLookbackSpin);
#ifdef SI_TRACE
        if (pending) {  // block, wave, word index, last seen tag, expected tag
          const uint64_t v = ld_agent64(p);
          g_si_trace[(size_t)blockIdx.x * kTraceSlots + 26] = blockIdx.x;
          g_si_trace[(size_t)blockIdx.x * kTraceSlots + 27] = threadIdx.x >> 6;
          g_si_trace[(size_t)blockIdx.x * kTraceSlots + 28] = (uint64_t)(size_t)p;
          g_si_trace[(size_t)blockIdx.x * kTraceSlots + 29] = v >> 32;
          g_si_trace[(size_t)blockIdx.x * kTraceSlots + 30] = tag;
        }
#endif
      } else {
        __builtin_amdgcn_s_sleep(1);
      }
    }
  }
  return out;
}

// Poll N*S wave-uniform tagged words at once (all requests in flight
// together) until each carries `tag`: word (r, t) lives at
// base[off[r] * S + t].  Entries r with bit r of `want` clear are skipped.
template <int N, int S>
__device__ inline void poll_batch(const uint64_t* base, const uint32_t (&off)[N], uint32_t want, uint32_t tag,
                                  uint32_t (&out)[N][S], uint32_t* hdr, bool& abort) {
  static_assert(N * S <= 64, "batch too large");
  uint64_t pending = 0;
#pragma unroll
  for (int r = 0; r < N; ++r)
    if ((want >> r) & 1) pending |= ((S == 64 ? ~0ull : ((1ull << S) - 1ull))) << (r * S);
  long spins = 0;
  while (pending && !abort) {
    uint64_t v[N][S];
#pragma unroll
    for (int r = 0; r < N; ++r)
#pragma unroll
      for (int t = 0; t < S; ++t)
        if ((pending >> (r * S + t)) & 1) v[r][t] = ld_agent64(base + (size_t)off[r] * S + t);
#pragma unroll
    for (int r = 0; r < N; ++r)
#pragma unroll
      for (int t = 0; t < S; ++t)
        if (((pending >> (r * S + t)) & 1) && (uint32_t)(v[r][t] >> 32) == tag) {
          out[r][t] = (uint32_t)v[r][t];
          pending &= ~(1ull << (r * S + t));
        }
    if (pending) {
      if (++spins > kPollLimit) {
        abort = true;
        atomicOr(&hdr[H_ERR], kErrLookbackSpin);
      } else {
        __builtin_amdgcn_s_sleep(1);
      }
    }
  }
}

// Index of the n-th (0-based) set bit of m; m must have more than n bits set.
__device__ inline int nth_set_bit(uint64_t m, int n) {
  int pos = 0;
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) {
    const uint64_t low = m & ((1ull << s) - 1ull);
    const int c = __popcll(low);
    if (n >= c) {
      n -= c;
      m >>= s;
      pos += s;
    } else {
      m = low;
    }
  }
  return pos;
}

// Wait until a readiness counter reaches `target` (one lane polls).
__device__ inline void wait_count(const uint32_t* p, uint32_t target, uint32_t* hdr, bool& abort) {
  if (abort) return;
  long spins = 0;
  while (ld_agent(p) < target) {
    if (++spins > kPollLimit) {
      abort = true;
      atomicOr(&hdr[H_ERR], kErrLookbackSpin);
      return;
    }
    __builtin_amdgcn_s_sleep(4);
  }
}

// Wave-wide look-back over the groups' posted counts (see predict.hip).
__device__ int layer_lookback(const uint64_t* status, int v, uint32_t tag, int lane, uint32_t* hdr) {
  int excl = 0;
  int j = v - 1;
  long spins = 0;
  while (j >= 0) {
    const int jj = j - lane;
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
      if (++spins > kPollLimit) {
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

// Gate/up of one kept row; `spec` requests the W_up row together with the
// W_gate row.  Returns h3 for the B tokens (in every lane) and whether the
// W_up row was read.
// Kept rows of a chunk of consecutive groups, as published by the groups'
// mask words.  Lane l < ng describes group g0 + l.
struct ChunkView {
  int g0, ng, E;    // first group, groups, kept rows of the chunk
  int pre_l;        // inclusive prefix of the kept counts up to this lane's group
  uint64_t kept_l;  // kept mask of this lane's group
  uint64_t conf_l;  // confident mask of this lane's group
};

__device__ inline ChunkView load_chunk(const uint64_t* lmask, int chunk, int gpc, int groups, uint32_t tag,
                                       uint32_t* hdr, bool& abort, int lane) {
  ChunkView c;
  c.g0 = chunk * gpc;
  c.ng = max(0, min(c.g0 + gpc, groups) - c.g0);
  const bool mw = lane < 4 * c.ng;
  const uint32_t mword = poll_lane(&lmask[(size_t)c.g0 * 4 + (mw ? lane : 0)], mw, tag, hdr, abort);
  const int gl = lane < c.ng ? lane : 0;
  c.kept_l = (uint64_t)__shfl(mword, 4 * gl, kWave) | ((uint64_t)__shfl(mword, 4 * gl + 1, kWave) << 32);
  c.conf_l = (uint64_t)__shfl(mword, 4 * gl + 2, kWave) | ((uint64_t)__shfl(mword, 4 * gl + 3, kWave) << 32);
  int pre = lane < c.ng ? __popcll(c.kept_l) : 0;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int v = __shfl_up(pre, o, kWave);
    if (lane >= o) pre += v;
  }
  c.pre_l = pre;
  const int last = __shfl(pre, c.ng > 0 ? c.ng - 1 : 0, kWave);
  c.E = c.ng > 0 ? last : 0;
  return c;
}

// Entry (conf << 31 | row) at position p (< E) of the chunk's kept list; p
// may differ between lanes.  All lanes must call it.
__device__ inline uint32_t chunk_entry(const ChunkView& c, int p) {
  int gi = 0;
  for (int gg = 0; gg < c.ng; ++gg) gi += (__shfl(c.pre_l, gg, kWave) <= p) ? 1 : 0;
  gi = min(gi, max(c.ng - 1, 0));
  // every lane takes part in the shuffles: reading an inactive lane yields 0
  const int pre_before = __shfl(c.pre_l, gi > 0 ? gi - 1 : 0, kWave);
  const int li = p - (gi > 0 ? pre_before : 0);
  const uint64_t km = __shfl(c.kept_l, gi, kWave);
  const uint64_t cm = __shfl(c.conf_l, gi, kWave);
  const int bit = (li >= 0 && li < __popcll(km)) ? nth_set_bit(km, li) : 0;
  return (uint32_t)((c.g0 + gi) * kRowGroup + bit) | (((cm >> bit) & 1ull) ? 0x80000000u : 0u);
}

// Gate/up of up to R kept rows at once (all their row requests in flight
// together).  Row r is valid for r < n.  spec[r] requests the W_up row with
// the W_gate row.  Returns h3 per row and token (in every lane) and whether
// the W_up row was read.
template <int B, int NU, int R>
__device__ inline void gate_up_rows(const u32x4* __restrict__ wg, const u32x4* __restrict__ wu,
                                    const int (&row)[R], const bool (&spec)[R], int n, int U, const u32x4* xs,
                                    int lane, bool no_as, float (&h)[R][B], bool (&up)[R]) {
  u32x4 a[R][NU], c[R][NU];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (r < n) {
      const u32x4* gr = wg + (size_t)row[r] * U;
#pragma unroll
      for (int j = 0; j < NU; ++j) {
        const int u = lane + kWave * j;
        if (u < U) a[r][j] = load_nt(gr + u);
      }
      if (spec[r]) {
        const u32x4* ur = wu + (size_t)row[r] * U;
#pragma unroll
        for (int j = 0; j < NU; ++j) {
          const int u = lane + kWave * j;
          if (u < U) c[r][j] = load_nt(ur + u);
        }
      }
    }
  }
  float g[R][B];
  bool need[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
#pragma unroll
    for (int t = 0; t < B; ++t) g[r][t] = 0.f;
    need[r] = false;
    if (r < n) {
#pragma unroll
      for (int j = 0; j < NU; ++j) {
        const int u = lane + kWave * j;
        if (u < U) {
#pragma unroll
          for (int t = 0; t < B; ++t) g[r][t] = dot8(a[r][j], xs[t * U + u], g[r][t]);
        }
      }
      bool any = false;
#pragma unroll
      for (int t = 0; t < B; ++t) {
        g[r][t] = fmaxf(wave_sum(g[r][t]), 0.f);
        any |= g[r][t] > 0.f;
      }
      need[r] = any || no_as;
      up[r] = need[r] || spec[r];
      // late W_up request where the gate value asks for it
      if (need[r] && !spec[r]) {
        const u32x4* ur = wu + (size_t)row[r] * U;
#pragma unroll
        for (int j = 0; j < NU; ++j) {
          const int u = lane + kWave * j;
          if (u < U) c[r][j] = load_nt(ur + u);
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
#pragma unroll
    for (int t = 0; t < B; ++t) h[r][t] = 0.f;
    if (r < n && need[r]) {
      float uu[B];
#pragma unroll
      for (int t = 0; t < B; ++t) uu[t] = 0.f;
#pragma unroll
      for (int j = 0; j < NU; ++j) {
        const int u = lane + kWave * j;
        if (u < U) {
#pragma unroll
          for (int t = 0; t < B; ++t) uu[t] = dot8(c[r][j], xs[t * U + u], uu[t]);
        }
      }
#pragma unroll
      for (int t = 0; t < B; ++t) h[r][t] = g[r][t] * wave_sum(uu[t]);
    }
  }
}

// Rows handled together by one gate/up wave (bounded by registers).
template <int B, int NU>
constexpr int gate_rows_in_flight() { return (B == 1 && NU <= 8) ? 2 : 1; }

template <int B, int NU>
__global__ __launch_bounds__(kLayerThreads) void k_layer(LayerArgs a) {
  constexpr int kDownBatch = kWave / 4;  // entries polled per batch by one down wave (one per lane)
  extern __shared__ u32x4 xs[];           // [B][d/8] fp16 tokens
  __shared__ __attribute__((aligned(16))) uint32_t xw[B * (kMaxD / 32)];
  __shared__ int cnt[B][kWave];
  __shared__ uint32_t kept[kRowGroup];  // conf << 31 | row
  __shared__ float red[B][kTile];
  __shared__ int s_nkept, s_up, s_down, s_adone;
  __shared__ uint32_t s_epoch;

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d = a.d, U = d >> 3, W = d >> 5, units = W >> 2;
  const int g = blockIdx.x, groups = gridDim.x;
  const int items = a.tiles * a.chunks;
  const bool has_item = g < items;
  const int tile = g % a.tiles, chunk = g / a.tiles;

  if (wv == 0) SI_TRACE_MARK(0);
#ifdef SI_TRACE
  if (tid == 0) g_si_trace[(size_t)blockIdx.x * kTraceSlots + 31] = (uint64_t)(size_t)a.h3e;
#endif
  // ---- packed-sign loads of this group, issued before anything else
  u32x4 sreg[kMaxSignUnitsPerWave];
  const u32x4* sg = a.signs + (size_t)g * units * kRowGroup + lane;
#pragma unroll
  for (int i = 0; i < kMaxSignUnitsPerWave; ++i) {
    const int q = wv + kLayerWaves * i;
    if (q < units) sreg[i] = load_nt(sg + (size_t)q * kRowGroup);
  }

  // ---- tokens -> LDS; clear the LDS accumulators; zero this block's tile of y
  for (int i = tid; i < B * U; i += kLayerThreads) xs[i] = reinterpret_cast<const u32x4*>(a.x)[i];
  for (int i = tid; i < B * kWave; i += kLayerThreads) (&cnt[0][0])[i] = 0;
  for (int i = tid; i < B * kTile; i += kLayerThreads) (&red[0][0])[i] = 0.f;
  if (tid == 0) {
    s_up = 0;
    s_down = 0;
    s_adone = 0;
    s_epoch = ld_agent(&a.hdr[H_EPOCH]);
  }
  const bool owns_tile = g < a.tiles;
  if (g == 0) {
    // the next call's readiness counters start from zero (this call's were
    // cleared by the previous call, or by the zero-filled workspace)
    const uint32_t nxt = (ld_agent(&a.hdr[H_EPOCH]) + 1u) & 1u;
    for (int i = tid; i < 2 * groups; i += kLayerThreads) a.ready[(size_t)nxt * 2 * groups + i] = 0u;
  }
  if (owns_tile) {
    for (int i = tid; i < B * kTile; i += kLayerThreads) {
      const int t = i / kTile, col = g * kTile + (i - t * kTile);
      if (col < d) __hip_atomic_store(&a.y[(size_t)t * d + col], 0.f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    wait_own_stores();
  }
  __syncthreads();
  const uint32_t epoch = s_epoch;
  const uint32_t tag = epoch_tag(epoch);
  if (wv == 0) SI_TRACE_MARK(1);
  if (owns_tile && tid == 0) st_agent64(&a.zflag[g], tagged(tag, 1u));
  for (int i = tid; i < B * W; i += kLayerThreads) {
    const int t = i / W, w = i - t * W;
    xw[i] = sign_word(&xs[t * U + 4 * w]);
  }
  __syncthreads();

  // ---- N_neg partial counts (XOR + popcount) added in LDS
  {
    int c[B];
#pragma unroll
    for (int t = 0; t < B; ++t) c[t] = 0;
    bool any_unit = false;
#pragma unroll
    for (int i = 0; i < kMaxSignUnitsPerWave; ++i) {
      const int q = wv + kLayerWaves * i;
      if (q < units) {
        any_unit = true;
#pragma unroll
        for (int t = 0; t < B; ++t) {
          const u32x4 xv = *reinterpret_cast<const u32x4*>(&xw[t * W + 4 * q]);
          c[t] += __popc(sreg[i].x ^ xv.x) + __popc(sreg[i].y ^ xv.y) + __popc(sreg[i].z ^ xv.z) +
                  __popc(sreg[i].w ^ xv.w);
        }
      }
    }
    if (any_unit) {
#pragma unroll
      for (int t = 0; t < B; ++t) atomicAdd(&cnt[t][lane], c[t]);
    }
  }
  __syncthreads();
  if (wv == 0) SI_TRACE_MARK(2);

  // ---- wave 0: Eq. (2), mask, kept list, publication
  if (wv == 0) {
    const int row = g * kRowGroup + lane;
    bool keep = false, conf = false;
#pragma unroll
    for (int t = 0; t < B; ++t) {
      const int n_neg = cnt[t][lane];
      keep |= n_neg < a.T;
      conf |= n_neg < a.T - a.margin;
    }
    keep = keep && row < a.k;
    if (row < a.k) a.mask[row] = keep ? 1 : 0;
    const uint64_t ballot = __ballot(keep);
    const int nk = __popcll(ballot);
    const int rank = __popcll(ballot & lanes_below(lane));
    const uint64_t cballot = __ballot(keep && conf);
    if (keep) kept[rank] = (conf ? 0x80000000u : 0u) | (uint32_t)row;
    if (lane < 4) {
      const uint64_t m = lane < 2 ? ballot : cballot;
      st_agent64(&a.lmask[(size_t)g * 4 + lane], tagged(tag, (uint32_t)(m >> (32 * (lane & 1)))));
    }
    wait_own_stores();
    if (lane == 0) {
      s_nkept = nk;
      st_agent64(&a.status[g], tagged(tag, (uint32_t)((g == 0 ? kFlagPrefix : kFlagAggregate) | (uint64_t)nk)));
      __hip_atomic_fetch_add(&a.ready[(size_t)(epoch & 1u) * 2 * groups + g / a.gpc], 1u, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  if (wv == 0) SI_TRACE_MARK(3);
  const int nkept = s_nkept;
  const bool no_as = (a.flags & kNoAS) != 0;

  if (wv == 0) {
    // ---- ordered compaction: every group posted its count right after
    // counting, so the look-back completes in a few round trips
    const int excl = g == 0 ? 0 : layer_lookback(a.status, g, tag, lane, a.hdr);
    if (lane == 0 && g > 0)
      st_agent64(&a.status[g], tagged(tag, (uint32_t)(kFlagPrefix | (uint64_t)(excl + nkept))));
    if (lane < nkept && a.idx) a.idx[excl + lane] = (int32_t)(kept[lane] & 0x7fffffffu);
    if (lane == 0 && g == groups - 1) {
      if (a.n_out) *a.n_out = excl + nkept;
      st_agent(&a.hdr[H_EPOCH], epoch + 1u);  // every group has posted: all blocks read this epoch
    }
    SI_TRACE_MARK(4);
#ifdef SI_TRACE
    if (lane == 0) g_si_trace[(size_t)blockIdx.x * kTraceSlots + 19] = nkept;
#endif
  } else if (wv <= kGateWaves) {
    // ---- gate/up, balanced inside the chunk of groups this group belongs
    // to: the chunk's kept rows (concatenated in group order) are split
    // evenly over its blocks, so a group with many kept rows does not hold
    // its chunk back.  Waves 1..7 take this block's positions round-robin,
    // R rows in flight per wave.
    constexpr int R = gate_rows_in_flight<B, NU>();
    constexpr int NGW = kGateWaves;
    bool abort = false;
    const ChunkView cv = load_chunk(a.lmask, g / a.gpc, a.gpc, groups, tag, a.hdr, abort, lane);
    const int mine = g - cv.g0;
    const int p_lo = (int)((long long)cv.E * mine / max(cv.ng, 1));
    const int p_hi = (int)((long long)cv.E * (mine + 1) / max(cv.ng, 1));
    int n_up = 0;
    const bool spec_ok = !(a.flags & kNoSpec) && NU <= 10;
    for (int i0 = p_lo + wv - 1; i0 < p_hi && !abort; i0 += NGW * R) {
      int rows[R];
      bool spec[R];
      int n = 0;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = i0 + NGW * r;
        const uint32_t e = chunk_entry(cv, i < p_hi ? i : p_lo);
        rows[r] = (int)(e & 0x7fffffffu);
        spec[r] = spec_ok && (e >> 31) != 0;
        if (i < p_hi) n = r + 1;
      }
      float h[R][B];
      bool up[R];
      gate_up_rows<B, NU, R>(a.wg, a.wu, rows, spec, n, U, xs, lane, no_as, h, up);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (r < n) {
          const int i = i0 + NGW * r;
          n_up += up[r] ? 1 : 0;
#pragma unroll
          for (int t = 0; t < B; ++t)
            if (lane == t)
              st_agent64(&a.h3e[((size_t)cv.g0 * kRowGroup + i) * B + t], tagged(tag, __float_as_uint(h[r][t])));
        }
      }
    }
    wait_own_stores();
    if (lane == 0) {
      if (n_up) atomicAdd(&s_up, n_up);
      if (atomicAdd(&s_adone, 1) == NGW - 1)  // last gate/up wave of the block
        __hip_atomic_fetch_add(&a.ready[(size_t)(epoch & 1u) * 2 * groups + groups + g / a.gpc], 1u,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    SI_TRACE_MARK(4 + wv);  // 5 .. 11
  } else if (has_item) {
    // ---- down-projection of (tile, chunk): this wave takes the chunk's list
    // positions [16 m + 64 j + 16 wb, +16), one entry per lane
    const int wb = wv - (kLayerWaves - kDownWaves);
    const int unit = tile * (kTile / 8) + lane;  // 16-byte unit of a W_down^T row: 8 columns
    const bool col_ok = unit < U;
    bool abort = false;
    const ChunkView cv = load_chunk(a.lmask, chunk, a.gpc, groups, tag, a.hdr, abort, lane);
    const int E = cv.E;
    if (wb == 0) SI_TRACE_MARK(12);
    float acc[B][8];
#pragma unroll
    for (int t = 0; t < B; ++t)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[t][q] = 0.f;
    int n_down = 0;
    const bool spec_ok = !(a.flags & kNoSpec);
    for (int base = wb * kDownBatch; base < E && !abort; base += kDownWaves * kDownBatch) {
      // lane r < 16 owns list position base + r
      const int p = base + lane;
      const bool mine = lane < kDownBatch && p < E;
      const uint32_t e = chunk_entry(cv, mine ? p : 0);
      const uint32_t off = (uint32_t)(cv.g0 * kRowGroup + p);  // h3 of position p
      if (wb == 0 && base == 0) SI_TRACE_MARK(13);
      const int nb = min(kDownBatch, E - base);
      u32x4 w[kDownBatch];
      uint32_t loaded = 0;
#pragma unroll
      for (int r = 0; r < kDownBatch; ++r) {
        w[r] = u32x4{0, 0, 0, 0};
        const uint32_t er = __shfl(e, r, kWave);
        const int row = (int)(er & 0x7fffffffu);
        if (r < nb && !abort && (unsigned)row < (unsigned)a.k && ((spec_ok && (er >> 31)) || no_as)) {
          if (col_ok) w[r] = load_nt(a.wdt + (size_t)row * U + unit);
          loaded |= 1u << r;
        }
      }
      float hl[B];
#pragma unroll
      for (int t = 0; t < B; ++t)
        hl[t] = __uint_as_float(poll_lane(&a.h3e[mine ? (size_t)off * B + t : 0], mine, tag, a.hdr, abort));
      if (wb == 0 && base == 0) SI_TRACE_MARK(14);
      float hv[kDownBatch][B];
#pragma unroll
      for (int r = 0; r < kDownBatch; ++r) {
        bool nz = false;
#pragma unroll
        for (int t = 0; t < B; ++t) {
          const float hr = __shfl(hl[t], r, kWave);
          hv[r][t] = (r < nb && !abort) ? hr : 0.f;
          nz |= hv[r][t] != 0.f;
        }
        const uint32_t er = __shfl(e, r, kWave);
        const int row = (int)(er & 0x7fffffffu);
        if (r < nb && !((loaded >> r) & 1) && nz && (unsigned)row < (unsigned)a.k) {
          if (col_ok) w[r] = load_nt(a.wdt + (size_t)row * U + unit);
          loaded |= 1u << r;
        }
      }
      n_down += __popc(loaded);
#pragma unroll
      for (int r = 0; r < kDownBatch; ++r) {
        const f16x2 p0h = as_h2(w[r].x), p1h = as_h2(w[r].y), p2h = as_h2(w[r].z), p3h = as_h2(w[r].w);
        const float f[8] = {(float)p0h.x, (float)p0h.y, (float)p1h.x, (float)p1h.y,
                            (float)p2h.x, (float)p2h.y, (float)p3h.x, (float)p3h.y};
#pragma unroll
        for (int t = 0; t < B; ++t)
#pragma unroll
          for (int q = 0; q < 8; ++q) acc[t][q] = fmaf(hv[r][t], f[q], acc[t][q]);
      }
    }
    if (col_ok) {
#pragma unroll
      for (int t = 0; t < B; ++t)
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (acc[t][q] != 0.f) atomicAdd(&red[t][lane * 8 + q], acc[t][q]);
    }
    if (lane == 0 && tile == 0 && n_down) atomicAdd(&s_down, n_down);
    SI_TRACE_MARK(15 + wb);  // 15 .. 18
  }
  __syncthreads();
  if (wv == 0) SI_TRACE_MARK(23);

  // ---- add the block's tile into y once block `tile` has zeroed it
  if (has_item) {
    if (wv == 0 && lane == 0) {
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
    if (wv == 0) SI_TRACE_MARK(24);
    for (int i = tid; i < B * kTile; i += kLayerThreads) {
      const int t = i / kTile, col = tile * kTile + (i - t * kTile);
      const float v = (&red[0][0])[i];
      if (col < d && v != 0.f) unsafeAtomicAdd(&a.y[(size_t)t * d + col], v);
    }
  }
  if (wv == 0) SI_TRACE_MARK(25);
  if (tid == 0) {
    a.counts[2 * g] = s_up;
    a.counts[2 * g + 1] = s_down;
  }
}

// Sum of the per-block work counts -> counters[3] = {n_gate, n_up, n_down}.
__global__ __launch_bounds__(256) void k_sum_counts(const int32_t* __restrict__ counts, int slots,
                                                    const int32_t* __restrict__ n_active, int k,
                                                    int32_t* __restrict__ counters) {
  __shared__ int s[2];
  const int tid = threadIdx.x, lane = tid & 63;
  if (tid < 2) s[tid] = 0;
  __syncthreads();
  int u = 0, dn = 0;
  for (int i = tid; i < slots; i += 256) { u += counts[2 * i]; dn += counts[2 * i + 1]; }
  u = wave_sum_int(u);
  dn = wave_sum_int(dn);
  if (lane == 0) { atomicAdd(&s[0], u); atomicAdd(&s[1], dn); }
  __syncthreads();
  if (tid == 0) {
    counters[0] = min(max(*n_active, 0), k);
    counters[1] = s[0];
    counters[2] = s[1];
  }
}

// Units of 16 bytes per lane that cover a row of d fp16 values (template
// bucket of the kernel).
inline int units_per_lane(int d) {
  const int nu = (d / 8 + kWave - 1) / kWave;
  return nu <= 1 ? 1 : nu <= 2 ? 2 : nu <= 4 ? 4 : nu <= 8 ? 8 : nu <= 10 ? 10 : 16;
}

// Work split of the down-projection: `tiles` column tiles times `chunks`
// chunks of `gpc` consecutive groups, at most one item per block.
struct LayerPlan {
  int groups, tiles, chunks, gpc;
};

static LayerPlan plan_layer(int k, int d) {
  LayerPlan p;
  p.groups = row_groups(k);
  p.tiles = (d + kTile - 1) / kTile;
  int want = p.groups / p.tiles;  // items = tiles * chunks must not exceed the blocks
  if (want < 1) want = 1;
  p.gpc = (p.groups + want - 1) / want;
  p.chunks = (p.groups + p.gpc - 1) / p.gpc;  // every chunk holds at least one group
  return p;
}

template <int B, int NU>
static int layer_capacity() {
  static int cap = -1;
  if (cap < 0) {
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    const size_t lds = (size_t)B * kMaxD * sizeof(uint16_t);  // dynamic LDS at the largest accepted d
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(&k_layer<B, NU>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
      return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(&k_layer<B, NU>),
                                                     kLayerThreads, lds) != hipSuccess)
      return 0;
    cap = per_cu * cus;
  }
  return cap;
}

// The single-kernel path applies when the x tokens fit the LDS budget, every
// block holds at most one down item, and all blocks can be resident at once.
bool layer_supported(int k, int d, int b) {
  if (b > kLayerMaxB) return false;
  const LayerPlan p = plan_layer(k, d);
  if (p.groups < p.tiles || p.gpc > kWave) return false;
  int cap = 0;
  const int nu = units_per_lane(d);
#define CAP(B)                                          \
  case B:                                               \
    cap = nu == 1   ? layer_capacity<B, 1>()            \
          : nu == 2 ? layer_capacity<B, 2>()            \
          : nu == 4 ? layer_capacity<B, 4>()            \
          : nu == 8 ? layer_capacity<B, 8>()            \
          : nu == 10 ? layer_capacity<B, 10>()          \
                     : layer_capacity<B, 16>();         \
    break;
  switch (b) {
    CAP(1) CAP(2)
    default: return false;
  }
#undef CAP
  return p.groups <= cap;
}

template <int B, int NU>
static hipError_t layer_b(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up,
                          const uint16_t* w_down_t, int k, int d, const uint16_t* x, int T, int margin,
                          uint8_t* mask, int32_t* idx, int32_t* n_out, float* y, void* ws, uint32_t flags,
                          int32_t* counters, hipStream_t s) {
  const WsLayout L = ws_layout(k, B);
  char* base = static_cast<char*>(ws);
  const LayerPlan p = plan_layer(k, d);
  LayerArgs a;
  a.signs = reinterpret_cast<const u32x4*>(signs);
  a.wg = reinterpret_cast<const u32x4*>(w_gate);
  a.wu = reinterpret_cast<const u32x4*>(w_up);
  a.wdt = reinterpret_cast<const u32x4*>(w_down_t);
  a.x = x;
  a.k = k;
  a.d = d;
  a.T = T;
  a.margin = margin;
  a.flags = flags;
  a.mask = mask;
  a.idx = idx;
  a.n_out = n_out;
  a.hdr = reinterpret_cast<uint32_t*>(base);
  a.status = reinterpret_cast<uint64_t*>(base + L.status);
  a.ready = reinterpret_cast<uint32_t*>(base + L.ready);
  a.lmask = reinterpret_cast<uint64_t*>(base + L.lmask);
  a.zflag = reinterpret_cast<uint64_t*>(base + L.zflag);
  a.h3e = reinterpret_cast<uint64_t*>(base + L.h3e);
  a.counts = reinterpret_cast<int32_t*>(base + L.counts);
  a.y = y;
  a.tiles = p.tiles;
  a.chunks = p.chunks;
  a.gpc = p.gpc;
  const size_t lds = (size_t)B * d * sizeof(uint16_t);
  k_layer<B, NU><<<p.groups, kLayerThreads, lds, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !counters) return e;
  k_sum_counts<<<1, 256, 0, s>>>(a.counts, p.groups, n_out, k, counters);
  return hipGetLastError();
}

hipError_t launch_layer(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up,
                        const uint16_t* w_down_t, int k, int d, const uint16_t* x, int b, int T, int margin,
                        uint8_t* mask, int32_t* idx, int32_t* n_out, float* y, void* ws, uint32_t flags,
                        int32_t* counters, hipStream_t s) {
  const int nu = units_per_lane(d);
#define ARGS signs, w_gate, w_up, w_down_t, k, d, x, T, margin, mask, idx, n_out, y, ws, flags, counters, s
#define CASE(B)                                          \
  case B:                                                \
    return nu == 1    ? layer_b<B, 1>(ARGS)              \
           : nu == 2  ? layer_b<B, 2>(ARGS)              \
           : nu == 4  ? layer_b<B, 4>(ARGS)              \
           : nu == 8  ? layer_b<B, 8>(ARGS)              \
           : nu == 10 ? layer_b<B, 10>(ARGS)             \
                      : layer_b<B, 16>(ARGS);
  switch (b) {
    CASE(1) CASE(2)
    default: return hipErrorInvalidValue;
  }
#undef CASE
#undef ARGS
}

}  // namespace si
