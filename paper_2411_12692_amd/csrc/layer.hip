// The whole per-token MLP path of one layer in a single kernel: sign-bit
// prediction (Section IV-A, Eq. (2)), ordered compaction, sparse gate/up with
// actual sparsity and sparse down-projection (Section IV-B 3)-4)).
//
// One block of 16 wavefronts per group of 64 rows (all blocks co-resident;
// the host only takes this path when they fit).  Roles inside a block:
//
//  all waves   issue the group's packed-sign loads first, stage x in LDS,
//              pack its sign words, and add their XOR/popcount partials.
//  wave 0      applies Eq. (2) (N_neg < T), writes the mask, publishes the
//              group's kept list, then runs the look-back that places the
//              group in the ascending kept list (active_idx) and, in the last
//              group, writes the count and advances the epoch.
//  waves 1-7   gate/up of the group's kept rows: W_gate row, and W_up row only
//              where some token's ReLU output is positive.  Rows whose count
//              is far inside the threshold (N_neg < T - margin) are almost
//              surely positive, so their W_up row is requested together with
//              the W_gate row instead of one memory round trip later.
//  waves 8-15  down-projection of one work item = (512-column tile of y,
//              chunk of consecutive groups).  They read the chunk's kept
//              lists as soon as they are published and request the W_down^T
//              row segments of the confident rows at once, overlapping the
//              gate/up phase, then collect h3 and finish the other rows.
//              The block's partial tile is reduced in LDS and added into y
//              with fp32 atomics; tile c is zeroed first by block c.
//
// Blocks exchange data through epoch-tagged 64-bit words (tag = call
// counter in the high half, payload in the low half) written and polled with
// agent-scope relaxed atomics: a consumer polls each word until it carries
// the current epoch, so no cache flushes or fences are needed, and the
// workspace is never cleared between calls.  Every poll has a spin limit that
// sets an error bit instead of hanging.
#include "si_device.h"
#include "si_launch.h"

namespace si {

constexpr int kLayerWaves = 16;
constexpr int kLayerThreads = kLayerWaves * kWave;
constexpr int kLayerMaxB = 2;  // larger batches take the two-kernel path (register budget)
constexpr int kGateWaves = 7;  // waves 1..7
constexpr int kDownWaves = 8;  // waves 8..15
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
  uint64_t* lhdr;    // [groups] tag | kept count
  uint64_t* lent;    // [groups][64] tag | conf << 31 | row
  uint64_t* h3e;     // [groups][64][B] tag | fp32 bits
  uint64_t* zflag;   // [tiles] tag once the tile of y is zero
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
template <int B, int NU>
__device__ inline bool gate_up_spec(const u32x4* __restrict__ wg, const u32x4* __restrict__ wu, int row, int U,
                                    const u32x4* xs, int lane, bool spec, bool no_as, float (&h)[B]) {
  constexpr int J = NU;                     // 16-byte units per lane
  constexpr int JC = NU <= 10 ? NU : 1;     // both rows in registers only up to d = 5120
  const u32x4* gr = wg + (size_t)row * U;
  const u32x4* ur = wu + (size_t)row * U;
  const bool two = spec && NU <= 10;
  u32x4 a[J], c[JC];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int u = lane + kWave * j;
    if (u < U) a[j] = load_nt(gr + u);
  }
  if (two) {
#pragma unroll
    for (int j = 0; j < JC; ++j) {
      const int u = lane + kWave * j;
      if (u < U) c[j] = load_nt(ur + u);
    }
  }
  float g[B];
#pragma unroll
  for (int t = 0; t < B; ++t) g[t] = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int u = lane + kWave * j;
    if (u < U) {
#pragma unroll
      for (int t = 0; t < B; ++t) g[t] = dot8(a[j], xs[t * U + u], g[t]);
    }
  }
  bool any = false;
#pragma unroll
  for (int t = 0; t < B; ++t) {
    g[t] = fmaxf(wave_sum(g[t]), 0.f);
    any |= g[t] > 0.f;
  }
#pragma unroll
  for (int t = 0; t < B; ++t) h[t] = 0.f;
  const bool up = any || no_as || two;
  if (any || no_as) {
    float u[B];
#pragma unroll
    for (int t = 0; t < B; ++t) u[t] = 0.f;
    if (two) {
#pragma unroll
      for (int j = 0; j < JC; ++j) {
        const int uu = lane + kWave * j;
        if (uu < U) {
#pragma unroll
          for (int t = 0; t < B; ++t) u[t] = dot8(c[j], xs[t * U + uu], u[t]);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const int uu = lane + kWave * j;
        if (uu < U) a[j] = load_nt(ur + uu);
      }
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const int uu = lane + kWave * j;
        if (uu < U) {
#pragma unroll
          for (int t = 0; t < B; ++t) u[t] = dot8(a[j], xs[t * U + uu], u[t]);
        }
      }
    }
#pragma unroll
    for (int t = 0; t < B; ++t) h[t] = g[t] * wave_sum(u[t]);
  }
  return up;
}

// W_down^T segments in flight per down wave (fewer for larger batches to
// bound the registers holding h3 values).
template <int B>
constexpr int down_batch() { return B == 1 ? 8 : 4; }

// Units of 16 bytes per lane that cover a row of d fp16 values (template
// bucket of the kernel).
inline int units_per_lane(int d) {
  const int nu = (d / 8 + kWave - 1) / kWave;
  return nu <= 1 ? 1 : nu <= 2 ? 2 : nu <= 4 ? 4 : nu <= 8 ? 8 : nu <= 10 ? 10 : 16;
}

template <int B, int NU>
__global__ __launch_bounds__(kLayerThreads) void k_layer(LayerArgs a) {
  constexpr int kDownBatch = down_batch<B>();
  extern __shared__ u32x4 xs[];  // [B][d/8] fp16 tokens
  __shared__ __attribute__((aligned(16))) uint32_t xw[B * (kMaxD / 32)];
  __shared__ int cnt[B][kWave];
  __shared__ uint32_t kept[kRowGroup];  // conf << 31 | row
  __shared__ float red[B][kTile];
  __shared__ int s_nkept, s_up, s_down;
  __shared__ uint32_t s_epoch;

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d = a.d, U = d >> 3, W = d >> 5, units = W >> 2;
  const int g = blockIdx.x, groups = gridDim.x;
  const int items = a.tiles * a.chunks;
  const bool has_item = g < items;
  const int tile = g % a.tiles, chunk = g / a.tiles;

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
    s_epoch = ld_agent(&a.hdr[H_PRED_EPOCH]);
  }
  const bool owns_tile = g < a.tiles;
  if (owns_tile) {
    for (int i = tid; i < B * kTile; i += kLayerThreads) {
      const int t = i / kTile, col = g * kTile + (i - t * kTile);
      if (col < d) a.y[(size_t)t * d + col] = 0.f;
    }
  }
  __syncthreads();
  const uint32_t epoch = s_epoch;
  const uint32_t tag = epoch_tag(epoch);
  if (owns_tile && tid == 0) {
    __hip_atomic_store(&a.zflag[g], tagged(tag, 1u), __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }
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
    if (keep) {
      const uint32_t e = (conf ? 0x80000000u : 0u) | (uint32_t)row;
      kept[rank] = e;
      st_agent64(&a.lent[(size_t)g * kRowGroup + rank], tagged(tag, e));
    }
    if (lane == 0) {
      s_nkept = nk;
      st_agent64(&a.lhdr[g], tagged(tag, (uint32_t)nk));
      st_agent64(&a.status[g], tagged(tag, (uint32_t)((g == 0 ? kFlagPrefix : kFlagAggregate) | (uint64_t)nk)));
    }
  }
  __syncthreads();
  const int nkept = s_nkept;
  const bool no_as = (a.flags & kNoAS) != 0;

  if (wv == 0) {
    // ---- ordered compaction
    const int excl = g == 0 ? 0 : layer_lookback(a.status, g, tag, lane, a.hdr);
    if (lane == 0 && g > 0) st_agent64(&a.status[g], tagged(tag, (uint32_t)(kFlagPrefix | (uint64_t)(excl + nkept))));
    if (lane < nkept && a.idx) a.idx[excl + lane] = (int32_t)(kept[lane] & 0x7fffffffu);
    if (lane == 0 && g == groups - 1) {
      if (a.n_out) *a.n_out = excl + nkept;
      st_agent(&a.hdr[H_PRED_EPOCH], epoch + 1u);  // every group has posted: all blocks read this epoch
    }
  } else if (wv <= kGateWaves) {
    // ---- gate/up of this group's kept rows
    int n_up = 0;
    for (int i = wv - 1; i < nkept; i += kGateWaves) {
      const uint32_t e = kept[i];
      const int row = (int)(e & 0x7fffffffu);
      const bool spec = (e >> 31) != 0 && !(a.flags & kNoSpec);
      float h[B];
      n_up += gate_up_spec<B, NU>(a.wg, a.wu, row, U, xs, lane, spec, no_as, h) ? 1 : 0;
#pragma unroll
      for (int t = 0; t < B; ++t)
        if (lane == t) st_agent64(&a.h3e[((size_t)g * kRowGroup + i) * B + t], tagged(tag, __float_as_uint(h[t])));
    }
    if (lane == 0 && n_up) atomicAdd(&s_up, n_up);
  } else if (has_item) {
    // ---- down-projection of (tile, chunk)
    const int wb = wv - (1 + kGateWaves);
    const int g0 = chunk * a.gpc;
    const int ng = max(0, min(g0 + a.gpc, groups) - g0);
    const int unit = tile * (kTile / 8) + lane;  // 16-byte unit of a W_down^T row: 8 columns
    const bool col_ok = unit < U;
    bool abort = false;
    // kept counts of the chunk's groups (lane l <-> group g0 + l) and their
    // inclusive prefix: positions of the chunk's concatenated kept list
    const int cnt_l = (int)poll_lane(&a.lhdr[g0 + (lane < ng ? lane : 0)], lane < ng, tag, a.hdr, abort);
    int pre_l = cnt_l;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int v = __shfl_up(pre_l, o, kWave);
      if (lane >= o) pre_l += v;
    }
    const int E = ng > 0 ? __shfl(pre_l, ng - 1, kWave) : 0;
    float acc[B][8];
#pragma unroll
    for (int t = 0; t < B; ++t)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[t][q] = 0.f;
    int n_down = 0;
    const bool spec_ok = !(a.flags & kNoSpec);
    for (int p0 = wb; p0 < E && !abort; p0 += kDownWaves * kDownBatch) {
      // list slots of this wave's positions p0 + 8r
      uint32_t off[kDownBatch];
      uint32_t want = 0;
#pragma unroll
      for (int r = 0; r < kDownBatch; ++r) {
        const int p = p0 + kDownWaves * r;
        const int gi = __popcll(__ballot(lane < ng && pre_l <= p));
        const int before = gi > 0 ? __shfl(pre_l, gi - 1, kWave) : 0;
        off[r] = (uint32_t)((g0 + gi) * kRowGroup + (p - before));
        if (p < E) want |= 1u << r;
      }
      uint32_t e[kDownBatch][1];
      poll_batch<kDownBatch, 1>(a.lent, off, want, tag, e, a.hdr, abort);
      u32x4 w[kDownBatch];
      uint32_t loaded = 0;
#pragma unroll
      for (int r = 0; r < kDownBatch; ++r) {
        w[r] = u32x4{0, 0, 0, 0};
        if (((want >> r) & 1) && !abort) {
          const int row = (int)(e[r][0] & 0x7fffffffu);
          if ((unsigned)row < (unsigned)a.k && ((spec_ok && (e[r][0] >> 31)) || no_as)) {
            if (col_ok) w[r] = load_nt(a.wdt + (size_t)row * U + unit);
            loaded |= 1u << r;
          }
        }
      }
      uint32_t hb[kDownBatch][B];
      poll_batch<kDownBatch, B>(a.h3e, off, want, tag, hb, a.hdr, abort);
      float hv[kDownBatch][B];
#pragma unroll
      for (int r = 0; r < kDownBatch; ++r) {
        bool nz = false;
#pragma unroll
        for (int t = 0; t < B; ++t) {
          hv[r][t] = ((want >> r) & 1) && !abort ? __uint_as_float(hb[r][t]) : 0.f;
          nz |= hv[r][t] != 0.f;
        }
        if (((want >> r) & 1) && !((loaded >> r) & 1) && nz) {
          const int row = (int)(e[r][0] & 0x7fffffffu);
          if ((unsigned)row < (unsigned)a.k) {
            if (col_ok) w[r] = load_nt(a.wdt + (size_t)row * U + unit);
            loaded |= 1u << r;
          }
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
  }
  __syncthreads();

  // ---- add the block's tile into y once block `tile` has zeroed it
  if (has_item) {
    if (wv == 0 && lane == 0) {
      long spins = 0;
      while ((uint32_t)(__hip_atomic_load(&a.zflag[tile], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) >> 32) !=
             tag) {
        if (++spins > kPollLimit) {
          atomicOr(&a.hdr[H_ERR], kErrLookbackSpin);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    __syncthreads();
    for (int i = tid; i < B * kTile; i += kLayerThreads) {
      const int t = i / kTile, col = tile * kTile + (i - t * kTile);
      const float v = (&red[0][0])[i];
      if (col < d && v != 0.f) unsafeAtomicAdd(&a.y[(size_t)t * d + col], v);
    }
  }
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
  char* lb = base + L.layer;
  const size_t groups = (size_t)p.groups;
  a.lhdr = reinterpret_cast<uint64_t*>(lb);
  lb += align256(groups * 8);
  a.lent = reinterpret_cast<uint64_t*>(lb);
  lb += align256(groups * kRowGroup * 8);
  a.h3e = reinterpret_cast<uint64_t*>(lb);
  lb += align256(groups * kRowGroup * B * 8);
  a.zflag = reinterpret_cast<uint64_t*>(lb);
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
