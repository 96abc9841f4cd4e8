// The whole per-token MLP path of one layer in a single kernel: sign-bit
// prediction (Section IV-A, Eq. (2)), the ordered list of kept rows, sparse
// gate/up with actual sparsity and the sparse down-projection (Section IV-B
// 3)-4)).
//
// One block of 16 wavefronts per compute unit, all blocks resident at once
// (the host takes this path only when they fit; each block asks for enough
// LDS that no two share a CU).
//
//  1. predict   block b counts N_neg for the 64-row groups b, b+P, ...
//               (lane per row, the group's units split over the waves),
//               applies Eq. (2) as N_neg < T, writes the mask and publishes
//               the group's kept mask and "confident" mask (N_neg < T -
//               margin: almost surely active) as four tagged words.
//  2. exchange  every block reads the published masks of all groups (one
//               poll per word, all in flight together) and forms the same
//               inclusive prefix of kept counts in LDS, so every block knows
//               the whole ascending list of kept rows without a serial scan.
//  3. gate/up   block b takes positions [n b / P, n (b+1) / P) of the list,
//               an even share whatever the groups' kept counts.  Each row is
//               cut into 1 KB pieces (one 16-byte unit per lane) dealt to
//               the 16 waves, so all of the block's row requests are in
//               flight together.  W_up pieces of confident rows are
//               requested with the W_gate pieces; other rows read W_up only
//               where some token's ReLU output is positive (actual
//               sparsity).  h3 is published per list position.
//  4. down      block b also owns one item (512-column tile of y, chunk of
//               list positions).  It requests the tile's W_down^T pieces of
//               the confident rows of its chunk before the gate/up work, so
//               they stream in together, then collects h3 of its positions,
//               fetches the remaining rows whose h3 is non-zero, reduces in
//               LDS and adds the tile into y with fp32 atomics once the
//               tile's owner has zeroed it in this call (about P / tiles
//               atomics per element of y).
//
// Blocks exchange data through 64-bit words: the high half is this call's
// tag (the workspace's call counter with the high bit set), the low half the
// payload.  They are written with agent-scope write-through stores and read
// with agent-scope loads; a word is valid once it carries the call's tag, so
// no cache flush or fence is needed and the workspace is never cleared
// between calls.  Block 0 advances the call counter once it has seen every
// block's first word (so every block has read the counter).  Every wait is
// bounded: past a spin limit the block sets an error bit in the workspace
// header and goes on without the data.

#include "si_device.h"
#include "si_launch.h"

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

constexpr int kLWaves = 16;
constexpr int kLThreads = kLWaves * kWave;
constexpr int kLayerMaxB = 2;       // larger batches take the two-kernel path (register budget)
constexpr int kMaxSignUnitsPerWave = kMaxD / 128 / kLWaves;  // 4
constexpr int kMaxLayerGroups = 960;  // masks of every group are held in LDS (k <= 61440)
constexpr int kMaxPollWords = 4 * kLThreads;
constexpr int kRoundRows = kLWaves / 2;    // gate/up rows per round: one (row, matrix) item per wave
constexpr int kDN = 4;                     // down pieces in flight per wave
constexpr int kDownRound = kLWaves * kDN;  // down positions per round
constexpr int kMaxSlice = 256;             // gate/up positions of one block (at most)
constexpr int kMaxDownItem = 4096;         // positions of one down item (at most)
constexpr int kLayerLdsBytes = 96 * 1024;  // per block: more than half of a CU's LDS
constexpr long kPollLimit = 1l << 16;
constexpr uint32_t kNoAS = 1u, kNoSpec = 2u;
static_assert(kTile == kWave * 8, "a down tile is one 16-byte unit per lane");

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
  uint64_t* pub;    // [groups][4] tag | kept mask low/high half, tag | confident mask low/high half
  uint64_t* alive;  // [blocks] tag, from blocks that own no group
  uint64_t* h3e;    // [k][B] tag | fp32 bits of h3, by list position
  uint64_t* zflag;  // [tiles] tag once the tile of y is zero
  int32_t* counts;  // [blocks][2] W_up rows read, W_down^T rows read (tile-0 items)
  float* y;
  int groups, tiles, chunks;
  double inv_blocks, inv_chunks;  // 1 / grid size, 1 / chunks (exact floors of n b / P, n c / C)
};

// Everything the block keeps in LDS, carved from the dynamic allocation.
template <int B>
struct LayerLds {
  // tokens (fp16); once the gate/up work is done, the down-projection's
  // per-wave tile sums: [8 wave pairs][B][512 columns]
  union {
    u32x4 xs[B * kMaxD / 8];
    float dpart[8][B][kTile];
  };
  uint32_t xw[B * kMaxD / 32];          // sign words of the tokens
  int cpart[kLWaves][B][kWave];         // per-wave N_neg partial counts of the current group
  uint32_t pm[4 * kMaxLayerGroups];     // published masks of every group
  int wtot[kLWaves];
  int pre[kMaxLayerGroups];             // inclusive prefix of the kept counts
  int gfirst[2];                        // group holding the first position of the slice / the down item
  float dots[kRoundRows][2][B];         // W_gate . x and W_up . x of the round's rows
  float h1[kRoundRows][B];
  uint32_t need[kRoundRows];            // round row needs a late W_up read
  uint32_t srow[kMaxSlice];             // conf << 31 | row of the block's gate/up positions
  uint32_t dent[kMaxDownItem];          // conf << 31 | row of the block's down positions
  float hs[kDownRound][B];              // h3 of the down round's positions
  int sc[8];                            // block scalars: n, lo, hi, dlo, dhi
  int n_late, n_up, n_down, zok;
  uint32_t epoch;
};

__device__ inline uint64_t tagged(uint32_t tag, uint32_t payload) { return ((uint64_t)tag << 32) | payload; }

template <int CTRL>
__device__ inline float dpp_add(float v) {
  return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

// Sum over the 64 lanes (wave-uniform result): DPP sums inside each row of 16
// lanes, then the four row sums.
__device__ inline float wave_total(float v) {
  v = dpp_add<0xB1>(v);   // quad_perm(1,0,3,2)
  v = dpp_add<0x4E>(v);   // quad_perm(2,3,0,1)
  v = dpp_add<0x141>(v);  // row_half_mirror
  v = dpp_add<0x140>(v);  // row_mirror
  const int iv = __builtin_bit_cast(int, v);
  return (__builtin_bit_cast(float, __builtin_amdgcn_readlane(iv, 0)) +
          __builtin_bit_cast(float, __builtin_amdgcn_readlane(iv, 16))) +
         (__builtin_bit_cast(float, __builtin_amdgcn_readlane(iv, 32)) +
          __builtin_bit_cast(float, __builtin_amdgcn_readlane(iv, 48)));
}

__device__ inline int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

template <int CTRL, int ROWS>
__device__ inline int dpp_get(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xF, true);
}

// Inclusive prefix sum over the 64 lanes: shifts by 1, 2, 4, 8 inside each
// row of 16 lanes, then the last lane of rows 0 and 1 broadcast forward.
__device__ inline int wave_incl_scan(int v) {
  v += dpp_get<0x111, 0xF>(v);  // row_shr:1
  v += dpp_get<0x112, 0xF>(v);  // row_shr:2
  v += dpp_get<0x114, 0xF>(v);  // row_shr:4
  v += dpp_get<0x118, 0xF>(v);  // row_shr:8
  v += dpp_get<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
  v += dpp_get<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
  return v;
}

// Poll one tagged word per lane (lanes may use different addresses) until it
// carries `tag`; returns the payload.  After the spin limit the wave stops
// waiting (`abort`) and the error bit is set.
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

// Dot products of a row held as NU 16-byte units per lane (unit lane + 64 j)
// with the B tokens in LDS; wave-uniform results.
template <int B, int NU>
__device__ inline void row_dots(const u32x4 (&v)[NU], const u32x4* xs, int U, int lane, float (&out)[B]) {
  float acc[B];
#pragma unroll
  for (int t = 0; t < B; ++t) acc[t] = 0.f;
#pragma unroll
  for (int j = 0; j < NU; ++j) {
    const int u = lane + kWave * j;
    if (u < U) {
#pragma unroll
      for (int t = 0; t < B; ++t) acc[t] = dot8(v[j], xs[t * U + u], acc[t]);
    }
  }
#pragma unroll
  for (int t = 0; t < B; ++t) out[t] = wave_total(acc[t]);
}

template <int NU>
__device__ inline void load_row(const u32x4* __restrict__ row, int U, int lane, u32x4 (&v)[NU]) {
#pragma unroll
  for (int j = 0; j < NU; ++j) {
    const int u = lane + kWave * j;
    if (u < U) v[j] = load_nt(row + u);
  }
}

template <int B, int NU>
__global__ __launch_bounds__(kLThreads) void k_layer(LayerArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  LayerLds<B>& L = *reinterpret_cast<LayerLds<B>*>(lds_raw);

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d = a.d, U = d >> 3, W = d >> 5, units = d >> 7;
  const int P = gridDim.x, blk = blockIdx.x, G = a.groups;
  const int T = a.tiles;
  const bool no_as = (a.flags & kNoAS) != 0;
  const bool spec_ok = (a.flags & kNoSpec) == 0;

  SI_TRACE_MARK(0);
  // ---- tokens, then the sign loads of the block's first group
  for (int i = tid; i < B * U; i += kLThreads) L.xs[i] = reinterpret_cast<const u32x4*>(a.x)[i];
  u32x4 sreg[kMaxSignUnitsPerWave];
  auto load_signs = [&](int g) {
    const u32x4* sg = a.signs + (size_t)g * units * kRowGroup + lane;
#pragma unroll
    for (int i = 0; i < kMaxSignUnitsPerWave; ++i) {
      const int q = wv + kLWaves * i;
      if (q < units) sreg[i] = load_nt(sg + (size_t)q * kRowGroup);
    }
  };
  if (blk < G) load_signs(blk);
  if (tid == 0) {
    L.n_up = 0;
    L.n_down = 0;
    L.zok = 0;
    L.epoch = ld_agent(&a.hdr[H_EPOCH]);
  }
  __syncthreads();
  const uint32_t epoch = uniform(L.epoch);
  const uint32_t tag = epoch_tag(epoch);
  for (int i = tid; i < B * W; i += kLThreads) {
    const int t = i / W, w = i - t * W;
    L.xw[i] = sign_word(&L.xs[t * U + 4 * w]);
  }
  __syncthreads();
  SI_TRACE_MARK(1);

  // ---- 1. predict the block's groups
  for (int g = blk; g < G; g += P) {
    if (g != blk) load_signs(g);
    int c[B];
#pragma unroll
    for (int t = 0; t < B; ++t) c[t] = 0;
    bool any_unit = false;
#pragma unroll
    for (int i = 0; i < kMaxSignUnitsPerWave; ++i) {
      const int q = wv + kLWaves * i;
      if (q < units) {
        any_unit = true;
#pragma unroll
        for (int t = 0; t < B; ++t) {
          const u32x4 xv = *reinterpret_cast<const u32x4*>(&L.xw[t * W + 4 * q]);
          c[t] += __popc(sreg[i].x ^ xv.x) + __popc(sreg[i].y ^ xv.y) + __popc(sreg[i].z ^ xv.z) +
                  __popc(sreg[i].w ^ xv.w);
        }
      }
    }
    if (any_unit) {
#pragma unroll
      for (int t = 0; t < B; ++t) L.cpart[wv][t][lane] = c[t];
    }
    __syncthreads();
    if (wv == 0) {
      const int row = g * kRowGroup + lane;
      const int nw = min(units, kLWaves);  // waves that counted units
      bool keep = false, conf = false;
#pragma unroll
      for (int t = 0; t < B; ++t) {
        int n_neg = 0;
        for (int w = 0; w < nw; ++w) n_neg += L.cpart[w][t][lane];
        keep |= n_neg < a.T;
        conf |= n_neg < a.T - a.margin;
      }
      keep = keep && row < a.k;
      if (row < a.k) a.mask[row] = keep ? 1 : 0;
      const uint64_t kb = __ballot(keep);
      const uint64_t cb = __ballot(keep && conf);
      if (lane < 4) {
        const uint64_t m = lane < 2 ? kb : cb;
        st_agent64(&a.pub[(size_t)g * 4 + lane], tagged(tag, (uint32_t)(m >> (32 * (lane & 1)))));
      }
    }
    __syncthreads();
  }
  if (blk >= G && tid == 0) st_agent64(&a.alive[blk], tagged(tag, 0u));
  // the tile of y this block owns is zeroed while the masks are exchanged
  const bool owns_tile = blk < T;
  if (owns_tile) {
    for (int i = tid; i < B * kTile; i += kLThreads) {
      const int t = i / kTile, col = blk * kTile + (i - t * kTile);
      if (col < d) __hip_atomic_store(&a.y[(size_t)t * d + col], 0.f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  SI_TRACE_MARK(2);

  // ---- 2. every group's masks (and the word of every block without a group)
  {
    const int NWp = 4 * G;
    const int NW = NWp + (P > G ? P - G : 0);
    uint64_t v[kMaxPollWords / kLThreads];
    uint32_t pending = 0;
#pragma unroll
    for (int i = 0; i < kMaxPollWords / kLThreads; ++i) {
      const int j = tid + kLThreads * i;
      if (j < NW) pending |= 1u << i;
    }
    long spins = 0;
    while (pending) {
#pragma unroll
      for (int i = 0; i < kMaxPollWords / kLThreads; ++i) {
        const int j = tid + kLThreads * i;
        if ((pending >> i) & 1u) v[i] = ld_agent64(j < NWp ? &a.pub[j] : &a.alive[G + (j - NWp)]);
      }
#pragma unroll
      for (int i = 0; i < kMaxPollWords / kLThreads; ++i) {
        const int j = tid + kLThreads * i;
        if (((pending >> i) & 1u) && (uint32_t)(v[i] >> 32) == tag) {
          if (j < NWp) L.pm[j] = (uint32_t)v[i];
          pending &= ~(1u << i);
        }
      }
      if (pending) {
        if (++spins > kPollLimit) {
          atomicOr(&a.hdr[H_ERR], kErrLookbackSpin);
#pragma unroll
          for (int i = 0; i < kMaxPollWords / kLThreads; ++i) {
            const int j = tid + kLThreads * i;
            if (((pending >> i) & 1u) && j < NWp) L.pm[j] = 0u;
          }
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
  }
  if (owns_tile) wait_own_stores();  // the y-zeroing stores of this wave have landed
  __syncthreads();
  if (tid == 0) {
    if (owns_tile) st_agent64(&a.zflag[blk], tagged(tag, 1u));
    if (blk == 0) st_agent(&a.hdr[H_EPOCH], epoch + 1u);  // every block has read the call counter
  }
  SI_TRACE_MARK(3);

  // ---- plan: kept count of every group (one group per thread) and their
  // block-wide prefix; the block's gate/up slice and down item; then one
  // wave per group that holds positions of them writes their list entries
  // (lane = row: rank among the group's kept rows)
  const int C = a.chunks;
  const bool has_item = blk < T * C;
  const int tile = has_item ? blk % T : 0, chunk = has_item ? blk / T : 0;
  {
    uint64_t km = 0;
    if (tid < G) km = (uint64_t)L.pm[4 * tid] | ((uint64_t)L.pm[4 * tid + 1] << 32);
    const int c = __popcll(km);
    const int incl = wave_incl_scan(c);
    if (lane == kWave - 1) L.wtot[wv] = incl;
    if (tid < 2) L.gfirst[tid] = G;
    __syncthreads();
    const int wt = wave_incl_scan(lane < kLWaves ? L.wtot[lane] : 0);  // lanes 0..15: prefix of wave totals
    const int n = uniform(__builtin_amdgcn_readlane(wt, kLWaves - 1));
    const int before = wv > 0 ? uniform(__builtin_amdgcn_readlane(wt, wv > 0 ? wv - 1 : 0)) : 0;
    // floor(n b / P) etc.: (x + 1/2) / P is at least 1 / (2P) away from an integer
    const int lo_ = (int)(((double)n * blk + 0.5) * a.inv_blocks);
    const int hi_ = (int)(((double)n * (blk + 1) + 0.5) * a.inv_blocks);
    const int dlo_ = has_item ? (int)(((double)n * chunk + 0.5) * a.inv_chunks) : 0;
    const int dhi_ = has_item ? (int)(((double)n * (chunk + 1) + 0.5) * a.inv_chunks) : 0;
    const int pi = before + incl, pe = pi - c;  // the group's kept rows hold positions [pe, pi)
    if (tid < G) {
      L.pre[tid] = pi;
      if (lo_ < hi_ && pe <= lo_ && lo_ < pi) L.gfirst[0] = tid;
      if (dlo_ < dhi_ && pe <= dlo_ && dlo_ < pi) L.gfirst[1] = tid;
    }
    if (tid == 0) {
      L.sc[1] = lo_;
      L.sc[2] = hi_;
      L.sc[3] = dlo_;
      L.sc[4] = dhi_;
      if (blk == 0) *a.n_out = n;
    }
    __syncthreads();
    // waves 0..7: groups from the slice's first; waves 8..15: from the down item's first
    const bool down_side = wv >= kLWaves / 2;
    const int rlo = down_side ? dlo_ : lo_, rhi = down_side ? dhi_ : hi_;
    for (int g = uniform(L.gfirst[down_side ? 1 : 0]) + (wv & 7); g < G; g += kLWaves / 2) {
      const int gpi = L.pre[g];
      const uint64_t gk = (uint64_t)L.pm[4 * g] | ((uint64_t)L.pm[4 * g + 1] << 32);
      const int gpe = gpi - __popcll(gk);
      if (gpe >= rhi) break;
      if (gpi <= rlo) continue;
      const uint64_t gc = (uint64_t)L.pm[4 * g + 2] | ((uint64_t)L.pm[4 * g + 3] << 32);
      const int q = gpe + __popcll(gk & lanes_below(lane));
      if (((gk >> lane) & 1ull) && q >= rlo && q < rhi) {
        const uint32_t e = (uint32_t)(g * kRowGroup + lane) | (((gc >> lane) & 1ull) ? 0x80000000u : 0u);
        if (down_side) {
          L.dent[q - rlo] = e;
        } else {
          L.srow[q - rlo] = e;
          a.idx[q] = g * kRowGroup + lane;
        }
      }
    }
  }
  __syncthreads();
  const int lo = uniform(L.sc[1]), hi = uniform(L.sc[2]);
  const int dlo = uniform(L.sc[3]), dhi = uniform(L.sc[4]);
  SI_TRACE_MARK(4);

  // ---- down requests of a round: this wave's positions q0 + wv + 16 j
  u32x4 vd[kDN];
  uint32_t dloaded = 0;
  const int dunit = tile * kWave + lane;
  const bool dcol_ok = dunit < U;
  auto issue_down = [&](int q0) {
    dloaded = 0;
#pragma unroll
    for (int j = 0; j < kDN; ++j) {
      vd[j] = u32x4{0, 0, 0, 0};
      const int q = wv + kLWaves * j;
      if (q0 + q < dhi) {
        const uint32_t e = L.dent[q0 - dlo + q];
        if ((spec_ok && (e >> 31)) || no_as) {
          if (dcol_ok) vd[j] = load_nt(a.wdt + (size_t)(e & 0x7fffffffu) * U + dunit);
          dloaded |= 1u << j;
        }
      }
    }
  };

  // ---- 3. gate/up: per round, wave wv owns item (row wv / 2, W_gate or W_up)
  const int ir = wv >> 1, imat = wv & 1;
  bool first = true;
  for (int r0 = lo; r0 < hi; r0 += kRoundRows) {
    const int mr = min(kRoundRows, hi - r0);
    const uint32_t* srow = &L.srow[r0 - lo];
    if (!first) __syncthreads();
    bool active = false;
    u32x4 v[NU];
    if (ir < mr) {
      const uint32_t e = srow[ir];
      active = imat == 0 || (spec_ok && (e >> 31));
      if (active) load_row<NU>((imat ? a.wu : a.wg) + (size_t)(e & 0x7fffffffu) * U, U, lane, v);
    }
    SI_TRACE_WAVE(0);
    if (active) {
      float dt[B];
      row_dots<B, NU>(v, L.xs, U, lane, dt);
      if (lane == 0) {
#pragma unroll
        for (int t = 0; t < B; ++t) L.dots[ir][imat][t] = dt[t];
      }
    }
    SI_TRACE_WAVE(1);
    // the down item's W_down^T pieces go out once this wave's gate/up data is
    // in, so they stream behind the loads that h3 depends on
    if (first && dlo < dhi) issue_down(dlo);
    first = false;
    __syncthreads();
    if (wv == 0) {  // rows of the round: one per lane (mr <= 8)
      bool any = no_as, spec = false;
      if (lane < mr) {
#pragma unroll
        for (int t = 0; t < B; ++t) {
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
    if (L.n_late) {  // W_up rows whose gate value asks for them
      if (imat == 1 && ir < mr && L.need[ir]) {
        load_row<NU>(a.wu + (size_t)(srow[ir] & 0x7fffffffu) * U, U, lane, v);
        float dt[B];
        row_dots<B, NU>(v, L.xs, U, lane, dt);
        if (lane == 0) {
#pragma unroll
          for (int t = 0; t < B; ++t) L.dots[ir][1][t] = dt[t];
        }
      }
      __syncthreads();
    }
    if (tid < mr * B) {
      const int r = tid / B, t = tid - r * B;
      const bool spec = spec_ok && (srow[r] >> 31);
      const float h = (L.need[r] || spec) ? L.h1[r][t] * L.dots[r][1][t] : 0.f;
      st_agent64(&a.h3e[(size_t)(r0 + r) * B + t], tagged(tag, __float_as_uint(h)));
    }
  }
  if (first && dlo < dhi) issue_down(dlo);  // blocks without gate/up rows
  SI_TRACE_MARK(6);

  // ---- 4. down-projection of (tile, chunk)
  float acc[B][8];
#pragma unroll
  for (int t = 0; t < B; ++t)
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[t][q] = 0.f;
  bool abort = false;
  int n_down = 0;
  for (int q0 = dlo; q0 < dhi; q0 += kDownRound) {
    const int nq = min(kDownRound, dhi - q0);
    if (q0 != dlo) {
      __syncthreads();  // the previous round's h3 values have been used
      issue_down(q0);
    }
    // wave 0 collects the round's h3 (contiguous words, one position per
    // lane); in the first round wave 1 checks the tile's zero flag
    if (wv == 0) {
#pragma unroll
      for (int t = 0; t < B; ++t) {
        const bool mine = lane < nq;
        const float h = __uint_as_float(poll_lane(&a.h3e[(size_t)(q0 + (mine ? lane : 0)) * B + t], mine, tag,
                                                  a.hdr, abort));
        if (mine) L.hs[lane][t] = abort ? 0.f : h;
      }
    } else if (wv == 1 && q0 == dlo) {
      poll_lane(&a.zflag[tile], lane == 0, tag, a.hdr, abort);
      if (lane == 0 && !abort) L.zok = 1;
    }
    __syncthreads();
    if (q0 == dlo) SI_TRACE_WAVE(3);
#pragma unroll
    for (int j = 0; j < kDN; ++j) {
      const int q = wv + kLWaves * j;
      float hv[B];
      bool nz = false;
#pragma unroll
      for (int t = 0; t < B; ++t) {
        hv[t] = q < nq ? L.hs[q][t] : 0.f;
        nz |= hv[t] != 0.f;
      }
      if (q < nq && !((dloaded >> j) & 1u) && nz) {  // late request
        if (dcol_ok) vd[j] = load_nt(a.wdt + (size_t)(L.dent[q0 - dlo + q] & 0x7fffffffu) * U + dunit);
        dloaded |= 1u << j;
      }
      const f16x2 p0 = as_h2(vd[j].x), p1 = as_h2(vd[j].y), p2 = as_h2(vd[j].z), p3 = as_h2(vd[j].w);
      const float f[8] = {(float)p0.x, (float)p0.y, (float)p1.x, (float)p1.y,
                          (float)p2.x, (float)p2.y, (float)p3.x, (float)p3.y};
#pragma unroll
      for (int t = 0; t < B; ++t)
#pragma unroll
        for (int qq = 0; qq < 8; ++qq) acc[t][qq] = fmaf(hv[t], f[qq], acc[t][qq]);
    }
    n_down += __popc(dloaded);
    if (q0 == dlo) SI_TRACE_WAVE(4);
  }
  // per-wave tile sums folded in LDS (plain stores; x is no longer needed)
  if (dlo < dhi) {
    if (wv < 8) {
#pragma unroll
      for (int t = 0; t < B; ++t)
#pragma unroll
        for (int q = 0; q < 8; ++q) L.dpart[wv][t][lane * 8 + q] = acc[t][q];
    }
    __syncthreads();
    if (wv >= 8) {
#pragma unroll
      for (int t = 0; t < B; ++t)
#pragma unroll
        for (int q = 0; q < 8; ++q) L.dpart[wv - 8][t][lane * 8 + q] += acc[t][q];
    }
  }
  if (lane == 0 && tile == 0 && n_down) atomicAdd(&L.n_down, n_down);
  SI_TRACE_MARK(8);
  __syncthreads();

  // ---- the block's tile into y (its owner zeroed it in this call)
  if (dlo < dhi) {
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
    for (int i = tid; i < B * kTile; i += kLThreads) {
      const int t = i / kTile, c = i - t * kTile, col = tile * kTile + c;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < 8; ++w) v += L.dpart[w][t][c];
      if (col < d && v != 0.f) unsafeAtomicAdd(&a.y[(size_t)t * d + col], v);
    }
  }
  SI_TRACE_MARK(10);
  if (tid == 0) {
    a.counts[2 * blk] = L.n_up;
    a.counts[2 * blk + 1] = L.n_down;
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
  for (int i = tid; i < slots; i += 256) {
    u += counts[2 * i];
    dn += counts[2 * i + 1];
  }
  u = wave_sum_int(u);
  dn = wave_sum_int(dn);
  if (lane == 0) {
    atomicAdd(&s[0], u);
    atomicAdd(&s[1], dn);
  }
  __syncthreads();
  if (tid == 0) {
    counters[0] = min(max(*n_active, 0), k);
    counters[1] = s[0];
    counters[2] = s[1];
  }
}

// 16-byte units per lane that cover a row of d fp16 values (template bucket).
inline int units_per_lane(int d) {
  const int nu = (d / 8 + kWave - 1) / kWave;
  return nu <= 1 ? 1 : nu <= 2 ? 2 : nu <= 4 ? 4 : nu <= 8 ? 8 : nu <= 10 ? 10 : 16;
}

// Grid of the single-kernel path: one block per compute unit (the LDS
// request keeps a second block off every CU), or 0 if the kernel cannot be
// resident on every CU.
template <int B, int NU>
static int layer_blocks() {
  static int blocks = -1;
  if (blocks < 0) {
    blocks = 0;
    int dev = 0, cus = 0, per_cu = 0;
    static_assert(sizeof(LayerLds<B>) <= (size_t)kLayerLdsBytes, "LDS budget");
    const void* fn = reinterpret_cast<const void*>(&k_layer<B, NU>);
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, kLayerLdsBytes) != hipSuccess) return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kLThreads, kLayerLdsBytes) != hipSuccess) return 0;
    if (per_cu >= 1) blocks = cus < kMaxLayerBlocks ? cus : kMaxLayerBlocks;
  }
  return blocks;
}

#define SI_LAYER_DISPATCH(B, CALL)          \
  switch (units_per_lane(d)) {             \
    case 1: return CALL(B, 1);             \
    case 2: return CALL(B, 2);             \
    case 4: return CALL(B, 4);             \
    case 8: return CALL(B, 8);             \
    case 10: return CALL(B, 10);           \
    default: return CALL(B, 16);           \
  }

static int blocks_for(int d, int b) {
#define BLOCKS(B, NU) layer_blocks<B, NU>()
  if (b == 1) { SI_LAYER_DISPATCH(1, BLOCKS) }
  if (b == 2) { SI_LAYER_DISPATCH(2, BLOCKS) }
  return 0;
#undef BLOCKS
}

// The single-kernel path applies for batches of at most two tokens, up to
// kMaxLayerGroups row groups (every group's masks fit in LDS and in one
// poll per thread), and when one block per CU can be resident.
bool layer_supported(int k, int d, int b) {
  if (b < 1 || b > kLayerMaxB) return false;
  const int G = row_groups(k);
  if (G > kMaxLayerGroups) return false;
  const int P = blocks_for(d, b);
  const int tiles = (d + kTile - 1) / kTile;
  if (P < tiles) return false;
  const int chunks = P / tiles;
  if ((k + P - 1) / P > kMaxSlice || (k + chunks - 1) / chunks > kMaxDownItem) return false;
  return 4 * G + (P > G ? P - G : 0) <= kMaxPollWords;
}

template <int B, int NU>
static hipError_t layer_b(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up,
                          const uint16_t* w_down_t, int k, int d, const uint16_t* x, int T, int margin,
                          uint8_t* mask, int32_t* idx, int32_t* n_out, float* y, void* ws, uint32_t flags,
                          int32_t* counters, hipStream_t s) {
  const WsLayout L = ws_layout(k, B);
  char* base = static_cast<char*>(ws);
  const int P = layer_blocks<B, NU>();
  if (P < 1) return hipErrorInvalidConfiguration;
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
  a.pub = reinterpret_cast<uint64_t*>(base + L.lmask);
  a.alive = reinterpret_cast<uint64_t*>(base + L.alive);
  a.zflag = reinterpret_cast<uint64_t*>(base + L.zflag);
  a.h3e = reinterpret_cast<uint64_t*>(base + L.h3e);
  a.counts = reinterpret_cast<int32_t*>(base + L.counts);
  a.y = y;
  a.groups = row_groups(k);
  a.tiles = (d + kTile - 1) / kTile;
  a.chunks = P / a.tiles;
  a.inv_blocks = 1.0 / P;
  a.inv_chunks = 1.0 / a.chunks;
  k_layer<B, NU><<<P, kLThreads, kLayerLdsBytes, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !counters) return e;
  k_sum_counts<<<1, 256, 0, s>>>(a.counts, P, n_out, k, counters);
  return hipGetLastError();
}

hipError_t launch_layer(const uint32_t* signs, const uint16_t* w_gate, const uint16_t* w_up,
                        const uint16_t* w_down_t, int k, int d, const uint16_t* x, int b, int T, int margin,
                        uint8_t* mask, int32_t* idx, int32_t* n_out, float* y, void* ws, uint32_t flags,
                        int32_t* counters, hipStream_t s) {
#define LAUNCH(B, NU) \
  layer_b<B, NU>(signs, w_gate, w_up, w_down_t, k, d, x, T, margin, mask, idx, n_out, y, ws, flags, counters, s)
  if (b == 1) { SI_LAYER_DISPATCH(1, LAUNCH) }
  if (b == 2) { SI_LAYER_DISPATCH(2, LAUNCH) }
  return hipErrorInvalidValue;
#undef LAUNCH
}
#undef SI_LAYER_DISPATCH

}  // namespace si
