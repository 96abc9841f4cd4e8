// The sparse gated MLP of one layer over a caller's list of kept rows in a
// single kernel (si_sparse_mlp with an active list): sparse gate/up with
// actual sparsity and the sparse down-projection (Section IV-B 3)-4)), for
// decode batches of up to 8 tokens.  (Predict and mask calls take the
// row-owning kernel of owned.hip.)
//
// One block of 16 wavefronts per compute unit, all blocks resident at once
// (the host takes this path only when they fit; each block asks for more
// than half of a CU's LDS so that no two share a CU).
//
//  1. plan      block b takes positions [n b / P, n (b+1) / P) of the list
//               for gate/up (an even share) and one down-projection item:
//               512-column tile (b mod T) of y and chunk (b / T) of the list.
//  2. gate/up   in rounds of 8 rows, wave w owns (row w/2, W_gate or W_up)
//               and requests all its 16-byte units at once.  W_up rows are
//               requested with W_gate (given rows count as confident unless
//               speculation is off); otherwise W_up is read only where some
//               token's ReLU output is positive (actual sparsity).  h3 is
//               published per list position and token.
//  3. down      the tile's W_down^T pieces of the item's rows are requested
//               once each wave's gate/up data is in; the item's h3 words are
//               collected, the remaining rows with non-zero h3 are fetched,
//               the per-wave partial tiles are folded in LDS (plain stores)
//               and the tile is added into y with fp32 atomics once the
//               tile's owner has zeroed it in this call.
//
// Blocks exchange data through 64-bit words: the high half is this call's
// tag (the workspace's call counter with the high bit set), the low half the
// payload.  They are written with agent-scope write-through stores and read
// with agent-scope loads; a word is valid once it carries the call's tag, so
// no cache flush or fence is needed and the workspace is never cleared
// between calls.  Block 0 advances the call counter once it has seen every
// block's "alive" word, i.e. once every block has read it.  Every wait is
// bounded: past a spin limit the block sets an error bit in the workspace
// header and goes on without the data.

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

constexpr int kMaxSlice = 256;             // gate/up positions of one block (at most)

struct LayerArgs {
  const u32x4* wg;
  const u32x4* wu;  // nullptr: the non-gated ReLU MLP (h3 = ReLU(g))
  const u32x4* wdt;
  const uint16_t* x;
  const int32_t* idx_in;  // the caller's ascending kept rows
  const int32_t* n_in;    // and their count (device)
  int k, d, b;
  uint32_t flags;
  uint32_t* hdr;
  uint64_t* h3e;    // [k][b] tag | fp32 bits of h3, by list position and token
  uint64_t* zflag;  // [tiles] tag once the tile of y is zero
  uint64_t* alive;  // [blocks] tag once the block has read the call counter
  int32_t* counts;  // [blocks][2] W_up rows read, W_down^T rows read (tile-0 items)
  float* y;
  int tiles, chunks;
  double inv_blocks, inv_chunks;  // 1 / grid size, 1 / chunks (exact floors of n b / P, n c / C)
};

// Everything the block keeps in LDS (carved from the dynamic allocation),
// sized for batches of up to BM tokens and rows of up to NU * 512 values.
template <int BM, int NU>
struct LayerLds {
  static constexpr int kUnits = NU * kWave;   // 16-byte units of a token
  static constexpr int kFold = kLWaves / BM;  // per-wave partial tiles held at once in the fold
  // tokens (fp16); once the gate/up work is done, the down-projection's
  // per-wave partial tiles
  union {
    u32x4 xs[BM * kUnits];
    float dpart[kFold][BM][kTile];
  };
  float dots[kRoundRows][2][BM];  // W_gate . x and W_up . x of the round's rows
  float h1[kRoundRows][BM];
  uint32_t need[kRoundRows];      // round row needs a late W_up read
  uint32_t srow[kMaxSlice];       // conf << 31 | row of the block's gate/up positions
  uint32_t dent[kMaxDownItem];    // conf << 31 | row of the block's down positions
  float hs[kDownRound * BM];      // h3 of the down round's positions
  int sc[8];                      // block scalars: lo, hi, dlo, dhi
  int n_late, n_up, n_down, zok;
  uint32_t epoch, err;
};

template <int BM, int NU>
constexpr int layer_lds_bytes() {
  const int need = (int)((sizeof(LayerLds<BM, NU>) + 1023) / 1024 * 1024);
  return need < kMinLds ? kMinLds : need;
}

template <int BM, int NU>
__global__ __launch_bounds__(kLThreads) void k_layer(LayerArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  LayerLds<BM, NU>& L = *reinterpret_cast<LayerLds<BM, NU>*>(lds_raw);

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d = a.d, U = d >> 3;
  const int b = a.b;  // tokens, 1..BM; tokens b..BM-1 are zero
  const int P = gridDim.x, blk = blockIdx.x;
  const int T = a.tiles;
  const bool no_as = (a.flags & kNoAS) != 0;
  const bool spec_ok = (a.flags & kNoSpec) == 0;
  const bool gated = a.wu != nullptr;  // else the non-gated ReLU MLP (no W_up)

  SI_TRACE_DECL;
  SI_TRACE_MARK(0);
  // ---- the tokens and (behind the first token requests, so that the wait
  // for it, which comes at once for an atomic load, also covers them) the
  // call counter; addresses are clamped so that the requests are
  // unconditional and go out back to back; tokens b..BM-1 are zero
  {
    // token t's unit u at xs[t * XS + u] (XS = NU * 64 >= U)
    constexpr int XS = LayerLds<BM, NU>::kUnits;
    const u32x4* xg = reinterpret_cast<const u32x4*>(a.x);
    const int nx = b * U;
    for (int i = tid; i < BM * XS; i += kLThreads) {
      const int t = i / XS, u = i - t * XS;
      const u32x4 xv = xg[min(t * U + u, nx - 1)];
      if (i == tid && tid == 0) {
        asm volatile("" ::: "memory");
        load_epoch(a.hdr, L.epoch, L.err);
        L.n_up = 0;
        L.n_down = 0;
        L.zok = 0;
      }
      L.xs[i] = (t < b && u < U) ? xv : u32x4{0, 0, 0, 0};
    }
  }
  // the tile of y this block owns is zeroed (announced after the plan)
  const bool owns_tile = blk < T;
  if (owns_tile) {
    for (int i = tid; i < b * kTile; i += kLThreads) {
      const int t = i / kTile, col = blk * kTile + (i - t * kTile);
      if (col < d) __hip_atomic_store(&a.y[(size_t)t * d + col], 0.f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  // a workspace left inconsistent by a call whose bounded wait gave up (its
  // sticky error word is set): nothing is computed until the workspace is
  // reset, and the owners of the tiles of y fill them with NaN (each thread
  // the columns it zeroed above)
  if (uniform(L.err) & kErrLookbackSpin) {
    if (owns_tile) {
      for (int i = tid; i < b * kTile; i += kLThreads) {
        const int t = i / kTile, col = blk * kTile + (i - t * kTile);
        if (col < d)
          __hip_atomic_store(&a.y[(size_t)t * d + col], __builtin_nanf(""), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    return;
  }
  const uint32_t epoch = uniform(L.epoch);
  const uint32_t tag = epoch_tag(epoch);
  if (tid == 0) st_agent64(&a.alive[blk], tagged(tag, 0u));  // this block has read the call counter
  SI_TRACE_MARK(1);

  // ---- 1. plan: the block's gate/up slice and down item, and the list
  // entries that fall in them
  const int C = a.chunks;
  const bool has_item = blk < T * C;
  const int tile = has_item ? blk % T : 0, chunk = has_item ? blk / T : 0;
  {
    const int n = min(max(*a.n_in, 0), a.k);
    // floor(n b / P) etc.: (x + 1/2) / P is at least 1 / (2P) away from an integer
    const int lo_ = (int)(((double)n * blk + 0.5) * a.inv_blocks);
    const int hi_ = (int)(((double)n * (blk + 1) + 0.5) * a.inv_blocks);
    const int dlo_ = has_item ? (int)(((double)n * chunk + 0.5) * a.inv_chunks) : 0;
    const int dhi_ = has_item ? (int)(((double)n * (chunk + 1) + 0.5) * a.inv_chunks) : 0;
    const uint32_t cbit = (spec_ok || no_as) ? 0x80000000u : 0u;  // given rows count as confident
    for (int q = tid; q < hi_ - lo_; q += kLThreads) {
      const int r = a.idx_in[lo_ + q];
      const bool ok = (unsigned)r < (unsigned)a.k;
      if (!ok) atomicOr(&a.hdr[H_ERR], kErrRow);
      L.srow[q] = ok ? ((uint32_t)r | cbit) : kBadRow;
    }
    for (int q = tid; q < dhi_ - dlo_; q += kLThreads) {
      const int r = a.idx_in[dlo_ + q];
      const bool ok = (unsigned)r < (unsigned)a.k;
      L.dent[q] = ok ? ((uint32_t)r | cbit) : kBadRow;
    }
    if (tid == 0) {
      L.sc[1] = lo_;
      L.sc[2] = hi_;
      L.sc[3] = dlo_;
      L.sc[4] = dhi_;
    }
  }
  // every load of this wave has been consumed by now; waiting here (at no
  // cost) also tells the compiler so, and it then issues the gate/up row
  // requests back to back (without waits between them); owners also know
  // their y-zeroing stores have landed
  wait_own_stores();
  __syncthreads();
  if (tid == 0 && owns_tile) st_agent64(&a.zflag[blk], tagged(tag, 1u));
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
        if (e != kBadRow && ((spec_ok && (e >> 31)) || no_as)) {
          if (dcol_ok) vd[j] = load_nt(a.wdt + (size_t)(e & 0x7fffffffu) * U + dunit);
          dloaded |= 1u << j;
        }
      }
    }
  };

  // ---- 4. gate/up: per round, wave wv owns item (row wv / 2, W_gate or W_up)
  const int ir = wv >> 1, imat = wv & 1;
  bool first = true;
  for (int r0 = lo; r0 < hi; r0 += kRoundRows) {
    const int mr = min(kRoundRows, hi - r0);
    const uint32_t* srow = &L.srow[r0 - lo];
    if (!first) __syncthreads();
    const uint32_t e = ir < mr ? srow[ir] : kBadRow;
    // the row's requests and their use sit in one branch, so that no request
    // is left outstanding across rounds (the compiler then issues them back
    // to back instead of waiting before each)
    if (e != kBadRow && (imat == 0 || (gated && spec_ok && (e >> 31)))) {
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
    // the down item's W_down^T pieces go out once this wave's gate/up data is
    // in, so they stream behind the loads that h3 depends on
    if (first && dlo < dhi) issue_down(dlo);
    first = false;
    __syncthreads();
    if (wv == 0) {  // rows of the round: one per lane (mr <= 8)
      bool any = no_as, spec = false, ok = false;
      if (lane < mr) {
        ok = srow[lane] != kBadRow;
#pragma unroll
        for (int t = 0; t < BM; ++t) {
          const float h = ok ? fmaxf(L.dots[lane][0][t], 0.f) : 0.f;
          L.h1[lane][t] = h;
          any |= h > 0.f;
        }
        any = any && ok && gated;  // W_up rows exist only in the gated MLP
        spec = ok && gated && spec_ok && (srow[lane] >> 31);
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
    for (int i = tid; i < mr * b; i += kLThreads) {
      const int r = i / b, t = i - r * b;
      const bool spec = srow[r] != kBadRow && spec_ok && (srow[r] >> 31);
      const float h = !gated ? L.h1[r][t] : (L.need[r] || spec) ? L.h1[r][t] * L.dots[r][1][t] : 0.f;
      st_agent64(&a.h3e[(size_t)(r0 + r) * b + t], tagged(tag, __float_as_uint(h)));
    }
  }
  if (first && dlo < dhi) issue_down(dlo);  // blocks without gate/up rows
  SI_TRACE_MARK(6);

  // ---- 5. down-projection of (tile, chunk)
  float acc[BM][8];
#pragma unroll
  for (int t = 0; t < BM; ++t)
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[t][q] = 0.f;
  int n_down = 0;
  bool epoch_done = false;
  for (int q0 = dlo; q0 < dhi; q0 += kDownRound) {
    const int nq = min(kDownRound, dhi - q0);
    if (q0 != dlo) {
      __syncthreads();  // the previous round's h3 values have been used
      issue_down(q0);
    }
    // waves 0..3 collect the round's h3 words (contiguous: positions x
    // tokens, all requests in flight together); in the first round wave 4
    // checks the tile's zero flag and waves 8.. of block 0
    // collect every block's alive word
    if (tid < kDownPollThreads) {
      constexpr int kPer = (kDownRound * BM + kDownPollThreads - 1) / kDownPollThreads;
      const int nw = nq * b;
      const uint64_t* base = &a.h3e[(size_t)q0 * b];
      uint64_t w[kPer];
      uint32_t pending = 0;
#pragma unroll
      for (int i = 0; i < kPer; ++i)
        if (tid + kDownPollThreads * i < nw) pending |= 1u << i;
      long spins = 0;
      while (pending) {
#pragma unroll
        for (int i = 0; i < kPer; ++i)
          if ((pending >> i) & 1u) w[i] = ld_agent64(base + tid + kDownPollThreads * i);
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
          if (((pending >> i) & 1u) && (uint32_t)(w[i] >> 32) == tag) {
            L.hs[tid + kDownPollThreads * i] = __uint_as_float((uint32_t)w[i]);
            pending &= ~(1u << i);
          }
        }
        if (pending) {
          if (++spins > kPollLimit) {
            atomicOr(&a.hdr[H_ERR], kErrLookbackSpin);
#pragma unroll
            for (int i = 0; i < kPer; ++i)
              if ((pending >> i) & 1u) L.hs[tid + kDownPollThreads * i] = 0.f;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
    } else if (q0 == dlo && wv == kDownPollThreads / kWave) {
      bool abort = false;
      poll_lane(&a.zflag[tile], lane == 0, tag, a.hdr, abort);
      if (lane == 0 && !abort) L.zok = 1;
    } else if (q0 == dlo && !epoch_done && blk == 0 && wv >= kLWaves / 2) {
      wait_alive(a.alive, P, tid - kLThreads / 2, kLThreads / 2, tag, a.hdr);
    }
    __syncthreads();
    if (q0 == dlo && !epoch_done && blk == 0 && tid == 0) advance_epoch(a.hdr, epoch);
    epoch_done = true;
    if (q0 == dlo) SI_TRACE_WAVE(3);
#pragma unroll
    for (int j = 0; j < kDN; ++j) {
      const int q = wv + kLWaves * j;
      float hv[BM];
      bool nz = false;
#pragma unroll
      for (int t = 0; t < BM; ++t) {
        hv[t] = (q < nq && t < b) ? L.hs[q * b + t] : 0.f;
        nz |= hv[t] != 0.f;
      }
      if (q < nq && !((dloaded >> j) & 1u) && nz) {  // late request
        const uint32_t e = L.dent[q0 - dlo + q];
        if (e != kBadRow) {
          if (dcol_ok) vd[j] = load_nt(a.wdt + (size_t)(e & 0x7fffffffu) * U + dunit);
          dloaded |= 1u << j;
        }
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
    if (q0 == dlo) SI_TRACE_WAVE(4);
  }
  // per-wave partial tiles folded in LDS (plain stores; x is no longer
  // needed): kFold waves store, the others add in turn
  constexpr int kFold = LayerLds<BM, NU>::kFold;
  if (dlo < dhi) {
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
    for (int i = tid; i < b * kTile; i += kLThreads) {
      const int t = i / kTile, c = i - t * kTile, col = tile * kTile + c;
      float v = 0.f;
#pragma unroll
      for (int s = 0; s < kFold; ++s) v += L.dpart[s][t][c];
      if (col < d && v != 0.f) unsafeAtomicAdd(&a.y[(size_t)t * d + col], v);
    }
  }
  if (!epoch_done && blk == 0) {  // no down round in block 0
    wait_alive(a.alive, P, tid, kLThreads, tag, a.hdr);
    __syncthreads();
    if (tid == 0) advance_epoch(a.hdr, epoch);
  }
  SI_TRACE_MARK(10);
  SI_TRACE_FLUSH;
  if (tid == 0) {
    a.counts[2 * blk] = L.n_up;
    a.counts[2 * blk + 1] = L.n_down;
    if (blk == 0) a.hdr[H_H3_FORM] = kH3ByPos;
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
hipError_t launch_sum_counts(const int32_t* counts, int slots, const int32_t* n_active, int k, int32_t* counters,
                             hipStream_t s) {
  k_sum_counts<<<1, 256, 0, s>>>(counts, slots, n_active, k, counters);
  return hipGetLastError();
}


// Grid of the single-kernel path: one block per compute unit, or 0 if the
// kernel's LDS does not fit or it cannot be resident on every CU.
template <int BM, int NU>
static int layer_blocks() {
  static std::atomic<int> cache[kMaxDevices];
  return per_device_once(cache, [](int dev) -> int {
    constexpr int lds = layer_lds_bytes<BM, NU>();
    if constexpr (lds > kMaxLds) {
      return 0;
    } else {
      int cus = 0, per_cu = 0;
      const void* fn = reinterpret_cast<const void*>(&k_layer<BM, NU>);
      if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
      if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess) return -1;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kLThreads, lds) != hipSuccess) return -1;
      return per_cu >= 1 ? (cus < kMaxLayerBlocks ? cus : kMaxLayerBlocks) : 0;
    }
  });
}

template <int BM, int NU>
static hipError_t layer_b(const LayerCall& c, hipStream_t s) {
  if constexpr (layer_lds_bytes<BM, NU>() > kMaxLds) {
    return hipErrorInvalidConfiguration;
  } else {
    const int k = c.k, d = c.d;
    const WsLayout L = ws_layout(k, c.b);
    char* base = static_cast<char*>(c.ws);
    const int P = layer_blocks<BM, NU>();
    if (P < 1) return hipErrorInvalidConfiguration;
    LayerArgs a;
    a.wg = reinterpret_cast<const u32x4*>(c.w_gate);
    a.wu = reinterpret_cast<const u32x4*>(c.w_up);
    a.wdt = reinterpret_cast<const u32x4*>(c.w_down_t);
    a.x = c.x;
    a.idx_in = c.idx_in;
    a.n_in = c.n_in;
    a.k = k;
    a.d = d;
    a.b = c.b;
    a.flags = c.flags;
    a.hdr = reinterpret_cast<uint32_t*>(base);
    a.zflag = reinterpret_cast<uint64_t*>(base + L.zflag);
    a.alive = reinterpret_cast<uint64_t*>(base + L.alive);
    a.h3e = reinterpret_cast<uint64_t*>(base + L.h3e);
    a.counts = reinterpret_cast<int32_t*>(base + L.counts);
    a.y = c.y;
    a.tiles = (d + kTile - 1) / kTile;
    a.chunks = P / a.tiles;
    a.inv_blocks = 1.0 / P;
    a.inv_chunks = 1.0 / a.chunks;
    k_layer<BM, NU><<<P, kLThreads, layer_lds_bytes<BM, NU>(), s>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !c.counters) return e;
    return launch_sum_counts(a.counts, P, c.n_in, k, c.counters, s);
  }
}

static int blocks_for(int d, int b) {
  if (b < 1 || b > kMaxB) return 0;
#define BLOCKS(BM, NU) layer_blocks<BM, NU>()
  SI_LAYER_DISPATCH(BLOCKS)
#undef BLOCKS
}

// The list kernel applies when one block per CU can be resident with the
// LDS that the batch and row width need, and a block's gate/up slice and
// down item fit their LDS lists.
bool layer_supported(int k, int d, int b) {
  const int P = blocks_for(d, b);
  const int tiles = (d + kTile - 1) / kTile;
  if (P < 1 || P < tiles) return false;
  const int chunks = P / tiles;
  return (k + P - 1) / P <= kMaxSlice && (k + chunks - 1) / chunks <= kMaxDownItem;
}

hipError_t launch_layer(const LayerCall& c, hipStream_t s) {
  const int d = c.d, b = c.b;
#define LAUNCH(BM, NU) layer_b<BM, NU>(c, s)
  SI_LAYER_DISPATCH(LAUNCH)
#undef LAUNCH
}
#undef SI_LAYER_DISPATCH
#undef SI_NU_DISPATCH

}  // namespace si
