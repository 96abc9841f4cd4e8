// Pieces shared by the single-launch layer kernels (layer.hip: list-driven
// and predictor-only calls; owned.hip: row-owning predict/mask calls):
// constants, wave-level reductions and scans, tagged exchange words, the
// row loads and dot products of the gate/up phase, and the host-side
// template dispatch.
#pragma once

#include "si_device.h"
#include "si_launch.h"

namespace si {

constexpr int kLWaves = 16;
constexpr int kLThreads = kLWaves * kWave;
constexpr int kMaxSignUnitsPerWave = (kMaxD / 128 + kLWaves - 1) / kLWaves;  // 4
constexpr int kRoundRows = kLWaves / 2;    // gate/up rows per round: one (row, matrix) item per wave
constexpr int kDN = 4;                     // down pieces in flight per wave
constexpr int kDownRound = kLWaves * kDN;  // down positions per round
constexpr int kMaxDownItem = 4096;         // positions of one down item (at most)
constexpr int kDownPollThreads = 256;      // waves 0..3 collect a round's h3 words
constexpr int kMinLds = 96 * 1024;         // more than half of a CU's LDS: one block per CU
constexpr int kMaxLds = 160 * 1024;
constexpr long kPollLimit = 1l << 16;
constexpr uint32_t kNoAS = 1u, kNoSpec = 2u;
constexpr uint32_t kBadRow = 0xffffffffu;  // list entry outside [0, k)
static_assert(kTile == kWave * 8, "a down tile is one 16-byte unit per lane");

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

// Threads [0, nthreads) wait until every block's alive word carries `tag`.
__device__ inline void wait_alive(const uint64_t* alive, int blocks, int t, int nthreads, uint32_t tag,
                                  uint32_t* hdr) {
  for (int j = t; j < blocks; j += nthreads) {
    long spins = 0;
    while ((uint32_t)(ld_agent64(&alive[j]) >> 32) != tag) {
      if (++spins > kPollLimit) {
        atomicOr(&hdr[H_ERR], kErrLookbackSpin);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
}

// Block 0, once every block has read the call counter: advance it.
// After a wait that gave up the counter is still advanced: otherwise the next
// call would carry this call's tag and take every word this call published as
// its own.  A late block may still tag its words for the next call, so the
// workspace is marked inconsistent (the sticky error word) until reset.
__device__ inline void advance_epoch(uint32_t* hdr, uint32_t epoch) { st_agent(&hdr[H_EPOCH], epoch + 1u); }

// The call counter and the sticky error word, in one request.
__device__ inline void load_epoch(const uint32_t* hdr, uint32_t& epoch, uint32_t& err) {
  const uint64_t w = ld_agent64(reinterpret_cast<const uint64_t*>(hdr));
  epoch = (uint32_t)w;
  err = (uint32_t)(w >> 32);
}

// A block's tile of y filled with NaN (one wave: lane = pair of columns).
__device__ inline void poison_tile(float* y, int b, int d, int tile, int lane) {
  const int half_cols = min(kTile, d - tile * kTile) / 2;
  const float nan = __builtin_nanf("");
  const uint64_t v = ((uint64_t)__float_as_uint(nan) << 32) | __float_as_uint(nan);
  for (int t = 0; t < b; ++t) {
    uint64_t* yt = reinterpret_cast<uint64_t*>(y + (size_t)t * d + tile * kTile);
    for (int c = lane; c < half_cols; c += kWave) st_agent64(yt + c, v);
  }
}

// Dot products of a row held as NU 16-byte units per lane (unit lane + 64 j)
// with the BM tokens in LDS (token t at xs[t * NU * 64], a compile-time
// stride, so that the tokens of a unit are read with immediate offsets from
// one address); wave-uniform results.
// Units past the row's end (u >= U) hold a repeat of its last unit and are
// left out with a select, not a branch.
template <int BM, int NU>
__device__ inline void row_dots(const u32x4 (&v)[NU], const u32x4* xs, int U, int lane, float (&out)[BM]) {
  float acc[BM];
#pragma unroll
  for (int t = 0; t < BM; ++t) acc[t] = 0.f;
#pragma unroll
  for (int j = 0; j < NU; ++j) {
    const int u = lane + kWave * j;
    const int uc = min(u, U - 1);
#pragma unroll
    for (int t = 0; t < BM; ++t) {
      const float s = dot8(v[j], xs[t * (NU * kWave) + uc], acc[t]);
      acc[t] = u < U ? s : acc[t];
    }
  }
#pragma unroll
  for (int t = 0; t < BM; ++t) out[t] = wave_total(acc[t]);
}

// All NU requests of a row in straight-line code (no per-unit branches, so
// the compiler can count them and issue them back to back); units past the
// row's end repeat its last unit.
template <int NU>
__device__ inline void load_row(const u32x4* __restrict__ row, int U, int lane, u32x4 (&v)[NU]) {
#pragma unroll
  for (int j = 0; j < NU; ++j) v[j] = load_nt(row + min(lane + kWave * j, U - 1));
}

// 16-byte units per lane that cover a row of d fp16 values (template bucket).
inline int units_per_lane(int d) {
  const int nu = (d / 8 + kWave - 1) / kWave;
  return nu <= 1 ? 1 : nu <= 2 ? 2 : nu <= 4 ? 4 : nu <= 8 ? 8 : nu <= 10 ? 10 : 16;
}

// Batch bucket of the kernel: the smallest of 1, 2, 4, 8 that holds b.
inline int batch_bucket(int b) { return b <= 1 ? 1 : b <= 2 ? 2 : b <= 4 ? 4 : 8; }

// Per-block work counts -> counters[3] = {n_gate, n_up, n_down}.
hipError_t launch_sum_counts(const int32_t* counts, int slots, const int32_t* n_active, int k, int32_t* counters,
                             hipStream_t s);

#define SI_NU_DISPATCH(BM, CALL)   \
  switch (units_per_lane(d)) {     \
    case 1: return CALL(BM, 1);    \
    case 2: return CALL(BM, 2);    \
    case 4: return CALL(BM, 4);    \
    case 8: return CALL(BM, 8);    \
    case 10: return CALL(BM, 10);  \
    default: return CALL(BM, 16);  \
  }

#define SI_LAYER_DISPATCH(CALL)        \
  switch (batch_bucket(b)) {           \
    case 1: SI_NU_DISPATCH(1, CALL)    \
    case 2: SI_NU_DISPATCH(2, CALL)    \
    case 4: SI_NU_DISPATCH(4, CALL)    \
    default: SI_NU_DISPATCH(8, CALL)   \
  }

}  // namespace si
