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
// INT8 weights (the kernel's third form): W_gate, W_up and W_down^T hold
// INT8 values with one float scale per output channel (rows of W_gate and
// W_up, columns of y for W_down^T).  The predictor reads the same packed
// signs (the MSBs of the INT8 weights), gate/up converts each row's INT8
// values exactly to fp16 in registers and scales the dot products, and the
// down-projection scales each column of y once, at the tile's add.
//
// No block waits for the whole grid: the only exchanges are inside a group.
// One block (the last, where the grid has a block without rows, else block 0)
// adds the published kept counts (the count of the call) and, having seen a
// word of this call from every block, advances the call counter.
// When the caller asks for the ascending kept list, each block adds the
// counts of the blocks before it at the end and writes its rows' entries.
//
// Exchange words are 64-bit: this call's tag (the workspace's call counter
// with the high bit set) in the high half, the payload in the low half,
// written with agent-scope write-through stores and read with agent-scope
// loads, so no cache flush or fence is needed and the workspace is never
// cleared between calls.  Every wait is bounded: past a spin limit the block
// sets an error bit in the workspace header and goes on without the data.

#include <type_traits>

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
constexpr int kMaxPairs = kWave;                   // (owner block, pass) pairs of one group
constexpr int kMaxChunkRows = 4096;                // kept rows of one group (at most)
constexpr int kWideGroupRows = 512;                // one token: groups larger than this take wider down batches
static_assert(kCountWord < kOwnPubStride, "published words of a block");

// Eight wavefronts per block (two per SIMD), so that a wave may hold up to
// 256 registers: a row of W_gate and of W_up in flight together, and the
// accumulators of 8 tokens, without spilling.
constexpr int kOW = 8;
constexpr int kOT = kOW * kWave;
constexpr int kOSignUnits = (kMaxD / 128 + kOW - 1) / kOW;  // sign units per wave and pass, at most (8)
constexpr int kFin = kOW - 1;      // the wave that finishes the prediction
constexpr int kTileWave = kOW - 2; // the wave that initialises the owner's tile of y
constexpr int kODN = 8;            // W_down^T pieces per wave and down round
// one token: W_down^T pieces per batch a wave takes, with INT8 weights, and
// in groups of more than kWideGroupRows rows (measured, us per call:
// 7B-shaped groups of 384 rows 12.33 / 12.23 / 12.18 / 12.41 with batches of
// 6 / 8 / 10 / 12, INT8 12.23 / 11.87 / 11.76 / 11.94 / 12.54 with 4 / 6 /
// 8 / 10 / 16; 13B-shaped groups of 560 rows 17.71 / 17.60 / 18.04 with
// 10 / 12 / 14; with the one-pass fold, on one box: 7B 12.12 / 12.16 /
// 12.13 / 12.21, decoder-block call 12.67 / 12.75 / 12.74 / 12.80, and the
// OPT-shaped non-gated call 13.18 / 12.70 / 12.45 / 12.63 with 7 / 8 / 9 /
// 10, while 11 was 0.05 us slower than 10 at 7B)
constexpr int kODN1 = 9;
constexpr int kODN1Int8 = 8;
constexpr int kODN1Wide = 12;
static_assert(kODN1 < kWave && kODN1Int8 < kWave && kODN1Wide < kWave, "a wave's last lane polls the tile's zero flag");
static_assert(kODN * kMaxB <= kWave, "a wave polls the h3 words of its pieces, one lane per (piece, token)");

// The down-projection on the matrix cores (4-8 tokens; INT8 pieces are
// turned into fp16, exactly, on their way into LDS): the group's rows in
// chunks of 32 (the K of one 16x16x32 fp16 MFMA), the tile's
// 512 columns split over the 8 waves (64 each, four 16-column blocks), the
// tokens padded to 16.  A chunk's W_down^T pieces pass through LDS, where
// transposing reads give each lane 8 rows of one column (the A operand); h3
// is the B operand, scaled per token and chunk by a power of two and split
// into two fp16 parts (hi + lo), so the products keep fp32 precision for any
// finite h3.
constexpr int kMRows = 32;                // rows per chunk
constexpr int kMInflight = 3;             // chunks whose pieces are in flight (3-4 tokens; one more with 5-8)
constexpr int kMPitch = kTile * 2 + 32;   // bytes per row of a chunk in LDS (padded against bank conflicts)
constexpr int kMTok = 16;                 // tokens of the MFMA (b <= 8 used)
static_assert(kMRows == 4 * kOW, "each wave stages 4 rows of a chunk (16 lanes per row)");
static_assert(kTile == 4 * 16 * kOW, "four 16-column blocks per wave");
template <int BM>
struct MfmaLds {
  unsigned char rows[kMRows * kMPitch];  // the chunk's pieces, row-major
  uint16_t bop[2][kMTok][kMRows];        // h3 (hi, lo) as fp16, token-major
};

struct OwnedArgs {
  const u32x4* signs;
  const u32x4* wg;
  const u32x4* wu;         // nullptr: the non-gated ReLU MLP (h3 = ReLU(g))
  const u32x4* wdt;
  const float* sg;         // INT8 form: scales of the rows of W_gate, W_up, and of the columns of y
  const float* su;
  const float* sd;
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
  const float* h;          // decoder-block mode: the residual stream [b][d] (x = RMSNorm(h) * norm_w)
  const float* norm_w;     // [d]
  float eps;
};

template <int BM, int NU>
struct OwnedLds {
  static constexpr int kUnits = NU * kWave;
  static constexpr int kFold = kOW / BM;  // per-wave partial tiles held at once in the fold
  // tokens (fp16); once the gate/up work is done, the per-wave partial tiles
  union {
    u32x4 xs[BM * kUnits];
    float dpart[kFold][BM][kTile];
    unsigned char mf_raw[BM >= 4 ? sizeof(MfmaLds<BM>) : 16];  // the down-projection on the matrix cores
  };
  uint32_t xw[BM * kUnits / 4];  // sign words of the tokens
  // per-wave N_neg partial counts during the prediction; the group's kept
  // rows in order afterwards
  union {
    int cpart[kOW][BM][kWave];
    uint32_t dent[kMaxChunkRows];  // conf << 31 | row
  };
  uint32_t pm[4 * kMaxPairs];  // the group's published mask words
  uint32_t srow[kMaxOwnRows];  // conf << 31 | row of the block's kept rows, ascending
  int wsum[kOW];
  float nsum[kOW][kMaxB];  // decoder-block mode: per-wave sums of squares of the tokens
  int n_own, n_up, n_down;
  int gpos;  // next gate/up position of the member's range not yet taken by a wave
  int dpos;    // one token: next down position not yet taken by a wave
  int issued;  // one token: waves whose first gate/up row is requested
  uint32_t epoch, err;
  uint32_t dmax[2][kMaxB];  // matrix-core down-projection: max |h3| bits per token (chunks alternate)
  float dinv[kMaxB];        // and the inverse of its scale
  // one token: the per-wave partial tiles, apart from the tokens, so that a
  // wave stores its tile as soon as its down batches are done (last, so
  // that the other fields keep their offsets)
  float dpart1[BM == 1 ? kOW : 1][BM == 1 ? kTile : 1];
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
  int t = lane < kOW ? L.wsum[lane] : 0;
  t = wave_sum_int(t);
  __syncthreads();
  return t;
}

// Sum of every block's published kept count (one poll per thread of the
// calling threads [t0, t0 + nt)); proof too that every block has read the
// call counter.
__device__ inline int census_part(const uint64_t* pub, int P, int t, int nt, uint32_t tag, uint32_t* hdr) {
  int sum = 0;
  for (int o = t; o < P; o += nt) {
    const uint64_t* src[1] = {&pub[(size_t)o * kOwnPubStride + kCountWord]};
    uint32_t v[1];
    poll_words<1>(src, 1, tag, hdr, v);
    sum += (int)v[0];
  }
  return sum;
}

// Dot products of two rows held as NU 16-byte units per lane (unit lane +
// 64 j) with the BM tokens in LDS (token t at xs[t * NU * 64]); each token
// unit is read once for both rows.  Wave-uniform results.
template <int BM, int NU>
__device__ inline void row_dots2(const u32x4 (&v)[NU], const u32x4 (&w)[NU], const u32x4* xs, int U, int lane,
                                 float (&o1)[BM], float (&o2)[BM]) {
  float a1[BM], a2[BM];
#pragma unroll
  for (int t = 0; t < BM; ++t) a1[t] = a2[t] = 0.f;
#pragma unroll
  for (int j = 0; j < NU; ++j) {
    const int u = lane + kWave * j;
    const int uc = min(u, U - 1);
#pragma unroll
    for (int t = 0; t < BM; ++t) {
      const u32x4 xv = xs[t * (NU * kWave) + uc];
      const float s1 = dot8(v[j], xv, a1[t]);
      const float s2 = dot8(w[j], xv, a2[t]);
      a1[t] = u < U ? s1 : a1[t];
      a2[t] = u < U ? s2 : a2[t];
    }
    // one unit's token values live at a time (with 8 tokens the scheduler
    // would otherwise hoist every unit's LDS reads and spill)
    if constexpr (BM >= 4) __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int t = 0; t < BM; ++t) {
    o1[t] = wave_total(a1[t]);
    o2[t] = wave_total(a2[t]);
  }
}

// The 16 INT8 values of a 16-byte unit as 16 fp16 values (two 16-byte
// vectors), exactly: each byte, offset by 128, becomes the low mantissa
// byte of the fp16 value 1024 + (q + 128), from which 1152 is subtracted
// (every value on the way is an integer below 2048).
__device__ inline uint32_t i8_pair(uint32_t biased) {
  return __builtin_bit_cast(uint32_t, as_h2(biased | 0x64006400u) - f16x2{(_Float16)1152.0f, (_Float16)1152.0f});
}
__device__ inline void i8_to_h16(u32x4 v, u32x4& lo, u32x4& hi) {
  const uint32_t a = v.x ^ 0x80808080u, b = v.y ^ 0x80808080u, c = v.z ^ 0x80808080u, e = v.w ^ 0x80808080u;
  auto p01 = [](uint32_t t) { return i8_pair((t & 0xffu) | ((t & 0xff00u) << 8)); };
  auto p23 = [](uint32_t t) { return i8_pair(((t >> 16) & 0xffu) | ((t >> 8) & 0xff0000u)); };
  lo = u32x4{p01(a), p23(a), p01(b), p23(b)};
  hi = u32x4{p01(c), p23(c), p01(e), p23(e)};
}

// Dot products of one or two INT8 rows held as (NU + 1) / 2 16-byte units
// per lane (unit lane + 64 j: 16 values, the tokens' fp16 units 2u and
// 2u + 1) with the BM tokens in LDS; unscaled, wave-uniform results.
template <int BM, int NU, bool TWO>
__device__ inline void row_dots_i8(const u32x4 (&v)[(NU + 1) / 2], const u32x4 (&w)[(NU + 1) / 2],
                                   const u32x4* xs, int U8, int lane, float (&o1)[BM], float (&o2)[BM]) {
  constexpr int NU8 = (NU + 1) / 2;
  float a1[BM], a2[BM];
#pragma unroll
  for (int t = 0; t < BM; ++t) a1[t] = a2[t] = 0.f;
#pragma unroll
  for (int j = 0; j < NU8; ++j) {
    const int u = lane + kWave * j;
    const int uc = min(u, U8 - 1);
    u32x4 vl, vh, wl, wh;
    i8_to_h16(v[j], vl, vh);
    if constexpr (TWO) i8_to_h16(w[j], wl, wh);
#pragma unroll
    for (int t = 0; t < BM; ++t) {
      const u32x4 x0 = xs[t * (NU * kWave) + 2 * uc], x1 = xs[t * (NU * kWave) + 2 * uc + 1];
      const float s1 = dot8(vh, x1, dot8(vl, x0, a1[t]));
      a1[t] = u < U8 ? s1 : a1[t];
      if constexpr (TWO) {
        const float s2 = dot8(wh, x1, dot8(wl, x0, a2[t]));
        a2[t] = u < U8 ? s2 : a2[t];
      }
    }
    if constexpr (BM >= 4) __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int t = 0; t < BM; ++t) {
    o1[t] = wave_total(a1[t]);
    o2[t] = TWO ? wave_total(a2[t]) : 0.f;
  }
}

// A W_down^T piece of one row for one lane: 8 columns (fp16: 16 bytes; INT8:
// 8 bytes) and their values as floats.
template <bool I8>
struct DownPiece {
  typedef u32x4 type;
  static __device__ inline type load(const u32x4* wdt, size_t row, int U, int unit) {
    return load_nt(wdt + row * U + unit);
  }
  static __device__ inline void values(type v, float (&f)[8]) {
    const f16x2 p0 = as_h2(v.x), p1 = as_h2(v.y), p2 = as_h2(v.z), p3 = as_h2(v.w);
    f[0] = (float)p0.x; f[1] = (float)p0.y; f[2] = (float)p1.x; f[3] = (float)p1.y;
    f[4] = (float)p2.x; f[5] = (float)p2.y; f[6] = (float)p3.x; f[7] = (float)p3.y;
  }
  // the 8 columns as fp16 (the matrix-core down-projection's A operand)
  static __device__ inline u32x4 as_f16(type v) { return v; }
};
template <>
struct DownPiece<true> {
  typedef uint32_t type __attribute__((ext_vector_type(2)));
  static __device__ inline type load(const u32x4* wdt, size_t row, int U, int unit) {
    return __builtin_nontemporal_load(reinterpret_cast<const type*>(wdt) + row * U + unit);
  }
  static __device__ inline void values(type v, float (&f)[8]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[i] = (float)(int8_t)(v.x >> (8 * i));
      f[4 + i] = (float)(int8_t)(v.y >> (8 * i));
    }
  }
  // the 8 INT8 values as fp16 (exact: |q| <= 128 < 2048), the column scales
  // being applied at the tile's add into y
  static __device__ inline u32x4 as_f16(type v) {
    float f[8];
    values(v, f);
    u32x4 r;
    r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(f[0], f[1]));
    r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(f[2], f[3]));
    r.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(f[4], f[5]));
    r.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(f[6], f[7]));
    return r;
  }
};

constexpr int kModePlain = 0;  // fp16 weights, x given
constexpr int kModeBlock = 1;  // fp16 weights, x = RMSNorm(h) * norm_w, y = h + MLP
constexpr int kModeInt8 = 2;   // INT8 weights with per-channel scales, x given

// MODE: the kernel's form (above); each is a separate instance so that the
// plain form carries none of the others' code (the decoder-block code alone
// cost the plain form 0.3 us per call)
// WIDE (one token): the down batches take kODN1Wide pieces instead of kODN1,
// for groups of more than kWideGroupRows rows (a separate instance: carrying
// both batch widths made the 7B call 0.25 us slower)
template <int BM, int NU, int MODE, bool WIDE>
__global__ __launch_bounds__(kOT) void k_owned(OwnedArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  OwnedLds<BM, NU>& L = *reinterpret_cast<OwnedLds<BM, NU>*>(lds_raw);

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d = a.d, U = d >> 3, W = d >> 5, units = d >> 7;
  const int b = a.b, k = a.k;
  const int P = gridDim.x, blk = blockIdx.x;
  const int T = a.tiles, R = a.R, nsub = a.nsub;
  const int r0 = blk * R;
  // the block that takes the census of the blocks' kept counts: one without
  // rows where the grid has one (the census waits for the last block to
  // publish, which a block with rows would wait for before its gate/up)
  const int cblk = a.groups * T < P ? P - 1 : 0;
  const int Rb = blk < a.groups * T ? max(0, min(R, k - r0)) : 0;  // rows this block owns
  const bool predict = a.mask_in == nullptr;
  const bool no_as = (a.flags & kNoAS) != 0;
  const bool spec_ok = (a.flags & kNoSpec) == 0;
  const bool gated = a.wu != nullptr;  // else the non-gated ReLU MLP (no W_up)
  const bool owns_tile = a.mlp && blk < T;

  SI_TRACE_DECL;
  SI_TRACE_MARK(0);
  // ---- the sign units (or mask bytes) of the first 64 owned rows are
  // requested, then the tokens and (behind the first token requests, so that
  // the wait for it, which comes at once for an atomic load, also covers
  // them) the call counter; addresses are clamped so that the requests are
  // unconditional and go out back to back; tokens b..BM-1 are zero
  // a row has d/128 <= 4 NU sign units, so a wave counts at most
  // ceil(NU / 2) of them per pass; the requests are unconditional (clamped
  // unit, the same line again where a wave has fewer) so that the counts
  // can start as the first ones arrive
  constexpr int kSU = (NU + 1) / 2;
  static_assert(kSU <= kOSignUnits, "sign units per wave");
  u32x4 sreg[kSU];
  const int kpad = (k + kRowGroup - 1) / kRowGroup * kRowGroup;  // rows of the packed layout
  auto load_signs = [&](int s) {
    const u32x4* sg = a.signs + r0 + min(s * kWave + lane, Rb - 1);
#pragma unroll
    for (int i = 0; i < kSU; ++i) {
      const int q = min(wv + kOW * i, units - 1);
      sreg[i] = load_nt(sg + (size_t)q * kpad);
    }
  };
  uint32_t mbyte = 0;
  if (Rb > 0) {
    if (predict) load_signs(0);
    else if (wv == kFin) mbyte = a.mask_in[r0 + min(lane, Rb - 1)];
  }
  // the owner of tile blk of y zeroes it (in decoder-block mode it copies
  // the residual in later); the same wave later announces it in the tile's
  // flag
  constexpr bool block_mode = MODE == kModeBlock;
  constexpr bool kI8 = MODE == kModeInt8;
  if (!block_mode && owns_tile && wv == kTileWave) {
    const int half_cols = min(kTile, d - blk * kTile) / 2;
    for (int t = 0; t < b; ++t) {
      uint64_t* yt = reinterpret_cast<uint64_t*>(a.y + (size_t)t * d + blk * kTile);
      for (int c = lane; c < half_cols; c += kWave) st_agent64(yt + c, 0ull);
    }
  }
  // decoder-block mode with one token: the tile wave requests its 8 values
  // of the residual h in the owner's tile now (lane = unit of the tile) and
  // stores them into y after the group exchange, so that neither the loads
  // nor the stores delay the published masks (with more tokens the tile is
  // copied while the finishing wave publishes: holding every token's values
  // until after the exchange was no faster)
  float4 htile[2] = {};
  const int tunit = blk * kWave + lane;  // the lane's unit (8 columns) of the tile
  if constexpr (block_mode && BM == 1) {
    if (owns_tile && wv == kTileWave && tunit < U) {
      const float4* hv4 = reinterpret_cast<const float4*>(a.h);
      htile[0] = hv4[2 * tunit];
      htile[1] = hv4[2 * tunit + 1];
    }
  }
  // token t's unit u at xs[t * XS + u] (XS = NU * 64 >= U)
  constexpr int XS = OwnedLds<BM, NU>::kUnits;
  // decoder-block mode: h and norm_w as 16-byte vectors; each thread's
  // units (two at most) are kept in registers from the sums of squares to
  // the scaling, which runs once the counts are done.  The units go to the
  // threads of waves 0..6 only: the finishing wave, which publishes the
  // masks, has no scaling to do after its stores (the compiler would wait
  // for those stores first)
  const float4* hg = reinterpret_cast<const float4*>(a.h);
  const float4* wg4 = reinterpret_cast<const float4*>(a.norm_w);
  constexpr int kXT = kOT - kWave;  // threads holding units of h
  static_assert(kFin == kOW - 1, "the finishing wave is the last one");
  constexpr int J = (BM * XS + kXT - 1) / kXT;  // units per thread (incl. padding)
  constexpr bool kKeep = J <= 2;
  float4 hr[kKeep ? J : 1][2], wr[kKeep ? J : 1][2];
  // otherwise (several tokens, or a wide row) thread tid takes the units
  // u = tid + j kOT of every token: the unit of norm_w is read once for all
  // tokens, and the b + 1 requests of a unit go out together.  Where they
  // fit, the values stay in registers from the sums of squares to the
  // scaling (which then runs right after the first barrier)
  constexpr int JU = (XS + kOT - 1) / kOT;
  constexpr bool kHold = JU * (BM + 1) * 8 <= 80;
  float4 hk[kHold ? JU : 1][BM][2], wk[kHold ? JU : 1][2];
  auto load_unit = [&](int u, float4 (&hv)[BM][2], float4 (&nv)[2]) {
    const int uc = min(u, U - 1);
    nv[0] = wg4[2 * uc];
    nv[1] = wg4[2 * uc + 1];
#pragma unroll
    for (int t = 0; t < BM; ++t) {
      const int i = min(t, b - 1) * U + uc;
      hv[t][0] = hg[2 * i];
      hv[t][1] = hg[2 * i + 1];
    }
  };
  // decoder-block mode: x = the fp16 rounding of h * r_t * norm_w, r_t the
  // token's RMS normaliser from the block's sums of squares (the units kept
  // in hr / wr)
  auto scale_x = [&]() {
    if (tid >= kXT) return;
    float r[BM];
#pragma unroll
    for (int t = 0; t < BM; ++t) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < kOW; ++w) v += L.nsum[w][t];
      r[t] = 1.0f / sqrtf(v / (float)d + a.eps);
    }
#pragma unroll
    for (int j = 0; j < (kKeep ? J : 0); ++j) {
      const int i = tid + j * kXT, t = i / XS, u = i - t * XS;
      if (i < BM * XS) {
        u32x4 xv{0, 0, 0, 0};
        if (t < b && u < U) {
          float rt = 0.f;
#pragma unroll
          for (int tt = 0; tt < BM; ++tt) rt = tt == t ? r[tt] : rt;
          const float4 p = hr[j][0], q = hr[j][1], wp = wr[j][0], wq = wr[j][1];
          xv.x = pack_h2((p.x * rt) * wp.x, (p.y * rt) * wp.y);
          xv.y = pack_h2((p.z * rt) * wp.z, (p.w * rt) * wp.w);
          xv.z = pack_h2((q.x * rt) * wq.x, (q.y * rt) * wq.y);
          xv.w = pack_h2((q.z * rt) * wq.z, (q.w * rt) * wq.w);
        }
        L.xs[i] = xv;
      }
    }
  };
  auto scale_units = [&]() {
    float r[BM];
#pragma unroll
    for (int t = 0; t < BM; ++t) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < kOW; ++w) v += L.nsum[w][t];
      r[t] = 1.0f / sqrtf(v / (float)d + a.eps);
    }
#pragma unroll
    for (int j = 0; j < JU; ++j) {
      const int u = tid + j * kOT;
      if (u < XS) {
        float4 hv[BM][2], nv[2];
        if constexpr (kHold) {
#pragma unroll
          for (int t = 0; t < BM; ++t) {
            hv[t][0] = hk[j][t][0];
            hv[t][1] = hk[j][t][1];
          }
          nv[0] = wk[j][0];
          nv[1] = wk[j][1];
        } else {
          load_unit(u, hv, nv);
        }
#pragma unroll
        for (int t = 0; t < BM; ++t) {
          u32x4 xv{0, 0, 0, 0};
          if (t < b && u < U) {
            const float4 p = hv[t][0], q = hv[t][1], wp = nv[0], wq = nv[1];
            const float rt = r[t];
            xv.x = pack_h2((p.x * rt) * wp.x, (p.y * rt) * wp.y);
            xv.y = pack_h2((p.z * rt) * wp.z, (p.w * rt) * wp.w);
            xv.z = pack_h2((q.x * rt) * wq.x, (q.y * rt) * wq.y);
            xv.w = pack_h2((q.z * rt) * wq.z, (q.w * rt) * wq.w);
          }
          L.xs[t * XS + u] = xv;
        }
      }
    }
  };
  if constexpr (!block_mode && BM == 1) {
    const u32x4* xg = reinterpret_cast<const u32x4*>(a.x);
    for (int i = tid; i < XS; i += kOT) {
      const u32x4 xv = xg[min(i, U - 1)];
      if (i == tid && tid == 0) {
        asm volatile("" ::: "memory");
        load_epoch(a.hdr, L.epoch, L.err);
        L.n_up = 0;
        L.n_down = 0;
      }
      L.xs[i] = i < U ? xv : u32x4{0, 0, 0, 0};
    }
  } else if constexpr (!block_mode) {
    // with 2-8 tokens every unit of the thread is requested before any is
    // stored, so that the requests travel together (a load-store loop
    // waits once per unit: 2 us of 64 KB with 8 tokens)
    const u32x4* xg = reinterpret_cast<const u32x4*>(a.x);
    const int nx = b * U;
    constexpr int JX = (BM * XS + kOT - 1) / kOT;
    if constexpr (BM == 4) {
      // 3-4 tokens: the units go straight from memory into LDS
      // (global_load_lds, 16 bytes per lane, a wave's 64 consecutive units of
      // xs) without passing through registers; units past a token's d or of
      // tokens b..BM-1 are zeroed once the copies have landed.  (The 4-token
      // mask call 24.37 -> 23.76 us; with 2 and 8 tokens the same copies were
      // 0.1-0.3 us slower than the loads below.)
      static_assert(XS % kWave == 0, "a wave's units of xs lie within one token");
#pragma unroll
      for (int j = 0; j < JX; ++j) {
        const int base = wv * kWave + j * kOT;  // the wave's first unit (wave-uniform)
        if (base < BM * XS) {
          const int i = base + lane, t = i / XS, u = i - t * XS;
          __builtin_amdgcn_global_load_lds(xg + min(t * U + u, nx - 1),
                                           (__attribute__((address_space(3))) void*)(&L.xs[base]), 16, 0, 0);
        }
      }
      if (tid == 0) {
        asm volatile("" ::: "memory");
        load_epoch(a.hdr, L.epoch, L.err);
        L.n_up = 0;
        L.n_down = 0;
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
      for (int j = 0; j < JX; ++j) {
        const int i = tid + j * kOT, t = i / XS, u = i - t * XS;
        if (i < BM * XS && !(t < b && u < U)) L.xs[i] = u32x4{0, 0, 0, 0};
      }
    } else {
      u32x4 xv[JX];
#pragma unroll
      for (int j = 0; j < JX; ++j) {
        const int i = tid + j * kOT, t = i / XS, u = i - t * XS;
        xv[j] = xg[min(t * U + u, nx - 1)];
      }
      if (tid == 0) {
        asm volatile("" ::: "memory");
        load_epoch(a.hdr, L.epoch, L.err);
        L.n_up = 0;
        L.n_down = 0;
      }
#pragma unroll
      for (int j = 0; j < JX; ++j) {
        const int i = tid + j * kOT, t = i / XS, u = i - t * XS;
        if (i < BM * XS) L.xs[i] = (t < b && u < U) ? xv[j] : u32x4{0, 0, 0, 0};
      }
    }
  } else {
    // decoder-block mode: x = RMSNorm(h) * norm_w in fp16, formed here from
    // the fp32 residual stream: the sums of squares over the block, then
    // every unit of 8 values scaled and rounded.  Where a thread has at most
    // two units (b * d <= 8192) its h and norm_w values stay in registers
    // between the two steps; otherwise the units go one per thread and
    // token column (above).
    float ss[BM];
#pragma unroll
    for (int t = 0; t < BM; ++t) ss[t] = 0.f;
    // the sign byte of x's unit: the XOR of the signs of h and norm_w (the
    // scale is positive, and rounding to fp16 keeps the sign, zeros
    // included), so the predictor's sign words need no norm
    auto sign_byte = [](float4 p, float4 q) -> uint32_t {
      return (__float_as_uint(p.x) >> 31) | ((__float_as_uint(p.y) >> 31) << 1) |
             ((__float_as_uint(p.z) >> 31) << 2) | ((__float_as_uint(p.w) >> 31) << 3) |
             ((__float_as_uint(q.x) >> 31) << 4) | ((__float_as_uint(q.y) >> 31) << 5) |
             ((__float_as_uint(q.z) >> 31) << 6) | ((__float_as_uint(q.w) >> 31) << 7);
    };
    if constexpr (!kKeep) {
#pragma unroll
      for (int j = 0; j < JU; ++j) {
        const int u = tid + j * kOT;
        float4 hv[BM][2], nv[2];
        load_unit(u, hv, nv);
        if (u < U) {
          const uint32_t wb = sign_byte(nv[0], nv[1]);
#pragma unroll
          for (int t = 0; t < BM; ++t) {
            if (t < b) {
              const float4 p = hv[t][0], q = hv[t][1];
              ss[t] += p.x * p.x + p.y * p.y + p.z * p.z + p.w * p.w + q.x * q.x + q.y * q.y + q.z * q.z + q.w * q.w;
              reinterpret_cast<uint8_t*>(L.xw)[t * 4 * W + u] = (uint8_t)(sign_byte(p, q) ^ wb);
            }
          }
        }
        if constexpr (kHold) {
#pragma unroll
          for (int t = 0; t < BM; ++t) {
            hk[j][t][0] = hv[t][0];
            hk[j][t][1] = hv[t][1];
          }
          wk[j][0] = nv[0];
          wk[j][1] = nv[1];
        }
      }
    }
#pragma unroll
    for (int j = 0; j < (kKeep ? J : 0); ++j) {
      const int i = tid + j * kXT, t = i / XS, u = i - t * XS;
      if (tid < kXT && i < BM * XS && t < b && u < U) {
        const float4 p = hg[2 * (t * U + u)], q = hg[2 * (t * U + u) + 1];
        if constexpr (kKeep) {
          hr[j][0] = p;
          hr[j][1] = q;
        }
        const float v = p.x * p.x + p.y * p.y + p.z * p.z + p.w * p.w + q.x * q.x + q.y * q.y + q.z * q.z + q.w * q.w;
#pragma unroll
        for (int tt = 0; tt < BM; ++tt) ss[tt] += tt == t ? v : 0.f;
        // the predictor's sign byte of this unit (byte u of the token's
        // sign words)
        const float4 wp = wg4[2 * u], wq = wg4[2 * u + 1];
        if constexpr (kKeep) {
          wr[j][0] = wp;
          wr[j][1] = wq;
        }
        reinterpret_cast<uint8_t*>(L.xw)[t * 4 * W + u] = (uint8_t)(sign_byte(p, q) ^ sign_byte(wp, wq));
      }
    }
    if (tid == 0) {
      asm volatile("" ::: "memory");
      load_epoch(a.hdr, L.epoch, L.err);
      L.n_up = 0;
      L.n_down = 0;
    }
#pragma unroll
    for (int t = 0; t < BM; ++t) {
      const float v = wave_total(ss[t]);
      if (lane == 0) L.nsum[wv][t] = v;
    }
  }
  __syncthreads();
  // a workspace left inconsistent by a call whose bounded wait gave up (its
  // sticky error word is set): nothing is computed until the workspace is
  // reset, and the owners of the tiles of y fill them with NaN
  if (uniform(L.err) & kErrLookbackSpin) {
    if (owns_tile && wv == kTileWave) poison_tile(a.y, b, d, blk, lane);
    return;
  }
  if constexpr (block_mode && !kKeep) scale_units();  // before the counts, not behind the publishing stores
  const uint32_t epoch = uniform(L.epoch);
  const uint32_t tag = epoch_tag(epoch);
  // consumed here, where the wait for it is covered by the token requests (a
  // load left outstanding into the loop below would make the compiler wait
  // for every outstanding request, stores included, inside it)
  bool mkeep = mbyte != 0;
  if constexpr (!block_mode) {  // (written with the norm, before the barrier above, in decoder-block mode)
    if (predict) {
      for (int i = tid; i < BM * W; i += kOT) {  // tokens b..BM-1 are zero
        const int t = i / W, w = i - t * W;
        L.xw[i] = sign_word(&L.xs[t * OwnedLds<BM, NU>::kUnits + 4 * w]);
      }
    }
    __syncthreads();
  }
  SI_TRACE_MARK(1);

  // ---- 1. kept and confident masks of the owned rows, 64 rows per pass;
  // the finishing wave applies the rule, lists the kept rows in order and
  // publishes, so no wave with gate/up work waits for those stores
  int n_own = 0;  // finishing wave
  for (int s = 0; s < nsub; ++s) {
    const bool any_rows = s * kWave < Rb;
    if (predict && any_rows) {
      if (s > 0) load_signs(s);
      int c[BM];
#pragma unroll
      for (int t = 0; t < BM; ++t) c[t] = 0;
#pragma unroll
      for (int i = 0; i < kSU; ++i) {
        const int q = wv + kOW * i;
        const int qc = min(q, units - 1);
#pragma unroll
        for (int t = 0; t < BM; ++t) {
          const u32x4 xv = *reinterpret_cast<const u32x4*>(&L.xw[t * W + 4 * qc]);
          const int n = __popc(sreg[i].x ^ xv.x) + __popc(sreg[i].y ^ xv.y) + __popc(sreg[i].z ^ xv.z) +
                        __popc(sreg[i].w ^ xv.w);
          c[t] += q < units ? n : 0;
        }
      }
      // every wave stores its partial counts (zero without units)
#pragma unroll
      for (int t = 0; t < BM; ++t) L.cpart[wv][t][lane] = c[t];
      __syncthreads();
      if (s == 0) SI_TRACE_MARK(2);
    }
    if (wv == kFin) {
      // every request of this wave has completed here (the sign units for
      // the counts, the tile's zeroing stores before the tokens); said
      // explicitly so that the publishing stores below are not waited for
      wait_all_requests();
      const int i = s * kWave + lane;
      const int row = r0 + i;
      const bool valid = i < Rb;
      bool keep = false, conf = false;
      if (predict) {
        if (any_rows) {
#pragma unroll
          for (int t = 0; t < BM; ++t) {
            int n_neg = 0;
#pragma unroll
            for (int w = 0; w < kOW; ++w) n_neg += L.cpart[w][t][lane];
            keep |= t < b && n_neg < a.T;
            conf |= t < b && n_neg < a.T - a.margin;
          }
        }
      } else if (any_rows) {
        if (s > 0) mkeep = a.mask_in[r0 + min(i, Rb - 1)] != 0;
        keep = mkeep;
        conf = keep;
      }
      keep = keep && valid;
      const uint64_t kb = __ballot(keep);
      const uint64_t cb = __ballot(keep && conf);
      if (keep) L.srow[n_own + __popcll(kb & lanes_below(lane))] = (uint32_t)row | (conf ? 0x80000000u : 0u);
      n_own += __popcll(kb);
      // lanes 0-3: this pass's kept and confident words; after the last
      // pass lane 4 also publishes the block's kept count (in the same
      // store instruction, before any later request of this wave)
      const bool last = s + 1 == nsub;
      if (lane < 4 || (last && lane == 4)) {
        const uint64_t m = lane < 2 ? kb : cb;
        const uint32_t v = lane < 4 ? (uint32_t)(m >> (32 * (lane & 1))) : (uint32_t)n_own;
        st_agent64(&a.pub[(size_t)blk * kOwnPubStride + (lane < 4 ? 4 * s + lane : kCountWord)], tagged(tag, v));
      }
      if (valid && a.mask) a.mask[row] = keep ? 1 : 0;
      if (last && lane == 0) L.n_own = n_own;
    }
    if (predict && any_rows && s + 1 < nsub) __syncthreads();  // the partial counts are reused
  }
  // decoder-block mode with several tokens: the owner's tile of y starts as
  // the residual h (lane = unit of the tile; every token's unit is requested
  // before any is stored)
  if constexpr (block_mode && BM > 1) {
    if (owns_tile && wv == kTileWave && tunit < U) {
      float4 hv[BM][2];
#pragma unroll
      for (int t = 0; t < BM; ++t) {
        const size_t i = (size_t)min(t, b - 1) * U + tunit;
        hv[t][0] = hg[2 * i];
        hv[t][1] = hg[2 * i + 1];
      }
#pragma unroll
      for (int t = 0; t < BM; ++t) {
        if (t < b) {
          uint64_t* yu = reinterpret_cast<uint64_t*>(a.y + (size_t)t * d) + 4 * (size_t)tunit;
          st_agent64(yu, ((uint64_t)__float_as_uint(hv[t][0].y) << 32) | __float_as_uint(hv[t][0].x));
          st_agent64(yu + 1, ((uint64_t)__float_as_uint(hv[t][0].w) << 32) | __float_as_uint(hv[t][0].z));
          st_agent64(yu + 2, ((uint64_t)__float_as_uint(hv[t][1].y) << 32) | __float_as_uint(hv[t][1].x));
          st_agent64(yu + 3, ((uint64_t)__float_as_uint(hv[t][1].w) << 32) | __float_as_uint(hv[t][1].z));
        }
      }
    }
  }
  __syncthreads();
  n_own = uniform(L.n_own);
  SI_TRACE_MARK(3);
  // decoder-block mode: x itself, needed only at gate/up, is scaled and
  // rounded from the registers while the group exchange is under way
  if constexpr (block_mode && kKeep) scale_x();

  bool census_done = false;
  if (tid < 2 * kMaxB) L.dmax[tid / kMaxB][tid % kMaxB] = 0u;
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
    // the census block's waves 4..7 meanwhile take the census: every block's
    // kept count (the call's count, and proof that every block has read the
    // call counter, which the census block then advances)
    if (tid < 4 * npairs) {
      const int p = tid >> 2;
      const int o = g * T + p / nsub, sb = p - (p / nsub) * nsub;
      const uint64_t* src[1] = {&a.pub[(size_t)o * kOwnPubStride + 4 * sb + (tid & 3)]};
      uint32_t v[1];
      poll_words<1>(src, 1, tag, a.hdr, v);
      L.pm[tid] = v[0];
    } else if (blk == cblk && tid >= kOT / 2) {
      const int sum = wave_sum_int(census_part(a.pub, P, tid - kOT / 2, kOT / 2, tag, a.hdr));
      if (lane == 0) L.wsum[wv] = sum;
    }
    __syncthreads();
    if (blk == cblk && tid == 0) {
      int sum = 0;
      for (int w = kOW / 2; w < kOW; ++w) sum += L.wsum[w];
      if (a.n_out) *a.n_out = sum;
      advance_epoch(a.hdr, epoch);
    }
    census_done = true;
    if (owns_tile && wv == kTileWave) {  // the tile's first stores have landed by now
      if constexpr (block_mode && BM == 1) {
        if (tunit < U) {
          uint64_t* yu = reinterpret_cast<uint64_t*>(a.y) + 4 * (size_t)tunit;
          st_agent64(yu, ((uint64_t)__float_as_uint(htile[0].y) << 32) | __float_as_uint(htile[0].x));
          st_agent64(yu + 1, ((uint64_t)__float_as_uint(htile[0].w) << 32) | __float_as_uint(htile[0].z));
          st_agent64(yu + 2, ((uint64_t)__float_as_uint(htile[1].y) << 32) | __float_as_uint(htile[1].x));
          st_agent64(yu + 3, ((uint64_t)__float_as_uint(htile[1].w) << 32) | __float_as_uint(htile[1].z));
        }
      }
      wait_own_stores();
      if (lane == 0) st_agent64(&a.zflag[blk], tagged(tag, 1u));
    }
    // the group's kept rows in order: every wave forms the prefix of the
    // pairs' kept counts (lane = pair), then one wave per pair writes its
    // rows' entries (lane = row)
    const int cnt = lane < npairs ? __popc(L.pm[4 * lane]) + __popc(L.pm[4 * lane + 1]) : 0;
    const int incl = wave_incl_scan(cnt);
    const int pre = incl - cnt;
    const int n = min(uniform(__builtin_amdgcn_readlane(incl, kWave - 1)), kMaxChunkRows);
    for (int p = wv; p < npairs; p += kOW) {
      const uint64_t kb = (uint64_t)L.pm[4 * p] | ((uint64_t)L.pm[4 * p + 1] << 32);
      const uint64_t cb = (uint64_t)L.pm[4 * p + 2] | ((uint64_t)L.pm[4 * p + 3] << 32);
      const int q0p = __builtin_amdgcn_readlane(pre, p);
      if ((kb >> lane) & 1ull) {
        const int o = g * T + p / nsub, sb = p - (p / nsub) * nsub;
        const uint32_t row = (uint32_t)(o * R + sb * kWave + lane);
        const int q = q0p + __popcll(kb & lanes_below(lane));
        if (q < kMaxChunkRows) L.dent[q] = row | (((cb >> lane) & 1ull) ? 0x80000000u : 0u);
      }
    }
    const int lo = (n * m) / T, hi = (n * (m + 1)) / T;  // this member's gate/up positions
    const int dN = n;                                     // the down item's positions
    if (tid == 0) {
      L.gpos = lo + kOW;
      L.dpos = 0;
      L.issued = 0;
      L.wsum[0] = 0;
      if constexpr (BM == 1 && kI8) L.wsum[1] = 0;  // waves done with their gate/up rows
    }
    __syncthreads();
    SI_TRACE_MARK(4);

    // ---- 2. gate/up: wave w takes position lo + w, then the next position
    // no wave has taken yet, and for each its W_gate row and (for confident rows, or without actual
    // sparsity) its W_up row at once; other rows read W_up only where some
    // token's ReLU output is positive.  Each wave works through its rows on
    // its own (no block barrier) and publishes h3 per row and token.
    int n_up = 0;
    // one token: a wave announces (LDS counter) that its first row's
    // requests are out, so that the waves without a row can queue their
    // W_down^T pieces behind them
    bool first = BM == 1;
    auto announce = [&]() {
      if constexpr (BM == 1) {
        if (first) {
          asm volatile("" ::: "memory");
          if (lane == 0) atomicAdd(&L.issued, 1);
          first = false;
        }
      }
    };
    for (int pos = lo + wv; pos < hi;) {
      const uint32_t e = L.dent[pos];
      const uint32_t row = e & 0x7fffffffu;
      float g[BM], u[BM];
      bool up;
      // with 4 or 8 tokens the per-lane unit addresses of the row loads and
      // token reads are formed again in every iteration (a few integer
      // operations) rather than kept live across the loop, where they were
      // spilled to scratch memory and read back in every iteration
      int ln = lane;
      if constexpr (BM >= 4) asm volatile("" : "+v"(ln));
      // a row's requests and their use sit in one branch (row-uniform)
      if constexpr (kI8) {
        // INT8 rows: U8 = d / 16 units of 16 values; scales read as the row's
        // requests go out, applied to the dot products
        constexpr int NU8 = (NU + 1) / 2;
        const int U8 = d >> 4;
        const uint32_t urow = uniform(row);
        if (gated && ((spec_ok && (e >> 31)) || no_as)) {
          u32x4 vg[NU8], vu[NU8];
          load_row<NU8>(a.wg + (size_t)urow * U8, U8, ln, vg);
          load_row<NU8>(a.wu + (size_t)urow * U8, U8, ln, vu);
          announce();
          const float sgv = a.sg[urow], suv = a.su[urow];
          row_dots_i8<BM, NU, true>(vg, vu, L.xs, U8, ln, g, u);
#pragma unroll
          for (int t = 0; t < BM; ++t) {
            g[t] *= sgv;
            u[t] *= suv;
          }
          up = true;
        } else {
          u32x4 vg[NU8];
          load_row<NU8>(a.wg + (size_t)urow * U8, U8, ln, vg);
          announce();
          const float sgv = a.sg[urow];
          row_dots_i8<BM, NU, false>(vg, vg, L.xs, U8, ln, g, u);
          bool any = false;
#pragma unroll
          for (int t = 0; t < BM; ++t) {
            g[t] *= sgv;
            any |= g[t] > 0.f;
          }
          up = gated && any;
          if (up) {
            u32x4 vu[NU8];
            load_row<NU8>(a.wu + (size_t)urow * U8, U8, ln, vu);
            if constexpr (BM >= 2) asm volatile("" ::: "memory");
            const float suv = a.su[urow];
            float unused[BM];
            row_dots_i8<BM, NU, false>(vu, vu, L.xs, U8, ln, u, unused);
#pragma unroll
            for (int t = 0; t < BM; ++t) u[t] *= suv;
          } else {
#pragma unroll
            for (int t = 0; t < BM; ++t) u[t] = gated ? 0.f : 1.f;
          }
        }
      } else if (gated && ((spec_ok && (e >> 31)) || no_as)) {
        u32x4 vg[NU], vu[NU];
        load_row<NU>(a.wg + (size_t)row * U, U, ln, vg);
        load_row<NU>(a.wu + (size_t)row * U, U, ln, vu);
        announce();
        SI_TRACE_WAVE(0);
        row_dots2<BM, NU>(vg, vu, L.xs, U, ln, g, u);
        up = true;
      } else {
        u32x4 vg[NU];
        load_row<NU>(a.wg + (size_t)row * U, U, ln, vg);
        announce();
        row_dots<BM, NU>(vg, L.xs, U, ln, g);
        bool any = false;
#pragma unroll
        for (int t = 0; t < BM; ++t) any |= g[t] > 0.f;
        up = gated && any;
        if (up) {
          u32x4 vu[NU];
          load_row<NU>(a.wu + (size_t)row * U, U, ln, vu);
          // the tokens are read from LDS again: kept from the gate products,
          // 2..8 tokens' units would not fit in registers and were spilled
          if constexpr (BM >= 2) asm volatile("" ::: "memory");
          row_dots<BM, NU>(vu, L.xs, U, ln, u);
        } else {  // h3 = ReLU(g) * 1 without W_up
#pragma unroll
          for (int t = 0; t < BM; ++t) u[t] = gated ? 0.f : 1.f;
        }
      }
      n_up += up ? 1 : 0;
      float hv = 0.f;  // lane t holds token t's h3
#pragma unroll
      for (int t = 0; t < BM; ++t) hv = lane == t ? fmaxf(g[t], 0.f) * u[t] : hv;
      if (lane < b) st_agent64(&a.h3e[(size_t)row * b + lane], tagged(tag, __float_as_uint(hv)));
      // the next free position of the member's range: the waves that the
      // CU serves first take more rows (with a fixed stride the second wave
      // of each SIMD finished its rows up to 10 us after the first); with at
      // most one position per wave there is none, and no wave waits for
      // the counter
      int nxt = hi;
      if (lo + kOW < hi) {
        if (lane == 0) nxt = atomicAdd(&L.gpos, 1);
        nxt = __builtin_amdgcn_readfirstlane(nxt);
      }
      pos = nxt;
    }
    SI_TRACE_WAVE(1);
    if constexpr (BM == 1 && kI8) {
      if (lane == 0 && lo + wv < hi) atomicAdd(&L.wsum[1], 1);
    }
    if (lane == 0 && n_up) atomicAdd(&L.n_up, n_up);
    SI_TRACE_MARK(6);
    SI_TRACE_WAVE(2);

    // ---- 3. down-projection of (tile, the group's rows): per round, wave w
    // takes positions q0 + w + 8 j (j < 8); it requests the tile's W_down^T
    // pieces of the confident ones, then polls their h3 words (lane = piece
    // x token; in the first round wave 0's last lane polls the tile's zero
    // flag in the same requests), fetches the non-confident pieces whose h3
    // is non-zero, and accumulates
    float acc[BM][8];
#pragma unroll
    for (int t = 0; t < BM; ++t)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[t][q] = 0.f;
    int n_down = 0;
    bool zok = false;
    const int dunit = tile * kWave + lane;
    const bool dcol_ok = dunit < U;
    constexpr bool kZLane = BM == 1 || kODN * BM < kWave;  // lane 63 of a wave's first round is free for the zero flag
    typedef DownPiece<kI8> DP;
    // with 2..8 tokens the rounds are pipelined: once round r's h3 words are
    // in (which also waits for its pieces), round r+1's pieces are requested
    // and round r's products (8 tokens x 8 columns per piece, the down
    // projection's arithmetic) run while they are in flight.  Every kept
    // row's pieces are requested (with several tokens a kept row almost
    // always has a non-zero h3; without speculation the rounds below run)
    bool pipelined = false;
    constexpr bool kMfma = BM >= 4;
    bool mdone = false;      // the down item ran on the matrix cores (its tile is in macc)
    float macc[4][4] = {};   // column block cb of the wave, D[4 g + i][token]: column 64 wv + 16 cb + 4 g + i
    if constexpr (kMfma) {
      if (spec_ok && dN > 0) {
        pipelined = true;
        mdone = true;
        MfmaLds<BM>& M = *reinterpret_cast<MfmaLds<BM>*>(L.mf_raw);
        const int nch = (dN + kMRows - 1) / kMRows;
        // chunks in flight: 4 with 5-8 tokens (the fused 8-token call 58.6 ->
        // 57.7 us), 3 with 3-4 (4 made the 4-token call 0.4 us slower)
        constexpr int kMI = BM >= 8 ? kMInflight + 1 : kMInflight;
        // pieces: the thread stages row 4 wv + lane / 16 of each chunk, its
        // 16-byte units lane % 16 + 16 j (j < 4) of the tile
        const int prow = 4 * wv + (lane >> 4), pslot = lane & 15;
        // h3 words: thread (row tid / BM, token tid % BM) for tid < 32 BM
        // (whole waves); the last wave reads the tile's zero flag with the
        // first chunk
        const int hrow = tid / BM, htok = tid - (tid / BM) * BM;
        const bool hwave = uniform(wv) < kMRows * BM / kWave;
        const bool zwave = uniform(wv) == kOW - 1;
        static_assert(kMRows * kMaxB / kWave < kOW, "the zero-flag wave reads no h3 words");
        const int tcu = tile * kWave;  // the tile's first 16-byte unit of a row
        typedef typename DP::type PT;
        auto request = [&](int c, PT(&pc)[4], uint64_t& w) {
          const int q = min(c * kMRows + prow, dN - 1);
          const size_t row = L.dent[q] & 0x7fffffffu;
#pragma unroll
          for (int j = 0; j < 4; ++j) pc[j] = DP::load(a.wdt, row, U, min(tcu + pslot + 16 * j, U - 1));
          // the first read of the chunk's h3 words goes out right behind its
          // pieces (a poll issued later would wait for every request before it)
          if (hwave) {
            const int hq = min(c * kMRows + hrow, dN - 1);
            w = ld_agent64(a.h3e + (size_t)(L.dent[hq] & 0x7fffffffu) * b + min(htok, b - 1));
          } else if (zwave && c == 0) {
            w = ld_agent64(&a.zflag[tile]);
          }
        };
        auto chunk = [&](int c, PT(&pc)[4], uint64_t& w) {
          float v = 0.f;
          if (hwave) {
            const int hq = c * kMRows + hrow;
            const bool ok = htok < b && hq < dN;
            uint32_t payload = (uint32_t)w;
            if (ok && (uint32_t)(w >> 32) != tag) {  // not published at the first read
              const uint64_t* src[1] = {a.h3e + (size_t)(L.dent[hq] & 0x7fffffffu) * b + htok};
              uint32_t o[1];
              poll_words<1>(src, 1, tag, a.hdr, o);
              payload = o[0];
            }
            v = ok ? __uint_as_float(payload) : 0.f;
            if (ok) atomicMax(&L.dmax[c & 1][htok], __float_as_uint(v) & 0x7fffffffu);
          } else if (zwave && c == 0) {
            zok = (uint32_t)(w >> 32) == tag && (uint32_t)w == 1u;
          }
          if (c == 0) SI_TRACE_WAVE(3);
          __syncthreads();  // (the first: every wave is past its gate/up, so x's LDS is free)
          unsigned char* rb = M.rows + prow * kMPitch;
#pragma unroll
          for (int j = 0; j < 4; ++j) *reinterpret_cast<u32x4*>(rb + (pslot + 16 * j) * 16) = DP::as_f16(pc[j]);
          if (hwave) {
            // scale 2^(se - 127): the token's largest |h3| of the chunk
            // lands in [2^14, 2^15), within fp16's range
            const int e8 = (int)(L.dmax[c & 1][htok] >> 23);
            const int se = min(268 - e8, 253);
            const float vs = v * __uint_as_float((uint32_t)se << 23);
            const _Float16 hi = (_Float16)vs;
            const _Float16 lo = (_Float16)(vs - (float)hi);
            M.bop[0][htok][hrow] = __builtin_bit_cast(uint16_t, hi);
            M.bop[1][htok][hrow] = __builtin_bit_cast(uint16_t, lo);
            if (hrow == 0) L.dinv[htok] = __uint_as_float((uint32_t)(254 - se) << 23);
          }
          if (tid < kMaxB) L.dmax[(c + 1) & 1][tid] = 0u;
          if (c == 0)  // tokens BM..15 of the B operand stay zero
            for (int i = tid; i < 2 * (kMTok - BM) * kMRows; i += kOT) {
              const int hlf = i / ((kMTok - BM) * kMRows), r = i - hlf * ((kMTok - BM) * kMRows);
              M.bop[hlf][BM + r / kMRows][r % kMRows] = 0;
            }
          if (c + kMI < nch) request(c + kMI, pc, w);
          __syncthreads();
          // lane (g = lane / 16, j16 = lane % 16): B = token j16's rows
          // 8 g .. 8 g + 7; A = those rows of column j16 of the block, from
          // two transposing reads (the 16 lanes of a group point at 4 rows x
          // 4 column quads; lane 4 p + q receives column 4 p + q of each row)
          const int g = lane >> 4, j16 = lane & 15;
          typedef _Float16 h8 __attribute__((ext_vector_type(8)));
          typedef _Float16 h4 __attribute__((ext_vector_type(4)));
          typedef float f4 __attribute__((ext_vector_type(4)));
          typedef short s4 __attribute__((ext_vector_type(4)));
          typedef __attribute__((address_space(3))) s4 lds_s4;
          const h8 bh = *reinterpret_cast<const h8*>(&M.bop[0][j16][8 * g]);
          const h8 bl = *reinterpret_cast<const h8*>(&M.bop[1][j16][8 * g]);
          const float inv = j16 < BM ? L.dinv[j16] : 0.f;
          const unsigned char* ab = M.rows + (8 * g + (j16 >> 2)) * kMPitch + (64 * wv + 4 * (j16 & 3)) * 2;
#pragma unroll
          for (int cb = 0; cb < 4; ++cb) {
            const h4 a0 = __builtin_bit_cast(h4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(ab + 32 * cb)));
            const h4 a1 =
                __builtin_bit_cast(h4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(ab + 32 * cb + 4 * kMPitch)));
            const h8 av = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
            f4 dv = {0.f, 0.f, 0.f, 0.f};
            dv = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bh, dv, 0, 0, 0);
            dv = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bl, dv, 0, 0, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i) macc[cb][i] = fmaf(dv[i], inv, macc[cb][i]);
          }
          if (c == 0) SI_TRACE_WAVE(4);
        };
        if constexpr (kMI == 4) {
          PT p0[4], p1[4], p2[4], p3[4];
          uint64_t w0 = 0, w1 = 0, w2 = 0, w3 = 0;
          request(0, p0, w0);
          if (1 < nch) request(1, p1, w1);
          if (2 < nch) request(2, p2, w2);
          if (3 < nch) request(3, p3, w3);
          for (int c = 0; c < nch; c += kMI) {
            chunk(c, p0, w0);
            if (c + 1 < nch) chunk(c + 1, p1, w1);
            if (c + 2 < nch) chunk(c + 2, p2, w2);
            if (c + 3 < nch) chunk(c + 3, p3, w3);
          }
        } else {
          PT p0[4], p1[4], p2[4];
          uint64_t w0 = 0, w1 = 0, w2 = 0;
          static_assert(kMI == 3, "three chunks in flight");
          request(0, p0, w0);
          if (1 < nch) request(1, p1, w1);
          if (2 < nch) request(2, p2, w2);
          for (int c = 0; c < nch; c += kMI) {
            chunk(c, p0, w0);
            if (c + 1 < nch) chunk(c + 1, p1, w1);
            if (c + 2 < nch) chunk(c + 2, p2, w2);
          }
        }
        n_down = wv == 0 ? dN : 0;
      }
    }
    if constexpr (BM >= 2 && !kMfma) {
      // a down item that one round of kODN pieces per wave does not cover but
      // one of 12 does takes that single round, all others pipelined rounds of
      // kODN (two tokens, the union of planted sets at s = 0.9, about 72
      // positions per group: 16.9 -> 15.9 us per 7B call; rounds of 12 for
      // every item made the longer items of the fused call and of s = 0.5
      // 0.6-1.5 us slower, and the shorter ones of s = 0.95-0.97 1 us slower)
      auto piped = [&](auto pn) {
        constexpr int kPN = decltype(pn)::value, kPRound = kOW * kPN;
        const int dcu = min(dunit, U - 1);  // column unit of the loads (in the row even past d)
        typename DP::type va[kPN], vb[kPN];
        auto request = [&](int q0, typename DP::type(&v)[kPN]) {
#pragma unroll
          for (int j = 0; j < kPN; ++j) {
            const int q = min(q0 + wv + kOW * j, dN - 1);
            v[j] = DP::load(a.wdt, L.dent[q] & 0x7fffffffu, U, dcu);
          }
        };
        auto round = [&](int q0, typename DP::type(&cur)[kPN], typename DP::type(&nxt)[kPN]) {
          const int pj = lane / BM, pt = lane - pj * BM;
          const int pq = q0 + wv + kOW * pj;
          const bool pok = pj < kPN && pq < dN && pt < b;
          const bool zlane = kZLane && q0 == 0 && wv == 0 && lane == kWave - 1;
          const uint64_t* src[1] = {zlane ? &a.zflag[tile]
                                          : a.h3e + (size_t)(L.dent[pok ? pq : q0] & 0x7fffffffu) * b + (pok ? pt : 0)};
          uint32_t hw[1];
          poll_words<1>(src, (pok || zlane) ? 1 : 0, tag, a.hdr, hw);
          if (q0 == 0 && wv == 0) zok = __builtin_amdgcn_readlane(hw[0], kWave - 1) == 1u && kZLane;
          if (q0 == 0) SI_TRACE_WAVE(3);
          if (q0 + kPRound < dN) request(q0 + kPRound, nxt);
#pragma unroll
          for (int j = 0; j < kPN; ++j) {
            const int q = q0 + wv + kOW * j;
            float hv[BM];
#pragma unroll
            for (int t = 0; t < BM; ++t)
              hv[t] = (j * BM + t < kWave && q < dN && t < b)
                          ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(hw[0], min(j * BM + t, kWave - 1)))
                          : 0.f;
            n_down += q < dN ? 1 : 0;
            float f[8];
            DP::values(cur[j], f);
#pragma unroll
            for (int t = 0; t < BM; ++t)
#pragma unroll
              for (int qq = 0; qq < 8; ++qq) acc[t][qq] = fmaf(hv[t], f[qq], acc[t][qq]);
          }
          if (q0 == 0) SI_TRACE_WAVE(4);
        };
        request(0, va);
        for (int q0 = 0; q0 < dN; q0 += 2 * kPRound) {
          round(q0, va, vb);
          if (q0 + kPRound < dN) round(q0 + kPRound, vb, va);
        }
      };
      if (spec_ok && dN > 0) {
        pipelined = true;
        if (dN > kOW * kODN && dN <= kOW * 12)
          piped(std::integral_constant<int, 12>{});
        else
          piped(std::integral_constant<int, kODN>{});
      }
    }
    // the unpipelined rounds, kDN pieces per wave and round (kODN, or with
    // one token kODN1 / kODN1Int8 / kODN1Wide).  With one token a wave takes
    // kDN consecutive positions at a time from an LDS counter; a wave without
    // a gate/up row starts at once, but only after the block's first gate/up
    // rows are requested (a CU's requests come back in order, and the pieces
    // must not delay them), and the waves with rows join in as they finish
    // them (with positions dealt w + 8 j the waves with a gate/up row
    // requested their pieces only after it, 0.35 us later per 7B call).
    // With more tokens wave w takes positions q0 + w + 8 j.
    auto down_rounds = [&](auto dn) {
      constexpr int kDN = decltype(dn)::value;
      static_assert(kDN * BM <= kWave, "a wave polls the h3 words of its pieces, one lane per (piece, token)");
      auto take = [&](int q0) -> int {
        if constexpr (BM == 1) {
          int v = 0;
          if (lane == 0) v = atomicAdd(&L.dpos, kDN);
          return __builtin_amdgcn_readfirstlane(v);
        } else {
          return q0 + kOW * kDN;
        }
      };
      if constexpr (BM == 1) {
        const int nwork = min(kOW, hi - lo);  // waves with a first gate/up row
        if (lo + wv >= hi && nwork > 0) {
          int spins = 0;  // an ordering aid only: the wait may give up
          while (__hip_atomic_load(&L.issued, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) < nwork &&
                 ++spins < 4096)
            __builtin_amdgcn_s_sleep(1);
        }
      }
      [[maybe_unused]] bool fb = true;  // the wave's first batch (phase-trace marks)
      for (int q0 = BM == 1 ? take(0) : 0; q0 < dN; q0 = take(q0)) {
        typename DP::type vd[kDN];
        uint32_t dl = 0;
#pragma unroll
        for (int j = 0; j < kDN; ++j) {
          vd[j] = typename DP::type{};
          const int q = BM == 1 ? q0 + j : q0 + wv + kOW * j;
          if (q < dN) {
            const uint32_t e = L.dent[q];
            if ((spec_ok && (e >> 31)) || no_as) {
              if (dcol_ok) vd[j] = DP::load(a.wdt, e & 0x7fffffffu, U, dunit);
              dl |= 1u << j;
            }
          }
        }
        // h3 of (piece j, token t) in lane j * BM + t
        const int pj = lane / BM, pt = lane - pj * BM;
        const int pq = BM == 1 ? q0 + pj : q0 + wv + kOW * pj;
        const bool pok = pj < kDN && pq < dN && pt < b;
        const bool zw = q0 == 0 && (BM == 1 || wv == 0);  // the wave that polls the tile's zero flag
        const bool zlane = kZLane && zw && lane == kWave - 1;
        const uint64_t* src[1] = {zlane ? &a.zflag[tile]
                                        : a.h3e + (size_t)(L.dent[pok ? pq : q0] & 0x7fffffffu) * b + (pok ? pt : 0)};
        uint32_t hw[1];
        if constexpr (BM == 1 && kI8) {
          // INT8 rows: a wave without gate/up rows polls its first batch's
          // h3 words once the block's own gate/up rows are done (the half-size
          // pieces are in long before the words are published, and a poll
          // that comes back without them costs a round trip: 11.72 -> 11.48
          // us per 7B call; with fp16 rows the pieces come in after the
          // words, and the same wait cost the non-gated and 13B-shaped calls
          // 0.1 us)
          if (fb && lo + wv >= hi) {
            const int nwork = min(kOW, hi - lo);
            int spins = 0;  // bounded: the wait only orders the poll
            while (__hip_atomic_load(&L.wsum[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) < nwork &&
                   ++spins < 65536)
              __builtin_amdgcn_s_sleep(1);
          }
        }
        poll_words<1>(src, (pok || zlane) ? 1 : 0, tag, a.hdr, hw);
        if (zw) zok = __builtin_amdgcn_readlane(hw[0], kWave - 1) == 1u && kZLane;
        if (fb) SI_TRACE_WAVE(3);
#pragma unroll
        for (int j = 0; j < kDN; ++j) {
          const int q = BM == 1 ? q0 + j : q0 + wv + kOW * j;
          float hv[BM];
          bool nz = false;
#pragma unroll
          for (int t = 0; t < BM; ++t) {
            hv[t] = (j * BM + t < kWave && q < dN && t < b)
                        ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(hw[0], min(j * BM + t, kWave - 1)))
                        : 0.f;
            nz |= hv[t] != 0.f;
          }
          if (q < dN && !((dl >> j) & 1u) && nz) {  // late request
            const uint32_t e = L.dent[q];
            if (dcol_ok) vd[j] = DP::load(a.wdt, e & 0x7fffffffu, U, dunit);
            dl |= 1u << j;
          }
          float f[8];
          DP::values(vd[j], f);
#pragma unroll
          for (int t = 0; t < BM; ++t)
#pragma unroll
            for (int qq = 0; qq < 8; ++qq) acc[t][qq] = fmaf(hv[t], f[qq], acc[t][qq]);
        }
        n_down += __popc(dl);
        if (fb) SI_TRACE_WAVE(4);
        fb = false;
      }
    };
    if (!pipelined) {
      if constexpr (BM == 1 && WIDE)
        down_rounds(std::integral_constant<int, kODN1Wide>{});
      else if constexpr (BM == 1)
        down_rounds(std::integral_constant<int, kI8 ? kODN1Int8 : kODN1>{});
      else
        down_rounds(std::integral_constant<int, kODN>{});
    }
    SI_TRACE_WAVE(5);
    if (lane == 0 && tile == 0 && n_down) atomicAdd(&L.n_down, n_down);
    if constexpr (BM == 1) {
      if (zok && lane == 0) L.wsum[0] = 1;  // the wave that took position 0 (the word starts at 0)
      if (dN > 0) {
        *reinterpret_cast<float4*>(&L.dpart1[wv][lane * 8]) = float4{acc[0][0], acc[0][1], acc[0][2], acc[0][3]};
        *reinterpret_cast<float4*>(&L.dpart1[wv][lane * 8 + 4]) = float4{acc[0][4], acc[0][5], acc[0][6], acc[0][7]};
      }
    } else {
      if (wv == (mdone ? kOW - 1 : 0) && lane == 0) L.wsum[0] = zok ? 1 : 0;
    }
    // per-wave partial tiles folded in LDS: with one token each wave has
    // stored its tile in a slot of its own (above, as its down batches
    // ended), so one barrier precedes the sum (three before, with the tiles
    // in the space of x: 7B 12.23 -> 12.14 us per call, INT8 11.60 -> 11.34,
    // decoder-block call 12.92 -> 12.79); with more tokens (plain stores in
    // the space of x, no longer needed) kFold waves store, the others add
    // in turn
    constexpr int kFold = OwnedLds<BM, NU>::kFold;
    __syncthreads();
    const bool zok_all = L.wsum[0] != 0;
    if (mdone) {
      // every wave is past its chunks: its columns of the tile go to LDS in
      // the fold's layout (token, column), so that the atomics below run
      // over consecutive columns (in the MFMA's layout one atomic
      // instruction would touch about 32 lines of y)
      const int n = lane & 15;
      if (n < BM) {
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
          *reinterpret_cast<float4*>(&L.dpart[0][n][64 * wv + 16 * cb + 4 * (lane >> 4)]) =
              float4{macc[cb][0], macc[cb][1], macc[cb][2], macc[cb][3]};
      }
    }
    if constexpr (BM > 1) {
      if (dN > 0 && !mdone) {
#pragma unroll
        for (int pass = 0; pass < kOW / kFold; ++pass) {
          if (wv / kFold == pass) {
            const int s2 = wv - pass * kFold;
#pragma unroll
            for (int t = 0; t < BM; ++t)
#pragma unroll
              for (int q = 0; q < 8; ++q) {
                float& dst = L.dpart[s2][t][lane * 8 + q];
                dst = pass == 0 ? acc[t][q] : dst + acc[t][q];
              }
          }
          __syncthreads();
        }
      }
    }
    SI_TRACE_MARK(8);

    // ---- the item's tile into y (its owner zeroed it in this call)
    if (dN > 0) {
      // (one token: only when the flag was not seen; zok_all is block-uniform,
      // read from LDS after the barrier above)
      if (BM > 1 || !zok_all) {
        if (tid == 0 && !zok_all) {  // after a timed-out poll, or when no lane was free for it
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
      }
      SI_TRACE_MARK(9);
      for (int i = tid; i < b * kTile; i += kOT) {
        const int t = i / kTile, c = i - t * kTile, col = tile * kTile + c;
        float v = 0.f;
#pragma unroll
        for (int s2 = 0; s2 < kFold; ++s2) {
          if constexpr (BM == 1)
            v += L.dpart1[s2][c];
          else
            v += (mdone && s2 > 0) ? 0.f : L.dpart[s2][t][c];
        }
        if constexpr (kI8) {
          if (col < d && v != 0.f) unsafeAtomicAdd(&a.y[(size_t)t * d + col], v * a.sd[col]);
        } else {
          if (col < d && v != 0.f) unsafeAtomicAdd(&a.y[(size_t)t * d + col], v);
        }
      }
    }
    if (tid == 0) {
      a.counts[2 * blk] = L.n_up;
      a.counts[2 * blk + 1] = L.n_down;
    }
  }
  if (blk == cblk && !census_done) {  // the predictor alone: the census at the end
    const int sum = block_sum(L, census_part(a.pub, P, tid, kOT, tag, a.hdr), lane, wv);
    if (tid == 0) {
      if (a.n_out) *a.n_out = sum;
      advance_epoch(a.hdr, epoch);
    }
  }

  // ---- the ascending kept list: the counts of the blocks before this one
  if (a.idx) {
    int sum = 0;
    for (int o = tid; o < blk; o += kOT) {
      const uint64_t* src[1] = {&a.pub[(size_t)o * kOwnPubStride + kCountWord]};
      uint32_t v[1];
      poll_words<1>(src, 1, tag, a.hdr, v);
      sum += (int)v[0];
    }
    const int before = block_sum(L, sum, lane, wv);
    for (int q = tid; q < n_own; q += kOT) a.idx[before + q] = (int32_t)(L.srow[q] & 0x7fffffffu);
  }
  if (a.mlp && blk == 0 && tid == 0) a.hdr[H_H3_FORM] = kH3ByRow;
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

// Grid of the row-owning kernel on the current device: one block per compute
// unit, or 0 if its LDS does not fit or one block cannot be resident per CU.
template <int BM, int NU, int MODE = kModePlain, bool WIDE = false>
static int owned_blocks() {
  static std::atomic<int> cache[kMaxDevices];
  return per_device_once(cache, [](int dev) -> int {
    constexpr int lds = owned_lds_bytes<BM, NU>();
    if constexpr (lds > kMaxLds) {
      return 0;
    } else {
      int cus = 0, per_cu = 0;
      const void* fn = reinterpret_cast<const void*>(&k_owned<BM, NU, MODE, WIDE>);
      if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
      if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess) return -1;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kOT, lds) != hipSuccess) return -1;
      return per_cu >= 1 ? (cus < kMaxLayerBlocks ? cus : kMaxLayerBlocks) : 0;
    }
  });
}

template <int BM, int NU>
static hipError_t owned_b(const LayerCall& c, hipStream_t s) {
  if constexpr (owned_lds_bytes<BM, NU>() > kMaxLds) {
    return hipErrorInvalidConfiguration;
  } else {
    const int k = c.k, d = c.d;
    const WsLayout L = ws_layout(k, c.b);
    char* base = static_cast<char*>(c.ws);
    const int mode = c.i8 ? kModeInt8 : c.h != nullptr ? kModeBlock : kModePlain;
    const int P = mode == kModeInt8    ? owned_blocks<BM, NU, kModeInt8>()
                  : mode == kModeBlock ? owned_blocks<BM, NU, kModeBlock>()
                                       : owned_blocks<BM, NU, kModePlain>();
    if (P < 1) return hipErrorInvalidConfiguration;
    OwnedArgs a;
    a.signs = reinterpret_cast<const u32x4*>(c.signs);
    a.wg = reinterpret_cast<const u32x4*>(c.w_gate);
    a.wu = reinterpret_cast<const u32x4*>(c.w_up);
    a.wdt = reinterpret_cast<const u32x4*>(c.w_down_t);
    a.sg = c.s_gate;
    a.su = c.s_up;
    a.sd = c.s_down;
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
    a.h = c.h;
    a.norm_w = c.norm_w;
    a.eps = c.eps;
    constexpr int lds = owned_lds_bytes<BM, NU>();
    bool launched = false;
    if constexpr (BM == 1) {
      // one token, groups of more than kWideGroupRows rows: the instance with
      // kODN1Wide pieces per down batch
      if (a.tiles * a.R > kWideGroupRows) {
        const int Pw = mode == kModeInt8    ? owned_blocks<1, NU, kModeInt8, true>()
                       : mode == kModeBlock ? owned_blocks<1, NU, kModeBlock, true>()
                                            : owned_blocks<1, NU, kModePlain, true>();
        if (Pw != P) return hipErrorInvalidConfiguration;
        if (mode == kModeInt8)
          k_owned<1, NU, kModeInt8, true><<<P, kOT, lds, s>>>(a);
        else if (mode == kModeBlock)
          k_owned<1, NU, kModeBlock, true><<<P, kOT, lds, s>>>(a);
        else
          k_owned<1, NU, kModePlain, true><<<P, kOT, lds, s>>>(a);
        launched = true;
      }
    }
    if (!launched) {
      if (mode == kModeInt8)
        k_owned<BM, NU, kModeInt8, false><<<P, kOT, lds, s>>>(a);
      else if (mode == kModeBlock)
        k_owned<BM, NU, kModeBlock, false><<<P, kOT, lds, s>>>(a);
      else
        k_owned<BM, NU, kModePlain, false><<<P, kOT, lds, s>>>(a);
    }
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
