// gspar: gradient sparsification (Wangni, Wang, Liu, Zhang; arXiv 1710.09854) for MI355X / gfx950.
//
// Pipeline per call (all launches on the caller's stream, no host synchronisation). Workgroups
// never wait on one another inside a histogram pass: every cross-workgroup hand-off is a kernel
// boundary, because device-scope fences are expensive on a multi-XCD part.
//   k_init     clears the per-call workspace and writes each row's budget B = rho*d (for a
//              segmented call, one row per segment, also the maps that give each workgroup of the
//              later passes its segment, so that only workgroups holding coordinates are launched).
//   k_stats    one streaming pass over g: an LDS histogram over binades of the magnitude bit pattern
//              (count, exact significand sum, max), added into per-row global copies.
//   k_solve    one workgroup per row: sums the copies and runs the solver (Proposition 1;
//              Algorithm 2's criterion with a density budget, or Algorithm 3), which either
//              finishes the row or asks for a refinement window.
//   k_refine   (launched a fixed number of times, each followed by k_solve; exits at once unless
//              the solver asked for it) histograms only the magnitudes inside one binade (4096
//              sub-bins with their minima, and a direct count of the keys at or above the greedy
//              query key) or inside one sub-bin (2048 single bit patterns), so every threshold the
//              solvers need is resolved exactly.
//   k_sample   one streaming pass: Philox4x32-10 per group of four coordinates, Bernoulli selection,
//              amplification to g_i or sign(g_i)/lambda, order-preserving compaction with a
//              decoupled look-back across tiles.
//   k_probs    (probabilities entry points) writes p_i = min(lambda |g_i|, 1); k_probs_out writes
//              the per-row results.
// Separately, k_aggregate averages M workers' sparse lists into one dense vector (Algorithm 1,
// step 6), summing each coordinate in fp64 in worker order.
//
// Sums of magnitudes are exact: a magnitude's bit pattern (its "key") fixes its binade, bins never
// straddle a binade, so per-bin sums of 24-bit significands are exact integers and are combined
// in a 320-bit fixed-point accumulator (unit 2^-149) that is rounded once to double. Hence lambda,
// the capped set and every decision are independent of the launch geometry and of atomic order.
#include <hip/hip_runtime.h>

#include <climits>
#include <algorithm>
#include <mutex>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <type_traits>

#include "gspar.h"
#ifdef GSPAR_INSTRUMENT
#include <hip/hip_ext.h>

#include "gspar_instr.h"
#endif

#define GS_HD __host__ __device__ __forceinline__

namespace gspar {

constexpr uint32_t kKeyInf = 0x7F800000u;   // bit pattern of +inf: keys >= this are non-finite
constexpr uint32_t kNone = 0xFFFFFFFFu;
constexpr int kNT = 512;                    // threads of the histogram / solver workgroups
constexpr int kLaneCopies = 8;              // LDS copies of the statistics histogram (by lane)
constexpr int kC1 = 4;                      // global copies of the level-1 histogram per row
constexpr int kC23 = 2;                     // global copies of the level-2 / level-3 histograms
constexpr int kB1 = 256;                    // level 1: one bin per binade (key >> 23)
constexpr int kB2 = 4096;                   // level 2: one binade, 2^11 keys per bin
constexpr int kB3 = 2048;                   // level 3: one level-2 bin, one key per bin
constexpr int kTileThreads = 256;
constexpr int kTileGroups = 16;             // float4 groups per thread per tile
constexpr int kTileElems = kTileThreads * kTileGroups * 4;  // 16384 coordinates per tile
// Sample tiles resident at once (256 CUs x 7); larger grids give each workgroup two tiles (a build
// may lower the threshold to exercise that path on small inputs).
#ifndef GSPAR_SAMPLE_RESIDENT
#define GSPAR_SAMPLE_RESIDENT (256 * 7)
#endif
constexpr int64_t kSampleResident = GSPAR_SAMPLE_RESIDENT;
constexpr int kMaxIters = 64;
constexpr int64_t kMaxChunk = (1 << 20) - 4;  // LDS packing holds < 2^20 elements per workgroup

enum : uint32_t { kFlagInternal = 16 };

// ------------------------------------------------------------------------------------------
// 320-bit fixed point, value = x * 2^-149 (the smallest subnormal float).
// ------------------------------------------------------------------------------------------
struct Fx {
  uint64_t w[5];
};

GS_HD Fx fx_zero() {
  Fx r;
  for (int i = 0; i < 5; ++i) r.w[i] = 0;
  return r;
}
GS_HD void fx_add(Fx& a, const Fx& b) {
  uint64_t c = 0;
  for (int i = 0; i < 5; ++i) {
    uint64_t s = a.w[i] + b.w[i];
    uint64_t c1 = s < a.w[i];
    uint64_t s2 = s + c;
    uint64_t c2 = s2 < s;
    a.w[i] = s2;
    c = c1 | c2;
  }
}
GS_HD Fx fx_sub(const Fx& a, const Fx& b) {  // requires a >= b
  Fx r;
  uint64_t br = 0;
  for (int i = 0; i < 5; ++i) {
    uint64_t d1 = a.w[i] - b.w[i];
    uint64_t b1 = a.w[i] < b.w[i];
    uint64_t d2 = d1 - br;
    uint64_t b2 = d1 < br;
    r.w[i] = d2;
    br = b1 | b2;
  }
  return r;
}
// Limb i of a, with i in [0, 5) known only at run time; written as selects so the accumulator
// stays in registers (no dynamically indexed private array).
GS_HD uint64_t fx_limb(const Fx& a, int i) {
  uint64_t r = 0;
#pragma unroll
  for (int j = 0; j < 5; ++j) r = (j == i) ? a.w[j] : r;
  return r;
}
// v * 2^s for s in [0, 255] (every v < 2^64 then fits). A shift outside that range breaks an
// invariant of the callers (a binade index outside [0, 255]): it sets kFlagInternal in *err and
// gives 0, so the row is reported instead of being solved with a wrong sum.
GS_HD Fx fx_shifted(uint64_t v, int s, uint32_t* err) {
  if ((unsigned)s > 255u) {
    *err |= kFlagInternal;
    return fx_zero();
  }
  const int li = s >> 6, off = s & 63;
  const uint64_t lo = v << off;
  const uint64_t hi = off ? (v >> (64 - off)) : 0;
  Fx r;
#pragma unroll
  for (int j = 0; j < 5; ++j) r.w[j] = (j == li) ? lo : ((j == li + 1) ? hi : 0);
  return r;
}
GS_HD bool fx_bit(const Fx& a, int k) { return (fx_limb(a, k >> 6) >> (k & 63)) & 1; }
GS_HD bool fx_any_below(const Fx& a, int k) {  // any set bit at positions [0, k)
  if (k <= 0) return false;
  const int li = k >> 6, off = k & 63;
  bool any = false;
#pragma unroll
  for (int j = 0; j < 5; ++j) {
    const uint64_t m = j < li ? ~0ull : ((j == li && off) ? ((1ull << off) - 1) : 0ull);
    any = any || (a.w[j] & m) != 0;
  }
  return any;
}
// Round to the nearest double, ties to even.
GS_HD double fx_to_double(const Fx& a) {
  int top = -1;
#pragma unroll
  for (int i = 0; i < 5; ++i)
    if (a.w[i]) top = i * 64 + 63 - __builtin_clzll(a.w[i]);
  if (top < 0) return 0.0;
  if (top < 53) return ldexp((double)a.w[0], -149);
  const int lo = top - 52;
  const int li = lo >> 6, off = lo & 63;
  uint64_t m = fx_limb(a, li) >> off;
  if (off) m |= fx_limb(a, li + 1) << (64 - off);
  m &= (1ull << 53) - 1;
  const bool rnd = fx_bit(a, lo - 1);
  const bool sticky = fx_any_below(a, lo - 1);
  if (rnd && (sticky || (m & 1))) m += 1;
  return ldexp((double)m, lo - 149);
}

// ------------------------------------------------------------------------------------------
// 640-bit fixed point, value = x * 2^-298 (the square of the smallest subnormal float): exact sums
// of squared magnitudes for the variance-budget solver.
// ------------------------------------------------------------------------------------------
constexpr int kQ = 10;
struct Fq {
  uint64_t w[kQ];
};

GS_HD Fq fq_zero() {
  Fq r;
  for (int i = 0; i < kQ; ++i) r.w[i] = 0;
  return r;
}
GS_HD void fq_add(Fq& a, const Fq& b) {
  uint64_t c = 0;
  for (int i = 0; i < kQ; ++i) {
    uint64_t s = a.w[i] + b.w[i];
    uint64_t c1 = s < a.w[i];
    uint64_t s2 = s + c;
    uint64_t c2 = s2 < s;
    a.w[i] = s2;
    c = c1 | c2;
  }
}
GS_HD Fq fq_sub(const Fq& a, const Fq& b) {  // requires a >= b
  Fq r;
  uint64_t br = 0;
  for (int i = 0; i < kQ; ++i) {
    uint64_t d1 = a.w[i] - b.w[i];
    uint64_t b1 = a.w[i] < b.w[i];
    uint64_t d2 = d1 - br;
    uint64_t b2 = d1 < br;
    r.w[i] = d2;
    br = b1 | b2;
  }
  return r;
}
GS_HD uint64_t fq_limb(const Fq& a, int i) {
  uint64_t r = 0;
#pragma unroll
  for (int j = 0; j < kQ; ++j) r = (j == i) ? a.w[j] : r;
  return r;
}
// Squared significands summed per bin as qh * 2^24 + ql (each square m^2 < 2^48 split at bit 24;
// qh, ql < 2^55 for at most 2^31 values), times 2^(2 shift): the bin's exact sum of squares. The
// sum is below 2^80, so 2 shift in [0, 511] keeps it inside the 640 bits; any other shift sets
// kFlagInternal in *err and gives 0, like fx_shifted.
GS_HD Fq fq_squares(uint64_t qh, uint64_t ql, int shift, uint32_t* err) {
  const int sh = 2 * shift;
  if ((unsigned)sh > 511u) {
    *err |= kFlagInternal;
    return fq_zero();
  }
  const uint64_t lo0 = qh << 24;
  const uint64_t lo = lo0 + ql;
  const uint64_t hi = (qh >> 40) + (lo < lo0 ? 1 : 0);
  const int li = sh >> 6, off = sh & 63;
  const uint64_t w0 = lo << off;
  const uint64_t w1 = off ? ((lo >> (64 - off)) | (hi << off)) : hi;
  const uint64_t w2 = off ? (hi >> (64 - off)) : 0;
  Fq r;
#pragma unroll
  for (int j = 0; j < kQ; ++j) r.w[j] = j == li ? w0 : (j == li + 1 ? w1 : (j == li + 2 ? w2 : 0));
  return r;
}
GS_HD bool fq_bit(const Fq& a, int k) { return (fq_limb(a, k >> 6) >> (k & 63)) & 1; }
GS_HD bool fq_any_below(const Fq& a, int k) {
  if (k <= 0) return false;
  const int li = k >> 6, off = k & 63;
  bool any = false;
#pragma unroll
  for (int j = 0; j < kQ; ++j) {
    const uint64_t m = j < li ? ~0ull : ((j == li && off) ? ((1ull << off) - 1) : 0ull);
    any = any || (a.w[j] & m) != 0;
  }
  return any;
}
// Round to the nearest double, ties to even.
GS_HD double fq_to_double(const Fq& a) {
  int top = -1;
#pragma unroll
  for (int i = 0; i < kQ; ++i)
    if (a.w[i]) top = i * 64 + 63 - __builtin_clzll(a.w[i]);
  if (top < 0) return 0.0;
  if (top < 53) return ldexp((double)a.w[0], -298);
  const int lo = top - 52;
  const int li = lo >> 6, off = lo & 63;
  uint64_t m = fq_limb(a, li) >> off;
  if (off) m |= fq_limb(a, li + 1) << (64 - off);
  m &= (1ull << 53) - 1;
  const bool rnd = fq_bit(a, lo - 1);
  const bool sticky = fq_any_below(a, lo - 1);
  if (rnd && (sticky || (m & 1))) m += 1;
  return ldexp((double)m, lo - 298);
}

// ------------------------------------------------------------------------------------------
// Magnitude keys.
// ------------------------------------------------------------------------------------------
GS_HD uint32_t key_of(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  return u & 0x7FFFFFFFu;
}
GS_HD double key_value(uint32_t k) {
  float f;
  memcpy(&f, &k, 4);
  return (double)f;
}
GS_HD uint64_t key_sig(uint32_t key) {  // integer significand: value = sig * 2^(max(e,1) - 150)
  uint32_t e = key >> 23, m = key & 0x7FFFFFu;
  return e ? (uint64_t)(m | 0x800000u) : (uint64_t)m;
}
GS_HD int binade_shift(int e) { return (e > 0 ? e : 1) - 1; }  // in units of 2^-149

// Smallest key t with fl(lambda * value(t)) >= 1, i.e. capped <=> key >= t for p = min(lambda a, 1).
// kKeyInf when no finite magnitude is capped.
GS_HD uint32_t cap_key(double lam) {
  if (!(lam > 0.0)) return kKeyInf;
  if (lam == INFINITY) return 1;
  double x = 1.0 / lam;
  uint32_t k;
  if (x >= 3.4028234663852886e38) {
    k = kKeyInf;
  } else {
    k = key_of((float)x);
    if (k == 0) k = 1;
  }
  for (int it = 0; it < 4 && k > 1 && lam * key_value(k - 1) >= 1.0; ++it) --k;
  for (int it = 0; it < 4 && k < kKeyInf && !(lam * key_value(k) >= 1.0); ++it) ++k;
  return k;
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two 32x32->64 products on
// counter words 0 and 2, high halves crossed with words 1, 3 and the round key; the key advances
// by the golden-ratio and sqrt(3)-1 Weyl increments after each round.
// a ^ b ^ c (one three-input bitwise instruction on gfx950)
GS_HD uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
#else
  return a ^ b ^ c;
#endif
}

GS_HD void philox10(uint32_t& c0, uint32_t& c1, uint32_t& c2, uint32_t& c3, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    uint64_t m0 = (uint64_t)c0 * 0xD2511F53u;
    uint64_t m1 = (uint64_t)c2 * 0xCD9E8D57u;
    uint32_t x0 = xor3((uint32_t)(m1 >> 32), c1, k0);
    uint32_t x2 = xor3((uint32_t)(m0 >> 32), c3, k1);
    c1 = (uint32_t)m1;
    c3 = (uint32_t)m0;
    c0 = x0;
    c2 = x2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
}

// ------------------------------------------------------------------------------------------
// Workspace.
// ------------------------------------------------------------------------------------------
struct alignas(256) RowCtl {
  double B;          // rho * d
  double lam;        // greedy: current lambda; final: lambda of Proposition 1
  Fx S;              // exact sum of |g|
  Fx fbW;            // exact solver: capped sum of the best candidate found so far
  uint64_t fbK;      // exact solver: capped count of that candidate
  uint64_t zeros;    // zero entries of the row (d minus the histogram's population)
  uint64_t wK;       // exact solver, level 3: count of keys above the window
  Fx wW;             // and their exact sum
  float inv_lam;     // fl32(1/lambda): the amplified value off the capped set
  uint32_t fbTcap;   // exact solver: candidate's capped threshold key
  uint32_t fbValid;
  uint32_t tcap;     // final: coordinate capped (p = 1) iff key >= tcap
  uint32_t flags;
  uint32_t need;     // 0: none; 2 / 3: a level-2 / level-3 pass is requested
  uint32_t done;     // 1 once lambda and tcap are final
  uint32_t qkey;     // greedy: key whose count and sum above the level-2 pass also counts directly
  uint32_t src;      // 1: the requested window lies in the candidate band, its pass reads the candidates
  uint32_t l2exp;    // binade of the level-2 window (kNone: none)
  uint32_t l3base;   // first key of the level-3 window (kNone: none)
  int32_t iter;      // greedy rescale steps taken
  int32_t stage;     // 0 before the first solve; exact solver: next level to examine
  int32_t solver;
  int32_t T;
  uint32_t band_lo;  // candidate band [band_lo, band_hi) of keys (whole binades) the statistics pass
  uint32_t band_hi;  // collected, written by its first workgroup (equal bounds: no band)
  uint64_t cand_n;   // candidates collected (first solve; above the capacity: incomplete, unused)
  uint32_t qonly;    // greedy, last rescale step: the level-2 pass only counts the keys >= qkey
};
static_assert(sizeof(RowCtl) == 256, "RowCtl layout");
// offsets read by the tests to see which source a refinement pass used
static_assert(offsetof(RowCtl, src) == 192 && offsetof(RowCtl, band_lo) == 220 && offsetof(RowCtl, band_hi) == 224 &&
                  offsetof(RowCtl, cand_n) == 232,
              "RowCtl offsets known to the tests");

struct Hist1 {
  uint64_t cnt[kB1];
  uint64_t sig[kB1];
  uint32_t mx[kB1];
};
// Histogram of one refinement window: a level-2 window uses all kB2 bins (one binade, 2^11 keys per
// bin), a level-3 window the first kB3 (one key per bin).
struct alignas(256) WinHist {
  uint64_t cnt[kB2];
  uint64_t sig[kB2];
  uint32_t mx[kB2];
  uint32_t mnc[kB2];  // level 2: bitwise complement of the bin's minimum key (0: empty), so max-combined
  uint64_t qcnt;      // level 2: count of window keys >= the row's qkey
  uint64_t qsig;      // their significand sum
};

// The level-1 histogram summed over its copies, with per binade the count K and exact sum W of all
// keys in the binades above it.
struct alignas(16) L1Cache {
  uint64_t cnt[kB1];
  uint64_t sig[kB1];
  uint32_t mx[kB1];
  uint64_t K[kB1];
  Fx W[kB1];
};
static_assert(sizeof(L1Cache) % 16 == 0, "L1Cache is copied in 16-byte units");
// Variance-budget solver: per-bin sums of squared significands (see fq_squares) of the level-1
// histogram copies and of the level-2 window copies, and per row the exact total of squares and
// the square sums that go with the solver's stored counts and sums (above the requested window,
// and of the fallback candidate).
struct H1Q {
  uint64_t qh[kB1];
  uint64_t ql[kB1];
};
struct alignas(256) WinQ {
  uint64_t qh[kB2];
  uint64_t ql[kB2];
};
struct alignas(256) VarCtl {
  Fq A2;   // sum of a^2 over the row
  Fq wH;   // square sum above the requested window
  Fq fbH;  // square sum of the fallback candidate's capped set
};

// Per-row partial count of capped coordinates written by the probabilities pass, one per class.
struct alignas(128) CountLine {
  unsigned long long v;
  unsigned long long pad[15];
};

// Per-row histogram over binades of a systematic sample of the row (count and significand sum),
// from which every statistics workgroup predicts the band of keys the solvers will refine.
struct PreHist {
  uint64_t cnt[kB1];
  uint64_t sig[kB1];
};

GS_HD size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Layout {
  size_t ctl, h1, l1t, win, kc, status, bmap, tmap, h1q, winq, vctl, pre, ccnt, cand, total;
  int64_t tiles;     // tiles per row of the sample pass
  int64_t cand_cap;  // candidate keys per row (0: no candidate band)
};

constexpr int64_t kMinChunk = 8192;  // fewest coordinates per histogram workgroup (but the row's)

// Candidate band: rows of at least kCandMinRow coordinates predict, from a sample of the row, the
// binades holding every threshold the solvers will refine, and the statistics pass copies the keys
// inside them to a per-row buffer, so refinement passes read those keys instead of the row. The
// sample costs a launch (about 5 us) and the collection a few per cent of the statistics pass, a
// loss on rows whose passes over the row take about as long or that need no window at all, so
// only rows of 2^25 coordinates and more take the band (a build may lower the threshold to
// exercise the band on small inputs).
#ifndef GSPAR_CAND_MIN_ROW
#define GSPAR_CAND_MIN_ROW (1 << 25)
#endif
constexpr int64_t kCandMinRow = GSPAR_CAND_MIN_ROW;
static_assert(kCandMinRow >= 1024, "a row must hold at least 64 whole lines to be sampled");
constexpr int kPreWG = 64;              // sample workgroups per row
#ifndef GSPAR_PRE_LINES
#define GSPAR_PRE_LINES 256
#endif
constexpr int kPreLines = GSPAR_PRE_LINES;  // 64-byte lines sampled per workgroup (16384 per row)
// Lines of a row of length len that the sample reads: every line when the row has fewer.
GS_HD int64_t pre_lines(int64_t len) {
  const int64_t nl = len / 16, ns = (int64_t)kPreWG * kPreLines;
  return nl < ns ? nl : ns;
}
// Refinement over candidates: at least kCandShare keys per workgroup and at most kCandGroups
// workgroups per row (each workgroup adds its whole window into the global copies, so fewer,
// fuller workgroups cost fewer global atomics), read kCandLoads float4 per thread at a time.
constexpr int64_t kCandShare = 1 << 14;
constexpr int64_t kCandGroups = 128;
constexpr int kCandLoads = 8;
// keys a lane buffers in LDS before its wave flushes (an odd stride keeps the lanes on different
// banks); sized so that the statistics workgroup stays within a quarter of the LDS (four resident
// per compute unit)
constexpr int kCandLane = 7;
// Candidate capacity per row a full workspace provides.
GS_HD int64_t cand_cap_full(int64_t d) {
  if (d < kCandMinRow) return 0;
  int64_t c = d / 16;
  if (c < ((int64_t)1 << 20)) c = (int64_t)1 << 20;
  return (c < d ? c : d) & ~(int64_t)63;  // whole 256-byte blocks
}

// Histogram copies: row r's copy c of level 1 is h1 + (r * kC1 + c), of a refinement window
// win + (r * kC23 + c); the solve that requests a refinement pass clears the window's copies.
// cand_cap: candidate keys per row (the workspace ends with the candidate buffers, so a smaller
// capacity changes no other offset).
GS_HD Layout layout_of(int64_t rows, int64_t d, int64_t cand_cap) {
  Layout L;
  L.tiles = (d + kTileElems - 1) / kTileElems;
  size_t off = 256;  // header (reserved)
  L.ctl = off;
  off += align256((size_t)rows * sizeof(RowCtl));
  L.h1 = off;
  off += align256((size_t)rows * kC1 * sizeof(Hist1));
  L.l1t = off;
  off += align256((size_t)rows * sizeof(L1Cache));
  L.win = off;
  off += align256((size_t)rows * kC23 * sizeof(WinHist));
  L.kc = off;
  off += align256((size_t)rows * 8 * sizeof(CountLine));
  L.status = off;
  off += align256((size_t)rows * (size_t)L.tiles * sizeof(uint64_t));
  // segmented calls: workgroup -> (row, block) of the histogram passes and (row, first tile) of the
  // sample pass, for the workgroups that hold coordinates only
  L.bmap = off;
  off += align256((size_t)rows * (size_t)((d + kMinChunk - 1) / kMinChunk) * sizeof(uint64_t));
  L.tmap = off;
  off += align256((size_t)rows * (size_t)L.tiles * sizeof(uint64_t));
  // variance-budget solver only
  L.h1q = off;
  off += align256((size_t)rows * kC1 * sizeof(H1Q));
  L.winq = off;
  off += align256((size_t)rows * kC23 * sizeof(WinQ));
  L.vctl = off;
  off += align256((size_t)rows * sizeof(VarCtl));
  // candidate band
  L.pre = off;
  off += align256((size_t)rows * sizeof(PreHist));
  L.ccnt = off;  // per row: keys collected (reserved in the compact list)
  off += align256((size_t)rows * sizeof(CountLine));
  L.cand = off;  // per row: the compact candidate list, then the statistics workgroups' regions
  L.cand_cap = cand_cap;
  off += align256((size_t)rows * (size_t)cand_cap * 2 * sizeof(uint32_t));
  L.total = off;
  return L;
}

struct Args {
  const float* g;
  int64_t rows, d, ld;
  const double* rho_dev;  // per-row densities, or nullptr to use `rho`
  double rho;
  const uint64_t* seed_dev;
  uint64_t seed;
  int solver, T;
  char* ws;
  Layout lay;
  int nb;          // workgroups per row of the histogram passes
  int64_t chunk;   // elements per histogram workgroup (multiple of 4)
  int first;       // k_solve: the solve right after the statistics pass
  int32_t* idx;    // compaction: every survivor; hybrid coding: Q_A, the capped survivors
  float* val;
  int64_t cap;
  int64_t* nnz;
  int32_t* code_b;  // hybrid coding: Q_B, index | sign << 31 of every other survivor
  int64_t cap_b;
  int64_t* nnz_b;
  float* inv_out;   // hybrid coding: fp32 1/lambda per row
  int8_t* q;        // hybrid coding: optional dense ternary vector, leading dimension ld
  double* lam_out;
  int64_t* k_out;
  uint32_t* flags_out;
  float* p;
  // segmented calls: row r is g[seg[r], seg[r + 1]) (device offsets), d the longest segment
  const int64_t* seg;
  int64_t seg_total;  // the host's last offset: no segment may end beyond it
  int64_t seg_elems;  // the host's total segment length
  int64_t seg_chunk;  // host: histogram-pass chunk chosen from the segment lengths
  int64_t seg_tiles;  // host: sample tiles that hold coordinates, over all segments
  int64_t seg_blocks; // histogram-pass workgroups (the grid), from the host offsets
  int64_t seg_wgs;    // sample-pass workgroups (the grid), from the host offsets
  int seg_k;          // tiles per sample workgroup
  int seg_align;      // vector loads in use: every segment must start at a multiple of 4
  size_t ws_bytes;    // the workspace's size (the candidate buffers take what the rest leaves)
  int64_t cand_region;  // candidate keys per statistics workgroup (cand_cap / nb, a multiple of 64)
};

// Start and length of row r: row r of a strided batch (offset r * ld, length d), or segment r of a
// segmented call. A segment whose device offsets break the bounds the host checked (order, end,
// length, alignment of the vector path) reads as empty and returns false.
__device__ __forceinline__ bool row_span(const Args& a, int64_t r, int64_t& base, int64_t& len) {
  if (!a.seg) {
    base = r * a.ld;
    len = a.d;
    return true;
  }
  const int64_t b = a.seg[r], e = a.seg[r + 1];
  const bool ok = b >= 0 && e >= b && e <= a.seg_total && e - b <= a.d && (!a.seg_align || (b & 3) == 0);
  base = ok ? b : 0;
  len = ok ? e - b : 0;
  return ok;
}

// Segmented calls: the word k_init leaves in the workspace header, 1 when the workgroup maps built
// from the device offsets have exactly the host's shape (the launched grids), 2 when they do not
// (every segment is then flagged GSPAR_FLAG_BADSEG and skipped).
__device__ __forceinline__ uint32_t* segok_of(const Args& a) { return reinterpret_cast<uint32_t*>(a.ws); }

__device__ __forceinline__ RowCtl* ctl_of(const Args& a, int64_t r) {
  return reinterpret_cast<RowCtl*>(a.ws + a.lay.ctl) + r;
}
__device__ __forceinline__ Hist1* h1_of(const Args& a, int64_t r, int c = 0) {
  return reinterpret_cast<Hist1*>(a.ws + a.lay.h1) + r * kC1 + c;
}
__device__ __forceinline__ L1Cache* l1t_of(const Args& a, int64_t r) {
  return reinterpret_cast<L1Cache*>(a.ws + a.lay.l1t) + r;
}
__device__ __forceinline__ WinHist* win_of(const Args& a, int64_t r, int c = 0) {
  return reinterpret_cast<WinHist*>(a.ws + a.lay.win) + r * kC23 + c;
}

__device__ __forceinline__ H1Q* h1q_of(const Args& a, int64_t r, int c = 0) {
  return reinterpret_cast<H1Q*>(a.ws + a.lay.h1q) + r * kC1 + c;
}
__device__ __forceinline__ WinQ* winq_of(const Args& a, int64_t r, int c = 0) {
  return reinterpret_cast<WinQ*>(a.ws + a.lay.winq) + r * kC23 + c;
}
__device__ __forceinline__ VarCtl* vctl_of(const Args& a, int64_t r) {
  return reinterpret_cast<VarCtl*>(a.ws + a.lay.vctl) + r;
}

__device__ __forceinline__ CountLine* kc_of(const Args& a, int64_t r) {
  return reinterpret_cast<CountLine*>(a.ws + a.lay.kc) + r * 8;
}
__device__ __forceinline__ uint64_t* status_of(const Args& a) {
  return reinterpret_cast<uint64_t*>(a.ws + a.lay.status);
}
__device__ __forceinline__ PreHist* pre_of(const Args& a, int64_t r) {
  return reinterpret_cast<PreHist*>(a.ws + a.lay.pre) + r;
}
// Candidates of row r: the compact list (cand_cap keys), then the staging regions, where statistics
// workgroup b collects into keys [b * cand_region, (b + 1) * cand_region) before moving them to
// the list; the row's count line holds the keys reserved in the list.
__device__ __forceinline__ CountLine* ccnt_of(const Args& a, int64_t r) {
  return reinterpret_cast<CountLine*>(a.ws + a.lay.ccnt) + r;
}
__device__ __forceinline__ uint32_t* cand_of(const Args& a, int64_t r) {
  return reinterpret_cast<uint32_t*>(a.ws + a.lay.cand) + r * a.lay.cand_cap * 2;
}
__device__ __forceinline__ uint32_t* creg_of(const Args& a, int64_t r) { return cand_of(a, r) + a.lay.cand_cap; }



// Four consecutive coordinates 4q..4q+3 of a row; entries at or beyond `end` read as 0 and are
// flagged invalid in the returned mask (bit c set = coordinate 4q+c exists).
template <bool VEC>
__device__ __forceinline__ uint32_t load4(const float* __restrict__ row, int64_t q, int64_t end, float v[4]) {
  int64_t i = 4 * q;
  if (VEC && i + 3 < end) {
    float4 x = *reinterpret_cast<const float4*>(row + i);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
    return 0xF;
  }
  uint32_t m = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    bool ok = i + c < end;
    v[c] = ok ? row[i + c] : 0.0f;
    m |= (uint32_t)ok << c;
  }
  return m;
}

// Streaming accesses: g is read once per pass and the outputs are written once, so those loads,
// the probabilities' stores and the compaction's staged stores (whole runs of consecutive words)
// carry the non-temporal hint and do not displace what the caches keep (the level-1 copies,
// windows and status words). Stores that lanes make one word at a time to scattered places (the
// other emission paths, the hybrid coding's lists, the candidate band) keep the default policy:
// there the hint made the hybrid coding's sampling pass a third slower at rho = 0.1. On 2^28
// coordinates the hint takes the statistics pass from about 213 to 192 microseconds per call.
#if defined(__HIP_DEVICE_COMPILE__)
typedef float gs_f4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 load_stream(const float* p) {
  const gs_f4v v = __builtin_nontemporal_load(reinterpret_cast<const gs_f4v*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void store_stream(float* p, float4 x) {
  const gs_f4v v = {x.x, x.y, x.z, x.w};
  __builtin_nontemporal_store(v, reinterpret_cast<gs_f4v*>(p));
}
#define GS_STORE_STREAM(ptr, v) __builtin_nontemporal_store((v), (ptr))
#else
GS_HD float4 load_stream(const float* p) { return *reinterpret_cast<const float4*>(p); }
GS_HD void store_stream(float* p, float4 x) { *reinterpret_cast<float4*>(p) = x; }
#define GS_STORE_STREAM(ptr, v) (*(ptr) = (v))
#endif

// Visits the coordinates [beg, end) of one row (beg a multiple of 4) with the NT threads of a
// workgroup, calling f(q, v, m) for each float4 group q (m: bit c set when coordinate 4q+c exists).
// With vector loads, blocks of U groups per thread are loaded unconditionally, all issued before
// any group is processed, so U loads per thread stay in flight; the last block clamps its addresses
// to the last whole group and masks the values, and a trailing partial group is loaded by one
// thread with scalar loads and visited by the whole first wave. No memory access sits under a
// divergent branch, which would make the compiler wait for every outstanding load. With vector
// loads every call of f is made by whole waves, so f may use cross-lane operations.
template <bool VEC, int U, int NT, typename F>
__device__ __forceinline__ void stream_groups(const float* __restrict__ row, int64_t beg, int64_t end, F&& f) {
  if (!VEC) {
    for (int64_t q = beg / 4 + threadIdx.x; 4 * q < end; q += NT) {
      float v[4];
      const uint32_t m = load4<false>(row, q, end, v);
      f(q, v, m);
    }
    return;
  }
  const int64_t qfull = end / 4;  // groups [beg/4, qfull) lie entirely inside [beg, end)
  int64_t qb = beg / 4;
  for (; qb + (int64_t)U * NT <= qfull; qb += (int64_t)U * NT) {
    float4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = load_stream(row + 4 * (qb + threadIdx.x + u * NT));
    __builtin_amdgcn_sched_barrier(0);  // keep every load of the block ahead of the first use
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float v[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
      f(qb + threadIdx.x + u * NT, v, 0xFu);
    }
  }
  if (qb < qfull) {
    float4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t q = qb + threadIdx.x + u * NT;
      x[u] = *reinterpret_cast<const float4*>(row + 4 * (q < qfull ? q : qfull - 1));
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t q = qb + threadIdx.x + u * NT;
      const bool ok = q < qfull;
      float v[4] = {ok ? x[u].x : 0.0f, ok ? x[u].y : 0.0f, ok ? x[u].z : 0.0f, ok ? x[u].w : 0.0f};
      f(q, v, ok ? 0xFu : 0u);
    }
  }
  if (4 * qfull < end && threadIdx.x < 64) {
    // the last, partial group: visited by the whole first wave (its other lanes see no
    // coordinates), so a visitor may use cross-lane operations
    float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    uint32_t m = 0;
    if (threadIdx.x == 0) m = load4<false>(row, qfull, end, v);
    f(qfull, v, m);
  }
}

// ------------------------------------------------------------------------------------------
// The per-row solver, run by one workgroup of kNT threads per row (k_solve). Every helper is
// force-inlined so LDS and global pointers keep their address spaces and no call frames or scratch
// are needed.
// ------------------------------------------------------------------------------------------
#define GS_DI __device__ __attribute__((always_inline)) inline

// LDS of the statistics pass: per binade and lane class, (count << 44) | significand sum and the
// maximum key. Counts stay below 2^20 per workgroup, so significand sums stay below 2^44.
struct StatsLds {
  unsigned long long pk[kB1 * kLaneCopies];
  uint32_t mx[kB1 * kLaneCopies];
};
// with the squared significands of the variance-budget solver (split at bit 24, see fq_squares)
template <bool SQ>
struct StatsLdsT : StatsLds {};
template <>
struct StatsLdsT<true> : StatsLds {
  unsigned long long qh[kB1 * kLaneCopies];
  unsigned long long ql[kB1 * kLaneCopies];
};
// LDS of a refinement pass: one window of at most kB2 bins, same packing, and for a level-2 window
// the complemented bin minimum.
struct WinLds {
  unsigned long long pk[kB2];
  uint32_t mx[kB2];
  uint32_t mnc[kB2];
  uint64_t qc[kNT / 64];
  uint64_t qs[kNT / 64];
};
template <bool SQ>
struct WinLdsT : WinLds {};
template <>
struct WinLdsT<true> : WinLds {
  unsigned long long qh[kB2];
  unsigned long long ql[kB2];
};
struct BinInfo {
  uint64_t Kab;  // count of keys strictly above the bin (including above the window)
  Fx Wab;        // their exact sum
  uint64_t cnt;
  Fx Wb;
  uint32_t mx;
};
// The solver's working copies of the histograms, in LDS: level 1 (L1Cache, kept in global memory
// as well between solves); the level-2 and level-3 windows when they exist.
template <int N>
struct WinCache {
  uint32_t cnt[N];  // window counts never exceed d < 2^31
  uint64_t sig[N];
  uint32_t mx[N];
};
struct SolveLds {
  uint64_t sk[kNT / 64];  // per-wave partial results of block scans and reductions
  uint64_t ss[kNT / 64];
  Fx sw[kB1 / 64];
  int ired[kNT / 64];
  BinInfo bi;
  L1Cache l1;
  WinCache<kB2> w2;
  WinCache<kB3> w3;
  uint32_t err;         // kFlagInternal when a wide-arithmetic invariant broke during this solve
  uint64_t bcnt, bsig;  // a level-2 bin's totals, broadcast by its owner (greedy queries)
  uint32_t bmx, bmn;
  // variance-budget solver: partial square sums of scans, and broadcasts of square sums
  Fq sq[kB1 / 64];
  Fq hq[2];
  uint64_t sqh[kNT / 64];
  uint64_t sql[kNT / 64];
};
struct Hists {
  uint32_t* err;       // LDS word collecting kFlagInternal from the wide-arithmetic helpers
  L1Cache* l1;         // LDS
  WinCache<kB2>* w2;   // LDS
  WinCache<kB3>* w3;   // LDS
  L1Cache* l1g;        // the row's level-1 table in global memory, written by the first solve
  const Hist1* h1g;    // the row's global copies, filled by the histogram passes
  WinHist* wg;         // copies of the refinement window
  const H1Q* h1q;      // variance-budget solver: square sums of the level-1 copies
  WinQ* wq;            // and of the level-2 window copies
  VarCtl* vc;          // and its per-row state
  const CountLine* cc; // keys collected in the row's candidate band
  int64_t cand_cap;    // the candidate list's capacity (0: no band)
};

GS_DI int block_max(SolveLds& s, int v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
  if ((threadIdx.x & 63) == 0) s.ired[threadIdx.x >> 6] = v;
  __syncthreads();
  int r = s.ired[0];
  for (int i = 1; i < kNT / 64; ++i) r = max(r, s.ired[i]);
  __syncthreads();
  return r;
}
GS_DI int block_min(SolveLds& s, int v) {
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o));
  if ((threadIdx.x & 63) == 0) s.ired[threadIdx.x >> 6] = v;
  __syncthreads();
  int r = s.ired[0];
  for (int i = 1; i < kNT / 64; ++i) r = min(r, s.ired[i]);
  __syncthreads();
  return r;
}

// Inclusive suffix sums over the lanes of a wave: lane l receives the sum over lanes l..63.
GS_DI uint64_t wave_suffix(uint64_t x, int lane) {
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_down(x, (unsigned)o);
    if (lane + o < 64) x += y;
  }
  return x;
}
GS_DI Fx wave_suffix(Fx x, int lane) {
  for (int o = 1; o < 64; o <<= 1) {
    Fx y;
#pragma unroll
    for (int i = 0; i < 5; ++i) y.w[i] = __shfl_down(x.w[i], (unsigned)o);
    if (lane + o < 64) fx_add(x, y);
  }
  return x;
}

// Level 1 (one bin per binade): exclusive suffix sums over the 256 binades, exact, into the LDS
// cache. Threads 0..255 (waves 0..3) own one binade each: a suffix scan inside each wave, then the
// totals of the waves above.
GS_DI void l1_build(SolveLds& s, const Hists& H) {
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  uint64_t k = 0, ik = 0;
  Fx w = fx_zero(), iw = fx_zero();
  if (t < kB1) {  // whole waves
    k = H.l1->cnt[t];
    if (k) w = fx_shifted(H.l1->sig[t], binade_shift(t), H.err);
    ik = wave_suffix(k, lane);
    iw = wave_suffix(w, lane);
    if (lane == 0) {
      s.sk[wv] = ik;
      s.sw[wv] = iw;
    }
  }
  __syncthreads();
  if (t < kB1) {
    uint64_t K = ik - k;
    Fx W = fx_sub(iw, w);
    for (int i = wv + 1; i < kB1 / 64; ++i) {
      K += s.sk[i];
      fx_add(W, s.sw[i]);
    }
    H.l1->K[t] = K;
    H.l1->W[t] = W;
  }
  __syncthreads();
}

GS_DI BinInfo l1_info(const Hists& H, int e) {
  BinInfo i;
  i.Kab = H.l1->K[e];
  i.Wab = H.l1->W[e];
  i.cnt = H.l1->cnt[e];
  i.Wb = i.cnt ? fx_shifted(H.l1->sig[e], binade_shift(e), H.err) : fx_zero();
  i.mx = H.l1->mx[e];
  return i;
}

// A refinement level inside one binade E: bins b = 0..nbins-1, thread t owns bins
// [t*per, t*per + per). Within one binade, sums of significands are plain integers.
struct Lvl {
  const uint32_t* cnt;
  const uint64_t* sig;
  const uint32_t* mx;
  int nbins, per;
  int shift;     // binade_shift(E): value = significand * 2^shift (units of 2^-149)
  uint64_t Kaw;  // count of keys above the window
  Fx Waw;        // their exact sum
  uint32_t* err; // as in Hists
};
struct Walk {
  uint64_t exK;  // count above this thread's bins, inside the window
  uint64_t exS;  // significand sum above this thread's bins, inside the window
};

GS_DI Lvl lvl2(const Hists& H, uint32_t E, uint64_t Kaw, const Fx& Waw) {
  Lvl L;
  L.cnt = H.w2->cnt; L.sig = H.w2->sig; L.mx = H.w2->mx;
  L.nbins = kB2; L.per = kB2 / kNT; L.shift = binade_shift((int)E); L.Kaw = Kaw; L.Waw = Waw; L.err = H.err;
  return L;
}
GS_DI Lvl lvl3(const Hists& H, uint32_t E, uint64_t Kaw, const Fx& Waw) {
  Lvl L;
  L.cnt = H.w3->cnt; L.sig = H.w3->sig; L.mx = H.w3->mx;
  L.nbins = kB3; L.per = kB3 / kNT; L.shift = binade_shift((int)E); L.Kaw = Kaw; L.Waw = Waw; L.err = H.err;
  return L;
}

// Exclusive suffix scan over thread index of (count, significand sum): a suffix scan inside each
// wave, then the totals of the waves above.
GS_DI void lvl_scan(const Lvl& L, SolveLds& s, Walk& w) {
  uint64_t k = 0, sg = 0;
  const int b0 = threadIdx.x * L.per;
  for (int j = 0; j < L.per; ++j) {
    const int b = b0 + j;
    if (b < L.nbins) {
      k += (uint64_t)L.cnt[b];
      sg += (uint64_t)L.sig[b];
    }
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const uint64_t ik = wave_suffix(k, lane), is = wave_suffix(sg, lane);
  if (lane == 0) {
    s.sk[wv] = ik;
    s.ss[wv] = is;
  }
  __syncthreads();
  uint64_t ak = 0, as = 0;
  for (int i = wv + 1; i < kNT / 64; ++i) {
    ak += s.sk[i];
    as += s.ss[i];
  }
  w.exK = ik - k + ak;
  w.exS = is - sg + as;
  __syncthreads();
}

GS_DI Fx lvl_total(const Lvl& L, uint64_t K, uint64_t S, uint64_t& Kout) {
  Kout = L.Kaw + K;
  Fx W = L.Waw;
  if (S) fx_add(W, fx_shifted(S, L.shift, L.err));
  return W;
}

// Aggregates above bin b and the bin's own totals, broadcast to every thread (b uniform).
GS_DI void lvl_bin_info(const Lvl& L, const Walk& w, int b, SolveLds& s, BinInfo& out) {
  if ((int)threadIdx.x == b / L.per) {
    uint64_t K = w.exK, S = w.exS;
    for (int j = L.per - 1; j >= 0; --j) {
      const int bb = threadIdx.x * L.per + j;
      if (bb >= L.nbins) continue;
      const uint64_t c = (uint64_t)L.cnt[bb];
      const uint64_t sg = (uint64_t)L.sig[bb];
      if (bb == b) {
        s.bi.Wab = lvl_total(L, K, S, s.bi.Kab);
        s.bi.cnt = c;
        s.bi.Wb = c ? fx_shifted(sg, L.shift, L.err) : fx_zero();
        s.bi.mx = L.mx[bb];
        break;
      }
      K += c;
      S += sg;
    }
  }
  __syncthreads();
  out = s.bi;
  __syncthreads();
}

// The density-budget form of Algorithm 2's criterion at a data value v, with k = #{a > v} and
// W = exact sum{a > v}: (B - k) * v <= fl(S - W).
GS_DI bool criterion(double B, const Fx& S, uint64_t k, const Fx& W, uint32_t vkey) {
  return (B - (double)k) * key_value(vkey) <= fx_to_double(fx_sub(S, W));
}

// Exact solver step: b1 = highest non-empty bin whose maximum satisfies the criterion, b2 =
// lowest non-empty bin above b1 (INT_MAX if none).
GS_DI void l1_exact(const Hists& H, double B, const Fx& S, SolveLds& s, int& b1, int& b2) {
  const int t = threadIdx.x;
  int best = -1, occupied = INT_MAX;
  if (t < kB1 && H.l1->cnt[t]) {
    if (criterion(B, S, H.l1->K[t], H.l1->W[t], H.l1->mx[t])) best = t;
  }
  b1 = block_max(s, best);
  if (t < kB1 && t > b1 && H.l1->cnt[t]) occupied = t;
  b2 = block_min(s, occupied);
}
// Inside a window each thread walks its bins from the top. A double-precision screen decides the
// criterion at every bin whose margin exceeds 2^-46 S: T = S - W is approximated by
// fl(S) - (fl(W above the window) + fl(window sum above)), within 2^-50 S of fl(T), and the
// left-hand side is computed exactly as the criterion computes it, so the screen and the exact
// evaluation agree wherever the screen decides; the exact criterion decides the rest (the bins
// next to the threshold).
GS_DI void lvl_exact(const Lvl& L, const Walk& w, double B, const Fx& S, SolveLds& s, int& b1, int& b2) {
  int best = -1;
  uint64_t K = w.exK, Sg = w.exS;
  const double Sd = fx_to_double(S), Wawd = fx_to_double(L.Waw);
  const double tol = 0x1p-46 * Sd + 0x1p-1000;
#pragma unroll 1
  for (int j = L.per - 1; j >= 0 && best < 0; --j) {
    const int b = threadIdx.x * L.per + j;
    if (b >= L.nbins) continue;
    const uint64_t c = (uint64_t)L.cnt[b];
    if (!c) continue;
    const double lhs = (B - (double)(L.Kaw + K)) * key_value(L.mx[b]);
    const double Td = Sd - (Wawd + ldexp((double)Sg, L.shift - 149));
    int pass = lhs <= Td - tol ? 1 : (lhs > Td + tol ? 0 : -1);
    if (pass < 0) {
      uint64_t Kt;
      const Fx W = lvl_total(L, K, Sg, Kt);
      pass = criterion(B, S, Kt, W, L.mx[b]) ? 1 : 0;
    }
    if (pass) best = b;
    K += c;
    Sg += (uint64_t)L.sig[b];
  }
  b1 = block_max(s, best);
  int lowest = INT_MAX;
  for (int j = 0; j < L.per; ++j) {
    const int b = threadIdx.x * L.per + j;
    if (b < L.nbins && b > b1 && (uint64_t)L.cnt[b]) {
      lowest = b;
      break;
    }
  }
  b2 = block_min(s, lowest);
}

// The solver's control flow runs in every thread of the workgroup on a private copy of the row's
// control block: every decision depends only on data all threads see (the LDS tables and values
// broadcast through LDS by the block-wide steps), so the copies stay identical and no barrier is
// needed between scalar steps. Thread 0 writes the block back at the end.
GS_DI void sv_finalize(RowCtl& c, double lam, uint32_t tcap) {
  c.lam = lam;
  c.tcap = tcap;
  c.inv_lam = (lam > 0.0 && lam < INFINITY) ? (float)(1.0 / lam) : 0.0f;
  c.done = 1;
  c.need = 0;
}

// Ask for a histogram of binade E (level 2; the pass also counts the keys >= qkey directly, kNone
// for none) or of keys [base, base + 2048) (level 3; wK and wW count and sum the keys above it).
// Clears the window's copies (every thread of the workgroup takes part; the kernel boundary orders
// the stores before the pass).
GS_DI void sv_request(RowCtl& c, const Hists& H, int level, uint32_t E, uint32_t base, uint32_t qkey, uint64_t wK,
                      const Fx& wW) {
  // The greedy solver's query of its last rescale step is answered by the direct count alone (no
  // later query reads a bin of this window), so that pass builds no bins and only the direct
  // count's fields are cleared.
  const bool qonly = level == 2 && c.solver == GSPAR_GREEDY && c.iter + 1 >= c.T;
  if (qonly) {
    if (threadIdx.x < kC23) {
      H.wg[threadIdx.x].qcnt = 0;
      H.wg[threadIdx.x].qsig = 0;
    }
  } else {
    uint4 z;
    z.x = z.y = z.z = z.w = 0u;
    uint4* w = reinterpret_cast<uint4*>(H.wg);
    for (int i = threadIdx.x; i < (int)(kC23 * sizeof(WinHist) / 16); i += kNT) w[i] = z;
  }
  c.qonly = qonly ? 1u : 0u;
  c.need = level;
  if (level == 2) {
    c.l2exp = E;
    c.l3base = kNone;
    c.qkey = qkey;
  } else {
    c.l3base = base;
    c.wK = wK;
    c.wW = wW;
  }
  // a window inside the candidate band (whole binades) holds only collected keys: its pass reads
  // the candidates instead of the row
  const uint32_t e = level == 2 ? E : (base >> 23);
  c.src = (c.band_hi > c.band_lo && (e << 23) >= c.band_lo && ((e + 1) << 23) <= c.band_hi) ? 1u : 0u;
}

// Count and significand sum of the level-2 window's keys in bins above sb, summed straight from the
// global copies (thread t owns bins [t * per, t * per + per)); bin sb's own totals, maximum and
// minimum go to s.bcnt, s.bsig, s.bmx, s.bmn.
GS_DI void w2_above(SolveLds& s, const Hists& H, int sb, uint64_t& ka, uint64_t& sa) {
  constexpr int per = kB2 / kNT;
  const int b0 = threadIdx.x * per;
  uint64_t c[per], g[per];
#pragma unroll
  for (int j = 0; j < per; ++j) {
    c[j] = 0;
    g[j] = 0;
#pragma unroll
    for (int q = 0; q < kC23; ++q) {
      c[j] += H.wg[q].cnt[b0 + j];
      g[j] += H.wg[q].sig[b0 + j];
    }
  }
  uint64_t k = 0, sg = 0;
#pragma unroll
  for (int j = 0; j < per; ++j) {
    if (b0 + j > sb) {
      k += c[j];
      sg += g[j];
    } else if (b0 + j == sb) {
      uint32_t mx = 0, mc = 0;
      for (int q = 0; q < kC23; ++q) {
        mx = max(mx, H.wg[q].mx[sb]);
        mc = max(mc, H.wg[q].mnc[sb]);
      }
      s.bcnt = c[j];
      s.bsig = g[j];
      s.bmx = mx;
      s.bmn = ~mc;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    k += __shfl_xor(k, o);
    sg += __shfl_xor(sg, o);
  }
  if ((threadIdx.x & 63) == 0) {
    s.sk[threadIdx.x >> 6] = k;
    s.ss[threadIdx.x >> 6] = sg;
  }
  __syncthreads();
  ka = 0;
  sa = 0;
  for (int i = 0; i < kNT / 64; ++i) {
    ka += s.sk[i];
    sa += s.ss[i];
  }
  __syncthreads();
}

// Greedy query: count K and exact sum W of the keys >= t. Resolved from level 1 when t's binade
// is empty, lies below t or starts at t; else from the level-2 pass of that binade, which counted
// the keys >= its qkey directly (qcnt, qsig), or whose bin holding t has all its keys on one side
// of t (bin minimum and maximum). Otherwise a level-2 pass of t's binade counting the keys >= t is
// requested. Returns 0 when resolved, 2 after a request.
GS_DI int sv_query(SolveLds& s, RowCtl& c, const Hists& H, uint64_t qcnt, uint64_t qsig, uint32_t t, uint64_t& K,
                   Fx& W) {
  const int e = (int)(t >> 23);
  const BinInfo i1 = l1_info(H, e);
  if ((t & 0x7FFFFFu) == 0) {
    K = i1.Kab + i1.cnt; W = i1.Wab; fx_add(W, i1.Wb);
    return 0;
  }
  if (i1.cnt == 0 || i1.mx < t) {
    K = i1.Kab; W = i1.Wab;
    return 0;
  }
  if (c.l2exp == (uint32_t)e) {
    uint64_t kq = 0, sq = 0;
    bool ok = false;
    if (c.qkey == t) {
      kq = qcnt;
      sq = qsig;
      ok = true;
    } else {
      uint64_t ka, sa;
      w2_above(s, H, (int)((t >> 11) & (kB2 - 1)), ka, sa);
      if (s.bcnt == 0 || s.bmx < t) {
        kq = ka; sq = sa; ok = true;
      } else if (s.bmn >= t) {
        kq = ka + s.bcnt; sq = sa + s.bsig; ok = true;
      }
    }
    if (ok) {
      K = i1.Kab + kq;
      W = i1.Wab;
      if (sq) fx_add(W, fx_shifted(sq, binade_shift(e), H.err));
      return 0;
    }
  }
  sv_request(c, H, 2, (uint32_t)e, 0, t, 0, fx_zero());
  return 2;
}

// Algorithm 3 in scale form: lambda_{j+1} = (B - k_j) / U_j, stop when it does not grow.
GS_DI void sv_greedy(SolveLds& s, RowCtl& c, const Hists& H, uint64_t qcnt, uint64_t qsig) {
  while (c.iter < c.T) {
    const double lam = c.lam;
    uint64_t K;
    Fx W;
    if (sv_query(s, c, H, qcnt, qsig, cap_key(lam), K, W)) return;
    const double U = fx_to_double(fx_sub(c.S, W));
    if (U == 0.0) break;
    const double ln = (c.B - (double)K) / U;
    if (!(ln > lam)) break;
    c.lam = ln;
    c.iter += 1;
  }
  sv_finalize(c, c.lam, cap_key(c.lam));
}

// The capped set of Proposition 1 is {p_i = 1}: the magnitudes above the criterion's value v
// (keys >= tcap = key(v) + 1) and, should fl(lambda * a) reach 1 below them (a tied run at v when
// the criterion holds with equality), those too. Both sets are {key >= t} for some t, so the union
// is the smaller threshold; every pass tests key >= the final tcap.
GS_DI uint32_t capped_threshold(double lam, uint32_t tcap) {
  const uint32_t t = cap_key(lam);
  return t < tcap ? t : tcap;
}

GS_DI void sv_exact_finish(RowCtl& c, uint64_t K, const Fx& W, uint32_t tcap) {
  const double T1 = fx_to_double(fx_sub(c.S, W));
  const double lam = (c.B - (double)K) / T1;
  sv_finalize(c, lam, capped_threshold(lam, tcap));
}

// The exact solver descends levels: at each one it finds the highest bin whose maximum passes
// the criterion (b1) and the lowest occupied bin above it (b2); the answer is b1's maximum
// unless b2 holds two or more values that could still pass, in which case b2 is refined.
GS_DI void sv_exact(SolveLds& s, RowCtl& c, const Hists& H) {
  const int level = c.stage;
  int b1, b2;
  BinInfo c1, c2;  // the bins b1 and b2 at this level
  uint32_t E = 0;
  if (level == 1) {
    l1_exact(H, c.B, c.S, s, b1, b2);
    if (b1 >= 0) c1 = l1_info(H, b1);
    if (b2 != INT_MAX) c2 = l1_info(H, b2);
  } else {
    E = c.l2exp;
    Lvl L;
    if (level == 2) {
      const BinInfo iE = l1_info(H, (int)E);
      L = lvl2(H, E, iE.Kab, iE.Wab);
    } else {
      L = lvl3(H, E, c.wK, c.wW);
    }
    Walk w;
    lvl_scan(L, s, w);
    lvl_exact(L, w, c.B, c.S, s, b1, b2);
    if (b1 >= 0) lvl_bin_info(L, w, b1, s, c1);
    if (b2 != INT_MAX) lvl_bin_info(L, w, b2, s, c2);
  }
  // refine b2 when it holds two or more values, of which a smaller one may pass; also when no
  // bin's maximum passes at this level (b1 < 0): the lowest occupied bin may still hold a passing
  // value below its maximum (when the answer lies in the row's lowest binade, or in a window's
  // lowest bin), and the candidate from a level up, if any, stays the fallback
  if (b2 != INT_MAX && level < 3 && c2.cnt >= 2) {
    if (b1 >= 0) {
      c.fbValid = 1;
      c.fbK = c1.Kab;
      c.fbW = c1.Wab;
      c.fbTcap = c1.mx + 1;
    }
    c.stage = level + 1;
    if (level == 1) sv_request(c, H, 2, (uint32_t)b2, 0, kNone, 0, fx_zero());
    else sv_request(c, H, 3, 0, (E << 23) | ((uint32_t)b2 << 11), kNone, c2.Kab, c2.Wab);
    return;
  }
  if (b1 >= 0) {
    sv_exact_finish(c, c1.Kab, c1.Wab, c1.mx + 1);
  } else if (c.fbValid) {
    // no value in this window passes: the answer is the candidate found one level up
    sv_exact_finish(c, c.fbK, c.fbW, c.fbTcap);
  } else {
    c.flags |= kFlagInternal;
    sv_finalize(c, NAN, kKeyInf);
  }
}

// ------------------------------------------------------------------------------------------
// Variance-budget exact solver: Algorithm 2 as printed (budget (1 + eps) sum a^2 on the variance,
// eqs. 6-7). With the magnitudes sorted decreasingly, k is the smallest index with
// a_(k+1) T1_k <= eps A + T2_k, where A = sum a^2 and T1_k, T2_k are the sum and the sum of
// squares of the magnitudes after the first k; lambda = T1_k / (eps A + T2_k) and the capped set
// is {a > a_(k+1)}. Candidates are distinct values; moving down to the next smaller value never
// turns the criterion from true to false, so the same three-level search as the density form
// applies, with the square sums of the bins carried alongside the counts and sums.
// ------------------------------------------------------------------------------------------
GS_DI Fq wave_suffix(Fq x, int lane) {
  for (int o = 1; o < 64; o <<= 1) {
    Fq y;
#pragma unroll
    for (int i = 0; i < kQ; ++i) y.w[i] = __shfl_down(x.w[i], (unsigned)o);
    if (lane + o < 64) fq_add(x, y);
  }
  return x;
}

// The criterion at a data value v, with W and H the exact sum and square sum of the magnitudes
// above v: v * fl(S - W) <= fl(eps * fl(A2)) + fl(A2 - H), each operation rounded on its own (the
// pragma keeps the compiler from fusing the product and the sum). T1 and the right-hand side are
// returned for lambda.
GS_DI bool v_criterion(double eps, const Fx& S, const Fq& A2, const Fx& W, const Fq& H, uint32_t vkey, double& T1,
                       double& rhs) {
#pragma clang fp contract(off)
  T1 = fx_to_double(fx_sub(S, W));
  const double T2 = fq_to_double(fq_sub(A2, H));
  const double eA = eps * fq_to_double(A2);
  rhs = eA + T2;
  return key_value(vkey) * T1 <= rhs;
}

// A double-precision screen of the criterion from approximate sums (each within a few units of
// rounding of the exact value, all terms non-negative): 1 or 0 when the margin exceeds 2^-44 of
// v*S + (1 + eps)*A2, far above every rounding of either evaluation, so the exact criterion
// decides the same way; -1 when the exact evaluation must decide.
GS_DI int v_screen(double eps, double Sd, double A2d, double Wd, double Hd, double v) {
#pragma clang fp contract(off)
  const double lhs = v * (Sd - Wd);
  const double rhs = eps * A2d + (A2d - Hd);
  const double tol = 0x1p-44 * (v * Sd + (1.0 + eps) * A2d);
  if (lhs <= rhs - tol) return 1;
  if (lhs >= rhs + tol) return 0;
  return -1;
}

GS_DI void v_finish(RowCtl& c, const Fq& A2, const Fx& W, const Fq& H, uint32_t tcap) {
  double T1, rhs;
  v_criterion(c.B, c.S, A2, W, H, 1u, T1, rhs);
  const double lam = T1 / rhs;
  sv_finalize(c, lam, capped_threshold(lam, tcap));
}

// A bin of a level: keys above it (count, sum, square sum), its own count and maximum key.
struct VInfo {
  uint64_t K;
  Fx W;
  Fq H;
  uint64_t cnt;
  uint32_t mx;
};

// Asks for a refinement window like sv_request, clears the window's square sums for level 2 and
// keeps the square sum above the window.
GS_DI void v_request(RowCtl& c, const Hists& H, int level, uint32_t E, uint32_t base, uint64_t wK, const Fx& wW,
                     const Fq& wH) {
  sv_request(c, H, level, E, base, kNone, wK, wW);
  if (level == 2) {
    uint4 z;
    z.x = z.y = z.z = z.w = 0u;
    uint4* w = reinterpret_cast<uint4*>(H.wq);
    for (int i = threadIdx.x; i < (int)(kC23 * sizeof(WinQ) / 16); i += kNT) w[i] = z;
  }
  if (threadIdx.x == 0) H.vc->wH = wH;
}

// Level 1 (first solve): square sums of the binades from the global copies, the square sum above
// each binade (exclusive suffix over binades), the total A2, then b1 = highest occupied binade whose
// maximum passes the criterion and b2 = lowest occupied binade above b1.
GS_DI void v_level1(SolveLds& s, const RowCtl& c, const Hists& H, Fq& A2, int& b1, int& b2, VInfo& i1, VInfo& i2) {
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  Fq q = fq_zero(), iq = fq_zero();
  if (t < kB1) {  // whole waves
    uint64_t qh = 0, ql = 0;
    for (int k = 0; k < kC1; ++k) {
      qh += H.h1q[k].qh[t];
      ql += H.h1q[k].ql[t];
    }
    if (H.l1->cnt[t]) q = fq_squares(qh, ql, binade_shift(t), H.err);
    iq = wave_suffix(q, lane);
    if (lane == 0) s.sq[wv] = iq;
  }
  __syncthreads();
  Fq above = fq_zero();
  if (t < kB1) {
    above = fq_sub(iq, q);
    for (int i = wv + 1; i < kB1 / 64; ++i) fq_add(above, s.sq[i]);
    if (t == 0) {
      Fq tot = above;
      fq_add(tot, q);
      s.hq[0] = tot;
    }
  }
  __syncthreads();
  A2 = s.hq[0];
  int best = -1, occupied = INT_MAX;
  if (t < kB1 && H.l1->cnt[t]) {
    double T1, rhs;
    if (v_criterion(c.B, c.S, A2, H.l1->W[t], above, H.l1->mx[t], T1, rhs)) best = t;
  }
  b1 = block_max(s, best);
  if (t < kB1 && t > b1 && H.l1->cnt[t]) occupied = t;
  b2 = block_min(s, occupied);
  if (t == b1) s.hq[0] = above;
  if (t == b2) s.hq[1] = above;
  __syncthreads();
  if (b1 >= 0) {
    i1.K = H.l1->K[b1];
    i1.W = H.l1->W[b1];
    i1.H = s.hq[0];
    i1.cnt = H.l1->cnt[b1];
    i1.mx = H.l1->mx[b1];
  }
  if (b2 != INT_MAX) {
    i2.K = H.l1->K[b2];
    i2.W = H.l1->W[b2];
    i2.H = s.hq[1];
    i2.cnt = H.l1->cnt[b2];
    i2.mx = H.l1->mx[b2];
  }
  __syncthreads();
}

// Level 2 (a binade's 4096 bins, square sums from the global window copies) or level 3 (2048
// single keys from `base`, whose square sums follow from the counts): b1 and b2 as at level 1, the
// keys above the window given by (L.Kaw, L.Waw, Haw).
// The square-sum parts (see fq_squares) of bin b of a level: level 2 from the global window copies,
// level 3 (one key per bin) the count times the key's squared significand.
GS_DI void v_bin_squares(const Hists& H, const Lvl& L, bool level2, uint32_t base, int b, uint64_t& qh,
                         uint64_t& ql) {
  if (level2) {
    qh = 0;
    ql = 0;
#pragma unroll
    for (int k = 0; k < kC23; ++k) {
      qh += H.wq[k].qh[b];
      ql += H.wq[k].ql[b];
    }
  } else {
    const uint64_t m = key_sig(base + (uint32_t)b), m2 = m * m, cnt = (uint64_t)L.cnt[b];
    qh = cnt * (m2 >> 24);
    ql = cnt * (m2 & 0xFFFFFFu);
  }
}

// Level 2 (a binade's 4096 bins, square sums from the global window copies) or level 3 (2048
// single keys from `base`): b1 and b2 as at level 1, the keys above the window given by (L.Kaw,
// L.Waw, Haw). The thread's bins are walked again where needed instead of being held in registers.
GS_DI void v_level(SolveLds& s, const RowCtl& c, const Hists& H, const Lvl& L, bool level2, uint32_t base,
                   const Fq& A2, const Fq& Haw, int& b1, int& b2, VInfo& i1, VInfo& i2) {
  const int per = L.per, b0 = threadIdx.x * per;
  uint64_t tk = 0, ts = 0, tqh = 0, tql = 0;
  for (int j = 0; j < per; ++j) {
    const int b = b0 + j;
    if (b >= L.nbins) break;
    uint64_t qh, ql;
    v_bin_squares(H, L, level2, base, b, qh, ql);
    tk += (uint64_t)L.cnt[b];
    ts += (uint64_t)L.sig[b];
    tqh += qh;
    tql += ql;
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const uint64_t ik = wave_suffix(tk, lane), is = wave_suffix(ts, lane);
  const uint64_t iqh = wave_suffix(tqh, lane), iql = wave_suffix(tql, lane);
  if (lane == 0) {
    s.sk[wv] = ik;
    s.ss[wv] = is;
    s.sqh[wv] = iqh;
    s.sql[wv] = iql;
  }
  __syncthreads();
  uint64_t eK = ik - tk, eS = is - ts, eQH = iqh - tqh, eQL = iql - tql;  // above this thread's bins
  for (int i = wv + 1; i < kNT / 64; ++i) {
    eK += s.sk[i];
    eS += s.ss[i];
    eQH += s.sqh[i];
    eQL += s.sql[i];
  }
  __syncthreads();
  // this thread's bins from the top: the first (highest) passing one (a loop that is not unrolled:
  // the criterion's wide arithmetic is long, and one copy of it keeps the code in the instruction
  // cache). The double-precision screen decides all but the bins next to the threshold.
  int best = -1;
  {
    const double Sd = fx_to_double(c.S), A2d = fq_to_double(A2);
    const double Wawd = fx_to_double(L.Waw), Hawd = fq_to_double(Haw);
    uint64_t Sg = eS, QH = eQH, QL = eQL;
#pragma unroll 1
    for (int j = per - 1; j >= 0; --j) {
      const int b = b0 + j;
      if (b >= L.nbins) continue;
      const uint64_t cnt = (uint64_t)L.cnt[b];
      uint64_t qh, ql;
      v_bin_squares(H, L, level2, base, b, qh, ql);
      if (cnt) {
        const double Wd = Wawd + ldexp((double)Sg, L.shift - 149);
        const double Hd = Hawd + ldexp((double)QH, 2 * L.shift - 298 + 24) + ldexp((double)QL, 2 * L.shift - 298);
        int pass = v_screen(c.B, Sd, A2d, Wd, Hd, key_value(L.mx[b]));
        if (pass < 0) {
          Fx W = L.Waw;
          if (Sg) fx_add(W, fx_shifted(Sg, L.shift, L.err));
          Fq Hq = Haw;
          fq_add(Hq, fq_squares(QH, QL, L.shift, L.err));
          double T1, rhs;
          pass = v_criterion(c.B, c.S, A2, W, Hq, L.mx[b], T1, rhs) ? 1 : 0;
        }
        if (pass) {
          best = b;
          break;
        }
      }
      Sg += (uint64_t)L.sig[b];
      QH += qh;
      QL += ql;
    }
  }
  b1 = block_max(s, best);
  int lowest = INT_MAX;
  for (int j = 0; j < per; ++j) {
    const int b = b0 + j;
    if (b < L.nbins && b > b1 && (uint64_t)L.cnt[b]) {
      lowest = b;
      break;
    }
  }
  b2 = block_min(s, lowest);
  // the owners of b1 and b2 broadcast the aggregates above their bin
#pragma unroll 1
  for (int w = 0; w < 2; ++w) {
    const int bb = w == 0 ? b1 : b2;
    if (bb >= 0 && bb != INT_MAX && (int)threadIdx.x == bb / per) {
      uint64_t K = eK, Sg = eS, QH = eQH, QL = eQL;
#pragma unroll 1
      for (int j = per - 1; b0 + j > bb; --j) {
        const int b = b0 + j;
        if (b >= L.nbins) continue;
        uint64_t qh, ql;
        v_bin_squares(H, L, level2, base, b, qh, ql);
        K += (uint64_t)L.cnt[b];
        Sg += (uint64_t)L.sig[b];
        QH += qh;
        QL += ql;
      }
      s.bi.Kab = L.Kaw + K;
      Fx W = L.Waw;
      if (Sg) fx_add(W, fx_shifted(Sg, L.shift, L.err));
      s.bi.Wab = W;
      Fq Hq = Haw;
      fq_add(Hq, fq_squares(QH, QL, L.shift, L.err));
      s.hq[0] = Hq;
      s.bi.cnt = (uint64_t)L.cnt[bb];
      s.bi.mx = L.mx[bb];
    }
    __syncthreads();
    if (bb >= 0 && bb != INT_MAX) {
      VInfo o;
      o.K = s.bi.Kab;
      o.W = s.bi.Wab;
      o.H = s.hq[0];
      o.cnt = s.bi.cnt;
      o.mx = s.bi.mx;
      if (w == 0) i1 = o;
      else i2 = o;
    }
    __syncthreads();
  }
}

GS_DI void sv_variance(SolveLds& s, RowCtl& c, const Hists& H) {
  const int level = c.stage;
  int b1, b2;
  VInfo i1, i2;
  Fq A2;
  uint32_t E = 0;
  if (level == 1) {
    v_level1(s, c, H, A2, b1, b2, i1, i2);
    if (threadIdx.x == 0) H.vc->A2 = A2;
  } else {
    A2 = H.vc->A2;
    const Fq Haw = H.vc->wH;
    E = c.l2exp;
    Lvl L;
    if (level == 2) {
      const BinInfo iE = l1_info(H, (int)E);
      L = lvl2(H, E, iE.Kab, iE.Wab);
    } else {
      L = lvl3(H, E, c.wK, c.wW);
    }
    v_level(s, c, H, L, level == 2, level == 2 ? 0u : c.l3base, A2, Haw, b1, b2, i1, i2);
  }
  // refine b2 when it holds two or more values, of which a smaller one may pass (also when
  // nothing at this level passes: the lowest occupied bin may still hold a passing value)
  if (b2 != INT_MAX && level < 3 && i2.cnt >= 2) {
    if (b1 >= 0) {
      c.fbValid = 1;
      c.fbK = i1.K;
      c.fbW = i1.W;
      c.fbTcap = i1.mx + 1;
      if (threadIdx.x == 0) H.vc->fbH = i1.H;
    }
    c.stage = level + 1;
    if (level == 1) v_request(c, H, 2, (uint32_t)b2, 0, 0, fx_zero(), i2.H);
    else v_request(c, H, 3, 0, (E << 23) | ((uint32_t)b2 << 11), i2.K, i2.W, i2.H);
    return;
  }
  if (b1 >= 0 || c.fbValid) {
    // b1's maximum, else the candidate found one level up
    Fx W;
    Fq Hq;
    uint32_t tcap;
    if (b1 >= 0) {
      W = i1.W;
      Hq = i1.H;
      tcap = i1.mx + 1;
    } else {
      W = c.fbW;
      Hq = H.vc->fbH;
      tcap = c.fbTcap;
    }
    v_finish(c, A2, W, Hq, tcap);
  } else {
    // no value passes (possible only through rounding with eps = 0): every nonzero is capped
    sv_finalize(c, INFINITY, 1);
  }
}

// First solve after the statistics pass: totals and the special cases.
template <bool VAR>
GS_DI void sv_start(SolveLds& s, RowCtl& c, const Hists& H, int64_t d) {
  const BinInfo i0 = l1_info(H, 0);
  const BinInfo inf = l1_info(H, 255);
  // every finite key lies in binades 0..254; binade 255 counts only Inf/NaN
  Fx tot = i0.Wab;
  fx_add(tot, i0.Wb);
  if (inf.cnt) {
    tot = fx_sub(tot, inf.Wb);
    c.flags |= GSPAR_FLAG_NONFINITE;
  }
  c.S = tot;
  c.stage = 1;
  // zeros = d minus the histogram's population (every nonzero key, finite or not, is binned)
  c.zeros = (uint64_t)d - (i0.Kab + i0.cnt);
  const uint64_t nnz = (uint64_t)d - c.zeros;
  if (c.flags & (GSPAR_FLAG_NONFINITE | GSPAR_FLAG_BADRHO | GSPAR_FLAG_BADSEG)) {
    sv_finalize(c, NAN, kKeyInf);
    return;
  }
  if (nnz == 0) {
    c.flags |= GSPAR_FLAG_ALLZERO;
    sv_finalize(c, INFINITY, 1);
    return;
  }
  if constexpr (VAR) {
    sv_variance(s, c, H);
    return;
  }
  if (c.B >= (double)nnz) {
    sv_finalize(c, INFINITY, 1);
    return;
  }
  if (c.B == 0.0) {
    sv_finalize(c, 0.0, kKeyInf);
    return;
  }
  if (c.solver == GSPAR_GREEDY) {
    c.lam = c.B / fx_to_double(c.S);
    c.iter = 0;
    sv_greedy(s, c, H, 0, 0);
  } else {
    sv_exact(s, c, H);
  }
}

// Sums the global copies of a histogram (filled with atomics by an earlier kernel on the same
// stream) into an LDS cache. Every load of a thread is issued before the first sum, so the whole
// reduction costs one round trip to memory.
template <int COPIES, int NBINS, typename HistT, typename CntT>
GS_DI void reduce_into(const HistT* h, CntT* cnt, uint64_t* sig, uint32_t* mx) {
  static_assert(NBINS % kNT == 0 || NBINS < kNT, "bins per thread");
  constexpr int kPer = NBINS < kNT ? 1 : NBINS / kNT;
  uint64_t c[kPer][COPIES], g[kPer][COPIES];
  uint32_t m[kPer][COPIES];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int b = threadIdx.x + j * kNT;
#pragma unroll
    for (int k = 0; k < COPIES; ++k) {
      const bool ok = b < NBINS;
      c[j][k] = ok ? h[k].cnt[b] : 0;
      g[j][k] = ok ? h[k].sig[b] : 0;
      m[j][k] = ok ? h[k].mx[b] : 0;
    }
  }
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int b = threadIdx.x + j * kNT;
    uint64_t cs = 0, gs = 0;
    uint32_t ms = 0;
#pragma unroll
    for (int k = 0; k < COPIES; ++k) {
      cs += c[j][k];
      gs += g[j][k];
      ms = max(ms, m[j][k]);
    }
    if (b < NBINS) {
      cnt[b] = (CntT)cs;
      sig[b] = gs;
      mx[b] = ms;
    }
  }
}

// The row's solver, run by one workgroup per row after each histogram pass: it either finishes the
// row (lambda and the capped threshold become final) or requests the next refinement window.
// `first`: the solve right after the statistics pass.
// VAR: the variance-budget solver's instantiation (a kernel of its own, so that its registers do
// not weigh on the density-budget solvers).
template <bool VAR>
GS_DI void solve_row(SolveLds& s, RowCtl* gc, const Hists& H, int64_t d, bool first) {
  // The global reads of a solve are issued together, so they share one round trip: level 1
  // (summed from its copies by the first solve, which also builds the suffix sums and keeps the
  // table in global memory for the later solves) and the direct count of the last level-2 pass.
  RowCtl c = *gc;
  constexpr int n16 = (int)(sizeof(L1Cache) / 16);
  constexpr int per16 = (n16 + kNT - 1) / kNT;
  uint4 tab[per16];
  uint64_t qcnt = 0, qsig = 0;
  if (first) {
    reduce_into<kC1, kB1>(H.h1g, H.l1->cnt, H.l1->sig, H.l1->mx);
    // the candidate band is usable only if every key in it was kept (a statistics workgroup whose
    // region overflowed reserves more than the list holds)
    if (H.cand_cap) {
      c.cand_n = H.cc->v;
      if (c.cand_n > (uint64_t)H.cand_cap) c.band_lo = c.band_hi = 0;
    } else {
      c.band_lo = c.band_hi = 0;
    }
  } else {
    if (c.done) return;
    const uint4* src = reinterpret_cast<const uint4*>(H.l1g);
#pragma unroll
    for (int j = 0; j < per16; ++j) {
      const int i = threadIdx.x + j * kNT;
      if (i < n16) tab[j] = src[i];
    }
#pragma unroll
    for (int k = 0; k < kC23; ++k) {
      qcnt += H.wg[k].qcnt;
      qsig += H.wg[k].qsig;
    }
  }
  if (c.done) return;
  if (!first) {
    uint4* dst = reinterpret_cast<uint4*>(H.l1);
#pragma unroll
    for (int j = 0; j < per16; ++j) {
      const int i = threadIdx.x + j * kNT;
      if (i < n16) dst[i] = tab[j];
    }
  }
  // for the exact solver the level-2 / level-3 window the last pass filled (for the greedy solver
  // the bins of a level-2 window are read only if a query needs them)
  if (c.solver != GSPAR_GREEDY) {
    if (c.stage == 2) reduce_into<kC23, kB2>(H.wg, H.w2->cnt, H.w2->sig, H.w2->mx);
    if (c.stage == 3) reduce_into<kC23, kB3>(H.wg, H.w3->cnt, H.w3->sig, H.w3->mx);
  }
  c.need = 0;
  if (threadIdx.x == 0) s.err = 0;
  // every load above has returned before any thread can go on to clear the window it read
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (first) {
    l1_build(s, H);
    constexpr int n16 = (int)(sizeof(L1Cache) / 16);
    const uint4* src = reinterpret_cast<const uint4*>(H.l1);
    uint4* dst = reinterpret_cast<uint4*>(H.l1g);
    for (int i = threadIdx.x; i < n16; i += kNT) dst[i] = src[i];
    sv_start<VAR>(s, c, H, d);
  } else if constexpr (VAR) {
    sv_variance(s, c, H);
  } else if (c.solver == GSPAR_GREEDY) {
    sv_greedy(s, c, H, qcnt, qsig);
  } else {
    sv_exact(s, c, H);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    if (s.err) {
      // a broken invariant of the exact arithmetic: the row is reported, not sampled
      c.flags |= s.err;
      sv_finalize(c, NAN, kKeyInf);
    }
    *gc = c;
  }
}

// ------------------------------------------------------------------------------------------
// Kernels.
// ------------------------------------------------------------------------------------------
// Segmented calls: the workgroup maps of the histogram passes (row << 32 | block) and of the sample
// pass (row << 32 | workgroup within the row), built by one workgroup of 256 threads from the
// device offsets in row order, 256 rows at a time: an exclusive scan of the per-row counts, then
// every thread fills map entries, finding each entry's row by a binary search of the scan. Also
// the verdict whether the maps have exactly the launched (host) shape.
__device__ void seg_maps(const Args& a) {
  __shared__ int64_t s_tot[2][4];
  __shared__ int64_t s_pre[2][257];  // exclusive prefixes of the batch's rows (+ the batch total)
  uint64_t* bmap = reinterpret_cast<uint64_t*>(a.ws + a.lay.bmap);
  uint64_t* tmap = reinterpret_cast<uint64_t*>(a.ws + a.lay.tmap);
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  int64_t cb = 0, cw = 0;  // workgroups of the rows before this batch
  for (int64_t r0 = 0; r0 < a.rows; r0 += 256) {
    const int64_t r = r0 + t;
    int64_t nb = 0, nw = 0;
    if (r < a.rows) {
      int64_t base, len;
      row_span(a, r, base, len);
      nb = (len + a.chunk - 1) / a.chunk;
      const int64_t rt = len > kTileElems ? (len + kTileElems - 1) / kTileElems : 1;
      nw = (rt + a.seg_k - 1) / a.seg_k;
    }
    int64_t xb = nb, xw = nw;  // inclusive scans over the wave
    for (int o = 1; o < 64; o <<= 1) {
      const int64_t yb = __shfl_up(xb, o), yw = __shfl_up(xw, o);
      if (lane >= o) {
        xb += yb;
        xw += yw;
      }
    }
    if (lane == 63) {
      s_tot[0][wv] = xb;
      s_tot[1][wv] = xw;
    }
    __syncthreads();
    int64_t pb = xb - nb, pw = xw - nw, tb = 0, tw = 0;
    for (int w = 0; w < 4; ++w) {
      if (w < wv) {
        pb += s_tot[0][w];
        pw += s_tot[1][w];
      }
      tb += s_tot[0][w];
      tw += s_tot[1][w];
    }
    s_pre[0][t] = pb;
    s_pre[1][t] = pw;
    if (t == 0) {
      s_pre[0][256] = tb;
      s_pre[1][256] = tw;
    }
    __syncthreads();
    // entry e of the batch belongs to the last row whose prefix is <= e (rows past the end have
    // no entries and the prefix of a row with none equals the next row's)
    for (int m = 0; m < 2; ++m) {
      const int64_t tot = s_pre[m][256], c0 = m == 0 ? cb : cw, cap = m == 0 ? a.seg_blocks : a.seg_wgs;
      uint64_t* map = m == 0 ? bmap : tmap;
      for (int64_t e = t; e < tot && c0 + e < cap; e += 256) {
        int lo = 0, hi = 255;  // the row lies in [lo, hi]
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (s_pre[m][mid] <= e) lo = mid;
          else hi = mid - 1;
        }
        map[c0 + e] = ((uint64_t)(r0 + lo) << 32) | (uint64_t)(e - s_pre[m][lo]);
      }
    }
    cb += tb;
    cw += tw;
    __syncthreads();
  }
  if (t == 0) *segok_of(a) = (cb == a.seg_blocks && cw == a.seg_wgs) ? 1u : 2u;
}

__global__ void __launch_bounds__(256) k_init(Args a) {
  if (a.seg && blockIdx.x == 0) seg_maps(a);
  const int64_t tid = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  // level-1 histogram copies, capped-count lines, look-back status words
  uint64_t* h1 = reinterpret_cast<uint64_t*>(a.ws + a.lay.h1);
  const int64_t n1 = a.rows * kC1 * (int64_t)(sizeof(Hist1) / 8);
  for (int64_t i = tid; i < n1; i += stride) h1[i] = 0;
  uint64_t* kc = reinterpret_cast<uint64_t*>(a.ws + a.lay.kc);
  const int64_t nkc = (int64_t)((a.lay.status - a.lay.kc) / 8);
  for (int64_t i = tid; i < nkc; i += stride) kc[i] = 0;
  uint64_t* st = status_of(a);
  const int64_t ns = a.rows * a.lay.tiles;
  for (int64_t i = tid; i < ns; i += stride) st[i] = 0;
  if (a.solver == GSPAR_VARIANCE) {
    uint64_t* q = reinterpret_cast<uint64_t*>(a.ws + a.lay.h1q);
    const int64_t nq = a.rows * kC1 * (int64_t)(sizeof(H1Q) / 8);
    for (int64_t i = tid; i < nq; i += stride) q[i] = 0;
  }
  if (a.lay.cand_cap) {
    // sample histograms and candidate count lines (adjacent in the layout)
    uint64_t* pc = reinterpret_cast<uint64_t*>(a.ws + a.lay.pre);
    const int64_t np = (int64_t)((a.lay.cand - a.lay.pre) / 8);
    for (int64_t i = tid; i < np; i += stride) pc[i] = 0;
  }
  for (int64_t r = tid; r < a.rows; r += stride) {
    RowCtl c;
    memset(&c, 0, sizeof(c));
    const double rho = a.rho_dev ? a.rho_dev[r] : a.rho;
    int64_t base, len;
    const bool ok = row_span(a, r, base, len);
    if (a.solver == GSPAR_VARIANCE) {
      // the variance budget eps (any finite eps >= 0) in place of the density
      c.B = rho;
      if (!(rho >= 0.0 && rho < INFINITY)) c.flags = GSPAR_FLAG_BADRHO;
    } else {
      c.B = rho * (double)len;
      if (!(rho >= 0.0 && rho <= 1.0)) c.flags = GSPAR_FLAG_BADRHO;
    }
    if (!ok) c.flags |= GSPAR_FLAG_BADSEG;
    c.l2exp = kNone;
    c.l3base = kNone;
    c.qkey = kNone;
    c.solver = a.solver;
    c.T = a.T;
    *ctl_of(a, r) = c;
  }
}

// Row and block of a histogram-pass workgroup: rows * nb workgroups for a strided batch, the map
// built by k_init for a segmented call (false: nothing to do).
__device__ __forceinline__ bool hist_block(const Args& a, int64_t& row, int64_t& blk) {
  if (!a.seg) {
    row = blockIdx.x / a.nb;
    blk = blockIdx.x % a.nb;
    return true;
  }
  if (*segok_of(a) != 1) return false;
  const uint64_t e = reinterpret_cast<const uint64_t*>(a.ws + a.lay.bmap)[blockIdx.x];
  row = (int64_t)(e >> 32);
  blk = (int64_t)(e & 0xFFFFFFFFu);
  return true;
}

// A global-memory pointer every lane holds equally, moved to scalar registers (on the device:
// in the global address space, so stores take a scalar base and a 32-bit vector offset).
#if defined(__HIP_DEVICE_COMPILE__)
typedef __attribute__((address_space(1))) char gchar;
#define GS_GLOBAL(T) T __attribute__((address_space(1)))
__device__ __forceinline__ gchar* uniform_ptr(void* p) {
  const uint64_t u = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return (gchar*)(((uint64_t)hi << 32) | lo);
}
#else
typedef char gchar;
#define GS_GLOBAL(T) T
GS_HD gchar* uniform_ptr(void* p) { return static_cast<gchar*>(p); }
#endif

// popcount(m & bits of the lanes below this one)
__device__ __forceinline__ uint32_t lanes_below(unsigned long long m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
// Exclusive prefix over the lanes of a wave of x in [0, 2^B) from B ballots; `total` receives the
// wave's sum.
template <int B>
__device__ __forceinline__ uint32_t wave_prefix_bits(uint32_t x, uint32_t& total) {
  uint32_t pre = 0;
  total = 0;
#pragma unroll
  for (int b = 0; b < B; ++b) {
    const unsigned long long m = __ballot((x >> b) & 1);
    pre += lanes_below(m) << b;
    total += (uint32_t)__popcll(m) << b;
  }
  return pre;
}

// Systematic sample of each row for the candidate band: kPreWG workgroups per row each read
// kPreLines of the row's whole 64-byte lines, spread evenly over the row, and add a histogram over
// binades (count, significand sum) into the row's PreHist. Every load is issued before any is used.
__global__ void __launch_bounds__(256) k_presample(Args a) {
  static_assert(kB1 == 256 && kPreLines % 64 == 0, "one binade per thread, 64 lines per round");
  constexpr int kRounds = kPreLines / 64;
  constexpr int kCopies = 4;  // LDS copies by lane, to spread same-bin atomics
  __shared__ uint32_t s_cnt[kB1 * kCopies];
  __shared__ unsigned long long s_sig[kB1 * kCopies];
  const int64_t row = blockIdx.x / kPreWG;
  const int p = (int)(blockIdx.x % kPreWG);
  const int t = threadIdx.x;
  for (int i = t; i < kB1 * kCopies; i += 256) {
    s_cnt[i] = 0;
    s_sig[i] = 0;
  }
  __syncthreads();
  const float* __restrict__ gr = a.g + row * a.ld;
  const int64_t nl = a.d / 16;         // whole lines of the row
  const int64_t ns = pre_lines(a.d);   // lines sampled (ns <= nl)
  float4 x[kRounds];
#pragma unroll
  for (int j = 0; j < kRounds; ++j) {
    const int64_t i = (int64_t)p * kPreLines + j * 64 + (t >> 2);  // sample index
    const int64_t line = (i < ns ? i : ns - 1) * nl / ns;             // < nl
    x[j] = *reinterpret_cast<const float4*>(gr + 16 * line + 4 * (t & 3));
  }
  __builtin_amdgcn_sched_barrier(0);
  const int lc = t & (kCopies - 1);
#pragma unroll
  for (int j = 0; j < kRounds; ++j) {
    const int64_t i = (int64_t)p * kPreLines + j * 64 + (t >> 2);
    if (i >= ns) continue;  // past the sample (rows with fewer lines than a full sample)
    const float v[4] = {x[j].x, x[j].y, x[j].z, x[j].w};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint32_t key = key_of(v[c]);
      if (key != 0) {
        const uint32_t b = (key >> 23) * kCopies + lc;
        atomicAdd(&s_cnt[b], 1u);
        atomicAdd(&s_sig[b], (unsigned long long)key_sig(key));
      }
    }
  }
  __syncthreads();
  uint64_t cnt = 0, sg = 0;
#pragma unroll
  for (int k = 0; k < kCopies; ++k) {
    cnt += s_cnt[t * kCopies + k];
    sg += s_sig[t * kCopies + k];
  }
  if (cnt) {
    PreHist* h = pre_of(a, row);
    atomicAdd((unsigned long long*)&h->cnt[t], (unsigned long long)cnt);
    atomicAdd((unsigned long long*)&h->sig[t], (unsigned long long)sg);
  }
}

// LDS of the band prediction.
struct BandLds {
  double w[kNT / 64];
  uint64_t k[kNT / 64];
  int ired[kNT / 64];
  double ge;   // the sample's G at the lower edge of the binade of 1/lambda*
  double ge1;  // and at the lower edge of the next binade up
};
// G within this fraction of B at that edge: 1/lambda* may lie in the binade below.
constexpr double kBandNear = 0.125;

// The candidate band of a row, predicted from its sample histogram identically by every
// workgroup of the statistics pass (same data, same order of operations). With f = the row's
// length over the sampled count, the sums are scaled sample sums. Every threshold a solver will
// refine lies in [1/lambda*, 1/lambda_0]: 1/lambda_0 = S / B (Algorithm 3's start), and the exact
// 1/lambda* is where G(tau) = #{a >= tau} + (sum of the a < tau) / tau falls to B (Proposition 1:
// sum min(lambda a, 1) = B); G decreases in tau, so at binade edges its crossing gives the binade
// e* of 1/lambda*. The exact solver refines the binade of 1/lambda*, or the next occupied one
// above it when no key of that binade lies above 1/lambda* (only when the crossing is at its top),
// so its band is e*, with e* - 1 or e* + 1 too when the sample's G at e*'s lower or upper edge is
// within kBandNear of B (the sample may have misplaced the crossing); the greedy solver's
// thresholds run from 1/lambda_0 = S / B down towards 1/lambda*, so its band reaches up to the
// binade of 1.25 S / B (slack for the sample's estimate of S). Whole binades, so every refinement
// window inside the band is complete. No band when B = 0 or nothing was sampled. Threads 0..255
// own one binade each; every thread receives the result.
GS_DI void cand_band(const Args& a, const PreHist* ph, double B, int64_t len, BandLds& sm, uint32_t& blo,
                     uint32_t& bhi) {
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  uint64_t c = 0;
  double w = 0.0;
  if (t < kB1) {
    c = ph->cnt[t];
    w = c ? ldexp((double)ph->sig[t], binade_shift(t) - 149) : 0.0;
  }
  // inclusive suffix sums over binades (count and value sum of the binades >= t)
  uint64_t kc = c;
  double wc = w;
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t ky = __shfl_down(kc, (unsigned)o);
    const double wy = __shfl_down(wc, (unsigned)o);
    if (lane + o < 64) {
      kc += ky;
      wc += wy;
    }
  }
  if (lane == 0) {
    sm.k[wv] = kc;
    sm.w[wv] = wc;
  }
  __syncthreads();
  double tot = 0.0;
  for (int i = 0; i < kB1 / 64; ++i) tot += sm.w[i];
  for (int i = wv + 1; i < kB1 / 64; ++i) {
    kc += sm.k[i];
    wc += sm.w[i];
  }
  const double f = (double)len / (16.0 * (double)pre_lines(len));
  // the highest occupied binade of the sample
  int top = (t < kB1 - 1 && c) ? t : -1;
  for (int o = 32; o > 0; o >>= 1) top = max(top, __shfl_xor(top, o));
  if (lane == 0) sm.ired[wv] = top;
  __syncthreads();
  top = -1;
  for (int i = 0; i < kNT / 64; ++i) top = max(top, sm.ired[i]);
  __syncthreads();
  int best = -1;
  double G = 0.0;
  if (t >= 1 && t < kB1 - 1 && B > 0.0 && tot > 0.0) {
    // G at the binade's lower edge lo = 2^(t - 127): keys >= lo count whole, the rest by value / lo
    const double lo = ldexp(1.0, t - 127);
    G = f * ((double)kc + (tot - wc) / lo);
    if (G >= B) best = t;
  }
  for (int o = 32; o > 0; o >>= 1) best = max(best, __shfl_xor(best, o));
  if (lane == 0) sm.ired[wv] = best;
  __syncthreads();
  int e = -1;
  for (int i = 0; i < kNT / 64; ++i) e = max(e, sm.ired[i]);
  if (t == e) sm.ge = G;
  if (t == e + 1) sm.ge1 = G;
  __syncthreads();
  blo = bhi = 0;
  // Nothing looks capped (B times the sample's largest magnitude, bounded by its binade's top,
  // below half the estimated sum): the solvers should need no window, so no band is collected (a
  // row the sample misjudged refines over the row).
  const bool uncapped = top >= 0 && B * ldexp(1.0, top - 126) <= 0.5 * f * tot;
  if (e >= 1 && B > 0.0 && tot > 0.0 && !uncapped) {
    const uint32_t elo = (uint32_t)e - (sm.ge < (1.0 + kBandNear) * B ? 1u : 0u);
    uint32_t ehi = (uint32_t)e + (sm.ge1 >= (1.0 - kBandNear) * B ? 1u : 0u);
    if (a.solver == GSPAR_GREEDY) {
      const double t0 = 1.25 * f * tot / B;
      const uint32_t e0 = t0 < 3.0e38 ? (key_of((float)t0) >> 23) : 254u;
      ehi = e0 > ehi ? e0 : ehi;
    }
    blo = elo << 23;
    bhi = (ehi + 1) << 23;
    if (bhi > kKeyInf) bhi = kKeyInf;
  }
  __syncthreads();
}

// Streaming statistics pass. Grid: rows * nb workgroups of kNT threads. Each builds an LDS
// histogram over binades (count, exact significand sum, maximum key), kept in kLaneCopies copies
// by lane to spread same-address LDS atomics, and adds its nonempty bins into one of the row's kC1
// global copies (chosen by workgroup index) with atomics. k_solve runs next.
template <bool VEC, bool SQ, bool CAND>
__global__ void __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(4))) k_stats(Args a) {
  static_assert(VEC || !CAND, "candidates are collected with whole waves (vector loads)");
  __shared__ StatsLdsT<SQ> sm_st;
  StatsLdsT<SQ>& sm = sm_st;
  __shared__ BandLds s_band;
  // candidate band: per-wave buffers of collected keys, and the workgroup's region count
  __shared__ uint32_t s_cand[CAND ? kNT / 64 : 1][CAND ? 64 * kCandLane : 1];
  __shared__ uint32_t s_rcnt;
  __shared__ unsigned long long s_rbase;
  int64_t row, blk;
  if (!hist_block(a, row, blk)) return;
  int64_t base, len;
  row_span(a, row, base, len);
  const int64_t beg = blk * a.chunk;
  if (beg >= len) return;  // past the end of a shorter segment
  uint32_t blo = 0, bhi = 0;
  if constexpr (CAND) {
    cand_band(a, pre_of(a, row), ctl_of(a, row)->B, len, s_band, blo, bhi);
    if (blk == 0 && threadIdx.x == 0) {
      RowCtl* c = ctl_of(a, row);
      c->band_lo = blo;
      c->band_hi = bhi;
    }
  }
  // zero keys are never candidates (no window counts them): the band starts at key 1 at least
  const uint32_t blo1 = blo ? blo : 1u;
  const uint32_t bspan = bhi > blo1 ? bhi - blo1 : 0u;
  const int lane = threadIdx.x & 63;
  // Collected keys are buffered per lane in LDS (kCandLane slots, no cross-lane work per group).
  // When some lane could not take a whole group's keys the wave flushes every lane's buffer into
  // this workgroup's own region of the row's candidate buffer, at a place taken from an LDS
  // counter, lanes in order by a wave prefix; keys that would pass the region's end are dropped and
  // the region is marked overflowed, so the first solve does not use the band.
  uint32_t* const lbuf = &s_cand[CAND ? threadIdx.x >> 6 : 0][CAND ? lane * kCandLane : 0];
  uint32_t lcnt = 0;
  if (CAND && threadIdx.x == 0) s_rcnt = 0;
  auto flush = [&]() {
    uint32_t wtot;
    const uint32_t pre = wave_prefix_bits<3>(lcnt, wtot);
    uint32_t b0 = 0;
    if (lane == 0) b0 = atomicAdd(&s_rcnt, wtot);
    const uint32_t b = (uint32_t)__shfl((int)b0, 0) + pre;
    uint32_t* __restrict__ dst = creg_of(a, row) + blk * a.cand_region;
    for (uint32_t j = 0; j < lcnt; ++j)
      if ((int64_t)b + j < a.cand_region) dst[b + j] = lbuf[j];
    lcnt = 0;
  };
  for (int b = threadIdx.x; b < kB1 * kLaneCopies; b += kNT) {
    sm.pk[b] = 0;
    sm.mx[b] = 0;
    if constexpr (SQ) {
      sm.qh[b] = 0;
      sm.ql[b] = 0;
    }
  }
  __syncthreads();
  const float* __restrict__ gr = a.g + base;
  const int64_t end = min(len, beg + a.chunk);
  const uint32_t lc = threadIdx.x & (kLaneCopies - 1);
  auto hist = [&](const float v[4]) {
    // the group's additions first (atomics without return), then its four bin maxima read
    // together: one LDS round trip per group. The bin maximum only grows, so a read that already
    // covers the key skips the atomic. Zero keys (also the coordinates outside [beg, end), read as
    // 0) add nothing, and their bin-0 reads are not acted on.
    uint32_t key[4], f[4], cur[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      key[c] = key_of(v[c]);
      f[c] = (key[c] >> 23) * kLaneCopies + lc;
      if (key[c] != 0) {
        atomicAdd(&sm.pk[f[c]], (unsigned long long)((1ull << 44) + key_sig(key[c])));
        if constexpr (SQ) {
          const uint64_t m = key_sig(key[c]), m2 = m * m;
          atomicAdd(&sm.qh[f[c]], (unsigned long long)(m2 >> 24));
          atomicAdd(&sm.ql[f[c]], (unsigned long long)(m2 & 0xFFFFFFu));
        }
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) cur[c] = sm.mx[f[c]];
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (key[c] > cur[c]) atomicMax(&sm.mx[f[c]], key[c]);
  };
  // the candidate band's keys of a group into the lane's buffer (room for four made first); a wave
  // whose groups all lie below the band (most of them) skips the group
  auto collect = [&](const float v[4]) {
    const uint32_t kmax = max(max(key_of(v[0]), key_of(v[1])), max(key_of(v[2]), key_of(v[3])));
    if (!__ballot(kmax >= blo1)) return;
    if (__ballot(lcnt > (uint32_t)(kCandLane - 4))) flush();
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint32_t key = key_of(v[c]);
      if (key - blo1 < bspan) lbuf[lcnt++] = key;
    }
  };
  // rows long enough for a candidate band (2^25 coordinates and more) keep 8 loads per lane in flight,
  // shorter ones 4 (on 2^28 coordinates 8 save about 4 microseconds per pass; on 2.5 * 10^7 and
  // fewer they cost 1-3)
  constexpr int kU = CAND ? 8 : 4;
  if (CAND && bspan != 0) {
    stream_groups<VEC, kU, kNT>(gr, beg, end, [&](int64_t, const float v[4], uint32_t) {
      hist(v);
      collect(v);
    });
  } else {
    // no band (or none predicted for this row): the plain statistics loop
    stream_groups<VEC, kU, kNT>(gr, beg, end, [&](int64_t, const float v[4], uint32_t) { hist(v); });
  }
  if constexpr (CAND) {
    if (__ballot(lcnt != 0)) flush();
    __syncthreads();
    // move the region to the row's compact list: one reservation per workgroup (a region that
    // overflowed reserves past the list's capacity, which disables the band)
    if (bspan != 0) {
      const uint32_t n = s_rcnt;
      if (threadIdx.x == 0) {
        const unsigned long long want = (int64_t)n <= a.cand_region ? n : (unsigned long long)a.lay.cand_cap + 1;
        s_rbase = want ? atomicAdd(&ccnt_of(a, row)->v, want) : 0ull;
      }
      __syncthreads();
      const uint64_t b = s_rbase;
      if ((int64_t)n <= a.cand_region && b + n <= (uint64_t)a.lay.cand_cap) {
        const uint32_t* __restrict__ src = creg_of(a, row) + blk * a.cand_region;
        uint32_t* __restrict__ out = cand_of(a, row) + b;
        for (uint32_t j = threadIdx.x; j < n; j += kNT) out[j] = src[j];
      }
    }
  }
  __syncthreads();
  // flush one binade per thread into copy (blk mod kC1)
  if (threadIdx.x < kB1) {
    const int e = threadIdx.x;
    uint64_t cnt = 0, sg = 0;
    uint32_t mx = 0;
#pragma unroll
    for (int j = 0; j < kLaneCopies; ++j) {
      const uint64_t p = sm.pk[e * kLaneCopies + j];
      cnt += p >> 44;
      sg += p & ((1ull << 44) - 1);
      mx = max(mx, sm.mx[e * kLaneCopies + j]);
    }
    if (cnt) {
      Hist1* h = h1_of(a, row, (int)(blk % kC1));
      atomicAdd((unsigned long long*)&h->cnt[e], (unsigned long long)cnt);
      atomicAdd((unsigned long long*)&h->sig[e], (unsigned long long)sg);
      atomicMax(&h->mx[e], mx);
      if constexpr (SQ) {
        uint64_t qh = 0, ql = 0;
#pragma unroll
        for (int j = 0; j < kLaneCopies; ++j) {
          qh += sm.qh[e * kLaneCopies + j];
          ql += sm.ql[e * kLaneCopies + j];
        }
        H1Q* q = h1q_of(a, row, (int)(blk % kC1));
        atomicAdd((unsigned long long*)&q->qh[e], (unsigned long long)qh);
        atomicAdd((unsigned long long*)&q->ql[e], (unsigned long long)ql);
      }
    }
  }
}

// Refinement pass over one window of keys, for the rows whose solver asked for one.
template <bool VEC, bool SQ>
__global__ void __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(4))) k_refine(Args a) {
  __shared__ WinLdsT<SQ> sm_w;
  WinLdsT<SQ>& sm = sm_w;
  int64_t row, blk;
  if (!hist_block(a, row, blk)) return;
  const RowCtl* ctl = ctl_of(a, row);
  const uint32_t need = ctl->need;
  if (need != 2 && need != 3) return;
  int64_t base, len;
  row_span(a, row, base, len);
  const float* __restrict__ gr = a.g + base;
  int64_t beg = blk * a.chunk, end = min(len, beg + a.chunk);
  // the window lies in the candidate band: the row's collected keys, read as the non-negative
  // floats they are, in equal shares (whole groups of 4, at least kCandShare keys, at most
  // kCandGroups shares) by the first of the row's workgroups
  const bool from_cand = ctl->src != 0;
  if (from_cand) {
    const int64_t n = (int64_t)ctl->cand_n;
    const int64_t groups = min((int64_t)a.nb, kCandGroups);
    const int64_t share = max(kCandShare, (((n + groups - 1) / groups) + 3) & ~(int64_t)3);
    beg = blk * share;
    end = min(n, beg + share);
    gr = reinterpret_cast<const float*>(cand_of(a, row));
  }
  if (beg >= end) return;  // past the end of a shorter segment, or of the candidates
  uint32_t lo, shift;
  int nbins;
  const int cp = (int)(blk % kC23);
  WinHist* h = win_of(a, row, cp);
  if (need == 2) {
    lo = ctl->l2exp << 23;
    shift = 11;
    nbins = kB2;
  } else {
    lo = ctl->l3base;
    shift = 0;
    nbins = kB3;
  }
  const uint32_t span = (uint32_t)nbins << shift;
  // level 2 also keeps bin minima and counts the window's keys >= qkey directly (qkey lies in the
  // window when set; kNone matches no key)
  const bool l2 = need == 2;
  const uint32_t qkey = l2 ? ctl->qkey : kNone;
  // the greedy solver's last query needs the direct count only: no bins are built or flushed
  const bool bins = !(l2 && ctl->qonly);
  // the variance-budget solver's level-2 windows also sum squared significands (level 3 has one
  // key per bin, whose square follows from the count)
  const bool sq2 = SQ && l2 && bins;
  for (int b = threadIdx.x; bins && b < nbins; b += kNT) {
    sm.pk[b] = 0;
    sm.mx[b] = 0;
    sm.mnc[b] = 0;
    if constexpr (SQ) {
      sm.qh[b] = 0;
      sm.ql[b] = 0;
    }
  }
  __syncthreads();
  uint64_t qc = 0, qs = 0;
  auto visit = [&](int64_t, const float v[4], uint32_t) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint32_t key = key_of(v[c]);
      const uint32_t rel = key - lo;
      if (key != 0 && rel < span) {
        const uint32_t b = rel >> shift;
        const uint64_t sg = key_sig(key);
        if (bins) {
          atomicAdd(&sm.pk[b], (unsigned long long)((1ull << 44) + sg));
          // level-2 bin extremes (fire-and-forget atomics: a read of the bin first would make
          // every key wait on the LDS); a level-3 bin is one key, its own maximum
          if (l2) {
            atomicMax(&sm.mx[b], key);
            atomicMax(&sm.mnc[b], ~key);
          }
        }
        if (key >= qkey) {
          ++qc;
          qs += sg;
        }
        if constexpr (SQ) {
          if (sq2) {
            const uint64_t m2 = sg * sg;
            atomicAdd(&sm.qh[b], (unsigned long long)(m2 >> 24));
            atomicAdd(&sm.ql[b], (unsigned long long)(m2 & 0xFFFFFFu));
          }
        }
      }
    }
  };
  // (the variance-budget solver never collects candidates)
  if (!SQ && from_cand) stream_groups<VEC, SQ ? 4 : kCandLoads, kNT>(gr, beg, end, visit);
  else stream_groups<VEC, 4, kNT>(gr, beg, end, visit);
  if (l2) {
    for (int o = 32; o > 0; o >>= 1) {
      qc += __shfl_xor(qc, o);
      qs += __shfl_xor(qs, o);
    }
    if ((threadIdx.x & 63) == 0) {
      sm.qc[threadIdx.x >> 6] = qc;
      sm.qs[threadIdx.x >> 6] = qs;
    }
  }
  __syncthreads();
  // flush: workgroups start at different blocks of kNT bins, so they do not queue on the same
  // addresses at the same time
  static_assert(kB2 % kNT == 0 && kB3 % kNT == 0, "whole blocks of bins");
  const int nblk = bins ? nbins / kNT : 0;
  for (int i = 0; i < nblk; ++i) {
    const int b = ((i + (int)blk) % nblk) * kNT + threadIdx.x;
    const uint64_t p = sm.pk[b];
    if (p) {
      atomicAdd((unsigned long long*)&h->cnt[b], (unsigned long long)(p >> 44));
      atomicAdd((unsigned long long*)&h->sig[b], (unsigned long long)(p & ((1ull << 44) - 1)));
      atomicMax(&h->mx[b], l2 ? sm.mx[b] : lo + (uint32_t)b);
      if (l2) atomicMax(&h->mnc[b], sm.mnc[b]);
      if constexpr (SQ) {
        if (sq2) {
          WinQ* q = winq_of(a, row, cp);
          atomicAdd((unsigned long long*)&q->qh[b], (unsigned long long)sm.qh[b]);
          atomicAdd((unsigned long long*)&q->ql[b], (unsigned long long)sm.ql[b]);
        }
      }
    }
  }
  if (l2 && threadIdx.x == 0) {
    uint64_t tc = 0, ts = 0;
    for (int i = 0; i < kNT / 64; ++i) {
      tc += sm.qc[i];
      ts += sm.qs[i];
    }
    if (tc) {
      atomicAdd((unsigned long long*)&h->qcnt, (unsigned long long)tc);
      atomicAdd((unsigned long long*)&h->qsig, (unsigned long long)ts);
    }
  }
}

// The solver: one workgroup per row, after the statistics pass and after every refinement pass.
template <bool VAR>
__global__ void __launch_bounds__(kNT) k_solve(Args a) {
  __shared__ SolveLds sm;
  const int64_t row = blockIdx.x;
  if (a.seg && *segok_of(a) != 1) {
    // the workgroup maps of a segmented call do not have the launched shape: no histogram pass
    // ran and the sample pass does nothing, so the first solve skips the row and writes its results
    if (a.first && threadIdx.x == 0) {
      RowCtl* gc = ctl_of(a, row);
      RowCtl c = *gc;
      c.flags |= GSPAR_FLAG_BADSEG;
      sv_finalize(c, NAN, kKeyInf);
      *gc = c;
      if (a.nnz) a.nnz[row] = 0;
      if (a.nnz_b) a.nnz_b[row] = 0;
      if (a.inv_out) a.inv_out[row] = c.inv_lam;
      if (a.k_out) a.k_out[row] = 0;
      if (a.lam_out) a.lam_out[row] = c.lam;
      if (a.flags_out) a.flags_out[row] = c.flags;
    }
    return;
  }
  const Hists H{&sm.err, &sm.l1, &sm.w2, &sm.w3, l1t_of(a, row), h1_of(a, row), win_of(a, row),
                h1q_of(a, row), winq_of(a, row), vctl_of(a, row), ccnt_of(a, row), a.lay.cand_cap};
  int64_t base, len;
  row_span(a, row, base, len);
  solve_row<VAR>(sm, ctl_of(a, row), H, len, a.first != 0);
}

// Sampling, amplification and order-preserving compaction. Workgroup t handles tile t (kTileElems
// coordinates of one row, in row order); wave w of the workgroup owns the tile's w-th quarter and
// reads it as kTileGroups coalesced float4 loads per lane. Tile prefixes chain through a decoupled
// look-back whose status word packs (flag:2 | capped survivors:31 | survivors:31). A predecessor
// that has not published after a long back-off is counted by the waiting wave itself, so no
// ordering of workgroup dispatch is assumed and every wait ends.
constexpr uint64_t kStAgg = 1ull << 62, kStInc = 2ull << 62, kStVal = (1ull << 62) - 1;
// Look-back rounds before a waiting wave counts an unpublished predecessor itself (a build may
// lower it to exercise that path).
#ifndef GSPAR_LOOKBACK_POLLS
#define GSPAR_LOOKBACK_POLLS 4096
#endif
constexpr int kPolls = GSPAR_LOOKBACK_POLLS;
constexpr int kWaveElems = kTileElems / (kTileThreads / 64);  // coordinates per wave per tile

struct TileCtx {
  const float* row;
  int64_t d;
  double lam;
  uint32_t tcap;
  uint32_t k0, k1;
  bool live;
};

// Selection bits (bit c: coordinate 4q+c survives) and capped-survivor bits of group q, whose
// values v are given (m: bit c set when coordinate 4q+c exists).
__device__ __forceinline__ void decide_values(const TileCtx& c, int64_t q, const float v[4], uint32_t m, uint32_t& z,
                                              uint32_t& cz) {
  uint32_t x0 = (uint32_t)q, x1 = (uint32_t)((uint64_t)q >> 32), x2 = 0, x3 = 0;
  philox10(x0, x1, x2, x3, c.k0, c.k1);
  const uint32_t xr[4] = {x0, x1, x2, x3};
  z = 0;
  cz = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t key = key_of(v[k]);
    const bool capped = key >= c.tcap;
    const bool pick = capped || ((double)xr[k] * 0x1p-32 < c.lam * (double)fabsf(v[k]));
    const bool sel = c.live && ((m >> k) & 1) && key != 0 && pick;
    z |= (uint32_t)sel << k;
    cz |= (uint32_t)(sel && capped) << k;
  }
}

// The same for group q loaded here (entries past the row's end read as 0).
template <bool VEC>
__device__ __forceinline__ void decide_group(const TileCtx& c, int64_t q, float v[4], uint32_t& z, uint32_t& cz) {
  const uint32_t m = load4<VEC>(c.row, q, c.d, v);
  decide_values(c, q, v, m, z, cz);
}

// Aggregate (capped << 31 | survivors) of tile `part` computed by one wave (fallback path).
template <bool VEC>
__device__ uint64_t wave_tile_aggregate(const TileCtx& c, int64_t part, int lane) {
  uint64_t n = 0, nc = 0;
  for (int j = 0; j < kTileElems / 4 / 64; ++j) {
    const int64_t q = part * (kTileElems / 4) + j * 64 + lane;
    float v[4];
    uint32_t z, cz;
    decide_group<VEC>(c, q, v, z, cz);
    n += __popc(z);
    nc += __popc(cz);
  }
  for (int o = 32; o > 0; o >>= 1) {
    n += __shfl_xor(n, o);
    nc += __shfl_xor(nc, o);
  }
  return (nc << 31) | n;
}

// Phase 1: each lane decides kTileGroups groups of its wave's quarter (coalesced loads, one
// Philox block per group) and writes one byte per group to LDS: selection bits (low nibble) and
// sign bits (high nibble); capped survivors (emitted unscaled) append their value to the deciding
// lane's own LDS row, and a second byte array holds per group their bits and the lane's running
// count of them. The wave totals give the tile aggregate, published at once; wave 0 then looks back
// for the tile's prefix.
// Phase 2: thread t owns the tile's groups [16t, 16t + 16), i.e. 64 consecutive coordinates
// inside its own wave's quarter, so its survivors are contiguous in the output: one prefix over
// the wave's lanes places it, and it writes only its own set bits (for up to kStageEmit survivors
// per wave through an LDS staging area that the wave then stores with consecutive lanes on
// consecutive slots). Phase 2 reads no global memory (a load would wait for every store issued
// before it), except in a wave where some lane kept more capped values than its LDS row holds (a
// separate instantiation).
// Capped survivors' values are kept in LDS by the phase-1 lane that decided them, kLaneCap per
// lane and tile (rows padded to kLaneStride floats so that lanes fall on different banks); a wave
// with a lane past that reads its capped values from global memory in phase 2.
constexpr int kLaneCap = 8;
constexpr int kLaneStride = kLaneCap + 1;
constexpr int kSampleBatch = 8;  // float4 loads in flight per lane in the sampling pass
constexpr int kDenseEmit = 1024;  // survivors of a wave's quarter tile (of 4096) above which emission goes by groups
// Survivors of a wave's quarter tile up to which emission is staged in LDS: 4-byte entries in the
// quarter's 2 KB of code and capped-survivor bytes, free once every lane has read its own.
constexpr int kStageEmit = 512;
static_assert(kTileGroups % kSampleBatch == 0 && kTileGroups == 16, "tile shape");
static_assert(2 * kStageEmit <= kWaveElems / 4 && kTileElems <= 65536 && 64 * kLaneStride <= 1024,
              "a staged entry: 16-bit tile coordinate, 10-bit capped-value place, within the quarter's bytes");
// Below this lambda, lambda * 2^32 * |g| could round differently from (lambda * |g|) * 2^32.
constexpr double kLamScaledMin = 0x1p-900;

// Whole-tile decisions with the scaled threshold: coordinate i survives iff
// x_i < t_i = fl(lambda * 2^32 * |g_i|), which equals the comparison x_i < fl(lambda * |g_i|) * 2^32
// (exact scaling by a power of two) for lambda = 0 or lambda >= kLamScaledMin. A capped coordinate
// (key >= tcap, p_i = 1) always passes that test: either fl(lambda a) >= 1, so t_i >= 2^32 > x_i,
// or it lies above the exact criterion's value, where lambda a > 1 in exact arithmetic and the few
// roundings of lambda keep t_i above 2^32 - 1 >= x_i. So the capped bits are needed only in groups
// whose largest threshold reaches 2^32 - 1, and there they are the key test itself.
__device__ __forceinline__ void decide_fast(int64_t q, const float v[4], double lam32, uint32_t tcap, uint32_t k0,
                                            uint32_t k1, uint32_t& z, uint32_t& cz) {
  // rows are shorter than 2^31 coordinates, so the counter's high word floor(i/4) >> 32 is 0; with
  // that known the first rounds fold into fewer vector operations
  uint32_t x0 = (uint32_t)q, x1 = 0, x2 = 0, x3 = 0;
  philox10(x0, x1, x2, x3, k0, k1);
  const uint32_t xr[4] = {x0, x1, x2, x3};
  double t[4];
  z = 0;
  cz = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    t[k] = lam32 * (double)fabsf(v[k]);
    z |= (uint32_t)((double)xr[k] < t[k]) << k;
  }
  // capped coordinates are rare: test the group's largest threshold first
  if (fmax(fmax(t[0], t[1]), fmax(t[2], t[3])) >= 0x1p32 - 1.0) {
#pragma unroll
    for (int k = 0; k < 4; ++k) cz |= (uint32_t)(key_of(v[k]) >= tcap) << k;
  }
}

// A group's code byte: the selection bits z (bits 0-3) and the signs of its four values (bits 4-7).
// v_perm_b32's sign-replicating selectors (9: bit 31 of the low word of the pair, 11: of the high
// word) turn each sign into a 0x00 / 0xFF byte, one bit of each byte is kept, and v_sad_u8 adds
// the four bytes to z.
__device__ __forceinline__ uint32_t group_code(const float v[4], uint32_t z) {
  const uint32_t s01 = __builtin_amdgcn_perm(__float_as_uint(v[1]), __float_as_uint(v[0]), 0x0C0C0B09u);
  const uint32_t s23 = __builtin_amdgcn_perm(__float_as_uint(v[3]), __float_as_uint(v[2]), 0x0B090C0Cu);
  return __builtin_amdgcn_sad_u8((s01 | s23) & 0x80402010u, 0u, z);
}

// The nibbles of the eight bytes of (w0, w1), byte 0 of w0 first: lo holds their low nibbles and hi
// their high nibbles, byte k's at bits [4k, 4k + 4). v_perm_b32 gathers the even and the odd bytes
// (selectors 0-7 pick a byte of the pair, w1 above w0), and one bit-field insert interleaves each.
__device__ __forceinline__ void byte_nibbles(uint32_t w0, uint32_t w1, uint32_t& lo, uint32_t& hi) {
  const uint32_t ev = __builtin_amdgcn_perm(w1, w0, 0x06040200u);  // bytes 6, 4, 2, 0
  const uint32_t od = __builtin_amdgcn_perm(w1, w0, 0x07050301u);  // bytes 7, 5, 3, 1
  lo = (ev & 0x0F0F0F0Fu) | ((od << 4) & 0xF0F0F0F0u);
  hi = ((ev >> 4) & 0x0F0F0F0Fu) | (od & 0xF0F0F0F0u);
}

template <bool VEC, bool HYB, int K>
__global__ void __launch_bounds__(kTileThreads) k_sample(Args a) {
  __shared__ float s_capl[K][kTileThreads / 64][64 * kLaneStride];
  __shared__ alignas(16) uint8_t s_code[K][kTileElems / 4];  // per group: selection | sign << 4
  // per group: capped-survivor bits | the deciding lane's capped count before the group << 4
  __shared__ alignas(16) uint8_t s_capb[K][kTileElems / 4];
  __shared__ uint32_t s_wsel[K][kTileThreads / 64];
  __shared__ uint32_t s_wcap[K][kTileThreads / 64];
  __shared__ uint32_t s_wcl[K][kTileThreads / 64];
  __shared__ uint64_t s_excl;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  // workgroup -> K consecutive tiles [part0, part0 + nk) of one row. A row has
  // max(1, ceil(length / kTileElems)) tiles, all lay.tiles for rows of a strided batch; the
  // workgroups past a shorter segment's tiles have nothing to do (no later tile of the row waits on
  // them, and its last tile writes the row's results).
  int64_t row, part0;
  if (!a.seg) {
    const int64_t wpr = (a.lay.tiles + K - 1) / K;  // workgroups per row
    row = blockIdx.x / wpr;
    part0 = (blockIdx.x % wpr) * K;
  } else {
    // the map built by k_init holds only workgroups with tiles; a map that does not have the
    // launched shape leaves every row to the first solve
    if (*segok_of(a) != 1) return;
    const uint64_t e = reinterpret_cast<const uint64_t*>(a.ws + a.lay.tmap)[blockIdx.x];
    row = (int64_t)(e >> 32);
    part0 = (int64_t)(e & 0xFFFFFFFFu) * K;
  }
  TileCtx c;
  int64_t base;
  row_span(a, row, base, c.d);
  const int64_t rtiles = c.d > kTileElems ? (c.d + kTileElems - 1) / kTileElems : 1;
  if (part0 >= rtiles) return;
  const int nk = (int)min((int64_t)K, rtiles - part0);
  const int64_t t0 = row * a.lay.tiles + part0;  // status word of the first tile
  const RowCtl* ctl = ctl_of(a, row);
  c.row = a.g + base;
  c.lam = ctl->lam;
  c.tcap = ctl->tcap;
  c.live = ctl->done && !(ctl->flags & (GSPAR_FLAG_NONFINITE | GSPAR_FLAG_BADRHO | GSPAR_FLAG_BADSEG | kFlagInternal));
  const uint64_t seed = a.seed_dev ? a.seed_dev[row] : a.seed;
  c.k0 = (uint32_t)seed;
  c.k1 = (uint32_t)(seed >> 32);
  const float inv = ctl->inv_lam;
  const bool fast = c.live && (c.lam == 0.0 || c.lam >= kLamScaledMin);
  const double lam32 = c.lam * 0x1p32;
  uint64_t* st = status_of(a);
  // group j of this lane in a tile is tile group wv * (kWaveElems / 4) + 64 j + lane
  const int tg0 = wv * (kWaveElems / 4) + lane;
  uint64_t agg[K];  // per tile: (capped survivors << 31) | survivors
  // capped-survivor bytes start at zero, so phase 1 writes only the groups that have some
#pragma unroll
  for (int kk = 0; kk < K; ++kk) *reinterpret_cast<uint4*>(&s_capb[kk][16 * tid]) = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();

#pragma unroll
  for (int kk = 0; kk < K; ++kk) {
    if (kk >= nk) break;
    __builtin_amdgcn_sched_barrier(0);  // keep each tile's loads in its own iteration
    // phase 1 of tile part0 + kk
    const int64_t part = part0 + kk;
    const int64_t q0 = part * (kTileElems / 4) + tg0;
    uint32_t nsel = 0;
    uint32_t run = 0;  // this lane's capped survivors in the tile so far
    float* const capl = &s_capl[kk][wv][lane * kLaneStride];
    // cz lies inside z: a capped coordinate always passes its selection test
    auto record = [&](int j, const float v[4], uint32_t z, uint32_t cz) {
      s_code[kk][tg0 + 64 * j] = (uint8_t)group_code(v, z);
      nsel += (uint32_t)__popc(z);
      if (cz) {
        s_capb[kk][tg0 + 64 * j] = (uint8_t)(cz | (min(run, 15u) << 4));
        // every value goes to the next free slot (the row's pad slot once the row is full), and
        // only a capped one takes it, so no lane branches per coordinate
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          capl[min(run, (uint32_t)kLaneCap)] = v[k];
          run += (cz >> k) & 1u;
        }
      }
    };
    if (VEC && fast && (part + 1) * (int64_t)kTileElems <= c.d) {
      // whole tile inside the row: kSampleBatch unconditional loads in flight per lane
#pragma unroll
      for (int jb = 0; jb < kTileGroups; jb += kSampleBatch) {
        float4 x[kSampleBatch];
#pragma unroll
        for (int u = 0; u < kSampleBatch; ++u)
          x[u] = load_stream(c.row + 4 * (q0 + 64 * (jb + u)));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kSampleBatch; ++u) {
          const float v[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
          uint32_t z, cz;
          decide_fast(q0 + 64 * (jb + u), v, lam32, c.tcap, c.k0, c.k1, z, cz);
          record(jb + u, v, z, cz);
        }
      }
    } else {
      for (int j = 0; j < kTileGroups; ++j) {
        float v[4];
        uint32_t z = 0, cz = 0;
        // groups past the row's end (the tail of the last tile, and whole tiles past the end of a
        // shorter segment) hold no coordinates
        if (c.live && 4 * (q0 + 64 * j) < c.d) decide_group<VEC>(c, q0 + 64 * j, v, z, cz);
        else v[0] = v[1] = v[2] = v[3] = 0.0f;
        record(j, v, z, cz);
      }
    }
    const bool lane_over = run > (uint32_t)kLaneCap;
    uint32_t ncap = run;
    for (int o = 32; o > 0; o >>= 1) {
      nsel += __shfl_xor(nsel, o);
      ncap += __shfl_xor(ncap, o);
    }
    const bool wave_over = __ballot(lane_over) != 0;
    if (lane == 0) {
      s_wsel[kk][wv] = nsel;
      s_wcap[kk][wv] = ncap;
      s_wcl[kk][wv] = wave_over ? 1u : 0u;
    }
    __syncthreads();
    uint32_t tsel = 0, tcp = 0;
    for (int i = 0; i < kTileThreads / 64; ++i) {
      tsel += s_wsel[kk][i];
      tcp += s_wcap[kk][i];
    }
    agg[kk] = ((uint64_t)tcp << 31) | tsel;
    // publish at once: a row's first tile its inclusive prefix, every other tile its aggregate
    if (tid == 0)
      __hip_atomic_store(&st[t0 + kk], (part == 0 ? kStInc : kStAgg) | agg[kk], __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  }

  // decoupled look-back for the exclusive prefix of the first tile within its row
  if (part0 == 0) {
    if (tid == 0) s_excl = 0;
  } else {
    if (wv == 0) {
      const int64_t t = t0;
      const int64_t first = t - part0;
      int64_t look = t - 1;
      uint64_t ex = 0;
      while (true) {
        const int64_t i = look - lane;
        uint64_t sw = kStInc;
        if (i >= first) sw = __hip_atomic_load(&st[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // wait only for the predecessors between this tile and the nearest one whose inclusive
        // prefix is published (that boundary can only move closer while waiting)
        uint64_t incl_mask, missing;
        int stop;
        for (int polls = 0;; ++polls) {
          incl_mask = __ballot((sw >> 62) == 2);
          stop = incl_mask ? (__ffsll((unsigned long long)incl_mask) - 1) : 63;
          missing = __ballot((sw >> 62) == 0 && lane <= stop);
          if (!missing || polls == kPolls) break;
          __builtin_amdgcn_s_sleep(4);
          if ((sw >> 62) == 0 && lane <= stop) sw = __hip_atomic_load(&st[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        // predecessors up to `stop` that never published: count them here
        while (missing) {
          const int m = __ffsll((unsigned long long)missing) - 1;
          const uint64_t val = wave_tile_aggregate<VEC>(c, (look - m) - first, lane);
          if (lane == m) sw = kStAgg | val;
          missing &= missing - 1;
        }
        uint64_t contrib = lane <= stop ? (sw & kStVal) : 0;
        for (int o = 32; o > 0; o >>= 1) contrib += __shfl_xor(contrib, o);
        ex += contrib;
        if (incl_mask) break;
        look -= 64;
      }
      if (lane == 0) {
        s_excl = ex;
        uint64_t run = ex;
        for (int kk = 0; kk < nk; ++kk) {
          run += agg[kk];
          __hip_atomic_store(&st[t0 + kk], kStInc | run, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
  }
  if (part0 == 0 && tid == 0) {
    // the row's first workgroup: its later tiles' inclusive prefixes follow from its own aggregates
    uint64_t run = agg[0];
    for (int kk = 1; kk < nk; ++kk) {
      run += agg[kk];
      __hip_atomic_store(&st[t0 + kk], kStInc | run, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  uint64_t excl = s_excl;

  // phase 2, tile by tile: thread tid owns tile groups [16 tid, 16 tid + 16) (bit b of its masks
  // is tile coordinate 64 tid + b)
#pragma unroll
  for (int kk = 0; kk < K; ++kk) {
    if (kk >= nk) break;
    __builtin_amdgcn_sched_barrier(0);
    const int64_t part = part0 + kk;
    uint32_t wbase = 0, wbase_cap = 0;
    for (int i = 0; i < wv; ++i) {
      wbase += s_wsel[kk][i];
      wbase_cap += s_wcap[kk][i];
    }
    const int64_t e0 = part * (int64_t)kTileElems + 64 * tid;
    uint64_t sm = 0, nm = 0, cm = 0;  // selected, negative, capped-and-selected coordinates
    uint32_t cr = 0;                  // hybrid: rank of this thread's first capped survivor in its wave
    uint32_t cwd[4] = {0u, 0u, 0u, 0u};  // this thread's 16 capped-survivor bytes
    if (s_wsel[kk][wv]) {
      const uint4 cw = *reinterpret_cast<const uint4*>(&s_code[kk][16 * tid]);
      uint32_t s0, s1, n0, n1;
      byte_nibbles(cw.x, cw.y, s0, n0);
      byte_nibbles(cw.z, cw.w, s1, n1);
      sm = ((uint64_t)s1 << 32) | s0;
      nm = ((uint64_t)n1 << 32) | n0;
      if (s_wcap[kk][wv]) {
        const uint4 bw = *reinterpret_cast<const uint4*>(&s_capb[kk][16 * tid]);
        cwd[0] = bw.x;
        cwd[1] = bw.y;
        cwd[2] = bw.z;
        cwd[3] = bw.w;
        uint32_t c0, c1, u0, u1;
        byte_nibbles(bw.x, bw.y, c0, u0);
        byte_nibbles(bw.z, bw.w, c1, u1);
        cm = ((uint64_t)c1 << 32) | c0;
        if constexpr (HYB) {
          uint32_t ctot;
          cr = wave_prefix_bits<7>((uint32_t)__popcll(cm), ctot);
        }
      }
      const bool lds_values = s_wcl[kk][wv] == 0;
      // the value of capped survivor b (0..63) of this thread's coordinates: its group 16 tid + b/4
      // was decided by phase-1 lane (16 tid + b/4) mod 64, whose list holds it after the lane's
      // earlier capped survivors (the byte's high nibble) and the group's lower ones
      auto capval = [&](int b) -> float {
        const int gi = b >> 2;
        const uint32_t cb = (cwd[gi >> 2] >> (8 * (gi & 3))) & 0xFFu;
        const uint32_t slot = (cb >> 4) + (uint32_t)__popc(cb & ((1u << (b & 3)) - 1u));
        return s_capl[kk][wv][((16 * tid + gi) & 63) * kLaneStride + slot];
      };
      if constexpr (!HYB) {
        uint32_t wtot;
        uint64_t pos = (excl & 0x7FFFFFFFull) + wbase + wave_prefix_bits<7>((uint32_t)__popcll(sm), wtot);
        int32_t* __restrict__ oi = a.idx + row * a.cap;
        float* __restrict__ ov = a.val + row * a.cap;
        auto emit = [&](auto from_lds) {
          uint64_t m = sm;
          while (m) {
            const int b = __ffsll((unsigned long long)m) - 1;
            const uint64_t bit = 1ull << b;
            float val = (nm & bit) ? -inv : inv;
            if (cm & bit) {
              if constexpr (decltype(from_lds)::value) val = capval(b);
              else val = c.row[e0 + b];
            }
            if ((int64_t)pos < a.cap) {
              oi[pos] = (int32_t)(e0 + b);
              ov[pos] = val;
            }
            ++pos;
            m &= m - 1;
          }
        };
        const uint64_t wave_end = (excl & 0x7FFFFFFFull) + wbase + s_wsel[kk][wv];
        if (lds_values && s_wsel[kk][wv] <= (uint32_t)kStageEmit && wave_end <= (uint64_t)a.cap &&
            wave_end <= ((uint64_t)1 << 30)) {
          // the common case, staged: every survivor of the wave within the capacity and its capped
          // values in the lanes' LDS rows. Each lane writes its survivors' entries (tile coordinate,
          // 16 bits; value code: sign in bit 15, or bit 14 and the capped value's place in the LDS
          // rows) at its prefix in the wave's quarter of the code and capped-survivor bytes, which
          // every lane of the wave has read by now (LDS operations of a wave complete in order);
          // then lane l writes entries l, l + 64, ... so that each store covers consecutive
          // addresses, instead of one address per lane far apart.
          uint16_t* const si = reinterpret_cast<uint16_t*>(&s_code[kk][wv * (kWaveElems / 4)]);
          uint16_t* const sc = reinterpret_cast<uint16_t*>(&s_capb[kk][wv * (kWaveElems / 4)]);
          const uint64_t wpos = (excl & 0x7FFFFFFFull) + wbase;  // the wave's first output slot
          const uint32_t lpre = (uint32_t)(pos - wpos);
          __builtin_amdgcn_wave_barrier();
          uint32_t j = lpre;
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            uint32_t m = (uint32_t)(sm >> (32 * h));
            const uint32_t neg = (uint32_t)(nm >> (32 * h));
            const uint32_t c0 = (uint32_t)(64 * tid + 32 * h);
            while (m) {
              const int b = __builtin_ctz(m);
              si[j] = (uint16_t)(c0 + b);
              sc[j] = (uint16_t)(((neg >> b) & 1u) << 15);
              ++j;
              m &= m - 1u;
            }
          }
          uint64_t mc = cm;
          while (mc) {
            const int b = __ffsll((unsigned long long)mc) - 1;
            const uint32_t below = (uint32_t)__popcll(sm & ((1ull << b) - 1ull));
            const int gi = b >> 2;
            const uint32_t cb = (cwd[gi >> 2] >> (8 * (gi & 3))) & 0xFFu;
            const uint32_t slot = (cb >> 4) + (uint32_t)__popc(cb & ((1u << (b & 3)) - 1u));
            sc[lpre + below] = (uint16_t)(0x4000u | (uint32_t)(((16 * tid + gi) & 63) * kLaneStride + slot));
            mc &= mc - 1;
          }
          __builtin_amdgcn_wave_barrier();
          const uint32_t wn = s_wsel[kk][wv];
          const float* const capw = &s_capl[kk][wv][0];
          gchar* __restrict__ bi = uniform_ptr(oi) + 4u * (uint32_t)wpos;
          gchar* __restrict__ bv = uniform_ptr(ov) + 4u * (uint32_t)wpos;
          const int32_t t0c = (int32_t)(part * (int64_t)kTileElems);
          for (uint32_t i = (uint32_t)lane; i < wn; i += 64u) {
            const uint32_t x = si[i], cc = sc[i];
            const float cv = capw[cc & 0x3FFu];
            const float val = (cc & 0x4000u) ? cv : ((cc & 0x8000u) ? -inv : inv);
            GS_STORE_STREAM((GS_GLOBAL(int32_t)*)(bi + 4u * i), t0c + (int32_t)x);
            GS_STORE_STREAM((GS_GLOBAL(float)*)(bv + 4u * i), val);
          }
        } else if (lds_values && s_wsel[kk][wv] <= (uint32_t)kDenseEmit && wave_end <= (uint64_t)a.cap &&
                   wave_end <= ((uint64_t)1 << 30)) {
          // the same between kStageEmit and kDenseEmit survivors, unstaged (no store needs a bound
          // check): a first loop writes every survivor with the sign's +-1/lambda, a second
          // (capped survivors are few) overwrites the capped ones' values with g_i; both stores of
          // a value come from this lane in program order. 32-bit byte offsets from the row's
          // output arrays, masks in 32-bit halves.
          gchar* __restrict__ bi = uniform_ptr(oi);
          gchar* __restrict__ bv = uniform_ptr(ov);
          const uint32_t off0 = (uint32_t)pos * 4u;
          uint32_t off = off0;
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            uint32_t m = (uint32_t)(sm >> (32 * h));
            const uint32_t neg = (uint32_t)(nm >> (32 * h));
            const int32_t i0 = (int32_t)(e0 + 32 * h);
            while (m) {
              const int b = __builtin_ctz(m);
              *(GS_GLOBAL(int32_t)*)(bi + off) = i0 + b;
              *(GS_GLOBAL(float)*)(bv + off) = ((neg >> b) & 1u) ? -inv : inv;
              off += 4u;
              m &= m - 1u;
            }
          }
          uint64_t m = cm;
          while (m) {
            const int b = __ffsll((unsigned long long)m) - 1;
            const uint32_t below = (uint32_t)__popcll(sm & ((1ull << b) - 1ull));
            *(GS_GLOBAL(float)*)(bv + off0 + 4u * below) = capval(b);
            m &= m - 1;
          }
        } else if (s_wsel[kk][wv] > (uint32_t)kDenseEmit) {
          // many survivors: lane l takes the wave's groups 64 j + l (the order of phase 1 and of
          // this lane's capped-value row), one step j at a time, so the stores of a step fall on a
          // few consecutive lines instead of one line per lane
          const uint64_t base0 = (excl & 0x7FFFFFFFull) + wbase;
          uint32_t carry = 0;
          for (int j = 0; j < kTileGroups; ++j) {
            const int q = wv * (kWaveElems / 4) + 64 * j + lane;  // tile group (decided by this lane)
            const uint32_t code = s_code[kk][q];
            const uint32_t sel = code & 0xFu, neg = code >> 4;
            const uint32_t cb = s_capb[kk][q], cap = cb & sel;
            uint32_t stot;
            const uint32_t sp = wave_prefix_bits<3>((uint32_t)__popc(sel), stot);
            uint64_t p = base0 + carry + sp;
            const int64_t eq = part * (int64_t)kTileElems + 4 * (int64_t)q;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              if ((sel >> k) & 1) {
                float val = ((neg >> k) & 1) ? -inv : inv;
                if ((cap >> k) & 1)
                  val = lds_values ? s_capl[kk][wv][lane * kLaneStride + (cb >> 4) + __popc(cap & ((1u << k) - 1u))]
                                   : c.row[eq + k];
                if ((int64_t)p < a.cap) {
                  oi[p] = (int32_t)(eq + k);
                  ov[p] = val;
                }
                ++p;
              }
            }
            carry += stot;
          }
        } else if (lds_values) {
          emit(std::true_type{});
        } else {
          emit(std::false_type{});
        }
      } else {
        // hybrid coding (Section 3.3, eqs. 9-10): capped survivors go to Q_A as (index, g_i), the
        // others to Q_B as index | sign << 31 (their value is sign(g_i) / lambda)
        const uint64_t bm = sm & ~cm;
        uint32_t btot;
        const uint64_t excl_cap = (excl >> 31) & 0x7FFFFFFFull;
        uint64_t pa = excl_cap + wbase_cap + cr;
        uint64_t pb = (excl & 0x7FFFFFFFull) - excl_cap + (wbase - wbase_cap) +
                      wave_prefix_bits<7>((uint32_t)__popcll(bm), btot);
        int32_t* __restrict__ oa = a.idx + row * a.cap;
        float* __restrict__ va = a.val + row * a.cap;
        int32_t* __restrict__ ob = a.code_b + row * a.cap_b;
        auto emit_a = [&](auto from_lds) {
          uint64_t m = cm;
          while (m) {
            const int b = __ffsll((unsigned long long)m) - 1;
            float val;
            if constexpr (decltype(from_lds)::value) val = capval(b);
            else val = c.row[e0 + b];
            if ((int64_t)pa < a.cap) {
              oa[pa] = (int32_t)(e0 + b);
              va[pa] = val;
            }
            ++pa;
            m &= m - 1;
          }
        };
        if (s_wsel[kk][wv] > (uint32_t)kDenseEmit) {
          // many survivors: group by group in phase-1 order, as in the compaction above
          uint64_t pa0 = excl_cap + wbase_cap;
          uint64_t pb0 = (excl & 0x7FFFFFFFull) - excl_cap + (wbase - wbase_cap);
          for (int j = 0; j < kTileGroups; ++j) {
            const int q = wv * (kWaveElems / 4) + 64 * j + lane;  // tile group
            const uint32_t code = s_code[kk][q];
            const uint32_t sel = code & 0xFu, neg = code >> 4;
            const uint32_t cb = s_capb[kk][q], cap = cb & sel, oth = sel & ~cap;
            uint32_t atot, btot2;
            uint64_t qa = pa0 + wave_prefix_bits<3>((uint32_t)__popc(cap), atot);
            uint64_t qb = pb0 + wave_prefix_bits<3>((uint32_t)__popc(oth), btot2);
            const int64_t eq = part * (int64_t)kTileElems + 4 * (int64_t)q;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              if ((cap >> k) & 1) {
                const float val =
                    lds_values ? s_capl[kk][wv][lane * kLaneStride + (cb >> 4) + __popc(cap & ((1u << k) - 1u))]
                               : c.row[eq + k];
                if ((int64_t)qa < a.cap) {
                  oa[qa] = (int32_t)(eq + k);
                  va[qa] = val;
                }
                ++qa;
              } else if ((oth >> k) & 1) {
                if ((int64_t)qb < a.cap_b) ob[qb] = (int32_t)((uint32_t)(eq + k) | (((neg >> k) & 1u) << 31));
                ++qb;
              }
            }
            pa0 += atot;
            pb0 += btot2;
          }
        } else {
          if (cm) {
            if (lds_values) emit_a(std::true_type{});
            else emit_a(std::false_type{});
          }
          uint64_t m = bm;
          while (m) {
            const int b = __ffsll((unsigned long long)m) - 1;
            if ((int64_t)pb < a.cap_b) ob[pb] = (int32_t)((uint32_t)(e0 + b) | (uint32_t)(((nm >> b) & 1) << 31));
            ++pb;
            m &= m - 1;
          }
        }
      }
    }
    if constexpr (HYB) {
      // dense ternary vector (Section 3.3): 2 on the capped set, sign(g_i) for the other
      // survivors, 0 elsewhere; this thread's 64 coordinates
      if (a.q && e0 < c.d) {
        int8_t* __restrict__ qr = a.q + base + e0;
        uint32_t w[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          uint32_t x = 0;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int b = 4 * j + k;
            const uint32_t code = ((cm >> b) & 1) ? 2u : (((sm >> b) & 1) ? (((nm >> b) & 1) ? 0xFFu : 1u) : 0u);
            x |= code << (8 * k);
          }
          w[j] = x;
        }
        if (e0 + 64 <= c.d && ((uintptr_t)qr & 15) == 0) {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            uint4 v;
            v.x = w[4 * j]; v.y = w[4 * j + 1]; v.z = w[4 * j + 2]; v.w = w[4 * j + 3];
            reinterpret_cast<uint4*>(qr)[j] = v;
          }
        } else {
          const int64_t nb = min((int64_t)64, c.d - e0);
          for (int64_t b = 0; b < nb; ++b) qr[b] = (int8_t)((w[b >> 2] >> (8 * (b & 3))) & 0xFF);
        }
      }
    }
    excl += agg[kk];
  }
  if (part0 + nk == rtiles && tid == 0) {
    const uint64_t incl = excl;
    const int64_t n = (int64_t)(incl & 0x7FFFFFFFull);
    const int64_t kc = (int64_t)((incl >> 31) & 0x7FFFFFFFull);
    uint32_t fl = ctl->flags;
    if (!ctl->done) fl |= kFlagInternal;
    if constexpr (!HYB) {
      if (a.nnz) a.nnz[row] = n;
      if (n > a.cap) fl |= GSPAR_FLAG_OVERFLOW;
    } else {
      a.nnz[row] = kc;
      a.nnz_b[row] = n - kc;
      if (a.inv_out) a.inv_out[row] = inv;
      if (kc > a.cap || n - kc > a.cap_b) fl |= GSPAR_FLAG_OVERFLOW;
    }
    if (a.k_out) a.k_out[row] = kc;
    if (a.lam_out) a.lam_out[row] = ctl->lam;
    if (a.flags_out) a.flags_out[row] = fl;
  }
}

// p_i = min(lambda |g_i|, 1), exactly 1 on the capped set. Grid: rows * nb workgroups. Capped
// coordinates are counted per workgroup and added into one of eight per-row lines.
template <bool VEC>
__global__ void __launch_bounds__(256) k_probs(Args a) {
  __shared__ uint32_t s_cnt[4];
  int64_t row, blk;
  if (!hist_block(a, row, blk)) return;
  const RowCtl* ctl = ctl_of(a, row);
  const double lam = ctl->lam;
  const uint32_t tcap = ctl->tcap;
  const bool live =
      ctl->done && !(ctl->flags & (GSPAR_FLAG_NONFINITE | GSPAR_FLAG_BADRHO | GSPAR_FLAG_BADSEG | kFlagInternal));
  int64_t base, len;
  row_span(a, row, base, len);
  const int64_t beg = blk * a.chunk;
  if (beg >= len) return;  // past the end of a shorter segment
  const float* __restrict__ gr = a.g + base;
  float* __restrict__ pr = a.p ? a.p + base : nullptr;
  const int64_t end = min(len, beg + a.chunk);
  uint32_t kc = 0;
  stream_groups<VEC, 4, 256>(gr, beg, end, [&](int64_t q, const float v[4], uint32_t m) {
    float o[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint32_t key = key_of(v[c]);
      const bool capped = live && key != 0 && key >= tcap;
      double pv = capped ? 1.0 : (live ? fmin(lam * (double)fabsf(v[c]), 1.0) : 0.0);
      if (key == 0) pv = 0.0;
      o[c] = (float)pv;
      kc += capped && ((m >> c) & 1);
    }
    if (pr) {
      if (VEC && m == 0xF) {
        store_stream(pr + 4 * q, make_float4(o[0], o[1], o[2], o[3]));
      } else {
        for (int c = 0; c < 4; ++c)
          if ((m >> c) & 1) pr[4 * q + c] = o[c];
      }
    }
  });
  for (int o = 32; o > 0; o >>= 1) kc += __shfl_xor(kc, o);
  if ((threadIdx.x & 63) == 0) s_cnt[threadIdx.x >> 6] = kc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t tot = 0;
    for (int i = 0; i < (int)(blockDim.x / 64); ++i) tot += s_cnt[i];
    if (tot) atomicAdd(&kc_of(a, row)[blk & 7].v, (unsigned long long)tot);
  }
}

// Per-row outputs of the probabilities entry points (one thread per row).
__global__ void __launch_bounds__(64) k_probs_out(Args a) {
  const int64_t row = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (row >= a.rows) return;
  const RowCtl* ctl = ctl_of(a, row);
  const CountLine* kl = kc_of(a, row);
  uint64_t ktot = 0;
  for (int i = 0; i < 8; ++i) ktot += kl[i].v;
  if (a.lam_out) a.lam_out[row] = ctl->lam;
  if (a.k_out) a.k_out[row] = (int64_t)ktot;
  uint32_t fl = ctl->flags;
  if (!ctl->done) fl |= kFlagInternal;
  if (a.flags_out) a.flags_out[row] = fl;
}

// ------------------------------------------------------------------------------------------
// Host side.
// ------------------------------------------------------------------------------------------
// Kernel classes, in the order the instrumented build reports them.
enum KernelClass {
  kcSample = 0, kcStats, kcProbs, kcSolve, kcRefine, kcInit, kcAggregate, kcProbsOut, kcPresample, kcCount
};

#ifdef GSPAR_INSTRUMENT
// Measurement build only: while armed, each launch records a pair of HIP events taken by the
// dispatch itself (hipExtLaunchKernelGGL's start and stop events, the kernel's own execution
// interval), filed under its class.
struct Timing {
  int max = 0;
  int n = 0;
  hipEvent_t* ev = nullptr;
  int* cls = nullptr;
};
static Timing g_timing;
#endif

template <typename... KArgs, typename... Args>
static void launch(int cls, void (*kern)(KArgs...), dim3 grid, dim3 block, hipStream_t s, Args... args) {
#ifdef GSPAR_INSTRUMENT
  if (g_timing.ev && g_timing.n < g_timing.max) {
    const int i = g_timing.n++;
    g_timing.cls[i] = cls;
    hipExtLaunchKernelGGL(kern, grid, block, 0, s, g_timing.ev[2 * i], g_timing.ev[2 * i + 1], 0, args...);
    return;
  }
#endif
  (void)cls;
  hipLaunchKernelGGL(kern, grid, block, 0, s, args...);
}

// a density in [0, 1], or for the variance-budget solver a finite eps >= 0
static bool rho_ok(double rho, int solver = GSPAR_EXACT) {
  return solver == GSPAR_VARIANCE ? (rho >= 0.0 && rho < INFINITY) : (rho >= 0.0 && rho <= 1.0);
}

static int check_common(const float* g, int64_t rows, int64_t d, int64_t ld, int solver, int iters,
                        void* ws, size_t ws_bytes) {
  if (!g || rows < 1 || d < 1 || d > INT32_MAX || ld < d) return GSPAR_ERR_ARG;
  if (solver != GSPAR_GREEDY && solver != GSPAR_EXACT && solver != GSPAR_VARIANCE) return GSPAR_ERR_ARG;
  if (iters < 0 || iters > kMaxIters) return GSPAR_ERR_ARG;
  if (rows > (int64_t)1 << 24) return GSPAR_ERR_ARG;
  const Layout L = layout_of(rows, d, 0);  // the minimum: no candidate buffers
  if ((double)rows * (double)L.tiles >= 2147483647.0) return GSPAR_ERR_ARG;  // sample grid, tickets
  const int64_t min_chunk = d < kMaxChunk ? d : kMaxChunk;
  if ((double)rows * (double)((d + min_chunk - 1) / min_chunk) >= 2147483647.0) return GSPAR_ERR_ARG;
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < L.total) return GSPAR_ERR_WORKSPACE;
  return GSPAR_OK;
}

static bool vec_ok(const Args& a);

// Candidate keys per row: the full capacity for rows long enough to predict a band, within what
// the workspace holds beyond its fixed part, on the vector path of a strided batch with a density
// budget; 0 otherwise.
static int64_t cand_cap_of(const Args& a) {
  if (a.seg || a.solver == GSPAR_VARIANCE || !vec_ok(a)) return 0;
  const int64_t full = cand_cap_full(a.d);
  if (full == 0) return 0;
  const size_t fixed = layout_of(a.rows, a.d, 0).total;
  if (a.ws_bytes <= fixed) return 0;
  // each key of capacity takes a list slot and a staging slot
  int64_t fit = (int64_t)((a.ws_bytes - fixed) / (2 * sizeof(uint32_t) * (size_t)a.rows));
  fit &= ~(int64_t)63;
  const int64_t cap = fit < full ? fit : full;
  // a workspace that leaves fewer than 2^16 keys (or the full capacity, for shorter rows) runs
  // without a band
  return cap >= (full < (1 << 16) ? full : (1 << 16)) ? cap : 0;
}

static void plan(Args& a) {
  a.lay = layout_of(a.rows, a.d, cand_cap_of(a));
  const int64_t target = 512;
  int64_t chunk;
  if (a.seg) {
    // chosen from the segment lengths so that the nonempty workgroups are resident at once
    chunk = a.seg_chunk;
  } else {
    int64_t nbt = (target + a.rows - 1) / a.rows;
    if (nbt < 1) nbt = 1;
    chunk = (a.d + nbt - 1) / nbt;
  }
  chunk = (chunk + 3) & ~(int64_t)3;
  if (chunk < kMinChunk) chunk = kMinChunk;
  if (chunk > kMaxChunk) chunk = kMaxChunk;
  a.chunk = chunk;
  a.nb = (int)((a.d + chunk - 1) / chunk);
  a.cand_region = (a.lay.cand_cap / a.nb) & ~(int64_t)63;
  if (a.cand_region == 0) a.lay.cand_cap = 0;  // no room for a band
}

static bool vec_ok(const Args& a) {
  if (a.seg) return a.seg_align != 0;
  return ((uintptr_t)a.g % 16 == 0) && (a.ld % 4 == 0);
}

static int launch_solve(Args& a, hipStream_t s) {
  const bool vec = vec_ok(a);
  const int64_t zero_items = a.rows * kC1 * (int64_t)(sizeof(Hist1) / 8) + a.rows * a.lay.tiles;
  const bool sq = a.solver == GSPAR_VARIANCE;  // histogram passes that also sum squares
  int ib = (int)((zero_items + 255) / 256);
  if (ib > 1024) ib = 1024;
  if (ib < 1) ib = 1;
  launch(kcInit, k_init, dim3(ib), dim3(256), s, a);
  // rows long enough for a candidate band: a sample of each row predicts it
  const bool cand = a.lay.cand_cap > 0;
  if (cand) launch(kcPresample, k_presample, dim3((unsigned)(a.rows * kPreWG)), dim3(256), s, a);
  // a segmented call launches only the workgroups that hold coordinates (none if every segment
  // is empty)
  const int64_t nblocks = a.seg ? a.seg_blocks : a.rows * a.nb;
  const dim3 grid((unsigned)nblocks);
  if (nblocks > 0) {
    if (sq) launch(kcStats, vec ? k_stats<true, true, false> : k_stats<false, true, false>, grid, dim3(kNT), s, a);
    else if (cand) launch(kcStats, k_stats<true, false, true>, grid, dim3(kNT), s, a);  // cand implies vec
    else launch(kcStats, vec ? k_stats<true, false, false> : k_stats<false, false, false>, grid, dim3(kNT), s, a);
  }
  a.first = 1;
  launch(kcSolve, sq ? k_solve<true> : k_solve<false>, dim3((unsigned)a.rows), dim3(kNT), s, a);
  // each greedy step needs at most one level-2 pass (which counts its query key directly), the
  // exact solver at most a level-2 and a level-3 window
  const int R = a.solver == GSPAR_GREEDY ? a.T : 2;  // the variance form also needs at most two
  for (int r = 0; r < R; ++r) {
    a.first = 0;
    if (nblocks > 0) {
      if (sq) launch(kcRefine, vec ? k_refine<true, true> : k_refine<false, true>, grid, dim3(kNT), s, a);
      else launch(kcRefine, vec ? k_refine<true, false> : k_refine<false, false>, grid, dim3(kNT), s, a);
    }
    launch(kcSolve, sq ? k_solve<true> : k_solve<false>, dim3((unsigned)a.rows), dim3(kNT), s, a);
  }
  return hipGetLastError() == hipSuccess ? GSPAR_OK : GSPAR_ERR_HIP;
}

template <int K>
static void launch_sample(const Args& a, bool vec, hipStream_t s) {
  const dim3 grid((unsigned)(a.seg ? a.seg_wgs : a.rows * ((a.lay.tiles + K - 1) / K)));
  if (a.code_b) launch(kcSample, vec ? k_sample<true, true, K> : k_sample<false, true, K>, grid, dim3(kTileThreads), s, a);
  else launch(kcSample, vec ? k_sample<true, false, K> : k_sample<false, false, K>, grid, dim3(kTileThreads), s, a);
}

static int run_sample(Args& a, hipStream_t s) {
  plan(a);
  if ((double)a.rows * (double)a.nb >= 2147483647.0) return GSPAR_ERR_ARG;
  int rc = launch_solve(a, s);
  if (rc) return rc;
  const bool vec = vec_ok(a);
  // tiles per workgroup: 1 while every tile can be resident at once, else 2, so that a
  // workgroup's wait for its predecessors' prefix overlaps the decide phase of its second tile
  const int64_t tiles = a.seg ? a.seg_tiles : a.rows * a.lay.tiles;
  if (a.seg ? a.seg_k == 1 : tiles <= kSampleResident) launch_sample<1>(a, vec, s);
  else launch_sample<2>(a, vec, s);
  return hipGetLastError() == hipSuccess ? GSPAR_OK : GSPAR_ERR_HIP;
}

static int run_probs(Args& a, hipStream_t s) {
  plan(a);
  if ((double)a.rows * (double)a.nb >= 2147483647.0) return GSPAR_ERR_ARG;
  int rc = launch_solve(a, s);
  if (rc) return rc;
  const bool vec = vec_ok(a) && (!a.p || (uintptr_t)a.p % 16 == 0);
  const int64_t nblocks = a.seg ? a.seg_blocks : a.rows * a.nb;
  const dim3 grid((unsigned)nblocks);
  if (nblocks > 0) launch(kcProbs, vec ? k_probs<true> : k_probs<false>, grid, dim3(256), s, a);
  launch(kcProbsOut, k_probs_out, dim3((unsigned)((a.rows + 63) / 64)), dim3(64), s, a);
  return hipGetLastError() == hipSuccess ? GSPAR_OK : GSPAR_ERR_HIP;
}

static Args base_args(const float* g, int64_t rows, int64_t d, int64_t ld, int solver, int iters, void* ws,
                      size_t ws_bytes) {
  Args a;
  memset(&a, 0, sizeof(a));
  a.ws_bytes = ws_bytes;
  a.g = g;
  a.rows = rows;
  a.d = d;
  a.ld = ld;
  a.solver = solver;
  a.T = iters;
  a.ws = static_cast<char*>(ws);
  return a;
}

// ------------------------------------------------------------------------------------------
// Aggregation of the workers' sparsified gradients (Algorithm 1, step 6 on one device):
// v_i = (sum over workers m = 0..M-1, in that order, of Q(g^m)_i in fp64) / M, rounded to fp32.
// Input: each worker's ascending (index, value) list as written by the sampling pass.
//
// One workgroup per block of kAggBlock output coordinates, no workspace. For kAggGroup workers at
// a time the workgroup finds where each list enters and leaves its block (a 9-ary search by eight
// lanes per bound, about log_9(n) dependent loads), loads the first kAggThreads entries of every
// one of those ranges at once, then adds them into an fp64 LDS accumulator one worker after
// another (a barrier between workers), so each coordinate's sum is taken in worker order.
// ------------------------------------------------------------------------------------------
constexpr int kAggBlock = 2048;                   // output coordinates per workgroup
constexpr int kAggThreads = 256;
constexpr int kAggLanes = 8;                      // lanes per search
constexpr int kAggGroup = kAggThreads / kAggLanes / 2;  // workers per pass (two searches each)

struct AggArgs {
  const int32_t* idx;
  const float* val;
  int64_t cap;
  const int64_t* nnz;
  int64_t workers, d;
  float* v;
};

__device__ __forceinline__ int64_t agg_len(const AggArgs& a, int64_t m) {
  const int64_t n = a.nnz[m];
  return n < 0 ? 0 : (n < a.cap ? n : a.cap);
}

// Number of entries of id[0, n) below key when the list ascends (its lower bound), found by the
// eight lanes of an aligned lane group: each step probes eight cut points of [lo, hi) and keeps
// the part between the last probe below key and the first one at or above it. For any list the
// result lies in [0, n] and the loop ends, since [lo, hi) shrinks at every step. Every lane of the
// wave must call it (the loop condition is wave-wide).
__device__ int64_t agg_search(const int32_t* id, int64_t n, int64_t key, bool active) {
  const int lane = threadIdx.x & 63, k = lane & (kAggLanes - 1);
  const unsigned long long gmask = 0xFFull << (lane & ~(kAggLanes - 1));
  int64_t lo = 0, hi = active ? n : 0;
  while (__ballot(hi > lo)) {
    const int64_t w = hi - lo;
    const int64_t pk = lo + (w * (k + 1)) / (kAggLanes + 1);
    const bool below = w > 0 && (int64_t)id[pk] < key;
    const int c = __popcll(__ballot(below) & gmask);
    if (w > 0) {
      const int64_t nlo = c == 0 ? lo : lo + (w * c) / (kAggLanes + 1) + 1;
      const int64_t nhi = c == kAggLanes ? hi : lo + (w * (c + 1)) / (kAggLanes + 1);
      hi = nhi;
      lo = nlo < nhi ? nlo : nhi;
    }
  }
  return lo;
}

__global__ void __launch_bounds__(kAggThreads) k_aggregate(AggArgs a) {
  __shared__ double acc[kAggBlock];
  __shared__ int64_t rng[kAggGroup][2];
  const int t = threadIdx.x;
  const int64_t b0 = (int64_t)blockIdx.x * kAggBlock;
  for (int i = t; i < kAggBlock; i += kAggThreads) acc[i] = 0.0;
  for (int64_t m0 = 0; m0 < a.workers; m0 += kAggGroup) {
    const int64_t mg = a.workers - m0 < kAggGroup ? a.workers - m0 : kAggGroup;
    {
      const int q = t / kAggLanes;           // search q: worker m0 + q/2, bound q&1
      const int64_t m = m0 + (q >> 1);
      const bool act = (q >> 1) < mg;
      const int64_t n = act ? agg_len(a, m) : 0;
      const int64_t lb = agg_search(a.idx + (act ? m : 0) * a.cap, n, b0 + (q & 1) * kAggBlock, act);
      if (act && (t & (kAggLanes - 1)) == 0) rng[q >> 1][q & 1] = lb;
    }
    __syncthreads();
    // the first kAggThreads entries of every range, loaded before any is added
    int32_t r[kAggGroup];
    float x[kAggGroup];
#pragma unroll
    for (int k = 0; k < kAggGroup; ++k) {
      r[k] = -1;
      x[k] = 0.0f;
      if (k < mg) {
        const int64_t j = rng[k][0] + t;
        if (j < rng[k][1]) {
          const int64_t rr = (int64_t)a.idx[(m0 + k) * a.cap + j] - b0;
          r[k] = rr >= 0 && rr < kAggBlock ? (int32_t)rr : -1;
          x[k] = a.val[(m0 + k) * a.cap + j];
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kAggGroup; ++k) {
      if (k < mg) {
        if (r[k] >= 0) acc[r[k]] += (double)x[k];
        const int64_t hi = rng[k][1];
        for (int64_t j = rng[k][0] + t + kAggThreads; j < hi; j += kAggThreads) {
          const int64_t rr = (int64_t)a.idx[(m0 + k) * a.cap + j] - b0;
          if (rr >= 0 && rr < kAggBlock) acc[rr] += (double)a.val[(m0 + k) * a.cap + j];
        }
      }
      __syncthreads();
    }
  }
  const double M = (double)a.workers;
  for (int i = t; i < kAggBlock; i += kAggThreads)
    if (b0 + i < a.d) a.v[b0 + i] = (float)(acc[i] / M);
}

// Scratch memory of the no-allocation entry point: one fixed array per GPU, in the code object's
// device memory. Host code never passes the name `scratch` to a kernel (on the host it is only a
// stand-in for the symbol): the array's device address is looked up once per device and kept.
static __device__ __align__(256) unsigned char scratch[GSPAR_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static void* g_scratch_ptr[kMaxDevices];
static std::mutex g_scratch_mu;

// Device address of the current device's scratch array (nullptr if it cannot be obtained).
static void* scratch_of_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace gspar

using namespace gspar;

#ifdef GSPAR_INSTRUMENT
// ------------------------------------------------------------------------------------------
// Stream probes (measurement build only): the bandwidth a plain kernel reaches on the same
// buffers, to set the path's figures against. Laid out like the statistics pass of one row:
// kProbeGroups workgroups of kNT threads, each streaming one contiguous chunk through the same
// loop (stream_groups, four float4 loads in flight per thread); the read probe adds the values (so
// no load is dead) into one double per wave, the copy probe writes them to dst.
// ------------------------------------------------------------------------------------------
namespace gspar {
constexpr int kProbeGroups = 512;
__global__ void __launch_bounds__(kNT) k_probe_read(const float* __restrict__ src, int64_t n, double* sink) {
  const int64_t chunk = ((n + kProbeGroups - 1) / kProbeGroups + 3) & ~(int64_t)3;
  const int64_t beg = (int64_t)blockIdx.x * chunk, end = min(n, beg + chunk);
  float acc = 0.0f;
  if (beg < end)
    stream_groups<true, 4, kNT>(src, beg, end, [&](int64_t, const float v[4], uint32_t) {
      acc += (v[0] + v[1]) + (v[2] + v[3]);
    });
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) atomicAdd(sink, (double)acc);
}
__global__ void __launch_bounds__(kNT) k_probe_copy(const float* __restrict__ src, float* __restrict__ dst, int64_t n) {
  const int64_t chunk = ((n + kProbeGroups - 1) / kProbeGroups + 3) & ~(int64_t)3;
  const int64_t beg = (int64_t)blockIdx.x * chunk, end = min(n, beg + chunk);
  if (beg < end)
    stream_groups<true, 4, kNT>(src, beg, end, [&](int64_t q, const float v[4], uint32_t m) {
      if (m == 0xFu) *reinterpret_cast<float4*>(dst + 4 * q) = make_float4(v[0], v[1], v[2], v[3]);
    });
}
}  // namespace gspar
#endif  // GSPAR_INSTRUMENT

extern "C" {

size_t gspar_workspace_bytes(int64_t rows, int64_t d, int solver) {
  if (rows < 1 || d < 1) return 0;
  return layout_of(rows, d, solver == GSPAR_VARIANCE ? 0 : cand_cap_full(d)).total;
}

int64_t gspar_capacity_hint(int64_t d, double rho) {
  if (d < 1 || !rho_ok(rho)) return 0;
  const double B = rho * (double)d;
  double c = std::ceil(B + 8.0 * std::sqrt(B) + 64.0);
  if (c > (double)d) c = (double)d;
  return (int64_t)c;
}

int sparsify_probs(const float* g, int64_t d, double rho, int solver, int greedy_iters, float* p,
                   double* lambda, int64_t* k, uint32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!lambda || !rho_ok(rho, solver)) return GSPAR_ERR_ARG;
  int rc = check_common(g, 1, d, d, solver, greedy_iters, ws, ws_bytes);
  if (rc) return rc;
  Args a = base_args(g, 1, d, d, solver, greedy_iters, ws, ws_bytes);
  a.rho = rho;
  a.p = p;
  a.lam_out = lambda;
  a.k_out = k;
  a.flags_out = flags;
  return run_probs(a, (hipStream_t)stream);
}

int sparsify_sample_compact(const float* g, int64_t d, double rho, int solver, int greedy_iters, uint64_t seed,
                            int32_t* idx, float* val, int64_t capacity, int64_t* nnz, double* lambda, int64_t* k,
                            uint32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!nnz || capacity < 0 || (capacity > 0 && (!idx || !val)) || !rho_ok(rho, solver)) return GSPAR_ERR_ARG;
  int rc = check_common(g, 1, d, d, solver, greedy_iters, ws, ws_bytes);
  if (rc) return rc;
  Args a = base_args(g, 1, d, d, solver, greedy_iters, ws, ws_bytes);
  a.rho = rho;
  a.seed = seed;
  a.idx = idx;
  a.val = val;
  a.cap = capacity;
  a.nnz = nnz;
  a.lam_out = lambda;
  a.k_out = k;
  a.flags_out = flags;
  return run_sample(a, (hipStream_t)stream);
}

int sparsify_sample_hybrid_batched(const float* g, int64_t rows, int64_t d, int64_t ld, const double* rho,
                                   int solver, int greedy_iters, const uint64_t* seeds, int32_t* idx_a, float* val_a,
                                   int64_t cap_a, int64_t* n_a, int32_t* code_b, int64_t cap_b, int64_t* n_b,
                                   float* inv_lambda, int8_t* q, double* lambda, uint32_t* flags, void* ws,
                                   size_t ws_bytes, void* stream) {
  if (!rho || !seeds || !n_a || !n_b || cap_a < 0 || cap_b < 0 || (cap_a > 0 && (!idx_a || !val_a)) ||
      !code_b)
    return GSPAR_ERR_ARG;
  int rc = check_common(g, rows, d, ld, solver, greedy_iters, ws, ws_bytes);
  if (rc) return rc;
  Args a = base_args(g, rows, d, ld, solver, greedy_iters, ws, ws_bytes);
  a.rho_dev = rho;
  a.seed_dev = seeds;
  a.idx = idx_a;
  a.val = val_a;
  a.cap = cap_a;
  a.nnz = n_a;
  a.code_b = code_b;
  a.cap_b = cap_b;
  a.nnz_b = n_b;
  a.inv_out = inv_lambda;
  a.q = q;
  a.lam_out = lambda;
  a.flags_out = flags;
  return run_sample(a, (hipStream_t)stream);
}

int sparsify_sample_hybrid(const float* g, int64_t d, double rho, int solver, int greedy_iters, uint64_t seed,
                           int32_t* idx_a, float* val_a, int64_t cap_a, int64_t* n_a, int32_t* code_b, int64_t cap_b,
                           int64_t* n_b, float* inv_lambda, int8_t* q, double* lambda, uint32_t* flags, void* ws,
                           size_t ws_bytes, void* stream) {
  if (!n_a || !n_b || cap_a < 0 || cap_b < 0 || (cap_a > 0 && (!idx_a || !val_a)) || !code_b ||
      !rho_ok(rho, solver))
    return GSPAR_ERR_ARG;
  int rc = check_common(g, 1, d, d, solver, greedy_iters, ws, ws_bytes);
  if (rc) return rc;
  Args a = base_args(g, 1, d, d, solver, greedy_iters, ws, ws_bytes);
  a.rho = rho;
  a.seed = seed;
  a.idx = idx_a;
  a.val = val_a;
  a.cap = cap_a;
  a.nnz = n_a;
  a.code_b = code_b;
  a.cap_b = cap_b;
  a.nnz_b = n_b;
  a.inv_out = inv_lambda;
  a.q = q;
  a.lam_out = lambda;
  a.flags_out = flags;
  return run_sample(a, (hipStream_t)stream);
}

int gspar_coding_bits(int64_t d, int64_t n_a, int64_t n_b, int64_t n_b_neg, int float_bits, double* out) {
  if (!out || d < 1 || n_a < 0 || n_b < 0 || n_b_neg < 0 || n_b_neg > n_b || n_a > d || n_b > d - n_a ||
      float_bits < 1)
    return GSPAR_ERR_ARG;
  const double L = std::log2((double)d), b = (double)float_bits;
  // Q_A: index and value per entry; Q_B: index and sign per entry; one float for 1/lambda
  out[0] = (double)n_a * (b + L) + (double)n_b * (L + 1.0) + b;
  // entropy-coded ternary vector (symbols 2, -1, +1, 0) plus the values of Q_A and 1/lambda
  const double counts[4] = {(double)n_a, (double)n_b_neg, (double)(n_b - n_b_neg), (double)(d - n_a - n_b)};
  double h = 0.0;
  for (double c : counts)
    if (c > 0.0) h += c * std::log2((double)d / c);
  out[1] = h + (double)n_a * b + b;
  // the experiments' per-message cost, with the realised |Q_B| for the expected sum of p over it
  out[2] = (double)n_a * (b + L) + std::min(2.0 * (double)d, (double)n_b * L) + b;
  return GSPAR_OK;
}

int gspar_aggregate(const int32_t* idx, const float* val, int64_t cap, const int64_t* nnz, int64_t workers, int64_t d,
                    float* v, void* stream) {
  using namespace gspar;
  if (!nnz || !v || workers < 1 || workers > ((int64_t)1 << 20) || d < 1 || d > INT32_MAX || cap < 0 ||
      (cap > 0 && (!idx || !val)))
    return GSPAR_ERR_ARG;
  AggArgs a;
  a.idx = idx;
  a.val = val;
  a.cap = cap;
  a.nnz = nnz;
  a.workers = workers;
  a.d = d;
  a.v = v;
  hipStream_t s = (hipStream_t)stream;
  launch(kcAggregate, k_aggregate, dim3((unsigned)((d + kAggBlock - 1) / kAggBlock)), dim3(kAggThreads), s, a);
  return hipGetLastError() == hipSuccess ? GSPAR_OK : GSPAR_ERR_HIP;
}

int sparsify_probs_batched(const float* g, int64_t rows, int64_t d, int64_t ld, const double* rho, int solver,
                           int greedy_iters, float* p, double* lambda, int64_t* k, uint32_t* flags, void* ws,
                           size_t ws_bytes, void* stream) {
  if (!rho || !lambda) return GSPAR_ERR_ARG;
  int rc = check_common(g, rows, d, ld, solver, greedy_iters, ws, ws_bytes);
  if (rc) return rc;
  Args a = base_args(g, rows, d, ld, solver, greedy_iters, ws, ws_bytes);
  a.rho_dev = rho;
  a.p = p;
  a.lam_out = lambda;
  a.k_out = k;
  a.flags_out = flags;
  return run_probs(a, (hipStream_t)stream);
}

int sparsify_sample_compact_batched(const float* g, int64_t rows, int64_t d, int64_t ld, const double* rho,
                                    int solver, int greedy_iters, const uint64_t* seeds, int32_t* idx, float* val,
                                    int64_t cap_per_row, int64_t* nnz, double* lambda, int64_t* k, uint32_t* flags,
                                    void* ws, size_t ws_bytes, void* stream) {
  if (!rho || !seeds || !nnz || cap_per_row < 0 || (cap_per_row > 0 && (!idx || !val))) return GSPAR_ERR_ARG;
  int rc = check_common(g, rows, d, ld, solver, greedy_iters, ws, ws_bytes);
  if (rc) return rc;
  Args a = base_args(g, rows, d, ld, solver, greedy_iters, ws, ws_bytes);
  a.rho_dev = rho;
  a.seed_dev = seeds;
  a.idx = idx;
  a.val = val;
  a.cap = cap_per_row;
  a.nnz = nnz;
  a.lam_out = lambda;
  a.k_out = k;
  a.flags_out = flags;
  return run_sample(a, (hipStream_t)stream);
}

int sparsify_sample_compact_batched_noalloc(const float* g, int64_t rows, int64_t d, int64_t ld, const double* rho,
                                            int solver, int greedy_iters, const uint64_t* seeds, int32_t* idx,
                                            float* val, int64_t cap_per_row, int64_t* nnz, double* lambda, int64_t* k,
                                            uint32_t* flags, void* stream) {
  if (rows < 1 || d < 1) return GSPAR_ERR_ARG;
  if (layout_of(rows, d, 0).total > GSPAR_SCRATCH_BYTES) return GSPAR_ERR_TOO_LARGE;
  void* ws = scratch_of_current_device();
  if (!ws) return GSPAR_ERR_HIP;
  return sparsify_sample_compact_batched(g, rows, d, ld, rho, solver, greedy_iters, seeds, idx, val, cap_per_row,
                                         nnz, lambda, k, flags, ws, GSPAR_SCRATCH_BYTES, stream);
}

// Host check of segment offsets (off[0] >= 0, nondecreasing, every length below 2^31): the longest
// length (at least 1, the row length the workspace is sized for), the total length, and whether
// vector loads may be used (g 16-byte aligned and every start a multiple of 4).
static int check_segments(const float* g, const int64_t* off, const int64_t* off_dev, int64_t segs, int64_t& maxlen,
                          int64_t& total, bool& aligned) {
  if (!g || !off || !off_dev || segs < 1 || segs > ((int64_t)1 << 24) || off[0] < 0) return GSPAR_ERR_ARG;
  maxlen = 1;
  aligned = (uintptr_t)g % 16 == 0;
  for (int64_t r = 0; r < segs; ++r) {
    const int64_t len = off[r + 1] - off[r];
    if (off[r + 1] < off[r] || len > INT32_MAX) return GSPAR_ERR_ARG;
    if (len > maxlen) maxlen = len;
    if (off[r] & 3) aligned = false;
  }
  total = off[segs] - off[0];
  return GSPAR_OK;
}

static void set_segments(Args& a, const int64_t* off, const int64_t* off_dev, int64_t segs, int64_t total,
                         bool aligned) {
  a.seg = off_dev;
  a.seg_total = off[segs];
  a.seg_elems = total;
  a.seg_align = aligned ? 1 : 0;
  // histogram passes: the smallest chunk (a multiple of 4, at least kMinChunk) for which the
  // segments need at most 512 workgroups (two resident per CU); the grid holds exactly those
  auto blocks = [&](int64_t ch) {
    int64_t n = 0;
    for (int64_t r = 0; r < segs; ++r) n += (off[r + 1] - off[r] + ch - 1) / ch;
    return n;
  };
  int64_t lo = kMinChunk, hi = kMaxChunk & ~(int64_t)3;
  if (blocks(lo) <= 512) {
    hi = lo;
  } else if (blocks(hi) <= 512) {
    while (hi - lo > 4) {
      const int64_t mid = ((lo + hi) / 2) & ~(int64_t)3;
      if (blocks(mid) <= 512) hi = mid;
      else lo = mid;
    }
  }
  a.seg_chunk = hi;
  a.seg_blocks = blocks(hi);
  // sample pass: tiles per workgroup from the tiles that hold coordinates, and the workgroups
  a.seg_tiles = 0;
  for (int64_t r = 0; r < segs; ++r) {
    const int64_t len = off[r + 1] - off[r];
    a.seg_tiles += len > kTileElems ? (len + kTileElems - 1) / kTileElems : 1;
  }
  a.seg_k = a.seg_tiles <= kSampleResident ? 1 : 2;
  a.seg_wgs = 0;
  for (int64_t r = 0; r < segs; ++r) {
    const int64_t len = off[r + 1] - off[r];
    const int64_t rt = len > kTileElems ? (len + kTileElems - 1) / kTileElems : 1;
    a.seg_wgs += (rt + a.seg_k - 1) / a.seg_k;
  }
}

int sparsify_sample_compact_segmented(const float* g, int64_t segs, const int64_t* off, const int64_t* off_dev,
                                      const double* rho, int solver, int greedy_iters, const uint64_t* seeds,
                                      int32_t* idx, float* val, int64_t cap_per_seg, int64_t* nnz, double* lambda,
                                      int64_t* k, uint32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!rho || !seeds || !nnz || cap_per_seg < 0 || (cap_per_seg > 0 && (!idx || !val))) return GSPAR_ERR_ARG;
  int64_t maxlen, total;
  bool aligned;
  int rc = check_segments(g, off, off_dev, segs, maxlen, total, aligned);
  if (rc) return rc;
  rc = check_common(g, segs, maxlen, maxlen, solver, greedy_iters, ws, ws_bytes);
  if (rc) return rc;
  Args a = base_args(g, segs, maxlen, maxlen, solver, greedy_iters, ws, ws_bytes);
  set_segments(a, off, off_dev, segs, total, aligned);
  a.rho_dev = rho;
  a.seed_dev = seeds;
  a.idx = idx;
  a.val = val;
  a.cap = cap_per_seg;
  a.nnz = nnz;
  a.lam_out = lambda;
  a.k_out = k;
  a.flags_out = flags;
  return run_sample(a, (hipStream_t)stream);
}

int sparsify_sample_hybrid_segmented(const float* g, int64_t segs, const int64_t* off, const int64_t* off_dev,
                                     const double* rho, int solver, int greedy_iters, const uint64_t* seeds,
                                     int32_t* idx_a, float* val_a, int64_t cap_a, int64_t* n_a, int32_t* code_b,
                                     int64_t cap_b, int64_t* n_b, float* inv_lambda, int8_t* q, double* lambda,
                                     uint32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!rho || !seeds || !n_a || !n_b || cap_a < 0 || cap_b < 0 || (cap_a > 0 && (!idx_a || !val_a)) ||
      !code_b)
    return GSPAR_ERR_ARG;
  int64_t maxlen, total;
  bool aligned;
  int rc = check_segments(g, off, off_dev, segs, maxlen, total, aligned);
  if (rc) return rc;
  rc = check_common(g, segs, maxlen, maxlen, solver, greedy_iters, ws, ws_bytes);
  if (rc) return rc;
  Args a = base_args(g, segs, maxlen, maxlen, solver, greedy_iters, ws, ws_bytes);
  set_segments(a, off, off_dev, segs, total, aligned);
  a.rho_dev = rho;
  a.seed_dev = seeds;
  a.idx = idx_a;
  a.val = val_a;
  a.cap = cap_a;
  a.nnz = n_a;
  a.code_b = code_b;
  a.cap_b = cap_b;
  a.nnz_b = n_b;
  a.inv_out = inv_lambda;
  a.q = q;
  a.lam_out = lambda;
  a.flags_out = flags;
  return run_sample(a, (hipStream_t)stream);
}

int sparsify_probs_segmented(const float* g, int64_t segs, const int64_t* off, const int64_t* off_dev,
                             const double* rho, int solver, int greedy_iters, float* p, double* lambda, int64_t* k,
                             uint32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!rho || !lambda) return GSPAR_ERR_ARG;
  int64_t maxlen, total;
  bool aligned;
  int rc = check_segments(g, off, off_dev, segs, maxlen, total, aligned);
  if (rc) return rc;
  rc = check_common(g, segs, maxlen, maxlen, solver, greedy_iters, ws, ws_bytes);
  if (rc) return rc;
  Args a = base_args(g, segs, maxlen, maxlen, solver, greedy_iters, ws, ws_bytes);
  set_segments(a, off, off_dev, segs, total, aligned);
  a.rho_dev = rho;
  a.p = p;
  a.lam_out = lambda;
  a.k_out = k;
  a.flags_out = flags;
  return run_probs(a, (hipStream_t)stream);
}

const char* gspar_status_string(int status) {
  switch (status) {
    case GSPAR_OK: return "ok";
    case GSPAR_ERR_ARG: return "invalid argument";
    case GSPAR_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case GSPAR_ERR_HIP: return "HIP launch failed";
    case GSPAR_ERR_TOO_LARGE: return "problem too large for the library's fixed scratch array";
    default: return "unknown status";
  }
}

int gspar_version(void) { return 100; }

#ifdef GSPAR_INSTRUMENT
int gspar_prof_arm(int max_launches) {
  if (max_launches < 1) return GSPAR_ERR_ARG;
  gspar_prof_disarm();
  g_timing.ev = new hipEvent_t[2 * (size_t)max_launches];
  g_timing.cls = new int[(size_t)max_launches];
  for (int i = 0; i < 2 * max_launches; ++i) {
    if (hipEventCreate(&g_timing.ev[i]) != hipSuccess) {
      for (int j = 0; j < i; ++j) (void)hipEventDestroy(g_timing.ev[j]);
      delete[] g_timing.ev;
      delete[] g_timing.cls;
      g_timing = Timing();
      return GSPAR_ERR_HIP;
    }
  }
  g_timing.max = max_launches;
  g_timing.n = 0;
  return GSPAR_OK;
}

int gspar_prof_read(double* ms, int* launches) {
  if (!ms || !launches) return GSPAR_ERR_ARG;
  for (int c = 0; c < kcCount; ++c) {
    ms[c] = 0.0;
    launches[c] = 0;
  }
  if (!g_timing.ev || g_timing.n == 0) return GSPAR_OK;
  if (hipEventSynchronize(g_timing.ev[2 * g_timing.n - 1]) != hipSuccess) return GSPAR_ERR_HIP;
  for (int i = 0; i < g_timing.n; ++i) {
    float t = 0.f;
    if (hipEventElapsedTime(&t, g_timing.ev[2 * i], g_timing.ev[2 * i + 1]) != hipSuccess) return GSPAR_ERR_HIP;
    ms[g_timing.cls[i]] += t;
    launches[g_timing.cls[i]] += 1;
  }
  return GSPAR_OK;
}

int gspar_prof_disarm(void) {
  if (g_timing.ev) {
    for (int i = 0; i < 2 * g_timing.max; ++i) (void)hipEventDestroy(g_timing.ev[i]);
    delete[] g_timing.ev;
    delete[] g_timing.cls;
  }
  g_timing = Timing();
  return GSPAR_OK;
}

// Host-side checks of the device arithmetic (the same source compiled for the host): rounding of
// the exact accumulator, the shift invariant, the capped-threshold search and the generator.
double gspar_check_fx_round(const uint64_t* limbs5) {
  Fx f;
  for (int i = 0; i < 5; ++i) f.w[i] = limbs5[i];
  return fx_to_double(f);
}

uint32_t gspar_check_fx_shifted(uint64_t v, int s, uint64_t* limbs5) {
  uint32_t err = 0;
  const Fx f = fx_shifted(v, s, &err);
  for (int i = 0; i < 5; ++i) limbs5[i] = f.w[i];
  return err;
}

uint32_t gspar_check_fq_squares(uint64_t qh, uint64_t ql, int shift, uint64_t* limbs10) {
  uint32_t err = 0;
  const Fq f = fq_squares(qh, ql, shift, &err);
  for (int i = 0; i < kQ; ++i) limbs10[i] = f.w[i];
  return err;
}

double gspar_check_exact_sum(const float* x, int64_t n) {
  Fx acc = fx_zero();
  uint32_t err = 0;
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t key = key_of(x[i]);
    if (key == 0 || key >= kKeyInf) continue;
    fx_add(acc, fx_shifted(key_sig(key), binade_shift((int)(key >> 23)), &err));
  }
  return err ? NAN : fx_to_double(acc);
}

uint32_t gspar_check_cap_key(double lam) { return cap_key(lam); }

int gspar_probe_stream(const float* src, float* dst, int64_t n, double* sink, void* stream) {
  if (!src || n < 0 || n % 4 != 0 || (uintptr_t)src % 16 || (dst && (uintptr_t)dst % 16) || (!dst && !sink))
    return GSPAR_ERR_ARG;
  if (n == 0) return GSPAR_OK;
  hipStream_t s = (hipStream_t)stream;
  const dim3 grid(kProbeGroups), block(kNT);
  if (dst) hipLaunchKernelGGL(k_probe_copy, grid, block, 0, s, src, dst, n);
  else hipLaunchKernelGGL(k_probe_read, grid, block, 0, s, src, n, sink);
  return hipGetLastError() == hipSuccess ? GSPAR_OK : GSPAR_ERR_HIP;
}

void gspar_check_philox(const uint32_t* ctr, const uint32_t* key, uint32_t* out) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  philox10(c0, c1, c2, c3, key[0], key[1]);
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}
#endif  // GSPAR_INSTRUMENT

}  // extern "C"
