// Oracle for the gradient sparsifier of Wangni, Wang, Liu and Zhang, "Gradient Sparsification for
// Communication-Efficient Distributed Optimization" (arXiv 1710.09854).
//
// TEST INFRASTRUCTURE ONLY. This file is a plain, slow, double-precision CPU statement of what the
// sparsifier computes. Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
// load it. It shares no code, header, table or helper with the GPU library and includes nothing
// from it. The only library primitives used as steps are std::sort and std::nth_element.
//
// Notation follows the paper: g is the gradient, a_i = |g_i|, p the keep-probability vector,
// Z the selection vector, Q(g) the sparsified vector, B = rho*d the density budget, k the size of
// the capped set S_k (coordinates with p_i = 1), lambda the scale of Proposition 1.
//
// Parity status of each function is stated in its comment; every one is pinned by a test against
// a brute-force search, a closed form, an invariant or a published known answer.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <functional>
#include <vector>

namespace {

// ---------------------------------------------------------------------------------------------
// Exact accumulation of non-negative doubles (a fixed-point integer with LSB 2^-1074 and 2176
// bits, wide enough for any finite double plus 78 bits of carry headroom). The paper's sums
// (sums of |g_i|, of g_i^2, of p_i) are written as sums over sets; the oracle evaluates each as
// the exact real sum, rounded once to the nearest double (ties to even). Pinned against Python's
// math.fsum, which returns the correctly rounded sum.
// ---------------------------------------------------------------------------------------------
struct Exact {
  static const int L = 34;
  uint64_t w[L];
  Exact() { std::memset(w, 0, sizeof(w)); }

  void add(double x) {  // x >= 0, finite
    if (x == 0.0) return;
    int e;
    double f = std::frexp(x, &e);                    // x = f * 2^e, f in [0.5, 1)
    uint64_t m = (uint64_t)std::ldexp(f, 53);        // 53-bit integer mantissa
    int pos = e - 53 + 1074;                         // x = m * 2^(pos - 1074)
    if (pos < 0) {                                   // subnormal: m has trailing zeros to drop
      m >>= -pos;
      pos = 0;
    }
    int li = pos / 64, sh = pos % 64;
    uint64_t lo = m << sh;
    uint64_t hi = sh ? (m >> (64 - sh)) : 0;
    add_at(li, lo);
    if (hi) add_at(li + 1, hi);
  }
  void add_at(int li, uint64_t v) {
    for (int i = li; i < L && v; ++i) {
      uint64_t s = w[i] + v;
      v = (s < v) ? 1 : 0;
      w[i] = s;
    }
  }
  void add(const Exact& o) {
    uint64_t c = 0;
    for (int i = 0; i < L; ++i) {
      uint64_t s = w[i] + o.w[i];
      uint64_t c1 = s < w[i];
      uint64_t s2 = s + c;
      uint64_t c2 = s2 < s;
      w[i] = s2;
      c = c1 | c2;
    }
  }
  // this - o, requires this >= o
  Exact minus(const Exact& o) const {
    Exact r;
    uint64_t b = 0;
    for (int i = 0; i < L; ++i) {
      uint64_t d1 = w[i] - o.w[i];
      uint64_t b1 = w[i] < o.w[i];
      uint64_t d2 = d1 - b;
      uint64_t b2 = d1 < b;
      r.w[i] = d2;
      b = b1 | b2;
    }
    return r;
  }
  bool bit(int k) const { return (w[k / 64] >> (k % 64)) & 1; }
  // round to nearest double, ties to even
  double value() const {
    int top = -1;
    for (int i = L - 1; i >= 0; --i)
      if (w[i]) { top = i * 64 + 63 - __builtin_clzll(w[i]); break; }
    if (top < 0) return 0.0;
    int len = top + 1;
    if (len <= 53) return std::ldexp((double)w[0], -1074);  // exact: fits in the low limb
    // take bits [top-52, top]
    uint64_t m = 0;
    for (int k = top; k >= top - 52; --k) m = (m << 1) | (uint64_t)bit(k);
    bool rnd = bit(top - 53);
    bool sticky = false;  // any set bit at or below position top-54
    int sb = top - 54;
    if (sb >= 0) {
      int li = sb / 64, off = sb % 64;
      uint64_t mask = off == 63 ? ~0ull : ((1ull << (off + 1)) - 1);
      sticky = (w[li] & mask) != 0;
      for (int i = li - 1; i >= 0 && !sticky; --i) sticky = w[i] != 0;
    }
    int exp = top - 52 - 1074;
    if (rnd && (sticky || (m & 1))) {
      m += 1;
      if (m == (1ull << 53)) { m >>= 1; exp += 1; }
    }
    return std::ldexp((double)m, exp);
  }
};

inline bool finite_f(float x) { return std::isfinite(x); }

// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3",
// SC'11). Written from the published round function: each round multiplies counter words 0 and 2
// by the two round multipliers, crosses the high halves with words 1 and 3 and the round key, and
// the key is bumped by the two Weyl constants between rounds. Pinned against published known
// answers and against an independent engine in a test.
void philox(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int r = 0; r < 10; ++r) {
    uint64_t prod0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
    uint64_t prod1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
    uint32_t hi0 = (uint32_t)(prod0 >> 32), lo0 = (uint32_t)prod0;
    uint32_t hi1 = (uint32_t)(prod1 >> 32), lo1 = (uint32_t)prod1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    uint32_t n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

// The random word used for coordinate i of a row keyed by seed: Philox4x32-10 with
// key = (seed low 32, seed high 32), counter = (q low 32, q high 32, 0, 0) for q = floor(i/4),
// output word i mod 4.
uint32_t word_for(uint64_t seed, int64_t i) {
  uint64_t q = (uint64_t)i >> 2;
  uint32_t ctr[4] = {(uint32_t)q, (uint32_t)(q >> 32), 0u, 0u};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t out[4];
  philox(ctr, key, out);
  return out[i & 3];
}

enum { FLAG_NONFINITE = 1, FLAG_OVERFLOW = 2, FLAG_ALLZERO = 4 };

struct Sol {
  double lambda;     // scale of Proposition 1 (+inf when every nonzero coordinate is capped)
  int64_t k;         // size of the capped set
  int iters;         // greedy rescale steps taken
  uint32_t flags;
};

// Common preamble: magnitudes, budget, special cases (which make p the indicator of the support
// or identically zero). Returns true when the special case settled p.
bool preamble(const float* g, int64_t d, double rho, std::vector<double>& a, double& B,
              int64_t& nnz, double* p, Sol& s) {
  s.lambda = 0.0; s.k = 0; s.iters = 0; s.flags = 0;
  a.resize(d);
  nnz = 0;
  for (int64_t i = 0; i < d; ++i) {
    if (!finite_f(g[i])) { s.flags |= FLAG_NONFINITE; }
    a[i] = std::fabs((double)g[i]);
    if (a[i] > 0.0) ++nnz;
  }
  B = rho * (double)d;
  if (s.flags & FLAG_NONFINITE) {
    s.lambda = NAN;
    for (int64_t i = 0; i < d; ++i) p[i] = 0.0;
    return true;
  }
  if (nnz == 0) s.flags |= FLAG_ALLZERO;
  if (nnz == 0 || B >= (double)nnz) {
    // every nonzero coordinate kept with probability one: Q(g) = g exactly
    s.lambda = INFINITY;
    s.k = nnz;
    for (int64_t i = 0; i < d; ++i) p[i] = a[i] > 0.0 ? 1.0 : 0.0;
    return true;
  }
  if (B == 0.0) {  // rho = 0: nothing may be kept
    for (int64_t i = 0; i < d; ++i) p[i] = 0.0;
    return true;
  }
  return false;
}

}  // namespace

extern "C" {

void orc_philox4x32_10(const uint32_t* ctr, const uint32_t* key, uint32_t* out) { philox(ctr, key, out); }

void orc_words(uint64_t seed, int64_t d, uint32_t* x) {
  for (int64_t i = 0; i < d; ++i) x[i] = word_for(seed, i);
}

void orc_words_at(uint64_t seed, int64_t n, const int64_t* idx, uint32_t* x) {
  for (int64_t j = 0; j < n; ++j) x[j] = word_for(seed, idx[j]);
}

double orc_exact_sum(const double* x, int64_t n) {
  Exact e;
  for (int64_t i = 0; i < n; ++i) e.add(x[i]);
  return e.value();
}

// Exact solver, density form. Proposition 1 gives p_i = min(lambda*a_i, 1); the KKT argument
// (eq. 5) shows the capped set S_k is the k largest magnitudes. With the density budget
// sum_i p_i = B in place of the variance budget of problem (4) (same family of solutions), the
// criterion of Algorithm 2 becomes: with a_(1) >= a_(2) >= ... the nonzero magnitudes and
// T_k = sum_{i>k} a_(i), take the smallest k with (B - k) * a_(k+1) <= T_k, then
// lambda = (B - k) / T_k. The criterion is monotone in k and never holds strictly inside a run of
// equal magnitudes in exact arithmetic, so it is evaluated only where a_(k) > a_(k+1) (or k = 0);
// this keeps tied coordinates together in floating point as well. Then p_i = 1 for a_i > a_(k+1)
// and p_i = min(lambda * a_i, 1) otherwise; the capped set is {p_i = 1}, which also holds the run of
// magnitudes equal to a_(k+1) when the criterion holds with equality (lambda * a_(k+1) = 1).
// Uses partial sorting (the top floor(B)+1 magnitudes), as the paper notes.
int orc_exact_density(const float* g, int64_t d, double rho, double* p, double* lam, int64_t* kout,
                      uint32_t* flags) {
  std::vector<double> a;
  double B;
  int64_t nnz;
  Sol s;
  if (!preamble(g, d, rho, a, B, nnz, p, s)) {
    std::vector<double> nz;
    nz.reserve(nnz);
    Exact total;
    for (int64_t i = 0; i < d; ++i)
      if (a[i] > 0.0) { nz.push_back(a[i]); total.add(a[i]); }
    // In exact arithmetic the criterion already holds at k = floor(B), so the floor(B)+2 largest
    // magnitudes suffice; if rounding ever pushes the answer further, sort everything and rescan.
    int64_t kstar = -1;
    double T = 0.0;
    for (int pass = 0; pass < 2 && kstar < 0; ++pass) {
      int64_t m = pass == 0 ? std::min<int64_t>(nnz, (int64_t)std::floor(B) + 2) : nnz;
      std::nth_element(nz.begin(), nz.begin() + (m - 1), nz.end(), std::greater<double>());
      std::sort(nz.begin(), nz.begin() + m, std::greater<double>());
      Exact prefix;  // sum of a_(1..k)
      for (int64_t k = 0; k < m; ++k) {
        if (k == 0 || nz[k - 1] > nz[k]) {
          double Tk = total.minus(prefix).value();
          if ((B - (double)k) * nz[k] <= Tk) { kstar = k; T = Tk; break; }
        }
        prefix.add(nz[k]);
      }
    }
    if (kstar < 0) return -1;
    double vstar = nz[kstar];
    s.lambda = (B - (double)kstar) / T;
    // k is the size of the capped set {p_i = 1} of Proposition 1: the kstar magnitudes above
    // vstar, plus any others whose product lambda * a_i reaches 1 (a run of ties at vstar when the
    // criterion holds with equality)
    s.k = 0;
    for (int64_t i = 0; i < d; ++i) {
      if (a[i] > vstar) p[i] = 1.0;
      else p[i] = std::min(s.lambda * a[i], 1.0);
      s.k += (p[i] == 1.0);
    }
  }
  *lam = s.lambda;
  *kout = s.k;
  *flags = s.flags;
  return 0;
}

// Exact solver, variance form: Algorithm 2 as printed. Smallest k with
// a_(k+1) * T_k <= eps * sum_j g_j^2 + sum_{i>k} a_(i)^2   (eq. 6), then
// p_i = 1 on S_k and p_i = a_i * T_k / (eps * sum g^2 + sum_{i>k} a_(i)^2) off it (eq. 7).
// Same tie handling as the density form. Full sort (k is not bounded by a budget here).
int orc_exact_variance(const float* g, int64_t d, double eps, double* p, double* lam, int64_t* kout,
                       uint32_t* flags) {
  std::vector<double> a(d);
  uint32_t fl = 0;
  int64_t nnz = 0;
  for (int64_t i = 0; i < d; ++i) {
    if (!finite_f(g[i])) fl |= FLAG_NONFINITE;
    a[i] = std::fabs((double)g[i]);
    if (a[i] > 0) ++nnz;
  }
  *flags = fl;
  if (fl & FLAG_NONFINITE) { *lam = NAN; *kout = 0; for (int64_t i = 0; i < d; ++i) p[i] = 0; return 0; }
  if (nnz == 0) { *flags |= FLAG_ALLZERO; *lam = INFINITY; *kout = 0; for (int64_t i = 0; i < d; ++i) p[i] = 0; return 0; }
  std::vector<double> nz;
  Exact t1, t2;
  for (int64_t i = 0; i < d; ++i)
    if (a[i] > 0) { nz.push_back(a[i]); t1.add(a[i]); t2.add(a[i] * a[i]); }
  std::sort(nz.begin(), nz.end(), std::greater<double>());
  double A = t2.value();
  Exact p1, p2;
  int64_t kstar = nnz;  // if nothing holds, every nonzero is capped (only possible for eps = 0)
  double lamv = INFINITY;
  for (int64_t k = 0; k < nnz; ++k) {
    if (k == 0 || nz[k - 1] > nz[k]) {
      double T1 = t1.minus(p1).value();
      double T2 = t2.minus(p2).value();
      double rhs = eps * A + T2;
      if (nz[k] * T1 <= rhs) { kstar = k; lamv = T1 / rhs; break; }
    }
    p1.add(nz[k]);
    p2.add(nz[k] * nz[k]);
  }
  double vstar = kstar < nnz ? nz[kstar] : 0.0;
  int64_t kcap = 0;  // the capped set {p_i = 1}, as in the density form
  for (int64_t i = 0; i < d; ++i) {
    if (a[i] > vstar) p[i] = 1.0;
    else p[i] = std::min(lamv * a[i], 1.0);
    kcap += (p[i] == 1.0);
  }
  *lam = lamv;
  *kout = kcap;
  return 0;
}

// Greedy solver: Algorithm 3 as printed, on whole vectors.
//   p^0_i = min(rho*d*a_i / sum_i a_i, 1)
//   repeat T times: I = {i : p^j_i != 1}; c = (rho*d - d + |I|) / sum_{i in I} p^j_i;
//                   stop if c <= 1; p^{j+1}_i = min(c*p^j_i, 1).
// T counts rescale steps after the initialisation (the experiments use two). The equivalent
// scale lambda (p_i = min(lambda*a_i, 1)) is reported as lambda_0 times the product of the c's.
int orc_greedy_alg3(const float* g, int64_t d, double rho, int T, double* p, double* lam,
                    int64_t* kout, int* used, uint32_t* flags) {
  std::vector<double> a;
  double B;
  int64_t nnz;
  Sol s;
  if (!preamble(g, d, rho, a, B, nnz, p, s)) {
    Exact sa;
    for (int64_t i = 0; i < d; ++i) sa.add(a[i]);
    double S = sa.value();
    for (int64_t i = 0; i < d; ++i) p[i] = std::min(B * a[i] / S, 1.0);
    double scale = B / S;
    int j = 0;
    for (; j < T; ++j) {
      int64_t inI = 0;
      Exact sp;
      for (int64_t i = 0; i < d; ++i)
        if (p[i] != 1.0) { ++inI; sp.add(p[i]); }
      double den = sp.value();
      if (den == 0.0) break;
      double c = (B - (double)d + (double)inI) / den;
      if (c <= 1.0) break;
      for (int64_t i = 0; i < d; ++i) p[i] = std::min(c * p[i], 1.0);
      scale *= c;
    }
    int64_t k = 0;
    for (int64_t i = 0; i < d; ++i) k += (p[i] == 1.0);
    s.k = k;
    s.lambda = scale;
    s.iters = j;
  }
  *lam = s.lambda;
  *kout = s.k;
  *used = s.iters;
  *flags = s.flags;
  return 0;
}

// Greedy solver in scale form: the same iteration written through p^j = min(lambda_j * a, 1).
// With k_j = #{lambda_{j-1} a_i >= 1} and U_j = sum over the rest of a_i, Algorithm 3's
// c = (B - k_j) / (lambda_{j-1} U_j), so lambda_j = (B - k_j) / U_j, and c <= 1 is
// lambda_j <= lambda_{j-1}. Cross-check of the printed form; not a different method.
int orc_greedy_scale(const float* g, int64_t d, double rho, int T, double* p, double* lam,
                     int64_t* kout, int* used, uint32_t* flags) {
  std::vector<double> a;
  double B;
  int64_t nnz;
  Sol s;
  if (!preamble(g, d, rho, a, B, nnz, p, s)) {
    Exact sa;
    for (int64_t i = 0; i < d; ++i) sa.add(a[i]);
    double l = B / sa.value();
    int j = 0;
    for (; j < T; ++j) {
      int64_t kj = 0;
      Exact u;
      for (int64_t i = 0; i < d; ++i) {
        if (l * a[i] >= 1.0) ++kj;
        else u.add(a[i]);
      }
      double U = u.value();
      if (U == 0.0) break;
      double ln = (B - (double)kj) / U;
      if (ln <= l) break;
      l = ln;
    }
    int64_t k = 0;
    for (int64_t i = 0; i < d; ++i) {
      double q = l * a[i];
      p[i] = q >= 1.0 ? 1.0 : q;
      k += (q >= 1.0);
    }
    s.lambda = l;
    s.k = k;
    s.iters = j;
  }
  *lam = s.lambda;
  *kout = s.k;
  *used = s.iters;
  *flags = s.flags;
  return 0;
}

// Sampling, amplification and compaction (Section 3's protocol): Z_i = 1 with probability p_i,
// drawn as Z_i = [x_i < p_i * 2^32] from the word x_i of Philox4x32-10 described above;
// Q(g)_i = Z_i * g_i / p_i. Survivors are emitted in ascending index order as
// (int32 index, fp32 value = g_i / p_i computed in double). Returns the true count in *nnz; at most
// cap pairs are written.
int orc_sample(const float* g, const double* p, int64_t d, uint64_t seed, int32_t* idx, float* val,
               int64_t cap, int64_t* nnz) {
  int64_t n = 0;
  for (int64_t i = 0; i < d; ++i) {
    if (!(p[i] > 0.0)) continue;
    uint32_t x = word_for(seed, i);
    if ((double)x < p[i] * 4294967296.0) {
      if (n < cap) {
        idx[n] = (int32_t)i;
        val[n] = (float)((double)g[i] / p[i]);
      }
      ++n;
    }
  }
  *nnz = n;
  return 0;
}

}  // extern "C"
