// Per-row passes of the SAKI coupling path.  One workgroup of NT threads owns
// one row at a time; chunk c of the row (1024 entries) belongs to wave c % NW.
//
//  stats sweep   : max / log-sum-exp of s and t, teacher argmax, p-moments of
//                  d = t - s, min/max of d, per-chunk proposal masses.
//  lambda sweeps : sums over the row at one or two candidate lambdas, giving
//                  A(lambda) = log sum_v p_v exp(lambda x_v) (x = d - c), its
//                  first two derivatives, KL(q_lambda || p) = lambda A' - A and
//                  KL' = lambda A''.  A safeguarded Newton iteration on
//                  log KL(lambda) = log eps picks the next candidate.
//  final sweep   : TV(p, q) = sum_v p_v [q_v/p_v - 1]_+, residual chunk
//                  masses, and (optionally) the gradient row.
// (SAKI Sec. 3.2 Eq. bridge / Eq. trust_region; Sec. 3.3; Sec. 3.4; App. E.)
#pragma once

#include "device_util.hpp"

namespace saki {

constexpr int RED_MAX = 12;  // widest block reduction (doubles per thread)

template <int NT>
struct RowShared {
  static constexpr int NW = NT / WAVE;
  float chunk_a[MAX_CHUNKS];  // proposal: chunk max of s | residual: chunk mass
  float chunk_b[MAX_CHUNKS];  // proposal: chunk sum of exp(s - chunk max)
  double red_d[NW][RED_MAX];
  float red_f[NW][4];
  int red_i[NW][4];
};

// Row-uniform results of the stats sweep.
struct RowStats {
  float ms, mt;        // max s, max t
  double lse_s, lse_t; // log-sum-exp of s and t
  double sum_s;        // sum exp(s - ms)
  float c;             // centring constant: E_p[d] rounded to float
  double var;          // Var_p[d] = kappa_2 (starting point of the lambda search)
  double k3, k4;       // third and fourth cumulants of d under p
  double kl1_est;      // KL(pi || p) = E_pi[d] - (lse_t - lse_s), a first estimate
  float dmin, dmax;    // range of d = t - s
  float tmax;          // max t
  int vstar;           // argmax t, lowest index on ties
  bool finite;
};

// Result of one lambda evaluation.
struct LamEval {
  float lam;
  double A, Eq, Var, KL, KLp;
};

template <int NT>
struct Block {
  static constexpr int NW = NT / WAVE;
  int tid, lane, wave;
  RowShared<NT>& sh;
  __device__ Block(RowShared<NT>& s) : sh(s) {
    tid = threadIdx.x;
    lane = tid & (WAVE - 1);
    wave = tid / WAVE;
  }

  // Sums N doubles over the block; every thread gets the same bits.
  template <int N>
  __device__ void sum(double (&v)[N]) {
    static_assert(N <= RED_MAX, "block reduction wider than the LDS buffer");
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = wave_sum(v[i]);
    if (lane == 0) {
#pragma unroll
      for (int i = 0; i < N; ++i) sh.red_d[wave][i] = v[i];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < N; ++i) {
      double acc = 0.0;
      for (int w = 0; w < NW; ++w) acc += sh.red_d[w][i];
      v[i] = acc;
    }
    __syncthreads();
  }

  __device__ float max(float v) {
    v = wave_max(v);
    if (lane == 0) sh.red_f[wave][0] = v;
    __syncthreads();
    float m = -finf();
    for (int w = 0; w < NW; ++w) m = fmaxf(m, sh.red_f[w][0]);
    __syncthreads();
    return m;
  }

  __device__ float min(float v) { return -max(-v); }

  template <typename K>
  __device__ void argmin(K& key, int& idx) {
    wave_argmin(key, idx);
    if (lane == 0) {
      sh.red_d[wave][0] = static_cast<double>(key);
      sh.red_i[wave][0] = idx;
    }
    __syncthreads();
    double bk = sh.red_d[0][0];
    int bi = sh.red_i[0][0];
    for (int w = 1; w < NW; ++w) {
      const double k2 = sh.red_d[w][0];
      const int i2 = sh.red_i[w][0];
      if (k2 < bk || (k2 == bk && i2 < bi)) { bk = k2; bi = i2; }
    }
    __syncthreads();
    key = static_cast<K>(bk);
    idx = bi;
  }

  __device__ void argmax(float& val, int& idx) {
    wave_argmax(val, idx);
    if (lane == 0) {
      sh.red_f[wave][0] = val;
      sh.red_i[wave][0] = idx;
    }
    __syncthreads();
    float bv = sh.red_f[0][0];
    int bi = sh.red_i[0][0];
    for (int w = 1; w < NW; ++w) {
      const float v2 = sh.red_f[w][0];
      const int i2 = sh.red_i[w][0];
      if (v2 > bv || (v2 == bv && i2 < bi)) { bv = v2; bi = i2; }
    }
    __syncthreads();
    val = bv;
    idx = bi;
  }
};

// ---------------------------------------------------------------------------
// Stats sweep.
// ---------------------------------------------------------------------------
template <typename T, int NT, bool TAIL>
__device__ __forceinline__ void stats_chunk(const T* srow, const T* trow, int V, int c, int lane,
                                            bool keep_chunks, RowShared<NT>& sh, float& Ms,
                                            float& Mt, double& Ss, double& S1, double& S2,
                                            double& S3, double& S4, double& St, double& T1,
                                            float& tbest, int& tidx,
                                            float& dmin, float& dmax) {
  float s[EPL], t[EPL];
  uint32_t vm;
  load_lane<T, TAIL>(srow, c, lane, V, s, &vm);
  load_lane<T, TAIL>(trow, c, lane, V, t, &vm);
  float ls = -finf(), lt = -finf();
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    if (!TAIL || ((vm >> e) & 1u)) {
      ls = fmaxf(ls, s[e]);
      lt = fmaxf(lt, t[e]);
    }
  }
  const float cms = wave_max(ls), cmt = wave_max(lt);
  // exponent arguments as (x - max) * log2(e): the subtraction is exact, so
  // the largest terms carry no rounding from the shift
  double ps = 0.0, pt = 0.0;
  float p1 = 0.f, p2 = 0.f, p3 = 0.f, p4 = 0.f, t1 = 0.f;
  const int base = c * CHUNK;
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    if (!TAIL || ((vm >> e) & 1u)) {
      const float es = fexp2((s[e] - cms) * LOG2E);
      const float et = fexp2((t[e] - cmt) * LOG2E);
      const float d = t[e] - s[e];
      // the normalisers are summed in double per entry: next to an entry of
      // weight ~1 a float partial sum would lose the small remaining mass
      ps += static_cast<double>(es);
      pt += static_cast<double>(et);
      const float ed = es * d;
      const float ed2 = ed * d;
      const float ed3 = ed2 * d;
      p1 += ed;
      p2 += ed2;
      p3 += ed3;
      p4 = fmaf(ed3, d, p4);
      t1 = fmaf(et, d, t1);
      if (t[e] > tbest) {
        tbest = t[e];
        tidx = base + elem_offset(lane, e);
      }
      dmin = fminf(dmin, d);
      dmax = fmaxf(dmax, d);
    }
  }
  if (keep_chunks) {
    const float csum = static_cast<float>(wave_sum(ps));
    if (lane == 0) {
      sh.chunk_a[c] = cms;
      sh.chunk_b[c] = csum;
    }
  }
  // fold this chunk into the wave's running sums (all lanes share Ms, Mt)
  if (cms > Ms) {
    const double f = static_cast<double>(fexp2((Ms - cms) * LOG2E));
    Ss *= f; S1 *= f; S2 *= f; S3 *= f; S4 *= f;
    Ms = cms;
  }
  if (cmt > Mt) {
    const double f = static_cast<double>(fexp2((Mt - cmt) * LOG2E));
    St *= f; T1 *= f;
    Mt = cmt;
  }
  // chunks below the running maximum are rescaled; the chunk holding the
  // maximum is added unscaled (factor exactly 1)
  const double gs = (cms == Ms) ? 1.0 : static_cast<double>(fexp2((cms - Ms) * LOG2E));
  const double gt = (cmt == Mt) ? 1.0 : static_cast<double>(fexp2((cmt - Mt) * LOG2E));
  Ss += ps * gs;
  S1 += static_cast<double>(p1) * gs;
  S2 += static_cast<double>(p2) * gs;
  S3 += static_cast<double>(p3) * gs;
  S4 += static_cast<double>(p4) * gs;
  St += pt * gt;
  T1 += static_cast<double>(t1) * gt;
}

template <typename T, int NT>
__device__ RowStats stats_sweep(Block<NT>& B, const T* srow, const T* trow, int V, bool keep_chunks) {
  constexpr int NW = NT / WAVE;
  const int nchunks = (V + CHUNK - 1) / CHUNK;
  const bool ragged = (V % CHUNK) != 0;
  float Ms = -finf(), Mt = -finf();
  double Ss = 0, S1 = 0, S2 = 0, S3 = 0, S4 = 0, St = 0, T1 = 0;
  float tbest = -finf();
  int tidx = 0x7fffffff;
  float dmin = finf(), dmax = -finf();
  for (int c = B.wave; c < nchunks; c += NW) {
    if (ragged && c == nchunks - 1)
      stats_chunk<T, NT, true>(srow, trow, V, c, B.lane, keep_chunks, B.sh, Ms, Mt, Ss, S1, S2, S3,
                               S4, St, T1, tbest, tidx, dmin, dmax);
    else
      stats_chunk<T, NT, false>(srow, trow, V, c, B.lane, keep_chunks, B.sh, Ms, Mt, Ss, S1, S2, S3,
                                S4, St, T1, tbest, tidx, dmin, dmax);
  }
  RowStats R;
  R.ms = B.max(Ms);
  R.mt = B.max(Mt);
  // rescale each wave's sums to the row maxima, then add in a fixed order
  const double gs = (Ms == -finf()) ? 0.0 : (Ms == R.ms) ? 1.0 : static_cast<double>(fexp2((Ms - R.ms) * LOG2E));
  const double gt = (Mt == -finf()) ? 0.0 : (Mt == R.mt) ? 1.0 : static_cast<double>(fexp2((Mt - R.mt) * LOG2E));
  double v[7] = {Ss * gs, S1 * gs, S2 * gs, S3 * gs, S4 * gs, St * gt, T1 * gt};
  B.sum(v);
  B.argmax(tbest, tidx);
  R.dmin = B.min(dmin);
  R.dmax = B.max(dmax);
  R.tmax = tbest;
  R.vstar = tidx;
  R.sum_s = v[0];
  R.lse_s = static_cast<double>(R.ms) + log(v[0]);
  R.lse_t = static_cast<double>(R.mt) + log(v[5]);
  const double Ed = v[1] / v[0], E2 = v[2] / v[0], E3 = v[3] / v[0], E4 = v[4] / v[0];
  R.var = fmax(E2 - Ed * Ed, 0.0);
  R.k3 = E3 - 3.0 * Ed * E2 + 2.0 * Ed * Ed * Ed;
  R.k4 = (E4 - 4.0 * Ed * E3 + 6.0 * Ed * Ed * E2 - 3.0 * Ed * Ed * Ed * Ed) - 3.0 * R.var * R.var;
  R.kl1_est = v[6] / v[5] - (R.lse_t - R.lse_s);
  R.c = static_cast<float>(Ed);
  R.finite = isfinite(R.lse_s) && isfinite(R.lse_t) && isfinite(Ed) && isfinite(v[2]) &&
             isfinite(R.dmin) && isfinite(R.dmax) && isfinite(R.ms) &&
             isfinite(R.mt);
  return R;
}

// ---------------------------------------------------------------------------
// Lambda sweep: sums at NC candidate lambdas.  For candidate j the weights are
// w_v = p~_v * exp(lam_j x_v - sig_j), p~_v = exp(s_v - ms), x_v = d_v - c.
// With sig_j = 0 the sum of (w - p~) is kept instead of the sum of w, so that
// A(lam) = log1p(sum(w - p~) / sum p~) keeps its relative precision when lam
// is small.  sig_j > 0 only when lam_j * (dmax - c) could overflow float.
// ---------------------------------------------------------------------------
// exp(y) - 1 for |y| < 1/16 to ~1e-7 relative: the Taylor polynomial through
// y^4 / 24 (the next term is below y^5 / 120).
__device__ __forceinline__ float expm1_small(float y) {
  return y * fmaf(y, fmaf(y, fmaf(y, 1.0f / 24.0f, 1.0f / 6.0f), 0.5f), 1.0f);
}

template <typename T, int NT, int NC, bool TAIL, bool ACC>
__device__ __forceinline__ void lam_chunk(const T* srow, const T* trow, int V, int c, int lane,
                                          float ms, float cf, const float* lam, const float* sigl,
                                          double& B0, double (&W)[NC], double (&S1)[NC],
                                          double (&S2)[NC]) {
  float s[EPL], t[EPL];
  uint32_t vm;
  load_lane<T, TAIL>(srow, c, lane, V, s, &vm);
  load_lane<T, TAIL>(trow, c, lane, V, t, &vm);
  float b0 = 0.f, w0[NC], s1[NC], s2[NC];
#pragma unroll
  for (int j = 0; j < NC; ++j) { w0[j] = 0.f; s1[j] = 0.f; s2[j] = 0.f; }
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    if (!TAIL || ((vm >> e) & 1u)) {
      const float a = (s[e] - ms) * LOG2E;
      const float pt = fexp2(a);
      const float x = (t[e] - s[e]) - cf;
      const float xl = x * LOG2E;
      b0 += pt;
#pragma unroll
      for (int j = 0; j < NC; ++j) {
        if (ACC) {
          // w - p~ = p~ * expm1(lam x), with expm1 accurate for small |lam x|
          // (used when the KL being resolved is small; requires sig = 0)
          const float y = lam[j] * x;
          const float e = fexp2(y * LOG2E);
          const float em1 = (fabsf(y) < 0.0625f) ? expm1_small(y) : (e - 1.0f);
          const float w = pt * e;
          w0[j] = fmaf(pt, em1, w0[j]);
          const float wx = w * x;
          s1[j] += wx;
          s2[j] = fmaf(wx, x, s2[j]);
        } else {
          const float w = fexp2(fmaf(lam[j], xl, a) - sigl[j]);
          w0[j] += (sigl[j] == 0.f) ? (w - pt) : w;
          const float wx = w * x;
          s1[j] += wx;
          s2[j] = fmaf(wx, x, s2[j]);
        }
      }
    }
  }
  B0 += static_cast<double>(b0);
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    W[j] += static_cast<double>(w0[j]);
    S1[j] += static_cast<double>(s1[j]);
    S2[j] += static_cast<double>(s2[j]);
  }
}

template <typename T, int NT, int NC, bool ACC = false>
__device__ void lam_sweep(Block<NT>& B, const T* srow, const T* trow, int V, const RowStats& R,
                          const float (&lam)[NC], LamEval (&out)[NC]) {
  constexpr int NW = NT / WAVE;
  const int nchunks = (V + CHUNK - 1) / CHUNK;
  const bool ragged = (V % CHUNK) != 0;
  // overflow guard: keep lam * x - sig <= 60 (natural units) for every entry;
  // sigl is the shift in log2 units
  float sigl[NC];
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const double top = static_cast<double>(lam[j]) * (static_cast<double>(R.dmax) - R.c);
    sigl[j] = (!ACC && top > 60.0) ? static_cast<float>((top - 60.0) * static_cast<double>(LOG2E)) : 0.0f;
  }
  double B0 = 0, W[NC], S1[NC], S2[NC];
#pragma unroll
  for (int j = 0; j < NC; ++j) { W[j] = 0; S1[j] = 0; S2[j] = 0; }
  for (int c = B.wave; c < nchunks; c += NW) {
    if (ragged && c == nchunks - 1)
      lam_chunk<T, NT, NC, true, ACC>(srow, trow, V, c, B.lane, R.ms, R.c, lam, sigl, B0, W, S1, S2);
    else
      lam_chunk<T, NT, NC, false, ACC>(srow, trow, V, c, B.lane, R.ms, R.c, lam, sigl, B0, W, S1, S2);
  }
  double v[1 + 3 * NC];
  v[0] = B0;
#pragma unroll
  for (int j = 0; j < NC; ++j) { v[1 + 3 * j] = W[j]; v[2 + 3 * j] = S1[j]; v[3 + 3 * j] = S2[j]; }
  B.sum(v);
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const double b0 = v[0], w = v[1 + 3 * j], s1 = v[2 + 3 * j], s2 = v[3 + 3 * j];
    // sigl is in log2 units: the shift in natural units is sigl * ln 2
    const double sh = static_cast<double>(sigl[j]) * LN2_D;
    LamEval& E = out[j];
    E.lam = lam[j];
    double S0;
    if (sigl[j] == 0.f) {
      S0 = b0 + w;
      E.A = log1p(w / b0);
    } else {
      S0 = w;
      E.A = sh + log(w / b0);
    }
    E.Eq = s1 / S0;
    E.Var = fmax(s2 / S0 - E.Eq * E.Eq, 0.0);
    const double l = static_cast<double>(lam[j]);
    E.KL = fmax(l * E.Eq - E.A, 0.0);  // non-negative; rounding can give -1e-16 when p ~ pi
    E.KLp = l * E.Var;
  }
}

// Rows whose KL (the radius, or KL(pi||p) at the teacher endpoint) is below
// this use the expm1 forms of the sweeps.
constexpr double KL_ACCURATE = 0.01;

// Result of the lambda search.
struct LamResult {
  float lam;   // lambda*
  double A;    // A(lambda*) = log sum_v p_v exp(lambda* x_v), x = d - c
  double KL;   // KL(q_lambda* || p)
  float c;     // centring constant used by A (may differ from RowStats::c)
};

// Degree-8 Hermite interpolant of A(lambda) through three nodes carrying
// A, A' and A'' (Newton divided differences with each node repeated three
// times).  KL(lambda) = lambda A'(lambda) - A(lambda) on the interpolant.
struct Hermite3 {
  double z[9], a[9];
  __device__ void build(const LamEval (&E)[3]) {
    // in-place divided differences; order 1 and 2 differences over a repeated
    // node are A' and A'' / 2 at that node
    for (int i = 0; i < 9; ++i) {
      z[i] = E[i / 3].lam;
      a[i] = E[i / 3].A;
    }
    for (int j = 1; j < 9; ++j) {
      for (int i = 8; i >= j; --i) {
        if (z[i] == z[i - j]) {
          a[i] = (j == 1) ? E[i / 3].Eq : 0.5 * E[i / 3].Var;
        } else {
          a[i] = (a[i] - a[i - 1]) / (z[i] - z[i - j]);
        }
      }
    }
  }
  // A, A', A'' at l
  __device__ void eval(double l, double& p0, double& p1, double& p2) const {
    double p = a[8], dp = 0.0, ddp = 0.0;
    for (int j = 7; j >= 0; --j) {
      const double h = l - z[j];
      ddp = ddp * h + 2.0 * dp;
      dp = dp * h + p;
      p = p * h + a[j];
    }
    p0 = p; p1 = dp; p2 = ddp;
  }
  // |d/dl (l * T'(l) - T(l))|-style size of the top Newton term T, an
  // estimate of the interpolant's truncation error in KL at l
  __device__ double top_term(double l) const {
    double prod = a[8], dprod = 0.0;
    for (int j = 0; j < 8; ++j) {
      const double h = l - z[j];
      dprod = dprod * h + prod;
      prod = prod * h;
    }
    return fabs(l * dprod - prod);
  }
  // root of lambda A' - A = eps in [lo, hi], where KL(lo) <= eps < KL(hi)
  __device__ double solve(double eps, double lo, double hi) const {
    double l = 0.5 * (lo + hi);
    for (int it = 0; it < 60; ++it) {
      double A0, A1, A2;
      eval(l, A0, A1, A2);
      const double f = l * A1 - A0 - eps;
      if (f <= 0) lo = l; else hi = l;
      const double fp = l * A2;
      double nl = (fp > 0) ? l - f / fp : 0.5 * (lo + hi);
      if (!(nl > lo && nl < hi)) nl = 0.5 * (lo + hi);
      if (fabs(nl - l) <= 1e-15 * l) { l = nl; break; }
      l = nl;
    }
    return l;
  }
};

// Start of the search from the cumulants of d under p:
// KL(lam) = sum_n (n - 1) kappa_n lam^n / n! ~ k2 lam^2/2 + k3 lam^3/3 + k4 lam^4/8.
__device__ inline double cumulant_start(const RowStats& R, double eps) {
  if (!(R.var > 0)) return 0.5;
  const double l2 = sqrt(2.0 * eps / R.var);
  double l = l2;
  for (int it = 0; it < 20; ++it) {
    const double f = R.var * l * l / 2 + R.k3 * l * l * l / 3 + R.k4 * l * l * l * l / 8 - eps;
    const double fp = R.var * l + R.k3 * l * l + R.k4 * l * l * l / 2;
    if (!(fp > 0)) { l = l2; break; }
    const double nl = l - f / fp;
    if (!(nl > 0.25 * l2 && nl < 4.0 * l2)) { l = l2; break; }
    l = nl;
  }
  return l;
}

// Largest lambda in [0, 1] with KL(q_lambda || p) <= eps (Eq. trust_region).
// Each lambda sweep evaluates a symmetric three-node stencil {c - h, c, c + h}
// (shifted below 1 when it would pass the teacher endpoint).  When the nodes
// bracket the root, the Hermite interpolant of A gives lambda* and A(lambda*);
// its top Newton term bounds the truncation error, and a stencil whose
// estimate exceeds HERMITE_TOL * eps is followed by a tight +-2% stencil.
template <typename T, int NT>
__device__ LamResult lambda_search(Block<NT>& B, const T* srow, const T* trow, int V,
                                   const RowStats& R, double eps) {
  LamResult out;
  if (R.dmin == R.dmax) {
    // t - s constant: p = pi, KL = 0 for every lambda, lambda* = 1, q = p
    out.lam = 1.0f; out.A = 0.0; out.KL = 0.0; out.c = R.dmin;
    return out;
  }
  out.c = R.c;
  if (eps == 0.0) {
    out.lam = 0.0f; out.A = 0.0; out.KL = 0.0;
    return out;
  }
  // A KL below KL_ACCURATE is resolved with the expm1 form of the sweep: the
  // plain form carries ~2^-24 absolute error per weight, too much next to a
  // KL of that size.  Its overflow guard needs lam * (dmax - c) <= 60.
  const bool acc_ok = (static_cast<double>(R.dmax) - R.c) <= 60.0;
  bool acc = eps < KL_ACCURATE && acc_ok;
  constexpr double DELTA0 = 0.25;       // first stencil half-width, relative
  constexpr double DELTA_TIGHT = 0.02;  // refinement stencil half-width
  constexpr double HERMITE_TOL = 1e-6;  // accepted truncation estimate, relative to eps
  constexpr double LMAX = 1.0 - 1e-6;
  double lo = 0.0, hi = 1.0;  // KL(lo) <= eps < KL(hi) (hi = 1 until a node above is seen)
  LamEval feas;               // the largest evaluated lambda that is feasible (lambda = 0 is)
  feas.lam = 0.0f; feas.A = 0.0; feas.KL = 0.0;
  double lg = fmin(fmax(cumulant_start(R, eps), 1e-7), LMAX);
  double delta = DELTA0;
  bool try_one = R.kl1_est <= 1.05 * eps + 1e-5;
  for (int sweep = 0; sweep < 12; ++sweep) {
    double h = delta * lg;
    double c0 = lg;
    if (try_one) {
      h = delta / (1.0 + delta);
      c0 = 1.0 - h;
    } else if (lg + h > 1.0) {
      h = fmin(h, 0.49);
      c0 = 1.0 - h;
    }
    float L[3] = {static_cast<float>(c0 - h), static_cast<float>(c0),
                  static_cast<float>(fmin(c0 + h, 1.0))};
    if (!(L[0] > 0.0f && L[0] < L[1] && L[1] < L[2])) {  // spacing below float resolution
      L[1] = static_cast<float>(c0);
      L[0] = static_cast<float>(c0 * (1 - 4e-6));
      L[2] = static_cast<float>(fmin(c0 * (1 + 4e-6), 1.0));
    }
    LamEval E[3];
    if (acc) lam_sweep<T, NT, 3, true>(B, srow, trow, V, R, L, E);
    else lam_sweep<T, NT, 3>(B, srow, trow, V, R, L, E);
    if (L[2] == 1.0f && E[2].KL <= eps) {
      if (!acc && acc_ok && E[2].KL < KL_ACCURATE) {
        acc = true;  // resolve a small endpoint KL with the accurate form
        try_one = true;
        continue;
      }
      out.lam = 1.0f; out.A = E[2].A; out.KL = E[2].KL;
      return out;
    }
    try_one = false;
    for (int j = 0; j < 3; ++j) {
      if (E[j].KL <= eps) {
        if (static_cast<double>(L[j]) >= lo) { lo = L[j]; feas = E[j]; }
      } else {
        hi = fmin(hi, static_cast<double>(L[j]));
      }
    }
    if (E[0].KL <= eps && eps < E[2].KL) {
      Hermite3 H;
      H.build(E);
      const int k = (E[1].KL <= eps) ? 1 : 0;
      const double root = H.solve(eps, L[k], L[k + 1]);
      const double h0 = static_cast<double>(L[1]) - L[0], h1 = static_cast<double>(L[2]) - L[1];
      const bool regular = h1 <= 1.5 * h0 && h0 <= 1.5 * h1;
      const bool accurate = H.top_term(root) <= HERMITE_TOL * eps;
      if ((regular && (accurate || delta <= 1.05 * DELTA_TIGHT)) || sweep >= 10) {
        const float lf = static_cast<float>(root);
        double A0, A1, A2;
        H.eval(static_cast<double>(lf), A0, A1, A2);
        out.lam = lf;
        out.A = A0;
        out.KL = fmax(static_cast<double>(lf) * A1 - A0, 0.0);
        return out;
      }
      lg = fmin(root, LMAX);
      delta = DELTA_TIGHT;
      continue;
    }
    // root outside the stencil: Newton in log KL from the nearest node
    const bool above = E[2].KL < eps;
    const LamEval& n = above ? E[2] : E[0];
    double g = above ? 0.5 * (static_cast<double>(n.lam) + hi) : 0.5 * (lo + n.lam);
    if (n.KL > 0 && n.KLp > 0) {
      const double t = n.lam - (log(n.KL) - log(eps)) * n.KL / n.KLp;
      if (t > lo && t < hi) g = t;
    }
    g = fmin(fmax(g, 1e-7), LMAX);
    delta = fmin(fmax(fabs(g - n.lam) / g, DELTA_TIGHT), 0.3);
    lg = g;
    if (above && L[2] < 1.0f && hi >= 1.0) try_one = lg * (1.0 + delta) >= 1.0;
  }
  // not reached in practice (the bracket shrinks every sweep): keep the
  // largest feasible evaluated lambda
  out.lam = feas.lam; out.A = feas.A; out.KL = feas.KL;
  return out;
}

// ---------------------------------------------------------------------------
// Final sweep at lambda*: TV, residual chunk masses, gradient row.
//   p_v = p~_v / sum_s,  q_v / p_v = exp(lam* x_v - A*),
//   w_v = p_v [q_v/p_v - 1]_+ ;  grad_v = coef * (p_v - 1[v = hot]).
// ---------------------------------------------------------------------------
// Residual weight [q_v - p_v]_+ and p_v of one entry; the residual race uses
// the same function so that its weights are bit-identical to the chunk masses.
// With ACC the ratio minus one, q/p - 1 = expm1(lam x - A), uses the small-
// argument polynomial near zero (rows whose KL, and so every q/p - 1, is small).
template <bool ACC>
__device__ __forceinline__ float res_weight(float s, float t, float ms, float invS, float cf,
                                            float laml, float Al, float* p_out) {
  const float p = fexp2((s - ms) * LOG2E) * invS;
  const float x = (t - s) - cf;
  const float y2 = fmaf(laml, x, -Al);  // log2 of q/p
  *p_out = p;
  if (ACC) {
    const float y = y2 * LN2;
    const float em1 = (fabsf(y) < 0.0625f) ? expm1_small(y) : (fexp2(y2) - 1.0f);
    return p * fmaxf(em1, 0.0f);
  }
  return p * fmaxf(fexp2(y2) - 1.0f, 0.0f);
}

template <typename T, typename G, int NT, bool TAIL, bool GRAD, bool ACC>
__device__ __forceinline__ void final_chunk(const T* srow, const T* trow, G* grow, int V, int c,
                                            int lane, float ms, float invS, float cf, float laml,
                                            float Al, bool keep_res, float coef, int hot,
                                            RowShared<NT>& sh, double& TV) {
  float s[EPL], t[EPL];
  uint32_t vm;
  load_lane<T, TAIL>(srow, c, lane, V, s, &vm);
  load_lane<T, TAIL>(trow, c, lane, V, t, &vm);
  float tv = 0.f;
  float g[EPL];
  const int base = c * CHUNK;
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    float p;
    const float w = res_weight<ACC>(s[e], t[e], ms, invS, cf, laml, Al, &p);
    if (!TAIL || ((vm >> e) & 1u)) tv += w;
    if (GRAD) g[e] = coef * (p - ((base + elem_offset(lane, e) == hot) ? 1.0f : 0.0f));
  }
  if (keep_res) {
    const float m = wave_sum(tv);
    if (lane == 0) sh.chunk_a[c] = m;
  }
  TV += static_cast<double>(tv);
  if (GRAD) store_lane<G, TAIL>(grow, c, lane, V, g);
}

template <typename T, typename G, int NT, bool GRAD, bool ACC>
__device__ double final_sweep(Block<NT>& B, const T* srow, const T* trow, G* grow, int V,
                              const RowStats& R, const LamResult& L, bool keep_res, float coef,
                              int hot) {
  constexpr int NW = NT / WAVE;
  const int nchunks = (V + CHUNK - 1) / CHUNK;
  const bool ragged = (V % CHUNK) != 0;
  const float invS = static_cast<float>(1.0 / R.sum_s);
  const float laml = L.lam * LOG2E;
  const float Al = static_cast<float>(L.A * static_cast<double>(LOG2E));
  double TV = 0;
  for (int c = B.wave; c < nchunks; c += NW) {
    if (ragged && c == nchunks - 1)
      final_chunk<T, G, NT, true, GRAD, ACC>(srow, trow, grow, V, c, B.lane, R.ms, invS, L.c, laml,
                                             Al, keep_res, coef, hot, B.sh, TV);
    else
      final_chunk<T, G, NT, false, GRAD, ACC>(srow, trow, grow, V, c, B.lane, R.ms, invS, L.c, laml,
                                              Al, keep_res, coef, hot, B.sh, TV);
  }
  double v[1] = {TV};
  B.sum(v);
  return v[0];
}

// Gradient-only sweep for rows that carry no coupling (non-finite rows, or
// the standalone routed loss): grad_v = coef * (p_v - 1[v = hot]).
template <typename T, typename G, int NT, bool TAIL>
__device__ __forceinline__ void grad_chunk(const T* srow, G* grow, int V, int c, int lane, float ms,
                                           float invS, float coef, int hot, bool nan_row) {
  float s[EPL];
  uint32_t vm;
  load_lane<T, TAIL>(srow, c, lane, V, s, &vm);
  float g[EPL];
  const int base = c * CHUNK;
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    const float p = fexp2((s[e] - ms) * LOG2E) * invS;
    g[e] = nan_row ? __builtin_nanf("") : coef * (p - ((base + elem_offset(lane, e) == hot) ? 1.0f : 0.0f));
  }
  store_lane<G, TAIL>(grow, c, lane, V, g);
}

template <typename T, typename G, int NT>
__device__ void grad_sweep(Block<NT>& B, const T* srow, G* grow, int V, float ms, double sum_s,
                           float coef, int hot, bool nan_row) {
  constexpr int NW = NT / WAVE;
  const int nchunks = (V + CHUNK - 1) / CHUNK;
  const bool ragged = (V % CHUNK) != 0;
  const float invS = static_cast<float>(1.0 / sum_s);
  for (int c = B.wave; c < nchunks; c += NW) {
    if (ragged && c == nchunks - 1)
      grad_chunk<T, G, NT, true>(srow, grow, V, c, B.lane, ms, invS, coef, hot, nan_row);
    else
      grad_chunk<T, G, NT, false>(srow, grow, V, c, B.lane, ms, invS, coef, hot, nan_row);
  }
}

// ---------------------------------------------------------------------------
// Two-level exponential races (the sampler this library fixes for z ~ p and
// c ~ [q - p]_+): the chunk with the smallest E_c / W_c wins, then the entry
// of that chunk with the smallest E_v / w_v; ties to the lowest index.  Keys
// are compared as ln E - ln w.
// ---------------------------------------------------------------------------

// Chunk level.  logw(c) returns ln W_c up to a row constant, or -inf.
template <int NT, typename F>
__device__ int chunk_race(Block<NT>& B, int nchunks, uint64_t seed, uint32_t stream, uint64_t g,
                          F logw) {
  double best = __builtin_huge_val();
  int bi = 0x7fffffff;
  for (int c = B.tid; c < nchunks; c += NT) {
    const double lw = logw(c);
    if (lw > -__builtin_huge_val()) {
      const double u = static_cast<double>(philox_uniform(seed, stream, g, static_cast<uint32_t>(c)));
      const double key = log(-log(u)) - lw;
      if (key < best) { best = key; bi = c; }
    }
  }
  B.argmin(best, bi);
  return bi;
}

// Entry level inside chunk c.  logw(v) returns ln w_v up to a row constant, or -inf.
template <int NT, typename F>
__device__ int elem_race(Block<NT>& B, int c, int V, uint64_t seed, uint32_t stream, uint64_t g,
                         F logw) {
  float best = finf();
  int bi = 0x7fffffff;
  const int lo = c * CHUNK;
  const int hi = min(V, lo + CHUNK);
  for (int v = lo + B.tid; v < hi; v += NT) {
    const float lw = logw(v);
    if (lw > -finf()) {
      const float u = philox_uniform(seed, stream, g, static_cast<uint32_t>(v));
      const float E = -flog2(u) * LN2;
      const float key = flog2(E) * LN2 - lw;
      if (key < best) { best = key; bi = v; }
    }
  }
  B.argmin(best, bi);
  return bi;
}

}  // namespace saki
