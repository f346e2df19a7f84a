// Per-row passes of the SAKI coupling path.  One workgroup of NT threads owns
// one row at a time; chunk c of the row (1024 entries) belongs to wave c % NW,
// which streams its chunks with the loads of its next chunk in flight.
//
//  stats sweep   : max / log-sum-exp of s and t, teacher argmax, p-moments of
//                  d = t - s, min/max of d, per-chunk proposal masses.
//  lambda sweeps : sums over the row at three candidate lambdas, giving
//                  A(lambda) = log sum_v p_v exp(lambda x_v) (x = d - c), A'
//                  and A''; KL(q_lambda || p) = lambda A' - A, KL' = lambda A''.
//  final sweep   : TV(p, q) = sum_v p_v [q_v/p_v - 1]_+, residual chunk
//                  masses, and (optionally) the gradient row.
// Exponents are taken in log2 units: X = x log2(e), so p_v e^{lambda x_v} =
// p_v 2^{lambda X_v}, and every weight costs one exp2.
// (SAKI Sec. 3.2 Eq. bridge / Eq. trust_region; Sec. 3.3; Sec. 3.4; App. E.)
#pragma once

#include <type_traits>

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
  float cL;            // c log2(e) rounded to float; X = fma(d, log2 e, -cL)
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
  double lam, A, Eq, Var, KL, KLp;
};

template <int NT, typename SH = RowShared<NT>>
struct Block {
  static constexpr int NW = NT / WAVE;
  int tid, lane, wave;
  SH& sh;
  __device__ Block(SH& s) : sh(s) {
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
// Chunk streaming.  body(tail, s, t, vm, c) gets this lane's 16 entries of s
// and t in chunk c (elem_offset layout) and the valid mask vm; tail is a
// std::integral_constant<bool, TAIL> (TAIL: the ragged last chunk).  Full
// chunks are visited with the next chunk's loads already issued.
// ---------------------------------------------------------------------------
template <typename T, int NW, typename Body>
__device__ __forceinline__ void for_chunks(const T* srow, const T* trow, int V, int wave, int lane,
                                           Body&& body) {
  const int nfull = V / CHUNK;
  if (wave < nfull) {
    Frag<T> fs, ft;
    frag_load(fs, srow, wave, lane);
    frag_load(ft, trow, wave, lane);
    for (int c = wave; c < nfull; c += NW) {
      Frag<T> ns, nt;
      if (c + NW < nfull) {
        frag_load(ns, srow, c + NW, lane);
        frag_load(nt, trow, c + NW, lane);
      }
      float s[EPL], t[EPL];
      frag_unpack(fs, s);
      frag_unpack(ft, t);
      body(std::integral_constant<bool, false>(), s, t, 0xffffu, c);
      fs = ns;
      ft = nt;
    }
  }
  if ((V % CHUNK) != 0 && (nfull % NW) == wave) {
    float s[EPL], t[EPL];
    uint32_t vm;
    load_lane<T, true>(srow, nfull, lane, V, s, &vm);
    load_lane<T, true>(trow, nfull, lane, V, t, &vm);
    body(std::integral_constant<bool, true>(), s, t, vm, nfull);
  }
}

#define SAKI_VALID(e) (!TAIL || ((vm >> (e)) & 1u))

// ---------------------------------------------------------------------------
// Stats sweep.
// ---------------------------------------------------------------------------
struct StatsAcc {
  float Ms, Mt;                 // wave-uniform running maxima of s and t
  double Ss, St;                // per-lane sums of exp(s - Ms), exp(t - Mt)
  float S1, S2, S3, S4;         // per-lane p-weighted powers of d (relative to Ms)
  float T1;                     // per-lane pi-weighted sum of d (relative to Mt)
  int tidx;                     // wave-uniform lowest index of the running max of t
  float dmin, dmax;             // per-lane range of d
  __device__ void init() {
    Ms = -finf(); Mt = -finf();
    Ss = St = 0.0;
    S1 = S2 = S3 = S4 = T1 = 0.f;
    tidx = 0x7fffffff;
    dmin = finf(); dmax = -finf();
  }
};

// Exponents are taken relative to the wave's running maxima Ms, Mt, so the
// common chunk needs no cross-lane step before its exp2: only a chunk that
// raises a running maximum (the wave's first chunk, then rarely) reduces it
// over the wave and rescales the sums.  The arguments (x - M) log2(e) have
// an exact subtraction, so the largest terms carry no rounding from the shift.
// The proposal mass of chunk c is kept as (Ms, sum_c exp(s - Ms)).
template <bool TAIL>
__device__ __forceinline__ void stats_math(const float* s, const float* t, uint32_t vm, int c,
                                           int lane, bool keep_chunks, float* ca, float* cb,
                                           StatsAcc& a) {
  float ls = -finf(), lt = -finf(), lmin = finf(), lmax = -finf();
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    if (SAKI_VALID(e)) {
      const float d = t[e] - s[e];
      ls = fmaxf(ls, s[e]);
      lt = fmaxf(lt, t[e]);
      lmin = fminf(lmin, d);
      lmax = fmaxf(lmax, d);
    }
  }
  a.dmin = fminf(a.dmin, lmin);
  a.dmax = fmaxf(a.dmax, lmax);
  if (wave_any(ls > a.Ms)) {
    const float cms = wave_max(ls);
    const float f = fexp2((a.Ms - cms) * LOG2E);
    a.Ss *= static_cast<double>(f);
    a.S1 *= f; a.S2 *= f; a.S3 *= f; a.S4 *= f;
    a.Ms = cms;
  }
  if (wave_any(lt > a.Mt)) {
    // a new running maximum of t: its lowest index in this chunk
    const float cmt = wave_max(lt);
    int li = 0x7fffffff;
#pragma unroll
    for (int e = EPL - 1; e >= 0; --e)
      if (SAKI_VALID(e) && t[e] == cmt) li = c * CHUNK + elem_offset(lane, e);
    a.tidx = wave_min(li);
    const float f = fexp2((a.Mt - cmt) * LOG2E);
    a.St *= static_cast<double>(f);
    a.T1 *= f;
    a.Mt = cmt;
  }
  // normalisers: float sums of four entries (within three roundings each),
  // then double
  double ps = 0.0, pt = 0.0;
  float gs = 0.f, gt = 0.f, p1 = 0.f, p2 = 0.f, p3 = 0.f, p4 = 0.f, t1 = 0.f;
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    float es = fexp2((s[e] - a.Ms) * LOG2E);
    float et = fexp2((t[e] - a.Mt) * LOG2E);
    if (TAIL && !SAKI_VALID(e)) { es = 0.f; et = 0.f; }
    const float d = t[e] - s[e];
    const float ed = es * d;
    const float ed2 = ed * d;
    const float ed3 = ed2 * d;
    p1 += ed;
    p2 += ed2;
    p3 += ed3;
    p4 = fmaf(ed3, d, p4);
    t1 = fmaf(et, d, t1);
    gs += es;
    gt += et;
    if ((e & 3) == 3) {
      ps += static_cast<double>(gs);
      pt += static_cast<double>(gt);
      gs = 0.f;
      gt = 0.f;
    }
  }
  if (keep_chunks) {
    const float csum = static_cast<float>(wave_sum(ps));
    if (lane == 0) {
      *ca = a.Ms;
      *cb = csum;
    }
  }
  a.Ss += ps;
  a.S1 += p1;
  a.S2 += p2;
  a.S3 += p3;
  a.S4 += p4;
  a.St += pt;
  a.T1 += t1;
}

// The block's maxima, rescaled sums, argmax and range of d.
struct StatsBlock {
  float ms, mt;
  double Ss, S1, S2, S3, S4, St, T1;
  float tbest;
  int tidx;
  float dmin, dmax;
};

template <int NT, typename SH>
__device__ StatsBlock stats_combine_block(Block<NT, SH>& B, StatsAcc& a) {
  StatsBlock O;
  O.ms = B.max(a.Ms);
  O.mt = B.max(a.Mt);
  // rescale each wave's sums to the block maxima, then add in a fixed order
  const double gs = (a.Ms == -finf()) ? 0.0 : (a.Ms == O.ms) ? 1.0 : static_cast<double>(fexp2((a.Ms - O.ms) * LOG2E));
  const double gt = (a.Mt == -finf()) ? 0.0 : (a.Mt == O.mt) ? 1.0 : static_cast<double>(fexp2((a.Mt - O.mt) * LOG2E));
  double v[7] = {a.Ss * gs, static_cast<double>(a.S1) * gs, static_cast<double>(a.S2) * gs,
                 static_cast<double>(a.S3) * gs, static_cast<double>(a.S4) * gs, a.St * gt,
                 static_cast<double>(a.T1) * gt};
  B.sum(v);
  O.Ss = v[0]; O.S1 = v[1]; O.S2 = v[2]; O.S3 = v[3]; O.S4 = v[4]; O.St = v[5]; O.T1 = v[6];
  float tb = a.Mt;
  int ti = a.tidx;
  B.argmax(tb, ti);
  O.tbest = tb;
  O.tidx = ti;
  O.dmin = B.min(a.dmin);
  O.dmax = B.max(a.dmax);
  return O;
}

// Row statistics from the (combined) block statistics.
__device__ inline RowStats row_stats_from(const StatsBlock& O) {
  RowStats R;
  R.ms = O.ms;
  R.mt = O.mt;
  R.dmin = O.dmin;
  R.dmax = O.dmax;
  R.tmax = O.tbest;
  R.vstar = O.tidx;
  R.sum_s = O.Ss;
  R.lse_s = static_cast<double>(R.ms) + log(O.Ss);
  R.lse_t = static_cast<double>(R.mt) + log(O.St);
  const double Ed = O.S1 / O.Ss, E2 = O.S2 / O.Ss, E3 = O.S3 / O.Ss, E4 = O.S4 / O.Ss;
  R.var = fmax(E2 - Ed * Ed, 0.0);
  R.k3 = E3 - 3.0 * Ed * E2 + 2.0 * Ed * Ed * Ed;
  R.k4 = (E4 - 4.0 * Ed * E3 + 6.0 * Ed * Ed * E2 - 3.0 * Ed * Ed * Ed * Ed) - 3.0 * R.var * R.var;
  R.kl1_est = O.T1 / O.St - (R.lse_t - R.lse_s);
  R.c = static_cast<float>(Ed);
  if (!isfinite(R.c)) R.c = 0.0f;
  R.cL = R.c * LOG2E;
  R.finite = isfinite(R.lse_s) && isfinite(R.lse_t) && isfinite(R.dmin) && isfinite(R.dmax) &&
             isfinite(R.ms) && isfinite(R.mt);
  return R;
}

template <typename T, int NT>
__device__ RowStats stats_sweep(Block<NT>& B, const T* srow, const T* trow, int V, bool keep_chunks) {
  constexpr int NW = NT / WAVE;
  StatsAcc a;
  a.init();
  for_chunks<T, NW>(srow, trow, V, B.wave, B.lane,
                    [&](auto tail, const float* s, const float* t, uint32_t vm, int c) {
                      constexpr bool TAIL = decltype(tail)::value;
                      stats_math<TAIL>(s, t, vm, c, B.lane, keep_chunks, &B.sh.chunk_a[c],
                                       &B.sh.chunk_b[c], a);
                    });
  return row_stats_from(stats_combine_block(B, a));
}

// ---------------------------------------------------------------------------
// Lambda sweep: sums at three nodes lam_j = base + j step.  For node j the
// weights are w_v = p~_v 2^{lam_j X_v}, p~_v = 2^{a_v}, a_v = (s_v - ms) log2 e.
// The sums kept are W_j = sum (w - p~) (so that A = log1p(W_j / sum p~) keeps
// its relative precision when A is small), S1_j = sum w X, S2_j = sum w X^2.
//   FAST: w_0 = 2^{a + base X}, r = 2^{step X}, w_1 = w_0 r, w_2 = w_1 r
//         (two exp2 for the three nodes; no overflow shifts).
//   GEN : one exp2 per node, with a shift sigl_j (log2 units) where
//         lam_j (dmax - c) could overflow float.
//   ACC : w - p~ = p~ expm1(lam x), with expm1 accurate for small arguments
//         (rows whose KL is small).
// ---------------------------------------------------------------------------
enum LamMode { LAM_FAST = 0, LAM_GEN = 1, LAM_ACC = 2 };

// exp(y) - 1 for |y| < 1/16 to ~1e-7 relative: the Taylor polynomial through
// y^4 / 24 (the next term is below y^5 / 120).
__device__ __forceinline__ float expm1_small(float y) {
  return y * fmaf(y, fmaf(y, fmaf(y, 1.0f / 24.0f, 1.0f / 6.0f), 0.5f), 1.0f);
}

// exp(y) - 1 given e = exp(y): the polynomial where |y| < 1/16, e - 1
// elsewhere (both evaluated, then selected).
__device__ __forceinline__ float expm1_sel(float y, float e) {
  const float poly = expm1_small(y);
  const float em = e - 1.0f;
  return (fabsf(y) < 0.0625f) ? poly : em;
}

struct LamNodes {
  float base, step;  // nodes lam_j = base + j step, exact in float
  float sigl[3];     // GEN: per-node overflow shift (log2 units), else 0
};

template <int MODE, bool TAIL>
__device__ __forceinline__ void lam_math(const float* s, const float* t, uint32_t vm, float ms,
                                         float cL, const LamNodes& N, double (&W)[3],
                                         double (&S1)[3], double (&S2)[3]) {
  float w_[3] = {0.f, 0.f, 0.f}, a_[3] = {0.f, 0.f, 0.f}, q_[3] = {0.f, 0.f, 0.f};
  const float lam[3] = {N.base, N.base + N.step, N.base + 2.0f * N.step};
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    const float a = (s[e] - ms) * LOG2E;
    float pt = fexp2(a);
    const float X = fmaf(t[e] - s[e], LOG2E, -cL);
    float w[3], u[3];
    if (MODE == LAM_FAST) {
      w[0] = fexp2(fmaf(N.base, X, a));
      const float r = fexp2(N.step * X);
      if (TAIL && !SAKI_VALID(e)) { pt = 0.f; w[0] = 0.f; }
      w[1] = w[0] * r;
      w[2] = w[1] * r;
#pragma unroll
      for (int j = 0; j < 3; ++j) u[j] = w[j] - pt;
    } else if (MODE == LAM_GEN) {
#pragma unroll
      for (int j = 0; j < 3; ++j) {
        w[j] = fexp2(fmaf(lam[j], X, a) - N.sigl[j]);
        u[j] = (N.sigl[j] == 0.f) ? (w[j] - pt) : w[j];
        if (TAIL && !SAKI_VALID(e)) { w[j] = 0.f; u[j] = 0.f; }
      }
    } else {
#pragma unroll
      for (int j = 0; j < 3; ++j) {
        const float yl = lam[j] * X;
        const float ee = fexp2(yl);
        w[j] = pt * ee;
        u[j] = pt * expm1_sel(yl * LN2, ee);
        if (TAIL && !SAKI_VALID(e)) { w[j] = 0.f; u[j] = 0.f; }
      }
    }
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const float wx = w[j] * X;
      w_[j] += u[j];
      a_[j] += wx;
      q_[j] = fmaf(wx, X, q_[j]);
    }
  }
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    W[j] += static_cast<double>(w_[j]);
    S1[j] += static_cast<double>(a_[j]);
    S2[j] += static_cast<double>(q_[j]);
  }
}

// A, A', A'' (natural units), KL and KL' at the nodes from the row sums
// v = {W_j, S1_j, S2_j} and b0 = sum p~.
__device__ __forceinline__ void lam_finish(const double* v, double b0, const LamNodes& N,
                                           LamEval (&out)[3]) {
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    const double w = v[3 * j], s1 = v[3 * j + 1], s2 = v[3 * j + 2];
    LamEval& E = out[j];
    E.lam = static_cast<double>(N.base) + j * static_cast<double>(N.step);
    double S0;
    if (N.sigl[j] == 0.f) {
      S0 = b0 + w;
      E.A = log1p(w / b0);
    } else {
      // sigl is in log2 units: the shift in natural units is sigl ln 2
      S0 = w;
      E.A = static_cast<double>(N.sigl[j]) * LN2_D + log(w / b0);
    }
    const double m1 = s1 / S0;  // E_q[X]
    E.Eq = m1 * LN2_D;
    E.Var = fmax(s2 / S0 - m1 * m1, 0.0) * (LN2_D * LN2_D);
    E.KL = fmax(E.lam * E.Eq - E.A, 0.0);  // non-negative; rounding can give -1e-16 when p ~ pi
    E.KLp = E.lam * E.Var;
  }
}

template <typename T, int NT, int MODE>
__device__ void lam_sweep_mode(Block<NT>& B, const T* srow, const T* trow, int V, const RowStats& R,
                               const LamNodes& N, LamEval (&out)[3]) {
  constexpr int NW = NT / WAVE;
  double W[3] = {0, 0, 0}, S1[3] = {0, 0, 0}, S2[3] = {0, 0, 0};
  for_chunks<T, NW>(srow, trow, V, B.wave, B.lane,
                    [&](auto tail, const float* s, const float* t, uint32_t vm, int c) {
                      constexpr bool TAIL = decltype(tail)::value;
                      lam_math<MODE, TAIL>(s, t, vm, R.ms, R.cL, N, W, S1, S2);
                    });
  double v[9];
#pragma unroll
  for (int j = 0; j < 3; ++j) { v[3 * j] = W[j]; v[3 * j + 1] = S1[j]; v[3 * j + 2] = S2[j]; }
  B.sum(v);
  lam_finish(v, R.sum_s, N, out);
}

// Evaluates the nodes base + j step (j = 0, 1, 2) over the whole row; acc
// selects the expm1 form.  Every thread gets the same E.
template <typename T, int NT>
__device__ void lam_sweep(Block<NT>& B, const T* srow, const T* trow, int V, const RowStats& R,
                          float base, float step, bool acc, LamEval (&E)[3]) {
  LamNodes N;
  N.base = base;
  N.step = step;
  N.sigl[0] = N.sigl[1] = N.sigl[2] = 0.f;
  const double top = static_cast<double>(R.dmax) - R.c;  // largest x
  const double lam2 = static_cast<double>(base) + 2.0 * step;
  if (acc) {
    lam_sweep_mode<T, NT, LAM_ACC>(B, srow, trow, V, R, N, E);
  } else if (lam2 * top <= 60.0 && static_cast<double>(step) * top <= 20.0) {
    // no weight can overflow, and where a node-0 weight underflows the node 1
    // and 2 weights are below 2^-60 of the row sum
    lam_sweep_mode<T, NT, LAM_FAST>(B, srow, trow, V, R, N, E);
  } else {
    // keep lam_j x - sig_j <= 60 (natural units) for every entry
    for (int j = 0; j < 3; ++j) {
      const double tj = (static_cast<double>(base) + j * static_cast<double>(step)) * top;
      N.sigl[j] = (tj > 60.0) ? static_cast<float>((tj - 60.0) * static_cast<double>(LOG2E)) : 0.0f;
    }
    lam_sweep_mode<T, NT, LAM_GEN>(B, srow, trow, V, R, N, E);
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
  float cL;    // c log2(e) as used in X = fma(d, log2 e, -cL)
  bool qp;     // q = p exactly (eps = 0, or t - s constant): the sweeps use lambda 0
  // x of one entry exactly as the sweeps see it: X ln 2, X = fma(d, log2 e, -cL)
  __device__ double x_of(float s, float t) const {
    return (static_cast<double>(LOG2E) * (static_cast<double>(t) - static_cast<double>(s)) -
            static_cast<double>(cL)) * LN2_D;
  }
  // log q(v) - log p(v) = lam x_v - A (exactly 0 when q = p)
  __device__ double log_ratio(float s, float t) const {
    return qp ? 0.0 : static_cast<double>(lam) * x_of(s, t) - A;
  }
};

// Degree-8 Hermite interpolant of A(lambda) through three nodes carrying
// A, A' and A'' (Newton divided differences with each node repeated three
// times).  KL(lambda) = lambda A'(lambda) - A(lambda) on the interpolant.
struct Hermite3 {
  double z[9], a[9];
  __device__ void build(const LamEval (&E)[3]) {
    // in-place divided differences; order 1 and 2 differences over a repeated
    // node are A' and A'' / 2 at that node
#pragma unroll
    for (int i = 0; i < 9; ++i) {
      z[i] = E[i / 3].lam;
      a[i] = E[i / 3].A;
    }
#pragma unroll
    for (int j = 1; j < 9; ++j) {
#pragma unroll
      for (int i = 8; i >= j; --i) {
        if (i / 3 == (i - j) / 3) {
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
#pragma unroll
    for (int j = 7; j >= 0; --j) {
      const double h = l - z[j];
      ddp = ddp * h + 2.0 * dp;
      dp = dp * h + p;
      p = p * h + a[j];
    }
    p0 = p; p1 = dp; p2 = ddp;
  }
  // size of d/dl (l T'(l) - T(l)) for the top Newton term T: an estimate of
  // the interpolant's truncation error in KL at l
  __device__ double top_term(double l) const {
    double prod = a[8], dprod = 0.0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const double h = l - z[j];
      dprod = dprod * h + prod;
      prod = prod * h;
    }
    return fabs(l * dprod - prod);
  }
  // root of lambda A' - A = eps in [lo, hi], where KL(lo) <= eps < KL(hi):
  // safeguarded Newton from the secant point; stops once the step is below
  // 1e-13 relative (far under the float resolution lambda* is returned in)
  __device__ double solve(double eps, double lo, double hi, double flo, double fhi) const {
    double l = (flo < 0 && fhi > 0) ? lo + (hi - lo) * (-flo / (fhi - flo)) : 0.5 * (lo + hi);
    for (int it = 0; it < 40; ++it) {
      double A0, A1, A2;
      eval(l, A0, A1, A2);
      const double f = l * A1 - A0 - eps;
      if (f == 0.0) break;
      if (f < 0) lo = l; else hi = l;
      const double fp = l * A2;
      double nl = (fp > 0) ? l - f / fp : 0.5 * (lo + hi);
      if (!(nl > lo && nl < hi)) nl = 0.5 * (lo + hi);
      const bool done = fabs(nl - l) <= 1e-13 * l || (hi - lo) <= 1e-13 * l;
      l = nl;
      if (done) break;
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
// Each lambda sweep evaluates an evenly spaced three-node stencil
// {c - h, c, c + h} (shifted below 1 when it would pass the teacher
// endpoint).  base and step are multiples of q = 2^(floor(log2 c) - 19), so
// the nodes are exact in float and the endpoint node is exactly 1.  When the
// nodes bracket the root, the Hermite interpolant of A gives lambda* and
// A(lambda*); its top Newton term bounds the truncation error, and a stencil
// whose estimate exceeds HERMITE_TOL * eps is followed by a tight +-2% one.
// sweep3(base, step, acc, E) evaluates the three nodes over the whole row.
template <typename Sweep3>
__device__ LamResult lambda_search_with(const RowStats& R, double eps, Sweep3&& sweep3) {
  LamResult out;
  if (R.dmin == R.dmax) {
    // t - s constant: p = pi, KL = 0 for every lambda, lambda* = 1, q = p
    out.lam = 1.0f; out.A = 0.0; out.KL = 0.0; out.c = R.dmin; out.cL = R.dmin * LOG2E; out.qp = true;
    return out;
  }
  out.c = R.c;
  out.cL = R.cL;
  out.qp = false;
  if (eps == 0.0) {
    out.lam = 0.0f; out.A = 0.0; out.KL = 0.0; out.qp = true;
    return out;
  }
  // A KL below KL_ACCURATE is resolved with the expm1 form of the sweep: the
  // plain form carries ~2^-24 absolute error per weight, too much next to a
  // KL of that size.  Its overflow guard needs lam (dmax - c) <= 60.
  const bool acc_ok = (static_cast<double>(R.dmax) - R.c) <= 60.0;
  bool acc = eps < KL_ACCURATE && acc_ok;
  constexpr double DELTA0 = 0.25;       // first stencil half-width, relative
  constexpr double DELTA_TIGHT = 0.02;  // refinement stencil half-width
  constexpr double HERMITE_TOL = 1e-6;  // accepted truncation estimate, relative to eps
  constexpr double LMAX = 1.0 - 1e-6;
  double lo = 0.0, hi = 1.0;  // KL(lo) <= eps < KL(hi) (hi = 1 until a node above is seen)
  LamEval feas;               // the largest evaluated lambda that is feasible (lambda = 0 is)
  feas.lam = 0.0; feas.A = 0.0; feas.KL = 0.0;
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
    // nodes on the grid of q = 2^(floor(log2 c0) - 19)
    int ex;
    frexp(c0, &ex);
    const double q = ldexp(1.0, ex - 20);
    const double step = fmax(rint(h / q), 1.0) * q;
    double base = rint((c0 - step) / q) * q;
    if (try_one || base + 2.0 * step > 1.0) base = 1.0 - 2.0 * step;
    if (!(base > 0.0)) base = step;
    LamEval E[3];
    sweep3(static_cast<float>(base), static_cast<float>(step), acc, E);
    if (E[2].lam == 1.0 && E[2].KL <= eps) {
      if (!acc && acc_ok && E[2].KL < KL_ACCURATE) {
        acc = true;  // resolve a small endpoint KL with the accurate form
        try_one = true;
        continue;
      }
      out.lam = 1.0f; out.A = E[2].A; out.KL = E[2].KL;
      return out;
    }
    try_one = false;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      if (E[j].KL <= eps) {
        if (E[j].lam >= lo) { lo = E[j].lam; feas = E[j]; }
      } else {
        hi = fmin(hi, E[j].lam);
      }
    }
    if (E[0].KL <= eps && eps < E[2].KL) {
      Hermite3 H;
      H.build(E);
      const bool k1 = E[1].KL <= eps;
      const double root = k1 ? H.solve(eps, E[1].lam, E[2].lam, E[1].KL - eps, E[2].KL - eps)
                             : H.solve(eps, E[0].lam, E[1].lam, E[0].KL - eps, E[1].KL - eps);
      const bool accurate = H.top_term(root) <= HERMITE_TOL * eps;
      if (accurate || delta <= 1.05 * DELTA_TIGHT || sweep >= 10) {
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
    double g = above ? 0.5 * (n.lam + hi) : 0.5 * (lo + n.lam);
    if (n.KL > 0 && n.KLp > 0) {
      const double t = n.lam - (log(n.KL) - log(eps)) * n.KL / n.KLp;
      if (t > lo && t < hi) g = t;
    }
    g = fmin(fmax(g, 1e-7), LMAX);
    delta = fmin(fmax(fabs(g - n.lam) / g, DELTA_TIGHT), 0.3);
    lg = g;
    if (above && E[2].lam < 1.0 && hi >= 1.0) try_one = lg * (1.0 + delta) >= 1.0;
  }
  // not reached in practice (the bracket shrinks every sweep): keep the
  // largest feasible evaluated lambda
  out.lam = static_cast<float>(feas.lam); out.A = feas.A; out.KL = feas.KL;
  return out;
}

template <typename T, int NT>
__device__ LamResult lambda_search(Block<NT>& B, const T* srow, const T* trow, int V,
                                   const RowStats& R, double eps) {
  return lambda_search_with(R, eps, [&](float base, float step, bool acc, LamEval (&E)[3]) {
    lam_sweep<T, NT>(B, srow, trow, V, R, base, step, acc, E);
  });
}

// ---------------------------------------------------------------------------
// Final sweep at lambda*: TV, residual chunk masses, gradient row.
//   p_v = p~_v / sum_s,  q_v / p_v = 2^{lam* X_v - A* log2 e},
//   w_v = p_v [q_v/p_v - 1]_+ ;  grad_v = coef * (p_v - 1[v = hot]).
// ---------------------------------------------------------------------------
struct FinalConst {
  float ms, invS, cL, lam, AL;  // AL = A* log2(e)
  bool acc;                     // expm1 form (rows whose KL is small)
};

__device__ inline FinalConst final_const(const RowStats& R, const LamResult& L) {
  FinalConst F;
  F.ms = R.ms;
  F.invS = static_cast<float>(1.0 / R.sum_s);
  F.cL = L.cL;
  F.lam = L.qp ? 0.0f : L.lam;
  F.AL = L.qp ? 0.0f : static_cast<float>(L.A * static_cast<double>(LOG2E));
  F.acc = L.KL < KL_ACCURATE;
  return F;
}

// Residual weight [q_v - p_v]_+ and p_v of one entry; the residual race uses
// the same function, so its weights are bit-identical to the chunk masses'.
template <bool ACC>
__device__ __forceinline__ float res_weight(float s, float t, const FinalConst& F, float* p_out) {
  const float p = fexp2((s - F.ms) * LOG2E) * F.invS;
  const float X = fmaf(t - s, LOG2E, -F.cL);
  const float y2 = fmaf(F.lam, X, -F.AL);  // log2 of q/p
  const float ee = fexp2(y2);
  *p_out = p;
  const float em1 = ACC ? expm1_sel(y2 * LN2, ee) : (ee - 1.0f);
  return p * fmaxf(em1, 0.0f);
}

template <typename T, typename G, int NT, bool GRAD, bool ACC>
__device__ double final_sweep(Block<NT>& B, const T* srow, const T* trow, G* grow, int V,
                              const FinalConst& F, bool keep_res, float coef, int hot) {
  constexpr int NW = NT / WAVE;
  const int hot_chunk = hot >= 0 ? hot / CHUNK : -1;
  double TV = 0;
  for_chunks<T, NW>(srow, trow, V, B.wave, B.lane,
                    [&](auto tail, const float* s, const float* t, uint32_t vm, int c) {
                      constexpr bool TAIL = decltype(tail)::value;
                      float tv = 0.f, g[EPL];
#pragma unroll
                      for (int e = 0; e < EPL; ++e) {
                        float p;
                        const float w = res_weight<ACC>(s[e], t[e], F, &p);
                        if (SAKI_VALID(e)) tv += w;
                        if (GRAD) g[e] = coef * p;
                      }
                      if (GRAD && c == hot_chunk) {
                        // the one entry with the indicator (wave-uniform branch)
#pragma unroll
                        for (int e = 0; e < EPL; ++e) {
                          if (c * CHUNK + elem_offset(B.lane, e) == hot) {
                            float p;
                            res_weight<ACC>(s[e], t[e], F, &p);
                            g[e] = coef * (p - 1.0f);
                          }
                        }
                      }
                      if (keep_res) {
                        const float m = wave_sum(tv);
                        if (B.lane == 0) B.sh.chunk_a[c] = m;
                      }
                      TV += static_cast<double>(tv);
                      if (GRAD) store_lane<G, TAIL>(grow, c, B.lane, V, g);
                    });
  double v[1] = {TV};
  B.sum(v);
  return v[0];
}

#undef SAKI_VALID

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
// are compared as ln E - ln w.  One Philox block gives the uniforms of four
// consecutive indices.
// ---------------------------------------------------------------------------

// Chunk level.  logw(c) returns ln W_c up to a row constant, or -inf.
template <int NT, typename F>
__device__ int chunk_race(Block<NT>& B, int nchunks, uint64_t seed, uint32_t stream, uint64_t g,
                          F logw) {
  double best = __builtin_huge_val();
  int bi = 0x7fffffff;
  for (int j = B.tid; 4 * j < nchunks; j += NT) {
    const uint4 w = philox_block(seed, stream, g, static_cast<uint32_t>(j));
    const uint32_t words[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int c = 4 * j + k;
      if (c < nchunks) {
        const double lw = logw(c);
        if (lw > -__builtin_huge_val()) {
          const double u = static_cast<double>(word_to_uniform(words[k]));
          const double key = log(-log(u)) - lw;
          if (key < best) { best = key; bi = c; }
        }
      }
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
  for (int v0 = lo + 4 * B.tid; v0 < hi; v0 += 4 * NT) {
    const uint4 w = philox_block(seed, stream, g, static_cast<uint32_t>(v0 >> 2));
    const uint32_t words[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int v = v0 + k;
      if (v < hi) {
        const float lw = logw(v);
        if (lw > -finf()) {
          const float u = word_to_uniform(words[k]);
          const float E = -flog2(u) * LN2;
          const float key = flog2(E) * LN2 - lw;
          if (key < best) { best = key; bi = v; }
        }
      }
    }
  }
  B.argmin(best, bi);
  return bi;
}

}  // namespace saki
