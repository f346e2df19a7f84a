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

constexpr int RED_MAX = 16;  // widest block reduction (doubles per thread)

// The stats sweep also evaluates A and its first two derivatives at a middle
// lambda (the weights p^(1 - lam) pi^lam), so that the start of the lambda
// search interpolates A between lambda = 0, that node and 1 instead of
// extrapolating from the ends.  The node sits near where lambda* falls for the
// radius (lambda* ~ sqrt(2 eps / Var_p[d]), Var_p[d] of a few units).
// The stats sweep sums the p-moments of d through d^4 (K34: the third and
// fourth cumulants feed the starts) or through d^2 only.  They pay where
// lambda* is small, close to the node lambda = 0 they describe: radii below
// K34_EPS (lambda* ~ sqrt(2 eps / Var_p[d])); elsewhere the middle and end
// nodes place lambda* as well without them, and in float the higher moments
// of d (not centred) carry more noise than they add.
constexpr double K34_EPS = 0.03;
__host__ __device__ inline bool use_k34(double eps) { return eps < K34_EPS; }

__host__ __device__ inline float mid_lambda(double eps) {
  const double l = 0.5 * sqrt(eps > 0.0 ? eps : 0.0);
  return static_cast<float>(l < 0.05 ? 0.05 : l > 0.5 ? 0.5 : l);
}



// Row-uniform results of the stats sweep.
struct RowStats {
  float ms, mt;        // max s, max t
  double lse_s, lse_t; // log-sum-exp of s and t
  double sum_s;        // sum exp(s - ms)
  float c;             // centring constant: E_p[d] rounded to float
  float cL;            // c log2(e) rounded to float; X = fma(d, log2 e, -cL)
  double mean_p;       // E_p[d]
  double var;          // Var_p[d] = kappa_2 (starting point of the lambda search)
  double k3, k4;       // third and fourth cumulants of d under p
  double mean_pi;      // E_pi[d]
  double var_pi;       // Var_pi[d]
  double kl1_est;      // KL(pi || p) = E_pi[d] - (lse_t - lse_s), a first estimate
  float dmin, dmax;    // range of d = t - s
  float tmax;          // max t
  int vstar;           // argmax t, lowest index on ties
  float t_smax;        // t at an entry holding max s (the dominant entry of p)
  double pmax;         // max_v p_v = exp(ms - lse_s)
  float lam_mid;       // the middle node (mid_lambda)
  bool k34;            // k3, k4 were summed (else 0)
  double mid_A, mid_A1, mid_A2;  // A, A', A'' there
  bool finite;
};

// The row statistics as kept in LDS.
struct RowStatsLDS {
  RowStats r;
};

// MAXC: chunk capacity (rows of up to MAXC * CHUNK entries).  KC > 0 adds a
// row cache of KC chunks per wave (bf16 rows): the stats sweep stores the
// wave's last KC full chunks there and the later sweeps of the row read them
// from LDS instead of memory (4 KiB per chunk: 1 KiB each of s and t per half).
template <int NT, int MAXC = MAX_CHUNKS, int KC = 0>
struct RowShared {
  static constexpr int NW = NT / WAVE;
  static constexpr int CACHE_CHUNKS = KC;
  float chunk_a[MAXC];  // proposal: reference (log2 units) | residual: chunk mass
  float chunk_b[MAXC];  // proposal: chunk sum of 2^(s log2 e - reference)
  float chunk_c[MAXC];  // teacher draw: reference (log2 units)
  float chunk_d[MAXC];  // teacher draw: chunk sum of 2^(t log2 e - reference)
  double red_d[NW][RED_MAX];
  float red_f[NW][4];
  int red_i[NW][4];
  uint4 cache[KC > 0 ? NW * KC * 4 * WAVE : 1];  // [wave][slot][s0, s1, t0, t1][lane]
  RowStatsLDS rs;  // the current row's statistics (stats_sweep)
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

  // (key, index) minimum over the block, ties to the lower index, carrying
  // two floats of the winner along.
  __device__ void argmin_with(float& key, int& idx, float& pa, float& pb) {
#pragma unroll
    for (int o = WAVE / 2; o > 0; o >>= 1) {
      const float k2 = __shfl_xor(key, o, WAVE);
      const int i2 = __shfl_xor(idx, o, WAVE);
      const float a2 = __shfl_xor(pa, o, WAVE);
      const float b2 = __shfl_xor(pb, o, WAVE);
      if (k2 < key || (k2 == key && i2 < idx)) { key = k2; idx = i2; pa = a2; pb = b2; }
    }
    if (lane == 0) {
      sh.red_f[wave][0] = key;
      sh.red_f[wave][1] = pa;
      sh.red_f[wave][2] = pb;
      sh.red_i[wave][0] = idx;
    }
    __syncthreads();
    float bk = sh.red_f[0][0], ba = sh.red_f[0][1], bb = sh.red_f[0][2];
    int bi = sh.red_i[0][0];
    for (int w = 1; w < NW; ++w) {
      const float k2 = sh.red_f[w][0];
      const int i2 = sh.red_i[w][0];
      if (k2 < bk || (k2 == bk && i2 < bi)) { bk = k2; bi = i2; ba = sh.red_f[w][1]; bb = sh.red_f[w][2]; }
    }
    __syncthreads();
    key = bk;
    idx = bi;
    pa = ba;
    pb = bb;
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
// chunks are visited with the next chunk's loads already issued.  LAST marks
// the row's last pass: its loads do not allocate in the caches.
//
// Row cache (bf16 rows, cache != nullptr): the wave's full chunks are
// i = 0 .. nw-1 (chunk wave + i NW); the last kc of them are cached.
// CACHE_FILL (stats sweep) visits every chunk from memory and stores the
// cached ones in LDS; CACHE_USE visits the cached chunks from LDS first (while
// the first memory chunk's loads are in flight), then the others from memory.
// Each wave uses only its own slots, so no barrier is needed between sweeps.
// ---------------------------------------------------------------------------
enum CacheMode { CACHE_NONE = 0, CACHE_FILL = 1, CACHE_USE = 2 };

struct RowCache {
  uint4* lds;  // RowShared::cache, or nullptr
  int kc;      // cached chunks per wave
};

template <typename T, int NW, bool LAST = false, int CM = CACHE_NONE, typename Body>
__device__ __forceinline__ void for_chunks(const T* srow, const T* trow, int V, int wave, int lane,
                                           Body&& body, RowCache rc = RowCache{nullptr, 0}) {
  static_assert(CM == CACHE_NONE || sizeof(T) == 2, "the row cache holds bf16 chunks");
  const int nfull = V / CHUNK;
  const int nw = wave < nfull ? (nfull - 1 - wave) / NW + 1 : 0;  // this wave's full chunks
  const int ncache = (CM == CACHE_NONE || rc.lds == nullptr) ? 0 : min(rc.kc, nw);
  const int first_cached = nw - ncache;
  const int nmem = (CM == CACHE_USE) ? first_cached : nw;  // chunks read from memory
  auto slot = [&](int i, int part) { return rc.lds + ((wave * rc.kc + (i - first_cached)) * 4 + part) * WAVE + lane; };
  auto run = [&](const Frag<T>& fs, const Frag<T>& ft, int c) {
    if constexpr (CM == CACHE_FILL) {
      const int i = (c - wave) / NW;
      if (i >= first_cached) {
        *slot(i, 0) = fs.q[0];
        *slot(i, 1) = fs.q[1];
        *slot(i, 2) = ft.q[0];
        *slot(i, 3) = ft.q[1];
      }
    }
    float s[EPL], t[EPL];
    frag_unpack(fs, s);
    frag_unpack(ft, t);
    body(std::integral_constant<bool, false>(), s, t, 0xffffu, c);
  };
  // two fragment buffers used in turn: chunk c is processed while the
  // loads of the wave's next chunk are in flight, without register copies.
  // The next loads are issued on every path (on the wave's last chunk they
  // re-read chunk c, unused): a load under a branch leaves a join where
  // the compiler's wait counters must assume no younger loads, and it then
  // waits for the next chunk's first load before processing chunk c.
  Frag<T> as, at, bs, bt;
  if (nmem > 0) {
    frag_load<LAST>(as, srow, wave, lane);
    frag_load<LAST>(at, trow, wave, lane);
  }
  if constexpr (CM == CACHE_USE) {
    for (int i = first_cached; i < nw; ++i) {
      Frag<T> cs, ct;
      cs.q[0] = *slot(i, 0);
      cs.q[1] = *slot(i, 1);
      ct.q[0] = *slot(i, 2);
      ct.q[1] = *slot(i, 3);
      float s[EPL], t[EPL];
      frag_unpack(cs, s);
      frag_unpack(ct, t);
      body(std::integral_constant<bool, false>(), s, t, 0xffffu, wave + i * NW);
    }
  }
  if (nmem > 0) {
    const int clast = wave + (nmem - 1) * NW;  // the wave's last chunk read from memory
    int c = wave;
    for (;;) {
      const bool more_b = c < clast;
      const int cb = more_b ? c + NW : c;
      frag_load<LAST>(bs, srow, cb, lane);
      frag_load<LAST>(bt, trow, cb, lane);
      run(as, at, c);
      if (!more_b) break;
      c += NW;
      const bool more_a = c < clast;
      const int ca = more_a ? c + NW : c;
      frag_load<LAST>(as, srow, ca, lane);
      frag_load<LAST>(at, trow, ca, lane);
      run(bs, bt, c);
      if (!more_a) break;
      c += NW;
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

// The chunk loop over one array: body(tail, x, vm, c) gets this lane's 16
// entries of chunk c; full chunks with the next chunk's loads in flight.  The
// row cache works as in for_chunks, with two slots (the two halves of the
// array) per cached chunk: the wave's last kc full chunks.
template <typename T, int NW, int CM = CACHE_NONE, typename Body>
__device__ __forceinline__ void for_chunks1(const T* row, int V, int wave, int lane, Body&& body,
                                            RowCache rc = RowCache{nullptr, 0}) {
  static_assert(CM == CACHE_NONE || sizeof(T) == 2, "the row cache holds bf16 chunks");
  const int nfull = V / CHUNK;
  const int nw = wave < nfull ? (nfull - 1 - wave) / NW + 1 : 0;  // this wave's full chunks
  const int ncache = (CM == CACHE_NONE || rc.lds == nullptr) ? 0 : min(rc.kc, nw);
  const int first_cached = nw - ncache;
  const int nmem = (CM == CACHE_USE) ? first_cached : nw;  // chunks read from memory
  auto slot = [&](int i, int part) { return rc.lds + ((wave * rc.kc + (i - first_cached)) * 2 + part) * WAVE + lane; };
  auto run = [&](const Frag<T>& f, int c) {
    if constexpr (CM == CACHE_FILL) {
      const int i = (c - wave) / NW;
      if (i >= first_cached) {
        *slot(i, 0) = f.q[0];
        *slot(i, 1) = f.q[1];
      }
    }
    float x[EPL];
    frag_unpack(f, x);
    body(std::integral_constant<bool, false>(), x, 0xffffu, c);
  };
  Frag<T> fa, fb;
  if (nmem > 0) frag_load<false>(fa, row, wave, lane);
  if constexpr (CM == CACHE_USE) {
    for (int i = first_cached; i < nw; ++i) {
      Frag<T> cf;
      cf.q[0] = *slot(i, 0);
      cf.q[1] = *slot(i, 1);
      float x[EPL];
      frag_unpack(cf, x);
      body(std::integral_constant<bool, false>(), x, 0xffffu, wave + i * NW);
    }
  }
  if (nmem > 0) {
    const int clast = wave + (nmem - 1) * NW;  // the wave's last chunk read from memory
    int c = wave;
    for (;;) {
      const bool more_b = c < clast;
      frag_load<false>(fb, row, more_b ? c + NW : c, lane);
      run(fa, c);
      if (!more_b) break;
      c += NW;
      const bool more_a = c < clast;
      frag_load<false>(fa, row, more_a ? c + NW : c, lane);
      run(fb, c);
      if (!more_a) break;
      c += NW;
    }
  }
  if ((V % CHUNK) != 0 && (nfull % NW) == wave) {
    float x[EPL];
    uint32_t vm;
    load_lane<T, true>(row, nfull, lane, V, x, &vm);
    body(std::integral_constant<bool, true>(), x, vm, nfull);
  }
}

// The row cache of a workgroup's shared state (none when SH has no slots or
// the rows are not bf16).
template <typename T, typename SH>
__device__ __forceinline__ RowCache row_cache(SH& sh) {
  if constexpr (SH::CACHE_CHUNKS > 0 && sizeof(T) == 2) return RowCache{sh.cache, SH::CACHE_CHUNKS};
  return RowCache{nullptr, 0};
}
template <typename T, typename SH>
constexpr int fill_mode() { return (SH::CACHE_CHUNKS > 0 && sizeof(T) == 2) ? CACHE_FILL : CACHE_NONE; }
template <typename T, typename SH>
constexpr int use_mode() { return (SH::CACHE_CHUNKS > 0 && sizeof(T) == 2) ? CACHE_USE : CACHE_NONE; }

#define SAKI_VALID(e) (!TAIL || ((vm >> (e)) & 1u))

// ---------------------------------------------------------------------------
// Stats sweep.
// ---------------------------------------------------------------------------
// 2^-d0 for d0 = ms log2(e) - msL, the rounding of the float shift msL.
__device__ __forceinline__ double shift_correction(float ms, float msL) {
  const double d0 = static_cast<double>(LOG2E) * static_cast<double>(ms) - static_cast<double>(msL);
  return exp2(-d0);
}

struct StatsAcc {
  float Ms, Mt;                 // wave-uniform running maxima of s and t
  float MsL, MtL;               // Ms log2(e), Mt log2(e) rounded to float
  double Ss, St;                // per-lane sums of 2^(s log2 e - MsL), 2^(t log2 e - MtL)
  float S1, S2, S3, S4;         // per-lane p-weighted powers of d (relative to Ms)
  float T1, T2;                 // per-lane pi-weighted sums of d, d^2 (relative to Mt)
  double Sm;                    // per-lane sum of 2^((1 - lm) as + lm at), lm the middle node
  float Q1, Q2;                 // per-lane d, d^2 under those weights
  int tidx;                     // wave-uniform lowest index of the running max of t
  float t_smax;                 // wave-uniform: t at an entry holding the running max of s
  float dmin, dmax;             // per-lane range of d
  __device__ void init() {
    Ms = -finf(); Mt = -finf();
    MsL = -finf(); MtL = -finf();
    Ss = St = Sm = 0.0;
    S1 = S2 = S3 = S4 = T1 = T2 = 0.f;
    Q1 = Q2 = 0.f;
    tidx = 0x7fffffff;
    t_smax = 0.f;
    dmin = finf(); dmax = -finf();
  }
};

// Exponents are taken relative to the wave's running maxima Ms, Mt, so the
// common chunk needs no cross-lane step before its exp2: only a chunk that
// raises a running maximum (the wave's first chunk, then rarely) reduces it
// over the wave and rescales the sums.  Each exponent is one fma,
// fma(x, log2 e, -ML) with ML = M log2(e) rounded to float, rounded once, so
// the largest terms carry no rounding from the shift; the rounding of ML itself
// is one factor for every term sharing it, removed exactly once the row's
// maxima are known (shift_correction).  The proposal mass of chunk c is kept as
// (MsL, sum_c 2^(s log2 e - MsL)), i.e. ln W_c = MsL ln 2 + ln(sum).
// MID: also the middle node's sums (else the row carries no middle node and
// the lambda search starts from the ends alone); K34: the third and fourth
// p-moments of d.
template <bool TAIL, bool MID, bool K34, typename SH>
__device__ __forceinline__ void stats_math(const float* s, const float* t, uint32_t vm, int c,
                                           int lane, bool keep_chunks, bool keep_teacher, float lm, SH& sh,
                                           StatsAcc& a) {
  // this lane's maxima and range of d over the chunk: chains of three-input
  // max / min (EPL - 1 entries after the first, two per instruction)
  float ls, lt, lmin, lmax;
  {
    float ms[EPL], mt[EPL], dn[EPL], dx[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      const bool ok = SAKI_VALID(e);
      const float d = t[e] - s[e];
      ms[e] = ok ? s[e] : -finf();
      mt[e] = ok ? t[e] : -finf();
      dn[e] = ok ? d : finf();
      dx[e] = ok ? d : -finf();
    }
    static_assert(EPL % 2 == 0, "pairs of entries per max3");
    ls = ms[0]; lt = mt[0]; lmin = dn[0]; lmax = dx[0];
    // entry 0 twice in the first step keeps the chain at EPL / 2 instructions
#pragma unroll
    for (int e = 1; e < EPL; e += 2) {
      const int f = e + 1 < EPL ? e + 1 : e;
      ls = max3_raw(ls, ms[e], ms[f]);
      lt = max3_raw(lt, mt[e], mt[f]);
      lmin = min3_raw(lmin, dn[e], dn[f]);
      lmax = max3_raw(lmax, dx[e], dx[f]);
    }
  }
  a.dmin = fminf(a.dmin, lmin);
  a.dmax = fmaxf(a.dmax, lmax);
  if (wave_any(ls > a.Ms)) {
    const float cms = wave_max(ls);
    // a new running maximum of s: the largest t among the entries holding it
    float lt2 = -finf();
#pragma unroll
    for (int e = 0; e < EPL; ++e)
      if (SAKI_VALID(e) && s[e] == cms) lt2 = fmaxf(lt2, t[e]);
    a.t_smax = wave_max(lt2);
    // rounded product and difference, never contracted into one fma: the sums
    // so far are relative to exactly the MsL the later terms use
    const float cmsL = __fmul_rn(cms, LOG2E);
    const float dsl = __fsub_rn(a.MsL, cmsL);
    const float f = fexp2(dsl);
    a.Ss *= static_cast<double>(f);
    a.S1 *= f; a.S2 *= f; a.S3 *= f; a.S4 *= f;
    const float fm = fexp2((1.0f - lm) * dsl);
    a.Sm *= static_cast<double>(fm);
    a.Q1 *= fm; a.Q2 *= fm;
    a.Ms = cms;
    a.MsL = cmsL;
  }
  if (wave_any(lt > a.Mt)) {
    // a new running maximum of t: its lowest index in this chunk
    const float cmt = wave_max(lt);
    int li = 0x7fffffff;
#pragma unroll
    for (int e = EPL - 1; e >= 0; --e)
      if (SAKI_VALID(e) && t[e] == cmt) li = c * CHUNK + elem_offset(lane, e);
    a.tidx = wave_min(li);
    const float cmtL = __fmul_rn(cmt, LOG2E);
    const float dtl = __fsub_rn(a.MtL, cmtL);
    const float f = fexp2(dtl);
    a.St *= static_cast<double>(f);
    a.T1 *= f;
    a.T2 *= f;
    const float fm = fexp2(lm * dtl);
    a.Sm *= static_cast<double>(fm);
    a.Q1 *= fm; a.Q2 *= fm;
    a.Mt = cmt;
    a.MtL = cmtL;
  }
  // normalisers: float sums of eight entries (within seven roundings each),
  // then double; moments in float
  double ps = 0.0, pt = 0.0, pm = 0.0;
  float gs = 0.f, gt = 0.f, gm = 0.f, p1 = 0.f, p2 = 0.f, p3 = 0.f, p4 = 0.f, t1 = 0.f, t2 = 0.f;
  float q1 = 0.f, q2 = 0.f;
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    const float as = fmaf(s[e], LOG2E, -a.MsL);
    const float at = fmaf(t[e], LOG2E, -a.MtL);
    float es = fexp2(as);
    float et = fexp2(at);
    // the middle node's weight p~^(1 - lm) pi~^lm: its exponent is at most 0
    // (as, at <= 0), so it cannot overflow
    float em = MID ? fexp2(fmaf(lm, at - as, as)) : 0.0f;
    if (TAIL && !SAKI_VALID(e)) { es = 0.f; et = 0.f; em = 0.f; }
    const float d = t[e] - s[e];
    const float d2 = d * d;
    p1 = fmaf(es, d, p1);
    p2 = fmaf(es, d2, p2);
    if (K34) {
      const float ed2 = es * d2;
      p3 = fmaf(ed2, d, p3);
      p4 = fmaf(ed2, d2, p4);
    }
    t1 = fmaf(et, d, t1);
    t2 = fmaf(et, d2, t2);
    if (MID) {
      q1 = fmaf(em, d, q1);
      q2 = fmaf(em, d2, q2);
      gm += em;
    }
    gs += es;
    gt += et;
    if ((e & 7) == 7) {
      ps += static_cast<double>(gs);
      pt += static_cast<double>(gt);
      pm += static_cast<double>(gm);
      gs = 0.f;
      gt = 0.f;
      gm = 0.f;
    }
  }
  // chunk masses (stored as float) by a float reduction
  if (keep_chunks) {
    const float csum = wave_sum(static_cast<float>(ps));
    if (lane == 0) {
      sh.chunk_a[c] = a.MsL;
      sh.chunk_b[c] = csum;
    }
  }
  if (keep_teacher) {
    const float csum = wave_sum(static_cast<float>(pt));
    if (lane == 0) {
      sh.chunk_c[c] = a.MtL;
      sh.chunk_d[c] = csum;
    }
  }
  a.Ss += ps;
  a.S1 += p1;
  a.S2 += p2;
  a.S3 += p3;
  a.S4 += p4;
  a.St += pt;
  a.T1 += t1;
  a.T2 += t2;
  a.Sm += pm;
  a.Q1 += q1;
  a.Q2 += q2;
}

// The block's maxima, rescaled sums, argmax and range of d.
struct StatsBlock {
  float ms, mt;
  double Ss, S1, S2, S3, S4, St, T1, T2;
  double Sm, Q1, Q2;  // middle-node sums (relative to the row's maxima)
  float lm;           // the middle node
  float tbest;
  int tidx;
  float t_smax;
  float dmin, dmax;
};

// One exchange through LDS: each wave posts its sums (relative to its own
// running maxima), maxima, argmax and range of d (stats_post); after a
// barrier one thread combines the waves in a fixed order (stats_combine).
template <int NT, typename SH>
__device__ void stats_post(Block<NT, SH>& B, StatsAcc& a) {
  double v[11] = {a.Ss, static_cast<double>(a.S1), static_cast<double>(a.S2), static_cast<double>(a.S3),
                  static_cast<double>(a.S4), a.St, static_cast<double>(a.T1), static_cast<double>(a.T2),
                  a.Sm, static_cast<double>(a.Q1), static_cast<double>(a.Q2)};
#pragma unroll
  for (int i = 0; i < 11; ++i) v[i] = wave_sum(v[i]);
  const float wdmin = -wave_max(-a.dmin);
  const float wdmax = wave_max(a.dmax);
  if (B.lane == 0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) B.sh.red_d[B.wave][i] = v[i];
    B.sh.red_d[B.wave][8] = static_cast<double>(a.MsL);
    B.sh.red_d[B.wave][9] = static_cast<double>(a.MtL);
    B.sh.red_f[B.wave][0] = a.Ms;
    B.sh.red_f[B.wave][1] = a.Mt;
    B.sh.red_f[B.wave][2] = wdmin;
    B.sh.red_f[B.wave][3] = wdmax;
    B.sh.red_i[B.wave][0] = a.tidx;
    B.sh.red_d[B.wave][10] = static_cast<double>(a.t_smax);
#pragma unroll
    for (int i = 0; i < 3; ++i) B.sh.red_d[B.wave][11 + i] = v[8 + i];
  }
}

template <int NT, typename SH>
__device__ StatsBlock stats_combine(Block<NT, SH>& B, float lm) {
  constexpr int NW = NT / WAVE;
  StatsBlock O;
  O.ms = -finf();
  O.mt = -finf();
  O.dmin = finf();
  O.dmax = -finf();
  for (int w = 0; w < NW; ++w) {
    O.ms = fmaxf(O.ms, B.sh.red_f[w][0]);
    O.mt = fmaxf(O.mt, B.sh.red_f[w][1]);
    O.dmin = fminf(O.dmin, B.sh.red_f[w][2]);
    O.dmax = fmaxf(O.dmax, B.sh.red_f[w][3]);
  }
  double acc[11] = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
  float tb = -finf();
  int ti = 0x7fffffff;
  float st = -finf();
  // each wave's sums are relative to 2^(its MsL): rescale to the block's
  // msL = ms log2(e) rounded (the MsL of a wave holding the maximum), then
  // remove that rounding (shift_correction)
  const float msL = __fmul_rn(O.ms, LOG2E), mtL = __fmul_rn(O.mt, LOG2E);
  for (int w = 0; w < NW; ++w) {
    const float wMs = B.sh.red_f[w][0], wMt = B.sh.red_f[w][1];
    const float wMsL = static_cast<float>(B.sh.red_d[w][8]), wMtL = static_cast<float>(B.sh.red_d[w][9]);
    const double gs = (wMs == -finf()) ? 0.0 : (wMs == O.ms) ? 1.0 : static_cast<double>(fexp2(__fsub_rn(wMsL, msL)));
    const double gt = (wMt == -finf()) ? 0.0 : (wMt == O.mt) ? 1.0 : static_cast<double>(fexp2(__fsub_rn(wMtL, mtL)));
#pragma unroll
    for (int i = 0; i < 5; ++i) acc[i] += B.sh.red_d[w][i] * gs;
#pragma unroll
    for (int i = 5; i < 8; ++i) acc[i] += B.sh.red_d[w][i] * gt;
    // the middle node's sums are relative to 2^((1 - lm) wMsL + lm wMtL)
    const double gm = (wMs == -finf() || wMt == -finf()) ? 0.0 :
        exp2(static_cast<double>(1.0f - lm) * (static_cast<double>(wMsL) - static_cast<double>(msL)) +
             static_cast<double>(lm) * (static_cast<double>(wMtL) - static_cast<double>(mtL)));
#pragma unroll
    for (int i = 0; i < 3; ++i) acc[8 + i] += B.sh.red_d[w][11 + i] * gm;
    const int wi = B.sh.red_i[w][0];
    if (wMt > tb || (wMt == tb && wi < ti)) { tb = wMt; ti = wi; }
    if (wMs == O.ms) st = fmaxf(st, static_cast<float>(B.sh.red_d[w][10]));
  }
  const double cs = shift_correction(O.ms, msL), ct = shift_correction(O.mt, mtL);
  // The maximum's own term went into the sums as 2^d0 rounded to float (d0 =
  // the rounding of the shift, ~1e-6: a rounding of ~6e-8 next to 1); after
  // the shift correction it is exactly 1.  The log-probability of a dominant
  // entry (near 0 on a peaked row) needs that term exact.
  const double dom_s = 1.0 - static_cast<double>(fexp2(fmaf(O.ms, LOG2E, -msL))) * cs;
  const double dom_t = 1.0 - static_cast<double>(fexp2(fmaf(O.mt, LOG2E, -mtL))) * ct;
  O.Ss = acc[0] * cs + dom_s; O.S1 = acc[1] * cs; O.S2 = acc[2] * cs; O.S3 = acc[3] * cs; O.S4 = acc[4] * cs;
  O.St = acc[5] * ct + dom_t; O.T1 = acc[6] * ct; O.T2 = acc[7] * ct;
  // the middle node's weights carry cs^(1 - lm) ct^lm likewise
  const double cm = exp2(static_cast<double>(1.0f - lm) * log2(cs) + static_cast<double>(lm) * log2(ct));
  O.Sm = acc[8] * cm; O.Q1 = acc[9] * cm; O.Q2 = acc[10] * cm;
  O.lm = lm;
  O.tbest = tb;
  O.tidx = ti;
  O.t_smax = st;
  return O;
}

// Row statistics from the (combined) block statistics.
__device__ inline RowStats row_stats_from(const StatsBlock& O, bool k34) {
  RowStats R;
  R.ms = O.ms;
  R.mt = O.mt;
  R.dmin = O.dmin;
  R.dmax = O.dmax;
  R.tmax = O.tbest;
  R.vstar = O.tidx;
  R.t_smax = O.t_smax;
  R.sum_s = O.Ss;
  R.lse_s = static_cast<double>(R.ms) + log(O.Ss);
  R.lse_t = static_cast<double>(R.mt) + log(O.St);
  const double Ed = O.S1 / O.Ss, E2 = O.S2 / O.Ss, E3 = O.S3 / O.Ss, E4 = O.S4 / O.Ss;
  R.var = fmax(E2 - Ed * Ed, 0.0);
  R.k34 = k34;
  R.k3 = k34 ? E3 - 3.0 * Ed * E2 + 2.0 * Ed * Ed * Ed : 0.0;
  R.k4 = k34 ? (E4 - 4.0 * Ed * E3 + 6.0 * Ed * Ed * E2 - 3.0 * Ed * Ed * Ed * Ed) - 3.0 * R.var * R.var : 0.0;
  R.mean_p = Ed;
  R.mean_pi = O.T1 / O.St;
  R.var_pi = fmax(O.T2 / O.St - R.mean_pi * R.mean_pi, 0.0);
  R.kl1_est = R.mean_pi - (R.lse_t - R.lse_s);
  R.pmax = exp(static_cast<double>(R.ms) - R.lse_s);
  R.c = static_cast<float>(Ed);
  if (!isfinite(R.c)) R.c = 0.0f;
  R.cL = R.c * LOG2E;
  // A at the middle node lm: sum_v p_v e^{lm x_v} = e^{lm (mt - ms - c)}
  // sum_m / sum_s, with sum_m = sum e^{(1 - lm)(s - ms) + lm (t - mt)}; its
  // derivatives are the mean and variance of x under the tilted weights
  {
    const double lm = static_cast<double>(O.lm);
    const double M1 = O.Q1 / O.Sm, M2 = O.Q2 / O.Sm;
    R.lam_mid = O.Sm > 0.0 ? O.lm : 0.0f;
    R.mid_A = lm * (static_cast<double>(R.mt) - static_cast<double>(R.ms) - static_cast<double>(R.c)) +
              log(O.Sm) - log(O.Ss);
    R.mid_A1 = M1 - static_cast<double>(R.c);
    R.mid_A2 = fmax(M2 - M1 * M1, 0.0);
  }
  R.finite = isfinite(R.lse_s) && isfinite(R.lse_t) && isfinite(R.dmin) && isfinite(R.dmax) &&
             isfinite(R.ms) && isfinite(R.mt);
  return R;
}

// keep_chunks: store the proposal chunk masses (of p); keep_teacher: those of pi.
// The statistics are kept in the workgroup's LDS (thread 0 writes them): the
// caller reads its fields there where it needs them rather than holding the
// whole record in registers across the later sweeps.
template <typename T, int NT, bool MID = true, bool K34 = true, typename SH>
__device__ const RowStats& stats_sweep(Block<NT, SH>& B, const T* srow, const T* trow, int V, float lm,
                                       bool keep_chunks, bool keep_teacher = false) {
  constexpr int NW = NT / WAVE;
  StatsAcc a;
  a.init();
  for_chunks<T, NW, false, fill_mode<T, SH>()>(srow, trow, V, B.wave, B.lane,
                    [&](auto tail, const float* s, const float* t, uint32_t vm, int c) {
                      constexpr bool TAIL = decltype(tail)::value;
                      stats_math<TAIL, MID, K34>(s, t, vm, c, B.lane, keep_chunks, keep_teacher, lm, B.sh, a);
                    }, row_cache<T>(B.sh));
  stats_post(B, a);
  __syncthreads();
  if (B.tid == 0) B.sh.rs.r = row_stats_from(stats_combine(B, MID ? lm : 0.0f), K34);
  __syncthreads();
  return B.sh.rs.r;
}

// Thread of a workgroup of NT threads that holds entry v in the chunk sweeps
// (wave c % NW of chunk c = v / CHUNK, lane and slot by elem_offset).
template <int NT>
__device__ __forceinline__ int entry_owner(int v) {
  constexpr int NW = NT / WAVE;
  const int o = v % CHUNK;
  const int lane = (o < 512) ? (o >> 3) : ((o - 512) >> 3);
  return ((v / CHUNK) % NW) * WAVE + lane;
}

// ---------------------------------------------------------------------------
// Lambda sweep: the sums at one node lam over the row.  The weights are
// w_v = p~_v 2^{lam X_v}, p~_v = 2^{a_v}, a_v = (s_v - ms) log2 e, and the
// sums kept are W = sum (w - p~) (so that A = log1p(W / sum p~) keeps its
// relative precision when A is small) and S_k = sum w X^k, k = 1..4, which
// give A(lam) and its first four derivatives, the cumulants of x under q_lam.
//   FAST : w = 2^{a + lam X}.
//   ACC  : w - p~ = p~ expm1(lam x), with expm1 accurate for small arguments
//          (rows whose KL is small).
//   SHIFT: where lam (dmax - c) could overflow float, w' = 2^{a + lam X - sigl}
//          with a shift sigl (log2 units); W = sum w' (plain form), or in the
//          expm1 form sum (w' - p~') with w' - p~' = p~' expm1(lam x) where
//          |lam x| < 1/16 (p~' = 2^{a - sigl}), so the sums keep their
//          relative precision and do not overflow.  Rows need it rarely, so
//          one loop serves both forms.
// ---------------------------------------------------------------------------
enum LamMode { LAM_FAST = 0, LAM_ACC = 1, LAM_SHIFT = 2 };

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

// A(lam) and its derivatives (natural units), and KL = lam A' - A.
struct LamEval {
  double lam, A, A1, A2, A3, A4, KL;
  // a root of the node's Taylor model is accepted only within this relative
  // distance of the node (a node whose A4 is a bound rather than a sum
  // limits it)
  double reach;
};


// a = fma(s, log2 e, -msL) with msL = ms log2 e rounded to float: the rounding
// of the shift, d0 = ms log2 e - msL (exact in double), is one offset for every
// entry of the row, so every weight and every p~ carries the factor 2^d0; the
// row sums are multiplied by 2^-d0 once (shift_correction).
template <int MODE, bool TAIL>
__device__ __forceinline__ void lam_math(const float* s, const float* t, uint32_t vm, float msL,
                                         float cL, float lam, float sigl, bool accf, double (&acc)[5]) {
  float W = 0.f, S1 = 0.f, S2 = 0.f, S3 = 0.f, S4 = 0.f;
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    const float a = fmaf(s[e], LOG2E, -msL);
    float pt = fexp2(a);
    const float X = fmaf(t[e] - s[e], LOG2E, -cL);
    float w, u;
    if (MODE == LAM_FAST) {
      w = fexp2(fmaf(lam, X, a));
      u = w - pt;
    } else if (MODE == LAM_ACC) {
      const float yl = lam * X;
      const float ee = fexp2(yl);
      w = pt * ee;
      u = pt * expm1_sel(yl * LN2, ee);
    } else {  // LAM_SHIFT: exponents shifted by sigl; accf selects the expm1 form
      w = fexp2(fmaf(lam, X, a) - sigl);
      const float y = lam * X * LN2;
      const float ps = fexp2(a - sigl);
      u = !accf ? w : (fabsf(y) < 0.0625f) ? ps * expm1_small(y) : w - ps;
    }
    if (TAIL && !SAKI_VALID(e)) { w = 0.f; u = 0.f; }
    const float wx = w * X;
    const float wx2 = wx * X;
    const float wx3 = wx2 * X;
    W += u;
    S1 += wx;
    S2 += wx2;
    S3 += wx3;
    S4 = fmaf(wx3, X, S4);
  }
  acc[0] += static_cast<double>(W);
  acc[1] += static_cast<double>(S1);
  acc[2] += static_cast<double>(S2);
  acc[3] += static_cast<double>(S3);
  acc[4] += static_cast<double>(S4);
}

// A and its derivatives at lam from the row sums v = {W, S1..S4} (log2
// units) and b0 = sum p~.  acc: W = sum (w - p~), scaled by 2^-sigl when
// sigl != 0; otherwise W = sum w when sigl != 0.
__device__ inline LamEval lam_finish(const double (&v)[5], double b0, float lam, float sigl, bool acc) {
  LamEval E;
  E.lam = lam;
  double S0, r = 1.0;
  if (sigl == 0.f) {
    S0 = b0 + v[0];
    E.A = log1p(v[0] / b0);
  } else if (acc) {
    // the sums carry the factor 2^-sigl: undo it in double
    r = exp2(static_cast<double>(sigl));
    S0 = b0 + v[0] * r;
    E.A = log1p(v[0] * r / b0);
  } else {
    // sigl is in log2 units: the shift in natural units is sigl ln 2
    S0 = v[0];
    E.A = static_cast<double>(sigl) * LN2_D + log(v[0] / b0);
  }
  // raw moments of X under q, then its cumulants; x = X ln 2
  const double m1 = v[1] * r / S0, m2 = v[2] * r / S0, m3 = v[3] * r / S0, m4 = v[4] * r / S0;
  const double c2 = fmax(m2 - m1 * m1, 0.0);
  const double c3 = m3 - 3.0 * m1 * m2 + 2.0 * m1 * m1 * m1;
  const double c4 = m4 - 4.0 * m1 * m3 + 6.0 * m1 * m1 * m2 - 3.0 * m1 * m1 * m1 * m1 - 3.0 * c2 * c2;
  const double l1 = LN2_D, l2 = l1 * l1;
  E.A1 = m1 * l1;
  E.A2 = c2 * l2;
  E.A3 = c3 * l2 * l1;
  E.A4 = c4 * l2 * l2;
  E.KL = fmax(E.lam * E.A1 - E.A, 0.0);  // non-negative; rounding can give -1e-16 when p ~ pi
  E.reach = __builtin_huge_val();
  return E;
}

// The dominant entry of p (an entry holding max s) carries the largest
// rounding of the plain w - p~ (~6e-8 of its p~, a p~ near 1 on a peaked row).
// Every thread computes that entry's plain term exactly as the sweep did (the
// same float operations) and its exact value, p~ expm1(lam x) in double; the
// difference replaces it in the row sum.  Its own a is the shift's rounding
// (|a| ~ 1e-6), so 2^a is the quadratic below to rounding; only where
// |lam x| < 1/16 is the plain term's rounding large next to the term itself
// (expm1 by its series there).
__device__ __forceinline__ double dominant_fix(float s, float t, float msL, float cL, float lam) {
  const float a = fmaf(s, LOG2E, -msL);
  const float X = fmaf(t - s, LOG2E, -cL);
  const double y = static_cast<double>(lam) * static_cast<double>(X) * LN2_D;
  if (!(fabs(y) < 0.0625)) return 0.0;
  const float uf = fexp2(fmaf(lam, X, a)) - fexp2(a);
  const double al = static_cast<double>(a) * LN2_D;
  const double pt = 1.0 + al * (1.0 + 0.5 * al);
  const double em = y * (1.0 + y * (0.5 + y * (1.0 / 6 + y * (1.0 / 24 + y * (1.0 / 120 + y * (1.0 / 720 +
                    y * (1.0 / 5040)))))));
  return pt * em - static_cast<double>(uf);
}

template <typename T, int NT, int MODE, typename SH>
__device__ LamEval lam_sweep_mode(Block<NT, SH>& B, const T* srow, const T* trow, int V, const RowStats& R,
                                  float lam, float sigl, bool accf) {
  constexpr int NW = NT / WAVE;
  double v[5] = {0, 0, 0, 0, 0};
  const float msL = R.ms * LOG2E;
  for_chunks<T, NW, false, use_mode<T, SH>()>(srow, trow, V, B.wave, B.lane,
                    [&](auto tail, const float* s, const float* t, uint32_t vm, int c) {
                      constexpr bool TAIL = decltype(tail)::value;
                      lam_math<MODE, TAIL>(s, t, vm, msL, R.cL, lam, sigl, accf, v);
                    }, row_cache<T>(B.sh));
  B.sum(v);
  if constexpr (MODE == LAM_FAST) v[0] += dominant_fix(R.ms, R.t_smax, msL, R.cL, lam);
  const double corr = shift_correction(R.ms, msL);
#pragma unroll
  for (int j = 0; j < 5; ++j) v[j] *= corr;
  return lam_finish(v, R.sum_s, lam, sigl, accf);
}

// Evaluates A and its derivatives at lam over the whole row; acc selects the
// expm1 form.  Where lam x can exceed 60 (natural units) for some entry, the
// exponents are shifted by sigl so that lam x - sig <= 60 for every entry.
// Every thread gets the same result.
template <typename T, int NT, typename SH>
__device__ LamEval lam_sweep(Block<NT, SH>& B, const T* srow, const T* trow, int V, const RowStats& R,
                             float lam, bool acc) {
  const double top = static_cast<double>(lam) * (static_cast<double>(R.dmax) - R.c);  // largest lam x
  const float sigl = top <= 60.0 ? 0.0f : static_cast<float>((top - 60.0) * static_cast<double>(LOG2E));
  if (sigl != 0.0f) return lam_sweep_mode<T, NT, LAM_SHIFT>(B, srow, trow, V, R, lam, sigl, acc);
  if (acc) return lam_sweep_mode<T, NT, LAM_ACC>(B, srow, trow, V, R, lam, 0.0f, true);
  return lam_sweep_mode<T, NT, LAM_FAST>(B, srow, trow, V, R, lam, 0.0f, false);
}

// Rows whose KL (the radius, or KL(pi||p) at the teacher endpoint) is below
// this use the expm1 forms of the lambda sweeps.
constexpr double KL_ACCURATE = 0.01;
// ... and below this, the expm1 form of the final sweep: there 2^y - 1 carries
// ~6e-8 absolute error per entry, which summed over the positive residual is
// ~1e-5 of a TV near 0.01 (TV <= sqrt(KL / 2)).
constexpr double TV_ACCURATE = 0.1;
// In the plain forms each w - p~ (and q/p - 1) carries ~4e-8 of its p as
// rounding, so A carries ~4e-8 |p'|_2 (random over the entries) and TV as
// much.  The lambda sweep takes the dominant entry's term exactly, so p' is p
// without it (|p'|_2 <= sqrt(min(max p, 1 - max p) (1 - max p))); peaked rows
// (max p above P_PEAKED) take the final sweep in the expm1 form, where the
// dominant entry's q/p - 1 is exact to rounding.
constexpr double P_PEAKED = 0.25;
// A row resolved in a plain form whose TV is below TV_PLAIN_MIN times that
// bound of |p'|_2 (A's error then above ~2e-6 of TV) is resolved again in the
// expm1 forms.
constexpr double TV_PLAIN_MIN = 0.02;

// Result of the lambda search.
struct LamResult {
  float lam;   // lambda*
  double A;    // A(lambda*) = log sum_v p_v exp(lambda* x_v), x = d - c
  double KL;   // KL(q_lambda* || p)
  float c;     // centring constant used by A (may differ from RowStats::c)
  float cL;    // c log2(e) as used in X = fma(d, log2 e, -cL)
  bool qp;     // q = p exactly (eps = 0, or t - s constant): the sweeps use lambda 0
  bool acc;    // A and KL come from a sweep in the expm1 form
  int sweeps;  // lambda sweeps the search ran
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

// Quartic Taylor model of A around a node: A(l) ~ sum_k A_k (l - lam)^k / k!,
// and KL(l) = l A'(l) - A(l) on it.
struct TaylorA {
  LamEval n;
  __device__ void eval(double l, double& A, double& Ap) const {
    const double d = l - n.lam;
    A = n.A + d * (n.A1 + d * (0.5 * n.A2 + d * (n.A3 / 6.0 + d * (n.A4 / 24.0))));
    Ap = n.A1 + d * (n.A2 + d * (0.5 * n.A3 + d * (n.A4 / 6.0)));
  }
  __device__ double kl(double l) const {
    double A, Ap;
    eval(l, A, Ap);
    return l * Ap - A;
  }
  __device__ bool usable() const {
    return isfinite(n.A) && isfinite(n.A1) && isfinite(n.A2) && isfinite(n.A3) && isfinite(n.A4);
  }
};

// Starting points of the search.  Cumulant start: KL(lam) = sum_n (n - 1)
// kappa_n lam^n / n! ~ k2 lam^2/2 + k3 lam^3/3 + k4 lam^4/8 with the
// cumulants of d under p.  Two-ended start: the degree-7 polynomial A(lam)
// with A(0) = 0, A^(k)(0) = kappa_k (k = 1..4, of x = d - c under p) and
// A(1) = lse_t - lse_s - c, A'(1) = E_pi[x], A''(1) = Var_pi(x) at the teacher
// end; KL = eps is solved on it by bisection.
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
    const bool done = fabs(nl - l) <= 1e-10 * l;
    l = nl;
    if (done) break;
  }
  return l;
}

__device__ inline double two_ended_start(const RowStats& R, double eps) {
  double c[8];
  c[0] = 0.0;
  c[1] = R.mean_p - R.c;
  c[2] = R.var / 2.0;
  c[3] = R.k3 / 6.0;
  c[4] = R.k4 / 24.0;
  const double a1 = R.lse_t - R.lse_s - R.c, d1 = R.mean_pi - R.c, dd1 = R.var_pi;
  const double r0 = a1 - (c[1] + c[2] + c[3] + c[4]);
  const double r1 = d1 - (c[1] + 2.0 * c[2] + 3.0 * c[3] + 4.0 * c[4]);
  const double r2 = dd1 - (2.0 * c[2] + 6.0 * c[3] + 12.0 * c[4]);
  c[5] = 0.5 * (42.0 * r0 - 12.0 * r1 + r2);
  c[6] = 0.5 * (-70.0 * r0 + 22.0 * r1 - 2.0 * r2);
  c[7] = 0.5 * (30.0 * r0 - 10.0 * r1 + r2);
  auto kl = [&](double l) {
    double v = 0.0;
#pragma unroll
    for (int j = 7; j >= 2; --j) v = (v + (j - 1) * c[j]) * l;
    return v * l;
  };
  if (!(kl(1.0) > eps)) return -1.0;
  // 2^-14 resolution: below the error of the model itself (~1e-3)
  double lo = 0.0, hi = 1.0;
  for (int it = 0; it < 14; ++it) {
    const double m = 0.5 * (lo + hi);
    if (kl(m) <= eps) lo = m; else hi = m;
  }
  return lo;
}

// Interpolating start: the polynomial of degree N0 + 5 that matches A and its
// first N0 - 1 derivatives at lambda = 0 (the cumulants of x under p: four
// with k3, k4, else two), A, A', A'' at the middle node, and A, A', A'' at
// lambda = 1 (the teacher end), in Newton form over the confluent nodes.  On rows whose A is smooth on [0, 1] it places
// lambda* to ~1e-6 or better, where the ends alone (two_ended_start) leave
// ~1e-3; on spiky rows it can be far off, which the caller detects.
template <int N0>  // conditions at lambda = 0: 5 with k3, k4, else 3
struct HermiteA {
  static constexpr int N = N0 + 6;
  double z[N], c[N];
  __device__ explicit HermiteA(const RowStats& R) {
    const double lm = static_cast<double>(R.lam_mid);
    const double f0[5] = {0.0, R.mean_p - R.c, R.var, R.k3, R.k4};
    const double fm[3] = {R.mid_A, R.mid_A1, R.mid_A2};
    const double f1[3] = {R.lse_t - R.lse_s - R.c, R.mean_pi - R.c, R.var_pi};
    const double inv_fact[5] = {1.0, 1.0, 0.5, 1.0 / 6.0, 1.0 / 24.0};
    auto deriv = [&](int i, int j) { return i < N0 ? f0[j] : i < N0 + 3 ? fm[j - 0] : f1[j]; };
#pragma unroll
    for (int i = 0; i < N; ++i) {
      z[i] = i < N0 ? 0.0 : i < N0 + 3 ? lm : 1.0;
      c[i] = deriv(i, 0);
    }
    // divided differences in place: after step j, c[i] = f[z_{i-j} .. z_i]
    // (a repeated node takes the derivative / j! there); the spans z_i - z_{i-j}
    // are lm, 1 - lm or 1, so three reciprocals serve every step
    const double r_lm = 1.0 / lm, r_rest = 1.0 / (1.0 - lm);
    // fully unrolled: constant indices keep the tables in registers
#pragma unroll
    for (int j = 1; j < N; ++j)
#pragma unroll
      for (int i = N - 1; i >= j; --i) {
        const double span = z[i] - z[i - j];
        const double rs = span == 1.0 ? 1.0 : span == lm ? r_lm : r_rest;
        c[i] = (span == 0.0) ? deriv(i, j) * inv_fact[j] : (c[i] - c[i - 1]) * rs;
      }
  }
  // the polynomial and its first two derivatives at l
  __device__ void eval(double l, double& p, double& p1, double& p2) const {
    p = c[N - 1];
    p1 = 0.0;
    p2 = 0.0;
#pragma unroll
    for (int k = N - 2; k >= 0; --k) {
      const double dz = l - z[k];
      p2 = p2 * dz + 2.0 * p1;
      p1 = p1 * dz + p;
      p = p * dz + c[k];
    }
  }

};

// Where lambda* starts, and A there.
struct StartPoint {
  double lam;  // the first node
  double A;    // A(lam) predicted by the interpolant (herm only)
  bool herm;   // lam solves KL = eps on the interpolant, on the middle node's side
};

constexpr double LAM_MAX = 1.0 - 1e-6;

// The interpolant's root of KL = eps from l0 (S unchanged when it is not
// found, lies on the wrong side of the middle node, or the interpolant is not
// convex there).
template <int N0>
__device__ inline void hermite_refine(const RowStats& R, double eps, double l0, StartPoint& S) {
  const HermiteA<N0> H(R);
  double p, p1, p2;
  H.eval(1.0, p, p1, p2);
  if (!(p1 - p > eps)) return;  // the interpolant puts lambda* at 1
  // KL increases with lambda, so KL at the middle node (known from the stats
  // sweep, which the interpolant matches there) tells on which side of it
  // lambda* lies: the search keeps to that side.  The ends' starts can be far
  // off on rows whose largest d dominate q_lambda, where the interpolant is
  // still close, so l0 only seeds the search.
  const double lm = static_cast<double>(R.lam_mid);
  const bool above = lm * R.mid_A1 - R.mid_A <= eps;
  const double blo = above ? lm : 0.0, bhi = above ? 1.0 : lm;
  // safeguarded Newton on KL(l) = l A'(l) - A(l) = eps (KL' = l A''),
  // keeping the bracket KL(lo) <= eps < KL(hi)
  // (converged once the step is below 1e-10 of lambda: the interpolant's own
  // rounding, ~1e-12 of lambda near the root, would otherwise send a
  // tighter test into the bisection branch)
  double lo = blo, hi = bhi;
  // the search starts from l0, moved inside the bracket when outside it (to
  // its nearer end, so that Newton does not start among the interpolant's
  // other roots far from both)
  double l = fmin(fmax(l0, blo + 1e-6 * (bhi - blo)), bhi - 1e-6 * (bhi - blo));
  bool conv = false;
  for (int it = 0; it < 14; ++it) {
    H.eval(l, p, p1, p2);
    const double f = l * p1 - p - eps;
    if (f <= 0.0) lo = l; else hi = l;
    const double fp = l * p2;
    const double step = (fp > 0.0) ? -f / fp : __builtin_huge_val();
    if (fabs(step) <= 1e-10 * l || hi - lo <= 1e-8 * l) {
      conv = true;
      break;
    }
    double nl = l + step;
    if (!(nl > lo && nl < hi)) nl = 0.5 * (lo + hi);
    l = nl;
  }
  if (!conv || !(l > blo && l < bhi) || !(l < LAM_MAX)) return;
  H.eval(l, p, p1, p2);
  if (!(p2 > 0.0) || !isfinite(p)) return;
  S.lam = l;
  S.A = p;
  S.herm = true;
}

__device__ inline StartPoint start_point(const RowStats& R, double eps) {
  const double l_cum = cumulant_start(R, eps);
  const double l_two = two_ended_start(R, eps);
  double l0 = (l_two > 0.0 && fabs(l_two - l_cum) <= 0.3 * l_cum) ? l_two : l_cum;
  l0 = fmin(fmax(l0, 1e-7), LAM_MAX);
  StartPoint S;
  S.lam = l0;
  S.A = 0.0;
  S.herm = false;
  if (!(R.lam_mid > 0.0f)) return S;
  if (R.k34)
    hermite_refine<5>(R, eps, l0, S);
  else
    hermite_refine<3>(R, eps, l0, S);
  return S;
}

// Largest lambda in [0, 1] with KL(q_lambda || p) <= eps (Eq. trust_region).
// Each sweep evaluates A and its first four derivatives at one node; KL = eps
// is then solved on the quartic Taylor model around the node, inside the
// bracket [lo, hi] of evaluated nodes and within 30% of the node.  The root
// is accepted when five times the model's last term is below TAYLOR_TOL eps
// (the next term is smaller by about |l - node| times the cumulant growth);
// otherwise the next node is that root (or the edge of the trust interval).
// sweep1(lam, acc) evaluates one node over the whole row.
// force_acc: every sweep in the expm1 form; lam_hint > 0: the first node (a
// lambda* found before, resolved again in the accurate form); first: the
// first node already evaluated (by the fused sweep, at first->lam; in the
// expm1 form if first_acc), used in place of the first sweep.  out.sweeps
// counts the sweeps run here.
// no_sweep: stop where a sweep would be needed (out.sweeps = -1), so that one
// wave can settle the common case of an accepted first node alone.
template <typename Sweep1>
__device__ LamResult lambda_search_with(const RowStats& R, double eps, Sweep1&& sweep1, bool force_acc = false,
                                        float lam_hint = 0.0f, const LamEval* first = nullptr,
                                        bool first_acc = false, bool no_sweep = false) {
  LamResult out;
  out.acc = true;
  out.sweeps = 0;
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
  // KL of that size.
  bool acc = force_acc || eps < KL_ACCURATE || (first != nullptr && first_acc);
  out.acc = acc;
  constexpr double TAYLOR_TOL = 1e-7;
  constexpr double TRUST = 0.3;
  constexpr double LMAX = LAM_MAX;
  double lo = 0.0, hi = 1.0;  // KL(lo) <= eps < KL(hi) (hi = 1 until a node above is seen)
  LamEval feas;               // the largest evaluated lambda that is feasible (lambda = 0 is)
  feas.lam = 0.0; feas.A = 0.0; feas.KL = 0.0;
  double lg = (first == nullptr && !(lam_hint > 0.0f)) ? start_point(R, eps).lam : 0.0;
  bool try_one = R.kl1_est <= 1.05 * eps + 1e-5;
  if (lam_hint > 0.0f) {
    lg = lam_hint;
    try_one = lam_hint == 1.0f;
  }
  if (first != nullptr) {
    lg = first->lam;
    try_one = false;
  }
  // The first TRUST_SWEEPS sweeps step within TRUST of the node.  A row still
  // unresolved after them (a KL that rises steeply, e.g. a few entries with
  // tiny p and a large d) continues with safeguarded steps: the model's root
  // inside the bracket when it at least halves the step of two sweeps
  // before, the bracket's midpoint otherwise.
  constexpr int TRUST_SWEEPS = 4;
  constexpr int MAX_SWEEPS = 64;
  double step1 = 2.0, step2 = 2.0;  // the last two node steps (safeguard)
  for (int sweep = 0; sweep < MAX_SWEEPS; ++sweep) {
    const float lf = try_one ? 1.0f : static_cast<float>(lg);
    const bool given = sweep == 0 && first != nullptr;
    if (!given && no_sweep) {
      out.sweeps = -1;
      return out;
    }
    const LamEval E = given ? *first : sweep1(lf, acc);
    if (!given) ++out.sweeps;
    if (lf == 1.0f && E.KL <= eps) {
      if (!acc && E.KL < KL_ACCURATE) {
        acc = true;  // resolve a small endpoint KL with the accurate form
        out.acc = true;
        continue;
      }
      out.lam = 1.0f; out.A = E.A; out.KL = E.KL;
      return out;
    }
    try_one = false;
    if (E.KL <= eps) {
      if (E.lam >= lo) { lo = E.lam; feas = E; }
    } else {
      hi = fmin(hi, E.lam);
    }
    const bool trust = sweep < TRUST_SWEEPS;
    if (!trust) {
      // a feasible node at the radius, or a bracket at float resolution
      if (E.KL <= eps && eps - E.KL <= TAYLOR_TOL * eps) break;
      if (hi - lo <= 1e-7 * hi) break;
    }
    TaylorA M;
    M.n = E;
    if (!M.usable()) {
      lg = 0.5 * (lo + hi);
      continue;
    }
    // a node whose A'''' is a bound (reach-limited) takes a trust interval of
    // twice its reach: far from the node that term would bend the model's KL
    const double tr = fmin(TRUST, 2.0 * E.reach);
    const double a = trust ? fmax(lo, E.lam * (1.0 - tr)) : lo;
    const double b = trust ? fmin(hi, E.lam * (1.0 + tr)) : hi;
    const double fa = M.kl(a) - eps, fb = M.kl(b) - eps;
    if (fa <= 0.0 && fb > 0.0) {
      // safeguarded Newton on the model inside [a, b]
      double l = fmin(fmax(E.lam, a), b), xa = a, xb = b;
      for (int it = 0; it < 60; ++it) {
        double A, Ap;
        M.eval(l, A, Ap);
        const double f = l * Ap - A - eps;
        if (f == 0.0) break;
        if (f < 0.0) xa = l; else xb = l;
        const double dd = l - E.lam;
        const double fp = l * (E.A2 + dd * (E.A3 + dd * (0.5 * E.A4)));  // l A''
        double nl = (fp > 0.0) ? l - f / fp : 0.5 * (xa + xb);
        if (!(nl > xa && nl < xb)) nl = 0.5 * (xa + xb);
        const bool done = fabs(nl - l) <= 1e-14 * l || (xb - xa) <= 1e-14 * l;
        l = nl;
        if (done) break;
      }
      const double d = l - E.lam;
      const double err = 5.0 * fabs(E.A4) * d * d * d * d / 24.0;
      if (err <= TAYLOR_TOL * eps && fabs(d) <= E.reach * E.lam) {
        const float lr = static_cast<float>(l);
        double A, Ap;
        M.eval(static_cast<double>(lr), A, Ap);
        out.lam = lr;
        out.A = A;
        out.KL = fmax(static_cast<double>(lr) * Ap - A, 0.0);
        return out;
      }
      lg = l;
    } else if (trust) {
      // the model's root is outside the trust interval: go to its edge
      if (fb <= 0.0) {
        if (b >= 1.0 || E.lam * (1.0 + TRUST) >= 1.0) {
          try_one = hi >= 1.0;  // the teacher endpoint may be feasible
          lg = fmin(0.5 * (E.lam + hi), LMAX);
        } else {
          lg = b;
        }
      } else {
        lg = a;
      }
    } else {
      lg = 0.5 * (lo + hi);
    }
    if (!trust) {
      const double st = fabs(lg - E.lam);
      if (!(lg > lo && lg < hi) || st > 0.5 * step2) lg = 0.5 * (lo + hi);
      step2 = step1;
      step1 = fabs(lg - E.lam);
    }
    lg = fmin(fmax(lg, 1e-7), LMAX);
  }
  // the bracket has closed on the root (or the sweeps ran out): keep the
  // largest feasible evaluated lambda
  out.lam = static_cast<float>(feas.lam); out.A = feas.A; out.KL = feas.KL;
  return out;
}

template <typename T, int NT, typename SH>
__device__ LamResult lambda_search(Block<NT, SH>& B, const T* srow, const T* trow, int V,
                                   const RowStats& R, double eps, bool force_acc = false, float lam_hint = 0.0f) {
  return lambda_search_with(R, eps, [&](float lam, bool acc) {
    return lam_sweep<T, NT>(B, srow, trow, V, R, lam, acc);
  }, force_acc, lam_hint);
}

// A row resolved in a plain form whose TV is too small for that form's
// rounding (TV_PLAIN_MIN) is resolved again in the expm1 forms.
__device__ inline bool redo_accurate(const RowStats& R, const LamResult& L, bool final_acc, double TV) {
  if (L.qp || (L.acc && final_acc)) return false;
  const double rest = 1.0 - R.pmax;
  const double lam_err = L.acc ? 0.0 : sqrt(fmax(fmin(R.pmax, rest) * rest, 0.0));
  const double fin_err = final_acc ? 0.0 : sqrt(R.pmax);
  return TV < TV_PLAIN_MIN * fmax(lam_err, fin_err);
}

// ---------------------------------------------------------------------------
// Final sweep at lambda*: TV, residual chunk masses, gradient row.
//   p_v = p~_v / sum_s,  q_v / p_v = 2^{lam* X_v - A* log2 e},
//   w_v = p_v [q_v/p_v - 1]_+ ;  grad_v = coef * (p_v - 1[v = hot]).
// ---------------------------------------------------------------------------
struct FinalConst {
  float msL, invS, cL, lam, AL;  // msL = ms log2(e); AL = A* log2(e)
  bool acc;                      // expm1 form (rows whose KL is small)
  bool wide;                     // q/p can exceed 2^60 for some entry
};

// Forms of the final sweep's weights: FIN_FAST 2^y - 1, FIN_ACC its expm1
// form; FIN_WIDE (rows where q/p can overflow float) takes [q - p]_+ with
// q = 2^(a + y) / sum p~ for the entries with q/p > 2^64 (q <= 1 there while
// q/p would overflow), the FIN_FAST / FIN_ACC form (by F.acc) elsewhere.
enum FinMode { FIN_FAST = 0, FIN_ACC = 1, FIN_WIDE = 2 };

__device__ inline FinalConst final_const(const RowStats& R, const LamResult& L, bool force_acc = false) {
  FinalConst F;
  F.msL = R.ms * LOG2E;
  // p = 2^{fma(s, log2 e, -msL)} * invS: the shift's rounding is folded into invS
  F.invS = static_cast<float>(shift_correction(R.ms, F.msL) / R.sum_s);
  F.cL = L.cL;
  F.lam = L.qp ? 0.0f : L.lam;
  F.AL = L.qp ? 0.0f : static_cast<float>(L.A * static_cast<double>(LOG2E));
  F.acc = force_acc || L.KL < TV_ACCURATE || R.pmax > P_PEAKED;
  // largest log q/p over the row: lam* (dmax - c) - A*
  const double top = static_cast<double>(F.lam) * (static_cast<double>(R.dmax) - L.c) - (L.qp ? 0.0 : L.A);
  F.wide = top * static_cast<double>(LOG2E) > 60.0;
  return F;
}

// Residual weight [q_v - p_v]_+ and p_v of one entry; the residual race uses
// the same function, so its weights are bit-identical to the chunk masses'.
template <int MODE>
__device__ __forceinline__ float res_weight(float s, float t, const FinalConst& F, float* p_out) {
  const float a = fmaf(s, LOG2E, -F.msL);
  const float p = fexp2(a) * F.invS;
  const float X = fmaf(t - s, LOG2E, -F.cL);
  const float y2 = fmaf(F.lam, X, -F.AL);  // log2 of q/p
  *p_out = p;
  if constexpr (MODE == FIN_WIDE) {
    const float ee = fexp2(fminf(y2, 64.0f));
    const float em1 = F.acc ? expm1_sel(y2 * LN2, ee) : (ee - 1.0f);
    const float q = fexp2(a + y2) * F.invS;
    const float w = (y2 > 64.0f) ? q - p : p * em1;
    return fmaxf(w, 0.0f);
  } else {
    const float ee = fexp2(y2);
    const float em1 = (MODE == FIN_ACC) ? expm1_sel(y2 * LN2, ee) : (ee - 1.0f);
    return p * fmaxf(em1, 0.0f);
  }
}

// res_weight in the form F selects.
__device__ __forceinline__ float res_weight_any(float s, float t, const FinalConst& F, float* p_out) {
  if (F.wide) return res_weight<FIN_WIDE>(s, t, F, p_out);
  return F.acc ? res_weight<FIN_ACC>(s, t, F, p_out) : res_weight<FIN_FAST>(s, t, F, p_out);
}


// F is taken by value: the loop then holds its fields in registers, with no
// reloads through a pointer that the gradient stores might alias.  The
// gradient's indicator entry (hot, whose logit s_hot the caller already holds)
// is not special-cased inside the loop: after the sweep the thread that
// stored coef * p_hot overwrites it with coef * (p_hot - 1), p_hot computed by
// the same expression (same thread, same address, so the later store is the
// one that stays).
template <typename T, typename G, int NT, bool GRAD, int MODE, typename SH>
__device__ __forceinline__ double final_sweep(Block<NT, SH>& B, const T* srow, const T* trow, G* grow, int V,
                              const FinalConst F, bool keep_res, float coef, int hot, float s_hot) {
  constexpr int NW = NT / WAVE;
  double TV = 0;
  for_chunks<T, NW, true, use_mode<T, SH>()>(srow, trow, V, B.wave, B.lane,
                    [&](auto tail, const float* s, const float* t, uint32_t vm, int c) {
                      constexpr bool TAIL = decltype(tail)::value;
                      float tv = 0.f, g[EPL];
#pragma unroll
                      for (int e = 0; e < EPL; ++e) {
                        float p;
                        const float w = res_weight<MODE>(s[e], t[e], F, &p);
                        if (SAKI_VALID(e)) tv += w;
                        if (GRAD) g[e] = coef * p;
                      }
                      if (keep_res) {
                        const float m = wave_sum(tv);
                        if (B.lane == 0) B.sh.chunk_a[c] = m;
                      }
                      TV += static_cast<double>(tv);
                      if (GRAD) store_lane<G, TAIL>(grow, c, B.lane, V, g);
                    }, row_cache<T>(B.sh));
  if (GRAD && hot >= 0 && hot < V && B.tid == entry_owner<NT>(hot)) {
    const float p = fexp2(fmaf(s_hot, LOG2E, -F.msL)) * F.invS;
    Storer<G>::store1(grow + hot, coef * (p - 1.0f));
  }
  double v[1] = {TV};
  B.sum(v);
  return v[0];
}

// A gradient row of one value (rows without a usable coupling: NaN at a valid
// row with non-finite logits, exact zeros at a masked row whatever its
// logits); the logits are not read.
template <typename G, int NT>
__device__ void fill_row(int wave, int lane, G* grow, int V, float value) {
  constexpr int NW = NT / WAVE;
  const int nchunks = (V + CHUNK - 1) / CHUNK;
  const bool ragged = (V % CHUNK) != 0;
  float g[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) g[e] = value;
  for (int c = wave; c < nchunks; c += NW) {
    if (ragged && c == nchunks - 1)
      store_lane<G, true>(grow, c, lane, V, g);
    else
      store_lane<G, false>(grow, c, lane, V, g);
  }
}

// The final sweep in the form F selects.
template <typename T, typename G, int NT, bool GRAD, typename SH>
__device__ double final_sweep_any(Block<NT, SH>& B, const T* srow, const T* trow, G* grow, int V,
                                  const FinalConst& F, bool keep_res, float coef, int hot, float s_hot) {
  if (F.wide) return final_sweep<T, G, NT, GRAD, FIN_WIDE>(B, srow, trow, grow, V, F, keep_res, coef, hot, s_hot);
  if (F.acc) return final_sweep<T, G, NT, GRAD, FIN_ACC>(B, srow, trow, grow, V, F, keep_res, coef, hot, s_hot);
  return final_sweep<T, G, NT, GRAD, FIN_FAST>(B, srow, trow, grow, V, F, keep_res, coef, hot, s_hot);
}

// ---------------------------------------------------------------------------
// Fused sweep: one pass that evaluates the lambda node and, speculatively,
// what the final sweep needs.  Where the interpolating start places lambda*
// close to its node lam_g, with A(lam_g) predicted as AL (log2 units), each
// entry takes y = lam_g X - AL, e = 2^y (q/p at the node, up to the small
// error of AL) and r = p~ (e - 1):
//   node  : W = sum r, S_k = sum p~ e y^k (k = 1..3): A(lam_g) = AL ln 2 +
//           log1p(W / sum p~), and from the moments of y = lam_g X - AL
//           those of X, i.e. A', A'' and A''' (the model's step is accepted
//           only within FUSED_REACH lam_g of the node, against a bound on
//           A'''');
//   final : over P = {y > 0}: T0 = sum r, U0 = sum p~ e, U1 = sum p~ e y, and
//           the mass Bd = sum p~ e over the band |y| < FUSED_BAND; per chunk
//           (keep_res) the masses sum_P r and sum_P p~ e;
//   grad  : coef p_v under the accept decision taken at the start point.
// At lambda* (node and model) each exponent moves by h = dl X - dA = rho y +
// H0 (dl, dA the changes of lambda and of A log2 e; rho = dl / lam_g,
// H0 = rho AL - dA), so
//   sum [q - p]_+ (unnormalised) = T0 + ln 2 (rho U1 + H0 U0) + O(h^2 U0)
// plus the entries whose sign of y changes, all inside the band when the
// threshold moves less than FUSED_BAND (fused_tv bounds both).  A row whose
// lambda*, accept decision or bounds do not hold takes the final sweep after
// all (its gradient is then rewritten).
// ---------------------------------------------------------------------------
constexpr float FUSED_BAND = 1.0f / 1024.0f;
constexpr double FUSED_REACH = 0.02;
// largest bound on TV's error accepted from the fused sums (relative; the
// bound is a worst case, the error itself is far below it)
constexpr double FUSED_TV_TOL = 3e-6;

struct FusedConst {
  float msL, cL;  // as in the final sweep
  float lam;      // the node lam_g
  float AL;       // predicted A(lam_g) log2 e: the exponents are y = lam X - AL
  float gsc;      // coef / sum p~ (with the shift's rounding): grad_v = gsc p~_v
  float kL, K;    // y = fma(t - s, kL, -K): kL = lam log2 e, K = lam cL + AL
  // the node and centring these float constants give exactly: with
  // X = (t - s) log2 e - cL, y = lam_e X - AL_e (the roundings of kL and K
  // are shared by every entry, so they are taken out here, not bounded)
  double lam_e, AL_e;
  __device__ void set_y() {
    kL = lam * LOG2E;
    K = fmaf(lam, cL, AL);
    lam_e = static_cast<double>(kL) / static_cast<double>(LOG2E);
    AL_e = static_cast<double>(K) - lam_e * static_cast<double>(cL);
  }
};

struct FusedSums {
  double v[4];   // W, S1, S2, S3 (moments of y, relative to 2^AL)
  double T0, U0, U1, Bd;
};

template <typename T, typename G, int NT, bool GRAD, int MODE, typename SH>
__device__ __forceinline__ FusedSums fused_sweep(Block<NT, SH>& B, const T* srow, const T* trow, G* grow, int V,
                                                 const FusedConst C, bool keep_res, float coef, float invS,
                                                 int hot, float s_hot) {
  constexpr int NW = NT / WAVE;
  double acc[5] = {0, 0, 0, 0, 0};  // W, S1, S2, S3, T0
  float U0 = 0.f, U1 = 0.f, Bd = 0.f;
  for_chunks<T, NW, true, use_mode<T, SH>()>(srow, trow, V, B.wave, B.lane,
                    [&](auto tail, const float* s, const float* t, uint32_t vm, int c) {
                      constexpr bool TAIL = decltype(tail)::value;
                      float w = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f, t0 = 0.f, u0 = 0.f, u1 = 0.f, bd = 0.f;
                      float g[EPL];
#pragma unroll
                      for (int e = 0; e < EPL; ++e) {
                        const float a = fmaf(s[e], LOG2E, -C.msL);
                        const float pt = fexp2(a);
                        const float y = fmaf(t[e] - s[e], C.kL, -C.K);
                        const float ee = fexp2(y);
                        // r = p~ (e - 1), rounded once in either form
                        float r = (MODE == FIN_ACC) ? pt * expm1_sel(y * LN2, ee) : fmaf(pt, ee, -pt);
                        float pe = pt + r;
                        if (TAIL && !SAKI_VALID(e)) { r = 0.f; pe = 0.f; }
                        w += r;
                        const float y2 = y * y;
                        s1 = fmaf(pe, y, s1);
                        s2 = fmaf(pe, y2, s2);
                        s3 = fmaf(pe * y2, y, s3);
                        const bool pos = r > 0.0f;
                        t0 += pos ? r : 0.0f;
                        const float pp = pos ? pe : 0.0f;
                        u0 += pp;
                        u1 = fmaf(pp, y, u1);
                        bd += (fabsf(y) < FUSED_BAND) ? pe : 0.0f;
                        if (GRAD) g[e] = C.gsc * pt;
                      }
                      if (keep_res) {
                        const float m = wave_sum(t0);
                        const float q = wave_sum(u0);
                        if (B.lane == 0) {
                          B.sh.chunk_a[c] = m;
                          B.sh.chunk_b[c] = q;
                        }
                      }
                      acc[0] += static_cast<double>(w);
                      acc[1] += static_cast<double>(s1);
                      acc[2] += static_cast<double>(s2);
                      acc[3] += static_cast<double>(s3);
                      acc[4] += static_cast<double>(t0);
                      U0 += u0;
                      U1 += u1;
                      Bd += bd;
                      if (GRAD) store_lane<G, TAIL>(grow, c, B.lane, V, g);
                    }, row_cache<T>(B.sh));
  if (GRAD && hot >= 0 && hot < V && B.tid == entry_owner<NT>(hot)) {
    const float p = fexp2(fmaf(s_hot, LOG2E, -C.msL)) * invS;
    Storer<G>::store1(grow + hot, coef * (p - 1.0f));
  }
  double v[8] = {acc[0], acc[1], acc[2], acc[3], acc[4], static_cast<double>(U0), static_cast<double>(U1),
                 static_cast<double>(Bd)};
  B.sum(v);
  FusedSums S;
#pragma unroll
  for (int i = 0; i < 4; ++i) S.v[i] = v[i];
  S.T0 = v[4];
  S.U0 = v[5];
  S.U1 = v[6];
  S.Bd = v[7];
  return S;
}

template <typename T, typename G, int NT, bool GRAD, typename SH>
__device__ FusedSums fused_sweep_any(Block<NT, SH>& B, const T* srow, const T* trow, G* grow, int V,
                                     const FusedConst& C, bool acc, bool keep_res, float coef, float invS, int hot,
                                     float s_hot) {
  if (acc) return fused_sweep<T, G, NT, GRAD, FIN_ACC>(B, srow, trow, grow, V, C, keep_res, coef, invS, hot, s_hot);
  return fused_sweep<T, G, NT, GRAD, FIN_FAST>(B, srow, trow, grow, V, C, keep_res, coef, invS, hot, s_hot);
}

// The dominant entry's term of the fused sweep's W in the plain form: its
// float value as the sweep computes it and its value in double (as
// dominant_fix does for the lambda sweep); the difference corrects W.
__device__ inline double dominant_fix_fused(float s, float t, const FusedConst& C) {
  const float a = fmaf(s, LOG2E, -C.msL);
  const float y = fmaf(t - s, C.kL, -C.K);
  const float pt = fexp2(a);
  const float rf = fmaf(pt, fexp2(y), -pt);
  const double yd = (static_cast<double>(C.kL) * (static_cast<double>(t) - static_cast<double>(s)) -
                     static_cast<double>(C.K)) * LN2_D;
  return exp2(static_cast<double>(a)) * expm1(yd) - static_cast<double>(rf);
}

// The lambda node of the fused sums: sum_v p~ 2^{lam X} = 2^AL (sum p~ + W).
// A'''' is not summed: A4 holds the bound max_v (x_v - A')^2 A'' on its size
// (a fourth central moment is at most the squared range times the variance),
// which the model's acceptance test needs and whose term in the model itself
// is negligible within the node's reach (FUSED_REACH; none at the teacher end,
// whose node only settles lambda* = 1).
// acc: the sweep took the expm1 form (else the dominant entry's term of W is
// taken exactly).
__device__ inline LamEval fused_node(const RowStats& R, const FusedSums& S, const FusedConst& C, bool end_first,
                                     bool acc) {
  const float msL = R.ms * LOG2E;
  const double corr = shift_correction(R.ms, msL);
  const double w = (S.v[0] + (acc ? 0.0 : dominant_fix_fused(R.ms, R.t_smax, C))) * corr;
  const double S0 = R.sum_s + w;
  // moments of y under q_lam, then those of X = (y + AL) / lam; x = X ln 2
  const double m1 = S.v[1] * corr / S0, m2 = S.v[2] * corr / S0, m3 = S.v[3] * corr / S0;
  const double c2 = fmax(m2 - m1 * m1, 0.0);
  const double c3 = m3 - 3.0 * m1 * m2 + 2.0 * m1 * m1 * m1;
  const double lam = C.lam_e, il = LN2_D / lam;
  LamEval E;
  E.lam = lam;
  const double lw = log1p(w / R.sum_s);
  E.A = C.AL_e * LN2_D + lw;
  E.A1 = (m1 + C.AL_e) * il;
  E.A2 = c2 * il * il;
  E.A3 = c3 * il * il * il;
  // KL = lam A' - A = ln 2 m1 - log1p(W / sum p~): no cancellation against AL
  E.KL = fmax(LN2_D * m1 - lw, 0.0);
  const double xr = fmax(fabs(static_cast<double>(R.dmax) - R.c - E.A1), fabs(static_cast<double>(R.dmin) - R.c - E.A1));
  E.A4 = xr * xr * E.A2;
  E.reach = end_first ? 0.0 : FUSED_REACH;
  return E;
}

// What the fused sums give at lambda* (L, F): TV, with the bounds that make it
// usable.  hmax bounds |h| over the row; flip bounds the unnormalised mass of
// the entries whose sign of y changes.  false: take the final sweep.
struct FusedFinal {
  bool ok;
  double TV;
  double hmax, flip;
  int why;  // 0: ok; 1: lambda* or the form not from the node; 2: lambda moved too far; 3: TV bound
};

// acc: the sweep took the expm1 form, where each r carries ~1e-7 of itself as
// rounding; in the plain form each carries ~6e-8 of p~ e instead, which over
// P sums to as much as 1e-7 U0.
__device__ inline FusedFinal fused_tv(const RowStats& R, const LamResult& L, const FinalConst& F,
                                      const FusedConst& C, const FusedSums& S, bool acc) {
  FusedFinal out;
  out.ok = false;
  out.TV = 0.0;
  out.hmax = out.flip = 0.0;
  out.why = 1;
  if (L.sweeps != 0 || L.qp || F.wide || F.cL != C.cL || F.msL != C.msL) return out;
  out.why = 2;
  const double dl = static_cast<double>(F.lam) - C.lam_e;
  const double dA = static_cast<double>(F.AL) - C.AL_e;
  const double lg = C.lam_e;
  // |X| over the row (X = d log2 e - cL), with a margin for its rounding
  const double xa = fmax(fabs(static_cast<double>(R.dmax) * LOG2E - C.cL),
                         fabs(static_cast<double>(R.dmin) * LOG2E - C.cL)) * (1.0 + 1e-6) + 1e-6;
  const double hmax = fabs(dl) * xa + fabs(dA);
  // an entry's exponent moves by h = rho y + H0 (X = (y + AL) / lam_g): its
  // sign changes only where |y| <= |H0| / (1 - |rho|) (plus the rounding of y)
  const double rho = dl / lg;
  const double H0 = dl * C.AL_e / lg - dA;
  if (!(fabs(rho) < 0.5)) return out;
  const double Hf = fabs(H0) / (1.0 - fabs(rho)) + 1e-7;
  if (!(Hf < static_cast<double>(FUSED_BAND)) || !(hmax < 0.01)) return out;
  out.why = 3;
  // such an entry's residual at lambda* is below p~ e (2^Hf - 1) on either side
  const double flip = S.Bd * Hf * LN2_D * 1.02;
  const double tvu = S.T0 + LN2_D * (rho * S.U1 + H0 * S.U0);
  // the rest of 2^h - 1 after its linear term, at most (h ln 2)^2 / 2 (1 + h
  // ln 2): summed over P with (rho y + H0)^2 <= 2 rho^2 y^2 + 2 H0^2 and
  // sum_P p~ e y^2 <= S2 (every entry)
  const double h2 = hmax * LN2_D;
  const double sq = 2.0 * (rho * rho * fabs(S.v[2]) + H0 * H0 * S.U0);
  const double err = flip + 0.5 * LN2_D * LN2_D * sq * (1.0 + h2) + 1e-7 * ((acc ? S.T0 : S.U0) + S.U0 * h2);
  if (!(tvu > 0.0) || !(err <= FUSED_TV_TOL * tvu)) return out;
  out.ok = true;
  out.why = 0;
  out.TV = tvu * shift_correction(R.ms, C.msL) / R.sum_s;
  out.hmax = hmax;
  out.flip = flip;
  return out;
}

// What wave 0 settles for a row between sweeps, read by every thread after a
// barrier (the other waves skip the serial arithmetic).
struct RowPlan {
  StartPoint S0;
  LamResult L;
  FinalConst F;
  FusedFinal FF;
  int fused;   // the row takes the fused sweep
  int state;   // after it: 1 settled, 0 final sweep after all, -1 the search needs sweeps
  int C;       // the accept decision at lambda* (state >= 0)
  int z;       // the proposal, and its s and t (wave_proposal)
  float sz, tz;
};

// The chunk level of the residual race from masses known within bounds
// (mass_bound(c, m, b): |true mass - m| <= b, m >= 0): the winner by the
// masses m, or -1 when a chunk could still beat it within the bounds (the
// caller then takes the final sweep).  Keys and ties as in chunk_race.
template <int NT, typename SH, typename F>
__device__ int chunk_race_certain(Block<NT, SH>& B, int nchunks, uint64_t seed, uint32_t stream, uint64_t g,
                                  F mass_bound) {
  double best = __builtin_huge_val();
  int bi = 0x7fffffff;
  // ln E of this thread's first chunk, kept for the second pass
  auto ln_e = [&](int c) {
    return log(-log(static_cast<double>(philox_uniform(seed, stream, g, static_cast<uint32_t>(c)))));
  };
  const double le0 = B.tid < nchunks ? ln_e(B.tid) : 0.0;
  for (int c = B.tid; c < nchunks; c += NT) {
    double m, b;
    mass_bound(c, m, b);
    if (m > 0.0) {
      const double key = (c == B.tid ? le0 : ln_e(c)) - log(m);
      if (key < best) { best = key; bi = c; }
    }
  }
  B.argmin(best, bi);
  if (bi >= nchunks) return -1;
  double mw, bw;
  mass_bound(bi, mw, bw);
  if (!(mw - bw > 0.0)) return -1;
  const double key_hi = ln_e(bi) - log(mw - bw);
  float amb = 0.0f;
  for (int c = B.tid; c < nchunks; c += NT) {
    if (c == bi) continue;
    double m, b;
    mass_bound(c, m, b);
    if (m + b > 0.0 && (c == B.tid ? le0 : ln_e(c)) - log(m + b) <= key_hi) amb = 1.0f;
  }
  return B.max(amb) > 0.0f ? -1 : bi;
}

// Standalone routed loss, first sweep: the log-sum-exp of one array, with the
// next chunk's loads in flight.  Exponents are taken against the wave's
// running maximum as one fma, fma(s, log2 e, -MsL) with MsL = Ms log2(e)
// rounded once; a chunk that raises the maximum rescales the sum.  Returns S
// with sum_v e^(s_v) = 2^msL S for the block's msL (written to *msL_out), so
// that lse = msL ln 2 + ln S and p_v = 2^(s_v log2 e - msL) / S, the form the
// gradient sweep evaluates.
template <typename T, int NT, typename SH>
__device__ double lse_sweep(Block<NT, SH>& B, const T* srow, int V, float* msL_out) {
  constexpr int NW = NT / WAVE;
  float Ms = -finf(), MsL = -finf();
  double Ss = 0.0;
  for_chunks1<T, NW, fill_mode<T, SH>()>(srow, V, B.wave, B.lane, [&](auto tail, const float* s, uint32_t vm, int c) {
    constexpr bool TAIL = decltype(tail)::value;
    float ls = -finf();
#pragma unroll
    for (int e = 0; e < EPL; ++e)
      if (SAKI_VALID(e)) ls = fmaxf(ls, s[e]);
    if (wave_any(ls > Ms)) {
      const float cms = wave_max(ls);
      const float cmsL = __fmul_rn(cms, LOG2E);
      Ss *= static_cast<double>(fexp2(__fsub_rn(MsL, cmsL)));
      Ms = cms;
      MsL = cmsL;
    }
    double ps = 0.0;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      float es = fexp2(fmaf(s[e], LOG2E, -MsL));
      if (TAIL && !SAKI_VALID(e)) es = 0.f;
      ps += static_cast<double>(es);
    }
    Ss += ps;
  }, row_cache<T>(B.sh));
  const float ms = B.max(Ms);
  const float msL = __fmul_rn(ms, LOG2E);
  double v[1] = {(Ms == -finf()) ? 0.0 : (Ms == ms) ? Ss : Ss * static_cast<double>(fexp2(__fsub_rn(MsL, msL)))};
  B.sum(v);
  *msL_out = msL;
  // the maximum's own term exactly: 2^d0 (d0 = ms log2 e - msL, exact in
  // double) instead of its float rounding (see stats_combine)
  if (isfinite(ms)) {
    const double d0 = static_cast<double>(LOG2E) * static_cast<double>(ms) - static_cast<double>(msL);
    v[0] += exp2(d0) - static_cast<double>(fexp2(fmaf(ms, LOG2E, -msL)));
  }
  return v[0];
}

// Standalone routed loss, second sweep: grad_v = coef * p_v with the
// indicator entry (hot, logit s_hot) rewritten after the loop by the thread
// that stored it, as in the final sweep; a row flagged nan_row is all NaN and
// a row with coef = 0 all zeros.
template <typename T, typename G, int NT, typename SH>
__device__ void route_grad_sweep(Block<NT, SH>& B, const T* srow, G* grow, int V, float msL, float invS,
                                 float coef, int hot, float s_hot, bool nan_row) {
  constexpr int NW = NT / WAVE;
  if (!nan_row && coef == 0.0f) {
    // a masked row (or a zero weight): exact zeros whatever the logits
    fill_row<G, NT>(B.wave, B.lane, grow, V, 0.0f);
    return;
  }
  const float cf = nan_row ? __builtin_nanf("") : coef;
  for_chunks1<T, NW, use_mode<T, SH>()>(srow, V, B.wave, B.lane, [&](auto tail, const float* s, uint32_t vm, int c) {
    constexpr bool TAIL = decltype(tail)::value;
    float g[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) g[e] = cf * (fexp2(fmaf(s[e], LOG2E, -msL)) * invS);
    store_lane<G, TAIL>(grow, c, B.lane, V, g);
  }, row_cache<T>(B.sh));
  if (!nan_row && hot >= 0 && hot < V && B.tid == entry_owner<NT>(hot)) {
    const float p = fexp2(fmaf(s_hot, LOG2E, -msL)) * invS;
    Storer<G>::store1(grow + hot, coef * (p - 1.0f));
  }
}

#undef SAKI_VALID

// ---------------------------------------------------------------------------
// Two-level exponential races (the sampler this library fixes for z ~ p and
// c ~ [q - p]_+): the chunk with the smallest E_c / W_c wins, then the entry
// of that chunk with the smallest E_v / w_v; ties to the lowest index.  Keys
// are compared as ln E - ln w.  One Philox block gives the uniforms of four
// consecutive indices.
// ---------------------------------------------------------------------------

// Chunk level.  logw(c) returns ln W_c up to a row constant, or -inf.  One
// chunk per thread: the double-precision logs dominate, not the Philox block.
template <int NT, typename SH, typename F>
__device__ int chunk_race(Block<NT, SH>& B, int nchunks, uint64_t seed, uint32_t stream, uint64_t g,
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
template <int NT, typename SH, typename F>
__device__ int elem_race(Block<NT, SH>& B, int c, int V, uint64_t seed, uint32_t stream, uint64_t g,
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

// The entry-level race in two halves.  elem_fetch loads this thread's four
// consecutive entries of s and t in chunk c (one vector load per array), so
// that a caller can issue it before a long step and hide its latency;
// elem_pick then runs the race of elem_race on them (same uniforms, keys and
// ties) and returns the winner with its s and t, so no later load is needed.
// logw(s, t, v) returns ln w_v up to a row constant, or -inf.
// The entries are held as loaded (packed bf16 words, or floats) and unpacked
// when raced, so that a fetch kept across the lambda search holds few registers.
template <typename T>
struct ElemFetch;
template <>
struct ElemFetch<uint16_t> {
  uint2 qs, qt;
  int v0;  // first of this thread's entries
  __device__ float s(int k) const {
    const uint32_t w = (k < 2) ? qs.x : qs.y;
    return __uint_as_float((k & 1) ? (w & 0xffff0000u) : (w << 16));
  }
  __device__ float t(int k) const {
    const uint32_t w = (k < 2) ? qt.x : qt.y;
    return __uint_as_float((k & 1) ? (w & 0xffff0000u) : (w << 16));
  }
};
template <>
struct ElemFetch<float> {
  float4 qs, qt;
  int v0;
  __device__ float s(int k) const { return k == 0 ? qs.x : k == 1 ? qs.y : k == 2 ? qs.z : qs.w; }
  __device__ float t(int k) const { return k == 0 ? qt.x : k == 1 ? qt.y : k == 2 ? qt.z : qt.w; }
};

template <typename T, int NT>
__device__ __forceinline__ ElemFetch<T> elem_fetch(const T* srow, const T* trow, int c, int V, int tid) {
  static_assert(4 * NT >= CHUNK, "four entries per thread cover a chunk");
  ElemFetch<T> f;
  const int hi = min(V, c * CHUNK + CHUNK);
  f.v0 = c * CHUNK + 4 * tid;
  if (f.v0 + 4 <= hi) {
    if constexpr (sizeof(T) == 2) {
      f.qs = *reinterpret_cast<const uint2*>(srow + f.v0);
      f.qt = *reinterpret_cast<const uint2*>(trow + f.v0);
    } else {
      f.qs = *reinterpret_cast<const float4*>(srow + f.v0);
      f.qt = *reinterpret_cast<const float4*>(trow + f.v0);
    }
  } else {
    // the ragged end of the row: entries past it read as 0 (and are not raced)
    if constexpr (sizeof(T) == 2) {
      uint32_t ws[4], wt[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const bool in = f.v0 + k < hi;
        ws[k] = in ? static_cast<uint32_t>(srow[f.v0 + k]) : 0u;
        wt[k] = in ? static_cast<uint32_t>(trow[f.v0 + k]) : 0u;
      }
      f.qs = make_uint2(ws[0] | (ws[1] << 16), ws[2] | (ws[3] << 16));
      f.qt = make_uint2(wt[0] | (wt[1] << 16), wt[2] | (wt[3] << 16));
    } else {
      float xs[4], xt[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const bool in = f.v0 + k < hi;
        xs[k] = in ? srow[f.v0 + k] : 0.0f;
        xt[k] = in ? trow[f.v0 + k] : 0.0f;
      }
      f.qs = make_float4(xs[0], xs[1], xs[2], xs[3]);
      f.qt = make_float4(xt[0], xt[1], xt[2], xt[3]);
    }
  }
  return f;
}

template <int NT, typename SH, typename T, typename F>
__device__ int elem_pick(Block<NT, SH>& B, const ElemFetch<T>& f, int c, int V, uint64_t seed, uint32_t stream,
                         uint64_t g, F logw, float* s_win, float* t_win) {
  float best = finf(), bs = 0.0f, bt = 0.0f;
  int bi = 0x7fffffff;
  const int hi = min(V, c * CHUNK + CHUNK);
  if (f.v0 < hi) {
    const uint4 w = philox_block(seed, stream, g, static_cast<uint32_t>(f.v0 >> 2));
    const uint32_t words[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int v = f.v0 + k;
      if (v < hi) {
        const float sk = f.s(k), tk = f.t(k);
        const float lw = logw(sk, tk, v);
        if (lw > -finf()) {
          const float u = word_to_uniform(words[k]);
          const float E = -flog2(u) * LN2;
          const float key = flog2(E) * LN2 - lw;
          if (key < best) { best = key; bi = v; bs = sk; bt = tk; }
        }
      }
    }
  }
  B.argmin_with(best, bi, bs, bt);
  *s_win = bs;
  *t_win = bt;
  return bi;
}

// The two-level race of chunk_race and elem_race run by one wave alone (same
// uniforms, keys and ties), so that it can overlap other waves' serial
// steps: the chunk keys in double, chunks lane, lane + 64, ...; then the
// entries of the winning chunk, four consecutive ones per load as elem_fetch
// takes them (a lane covers the four quarter-chunks j = 0..3 of a 256-thread
// block's layout).  chunk_logw(c) as for chunk_race; logw(s, t, v) as for
// elem_pick.  Returns the winner (or >= V if no entry has weight) with its s
// and t, on every lane.
template <typename T, typename FC, typename FE>
__device__ int wave_proposal(const T* srow, const T* trow, int nchunks, int V, int lane, uint64_t seed,
                             uint32_t chunk_stream, uint32_t elem_stream, uint64_t g, FC chunk_logw, FE logw,
                             float* s_win, float* t_win) {
  double ck = __builtin_huge_val();
  int ci = 0x7fffffff;
  for (int c = lane; c < nchunks; c += WAVE) {
    const double lw = chunk_logw(c);
    if (lw > -__builtin_huge_val()) {
      const double u = static_cast<double>(philox_uniform(seed, chunk_stream, g, static_cast<uint32_t>(c)));
      const double key = log(-log(u)) - lw;
      if (key < ck) { ck = key; ci = c; }
    }
  }
  wave_argmin(ck, ci);
  const int c = ci < nchunks ? ci : 0;
  const int hi = min(V, c * CHUNK + CHUNK);
  float best = finf(), bs = 0.0f, bt = 0.0f;
  int bi = 0x7fffffff;
#pragma unroll
  for (int j = 0; j < CHUNK / (4 * WAVE); ++j) {
    const ElemFetch<T> f = elem_fetch<T, CHUNK / 4>(srow, trow, c, V, lane + WAVE * j);
    if (f.v0 < hi) {
      const uint4 w = philox_block(seed, elem_stream, g, static_cast<uint32_t>(f.v0 >> 2));
      const uint32_t words[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int v = f.v0 + k;
        if (v < hi) {
          const float sk = f.s(k), tk = f.t(k);
          const float lw = logw(sk, tk, v);
          if (lw > -finf()) {
            const float u = word_to_uniform(words[k]);
            const float E = -flog2(u) * LN2;
            const float key = flog2(E) * LN2 - lw;
            if (key < best) { best = key; bi = v; bs = sk; bt = tk; }
          }
        }
      }
    }
  }
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) {
    const float k2 = __shfl_xor(best, o, WAVE);
    const int i2 = __shfl_xor(bi, o, WAVE);
    const float a2 = __shfl_xor(bs, o, WAVE);
    const float b2 = __shfl_xor(bt, o, WAVE);
    if (k2 < best || (k2 == best && i2 < bi)) { best = k2; bi = i2; bs = a2; bt = b2; }
  }
  *s_win = bs;
  *t_win = bt;
  return bi;
}

}  // namespace saki
