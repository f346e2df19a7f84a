// Fixed-prefix probe metrics of the student S = softmax(s) against the
// teacher T = softmax(t) at each row (the paper's probe analysis):
//   C_1 = S(v*_T), C_k = sum of S over the teacher's Top-k set (ties to the
//   lower index), KL(T || S) = E_T[t - s] - (lse_t - lse_s), H(S).
// One workgroup per row.  A sweep gives the normalisers and moments, each
// thread's largest teacher logit and each chunk's.  L, the k-th largest of the
// threads' maxima, bounds the k-th largest logit from below, and the entries
// at or above L are gathered from the chunks whose maximum reaches L (a few
// chunks of the row).  When more entries than LDS holds reach L, the k-th
// largest logit is found by a search over the logits' order-preserving integer
// images (16 bits for bf16, 32 for f32) that counts four pivots per sweep;
// ties at the threshold go to the lowest indices (the same search over the
// index, only when the threshold value has more entries than are taken), and
// a last sweep gathers the Top-k set.
#pragma once

#include "row_engine.hpp"

namespace saki {

struct ProbeParams {
  const void* s;
  const void* t;
  int64_t n_rows;
  int64_t stride;
  int V;
  int k;
  float* c1;
  float* ck;
  float* kl_ts;
  float* entropy;
  int32_t* topk;      // [n_rows, k] or NULL
  uint8_t* row_status;
};

template <typename T>
struct OrderKey;
template <>
struct OrderKey<uint16_t> {
  static constexpr int BITS = 16;
  static __device__ __forceinline__ uint32_t of(float x) {
    const uint32_t u = x == 0.0f ? 0u : __float_as_uint(x);  // -0 and +0 tie
    return ((u >> 31) ? ~u : (u | 0x80000000u)) >> 16;
  }
};
template <>
struct OrderKey<float> {
  static constexpr int BITS = 32;
  static __device__ __forceinline__ uint32_t of(float x) {
    const uint32_t u = x == 0.0f ? 0u : __float_as_uint(x);  // -0 and +0 tie
    return (u >> 31) ? ~u : (u | 0x80000000u);
  }
};

// Entries the gathering sweep can hold: those above the threshold value and,
// when they fit, every entry at it (ties then need no index search).
constexpr int PROBE_SEL_CAP = NT;
static_assert(PROBE_SEL_CAP >= SAKI_MAX_PROBE_K, "the gathered set holds the Top-k");
// Rows of up to PROBE_MAXC chunks keep each chunk's largest teacher logit.
constexpr int PROBE_MAXC = 512;
// Workgroups per CU: three, so that while some are in a row's serial steps
// (reductions, the threshold, the gathering) the others stream.
constexpr int PROBE_WG_PER_CU = 3;

struct ProbeShared {
  double red_d[NT / WAVE][RED_MAX];
  float red_f[NT / WAVE][4];
  int red_i[NT / WAVE][4];
  int n_sel;
  float thread_max[NT];  // each thread's largest teacher logit of the row
  float chunk_tmax[PROBE_MAXC];  // each chunk's largest teacher logit
  int sel_idx[PROBE_SEL_CAP];   // gathered entries, in arrival order
  float sel_t[PROBE_SEL_CAP];
  int ord_idx[PROBE_SEL_CAP];   // the same entries by (t descending, index ascending)
};

// Pivots counted per sweep in the Top-k searches (one block sum of that many
// doubles).  Four keep the kernel free of register spills at three workgroups
// per CU; the searches run only when more than PROBE_SEL_CAP entries reach L.
constexpr int PROBE_PIVOTS = 4;

struct Pivots {
  uint32_t m[PROBE_PIVOTS];
};
struct PivotCounts {
  double n[PROBE_PIVOTS];
};

// One sweep over the teacher row, for every pivot i: #{v : key(t_v) >= m_i}
// (BY_INDEX false) or #{v : key(t_v) == K, v <= m_i} (BY_INDEX true), summed
// over the block (every thread gets the same counts).  Pivots and counts are
// passed by value so that they stay in registers.
template <bool BY_INDEX, typename T>
__device__ __forceinline__ PivotCounts probe_counts(Block<NT, ProbeShared>& B, const T* trow, int V, const Pivots pv,
                                                    uint32_t K) {
  constexpr int NW = NT / WAVE;
  uint32_t cnt[PROBE_PIVOTS];
#pragma unroll
  for (int i = 0; i < PROBE_PIVOTS; ++i) cnt[i] = 0u;
  for_chunks1<T, NW>(trow, V, B.wave, B.lane, [&](auto tail, const float* x, uint32_t vm, int c) {
    constexpr bool TAIL = decltype(tail)::value;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      const bool ok = !TAIL || ((vm >> e) & 1u);
      const uint32_t key = OrderKey<T>::of(x[e]);
      if (BY_INDEX) {
        // entries outside the row or off the threshold value get an index no pivot reaches
        const uint32_t v = (ok && key == K) ? static_cast<uint32_t>(c * CHUNK + elem_offset(B.lane, e)) : 0xffffffffu;
#pragma unroll
        for (int i = 0; i < PROBE_PIVOTS; ++i) cnt[i] += (v <= pv.m[i]) ? 1u : 0u;
      } else {
        // every pivot is >= 1 (key 0 is the image of a NaN, and rows with a
        // non-finite logit are not searched): key 0 is never counted
        const uint32_t kk = ok ? key : 0u;
#pragma unroll
        for (int i = 0; i < PROBE_PIVOTS; ++i) cnt[i] += (kk >= pv.m[i]) ? 1u : 0u;
      }
    }
  });
  double n[PROBE_PIVOTS];
#pragma unroll
  for (int i = 0; i < PROBE_PIVOTS; ++i) n[i] = static_cast<double>(cnt[i]);
  B.sum(n);
  PivotCounts out;
#pragma unroll
  for (int i = 0; i < PROBE_PIVOTS; ++i) out.n[i] = n[i];
  return out;
}

template <typename T>
__global__ __launch_bounds__(NT, PROBE_WG_PER_CU) void probe_kernel(ProbeParams P) {
  __shared__ ProbeShared sh;
  Block<NT, ProbeShared> B(sh);
  constexpr int NW = NT / WAVE;
  const int V = P.V, k = P.k;
  const int nch = (V + CHUNK - 1) / CHUNK;
  for (int64_t r = blockIdx.x; r < P.n_rows; r += gridDim.x) {
    const T* srow = static_cast<const T*>(P.s) + r * P.stride;
    const T* trow = static_cast<const T*>(P.t) + r * P.stride;
    // sums relative to the running maxima: Ss = sum e^{s-Ms}, Sa = sum e^{s-Ms} (s-Ms),
    // St = sum e^{t-Mt}, Td = sum e^{t-Mt} (t-s)
    float Ms = -finf(), Mt = -finf();
    double Ss = 0, Sa = 0, St = 0, Td = 0;
    float Lt = -finf();  // this thread's largest teacher logit
    bool finite = true;
    for_chunks<T, NW>(srow, trow, V, B.wave, B.lane,
                      [&](auto tail, const float* s, const float* t, uint32_t vm, int c) {
                        constexpr bool TAIL = decltype(tail)::value;
                        float ls = -finf(), lt = -finf();
                        bool fin = true;
#pragma unroll
                        for (int e = 0; e < EPL; ++e) {
                          if (!TAIL || ((vm >> e) & 1u)) {
                            ls = fmaxf(ls, s[e]);
                            lt = fmaxf(lt, t[e]);
                            fin = fin && isfinite(s[e]) && isfinite(t[e]);
                          }
                        }
                        finite = finite && !wave_any(!fin);
                        Lt = fmaxf(Lt, lt);
                        const float cmt = wave_max(lt);
                        if (c < PROBE_MAXC && B.lane == 0) sh.chunk_tmax[c] = cmt;
                        if (wave_any(ls > Ms)) {
                          const float m = wave_max(ls);
                          const double f = static_cast<double>(fexp2((Ms - m) * LOG2E));
                          // sum e^{s-m}(s-m) = f (sum e^{s-Ms}(s-Ms) - (m - Ms) sum e^{s-Ms})
                          Sa = (Ms == -finf()) ? 0.0 : f * (Sa - (static_cast<double>(m) - Ms) * Ss);
                          Ss *= f;
                          Ms = m;
                        }
                        if (cmt > Mt) {
                          const float m = cmt;
                          const double f = static_cast<double>(fexp2((Mt - m) * LOG2E));
                          St *= f;
                          Td *= f;
                          Mt = m;
                        }
                        float ss = 0.f, sa = 0.f, st = 0.f, td = 0.f;
#pragma unroll
                        for (int e = 0; e < EPL; ++e) {
                          if (!TAIL || ((vm >> e) & 1u)) {
                            const float a = s[e] - Ms;
                            const float es = fexp2(a * LOG2E);
                            const float et = fexp2((t[e] - Mt) * LOG2E);
                            ss += es;
                            sa = fmaf(es, a, sa);
                            st += et;
                            td = fmaf(et, t[e] - s[e], td);
                          }
                        }
                        Ss += ss; Sa += sa; St += st; Td += td;
                      });
    // combine the waves (rescaled to the block maxima)
    const float ms = B.max(Ms), mt = B.max(Mt);
    {
      const double fs = (Ms == -finf()) ? 0.0 : static_cast<double>(fexp2((Ms - ms) * LOG2E));
      const double ft = (Mt == -finf()) ? 0.0 : static_cast<double>(fexp2((Mt - mt) * LOG2E));
      const double dm = static_cast<double>(ms) - Ms;
      double v[5] = {Ss * fs, (Ms == -finf()) ? 0.0 : fs * (Sa - dm * Ss), St * ft, Td * ft,
                     finite ? 0.0 : 1.0};
      B.sum(v);
      Ss = v[0]; Sa = v[1]; St = v[2]; Td = v[3];
      finite = v[4] == 0.0;
    }
    const double lse_s = static_cast<double>(ms) + log(Ss);
    const double lse_t = static_cast<double>(mt) + log(St);
    if (!finite || !isfinite(lse_s) || !isfinite(lse_t)) {
      if (B.tid == 0) {
        if (P.c1) P.c1[r] = nanf_();
        if (P.ck) P.ck[r] = nanf_();
        if (P.kl_ts) P.kl_ts[r] = nanf_();
        if (P.entropy) P.entropy[r] = nanf_();
        if (P.row_status) P.row_status[r] = SAKI_ROW_NONFINITE;
      }
      if (P.topk)
        for (int j = B.tid; j < k; j += NT) P.topk[r * k + j] = -1;
      continue;
    }
    // The k-th largest key K: the largest x with #{key >= x} >= k, searched with
    // PROBE_PIVOTS pivots per sweep.  Invariants: #{key >= lo} = c_lo >= k and
    // #{key >= hi + 1} = c_up < k.
    // The search starts from [key(L), key(max t)]: L, the k-th largest of the
    // threads' own maxima (k distinct entries of the row), is at most the k-th
    // largest logit; #{key >= key(L)} is counted by the first sweep.
    sh.thread_max[B.tid] = Lt;
    __syncthreads();
    int n_ge = 0;
    for (int u = 0; u < NT; ++u) n_ge += (sh.thread_max[u] >= Lt) ? 1 : 0;
    const float L = B.max(n_ge >= k ? Lt : -finf());
    // Gathers into LDS the entries with KEEP(key, logit, index); every thread
    // gets the number that matched (the set holds the first PROBE_SEL_CAP).
    auto gather = [&](auto keep) {
      if (B.tid == 0) sh.n_sel = 0;
      __syncthreads();
      for_chunks1<T, NW>(trow, V, B.wave, B.lane, [&](auto tail, const float* x, uint32_t vm, int c) {
        constexpr bool TAIL = decltype(tail)::value;
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          if (!TAIL || ((vm >> e) & 1u)) {
            const int v = c * CHUNK + elem_offset(B.lane, e);
            if (keep(OrderKey<T>::of(x[e]), x[e], v)) {
              const int slot = atomicAdd(&sh.n_sel, 1);
              if (slot < PROBE_SEL_CAP) {
                sh.sel_idx[slot] = v;
                sh.sel_t[slot] = x[e];
              }
            }
          }
        }
      });
      __syncthreads();
      const int n = sh.n_sel;
      __syncthreads();  // read by every thread before the next gather clears it
      return n;
    };
    // First sweep: every entry >= L (in the float order of the ranking below,
    // so that -0 and +0 tie).  There are at least k of them, and when they fit
    // the set holds the Top-k with all its ties: no counting sweep is needed.
    int n_got;
    if (nch <= PROBE_MAXC) {
      // only the chunks whose maximum reaches L hold such entries; the test is
      // uniform in the wave that owns the chunk (and stored its maximum)
      if (B.tid == 0) sh.n_sel = 0;
      __syncthreads();
      for (int c = B.wave; c < nch; c += NW) {
        if (!(sh.chunk_tmax[c] >= L)) continue;
        float x[EPL];
        uint32_t vm;
        if (c < V / CHUNK)
          load_lane<T, false>(trow, c, B.lane, V, x, &vm);
        else
          load_lane<T, true>(trow, c, B.lane, V, x, &vm);
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          if (((vm >> e) & 1u) && x[e] >= L) {
            const int slot = atomicAdd(&sh.n_sel, 1);
            if (slot < PROBE_SEL_CAP) {
              sh.sel_idx[slot] = c * CHUNK + elem_offset(B.lane, e);
              sh.sel_t[slot] = x[e];
            }
          }
        }
      }
      __syncthreads();
      n_got = sh.n_sel;
      __syncthreads();  // read by every thread before a later gather clears it
    } else {
      n_got = gather([&](uint32_t, float x, int) { return x >= L; });
    }
    if (n_got > PROBE_SEL_CAP) {
      uint64_t lo = OrderKey<T>::of(L), hi = OrderKey<T>::of(mt);
      double c_lo = __builtin_huge_val(), c_up = 0.0;
      while (lo < hi) {
        Pivots pv;  // in (lo, hi], non-decreasing
#pragma unroll
        for (int i = 0; i < PROBE_PIVOTS; ++i)
          pv.m[i] = static_cast<uint32_t>(lo + 1 + (hi - lo) * static_cast<uint64_t>(i + 1) / (PROBE_PIVOTS + 1));
        if (c_lo == __builtin_huge_val()) {
          // first sweep: lo itself (its count), then lo + 1, lo + 2, lo + 4, ...:
          // L is usually the k-th largest logit itself (the Top-k entries lie in
          // different threads), and then this sweep ends the search
#pragma unroll
          for (int i = 0; i < PROBE_PIVOTS; ++i)
            pv.m[i] = static_cast<uint32_t>(i == 0 ? lo : (lo + (1ull << (i - 1)) < hi ? lo + (1ull << (i - 1)) : hi));
        }
        const PivotCounts pc = probe_counts<false>(B, trow, V, pv, 0u);
        const double* n = pc.n;
        const uint32_t* piv = pv.m;
        // counts fall as pivots rise: lo moves to the last pivot with count >= k,
        // hi below the first with count < k (static indices: no scratch arrays)
        uint64_t lo2 = lo, hi2 = hi;
        double c_lo2 = c_lo, c_up2 = c_up;
#pragma unroll
        for (int i = 0; i < PROBE_PIVOTS; ++i)
          if (n[i] >= k) { lo2 = piv[i]; c_lo2 = n[i]; }
#pragma unroll
        for (int i = PROBE_PIVOTS - 1; i >= 0; --i)
          if (n[i] < k) { hi2 = static_cast<uint64_t>(piv[i]) - 1; c_up2 = n[i]; }
        lo = lo2; hi = hi2; c_lo = c_lo2; c_up = c_up2;
      }
      const uint32_t K = static_cast<uint32_t>(lo);
      const double need = k - c_up;  // entries with key K to take, lowest indices first
      // the smallest J with #{key == K, v <= J} >= need.  Every entry with key K
      // is gathered when there are exactly need of them, or when all entries at
      // and above K fit the gathered set (the ordering then picks the lowest
      // indices); otherwise the index search finds J.
      const bool gather_all = c_lo - c_up == need || c_lo <= static_cast<double>(PROBE_SEL_CAP);
      int J = V - 1;
      if (!gather_all) {
        // invariants: #{key == K, v <= jhi} >= need > #{key == K, v < jlo}
        int jlo = 0, jhi = V - 1;
        while (jlo < jhi) {
          Pivots pv;  // in [jlo, jhi), non-decreasing
#pragma unroll
          for (int i = 0; i < PROBE_PIVOTS; ++i)
            pv.m[i] = static_cast<uint32_t>(jlo + static_cast<int>(static_cast<int64_t>(jhi - jlo) * (i + 1) / (PROBE_PIVOTS + 1)));
          const PivotCounts pc = probe_counts<true>(B, trow, V, pv, K);
          const double* n = pc.n;
          const uint32_t* piv = pv.m;
          // counts grow with the pivot: jlo moves past the last pivot with count
          // < need, jhi to the first with count >= need
          int jlo2 = jlo, jhi2 = jhi;
#pragma unroll
          for (int i = 0; i < PROBE_PIVOTS; ++i)
            if (n[i] < need) jlo2 = static_cast<int>(piv[i]) + 1;
#pragma unroll
          for (int i = PROBE_PIVOTS - 1; i >= 0; --i)
            if (n[i] >= need) jhi2 = static_cast<int>(piv[i]);
          jlo = jlo2;
          jhi = jhi2;
        }
        J = jlo;
      }
      n_got = gather([&](uint32_t key, float, int v) { return key > K || (key == K && v <= J); });
    }
    // rank sort of the gathered entries by (t descending, index ascending)
    const int n_all = min(n_got, PROBE_SEL_CAP);
    if (B.tid < n_all) {
      const int vi = sh.sel_idx[B.tid];
      const float ti = sh.sel_t[B.tid];
      int rank = 0;
      for (int j = 0; j < n_all; ++j) {
        const float tj = sh.sel_t[j];
        rank += (tj > ti || (tj == ti && sh.sel_idx[j] < vi)) ? 1 : 0;
      }
      sh.ord_idx[rank] = vi;
    }
    __syncthreads();
    const int n = min(n_all, k);
    // S over the Top-k set and at the teacher mode, summed over the block
    double pv2[2] = {0.0, 0.0};
    if (B.tid < n) {
      const double p = exp(static_cast<double>(Loader<T>::load1(srow + sh.ord_idx[B.tid])) - lse_s);
      pv2[0] = p;
      if (B.tid == 0) pv2[1] = p;
    }
    B.sum(pv2);
    if (B.tid == 0) {
      const double ck = pv2[0], c1 = pv2[1];
      const double kl = Td / St - (lse_t - lse_s);
      const double h = log(Ss) - Sa / Ss;  // lse_s - E_S[s]
      if (P.c1) P.c1[r] = static_cast<float>(c1);
      if (P.ck) P.ck[r] = static_cast<float>(ck);
      if (P.kl_ts) P.kl_ts[r] = static_cast<float>(fmax(kl, 0.0));
      if (P.entropy) P.entropy[r] = static_cast<float>(fmax(h, 0.0));
      if (P.row_status) P.row_status[r] = SAKI_ROW_OK;
      if (P.topk)
        for (int i = 0; i < k; ++i) P.topk[r * k + i] = i < n ? sh.ord_idx[i] : -1;
    }
    __syncthreads();
  }
}

}  // namespace saki
