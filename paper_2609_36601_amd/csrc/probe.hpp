// Fixed-prefix probe metrics of the student S = softmax(s) against the
// teacher T = softmax(t) at each row (the paper's probe analysis):
//   C_1 = S(v*_T), C_k = sum of S over the teacher's Top-k set (ties to the
//   lower index), KL(T || S) = E_T[t - s] - (lse_t - lse_s), H(S).
// One workgroup per row.  A sweep gives the normalisers and moments; the
// teacher's k-th largest logit is found by bisection over the logits'
// order-preserving integer images (16 bits for bf16, 32 for f32; one counting
// sweep per bit), ties at the threshold go to the lowest indices (bisection
// over the index), and a last sweep gathers the Top-k set.  Probe sets are
// small (thousands of positions), so the sweeps re-read rows freely.
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
    const uint32_t u = __float_as_uint(x);
    return ((u >> 31) ? ~u : (u | 0x80000000u)) >> 16;
  }
};
template <>
struct OrderKey<float> {
  static constexpr int BITS = 32;
  static __device__ __forceinline__ uint32_t of(float x) {
    const uint32_t u = __float_as_uint(x);
    return (u >> 31) ? ~u : (u | 0x80000000u);
  }
};

struct ProbeShared {
  double red_d[NT / WAVE][RED_MAX];
  float red_f[NT / WAVE][4];
  int red_i[NT / WAVE][4];
  int n_sel;
  int sel_idx[SAKI_MAX_PROBE_K];
  float sel_t[SAKI_MAX_PROBE_K];
};

// Number of entries v of the row with pred(key(t_v), v), summed over the block.
template <typename T, typename Pred>
__device__ double probe_count(Block<NT, ProbeShared>& B, const T* trow, int V, Pred pred) {
  double n = 0;
  for (int v = B.tid; v < V; v += NT) n += pred(OrderKey<T>::of(Loader<T>::load1(trow + v)), v) ? 1.0 : 0.0;
  double r[1] = {n};
  B.sum(r);
  return r[0];
}

template <typename T>
__global__ __launch_bounds__(NT, WG_PER_CU) void probe_kernel(ProbeParams P) {
  __shared__ ProbeShared sh;
  Block<NT, ProbeShared> B(sh);
  constexpr int NW = NT / WAVE;
  const int V = P.V, k = P.k;
  for (int64_t r = blockIdx.x; r < P.n_rows; r += gridDim.x) {
    const T* srow = static_cast<const T*>(P.s) + r * P.stride;
    const T* trow = static_cast<const T*>(P.t) + r * P.stride;
    // sums relative to the running maxima: Ss = sum e^{s-Ms}, Sa = sum e^{s-Ms} (s-Ms),
    // St = sum e^{t-Mt}, Td = sum e^{t-Mt} (t-s)
    float Ms = -finf(), Mt = -finf();
    double Ss = 0, Sa = 0, St = 0, Td = 0;
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
                        if (wave_any(ls > Ms)) {
                          const float m = wave_max(ls);
                          const double f = static_cast<double>(fexp2((Ms - m) * LOG2E));
                          // sum e^{s-m}(s-m) = f (sum e^{s-Ms}(s-Ms) - (m - Ms) sum e^{s-Ms})
                          Sa = (Ms == -finf()) ? 0.0 : f * (Sa - (static_cast<double>(m) - Ms) * Ss);
                          Ss *= f;
                          Ms = m;
                        }
                        if (wave_any(lt > Mt)) {
                          const float m = wave_max(lt);
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
    // the k-th largest key: the largest x with #{key >= x} >= k
    uint32_t lo = 0, hi = (OrderKey<T>::BITS == 32) ? 0xffffffffu : 0xffffu;
    while (lo < hi) {
      const uint32_t mid = lo + static_cast<uint32_t>((static_cast<uint64_t>(hi) - lo + 1) / 2);
      const double n = probe_count<T>(B, trow, V, [&](uint32_t key, int) { return key >= mid; });
      if (n >= k) lo = mid; else hi = mid - 1;
    }
    const uint32_t K = lo;
    const double n_gt = probe_count<T>(B, trow, V, [&](uint32_t key, int) { return key > K; });
    const double need = k - n_gt;  // entries with key K to take, lowest indices first
    // the smallest J with #{key == K, v <= J} >= need
    int jlo = 0, jhi = V - 1;
    while (jlo < jhi) {
      const int mid = jlo + (jhi - jlo) / 2;
      const double n = probe_count<T>(B, trow, V, [&](uint32_t key, int v) { return key == K && v <= mid; });
      if (n >= need) jhi = mid; else jlo = mid + 1;
    }
    const int J = jlo;
    if (B.tid == 0) sh.n_sel = 0;
    __syncthreads();
    for (int v = B.tid; v < V; v += NT) {
      const float tv = Loader<T>::load1(trow + v);
      const uint32_t key = OrderKey<T>::of(tv);
      if (key > K || (key == K && v <= J)) {
        const int slot = atomicAdd(&sh.n_sel, 1);
        if (slot < SAKI_MAX_PROBE_K) {
          sh.sel_idx[slot] = v;
          sh.sel_t[slot] = tv;
        }
      }
    }
    __syncthreads();
    if (B.tid == 0) {
      const int n = min(sh.n_sel, k);
      // order by (t descending, index ascending)
      for (int i = 1; i < n; ++i) {
        const int vi = sh.sel_idx[i];
        const float ti = sh.sel_t[i];
        int j = i - 1;
        while (j >= 0 && (sh.sel_t[j] < ti || (sh.sel_t[j] == ti && sh.sel_idx[j] > vi))) {
          sh.sel_idx[j + 1] = sh.sel_idx[j];
          sh.sel_t[j + 1] = sh.sel_t[j];
          --j;
        }
        sh.sel_idx[j + 1] = vi;
        sh.sel_t[j + 1] = ti;
      }
      double ck = 0.0, c1 = 0.0;
      for (int i = 0; i < n; ++i) {
        const double p = exp(static_cast<double>(Loader<T>::load1(srow + sh.sel_idx[i])) - lse_s);
        ck += p;
        if (i == 0) c1 = p;
      }
      const double kl = Td / St - (lse_t - lse_s);
      const double h = log(Ss) - Sa / Ss;  // lse_s - E_S[s]
      if (P.c1) P.c1[r] = static_cast<float>(c1);
      if (P.ck) P.ck[r] = static_cast<float>(ck);
      if (P.kl_ts) P.kl_ts[r] = static_cast<float>(fmax(kl, 0.0));
      if (P.entropy) P.entropy[r] = static_cast<float>(fmax(h, 0.0));
      if (P.row_status) P.row_status[r] = SAKI_ROW_OK;
      if (P.topk)
        for (int i = 0; i < k; ++i) P.topk[r * k + i] = i < n ? sh.sel_idx[i] : -1;
    }
    __syncthreads();
  }
}

}  // namespace saki
