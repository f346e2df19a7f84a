// SAKI coupling-and-routing kernels for gfx950 and the C ABI of include/saki.h.
//
// One workgroup of NT = 256 threads (4 waves) owns one row at a time and
// walks the grid's rows persistently; two workgroups share a compute unit, so
// one row's serial steps (reductions, the lambda search, the races) overlap
// the other's streaming sweeps.  The row engine (row_engine.hpp) runs the
// stats sweep, the lambda sweeps and the final sweep over a row.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>

#include <mutex>
#include <string>

#include "../../include/saki.h"
#include "row_engine.hpp"

namespace saki {

constexpr int NT = 256;
constexpr int WG_PER_CU = 2;
// bf16 rows of up to CACHED_MAXC chunks (262,144 entries) use the variant with
// a row cache of CACHE_KC chunks per wave: 4 KiB of chunk masses and 64 KiB of
// cached chunks per workgroup, two workgroups in the 160 KiB of LDS of a CU.
// The cached chunks are read once per row instead of three times.
constexpr int CACHED_MAXC = 256;
constexpr int CACHE_KC = 4;
template <int KC>
using RowSharedK = RowShared<NT, (KC > 0 ? CACHED_MAXC : MAX_CHUNKS), KC>;

struct CoupleParams {
  const void* s;
  const void* t;
  int64_t n_rows;
  int64_t stride;
  int64_t row_offset;
  int V;
  double eps;
  uint64_t seed;
  saki_couple_out out;
  // routing
  const uint8_t* valid;
  float grad_scale;
  float* row_loss;
  double* scaled_loss;  // workspace [n_rows] or NULL
  void* grad;
  int64_t grad_stride;
  int target_mode;      // SAKI_TARGET_MODE or SAKI_TARGET_SAMPLE
  unsigned int* next_row;  // work counter in the caller's workspace, zero at launch
  // Rows resolved in the plain forms whose TV turns out too small for their
  // rounding are listed (redo_list, redo_count, in the workspace) and processed
  // again by a second launch with every sweep in the expm1 form (redo_pass).
  unsigned int* redo_list;
  unsigned int* redo_count;
  int redo_pass;
};

__device__ __forceinline__ float nanf_() { return __builtin_nanf(""); }

// Clears the work counters at the start of a workspace (a kernel rather than
// a memset node, so that a captured graph replays it correctly).
__global__ void clear_counter_kernel(unsigned int* c) {
  if (threadIdx.x < 4) c[threadIdx.x] = 0u;
}

// Takes the next work item (row or block) for the whole workgroup: thread 0
// takes it from the counter with a device atomic and posts it in LDS, and
// readfirstlane makes the index, and so the caller's loop exit, uniform in
// every wave, so all threads reach the same barriers.
__device__ __forceinline__ unsigned int take_next(unsigned int* counter, unsigned int* slot) {
  if (threadIdx.x == 0) *slot = atomicAdd(counter, 1u);
  __syncthreads();
  const unsigned int v = static_cast<unsigned int>(__builtin_amdgcn_readfirstlane(static_cast<int>(*slot)));
  __syncthreads();
  return v;
}

// K34: the stats sweep sums k3, k4 (radii below K34_EPS).
template <typename T, typename G, bool ROUTE, bool GRAD, int KC, bool K34>
__global__ __launch_bounds__(NT, WG_PER_CU) void couple_kernel(CoupleParams P) {
  __shared__ RowSharedK<KC> sh;
  __shared__ RowPlan plan;
  Block<NT, RowSharedK<KC>> B(sh);
  const int V = P.V;
  const int nch = (V + CHUNK - 1) / CHUNK;
  // Workgroups take rows from a counter: their speeds differ (the two
  // workgroups of a CU, and CUs, get unequal shares of the memory system), so
  // a fixed stride left the slowest ones finishing ~15% after the median.
  // Each iteration takes a new row or ends the loop: at most n_rows + 1.
  __shared__ unsigned int next_r;
  // the second launch takes its rows from the list the first one made
  const unsigned int n_work = P.redo_pass
      ? static_cast<unsigned int>(__builtin_amdgcn_readfirstlane(static_cast<int>(*P.redo_count)))
      : static_cast<unsigned int>(P.n_rows);
  const bool force_acc = P.redo_pass != 0;
  for (int64_t it = 0; it <= P.n_rows; ++it) {
    const unsigned int ru = take_next(P.next_row, &next_r);
    // unsigned: n_rows < 2^31 and the counter stays below n_rows + grid
    if (ru >= n_work) break;
    const int64_t r = static_cast<int64_t>(P.redo_pass ? P.redo_list[ru] : ru);
    const T* srow = static_cast<const T*>(P.s) + r * P.stride;
    const T* trow = static_cast<const T*>(P.t) + r * P.stride;
    G* grow = GRAD ? static_cast<G*>(P.grad) + r * P.grad_stride : nullptr;
    const uint64_t g = static_cast<uint64_t>(P.row_offset + r);
    const float M = (ROUTE && P.valid) ? (P.valid[r] ? 1.0f : 0.0f) : 1.0f;

    const bool sample_target = ROUTE && P.target_mode == SAKI_TARGET_SAMPLE;
    const RowStats& R = stats_sweep<T, NT, true, K34>(B, srow, trow, V, mid_lambda(P.eps), true, sample_target);
    if (!R.finite) {
      if (GRAD) fill_row<G, NT>(B.wave, B.lane, grow, V, M != 0.0f ? nanf_() : 0.0f);
      if (B.tid == 0) {
        const saki_couple_out& o = P.out;
        if (o.lambda) o.lambda[r] = nanf_();
        if (o.kl) o.kl[r] = nanf_();
        if (o.tv) o.tv[r] = nanf_();
        if (o.accept_prob) o.accept_prob[r] = nanf_();
        if (o.margin) o.margin[r] = nanf_();
        if (o.logp_token) o.logp_token[r] = nanf_();
        if (o.logt_token) o.logt_token[r] = nanf_();
        if (o.logq_token) o.logq_token[r] = nanf_();
        if (o.proposal) o.proposal[r] = -1;
        if (o.token) o.token[r] = -1;
        if (o.teacher_argmax) o.teacher_argmax[r] = -1;
        if (o.target) o.target[r] = -1;
        if (o.corrected) o.corrected[r] = 0;
        if (o.row_status) o.row_status[r] = SAKI_ROW_NONFINITE;
        if (ROUTE) {
          const float l = (M != 0.0f) ? nanf_() : 0.0f;
          if (P.row_loss) P.row_loss[r] = l;
          if (P.scaled_loss) P.scaled_loss[r] = static_cast<double>(l);
        }
      }
      continue;
    }

    // The logit of the teacher mode (the loss and gradient at a correction) is
    // loaded early.
    const float s_vstar = Loader<T>::load1(srow + R.vstar);

    // Rows the interpolating start places well take the fused sweep (the
    // lambda node and a speculative final sweep in one pass), and so do rows
    // whose teacher end may be feasible (the node lambda = 1, where A is known
    // exactly); the others, and fused rows whose checks fail, the lambda
    // search and the final sweep.
    // The serial steps between sweeps run on one wave at a time: wave 0 the
    // start point while wave 1 draws the proposal z ~ p (the two-level race on
    // the stats sweep's chunk masses, then the entry race in the winning
    // chunk), which leaves the other waves' issue slots to the other
    // workgroup of the CU; the results go through LDS (plan).
    const bool end_first = R.kl1_est <= 1.05 * P.eps + 1e-5;
    if (B.wave == 0) {
      bool fu = !force_acc && P.eps > 0.0 && R.dmin != R.dmax;
      StartPoint S0;
      S0.lam = 1.0; S0.A = R.lse_t - R.lse_s - static_cast<double>(R.c); S0.herm = true;
      if (fu) {
        if (!end_first) S0 = start_point(R, P.eps);
        const double top = S0.lam * (static_cast<double>(R.dmax) - static_cast<double>(R.c));
        fu = S0.herm && top <= 56.0 && (top - S0.A) * static_cast<double>(LOG2E) <= 56.0;
      }
      if (B.lane == 0) {
        plan.S0 = S0;
        plan.fused = fu ? 1 : 0;
      }
    } else if (B.wave == 1) {
      float ws, wt;
      const int zz = wave_proposal<T>(srow, trow, nch, V, B.lane, P.seed, PROP_CHUNK, PROP_ELEM, g,
                                      [&](int c) {
                                        return static_cast<double>(sh.chunk_a[c]) * LN2_D +
                                               log(static_cast<double>(sh.chunk_b[c]));
                                      },
                                      [](float sv, float, int) { return sv; }, &ws, &wt);
      if (B.lane == 0) {
        plan.z = zz;
        plan.sz = ws;
        plan.tz = wt;
      }
    }
    __syncthreads();
    const bool fused = plan.fused != 0;

    float sz = plan.sz, tz = plan.tz;
    int z = plan.z;
    if (z >= V) {  // unreachable for finite rows: every chunk has a winner
      z = R.vstar;
      sz = s_vstar;
      tz = Loader<T>::load1(trow + z);
    }
    const double u = static_cast<double>(philox_uniform(P.seed, ACCEPT, g, 0));
    const double logp_z = static_cast<double>(sz) - R.lse_s;
    const double logt_z = static_cast<double>(tz) - R.lse_t;
    const double adv = logt_z - logp_z;
    auto coef_of = [&](bool corr) {
      return ROUTE ? static_cast<float>(static_cast<double>(P.grad_scale) * M * (corr ? 1.0 : adv)) : 0.0f;
    };
    // the gradient's indicator at a correction: the teacher mode, or a draw
    // from pi by the same two-level race on its own streams (teacher chunk
    // masses from the stats sweep); it does not depend on lambda
    int hot_c = R.vstar;
    float s_hot_c = s_vstar;
    bool have_hot_c = !sample_target;
    auto correction_target = [&]() {
      if (have_hot_c) return;
      have_hot_c = true;
      const int ct = chunk_race<NT>(B, nch, P.seed, TS_CHUNK, g, [&](int c) {
        return static_cast<double>(sh.chunk_c[c]) * LN2_D + log(static_cast<double>(sh.chunk_d[c]));
      });
      const int cc = ct < nch ? ct : 0;
      const ElemFetch<T> ft = elem_fetch<T, NT>(srow, trow, cc, V, B.tid);
      float sv, tv;
      const int vt = elem_pick<NT>(B, ft, cc, V, P.seed, TS_ELEM, g,
                                   [&](float, float tl, int) { return tl; }, &sv, &tv);
      if (vt < V) {
        hot_c = vt;
        s_hot_c = sv;
      }
    };
    auto sweep1 = [&](float lam, bool acc) { return lam_sweep<T, NT>(B, srow, trow, V, R, lam, acc); };

    LamResult L;
    FinalConst F;
    bool C;
    double TV = 0.0;
    bool tv_acc = false;   // the fused sweep's form (the final sweep's is F.acc)
    bool settled = false;  // TV, the residual chunk and the gradient row come from the fused sweep
    int res_chunk = nch;
    if (fused) {
      // accept decision at the start point: it sets the gradient the fused
      // sweep writes, and must agree with the one at lambda*
      const double xz = (static_cast<double>(LOG2E) * (static_cast<double>(tz) - static_cast<double>(sz)) -
                         static_cast<double>(R.cL)) * LN2_D;
      const bool Cg = !(u < exp(fmin(0.0, plan.S0.lam * xz - plan.S0.A)));
      if (Cg) correction_target();
      const float coef_g = coef_of(Cg);
      FusedConst FC;
      FC.msL = R.ms * LOG2E;
      FC.cL = R.cL;
      FC.lam = static_cast<float>(plan.S0.lam);
      FC.AL = static_cast<float>(plan.S0.A * static_cast<double>(LOG2E));
      const float invS = static_cast<float>(shift_correction(R.ms, FC.msL) / R.sum_s);
      FC.gsc = coef_g * invS;
      FC.set_y();
      // the expm1 form where the lambda sweep would take it (KL below
      // KL_ACCURATE: the radius, or KL(pi || p) at the teacher end) and on
      // peaked rows, whose TV the plain form would often leave too imprecise;
      // elsewhere a row whose TV turns out too small for the plain form is
      // listed for the accurate second launch (redo_accurate)
      const bool facc = (end_first ? R.kl1_est < 1.01 * KL_ACCURATE : P.eps < KL_ACCURATE) || R.pmax > P_PEAKED;
      tv_acc = facc;
      const FusedSums FS = fused_sweep_any<T, G, NT, GRAD>(B, srow, trow, grow, V, FC, facc, Cg, coef_g, invS,
                                                          Cg ? hot_c : z, Cg ? s_hot_c : sz);
      // wave 0: lambda* from the node's model when it needs no sweep, the
      // accept decision there and TV from the fused sums
      if (B.wave == 0) {
        const LamEval E0 = fused_node(R, FS, FC, end_first, facc);
        const LamResult L0 = lambda_search_with(R, P.eps, [](float, bool) { LamEval e{}; return e; }, false, 0.0f,
                                                &E0, facc, true);
        int state = -1, C0 = 0;
        FinalConst F0{};
        FusedFinal FF0{};
        if (L0.sweeps == 0) {
          F0 = final_const(R, L0, false);
          C0 = !(u < exp(fmin(0.0, L0.log_ratio(sz, tz)))) ? 1 : 0;
          FF0 = fused_tv(R, L0, F0, FC, FS, facc);
          state = (FF0.ok && (C0 != 0) == Cg) ? 1 : 0;
        }
        if (B.lane == 0) {
          plan.L = L0;
          plan.F = F0;
          plan.FF = FF0;
          plan.state = state;
          plan.C = C0;
        }
      }
      __syncthreads();
      if (plan.state < 0) {
        // the node's model did not settle lambda*: the search goes on with
        // lambda sweeps from that node
        const LamEval E0 = fused_node(R, FS, FC, end_first, facc);
        L = lambda_search_with(R, P.eps, sweep1, false, 0.0f, &E0, facc);
        F = final_const(R, L, false);
        C = !(u < exp(fmin(0.0, L.log_ratio(sz, tz))));
      } else {
        L = plan.L;
        F = plan.F;
        C = plan.C != 0;
        if (plan.state == 1) {
          TV = plan.FF.TV;
          settled = true;
          if (C) {
            // the residual chunk from the masses at the node, each within
            // (2^hmax - 1) of its positive mass plus the sign-change bound
            const double hb = expm1(plan.FF.hmax * LN2_D) * 1.02 + 2e-6;
            const double flip = plan.FF.flip;
            res_chunk = chunk_race_certain<NT>(B, nch, P.seed, RES_CHUNK, g, [&](int c, double& m, double& b) {
              m = fmax(static_cast<double>(sh.chunk_a[c]), 0.0);
              b = hb * static_cast<double>(sh.chunk_b[c]) + flip;
            });
            if (res_chunk < 0) {
              settled = false;
              res_chunk = nch;
            }
          }
        }
      }
    } else {
      L = lambda_search<T, NT>(B, srow, trow, V, R, P.eps, force_acc);
      F = final_const(R, L, force_acc);
      C = !(u < exp(fmin(0.0, L.log_ratio(sz, tz))));
    }

    // accept test, Eq. accept in the log form exp(min(0, log q(z) - log p(z)))
    const double alpha = exp(fmin(0.0, L.log_ratio(sz, tz)));
    if (C) correction_target();
    const float coef = coef_of(C);
    const int hot = C ? hot_c : z;
    const float s_hot = C ? s_hot_c : sz;

    if (!settled) {
      TV = final_sweep_any<T, G, NT, GRAD>(B, srow, trow, grow, V, F, C, coef, hot, s_hot);
      if (C) {
        res_chunk = chunk_race<NT>(B, nch, P.seed, RES_CHUNK, g, [&](int c) {
          const float m = sh.chunk_a[c];
          return m > 0.0f ? log(static_cast<double>(m)) : -__builtin_huge_val();
        });
      }
    }
    if (!force_acc && redo_accurate(R, L, settled ? tv_acc : F.acc, TV)) {
      // listed for the second launch, which rewrites the row's gradient and
      // writes its outputs
      if (B.tid == 0) P.redo_list[atomicAdd(P.redo_count, 1u)] = static_cast<unsigned int>(r);
      continue;
    }

    int y = z;
    float sy = sz, ty = tz;
    if (C) {
      // a residual that rounds to zero everywhere in float (lambda* x within
      // rounding of A*) leaves no chunk with mass; the proposal is kept then
      const int c1 = res_chunk;
      if (c1 < nch) {
        const ElemFetch<T> fr = elem_fetch<T, NT>(srow, trow, c1, V, B.tid);
        float sw, tw;
        const int yc = elem_pick<NT>(B, fr, c1, V, P.seed, RES_ELEM, g, [&](float sv, float tv, int) {
          float p;
          const float w = res_weight_any(sv, tv, F, &p);
          return w > 0.0f ? flog2(w) * LN2 : -finf();
        }, &sw, &tw);
        if (yc < V) {
          y = yc;
          sy = sw;
          ty = tw;
        }
      }
    }

    if (B.tid == 0) {
      const double logp_y = static_cast<double>(sy) - R.lse_s;
      const double logt_y = static_cast<double>(ty) - R.lse_t;
      const double logq_y = logp_y + L.log_ratio(sy, ty);
      const saki_couple_out& o = P.out;
      if (o.lambda) o.lambda[r] = L.lam;
      if (o.kl) o.kl[r] = static_cast<float>(L.KL);
      if (o.tv) o.tv[r] = static_cast<float>(TV);
      if (o.accept_prob) o.accept_prob[r] = static_cast<float>(alpha);
      if (o.margin) o.margin[r] = static_cast<float>(fabs(u - alpha));
      if (o.logp_token) o.logp_token[r] = static_cast<float>(logp_y);
      if (o.logt_token) o.logt_token[r] = static_cast<float>(logt_y);
      if (o.logq_token) o.logq_token[r] = static_cast<float>(logq_y);
      if (o.proposal) o.proposal[r] = z;
      if (o.token) o.token[r] = y;
      if (o.teacher_argmax) o.teacher_argmax[r] = R.vstar;
      if (o.target) o.target[r] = hot;
      if (o.corrected) o.corrected[r] = C ? 1 : 0;
      if (o.row_status) o.row_status[r] = SAKI_ROW_OK;
      if (ROUTE) {
        double l = 0.0;
        if (M != 0.0f) {
          if (C) {
            const double logp_v = static_cast<double>(s_hot) - R.lse_s;
            l = -logp_v;
          } else {
            l = -adv * logp_z;
          }
        }
        if (P.row_loss) P.row_loss[r] = static_cast<float>(l);
        if (P.scaled_loss) P.scaled_loss[r] = static_cast<double>(P.grad_scale) * l;
      }
    }
  }
}

}  // namespace saki

#include "probe.hpp"

namespace saki {

// ---------------------------------------------------------------------------
// Speculative verification: one workgroup per block, positions in order.
// ---------------------------------------------------------------------------
struct VerifyParams {
  const void* s;
  const void* t;
  int64_t n_blocks;
  int64_t stride;
  int64_t row_offset;
  int V;
  int k;
  const int32_t* draft;
  double eps;
  uint64_t seed;
  int eos;
  int32_t* accepted_len;
  int32_t* correction;
  saki_couple_out pp;  // per-position outputs (fields may be NULL)
  int has_pp;
  unsigned int* next_block;  // work counter in the caller's workspace, zero at launch
};

__device__ void write_skipped(const saki_couple_out& o, int64_t r, int32_t draft, uint8_t status) {
  if (o.lambda) o.lambda[r] = nanf_();
  if (o.kl) o.kl[r] = nanf_();
  if (o.tv) o.tv[r] = nanf_();
  if (o.accept_prob) o.accept_prob[r] = nanf_();
  if (o.margin) o.margin[r] = nanf_();
  if (o.logp_token) o.logp_token[r] = nanf_();
  if (o.logt_token) o.logt_token[r] = nanf_();
  if (o.logq_token) o.logq_token[r] = nanf_();
  if (o.proposal) o.proposal[r] = draft;
  if (o.token) o.token[r] = -1;
  if (o.teacher_argmax) o.teacher_argmax[r] = -1;
  if (o.target) o.target[r] = -1;
  if (o.corrected) o.corrected[r] = 0;
  if (o.row_status) o.row_status[r] = status;
}

// VNT threads per workgroup: 256 (two workgroups per CU) for large batches,
// 512 (one per CU) when a call has no more blocks than CUs, as in rollouts,
// so that each position's sweeps are spread over eight waves.
template <typename T, int KC, int VNT, bool K34>
__global__ __launch_bounds__(VNT, VNT == 256 ? 2 : 1) void verify_kernel(VerifyParams P) {
  using SH = RowShared<VNT, (KC > 0 ? CACHED_MAXC : MAX_CHUNKS), KC>;
  __shared__ SH sh;
  __shared__ RowPlan plan;
  Block<VNT, SH> B(sh);
  const int V = P.V;
  const int nch = (V + CHUNK - 1) / CHUNK;
  const saki_couple_out& o = P.pp;
  const bool need_tv = P.has_pp && o.tv != nullptr;
  // outputs that need lambda* at an accepted position
  const bool need_lam = P.has_pp && (o.lambda || o.kl || o.tv || o.accept_prob || o.margin || o.logq_token);
  // Blocks cost one to k positions, so workgroups take them from a counter
  // (dynamic scheduling) rather than with a fixed stride.  Each iteration
  // takes a new block or ends the loop, so at most n_blocks + 1 iterations run.
  __shared__ unsigned int next_b;
  for (int64_t it = 0; it <= P.n_blocks; ++it) {
    const unsigned int bu = take_next(P.next_block, &next_b);
    // unsigned: n_blocks < 2^31 and the counter stays below n_blocks + grid
    if (bu >= static_cast<unsigned int>(P.n_blocks)) break;
    const int64_t b = static_cast<int64_t>(bu);
    int n = P.k;
    int corr = -1;
    int next_unwritten = P.k;  // first position whose per-position outputs are not yet written
    // a position resolved in a plain form whose TV turns out too small for
    // that form's rounding is processed again with every sweep in the expm1
    // form (rare): force_acc is all that crosses the restart
    bool force_acc = false;
    for (int j = 0; j < P.k; ++j) {
      const int64_t r = b * P.k + j;
      const T* srow = static_cast<const T*>(P.s) + r * P.stride;
      const T* trow = static_cast<const T*>(P.t) + r * P.stride;
      const uint64_t g = static_cast<uint64_t>(P.row_offset + r);
      const int z = P.draft[r];
      if (z < 0 || z >= V) {
        if (P.has_pp && B.tid == 0) write_skipped(o, r, z, SAKI_ROW_BAD_DRAFT);
        n = j;
        next_unwritten = j + 1;
        break;
      }
      const RowStats& R = stats_sweep<T, VNT, true, K34>(B, srow, trow, V, mid_lambda(P.eps), false);
      if (!R.finite) {
        if (P.has_pp && B.tid == 0) write_skipped(o, r, z, SAKI_ROW_NONFINITE);
        n = j;
        next_unwritten = j + 1;
        break;
      }
      const float sz = Loader<T>::load1(srow + z), tz = Loader<T>::load1(trow + z);
      const double u = static_cast<double>(philox_uniform(P.seed, ACCEPT, g, 0));
      // g(lam) = lam x_z - A(lam) = log q(z) - log p(z) is concave in lam with
      // g(0) = 0, so on a bracket [la, lb] of lambda* it lies above min(g(la),
      // g(lb)): a draft with u below exp of that is accepted whatever lambda*
      // is, and when no output needs lambda* its search is skipped.  The
      // bracket is [0, 1] (g(1) = log pi(z) - log p(z)), or split at the
      // middle node by the sign of KL(lm) - eps; the middle node's values come
      // from float sums, so that bound keeps a margin of 2e-6.
      if (!need_lam) {
        const double lr1 = (static_cast<double>(tz) - R.lse_t) - (static_cast<double>(sz) - R.lse_s);
        double gmin = fmin(0.0, lr1);
        if (R.lam_mid > 0.0f) {
          const double lm = static_cast<double>(R.lam_mid);
          const double xz = static_cast<double>(tz) - static_cast<double>(sz) - static_cast<double>(R.c);
          const double gm = lm * xz - R.mid_A;
          const double klm = lm * R.mid_A1 - R.mid_A;
          // Above the middle node the bracket can end below 1, where
          // convexity alone forces KL > eps.  With A and A' known at lm and 1, the
          // tangent of A at lambda lies below A at lm, so A'(lambda) >=
          // (A(lambda) - A(lm)) / (lambda - lm), and A(lambda) lies above the
          // tangent at 1; together KL(lambda) >= (lm T1(lambda) - lambda A(lm))
          // / (lambda - lm), T1 that tangent, which passes eps at lh below.
          // On [lm, lh] g lies above lambda x_z minus the chord of A from lm
          // to 1 (A is convex), a line: its smaller end value bounds g.
          // Guards keep lh away from cancellations in the float sums.
          const double A1 = R.lse_t - R.lse_s - static_cast<double>(R.c);
          const double D1 = R.mean_pi - static_cast<double>(R.c);
          const double num = R.kl1_est - P.eps, den = lm * D1 - R.mid_A - P.eps;
          double g_hi = lr1;
          if (num > 1e-2 * (fabs(R.kl1_est) + P.eps) &&
              den > 1e-2 * (fabs(lm * D1) + fabs(R.mid_A) + P.eps)) {
            const double lh = fmax(lm, lm * num / den * (1.0 + 1e-3) + 1e-6);
            if (lh < 1.0) g_hi = lh * xz - (R.mid_A + (A1 - R.mid_A) * (lh - lm) / (1.0 - lm));
          }
          const double lo_side = fmin(0.0, gm), hi_side = fmin(gm, g_hi);
          const double gb = (klm < P.eps * (1.0 - 1e-3)) ? hi_side : (klm > P.eps * (1.0 + 1e-3)) ? lo_side
                                                                     : fmin(lo_side, hi_side);
          gmin = fmax(gmin, gb - 2e-6);
        }
        if (u < exp(gmin)) {
          if (P.has_pp && B.tid == 0) {
            if (o.logp_token) o.logp_token[r] = static_cast<float>(static_cast<double>(sz) - R.lse_s);
            if (o.logt_token) o.logt_token[r] = static_cast<float>(static_cast<double>(tz) - R.lse_t);
            if (o.proposal) o.proposal[r] = z;
            if (o.token) o.token[r] = z;
            if (o.teacher_argmax) o.teacher_argmax[r] = R.vstar;
            if (o.target) o.target[r] = z;
            if (o.corrected) o.corrected[r] = 0;
            if (o.row_status) o.row_status[r] = SAKI_ROW_OK;
          }
          if (P.eos >= 0 && z == P.eos) {
            n = j + 1;
            next_unwritten = j + 1;
            break;
          }
          continue;
        }
      }
      // Positions the interpolating start places well take the fused sweep
      // (the lambda node, and the residual chunk masses where the start
      // predicts a rejection); the others the lambda search and, when
      // rejected or when TV is asked for, the final sweep.  With one
      // workgroup per CU (rollout waves) a position's steps are not hidden
      // behind another workgroup's, and the fused sweep's serial start and
      // settling cost more than the lambda sweep they replace: every position
      // takes the search there.
      const bool end_first = R.kl1_est <= 1.05 * P.eps + 1e-5;
      if (B.wave == 0) {
        bool fu = VNT == 256 && !force_acc && P.eps > 0.0 && R.dmin != R.dmax;
        StartPoint S0;
        S0.lam = 1.0; S0.A = R.lse_t - R.lse_s - static_cast<double>(R.c); S0.herm = true;
        if (fu) {
          if (!end_first) S0 = start_point(R, P.eps);
          const double top = S0.lam * (static_cast<double>(R.dmax) - static_cast<double>(R.c));
          fu = S0.herm && top <= 56.0 && (top - S0.A) * static_cast<double>(LOG2E) <= 56.0;
        }
        if (B.lane == 0) {
          plan.S0 = S0;
          plan.fused = fu ? 1 : 0;
        }
      }
      __syncthreads();
      LamResult L;
      FinalConst F;
      double TV = __builtin_nan("");
      bool settled = false;  // lambda*, the decision, TV (if valid) and the residual chunk from the fused sweep
      bool tv_ok = false;
      bool tv_acc = false;   // the fused sweep's form (the final sweep's is F.acc)
      int res_chunk = nch;
      auto sweep1 = [&](float lam, bool acc) { return lam_sweep<T, VNT>(B, srow, trow, V, R, lam, acc); };
      if (plan.fused != 0) {
        const double xz = (static_cast<double>(LOG2E) * (static_cast<double>(tz) - static_cast<double>(sz)) -
                           static_cast<double>(R.cL)) * LN2_D;
        const bool reject_g = !(u < exp(fmin(0.0, plan.S0.lam * xz - plan.S0.A)));
        FusedConst FC;
        FC.msL = R.ms * LOG2E;
        FC.cL = R.cL;
        FC.lam = static_cast<float>(plan.S0.lam);
        FC.AL = static_cast<float>(plan.S0.A * static_cast<double>(LOG2E));
        FC.gsc = 0.0f;
        FC.set_y();
        const bool facc = (end_first ? R.kl1_est < 1.01 * KL_ACCURATE : P.eps < KL_ACCURATE) || R.pmax > P_PEAKED;
        tv_acc = facc;
        const FusedSums FS = fused_sweep_any<T, float, VNT, false>(B, srow, trow, nullptr, V, FC, facc, reject_g,
                                                                  0.0f, 0.0f, -1, 0.0f);
        if (B.wave == 0) {
          const LamEval E0 = fused_node(R, FS, FC, end_first, facc);
          const LamResult L0 = lambda_search_with(R, P.eps, [](float, bool) { LamEval e{}; return e; }, false, 0.0f,
                                                  &E0, facc, true);
          int state = -1, C0 = 0;
          FinalConst F0{};
          FusedFinal FF0{};
          if (L0.sweeps == 0) {
            F0 = final_const(R, L0, false);
            C0 = !(u < exp(fmin(0.0, L0.log_ratio(sz, tz)))) ? 1 : 0;
            FF0 = fused_tv(R, L0, F0, FC, FS, facc);
            // settled unless the decision or TV needs the final sweep: a
            // rejection needs valid residual masses (kept only where the
            // start predicted it), TV a valid correction
            const bool need_final = (C0 != 0) ? !(FF0.ok && reject_g) : (need_tv && !FF0.ok);
            state = need_final ? 0 : 1;
          }
          if (B.lane == 0) {
            plan.L = L0;
            plan.F = F0;
            plan.FF = FF0;
            plan.state = state;
            plan.C = C0;
          }
        }
        __syncthreads();
        if (plan.state < 0) {
          const LamEval E0 = fused_node(R, FS, FC, end_first, facc);
          L = lambda_search_with(R, P.eps, sweep1, false, 0.0f, &E0, facc);
          F = final_const(R, L, false);
        } else {
          L = plan.L;
          F = plan.F;
          if (plan.state == 1) {
            settled = true;
            tv_ok = plan.FF.ok;
            if (tv_ok) TV = plan.FF.TV;
            if (plan.C != 0) {
              const double hb = expm1(plan.FF.hmax * LN2_D) * 1.02 + 2e-6;
              const double flip = plan.FF.flip;
              res_chunk = chunk_race_certain<VNT>(B, nch, P.seed, RES_CHUNK, g, [&](int c, double& m, double& bb) {
                m = fmax(static_cast<double>(sh.chunk_a[c]), 0.0);
                bb = hb * static_cast<double>(sh.chunk_b[c]) + flip;
              });
              if (res_chunk < 0) {
                settled = false;
                res_chunk = nch;
              }
            }
          }
        }
      } else {
        L = lambda_search<T, VNT>(B, srow, trow, V, R, P.eps, force_acc);
        F = final_const(R, L, force_acc);
      }
      const double alpha = exp(fmin(0.0, L.log_ratio(sz, tz)));
      const bool accept = u < alpha;
      if (!settled && (need_tv || !accept)) {
        TV = final_sweep_any<T, float, VNT, false>(B, srow, trow, nullptr, V, F, !accept, 0.0f, -1, 0.0f);
        tv_ok = true;
        if (!accept) {
          res_chunk = chunk_race<VNT>(B, nch, P.seed, RES_CHUNK, g, [&](int c) {
            const float m = sh.chunk_a[c];
            return m > 0.0f ? log(static_cast<double>(m)) : -__builtin_huge_val();
          });
        }
      }
      if ((need_tv || !accept) && tv_ok && !force_acc && redo_accurate(R, L, settled ? tv_acc : F.acc, TV)) {
        force_acc = true;
        --j;
        continue;
      }
      force_acc = false;
      int y = z;
      float sy = sz, ty = tz;
      if (!accept) {
        const int c1 = res_chunk;
        if (c1 < nch) {
          const ElemFetch<T> fr = elem_fetch<T, VNT>(srow, trow, c1, V, B.tid);
          float sw, tw;
          const int yc = elem_pick<VNT>(B, fr, c1, V, P.seed, RES_ELEM, g, [&](float sv, float tv, int) {
            float p;
            const float w = res_weight_any(sv, tv, F, &p);
            return w > 0.0f ? flog2(w) * LN2 : -finf();
          }, &sw, &tw);
          if (yc < V) {
            y = yc;
            sy = sw;
            ty = tw;
          }
        }
      }
      if (P.has_pp && B.tid == 0) {
        const double logp_y = static_cast<double>(sy) - R.lse_s;
        const double logt_y = static_cast<double>(ty) - R.lse_t;
        if (o.lambda) o.lambda[r] = L.lam;
        if (o.kl) o.kl[r] = static_cast<float>(L.KL);
        if (o.tv) o.tv[r] = static_cast<float>(TV);
        if (o.accept_prob) o.accept_prob[r] = static_cast<float>(alpha);
        if (o.margin) o.margin[r] = static_cast<float>(fabs(u - alpha));
        if (o.logp_token) o.logp_token[r] = static_cast<float>(logp_y);
        if (o.logt_token) o.logt_token[r] = static_cast<float>(logt_y);
        if (o.logq_token) o.logq_token[r] = static_cast<float>(logp_y + L.log_ratio(sy, ty));
        if (o.proposal) o.proposal[r] = z;
        if (o.token) o.token[r] = y;
        if (o.teacher_argmax) o.teacher_argmax[r] = R.vstar;
        if (o.target) o.target[r] = accept ? z : R.vstar;
        if (o.corrected) o.corrected[r] = accept ? 0 : 1;
        if (o.row_status) o.row_status[r] = SAKI_ROW_OK;
      }
      if (!accept) {
        n = j;
        corr = y;
        next_unwritten = j + 1;
        break;
      }
      if (P.eos >= 0 && z == P.eos) {
        n = j + 1;
        next_unwritten = j + 1;
        break;
      }
    }
    if (B.tid == 0) {
      P.accepted_len[b] = n;
      P.correction[b] = corr;
      if (P.has_pp) {
        // positions after the end of the block's committed prefix
        for (int jj = next_unwritten; jj < P.k; ++jj) {
          const int64_t r = b * P.k + jj;
          write_skipped(o, r, P.draft[r], SAKI_ROW_SKIPPED);
        }
      }
    }
  }
}

#include "rollout.hpp"

// ---------------------------------------------------------------------------
// Standalone routed loss and gradient from given events.
// ---------------------------------------------------------------------------
struct RouteParams {
  const void* s;
  int64_t n_rows;
  int64_t stride;
  int V;
  const int32_t* token;
  const uint8_t* corrected;
  const int32_t* vstar;
  const float* advantage;
  const uint8_t* valid;
  float grad_scale;
  float* row_loss;
  double* scaled_loss;
  void* grad;
  int64_t grad_stride;
  unsigned int* next_row;  // work counter in the caller's workspace, zero at launch
};

// Shared state of the standalone routed loss: the block reductions and, for
// bf16 rows, a row cache of KC chunks of s per wave (the log-sum-exp sweep
// stores the wave's last KC full chunks, the gradient sweep reads them).
template <int NT_, int KC>
struct RouteShared {
  static constexpr int NW = NT_ / WAVE;
  static constexpr int CACHE_CHUNKS = KC;
  double red_d[NW][RED_MAX];
  float red_f[NW][4];
  int red_i[NW][4];
  uint4 cache[KC > 0 ? NW * KC * 2 * WAVE : 1];  // [wave][slot][half][lane]
};
// 9 chunks per wave: 72 KiB, two workgroups per CU
constexpr int ROUTE_KC = 9;

// Standalone routed loss: two sweeps over s per row (log-sum-exp, then the
// gradient), the loss from the logit of the supervised entry.  Workgroups take
// rows from a counter, as in the coupling kernel.
template <typename T, typename G, bool GRAD>
__global__ __launch_bounds__(NT, WG_PER_CU) void route_kernel(RouteParams P) {
  using SH = RouteShared<NT, (sizeof(T) == 2 ? ROUTE_KC : 0)>;
  __shared__ SH sh;
  Block<NT, SH> B(sh);
  const int V = P.V;
  __shared__ unsigned int next_r;
  for (int64_t it = 0; it <= P.n_rows; ++it) {
    const unsigned int ru = take_next(P.next_row, &next_r);
    // unsigned: n_rows < 2^31 and the counter stays below n_rows + grid
    if (ru >= static_cast<unsigned int>(P.n_rows)) break;
    const int64_t r = static_cast<int64_t>(ru);
    const T* srow = static_cast<const T*>(P.s) + r * P.stride;
    G* grow = GRAD ? static_cast<G*>(P.grad) + r * P.grad_stride : nullptr;
    const bool M = P.valid ? (P.valid[r] != 0) : true;
    const bool C = P.corrected[r] != 0;
    const int hot = C ? P.vstar[r] : P.token[r];
    const bool hot_ok = hot >= 0 && hot < V;
    // the supervised entry's logit, loaded before the sweeps
    const float s_hot = hot_ok ? Loader<T>::load1(srow + hot) : 0.0f;
    float msL;
    const double S = lse_sweep<T, NT>(B, srow, V, &msL);
    const double lse = static_cast<double>(msL) * LN2_D + log(S);
    const bool bad = M && (!hot_ok || !isfinite(lse));
    const double A = C ? 0.0 : static_cast<double>(P.advantage[r]);
    float coef = 0.0f;
    if (M && !bad) coef = static_cast<float>(static_cast<double>(P.grad_scale) * (C ? 1.0 : A));
    if (GRAD)
      route_grad_sweep<T, G, NT>(B, srow, grow, V, msL, static_cast<float>(1.0 / S), coef, hot_ok ? hot : -1,
                                 s_hot, bad);
    if (B.tid == 0) {
      double l = 0.0;
      if (bad) {
        l = __builtin_nan("");
      } else if (M) {
        const double logp_h = static_cast<double>(s_hot) - lse;
        l = C ? -logp_h : -A * logp_h;
      }
      if (P.row_loss) P.row_loss[r] = static_cast<float>(l);
      if (P.scaled_loss) P.scaled_loss[r] = static_cast<double>(P.grad_scale) * l;
    }
  }
}

// Deterministic sum of the scaled row losses: fixed per-thread strides, then a
// fixed-order block tree.
__global__ __launch_bounds__(1024) void loss_sum_kernel(const double* x, int64_t n, double* out) {
  __shared__ double part[1024];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 1024) acc += x[i];
  part[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if (static_cast<int>(threadIdx.x) < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = part[0];
}


// ---------------------------------------------------------------------------
// Placement controls (Random-TM, TV-Weighted-TM): per trajectory, select
// m = corrections among the valid positions.  Keys in double: ln E with
// E = -ln U (Random-TM, and the uniform fill of TV-Weighted-TM from the
// positions with TV = 0), ln E - ln TV for the positions with TV > 0.  The k
// smallest keys of a tier are found exactly: bisection over the keys'
// order-preserving 64-bit images gives the k-th smallest, ties to the lower row.
// ---------------------------------------------------------------------------
constexpr int SNT = 256;

struct SelectParams {
  int mode;
  int64_t n_traj;
  int64_t n_rows;
  const int64_t* off;
  const float* tv;
  const uint8_t* corrected;
  const uint8_t* valid;
  uint64_t seed;
  int64_t row_offset;
  uint8_t* sel;   // holds each row's tier (0, 1; 2 = not valid) until the end
  double* keys;   // workspace [n_rows]
};

struct SelShared {
  double red_d[SNT / WAVE][RED_MAX];
  float red_f[SNT / WAVE][4];
  int red_i[SNT / WAVE][4];
  int scan[SNT];
};

__device__ __forceinline__ uint64_t order_bits(double k) {
  const uint64_t u = __builtin_bit_cast(uint64_t, k);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Number of rows of tier `tier` in [a, b) whose key image is <= x (or < x).
__device__ __forceinline__ double count_le(const SelectParams& P, int64_t a, int64_t b, int tier,
                                           uint64_t x, bool strict) {
  double n = 0;
  for (int64_t r = a; r < b; ++r) {
    if (P.sel[r] != tier) continue;
    const uint64_t o = order_bits(P.keys[r]);
    n += strict ? (o < x) : (o <= x);
  }
  return n;
}

// Marks (sel = 3) the k smallest rows of `tier` in the trajectory; thread j
// owns rows [a, b), contiguous and in order across threads.
__device__ void select_smallest(Block<SNT, SelShared>& B, const SelectParams& P, int64_t a, int64_t b,
                                int tier, double k) {
  uint64_t lo = 0, hi = ~0ull;
  while (lo < hi) {
    const uint64_t mid = lo + (hi - lo) / 2;
    double v[1] = {count_le(P, a, b, tier, mid, false)};
    B.sum(v);
    if (v[0] >= k) hi = mid; else lo = mid + 1;
  }
  const uint64_t T = lo;
  double v[1] = {count_le(P, a, b, tier, T, true)};
  B.sum(v);
  const int need = static_cast<int>(k - v[0]);  // rows with key image T to take, lowest rows first
  int eq = 0;
  for (int64_t r = a; r < b; ++r) eq += (P.sel[r] == tier && order_bits(P.keys[r]) == T);
  B.sh.scan[B.tid] = eq;
  __syncthreads();
  int before = 0;
  for (int j = 0; j < B.tid; ++j) before += B.sh.scan[j];
  __syncthreads();
  for (int64_t r = a; r < b; ++r) {
    if (P.sel[r] != tier) continue;
    const uint64_t o = order_bits(P.keys[r]);
    if (o < T || (o == T && before++ < need)) P.sel[r] = 3;
  }
  __syncthreads();
}

__global__ __launch_bounds__(SNT) void select_kernel(SelectParams P) {
  __shared__ SelShared sh;
  Block<SNT, SelShared> B(sh);
  for (int64_t i = blockIdx.x; i < P.n_traj; i += gridDim.x) {
    const int64_t lo = P.off[i], hi = P.off[i + 1];
    if (lo < 0 || hi < lo || hi > P.n_rows) continue;  // malformed range: rows left unwritten
    const int64_t per = (hi - lo + SNT - 1) / SNT;
    const int64_t a = min(hi, lo + B.tid * per), b = min(hi, a + per);
    double cnt[2] = {0, 0};  // corrections among valid rows, rows of tier 0
    for (int64_t r = a; r < b; ++r) {
      const bool M = P.valid ? (P.valid[r] != 0) : true;
      uint8_t tier = 2;
      double key = __builtin_huge_val();
      if (M) {
        const double u = static_cast<double>(philox_uniform(P.seed, SELECT, static_cast<uint64_t>(P.row_offset + r), 0));
        const double lE = log(-log(u));
        const double d = static_cast<double>(P.tv[r]);
        if (P.mode == SAKI_SELECT_RANDOM) {
          tier = 0; key = lE;
        } else if (d > 0.0) {
          tier = 0; key = lE - log(d);
        } else {
          tier = 1; key = lE;
        }
        cnt[0] += (P.corrected[r] != 0);
        cnt[1] += (tier == 0);
      }
      P.keys[r] = key;
      P.sel[r] = tier;
    }
    __syncthreads();
    B.sum(cnt);
    const double m = cnt[0], n0 = cnt[1];
    if (m > 0) {
      if (m <= n0) {
        select_smallest(B, P, a, b, 0, m);
      } else {
        for (int64_t r = a; r < b; ++r)
          if (P.sel[r] == 0) P.sel[r] = 3;
        __syncthreads();
        select_smallest(B, P, a, b, 1, m - n0);
      }
    }
    for (int64_t r = a; r < b; ++r) P.sel[r] = (P.sel[r] == 3) ? 1 : 0;
    __syncthreads();
  }
}

}  // namespace saki

// ===========================================================================
// C ABI
// ===========================================================================
namespace {

thread_local std::string g_last_error;

saki_status fail(saki_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

saki_status ok() {
  g_last_error.clear();
  return SAKI_OK;
}

int elem_size(int32_t dt) { return dt == SAKI_BF16 ? 2 : 4; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

saki_status device_cus(int* cus) {
  static std::mutex mu;
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return fail(SAKI_E_DEVICE, "hipGetDevice failed");
  std::lock_guard<std::mutex> lock(mu);
  if (dev < 64 && cache[dev] > 0) {
    *cus = cache[dev];
    return SAKI_OK;
  }
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    return fail(SAKI_E_DEVICE, "hipDeviceGetAttribute(MultiprocessorCount) failed");
  if (dev < 64) cache[dev] = n;
  *cus = n;
  return SAKI_OK;
}

saki_status check_rows(const saki_rows* in, bool need_teacher = true) {
  if (!in) return fail(SAKI_E_NULLPTR, "rows descriptor is NULL");
  if (in->dtype != SAKI_F32 && in->dtype != SAKI_BF16) return fail(SAKI_E_DTYPE, "unknown logits dtype");
  if (in->reserved != 0) return fail(SAKI_E_VALUE, "saki_rows.reserved must be 0");
  if (in->n_rows < 0) return fail(SAKI_E_SHAPE, "n_rows < 0");
  if (in->vocab < 1 || in->vocab > SAKI_MAX_VOCAB) return fail(SAKI_E_SHAPE, "vocab outside [1, SAKI_MAX_VOCAB]");
  if (in->row_stride < in->vocab) return fail(SAKI_E_SHAPE, "row_stride < vocab");
  if (in->row_offset < 0) return fail(SAKI_E_VALUE, "row_offset < 0");
  if (in->n_rows == 0) return SAKI_OK;
  if (!in->student || (need_teacher && !in->teacher))
    return fail(SAKI_E_NULLPTR, "student or teacher pointer is NULL");
  if (!aligned16(in->student) || (need_teacher && !aligned16(in->teacher)) ||
      (in->row_stride * elem_size(in->dtype)) % 16 != 0)
    return fail(SAKI_E_ALIGN, "logit base pointers and row pitch must be 16-byte aligned");
  return SAKI_OK;
}

saki_status check_route(const saki_route_args* rt, int64_t vocab, bool* want_loss_sum) {
  *want_loss_sum = false;
  if (!rt) return SAKI_OK;
  if (!isfinite(rt->grad_scale)) return fail(SAKI_E_VALUE, "grad_scale is not finite");
  if (rt->correction_target != SAKI_TARGET_MODE && rt->correction_target != SAKI_TARGET_SAMPLE)
    return fail(SAKI_E_VALUE, "unknown correction_target");
  if (rt->grad) {
    if (rt->grad_dtype != SAKI_F32 && rt->grad_dtype != SAKI_BF16) return fail(SAKI_E_DTYPE, "unknown grad dtype");
    if (rt->grad_stride < vocab) return fail(SAKI_E_SHAPE, "grad_stride < vocab");
    if (!aligned16(rt->grad) || (rt->grad_stride * elem_size(rt->grad_dtype)) % 16 != 0)
      return fail(SAKI_E_ALIGN, "grad base pointer and row pitch must be 16-byte aligned");
  }
  *want_loss_sum = rt->loss_sum != nullptr;
  return SAKI_OK;
}

size_t loss_ws_bytes(int64_t n_rows) {
  const size_t b = static_cast<size_t>(n_rows) * sizeof(double);
  return (b + 255) & ~static_cast<size_t>(255);
}

size_t list_ws_bytes(int64_t n_rows) {
  const size_t b = static_cast<size_t>(n_rows) * sizeof(unsigned int);
  return (b + 255) & ~static_cast<size_t>(255);
}

saki_status launched(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(SAKI_E_LAUNCH, std::string(what) + ": " + hipGetErrorString(e));
  return SAKI_OK;
}

template <bool K34>
void launch_verify(const saki::VerifyParams& P, int cus, int grid, bool cached, bool bf16, hipStream_t hs) {
  if (P.n_blocks <= cus) {
    // no more blocks than CUs: one 512-thread workgroup per block
    const dim3 g1(static_cast<unsigned>(P.n_blocks)), b1(512);
    if (cached)
      hipLaunchKernelGGL((saki::verify_kernel<uint16_t, saki::CACHE_KC, 512, K34>), g1, b1, 0, hs, P);
    else if (bf16)
      hipLaunchKernelGGL((saki::verify_kernel<uint16_t, 0, 512, K34>), g1, b1, 0, hs, P);
    else
      hipLaunchKernelGGL((saki::verify_kernel<float, 0, 512, K34>), g1, b1, 0, hs, P);
  } else if (cached) {
    hipLaunchKernelGGL((saki::verify_kernel<uint16_t, saki::CACHE_KC, 256, K34>), dim3(grid), dim3(256), 0, hs, P);
  } else if (bf16) {
    hipLaunchKernelGGL((saki::verify_kernel<uint16_t, 0, 256, K34>), dim3(grid), dim3(256), 0, hs, P);
  } else {
    hipLaunchKernelGGL((saki::verify_kernel<float, 0, 256, K34>), dim3(grid), dim3(256), 0, hs, P);
  }
}

template <typename T, typename G, bool ROUTE, bool GRAD, bool K34>
saki_status launch_couple_k(const saki::CoupleParams& P, int grid, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    if ((P.V + saki::CHUNK - 1) / saki::CHUNK <= saki::CACHED_MAXC) {
      hipLaunchKernelGGL((saki::couple_kernel<T, G, ROUTE, GRAD, saki::CACHE_KC, K34>), dim3(grid), dim3(saki::NT), 0,
                         st, P);
      return launched("couple_kernel");
    }
  }
  hipLaunchKernelGGL((saki::couple_kernel<T, G, ROUTE, GRAD, 0, K34>), dim3(grid), dim3(saki::NT), 0, st, P);
  return launched("couple_kernel");
}

template <typename T, typename G, bool ROUTE, bool GRAD>
saki_status launch_couple(const saki::CoupleParams& P, int grid, hipStream_t st) {
  return saki::use_k34(P.eps) ? launch_couple_k<T, G, ROUTE, GRAD, true>(P, grid, st)
                              : launch_couple_k<T, G, ROUTE, GRAD, false>(P, grid, st);
}

template <typename T>
saki_status dispatch_couple(const saki::CoupleParams& P, bool route, bool grad, int32_t gdt, int grid,
                            hipStream_t st) {
  if (!route) return launch_couple<T, float, false, false>(P, grid, st);
  if (!grad) return launch_couple<T, float, true, false>(P, grid, st);
  if (gdt == SAKI_BF16) return launch_couple<T, uint16_t, true, true>(P, grid, st);
  return launch_couple<T, float, true, true>(P, grid, st);
}

template <typename T, typename G, bool GRAD>
saki_status launch_route(const saki::RouteParams& P, int grid, hipStream_t st) {
  hipLaunchKernelGGL((saki::route_kernel<T, G, GRAD>), dim3(grid), dim3(saki::NT), 0, st, P);
  return launched("route_kernel");
}

}  // namespace

extern "C" {

size_t saki_workspace_bytes(int op, int64_t n_rows, int64_t vocab) {
  (void)vocab;
  if (n_rows <= 0) return 0;
  switch (op) {
    case SAKI_OP_COUPLE:
      // the counters, the scaled row losses, the list of rows for the
      // second (expm1-form) launch
      return 256 + loss_ws_bytes(n_rows) + list_ws_bytes(n_rows);
    case SAKI_OP_ROUTE:
      return 256 + loss_ws_bytes(n_rows);  // the row counter, then the scaled row losses
    case SAKI_OP_VERIFY:
      return 256;  // the work counter
    case SAKI_OP_SELECT:
      return loss_ws_bytes(n_rows);
    default:
      return 0;
  }
}

}  // extern "C"

// The library's own scratch for saki_couple_static: the work counters (256
// bytes), one double per row for the scaled row losses, one index per row for
// the list of rows the second launch processes in the expm1 forms.  Each GPU the
// library runs on holds its own copy until the process ends.  In host code
// `scratch` names a host-side stand-in, not the device array: only the
// address from hipGetSymbolAddress (static_scratch) is passed to kernels.
static __device__ __align__(256) unsigned char scratch[256 + SAKI_STATIC_MAX_ROWS * (sizeof(double) + sizeof(unsigned int))];

namespace {

constexpr size_t STATIC_SCRATCH_BYTES =
    256 + static_cast<size_t>(SAKI_STATIC_MAX_ROWS) * (sizeof(double) + sizeof(unsigned int));

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
saki_status static_scratch(void** ptr) {
  static std::mutex mu;
  static void* cache[64] = {nullptr};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return fail(SAKI_E_DEVICE, "hipGetDevice failed");
  if (dev >= 64) return fail(SAKI_E_DEVICE, "device index above 63");
  std::lock_guard<std::mutex> lock(mu);
  if (cache[dev] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(SAKI_E_DEVICE, std::string("hipGetSymbolAddress(scratch) failed: ") + hipGetErrorString(e));
    cache[dev] = p;
  }
  *ptr = cache[dev];
  return SAKI_OK;
}

// use_static: the workspace is the static scratch (ws and ws_bytes unused),
// looked up after every argument check.
saki_status couple_impl(const saki_rows* in, double eps, uint64_t seed, const saki_couple_out* out,
                        const saki_route_args* route, void* ws, size_t ws_bytes, saki_stream_t stream,
                        bool use_static);

}  // namespace

extern "C" {

saki_status saki_couple(const saki_rows* in, double eps, uint64_t seed, const saki_couple_out* out,
                        const saki_route_args* route, void* ws, size_t ws_bytes, saki_stream_t stream) {
  return couple_impl(in, eps, seed, out, route, ws, ws_bytes, stream, false);
}

saki_status saki_couple_static(const saki_rows* in, double eps, uint64_t seed, const saki_couple_out* out,
                               const saki_route_args* route, saki_stream_t stream) {
  return couple_impl(in, eps, seed, out, route, nullptr, 0, stream, true);
}

}  // extern "C"

namespace {

saki_status couple_impl(const saki_rows* in, double eps, uint64_t seed, const saki_couple_out* out,
                        const saki_route_args* route, void* ws, size_t ws_bytes, saki_stream_t stream,
                        bool use_static) {
  saki_status st = check_rows(in);
  if (st != SAKI_OK) return st;
  if (!out) return fail(SAKI_E_NULLPTR, "out is NULL");
  if (!(eps >= 0.0) || !isfinite(eps)) return fail(SAKI_E_VALUE, "eps must be finite and >= 0");
  bool want_sum = false;
  st = check_route(route, in->vocab, &want_sum);
  if (st != SAKI_OK) return st;
  if (use_static && in->n_rows > SAKI_STATIC_MAX_ROWS)
    return fail(SAKI_E_SHAPE, "n_rows above SAKI_STATIC_MAX_ROWS (the static scratch holds one double per row)");
  if (in->n_rows == 0) return ok();
  if (in->n_rows >= (int64_t{1} << 31)) return fail(SAKI_E_SHAPE, "more than 2^31 - 1 rows in one call");
  if (use_static) {
    st = static_scratch(&ws);
    if (st != SAKI_OK) return st;
    ws_bytes = STATIC_SCRATCH_BYTES;
  }
  if (!ws) return fail(SAKI_E_WORKSPACE, "workspace is NULL");
  if (ws_bytes < saki_workspace_bytes(SAKI_OP_COUPLE, in->n_rows, in->vocab))
    return fail(SAKI_E_WORKSPACE, "workspace smaller than saki_workspace_bytes(SAKI_OP_COUPLE)");
  if ((reinterpret_cast<uintptr_t>(ws) & 7u) != 0) return fail(SAKI_E_ALIGN, "workspace must be 8-byte aligned");
  double* const row_losses = reinterpret_cast<double*>(static_cast<char*>(ws) + 256);
  int cus = 0;
  st = device_cus(&cus);
  if (st != SAKI_OK) return st;
  saki::CoupleParams P{};
  P.s = in->student;
  P.t = in->teacher;
  P.n_rows = in->n_rows;
  P.stride = in->row_stride;
  P.row_offset = in->row_offset;
  P.V = static_cast<int>(in->vocab);
  P.eps = eps;
  P.seed = seed;
  P.out = *out;
  if (route) {
    P.valid = route->valid_mask;
    P.grad_scale = route->grad_scale;
    P.row_loss = route->row_loss;
    P.scaled_loss = want_sum ? row_losses : nullptr;
    P.grad = route->grad;
    P.grad_stride = route->grad_stride;
    P.target_mode = route->correction_target;
  }
  // workspace: [0] row counter, [1] second launch's row counter, [2] listed
  // rows; then the scaled row losses; then the list
  unsigned int* const counters = static_cast<unsigned int*>(ws);
  P.next_row = counters;
  P.redo_count = counters + 2;
  P.redo_list = reinterpret_cast<unsigned int*>(static_cast<char*>(ws) + 256 + loss_ws_bytes(in->n_rows));
  P.redo_pass = 0;
  const int grid = static_cast<int>(std::min<int64_t>(in->n_rows, static_cast<int64_t>(cus) * saki::WG_PER_CU));
  hipStream_t hs = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(saki::clear_counter_kernel, dim3(1), dim3(64), 0, hs, counters);
  st = launched("clear_counter_kernel");
  if (st != SAKI_OK) return st;
  const bool grad = route && route->grad;
  for (int pass = 0; pass < 2; ++pass) {
    // the second launch: the listed rows, every sweep in the expm1 form
    if (pass == 1) {
      P.redo_pass = 1;
      P.next_row = counters + 1;
    }
    st = (in->dtype == SAKI_BF16)
             ? dispatch_couple<uint16_t>(P, route != nullptr, grad, route ? route->grad_dtype : 0, grid, hs)
             : dispatch_couple<float>(P, route != nullptr, grad, route ? route->grad_dtype : 0, grid, hs);
    if (st != SAKI_OK) return st;
  }
  if (want_sum) {
    hipLaunchKernelGGL(saki::loss_sum_kernel, dim3(1), dim3(1024), 0, hs,
                       static_cast<const double*>(row_losses), in->n_rows, route->loss_sum);
    st = launched("loss_sum_kernel");
    if (st != SAKI_OK) return st;
  }
  return ok();
}

}  // namespace

extern "C" {

saki_status saki_route_loss(const void* student, int32_t dtype, int64_t n_rows, int64_t vocab,
                            int64_t row_stride, const int32_t* token, const uint8_t* corrected,
                            const int32_t* teacher_argmax, const float* advantage,
                            const saki_route_args* route, void* ws, size_t ws_bytes,
                            saki_stream_t stream) {
  if (dtype != SAKI_F32 && dtype != SAKI_BF16) return fail(SAKI_E_DTYPE, "unknown logits dtype");
  if (n_rows < 0) return fail(SAKI_E_SHAPE, "n_rows < 0");
  if (vocab < 1 || vocab > SAKI_MAX_VOCAB) return fail(SAKI_E_SHAPE, "vocab outside [1, SAKI_MAX_VOCAB]");
  if (row_stride < vocab) return fail(SAKI_E_SHAPE, "row_stride < vocab");
  if (!route) return fail(SAKI_E_NULLPTR, "route is NULL");
  bool want_sum = false;
  saki_status st = check_route(route, vocab, &want_sum);
  if (st != SAKI_OK) return st;
  if (n_rows >= (int64_t{1} << 31)) return fail(SAKI_E_SHAPE, "more than 2^31 - 1 rows in one call");
  if (n_rows == 0) return ok();
  if (!student || !token || !corrected || !teacher_argmax || !advantage)
    return fail(SAKI_E_NULLPTR, "student, token, corrected, teacher_argmax and advantage are required");
  if (!ws) return fail(SAKI_E_WORKSPACE, "workspace is NULL");
  if (ws_bytes < saki_workspace_bytes(SAKI_OP_ROUTE, n_rows, vocab)) return fail(SAKI_E_WORKSPACE, "workspace too small");
  if ((reinterpret_cast<uintptr_t>(ws) & 7u) != 0) return fail(SAKI_E_ALIGN, "workspace must be 8-byte aligned");
  double* row_losses = reinterpret_cast<double*>(static_cast<char*>(ws) + 256);
  if (!aligned16(student) || (row_stride * elem_size(dtype)) % 16 != 0)
    return fail(SAKI_E_ALIGN, "student base pointer and row pitch must be 16-byte aligned");
  int cus = 0;
  st = device_cus(&cus);
  if (st != SAKI_OK) return st;
  saki::RouteParams P{};
  P.s = student;
  P.n_rows = n_rows;
  P.stride = row_stride;
  P.V = static_cast<int>(vocab);
  P.token = token;
  P.corrected = corrected;
  P.vstar = teacher_argmax;
  P.advantage = advantage;
  P.valid = route->valid_mask;
  P.grad_scale = route->grad_scale;
  P.row_loss = route->row_loss;
  P.scaled_loss = want_sum ? row_losses : nullptr;
  P.grad = route->grad;
  P.grad_stride = route->grad_stride;
  P.next_row = static_cast<unsigned int*>(ws);
  const int grid = static_cast<int>(std::min<int64_t>(n_rows, static_cast<int64_t>(cus) * saki::WG_PER_CU));
  hipStream_t hs = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(saki::clear_counter_kernel, dim3(1), dim3(64), 0, hs, P.next_row);
  st = launched("clear_counter_kernel");
  if (st != SAKI_OK) return st;
  const bool grad = route->grad != nullptr;
  const bool gbf = route->grad_dtype == SAKI_BF16;
  if (dtype == SAKI_BF16) {
    st = !grad ? launch_route<uint16_t, float, false>(P, grid, hs)
         : gbf ? launch_route<uint16_t, uint16_t, true>(P, grid, hs)
               : launch_route<uint16_t, float, true>(P, grid, hs);
  } else {
    st = !grad ? launch_route<float, float, false>(P, grid, hs)
         : gbf ? launch_route<float, uint16_t, true>(P, grid, hs)
               : launch_route<float, float, true>(P, grid, hs);
  }
  if (st != SAKI_OK) return st;
  if (want_sum) {
    hipLaunchKernelGGL(saki::loss_sum_kernel, dim3(1), dim3(1024), 0, hs, row_losses, n_rows,
                       route->loss_sum);
    st = launched("loss_sum_kernel");
    if (st != SAKI_OK) return st;
  }
  return ok();
}

saki_status saki_spec_verify(const saki_rows* in, int32_t k, const int32_t* draft, double eps,
                             uint64_t seed, int32_t eos_id, int32_t* accepted_len,
                             int32_t* correction, const saki_couple_out* per_pos, void* ws,
                             size_t ws_bytes, saki_stream_t stream) {
  saki_status st = check_rows(in);
  if (st != SAKI_OK) return st;
  if (k < 1 || k > SAKI_MAX_BLOCK_K) return fail(SAKI_E_SHAPE, "k outside [1, SAKI_MAX_BLOCK_K]");
  if (in->n_rows % k != 0) return fail(SAKI_E_SHAPE, "n_rows is not a multiple of k");
  if (!(eps >= 0.0) || !isfinite(eps)) return fail(SAKI_E_VALUE, "eps must be finite and >= 0");
  if (in->n_rows == 0) return ok();
  if (!draft || !accepted_len || !correction)
    return fail(SAKI_E_NULLPTR, "draft, accepted_len and correction are required");
  if (in->n_rows / k >= (int64_t{1} << 31)) return fail(SAKI_E_SHAPE, "more than 2^31 - 1 blocks");
  if (!ws || ws_bytes < saki_workspace_bytes(SAKI_OP_VERIFY, in->n_rows, in->vocab))
    return fail(SAKI_E_WORKSPACE, "workspace NULL or smaller than saki_workspace_bytes(SAKI_OP_VERIFY)");
  if ((reinterpret_cast<uintptr_t>(ws) & 3u) != 0) return fail(SAKI_E_ALIGN, "workspace must be 4-byte aligned");
  int cus = 0;
  st = device_cus(&cus);
  if (st != SAKI_OK) return st;
  saki::VerifyParams P{};
  P.s = in->student;
  P.t = in->teacher;
  P.n_blocks = in->n_rows / k;
  P.stride = in->row_stride;
  P.row_offset = in->row_offset;
  P.V = static_cast<int>(in->vocab);
  P.k = k;
  P.draft = draft;
  P.eps = eps;
  P.seed = seed;
  P.eos = eos_id;
  P.accepted_len = accepted_len;
  P.correction = correction;
  if (per_pos) {
    P.pp = *per_pos;
    P.has_pp = 1;
  }
  P.next_block = static_cast<unsigned int*>(ws);
  const int grid = static_cast<int>(std::min<int64_t>(P.n_blocks, static_cast<int64_t>(cus) * saki::WG_PER_CU));
  hipStream_t hs = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(saki::clear_counter_kernel, dim3(1), dim3(64), 0, hs, P.next_block);
  st = launched("clear_counter_kernel");
  if (st != SAKI_OK) return st;
  const bool cached = in->dtype == SAKI_BF16 && (P.V + saki::CHUNK - 1) / saki::CHUNK <= saki::CACHED_MAXC;
  if (saki::use_k34(P.eps))
    launch_verify<true>(P, cus, grid, cached, in->dtype == SAKI_BF16, hs);
  else
    launch_verify<false>(P, cus, grid, cached, in->dtype == SAKI_BF16, hs);
  st = launched("verify_kernel");
  if (st != SAKI_OK) return st;
  return ok();
}

saki_status saki_sample(const saki_rows* in, int64_t row_step, uint64_t seed, int32_t* token,
                        uint8_t* row_status, saki_stream_t stream) {
  saki_status st = check_rows(in, false);
  if (st != SAKI_OK) return st;
  if (row_step < 1) return fail(SAKI_E_VALUE, "row_step < 1");
  if (in->n_rows > 0 && (in->n_rows - 1) > (INT64_MAX - in->row_offset) / row_step)
    return fail(SAKI_E_VALUE, "row_offset + (n_rows - 1) * row_step overflows");
  if (in->n_rows == 0) return ok();
  if (!token) return fail(SAKI_E_NULLPTR, "token is required");
  int cus = 0;
  st = device_cus(&cus);
  if (st != SAKI_OK) return st;
  saki::SampleParams P{};
  P.s = in->student;
  P.n_rows = in->n_rows;
  P.stride = in->row_stride;
  P.row_offset = in->row_offset;
  P.row_step = row_step;
  P.V = static_cast<int>(in->vocab);
  P.seed = seed;
  P.token = token;
  P.status = row_status;
  const int grid = static_cast<int>(std::min<int64_t>(P.n_rows, static_cast<int64_t>(cus)));
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (in->dtype == SAKI_BF16)
    hipLaunchKernelGGL(saki::sample_kernel<uint16_t>, dim3(grid), dim3(saki::SAMPLE_NT), 0, hs, P);
  else
    hipLaunchKernelGGL(saki::sample_kernel<float>, dim3(grid), dim3(saki::SAMPLE_NT), 0, hs, P);
  st = launched("sample_kernel");
  if (st != SAKI_OK) return st;
  return ok();
}

saki_status saki_commit(const saki_traj* traj, int32_t k, int32_t eos_id,
                        const int32_t* accepted_len, const int32_t* correction,
                        const saki_couple_out* per_pos, int32_t* n_commit, saki_stream_t stream) {
  if (!traj) return fail(SAKI_E_NULLPTR, "trajectory descriptor is NULL");
  if (k < 1 || k > SAKI_MAX_BLOCK_K) return fail(SAKI_E_SHAPE, "k outside [1, SAKI_MAX_BLOCK_K]");
  if (traj->n_seq < 0) return fail(SAKI_E_SHAPE, "n_seq < 0");
  if (traj->max_len < 0 || traj->max_len > INT32_MAX) return fail(SAKI_E_SHAPE, "max_len outside [0, 2^31 - 1]");
  if (traj->n_seq == 0) return ok();
  if (!traj->tokens || !traj->length || !traj->done)
    return fail(SAKI_E_NULLPTR, "tokens, length and done are required");
  if (!accepted_len || !correction || !per_pos || !per_pos->token)
    return fail(SAKI_E_NULLPTR, "accepted_len, correction and per_pos->token are required");
  saki::CommitParams P{};
  P.tr = *traj;
  P.k = k;
  P.eos = eos_id;
  P.accepted_len = accepted_len;
  P.correction = correction;
  P.pp = *per_pos;
  P.n_commit = n_commit;
  const int64_t grid = (traj->n_seq + 255) / 256;
  if (grid > INT32_MAX) return fail(SAKI_E_SHAPE, "n_seq too large");
  hipLaunchKernelGGL(saki::commit_kernel, dim3(static_cast<unsigned>(grid)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), P);
  saki_status st = launched("commit_kernel");
  if (st != SAKI_OK) return st;
  return ok();
}

saki_status saki_probe_metrics(const saki_rows* in, int32_t k, float* c1, float* ck, float* kl_ts,
                               float* entropy, int32_t* topk, uint8_t* row_status,
                               saki_stream_t stream) {
  saki_status st = check_rows(in);
  if (st != SAKI_OK) return st;
  if (k < 1 || k > SAKI_MAX_PROBE_K || k > in->vocab) return fail(SAKI_E_SHAPE, "k outside [1, min(SAKI_MAX_PROBE_K, vocab)]");
  if (in->n_rows == 0) return ok();
  int cus = 0;
  st = device_cus(&cus);
  if (st != SAKI_OK) return st;
  saki::ProbeParams P{};
  P.s = in->student;
  P.t = in->teacher;
  P.n_rows = in->n_rows;
  P.stride = in->row_stride;
  P.V = static_cast<int>(in->vocab);
  P.k = k;
  P.c1 = c1;
  P.ck = ck;
  P.kl_ts = kl_ts;
  P.entropy = entropy;
  P.topk = topk;
  P.row_status = row_status;
  const int grid = static_cast<int>(std::min<int64_t>(in->n_rows, static_cast<int64_t>(cus) * saki::PROBE_WG_PER_CU));
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (in->dtype == SAKI_BF16)
    hipLaunchKernelGGL(saki::probe_kernel<uint16_t>, dim3(grid), dim3(saki::NT), 0, hs, P);
  else
    hipLaunchKernelGGL(saki::probe_kernel<float>, dim3(grid), dim3(saki::NT), 0, hs, P);
  st = launched("probe_kernel");
  if (st != SAKI_OK) return st;
  return ok();
}

saki_status saki_select_positions(int32_t mode, int64_t n_traj, int64_t n_rows,
                                  const int64_t* traj_offsets, const float* tv,
                                  const uint8_t* corrected, const uint8_t* valid_mask, uint64_t seed,
                                  int64_t row_offset, uint8_t* selected, void* ws, size_t ws_bytes,
                                  saki_stream_t stream) {
  if (mode != SAKI_SELECT_RANDOM && mode != SAKI_SELECT_TV_WEIGHTED) return fail(SAKI_E_VALUE, "unknown mode");
  if (n_traj < 0 || n_rows < 0) return fail(SAKI_E_SHAPE, "n_traj < 0 or n_rows < 0");
  if (row_offset < 0) return fail(SAKI_E_VALUE, "row_offset < 0");
  if (n_traj == 0 || n_rows == 0) return ok();
  if (!traj_offsets || !tv || !corrected || !selected)
    return fail(SAKI_E_NULLPTR, "traj_offsets, tv, corrected and selected are required");
  if (!ws) return fail(SAKI_E_WORKSPACE, "workspace is NULL");
  if (ws_bytes < loss_ws_bytes(n_rows)) return fail(SAKI_E_WORKSPACE, "workspace too small");
  if ((reinterpret_cast<uintptr_t>(ws) & 7u) != 0) return fail(SAKI_E_ALIGN, "workspace must be 8-byte aligned");
  int cus = 0;
  saki_status st = device_cus(&cus);
  if (st != SAKI_OK) return st;
  saki::SelectParams P{};
  P.mode = mode;
  P.n_traj = n_traj;
  P.n_rows = n_rows;
  P.off = traj_offsets;
  P.tv = tv;
  P.corrected = corrected;
  P.valid = valid_mask;
  P.seed = seed;
  P.row_offset = row_offset;
  P.sel = selected;
  P.keys = static_cast<double*>(ws);
  const int grid = static_cast<int>(std::min<int64_t>(n_traj, static_cast<int64_t>(cus) * 4));
  hipLaunchKernelGGL(saki::select_kernel, dim3(grid), dim3(saki::SNT), 0, static_cast<hipStream_t>(stream), P);
  st = launched("select_kernel");
  if (st != SAKI_OK) return st;
  return ok();
}

const char* saki_status_str(saki_status s) {
  switch (s) {
    case SAKI_OK: return "ok";
    case SAKI_E_NULLPTR: return "a required pointer is NULL";
    case SAKI_E_SHAPE: return "invalid shape";
    case SAKI_E_VALUE: return "invalid value";
    case SAKI_E_DTYPE: return "unknown dtype";
    case SAKI_E_ALIGN: return "pointer or pitch not 16-byte aligned";
    case SAKI_E_WORKSPACE: return "workspace missing or too small";
    case SAKI_E_DEVICE: return "HIP device error";
    case SAKI_E_LAUNCH: return "kernel launch failed";
  }
  return "unknown status";
}

const char* saki_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
