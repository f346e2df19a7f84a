/*
 * saki.h -- C ABI of the SAKI coupling-and-routing library for AMD MI355X (gfx950).
 *
 * Per position (one row of [positions x vocab] logits) the library
 *   1. forms the student p = softmax(s) and teacher pi = softmax(t);
 *   2. finds the trust-region bridge coefficient lambda*, the largest lambda in
 *      [0, 1] with KL(q_lambda || p) <= eps, where q_lambda is proportional to
 *      p^(1-lambda) * pi^lambda                     (SAKI Sec. 3.2, Eq. bridge,
 *                                                    Eq. trust_region, App. A);
 *   3. realises q = q_lambda* by maximal coupling with p: z ~ p, accept with
 *      probability min(1, q(z)/p(z)), else draw a correction from the normalised
 *      positive residual [q - p]_+                (Sec. 3.3, Eq. accept, Eq. residual);
 *   4. routes the loss: sampled-token reverse KL at accepted rows, the teacher
 *      argmax cross-entropy at corrections, and writes its gradient with respect
 *      to the student logits                      (Sec. 3.4, Eq. general_objective, App. H);
 *   5. for speculative blocks of k drafted tokens, commits the longest accepted
 *      prefix and draws the correction at the first rejection
 *                                                 (Sec. 3.5, App. F, App. I);
 *   6. supervision variants: a correction target drawn from the teacher
 *      instead of its mode (App. C), and the Random-TM / TV-Weighted-TM
 *      placement controls (Sec. 4.1, placement-control appendix);
 *   7. the other steps of a speculative rollout wave: student draft sampling,
 *      and the first-rejection commit with token-aligned metadata packing
 *                                                 (App. I; App. F, Prop. spec_exact).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.     Every array argument is DEVICE memory owned by the caller.  The
 *             library never allocates, frees or synchronises; scratch space is
 *             the caller's workspace, sized by saki_workspace_bytes().
 * Streams.    Every call only enqueues work on `stream` (a hipStream_t; NULL is
 *             the default stream) and returns without waiting for it.
 * Layout.     Logit rows are row-major, contiguous in the vocabulary:
 *             element (r, v) is at base[r * row_stride + v].  The base pointer
 *             must be 16-byte aligned and row_stride * sizeof(element) a
 *             multiple of 16.  1 <= vocab <= SAKI_MAX_VOCAB, row_stride >= vocab.
 * Randomness. Draws come from Philox-4x32-10 (Salmon et al., SC'11) keyed by
 *             (seed, stream id, global row g = row_offset + r), so results are
 *             a deterministic function of (input bits, eps, seed, g) and do not
 *             depend on launch geometry or on how rows are split into calls.
 * Errors.     Argument errors are found on the host before anything is
 *             enqueued and return a SAKI_E_* code (details: saki_last_error()).
 *             Data errors found on the device never abort: the row gets a
 *             non-zero row_status, NaN in its float outputs and -1 in its index
 *             outputs, and other rows are unaffected.  No C++ exception crosses
 *             this interface.  n_rows == 0 returns SAKI_OK and enqueues nothing.
 */
#ifndef SAKI_H
#define SAKI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SAKI_MAX_VOCAB (1 << 21) /* 2,097,152 entries per row */
#define SAKI_CHUNK 1024          /* vocab entries per race chunk (sampler definition) */
#define SAKI_MAX_BLOCK_K 64      /* largest speculative block length */
#define SAKI_MAX_PROBE_K 64      /* largest teacher Top-k of the probe metrics */

typedef void *saki_stream_t; /* a hipStream_t; NULL = the default stream */

typedef enum { SAKI_F32 = 0, SAKI_BF16 = 1 } saki_dtype;

typedef enum {
  SAKI_OK = 0,
  SAKI_E_NULLPTR = 1,   /* a required pointer is NULL */
  SAKI_E_SHAPE = 2,     /* n_rows < 0, vocab outside [1, SAKI_MAX_VOCAB], row_stride < vocab, bad k */
  SAKI_E_VALUE = 3,     /* eps < 0 or NaN, grad_scale not finite, row_offset < 0 */
  SAKI_E_DTYPE = 4,     /* unknown saki_dtype */
  SAKI_E_ALIGN = 5,     /* base pointer or row pitch not 16-byte aligned */
  SAKI_E_WORKSPACE = 6, /* workspace NULL or smaller than saki_workspace_bytes() */
  SAKI_E_DEVICE = 7,    /* no usable HIP device, or a HIP call failed */
  SAKI_E_LAUNCH = 8     /* a kernel launch failed */
} saki_status;

/* Row status codes written to saki_couple_out.row_status. */
#define SAKI_ROW_OK 0
#define SAKI_ROW_NONFINITE 1 /* a student or teacher logit is NaN or infinite */
#define SAKI_ROW_BAD_DRAFT 2 /* a draft token id is outside [0, vocab) */
#define SAKI_ROW_SKIPPED 3   /* verify: position after the end of the committed prefix */

/* Student and teacher logits for n_rows positions (Sec. 3.1: p at prefix h_t and
 * pi_T at the same prefix).  Both arrays have the same dtype, shape and stride. */
typedef struct {
  const void *student; /* [n_rows, row_stride]; p = softmax(student row)            */
  const void *teacher; /* [n_rows, row_stride]; pi = softmax(teacher row)           */
  int32_t dtype;       /* saki_dtype of both arrays                                */
  int32_t reserved;    /* must be 0                                                */
  int64_t n_rows;      /* number of positions, >= 0                                */
  int64_t vocab;       /* entries per row used, 1 .. SAKI_MAX_VOCAB                */
  int64_t row_stride;  /* elements between consecutive rows, >= vocab              */
  int64_t row_offset;  /* global index of row 0 (keys the random draws), >= 0      */
} saki_rows;

/* Per-row outputs of the coupling (token-aligned metadata, Sec. 3.5 and App. I).
 * Every pointer may be NULL, in which case that output is not written. Arrays
 * have n_rows entries. */
typedef struct {
  float *lambda;          /* lambda*                                                   */
  float *kl;              /* KL(q_lambda* || p)                                         */
  float *tv;              /* TV(p, q) = sum_v [q(v) - p(v)]_+ = Pr(correction) (Prop. 1)  */
  float *accept_prob;     /* alpha = min(1, q(z)/p(z)) at the proposal z                */
  float *margin;          /* |u - alpha|, distance of the accept decision from a tie    */
  float *logp_token;      /* log p(y) of the committed token y                          */
  float *logt_token;      /* log pi_T(y)                                                 */
  float *logq_token;      /* log q(y)                                                    */
  int32_t *proposal;      /* z, the student proposal                                    */
  int32_t *token;         /* y, the committed token (z if accepted, else the correction) */
  int32_t *teacher_argmax;/* v* = argmax_v t_v, lowest index on ties                    */
  uint8_t *corrected;     /* C: 1 if the proposal was rejected                          */
  uint8_t *row_status;    /* SAKI_ROW_*                                                  */
  int32_t *target;        /* index of the gradient's indicator: y at accepted rows; at a
                             correction v*, or the teacher draw v~ with
                             SAKI_TARGET_SAMPLE; -1 at rows without outputs         */
} saki_couple_out;

/* Routing arguments (Eq. general_objective).  row loss
 *   l_r = M_r * [ (1 - C_r) * (-A_r) * log p(y_r) + C_r * (-log p(v*_r)) ],
 *   A_r = log pi_T(y_r) - log p(y_r)   (detached advantage, Eq. k1_advantage_token),
 * gradient  g[r, j] = grad_scale * M_r * d l_r / d s[r, j]
 *         = grad_scale * M_r * [ (1 - C_r) * (-A_r) * (1[j = y_r] - p_j) + C_r * (p_j - 1[j = v*_r]) ]. */
/* Supervision target at corrections (saki_route_args.correction_target). */
#define SAKI_TARGET_MODE 0   /* v* = argmax t (Eq. teacher_mode_loss)                        */
#define SAKI_TARGET_SAMPLE 1 /* v~ ~ pi_T, L_TS = -log pi_theta(v~) (App. C, teacher-sampled
                                supervision): the two-level exponential race of the coupling
                                on log pi_T with Philox streams 5 (chunks) and 6 (entries)  */

typedef struct {
  const uint8_t *valid_mask; /* M, [n_rows] (0 / non-zero); NULL = every row valid        */
  float grad_scale;          /* the caller's 1 / N_valid over the WHOLE batch (App. H)    */
  int32_t grad_dtype;        /* saki_dtype of grad                                        */
  float *row_loss;           /* [n_rows] unscaled l_r, or NULL                            */
  double *loss_sum;          /* one double: OVERWRITTEN with sum_r grad_scale * l_r, or NULL */
  void *grad;                /* [n_rows, grad_stride] gradient, or NULL (loss only)       */
  int64_t grad_stride;       /* elements between gradient rows, >= vocab                  */
  int32_t correction_target; /* SAKI_TARGET_MODE or SAKI_TARGET_SAMPLE (saki_couple; the
                                standalone saki_route_loss takes its targets as input)    */
} saki_route_args;

/* Operation codes for saki_workspace_bytes. */
#define SAKI_OP_COUPLE 0
#define SAKI_OP_ROUTE 1
#define SAKI_OP_VERIFY 2
#define SAKI_OP_SELECT 3

/* Bytes of caller workspace that one call of `op` on n_rows rows of `vocab`
 * entries needs (device memory, any contents, 256-byte aligned).  For
 * SAKI_OP_VERIFY n_rows is the number of blocks times k. */
size_t saki_workspace_bytes(int op, int64_t n_rows, int64_t vocab);

/* Coupling for every row (Sec. 3.2-3.3) and, when route != NULL, the routed
 * loss and gradient fused into the same pass (Sec. 3.4).
 *   in     rows of student / teacher logits
 *   eps    trust-region radius, eps >= 0 (eps = 0 gives q = p and no corrections)
 *   seed   64-bit Philox key
 *   out    per-row outputs (any field may be NULL); out itself may not be NULL
 *   route  NULL for coupling only
 *   ws     required when n_rows > 0: ws_bytes >= saki_workspace_bytes(SAKI_OP_COUPLE,
 *          n_rows, vocab), 8-byte aligned.  Its first 256 bytes hold the counters
 *          from which workgroups take rows (cleared by the call on `stream`); the
 *          scaled row losses follow (with route->loss_sum), then the list of rows
 *          a second launch of the call resolves again with every sweep in its
 *          expm1 form (rows whose TV turns out too small for the plain forms'
 *          rounding; rare).  Calls that may run at the same time need separate
 *          workspaces.
 * More than 2^31 - 1 rows in one call is SAKI_E_SHAPE (split the rows into calls
 * with row_offset; results do not change). */
saki_status saki_couple(const saki_rows *in, double eps, uint64_t seed, const saki_couple_out *out,
                        const saki_route_args *route, void *ws, size_t ws_bytes,
                        saki_stream_t stream);

/* Largest n_rows of one saki_couple_static call. */
#define SAKI_STATIC_MAX_ROWS 262144

/* saki_couple for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  Same
 * arguments, kernels and results as saki_couple, without the workspace: the
 * work counters, the scaled row losses and the list of rows for the second
 * launch live in a static device array of the library (256 + 12 *
 * SAKI_STATIC_MAX_ROWS bytes = 3 MiB + 256 B), which each GPU the library runs
 * on holds until the process ends.  Its device
 * address is looked up once per device, on the first call made with that
 * device current.  The call allocates and frees nothing.
 *   n_rows > SAKI_STATIC_MAX_ROWS  SAKI_E_SHAPE, nothing enqueued (split the
 *                                  rows into calls with row_offset)
 * The array keeps the last call's contents; each call clears the counters
 * itself (a kernel on `stream`), writes every scaled row loss before summing
 * them and every list entry before the second launch reads it.  All calls on one GPU share the array: calls whose work can
 * overlap in time on one GPU (other streams, concurrent graph replays) race
 * and give wrong results; serialise them, or use saki_couple with separate
 * workspaces. */
saki_status saki_couple_static(const saki_rows *in, double eps, uint64_t seed,
                               const saki_couple_out *out, const saki_route_args *route,
                               saki_stream_t stream);

/* Routed loss and gradient from given events (Sec. 3.4), for callers that
 * already hold the coupling results.  student: [n_rows, row_stride] logits of
 * pi_theta (= p).  token y, corrected C, teacher_argmax v* and advantage A
 * (= log pi_T(y) - log p(y), read only at rows with C = 0) are [n_rows] device
 * arrays.  A token or v* outside [0, vocab) at a valid row gives that row a NaN
 * loss and a NaN gradient row.
 *   ws  required when n_rows > 0: ws_bytes >= saki_workspace_bytes(SAKI_OP_ROUTE,
 *       n_rows, vocab), 8-byte aligned.  Its first 256 bytes hold the counter from
 *       which workgroups take rows (cleared by the call on `stream`); with
 *       route->loss_sum the scaled row losses follow.  Calls that may run at the
 *       same time need separate workspaces.
 * More than 2^31 - 1 rows in one call is SAKI_E_SHAPE. */
saki_status saki_route_loss(const void *student, int32_t dtype, int64_t n_rows, int64_t vocab,
                            int64_t row_stride, const int32_t *token, const uint8_t *corrected,
                            const int32_t *teacher_argmax, const float *advantage,
                            const saki_route_args *route, void *ws, size_t ws_bytes,
                            saki_stream_t stream);

/* Speculative block verification (Sec. 3.5, App. F, App. I).  Rows are
 * block-major: row b*k + j holds position j of block b, whose student draft is
 * draft[b*k + j].  Positions are examined in order; position j is accepted iff
 * u_j < alpha_j(draft_j) with u_j the ACCEPT uniform of its global row; the
 * block commits the accepted prefix of length n and, if n < k, the correction
 * drawn from [q_n - p_n]_+ at position n.  With eos_id >= 0 an accepted draft
 * equal to eos_id at position j ends the block: n = j + 1, no correction.  A
 * position with bad data (non-finite logits, draft outside the vocabulary) ends
 * the block before it with no correction.
 *   accepted_len [n_blocks]  n
 *   correction   [n_blocks]  the correction token, or -1
 *   per_pos      optional per-position outputs ([n_rows], fields may be NULL):
 *                positions after the end of the committed prefix get NaN / -1
 *                and row_status SAKI_ROW_SKIPPED; proposal = the draft, token =
 *                the committed token.
 *   ws           required: ws_bytes >= saki_workspace_bytes(SAKI_OP_VERIFY, n_rows,
 *                vocab) (256 bytes), 4-byte aligned; it holds the counter from
 *                which workgroups take blocks, cleared by the call on `stream`.
 *                Calls that may run at the same time need separate workspaces.
 * More than 2^31 - 1 blocks is SAKI_E_SHAPE. */
saki_status saki_spec_verify(const saki_rows *in, int32_t k, const int32_t *draft, double eps,
                             uint64_t seed, int32_t eos_id, int32_t *accepted_len,
                             int32_t *correction, const saki_couple_out *per_pos, void *ws,
                             size_t ws_bytes, saki_stream_t stream);

/* Student draft sampling for speculative rollouts (App. I, step 1).
 * z_r ~ p_r = softmax(student row r) by the coupling's two-level exponential
 * race on the proposal streams (0: chunks, 1: entries) of the global row
 * g = in->row_offset + r * row_step, so a draft equals the proposal that
 * saki_couple draws at row g (up to float rounding of near-tied race keys).
 * With row_step = k, drafting position j of a wave whose verification rows
 * start at G uses row_offset = G + j: draft j of sequence b is keyed by the row
 * b*k + j that verifies it.  in->teacher is not read and may be NULL.
 *   token      [n_rows] z_r, or -1 for a row with a non-finite student logit
 *   row_status [n_rows] SAKI_ROW_OK / SAKI_ROW_NONFINITE, or NULL
 * row_step >= 1; the last row's g must stay below 2^63. */
saki_status saki_sample(const saki_rows *in, int64_t row_step, uint64_t seed, int32_t *token,
                        uint8_t *row_status, saki_stream_t stream);

/* Token-aligned trajectories of a speculative rollout (App. I, steps 7-8).
 * Arrays of [n_seq, max_len] entries are row-major per sequence; position
 * i of sequence b is entry b * max_len + i.  Optional arrays may be NULL. */
#define SAKI_SEQ_RUNNING 0
#define SAKI_SEQ_FINISHED 1 /* reached max_len, or committed eos_id                       */
#define SAKI_SEQ_STOPPED 2  /* a wave committed nothing (bad logits or an out-of-vocabulary
                               draft at the block's first position), or length was invalid */
typedef struct {
  int64_t n_seq;           /* sequences, >= 0                                               */
  int64_t max_len;         /* positions per sequence, 0 .. 2^31 - 1                         */
  int32_t *tokens;         /* [n_seq, max_len] committed tokens (required)                  */
  uint8_t *corrected;      /* [n_seq, max_len] 1 at a correction, 0 at an accepted draft     */
  float *lambda;           /* [n_seq, max_len] lambda* at the position                      */
  float *kl;               /* [n_seq, max_len] KL(q || p)                                   */
  float *tv;               /* [n_seq, max_len] TV(p, q)                                     */
  float *logp_token;       /* [n_seq, max_len] log p(y)                                     */
  float *logt_token;       /* [n_seq, max_len] log pi_T(y)                                  */
  int32_t *teacher_argmax; /* [n_seq, max_len] v*                                           */
  int32_t *length;         /* [n_seq] committed tokens so far; read and updated (required)  */
  uint8_t *done;           /* [n_seq] SAKI_SEQ_*; read and updated (required)               */
} saki_traj;

/* First-rejection commit of one speculative wave (App. I, steps 7-8; App. F).
 * Inputs are the outputs of saki_spec_verify over n_seq blocks of k positions
 * (block b = sequence b): accepted_len and correction [n_seq], and per_pos, its
 * per-position outputs [n_seq * k], of which token is required and lambda, kl,
 * tv, logp_token, logt_token, teacher_argmax are copied where both sides are
 * non-NULL (NaN / -1 where only the destination is).  For each sequence with
 * done == SAKI_SEQ_RUNNING, the n accepted drafts and, if n < k and
 * correction >= 0, the correction are appended at positions length .. in token
 * order, at most max_len - length of them; every later position of the block
 * is discarded.  Then length grows by the count m, and done becomes
 * SAKI_SEQ_FINISHED when length reaches max_len or the last committed token is
 * eos_id (eos_id >= 0), SAKI_SEQ_STOPPED when m = 0.  Sequences not running
 * are left as they are.
 *   n_commit  [n_seq] m (0 for sequences not running), or NULL
 * The caller's model continues sequence b from the state after its committed
 * prefix: the draft state after m - 1 drafts, advanced by the last committed
 * token (this is the rollback of every later speculative state).
 * Requirements: 1 <= k <= SAKI_MAX_BLOCK_K, max_len <= 2^31 - 1. */
saki_status saki_commit(const saki_traj *traj, int32_t k, int32_t eos_id,
                        const int32_t *accepted_len, const int32_t *correction,
                        const saki_couple_out *per_pos, int32_t *n_commit, saki_stream_t stream);

/* Placement controls (Sec. 4.1; placement-control appendix).  Rows are grouped
 * into trajectories: trajectory i holds rows [traj_offsets[i], traj_offsets[i+1])
 * (device int64 array of n_traj + 1 non-decreasing entries in [0, n_rows]; a
 * trajectory whose range is malformed is skipped and its rows are not written).
 * For each trajectory with valid rows V_i (valid_mask non-zero, or every row
 * when valid_mask is NULL), m_i = sum over V_i of corrected, and exactly m_i
 * rows of V_i get selected = 1, every other row 0:
 *   SAKI_SELECT_RANDOM       m_i rows of V_i uniformly without replacement;
 *   SAKI_SELECT_TV_WEIGHTED  m_i rows without replacement with weights tv
 *                            (keys -log U / tv, the m_i smallest win); when fewer
 *                            than m_i valid rows have tv > 0, the rest are filled
 *                            uniformly from the rows with tv = 0 (or NaN).
 * U is the Philox uniform of stream 7, index 0, of the global row row_offset + r.
 * Selected rows take the teacher-mode loss and the others keep RKL: pass
 * `selected` as `corrected` to saki_route_loss.  tv, corrected (uint8) and
 * selected are [n_rows] device arrays; ws holds one double per row
 * (saki_workspace_bytes(SAKI_OP_SELECT, n_rows, 0)), 8-byte aligned. */
#define SAKI_SELECT_RANDOM 0
#define SAKI_SELECT_TV_WEIGHTED 1
saki_status saki_select_positions(int32_t mode, int64_t n_traj, int64_t n_rows,
                                  const int64_t *traj_offsets, const float *tv,
                                  const uint8_t *corrected, const uint8_t *valid_mask,
                                  uint64_t seed, int64_t row_offset, uint8_t *selected,
                                  void *ws, size_t ws_bytes, saki_stream_t stream);

/* Fixed-prefix probe metrics (the paper's probe analysis), per row of
 * student / teacher logits: S = softmax(student), T = softmax(teacher),
 *   c1[r]      = S(v*), v* the teacher's Top-1 (lowest index on ties);
 *   ck[r]      = sum of S over the teacher's Top-k set (the k largest teacher
 *                logits, ties to the lower index; k = 16 in the paper);
 *   kl_ts[r]   = KL(T || S) = E_T[t - s] - (lse_t - lse_s), the conflict measure
 *                (accumulated in double from float partial sums: relative error
 *                ~1e-7 x E_T[t - s] / KL);
 *   entropy[r] = H(S);
 *   topk       = [n_rows, k] the Top-k indices, best first.
 * Every output may be NULL.  1 <= k <= min(SAKI_MAX_PROBE_K, vocab).  Rows with a
 * non-finite logit get NaN metrics, topk -1 and row_status SAKI_ROW_NONFINITE.
 * One workgroup per row: one sweep over both rows, then only the teacher
 * chunks whose maximum reaches a lower bound of the k-th largest logit (a few
 * per row); a row where more than 256 teacher entries reach that bound (heavy
 * ties) takes a counting search of several more sweeps of the teacher row. */
saki_status saki_probe_metrics(const saki_rows *in, int32_t k, float *c1, float *ck, float *kl_ts,
                               float *entropy, int32_t *topk, uint8_t *row_status,
                               saki_stream_t stream);

/* Static description of a status code. */
const char *saki_status_str(saki_status s);

/* Detail of the last non-OK status returned on the calling thread ("" if none). */
const char *saki_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SAKI_H */
