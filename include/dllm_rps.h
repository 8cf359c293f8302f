/*
 * dllm_rps.h - C ABI of the MI355X (gfx950) library for one batched denoising
 * step of Ripple-Pivot Search (RPS) over a bidirectional masked-diffusion
 * transformer.
 *
 * The paper (Ripple-Pivot Search: Active Parallel Decoding for Diffusion
 * Large Language Models) treats the model as a black box that returns, in one
 * forward pass over [y || x], a predictive distribution p_i for every masked
 * response position i (Section 3, Notation).  A scheduler then commits
 * positions (Eq. 1 and Eq. 2), picks a mid-entropy pivot (Eq. 3), evaluates
 * candidate tokens for it by lookahead (Eq. 4) and commits or abstains,
 * carrying the chosen branch's distributions to the next step (Section 4.1,
 * Algorithm 1).  This header exposes those operations as device calls.
 *
 * Conventions (every entry point):
 *  - Every tensor argument is a DEVICE pointer owned by the caller; the
 *    library only borrows it for the stream-ordered duration of the call.
 *    Struct arguments (dllm_stats, rps_params, ...) are HOST structs, read
 *    during the call; the pointers inside them are device pointers.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL means the
 *    default stream) and enqueues kernels only: no allocation, no host
 *    synchronisation.  The caller provides scratch memory as `ws` of at least
 *    the size the matching *_workspace_bytes function returns.
 *  - Arguments are validated on the host before anything is enqueued.  On
 *    error nothing is enqueued, the status is returned and
 *    dllm_last_error() describes it (thread-local).  Nothing aborts or throws
 *    across the ABI.  Asynchronous device faults surface as DLLM_EHIP from a
 *    later call.
 *  - Matrices are row-major.  Weights use the [out_features][in_features]
 *    layout, so a projection computes y = x W^T.
 *  - A model handle may be used by one stream at a time.
 */
#ifndef DLLM_RPS_H
#define DLLM_RPS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DLLM_ABI_VERSION 1
#define DLLM_MAX_TOPK 16       /* top-K entries kept per position */
#define RPS_MAX_PIVOTS 16
#define RPS_MAX_BRANCH 16      /* lookahead branches per step */
#define RPS_MAX_MASKED 1024    /* masked positions per step */

typedef enum {
    DLLM_OK = 0,
    DLLM_EINVAL = 1,        /* null pointer or out-of-range scalar */
    DLLM_ESHAPE = 2,        /* unsupported or inconsistent sizes */
    DLLM_EDTYPE = 3,        /* unknown dtype */
    DLLM_ENOMEM = 4,        /* workspace smaller than required */
    DLLM_EHIP = 5,          /* HIP runtime error (launch or earlier async fault) */
    DLLM_EUNSUPPORTED = 6
} dllm_status;

typedef enum { DLLM_F32 = 0, DLLM_BF16 = 1 } dllm_dtype;

typedef void* dllm_stream;  /* hipStream_t */

/* Model shape.  The architecture (the paper does not fix one) is a
 * bidirectional pre-RMSNorm transformer with rotate-half RoPE, full
 * non-causal softmax attention, SwiGLU feed-forward, untied embedding and LM
 * head, unit RMSNorm gains and no biases.  Requirements: d_model =
 * n_heads * head_dim, head_dim in {64, 128}, d_model % 256 == 0, d_model <= 8192,
 * d_ffn % 128 == 0, 0 <= mask_id < vocab. */
typedef struct {
    int32_t n_layers, d_model, n_heads, head_dim, d_ffn, vocab, mask_id;
    float rope_base;        /* e.g. 10000 */
    float rms_eps;          /* e.g. 1e-5 */
    int32_t dtype;          /* dllm_dtype of weights and activations */
    int32_t max_pos;        /* RoPE table size: largest position id + 1 */
} dllm_model_desc;

/* Weights, device pointers of the model dtype.  The per-layer arrays are host
 * arrays of n_layers device pointers; the handle copies the arrays and
 * borrows the device memory until dllm_model_destroy. */
typedef struct {
    const void* emb;                 /* [vocab][d] */
    const void* lm_head;             /* [vocab][d] */
    const void* const* wqkv;         /* [3d][d]: rows Q, then K, then V */
    const void* const* wo;           /* [d][d] */
    const void* const* wgu;          /* [2F][d]: rows gate, then up */
    const void* const* wdown;        /* [d][F] */
} dllm_weights;

/* Per-position statistics of the predictive distributions (Section 3,
 * Notation), struct of arrays over R rows.  Computed over the vocabulary
 * without [MASK] (its logit is -inf).  Natural log, entropies in nats.
 *   lmax   largest scaled logit          lse  log sum_v exp(logit_v)
 *   H      -sum_v p_v log p_v            argmax  token of lmax, lowest id on ties
 *   topk_id / topk_logit  [R][k]: tokens by logit descending, lower id first
 *                          on ties, and their scaled logits; log p = logit - lse.
 * P^max = exp(lmax - lse). */
typedef struct {
    float* H;
    float* lse;
    float* lmax;
    int32_t* argmax;
    int32_t* topk_id;
    float* topk_logit;
    int32_t k;              /* entries per row (row stride), 1..DLLM_MAX_TOPK */
} dllm_stats;

/* Cached keys/values of a prefix (the block-wise prefix cache used with RPS
 * in Section 5.3).  k: [n_layers][n_heads][cap][head_dim], post-RoPE;
 * vt: [n_layers][n_heads][head_dim][cap] (values transposed).  k in the
 * model dtype; vt float32 for f32 models and IEEE binary16 (values saturated
 * to +-65504) for bf16 models, the type the attention's P V product uses. */
typedef struct {
    void* k;
    void* vt;
    int32_t len;            /* valid prefix positions 0 .. len-1 */
    int32_t cap;            /* allocated positions per (layer, head) */
} dllm_kv_cache;

/* Scaled logits of chosen (row, token) pairs, e.g. p_anchor(c) at the pivot
 * for tokens outside the stored top-K (Eq. 4's plausibility term). */
typedef struct {
    const int32_t* row;     /* [n] output-stats row index */
    const int32_t* token;   /* [n] */
    float* logit;           /* [n] out: scaled logit */
    int32_t n;
} dllm_probe;

typedef struct dllm_model dllm_model;

/* ---------------------------------------------------------------- library */

int32_t dllm_abi_version(void);
const char* dllm_last_error(void);
const char* dllm_status_string(dllm_status s);

/* Create a model handle.  Copies desc and the weight-pointer arrays; uploads
 * a RoPE cos/sin table (computed in double on the host) to the current
 * device.  This is the only call that allocates device memory. */
dllm_status dllm_model_create(const dllm_model_desc* desc, const dllm_weights* w, dllm_model** out);
void dllm_model_destroy(dllm_model* m);

/* Workspace of dllm_forward for `batch` sequences of `seq` positions with
 * statistics at n_lm_pos positions of each sequence. */
size_t dllm_workspace_bytes(const dllm_model* m, int32_t batch, int32_t seq, int32_t n_lm_pos);

/* One denoising forward (the model call of Algorithm 1) over a batch of
 * sequences, ending in the LM head and the fused statistics.
 *   tokens      [batch][seq] int32, values in [0, vocab) (others are clamped).
 *   pos_offset  position id of column 0 (the cached prefix length when
 *               kv_prefix is given, else usually 0).
 *   kv_prefix   nullable; every sequence's positions attend to the cached
 *               prefix keys 0 .. len-1 followed by its own keys.
 *   kv_out      nullable; writes this call's post-RoPE K and V^T at cache
 *               positions pos_offset .. pos_offset+seq-1 (batch must be 1).
 *   lm_pos      [n_lm_pos] int32 positions (0 .. seq-1, clamped) that get the LM
 *               head; output row b * n_lm_pos + j is sequence b, lm_pos[j].
 *   row_scale   nullable [seq] float: per-position logit scale, indexed by
 *               position; logits = scale * row_scale[lm_pos[j]] * (h W_lm^T).
 *   probe       nullable; rows index the output statistics.
 *   out         statistics of batch * n_lm_pos rows.
 * seq % 8 == 0 is not required; seq >= 1, batch >= 1, n_lm_pos >= 1. */
dllm_status dllm_forward(dllm_model* m, const int32_t* tokens, int32_t batch, int32_t seq,
                         int32_t pos_offset, const dllm_kv_cache* kv_prefix, const dllm_kv_cache* kv_out,
                         const int32_t* lm_pos, int32_t n_lm_pos, const float* row_scale, float scale,
                         const dllm_probe* probe, const dllm_stats* out,
                         void* ws, size_t ws_bytes, dllm_stream stream);

/* Packed lookahead forward (Section 4.1, lookahead scoring and Algorithm 1's
 * x_ahead = [x || x_b^(c_1) || ... ]): one sequence holding the shared
 * sequence (the anchor: prompt and response, pivot still masked) followed by
 * n_branch copies of the current block, each with its pivot filled by one
 * candidate, evaluated in one forward with a branch-isolating attention mask.
 *   tokens       [shared_len + n_branch * block_len] int32.
 *   block_start  first position of the current block in the shared sequence;
 *                branch rows reuse the block's position ids.
 *   mask         shared rows attend to the shared rows only; the rows of a
 *                branch attend to the shared rows outside the block they stand
 *                in for (block_start .. block_start+block_len-1) and to their
 *                own block, never to another branch.  With one layer a
 *                branch's rows equal an independent forward of the shared
 *                sequence with the block replaced; with more layers the shared
 *                rows' keys and values are those of the anchor (the packing
 *                approximation).
 *   lm_pos       [n_lm_pos] positions of the shared sequence (clamped to
 *                0 .. shared_len-1).  `out` receives (1 + n_branch) * n_lm_pos
 *                rows, in the order of the unpacked lookahead batch: rows
 *                0 .. n_lm_pos-1 are the shared sequence at lm_pos, rows
 *                (1+c)*n_lm_pos + j are branch c at lm_pos[j] (the shared row
 *                when lm_pos[j] lies outside the block).  probe rows index
 *                these rows.
 *   row_scale    nullable [shared_len] float indexed by in-sequence position
 *                (a branch row uses the scale of the position it copies).
 *   kv_prefix    nullable cached prefix (Section 5.3's prefix cache) that every
 *                row of the packed sequence attends to in full; the packed
 *                rows then start at position pos_offset (typically the block:
 *                shared sequence = the block and the masked suffix, with
 *                block_start 0).
 *   Other arguments as dllm_forward (batch 1, no kv_out).  The workspace is
 *   dllm_workspace_bytes_packed(m, shared_len, block_len, n_branch, n_lm_pos).
 * Errors: DLLM_ESHAPE unless 1 <= n_lm_pos <= shared_len, block_len is a
 *   power of two, n_branch >= 0, 0 <= block_start, block_start + block_len <=
 *   shared_len and pos_offset + shared_len <= max_pos. */
size_t dllm_workspace_bytes_packed(const dllm_model* m, int32_t shared_len, int32_t block_len, int32_t n_branch,
                                   int32_t n_lm_pos);
dllm_status dllm_forward_packed(dllm_model* m, const int32_t* tokens, int32_t shared_len, int32_t block_start,
                                int32_t block_len, int32_t n_branch, int32_t pos_offset, const dllm_kv_cache* kv_prefix,
                                const int32_t* lm_pos, int32_t n_lm_pos, const float* row_scale, float scale,
                                const dllm_probe* probe, const dllm_stats* out, void* ws, size_t ws_bytes,
                                dllm_stream stream);

/* LM head with fused vocabulary statistics (the per-position quantities of
 * Section 3, Notation, that Eq. 1-4 consume): for each of R rows of final
 * normed hidden states, logits = scale * row_scale[r] * (hidden[r] W_lm^T),
 * logit[mask_id] = -inf (mask_id < 0: none), then H, lse, lmax, argmax and
 * top-k.  The [R][vocab] logits are never written to memory.
 *   hidden [R][d], w_lm [vocab][d], dtype of both = `dtype`.  d % 64 == 0
 *   (bf16) or d % 32 == 0 (f32). */
size_t vocab_entropy_topk_workspace_bytes(int32_t R, int32_t vocab);
dllm_status vocab_entropy_topk(const void* hidden, const void* w_lm, int32_t R, int32_t d, int32_t vocab,
                               int32_t dtype, const float* row_scale, float scale, int32_t mask_id,
                               const dllm_stats* out, void* ws, size_t ws_bytes, dllm_stream stream);

/* Allocation-free variant of vocab_entropy_topk, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same kernels and results, with the
 * partial statistics in a device scratch array that the library holds on
 * every device it runs on (DLLM_NOALLOC_SCRATCH_BYTES, until the process
 * ends) instead of a caller workspace.  Arguments as vocab_entropy_topk; the
 * caller still owns hidden, w_lm, row_scale and out.  The device is the
 * stream's (the current device for the NULL stream); the first call on a
 * device looks the scratch up (hipGetSymbolAddress), no call allocates.
 * All calls on one device share its scratch: calls that overlap on one
 * device (concurrent streams, threads) race and must be serialised by the
 * caller.  Errors: those of vocab_entropy_topk, and DLLM_ENOMEM when
 * vocab_entropy_topk_workspace_bytes(R, vocab) exceeds the scratch
 * (beyond about 180 000 rows). */
#define DLLM_NOALLOC_SCRATCH_BYTES (48u << 20)
dllm_status vocab_entropy_topk_noalloc(const void* hidden, const void* w_lm, int32_t R, int32_t d, int32_t vocab,
                                       int32_t dtype, const float* row_scale, float scale, int32_t mask_id,
                                       const dllm_stats* out, dllm_stream stream);

/* Kernel timing for benchmarks.  Between dllm_profile_begin and
 * dllm_profile_end every kernel that dllm_forward launches is bracketed by
 * HIP events on the launch stream (for at most max_launches launches).
 * dllm_profile_end waits for those events and returns, per kernel class,
 * the summed duration in ms and the launch count (arrays of
 * DLLM_PROF_CLASSES entries, host memory).  begin creates the events (it
 * allocates); the forward itself does not. */
#define DLLM_PROF_CLASSES 10
typedef enum {
    DLLM_PROF_EMBED = 0, DLLM_PROF_RMSNORM = 1, DLLM_PROF_GEMM_QKV = 2, DLLM_PROF_ATTENTION = 3,
    DLLM_PROF_GEMM_O = 4, DLLM_PROF_GEMM_GATEUP = 5, DLLM_PROF_GEMM_DOWN = 6, DLLM_PROF_LMHEAD = 7,
    DLLM_PROF_LMHEAD_MERGE = 8, DLLM_PROF_OTHER = 9
} dllm_prof_class;
dllm_status dllm_profile_begin(dllm_model* m, int32_t max_launches);
/* As dllm_profile_begin, bracketing only the launches of the classes whose
 * bit (1 << class) is set in class_mask: each pair of events costs a few
 * microseconds of stream time, so a benchmark that times whole steps
 * brackets only the kernel it reports on.  class_mask == 0 is EINVAL. */
dllm_status dllm_profile_begin_classes(dllm_model* m, int32_t max_launches, uint32_t class_mask);
dllm_status dllm_profile_end(dllm_model* m, float* ms, int32_t* launches);
/* Benchmark calibration, not part of the method: the bf16 MFMA rate this
 * device sustains on a register-only loop of v_mfma_f32_16x16x32_bf16 (no
 * memory traffic), in TFLOP/s, written to *tflops (host memory).  With
 * random_operands != 0 every MFMA takes different random bf16 operands, as a
 * GEMM on real data does: the datapath then draws more power and the
 * sustained clock drops, so this is the attainable ceiling against which a
 * GEMM's rate is judged (the published 2.5 PFLOP/s assumes the peak clock).
 * Runs about 25 ms of work on `stream` and waits for it; creates and destroys
 * two events. */
dllm_status dllm_mfma_ceiling(int32_t random_operands, float* tflops, dllm_stream stream);

/* ---------------------------------------------------------------- scheduler */

typedef enum {
    RPS_PIVOT_PAPER = 0,   /* Eq. 3: feasible iff top-k_max mass >= tau_pivot */
    RPS_PIVOT_BAND = 1     /* feasible iff H within [pct_lo, pct_hi] percentiles of H over M */
} rps_pivot_mode;

typedef struct {
    int32_t mode;          /* rps_pivot_mode */
    int32_t k_max;         /* truncated support size, <= stats k */
    float tau_pivot;       /* mass threshold (paper mode), inclusive */
    float pct_lo, pct_hi;  /* band percentiles in [0, 100] (band mode), inclusive */
    int32_t n_pivots;      /* pivots taken, by truncated entropy (1 in paper mode) */
    float r;               /* reachability ratio: keep c if p(c) >= r * P^max */
    int32_t n_cand;        /* candidates per pivot, <= k_max */
    int32_t max_branch;    /* total lookahead branches, <= RPS_MAX_BRANCH */
} rps_params;

/* Device-resident lookahead plan written by rps_select_pivots.  Branches are
 * ordered pivot by pivot (pivot rank order), candidates in rank order. */
typedef struct {
    int32_t n_pivots;                    /* 0: skip the lookahead (Algorithm 1 skip rules) */
    int32_t n_branch;
    int32_t pivot_row[RPS_MAX_PIVOTS];   /* index into the masked list */
    int32_t pivot_pos[RPS_MAX_PIVOTS];   /* absolute position */
    int32_t n_cand[RPS_MAX_PIVOTS];
    int32_t br_pivot[RPS_MAX_BRANCH];    /* pivot slot of the branch */
    int32_t br_row[RPS_MAX_BRANCH];
    int32_t br_pos[RPS_MAX_BRANCH];
    int32_t br_token[RPS_MAX_BRANCH];
    float br_logp[RPS_MAX_BRANCH];       /* log p(candidate) under the statistics the plan came from */
} rps_plan;

/* Device-resident decision written by rps_lookahead_score. */
typedef struct {
    int32_t commit;        /* 1: commit token at pivot_pos; 0: abstain or no branch */
    int32_t branch;        /* winning branch in plan order, -1 if none */
    int32_t pivot_row;
    int32_t pivot_pos;
    int32_t token;
    float delta;           /* best Eq. 4 margin over the pivot's [MASK] score */
    float second_delta;    /* runner-up margin (near-tie reporting) */
    int32_t n_masked;      /* |M| the decision was taken over */
} rps_decision;

/* Pivot selection (Eq. 3, or the percentile band) and adaptive candidate
 * sets (Section 4.1) over the n_m masked positions of the current block.
 *   base   statistics, row j <-> position m_pos[j] (ascending positions).
 *   m_pos  [n_m] int32.   1 <= n_m <= RPS_MAX_MASKED.
 * Ties: larger truncated entropy first, then the lower position.  A pivot
 * with at most one candidate is dropped; n_m <= 1 gives an empty plan. */
dllm_status rps_select_pivots(const dllm_stats* base, const int32_t* m_pos, int32_t n_m,
                              const rps_params* prm, rps_plan* plan, dllm_stream stream);

/* Lookahead batch construction: out[slot][seq] int32 for `capacity` slots.
 * With anchor_first, slot 0 is `tokens` unchanged (the anchor branch keeps
 * the pivot masked) and branch b fills slot 1 + b; otherwise branch b fills
 * slot b.  Branch b is `tokens` with br_pos[b] := br_token[b].  Slots beyond
 * the plan's branches repeat `tokens`. */
dllm_status rps_build_branches(const int32_t* tokens, int32_t seq, const rps_plan* plan,
                               int32_t anchor_first, int32_t capacity, int32_t* out, dllm_stream stream);

/* Packed lookahead sequence x_ahead = [x || x_b^(c_1) || ... ] (Algorithm 1,
 * Section 4.1) for dllm_forward_packed: out[seq + capacity * block_len] int32
 * is `tokens`, then for slot b the block block_start .. block_start +
 * block_len - 1 of `tokens` with br_pos[b] := br_token[b] (the unchanged block
 * for slots beyond the plan's branches).  Errors: DLLM_ESHAPE unless 0 <=
 * capacity <= RPS_MAX_BRANCH and the block lies inside 0 .. seq-1. */
dllm_status rps_build_packed(const int32_t* tokens, int32_t seq, const rps_plan* plan, int32_t block_start,
                             int32_t block_len, int32_t capacity, int32_t* out, dllm_stream stream);

/* Lookahead scoring (Eq. 4) and the commit/abstain decision.
 *   anchor    statistics of the anchor branch (pivot still masked), n_m rows.
 *   branches  statistics of the lookahead batch: branch b is stats rows
 *             (branch_offset + b) * n_m .. +n_m-1.
 *   anchor_logit  nullable [n_branch]: scaled anchor logit of each branch's
 *             token at its pivot (a dllm_probe output); if NULL the plan's
 *             br_logp is log p_anchor(c).
 *   scores    nullable [RPS_MAX_BRANCH] out: Eq. 4 score of each branch.
 *   deltas    nullable [RPS_MAX_BRANCH] out: score minus the pivot's [MASK] score.
 * S(c) = -(1/(n_m-1)) sum_{i != pivot} H(p_i^c) + lambda log a_c with
 * a_[MASK] = P^max of the anchor at the pivot.  The winner is the largest
 * margin (lowest branch index on ties); it is committed iff its margin is > 0
 * (a tie with [MASK] abstains). */
dllm_status rps_lookahead_score(const dllm_stats* anchor, const dllm_stats* branches, int32_t branch_offset,
                                int32_t n_m, const rps_plan* plan, const float* anchor_logit, float lambda,
                                float* scores, float* deltas, rps_decision* dec, dllm_stream stream);

/* Commit step (Eq. 1; Algorithm 1's pivot commit, carry-over and standard
 * commit), in this order:
 *  1. if dec is non-NULL and dec->commit: tokens[pivot_pos] = token and the
 *     pivot leaves M; the carried statistics become the winning branch's rows
 *     (branches, branch_offset as in rps_lookahead_score).  If dec is
 *     non-NULL and abstains, the carried statistics become `anchor`'s rows
 *     (when anchor is non-NULL) or stay `base`.
 *  2. if tau >= 0: confidence-aware commit (Eq. 2, third case) on the carried
 *     statistics: every row with P^max >= tau, or the single most confident
 *     row (lowest position on ties) if none; tokens = argmax (Eq. 1).
 *  3. m_pos and base are compacted in place to the remaining masked rows.
 *   tokens [seq] int32 (one sequence), m_pos [n_m] (positions outside
 *   0 .. seq-1 are clamped), base: n_m rows.
 *   n_m_out (device int32) receives the new |M|; committed [n_m] receives the
 *   committed positions (pivot first) and n_committed (device int32) their
 *   count. */
dllm_status rps_commit(int32_t* tokens, int32_t seq, int32_t* m_pos, int32_t n_m, const dllm_stats* base,
                       const rps_decision* dec, const dllm_stats* branches, int32_t branch_offset,
                       const dllm_stats* anchor, float tau, int32_t* n_m_out,
                       int32_t* committed, int32_t* n_committed, dllm_stream stream);

/* Baseline scheduler commit (Section 3, Eq. 2, first two cases; Eq. 1 for
 * the assignment): the masked rows with the k highest confidences
 * P^max = exp(lmax - lse) (SCHED_TOP_CONFIDENCE; k = 1 is the one-token-per-
 * step Default decoder), or with the k lowest entropies H (SCHED_LOW_ENTROPY),
 * ties to the lower row, i.e. the lower position (m_pos ascending).  The
 * third case of Eq. 2, the confidence threshold, is rps_commit with
 * dec = NULL and tau >= 0.
 *   min(k, n_m) rows are committed: tokens[m_pos[j]] = stats->argmax[j];
 *   m_pos and stats are compacted in place to the remaining rows, n_m_out
 *   (device int32) receives the new |M|, committed [n_m] the committed
 *   positions in row order and n_committed (device int32) their count.
 * Errors: DLLM_EINVAL for NULL arguments, a rule outside the enum or k < 1;
 * DLLM_ESHAPE for n_m outside 1 .. RPS_MAX_MASKED or seq < 1. */
enum { SCHED_TOP_CONFIDENCE = 0, SCHED_LOW_ENTROPY = 1 };
dllm_status sched_commit(int32_t* tokens, int32_t seq, int32_t* m_pos, int32_t n_m, const dllm_stats* stats,
                         int32_t rule, int32_t k, int32_t* n_m_out, int32_t* committed, int32_t* n_committed,
                         dllm_stream stream);

#ifdef __cplusplus
}
#endif
#endif /* DLLM_RPS_H */
