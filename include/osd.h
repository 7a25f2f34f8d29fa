/*
 * osd.h -- C ABI of the MI355X (gfx950) library for the vocabulary-wide logits
 * path of online speculative decoding (Liu et al., "Online Speculative
 * Decoding", ICML 2024, arXiv:2310.07177).
 *
 * Two operations (and their fused, sampling and vocabulary-sharded forms):
 *   osd_verify             speculative-sampling verification of k proposed
 *                          tokens against the target (Appendix A.1, Eq. 5;
 *                          Algorithm 1, the verification step);
 *   osd_distill_loss_grad  the distillation divergence of Eq. 3 (forward KL,
 *                          reverse KL, JSD[beta]) and its gradient with
 *                          respect to the draft (student) logits (Section 4.1,
 *                          Eq. 2-4).
 *
 * Conventions shared by every entry point:
 *   - All array arguments are DEVICE pointers owned by the caller; the library
 *     never allocates, frees or synchronises.  Work is enqueued on `stream`
 *     (a hipStream_t passed as void*; NULL is the default stream) and the call
 *     returns without waiting for it.
 *   - Logit arrays are row-major with the vocabulary axis contiguous, in the
 *     dtype given by `dtype` (OSD_F32: IEEE float; OSD_BF16: bfloat16 bit
 *     patterns).  Rows whose byte address and length are multiples of 16 take
 *     the vectorised path; others are accepted and read element by element.
 *   - Host-checkable mistakes (null required pointer, non-positive sizes,
 *     K > OSD_MAX_K, V above osd_max_vocab, NaN or out-of-range scalars, an
 *     unknown enum, a workspace that is too small) return a negative status
 *     and enqueue nothing.  A failed launch returns OSD_ERR_DEVICE.
 *   - Workspaces: the caller allocates `*_workspace_bytes(...)` bytes of
 *     device memory and fills them with zeros ONCE before first use; every
 *     call leaves its workspace zeroed again when its kernels finish.  Calls
 *     that may run concurrently need distinct workspaces.  (A workspace that
 *     is not zero -- fresh from an uninitialised allocation, or shared by
 *     calls in flight on two streams -- is not detected: the outputs are then
 *     wrong, with no status to say so.)
 *   - Thread-safe: apart from osd_verify_noalloc's per-GPU scratch array
 *     (see there), the library holds no mutable global state.
 */
#ifndef OSD_H
#define OSD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    OSD_OK = 0,
    OSD_ERR_INVALID_ARG = -1,
    OSD_ERR_UNSUPPORTED = -2,
    OSD_ERR_DEVICE = -3,
    OSD_ERR_WORKSPACE = -4,
    OSD_ERR_SCRATCH = -5
} osd_status;

typedef enum { OSD_F32 = 0, OSD_BF16 = 1 } osd_dtype;

typedef enum { OSD_FKL = 0, OSD_RKL = 1, OSD_JSD = 2 } osd_divergence;

#define OSD_MAX_K 16

/* Largest vocabulary size the row-resident kernels accept for `dtype`
 * (0 for an unknown dtype). */
int osd_max_vocab(int dtype);

/* Human-readable name of a status code (static storage). */
const char* osd_status_string(int status);

/* Workspace needed by osd_verify for B sequences of up to K proposals. */
size_t osd_verify_workspace_bytes(int B, int K);

/*
 * osd_verify -- one speculative-decoding verification step for B sequences
 * (Appendix A.1: with i rising from 1 to k, accept proposal y_i when
 * u < p(y_i)/q(y_i) and stop at the first rejection; Eq. 5: then draw one
 * more token from norm(max(0, p - q)) at the rejected position, or from p at
 * position k+1 when all k were accepted).
 *
 * target_logits [B, K+1, V]  row i (0-based) holds the target logits that
 *                            score proposal i, row k_b is the bonus row
 * draft_logits  [B, K, V]    row i holds the draft logits proposal i was
 *                            drawn from; may be NULL when temperature == 0
 * draft_tokens  [B, K] int32 the proposals y
 * draft_len     [B] int32    k_b in 1..K (ragged proposals), or NULL for K;
 *                            rows past k_b are padding and are never read
 * u_accept      [B, K] fp32  acceptance uniforms in [0,1); NULL iff T == 0
 * u_resample    [B] fp32     the uniform of the extra token; NULL iff T == 0
 * temperature   T > 0: logits are divided by T before the softmax (the same T
 *               for target and draft); T == 0: greedy verification, proposals
 *               are accepted while they equal the target argmax (lowest index
 *               on ties) and the extra token is that argmax
 * accepted_len  out [B] int32      a_b in 0..k_b, or -1 for an invalid row
 *                                  (k_b outside 1..K, a token outside [0,V),
 *                                  or a row that is read and has no finite
 *                                  logit)
 * out_tokens    out [B, K+1] int32 y_1..y_a, the extra token, then -1
 * reject_mask   out [B, K] uint8   nullable; 1 at i == a_b when a_b < k_b
 *                                  (the error index recorded for
 *                                  distillation), else 0
 * workspace     osd_verify_workspace_bytes(B, K) zero-initialised bytes
 *
 * Decisions are taken in fp32 arithmetic with fp64 scalars; they agree with
 * an exact computation except where u lies within about 1e-7 of p(y)/q(y) or
 * u*Z within about 1e-7 (in probability mass) of a CDF edge.
 */
int osd_verify(const void* target_logits, const void* draft_logits, int dtype,
               int B, int K, int V,
               const int32_t* draft_tokens, const int32_t* draft_len,
               const float* u_accept, const float* u_resample,
               float temperature,
               int32_t* accepted_len, int32_t* out_tokens,
               uint8_t* reject_mask,
               void* workspace, size_t workspace_bytes, void* stream);

/*
 * osd_verify_noalloc -- osd_verify for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same arguments without the workspace, and the same
 * results.  Its scratch is a device array the library holds, one per GPU, of
 * OSD_VERIFY_NOALLOC_SCRATCH_BYTES bytes, kept until the process ends; the
 * call itself allocates nothing.  Calls with
 * osd_verify_workspace_bytes(B, K) > OSD_VERIFY_NOALLOC_SCRATCH_BYTES
 * (about B * (K + 1) > 10000 rows) return OSD_ERR_SCRATCH and enqueue
 * nothing.  Every call on one GPU shares that GPU's array: each call clears
 * the part it needs on its own stream first, and calls that may overlap on
 * one GPU (concurrent streams, other host threads) race and must not be made
 * -- give those osd_verify with separate workspaces.  Other errors as
 * osd_verify.
 */
#define OSD_VERIFY_NOALLOC_SCRATCH_BYTES (4u << 20)
int osd_verify_noalloc(const void* target_logits, const void* draft_logits, int dtype,
                       int B, int K, int V,
                       const int32_t* draft_tokens, const int32_t* draft_len,
                       const float* u_accept, const float* u_resample,
                       float temperature,
                       int32_t* accepted_len, int32_t* out_tokens,
                       uint8_t* reject_mask, void* stream);

/* Workspace needed by osd_distill_loss_grad for B*K rows. */
size_t osd_distill_workspace_bytes(int B, int K);

/*
 * osd_distill_loss_grad -- masked distillation divergence between teacher
 * (target) and student (draft) distributions at temperature tau and its
 * gradient with respect to the student logits (Section 4.1, Eq. 3):
 *   FKL  KL(p || q)                 gradient (q - p) / tau
 *   RKL  KL(q || p)                 gradient q (log q - log p - KL(q||p)) / tau
 *   JSD  beta KL(p || m) + (1-beta) KL(q || m),  m = beta p + (1-beta) q,
 *                                   gradient (1-beta) q (log q - log m - KL(q||m)) / tau
 * with p = softmax(teacher / tau), q = softmax(student / tau), 0 log 0 = 0.
 *
 * teacher_logits  row (b, i) starts at element b*teacher_batch_stride + i*V
 *                 (pass (K+1)*V to distil the first K rows of a verify target)
 * student_logits  row (b, i) starts at element b*student_batch_stride + i*V
 * mask            [B, K] uint8 0/1, or NULL for all ones
 * kind            OSD_FKL / OSD_RKL / OSD_JSD;  beta in [0,1] weights the
 *                 teacher in the JSD mixture;  tau > 0
 * loss_out        out [2] fp32: {sum(mask*D)/sum(mask) (0 if the mask is
 *                 empty), sum(mask*D)} (Eq. 2's batch mean and Eq. 4's sum);
 *                 reduced in a fixed order in fp64, so bitwise deterministic
 * row_loss_out    out [B, K] fp32, nullable: D per row, 0 where mask is 0
 * grad_out        out [B, K, V] in `dtype`, contiguous, nullable: the
 *                 gradient of sum(mask*D); rows with mask 0 are written as 0
 * workspace       osd_distill_workspace_bytes(B, K) zero-initialised bytes
 */
int osd_distill_loss_grad(const void* teacher_logits, int64_t teacher_batch_stride,
                          const void* student_logits, int64_t student_batch_stride,
                          int dtype, int B, int K, int V,
                          const uint8_t* mask, int kind, float beta, float tau,
                          float* loss_out, float* row_loss_out, void* grad_out,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Workspace needed by osd_verify_distill for B sequences of up to K proposals. */
size_t osd_verify_distill_workspace_bytes(int B, int K);

/*
 * osd_verify_distill -- one speculative step's verification and
 * distillation in a single pass over the row pairs (Algorithm 1 verifies the
 * proposals and records, at the error index, what distillation later trains
 * on; Section 4.1 and Eq. 2-4 give the divergence).  The results are those
 * of
 *   osd_verify(target, draft, ..., temperature, ...) and
 *   osd_distill_loss_grad(target, (K+1)*V, draft, K*V, dtype, B, K, V,
 *                         distill_mask, kind, beta, temperature, ...):
 * teacher = target rows 0..K-1, student = draft rows, tau = temperature.
 * Both read the same row pairs; done together they are read once and their
 * softmax normalisers are computed once.
 *
 * Arguments as in osd_verify and osd_distill_loss_grad, with:
 * temperature   T > 0: verification temperature and distillation tau
 * distill_mask  [B, K] uint8 0/1, or NULL for all rows: which rows are
 *               distilled (independent of the verification outcome)
 * workspace     osd_verify_distill_workspace_bytes(B, K) zero-initialised
 *               bytes
 *
 * Verification decisions have the same guarantee as osd_verify's (their
 * masses are formed from the distillation's cached exponents, so a draw that
 * sits within ~1e-7 of a CDF edge may differ from osd_verify's); losses and
 * gradients match osd_distill_loss_grad's within fp32 rounding (the fp64 loss
 * sum is taken in a different fixed order).
 */
int osd_verify_distill(const void* target_logits, const void* draft_logits, int dtype,
                       int B, int K, int V,
                       const int32_t* draft_tokens, const int32_t* draft_len,
                       const float* u_accept, const float* u_resample,
                       float temperature,
                       int32_t* accepted_len, int32_t* out_tokens, uint8_t* reject_mask,
                       const uint8_t* distill_mask, int kind, float beta,
                       float* loss_out, float* row_loss_out, void* grad_out,
                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * osd_verify_distill_rejected -- osd_verify_distill whose distilled rows are
 * the verification's own outcome: the row pair at each sequence's first
 * rejection a_b (the error index at which Algorithm 1 records the target for
 * distillation; Fig. 1: the positions where the draft proposed a wrong
 * token), and no other.  The results are those of
 *   osd_verify(target, draft, ..., temperature, ..., reject_mask, ...) then
 *   osd_distill_loss_grad(target, (K+1)*V, draft, K*V, dtype, B, K, V,
 *                         reject_mask, kind, beta, temperature, ...):
 * loss_out = {sum of D over the distilled rows / their number (0 if none),
 * that sum}; row_loss_out and grad_out hold zeros on every other row.  The
 * rejected row pair is read once: the workgroup that finds a sequence's
 * first rejection draws the correction and distils the row from what it
 * already holds.  (A workgroup that cannot learn in time whether an earlier
 * position rejected distils its row anyway; if it was not the first, the
 * call's last workgroup zeroes that row again.)
 *
 * Arguments as in osd_verify_distill, without distill_mask; reject_mask is
 * nullable.  workspace: osd_verify_distill_workspace_bytes(B, K)
 * zero-initialised bytes (one workspace serves both fused entry points).
 * Decisions, losses and gradients have osd_verify_distill's accuracy.
 */
int osd_verify_distill_rejected(const void* target_logits, const void* draft_logits, int dtype,
                                int B, int K, int V,
                                const int32_t* draft_tokens, const int32_t* draft_len,
                                const float* u_accept, const float* u_resample,
                                float temperature,
                                int32_t* accepted_len, int32_t* out_tokens, uint8_t* reject_mask,
                                int kind, float beta,
                                float* loss_out, float* row_loss_out, void* grad_out,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * osd_verify_tree -- multi-candidate (tree) verification.  The paper applies
 * its online updates to Medusa, which proposes several candidate tokens per
 * position arranged in a tree (Section 5, "OSD and Medusa", Table 4), and
 * states no verification rule for it; this call takes the rule that keeps
 * Appendix A.1's exactness (the emitted tokens follow the target): the
 * children of a node are candidates drawn independently from the draft
 * distribution q at that node and are tested in ascending node order,
 * candidate c accepted when u_c < R(y_c) / q(y_c), with R = p for the first
 * and, after each rejection, R <- norm(max(0, R - q)) (Eq. 5's residual).
 * The walk continues at the first accepted child; where every child is
 * rejected one token is drawn from the last residual max(0, R - q), and at a
 * node without children one token is drawn from p (the bonus token).  The
 * draws are the inverse CDF of osd_verify.  T == 0: the first child whose
 * token is the target argmax (lowest index on ties) is accepted and the
 * argmax is emitted where the walk stops.  A chain (one child per node) is
 * osd_verify.
 *
 * target_logits [B, N, V]  row n: target logits after the prefix ending at
 *                          node n (it scores node n's children; at a node
 *                          without children it is the bonus distribution)
 * draft_logits  [B, N, V]  row n: draft logits node n's children were drawn
 *                          from; not read at leaves; may be NULL at T == 0
 * parent        [B, N] int32  node 0 is the root (the accepted context; its
 *                          entry is ignored); 0 <= parent[n] < n for n >= 1
 * node_tokens   [B, N] int32  the candidate token of node n (node 0 ignored)
 * u_accept      [B, N] fp32  u_accept[b, n] tests node n; NULL iff T == 0
 * u_resample    [B] fp32    the extra token's uniform; NULL iff T == 0
 * accepted_len  out [B] int32  number of accepted candidates, or -1 for an
 *                          invalid tree (a parent or token out of range) or
 *                          a reached row without finite logits
 * out_tokens    out [B, N] int32  accepted tokens, the extra token, then -1
 * path_nodes    out [B, N] int32, nullable: the accepted nodes, then -1
 * workspace     osd_verify_tree_workspace_bytes(B, N) zero-initialised bytes
 *
 * N <= OSD_MAX_TREE_NODES; V up to 32768 (bf16) or 16384 (fp32), otherwise
 * OSD_ERR_UNSUPPORTED.  Every node's rows are read once, whether or not the
 * walk reaches it: one workgroup per (sequence, node), or, for 16-byte
 * aligned rows at T > 0, about one workgroup per CU walking the nodes.
 */
#define OSD_MAX_TREE_NODES 64
size_t osd_verify_tree_workspace_bytes(int B, int N);
int osd_verify_tree(const void* target_logits, const void* draft_logits, int dtype,
                    int B, int N, int V,
                    const int32_t* parent, const int32_t* node_tokens,
                    const float* u_accept, const float* u_resample,
                    float temperature,
                    int32_t* accepted_len, int32_t* out_tokens, int32_t* path_nodes,
                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * osd_sample -- token sampling: the draft model's proposals y ~ q
 * (Algorithm 1) and the mixed sampling y ~ beta p + (1 - beta) q that
 * Section 4.1 uses to generate distillation data (beta weights the target
 * p).  For each row n:
 *   pi_n = beta softmax(p_n / T) + (1 - beta) softmax(q_n / T)
 * and out_tokens[n] is the smallest token id j whose running sum of pi_n
 * (ascending j) exceeds u[n] * sum(pi_n) -- the inverse CDF of osd_verify's
 * extra token.  T == 0 takes the argmax (lowest index on ties) of the row
 * with weight 1.
 *
 * p_logits      [N, V] dtype rows, row n at element offset n * p_row_stride;
 *               not read (may be NULL) when beta == 0
 * q_logits      [N, V] dtype rows, row stride q_row_stride elements; not read
 *               (may be NULL) when beta == 1
 * p_row_stride, q_row_stride  elements between rows, >= V (e.g. V for
 *               [N, V], or (K+1)*V for one position of every sequence of a
 *               [B, K+1, V] tensor)
 * temperature   T > 0 samples; T == 0 needs beta == 0 or beta == 1
 * beta          in [0, 1]
 * u             [N] float uniforms in [0, 1) (unused, may be NULL, at T == 0)
 * out_tokens    out [N] int32: the token, or -1 for a row with weight > 0
 *               that has no finite logit
 *
 * workspace     NULL, or at least osd_sample_workspace_bytes(N) bytes,
 *               16-byte aligned, zero before the first call; every call
 *               leaves it zero.  Calls that may overlap (other streams) need
 *               their own.  With a workspace, one-row sampling (T > 0, beta
 *               0 or 1) of fewer rows than two per CU, rows 16-byte aligned
 *               with 16-byte multiple strides and lengths, splits each row
 *               over several workgroups that exchange two words each through
 *               it; every other call (and every call without one) runs one
 *               workgroup per row.  The token is the same rule's either way;
 *               the two can differ only where u * sum(pi) lies within fp32
 *               rounding of a boundary between tokens.
 *
 * Errors: OSD_ERR_INVALID_ARG for N <= 0, V <= 0, a bad dtype, T < 0, inf
 * or NaN, beta outside [0, 1], T == 0 with 0 < beta < 1, a needed pointer
 * NULL or a row stride < V; OSD_ERR_UNSUPPORTED for V > osd_max_vocab(dtype);
 * OSD_ERR_WORKSPACE for a workspace that is too small or misaligned;
 * OSD_ERR_DEVICE if the launch fails.  Nothing is enqueued on an error.
 * Rows that are 16-byte aligned with 16-byte multiple strides and lengths
 * take 16-byte loads.
 */
size_t osd_sample_workspace_bytes(int N);
int osd_sample(const void* p_logits, int64_t p_row_stride,
               const void* q_logits, int64_t q_row_stride,
               int dtype, int N, int V, float temperature, float beta,
               const float* u, int32_t* out_tokens, void* workspace, size_t workspace_bytes,
               void* stream);

/*
 * Vocabulary-sharded verification.  When the target and draft LM heads are
 * split by vocabulary over G ranks (tensor parallelism), rank g holds columns
 * [v_begin_g, v_begin_g + V_g) of every logit row, and no rank sees a whole
 * row.  The verification of osd_verify (Appendix A.1, Eq. 5) then runs in
 * three phases with one exchange after each:
 *
 *   1. osd_shard_verify_stats   each rank reduces its slice of every row to an
 *                               osd_shard_row_stats record;
 *      -> all-gather of the records over the G ranks, in rank order
 *         (stats_all [G, B, K+1]);
 *   2. osd_shard_verify_mass    every rank merges the G records of each row
 *                               (identically, in rank order), takes the
 *                               acceptance tests, finds the first rejection a_b,
 *                               and sums the extra draw's mass over its own
 *                               slice of row a_b into an osd_shard_mass record;
 *      -> all-gather of those records (mass_all [G, B]);
 *   3. osd_shard_verify_draw    every rank finds which slice holds the point
 *                               u * Z of the whole row's CDF; that rank draws
 *                               the token from its slice.  Every rank writes
 *                               the same accepted_len and reject_mask and an
 *                               out_tokens row whose extra token is -1 except
 *                               on the drawing rank;
 *      -> all-reduce MAX of out_tokens gives every rank the result.
 *
 * The result is osd_verify's on the whole rows: masses are summed in exact
 * fixed point, so how the vocabulary is split changes no decision beyond the
 * fp32 rounding that osd_verify documents.  The slices must partition
 * [0, V) in rank order (v_begin_0 = 0, v_begin_{g+1} = v_begin_g + V_g).
 * Greedy verification (T == 0) needs phases 1-3 too; its phase 2 finds the
 * extra token itself (the argmax) and phase 3 draws nothing.
 *
 * Shard logits are row-major [B, K+1, V_g] (target) and [B, K, V_g] (draft),
 * each row contiguous.  Arguments shared with osd_verify (draft_tokens as
 * global ids, draft_len, u_accept, u_resample, temperature, the outputs) have
 * its meaning.  Records are 8-byte aligned device arrays owned by the caller;
 * rows past k_b are neither read nor written.  No workspace.  Errors:
 * OSD_ERR_INVALID_ARG for a bad dtype, sizes <= 0, K > OSD_MAX_K, G outside
 * 1..OSD_MAX_SHARDS, shard outside [0, G), a slice outside [0, V), T < 0 or
 * not finite, a needed NULL pointer or a misaligned record array;
 * OSD_ERR_UNSUPPORTED for V_g above 65536 (bf16) or 32768 (fp32) -- a rank
 * holds its slice in registers -- or V > 524288 (the whole row's
 * fixed-point mass must stay below 2^63); OSD_ERR_DEVICE for a failed
 * launch.  Nothing is enqueued on an error.
 */
#define OSD_MAX_SHARDS 64

/* One rank's reduction of its slice of one logit row pair (40 bytes). */
typedef struct {
    double s_target;  /* T > 0: sum over the slice of 2^(t_j log2(e)/T - k_target) */
    double s_draft;   /* T > 0: the same for the draft row (proposal rows only)   */
    float k_target;   /* T > 0: whole-number shift >= max_j t_j log2(e)/T, -inf if
                         the slice has no finite logit; T == 0: max_j t_j      */
    float k_draft;    /* T > 0: the draft row's shift                           */
    float t_y, d_y;   /* T > 0: target and draft logits of the proposal y_i when
                         this slice holds it                                   */
    int32_t argmax;   /* T == 0: global id of the slice's largest target logit
                         (lowest id on ties), -1 if the slice has none           */
    int32_t flags;    /* bit 0: the slice holds y_i; bit 1: y_i lies outside [0, V) */
} osd_shard_row_stats;

/* One rank's part of a sequence's extra draw (48 bytes). */
typedef struct {
    uint64_t z;        /* mass of max(0, p - q) (of p at the bonus row) over the
                          slice, 2^-44 fixed point in units of the target row's
                          sum of exponentials                                  */
    uint64_t z_p;      /* mass of p over the slice, same units (used should the
                          whole row's residual mass round to 0)                 */
    double s_target, s_draft;  /* merged sums of row a_b (whole row)           */
    float k_target, k_draft;   /* their shifts                                 */
    int32_t accepted;  /* a_b, or -1 for an invalid sequence                   */
    int32_t token;     /* T == 0: the extra token (global id); else -1         */
} osd_shard_mass;

int osd_shard_verify_stats(const void* target_shard, const void* draft_shard, int dtype,
                           int B, int K, int V_shard, int v_begin, int V,
                           const int32_t* draft_tokens, const int32_t* draft_len,
                           float temperature,
                           osd_shard_row_stats* stats, /* out [B, K+1] */
                           void* stream);

int osd_shard_verify_mass(const void* target_shard, const void* draft_shard, int dtype,
                          int B, int K, int V_shard, int G,
                          const int32_t* draft_tokens, const int32_t* draft_len,
                          const float* u_accept, float temperature,
                          const osd_shard_row_stats* stats_all, /* [G, B, K+1] */
                          osd_shard_mass* mass,                 /* out [B]      */
                          void* stream);

int osd_shard_verify_draw(const void* target_shard, const void* draft_shard, int dtype,
                          int B, int K, int V_shard, int v_begin, int G, int shard,
                          const int32_t* draft_tokens, const int32_t* draft_len,
                          const float* u_resample, float temperature,
                          const osd_shard_mass* mass_all,       /* [G, B] */
                          int32_t* accepted_len, int32_t* out_tokens,
                          uint8_t* reject_mask, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OSD_H */
