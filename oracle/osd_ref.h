/*
 * osd_ref.h -- plain fp64 CPU oracle for the vocabulary-wide logits path of
 * online speculative decoding (Liu et al., "Online Speculative Decoding",
 * ICML 2024, arXiv:2310.07177).
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists so that the GPU path can be
 * checked against a slow, obviously correct restatement of the paper.  Only
 * the test-suite, the smoke check and the CPU-baseline leg of the benchmark
 * may load it.  It shares no source, header, table or helper with the HIP
 * library; it is built with the host compiler alone.
 *
 * All arithmetic is IEEE fp64 in plain sequential loops.  Inputs are read as
 * fp32, bf16 (raw 16-bit patterns) or fp64 (fp64 is an oracle-only input type
 * used by the finite-difference and enumeration pins), and converted exactly
 * to fp64.  Every pointer is a HOST pointer owned by the caller.  Layouts are
 * row-major with the vocabulary axis contiguous.
 *
 * Return value: 0 on success, -1 for an argument the caller got wrong.
 */
#ifndef OSD_REF_H
#define OSD_REF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { OSD_REF_F32 = 0, OSD_REF_BF16 = 1, OSD_REF_F64 = 2 };
enum { OSD_REF_FKL = 0, OSD_REF_RKL = 1, OSD_REF_JSD = 2 };

/*
 * Speculative-sampling verification (Appendix A.1 and its Eq. 5; Algorithm 1,
 * the "determine number of accepted tokens and sample one more" step).
 *
 * target        [B, K+1, V]  row i is p(. | x, y_<=i) before temperature
 * draft         [B, K,   V]  row i is q(. | x, y_<=i) before temperature
 * draft_tokens  [B, K]       y_{i+1}, proposed from draft row i
 * draft_len     [B] or NULL  k_b in 1..K (ragged proposals); NULL means all K
 * u_accept      [B, K]       acceptance uniforms in [0,1); unused when T == 0
 * u_resample    [B]          one uniform per sequence for the final sample
 * temperature   T > 0 samples at softmax(z/T); T == 0 is greedy verification
 * accepted_len  out [B]      a_b, or -1 for an invalid row
 * out_tokens    out [B, K+1] y_1..y_a, then the correction/bonus token, then -1
 * reject_mask   out [B, K]   nullable; 1 at i == a_b when a_b < k_b
 * margin_accept out [B, K]   nullable; |u - p(y)/q(y)| for every acceptance
 *                            test actually evaluated, NaN elsewhere
 * margin_cdf    out [B]      nullable; distance, in absolute probability
 *                            mass (not divided by Z), from u*Z to the nearer
 *                            edge of the chosen token's CDF interval (NaN for
 *                            greedy and invalid rows)
 * z_fallback    out [B]      nullable; 1 where a rejection met Z == 0 and the
 *                            sample fell back to p
 */
int osd_ref_verify(const void* target, const void* draft, int dtype,
                   int B, int K, int V,
                   const int32_t* draft_tokens, const int32_t* draft_len,
                   const float* u_accept, const float* u_resample,
                   float temperature,
                   int32_t* accepted_len, int32_t* out_tokens,
                   uint8_t* reject_mask,
                   double* margin_accept, double* margin_cdf,
                   int32_t* z_fallback);

/*
 * Distillation divergence and its gradient with respect to the student
 * (draft) logits (Section 4.1, Eq. 2-4).
 *
 * teacher  [B, K, V] with batch stride teacher_batch_stride (elements)
 * student  [B, K, V] with batch stride student_batch_stride (elements)
 * mask     [B, K] 0/1 or NULL (all ones)
 * kind     OSD_REF_FKL / OSD_REF_RKL / OSD_REF_JSD; beta weights the teacher
 *          in the JSD mixture; tau > 0 is the softmax temperature
 * loss_out out [2]       {masked mean, masked sum} of the per-row divergence
 * row_loss out [B, K]    nullable; per-row divergence, 0 where mask is 0
 * grad     out [B, K, V] nullable; fp64 d(sum_n mask_n D_n)/d student logits
 */
int osd_ref_distill_loss_grad(const void* teacher, int64_t teacher_batch_stride,
                              const void* student, int64_t student_batch_stride,
                              int dtype, int B, int K, int V,
                              const uint8_t* mask, int kind,
                              double beta, double tau,
                              double* loss_out, double* row_loss,
                              double* grad);

/*
 * Multi-candidate (tree) verification (Section 5, "OSD and Medusa": several
 * candidates per position; the rule is the recursive form of Appendix A.1's
 * test, see osd_ref.cpp).
 *
 * target       [B, N, V]  row n: target logits after the prefix ending at
 *                         node n (it scores node n's children; at a node
 *                         without children it is the bonus distribution)
 * draft        [B, N, V]  row n: draft logits node n's children were drawn
 *                         from (i.i.d.); unused at T == 0 and at leaves
 * parent       [B, N]     parent node of each node; node 0 is the root
 *                         (its entry is ignored); 0 <= parent[n] < n
 * node_tokens  [B, N]     the candidate token of each node (node 0 ignored)
 * u_accept     [B, N]     the uniform that tests node n; u_resample [B]
 * accepted_len out [B]    number of accepted candidates (path length), -1
 *                         for an invalid tree or a reached row without a
 *                         finite logit
 * out_tokens   out [B, N] the accepted candidates' tokens, the extra token,
 *                         then -1
 * path_nodes   out [B, N] nullable: the accepted nodes, then -1
 * margin_accept out [B, N] nullable: |u - ratio| of every tested candidate
 * margin_cdf   out [B]    nullable: the extra draw's CDF margin (absolute)
 * z_fallback   out [B]    nullable: 1 where a residual had no mass
 */
int osd_ref_verify_tree(const void* target, const void* draft, int dtype,
                        int B, int N, int V,
                        const int32_t* parent, const int32_t* node_tokens,
                        const float* u_accept, const float* u_resample,
                        float temperature, int32_t* accepted_len,
                        int32_t* out_tokens, int32_t* path_nodes,
                        double* margin_accept, double* margin_cdf,
                        int32_t* z_fallback);

/*
 * Token sampling: the draft's proposals y ~ q (Algorithm 1) and mixed
 * sampling y ~ beta p + (1 - beta) q (Section 4.1).
 *
 * p, q        [N, V] rows, row strides p_stride, q_stride (elements, >= V);
 *             a row set whose weight is 0 (p when beta == 0, q when
 *             beta == 1) is not read and may be NULL
 * temperature T > 0: pi = beta softmax(p_n / T) + (1 - beta) softmax(q_n / T),
 *             token = smallest j whose running sum (ascending j) exceeds
 *             u[n] * Z, Z = sum pi; T == 0: argmax of the row with weight 1
 *             (lowest index on ties), beta must then be 0 or 1
 * u           [N] in [0, 1); unused (may be NULL) when T == 0
 * out         [N] the token, -1 when a row with non-zero weight has no
 *             finite logit
 * margin      [N] nullable; distance in probability mass from u*Z to the
 *             nearer edge of the chosen token's interval (NaN for greedy and
 *             invalid rows)
 */
int osd_ref_sample(const void* p, int64_t p_stride, const void* q, int64_t q_stride,
                   int dtype, int N, int V, float temperature, double beta,
                   const float* u, int32_t* out, double* margin);

/* Round fp64 values to bf16 bit patterns, round-to-nearest-even, directly
 * (no intermediate fp32 rounding). */
void osd_ref_round_bf16(const double* x, uint16_t* out, int64_t n);

/* flag[i] = 1 where x[i] lies within rel*|x[i]| of a bf16 rounding midpoint,
 * i.e. where a correctly computed fp32 value could legitimately round to
 * either neighbouring bf16 value. */
void osd_ref_bf16_midpoint_flags(const double* x, uint8_t* flag, int64_t n,
                                 double rel);

#ifdef __cplusplus
}
#endif

#endif /* OSD_REF_H */
