/*
 * osd_ref.cpp -- plain fp64 CPU oracle (test infrastructure only).
 *
 * Restates, loop by loop, what the verification and distillation steps of
 * online speculative decoding compute (arXiv:2310.07177).  Nothing here is
 * blocked, fused or reordered: each function follows the definition it
 * cites, so that a reader can check it against the paper by eye.  It shares
 * no code with the HIP library.
 *
 * Readings of points the paper leaves open are stated where they are used:
 *   - acceptance is "u < p(y)/q(y)" with u in [0,1) (Appendix A.1 writes
 *     u <= p/q; the two agree except on a set of u of measure zero);
 *   - the extra token is drawn by inverse CDF over ascending token id with a
 *     strict ">" so that zero-mass tokens are never drawn (Eq. 5 names the
 *     distribution, not the sampler);
 *   - the same temperature scales target and draft logits (Section 4.1);
 *   - temperature 0 means greedy verification: accept while the draft token
 *     equals the target argmax (lowest index on ties), emit that argmax;
 *   - the gradient is the exact derivative with respect to the raw student
 *     logits, including the 1/tau factor of the temperature softmax.
 */
#include "osd_ref.h"

#include <cmath>
#include <cstring>
#include <limits>
#include <vector>

namespace {

const double kInf = std::numeric_limits<double>::infinity();
const double kNaN = std::numeric_limits<double>::quiet_NaN();

/* One logit, converted exactly to fp64. */
double load_logit(const void* base, int dtype, int64_t idx) {
    if (dtype == OSD_REF_F32) {
        return (double)((const float*)base)[idx];
    }
    if (dtype == OSD_REF_BF16) {
        uint32_t bits = (uint32_t)((const uint16_t*)base)[idx] << 16;
        float f;
        std::memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
    return ((const double*)base)[idx];
}

/* A row of V logits starting at element offset `off`. */
std::vector<double> load_row(const void* base, int dtype, int64_t off, int V) {
    std::vector<double> z((size_t)V);
    for (int j = 0; j < V; ++j) z[(size_t)j] = load_logit(base, dtype, off + j);
    return z;
}

/*
 * Temperature softmax, softmax(z / T), and its log (Section 4.1 uses a
 * tunable temperature on the logits before the softmax).  The maximum is
 * subtracted before exponentiating; that leaves the value unchanged in exact
 * arithmetic.  Returns false when the row has no finite logit (every
 * probability would be 0/0).
 */
bool temperature_softmax(const std::vector<double>& z, double T,
                         std::vector<double>& prob,
                         std::vector<double>& logprob) {
    const size_t V = z.size();
    double m = -kInf;
    for (size_t j = 0; j < V; ++j) {
        double x = z[j] / T;
        if (x > m) m = x;
    }
    if (!(m > -kInf) || !std::isfinite(m)) return false;
    double s = 0.0;
    for (size_t j = 0; j < V; ++j) s += std::exp(z[j] / T - m);
    double lse = m + std::log(s);
    prob.assign(V, 0.0);
    logprob.assign(V, 0.0);
    for (size_t j = 0; j < V; ++j) {
        prob[j] = std::exp(z[j] / T - m) / s;
        logprob[j] = z[j] / T - lse;
    }
    return true;
}

/*
 * Inverse-CDF draw from the unnormalised weights r (all >= 0) with total Z:
 * the smallest j whose running sum C_j exceeds c = u * Z, walking ascending
 * token ids.  If rounding leaves c at or beyond the last running sum, the
 * last token with r_j > 0 is taken.  *margin receives
 * min(C_j - c, c - C_{j-1}), the distance from c to the nearer edge of the
 * chosen interval in absolute probability mass (r_j = max(0, p_j - q_j) or
 * p_j, so Z <= 1), NOT divided by Z: a kernel that forms these masses in
 * fp32 errs by an amount of order 1e-7 in absolute mass whatever Z is, so
 * the absolute distance is the one that says whether such a kernel can land
 * on the other side of an edge.
 */
int inverse_cdf(const std::vector<double>& r, double Z, float u,
                double* margin) {
    const double c = (double)u * Z;
    double C = 0.0;
    for (size_t j = 0; j < r.size(); ++j) {
        double prev = C;
        C += r[j];
        if (C > c) {
            double a = C - c, b = c - prev;
            *margin = a < b ? a : b;
            return (int)j;
        }
    }
    for (size_t j = r.size(); j-- > 0;) {
        if (r[j] > 0.0) {
            *margin = 0.0;
            return (int)j;
        }
    }
    *margin = 0.0;
    return -1;
}

/* Greedy reading: the target argmax, lowest index on ties.  -1 if the row has
 * no finite logit. */
int row_argmax(const std::vector<double>& z) {
    int best = -1;
    double bv = -kInf;
    for (size_t j = 0; j < z.size(); ++j) {
        if (z[j] > bv) {
            bv = z[j];
            best = (int)j;
        }
    }
    if (best >= 0 && !std::isfinite(bv)) return -1;
    return best;
}

void mark_invalid(int b, int K, int32_t* accepted_len, int32_t* out_tokens,
                  uint8_t* reject_mask) {
    accepted_len[b] = -1;
    for (int i = 0; i <= K; ++i) out_tokens[(size_t)b * (K + 1) + i] = -1;
    if (reject_mask)
        for (int i = 0; i < K; ++i) reject_mask[(size_t)b * K + i] = 0;
}

}  // namespace

extern "C" int osd_ref_verify(const void* target, const void* draft, int dtype,
                              int B, int K, int V,
                              const int32_t* draft_tokens,
                              const int32_t* draft_len,
                              const float* u_accept, const float* u_resample,
                              float temperature, int32_t* accepted_len,
                              int32_t* out_tokens, uint8_t* reject_mask,
                              double* margin_accept, double* margin_cdf,
                              int32_t* z_fallback) {
    if (!target || !draft_tokens || !accepted_len || !out_tokens) return -1;
    if (B <= 0 || K <= 0 || V <= 0) return -1;
    if (dtype != OSD_REF_F32 && dtype != OSD_REF_BF16 && dtype != OSD_REF_F64)
        return -1;
    if (!(temperature >= 0.0f) || std::isinf(temperature)) return -1;
    const bool greedy = temperature == 0.0f;
    if (!greedy && (!draft || !u_accept || !u_resample)) return -1;
    const double T = (double)temperature;
    const int64_t tstride = (int64_t)(K + 1) * V, dstride = (int64_t)K * V;

    for (int b = 0; b < B; ++b) {
        if (margin_accept)
            for (int i = 0; i < K; ++i) margin_accept[(size_t)b * K + i] = kNaN;
        if (margin_cdf) margin_cdf[b] = kNaN;
        if (z_fallback) z_fallback[b] = 0;
        if (reject_mask)
            for (int i = 0; i < K; ++i) reject_mask[(size_t)b * K + i] = 0;

        /* Ragged proposals: k_b tokens were proposed; target row k_b is the
         * bonus row.  Anything past k_b is padding and is never read. */
        const int kb = draft_len ? draft_len[b] : K;
        if (kb < 1 || kb > K) {
            mark_invalid(b, K, accepted_len, out_tokens, reject_mask);
            continue;
        }
        const int32_t* y = draft_tokens + (size_t)b * K;
        bool ok = true;
        for (int i = 0; i < kb; ++i)
            if (y[i] < 0 || y[i] >= V) ok = false;
        if (!ok) {
            mark_invalid(b, K, accepted_len, out_tokens, reject_mask);
            continue;
        }

        int a = kb;       /* number of accepted draft tokens */
        int extra = -1;   /* the one additional token */

        if (greedy) {
            /* Accept while the proposal equals the target argmax; the extra
             * token is the target argmax at the first mismatch, or at the
             * bonus row. */
            for (int i = 0; i <= kb && ok; ++i) {
                std::vector<double> t =
                    load_row(target, dtype, b * tstride + (int64_t)i * V, V);
                int g = row_argmax(t);
                if (g < 0) {
                    ok = false;
                    break;
                }
                if (i == kb || y[i] != g) {
                    a = i;
                    extra = g;
                    break;
                }
            }
        } else {
            /* Appendix A.1: with i rising from 1 to k, accept y_i if
             * u < p(y_i)/q(y_i); otherwise stop.  Rows are 0-based here:
             * row i scores proposal y[i]. */
            std::vector<double> P, logP, Q, logQ;
            bool rejected = false;
            for (int i = 0; i < kb; ++i) {
                std::vector<double> t =
                    load_row(target, dtype, b * tstride + (int64_t)i * V, V);
                std::vector<double> d =
                    load_row(draft, dtype, b * dstride + (int64_t)i * V, V);
                if (!temperature_softmax(t, T, P, logP) ||
                    !temperature_softmax(d, T, Q, logQ)) {
                    ok = false;
                    break;
                }
                const double py = P[(size_t)y[i]], qy = Q[(size_t)y[i]];
                double ratio;
                if (qy > 0.0)
                    ratio = py / qy;
                else
                    ratio = py > 0.0 ? kInf : 0.0;
                const float u = u_accept[(size_t)b * K + i];
                if (margin_accept)
                    margin_accept[(size_t)b * K + i] = std::fabs((double)u - ratio);
                if (!((double)u < ratio)) {
                    a = i;
                    rejected = true;
                    break;
                }
            }
            if (ok) {
                /* Eq. 5: after a rejection at a the extra token comes from
                 * norm(max(0, p - q)) at row a; after k_b acceptances it
                 * comes from p at the bonus row k_b. */
                std::vector<double> r((size_t)V);
                double Z = 0.0;
                if (rejected) {
                    for (int j = 0; j < V; ++j) {
                        double diff = P[(size_t)j] - Q[(size_t)j];
                        r[(size_t)j] = diff > 0.0 ? diff : 0.0;
                    }
                    for (int j = 0; j < V; ++j) Z += r[(size_t)j];
                    if (!(Z > 0.0)) {
                        /* Exact arithmetic rules this out (a rejection needs
                         * p(y) < q(y), so some other p_j > q_j); under
                         * rounding the draw falls back to p. */
                        r = P;
                        Z = 0.0;
                        for (int j = 0; j < V; ++j) Z += r[(size_t)j];
                        if (z_fallback) z_fallback[b] = 1;
                    }
                } else {
                    std::vector<double> t =
                        load_row(target, dtype, b * tstride + (int64_t)kb * V, V);
                    if (!temperature_softmax(t, T, P, logP)) {
                        ok = false;
                    } else {
                        r = P;
                        for (int j = 0; j < V; ++j) Z += r[(size_t)j];
                    }
                }
                if (ok) {
                    double margin = 0.0;
                    extra = inverse_cdf(r, Z, u_resample[b], &margin);
                    if (margin_cdf) margin_cdf[b] = margin;
                    if (extra < 0) ok = false;
                }
            }
        }

        if (!ok) {
            mark_invalid(b, K, accepted_len, out_tokens, reject_mask);
            if (margin_cdf) margin_cdf[b] = kNaN;
            continue;
        }
        /* Emit y_1..y_a and the extra token (Algorithm 1: a + 1 new tokens);
         * record the error index a when a proposal was rejected. */
        accepted_len[b] = a;
        int32_t* out = out_tokens + (size_t)b * (K + 1);
        for (int i = 0; i <= K; ++i) out[i] = -1;
        for (int i = 0; i < a; ++i) out[i] = y[i];
        out[a] = extra;
        if (reject_mask && a < kb) reject_mask[(size_t)b * K + a] = 1;
    }
    return 0;
}

extern "C" int osd_ref_distill_loss_grad(const void* teacher,
                                         int64_t teacher_batch_stride,
                                         const void* student,
                                         int64_t student_batch_stride,
                                         int dtype, int B, int K, int V,
                                         const uint8_t* mask, int kind,
                                         double beta, double tau,
                                         double* loss_out, double* row_loss,
                                         double* grad) {
    if (!teacher || !student || !loss_out) return -1;
    if (B <= 0 || K <= 0 || V <= 0) return -1;
    if (dtype != OSD_REF_F32 && dtype != OSD_REF_BF16 && dtype != OSD_REF_F64)
        return -1;
    if (kind != OSD_REF_FKL && kind != OSD_REF_RKL && kind != OSD_REF_JSD)
        return -1;
    if (!(tau > 0.0) || std::isinf(tau)) return -1;
    if (!(beta >= 0.0 && beta <= 1.0)) return -1;

    double loss_sum = 0.0, count = 0.0;
    std::vector<double> P, logP, Q, logQ;
    for (int b = 0; b < B; ++b) {
        for (int i = 0; i < K; ++i) {
            const size_t n = (size_t)b * K + i;
            double* g = grad ? grad + n * (size_t)V : nullptr;
            const bool on = mask ? mask[n] != 0 : true;
            if (!on) {
                if (row_loss) row_loss[n] = 0.0;
                if (g)
                    for (int j = 0; j < V; ++j) g[j] = 0.0;
                continue;
            }
            std::vector<double> t = load_row(
                teacher, dtype, b * teacher_batch_stride + (int64_t)i * V, V);
            std::vector<double> s = load_row(
                student, dtype, b * student_batch_stride + (int64_t)i * V, V);
            double D = kNaN;
            bool ok = temperature_softmax(t, tau, P, logP) &&
                      temperature_softmax(s, tau, Q, logQ);
            if (ok && kind == OSD_REF_FKL) {
                /* Eq. 3: KL(p || q) = sum_j p_j (log p_j - log q_j), with
                 * 0 log 0 = 0.  d/ds_j = (q_j - p_j) / tau. */
                D = 0.0;
                for (int j = 0; j < V; ++j)
                    if (P[(size_t)j] > 0.0)
                        D += P[(size_t)j] * (logP[(size_t)j] - logQ[(size_t)j]);
                if (g)
                    for (int j = 0; j < V; ++j)
                        g[j] = (Q[(size_t)j] - P[(size_t)j]) / tau;
            } else if (ok && kind == OSD_REF_RKL) {
                /* Eq. 3: KL(q || p).  d/ds_j = q_j (log q_j - log p_j - KL) / tau. */
                D = 0.0;
                for (int j = 0; j < V; ++j)
                    if (Q[(size_t)j] > 0.0)
                        D += Q[(size_t)j] * (logQ[(size_t)j] - logP[(size_t)j]);
                if (g)
                    for (int j = 0; j < V; ++j)
                        g[j] = Q[(size_t)j] > 0.0
                                   ? Q[(size_t)j] *
                                         (logQ[(size_t)j] - logP[(size_t)j] - D) /
                                         tau
                                   : 0.0;
            } else if (ok) {
                /* Eq. 3: JSD[beta] = beta KL(p || m) + (1-beta) KL(q || m) with
                 * m = beta p + (1-beta) q (beta weights the teacher).
                 * d/ds_j = (1-beta) q_j (log q_j - log m_j - KL(q || m)) / tau.
                 * A term whose weight is 0 is left out rather than multiplied
                 * by 0: at beta = 1 KL(q || m) = KL(q || p) may be infinite,
                 * at beta = 0 KL(p || m) = KL(p || q) may be, and 0 * inf is
                 * not the 0 the printed formula means.  With that reading
                 * JSD is identically 0 at both ends (m equals the one
                 * distribution left in the sum). */
                const double wp = beta, wq = 1.0 - beta;
                std::vector<double> logM((size_t)V);
                for (int j = 0; j < V; ++j)
                    logM[(size_t)j] =
                        std::log(wp * P[(size_t)j] + wq * Q[(size_t)j]);
                double kl_pm = 0.0, kl_qm = 0.0;
                if (wp > 0.0)
                    for (int j = 0; j < V; ++j)
                        if (P[(size_t)j] > 0.0)
                            kl_pm += P[(size_t)j] * (logP[(size_t)j] - logM[(size_t)j]);
                if (wq > 0.0)
                    for (int j = 0; j < V; ++j)
                        if (Q[(size_t)j] > 0.0)
                            kl_qm += Q[(size_t)j] * (logQ[(size_t)j] - logM[(size_t)j]);
                D = 0.0;
                if (wp > 0.0) D += wp * kl_pm;
                if (wq > 0.0) D += wq * kl_qm;
                if (g)
                    for (int j = 0; j < V; ++j)
                        g[j] = (wq > 0.0 && Q[(size_t)j] > 0.0)
                                   ? wq * Q[(size_t)j] *
                                         (logQ[(size_t)j] - logM[(size_t)j] - kl_qm) /
                                         tau
                                   : 0.0;
            } else if (g) {
                for (int j = 0; j < V; ++j) g[j] = kNaN;
            }
            if (row_loss) row_loss[n] = D;
            /* Eq. 2 averages over the batch; Eq. 4 sums over positions: the
             * loss is reported as both, the gradient is of the sum. */
            loss_sum += D;
            count += 1.0;
        }
    }
    loss_out[0] = count > 0.0 ? loss_sum / count : 0.0;
    loss_out[1] = loss_sum;
    return 0;
}

/*
 * Multi-candidate (tree) verification.  The paper applies online updates to
 * Medusa, which proposes several candidate tokens per position arranged in a
 * tree, and states no verification rule for it (Section 5, "OSD and
 * Medusa", Table 4).  The rule used here keeps the exactness that the
 * paper's verification has (the emitted tokens follow the target): the
 * children of a node are candidates drawn independently from the draft
 * distribution q at that node, and they are tested one after another by the
 * same accept/resample step as Appendix A.1, where after each rejection the
 * distribution the next candidate is tested against becomes the residual
 * norm(max(0, p - q)) of Eq. 5.  The first accepted candidate is emitted and
 * the walk continues at its node; when every child of a node is rejected,
 * one token is drawn from the last residual, and at a node without children
 * one token is drawn from p (the bonus token).  At T == 0 the first child
 * whose token is the target argmax is accepted, and the argmax is emitted
 * where the walk stops.
 */
extern "C" int osd_ref_verify_tree(const void* target, const void* draft, int dtype,
                                   int B, int N, int V,
                                   const int32_t* parent, const int32_t* node_tokens,
                                   const float* u_accept, const float* u_resample,
                                   float temperature, int32_t* accepted_len,
                                   int32_t* out_tokens, int32_t* path_nodes,
                                   double* margin_accept, double* margin_cdf,
                                   int32_t* z_fallback) {
    if (!target || !parent || !node_tokens || !accepted_len || !out_tokens) return -1;
    if (B <= 0 || N <= 0 || V <= 0) return -1;
    if (dtype != OSD_REF_F32 && dtype != OSD_REF_BF16 && dtype != OSD_REF_F64)
        return -1;
    if (!(temperature >= 0.0f) || std::isinf(temperature)) return -1;
    const bool greedy = temperature == 0.0f;
    if (!greedy && (!draft || !u_accept || !u_resample)) return -1;
    const double T = (double)temperature;
    const int64_t stride = (int64_t)N * V;

    for (int b = 0; b < B; ++b) {
        int32_t* out = out_tokens + (size_t)b * N;
        int32_t* pn = path_nodes ? path_nodes + (size_t)b * N : nullptr;
        for (int n = 0; n < N; ++n) {
            out[n] = -1;
            if (pn) pn[n] = -1;
            if (margin_accept) margin_accept[(size_t)b * N + n] = kNaN;
        }
        if (margin_cdf) margin_cdf[b] = kNaN;
        if (z_fallback) z_fallback[b] = 0;
        accepted_len[b] = -1;

        /* The tree: node 0 is the root (the accepted context); every other
         * node names an earlier node as its parent and carries a token. */
        const int32_t* par = parent + (size_t)b * N;
        const int32_t* tok = node_tokens + (size_t)b * N;
        bool ok = true;
        for (int n = 1; n < N; ++n)
            if (par[n] < 0 || par[n] >= n || tok[n] < 0 || tok[n] >= V) ok = false;
        if (!ok) continue;

        std::vector<int> path;
        int extra = -1;
        int v = 0;
        for (;;) {
            std::vector<int> kids;
            for (int n = v + 1; n < N; ++n)
                if (par[n] == v) kids.push_back(n);
            std::vector<double> t = load_row(target, dtype, b * stride + (int64_t)v * V, V);
            if (greedy) {
                const int g = row_argmax(t);
                if (g < 0) {
                    ok = false;
                    break;
                }
                int next = -1;
                for (int c : kids)
                    if (tok[c] == g) {
                        next = c;
                        break;
                    }
                if (next < 0) {
                    extra = g;
                    break;
                }
                path.push_back(next);
                v = next;
                continue;
            }
            std::vector<double> P, logP;
            if (!temperature_softmax(t, T, P, logP)) {
                ok = false;
                break;
            }
            if (kids.empty()) {
                /* no candidate below this node: the bonus token from p */
                double Z = 0.0;
                for (int j = 0; j < V; ++j) Z += P[(size_t)j];
                double m = 0.0;
                extra = inverse_cdf(P, Z, u_resample[b], &m);
                if (margin_cdf) margin_cdf[b] = m;
                if (extra < 0) ok = false;
                break;
            }
            std::vector<double> Q, logQ;
            std::vector<double> d = load_row(draft, dtype, b * stride + (int64_t)v * V, V);
            if (!temperature_softmax(d, T, Q, logQ)) {
                ok = false;
                break;
            }
            /* Candidates in order; R is the distribution the next one is
             * tested against: p, then after each rejection the normalised
             * residual max(0, R - q). */
            std::vector<double> R = P;
            /* the last rejection's residual max(0, R - q) before it is
             * normalised, and its total: the extra token is drawn from it,
             * so that its CDF margin is in the same units as Eq. 5's single
             * residual (one candidate per node gives exactly that draw) */
            std::vector<double> last_r;
            double last_Z = 0.0;
            int next = -1;
            for (int c : kids) {
                const double rc = R[(size_t)tok[c]], qc = Q[(size_t)tok[c]];
                double ratio;
                if (qc > 0.0)
                    ratio = rc / qc;
                else
                    ratio = rc > 0.0 ? kInf : 0.0;
                const float u = u_accept[(size_t)b * N + c];
                if (margin_accept) margin_accept[(size_t)b * N + c] = std::fabs((double)u - ratio);
                if ((double)u < ratio) {
                    next = c;
                    break;
                }
                std::vector<double> r((size_t)V);
                double Z = 0.0;
                for (int j = 0; j < V; ++j) {
                    const double diff = R[(size_t)j] - Q[(size_t)j];
                    r[(size_t)j] = diff > 0.0 ? diff : 0.0;
                }
                for (int j = 0; j < V; ++j) Z += r[(size_t)j];
                if (!(Z > 0.0)) {
                    /* impossible in exact arithmetic (a rejection needs
                     * R(y) < q(y)); under rounding R is kept */
                    if (z_fallback) z_fallback[b] = 1;
                    last_r.clear();
                    continue;
                }
                last_r = r;
                last_Z = Z;
                for (int j = 0; j < V; ++j) R[(size_t)j] = r[(size_t)j] / Z;
            }
            if (next >= 0) {
                path.push_back(next);
                v = next;
                continue;
            }
            /* every candidate rejected: one token from the last residual */
            if (last_r.empty()) {
                last_r = R;
                last_Z = 0.0;
                for (int j = 0; j < V; ++j) last_Z += R[(size_t)j];
            }
            double m = 0.0;
            extra = inverse_cdf(last_r, last_Z, u_resample[b], &m);
            if (margin_cdf) margin_cdf[b] = m;
            if (extra < 0) ok = false;
            break;
        }
        if (!ok) {
            for (int n = 0; n < N; ++n) {
                out[n] = -1;
                if (pn) pn[n] = -1;
            }
            if (margin_cdf) margin_cdf[b] = kNaN;
            continue;
        }
        accepted_len[b] = (int32_t)path.size();
        for (size_t i = 0; i < path.size(); ++i) {
            out[i] = tok[path[i]];
            if (pn) pn[i] = path[i];
        }
        out[path.size()] = extra;
    }
    return 0;
}

/*
 * Token sampling: the draft's proposals y ~ q (Algorithm 1) and the mixed
 * sampling y ~ beta p + (1 - beta) q of Section 4.1.  Per row n the
 * distribution is pi = beta softmax(p_n / T) + (1 - beta) softmax(q_n / T)
 * (a row whose weight is 0 is not read), and the token is drawn by the same
 * inverse CDF as the verification's extra token: ascending token ids, the
 * first running sum strictly above u * Z.  T == 0 takes the argmax of the
 * one row with weight 1.
 */
extern "C" int osd_ref_sample(const void* p, int64_t p_stride, const void* q, int64_t q_stride,
                              int dtype, int N, int V, float temperature, double beta,
                              const float* u, int32_t* out, double* margin) {
    if (N <= 0 || V <= 0 || !out) return -1;
    if (!(temperature >= 0.0f) || !(beta >= 0.0 && beta <= 1.0)) return -1;
    const bool use_p = beta > 0.0, use_q = beta < 1.0;
    if ((use_p && (!p || p_stride < V)) || (use_q && (!q || q_stride < V))) return -1;
    const bool greedy = temperature == 0.0f;
    if (greedy && use_p && use_q) return -1;  /* argmax of a mixture: not defined here */
    if (!greedy && !u) return -1;
    const double temp = (double)temperature;
    for (int n = 0; n < N; ++n) {
        out[n] = -1;
        if (margin) margin[n] = kNaN;
        if (greedy) {
            const std::vector<double> z = use_p ? load_row(p, dtype, (int64_t)n * p_stride, V)
                                                : load_row(q, dtype, (int64_t)n * q_stride, V);
            out[n] = row_argmax(z);
            continue;
        }
        std::vector<double> P, logP, Q, logQ;
        if (use_p && !temperature_softmax(load_row(p, dtype, (int64_t)n * p_stride, V), temp, P, logP))
            continue;
        if (use_q && !temperature_softmax(load_row(q, dtype, (int64_t)n * q_stride, V), temp, Q, logQ))
            continue;
        std::vector<double> pi((size_t)V, 0.0);
        double Z = 0.0;
        for (int j = 0; j < V; ++j) {
            double w = 0.0;
            if (use_p) w += beta * P[(size_t)j];
            if (use_q) w += (1.0 - beta) * Q[(size_t)j];
            pi[(size_t)j] = w;
            Z += w;
        }
        double m = 0.0;
        out[n] = inverse_cdf(pi, Z, u[n], &m);
        if (margin) margin[n] = m;
    }
    return 0;
}

namespace {

/* Spacing of bf16 values around |x| (8 significant bits; the subnormal
 * spacing below 2^-126). */
double bf16_quantum(double x) {
    int e;
    std::frexp(x, &e); /* |x| = f * 2^e, f in [0.5, 1) */
    double q = std::ldexp(1.0, e - 8);
    double qmin = std::ldexp(1.0, -133);
    return q > qmin ? q : qmin;
}

}  // namespace

extern "C" void osd_ref_round_bf16(const double* x, uint16_t* out, int64_t n) {
    for (int64_t i = 0; i < n; ++i) {
        double v = x[i];
        float f;
        if (std::isnan(v)) {
            f = std::numeric_limits<float>::quiet_NaN();
        } else if (std::isinf(v) || v == 0.0) {
            f = (float)v;
        } else {
            double q = bf16_quantum(v);
            /* nearbyint rounds half to even in the default mode */
            double r = std::nearbyint(v / q) * q;
            /* exact: r has at most 8 significant bits; a value that rounds
             * up to 2^128 becomes infinity, as RNE to bf16 requires */
            f = (float)r;
        }
        uint32_t bits;
        std::memcpy(&bits, &f, sizeof bits);
        out[i] = (uint16_t)(bits >> 16);
    }
}

extern "C" void osd_ref_bf16_midpoint_flags(const double* x, uint8_t* flag,
                                            int64_t n, double rel) {
    for (int64_t i = 0; i < n; ++i) {
        double v = x[i];
        if (!std::isfinite(v) || v == 0.0) {
            flag[i] = 0;
            continue;
        }
        double q = bf16_quantum(v);
        double k = std::floor(v / q);
        double mid = (k + 0.5) * q;
        flag[i] = std::fabs(v - mid) <= rel * std::fabs(v) ? 1 : 0;
    }
}
