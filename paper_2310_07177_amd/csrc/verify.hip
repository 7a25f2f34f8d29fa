// verify.hip -- speculative-sampling verification on gfx950.
//
// Method (Appendix A.1 and Eq. 5 of arXiv:2310.07177; Algorithm 1, the step
// that determines the accepted count and samples one more token): proposals
// y_1..y_k are tested in order, y_i is accepted when u_i < p(y_i)/q(y_i), the
// first rejection at position a ends the test, and one extra token is drawn
// from norm(max(0, p - q)) at row a, or from p at the bonus row when all k
// were accepted.  p and q are temperature softmaxes of the logits.
//
// Work layout.  One workgroup per (sequence b, proposal row i), numbered
// position-major, then one workgroup per bonus row.  A proposal workgroup
// reads its target and draft rows from HBM exactly once into registers,
// reduces the row maxima and sums of exponentials, and takes the acceptance
// test.  A rejecting workgroup announces the rejection at once, then learns
// (by polling the records of the earlier positions of its sequence, with a
// bounded number of polls) whether it is the first rejection; only the first
// draws the correction token, from the rows it already holds.  If the polls
// run out it draws anyway, which is always correct.  A bonus workgroup first
// checks whether an earlier position has already rejected and, if so, skips
// its row entirely.  Every workgroup publishes a one-word record; the last of
// the k_b + 1 workgroups of a sequence to arrive selects the first rejection,
// writes the outputs, and clears the records and the counter.
#include "osd_device.hpp"
#include "osd_internal.hpp"
#include "row_draw.hpp"

namespace osd {
namespace {

// Record word: state in bits 31..28, token in bits 27..0.
enum : uint32_t {
    kRecEmpty = 0,
    kRecAccept = 1,
    kRecReject = 2,          // rejected, correction token attached
    kRecRejectSkipped = 3,   // rejected after an earlier rejection was seen
    kRecBadRow = 4,          // no finite logit in a row that was read
    kRecBadToken = 5,        // proposal outside [0, V)
    kRecBonus = 6,           // bonus token attached
    kRecBonusSkipped = 7,    // an earlier rejection was seen
    kRecRejectPending = 8,   // rejected, correction not yet decided
};

__device__ inline uint32_t make_rec(uint32_t state, uint32_t tok) {
    return (state << 28) | (tok & 0x0FFFFFFFu);
}
__device__ inline uint32_t rec_state(uint32_t r) { return r >> 28; }
__device__ inline int rec_token(uint32_t r) { return int(r & 0x0FFFFFFFu); }
__device__ inline bool rejects(uint32_t s) {
    return s == kRecReject || s == kRecRejectSkipped || s == kRecRejectPending || s == kRecBadToken;
}

// Residual masses are handled in units of S_t (the target row's sum of
// exponentials), where every element is at most about 1: chunk sums stay
// below 16 and row totals below 2^17, so a 2^-44 fixed point never overflows.
constexpr int kFixedShift = 44;
// Looks at the earlier positions' records before a rejecting workgroup draws
// speculatively (a speculative draw is always correct: the finalizer takes
// the first rejection's token).  Each look is one device-coherent round trip.
// The row-resident kernel looks once: its draw works on registers it already
// holds, and waiting for a late earlier row costs more than drawing (a
// measured 0.4 us at B = 64, k = 8).  The streamed kernel, whose draw reads
// the row pair again, waits longer (24 looks with a short sleep).
constexpr int kMaxPolls = 1;
constexpr int kMaxLongPolls = 24;

struct VerifyArgs {
    const void* target;
    const void* draft;
    int B, K, V;
    const int32_t* tokens;
    const int32_t* draft_len;
    const float* u_accept;
    const float* u_resample;
    float c2;        // log2(e) / T, the scale of every exponent
    double c2d;      // the same value in fp64
    int32_t* accepted_len;
    int32_t* out_tokens;
    uint8_t* reject_mask;
    uint32_t* records;
    uint32_t* counters;
};

__device__ void write_invalid(const VerifyArgs& a, int b) {
    const int K = a.K;
    for (int j = threadIdx.x; j <= K; j += blockDim.x) {
        a.out_tokens[int64_t(b) * (K + 1) + j] = -1;
        if (a.reject_mask && j < K) a.reject_mask[int64_t(b) * K + j] = 0;
    }
    if (threadIdx.x == 0) a.accepted_len[b] = -1;
}

// Executed by all 64 lanes of one wave with the same `record`: publish this
// row's final record, and if it is the last of the k_b + 1 rows of sequence b
// to arrive, emit the outputs.  Lane j handles position j (K < 64).
__device__ void publish(const VerifyArgs& a, int b, int i, int kb, uint32_t record) {
    const int K = a.K;
    const int lane = threadIdx.x & (kWave - 1);
    uint32_t* recs = a.records + int64_t(b) * (K + 1);
    uint32_t prev = 0;
    if (lane == 0) {
        publish_u32(&recs[i], record);
        prev = arrive(&a.counters[b]);
    }
    prev = __shfl(prev, 0, kWave);
    if (prev != uint32_t(kb)) return;

    // First rejection (Appendix A.1: the test stops there).  A proposal
    // outside the vocabulary invalidates the sequence wherever it sits; a row
    // without finite logits only if the test reaches it.  Records are read
    // and cleared in one step.
    const uint32_t r = lane <= kb ? take_u32(&recs[lane]) : 0u;
    const uint32_t s = rec_state(r);
    const bool bad_token = __ballot(lane < kb && s == kRecBadToken) != 0;
    const uint64_t stop = __ballot(lane < kb && s != kRecAccept);
    int acc = kb;
    if (stop) acc = __builtin_ctzll(stop);
    const uint32_t ra = __shfl(r, acc, kWave);
    bool bad = bad_token;
    int extra = -1;
    if (!bad) {
        const uint32_t sa = rec_state(ra);
        if (acc < kb ? sa == kRecReject : sa == kRecBonus)
            extra = rec_token(ra);
        else
            bad = true;  // a row without finite logits
    }
    const int32_t* y = a.tokens + int64_t(b) * K;
    if (lane <= K) {
        int32_t o = -1;
        if (!bad) o = lane < acc ? y[lane] : (lane == acc ? extra : -1);
        a.out_tokens[int64_t(b) * (K + 1) + lane] = o;
        if (a.reject_mask && lane < K)
            a.reject_mask[int64_t(b) * K + lane] = (!bad && lane == acc && acc < kb) ? 1 : 0;
    }
    if (lane == 0) {
        a.accepted_len[b] = bad ? -1 : acc;
        take_u32(&a.counters[b]);
    }
}

// Called by all lanes of a wave.  Looks at the records of positions 0..i-1:
// returns 2 if one of them rejected (or proposed an invalid token), 1 if all
// accepted, 0 if still undecided after `polls` looks.
__device__ int poll_earlier(const VerifyArgs& a, int b, int i, int polls) {
    const int lane = threadIdx.x & (kWave - 1);
    const uint32_t* recs = a.records + int64_t(b) * (a.K + 1);
    for (int p = 0;; ++p) {
        const uint32_t s = lane < i ? rec_state(load_relaxed(&recs[lane])) : uint32_t(kRecAccept);
        if (__ballot(rejects(s)) != 0) return 2;
        if (__ballot(s != kRecAccept) == 0) return 1;
        if (p + 1 >= polls) return 0;
        __builtin_amdgcn_s_sleep(8);
    }
}

template <typename Fmt, int W, int CPT, bool VEC, bool GREEDY>
__global__ __launch_bounds__(W, min_waves_per_simd(W, CPT)) void verify_kernel(VerifyArgs a) {
    constexpr int NW = W / kWave;
    constexpr int EPC = Fmt::kPerChunk;
    __shared__ float s_max[2][NW];
    __shared__ double s_sum[2][NW];
    __shared__ int s_idx[NW];
    __shared__ int s_flag;
    __shared__ int s_tok;
    __shared__ unsigned long long s_tot[CPT * NW];
    __shared__ DrawShared s_draw;
    __shared__ chunk_t s_stage[GREEDY ? 1 : 2 * CPT * kWave];

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int B = a.B, K = a.K, V = a.V;
    const bool bonus = int(blockIdx.x) >= B * K;
    int b, i;
    if (!bonus) {
        i = blockIdx.x / B;
        b = blockIdx.x - i * B;
    } else {
        b = blockIdx.x - B * K;
        i = -1;
    }
    const int kb = a.draft_len ? a.draft_len[b] : K;
    if (kb < 1 || kb > K) {
        if (bonus) write_invalid(a, b);
        return;
    }
    if (bonus) {
        i = kb;
    } else if (i >= kb) {
        return;  // padding row of a short proposal
    }
    const int y = bonus ? 0 : a.tokens[int64_t(b) * K + i];
    if (!bonus && (y < 0 || y >= V)) {
        if (wid == 0) publish(a, b, i, kb, make_rec(kRecBadToken, 0));
        return;
    }
    if (bonus) {
        // The bonus row matters only if every proposal is accepted: skip it
        // when a rejection is already visible.
        if (wid == 0) {
            const int st = poll_earlier(a, b, i, 1);
            if (lane == 0) s_flag = st;
            if (st == 2) publish(a, b, i, kb, make_rec(kRecBonusSkipped, 0));
        }
        __syncthreads();
        if (s_flag == 2) return;
    }

    const char* trow = static_cast<const char*>(a.target) +
                       (int64_t(b) * (K + 1) + i) * int64_t(V) * Fmt::kBytes;
    // A bonus row has no draft row: its draft loads re-read the target row
    // (ignored), so that every workgroup issues the same loads without a
    // branch and the compiler can wait for each chunk exactly.
    const char* drow = GREEDY || bonus
                           ? trow
                           : static_cast<const char*>(a.draft) + (int64_t(b) * K + i) * int64_t(V) * Fmt::kBytes;
    // The logits of the proposal itself, for the acceptance test, requested
    // before the rows and converted only after the statistics: loads complete
    // in issue order, so a value used early that was loaded after the rows
    // would make the sweeps wait for the whole row pair.
    uint32_t ty_raw = 0u, dy_raw = 0u;
    if constexpr (!GREEDY) {
        ty_raw = Fmt::load_raw(trow, bonus ? 0 : y);
        dy_raw = Fmt::load_raw(drow, bonus ? 0 : y);
    }
    __builtin_amdgcn_sched_barrier(0);
    // Sampling with 16-byte rows: the rows are loaded without padding and the
    // statistics pad each chunk as they take it, so they fold in as the
    // loads land; the register copy is padded afterwards for the draw.
    constexpr bool kFold = VEC && !GREEDY;
    const int nchunks = (V + EPC - 1) / EPC;
    chunk_t tv[CPT];
    if constexpr (!kFold) load_row<Fmt, W, CPT, VEC>(tv, trow, V);

    if constexpr (GREEDY) {
        // Target argmax, lowest index on ties: within a thread indices grow
        // with (n, e), so a strict ">" keeps the first maximum.
        float best = kNegInf;
        int bi = 0x7FFFFFFF;
#pragma unroll
        for (int n = 0; n < CPT; ++n)
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float x = Fmt::get(tv[n], e);
                if (x > best) {
                    best = x;
                    bi = (n * W + tid) * EPC + e;
                }
            }
        wave_argmax(best, bi);
        if (lane == 0) {
            s_max[0][wid] = best;
            s_idx[wid] = bi;
        }
        __syncthreads();
        if (wid == 0) {
            float bv = s_max[0][0];
            int g = s_idx[0];
            for (int w = 1; w < NW; ++w)
                if (s_max[0][w] > bv || (s_max[0][w] == bv && s_idx[w] < g)) {
                    bv = s_max[0][w];
                    g = s_idx[w];
                }
            uint32_t r;
            if (!(bv > kNegInf) || bv == -kNegInf)
                r = make_rec(kRecBadRow, 0);
            else if (bonus)
                r = make_rec(kRecBonus, uint32_t(g));
            else
                r = make_rec(y == g ? kRecAccept : kRecReject, uint32_t(g));
            publish(a, b, i, kb, r);
        }
        return;
    } else {
        const float c2 = a.c2;
        // The draft row is read only for proposal rows.
        chunk_t dv[CPT];
        if constexpr (kFold)
            load_rows_interleaved<W, CPT>(tv, dv, trow, drow, nchunks);
        else
            load_row<Fmt, W, CPT, VEC>(dv, drow, V);

        // Row statistics (K, S), folded in chunk by chunk as the loads land.
        float Kt = kNegInf, Kd = kNegInf;
        {
            float st = 0.0f, sd = 0.0f;
            if constexpr (kFold) {
                row_stats2_tail<Fmt, W, CPT>(tv, dv, nchunks, c2, !bonus, Kt, st, Kd, sd);
                pad_row_tail<Fmt, W, CPT>(tv, nchunks);
                pad_row_tail<Fmt, W, CPT>(dv, nchunks);
            } else {
                row_stats<Fmt, CPT>(tv, c2, Kt, st);
                if (!bonus) row_stats<Fmt, CPT>(dv, c2, Kd, sd);
            }
            double dt = st, dd = sd;
            wave_merge_stats(Kt, dt);
            wave_merge_stats(Kd, dd);
            if (lane == 0) {
                s_max[0][wid] = Kt;
                s_max[1][wid] = Kd;
                s_sum[0][wid] = dt;
                s_sum[1][wid] = dd;
            }
        }
        if (tid == 0) s_tok = -1;
        __syncthreads();
        Kt = s_max[0][0];
        Kd = s_max[1][0];
#pragma unroll
        for (int w = 1; w < NW; ++w) {
            Kt = fmaxf(Kt, s_max[0][w]);
            Kd = fmaxf(Kd, s_max[1][w]);
        }
        double St = 0.0, Sd = 0.0;
        for (int w = 0; w < NW; ++w) {
            St += rescale(s_sum[0][w], s_max[0][w], Kt);
            Sd += rescale(s_sum[1][w], s_max[1][w], Kd);
        }
        // A row without finite logits, or with a NaN logit (its sum is NaN),
        // cannot be tested or drawn from.
        const bool bad = !(Kt > kNegInf && Kt < -kNegInf) || !usable_sum(St) ||
                         (!bonus && (!(Kd > kNegInf && Kd < -kNegInf) || !usable_sum(Sd)));
        if (bad) {
            if (wid == 0) publish(a, b, i, kb, make_rec(kRecBadRow, 0));
            return;
        }

        // Wave 0 decides whether this workgroup draws a token.
        if (wid == 0) {
            int flag = 1;
            if (!bonus) {
                // Acceptance test: p(y)/q(y) = 2^e * S_d / S_t with
                // e = (t_y c2 - K_t) - (d_y c2 - K_d) in fp64; 2^e is split
                // into an exact power of two and 2^frac (v_exp_f32, 1 ulp).
                asm volatile("" : "+v"(ty_raw), "+v"(dy_raw));  // converted here, not at the load
                const float ty = Fmt::from_raw(ty_raw), dy = Fmt::from_raw(dy_raw);
                const double e = (double(ty) * a.c2d - double(Kt)) - (double(dy) * a.c2d - double(Kd));
                double ratio;
                if (!(e > -2000.0)) {
                    ratio = 0.0;  // p(y) = 0 (or both probabilities 0)
                } else if (e > 2000.0) {
                    ratio = __builtin_huge_val();
                } else {
                    const double n = floor(e);
                    ratio = __builtin_ldexp(double(exp2_fast(float(e - n))), int(n)) * (Sd / St);
                }
                const double u = a.u_accept[int64_t(b) * K + i];
                if (u < ratio) {
                    flag = 0;
                    publish(a, b, i, kb, make_rec(kRecAccept, 0));
                } else {
                    // Announce the rejection, then find out whether it is the
                    // first one of the sequence.
                    if (lane == 0)
                        publish_u32(a.records + int64_t(b) * (K + 1) + i, make_rec(kRecRejectPending, 0));
                    if (i > 0 && poll_earlier(a, b, i, kMaxPolls) == 2) {
                        flag = 0;
                        publish(a, b, i, kb, make_rec(kRecRejectSkipped, 0));
                    }
                }
            } else if (poll_earlier(a, b, i, kMaxPolls) == 2) {
                flag = 0;
                publish(a, b, i, kb, make_rec(kRecBonusSkipped, 0));
            }
            if (lane == 0) s_flag = flag;
        }
        __syncthreads();
        if (s_flag == 0) return;

        // Draw the extra token: from max(0, p - q) after a rejection, from p
        // at the bonus row (and, should max(0, p - q) have no mass after
        // rounding, from p as well).  Masses are in units of S_t:
        //   p_j S_t = 2^(t_j c2 - K_t),  q_j S_t = 2^(d_j c2 - K_d) (S_t / S_d).
        const float rho = bonus ? 0.0f : float(St / Sd);
        const float u = a.u_resample[b];
        bool use_p = bonus;
        for (int attempt = 0; attempt < 2; ++attempt) {
            // Opaque copies of the shifts, fresh in each attempt: without them
            // the compiler may keep exponentials alive across passes (to reuse
            // them) and spill.
            float mtc_d = Kt, mdc_d = Kd;
            asm volatile("" : "+v"(mtc_d), "+v"(mdc_d));
            opaque(tv);
            if (!use_p) opaque(dv);
            const bool p_only = use_p;
            auto mass = [=](const chunk_t& tc, const chunk_t& dc, int e) -> float {
                const float pt = exp2_fast(__builtin_fmaf(Fmt::get(tc, e), c2, -mtc_d));
                if (p_only) return pt;
                const float qt = exp2_fast(__builtin_fmaf(Fmt::get(dc, e), c2, -mdc_d));
                return fmaxf(__builtin_fmaf(-qt, rho, pt), 0.0f);
            };
            bool z_zero = false;
            const int tok = draw_inverse_cdf<kFixedShift, W, CPT, EPC>(tv, dv, mass, u, s_tot, &s_draw, s_stage, &z_zero);
            if (tok >= 0) s_tok = tok;
            if (!z_zero || use_p) break;
            use_p = true;
        }
        __syncthreads();
        if (wid == 0) {
            const int tok = s_tok;
            uint32_t r;
            if (tok >= 0)
                r = make_rec(bonus ? kRecBonus : kRecReject, uint32_t(tok));
            else
                r = make_rec(kRecBadRow, 0);  // no mass anywhere
            publish(a, b, i, kb, r);
        }
    }
}

// Rows too long to hold (more than 8 chunks per thread of a 1024-thread
// workgroup): the same per-row protocol as verify_kernel, with the rows
// streamed from memory.  The statistics take one pass over the row pair (four
// rounds of loads in flight per thread); the workgroup that draws streams the
// row pair again (pass A of draw_inverse_cdf_streamed) and its winning wave
// reloads one round (pass B).  Nothing is held across passes but (K, S), so
// no register spills at any row length.
constexpr int kLongW = 1024;
constexpr int kLongUnroll = 4;

template <typename Fmt, bool VEC>
__global__ __launch_bounds__(kLongW, 1) void verify_long_kernel(VerifyArgs a) {
    constexpr int W = kLongW, NW = W / kWave, EPC = Fmt::kPerChunk, U = kLongUnroll;
    __shared__ float s_max[2][NW];
    __shared__ double s_sum[2][NW];
    __shared__ int s_flag;
    __shared__ int s_tok;
    __shared__ unsigned long long s_tot[kMaxStreamRounds * NW];
    __shared__ DrawShared s_draw;

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int B = a.B, K = a.K, V = a.V;
    const bool bonus = int(blockIdx.x) >= B * K;
    int b, i;
    if (!bonus) {
        i = blockIdx.x / B;
        b = blockIdx.x - i * B;
    } else {
        b = blockIdx.x - B * K;
        i = -1;
    }
    const int kb = a.draft_len ? a.draft_len[b] : K;
    if (kb < 1 || kb > K) {
        if (bonus) write_invalid(a, b);
        return;
    }
    if (bonus) {
        i = kb;
    } else if (i >= kb) {
        return;
    }
    const int y = bonus ? 0 : a.tokens[int64_t(b) * K + i];
    if (!bonus && (y < 0 || y >= V)) {
        if (wid == 0) publish(a, b, i, kb, make_rec(kRecBadToken, 0));
        return;
    }
    if (bonus) {
        if (wid == 0) {
            const int st = poll_earlier(a, b, i, 1);
            if (lane == 0) s_flag = st;
            if (st == 2) publish(a, b, i, kb, make_rec(kRecBonusSkipped, 0));
        }
        __syncthreads();
        if (s_flag == 2) return;
    }
    const char* trow = static_cast<const char*>(a.target) + (int64_t(b) * (K + 1) + i) * int64_t(V) * Fmt::kBytes;
    const char* drow =
        bonus ? trow : static_cast<const char*>(a.draft) + (int64_t(b) * K + i) * int64_t(V) * Fmt::kBytes;
    uint32_t ty_raw = 0u, dy_raw = 0u;
    if (!bonus) {
        ty_raw = Fmt::load_raw(trow, y);
        dy_raw = Fmt::load_raw(drow, y);
    }
    const float c2 = a.c2;
    const int nchunks = (V + EPC - 1) / EPC;
    const int R = (nchunks + W - 1) / W;

    // Statistics, U rounds of loads at a time.
    float Kt = kNegInf, Kd = kNegInf, st = 0.0f, sd = 0.0f;
    for (int r0 = 0; r0 < R; r0 += U) {
        chunk_t xt[U], xd[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int ch = (r0 + u) * W + tid;
            xt[u] = stream_chunk<Fmt, VEC>(trow, ch, nchunks, V);
            if (!bonus) xd[u] = stream_chunk<Fmt, VEC>(drow, ch, nchunks, V);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            fold_chunk<Fmt>(xt[u], c2, Kt, st);
            if (!bonus) fold_chunk<Fmt>(xd[u], c2, Kd, sd);
        }
    }
    {
        double dt = st, dd = sd;
        wave_merge_stats(Kt, dt);
        wave_merge_stats(Kd, dd);
        if (lane == 0) {
            s_max[0][wid] = Kt;
            s_max[1][wid] = Kd;
            s_sum[0][wid] = dt;
            s_sum[1][wid] = dd;
        }
    }
    if (tid == 0) s_tok = -1;
    __syncthreads();
    Kt = s_max[0][0];
    Kd = s_max[1][0];
#pragma unroll
    for (int w = 1; w < NW; ++w) {
        Kt = fmaxf(Kt, s_max[0][w]);
        Kd = fmaxf(Kd, s_max[1][w]);
    }
    double St = 0.0, Sd = 0.0;
    for (int w = 0; w < NW; ++w) {
        St += rescale(s_sum[0][w], s_max[0][w], Kt);
        Sd += rescale(s_sum[1][w], s_max[1][w], Kd);
    }
    const bool bad = !(Kt > kNegInf && Kt < -kNegInf) || !usable_sum(St) ||
                     (!bonus && (!(Kd > kNegInf && Kd < -kNegInf) || !usable_sum(Sd)));
    if (bad) {
        if (wid == 0) publish(a, b, i, kb, make_rec(kRecBadRow, 0));
        return;
    }
    // Wave 0 decides whether this workgroup draws (as verify_kernel).
    if (wid == 0) {
        int flag = 1;
        if (!bonus) {
            const float ty = Fmt::from_raw(ty_raw), dy = Fmt::from_raw(dy_raw);
            const double e = (double(ty) * a.c2d - double(Kt)) - (double(dy) * a.c2d - double(Kd));
            double ratio;
            if (!(e > -2000.0)) {
                ratio = 0.0;
            } else if (e > 2000.0) {
                ratio = __builtin_huge_val();
            } else {
                const double n = floor(e);
                ratio = __builtin_ldexp(double(exp2_fast(float(e - n))), int(n)) * (Sd / St);
            }
            const double u = a.u_accept[int64_t(b) * K + i];
            if (u < ratio) {
                flag = 0;
                publish(a, b, i, kb, make_rec(kRecAccept, 0));
            } else {
                if (lane == 0) publish_u32(a.records + int64_t(b) * (K + 1) + i, make_rec(kRecRejectPending, 0));
                if (i > 0 && poll_earlier(a, b, i, kMaxLongPolls) == 2) {
                    flag = 0;
                    publish(a, b, i, kb, make_rec(kRecRejectSkipped, 0));
                }
            }
        } else if (poll_earlier(a, b, i, kMaxLongPolls) == 2) {
            flag = 0;
            publish(a, b, i, kb, make_rec(kRecBonusSkipped, 0));
        }
        if (lane == 0) s_flag = flag;
    }
    __syncthreads();
    if (s_flag == 0) return;

    // The draw, the masses of verify_kernel on the streamed chunks.
    const float rho = bonus ? 0.0f : float(St / Sd);
    const float u = a.u_resample[b];
    bool use_p = bonus;
    for (int attempt = 0; attempt < 2; ++attempt) {
        const bool p_only = use_p;
        const float kt = Kt, kd = Kd;
        auto masses = [&](int r, float (&m)[EPC]) {
            const int ch = r * W + tid;
            const chunk_t tc = stream_chunk<Fmt, VEC>(trow, ch, nchunks, V);
            const chunk_t dc = p_only ? tc : stream_chunk<Fmt, VEC>(drow, ch, nchunks, V);
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float pt = exp2_fast(__builtin_fmaf(Fmt::get(tc, e), c2, -kt));
                if (p_only) {
                    m[e] = pt;
                } else {
                    const float qt = exp2_fast(__builtin_fmaf(Fmt::get(dc, e), c2, -kd));
                    m[e] = fmaxf(__builtin_fmaf(-qt, rho, pt), 0.0f);
                }
            }
        };
        bool z_zero = false;
        const int tok = draw_inverse_cdf_streamed<kFixedShift, W, EPC>(R, masses, u, s_tot, &s_draw, &z_zero);
        if (tok >= 0) s_tok = tok;
        if (!z_zero || use_p) break;
        use_p = true;
        __syncthreads();  // s_tot and s_draw are reused
    }
    __syncthreads();
    if (wid == 0) {
        const int tok = s_tok;
        publish(a, b, i, kb, tok >= 0 ? make_rec(bonus ? kRecBonus : kRecReject, uint32_t(tok)) : make_rec(kRecBadRow, 0));
    }
}

template <typename Fmt>
hipError_t launch_long(const VerifyLaunch& L, const VerifyArgs& a) {
    const dim3 grid(unsigned(L.B) * unsigned(L.K + 1)), block(kLongW);
    return L.vec ? launch_kernel(&verify_long_kernel<Fmt, true>, grid, block, 0, L.stream, a)
                 : launch_kernel(&verify_long_kernel<Fmt, false>, grid, block, 0, L.stream, a);
}

template <typename Fmt, int W, int CPT>
hipError_t launch_tile(const VerifyLaunch& L, const VerifyArgs& a) {
    const dim3 grid(unsigned(L.B) * unsigned(L.K + 1)), block(W);
    const bool greedy = L.temperature == 0.0f;
    hipError_t e;
    if (L.vec) {
        if (greedy)
            e = launch_kernel(&verify_kernel<Fmt, W, CPT, true, true>, grid, block, 0, L.stream, a);
        else
            e = launch_kernel(&verify_kernel<Fmt, W, CPT, true, false>, grid, block, 0, L.stream, a);
    } else {
        if (greedy)
            e = launch_kernel(&verify_kernel<Fmt, W, CPT, false, true>, grid, block, 0, L.stream, a);
        else
            e = launch_kernel(&verify_kernel<Fmt, W, CPT, false, false>, grid, block, 0, L.stream, a);
    }
    return e;
}

template <typename Fmt>
hipError_t launch_fmt(const VerifyLaunch& L, const VerifyArgs& a) {
    RowTile t;
    if (!pick_tile(L.V, Fmt::kPerChunk, &t)) {
        if (L.V > max_vocab_for(Fmt::kPerChunk)) return hipErrorInvalidValue;
        // Rows longer than the largest resident tile: streamed (sampling).
        // Greedy rows of that length take the resident 1024 x 16 tile, which
        // holds one row per thread without spilling.
        if (L.temperature > 0.0f) return launch_long<Fmt>(L, a);
        const dim3 grid(unsigned(L.B) * unsigned(L.K + 1)), block(1024);
        return L.vec ? launch_kernel(&verify_kernel<Fmt, 1024, 16, true, true>, grid, block, 0, L.stream, a)
                     : launch_kernel(&verify_kernel<Fmt, 1024, 16, false, true>, grid, block, 0, L.stream, a);
    }
    switch (t.W * 100 + t.CPT) {
        case 25601: return launch_tile<Fmt, 256, 1>(L, a);
        case 25602: return launch_tile<Fmt, 256, 2>(L, a);
        case 25604: return launch_tile<Fmt, 256, 4>(L, a);
        case 51204: return launch_tile<Fmt, 512, 4>(L, a);
        case 51208: return launch_tile<Fmt, 512, 8>(L, a);
        case 102408: return launch_tile<Fmt, 1024, 8>(L, a);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

// The largest row every entry point takes: 16 rounds of 1024 threads
// (131072 bf16 or 65536 fp32 logits); the streamed kernels' cell tables are
// sized for it.
int max_vocab_for(int per_chunk) { return 1024 * kMaxStreamRounds * per_chunk; }

// Register-resident tiles (a row pair in registers, at most 8 chunks per
// thread); longer rows are streamed.
bool pick_tile(int V, int per_chunk, RowTile* t) {
    static const RowTile tiles[] = {{256, 1}, {256, 2}, {256, 4}, {512, 4},
                                    {512, 8}, {1024, 8}};
    for (const RowTile& c : tiles)
        if (int64_t(V) <= int64_t(c.W) * c.CPT * per_chunk) {
            *t = c;
            return true;
        }
    return false;
}

hipError_t launch_verify(const VerifyLaunch& L) {
    VerifyArgs a{};
    a.target = L.target;
    a.draft = L.draft;
    a.B = L.B;
    a.K = L.K;
    a.V = L.V;
    a.tokens = L.tokens;
    a.draft_len = L.draft_len;
    a.u_accept = L.u_accept;
    a.u_resample = L.u_resample;
    a.c2 = L.temperature > 0.0f ? float(1.4426950408889634 / double(L.temperature)) : 0.0f;
    a.c2d = double(a.c2);
    a.accepted_len = L.accepted_len;
    a.out_tokens = L.out_tokens;
    a.reject_mask = L.reject_mask;
    a.records = L.records;
    a.counters = L.counters;
    return L.dtype == 1 ? launch_fmt<BF16>(L, a) : launch_fmt<F32>(L, a);
}

}  // namespace osd
