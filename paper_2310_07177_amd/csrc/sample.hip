// sample.hip -- token sampling on gfx950: the draft's proposals y ~ q
// (Algorithm 1 of arXiv:2310.07177) and the mixed sampling
// y ~ beta p + (1 - beta) q that Section 4.1 uses to generate distillation
// data, at temperature T (T = 0: argmax).
//
// Work layout: one workgroup per sampled row n, the row (or the row pair of a
// mixture) read once from HBM into registers with the tile of the
// verification kernel; the softmax statistics (K, S) are folded in chunk by
// chunk and merged over lanes and waves; the token is drawn with the exact
// fixed-point inverse CDF of row_draw.hpp.  Masses:
//   one row:  2^(x c2 - K), in units of S (the verification's bonus draw);
//   mixture:  beta 2^(t c2 - K_p)/S_p + (1 - beta) 2^(d c2 - K_q)/S_q, in
//             probability units (each element is at most 1, every partial
//             sum at most 1 + rounding, so 2^-60 fixed point cannot overflow).
#include "osd.h"
#include "osd_device.hpp"
#include "osd_internal.hpp"
#include "row_draw.hpp"

namespace osd {
namespace {

constexpr int kShiftOne = 44;  // units of S: elements <= 1, row total <= V
constexpr int kShiftMix = 60;  // probability units: total 1

enum : int { kModeGreedy = 0, kModeOne = 1, kModeMix = 2 };

struct SampleArgs {
    const char* p;        // the row with weight beta (one-row modes: the row sampled)
    const char* q;        // the row with weight 1 - beta (mixture only)
    int64_t p_stride;     // row strides, bytes
    int64_t q_stride;
    int N, V;
    float c2;             // log2(e) / T
    float beta;
    const float* u;       // [N]
    int32_t* out;         // [N]
};

template <typename Fmt, int W, int CPT, bool VEC, int MODE>
__global__ __launch_bounds__(W, min_waves_per_simd(W, CPT)) void sample_kernel(SampleArgs a) {
    constexpr int NW = W / kWave;
    constexpr int EPC = Fmt::kPerChunk;
    constexpr bool MIX = MODE == kModeMix;
    __shared__ float s_max[2][NW];
    __shared__ double s_sum[2][NW];
    __shared__ int s_idx[NW];
    __shared__ int s_tok;
    __shared__ unsigned long long s_tot[CPT * NW];
    __shared__ DrawShared s_draw;
    __shared__ chunk_t s_stage[MODE == kModeGreedy ? 1 : 2 * CPT * kWave];

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int n = blockIdx.x;
    chunk_t tv[CPT], dv[CPT];
    // Sampling from 16-byte rows: loads without padding (a row pair
    // interleaved chunk by chunk), so that the statistics fold in as they
    // land; the register copy is padded afterwards for the draw.
    constexpr bool kFold = VEC && MODE != kModeGreedy;
    const int nchunks = (a.V + EPC - 1) / EPC;
    if constexpr (kFold && MIX) {
        load_rows_interleaved<W, CPT>(tv, dv, a.p + int64_t(n) * a.p_stride, a.q + int64_t(n) * a.q_stride, nchunks);
    } else if constexpr (kFold) {
        load_row_clamped<W, CPT>(tv, a.p + int64_t(n) * a.p_stride, nchunks);
    } else {
        load_row<Fmt, W, CPT, VEC>(tv, a.p + int64_t(n) * a.p_stride, a.V);
        if constexpr (MIX) load_row<Fmt, W, CPT, VEC>(dv, a.q + int64_t(n) * a.q_stride, a.V);
    }

    if constexpr (MODE == kModeGreedy) {
        // Argmax, lowest index on ties: within a thread indices grow with
        // (round, element), so a strict ">" keeps the first maximum.
        float best = kNegInf;
        int bi = 0x7FFFFFFF;
#pragma unroll
        for (int r = 0; r < CPT; ++r)
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float x = Fmt::get(tv[r], e);
                if (x > best) {
                    best = x;
                    bi = (r * W + tid) * EPC + e;
                }
            }
        wave_argmax(best, bi);
        if (lane == 0) {
            s_max[0][wid] = best;
            s_idx[wid] = bi;
        }
        __syncthreads();
        if (tid == 0) {
            float bv = s_max[0][0];
            int g = s_idx[0];
            for (int w = 1; w < NW; ++w)
                if (s_max[0][w] > bv || (s_max[0][w] == bv && s_idx[w] < g)) {
                    bv = s_max[0][w];
                    g = s_idx[w];
                }
            a.out[n] = (bv > kNegInf && bv < -kNegInf) ? g : -1;
        }
        return;
    } else {
        const float c2 = a.c2;
        float Kp = kNegInf, Kq = kNegInf;
        {
            float sp = 0.0f, sq = 0.0f;
            if constexpr (kFold && MIX) {
                row_stats2_tail<Fmt, W, CPT>(tv, dv, nchunks, c2, true, Kp, sp, Kq, sq);
                pad_row_tail<Fmt, W, CPT>(tv, nchunks);
                pad_row_tail<Fmt, W, CPT>(dv, nchunks);
            } else if constexpr (kFold) {
                row_stats_tail<Fmt, W, CPT>(tv, nchunks, c2, Kp, sp);
                pad_row_tail<Fmt, W, CPT>(tv, nchunks);
            } else {
                row_stats<Fmt, CPT>(tv, c2, Kp, sp);
                if constexpr (MIX) row_stats<Fmt, CPT>(dv, c2, Kq, sq);
            }
            double dp = sp, dq = sq;
            wave_merge_stats(Kp, dp);
            if constexpr (MIX) wave_merge_stats(Kq, dq);
            if (lane == 0) {
                s_max[0][wid] = Kp;
                s_max[1][wid] = Kq;
                s_sum[0][wid] = dp;
                s_sum[1][wid] = dq;
            }
        }
        if (tid == 0) s_tok = -1;
        __syncthreads();
        Kp = s_max[0][0];
        Kq = s_max[1][0];
#pragma unroll
        for (int w = 1; w < NW; ++w) {
            Kp = fmaxf(Kp, s_max[0][w]);
            Kq = fmaxf(Kq, s_max[1][w]);
        }
        double Sp = 0.0, Sq = 0.0;
        for (int w = 0; w < NW; ++w) {
            Sp += rescale(s_sum[0][w], s_max[0][w], Kp);
            if constexpr (MIX) Sq += rescale(s_sum[1][w], s_max[1][w], Kq);
        }
        const bool bad = !(Kp > kNegInf && Kp < -kNegInf) || !usable_sum(Sp) ||
                         (MIX && (!(Kq > kNegInf && Kq < -kNegInf) || !usable_sum(Sq)));
        if (bad) {
            if (tid == 0) a.out[n] = -1;
            return;
        }
        // Opaque copies of the shifts and rows: the compiler must not keep
        // the statistics pass's exponentials alive for the draw.
        float kp = Kp, kq = Kq;
        asm volatile("" : "+v"(kp), "+v"(kq));
        opaque(tv);
        if constexpr (MIX) opaque(dv);
        const float wp = MIX ? float(double(a.beta) / Sp) : 1.0f;
        const float wq = MIX ? float((1.0 - double(a.beta)) / Sq) : 0.0f;
        auto mass = [=](const chunk_t& tc, const chunk_t& dc, int e) -> float {
            const float et = exp2_fast(__builtin_fmaf(Fmt::get(tc, e), c2, -kp));
            if constexpr (!MIX) {
                return et;
            } else {
                const float ed = exp2_fast(__builtin_fmaf(Fmt::get(dc, e), c2, -kq));
                return __builtin_fmaf(wp, et, wq * ed);
            }
        };
        bool z_zero = false;
        const int tok = draw_inverse_cdf<MIX ? kShiftMix : kShiftOne, W, CPT, EPC>(
            tv, dv, mass, a.u[n], s_tot, &s_draw, s_stage, &z_zero);
        if (tok >= 0) s_tok = tok;
        __syncthreads();
        if (tid == 0) a.out[n] = s_tok;  // -1 when no element carries mass
    }
}

template <typename Fmt, int W, int CPT, int MODE>
hipError_t launch_mode(const SampleLaunch& L, const SampleArgs& a) {
    const dim3 grid(unsigned(L.N)), block(W);
    hipError_t e;
    if (L.vec)
        e = launch_kernel(&sample_kernel<Fmt, W, CPT, true, MODE>, grid, block, 0, L.stream, a);
    else
        e = launch_kernel(&sample_kernel<Fmt, W, CPT, false, MODE>, grid, block, 0, L.stream, a);
    return e;
}

// A mixture of rows too long to hold as a pair (beyond 8 chunks per thread of
// 1024 threads): the statistics and the draw of sample_kernel with both rows
// streamed from memory, one 1024-thread workgroup per row pair.
constexpr int kLongW = 1024;
constexpr int kLongUnroll = 4;

template <typename Fmt, bool VEC>
__global__ __launch_bounds__(kLongW, 1) void sample_mix_long_kernel(SampleArgs a) {
    constexpr int W = kLongW, NW = W / kWave, EPC = Fmt::kPerChunk, U = kLongUnroll;
    __shared__ float s_max[2][NW];
    __shared__ double s_sum[2][NW];
    __shared__ int s_tok;
    __shared__ unsigned long long s_tot[kMaxStreamRounds * NW];
    __shared__ DrawShared s_draw;

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int n = blockIdx.x;
    const int V = a.V;
    const char* prow = a.p + int64_t(n) * a.p_stride;
    const char* qrow = a.q + int64_t(n) * a.q_stride;
    const int nchunks = (V + EPC - 1) / EPC;
    const int R = (nchunks + W - 1) / W;
    const float c2 = a.c2;
    float Kp = kNegInf, Kq = kNegInf, sp = 0.0f, sq = 0.0f;
    for (int r0 = 0; r0 < R; r0 += U) {
        chunk_t xp[U], xq[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            xp[u] = stream_chunk<Fmt, VEC>(prow, (r0 + u) * W + tid, nchunks, V);
            xq[u] = stream_chunk<Fmt, VEC>(qrow, (r0 + u) * W + tid, nchunks, V);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            fold_chunk<Fmt>(xp[u], c2, Kp, sp);
            fold_chunk<Fmt>(xq[u], c2, Kq, sq);
        }
    }
    {
        double dp = sp, dq = sq;
        wave_merge_stats(Kp, dp);
        wave_merge_stats(Kq, dq);
        if (lane == 0) {
            s_max[0][wid] = Kp;
            s_max[1][wid] = Kq;
            s_sum[0][wid] = dp;
            s_sum[1][wid] = dq;
        }
    }
    if (tid == 0) s_tok = -1;
    __syncthreads();
    Kp = s_max[0][0];
    Kq = s_max[1][0];
#pragma unroll
    for (int w = 1; w < NW; ++w) {
        Kp = fmaxf(Kp, s_max[0][w]);
        Kq = fmaxf(Kq, s_max[1][w]);
    }
    double Sp = 0.0, Sq = 0.0;
    for (int w = 0; w < NW; ++w) {
        Sp += rescale(s_sum[0][w], s_max[0][w], Kp);
        Sq += rescale(s_sum[1][w], s_max[1][w], Kq);
    }
    const bool bad = !(Kp > kNegInf && Kp < -kNegInf) || !usable_sum(Sp) || !(Kq > kNegInf && Kq < -kNegInf) ||
                     !usable_sum(Sq);
    if (bad) {
        if (tid == 0) a.out[n] = -1;
        return;
    }
    const float wp = float(double(a.beta) / Sp), wq = float((1.0 - double(a.beta)) / Sq);
    const float kp = Kp, kq = Kq;
    auto masses = [&](int r, float (&m)[EPC]) {
        const int ch = r * W + tid;
        const chunk_t tc = stream_chunk<Fmt, VEC>(prow, ch, nchunks, V);
        const chunk_t dc = stream_chunk<Fmt, VEC>(qrow, ch, nchunks, V);
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
            const float et = exp2_fast(__builtin_fmaf(Fmt::get(tc, e), c2, -kp));
            const float ed = exp2_fast(__builtin_fmaf(Fmt::get(dc, e), c2, -kq));
            m[e] = __builtin_fmaf(wp, et, wq * ed);
        }
    };
    bool z_zero = false;
    const int tok = draw_inverse_cdf_streamed<kShiftMix, W, EPC>(R, masses, a.u[n], s_tot, &s_draw, &z_zero);
    if (tok >= 0) s_tok = tok;
    __syncthreads();
    if (tid == 0) a.out[n] = s_tok;
}

template <typename Fmt, int W, int CPT>
hipError_t launch_tile(const SampleLaunch& L, const SampleArgs& a) {
    if (L.temperature == 0.0f) return launch_mode<Fmt, W, CPT, kModeGreedy>(L, a);
    if (L.beta > 0.0f && L.beta < 1.0f) return launch_mode<Fmt, W, CPT, kModeMix>(L, a);
    return launch_mode<Fmt, W, CPT, kModeOne>(L, a);
}

template <typename Fmt>
hipError_t launch_fmt(const SampleLaunch& L, const SampleArgs& a) {
    RowTile t;
    if (!pick_tile(L.V, Fmt::kPerChunk, &t)) {
        // Longer rows: a mixture streams its row pair; one row (or an
        // argmax) fits the resident 1024 x 16 tile without spilling.
        const bool mix = L.temperature > 0.0f && L.beta > 0.0f && L.beta < 1.0f;
        const dim3 grid(unsigned(L.N)), block(kLongW);
        if (mix)
            return L.vec ? launch_kernel(&sample_mix_long_kernel<Fmt, true>, grid, block, 0, L.stream, a)
                         : launch_kernel(&sample_mix_long_kernel<Fmt, false>, grid, block, 0, L.stream, a);
        if (L.temperature == 0.0f) return launch_mode<Fmt, 1024, 16, kModeGreedy>(L, a);
        return launch_mode<Fmt, 1024, 16, kModeOne>(L, a);
    }
    // Fewer rows than two per CU: the rows' latency is the cost, so each row
    // gets the widest workgroup (half the elements per thread).
    if (L.N < 2 * L.cus && t.W < 1024) {
        const int per = 1024 * Fmt::kPerChunk;
        t = RowTile{1024, L.V <= 2 * per ? 2 : (L.V <= 4 * per ? 4 : 8)};
    }
    switch (t.W * 100 + t.CPT) {
        case 102402: return launch_tile<Fmt, 1024, 2>(L, a);
        case 102404: return launch_tile<Fmt, 1024, 4>(L, a);
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

hipError_t launch_sample(const SampleLaunch& L) {
    SampleArgs a{};
    // One-row modes sample the row with weight 1: p when beta == 1, q when
    // beta == 0 (the row with weight 0 is never read).
    const bool q_only = L.beta == 0.0f;
    a.p = static_cast<const char*>(q_only ? L.q : L.p);
    a.q = static_cast<const char*>(L.q);
    const int64_t elem = L.dtype == 1 ? 2 : 4;
    a.p_stride = (q_only ? L.q_stride : L.p_stride) * elem;
    a.q_stride = L.q_stride * elem;
    a.N = L.N;
    a.V = L.V;
    a.c2 = L.temperature > 0.0f ? float(1.4426950408889634 / double(L.temperature)) : 0.0f;
    a.beta = L.beta;
    a.u = L.u;
    a.out = L.out;
    return L.dtype == 1 ? launch_fmt<BF16>(L, a) : launch_fmt<F32>(L, a);
}

}  // namespace osd
