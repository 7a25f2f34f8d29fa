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
#include <stdlib.h>

#include "osd.h"
#include "osd_device.hpp"
#include "osd_internal.hpp"
#include "row_draw.hpp"
#include "stream_device.hpp"

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

// One-row sampling of few rows (fewer than two per CU), each row split over S
// segment workgroups of 256 threads (CPT chunks per thread, SEG = CPT*256
// chunks per segment).  The inverse CDF needs no global normaliser: for any
// common shift K, token j is the first whose running sum of 2^(x c2 - K)
// exceeds u times the total.  Each segment therefore works alone:
//   1. shift k_s = ceil(max over the segment * c2); masses 2^(x c2 - k_s);
//      each thread's chunk sums become 2^-40 fixed point (whole numbers in
//      fp64, exact below 2^53), summed into cells (round, wave) and the
//      segment total T_s;
//   2. it publishes (k_s, T_s) and reads its siblings' (bounded polls; a
//      workgroup that runs out of polls computes the missing records itself
//      from the rows in memory, bit for bit as their owners do);
//   3. every segment combines the S records in segment order, identically:
//      K = max k_s over segments with a finite logit, weights
//      W_s = floor(T_s 2^(k_s - K)) (u64), Z = sum W_s, the point
//      c = floor(u Z), and the segment s* whose weight interval holds c;
//   4. s* maps c into its own units (an exact shift: the local offset stays
//      below T_s*) and walks its cells, its lanes and its elements.
// The cells partition [0, Z) exactly, so the token is always one with mass;
// it can differ from the one-workgroup kernel's only where u*Z lies within
// the fp32 rounding of a boundary.  Records are two never-zero words per
// segment (the shift's bits with the top bit set; the total's bits
// inverted); each workgroup arrives at its row's counter once it holds all
// S records, and the last to arrive clears the row's words and counter.
constexpr int kSegSampleW = 256;
constexpr int kMaxSampleSegments = 16;
constexpr int kSamplePolls = 256;

struct SplitSampleArgs {
    const char* row;   // row 0 of the sampled rows
    int64_t stride;    // bytes between rows
    int N, V, nchunks, S, polls;
    float c2;
    const float* u;
    int32_t* out;
    uint64_t* rec;     // [N, kMaxSampleSegments, 2], zero between calls
    uint32_t* cnt;     // [N, 4] (word 0: arrivals), zero between calls
};

__device__ inline double fixed40(float x) { return floor(double(x) * 0x1p40); }

// Statistics of one segment held in x (chunk r of this thread is segment
// chunk r*W + tid): the shift, the cell totals (s_cell[r*NW + w]) and their
// exclusive prefix in segment order (s_excl), the total and whether the
// segment has any finite logit.  Each thread also keeps what a walk to a
// point inside its chunks needs: the chunk masses m, their fixed-point sums
// f and the sum of the lower lanes' sums in the same cell (off).  All
// threads call it; it ends with the cell values visible to every thread.
template <typename Fmt, int CPT>
__device__ void segment_stats(const chunk_t (&x)[CPT], float c2, float* s_mx, double* s_cell, double* s_excl,
                              double* s_tot, float& k, double& T, bool& empty, float (&m)[CPT][Fmt::kPerChunk],
                              double (&f)[CPT], double (&off)[CPT]) {
    constexpr int W = kSegSampleW, NW = W / kWave, EPC = Fmt::kPerChunk, CELLS = CPT * NW;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    float mx = chunk_max<Fmt>(x[0]);
#pragma unroll
    for (int r = 1; r < CPT; ++r) mx = fmaxf(mx, chunk_max<Fmt>(x[r]));
    mx = wave_max_u(mx);
    if (lane == 0) s_mx[wid] = mx;
    __syncthreads();
    mx = s_mx[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) mx = fmaxf(mx, s_mx[w]);
    empty = !(mx > kNegInf);
    k = shift_of_max(mx, c2);
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
        m[r][0] = exp2_fast(__builtin_fmaf(Fmt::get(x[r], 0), c2, -k));
        float sm = m[r][0];
#pragma unroll
        for (int e = 1; e < EPC; ++e) {
            m[r][e] = exp2_fast(__builtin_fmaf(Fmt::get(x[r], e), c2, -k));
            sm = sm + m[r][e];
        }
        f[r] = fixed40(sm);
        const double t = wave_scan_add(f[r]);
        off[r] = t - f[r];
        if (lane == kWave - 1) s_cell[r * NW + wid] = t;
        __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    if (wid == 0) {
        const double cv = lane < CELLS ? s_cell[lane] : 0.0;
        const double ci = wave_scan_add(cv);
        if (lane < CELLS) s_excl[lane] = ci - cv;
        if (lane == kWave - 1) *s_tot = ci;
    }
    __syncthreads();
    T = *s_tot;
}

template <typename Fmt, int CPT>
__global__ __launch_bounds__(kSegSampleW) void sample_split_kernel(SplitSampleArgs a) {
    constexpr int W = kSegSampleW, NW = W / kWave, EPC = Fmt::kPerChunk, SEG = CPT * W, CELLS = CPT * NW;
    static_assert(CELLS <= kWave, "one wave scans the cells");
    __shared__ float s_mx[NW];
    __shared__ double s_cell[CELLS];
    __shared__ double s_excl[CELLS];
    __shared__ double s_tot;
    __shared__ float s_k[kMaxSampleSegments];
    __shared__ double s_T[kMaxSampleSegments];
    __shared__ int s_ok;
    __shared__ int s_tok;

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int S = a.S, n = blockIdx.x / S, s = blockIdx.x - n * S;
    const char* row = a.row + int64_t(n) * a.stride;
    uint64_t* rec = a.rec + int64_t(n) * kMaxSampleSegments * 2;
    const float c2 = a.c2;

    // The row's uniform is read with the chunks (a load after the exchange
    // would wait for the exchange's own memory operations).
    const float un = a.u[n];
    chunk_t x[CPT];
#pragma unroll
    for (int r = 0; r < CPT; ++r) x[r] = stream_chunk<Fmt, true>(row, s * SEG + r * W + tid, a.nchunks, a.V);
    if (tid == 0) s_tok = -1;  // ordered before the walk by the statistics' barriers
    float k;
    double T;
    bool empty;
    float mass[CPT][EPC];
    double fx[CPT], off[CPT];
    segment_stats<Fmt, CPT>(x, c2, s_mx, s_cell, s_excl, &s_tot, k, T, empty, mass, fx, off);
    if (tid == 0) {
        s_k[s] = empty ? kNegInf : k;
        s_T[s] = T;
        // Both words issued before either completion is waited for.
        const uint64_t o0 = __hip_atomic_exchange(&rec[2 * s], (1ull << 63) | __float_as_uint(empty ? kNegInf : k),
                                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t o1 = __hip_atomic_exchange(&rec[2 * s + 1], ~uint64_t(__double_as_longlong(T)),
                                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        asm volatile("" ::"v"(o0), "v"(o1));
    }
    // The siblings' records: wave 0, lane j reads segment j's two words.
    if (wid == 0) {
        const bool mine = lane < S && lane != s;
        bool ok = false;
        uint64_t w0 = 0, w1 = 0;
        for (int p = 0; p < a.polls; ++p) {
            if (p > 0) __builtin_amdgcn_s_sleep(4);
            bool ready = true;
            if (mine) {
                w0 = poll_u64(&rec[2 * lane]);
                w1 = poll_u64(&rec[2 * lane + 1]);
                ready = w0 != 0 && w1 != 0;
            }
            if (__ballot(!ready) == 0) {
                ok = true;
                break;
            }
        }
        if (ok && mine) {
            s_k[lane] = __uint_as_float(uint32_t(w0));
            s_T[lane] = __longlong_as_double(~w1);
        }
        if (lane == 0) s_ok = ok;
    }
    __syncthreads();
    if (!s_ok) {
        // Out of polls: every other segment's record from the row itself.
        __shared__ double s_cellx[CELLS], s_exclx[CELLS];
        for (int j = 0; j < S; ++j) {
            if (j == s) continue;
            chunk_t y[CPT];
#pragma unroll
            for (int r = 0; r < CPT; ++r) y[r] = stream_chunk<Fmt, true>(row, j * SEG + r * W + tid, a.nchunks, a.V);
            float kj;
            double Tj;
            bool ej;
            float mj[CPT][EPC];
            double fj[CPT], oj[CPT];
            segment_stats<Fmt, CPT>(y, c2, s_mx, s_cellx, s_exclx, &s_tot, kj, Tj, ej, mj, fj, oj);
            if (tid == 0) {
                s_k[j] = ej ? kNegInf : kj;
                s_T[j] = Tj;
            }
        }
        __syncthreads();
    }
    // Arrival at the row's counter, once this workgroup holds every record:
    // issued here, its count awaited only at the end (s* walks meanwhile);
    // the last to arrive leaves the row's words zero.  (This workgroup's
    // records went out before its polls, whose waits covered them.)
    uint32_t prev = 0;
    if (tid == 0) prev = __hip_atomic_fetch_add(&a.cnt[int64_t(n) * 4], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    auto arrive_row = [&]() {
        if (tid == 0 && prev == uint32_t(S - 1)) {
            for (int j = 0; j < S; ++j) {
                take_u64(&rec[2 * j]);
                take_u64(&rec[2 * j + 1]);
            }
            take_u32(&a.cnt[int64_t(n) * 4]);
        }
    };
    // The combine, identical in every segment and every wave (no barrier):
    // lane j holds segment j's record; the shift K is their maximum, the
    // weights are scanned in segment order, and s* is the lane whose weight
    // interval holds c.
    const bool have = lane < S;
    const float kj = have ? s_k[lane] : kNegInf;
    const double Tj = have ? s_T[lane] : 0.0;
    const bool bad = __ballot(have && !(Tj >= 0.0 && Tj < 0x1p60)) != 0;
    const float K = wave_max_u(kj);
    uint64_t wj = 0;
    if (have && kj > kNegInf && !bad) wj = uint64_t(floor(__builtin_ldexp(Tj, int(fmaxf(kj - K, -2048.0f)))));
    const uint64_t incl = wave_scan_add(wj);
    const uint64_t Z = readlane_u64(incl, kWave - 1);
    if (bad || Z == 0) {
        if (s == 0 && tid == 0) a.out[n] = -1;
        arrive_row();
        return;
    }
    uint64_t c = uint64_t(double(un) * double(Z));
    if (c >= Z) c = Z - 1;
    const uint64_t hit = __ballot(wj > 0 && incl - wj <= c && c < incl);
    const int sstar = hit ? __builtin_ctzll(hit) : -1;
    if (s != sstar) {
        arrive_row();
        return;
    }
    const uint64_t lo = readlane_u64(incl - wj, sstar);
    // This segment holds the point: its offset in the segment's own units.
    // The cell (round r of this wave) and the lane that hold it, from the
    // prefixes prepared before the exchange; that lane walks its chunk with
    // the same fp32 sums of the same masses.
    const double target = __builtin_ldexp(double(c - lo), int(K - k));
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
        const double cl = s_excl[r * NW + wid];
        if (cl <= target && target < cl + s_cell[r * NW + wid]) {
            const double mylo = cl + off[r];
            if (fx[r] > 0.0 && mylo <= target && target < mylo + fx[r]) {
                const double want = target - mylo;
                float racc = mass[r][0];
                int pick = fixed40(racc) > want ? 0 : -1, last_pos = mass[r][0] > 0.0f ? 0 : -1;
#pragma unroll
                for (int e = 1; e < EPC; ++e) {
                    racc = racc + mass[r][e];
                    if (mass[r][e] > 0.0f) last_pos = e;
                    if (pick < 0 && fixed40(racc) > want) pick = e;
                }
                if (pick < 0) pick = last_pos >= 0 ? last_pos : 0;
                s_tok = ((s * SEG + r * W + tid) * EPC) + pick;
            }
        }
    }
    __syncthreads();
    if (tid == 0) a.out[n] = s_tok;
    arrive_row();
}

// kSamplePolls, or the value of OSD_SAMPLE_POLLS (read once; 0 makes every
// workgroup compute its siblings' records itself).
int sample_polls() {
    static const int v = [] {
        const char* e = getenv("OSD_SAMPLE_POLLS");
        if (e == nullptr || *e == 0) return kSamplePolls;
        const int k = atoi(e);
        return k < 0 ? kSamplePolls : (k > 65536 ? 65536 : k);
    }();
    return v;
}

template <typename Fmt, int CPT>
hipError_t launch_split(const SampleLaunch& L, const SampleArgs& a, int nchunks, int S) {
    SplitSampleArgs sa{};
    sa.row = a.p;
    sa.stride = a.p_stride;
    sa.N = a.N;
    sa.V = a.V;
    sa.nchunks = nchunks;
    sa.S = S;
    sa.polls = sample_polls();
    sa.c2 = a.c2;
    sa.u = a.u;
    sa.out = a.out;
    char* w = static_cast<char*>(L.workspace);
    sa.rec = reinterpret_cast<uint64_t*>(w);
    sa.cnt = reinterpret_cast<uint32_t*>(w + size_t(L.N) * kMaxSampleSegments * 16);
    return launch_kernel(&sample_split_kernel<Fmt, CPT>, dim3(unsigned(L.N) * unsigned(S)), dim3(kSegSampleW), 0,
                         L.stream, sa);
}

// The split applies to one-row sampling (T > 0, beta 0 or 1) of 16-byte rows
// when one workgroup per row would leave most CUs idle.
template <typename Fmt>
bool try_split(const SampleLaunch& L, const SampleArgs& a, hipError_t* e) {
    if (!L.workspace || !L.vec || !(L.temperature > 0.0f) || (L.beta > 0.0f && L.beta < 1.0f)) return false;
    if (L.N >= 2 * L.cus) return false;
    const int nchunks = (L.V + Fmt::kPerChunk - 1) / Fmt::kPerChunk;
    const int s2 = (nchunks + 2 * kSegSampleW - 1) / (2 * kSegSampleW);
    const int s4 = (nchunks + 4 * kSegSampleW - 1) / (4 * kSegSampleW);
    if (s2 >= 2 && s2 <= kMaxSampleSegments && int64_t(L.N) * s2 <= 4 * int64_t(L.cus)) {
        *e = launch_split<Fmt, 2>(L, a, nchunks, s2);
        return true;
    }
    if (s4 >= 2 && s4 <= kMaxSampleSegments && int64_t(L.N) * s4 <= 4 * int64_t(L.cus)) {
        *e = launch_split<Fmt, 4>(L, a, nchunks, s4);
        return true;
    }
    return false;
}

template <typename Fmt, int W, int CPT>
hipError_t launch_tile(const SampleLaunch& L, const SampleArgs& a) {
    if (L.temperature == 0.0f) return launch_mode<Fmt, W, CPT, kModeGreedy>(L, a);
    if (L.beta > 0.0f && L.beta < 1.0f) return launch_mode<Fmt, W, CPT, kModeMix>(L, a);
    return launch_mode<Fmt, W, CPT, kModeOne>(L, a);
}

template <typename Fmt>
hipError_t launch_fmt(const SampleLaunch& L, const SampleArgs& a) {
    hipError_t se;
    if (try_split<Fmt>(L, a, &se)) return se;
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
