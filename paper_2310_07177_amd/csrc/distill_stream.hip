// distill_stream.hip -- distillation divergence and its gradient with respect
// to the student logits on gfx950, streaming form (persistent workgroups)
// (Section 4.1, Eq. 2-4 of arXiv:2310.07177).
//
// For each row n = (b, i) with mask 1, with p = softmax(t / tau) (teacher) and
// q = softmax(s / tau) (student):
//   FKL  D = sum p (log p - log q)                  g = (q - p) / tau
//   RKL  D = sum q (log q - log p)                  g = q (log q - log p - D) / tau
//   JSD  D = beta KL(p || m) + (1-beta) KL(q || m)   g = (1-beta) q (log q - log m - KL(q || m)) / tau
//        with m = beta p + (1-beta) q
// and 0 log 0 = 0.  Rows with mask 0 get D = 0 and a zero gradient row.
//
// Work layout.  About one workgroup per CU walks the rows n = g, g+G, ...
// Each thread owns chunks n*W + tid of both rows.  The statistics pass
// consumes the raw chunks of row j while each register chunk is reloaded with
// the same chunk of row j+G; what the later passes need is kept per element in
// a cache of two floats (c0 in LDS, in thread-private float4 slots; c1 in
// registers), so the loss and gradient passes of row j run while row j+G is
// landing.  The statistics pass caches both exponents, (t c2 - K_t,
// s c2 - K_s), for every kind; the loss pass replaces them by
//   JSD  (log2 q - log2 m, q)
//   FKL  (p, log2 q)
//   RKL  (log2 p - log2 q, q)
// (c2 = log2(e)/tau, K a whole number per thread and row).  The log-ratio of
// FKL and RKL is the difference of the two cached exponents less the
// difference of the normalisers (taken in fp64), so it carries no rounding
// of the (much larger) normalisers themselves.
//
// Each workgroup adds the D of its rows in fp64 in row order and posts the
// partial at the device-wide coherence point; the last workgroup to finish
// adds the partials in workgroup order, so the loss is reproducible for a
// given grid.
#include "osd_device.hpp"
#include "osd_internal.hpp"
#include "stream_device.hpp"
#include "distill_common.hpp"

namespace osd {
namespace {

struct StreamDistillArgs {
    const void* teacher;
    int64_t tstride;
    const void* student;
    int64_t sstride;
    int B, K, V;
    const uint8_t* mask;
    float beta;
    float c2;       // log2(e) / tau
    float inv_tau;  // 1 / tau
    float* row_loss_out;
    void* grad_out;
    double* row_ws;     // [grid] per-workgroup loss partials, zero between calls
    uint32_t* done;     // workgroups finished, zero between calls
    float* loss_out;    // {masked mean, masked sum}
    int nrows;
    int nchunks;
    uint32_t row_bytes;
    int G;  // workgroups in the grid
};

struct Row {
    bool on;
    const char* trow;
    const char* srow;
};

// Row n, with its mask flag `on` (rows out of range are off).
template <typename Fmt>
__device__ inline Row decode_row(const StreamDistillArgs& a, int n, bool on) {
    Row r;
    r.on = false;
    r.trow = nullptr;
    r.srow = nullptr;
    if (n < 0 || n >= a.nrows) return r;
    r.on = on;
    const int b = n / a.K, i = n - b * a.K;
    r.trow = static_cast<const char*>(a.teacher) + (int64_t(b) * a.tstride + int64_t(i) * a.V) * Fmt::kBytes;
    r.srow = static_cast<const char*>(a.student) + (int64_t(b) * a.sstride + int64_t(i) * a.V) * Fmt::kBytes;
    return r;
}

template <typename Fmt, int W, int CPT, int KIND>
__global__ __launch_bounds__(W, 1) void distill_stream_kernel(StreamDistillArgs a) {
    constexpr int NW = W / kWave, EPC = Fmt::kPerChunk, NG = EPC / 4;
    // JSD caches exponentials (the others, exponents): see the statistics pass.
    constexpr bool XV = KIND == 2;
    __shared__ float s_k[2 * NW];
    __shared__ double s_s[2 * NW];
    __shared__ RowPair s_rp;
    __shared__ double s_a[2 * NW];
    __shared__ uint8_t s_on[W];
    __shared__ double s_part[1];  // sum of this workgroup's row divergences
    __shared__ LossTail s_tail;
    __shared__ f32x4_t s_c0[CPT * NG * W];
    const LdsCache<W, EPC> lc{s_c0};

    // Every argument word, requested together: each dependent request would
    // cost a round trip to the argument buffer (about a microsecond).
    asm volatile("" ::"s"(a.teacher), "s"(a.tstride), "s"(a.student), "s"(a.sstride), "s"(a.B), "s"(a.K), "s"(a.V),
                 "s"(a.mask), "s"(a.beta), "s"(a.c2), "s"(a.inv_tau));
    asm volatile("" ::"s"(a.row_loss_out), "s"(a.grad_out), "s"(a.row_ws), "s"(a.done), "s"(a.loss_out), "s"(a.nrows),
                 "s"(a.nchunks), "s"(a.row_bytes), "s"(a.G));
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int G = a.G;
    const float c2 = a.c2;
    const bool last_ok = (CPT - 1) * W + tid < a.nchunks;
    const float beta = a.beta, omb = 1.0f - a.beta;

    chunk_t rt[CPT], rs[CPT];
    float c1[CPT][EPC];

    // The mask flags of this workgroup's rows (thread j: row blockIdx.x +
    // j*G), loaded before any row data so that waiting for them never waits
    // for rows, and staged in LDS by step -1.  Nothing in the row loop then
    // reads global memory except the rows themselves (a scalar load there
    // would share its wait counter with LDS traffic).
    const int nk = (a.nrows - int(blockIdx.x) + G - 1) / G;
    if (tid == 0) {
        s_part[0] = 0.0;  // read and written by thread 0 only
        s_tail.row_ws = a.row_ws;
        s_tail.done = a.done;
        s_tail.loss_out = a.loss_out;
        s_tail.mask = a.mask;
        s_tail.nrows = a.nrows;
        s_tail.G = a.G;
    }
    uint32_t mine = 1u;
    if (a.mask && tid < nk) mine = a.mask[int(blockIdx.x) + tid * G];
    // The pipeline starts one step early: step -1 computes nothing; it issues
    // the loads of the workgroup's first row (read whatever its mask, which is
    // not known yet), from the same code as every later step (so the compiler
    // sees one load order throughout).
    Row cur;
    cur.on = false;
    cur.trow = nullptr;
    cur.srow = nullptr;
    for (int k = -1, n = int(blockIdx.x) - G; n < a.nrows; n += G, ++k) {
        const bool non = k < 0 ? true : (k + 1 < nk && s_on[k + 1] != 0);
        const Row nxt = decode_row<Fmt>(a, n + G, non);
        const rsrc_t ntr = make_rsrc(nxt.on ? nxt.trow : a.teacher, nxt.on ? a.row_bytes : 0u);
        const rsrc_t nsr = make_rsrc(nxt.on ? nxt.srow : a.student, nxt.on ? a.row_bytes : 0u);
        if (k >= 0) cur = decode_row<Fmt>(a, n, s_on[k] != 0);
        // The gradient row of the current row (0 bytes before the first row:
        // nothing is written).
        const bool has_row = n >= 0;
        const rsrc_t gr = make_rsrc(a.grad_out && has_row ? static_cast<char*>(a.grad_out) + int64_t(n) * a.row_bytes
                                                          : static_cast<char*>(nullptr),
                                    a.grad_out && has_row ? a.row_bytes : 0u);
        double D = 0.0;
        // ---- statistics pass: consumes the raw chunks and reloads each
        // with the next row's.  The loads are issued whether or not the row
        // is computed: a branch around them would make the compiler copy
        // registers with loads still in flight, which waits for all of them.
        const bool live = cur.on;
        float kc_t = 0.0f, kc_s = 0.0f;
        double S_t = 0.0, S_s = 0.0;
        if constexpr (XV) {
            // JSD caches each element's 2^(x c2 - k) itself, so the thread's
            // shift k is taken over all its chunks: every cached value is at
            // most 1 and no sum leaves the fp32 range.
            if (live) {
                const float mt = chunks_max<Fmt, CPT>(rt, !last_ok);
                const float ms = chunks_max<Fmt, CPT>(rs, !last_ok);
                kc_t = shift_of_max(mt, c2);
                kc_s = shift_of_max(ms, c2);
            }
        }
#pragma unroll
        for (int r = 0; r < CPT; ++r) {
            if (live) {
                chunk_t xt = rt[r], xs = rs[r];
                if (r == CPT - 1 && !last_ok) {
                    xt = pad_chunk<Fmt>();
                    xs = pad_chunk<Fmt>();
                }
                if (!XV && r == 0) {
                    kc_t = first_chunk_shift<Fmt>(xt, c2);
                    kc_s = first_chunk_shift<Fmt>(xs, c2);
                }
                float st = 0.0f, ss = 0.0f;
#pragma unroll
                for (int g = 0; g < NG; ++g) {
                    float c0v[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int e = 4 * g + j;
                        const float t = Fmt::get(xt, e), s = Fmt::get(xs, e);
                        const float vt = __builtin_fmaf(t, c2, -kc_t);
                        const float vs = __builtin_fmaf(s, c2, -kc_s);
                        const float et = exp2_fast(vt), es = exp2_fast(vs);
                        // (the first term starts the sums: 0 + x would cost an add)
                        st = e == 0 ? et : st + et;
                        ss = e == 0 ? es : ss + es;
                        if constexpr (XV) {
                            c0v[j] = et;
                            c1[r][e] = es;
                        } else {
                            // Both exponents: each side's probability is
                            // rebuilt from its own exponent, so a -inf logit
                            // on either side alone gives that side 0 and the
                            // other its true value.  One floor suffices: with
                            // the target's exponent finite, a draft exponent
                            // of -inf still gives q = 0, and two -inf
                            // exponents give a finite difference.
                            c0v[j] = fmaxf(vt, kLogFloor);
                            c1[r][e] = vs;
                        }
                    }
                    lc.store(r, g, f32x4_t{c0v[0], c0v[1], c0v[2], c0v[3]});
                }
                // Keep each round's sums in the round (without this the
                // compiler may defer one row's exponentials past the loop).
                asm volatile("" : "+v"(st), "+v"(ss));
                S_t = r == 0 ? double(st) : S_t + double(st);
                S_s = r == 0 ? double(ss) : S_s + double(ss);
            }
            rt[r] = load_chunk<W>(ntr, r);
            rs[r] = load_chunk<W>(nsr, r);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (k < 0) {  // step -1: stage the mask flags
            if (tid < nk) s_on[tid] = uint8_t(mine);  // the raw byte: no compare next to the load
            __syncthreads();
        }
        if (!live) {
            if (a.grad_out && has_row) {
#pragma unroll
                for (int r = 0; r < CPT; ++r) store_chunk<W>(gr, r, chunk_t{0u, 0u, 0u, 0u});
            }
        } else {
            // Exponent range exceeded by an element far above the first
            // chunk's maximum: rescale exactly from the cached exponents.
            float ks_t = kc_t, ks_s = kc_s;
            if (!XV && S_t >= 1.0e300) {  // (a NaN sum stays NaN: it marks a NaN logit)
                ks_t = kc_t + rescue_sum<CPT, EPC>(S_t, [&](int r, int e) -> float { return lc.load(r, e / 4)[e % 4]; });
            }
            if (!XV && S_s >= 1.0e300) {
                ks_s = kc_s + rescue_sum<CPT, EPC>(S_s, [&](int r, int e) -> float { return c1[r][e]; });
            }
            const RowPair rp = merge_row_pair<NW>(ks_t, S_t, ks_s, S_s, s_k, s_s, &s_rp);
            const float Kt = rp.kt, Ks = rp.ks;
            // log2 p_j = (t_j c2 - K_t) - (K_row_t - K_t + log2 S_t) = c - ct, likewise q.
            // T = K + log2 S, the rows' log2 normalisers; only their
            // difference is needed in fp64 (from the ratio of the sums).
            const double dTd = rp.dtd;
            const float ct = float(double(Kt - kc_t) + rp.lt), cs = float(double(Ks - kc_s) + rp.ls);
            // FKL/RKL: log2(p/q) = (v_t - v_s) - dTk, from the same rounded
            // exponents as the sums (so the normalisers and the log-ratios
            // agree: rows with p ~ q keep their small divergence accurate).
            const float dTk = float(dTd - double(kc_t - kc_s));
            // JSD: p = e_t at and q = e_s as, the cached values times the
            // thread's scale 2^(k - K) / S (fp64, rounded once).
            const float at = float(__builtin_ldexp(rp.ist, int(fmaxf(kc_t - Kt, -2048.0f))));
            const float as = float(__builtin_ldexp(rp.iss, int(fmaxf(kc_s - Ks, -2048.0f))));

            // ---- loss pass (from the cache) ----
            float acc0 = 0.0f, acc1 = 0.0f;
#pragma unroll
            for (int r = 0; r < CPT; ++r) {
                float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
                for (int g = 0; g < NG; ++g) {
                    const f32x4_t v = lc.load(r, g);
                    float c0v[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int e = 4 * g + j;
                        if constexpr (KIND == 2) {
                            const float p = c0v[j] * at, q = c1[r][e] * as;
                            // rho = q/p, clamped to 2^+-126 (both limits stay exact enough:
                            // the vanishing side carries no weight).  log2 m = log2 p + L,
                            // L = log2(beta + (1 - beta) rho): the mixture's log relative
                            // to p, a number near 0 when p ~ q, so the rounding of a log
                            // does not bias every term of a small divergence.  At beta = 0,
                            // L is d itself (the same log of the same value): x = 0.
                            const float rho = __builtin_amdgcn_fmed3f(
                                q * __builtin_amdgcn_rcpf(fmaxf(p, 0x1p-126f)), 0x1p-126f, 0x1p126f);
                            const float d = log2_fast(rho);
                            const float L = log2_fast(__builtin_fmaf(omb, rho, beta));
                            const float x = d - L;  // log2(q/m)
                            a0 = __builtin_fmaf(p, -L, a0);
                            a1 = __builtin_fmaf(q, x, a1);
                            c0v[j] = x;
                            c1[r][e] = q;
                        } else {
                            // log2(p/q) from the difference of the two
                            // exponents, clamped so that a zero probability
                            // times an infinite log-ratio stays 0.
                            const float lr = fmaxf(fminf((c0v[j] - c1[r][e]) - dTk, -kLogFloor), kLogFloor);
                            if constexpr (KIND == 0) {
                                const float p = exp2_fast(c0v[j] - ct);
                                a0 = __builtin_fmaf(p, lr, a0);
                                c0v[j] = p;
                                c1[r][e] = c1[r][e] - cs;  // log2 q
                            } else {
                                const float q = exp2_fast(c1[r][e] - cs);
                                a0 = __builtin_fmaf(q, lr, a0);
                                c0v[j] = lr;
                                c1[r][e] = q;
                            }
                        }
                    }
                    lc.store(r, g, f32x4_t{c0v[0], c0v[1], c0v[2], c0v[3]});
                }
                acc0 = acc0 + a0;
                acc1 = acc1 + a1;
                __builtin_amdgcn_sched_barrier(0);
            }
            double A0 = double(acc0), A1 = KIND == 2 ? double(acc1) : 0.0;
            block_sum2<NW>(A0, A1, s_a);
            // Terms were accumulated in log2 units.
            if constexpr (KIND == 2)
                D = kLn2 * (double(a.beta) * A0 + (1.0 - double(a.beta)) * A1);
            else if constexpr (KIND == 0)
                D = kLn2 * A0;
            else
                D = -kLn2 * A0;

            // ---- gradient pass (from the cache) ----
            if (a.grad_out) {
                const float ln2 = float(kLn2);
                // JSD: (1-beta) ln2/tau * q * (x - KL2);  RKL: ln2/tau * q * (A0 - lr)
                const float scale = KIND == 2 ? omb * ln2 * a.inv_tau : ln2 * a.inv_tau;
                const float shift = KIND == 2 ? float(A1) : float(A0);
#pragma unroll
                for (int r = 0; r < CPT; ++r) {
                    float g[EPC];
#pragma unroll
                    for (int q4 = 0; q4 < NG; ++q4) {
                        const f32x4_t v = lc.load(r, q4);
                        const float c0v[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const int e = 4 * q4 + j;
                            if constexpr (KIND == 0)
                                g[e] = (exp2_fast(c1[r][e]) - c0v[j]) * a.inv_tau;
                            else if constexpr (KIND == 2)
                                g[e] = (c1[r][e] * scale) * (c0v[j] - shift);
                            else
                                g[e] = (c1[r][e] * scale) * (shift - c0v[j]);
                        }
                    }
                    store_chunk<W>(gr, r, pack_grad<Fmt>(g));
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
        if (tid == 0 && n >= 0) {
            if (a.row_loss_out) a.row_loss_out[n] = float(D);
            s_part[0] += D;  // this workgroup's rows, in row order
        }
        cur = nxt;
    }
    finish_loss<W>(s_tail, s_part);
}

template <typename Fmt, int W, int CPT, int KIND>
int blocks_per_cu() {
    static const int v = [] {
        int nb = 0;
        const hipError_t e =
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, distill_stream_kernel<Fmt, W, CPT, KIND>, W, 0);
        return (e != hipSuccess || nb < 1) ? 1 : nb;
    }();
    return v;
}

template <typename Fmt, int W, int CPT, int KIND>
hipError_t launch_kind(const DistillLaunch& L, const StreamDistillArgs& a) {
    int64_t want = int64_t(L.cus) * blocks_per_cu<Fmt, W, CPT, KIND>();
    // At most W rows per workgroup: their mask flags are staged one per thread.
    const int64_t min_grid = (int64_t(a.nrows) + W - 1) / W;
    if (want < min_grid) want = min_grid;
    const unsigned grid = unsigned(want < a.nrows ? want : a.nrows);
    StreamDistillArgs ag = a;
    ag.G = int(grid);
    const hipError_t e = launch_kernel(&distill_stream_kernel<Fmt, W, CPT, KIND>, dim3(grid), dim3(W), 0, L.stream, ag);
    return e;
}

template <typename Fmt, int W, int CPT>
hipError_t launch_tile(const DistillLaunch& L, const StreamDistillArgs& a) {
    switch (L.kind) {
        case 0: return launch_kind<Fmt, W, CPT, 0>(L, a);
        case 1: return launch_kind<Fmt, W, CPT, 1>(L, a);
        default: return launch_kind<Fmt, W, CPT, 2>(L, a);
    }
}

template <typename Fmt>
hipError_t launch_fmt(const DistillLaunch& L, const StreamDistillArgs& a) {
    RowTile t;
    if (!pick_stream_tile(L.V, Fmt::kPerChunk, &t)) return hipErrorInvalidValue;
    switch (t.W * 100 + t.CPT) {
        case 25601: return launch_tile<Fmt, 256, 1>(L, a);
        case 51201: return launch_tile<Fmt, 512, 1>(L, a);
        case 102401: return launch_tile<Fmt, 1024, 1>(L, a);
        case 102402: return launch_tile<Fmt, 1024, 2>(L, a);
        case 102403: return launch_tile<Fmt, 1024, 3>(L, a);
        case 102404: return launch_tile<Fmt, 1024, 4>(L, a);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

// Streaming tiles, smallest first: up to 32768 bf16 or 16384 fp32 logits per
// row.  Registers hold the raw chunks in flight (and, in the distillation
// kernel, one float per element); the rest of a row's state lives in LDS.
bool pick_stream_tile(int V, int per_chunk, RowTile* t) {
    static const RowTile tiles[] = {{256, 1}, {512, 1}, {1024, 1}, {1024, 2}, {1024, 3}, {1024, 4}};
    for (const RowTile& c : tiles)
        if (int64_t(V) <= int64_t(c.W) * c.CPT * per_chunk) {
            *t = c;
            return true;
        }
    return false;
}

hipError_t launch_distill_stream(const DistillLaunch& L) {
    StreamDistillArgs a{};
    a.teacher = L.teacher;
    a.tstride = L.teacher_stride;
    a.student = L.student;
    a.sstride = L.student_stride;
    a.B = L.B;
    a.K = L.K;
    a.V = L.V;
    a.mask = L.mask;
    a.beta = L.beta;
    a.c2 = float(1.4426950408889634 / double(L.tau));
    a.inv_tau = float(1.0 / double(L.tau));
    a.row_loss_out = L.row_loss_out;
    a.grad_out = L.grad_out;
    a.row_ws = L.row_loss_ws;
    a.done = L.done_counter;
    a.loss_out = L.loss_out;
    a.nrows = L.B * L.K;
    const int eb = L.dtype == 1 ? 2 : 4;
    a.nchunks = int((int64_t(L.V) * eb) / 16);
    a.row_bytes = uint32_t(int64_t(L.V) * eb);
    return L.dtype == 1 ? launch_fmt<BF16>(L, a) : launch_fmt<F32>(L, a);
}

}  // namespace osd
