// distill.hip -- distillation divergence and its gradient with respect to the
// student logits on gfx950 (Section 4.1, Eq. 2-4 of arXiv:2310.07177).
//
// For each row n = (b, i) with mask 1, with p = softmax(t / tau) (teacher) and
// q = softmax(s / tau) (student):
//   FKL  D = sum p (log p - log q)                  g = (q - p) / tau
//   RKL  D = sum q (log q - log p)                  g = q (log q - log p - D) / tau
//   JSD  D = beta KL(p || m) + (1-beta) KL(q || m)   g = (1-beta) q (log q - log m - KL(q || m)) / tau
//        with m = beta p + (1-beta) q
// and 0 log 0 = 0.  Rows with mask 0 get D = 0 and a zero gradient row.
//
// One workgroup per row.  Both rows are read from HBM once, 16 bytes per
// load, into registers; the row maxima and sums of exponentials are reduced
// across the workgroup, the divergence terms are accumulated in fp32 per
// thread and in fp64 across threads, and the gradient is written with 16-byte
// stores.  The scalar loss is reduced without floating-point atomics: each
// row stores its D, the last row of every 64-row slab to arrive sums its slab
// in a fixed order, and the last slab to arrive sums the slabs in a fixed
// order -- the result is bitwise reproducible.
#include "osd_device.hpp"
#include "osd_internal.hpp"

namespace osd {
namespace {

struct DistillArgs {
    const void* teacher;
    int64_t tstride;
    const void* student;
    int64_t sstride;
    int B, K, V;
    const uint8_t* mask;
    float beta;
    float c2;       // log2(e) / tau
    float inv_tau;  // 1 / tau
    float* loss_out;
    float* row_loss_out;
    void* grad_out;
    double* row_ws;    // [B*K]
    double* slab_ws;   // [2*nslabs]: {sum, count} per slab
    uint32_t* slab_cnt;
    uint32_t* done_cnt;
    int nslabs;
};

template <typename Fmt>
__device__ inline chunk_t pack_grad(const float (&g)[Fmt::kPerChunk]) {
    if constexpr (Fmt::kPerChunk == 8) {
        return chunk_t{pack_bf16x2(g[0], g[1]), pack_bf16x2(g[2], g[3]),
                       pack_bf16x2(g[4], g[5]), pack_bf16x2(g[6], g[7])};
    } else {
        return chunk_t{__float_as_uint(g[0]), __float_as_uint(g[1]),
                       __float_as_uint(g[2]), __float_as_uint(g[3])};
    }
}

template <typename Fmt, int W, int CPT, bool VEC>
__device__ inline void store_grad_chunk(void* row, int n, const chunk_t& c, int V) {
    const int nchunks = (V + Fmt::kPerChunk - 1) / Fmt::kPerChunk;
    const int ch = n * W + static_cast<int>(threadIdx.x);
    if (ch >= nchunks) return;
    if constexpr (VEC) {
        __builtin_nontemporal_store(c, static_cast<chunk_t*>(row) + ch);
    } else {
        const int64_t first = int64_t(ch) * Fmt::kPerChunk;
        if constexpr (Fmt::kPerChunk == 8) {
            uint16_t* p = static_cast<uint16_t*>(row);
            const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (first + e < V) p[first + e] = uint16_t((w[e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
        } else {
            uint32_t* p = static_cast<uint32_t*>(row);
            const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (first + e < V) p[first + e] = w[e];
        }
    }
}

// Wave-wide fp64 sum with a fixed butterfly: every lane ends with the same,
// run-to-run reproducible value.
__device__ inline double wave_sum_fixed(double v) { return wave_sum(v); }

// Executed by all lanes of wave 0: record D for row n and fold it into the
// masked sum once every row has arrived.  Up to kOneLevelRows rows, the last
// row to arrive sums them all (each lane a fixed strided subset, then a fixed
// butterfly); beyond that, rows are summed per 64-row slab first and the last
// slab to arrive sums the slabs.  Every order is fixed, so the result is
// reproducible bit for bit.
__device__ void finish_loss(const DistillArgs& a, double sum, double count) {
    const int lane = threadIdx.x & (kWave - 1);
    if (lane == 0) {
        a.loss_out[0] = count > 0.0 ? float(sum / count) : 0.0f;
        a.loss_out[1] = float(sum);
    }
}

__device__ void reduce_loss(const DistillArgs& a, int n, double D) {
    const int lane = threadIdx.x & (kWave - 1);
    const int rows = a.B * a.K;
    uint32_t prev = 0;
    if (rows <= kOneLevelRows) {
        if (lane == 0) {
            publish_f64(&a.row_ws[n], D);
            prev = arrive(a.done_cnt);
        }
        prev = __shfl(prev, 0, kWave);
        if (prev != uint32_t(rows - 1)) return;
        double v[kOneLevelRows / kWave];
#pragma unroll
        for (int k = 0; k < kOneLevelRows / kWave; ++k) {
            const int r = k * kWave + lane;
            v[k] = r < rows ? take_f64(&a.row_ws[r]) : 0.0;  // read and clear
        }
        double s = 0.0, c = 0.0;
#pragma unroll
        for (int k = 0; k < kOneLevelRows / kWave; ++k) {
            const int r = k * kWave + lane;
            s += v[k];
            c += (r < rows && (a.mask == nullptr || a.mask[r] != 0)) ? 1.0 : 0.0;
        }
        s = wave_sum_fixed(s);
        c = wave_sum_fixed(c);
        finish_loss(a, s, c);
        if (lane == 0) take_u32(a.done_cnt);
        return;
    }
    const int slab = n / kSlabRows;
    const int first = slab * kSlabRows;
    const int in_slab = min(kSlabRows, rows - first);
    if (lane == 0) {
        publish_f64(&a.row_ws[n], D);
        prev = arrive(&a.slab_cnt[slab]);
    }
    prev = __shfl(prev, 0, kWave);
    if (prev != uint32_t(in_slab - 1)) return;
    double v = 0.0, c = 0.0;
    if (lane < in_slab) {
        v = take_f64(&a.row_ws[first + lane]);  // read and clear
        c = (a.mask == nullptr || a.mask[first + lane] != 0) ? 1.0 : 0.0;
    }
    const double slab_sum = wave_sum_fixed(v);
    const double slab_cnt = wave_sum_fixed(c);
    if (lane == 0) {
        publish_f64(&a.slab_ws[2 * slab], slab_sum);
        publish_f64(&a.slab_ws[2 * slab + 1], slab_cnt);
        take_u32(&a.slab_cnt[slab]);
        prev = arrive(a.done_cnt);
    }
    prev = __shfl(prev, 0, kWave);
    if (prev != uint32_t(a.nslabs - 1)) return;
    double ts = 0.0, tc = 0.0;
    for (int s = lane; s < a.nslabs; s += kWave) {
        ts += take_f64(&a.slab_ws[2 * s]);
        tc += take_f64(&a.slab_ws[2 * s + 1]);
    }
    ts = wave_sum_fixed(ts);
    tc = wave_sum_fixed(tc);
    finish_loss(a, ts, tc);
    if (lane == 0) take_u32(a.done_cnt);
}

// Largest finite fp32 magnitude used to stand in for log2(0) = -inf, so that
// p * log2(p) stays 0 * finite = 0 for logits of -inf.
constexpr float kLogFloor = -1.0e30f;

template <typename Fmt, int W, int CPT, bool VEC, int KIND>
__global__ __launch_bounds__(W, min_waves_per_simd(W, CPT)) void distill_kernel(DistillArgs a) {
    constexpr int NW = W / kWave;
    constexpr int EPC = Fmt::kPerChunk;
    __shared__ float s_max[2][NW];
    __shared__ double s_sum[2][NW];

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int K = a.K, V = a.V;
    const int n = blockIdx.x;
    const int b = n / K, i = n - b * K;
    const bool on = a.mask == nullptr || a.mask[n] != 0;
    void* grow = a.grad_out ? static_cast<char*>(a.grad_out) + int64_t(n) * V * Fmt::kBytes : nullptr;
    double D = 0.0;

    if (!on) {
        if (grow) {
#pragma unroll
            for (int c = 0; c < CPT; ++c)
                store_grad_chunk<Fmt, W, CPT, VEC>(grow, c, chunk_t{0u, 0u, 0u, 0u}, V);
        }
    } else {
        const char* trow = static_cast<const char*>(a.teacher) +
                           (int64_t(b) * a.tstride + int64_t(i) * V) * Fmt::kBytes;
        const char* srow = static_cast<const char*>(a.student) +
                           (int64_t(b) * a.sstride + int64_t(i) * V) * Fmt::kBytes;
        chunk_t tv[CPT], sv[CPT];
        load_row<Fmt, W, CPT, VEC>(tv, trow, V);
        load_row<Fmt, W, CPT, VEC>(sv, srow, V);
        const float c2 = a.c2;

        // Row statistics (K, S), folded in chunk by chunk as the loads land.
        // FKL and RKL are first-order sensitive to the normaliser (an error s
        // in S shifts every log-ratio by s), so they accumulate every term in
        // fp64; JSD is not (the mixture absorbs a common scale error), so it
        // sums pairwise in fp32 within a chunk.
        float Kt = kNegInf, Ks = kNegInf;
        {
            double dt = 0.0, ds = 0.0;
            if constexpr (KIND == 2) {
                float ft = 0.0f, fs = 0.0f;
                row_stats<Fmt, CPT>(tv, c2, Kt, ft);
                row_stats<Fmt, CPT>(sv, c2, Ks, fs);
                dt = ft;
                ds = fs;
            } else {
                row_stats<Fmt, CPT>(tv, c2, Kt, dt);
                row_stats<Fmt, CPT>(sv, c2, Ks, ds);
            }
            wave_merge_stats(Kt, dt);
            wave_merge_stats(Ks, ds);
            if (lane == 0) {
                s_max[0][wid] = Kt;
                s_max[1][wid] = Ks;
                s_sum[0][wid] = dt;
                s_sum[1][wid] = ds;
            }
        }
        __syncthreads();
        Kt = s_max[0][0];
        Ks = s_max[1][0];
#pragma unroll
        for (int w = 1; w < NW; ++w) {
            Kt = fmaxf(Kt, s_max[0][w]);
            Ks = fmaxf(Ks, s_max[1][w]);
        }
        double St = 0.0, Ss = 0.0;
        for (int w = 0; w < NW; ++w) {
            St += rescale(s_sum[0][w], s_max[0][w], Kt);
            Ss += rescale(s_sum[1][w], s_max[1][w], Ks);
        }
        // log2 p_j = t_j c2 - (K_t + log2 S_t) and p_j = 2^(log2 p_j): one
        // fma and one exponential per element; likewise for q.
        const double ktd = double(Kt) + log2(St), ksd = double(Ks) + log2(Ss);
        const float kt = float(ktd), ks = float(ksd);
        // log2(p_j / q_j) = (t_j - s_j) c2 - (k_t - k_s): the difference of the
        // two constants is taken in fp64, so the loss of FKL and RKL carries no
        // rounding of the (much larger) constants themselves.
        const float dk = float(ktd - ksd);
        const float beta = a.beta, omb = 1.0f - a.beta;
        const bool q_only = a.beta == 0.0f;  // JSD at beta = 0: m = q, log2(q/m) = 0
        const float ln2 = float(kLn2);

        // Divergence terms, in log2 units.
        float kt_c = kt, ks_c = ks, dk_c = dk;
        asm volatile("" : "+v"(kt_c), "+v"(ks_c), "+v"(dk_c));
        opaque(tv);
        opaque(sv);
        float acc0 = 0.0f, acc1 = 0.0f;
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
            float c0 = 0.0f, c1 = 0.0f;
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float t = Fmt::get(tv[c], e), sx = Fmt::get(sv[c], e);
                if constexpr (KIND == 0 || KIND == 1) {
                    // log2(p/q), clamped so that a zero probability times an
                    // infinite log-ratio stays 0.
                    const float lr = fmaxf(fminf(__builtin_fmaf(t - sx, c2, -dk_c), -kLogFloor), kLogFloor);
                    if constexpr (KIND == 0) {
                        const float p = exp2_fast(__builtin_fmaf(t, c2, -kt_c));
                        c0 = __builtin_fmaf(p, lr, c0);
                    } else {
                        const float q = exp2_fast(__builtin_fmaf(sx, c2, -ks_c));
                        c0 = __builtin_fmaf(-q, lr, c0);
                    }
                } else {
                    const float lp = fmaxf(__builtin_fmaf(t, c2, -kt_c), kLogFloor);
                    const float lq = fmaxf(__builtin_fmaf(sx, c2, -ks_c), kLogFloor);
                    const float p = exp2_fast(lp), q = exp2_fast(lq);
                    // log2 m = lp + L, the mixture's log relative to p (near 0
                    // when p ~ q): its rounding does not bias a small JSD.
                    const float d = __builtin_amdgcn_fmed3f(lq - lp, -126.0f, 126.0f);
                    const float L = log2_fast(__builtin_fmaf(omb, exp2_fast(d), beta));
                    c0 = __builtin_fmaf(p, -L, c0);
                    c1 = __builtin_fmaf(q, q_only ? 0.0f : d - L, c1);  // log2(q/m); m = q at beta = 0
                }
                if ((e & 3) == 3) __builtin_amdgcn_sched_barrier(0);  // 4 elements in flight
            }
            acc0 = acc0 + c0;
            acc1 = acc1 + c1;
            __builtin_amdgcn_sched_barrier(0);
        }
        {
            const double d0 = wave_sum(double(acc0));
            const double d1 = wave_sum(double(acc1));
            __syncthreads();  // s_sum is reused
            if (lane == 0) {
                s_sum[0][wid] = d0;
                s_sum[1][wid] = d1;
            }
        }
        __syncthreads();
        double A0 = 0.0, A1 = 0.0;
        for (int w = 0; w < NW; ++w) {
            A0 += s_sum[0][w];
            A1 += s_sum[1][w];
        }
        // Terms were accumulated in log2 units.
        if constexpr (KIND == 2)
            D = kLn2 * (double(a.beta) * A0 + (1.0 - double(a.beta)) * A1);
        else
            D = kLn2 * A0;

        if (grow) {
            // FKL: g = (q - p) / tau;  RKL: g = q (ln q - ln p - D) / tau;
            // JSD: g = (1-beta) q (ln q - ln m - KL(q||m)) / tau.
            const float shift = KIND == 1 ? float(D) : float(kLn2 * A1);
            const float scale = (KIND == 2 ? omb : 1.0f) * a.inv_tau;
            float kt_g = kt, ks_g = ks;
            asm volatile("" : "+v"(kt_g), "+v"(ks_g));
            opaque(tv);
            opaque(sv);
#pragma unroll
            for (int c = 0; c < CPT; ++c) {
                float g[EPC];
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    const float lp = fmaxf(__builtin_fmaf(Fmt::get(tv[c], e), c2, -kt_g), kLogFloor);
                    const float lq = fmaxf(__builtin_fmaf(Fmt::get(sv[c], e), c2, -ks_g), kLogFloor);
                    const float q = exp2_fast(lq);
                    if constexpr (KIND == 0) {
                        g[e] = (q - exp2_fast(lp)) * scale;
                    } else {
                        float lr;
                        if constexpr (KIND == 1) {
                            lr = lq - lp;
                        } else {
                            // log2(q/m), as in the loss pass
                            const float d = __builtin_amdgcn_fmed3f(lq - lp, -126.0f, 126.0f);
                            lr = q_only ? 0.0f : d - log2_fast(__builtin_fmaf(omb, exp2_fast(d), beta));
                        }
                        g[e] = (q * scale) * __builtin_fmaf(lr, ln2, -shift);
                    }
                    if ((e & 3) == 3) __builtin_amdgcn_sched_barrier(0);
                }
                store_grad_chunk<Fmt, W, CPT, VEC>(grow, c, pack_grad<Fmt>(g), V);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }

    if (a.row_loss_out && tid == 0) a.row_loss_out[n] = float(D);
    if (wid == 0) reduce_loss(a, n, D);
}

// Rows too long to hold (beyond 8 chunks per thread of 1024 threads) are
// split into segments of kSegChunks chunks, each its own 256-thread
// workgroup, and the row is reduced across its segments in phases, one kernel
// each (so every row, masked or not, spreads over many CUs):
//   1. statistics: each segment's (K, S) of both rows -> SegRec; segments of
//      rows with mask 0 write their part of the zero gradient row instead;
//   2. divergence: each segment merges its row's S records in segment order
//      (every segment obtains the same normalisers), re-reads its part of the
//      row pair and sums its divergence terms -> SegPart; FKL, whose gradient
//      needs only the normalisers, writes its gradient segment here;
//   3. (RKL, JSD) gradient: each segment adds the row's partials in segment
//      order and writes its gradient segment;
//   F. one wave per row adds the partials (in the same order), writes the
//      row's divergence, enters the masked-loss reduction, and clears the
//      records and partials it read (the workspace is left zero; every
//      record and partial a phase reads was written by an earlier phase of
//      the same call, so nothing depends on that).
// The formulas are distill_kernel's.  Re-reads of a segment follow its first
// read closely (Infinity Cache).
constexpr int kSegW = 256;
constexpr int kSegCPT = 4;
constexpr int kSegChunks = kSegW * kSegCPT;

struct SegRec {
    double st, ss;
    float kt, ks;
    double pad;
};
static_assert(sizeof(SegRec) == 32, "two records per 64 bytes");

struct SplitArgs {
    DistillArgs d;
    SegRec* rec;     // [rows, nseg]
    double* part;    // [rows, nseg, 2]
    int nseg;
    int nchunks;
};

__device__ inline bool row_on(const DistillArgs& a, int n) { return a.mask == nullptr || a.mask[n] != 0; }

template <typename Fmt>
__device__ inline const char* row_ptr(const void* base, int64_t stride, int n, int K, int V) {
    const int b = n / K, i = n - b * K;
    return static_cast<const char*>(base) + (int64_t(b) * stride + int64_t(i) * V) * Fmt::kBytes;
}

// The row's normalisers from its segments' records, merged in segment order
// (the same result in every workgroup that reads them).
__device__ inline void merge_records(const SegRec* r, int nseg, float& Kt, double& St, float& Ks, double& Ss) {
    Kt = Ks = kNegInf;
    for (int s = 0; s < nseg; ++s) {
        Kt = fmaxf(Kt, r[s].kt);
        Ks = fmaxf(Ks, r[s].ks);
    }
    St = Ss = 0.0;
    for (int s = 0; s < nseg; ++s) {
        St += rescale(r[s].st, r[s].kt, Kt);
        Ss += rescale(r[s].ss, r[s].ks, Ks);
    }
}

// The row's divergence from its segments' partials, in segment order.
template <int KIND>
__device__ inline double row_divergence(const double* part, int nseg, float beta, double& A1) {
    double A0 = 0.0;
    A1 = 0.0;
    for (int s = 0; s < nseg; ++s) {
        A0 += part[2 * s];
        A1 += part[2 * s + 1];
    }
    if constexpr (KIND == 2)
        return kLn2 * (double(beta) * A0 + (1.0 - double(beta)) * A1);
    else
        return kLn2 * A0;
}

// Chunk r of this thread in segment s.
__device__ inline int seg_chunk(int s, int r) { return s * kSegChunks + r * kSegW + int(threadIdx.x); }

template <typename Fmt, bool VEC>
__device__ inline void put_chunk(void* row, int ch, int nchunks, const chunk_t& c, int V) {
    if (ch >= nchunks) return;
    if constexpr (VEC) {
        __builtin_nontemporal_store(c, static_cast<chunk_t*>(row) + ch);
    } else {
        const int64_t first = int64_t(ch) * Fmt::kPerChunk;
        const uint32_t w[4] = {c.x, c.y, c.z, c.w};
        if constexpr (Fmt::kPerChunk == 8) {
            uint16_t* p = static_cast<uint16_t*>(row);
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (first + e < V) p[first + e] = uint16_t((w[e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
        } else {
            uint32_t* p = static_cast<uint32_t*>(row);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (first + e < V) p[first + e] = w[e];
        }
    }
}

// Workgroup totals of two doubles (every thread gets them).
__device__ inline void seg_sum2(double& x, double& y, double* s_a) {
    constexpr int NW = kSegW / kWave;
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    x = wave_sum(x);
    y = wave_sum(y);
    if (lane == 0) {
        s_a[wid] = x;
        s_a[NW + wid] = y;
    }
    __syncthreads();
    x = 0.0;
    y = 0.0;
    for (int w = 0; w < NW; ++w) {
        x += s_a[w];
        y += s_a[NW + w];
    }
}

template <typename Fmt, bool VEC, int KIND>
__global__ __launch_bounds__(kSegW) void split_stats_kernel(SplitArgs sa) {
    constexpr int NW = kSegW / kWave, EPC = Fmt::kPerChunk;
    __shared__ float s_k[2][NW];
    __shared__ double s_s[2][NW];
    const DistillArgs& a = sa.d;
    const int n = blockIdx.x / sa.nseg, s = blockIdx.x - n * sa.nseg;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int K = a.K, V = a.V, nchunks = sa.nchunks;
    if (!row_on(a, n)) {
        if (a.grad_out) {
            void* grow = static_cast<char*>(a.grad_out) + int64_t(n) * V * Fmt::kBytes;
#pragma unroll
            for (int r = 0; r < kSegCPT; ++r) put_chunk<Fmt, VEC>(grow, seg_chunk(s, r), nchunks, chunk_t{0u, 0u, 0u, 0u}, V);
        }
        return;
    }
    const char* trow = row_ptr<Fmt>(a.teacher, a.tstride, n, K, V);
    const char* srow = row_ptr<Fmt>(a.student, a.sstride, n, K, V);
    chunk_t xt[kSegCPT], xs[kSegCPT];
#pragma unroll
    for (int r = 0; r < kSegCPT; ++r) {
        xt[r] = stream_chunk<Fmt, VEC>(trow, seg_chunk(s, r), nchunks, V);
        xs[r] = stream_chunk<Fmt, VEC>(srow, seg_chunk(s, r), nchunks, V);
    }
    const float c2 = a.c2;
    float Kt = kNegInf, Ks = kNegInf;
    double dt = 0.0, ds = 0.0;
    if constexpr (KIND == 2) {
        float ft = 0.0f, fs = 0.0f;
#pragma unroll
        for (int r = 0; r < kSegCPT; ++r) {
            fold_chunk<Fmt>(xt[r], c2, Kt, ft);
            fold_chunk<Fmt>(xs[r], c2, Ks, fs);
        }
        dt = ft;
        ds = fs;
    } else {
#pragma unroll
        for (int r = 0; r < kSegCPT; ++r) {
            fold_chunk<Fmt>(xt[r], c2, Kt, dt);
            fold_chunk<Fmt>(xs[r], c2, Ks, ds);
        }
    }
    wave_merge_stats(Kt, dt);
    wave_merge_stats(Ks, ds);
    if (lane == 0) {
        s_k[0][wid] = Kt;
        s_k[1][wid] = Ks;
        s_s[0][wid] = dt;
        s_s[1][wid] = ds;
    }
    __syncthreads();
    if (tid == 0) {
        float kt = s_k[0][0], ks = s_k[1][0];
        for (int w = 1; w < NW; ++w) {
            kt = fmaxf(kt, s_k[0][w]);
            ks = fmaxf(ks, s_k[1][w]);
        }
        double St = 0.0, Ss = 0.0;
        for (int w = 0; w < NW; ++w) {
            St += rescale(s_s[0][w], s_k[0][w], kt);
            Ss += rescale(s_s[1][w], s_k[1][w], ks);
        }
        SegRec r;
        r.st = St;
        r.ss = Ss;
        r.kt = kt;
        r.ks = ks;
        r.pad = 0.0;
        sa.rec[int64_t(n) * sa.nseg + s] = r;
    }
}

// The row's normalisers in the forms distill_kernel uses.
struct RowNorm {
    float kt, ks, dk;
};
__device__ inline RowNorm row_norm(const SplitArgs& sa, int n) {
    float Kt, Ks;
    double St, Ss;
    merge_records(sa.rec + int64_t(n) * sa.nseg, sa.nseg, Kt, St, Ks, Ss);
    const double ktd = double(Kt) + log2(St), ksd = double(Ks) + log2(Ss);
    return RowNorm{float(ktd), float(ksd), float(ktd - ksd)};
}

template <typename Fmt, bool VEC, int KIND>
__global__ __launch_bounds__(kSegW) void split_loss_kernel(SplitArgs sa) {
    constexpr int NW = kSegW / kWave, EPC = Fmt::kPerChunk;
    __shared__ double s_a[2 * NW];
    const DistillArgs& a = sa.d;
    const int n = blockIdx.x / sa.nseg, s = blockIdx.x - n * sa.nseg;
    if (!row_on(a, n)) return;
    const int K = a.K, V = a.V, nchunks = sa.nchunks;
    const char* trow = row_ptr<Fmt>(a.teacher, a.tstride, n, K, V);
    const char* srow = row_ptr<Fmt>(a.student, a.sstride, n, K, V);
    chunk_t xt[kSegCPT], xs[kSegCPT];
#pragma unroll
    for (int r = 0; r < kSegCPT; ++r) {
        xt[r] = stream_chunk<Fmt, VEC>(trow, seg_chunk(s, r), nchunks, V);
        xs[r] = stream_chunk<Fmt, VEC>(srow, seg_chunk(s, r), nchunks, V);
    }
    const RowNorm rn = row_norm(sa, n);
    const float c2 = a.c2, beta = a.beta, omb = 1.0f - a.beta;
    const bool q_only = a.beta == 0.0f;
    void* grow = a.grad_out ? static_cast<char*>(a.grad_out) + int64_t(n) * V * Fmt::kBytes : nullptr;
    float acc0 = 0.0f, acc1 = 0.0f;
#pragma unroll
    for (int r = 0; r < kSegCPT; ++r) {
        float c0 = 0.0f, c1 = 0.0f;
        float g[EPC];
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
            const float t = Fmt::get(xt[r], e), sx = Fmt::get(xs[r], e);
            if constexpr (KIND == 0 || KIND == 1) {
                const float lr = fmaxf(fminf(__builtin_fmaf(t - sx, c2, -rn.dk), -kLogFloor), kLogFloor);
                if constexpr (KIND == 0) {
                    const float p = exp2_fast(__builtin_fmaf(t, c2, -rn.kt));
                    c0 = __builtin_fmaf(p, lr, c0);
                    const float q = exp2_fast(fmaxf(__builtin_fmaf(sx, c2, -rn.ks), kLogFloor));
                    g[e] = (q - p) * a.inv_tau;
                } else {
                    const float q = exp2_fast(__builtin_fmaf(sx, c2, -rn.ks));
                    c0 = __builtin_fmaf(-q, lr, c0);
                }
            } else {
                const float lp = fmaxf(__builtin_fmaf(t, c2, -rn.kt), kLogFloor);
                const float lq = fmaxf(__builtin_fmaf(sx, c2, -rn.ks), kLogFloor);
                const float p = exp2_fast(lp), q = exp2_fast(lq);
                const float d = __builtin_amdgcn_fmed3f(lq - lp, -126.0f, 126.0f);
                const float L = log2_fast(__builtin_fmaf(omb, exp2_fast(d), beta));
                c0 = __builtin_fmaf(p, -L, c0);
                c1 = __builtin_fmaf(q, q_only ? 0.0f : d - L, c1);
            }
        }
        acc0 = acc0 + c0;
        acc1 = acc1 + c1;
        if constexpr (KIND == 0) {
            if (grow) put_chunk<Fmt, VEC>(grow, seg_chunk(s, r), nchunks, pack_grad<Fmt>(g), V);
        }
    }
    double A0 = double(acc0), A1 = double(acc1);
    seg_sum2(A0, A1, s_a);
    if (threadIdx.x == 0) {
        double* p = sa.part + (int64_t(n) * sa.nseg + s) * 2;
        p[0] = A0;
        p[1] = A1;
    }
}

template <typename Fmt, bool VEC, int KIND>
__global__ __launch_bounds__(kSegW) void split_grad_kernel(SplitArgs sa) {
    constexpr int EPC = Fmt::kPerChunk;
    const DistillArgs& a = sa.d;
    const int n = blockIdx.x / sa.nseg, s = blockIdx.x - n * sa.nseg;
    if (!row_on(a, n) || !a.grad_out) return;
    const int K = a.K, V = a.V, nchunks = sa.nchunks;
    const char* trow = row_ptr<Fmt>(a.teacher, a.tstride, n, K, V);
    const char* srow = row_ptr<Fmt>(a.student, a.sstride, n, K, V);
    chunk_t xt[kSegCPT], xs[kSegCPT];
#pragma unroll
    for (int r = 0; r < kSegCPT; ++r) {
        xt[r] = stream_chunk<Fmt, VEC>(trow, seg_chunk(s, r), nchunks, V);
        xs[r] = stream_chunk<Fmt, VEC>(srow, seg_chunk(s, r), nchunks, V);
    }
    const RowNorm rn = row_norm(sa, n);
    double A1;
    const double D = row_divergence<KIND>(sa.part + int64_t(n) * sa.nseg * 2, sa.nseg, a.beta, A1);
    const float c2 = a.c2, beta = a.beta, omb = 1.0f - a.beta;
    const bool q_only = a.beta == 0.0f;
    const float ln2 = float(kLn2);
    const float shift = KIND == 1 ? float(D) : float(kLn2 * A1);
    const float scale = (KIND == 2 ? omb : 1.0f) * a.inv_tau;
    void* grow = static_cast<char*>(a.grad_out) + int64_t(n) * V * Fmt::kBytes;
#pragma unroll
    for (int r = 0; r < kSegCPT; ++r) {
        float g[EPC];
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
            const float lp = fmaxf(__builtin_fmaf(Fmt::get(xt[r], e), c2, -rn.kt), kLogFloor);
            const float lq = fmaxf(__builtin_fmaf(Fmt::get(xs[r], e), c2, -rn.ks), kLogFloor);
            const float q = exp2_fast(lq);
            float lr;
            if constexpr (KIND == 1) {
                lr = lq - lp;
            } else {
                const float d = __builtin_amdgcn_fmed3f(lq - lp, -126.0f, 126.0f);
                lr = q_only ? 0.0f : d - log2_fast(__builtin_fmaf(omb, exp2_fast(d), beta));
            }
            g[e] = (q * scale) * __builtin_fmaf(lr, ln2, -shift);
        }
        put_chunk<Fmt, VEC>(grow, seg_chunk(s, r), nchunks, pack_grad<Fmt>(g), V);
    }
}

// One wave per row: the row's divergence, the masked-loss reduction, and the
// records and partials cleared.
template <int KIND>
__global__ __launch_bounds__(kWave) void split_finish_kernel(SplitArgs sa) {
    const DistillArgs& a = sa.d;
    const int n = blockIdx.x;
    const int lane = threadIdx.x;
    const bool on = row_on(a, n);
    double D = 0.0;
    if (on) {
        double A1;
        D = row_divergence<KIND>(sa.part + int64_t(n) * sa.nseg * 2, sa.nseg, a.beta, A1);
    }
    if (a.row_loss_out && lane == 0) a.row_loss_out[n] = float(D);
    if (on) {
        // Rows with mask 0 wrote neither.
        for (int j = lane; j < sa.nseg; j += kWave) {
            SegRec z;
            z.st = z.ss = 0.0;
            z.kt = z.ks = 0.0f;
            z.pad = 0.0;
            sa.rec[int64_t(n) * sa.nseg + j] = z;
            sa.part[(int64_t(n) * sa.nseg + j) * 2] = 0.0;
            sa.part[(int64_t(n) * sa.nseg + j) * 2 + 1] = 0.0;
        }
    }
    reduce_loss(a, n, D);
}

template <typename Fmt, bool VEC, int KIND>
hipError_t launch_split_kind(const DistillLaunch& L, const SplitArgs& sa) {
    const unsigned rows = unsigned(L.B) * unsigned(L.K);
    const dim3 grid(rows * unsigned(sa.nseg)), block(kSegW);
    hipError_t e = launch_kernel(&split_stats_kernel<Fmt, VEC, KIND>, grid, block, 0, L.stream, sa);
    if (e != hipSuccess) return e;
    e = launch_kernel(&split_loss_kernel<Fmt, VEC, KIND>, grid, block, 0, L.stream, sa);
    if (e != hipSuccess) return e;
    if constexpr (KIND != 0) {
        e = launch_kernel(&split_grad_kernel<Fmt, VEC, KIND>, grid, block, 0, L.stream, sa);
        if (e != hipSuccess) return e;
    }
    return launch_kernel(&split_finish_kernel<KIND>, dim3(rows), dim3(kWave), 0, L.stream, sa);
}

template <typename Fmt, bool VEC>
hipError_t launch_split(const DistillLaunch& L, const DistillArgs& a) {
    SplitArgs sa;
    sa.d = a;
    sa.nchunks = (L.V + Fmt::kPerChunk - 1) / Fmt::kPerChunk;
    sa.nseg = (sa.nchunks + kSegChunks - 1) / kSegChunks;
    if (sa.nseg > kMaxSplitSegments) return hipErrorInvalidValue;
    sa.rec = static_cast<SegRec*>(L.split_ws);
    sa.part = reinterpret_cast<double*>(static_cast<char*>(L.split_ws) +
                                        size_t(L.B) * size_t(L.K) * kMaxSplitSegments * sizeof(SegRec));
    switch (L.kind) {
        case 0: return launch_split_kind<Fmt, VEC, 0>(L, sa);
        case 1: return launch_split_kind<Fmt, VEC, 1>(L, sa);
        default: return launch_split_kind<Fmt, VEC, 2>(L, sa);
    }
}

template <typename Fmt, int W, int CPT, bool VEC>
hipError_t launch_kind(const DistillLaunch& L, const DistillArgs& a) {
    const dim3 grid(unsigned(L.B) * unsigned(L.K)), block(W);
    hipError_t e;
    switch (L.kind) {
        case 0: e = launch_kernel(&distill_kernel<Fmt, W, CPT, VEC, 0>, grid, block, 0, L.stream, a); break;
        case 1: e = launch_kernel(&distill_kernel<Fmt, W, CPT, VEC, 1>, grid, block, 0, L.stream, a); break;
        default: e = launch_kernel(&distill_kernel<Fmt, W, CPT, VEC, 2>, grid, block, 0, L.stream, a); break;
    }
    return e;
}

template <typename Fmt, int W, int CPT>
hipError_t launch_tile(const DistillLaunch& L, const DistillArgs& a) {
    return L.vec ? launch_kind<Fmt, W, CPT, true>(L, a) : launch_kind<Fmt, W, CPT, false>(L, a);
}

template <typename Fmt>
hipError_t launch_fmt(const DistillLaunch& L, const DistillArgs& a) {
    RowTile t;
    if (!pick_tile(L.V, Fmt::kPerChunk, &t))
        return L.vec ? launch_split<Fmt, true>(L, a) : launch_split<Fmt, false>(L, a);
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

hipError_t launch_distill(const DistillLaunch& L) {
    DistillArgs a;
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
    a.loss_out = L.loss_out;
    a.row_loss_out = L.row_loss_out;
    a.grad_out = L.grad_out;
    a.row_ws = L.row_loss_ws;
    a.slab_ws = L.slab_ws;
    a.slab_cnt = L.slab_counters;
    a.done_cnt = L.done_counter;
    a.nslabs = (L.B * L.K + kSlabRows - 1) / kSlabRows;
    return L.dtype == 1 ? launch_fmt<BF16>(L, a) : launch_fmt<F32>(L, a);
}

}  // namespace osd
