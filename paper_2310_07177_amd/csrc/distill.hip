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
// split into segments of kSegChunks chunks, one 256-thread workgroup each,
// which keeps its segment of both rows in registers and cooperates with the
// other segments of its row through device memory:
//   1. each segment folds its (K, S) pair of both rows and publishes it;
//      every segment reads all the row's records and merges them in segment
//      order (the same normalisers in every workgroup);
//   2. each segment sums its divergence terms and publishes the partials;
//      FKL's gradient needs only the normalisers and is written here;
//   3. RKL and JSD read all the row's partials, add them in segment order and
//      write their gradient segment.
// Published words go out as plain agent-scope atomic stores that are never
// zero (each value is stored bit-inverted, and no value a segment publishes
// has all bits set), so a reader polls the words themselves: a zero word is
// not yet published.  Once a segment has read everything it needs it
// arrives at the row's counter; the last arriver adds the partials in
// segment order, writes the row's divergence, enters the masked-loss
// reduction and clears the row's words and counter (the workspace is left
// zero).  Rows with mask 0 write their zero gradient segments and take no
// part in the exchange.
//
// A wait is bounded (kSplitPolls polls, or the value of OSD_SPLIT_POLLS).  A
// workgroup whose siblings have not all published in time computes the
// missing records (or partials) itself, re-reading every segment of the row
// with the same thread layout and reduction order, so that the result is the
// same bit for bit; it still publishes and arrives, so the row completes as
// usual.
// The formulas are distill_kernel's.
constexpr int kSegW = 256;
constexpr int kSegCPT = 4;
constexpr int kSegChunks = kSegW * kSegCPT;
constexpr int kSplitPolls = 256;
constexpr int kSegNW = kSegW / kWave;

struct SplitArgs {
    DistillArgs d;
    uint64_t* rec;   // [rows, kMaxSplitSegments, 3]: ~S_t, ~S_s, ~(K_t | K_s << 32) (bits)
    uint64_t* part;  // [rows, kMaxSplitSegments, 2]: ~A0, ~A1 (bits)
    uint32_t* cnt;   // [rows, 4]: arrivals (word 0)
    int nseg;
    int nchunks;
    int polls;
};

struct SegShared {
    float k[2][kSegNW];
    double s[2][kSegNW];
    float rk[kMaxSplitSegments][2];   // records merged by this workgroup
    double rs[kMaxSplitSegments][2];
    double pa[kMaxSplitSegments][2];  // partials
    int flag;
};

__device__ inline bool row_on(const DistillArgs& a, int n) { return a.mask == nullptr || a.mask[n] != 0; }

template <typename Fmt>
__device__ inline const char* row_ptr(const void* base, int64_t stride, int n, int K, int V) {
    const int b = n / K, i = n - b * K;
    return static_cast<const char*>(base) + (int64_t(b) * stride + int64_t(i) * V) * Fmt::kBytes;
}

// Chunk r of this thread in segment s.
__device__ inline int seg_chunk(int s, int r) { return s * kSegChunks + r * kSegW + int(threadIdx.x); }

template <typename Fmt, bool VEC>
__device__ inline void seg_load(chunk_t (&x)[kSegCPT], const char* row, int s, int nchunks, int V) {
#pragma unroll
    for (int r = 0; r < kSegCPT; ++r) x[r] = stream_chunk<Fmt, VEC>(row, seg_chunk(s, r), nchunks, V);
}

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

// Segment statistics of both rows, reduced over the workgroup; slot `slot`
// of sh.rk / sh.rs receives them.  Opens with a barrier (sh.k, sh.s reuse).
// A segment's chunks come from a source: src(r, t, s) yields chunk r of
// this thread for both rows (held in registers, or loaded on demand -- the
// arithmetic is the same either way).
template <typename Fmt, int KIND, typename Src>
__device__ inline void seg_stats(Src src, float c2, SegShared& sh, int slot) {
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    float Kt = kNegInf, Ks = kNegInf;
    double dt = 0.0, ds = 0.0;
    if constexpr (KIND == 2) {
        float ft = 0.0f, fs = 0.0f;
#pragma unroll
        for (int r = 0; r < kSegCPT; ++r) {
            chunk_t ct, cs;
            src(r, ct, cs);
            fold_chunk<Fmt>(ct, c2, Kt, ft);
            fold_chunk<Fmt>(cs, c2, Ks, fs);
        }
        dt = ft;
        ds = fs;
    } else {
#pragma unroll
        for (int r = 0; r < kSegCPT; ++r) {
            chunk_t ct, cs;
            src(r, ct, cs);
            fold_chunk<Fmt>(ct, c2, Kt, dt);
            fold_chunk<Fmt>(cs, c2, Ks, ds);
        }
    }
    wave_merge_stats(Kt, dt);
    wave_merge_stats(Ks, ds);
    __syncthreads();
    if (lane == 0) {
        sh.k[0][wid] = Kt;
        sh.k[1][wid] = Ks;
        sh.s[0][wid] = dt;
        sh.s[1][wid] = ds;
    }
    __syncthreads();
    if (tid == 0) {  // one value at a time: few registers beside the held segment
        float kt = sh.k[0][0], ks = sh.k[1][0];
#pragma unroll 1
        for (int w = 1; w < kSegNW; ++w) {
            kt = fmaxf(kt, sh.k[0][w]);
            ks = fmaxf(ks, sh.k[1][w]);
        }
        double St = 0.0, Ss = 0.0;
#pragma unroll 1
        for (int w = 0; w < kSegNW; ++w) {
            St += rescale(sh.s[0][w], sh.k[0][w], kt);
            Ss += rescale(sh.s[1][w], sh.k[1][w], ks);
        }
        sh.rk[slot][0] = kt;
        sh.rk[slot][1] = ks;
        sh.rs[slot][0] = St;
        sh.rs[slot][1] = Ss;
    }
}

// A value every thread of the workgroup holds alike, kept in a scalar register.
__device__ inline float uniform_f32(float v) {
    return __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(v)));
}

// The row's normalisers in the forms distill_kernel uses, from the records
// in sh, merged in segment order.
struct RowNorm {
    float kt, ks, dk;
};
__device__ inline RowNorm merge_norm(const SegShared& sh, int nseg) {
    float Kt = kNegInf, Ks = kNegInf;
#pragma unroll 2
    for (int s = 0; s < nseg; ++s) {
        Kt = fmaxf(Kt, sh.rk[s][0]);
        Ks = fmaxf(Ks, sh.rk[s][1]);
    }
    double St = 0.0, Ss = 0.0;
#pragma unroll 2
    for (int s = 0; s < nseg; ++s) {
        St += rescale(sh.rs[s][0], sh.rk[s][0], Kt);
        Ss += rescale(sh.rs[s][1], sh.rk[s][1], Ks);
    }
    const double ktd = double(Kt) + log2(St), ksd = double(Ks) + log2(Ss);
    return RowNorm{uniform_f32(float(ktd)), uniform_f32(float(ksd)), uniform_f32(float(ktd - ksd))};
}

// The row's divergence from the partials in sh, added in segment order.
template <int KIND>
__device__ inline double merge_divergence(const SegShared& sh, int nseg, float beta, double& A1) {
    double A0 = 0.0;
    A1 = 0.0;
#pragma unroll 2
    for (int s = 0; s < nseg; ++s) {
        A0 += sh.pa[s][0];
        A1 += sh.pa[s][1];
    }
    if constexpr (KIND == 2)
        return kLn2 * (double(beta) * A0 + (1.0 - double(beta)) * A1);
    else
        return kLn2 * A0;
}

// The segment's divergence partials, reduced over the workgroup into slot
// `slot` of sh.pa.
template <typename Fmt, int KIND, typename Src>
__device__ inline void seg_partial(Src src, const RowNorm& rn, const DistillArgs& a, SegShared& sh, int slot) {
    constexpr int EPC = Fmt::kPerChunk;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const float c2 = a.c2, beta = a.beta, omb = 1.0f - a.beta;
    const bool q_only = a.beta == 0.0f;
    float acc0 = 0.0f, acc1 = 0.0f;
#pragma unroll
    for (int r = 0; r < kSegCPT; ++r) {
        float c0 = 0.0f, c1 = 0.0f;
        chunk_t ct, cs;
        src(r, ct, cs);
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
            const float t = Fmt::get(ct, e), sx = Fmt::get(cs, e);
            if constexpr (KIND == 0 || KIND == 1) {
                const float lr = fmaxf(fminf(__builtin_fmaf(t - sx, c2, -rn.dk), -kLogFloor), kLogFloor);
                if constexpr (KIND == 0) {
                    const float p = exp2_fast(__builtin_fmaf(t, c2, -rn.kt));
                    c0 = __builtin_fmaf(p, lr, c0);
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
            if ((e & 3) == 3) __builtin_amdgcn_sched_barrier(0);  // 4 elements in flight
        }
        acc0 = acc0 + c0;
        acc1 = acc1 + c1;
        __builtin_amdgcn_sched_barrier(0);
    }
    const double d0 = wave_sum(double(acc0)), d1 = wave_sum(double(acc1));
    __syncthreads();
    if (lane == 0) {
        sh.s[0][wid] = d0;
        sh.s[1][wid] = d1;
    }
    __syncthreads();
    if (tid == 0) {
        double A0 = 0.0, A1 = 0.0;
#pragma unroll 1
        for (int w = 0; w < kSegNW; ++w) {
            A0 += sh.s[0][w];
            A1 += sh.s[1][w];
        }
        sh.pa[slot][0] = A0;
        sh.pa[slot][1] = A1;
    }
}

template <typename Fmt, bool VEC, int KIND>
__device__ inline void seg_grad(const chunk_t (&xt)[kSegCPT], const chunk_t (&xs)[kSegCPT], const RowNorm& rn,
                                const DistillArgs& a, double D, double A1, void* grow, int s, int nchunks) {
    constexpr int EPC = Fmt::kPerChunk;
    const float c2 = a.c2, beta = a.beta, omb = 1.0f - a.beta;
    const bool q_only = a.beta == 0.0f;
    const float ln2 = float(kLn2);
    const float shift = uniform_f32(KIND == 1 ? float(D) : float(kLn2 * A1));
    const float scale = (KIND == 2 ? omb : 1.0f) * a.inv_tau;
#pragma unroll
    for (int r = 0; r < kSegCPT; ++r) {
        float g[EPC];
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
            const float lp = fmaxf(__builtin_fmaf(Fmt::get(xt[r], e), c2, -rn.kt), kLogFloor);
            const float lq = fmaxf(__builtin_fmaf(Fmt::get(xs[r], e), c2, -rn.ks), kLogFloor);
            const float q = exp2_fast(lq);
            if constexpr (KIND == 0) {
                g[e] = (q - exp2_fast(lp)) * scale;
            } else {
                float lr;
                if constexpr (KIND == 1) {
                    lr = lq - lp;
                } else {
                    const float d = __builtin_amdgcn_fmed3f(lq - lp, -126.0f, 126.0f);
                    lr = q_only ? 0.0f : d - log2_fast(__builtin_fmaf(omb, exp2_fast(d), beta));
                }
                g[e] = (q * scale) * __builtin_fmaf(lr, ln2, -shift);
            }
            if ((e & 3) == 3) __builtin_amdgcn_sched_barrier(0);
        }
        put_chunk<Fmt, VEC>(grow, seg_chunk(s, r), nchunks, pack_grad<Fmt>(g), a.V);
        __builtin_amdgcn_sched_barrier(0);
    }
}

__device__ inline uint64_t load_u64(const uint64_t* p) {
    return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void store_u64(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t pack_k(float kt, float ks) {
    return uint64_t(__float_as_uint(kt)) | (uint64_t(__float_as_uint(ks)) << 32);
}

// Wave 0 polls the published words of the row's other segments: lane j < nseg
// (j != s) reads the `words` words of segment j until every one is non-zero
// or the polls run out.  On success, lane j leaves them (un-inverted) in
// w[0..words).  Every thread gets the outcome.
template <int WORDS>
__device__ inline bool poll_words(const uint64_t* base, int nseg, int s, int polls, uint64_t (&w)[WORDS],
                                  SegShared& sh) {
    const int tid = threadIdx.x;
    if (tid < kWave) {
        const bool mine = tid < nseg && tid != s;
        bool ok = false;
        for (int p = 0; p < polls; ++p) {
            if (p > 0) __builtin_amdgcn_s_sleep(8);
            bool ready = true;
            if (mine) {
#pragma unroll
                for (int k = 0; k < WORDS; ++k) {
                    w[k] = load_u64(base + int64_t(tid) * WORDS + k);
                    ready = ready && w[k] != 0;
                }
            }
            if (__ballot(!ready) == 0) {
                ok = true;
                break;
            }
        }
#pragma unroll
        for (int k = 0; k < WORDS; ++k) w[k] = ~w[k];
        if (tid == 0) sh.flag = ok;
    }
    __syncthreads();
    return sh.flag != 0;
}

// Arrival at the row's counter once this workgroup's published words are
// complete; the returned count is awaited only where it is used.
__device__ inline uint32_t arrive_row(uint32_t* counter) {
    wait_memory();
    return __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename Fmt, bool VEC, int KIND>
__global__ __launch_bounds__(kSegW) void split_row_kernel(SplitArgs sa) {
    __shared__ SegShared sh;
    const DistillArgs& a = sa.d;
    const int nseg = sa.nseg, nchunks = sa.nchunks, V = a.V;
    const int n = blockIdx.x / nseg, s = blockIdx.x - n * nseg;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    void* grow = a.grad_out ? static_cast<char*>(a.grad_out) + int64_t(n) * V * Fmt::kBytes : nullptr;
    if (!row_on(a, n)) {
        if (grow) {
#pragma unroll
            for (int r = 0; r < kSegCPT; ++r) put_chunk<Fmt, VEC>(grow, seg_chunk(s, r), nchunks, chunk_t{0u, 0u, 0u, 0u}, V);
        }
        if (s == 0 && wid == 0) {
            if (a.row_loss_out && lane == 0) a.row_loss_out[n] = 0.0f;
            reduce_loss(a, n, 0.0);
        }
        return;
    }
    const char* trow = row_ptr<Fmt>(a.teacher, a.tstride, n, a.K, V);
    const char* srow = row_ptr<Fmt>(a.student, a.sstride, n, a.K, V);
    uint64_t* rec = sa.rec + int64_t(n) * kMaxSplitSegments * 3;
    uint64_t* part = sa.part + int64_t(n) * kMaxSplitSegments * 2;
    uint32_t* cnt = sa.cnt + int64_t(n) * 4;
    const float c2 = a.c2;

    chunk_t xt[kSegCPT], xs[kSegCPT];
    seg_load<Fmt, VEC>(xt, trow, s, nchunks, V);
    seg_load<Fmt, VEC>(xs, srow, s, nchunks, V);
    const auto held = [&](int r, chunk_t& ct, chunk_t& cs) {
        ct = xt[r];
        cs = xs[r];
    };

    // 1. statistics
    seg_stats<Fmt, KIND>(held, c2, sh, s);
    if (tid == 0) {
        store_u64(&rec[3 * s], ~uint64_t(__double_as_longlong(sh.rs[s][0])));
        store_u64(&rec[3 * s + 1], ~uint64_t(__double_as_longlong(sh.rs[s][1])));
        store_u64(&rec[3 * s + 2], ~pack_k(sh.rk[s][0], sh.rk[s][1]));
    }
    {
        uint64_t w[3];
        const bool ok = poll_words<3>(rec, nseg, s, sa.polls, w, sh);
        if (ok) {
            if (tid < nseg && tid != s) {
                sh.rs[tid][0] = __longlong_as_double(w[0]);
                sh.rs[tid][1] = __longlong_as_double(w[1]);
                sh.rk[tid][0] = __uint_as_float(uint32_t(w[2]));
                sh.rk[tid][1] = __uint_as_float(uint32_t(w[2] >> 32));
            }
        } else {
            for (int j = 0; j < nseg; ++j) {
                if (j == s) continue;
                const auto loaded = [&](int r, chunk_t& ct, chunk_t& cs) {
                    ct = stream_chunk<Fmt, VEC>(trow, seg_chunk(j, r), nchunks, V);
                    cs = stream_chunk<Fmt, VEC>(srow, seg_chunk(j, r), nchunks, V);
                };
                seg_stats<Fmt, KIND>(loaded, c2, sh, j);
            }
            // the segment is read again rather than held across the loop above
            seg_load<Fmt, VEC>(xt, trow, s, nchunks, V);
            seg_load<Fmt, VEC>(xs, srow, s, nchunks, V);
        }
    }
    __syncthreads();
    const RowNorm rn = merge_norm(sh, nseg);
    opaque(xt);  // each pass unpacks the held chunks afresh (bounded VGPRs)
    opaque(xs);

    // 2. divergence
    seg_partial<Fmt, KIND>(held, rn, a, sh, s);
    if (tid == 0) {
        store_u64(&part[2 * s], ~uint64_t(__double_as_longlong(sh.pa[s][0])));
        store_u64(&part[2 * s + 1], ~uint64_t(__double_as_longlong(sh.pa[s][1])));
    }
    uint32_t prev = 0;
    double D = 0.0, A1 = 0.0;
    if constexpr (KIND == 0) {
        if (tid == 0) prev = arrive_row(&cnt[0]);
        opaque(xt);
        opaque(xs);
        if (grow) seg_grad<Fmt, VEC, KIND>(xt, xs, rn, a, 0.0, 0.0, grow, s, nchunks);
    } else {
        // 3. gradient
        uint64_t w[2];
        const bool ok = poll_words<2>(part, nseg, s, sa.polls, w, sh);
        if (ok) {
            if (tid < nseg && tid != s) {
                sh.pa[tid][0] = __longlong_as_double(w[0]);
                sh.pa[tid][1] = __longlong_as_double(w[1]);
            }
        } else {
            for (int j = 0; j < nseg; ++j) {
                if (j == s) continue;
                const auto loaded = [&](int r, chunk_t& ct, chunk_t& cs) {
                    ct = stream_chunk<Fmt, VEC>(trow, seg_chunk(j, r), nchunks, V);
                    cs = stream_chunk<Fmt, VEC>(srow, seg_chunk(j, r), nchunks, V);
                };
                seg_partial<Fmt, KIND>(loaded, rn, a, sh, j);
            }
            seg_load<Fmt, VEC>(xt, trow, s, nchunks, V);
            seg_load<Fmt, VEC>(xs, srow, s, nchunks, V);
        }
        __syncthreads();
        if (tid == 0) prev = arrive_row(&cnt[0]);
        D = merge_divergence<KIND>(sh, nseg, a.beta, A1);
        opaque(xt);
        opaque(xs);
        if (grow) seg_grad<Fmt, VEC, KIND>(xt, xs, rn, a, D, A1, grow, s, nchunks);
    }
    if (tid == 0) sh.flag = prev == uint32_t(nseg - 1);
    __syncthreads();
    if (sh.flag == 0) return;
    // The row's last arriver: every segment has read what it needed.
    if constexpr (KIND == 0) {
        if (tid < nseg && tid != s) {
            sh.pa[tid][0] = __longlong_as_double(~load_u64(&part[2 * tid]));
            sh.pa[tid][1] = __longlong_as_double(~load_u64(&part[2 * tid + 1]));
        }
        __syncthreads();
        D = merge_divergence<KIND>(sh, nseg, a.beta, A1);
    }
    if (tid < nseg) {
        store_u64(&rec[3 * tid], 0ull);
        store_u64(&rec[3 * tid + 1], 0ull);
        store_u64(&rec[3 * tid + 2], 0ull);
        store_u64(&part[2 * tid], 0ull);
        store_u64(&part[2 * tid + 1], 0ull);
    }
    if (tid == 0) __hip_atomic_store(&cnt[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (wid == 0) {
        if (a.row_loss_out && lane == 0) a.row_loss_out[n] = float(D);
        reduce_loss(a, n, D);
    }
}

template <typename Fmt, bool VEC, int KIND>
hipError_t launch_split_kind(const DistillLaunch& L, const SplitArgs& sa) {
    const unsigned rows = unsigned(L.B) * unsigned(L.K);
    return launch_kernel(&split_row_kernel<Fmt, VEC, KIND>, dim3(rows * unsigned(sa.nseg)), dim3(kSegW), 0, L.stream,
                         sa);
}

// kSplitPolls, or the value of OSD_SPLIT_POLLS (read once; 0 makes every
// workgroup compute its row's records and partials itself).
int split_polls() {
    static const int v = [] {
        const char* e = getenv("OSD_SPLIT_POLLS");
        if (e == nullptr || *e == 0) return kSplitPolls;
        const int k = atoi(e);
        return k < 0 ? kSplitPolls : (k > 65536 ? 65536 : k);
    }();
    return v;
}

template <typename Fmt, bool VEC>
hipError_t launch_split(const DistillLaunch& L, const DistillArgs& a) {
    SplitArgs sa;
    sa.d = a;
    sa.nchunks = (L.V + Fmt::kPerChunk - 1) / Fmt::kPerChunk;
    sa.nseg = (sa.nchunks + kSegChunks - 1) / kSegChunks;
    if (sa.nseg > kMaxSplitSegments) return hipErrorInvalidValue;
    const size_t rows = size_t(L.B) * size_t(L.K);
    char* w = static_cast<char*>(L.split_ws);
    sa.rec = reinterpret_cast<uint64_t*>(w);
    sa.part = reinterpret_cast<uint64_t*>(w + rows * kMaxSplitSegments * 24);
    sa.cnt = reinterpret_cast<uint32_t*>(w + rows * kMaxSplitSegments * 40);
    sa.polls = split_polls();
    if (rows * size_t(sa.nseg) > size_t(0x7FFFFFFF)) return hipErrorInvalidValue;
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
    DistillArgs a{};
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
