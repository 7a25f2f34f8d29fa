// distill_common.hpp -- pieces shared by the streaming distillation kernel
// and the fused verification + distillation kernel (gfx950): numerical
// floors, the bf16 gradient packer, the exponent-range rescue, the LDS half of
// the per-element cache, and the last-workgroup loss reduction.
#pragma once

#include "osd_device.hpp"
#include "stream_device.hpp"

namespace osd {

// Largest finite fp32 magnitude used to stand in for log2(0) = -inf, so that
// p * log2(p) stays 0 * finite = 0 for logits of -inf.
constexpr float kLogFloor = -1.0e30f;

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

// Rescale a thread's sum of 2^v over its cached exponents when the first
// chunk's shift left the fp32 range: returns the extra whole-number shift o
// and replaces S by sum 2^(v - o).  v(r, e) reads the exponent of element e
// of round r; rounds are processed one at a time (a scheduling barrier after
// each) so that the rarely taken branch adds few live registers.
template <int CPT, int EPC, typename VFn>
__device__ inline float rescue_sum(double& S, VFn v) {
    float m = kNegInf;
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
#pragma unroll
        for (int e = 0; e < EPC; ++e) m = fmaxf(m, v(r, e));
        __builtin_amdgcn_sched_barrier(0);
    }
    const float o = (m > -3.0e38f && m < 3.0e38f) ? ceilf(m) : 0.0f;
    S = 0.0;
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
        float t = 0.0f;
#pragma unroll
        for (int e = 0; e < EPC; ++e) t = t + exp2_fast(v(r, e) - o);
        S += double(t);
        __builtin_amdgcn_sched_barrier(0);
    }
    return o;
}

// A row pair's merged softmax statistics and the row-uniform values derived
// from them (fp64), computed once per row pair by wave 0 and read from LDS by
// every thread: K, S of each row, T_t - T_s (T = K + log2 S, the log2
// normalisers), 1/S and log2 S.
struct RowPair {
    float kt, ks;
    double st, ss, dtd, ist, iss, lt, ls;
};

// Every wave merges its lanes' (K, S) pairs and posts them; after one
// barrier wave 0 merges the waves' pairs and derives the row values; after a
// second, every thread reads them.  The values are those of block_merge2
// followed by the same formulas, bit for bit.
template <int NW>
__device__ inline RowPair merge_row_pair(float Kt, double St, float Ks, double Ss, float* s_k, double* s_s,
                                         RowPair* s_r) {
    static_assert(NW <= 16, "the posted pairs fit one DPP row");
    const int t = opaque_tid(), lane = t & (kWave - 1), wid = t / kWave;
    wave_merge_stats_u(Kt, St);
    wave_merge_stats_u(Ks, Ss);
    if (lane == 0) {
        s_k[wid] = Kt;
        s_k[NW + wid] = Ks;
        s_s[wid] = St;
        s_s[NW + wid] = Ss;
    }
    __syncthreads();
    if (wid == 0) {
        float k0 = kNegInf, k1 = kNegInf;
        double t0 = 0.0, t1 = 0.0;
        if (lane < NW) {
            k0 = s_k[lane];
            k1 = s_k[NW + lane];
            t0 = s_s[lane];
            t1 = s_s[NW + lane];
        }
        row0_merge_stats_u(k0, t0);
        row0_merge_stats_u(k1, t1);
        // The three quotients and the three logarithms are taken side by side
        // in lanes 0-2 (one division and one log2_pos in sequence instead of
        // three and three): lane 0 t0/t1, lane 1 1/t0, lane 2 1/t1, then the
        // log2 of t0/t1, t0 and t1.  Each value is the one the scalar formula
        // gives.
        const double qv = (lane == 0 ? t0 : 1.0) / (lane == 1 ? t0 : t1);
        const double lv = log2_pos(lane == 0 ? qv : (lane == 1 ? t0 : t1));
        const double l_q = readlane_f64(lv, 0), l_t = readlane_f64(lv, 1), l_s = readlane_f64(lv, 2);
        const double i_t = readlane_f64(qv, 1), i_s = readlane_f64(qv, 2);
        if (lane == 0) {
            RowPair r;
            r.kt = k0;
            r.ks = k1;
            r.st = t0;
            r.ss = t1;
            r.dtd = double(k0 - k1) + (t0 == t1 ? 0.0 : l_q);
            r.ist = i_t;
            r.iss = i_s;
            r.lt = l_t;
            r.ls = l_s;
            *s_r = r;
        }
    }
    __syncthreads();
    return *s_r;
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// The LDS half of the cache: element e of chunk r of this thread, in float4
// slots laid out [r][e/4][tid] so that a wave's accesses are contiguous.
template <int W, int EPC>
struct LdsCache {
    f32x4_t* base;
    __device__ f32x4_t load(int r, int g) const { return base[(r * (EPC / 4) + g) * W + threadIdx.x]; }
    __device__ void store(int r, int g, const f32x4_t& v) const { base[(r * (EPC / 4) + g) * W + threadIdx.x] = v; }
};

// Masked sum and mean of the row divergences.  Each workgroup adds its rows
// in row order (D = 0 for masked-out rows) and posts the partial at the
// device-wide coherence point; the last workgroup to finish adds the
// partials in workgroup order, counts the mask, writes the loss and zeroes
// what it read.  The result depends only on the grid size.
// What the tail needs, staged in LDS at kernel start so that none of it stays
// in registers across the row loop.
struct LossTail {
    double* row_ws;
    uint32_t* done;
    float* loss_out;
    const uint8_t* mask;
    int nrows;
    int G;  // workgroups in the grid
};

template <int W>
__device__ inline void finish_loss(const LossTail& a, const double* s_part) {
    __shared__ int s_last;
    __shared__ double s_sum[W / kWave], s_cnt[W / kWave];
    // Thread indices recomputed from an opaque copy: values derived from them
    // before the row loop are then not kept alive across it.
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & (kWave - 1), wid = tid / kWave;
    const int G = a.G;
    __syncthreads();
    if (tid == 0) {
        __hip_atomic_exchange(&a.row_ws[blockIdx.x], s_part[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = int(arrive(a.done)) == G - 1;  // after the post completed
    }
    __syncthreads();
    if (!s_last) return;
    // Thread t adds partials t, t+W, ... (one each when G <= W).
    double sm = 0.0, cn = 0.0;
    for (int g = tid; g < G; g += W) sm += take_f64(&a.row_ws[g]);
    for (int r = tid; r < a.nrows; r += W) cn += (a.mask == nullptr || a.mask[r] != 0) ? 1.0 : 0.0;
    sm = wave_sum(sm);
    cn = wave_sum(cn);
    if (lane == 0) {
        s_sum[wid] = sm;
        s_cnt[wid] = cn;
    }
    __syncthreads();
    if (tid == 0) {
        double ts = 0.0, tc = 0.0;
        for (int w = 0; w < W / kWave; ++w) {
            ts += s_sum[w];
            tc += s_cnt[w];
        }
        a.loss_out[0] = tc > 0.0 ? float(ts / tc) : 0.0f;
        a.loss_out[1] = float(ts);
        take_u32(a.done);
    }
}

}  // namespace osd
