// verify_greedy.hip -- greedy verification (T = 0) on gfx950.
//
// Method: with T = 0 the target distribution is its argmax (lowest index on
// ties); proposal y_i is accepted while it equals the argmax of target row
// i, the first mismatch at position a ends the test (the exit of the
// acceptance loop in Appendix A.1), and the extra token is the argmax of row
// a, or of the bonus row k_b when every proposal matched.  Only target rows
// are read.
//
// Work layout: two flat grids of small workgroups, so the hardware
// dispatcher balances the work over every CU whatever B and k are.
//  1. verify_greedy_stats -- one workgroup per (target row, vocabulary
//     segment of kW*4 chunks): the segment's (max, lowest index) partial.
//     This kernel moves every byte the method reads.
//  2. verify_greedy_decide -- one workgroup per sequence: stages the
//     partials of rows 0..k_b in LDS, merges them in segment order, finds the
//     first mismatch and writes the outputs, then zeroes the partials.
#include "osd.h"
#include "osd_device.hpp"
#include "osd_internal.hpp"
#include "stream_device.hpp"

namespace osd {
namespace {

constexpr int kW = 256;          // threads per workgroup
constexpr int kNW = kW / kWave;  // waves per workgroup
// Workgroups per launch (grid sizes stay far below the 2^32 work-item limit).
constexpr int64_t kMaxGrid = int64_t(1) << 22;

struct SegArgs {
    const void* target;        // [B, K+1, V]
    int B, K, V;
    const int32_t* tokens;     // [B, K]
    const int32_t* draft_len;  // [B] or null
    int nseg;                  // segments per row
    int nchunks;               // 16-byte chunks per row
    uint32_t row_bytes;
    int64_t first;             // first work unit of this launch
    SegStats* stats;           // [B*(K+1), kMaxSeg] argmax partials, zero between calls
    int32_t* accepted_len;
    int32_t* out_tokens;
    uint8_t* reject_mask;
};

// Load this thread's chunks of segment `s` of a row (zeros past the end of
// the row: the caller pads them).  A null row issues loads of 0 bytes.
template <int CPT>
__device__ inline void load_segment(chunk_t (&x)[CPT], const char* row, const SegArgs& a, int s) {
    const uint32_t off = uint32_t(s) * uint32_t(kW * CPT * 16);
    const rsrc_t r = make_rsrc(row ? row + off : static_cast<const char*>(a.target), row ? a.row_bytes - off : 0u);
#pragma unroll
    for (int n = 0; n < CPT; ++n) x[n] = load_chunk<kW>(r, n);
}

// Chunks past the end of the row become -inf (zero probability).
template <typename Fmt, int CPT>
__device__ inline void pad_segment(chunk_t (&x)[CPT], const SegArgs& a, int s) {
#pragma unroll
    for (int n = 0; n < CPT; ++n)
        if (s * kW * CPT + n * kW + int(threadIdx.x) >= a.nchunks) x[n] = pad_chunk<Fmt>();
}

__device__ inline int seq_k(const SegArgs& a, int b) { return a.draft_len ? scalar_load(a.draft_len + b) : a.K; }

// Every argument word, requested together on entry: each dependent request
// would cost a round trip to the argument buffer (about a microsecond).
__device__ inline void request_args(const SegArgs& a) {
    asm volatile("" ::"s"(a.target), "s"(a.B), "s"(a.K), "s"(a.V), "s"(a.tokens), "s"(a.draft_len), "s"(a.nseg),
                 "s"(a.nchunks), "s"(a.row_bytes), "s"(a.first), "s"(a.stats));
    asm volatile("" ::"s"(a.accepted_len), "s"(a.out_tokens), "s"(a.reject_mask));
}

template <typename Fmt, int CPT>
__global__ __launch_bounds__(kW) void verify_greedy_stats(SegArgs a) {
    constexpr int EPC = Fmt::kPerChunk;
    __shared__ float s_k[kNW];
    __shared__ int s_i[kNW];

    request_args(a);
    const int tid = threadIdx.x;
    const int64_t unit = a.first + blockIdx.x;
    const int s = int(unit % a.nseg);
    const int64_t pair = unit / a.nseg;  // b*(K+1) + i
    const int b = int(pair / (a.K + 1));
    const int i = int(pair - int64_t(b) * (a.K + 1));
    const int kb = seq_k(a, b);
    if (kb < 1 || kb > a.K || i > kb) return;  // invalid k_b (reported later) or a padding row

    const char* trow = static_cast<const char*>(a.target) + pair * int64_t(a.V) * Fmt::kBytes;
    chunk_t xt[CPT];
    load_segment<CPT>(xt, trow, a, s);
    pad_segment<Fmt, CPT>(xt, a, s);
    const int c0 = s * kW * CPT + tid;  // this thread's first chunk in the row
    // Within a thread indices grow with (n, e): a strict ">" keeps the first
    // maximum.
    float best = kNegInf;
    int bi = 0x7FFFFFFF;
#pragma unroll
    for (int n = 0; n < CPT; ++n)
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
            const float v = Fmt::get(xt[n], e);
            if (v > best) {
                best = v;
                bi = (c0 + n * kW) * EPC + e;
            }
        }
    const int lane = tid & (kWave - 1), wid = tid / kWave;
    wave_argmax_u(best, bi);
    if (lane == 0) {
        s_k[wid] = best;
        s_i[wid] = bi;
    }
    __syncthreads();
    if (tid == 0) {
        float bv = s_k[0];
        int bx = s_i[0];
        for (int w = 1; w < kNW; ++w)
            if (s_k[w] > bv || (s_k[w] == bv && s_i[w] < bx)) {
                bv = s_k[w];
                bx = s_i[w];
            }
        SegStats r;
        r.st = 0.0;
        r.sd = 0.0;
        r.kt = bv;
        r.kd = __int_as_float(bx);
        a.stats[pair * kMaxSeg + s] = r;
    }
}


// Outputs of sequence b, written by wave 0 (lane j handles position j; K < 64).
__device__ inline void write_outputs(const SegArgs& a, int b, int kb, int acc, bool bad, int extra) {
    const int lane = threadIdx.x & (kWave - 1);
    const int K = a.K;
    if (lane <= K) {
        int32_t o = -1;
        if (!bad) o = lane < acc ? a.tokens[int64_t(b) * K + lane] : (lane == acc ? extra : -1);
        a.out_tokens[int64_t(b) * (K + 1) + lane] = o;
        if (a.reject_mask && lane < K)
            a.reject_mask[int64_t(b) * K + lane] = (!bad && lane == acc && acc < kb) ? 1 : 0;
    }
    if (lane == 0) a.accepted_len[b] = bad ? -1 : acc;
}

// Zero the argmax partials of sequence b (lane i: row i), once nothing reads
// them any more.
__device__ inline void clear_stats(const SegArgs& a, int b, int kb) {
    const int i = threadIdx.x & (kWave - 1);
    if (kb < 1 || kb > a.K || i > kb) return;
    const int64_t pi = int64_t(b) * (a.K + 1) + i;
    SegStats z;
    z.st = 0.0;
    z.sd = 0.0;
    z.kt = 0.0f;
    z.kd = 0.0f;
    for (int s = 0; s < a.nseg; ++s) a.stats[pi * kMaxSeg + s] = z;
}

// Greedy decision: merge the argmax partials of rows 0..k_b (lowest index on
// ties), accept while y_i equals the argmax, emit the argmax where the test
// stops.
template <typename Fmt>
__global__ __launch_bounds__(kW) void verify_greedy_decide(SegArgs a) {
    __shared__ SegStats s_st[(OSD_MAX_K + 1) * kMaxSeg];
    request_args(a);
    const int tid = threadIdx.x;
    const int b = int(a.first + blockIdx.x);
    const int K = a.K;
    const int kb = seq_k(a, b);
    {
        const SegStats* st = a.stats + int64_t(b) * (K + 1) * kMaxSeg;
        for (int j = tid; j < (K + 1) * kMaxSeg; j += kW)
            if ((j % kMaxSeg) < a.nseg) s_st[j] = st[j];
    }
    __syncthreads();
    if (tid >= kWave) return;
    const int lane = tid;
    const bool kb_ok = kb >= 1 && kb <= K;
    const int i = lane;
    float best = kNegInf;
    int g = 0x7FFFFFFF;
    if (kb_ok && i <= kb) {
        const SegStats* st = s_st + i * kMaxSeg;
        for (int s = 0; s < a.nseg; ++s) {
            const float v = st[s].kt;
            const int x = __float_as_int(st[s].kd);
            if (v > best) {  // segments hold increasing indices
                best = v;
                g = x;
            }
        }
    }
    clear_stats(a, b, kb);  // this workgroup is the only reader
    const bool bad_row = !(best > kNegInf) || best == -kNegInf;
    int y = 0;
    if (kb_ok && i < kb) y = a.tokens[int64_t(b) * K + i];
    const uint64_t tok_bad = __ballot(kb_ok && i < kb && (y < 0 || y >= a.V));
    const uint64_t stop = __ballot(kb_ok && i < kb && (bad_row || y != g));
    const int acc = stop ? __builtin_ctzll(stop) : (kb_ok ? kb : 0);
    const uint64_t row_bad = __ballot(kb_ok && i <= kb && bad_row);
    const bool bad = !kb_ok || tok_bad != 0 || ((row_bad >> acc) & 1ull) != 0;
    const int extra = __shfl(g, acc, kWave);
    write_outputs(a, b, kb, acc, bad, extra);
}

template <typename Fmt>
hipError_t launch_fmt(const VerifyLaunch& L, SegArgs a) {
    if (!greedy_segments(L.V, Fmt::kPerChunk, &a.nseg)) return hipErrorInvalidValue;
    const int64_t units = int64_t(a.B) * (a.K + 1) * a.nseg;
    for (int64_t f = 0; f < units; f += kMaxGrid) {
        a.first = f;
        const unsigned g = unsigned(units - f < kMaxGrid ? units - f : kMaxGrid);
        const hipError_t e = launch_kernel(&verify_greedy_stats<Fmt, 4>, dim3(g), dim3(kW), 0, L.stream, a);
        if (e != hipSuccess) return e;
    }
    for (int64_t f = 0; f < a.B; f += kMaxGrid) {
        a.first = f;
        const unsigned g = unsigned(a.B - f < kMaxGrid ? a.B - f : kMaxGrid);
        const hipError_t e = launch_kernel(&verify_greedy_decide<Fmt>, dim3(g), dim3(kW), 0, L.stream, a);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

// Segments of a row for greedy verification: kW threads x 4 chunks each
// (8192 bf16 or 4096 fp32 logits), at most kMaxSeg of them.
bool greedy_segments(int V, int per_chunk, int* nseg) {
    const int64_t nchunks = (int64_t(V) + per_chunk - 1) / per_chunk;
    const int64_t n = (nchunks + int64_t(kW) * 4 - 1) / (int64_t(kW) * 4);
    if (n > kMaxSeg) return false;
    *nseg = int(n);
    return true;
}

hipError_t launch_verify_greedy(const VerifyLaunch& L) {
    SegArgs a{};
    a.target = L.target;
    a.B = L.B;
    a.K = L.K;
    a.V = L.V;
    a.tokens = L.tokens;
    a.draft_len = L.draft_len;
    const int eb = L.dtype == 1 ? 2 : 4;
    a.nchunks = int((int64_t(L.V) * eb) / 16);
    a.row_bytes = uint32_t(int64_t(L.V) * eb);
    a.first = 0;
    a.stats = L.seg_stats;
    a.accepted_len = L.accepted_len;
    a.out_tokens = L.out_tokens;
    a.reject_mask = L.reject_mask;
    return L.dtype == 1 ? launch_fmt<BF16>(L, a) : launch_fmt<F32>(L, a);
}

}  // namespace osd
