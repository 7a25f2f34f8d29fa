// verify_seg.hip -- speculative-sampling verification on gfx950, segmented
// form.
//
// Method (Appendix A.1 and Eq. 5 of arXiv:2310.07177; the verification step
// of Algorithm 1): proposals y_1..y_k are tested in order, y_i is accepted
// when u_i < p(y_i)/q(y_i), the first rejection at position a ends the test,
// and one extra token is drawn from norm(max(0, p - q)) at row a, or from p at
// the bonus row when all k were accepted.  p and q are temperature softmaxes
// of the target and draft logits.
//
// Work layout: two kernels, each a flat grid of small workgroups, so the
// hardware dispatcher balances the work over every CU whatever B and k are.
//
//  1. verify_seg_stats -- one workgroup per (row pair, vocabulary segment).
//     It reads its segment of target row i and draft row i once (coalesced
//     16-byte loads), and posts the segment's softmax statistics (K, S) for
//     both rows: K a whole number at least ceil(max x log2(e)/T), S the sum
//     of 2^(x log2(e)/T - K) in fp64.  The workgroup whose segment holds the
//     proposal y_i also posts t_i[y_i] and d_i[y_i].  This kernel moves every
//     byte the method has to read.
//
//  2. verify_seg_draw -- one workgroup per (sequence, segment).  Every
//     workgroup of a sequence merges the segment statistics of the
//     sequence's rows in a fixed order, takes the acceptance tests of
//     positions 0..k_b-1 and finds the first rejection a (all of them reach
//     the same decision from the same numbers).  Each then computes the
//     masses of its own segment of row pair a -- max(0, p - q), or p for the
//     bonus row -- as fixed-point integers, posts the segment's total, and
//     the last of the sequence's workgroups to arrive finds the segment that
//     holds u * Z, walks it and writes the outputs.  The segment of row pair
//     0 (the most frequent first rejection) is loaded before the decision is
//     known; any other row pair is loaded after it.
//
// Greedy verification (T = 0) uses the same two steps with argmax partials
// (target rows only) and no draw.
#include "osd.h"
#include "osd_device.hpp"
#include "osd_internal.hpp"
#include "stream_device.hpp"

namespace osd {
namespace {

constexpr int kW = 256;          // threads per workgroup
constexpr int kNW = kW / kWave;  // waves per workgroup
// Residual and bonus masses are probabilities (at most 1 per element, about 1
// per row); chunk sums are converted exactly to 2^-40 fixed point, so every
// partial sum of the CDF is an exact integer and the totals do not depend on
// the reduction order.
constexpr int kFixedShift = 40;
// Workgroups per launch (grid sizes stay far below the 2^32 work-item limit).
constexpr int64_t kMaxGrid = int64_t(1) << 22;

struct SegArgs {
    const void* target;  // [B, K+1, V]
    const void* draft;   // [B, K, V] (unused when greedy)
    int B, K, V;
    const int32_t* tokens;     // [B, K]
    const int32_t* draft_len;  // [B] or null
    const float* u_accept;     // [B, K]
    const float* u_resample;   // [B]
    float c2;                  // log2(e) / T
    double c2d;                // the same value in fp64
    int nseg;                  // segments per row
    int nchunks;               // 16-byte chunks per row
    uint32_t row_bytes;
    int64_t first;             // first work unit of this launch
    SegStats* stats;           // [B*(K+1), kMaxSeg]
    float* yv;                 // [B*(K+1), 2]: t_i[y_i], d_i[y_i]
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

// ---------------------------------------------------------------------------
// Kernel 1: segment statistics
// ---------------------------------------------------------------------------
template <typename Fmt, int CPT, bool GREEDY>
__global__ __launch_bounds__(kW) void verify_seg_stats(SegArgs a) {
    constexpr int EPC = Fmt::kPerChunk;
    __shared__ float s_k[2 * kNW];
    __shared__ double s_s[2 * kNW];
    __shared__ int s_i[kNW];

    const int tid = threadIdx.x;
    const int64_t unit = a.first + blockIdx.x;
    const int s = int(unit % a.nseg);
    const int64_t pair = unit / a.nseg;  // b*(K+1) + i
    const int b = int(pair / (a.K + 1));
    const int i = int(pair - int64_t(b) * (a.K + 1));
    // (Without a length array every row below K+1 is live, and the loads
    // below do not wait for a length.)
    const int kb = seq_k(a, b);
    if (kb < 1 || kb > a.K || i > kb) return;  // invalid k_b (reported later) or a padding row
    const bool bonus = i == kb;

    const char* trow = static_cast<const char*>(a.target) + pair * int64_t(a.V) * Fmt::kBytes;
    const char* drow = (GREEDY || bonus) ? nullptr
                                         : static_cast<const char*>(a.draft) +
                                               (int64_t(b) * a.K + i) * int64_t(a.V) * Fmt::kBytes;
    chunk_t xt[CPT], xd[CPT];
    load_segment<CPT>(xt, trow, a, s);
    if (!GREEDY) load_segment<CPT>(xd, drow, a, s);
    pad_segment<Fmt, CPT>(xt, a, s);
    if (!GREEDY) pad_segment<Fmt, CPT>(xd, a, s);
    const int c0 = s * kW * CPT + tid;  // this thread's first chunk in the row

    if constexpr (GREEDY) {
        // Within a thread indices grow with (n, e): a strict ">" keeps the
        // first maximum.
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
        return;
    } else {
        // The proposal's logits, posted by the thread that holds them.
        if (!bonus) {
            const int y = scalar_load(a.tokens + int64_t(b) * a.K + i);
            const int yc = y / EPC - c0;  // chunk offset from this thread's first chunk
            if (y >= 0 && y < a.V && yc >= 0 && yc < kW * CPT && yc % kW == 0) {
#pragma unroll
                for (int n = 0; n < CPT; ++n)
                    if (yc == n * kW) {
                        a.yv[2 * pair] = Fmt::get(xt[n], y % EPC);
                        a.yv[2 * pair + 1] = Fmt::get(xd[n], y % EPC);
                    }
            }
        }
        // Thread maxima first (all chunks are resident), then every
        // exponential is at most 1 and the thread sums cannot overflow.
        float mt = kNegInf, md = kNegInf;
#pragma unroll
        for (int n = 0; n < CPT; ++n) {
            mt = fmaxf(mt, chunk_max<Fmt>(xt[n]));
            md = fmaxf(md, chunk_max<Fmt>(xd[n]));
        }
        // A thread that saw only -inf: a finite stand-in for its shift keeps
        // 2^(x c2 - k) at 0 instead of NaN.
        float kt = fmaxf(ceilf(mt * a.c2), -3.0e38f);
        float kd = fmaxf(ceilf(md * a.c2), -3.0e38f);
        float st = 0.0f, sd = 0.0f;
#pragma unroll
        for (int n = 0; n < CPT; ++n)
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                st = st + exp2_fast(__builtin_fmaf(Fmt::get(xt[n], e), a.c2, -kt));
                if (!bonus) sd = sd + exp2_fast(__builtin_fmaf(Fmt::get(xd[n], e), a.c2, -kd));
            }
        double St = st, Sd = sd;
        block_merge2<kNW>(kt, St, kd, Sd, s_k, s_s);
        if (tid == 0) {
            SegStats r;
            r.st = St;
            r.sd = Sd;
            r.kt = kt;
            r.kd = kd;
            a.stats[pair * kMaxSeg + s] = r;
        }
    }
}

// ---------------------------------------------------------------------------
// Kernel 2: decision, draw and outputs
// ---------------------------------------------------------------------------

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

// Merge the segment statistics of one row in segment order (fp64, exact
// power-of-two shifts), so every workgroup gets the same numbers.
__device__ inline void merge_row(const SegStats* st, int nseg, bool draft, float& K, double& S) {
    float k = -3.0e38f;
    for (int s = 0; s < nseg; ++s) k = fmaxf(k, draft ? st[s].kd : st[s].kt);
    double acc = 0.0;
    for (int s = 0; s < nseg; ++s) acc += rescale(draft ? st[s].sd : st[s].st, draft ? st[s].kd : st[s].kt, k);
    K = k;
    S = acc;
}

// Element masses of row pair a in fp32: p = 2^(t c2 - K_t) / S_t, and for
// the residual max(0, p - 2^(d c2 - K_d) / S_d).  The pass that sums the
// masses and the walk that picks the token evaluate exactly this code on the
// same numbers.
template <typename Fmt>
struct Masses {
    float c2, kt, kd, at, ad;
    __device__ inline float p(const chunk_t& t, int e) const {
        return exp2_fast(__builtin_fmaf(Fmt::get(t, e), c2, -kt)) * at;
    }
    __device__ inline float get(const chunk_t& t, const chunk_t& d, int e, bool residual) const {
        const float pv = p(t, e);
        if (!residual) return pv;
        return fmaxf(pv - exp2_fast(__builtin_fmaf(Fmt::get(d, e), c2, -kd)) * ad, 0.0f);
    }
    // Sum of a chunk's masses, left to right in fp32, exactly in 2^-40 units.
    __device__ inline uint64_t chunk(const chunk_t& t, const chunk_t& d, bool residual) const {
        float sm = 0.0f;
#pragma unroll
        for (int e = 0; e < Fmt::kPerChunk; ++e) sm = sm + get(t, d, e, residual);
        return to_fixed<kFixedShift>(sm);
    }
};

// Zero the segment statistics and proposal logits of sequence b (lane i:
// row i), once nothing reads them any more.
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
    a.yv[2 * pi] = 0.0f;
    a.yv[2 * pi + 1] = 0.0f;
}

struct Decision {
    int acc;
    int bad;
    float kt, kd;
    double st, sd;
};

// The draw workgroup: kDW threads, thread tid owns chunks n*kDW + tid
// (n < NCH) of row pair a; they are processed kGroup at a time.
constexpr int kDW = 1024;
constexpr int kDNW = kDW / kWave;
constexpr int kGroup = 4;

template <typename Fmt, int GC>
__device__ inline void load_group(chunk_t (&xt)[GC], chunk_t (&xd)[GC], rsrc_t tr, rsrc_t dr, int g,
                                  int nchunks) {
#pragma unroll
    for (int n = 0; n < GC; ++n) {
        xt[n] = load_chunk<kDW>(tr, g * GC + n);
        xd[n] = load_chunk<kDW>(dr, g * GC + n);
    }
#pragma unroll
    for (int n = 0; n < GC; ++n)
        if ((g * GC + n) * kDW + int(threadIdx.x) >= nchunks) {
            xt[n] = pad_chunk<Fmt>();
            xd[n] = pad_chunk<Fmt>();
        }
}

// One workgroup per sequence: decision, then the draw over row pair a.
//  - the segment statistics of rows 0..K are staged in LDS by all threads;
//    wave 0 merges them (fixed order), takes the acceptance tests and finds
//    the first rejection a;
//  - the chunk masses of row pair a are summed per thread as exact
//    fixed-point cells; cells are ordered (round n, wave, lane), which is
//    token order; one scan of the per-(round, wave) totals gives every cell
//    its prefix, and the thread whose cell holds u*Z walks its elements.
// The first group of row pair 0 (the most frequent first rejection) is
// loaded before the decision is known.
template <typename Fmt, int NCH>
__global__ __launch_bounds__(kDW) void verify_seg_draw(SegArgs a) {
    constexpr int EPC = Fmt::kPerChunk;
    constexpr int GC = NCH < kGroup ? NCH : kGroup;  // chunks per group
    constexpr int NG = NCH / GC;                      // groups
    constexpr int CELLS = NCH * kDNW;                 // (round, wave) cells
    __shared__ SegStats s_st[(OSD_MAX_K + 1) * kMaxSeg];
    __shared__ Decision s_dec;
    __shared__ unsigned long long s_cell[CELLS];
    __shared__ unsigned long long s_w[kDNW];
    __shared__ int s_tok;

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int b = int(a.first + blockIdx.x);
    const int K = a.K;
    const int kb = seq_k(a, b);
    const int64_t row_elems = int64_t(a.V) * Fmt::kBytes;
    const char* t0 = static_cast<const char*>(a.target) + int64_t(b) * (K + 1) * row_elems;
    const char* d0 = static_cast<const char*>(a.draft) + int64_t(b) * K * row_elems;

    chunk_t xt[GC], xd[GC];
    load_group<Fmt, GC>(xt, xd, make_rsrc(t0, a.row_bytes), make_rsrc(d0, a.row_bytes), 0, a.nchunks);
    {
        const SegStats* st = a.stats + int64_t(b) * (K + 1) * kMaxSeg;
        for (int j = tid; j < (K + 1) * kMaxSeg; j += kDW)
            if ((j % kMaxSeg) < a.nseg) s_st[j] = st[j];
    }
    __syncthreads();

    // ---- decision (wave 0; lane i = position i) ----
    if (wid == 0) {
        const bool kb_ok = kb >= 1 && kb <= K;
        const int i = lane;
        float kt = -3.0e38f, kd = -3.0e38f;
        double St = 0.0, Sd = 0.0;
        bool accept = false, bad_tok = false, bad_row = false;
        if (kb_ok && i <= kb) {
            const SegStats* st = s_st + i * kMaxSeg;
            merge_row(st, a.nseg, false, kt, St);
            bad_row = !(St > 0.0 && St < 1.0e300);
            if (i < kb) {
                merge_row(st, a.nseg, true, kd, Sd);
                bad_row = bad_row || !(Sd > 0.0 && Sd < 1.0e300);
                const int y = a.tokens[int64_t(b) * K + i];
                bad_tok = y < 0 || y >= a.V;
                if (!bad_tok && !bad_row) {
                    // p(y)/q(y) = 2^e * S_d / S_t, e = (t_y c2 - K_t) - (d_y c2 - K_d)
                    // in fp64; 2^e is split into an exact power of two and
                    // 2^frac (v_exp_f32).
                    const int64_t pi = int64_t(b) * (K + 1) + i;
                    const double e = (double(a.yv[2 * pi]) * a.c2d - double(kt)) -
                                     (double(a.yv[2 * pi + 1]) * a.c2d - double(kd));
                    double ratio;
                    if (!(e > -2000.0)) {
                        ratio = 0.0;  // p(y) = 0
                    } else if (e > 2000.0) {
                        ratio = __builtin_huge_val();
                    } else {
                        const double fl = floor(e);
                        ratio = __builtin_ldexp(double(exp2_fast(float(e - fl))), int(fl)) * (Sd / St);
                    }
                    accept = double(a.u_accept[int64_t(b) * K + i]) < ratio;
                }
            }
        }
        // A proposal outside the vocabulary invalidates the sequence wherever
        // it sits; a row without finite logits only if the test reaches it.
        const uint64_t tok_bad = __ballot(kb_ok && i < kb && bad_tok);
        const uint64_t stop = __ballot(kb_ok && i < kb && !accept);
        const int acc = stop ? __builtin_ctzll(stop) : (kb_ok ? kb : 0);
        const uint64_t row_bad = __ballot(kb_ok && i <= kb && bad_row);
        const bool bad = !kb_ok || tok_bad != 0 || ((row_bad >> acc) & 1ull) != 0;
        if (lane == acc) {
            s_dec.acc = acc;
            s_dec.bad = bad ? 1 : 0;
            s_dec.kt = kt;
            s_dec.kd = kd;
            s_dec.st = St;
            s_dec.sd = Sd;
        }
        clear_stats(a, b, kb);  // LDS holds what is still needed
    }
    __syncthreads();
    const Decision dec = s_dec;
    const int acc = __builtin_amdgcn_readfirstlane(dec.acc);
    if (dec.bad) {
        if (wid == 0) write_outputs(a, b, kb, acc, true, -1);
        return;
    }
    const bool bonus = acc == kb;
    const rsrc_t tr = make_rsrc(t0 + int64_t(acc) * row_elems, a.row_bytes);
    const rsrc_t dr = make_rsrc(bonus ? t0 : d0 + int64_t(acc) * row_elems, bonus ? 0u : a.row_bytes);
    if (acc != 0) load_group<Fmt, GC>(xt, xd, tr, dr, 0, a.nchunks);

    Masses<Fmt> m;
    m.c2 = a.c2;
    m.kt = dec.kt;
    m.kd = dec.kd;
    m.at = float(1.0 / dec.st);
    m.ad = bonus ? 0.0f : float(1.0 / dec.sd);

    // Cell masses of the whole row pair; the workgroup total.  A residual
    // with no mass left after rounding (p = q to fp32 accuracy) is drawn from
    // p instead.
    uint64_t f[NCH];
    bool residual = !bonus;
    uint64_t Z = 0;
    for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
        for (int g = 0; g < NG; ++g) {
            if (g > 0 || pass > 0) {
                if (NG > 1) load_group<Fmt, GC>(xt, xd, tr, dr, g, a.nchunks);
            }
#pragma unroll
            for (int n = 0; n < GC; ++n) f[g * GC + n] = m.chunk(xt[n], xd[n], residual);
        }
        uint64_t t = 0;
#pragma unroll
        for (int n = 0; n < NCH; ++n) t += f[n];
        t = readlane_u64(wave_scan_add(t), kWave - 1);
        if (lane == 0) s_w[wid] = t;
        __syncthreads();
        Z = 0;
#pragma unroll
        for (int w = 0; w < kDNW; ++w) Z += s_w[w];
        __syncthreads();  // s_w is rewritten by a second pass
        if (Z > 0 || !residual) break;
        residual = false;
    }
    if (Z == 0) {  // no mass at all (cannot happen for a row with a finite logit)
        if (wid == 0) write_outputs(a, b, kb, acc, true, -1);
        return;
    }
    uint64_t target = static_cast<uint64_t>(double(a.u_resample[b]) * double(Z));
    if (target >= Z) target = Z - 1;

    // ---- prefixes of the (round, wave) cells, in token order ----
#pragma unroll
    for (int n = 0; n < NCH; ++n) {
        const uint64_t incl = wave_scan_add(f[n]);
        if (lane == kWave - 1) s_cell[n * kDNW + wid] = incl;
    }
    if (tid == 0) s_tok = -1;
    __syncthreads();
    if (wid == 0) {  // exclusive scan in place, 64 cells at a time
        uint64_t carry = 0;
        for (int q = 0; q < CELLS; q += kWave) {
            const uint64_t v = q + lane < CELLS ? uint64_t(s_cell[q + lane]) : 0;
            const uint64_t incl = wave_scan_add(v);
            if (q + lane < CELLS) s_cell[q + lane] = carry + incl - v;
            carry += readlane_u64(incl, kWave - 1);
        }
    }
    __syncthreads();
#pragma unroll
    for (int n = 0; n < NCH; ++n) {
        const uint64_t incl = wave_scan_add(f[n]);
        const uint64_t lo = uint64_t(s_cell[n * kDNW + wid]) + incl - f[n];
        if (f[n] > 0 && lo <= target && target < lo + f[n]) {
            chunk_t ct, cd;
            if constexpr (NG == 1) {
                ct = xt[n % GC];
                cd = xd[n % GC];
            } else {  // reload this one chunk pair
                ct = load_chunk<kDW>(tr, n);
                cd = load_chunk<kDW>(dr, n);
                if (n * kDW + tid >= a.nchunks) {
                    ct = pad_chunk<Fmt>();
                    cd = pad_chunk<Fmt>();
                }
            }
            const uint64_t want = target - lo;
            float racc = 0.0f;
            int pick = -1, last_pos = -1;
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float v = m.get(ct, cd, e, residual);
                racc = racc + v;
                if (v > 0.0f) last_pos = e;
                if (pick < 0 && to_fixed<kFixedShift>(racc) > want) pick = e;
            }
            if (pick < 0) pick = last_pos >= 0 ? last_pos : 0;
            s_tok = (n * kDW + tid) * EPC + pick;
        }
    }
    __syncthreads();
    if (wid == 0) {
        const int tok = s_tok;
        write_outputs(a, b, kb, acc, tok < 0 || tok >= a.V, tok);
    }
}

// Greedy decision: merge the argmax partials of rows 0..k_b (lowest index on
// ties), accept while y_i equals the argmax, emit the argmax where the test
// stops.
template <typename Fmt>
__global__ __launch_bounds__(kW) void verify_seg_greedy(SegArgs a) {
    __shared__ SegStats s_st[(OSD_MAX_K + 1) * kMaxSeg];
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

template <typename Fmt, int CPT, int NCH>
hipError_t launch_tiles(const VerifyLaunch& L, SegArgs a) {
    const bool greedy = L.temperature == 0.0f;
    const int64_t units = int64_t(a.B) * (a.K + 1) * a.nseg;
    for (int64_t f = 0; f < units; f += kMaxGrid) {
        a.first = f;
        const unsigned g = unsigned(units - f < kMaxGrid ? units - f : kMaxGrid);
        if (greedy)
            hipLaunchKernelGGL((verify_seg_stats<Fmt, CPT, true>), dim3(g), dim3(kW), 0, L.stream, a);
        else
            hipLaunchKernelGGL((verify_seg_stats<Fmt, CPT, false>), dim3(g), dim3(kW), 0, L.stream, a);
    }
    for (int64_t f = 0; f < a.B; f += kMaxGrid) {
        a.first = f;
        const unsigned g = unsigned(a.B - f < kMaxGrid ? a.B - f : kMaxGrid);
        if (greedy)
            hipLaunchKernelGGL((verify_seg_greedy<Fmt>), dim3(g), dim3(kW), 0, L.stream, a);
        else
            hipLaunchKernelGGL((verify_seg_draw<Fmt, NCH>), dim3(g), dim3(kDW), 0, L.stream, a);
    }
    return hipGetLastError();
}

template <typename Fmt>
hipError_t launch_fmt(const VerifyLaunch& L, SegArgs a) {
    int cpt = 0;
    if (!pick_seg_cpt(L.V, Fmt::kPerChunk, &cpt, &a.nseg) || cpt != 4) return hipErrorInvalidValue;
    // Chunks per thread of the draw workgroup.
    const int need = (a.nchunks + kDW - 1) / kDW;
    if (need <= 1) return launch_tiles<Fmt, 4, 1>(L, a);
    if (need <= 2) return launch_tiles<Fmt, 4, 2>(L, a);
    if (need <= 4) return launch_tiles<Fmt, 4, 4>(L, a);
    if (need <= 8) return launch_tiles<Fmt, 4, 8>(L, a);
    if (need <= 16) return launch_tiles<Fmt, 4, 16>(L, a);
    return hipErrorInvalidValue;
}

}  // namespace

// Chunks per thread of a segment: 4 (32 bf16 or 16 fp32 logits per row per
// thread), enough work to amortise the workgroup's merge of its statistics.
// Segments per row: as many as V needs, at most kMaxSeg.
bool pick_seg_cpt(int V, int per_chunk, int* cpt, int* nseg) {
    constexpr int kCpt = 4;
    const int64_t nchunks = (int64_t(V) + per_chunk - 1) / per_chunk;
    const int64_t n = (nchunks + int64_t(kW) * kCpt - 1) / (int64_t(kW) * kCpt);
    if (n > kMaxSeg) return false;
    *cpt = kCpt;
    *nseg = int(n);
    return true;
}

hipError_t launch_verify_seg(const VerifyLaunch& L) {
    SegArgs a;
    a.target = L.target;
    a.draft = L.draft ? L.draft : L.target;
    a.B = L.B;
    a.K = L.K;
    a.V = L.V;
    a.tokens = L.tokens;
    a.draft_len = L.draft_len;
    a.u_accept = L.u_accept;
    a.u_resample = L.u_resample;
    a.c2 = L.temperature > 0.0f ? float(1.4426950408889634 / double(L.temperature)) : 0.0f;
    a.c2d = double(a.c2);
    const int eb = L.dtype == 1 ? 2 : 4;
    a.nchunks = int((int64_t(L.V) * eb) / 16);
    a.row_bytes = uint32_t(int64_t(L.V) * eb);
    a.first = 0;
    a.stats = L.seg_stats;
    a.yv = L.seg_y;
    a.accepted_len = L.accepted_len;
    a.out_tokens = L.out_tokens;
    a.reject_mask = L.reject_mask;
    return L.dtype == 1 ? launch_fmt<BF16>(L, a) : launch_fmt<F32>(L, a);
}

}  // namespace osd
