// osd_device.hpp -- device-side building blocks shared by the verification and
// distillation kernels (gfx950, wave64).
//
// Rows are read as 16-byte chunks (8 bf16 or 4 fp32 logits).  A workgroup of W
// threads holds a row in registers as CPT chunks per thread: chunk n*W + tid
// for round n, so each round is one fully coalesced sweep over W*16 bytes and
// token ids grow with (round, thread, element).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace osd {

constexpr int kWave = 64;

// One 16-byte chunk of a row (a native vector so that loads stay dwordx4).
typedef uint32_t chunk_t __attribute__((ext_vector_type(4)));
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLog2e = 1.4426950408889634f;
constexpr double kLn2 = 0.69314718055994530942;

// ---------------------------------------------------------------------------
// Exponentials.  v_exp_f32 computes 2^x; scaled logits are formed as
// (x - max) * log2(e)/T so that the term carrying the mass is exact-ish.
// ---------------------------------------------------------------------------
__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ inline float log2_fast(float x) { return __builtin_amdgcn_logf(x); }

// ---------------------------------------------------------------------------
// Logit formats
// ---------------------------------------------------------------------------
struct BF16 {
    static constexpr int kPerChunk = 8;
    static constexpr int kBytes = 2;
    // One padding element: -inf has zero probability and never wins a max.
    static constexpr uint16_t kPad = 0xFF80u;
    __device__ static inline float get(const chunk_t& c, int e) {
        const uint32_t w = (e >> 1) == 0 ? c.x : (e >> 1) == 1 ? c.y : (e >> 1) == 2 ? c.z : c.w;
        return (e & 1) ? __uint_as_float(w & 0xFFFF0000u) : __uint_as_float(w << 16);
    }
    __device__ static inline float load_one(const void* row, int j) {
        return __uint_as_float(uint32_t(static_cast<const uint16_t*>(row)[j]) << 16);
    }
    // The bits of element j, and their value (a load kept apart from its use).
    __device__ static inline uint32_t load_raw(const void* row, int j) { return static_cast<const uint16_t*>(row)[j]; }
    __device__ static inline float from_raw(uint32_t r) { return __uint_as_float(r << 16); }
    __device__ static inline chunk_t load_scalar(const void* row, int64_t first, int V) {
        const uint16_t* p = static_cast<const uint16_t*>(row);
        uint16_t v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (first + e < V) ? p[first + e] : kPad;
        chunk_t c;
        c.x = v[0] | (uint32_t(v[1]) << 16);
        c.y = v[2] | (uint32_t(v[3]) << 16);
        c.z = v[4] | (uint32_t(v[5]) << 16);
        c.w = v[6] | (uint32_t(v[7]) << 16);
        return c;
    }
};

struct F32 {
    static constexpr int kPerChunk = 4;
    static constexpr int kBytes = 4;
    __device__ static inline float get(const chunk_t& c, int e) {
        const uint32_t w = e == 0 ? c.x : e == 1 ? c.y : e == 2 ? c.z : c.w;
        return __uint_as_float(w);
    }
    __device__ static inline float load_one(const void* row, int j) {
        return static_cast<const float*>(row)[j];
    }
    __device__ static inline uint32_t load_raw(const void* row, int j) { return static_cast<const uint32_t*>(row)[j]; }
    __device__ static inline float from_raw(uint32_t r) { return __uint_as_float(r); }
    __device__ static inline chunk_t load_scalar(const void* row, int64_t first, int V) {
        const float* p = static_cast<const float*>(row);
        uint32_t v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[e] = (first + e < V) ? __float_as_uint(p[first + e]) : 0xFF800000u;
        return chunk_t{v[0], v[1], v[2], v[3]};
    }
};

// Whole chunk of padding (past the end of the row).
template <typename Fmt>
__device__ inline chunk_t pad_chunk() {
    if constexpr (Fmt::kPerChunk == 8)
        return chunk_t{0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u};
    else
        return chunk_t{0xFF800000u, 0xFF800000u, 0xFF800000u, 0xFF800000u};
}

// Load the CPT chunks of one row owned by this thread.  VEC: the row is
// 16-byte aligned and V is a multiple of the chunk size.
// VEC loads are issued without branches (a chunk past the row reloads the
// row's last chunk and is replaced by padding): with every load in one basic
// block the compiler waits for exactly the chunk a sweep consumes next, so
// the statistics fold in as the loads land instead of after the last one.
template <typename Fmt, int W, int CPT, bool VEC>
__device__ inline void load_row(chunk_t (&c)[CPT], const void* row, int V) {
    const int nchunks = (V + Fmt::kPerChunk - 1) / Fmt::kPerChunk;
#pragma unroll
    for (int n = 0; n < CPT; ++n) {
        const int ch = n * W + static_cast<int>(threadIdx.x);
        if constexpr (VEC) {
            const bool in = ch < nchunks;
            const chunk_t v = __builtin_nontemporal_load(static_cast<const chunk_t*>(row) + (in ? ch : nchunks - 1));
            const chunk_t pad = pad_chunk<Fmt>();
            c[n] = chunk_t{in ? v.x : pad.x, in ? v.y : pad.y, in ? v.z : pad.z, in ? v.w : pad.w};
        } else {
            c[n] = ch < nchunks ? Fmt::load_scalar(row, int64_t(ch) * Fmt::kPerChunk, V) : pad_chunk<Fmt>();
        }
    }
}

// The loads of load_row<VEC> without the padding: a chunk past the row
// re-reads the row's last chunk and stays as loaded.  Consumers apply the
// padding where they use a chunk (row_stats_tail, pad_row_tail), so no
// instruction right after the loads needs their data and each sweep waits
// only for the chunk it takes next.
template <int W, int CPT>
__device__ inline void load_row_clamped(chunk_t (&c)[CPT], const void* row, int nchunks) {
#pragma unroll
    for (int n = 0; n < CPT; ++n) {
        const int ch = n * W + static_cast<int>(threadIdx.x);
        c[n] = __builtin_nontemporal_load(static_cast<const chunk_t*>(row) + (ch < nchunks ? ch : nchunks - 1));
    }
}

// Two rows loaded as load_row_clamped loads each, chunk by chunk in turn
// (a0, b0, a1, b1, ...), the order in which row_stats2_tail takes them.
template <int W, int CPT>
__device__ inline void load_rows_interleaved(chunk_t (&a)[CPT], chunk_t (&b)[CPT], const void* ra, const void* rb,
                                             int nchunks) {
#pragma unroll
    for (int n = 0; n < CPT; ++n) {
        const int ch = n * W + static_cast<int>(threadIdx.x);
        const int cl = ch < nchunks ? ch : nchunks - 1;
        a[n] = __builtin_nontemporal_load(static_cast<const chunk_t*>(ra) + cl);
        b[n] = __builtin_nontemporal_load(static_cast<const chunk_t*>(rb) + cl);
    }
}

// Chunk n of this thread, or padding if it lies past the row.
template <typename Fmt, int W>
__device__ inline chunk_t chunk_or_pad(const chunk_t& c, int n, int nchunks) {
    const bool in = n * W + static_cast<int>(threadIdx.x) < nchunks;
    const chunk_t pad = pad_chunk<Fmt>();
    return chunk_t{in ? c.x : pad.x, in ? c.y : pad.y, in ? c.z : pad.z, in ? c.w : pad.w};
}

// Replace the chunks of load_row_clamped that lie past the row by padding.
template <typename Fmt, int W, int CPT>
__device__ inline void pad_row_tail(chunk_t (&c)[CPT], int nchunks) {
#pragma unroll
    for (int n = 0; n < CPT; ++n) c[n] = chunk_or_pad<Fmt, W>(c[n], n, nchunks);
}

// Make register-resident chunks opaque to the optimiser at the start of a
// sweep.  Unpacking a bf16 pair costs one instruction; without this the
// compiler keeps every unpacked value of an earlier sweep alive to reuse it,
// which doubles the register footprint of a row and spills.
template <int CPT>
__device__ inline void opaque(chunk_t (&c)[CPT]) {
#pragma unroll
    for (int n = 0; n < CPT; ++n) asm volatile("" : "+v"(c[n]));
}

// ---------------------------------------------------------------------------
// Wave64 reductions and scans on DPP (data-parallel primitives: operand lane
// permutations inside the vector ALU).  Lane shuffles compile to LDS permute
// round trips; these do not.  Steps: row_shr 1, 2, 4, 8 form inclusive
// prefixes inside each row of 16 lanes, then row_bcast 15 and 31 carry the row
// totals into the later rows.  Lanes whose source is outside the row (or a
// disabled row) take the identity.  The order of operations is fixed, so
// results are reproducible.  The total ends in lane 63; readlane broadcasts it.
// ---------------------------------------------------------------------------
enum : int { kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118,
             kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143 };

template <int CTRL, int ROWS>
__device__ inline uint32_t dpp(uint32_t identity, uint32_t v) {
    return uint32_t(__builtin_amdgcn_update_dpp(int(identity), int(v), CTRL, ROWS, 0xF, false));
}
__device__ inline uint32_t readlane_u32(uint32_t v, int lane) {
    return uint32_t(__builtin_amdgcn_readlane(int(v), lane));
}
__device__ inline float readlane_f32(float v, int lane) {
    return __uint_as_float(readlane_u32(__float_as_uint(v), lane));
}
__device__ inline uint64_t readlane_u64(uint64_t v, int lane) {
    return uint64_t(readlane_u32(uint32_t(v), lane)) | (uint64_t(readlane_u32(uint32_t(v >> 32), lane)) << 32);
}
__device__ inline double readlane_f64(double v, int lane) {
    return __builtin_bit_cast(double, readlane_u64(__builtin_bit_cast(uint64_t, v), lane));
}

// Floats as unsigned keys in the same order (no NaN): a float maximum over
// lanes becomes an unsigned one, which the DPP move folds into (identity 0)
// and which needs no NaN quieting of each operand.
__device__ inline uint32_t float_key(float f) {
    const uint32_t b = __float_as_uint(f);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ inline float key_float(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}
template <int CTRL, int ROWS>
__device__ inline uint32_t dpp_umax_step(uint32_t k) {
    const uint32_t o = dpp<CTRL, ROWS>(0u, k);
    return k > o ? k : o;
}
// A 32-bit lane permutation for a sum (identity 0).  Every row enabled
// (the row shifts): lanes whose source is outside the row read 0 through
// the bound control, and no register has to be preset to the identity.
template <int CTRL, int ROWS>
__device__ inline uint32_t dpp_sum_src(uint32_t v) {
    if constexpr (ROWS == 0xF)
        return uint32_t(__builtin_amdgcn_mov_dpp(int(v), CTRL, 0xF, 0xF, true));
    else
        return dpp<CTRL, ROWS>(0u, v);
}
template <int CTRL, int ROWS>
__device__ inline double dpp_add_step(double v) {
    const uint64_t b = __builtin_bit_cast(uint64_t, v);
    const uint64_t o = uint64_t(dpp_sum_src<CTRL, ROWS>(uint32_t(b))) |
                       (uint64_t(dpp_sum_src<CTRL, ROWS>(uint32_t(b >> 32))) << 32);
    return v + __builtin_bit_cast(double, o);
}
template <int CTRL, int ROWS>
__device__ inline uint64_t dpp_add_step(uint64_t v) {
    const uint64_t o = uint64_t(dpp_sum_src<CTRL, ROWS>(uint32_t(v))) |
                       (uint64_t(dpp_sum_src<CTRL, ROWS>(uint32_t(v >> 32))) << 32);
    return v + o;
}

// Inclusive scans over the wave (lane 63 holds the total).
template <typename T>
__device__ inline T wave_scan_add(T v) {
    v = dpp_add_step<kDppRowShr1, 0xF>(v);
    v = dpp_add_step<kDppRowShr2, 0xF>(v);
    v = dpp_add_step<kDppRowShr4, 0xF>(v);
    v = dpp_add_step<kDppRowShr8, 0xF>(v);
    v = dpp_add_step<kDppRowBcast15, 0xA>(v);
    v = dpp_add_step<kDppRowBcast31, 0xC>(v);
    return v;
}


// Wave totals and scans on the primitives above; every lane gets the total.
__device__ inline float wave_max(float v) {  // values without NaN
    uint32_t k = float_key(v);
    k = dpp_umax_step<kDppRowShr1, 0xF>(k);
    k = dpp_umax_step<kDppRowShr2, 0xF>(k);
    k = dpp_umax_step<kDppRowShr4, 0xF>(k);
    k = dpp_umax_step<kDppRowShr8, 0xF>(k);
    k = dpp_umax_step<kDppRowBcast15, 0xA>(k);
    k = dpp_umax_step<kDppRowBcast31, 0xC>(k);
    return key_float(readlane_u32(k, kWave - 1));
}
__device__ inline double wave_sum(double v) { return readlane_f64(wave_scan_add(v), kWave - 1); }
__device__ inline uint64_t wave_sum(uint64_t v) { return readlane_u64(wave_scan_add(v), kWave - 1); }
__device__ inline uint64_t wave_inclusive_scan(uint64_t v) { return wave_scan_add(v); }

// Max value, lowest index among equal maxima.
__device__ inline void wave_argmax(float& v, int& idx) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float ov = __shfl_xor(v, o, kWave);
        const int oi = __shfl_xor(idx, o, kWave);
        if (ov > v || (ov == v && oi < idx)) {
            v = ov;
            idx = oi;
        }
    }
}

// ---------------------------------------------------------------------------
// Streaming softmax statistics of a register-resident row.
//
// Each thread keeps S = sum_j 2^(x_j c2 - K) over its elements, where c2 =
// log2(e)/T and the shift K is a whole number at least ceil(max_j x_j c2).
// Chunks are folded in as their loads land (no barrier between the maximum
// and the sum); raising K rescales S by an exact power of two (ldexp), so
// the statistics carry no rounding from the shift.  Lanes and waves merge
// the same way.  A row without finite logits ends with K = -inf, S = 0.
// ---------------------------------------------------------------------------
template <typename Fmt>
__device__ inline float chunk_max(const chunk_t& c) {
    float m = Fmt::get(c, 0);
#pragma unroll
    for (int e = 1; e < Fmt::kPerChunk; ++e) m = fmaxf(m, Fmt::get(c, e));
    return m;
}

// 2^(from - to) * S for whole numbers from <= to (exact; -inf/NaN -> 0).
__device__ inline float rescale(float S, float from, float to) {
    return __builtin_ldexpf(S, int(fmaxf(from - to, -256.0f)));
}
__device__ inline double rescale(double S, float from, float to) {
    return __builtin_ldexp(S, int(fmaxf(from - to, -2048.0f)));
}

// fp32 accumulation, pairwise within a chunk.
template <typename Fmt, int CPT>
__device__ inline void row_stats(const chunk_t (&c)[CPT], float c2, float& K, float& S) {
    constexpr int EPC = Fmt::kPerChunk;
#pragma unroll
    for (int n = 0; n < CPT; ++n) {
        const float kn = fmaxf(K, ceilf(chunk_max<Fmt>(c[n]) * c2));
        S = rescale(S, K, kn);
        K = kn;
        // While K is still -inf every element seen is -inf: a finite stand-in
        // keeps 2^(x c2 - K) at 2^-inf = 0 instead of -inf + inf = NaN.
        const float kx = fmaxf(K, -3.0e38f);
        float e8[EPC];
#pragma unroll
        for (int e = 0; e < EPC; ++e) e8[e] = exp2_fast(__builtin_fmaf(Fmt::get(c[n], e), c2, -kx));
#pragma unroll
        for (int w = 1; w < EPC; w <<= 1)
#pragma unroll
            for (int e = 0; e < EPC; e += 2 * w) e8[e] = e8[e] + e8[e + w];
        S = S + e8[0];
        __builtin_amdgcn_sched_barrier(0);  // one chunk in flight: bounded VGPRs
    }
}

// row_stats over chunks from load_row_clamped: each chunk is padded as the
// sweep takes it (after its load has landed).
template <typename Fmt, int W, int CPT>
__device__ inline void row_stats_tail(const chunk_t (&c)[CPT], int nchunks, float c2, float& K, float& S) {
    constexpr int EPC = Fmt::kPerChunk;
#pragma unroll
    for (int n = 0; n < CPT; ++n) {
        const chunk_t x = chunk_or_pad<Fmt, W>(c[n], n, nchunks);
        const float kn = fmaxf(K, ceilf(chunk_max<Fmt>(x) * c2));
        S = rescale(S, K, kn);
        K = kn;
        const float kx = fmaxf(K, -3.0e38f);  // see row_stats
        float e8[EPC];
#pragma unroll
        for (int e = 0; e < EPC; ++e) e8[e] = exp2_fast(__builtin_fmaf(Fmt::get(x, e), c2, -kx));
#pragma unroll
        for (int w = 1; w < EPC; w <<= 1)
#pragma unroll
            for (int e = 0; e < EPC; e += 2 * w) e8[e] = e8[e] + e8[e + w];
        S = S + e8[0];
        __builtin_amdgcn_sched_barrier(0);  // one chunk in flight: bounded VGPRs
    }
}

// Two rows from load_rows_interleaved swept together: chunk n of both rows
// in iteration n, in the order the loads were issued, each row folded exactly
// as row_stats_tail folds it.  With second == false only the first row is
// folded (its partner's loads are ignored).
template <typename Fmt, int W, int CPT>
__device__ inline void row_stats2_tail(const chunk_t (&a)[CPT], const chunk_t (&b)[CPT], int nchunks, float c2,
                                       bool second, float& Ka, float& Sa, float& Kb, float& Sb) {
    constexpr int EPC = Fmt::kPerChunk;
#pragma unroll
    for (int n = 0; n < CPT; ++n) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            if (r == 1 && !second) continue;
            const chunk_t x = chunk_or_pad<Fmt, W>(r == 0 ? a[n] : b[n], n, nchunks);
            float& K = r == 0 ? Ka : Kb;
            float& S = r == 0 ? Sa : Sb;
            const float kn = fmaxf(K, ceilf(chunk_max<Fmt>(x) * c2));
            S = rescale(S, K, kn);
            K = kn;
            const float kx = fmaxf(K, -3.0e38f);  // see row_stats
            float e8[EPC];
#pragma unroll
            for (int e = 0; e < EPC; ++e) e8[e] = exp2_fast(__builtin_fmaf(Fmt::get(x, e), c2, -kx));
#pragma unroll
            for (int w = 1; w < EPC; w <<= 1)
#pragma unroll
                for (int e = 0; e < EPC; e += 2 * w) e8[e] = e8[e] + e8[e + w];
            S = S + e8[0];
        }
        __builtin_amdgcn_sched_barrier(0);  // one chunk pair in flight: bounded VGPRs
    }
}

// Fold one chunk into a thread's (K, S) exactly as row_stats does for each
// of its chunks (for rows streamed from memory rather than held).
template <typename Fmt>
__device__ inline void fold_chunk(const chunk_t& x, float c2, float& K, float& S) {
    constexpr int EPC = Fmt::kPerChunk;
    const float kn = fmaxf(K, ceilf(chunk_max<Fmt>(x) * c2));
    S = rescale(S, K, kn);
    K = kn;
    const float kx = fmaxf(K, -3.0e38f);  // see row_stats
    float e8[EPC];
#pragma unroll
    for (int e = 0; e < EPC; ++e) e8[e] = exp2_fast(__builtin_fmaf(Fmt::get(x, e), c2, -kx));
#pragma unroll
    for (int w = 1; w < EPC; w <<= 1)
#pragma unroll
        for (int e = 0; e < EPC; e += 2 * w) e8[e] = e8[e] + e8[e + w];
    S = S + e8[0];
}

// fold_chunk with every term accumulated in fp64 (as the fp64 row_stats).
template <typename Fmt>
__device__ inline void fold_chunk(const chunk_t& x, float c2, float& K, double& S) {
    constexpr int EPC = Fmt::kPerChunk;
    const float kn = fmaxf(K, ceilf(chunk_max<Fmt>(x) * c2));
    S = rescale(S, K, kn);
    K = kn;
    const float kx = fmaxf(K, -3.0e38f);
    double s0 = 0.0, s1 = 0.0;
#pragma unroll
    for (int e = 0; e < EPC; e += 2) {
        s0 += double(exp2_fast(__builtin_fmaf(Fmt::get(x, e), c2, -kx)));
        s1 += double(exp2_fast(__builtin_fmaf(Fmt::get(x, e + 1), c2, -kx)));
    }
    S += s0 + s1;
}

// Chunk ch of a row streamed from memory, or padding past its end.  VEC:
// a 16-byte load (a chunk past the row re-reads the last one, replaced by
// padding); otherwise element loads.
template <typename Fmt, bool VEC>
__device__ inline chunk_t stream_chunk(const void* row, int ch, int nchunks, int V) {
    if constexpr (VEC) {
        const bool in = ch < nchunks;
        const chunk_t v = __builtin_nontemporal_load(static_cast<const chunk_t*>(row) + (in ? ch : nchunks - 1));
        const chunk_t pad = pad_chunk<Fmt>();
        return chunk_t{in ? v.x : pad.x, in ? v.y : pad.y, in ? v.z : pad.z, in ? v.w : pad.w};
    } else {
        return ch < nchunks ? Fmt::load_scalar(row, int64_t(ch) * Fmt::kPerChunk, V) : pad_chunk<Fmt>();
    }
}

// fp64 accumulation of every term (for quantities first-order sensitive to
// the normaliser).
template <typename Fmt, int CPT>
__device__ inline void row_stats(const chunk_t (&c)[CPT], float c2, float& K, double& S) {
    constexpr int EPC = Fmt::kPerChunk;
#pragma unroll
    for (int n = 0; n < CPT; ++n) {
        const float kn = fmaxf(K, ceilf(chunk_max<Fmt>(c[n]) * c2));
        S = rescale(S, K, kn);
        K = kn;
        const float kx = fmaxf(K, -3.0e38f);  // see the fp32 version
        double s0 = 0.0, s1 = 0.0;
#pragma unroll
        for (int e = 0; e < EPC; e += 2) {
            s0 += double(exp2_fast(__builtin_fmaf(Fmt::get(c[n], e), c2, -kx)));
            s1 += double(exp2_fast(__builtin_fmaf(Fmt::get(c[n], e + 1), c2, -kx)));
        }
        S += s0 + s1;
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Merge (K, S) across the wave; every lane returns the wave's pair.
template <typename Acc>
__device__ inline void wave_merge_stats(float& K, Acc& S) {
    const float kw = wave_max(K);
    S = wave_sum(rescale(S, K, kw));
    K = kw;
}

// ---------------------------------------------------------------------------
// Fixed-point probability mass.  A non-negative fp32 value x < 2^(63-SH) maps
// to floor(x * 2^SH); the conversion is exact for x >= 2^(23-SH) (the
// mantissa is shifted, not rounded).  Integer sums of such values are
// associative, so every reduction order partitions a CDF identically.
// Values outside the domain never shift by 64 or more: negatives and
// subnormals give 0, and anything at or above 2^(63-SH) -- infinities and
// NaN included -- saturates at 2^39 * (2^24 - 1) < 2^63.  (Callers reject
// rows whose sums are not finite before they draw, so none reaches a draw.)
// ---------------------------------------------------------------------------
template <int SH>
__device__ inline uint64_t mass_to_fixed(float x) {
    const uint32_t b = __float_as_uint(x);
    const int e = int((b >> 23) & 0xFF) - 127;
    if (e < -126 || (b >> 31)) return 0;  // zero, subnormal or negative
    const uint64_t m = uint64_t((b & 0x7FFFFFu) | 0x800000u);
    int sh = e + SH - 23;  // x * 2^SH = m * 2^(e - 23 + SH)
    if (sh > 39) sh = 39;  // beyond the domain: saturate below 2^63
    if (sh >= 0) return m << sh;
    if (sh <= -64) return 0;
    return m >> (-sh);
}

// A row's sum of exponentials that a draw or a test can use: positive and
// finite (a NaN logit makes it NaN, an overflow makes it infinite).
__device__ inline bool usable_sum(double s) { return s > 0.0 && s < 1.0e300; }

// Two fp32 values to a packed pair of bf16, round to nearest even, with the
// native v_cvt_pk_bf16_f32 of gfx950.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
    const f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// ---------------------------------------------------------------------------
// Cross-workgroup hand-off through device memory, without cache flushes.
//
// Every word that crosses workgroups is written and read with agent-scope
// atomic read-modify-write operations, which the hardware performs at the
// device-wide coherence point (not in an XCD's private L2).  A publisher
// waits for its payload RMW to complete (s_waitcnt) before it bumps the
// arrival counter; the last arriver reads (and clears) the payloads with RMWs
// issued after its counter RMW returned.  Release/acquire fences would instead
// write back and invalidate the whole L2 of the XCD on every arrival.
// ---------------------------------------------------------------------------
__device__ inline void wait_memory() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// The publishing RMWs return their old value (consumed by an empty asm) so
// that the hardware reports their completion to the waiting s_waitcnt.
__device__ inline void publish_u32(uint32_t* p, uint32_t v) {
    uint32_t old = __hip_atomic_exchange(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    asm volatile("" ::"v"(old));
}
__device__ inline uint32_t take_u32(uint32_t* p) {  // read and clear
    return __hip_atomic_exchange(p, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void publish_f64(double* p, double v) {
    double old = __hip_atomic_exchange(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    asm volatile("" ::"v"(old));
}
__device__ inline double take_f64(double* p) {
    return __hip_atomic_exchange(p, 0.0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void publish_u64(uint64_t* p, uint64_t v) {
    uint64_t old = __hip_atomic_exchange(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    asm volatile("" ::"v"(old));
}
__device__ inline uint64_t take_u64(uint64_t* p) {  // read and clear
    return __hip_atomic_exchange(p, uint64_t(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t poll_u64(const uint64_t* p) {
    return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint32_t load_relaxed(const uint32_t* p) {
    return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Arrive at a counter; returns the number of earlier arrivals.  The caller's
// payload RMWs have completed before the add is issued.
__device__ inline uint32_t arrive(uint32_t* counter) {
    wait_memory();
    const uint32_t prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    wait_memory();
    return prev;
}

}  // namespace osd
