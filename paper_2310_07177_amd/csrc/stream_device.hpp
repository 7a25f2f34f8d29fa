// stream_device.hpp -- building blocks of the persistent streaming kernels
// (gfx950, wave64).
//
// A persistent workgroup walks a list of rows.  Each thread owns the 16-byte
// chunks n*W + tid (n = 0..CPT-1) of every row, so each round n is one
// coalesced sweep over W*16 bytes.  Rows are read through buffer descriptors:
// a descriptor of 0 bytes turns every load into a no-op that returns zeros
// without touching memory, so the instruction stream is the same whether or
// not the next row exists.  That keeps the hardware load counter in a fixed
// order, which lets the compiler wait for exactly the chunk it needs while
// the prefetch of the next row stays in flight.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "osd_device.hpp"

namespace osd {

typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Fourth descriptor word for raw (untyped) buffer access on gfx9-class parts:
// 32-bit data format, no swizzle, no index stride.
constexpr int kRsrcWord3 = 0x00020000;
// Cache policy of streaming loads and stores: non-temporal (the data is used
// once per call).
constexpr int kStreamAux = 2;

__device__ inline rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), kRsrcWord3);
}

// Chunk n of this thread (byte offset (n*W + tid)*16).  Out-of-range chunks
// read as zeros.
template <int W>
__device__ inline chunk_t load_chunk(rsrc_t r, int n) {
    const int off = (n * W + static_cast<int>(threadIdx.x)) * 16;
    return __builtin_bit_cast(chunk_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kStreamAux));
}

template <int W>
__device__ inline void store_chunk(rsrc_t r, int n, const chunk_t& c) {
    const int off = (n * W + static_cast<int>(threadIdx.x)) * 16;
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((ext_vector_type(4))) int, c),
                                           r, off, 0, kStreamAux);
}

// Chunk c of a row, whoever holds it (byte offset c*16).
__device__ inline void store_chunk_at(rsrc_t r, int c, const chunk_t& v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((ext_vector_type(4))) int, v), r, c * 16,
                                           0, kStreamAux);
}

// Uniform (scalar-cache) loads of small per-row arguments.  The address must
// be the same in every lane; the value lands in a scalar register and its
// wait does not depend on the vector loads in flight.
template <typename T>
__device__ inline T scalar_load(const T* p) {
    return *(const __attribute__((address_space(4))) T*)(p);
}

// Byte i of a uint8 array, through the aligned dword that holds it.
__device__ inline uint32_t scalar_load_u8(const uint8_t* base, int64_t i) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(base) + uintptr_t(i);
    const uint32_t w = scalar_load(reinterpret_cast<const uint32_t*>(a & ~uintptr_t(3)));
    return (w >> (8 * (a & 3))) & 0xFFu;
}

// Element j of a logit row as fp32, through the aligned dword that holds it
// (the row itself is 16-byte aligned on the streaming path).
template <typename Fmt>
__device__ inline float scalar_load_logit(const void* row, int j) {
    if constexpr (Fmt::kBytes == 2) {
        const uint32_t w = scalar_load(static_cast<const uint32_t*>(row) + (j >> 1));
        return (j & 1) ? __uint_as_float(w & 0xFFFF0000u) : __uint_as_float(w << 16);
    } else {
        return scalar_load(static_cast<const float*>(row) + j);
    }
}

// The per-thread shift of a row: the whole number ceil(max * c2) over the
// thread's first chunk, or 0 when that chunk has no finite logit.  Every
// later exponent is taken relative to it; a row whose later elements exceed
// it by more than the fp32 exponent range is caught by the caller (the sum
// overflows) and rescaled exactly.
// The shift of a maximum m: ceil(m * c2), or 0 when m is not finite.
__device__ inline float shift_of_max(float m, float c2) {
    const float k = ceilf(m * c2);
    return (k > -3.0e38f && k < 3.0e38f) ? k : 0.0f;
}

template <typename Fmt>
__device__ inline float first_chunk_shift(const chunk_t& c, float c2) {
    return shift_of_max(chunk_max<Fmt>(c), c2);
}

// The largest element of a thread's CPT chunks of one row (pad_last: the
// last chunk is padding), element by element.
template <typename Fmt, int CPT>
__device__ inline float chunks_max_exact(const chunk_t (&x)[CPT], bool pad_last) {
    float m = kNegInf;
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
        const chunk_t c = (r == CPT - 1 && pad_last) ? pad_chunk<Fmt>() : x[r];
        m = fmaxf(m, chunk_max<Fmt>(c));
    }
    return m;
}

// The same maximum.  For bf16 the chunks' 16-bit patterns are first compared
// as f16 numbers, two per packed instruction with three operands: both
// formats are sign-magnitude with the exponent above the mantissa, so the
// two orders agree wherever the f16 reading is finite, that is for bf16
// magnitudes below 2^121, and the winning pattern is the bf16 maximum.  The
// f16 maximum propagates NaN, so a thread holding a pattern outside that
// range (an infinity, a NaN, a magnitude of 2^121 or more) or only padding
// (f16 -inf) gets an unusable result and is decided element by element.
// Either way the value is the exact maximum.
template <typename Fmt, int CPT>
__device__ inline float chunks_max(const chunk_t (&x)[CPT], bool pad_last) {
    if constexpr (Fmt::kPerChunk == 8) {
        typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
        constexpr uint32_t kNegInfPair = 0xFC00FC00u;  // f16 -inf in both halves
        const auto H = [](uint32_t w) { return __builtin_bit_cast(h2_t, w); };
        const auto mx = [](h2_t u, h2_t v) { return __builtin_elementwise_maximum(u, v); };
        h2_t m = H(kNegInfPair);
#pragma unroll
        for (int r = 0; r < CPT - 1; ++r)
            m = mx(mx(mx(m, H(x[r].x)), mx(H(x[r].y), H(x[r].z))), H(x[r].w));
        // The last chunk joins unless it is padding (one select).
        const chunk_t& l = x[CPT - 1];
        const h2_t ml = mx(mx(mx(m, H(l.x)), mx(H(l.y), H(l.z))), H(l.w));
        m = pad_last ? m : ml;
        const uint32_t b = __builtin_bit_cast(uint32_t, m);
        const float lo = __uint_as_float(b << 16), hi = __uint_as_float(b & 0xFFFF0000u);
        if (__builtin_fabsf(lo) < 0x1p121f && __builtin_fabsf(hi) < 0x1p121f) return fmaxf(lo, hi);
    }
    return chunks_max_exact<Fmt, CPT>(x, pad_last);
}

// The thread index through an opaque copy: lane and wave numbers derived from
// it are recomputed where they are used instead of being kept alive (or
// spilled) across a long loop.
__device__ inline int opaque_tid() {
    int t = threadIdx.x;
    asm volatile("" : "+v"(t));
    return t;
}

// Wave totals, uniform.  (The maximum of values without NaN.)
__device__ inline float wave_max_u(float v) {
    uint32_t k = float_key(v);
    k = dpp_umax_step<kDppRowShr1, 0xF>(k);
    k = dpp_umax_step<kDppRowShr2, 0xF>(k);
    k = dpp_umax_step<kDppRowShr4, 0xF>(k);
    k = dpp_umax_step<kDppRowShr8, 0xF>(k);
    k = dpp_umax_step<kDppRowBcast15, 0xA>(k);
    k = dpp_umax_step<kDppRowBcast31, 0xC>(k);
    return key_float(readlane_u32(k, kWave - 1));
}
__device__ inline double wave_sum_u(double v) { return readlane_f64(wave_scan_add(v), kWave - 1); }

// log2 of a positive finite double to within about 6e-8 (absolute): the
// binary exponent, v_log_f32 of the fp32 rounding of the mantissa taken in
// [sqrt(1/2), sqrt(2)) (so a ratio near 1 keeps its relative accuracy; the
// instruction is within one unit in the last place of its result there),
// and the first-order term of that rounding.  A fraction of the fp64
// library routine's cost.
__device__ inline double log2_pos(double x) {
    int ex;
    double m = __builtin_frexp(x, &ex);  // [0.5, 1)
    if (m < 0.70710678118654752) {
        m *= 2.0;
        ex -= 1;
    }
    const float mf = float(m);
    const float corr = float(m - double(mf)) * (1.44269504f * __builtin_amdgcn_rcpf(mf));
    return double(ex) + double(__builtin_amdgcn_logf(mf)) + double(corr);
}

// Totals of lanes 0..15 when every other lane holds the identity: the row
// steps of the scans alone.  Equal, bit for bit, to the wave totals above
// (the remaining steps only combine identities).
__device__ inline float row0_max_u(float v) {
    uint32_t k = float_key(v);
    k = dpp_umax_step<kDppRowShr1, 0xF>(k);
    k = dpp_umax_step<kDppRowShr2, 0xF>(k);
    k = dpp_umax_step<kDppRowShr4, 0xF>(k);
    k = dpp_umax_step<kDppRowShr8, 0xF>(k);
    return key_float(readlane_u32(k, 15));
}
__device__ inline double row0_sum_u(double v) {
    v = dpp_add_step<kDppRowShr1, 0xF>(v);
    v = dpp_add_step<kDppRowShr2, 0xF>(v);
    v = dpp_add_step<kDppRowShr4, 0xF>(v);
    v = dpp_add_step<kDppRowShr8, 0xF>(v);
    return readlane_f64(v, 15);
}

// Merge (K, S) pairs over the wave: K = max K, S = sum S 2^(K_lane - K).
// Every lane gets the wave's pair.
__device__ inline void wave_merge_stats_u(float& K, double& S) {
    const float kw = wave_max_u(K);
    S = wave_sum_u(rescale(S, K, kw));
    K = kw;
}
// The same for pairs held by lanes 0..15 (identity elsewhere).
__device__ inline void row0_merge_stats_u(float& K, double& S) {
    const float kw = row0_max_u(K);
    S = row0_sum_u(rescale(S, K, kw));
    K = kw;
}

// Workgroup merge of the (K, S) pairs of two rows.  Each wave merges its
// lanes; lane 0 of every wave posts the wave's pairs to LDS; after one
// barrier every wave merges the NW posted pairs the same way (so all agree,
// bit for bit).  s_k: [2*NW] floats, s_s: [2*NW] doubles, not written again
// before the caller's next barrier.
template <int NW>
__device__ inline void block_merge2(float& K0, double& S0, float& K1, double& S1, float* s_k, double* s_s) {
    static_assert(NW <= 16, "the posted pairs fit one DPP row");
    const int t = opaque_tid(), lane = t & (kWave - 1), wid = t / kWave;
    wave_merge_stats_u(K0, S0);
    wave_merge_stats_u(K1, S1);
    if (lane == 0) {
        s_k[wid] = K0;
        s_k[NW + wid] = K1;
        s_s[wid] = S0;
        s_s[NW + wid] = S1;
    }
    __syncthreads();
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
    K0 = k0;
    S0 = t0;
    K1 = k1;
    S1 = t1;
}

// Workgroup sums of two doubles, the same way (one barrier).
template <int NW>
__device__ inline void block_sum2(double& A0, double& A1, double* s_a) {
    static_assert(NW <= 16, "the posted sums fit one DPP row");
    const int t = opaque_tid(), lane = t & (kWave - 1), wid = t / kWave;
    A0 = wave_sum_u(A0);
    A1 = wave_sum_u(A1);
    if (lane == 0) {
        s_a[wid] = A0;
        s_a[NW + wid] = A1;
    }
    __syncthreads();
    double t0 = lane < NW ? s_a[lane] : 0.0;
    double t1 = lane < NW ? s_a[NW + lane] : 0.0;
    A0 = row0_sum_u(t0);
    A1 = row0_sum_u(t1);
}

// Argmax step: the larger value, the lower index among equal values.
template <int CTRL, int ROWS>
__device__ inline void dpp_argmax_step(float& v, int& idx) {
    const float ov = __uint_as_float(dpp<CTRL, ROWS>(0xFF800000u, __float_as_uint(v)));
    const int oi = int(dpp<CTRL, ROWS>(0x7FFFFFFFu, uint32_t(idx)));
    if (ov > v || (ov == v && oi < idx)) {
        v = ov;
        idx = oi;
    }
}
// Max value, lowest index among equal maxima; uniform result.
__device__ inline void wave_argmax_u(float& v, int& idx) {
    dpp_argmax_step<kDppRowShr1, 0xF>(v, idx);
    dpp_argmax_step<kDppRowShr2, 0xF>(v, idx);
    dpp_argmax_step<kDppRowShr4, 0xF>(v, idx);
    dpp_argmax_step<kDppRowShr8, 0xF>(v, idx);
    dpp_argmax_step<kDppRowBcast15, 0xA>(v, idx);
    dpp_argmax_step<kDppRowBcast31, 0xC>(v, idx);
    v = readlane_f32(v, kWave - 1);
    idx = int(readlane_u32(uint32_t(idx), kWave - 1));
}

// Exact fp32 -> fixed point with SH fractional bits (x >= 0, x < 2^(63-SH)).
template <int SH>
__device__ inline uint64_t to_fixed(float x) { return mass_to_fixed<SH>(x); }


}  // namespace osd
