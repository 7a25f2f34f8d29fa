// row_draw.hpp -- inverse-CDF draw over a register-resident row (pair), the
// sampling rule of the verification's extra token (Eq. 5 of
// arXiv:2310.07177, Appendix A.1) and of token sampling.
//
// Element masses are fp32; each thread's chunk sums are converted exactly to
// 2^-SH fixed point, so every partial sum of the CDF is an exact integer and
// the cells partition [0, Z) without gaps or overlaps whatever the reduction
// order.  The token is the first element (ascending id) whose running sum
// exceeds u*Z.
#pragma once

#include "osd_device.hpp"

namespace osd {

// x 2^SH as a whole number held in fp64: for masses of at most 1 per element
// (chunk sums at most 8) and SH <= 44, every chunk value is below 2^47 and
// every wave sum at most 2^53, so each is exact -- and equal to
// mass_to_fixed<SH>(x), which takes more instructions.
template <int SH>
__device__ inline double fixed_f64(float x) {
    static_assert(SH <= 44, "exact below 2^53 only for SH <= 44");
    return floor(double(x) * double(1ull << SH));
}

struct DrawShared {
    int cell_round, cell_wave;
    unsigned long long target;  // offset of u*Z inside the winning cell
};

// The winning wave's last step (both draws): this lane's chunk of round
// nstar has masses m[] (sum s, added left to right from 0); target is the
// point's offset inside the wave's cell.  The lanes' fixed-point chunk sums
// are scanned to find the lane holding the target, which walks its elements
// with the same left-to-right fp32 sums.  Returns the token on that lane and
// -1 on the others.
template <int SH, int W, int EPC>
__device__ inline int walk_chunk(const float (&m)[EPC], float s, uint64_t target, int nstar) {
    const int tid = threadIdx.x;
    int pick = -1, last_pos = -1;
    if constexpr (SH <= 44) {
        // Offsets inside one cell stay below 2^53: exact in fp64.
        const double v = fixed_f64<SH>(s);
        const double incl = wave_scan_add(v);
        const double lo = incl - v, t = double(target);
        if (!(v > 0.0 && lo <= t && t < incl)) return -1;
        const double want = t - lo;
        float run = 0.0f;
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
            run = run + m[e];
            if (m[e] > 0.0f) last_pos = e;
            if (pick < 0 && fixed_f64<SH>(run) > want) pick = e;
        }
    } else {
        const uint64_t v = mass_to_fixed<SH>(s);
        const uint64_t incl = wave_inclusive_scan(v);
        const uint64_t lo = incl - v;
        if (!(v > 0 && lo <= target && target < incl)) return -1;
        const uint64_t want = target - lo;
        float run = 0.0f;
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
            run = run + m[e];
            if (m[e] > 0.0f) last_pos = e;
            if (pick < 0 && mass_to_fixed<SH>(run) > want) pick = e;
        }
    }
    if (pick < 0) pick = last_pos >= 0 ? last_pos : 0;
    return (nstar * W + tid) * EPC + pick;
}

// Inverse-CDF draw over a register-resident row pair.  mass(t, d, e) returns
// the non-negative fp32 mass of element e of the chunks t, d (0 for padding).
// Returns the drawn token on exactly one thread and -1 on every other thread;
// *z_zero is set (uniformly) when the total mass is zero.  The point drawn is
// floor(u * Z) in fixed point, or, when c_given >= 0, c_given itself (a point
// already chosen in a larger CDF of which this row is one part); either is
// clamped to Z - 1.
//
// Token order is (round n, wave w, lane, element e).  Chunk masses are summed
// left to right in fp32 and converted exactly to fixed point, so every partial
// sum below is an exact integer and the CDF cells (n, w) partition [0, Z)
// without gaps or overlaps whatever the reduction order.  The winning wave
// stages its chunks through LDS (s_stage, 2*CPT*64 chunks) so that the
// winning round is selected by address, never by register index.
template <int SH, int W, int CPT, int EPC, typename MassFn>
__device__ int draw_inverse_cdf(const chunk_t (&tv)[CPT], const chunk_t (&dv)[CPT], MassFn mass,
                                float u, unsigned long long* s_tot, DrawShared* s_draw,
                                chunk_t* s_stage, bool* z_zero, long long c_given = -1) {
    constexpr int NW = W / kWave;
    constexpr int CELLS = CPT * NW;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;

#pragma unroll
    for (int n = 0; n < CPT; ++n) {
        float s = 0.0f;
#pragma unroll
        for (int e = 0; e < EPC; ++e) s = s + mass(tv[n], dv[n], e);
        uint64_t t;
        if constexpr (SH <= 44)
            t = uint64_t(wave_sum(fixed_f64<SH>(s)));
        else
            t = wave_sum(mass_to_fixed<SH>(s));
        if (lane == 0) s_tot[n * NW + wid] = t;
        __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    if (wid == 0) {
        uint64_t z = 0;
        for (int c0 = lane; c0 < CELLS; c0 += kWave) z += s_tot[c0];
        z = wave_sum(z);
        if (lane == 0) s_draw->cell_round = -1;
        if (z > 0) {
            uint64_t c = c_given >= 0 ? static_cast<uint64_t>(c_given)
                                      : static_cast<uint64_t>(double(u) * double(z));
            if (c >= z) c = z - 1;
            uint64_t carry = 0;
            for (int base = 0; base < CELLS; base += kWave) {
                const int idx = base + lane;
                const uint64_t v = idx < CELLS ? uint64_t(s_tot[idx]) : 0;
                const uint64_t incl = wave_inclusive_scan(v) + carry;
                const uint64_t lo = incl - v;
                if (v > 0 && lo <= c && c < incl) {
                    s_draw->cell_round = idx / NW;
                    s_draw->cell_wave = idx % NW;
                    s_draw->target = c - lo;
                }
                carry = static_cast<uint64_t>(__shfl(static_cast<unsigned long long>(incl), kWave - 1, kWave));
            }
        }
    }
    __syncthreads();
    const int nstar = s_draw->cell_round;
    *z_zero = nstar < 0;
    if (nstar < 0 || wid != s_draw->cell_wave) return -1;

    // Winning wave: stage every round through LDS, pick round nstar by address.
#pragma unroll
    for (int n = 0; n < CPT; ++n) {
        s_stage[n * kWave + lane] = tv[n];
        s_stage[(CPT + n) * kWave + lane] = dv[n];
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const chunk_t tc = s_stage[nstar * kWave + lane];
    const chunk_t dc = s_stage[(CPT + nstar) * kWave + lane];
    float m[EPC];
    float s = 0.0f;
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
        m[e] = mass(tc, dc, e);
        s = s + m[e];
    }
    return walk_chunk<SH, W, EPC>(m, s, s_draw->target, nstar);
}

}  // namespace osd

namespace osd {

// Rounds of a row streamed by a workgroup of W threads: chunk r*W + tid in
// round r.  The streamed kernels hold at most kMaxStreamRounds rounds' worth of
// cell totals in LDS (16 rounds of 1024 threads: 131072 bf16 or 65536 fp32
// logits per row).
constexpr int kMaxStreamRounds = 16;

// Inverse-CDF draw over a row that is streamed from memory instead of held in
// registers.  masses(r, m) fills m[0..EPC) with the non-negative fp32 masses
// of this thread's chunk in round r (0 for padding); it is called once per
// round in pass A and once more, for the winning round, by the winning wave in
// pass B, and must return the same values both times.  Cells are (round,
// wave); chunk masses are summed left to right in fp32 and converted exactly
// to 2^-SH fixed point, as in draw_inverse_cdf, so the CDF cells partition
// [0, Z) exactly.  Returns the token on one thread and -1 on the others;
// *z_zero is set (uniformly) when the total mass is zero.  s_tot holds
// R * (W / 64) cells.  All threads call it.
template <int SH, int W, int EPC, typename MassFn>
__device__ int draw_inverse_cdf_streamed(int R, MassFn masses, float u, unsigned long long* s_tot,
                                         DrawShared* s_draw, bool* z_zero) {
    constexpr int NW = W / kWave;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int cells = R * NW;
    for (int r = 0; r < R; ++r) {
        float m[EPC];
        masses(r, m);
        float s = 0.0f;
#pragma unroll
        for (int e = 0; e < EPC; ++e) s = s + m[e];
        uint64_t t;
        if constexpr (SH <= 44)
            t = uint64_t(wave_sum(fixed_f64<SH>(s)));
        else
            t = wave_sum(mass_to_fixed<SH>(s));
        if (lane == 0) s_tot[r * NW + wid] = t;
    }
    __syncthreads();
    if (wid == 0) {
        uint64_t z = 0;
        for (int c0 = lane; c0 < cells; c0 += kWave) z += s_tot[c0];
        z = wave_sum(z);
        if (lane == 0) s_draw->cell_round = -1;
        if (z > 0) {
            uint64_t c = static_cast<uint64_t>(double(u) * double(z));
            if (c >= z) c = z - 1;
            uint64_t carry = 0;
            for (int base = 0; base < cells; base += kWave) {
                const int idx = base + lane;
                const uint64_t v = idx < cells ? uint64_t(s_tot[idx]) : 0;
                const uint64_t incl = wave_inclusive_scan(v) + carry;
                const uint64_t lo = incl - v;
                if (v > 0 && lo <= c && c < incl) {
                    s_draw->cell_round = idx / NW;
                    s_draw->cell_wave = idx % NW;
                    s_draw->target = c - lo;
                }
                carry = static_cast<uint64_t>(__shfl(static_cast<unsigned long long>(incl), kWave - 1, kWave));
            }
        }
    }
    __syncthreads();
    const int nstar = s_draw->cell_round;
    *z_zero = nstar < 0;
    if (nstar < 0 || wid != s_draw->cell_wave) return -1;
    float m[EPC];
    masses(nstar, m);
    float s = 0.0f;
#pragma unroll
    for (int e = 0; e < EPC; ++e) s = s + m[e];
    return walk_chunk<SH, W, EPC>(m, s, s_draw->target, nstar);
}

}  // namespace osd
