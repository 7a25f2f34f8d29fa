// cache_draw.hpp -- inverse-CDF draw over a row whose element masses are
// held on chip (an LDS and a register half, or LDS alone), the sampling rule
// of the extra token (Eq. 5 of arXiv:2310.07177, Appendix A.1) as the
// streaming kernels take it.
#pragma once

#include "osd_device.hpp"
#include "stream_device.hpp"

namespace osd {

// Inverse-CDF draw over a cached row.  mass(r, e) gives the fp32
// mass of element e of round r (RESIDUAL: max(0, p - q); else p) and
// mass_at(rr, e) the same for a round rr known only at run time.  Token order
// is chunk order c = r*W + tid, then element; the cells are (round r, wave w,
// lane).  Masses become 2^-40 fixed point, held as whole numbers in fp64
// (every sum below stays under 2^53, so each is exact): the chunk sum x, an
// fp32 sum of at most 8 masses of at most 1, becomes floor(x 2^40).  Pass A
// posts each (round, wave) total; one wave scans them (CPT*NW <= 64 cells).
// The wave whose cell holds u*Z recomputes that round's chunk sums -- the
// same fp32 additions of the same values -- finds the lane, and the lane
// walks its elements.  Returns the token (uniform), or -1 if there is no mass
// at all.  All threads call it.
__device__ inline double fixed40(float x) { return floor(double(x) * 0x1p40); }

template <int W, int CPT, int EPC, bool RESIDUAL, typename MassFn, typename MassAtFn>
__device__ int draw_cached(MassFn mass, MassAtFn mass_at, float u, double* s_cell, double* s_z, int* s_tok) {
    constexpr int NW = W / kWave, CELLS = CPT * NW;
    static_assert(CELLS <= kWave, "one wave scans the cells");
    const int tid = opaque_tid(), lane = tid & (kWave - 1), wid = tid / kWave;
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
        float sm = 0.0f;
#pragma unroll
        for (int e = 0; e < EPC; ++e) sm = sm + mass(r, e);
        const double incl = wave_scan_add(fixed40(sm));
        if (lane == kWave - 1) s_cell[r * NW + wid] = incl;
        __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    if (wid == 0) {
        const double cv = lane < CELLS ? s_cell[lane] : 0.0;
        const double ci = wave_scan_add(cv);
        if (lane < CELLS) s_cell[lane] = ci - cv;  // exclusive prefix
        if (lane == kWave - 1) *s_z = ci;
        if (lane == 0) *s_tok = -1;
    }
    __syncthreads();
    const double Z = *s_z;
    int tok = -1;
    if (Z > 0.0) {
        double target = floor(double(u) * Z);
        if (target >= Z) target = Z - 1.0;
        // The round whose cell of this wave holds the target (uniform).
        int rr = -1;
        double lo = 0.0;
        for (int r = 0; r < CPT; ++r) {
            const int c = r * NW + wid;
            const double l = s_cell[c];
            const double h = c + 1 < CELLS ? s_cell[c + 1] : Z;
            if (l <= target && target < h) {
                rr = r;
                lo = l;
            }
        }
        if (rr >= 0) {
            float sm = 0.0f;
#pragma unroll
            for (int e = 0; e < EPC; ++e) sm = sm + mass_at(rr, e);
            const double f = fixed40(sm);
            const double mylo = lo + (wave_scan_add(f) - f);
            if (f > 0.0 && mylo <= target && target < mylo + f) {
                // The lane's masses again (the same values: held across the
                // scan they would cost EPC registers).
                const double want = target - mylo;
                float racc = 0.0f;
                int pick = -1, last_pos = -1;
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    const float me = mass_at(rr, e);
                    racc = racc + me;
                    if (me > 0.0f) last_pos = e;
                    if (pick < 0 && fixed40(racc) > want) pick = e;
                }
                if (pick < 0) pick = last_pos >= 0 ? last_pos : 0;
                *s_tok = (rr * W + tid) * EPC + pick;
            }
        }
        __syncthreads();
        tok = *s_tok;
    }
    __syncthreads();  // s_cell, s_z and s_tok are rewritten by the next draw
    return tok;
}

}  // namespace osd
