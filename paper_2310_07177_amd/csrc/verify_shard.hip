// verify_shard.hip -- speculative-sampling verification with the vocabulary
// split over G ranks (a tensor-parallel LM head), on gfx950.
//
// Method: the verification of Appendix A.1 and Eq. 5 of arXiv:2310.07177
// (accept y_i while u_i < p(y_i)/q(y_i); at the first rejection a draw one
// token from norm(max(0, p - q)); if all k_b proposals pass, draw from p at
// the bonus row).  No rank holds a whole row, so the work runs in three
// phases with an exchange of small records between them:
//
//   shard_stats_kernel  one workgroup per row pair (b, i), i <= k_b: reduce the
//                       rank's slice of the target (and draft) row to a base-2
//                       shift and sum of exponentials -- the same streaming
//                       statistics as the whole-row kernels -- and pick up the
//                       proposal's logits where the slice holds it;
//   shard_mass_kernel   one workgroup per sequence: stage the G records of the
//                       rows 0..k_b in LDS, merge them in rank order (exact
//                       power-of-two rescaling, fp64 sums in a fixed DPP order,
//                       so every rank gets bit-identical normalisers), take the
//                       acceptance tests in order and stop at the first
//                       rejection a; then sum the extra draw's mass over the
//                       rank's slice of row a in 2^-44 fixed point;
//   shard_draw_kernel   one workgroup per sequence: add the G slice masses
//                       (exact integers), place u*Z, and let the one rank whose
//                       slice holds it walk its slice with the inverse CDF of
//                       the whole-row kernels.
//
// Because every chunk mass is converted exactly to an integer before it is
// summed, the whole row's CDF is the concatenation of the slices' CDFs, and
// the token drawn does not depend on how the vocabulary is split.
#include "osd.h"
#include "osd_device.hpp"
#include "osd_internal.hpp"
#include "row_draw.hpp"

namespace osd {
namespace {

static_assert(sizeof(osd_shard_row_stats) == 40, "record layout");
static_assert(sizeof(osd_shard_mass) == 48, "record layout");

// 2^-44 fixed point, as the whole-row verification: an element's mass is at
// most 1 unit, so a whole row of V <= 2^19 tokens totals below 2^63.
constexpr int kFixedShift = 44;
constexpr int kRecWords = sizeof(osd_shard_row_stats) / 4;

enum : int32_t { kHoldsY = 1, kBadToken = 2 };

// The extra draw's mass of element e, in units of the target row's sum of
// exponentials: p_j S_t = 2^(t_j c2 - K_t), q_j S_t = 2^(d_j c2 - K_d) S_t/S_d.
// The mass and the draw kernels evaluate it with this one expression, so the
// chunk sums that the draw walks are the ones whose totals were exchanged.
template <typename Fmt>
struct SliceMass {
    float c2, kt, kd, rho;
    bool p_only;
    __device__ float operator()(const chunk_t& tc, const chunk_t& dc, int e) const {
        const float pt = exp2_fast(__builtin_fmaf(Fmt::get(tc, e), c2, -kt));
        if (p_only) return pt;
        const float qt = exp2_fast(__builtin_fmaf(Fmt::get(dc, e), c2, -kd));
        return fmaxf(__builtin_fmaf(-qt, rho, pt), 0.0f);
    }
};

__device__ inline int draft_len_of(const int32_t* draft_len, int b, int K) {
    return draft_len ? draft_len[b] : K;
}

// ---------------------------------------------------------------------------
// Phase 1: slice statistics.
// ---------------------------------------------------------------------------
struct StatsArgs {
    const void* target;
    const void* draft;
    int B, K, Vs, v_begin, V;
    const int32_t* tokens;
    const int32_t* draft_len;
    float c2;
    osd_shard_row_stats* stats;
};

template <typename Fmt, int W, int CPT, bool VEC, bool GREEDY>
__global__ __launch_bounds__(W, 4) void shard_stats_kernel(StatsArgs a) {
    constexpr int NW = W / kWave;
    constexpr int EPC = Fmt::kPerChunk;
    __shared__ float s_k[2][NW];
    __shared__ double s_s[2][NW];
    __shared__ int s_idx[NW];

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int B = a.B, K = a.K, Vs = a.Vs;
    const int i = blockIdx.x / B, b = blockIdx.x - i * B;
    const int kb = draft_len_of(a.draft_len, b, K);
    if (kb < 1 || kb > K || i > kb) return;  // padding row, or a sequence phase 2 rejects
    const bool bonus = i == kb;

    int32_t flags = 0;
    int yl = -1;
    if (!bonus) {
        const int y = a.tokens[int64_t(b) * K + i];
        if (y < 0 || y >= a.V) {
            flags |= kBadToken;
        } else if (y >= a.v_begin && y - a.v_begin < Vs) {
            flags |= kHoldsY;
            yl = y - a.v_begin;
        }
    }
    const char* trow = static_cast<const char*>(a.target) + (int64_t(b) * (K + 1) + i) * int64_t(Vs) * Fmt::kBytes;
    chunk_t tv[CPT];
    load_row<Fmt, W, CPT, VEC>(tv, trow, Vs);
    osd_shard_row_stats* out = a.stats + int64_t(b) * (K + 1) + i;

    if constexpr (GREEDY) {
        // Slice argmax, lowest index on ties (indices grow with (n, e) in a
        // thread, so a strict ">" keeps the first maximum).
        float best = kNegInf;
        int bi = 0x7FFFFFFF;
#pragma unroll
        for (int n = 0; n < CPT; ++n)
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float x = Fmt::get(tv[n], e);
                if (x > best) {
                    best = x;
                    bi = (n * W + tid) * EPC + e;
                }
            }
        wave_argmax(best, bi);
        if (lane == 0) {
            s_k[0][wid] = best;
            s_idx[wid] = bi;
        }
        __syncthreads();
        if (tid == 0) {
            float bv = s_k[0][0];
            int g = s_idx[0];
            for (int w = 1; w < NW; ++w)
                if (s_k[0][w] > bv || (s_k[0][w] == bv && s_idx[w] < g)) {
                    bv = s_k[0][w];
                    g = s_idx[w];
                }
            osd_shard_row_stats r = {};
            r.k_target = bv;
            r.k_draft = kNegInf;
            r.argmax = bv > kNegInf ? a.v_begin + g : -1;
            r.flags = flags;
            *out = r;
        }
    } else {
        const float c2 = a.c2;
        chunk_t dv[CPT];
        const char* drow = static_cast<const char*>(a.draft) + (int64_t(b) * K + i) * int64_t(Vs) * Fmt::kBytes;
        if (!bonus) load_row<Fmt, W, CPT, VEC>(dv, drow, Vs);
        float Kt = kNegInf, Kd = kNegInf;
        float st = 0.0f, sd = 0.0f;
        row_stats<Fmt, CPT>(tv, c2, Kt, st);
        if (!bonus) row_stats<Fmt, CPT>(dv, c2, Kd, sd);
        double dt = st, dd = sd;
        wave_merge_stats(Kt, dt);
        wave_merge_stats(Kd, dd);
        if (lane == 0) {
            s_k[0][wid] = Kt;
            s_k[1][wid] = Kd;
            s_s[0][wid] = dt;
            s_s[1][wid] = dd;
        }
        __syncthreads();
        if (tid == 0) {
            float kt = s_k[0][0], kd = s_k[1][0];
            for (int w = 1; w < NW; ++w) {
                kt = fmaxf(kt, s_k[0][w]);
                kd = fmaxf(kd, s_k[1][w]);
            }
            double St = 0.0, Sd = 0.0;
            for (int w = 0; w < NW; ++w) {
                St += rescale(s_s[0][w], s_k[0][w], kt);
                Sd += rescale(s_s[1][w], s_k[1][w], kd);
            }
            osd_shard_row_stats r = {};
            r.s_target = St;
            r.s_draft = Sd;
            r.k_target = kt;
            r.k_draft = kd;
            r.argmax = -1;
            r.flags = flags;
            if (flags & kHoldsY) {
                r.t_y = Fmt::load_one(trow, yl);
                r.d_y = Fmt::load_one(drow, yl);
            }
            *out = r;
        }
    }
}

// ---------------------------------------------------------------------------
// Phase 2: merge, decide, and this slice's mass of the extra draw.
// ---------------------------------------------------------------------------
struct MassArgs {
    const void* target;
    const void* draft;
    int B, K, Vs, G;
    const int32_t* tokens;
    const int32_t* draft_len;
    const float* u_accept;
    float c2;
    double c2d;
    const osd_shard_row_stats* stats_all;
    osd_shard_mass* mass;
};

struct Decision {
    int acc;  // a_b, or -1
    int token;
    float kt, kd;
    double st, sd;
};

__device__ inline bool finite_shift(float k) { return k > kNegInf && k < -kNegInf; }

template <typename Fmt, int W, int CPT, bool VEC, bool GREEDY>
__global__ __launch_bounds__(W, 4) void shard_mass_kernel(MassArgs a) {
    constexpr int NW = W / kWave;
    constexpr int EPC = Fmt::kPerChunk;
    extern __shared__ osd_shard_row_stats s_rec[];  // [G][k_b + 1], sized at launch for G (K + 1)
    __shared__ Decision s_dec;
    __shared__ unsigned long long s_z[2][NW];

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int B = a.B, K = a.K, Vs = a.Vs, G = a.G;
    const int b = blockIdx.x;
    const int kb = draft_len_of(a.draft_len, b, K);
    osd_shard_mass* out = a.mass + b;
    if (kb < 1 || kb > K) {
        if (tid == 0) {
            osd_shard_mass r = {};
            r.accepted = -1;
            r.token = -1;
            *out = r;
        }
        return;
    }

    // Stage the records of rows 0..k_b of every rank: [g][i], word by word.
    {
        const int per_rank = (kb + 1) * kRecWords;
        uint32_t* dst = reinterpret_cast<uint32_t*>(s_rec);
        for (int t = tid; t < G * per_rank; t += W) {
            const int g = t / per_rank, r = t - g * per_rank;
            const uint32_t* src =
                reinterpret_cast<const uint32_t*>(a.stats_all + (int64_t(g) * B + b) * (K + 1));
            dst[g * per_rank + r] = src[r];
        }
    }
    __syncthreads();

    if (wid == 0) {
        const bool mine = lane < G;
        auto rec = [&](int i) -> const osd_shard_row_stats& { return s_rec[(mine ? lane : 0) * (kb + 1) + i]; };
        Decision d;
        d.acc = -1;
        d.token = -1;
        d.kt = d.kd = kNegInf;
        d.st = d.sd = 0.0;
        // A proposal outside the vocabulary invalidates the sequence wherever
        // it sits (every rank flags it).
        bool bad = false;
        for (int i = 0; i < kb; ++i)
            if (__ballot(mine && (rec(i).flags & kBadToken)) != 0) bad = true;
        const int32_t* y = a.tokens + int64_t(b) * K;
        for (int i = 0; i <= kb && !bad; ++i) {
            const bool bonus_row = i == kb;
            if constexpr (GREEDY) {
                // Merged argmax: larger value, else lower id (ranks in order).
                float v = mine ? rec(i).k_target : kNegInf;
                int g = mine && rec(i).argmax >= 0 ? rec(i).argmax : 0x7FFFFFFF;
                wave_argmax(v, g);
                if (!finite_shift(v)) {
                    bad = true;
                    break;
                }
                if (bonus_row || y[i] != g) {
                    d.acc = i;
                    d.token = g;
                    break;
                }
            } else {
                float kt = mine ? rec(i).k_target : kNegInf;
                double st = mine ? rec(i).s_target : 0.0;
                wave_merge_stats(kt, st);
                float kd = kNegInf;
                double sd = 0.0;
                if (!bonus_row) {
                    kd = mine ? rec(i).k_draft : kNegInf;
                    sd = mine ? rec(i).s_draft : 0.0;
                    wave_merge_stats(kd, sd);
                }
                if (!finite_shift(kt) || !usable_sum(st) ||
                    (!bonus_row && (!finite_shift(kd) || !usable_sum(sd)))) {
                    bad = true;  // a row the test reaches has no finite logit (or a NaN)
                    break;
                }
                d.kt = kt;
                d.kd = kd;
                d.st = st;
                d.sd = sd;
                if (bonus_row) {
                    d.acc = i;
                    break;
                }
                const uint64_t holders = __ballot(mine && (rec(i).flags & kHoldsY));
                if (holders == 0) {
                    bad = true;  // the slices do not cover the proposal's id
                    break;
                }
                const int h = __builtin_ctzll(holders);
                const float ty = readlane_f32(rec(i).t_y, h), dy = readlane_f32(rec(i).d_y, h);
                // Acceptance test as the whole-row kernels: p(y)/q(y) = 2^e S_d/S_t.
                const double e = (double(ty) * a.c2d - double(kt)) - (double(dy) * a.c2d - double(kd));
                double ratio;
                if (!(e > -2000.0)) {
                    ratio = 0.0;
                } else if (e > 2000.0) {
                    ratio = __builtin_huge_val();
                } else {
                    const double n = floor(e);
                    ratio = __builtin_ldexp(double(exp2_fast(float(e - n))), int(n)) * (sd / st);
                }
                if (!(double(a.u_accept[int64_t(b) * K + i]) < ratio)) {
                    d.acc = i;
                    break;
                }
            }
        }
        if (bad) d.acc = -1;
        if (lane == 0) s_dec = d;
    }
    __syncthreads();
    const Decision d = s_dec;

    uint64_t z = 0, zp = 0;
    if (!GREEDY && d.acc >= 0) {
        const bool p_only = d.acc == kb;
        const char* trow = static_cast<const char*>(a.target) + (int64_t(b) * (K + 1) + d.acc) * int64_t(Vs) * Fmt::kBytes;
        const char* drow = static_cast<const char*>(a.draft) + (int64_t(b) * K + d.acc) * int64_t(Vs) * Fmt::kBytes;
        chunk_t tv[CPT], dv[CPT];
        load_row<Fmt, W, CPT, VEC>(tv, trow, Vs);
        if (!p_only) load_row<Fmt, W, CPT, VEC>(dv, drow, Vs);
        const SliceMass<Fmt> mass{a.c2, d.kt, d.kd, p_only ? 0.0f : float(d.st / d.sd), p_only};
        const SliceMass<Fmt> pmass{a.c2, d.kt, d.kd, 0.0f, true};
#pragma unroll
        for (int n = 0; n < CPT; ++n) {
            float s = 0.0f, sp = 0.0f;
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                s = s + mass(tv[n], dv[n], e);
                if (!p_only) sp = sp + pmass(tv[n], dv[n], e);
            }
            z += mass_to_fixed<kFixedShift>(s);
            if (!p_only) zp += mass_to_fixed<kFixedShift>(sp);
        }
        if (p_only) zp = z;
        z = wave_sum(z);
        zp = wave_sum(zp);
        if (lane == 0) {
            s_z[0][wid] = z;
            s_z[1][wid] = zp;
        }
        __syncthreads();
        z = zp = 0;
        for (int w = 0; w < NW; ++w) {
            z += s_z[0][w];
            zp += s_z[1][w];
        }
    }
    if (tid == 0) {
        osd_shard_mass r = {};
        r.z = z;
        r.z_p = zp;
        r.s_target = d.st;
        r.s_draft = d.sd;
        r.k_target = d.kt;
        r.k_draft = d.kd;
        r.accepted = d.acc;
        r.token = GREEDY ? d.token : -1;
        *out = r;
    }
}

// ---------------------------------------------------------------------------
// Phase 3: place u*Z, draw on the rank that holds it, write the outputs.
// ---------------------------------------------------------------------------
struct DrawArgs {
    const void* target;
    const void* draft;
    int B, K, Vs, v_begin, G, shard;
    const int32_t* tokens;
    const int32_t* draft_len;
    const float* u_resample;
    float c2;
    const osd_shard_mass* mass_all;
    int32_t* accepted_len;
    int32_t* out_tokens;
    uint8_t* reject_mask;
};

struct Placement {
    int acc;        // a_b, or -1
    int token;      // greedy token, or -1
    int draw;       // 1: this rank draws
    int p_only;
    long long c;    // the point inside this rank's slice
};

template <typename Fmt, int W, int CPT, bool VEC, bool GREEDY>
__global__ __launch_bounds__(W, 4) void shard_draw_kernel(DrawArgs a) {
    constexpr int EPC = Fmt::kPerChunk;
    __shared__ Placement s_pl;
    __shared__ int s_tok;
    __shared__ unsigned long long s_tot[CPT * (W / kWave)];
    __shared__ DrawShared s_draw;
    __shared__ chunk_t s_stage[2 * CPT * kWave];

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int B = a.B, K = a.K, Vs = a.Vs, G = a.G;
    const int b = blockIdx.x;
    const int kb = draft_len_of(a.draft_len, b, K);
    const osd_shard_mass& own = a.mass_all[int64_t(a.shard) * B + b];

    if (wid == 0) {
        Placement pl;
        pl.acc = (kb < 1 || kb > K) ? -1 : own.accepted;
        pl.token = -1;
        pl.draw = 0;
        pl.p_only = 0;
        pl.c = 0;
        if (pl.acc >= 0) {
            if constexpr (GREEDY) {
                pl.token = own.token;
            } else {
                const bool mine = lane < G;
                const osd_shard_mass& m = a.mass_all[int64_t(mine ? lane : 0) * B + b];
                uint64_t zl = mine ? m.z : 0;
                uint64_t Z = wave_sum(zl);
                if (Z == 0) {
                    // No residual mass anywhere after rounding: draw from p.
                    zl = mine ? m.z_p : 0;
                    Z = wave_sum(zl);
                    pl.p_only = 1;
                }
                if (Z == 0) {
                    pl.acc = -1;  // no mass anywhere: the row has no finite logit
                } else {
                    uint64_t c = static_cast<uint64_t>(double(a.u_resample[b]) * double(Z));
                    if (c >= Z) c = Z - 1;
                    const uint64_t incl = wave_inclusive_scan(zl);
                    const uint64_t lo = readlane_u64(incl - zl, a.shard);
                    const uint64_t zs = readlane_u64(zl, a.shard);
                    if (zs > 0 && lo <= c && c - lo < zs) {
                        pl.draw = 1;
                        pl.c = static_cast<long long>(c - lo);
                    }
                }
            }
        }
        if (lane == 0) {
            s_pl = pl;
            s_tok = -1;
        }
    }
    __syncthreads();
    const Placement pl = s_pl;

    if (!GREEDY && pl.draw) {
        const int acc = pl.acc;
        const bool p_only = pl.p_only || acc == kb;
        const char* trow = static_cast<const char*>(a.target) + (int64_t(b) * (K + 1) + acc) * int64_t(Vs) * Fmt::kBytes;
        const char* drow = static_cast<const char*>(a.draft) + (int64_t(b) * K + acc) * int64_t(Vs) * Fmt::kBytes;
        chunk_t tv[CPT], dv[CPT];
        load_row<Fmt, W, CPT, VEC>(tv, trow, Vs);
        if (!p_only) {
            load_row<Fmt, W, CPT, VEC>(dv, drow, Vs);
        } else {
#pragma unroll
            for (int n = 0; n < CPT; ++n) dv[n] = pad_chunk<Fmt>();
        }
        const SliceMass<Fmt> mass{a.c2, own.k_target, own.k_draft,
                                  p_only ? 0.0f : float(own.s_target / own.s_draft), p_only};
        bool z_zero = false;
        const int t = draw_inverse_cdf<kFixedShift, W, CPT, EPC>(tv, dv, mass, 0.0f, s_tot, &s_draw, s_stage,
                                                                 &z_zero, pl.c);
        if (t >= 0) s_tok = a.v_begin + t;
        __syncthreads();
    }

    if (wid == 0) {
        const int acc = pl.acc;
        const int extra = GREEDY ? pl.token : (pl.draw ? s_tok : -1);
        const int32_t* y = a.tokens + int64_t(b) * K;
        for (int j = lane; j <= K; j += kWave) {
            int32_t o = -1;
            if (acc >= 0) o = j < acc ? y[j] : (j == acc ? extra : -1);
            a.out_tokens[int64_t(b) * (K + 1) + j] = o;
            if (a.reject_mask && j < K) a.reject_mask[int64_t(b) * K + j] = (acc >= 0 && j == acc && acc < kb) ? 1 : 0;
        }
        if (lane == 0) a.accepted_len[b] = acc;
    }
}

template <typename Fmt, int W, int CPT, bool VEC>
hipError_t launch_tile(const ShardLaunch& L) {
    const bool greedy = L.temperature == 0.0f;
    const float c2 = greedy ? 0.0f : float(1.4426950408889634 / double(L.temperature));
    const dim3 block(W);
    hipError_t e;
    if (L.phase == 1) {
        StatsArgs a{L.target, L.draft, L.B, L.K, L.Vs, L.v_begin, L.V, L.tokens, L.draft_len, c2, L.stats};
        const dim3 grid(unsigned(L.B) * unsigned(L.K + 1));
        if (greedy)
            e = launch_kernel(&shard_stats_kernel<Fmt, W, CPT, VEC, true>, grid, block, 0, L.stream, a);
        else
            e = launch_kernel(&shard_stats_kernel<Fmt, W, CPT, VEC, false>, grid, block, 0, L.stream, a);
    } else if (L.phase == 2) {
        MassArgs a{L.target, L.draft, L.B, L.K, L.Vs, L.G, L.tokens, L.draft_len, L.u_accept, c2, double(c2),
                   L.stats_in, L.mass};
        const size_t lds = size_t(L.G) * size_t(L.K + 1) * sizeof(osd_shard_row_stats);
        if (greedy)
            e = launch_kernel(&shard_mass_kernel<Fmt, W, CPT, VEC, true>, dim3(L.B), block, lds, L.stream, a);
        else
            e = launch_kernel(&shard_mass_kernel<Fmt, W, CPT, VEC, false>, dim3(L.B), block, lds, L.stream, a);
    } else {
        DrawArgs a{L.target, L.draft, L.B, L.K, L.Vs, L.v_begin, L.G, L.shard, L.tokens, L.draft_len,
                   L.u_resample, c2, L.mass_in, L.accepted_len, L.out_tokens, L.reject_mask};
        if (greedy)
            e = launch_kernel(&shard_draw_kernel<Fmt, W, CPT, VEC, true>, dim3(L.B), block, 0, L.stream, a);
        else
            e = launch_kernel(&shard_draw_kernel<Fmt, W, CPT, VEC, false>, dim3(L.B), block, 0, L.stream, a);
    }
    return e;
}

template <typename Fmt, bool VEC>
hipError_t launch_fmt(const ShardLaunch& L) {
    RowTile t;
    if (!pick_tile(L.Vs, Fmt::kPerChunk, &t)) return hipErrorInvalidValue;
    switch (t.W * 100 + t.CPT) {
        case 25601: return launch_tile<Fmt, 256, 1, VEC>(L);
        case 25602: return launch_tile<Fmt, 256, 2, VEC>(L);
        case 25604: return launch_tile<Fmt, 256, 4, VEC>(L);
        case 51204: return launch_tile<Fmt, 512, 4, VEC>(L);
        case 51208: return launch_tile<Fmt, 512, 8, VEC>(L);
        case 102408: return launch_tile<Fmt, 1024, 8, VEC>(L);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_verify_shard(const ShardLaunch& L) {
    if (L.dtype == 1) return L.vec ? launch_fmt<BF16, true>(L) : launch_fmt<BF16, false>(L);
    return L.vec ? launch_fmt<F32, true>(L) : launch_fmt<F32, false>(L);
}

}  // namespace osd
