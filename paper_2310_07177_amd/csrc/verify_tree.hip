// verify_tree.hip -- multi-candidate (tree) verification on gfx950.
//
// The paper applies online updates to Medusa, whose heads propose several
// candidate tokens per position arranged in a tree (Section 5, "OSD and
// Medusa", Table 4); it gives no verification rule for such a tree.  The
// rule here keeps the exactness of Appendix A.1 (the emitted tokens follow
// the target): a node's children are candidates drawn independently from
// the draft distribution q at the node and are tested one after another;
// candidate c is accepted when u_c < R(y_c)/q(y_c), where R is p at the first
// test and, after each rejection, the normalised residual max(0, R - q) of
// Eq. 5.  The walk continues at the first accepted child; where every child
// is rejected, one token is drawn from the last residual, and at a node
// without children one token is drawn from p (the bonus token).  At T == 0
// the first child whose token is the target argmax is accepted and the
// argmax is emitted where the walk stops.
//
// Work layout.  One workgroup per (sequence b, node n), numbered node-major
// (every root first).  Each node's outcome depends only on its own row pair
// and its children's tokens and uniforms, so every node is decided in
// parallel from one read of its rows: the workgroup reads the target and
// draft rows into registers, turns them into the masses p S_t and q S_t
// (cached as floats), tests the children in order -- each rejection
// replaces the cached p by max(0, R - q) and sums it (one workgroup
// reduction) -- and, if no child is accepted, draws from the last residual
// (or from p at a leaf) by the exact fixed-point inverse CDF.  It publishes
// one record (accepted child, or drawn token); the last of the N workgroups
// of a sequence to arrive walks the records from the root and writes the
// outputs.  Nodes off the accepted path are computed too: the price of not
// waiting for the path.
#include "osd_device.hpp"
#include "osd_internal.hpp"
#include "row_draw.hpp"

namespace osd {
namespace {

// Record word: state in bits 31..28, payload (child node or token) in 27..0.
enum : uint32_t { kNodeAccept = 1, kNodeDraw = 2, kNodeBad = 3 };
__device__ inline uint32_t node_rec(uint32_t s, uint32_t v) { return (s << 28) | (v & 0x0FFFFFFFu); }

// Masses are in units of S_t (the target row's sum of exponentials): every
// residual is rescaled to total S_t <= V <= 2^17, so no element or sum
// exceeds 2^17 and 2^-44 fixed point cannot overflow.
constexpr int kFixedShift = 44;

struct TreeArgs {
    const void* target;  // [B, N, V]
    const void* draft;   // [B, N, V]
    int B, N, V;
    const int32_t* parent;       // [B, N]
    const int32_t* node_tokens;  // [B, N]
    const float* u_accept;       // [B, N]
    const float* u_resample;     // [B]
    float c2;
    int32_t* accepted_len;  // [B]
    int32_t* out_tokens;    // [B, N]
    int32_t* path_nodes;    // [B, N] or null
    uint32_t* records;      // [B, N]   zero between calls
    uint32_t* counters;     // [B]      zero between calls
};

// The last of the N node workgroups of sequence b: validate the tree, walk
// the records from the root, write the outputs, clear the records and the
// counter.  All 64 lanes of one wave (lane j: node j; N <= 64).
__device__ void finish_tree(const TreeArgs& a, int b) {
    const int lane = threadIdx.x & (kWave - 1), N = a.N;
    const bool mine = lane < N;
    const uint32_t r = mine ? take_u32(&a.records[int64_t(b) * N + lane]) : 0u;
    const int par = mine ? a.parent[int64_t(b) * N + lane] : 0;
    const int tok = mine ? a.node_tokens[int64_t(b) * N + lane] : 0;
    bool bad = __ballot(mine && lane > 0 && (par < 0 || par >= lane || tok < 0 || tok >= a.V)) != 0;
    int v = 0, len = 0, extra = -1, at = -1;  // at: this lane's path node
    for (int step = 0; step < N && !bad; ++step) {
        const uint32_t rv = uint32_t(__shfl(int(r), v, kWave));
        const uint32_t st = rv >> 28, pay = rv & 0x0FFFFFFFu;
        if (st == kNodeAccept && int(pay) > v && int(pay) < N) {
            if (lane == len) at = int(pay);
            ++len;
            v = int(pay);
        } else if (st == kNodeDraw) {
            extra = int(pay);
            break;
        } else {
            bad = true;
        }
    }
    if (extra < 0) bad = true;
    const int ptok = __shfl(tok, at >= 0 ? at : 0, kWave);
    if (mine) {
        int32_t o = -1;
        if (!bad) o = lane < len ? ptok : (lane == len ? extra : -1);
        a.out_tokens[int64_t(b) * N + lane] = o;
        if (a.path_nodes) a.path_nodes[int64_t(b) * N + lane] = (!bad && lane < len) ? at : -1;
    }
    if (lane == 0) {
        a.accepted_len[b] = bad ? -1 : len;
        take_u32(&a.counters[b]);
    }
}

// Wave 0 of a node workgroup: publish the node's record; the last of the
// sequence's N workgroups writes the outputs.
__device__ void publish_node(const TreeArgs& a, int b, int n, uint32_t record) {
    const int lane = threadIdx.x & (kWave - 1);
    uint32_t prev = 0;
    if (lane == 0) {
        publish_u32(&a.records[int64_t(b) * a.N + n], record);
        prev = arrive(&a.counters[b]);
    }
    prev = uint32_t(__shfl(int(prev), 0, kWave));
    if (prev == uint32_t(a.N - 1)) finish_tree(a, b);
}

// Floats of a cached row: element e of round r lives in lane (e & 3) of
// chunk lo[r] (e < 4) or hi[r] (e >= 4).
template <int EPC>
__device__ inline float cache_get(const chunk_t& lo, const chunk_t& hi, int e) {
    const chunk_t& c = (EPC == 8 && e >= 4) ? hi : lo;
    const int k = e & 3;
    return __uint_as_float(k == 0 ? c.x : k == 1 ? c.y : k == 2 ? c.z : c.w);
}
__device__ inline void cache_set(chunk_t& lo, chunk_t& hi, int e, float v, int epc) {
    chunk_t& c = (epc == 8 && e >= 4) ? hi : lo;
    const uint32_t u = __float_as_uint(v);
    switch (e & 3) {
        case 0: c.x = u; break;
        case 1: c.y = u; break;
        case 2: c.z = u; break;
        default: c.w = u; break;
    }
}

template <typename Fmt, int W, int CPT, bool VEC, bool GREEDY>
__global__ __launch_bounds__(W, min_waves_per_simd(W, CPT)) void tree_node_kernel(TreeArgs a) {
    constexpr int NW = W / kWave;
    constexpr int EPC = Fmt::kPerChunk;
    __shared__ float s_max[2][NW];
    __shared__ double s_sum[2][NW];
    __shared__ int s_idx[NW];
    __shared__ unsigned long long s_kids;
    __shared__ int s_ktok[kWave];
    __shared__ float s_y[2];
    __shared__ double s_z[NW];
    __shared__ unsigned long long s_tot[CPT * NW];
    __shared__ DrawShared s_draw;
    __shared__ int s_tok;
    __shared__ chunk_t s_stage[GREEDY ? 1 : 2 * CPT * kWave];

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int B = a.B, N = a.N, V = a.V;
    const int n = blockIdx.x / B, b = blockIdx.x - n * B;

    // The node's children (ascending node id) and their tokens.
    if (wid == 0) {
        const bool in = lane < N;
        const int par = in ? a.parent[int64_t(b) * N + lane] : -1;
        const int tok = in ? a.node_tokens[int64_t(b) * N + lane] : -1;
        const uint64_t kids = __ballot(in && lane > n && par == n);
        // A child token outside the vocabulary invalidates the tree (the
        // last workgroup checks it); it is never used to index a row.
        const bool tok_bad = __ballot(in && lane > n && par == n && (tok < 0 || tok >= V)) != 0;
        if (lane == 0) s_kids = tok_bad ? ~0ull : kids;
        s_ktok[lane] = tok;
        if (tid == 0) s_tok = -1;
    }
    __syncthreads();
    const uint64_t kids = s_kids;
    if (kids == ~0ull) {
        if (wid == 0) publish_node(a, b, n, node_rec(kNodeBad, 0));
        return;
    }
    const bool leaf = kids == 0;
    const char* trow = static_cast<const char*>(a.target) + (int64_t(b) * N + n) * int64_t(V) * Fmt::kBytes;
    const char* drow = (GREEDY || leaf) ? trow
                                        : static_cast<const char*>(a.draft) + (int64_t(b) * N + n) * int64_t(V) * Fmt::kBytes;
    const int nchunks = (V + EPC - 1) / EPC;
    chunk_t tv[CPT], dv[CPT];
    // A leaf (and greedy verification) reads the target row alone.
    const bool pair = !GREEDY && !leaf;
    if constexpr (VEC) {
        if (pair) {
            load_rows_interleaved<W, CPT>(tv, dv, trow, drow, nchunks);
        } else {
            load_row_clamped<W, CPT>(tv, trow, nchunks);
#pragma unroll
            for (int r = 0; r < CPT; ++r) dv[r] = pad_chunk<Fmt>();
        }
    } else {
        load_row<Fmt, W, CPT, VEC>(tv, trow, V);
        if (pair)
            load_row<Fmt, W, CPT, VEC>(dv, drow, V);
        else
#pragma unroll
            for (int r = 0; r < CPT; ++r) dv[r] = pad_chunk<Fmt>();
    }

    if constexpr (GREEDY) {
        if constexpr (VEC) pad_row_tail<Fmt, W, CPT>(tv, nchunks);
        (void)drow;
        float best = kNegInf;
        int bi = 0x7FFFFFFF;
#pragma unroll
        for (int r = 0; r < CPT; ++r)
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float x = Fmt::get(tv[r], e);
                if (x > best) {
                    best = x;
                    bi = (r * W + tid) * EPC + e;
                }
            }
        wave_argmax(best, bi);
        if (lane == 0) {
            s_max[0][wid] = best;
            s_idx[wid] = bi;
        }
        __syncthreads();
        if (wid == 0) {
            float bv = s_max[0][0];
            int g = s_idx[0];
            for (int w = 1; w < NW; ++w)
                if (s_max[0][w] > bv || (s_max[0][w] == bv && s_idx[w] < g)) {
                    bv = s_max[0][w];
                    g = s_idx[w];
                }
            uint32_t rec;
            if (!(bv > kNegInf) || bv == -kNegInf) {
                rec = node_rec(kNodeBad, 0);
            } else {
                // the first child whose token is the argmax
                const uint64_t hit = __ballot(((kids >> lane) & 1ull) && s_ktok[lane] == g);
                rec = hit ? node_rec(kNodeAccept, uint32_t(__builtin_ctzll(hit))) : node_rec(kNodeDraw, uint32_t(g));
            }
            publish_node(a, b, n, rec);
        }
        return;
    } else {
        const float c2 = a.c2;
        float Kt = kNegInf, Kd = kNegInf;
        {
            float st = 0.0f, sd = 0.0f;
            if constexpr (VEC) {
                row_stats2_tail<Fmt, W, CPT>(tv, dv, nchunks, c2, !leaf, Kt, st, Kd, sd);
                pad_row_tail<Fmt, W, CPT>(tv, nchunks);
                pad_row_tail<Fmt, W, CPT>(dv, nchunks);
            } else {
                row_stats<Fmt, CPT>(tv, c2, Kt, st);
                if (!leaf) row_stats<Fmt, CPT>(dv, c2, Kd, sd);
            }
            double dt = st, dd = sd;
            wave_merge_stats(Kt, dt);
            wave_merge_stats(Kd, dd);
            if (lane == 0) {
                s_max[0][wid] = Kt;
                s_max[1][wid] = Kd;
                s_sum[0][wid] = dt;
                s_sum[1][wid] = dd;
            }
        }
        __syncthreads();
        Kt = s_max[0][0];
        Kd = s_max[1][0];
#pragma unroll
        for (int w = 1; w < NW; ++w) {
            Kt = fmaxf(Kt, s_max[0][w]);
            Kd = fmaxf(Kd, s_max[1][w]);
        }
        double St = 0.0, Sd = 0.0;
        for (int w = 0; w < NW; ++w) {
            St += rescale(s_sum[0][w], s_max[0][w], Kt);
            Sd += rescale(s_sum[1][w], s_max[1][w], Kd);
        }
        const bool bad = !(Kt > kNegInf && Kt < -kNegInf) || !usable_sum(St) ||
                         (!leaf && (!(Kd > kNegInf && Kd < -kNegInf) || !usable_sum(Sd)));
        if (bad) {
            if (wid == 0) publish_node(a, b, n, node_rec(kNodeBad, 0));
            return;
        }
        // The cache: P (p S_t, later the residuals) and Q (q S_t), as floats.
        // The raw target chunks are kept for the fallback draw from p.
        const float rho = leaf ? 0.0f : float(St / Sd);
        chunk_t plo[CPT], phi[CPT], qlo[CPT], qhi[CPT];
#pragma unroll
        for (int r = 0; r < CPT; ++r) {
            plo[r] = phi[r] = qlo[r] = qhi[r] = chunk_t{0u, 0u, 0u, 0u};
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float p = exp2_fast(__builtin_fmaf(Fmt::get(tv[r], e), c2, -Kt));
                const float q = leaf ? 0.0f : exp2_fast(__builtin_fmaf(Fmt::get(dv[r], e), c2, -Kd)) * rho;
                cache_set(plo[r], phi[r], e, p, EPC);
                cache_set(qlo[r], qhi[r], e, q, EPC);
            }
        }
        // Test the children in order.  The cached P is the residual
        // before scaling; `scale` makes it total S_t (the normalised
        // distribution the next child is tested against, in S_t units).
        float scale = 1.0f;
        uint32_t rec = 0u;
        uint64_t left = kids;
        while (left) {
            const int c = __builtin_ctzll(left);
            left &= left - 1;
            const int y = s_ktok[c];
            // the holder of y posts R(y) and Q(y)
            {
                const int ch = y / EPC, ey = y - ch * EPC;
                const int rr = ch / W, th = ch - rr * W;
#pragma unroll
                for (int r = 0; r < CPT; ++r)
                    if (r == rr && tid == th) {
                        s_y[0] = cache_get<EPC>(plo[r], phi[r], ey) * scale;
                        s_y[1] = cache_get<EPC>(qlo[r], qhi[r], ey);
                    }
            }
            __syncthreads();
            const double ry = double(s_y[0]), qy = double(s_y[1]);
            const double ratio = qy > 0.0 ? ry / qy : (ry > 0.0 ? __builtin_huge_val() : 0.0);
            const double u = a.u_accept[int64_t(b) * N + c];
            if (u < ratio) {
                rec = node_rec(kNodeAccept, uint32_t(c));
                break;
            }
            // Rejected: P <- max(0, scale P - Q), summed over the row.
            float part = 0.0f;
#pragma unroll
            for (int r = 0; r < CPT; ++r) {
                float s = 0.0f;
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    const float v = fmaxf(__builtin_fmaf(cache_get<EPC>(plo[r], phi[r], e), scale,
                                                         -cache_get<EPC>(qlo[r], qhi[r], e)),
                                          0.0f);
                    cache_set(plo[r], phi[r], e, v, EPC);
                    s = s + v;
                }
                part = part + s;
            }
            double z = wave_sum(double(part));
            __syncthreads();  // s_y and s_z are read before they are rewritten
            if (lane == 0) s_z[wid] = z;
            __syncthreads();
            z = 0.0;
            for (int w = 0; w < NW; ++w) z += s_z[w];
            // No residual mass after rounding (R = q to fp32 accuracy): the
            // cache is left at zero and the draw below falls back to p.
            scale = z > 0.0 ? float(St / z) : 1.0f;
        }
        if (rec == 0u) {
            // Every child rejected (or a leaf): the token from the cached
            // residual (from p at a leaf), or from p should it have no mass.
            bool use_p = leaf;
            for (int attempt = 0; attempt < 2; ++attempt) {
                bool z_zero = false;
                int tok;
                if (use_p) {
                    float kt = Kt;
                    asm volatile("" : "+v"(kt));
                    auto mass = [=](const chunk_t& tc, const chunk_t&, int e) -> float {
                        return exp2_fast(__builtin_fmaf(Fmt::get(tc, e), c2, -kt));
                    };
                    tok = draw_inverse_cdf<kFixedShift, W, CPT, EPC>(tv, dv, mass, a.u_resample[b], s_tot,
                                                                    &s_draw, s_stage, &z_zero);
                } else {
                    auto mass = [](const chunk_t& lo, const chunk_t& hi, int e) -> float {
                        return cache_get<EPC>(lo, hi, e);
                    };
                    tok = draw_inverse_cdf<kFixedShift, W, CPT, EPC>(plo, phi, mass, a.u_resample[b], s_tot,
                                                                    &s_draw, s_stage, &z_zero);
                }
                if (tok >= 0) s_tok = tok;
                if (!z_zero || use_p) break;
                use_p = true;
            }
            __syncthreads();
            const int t = s_tok;
            rec = (t >= 0 && t < V) ? node_rec(kNodeDraw, uint32_t(t)) : node_rec(kNodeBad, 0);
        }
        if (wid == 0) publish_node(a, b, n, rec);
    }
}

template <typename Fmt, int W, int CPT>
hipError_t launch_tile(const TreeLaunch& L, const TreeArgs& a) {
    const dim3 grid(unsigned(L.B) * unsigned(L.N)), block(W);
    const bool greedy = L.temperature == 0.0f;
    hipError_t e;
    if (L.vec) {
        if (greedy)
            e = launch_kernel(&tree_node_kernel<Fmt, W, CPT, true, true>, grid, block, 0, L.stream, a);
        else
            e = launch_kernel(&tree_node_kernel<Fmt, W, CPT, true, false>, grid, block, 0, L.stream, a);
    } else {
        if (greedy)
            e = launch_kernel(&tree_node_kernel<Fmt, W, CPT, false, true>, grid, block, 0, L.stream, a);
        else
            e = launch_kernel(&tree_node_kernel<Fmt, W, CPT, false, false>, grid, block, 0, L.stream, a);
    }
    return e;
}

template <typename Fmt>
hipError_t launch_fmt(const TreeLaunch& L, const TreeArgs& a) {
    RowTile t;
    if (!pick_tree_tile(L.V, Fmt::kPerChunk, &t)) return hipErrorInvalidValue;
    switch (t.W * 100 + t.CPT) {
        case 25601: return launch_tile<Fmt, 256, 1>(L, a);
        case 25602: return launch_tile<Fmt, 256, 2>(L, a);
        case 51202: return launch_tile<Fmt, 512, 2>(L, a);
        case 102402: return launch_tile<Fmt, 1024, 2>(L, a);
        case 102404: return launch_tile<Fmt, 1024, 4>(L, a);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

// Tiles of the tree kernel: at most 4 chunks per thread, since each element
// keeps two cached floats besides the raw chunks (up to 32768 bf16 or 16384
// fp32 logits per row).
bool pick_tree_tile(int V, int per_chunk, RowTile* t) {
    static const RowTile tiles[] = {{256, 1}, {256, 2}, {512, 2}, {1024, 2}, {1024, 4}};
    for (const RowTile& c : tiles)
        if (int64_t(V) <= int64_t(c.W) * c.CPT * per_chunk) {
            *t = c;
            return true;
        }
    return false;
}

hipError_t launch_verify_tree(const TreeLaunch& L) {
    TreeArgs a{};
    a.target = L.target;
    a.draft = L.draft;
    a.B = L.B;
    a.N = L.N;
    a.V = L.V;
    a.parent = L.parent;
    a.node_tokens = L.node_tokens;
    a.u_accept = L.u_accept;
    a.u_resample = L.u_resample;
    a.c2 = L.temperature > 0.0f ? float(1.4426950408889634 / double(L.temperature)) : 0.0f;
    a.accepted_len = L.accepted_len;
    a.out_tokens = L.out_tokens;
    a.path_nodes = L.path_nodes;
    a.records = L.records;
    a.counters = L.counters;
    return L.dtype == 1 ? launch_fmt<BF16>(L, a) : launch_fmt<F32>(L, a);
}

}  // namespace osd
