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
//
// Rows with 16-byte alignment at T > 0 take the streaming layout instead
// (tree_stream_kernel, below): about one workgroup per CU walks its node
// items while the next item's rows are in flight.
#include "osd_device.hpp"
#include "osd_internal.hpp"
#include "row_draw.hpp"
#include "stream_device.hpp"
#include "distill_common.hpp"
#include "cache_draw.hpp"

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
    // streaming layout only
    int G;               // workgroups in the grid
    int nitems;          // B * N
    int nchunks;         // 16-byte chunks per row
    uint32_t row_bytes;  // bytes per row
};

// The last of the N node workgroups of sequence b: validate the tree, walk
// the records from the root, write the outputs, clear the records and the
// counter.  All 64 lanes of one wave (lane j: node j; N <= 64).
__device__ void finish_tree(const TreeArgs& a, int b) {
    const int lane = opaque_tid() & (kWave - 1), N = a.N;  // (recomputed here: nothing lane-derived is kept across a caller's loop)
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

// ---------------------------------------------------------------------------
// Streaming layout (16-byte rows, T > 0).  About one workgroup per CU walks
// the node items j = g, g + G, ... (item j is node j / B of sequence j % B,
// so the roots come first).  While an item is computed the next item's rows
// are in flight: each register chunk is reloaded with the same chunk of the
// next item as soon as the statistics pass has consumed it, so the loads of
// one item overlap the arithmetic of the one before.  Per item the cache
// holds 2^(t c2 - k_t) for every target element (LDS, thread-private float4
// slots) and 2^(d c2 - k_d) for every draft element (registers), k being the
// thread's shifts over its chunks (every cached value is at most 1); after
// the workgroup merge of the normalisers p and q are these values times one
// per-thread scale each.  The children are tested against R = p and then
// against the residuals, each of the form max(0, p - s q) / Z with two
// scalars s, Z, so a rejection costs one sum over the cache and nothing is
// rewritten.  Where no child is accepted, the token is drawn from the last
// residual over the cache (exact fixed point, as the fused kernel draws), or
// from p should that residual have no mass after rounding.  Each item posts
// its record and arrives at its sequence's counter without waiting for
// either; the arrival's count is read at the start of the next item (it
// returns after that item's rows, which the statistics wait for anyway), and
// the item whose arrival is its sequence's last writes the outputs
// (finish_tree_polled, which waits for records still on their way).  No item
// waits for another.
constexpr int kTreeRecordPolls = 4096;
constexpr int kMaxTreeItems = 128;  // items staged per workgroup (the grid grows beyond)

__device__ inline float f4_get(const f32x4_t& v, int i) { return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w; }

__device__ inline uint64_t uniform_u64(uint64_t v) {
    const uint32_t lo = uint32_t(__builtin_amdgcn_readfirstlane(int(uint32_t(v))));
    const uint32_t hi = uint32_t(__builtin_amdgcn_readfirstlane(int(uint32_t(v >> 32))));
    return (uint64_t(hi) << 32) | lo;
}

// finish_tree for records posted without a wait before the arrival: each
// lane first waits (bounded) until its node's record is there.  A record
// still missing after the polls makes the tree invalid.
__device__ void finish_tree_polled(const TreeArgs& a, int b) {
    const int lane = opaque_tid() & (kWave - 1);
    bool missing = false;
    if (lane < a.N) {
        const uint32_t* rp = &a.records[int64_t(b) * a.N + lane];
        int p = 0;
        while (load_relaxed(rp) == 0u && p < kTreeRecordPolls) {
            __builtin_amdgcn_s_sleep(2);
            ++p;
        }
        missing = p >= kTreeRecordPolls;
    }
    if (__ballot(missing) != 0) {
        // (not reached in practice: every record is posted before its arrival)
        if (lane < a.N) {
            take_u32(&a.records[int64_t(b) * a.N + lane]);
            a.out_tokens[int64_t(b) * a.N + lane] = -1;
            if (a.path_nodes) a.path_nodes[int64_t(b) * a.N + lane] = -1;
        }
        if (lane == 0) {
            a.accepted_len[b] = -1;
            take_u32(&a.counters[b]);
        }
        return;
    }
    finish_tree(a, b);
}

template <typename Fmt, int W, int CPT>
__global__ __launch_bounds__(W, 1) void tree_stream_kernel(TreeArgs a) {
    constexpr int NW = W / kWave, EPC = Fmt::kPerChunk, NG = EPC / 4;
    __shared__ f32x4_t s_c0[CPT * NG * W];
    __shared__ uint64_t s_kids[kMaxTreeItems];
    __shared__ float s_k[2 * NW];
    __shared__ double s_s[2 * NW];
    __shared__ RowPair s_rp;
    // Per-item scratch written before the item's first barrier is
    // double-buffered by item parity: a wave can still be reading the
    // previous item's while another writes this one's.
    __shared__ int s_ktok[2][kWave];
    __shared__ float s_ku[2][kWave];
    __shared__ float s_y[2];
    __shared__ double s_z[NW];
    __shared__ double s_cell[CPT * NW];
    __shared__ double s_dz;
    __shared__ int s_tok;
    const LdsCache<W, EPC> lc{s_c0};

    // Every argument word, requested together on entry.
    asm volatile("" ::"s"(a.target), "s"(a.draft), "s"(a.B), "s"(a.N), "s"(a.V), "s"(a.parent), "s"(a.node_tokens),
                 "s"(a.u_accept), "s"(a.u_resample), "s"(a.c2));
    asm volatile("" ::"s"(a.accepted_len), "s"(a.out_tokens), "s"(a.path_nodes), "s"(a.records), "s"(a.counters),
                 "s"(a.G), "s"(a.nitems), "s"(a.nchunks), "s"(a.row_bytes));
    const int tid = threadIdx.x;
    const int g = blockIdx.x, G = a.G, B = a.B, N = a.N;
    const float c2 = a.c2;
    const bool last_ok = (CPT - 1) * W + tid < a.nchunks;
    const int nk = g < a.nitems ? (a.nitems - 1 - g) / G + 1 : 0;  // <= kMaxTreeItems (launch)
    const char* const tbase = static_cast<const char*>(a.target);
    const char* const dbase = static_cast<const char*>(a.draft);

    chunk_t rt[CPT], rs[CPT];
    float c1[CPT][EPC];
    // The first item's rows, before its children are known (a leaf's draft
    // row is read then too; it is in bounds either way).
    {
        const int n = g / B, b = g - n * B;
        const bool on = nk > 0;
        const int64_t row = int64_t(b) * N + n;
        const rsrc_t tr = make_rsrc(on ? tbase + row * a.row_bytes : tbase, on ? a.row_bytes : 0u);
        const rsrc_t dr = make_rsrc(on ? dbase + row * a.row_bytes : tbase, on ? a.row_bytes : 0u);
#pragma unroll
        for (int r = 0; r < CPT; ++r) {
            rt[r] = load_chunk<W>(tr, r);
            rs[r] = load_chunk<W>(dr, r);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // The children of every item, staged once (wave w takes items w, w + NW,
    // ...): a bit mask of the node's children, ~0 when one of them carries a
    // token outside the vocabulary (the tree is then invalid; the last
    // workgroup of the sequence reports it).
    for (int k = opaque_tid() / kWave; k < nk; k += NW) {
        const int lane = opaque_tid() & (kWave - 1);
        const int j = g + k * G, n = j / B, b = j - n * B;
        const bool in = lane < N;
        const int par = in ? a.parent[int64_t(b) * N + lane] : -1;
        const int tok = in ? a.node_tokens[int64_t(b) * N + lane] : -1;
        const bool kid = in && lane > n && par == n;
        const uint64_t kids = __ballot(kid);
        const bool tok_bad = __ballot(kid && (tok < 0 || tok >= a.V)) != 0;
        if (lane == 0) s_kids[k] = tok_bad ? ~0ull : kids;
    }
    __syncthreads();

    // Wave 0's pending arrival (the previous item's): its sequence and the
    // number of earlier arrivals, read at the start of the next item.
    int pend_b = -1;
    uint32_t pend = 0u;
    for (int k = 0; k < nk; ++k) {
        const int j = g + k * G, n = j / B, b = j - n * B, par = k & 1;
        const uint64_t kids = uniform_u64(s_kids[k]);
        const bool bad_tree = kids == ~0ull, leaf = kids == 0ull, live = !bad_tree;
        // The next item's rows (its draft row only if it has children).
        const bool more = k + 1 < nk;
        const uint64_t kn = more ? uniform_u64(s_kids[k + 1]) : ~0ull;
        const bool nload = more && kn != ~0ull, ndraft = nload && kn != 0ull;
        const int jn = j + G, nn = jn / B, bn = jn - nn * B;
        const int64_t nrow = int64_t(bn) * N + nn;
        const rsrc_t ntr = make_rsrc(nload ? tbase + nrow * a.row_bytes : tbase, nload ? a.row_bytes : 0u);
        const rsrc_t nsr = make_rsrc(ndraft ? dbase + nrow * a.row_bytes : tbase, ndraft ? a.row_bytes : 0u);
        // Wave 0: the previous item's arrival (it returns after this item's
        // rows, which the statistics wait for anyway; it may complete that
        // sequence), then this item's candidate tokens and uniforms (lane c:
        // node c), requested now and used after the statistics.
        int ktok = -1;
        float ku = 0.0f;
        if (opaque_tid() < kWave) {
            if (pend_b >= 0 && uint32_t(__shfl(int(pend), 0, kWave)) == uint32_t(N - 1)) finish_tree_polled(a, pend_b);
            pend_b = -1;
            const int lane = opaque_tid();
            if (live && !leaf && lane < N) {
                ktok = a.node_tokens[int64_t(b) * N + lane];
                ku = a.u_accept[int64_t(b) * N + lane];
            }
        }
        const float ures = scalar_load(a.u_resample + b);

        // ---- statistics pass (and the cache), reloading each chunk with the
        // next item's ----
        float kc_t = 0.0f, kc_s = 0.0f;
        double S_t = 0.0, S_s = 0.0;
        if (live) {
            kc_t = shift_of_max(chunks_max<Fmt, CPT>(rt, !last_ok), c2);
            if (!leaf) kc_s = shift_of_max(chunks_max<Fmt, CPT>(rs, !last_ok), c2);
        }
#pragma unroll
        for (int r = 0; r < CPT; ++r) {
            if (live) {
                chunk_t xt = rt[r], xs = rs[r];
                if (r == CPT - 1 && !last_ok) {
                    xt = pad_chunk<Fmt>();
                    xs = pad_chunk<Fmt>();
                }
                float st = 0.0f, ss = 0.0f;
#pragma unroll
                for (int q4 = 0; q4 < NG; ++q4) {
                    float c0v[4];
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) {
                        const int e = 4 * q4 + jj;
                        const float et = exp2_fast(__builtin_fmaf(Fmt::get(xt, e), c2, -kc_t));
                        const float es = exp2_fast(__builtin_fmaf(Fmt::get(xs, e), c2, -kc_s));
                        st = e == 0 ? et : st + et;
                        ss = e == 0 ? es : ss + es;
                        c0v[jj] = et;
                        c1[r][e] = es;
                    }
                    lc.store(r, q4, f32x4_t{c0v[0], c0v[1], c0v[2], c0v[3]});
                }
                asm volatile("" : "+v"(st), "+v"(ss));
                S_t = r == 0 ? double(st) : S_t + double(st);
                S_s = r == 0 ? double(ss) : S_s + double(ss);
            }
            rt[r] = load_chunk<W>(ntr, r);
            rs[r] = load_chunk<W>(nsr, r);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (opaque_tid() < kWave) {
            s_ktok[par][opaque_tid()] = ktok;
            s_ku[par][opaque_tid()] = ku;
        }

        uint32_t rec = node_rec(kNodeBad, 0);
        if (!live) {
            __syncthreads();  // every item has a barrier (the live ones: the merge), so no wave runs two items ahead
        } else {
            const RowPair rp = merge_row_pair<NW>(kc_t, S_t, kc_s, S_s, s_k, s_s, &s_rp);
            const bool bad = !usable_sum(rp.st) || (!leaf && !usable_sum(rp.ss));
            if (!bad) {
                // p = e_t at, q = e_s as (the thread's scales, fp64 rounded once).
                const float at = float(__builtin_ldexp(rp.ist, int(fmaxf(kc_t - rp.kt, -2048.0f))));
                const float as = leaf ? 0.0f : float(__builtin_ldexp(rp.iss, int(fmaxf(kc_s - rp.ks, -2048.0f))));
                // The candidates in order.  R = max(0, p - s q) / Z: the first
                // test has s = 0, Z = 1, and a rejection takes s <- s + Z,
                // Z <- sum_j max(0, p_j - s q_j).  This is Eq. 5's residual of
                // the residual, unrolled: by induction max(0, R - q) / z =
                // max(0, p - (s + Z) q) / (Z z), and Z z is that sum.  So the
                // cache is never rewritten, and a rejection costs one sum.
                // Z = 0 (no residual mass after rounding) leaves R = 0: every
                // later candidate is rejected and the draw falls back to p.
                double s_c = 0.0, Z_c = 1.0;
                rec = 0u;
                uint64_t left = kids;
                while (left) {
                    const int c = __builtin_ctzll(left);
                    left &= left - 1;
                    const int y = __builtin_amdgcn_readfirstlane(s_ktok[par][c]);
                    {
                        // The holder of y posts R(y) and Q(y).
                        const int ch = y / EPC, ey = y - ch * EPC, rr = ch / W, th = ch - rr * W;
                        if (opaque_tid() == th) {
                            float ev = 0.0f;
#pragma unroll
                            for (int r = 0; r < CPT; ++r)
#pragma unroll
                                for (int e = 0; e < EPC; ++e)
                                    if (r == rr && e == ey) ev = c1[r][e];
                            const float pv = f4_get(lc.load(rr, ey >> 2), ey & 3) * at, qv = ev * as;
                            const float d = fmaxf(__builtin_fmaf(-float(s_c), qv, pv), 0.0f);
                            s_y[0] = Z_c > 0.0 ? float(double(d) / Z_c) : 0.0f;
                            s_y[1] = qv;
                        }
                    }
                    __syncthreads();
                    const double ry = double(s_y[0]), qy = double(s_y[1]);
                    const double ratio = qy > 0.0 ? ry / qy : (ry > 0.0 ? __builtin_huge_val() : 0.0);
                    const bool accept = __builtin_amdgcn_readfirstlane(double(s_ku[par][c]) < ratio ? 1 : 0) != 0;
                    if (accept) {
                        rec = node_rec(kNodeAccept, uint32_t(c));
                        break;
                    }
                    if (Z_c > 0.0) {
                        s_c += Z_c;
                        // p - s q = at (e_t - k e_s), summed where positive.
                        const float k = at > 0.0f ? float(s_c * double(as) / double(at)) : 0.0f;
                        float part = 0.0f;
#pragma unroll
                        for (int r = 0; r < CPT; ++r) {
                            float sr = 0.0f;
#pragma unroll
                            for (int q4 = 0; q4 < NG; ++q4) {
                                const f32x4_t v = lc.load(r, q4);
                                const float c0v[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                                for (int jj = 0; jj < 4; ++jj)
                                    sr = sr + fmaxf(__builtin_fmaf(-k, c1[r][4 * q4 + jj], c0v[jj]), 0.0f);
                            }
                            part = part + sr;
                        }
                        const double zw = wave_sum(double(at) * double(part));
                        if ((opaque_tid() & (kWave - 1)) == 0) s_z[opaque_tid() / kWave] = zw;
                        __syncthreads();
                        double z = 0.0;
#pragma unroll
                        for (int w = 0; w < NW; ++w) z += s_z[w];
                        Z_c = readlane_f64(z, 0);  // uniform: held in scalar registers
                    }
                }
                if (rec == 0u) {
                    // Every candidate rejected (or a leaf): the token from the
                    // last residual (from p at a leaf, and should the residual
                    // have no mass).  Element mass max(0, e_t - k e_s) m.
                    const bool from_p = !(Z_c > 0.0);
                    float k = 0.0f, m = at;
                    if (!from_p) {
                        k = at > 0.0f ? float(s_c * double(as) / double(at)) : 0.0f;
                        m = float(double(at) / Z_c);
                    }
                    auto mass = [&](int r, int e) -> float {
                        return fmaxf(__builtin_fmaf(-k, c1[r][e], f4_get(lc.load(r, e >> 2), e & 3)), 0.0f) * m;
                    };
                    // Round rr known at run time: the register half is picked
                    // with opaque bit masks (an indexed access would move it to
                    // scratch memory).
                    auto mass_at = [&](int rr, int e) -> float {
                        uint32_t bits = 0u;
#pragma unroll
                        for (int r = 0; r < CPT; ++r) {
                            uint32_t msk = 0u - uint32_t(rr == r);
                            asm volatile("" : "+v"(msk));
                            bits |= __float_as_uint(c1[r][e]) & msk;
                        }
                        return fmaxf(__builtin_fmaf(-k, __uint_as_float(bits), f4_get(lc.load(rr, e >> 2), e & 3)),
                                     0.0f) * m;
                    };
                    int tok = draw_cached<W, CPT, EPC, true>(mass, mass_at, ures, s_cell, &s_dz, &s_tok);
                    if (tok < 0 && !from_p) {
                        k = 0.0f;
                        m = at;
                        tok = draw_cached<W, CPT, EPC, false>(mass, mass_at, ures, s_cell, &s_dz, &s_tok);
                    }
                    rec = (tok >= 0 && tok < a.V) ? node_rec(kNodeDraw, uint32_t(tok)) : node_rec(kNodeBad, 0);
                }
            }
        }
        // The record and the arrival, without waiting for either.
        if (opaque_tid() < kWave) {
            if (opaque_tid() == 0) {
                __hip_atomic_exchange(&a.records[int64_t(b) * N + n], rec, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                pend = __hip_atomic_fetch_add(&a.counters[b], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            pend_b = b;
        }
    }
    if (opaque_tid() < kWave && pend_b >= 0 && uint32_t(__shfl(int(pend), 0, kWave)) == uint32_t(N - 1))
        finish_tree_polled(a, pend_b);
}

template <typename Fmt, int W, int CPT>
int tree_stream_blocks_per_cu() {
    static const int v = [] {
        int nb = 0;
        const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, tree_stream_kernel<Fmt, W, CPT>, W, 0);
        return (e != hipSuccess || nb < 1) ? 1 : nb;
    }();
    return v;
}

template <typename Fmt, int W, int CPT>
hipError_t launch_stream(const TreeLaunch& L, TreeArgs a) {
    int64_t grid = int64_t(L.cus) * tree_stream_blocks_per_cu<Fmt, W, CPT>();
    const int64_t min_grid = (int64_t(a.nitems) + kMaxTreeItems - 1) / kMaxTreeItems;
    if (grid < min_grid) grid = min_grid;
    if (grid > a.nitems) grid = a.nitems;
    a.G = int(grid);
    return launch_kernel(&tree_stream_kernel<Fmt, W, CPT>, dim3(unsigned(grid)), dim3(W), 0, L.stream, a);
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
    RowTile s;
    if (L.vec && L.temperature > 0.0f && pick_stream_tile(L.V, Fmt::kPerChunk, &s)) {
        switch (s.W * 100 + s.CPT) {
            case 25601: return launch_stream<Fmt, 256, 1>(L, a);
            case 51201: return launch_stream<Fmt, 512, 1>(L, a);
            case 102401: return launch_stream<Fmt, 1024, 1>(L, a);
            case 102402: return launch_stream<Fmt, 1024, 2>(L, a);
            case 102403: return launch_stream<Fmt, 1024, 3>(L, a);
            case 102404: return launch_stream<Fmt, 1024, 4>(L, a);
            default: break;
        }
    }
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
    a.nitems = L.B * L.N;
    const int eb = L.dtype == 1 ? 2 : 4;
    a.row_bytes = uint32_t(int64_t(L.V) * eb);
    a.nchunks = int(a.row_bytes / 16u);
    return L.dtype == 1 ? launch_fmt<BF16>(L, a) : launch_fmt<F32>(L, a);
}

}  // namespace osd
