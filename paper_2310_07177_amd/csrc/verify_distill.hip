// verify_distill.hip -- verification and distillation of one speculative
// step in a single pass over the row pairs (gfx950).
//
// Method.  Verification: Appendix A.1 and Eq. 5 of arXiv:2310.07177 (the
// verification step of Algorithm 1) -- proposals y_1..y_k are tested in
// order, y_i is accepted when u_i < p(y_i)/q(y_i), the first rejection at
// position a ends the test, and one more token is drawn from
// norm(max(0, p - q)) at row a, or from p at the bonus row k_b when all were
// accepted.  Distillation: Section 4.1, Eq. 2-4 -- the divergence D (FKL,
// RKL or JSD with weight beta) between the target distribution p and the
// draft distribution q of each masked row, and its gradient with respect to
// the draft logits.  Both use the same temperature T, so the softmax
// normalisers of a row pair are computed once and serve both.
//
// Work layout: the streaming layout of distill_stream.hip.  About one
// workgroup per CU walks the items g, g+G, ...: the B*K row pairs
// (target row i, draft row i) numbered position-major (item i*B + b), then
// the B bonus rows (target row k_b).  While one item is computed, the next
// one's chunks are in flight.  Per row pair:
//   1. statistics pass (max and sum of exponentials of both rows; fills the
//      per-element cache; the thread holding y_i posts t_i[y_i], d_i[y_i]);
//   2. workgroup merge of the normalisers;
//   3. acceptance test; if the proposal is rejected and no earlier rejection
//      of the sequence is known to this workgroup, the correction draw from
//      the cache (exact fixed-point inverse CDF);
//   4. loss and gradient passes from the cache, for rows with mask 1.
// Bonus rows run 1-3 on the target row alone, and are not read at all when
// an earlier rejection of their sequence is known.  Each item posts a
// one-word record; the last workgroup to finish reduces the loss and turns
// the records of every sequence into the outputs.
#include <stdlib.h>

#include <type_traits>

#include "osd.h"
#include "osd_device.hpp"
#include "osd_internal.hpp"
#include "stream_device.hpp"
#include "distill_common.hpp"
#include "cache_draw.hpp"

namespace osd {
namespace {

// Record word: state in bits 31..28, token in bits 27..0.
enum : uint32_t {
    kRecAccept = 1,
    kRecReject = 2,          // rejected, correction token attached
    kRecRejectSkipped = 3,   // rejected after a known earlier rejection
    kRecBadRow = 4,          // no finite logit in a row that was read
    kRecBadToken = 5,        // proposal outside [0, V)
    kRecBonus = 6,           // bonus token attached
    kRecBonusSkipped = 7,    // an earlier rejection was known
    kRecRejectSpec = 8,      // rejected, correction attached, drawn before the
                             // earlier positions' outcomes were known (in the
                             // error-index mode its row was also distilled)
};
// Decision word of a tested position, posted as soon as the acceptance test
// is taken (before the draw and the distillation), so that a later position
// of the sequence can learn early whether it holds the first rejection.
enum : uint32_t { kDecAccept = 1, kDecStop = 2 };
__device__ inline uint32_t make_rec(uint32_t state, uint32_t tok) { return (state << 28) | (tok & 0x0FFFFFFFu); }

// Masses are probabilities (at most 1 per element); chunk sums become exact
// 2^-40 fixed point, so every partial sum of the CDF is an exact integer.
constexpr int kFixedShift = 40;
// Items per workgroup (their arguments are staged in LDS) and the outcomes a
// workgroup remembers.
constexpr int kMaxItems = 256;
// Looks at the earlier positions' decisions before a rejecting workgroup
// draws without knowing whether it holds the first rejection.  Each look is
// one device-coherent round trip plus a short sleep; the bound keeps every
// wait finite whatever the dispatch order.  (The environment variable
// OSD_FUSED_POLLS overrides it, for tests: 0 makes every such workgroup draw
// without looking.)
constexpr int kMaxPolls = 32;

struct FusedArgs {
    // Every word is requested at once on entry (one round trip to the
    // argument buffer); those the prologue needs come first.
    const void* target;        // [B, K+1, V]
    const void* draft;         // [B, K, V]
    const int32_t* tokens;     // [B, K]
    const int32_t* draft_len;  // [B] or null
    const float* u_accept;     // [B, K]
    const float* u_resample;   // [B]
    const uint8_t* mask;       // [B, K] distillation mask or null (all rows)
    int B, K, V;
    int G;                     // workgroups in the grid
    int nitems;                // B*K + B
    int nchunks;
    uint32_t row_bytes;
    int seq_step;              // items k and k - seq_step of a workgroup share a sequence
    int erridx;                // distil the first rejected row of each sequence (not `mask`)
    int max_polls;             // looks at the earlier decisions before drawing speculatively
    float c2;                  // log2(e) / T
    float inv_tau;             // 1 / T
    float beta;
    double c2d;
    double betad, ombd;        // beta and 1 - beta in fp64 (scalar operands of the JSD combination)
    uint32_t* records;         // [B, K+1], zero between calls
    uint32_t* dec;             // [B, K+1] decisions, zero between calls
    int32_t* accepted_len;
    int32_t* out_tokens;
    uint8_t* reject_mask;
    float* row_loss_out;       // [B, K] or null
    void* grad_out;            // [B, K, V] or null
    double* part_ws;           // [G] loss partials ([B*K] row losses in the error-index mode), zero between calls
    uint32_t* done;            // workgroups finished, zero between calls
    float* loss_out;
};

// Per-item arguments, loaded once per workgroup (thread j: its j-th item)
// and staged in LDS, so nothing in the item loop reads global memory except
// the rows (a scalar load there would share its wait counter with LDS).
struct Meta {
    int kb, y;
    float u, u_res;
    int on;  // distillation mask flag; in the error-index mode: every proposal of the sequence is in [0, V)
};

// An item's arguments in two steps, so that the loads are issued before the
// first rows and waited for after them: issue_meta reads every word the
// item needs (in the error-index mode also all K proposals of its sequence,
// K <= 16), finish_meta combines them.
struct MetaLoads {
    Meta m;
    int32_t seq[OSD_MAX_K];
};

__device__ inline MetaLoads issue_meta(const FusedArgs& a, int it) {
    MetaLoads r;
    Meta& m = r.m;
    const int BK = a.B * a.K;
    const bool bonus = it >= BK;
    const int i = bonus ? 0 : it / a.B;
    const int b = bonus ? it - BK : it - i * a.B;
    m.kb = a.draft_len ? a.draft_len[b] : a.K;
    const int64_t ti = int64_t(b) * a.K + i;
    m.y = bonus ? 0 : a.tokens[ti];
    m.u = bonus ? 0.0f : a.u_accept[ti];
    m.u_res = a.u_resample[b];
    m.on = a.erridx ? 0 : (bonus ? 0 : (a.mask ? int(a.mask[ti]) : 1));
#pragma unroll
    for (int j = 0; j < OSD_MAX_K; ++j) r.seq[j] = (a.erridx && j < a.K) ? a.tokens[int64_t(b) * a.K + j] : 0;
    return r;
}

__device__ inline Meta finish_meta(const FusedArgs& a, const MetaLoads& r) {
    Meta m = r.m;
    if (a.erridx) {
        // A proposal outside the vocabulary invalidates the whole sequence,
        // wherever it sits: its rejected row is then not distilled.
        int ok = m.kb >= 1 && m.kb <= a.K;
#pragma unroll
        for (int j = 0; j < OSD_MAX_K; ++j)
            if (j < m.kb) ok = ok && r.seq[j] >= 0 && r.seq[j] < a.V;
        m.on = ok;
    }
    return m;
}

enum : int { kItemNone = 0, kItemBadToken = 1, kItemLive = 2 };

struct Item {
    int row;      // b*(K+1) + i: the target row, and the item's decision and record slot
    int i;        // position (k_b for a bonus row)
    bool bonus;
    int vkind;    // verification: none, bad token or live
    bool dist;    // distillation row with mask 1 (error-index mode: decided after the test)
    bool seq_ok;  // error-index mode: every proposal of the sequence is valid
    int y;
    float u, u_res;
    const char* trow;
    const char* drow;
    int grow;     // gradient and row-loss index b*K + i, or -1 (bonus row)
};

template <typename Fmt>
__device__ inline Item decode_item(const FusedArgs& a, int it, const Meta& m) {
    Item t;
    t.vkind = kItemNone;
    t.dist = false;
    t.seq_ok = a.erridx ? m.on != 0 : true;
    t.trow = nullptr;
    t.drow = nullptr;
    t.grow = -1;
    t.y = m.y;
    t.u = m.u;
    t.u_res = m.u_res;
    const int BK = a.B * a.K;
    t.bonus = it >= BK;
    const int i = t.bonus ? 0 : it / a.B;
    const int b = t.bonus ? it - BK : it - i * a.B;
    t.i = t.bonus ? m.kb : i;
    t.row = b * (a.K + 1) + t.i;
    if (it < 0 || it >= a.nitems) return t;
    const bool kb_ok = m.kb >= 1 && m.kb <= a.K;
    if (!t.bonus) {
        t.grow = b * a.K + i;
        t.dist = !a.erridx && m.on != 0;
        if (kb_ok && i < m.kb) t.vkind = (m.y < 0 || m.y >= a.V) ? kItemBadToken : kItemLive;
    } else if (kb_ok) {
        t.vkind = kItemLive;
    }
    if (t.vkind == kItemLive || t.dist) {
        t.trow = static_cast<const char*>(a.target) + int64_t(t.row) * int64_t(a.V) * Fmt::kBytes;
        if (!t.bonus) t.drow = static_cast<const char*>(a.draft) + int64_t(t.grow) * int64_t(a.V) * Fmt::kBytes;
    }
    return t;
}

// The items of workgroup g of G: the row pairs g, g + G, ... below B*K, then
// the bonus rows b < B with (K-1)*B + b = g (mod G).  Each bonus row goes to
// the workgroup that tests position K-1 of its sequence: by the time that
// position is tested an earlier rejection of the sequence is usually posted,
// so its items seldom draw, while the workgroups of position 0 draw for most
// sequences.  Row pairs k and k - seq_step of a workgroup share a sequence;
// a bonus row shares its sequence with the workgroup's row pair at position
// K-1.  Every field is uniform over the workgroup.
struct Schedule {
    int g, G, B, BK, nrp, b0, nk, seq_step;
    __device__ int item(int k) const { return k < nrp ? g + k * G : BK + b0 + (k - nrp) * G; }
    // The latest earlier item of the workgroup in the same sequence, or < 0.
    __device__ int prev_same(int k) const {
        if (k < nrp) return k - seq_step;
        const int b = b0 + (k - nrp) * G;
        return (BK - B + b - g) / G;
    }
};

__device__ inline Schedule make_schedule(const FusedArgs& a, int g, int G) {
    Schedule s;
    s.g = g;
    s.G = G;
    s.B = a.B;
    s.BK = a.B * a.K;
    s.nrp = g < s.BK ? (s.BK - g + G - 1) / G : 0;
    s.b0 = ((g - (s.BK - a.B)) % G + G) % G;
    s.nk = s.nrp + (s.b0 < a.B ? (a.B - s.b0 + G - 1) / G : 0);
    s.seq_step = a.seq_step;
    return s;
}

// s_rej[k] = 1 if item k of this workgroup or an earlier item of the same
// sequence ended the test (or could not be tested).  Read after a barrier of
// item k (every item has one), the entries up to k - 1 are visible.  Items
// end without a workgroup barrier, so when item k - 1 starts only the entries
// up to k - 3 are certainly visible to every wave (entry j is written by
// thread 0 at the end of item j, before it reaches a barrier of item j + 1):
// the link consulted there, to decide whether item k's rows are read, is the
// latest earlier item of the sequence at or below k - 3.

// An item as the prologue stages it in LDS (thread k decodes item k of its
// workgroup, once), so that the item loop takes each item's fields from two
// uniform LDS reads instead of recomputing them from the schedule and the
// arguments in scalar code.  links holds the entries of the workgroup's
// outcome flags consulted for the item: its latest earlier item of the same
// sequence (bits 0-15) and the one consulted a step ahead (bits 16-31), each
// -1 if none.
struct ItemRec {
    int row, i, y;
    float u, u_res;
    int grow;
    uint32_t flags;  // bit 0 bonus, bits 1-2 vkind, bit 3 dist, bit 4 seq_ok, bit 5 target row read, bit 6 draft row read
    int links;
};
static_assert(sizeof(ItemRec) == 32, "two 16-byte LDS reads per item");

__device__ inline int link_of(int kk) { return kk >= 0 && kk < kMaxItems ? kk : -1; }

template <typename Fmt>
__device__ inline ItemRec encode_item(const FusedArgs& a, const Schedule& sc, int k, const Meta& m) {
    const Item t = decode_item<Fmt>(a, sc.item(k), m);
    ItemRec r;
    r.row = t.row;
    r.i = t.i;
    r.y = t.y;
    r.u = t.u;
    r.u_res = t.u_res;
    r.grow = t.grow;
    r.flags = (t.bonus ? 1u : 0u) | (uint32_t(t.vkind) << 1) | (t.dist ? 8u : 0u) | (t.seq_ok ? 16u : 0u) |
              (t.trow != nullptr ? 32u : 0u) | (t.drow != nullptr ? 64u : 0u);
    int kk = sc.prev_same(k);
    const int prev = link_of(kk);
    while (kk > k - 3) kk = sc.prev_same(kk);
    r.links = int((uint32_t(prev) & 0xFFFFu) | (uint32_t(link_of(kk)) << 16));
    return r;
}

// Item k from the staged records (uniform); prev and ahead receive its links.
template <typename Fmt>
__device__ inline Item item_at(const FusedArgs& a, const ItemRec* s_items, int k, int* prev, int* ahead) {
    const ItemRec v = s_items[k];
    const auto rfl = [](int x) { return __builtin_amdgcn_readfirstlane(x); };
    Item t;
    t.row = rfl(v.row);
    t.i = rfl(v.i);
    t.y = rfl(v.y);
    t.u = __int_as_float(rfl(__float_as_int(v.u)));
    t.u_res = __int_as_float(rfl(__float_as_int(v.u_res)));
    t.grow = rfl(v.grow);
    const uint32_t f = uint32_t(rfl(int(v.flags)));
    const int l = rfl(v.links);
    t.bonus = (f & 1u) != 0;
    t.vkind = int((f >> 1) & 3u);
    t.dist = (f & 8u) != 0;
    t.seq_ok = (f & 16u) != 0;
    t.trow = (f & 32u) ? static_cast<const char*>(a.target) + int64_t(t.row) * a.row_bytes : nullptr;
    t.drow = (f & 64u) ? static_cast<const char*>(a.draft) + int64_t(t.grow) * a.row_bytes : nullptr;
    *prev = int(int16_t(l & 0xFFFF));
    *ahead = l >> 16;
    return t;
}

__device__ inline bool rejected_at(const uint8_t* s_rej, int link) { return link >= 0 && s_rej[link] != 0; }

// Wave 0: the decisions of positions 0..i-1 of one sequence (lane j:
// position j).  2 if one of them stopped the test, 1 if all accepted, 0 if
// still undecided after kMaxPolls looks.
__device__ inline int poll_decisions(const uint32_t* dec, int i, int polls) {
    const int lane = opaque_tid() & (kWave - 1);
    for (int p = 0; p < polls; ++p) {
        if (p > 0) __builtin_amdgcn_s_sleep(8);
        const uint32_t d = lane < i ? load_relaxed(&dec[lane]) : uint32_t(kDecAccept);
        if (__ballot(d == kDecStop) != 0) return 2;
        if (__ballot(d != kDecAccept) == 0) return 1;
    }
    return 0;
}

// What the last workgroup needs, staged in LDS at kernel start so that none
// of it stays in registers across the item loop.
struct FusedTail {
    double* part_ws;
    uint32_t* done;
    float* loss_out;
    const uint8_t* mask;
    int nrows;
    uint32_t* records;
    uint32_t* dec;
    const int32_t* draft_len;
    const int32_t* tokens;
    int32_t* accepted_len;
    int32_t* out_tokens;
    uint8_t* reject_mask;
    float* row_loss_out;
    void* grad_out;
    uint32_t row_bytes;
    int erridx;
    int B, K;
    int G;
};

// Rows whose gradient the last workgroup clears (error-index mode): rows
// distilled before the earlier positions' outcomes were known that turn out
// not to hold the first rejection.  One pass of the finalizer covers at most
// W/16 sequences of at most 15 proposals or W/32 of 16, so at most 1024 rows
// at W = 1024: the list is emptied after every pass.
constexpr int kMaxExtraRows = 1024;

// Every workgroup posts its loss partial and arrives; the last one
//  - turns each sequence's records into the outputs (one segment of 16 or
//    32 lanes per sequence, lane j = position j): the first position whose
//    record is not an acceptance ends the test; a proposal outside the
//    vocabulary invalidates the sequence wherever it sits, a row without
//    finite logits only if the test reaches it;
//  - adds the partials in workgroup order and counts the mask (fixed order,
//    fp64), writing {mean, sum}; in the error-index mode it adds instead
//    the divergence of each sequence's first rejected row, in sequence
//    order, and clears the gradient rows and row losses of rows that were
//    distilled speculatively and turn out not to be first;
//  - reads every record, decision and partial with an exchange that leaves
//    zero.
// All of a pass's reads are issued before any is used (one round trip per
// pass; positions beyond k_b were never posted and read as zero).
template <int W>
__device__ inline void finish_fused(const FusedTail& a, const double* s_part) {
    constexpr int NW = W / kWave;
    static_assert(W <= kMaxExtraRows, "one pass adds at most one row per thread to the list");
    __shared__ int s_last;
    __shared__ double s_sum[NW], s_cnt[NW];
    __shared__ int s_nextra;
    __shared__ int s_extra[kMaxExtraRows];
    // Thread indices from an opaque copy: nothing derived from them before
    // the item loop is kept alive across it.
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & (kWave - 1), wid = tid / kWave;
    const int G = a.G;
    __syncthreads();
    if (tid == 0) {
        if (!a.erridx)
            __hip_atomic_exchange(&a.part_ws[blockIdx.x], s_part[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = int(arrive(a.done)) == G - 1;  // after this workgroup's posts completed
        s_nextra = 0;
    }
    __syncthreads();
    if (!s_last) return;
    // Error-index mode: rows distilled speculatively were released to memory
    // before their records were posted; see them before clearing any.
    if (a.erridx) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    const int K = a.K;
    const int seg = K + 1 <= 16 ? 16 : 32;  // K <= 16
    const int per_pass = W / seg;
    const int j = tid & (seg - 1), base = lane & ~(seg - 1);
    const uint64_t segmask = (seg == 32 ? 0xFFFFFFFFull : 0xFFFFull) << base;
    const int nchunks = int(a.row_bytes / 16);
    // The loss partials and the mask are requested before the records, so
    // that one round trip brings all of them.
    double sm = 0.0, cn = 0.0;
    if (!a.erridx) {
        for (int g = tid; g < G; g += W) sm += take_f64(&a.part_ws[g]);
        for (int r = tid; r < a.nrows; r += W) cn += (a.mask == nullptr || a.mask[r] != 0) ? 1.0 : 0.0;
    }
    double esum = 0.0, ecnt = 0.0;  // error-index mode: this thread's sequences, in order
    for (int b0 = 0; b0 < a.B; b0 += per_pass) {
        const int b = b0 + tid / seg;
        const bool on = b < a.B;
        const int kb = on ? (a.draft_len ? a.draft_len[b] : K) : 0;
        const uint32_t r = on && j <= K ? take_u32(&a.records[int64_t(b) * (K + 1) + j]) : 0u;
        if (on && j < K) take_u32(&a.dec[int64_t(b) * (K + 1) + j]);
        const int32_t tk = on && j < K ? a.tokens[int64_t(b) * K + j] : -1;
        const bool kb_ok = kb >= 1 && kb <= K;
        const uint32_t st = r >> 28;
        const bool drew = st == kRecReject || st == kRecRejectSpec;
        double dj = 0.0;
        if (a.erridx && on && j < K && drew) dj = take_f64(&a.part_ws[int64_t(b) * K + j]);
        const bool bad_token = (__ballot(j < kb && st == kRecBadToken) & segmask) != 0;
        const uint64_t stop = (__ballot(j < kb && st != kRecAccept) & segmask) >> base;
        const int acc = stop ? __builtin_ctzll(stop) : kb;
        const uint32_t ra = __shfl(r, base + (kb_ok ? acc : 0), kWave);
        const uint32_t sa = ra >> 28;
        bool bad = !kb_ok || bad_token;
        int extra = -1;
        if (!bad) {
            if (acc < kb ? (sa == kRecReject || sa == kRecRejectSpec) : sa == kRecBonus)
                extra = int(ra & 0x0FFFFFFFu);
            else
                bad = true;  // a row without finite logits where the test stopped
        }
        if (on && j <= K) {
            const int32_t o = bad ? -1 : (j < acc ? tk : (j == acc ? extra : -1));
            a.out_tokens[int64_t(b) * (K + 1) + j] = o;
            if (a.reject_mask && j < K)
                a.reject_mask[int64_t(b) * K + j] = (!bad && j == acc && acc < kb) ? 1 : 0;
            if (j == 0) a.accepted_len[b] = bad ? -1 : acc;
        }
        if (a.erridx && on && j < K && drew) {
            if (!bad && j == acc) {
                esum += dj;  // the first rejection: its row is the one distilled
                ecnt += 1.0;
            } else {
                // distilled speculatively, not first: its outputs become zero
                if (a.row_loss_out) a.row_loss_out[int64_t(b) * K + j] = 0.0f;
                s_extra[atomicAdd(&s_nextra, 1)] = b * K + j;
            }
        }
        if (a.erridx) {
            __syncthreads();
            const int n = s_nextra;
            if (n > 0 && a.grad_out) {
                for (int e = 0; e < n; ++e) {
                    const rsrc_t gr =
                        make_rsrc(static_cast<char*>(a.grad_out) + int64_t(s_extra[e]) * a.row_bytes, a.row_bytes);
                    for (int c = tid; c < nchunks; c += W) store_chunk_at(gr, c, chunk_t{0u, 0u, 0u, 0u});
                }
            }
            __syncthreads();
            if (tid == 0) s_nextra = 0;
        }
    }
    if (a.erridx) {
        sm = esum;
        cn = ecnt;
    }
    sm = wave_sum(sm);
    cn = wave_sum(cn);
    if (lane == 0) {
        s_sum[wid] = sm;
        s_cnt[wid] = cn;
    }
    __syncthreads();
    if (tid == 0) {
        double ts = 0.0, tc = 0.0;
        for (int w = 0; w < NW; ++w) {
            ts += s_sum[w];
            tc += s_cnt[w];
        }
        a.loss_out[0] = tc > 0.0 ? float(ts / tc) : 0.0f;
        a.loss_out[1] = float(ts);
        take_u32(a.done);
    }
}

template <typename Fmt, int W, int CPT, int KIND>
__global__ __launch_bounds__(W, 1) void verify_distill_kernel(FusedArgs a) {
    constexpr int NW = W / kWave, EPC = Fmt::kPerChunk, NG = EPC / 4;
    // JSD caches exponentials (the others, exponents): see the statistics pass.
    constexpr bool XV = KIND == 2;
    // Items end without a barrier, so a wave can be one item ahead of
    // another: the scratch written once per item is double-buffered by item
    // parity (every item has at least one barrier, so never two ahead).
    __shared__ float s_k[2][2 * NW];
    __shared__ double s_s[2][2 * NW];
    __shared__ RowPair s_rp[2];
    __shared__ double s_a[2 * NW];
    __shared__ ItemRec s_items[kMaxItems];
    __shared__ uint8_t s_rej[kMaxItems];
    __shared__ int s_flag[2];
    __shared__ float s_y[2][2];
    __shared__ double s_cell[CPT * NW];
    __shared__ double s_z;
    __shared__ int s_tok;
    __shared__ double s_part[1];
    __shared__ FusedTail s_tail;
    __shared__ f32x4_t s_c0[CPT * NG * W];
    __shared__ double s_ln2;
    const LdsCache<W, EPC> lc{s_c0};

    // Every argument word the kernel reads, requested together: each
    // dependent request would cost a round trip to the argument buffer
    // (about a microsecond), and no argument is read again later.
    asm volatile("" ::"s"(a.target), "s"(a.draft), "s"(a.tokens), "s"(a.draft_len), "s"(a.u_accept),
                 "s"(a.u_resample), "s"(a.mask));
    asm volatile("" ::"s"(a.B), "s"(a.K), "s"(a.V), "s"(a.G), "s"(a.nitems), "s"(a.nchunks), "s"(a.row_bytes),
                 "s"(a.seq_step), "s"(a.erridx), "s"(a.max_polls), "s"(a.c2), "s"(a.inv_tau), "s"(a.beta));
    asm volatile("" ::"s"(a.c2d), "s"(a.betad), "s"(a.ombd), "s"(a.records), "s"(a.dec), "s"(a.row_loss_out),
                 "s"(a.grad_out), "s"(a.part_ws));
    asm volatile("" ::"s"(a.accepted_len), "s"(a.out_tokens), "s"(a.reject_mask), "s"(a.done), "s"(a.loss_out));
    const int tid = threadIdx.x;
    const int G = a.G;
    const float c2 = a.c2;
    const bool last_ok = (CPT - 1) * W + tid < a.nchunks;
    const float beta = a.beta, omb = 1.0f - a.beta;

    chunk_t rt[CPT], rs[CPT];
    float c1[CPT][EPC];

    const Schedule sc = make_schedule(a, int(blockIdx.x), G);
    const int nk = sc.nk;
    for (int j = tid; j < kMaxItems; j += W) s_rej[j] = 0;  // ordered before any read by the staging barrier
    if (tid == 0) {
        s_ln2 = kLn2;     // ordered before any read by the prologue's barrier
        s_part[0] = 0.0;  // read and written by thread 0 only
        // What the last workgroup needs (from the arguments already read).
        s_tail.part_ws = a.part_ws;
        s_tail.done = a.done;
        s_tail.loss_out = a.loss_out;
        s_tail.mask = a.mask;
        s_tail.nrows = a.B * a.K;
        s_tail.records = a.records;
        s_tail.dec = a.dec;
        s_tail.row_loss_out = a.row_loss_out;
        s_tail.grad_out = a.grad_out;
        s_tail.row_bytes = a.row_bytes;
        s_tail.erridx = a.erridx;
        s_tail.draft_len = a.draft_len;
        s_tail.tokens = a.tokens;
        s_tail.accepted_len = a.accepted_len;
        s_tail.out_tokens = a.out_tokens;
        s_tail.reject_mask = a.reject_mask;
        s_tail.B = a.B;
        s_tail.K = a.K;
        s_tail.G = a.G;
    }
    // Prologue: the item arguments are requested first (a few words per
    // item), then the first item's rows, so that waiting for the arguments
    // does not wait for the rows (loads complete in order) and the first
    // statistics pass folds its chunks in as they land.  The first item's
    // rows are requested before its arguments are known (in bounds either
    // way; a bonus row, whose index is k_b, reads k_b directly).
    {
        const int t = opaque_tid();
        MetaLoads ml{};
        if (t < nk) ml = issue_meta(a, sc.item(t));
        Meta m0;
        m0.kb = a.K;
        m0.y = 0;
        m0.u = 0.0f;
        m0.u_res = 0.0f;
        m0.on = 1;
        const int it0 = sc.item(0);
        if (it0 >= sc.BK && it0 < a.nitems && a.draft_len) m0.kb = scalar_load(a.draft_len + (it0 - sc.BK));
        const Item first = decode_item<Fmt>(a, it0, m0);
        const bool fload = first.trow != nullptr;
        const rsrc_t ftr = make_rsrc(fload ? first.trow : a.target, fload ? a.row_bytes : 0u);
        const rsrc_t fsr =
            make_rsrc(fload && first.drow ? first.drow : a.target, fload && first.drow ? a.row_bytes : 0u);
#pragma unroll
        for (int r = 0; r < CPT; ++r) {
            rt[r] = load_chunk<W>(ftr, r);
            rs[r] = load_chunk<W>(fsr, r);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (t < nk) s_items[t] = encode_item<Fmt>(a, sc, t, finish_meta(a, ml));
        __syncthreads();
    }
    Item cur;
    cur.vkind = kItemNone;
    cur.dist = false;
    cur.bonus = false;
    cur.row = 0;
    cur.i = 0;
    cur.y = 0;
    cur.u = 0.0f;
    cur.u_res = 0.0f;
    cur.trow = nullptr;
    cur.drow = nullptr;
    cur.grow = -1;
    int cur_skip = 0;
    for (int k = 0; k < nk; ++k) {
        Item nxt;
        nxt.bonus = false;
        nxt.trow = nullptr;
        nxt.drow = nullptr;
        int nxt_skip = 0;
        if (k + 1 < nk) {
            int nprev, nahead;
            nxt = item_at<Fmt>(a, s_items, k + 1, &nprev, &nahead);
            // A bonus row whose sequence already stopped here is not read
            // (the current item's outcome is not known yet).
            if (nxt.trow != nullptr && nxt.bonus && rejected_at(s_rej, nahead)) {
                nxt.trow = nullptr;
                nxt_skip = 1;
            }
        }
        const bool nload = nxt.trow != nullptr;
        const rsrc_t ntr = make_rsrc(nload ? nxt.trow : a.target, nload ? a.row_bytes : 0u);
        const rsrc_t nsr = make_rsrc(nload && nxt.drow ? nxt.drow : a.target, nload && nxt.drow ? a.row_bytes : 0u);
        int cprev, cahead;
        cur = item_at<Fmt>(a, s_items, k, &cprev, &cahead);
        // A bonus row is needed only if every proposal of its sequence is
        // accepted.  Besides this workgroup's own outcomes, the decisions
        // that any workgroup has posted so far are consulted (each is
        // written once per call; zero: not posted yet): a stop means the row
        // is not needed.  Wave 0 reads them (k_b <= 16 lanes); the bonus
        // rows come last, when most are posted.
        bool bonus_stop = false;
        if (cur.bonus && cur.vkind == kItemLive && !cur_skip) {
            const int t = opaque_tid();  // nothing tid-derived is kept across the loop
            if (t < kWave) {
                uint32_t d = 0u;
                if (t < cur.i) d = load_relaxed(&a.dec[int64_t(cur.row - cur.i) + t]);
                const uint64_t m = __ballot(d == kDecStop);
                if (t == 0) s_flag[k & 1] = m != 0 ? 1 : 0;
            }
            __syncthreads();
            bonus_stop = s_flag[k & 1] != 0 || rejected_at(s_rej, cprev);
        }
        const bool vlive = cur.vkind == kItemLive && !cur_skip && !bonus_stop;
        const bool live = vlive || cur.dist;
        const int ychunk = cur.y / EPC;
        const rsrc_t gr = make_rsrc(a.grad_out && cur.grow >= 0
                                        ? static_cast<char*>(a.grad_out) + int64_t(cur.grow) * a.row_bytes
                                        : static_cast<char*>(nullptr),
                                    a.grad_out && cur.grow >= 0 ? a.row_bytes : 0u);
        double D = 0.0;
        // ---- statistics pass: consumes the raw chunks and reloads each with
        // the next item's (one load sequence for every item: a branch around
        // the loads would make the compiler wait for all of them) ----
        float kc_t = 0.0f, kc_s = 0.0f;
        double S_t = 0.0, S_s = 0.0;
        if constexpr (XV) {
            // JSD caches each element's 2^(x c2 - k) itself, so the thread's
            // shift k is taken over all its chunks: every cached value is at
            // most 1 and no sum leaves the fp32 range.
            if (live) {
                const float mt = chunks_max<Fmt, CPT>(rt, !last_ok);
                const float ms = chunks_max<Fmt, CPT>(rs, !last_ok);
                kc_t = shift_of_max(mt, c2);
                kc_s = shift_of_max(ms, c2);
            }
        }
#pragma unroll
        for (int r = 0; r < CPT; ++r) {
            if (live) {
                chunk_t xt = rt[r], xs = rs[r];
                if (r == CPT - 1 && !last_ok) {
                    xt = pad_chunk<Fmt>();
                    xs = pad_chunk<Fmt>();
                }
                if (vlive && !cur.bonus && r * W + tid == ychunk) {
                    s_y[k & 1][0] = Fmt::get(xt, cur.y - ychunk * EPC);
                    s_y[k & 1][1] = Fmt::get(xs, cur.y - ychunk * EPC);
                }
                if (!XV && r == 0) {
                    kc_t = first_chunk_shift<Fmt>(xt, c2);
                    kc_s = first_chunk_shift<Fmt>(xs, c2);
                }
                float st = 0.0f, ss = 0.0f;
#pragma unroll
                for (int g = 0; g < NG; ++g) {
                    float c0v[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int e = 4 * g + j;
                        const float t = Fmt::get(xt, e), s = Fmt::get(xs, e);
                        const float vt = __builtin_fmaf(t, c2, -kc_t);
                        const float vs = __builtin_fmaf(s, c2, -kc_s);
                        const float et = exp2_fast(vt), es = exp2_fast(vs);
                        // (the first term starts the sums: 0 + x would cost an add)
                        st = e == 0 ? et : st + et;
                        ss = e == 0 ? es : ss + es;
                        if constexpr (XV) {
                            c0v[j] = et;
                            c1[r][e] = es;
                        } else {
                            // Both exponents: each side's probability is
                            // rebuilt from its own exponent, so a -inf logit
                            // on either side alone gives that side 0 and the
                            // other its true value.  One floor suffices: with
                            // the target's exponent finite, a draft exponent
                            // of -inf still gives q = 0, and two -inf
                            // exponents give a finite difference.
                            c0v[j] = fmaxf(vt, kLogFloor);
                            c1[r][e] = vs;
                        }
                    }
                    lc.store(r, g, f32x4_t{c0v[0], c0v[1], c0v[2], c0v[3]});
                }
                // Keep each round's sums in the round.
                asm volatile("" : "+v"(st), "+v"(ss));
                S_t = r == 0 ? double(st) : S_t + double(st);
                S_s = r == 0 ? double(ss) : S_s + double(ss);
            }
            rt[r] = load_chunk<W>(ntr, r);
            rs[r] = load_chunk<W>(nsr, r);
            __builtin_amdgcn_sched_barrier(0);
        }
        // The record of an item that is not tested (a proposal outside the
        // vocabulary, or a bonus row known to be unneeded); a tested item
        // replaces it below.  Its row may still be distilled.
        uint32_t record = 0u;
        bool stopped = false;  // this item ended the test (or could not be tested)
        bool distilled = false;
        bool release_rows = false;  // error-index mode: this item's outputs may be cleared by the last workgroup
        uint32_t* const dec_at = a.dec + cur.row;
        if (cur.vkind == kItemBadToken) {
            record = make_rec(kRecBadToken, 0);
            stopped = true;
            if (opaque_tid() == 0) __hip_atomic_exchange(dec_at, uint32_t(kDecStop), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else if (cur.vkind == kItemLive && !vlive) {
            record = make_rec(kRecBonusSkipped, 0);
            stopped = true;
        }
        if (!live) {
            if (cur.grow >= 0 && a.grad_out) {
#pragma unroll
                for (int r = 0; r < CPT; ++r) store_chunk<W>(gr, r, chunk_t{0u, 0u, 0u, 0u});
            }
            __syncthreads();  // every item has a barrier (the live ones: the merge)
        } else {
            // Exponent range exceeded by an element far above the first
            // chunk's maximum: rescale exactly from the cache.
            float ks_t = kc_t, ks_s = kc_s;
            if (!XV && S_t >= 1.0e300) {  // (a NaN sum stays NaN: it marks a NaN logit)
                ks_t = kc_t + rescue_sum<CPT, EPC>(S_t, [&](int r, int e) -> float { return lc.load(r, e / 4)[e % 4]; });
            }
            if (!XV && S_s >= 1.0e300) {
                ks_s = kc_s + rescue_sum<CPT, EPC>(S_s, [&](int r, int e) -> float { return c1[r][e]; });
            }
            const RowPair rp = merge_row_pair<NW>(ks_t, S_t, ks_s, S_s, s_k[k & 1], s_s[k & 1], &s_rp[k & 1]);
            const float Kt = rp.kt, Ks = rp.ks;
            const double St = rp.st, Ss = rp.ss;
            // log2 p_j = (t_j c2 - K_t) - (K_row_t - K_t + log2 S_t) = c - ct, likewise q.
            // T = K + log2 S, the rows' log2 normalisers; only their
            // difference is needed in fp64 (from the ratio of the sums).
            const double dTd = rp.dtd;
            const float ct = float(double(Kt - kc_t) + rp.lt), cs = float(double(Ks - kc_s) + rp.ls);
            // FKL/RKL: log2(p/q) = (v_t - v_s) - dTk, from the same rounded
            // exponents as the sums (so the normalisers and the log-ratios
            // agree: rows with p ~ q keep their small divergence accurate).
            const float dTk = float(dTd - double(kc_t - kc_s));
            // JSD: p = e_t at and q = e_s as, the cached values times the
            // thread's scale 2^(k - K) / S (fp64, rounded once).
            const float at = float(__builtin_ldexp(rp.ist, int(fmaxf(kc_t - Kt, -2048.0f))));
            const float as = float(__builtin_ldexp(rp.iss, int(fmaxf(kc_s - Ks, -2048.0f))));

            // ---- verification ----
            bool spec = false;  // drew without knowing the earlier positions' outcomes
            if (vlive) {
                const bool bad = !(St > 0.0 && St < 1.0e300) || (!cur.bonus && !(Ss > 0.0 && Ss < 1.0e300));
                const bool earlier = rejected_at(s_rej, cprev);
                bool want_draw = false;
                if (bad) {
                    record = make_rec(kRecBadRow, 0);
                    stopped = true;
                    if (!cur.bonus && opaque_tid() == 0)
                        __hip_atomic_exchange(dec_at, uint32_t(kDecStop), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                } else if (!cur.bonus) {
                    // p(y)/q(y) = 2^e with e = (t_y - d_y) c2 - (T_t - T_s)
                    // in fp64; 2^e is split into an exact power of two and
                    // 2^frac (v_exp_f32).
                    const double e = (double(s_y[k & 1][0]) - double(s_y[k & 1][1])) * a.c2d - dTd;
                    double ratio;
                    if (!(e > -2000.0)) {
                        ratio = 0.0;  // p(y) = 0
                    } else if (e > 2000.0) {
                        ratio = __builtin_huge_val();
                    } else {
                        const double fl = floor(e);
                        ratio = __builtin_ldexp(double(exp2_fast(float(e - fl))), int(fl));
                    }
                    const bool accept = double(cur.u) < ratio;
                    // Posted now, so that later positions learn it before
                    // this item's draw and distillation.
                    if (opaque_tid() == 0)
                        __hip_atomic_exchange(dec_at, uint32_t(accept ? kDecAccept : kDecStop), __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
                    stopped = !accept;
                    want_draw = !accept && !earlier && cur.seq_ok;
                    record = accept ? make_rec(kRecAccept, 0) : make_rec(kRecRejectSkipped, 0);
                    if (want_draw && cur.i > 0) {
                        // Only the first rejection of a sequence draws (and,
                        // in the error-index mode, is distilled): wave 0
                        // looks at the earlier positions' decisions.
                        if (opaque_tid() < kWave) {
                            const int st = poll_decisions(a.dec + (cur.row - cur.i), cur.i, a.max_polls);
                            if (opaque_tid() == 0) s_flag[k & 1] = st;
                        }
                        __syncthreads();
                        const int st = s_flag[k & 1];
                        want_draw = st != 2;
                        spec = st == 0;
                    }
                } else {
                    stopped = true;
                    want_draw = !earlier;
                    record = make_rec(kRecBonusSkipped, 0);
                }
                if (want_draw) {
                    // Element masses from the cache; the sums and the walk
                    // evaluate exactly this formula on the same values.
                    auto formula = [&](float c0, float cc1, bool residual) -> float {
                        if constexpr (XV) {
                            const float p = c0 * at;
                            if (!residual) return p;
                            return fmaxf(p - cc1 * as, 0.0f);
                        } else {
                            const float lp = c0 - ct, lq = cc1 - cs;
                            const float p = exp2_fast(lp);
                            if (!residual) return p;
                            return fmaxf(p - exp2_fast(lq), 0.0f);
                        }
                    };
                    auto mass = [&](auto res_tag) {
                        return [&](int r, int e) -> float {
                            return formula(lc.load(r, e / 4)[e % 4], c1[r][e], decltype(res_tag)::value);
                        };
                    };
                    // Round rr known at run time: the register half of the
                    // cache is picked with opaque bit masks, so that the
                    // compiler cannot turn the pick into an indexed access
                    // (which would move the whole cache to scratch memory).
                    auto mass_at = [&](auto res_tag) {
                        return [&](int rr, int e) -> float {
                            uint32_t bits = 0u;
#pragma unroll
                            for (int r = 0; r < CPT; ++r) {
                                uint32_t m = 0u - uint32_t(rr == r);
                                asm volatile("" : "+v"(m));
                                bits |= __float_as_uint(c1[r][e]) & m;
                            }
                            return formula(lc.load(rr, e / 4)[e % 4], __uint_as_float(bits),
                                           decltype(res_tag)::value);
                        };
                    };
                    // No residual mass left after rounding (p = q to fp32
                    // accuracy): draw from p.
                    using kResidual = std::integral_constant<bool, true>;
                    using kTarget = std::integral_constant<bool, false>;
                    int tok = -1;
                    if (!cur.bonus)
                        tok = draw_cached<W, CPT, EPC, true>(mass(kResidual{}), mass_at(kResidual{}), cur.u_res,
                                                             s_cell, &s_z, &s_tok);
                    if (tok < 0)
                        tok = draw_cached<W, CPT, EPC, false>(mass(kTarget{}), mass_at(kTarget{}), cur.u_res,
                                                              s_cell, &s_z, &s_tok);
                    if (tok < 0 || tok >= a.V)
                        record = make_rec(kRecBadRow, 0);
                    else
                        record = make_rec(cur.bonus ? kRecBonus : (spec ? kRecRejectSpec : kRecReject), uint32_t(tok));
                }
                stopped = stopped || earlier;
            }
            // The error-index mode distils the row whose draw made the
            // correction (the first rejection, or a speculative one).
            const uint32_t rst = record >> 28;
            const bool dist_now = a.erridx ? (rst == kRecReject || rst == kRecRejectSpec) : cur.dist;
            distilled = dist_now;

            // ---- distillation ----
            if (dist_now) {
                float acc0 = 0.0f, acc1 = 0.0f;
#pragma unroll
                for (int r = 0; r < CPT; ++r) {
                    float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
                    for (int g = 0; g < NG; ++g) {
                        const f32x4_t v = lc.load(r, g);
                        float c0v[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const int e = 4 * g + j;
                            if constexpr (KIND == 2) {
                                const float p = c0v[j] * at, q = c1[r][e] * as;
                                // rho = q/p, clamped to 2^+-126 (both limits stay exact enough:
                                // the vanishing side carries no weight).  log2 m = log2 p + L,
                                // L = log2(beta + (1 - beta) rho): the mixture's log relative
                                // to p, a number near 0 when p ~ q, so the rounding of a log
                                // does not bias every term of a small divergence.  At beta = 0,
                                // L is d itself (the same log of the same value): x = 0.
                                const float rho = __builtin_amdgcn_fmed3f(
                                    q * __builtin_amdgcn_rcpf(fmaxf(p, 0x1p-126f)), 0x1p-126f, 0x1p126f);
                                const float d = log2_fast(rho);
                                const float L = log2_fast(__builtin_fmaf(omb, rho, beta));
                                const float x = d - L;  // log2(q/m)
                                a0 = __builtin_fmaf(p, -L, a0);
                                a1 = __builtin_fmaf(q, x, a1);
                                c0v[j] = x;
                                c1[r][e] = q;
                            } else {
                                // log2(p/q) from the difference of the two
                                // exponents, clamped so that a zero probability
                                // times an infinite log-ratio stays 0.
                                const float lr = fmaxf(fminf((c0v[j] - c1[r][e]) - dTk, -kLogFloor), kLogFloor);
                                if constexpr (KIND == 0) {
                                    const float p = exp2_fast(c0v[j] - ct);
                                    a0 = __builtin_fmaf(p, lr, a0);
                                    c0v[j] = p;
                                    c1[r][e] = c1[r][e] - cs;  // log2 q
                                } else {
                                    const float q = exp2_fast(c1[r][e] - cs);
                                    a0 = __builtin_fmaf(q, lr, a0);
                                    c0v[j] = lr;
                                    c1[r][e] = q;
                                }
                            }
                        }
                        lc.store(r, g, f32x4_t{c0v[0], c0v[1], c0v[2], c0v[3]});
                    }
                    acc0 = acc0 + a0;
                    acc1 = acc1 + a1;
                    __builtin_amdgcn_sched_barrier(0);
                }
                double A0 = double(acc0), A1 = KIND == 2 ? double(acc1) : 0.0;
                block_sum2<NW>(A0, A1, s_a);
                // Terms were accumulated in log2 units.  (ln 2 is read from
                // LDS here rather than held in registers across the item loop.)
                const double ln2d = s_ln2;
                if constexpr (KIND == 2)
                    D = ln2d * (a.betad * A0 + a.ombd * A1);
                else if constexpr (KIND == 0)
                    D = ln2d * A0;
                else
                    D = -ln2d * A0;
                if (a.grad_out && distilled) {
                    const float ln2 = float(kLn2);
                    // JSD: (1-beta) ln2/tau * q * (x - KL2);  RKL: ln2/tau * q * (A0 - lr)
                    const float scale = KIND == 2 ? omb * ln2 * a.inv_tau : ln2 * a.inv_tau;
                    const float shift = KIND == 2 ? float(A1) : float(A0);
#pragma unroll
                    for (int r = 0; r < CPT; ++r) {
                        float g[EPC];
#pragma unroll
                        for (int q4 = 0; q4 < NG; ++q4) {
                            const f32x4_t v = lc.load(r, q4);
                            const float c0v[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                            for (int j = 0; j < 4; ++j) {
                                const int e = 4 * q4 + j;
                                if constexpr (KIND == 0)
                                    g[e] = (exp2_fast(c1[r][e]) - c0v[j]) * a.inv_tau;
                                else if constexpr (KIND == 2)
                                    g[e] = (c1[r][e] * scale) * (c0v[j] - shift);
                                else
                                    g[e] = (c1[r][e] * scale) * (shift - c0v[j]);
                            }
                        }
                        store_chunk<W>(gr, r, pack_grad<Fmt>(g));
                        __builtin_amdgcn_sched_barrier(0);
                    }
                }
            }
            if (!distilled && cur.grow >= 0 && a.grad_out) {
#pragma unroll
                for (int r = 0; r < CPT; ++r) store_chunk<W>(gr, r, chunk_t{0u, 0u, 0u, 0u});
            }
            release_rows = a.erridx && spec && distilled;
        }
        if (release_rows) {  // every wave's gradient stores complete before the release below
            wait_memory();
            __syncthreads();
        }
        if (tid == 0) {
            if (cur.grow >= 0) {
                if (a.row_loss_out) a.row_loss_out[cur.grow] = float(D);
                if (!a.erridx)
                    s_part[0] += D;  // this workgroup's rows, in item order
                else if (distilled)  // the last workgroup adds the first rejections' in sequence order
                    __hip_atomic_exchange(&a.part_ws[cur.grow], D, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            // A speculative row's outputs are written back to memory before
            // its record says so: the last workgroup may overwrite them.
            if (release_rows) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            if (cur.vkind != kItemNone)  // posted at the coherence point; waited for once, at the end
                __hip_atomic_exchange(&a.records[cur.row], record, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (k < kMaxItems) s_rej[k] = (stopped || rejected_at(s_rej, cprev)) ? 1 : 0;
        }
        cur_skip = nxt_skip;
    }
    finish_fused<W>(s_tail, s_part);
}

template <typename Fmt, int W, int CPT, int KIND>
int blocks_per_cu() {
    static const int v = [] {
        int nb = 0;
        const hipError_t e =
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, verify_distill_kernel<Fmt, W, CPT, KIND>, W, 0);
        return (e != hipSuccess || nb < 1) ? 1 : nb;
    }();
    return v;
}

template <typename Fmt, int W, int CPT, int KIND>
hipError_t launch_kind(const FusedLaunch& L, FusedArgs a) {
    int64_t want = int64_t(L.cus) * blocks_per_cu<Fmt, W, CPT, KIND>();
    // Each workgroup stages at most ceil(BK/G) + ceil(B/G) <= nitems/G + 2 items.
    const int64_t min_grid = (int64_t(a.nitems) + kMaxItems - 3) / (kMaxItems - 2);
    if (want < min_grid) want = min_grid;
    const int64_t BK = int64_t(a.B) * a.K;
    const unsigned grid = unsigned(want < BK ? want : BK);
    int g = int(grid), r = a.B;
    while (r != 0) {
        const int t = g % r;
        g = r;
        r = t;
    }
    a.seq_step = a.B / g;
    a.G = int(grid);
    const hipError_t e = launch_kernel(&verify_distill_kernel<Fmt, W, CPT, KIND>, dim3(grid), dim3(W), 0, L.stream, a);
    return e;
}

template <typename Fmt, int W, int CPT>
hipError_t launch_tile(const FusedLaunch& L, const FusedArgs& a) {
    switch (L.kind) {
        case 0: return launch_kind<Fmt, W, CPT, 0>(L, a);
        case 1: return launch_kind<Fmt, W, CPT, 1>(L, a);
        default: return launch_kind<Fmt, W, CPT, 2>(L, a);
    }
}

template <typename Fmt>
hipError_t launch_fmt(const FusedLaunch& L, const FusedArgs& a) {
    RowTile t;
    if (!pick_stream_tile(L.V, Fmt::kPerChunk, &t)) return hipErrorInvalidValue;
    switch (t.W * 100 + t.CPT) {
        case 25601: return launch_tile<Fmt, 256, 1>(L, a);
        case 51201: return launch_tile<Fmt, 512, 1>(L, a);
        case 102401: return launch_tile<Fmt, 1024, 1>(L, a);
        case 102402: return launch_tile<Fmt, 1024, 2>(L, a);
        case 102403: return launch_tile<Fmt, 1024, 3>(L, a);
        case 102404: return launch_tile<Fmt, 1024, 4>(L, a);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

// kMaxPolls, or the value of OSD_FUSED_POLLS (read once).
int fused_max_polls() {
    static const int v = [] {
        const char* e = getenv("OSD_FUSED_POLLS");
        if (e == nullptr || *e == 0) return kMaxPolls;
        const int n = atoi(e);
        return n < 0 ? kMaxPolls : (n > 4096 ? 4096 : n);
    }();
    return v;
}

hipError_t launch_verify_distill(const FusedLaunch& L) {
    FusedArgs a{};
    a.target = L.target;
    a.draft = L.draft;
    a.B = L.B;
    a.K = L.K;
    a.V = L.V;
    a.tokens = L.tokens;
    a.draft_len = L.draft_len;
    a.u_accept = L.u_accept;
    a.u_resample = L.u_resample;
    a.mask = L.mask;
    a.c2 = float(1.4426950408889634 / double(L.temperature));
    a.c2d = double(a.c2);
    a.beta = L.beta;
    a.betad = double(L.beta);
    a.ombd = 1.0 - double(L.beta);
    a.inv_tau = float(1.0 / double(L.temperature));
    a.records = L.records;
    a.dec = L.dec;
    a.erridx = L.erridx;
    a.max_polls = fused_max_polls();
    a.accepted_len = L.accepted_len;
    a.out_tokens = L.out_tokens;
    a.reject_mask = L.reject_mask;
    a.row_loss_out = L.row_loss_out;
    a.grad_out = L.grad_out;
    a.part_ws = L.part_ws;
    a.done = L.done;
    a.loss_out = L.loss_out;
    a.nitems = L.B * L.K + L.B;
    const int eb = L.dtype == 1 ? 2 : 4;
    a.nchunks = int((int64_t(L.V) * eb) / 16);
    a.row_bytes = uint32_t(int64_t(L.V) * eb);
    a.seq_step = 1;
    return L.dtype == 1 ? launch_fmt<BF16>(L, a) : launch_fmt<F32>(L, a);
}

}  // namespace osd
