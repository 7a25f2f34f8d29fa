// osd_api.hip -- the C ABI of libosd (declared in include/osd.h): argument
// validation, workspace carving and kernel dispatch.  No allocation, no
// synchronisation; the only global state is the allocation-free entry
// point's scratch array and its per-device address (end of this file).
#include <math.h>

#include <mutex>

#include "osd.h"
#include "osd_internal.hpp"

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int per_chunk(int dtype) { return dtype == OSD_BF16 ? 8 : (dtype == OSD_F32 ? 4 : 0); }
int elem_bytes(int dtype) { return dtype == OSD_BF16 ? 2 : 4; }

// Counters and records of the row-resident kernel, then the argmax partials
// of the segmented greedy kernels.  Every call leaves all of it zero.
struct VerifyWs {
    size_t records, counters, stats, total;
};
VerifyWs verify_layout(int B, int K) {
    VerifyWs w;
    const size_t rows = size_t(B) * size_t(K + 1);
    w.counters = 0;
    w.records = round_up(size_t(B) * 4, kAlign);
    w.stats = w.records + round_up(rows * 4, kAlign);
    w.total = w.stats + round_up(rows * osd::kMaxSeg * sizeof(osd::SegStats), kAlign);
    return w;
}

struct DistillWs {
    size_t done, slab_cnt, slabs, rows, split, total;
    int nslabs;
};
// Counters first, at offsets that do not depend on B*K beyond their own
// count, then the fp64 partial sums; the kernels leave every byte zero.
DistillWs distill_layout(int B, int K) {
    DistillWs w;
    const size_t R = size_t(B) * size_t(K);
    w.nslabs = int((R + osd::kSlabRows - 1) / osd::kSlabRows);
    w.done = 0;
    w.slab_cnt = 16;
    w.slabs = round_up(w.slab_cnt + size_t(w.nslabs) * 4, kAlign);
    w.rows = w.slabs + round_up(size_t(w.nslabs) * 16, kAlign);
    w.split = w.rows + round_up(R * 8, kAlign);
    w.total = w.split + round_up(R * osd::kSplitBytesPerRow, kAlign);
    return w;
}

// The fused entry points: the verify workspace, then the distill workspace
// (both used as they are by the two-call path; the fused kernel keeps its
// per-position decisions where the greedy partials go), then per-workgroup
// loss partials of the fused kernel (at most one per item; per-row losses in
// the error-index mode), then a [B, K] mask for the error-index mode's
// two-call path when the caller passes no reject_mask.
struct FusedWs {
    size_t verify, distill, part, mask, total;
};
FusedWs fused_layout(int B, int K) {
    FusedWs w;
    w.verify = 0;
    w.distill = round_up(verify_layout(B, K).total, kAlign);
    w.part = w.distill + round_up(distill_layout(B, K).total, kAlign);
    w.mask = w.part + round_up(size_t(B) * size_t(K + 1) * 8, kAlign);
    w.total = w.mask + round_up(size_t(B) * size_t(K), kAlign);
    return w;
}

// Compute units of the device that runs `stream` (queried once per device).
int device_cus(hipStream_t stream) {
    static int cache[64] = {0};
    int dev = 0;
    if (stream == nullptr || hipStreamGetDevice(stream, &dev) != hipSuccess) {
        if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    }
    if (dev < 0 || dev >= 64) dev = 0;
    int n = __atomic_load_n(&cache[dev], __ATOMIC_RELAXED);
    if (n <= 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        __atomic_store_n(&cache[dev], n, __ATOMIC_RELAXED);
    }
    return n;
}

// Zero n 32-bit words (a kernel rather than a memset: it may be captured
// into a graph).
__global__ void clear_words(uint32_t* p, int n) {
    for (int i = int(blockIdx.x * blockDim.x + threadIdx.x); i < n; i += int(gridDim.x * blockDim.x)) p[i] = 0u;
}

hipError_t launch_clear_words(uint32_t* p, int n, hipStream_t s) {
    const int threads = 256, want = (n + threads - 1) / threads, blocks = want < 1024 ? (want > 0 ? want : 1) : 1024;
    return osd::launch_kernel(&clear_words, dim3(blocks), dim3(threads), 0, s, p, n);
}

bool sizes_ok(int B, int K, int V, int dtype) {
    if (B <= 0 || K <= 0 || V <= 0 || K > OSD_MAX_K) return false;
    if (per_chunk(dtype) == 0) return false;
    if (V > osd::max_vocab_for(per_chunk(dtype))) return false;
    // grid.x = B * (K + 1) must fit in 31 bits
    if (int64_t(B) * int64_t(K + 1) > 0x7FFFFFFFll) return false;
    return true;
}

}  // namespace

extern "C" {

int osd_max_vocab(int dtype) {
    return per_chunk(dtype) ? osd::max_vocab_for(per_chunk(dtype)) : 0;
}

const char* osd_status_string(int status) {
    switch (status) {
        case OSD_OK: return "OSD_OK";
        case OSD_ERR_INVALID_ARG: return "OSD_ERR_INVALID_ARG: an argument is out of range or a required pointer is NULL";
        case OSD_ERR_UNSUPPORTED: return "OSD_ERR_UNSUPPORTED: the vocabulary size or dtype is not supported";
        case OSD_ERR_DEVICE: return "OSD_ERR_DEVICE: the HIP runtime failed to launch a kernel";
        case OSD_ERR_WORKSPACE: return "OSD_ERR_WORKSPACE: the workspace is NULL or smaller than required";
        case OSD_ERR_SCRATCH:
            return "OSD_ERR_SCRATCH: the call needs more scratch than the allocation-free entry point holds "
                   "(osd_verify_workspace_bytes(B, K) > OSD_VERIFY_NOALLOC_SCRATCH_BYTES)";
        default: return "unknown osd status";
    }
}

size_t osd_verify_workspace_bytes(int B, int K) {
    if (B <= 0 || K <= 0 || K > OSD_MAX_K) return 0;
    return verify_layout(B, K).total;
}

int osd_verify(const void* target_logits, const void* draft_logits, int dtype, int B, int K,
               int V, const int32_t* draft_tokens, const int32_t* draft_len,
               const float* u_accept, const float* u_resample, float temperature,
               int32_t* accepted_len, int32_t* out_tokens, uint8_t* reject_mask,
               void* workspace, size_t workspace_bytes, void* stream) {
    if (dtype != OSD_F32 && dtype != OSD_BF16) return OSD_ERR_INVALID_ARG;
    if (B <= 0 || K <= 0 || V <= 0 || K > OSD_MAX_K) return OSD_ERR_INVALID_ARG;
    if (!sizes_ok(B, K, V, dtype)) return OSD_ERR_UNSUPPORTED;
    if (!(temperature >= 0.0f) || isinf(temperature)) return OSD_ERR_INVALID_ARG;
    const bool greedy = temperature == 0.0f;
    if (!target_logits || !draft_tokens || !accepted_len || !out_tokens) return OSD_ERR_INVALID_ARG;
    if (!greedy && (!draft_logits || !u_accept || !u_resample)) return OSD_ERR_INVALID_ARG;
    const VerifyWs ws = verify_layout(B, K);
    if (!workspace || workspace_bytes < ws.total || (reinterpret_cast<uintptr_t>(workspace) & 15u))
        return OSD_ERR_WORKSPACE;

    osd::VerifyLaunch L;
    L.target = target_logits;
    L.draft = greedy ? nullptr : draft_logits;
    L.dtype = dtype;
    L.B = B;
    L.K = K;
    L.V = V;
    L.tokens = draft_tokens;
    L.draft_len = draft_len;
    L.u_accept = u_accept;
    L.u_resample = u_resample;
    L.temperature = temperature;
    L.accepted_len = accepted_len;
    L.out_tokens = out_tokens;
    L.reject_mask = reject_mask;
    char* w = static_cast<char*>(workspace);
    L.records = reinterpret_cast<uint32_t*>(w + ws.records);
    L.counters = reinterpret_cast<uint32_t*>(w + ws.counters);
    L.seg_stats = reinterpret_cast<osd::SegStats*>(w + ws.stats);
    L.vec = (int64_t(V) * elem_bytes(dtype)) % 16 == 0 && aligned16(target_logits) &&
            (greedy || aligned16(draft_logits));
    L.stream = static_cast<hipStream_t>(stream);
    // Greedy: segmented kernels (balanced over every CU).  Sampling: the
    // row-resident kernel, which draws from rows it already holds.
    int nseg = 0;
    const bool segmented = greedy && L.vec && osd::greedy_segments(V, per_chunk(dtype), &nseg);
    const hipError_t e = segmented ? osd::launch_verify_greedy(L) : osd::launch_verify(L);
    return e == hipSuccess ? OSD_OK : OSD_ERR_DEVICE;
}

size_t osd_distill_workspace_bytes(int B, int K) {
    if (B <= 0 || K <= 0) return 0;
    if (int64_t(B) * int64_t(K) > 0x7FFFFFFFll) return 0;
    return distill_layout(B, K).total;
}

int osd_distill_loss_grad(const void* teacher_logits, int64_t teacher_batch_stride,
                          const void* student_logits, int64_t student_batch_stride, int dtype,
                          int B, int K, int V, const uint8_t* mask, int kind, float beta,
                          float tau, float* loss_out, float* row_loss_out, void* grad_out,
                          void* workspace, size_t workspace_bytes, void* stream) {
    if (dtype != OSD_F32 && dtype != OSD_BF16) return OSD_ERR_INVALID_ARG;
    if (B <= 0 || K <= 0 || V <= 0) return OSD_ERR_INVALID_ARG;
    if (int64_t(B) * int64_t(K) > 0x7FFFFFFFll) return OSD_ERR_INVALID_ARG;
    if (per_chunk(dtype) == 0 || V > osd::max_vocab_for(per_chunk(dtype))) return OSD_ERR_UNSUPPORTED;
    if (kind != OSD_FKL && kind != OSD_RKL && kind != OSD_JSD) return OSD_ERR_INVALID_ARG;
    if (!(tau > 0.0f) || isinf(tau)) return OSD_ERR_INVALID_ARG;
    if (!(beta >= 0.0f && beta <= 1.0f)) return OSD_ERR_INVALID_ARG;
    if (!teacher_logits || !student_logits || !loss_out) return OSD_ERR_INVALID_ARG;
    // The K rows of one sequence must not overlap those of the next.
    if (B > 1 && (teacher_batch_stride < int64_t(K) * V || student_batch_stride < int64_t(K) * V))
        return OSD_ERR_INVALID_ARG;
    const DistillWs ws = distill_layout(B, K);
    if (!workspace || workspace_bytes < ws.total || (reinterpret_cast<uintptr_t>(workspace) & 15u))
        return OSD_ERR_WORKSPACE;

    osd::DistillLaunch L;
    L.teacher = teacher_logits;
    L.teacher_stride = teacher_batch_stride;
    L.student = student_logits;
    L.student_stride = student_batch_stride;
    L.dtype = dtype;
    L.B = B;
    L.K = K;
    L.V = V;
    L.mask = mask;
    L.kind = kind;
    L.beta = beta;
    L.tau = tau;
    L.loss_out = loss_out;
    L.row_loss_out = row_loss_out;
    L.grad_out = grad_out;
    char* w = static_cast<char*>(workspace);
    L.row_loss_ws = reinterpret_cast<double*>(w + ws.rows);
    L.split_ws = w + ws.split;
    L.slab_ws = reinterpret_cast<double*>(w + ws.slabs);
    L.slab_counters = reinterpret_cast<uint32_t*>(w + ws.slab_cnt);
    L.done_counter = reinterpret_cast<uint32_t*>(w + ws.done);
    const int eb = elem_bytes(dtype);
    L.vec = (int64_t(V) * eb) % 16 == 0 && (teacher_batch_stride * eb) % 16 == 0 &&
            (student_batch_stride * eb) % 16 == 0 && aligned16(teacher_logits) &&
            aligned16(student_logits) && (grad_out == nullptr || aligned16(grad_out));
    L.stream = static_cast<hipStream_t>(stream);
    L.cus = device_cus(L.stream);
    osd::RowTile t;
    const bool streaming = L.vec && osd::pick_stream_tile(V, per_chunk(dtype), &t);
    const hipError_t e = streaming ? osd::launch_distill_stream(L) : osd::launch_distill(L);
    return e == hipSuccess ? OSD_OK : OSD_ERR_DEVICE;
}

size_t osd_verify_distill_workspace_bytes(int B, int K) {
    if (B <= 0 || K <= 0 || K > OSD_MAX_K) return 0;
    if (int64_t(B) * int64_t(K + 1) > 0x7FFFFFFFll) return 0;
    return fused_layout(B, K).total;
}

}  // extern "C"

namespace {

// Both fused entry points: erridx = 0 distils the caller's mask, 1 the row
// at each sequence's first rejection (the error index).
int verify_distill_impl(const void* target_logits, const void* draft_logits, int dtype, int B, int K, int V,
                        const int32_t* draft_tokens, const int32_t* draft_len, const float* u_accept,
                        const float* u_resample, float temperature, int32_t* accepted_len, int32_t* out_tokens,
                        uint8_t* reject_mask, const uint8_t* distill_mask, int erridx, int kind, float beta,
                        float* loss_out, float* row_loss_out, void* grad_out, void* workspace,
                        size_t workspace_bytes, void* stream) {
    if (dtype != OSD_F32 && dtype != OSD_BF16) return OSD_ERR_INVALID_ARG;
    if (B <= 0 || K <= 0 || V <= 0 || K > OSD_MAX_K) return OSD_ERR_INVALID_ARG;
    if (!sizes_ok(B, K, V, dtype)) return OSD_ERR_UNSUPPORTED;
    if (!(temperature > 0.0f) || isinf(temperature)) return OSD_ERR_INVALID_ARG;
    if (kind != OSD_FKL && kind != OSD_RKL && kind != OSD_JSD) return OSD_ERR_INVALID_ARG;
    if (!(beta >= 0.0f && beta <= 1.0f)) return OSD_ERR_INVALID_ARG;
    if (!target_logits || !draft_logits || !draft_tokens || !u_accept || !u_resample || !accepted_len ||
        !out_tokens || !loss_out)
        return OSD_ERR_INVALID_ARG;
    const FusedWs ws = fused_layout(B, K);
    if (!workspace || workspace_bytes < ws.total || (reinterpret_cast<uintptr_t>(workspace) & 15u))
        return OSD_ERR_WORKSPACE;
    char* w = static_cast<char*>(workspace);
    const int eb = elem_bytes(dtype);
    osd::RowTile t;
    const bool fused = (int64_t(V) * eb) % 16 == 0 && aligned16(target_logits) && aligned16(draft_logits) &&
                       (grad_out == nullptr || aligned16(grad_out)) && osd::pick_stream_tile(V, per_chunk(dtype), &t);
    if (!fused) {  // the two calls, each on its own part of the workspace
        const VerifyWs vw = verify_layout(B, K);
        const DistillWs dw = distill_layout(B, K);
        uint8_t* rmask = reject_mask;
        if (erridx && !rmask) rmask = reinterpret_cast<uint8_t*>(w + ws.mask);
        int st = osd_verify(target_logits, draft_logits, dtype, B, K, V, draft_tokens, draft_len, u_accept,
                            u_resample, temperature, accepted_len, out_tokens, rmask, w + ws.verify, vw.total,
                            stream);
        if (st != OSD_OK) return st;
        st = osd_distill_loss_grad(target_logits, int64_t(K + 1) * V, draft_logits, int64_t(K) * V, dtype, B, K, V,
                                   erridx ? rmask : distill_mask, kind, beta, temperature, loss_out, row_loss_out,
                                   grad_out, w + ws.distill, dw.total, stream);
        if (st != OSD_OK || rmask == reject_mask) return st;
        // The mask kept in the workspace: every call leaves its workspace zero.
        const int words = int((size_t(B) * size_t(K) + 3) / 4);
        return launch_clear_words(reinterpret_cast<uint32_t*>(rmask), words, static_cast<hipStream_t>(stream)) ==
                       hipSuccess
                   ? OSD_OK
                   : OSD_ERR_DEVICE;
    }
    osd::FusedLaunch L;
    L.target = target_logits;
    L.draft = draft_logits;
    L.dtype = dtype;
    L.B = B;
    L.K = K;
    L.V = V;
    L.tokens = draft_tokens;
    L.draft_len = draft_len;
    L.u_accept = u_accept;
    L.u_resample = u_resample;
    L.temperature = temperature;
    L.mask = erridx ? nullptr : distill_mask;
    L.kind = kind;
    L.beta = beta;
    L.accepted_len = accepted_len;
    L.out_tokens = out_tokens;
    L.reject_mask = reject_mask;
    L.loss_out = loss_out;
    L.row_loss_out = row_loss_out;
    L.grad_out = grad_out;
    const VerifyWs vw = verify_layout(B, K);
    L.records = reinterpret_cast<uint32_t*>(w + ws.verify + vw.records);
    L.dec = reinterpret_cast<uint32_t*>(w + ws.verify + vw.stats);
    L.erridx = erridx;
    L.done = reinterpret_cast<uint32_t*>(w + ws.distill + distill_layout(B, K).done);
    L.part_ws = reinterpret_cast<double*>(w + ws.part);
    L.stream = static_cast<hipStream_t>(stream);
    L.cus = device_cus(L.stream);
    return osd::launch_verify_distill(L) == hipSuccess ? OSD_OK : OSD_ERR_DEVICE;
}

}  // namespace

extern "C" {

int osd_verify_distill(const void* target_logits, const void* draft_logits, int dtype, int B, int K,
                       int V, const int32_t* draft_tokens, const int32_t* draft_len,
                       const float* u_accept, const float* u_resample, float temperature,
                       int32_t* accepted_len, int32_t* out_tokens, uint8_t* reject_mask,
                       const uint8_t* distill_mask, int kind, float beta, float* loss_out,
                       float* row_loss_out, void* grad_out, void* workspace, size_t workspace_bytes,
                       void* stream) {
    return verify_distill_impl(target_logits, draft_logits, dtype, B, K, V, draft_tokens, draft_len, u_accept,
                               u_resample, temperature, accepted_len, out_tokens, reject_mask, distill_mask, 0,
                               kind, beta, loss_out, row_loss_out, grad_out, workspace, workspace_bytes, stream);
}

int osd_verify_distill_rejected(const void* target_logits, const void* draft_logits, int dtype, int B, int K,
                                int V, const int32_t* draft_tokens, const int32_t* draft_len,
                                const float* u_accept, const float* u_resample, float temperature,
                                int32_t* accepted_len, int32_t* out_tokens, uint8_t* reject_mask, int kind,
                                float beta, float* loss_out, float* row_loss_out, void* grad_out,
                                void* workspace, size_t workspace_bytes, void* stream) {
    return verify_distill_impl(target_logits, draft_logits, dtype, B, K, V, draft_tokens, draft_len, u_accept,
                               u_resample, temperature, accepted_len, out_tokens, reject_mask, nullptr, 1, kind,
                               beta, loss_out, row_loss_out, grad_out, workspace, workspace_bytes, stream);
}

size_t osd_sample_workspace_bytes(int N) {
    if (N <= 0) return 0;
    return size_t(N) * osd::kSampleWsPerRow;
}

int osd_sample(const void* p_logits, int64_t p_row_stride, const void* q_logits, int64_t q_row_stride,
               int dtype, int N, int V, float temperature, float beta, const float* u,
               int32_t* out_tokens, void* workspace, size_t workspace_bytes, void* stream) {
    if (dtype != OSD_F32 && dtype != OSD_BF16) return OSD_ERR_INVALID_ARG;
    if (N <= 0 || V <= 0) return OSD_ERR_INVALID_ARG;
    if (V > osd_max_vocab(dtype)) return OSD_ERR_UNSUPPORTED;
    if (!(temperature >= 0.0f) || isinf(temperature)) return OSD_ERR_INVALID_ARG;
    if (!(beta >= 0.0f && beta <= 1.0f)) return OSD_ERR_INVALID_ARG;
    const bool greedy = temperature == 0.0f;
    const bool use_p = beta > 0.0f, use_q = beta < 1.0f;
    if (greedy && use_p && use_q) return OSD_ERR_INVALID_ARG;
    if (!out_tokens || (!greedy && !u)) return OSD_ERR_INVALID_ARG;
    if (use_p && (!p_logits || p_row_stride < V)) return OSD_ERR_INVALID_ARG;
    if (use_q && (!q_logits || q_row_stride < V)) return OSD_ERR_INVALID_ARG;
    if (workspace && (workspace_bytes < osd_sample_workspace_bytes(N) ||
                      (reinterpret_cast<uintptr_t>(workspace) & 15u)))
        return OSD_ERR_WORKSPACE;
    const int64_t eb = elem_bytes(dtype);
    osd::SampleLaunch L;
    L.p = use_p ? p_logits : nullptr;
    L.p_stride = use_p ? p_row_stride : 0;
    L.q = use_q ? q_logits : nullptr;
    L.q_stride = use_q ? q_row_stride : 0;
    L.dtype = dtype;
    L.N = N;
    L.V = V;
    L.temperature = temperature;
    L.beta = beta;
    L.u = u;
    L.out = out_tokens;
    L.workspace = workspace;
    L.vec = (int64_t(V) * eb) % 16 == 0 && (!use_p || (aligned16(p_logits) && (p_row_stride * eb) % 16 == 0)) &&
            (!use_q || (aligned16(q_logits) && (q_row_stride * eb) % 16 == 0));
    L.stream = static_cast<hipStream_t>(stream);
    L.cus = device_cus(L.stream);
    return osd::launch_sample(L) == hipSuccess ? OSD_OK : OSD_ERR_DEVICE;
}

}  // extern "C"

namespace {

// Vocabulary-sharded verification: the checks every phase shares.  The whole
// row's fixed-point mass stays below 2^63 for V <= 2^19.
constexpr int kMaxShardedVocab = 1 << 19;

int shard_common(const void* target, int dtype, int B, int K, int V_shard, float temperature,
                 const int32_t* draft_tokens) {
    if (dtype != OSD_F32 && dtype != OSD_BF16) return OSD_ERR_INVALID_ARG;
    if (B <= 0 || K <= 0 || V_shard <= 0 || K > OSD_MAX_K) return OSD_ERR_INVALID_ARG;
    if (!sizes_ok(B, K, V_shard, dtype)) return OSD_ERR_UNSUPPORTED;
    // A rank's slice is held in registers: at most 8 chunks per thread of a
    // 1024-thread workgroup (65536 bf16 or 32768 fp32 logits).
    osd::RowTile t;
    if (!osd::pick_tile(V_shard, per_chunk(dtype), &t)) return OSD_ERR_UNSUPPORTED;
    if (!(temperature >= 0.0f) || isinf(temperature)) return OSD_ERR_INVALID_ARG;
    if (!target || !draft_tokens) return OSD_ERR_INVALID_ARG;
    return OSD_OK;
}

bool aligned8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }

osd::ShardLaunch shard_launch(int phase, const void* target, const void* draft, int dtype, int B, int K,
                              int V_shard, float temperature, const int32_t* tokens, const int32_t* draft_len,
                              void* stream) {
    osd::ShardLaunch L = {};
    L.phase = phase;
    L.target = target;
    L.draft = temperature == 0.0f ? nullptr : draft;
    L.dtype = dtype;
    L.B = B;
    L.K = K;
    L.Vs = V_shard;
    L.tokens = tokens;
    L.draft_len = draft_len;
    L.temperature = temperature;
    L.vec = (int64_t(V_shard) * elem_bytes(dtype)) % 16 == 0 && aligned16(target) &&
            (L.draft == nullptr || aligned16(L.draft));
    L.stream = static_cast<hipStream_t>(stream);
    return L;
}

}  // namespace

extern "C" {

int osd_shard_verify_stats(const void* target_shard, const void* draft_shard, int dtype, int B, int K,
                           int V_shard, int v_begin, int V, const int32_t* draft_tokens,
                           const int32_t* draft_len, float temperature, osd_shard_row_stats* stats,
                           void* stream) {
    const int st = shard_common(target_shard, dtype, B, K, V_shard, temperature, draft_tokens);
    if (st != OSD_OK) return st;
    if (V <= 0 || v_begin < 0 || int64_t(v_begin) + V_shard > V) return OSD_ERR_INVALID_ARG;
    if (V > kMaxShardedVocab) return OSD_ERR_UNSUPPORTED;
    if (temperature > 0.0f && !draft_shard) return OSD_ERR_INVALID_ARG;
    if (!stats || !aligned8(stats)) return OSD_ERR_INVALID_ARG;
    osd::ShardLaunch L = shard_launch(1, target_shard, draft_shard, dtype, B, K, V_shard, temperature,
                                      draft_tokens, draft_len, stream);
    L.v_begin = v_begin;
    L.V = V;
    L.stats = stats;
    return osd::launch_verify_shard(L) == hipSuccess ? OSD_OK : OSD_ERR_DEVICE;
}

int osd_shard_verify_mass(const void* target_shard, const void* draft_shard, int dtype, int B, int K,
                          int V_shard, int G, const int32_t* draft_tokens, const int32_t* draft_len,
                          const float* u_accept, float temperature, const osd_shard_row_stats* stats_all,
                          osd_shard_mass* mass, void* stream) {
    const int st = shard_common(target_shard, dtype, B, K, V_shard, temperature, draft_tokens);
    if (st != OSD_OK) return st;
    if (G < 1 || G > OSD_MAX_SHARDS) return OSD_ERR_INVALID_ARG;
    if (temperature > 0.0f && (!draft_shard || !u_accept)) return OSD_ERR_INVALID_ARG;
    if (!stats_all || !mass || !aligned8(stats_all) || !aligned8(mass)) return OSD_ERR_INVALID_ARG;
    osd::ShardLaunch L = shard_launch(2, target_shard, draft_shard, dtype, B, K, V_shard, temperature,
                                      draft_tokens, draft_len, stream);
    L.G = G;
    L.u_accept = u_accept;
    L.stats_in = stats_all;
    L.mass = mass;
    return osd::launch_verify_shard(L) == hipSuccess ? OSD_OK : OSD_ERR_DEVICE;
}

int osd_shard_verify_draw(const void* target_shard, const void* draft_shard, int dtype, int B, int K,
                          int V_shard, int v_begin, int G, int shard, const int32_t* draft_tokens,
                          const int32_t* draft_len, const float* u_resample, float temperature,
                          const osd_shard_mass* mass_all, int32_t* accepted_len, int32_t* out_tokens,
                          uint8_t* reject_mask, void* stream) {
    const int st = shard_common(target_shard, dtype, B, K, V_shard, temperature, draft_tokens);
    if (st != OSD_OK) return st;
    if (G < 1 || G > OSD_MAX_SHARDS || shard < 0 || shard >= G) return OSD_ERR_INVALID_ARG;
    if (v_begin < 0 || int64_t(v_begin) + V_shard > kMaxShardedVocab) return OSD_ERR_INVALID_ARG;
    if (temperature > 0.0f && (!draft_shard || !u_resample)) return OSD_ERR_INVALID_ARG;
    if (!mass_all || !aligned8(mass_all) || !accepted_len || !out_tokens) return OSD_ERR_INVALID_ARG;
    osd::ShardLaunch L = shard_launch(3, target_shard, draft_shard, dtype, B, K, V_shard, temperature,
                                      draft_tokens, draft_len, stream);
    L.v_begin = v_begin;
    L.G = G;
    L.shard = shard;
    L.u_resample = u_resample;
    L.mass_in = mass_all;
    L.accepted_len = accepted_len;
    L.out_tokens = out_tokens;
    L.reject_mask = reject_mask;
    return osd::launch_verify_shard(L) == hipSuccess ? OSD_OK : OSD_ERR_DEVICE;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Allocation-free verification.  The scratch of osd_verify (arrival counters,
// per-row records, greedy argmax partials) lives in a device array that the
// library holds for the life of the process, one copy per GPU.  In host code
// `scratch` names a host-side stand-in, not device memory: its device address
// on each GPU comes from hipGetSymbolAddress, taken once per device with that
// device current, and only that address is handed to kernels.
// ---------------------------------------------------------------------------
namespace {

static __device__ __align__(256) unsigned char scratch[OSD_VERIFY_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

// The device address of `scratch` on device dev (nullptr on failure).
void* scratch_on(int dev) {
    if (dev < 0 || dev >= kMaxDevices) return nullptr;
    std::call_once(g_scratch_once[dev], [dev] {
        int cur = -1;
        hipError_t e = hipGetDevice(&cur);
        if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
        void* ptr = nullptr;
        if (e == hipSuccess) e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur >= 0 && cur != dev) (void)hipSetDevice(cur);
        g_scratch_err[dev] = e;
        g_scratch_ptr[dev] = e == hipSuccess ? ptr : nullptr;
    });
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" int osd_verify_noalloc(const void* target_logits, const void* draft_logits, int dtype, int B, int K,
                                  int V, const int32_t* draft_tokens, const int32_t* draft_len,
                                  const float* u_accept, const float* u_resample, float temperature,
                                  int32_t* accepted_len, int32_t* out_tokens, uint8_t* reject_mask,
                                  void* stream) {
    // Argument checks first (nothing is enqueued on an error), then the size.
    if (dtype != OSD_F32 && dtype != OSD_BF16) return OSD_ERR_INVALID_ARG;
    if (B <= 0 || K <= 0 || V <= 0 || K > OSD_MAX_K) return OSD_ERR_INVALID_ARG;
    if (!sizes_ok(B, K, V, dtype)) return OSD_ERR_UNSUPPORTED;
    if (!(temperature >= 0.0f) || isinf(temperature)) return OSD_ERR_INVALID_ARG;
    if (!target_logits || !draft_tokens || !accepted_len || !out_tokens) return OSD_ERR_INVALID_ARG;
    if (temperature > 0.0f && (!draft_logits || !u_accept || !u_resample)) return OSD_ERR_INVALID_ARG;
    const VerifyWs ws = verify_layout(B, K);
    if (ws.total > size_t(OSD_VERIFY_NOALLOC_SCRATCH_BYTES)) return OSD_ERR_SCRATCH;

    hipStream_t s = static_cast<hipStream_t>(stream);
    int dev = 0;
    if (s == nullptr || hipStreamGetDevice(s, &dev) != hipSuccess) {
        if (hipGetDevice(&dev) != hipSuccess) return OSD_ERR_DEVICE;
    }
    void* ptr = scratch_on(dev);
    if (!ptr) return OSD_ERR_DEVICE;
    // The counters and records must start at zero.  osd_verify's kernels
    // leave them zero, but the array keeps whatever the previous call on this
    // GPU left, so they are cleared here on the call's own stream.  (The
    // greedy partials are written before they are read.)
    if (launch_clear_words(static_cast<uint32_t*>(ptr), int(ws.stats / 4), s) != hipSuccess) return OSD_ERR_DEVICE;
    return osd_verify(target_logits, draft_logits, dtype, B, K, V, draft_tokens, draft_len, u_accept, u_resample,
                      temperature, accepted_len, out_tokens, reject_mask, ptr, ws.total, stream);
}

// ---------------------------------------------------------------------------
// Multi-candidate (tree) verification.
// ---------------------------------------------------------------------------
namespace {

struct TreeWs {
    size_t counters, records, total;
};
TreeWs tree_layout(int B, int N) {
    TreeWs w;
    w.counters = 0;
    w.records = round_up(size_t(B) * 4, kAlign);
    w.total = w.records + round_up(size_t(B) * size_t(N) * 4, kAlign);
    return w;
}

}  // namespace

extern "C" {

size_t osd_verify_tree_workspace_bytes(int B, int N) {
    if (B <= 0 || N <= 0 || N > OSD_MAX_TREE_NODES) return 0;
    if (int64_t(B) * int64_t(N) > 0x7FFFFFFFll) return 0;
    return tree_layout(B, N).total;
}

int osd_verify_tree(const void* target_logits, const void* draft_logits, int dtype, int B, int N, int V,
                    const int32_t* parent, const int32_t* node_tokens, const float* u_accept,
                    const float* u_resample, float temperature, int32_t* accepted_len, int32_t* out_tokens,
                    int32_t* path_nodes, void* workspace, size_t workspace_bytes, void* stream) {
    if (dtype != OSD_F32 && dtype != OSD_BF16) return OSD_ERR_INVALID_ARG;
    if (B <= 0 || N <= 0 || V <= 0 || N > OSD_MAX_TREE_NODES) return OSD_ERR_INVALID_ARG;
    if (int64_t(B) * int64_t(N) > 0x7FFFFFFFll) return OSD_ERR_INVALID_ARG;
    osd::RowTile t;
    if (!osd::pick_tree_tile(V, per_chunk(dtype), &t)) return OSD_ERR_UNSUPPORTED;
    if (!(temperature >= 0.0f) || isinf(temperature)) return OSD_ERR_INVALID_ARG;
    const bool greedy = temperature == 0.0f;
    if (!target_logits || !parent || !node_tokens || !accepted_len || !out_tokens) return OSD_ERR_INVALID_ARG;
    if (!greedy && (!draft_logits || !u_accept || !u_resample)) return OSD_ERR_INVALID_ARG;
    const TreeWs ws = tree_layout(B, N);
    if (!workspace || workspace_bytes < ws.total || (reinterpret_cast<uintptr_t>(workspace) & 15u))
        return OSD_ERR_WORKSPACE;
    osd::TreeLaunch L;
    L.target = target_logits;
    L.draft = greedy ? nullptr : draft_logits;
    L.dtype = dtype;
    L.B = B;
    L.N = N;
    L.V = V;
    L.parent = parent;
    L.node_tokens = node_tokens;
    L.u_accept = u_accept;
    L.u_resample = u_resample;
    L.temperature = temperature;
    L.accepted_len = accepted_len;
    L.out_tokens = out_tokens;
    L.path_nodes = path_nodes;
    char* w = static_cast<char*>(workspace);
    L.counters = reinterpret_cast<uint32_t*>(w + ws.counters);
    L.records = reinterpret_cast<uint32_t*>(w + ws.records);
    L.vec = (int64_t(V) * elem_bytes(dtype)) % 16 == 0 && aligned16(target_logits) &&
            (greedy || aligned16(draft_logits));
    L.stream = static_cast<hipStream_t>(stream);
    L.cus = device_cus(L.stream);
    return osd::launch_verify_tree(L) == hipSuccess ? OSD_OK : OSD_ERR_DEVICE;
}

}  // extern "C"
