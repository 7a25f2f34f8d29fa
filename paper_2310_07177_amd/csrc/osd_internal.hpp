// osd_internal.hpp -- host-side launch interface between the C ABI layer and
// the kernel translation units.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "osd.h"

namespace osd {

template <typename T>
struct same_type {
    using type = T;
};

// Enqueue kernel<<<grid, block, lds, stream>>>(args...) and return the status
// of this launch alone (hipGetLastError would also report an earlier failure
// of some other call made by the same thread).
template <typename... P>
inline hipError_t launch_kernel(void (*kernel)(P...), dim3 grid, dim3 block, size_t lds, hipStream_t stream,
                                typename same_type<P>::type... args) {
    void* ptrs[] = {static_cast<void*>(&args)..., nullptr};
    return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, lds, stream);
}

// Kernel tile shape chosen from V: W threads per workgroup, CPT 16-byte chunks
// per thread per row.
struct RowTile {
    int W;
    int CPT;
};

// Occupancy target of a row-resident tile (waves per SIMD the compiler must
// leave room for): 4, i.e. up to 128 VGPRs -- two 512-thread workgroups or
// one 1024-thread workgroup per CU.  (Eight waves per SIMD would cap a wave at
// 64 VGPRs, and the spills that forces cost more than the occupancy gains.)
constexpr int min_waves_per_simd(int W, int CPT) { return (void)W, (void)CPT, 4; }

// Argmax partial of one vocabulary segment of a target row (segmented greedy
// verification): (max, lowest index) in (kt, kd's bits).
struct SegStats {
    double st, sd;
    float kt, kd;
};
// Segments per row in the segmented greedy kernels (at most).
constexpr int kMaxSeg = 16;

struct VerifyLaunch {
    const void* target;
    const void* draft;
    int dtype;  // 0 fp32, 1 bf16
    int B, K, V;
    const int32_t* tokens;
    const int32_t* draft_len;
    const float* u_accept;
    const float* u_resample;
    float temperature;
    int32_t* accepted_len;
    int32_t* out_tokens;
    uint8_t* reject_mask;
    uint32_t* records;   // [B*(K+1)] zero on entry and exit
    uint32_t* counters;  // [B]       zero on entry and exit
    SegStats* seg_stats;  // [B*(K+1)*kMaxSeg] greedy argmax partials, zero on entry and exit
    bool vec;            // rows 16-byte aligned
    hipStream_t stream;
};

struct DistillLaunch {
    const void* teacher;
    int64_t teacher_stride;
    const void* student;
    int64_t student_stride;
    int dtype;
    int B, K, V;
    const uint8_t* mask;
    int kind;
    float beta, tau;
    float* loss_out;
    float* row_loss_out;
    void* grad_out;
    void* split_ws;            // rows longer than the resident tiles: per-segment records, zero on entry and exit
    double* row_loss_ws;       // [B*K]
    double* slab_ws;           // [nslabs]
    uint32_t* slab_counters;   // [nslabs] zero on entry and exit
    uint32_t* done_counter;    // [1]      zero on entry and exit
    bool vec;
    int cus;
    hipStream_t stream;
};

constexpr int kSlabRows = 64;
// Segments per row of the split distillation (16 x 8192 bf16 or 16 x 4096 fp32
// logits) and the workspace bytes per row they take: a 24-byte record and two
// fp64 partials per segment, and four 32-bit counters.
constexpr int kMaxSplitSegments = 16;
constexpr size_t kSplitBytesPerRow = size_t(kMaxSplitSegments) * (24 + 16) + 16;
// Row counts up to this are reduced in one level (see distill.hip).
constexpr int kOneLevelRows = 1024;

// Largest V handled by the row-resident tiles for a chunk of `per_chunk`
// elements.
int max_vocab_for(int per_chunk);
bool pick_tile(int V, int per_chunk, RowTile* t);

hipError_t launch_verify(const VerifyLaunch& L);
hipError_t launch_distill(const DistillLaunch& L);

// Segmented greedy verification: rows whose byte length and base are
// 16-byte multiples.  Segments per row for V (false: V too large).
bool greedy_segments(int V, int per_chunk, int* nseg);
hipError_t launch_verify_greedy(const VerifyLaunch& L);

// Fused verification + distillation of one step (streaming layout), the
// distillation at the verification temperature: teacher = target rows
// 0..K-1, student = draft rows.
struct FusedLaunch {
    const void* target;
    const void* draft;
    int dtype;
    int B, K, V;
    const int32_t* tokens;
    const int32_t* draft_len;
    const float* u_accept;
    const float* u_resample;
    float temperature;
    const uint8_t* mask;  // distillation mask [B, K] or null
    int kind;
    float beta;
    int32_t* accepted_len;
    int32_t* out_tokens;
    uint8_t* reject_mask;
    float* loss_out;
    float* row_loss_out;
    void* grad_out;
    uint32_t* records;  // [B*(K+1)]     zero on entry and exit
    uint32_t* dec;      // [B*(K+1)]     zero on entry and exit
    int erridx;         // distil each sequence's first rejected row instead of `mask`
    double* part_ws;    // [B*(K+1)]     zero on entry and exit
    uint32_t* done;     // [1]           zero on entry and exit
    int cus;
    hipStream_t stream;
};
hipError_t launch_verify_distill(const FusedLaunch& L);

// Multi-candidate (tree) verification: one workgroup per (sequence, node).
struct TreeLaunch {
    const void* target;  // [B, N, V]
    const void* draft;   // [B, N, V]
    int dtype;
    int B, N, V;
    const int32_t* parent;
    const int32_t* node_tokens;
    const float* u_accept;
    const float* u_resample;
    float temperature;
    int32_t* accepted_len;
    int32_t* out_tokens;
    int32_t* path_nodes;
    uint32_t* records;   // [B*N] zero on entry and exit
    uint32_t* counters;  // [B]   zero on entry and exit
    bool vec;
    int cus;  // compute units of the device
    hipStream_t stream;
};
bool pick_tree_tile(int V, int per_chunk, RowTile* t);
hipError_t launch_verify_tree(const TreeLaunch& L);

// Token sampling: one workgroup per row, pi = beta softmax(p/T) +
// (1 - beta) softmax(q/T) (a row with weight 0 is not read); T == 0 takes
// the argmax of the row with weight 1.
struct SampleLaunch {
    const void* p;
    int64_t p_stride;  // elements
    const void* q;
    int64_t q_stride;
    int dtype;
    int N, V;
    float temperature;
    float beta;
    const float* u;
    int32_t* out;
    bool vec;  // every row 16-byte aligned and V a whole number of chunks
    int cus;
    void* workspace;  // null, or sample_workspace_bytes(N) zeroed bytes: rows split over workgroups
    hipStream_t stream;
};
hipError_t launch_sample(const SampleLaunch& L);
// Workspace of the split sampling: per row, 16 segment records of 16 bytes
// and a 16-byte counter slot.
constexpr size_t kSampleWsPerRow = 16 * 16 + 16;

// Streaming (persistent-workgroup) distillation: rows whose byte length and
// base are 16-byte multiples and whose V fits one of the streaming tiles.
bool pick_stream_tile(int V, int per_chunk, RowTile* t);
hipError_t launch_distill_stream(const DistillLaunch& L);

// Vocabulary-sharded verification, one phase per call (1 stats, 2 mass,
// 3 draw).  Records are the public osd_shard_row_stats / osd_shard_mass.
struct ShardLaunch {
    int phase;
    const void* target;  // this rank's slice [B, K+1, Vs]
    const void* draft;   // [B, K, Vs]
    int dtype;
    int B, K, Vs, v_begin, V, G, shard;
    const int32_t* tokens;
    const int32_t* draft_len;
    const float* u_accept;
    const float* u_resample;
    float temperature;
    osd_shard_row_stats* stats;          // phase 1 out [B, K+1]
    const osd_shard_row_stats* stats_in;  // phase 2 in [G, B, K+1]
    osd_shard_mass* mass;                 // phase 2 out [B]
    const osd_shard_mass* mass_in;        // phase 3 in [G, B]
    int32_t* accepted_len;
    int32_t* out_tokens;
    uint8_t* reject_mask;
    bool vec;
    hipStream_t stream;
};
hipError_t launch_verify_shard(const ShardLaunch& L);

}  // namespace osd
