// read_ceiling.hip -- a pure-read kernel used by the benchmark to measure what
// one launch that only reads a buffer of a given size achieves on this GPU
// (the ceiling the path's kernels are compared with, beside the 8 TB/s
// peak).  Not part of libosd: it is built into its own small library.
//
// Each thread reads 16-byte chunks of the buffer with non-temporal loads,
// UNROLL chunks in flight, in a grid-stride loop, and folds them into one
// word; one word per workgroup is written so that nothing is optimised away.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t chunk_t __attribute__((ext_vector_type(4)));

template <int UNROLL>
__global__ __launch_bounds__(256) void read_kernel(const chunk_t* p, int64_t nchunks, uint32_t* sink) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    uint32_t acc = 0u;
    for (; i + (UNROLL - 1) * stride < nchunks; i += UNROLL * stride) {
        chunk_t v[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < nchunks; i += stride) {
        const chunk_t v = __builtin_nontemporal_load(p + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    // one word per workgroup (the fold of every lane's word)
    __shared__ uint32_t s_acc;
    if (threadIdx.x == 0) s_acc = 0u;
    __syncthreads();
    atomicXor(&s_acc, acc);
    __syncthreads();
    if (threadIdx.x == 0) sink[blockIdx.x] = s_acc;
}

}  // namespace

// Read `bytes` (a multiple of 16, 16-byte aligned) from `buf` with `blocks`
// workgroups of 256 threads and `unroll` (1, 2, 4 or 8) chunks in flight per
// thread; `sink` holds `blocks` words.  Returns 0 when enqueued.
extern "C" int osd_probe_read(const void* buf, int64_t bytes, int blocks, int unroll, uint32_t* sink,
                              void* stream) {
    if (!buf || !sink || bytes <= 0 || (bytes & 15) || blocks <= 0) return -1;
    const chunk_t* p = static_cast<const chunk_t*>(buf);
    const int64_t n = bytes / 16;
    hipStream_t s = static_cast<hipStream_t>(stream);
    void* args[] = {&p, const_cast<int64_t*>(&n), &sink};
    const void* k;
    switch (unroll) {
        case 1: k = reinterpret_cast<const void*>(&read_kernel<1>); break;
        case 2: k = reinterpret_cast<const void*>(&read_kernel<2>); break;
        case 4: k = reinterpret_cast<const void*>(&read_kernel<4>); break;
        case 8: k = reinterpret_cast<const void*>(&read_kernel<8>); break;
        default: return -1;
    }
    return hipLaunchKernel(k, dim3(blocks), dim3(256), args, 0, s) == hipSuccess ? 0 : -3;
}
