// probe.hip -- measurement aids for the benchmark (not part of the attention
// path): the HBM read bandwidth the device reaches with a plain streaming
// kernel, the rate at which one CU reads L2-resident data, the cost of an
// empty launch, and the latency of the memory operations a cross-workgroup
// hand-off is built from.  The decode kernels'
// fractions of peak are reported against the published 8 TB/s and against the
// streaming figure measured here.
#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

// Streaming read: workgroup w reads its own contiguous range of the buffer,
// every thread keeping 8 nontemporal 16-byte loads in flight (consecutive
// threads on consecutive 16-byte chunks); the xor of the data decides a store
// that never happens in practice, which keeps the loads alive.
__global__ __launch_bounds__(256) void stream_read_kernel(const uint4 *src, size_t n16, unsigned *sink) {
    typedef unsigned u4v __attribute__((ext_vector_type(4)));
    const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
    const size_t lo = (size_t)blockIdx.x * per;
    const size_t hi = lo + per < n16 ? lo + per : n16;
    uint32_t acc = 0;
    for (size_t base = lo + threadIdx.x; base < hi; base += 8 * 256) {
        u4v v[8];
        #pragma unroll
        for (int i = 0; i < 8; ++i) {
            const size_t idx = base + (size_t)i * 256;
            v[i] = idx < hi ? __builtin_nontemporal_load(reinterpret_cast<const u4v *>(src + idx)) : u4v{0u, 0u, 0u, 0u};
        }
        #pragma unroll
        for (int i = 0; i < 8; ++i) acc ^= v[i].x ^ v[i].y ^ v[i].z ^ v[i].w;
    }
    if (acc == 0x9e3779b9u && sink) sink[0] = acc;
}

// Shared read: every workgroup reads the same bytes (16-byte loads into
// registers, consecutive threads on consecutive 16 bytes, 16 loads in flight
// per thread).  After the first touch the data is L2-resident, so the time
// per launch gives the rate at which one CU pulls L2-resident data, by the
// number of waves of its workgroup.
__global__ __launch_bounds__(1024) void shared_read_kernel(const uint4 *src, size_t n16, unsigned *sink) {
    typedef unsigned u4v __attribute__((ext_vector_type(4)));
    const size_t nt = blockDim.x;
    uint32_t acc = 0;
    for (size_t base = threadIdx.x; base < n16; base += 16 * nt) {
        u4v v[16];
        #pragma unroll
        for (int i = 0; i < 16; ++i) {
            const size_t idx = base + (size_t)i * nt;
            v[i] = idx < n16 ? *reinterpret_cast<const u4v *>(src + idx) : u4v{0u, 0u, 0u, 0u};
        }
        #pragma unroll
        for (int i = 0; i < 16; ++i) acc ^= v[i].x ^ v[i].y ^ v[i].z ^ v[i].w;
    }
    if (acc == 0x9e3779b9u && sink) sink[0] = acc;
}

__global__ void empty_kernel() {}

// One thread times each primitive with the shader clock, on a fresh 256-byte
// line per repetition; the value of every load or atomic is awaited before the
// second clock read.  Row k of `cycles` ([8][reps]) holds kind k.
__device__ __forceinline__ unsigned long long clk() { return __builtin_readcyclecounter(); }
__device__ __forceinline__ unsigned landed(unsigned x) {
    asm volatile("s_waitcnt vmcnt(0)" : "+v"(x)::"memory");
    return x;
}
__global__ void handoff_latency_kernel(unsigned *buf, unsigned long long *cycles, int reps) {
    if (threadIdx.x != 0) return;
    unsigned sink = 0;
    for (int r = 0; r < reps; ++r) {
        unsigned *q = buf + (size_t)r * 64;
        unsigned long long *o = cycles + r, t0, t1;
        t0 = clk(); q[0] = r; __builtin_amdgcn_s_waitcnt(0x0f70); t1 = clk(); o[0 * (size_t)reps] = t1 - t0;
        t0 = clk(); __hip_atomic_store(q + 1, (unsigned)r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __builtin_amdgcn_s_waitcnt(0x0f70); t1 = clk(); o[1 * (size_t)reps] = t1 - t0;
        t0 = clk(); sink += landed(__hip_atomic_fetch_add(q + 2, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        t1 = clk(); o[2 * (size_t)reps] = t1 - t0;
        t0 = clk(); sink += landed(__hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        t1 = clk(); o[3 * (size_t)reps] = t1 - t0;
        t0 = clk(); sink += landed(*(volatile unsigned *)(q + 0)); t1 = clk(); o[4 * (size_t)reps] = t1 - t0;
        t0 = clk(); sink += landed(*(volatile unsigned *)(q + 32)); t1 = clk(); o[5 * (size_t)reps] = t1 - t0;
        o[6 * (size_t)reps] = __builtin_amdgcn_s_memrealtime();
        o[7 * (size_t)reps] = clk();
    }
    if (sink == 0x9e3779b9u) cycles[0] = sink;
}

}  // namespace mad

extern "C" {

int mad_probe_stream_read(const void *src, size_t bytes, unsigned *sink, int n_workgroups, void *stream) {
    if (!src || bytes < 16 || bytes % 16 || ((uintptr_t)src & 15u) || n_workgroups < 1) return MAD_EINVAL;
    hipLaunchKernelGGL(mad::stream_read_kernel, dim3((unsigned)n_workgroups), dim3(256), 0, (hipStream_t)stream,
                       reinterpret_cast<const uint4 *>(src), bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? MAD_OK : MAD_EHIP;
}

int mad_probe_shared_read(const void *src, size_t bytes, unsigned *sink, int n_workgroups, int threads,
                          void *stream) {
    if (!src || bytes < 16 || bytes % 16 || ((uintptr_t)src & 15u) || n_workgroups < 1 || threads < 64 ||
        threads > 1024 || threads % 64)
        return MAD_EINVAL;
    hipLaunchKernelGGL(mad::shared_read_kernel, dim3((unsigned)n_workgroups), dim3((unsigned)threads), 0,
                       (hipStream_t)stream, reinterpret_cast<const uint4 *>(src), bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? MAD_OK : MAD_EHIP;
}

int mad_probe_empty(int n_workgroups, int threads, void *stream) {
    if (n_workgroups < 1 || threads < 1 || threads > 1024) return MAD_EINVAL;
    hipLaunchKernelGGL(mad::empty_kernel, dim3((unsigned)n_workgroups), dim3((unsigned)threads), 0,
                       (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? MAD_OK : MAD_EHIP;
}

int mad_probe_handoff_latency(void *buf, size_t buf_bytes, unsigned long long *cycles, int reps, void *stream) {
    if (!buf || !cycles || reps < 2 || buf_bytes < (size_t)reps * 256 + 256) return MAD_EINVAL;
    hipLaunchKernelGGL(mad::handoff_latency_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream,
                       reinterpret_cast<unsigned *>(buf), cycles, reps);
    return hipGetLastError() == hipSuccess ? MAD_OK : MAD_EHIP;
}

}  // extern "C"
