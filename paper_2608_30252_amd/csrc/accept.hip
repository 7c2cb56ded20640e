// accept.hip -- greedy accept/reject (Sec. 2.1; greedy decoding, Sec. 4.1).
//
// For every sequence b: am[t] = argmax_v logits[b][t][v]; the drafted tokens
// are accepted up to the first t with draft[b][t] != am[t]; the target's
// token at that position (a correction, or the bonus token when everything
// was accepted) is emitted next.
//
// Argmax is made exact and independent of reduction order by mapping each
// (value, index) to one 64-bit key: an order-preserving 32-bit image of the
// float (NaN above +inf, -0 folded into +0) in the high word and the inverted
// index in the low word.  The row argmax is then the maximum key: ties go to
// the lowest index, the first NaN wins.
//
// One launch: workgroup (chunk, row) reduces a chunk of the vocabulary; the
// last chunk of a row (arrival counter) reduces the row; the last row to
// finish applies the accept rule for every sequence.
#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

__device__ __forceinline__ uint64_t argmax_key(float x, int idx) {
    uint32_t u = __float_as_uint(x);
    uint32_t ord;
    if ((u & 0x7fffffffu) > 0x7f800000u) ord = 0xffffffffu;      // NaN: above everything
    else if ((u & 0x7fffffffu) == 0u) ord = 0x80000000u;         // +0 and -0 compare equal
    else ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((uint64_t)ord << 32) | (uint64_t)(0xffffffffu - (uint32_t)idx);
}
__device__ __forceinline__ int key_index(uint64_t k) { return (int)(0xffffffffu - (uint32_t)k); }

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    const int lo = __shfl_xor((int)(uint32_t)v, m, 64);
    const int hi = __shfl_xor((int)(uint32_t)(v >> 32), m, 64);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
    #pragma unroll
    for (int m = 1; m < 64; m <<= 1) {
        const uint64_t o = shfl_xor_u64(v, m);
        v = o > v ? o : v;
    }
    return v;
}
__device__ __forceinline__ void store_agent_u64(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t load_agent_u64(const uint64_t *p) {
    return __hip_atomic_load(const_cast<uint64_t *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename T>
__global__ __launch_bounds__(256) void accept_kernel(const AcceptArgs a) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rows = a.B * a.T;
    const int row = blockIdx.x % rows, chunk = blockIdx.x / rows;
    const int v0 = chunk * kAcceptChunk;
    const int v1 = min(a.V, v0 + kAcceptChunk);
    const T *x = reinterpret_cast<const T *>(a.logits) + (size_t)row * a.V;

    uint64_t best = 0;   // below every real key (index 0xffffffff is never used)
    constexpr int VEC = Elem<T>::VEC;                   // elements per 16-byte load
    constexpr int NV = kAcceptChunk / (256 * VEC);      // 16-byte loads per thread per chunk
    if (a.vec16) {
        // rows start on 16-byte boundaries and V is a multiple of VEC: every
        // load of the chunk is issued before any is used
        uint4 v[NV];
        #pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int e = v0 + (tid + 256 * k) * VEC;
            v[k] = e < v1 ? *reinterpret_cast<const uint4 *>(x + e) : make_uint4(0u, 0u, 0u, 0u);
        }
        #pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int e = v0 + (tid + 256 * k) * VEC;
            if (e < v1) {
                float f[VEC];
                unpack16(v[k], f, T());
                #pragma unroll
                for (int q = 0; q < VEC; ++q) {
                    const uint64_t key = argmax_key(f[q], e + q);
                    best = key > best ? key : best;
                }
            }
        }
    } else {
        for (int i = v0 + tid; i < v1; i += 256) {
            const uint64_t k = argmax_key(Elem<T>::load1(x + i), i);
            best = k > best ? k : best;
        }
    }
    best = wave_max_u64(best);
    __shared__ uint64_t s_w[4];
    __shared__ int s_flag;
    if (lane == 0) s_w[wave] = best;
    __syncthreads();
    if (tid == 0) {
        uint64_t m = s_w[0];
        for (int w = 1; w < 4; ++w) m = s_w[w] > m ? s_w[w] : m;
        store_agent_u64(a.part + (size_t)row * a.n_chunks + chunk, m);
    }
    wait_vm_stores();
    __syncthreads();
    if (tid == 0) {
        unsigned *cnt = a.counters + (size_t)row * kCounterStride;
        const int last = arrive(cnt) == (unsigned)(a.n_chunks - 1);
        if (last) reset_counter(cnt);
        s_flag = last;
    }
    __syncthreads();
    if (!s_flag) return;

    // ---- last chunk of this row: reduce the row ----
    uint64_t rb = 0;
    for (int c = tid; c < a.n_chunks; c += 256) {
        const uint64_t k = load_agent_u64(a.part + (size_t)row * a.n_chunks + c);
        rb = k > rb ? k : rb;
    }
    rb = wave_max_u64(rb);
    if (lane == 0) s_w[wave] = rb;
    __syncthreads();
    if (tid == 0) {
        uint64_t m = s_w[0];
        for (int w = 1; w < 4; ++w) m = s_w[w] > m ? s_w[w] : m;
        store_agent_u64(a.row_best + row, m);
    }
    wait_vm_stores();
    __syncthreads();
    if (tid == 0) {
        unsigned *cnt = a.counters + (size_t)rows * kCounterStride;
        const int last = arrive(cnt) == (unsigned)(rows - 1);
        if (last) reset_counter(cnt);
        s_flag = last;
    }
    __syncthreads();
    if (!s_flag) return;

    // ---- last row overall: the accept rule for every sequence ----
    for (int b = tid; b < a.B; b += 256) {
        int acc = 0;
        const uint64_t *rbp = a.row_best + (size_t)b * a.T;
        while (acc < a.T - 1 && a.draft[(size_t)b * (a.T - 1) + acc] == key_index(load_agent_u64(rbp + acc))) ++acc;
        a.n_accept[b] = acc;
        a.next_tok[b] = key_index(load_agent_u64(rbp + acc));
    }
}

// ------------------------------------------------------------------ host ----

size_t accept_ws_bytes(int B, int T, int V) {
    const size_t rows = (size_t)B * T;
    const size_t chunks = ((size_t)V + kAcceptChunk - 1) / kAcceptChunk;
    return kCounterRegionBytes + align256(rows * chunks * 8) + align256(rows * 8);
}

void accept_ws_layout(int B, int T, int V, size_t *off_part, size_t *off_rows) {
    const size_t rows = (size_t)B * T;
    const size_t chunks = ((size_t)V + kAcceptChunk - 1) / kAcceptChunk;
    *off_part = kCounterRegionBytes;
    *off_rows = kCounterRegionBytes + align256(rows * chunks * 8);
}

hipError_t launch_accept(const AcceptArgs &a, int dtype, hipStream_t st) {
    dim3 grid((unsigned)(a.B * a.T * a.n_chunks)), block(256);
    if (dtype == MAD_BF16) hipLaunchKernelGGL(accept_kernel<bf16_t>, grid, block, 0, st, a);
    else hipLaunchKernelGGL(accept_kernel<float>, grid, block, 0, st, a);
    return hipGetLastError();
}

}  // namespace mad
