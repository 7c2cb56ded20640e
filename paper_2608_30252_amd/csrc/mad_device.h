// mad_device.h -- small device helpers shared by the libmad kernels (gfx950).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mad {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// bf16 is carried as raw uint16_t bits; conversions are written out.
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// fp32 -> bf16, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// The same rounding (nearest even) by the hardware conversion, one instruction
// for two values; for finite inputs it equals pack_bf16x2.
typedef __bf16 bf16x2_cvt_v __attribute__((ext_vector_type(2)));
typedef float f32x2_cvt_v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_cvt_v{lo, hi}), bf16x2_cvt_v));
}

// Element type traits: T = float or bf16_t; a 16-byte vector holds VEC elements.
template <typename T> struct Elem;
template <> struct Elem<float> {
    static constexpr int VEC = 4;
    __device__ __forceinline__ static float load1(const float *p) { return *p; }
    __device__ __forceinline__ static void store1(float *p, float v) { *p = v; }
};
template <> struct Elem<bf16_t> {
    static constexpr int VEC = 8;
    __device__ __forceinline__ static float load1(const bf16_t *p) { return bf16_to_f32(p->bits); }
    __device__ __forceinline__ static void store1(bf16_t *p, float v) { p->bits = f32_to_bf16(v); }
};

// Unpack a 16-byte vector into fp32 values.
__device__ __forceinline__ void unpack16(const uint4 &u, float (&f)[4], float) {
    f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y);
    f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
}
__device__ __forceinline__ void unpack16(const uint4 &u, float (&f)[8], bf16_t) {
    f[0] = bf16_lo(u.x); f[1] = bf16_hi(u.x); f[2] = bf16_lo(u.y); f[3] = bf16_hi(u.y);
    f[4] = bf16_lo(u.z); f[5] = bf16_hi(u.z); f[6] = bf16_lo(u.w); f[7] = bf16_hi(u.w);
}

// Cross-lane exchange inside a wave64, all on the vector ALU (no LDS
// crossbar).  Patterns 1 and 2 use DPP quad permutes, 4 and 8 use DPP row
// mirrors (valid for sum/max reductions over aligned groups); across 16 and
// 32 lanes the gfx950 lane swaps v_permlane16_swap / v_permlane32_swap give
// every lane the values of lanes l & ~X and l | X (pair_sum, pair_max).
template <int X> __device__ __forceinline__ float xor_lane(float v);
template <> __device__ __forceinline__ float xor_lane<1>(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, true));
}
template <> __device__ __forceinline__ float xor_lane<2>(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, true));
}
// row_half_mirror: lane i of each 8-lane half row <-> lane 7-i.  After the
// groups of 4 are reduced this pairs every lane with the other quad.
template <> __device__ __forceinline__ float xor_lane<4>(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xF, 0xF, true));
}
// row_mirror: lane i of each 16-lane row <-> lane 15-i (pairs the two halves of
// the row once each half is reduced).
template <> __device__ __forceinline__ float xor_lane<8>(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xF, 0xF, true));
}
// v + v[l ^ X] for X = 16 or 32, the operands in the same order in both lanes
// of a pair (the two lanes' results are bitwise equal)
template <int X> __device__ __forceinline__ float pair_sum(float v) {
    if constexpr (X == 16) {
        const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        return __uint_as_float(p[0]) + __uint_as_float(p[1]);
    } else {
        const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        return __uint_as_float(p[0]) + __uint_as_float(p[1]);
    }
}
template <int X> __device__ __forceinline__ float pair_max(float v) {
    if constexpr (X == 16) {
        const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
    } else {
        const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
    }
}

// Reduce over aligned groups of N consecutive lanes (N a power of two <= 64).
// Valid only as an all-reduce of a commutative, associative op when applied
// from the smallest pattern upward (the mirrors rely on it).
template <int N> __device__ __forceinline__ float group_sum(float v) {
    if constexpr (N >= 2) v += xor_lane<1>(v);
    if constexpr (N >= 4) v += xor_lane<2>(v);
    if constexpr (N >= 8) v += xor_lane<4>(v);
    if constexpr (N >= 16) v += xor_lane<8>(v);
    if constexpr (N >= 32) v = pair_sum<16>(v);
    if constexpr (N >= 64) v = pair_sum<32>(v);
    return v;
}
template <int N> __device__ __forceinline__ float group_max(float v) {
    if constexpr (N >= 2) v = fmaxf(v, xor_lane<1>(v));
    if constexpr (N >= 4) v = fmaxf(v, xor_lane<2>(v));
    if constexpr (N >= 8) v = fmaxf(v, xor_lane<4>(v));
    if constexpr (N >= 16) v = fmaxf(v, xor_lane<8>(v));
    if constexpr (N >= 32) v = pair_max<16>(v);
    if constexpr (N >= 64) v = pair_max<32>(v);
    return v;
}

// Rotate-half RoPE: theta_j = base^(-2j/d) in double precision (a kernel may
// tabulate it), the angle pos * theta_j formed and reduced modulo 2 pi in double
// precision (Cody-Waite with a two-part 2 pi), its sine and cosine taken in
// single precision on the reduced angle in [-pi, pi].
__device__ __forceinline__ double rope_theta(int j, int d, double log2_base) {
    return exp2(-2.0 * (double)j / (double)d * log2_base);
}
// a - n * 2 pi with n = rint(a / (2 pi)): 2 pi split as hi + lo, hi the double
// nearest 2 pi and lo the double nearest 2 pi - hi.  The inner fma forms
// a - n * hi with a single rounding (its product is exact inside the fma), the
// outer one subtracts n * lo, so the reduced angle is within a few ulps of the
// exact a - n * 2 pi for every angle a position id reaches.
__host__ __device__ inline double rope_reduce(double a) {
    const double n = rint(a * 0.15915494309189535);            // 1 / (2 pi)
    return fma(-n, 2.4492935982947064e-16, fma(-n, 6.283185307179586, a));
}
// The rotation in two parts, so that a kernel can take the cosine and sine
// before the pair is known; the products are fused explicitly so that every
// kernel rounds the rotation the same way.
__device__ __forceinline__ void rope_cs(int pos, double theta, float *c, float *s) {
    const double r = rope_reduce((double)pos * theta);
    sincosf((float)r, s, c);
}
__device__ __forceinline__ void rope_apply(float y0, float y1, float c, float s, float *k0, float *k1) {
    *k0 = fmaf(y0, c, -(y1 * s));
    *k1 = fmaf(y1, c, y0 * s);
}
__device__ __forceinline__ void rope_rotate(float y0, float y1, int pos, double theta, float *k0, float *k1) {
    float c, s;
    rope_cs(pos, theta, &c, &s);
    rope_apply(y0, y1, c, s, k0, k1);
}

// ---- cross-workgroup hand-off without cache maintenance -------------------
// Split partials are written with agent-scope atomic stores (write-through to
// the device-coherent level, past the per-XCD L2), the writer waits for their
// completion (vmcnt(0)), and only then bumps the arrival counter.  The last
// arriving workgroup reads the partials with agent-scope atomic loads.  This
// is the ordering the memory model's own release sequence relies on, without
// its L2 writeback and -- worse for a streaming kernel -- the whole-L2
// invalidate that a full __threadfence() performs in every workgroup.
__device__ __forceinline__ void store_agent(float *p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Two adjacent floats (8-byte aligned) in one device-coherent store.
__device__ __forceinline__ void store_agent2(float *p, float a, float b) {
    const uint64_t v = (uint64_t)__float_as_uint(a) | ((uint64_t)__float_as_uint(b) << 32);
    __hip_atomic_store(reinterpret_cast<uint64_t *>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t load_agent64(const uint64_t *p) {
    return __hip_atomic_load(const_cast<uint64_t *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_agent(const float *p) {
    return __hip_atomic_load(const_cast<float *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void wait_vm_stores() { __builtin_amdgcn_s_waitcnt(0x0F70); /* vmcnt(0) */ }
// Keeps a wave-uniform pointer (as an integer) in SGPRs from this point on
// (the empty asm): the compiler neither re-reads the kernel argument it came
// from where it is used nor knows its address space afterwards, so the
// one-lane hand-off atomics through it are issued as flat atomics (the same
// agent-scope semantics) without the wave-reduction wrapper the compiler puts
// around a global atomic -- measured 0.09 us shorter on the decode arrival.
// The value must be wave-uniform; it is taken from the first active lane
// (readfirstlane returns int: each half goes through uint32_t, so the low
// half is never sign-extended into the high one).
__device__ __forceinline__ void pin_sgpr(uint64_t &v) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    v = ((uint64_t)hi << 32) | (uint64_t)lo;
    asm volatile("" : "+s"(v));
}
template <typename P> __device__ __forceinline__ uint64_t ptr_bits(P *p) { return (uint64_t)(uintptr_t)p; }
template <typename P> __device__ __forceinline__ P *bits_ptr(uint64_t v) { return reinterpret_cast<P *>((uintptr_t)v); }
__device__ __forceinline__ unsigned arrive(unsigned *counter) {
    return __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void reset_counter(unsigned *counter) {
    __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// s_waitcnt vmcnt(n), n in [0, 63] (gfx9 encoding: vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14)
__device__ __forceinline__ void wait_vm(int n) {
    switch (n) {
        case 0: __builtin_amdgcn_s_waitcnt(0x0f70); break;
        case 1: __builtin_amdgcn_s_waitcnt(0x0f71); break;
        case 2: __builtin_amdgcn_s_waitcnt(0x0f72); break;
        case 3: __builtin_amdgcn_s_waitcnt(0x0f73); break;
        case 4: __builtin_amdgcn_s_waitcnt(0x0f74); break;
        case 5: __builtin_amdgcn_s_waitcnt(0x0f75); break;
        case 6: __builtin_amdgcn_s_waitcnt(0x0f76); break;
        case 7: __builtin_amdgcn_s_waitcnt(0x0f77); break;
        case 8: __builtin_amdgcn_s_waitcnt(0x0f78); break;
        case 9: __builtin_amdgcn_s_waitcnt(0x0f79); break;
        case 10: __builtin_amdgcn_s_waitcnt(0x0f7a); break;
        case 11: __builtin_amdgcn_s_waitcnt(0x0f7b); break;
        case 12: __builtin_amdgcn_s_waitcnt(0x0f7c); break;
        case 13: __builtin_amdgcn_s_waitcnt(0x0f7d); break;
        case 14: __builtin_amdgcn_s_waitcnt(0x0f7e); break;
        case 15: __builtin_amdgcn_s_waitcnt(0x0f7f); break;
        case 16: __builtin_amdgcn_s_waitcnt(0x4f70); break;
        case 17: __builtin_amdgcn_s_waitcnt(0x4f71); break;
        case 18: __builtin_amdgcn_s_waitcnt(0x4f72); break;
        case 19: __builtin_amdgcn_s_waitcnt(0x4f73); break;
        case 20: __builtin_amdgcn_s_waitcnt(0x4f74); break;
        case 21: __builtin_amdgcn_s_waitcnt(0x4f75); break;
        case 22: __builtin_amdgcn_s_waitcnt(0x4f76); break;
        case 23: __builtin_amdgcn_s_waitcnt(0x4f77); break;
        case 24: __builtin_amdgcn_s_waitcnt(0x4f78); break;
        case 25: __builtin_amdgcn_s_waitcnt(0x4f79); break;
        case 26: __builtin_amdgcn_s_waitcnt(0x4f7a); break;
        case 27: __builtin_amdgcn_s_waitcnt(0x4f7b); break;
        case 28: __builtin_amdgcn_s_waitcnt(0x4f7c); break;
        case 29: __builtin_amdgcn_s_waitcnt(0x4f7d); break;
        case 30: __builtin_amdgcn_s_waitcnt(0x4f7e); break;
        case 31: __builtin_amdgcn_s_waitcnt(0x4f7f); break;
        case 32: __builtin_amdgcn_s_waitcnt(0x8f70); break;
        case 33: __builtin_amdgcn_s_waitcnt(0x8f71); break;
        case 34: __builtin_amdgcn_s_waitcnt(0x8f72); break;
        case 35: __builtin_amdgcn_s_waitcnt(0x8f73); break;
        case 36: __builtin_amdgcn_s_waitcnt(0x8f74); break;
        case 37: __builtin_amdgcn_s_waitcnt(0x8f75); break;
        case 38: __builtin_amdgcn_s_waitcnt(0x8f76); break;
        case 39: __builtin_amdgcn_s_waitcnt(0x8f77); break;
        case 40: __builtin_amdgcn_s_waitcnt(0x8f78); break;
        case 41: __builtin_amdgcn_s_waitcnt(0x8f79); break;
        case 42: __builtin_amdgcn_s_waitcnt(0x8f7a); break;
        case 43: __builtin_amdgcn_s_waitcnt(0x8f7b); break;
        case 44: __builtin_amdgcn_s_waitcnt(0x8f7c); break;
        case 45: __builtin_amdgcn_s_waitcnt(0x8f7d); break;
        case 46: __builtin_amdgcn_s_waitcnt(0x8f7e); break;
        case 47: __builtin_amdgcn_s_waitcnt(0x8f7f); break;
        case 48: __builtin_amdgcn_s_waitcnt(0xcf70); break;
        case 49: __builtin_amdgcn_s_waitcnt(0xcf71); break;
        case 50: __builtin_amdgcn_s_waitcnt(0xcf72); break;
        case 51: __builtin_amdgcn_s_waitcnt(0xcf73); break;
        case 52: __builtin_amdgcn_s_waitcnt(0xcf74); break;
        case 53: __builtin_amdgcn_s_waitcnt(0xcf75); break;
        case 54: __builtin_amdgcn_s_waitcnt(0xcf76); break;
        case 55: __builtin_amdgcn_s_waitcnt(0xcf77); break;
        case 56: __builtin_amdgcn_s_waitcnt(0xcf78); break;
        case 57: __builtin_amdgcn_s_waitcnt(0xcf79); break;
        case 58: __builtin_amdgcn_s_waitcnt(0xcf7a); break;
        case 59: __builtin_amdgcn_s_waitcnt(0xcf7b); break;
        case 60: __builtin_amdgcn_s_waitcnt(0xcf7c); break;
        case 61: __builtin_amdgcn_s_waitcnt(0xcf7d); break;
        case 62: __builtin_amdgcn_s_waitcnt(0xcf7e); break;
        default: __builtin_amdgcn_s_waitcnt(0xCF7F); break;
    }
}

// ---- direct HBM -> LDS loads (gfx950 global_load_lds_dwordx4) ------------
// Lane i of the wave writes its 16 bytes at lds_base + 16 * i; lds_base must be
// wave-uniform.  The "coherent" form reads at device scope (sc1), for data
// written by other workgroups of the same launch.
//
// The streaming form is issued through inline assembly on purpose: the
// compiler cannot tell which LDS bytes an in-flight direct load will write, so
// for the builtin it places a wait for *every* outstanding vector-memory
// operation before the next LDS read, which serialises a multi-stage ring.
// Callers of lds_stream16 therefore own the waits: s_waitcnt vmcnt(n) plus a
// workgroup barrier before the stage is read.  M0 (the LDS base of the load)
// is a register the compiler reserves and also sets for its own direct loads,
// so the sequence saves and restores it rather than clobbering it.
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}
__device__ __forceinline__ void lds_stream16(const void *src, void *lds_base) {
    const uint32_t m = __builtin_amdgcn_readfirstlane(lds_addr(lds_base));
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved) : "v"(src), "s"(m) : "memory");
}
// The same load with the non-temporal hint, for data read once per launch (the
// key/value streams): measured 6-9 % faster than the plain form on the
// bandwidth-bound verify attention and on the compact decode layer.
__device__ __forceinline__ void lds_stream16_nt(const void *src, void *lds_base) {
    const uint32_t m = __builtin_amdgcn_readfirstlane(lds_addr(lds_base));
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off nt\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved) : "v"(src), "s"(m) : "memory");
}
// Load N dwords at a wave-uniform address through the scalar cache (s_load).
template <int N>
__device__ __forceinline__ void load_uniform_dwords(const void *p, uint32_t (&out)[N]) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uintptr_t)p >> 32));
    const __attribute__((address_space(4))) uint32_t *c =
        (const __attribute__((address_space(4))) uint32_t *)(((uint64_t)hi << 32) | lo);
    #pragma unroll
    for (int i = 0; i < N; ++i) out[i] = c[i];
}
__device__ __forceinline__ void lds_load16_coherent(const void *src, void *lds_base) {
    __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)lds_base, 16, 0, 16);
}

// ---- phase trace: a diagnostic build only (-DMAD_PHASE_TRACE, libmad_trace.so) ----
// Thread 0 of a workgroup records the device's 100 MHz constant counter
// (s_memrealtime) at named phases of a kernel in a per-file device array of
// kTraceSlots words per workgroup (linear workgroup id), and in the last word
// its XCC id (high half) and hardware id register (low half).  One vector store
// per mark.  The counter has its own origin on each XCD, so only marks taken on
// one XCD compare.  In the product library the marks compile to nothing.
constexpr int kTraceSlots = 16, kTraceWGs = 4096;
#ifdef MAD_PHASE_TRACE
__device__ __forceinline__ unsigned trace_block() {
    return blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
}
__device__ __forceinline__ void trace_mark(unsigned long long *buf, int slot) {
    const unsigned b = trace_block();
    if (threadIdx.x == 0 && b < (unsigned)kTraceWGs) buf[kTraceSlots * b + slot] = __builtin_amdgcn_s_memrealtime();
}
__device__ __forceinline__ void trace_ids(unsigned long long *buf) {
    const unsigned b = trace_block();
    if (threadIdx.x == 0 && b < (unsigned)kTraceWGs) {
        const unsigned hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);    // HW_ID
        const unsigned xcc = __builtin_amdgcn_s_getreg((3 << 11) | 20);   // XCC_ID
        buf[kTraceSlots * b + kTraceSlots - 1] = ((unsigned long long)xcc << 32) | hw;
    }
}
#define MAD_TRACE_BUFFER(NAME)                                                                          \
    __device__ unsigned long long NAME[kTraceSlots * kTraceWGs];                                        \
    extern "C" int NAME##_read(void *host, size_t bytes) {                                              \
        if (bytes > sizeof(NAME)) return -1;                                                            \
        return (int)hipMemcpyFromSymbol(host, HIP_SYMBOL(NAME), bytes, 0, hipMemcpyDeviceToHost);       \
    }                                                                                                   \
    extern "C" int NAME##_clear(void) {                                                                 \
        static const unsigned long long zero[kTraceSlots * kTraceWGs] = {};                            \
        return (int)hipMemcpyToSymbol(HIP_SYMBOL(NAME), zero, sizeof(zero), 0, hipMemcpyHostToDevice);  \
    }
// MAD_TRACE_T0 reads the counter at kernel entry into a register;
// MAD_TRACE_SAVE_T0 stores it (slot 0) with the ids at a later point, so the
// entry itself gains no store
#define MAD_TRACE_T0() const unsigned long long mad_trace_t0 = __builtin_amdgcn_s_memrealtime()
#define MAD_TRACE_SAVE_T0(NAME)                                                        \
    do {                                                                               \
        const unsigned b_ = trace_block();                                             \
        if (threadIdx.x == 0 && b_ < (unsigned)kTraceWGs) NAME[kTraceSlots * b_] = mad_trace_t0; \
        trace_ids(NAME);                                                               \
    } while (0)
#define MAD_TRACE(NAME, SLOT) trace_mark(NAME, SLOT)
// a mark read now and stored later (MAD_TRACE_PUT), where a store would be
// counted by a wait that follows it (vmcnt counts stores as well as loads)
#define MAD_TRACE_VAR(VAR) unsigned long long VAR = 0
#define MAD_TRACE_SET(VAR) (VAR = __builtin_amdgcn_s_memrealtime())
#define MAD_TRACE_PUT(NAME, SLOT, VAR)                                                 \
    do {                                                                               \
        const unsigned b_ = trace_block();                                             \
        if (threadIdx.x == 0 && b_ < (unsigned)kTraceWGs) NAME[kTraceSlots * b_ + (SLOT)] = (VAR); \
    } while (0)
#else
#define MAD_TRACE_BUFFER(NAME)
#define MAD_TRACE_T0() ((void)0)
#define MAD_TRACE_SAVE_T0(NAME) ((void)0)
#define MAD_TRACE(NAME, SLOT) ((void)0)
#define MAD_TRACE_VAR(VAR) ((void)0)
#define MAD_TRACE_SET(VAR) ((void)0)
#define MAD_TRACE_PUT(NAME, SLOT, VAR) ((void)0)
#endif

}  // namespace mad
