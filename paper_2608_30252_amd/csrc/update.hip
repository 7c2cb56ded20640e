// update.hip -- memory update by the MASW memory adaptor (Sec. 3.2).
//
// For every new memory slot row r = (sequence b, slot i) the mirrored
// projections give  [k~ | v] = x[r] . [W_K,g ; W_V,g]^T,  the key is rotated at
// the slot's position id (the id of the raw token that follows the slot), and
// the pair is appended at memory row len[b] + i.  Rows of sequences whose fire
// flag is 0 are computed but not written (per-sequence masks of heterogeneous
// batches, Sec. 4.1).
//
// BF16: the projection Y[R x N] = X[R x D] W^T runs on the matrix cores
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation).  Workgroup (head block hb,
// k-split ks) owns the d output features of one K or V head and a slice of the
// input width; every wave covers d/4 features for all rows.  W is streamed
// once from HBM straight into the MFMA operand registers (16 bytes a lane).
// Split partials go to the workspace with device-coherent stores; the last
// workgroup of a head block (arrival counter) pulls them into LDS in one round
// trip, sums them, applies RoPE with fp64 angles and writes bf16 rows.
// F32: a vector-ALU kernel, one thread per (row, rotation pair).
#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_v;
typedef __attribute__((ext_vector_type(4))) float f32x4_v;

// Rotate-half RoPE of one feature pair (j, j + d/2) at integer position pos;
// the angle pos * base^(-2j/d) is formed and reduced in double precision.
__device__ __forceinline__ void rope_pair(double y0, double y1, int j, int d, int pos, double log2_base,
                                          double *k0, double *k1) {
    const double theta = exp2(-2.0 * (double)j / (double)d * log2_base);
    double s, c;
    sincos((double)pos * theta, &s, &c);
    *k0 = y0 * c - y1 * s;
    *k1 = y1 * c + y0 * s;
}

template <int D>
__global__ __launch_bounds__(256) void update_mfma_kernel(const UpdateArgs a) {
    constexpr int CT = D / 64;   // 16-feature column tiles per wave
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int NH = 2 * a.Hkv;
    const int hb = blockIdx.x % NH, ks = blockIdx.x / NH;
    const int R = a.R;
    const int RT = (R + 15) / 16;
    const int k_lo = ks * a.kc;
    const bf16_t *x = reinterpret_cast<const bf16_t *>(a.x);
    const bf16_t *w = reinterpret_cast<const bf16_t *>(a.w) + (size_t)hb * D * a.D;

    f32x4_v acc[4][CT];
    #pragma unroll
    for (int rt = 0; rt < 4; ++rt)
        #pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = f32x4_v{0.f, 0.f, 0.f, 0.f};

    const int kq = 8 * (lane >> 4);   // this lane's 8-element slice of a 32-wide k step
    for (int k0 = k_lo; k0 < k_lo + a.kc; k0 += 32) {
        bf16x8_v bop[CT];
        #pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            const int col = wave * (D / 4) + ct * 16 + (lane & 15);
            bop[ct] = *reinterpret_cast<const bf16x8_v *>(w + (size_t)col * a.D + k0 + kq);
        }
        #pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            if (rt < RT) {
                const int row = rt * 16 + (lane & 15);
                bf16x8_v aop;
                if (row < R) aop = *reinterpret_cast<const bf16x8_v *>(x + (size_t)row * a.D + k0 + kq);
                else aop = bf16x8_v{0, 0, 0, 0, 0, 0, 0, 0};
                #pragma unroll
                for (int ct = 0; ct < CT; ++ct)
                    acc[rt][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aop, bop[ct], acc[rt][ct], 0, 0, 0);
            }
        }
    }

    // ---- partial [hb][ks][R][D] with device-coherent stores ----
    float *blk = a.part + (size_t)hb * a.part_stride;
    float *pp = blk + (size_t)ks * R * D;
    #pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
        if (rt < RT) {
            #pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                const int col = wave * (D / 4) + ct * 16 + (lane & 15);
                #pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = rt * 16 + 4 * (lane >> 4) + i;
                    if (row < R) store_agent(pp + (size_t)row * D + col, acc[rt][ct][i]);
                }
            }
        }
    }
    wait_vm_stores();
    __syncthreads();
    __shared__ int s_last;
    if (tid == 0) {
        unsigned *cnt = a.counters + (size_t)hb * kCounterStride;
        const int last = arrive(cnt) == (unsigned)(a.KS - 1);
        if (last) reset_counter(cnt);
        s_last = last;
    }
    __syncthreads();
    if (!s_last) return;

    // ---- last workgroup of the head block: sum the splits, rotate, append ----
    extern __shared__ __align__(16) unsigned char smem[];
    const int nbytes = (a.KS * R * D * 4 + 15) & ~15;
    for (int off = wave * 1024; off < nbytes; off += 4096)
        if (off + lane * 16 < nbytes)
            lds_load16_coherent(reinterpret_cast<const unsigned char *>(blk) + off + lane * 16, smem + off);
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
    const float *sp = reinterpret_cast<const float *>(smem);
    const bool is_k = hb < a.Hkv;
    const int h = is_k ? hb : hb - a.Hkv;
    bf16_t *dst_base = reinterpret_cast<bf16_t *>(is_k ? a.mk : a.mv) + (size_t)h * a.m_head;
    for (int idx = tid; idx < R * (D / 2); idx += 256) {
        const int r = idx / (D / 2), j = idx % (D / 2);
        float y0 = 0.f, y1 = 0.f;
        for (int s = 0; s < a.KS; ++s) {
            y0 += sp[((size_t)s * R + r) * D + j];
            y1 += sp[((size_t)s * R + r) * D + j + D / 2];
        }
        const int b = r / a.n_new, i = r - b * a.n_new;
        if (!a.fire[b]) continue;
        double o0 = y0, o1 = y1;
        if (is_k) rope_pair(y0, y1, j, D, a.pos[r], a.log2_base, &o0, &o1);
        bf16_t *dst = dst_base + (size_t)b * a.m_seq + (size_t)(a.mlen[b] + i) * D;
        dst[j].bits = f32_to_bf16((float)o0);
        dst[j + D / 2].bits = f32_to_bf16((float)o1);
    }
}

// fp32: one thread per (row r, head h of K or V, feature pair j).
__global__ __launch_bounds__(256) void update_f32_kernel(const UpdateArgs a) {
    const int d = a.d, half = d / 2;
    const int NH = 2 * a.Hkv;
    const int total = a.R * NH * half;
    const int idx = blockIdx.x * 256 + threadIdx.x;
    if (idx >= total) return;
    const int j = idx % half, hb = (idx / half) % NH, r = idx / (half * NH);
    const float *x = reinterpret_cast<const float *>(a.x) + (size_t)r * a.D;
    const float *w0 = reinterpret_cast<const float *>(a.w) + ((size_t)hb * d + j) * a.D;
    const float *w1 = w0 + (size_t)half * a.D;
    float y0 = 0.f, y1 = 0.f;
    for (int k = 0; k < a.D; k += 4) {
        const float4 xv = *reinterpret_cast<const float4 *>(x + k);
        const float4 a0 = *reinterpret_cast<const float4 *>(w0 + k);
        const float4 a1 = *reinterpret_cast<const float4 *>(w1 + k);
        y0 = fmaf(xv.x, a0.x, y0); y0 = fmaf(xv.y, a0.y, y0); y0 = fmaf(xv.z, a0.z, y0); y0 = fmaf(xv.w, a0.w, y0);
        y1 = fmaf(xv.x, a1.x, y1); y1 = fmaf(xv.y, a1.y, y1); y1 = fmaf(xv.z, a1.z, y1); y1 = fmaf(xv.w, a1.w, y1);
    }
    const int b = r / a.n_new, i = r - b * a.n_new;
    if (!a.fire[b]) return;
    const bool is_k = hb < a.Hkv;
    const int h = is_k ? hb : hb - a.Hkv;
    double o0 = y0, o1 = y1;
    if (is_k) rope_pair(y0, y1, j, d, a.pos[r], a.log2_base, &o0, &o1);
    float *dst = reinterpret_cast<float *>(is_k ? a.mk : a.mv) + (size_t)b * a.m_seq + (size_t)h * a.m_head +
                 (size_t)(a.mlen[b] + i) * d;
    dst[j] = (float)o0;
    dst[j + half] = (float)o1;
}

// ------------------------------------------------------------------ host ----

UpdatePlan plan_update(int R, int D, int Hkv, int d) {
    UpdatePlan p;
    const int NH = 2 * Hkv;
    const int ksteps = D / 32;
    int ks = (256 + NH - 1) / NH;                               // aim at ~256 workgroups
    const int lds_cap = (int)(kUpdateMergeBytes / ((size_t)R * d * 4));
    if (ks > lds_cap) ks = lds_cap;
    if (ks > ksteps) ks = ksteps;
    if (ks < 1) ks = 1;
    while (ksteps % ks) --ks;                                   // equal k chunks of whole steps
    p.KS = ks;
    p.kc = D / ks;
    return p;
}

size_t update_ws_bytes(int R, int D, int Hkv, int d) {
    UpdatePlan p = plan_update(R, D, Hkv, d);
    return kCounterRegionBytes + (size_t)2 * Hkv * update_part_stride(R, d, p.KS) * 4 + 256;
}

size_t update_part_stride(int R, int d, int KS) { return ((size_t)KS * R * d + 63) / 64 * 64; }

hipError_t launch_update(const UpdateArgs &a, int dtype, hipStream_t st) {
    if (dtype == MAD_BF16) {
        dim3 grid((unsigned)(2 * a.Hkv * a.KS)), block(256);
        const size_t lds = (size_t)a.KS * a.R * a.d * 4 + 16;
        if (a.d == 64) hipLaunchKernelGGL(update_mfma_kernel<64>, grid, block, lds, st, a);
        else hipLaunchKernelGGL(update_mfma_kernel<128>, grid, block, lds, st, a);
    } else {
        const int total = a.R * 2 * a.Hkv * (a.d / 2);
        dim3 grid((unsigned)((total + 255) / 256)), block(256);
        hipLaunchKernelGGL(update_f32_kernel, grid, block, 0, st, a);
    }
    return hipGetLastError();
}

}  // namespace mad
