// layer.hip -- the linear maps of a draft decoder layer around its attention:
// RMSNorm + fused Q/K/V projection with RoPE, the output projection with the
// residual, RMSNorm + the SwiGLU gate/up projection, and the down projection
// with the residual.  These chain the hidden states of raw tokens and of
// memory slots through the layers (Sec. 3.2: a slot token runs through the
// same transformer blocks; its hidden state entering layer l feeds the
// mirrored projections of layer l) and carry the weight-streaming term of the
// draft's per-token cost (Sec. 2.3, Eq. latency_decomp).
//
// At decode time a call has R <= 8 rows (the raw token, plus the slot tokens
// of a materialisation pass), so every map is a weight stream: y = x W^T with
// W [N][D] bf16 read once from HBM, fp32 accumulation.  A workgroup of 256
// threads owns NC output features; thread t owns the 16-byte chunks t, t+256,
// ... of every row, so one feature's row of W is read by the whole workgroup
// in 4 KB coalesced sweeps and every thread has NC x D/2048 loads in flight.
// Row sums: DPP/swizzle reductions inside each wave, then one LDS exchange of
// the four waves' partials.  Epilogues:
//   QKV     features grouped as rotate-half pairs (j, j + d/2) of one head, so
//           RoPE at the row's position id is local; q, k, v go to separate
//           [R][H][d] outputs; k and v of row 0 may be written to every row
//           (the current token's K/V, which the rows of a fused step share)
//   RES     y = residual + x W^T
//   SWIGLU  W = [W_gate ; W_up] (2F rows): y_j = silu(g_j) * u_j
// The normalised rows (bf16, as the projection consumes them) can be stored
// for the memory adaptor, which projects the same normalised slot rows.
#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

constexpr int kLinQKV = 0, kLinRes = 1, kLinSwiglu = 2;

__device__ __forceinline__ float lin_dot8(const uint4 &w, const uint4 &x, float acc) {
    typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, w.x), __builtin_bit_cast(bf16x2_v, x.x), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, w.y), __builtin_bit_cast(bf16x2_v, x.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, w.z), __builtin_bit_cast(bf16x2_v, x.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, w.w), __builtin_bit_cast(bf16x2_v, x.w), acc, false);
    return acc;
}

template <int MODE, int RR, int NC, int KD>
__global__ __launch_bounds__(256) void linear_kernel(const LinearArgs a) {
    constexpr bool NORM = MODE != kLinRes;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int R = a.R, D = a.D;
    __shared__ float s_red[4][NC * RR];
    __shared__ float s_sq[4][RR];

    // ---- input rows: thread t holds chunks t + 256 j (8 features each) ----
    // Rows past R read row R - 1 (their results are never stored): an
    // unconditional load, where a conditional one is waited for inside its
    // branch, before any weight load is issued.
    const bf16_t *x = reinterpret_cast<const bf16_t *>(a.x);
    uint4 xr[RR][KD];
    #pragma unroll
    for (int r = 0; r < RR; ++r)
        #pragma unroll
        for (int j = 0; j < KD; ++j)
            xr[r][j] = *reinterpret_cast<const uint4 *>(x + (size_t)min(r, R - 1) * D + (tid + 256 * j) * 8);

    // ---- this workgroup's features and the first weight loads ----
    int col[NC];
    #pragma unroll
    for (int c = 0; c < NC; ++c) {
        if constexpr (MODE == kLinQKV) {
            // pair q = blockIdx * NC/2 + c % (NC/2): head q / (d/2), offset q % (d/2)
            const int q = blockIdx.x * (NC / 2) + (c % (NC / 2));
            const int hd = a.head_dim / 2;
            col[c] = (q / hd) * a.head_dim + (q % hd) + (c >= NC / 2 ? hd : 0);
        } else if constexpr (MODE == kLinSwiglu) {
            col[c] = c < NC / 2 ? blockIdx.x * (NC / 2) + c : a.N + blockIdx.x * (NC / 2) + c - NC / 2;
        } else {
            col[c] = blockIdx.x * NC + c;
        }
    }
    const bf16_t *w = reinterpret_cast<const bf16_t *>(a.w);
    uint4 wr[NC][KD];
    #pragma unroll
    for (int c = 0; c < NC; ++c)
        #pragma unroll
        for (int j = 0; j < KD; ++j)
            wr[c][j] = *reinterpret_cast<const uint4 *>(w + (size_t)col[c] * D + (tid + 256 * j) * 8);

    // the norm weights, loaded with everything else rather than after the barrier
    uint4 gr[KD];
    if constexpr (NORM) {
        const bf16_t *gm = reinterpret_cast<const bf16_t *>(a.gamma);
        #pragma unroll
        for (int j = 0; j < KD; ++j) gr[j] = *reinterpret_cast<const uint4 *>(gm + (tid + 256 * j) * 8);
    }

    // ---- RMSNorm of the input rows (fp32), rounded to bf16 for the product ----
    if constexpr (NORM) {
        float ss[RR];
        #pragma unroll
        for (int r = 0; r < RR; ++r) {
            ss[r] = 0.f;
            #pragma unroll
            for (int j = 0; j < KD; ++j) {
                const uint32_t u4[4] = {xr[r][j].x, xr[r][j].y, xr[r][j].z, xr[r][j].w};
                #pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float lo = bf16_lo(u4[e]), hi = bf16_hi(u4[e]);
                    ss[r] = fmaf(lo, lo, fmaf(hi, hi, ss[r]));
                }
            }
            ss[r] = group_sum<64>(ss[r]);
            if (lane == 0) s_sq[wave][r] = ss[r];
        }
        __syncthreads();
        #pragma unroll
        for (int r = 0; r < RR; ++r) {
            const float tot = s_sq[0][r] + s_sq[1][r] + s_sq[2][r] + s_sq[3][r];
            const float inv = 1.f / sqrtf(tot / (float)D + a.eps);
            #pragma unroll
            for (int j = 0; j < KD; ++j) {
                uint32_t u4[4] = {xr[r][j].x, xr[r][j].y, xr[r][j].z, xr[r][j].w};
                const uint32_t g4[4] = {gr[j].x, gr[j].y, gr[j].z, gr[j].w};
                #pragma unroll
                for (int e = 0; e < 4; ++e)
                    u4[e] = cvt_pk_bf16(bf16_lo(u4[e]) * inv * bf16_lo(g4[e]), bf16_hi(u4[e]) * inv * bf16_hi(g4[e]));
                xr[r][j] = make_uint4(u4[0], u4[1], u4[2], u4[3]);
                if (MODE == kLinQKV && a.xn && blockIdx.x == 0 && r < R)
                    *reinterpret_cast<uint4 *>(reinterpret_cast<bf16_t *>(a.xn) + (size_t)r * D + (tid + 256 * j) * 8) =
                        xr[r][j];
            }
        }
    }

    // ---- products and row sums ----
    float acc[NC][RR];
    #pragma unroll
    for (int c = 0; c < NC; ++c)
        #pragma unroll
        for (int r = 0; r < RR; ++r) {
            float s = 0.f;
            #pragma unroll
            for (int j = 0; j < KD; ++j) s = lin_dot8(wr[c][j], xr[r][j], s);
            acc[c][r] = s;
        }
    #pragma unroll
    for (int c = 0; c < NC; ++c)
        #pragma unroll
        for (int r = 0; r < RR; ++r) {
            const float s = group_sum<64>(acc[c][r]);
            if (lane == 0) s_red[wave][c * RR + r] = s;
        }
    __syncthreads();

    // ---- epilogues ----
    if constexpr (MODE == kLinQKV) {
        // thread (pair p, row r): features col[p], col[p + NC/2]
        constexpr int NP = NC / 2;
        if (tid < NP * RR) {
            const int p = tid / RR, r = tid % RR;
            if (r < R) {
                float y0 = 0.f, y1 = 0.f;
                #pragma unroll
                for (int wv = 0; wv < 4; ++wv) {
                    y0 += s_red[wv][p * RR + r];
                    y1 += s_red[wv][(p + NP) * RR + r];
                }
                const int hd = a.head_dim, q = blockIdx.x * NP + p;
                const int head = q / (hd / 2), jj = q % (hd / 2);   // feature pair (jj, jj + d/2) of `head`
                if (head < a.Hq + a.Hkv) rope_rotate(y0, y1, a.pos[r], rope_theta(jj, hd, a.log2_base), &y0, &y1);
                const uint16_t b0 = f32_to_bf16(y0), b1 = f32_to_bf16(y1);
                if (head < a.Hq) {
                    bf16_t *dst = reinterpret_cast<bf16_t *>(a.q) + ((size_t)r * a.Hq + head) * hd;
                    dst[jj].bits = b0;
                    dst[jj + hd / 2].bits = b1;
                } else if (!a.kv_from_row0 || r == 0) {
                    // K or V head; with kv_from_row0 row 0's values go to every row
                    const bool isk = head < a.Hq + a.Hkv;
                    const int hk = head - a.Hq - (isk ? 0 : a.Hkv);
                    bf16_t *base = reinterpret_cast<bf16_t *>(isk ? a.k : a.v);
                    const int r_lo = a.kv_from_row0 ? 0 : r, r_hi = a.kv_from_row0 ? R : r + 1;
                    for (int rr = r_lo; rr < r_hi; ++rr) {
                        bf16_t *dst = base + ((size_t)rr * a.Hkv + hk) * hd;
                        dst[jj].bits = b0;
                        dst[jj + hd / 2].bits = b1;
                    }
                }
            }
        }
    } else {
        const int ncol = MODE == kLinSwiglu ? NC / 2 : NC;
        if (tid < ncol * RR) {
            const int c = tid / RR, r = tid % RR;
            if (r < R) {
                float y = 0.f;
                #pragma unroll
                for (int wv = 0; wv < 4; ++wv) y += s_red[wv][c * RR + r];
                const int n = blockIdx.x * ncol + c;
                if constexpr (MODE == kLinSwiglu) {
                    float u = 0.f;
                    #pragma unroll
                    for (int wv = 0; wv < 4; ++wv) u += s_red[wv][(c + NC / 2) * RR + r];
                    y = y / (1.f + __expf(-y)) * u;
                } else {
                    y += bf16_to_f32(reinterpret_cast<const bf16_t *>(a.res)[(size_t)r * a.N + n].bits);
                }
                reinterpret_cast<bf16_t *>(a.out)[(size_t)r * a.N + n].bits = f32_to_bf16(y);
            }
        }
    }
}

// ------------------------------------------------------------------ host ----

template <int MODE, int NC, int KD>
static hipError_t launch_rr(const LinearArgs &a, int grid, hipStream_t st) {
    if (a.R == 1) {
        hipLaunchKernelGGL((linear_kernel<MODE, 1, NC, KD>), dim3(grid), dim3(256), 0, st, a);
    } else {
        hipLaunchKernelGGL((linear_kernel<MODE, kMaxLinRows, NC, KD>), dim3(grid), dim3(256), 0, st, a);
    }
    return hipGetLastError();
}

template <int MODE, int NC>
static hipError_t launch_kd(const LinearArgs &a, int grid, hipStream_t st) {
    switch (a.D / 2048) {
        case 1: return launch_rr<MODE, NC, 1>(a, grid, st);
        case 2: return launch_rr<MODE, NC, 2>(a, grid, st);
    }
    return hipErrorInvalidValue;
}

// Features per workgroup (measured): 2 for Q/K/V (one rotation pair each,
// 1536 workgroups; 5% faster than two pairs), 8 for the output projection (one
// workgroup per CU; 2 and 4 measure the same), 2 for the wide down projection
// (1024 workgroups; 3% faster than 4), 8 (4 gate + 4 up) for the SwiGLU map (4
// and 16 are slower).
hipError_t launch_linear(const LinearArgs &a, int mode, hipStream_t st) {
    if (mode == kLinQKV) return launch_kd<kLinQKV, 2>(a, a.N / 2, st);
    if (mode == kLinSwiglu) return launch_kd<kLinSwiglu, 8>(a, a.N / 4, st);
    if (mode == kLinRes) {
        if (a.D / 2048 == 4) return launch_rr<kLinRes, 2, 4>(a, a.N / 2, st);
        if (a.N % 8 == 0) return launch_kd<kLinRes, 8>(a, a.N / 8, st);
        return launch_kd<kLinRes, 4>(a, a.N / 4, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace mad
