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
// input width.  Its X and W slices stream from HBM straight into LDS
// (global_load_lds_dwordx4) in 64-wide k chunks through a two-stage ring, 16-byte
// chunks XOR-swizzled by row so the MFMA operand reads are conflict-free; every
// wave covers d/4 features for all rows.  Split partials go to the workspace
// with device-coherent stores; the last workgroup of a head block (arrival
// counter) pulls them into LDS in one round trip, sums them, applies RoPE with
// fp64 angles and writes bf16 rows.
// BF16 with at most 8 rows (a single sequence's update, or a few): a weight
// stream instead (update_gemv_kernel).  The projection is then a matrix-vector
// product per row, bound by reading W once; a workgroup owns NC output
// features -- rotate-half pairs (j, j + d/2) of one K or V head -- over the
// whole input width, so no split partials and no merge: thread t holds the
// 16-byte chunks t, t + 256, ... of every row and of the NC weight rows (all
// loads issued together), products by v_dot2_f32_bf16, wave and workgroup
// sums, then RoPE on the K pairs and the append.
// F32: a vector-ALU kernel, one thread per (row, rotation pair).
#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_v;
typedef __attribute__((ext_vector_type(4))) float f32x4_v;


constexpr int kUpdSubK = 64;                 // k elements per ring stage (8 chunks of 16 bytes a row)

// LDS of the merged rows [KS][R][d] fp32, 16-byte aligned; the angle table follows.
__host__ __device__ __forceinline__ size_t update_merge_bytes(int KS, int R, int d) {
    return ((size_t)KS * R * d * 4 + 15) / 16 * 16;
}
constexpr int kUpdRowBytes = kUpdSubK * 2;   // 128 bytes of X or W row per stage

template <int D>
__global__ __launch_bounds__(256) void update_mfma_kernel(const UpdateArgs a) {
    constexpr int CT = D / 64;   // 16-feature column tiles per wave
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int NH = 2 * a.Hkv;
    const int hb = blockIdx.x % NH, ks = blockIdx.x / NH;
    const int R = a.R;
    const int RT = (R + 15) / 16;
    const int k_lo = ks * a.kc;
    const bf16_t *x = reinterpret_cast<const bf16_t *>(a.x);
    const bf16_t *w = reinterpret_cast<const bf16_t *>(a.w) + (size_t)hb * D * a.D;

    // ---- stage layout: [X rows 0..R-1 | W rows 0..D-1], 128 bytes each ----
    const int rows = R + D;
    const int chunks = rows * (kUpdRowBytes / 16);              // 16-byte pieces per stage
    const int per_round = 256;                                  // one piece per thread per round
    const int rounds = (chunks + per_round - 1) / per_round;    // load instructions per thread per stage
    const int stage_bytes = rounds * per_round * 16;
    const int nsub = a.kc / kUpdSubK;
    const int S = a.stages;                                     // ring stages (all slices at once when they fit)
    auto issue = [&](int sub, int stage) {
        unsigned char *st = smem + stage * stage_bytes;
        const int kb = k_lo + sub * kUpdSubK;
        for (int rd = 0; rd < rounds; ++rd) {
            const int inst = rd * 4 + wave;                      // 1 KB block of the stage
            int piece = inst * 64 + lane;
            if (piece >= chunks) piece = chunks - 1;             // padding lanes fetch a valid piece again
            const int r = piece >> 3, slot = piece & 7;
            const int c = slot ^ (r & 7);                        // LDS slot `slot` of row r holds chunk c
            const bf16_t *src = r < R ? x + (size_t)r * a.D : w + (size_t)(r - R) * a.D;
            lds_stream16(src + kb + c * 8, st + inst * 1024);
        }
    };

    f32x4_v acc[4][CT];
    #pragma unroll
    for (int rt = 0; rt < 4; ++rt)
        #pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = f32x4_v{0.f, 0.f, 0.f, 0.f};

    int issued = 0;
    for (; issued < nsub && issued < S; ++issued) issue(issued, issued);
    const int kq = lane >> 4;   // this lane's chunk within a 32-wide k step (8 elements)
    for (int t = 0; t < nsub; ++t) {
        wait_vm(rounds * (issued - t - 1));
        __syncthreads();   // slice t is in LDS
        const unsigned char *st = smem + (t % S) * stage_bytes;
        #pragma unroll
        for (int kst = 0; kst < kUpdSubK / 32; ++kst) {
            const int c = kst * 4 + kq;
            bf16x8_v bop[CT];
            #pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                const int fr = R + wave * (D / 4) + ct * 16 + (lane & 15);   // stage row of the feature
                bop[ct] = *reinterpret_cast<const bf16x8_v *>(st + (size_t)fr * kUpdRowBytes + ((c ^ (fr & 7)) << 4));
            }
            #pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                if (rt < RT) {
                    const int row = rt * 16 + (lane & 15);
                    bf16x8_v aop = bf16x8_v{0, 0, 0, 0, 0, 0, 0, 0};
                    if (row < R) aop = *reinterpret_cast<const bf16x8_v *>(st + (size_t)row * kUpdRowBytes + ((c ^ (row & 7)) << 4));
                    #pragma unroll
                    for (int ct = 0; ct < CT; ++ct)
                        acc[rt][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aop, bop[ct], acc[rt][ct], 0, 0, 0);
                }
            }
        }
        if (issued < nsub) {
            __syncthreads();   // every wave is done with stage t % S
            issue(issued, issued % S);
            ++issued;
        }
    }

    __syncthreads();   // every wave is done with the stages
    // ---- the head block's rows y [R][D]: in LDS directly (one split) or via
    // device-coherent partials [ks][R][D] and the last-arriving workgroup ----
    float *blk = a.part + (size_t)hb * a.part_stride;
    float *ys = reinterpret_cast<float *>(smem);
    const bool single = a.KS == 1;
    #pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
        if (rt < RT) {
            #pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                const int col = wave * (D / 4) + ct * 16 + (lane & 15);
                #pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = rt * 16 + 4 * (lane >> 4) + i;
                    if (row < R) {
                        if (single) ys[(size_t)row * D + col] = acc[rt][ct][i];
                        else store_agent(blk + ((size_t)ks * R + row) * D + col, acc[rt][ct][i]);
                    }
                }
            }
        }
    }
    if (!single) {
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
        // ---- last workgroup of the head block: pull every split into LDS ----
        const int nbytes = (a.KS * R * D * 4 + 15) & ~15;
        for (int off = wave * 1024; off < nbytes; off += 4096)
            if (off + lane * 16 < nbytes)
                lds_load16_coherent(reinterpret_cast<const unsigned char *>(blk) + off + lane * 16, smem + off);
        __builtin_amdgcn_s_waitcnt(0x0F70);
    }
    __syncthreads();

    // ---- sum the splits, rotate the K half at the slot positions, append ----
    // thread <-> (row r, four consecutive rotation pairs j..j+3); the 2 x KS
    // 16-byte reads of an item are issued together
    const float *sp = reinterpret_cast<const float *>(smem);
    double *theta = reinterpret_cast<double *>(smem + update_merge_bytes(a.KS, R, D));
    const bool is_k = hb < a.Hkv;
    if (is_k && tid < D / 2) theta[tid] = rope_theta(tid, D, a.log2_base);
    __syncthreads();
    const int h = is_k ? hb : hb - a.Hkv;
    bf16_t *dst_base = reinterpret_cast<bf16_t *>(is_k ? a.mk : a.mv) + (size_t)h * a.m_head;
    constexpr int Q = D / 8;   // groups of four pairs per row
    for (int idx = tid; idx < R * Q; idx += 256) {
        const int r = idx / Q, j = (idx % Q) * 4;
        float4 y0 = make_float4(0.f, 0.f, 0.f, 0.f), y1 = y0;
        for (int s0 = 0; s0 < a.KS; s0 += 8) {
            float4 u[8], v[8];
            #pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int sidx = s0 + t < a.KS ? s0 + t : a.KS - 1;
                u[t] = *reinterpret_cast<const float4 *>(sp + ((size_t)sidx * R + r) * D + j);
                v[t] = *reinterpret_cast<const float4 *>(sp + ((size_t)sidx * R + r) * D + j + D / 2);
            }
            #pragma unroll
            for (int t = 0; t < 8; ++t) {
                if (s0 + t < a.KS) {
                    y0.x += u[t].x; y0.y += u[t].y; y0.z += u[t].z; y0.w += u[t].w;
                    y1.x += v[t].x; y1.y += v[t].y; y1.z += v[t].z; y1.w += v[t].w;
                }
            }
        }
        const int b = r / a.n_new, i = r - b * a.n_new;
        if (!a.fire[b]) continue;
        float o0[4] = {y0.x, y0.y, y0.z, y0.w}, o1[4] = {y1.x, y1.y, y1.z, y1.w};
        if (is_k) {
            #pragma unroll
            for (int e = 0; e < 4; ++e) rope_rotate(o0[e], o1[e], a.pos[r], theta[j + e], &o0[e], &o1[e]);
        }
        bf16_t *dst = dst_base + (size_t)b * a.m_seq + (size_t)(a.mlen[b] + i) * D;
        reinterpret_cast<uint2 *>(dst + j)[0] = make_uint2(pack_bf16x2(o0[0], o0[1]), pack_bf16x2(o0[2], o0[3]));
        reinterpret_cast<uint2 *>(dst + j + D / 2)[0] = make_uint2(pack_bf16x2(o1[0], o1[1]), pack_bf16x2(o1[2], o1[3]));
    }
}

template <int RR, int NC, int KD>
__global__ __launch_bounds__(256) void update_gemv_kernel(const UpdateArgs a) {
    constexpr int NP = NC / 2;   // rotation pairs per workgroup
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int R = a.R, D = a.D, d = a.d, hd = d / 2;
    __shared__ float s_red[4][NC * RR];

    // ---- rows and weights: chunk t + 256 j (8 inputs) of each ----
    const bf16_t *x = reinterpret_cast<const bf16_t *>(a.x);
    const bf16_t *w = reinterpret_cast<const bf16_t *>(a.w);
    int wrow[NC];   // W row of feature c: pair q = blockIdx * NP + c % NP of head q / hd
    #pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int q = blockIdx.x * NP + (c % NP);
        wrow[c] = (q / hd) * d + (q % hd) + (c >= NP ? hd : 0);
    }
    uint4 wr[NC][KD], xr[RR][KD];
    #pragma unroll
    for (int j = 0; j < KD; ++j) {
        const int e = (tid + 256 * j) * 8;
        const bool in = e < D;
        #pragma unroll
        for (int c = 0; c < NC; ++c)
            wr[c][j] = in ? *reinterpret_cast<const uint4 *>(w + (size_t)wrow[c] * D + e) : make_uint4(0u, 0u, 0u, 0u);
        #pragma unroll
        for (int r = 0; r < RR; ++r)
            xr[r][j] = in && r < R ? *reinterpret_cast<const uint4 *>(x + (size_t)r * D + e) : make_uint4(0u, 0u, 0u, 0u);
    }
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    auto dot8 = [](const uint4 &u, const uint4 &v, float acc) {
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u.x), __builtin_bit_cast(bf16x2_t, v.x), acc, false);
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u.y), __builtin_bit_cast(bf16x2_t, v.y), acc, false);
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u.z), __builtin_bit_cast(bf16x2_t, v.z), acc, false);
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u.w), __builtin_bit_cast(bf16x2_t, v.w), acc, false);
    };
    #pragma unroll
    for (int c = 0; c < NC; ++c)
        #pragma unroll
        for (int r = 0; r < RR; ++r) {
            float acc = 0.f;
            #pragma unroll
            for (int j = 0; j < KD; ++j) acc = dot8(wr[c][j], xr[r][j], acc);
            acc = group_sum<64>(acc);
            if (lane == 0) s_red[wave][c * RR + r] = acc;
        }
    __syncthreads();

    // ---- thread (pair p, row r): sum the waves, rotate a K pair, append ----
    if (tid < NP * RR) {
        const int p = tid / RR, r = tid % RR;
        if (r >= R) return;
        const int b = r / a.n_new, i = r - b * a.n_new;
        if (!a.fire[b]) return;
        float y0 = 0.f, y1 = 0.f;
        #pragma unroll
        for (int wv = 0; wv < 4; ++wv) {
            y0 += s_red[wv][p * RR + r];
            y1 += s_red[wv][(p + NP) * RR + r];
        }
        const int q = blockIdx.x * NP + p, head = q / hd, jj = q % hd;
        const bool is_k = head < a.Hkv;
        if (is_k) rope_rotate(y0, y1, a.pos[r], rope_theta(jj, d, a.log2_base), &y0, &y1);
        bf16_t *dst = reinterpret_cast<bf16_t *>(is_k ? a.mk : a.mv) + (size_t)(is_k ? head : head - a.Hkv) * a.m_head +
                      (size_t)b * a.m_seq + (size_t)(a.mlen[b] + i) * d;
        dst[jj].bits = f32_to_bf16(y0);
        dst[jj + hd].bits = f32_to_bf16(y1);
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
    float o0 = y0, o1 = y1;
    if (is_k) rope_rotate(y0, y1, a.pos[r], rope_theta(j, d, a.log2_base), &o0, &o1);
    float *dst = reinterpret_cast<float *>(is_k ? a.mk : a.mv) + (size_t)b * a.m_seq + (size_t)h * a.m_head +
                 (size_t)(a.mlen[b] + i) * d;
    dst[j] = o0;
    dst[j + half] = o1;
}

// ------------------------------------------------------------------ host ----

// Bytes of LDS a bf16 update workgroup needs: the two-stage ring, or the
// merge of all KS partials, whichever is larger.
static size_t update_stage_bytes(int R, int d) {
    const size_t pieces = (size_t)(R + d) * (kUpdRowBytes / 16);
    return (pieces + 255) / 256 * 256 * 16;
}
static int update_rounds(int R, int d) { return (int)(update_stage_bytes(R, d) / 4096); }
// Ring stages: every k slice of the workgroup at once when LDS and the vmcnt
// range allow it, else as many as fit (at least two).
static int update_stages(int R, int d, int KS, int D) {
    const int nsub = D / KS / kUpdSubK;
    int s = nsub;
    const int by_lds = (int)((kUpdateMaxLds - (size_t)d / 2 * 8 - 16) / update_stage_bytes(R, d));
    const int by_cnt = 62 / update_rounds(R, d) + 1;
    if (s > by_lds) s = by_lds;
    if (s > by_cnt) s = by_cnt;
    if (s < 2) s = 2;
    return s;
}
static size_t update_lds_bytes(int R, int d, int KS, int stages) {
    const size_t ring = (size_t)stages * update_stage_bytes(R, d);
    const size_t merge = update_merge_bytes(KS, R, d);
    return (ring > merge ? ring : merge) + (size_t)d / 2 * 8 + 16;   // + the RoPE angle table
}

UpdatePlan plan_update(int R, int D, int Hkv, int d) {
    UpdatePlan p;
    const int NH = 2 * Hkv;
    const int nk = D / kUpdSubK;                                // 64-wide k chunks
    int ks = (kUpdateTargetWGs + NH - 1) / NH;
    while (ks > 1 && update_lds_bytes(R, d, ks, 2) > kUpdateMaxLds) --ks;
    if (ks > nk) ks = nk;
    if (ks < 1) ks = 1;
    while (nk % ks) --ks;                                       // equal k slices of whole chunks
    p.KS = ks;
    p.kc = D / ks;
    p.stages = update_stages(R, d, ks, D);
    return p;
}

size_t update_ws_bytes(int R, int D, int Hkv, int d) {
    UpdatePlan p = plan_update(R, D, Hkv, d);
    return kCounterRegionBytes + (size_t)2 * Hkv * update_part_stride(R, d, p.KS) * 4 + 256;
}

size_t update_part_stride(int R, int d, int KS) { return ((size_t)KS * R * d + 63) / 64 * 64; }

template <int RR, int KD>
static hipError_t launch_gemv(const UpdateArgs &a, hipStream_t st) {
    constexpr int NC = 4;
    hipLaunchKernelGGL((update_gemv_kernel<RR, NC, KD>), dim3((unsigned)(2 * a.Hkv * a.d / NC)), dim3(256), 0, st, a);
    return hipGetLastError();
}
template <int RR>
static hipError_t launch_gemv_kd(const UpdateArgs &a, hipStream_t st) {
    const int kd = (a.D + 2047) / 2048;
    if (kd == 1) return launch_gemv<RR, 1>(a, st);
    if (kd == 2) return launch_gemv<RR, 2>(a, st);
    return launch_gemv<RR, 4>(a, st);
}

bool update_uses_gemv(int R, int D, int dtype) { return dtype == MAD_BF16 && R <= kUpdateGemvRows && D <= 8192; }

hipError_t launch_update(const UpdateArgs &a, int dtype, hipStream_t st) {
    if (update_uses_gemv(a.R, a.D, dtype)) {
        if (a.R == 1) return launch_gemv_kd<1>(a, st);
        if (a.R <= 4) return launch_gemv_kd<4>(a, st);
        return launch_gemv_kd<8>(a, st);
    }
    if (dtype == MAD_BF16) {
        dim3 grid((unsigned)(2 * a.Hkv * a.KS)), block(256);
        const size_t lds = update_lds_bytes(a.R, a.d, a.KS, a.stages);
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
