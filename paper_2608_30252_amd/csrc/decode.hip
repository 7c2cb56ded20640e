// decode.hip -- draft decode attention over the compact MASW memory.
//
// One launch computes, for every (sequence b, KV head c), the attention of the
// G = Hq/Hkv query heads of the current token over the logical key sequence
//     [ memory rows 0..mlen-1 (sinks, then slots) | window ring rows 0..wlen-1 | new token ]
// (the working memory M_t of Sec. 3.1) and appends the new token's K/V to the
// window ring in the same pass (Sec. 3.2).
//
// Work decomposition (split-K / flash-decoding):
//   grid = n_splits * units workgroups, units = B * Hkv, 1-D.  Workgroup w
//   handles unit u = w % units and split s = w / units, a contiguous range of
//   `chunk` keys.  When units is a multiple of 8 every split of one unit lands
//   on the same XCD (workgroups are dealt round-robin to the 8 XCDs), so a
//   unit's partial results and its arrival counter stay in one L2.
//   Inside a workgroup (256 threads) keys stream through LDS in tiles:
//     1. every thread loads 16-byte pieces of the tile's K and V rows into
//        registers (coalesced, issued one tile ahead of use) and stores them to
//        LDS; K rows are XOR-swizzled by 16-byte chunk to keep the QK reads
//        bank-conflict free;
//     2. QK: thread <-> (key, query head) pair, full dot product from LDS with
//        the query kept in registers (K is read once from HBM and shared by
//        the G heads of the group);
//     3. online softmax: per-head tile max by wave shuffles + a 4-wave LDS
//        exchange, exp2 of pre-scaled scores, running (max, sum) rescaling;
//     4. PV: thread <-> (feature pair, key subset) accumulating all G heads,
//        V read once from LDS per thread and key.
//   The last workgroup of a unit to finish (arrival counter) merges the
//   n_splits partial (o, max, sum) triples with the log-sum-exp rule and
//   writes the output, so the whole operation is a single launch.
#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

constexpr int kNT = 256;

template <typename T, int D, int G>
struct DecodeCfg {
    static constexpr int ESZ = (int)sizeof(T);
    static constexpr int VEC = 16 / ESZ;                        // elements per 16-byte chunk
    static constexpr int CPR = D / VEC;                         // chunks per row
    static constexpr int TILE = (16384 / (D * ESZ)) < 64 ? (16384 / (D * ESZ)) : 64;
    static constexpr int RPL = kNT / CPR;                       // rows per load sweep
    static constexpr int NLD = TILE / RPL;                      // load sweeps per tile
    static constexpr int SW = (CPR < 8 ? CPR : 8) - 1;          // swizzle mask
    static constexpr int PAIRS = TILE * G;
    static constexpr int PPT = (PAIRS + kNT - 1) / kNT;         // score pairs per thread
    static constexpr int DP = D / 2;                            // feature pairs
    static constexpr int KS = kNT / DP;                         // key subsets in PV
    static constexpr int KPS = TILE / KS;                       // keys per subset per tile
    static constexpr int NW = kNT / 64;
    // LDS carve-up (bytes): a fixed head for reductions, then one region
    // shared by the tile buffers, the final reduction and the split merge.
    static constexpr int SZ_HEAD = ((2 * NW + 2) * G * 4 + 15) / 16 * 16;
    static constexpr int SZ_K = TILE * D * ESZ;
    static constexpr int SZ_TILE = 2 * SZ_K + TILE * G * 4;
    static constexpr int SZ_FIN = KS * G * D * 4;
    static constexpr int SZ_CMB = kDecodeMaxSplits * G * 8;
    static constexpr int SZ_UNI = SZ_TILE > SZ_FIN ? (SZ_TILE > SZ_CMB ? SZ_TILE : SZ_CMB)
                                                   : (SZ_FIN > SZ_CMB ? SZ_FIN : SZ_CMB);
    static constexpr int SMEM = SZ_HEAD + SZ_UNI;
    static_assert((2 * NW + 2) * G * 4 <= SZ_HEAD, "lds head");
    static_assert(D % VEC == 0 && kNT % CPR == 0 && TILE % RPL == 0, "tile shape");
    static_assert(kNT % DP == 0 && TILE % KS == 0, "pv shape");
    static_assert(kNT % G == 0, "group");
};

// q . k over one 16-byte chunk (VEC elements), q held as fp32 (F32) or as
// packed bf16 pairs (BF16), accumulated in fp32.
__device__ __forceinline__ float chunk_dot(const float *qf, const uint4 &kv, float acc, float) {
    acc = fmaf(qf[0], __uint_as_float(kv.x), acc);
    acc = fmaf(qf[1], __uint_as_float(kv.y), acc);
    acc = fmaf(qf[2], __uint_as_float(kv.z), acc);
    acc = fmaf(qf[3], __uint_as_float(kv.w), acc);
    return acc;
}

typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, a),
                                           __builtin_bit_cast(bf16x2_v, b), c, false);
}
__device__ __forceinline__ float chunk_dot(const uint32_t *qp, const uint4 &kv, float acc, bf16_t) {
    acc = dot2_bf16(qp[0], kv.x, acc);
    acc = dot2_bf16(qp[1], kv.y, acc);
    acc = dot2_bf16(qp[2], kv.z, acc);
    acc = dot2_bf16(qp[3], kv.w, acc);
    return acc;
}

template <typename T> struct QReg;
template <> struct QReg<float> { typedef float type; static constexpr int PER_CHUNK = 4; };
template <> struct QReg<bf16_t> { typedef uint32_t type; static constexpr int PER_CHUNK = 4; };

template <typename T, int D, int G>
__global__ __launch_bounds__(kNT) void decode_kernel(const DecodeArgs a) {
    using C = DecodeCfg<T, D, G>;
    using QT = typename QReg<T>::type;
    __shared__ __align__(16) unsigned char smem[C::SMEM];
    // fixed head of LDS: per-wave reductions and per-head totals
    float *sRedM = reinterpret_cast<float *>(smem);                  // [NW][G]
    float *sRedL = sRedM + C::NW * G;                                 // [NW][G]
    float *sFin = sRedL + C::NW * G;                                  // [G][2] (max, sum)
    unsigned char *uni = smem + C::SZ_HEAD;                           // union region
    uint4 *sK = reinterpret_cast<uint4 *>(uni);                       // [TILE][CPR] swizzled
    uint4 *sV = reinterpret_cast<uint4 *>(uni + C::SZ_K);             // [TILE][CPR]
    float *sP = reinterpret_cast<float *>(uni + 2 * C::SZ_K);         // [TILE][G]
    float *sO = reinterpret_cast<float *>(uni);                       // [KS][G][D] after the tiles
    float2 *sML = reinterpret_cast<float2 *>(uni);                    // [n_splits][G] in the merge

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int units = a.units;
    const int u = blockIdx.x % units, s = blockIdx.x / units;
    const int b = u / a.Hkv, c = u - b * a.Hkv;
    const int mlen = a.mlen[b], wlen = a.wlen[b], wst = a.wstart[b];
    const bool has_new = a.kn != nullptr;
    const int n = mlen + wlen + (has_new ? 1 : 0);
    const int k0 = s * a.chunk;
    const int k1 = min(n, k0 + a.chunk);
    const int w_cap = a.w_cap;

    const T *mk = reinterpret_cast<const T *>(a.mk) + b * a.m_seq + c * a.m_head;
    const T *mv = reinterpret_cast<const T *>(a.mv) + b * a.m_seq + c * a.m_head;
    T *wk = reinterpret_cast<T *>(a.wk) + b * a.w_seq + c * a.w_head;
    T *wv = reinterpret_cast<T *>(a.wv) + b * a.w_seq + c * a.w_head;
    const size_t nrow = ((size_t)b * a.Hkv + c) * D;
    const T *nk = has_new ? reinterpret_cast<const T *>(a.kn) + nrow : nullptr;
    const T *nv = has_new ? reinterpret_cast<const T *>(a.vn) + nrow : nullptr;

    // the workgroup whose range holds the new token appends it to the window ring
    if (has_new && k0 <= n - 1 && n - 1 < k1 && tid < 2 * C::CPR) {
        int r = wst + wlen;
        if (r >= w_cap) r -= w_cap;
        const int ch = tid % C::CPR;
        if (tid < C::CPR)
            reinterpret_cast<uint4 *>(wk + (size_t)r * D)[ch] = reinterpret_cast<const uint4 *>(nk)[ch];
        else
            reinterpret_cast<uint4 *>(wv + (size_t)r * D)[ch] = reinterpret_cast<const uint4 *>(nv)[ch];
    }

    // ---- query of this thread's head (fixed per thread: kNT % G == 0) ----
    const int g_me = tid % G;
    QT qreg[C::CPR * 4];
    {
        const uint4 *qsrc = reinterpret_cast<const uint4 *>(
            reinterpret_cast<const T *>(a.q) + ((size_t)b * a.Hq + (size_t)c * G + g_me) * D);
        #pragma unroll
        for (int ch = 0; ch < C::CPR; ++ch) {
            uint4 v = qsrc[ch];
            qreg[ch * 4 + 0] = __builtin_bit_cast(QT, v.x);
            qreg[ch * 4 + 1] = __builtin_bit_cast(QT, v.y);
            qreg[ch * 4 + 2] = __builtin_bit_cast(QT, v.z);
            qreg[ch * 4 + 3] = __builtin_bit_cast(QT, v.w);
        }
    }

    // ---- running softmax state (identical in every thread) and accumulators ----
    float m_run[G];
    float l_acc = 0.f;           // partial sum for head g_me over this thread's pairs
    float o_acc[G][2];
    #pragma unroll
    for (int g = 0; g < G; ++g) { m_run[g] = -INFINITY; o_acc[g][0] = o_acc[g][1] = 0.f; }

    const int ld_row = tid / C::CPR, ld_ch = tid % C::CPR;
    const int pv_dp = tid % C::DP, pv_ks = tid / C::DP;

    // address of logical key row kidx (K or V) of this unit
    auto row_ptr = [&](int kidx, const T *mb, const T *wb, const T *nb) -> const T * {
        if (kidx < mlen) return mb + (size_t)kidx * D;
        int i = kidx - mlen;
        if (i < wlen) {
            int r = wst + i;
            if (r >= w_cap) r -= w_cap;
            return wb + (size_t)r * D;
        }
        return nb;
    };

    uint4 kreg[C::NLD], vreg[C::NLD];
    auto load_tile = [&](int base) {
        #pragma unroll
        for (int l = 0; l < C::NLD; ++l) {
            int kidx = base + l * C::RPL + ld_row;
            if (kidx < k1) {
                kreg[l] = reinterpret_cast<const uint4 *>(row_ptr(kidx, mk, wk, nk))[ld_ch];
                vreg[l] = reinterpret_cast<const uint4 *>(row_ptr(kidx, mv, wv, nv))[ld_ch];
            } else {
                kreg[l] = make_uint4(0, 0, 0, 0);
                vreg[l] = make_uint4(0, 0, 0, 0);
            }
        }
    };

    if (k0 < k1) load_tile(k0);

    for (int base = k0; base < k1; base += C::TILE) {
        __syncthreads();  // the previous tile is fully consumed
        #pragma unroll
        for (int l = 0; l < C::NLD; ++l) {
            int row = l * C::RPL + ld_row;
            sK[row * C::CPR + (ld_ch ^ (row & C::SW))] = kreg[l];
            sV[row * C::CPR + ld_ch] = vreg[l];
        }
        if (base + C::TILE < k1) load_tile(base + C::TILE);   // prefetch the next tile
        __syncthreads();

        // ---- QK: scores of (key j, head g) pairs, j = pr / G, g = pr % G ----
        float sc[C::PPT];
        float tmax = -INFINITY;
        #pragma unroll
        for (int pp = 0; pp < C::PPT; ++pp) {
            int pr = tid + pp * kNT;
            sc[pp] = -INFINITY;
            if (pr < C::PAIRS) {
                int j = pr / G;
                float acc = 0.f;
                #pragma unroll
                for (int ch = 0; ch < C::CPR; ++ch) {
                    uint4 kv = sK[j * C::CPR + (ch ^ (j & C::SW))];
                    acc = chunk_dot(&qreg[ch * 4], kv, acc, T{});
                }
                if (base + j < k1) sc[pp] = acc * a.scale_log2;
            }
            tmax = fmaxf(tmax, sc[pp]);
        }
        // per-head tile max: lanes sharing lane % G hold the same head
        tmax = strided_max<G>(tmax);
        if (lane < G) sRedM[wave * G + lane] = tmax;
        __syncthreads();
        float alpha[G];
        float m_me = 0.f, alpha_me = 0.f;
        #pragma unroll
        for (int g = 0; g < G; ++g) {
            float mt = sRedM[g];
            #pragma unroll
            for (int w = 1; w < C::NW; ++w) mt = fmaxf(mt, sRedM[w * G + g]);
            float mn = fmaxf(m_run[g], mt);
            alpha[g] = exp2f(m_run[g] - mn);   // 0 while m_run is -inf
            m_run[g] = mn;
            if (g == g_me) { m_me = mn; alpha_me = alpha[g]; }
        }
        float lsum = 0.f;
        #pragma unroll
        for (int pp = 0; pp < C::PPT; ++pp) {
            int pr = tid + pp * kNT;
            if (pr < C::PAIRS) {
                float p = exp2f(sc[pp] - m_me);
                sP[pr] = p;
                lsum += p;
            }
        }
        l_acc = l_acc * alpha_me + lsum;
        __syncthreads();

        // ---- PV: o[g][2dp..2dp+1] += sum over this subset's keys of p[j][g] * V[j] ----
        #pragma unroll
        for (int g = 0; g < G; ++g) { o_acc[g][0] *= alpha[g]; o_acc[g][1] *= alpha[g]; }
        #pragma unroll 4
        for (int kk = 0; kk < C::KPS; ++kk) {
            int j = pv_ks * C::KPS + kk;
            float v0, v1;
            if constexpr (sizeof(T) == 2) {
                uint32_t w = reinterpret_cast<const uint32_t *>(sV)[j * (D / 2) + pv_dp];
                v0 = bf16_lo(w); v1 = bf16_hi(w);
            } else {
                float2 w = reinterpret_cast<const float2 *>(sV)[j * (D / 2) + pv_dp];
                v0 = w.x; v1 = w.y;
            }
            const float *pj = sP + j * G;
            #pragma unroll
            for (int g = 0; g < G; ++g) {
                float p = pj[g];
                o_acc[g][0] = fmaf(p, v0, o_acc[g][0]);
                o_acc[g][1] = fmaf(p, v1, o_acc[g][1]);
            }
        }
    }

    // ---- reduce inside the workgroup ----
    l_acc = strided_sum<G>(l_acc);
    if (lane < G) sRedL[wave * G + lane] = l_acc;
    __syncthreads();   // tiles consumed, sRedL complete
    if (tid < G) {
        float t = 0.f;
        #pragma unroll
        for (int w = 0; w < C::NW; ++w) t += sRedL[w * G + tid];
        float mm = 0.f;
        #pragma unroll
        for (int g = 0; g < G; ++g) if (g == tid) mm = m_run[g];
        sFin[2 * tid] = mm;
        sFin[2 * tid + 1] = t;
    }
    #pragma unroll
    for (int g = 0; g < G; ++g) {
        sO[(pv_ks * G + g) * D + 2 * pv_dp] = o_acc[g][0];
        sO[(pv_ks * G + g) * D + 2 * pv_dp + 1] = o_acc[g][1];
    }
    __syncthreads();

    const int n_splits = a.n_splits;
    const size_t head0 = (size_t)b * a.Hq + (size_t)c * G;
    T *out = reinterpret_cast<T *>(a.out) + head0 * D;
    if (n_splits == 1) {
        for (int idx = tid; idx < G * D; idx += kNT) {
            int g = idx / D;
            float o = 0.f;
            #pragma unroll
            for (int ks = 0; ks < C::KS; ++ks) o += sO[ks * G * D + idx];
            float mm = sFin[2 * g], l = sFin[2 * g + 1];
            Elem<T>::store1(out + idx, l > 0.f ? o / l : 0.f);
            if (a.lse && (idx % D) == 0) a.lse[head0 + g] = l > 0.f ? (mm + log2f(l)) * kLn2 : -INFINITY;
        }
        return;
    }

    // ---- write this split's partial (unnormalised o, running max, running sum) ----
    float *po = a.part_o + ((size_t)u * n_splits + s) * G * D;
    for (int idx = tid; idx < G * D; idx += kNT) {
        float o = 0.f;
        #pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) o += sO[ks * G * D + idx];
        po[idx] = o;
    }
    if (tid < G)
        reinterpret_cast<float2 *>(a.part_ml)[((size_t)u * n_splits + s) * G + tid] =
            make_float2(sFin[2 * tid], sFin[2 * tid + 1]);
    __threadfence();           // release the partials at device scope
    __syncthreads();
    __shared__ int s_last;
    if (tid == 0) {
        unsigned prev = atomicAdd(&a.counters[u], 1u);
        s_last = (prev == (unsigned)(n_splits - 1));
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();           // acquire the other workgroups' partials

    // ---- last workgroup of the unit: log-sum-exp merge of the splits ----
    const float2 *pml = reinterpret_cast<const float2 *>(a.part_ml) + (size_t)u * n_splits * G;
    for (int idx = tid; idx < n_splits * G; idx += kNT) sML[idx] = pml[idx];
    __syncthreads();
    const float *pob = a.part_o + (size_t)u * n_splits * G * D;
    for (int idx = tid; idx < G * D; idx += kNT) {
        int g = idx / D;
        float M = -INFINITY;
        for (int sp = 0; sp < n_splits; ++sp) M = fmaxf(M, sML[sp * G + g].x);
        float acc = 0.f, L = 0.f;
        if (M != -INFINITY) {
            #pragma unroll 8
            for (int sp = 0; sp < n_splits; ++sp) {
                float2 ml = sML[sp * G + g];
                float wgt = exp2f(ml.x - M);
                L = fmaf(wgt, ml.y, L);
                acc = fmaf(wgt, pob[(size_t)sp * G * D + idx], acc);
            }
        }
        Elem<T>::store1(out + idx, L > 0.f ? acc / L : 0.f);
        if (a.lse && (idx % D) == 0) a.lse[head0 + g] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
    }
    if (tid == 0) a.counters[u] = 0u;   // leave the counter ready for the next call
}

// ------------------------------------------------------------------ host ----

DecodePlan plan_decode(int B, int Hkv, const int *n_keys) {
    DecodePlan p;
    p.units = B * Hkv;
    p.n_max = 0;
    for (int b = 0; b < B; ++b) p.n_max = n_keys[b] > p.n_max ? n_keys[b] : p.n_max;
    int fill = (kDecodeTargetWGs + p.units - 1) / p.units;
    if (fill > kDecodeMaxSplits) fill = kDecodeMaxSplits;
    if (fill < 1) fill = 1;
    int chunk = (p.n_max + fill - 1) / fill;
    chunk = ((chunk + kDecodeChunkQuant - 1) / kDecodeChunkQuant) * kDecodeChunkQuant;
    if (chunk < kDecodeMinChunk) chunk = kDecodeMinChunk;
    int ns = (p.n_max + chunk - 1) / chunk;
    if (ns < 1) ns = 1;
    p.n_splits = ns;
    p.chunk = chunk;
    return p;
}

size_t decode_ws_bytes(int B, int Hq, int Hkv, int d) {
    size_t units = (size_t)B * Hkv;
    int G = Hq / Hkv;
    size_t fill = (kDecodeTargetWGs + units - 1) / units;
    if (fill > (size_t)kDecodeMaxSplits) fill = kDecodeMaxSplits;
    return align256(units * 4) + align256(units * fill * G * d * 4) + align256(units * fill * G * 8);
}

template <typename T, int D, int G>
static hipError_t launch_t(const DecodeArgs &a, hipStream_t st) {
    dim3 grid((unsigned)(a.units * a.n_splits)), block(kNT);
    hipLaunchKernelGGL((decode_kernel<T, D, G>), grid, block, 0, st, a);
    return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_g(const DecodeArgs &a, int G, hipStream_t st) {
    switch (G) {
        case 1: return launch_t<T, D, 1>(a, st);
        case 2: return launch_t<T, D, 2>(a, st);
        case 4: return launch_t<T, D, 4>(a, st);
        case 8: return launch_t<T, D, 8>(a, st);
        case 16: return launch_t<T, D, 16>(a, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_decode(const DecodeArgs &a, int dtype, int d, int G, hipStream_t st) {
    if (dtype == MAD_BF16) {
        if (d == 64) return launch_g<bf16_t, 64>(a, G, st);
        if (d == 128) return launch_g<bf16_t, 128>(a, G, st);
    } else {
        if (d == 64) return launch_g<float, 64>(a, G, st);
        if (d == 128) return launch_g<float, 128>(a, G, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace mad
