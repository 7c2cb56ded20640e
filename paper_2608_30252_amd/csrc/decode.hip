// decode.hip -- draft decode attention over the compact MASW memory.
//
// One launch computes, for every (sequence b, KV head c), the attention of the
// G = Hq/Hkv query heads of the current token over the logical key sequence
//     [ memory rows 0..mlen-1 (sinks, then slots) | window ring rows 0..wlen-1 | new token ]
// (the working memory M_t of Sec. 3.1) and appends the new token's K/V to the
// window ring in the same pass (Sec. 3.2).
//
// Work decomposition (split-K / flash-decoding), grid = n_splits * units
// workgroups of 256 threads, units = B * Hkv; workgroup w handles unit
// u = w % units and the s = w / units-th range of `chunk` keys.
//
// Inside a workgroup keys stream through LDS in tiles of 8 KB of K + 8 KB of V
// (64 keys for bf16, head_dim 64):
//   * loads go straight from HBM into LDS (global_load_lds_dwordx4, 16 bytes a
//     lane, no VGPR round trip) through a 4-stage ring, so up to three tiles
//     are in flight while one is consumed; K rows are XOR-swizzled by 16-byte
//     chunk on the way in so the QK reads are bank-conflict free;
//   * QK: one wave per query head of the GQA group, one lane per key; the
//     full head_dim dot product comes from LDS (K is read once from HBM and
//     shared by the G heads);
//   * online softmax on exp2 of pre-scaled scores; the per-head tile max is a
//     single in-wave DPP/swizzle reduction; for the PV product the
//     probabilities are rounded to bf16 and packed in key pairs (the softmax
//     normaliser keeps the fp32 values);
//   * PV: thread <-> (feature pair, key subset) for all G heads at once, two
//     keys per v_dot2_f32_bf16 (fp32 accumulation);
//   * the last workgroup of a unit (one arrival counter per unit, on its own
//     256-byte line) pulls every split's partial (o, max, sum) into LDS with
//     device-coherent direct loads in a single round trip and merges them with
//     the log-sum-exp rule.
#include <type_traits>

#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

constexpr int kNT = 256;
constexpr int kStages = 4;
constexpr int kStageBytes = 16384;   // 8 KB of K + 8 KB of V

template <typename T, int D, int G>
struct DecodeCfg {
    static constexpr int ESZ = (int)sizeof(T);
    static constexpr int RB = D * ESZ;                 // bytes per K/V row
    static constexpr int TILE = 8192 / RB;             // keys per tile
    static constexpr int CPR = RB / 16;                // 16-byte chunks per row
    static constexpr int SW = (CPR < 8 ? CPR : 8) - 1; // K swizzle mask
    static constexpr int RPI = 1024 / RB;              // rows per wave load (64 lanes x 16 B)
    static constexpr int LPT = 2;                      // K (and V) loads per thread per tile
    static constexpr int PAIRS = TILE * G;             // (head, key) score pairs per tile
    static constexpr int PPT = (PAIRS + kNT - 1) / kNT;
    static constexpr int DP = D / 2;                   // feature pairs
    static constexpr int KS = kNT / DP;                // key subsets in PV
    static constexpr int KPS = TILE / KS;              // keys per subset per tile
    static constexpr bool BF = std::is_same<T, bf16_t>::value;
    // LDS layout: [stages | P | alpha | fin | O]; the merge reuses [stages]
    static constexpr int OFF_P = kStages * kStageBytes;
    static constexpr int SZ_P = TILE * G * 4;
    static constexpr int OFF_ALPHA = OFF_P + SZ_P;
    static constexpr int OFF_FIN = OFF_ALPHA + G * 4;
    static constexpr int OFF_O = OFF_FIN + G * 8;
    static constexpr int SZ_O = KS * G * D * 4;
    static constexpr int SMEM = OFF_O + SZ_O;
    static_assert(TILE * RB == 8192 && kNT / 64 * LPT * 1024 == 8192, "tile = 8 KB per tensor");
    static_assert(KPS % 2 == 0 && kNT % DP == 0 && TILE % KS == 0, "pv shape");
    static_assert(PAIRS % TILE == 0 && (kNT % TILE == 0), "score pair groups");
};

// vmcnt(n) for n in {0, 4, 8, 12} (the tile loads are the only vector memory
// operations in flight inside the pipeline; 4 per tile and thread).
__device__ __forceinline__ void wait_vmcnt(int n) {
    switch (n) {
        case 0: __builtin_amdgcn_s_waitcnt(0x0F70); break;
        case 4: __builtin_amdgcn_s_waitcnt(0x0F74); break;
        case 8: __builtin_amdgcn_s_waitcnt(0x0F78); break;
        default: __builtin_amdgcn_s_waitcnt(0x0F7C); break;   // 12
    }
}

typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, a), __builtin_bit_cast(bf16x2_v, b), c,
                                           false);
}

// Max over aligned groups of N consecutive lanes (all lanes must be active).
template <int N> __device__ __forceinline__ float group_max(float v) {
    if constexpr (N >= 2) v = fmaxf(v, xor_lane<1>(v));
    if constexpr (N >= 4) v = fmaxf(v, xor_lane<2>(v));
    if constexpr (N >= 8) v = fmaxf(v, xor_lane<4>(v));
    if constexpr (N >= 16) v = fmaxf(v, xor_lane<8>(v));
    if constexpr (N >= 32) v = fmaxf(v, xor_lane<16>(v));
    if constexpr (N >= 64) v = fmaxf(v, xor_lane<32>(v));
    return v;
}

template <typename T, int D, int G>
__global__ __launch_bounds__(kNT, 2) void decode_kernel(const DecodeArgs a) {
    using C = DecodeCfg<T, D, G>;
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char *sStage = smem;
    float *sAlpha = reinterpret_cast<float *>(smem + C::OFF_ALPHA);   // [G]
    float *sFin = reinterpret_cast<float *>(smem + C::OFF_FIN);       // [G][2]: max, sum
    float *sO = reinterpret_cast<float *>(smem + C::OFF_O);           // [KS][G][D]

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

    // ---- queries of this thread's score pairs (head g = pair / TILE) ----
    // With 64-key tiles a wave's score pairs share one head, so its query row is
    // wave-uniform and comes through the scalar cache (no vector-memory wait);
    // otherwise each lane loads its own row.
    constexpr int QW = D * C::ESZ / 4;   // 32-bit words of one query row
    uint32_t qreg[C::PPT][QW];
    #pragma unroll
    for (int pp = 0; pp < C::PPT; ++pp) {
        const int pr = tid + pp * kNT;
        const int g = (pr < C::PAIRS ? pr : 0) / C::TILE;
        const T *qrow = reinterpret_cast<const T *>(a.q) + ((size_t)b * a.Hq + (size_t)c * G + g) * D;
        if constexpr (C::TILE == 64) {
            load_uniform_dwords<QW>(qrow, qreg[pp]);
        } else {
            const uint4 *qs = reinterpret_cast<const uint4 *>(qrow);
            #pragma unroll
            for (int ch = 0; ch < C::CPR; ++ch) {
                const uint4 v = qs[ch];
                qreg[pp][4 * ch + 0] = v.x; qreg[pp][4 * ch + 1] = v.y;
                qreg[pp][4 * ch + 2] = v.z; qreg[pp][4 * ch + 3] = v.w;
            }
        }
    }

    // ---- append the new token to the window ring (the workgroup holding it) ----
    if (has_new && k0 <= n - 1 && n - 1 < k1) {
        if (tid < 2 * C::CPR) {
            int r = wst + wlen;
            if (r >= w_cap) r -= w_cap;
            const int ch = tid % C::CPR;
            if (tid < C::CPR)
                reinterpret_cast<uint4 *>(wk + (size_t)r * D)[ch] = reinterpret_cast<const uint4 *>(nk)[ch];
            else
                reinterpret_cast<uint4 *>(wv + (size_t)r * D)[ch] = reinterpret_cast<const uint4 *>(nv)[ch];
        }
    }
    // Vector-memory operations issued above are older than every tile load, so
    // the per-tile vmcnt waits below also cover them.

    // ---- tile loader: direct HBM -> LDS, 2 K + 2 V instructions per thread ----
    auto row_src = [&](int kidx, bool is_v) -> const T * {
        if (kidx >= k1) kidx = k1 - 1;   // rows past the range load a valid row (weight 0)
        if (kidx < mlen) return (is_v ? mv : mk) + (size_t)kidx * D;
        const int i = kidx - mlen;
        if (i < wlen) {
            int r = wst + i;
            if (r >= w_cap) r -= w_cap;
            return (is_v ? wv : wk) + (size_t)r * D;
        }
        return is_v ? nv : nk;
    };
    auto issue_tile = [&](int tile_base, int stage) {
        unsigned char *st = sStage + stage * kStageBytes;
        #pragma unroll
        for (int l = 0; l < C::LPT; ++l) {
            const int inst = l * 4 + wave;                 // 1 KB block of the 8 KB tensor tile
            const int row = inst * C::RPI + lane / C::CPR;
            const int slot = lane % C::CPR;
            const int kidx = tile_base + row;
            const T *kp = row_src(kidx, false);
            const T *vp = row_src(kidx, true);
            // K: LDS slot `slot` of row `row` holds global chunk slot ^ (row & SW)
            lds_stream16(reinterpret_cast<const uint4 *>(kp) + (slot ^ (row & C::SW)), st + inst * 1024);
            lds_stream16(reinterpret_cast<const uint4 *>(vp) + slot, st + 8192 + inst * 1024);
        }
    };

    // ---- running state ----
    float m_run[C::PPT], l_lane[C::PPT];
    #pragma unroll
    for (int pp = 0; pp < C::PPT; ++pp) { m_run[pp] = -INFINITY; l_lane[pp] = 0.f; }
    float o_acc[G][2];
    #pragma unroll
    for (int g = 0; g < G; ++g) o_acc[g][0] = o_acc[g][1] = 0.f;
    const int pv_dp = tid % C::DP, pv_ks = tid / C::DP;

    const int ntiles = (k1 > k0) ? (k1 - k0 + C::TILE - 1) / C::TILE : 0;
    int issued = 0;
    for (; issued < ntiles && issued < kStages - 1; ++issued) issue_tile(k0 + issued * C::TILE, issued);

    for (int t = 0; t < ntiles; ++t) {
        wait_vmcnt(4 * (issued - t - 1));
        __syncthreads();   // tile t is in LDS for every wave; stage (t-1) % kStages is free
        if (issued < ntiles) {
            issue_tile(k0 + issued * C::TILE, issued % kStages);
            ++issued;
        }
        const unsigned char *st = sStage + (t % kStages) * kStageBytes;
        const int base = k0 + t * C::TILE;

        // ---- QK and softmax statistics: pair (g = pr / TILE, j = pr % TILE) ----
        #pragma unroll
        for (int pp = 0; pp < C::PPT; ++pp) {
            const int pr = tid + pp * kNT;
            const bool act = pr < C::PAIRS;
            const int j = pr % C::TILE, g = (act ? pr : 0) / C::TILE;
            float acc = 0.f;
            const uint4 *krow = reinterpret_cast<const uint4 *>(st + j * C::RB);
            #pragma unroll
            for (int ch = 0; ch < C::CPR; ++ch) {
                const uint4 kv = krow[ch ^ (j & C::SW)];
                if constexpr (C::BF) {
                    acc = dot2_bf16(qreg[pp][4 * ch + 0], kv.x, acc);
                    acc = dot2_bf16(qreg[pp][4 * ch + 1], kv.y, acc);
                    acc = dot2_bf16(qreg[pp][4 * ch + 2], kv.z, acc);
                    acc = dot2_bf16(qreg[pp][4 * ch + 3], kv.w, acc);
                } else {
                    acc = fmaf(__uint_as_float(qreg[pp][4 * ch + 0]), __uint_as_float(kv.x), acc);
                    acc = fmaf(__uint_as_float(qreg[pp][4 * ch + 1]), __uint_as_float(kv.y), acc);
                    acc = fmaf(__uint_as_float(qreg[pp][4 * ch + 2]), __uint_as_float(kv.z), acc);
                    acc = fmaf(__uint_as_float(qreg[pp][4 * ch + 3]), __uint_as_float(kv.w), acc);
                }
            }
            const float sc = (base + j < k1) ? acc * a.scale_log2 : -INFINITY;
            const float tmax = group_max<C::TILE>(sc);
            const float mn = fmaxf(m_run[pp], tmax);      // finite: every tile holds a valid key
            const float alpha = exp2f(m_run[pp] - mn);
            m_run[pp] = mn;
            const float p = exp2f(sc - mn);
            if constexpr (C::BF) {
                // PV consumes the probabilities rounded to bf16 and packed by key
                // pairs; the normaliser below sums the fp32 values
                const uint32_t pb = (uint32_t)f32_to_bf16(p);
                const uint32_t pn = (uint32_t)__float_as_int(xor_lane<1>(__int_as_float((int)pb)));
                if (act && (j & 1) == 0)
                    reinterpret_cast<uint32_t *>(smem + C::OFF_P)[(j >> 1) * G + g] = pb | (pn << 16);
            } else {
                if (act) reinterpret_cast<float *>(smem + C::OFF_P)[j * G + g] = p;
            }
            l_lane[pp] = fmaf(l_lane[pp], alpha, p);
            if (act && j == 0) sAlpha[g] = alpha;
        }
        __syncthreads();   // P and alpha ready

        // ---- PV ----
        float al[G];
        #pragma unroll
        for (int g = 0; g < G; ++g) al[g] = sAlpha[g];
        #pragma unroll
        for (int g = 0; g < G; ++g) { o_acc[g][0] *= al[g]; o_acc[g][1] *= al[g]; }
        const unsigned char *sv = st + 8192;
        #pragma unroll
        for (int kk = 0; kk < C::KPS; kk += 2) {
            const int j0 = pv_ks * C::KPS + kk;
            if constexpr (C::BF) {
                const uint32_t w0 = reinterpret_cast<const uint32_t *>(sv + j0 * C::RB)[pv_dp];
                const uint32_t w1 = reinterpret_cast<const uint32_t *>(sv + (j0 + 1) * C::RB)[pv_dp];
                const uint32_t lo = __builtin_amdgcn_perm(w1, w0, 0x05040100u);   // feature 2dp, keys j0 | j0+1
                const uint32_t hi = __builtin_amdgcn_perm(w1, w0, 0x07060302u);   // feature 2dp+1
                const uint32_t *pj = reinterpret_cast<const uint32_t *>(smem + C::OFF_P) + (j0 >> 1) * G;
                #pragma unroll
                for (int g = 0; g < G; ++g) {
                    const uint32_t pg = pj[g];
                    o_acc[g][0] = dot2_bf16(pg, lo, o_acc[g][0]);
                    o_acc[g][1] = dot2_bf16(pg, hi, o_acc[g][1]);
                }
            } else {
                #pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const float2 w = reinterpret_cast<const float2 *>(sv + (j0 + e) * C::RB)[pv_dp];
                    const float *pj = reinterpret_cast<const float *>(smem + C::OFF_P) + (j0 + e) * G;
                    #pragma unroll
                    for (int g = 0; g < G; ++g) {
                        o_acc[g][0] = fmaf(pj[g], w.x, o_acc[g][0]);
                        o_acc[g][1] = fmaf(pj[g], w.y, o_acc[g][1]);
                    }
                }
            }
        }
    }

    // ---- per-head totals: lanes of one pair group share a head ----
    #pragma unroll
    for (int pp = 0; pp < C::PPT; ++pp) {
        const int pr = tid + pp * kNT;
        float lt = l_lane[pp];
        #pragma unroll
        for (int k = 1; k < C::TILE; k <<= 1) lt += __shfl_xor(lt, k, 64);
        if (pr < C::PAIRS && pr % C::TILE == 0) {
            const int g = pr / C::TILE;
            sFin[2 * g] = m_run[pp];   // -inf when this split had no keys
            sFin[2 * g + 1] = lt;
        }
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
            const int g = idx / D;
            float o = 0.f;
            #pragma unroll
            for (int ks = 0; ks < C::KS; ++ks) o += sO[ks * G * D + idx];
            const float mm = sFin[2 * g], l = sFin[2 * g + 1];
            Elem<T>::store1(out + idx, l > 0.f ? o / l : 0.f);
            if (a.lse && (idx % D) == 0) a.lse[head0 + g] = l > 0.f ? (mm + log2f(l)) * kLn2 : -INFINITY;
        }
        return;
    }

    // ---- partial of this split: unit block = [o: n_splits][G][D] [ml: n_splits][G][2] ----
    float *blk = a.part + (size_t)u * a.part_stride;
    float *po = blk + (size_t)s * G * D;
    for (int idx = tid; idx < G * D; idx += kNT) {
        float o = 0.f;
        #pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) o += sO[ks * G * D + idx];
        store_agent(po + idx, o);
    }
    if (tid < 2 * G) store_agent(blk + (size_t)n_splits * G * D + (size_t)s * 2 * G + tid, sFin[tid]);
    wait_vm_stores();
    __syncthreads();
    __shared__ int s_last;
    if (tid == 0) {
        unsigned *cnt = a.counters + (size_t)u * kCounterStride;
        const int last = arrive(cnt) == (unsigned)(n_splits - 1);
        if (last) reset_counter(cnt);
        s_last = last;
    }
    __syncthreads();
    if (!s_last) return;

    // ---- last workgroup: pull all partials into LDS in one round trip ----
    const int nbytes = (n_splits * G * (D + 2) * 4 + 15) & ~15;   // inside the 256-byte padded block
    for (int off = wave * 1024; off < nbytes; off += 4096) {
        if (off + lane * 16 < nbytes)
            lds_load16_coherent(reinterpret_cast<const unsigned char *>(blk) + off + lane * 16, sStage + off);
    }
    wait_vmcnt(0);
    __syncthreads();
    const float *lo = reinterpret_cast<const float *>(sStage);
    const float *lml = lo + (size_t)n_splits * G * D;
    for (int idx = tid; idx < G * D; idx += kNT) {
        const int g = idx / D;
        float M = -INFINITY;
        for (int sp = 0; sp < n_splits; ++sp) M = fmaxf(M, lml[sp * 2 * G + 2 * g]);
        float acc = 0.f, L = 0.f;
        if (M != -INFINITY) {
            for (int sp = 0; sp < n_splits; ++sp) {
                const float wgt = exp2f(lml[sp * 2 * G + 2 * g] - M);
                L = fmaf(wgt, lml[sp * 2 * G + 2 * g + 1], L);
                acc = fmaf(wgt, lo[(size_t)sp * G * D + idx], acc);
            }
        }
        Elem<T>::store1(out + idx, L > 0.f ? acc / L : 0.f);
        if (a.lse && (idx % D) == 0) a.lse[head0 + g] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
    }
}

// ------------------------------------------------------------------ host ----

int decode_max_splits(int d, int G) {
    const int cap = kStages * kStageBytes / (G * (d + 2) * 4);   // merge block must fit the stage LDS
    return cap < kDecodeMaxSplits ? cap : kDecodeMaxSplits;
}

static int decode_tile(int dtype, int d) { return 8192 / (d * (dtype == MAD_BF16 ? 2 : 4)); }

DecodePlan plan_decode(int B, int Hkv, int G, int d, int dtype, const int *n_keys) {
    DecodePlan p;
    p.units = B * Hkv;
    p.n_max = 0;
    for (int b = 0; b < B; ++b) p.n_max = n_keys[b] > p.n_max ? n_keys[b] : p.n_max;
    const int tile = decode_tile(dtype, d);
    int ns = (kDecodeTargetWGs + p.units - 1) / p.units;
    const int cap = decode_max_splits(d, G);
    if (ns > cap) ns = cap;
    if (ns < 1) ns = 1;
    int chunk = (p.n_max + ns - 1) / ns;
    chunk = ((chunk + tile - 1) / tile) * tile;
    if (chunk < tile) chunk = tile;
    ns = (p.n_max + chunk - 1) / chunk;
    p.n_splits = ns < 1 ? 1 : ns;
    p.chunk = chunk;
    return p;
}

// floats per unit block, rounded to 256 bytes (the merge loads whole 16-byte pieces)
size_t decode_part_stride(int d, int G) {
    return ((size_t)decode_max_splits(d, G) * G * (d + 2) + 63) / 64 * 64;
}

size_t decode_ws_bytes(int B, int Hq, int Hkv, int d) {
    return kCounterRegionBytes + (size_t)B * Hkv * decode_part_stride(d, Hq / Hkv) * 4 + 256;
}

template <typename T, int D, int G>
static hipError_t launch_t(const DecodeArgs &a, hipStream_t st) {
    using C = DecodeCfg<T, D, G>;
    dim3 grid((unsigned)(a.units * a.n_splits)), block(kNT);
    hipLaunchKernelGGL((decode_kernel<T, D, G>), grid, block, C::SMEM, st, a);
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
