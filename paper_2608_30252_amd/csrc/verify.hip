// verify.hip -- the target's (gamma+1)-query verify attention over its full KV
// cache (Sec. 2.1 draft-verify paradigm; Sec. 3.3: the verifier keeps the full
// KV).  The T = gamma+1 new tokens' K/V sit at rows len-T .. len-1; query t
// sees rows 0 .. len-T+t.
//
// Both products of attention run on the matrix cores
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation):
//   * the query tile of one (sequence, KV head) unit is the T*G rows
//     (t, g) -> row t*G + g, padded to 16-row blocks;
//   * S^T = K Q^T takes K rows as the A operand.  Key rows are assigned to the
//     A rows with a fixed permutation so that the S^T accumulator already holds,
//     in every lane, the 8 consecutive keys that the next product needs;
//   * O^T = V^T P^T takes its A operand (8 consecutive keys of one feature)
//     either from the verifier's V cache in its natural layout (rows of d
//     features: staged in LDS as they are, 16-byte chunks XOR-swizzled by row,
//     and read back with two transposing LDS reads, ds_read_b64_tr_b16) or from
//     a key-contiguous V^T cache (one run of cap keys per feature: 16 bytes a
//     lane straight from memory); the probabilities come from the lane's own
//     scores (rounded to bf16);
//   * online softmax per query row: the row's 8 scores sit in one lane, the
//     row max needs two cross-lane exchanges.
// Each wave of a workgroup streams its own 32-key slabs (K rows and V^T
// columns, 16 bytes a lane) straight into registers, DEPTH slabs deep:
// the loads of slab i + DEPTH - 1 are issued before slab i is used, so about
// (DEPTH - 1) x 16 KB per wave are in flight -- the register file is a far
// larger buffer than LDS.  The four waves' (max, sum, o) are merged in LDS into
// one split partial; a second small kernel merges the splits of every query row
// with the log-sum-exp rule.
#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

// phase marks of the diagnostic trace build (verify_lds_kernel): 0 entry,
// 1 the split's partial written
MAD_TRACE_BUFFER(mad_trace_verify)

constexpr int kVerifyLdsMinNb = 2;   // query row blocks from which the LDS-staged kernel is used

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_v;
typedef __attribute__((ext_vector_type(4))) float f32x4_v;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_v;

// Lanes l, l^16, l^32, l^48 hold the same query row.  v_permlane16_swap and
// v_permlane32_swap (VALU lane swaps of gfx950) give every lane the values of
// lanes l & ~16 and l | 16 (resp. 32), so two swaps reduce over the four.
__device__ __forceinline__ float max_over_row_lanes(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float sum_over_row_lanes(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// slabs per wave in flight or in use: three where the registers allow it
template <int D, int NB> constexpr int verify_depth() { return D == 128 ? (NB >= 4 ? 1 : NB == 3 ? 2 : 3) : 3; }

template <int D, int NB>
__global__ __launch_bounds__(256) void verify_split_kernel(const VerifyArgs a) {
    constexpr int KST = D / 32;   // 32-feature k steps of the QK product
    constexpr int DB = D / 16;    // 16-feature output blocks of the PV product
    constexpr int RP = NB * 16;   // padded query rows
    constexpr int DEPTH = verify_depth<D, NB>();
    extern __shared__ __align__(16) unsigned char smem[];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u = blockIdx.x % a.units, s = blockIdx.x / a.units;
    const int b = u / a.Hkv, c = u - b * a.Hkv;
    const int len = a.len[b], T = a.T, G = a.G, R = T * G;
    const int k0 = s * a.chunk;
    const int k1 = min(len, k0 + a.chunk);
    const int cap = a.cap;
    const bf16_t *K = reinterpret_cast<const bf16_t *>(a.k) + b * a.seq + c * a.head;
    // V: natural rows [cap][D] (VNAT) or one run of cap keys per feature [D][cap]
    const bf16_t *VT = reinterpret_cast<const bf16_t *>(a.vt) + b * a.seq + c * a.head;
    const int lr = lane & 15, lg = lane >> 4;   // row within a 16-block, lane group

    // ---- query fragments (B operand of S^T = K Q^T) and causal limits ----
    bf16x8_v qf[NB][KST];
    int lim[NB];
    #pragma unroll
    for (int rb = 0; rb < NB; ++rb) {
        const int row = rb * 16 + lr;
        if (row < R) {
            const int t = row / G, g = row - t * G;
            const bf16_t *qrow = reinterpret_cast<const bf16_t *>(a.q) + (((size_t)b * T + t) * a.Hq + c * G + g) * D;
            #pragma unroll
            for (int ks = 0; ks < KST; ++ks) qf[rb][ks] = *reinterpret_cast<const bf16x8_v *>(qrow + ks * 32 + 8 * lg);
            lim[rb] = len - T + t;
        } else {
            #pragma unroll
            for (int ks = 0; ks < KST; ++ks) qf[rb][ks] = bf16x8_v{0, 0, 0, 0, 0, 0, 0, 0};
            lim[rb] = 0x7fffffff;
        }
    }

    int lim_min = lim[0];
    #pragma unroll
    for (int rb = 1; rb < NB; ++rb) lim_min = min(lim_min, lim[rb]);

    // ---- this wave's slabs: keys kb = k0 + 32 wave + 128 i ----
    const int nsl = (k1 > k0 + wave * 32) ? (k1 - k0 - wave * 32 + 127) / 128 : 0;
    // K rows of the two 16-key blocks: A row m of block blk holds key
    // kb + 8*(m/4) + 4*blk + m%4, so accumulator element i of lane group lg is
    // key kb + 8*lg + 4*blk + i.  V^T: feature db*16 + lr, keys kb + 8*lg .. +7.
    bf16x8_v kf[DEPTH][2][KST];
    u32x4_v vw[DEPTH][DB];
    auto load = [&](int i, int buf_k, int buf_v) {
        (void)buf_v;
        const int kb = k0 + wave * 32 + i * 128;
        #pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
            const int key = min(kb + 8 * (lr >> 2) + 4 * blk + (lr & 3), len - 1);   // past len: a valid row, masked
            const bf16_t *krow = K + (size_t)key * D + 8 * lg;
            #pragma unroll
            for (int ks = 0; ks < KST; ++ks) kf[buf_k][blk][ks] = *reinterpret_cast<const bf16x8_v *>(krow + ks * 32);
        }
        int kg = kb + 8 * lg;
        if (kg >= len) kg = (len - 1) & ~7;   // past len: any valid chunk (zeroed when used)
        #pragma unroll
        for (int db = 0; db < DB; ++db)
            vw[buf_v][db] = *reinterpret_cast<const u32x4_v *>(VT + (size_t)(db * 16 + lr) * cap + kg);
    };

    f32x4_v o[DB][NB];
    float m_run[NB], l_run[NB];
    #pragma unroll
    for (int rb = 0; rb < NB; ++rb) {
        m_run[rb] = -INFINITY;
        l_run[rb] = 0.f;
        #pragma unroll
        for (int db = 0; db < DB; ++db) o[db][rb] = f32x4_v{0.f, 0.f, 0.f, 0.f};
    }

    auto compute = [&](int i, int buf) {
        const int kb = k0 + wave * 32 + i * 128;
        const int kg = kb + 8 * lg;
        bf16x8_v vf[DB];
        #pragma unroll
        for (int db = 0; db < DB; ++db) {
            u32x4_v w = vw[buf][db];
            if (kg + 8 > len) {   // zero the values of keys past len (they may be stale)
                #pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int kk = kg + 2 * e;
                    if (kk >= len) w[e] = 0u;
                    else if (kk + 1 >= len) w[e] &= 0x0000ffffu;
                }
            }
            vf[db] = __builtin_bit_cast(bf16x8_v, w);
        }
        // S^T
        f32x4_v sacc[2][NB];
        #pragma unroll
        for (int blk = 0; blk < 2; ++blk)
            #pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                sacc[blk][rb] = f32x4_v{0.f, 0.f, 0.f, 0.f};
                #pragma unroll
                for (int ks = 0; ks < KST; ++ks)
                    sacc[blk][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[buf][blk][ks], qf[rb][ks], sacc[blk][rb], 0, 0, 0);
            }
        // online softmax and PV, per 16-row block
        // the running max is kept on unscaled scores (the scale is positive):
        // p = 2^(s c - m c) is one fma into the exponential.  A slab that is
        // visible to every row of the wave skips the masks, and a row block
        // whose max did not move in any lane skips the rescale of o.
        const float cs = a.scale_log2;
        const bool full = __all(kg + 8 <= k1 && kg + 7 <= lim_min);
        #pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            float sv[8];
            float mt = -INFINITY;
            if (full) {   // wave-uniform: no masks
                #pragma unroll
                for (int j = 0; j < 8; ++j) {
                    sv[j] = sacc[j >> 2][rb][j & 3];
                    mt = fmaxf(mt, sv[j]);
                }
            } else {
                #pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int key = kg + j;
                    const bool ok = (key < k1) & (key <= lim[rb]);   // no short circuit: straight-line selects
                    sv[j] = ok ? sacc[j >> 2][rb][j & 3] : -INFINITY;
                    mt = fmaxf(mt, sv[j]);
                }
            }
            mt = max_over_row_lanes(mt);
            const float mn = fmaxf(m_run[rb], mt);
            const bool same = mn == m_run[rb];
            const float ms = (mn == -INFINITY) ? 0.f : mn * cs;
            const float alpha = same ? 1.f : __builtin_amdgcn_exp2f(fmaf(m_run[rb], cs, -ms));
            m_run[rb] = mn;
            float ps = 0.f;
            uint32_t pk[4];
            #pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float p0 = __builtin_amdgcn_exp2f(fmaf(sv[2 * e], cs, -ms));
                const float p1 = __builtin_amdgcn_exp2f(fmaf(sv[2 * e + 1], cs, -ms));
                ps += p0 + p1;
                pk[e] = cvt_pk_bf16(p0, p1);
            }
            l_run[rb] = fmaf(l_run[rb], alpha, ps);
            const bf16x8_v pf = __builtin_bit_cast(bf16x8_v, u32x4_v{pk[0], pk[1], pk[2], pk[3]});
            if (!__all(same)) {
                #pragma unroll
                for (int db = 0; db < DB; ++db) o[db][rb] *= alpha;
            }
            #pragma unroll
            for (int db = 0; db < DB; ++db)
                o[db][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[db], pf, o[db][rb], 0, 0, 0);
        }
    };

    // software pipeline: slab i lives in buffer i % DEPTH
    #pragma unroll
    for (int d = 0; d < DEPTH - 1; ++d)
        if (d < nsl) load(d, d, d);
    for (int i0 = 0; i0 < nsl; i0 += DEPTH) {
        #pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int i = i0 + d;
            if (i + DEPTH - 1 < nsl) load(i + DEPTH - 1, (d + DEPTH - 1) % DEPTH, (d + DEPTH - 1) % DEPTH);
            if (i < nsl) compute(i, d);
        }
    }

    // ---- merge the four waves in LDS ----
    float *sML = reinterpret_cast<float *>(smem);          // [4 waves][RP][2]
    float *sO = sML + 4 * RP * 2;                          // [4 waves][RP][D]
    #pragma unroll
    for (int rb = 0; rb < NB; ++rb) {
        const float lt = sum_over_row_lanes(l_run[rb]);
        if (lg == 0) {
            sML[(wave * RP + rb * 16 + lr) * 2] = m_run[rb] == -INFINITY ? -INFINITY : m_run[rb] * a.scale_log2;
            sML[(wave * RP + rb * 16 + lr) * 2 + 1] = lt;
        }
        #pragma unroll
        for (int db = 0; db < DB; ++db)
            #pragma unroll
            for (int i = 0; i < 4; ++i) sO[((size_t)wave * RP + rb * 16 + lr) * D + db * 16 + 4 * lg + i] = o[db][rb][i];
    }
    __syncthreads();
    float *po = a.part + ((size_t)u * a.n_splits + s) * a.part_rows * D;
    float *pml = a.part_ml + ((size_t)u * a.n_splits + s) * a.part_rows * 2;
    for (int idx = tid; idx < R * D; idx += 256) {
        const int r = idx / D, col = idx - r * D;
        float M = -INFINITY;
        #pragma unroll
        for (int w = 0; w < 4; ++w) M = fmaxf(M, sML[(w * RP + r) * 2]);
        const float Ms = (M == -INFINITY) ? 0.f : M;
        float acc = 0.f, L = 0.f;
        #pragma unroll
        for (int w = 0; w < 4; ++w) {
            const float wt = __builtin_amdgcn_exp2f(sML[(w * RP + r) * 2] - Ms);
            acc = fmaf(wt, sO[((size_t)w * RP + r) * D + col], acc);
            L = fmaf(wt, sML[(w * RP + r) * 2 + 1], L);
        }
        po[idx] = acc;
        if (col == 0) {
            pml[2 * r] = M;
            pml[2 * r + 1] = L;
        }
    }
}

// ---------------------------------------------------------------------------
// LDS-staged split kernel.  The register-resident kernel above keeps a full
// copy of the output accumulators in every wave (the waves split keys), which
// leaves room for one or two 32-key slabs in flight per wave: with HBM latency
// under load of several microseconds that caps the stream.  Here the waves
// split the query rows and the keys of every slab -- wave w < 2 NB owns 16-row
// block w % NB and the 32-key half w / NB of each 64-key slab; with two waves
// per SIMD one wave's exponentials and matrix products overlap another's -- and share
// every K/V slab through a deep LDS ring filled by direct loads
// (global_load_lds_dwordx4, issued by all eight waves), so about
// (NST - 1) x 32 KB are in flight per workgroup:
//   * K rows land with their 16-byte chunks XOR-swizzled by row, so the
//     permuted-row A operand reads of S^T = K Q^T are conflict-free;
//   * V^T rows (one feature, the slab's 64 keys) land with their 16-byte
//     key chunks swizzled by feature for the A operand of O^T = V^T P^T;
//   * one barrier per slab; at the end the two key halves of each row block
//     are merged in LDS and the rows' partial (max, sum, o) is written.
template <int D>
struct VerifyLdsCfg {
    static constexpr int SLAB = 64;                        // keys per slab (128 contiguous bytes of each V^T row)
    static constexpr int RB = D * 2;                       // bytes per K row
    static constexpr int KBYTES = SLAB * RB;               // K bytes per slab (= V^T bytes)
    static constexpr int VROW = SLAB * 2;                  // bytes per V^T row in a stage
    static constexpr int STAGE = 2 * KBYTES;
    static constexpr int NST = D == 128 ? 4 : 8;           // ring stages (128 KB)
    static constexpr int NWV = 8;                          // waves: 4 row blocks x 2 key halves
    static constexpr int IPW = STAGE / 1024 / NWV;         // direct loads per wave per slab
    static constexpr int SMEM = NST * STAGE;
    static_assert(IPW % 2 == 0, "K and V loads per wave");
};

__device__ __forceinline__ int vk_swz(int k) { return (k & 3) | (((k >> 3) & 1) << 2); }
// natural V rows: 16-byte chunk c of key row k sits at chunk c ^ vn_swz(k); a
// transposing read of 16 lanes covers rows k0 .. k0+3 (k0 a multiple of 4) x
// two adjacent chunks, and XOR with 2 (k mod 4) puts the eight (row, chunk)
// pairs on distinct banks
__device__ __forceinline__ int vn_swz(int k) { return (k & 3) << 1; }
typedef short v4s_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ v4s_t lds_read_tr16(const unsigned char *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s_t *)(p));
}

template <int D, int NB, bool VNAT>
__global__ __launch_bounds__(512, 1) void verify_lds_kernel(const VerifyArgs a) {
    using C = VerifyLdsCfg<D>;
    constexpr int KST = D / 32, DB = D / 16, CPR = D / 8;
    extern __shared__ __align__(16) unsigned char smem[];
    MAD_TRACE_T0();

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u = blockIdx.x % a.units, s = blockIdx.x / a.units;
    const int b = u / a.Hkv, c = u - b * a.Hkv;
    const int len = a.len[b], T = a.T, G = a.G, R = T * G;
    const int k0 = s * a.chunk;
    const int k1 = min(len, k0 + a.chunk);
    const int cap = a.cap;
    const bf16_t *K = reinterpret_cast<const bf16_t *>(a.k) + b * a.seq + c * a.head;
    // V: natural rows [cap][D] (VNAT) or one run of cap keys per feature [D][cap]
    const bf16_t *VT = reinterpret_cast<const bf16_t *>(a.vt) + b * a.seq + c * a.head;
    const int lr = lane & 15, lg = lane >> 4;
    // waves 0 .. 2 NB - 1 compute (row block wave % NB, key half wave / NB), so
    // consecutive waves -- on different SIMDs -- take different row blocks
    const int rbw = wave % NB, kh = wave / NB;
    const bool active = wave < 2 * NB;

    // ---- this wave's query fragments and causal limit (row block rbw) ----
    bf16x8_v qf[KST];
    const int row = rbw * 16 + lr;
    int lim = 0x7fffffff;
    if (active && row < R) {
        const int t = row / G, g = row - t * G;
        const bf16_t *qrow = reinterpret_cast<const bf16_t *>(a.q) + (((size_t)b * T + t) * a.Hq + c * G + g) * D;
        #pragma unroll
        for (int ks = 0; ks < KST; ++ks) qf[ks] = *reinterpret_cast<const bf16x8_v *>(qrow + ks * 32 + 8 * lg);
        lim = len - T + t;
    } else {
        #pragma unroll
        for (int ks = 0; ks < KST; ++ks) qf[ks] = bf16x8_v{0, 0, 0, 0, 0, 0, 0, 0};
    }
    // the query loads complete here, before any direct load is in flight, so
    // no wait the compiler places for them can drain the ring later
    #pragma unroll
    for (int ks = 0; ks < KST; ++ks) asm volatile("" : : "v"(qf[ks]));

    const int nsl = k1 > k0 ? (k1 - k0 + C::SLAB - 1) / C::SLAB : 0;
    auto issue = [&](int i) {
        unsigned char *st = smem + (i % C::NST) * C::STAGE;
        const int kb = k0 + i * C::SLAB;
        #pragma unroll
        for (int j = 0; j < C::IPW / 2; ++j) {
            const int inst = wave * (C::IPW / 2) + j;
            const int cidx = inst * 64 + lane;
            // K: row cidx / CPR, LDS slot cidx % CPR holds global chunk slot ^ swz(row)
            const int kr = cidx / CPR, slot = cidx % CPR;
            const int key = min(kb + kr, len - 1);   // rows past len: a valid row, masked
            lds_stream16_nt(K + (size_t)key * D + (slot ^ vk_swz(kr)) * 8, st + inst * 1024);
            if constexpr (VNAT) {
                // V rows like K rows (the same clamp), chunk slot holds global chunk slot ^ vn_swz(row)
                lds_stream16_nt(VT + (size_t)key * D + (slot ^ vn_swz(kr)) * 8, st + C::KBYTES + inst * 1024);
            } else {
                // V^T: feature cidx / 8, LDS slot cidx % 8 holds key chunk slot ^ (f & 7)
                const int f = cidx >> 3, vs = cidx & 7;
                int kc = kb + ((vs ^ (f & 7)) << 3);
                if (kc + 8 > cap) kc = cap - 8;          // chunks past the cache: any valid chunk (zeroed when used)
                lds_stream16_nt(VT + (size_t)f * cap + kc, st + C::KBYTES + inst * 1024);
            }
        }
    };

    f32x4_v o[DB];
    #pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x4_v{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;
    const float cs = a.scale_log2;

    auto compute = [&](int i) {
        const unsigned char *st = smem + (i % C::NST) * C::STAGE;
        const int kb = k0 + i * C::SLAB;
        // S^T for this wave's 32-key half: A row m of block blk is key
        // 32 kh + 8(m/4) + 4 blk + m%4 of the slab, so accumulator element e&3 of
        // block e>>2 is key 32 kh + 8 lg + e
        f32x4_v sacc[2];
        #pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
            const int kr = 32 * kh + 8 * (lr >> 2) + 4 * blk + (lr & 3);
            sacc[blk] = f32x4_v{0.f, 0.f, 0.f, 0.f};
            #pragma unroll
            for (int ks = 0; ks < KST; ++ks) {
                const bf16x8_v kf =
                    *reinterpret_cast<const bf16x8_v *>(st + kr * C::RB + (((4 * ks + lg) ^ vk_swz(kr)) << 4));
                sacc[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks], sacc[blk], 0, 0, 0);
            }
        }
        float sv[8];
        float mt = -INFINITY;
        const int kg = kb + 32 * kh + 8 * lg;
        if (__all(kb + C::SLAB <= k1 && kb + C::SLAB - 1 <= lim)) {
            #pragma unroll
            for (int j = 0; j < 8; ++j) {
                sv[j] = sacc[j >> 2][j & 3];
                mt = fmaxf(mt, sv[j]);
            }
        } else {
            #pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int key = kg + j;
                const bool ok = (key < k1) & (key <= lim);
                sv[j] = ok ? sacc[j >> 2][j & 3] : -INFINITY;
                mt = fmaxf(mt, sv[j]);
            }
        }
        mt = max_over_row_lanes(mt);
        const float mn = fmaxf(m_run, mt);
        const bool same = mn == m_run;
        const float ms = (mn == -INFINITY) ? 0.f : mn * cs;
        const float alpha = same ? 1.f : __builtin_amdgcn_exp2f(fmaf(m_run, cs, -ms));
        m_run = mn;
        float ps = 0.f;
        uint32_t pk[4];
        #pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float p0 = __builtin_amdgcn_exp2f(fmaf(sv[2 * e], cs, -ms));
            const float p1 = __builtin_amdgcn_exp2f(fmaf(sv[2 * e + 1], cs, -ms));
            ps += p0 + p1;
            pk[e] = cvt_pk_bf16(p0, p1);
        }
        const bf16x8_v pf = __builtin_bit_cast(bf16x8_v, u32x4_v{pk[0], pk[1], pk[2], pk[3]});
        l_run = fmaf(l_run, alpha, ps);
        if (!__all(same)) {
            #pragma unroll
            for (int db = 0; db < DB; ++db) o[db] *= alpha;
        }
        if constexpr (VNAT) {
            // A = V^T rows (features db*16 + lr), keys 32 kh + 8 lg .. +7, from
            // the transposing reads of key rows 32 kh + 8 lg + {0..3} and {4..7}
            // (rows past len hold the clamped row len - 1, weighted 0)
            const unsigned char *sv = st + C::KBYTES;
            const int tr_row = 32 * kh + 8 * lg + (lr >> 2), tr_byte = 8 * (lr & 3);
            #pragma unroll
            for (int db = 0; db < DB; ++db) {
                const int byte = db * 32 + tr_byte, chunk = byte >> 4, half = byte & 8;
                const int r0 = tr_row, r1 = tr_row + 4;
                const v4s_t lo = lds_read_tr16(sv + r0 * C::RB + ((chunk ^ vn_swz(r0)) << 4) + half);
                const v4s_t hi = lds_read_tr16(sv + r1 * C::RB + ((chunk ^ vn_swz(r1)) << 4) + half);
                const bf16x8_v vf = __builtin_bit_cast(bf16x8_v, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[db], 0, 0, 0);
            }
        } else {
            #pragma unroll
            for (int db = 0; db < DB; ++db) {
                const int f = db * 16 + lr;
                u32x4_v w = *reinterpret_cast<const u32x4_v *>(st + C::KBYTES + f * C::VROW + (((4 * kh + lg) ^ (f & 7)) << 4));
                if (kg + 8 > len) {   // values of keys past len may be anything: zero them
                    #pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int kk = kg + 2 * e;
                        if (kk >= len) w[e] = 0u;
                        else if (kk + 1 >= len) w[e] &= 0x0000ffffu;
                    }
                }
                o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_v, w), pf, o[db], 0, 0, 0);
            }
        }
    };

    int issued = 0;
    for (; issued < nsl && issued < C::NST - 1; ++issued) issue(issued);
    for (int i = 0; i < nsl; ++i) {
        wait_vm(C::IPW * (issued - 1 - i));   // slab i has landed (this wave's part)
        __syncthreads();                      // ... every wave's part; stage (i-1) % NST is free
        if (issued < nsl) {
            issue(issued);
            ++issued;
        }
        if (active) compute(i);
    }

    // ---- merge the two key halves of each row block, then the rows' partial
    // (max in log2 units, sum, unnormalised o) ----
    const float lt = sum_over_row_lanes(l_run);
    const float msc = m_run == -INFINITY ? -INFINITY : m_run * cs;
    __syncthreads();   // every wave is done with the ring
    float *xo = reinterpret_cast<float *>(smem);   // [4][16][D]: the second halves' o
    float *xml = xo + 4 * 16 * D;                  // [4][16][2]: their (max, sum)
    if (active && kh == 1) {
        #pragma unroll
        for (int db = 0; db < DB; ++db)
            *reinterpret_cast<float4 *>(xo + (size_t)row * D + db * 16 + 4 * lg) = make_float4(o[db][0], o[db][1], o[db][2], o[db][3]);
        if (lg == 0) {
            xml[2 * row] = msc;
            xml[2 * row + 1] = lt;
        }
    }
    __syncthreads();
    MAD_TRACE_SAVE_T0(mad_trace_verify);   // the workgroup's partial is written below; thread 0 marks it
    if (!active || kh == 1 || row >= R) return;
    const float m1 = xml[2 * row], l1 = xml[2 * row + 1];
    const float M = fmaxf(msc, m1);
    const float w0 = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(msc - M);
    const float w1 = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - M);
    float *po = a.part + (((size_t)u * a.n_splits + s) * a.part_rows + row) * D;
    float *pml = a.part_ml + (((size_t)u * a.n_splits + s) * a.part_rows + row) * 2;
    // the partial leaves with non-temporal stores: the merge kernel reads it
    // once, and no dirty L2 lines are left for the end of the launch (0.7 us
    // less at the 70B shape)
    typedef float f4v __attribute__((ext_vector_type(4)));
    #pragma unroll
    for (int db = 0; db < DB; ++db) {
        const float4 x = *reinterpret_cast<const float4 *>(xo + (size_t)row * D + db * 16 + 4 * lg);
        __builtin_nontemporal_store(f4v{fmaf(w0, o[db][0], w1 * x.x), fmaf(w0, o[db][1], w1 * x.y),
                                        fmaf(w0, o[db][2], w1 * x.z), fmaf(w0, o[db][3], w1 * x.w)},
                                    reinterpret_cast<f4v *>(po + db * 16 + 4 * lg));
    }
    if (lg == 0) {
        __builtin_nontemporal_store(M, pml);
        __builtin_nontemporal_store(fmaf(w0, lt, w1 * l1), pml + 1);
    }
    MAD_TRACE(mad_trace_verify, 1);
}

// One workgroup (D threads) per (unit, query row): log-sum-exp merge of the
// splits.  Every thread first issues the reads of its feature in the first MB
// splits (they do not depend on the weights, so their round trip overlaps the
// one of the (max, sum) pairs), the threads turn the splits' (max, sum) into
// weights in parallel, then every thread sums its feature over the splits.
template <int D>
__global__ __launch_bounds__(D) void verify_merge_kernel(const VerifyArgs a) {
    const int R = a.T * a.G;
    const int u = blockIdx.x / R, r = blockIdx.x - u * R;
    const int b = u / a.Hkv, c = u - b * a.Hkv;
    const int t = r / a.G, g = r - t * a.G;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int NW = D / 64;
    const int ns = a.n_splits;
    const float *po = a.part + (size_t)u * ns * a.part_rows * D + (size_t)r * D + tid;
    const float *pml = a.part_ml + (size_t)u * ns * a.part_rows * 2 + 2 * r;
    const size_t so = (size_t)a.part_rows * D, sml = (size_t)a.part_rows * 2;
    __shared__ float s_w[kVerifyMaxSplits];
    __shared__ float s_red[2][NW];

    constexpr int MB = 32;   // splits whose feature values are read ahead
    float v[MB];
    #pragma unroll
    for (int e = 0; e < MB; ++e) v[e] = e < ns ? po[e * so] : 0.f;

    // split weights: thread i handles splits i and i + D (ns <= kVerifyMaxSplits <= 2 D)
    float m0 = -INFINITY, m1 = -INFINITY, l0 = 0.f, l1 = 0.f;
    if (tid < ns) { m0 = pml[tid * sml]; l0 = pml[tid * sml + 1]; }
    if (tid + D < ns) { m1 = pml[(tid + D) * sml]; l1 = pml[(tid + D) * sml + 1]; }
    const float m = group_max<64>(fmaxf(m0, m1));
    if (lane == 0) s_red[0][wave] = m;
    __syncthreads();
    float M = s_red[0][0];
    #pragma unroll
    for (int w = 1; w < NW; ++w) M = fmaxf(M, s_red[0][w]);
    const float w0 = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m0 - M);
    const float w1 = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m1 - M);
    const float lsum = group_sum<64>(w0 * l0 + w1 * l1);
    if (lane == 0) s_red[1][wave] = lsum;
    __syncthreads();
    float L = 0.f;
    #pragma unroll
    for (int w = 0; w < NW; ++w) L += s_red[1][w];
    const float inv = L > 0.f ? 1.f / L : 0.f;
    if (tid < ns) s_w[tid] = w0 * inv;
    if (tid + D < ns) s_w[tid + D] = w1 * inv;
    __syncthreads();

    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    #pragma unroll
    for (int e = 0; e < MB; ++e)
        if (e < ns) acc[e & 3] = fmaf(s_w[e], v[e], acc[e & 3]);
    for (int s0 = MB; s0 < ns; s0 += 8) {
        float x[8];
        #pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = s0 + e < ns ? po[(s0 + e) * so] : 0.f;
        #pragma unroll
        for (int e = 0; e < 8; ++e) if (s0 + e < ns) acc[e & 3] = fmaf(s_w[s0 + e], x[e], acc[e & 3]);
    }
    const float accs = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    const size_t head = ((size_t)b * a.T + t) * a.Hq + (size_t)c * a.G + g;
    reinterpret_cast<bf16_t *>(a.out)[head * D + tid].bits = f32_to_bf16(accs);
    if (a.lse && tid == 0) a.lse[head] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
}

// ------------------------------------------------------------------ host ----

VerifyPlan plan_verify(int B, int Hkv, int G, int T, const int *len, bool vnat) {
    VerifyPlan p;
    p.units = B * Hkv;
    int n_max = 0;
    for (int b = 0; b < B; ++b) n_max = len[b] > n_max ? len[b] : n_max;
    int ns = (kVerifyTargetWGs + p.units - 1) / p.units;
    if (ns > kVerifyMaxSplits) ns = kVerifyMaxSplits;
    if (ns < 1) ns = 1;
    int chunk = (n_max + ns - 1) / ns;
    // whole slabs: 4 x 32 keys for the register-resident kernel, 64 for the LDS-staged one
    const int gran = (vnat || (T * G + 15) / 16 >= kVerifyLdsMinNb) ? 64 : 128;
    chunk = (chunk + gran - 1) / gran * gran;
    if (chunk < gran) chunk = gran;
    p.chunk = chunk;
    p.n_splits = (n_max + chunk - 1) / chunk;
    if (p.n_splits < 1) p.n_splits = 1;
    return p;
}

static int verify_max_splits(int units) {
    int ns = (kVerifyTargetWGs + units - 1) / units;
    return ns > kVerifyMaxSplits ? kVerifyMaxSplits : (ns < 1 ? 1 : ns);
}

size_t verify_ws_bytes(int B, int Hq, int Hkv, int d, int T) {
    const size_t units = (size_t)B * Hkv;
    const size_t rows = (size_t)T * (Hq / Hkv);
    const size_t ns = (size_t)verify_max_splits((int)units);
    const size_t bf = kCounterRegionBytes + align256(units * ns * rows * d * 4) + align256(units * ns * rows * 2 * 4);
    // fp32 verify runs the decode kernel once per sequence, its T query rows as the rows
    const size_t f32 = decode_ws_bytes(T, Hq, Hkv, d);
    return bf > f32 ? bf : f32;
}

void verify_ws_layout(int B, int Hq, int Hkv, int d, int T, size_t *off_o, size_t *off_ml) {
    const size_t units = (size_t)B * Hkv;
    const size_t rows = (size_t)T * (Hq / Hkv);
    const size_t ns = (size_t)verify_max_splits((int)units);
    *off_o = kCounterRegionBytes;
    *off_ml = kCounterRegionBytes + align256(units * ns * rows * d * 4);
}

template <int D, int NB>
static hipError_t launch_split(const VerifyArgs &a, hipStream_t st) {
    if (a.vnat) {
        hipLaunchKernelGGL((verify_lds_kernel<D, NB, true>), dim3((unsigned)(a.units * a.n_splits)),
                           dim3(64 * VerifyLdsCfg<D>::NWV), VerifyLdsCfg<D>::SMEM, st, a);
        return hipGetLastError();
    }
    if (NB >= kVerifyLdsMinNb) {
        hipLaunchKernelGGL((verify_lds_kernel<D, NB, false>), dim3((unsigned)(a.units * a.n_splits)),
                           dim3(64 * VerifyLdsCfg<D>::NWV), VerifyLdsCfg<D>::SMEM, st, a);
        return hipGetLastError();
    }
    constexpr int RP = NB * 16;
    const size_t lds = (size_t)4 * RP * 2 * 4 + (size_t)4 * RP * D * 4;
    hipLaunchKernelGGL((verify_split_kernel<D, NB>), dim3((unsigned)(a.units * a.n_splits)), dim3(256), lds, st, a);
    return hipGetLastError();
}

template <int D>
static hipError_t launch_d(const VerifyArgs &a, hipStream_t st) {
    const int NB = (a.T * a.G + 15) / 16;
    hipError_t e;
    switch (NB) {
        case 1: e = launch_split<D, 1>(a, st); break;
        case 2: e = launch_split<D, 2>(a, st); break;
        case 3: e = launch_split<D, 3>(a, st); break;
        case 4: e = launch_split<D, 4>(a, st); break;
        default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((verify_merge_kernel<D>), dim3((unsigned)(a.units * a.T * a.G)), dim3(D), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_verify(const VerifyArgs &a, hipStream_t st) {
    if (a.d == 64) return launch_d<64>(a, st);
    if (a.d == 128) return launch_d<128>(a, st);
    return hipErrorInvalidValue;
}

}  // namespace mad
