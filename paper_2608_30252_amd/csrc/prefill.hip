// prefill.hip -- memory-prefill attention: the draft's one masked pass over a
// prefix that builds its initial compact memory (Sec. 3.3 prefill; the
// appendix on memory prefill).
//
// The prefill mask applies the same write policy as decoding, so every query
// of the pass attends exactly the set it would attend during decoding:
//   raw token at position p : sinks [0, min(S, p+1)), the slots materialised
//                             in passes of earlier tokens (1 .. slots_after(p)),
//                             and the window [max(S, p-W+1), p];
//   memory slot g_m         : the sinks, slots 1..m (itself included) and the
//                             W raw tokens before its position id b_m = S + m r:
//                             [max(S, b_m - W), b_m - 1].
// Keys come from two places: the memory segment (sinks in rows 0..S-1, slot m
// in row S + m - 1) and the prefix's raw K/V (position x in row x).  For every
// query the visible keys are one prefix of the memory segment, [0, mem_hi),
// and one interval of raw rows, [raw_lo, raw_hi).
//
// Both products run on the matrix cores (v_mfma_f32_16x16x32_bf16, fp32
// accumulation).  A workgroup of four waves owns one (sequence, KV head) unit
// and a block of query tokens; its rows are (token, query head of the GQA
// group) pairs in 16-token blocks, each wave holding NB of them with their
// query fragments in registers for the whole pass.  Keys stream in 64-key
// tiles through two LDS stages, loaded into registers one tile ahead:
//   * K rows are stored with their 16-byte chunks XOR-swizzled so the A
//     operand reads of S^T = K Q^T are conflict-free; the A rows are permuted
//     so that each lane's S^T accumulators hold the 8 consecutive keys that
//     the PV product's B operand needs (no shuffle of probabilities);
//   * V rows are stored as they are (16-byte chunks XOR-swizzled by row), and
//     the A operand of O^T = V^T P^T -- 8 consecutive keys of one feature --
//     comes from two transposing LDS reads (ds_read_b64_tr_b16: lane 4e + a of
//     a 16-lane group names features 4a .. 4a+3 of key row e, and lane 4a + b
//     receives feature 4a + b of the four rows);
//   * online softmax per query row (16 scores per lane per tile, two
//     cross-lane lane swaps), masks applied in place on edge tiles only, and
//     a lazy rescale: the reference maximum of a row block moves only when a
//     row gains more than 2^8, so most tiles skip the exponential of the
//     correction and the rescale of o; one barrier per tile.
// Query blocks of every unit are dealt round-robin over the units (with a
// multiple of 8 units all blocks of one KV head share an XCD and its L2), the
// heaviest blocks first.
#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_v;
typedef __attribute__((ext_vector_type(4))) float f32x4_v;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_v;

template <int D>
struct PrefillCfg {
    static constexpr int KT = 64;                     // keys per tile (128 spills registers at d 64)
    static constexpr int KH = KT / 32;                 // 32-key halves of a tile
    static constexpr int RB = D * 2;                   // bytes per K row
    static constexpr int CPR = RB / 16;                // 16-byte chunks per K row
    static constexpr int KTILE = KT * RB;              // K tile bytes
    static constexpr int STAGE = 2 * KTILE;            // K tile + V tile (same size)
    static constexpr int SMEM = 2 * STAGE;
    static constexpr int KCH = KT * CPR / 256;         // K chunks per thread per tile
    static constexpr int VCH = KCH;                    // V chunks per thread per tile
};

// swizzle of K row k's 16-byte chunks: distinct for the 8 rows one group of
// eight lanes reads (k mod 4 and bit 3 of k vary across them)
__device__ __forceinline__ int k_swz(int k) { return (k & 3) | (((k >> 3) & 1) << 2); }
// swizzle of V row k's 16-byte chunks: a transposing read of 16 lanes covers
// rows k0 .. k0+3 (k0 a multiple of 4) x two adjacent chunks; XOR with
// 2 (k mod 4) spreads the eight (row, chunk) pairs over distinct banks
__device__ __forceinline__ int v_swz(int k) { return (k & 3) << 1; }
typedef short v4s_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ v4s_t lds_read_tr16(const unsigned char *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s_t *)(p));
}

// Lanes l, l^16, l^32, l^48 hold the same query row.  v_permlane16_swap and
// v_permlane32_swap (VALU lane swaps, no LDS round trip) give every lane the
// values of lanes l & ~16 and l | 16 (resp. 32), so two swaps reduce over the four.
__device__ __forceinline__ float prefill_row_max(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float prefill_row_sum(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

constexpr float kLazyLog2 = 8.f;   // rescale threshold of the online softmax, log2 units

__device__ __forceinline__ int prefill_slots_after(int t, int S, int ru, int u) {
    return t <= S ? 0 : (t - S) / ru * u;
}

// Occupancy: three waves per SIMD at head_dim 64 (the compiler then keeps the
// kernel within 168 registers; measured 8% faster than two), two at 128.
template <int D, int G, int NB>
__global__ __launch_bounds__(256, NB == 2 ? (D == 64 ? 3 : 2) : 1) void prefill_kernel(const PrefillArgs a) {
    using C = PrefillCfg<D>;
    constexpr int KST = D / 32, DB = D / 16;
    constexpr int TBW = 4 * NB / G;   // 16-token blocks per workgroup
    constexpr int QT = 16 * TBW;      // query tokens per workgroup
    static_assert(4 * NB % G == 0, "row blocks cover whole token blocks");
    extern __shared__ __align__(16) unsigned char smem[];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lr = lane & 15, lg = lane >> 4;
    const int unit = blockIdx.x % a.units;
    const int qb = a.nrb + a.nsb - 1 - (int)(blockIdx.x / a.units);   // slot blocks, then raw blocks, late first
    const int b = unit / a.Hkv, c = unit - b * a.Hkv;
    const bool slot_kind = qb >= a.nrb;
    const int S = a.S, W = a.W, r = a.r, u = a.u, ru = a.r * a.u;
    const int nq = slot_kind ? a.Mtot[b] : a.P[b];
    const int q0 = (slot_kind ? qb - a.nrb : qb) * QT;   // first token: raw position, or slot index - 1
    if (q0 >= nq) return;                                 // the whole workgroup: no barrier crossed
    const int qlast = min(nq, q0 + QT) - 1;

    // ---- the workgroup's key ranges: the union of its rows' ranges ----
    int mem_hi, raw_lo, raw_hi;
    if (!slot_kind) {
        mem_hi = qlast < S ? qlast + 1 : S + prefill_slots_after(qlast, S, ru, u);
        raw_lo = max(S, q0 - W + 1);
        raw_hi = qlast + 1;
    } else {
        mem_hi = S + qlast + 1;
        raw_lo = max(S, S + (q0 + 1) * r - W);
        raw_hi = S + (qlast + 1) * r;
    }
    if (raw_hi < raw_lo) raw_hi = raw_lo;
    const int n_mem_t = (mem_hi + C::KT - 1) / C::KT;
    const int nt = n_mem_t + (raw_hi - raw_lo + C::KT - 1) / C::KT;

    const bf16_t *mk = reinterpret_cast<const bf16_t *>(a.mk) + b * a.m_seq + c * a.m_head;
    const bf16_t *mv = reinterpret_cast<const bf16_t *>(a.mv) + b * a.m_seq + c * a.m_head;
    const bf16_t *rk = reinterpret_cast<const bf16_t *>(a.rk) + b * a.r_seq + c * a.r_head;
    const bf16_t *rv = reinterpret_cast<const bf16_t *>(a.rv) + b * a.r_seq + c * a.r_head;
    const bf16_t *qbase = reinterpret_cast<const bf16_t *>(slot_kind ? a.q_slot : a.q_raw) +
                          (size_t)b * (slot_kind ? a.slot_cap : a.q_cap) * a.Hq * D;

    // ---- this lane's rows: query fragments and visible ranges ----
    bf16x8_v qf[NB][KST];
    int m_lim[NB], r_lo[NB], r_hi[NB];
    #pragma unroll
    for (int i = 0; i < NB; ++i) {
        const int j = wave + 4 * i, g = j % G, tb = j / G;
        const int tok = q0 + tb * 16 + lr;
        if (tok <= qlast) {
            const bf16_t *qrow = qbase + ((size_t)tok * a.Hq + c * G + g) * D;
            #pragma unroll
            for (int ks = 0; ks < KST; ++ks) qf[i][ks] = *reinterpret_cast<const bf16x8_v *>(qrow + ks * 32 + 8 * lg);
            if (!slot_kind) {
                m_lim[i] = tok < S ? tok + 1 : S + prefill_slots_after(tok, S, ru, u);
                r_lo[i] = max(S, tok - W + 1);
                r_hi[i] = tok < S ? r_lo[i] : tok + 1;
            } else {
                const int bm = S + (tok + 1) * r;
                m_lim[i] = S + tok + 1;
                r_lo[i] = max(S, bm - W);
                r_hi[i] = bm;
            }
        } else {
            #pragma unroll
            for (int ks = 0; ks < KST; ++ks) qf[i][ks] = bf16x8_v{0, 0, 0, 0, 0, 0, 0, 0};
            m_lim[i] = 0;
            r_lo[i] = r_hi[i] = 0;
        }
    }

    // ---- tile loader: registers one tile ahead, then LDS ----
    // one tile's K and V chunks of this thread, staged in registers
    struct StageRegs {
        uint4 k[C::KCH], v[C::VCH];
    };
    auto tile_base = [&](int t, bool &is_mem, int &end) -> int {
        is_mem = t < n_mem_t;
        if (is_mem) {
            end = mem_hi;
            return t * C::KT;
        }
        end = raw_hi;
        return raw_lo + (t - n_mem_t) * C::KT;
    };
    auto load_regs = [&](int t) -> StageRegs {
        StageRegs r;
        bool is_mem;
        int end;
        const int base = tile_base(t, is_mem, end);
        const bf16_t *ks = is_mem ? mk : rk, *vs = is_mem ? mv : rv;
        #pragma unroll
        for (int i = 0; i < C::KCH; ++i) {
            const int idx = tid + 256 * i, row = idx / C::CPR, ch = idx % C::CPR;
            const int key = min(base + row, end - 1);   // rows past the range load a valid row (masked)
            r.k[i] = *reinterpret_cast<const uint4 *>(ks + (size_t)key * D + ch * 8);
        }
        #pragma unroll
        for (int i = 0; i < C::VCH; ++i) {
            const int idx = tid + 256 * i, row = idx / C::CPR, ch = idx % C::CPR;
            const int key = min(base + row, end - 1);
            r.v[i] = *reinterpret_cast<const uint4 *>(vs + (size_t)key * D + ch * 8);
        }
        return r;
    };
    auto store_lds = [&](int stage, const StageRegs &r) {
        unsigned char *sk = smem + stage * C::STAGE, *sv = sk + C::KTILE;
        #pragma unroll
        for (int i = 0; i < C::KCH; ++i) {
            const int idx = tid + 256 * i, row = idx / C::CPR, ch = idx % C::CPR;
            *reinterpret_cast<uint4 *>(sk + row * C::RB + ((ch ^ k_swz(row)) << 4)) = r.k[i];
        }
        #pragma unroll
        for (int i = 0; i < C::VCH; ++i) {
            const int idx = tid + 256 * i, row = idx / C::CPR, ch = idx % C::CPR;
            *reinterpret_cast<uint4 *>(sv + row * C::RB + ((ch ^ v_swz(row)) << 4)) = r.v[i];
        }
    };

    f32x4_v o[DB][NB];
    float m_run[NB], l_run[NB];
    #pragma unroll
    for (int i = 0; i < NB; ++i) {
        m_run[i] = -INFINITY;
        l_run[i] = 0.f;
        #pragma unroll
        for (int db = 0; db < DB; ++db) o[db][i] = f32x4_v{0.f, 0.f, 0.f, 0.f};
    }

    auto compute = [&](int t, int stage) {
        const unsigned char *sk = smem + stage * C::STAGE, *sv = sk + C::KTILE;
        bool is_mem;
        int end;
        const int base = tile_base(t, is_mem, end);
        // S^T = K Q^T for the tile's keys: half h holds keys 32h .. 32h+31;
        // A row m of block blk of pair h is key 32h + 8(m/4) + 4 blk + m%4, so
        // accumulator element e&3 of block e>>2 in lane group lg is key 32h + 8 lg + e
        f32x4_v sacc[C::KH][2][NB];
        #pragma unroll
        for (int h = 0; h < C::KH; ++h)
            #pragma unroll
            for (int blk = 0; blk < 2; ++blk) {
                const int kr = 32 * h + 8 * (lr >> 2) + 4 * blk + (lr & 3);
                bf16x8_v kf[KST];
                #pragma unroll
                for (int ks = 0; ks < KST; ++ks)
                    kf[ks] = *reinterpret_cast<const bf16x8_v *>(sk + kr * C::RB + (((4 * ks + lg) ^ k_swz(kr)) << 4));
                #pragma unroll
                for (int i = 0; i < NB; ++i) {
                    sacc[h][blk][i] = f32x4_v{0.f, 0.f, 0.f, 0.f};
                    #pragma unroll
                    for (int ks = 0; ks < KST; ++ks)
                        sacc[h][blk][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ks], qf[i][ks], sacc[h][blk][i], 0, 0, 0);
                }
            }
        // online softmax per row block; probabilities become the B operand of PV.
        // The running max is kept on unscaled scores (the scale is positive);
        // p = 2^(s c - m c) is one fma into the exponential.  A tile inside
        // every row's visible range of this wave skips the masks.
        bf16x8_v pf[NB][C::KH];
        const float cs = a.scale_log2;
        #pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int lo = is_mem ? 0 : r_lo[i];
            const int hi = min(end, is_mem ? m_lim[i] : r_hi[i]);
            if (!__all(base >= lo && base + C::KT <= hi)) {
                // edge tile: element e of half h is key base + 32h + 8lg + e; mask in place
                const int k0 = base + 8 * lg, a0 = lo - k0, b0 = hi - k0;
                #pragma unroll
                for (int h = 0; h < C::KH; ++h)
                    #pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int kk = 32 * h + e;
                        const bool ok = (kk >= a0) & (kk < b0);   // no short circuit: straight-line selects
                        sacc[h][e >> 2][i][e & 3] = ok ? sacc[h][e >> 2][i][e & 3] : -INFINITY;
                    }
            }
            float mt = -INFINITY;
            #pragma unroll
            for (int h = 0; h < C::KH; ++h)
                #pragma unroll
                for (int e = 0; e < 8; ++e) mt = fmaxf(mt, sacc[h][e >> 2][i][e & 3]);
            mt = prefill_row_max(mt);
            // lazy rescale: the reference maximum moves only when some row of the
            // block gains more than kLazyLog2 (in log2 units); until then the
            // probabilities stay below 2^kLazyLog2, and o and l share one reference
            const bool grow = mt > m_run[i] && (m_run[i] == -INFINITY || (mt - m_run[i]) * cs > kLazyLog2);
            if (__any(grow)) {
                const float mn = fmaxf(m_run[i], mt);
                const float alpha = __builtin_amdgcn_exp2f(fmaf(m_run[i], cs, mn == -INFINITY ? 0.f : -mn * cs));
                m_run[i] = mn;
                l_run[i] *= alpha;
                #pragma unroll
                for (int db = 0; db < DB; ++db) o[db][i] *= alpha;
            }
            const float ms = m_run[i] == -INFINITY ? 0.f : m_run[i] * cs;
            float ps = 0.f;
            #pragma unroll
            for (int h = 0; h < C::KH; ++h) {
                uint32_t pk[4];
                #pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[h][(2 * e) >> 2][i][(2 * e) & 3], cs, -ms));
                    const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[h][(2 * e + 1) >> 2][i][(2 * e + 1) & 3], cs, -ms));
                    ps += p0 + p1;
                    pk[e] = cvt_pk_bf16(p0, p1);
                }
                pf[i][h] = __builtin_bit_cast(bf16x8_v, u32x4_v{pk[0], pk[1], pk[2], pk[3]});
            }
            l_run[i] += ps;
        }
        // O^T += V^T P^T: A = V^T rows (features db*16 + lr), keys 32h + 8 lg .. +7,
        // from the transposing reads of key rows 32h + 8 lg + {0..3} and {4..7}
        const int tr_row = 8 * lg + (lr >> 2), tr_byte = 8 * (lr & 3);
        #pragma unroll
        for (int h = 0; h < C::KH; ++h)
            #pragma unroll
            for (int db = 0; db < DB; ++db) {
                const int byte = db * 32 + tr_byte, chunk = byte >> 4, half = byte & 8;
                const int r0 = 32 * h + tr_row, r1 = r0 + 4;
                const v4s_t lo = lds_read_tr16(sv + r0 * C::RB + ((chunk ^ v_swz(r0)) << 4) + half);
                const v4s_t hi = lds_read_tr16(sv + r1 * C::RB + ((chunk ^ v_swz(r1)) << 4) + half);
                const bf16x8_v vf = __builtin_bit_cast(bf16x8_v, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                #pragma unroll
                for (int i = 0; i < NB; ++i) o[db][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[i][h], o[db][i], 0, 0, 0);
            }
    };

    store_lds(0, load_regs(0));
    __syncthreads();
    // Unconditional: the last pass reloads and restages its own tile into the
    // idle stage (nothing reads it), so the staging registers stay registers
    // (a conditional fill and drain sent them to scratch memory).
    for (int t = 0; t < nt; ++t) {
        const StageRegs next = load_regs(t + 1 < nt ? t + 1 : t);
        compute(t, t & 1);
        store_lds((t + 1) & 1, next);
        __syncthreads();
    }

    // ---- normalise and store: lane (lr, lg) holds features db*16 + 4 lg .. +3 of row lr ----
    bf16_t *obase = reinterpret_cast<bf16_t *>(slot_kind ? a.o_slot : a.o_raw) +
                    (size_t)b * (slot_kind ? a.slot_cap : a.q_cap) * a.Hq * D;
    float *lbase = slot_kind ? a.lse_slot : a.lse_raw;
    #pragma unroll
    for (int i = 0; i < NB; ++i) {
        const int j = wave + 4 * i, g = j % G, tb = j / G;
        const int tok = q0 + tb * 16 + lr;
        const float lt = prefill_row_sum(l_run[i]);
        if (tok > qlast) continue;
        const float inv = lt > 0.f ? 1.f / lt : 0.f;
        const size_t head = (size_t)tok * a.Hq + c * G + g;
        #pragma unroll
        for (int db = 0; db < DB; ++db) {
            const f32x4_v v = o[db][i];
            *reinterpret_cast<uint2 *>(obase + head * D + db * 16 + 4 * lg) =
                make_uint2(cvt_pk_bf16(v[0] * inv, v[1] * inv), cvt_pk_bf16(v[2] * inv, v[3] * inv));
        }
        if (lbase && lg == 0)
            lbase[(size_t)b * (slot_kind ? a.slot_cap : a.q_cap) * a.Hq + head] =
                lt > 0.f ? (m_run[i] * a.scale_log2 + log2f(lt)) * kLn2 : -INFINITY;
    }
}

// ------------------------------------------------------------------ host ----

// 16-row blocks per wave (two workgroups per CU)
static constexpr int prefill_nb(int) { return 2; }

int prefill_tokens_per_block(int d, int G) { return 16 * 4 * prefill_nb(d) / G; }

template <int D, int G>
static hipError_t launch_t(const PrefillArgs &a, hipStream_t st) {
    using C = PrefillCfg<D>;
    constexpr int NB = prefill_nb(D);
    dim3 grid((unsigned)(a.units * (a.nrb + a.nsb))), block(256);
    hipLaunchKernelGGL((prefill_kernel<D, G, NB>), grid, block, C::SMEM, st, a);
    return hipGetLastError();
}

template <int D>
static hipError_t launch_g(const PrefillArgs &a, int G, hipStream_t st) {
    switch (G) {
        case 1: return launch_t<D, 1>(a, st);
        case 2: return launch_t<D, 2>(a, st);
        case 4: return launch_t<D, 4>(a, st);
        case 8: return launch_t<D, 8>(a, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_prefill(const PrefillArgs &a, int d, int G, hipStream_t st) {
    if (d == 64) return launch_g<64>(a, G, st);
    if (d == 128) return launch_g<128>(a, G, st);
    return hipErrorInvalidValue;
}

}  // namespace mad
