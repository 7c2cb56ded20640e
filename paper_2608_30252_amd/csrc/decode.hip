// decode.hip -- draft decode attention over the compact MASW memory.
//
// One launch computes, for every (sequence b, KV head c), the attention of the
// G = Hq/Hkv query heads of the current token over the logical key sequence
//     [ memory rows 0..mlen-1 (sinks, then slots) | window ring rows 0..wlen-1 | new token ]
// (the working memory M_t of Sec. 3.1) and appends the new token's K/V to the
// window ring in the same pass (Sec. 3.2).  Per row the new token can also be
// attended without being appended (a slot's write scope that ends at the
// current token) or left out, so one launch serves a raw query and the write
// scopes of the slots made in the same pass.
//
// Work decomposition (split-K / flash-decoding): a (Hkv, B, n_splits) grid,
// so workgroup (c, b, z) finds its row's record from its own indices, in the
// same batch of argument reads as everything else its prologue needs.  It
// handles unit u = b * Hkv + c of the units = B * Hkv and key range
// s = n_splits - 1 - z (the last range, which holds the new token, is
// dispatched first).  Workgroups are dealt to the 8 XCDs
// round-robin by their linear id z * units + u, so with units a multiple of 8
// every split of a unit runs on one XCD.
//
// A workgroup is NSUB groups of four waves.  Keys stream through LDS in
// super-tiles of NSUB tiles, a tile being 8 KB of K + 8 KB of V (64 keys for
// bf16 with head_dim 64); group j owns tile j of every super-tile:
//   * all waves load each super-tile together straight from HBM into LDS
//     (global_load_lds_dwordx4, 16 bytes a lane, no VGPR round trip) through a
//     ring of stages; K rows are XOR-swizzled by 16-byte chunk on the way in so
//     the QK reads are bank-conflict free; a super-tile inside one segment
//     (memory, or the ring without a wrap) takes a uniform address path;
//   * everything after the load is wave-local: wave w of a group owns query
//     heads w, w+4, ... of the GQA group.  QK puts one key on each lane (query
//     rows in SGPRs or VGPRs, K chunks read from LDS in one burst), the tile
//     maximum of a head is a DPP row reduction plus row broadcasts and a
//     readlane, and PV runs over (feature pair, key subset) lanes, two keys per
//     v_dot2_f32_bf16 on bf16-rounded probabilities that the wave passes to
//     itself through a private LDS slice (the softmax normaliser keeps the
//     fp32 values).  One barrier per super-tile: the one that says it landed;
//   * the groups' running (max, sum, o) are merged in LDS into one partial per
//     workgroup;
//   * the last workgroup of a unit (one arrival counter per unit, on its own
//     256-byte line) pulls every split's partial into LDS with device-coherent
//     direct loads in a single round trip and merges them with the
//     log-sum-exp rule, one wave per head: all splits of the head in parallel
//     lanes for the weights, then the features in parallel lanes.
#include <type_traits>

#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

// phase marks of the diagnostic trace build: 0 entry, 1 partial stored and
// acknowledged, 2 arrival counter returned, 3 (merging workgroup) partials in
// LDS, 4 its first head merged, 5 merge done, 6 the first tiles' loads
// issued, 7 the first tile landed, 8 the prologue's kernel arguments read
MAD_TRACE_BUFFER(mad_trace_decode)

constexpr int kTileBytes = 16384;   // 8 KB of K + 8 KB of V
constexpr int kMergeLds = 69632;    // LDS that holds a unit's split partials in the merge (64 splits at G 4, d 64)

template <typename T, int D, int G, int NSUB>
struct DecodeCfg {
    static constexpr bool BF = std::is_same<T, bf16_t>::value;
    static constexpr int NT = 256 * NSUB;              // threads per workgroup
    static constexpr int NW = 4 * NSUB;                // waves
    static constexpr int ESZ = (int)sizeof(T);
    static constexpr int RB = D * ESZ;                 // bytes per K/V row
    static constexpr int TILE = 8192 / RB;             // keys per tile: 64, 32 or 16
    static constexpr int SUPER = NSUB * TILE;          // keys per super-tile
    static constexpr int STAGES = NSUB == 1 ? 4 : 2;   // super-tiles in the LDS ring
    static constexpr int SB = NSUB * kTileBytes;       // bytes per stage: [K: NSUB x 8 KB][V: NSUB x 8 KB]
    static constexpr int CPR = RB / 16;                // 16-byte chunks per row (>= 8)
    static constexpr int SW = 7;                       // K swizzle: chunk ^ (row & 7)
    static constexpr int RPI = 1024 / RB;              // rows per wave load (64 lanes x 16 B)
    static constexpr int LPT = 2;                      // K (and V) loads per thread per super-tile
    static constexpr int HPP = 64 / TILE;              // heads per QK pass of a wave
    static constexpr int HW = (G + 3) / 4;             // heads per wave
    static constexpr int NPASS = (HW + HPP - 1) / HPP; // QK passes per tile
    static constexpr int QW = RB / 4;                  // 32-bit words of one query row
    static constexpr int KB = 8;                       // K chunks read per batch
    static constexpr int DW = D / 2;                   // PV: each lane owns two features
    static constexpr int KSW = 64 / DW;                // PV key subsets per wave
    static constexpr int KPL = TILE / KSW;             // PV keys per lane per tile
    // a 64-key tile gives every wave one head per pass: its query rows (at most
    // two) come through the scalar cache, loaded at kernel start
    static constexpr bool QS = TILE == 64 && HW <= 2;
    // LDS: [stages (also the merge buffer) | Q: the unit's query rows | P: per-wave probabilities]
    static constexpr int SZ_ST = STAGES * SB;
    static constexpr int OFF_Q = SZ_ST > kMergeLds ? SZ_ST : kMergeLds;
    static constexpr int SZ_Q = (G * RB + 1023) / 1024 * 1024;
    static constexpr int OFF_P = OFF_Q + SZ_Q;
    static constexpr int SZ_P = NW * TILE * HW * 4;
    static constexpr int SMEM = OFF_P + SZ_P;
    static_assert(TILE * RB == 8192 && 4 * LPT * 1024 == 8192, "tile = 8 KB per tensor");
    static_assert(CPR % KB == 0 && KPL % 2 == 0 && 64 % DW == 0, "shape");
    static_assert(NSUB * G * (D + 2) * 4 <= SZ_ST, "group merge buffer fits the stages");
};

typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, a), __builtin_bit_cast(bf16x2_v, b), c,
                                           false);
}

// Max over aligned groups of N in {16, 32, 64} lanes, returned to every lane
// of the group.  A 16-lane row is reduced with DPP; rows are then folded with
// the row broadcasts (row 1 <- lane 15, row 3 <- lane 47 under row mask 0xa;
// rows 2 and 3 <- lane 31 under mask 0xc) and the group's last lane is read
// back as a wave-uniform value.
__device__ __forceinline__ float row_bcast15(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x142, 0xA, 0xF, false));
}
__device__ __forceinline__ float row_bcast31(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x143, 0xC, 0xF, false));
}
__device__ __forceinline__ float read_lane(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
template <int N> __device__ __forceinline__ float group_max_b(float v, int lane) {
    v = fmaxf(v, xor_lane<1>(v));
    v = fmaxf(v, xor_lane<2>(v));
    v = fmaxf(v, xor_lane<4>(v));
    v = fmaxf(v, xor_lane<8>(v));
    if constexpr (N == 16) {
        return v;
    } else if constexpr (N == 32) {
        v = fmaxf(v, row_bcast15(v));
        const float a = read_lane(v, 31), b = read_lane(v, 63);
        return lane < 32 ? a : b;
    } else {
        v = fmaxf(v, row_bcast15(v));
        v = fmaxf(v, row_bcast31(v));
        return read_lane(v, 63);
    }
}

// Where feature f of split s sits in the split's partial row: the D/4 feature
// quads rotated by (s mod SG) * 16 / SG places, SG = 256 / D.  The merge reads
// feature quad fq of splits s, s + 1, ... (s mod SG = 0) with consecutive lanes
// (lane = fq * SG + s mod SG), and with the rotation every 16 consecutive lanes
// touch 16 different 16-byte bank groups of the LDS.
template <int D> __device__ __forceinline__ int part_pos(int f, int s) {
    constexpr int FQ = D / 4, SG = 64 / FQ;
    return ((f / 4 + (s % SG) * (16 / SG)) % FQ) * 4 + f % 4;
}

// One batch of U splits of a lane, U consecutive ones of its split group (OS /
// MS bytes apart in the o / (m, l) arrays), folded into the lane's running
// (m, l, acc).  RAGGED: only the first `valid` are the unit's (the rest are
// repeats of a real split read with weight 0).  FIRST: the running state is
// still empty, so it needs no rescale.
template <int U, bool FIRST, bool RAGGED>
__device__ __forceinline__ void merge_batch(const float4 (&ov)[U], const float2 (&ml)[U], int valid, float &m,
                                            float &l, float4 &acc) {
    float mb = m;
    #pragma unroll
    for (int u = 0; u < U; ++u)
        if (!RAGGED || u < valid) mb = FIRST && u == 0 ? ml[0].x : __builtin_amdgcn_fmed3f(mb, ml[u].x, INFINITY);
    const float mr = mb == -INFINITY ? 0.f : mb;   // every weight 0 when the batch has no key
    if constexpr (!FIRST) {
        const float c = __builtin_amdgcn_exp2f(m - mr);
        l *= c;
        acc.x *= c; acc.y *= c; acc.z *= c; acc.w *= c;
    }
    #pragma unroll
    for (int u = 0; u < U; ++u) {
        float w = __builtin_amdgcn_exp2f(ml[u].x - mr);
        if (RAGGED && u >= valid) w = 0.f;
        if (FIRST && u == 0) {
            l = w * ml[u].y;
            acc = make_float4(w * ov[u].x, w * ov[u].y, w * ov[u].z, w * ov[u].w);
        } else {
            l = fmaf(w, ml[u].y, l);
            acc.x = fmaf(w, ov[u].x, acc.x);
            acc.y = fmaf(w, ov[u].y, acc.y);
            acc.z = fmaf(w, ov[u].z, acc.z);
            acc.w = fmaf(w, ov[u].w, acc.w);
        }
    }
    m = mb;
}

// Merge of a unit's split partials by its last-arriving workgroup (NT threads).
//   blk   unit block in the workspace: [o: n_splits][G][D] (features placed by
//         part_pos) [ml: n_splits][G][2]
//   lds   >= n_splits * G * (D + 2) * 4 bytes of LDS (16-byte aligned)
// One round trip pulls the whole block into LDS; then each wave merges whole
// heads on its own, with no further barrier.  Lane (fq, j) = lane fq * SG + j
// takes feature quad fq of the splits j, j + SG, j + 2 SG, ... with their
// (m, l) pairs, every read of a batch issued at once (a batch holds up to 8
// splits per lane; when SG divides the split count every lane has the same
// splits at fixed offsets).  The SG lanes of a quad then take their common
// maximum, rescale to it and sum, by DPP within the lane quad or pair; no split
// is read one at a time.
template <typename T, int D, int G, int NT>
__device__ __forceinline__ void merge_splits(const float *blk, int n_splits, unsigned char *lds, T *out, float *lse) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int FQ = D / 4;     // feature quads
    constexpr int SG = 64 / FQ;   // split groups: 4 at d 64, 2 at d 128
    static_assert(SG == 2 || SG == 4, "merge lane layout assumes d 64 or 128");
    constexpr int OS = SG * G * D * 4, MS = SG * G * 8;   // bytes from split s to s + SG
    const int fq = lane / SG, sg = lane % SG;
    const int slot = (fq + sg * (16 / SG)) % FQ;          // where quad fq sits in split sg's rows
    const int nbytes = (n_splits * G * (D + 2) * 4 + 15) & ~15;   // inside the 256-byte padded block
    // whole 1 KB pieces, a wave-uniform trip count; lanes past the block load
    // its last 16 bytes again into LDS past the block (never read)
    const int npieces = (nbytes + 1023) >> 10;
    const unsigned char *src = reinterpret_cast<const unsigned char *>(blk);
    #pragma unroll 4
    for (int pc = wave; pc < npieces; pc += NT / 64)
        lds_load16_coherent(src + min(pc * 1024 + lane * 16, nbytes - 16), lds + pc * 1024);
    const int ml_base = n_splits * G * D * 4;
    const int per_lane = n_splits / SG;   // whole batches of every lane when SG divides n_splits
    const bool even = per_lane * SG == n_splits && (per_lane <= 8 || per_lane % 8 == 0);
    wait_vm(0);
    __syncthreads();
    MAD_TRACE(mad_trace_decode, 3);

    for (int g = wave; g < G; g += NT / 64) {
        const unsigned char *po = lds + ((size_t)(sg * G + g) * D + slot * 4) * 4;   // split sg, head g, quad fq
        const unsigned char *pm = lds + ml_base + (size_t)(sg * G + g) * 8;
        float m = -INFINITY, l = 0.f;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        auto even_run = [&](auto u_const) {   // per_lane == U, or whole batches of U == 8
            constexpr int U = decltype(u_const)::value;
            for (int b = 0; b < per_lane; b += U) {
                float2 ml[U];
                float4 ov[U];
                #pragma unroll
                for (int u = 0; u < U; ++u) {
                    ml[u] = *reinterpret_cast<const float2 *>(pm + (size_t)(b + u) * MS);
                    ov[u] = *reinterpret_cast<const float4 *>(po + (size_t)(b + u) * OS);
                }
                if (b == 0) merge_batch<U, true, false>(ov, ml, U, m, l, acc);
                else merge_batch<U, false, false>(ov, ml, U, m, l, acc);
            }
        };
        if (even) {
            switch (per_lane) {
                case 1: even_run(std::integral_constant<int, 1>()); break;
                case 2: even_run(std::integral_constant<int, 2>()); break;
                case 3: even_run(std::integral_constant<int, 3>()); break;
                case 4: even_run(std::integral_constant<int, 4>()); break;
                case 5: even_run(std::integral_constant<int, 5>()); break;
                case 6: even_run(std::integral_constant<int, 6>()); break;
                case 7: even_run(std::integral_constant<int, 7>()); break;
                default: even_run(std::integral_constant<int, 8>()); break;
            }
        } else {
            // any split count: batches of 8 per lane, reads past the unit's
            // splits clamped to its last split and weighted 0
            constexpr int U = 8;
            const int mine = (n_splits - sg + SG - 1) / SG;   // this lane's splits
            for (int b = 0; b * SG < n_splits; b += U) {
                float2 ml[U];
                float4 ov[U];
                #pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int sp = min(sg + SG * (b + u), n_splits - 1);
                    ml[u] = *reinterpret_cast<const float2 *>(lds + ml_base + (size_t)(sp * G + g) * 8);
                    ov[u] = *reinterpret_cast<const float4 *>(lds + ((size_t)(sp * G + g) * D + slot * 4) * 4);
                }
                merge_batch<U, false, true>(ov, ml, mine - b, m, l, acc);
            }
        }
        // the SG lanes of a feature quad: common maximum, rescale, sums
        const float M = group_max<SG>(m);
        const float c = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M);
        const float L = group_sum<SG>(l * c);
        acc.x = group_sum<SG>(acc.x * c);
        acc.y = group_sum<SG>(acc.y * c);
        acc.z = group_sum<SG>(acc.z * c);
        acc.w = group_sum<SG>(acc.w * c);
        const float inv = L > 0.f ? __builtin_amdgcn_rcpf(L) : 0.f;
        if (g == 0) MAD_TRACE(mad_trace_decode, 4);
        if (sg == 0) {
            T *og = out + (size_t)g * D + 4 * fq;
            if constexpr (std::is_same<T, bf16_t>::value) {
                *reinterpret_cast<uint2 *>(og) = make_uint2(pack_bf16x2(acc.x * inv, acc.y * inv),
                                                            pack_bf16x2(acc.z * inv, acc.w * inv));
            } else {
                *reinterpret_cast<float4 *>(og) = make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
            }
        }
        if (lse && lane == 0) lse[g] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
    }
}

template <typename T, int D, int G, int NSUB>
__global__ __launch_bounds__(256 * NSUB, NSUB == 4 ? 1 : 2) void decode_kernel(const DecodeArgs a) {
    using C = DecodeCfg<T, D, G, NSUB>;
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char *sStage = smem;
    MAD_TRACE_T0();

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int grp = wave >> 2, wq = wave & 3;   // wave group (tile of the super-tile), wave in group
    // grid (KV head, row, split); the last split (the one holding the new token) is dispatched first
    const int c = blockIdx.x, b = blockIdx.y;
    // every kernel argument the prologue needs, read in one batch (one wait):
    // left to itself the compiler spreads these reads over six dependent
    // rounds (0.06 us on the compact layer).  With 8 or more query heads per KV
    // head the kernel has no SGPRs to spare for it.
    if constexpr (G <= 4) {
        const int4 sq0 = a.seq[b];
        asm volatile("" ::"s"(a.q), "s"(a.mk), "s"(a.mv), "s"(a.wk), "s"(a.wv), "s"(a.kn), "s"(a.vn),
                     "s"(a.m_seq), "s"(a.m_head), "s"(a.w_seq), "s"(a.w_head), "s"(a.chunk), "s"(a.w_cap),
                     "s"(a.n_splits), "s"(a.Hq), "s"(a.fold), "s"(sq0.x), "s"(sq0.y), "s"(sq0.z), "s"(sq0.w),
                     "s"(gridDim.x), "s"(gridDim.z));
    }
    MAD_TRACE_VAR(t_args);
    MAD_TRACE_SET(t_args);
    const int u = b * (int)gridDim.x + c, s = (int)gridDim.z - 1 - (int)blockIdx.z;
    const int4 sq = a.seq[b];
    const int mlen = sq.x, wlen = sq.y, wst = sq.z;
    const int nmode = a.kn != nullptr ? sq.w : 0;
    const bool has_new = nmode >= 1;      // the key sequence ends with the current token
    const bool appends = nmode == 2;      // ... which this row also writes into its ring
    const int n = mlen + wlen + (has_new ? 1 : 0);
    const int k0 = s * a.chunk;
    const int k1 = (a.fold && s == a.n_splits - 1) ? n : min(n, k0 + a.chunk);
    const int w_cap = a.w_cap;

    // the unit's arrival counter, taken at entry and pinned in SGPRs (pin_sgpr):
    // not re-read between a split's last partial store and its arrival, which
    // becomes a flat atomic -- 7.09 -> 7.00 us on the compact layer (pinning
    // it as a global pointer gained nothing).  With 8 or more query heads per
    // KV head the kernel has no SGPRs to spare for it.
    uint64_t cnt_addr = 0;
    if constexpr (G <= 4) {
        cnt_addr = ptr_bits(a.counters + (size_t)u * kCounterStride);
        pin_sgpr(cnt_addr);
    }
    const T *mk = reinterpret_cast<const T *>(a.mk) + b * a.m_seq + c * a.m_head;
    const T *mv = reinterpret_cast<const T *>(a.mv) + b * a.m_seq + c * a.m_head;
    T *wk = reinterpret_cast<T *>(a.wk) + b * a.w_seq + c * a.w_head;
    T *wv = reinterpret_cast<T *>(a.wv) + b * a.w_seq + c * a.w_head;
    const size_t nrow = ((size_t)b * a.Hkv + c) * D;
    const T *nk = has_new ? reinterpret_cast<const T *>(a.kn) + nrow : nullptr;
    const T *nv = has_new ? reinterpret_cast<const T *>(a.vn) + nrow : nullptr;
    const size_t head0 = (size_t)b * a.Hq + (size_t)c * G;

    // ---- query rows ----
    // QS: each wave's rows in SGPRs.  Otherwise the unit's G rows go to LDS by
    // the same direct loads as the tiles (older than every tile load, so the
    // first tile's wait covers them; lanes past the rows fetch the last chunk
    // again into the padding of the region) and each lane copies its row out.
    uint32_t qsr[C::QS ? C::HW : 1][C::QW];
    if constexpr (C::QS) {
        #pragma unroll
        for (int hi = 0; hi < C::HW; ++hi) {
            const int g = wq + 4 * hi;
            load_uniform_dwords<C::QW>(reinterpret_cast<const T *>(a.q) + (head0 + (g < G ? g : 0)) * D, qsr[hi]);
        }
    } else {
        const unsigned char *qsrc = reinterpret_cast<const unsigned char *>(a.q) + head0 * C::RB;
        for (int off = wave * 1024; off < G * C::RB; off += C::NT * 16) {
            const int o = min(off + lane * 16, G * C::RB - 16);
            lds_stream16(qsrc + o, smem + C::OFF_Q + off);
        }
    }
    const int qj = lane % C::TILE, qhs = lane / C::TILE;
    uint32_t qv[C::QS ? 1 : C::NPASS][C::QW];

    // ---- super-tile loader: direct HBM -> LDS, 2 K + 2 V instructions per thread ----
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
    auto issue = [&](int tb, int stage) {
        unsigned char *st = sStage + stage * C::SB;
        // a full super-tile inside one segment (memory, or the ring without a
        // wrap) has one base address for all its rows: a wave-uniform test
        const T *kb = nullptr, *vb = nullptr;
        if (tb + C::SUPER <= k1) {
            if (tb + C::SUPER <= mlen) {
                kb = mk + (size_t)tb * D;
                vb = mv + (size_t)tb * D;
            } else if (tb >= mlen && tb + C::SUPER <= mlen + wlen) {
                int r0 = wst + (tb - mlen);
                if (r0 >= w_cap) r0 -= w_cap;
                if (r0 + C::SUPER <= w_cap) {
                    kb = wk + (size_t)r0 * D;
                    vb = wv + (size_t)r0 * D;
                }
            }
        }
        #pragma unroll
        for (int l = 0; l < C::LPT; ++l) {
            const int inst = l * C::NW + wave;             // 1 KB block of the NSUB x 8 KB tensor super-tile
            const int row = inst * C::RPI + lane / C::CPR;
            const int slot = lane % C::CPR;
            const T *kp, *vp;
            if (kb != nullptr) {
                kp = kb + (size_t)row * D;
                vp = vb + (size_t)row * D;
            } else {
                kp = row_src(tb + row, false);
                vp = row_src(tb + row, true);
            }
            // K: LDS slot `slot` of row `row` holds global chunk slot ^ (row & SW)
            lds_stream16_nt(reinterpret_cast<const uint4 *>(kp) + (slot ^ (row & C::SW)), st + inst * 1024);
            lds_stream16_nt(reinterpret_cast<const uint4 *>(vp) + slot, st + NSUB * 8192 + inst * 1024);
        }
    };

    // ---- running state of this wave (heads wq + 4 hi, keys of tile `grp`) ----
    float m_run[C::NPASS], l_lane[C::NPASS];
    #pragma unroll
    for (int p = 0; p < C::NPASS; ++p) { m_run[p] = -INFINITY; l_lane[p] = 0.f; }
    float o_acc[C::HW][2];
    #pragma unroll
    for (int hi = 0; hi < C::HW; ++hi) o_acc[hi][0] = o_acc[hi][1] = 0.f;
    const int pv_dp = lane % C::DW, pv_ks = lane / C::DW;
    unsigned char *sP = smem + C::OFF_P + wave * (C::TILE * C::HW * 4);   // this wave's slice
    const bool wave_active = wq < G;

    const int nst = (k1 > k0) ? (k1 - k0 + C::SUPER - 1) / C::SUPER : 0;
    int issued = 0;
    for (; issued < nst && issued < C::STAGES - 1; ++issued) issue(k0 + issued * C::SUPER, issued);
    MAD_TRACE_VAR(t_issued);
    MAD_TRACE_SET(t_issued);
    MAD_TRACE_VAR(t_landed);

    for (int t = 0; t < nst; ++t) {
        wait_vm(4 * (issued - t - 1));
        __syncthreads();   // super-tile t is in LDS for every wave; stage (t-1) % STAGES is free
        if (t == 0) MAD_TRACE_SET(t_landed);
        if (issued < nst) {
            issue(k0 + issued * C::SUPER, issued % C::STAGES);
            ++issued;
        }
        const int base = k0 + t * C::SUPER + grp * C::TILE;   // first key of this group's tile
        if (!wave_active || base >= k1) continue;
        if (!C::QS && t == 0) {
            // this lane's query row in each QK pass: head wq + 4 (pass * HPP + lane / TILE)
            #pragma unroll
            for (int p = 0; p < C::NPASS; ++p) {
                const int hi = p * C::HPP + qhs, g = wq + 4 * hi;
                const uint4 *qs = reinterpret_cast<const uint4 *>(smem + C::OFF_Q + ((hi < C::HW && g < G) ? g : 0) * C::RB);
                #pragma unroll
                for (int ch = 0; ch < C::QW / 4; ++ch) {
                    const uint4 v = qs[ch];
                    qv[p][4 * ch + 0] = v.x; qv[p][4 * ch + 1] = v.y; qv[p][4 * ch + 2] = v.z; qv[p][4 * ch + 3] = v.w;
                }
            }
        }
        const unsigned char *st = sStage + (t % C::STAGES) * C::SB;
        const unsigned char *sk = st + grp * 8192;
        const unsigned char *sv = st + NSUB * 8192 + grp * 8192;

        // ---- QK, softmax statistics and the probabilities, pass by pass ----
        float al[C::HW];
        #pragma unroll
        for (int p = 0; p < C::NPASS; ++p) {
            const int hi = p * C::HPP + qhs;
            const bool act = hi < C::HW && wq + 4 * hi < G;
            const uint4 *krow = reinterpret_cast<const uint4 *>(sk + qj * C::RB);
            float acc0 = 0.f, acc1 = 0.f;
            #pragma unroll
            for (int cb = 0; cb < C::CPR; cb += C::KB) {
                uint4 kc[C::KB];
                #pragma unroll
                for (int i = 0; i < C::KB; ++i) kc[i] = krow[(cb + i) ^ (qj & C::SW)];
                #pragma unroll
                for (int i = 0; i < C::KB; ++i) {
                    const uint32_t *qq = C::QS ? &qsr[p][4 * (cb + i)] : &qv[p][4 * (cb + i)];
                    float &acc = (i & 1) ? acc1 : acc0;
                    if constexpr (C::BF) {
                        acc = dot2_bf16(qq[0], kc[i].x, acc);
                        acc = dot2_bf16(qq[1], kc[i].y, acc);
                        acc = dot2_bf16(qq[2], kc[i].z, acc);
                        acc = dot2_bf16(qq[3], kc[i].w, acc);
                    } else {
                        acc = fmaf(__uint_as_float(qq[0]), __uint_as_float(kc[i].x), acc);
                        acc = fmaf(__uint_as_float(qq[1]), __uint_as_float(kc[i].y), acc);
                        acc = fmaf(__uint_as_float(qq[2]), __uint_as_float(kc[i].z), acc);
                        acc = fmaf(__uint_as_float(qq[3]), __uint_as_float(kc[i].w), acc);
                    }
                }
            }
            const float sc = (act && base + qj < k1) ? (acc0 + acc1) * a.scale_log2 : -INFINITY;
            const float tmax = group_max_b<C::TILE>(sc, lane);
            const float mn = fmaxf(m_run[p], tmax);
            const bool live = mn != -INFINITY;   // false only for heads this lane does not own
            const float alpha = live ? __builtin_amdgcn_exp2f(m_run[p] - mn) : 1.f;
            const float pr = live ? __builtin_amdgcn_exp2f(sc - mn) : 0.f;
            m_run[p] = mn;
            l_lane[p] = fmaf(l_lane[p], alpha, pr);
            if constexpr (C::BF) {
                // PV consumes the probabilities rounded to bf16 and packed by key pairs
                const uint32_t pb = (uint32_t)f32_to_bf16(pr);
                const uint32_t pn = (uint32_t)__float_as_int(xor_lane<1>(__int_as_float((int)pb)));
                if (act && (qj & 1) == 0)
                    reinterpret_cast<uint32_t *>(sP)[(qj >> 1) * C::HW + hi] = pb | (pn << 16);
            } else {
                if (act) reinterpret_cast<float *>(sP)[qj * C::HW + hi] = pr;
            }
            #pragma unroll
            for (int hs = 0; hs < C::HPP; ++hs)
                if (p * C::HPP + hs < C::HW) al[p * C::HPP + hs] = read_lane(alpha, hs * C::TILE);
        }

        // ---- PV over this wave's heads ----
        #pragma unroll
        for (int hi = 0; hi < C::HW; ++hi) { o_acc[hi][0] *= al[hi]; o_acc[hi][1] *= al[hi]; }
        if constexpr (C::BF) {
            // all V words and probabilities of the tile first, then the products
            // (one LDS round trip instead of one per key pair)
            uint32_t vw[C::KPL], pw[C::KPL / 2][C::HW];
            #pragma unroll
            for (int k = 0; k < C::KPL; ++k)
                vw[k] = reinterpret_cast<const uint32_t *>(sv + (pv_ks * C::KPL + k) * C::RB)[pv_dp];
            #pragma unroll
            for (int k = 0; k < C::KPL / 2; ++k)
                #pragma unroll
                for (int hi = 0; hi < C::HW; ++hi)
                    pw[k][hi] = reinterpret_cast<const uint32_t *>(sP)[((pv_ks * C::KPL >> 1) + k) * C::HW + hi];
            #pragma unroll
            for (int k = 0; k < C::KPL / 2; ++k) {
                const uint32_t lo = __builtin_amdgcn_perm(vw[2 * k + 1], vw[2 * k], 0x05040100u);   // feature 2dp
                const uint32_t hi2 = __builtin_amdgcn_perm(vw[2 * k + 1], vw[2 * k], 0x07060302u);  // feature 2dp+1
                #pragma unroll
                for (int hi = 0; hi < C::HW; ++hi) {
                    o_acc[hi][0] = dot2_bf16(pw[k][hi], lo, o_acc[hi][0]);
                    o_acc[hi][1] = dot2_bf16(pw[k][hi], hi2, o_acc[hi][1]);
                }
            }
        } else {
            float2 vf[C::KPL];
            #pragma unroll
            for (int k = 0; k < C::KPL; ++k)
                vf[k] = reinterpret_cast<const float2 *>(sv + (pv_ks * C::KPL + k) * C::RB)[pv_dp];
            #pragma unroll
            for (int k = 0; k < C::KPL; ++k) {
                const float *pj = reinterpret_cast<const float *>(sP) + (pv_ks * C::KPL + k) * C::HW;
                #pragma unroll
                for (int hi = 0; hi < C::HW; ++hi) {
                    const float pf = pj[hi];
                    o_acc[hi][0] = fmaf(pf, vf[k].x, o_acc[hi][0]);
                    o_acc[hi][1] = fmaf(pf, vf[k].y, o_acc[hi][1]);
                }
            }
        }
    }

    // ---- append the new token to the window ring (the workgroup holding it) ----
    // Its row is outside every window of this launch (the window ends just
    // before it), and attention above read the token from k_new / v_new.
    if (appends && k0 <= n - 1 && n - 1 < k1) {
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

    // ---- this wave's per-head (max, sum, o) ----
    const int n_splits = a.n_splits;
    T *out = reinterpret_cast<T *>(a.out) + head0 * D;
    float *blk = a.part + (size_t)u * a.part_stride;
    // group results go to LDS ([group][G][D] o, then [group][G] (max, sum)) and
    // are merged there; one group writes them straight out
    float *go = reinterpret_cast<float *>(sStage);
    float2 *gml = reinterpret_cast<float2 *>(go + NSUB * G * D);
    if constexpr (NSUB > 1) __syncthreads();   // every wave is done with the stages
    if (wave_active) {
        float l_tot[C::NPASS];
        #pragma unroll
        for (int p = 0; p < C::NPASS; ++p) l_tot[p] = group_sum<C::TILE>(l_lane[p]);
        #pragma unroll
        for (int hi = 0; hi < C::HW; ++hi) {
            if constexpr (C::KSW == 2) {
                o_acc[hi][0] = pair_sum<32>(o_acc[hi][0]);
                o_acc[hi][1] = pair_sum<32>(o_acc[hi][1]);
            }
        }
        #pragma unroll
        for (int hi = 0; hi < C::HW; ++hi) {
            const int g = wq + 4 * hi;
            if (g >= G) continue;
            const int p = hi / C::HPP, hs = hi % C::HPP;
            const float mm = read_lane(m_run[p], hs * C::TILE);   // -inf when the group had no keys
            const float l = read_lane(l_tot[p], hs * C::TILE);
            if constexpr (NSUB > 1) {
                if (pv_ks == 0)
                    reinterpret_cast<float2 *>(go + ((size_t)grp * G + g) * D)[pv_dp] = make_float2(o_acc[hi][0], o_acc[hi][1]);
                if (lane == 0) gml[grp * G + g] = make_float2(mm, l);
            } else if (n_splits == 1) {
                if (pv_ks == 0) {
                    const float inv = l > 0.f ? 1.f / l : 0.f;
                    Elem<T>::store1(out + g * D + 2 * pv_dp, o_acc[hi][0] * inv);
                    Elem<T>::store1(out + g * D + 2 * pv_dp + 1, o_acc[hi][1] * inv);
                }
                if (a.lse && lane == 0) a.lse[head0 + g] = l > 0.f ? (mm + log2f(l)) * kLn2 : -INFINITY;
            } else {
                // partial of this split: unit block = [o: n_splits][G][D] [ml: n_splits][G][2]
                float *po = blk + ((size_t)s * G + g) * D;
                if (pv_ks == 0) store_agent2(po + part_pos<D>(2 * pv_dp, s), o_acc[hi][0], o_acc[hi][1]);
                if (lane == 0) store_agent2(blk + (size_t)n_splits * G * D + ((size_t)s * G + g) * 2, mm, l);
            }
        }
    }
    if constexpr (NSUB > 1) {
        __syncthreads();
        // merge the groups: per (head g, feature d), weights 2^(m_j - M)
        for (int idx = tid; idx < G * D; idx += C::NT) {
            const int g = idx / D;
            float mj[NSUB], M = -INFINITY;
            #pragma unroll
            for (int j = 0; j < NSUB; ++j) { mj[j] = gml[j * G + g].x; M = fmaxf(M, mj[j]); }
            float L = 0.f, O = 0.f;
            #pragma unroll
            for (int j = 0; j < NSUB; ++j) {
                const float w = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mj[j] - M);
                L = fmaf(w, gml[j * G + g].y, L);
                O = fmaf(w, go[(size_t)j * G * D + idx], O);
            }
            if (n_splits == 1) {
                Elem<T>::store1(out + idx, L > 0.f ? O / L : 0.f);
                if (a.lse && idx % D == 0) a.lse[head0 + g] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
            } else {
                store_agent(blk + ((size_t)s * G + g) * D + part_pos<D>(idx % D, s), O);
                if (idx % D == 0) store_agent2(blk + (size_t)n_splits * G * D + ((size_t)s * G + g) * 2, M, L);
            }
        }
    }
    if (n_splits == 1) return;
    // every head g < G belongs to exactly one active wave: the block is complete
    wait_vm_stores();
    __syncthreads();
    MAD_TRACE_VAR(t_arrive);
    MAD_TRACE_SET(t_arrive);   // stored after the atomic, whose wait would count the store
    __shared__ int s_last;
    if (tid == 0) {
        unsigned *cnt = G <= 4 ? bits_ptr<unsigned>(cnt_addr) : a.counters + (size_t)u * kCounterStride;
        const int last = arrive(cnt) == (unsigned)(n_splits - 1);
        MAD_TRACE(mad_trace_decode, 2);
        MAD_TRACE_SAVE_T0(mad_trace_decode);
        MAD_TRACE_PUT(mad_trace_decode, 1, t_arrive);
        MAD_TRACE_PUT(mad_trace_decode, 6, t_issued);
        MAD_TRACE_PUT(mad_trace_decode, 7, t_landed);
        MAD_TRACE_PUT(mad_trace_decode, 8, t_args);
        if (last) reset_counter(cnt);
        s_last = last;
    }
    __syncthreads();
    if (!s_last) return;
    merge_splits<T, D, G, C::NT>(blk, n_splits, sStage, out, a.lse ? a.lse + head0 : nullptr);
    MAD_TRACE(mad_trace_decode, 5);
}

// ------------------------------------------------------------------ host ----

int decode_max_splits(int d, int G) {
    const int cap = kMergeLds / (G * (d + 2) * 4);   // merge block must fit its LDS
    return cap < kDecodeMaxSplits ? cap : kDecodeMaxSplits;
}

static int decode_tile(int dtype, int d) { return 8192 / (d * (dtype == MAD_BF16 ? 2 : 4)); }

// Two-group workgroups (8 waves, two per CU) for bf16 with head_dim 64 and at
// most 4 query heads per KV head when the launch holds many keys (long
// streams or many sequences, where two tiles in flight per workgroup and fewer
// partials pay); one-group workgroups (4 waves, about two tiles per split)
// for short streams, where the first loads are spread over as many CUs as
// possible.
static int decode_nsub(int units, int n_max, int G, int d, int dtype) {
    if (!(dtype == MAD_BF16 && d == 64 && G <= 4)) return 1;
    const bool wide = (int64_t)units * n_max >= kDecodeWideKeys;
    return wide ? 2 : 1;
}

DecodePlan plan_decode(int B, int Hkv, int G, int d, int dtype, const int *n_keys) {
    DecodePlan p;
    p.units = B * Hkv;
    p.n_max = 0;
    for (int b = 0; b < B; ++b) p.n_max = n_keys[b] > p.n_max ? n_keys[b] : p.n_max;
    p.nsub = decode_nsub(p.units, p.n_max, G, d, dtype);
    const int super = p.nsub * decode_tile(dtype, d);
    // workgroups to aim for: two per CU with 8 waves; with 4 waves one per CU
    // for a short stream (the first loads spread over every CU decide the time),
    // two per CU when there is enough work to need the loads in flight of both
    const int64_t total = (int64_t)p.units * p.n_max;
    const int per_cu = p.nsub == 2 ? 2 : (total >= kDecodeWideKeys ? 2 : 1);
    const int target = per_cu * kDecodeCUs;
    int ns = (target + p.units - 1) / p.units;
    const int cap = decode_max_splits(d, G);
    if (ns > cap) ns = cap;
    if (ns < 1) ns = 1;
    // Whole super-tiles per split.  Rounding the even share down leaves a few
    // keys (e.g. the new token) for one short extra split per unit, which the
    // grid dispatches first -- unless the extra workgroups would not all be
    // resident at once (two per CU), where they would start only as others
    // finish: then the last split takes those keys (one more, mostly masked,
    // super-tile), and every CU keeps the same share (the full 32K KV: 64
    // splits of 512 keys, 512 workgroups, against 52 of 640 whose 416
    // workgroups put two on some CUs and one on others).  When the leftover
    // is more than a sliver the share is rounded up instead (one split fewer,
    // the last one short).
    const int share = p.n_max / ns;
    const int down = share / super * super;
    int chunk;
    p.fold = 0;
    if (down >= super && p.n_max - ns * down <= down / 8) {
        chunk = down;
        if (p.n_max > ns * down && (int64_t)p.units * (ns + 1) > 2 * kDecodeCUs) {
            p.n_splits = ns;
            p.chunk = chunk;
            p.fold = 1;
            return p;
        }
    } else {
        chunk = ((p.n_max + ns - 1) / ns + super - 1) / super * super;
    }
    if (chunk < super) chunk = super;
    ns = (p.n_max + chunk - 1) / chunk;
    if (ns > cap) {   // the extra split would not fit the merge
        chunk = ((p.n_max + cap - 1) / cap + super - 1) / super * super;
        ns = (p.n_max + chunk - 1) / chunk;
    }
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

template <typename T, int D, int G, int NSUB>
static hipError_t launch_t(const DecodeArgs &a, hipStream_t st) {
    using C = DecodeCfg<T, D, G, NSUB>;
    dim3 grid((unsigned)a.Hkv, (unsigned)(a.units / a.Hkv), (unsigned)a.n_splits), block(C::NT);
    hipLaunchKernelGGL((decode_kernel<T, D, G, NSUB>), grid, block, C::SMEM, st, a);
    return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_g(const DecodeArgs &a, int G, hipStream_t st) {
    if constexpr (std::is_same<T, bf16_t>::value && D == 64) {
        if (a.nsub == 2) {
            switch (G) {
                case 1: return launch_t<T, D, 1, 2>(a, st);
                case 2: return launch_t<T, D, 2, 2>(a, st);
                case 4: return launch_t<T, D, 4, 2>(a, st);
            }
            return hipErrorInvalidValue;
        }
    }
    if (a.nsub != 1) return hipErrorInvalidValue;
    switch (G) {
        case 1: return launch_t<T, D, 1, 1>(a, st);
        case 2: return launch_t<T, D, 2, 1>(a, st);
        case 4: return launch_t<T, D, 4, 1>(a, st);
        case 8: return launch_t<T, D, 8, 1>(a, st);
        case 16: return launch_t<T, D, 16, 1>(a, st);
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
