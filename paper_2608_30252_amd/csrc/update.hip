// update.hip -- memory update by the MASW memory adaptor (Sec. 3.2).
//
// For every new memory slot row r = (sequence b, slot i) the mirrored
// projections give  [k~ | v] = x[r] . [W_K,g ; W_V,g]^T,  the key is rotated at
// the slot's position id (the id of the raw token that follows the slot), and
// the pair is appended at memory row len[b] + i.  Rows of sequences whose fire
// flag is 0 are computed but not written (per-sequence masks of heterogeneous
// batches, Sec. 4.1).
//
// BF16 with at most 8 rows (a single sequence's update, or a few): a weight
// stream (update_gemv_kernel).  The projection is then a matrix-vector
// product per row, bound by reading W once; a workgroup owns NC output
// features -- rotate-half pairs (j, j + d/2) of one K or V head -- over the
// whole input width, so no split partials and no merge: thread t holds the
// 16-byte chunks t, t + 256, ... of every row and of the NC weight rows (all
// loads issued together), products by v_dot2_f32_bf16, wave and workgroup
// sums, then RoPE on the K pairs and the append.
// BF16 with more rows: the projection Y[R x 2 Hkv d] = X W^T runs on the
// matrix cores (v_mfma_f32_16x16x32_bf16, fp32 accumulation) in 16 x 16 output
// tiles, each over the whole input width (update_rows_kernel): again no split
// partials, no merge and no workspace.  The tile's 32 input rows go through
// LDS: a CU pulls them from L2 fastest as whole 1-KB row pieces per wave load
// with many waves in flight, which the MFMA operand layout (16 rows per load)
// does not give; when the whole width fits LDS at once they are loaded
// straight into it (global_load_lds_dwordx4) and the products follow them
// block by block.
// F32: a vector-ALU kernel, one thread per (row, rotation pair).
#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

// phase marks of the diagnostic trace build (update_rows_kernel): 0 entry,
// 1 the first rows in LDS, 2 products done, 4 partial tiles in LDS, 5 tile
// summed (thread 0's rows), 6 summed tile in LDS, 3 stored
MAD_TRACE_BUFFER(mad_trace_update)

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_v;
typedef __attribute__((ext_vector_type(4))) float f32x4_v;


// BF16 with more than 8 rows: workgroup (feature block fb, row tile rt) owns a
// 16 x 16 tile of Y -- 16 slot rows by 8 rotate-half pairs (j, j + d/2) of one
// K or V head -- over the whole input width, so no split partials and no merge.
// Each round copies 2048 columns of the tile's 16 W rows and 16 X rows into LDS
// (every wave load is 1 KB of one row, consecutive lanes on consecutive 16
// bytes; rows padded by 16 bytes so the operand reads below are free of bank
// conflicts); wave w then runs the 32-wide k-steps w, w + NW, ... of the round
// from LDS in the MFMA register layout (lane l: row / feature l % 16, k chunk
// l / 16), and the NW partial tiles are summed through LDS.  An input width of
// at most one round (DIRECT) is loaded straight into LDS by 512-column block
// and each block's k-steps start as soon as it has landed; wider inputs go
// through registers, the next round's loads issued before this round's
// MFMAs.  Both run the k-steps of a wave in the same order (bit-identical
// results).  The row tiles of one feature
// block are dealt to one XCD (workgroups go round-robin over the 8 XCDs, so
// blockIdx mod 8 is kept), where they share its weight rows in L2; the order
// affects only where data is cached, never the result.  The RoPE angles and
// the epilogue's kernel arguments are taken at entry, while the rows are in
// flight, and each tile row leaves as two 16-byte stores.
template <int NW, bool DIRECT>
__global__ __launch_bounds__(64 * NW) void update_rows_kernel(const UpdateArgs a) {
    constexpr int KR = 2048, PITCH = 2 * KR + 16, PIECES = 32 * KR / 512, PW = PIECES / NW;
    static_assert(PIECES % NW == 0, "whole pieces per wave");
    __shared__ __attribute__((aligned(16))) unsigned char s_rows[32 * PITCH];   // rows 0-15: W, 16-31: X
    __shared__ f32x4_v s_acc[NW][64];
    __shared__ __attribute__((aligned(16))) uint16_t s_out[16][16];   // [tile row][pair | pair + 8]
    MAD_TRACE_T0();
    MAD_TRACE_VAR(t_rows);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // The kernel arguments come in two batches, each read with one wait and
    // kept as opaque copies (left to the compiler, the reads are spread over
    // dependent rounds, and the epilogue's are issued after the last barrier):
    // what the row loads need, here; what the epilogue needs, once the row
    // loads are issued.
    uint64_t xb = ptr_bits(a.x), wb = ptr_bits(a.w);
    int R = a.R, D = a.D, d = a.d, Hkv = a.Hkv, n_new = a.n_new;
    asm volatile("" : "+s"(xb), "+s"(wb), "+s"(R), "+s"(D), "+s"(d), "+s"(Hkv), "+s"(n_new));
    uint64_t mkb = 0, mvb = 0;
    int64_t m_head = 0, m_seq = 0;
    auto epilogue_args = [&]() {
        mkb = ptr_bits(a.mk);
        mvb = ptr_bits(a.mv);
        m_head = a.m_head;
        m_seq = a.m_seq;
        asm volatile("" : "+s"(mkb), "+s"(mvb), "+s"(m_head), "+s"(m_seq));
    };
    const int hd = d / 2;
    const int RT = (R + 15) >> 4;
    const int li = blockIdx.x >> 3;   // grid = (2 Hkv d / 16) feature blocks (a multiple of 8) x RT
    const int fb = 8 * (li / RT) + (blockIdx.x & 7), rt = li % RT;
    const int hb = fb / (d / 16), j0 = (fb % (d / 16)) * 8;
    const bool is_k = hb < Hkv;
    const int c = lane & 15, kq = lane >> 4;

    // thread t < 128 rotates pair t % 8 of tile row t / 8; thread t < 32 stores half t % 2 of tile row t / 2.
    // Its angle is taken once the row loads are issued, and its row's position
    // comes through the scalar cache (the tile's 16 positions, a wave-uniform
    // read) and a lane permute: a vector-memory read would need a wait that
    // also waits for the row loads.
    int tpos[16];
    #pragma unroll
    for (int i = 0; i < 16; ++i) tpos[i] = a.pos[rt * 16 + i];   // rows past R: never stored
    float rc = 1.f, rs = 0.f;
    auto rope_angles = [&]() {
        if (is_k && tid < 128) {
            int pv = 0;
            #pragma unroll
            for (int i = 0; i < 16; ++i)   // lane i: row i
                asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(pv) : "s"(tpos[i]), "n"(i));
            pv = __builtin_amdgcn_ds_bpermute(((tid >> 3) & 15) << 2, pv);
            rope_cs(pv, rope_theta(j0 + (tid & 7), d, a.log2_base), &rc, &rs);
        }
    };
    const int s_row = rt * 16 + ((tid >> 1) & 15), s_b = min(s_row, R - 1) / n_new;
    const int s_fire = a.fire[s_b], s_mlen = a.mlen[s_b];

    const bf16_t *w = bits_ptr<const bf16_t>(wb);
    const bf16_t *x = bits_ptr<const bf16_t>(xb);
    f32x4_v acc = f32x4_v{0.f, 0.f, 0.f, 0.f};
    if constexpr (DIRECT) {
        // one round (D <= KR): the pieces go straight from memory into LDS
        // (global_load_lds_dwordx4: no VGPR hop, no LDS write instructions),
        // issued by 512-column block -- wave w loads block b of rows w and
        // w + 16 as its loads 2b and 2b + 1 -- so the products of block b start
        // while the later blocks are still arriving.  Lanes past D load the
        // row's last chunk again (never read) so every wave issues all PW loads
        // and the counted waits hold.
        static_assert(PW == 8 && NW == 16, "two rows x four column blocks per wave");
        #pragma unroll
        for (int i = 0; i < PW; ++i) {
            const int row = wave + 16 * (i & 1), cb = i >> 1;
            const bf16_t *rp = row < 16 ? w + (size_t)(hb * d + (row < 8 ? j0 + row : hd + j0 + row - 8)) * D
                                        : x + (size_t)min(rt * 16 + row - 16, R - 1) * D;
            lds_stream16(rp + min(cb * 512 + lane * 8, D - 8), s_rows + row * PITCH + cb * 1024);
        }
        // the epilogue's arguments and the RoPE angles while the rows are in flight
        epilogue_args();
        rope_angles();
        const int nst = D >> 5;
        #pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
            wait_vm(PW - 2 * (cb + 1));   // this wave's loads of blocks 0 .. cb have landed
            __syncthreads();              // ... every wave's
            if (cb == 0) MAD_TRACE_SET(t_rows);
            const int t = cb * NW + wave;
            if (t < nst) {
                const bf16x8_v bv = *reinterpret_cast<const bf16x8_v *>(s_rows + c * PITCH + t * 64 + kq * 16);
                const bf16x8_v av = *reinterpret_cast<const bf16x8_v *>(s_rows + (16 + c) * PITCH + t * 64 + kq * 16);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
            }
        }
    } else {
        // piece pc = wave + NW i: row pc / 4, columns 512 (pc % 4) .. + 511 of
        // the round, through registers so the next round's loads overlap this
        // round's products
        const bf16_t *src[PW];
        #pragma unroll
        for (int i = 0; i < PW; ++i) {
            const int row = (wave + NW * i) >> 2;
            src[i] = row < 16 ? w + (size_t)(hb * d + (row < 8 ? j0 + row : hd + j0 + row - 8)) * D
                              : x + (size_t)min(rt * 16 + row - 16, R - 1) * D;
        }
        uint4 buf[PW];
        auto load = [&](int r0) {
            #pragma unroll
            for (int i = 0; i < PW; ++i) {
                const int col = r0 + ((wave + NW * i) & 3) * 512 + lane * 8;
                buf[i] = col < D ? *reinterpret_cast<const uint4 *>(src[i] + col) : make_uint4(0u, 0u, 0u, 0u);
            }
        };
        load(0);
        epilogue_args();
        rope_angles();
        for (int r0 = 0; r0 < D; r0 += KR) {
            #pragma unroll
            for (int i = 0; i < PW; ++i) {
                const int pc = wave + NW * i;
                *reinterpret_cast<uint4 *>(s_rows + (pc >> 2) * PITCH + (pc & 3) * 1024 + lane * 16) = buf[i];
            }
            __syncthreads();
            if (r0 == 0) MAD_TRACE_SET(t_rows);
            if (r0 + KR < D) load(r0 + KR);
            const int nst = min(KR, D - r0) >> 5;
            for (int t = wave; t < nst; t += NW) {
                const bf16x8_v bv = *reinterpret_cast<const bf16x8_v *>(s_rows + c * PITCH + t * 64 + kq * 16);
                const bf16x8_v av = *reinterpret_cast<const bf16x8_v *>(s_rows + (16 + c) * PITCH + t * 64 + kq * 16);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
            }
            __syncthreads();
        }
    }
    MAD_TRACE_VAR(t_prod);
    MAD_TRACE_SET(t_prod);
    // lane l holds Y[row 4 (l / 16) + e][column l % 16], e < 4
    s_acc[wave][lane] = acc;
    __syncthreads();
    MAD_TRACE_VAR(t_acc);
    MAD_TRACE_SET(t_acc);
    MAD_TRACE_VAR(t_red);
    if (tid < 128) {
        const int r = tid >> 3, p = tid & 7, l0 = 16 * (r >> 2) + p, e = r & 3;
        // every read first, then a pairwise sum (no serial chain of reads)
        float v0[NW], v1[NW];
        #pragma unroll
        for (int wv = 0; wv < NW; ++wv) {
            v0[wv] = s_acc[wv][l0][e];
            v1[wv] = s_acc[wv][l0 + 8][e];
        }
        #pragma unroll
        for (int h = NW / 2; h > 0; h /= 2)
            #pragma unroll
            for (int wv = 0; wv < h; ++wv) {
                v0[wv] += v0[wv + h];
                v1[wv] += v1[wv + h];
            }
        float y0 = v0[0], y1 = v1[0];
        if (is_k) rope_apply(y0, y1, rc, rs, &y0, &y1);
        s_out[r][p] = f32_to_bf16(y0);
        s_out[r][p + 8] = f32_to_bf16(y1);
        MAD_TRACE_SET(t_red);
    }
    __syncthreads();
    MAD_TRACE_VAR(t_bar);
    MAD_TRACE_SET(t_bar);
    if (tid < 32 && s_row < R && s_fire) {
        const int h = tid & 1, i = s_row - s_b * n_new;
        bf16_t *dst = bits_ptr<bf16_t>(is_k ? mkb : mvb) + (size_t)(is_k ? hb : hb - Hkv) * m_head +
                      (size_t)s_b * m_seq + (size_t)(s_mlen + i) * d + h * hd + j0;
        *reinterpret_cast<uint4 *>(dst) = *reinterpret_cast<const uint4 *>(&s_out[tid >> 1][8 * h]);
    }
    // the marks are stored only now: a store earlier would be counted by the row loads' waits
    MAD_TRACE_SAVE_T0(mad_trace_update);
    MAD_TRACE_PUT(mad_trace_update, 1, t_rows);
    MAD_TRACE_PUT(mad_trace_update, 2, t_prod);
    MAD_TRACE_PUT(mad_trace_update, 4, t_acc);
    MAD_TRACE_PUT(mad_trace_update, 5, t_red);
    MAD_TRACE_PUT(mad_trace_update, 6, t_bar);
    MAD_TRACE(mad_trace_update, 3);
}

template <int RR, int NC, int KD>
__global__ __launch_bounds__(256) void update_gemv_kernel(const UpdateArgs a) {
    constexpr int NP = NC / 2;   // rotation pairs per workgroup
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int R = a.R, D = a.D, d = a.d, hd = d / 2;
    __shared__ float s_red[4][NC * RR];

    // thread t < NP * RR finishes pair t / RR of row t % RR: its kernel
    // arguments and RoPE angle are taken now, while the loads are in flight
    const int ep = tid / RR, er = tid % RR;
    const int eq = blockIdx.x * NP + ep, ehead = eq / hd, ejj = eq % hd;
    const bool e_is_k = ehead < a.Hkv;
    const int e_b = min(er, R - 1) / a.n_new;
    int e_fire = 0, e_mlen = 0;
    float rc = 1.f, rs = 0.f;
    if (tid < NP * RR) {
        e_fire = a.fire[e_b];
        e_mlen = a.mlen[e_b];
        if (e_is_k) rope_cs(a.pos[min(er, R - 1)], rope_theta(ejj, d, a.log2_base), &rc, &rs);
    }

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
    if (tid < NP * RR && er < R && e_fire) {
        const int p = ep, r = er, i = r - e_b * a.n_new;
        float y0 = 0.f, y1 = 0.f;
        #pragma unroll
        for (int wv = 0; wv < 4; ++wv) {
            y0 += s_red[wv][p * RR + r];
            y1 += s_red[wv][(p + NP) * RR + r];
        }
        if (e_is_k) rope_apply(y0, y1, rc, rs, &y0, &y1);
        bf16_t *dst = reinterpret_cast<bf16_t *>(e_is_k ? a.mk : a.mv) +
                      (size_t)(e_is_k ? ehead : ehead - a.Hkv) * a.m_head + (size_t)e_b * a.m_seq +
                      (size_t)(e_mlen + i) * d;
        dst[ejj].bits = f32_to_bf16(y0);
        dst[ejj + hd].bits = f32_to_bf16(y1);
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

template <int RR, int KD>
static hipError_t launch_gemv(const UpdateArgs &a, hipStream_t st) {
    constexpr int NC = 2;   // one rotation pair per workgroup (measured: 4.2 us for 4 rows, against 4.6 with two pairs, 5.8 with four)
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
        // sixteen waves: eight 1-KB row pieces of each in flight per round
        // (measured at 64 rows, D 2048, through registers: 5.6 us, against
        // 5.8 with eight waves and 7.4 for loads straight into the MFMA
        // layout; straight into LDS by column block: 5.3 us)
        const int RT = (a.R + 15) / 16;
        const dim3 grid((unsigned)(2 * a.Hkv * a.d / 16 * RT));
        if (a.D <= 2048)
            hipLaunchKernelGGL((update_rows_kernel<16, true>), grid, dim3(1024), 0, st, a);
        else
            hipLaunchKernelGGL((update_rows_kernel<16, false>), grid, dim3(1024), 0, st, a);
    } else {
        const int total = a.R * 2 * a.Hkv * (a.d / 2);
        dim3 grid((unsigned)((total + 255) / 256)), block(256);
        hipLaunchKernelGGL(update_f32_kernel, grid, block, 0, st, a);
    }
    return hipGetLastError();
}

}  // namespace mad
