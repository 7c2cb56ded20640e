// accept.hip -- greedy accept/reject (Sec. 2.1; greedy decoding, Sec. 4.1).
//
// For every sequence b: am[t] = argmax_v logits[b][t][v]; the drafted tokens
// are accepted up to the first t with draft[b][t] != am[t]; the target's
// token at that position (a correction, or the bonus token when everything
// was accepted) is emitted next.
//
// Argmax is made exact and independent of reduction order by mapping each
// (value, index) to one 64-bit key: an order-preserving 32-bit image of the
// float (NaN above +inf, -0 folded into +0) in the high word and the inverted
// index in the low word.  The row argmax is then the maximum key: ties go to
// the lowest index, the first NaN wins.
//
// One launch: workgroup (chunk, row) reduces a chunk of the vocabulary and
// folds its key into the row's key with a 64-bit atomic max; the last
// workgroup of a sequence (arrival counter over its T rows and all chunks)
// applies the accept rule to the sequence and clears the row keys for the
// next call.
//
// Stochastic accept/reject (the rejection-sampling rule the target applies,
// Sec. 2.1 and Sec. 3.3) with caller-supplied uniforms: drafted token x_i is
// accepted while u_i q_i(x_i) < p_i(x_i) (exact in double precision); the
// emitted token is the inverse-CDF draw with u_{T-1} from max(0, p_a - q_a)
// after the first rejection a, or from p_{T-1} when all were accepted.  One
// launch: workgroup (chunk, sequence) re-derives a from the T-1 drafted
// tokens, sums its vocabulary chunk of the draw's weights (and of p_a, the
// fallback when the residual is empty) in double precision; the last chunk of
// the sequence locates the chunk where the running sum passes u_{T-1} Z and
// scans it.
#include "mad_device.h"
#include "mad_internal.h"

namespace mad {

__device__ __forceinline__ uint64_t argmax_key(float x, int idx) {
    uint32_t u = __float_as_uint(x);
    uint32_t ord;
    if ((u & 0x7fffffffu) > 0x7f800000u) ord = 0xffffffffu;      // NaN: above everything
    else if ((u & 0x7fffffffu) == 0u) ord = 0x80000000u;         // +0 and -0 compare equal
    else ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((uint64_t)ord << 32) | (uint64_t)(0xffffffffu - (uint32_t)idx);
}
__device__ __forceinline__ int key_index(uint64_t k) { return (int)(0xffffffffu - (uint32_t)k); }

// Cross-lane exchanges of 64-bit values (two 32-bit halves) on the vector ALU,
// without an LDS round trip: DPP within rows of 16 lanes, then the gfx950
// lane swaps between rows.  dpp_u64<CTRL, ROWS>: the DPP move CTRL into the
// rows of ROWS; lanes without a source, and rows outside ROWS, read 0.
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, ROWS, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, ROWS, 0xF, false);
    return ((uint64_t)hi << 32) | lo;
}
// the values of lanes l & ~W and l | W (W = 16 or 32), in that order
template <int W>
__device__ __forceinline__ void lane_pair_u64(uint64_t v, uint64_t &a, uint64_t &b) {
    const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    if constexpr (W == 16) {
        const auto l = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
        const auto h = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
        a = ((uint64_t)h[0] << 32) | l[0];
        b = ((uint64_t)h[1] << 32) | l[1];
    } else {
        const auto l = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
        const auto h = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
        a = ((uint64_t)h[0] << 32) | l[0];
        b = ((uint64_t)h[1] << 32) | l[1];
    }
}
// f folded over the 64 lanes, the same value in every lane: pairs within a
// quad, then the two quads of 8 lanes (half mirror), the two 8s of a row
// (mirror), the two 16s of 32 lanes, the two 32s.  Every lane combines the same
// operands in the same order, so a floating-point sum is bitwise uniform.
template <typename F>
__device__ __forceinline__ uint64_t wave_fold_u64(uint64_t v, F f) {
    v = f(v, dpp_u64<0xB1>(v));    // quad_perm [1, 0, 3, 2]
    v = f(v, dpp_u64<0x4E>(v));    // quad_perm [2, 3, 0, 1]
    v = f(v, dpp_u64<0x141>(v));   // row_half_mirror
    v = f(v, dpp_u64<0x140>(v));   // row_mirror
    uint64_t a, b;
    lane_pair_u64<16>(v, a, b);
    v = f(a, b);
    lane_pair_u64<32>(v, a, b);
    return f(a, b);
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
    return wave_fold_u64(v, [](uint64_t x, uint64_t y) { return x > y ? x : y; });
}
__device__ __forceinline__ void store_agent_u64(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t load_agent_u64(const uint64_t *p) {
    return __hip_atomic_load(const_cast<uint64_t *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t max_agent_u64(uint64_t *p, uint64_t v) {
    return __hip_atomic_fetch_max(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename T>
__global__ __launch_bounds__(256) void accept_kernel(const AcceptArgs a) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rows = a.B * a.T;
    const int row = blockIdx.x % rows, chunk = blockIdx.x / rows;
    const int v0 = chunk * kAcceptChunk;
    const int v1 = min(a.V, v0 + kAcceptChunk);
    const T *x = reinterpret_cast<const T *>(a.logits) + (size_t)row * a.V;

    uint64_t best = 0;   // below every real key (index 0xffffffff is never used)
    constexpr int VEC = Elem<T>::VEC;                   // elements per 16-byte load
    constexpr int NV = kAcceptChunk / (256 * VEC);      // 16-byte loads per thread per chunk
    if (a.vec16) {
        // rows start on 16-byte boundaries and V is a multiple of VEC: every
        // load of the chunk is issued before any is used
        uint4 v[NV];
        #pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int e = v0 + (tid + 256 * k) * VEC;
            v[k] = e < v1 ? *reinterpret_cast<const uint4 *>(x + e) : make_uint4(0u, 0u, 0u, 0u);
        }
        #pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int e = v0 + (tid + 256 * k) * VEC;
            if (e < v1) {
                float f[VEC];
                unpack16(v[k], f, T());
                #pragma unroll
                for (int q = 0; q < VEC; ++q) {
                    const uint64_t key = argmax_key(f[q], e + q);
                    best = key > best ? key : best;
                }
            }
        }
    } else {
        for (int i = v0 + tid; i < v1; i += 256) {
            const uint64_t k = argmax_key(Elem<T>::load1(x + i), i);
            best = k > best ? k : best;
        }
    }
    best = wave_max_u64(best);
    __shared__ uint64_t s_w[4];
    __shared__ int s_flag;
    if (lane == 0) s_w[wave] = best;
    __syncthreads();
    if (tid == 0) {
        uint64_t m = s_w[0];
        for (int w = 1; w < 4; ++w) m = s_w[w] > m ? s_w[w] : m;
        // the maximum must have been performed at device scope before the
        // arrival is counted: the atomic's result is not used, so the compiler
        // may issue its no-return form; vmcnt(0) waits for it either way
        (void)max_agent_u64(a.row_best + row, m);
        wait_vm_stores();
        const int b = row / a.T;
        unsigned *cnt = a.counters + (size_t)b * kCounterStride;
        const int last = arrive(cnt) == (unsigned)(a.T * a.n_chunks - 1);
        if (last) reset_counter(cnt);
        s_flag = last;
    }
    __syncthreads();
    if (!s_flag) return;

    // ---- last workgroup of sequence b: the accept rule, then clear its row keys ----
    // thread t reads row t's key (all in one round trip); the first t < T-1
    // whose drafted token differs from the row's argmax is the rejection
    __shared__ int s_first;
    __shared__ uint64_t s_keys[kAcceptMaxT];
    const int b = row / a.T;
    uint64_t *rbp = a.row_best + (size_t)b * a.T;
    if (tid == 0) s_first = a.T - 1;
    __syncthreads();
    if (tid < a.T) {
        const uint64_t k = load_agent_u64(rbp + tid);
        s_keys[tid] = k;
        if (tid < a.T - 1 && a.draft[(size_t)b * (a.T - 1) + tid] != key_index(k)) atomicMin(&s_first, tid);
        store_agent_u64(rbp + tid, 0);   // the next call starts from zero keys
    }
    __syncthreads();
    if (tid == 0) {
        const int acc = s_first;
        a.n_accept[b] = acc;
        a.next_tok[b] = key_index(s_keys[acc]);
    }
}

// ------------------------------------------------------------------ host ----

// Only the counter region: line b holds sequence b's arrivals, and the row
// keys sit in the lines after line B-1.  That region is zero between calls
// (every kernel of the library leaves it so), which the atomic maxima need;
// the rest of a shared workspace holds other calls' partials.
size_t accept_ws_bytes(int B, int T, int V) {
    (void)B;
    (void)T;
    (void)V;
    return kCounterRegionBytes;
}

// ---------------------------------------------------------- stochastic ----

__device__ __forceinline__ uint64_t add_f64_bits(uint64_t x, uint64_t y) {
    return (uint64_t)__double_as_longlong(__longlong_as_double((long long)x) + __longlong_as_double((long long)y));
}
// inclusive prefix sum over the 64 lanes of a wave (lane order): shifts by 1,
// 2, 4, 8 within each row of 16, then row 0's total into row 1 and row 2's
// into row 3 (row_bcast:15), then rows 0-1's total into rows 2-3 (row_bcast:31)
__device__ __forceinline__ double wave_scan_f64(double v) {
    uint64_t u = (uint64_t)__double_as_longlong(v);
    u = add_f64_bits(u, dpp_u64<0x111>(u));
    u = add_f64_bits(u, dpp_u64<0x112>(u));
    u = add_f64_bits(u, dpp_u64<0x114>(u));
    u = add_f64_bits(u, dpp_u64<0x118>(u));
    u = add_f64_bits(u, dpp_u64<0x142, 0xA>(u));
    u = add_f64_bits(u, dpp_u64<0x143, 0xC>(u));
    return __longlong_as_double((long long)u);
}
__device__ __forceinline__ double read_lane_f64(double v, int l) {
    const uint64_t u = __double_as_longlong(v);
    const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)u, l);
    const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ double wave_sum_f64(double v) {
    return __longlong_as_double((long long)wave_fold_u64((uint64_t)__double_as_longlong(v), add_f64_bits));
}
// weight of entry v in the draw: max(0, p - q) (q given) or max(0, p)
__device__ __forceinline__ double draw_weight(float p, float q, bool resid) {
    const double r = resid ? (double)p - (double)q : (double)p;
    return r > 0.0 ? r : 0.0;
}

// VEC16: every row starts 16-byte aligned and V is a multiple of 4, so the
// rows are read as float4; the element-wise form is its own instantiation so
// that the aligned kernel carries none of its code
template <bool VEC16>
__global__ __launch_bounds__(256) void stoch_kernel(const StochArgs a) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int b = blockIdx.x % a.B, chunk = blockIdx.x / a.B;
    const int T = a.T, V = a.V;
    __shared__ int s_a;
    __shared__ double s_w[2][4];
    __shared__ int s_flag;
    // ---- the first rejection a (every workgroup of the sequence derives it) ----
    if (wave == 0) {
        bool rej = false;
        if (lane < T - 1) {
            const int x = a.draft[(size_t)b * (T - 1) + lane];
            if (x < 0 || x >= V) {
                rej = true;   // not a token
            } else {
                const double px = a.p[((size_t)b * T + lane) * V + x];
                const double qx = a.q[((size_t)b * (T - 1) + lane) * V + x];
                rej = !((double)a.u[(size_t)b * T + lane] * qx < px);
            }
        }
        const unsigned long long m = __ballot(rej);
        if (lane == 0) s_a = m ? __ffsll((long long)m) - 1 : T - 1;
    }
    __syncthreads();
    const int acc = s_a;
    const bool resid = acc < T - 1;
    const float *pr = a.p + ((size_t)b * T + acc) * V;
    const float *qr = resid ? a.q + ((size_t)b * (T - 1) + acc) * V : pr;

    // ---- this chunk's sums of the draw weights and of p_a ----
    const int v0 = chunk * kAcceptChunk, v1 = min(V, v0 + kAcceptChunk);
    double sr = 0.0, sp = 0.0;
    if constexpr (VEC16) {
        // every load unconditional (a piece past the chunk reads its last
        // piece again and is skipped below; q reads the p row when unused), so
        // no branch -- and no wait the compiler places inside one -- splits
        // them: all 2 NV loads are in flight together
        constexpr int NV = kAcceptChunk / (256 * 4);
        float4 pv[NV], qv[NV];
        #pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int e = min(v0 + (tid + 256 * k) * 4, v1 - 4);
            pv[k] = *reinterpret_cast<const float4 *>(pr + e);
            qv[k] = *reinterpret_cast<const float4 *>(qr + e);
        }
        #pragma unroll
        for (int k = 0; k < NV; ++k) {
            if (v0 + (tid + 256 * k) * 4 >= v1) continue;
            sr += draw_weight(pv[k].x, qv[k].x, resid) + draw_weight(pv[k].y, qv[k].y, resid) +
                  draw_weight(pv[k].z, qv[k].z, resid) + draw_weight(pv[k].w, qv[k].w, resid);
            sp += draw_weight(pv[k].x, 0.f, false) + draw_weight(pv[k].y, 0.f, false) +
                  draw_weight(pv[k].z, 0.f, false) + draw_weight(pv[k].w, 0.f, false);
        }
    } else {
        // element by element, the loads again unconditional (an index past
        // the chunk reads its last entry, skipped in the sums)
        constexpr int NE = kAcceptChunk / 256;
        float pv[NE], qv[NE];
        #pragma unroll
        for (int k = 0; k < NE; ++k) {
            const int v = min(v0 + tid + 256 * k, v1 - 1);
            pv[k] = pr[v];
            qv[k] = qr[v];
        }
        #pragma unroll
        for (int k = 0; k < NE; ++k) {
            if (v0 + tid + 256 * k >= v1) continue;
            sr += draw_weight(pv[k], qv[k], resid);
            sp += draw_weight(pv[k], 0.f, false);
        }
    }
    sr = wave_sum_f64(sr);
    sp = wave_sum_f64(sp);
    if (lane == 0) { s_w[0][wave] = sr; s_w[1][wave] = sp; }
    __syncthreads();
    double *sums = a.sums + (size_t)b * a.n_chunks * 2;
    if (tid == 0) {
        const double cr = s_w[0][0] + s_w[0][1] + s_w[0][2] + s_w[0][3];
        const double cp = s_w[1][0] + s_w[1][1] + s_w[1][2] + s_w[1][3];
        __hip_atomic_store(reinterpret_cast<uint64_t *>(sums + 2 * chunk), (uint64_t)__double_as_longlong(cr),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(reinterpret_cast<uint64_t *>(sums + 2 * chunk + 1), (uint64_t)__double_as_longlong(cp),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    wait_vm_stores();
    __syncthreads();
    if (tid == 0) {
        unsigned *cnt = a.counters + (size_t)b * kCounterStride;
        const int last = arrive(cnt) == (unsigned)(a.n_chunks - 1);
        if (last) reset_counter(cnt);
        s_flag = last;
    }
    __syncthreads();
    if (!s_flag) return;

    // ---- last chunk of the sequence: locate the chunk, then the token ----
    // (1) one wave reads the chunk sums (64 per pass), totals them and finds,
    // by a prefix sum over chunks, the first chunk of positive weight whose
    // running sum passes the target u * Z
    __shared__ int s_c, s_mode, s_fb;
    __shared__ double s_t;
    if (wave == 0) {
        const int nc = a.n_chunks;
        auto chunk_sum = [&](int c, int which) -> double {
            return __longlong_as_double(
                (long long)load_agent_u64(reinterpret_cast<const uint64_t *>(sums + 2 * c + which)));
        };
        double zr = 0.0, zp = 0.0;
        for (int c0 = 0; c0 < nc; c0 += 64)
            if (c0 + lane < nc) {
                zr += chunk_sum(c0 + lane, 0);
                zp += chunk_sum(c0 + lane, 1);
            }
        const double Zr = wave_sum_f64(zr), Zp = wave_sum_f64(zp);
        const int use_p = Zr == 0.0;   // empty residual: the draw uses p_a
        const double t = (double)a.u[(size_t)b * T + T - 1] * (use_p ? Zp : Zr);
        double carry = 0.0, before = 0.0;
        int cs = -1, clast = -1;
        for (int c0 = 0; c0 < nc; c0 += 64) {
            const double w = c0 + lane < nc ? chunk_sum(c0 + lane, use_p) : 0.0;
            const double incl = wave_scan_f64(w);
            const unsigned long long pos = __ballot(w > 0.0);
            const unsigned long long hit = __ballot(w > 0.0 && carry + incl > t);
            if (pos) clast = c0 + 63 - __clzll((long long)pos);
            if (hit) {
                const int l = __ffsll((long long)hit) - 1;
                cs = c0 + l;
                before = carry + read_lane_f64(incl, l) - read_lane_f64(w, l);
                break;
            }
            carry += read_lane_f64(incl, 63);
        }
        if (lane == 0) {
            const int fb = cs < 0;   // no chunk passes t: the last positive entry is drawn
            s_c = fb ? (clast >= 0 ? clast : 0) : cs;
            s_mode = use_p;
            s_fb = fb;
            s_t = fb ? 0.0 : t - before;   // target measured from the chunk's start
        }
    }
    __syncthreads();
    const int cs = s_c;
    const bool wres = resid && !s_mode;
    // (2) runs of RUN consecutive entries of the chunk, one per thread, kept in
    // registers; a block prefix sum over the runs finds the run where the
    // running sum passes the target, and that thread walks its run in order
    constexpr int RUN = kAcceptChunk / 256;
    const int cbeg = cs * kAcceptChunk, cend = min(V, cbeg + kAcceptChunk);
    const int r0 = cbeg + tid * RUN;
    double w[RUN];
    double mine = 0.0;
    int lastpos = -1;
    if constexpr (VEC16) {
        // runs start on multiples of RUN and V is a multiple of 4, so a float4
        // piece lies wholly inside the chunk or wholly past it: a piece past
        // it reads the chunk's last piece and gets weight 0 (a product, not a
        // branch, so the loads stay together)
        #pragma unroll
        for (int k = 0; k < RUN / 4; ++k) {
            const int e = min(r0 + 4 * k, cend - 4);
            const double in = (double)(r0 + 4 * k < cend);
            // q read unconditionally (the p row when the draw does not use it)
            const float4 pv = *reinterpret_cast<const float4 *>(pr + e);
            const float4 qv = *reinterpret_cast<const float4 *>(qr + e);
            w[4 * k + 0] = draw_weight(pv.x, qv.x, wres) * in;
            w[4 * k + 1] = draw_weight(pv.y, qv.y, wres) * in;
            w[4 * k + 2] = draw_weight(pv.z, qv.z, wres) * in;
            w[4 * k + 3] = draw_weight(pv.w, qv.w, wres) * in;
        }
    } else {
        #pragma unroll
        for (int i = 0; i < RUN; ++i) {   // unconditional loads (past the chunk: its last entry, weight 0)
            const int v = min(r0 + i, cend - 1);
            const float pv = pr[v], qv = qr[v];
            // masked by a product, not a branch (a branch would take the loads into it)
            w[i] = draw_weight(pv, qv, wres) * (double)(r0 + i < cend);
        }
    }
    #pragma unroll
    for (int i = 0; i < RUN; ++i) {
        mine += w[i];
        if (w[i] > 0.0) lastpos = r0 + i;
    }
    __shared__ double s_wt[4];
    __shared__ int s_first[4], s_last[4];
    const double incl = wave_scan_f64(mine);
    if (lane == 63) s_wt[wave] = incl;
    __syncthreads();
    double excl = incl - mine;
    for (int k = 0; k < wave; ++k) excl += s_wt[k];
    const double tt = s_t;
    const bool hit = !s_fb && mine > 0.0 && excl + mine > tt;
    const unsigned long long hm = __ballot(hit);
    const int lp = (int)wave_max_u64((uint64_t)(lastpos + 1)) - 1;   // lastpos >= -1
    if (lane == 0) {
        s_first[wave] = hm ? wave * 64 + __ffsll((long long)hm) - 1 : 0x7fffffff;
        s_last[wave] = lp;
    }
    __syncthreads();
    const int first = min(min(s_first[0], s_first[1]), min(s_first[2], s_first[3]));
    if (first == 0x7fffffff) {   // fallback: the chunk's last positive entry
        if (tid == 0) {
            const int la = max(max(s_last[0], s_last[1]), max(s_last[2], s_last[3]));
            a.n_accept[b] = acc;
            a.next_tok[b] = la >= 0 ? la : cbeg;
        }
    } else if (tid == first) {
        int v_out = lastpos;   // if rounding keeps the target above the run's own sum
        double e = excl;
        #pragma unroll
        for (int i = 0; i < RUN; ++i) {
            if (w[i] > 0.0) {
                e += w[i];
                if (e > tt) {
                    v_out = r0 + i;
                    break;
                }
            }
        }
        a.n_accept[b] = acc;
        a.next_tok[b] = v_out;
    }
}

size_t stoch_ws_bytes(int B, int V) {
    const size_t chunks = ((size_t)V + kAcceptChunk - 1) / kAcceptChunk;
    return kCounterRegionBytes + align256((size_t)B * chunks * 16);
}

hipError_t launch_stoch(const StochArgs &a, hipStream_t st) {
    if (a.vec16)
        hipLaunchKernelGGL(stoch_kernel<true>, dim3((unsigned)(a.B * a.n_chunks)), dim3(256), 0, st, a);
    else
        hipLaunchKernelGGL(stoch_kernel<false>, dim3((unsigned)(a.B * a.n_chunks)), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_accept(const AcceptArgs &a, int dtype, hipStream_t st) {
    dim3 grid((unsigned)(a.B * a.T * a.n_chunks)), block(256);
    if (dtype == MAD_BF16) hipLaunchKernelGGL(accept_kernel<bf16_t>, grid, block, 0, st, a);
    else hipLaunchKernelGGL(accept_kernel<float>, grid, block, 0, st, a);
    return hipGetLastError();
}

}  // namespace mad
