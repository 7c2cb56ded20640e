/*
 * mad.h -- C ABI of libmad: the data-parallel hot path of memory-augmented
 * sliding-window (MASW) drafting for long-context speculative decoding, on
 * AMD Instinct MI355X (gfx950).
 *
 * What the library computes (paper: "Strong Drafts Need Compact Memories"):
 *   - the draft model's per-step decode attention over its compact memory
 *     (sink + memory slots, then the exact local window)          Sec. 3.1
 *   - the memory adaptor's update: mirrored K/V projection of new slot
 *     hidden states, RoPE at the slot's position id, append-only write Sec. 3.2
 *   - the target's (gamma+1)-query verify attention over its full KV  Sec. 2.1, 3.3
 *   - the greedy and the stochastic accept/reject rules              Sec. 2.1, 4.1
 *   - the draft's memory-prefill attention                          Sec. 3.3, App.
 *   - the linear maps of a draft decoder layer around the attention  Sec. 2.3, 3.2
 *
 * Conventions shared by every entry point
 *   - Tensors are DEVICE memory owned by the caller, row-major; a key/value row
 *     (head_dim elements) is contiguous.  Per-sequence lengths, starts,
 *     positions and fire flags are HOST arrays, copied into kernel arguments,
 *     so every argument is validated synchronously before anything is
 *     enqueued; on an error nothing is launched and no buffer is touched.
 *   - dtype: MAD_F32 or MAD_BF16 (inputs and outputs share it; arithmetic
 *     accumulates in fp32; lse outputs are always fp32).
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls enqueue
 *     work and return; nothing synchronises the host.
 *   - Workspace `ws`: device scratch of at least mad_workspace_bytes(...)
 *     bytes.  It holds split partial results and arrival counters.  It must be
 *     zero-filled once before its first use; every call leaves the counters at
 *     zero again when its kernels finish.  Calls that share a workspace must
 *     be ordered (same stream); concurrent calls on one workspace race.
 *   - The library allocates no device memory and keeps no state besides a
 *     thread-local error string.  No C++ exception crosses the ABI.
 *   - Return value: MAD_OK or a negative MAD_E* code; mad_last_error() then
 *     describes the failure.
 *   - Limits: B <= MAD_MAX_BATCH; head_dim in {64, 128}; 1 <= Hq/Hkv <= 16.
 */
#ifndef MAD_H
#define MAD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MAD_OK 0
#define MAD_EINVAL (-1)  /* bad pointer, shape, length, capacity or workspace argument */
#define MAD_ENOTSUP (-2) /* valid but unsupported: head_dim, group size, dtype */
#define MAD_EHIP (-3)    /* a HIP launch failed; the message carries hipGetErrorString */
#define MAD_EWS (-4)     /* workspace smaller than mad_workspace_bytes() asks */

#define MAD_F32 0
#define MAD_BF16 1

#define MAD_MAX_BATCH 64
#define MAD_MAX_UPDATE_ROWS 64 /* B * n_new per mad_memory_update call */
#define MAD_MAX_VERIFY_ROWS 64 /* T * (Hq / Hkv) per mad_verify_attn call */
#define MAD_MAX_LAYER_ROWS 8   /* rows (raw token + slot tokens) per draft-layer linear map */

#define MAD_OP_DECODE 0
#define MAD_OP_UPDATE 1 /* takes no workspace: 0 bytes */
#define MAD_OP_VERIFY 2
#define MAD_OP_ACCEPT 3
#define MAD_OP_ACCEPT_STOCH 4

/*
 * A per-sequence, per-KV-head run of key/value rows in device memory.
 * Row i of sequence b, KV head h lives at
 *     k + b * seq_stride + h * head_stride + i * head_dim   (elements of dtype)
 * and likewise for v.  seq_stride may be 0 (every sequence index aliases the
 * same buffer, e.g. several queries of one sequence with different visible
 * ranges); head_stride >= cap * head_dim.
 *   cap    rows available per (sequence, head)
 *   start  HOST int32[B], ring start of each sequence (NULL = all 0); used by
 *          the local window only, must satisfy 0 <= start < cap
 *   len    HOST int32[B], number of valid rows, 0 <= len <= cap
 */
typedef struct mad_kv_view {
    void *k;
    void *v;
    int64_t seq_stride;
    int64_t head_stride;
    int32_t cap;
    const int32_t *start;
    const int32_t *len;
} mad_kv_view;

/*
 * Draft decode attention over the compact memory (Sec. 3.1: the working
 * memory M_t = M_sink u M_local,t u M_slot,t; the draft reads only this
 * compact memory, Sec. 3.3).  For each sequence b and query head h, with
 * G = Hq / Hkv and KV head c = h / G (consecutive query heads share a KV head):
 *
 *   keys  = mem rows [0, mem.len[b])                       (sinks, then slots)
 *         ++ window rows i = 0 .. win.len[b]-1 at ring row (win.start[b] + i) % win.cap
 *         ++ the new token (k_new, v_new) when k_new != NULL
 *   out[b][h] = sum_j softmax_j(scale * q[b][h] . K_j) V_j,
 *   lse[b][h] = log sum_j exp(scale * q[b][h] . K_j)        (natural log)
 *
 * When k_new/v_new are given ([B][Hkv][d], dtype) the new token's K/V are
 * also written into the window ring at row (start + len) % cap -- the append
 * of the current token into the local window in the same pass (Sec. 3.2);
 * this requires win.len[b] + 1 <= win.cap.  Eviction is the caller's
 * bookkeeping: advancing win.start / shrinking win.len; evicted rows stay in
 * the ring until overwritten, which is what the raw-KV rollback window keeps.
 *   q    device [B][Hq][d], dtype          out  device [B][Hq][d], dtype
 *   lse  device fp32 [B][Hq] or NULL
 *   mem  linear view (start ignored) or NULL = empty; win  ring view or NULL
 * A sequence with no keys at all gets out = 0 and lse = -inf.
 * The full-KV draft (the uncompressed comparison) is the same call with an
 * empty mem and the whole prefix in the window.
 * Supports dtype F32 and BF16, d in {64, 128}, G in {1, 2, 4, 8, 16}.
 */
int mad_draft_decode_attn(const void *q, int B, int Hq, int Hkv, int d, int dtype, float scale,
                          const mad_kv_view *mem, const mad_kv_view *win,
                          const void *k_new, const void *v_new,
                          void *out, float *lse,
                          void *ws, size_t ws_bytes, void *stream);

/*
 * The draft decode attention of mad_draft_decode_attn without a workspace and
 * without any allocation, for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Arguments, results, layouts and errors are those of
 * mad_draft_decode_attn (the same kernels run); the split partials and
 * arrival counters live in a library-owned device array of
 * MAD_NOALLOC_SCRATCH_BYTES per GPU, held until the process ends.
 *   - The first call on a device looks up the array's address and clears its
 *     counter region with a small kernel on `stream`; every call leaves the
 *     counters at zero again.
 *   - Calls whose workspace need, mad_workspace_bytes(MAD_OP_DECODE, B, Hq,
 *     Hkv, d, ...), exceeds MAD_NOALLOC_SCRATCH_BYTES return MAD_EINVAL before
 *     anything is launched (16 MiB holds B * Hkv up to 240 units at d 64 and
 *     G 4; the 16-sequence, 8-KV-head launch needs 9 MiB).
 *   - Every call on one GPU shares its array: calls ordered on one stream are
 *     safe; calls that overlap in time on one GPU (other streams, threads)
 *     race and must not be issued.
 *   - Errors: as mad_draft_decode_attn, plus MAD_EHIP if the array's address
 *     cannot be obtained on the current device.
 */
#define MAD_NOALLOC_SCRATCH_BYTES (16u << 20)
int mad_draft_decode_attn_noalloc(const void *q, int B, int Hq, int Hkv, int d, int dtype, float scale,
                                  const mad_kv_view *mem, const mad_kv_view *win,
                                  const void *k_new, const void *v_new,
                                  void *out, float *lse, void *stream);

/*
 * The same attention with a per-row choice for the new token, so that one
 * launch serves the raw query of a step and the write-scope queries of the
 * memory slots materialised in that step (Sec. 3.2: a slot is an extra
 * position of the pass; its write scope is the sinks, the slots up to it and
 * the W raw tokens before its position id, which for the newest slot end at
 * the current token).
 *   new_mode  host uint8 [B]: 0 = the row has no new token; 1 = the row's key
 *             sequence ends with k_new/v_new[b] (not written anywhere);
 *             2 = as 1, and the token is appended to the row's window ring at
 *             (start + len) % cap, as mad_draft_decode_attn does.
 * Rows may alias one sequence's buffers (seq_stride 0); at most one row of a
 * shared ring may append, and no row's window may include the ring row being
 * appended (the window of a mode-1 row stops before the current token, which
 * it reads from k_new/v_new instead).  k_new/v_new are required when any row
 * has mode 1 or 2.  Everything else (layouts, workspace, errors) is as for
 * mad_draft_decode_attn.
 */
int mad_draft_step_attn(const void *q, int B, int Hq, int Hkv, int d, int dtype, float scale,
                        const mad_kv_view *mem, const mad_kv_view *win, const void *k_new, const void *v_new,
                        const uint8_t *new_mode, void *out, float *lse, void *ws, size_t ws_bytes, void *stream);

/*
 * Memory update by the memory adaptor (Sec. 3.2, projection and KV
 * materialisation): for every firing sequence b and slot i < n_new,
 *   [k~ | v] = x[b][i] . [W_K,g ; W_V,g]^T          (mirrored projections)
 *   k        = RoPE(k~, pos[b][i])                   (rotate-half pairs (j, j+d/2),
 *              angle pos * base^(-2j/d), computed in fp64)
 * and the pair is appended at mem row mem.len[b] + i (append-only: rows below
 * mem.len[b] are never written).  The caller then raises mem.len[b] by n_new.
 *   x      device [B][n_new][D], dtype (slot hidden states entering the layer)
 *   w_kv   device [2*Hkv*d][D], dtype: the Hkv*d rows of W_K,g then the Hkv*d
 *          rows of W_V,g (one row per output feature, nn.Linear layout)
 *   pos    HOST int32[B][n_new] position ids (a slot shares the id of the raw
 *          token after it)
 *   fire   HOST uint8[B] or NULL (= all fire); fire[b] == 0 leaves sequence b
 *          untouched (the per-sequence mask of heterogeneous batches, Sec. 4.1)
 *   mem    linear view to append to; requires mem.len[b] + n_new <= mem.cap
 * B * n_new <= MAD_MAX_UPDATE_ROWS; D a multiple of 64; d in {64, 128}.
 * BF16 runs the projection as a weight stream (at most 8 rows) or on the
 * matrix cores; F32 on the vector ALUs.  No workspace: every output element is
 * produced by one workgroup.
 * Errors: MAD_EINVAL (null pointers, B, n_new, D, Hkv, rope_base <= 1 or not
 * finite, a firing sequence's len + n_new above cap), MAD_ENOTSUP (d, dtype).
 */
int mad_memory_update(const void *x, const void *w_kv, const int32_t *pos, const uint8_t *fire,
                      int B, int n_new, int D, int Hkv, int d, int dtype, double rope_base,
                      const mad_kv_view *mem, void *stream);

/*
 * Target verify attention (Sec. 2.1: the target scores the drafted block in
 * one parallel pass; Sec. 3.3: over its full KV cache, which the compact draft
 * memory leaves unchanged).  The T = gamma+1 new tokens' K/V are already
 * stored at rows len[b]-T .. len[b]-1; query t sees rows 0 .. len[b]-T+t (the
 * prefix and new tokens 0..t).
 *   q    device [B][T][Hq][d], dtype     out  device [B][T][Hq][d], dtype
 *   lse  device fp32 [B][T][Hq] or NULL
 *   kv   the verifier's cache as it is: a linear mad_kv_view (start NULL),
 *        K and V rows of d elements, kv->len[b] in [T, cap]
 * T * G <= MAD_MAX_VERIFY_ROWS; d in {64, 128}.  dtype BF16: both products on
 * the matrix cores.  dtype F32: on the vector ALUs, one decode-attention launch
 * per sequence (its T queries as the rows, query t over rows 0 .. len-T+t),
 * all on `stream` with the same workspace.  Workspace MAD_OP_VERIFY (sized for
 * both).
 */
int mad_verify_attn(const void *q, int B, int T, int Hq, int Hkv, int d, int dtype, float scale,
                    const mad_kv_view *kv, void *out, float *lse, void *ws, size_t ws_bytes, void *stream);

/*
 * The same verify attention for a verifier that keeps its V cache transposed,
 * one run of cap keys per feature (key-contiguous), so that the A operand of
 * the PV product (8 consecutive keys of one feature) is one 16-byte load:
 *   k   device keys, rows of d:      k  + b*seq_stride + h*head_stride + i*d
 *   vt  device values TRANSPOSED:    vt + b*seq_stride + h*head_stride + c*cap + i
 *   len HOST int32[B], T <= len[b] <= cap; cap a multiple of 8
 * dtype BF16 only (MAD_ENOTSUP otherwise).  Everything else as mad_verify_attn.
 */
int mad_verify_attn_vt(const void *q, int B, int T, int Hq, int Hkv, int d, int dtype, float scale,
                       const void *k, const void *vt, int64_t seq_stride, int64_t head_stride,
                       int32_t cap, const int32_t *len,
                       void *out, float *lse, void *ws, size_t ws_bytes, void *stream);

/*
 * Greedy accept/reject (Sec. 2.1; greedy decoding at temperature 0, Sec. 4.1).
 * For each sequence b, with am[t] = argmax_v logits[b][t][v] (ties -> lowest
 * index, a NaN ranks above every number):
 *   n_accept[b] = first t < T-1 with draft_tok[b][t] != am[t], else T-1
 *   next_tok[b] = am[n_accept[b]]   (the correction, or the bonus token)
 * The iteration emits n_accept[b] + 1 tokens.
 *   logits    device [B][T][V], dtype F32 or BF16
 *   draft_tok device int32 [B][T-1] (may be NULL when T == 1)
 *   n_accept, next_tok  device int32 [B]
 * V >= 1, 1 <= T <= 256.
 */
int mad_accept_greedy(const void *logits, int dtype, const int32_t *draft_tok,
                      int B, int T, int V, int32_t *n_accept, int32_t *next_tok,
                      void *ws, size_t ws_bytes, void *stream);

/*
 * Stochastic accept/reject: the rejection-sampling rule of speculative
 * decoding, which the target applies unchanged (Sec. 2.1, Sec. 3.3), with
 * uniforms supplied by the caller (so a host and the device can share one
 * random stream).  For each sequence b, in double precision:
 *   n_accept[b] = a = first i < T-1 with NOT (u[b][i] q_i(x_i) < p_i(x_i)),
 *                 x_i = draft_tok[b][i] (a value outside [0, V) is rejected),
 *                 else T-1;
 *   next_tok[b] = the inverse-CDF draw with u[b][T-1] from the weights
 *                 max(0, p_a - q_a) when a < T-1 (the correction), or
 *                 max(0, p_{T-1}) when all drafts were accepted (the bonus
 *                 token): the smallest v whose running weight sum exceeds
 *                 u[b][T-1] * Z, Z the total weight.  An empty residual
 *                 (Z = 0) draws from p_a; if no index qualifies, the last
 *                 index of positive weight is returned.
 * The running sums are formed in a different order than a sequential scan,
 * so a draw can differ from one only when u[b][T-1] * Z lies within rounding
 * of a bin edge.
 *   p         device float32 [B][T][V] target probabilities
 *   q         device float32 [B][T-1][V] draft probabilities (NULL when T == 1)
 *   draft_tok device int32 [B][T-1] (NULL when T == 1)
 *   u         device float32 [B][T] uniforms in [0, 1)
 *   n_accept, next_tok  device int32 [B]
 * The workspace (MAD_OP_ACCEPT_STOCH) holds per-chunk sums and arrival
 * counters; it follows the same rules as the other workspaces.
 */
int mad_accept_stochastic(const float *p, const float *q, const int32_t *draft_tok, const float *u, int B, int T,
                          int V, int32_t *n_accept, int32_t *next_tok, void *ws, size_t ws_bytes, void *stream);

/*
 * Memory-prefill attention (Sec. 3.3, prefill; the appendix on memory
 * prefill): the draft's single masked pass over a prefix, which builds its
 * initial compact memory.  The mask applies the write policy of decoding, so
 * every query of the pass attends exactly what it would attend while
 * decoding.  With s(t) = u * floor((t - S) / (u r)) for t > S, else 0 (the
 * slots materialised once raw tokens 0..t-1 are processed; u = slots per
 * update, 1 = one slot per boundary), for sequence b and KV head c = h / G:
 *   raw token p < P[b]:  keys = sinks [0, min(S, p+1)), slots 1..s(p) and the
 *                        raw tokens [max(S, p-W+1), p];
 *   slot m <= M[b]:      keys = sinks [0, S), slots 1..m (itself included) and
 *                        the raw tokens [max(S, b_m - W), b_m - 1], b_m = S + m r
 *                        (its write scope);
 * where M[b] = s(P[b]) is the number of slots the prefix materialises.  Sinks
 * are read from mem rows 0..S-1, slot m from mem row S + m - 1, raw token x
 * from raw row x.  Outputs and lse are as for mad_draft_decode_attn.
 *   q_raw     device [B][q_cap][Hq][d]: row p of sequence b for p < P[b]
 *   out_raw   device [B][q_cap][Hq][d]; lse_raw device fp32 [B][q_cap][Hq] or NULL
 *   q_slot    device [B][slot_cap][Hq][d], row m-1 for slot m; NULL = no slot
 *             queries (out_slot and lse_slot are then ignored)
 *   out_slot  device [B][slot_cap][Hq][d]; lse_slot fp32 [B][slot_cap][Hq] or NULL
 *   P         HOST int32[B], 0 <= P[b] <= q_cap
 *   mem       linear view (start ignored): len[b] >= S + M[b] (>= P[b] when
 *             P[b] <= S)
 *   raw       linear view of the prefix's raw K/V (start must be NULL):
 *             len[b] >= P[b]
 *   S >= 0 sinks, W >= 1 window, r >= 1 slot interval, u >= 1 slots per update
 * dtype BF16 only (the products run on the matrix cores), d in {64, 128},
 * G in {1, 2, 4, 8}.  No workspace.  A slot count M[b] > slot_cap (with slot
 * queries) is MAD_EINVAL.
 */
int mad_memory_prefill_attn(const void *q_raw, const void *q_slot, int B, int Hq, int Hkv, int d, int dtype,
                            float scale, const int32_t *P, int q_cap, int slot_cap, int S, int W, int r, int u,
                            const mad_kv_view *mem, const mad_kv_view *raw, void *out_raw, float *lse_raw,
                            void *out_slot, float *lse_slot, void *stream);

/*
 * The linear maps of a draft decoder layer around its attention.  A decode
 * step runs, per layer, for R rows: the raw token and, in a materialisation
 * pass, the memory-slot tokens, which go through the same transformer blocks
 * and whose hidden states leaving layer l enter layer l+1 (Sec. 3.2); these
 * maps stream the layer's weights, the alpha d^2 term of the draft's cost
 * (Sec. 2.3, Eq. latency_decomp).  A pre-norm (RMSNorm) layer with a SwiGLU
 * MLP, the Llama family the paper uses (Sec. 4.1):
 *   xn  = rmsnorm(x) * gamma1        (fp32, rounded to bf16)
 *   q, k, v = xn W_qkv^T; q and k rotated at pos[r] (rotate-half RoPE, base)
 *   o   = attention(q, ...)          (mad_draft_decode_attn / _step_attn)
 *   h   = x + o W_o^T
 *   a   = silu(hn W_gate^T) * (hn W_up^T),  hn = rmsnorm(h) * gamma2
 *   y   = h + a W_down^T
 * Every tensor is BF16, row-major; weights in nn.Linear layout [out][in];
 * products accumulate in fp32.  R <= MAD_MAX_LAYER_ROWS.
 *
 * mad_rmsnorm_qkv_rope: x [R][D]; gamma [D]; w_qkv [(Hq + 2 Hkv) d][D] (the
 *   rows of W_q, then W_k, then W_v); pos HOST int32[R] position ids;
 *   outputs q [R][Hq][d], k and v [R][Hkv][d]; xn [R][D] or NULL receives the
 *   normalised rows (the input of the memory adaptor for slot rows).  With
 *   kv_from_row0 != 0 every row's k and v are row 0's (the current token's,
 *   which the rows of a fused step attend).  D in {2048, 4096}; d in {64, 128}.
 * mad_linear_residual: out [R][N] = res + x W^T, x [R][D], w [N][D],
 *   res [R][N]; D in {2048, 4096, 8192}; N a multiple of 4.
 *   out may be res; it must not overlap x.
 * mad_rmsnorm_swiglu: out [R][F] = silu(xn W_gate^T) * (xn W_up^T),
 *   xn = rmsnorm(x) * gamma, w_gate_up [2F][D] (W_gate rows, then W_up);
 *   D in {2048, 4096}; F a multiple of 4.
 * Errors: MAD_EINVAL (null or unaligned pointers, R, sizes), MAD_ENOTSUP
 * (dtype is implied BF16; D or d outside the sets above).  No workspace.
 */
int mad_rmsnorm_qkv_rope(const void *x, const void *gamma, float eps, const void *w_qkv, const int32_t *pos, int R,
                         int D, int Hq, int Hkv, int d, double rope_base, int kv_from_row0, void *q, void *k,
                         void *v, void *xn, void *stream);
int mad_linear_residual(const void *x, const void *w, const void *res, int R, int D, int N, void *out, void *stream);
int mad_rmsnorm_swiglu(const void *x, const void *gamma, float eps, const void *w_gate_up, int R, int D, int F,
                       void *out, void *stream);

/*
 * Measurement aids (not part of the attention path), used by the benchmark to
 * put the kernels' times next to what the device itself delivers:
 * mad_probe_stream_read: reads `bytes` (a multiple of 16; src 16-byte
 *   aligned) with n_workgroups x 256 threads, each workgroup a contiguous
 *   range, 8 nontemporal 16-byte loads in flight per thread; the HBM read
 *   bandwidth a plain streaming kernel reaches.  sink: device unsigned, written only if an xor of the data
 *   hits one particular value (keeps the loads), may be NULL.
 * mad_probe_shared_read: every one of n_workgroups workgroups of `threads`
 *   threads (a multiple of 64, at most 1024) reads the same `bytes` (a
 *   multiple of 16; src 16-byte aligned), 16 loads of 16 bytes in flight per
 *   thread; after the first touch the data is L2-resident, so the launch time
 *   gives the rate at which one CU reads from L2.  sink as above.
 * mad_probe_empty: an empty kernel of n_workgroups x threads (the launch floor).
 * mad_probe_handoff_latency: one thread times, in shader-clock cycles, `reps`
 *   repetitions (reps >= 2) of: row 0 a plain store until acknowledged; 1 a
 *   device-scope store until acknowledged; 2 a device-scope atomic add (value
 *   returned); 3 a device-scope load of the word row 1 stored; 4 a plain load
 *   of the word row 0 stored; 5 a plain load of an untouched line; rows 6 and 7
 *   the 100 MHz real-time counter and the shader clock at the end of each
 *   repetition (their ratio gives the clock rate).  buf: device, at least
 *   reps * 256 + 256 bytes, fresh lines; cycles: device uint64 [8][reps].
 * Errors: MAD_EINVAL for bad arguments, MAD_EHIP for a failed launch.
 */
int mad_probe_stream_read(const void *src, size_t bytes, unsigned *sink, int n_workgroups, void *stream);
int mad_probe_shared_read(const void *src, size_t bytes, unsigned *sink, int n_workgroups, int threads,
                          void *stream);
int mad_probe_empty(int n_workgroups, int threads, void *stream);
int mad_probe_handoff_latency(void *buf, size_t buf_bytes, unsigned long long *cycles, int reps, void *stream);

/*
 * Workspace bytes needed by op (MAD_OP_*) for calls with at most these sizes:
 *   DECODE: B, Hq, Hkv, d                       (T, max_keys ignored)
 *   VERIFY: B, Hq, Hkv, d, T                    (max_keys ignored)
 *   ACCEPT: B, T, max_keys = V                  (Hq, Hkv, d ignored)
 *   ACCEPT_STOCH: B, max_keys = V               (Hq, Hkv, d, T ignored)
 * Returns 0 for an unknown op or invalid sizes.  The memory update and the
 * draft-layer maps take no workspace (MAD_OP_UPDATE is 0 bytes).
 */
size_t mad_workspace_bytes(int op, int B, int Hq, int Hkv, int d, int T, int max_keys);

/* Thread-local description of the last failure in this thread ("" if none). */
const char *mad_last_error(void);

/* Library version string. */
const char *mad_version(void);

#ifdef __cplusplus
}
#endif
#endif /* MAD_H */
