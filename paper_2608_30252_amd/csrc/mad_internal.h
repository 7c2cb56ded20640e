// mad_internal.h -- kernel argument blocks and launchers shared between the
// C-ABI layer (mad_api.hip) and the kernels.  Not installed; not part of the ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "mad.h"

namespace mad {

constexpr int kMaxB = MAD_MAX_BATCH;

// ---------------------------------------------------------------- decode ----
// The split count aims at one 4-wave or two 8-wave workgroups per CU; splits
// are whole super-tiles (see plan_decode).
constexpr int kDecodeCUs = 256;        // compute units of the device the split plan is sized for
constexpr int kDecodeWideKeys = 65536;      // 8-wave workgroups: launches holding at least this many keys
constexpr int kDecodeMaxSplits = 256;
// Every workspace starts with a fixed counter region that holds nothing but
// arrival counters (one per 256-byte line) and that every kernel leaves at
// zero.  Its layout therefore never overlaps the partial results of a call
// with other shapes.  Split partials follow it.
constexpr size_t kCounterRegionBytes = (size_t)1 << 20;
constexpr int kCounterStride = 64;   // unsigned ints per counter line
constexpr int kCounterLines = (int)(kCounterRegionBytes / (kCounterStride * 4));

struct DecodeArgs {
    const void *q;
    void *out;
    float *lse;
    const void *mk, *mv;  // memory segment (sinks, slots): linear
    int64_t m_seq, m_head;
    void *wk, *wv;        // local window: ring
    int64_t w_seq, w_head;
    const void *kn, *vn;  // current token K/V [B][Hkv][D] or null
    float *part;          // split partials, one block of part_stride floats per unit
    int64_t part_stride;
    unsigned *counters;   // counter region: unit u on line u
    float scale_log2;     // softmax scale * log2(e)
    int Hq, Hkv, units, n_splits, chunk, w_cap;
    int nsub;             // wave groups per workgroup (1 or 2)
    int fold;             // 1: the last split runs to the end of the row (keys past n_splits * chunk)
    // per row, one 16-byte record read by a single scalar load: memory length,
    // window length, ring start, new-token mode (0 none, 1 attend, 2 attend and append)
    int4 seq[kMaxB];
};

struct DecodePlan {
    int units, n_splits, chunk, n_max, nsub;
    int fold;   // 1: the last split also takes the few keys past n_splits * chunk
};

DecodePlan plan_decode(int B, int Hkv, int G, int d, int dtype, const int *n_keys);
int decode_max_splits(int d, int G);
size_t decode_part_stride(int d, int G);
size_t decode_ws_bytes(int B, int Hq, int Hkv, int d);
hipError_t launch_decode(const DecodeArgs &a, int dtype, int d, int G, hipStream_t st);

// ---------------------------------------------------------------- update ----
struct UpdateArgs {
    const void *x, *w;    // [R][D] slot rows, [2*Hkv*d][D] mirrored projections
    void *mk, *mv;        // memory segment to append to
    int64_t m_seq, m_head;
    double log2_base;     // log2 of the RoPE base
    int R, n_new, D, Hkv, d;
    int mlen[kMaxB];
    int pos[MAD_MAX_UPDATE_ROWS];
    unsigned char fire[kMaxB];
};

hipError_t launch_update(const UpdateArgs &a, int dtype, hipStream_t st);
constexpr int kUpdateGemvRows = 8;   // bf16 updates of at most this many rows take the weight stream
bool update_uses_gemv(int R, int D, int dtype);

// ---------------------------------------------------------------- verify ----
constexpr int kVerifyTargetWGs = 256;   // workgroups the split count aims at (one per CU)
constexpr int kVerifyMaxSplits = 128;

struct VerifyArgs {
    const void *q, *k, *vt;   // vt: V in natural rows [cap][d] when vnat, else one run of cap keys per feature
    void *out;
    float *lse;
    int64_t seq, head;    // element strides of sequences and KV heads (K and V^T alike)
    float *part;          // [units][n_splits][part_rows][d] split partials (unnormalised o)
    float *part_ml;       // [units][n_splits][part_rows][2] (max, sum)
    float scale_log2;
    int cap, Hq, Hkv, G, T, d, units, n_splits, chunk, part_rows;
    int vnat;             // 1: V stored in natural rows
    int len[kMaxB];
};

// ----------------------------------------------------------------- layer ----
constexpr int kMaxLinRows = MAD_MAX_LAYER_ROWS;

struct LinearArgs {
    const void *x, *w, *gamma, *res;
    void *out, *xn, *q, *k, *v;
    float eps;
    double log2_base;
    int R, D, N, Hq, Hkv, head_dim, kv_from_row0;
    int pos[kMaxLinRows];
};

hipError_t launch_linear(const LinearArgs &a, int mode, hipStream_t st);

// --------------------------------------------------------------- prefill ----
struct PrefillArgs {
    const void *q_raw, *q_slot;
    void *o_raw, *o_slot;
    float *lse_raw, *lse_slot;
    const void *mk, *mv;  // memory segment: sinks, then slots
    int64_t m_seq, m_head;
    const void *rk, *rv;  // the prefix's raw K/V, position x in row x
    int64_t r_seq, r_head;
    float scale_log2;
    int q_cap, slot_cap, Hq, Hkv, units, nrb, nsb;
    int S, W, r, u;
    int P[kMaxB], Mtot[kMaxB];
};

int prefill_tokens_per_block(int d, int G);
hipError_t launch_prefill(const PrefillArgs &a, int d, int G, hipStream_t st);

struct VerifyPlan {
    int units, n_splits, chunk;
};

VerifyPlan plan_verify(int B, int Hkv, int G, int T, const int *len, bool vnat);
size_t verify_ws_bytes(int B, int Hq, int Hkv, int d, int T);
void verify_ws_layout(int B, int Hq, int Hkv, int d, int T, size_t *off_o, size_t *off_ml);
hipError_t launch_verify(const VerifyArgs &a, hipStream_t st);

// ---------------------------------------------------------------- accept ----
constexpr int kAcceptChunk = 8192;   // vocabulary entries per workgroup
constexpr int kAcceptMaxT = 256;     // rows per sequence of the greedy rule (one workgroup applies it)
static_assert((size_t)kMaxB * kCounterStride * 4 + (size_t)kMaxB * kAcceptMaxT * 8 <= kCounterRegionBytes,
              "greedy-accept counters and row keys fit the counter region");

struct AcceptArgs {
    const void *logits;
    const int32_t *draft;      // [B][T-1] device
    int32_t *n_accept, *next_tok;
    uint64_t *row_best;        // [rows] row argmax keys, in the counter region after line B-1 (zero between calls)
    unsigned *counters;        // line b: arrivals of sequence b's workgroups
    int B, T, V, n_chunks;
    int vec16;                 // rows 16-byte aligned and V a multiple of 16 / element size
};

size_t accept_ws_bytes(int B, int T, int V);
hipError_t launch_accept(const AcceptArgs &a, int dtype, hipStream_t st);

struct StochArgs {
    const float *p, *q, *u;    // [B][T][V], [B][T-1][V], [B][T]
    const int32_t *draft;      // [B][T-1]
    int32_t *n_accept, *next_tok;
    double *sums;              // [B][n_chunks][2]: chunk sums of the draw's r and of p_a
    unsigned *counters;        // line b: arrivals of sequence b's chunks
    int B, T, V, n_chunks;
    int vec16;                 // rows of p and q 16-byte aligned (V % 4 == 0, aligned bases)
};
size_t stoch_ws_bytes(int B, int V);
hipError_t launch_stoch(const StochArgs &a, hipStream_t st);

// ws layout helpers: counters first (256-byte aligned), then partials.
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace mad
