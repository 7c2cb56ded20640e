// mad_internal.h -- kernel argument blocks and launchers shared between the
// C-ABI layer (mad_api.hip) and the kernels.  Not installed; not part of the ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/mad.h"

namespace mad {

constexpr int kMaxB = MAD_MAX_BATCH;

// ---------------------------------------------------------------- decode ----
// Keys per split are a multiple of kDecodeChunkQuant and at least
// kDecodeMinChunk; the split count aims at kDecodeTargetWGs workgroups.
#ifndef MAD_DECODE_TARGET_WGS
#define MAD_DECODE_TARGET_WGS 1024
#endif
#ifndef MAD_DECODE_MIN_CHUNK
#define MAD_DECODE_MIN_CHUNK 32
#endif
#ifndef MAD_DECODE_CHUNK_QUANT
#define MAD_DECODE_CHUNK_QUANT 16
#endif
constexpr int kDecodeTargetWGs = MAD_DECODE_TARGET_WGS;
constexpr int kDecodeMinChunk = MAD_DECODE_MIN_CHUNK;
constexpr int kDecodeChunkQuant = MAD_DECODE_CHUNK_QUANT;
constexpr int kDecodeMaxSplits = 256;

struct DecodeArgs {
    const void *q;
    void *out;
    float *lse;
    const void *mk, *mv;  // memory segment (sinks, slots): linear
    int64_t m_seq, m_head;
    void *wk, *wv;        // local window: ring
    int64_t w_seq, w_head;
    const void *kn, *vn;  // current token K/V [B][Hkv][D] or null
    float *part_o;        // [units][n_splits][G][D]
    float *part_ml;       // [units][n_splits][G][2]
    unsigned *counters;   // [units]
    float scale_log2;     // softmax scale * log2(e)
    int Hq, Hkv, units, n_splits, chunk, w_cap;
    int mlen[kMaxB], wstart[kMaxB], wlen[kMaxB];
};

struct DecodePlan {
    int units, n_splits, chunk, n_max;
};

DecodePlan plan_decode(int B, int Hkv, const int *n_keys);
size_t decode_ws_bytes(int B, int Hq, int Hkv, int d);
hipError_t launch_decode(const DecodeArgs &a, int dtype, int d, int G, hipStream_t st);

// ws layout helpers: counters first (256-byte aligned), then partials.
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace mad
