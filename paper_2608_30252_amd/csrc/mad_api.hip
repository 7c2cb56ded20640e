// mad_api.hip -- the C ABI of libmad: argument validation, split planning,
// workspace accounting and kernel launch.  Every check runs on the host before
// anything is enqueued; no exception leaves this file.
#include <stdarg.h>
#include <stdio.h>
#include <math.h>
#include <string.h>

#include <mutex>

#include "mad_internal.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_err[0] = '\0';
    return MAD_OK;
}

int hip_status(hipError_t e, const char *what) {
    if (e != hipSuccess) return fail(MAD_EHIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int elem_size(int dtype) { return dtype == MAD_BF16 ? 2 : 4; }

bool pow2_group(int G) { return G == 1 || G == 2 || G == 4 || G == 8 || G == 16; }

// Common shape checks for attention entry points.
int check_heads(int B, int Hq, int Hkv, int d, int dtype) {
    if (B < 1 || B > MAD_MAX_BATCH) return fail(MAD_EINVAL, "B=%d outside [1, %d]", B, MAD_MAX_BATCH);
    if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0)
        return fail(MAD_EINVAL, "Hq=%d must be a positive multiple of Hkv=%d", Hq, Hkv);
    if (dtype != MAD_F32 && dtype != MAD_BF16) return fail(MAD_ENOTSUP, "dtype %d not supported", dtype);
    if (d != 64 && d != 128) return fail(MAD_ENOTSUP, "head_dim %d not supported (64 or 128)", d);
    if (!pow2_group(Hq / Hkv)) return fail(MAD_ENOTSUP, "group size %d not supported (1,2,4,8,16)", Hq / Hkv);
    return MAD_OK;
}

// Validate a kv view for B sequences; `ring` enables the start array check;
// rows with append[b] != 0 need room for one more row.
int check_view(const mad_kv_view *v, const char *name, int B, int Hkv, int d, int dtype, bool ring,
               const unsigned char *append) {
    if (!v->k || !v->v) return fail(MAD_EINVAL, "%s: null k or v", name);
    if (!aligned16(v->k) || !aligned16(v->v)) return fail(MAD_EINVAL, "%s: k/v not 16-byte aligned", name);
    if (v->cap < 1) return fail(MAD_EINVAL, "%s: cap=%d", name, v->cap);
    if (!v->len) return fail(MAD_EINVAL, "%s: null len", name);
    const int vec = 16 / elem_size(dtype);
    if (v->seq_stride < 0 || v->head_stride < (int64_t)v->cap * d || v->seq_stride % vec || v->head_stride % vec)
        return fail(MAD_EINVAL, "%s: bad strides (seq %lld, head %lld) for cap %d, d %d", name,
                    (long long)v->seq_stride, (long long)v->head_stride, v->cap, d);
    if (v->seq_stride != 0 && v->seq_stride < (int64_t)Hkv * v->head_stride && B > 1)
        return fail(MAD_EINVAL, "%s: seq_stride %lld overlaps heads", name, (long long)v->seq_stride);
    for (int b = 0; b < B; ++b) {
        int len = v->len[b];
        int room = (append && append[b]) ? 1 : 0;
        if (len < 0 || len + room > v->cap)
            return fail(MAD_EINVAL, "%s: len[%d]=%d (+%d) exceeds cap %d", name, b, len, room, v->cap);
        if (ring && v->start) {
            int st = v->start[b];
            if (st < 0 || st >= v->cap) return fail(MAD_EINVAL, "%s: start[%d]=%d outside [0, cap)", name, b, st);
        }
    }
    return MAD_OK;
}

}  // namespace

extern "C" {

const char *mad_last_error(void) { return g_err; }

const char *mad_version(void) { return "libmad 0.1 (gfx950)"; }

size_t mad_workspace_bytes(int op, int B, int Hq, int Hkv, int d, int T, int max_keys) {
    (void)max_keys;
    switch (op) {
        case MAD_OP_DECODE:
            if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || (d != 64 && d != 128)) return 0;
            return mad::decode_ws_bytes(B, Hq, Hkv, d);
        case MAD_OP_VERIFY:
            if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || (d != 64 && d != 128) || T < 1) return 0;
            return mad::verify_ws_bytes(B, Hq, Hkv, d, T);
        case MAD_OP_ACCEPT_STOCH:   // B, max_keys = V
            if (B < 1 || B > MAD_MAX_BATCH || max_keys < 1) return 0;
            return mad::stoch_ws_bytes(B, max_keys);
        case MAD_OP_ACCEPT:   // B, T, max_keys = V
            if (B < 1 || B > MAD_MAX_BATCH || T < 1 || T > mad::kAcceptMaxT || max_keys < 1) return 0;
            return mad::accept_ws_bytes(B, T, max_keys);
        default:
            return 0;
    }
}

}  // extern "C"

namespace {

// The draft decode attention with a per-row new-token mode (0: none, 1: attend
// k_new/v_new, 2: attend and append to the ring); both entry points use it.
int decode_impl(const void *q, int B, int Hq, int Hkv, int d, int dtype, float scale, const mad_kv_view *mem,
                const mad_kv_view *win, const void *k_new, const void *v_new, const unsigned char *mode, void *out,
                float *lse, void *ws, size_t ws_bytes, void *stream) {
    int rc = check_heads(B, Hq, Hkv, d, dtype);
    if (rc) return rc;
    if (!q || !out) return fail(MAD_EINVAL, "null q or out");
    if (!aligned16(q) || !aligned16(out)) return fail(MAD_EINVAL, "q/out not 16-byte aligned");
    if ((k_new == nullptr) != (v_new == nullptr)) return fail(MAD_EINVAL, "k_new and v_new must both be given or both null");
    if (k_new && (!aligned16(k_new) || !aligned16(v_new))) return fail(MAD_EINVAL, "k_new/v_new not 16-byte aligned");
    unsigned char append[MAD_MAX_BATCH];
    int n_append = 0;
    for (int b = 0; b < B; ++b) {
        if (mode[b] > 2) return fail(MAD_EINVAL, "new_mode[%d]=%d outside {0, 1, 2}", b, (int)mode[b]);
        if (mode[b] && !k_new) return fail(MAD_EINVAL, "new_mode[%d]=%d needs k_new and v_new", b, (int)mode[b]);
        append[b] = mode[b] == 2;
        n_append += append[b];
    }
    if (n_append && !win) return fail(MAD_EINVAL, "appending the new token needs a window ring");
    if (n_append > 1 && win->seq_stride == 0)
        return fail(MAD_EINVAL, "rows that share one window ring (seq_stride 0) cannot all append to it");
    if (!(scale > 0.f) || scale != scale) return fail(MAD_EINVAL, "scale must be positive");
    if (mem && (rc = check_view(mem, "mem", B, Hkv, d, dtype, false, nullptr))) return rc;
    if (win && (rc = check_view(win, "win", B, Hkv, d, dtype, true, append))) return rc;
    const int G = Hq / Hkv;
    if ((size_t)B * Hkv > (size_t)mad::kCounterLines)
        return fail(MAD_ENOTSUP, "B*Hkv=%d too large for the counter region", B * Hkv);

    mad::DecodeArgs a;
    memset(&a, 0, sizeof(a));
    int n_keys[MAD_MAX_BATCH];
    for (int b = 0; b < B; ++b) {
        a.seq[b].x = mem ? mem->len[b] : 0;
        a.seq[b].y = win ? win->len[b] : 0;
        a.seq[b].z = (win && win->start) ? win->start[b] : 0;
        a.seq[b].w = mode[b];
        n_keys[b] = a.seq[b].x + a.seq[b].y + (mode[b] ? 1 : 0);
    }
    mad::DecodePlan p = mad::plan_decode(B, Hkv, G, d, dtype, n_keys);
    size_t need = p.n_splits > 1 ? mad::decode_ws_bytes(B, Hq, Hkv, d) : 0;
    if (need > 0) {
        if (!ws) return fail(MAD_EWS, "workspace required (%zu bytes)", need);
        if (ws_bytes < need) return fail(MAD_EWS, "workspace %zu bytes < %zu", ws_bytes, need);
        if (!aligned16(ws)) return fail(MAD_EINVAL, "workspace not 16-byte aligned");
    }
    a.q = q;
    a.out = out;
    a.lse = lse;
    if (mem) {
        a.mk = mem->k; a.mv = mem->v; a.m_seq = mem->seq_stride; a.m_head = mem->head_stride;
    }
    if (win) {
        a.wk = win->k; a.wv = win->v; a.w_seq = win->seq_stride; a.w_head = win->head_stride;
        a.w_cap = win->cap;
    } else {
        a.w_cap = 1;
    }
    a.kn = k_new;
    a.vn = v_new;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.units = p.units;
    a.n_splits = p.n_splits;
    a.nsub = p.nsub;
    a.chunk = p.chunk;
    a.fold = p.fold;
    if (need > 0) {
        a.counters = (unsigned *)ws;
        a.part = (float *)((char *)ws + mad::kCounterRegionBytes);
        a.part_stride = (int64_t)mad::decode_part_stride(d, G);
    }
    return hip_status(mad::launch_decode(a, dtype, d, G, (hipStream_t)stream), "decode launch");
}

}  // namespace

extern "C" {

int mad_draft_decode_attn(const void *q, int B, int Hq, int Hkv, int d, int dtype, float scale,
                          const mad_kv_view *mem, const mad_kv_view *win, const void *k_new,
                          const void *v_new, void *out, float *lse, void *ws, size_t ws_bytes,
                          void *stream) {
    if (B < 1 || B > MAD_MAX_BATCH) return fail(MAD_EINVAL, "B=%d outside [1, %d]", B, MAD_MAX_BATCH);
    if (k_new && !win) return fail(MAD_EINVAL, "k_new needs a window ring to append to");
    unsigned char mode[MAD_MAX_BATCH];
    for (int b = 0; b < B; ++b) mode[b] = k_new ? 2 : 0;
    return decode_impl(q, B, Hq, Hkv, d, dtype, scale, mem, win, k_new, v_new, mode, out, lse, ws, ws_bytes,
                       stream);
}

}  // extern "C"

namespace {

// ---- the no-allocation decode entry point's scratch -----------------------
// One library-owned device array per GPU (every device that runs the library
// holds its own copy until the process ends): the counter region followed by
// split partials, the same layout as a caller workspace.  In host code the
// array's name only names the symbol; its device address on the current GPU
// comes from hipGetSymbolAddress, looked up once per device and kept.
constexpr size_t kNoallocScratchBytes = (size_t)MAD_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

__global__ void zero_words(unsigned *p, unsigned n) {
    for (unsigned i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0u;
}

// The current device's scratch address; on the first call on a device, look it
// up and clear the counter region with a kernel on `stream` (the kernels leave
// it at zero after every call, so this happens once).
int scratch_of_current_device(hipStream_t stream, void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(MAD_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return fail(MAD_EHIP, "device ordinal %d outside [0, %d)", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(MAD_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
        hipLaunchKernelGGL(zero_words, dim3(256), dim3(256), 0, stream, (unsigned *)p,
                           (unsigned)(mad::kCounterRegionBytes / 4));
        e = hipGetLastError();
        if (e != hipSuccess) return fail(MAD_EHIP, "scratch clear launch: %s", hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return MAD_OK;
}

}  // namespace

extern "C" {

int mad_draft_decode_attn_noalloc(const void *q, int B, int Hq, int Hkv, int d, int dtype, float scale,
                                  const mad_kv_view *mem, const mad_kv_view *win, const void *k_new,
                                  const void *v_new, void *out, float *lse, void *stream) {
    if (B < 1 || B > MAD_MAX_BATCH) return fail(MAD_EINVAL, "B=%d outside [1, %d]", B, MAD_MAX_BATCH);
    int rc = check_heads(B, Hq, Hkv, d, dtype);
    if (rc) return rc;
    const size_t need = mad::decode_ws_bytes(B, Hq, Hkv, d);
    if (need > kNoallocScratchBytes)
        return fail(MAD_EINVAL, "B=%d, Hkv=%d, d=%d need %zu bytes of scratch, above the %zu-byte limit of the "
                    "no-allocation entry point (use mad_draft_decode_attn with a workspace)", B, Hkv, d, need,
                    kNoallocScratchBytes);
    if (k_new && !win) return fail(MAD_EINVAL, "k_new needs a window ring to append to");
    void *ws = nullptr;
    if ((rc = scratch_of_current_device((hipStream_t)stream, &ws))) return rc;
    unsigned char mode[MAD_MAX_BATCH];
    for (int b = 0; b < B; ++b) mode[b] = k_new ? 2 : 0;
    return decode_impl(q, B, Hq, Hkv, d, dtype, scale, mem, win, k_new, v_new, mode, out, lse, ws,
                       kNoallocScratchBytes, stream);
}

int mad_draft_step_attn(const void *q, int B, int Hq, int Hkv, int d, int dtype, float scale,
                        const mad_kv_view *mem, const mad_kv_view *win, const void *k_new, const void *v_new,
                        const uint8_t *new_mode, void *out, float *lse, void *ws, size_t ws_bytes, void *stream) {
    if (B < 1 || B > MAD_MAX_BATCH) return fail(MAD_EINVAL, "B=%d outside [1, %d]", B, MAD_MAX_BATCH);
    if (!new_mode) return fail(MAD_EINVAL, "null new_mode");
    return decode_impl(q, B, Hq, Hkv, d, dtype, scale, mem, win, k_new, v_new, new_mode, out, lse, ws, ws_bytes,
                       stream);
}

int mad_memory_update(const void *x, const void *w_kv, const int32_t *pos, const uint8_t *fire, int B, int n_new,
                      int D, int Hkv, int d, int dtype, double rope_base, const mad_kv_view *mem, void *stream) {
    if (B < 1 || B > MAD_MAX_BATCH) return fail(MAD_EINVAL, "B=%d outside [1, %d]", B, MAD_MAX_BATCH);
    if (n_new < 1 || B * n_new > MAD_MAX_UPDATE_ROWS)
        return fail(MAD_EINVAL, "B*n_new=%d outside [1, %d]", B * n_new, MAD_MAX_UPDATE_ROWS);
    if (dtype != MAD_F32 && dtype != MAD_BF16) return fail(MAD_ENOTSUP, "dtype %d not supported", dtype);
    if (d != 64 && d != 128) return fail(MAD_ENOTSUP, "head_dim %d not supported (64 or 128)", d);
    if (Hkv < 1 || 2 * Hkv > mad::kCounterLines) return fail(MAD_EINVAL, "Hkv=%d", Hkv);
    if (D < 64 || D % 64) return fail(MAD_EINVAL, "D=%d must be a positive multiple of 64", D);
    if (!x || !w_kv || !pos || !mem) return fail(MAD_EINVAL, "null x, w_kv, pos or mem");
    if (!aligned16(x) || !aligned16(w_kv)) return fail(MAD_EINVAL, "x/w_kv not 16-byte aligned");
    if (!(rope_base > 1.0) || rope_base != rope_base || rope_base > 1e300)
        return fail(MAD_EINVAL, "rope_base must be finite and > 1");
    int rc = check_view(mem, "mem", B, Hkv, d, dtype, false, nullptr);
    if (rc) return rc;
    for (int b = 0; b < B; ++b) {
        const bool f = fire ? fire[b] != 0 : true;
        if (f && mem->len[b] + n_new > mem->cap)
            return fail(MAD_EINVAL, "mem: len[%d]=%d + n_new=%d exceeds cap %d", b, mem->len[b], n_new, mem->cap);
    }
    const int R = B * n_new;
    mad::UpdateArgs a;
    memset(&a, 0, sizeof(a));
    a.x = x;
    a.w = w_kv;
    a.mk = mem->k;
    a.mv = mem->v;
    a.m_seq = mem->seq_stride;
    a.m_head = mem->head_stride;
    a.log2_base = log2(rope_base);
    a.R = R;
    a.n_new = n_new;
    a.D = D;
    a.Hkv = Hkv;
    a.d = d;
    for (int b = 0; b < B; ++b) {
        a.mlen[b] = mem->len[b];
        a.fire[b] = (unsigned char)(fire ? (fire[b] != 0) : 1);
    }
    for (int r = 0; r < R; ++r) a.pos[r] = pos[r];
    return hip_status(mad::launch_update(a, dtype, (hipStream_t)stream), "memory update launch");
}

}  // extern "C"

namespace {

// The verify attention over either V layout; K and V share the strides.
int verify_impl(const void *q, int B, int T, int Hq, int Hkv, int d, int dtype, float scale, const void *k,
                const void *v, bool vnat, int64_t seq_stride, int64_t head_stride, int32_t cap, const int32_t *len,
                void *out, float *lse, void *ws, size_t ws_bytes, void *stream) {
    int rc = check_heads(B, Hq, Hkv, d, dtype);
    if (rc) return rc;
    if (dtype != MAD_BF16 && !(dtype == MAD_F32 && vnat))
        return fail(MAD_ENOTSUP, "the transposed-V verify runs in bf16 only (matrix cores)");
    const int G = Hq / Hkv;
    if (T < 1 || T * G > MAD_MAX_VERIFY_ROWS)
        return fail(MAD_EINVAL, "T=%d: T*G=%d must be in [1, %d]", T, T * G, MAD_MAX_VERIFY_ROWS);
    if (!q || !k || !v || !out || !len) return fail(MAD_EINVAL, "null q, k, v, out or len");
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
        return fail(MAD_EINVAL, "q/k/v/out not 16-byte aligned");
    if (!(scale > 0.f) || scale != scale) return fail(MAD_EINVAL, "scale must be positive");
    if (vnat) {
        if (cap < 1) return fail(MAD_EINVAL, "cap=%d", cap);
    } else if (cap < 8 || cap % 8) {
        return fail(MAD_EINVAL, "cap=%d must be a positive multiple of 8 (transposed V)", cap);
    }
    if (head_stride < (int64_t)cap * d || head_stride % 8 || seq_stride < 0 || seq_stride % 8)
        return fail(MAD_EINVAL, "bad strides (seq %lld, head %lld) for cap %d, d %d", (long long)seq_stride,
                    (long long)head_stride, cap, d);
    if (B > 1 && seq_stride != 0 && seq_stride < (int64_t)Hkv * head_stride)
        return fail(MAD_EINVAL, "seq_stride %lld overlaps heads", (long long)seq_stride);
    for (int b = 0; b < B; ++b)
        if (len[b] < T || len[b] > cap) return fail(MAD_EINVAL, "len[%d]=%d outside [T=%d, cap=%d]", b, len[b], T, cap);
    const size_t need = mad::verify_ws_bytes(B, Hq, Hkv, d, T);
    if (!ws) return fail(MAD_EWS, "workspace required (%zu bytes)", need);
    if (ws_bytes < need) return fail(MAD_EWS, "workspace %zu bytes < %zu", ws_bytes, need);
    if (!aligned16(ws)) return fail(MAD_EINVAL, "workspace not 16-byte aligned");
    if (dtype == MAD_F32) {
        // fp32 (on the vector ALUs): per sequence b, one decode launch whose T rows
        // are the T queries, all reading b's cache (row stride 0) with query t
        // limited to rows 0 .. len-T+t; launches on one stream, one workspace
        const size_t qrow = (size_t)T * Hq * d * 4;
        for (int b = 0; b < B; ++b) {
            int32_t lens[MAD_MAX_BATCH];
            for (int t = 0; t < T; ++t) lens[t] = len[b] - T + t + 1;
            mad_kv_view kv;
            memset(&kv, 0, sizeof(kv));
            kv.k = (char *)k + (size_t)b * seq_stride * 4;
            kv.v = (char *)v + (size_t)b * seq_stride * 4;
            kv.seq_stride = 0;
            kv.head_stride = head_stride;
            kv.cap = cap;
            kv.start = nullptr;
            kv.len = lens;
            unsigned char mode[MAD_MAX_BATCH] = {0};
            rc = decode_impl((const char *)q + b * qrow, T, Hq, Hkv, d, MAD_F32, scale, &kv, nullptr, nullptr,
                             nullptr, mode, (char *)out + b * qrow, lse ? lse + (size_t)b * T * Hq : nullptr, ws,
                             ws_bytes, stream);
            if (rc) return rc;
        }
        return MAD_OK;
    }
    mad::VerifyPlan p = mad::plan_verify(B, Hkv, G, T, len, vnat);
    mad::VerifyArgs a;
    memset(&a, 0, sizeof(a));
    a.q = q;
    a.k = k;
    a.vt = v;
    a.vnat = vnat ? 1 : 0;
    a.out = out;
    a.lse = lse;
    a.seq = seq_stride;
    a.head = head_stride;
    size_t off_o, off_ml;
    mad::verify_ws_layout(B, Hq, Hkv, d, T, &off_o, &off_ml);
    a.part = (float *)((char *)ws + off_o);
    a.part_ml = (float *)((char *)ws + off_ml);
    a.scale_log2 = scale * 1.4426950408889634f;
    a.cap = cap;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.G = G;
    a.T = T;
    a.d = d;
    a.units = p.units;
    a.n_splits = p.n_splits;
    a.chunk = p.chunk;
    a.part_rows = T * G;
    for (int b = 0; b < B; ++b) a.len[b] = len[b];
    return hip_status(mad::launch_verify(a, (hipStream_t)stream), "verify launch");
}

}  // namespace

extern "C" {

int mad_verify_attn(const void *q, int B, int T, int Hq, int Hkv, int d, int dtype, float scale,
                    const mad_kv_view *kv, void *out, float *lse, void *ws, size_t ws_bytes, void *stream) {
    if (!kv) return fail(MAD_EINVAL, "null kv");
    if (kv->start) return fail(MAD_EINVAL, "kv: the verifier's cache is linear (start must be NULL)");
    if (!kv->len) return fail(MAD_EINVAL, "kv: null len");
    return verify_impl(q, B, T, Hq, Hkv, d, dtype, scale, kv->k, kv->v, true, kv->seq_stride, kv->head_stride,
                       kv->cap, kv->len, out, lse, ws, ws_bytes, stream);
}

int mad_verify_attn_vt(const void *q, int B, int T, int Hq, int Hkv, int d, int dtype, float scale, const void *k,
                       const void *vt, int64_t seq_stride, int64_t head_stride, int32_t cap, const int32_t *len,
                       void *out, float *lse, void *ws, size_t ws_bytes, void *stream) {
    return verify_impl(q, B, T, Hq, Hkv, d, dtype, scale, k, vt, false, seq_stride, head_stride, cap, len, out, lse,
                       ws, ws_bytes, stream);
}

int mad_memory_prefill_attn(const void *q_raw, const void *q_slot, int B, int Hq, int Hkv, int d, int dtype,
                            float scale, const int32_t *P, int q_cap, int slot_cap, int S, int W, int r, int u,
                            const mad_kv_view *mem, const mad_kv_view *raw, void *out_raw, float *lse_raw,
                            void *out_slot, float *lse_slot, void *stream) {
    int rc = check_heads(B, Hq, Hkv, d, dtype);
    if (rc) return rc;
    if (dtype != MAD_BF16) return fail(MAD_ENOTSUP, "memory-prefill attention runs in bf16 only");
    const int G = Hq / Hkv;
    if (G > 8) return fail(MAD_ENOTSUP, "group size %d not supported by the prefill (1, 2, 4, 8)", G);
    if (!q_raw || !out_raw || !P || !mem || !raw) return fail(MAD_EINVAL, "null q_raw, out_raw, P, mem or raw");
    if (q_slot && !out_slot) return fail(MAD_EINVAL, "q_slot given without out_slot");
    if (!aligned16(q_raw) || !aligned16(out_raw) || (q_slot && (!aligned16(q_slot) || !aligned16(out_slot))))
        return fail(MAD_EINVAL, "q/out not 16-byte aligned");
    if (!(scale > 0.f) || scale != scale) return fail(MAD_EINVAL, "scale must be positive");
    if (S < 0 || W < 1 || r < 1 || u < 1) return fail(MAD_EINVAL, "S=%d W=%d r=%d u=%d", S, W, r, u);
    if (q_cap < 1 || (q_slot && slot_cap < 1)) return fail(MAD_EINVAL, "q_cap=%d slot_cap=%d", q_cap, slot_cap);
    if (raw->start) return fail(MAD_EINVAL, "raw: the prefix's K/V are linear (start must be NULL)");
    if ((rc = check_view(mem, "mem", B, Hkv, d, dtype, false, nullptr))) return rc;
    if ((rc = check_view(raw, "raw", B, Hkv, d, dtype, false, nullptr))) return rc;
    if ((size_t)r * (size_t)u > 0x3fffffff) return fail(MAD_EINVAL, "r*u too large");
    int Mtot[MAD_MAX_BATCH];
    int P_max = 0, M_max = 0;
    for (int b = 0; b < B; ++b) {
        if (P[b] < 0 || P[b] > q_cap) return fail(MAD_EINVAL, "P[%d]=%d outside [0, q_cap=%d]", b, P[b], q_cap);
        Mtot[b] = P[b] <= S ? 0 : (P[b] - S) / (r * u) * u;
        const int need_mem = P[b] <= S ? P[b] : S + Mtot[b];
        if (mem->len[b] < need_mem)
            return fail(MAD_EINVAL, "mem: len[%d]=%d < %d rows (sinks + slots of the prefix)", b, mem->len[b], need_mem);
        if (raw->len[b] < P[b]) return fail(MAD_EINVAL, "raw: len[%d]=%d < P=%d", b, raw->len[b], P[b]);
        if (q_slot && Mtot[b] > slot_cap)
            return fail(MAD_EINVAL, "sequence %d has %d slots > slot_cap=%d", b, Mtot[b], slot_cap);
        P_max = P[b] > P_max ? P[b] : P_max;
        M_max = Mtot[b] > M_max ? Mtot[b] : M_max;
    }
    if (P_max == 0) return ok();
    const int QT = mad::prefill_tokens_per_block(d, G);
    mad::PrefillArgs a;
    memset(&a, 0, sizeof(a));
    a.q_raw = q_raw;
    a.q_slot = q_slot;
    a.o_raw = out_raw;
    a.o_slot = out_slot;
    a.lse_raw = lse_raw;
    a.lse_slot = q_slot ? lse_slot : nullptr;
    a.mk = mem->k;
    a.mv = mem->v;
    a.m_seq = mem->seq_stride;
    a.m_head = mem->head_stride;
    a.rk = raw->k;
    a.rv = raw->v;
    a.r_seq = raw->seq_stride;
    a.r_head = raw->head_stride;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.q_cap = q_cap;
    a.slot_cap = q_slot ? slot_cap : 0;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.units = B * Hkv;
    a.nrb = (P_max + QT - 1) / QT;
    a.nsb = q_slot ? (M_max + QT - 1) / QT : 0;
    a.S = S;
    a.W = W;
    a.r = r;
    a.u = u;
    for (int b = 0; b < B; ++b) {
        a.P[b] = P[b];
        a.Mtot[b] = Mtot[b];
    }
    return hip_status(mad::launch_prefill(a, d, G, (hipStream_t)stream), "memory prefill launch");
}

int mad_rmsnorm_qkv_rope(const void *x, const void *gamma, float eps, const void *w_qkv, const int32_t *pos, int R,
                         int D, int Hq, int Hkv, int d, double rope_base, int kv_from_row0, void *q, void *k,
                         void *v, void *xn, void *stream) {
    if (R < 1 || R > MAD_MAX_LAYER_ROWS) return fail(MAD_EINVAL, "R=%d outside [1, %d]", R, MAD_MAX_LAYER_ROWS);
    if (D != 2048 && D != 4096) return fail(MAD_ENOTSUP, "D=%d not supported (2048, 4096)", D);
    if (d != 64 && d != 128) return fail(MAD_ENOTSUP, "head_dim %d not supported (64 or 128)", d);
    if (Hq < 1 || Hkv < 1 || Hq % Hkv) return fail(MAD_EINVAL, "Hq=%d must be a positive multiple of Hkv=%d", Hq, Hkv);
    if (!x || !gamma || !w_qkv || !pos || !q || !k || !v) return fail(MAD_EINVAL, "null x, gamma, w_qkv, pos, q, k or v");
    if (!aligned16(x) || !aligned16(gamma) || !aligned16(w_qkv) || (xn && !aligned16(xn)))
        return fail(MAD_EINVAL, "x/gamma/w_qkv/xn not 16-byte aligned");
    if (!(eps > 0.f) || !(rope_base > 1.0) || rope_base != rope_base || isinf(rope_base))
        return fail(MAD_EINVAL, "eps must be positive and rope_base finite and > 1");
    mad::LinearArgs a;
    memset(&a, 0, sizeof(a));
    a.x = x;
    a.w = w_qkv;
    a.gamma = gamma;
    a.q = q;
    a.k = k;
    a.v = v;
    a.xn = xn;
    a.eps = eps;
    a.log2_base = log2(rope_base);
    a.R = R;
    a.D = D;
    a.N = (Hq + 2 * Hkv) * d;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.head_dim = d;
    a.kv_from_row0 = kv_from_row0 ? 1 : 0;
    for (int r = 0; r < R; ++r) a.pos[r] = pos[r];
    return hip_status(mad::launch_linear(a, 0, (hipStream_t)stream), "qkv projection launch");
}

int mad_linear_residual(const void *x, const void *w, const void *res, int R, int D, int N, void *out, void *stream) {
    if (R < 1 || R > MAD_MAX_LAYER_ROWS) return fail(MAD_EINVAL, "R=%d outside [1, %d]", R, MAD_MAX_LAYER_ROWS);
    if (D != 2048 && D != 4096 && D != 8192) return fail(MAD_ENOTSUP, "D=%d not supported (2048, 4096, 8192)", D);
    if (N < 4 || N % 4) return fail(MAD_EINVAL, "N=%d must be a positive multiple of 4", N);
    if (!x || !w || !res || !out) return fail(MAD_EINVAL, "null x, w, res or out");
    if (!aligned16(x) || !aligned16(w)) return fail(MAD_EINVAL, "x/w not 16-byte aligned");
    const char *xb = (const char *)x, *ob = (const char *)out;
    if (ob < xb + (size_t)R * D * 2 && xb < ob + (size_t)R * N * 2) return fail(MAD_EINVAL, "out overlaps x");
    mad::LinearArgs a;
    memset(&a, 0, sizeof(a));
    a.x = x;
    a.w = w;
    a.res = res;
    a.out = out;
    a.R = R;
    a.D = D;
    a.N = N;
    return hip_status(mad::launch_linear(a, 1, (hipStream_t)stream), "linear launch");
}

int mad_rmsnorm_swiglu(const void *x, const void *gamma, float eps, const void *w_gate_up, int R, int D, int F,
                       void *out, void *stream) {
    if (R < 1 || R > MAD_MAX_LAYER_ROWS) return fail(MAD_EINVAL, "R=%d outside [1, %d]", R, MAD_MAX_LAYER_ROWS);
    if (D != 2048 && D != 4096) return fail(MAD_ENOTSUP, "D=%d not supported (2048, 4096)", D);
    if (F < 4 || F % 4) return fail(MAD_EINVAL, "F=%d must be a positive multiple of 4", F);
    if (!x || !gamma || !w_gate_up || !out) return fail(MAD_EINVAL, "null x, gamma, w_gate_up or out");
    if (!aligned16(x) || !aligned16(gamma) || !aligned16(w_gate_up)) return fail(MAD_EINVAL, "x/gamma/w not 16-byte aligned");
    if (!(eps > 0.f)) return fail(MAD_EINVAL, "eps must be positive");
    const char *xb = (const char *)x, *ob = (const char *)out;
    if (ob < xb + (size_t)R * D * 2 && xb < ob + (size_t)R * F * 2) return fail(MAD_EINVAL, "out overlaps x");
    mad::LinearArgs a;
    memset(&a, 0, sizeof(a));
    a.x = x;
    a.w = w_gate_up;
    a.gamma = gamma;
    a.out = out;
    a.eps = eps;
    a.R = R;
    a.D = D;
    a.N = F;
    return hip_status(mad::launch_linear(a, 2, (hipStream_t)stream), "swiglu projection launch");
}

int mad_accept_greedy(const void *logits, int dtype, const int32_t *draft_tok, int B, int T, int V,
                      int32_t *n_accept, int32_t *next_tok, void *ws, size_t ws_bytes, void *stream) {
    if (B < 1 || B > MAD_MAX_BATCH) return fail(MAD_EINVAL, "B=%d outside [1, %d]", B, MAD_MAX_BATCH);
    if (T < 1 || T > mad::kAcceptMaxT) return fail(MAD_EINVAL, "T=%d outside [1, %d]", T, mad::kAcceptMaxT);
    if (V < 1) return fail(MAD_EINVAL, "V=%d", V);
    if (dtype != MAD_F32 && dtype != MAD_BF16) return fail(MAD_ENOTSUP, "dtype %d not supported", dtype);
    if (!logits || !n_accept || !next_tok) return fail(MAD_EINVAL, "null logits, n_accept or next_tok");
    if (T > 1 && !draft_tok) return fail(MAD_EINVAL, "draft_tok required when T > 1");
    const size_t need = mad::accept_ws_bytes(B, T, V);
    if (!ws) return fail(MAD_EWS, "workspace required (%zu bytes)", need);
    if (ws_bytes < need) return fail(MAD_EWS, "workspace %zu bytes < %zu", ws_bytes, need);
    if (((uintptr_t)ws & 255u) != 0) return fail(MAD_EINVAL, "workspace not 256-byte aligned");
    mad::AcceptArgs a;
    memset(&a, 0, sizeof(a));
    a.logits = logits;
    a.draft = draft_tok;
    a.n_accept = n_accept;
    a.next_tok = next_tok;
    a.row_best = (uint64_t *)((char *)ws + (size_t)B * mad::kCounterStride * 4);   // inside the counter region
    a.counters = (unsigned *)ws;
    a.B = B;
    a.T = T;
    a.V = V;
    a.n_chunks = (V + mad::kAcceptChunk - 1) / mad::kAcceptChunk;
    const size_t esz = dtype == MAD_BF16 ? 2 : 4;
    a.vec16 = aligned16(logits) && ((size_t)V * esz) % 16 == 0;
    return hip_status(mad::launch_accept(a, dtype, (hipStream_t)stream), "accept launch");
}

int mad_accept_stochastic(const float *p, const float *q, const int32_t *draft_tok, const float *u, int B, int T,
                          int V, int32_t *n_accept, int32_t *next_tok, void *ws, size_t ws_bytes, void *stream) {
    if (B < 1 || B > MAD_MAX_BATCH) return fail(MAD_EINVAL, "B=%d outside [1, %d]", B, MAD_MAX_BATCH);
    if (T < 1 || T > 64) return fail(MAD_EINVAL, "T=%d outside [1, 64]", T);
    if (V < 1) return fail(MAD_EINVAL, "V=%d", V);
    if (!p || !u || !n_accept || !next_tok) return fail(MAD_EINVAL, "null p, u, n_accept or next_tok");
    if (T > 1 && (!q || !draft_tok)) return fail(MAD_EINVAL, "q and draft_tok required when T > 1");
    if ((size_t)B > (size_t)mad::kCounterLines) return fail(MAD_EINVAL, "B=%d", B);
    const size_t need = mad::stoch_ws_bytes(B, V);
    if (!ws) return fail(MAD_EWS, "workspace required (%zu bytes)", need);
    if (ws_bytes < need) return fail(MAD_EWS, "workspace %zu bytes < %zu", ws_bytes, need);
    if (((uintptr_t)ws & 255u) != 0) return fail(MAD_EINVAL, "workspace not 256-byte aligned");
    mad::StochArgs a;
    memset(&a, 0, sizeof(a));
    a.p = p;
    a.q = q;
    a.u = u;
    a.draft = draft_tok;
    a.n_accept = n_accept;
    a.next_tok = next_tok;
    a.counters = (unsigned *)ws;
    a.sums = (double *)((char *)ws + mad::kCounterRegionBytes);
    a.B = B;
    a.T = T;
    a.V = V;
    a.n_chunks = (V + mad::kAcceptChunk - 1) / mad::kAcceptChunk;
    a.vec16 = aligned16(p) && (T == 1 || aligned16(q)) && V % 4 == 0;
    return hip_status(mad::launch_stoch(a, (hipStream_t)stream), "stochastic accept launch");
}

}  // extern "C"
