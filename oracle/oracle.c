/*
 * oracle.c -- plain, slow, fp64 CPU reference for the MASW hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product (the HIP library or its
 * Python binding) may include, link, load or call this file.  Only the test
 * suite, the smoke check and the CPU-baseline leg of the benchmark use it.
 * It shares no code, header, table or constant with the GPU path.
 *
 * Every routine is the textbook definition written out in double precision,
 * without blocking, splitting, online rescaling or fusion, so that it can be
 * read against the paper by eye:
 *
 *   oracle_attend          softmax(s * q K^T) V over one explicit key list
 *                          (the draft reads its compact memory "sink + slots +
 *                          local window" with ordinary attention: Sec. 3.1,
 *                          Eq. three_part_memory and the local-window set; the
 *                          working set size S + W + floor(t/r)).
 *   oracle_attend_batched  the same for every (sequence, KV head) unit, GQA
 *                          head h reading KV head floor(h / G).
 *   oracle_verify          the target's parallel verification pass over its full
 *                          KV (Sec. 2.1 draft-verify paradigm, Sec. 3.3): query
 *                          t of the T = gamma+1 new tokens sees every prefix key
 *                          and the new tokens 0..t.
 *   oracle_project         mirrored projection y = x W_g^T (Sec. 3.2, the
 *                          projection equations K_g = H_g W_K,g, V_g = H_g W_V,g).
 *   oracle_rope            rotary position embedding at integer position ids;
 *                          a slot shares the position id of the raw token that
 *                          follows it (Sec. 3.2, memory update cycle).
 *   oracle_argmax          row argmax (ties -> lowest index, NaN ranks highest).
 *   oracle_accept_greedy   greedy (T = 0) accept/reject: accept the longest
 *                          prefix of drafted tokens equal to the target's argmax,
 *                          then emit one target token (Sec. 2.1, Eq. sd_speedup's
 *                          L_acc + 1; Sec. 4.1 greedy decoding).
 *   oracle_accept_stochastic  the rejection-sampling rule with caller-supplied
 *                          uniforms (Sec. 2.1, Sec. 3.3).
 *
 * Parallelism: OpenMP over independent units only; every unit is computed by
 * one thread in the order written here, so results do not depend on the
 * thread count.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>
#include <stdlib.h>

/* ------------------------------------------------------------------------ */
/* Attention over one explicit key list.                                     */
/*   q    [G][d]    G query vectors that share the key list                  */
/*   k, v [n][d]    keys and values                                          */
/*   o    [G][d]    output; lse [G] = log sum_j exp(s_j); wsum [G] = sum of  */
/*                  the normalised weights (a debug value, exactly 1 in real */
/*                  arithmetic) -- lse and wsum may be NULL.                 */
/* n == 0 gives o = 0, lse = -inf, wsum = 0.                                 */
/* ------------------------------------------------------------------------ */
void oracle_attend(int G, int d, const double *q, int n, const double *k, const double *v,
                   double scale, double *o, double *lse, double *wsum)
{
    double *s = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    for (int g = 0; g < G; ++g) {
        const double *qg = q + (size_t)g * d;
        double *og = o + (size_t)g * d;
        for (int c = 0; c < d; ++c) og[c] = 0.0;
        if (n == 0) {
            if (lse) lse[g] = -INFINITY;
            if (wsum) wsum[g] = 0.0;
            continue;
        }
        /* pass 1: scaled scores and their maximum */
        double m = -INFINITY;
        for (int j = 0; j < n; ++j) {
            double acc = 0.0;
            for (int c = 0; c < d; ++c) acc += qg[c] * k[(size_t)j * d + c];
            s[j] = scale * acc;
            if (s[j] > m) m = s[j];
        }
        /* pass 2: normaliser */
        double z = 0.0;
        for (int j = 0; j < n; ++j) z += exp(s[j] - m);
        /* pass 3: weighted sum of values with the normalised weights */
        double ws = 0.0;
        for (int j = 0; j < n; ++j) {
            double p = exp(s[j] - m) / z;
            ws += p;
            for (int c = 0; c < d; ++c) og[c] += p * v[(size_t)j * d + c];
        }
        if (lse) lse[g] = m + log(z);
        if (wsum) wsum[g] = ws;
    }
    free(s);
}

/* ------------------------------------------------------------------------ */
/* Batched attention over gathered key lists.                               */
/*   q [B][Hq][d]; k, v [B][Hkv][nmax][d] (rows 0..n[b]-1 used);            */
/*   o [B][Hq][d]; lse [B][Hq] (may be NULL).  Query head h reads KV head    */
/*   h / G with G = Hq / Hkv (consecutive query heads share a KV head).      */
/* ------------------------------------------------------------------------ */
void oracle_attend_batched(int B, int Hq, int Hkv, int d, const double *q,
                           int nmax, const int *n, const double *k, const double *v,
                           double scale, double *o, double *lse)
{
    const int G = Hq / Hkv;
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < Hkv; ++h) {
            size_t kv_off = ((size_t)b * Hkv + h) * (size_t)nmax * d;
            size_t q_off = ((size_t)b * Hq + (size_t)h * G) * d;
            oracle_attend(G, d, q + q_off, n[b], k + kv_off, v + kv_off, scale,
                          o + q_off, lse ? lse + (size_t)b * Hq + (size_t)h * G : NULL, NULL);
        }
}

/* ------------------------------------------------------------------------ */
/* Verify attention.  q [B][T][Hq][d]; k, v [B][Hkv][cap][d] with the T new  */
/* tokens already stored at rows len[b]-T .. len[b]-1.  Query t sees rows    */
/* 0 .. len[b]-T+t (the prefix and new tokens 0..t).                         */
/* o [B][T][Hq][d]; lse [B][T][Hq] (may be NULL).                            */
/* ------------------------------------------------------------------------ */
void oracle_verify(int B, int T, int Hq, int Hkv, int d, const double *q,
                   int cap, const int *len, const double *k, const double *v,
                   double scale, double *o, double *lse)
{
    const int G = Hq / Hkv;
    #pragma omp parallel for collapse(3) schedule(dynamic)
    for (int b = 0; b < B; ++b)
        for (int t = 0; t < T; ++t)
            for (int h = 0; h < Hkv; ++h) {
                size_t kv_off = ((size_t)b * Hkv + h) * (size_t)cap * d;
                size_t q_off = (((size_t)b * T + t) * Hq + (size_t)h * G) * d;
                int n = len[b] - T + t + 1;
                oracle_attend(G, d, q + q_off, n, k + kv_off, v + kv_off, scale, o + q_off,
                              lse ? lse + ((size_t)b * T + t) * Hq + (size_t)h * G : NULL, NULL);
            }
}

/* ------------------------------------------------------------------------ */
/* Mirrored projection: y[r][c] = sum_i x[r][i] * w[c][i].                   */
/*   x [R][D] slot hidden states; w [N][D] (one row per output feature, the  */
/*   K_g rows then the V_g rows); y [R][N].                                  */
/* ------------------------------------------------------------------------ */
void oracle_project(int R, int D, int N, const double *x, const double *w, double *y)
{
    #pragma omp parallel for collapse(2)
    for (int r = 0; r < R; ++r)
        for (int c = 0; c < N; ++c) {
            double acc = 0.0;
            for (int i = 0; i < D; ++i) acc += x[(size_t)r * D + i] * w[(size_t)c * D + i];
            y[(size_t)r * N + c] = acc;
        }
}

/* ------------------------------------------------------------------------ */
/* Rotary position embedding, rotate-half pairing, in place.                 */
/*   k [R][H][d]; pos [R].  For i < d/2, with theta_i = base^(-2i/d) and      */
/*   a = pos * theta_i:                                                      */
/*     k'[i]       = k[i] cos a - k[i + d/2] sin a                           */
/*     k'[i + d/2] = k[i + d/2] cos a + k[i] sin a                           */
/* ------------------------------------------------------------------------ */
void oracle_rope(int R, int H, int d, double *k, const int *pos, double base)
{
    const int half = d / 2;
    for (int r = 0; r < R; ++r)
        for (int h = 0; h < H; ++h) {
            double *kh = k + ((size_t)r * H + h) * d;
            for (int i = 0; i < half; ++i) {
                double theta = pow(base, -2.0 * (double)i / (double)d);
                double a = (double)pos[r] * theta;
                double c = cos(a), s = sin(a);
                double x0 = kh[i], x1 = kh[i + half];
                kh[i] = x0 * c - x1 * s;
                kh[i + half] = x1 * c + x0 * s;
            }
        }
}

/* ------------------------------------------------------------------------ */
/* Row argmax over float logits [rows][V]: the index of the largest value;   */
/* ties go to the lowest index; a NaN ranks above every number (the first    */
/* NaN wins).                                                                */
/* ------------------------------------------------------------------------ */
static int better(float a, int ia, float b, int ib)
{
    int an = isnan(a), bn = isnan(b);
    if (an || bn) {
        if (an && bn) return ia < ib;
        return an;
    }
    if (a != b) return a > b;
    return ia < ib;
}

void oracle_argmax(int rows, int V, const float *logits, int *idx)
{
    for (int r = 0; r < rows; ++r) {
        const float *x = logits + (size_t)r * V;
        int best = 0;
        for (int j = 1; j < V; ++j)
            if (better(x[j], j, x[best], best)) best = j;
        idx[r] = best;
    }
}

/* ------------------------------------------------------------------------ */
/* Greedy accept.  logits [B][T][V] are the target's scores at the T verify  */
/* positions; draft [B][T-1] are the drafted tokens.  For each sequence:     */
/*   a    = first i < T-1 with draft[i] != argmax(logits[i]), else T-1       */
/*   next = argmax(logits[a])  (correction token, or bonus token if a = T-1) */
/* n_accept[b] = a; the iteration emits a + 1 tokens.                        */
/* ------------------------------------------------------------------------ */
void oracle_accept_greedy(int B, int T, int V, const float *logits, const int *draft,
                          int *n_accept, int *next)
{
    int *am = (int *)malloc(sizeof(int) * (size_t)B * T);
    oracle_argmax(B * T, V, logits, am);
    for (int b = 0; b < B; ++b) {
        int a = 0;
        while (a < T - 1 && draft[(size_t)b * (T - 1) + a] == am[(size_t)b * T + a]) ++a;
        n_accept[b] = a;
        next[b] = am[(size_t)b * T + a];
    }
    free(am);
}

/* ------------------------------------------------------------------------ */
/* Stochastic accept/reject (the standard speculative-sampling rule that the */
/* target applies, Sec. 2.1 and Sec. 3.3; it keeps the target's output       */
/* distribution).  p [B][T][V] target probabilities, q [B][T-1][V] draft     */
/* probabilities, draft [B][T-1] drafted tokens, u [B][T] uniforms in [0,1). */
/* For each sequence, in double precision:                                   */
/*   a = first i < T-1 with NOT (u[i] * q_i(x_i) < p_i(x_i)), x_i = draft[i], */
/*       else T-1 (every drafted token accepted); a drafted value outside    */
/*       [0, V) is not a token and is rejected;                               */
/*   the emitted token is drawn by inverse CDF with u[T-1] from              */
/*     r(v) = max(0, p_a(v) - q_a(v))  after a rejection (a < T-1), or       */
/*     r(v) = p_a(v)                   when everything was accepted,         */
/*   i.e. the smallest v with r(0) + ... + r(v) > u[T-1] * Z, Z = sum_v r(v) */
/*   (summed in index order).  If Z == 0 the draw uses p_a; if no index       */
/*   qualifies (u[T-1] * Z >= the running total) the last v with r(v) > 0.   */
/* n_accept[b] = a, next[b] = the drawn token.                               */
/* ------------------------------------------------------------------------ */
static int inverse_cdf(int V, const float *p, const float *q, double u)
{
    double Z = 0.0;
    for (int v = 0; v < V; ++v) {
        double r = q ? (double)p[v] - (double)q[v] : (double)p[v];
        if (r > 0.0) Z += r;
    }
    if (Z == 0.0 && q) return inverse_cdf(V, p, NULL, u);
    const double t = u * Z;
    double c = 0.0;
    int last = 0;
    for (int v = 0; v < V; ++v) {
        double r = q ? (double)p[v] - (double)q[v] : (double)p[v];
        if (r <= 0.0) continue;
        c += r;
        last = v;
        if (c > t) return v;
    }
    return last;
}

void oracle_accept_stochastic(int B, int T, int V, const float *p, const float *q, const int *draft,
                              const float *u, int *n_accept, int *next)
{
    for (int b = 0; b < B; ++b) {
        const float *ub = u + (size_t)b * T;
        int a = 0;
        while (a < T - 1) {
            const int x = draft[(size_t)b * (T - 1) + a];
            if (x < 0 || x >= V) break;           /* not a token: rejected */
            const double px = p[((size_t)b * T + a) * V + x];
            const double qx = q[((size_t)b * (T - 1) + a) * V + x];
            if (!((double)ub[a] * qx < px)) break;
            ++a;
        }
        n_accept[b] = a;
        const float *pa = p + ((size_t)b * T + a) * V;
        const float *qa = a < T - 1 ? q + ((size_t)b * (T - 1) + a) * V : NULL;
        next[b] = inverse_cdf(V, pa, qa, (double)ub[T - 1]);
    }
}

/* Number of OpenMP threads the batched routines use (1 without OpenMP). */
#ifdef _OPENMP
#include <omp.h>
int oracle_num_threads(void) { return omp_get_max_threads(); }
/* threads of the parallel loops from now on (timing of the oracle itself only) */
void oracle_set_threads(int n) { if (n > 0) omp_set_num_threads(n); }
#else
int oracle_num_threads(void) { return 1; }
void oracle_set_threads(int n) { (void)n; }
#endif
