/*
 * CPU oracle: forward pass of the decoder-only transformer that DVI splits
 * into a draft path (layers 1..k) and a target path (layers k+1..L)
 * (paper Section 3.1, "Preliminaries and Notation").
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may load this file's
 * library; only tests, the smoke check and the CPU-baseline leg of the
 * benchmark do.
 *
 * The paper names the backbone only as a decoder-only language model; the
 * layer below is the Llama-style pre-norm block the measured workloads name
 * (RMSNorm, rotary position embedding, SwiGLU MLP, no biases):
 *
 *   a  = RMSNorm(h; g_attn)
 *   q,k,v = Wq a, Wk a, Wv a ;  q,k rotated by position p (rotate-half RoPE)
 *   o  = softmax(q K^T / sqrt(hd)) V   over keys 0..p  (head -> kv head by group)
 *   h += Wo o
 *   b  = RMSNorm(h; g_mlp)
 *   h += Wd (silu(Wg b) * (Wu b))
 *
 * Everything is float64.  Weights are read as their exact values (bf16 bit
 * patterns widened bit-for-bit, or float32).  Every output element is one sum
 * taken in increasing index order, computed by the same code whatever the
 * number of rows processed together, so processing a block of tokens gives
 * bitwise the same numbers as processing them one at a time.  Build without
 * -ffast-math and with -ffp-contract=off.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t n_layers, d, n_heads, n_kv_heads, head_dim, ffn, vocab, bf16;
    double eps, theta;
    const void *tok_emb;     /* [V, d] */
    const void *final_norm;  /* [d] */
    const void *lm_head;     /* [V, d]  W^(V), also the frozen base W^(S) of the draft head */
    const void *const *attn_norm, *const *wq, *const *wk, *const *wv, *const *wo;
    const void *const *mlp_norm, *const *wg, *const *wu, *const *wd;
} orc_model;

static inline double wget(const void *w, int bf16, size_t i) {
    if (bf16) {
        uint32_t u = ((uint32_t)((const uint16_t *)w)[i]) << 16;
        float f;
        memcpy(&f, &u, 4);
        return (double)f;
    }
    return (double)((const float *)w)[i];
}

/*
 * Y[t][j] = sum_{c=0}^{K-1} W[j][c] * X[t][c]   (W row-major [N][K]),
 * each sum taken in increasing c, one multiply and one add per term (no
 * fused multiply-add: built with -ffp-contract=off).  Rows of W are widened
 * to double RB at a time and tokens are taken TB at a time only to keep the
 * CPU busy: the TB sums of a row are independent, so they may share SIMD
 * lanes, and every Y[t][j] still sees exactly the same sequence of
 * multiplies and adds.  The result therefore does not depend on the block
 * sizes, the thread count, the SIMD width or how many tokens are processed
 * together.  An AVX2 body is used where the CPU has it; the plain body
 * evaluates the same operations in the same order.
 */
#include <immintrin.h>
#define TB 8      /* tokens per SIMD block (two 4-wide vectors) */
#define TSUB 4    /* token blocks sharing one widened row panel */
#define RB 4      /* rows per panel */
#define RV 8      /* rows per panel of the one-token product */

/* dst[c] = W[row][c] as double, c < K */
__attribute__((target("avx2")))
static void widen_row_avx2(const void *W, int bf16, size_t row, int K, double *dst) {
    int c = 0;
    if (bf16) {
        const uint16_t *src = (const uint16_t *)W + row * K;
        for (; c + 8 <= K; c += 8) {
            const __m256i w = _mm256_slli_epi32(_mm256_cvtepu16_epi32(_mm_loadu_si128((const __m128i *)(src + c))), 16);
            const __m256 f = _mm256_castsi256_ps(w);
            _mm256_storeu_pd(dst + c, _mm256_cvtps_pd(_mm256_castps256_ps128(f)));
            _mm256_storeu_pd(dst + c + 4, _mm256_cvtps_pd(_mm256_extractf128_ps(f, 1)));
        }
    } else {
        const float *src = (const float *)W + row * K;
        for (; c + 4 <= K; c += 4) _mm256_storeu_pd(dst + c, _mm256_cvtps_pd(_mm_loadu_ps(src + c)));
    }
    for (; c < K; ++c) dst[c] = wget(W, bf16, row * K + c);
}

static void widen_row_plain(const void *W, int bf16, size_t row, int K, double *dst) {
    for (int c = 0; c < K; ++c) dst[c] = wget(W, bf16, row * K + c);
}

/* acc[jj][t] = sum_c P[jj][c] * XT[c*xs + t], jj < RB, t < TB; P is [RB][K] */
__attribute__((target("avx2")))
static void panel_avx2(const double *P, int K, const double *XT, int xs, double (*acc)[TB]) {
    const double *p0 = P, *p1 = P + K, *p2 = P + 2 * (size_t)K, *p3 = P + 3 * (size_t)K;
    __m256d a00 = _mm256_setzero_pd(), a01 = _mm256_setzero_pd(), a10 = _mm256_setzero_pd(), a11 = _mm256_setzero_pd();
    __m256d a20 = _mm256_setzero_pd(), a21 = _mm256_setzero_pd(), a30 = _mm256_setzero_pd(), a31 = _mm256_setzero_pd();
    for (int c = 0; c < K; ++c) {
        const __m256d x0 = _mm256_loadu_pd(XT + (size_t)c * xs), x1 = _mm256_loadu_pd(XT + (size_t)c * xs + 4);
        __m256d w = _mm256_broadcast_sd(p0 + c);
        a00 = _mm256_add_pd(a00, _mm256_mul_pd(w, x0));
        a01 = _mm256_add_pd(a01, _mm256_mul_pd(w, x1));
        w = _mm256_broadcast_sd(p1 + c);
        a10 = _mm256_add_pd(a10, _mm256_mul_pd(w, x0));
        a11 = _mm256_add_pd(a11, _mm256_mul_pd(w, x1));
        w = _mm256_broadcast_sd(p2 + c);
        a20 = _mm256_add_pd(a20, _mm256_mul_pd(w, x0));
        a21 = _mm256_add_pd(a21, _mm256_mul_pd(w, x1));
        w = _mm256_broadcast_sd(p3 + c);
        a30 = _mm256_add_pd(a30, _mm256_mul_pd(w, x0));
        a31 = _mm256_add_pd(a31, _mm256_mul_pd(w, x1));
    }
    _mm256_storeu_pd(acc[0], a00); _mm256_storeu_pd(acc[0] + 4, a01);
    _mm256_storeu_pd(acc[1], a10); _mm256_storeu_pd(acc[1] + 4, a11);
    _mm256_storeu_pd(acc[2], a20); _mm256_storeu_pd(acc[2] + 4, a21);
    _mm256_storeu_pd(acc[3], a30); _mm256_storeu_pd(acc[3] + 4, a31);
}

static void panel_plain(const double *P, int K, const double *XT, int xs, double (*acc)[TB]) {
    for (int jj = 0; jj < RB; ++jj)
        for (int t = 0; t < TB; ++t) {
            double s = 0.0;
            for (int c = 0; c < K; ++c) s += P[(size_t)jj * K + c] * XT[(size_t)c * xs + t];
            acc[jj][t] = s;
        }
}

static void matmul(const void *W, int bf16, int N, int K, int n, const double *X, double *Y) {
    const int avx2 = __builtin_cpu_supports("avx2");
    if (n == 1) {
        /* one token: RV independent row sums, each in increasing c */
#pragma omp parallel
        {
            double *P = (double *)malloc(sizeof(double) * (size_t)RV * K);
#pragma omp for schedule(static)
            for (int j = 0; j < N; j += RV) {
                const int jn = N - j < RV ? N - j : RV;
                for (int jj = 0; jj < jn; ++jj)
                    (avx2 ? widen_row_avx2 : widen_row_plain)(W, bf16, (size_t)(j + jj), K, P + (size_t)jj * K);
                double acc[RV] = {0.0};
                for (int c = 0; c < K; ++c) {
                    const double xc = X[c];
                    for (int jj = 0; jj < RV; ++jj)
                        if (jj < jn) acc[jj] += P[(size_t)jj * K + c] * xc;
                }
                for (int jj = 0; jj < jn; ++jj) Y[j + jj] = acc[jj];
            }
            free(P);
        }
        return;
    }
    const int TBB = TB * TSUB;
    double *XT = (double *)malloc(sizeof(double) * (size_t)K * TBB);
    for (int t0 = 0; t0 < n; t0 += TBB) {
        const int nb = n - t0 < TBB ? n - t0 : TBB;
        /* X block transposed to [K][TBB]; lanes past the block are zero and never stored */
        for (int c = 0; c < K; ++c)
            for (int t = 0; t < TBB; ++t) XT[(size_t)c * TBB + t] = t < nb ? X[(size_t)(t0 + t) * K + c] : 0.0;
#pragma omp parallel
        {
            double *P = (double *)calloc((size_t)RB * K, sizeof(double));
#pragma omp for schedule(static)
            for (int j = 0; j < N; j += RB) {
                const int jn = N - j < RB ? N - j : RB;
                for (int jj = 0; jj < RB; ++jj) {
                    if (jj < jn)
                        (avx2 ? widen_row_avx2 : widen_row_plain)(W, bf16, (size_t)(j + jj), K, P + (size_t)jj * K);
                    else
                        memset(P + (size_t)jj * K, 0, sizeof(double) * K);
                }
                for (int sb = 0; sb < TSUB && sb * TB < nb; ++sb) {
                    double acc[RB][TB];
                    (avx2 ? panel_avx2 : panel_plain)(P, K, XT + sb * TB, TBB, acc);
                    for (int jj = 0; jj < jn; ++jj)
                        for (int t = 0; t < TB && sb * TB + t < nb; ++t) Y[(size_t)(t0 + sb * TB + t) * N + j + jj] = acc[jj][t];
                }
            }
            free(P);
        }
    }
    free(XT);
}

/* y = x / sqrt(mean(x^2) + eps) * g */
static void rmsnorm(const double *x, const void *g, int bf16, int d, double eps, double *y) {
    double ss = 0.0;
    for (int i = 0; i < d; ++i) ss += x[i] * x[i];
    double inv = 1.0 / sqrt(ss / (double)d + eps);
    for (int i = 0; i < d; ++i) y[i] = x[i] * inv * wget(g, bf16, i);
}

/*
 * Rotary embedding, rotate-half convention: for i < hd/2 the pair
 * (x[i], x[i+hd/2]) is rotated by the angle p * theta^(-2i/hd).
 */
static void rope(double *x, int hd, int pos, double theta) {
    int half = hd / 2;
    for (int i = 0; i < half; ++i) {
        double ang = (double)pos * pow(theta, -2.0 * (double)i / (double)hd);
        double c = cos(ang), s = sin(ang);
        double a = x[i], b = x[i + half];
        x[i] = a * c - b * s;
        x[i + half] = a * s + b * c;
    }
}

static inline double silu(double x) { return x / (1.0 + exp(-x)); }

/* h[t][:] = E[tok[t]][:] */
void orc_embed(const orc_model *m, const int32_t *tok, int n, double *h) {
    for (int t = 0; t < n; ++t)
        for (int i = 0; i < m->d; ++i) h[(size_t)t * m->d + i] = wget(m->tok_emb, m->bf16, (size_t)tok[t] * m->d + i);
}

/*
 * Run layers [l0, l1) (0-based) on n consecutive tokens of one sequence at
 * positions pos0 .. pos0+n-1.  h is [n][d] in/out.  kc/vc are this
 * sequence's caches, [n_layers][s_max][kv_dim]; the block's own keys and
 * values are written before attention, so token t sees keys 0..pos0+t.
 */
void orc_layers(const orc_model *m, double *kc, double *vc, int s_max, int pos0, int n,
                int l0, int l1, double *h) {
    const int d = m->d, H = m->n_heads, Hkv = m->n_kv_heads, hd = m->head_dim, F = m->ffn;
    const int qd = H * hd, kvd = Hkv * hd, grp = H / Hkv;
    double *a = (double *)malloc(sizeof(double) * (size_t)n * d);
    double *q = (double *)malloc(sizeof(double) * (size_t)n * qd);
    double *k = (double *)malloc(sizeof(double) * (size_t)n * kvd);
    double *v = (double *)malloc(sizeof(double) * (size_t)n * kvd);
    double *o = (double *)malloc(sizeof(double) * (size_t)n * qd);
    double *y = (double *)malloc(sizeof(double) * (size_t)n * d);
    double *gt = (double *)malloc(sizeof(double) * (size_t)n * F);
    double *up = (double *)malloc(sizeof(double) * (size_t)n * F);
    const double scale = 1.0 / sqrt((double)hd);

    for (int l = l0; l < l1; ++l) {
        double *K = kc + (size_t)l * s_max * kvd;
        double *V = vc + (size_t)l * s_max * kvd;
        for (int t = 0; t < n; ++t) rmsnorm(h + (size_t)t * d, m->attn_norm[l], m->bf16, d, m->eps, a + (size_t)t * d);
        matmul(m->wq[l], m->bf16, qd, d, n, a, q);
        matmul(m->wk[l], m->bf16, kvd, d, n, a, k);
        matmul(m->wv[l], m->bf16, kvd, d, n, a, v);
        for (int t = 0; t < n; ++t) {
            for (int hh = 0; hh < H; ++hh) rope(q + (size_t)t * qd + hh * hd, hd, pos0 + t, m->theta);
            for (int hh = 0; hh < Hkv; ++hh) rope(k + (size_t)t * kvd + hh * hd, hd, pos0 + t, m->theta);
            memcpy(K + (size_t)(pos0 + t) * kvd, k + (size_t)t * kvd, sizeof(double) * kvd);
            memcpy(V + (size_t)(pos0 + t) * kvd, v + (size_t)t * kvd, sizeof(double) * kvd);
        }
#pragma omp parallel for schedule(dynamic) collapse(2)
        for (int t = 0; t < n; ++t) {
            for (int hh = 0; hh < H; ++hh) {
                const int p = pos0 + t, kvh = hh / grp;
                const double *qv = q + (size_t)t * qd + hh * hd;
                double *s = (double *)malloc(sizeof(double) * (size_t)(p + 1));
                double mx = -INFINITY;
                for (int j = 0; j <= p; ++j) {
                    const double *kj = K + (size_t)j * kvd + kvh * hd;
                    double dot = 0.0;
                    for (int e = 0; e < hd; ++e) dot += qv[e] * kj[e];
                    s[j] = dot * scale;
                    if (s[j] > mx) mx = s[j];
                }
                double z = 0.0;
                for (int j = 0; j <= p; ++j) { s[j] = exp(s[j] - mx); z += s[j]; }
                double *ov = o + (size_t)t * qd + hh * hd;
                for (int e = 0; e < hd; ++e) ov[e] = 0.0;
                for (int j = 0; j <= p; ++j) {
                    const double w = s[j] / z;
                    const double *vj = V + (size_t)j * kvd + kvh * hd;
                    for (int e = 0; e < hd; ++e) ov[e] += w * vj[e];
                }
                free(s);
            }
        }
        matmul(m->wo[l], m->bf16, d, qd, n, o, y);
        for (size_t i = 0; i < (size_t)n * d; ++i) h[i] += y[i];
        for (int t = 0; t < n; ++t) rmsnorm(h + (size_t)t * d, m->mlp_norm[l], m->bf16, d, m->eps, a + (size_t)t * d);
        matmul(m->wg[l], m->bf16, F, d, n, a, gt);
        matmul(m->wu[l], m->bf16, F, d, n, a, up);
        for (size_t i = 0; i < (size_t)n * F; ++i) gt[i] = silu(gt[i]) * up[i];
        matmul(m->wd[l], m->bf16, d, F, n, gt, y);
        for (size_t i = 0; i < (size_t)n * d; ++i) h[i] += y[i];
    }
    free(a); free(q); free(k); free(v); free(o); free(y); free(gt); free(up);
}

/* hn[t] = RMSNorm(h[t]; g_final): the input both vocabulary heads read */
void orc_final_norm(const orc_model *m, const double *h, int n, double *hn) {
    for (int t = 0; t < n; ++t) rmsnorm(h + (size_t)t * m->d, m->final_norm, m->bf16, m->d, m->eps, hn + (size_t)t * m->d);
}

/* Target head, logits^phi = W^(V) hn  (Section 3.1). out [n][V] */
void orc_target_logits(const orc_model *m, const double *hn, int n, double *out) {
    matmul(m->lm_head, m->bf16, m->vocab, m->d, n, hn, out);
}

/*
 * Draft head, logits^theta = (W^(S) + gamma A_s B_s) hn  (Section 3.1), with
 * W^(S) = W^(V).  Evaluated as W hn + gamma * A_s (B_s hn):
 *   u[c] = sum_i B_s[c][i] hn[i]              (B_s [r][d])
 *   out[v] = (W hn)[v] + gamma * sum_c A_s[v][c] u[c]   (A_s [V][r])
 */
void orc_draft_logits(const orc_model *m, const double *hn, int n, const double *A, const double *B,
                      int r, double gamma, double *out) {
    const int d = m->d, V = m->vocab;
    matmul(m->lm_head, m->bf16, V, d, n, hn, out);
    double *u = (double *)malloc(sizeof(double) * (size_t)r);
    for (int t = 0; t < n; ++t) {
        const double *x = hn + (size_t)t * d;
        for (int c = 0; c < r; ++c) {
            double s = 0.0;
            for (int i = 0; i < d; ++i) s += B[(size_t)c * d + i] * x[i];
            u[c] = s;
        }
        double *o = out + (size_t)t * V;
        for (int vv = 0; vv < V; ++vv) {
            double s = 0.0;
            for (int c = 0; c < r; ++c) s += A[(size_t)vv * r + c] * u[c];
            o[vv] += gamma * s;
        }
    }
    free(u);
}
