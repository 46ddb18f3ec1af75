/*
 * CPU oracle for Jacobi decoding with a KV cache -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg load this
 * library. The GPU product path never calls it, and it shares no code with the GPU path:
 * the two sides implement the same written contract independently.
 *
 * What it computes (CLLMs, Section 3.1 "Preliminary: Jacobi Decoding"):
 *   - greedy autoregressive decoding, eq. (ar_decoding): y_i = argmax_y p(y | y_<i, x);
 *   - the Jacobi fixed-point iteration, eq. (jacobi_decoding), where one causal forward pass
 *     over the n-token block yields all n argmaxes at once;
 *   - Jacobi decoding with a KV cache, Appendix algorithm "Jacobi Decoding with KV Cache":
 *     prefill gives the first token, each iteration forwards the unfixed block against the
 *     cache, accepts the converged prefix, keeps its K/V and shrinks the state.
 *
 * The paper does not print the architecture of its 7B models (Section 4 names LLaMA-2-7B and
 * Deepseek-coder-7B). The decoder below is the LLaMA-style one: pre-norm RMSNorm,
 * rotate-half RoPE, causal softmax attention, SwiGLU FFN, untied LM head, no biases.
 *
 * Precision: every intermediate is a double. With round_bf16 set (the bf16 precision contract),
 * the weights hold bf16 values and the keys and values written to the cache (after RoPE) are
 * rounded to bfloat16 (round to nearest, ties to even); no other value is rounded. Each
 * RMSNorm is applied as written, x / sqrt(mean(x^2) + eps) (.) g, and its output is the input
 * of the product that follows. Argmax decisions are taken on the logits rounded to fp32, the
 * precision the GPU path decides in; ties go to the lowest id.
 *
 * Reading of the acceptance rule (the algorithm's fast-forward count): the block z holds the
 * known-correct pending token at index 0, the model's output at row k is the prediction for
 * the token after z[k], and the accepted length is a = 1 + the number of leading k >= 1 with
 * z[k] equal to the prediction of row k-1. The printed set {0, .., len-1} compared without a
 * shift would accept nothing and stall, so the shifted comparison is used.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct orc_config {
    int32_t n_layers, d_model, n_heads, head_dim, ffn_dim, vocab;
    double rms_eps, rope_base;
    int32_t round_bf16;
} orc_config;

/* Weights as fp32 arrays, row-major [out][in]; the caller keeps them alive. */
typedef struct orc_model {
    orc_config c;
    const float *embed, *final_norm, *lm_head;
    const float **attn_norm, **wq, **wk, **wv, **wo, **ffn_norm, **wg, **wu, **wd;
} orc_model;

/* Decoding state of one sequence: the KV cache and the committed length. */
typedef struct orc_state {
    const orc_model *m;
    int32_t max_ctx;
    double *k, *v;   /* [layer][pos][d_model] */
    int32_t L;       /* committed length (prompt + accepted tokens) */
    int32_t pending; /* the next token, known correct, not yet in the cache */
    int32_t prefilled;
} orc_state;

/* Initial-guess and iteration policies. */
typedef struct orc_guess_spec {
    int32_t policy;        /* 0 uniform ids, 1 corrupted stream, 2 corrupted stream re-drawn every step */
    int32_t block_policy;  /* 0 shrink (the algorithm as printed), 1 slide (window of n) */
    const int32_t *stream; /* reference continuation, indexed by output position */
    int32_t stream_len;
    uint64_t thr53;        /* corrupt when the top 53 bits of the draw are below thr53 (p * 2^53) */
    uint64_t seed;
} orc_guess_spec;

/* Optional trajectory of a decode: per iteration t < cap the committed length L before the
 * iteration, the output position e of the block's first token, the first output position b0
 * of the current block (shrink policy; the slide policy keeps b0 = e), and the block tokens z
 * and predictions pred (stride n; entries past the iteration's m are left unwritten). */
typedef struct orc_traj {
    int32_t *L, *e, *b0, *z, *pred;
    int32_t cap;
} orc_traj;

typedef struct orc_stats {
    int64_t steps, blocks, tokens;
    int64_t accept_hist[257];
} orc_stats;

int32_t orc_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------------------- */
/* Scalar helpers                                                                         */

/* Nearest bfloat16 value of x (8 significant bits, ties to even), from the definition of the
 * format: scale the significand to 8 bits, round to the nearest integer (the default rounding
 * mode rounds ties to even), scale back. Subnormals have a fixed spacing of 2^-133. */
double orc_bf16(double x) {
    if (x == 0.0 || !isfinite(x)) return x;
    int e;
    double f = frexp(x, &e); /* x = f * 2^e, 0.5 <= |f| < 1 */
    double r;
    if (e - 1 < -126) {
        r = ldexp(nearbyint(ldexp(x, 133)), -133);
    } else {
        r = ldexp(nearbyint(ldexp(f, 8)), e - 8);
    }
    if (fabs(r) > 3.3895313892515355e38) r = copysign(INFINITY, x);
    return r;
}

/* Rounding of a key or value stored in the cache (bf16 contract). */
static inline double rnd_cache(const orc_model *m, double x) { return m->c.round_bf16 ? orc_bf16(x) : x; }

/* RMSNorm row factor: 1 / sqrt(mean(x^2) + eps). */
double orc_rms_inv(const double *x, int32_t n, double eps) {
    double ss = 0.0;
    for (int32_t k = 0; k < n; ++k) ss += x[k] * x[k];
    return 1.0 / sqrt(ss / n + eps);
}

/* RMSNorm: out_k = x_k / sqrt(mean(x^2) + eps) * g_k (rounded to bf16 if asked). */
void orc_rmsnorm(const double *x, int32_t n, const float *g, double eps, int32_t round_bf16, double *out) {
    double inv = orc_rms_inv(x, n, eps);
    for (int32_t k = 0; k < n; ++k) {
        double y = x[k] * inv * (double)g[k];
        out[k] = round_bf16 ? orc_bf16(y) : y;
    }
}

/* Rotate-half RoPE at absolute position t: the pair (x_j, x_{j+hd/2}) is rotated by the angle
 * t * base^(-2j/hd). */
void orc_rope(double *x, int32_t hd, int32_t t, double base) {
    int32_t h2 = hd / 2;
    for (int32_t j = 0; j < h2; ++j) {
        double theta = pow(base, -2.0 * (double)j / (double)hd);
        double ang = (double)t * theta;
        double c = cos(ang), s = sin(ang);
        double a = x[j], b = x[j + h2];
        x[j] = a * c - b * s;
        x[j + h2] = b * c + a * s;
    }
}

/* Softmax attention of one query over n_keys keys (rows of K and V, stride ld):
 * out = sum_u softmax_u(q . k_u / sqrt(hd)) v_u. */
void orc_attention_row(const double *q, const double *K, const double *V, int32_t n_keys, int32_t ld,
                       int32_t hd, double *out) {
    double *s = (double *)malloc(sizeof(double) * (size_t)(n_keys > 0 ? n_keys : 1));
    double mx = -INFINITY;
    double scale = 1.0 / sqrt((double)hd);
    for (int32_t u = 0; u < n_keys; ++u) {
        double acc = 0.0;
        for (int32_t d = 0; d < hd; ++d) acc += q[d] * K[(size_t)u * ld + d];
        s[u] = acc * scale;
        if (s[u] > mx) mx = s[u];
    }
    double den = 0.0;
    for (int32_t u = 0; u < n_keys; ++u) {
        s[u] = exp(s[u] - mx);
        den += s[u];
    }
    for (int32_t d = 0; d < hd; ++d) {
        double acc = 0.0;
        for (int32_t u = 0; u < n_keys; ++u) acc += s[u] * V[(size_t)u * ld + d];
        out[d] = acc / den;
    }
    free(s);
}

double orc_silu(double x) { return x / (1.0 + exp(-x)); }

/* Greedy choice over one row of logits, decided on the fp32 values; ties go to the lowest id.
 * Returns -1 if a logit is NaN. */
int32_t orc_argmax(const double *logits, int32_t n) {
    int32_t best = 0;
    float bv = (float)logits[0];
    if (isnan(bv)) return -1;
    for (int32_t v = 1; v < n; ++v) {
        float x = (float)logits[v];
        if (isnan(x)) return -1;
        if (x > bv) {
            bv = x;
            best = v;
        }
    }
    return best;
}

/* Accepted length of one iteration: 1 + leading matches z[k] == pred[k-1] for k in [1, m). */
int32_t orc_accept_len(const int32_t *z, const int32_t *pred, int32_t m) {
    int32_t a = 1;
    while (a < m && z[a] == pred[a - 1]) ++a;
    return a;
}

/* SplitMix64 output function on state x (Steele, Lea and Flood, OOPSLA 2014). */
uint64_t orc_mix(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Guess for output position t of sequence seq at draw d. Without a stream: a uniform id.
 * With a stream: stream[t], replaced by a uniform id other than stream[t] when the draw
 * falls below the corruption threshold. */
int32_t orc_guess(const orc_guess_spec *g, int32_t seq, int32_t t, int32_t d, int32_t vocab) {
    uint64_t h = orc_mix(orc_mix(orc_mix(orc_mix(g->seed) ^ (uint64_t)(uint32_t)seq) ^ (uint64_t)(uint32_t)t) ^
                         (uint64_t)(uint32_t)d);
    if (!g->stream || g->policy == 0) return (int32_t)(((h >> 32) * (uint64_t)(uint32_t)vocab) >> 32);
    int32_t s = (t < g->stream_len) ? g->stream[t] : 0;
    if ((h >> 11) < g->thr53) {
        uint64_t h2 = orc_mix(h);
        int32_t r = (int32_t)(((h2 >> 32) * (uint64_t)(uint32_t)(vocab - 1)) >> 32);
        return (int32_t)(((int64_t)s + 1 + r) % vocab);
    }
    return s;
}

/* ------------------------------------------------------------------------------------- */
/* Model                                                                                  */

/* tensors: embed, then per layer (attn_norm, wq, wk, wv, wo, ffn_norm, w_gate, w_up, w_down),
 * then final_norm, lm_head. */
orc_model *orc_model_new(const orc_config *c, const float *const *tensors) {
    orc_model *m = (orc_model *)calloc(1, sizeof(orc_model));
    if (!m) return NULL;
    m->c = *c;
    int32_t L = c->n_layers;
    const float ***slots[9] = {&m->attn_norm, &m->wq, &m->wk, &m->wv, &m->wo, &m->ffn_norm, &m->wg, &m->wu, &m->wd};
    for (int s = 0; s < 9; ++s) *slots[s] = (const float **)calloc((size_t)(L > 0 ? L : 1), sizeof(float *));
    m->embed = tensors[0];
    for (int32_t l = 0; l < L; ++l)
        for (int s = 0; s < 9; ++s) (*slots[s])[l] = tensors[1 + 9 * l + s];
    m->final_norm = tensors[1 + 9 * L];
    m->lm_head = tensors[2 + 9 * L];
    return m;
}

void orc_model_free(orc_model *m) {
    if (!m) return;
    free(m->attn_norm); free(m->wq); free(m->wk); free(m->wv); free(m->wo);
    free(m->ffn_norm); free(m->wg); free(m->wu); free(m->wd);
    free(m);
}

/* y[r][o] = sum_i a[r][i] * W[o][i] for rows r < rows; every sum is taken over i in increasing
 * order, one multiply and one add per term (no fused multiply-add: the build has none). For
 * speed each thread owns a contiguous range of outputs o and takes the rows eight at a time
 * (copied side by side, so that one pass over a weight row feeds eight independent sums); the
 * value of every sum is that of the plain loop. */
#define ORC_ROWS 8
static void linear(const double *a, int32_t rows, const float *W, int32_t in, int32_t out, double *y) {
#pragma omp parallel
    {
#ifdef _OPENMP
        const int nt = omp_get_num_threads(), t = omp_get_thread_num();
#else
        const int nt = 1, t = 0;
#endif
        const int32_t o0 = (int32_t)((int64_t)out * t / nt), o1 = (int32_t)((int64_t)out * (t + 1) / nt);
        double *xt = (double *)malloc(sizeof(double) * (size_t)(in > 0 ? in : 1) * ORC_ROWS);
        for (int32_t r0 = 0; xt && r0 < rows; r0 += ORC_ROWS) {
            const int32_t nr = rows - r0 < ORC_ROWS ? rows - r0 : ORC_ROWS;
            for (int32_t i = 0; i < in; ++i)
                for (int32_t r = 0; r < ORC_ROWS; ++r)
                    xt[(size_t)i * ORC_ROWS + r] = r < nr ? a[(size_t)(r0 + r) * in + i] : 0.0;
            for (int32_t o = o0; o < o1; ++o) {
                const float *w = W + (size_t)o * in;
                double acc[ORC_ROWS] = {0.0};
                for (int32_t i = 0; i < in; ++i) {
                    const double wi = (double)w[i];
                    for (int32_t r = 0; r < ORC_ROWS; ++r) acc[r] += xt[(size_t)i * ORC_ROWS + r] * wi;
                }
                for (int32_t r = 0; r < nr; ++r) y[(size_t)(r0 + r) * out + o] = acc[r];
            }
        }
        free(xt);
    }
}

/* Forward of m tokens at positions pos0 .. pos0+m-1 against cache rows 0 .. pos0-1. Row i
 * attends to cache positions 0 .. pos0+i; its own key and value are written to the cache at
 * position pos0+i first (the causal mask over the block, Section 3.1). If logits is not NULL it
 * receives the logits of rows lm0 .. m-1 ((m - lm0) x vocab; the LM head runs on those rows
 * only); if hidden is not NULL it receives the LM head's input rows RMSNorm(x) (.) g_final of
 * every row (m x d_model). */
static int forward_rows(orc_state *st, const int32_t *tok, int32_t m, int32_t pos0, double *logits, int32_t lm0,
                        double *hidden) {
    const orc_model *M = st->m;
    const orc_config *c = &M->c;
    int32_t d = c->d_model, F = c->ffn_dim, H = c->n_heads, hd = c->head_dim, V = c->vocab;
    if (pos0 + m > st->max_ctx || lm0 < 0 || lm0 >= m) return -1;
    double *h = (double *)calloc((size_t)m * d, sizeof(double));
    double *a = (double *)calloc((size_t)m * d, sizeof(double));
    double *q = (double *)calloc((size_t)m * d, sizeof(double));
    double *kk = (double *)calloc((size_t)m * d, sizeof(double));
    double *vv = (double *)calloc((size_t)m * d, sizeof(double));
    double *o = (double *)calloc((size_t)m * d, sizeof(double));
    double *y = (double *)calloc((size_t)m * d, sizeof(double));
    double *g = (double *)calloc((size_t)m * F, sizeof(double));
    double *u = (double *)calloc((size_t)m * F, sizeof(double));
    if (!h || !a || !q || !kk || !vv || !o || !y || !g || !u) {
        free(h); free(a); free(q); free(kk); free(vv); free(o); free(y); free(g); free(u);
        return -2;
    }

    for (int32_t i = 0; i < m; ++i)
        for (int32_t k = 0; k < d; ++k) h[(size_t)i * d + k] = (double)M->embed[(size_t)tok[i] * d + k];

    for (int32_t l = 0; l < c->n_layers; ++l) {
        double *Kc = st->k + (size_t)l * st->max_ctx * d;
        double *Vc = st->v + (size_t)l * st->max_ctx * d;
        /* attention sub-layer */
        for (int32_t i = 0; i < m; ++i)
            orc_rmsnorm(h + (size_t)i * d, d, M->attn_norm[l], c->rms_eps, 0, a + (size_t)i * d);
        linear(a, m, M->wq[l], d, d, q);
        linear(a, m, M->wk[l], d, d, kk);
        linear(a, m, M->wv[l], d, d, vv);
        for (int32_t i = 0; i < m; ++i) {
            for (int32_t hh = 0; hh < H; ++hh) {
                orc_rope(q + (size_t)i * d + hh * hd, hd, pos0 + i, c->rope_base);
                orc_rope(kk + (size_t)i * d + hh * hd, hd, pos0 + i, c->rope_base);
            }
            for (int32_t k = 0; k < d; ++k) {
                size_t ix = (size_t)i * d + k;
                Kc[(size_t)(pos0 + i) * d + k] = rnd_cache(M, kk[ix]);
                Vc[(size_t)(pos0 + i) * d + k] = rnd_cache(M, vv[ix]);
            }
        }
#pragma omp parallel for collapse(2) schedule(static)
        for (int32_t i = 0; i < m; ++i)
            for (int32_t hh = 0; hh < H; ++hh)
                orc_attention_row(q + (size_t)i * d + hh * hd, Kc + hh * hd, Vc + hh * hd, pos0 + i + 1, d, hd,
                                  o + (size_t)i * d + hh * hd);
        linear(o, m, M->wo[l], d, d, y);
        for (size_t ix = 0; ix < (size_t)m * d; ++ix) h[ix] += y[ix];
        /* SwiGLU feed-forward sub-layer */
        for (int32_t i = 0; i < m; ++i)
            orc_rmsnorm(h + (size_t)i * d, d, M->ffn_norm[l], c->rms_eps, 0, a + (size_t)i * d);
        linear(a, m, M->wg[l], d, F, g);
        linear(a, m, M->wu[l], d, F, u);
        for (size_t ix = 0; ix < (size_t)m * F; ++ix) g[ix] = orc_silu(g[ix]) * u[ix];
        linear(g, m, M->wd[l], F, d, y);
        for (size_t ix = 0; ix < (size_t)m * d; ++ix) h[ix] += y[ix];
    }
    if (logits || hidden) {
        for (int32_t i = 0; i < m; ++i)
            orc_rmsnorm(h + (size_t)i * d, d, M->final_norm, c->rms_eps, 0, a + (size_t)i * d);
        if (hidden) memcpy(hidden, a, sizeof(double) * (size_t)m * d);
        if (logits) linear(a + (size_t)lm0 * d, m - lm0, M->lm_head, d, V, logits);
    }
    free(h); free(a); free(q); free(kk); free(vv); free(o); free(y); free(g); free(u);
    return 0;
}

/* Exported form of the matrix product used by the forward pass (for pinning). */
void orc_linear(const double *a, int32_t rows, const float *W, int32_t in, int32_t out, double *y) {
    linear(a, rows, W, in, out, y);
}

/* ------------------------------------------------------------------------------------- */
/* Decoding state                                                                         */

orc_state *orc_state_new(const orc_model *m, int32_t max_ctx) {
    orc_state *st = (orc_state *)calloc(1, sizeof(orc_state));
    if (!st) return NULL;
    st->m = m;
    st->max_ctx = max_ctx;
    size_t n = (size_t)m->c.n_layers * (size_t)max_ctx * (size_t)m->c.d_model;
    st->k = (double *)calloc(n ? n : 1, sizeof(double));
    st->v = (double *)calloc(n ? n : 1, sizeof(double));
    if (!st->k || !st->v) {
        free(st->k); free(st->v); free(st);
        return NULL;
    }
    return st;
}

void orc_state_free(orc_state *st) {
    if (!st) return;
    free(st->k); free(st->v); free(st);
}

int32_t orc_state_len(const orc_state *st) { return st->L; }
int32_t orc_state_pending(const orc_state *st) { return st->pending; }

/* Prefill (the algorithm's first forward: the prompt's cache and the first token y0).
 * Returns y0, or a negative code. logits_last (vocab doubles) may be NULL. */
int32_t orc_prefill(orc_state *st, const int32_t *prompt, int32_t len, double *logits_last) {
    const orc_config *c = &st->m->c;
    if (len < 1 || len > st->max_ctx) return -1;
    double *lg = (double *)malloc(sizeof(double) * (size_t)c->vocab);
    if (!lg) return -2;
    int rc = forward_rows(st, prompt, len, 0, lg, len - 1, NULL);
    if (rc) { free(lg); return -3; }
    int32_t y0 = orc_argmax(lg, c->vocab);
    if (logits_last) memcpy(logits_last, lg, sizeof(double) * c->vocab);
    free(lg);
    if (y0 < 0) return -4;
    st->L = len;
    st->pending = y0;
    st->prefilled = 1;
    return y0;
}

/* Logits of one iteration over block[0..m) at positions L .. L+m-1 (keys and values of the
 * block are written to the cache provisionally; nothing is committed). */
int32_t orc_eval_block(orc_state *st, const int32_t *block, int32_t m, double *logits) {
    if (!st->prefilled || m < 1 || st->L + m > st->max_ctx) return -1;
    return forward_rows(st, block, m, st->L, logits, 0, NULL) ? -3 : 0;
}

/* The LM head's input rows (m x d_model) of an iteration over block[0..m) at positions
 * L .. L+m-1 (as orc_eval_block: nothing is committed). */
int32_t orc_eval_block_hidden(orc_state *st, const int32_t *block, int32_t m, double *hidden) {
    if (!st->prefilled || m < 1 || st->L + m > st->max_ctx) return -1;
    return forward_rows(st, block, m, st->L, NULL, 0, hidden) ? -3 : 0;
}

/* Commit a accepted tokens (their cache rows become permanent) and set the pending token. */
int32_t orc_commit(orc_state *st, int32_t a, int32_t pending) {
    if (a < 1 || st->L + a > st->max_ctx) return -1;
    st->L += a;
    st->pending = pending;
    return 0;
}

/* One Jacobi iteration: the block's greedy predictions, the accepted length and the commit.
 * block_in[0] must be the pending token. logits (m x vocab) may be NULL. */
int32_t orc_jacobi_step(orc_state *st, const int32_t *block_in, int32_t m, int32_t *block_out, int32_t *accepted,
                        double *logits) {
    const orc_config *c = &st->m->c;
    if (!st->prefilled || m < 1 || block_in[0] != st->pending) return -1;
    double *lg = logits ? logits : (double *)malloc(sizeof(double) * (size_t)m * c->vocab);
    if (!lg) return -2;
    int32_t rc = orc_eval_block(st, block_in, m, lg);
    if (rc == 0) {
        for (int32_t k = 0; k < m; ++k) {
            block_out[k] = orc_argmax(lg + (size_t)k * c->vocab, c->vocab);
            if (block_out[k] < 0) rc = -4;
        }
    }
    if (!logits) free(lg);
    if (rc) return rc;
    int32_t a = orc_accept_len(block_in, block_out, m);
    *accepted = a;
    return orc_commit(st, a, block_out[a - 1]);
}

/* Full forward of tokens[0..T) from an empty cache (no reuse): logits T x vocab. */
int32_t orc_forward_full(const orc_model *m, const int32_t *tokens, int32_t T, double *logits) {
    orc_state *st = orc_state_new(m, T);
    if (!st) return -2;
    int rc = forward_rows(st, tokens, T, 0, logits, 0, NULL);
    orc_state_free(st);
    return rc ? -3 : 0;
}

/* ------------------------------------------------------------------------------------- */
/* Decoders                                                                               */

/* Greedy AR decoding, eq. (ar_decoding): y0 from the prefill, then one token per forward.
 * out holds max_new tokens. */
int32_t orc_ar_decode(const orc_model *m, const int32_t *prompt, int32_t len, int32_t max_new, int32_t *out) {
    if (max_new < 1) return -1;
    orc_state *st = orc_state_new(m, len + max_new);
    if (!st) return -2;
    int32_t rc = 0;
    int32_t y = orc_prefill(st, prompt, len, NULL);
    if (y < 0) rc = -3;
    double *lg = (double *)malloc(sizeof(double) * m->c.vocab);
    for (int32_t t = 0; rc == 0 && t < max_new; ++t) {
        out[t] = y;
        if (t + 1 == max_new) break;
        if (forward_rows(st, &y, 1, st->L, lg, 0, NULL)) { rc = -3; break; }
        st->L += 1;
        y = orc_argmax(lg, m->c.vocab);
        if (y < 0) rc = -4;
    }
    free(lg);
    orc_state_free(st);
    return rc;
}

/* Jacobi decoding with a KV cache (the appendix algorithm), blockwise over max_new tokens
 * (Section 3.2.1: long responses are decoded one n-token truncation after another).
 * Block policy 0 (shrink): after an iteration that accepts a < m tokens the state becomes the
 * pending token followed by the unaccepted predictions; a block ends when all of it is fixed.
 * Block policy 1 (slide): the state is always the next min(n, remaining) positions.
 * Guess policy 2 re-draws every unfixed position from the corrupted stream after each
 * iteration instead of keeping the model's predictions.
 * step_m / step_a (capacity max_steps, may be NULL) record the trajectory's sizes. */
int32_t orc_jacobi_decode(const orc_model *m, const int32_t *prompt, int32_t len, int32_t n, int32_t max_new,
                          const orc_guess_spec *gs, int32_t seq, int32_t *out, orc_stats *stats, int32_t *step_m,
                          int32_t *step_a, int32_t max_steps, const orc_traj *tr) {
    const int32_t V = m->c.vocab;
    if (n < 1 || max_new < 1 || !gs) return -1;
    orc_state *st = orc_state_new(m, len + max_new + n);
    if (!st) return -2;
    int32_t *z = (int32_t *)malloc(sizeof(int32_t) * n);
    int32_t *pred = (int32_t *)malloc(sizeof(int32_t) * n);
    int32_t *nz = (int32_t *)malloc(sizeof(int32_t) * n);
    orc_stats loc;
    memset(&loc, 0, sizeof(loc));
    int32_t rc = 0;
    int32_t y0 = orc_prefill(st, prompt, len, NULL);
    if (y0 < 0) rc = -3;
    int32_t e = 0;          /* tokens emitted (fixed) */
    int32_t b0 = 0;         /* first output position of the current block */
    int32_t nb = n < max_new ? n : max_new;
    int32_t mlen = nb;
    z[0] = y0;
    for (int32_t j = 1; j < mlen; ++j) z[j] = orc_guess(gs, seq, j, 0, V);
    loc.blocks = 1;
    while (rc == 0 && e < max_new) {
        int32_t a;
        const int32_t L_before = st->L;
        if (orc_jacobi_step(st, z, mlen, pred, &a, NULL)) { rc = -4; break; }
        if (tr && loc.steps < tr->cap) {
            const int64_t t = loc.steps;
            tr->L[t] = L_before;
            tr->e[t] = e;
            tr->b0[t] = gs->block_policy == 0 ? b0 : e;
            for (int32_t k = 0; k < mlen; ++k) {
                tr->z[t * n + k] = z[k];
                tr->pred[t * n + k] = pred[k];
            }
        }
        for (int32_t k = 0; k < a; ++k) out[e + k] = z[k];
        if (step_m && loc.steps < max_steps) { step_m[loc.steps] = mlen; step_a[loc.steps] = a; }
        e += a;
        loc.steps += 1;
        loc.accept_hist[a < 256 ? a : 256] += 1;
        if (e >= max_new) break;
        int32_t draw = (gs->policy == 2) ? (int32_t)loc.steps : 0;
        int32_t newm;
        if (gs->block_policy == 0) {
            if (e == b0 + nb) { /* block converged: its last prediction seeds the next block */
                b0 = e;
                nb = (max_new - e) < n ? (max_new - e) : n;
                newm = nb;
                loc.blocks += 1;
                nz[0] = st->pending;
                for (int32_t j = 1; j < newm; ++j) nz[j] = orc_guess(gs, seq, e + j, draw, V);
            } else {
                newm = b0 + nb - e;
                nz[0] = st->pending;
                for (int32_t j = 1; j < newm; ++j)
                    nz[j] = (gs->policy == 2) ? orc_guess(gs, seq, e + j, draw, V) : pred[a - 1 + j];
            }
        } else {
            newm = (max_new - e) < n ? (max_new - e) : n;
            nz[0] = st->pending;
            for (int32_t j = 1; j < newm; ++j) {
                int32_t src = a - 1 + j; /* prediction index for output position e + j */
                if (gs->policy != 2 && src < mlen)
                    nz[j] = pred[src];
                else
                    nz[j] = orc_guess(gs, seq, e + j, draw, V);
            }
        }
        mlen = newm;
        memcpy(z, nz, sizeof(int32_t) * newm);
    }
    loc.tokens = e;
    if (stats) *stats = loc;
    free(z); free(pred); free(nz);
    orc_state_free(st);
    return rc;
}
