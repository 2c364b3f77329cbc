/*
 * hbsjd_oracle.c - plain, slow, fp32 CPU oracle of the batched
 * speculative-Jacobi (SJD) rollout.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing on the product path may call, link or
 * load this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do. It shares no code, header or table with the HIP library.
 *
 * Every floating-point operation is fp32 with one rounding per operation
 * (compiled with -ffp-contract=off, no fast-math), every dot product and sum
 * runs sequentially in index order, and every row is computed on its own, so
 * the result of a row never depends on which other rows are processed.
 *
 * What it follows (paper sections / equations):
 *  - the student distribution is the AR factorisation p(x_t | x_<t)  (Sec. 3.1, Eq. 1);
 *    the rollout suffix must follow the mixed distribution of Eq. 2;
 *  - independent per-image state: committed cursor plus a window of W drafts;
 *    first draft sampled from the student after prefill; later windows reuse the
 *    previous verification's predictions and fill the rest with committed tokens
 *    at history offset H  (Sec. 4.2, "Independent rollout states");
 *  - batched verifier input = last committed token followed by the window
 *    (Sec. 4.2, "Batched verification");
 *  - probabilistic acceptance min(1, p(z)/q(z)), resampling from the residual
 *    [p - q]_+ on rejection  (Sec. 4.2, Eq. 5);
 *  - greedy acceptance z = argmax p, argmax committed at the first mismatch
 *    (Sec. 4.2, Eq. 4);
 *  - independent commit; the replacement token opens the next round, whose
 *    forward recomputes the cache after the rejection point  (Sec. 4.2,
 *    "Independent progress"); CFG branches share one state and verify on the
 *    fused guided logits (same paragraph);
 *  - Full vs Compact execution differ only in which rows are physically
 *    processed; the per-round choice is Full iff A > gamma  (Sec. 4.3, Eq. 6);
 *  - the Batch-Synchronous SJD ablation (Sec. 4.1 "From Single-Sequence to
 *    Batched SJD", Fig. 2a, Table 2): every image works through the same
 *    sequence of Jacobi windows; an image that has committed its whole current
 *    window waits until every active image has done so, and only then does the
 *    batch move on to the next window.
 *
 * Where the paper is silent the oracle takes these readings: the decoder is a
 * LlamaGen-style pre-norm transformer (RMSNorm eps 1e-5, 2D RoPE on adjacent
 * pairs, first half of the pairs rotated by the grid row, second half by the
 * grid column, class token at position 0 unrotated, SwiGLU MLP, no biases except
 * an optional lm_head bias); the verifier sees W+1 rows and commits between 1
 * and min(W, T-n) tokens (no bonus token); a reused prediction is a sample from
 * that row's distribution with that row as its proposal; a history draft takes
 * the token H positions back (one back when that is before position 1) and has a
 * point-mass proposal; the transform applies CFG, then temperature, then top-k
 * (ties kept), then softmax; Philox4x32-10 keyed by the seed with counter
 * (image, position, 0, 0) gives the draft, accept and resample uniforms; every
 * sum over the vocabulary is associated as sequential sums inside consecutive
 * 64-entry chunks, chunk totals then added sequentially; the inverse CDF returns
 * the first entry whose inclusive prefix exceeds u * total. For the
 * batch-synchronous ablation, window w of image b spans positions
 * k_b + wW + 1 .. min(k_b + (w+1)W, T) (each image counts windows from its own
 * prefix); an image waiting at the boundary still forwards its last committed
 * token and re-draws its first draft from that row, committing nothing.
 *
 * om_rollout can also record every image's window (drafts and the proposal
 * probability q(z) of each) after the prefill and after every round, so that
 * tests can compare the refresh step round by round.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OM_CHUNK 64

typedef struct {
    int n_layers, d, n_heads, f, V, C, G, has_bias;
    float eps, rope_base;
} om_desc;

typedef struct {
    om_desc m;
    int dh, T;
    float *tok_emb, *cls_emb;               /* [V][d], [(C+1)][d] */
    float **g_attn, **g_ffn;                /* [d] per layer */
    float **wqkv_t, **wo_t, **w1_t, **w3_t, **w2_t; /* transposed: [in][out] */
    float *g_out, *wlm_t, *b_lm;            /* [d], [d][V], [V] or NULL */
    float *rope_cos, *rope_sin;             /* [(T+1)][dh/2] */
} om_model;

/* planted mistakes for the oracle's own power tests (never set otherwise) */
static int g_debug = 0;
void om_set_debug(int flags) { g_debug = flags; }
#define DBG_RESIDUAL_DROPS_Q 1
#define DBG_INVERTED_RATIO 2
#define DBG_ROPE_SIGN 4
#define DBG_HISTORY_SHIFT 8   /* history token one position later: S[pos - H + 1] */
#define DBG_REUSE_SHIFT 16    /* reused prediction taken from the next row */

/* ---------------------------------------------------------------- utils */

static float* fdup(const float* src, long n) {
    float* p = (float*)malloc(sizeof(float) * (size_t)n);
    memcpy(p, src, sizeof(float) * (size_t)n);
    return p;
}

/* W is [out][in]; returns Wt [in][out] so that y[n] = sum_k x[k] Wt[k][n]. */
static float* transpose(const float* w, int out, int in) {
    float* t = (float*)malloc(sizeof(float) * (size_t)out * in);
    for (int o = 0; o < out; ++o)
        for (int i = 0; i < in; ++i) t[(size_t)i * out + o] = w[(size_t)o * in + i];
    return t;
}

/* y[n] = sum_{k=0}^{K-1} x[k] * Wt[k][n], summed in k order for every n. */
static void matvec(const float* x, const float* wt, int K, int N, float* y) {
    for (int n = 0; n < N; ++n) y[n] = 0.0f;
    for (int k = 0; k < K; ++k) {
        const float xk = x[k];
        const float* row = wt + (size_t)k * N;
        for (int n = 0; n < N; ++n) y[n] = y[n] + xk * row[n];
    }
}

static float dot(const float* a, const float* b, int n) {
    float s = 0.0f;
    for (int i = 0; i < n; ++i) s = s + a[i] * b[i];
    return s;
}

/* RMSNorm(x) * g: x / sqrt(mean(x^2) + eps), then the gain. */
static void rmsnorm(const float* x, const float* g, int d, float eps, float* y) {
    float ss = 0.0f;
    for (int i = 0; i < d; ++i) ss = ss + x[i] * x[i];
    const float r = 1.0f / sqrtf(ss / (float)d + eps);
    for (int i = 0; i < d; ++i) y[i] = (x[i] * r) * g[i];
}

/* ---------------------------------------------------------------- model */

om_model* om_create(const om_desc* desc, const float* blob, long n_floats) {
    const om_desc m = *desc;
    if (m.d % m.n_heads) return NULL;
    const int dh = m.d / m.n_heads;
    if (dh % 4) return NULL;
    long need = (long)m.V * m.d + (long)(m.C + 1) * m.d +
                (long)m.n_layers * (2L * m.d + 3L * m.d * m.d + (long)m.d * m.d +
                                    3L * m.f * m.d) +
                m.d + (long)m.V * m.d + (m.has_bias ? m.V : 0);
    if (need != n_floats) return NULL;
    om_model* o = (om_model*)calloc(1, sizeof(om_model));
    o->m = m;
    o->dh = dh;
    o->T = m.G * m.G;
    const float* p = blob;
    o->tok_emb = fdup(p, (long)m.V * m.d); p += (long)m.V * m.d;
    o->cls_emb = fdup(p, (long)(m.C + 1) * m.d); p += (long)(m.C + 1) * m.d;
    const int L = m.n_layers, d = m.d, f = m.f;
    o->g_attn = (float**)calloc(L, sizeof(float*));
    o->g_ffn = (float**)calloc(L, sizeof(float*));
    o->wqkv_t = (float**)calloc(L, sizeof(float*));
    o->wo_t = (float**)calloc(L, sizeof(float*));
    o->w1_t = (float**)calloc(L, sizeof(float*));
    o->w3_t = (float**)calloc(L, sizeof(float*));
    o->w2_t = (float**)calloc(L, sizeof(float*));
    for (int l = 0; l < L; ++l) {
        o->g_attn[l] = fdup(p, d); p += d;
        o->wqkv_t[l] = transpose(p, 3 * d, d); p += 3L * d * d;
        o->wo_t[l] = transpose(p, d, d); p += (long)d * d;
        o->g_ffn[l] = fdup(p, d); p += d;
        o->w1_t[l] = transpose(p, f, d); p += (long)f * d;
        o->w3_t[l] = transpose(p, f, d); p += (long)f * d;
        o->w2_t[l] = transpose(p, d, f); p += (long)d * f;
    }
    o->g_out = fdup(p, d); p += d;
    o->wlm_t = transpose(p, m.V, d); p += (long)m.V * d;
    o->b_lm = m.has_bias ? fdup(p, m.V) : NULL;
    /* 2D RoPE angles: position s >= 1 is grid cell s-1 = (row, col); pairs
       i < dh/4 turn by row * theta_i, pairs dh/4 <= i < dh/2 by
       col * theta_{i - dh/4}, theta_i = base^(-4 i / dh). Position 0 is not turned. */
    const int half = dh / 2, quarter = dh / 4;
    o->rope_cos = (float*)malloc(sizeof(float) * (size_t)(o->T + 1) * half);
    o->rope_sin = (float*)malloc(sizeof(float) * (size_t)(o->T + 1) * half);
    for (int s = 0; s <= o->T; ++s) {
        const int row = s >= 1 ? (s - 1) / m.G : 0;
        const int col = s >= 1 ? (s - 1) % m.G : 0;
        for (int i = 0; i < half; ++i) {
            double ang = 0.0;
            if (s >= 1) {
                const int ii = i < quarter ? i : i - quarter;
                const double theta = pow((double)m.rope_base, -4.0 * ii / (double)dh);
                ang = (i < quarter ? row : col) * theta;
            }
            o->rope_cos[(size_t)s * half + i] = (float)cos(ang);
            o->rope_sin[(size_t)s * half + i] = (float)sin(ang);
        }
    }
    return o;
}

void om_free(om_model* o) {
    if (!o) return;
    for (int l = 0; l < o->m.n_layers; ++l) {
        free(o->g_attn[l]); free(o->g_ffn[l]); free(o->wqkv_t[l]); free(o->wo_t[l]);
        free(o->w1_t[l]); free(o->w3_t[l]); free(o->w2_t[l]);
    }
    free(o->g_attn); free(o->g_ffn); free(o->wqkv_t); free(o->wo_t);
    free(o->w1_t); free(o->w3_t); free(o->w2_t);
    free(o->tok_emb); free(o->cls_emb); free(o->g_out); free(o->wlm_t); free(o->b_lm);
    free(o->rope_cos); free(o->rope_sin);
    free(o);
}

/* Rotate one head vector u (length dh) for sequence position s (clamped to T). */
static void rope_apply(const om_model* o, float* u, int s) {
    if (s > o->T) s = o->T;
    const int half = o->dh / 2;
    const float* cs = o->rope_cos + (size_t)s * half;
    const float* sn = o->rope_sin + (size_t)s * half;
    for (int i = 0; i < half; ++i) {
        const float a = u[2 * i], b = u[2 * i + 1];
        if (g_debug & DBG_ROPE_SIGN) {
            u[2 * i] = a * cs[i] + b * sn[i];
            u[2 * i + 1] = b * cs[i] - a * sn[i];
        } else {
            u[2 * i] = a * cs[i] - b * sn[i];
            u[2 * i + 1] = a * sn[i] + b * cs[i];
        }
    }
}

void om_rope(const om_model* o, float* u, int s) { rope_apply(o, u, s); }

/* KV cache of one sequence: K[l][pos][d], V[l][pos][d] for pos < cap. */
typedef struct {
    int cap;
    float *k, *v;
} om_cache;

static void cache_init(om_cache* c, const om_model* o, int cap) {
    c->cap = cap;
    size_t n = (size_t)o->m.n_layers * cap * o->m.d;
    c->k = (float*)calloc(n, sizeof(float));
    c->v = (float*)calloc(n, sizeof(float));
}
static void cache_free(om_cache* c) { free(c->k); free(c->v); c->k = c->v = NULL; }

typedef struct {
    float *h, *a, *qkv, *att, *g, *u, *act, *tmp, *scores;
} om_scratch;

static void scratch_init(om_scratch* s, const om_model* o, int max_ctx) {
    const int d = o->m.d, f = o->m.f;
    s->h = (float*)malloc(sizeof(float) * d);
    s->a = (float*)malloc(sizeof(float) * d);
    s->qkv = (float*)malloc(sizeof(float) * 3 * d);
    s->att = (float*)malloc(sizeof(float) * d);
    s->g = (float*)malloc(sizeof(float) * f);
    s->u = (float*)malloc(sizeof(float) * f);
    s->act = (float*)malloc(sizeof(float) * f);
    s->tmp = (float*)malloc(sizeof(float) * d);
    s->scores = (float*)malloc(sizeof(float) * (max_ctx + 1));
}
static void scratch_free(om_scratch* s) {
    free(s->h); free(s->a); free(s->qkv); free(s->att); free(s->g); free(s->u);
    free(s->act); free(s->tmp); free(s->scores);
}

/*
 * One decoder row: the token at sequence position `pos` (token >= 0 is an image
 * token; token < 0 encodes class -(token+1) at position 0). Writes its K and V
 * into the cache at `pos` and attends causally over cache positions 0..pos.
 * Writes V logits when `logits` is not NULL.
 */
static void om_step(const om_model* o, om_cache* c, om_scratch* s, int pos, int token,
                    float* logits) {
    const int d = o->m.d, f = o->m.f, H = o->m.n_heads, dh = o->dh;
    const float scale = 1.0f / sqrtf((float)dh);
    const float* emb = token >= 0 ? o->tok_emb + (size_t)token * d
                                  : o->cls_emb + (size_t)(-(token + 1)) * d;
    memcpy(s->h, emb, sizeof(float) * d);
    for (int l = 0; l < o->m.n_layers; ++l) {
        rmsnorm(s->h, o->g_attn[l], d, o->m.eps, s->a);
        matvec(s->a, o->wqkv_t[l], d, 3 * d, s->qkv);
        float* q = s->qkv;
        float* k = s->qkv + d;
        float* v = s->qkv + 2 * d;
        for (int hh = 0; hh < H; ++hh) {
            rope_apply(o, q + hh * dh, pos);
            rope_apply(o, k + hh * dh, pos);
        }
        float* kc = c->k + ((size_t)l * c->cap) * d;
        float* vc = c->v + ((size_t)l * c->cap) * d;
        memcpy(kc + (size_t)pos * d, k, sizeof(float) * d);
        memcpy(vc + (size_t)pos * d, v, sizeof(float) * d);
        for (int hh = 0; hh < H; ++hh) {
            const float* qh = q + hh * dh;
            float mx = -INFINITY;
            for (int j = 0; j <= pos; ++j) {
                const float sc = dot(qh, kc + (size_t)j * d + hh * dh, dh) * scale;
                s->scores[j] = sc;
                if (sc > mx) mx = sc;
            }
            float z = 0.0f;
            for (int j = 0; j <= pos; ++j) {
                s->scores[j] = expf(s->scores[j] - mx);
                z = z + s->scores[j];
            }
            float* out = s->att + hh * dh;
            for (int e = 0; e < dh; ++e) out[e] = 0.0f;
            for (int j = 0; j <= pos; ++j) {
                const float w = s->scores[j] / z;
                const float* vj = vc + (size_t)j * d + hh * dh;
                for (int e = 0; e < dh; ++e) out[e] = out[e] + w * vj[e];
            }
        }
        matvec(s->att, o->wo_t[l], d, d, s->tmp);
        for (int i = 0; i < d; ++i) s->h[i] = s->h[i] + s->tmp[i];
        rmsnorm(s->h, o->g_ffn[l], d, o->m.eps, s->a);
        matvec(s->a, o->w1_t[l], d, f, s->g);
        matvec(s->a, o->w3_t[l], d, f, s->u);
        for (int i = 0; i < f; ++i) {
            const float gi = s->g[i];
            const float silu = gi / (1.0f + expf(-gi));
            s->act[i] = silu * s->u[i];
        }
        matvec(s->act, o->w2_t[l], f, d, s->tmp);
        for (int i = 0; i < d; ++i) s->h[i] = s->h[i] + s->tmp[i];
    }
    if (logits) {
        rmsnorm(s->h, o->g_out, d, o->m.eps, s->a);
        matvec(s->a, o->wlm_t, d, o->m.V, logits);
        if (o->b_lm)
            for (int v = 0; v < o->m.V; ++v) logits[v] = logits[v] + o->b_lm[v];
    }
}

/* Teacher-forced forward of one sequence [class, x_1..x_n]; logits for
   positions 0..n into out[(n+1) x V]. */
int om_forward_seq(const om_model* o, int cls, const int* tok, int n, float* out) {
    if (n < 0 || n > o->T) return -1;
    om_cache c;
    om_scratch s;
    cache_init(&c, o, n + 1);
    scratch_init(&s, o, n + 1);
    for (int p = 0; p <= n; ++p)
        om_step(o, &c, &s, p, p == 0 ? -(cls + 1) : tok[p - 1], out + (size_t)p * o->m.V);
    scratch_free(&s);
    cache_free(&c);
    return 0;
}

/* Teacher-forced forwards of n independent sequences (one per OpenMP task):
   sequence s is [cls[s], tok[off[s]] .. tok[off[s] + len[s] - 1]], its logits go
   to out rows row0[s] .. row0[s] + len[s]. */
int om_forward_batch(const om_model* o, int n, const int* cls, const int* tok, const int* off,
                     const int* len, const long* row0, float* out) {
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int s = 0; s < n; ++s)
        bad |= om_forward_seq(o, cls[s], tok + off[s], len[s], out + row0[s] * o->m.V) != 0;
    return bad ? -1 : 0;
}

/* ---------------------------------------------------------------- RNG */

/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of the
   multiply-xor bijection with the Weyl key schedule. */
void om_philox(uint64_t seed, const uint32_t ctr[4], uint32_t out[4]) {
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        const uint32_t n1 = (uint32_t)p1;
        const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        const uint32_t n3 = (uint32_t)p0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* 24 high bits as a uniform on [0, 1 - 2^-24]. */
static float u01(uint32_t x) { return (float)(x >> 8) * (1.0f / 16777216.0f); }

typedef struct { float draft, acc, res; } om_uniforms;

static om_uniforms uniforms(uint64_t seed, int b, int t) {
    uint32_t ctr[4] = {(uint32_t)b, (uint32_t)t, 0u, 0u}, o4[4];
    om_philox(seed, ctr, o4);
    om_uniforms u = {u01(o4[0]), u01(o4[1]), u01(o4[2])};
    return u;
}

void om_uniforms3(uint64_t seed, int b, int t, float out[3]) {
    om_uniforms u = uniforms(seed, b, t);
    out[0] = u.draft; out[1] = u.acc; out[2] = u.res;
}

/* ---------------------------------------------------------------- sampling */

/* sum of w[0..n): sequential inside 64-entry chunks, chunk totals sequential */
float om_pinned_sum(const float* w, int n) {
    float total = 0.0f;
    for (int c0 = 0; c0 < n; c0 += OM_CHUNK) {
        const int c1 = c0 + OM_CHUNK < n ? c0 + OM_CHUNK : n;
        float t = 0.0f;
        for (int v = c0; v < c1; ++v) t = t + w[v];
        total = total + t;
    }
    return total;
}

/* Inverse CDF over non-negative weights: the smallest v whose inclusive prefix
   (chunk prefix + in-chunk prefix) exceeds u * total; if rounding leaves none,
   the largest v with positive weight; -1 if every weight is zero. */
int om_inv_cdf(const float* w, int n, float u) {
    const float target = u * om_pinned_sum(w, n);
    float before = 0.0f;
    for (int c0 = 0; c0 < n; c0 += OM_CHUNK) {
        const int c1 = c0 + OM_CHUNK < n ? c0 + OM_CHUNK : n;
        float inner = 0.0f;
        for (int v = c0; v < c1; ++v) {
            inner = inner + w[v];
            if (before + inner > target) return v;
        }
        before = before + inner;
    }
    for (int v = n - 1; v >= 0; --v)
        if (w[v] > 0.0f) return v;
    return -1;
}

static int cmp_desc(const void* a, const void* b) {
    const float x = *(const float*)a, y = *(const float*)b;
    return (x < y) - (x > y);
}

/* Distribution transform: y = l / tau; keep the top_k largest (ties with the
   k-th kept; 0 or >= V keeps all); softmax over the kept entries. */
void om_transform(const float* l, int V, float tau, int top_k, float* p) {
    float* y = p;
    for (int v = 0; v < V; ++v) y[v] = l[v] / tau;
    float thr = -INFINITY;
    if (top_k > 0 && top_k < V) {
        float* tmp = fdup(y, V);
        qsort(tmp, V, sizeof(float), cmp_desc);
        thr = tmp[top_k - 1];
        free(tmp);
    }
    float mx = -INFINITY;
    for (int v = 0; v < V; ++v)
        if (y[v] >= thr && y[v] > mx) mx = y[v];
    for (int v = 0; v < V; ++v) y[v] = y[v] >= thr ? expf(y[v] - mx) : 0.0f;
    const float z = om_pinned_sum(y, V);
    for (int v = 0; v < V; ++v) p[v] = y[v] / z;
}

/* CFG guided logits: l_u + s * (l_c - l_u). */
void om_cfg_combine(const float* lc, const float* lu, int V, float s, float* out) {
    for (int v = 0; v < V; ++v) out[v] = lu[v] + s * (lc[v] - lu[v]);
}

int om_argmax(const float* l, int V) {
    int best = 0;
    for (int v = 1; v < V; ++v)
        if (l[v] > l[best]) best = v;
    return best;
}

/* One probabilistic verification of a window against explicit rows.
   p[j], q[j] are the target and proposal rows for draft j (j = 0..n-1); q may
   be NULL for a draft whose proposal is a point mass (qmass[j] != 0).
   Returns the count committed (accepted drafts plus the replacement). */
static int verify_window(int n, int V, const float* const* p, const float* const* q,
                         const int* qmass, const int* drafts, const float* u_acc,
                         const float* u_res, float* resid, int* out_tokens,
                         int* rejected) {
    for (int j = 0; j < n; ++j) {
        const int z = drafts[j];
        const float P = p[j][z];
        const float Q = qmass[j] ? 1.0f : q[j][z];
        int accept;
        if (g_debug & DBG_INVERTED_RATIO)
            accept = (Q >= P) || (u_acc[j] < Q / P);
        else
            accept = (P >= Q) || (u_acc[j] < P / Q);
        if (accept) {
            out_tokens[j] = z;
            continue;
        }
        for (int v = 0; v < V; ++v) {
            const float qv = qmass[j] ? (v == z ? 1.0f : 0.0f) : q[j][v];
            const float r = (g_debug & DBG_RESIDUAL_DROPS_Q) ? p[j][v] : p[j][v] - qv;
            resid[v] = r > 0.0f ? r : 0.0f;
        }
        int tok;
        if (om_pinned_sum(resid, V) > 0.0f)
            tok = om_inv_cdf(resid, V, u_res[j]);
        else
            tok = om_inv_cdf(p[j], V, u_res[j]);
        out_tokens[j] = tok;
        *rejected = 1;
        return j + 1;
    }
    *rejected = 0;
    return n;
}

/* Verification on caller-supplied rows: p, q [B][W][V], drafts and u_acc
   [B][W], u_res [B] (used at the first rejection). Outputs counts [B] and the
   committed tokens [B][W] (entries past the count are left as -1). */
void om_verify_probs(int B, int W, int V, const float* p, const float* q,
                     const int* drafts, const float* u_acc, const float* u_res,
                     int* counts, int* tokens) {
    const float** pr = (const float**)malloc(sizeof(float*) * W);
    const float** qr = (const float**)malloc(sizeof(float*) * W);
    int* qmass = (int*)calloc(W, sizeof(int));
    float* ures = (float*)malloc(sizeof(float) * W);
    float* resid = (float*)malloc(sizeof(float) * V);
    for (int b = 0; b < B; ++b) {
        for (int j = 0; j < W; ++j) {
            pr[j] = p + ((size_t)b * W + j) * V;
            qr[j] = q + ((size_t)b * W + j) * V;
            ures[j] = u_res[b];
        }
        for (int j = 0; j < W; ++j) tokens[(size_t)b * W + j] = -1;
        int rej;
        counts[b] = verify_window(W, V, pr, qr, qmass, drafts + (size_t)b * W,
                                  u_acc + (size_t)b * W, ures, resid,
                                  tokens + (size_t)b * W, &rej);
    }
    free(pr); free(qr); free(qmass); free(ures); free(resid);
}

/* ---------------------------------------------------------------- rollout */

typedef struct {
    int B;
    const int* prefix_tokens;   /* [B][T] */
    const int* prefix_len;      /* [B] */
    const int* labels;          /* [B] */
    const float* temperature;   /* [B] */
    int W, H, top_k;
    float cfg_scale;            /* 0 = no CFG */
    uint64_t seed;
    int greedy;                 /* 0 = probabilistic (Eq. 5), 1 = greedy (Eq. 4) */
    int exec_mode;              /* 0 Full, 1 Compact, 2 Auto (Eq. 6) */
    int gamma;
    int max_rounds;
    int sync;                   /* 0 = independent progress, 1 = batch-synchronous windows */
} om_rollout_args;

typedef struct {
    int* tokens;        /* [B][T] */
    int* counts;        /* [max_rounds][B], 0 when inactive */
    int* rounds;        /* 1 */
    int* active_hist;   /* [max_rounds] or NULL */
    int* mode_hist;     /* [max_rounds] or NULL: 0 Full, 1 Compact */
    long* stats;        /* [3] or NULL: drafts verified, drafts rejected, image-rounds */
    /* the window after the prefill (entry 0) and after each round r (entry r+1),
       or NULL: [max_rounds + 1][B][W] drafts at positions n_b + 1 + m (-1 past T
       or once the image is complete) and their proposal probability q(z):
       the reused row's p(z), 1 for a point-mass (history) proposal and in
       greedy mode, 0 where the draft is -1 */
    int* trace_drafts;
    float* trace_q;
} om_rollout_out;

typedef struct {
    int n, active, k;
    int e;               /* batch-synchronous mode: end of the current window */
    int* x;              /* [T+1], x[1..n] committed */
    int* wz;             /* [W]: draft at position n + 1 + m */
    int* wmass;          /* [W]: 1 if its proposal is a point mass */
    float* wq;           /* [W][V]: proposal rows of reused drafts */
    int* nz; int* nmass; float* nq;   /* next-window staging */
    float* logits;       /* [cfg][W+1][V] */
    float* guided;       /* [W+1][V] */
    float* p;            /* [W+1][V] */
    float* resid;        /* [V] */
    om_cache cache[2];
    om_scratch s;
    long verified, rejected;
} om_img;

/* Refill the window for positions n_new+1 .. n_new+min(W, T-n_new): a position
   predicted by row i (row i predicts base+i+1, i < nrows) gets a reused
   prediction from that row; the rest take the history token. */
static void refresh_window(const om_model* o, const om_rollout_args* a, om_img* st, int b,
                           int n_new, int base, int nrows) {
    const int T = o->T, V = o->m.V, W = a->W;
    const int span = W < T - n_new ? W : T - n_new;
    for (int m = 1; m <= span; ++m) {
        const int pos = n_new + m;
        const int i = pos - base - 1 + ((g_debug & DBG_REUSE_SHIFT) ? 1 : 0);
        if (i >= 0 && i < nrows) {
            if (a->greedy) {
                st->nz[m - 1] = om_argmax(st->guided + (size_t)i * V, V);
            } else {
                const om_uniforms u = uniforms(a->seed, b, pos);
                st->nz[m - 1] = om_inv_cdf(st->p + (size_t)i * V, V, u.draft);
                memcpy(st->nq + (size_t)(m - 1) * V, st->p + (size_t)i * V, sizeof(float) * V);
            }
            st->nmass[m - 1] = 0;
        } else {
            const int H = (g_debug & DBG_HISTORY_SHIFT) ? a->H - 1 : a->H;
            const int src = pos - H >= 1 ? pos - H : pos - 1;
            st->nz[m - 1] = src <= n_new ? st->x[src] : st->nz[src - n_new - 1];
            st->nmass[m - 1] = 1;
        }
    }
    int* t = st->wz; st->wz = st->nz; st->nz = t;
    t = st->wmass; st->wmass = st->nmass; st->nmass = t;
    float* q = st->wq; st->wq = st->nq; st->nq = q;
}

/* Forward rows i = 0..nrows-1 of one image at positions n+i for each CFG branch
   and turn them into guided logits and (probabilistic mode) distributions. */
static void window_forward(const om_model* o, const om_rollout_args* a, om_img* st, int b,
                           int n, int nrows, const int* row_tokens, int compute_p) {
    const int V = o->m.V;
    const int ncfg = a->cfg_scale != 0.0f ? 2 : 1;
    for (int br = 0; br < ncfg; ++br) {
        for (int i = 0; i < nrows; ++i) {
            int tok = row_tokens[i];
            if (tok < 0) tok = br == 0 ? -(a->labels[b] + 1) : -(o->m.C + 1);
            om_step(o, &st->cache[br], &st->s, n + i, tok,
                    st->logits + ((size_t)br * (a->W + 1) + i) * V);
        }
    }
    for (int i = 0; i < nrows; ++i) {
        float* g = st->guided + (size_t)i * V;
        const float* lc = st->logits + (size_t)i * V;
        if (ncfg == 2)
            om_cfg_combine(lc, st->logits + ((size_t)(a->W + 1) + i) * V, V, a->cfg_scale, g);
        else
            memcpy(g, lc, sizeof(float) * V);
        if (compute_p)
            om_transform(g, V, a->temperature[b], a->top_k, st->p + (size_t)i * V);
    }
}

static void img_alloc(om_img* st, const om_model* o, const om_rollout_args* a) {
    const int V = o->m.V, W = a->W, T = o->T;
    const int ncfg = a->cfg_scale != 0.0f ? 2 : 1;
    memset(st, 0, sizeof(*st));
    st->x = (int*)calloc(T + 1, sizeof(int));
    st->wz = (int*)calloc(W, sizeof(int));
    st->nz = (int*)calloc(W, sizeof(int));
    st->wmass = (int*)calloc(W, sizeof(int));
    st->nmass = (int*)calloc(W, sizeof(int));
    st->wq = (float*)calloc((size_t)W * V, sizeof(float));
    st->nq = (float*)calloc((size_t)W * V, sizeof(float));
    st->logits = (float*)calloc((size_t)ncfg * (W + 1) * V, sizeof(float));
    st->guided = (float*)calloc((size_t)(W + 1) * V, sizeof(float));
    st->p = (float*)calloc((size_t)(W + 1) * V, sizeof(float));
    st->resid = (float*)calloc(V, sizeof(float));
    for (int br = 0; br < ncfg; ++br) cache_init(&st->cache[br], o, T + W + 1);
    scratch_init(&st->s, o, T + W + 1);
}

static void img_free(om_img* st, const om_rollout_args* a) {
    const int ncfg = a->cfg_scale != 0.0f ? 2 : 1;
    free(st->x); free(st->wz); free(st->nz); free(st->wmass); free(st->nmass);
    free(st->wq); free(st->nq); free(st->logits); free(st->guided); free(st->p);
    free(st->resid);
    for (int br = 0; br < ncfg; ++br) cache_free(&st->cache[br]);
    scratch_free(&st->s);
}

/* Prefill [class, x_1..x_k] and draw the first window. */
static void img_prefill(const om_model* o, const om_rollout_args* a, om_img* st, int b) {
    const int T = o->T;
    const int k = a->prefix_len[b];
    st->k = k;
    st->n = k;
    for (int t = 1; t <= k; ++t) st->x[t] = a->prefix_tokens[(size_t)b * T + t - 1];
    st->active = k < T;
    st->e = k + a->W < T ? k + a->W : T;
    if (!st->active) return;
    const int ncfg = a->cfg_scale != 0.0f ? 2 : 1;
    /* positions 0..k-1 go through the cache only; position k gives the logits */
    for (int br = 0; br < ncfg; ++br) {
        for (int p = 0; p < k; ++p) {
            const int tok = p == 0 ? (br == 0 ? -(a->labels[b] + 1) : -(o->m.C + 1))
                                   : st->x[p];
            om_step(o, &st->cache[br], &st->s, p, tok, NULL);
        }
    }
    int last = k == 0 ? -1 : st->x[k];
    window_forward(o, a, st, b, k, 1, &last, !a->greedy);
    refresh_window(o, a, st, b, k, k, 1);
}

/* One round for one active image: forward, verify, commit, refresh. */
static int img_round(const om_model* o, const om_rollout_args* a, om_img* st, int b) {
    const int T = o->T, V = o->m.V, W = a->W;
    const int n = st->n;
    const int lim = a->sync ? st->e : T;
    const int We = W < lim - n ? W : lim - n;
    if (We == 0) {
        /* waiting at a shared window boundary: row 0 only, nothing verified */
        const int last = n == 0 ? -1 : st->x[n];
        window_forward(o, a, st, b, n, 1, &last, !a->greedy);
        refresh_window(o, a, st, b, n, n, 1);
        return 0;
    }
    int* rt = (int*)malloc(sizeof(int) * (We + 1));
    rt[0] = n == 0 ? -1 : st->x[n];
    for (int i = 1; i <= We; ++i) rt[i] = st->wz[i - 1];
    window_forward(o, a, st, b, n, We + 1, rt, !a->greedy);
    free(rt);
    int count = We, rejected = 0;
    int* committed = (int*)malloc(sizeof(int) * We);
    if (a->greedy) {
        for (int j = 1; j <= We; ++j) {
            const int am = om_argmax(st->guided + (size_t)(j - 1) * V, V);
            committed[j - 1] = am;
            if (am != st->wz[j - 1]) {
                count = j;
                rejected = 1;
                break;
            }
        }
    } else {
        const float** pr = (const float**)malloc(sizeof(float*) * We);
        const float** qr = (const float**)malloc(sizeof(float*) * We);
        float* ua = (float*)malloc(sizeof(float) * We);
        float* ur = (float*)malloc(sizeof(float) * We);
        for (int j = 1; j <= We; ++j) {
            pr[j - 1] = st->p + (size_t)(j - 1) * V;
            qr[j - 1] = st->wq + (size_t)(j - 1) * V;
            const om_uniforms u = uniforms(a->seed, b, n + j);
            ua[j - 1] = u.acc;
            ur[j - 1] = u.res;
        }
        count = verify_window(We, V, pr, qr, st->wmass, st->wz, ua, ur, st->resid, committed,
                              &rejected);
        free(pr); free(qr); free(ua); free(ur);
    }
    for (int j = 1; j <= count; ++j) st->x[n + j] = committed[j - 1];
    free(committed);
    st->verified += count;
    st->rejected += rejected;
    st->n = n + count;
    if (st->n >= T) {
        st->active = 0;
    } else {
        refresh_window(o, a, st, b, st->n, n, We + 1);
    }
    return count;
}

/* Full execution also runs finished images' rows (positions T..T+W) without
   touching their state; the outputs are thrown away. */
static void img_wasted_rows(const om_model* o, const om_rollout_args* a, om_img* st, int b) {
    const int T = o->T, W = a->W;
    int* rt = (int*)calloc(W + 1, sizeof(int));
    rt[0] = T >= 1 ? st->x[T] : -1;
    window_forward(o, a, st, b, T, W + 1, rt, 0);
    free(rt);
}

static void record_window(const om_model* o, const om_rollout_args* a, const om_img* st,
                          int* dr, float* q) {
    const int W = a->W, T = o->T, V = o->m.V;
    for (int b = 0; b < a->B; ++b) {
        const om_img* s = &st[b];
        const int span = s->n < T ? (W < T - s->n ? W : T - s->n) : 0;
        for (int m = 0; m < W; ++m) {
            int z = -1;
            float qz = 0.0f;
            if (m < span) {
                z = s->wz[m];
                qz = (a->greedy || s->wmass[m]) ? 1.0f : s->wq[(size_t)m * V + z];
            }
            dr[(size_t)b * W + m] = z;
            q[(size_t)b * W + m] = qz;
        }
    }
}

int om_rollout(const om_model* o, const om_rollout_args* a, om_rollout_out* out) {
    const int B = a->B, T = o->T;
    if (a->W < 1 || a->H < 1 || B < 1) return -1;
    om_img* st = (om_img*)calloc(B, sizeof(om_img));
    for (int b = 0; b < B; ++b) img_alloc(&st[b], o, a);
#pragma omp parallel for schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) img_prefill(o, a, &st[b], b);
    const size_t tw = (size_t)B * a->W;
    if (out->trace_drafts && out->trace_q)
        record_window(o, a, st, out->trace_drafts, out->trace_q);
    int rounds = 0, status = 0;
    for (;;) {
        int A = 0;
        for (int b = 0; b < B; ++b) A += st[b].active;
        if (A == 0) break;
        if (rounds >= a->max_rounds) { status = -2; break; }
        if (a->sync) {
            /* the batch moves to the next window once no active image has
               drafts of the current one left to verify */
            int pending = 0;
            for (int b = 0; b < B; ++b) pending |= st[b].active && st[b].n < st[b].e;
            if (!pending)
                for (int b = 0; b < B; ++b) st[b].e = st[b].e + a->W < T ? st[b].e + a->W : T;
        }
        const int full = a->exec_mode == 0 || (a->exec_mode == 2 && A > a->gamma);
        if (out->active_hist) out->active_hist[rounds] = A;
        if (out->mode_hist) out->mode_hist[rounds] = full ? 0 : 1;
        int* cnt = out->counts + (size_t)rounds * B;
#pragma omp parallel for schedule(dynamic, 1)
        for (int b = 0; b < B; ++b) {
            cnt[b] = 0;
            if (st[b].active)
                cnt[b] = img_round(o, a, &st[b], b);
            else if (full)
                img_wasted_rows(o, a, &st[b], b);
        }
        ++rounds;
        if (out->trace_drafts && out->trace_q)
            record_window(o, a, st, out->trace_drafts + rounds * tw, out->trace_q + rounds * tw);
    }
    *out->rounds = rounds;
    long verified = 0, rejected = 0, imgrounds = 0;
    for (int b = 0; b < B; ++b) {
        for (int t = 1; t <= T; ++t) out->tokens[(size_t)b * T + t - 1] = st[b].x[t];
        verified += st[b].verified;
        rejected += st[b].rejected;
    }
    for (int r = 0; r < rounds; ++r)
        for (int b = 0; b < B; ++b) imgrounds += out->counts[(size_t)r * B + b] > 0;
    if (out->stats) {
        out->stats[0] = verified;
        out->stats[1] = rejected;
        out->stats[2] = imgrounds;
    }
    for (int b = 0; b < B; ++b) img_free(&st[b], a);
    free(st);
    return status;
}

/* Token-by-token reference: x_t = F^-1(D(logits at t-1), u_draft(b, t)), or the
   argmax in greedy mode, for t = k_b+1..T. */
int om_rollout_ar(const om_model* o, const om_rollout_args* a, int* tokens) {
    const int B = a->B, T = o->T, V = o->m.V;
    const int ncfg = a->cfg_scale != 0.0f ? 2 : 1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
        om_cache c[2];
        om_scratch s;
        for (int br = 0; br < ncfg; ++br) cache_init(&c[br], o, T + 1);
        scratch_init(&s, o, T + 1);
        float* lg = (float*)malloc(sizeof(float) * 2 * V);
        float* g = (float*)malloc(sizeof(float) * V);
        float* p = (float*)malloc(sizeof(float) * V);
        int* x = tokens + (size_t)b * T;
        const int k = a->prefix_len[b];
        for (int t = 0; t < k; ++t) x[t] = a->prefix_tokens[(size_t)b * T + t];
        for (int pos = 0; pos < T; ++pos) {
            for (int br = 0; br < ncfg; ++br) {
                const int tok = pos == 0 ? (br == 0 ? -(a->labels[b] + 1) : -(o->m.C + 1))
                                         : x[pos - 1];
                om_step(o, &c[br], &s, pos, tok, pos >= k ? lg + (size_t)br * V : NULL);
            }
            if (pos < k) continue;
            if (ncfg == 2)
                om_cfg_combine(lg, lg + V, V, a->cfg_scale, g);
            else
                memcpy(g, lg, sizeof(float) * V);
            int tok;
            if (a->greedy) {
                tok = om_argmax(g, V);
            } else {
                om_transform(g, V, a->temperature[b], a->top_k, p);
                tok = om_inv_cdf(p, V, uniforms(a->seed, b, pos + 1).draft);
            }
            x[pos] = tok;
        }
        for (int br = 0; br < ncfg; ++br) cache_free(&c[br]);
        scratch_free(&s);
        free(lg); free(g); free(p);
    }
    return 0;
}
