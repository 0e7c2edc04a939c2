/*
 * rl_oracle.c -- plain, slow, CPU reference of one RL-rollout decode step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or constant
 * generator with the GPU library.
 *
 * What it computes (the paper, RLinf, arXiv 2509.15965):
 *   - Generation in a GRPO iteration samples several responses per query,
 *     and the per-token log-probabilities of those responses are what the
 *     RL loss consumes (Sec. 2.1, GRPO workflow: Generation / Inference).
 *   - One forward pass yields both the sampled action token and its
 *     log-probability (Sec. 5.1.2, LIBERO results).
 *   - Sampling temperature is a knob (0.6 and 1.0 in Sec. 5.2).
 *   The paper never writes out the policy network.  The policy models it
 *   trains (Qwen2.5 in Sec. 5.1.1, OpenVLA on a Llama-2 backbone in
 *   Sec. 5.1.2) are pre-norm decoders with RMSNorm, rotate-half RoPE,
 *   grouped-query attention, SwiGLU MLP and an untied LM head; that is the
 *   function written out below, with no biases.  The mixture-of-experts
 *   policy it also names (Qwen3-30B-A3B, Sec. 5.1.1) replaces each layer's
 *   MLP by E SwiGLU experts of which each token uses its top k: a router
 *   row r = h . W_r^T (stored fp32), the k largest entries of r (equal
 *   values: the lower expert first), weights w = softmax of those k entries,
 *   MLP output = sum_j w_j * expert_{e_j}(h) in selection order.
 *
 * Precision model (the same function the GPU path must compute):
 *   - every dot product, norm statistic, softmax and log-sum-exp is
 *     accumulated in fp64;
 *   - values are rounded to the model storage type ("bf()") exactly where
 *     the GPU stores them: GEMM/attention inputs, the KV cache, q after
 *     RoPE, the attention output and the SwiGLU product;
 *   - the residual stream and the logits are stored as fp32.
 *   mode ORC_FP64 skips every rounding (used to compare with a brute-force
 *   full-sequence forward), ORC_FP32 rounds to fp32, ORC_BF16 rounds to
 *   bf16 with round-to-nearest-even.
 *
 * Sampling (Gumbel-max, counter-based noise):
 *   zt_v = fl32(z_v / T); logp(y) = zt_y - LSE(zt);
 *   u_v  = (x_v + 1/2) * 2^-32, x_v a Philox4x32-10 output word;
 *   g_v  = fl32(-log(-log(u_v))) evaluated in fp64;
 *   y    = argmax_v fl32(zt_v + g_v), exact ties to the lowest v;
 *   T == 0 selects argmax_v z_v and reports the T = 1 log-probability.
 *   Philox4x32-10 is taken from Salmon, Moraes, Dror, Shaw, "Parallel
 *   random numbers: as easy as 1, 2, 3" (SC'11): key (seed lo, seed hi),
 *   counter (v / 4, position of the new token, uid lo, uid hi), word v % 4.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_FP64 = 0, ORC_FP32 = 1, ORC_BF16 = 2 };   /* storage mode   */
enum { ORC_W_F32 = 0, ORC_W_BF16 = 1 };               /* weight encoding */

/* ------------------------------------------------------------------ */
/* rounding helpers                                                    */
/* ------------------------------------------------------------------ */

/* Round a double to the nearest bf16 value (ties to even), returned as a
 * double.  bf16 keeps 8 significant bits: drop the low 45 of the 52
 * stored double mantissa bits with round-to-nearest-even. */
double orc_round_bf16(double x)
{
    if (isnan(x) || isinf(x) || x == 0.0) return x;
    if (fabs(x) < 1.1754943508222875e-38) {          /* below fp32 normal range */
        float f = (float)x;                           /* subnormal: via fp32   */
        uint32_t u; memcpy(&u, &f, 4);
        uint32_t lsb = (u >> 16) & 1u;
        u += 0x7FFFu + lsb; u &= 0xFFFF0000u;
        memcpy(&f, &u, 4);
        return (double)f;
    }
    uint64_t u; memcpy(&u, &x, 8);
    uint64_t lsb = (u >> 45) & 1ull;
    u += ((1ull << 44) - 1ull) + lsb;
    u &= ~((1ull << 45) - 1ull);
    double r; memcpy(&r, &u, 8);
    if (fabs(r) > 3.3895313892515355e38) r = copysign(INFINITY, x);  /* > bf16 max */
    return r;
}

static double store_round(int mode, double x)   /* bf() */
{
    if (mode == ORC_FP64) return x;
    if (mode == ORC_FP32) return (double)(float)x;
    return orc_round_bf16(x);
}

static double resid_round(int mode, double x)   /* fp32 residual / logits */
{
    return mode == ORC_FP64 ? x : (double)(float)x;
}

static double bf16_bits_to_double(uint16_t b)
{
    uint32_t u = ((uint32_t)b) << 16;
    float f; memcpy(&f, &u, 4);
    return (double)f;
}

static double wget(int wdt, const void* p, size_t i)
{
    if (wdt == ORC_W_BF16) return bf16_bits_to_double(((const uint16_t*)p)[i]);
    return (double)((const float*)p)[i];
}

/* ------------------------------------------------------------------ */
/* Philox4x32-10 (SC'11)                                               */
/* ------------------------------------------------------------------ */

void orc_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;   /* round multipliers */
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;   /* Weyl key bumps    */
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) { k0 += W0; k1 += W1; }
        uint64_t p0 = (uint64_t)M0 * (uint64_t)c0;
        uint64_t p1 = (uint64_t)M1 * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* 32-bit noise word for vocabulary entry v of the token at position
 * pos_new of sequence uid. */
uint32_t orc_noise_word(uint64_t seed, uint64_t uid, int32_t pos_new, int64_t v)
{
    uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
    uint32_t ctr[4] = { (uint32_t)(v / 4), (uint32_t)pos_new, (uint32_t)uid, (uint32_t)(uid >> 32) };
    uint32_t out[4];
    orc_philox4x32_10(ctr, key, out);
    return out[v % 4];
}

/* Gumbel noise of one 32-bit word: fp64 evaluation, rounded to fp32. */
float orc_gumbel_of_word(uint32_t x)
{
    double u = ((double)x + 0.5) * 2.3283064365386963e-10;   /* 2^-32 */
    return (float)(-log(-log(u)));
}

/* Gumbel-max with caller-given uniforms u[V] (for hand-built cases).
 * Returns the selected index; ties go to the lowest index. */
int32_t orc_gumbel_argmax_u(const float* z, const double* u, int32_t V, float T)
{
    int32_t best = 0; float bests = 0.f;
    for (int32_t v = 0; v < V; ++v) {
        float zt = z[v] / T;
        float g = (float)(-log(-log(u[v])));
        float s = zt + g;
        if (v == 0 || s > bests) { bests = s; best = v; }
    }
    return best;
}

/* Sample one token from fp32 logits z[V] and report a log-probability.
 * forced >= 0 selects whose log-probability is reported. */
void orc_sample(const float* z, int32_t V, float T, uint64_t seed, uint64_t uid,
                int32_t pos_new, int32_t forced, int32_t* tok_out, double* logp_out)
{
    int32_t y = 0;
    double lse;
    if (T == 0.0f) {
        float best = z[0];
        for (int32_t v = 1; v < V; ++v) if (z[v] > best) { best = z[v]; y = v; }
        double m = (double)best, s = 0.0;
        for (int32_t v = 0; v < V; ++v) s += exp((double)z[v] - m);
        lse = m + log(s);
        int32_t r = forced >= 0 ? forced : y;
        *tok_out = y;
        *logp_out = (double)z[r] - lse;
        return;
    }
    float bests = 0.f;
    double m = -INFINITY;
    for (int32_t v = 0; v < V; ++v) {
        float zt = z[v] / T;
        if ((double)zt > m) m = (double)zt;
        float g = orc_gumbel_of_word(orc_noise_word(seed, uid, pos_new, v));
        float s = zt + g;
        if (v == 0 || s > bests) { bests = s; y = v; }
    }
    double s = 0.0;
    for (int32_t v = 0; v < V; ++v) s += exp((double)(z[v] / T) - m);
    lse = m + log(s);
    int32_t r = forced >= 0 ? forced : y;
    *tok_out = y;
    *logp_out = (double)(z[r] / T) - lse;
}

/* Log-probability of token y under temperature T: fl32(z_y / T) - LSE(fl32(z / T)),
 * the same quantity the sampler reports, with no draw.  This is what the
 * inference stage computes for every generated token (Sec. 2.1, GRPO: the
 * log-probabilities of the responses, from a forward pass over them).
 * T == 0 reports the T = 1 value (as the arg-max sampler does).
 * y outside [0, V) returns NaN. */
double orc_logprob(const float* z, int32_t V, float T, int32_t y)
{
    if (y < 0 || y >= V) return NAN;
    const int scaled = T != 0.0f;
    double m = -INFINITY;
    for (int32_t v = 0; v < V; ++v) {
        double zt = scaled ? (double)(z[v] / T) : (double)z[v];
        if (zt > m) m = zt;
    }
    double s = 0.0;
    for (int32_t v = 0; v < V; ++v) {
        double zt = scaled ? (double)(z[v] / T) : (double)z[v];
        s += exp(zt - m);
    }
    double zy = scaled ? (double)(z[y] / T) : (double)z[y];
    return zy - (m + log(s));
}

/* Top-two perturbed scores of a draw (used to excuse near-tie flips). */
void orc_sample_margin(const float* z, int32_t V, float T, uint64_t seed, uint64_t uid,
                       int32_t pos_new, int32_t* first, int32_t* second, double* margin)
{
    float s1 = -INFINITY, s2 = -INFINITY; int32_t i1 = -1, i2 = -1;
    for (int32_t v = 0; v < V; ++v) {
        float s;
        if (T == 0.0f) s = z[v];
        else s = z[v] / T + orc_gumbel_of_word(orc_noise_word(seed, uid, pos_new, v));
        if (i1 < 0 || s > s1) { s2 = s1; i2 = i1; s1 = s; i1 = v; }
        else if (i2 < 0 || s > s2) { s2 = s; i2 = v; }
    }
    *first = i1; *second = i2; *margin = (double)s1 - (double)s2;
}

/* ------------------------------------------------------------------ */
/* building blocks                                                     */
/* ------------------------------------------------------------------ */

/* out = bf( x / sqrt(mean(x^2) + eps) * g ) */
void orc_rmsnorm(const double* x, int wdt, const void* g, size_t g_off, int32_t H,
                 double eps, int mode, double* out)
{
    double ss = 0.0;
    for (int32_t i = 0; i < H; ++i) ss += x[i] * x[i];
    double r = 1.0 / sqrt(ss / (double)H + eps);
    for (int32_t i = 0; i < H; ++i)
        out[i] = store_round(mode, x[i] * r * wget(wdt, g, g_off + (size_t)i));
}

/* y[r] = sum_k W[w_off + r*K + k] * x[k] for r in [0, R): fp64 accumulation */
void orc_matvec(int wdt, const void* W, size_t w_off, int32_t R, int32_t K,
                const double* x, double* y)
{
    #pragma omp parallel for schedule(static)
    for (int32_t r = 0; r < R; ++r) {
        double acc = 0.0;
        size_t base = w_off + (size_t)r * (size_t)K;
        if (wdt == ORC_W_BF16) {
            const uint16_t* w = (const uint16_t*)W + base;
            for (int32_t k = 0; k < K; ++k) acc += bf16_bits_to_double(w[k]) * x[k];
        } else {
            const float* w = (const float*)W + base;
            for (int32_t k = 0; k < K; ++k) acc += (double)w[k] * x[k];
        }
        y[r] = acc;
    }
}

/* cos and sin of the RoPE angle pos * theta^(-2i/D), angle in fp64,
 * results rounded to fp32. */
void orc_rope_cos_sin(int32_t pos, int32_t i, int32_t D, double theta, double* c, double* s)
{
    double w = pow(theta, -2.0 * (double)i / (double)D);
    double a = (double)pos * w;
    *c = (double)(float)cos(a);
    *s = (double)(float)sin(a);
}

/* rotate-half RoPE of one head vector v[D] in place (pairs i, i + D/2) */
void orc_rope(double* v, int32_t D, int32_t pos, double theta)
{
    int32_t h = D / 2;
    for (int32_t i = 0; i < h; ++i) {
        double c, s;
        orc_rope_cos_sin(pos, i, D, theta, &c, &s);
        double a = v[i], b = v[i + h];
        v[i] = a * c - b * s;
        v[i + h] = b * c + a * s;
    }
}

/* single-query softmax attention over n cached rows: out = softmax(q.K^T / sqrt(D)) V.
 * K and V rows are at K + t*stride, V + t*stride. */
void orc_attend(const double* q, const double* K, const double* Vv, int64_t stride,
                int32_t n, int32_t D, double* out)
{
    double* s = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    double m = -INFINITY;
    double scale = 1.0 / sqrt((double)D);
    for (int32_t t = 0; t < n; ++t) {
        double d = 0.0;
        for (int32_t i = 0; i < D; ++i) d += q[i] * K[(int64_t)t * stride + i];
        s[t] = d * scale;
        if (s[t] > m) m = s[t];
    }
    double l = 0.0;
    for (int32_t t = 0; t < n; ++t) { s[t] = exp(s[t] - m); l += s[t]; }
    for (int32_t i = 0; i < D; ++i) out[i] = 0.0;
    for (int32_t t = 0; t < n; ++t) {
        double a = s[t] / l;
        for (int32_t i = 0; i < D; ++i) out[i] += a * Vv[(int64_t)t * stride + i];
    }
    free(s);
}

/* ------------------------------------------------------------------ */
/* model and sequence state                                            */
/* ------------------------------------------------------------------ */

typedef struct {
    int32_t L, H, Hq, Hkv, D, F, V;
    double eps, theta;
    int32_t mode;    /* ORC_FP64 / ORC_FP32 / ORC_BF16 */
    int32_t wdt;     /* ORC_W_F32 / ORC_W_BF16 */
    /* weights, row-major [out][in]; layer tensors stacked over layers */
    const void* embed;      /* [V][H]                */
    const void* attn_norm;  /* [L][H]                */
    const void* w_qkv;      /* [L][(Hq+2Hkv)D][H]    */
    const void* w_o;        /* [L][H][Hq*D]          */
    const void* mlp_norm;   /* [L][H]                */
    const void* w_gate_up;  /* [L][2F][H], gate rows first */
    const void* w_down;     /* [L][H][F]             */
    const void* final_norm; /* [H]                   */
    const void* lm_head;    /* [V][H]                */
    /* mixture of experts (E > 0: replaces w_gate_up / w_down) */
    int32_t E, topk, Fe;
    const void* w_router;       /* [L][E][H]            */
    const void* w_exp_gate_up;  /* [L][E][2Fe][H], gate rows first */
    const void* w_exp_down;     /* [L][E][H][Fe]        */
} orc_model;

/* Top-k routing of one row: the k largest r[e] (equal values: lower e
 * first) in decreasing order, and their softmax weights. */
void orc_route(const double* r, int32_t E, int32_t k, int32_t* sel, double* w)
{
    for (int32_t j = 0; j < k; ++j) {
        int32_t best = -1;
        for (int32_t e = 0; e < E; ++e) {
            int taken = 0;
            for (int32_t i = 0; i < j; ++i) taken |= sel[i] == e;
            if (!taken && (best < 0 || r[e] > r[best])) best = e;
        }
        sel[j] = best;
    }
    double m = r[sel[0]], sum = 0.0;
    for (int32_t j = 0; j < k; ++j) { w[j] = exp(r[sel[j]] - m); sum += w[j]; }
    for (int32_t j = 0; j < k; ++j) w[j] /= sum;
}

typedef struct {
    int32_t max_ctx;
    int32_t len;         /* tokens already in the cache */
    double* K;           /* [L][max_ctx][Hkv][D] */
    double* Vc;          /* [L][max_ctx][Hkv][D] */
    double route_margin; /* smallest gap between a chosen router logit and the
                            largest one left out, over every routing so far
                            (a check that a test's routing has no near ties) */
} orc_seq;

orc_seq* orc_seq_create(const orc_model* m, int32_t max_ctx)
{
    orc_seq* s = (orc_seq*)calloc(1, sizeof(orc_seq));
    size_t n = (size_t)m->L * (size_t)max_ctx * (size_t)m->Hkv * (size_t)m->D;
    s->max_ctx = max_ctx;
    s->len = 0;
    s->route_margin = INFINITY;
    s->K = (double*)calloc(n, sizeof(double));
    s->Vc = (double*)calloc(n, sizeof(double));
    if (!s->K || !s->Vc) { free(s->K); free(s->Vc); free(s); return NULL; }
    return s;
}

void orc_seq_destroy(orc_seq* s)
{
    if (!s) return;
    free(s->K); free(s->Vc); free(s);
}

/* Duplicate a sequence's cache and length (same max_ctx and model). */
orc_seq* orc_seq_clone(const orc_model* m, const orc_seq* src)
{
    orc_seq* d = orc_seq_create(m, src->max_ctx);
    if (!d) return NULL;
    size_t n = (size_t)m->L * (size_t)src->max_ctx * (size_t)m->Hkv * (size_t)m->D;
    memcpy(d->K, src->K, n * sizeof(double));
    memcpy(d->Vc, src->Vc, n * sizeof(double));
    d->len = src->len;
    d->route_margin = src->route_margin;
    return d;
}

double orc_seq_route_margin(const orc_seq* s) { return s->route_margin; }

int32_t orc_seq_len(const orc_seq* s) { return s->len; }
void orc_seq_set_len(orc_seq* s, int32_t len) { s->len = len; }

static size_t kv_index(const orc_model* m, const orc_seq* s, int32_t l, int32_t t, int32_t g)
{
    return (((size_t)l * (size_t)s->max_ctx + (size_t)t) * (size_t)m->Hkv + (size_t)g) * (size_t)m->D;
}

/* Store given K and V rows (already in storage precision) at (layer, pos, kv-head). */
void orc_seq_set_kv(const orc_model* m, orc_seq* s, int32_t l, int32_t t, int32_t g,
                    const double* k, const double* v)
{
    size_t b = kv_index(m, s, l, t, g);
    memcpy(s->K + b, k, sizeof(double) * (size_t)m->D);
    memcpy(s->Vc + b, v, sizeof(double) * (size_t)m->D);
}

/* Store n consecutive positions 0..n-1 of (layer, kv-head): K and V are
 * [n][D] row-major, already in storage precision. */
void orc_seq_set_kv_block(const orc_model* m, orc_seq* s, int32_t l, int32_t g, int32_t n,
                          const double* K, const double* V)
{
    for (int32_t t = 0; t < n; ++t) {
        size_t b = kv_index(m, s, l, t, g);
        memcpy(s->K + b, K + (size_t)t * (size_t)m->D, sizeof(double) * (size_t)m->D);
        memcpy(s->Vc + b, V + (size_t)t * (size_t)m->D, sizeof(double) * (size_t)m->D);
    }
}

void orc_seq_get_kv(const orc_model* m, const orc_seq* s, int32_t l, int32_t t, int32_t g,
                    double* k, double* v)
{
    size_t b = kv_index(m, s, l, t, g);
    memcpy(k, s->K + b, sizeof(double) * (size_t)m->D);
    memcpy(v, s->Vc + b, sizeof(double) * (size_t)m->D);
}

/* Run one token through the decoder at position s->len, append its K/V,
 * advance s->len and write the fp32 logits (as doubles) to logits[V].
 *   tok >= 0 : embedding row tok
 *   tok <  0 : the given row `embed_row` (model weight encoding, H values)
 * Returns 0 on success, -1 if the cache is full, -2 on allocation failure. */
int orc_forward_token(const orc_model* m, orc_seq* s, int32_t tok, const void* embed_row,
                      double* logits)
{
    const int32_t H = m->H, Hq = m->Hq, Hkv = m->Hkv, D = m->D, F = m->F, V = m->V;
    const int32_t G = Hq / Hkv;
    const int32_t pos = s->len;
    const int32_t NQKV = (Hq + 2 * Hkv) * D;
    const int mode = m->mode, wdt = m->wdt;
    if (pos >= s->max_ctx) return -1;

    double* x    = (double*)malloc(sizeof(double) * (size_t)H);
    double* h    = (double*)malloc(sizeof(double) * (size_t)H);
    double* qkv  = (double*)malloc(sizeof(double) * (size_t)NQKV);
    double* att  = (double*)malloc(sizeof(double) * (size_t)Hq * (size_t)D);
    const int32_t E = m->E, Fe = m->Fe, FF = E > 0 ? Fe : F;
    double* y    = (double*)malloc(sizeof(double) * (size_t)(H > 2 * FF ? H : 2 * FF));
    double* mm   = (double*)malloc(sizeof(double) * (size_t)FF);
    double* r    = (double*)malloc(sizeof(double) * (size_t)(E > 0 ? E : 1));
    double* acc  = (double*)malloc(sizeof(double) * (size_t)H);
    double* y2   = (double*)malloc(sizeof(double) * (size_t)H);
    int32_t* sel = (int32_t*)malloc(sizeof(int32_t) * (size_t)(m->topk > 0 ? m->topk : 1));
    double* wsel = (double*)malloc(sizeof(double) * (size_t)(m->topk > 0 ? m->topk : 1));
    if (!x || !h || !qkv || !att || !y || !mm || !r || !acc || !y2 || !sel || !wsel) {
        free(x); free(h); free(qkv); free(att); free(y); free(mm);
        free(r); free(acc); free(y2); free(sel); free(wsel);
        return -2;
    }

    /* 1. embedding into the fp32 residual stream */
    for (int32_t i = 0; i < H; ++i) {
        double e = tok >= 0 ? wget(wdt, m->embed, (size_t)tok * (size_t)H + (size_t)i)
                            : wget(wdt, embed_row, (size_t)i);
        x[i] = resid_round(mode, e);
    }

    for (int32_t l = 0; l < m->L; ++l) {
        /* 2a. attention RMSNorm */
        orc_rmsnorm(x, wdt, m->attn_norm, (size_t)l * (size_t)H, H, m->eps, mode, h);
        /* 2b. fused q|k|v projection */
        orc_matvec(wdt, m->w_qkv, (size_t)l * (size_t)NQKV * (size_t)H, NQKV, H, h, qkv);
        double* q = qkv;
        double* k = qkv + (size_t)Hq * D;
        double* v = k + (size_t)Hkv * D;
        /* 2c. RoPE on q and k, then storage rounding; 2d. append to the cache */
        for (int32_t j = 0; j < Hq; ++j) {
            orc_rope(q + (size_t)j * D, D, pos, m->theta);
            for (int32_t i = 0; i < D; ++i) q[(size_t)j * D + i] = store_round(mode, q[(size_t)j * D + i]);
        }
        for (int32_t g = 0; g < Hkv; ++g) {
            orc_rope(k + (size_t)g * D, D, pos, m->theta);
            size_t b = kv_index(m, s, l, pos, g);
            for (int32_t i = 0; i < D; ++i) {
                s->K[b + i]  = store_round(mode, k[(size_t)g * D + i]);
                s->Vc[b + i] = store_round(mode, v[(size_t)g * D + i]);
            }
        }
        /* 2e. grouped-query attention over positions 0..pos; q-head j reads
         *     kv-head j / G (contiguous groups) */
        #pragma omp parallel for schedule(static)
        for (int32_t j = 0; j < Hq; ++j) {
            int32_t g = j / G;
            size_t b0 = kv_index(m, s, l, 0, g);
            orc_attend(q + (size_t)j * D, s->K + b0, s->Vc + b0, (int64_t)Hkv * D,
                       pos + 1, D, att + (size_t)j * D);
        }
        for (int32_t i = 0; i < Hq * D; ++i) att[i] = store_round(mode, att[i]);
        /* 2f. output projection into the residual stream */
        orc_matvec(wdt, m->w_o, (size_t)l * (size_t)H * (size_t)Hq * (size_t)D, H, Hq * D, att, y);
        for (int32_t i = 0; i < H; ++i) x[i] = resid_round(mode, x[i] + y[i]);
        /* 2g. SwiGLU MLP */
        orc_rmsnorm(x, wdt, m->mlp_norm, (size_t)l * (size_t)H, H, m->eps, mode, h);
        if (E == 0) {
            orc_matvec(wdt, m->w_gate_up, (size_t)l * 2u * (size_t)F * (size_t)H, 2 * F, H, h, y);
            for (int32_t i = 0; i < F; ++i) {
                double a = y[i], b = y[F + i];
                double silu = a / (1.0 + exp(-a));
                mm[i] = store_round(mode, silu * b);
            }
            orc_matvec(wdt, m->w_down, (size_t)l * (size_t)H * (size_t)F, H, F, mm, y);
            for (int32_t i = 0; i < H; ++i) x[i] = resid_round(mode, x[i] + y[i]);
        } else {
            /* 2g'. mixture of experts: route, then the selected SwiGLU experts */
            orc_matvec(wdt, m->w_router, (size_t)l * (size_t)E * (size_t)H, E, H, h, r);
            for (int32_t e = 0; e < E; ++e) r[e] = resid_round(mode, r[e]);
            orc_route(r, E, m->topk, sel, wsel);
            for (int32_t e = 0; e < E; ++e) {
                int chosen = 0;
                for (int32_t j = 0; j < m->topk; ++j) chosen |= sel[j] == e;
                if (!chosen && r[sel[m->topk - 1]] - r[e] < s->route_margin) s->route_margin = r[sel[m->topk - 1]] - r[e];
            }
            for (int32_t i = 0; i < H; ++i) acc[i] = 0.0;
            for (int32_t j = 0; j < m->topk; ++j) {
                const size_t ex = (size_t)l * (size_t)E + (size_t)sel[j];
                orc_matvec(wdt, m->w_exp_gate_up, ex * 2u * (size_t)Fe * (size_t)H, 2 * Fe, H, h, y);
                for (int32_t i = 0; i < Fe; ++i) {
                    double a = y[i], b = y[Fe + i];
                    double silu = a / (1.0 + exp(-a));
                    mm[i] = store_round(mode, silu * b);
                }
                orc_matvec(wdt, m->w_exp_down, ex * (size_t)H * (size_t)Fe, H, Fe, mm, y2);
                for (int32_t i = 0; i < H; ++i) acc[i] += wsel[j] * y2[i];
            }
            for (int32_t i = 0; i < H; ++i) x[i] = resid_round(mode, x[i] + acc[i]);
        }
    }

    /* 3. final norm and LM head (fp32 logits) */
    orc_rmsnorm(x, wdt, m->final_norm, 0, H, m->eps, mode, h);
    orc_matvec(wdt, m->lm_head, 0, V, H, h, logits);
    for (int32_t v = 0; v < V; ++v) logits[v] = resid_round(mode, logits[v]);

    s->len = pos + 1;
    free(x); free(h); free(qkv); free(att); free(y); free(mm);
    free(r); free(acc); free(y2); free(sel); free(wsel);
    return 0;
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void orc_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

size_t orc_model_size(void) { return sizeof(orc_model); }
