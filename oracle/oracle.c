/*
 * Plain CPU oracle for the sparse parameter-store training step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the tests, the package's smoke check and the
 * benchmark's CPU-baseline leg do.  It shares no code, header, table or
 * helper with the GPU library; the two meet only in the seeded inputs the
 * tests hand to both.
 *
 * What it computes (one deterministic synchronous minibatch step):
 *   1. every worker reads the rows it needs from the store by key
 *      (the parameter manager's global read access, Section 1 and the
 *      co-located store of Section 4 / Figure 3);
 *   2. per-occurrence gradients are computed from those pre-step values for
 *      the task at hand (Appendix C, "Task details": MF, ComplEx KGE,
 *      skip-gram word vectors, CTR embeddings);
 *   3. the updates of all occurrences of one key are merged (the owner
 *      "merges the replica updates into its parameter store", Appendix B.1.2)
 *      here by a sum, in occurrence order, in double precision;
 *   4. one AdaGrad step per key (all five tasks train "SGD with AdaGrad",
 *      Appendix C) with a per-element float accumulator.
 * The paper gives none of these formulas; the readings taken where it is
 * silent are: diagonal AdaGrad with eps outside the square root and a zero
 * initial accumulator, a sum over duplicate keys, fp64 accumulation of every
 * multi-term sum with one fp32 rounding, and the task losses written below.
 *
 * Everything is written for clarity, not speed: one thread, qsort for the
 * stable sort (ties broken by occurrence index), materialized per-occurrence
 * gradient rows, sequential sums.  Compile with -ffp-contract=off and without
 * -ffast-math so that every float operation rounds exactly once, in the
 * order written.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_API __attribute__((visibility("default")))

/* ------------------------------------------------------------------------ */
/* small scalar helpers                                                      */
/* ------------------------------------------------------------------------ */

/* logistic function 1/(1+e^-x), evaluated without overflow */
static double sigmoid(double x)
{
    if (x >= 0.0) return 1.0 / (1.0 + exp(-x));
    double e = exp(x);
    return e / (1.0 + e);
}

/* softplus(x) = log(1 + e^x), evaluated without overflow */
static double softplus(double x)
{
    if (x > 0.0) return x + log1p(exp(-x));
    return log1p(exp(x));
}

static int key_ok(int64_t key, int64_t num_keys) { return key >= 0 && key < num_keys; }

/* ------------------------------------------------------------------------ */
/* read access: out[i] = W[keys[i]]  (Section 1, global read access)         */
/* A key outside [0, num_keys) yields a zero row and is counted.             */
/* ------------------------------------------------------------------------ */
ORC_API int64_t orc_pull(const float* W, int64_t num_keys, int32_t dim,
                         const int64_t* keys, int64_t n, float* out)
{
    int64_t bad = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (key_ok(keys[i], num_keys)) {
            memcpy(out + i * dim, W + keys[i] * dim, sizeof(float) * (size_t)dim);
        } else {
            memset(out + i * dim, 0, sizeof(float) * (size_t)dim);
            ++bad;
        }
    }
    return bad;
}

/* ------------------------------------------------------------------------ */
/* duplicate-key merge order: stable sort of occurrences by key              */
/* (Appendix B.1.2: updates to one parameter are merged at its store).       */
/* Invalid keys are given the sentinel num_keys, so they sort after every    */
/* valid key, keep their occurrence order, and belong to no segment.         */
/* ------------------------------------------------------------------------ */
typedef struct {
    int64_t key;
    int64_t idx;
} occ_t;

static int occ_cmp(const void* pa, const void* pb)
{
    const occ_t* a = (const occ_t*)pa;
    const occ_t* b = (const occ_t*)pb;
    if (a->key != b->key) return a->key < b->key ? -1 : 1;
    if (a->idx != b->idx) return a->idx < b->idx ? -1 : 1;
    return 0;
}

/* Sorted occurrence list; returns the number of invalid keys. */
static int64_t sort_occurrences(int64_t num_keys, const int64_t* keys, int64_t n, occ_t* occ)
{
    int64_t bad = 0;
    for (int64_t i = 0; i < n; ++i) {
        int ok = key_ok(keys[i], num_keys);
        occ[i].key = ok ? keys[i] : num_keys;
        occ[i].idx = i;
        bad += !ok;
    }
    qsort(occ, (size_t)n, sizeof(occ_t), occ_cmp);
    return bad;
}

/* uniq[u]      : the u-th distinct valid key, ascending
 * perm[j]      : occurrence index at sorted position j (all n positions)
 * offsets[u]   : first sorted position of key uniq[u]; offsets[U] = #valid
 * *num_unique  : U
 * returns the number of invalid keys                                        */
ORC_API int64_t orc_dedup(int64_t num_keys, const int64_t* keys, int64_t n,
                          int64_t* uniq, int32_t* perm, int32_t* offsets, int32_t* num_unique)
{
    occ_t* occ = (occ_t*)malloc(sizeof(occ_t) * (size_t)(n > 0 ? n : 1));
    int64_t bad = sort_occurrences(num_keys, keys, n, occ);
    int32_t u = 0;
    int64_t j = 0;
    for (; j < n && occ[j].key < num_keys; ++j) {
        if (j == 0 || occ[j].key != occ[j - 1].key) {
            uniq[u] = occ[j].key;
            offsets[u] = (int32_t)j;
            ++u;
        }
    }
    offsets[u] = (int32_t)j;
    for (int64_t i = 0; i < n; ++i) perm[i] = (int32_t)occ[i].idx;
    *num_unique = u;
    free(occ);
    return bad;
}

/* ------------------------------------------------------------------------ */
/* AdaGrad on one row (Appendix C: every task trains with AdaGrad).          */
/* Diagonal form, fp32, in exactly this order for every element:             */
/*   G <- G + g*g ;  W <- W - lr * ( g / (sqrt(G) + eps) )                   */
/* ------------------------------------------------------------------------ */
ORC_API void orc_adagrad_row(float* w, float* acc, const float* g, int32_t dim, float lr, float eps)
{
    for (int32_t c = 0; c < dim; ++c) {
        float t = g[c] * g[c];
        float a = acc[c] + t;
        float s = sqrtf(a);
        float den = s + eps;
        float q = g[c] / den;
        float step = lr * q;
        acc[c] = a;
        w[c] = w[c] - step;
    }
}

/* ------------------------------------------------------------------------ */
/* Row-wise AdaGrad, an update variant with one accumulator per row instead  */
/* of one per element (a reading: the paper names AdaGrad only).  For the    */
/* merged gradient row g of a key, with its accumulator a (fp32):            */
/*   t = fp32( (sum_c g_c*g_c) / dim )   (products exact, sum in fp64)       */
/*   a <- a + t ;  then per element  W <- W - lr * ( g / (sqrt(a) + eps) )   */
/* in the same fp32 operation order as the per-element form.                 */
/* ------------------------------------------------------------------------ */
ORC_API void orc_adagrad_rowwise(float* w, float* acc, const float* g, int32_t dim, float lr, float eps)
{
    double sq = 0.0;
    for (int32_t c = 0; c < dim; ++c) sq += (double)g[c] * (double)g[c];
    float t = (float)(sq / (double)dim);
    float a = *acc + t;
    float s = sqrtf(a);
    float den = s + eps;
    for (int32_t c = 0; c < dim; ++c) {
        float q = g[c] / den;
        float step = lr * q;
        w[c] = w[c] - step;
    }
    *acc = a;
}

/* ------------------------------------------------------------------------ */
/* write access with merging: per distinct key, the fp64 sum of its          */
/* occurrences' gradient rows in occurrence order, rounded once to fp32,     */
/* then one AdaGrad step.  Invalid keys are ignored and counted.             */
/* ------------------------------------------------------------------------ */
ORC_API int64_t orc_push(float* W, float* G, int64_t num_keys, int32_t dim, float lr, float eps,
                         const int64_t* keys, int64_t n, const float* grads)
{
    occ_t* occ = (occ_t*)malloc(sizeof(occ_t) * (size_t)(n > 0 ? n : 1));
    double* sum = (double*)malloc(sizeof(double) * (size_t)dim);
    float* g32 = (float*)malloc(sizeof(float) * (size_t)dim);
    int64_t bad = sort_occurrences(num_keys, keys, n, occ);
    int64_t j = 0;
    while (j < n && occ[j].key < num_keys) {
        int64_t key = occ[j].key;
        for (int32_t c = 0; c < dim; ++c) sum[c] = 0.0;
        for (; j < n && occ[j].key == key; ++j) {
            const float* row = grads + occ[j].idx * dim;
            for (int32_t c = 0; c < dim; ++c) sum[c] += (double)row[c];
        }
        for (int32_t c = 0; c < dim; ++c) g32[c] = (float)sum[c];
        orc_adagrad_row(W + key * dim, G + key * dim, g32, dim, lr, eps);
    }
    free(g32);
    free(sum);
    free(occ);
    return bad;
}

/* ------------------------------------------------------------------------ */
/* Write access without merging: the asynchronous update semantics of the    */
/* paper's experiments (Section 5.1: asynchronous SGD; each worker's update   */
/* reaches the store on its own, with no merging of concurrent updates).    */
/* Reading: every occurrence's gradient row is its own AdaGrad step on its   */
/* key's row, the occurrences applied one after another in the order        */
/* order[0..n) (occurrence indices; NULL: index order).  A store that       */
/* applies them concurrently, each element atomically, ends, element by     */
/* element, where some such order ends.  Invalid keys are ignored, counted. */
/* ------------------------------------------------------------------------ */
ORC_API int64_t orc_push_sequential(float* W, float* G, int64_t num_keys, int32_t dim, float lr, float eps,
                                    const int64_t* keys, int64_t n, const float* grads, const int64_t* order)
{
    int64_t bad = 0;
    for (int64_t t = 0; t < n; ++t) {
        int64_t i = order ? order[t] : t;
        int64_t key = keys[i];
        if (!key_ok(key, num_keys)) {
            ++bad;
            continue;
        }
        orc_adagrad_row(W + key * dim, G + key * dim, grads + i * dim, dim, lr, eps);
    }
    return bad;
}

/* The same with row-wise AdaGrad: Gr holds one accumulator per key.         */
ORC_API int64_t orc_push_sequential_rowwise(float* W, float* Gr, int64_t num_keys, int32_t dim, float lr,
                                            float eps, const int64_t* keys, int64_t n, const float* grads,
                                            const int64_t* order)
{
    int64_t bad = 0;
    for (int64_t t = 0; t < n; ++t) {
        int64_t i = order ? order[t] : t;
        int64_t key = keys[i];
        if (!key_ok(key, num_keys)) {
            ++bad;
            continue;
        }
        orc_adagrad_rowwise(W + key * dim, Gr + key, grads + i * dim, dim, lr, eps);
    }
    return bad;
}

/* The same merge with row-wise AdaGrad: Gr holds one accumulator per key.   */
ORC_API int64_t orc_push_rowwise(float* W, float* Gr, int64_t num_keys, int32_t dim, float lr, float eps,
                                 const int64_t* keys, int64_t n, const float* grads)
{
    occ_t* occ = (occ_t*)malloc(sizeof(occ_t) * (size_t)(n > 0 ? n : 1));
    double* sum = (double*)malloc(sizeof(double) * (size_t)dim);
    float* g32 = (float*)malloc(sizeof(float) * (size_t)dim);
    int64_t bad = sort_occurrences(num_keys, keys, n, occ);
    int64_t j = 0;
    while (j < n && occ[j].key < num_keys) {
        int64_t key = occ[j].key;
        for (int32_t c = 0; c < dim; ++c) sum[c] = 0.0;
        for (; j < n && occ[j].key == key; ++j) {
            const float* row = grads + occ[j].idx * dim;
            for (int32_t c = 0; c < dim; ++c) sum[c] += (double)row[c];
        }
        for (int32_t c = 0; c < dim; ++c) g32[c] = (float)sum[c];
        orc_adagrad_rowwise(W + key * dim, Gr + key, g32, dim, lr, eps);
    }
    free(g32);
    free(sum);
    free(occ);
    return bad;
}

/* ------------------------------------------------------------------------ */
/* bf16 value storage, an update variant that halves the bytes of a value:  */
/* a bf16 word is the upper half of an fp32 word, so widening is exact;     */
/* narrowing rounds to the nearest bf16, ties to the even one (NaN stays a  */
/* quiet NaN).  Accumulators stay fp32; the updated value is narrowed once. */
/* ------------------------------------------------------------------------ */
ORC_API float orc_bf16_to_f32(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

ORC_API uint16_t orc_f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    uint32_t lower = u & 0xffffu;          /* the bits that are dropped */
    uint32_t upper = u >> 16;
    if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u))) upper += 1u;   /* carries into the exponent */
    return (uint16_t)upper;
}

ORC_API void orc_f32_to_bf16_array(const float* x, uint16_t* out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) out[i] = orc_f32_to_bf16(x[i]);
}

ORC_API int64_t orc_push_bf16(uint16_t* W, float* G, int64_t num_keys, int32_t dim, float lr, float eps,
                              const int64_t* keys, int64_t n, const float* grads)
{
    occ_t* occ = (occ_t*)malloc(sizeof(occ_t) * (size_t)(n > 0 ? n : 1));
    double* sum = (double*)malloc(sizeof(double) * (size_t)dim);
    float* g32 = (float*)malloc(sizeof(float) * (size_t)dim);
    float* w32 = (float*)malloc(sizeof(float) * (size_t)dim);
    int64_t bad = sort_occurrences(num_keys, keys, n, occ);
    int64_t j = 0;
    while (j < n && occ[j].key < num_keys) {
        int64_t key = occ[j].key;
        for (int32_t c = 0; c < dim; ++c) sum[c] = 0.0;
        for (; j < n && occ[j].key == key; ++j) {
            const float* row = grads + occ[j].idx * dim;
            for (int32_t c = 0; c < dim; ++c) sum[c] += (double)row[c];
        }
        for (int32_t c = 0; c < dim; ++c) {
            g32[c] = (float)sum[c];
            w32[c] = orc_bf16_to_f32(W[key * dim + c]);
        }
        orc_adagrad_row(w32, G + key * dim, g32, dim, lr, eps);
        for (int32_t c = 0; c < dim; ++c) W[key * dim + c] = orc_f32_to_bf16(w32[c]);
    }
    free(w32);
    free(g32);
    free(sum);
    free(occ);
    return bad;
}

/* ------------------------------------------------------------------------ */
/* Matrix factorization (Appendix C, "Matrix factorization"; Table 3).       */
/* Entry (i, j, v): u = W[i], m = W[col_off + j].                            */
/*   e = v - <u, m>                                                          */
/*   loss  = e^2/2 + lam/2 (|u|^2 + |m|^2)                                   */
/*   grad_u = lam*u - e*m ,  grad_m = lam*m - e*u                            */
/* Occurrences 2b (row key) and 2b+1 (column key).  An entry with a key      */
/* outside the table contributes nothing: its occurrence keys are -1.        */
/* Returns the loss; *bad gets the number of skipped entries.                */
/* ------------------------------------------------------------------------ */
ORC_API double orc_grad_mf(const float* W, int64_t num_keys, int32_t dim,
                           const int32_t* row, const int32_t* col, const float* val, int64_t B,
                           int64_t col_off, float lam, int64_t* okeys, float* ograds, int64_t* bad)
{
    double loss = 0.0;
    double lamd = (double)lam;
    *bad = 0;
    for (int64_t b = 0; b < B; ++b) {
        int64_t ku = (int64_t)row[b];
        int64_t km = col_off + (int64_t)col[b];
        float* gu = ograds + (2 * b) * dim;
        float* gm = ograds + (2 * b + 1) * dim;
        /* row factors occupy keys [0, col_off), column factors [col_off, num_keys) */
        if (!key_ok(ku, num_keys) || ku >= col_off || !key_ok(km, num_keys) || row[b] < 0 || col[b] < 0) {
            okeys[2 * b] = -1;
            okeys[2 * b + 1] = -1;
            memset(gu, 0, sizeof(float) * (size_t)dim);
            memset(gm, 0, sizeof(float) * (size_t)dim);
            ++*bad;
            continue;
        }
        const float* u = W + ku * dim;
        const float* m = W + km * dim;
        double dot = 0.0, nu = 0.0, nm = 0.0;
        for (int32_t c = 0; c < dim; ++c) {
            dot += (double)u[c] * (double)m[c];
            nu += (double)u[c] * (double)u[c];
            nm += (double)m[c] * (double)m[c];
        }
        double e = (double)val[b] - dot;
        loss += 0.5 * e * e + 0.5 * lamd * (nu + nm);
        for (int32_t c = 0; c < dim; ++c) {
            gu[c] = (float)(lamd * (double)u[c] - e * (double)m[c]);
            gm[c] = (float)(lamd * (double)m[c] - e * (double)u[c]);
        }
        okeys[2 * b] = ku;
        okeys[2 * b + 1] = km;
    }
    return loss;
}

/* ------------------------------------------------------------------------ */
/* ComplEx knowledge-graph embeddings (Appendix C, "Knowledge graph          */
/* embeddings": ComplEx trained with AdaGrad and uniform negative sampling). */
/* A row holds [Re(0..C-1) | Im(0..C-1)].  The ComplEx score is the real     */
/* part of sum_k s_k r_k conj(o_k):                                          */
/*   phi = sum_k sR rR oR + sI rR oI + sR rI oI - sI rI oR                   */
/* Logistic loss softplus(-y*phi) with y = +1 for the true triple and -1 for */
/* each corrupted one; d loss / d phi = -y * sigmoid(-y*phi).                */
/* Per triple: the true triple, n_head_neg triples with the head replaced by */
/* neg[j], then the rest with the tail replaced by neg[j].                   */
/* Occurrence order per triple: s, r, o, then one row per negative.          */
/* ------------------------------------------------------------------------ */
ORC_API double orc_complex_score(const float* s, const float* r, const float* o, int32_t cdim)
{
    const float *sR = s, *sI = s + cdim, *rR = r, *rI = r + cdim, *oR = o, *oI = o + cdim;
    double phi = 0.0;
    for (int32_t k = 0; k < cdim; ++k) {
        phi += (double)sR[k] * (double)rR[k] * (double)oR[k];
        phi += (double)sI[k] * (double)rR[k] * (double)oI[k];
        phi += (double)sR[k] * (double)rI[k] * (double)oI[k];
        phi -= (double)sI[k] * (double)rI[k] * (double)oR[k];
    }
    return phi;
}

/* acc += coef * d phi / d s  (depends on r, o) */
static void add_dphi_ds(double* acc, double coef, const float* r, const float* o, int32_t cdim)
{
    const float *rR = r, *rI = r + cdim, *oR = o, *oI = o + cdim;
    for (int32_t k = 0; k < cdim; ++k) {
        acc[k] += coef * ((double)rR[k] * (double)oR[k] + (double)rI[k] * (double)oI[k]);
        acc[cdim + k] += coef * ((double)rR[k] * (double)oI[k] - (double)rI[k] * (double)oR[k]);
    }
}

/* acc += coef * d phi / d r  (depends on s, o) */
static void add_dphi_dr(double* acc, double coef, const float* s, const float* o, int32_t cdim)
{
    const float *sR = s, *sI = s + cdim, *oR = o, *oI = o + cdim;
    for (int32_t k = 0; k < cdim; ++k) {
        acc[k] += coef * ((double)sR[k] * (double)oR[k] + (double)sI[k] * (double)oI[k]);
        acc[cdim + k] += coef * ((double)sR[k] * (double)oI[k] - (double)sI[k] * (double)oR[k]);
    }
}

/* acc += coef * d phi / d o  (depends on s, r) */
static void add_dphi_do(double* acc, double coef, const float* s, const float* r, int32_t cdim)
{
    const float *sR = s, *sI = s + cdim, *rR = r, *rI = r + cdim;
    for (int32_t k = 0; k < cdim; ++k) {
        acc[k] += coef * ((double)sR[k] * (double)rR[k] - (double)sI[k] * (double)rI[k]);
        acc[cdim + k] += coef * ((double)sI[k] * (double)rR[k] + (double)sR[k] * (double)rI[k]);
    }
}

static void round_row(float* dst, const double* src, int32_t dim)
{
    for (int32_t c = 0; c < dim; ++c) dst[c] = (float)src[c];
}

ORC_API double orc_grad_kge(const float* W, int64_t num_keys, int32_t dim,
                            const int32_t* head, const int32_t* rel, const int32_t* tail,
                            const int32_t* neg, int64_t B, int32_t n_neg, int32_t n_head_neg,
                            int64_t rel_off, int64_t* okeys, float* ograds, int64_t* bad)
{
    const int32_t cdim = dim / 2;
    const int64_t per = 3 + (int64_t)n_neg;
    double* gs = (double*)malloc(sizeof(double) * (size_t)dim);
    double* gr = (double*)malloc(sizeof(double) * (size_t)dim);
    double* go = (double*)malloc(sizeof(double) * (size_t)dim);
    double* gn = (double*)malloc(sizeof(double) * (size_t)dim);
    double loss = 0.0;
    *bad = 0;
    for (int64_t t = 0; t < B; ++t) {
        int64_t* kk = okeys + t * per;
        float* gg = ograds + t * per * dim;
        int64_t ks = head[t], kr = rel_off + (int64_t)rel[t], ko = tail[t];
        int ok = key_ok(ks, num_keys) && key_ok(kr, num_keys) && key_ok(ko, num_keys) && rel[t] >= 0;
        for (int32_t j = 0; j < n_neg; ++j) ok = ok && key_ok(neg[t * n_neg + j], num_keys);
        if (!ok) {
            for (int64_t q = 0; q < per; ++q) kk[q] = -1;
            memset(gg, 0, sizeof(float) * (size_t)(per * dim));
            ++*bad;
            continue;
        }
        const float* s = W + ks * dim;
        const float* r = W + kr * dim;
        const float* o = W + ko * dim;
        for (int32_t c = 0; c < dim; ++c) gs[c] = gr[c] = go[c] = 0.0;

        /* the true triple, y = +1 */
        double phi = orc_complex_score(s, r, o, cdim);
        double coef = -sigmoid(-phi);
        loss += softplus(-phi);
        add_dphi_ds(gs, coef, r, o, cdim);
        add_dphi_dr(gr, coef, s, o, cdim);
        add_dphi_do(go, coef, s, r, cdim);

        /* corrupted triples, y = -1 */
        for (int32_t j = 0; j < n_neg; ++j) {
            int64_t kn = neg[t * n_neg + j];
            const float* x = W + kn * dim;
            for (int32_t c = 0; c < dim; ++c) gn[c] = 0.0;
            if (j < n_head_neg) {          /* (x, r, o) */
                phi = orc_complex_score(x, r, o, cdim);
                coef = sigmoid(phi);
                add_dphi_ds(gn, coef, r, o, cdim);
                add_dphi_dr(gr, coef, x, o, cdim);
                add_dphi_do(go, coef, x, r, cdim);
            } else {                       /* (s, r, x) */
                phi = orc_complex_score(s, r, x, cdim);
                coef = sigmoid(phi);
                add_dphi_do(gn, coef, s, r, cdim);
                add_dphi_ds(gs, coef, r, x, cdim);
                add_dphi_dr(gr, coef, s, x, cdim);
            }
            loss += softplus(phi);
            kk[3 + j] = kn;
            round_row(gg + (3 + j) * dim, gn, dim);
        }
        kk[0] = ks;
        kk[1] = kr;
        kk[2] = ko;
        round_row(gg, gs, dim);
        round_row(gg + dim, gr, dim);
        round_row(gg + 2 * dim, go, dim);
    }
    free(gn);
    free(go);
    free(gr);
    free(gs);
    return loss;
}

/* ------------------------------------------------------------------------ */
/* Skip-gram with negative sampling (Appendix C, "Word vectors": word2vec    */
/* skip-gram, AdaGrad, negative sampling, window 5).  Input vectors have     */
/* keys [0, V), output vectors keys out_off + id.  For centre c with input   */
/* vector v and each context slot q (ctx id, or -1 = outside the stream):    */
/*   positive x = <u_ctx, v>:  loss softplus(-x), a = -sigmoid(-x)           */
/*   negative x = <u_n, v>  :  loss softplus(x),  a =  sigmoid(x)            */
/*   grad u (per occurrence) = a * v ;  grad v = sum over all pairs a * u    */
/* Occurrence order per centre: v, then per slot the context and its         */
/* negatives.  Absent slots get key -1 (no occurrence, no error).            */
/* ------------------------------------------------------------------------ */
static double dot_f(const float* a, const float* b, int32_t dim)
{
    double s = 0.0;
    for (int32_t c = 0; c < dim; ++c) s += (double)a[c] * (double)b[c];
    return s;
}

ORC_API double orc_grad_sgns(const float* W, int64_t num_keys, int32_t dim,
                             const int32_t* centre, const int32_t* ctx, const int32_t* neg,
                             int64_t B, int32_t window, int32_t n_neg, int64_t out_off,
                             int64_t* okeys, float* ograds, int64_t* bad)
{
    const int32_t slots = 2 * window;
    const int64_t per = 1 + (int64_t)slots * (1 + n_neg);
    double* gv = (double*)malloc(sizeof(double) * (size_t)dim);
    double loss = 0.0;
    *bad = 0;
    for (int64_t b = 0; b < B; ++b) {
        int64_t* kk = okeys + b * per;
        float* gg = ograds + b * per * dim;
        /* word2vec keeps two tables: centre words index the input vectors
         * [0, out_off), context and noise words the output vectors
         * [out_off, num_keys); a unit with an id outside its table is skipped */
        int64_t kc = centre[b];
        int ok = kc >= 0 && kc < out_off && key_ok(kc, num_keys);
        for (int32_t q = 0; q < slots; ++q) {
            int32_t cx = ctx[b * slots + q];
            if (cx == -1) continue;
            ok = ok && cx >= 0 && key_ok(out_off + cx, num_keys);
            for (int32_t k = 0; k < n_neg; ++k) {
                int32_t nx = neg[(b * slots + q) * n_neg + k];
                ok = ok && nx >= 0 && key_ok(out_off + nx, num_keys);
            }
        }
        for (int64_t q = 0; q < per; ++q) kk[q] = -1;
        memset(gg, 0, sizeof(float) * (size_t)(per * dim));
        if (!ok) {
            ++*bad;
            continue;
        }
        const float* v = W + kc * dim;
        for (int32_t c = 0; c < dim; ++c) gv[c] = 0.0;
        for (int32_t q = 0; q < slots; ++q) {
            int32_t cx = ctx[b * slots + q];
            if (cx == -1) continue;
            for (int32_t k = -1; k < n_neg; ++k) {
                int64_t key = out_off + (k < 0 ? cx : neg[(b * slots + q) * n_neg + k]);
                const float* u = W + key * dim;
                double x = dot_f(u, v, dim);
                double a;
                if (k < 0) {
                    a = -sigmoid(-x);
                    loss += softplus(-x);
                } else {
                    a = sigmoid(x);
                    loss += softplus(x);
                }
                int64_t occ = 1 + (int64_t)q * (1 + n_neg) + (k + 1);
                kk[occ] = key;
                float* go = gg + occ * dim;
                for (int32_t c = 0; c < dim; ++c) {
                    go[c] = (float)(a * (double)v[c]);
                    gv[c] += a * (double)u[c];
                }
            }
        }
        kk[0] = kc;
        round_row(gg, gv, dim);
    }
    free(gv);
    return loss;
}

/* ------------------------------------------------------------------------ */
/* CTR embeddings (Appendix C, "Click-through-rate prediction", embedding    */
/* part only): sample keys k_0..k_{F-1}, label y in {0,1}, e_f = W[k_f].     */
/*   S = sum_f e_f ,  z = sum_{f<g} <e_f, e_g>                               */
/*   loss = softplus(z) - y z ,  a = sigmoid(z) - y                          */
/*   grad e_f = a (S - e_f)   (one occurrence per field)                     */
/* ------------------------------------------------------------------------ */
ORC_API double orc_grad_ctr(const float* W, int64_t num_keys, int32_t dim,
                            const int64_t* keys, const float* label, int64_t B, int32_t F,
                            int64_t* okeys, float* ograds, int64_t* bad)
{
    double* S = (double*)malloc(sizeof(double) * (size_t)dim);
    double loss = 0.0;
    *bad = 0;
    for (int64_t b = 0; b < B; ++b) {
        const int64_t* kb = keys + b * F;
        int64_t* kk = okeys + b * F;
        float* gg = ograds + b * F * dim;
        int ok = 1;
        for (int32_t f = 0; f < F; ++f) ok = ok && key_ok(kb[f], num_keys);
        if (!ok) {
            for (int32_t f = 0; f < F; ++f) kk[f] = -1;
            memset(gg, 0, sizeof(float) * (size_t)(F * dim));
            ++*bad;
            continue;
        }
        for (int32_t c = 0; c < dim; ++c) S[c] = 0.0;
        for (int32_t f = 0; f < F; ++f)
            for (int32_t c = 0; c < dim; ++c) S[c] += (double)W[kb[f] * dim + c];
        double z = 0.0;
        for (int32_t f = 0; f < F; ++f)
            for (int32_t g = f + 1; g < F; ++g) z += dot_f(W + kb[f] * dim, W + kb[g] * dim, dim);
        double y = (double)label[b];
        loss += softplus(z) - y * z;
        double a = sigmoid(z) - y;
        for (int32_t f = 0; f < F; ++f) {
            const float* e = W + kb[f] * dim;
            for (int32_t c = 0; c < dim; ++c) gg[f * dim + c] = (float)(a * (S[c] - (double)e[c]));
            kk[f] = kb[f];
        }
    }
    free(S);
    return loss;
}

/* ------------------------------------------------------------------------ */
/* Full steps: gradients from the pre-step table, then the merging push.     */
/* Each returns the summed loss; *bad gets the number of skipped units.      */
/* ------------------------------------------------------------------------ */
static void* xmalloc(size_t bytes) { return malloc(bytes ? bytes : 1); }

ORC_API double orc_step_mf(float* W, float* G, int64_t num_keys, int32_t dim, float lr, float eps,
                           const int32_t* row, const int32_t* col, const float* val, int64_t B,
                           int64_t col_off, float lam, int64_t* bad)
{
    int64_t n = 2 * B;
    int64_t* k = (int64_t*)xmalloc(sizeof(int64_t) * (size_t)n);
    float* g = (float*)xmalloc(sizeof(float) * (size_t)(n * dim));
    double loss = orc_grad_mf(W, num_keys, dim, row, col, val, B, col_off, lam, k, g, bad);
    orc_push(W, G, num_keys, dim, lr, eps, k, n, g);
    free(g);
    free(k);
    return loss;
}

ORC_API double orc_step_kge(float* W, float* G, int64_t num_keys, int32_t dim, float lr, float eps,
                            const int32_t* head, const int32_t* rel, const int32_t* tail,
                            const int32_t* neg, int64_t B, int32_t n_neg, int32_t n_head_neg,
                            int64_t rel_off, int64_t* bad)
{
    int64_t n = B * (3 + (int64_t)n_neg);
    int64_t* k = (int64_t*)xmalloc(sizeof(int64_t) * (size_t)n);
    float* g = (float*)xmalloc(sizeof(float) * (size_t)(n * dim));
    double loss = orc_grad_kge(W, num_keys, dim, head, rel, tail, neg, B, n_neg, n_head_neg,
                               rel_off, k, g, bad);
    orc_push(W, G, num_keys, dim, lr, eps, k, n, g);
    free(g);
    free(k);
    return loss;
}

ORC_API double orc_step_sgns(float* W, float* G, int64_t num_keys, int32_t dim, float lr, float eps,
                             const int32_t* centre, const int32_t* ctx, const int32_t* neg,
                             int64_t B, int32_t window, int32_t n_neg, int64_t out_off, int64_t* bad)
{
    int64_t n = B * (1 + 2 * (int64_t)window * (1 + n_neg));
    int64_t* k = (int64_t*)xmalloc(sizeof(int64_t) * (size_t)n);
    float* g = (float*)xmalloc(sizeof(float) * (size_t)n * (size_t)dim);
    double loss = orc_grad_sgns(W, num_keys, dim, centre, ctx, neg, B, window, n_neg, out_off,
                                k, g, bad);
    /* absent slots carry key -1: drop them before the push */
    int64_t m = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (k[i] < 0) continue;
        if (m != i) {
            k[m] = k[i];
            memmove(g + m * dim, g + i * dim, sizeof(float) * (size_t)dim);
        }
        ++m;
    }
    orc_push(W, G, num_keys, dim, lr, eps, k, m, g);
    free(g);
    free(k);
    return loss;
}

ORC_API double orc_step_ctr(float* W, float* G, int64_t num_keys, int32_t dim, float lr, float eps,
                            const int64_t* keys, const float* label, int64_t B, int32_t F,
                            int64_t* bad)
{
    int64_t n = B * (int64_t)F;
    int64_t* k = (int64_t*)xmalloc(sizeof(int64_t) * (size_t)n);
    float* g = (float*)xmalloc(sizeof(float) * (size_t)(n * dim));
    double loss = orc_grad_ctr(W, num_keys, dim, keys, label, B, F, k, g, bad);
    orc_push(W, G, num_keys, dim, lr, eps, k, n, g);
    free(g);
    free(k);
    return loss;
}
