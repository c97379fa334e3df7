/* Drives every entry point of the CPU oracle (oracle/oracle.c, compiled into
 * this program) on small random inputs with the edge cases the tests use:
 * invalid keys, empty calls, absent skip-gram slots, units skipped for an
 * out-of-range id.  Built with address and undefined-behaviour sanitizers,
 * it exits non-zero on the first report.  Prints a checksum of the results. */
#include "../oracle/oracle.c"

#include <stdio.h>

static uint64_t rng = 88172645463325252ull;
static uint64_t next_u64(void) {
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return rng;
}
static int64_t rnd(int64_t n) { return (int64_t)(next_u64() % (uint64_t)n); }
static float rndf(void) { return (float)((double)(next_u64() >> 11) * 0x1p-53 - 0.5); }

static float* table(int64_t rows, int32_t dim) {
    float* t = (float*)malloc(sizeof(float) * (size_t)(rows * dim));
    for (int64_t i = 0; i < rows * dim; ++i) t[i] = rndf() * 0.2f;
    return t;
}

static double sum(const float* x, int64_t n) {
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) s += x[i];
    return s;
}

int main(void) {
    double check = 0.0;
    for (int round = 0; round < 40; ++round) {
        const int64_t K = 1 + rnd(300);
        const int32_t d = 1 + (int32_t)rnd(24);
        const int64_t n = rnd(500);
        float* W = table(K, d);
        float* G = table(K, d);
        for (int64_t i = 0; i < K * d; ++i) G[i] = G[i] * G[i];
        int64_t* keys = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n + 1));
        for (int64_t i = 0; i < n; ++i) keys[i] = rnd(K + 4) - 2;       /* some out of range */
        float* grads = table(n + 1, d);
        float* out = (float*)malloc(sizeof(float) * (size_t)((n + 1) * d));
        check += (double)orc_pull(W, K, d, keys, n, out) + sum(out, n * d);
        int64_t* uniq = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n + 1));
        int32_t* perm = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n + 1));
        int32_t* offs = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n + 2));
        int32_t nu = 0;
        check += (double)orc_dedup(K, keys, n, uniq, perm, offs, &nu) + nu;
        check += (double)orc_push(W, G, K, d, 0.1f, 1e-10f, keys, n, grads);
        float* Gr = table(K, 1);
        for (int64_t i = 0; i < K; ++i) Gr[i] = Gr[i] * Gr[i];
        check += (double)orc_push_rowwise(W, Gr, K, d, 0.1f, 1e-10f, keys, n, grads);
        int64_t* order = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n + 1));
        for (int64_t i = 0; i < n; ++i) order[i] = n - 1 - i;
        check += (double)orc_push_sequential(W, G, K, d, 0.1f, 1e-10f, keys, n, grads, order);
        check += (double)orc_push_sequential(W, G, K, d, 0.1f, 1e-10f, keys, n, grads, NULL);
        check += (double)orc_push_sequential_rowwise(W, Gr, K, d, 0.1f, 1e-10f, keys, n, grads, order);
        uint16_t* Wb = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)(K * d));
        orc_f32_to_bf16_array(W, Wb, K * d);
        check += (double)orc_push_bf16(Wb, G, K, d, 0.1f, 1e-10f, keys, n, grads) + orc_bf16_to_f32(Wb[0]);
        check += sum(W, K * d) + sum(G, K * d) + sum(Gr, K);

        /* MF: rows [0, R), columns [R, K) */
        const int64_t B = rnd(200), R = K / 2 + 1 > K ? K : K / 2 + 1;
        int32_t* row = (int32_t*)malloc(sizeof(int32_t) * (size_t)(B + 1));
        int32_t* col = (int32_t*)malloc(sizeof(int32_t) * (size_t)(B + 1));
        float* val = table(B + 1, 1);
        for (int64_t b = 0; b < B; ++b) {
            row[b] = (int32_t)(rnd(R + 2) - 1);
            col[b] = (int32_t)(rnd(K - R + 2) - 1);
        }
        int64_t* okeys = (int64_t*)malloc(sizeof(int64_t) * (size_t)(2 * B + 1));
        float* og = (float*)malloc(sizeof(float) * (size_t)((2 * B + 1) * d));
        int64_t bad = 0;
        check += orc_grad_mf(W, K, d, row, col, val, B, R, 1e-2f, okeys, og, &bad) + (double)bad;
        check += orc_step_mf(W, G, K, d, 0.1f, 1e-10f, row, col, val, B, R, 1e-2f, &bad) + (double)bad;

        /* ComplEx: even rows, relations after the entities */
        const int32_t dk = 2 * (1 + (int32_t)rnd(8));
        const int64_t E = 2 + rnd(100), Rn = 1 + rnd(5), Bk = rnd(30);
        const int32_t nneg = (int32_t)rnd(7), nhead = nneg ? (int32_t)rnd(nneg + 1) : 0;
        float* Wk = table(E + Rn, dk);
        float* Gk = table(E + Rn, dk);
        for (int64_t i = 0; i < (E + Rn) * dk; ++i) Gk[i] = Gk[i] * Gk[i];
        int32_t* h = (int32_t*)malloc(sizeof(int32_t) * (size_t)(Bk + 1));
        int32_t* r = (int32_t*)malloc(sizeof(int32_t) * (size_t)(Bk + 1));
        int32_t* t = (int32_t*)malloc(sizeof(int32_t) * (size_t)(Bk + 1));
        int32_t* ng = (int32_t*)malloc(sizeof(int32_t) * (size_t)(Bk * nneg + 1));
        for (int64_t b = 0; b < Bk; ++b) {
            h[b] = (int32_t)rnd(E);
            r[b] = (int32_t)(rnd(Rn + 1) - (b == 3 ? 1 : 0));
            t[b] = (int32_t)rnd(E + 1);
        }
        for (int64_t i = 0; i < Bk * nneg; ++i) ng[i] = (int32_t)rnd(E);
        const int64_t perk = 3 + nneg;
        int64_t* kk = (int64_t*)malloc(sizeof(int64_t) * (size_t)(Bk * perk + 1));
        float* kg = (float*)malloc(sizeof(float) * (size_t)((Bk * perk + 1) * dk));
        check += orc_grad_kge(Wk, E + Rn, dk, h, r, t, ng, Bk, nneg, nhead, E, kk, kg, &bad) + (double)bad;
        check += orc_step_kge(Wk, Gk, E + Rn, dk, 0.1f, 1e-10f, h, r, t, ng, Bk, nneg, nhead, E, &bad);
        if (Bk > 0) check += orc_complex_score(Wk, Wk + dk, Wk + 2 * (E > 2 ? dk : 0), dk / 2);

        /* skip-gram: input rows [0, V), output rows [V, 2V) */
        const int64_t V = 2 + rnd(60), Bs = rnd(20);
        const int32_t win = (int32_t)rnd(4), kneg = (int32_t)rnd(5);
        const int32_t slots = 2 * win;
        float* Ws = table(2 * V, d);
        float* Gs = table(2 * V, d);
        for (int64_t i = 0; i < 2 * V * d; ++i) Gs[i] = Gs[i] * Gs[i];
        int32_t* cen = (int32_t*)malloc(sizeof(int32_t) * (size_t)(Bs + 1));
        int32_t* ctx = (int32_t*)malloc(sizeof(int32_t) * (size_t)(Bs * slots + 1));
        int32_t* sn = (int32_t*)malloc(sizeof(int32_t) * (size_t)(Bs * slots * kneg + 1));
        for (int64_t b = 0; b < Bs; ++b) cen[b] = (int32_t)rnd(V + (b == 2 ? V : 0));
        for (int64_t i = 0; i < Bs * slots; ++i) ctx[i] = (int32_t)(rnd(V + 1) - 1);   /* -1: absent */
        for (int64_t i = 0; i < Bs * slots * kneg; ++i) sn[i] = (int32_t)rnd(V);
        const int64_t pers = 1 + (int64_t)slots * (1 + kneg);
        int64_t* sk = (int64_t*)malloc(sizeof(int64_t) * (size_t)(Bs * pers + 1));
        float* sg = (float*)malloc(sizeof(float) * (size_t)((Bs * pers + 1) * d));
        check += orc_grad_sgns(Ws, 2 * V, d, cen, ctx, sn, Bs, win, kneg, V, sk, sg, &bad) + (double)bad;
        check += orc_step_sgns(Ws, Gs, 2 * V, d, 0.1f, 1e-10f, cen, ctx, sn, Bs, win, kneg, V, &bad);

        /* CTR: F fields per sample */
        const int64_t Bc = rnd(40);
        const int32_t F = 1 + (int32_t)rnd(27);
        int64_t* ck = (int64_t*)malloc(sizeof(int64_t) * (size_t)(Bc * F + 1));
        float* lab = (float*)malloc(sizeof(float) * (size_t)(Bc + 1));
        for (int64_t i = 0; i < Bc * F; ++i) ck[i] = rnd(K + 1) - (i == 5 ? 3 : 0);
        for (int64_t b = 0; b < Bc; ++b) lab[b] = (float)rnd(2);
        int64_t* cko = (int64_t*)malloc(sizeof(int64_t) * (size_t)(Bc * F + 1));
        float* cg = (float*)malloc(sizeof(float) * (size_t)((Bc * F + 1) * d));
        check += orc_grad_ctr(W, K, d, ck, lab, Bc, F, cko, cg, &bad) + (double)bad;
        check += orc_step_ctr(W, G, K, d, 0.1f, 1e-10f, ck, lab, Bc, F, &bad);

        free(W); free(G); free(keys); free(grads); free(out); free(uniq); free(perm); free(offs); free(Gr);
        free(order); free(Wb); free(row); free(col); free(val); free(okeys); free(og); free(Wk); free(Gk);
        free(h); free(r); free(t); free(ng); free(kk); free(kg); free(Ws); free(Gs); free(cen); free(ctx);
        free(sn); free(sk); free(sg); free(ck); free(lab); free(cko); free(cg);
    }
    printf("checksum %.6e\n", check);
    return 0;
}
