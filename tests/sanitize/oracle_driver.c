/* Host driver for a sanitizer build (AddressSanitizer + UndefinedBehaviorSanitizer)
 * of the CPU oracle, which it includes as one translation unit. Test
 * infrastructure only.
 *
 * usage: oracle_driver <graphs file> <seed>
 * For each of the five models, random small parameter arrays of exactly the
 * shapes the model reads (so that any read past them is caught) and random
 * batches: every built-in structure with valid and out-of-range ids, every
 * graph of the file (one line per graph: node count, then 6 ints per node,
 * malformed graphs included), top-k with valid and invalid k, and filtered
 * ranks with random answer lists (out-of-range ids included). */
#include <stdio.h>
#include <stdlib.h>

#include "../../oracle/kgq_oracle.c"

static unsigned long long g_state;
static unsigned rnd(void)
{
    g_state = g_state * 6364136223846793005ULL + 1442695040888963407ULL;
    return (unsigned)(g_state >> 33);
}
static double unif(double lo, double hi) { return lo + (hi - lo) * (rnd() / 2147483648.0); }

static float* arr(size_t n, double lo, double hi)
{
    float* p = (float*)malloc(sizeof(float) * (n ? n : 1));
    for (size_t i = 0; i < n; ++i) p[i] = (float)unif(lo, hi);
    return p;
}

typedef struct {
    int n;
    int32_t* g;
} graph_t;

int main(int argc, char** argv)
{
    if (argc < 3) {
        fprintf(stderr, "usage: %s <graphs> <seed>\n", argv[0]);
        return 2;
    }
    g_state = strtoull(argv[2], NULL, 10) * 2654435761ULL + 1;
    FILE* f = fopen(argv[1], "r");
    if (!f) return 2;
    graph_t graphs[512];
    int ng = 0, n;
    while (ng < 512 && fscanf(f, "%d", &n) == 1) {
        if (n < 0 || n > 300) break;
        graphs[ng].n = n;
        graphs[ng].g = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1) * KGO_NODE_WORDS);
        for (int i = 0; i < n * KGO_NODE_WORDS; ++i)
            if (fscanf(f, "%d", &graphs[ng].g[i]) != 1) return 2;
        ++ng;
    }
    fclose(f);
    long ok = 0, refused = 0;
    for (int trial = 0; trial < 10; ++trial) {
        for (int model = 0; model < 5; ++model) {
            kgo_model m;
            memset(&m, 0, sizeof(m));
            const int d = 4 + 4 * (int)(rnd() % 3);
            const int N = 5 + (int)(rnd() % 36), R = 2 + (int)(rnd() % 6);
            m.model = model;
            m.dim = d;
            m.n_entities = N;
            m.n_relations = R;
            m.gamma = 12.0;
            m.center_reg = 0.02;
            m.modulus = 0.1;
            m.tnorm = (int)(rnd() % 3);
            const int w = model == KGO_GQE ? d : 2 * d;
            if (model == KGO_BETAE) m.entity = arr((size_t)N * 2 * d, 0.05, 3.0);
            else if (model == KGO_LOGICE) m.entity = arr((size_t)N * 2 * d, 0.0, 1.0);
            else if (model == KGO_CONE) m.entity = arr((size_t)N * d, -3.14, 3.14);
            else m.entity = arr((size_t)N * d, -0.5, 0.5);
            m.relation = arr((size_t)R * (model == KGO_BETAE || model == KGO_CONE ? 2 * d : d), -0.5, 0.5);
            if (model == KGO_Q2B) m.offset_raw = arr((size_t)R * d, -2.0, 0.0);
            if (model == KGO_GQE || model == KGO_Q2B) {
                m.att_w1 = arr((size_t)d * d, -0.3, 0.3); m.att_b1 = arr(d, -0.1, 0.1);
                m.att_w2 = arr((size_t)d * d, -0.3, 0.3); m.att_b2 = arr(d, -0.1, 0.1);
            }
            if (model == KGO_Q2B) {
                m.off_w1 = arr((size_t)d * d, -0.3, 0.3); m.off_b1 = arr(d, -0.1, 0.1);
                m.off_w2 = arr((size_t)d * d, -0.3, 0.3); m.off_b2 = arr(d, -0.1, 0.1);
            }
            if (model == KGO_BETAE) {
                m.att_w1 = arr((size_t)2 * d * 2 * d, -0.3, 0.3); m.att_b1 = arr(2 * d, -0.1, 0.1);
                m.att_w2 = arr((size_t)d * 2 * d, -0.3, 0.3); m.att_b2 = arr(d, -0.1, 0.1);
            }
            if (model == KGO_CONE) {
                m.att_w1 = arr((size_t)d * 2 * d, -0.3, 0.3); m.att_b1 = arr(d, -0.1, 0.1);
                m.att_w2 = arr((size_t)d * d, -0.3, 0.3); m.att_b2 = arr(d, -0.1, 0.1);
                m.off_w1 = arr((size_t)d * 2 * d, -0.3, 0.3); m.off_b1 = arr(d, -0.1, 0.1);
                m.off_w2 = arr((size_t)d * d, -0.3, 0.3); m.off_b2 = arr(d, -0.1, 0.1);
            }
            if (model >= KGO_BETAE) {
                const int in_w = model == KGO_LOGICE ? 3 * d : 2 * d, h = 4 * d;
                m.proj_w1 = arr((size_t)h * in_w, -0.2, 0.2); m.proj_b1 = arr(h, -0.1, 0.1);
                m.proj_w2 = arr((size_t)h * h, -0.2, 0.2); m.proj_b2 = arr(h, -0.1, 0.1);
                m.proj_w3 = arr((size_t)2 * d * h, -0.2, 0.2); m.proj_b3 = arr(2 * d, -0.1, 0.1);
            }
            (void)w;
            /* built-in structures, valid ids and some out of range */
            const int B = 1 + (int)(rnd() % 9);
            int32_t sid[16], an[16 * 3], rl[16 * 3];
            for (int q = 0; q < B; ++q) {
                sid[q] = (int32_t)(rnd() % 15) - (rnd() % 8 == 0 ? 1 : 0);
                for (int k = 0; k < 3; ++k) {
                    an[q * 3 + k] = (int32_t)(rnd() % (N + (trial == 0 ? 2 : 0)));
                    rl[q * 3 + k] = (int32_t)(rnd() % (R + (trial == 1 ? 2 : 0)));
                }
            }
            double* sc = (double*)malloc(sizeof(double) * (size_t)B * N);
            double* mg = (double*)malloc(sizeof(double) * (size_t)B);
            if (kgo_scores(&m, B, sid, an, 3, rl, 3, sc, mg, 2) == 0) {
                ++ok;
                const int k = 1 + (int)(rnd() % (N + 1));
                int32_t* idx = (int32_t*)malloc(sizeof(int32_t) * (size_t)B * (k > N ? 1 : k));
                double* val = (double*)malloc(sizeof(double) * (size_t)B * (k > N ? 1 : k));
                if (kgo_topk(sc, B, N, k, idx, val, 2) == 0) ++ok; else ++refused;
                free(idx);
                free(val);
                /* ranks: random CSR lists, some ids out of range */
                int32_t off[17], ids[16 * 8], hard[16 * 8], rk[16 * 8];
                float* scf = (float*)malloc(sizeof(float) * (size_t)B * N);
                for (int i = 0; i < B * N; ++i) scf[i] = (float)sc[i];
                off[0] = 0;
                for (int q = 0; q < B; ++q) {
                    const int len = (int)(rnd() % 8);
                    for (int i = 0; i < len; ++i) {
                        ids[off[q] + i] = (int32_t)(rnd() % (N + 1));
                        hard[off[q] + i] = (int32_t)(rnd() % 2);
                    }
                    off[q + 1] = off[q] + len;
                }
                double met[16 * 4];
                if (kgo_rank_answers(scf, B, N, off, ids, hard, rk, met, 2) == 0) ++ok; else ++refused;
                free(scf);
            } else {
                ++refused;
            }
            free(sc);
            free(mg);
            /* graphs of the file */
            for (int gi = 0; gi < ng; ++gi) {
                int na, nr, nt;
                if (kgo_graph_check(&m, graphs[gi].g, graphs[gi].n, &na, &nr, &nt) != 0) {
                    ++refused;
                    continue;
                }
                const int Bg = 2;
                int32_t ga[2 * 8], gr[2 * 8];
                for (int i = 0; i < 2 * 8; ++i) {
                    ga[i] = (int32_t)(rnd() % N);
                    gr[i] = (int32_t)(rnd() % R);
                }
                double* gs = (double*)malloc(sizeof(double) * (size_t)Bg * N);
                double* gm = (double*)malloc(sizeof(double) * Bg);
                if (na <= 8 && nr <= 8 && kgo_graph_scores(&m, graphs[gi].g, graphs[gi].n, Bg, ga, 8, gr, 8, gs, gm, 2) == 0)
                    ++ok;
                else
                    ++refused;
                free(gs);
                free(gm);
            }
            free((void*)m.entity); free((void*)m.relation); free((void*)m.offset_raw);
            free((void*)m.att_w1); free((void*)m.att_b1); free((void*)m.att_w2); free((void*)m.att_b2);
            free((void*)m.off_w1); free((void*)m.off_b1); free((void*)m.off_w2); free((void*)m.off_b2);
            free((void*)m.proj_w1); free((void*)m.proj_b1); free((void*)m.proj_w2); free((void*)m.proj_b2);
            free((void*)m.proj_w3); free((void*)m.proj_b3);
        }
    }
    for (int gi = 0; gi < ng; ++gi) free(graphs[gi].g);
    printf("ok %ld refused %ld graphs %d\n", ok, refused, ng);
    return 0;
}
