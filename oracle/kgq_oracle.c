/*
 * kgq_oracle.c -- CPU oracle for batched complex-logical-query answering.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the slow, plain reference against
 * which the GPU library is checked. It is called from the test suite, from
 * the smoke check and from the benchmark's CPU-baseline leg, never from the
 * product path. It shares no code, header, table or constant with the GPU
 * library.
 *
 * Arithmetic: every operator is evaluated one node at a time in double
 * precision from the float32 (or bfloat16-decoded) inputs, with no fusion
 * and no algebraic regrouping. The paper's operator fusion is stated to
 * leave the output unchanged (Methodology, Operator Fuser), so the fused GPU
 * result must equal this node-by-node evaluation.
 *
 * What the paper fixes and what it leaves open:
 *  - Query computation graph and its mapping from a first-order query
 *    (Preliminaries, Query Computation Graph; Methodology, Graph Capturer,
 *    Eq. 2): entities become value nodes, each relation becomes a projection
 *    operator node, and conjunction / disjunction / negation become
 *    intersection / union / negation functions.
 *  - Disjunctive normal form (Preliminaries, Eq. 1): a union is evaluated as
 *    separate conjunctive branches whose entity scores are combined by max.
 *  - Beta embeddings (Methodology, Pattern Recognizer, Eq. 3) and the BetaE
 *    projection as three matmul+bias layers with ReLU between them (Eq. 4).
 *    Eq. 4 prints a softmax as the last operator; here the last operator is
 *    the regulariser clamp(y + 1, 0.05, 1e9), because a softmax would force
 *    the shape parameters of each query to sum to one.
 *  - Reasoning time is operator execution plus the entity-similarity query,
 *    i.e. scoring every entity (Experiments, Metrics).
 *  - GQE and Query2Box are named (Related Work; Experiments, Baselines) but
 *    their operators are not written out in the paper. The forms used here:
 *      GQE:   anchor q = E[a]; projection q + Rel[r]; intersection by
 *             attention over branches; score gamma - ||q - e||_1.
 *      Q2B:   anchor box (E[a], 0); projection (c + C[r], o + softplus(O[r]));
 *             intersection: attention over centers, offset
 *             min_j(o_j) * sigmoid(W4 mean_j ReLU(W3 o_j + b3) + b4);
 *             score gamma - (dist_out + center_reg * dist_in).
 *      BetaE: negation (alpha, beta) -> (1/alpha, 1/beta), no clamp after;
 *             intersection: attention over branches on [alpha; beta];
 *             score gamma - sum_i KL(Beta(entity_i) || Beta(query_i)).
 *      ConE and LogicE are named as well (Related Work; Experiments,
 *      Baselines; Table 1) without their operators; the forms used here are
 *      those of the two models' own papers, read as follows.
 *      ConE:  a query is a product of d two-dimensional sector cones, axis
 *             theta in [-pi, pi) and half-aperture psi in [0, pi] per
 *             dimension (state [theta; psi]); an entity is a cone of
 *             aperture 0 (its axis). Projection: x = [theta + theta_r;
 *             psi + psi_r] -> three dense layers (ReLU between) -> theta =
 *             pi tanh(y_theta), psi = (pi / 2)(tanh(2 y_psi) + 1).
 *             Intersection: u_j = [theta_j - psi_j; theta_j + psi_j];
 *             attention logits from an MLP on u_j (2d -> d -> d), softmax
 *             across branches per dimension, axis = the angle of the
 *             weighted mean of the unit vectors (cos theta_j, sin theta_j);
 *             half-aperture = min_j psi_j times a sigmoid gate computed from
 *             the mean over branches of ReLU(W3 u_j + b3). Negation: the
 *             complementary cone, axis moved by pi (theta - pi if theta >= 0,
 *             else theta + pi), half-aperture pi - psi. Score: gamma -
 *             modulus (sum_i d_out + center_reg sum_i d_in), with
 *             t = theta_e - theta, d_in = min(|sin(t/2)|, |sin(psi/2)|) and
 *             d_out = 0 inside the sector (|sin(t/2)| < |sin(psi/2)|), else
 *             the smaller of |sin((t + psi)/2)| and |sin((t - psi)/2)|.
 *      LogicE: a query is a vector of truth-value bounds [l; u] in [0, 1]^2d
 *             with l <= u; an entity is such a vector too. Projection:
 *             x = [l; u; Rel[r]] (concatenation, width 3d) -> three dense
 *             layers -> l = sigmoid(y_l), u = l + sigmoid(y_u)(1 - l).
 *             Intersection: a t-norm applied coordinate-wise to the lower
 *             bounds and to the upper bounds of the branches, folded from the
 *             first branch on (product a*b, minimum, or Lukasiewicz
 *             max(0, a + b - 1)). Negation: [l; u] -> [1 - u; 1 - l].
 *             Score: gamma - ||e - q||_1 / (2d) over the 2d bounds.
 *  - The 14 query shapes are named in the paper (Introduction; Experiments,
 *    Datasets & Tasks) but drawn only in a figure that is not available;
 *    the shapes below are the standard ones of the BetaE benchmark that the
 *    paper adopts. pin negates the one-hop branch, pni the two-hop branch.
 *
 * Parity pins: every function below is checked in the CPU test suite against
 * closed forms, identities, worked examples, special cases that reduce to a
 * library routine, or brute force (see the tests named test_oracle_*).
 */

#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define KGO_GQE 0
#define KGO_Q2B 1
#define KGO_BETAE 2
#define KGO_CONE 3
#define KGO_LOGICE 4

#define KGO_TNORM_PRODUCT 0
#define KGO_TNORM_MIN 1
#define KGO_TNORM_LUKASIEWICZ 2

#define KGO_PI 3.14159265358979323846

typedef struct {
    int32_t model;
    int32_t dim;
    int64_t n_entities;
    int32_t n_relations;
    int32_t pad_;
    double gamma;
    double center_reg;
    const float* entity;     /* GQE/Q2B [N x d]; BetaE [N x 2d], alpha then beta;
                                ConE [N x d] axes; LogicE [N x 2d], l then u */
    const float* relation;   /* GQE [R x d]; Q2B centers [R x d]; BetaE, ConE [R x 2d];
                                LogicE [R x d] */
    const float* offset_raw; /* Q2B [R x d], offsets before softplus */
    const float* att_w1;     /* intersection attention layer 1 [h x in] */
    const float* att_b1;
    const float* att_w2;     /* intersection attention layer 2 [d x h] */
    const float* att_b2;
    const float* off_w1;     /* Q2B offset set-function layers [d x d];
                                ConE aperture set function [d x 2d], [d x d] */
    const float* off_b1;
    const float* off_w2;
    const float* off_b2;
    const float* proj_w1;    /* projection MLP [4d x in], [4d x 4d], [2d x 4d]; in = 2d (BetaE,
                                ConE) or 3d (LogicE) */
    const float* proj_b1;
    const float* proj_w2;
    const float* proj_b2;
    const float* proj_w3;
    const float* proj_b3;
    int32_t tnorm;           /* LogicE intersection t-norm (KGO_TNORM_*) */
    int32_t pad2_;
    double modulus;          /* ConE distance scale */
} kgo_model;

/* Models with a negation operator (the paper: GQE and Query2Box run only
 * the 9 structures without one; Experiments, Baselines). */
static int has_negation(const kgo_model* m)
{
    return m->model == KGO_BETAE || m->model == KGO_CONE || m->model == KGO_LOGICE;
}

/* Closest approach, in the query being evaluated, to a point where ConE's
 * operators are discontinuous: a negated axis at 0 (the complement moves it
 * by -pi or +pi by its sign) and an intersection axis on the branch cut of
 * the angle (weighted mean vector on the negative x axis). There a float32
 * evaluation can land on the other side, with a different but equally
 * correct result. Reset per query; +inf when no such operator runs. */
static __thread double g_margin;

static void note_margin(double v)
{
    if (v < g_margin) g_margin = v;
}

/* A query state: GQE uses x[0..d); Q2B holds center x[0..d) and offset
 * x[d..2d); BetaE holds alpha x[0..d) and beta x[d..2d). */
#define KGO_MAX_DIM 4096

/* ------------------------------------------------------------------ */
/* Special functions                                                   */
/* ------------------------------------------------------------------ */

/* Digamma psi(x) for x > 0: raise the argument with psi(x) = psi(x+1) - 1/x
 * until it is at least 10, then apply the asymptotic expansion
 * psi(x) ~ ln x - 1/(2x) - sum_n B_2n / (2n x^(2n)) through B_12
 * (Abramowitz & Stegun 6.3.18). The first omitted term is below 1e-16 at
 * x >= 10. */
double kgo_digamma(double x)
{
    double acc = 0.0;
    while (x < 10.0) {
        acc -= 1.0 / x;
        x += 1.0;
    }
    double r = 1.0 / x;
    double r2 = r * r;
    /* B2 = 1/6, B4 = -1/30, B6 = 1/42, B8 = -1/30, B10 = 5/66, B12 = -691/2730 */
    double series = r2 * (1.0 / 12.0
                  - r2 * (1.0 / 120.0
                  - r2 * (1.0 / 252.0
                  - r2 * (1.0 / 240.0
                  - r2 * (1.0 / 132.0
                  - r2 * (691.0 / 32760.0))))));
    return acc + log(x) - 0.5 * r - series;
}

double kgo_lgamma(double x)
{
    int sign;
    return lgamma_r(x, &sign);
}

/* ln B(a, b) with B the Beta function of Eq. 3. */
double kgo_lnbeta(double a, double b)
{
    return kgo_lgamma(a) + kgo_lgamma(b) - kgo_lgamma(a + b);
}

/* KL( Beta(a1, b1) || Beta(a2, b2) ) for the densities of Eq. 3. */
double kgo_kl_beta(double a1, double b1, double a2, double b2)
{
    return kgo_lnbeta(a2, b2) - kgo_lnbeta(a1, b1)
         + (a1 - a2) * kgo_digamma(a1)
         + (b1 - b2) * kgo_digamma(b1)
         + (a2 - a1 + b2 - b1) * kgo_digamma(a1 + b1);
}

double kgo_softplus(double x)
{
    return (x > 0.0 ? x : 0.0) + log1p(exp(-fabs(x)));
}

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/* y = W x + b for W stored [out x in] row-major (one dense layer of Eq. 4). */
static void dense(const float* W, const float* b, int out, int in, const double* x, double* y)
{
    for (int i = 0; i < out; ++i) {
        double s = (double)b[i];
        const float* w = W + (size_t)i * in;
        for (int j = 0; j < in; ++j) s += (double)w[j] * x[j];
        y[i] = s;
    }
}

static void relu_inplace(double* x, int n)
{
    for (int i = 0; i < n; ++i) if (x[i] < 0.0) x[i] = 0.0;
}

/* ------------------------------------------------------------------ */
/* Operators                                                           */
/* ------------------------------------------------------------------ */

int kgo_state_width(const kgo_model* m)
{
    return m->model == KGO_GQE ? m->dim : 2 * m->dim;
}

static double sigmoid_d(double x) { return 1.0 / (1.0 + exp(-x)); }

/* The three t-norms of LogicE's intersection, as binary operations. */
static double tnorm2(int kind, double a, double b)
{
    if (kind == KGO_TNORM_MIN) return a < b ? a : b;
    if (kind == KGO_TNORM_LUKASIEWICZ) {
        double v = a + b - 1.0;
        return v > 0.0 ? v : 0.0;
    }
    return a * b;
}

/* Anchor entity -> value node (Eq. 2, first rule). */
void kgo_anchor(const kgo_model* m, int64_t e, double* st)
{
    int d = m->dim;
    if (m->model == KGO_GQE) {
        for (int i = 0; i < d; ++i) st[i] = m->entity[(size_t)e * d + i];
    } else if (m->model == KGO_Q2B || m->model == KGO_CONE) {
        /* Q2B: a point is a box of zero offset; ConE: a cone of zero aperture */
        for (int i = 0; i < d; ++i) { st[i] = m->entity[(size_t)e * d + i]; st[d + i] = 0.0; }
    } else {
        for (int i = 0; i < 2 * d; ++i) st[i] = m->entity[(size_t)e * 2 * d + i];
    }
}

/* Relation projection (Eq. 2, relation rule; BetaE: Eq. 4). in and out may alias. */
void kgo_project(const kgo_model* m, const double* in, int32_t r, double* out)
{
    int d = m->dim;
    if (m->model == KGO_GQE) {
        for (int i = 0; i < d; ++i) out[i] = in[i] + (double)m->relation[(size_t)r * d + i];
        return;
    }
    if (m->model == KGO_Q2B) {
        for (int i = 0; i < d; ++i) {
            out[i] = in[i] + (double)m->relation[(size_t)r * d + i];
            out[d + i] = in[d + i] + kgo_softplus((double)m->offset_raw[(size_t)r * d + i]);
        }
        return;
    }
    /* BetaE, ConE: x = state + Rel[r] (width 2d); LogicE: x = [state; Rel[r]]
     * (width 3d). Three dense layers with ReLU between, then the model's
     * output map. */
    int w = 2 * d, h = 4 * d;
    int in_w = m->model == KGO_LOGICE ? 3 * d : w;
    double* x = (double*)malloc(sizeof(double) * (size_t)(in_w + h + h + w));
    double* h1 = x + in_w;
    double* h2 = h1 + h;
    double* y = h2 + h;
    if (m->model == KGO_LOGICE) {
        for (int i = 0; i < w; ++i) x[i] = in[i];
        for (int i = 0; i < d; ++i) x[w + i] = (double)m->relation[(size_t)r * d + i];
    } else {
        for (int i = 0; i < w; ++i) x[i] = in[i] + (double)m->relation[(size_t)r * w + i];
    }
    dense(m->proj_w1, m->proj_b1, h, in_w, x, h1);
    relu_inplace(h1, h);
    dense(m->proj_w2, m->proj_b2, h, h, h1, h2);
    relu_inplace(h2, h);
    dense(m->proj_w3, m->proj_b3, w, h, h2, y);
    if (m->model == KGO_BETAE) {
        for (int i = 0; i < w; ++i) {
            double v = y[i] + 1.0;
            if (v < 0.05) v = 0.05;
            if (v > 1e9) v = 1e9;
            out[i] = v;
        }
    } else if (m->model == KGO_CONE) {
        for (int i = 0; i < d; ++i) {
            out[i] = KGO_PI * tanh(y[i]);
            out[d + i] = 0.5 * KGO_PI * (tanh(2.0 * y[d + i]) + 1.0);
        }
    } else {
        for (int i = 0; i < d; ++i) {
            double l = sigmoid_d(y[i]);
            out[i] = l;
            out[d + i] = l + sigmoid_d(y[d + i]) * (1.0 - l);
        }
    }
    free(x);
}

/* Negation (f_not of Eq. 2), for the models that have one. BetaE: the
 * reciprocal of both shape parameters. ConE: the complementary cone. LogicE:
 * the complement of the truth bounds. in and out may alias. */
void kgo_negate(const kgo_model* m, const double* in, double* out)
{
    int d = m->dim, w = 2 * d;
    if (m->model == KGO_CONE) {
        for (int i = 0; i < d; ++i) {
            double t = in[i];
            note_margin(fabs(t));
            out[i] = t >= 0.0 ? t - KGO_PI : t + KGO_PI;
            out[d + i] = KGO_PI - in[d + i];
        }
        return;
    }
    if (m->model == KGO_LOGICE) {
        for (int i = 0; i < d; ++i) {
            double l = in[i], u = in[d + i];
            out[i] = 1.0 - u;
            out[d + i] = 1.0 - l;
        }
        return;
    }
    for (int i = 0; i < w; ++i) out[i] = 1.0 / in[i];
}

/* ConE intersection: semantic average of the axes, gated minimum of the
 * half-apertures. */
static void cone_intersect(const kgo_model* m, int n, const double* const* br, double* out)
{
    int d = m->dim, w = 2 * d;
    double* u = (double*)malloc(sizeof(double) * (size_t)w);
    double* hid = (double*)malloc(sizeof(double) * (size_t)d);
    double* logits = (double*)malloc(sizeof(double) * (size_t)n * d);
    double* mean = (double*)calloc((size_t)d, sizeof(double));
    double* g = (double*)malloc(sizeof(double) * (size_t)d);
    double* wts = (double*)malloc(sizeof(double) * (size_t)n);
    for (int j = 0; j < n; ++j) {
        for (int i = 0; i < d; ++i) {
            u[i] = br[j][i] - br[j][d + i];
            u[d + i] = br[j][i] + br[j][d + i];
        }
        dense(m->att_w1, m->att_b1, d, w, u, hid);
        relu_inplace(hid, d);
        dense(m->att_w2, m->att_b2, d, d, hid, logits + (size_t)j * d);
        dense(m->off_w1, m->off_b1, d, w, u, hid);
        relu_inplace(hid, d);
        for (int i = 0; i < d; ++i) mean[i] += hid[i];
    }
    for (int i = 0; i < d; ++i) mean[i] /= (double)n;
    dense(m->off_w2, m->off_b2, d, d, mean, g);
    for (int i = 0; i < d; ++i) {
        double mx = logits[i];
        for (int j = 1; j < n; ++j) if (logits[(size_t)j * d + i] > mx) mx = logits[(size_t)j * d + i];
        double z = 0.0;
        for (int j = 0; j < n; ++j) { wts[j] = exp(logits[(size_t)j * d + i] - mx); z += wts[j]; }
        double cx = 0.0, sy = 0.0, mn = br[0][d + i];
        for (int j = 0; j < n; ++j) {
            double wj = wts[j] / z;
            cx += wj * cos(br[j][i]);
            sy += wj * sin(br[j][i]);
            if (br[j][d + i] < mn) mn = br[j][d + i];
        }
        if (cx < 0.0) note_margin(fabs(sy));
        out[i] = atan2(sy, cx);
        out[d + i] = mn * sigmoid_d(g[i]);
    }
    free(u); free(hid); free(logits); free(mean); free(g); free(wts);
}

/* Intersection (f_and of Eq. 2) of n >= 1 branch states. */
void kgo_intersect(const kgo_model* m, int n, const double* const* br, double* out)
{
    int d = m->dim;
    if (m->model == KGO_CONE) {
        cone_intersect(m, n, br, out);
        return;
    }
    if (m->model == KGO_LOGICE) {
        for (int i = 0; i < 2 * d; ++i) {
            double v = br[0][i];
            for (int j = 1; j < n; ++j) v = tnorm2(m->tnorm, v, br[j][i]);
            out[i] = v;
        }
        return;
    }
    int in_w = (m->model == KGO_BETAE) ? 2 * d : d;   /* attention input width */
    int hid = in_w;                                    /* attention hidden width */
    double* hbuf = (double*)malloc(sizeof(double) * (size_t)hid);
    double* logits = (double*)malloc(sizeof(double) * (size_t)n * d);
    double* wts = (double*)malloc(sizeof(double) * (size_t)n);
    for (int j = 0; j < n; ++j) {
        /* GQE: the query vector; Q2B: the center; BetaE: [alpha; beta]. */
        dense(m->att_w1, m->att_b1, hid, in_w, br[j], hbuf);
        relu_inplace(hbuf, hid);
        dense(m->att_w2, m->att_b2, d, hid, hbuf, logits + (size_t)j * d);
    }
    for (int i = 0; i < d; ++i) {
        double mx = logits[i];
        for (int j = 1; j < n; ++j) if (logits[(size_t)j * d + i] > mx) mx = logits[(size_t)j * d + i];
        double z = 0.0;
        for (int j = 0; j < n; ++j) { wts[j] = exp(logits[(size_t)j * d + i] - mx); z += wts[j]; }
        for (int j = 0; j < n; ++j) wts[j] /= z;
        if (m->model == KGO_BETAE) {
            double a = 0.0, b = 0.0;
            for (int j = 0; j < n; ++j) { a += wts[j] * br[j][i]; b += wts[j] * br[j][d + i]; }
            out[i] = a;
            out[d + i] = b;
        } else {
            double c = 0.0;
            for (int j = 0; j < n; ++j) c += wts[j] * br[j][i];
            out[i] = c;
        }
    }
    if (m->model == KGO_Q2B) {
        /* Offset: elementwise minimum over branches, shrunk by a sigmoid gate
         * computed from the mean of per-branch set-function features. */
        double* z = (double*)malloc(sizeof(double) * (size_t)d);
        double* mean = (double*)calloc((size_t)d, sizeof(double));
        double* g = (double*)malloc(sizeof(double) * (size_t)d);
        for (int j = 0; j < n; ++j) {
            dense(m->off_w1, m->off_b1, d, d, br[j] + d, z);
            relu_inplace(z, d);
            for (int i = 0; i < d; ++i) mean[i] += z[i];
        }
        for (int i = 0; i < d; ++i) mean[i] /= (double)n;
        dense(m->off_w2, m->off_b2, d, d, mean, g);
        for (int i = 0; i < d; ++i) {
            double mn = br[0][d + i];
            for (int j = 1; j < n; ++j) if (br[j][d + i] < mn) mn = br[j][d + i];
            out[d + i] = mn * sigmoid(g[i]);
        }
        free(z); free(mean); free(g);
    }
    free(hbuf);
    free(logits);
    free(wts);
}

/* Score of one entity against one query state (entity-similarity query). */
double kgo_score(const kgo_model* m, const double* st, int64_t e)
{
    int d = m->dim;
    if (m->model == KGO_GQE) {
        double s = 0.0;
        for (int i = 0; i < d; ++i) s += fabs(st[i] - (double)m->entity[(size_t)e * d + i]);
        return m->gamma - s;
    }
    if (m->model == KGO_Q2B) {
        double out = 0.0, in = 0.0;
        for (int i = 0; i < d; ++i) {
            double v = m->entity[(size_t)e * d + i];
            double c = st[i], o = st[d + i];
            double lo = c - o, hi = c + o;
            double mm = v > lo ? v : lo;       /* max(c - o, v) */
            if (mm > hi) mm = hi;              /* min(c + o, .) */
            out += fabs(v - mm);
            in += fabs(c - mm);
        }
        return m->gamma - (out + m->center_reg * in);
    }
    if (m->model == KGO_CONE) {
        double out = 0.0, in = 0.0;
        for (int i = 0; i < d; ++i) {
            double t = (double)m->entity[(size_t)e * d + i] - st[i];
            double psi = st[d + i];
            double to_axis = fabs(sin(0.5 * t));
            double base = fabs(sin(0.5 * psi));
            if (!(to_axis < base)) {
                double lo = fabs(sin(0.5 * (t + psi))), hi = fabs(sin(0.5 * (t - psi)));
                out += lo < hi ? lo : hi;
            }
            in += to_axis < base ? to_axis : base;
        }
        return m->gamma - m->modulus * (out + m->center_reg * in);
    }
    if (m->model == KGO_LOGICE) {
        double s = 0.0;
        for (int i = 0; i < 2 * d; ++i) s += fabs(st[i] - (double)m->entity[(size_t)e * 2 * d + i]);
        return m->gamma - s / (2.0 * d);
    }
    double kl = 0.0;
    for (int i = 0; i < d; ++i) {
        double ae = m->entity[(size_t)e * 2 * d + i], be = m->entity[(size_t)e * 2 * d + d + i];
        kl += kgo_kl_beta(ae, be, st[i], st[d + i]);
    }
    return m->gamma - kl;
}

/* ------------------------------------------------------------------ */
/* Query structures                                                    */
/* ------------------------------------------------------------------ */

enum { S_1P, S_2P, S_3P, S_2I, S_3I, S_PI, S_IP, S_2U, S_UP,
       S_2IN, S_3IN, S_INP, S_PIN, S_PNI, S_COUNT };

static const int ARITY_A[S_COUNT] = {1, 1, 1, 2, 3, 2, 2, 2, 2, 2, 3, 2, 2, 2};
static const int ARITY_R[S_COUNT] = {1, 2, 3, 2, 3, 3, 3, 2, 3, 2, 3, 3, 3, 3};

int kgo_arity(int s, int* na, int* nr)
{
    if (s < 0 || s >= S_COUNT) return -1;
    *na = ARITY_A[s];
    *nr = ARITY_R[s];
    return 0;
}

/* a0..a2 / r0..r2 refer to the query's anchor and relation slots in order. */
#define ANCHOR(st, k) kgo_anchor(m, a[k], st)
#define PROJ(st, k) kgo_project(m, st, r[k], st)

/* Evaluate one query; writes 1 or 2 final states (2 for a union, whose
 * entity score is the max over the two conjunctive branches of its DNF).
 * Returns the number of states, or -1 for an unknown or unsupported shape. */
int kgo_query_states(const kgo_model* m, int s, const int32_t* a, const int32_t* r, double* out)
{
    int w = kgo_state_width(m);
    g_margin = INFINITY;
    if (s < 0 || s >= S_COUNT) return -1;
    if (s >= S_2IN && !has_negation(m)) return -1;
    double* b0 = (double*)malloc(sizeof(double) * (size_t)w * 3);
    double* b1 = b0 + w;
    double* b2 = b1 + w;
    const double* br[3] = {b0, b1, b2};
    int nout = 1;
    switch (s) {
    case S_1P: ANCHOR(b0, 0); PROJ(b0, 0); memcpy(out, b0, sizeof(double) * w); break;
    case S_2P: ANCHOR(b0, 0); PROJ(b0, 0); PROJ(b0, 1); memcpy(out, b0, sizeof(double) * w); break;
    case S_3P: ANCHOR(b0, 0); PROJ(b0, 0); PROJ(b0, 1); PROJ(b0, 2);
               memcpy(out, b0, sizeof(double) * w); break;
    case S_2I: ANCHOR(b0, 0); PROJ(b0, 0); ANCHOR(b1, 1); PROJ(b1, 1);
               kgo_intersect(m, 2, br, out); break;
    case S_3I: ANCHOR(b0, 0); PROJ(b0, 0); ANCHOR(b1, 1); PROJ(b1, 1); ANCHOR(b2, 2); PROJ(b2, 2);
               kgo_intersect(m, 3, br, out); break;
    case S_PI: ANCHOR(b0, 0); PROJ(b0, 0); PROJ(b0, 1); ANCHOR(b1, 1); PROJ(b1, 2);
               kgo_intersect(m, 2, br, out); break;
    case S_IP: ANCHOR(b0, 0); PROJ(b0, 0); ANCHOR(b1, 1); PROJ(b1, 1);
               kgo_intersect(m, 2, br, out); kgo_project(m, out, r[2], out); break;
    case S_2U: ANCHOR(b0, 0); PROJ(b0, 0); ANCHOR(b1, 1); PROJ(b1, 1);
               memcpy(out, b0, sizeof(double) * w); memcpy(out + w, b1, sizeof(double) * w);
               nout = 2; break;
    case S_UP: /* DNF: (a0.r0 v a1.r1).r2 = (a0.r0.r2) v (a1.r1.r2) */
               ANCHOR(b0, 0); PROJ(b0, 0); PROJ(b0, 2); ANCHOR(b1, 1); PROJ(b1, 1); PROJ(b1, 2);
               memcpy(out, b0, sizeof(double) * w); memcpy(out + w, b1, sizeof(double) * w);
               nout = 2; break;
    case S_2IN: ANCHOR(b0, 0); PROJ(b0, 0); ANCHOR(b1, 1); PROJ(b1, 1); kgo_negate(m, b1, b1);
                kgo_intersect(m, 2, br, out); break;
    case S_3IN: ANCHOR(b0, 0); PROJ(b0, 0); ANCHOR(b1, 1); PROJ(b1, 1); ANCHOR(b2, 2); PROJ(b2, 2);
                kgo_negate(m, b2, b2); kgo_intersect(m, 3, br, out); break;
    case S_INP: ANCHOR(b0, 0); PROJ(b0, 0); ANCHOR(b1, 1); PROJ(b1, 1); kgo_negate(m, b1, b1);
                kgo_intersect(m, 2, br, out); kgo_project(m, out, r[2], out); break;
    case S_PIN: ANCHOR(b0, 0); PROJ(b0, 0); PROJ(b0, 1); ANCHOR(b1, 1); PROJ(b1, 2);
                kgo_negate(m, b1, b1); kgo_intersect(m, 2, br, out); break;
    case S_PNI: ANCHOR(b0, 0); PROJ(b0, 0); PROJ(b0, 1); kgo_negate(m, b0, b0);
                ANCHOR(b1, 1); PROJ(b1, 2); kgo_intersect(m, 2, br, out); break;
    }
    free(b0);
    return nout;
}

#undef ANCHOR
#undef PROJ

/* Margin (see g_margin) of the query last evaluated on this thread by
 * kgo_query_states or kgo_graph_states. */
double kgo_last_margin(void) { return g_margin; }

/* ------------------------------------------------------------------ */
/* Batched scoring and top-k                                           */
/* ------------------------------------------------------------------ */

static int set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
    return omp_get_max_threads();
#else
    (void)nthreads;
    return 1;
#endif
}

int kgo_max_threads(int nthreads) { return set_threads(nthreads); }

/* Entity-similarity query over all N entities for B queries whose answer
 * variable has nst[q] conjunctive terms (DNF, Eq. 1): the score of an
 * entity is the maximum of its scores against the terms. states is
 * [B][T][w] (term t of query q at (q * T + t) * w), scores is [B x N].
 * Entities are processed in chunks so that BetaE's per-entity function
 * values (psi, ln B) are computed once per chunk and then reused for every
 * query; the KL formula itself is unchanged. */
static void score_terms(const kgo_model* m, int32_t B, const double* states, const int* nst, int T,
                        double* scores)
{
    int w = kgo_state_width(m);
    int64_t N = m->n_entities;
    int d = m->dim;
    const int64_t CH = 256;
    int64_t nch = (N + CH - 1) / CH;
#pragma omp parallel
    {
        double* memo = NULL;
        if (m->model == KGO_BETAE) memo = (double*)malloc(sizeof(double) * (size_t)CH * d * 4);
#pragma omp for schedule(dynamic, 1)
        for (int64_t c = 0; c < nch; ++c) {
            int64_t e0 = c * CH, e1 = e0 + CH < N ? e0 + CH : N;
            if (m->model != KGO_BETAE) {
                for (int32_t q = 0; q < B; ++q) {
                    for (int64_t e = e0; e < e1; ++e) {
                        double best = 0.0;
                        for (int t = 0; t < nst[q]; ++t) {
                            double s = kgo_score(m, states + ((size_t)q * T + t) * w, e);
                            if (t == 0 || s > best) best = s;
                        }
                        scores[(size_t)q * N + e] = best;
                    }
                }
                continue;
            }
            /* BetaE: memo[(e-e0)*d + i] slots: lnB(a,b), psi(a), psi(b), psi(a+b). */
            for (int64_t e = e0; e < e1; ++e) {
                const float* ab = m->entity + (size_t)e * 2 * d;
                double* mm = memo + (size_t)(e - e0) * d * 4;
                for (int i = 0; i < d; ++i) {
                    double a1 = ab[i], b1 = ab[d + i];
                    mm[4 * i + 0] = kgo_lnbeta(a1, b1);
                    mm[4 * i + 1] = kgo_digamma(a1);
                    mm[4 * i + 2] = kgo_digamma(b1);
                    mm[4 * i + 3] = kgo_digamma(a1 + b1);
                }
            }
            double* lnbq = (double*)malloc(sizeof(double) * (size_t)d * 2);
            for (int32_t q = 0; q < B; ++q) {
                for (int t = 0; t < nst[q]; ++t) {
                    const double* st = states + ((size_t)q * T + t) * w;
                    for (int i = 0; i < d; ++i) lnbq[i] = kgo_lnbeta(st[i], st[d + i]);
                    for (int64_t e = e0; e < e1; ++e) {
                        const float* ab = m->entity + (size_t)e * 2 * d;
                        const double* mm = memo + (size_t)(e - e0) * d * 4;
                        double kl = 0.0;
                        for (int i = 0; i < d; ++i) {
                            double a1 = ab[i], b1 = ab[d + i], a2 = st[i], b2 = st[d + i];
                            /* KL(Beta(a1,b1) || Beta(a2,b2)) with memoised
                             * values of lnB and psi. */
                            kl += lnbq[i] - mm[4 * i + 0]
                                + (a1 - a2) * mm[4 * i + 1]
                                + (b1 - b2) * mm[4 * i + 2]
                                + (a2 - a1 + b2 - b1) * mm[4 * i + 3];
                        }
                        double s = m->gamma - kl;
                        if (t == 0 || s > scores[(size_t)q * N + e]) scores[(size_t)q * N + e] = s;
                    }
                }
            }
            free(lnbq);
        }
        free(memo);
    }
}

/* Scores of every entity for B queries. Query q has structure sid[q], anchors
 * anchors[q*astride ..] and relations rels[q*rstride ..]. scores is [B x N].
 * Returns 0, or -1 if any query has an unknown/unsupported structure or an
 * id outside the tables. */
int kgo_scores(const kgo_model* m, int32_t B, const int32_t* sid, const int32_t* anchors,
               int32_t astride, const int32_t* rels, int32_t rstride, double* scores,
               double* margin, int nthreads)
{
    int w = kgo_state_width(m);
    int64_t N = m->n_entities;
    if (m->dim > KGO_MAX_DIM) return -1;
    for (int32_t q = 0; q < B; ++q) {
        int na, nr;
        if (kgo_arity(sid[q], &na, &nr)) return -1;
        if (sid[q] >= S_2IN && !has_negation(m)) return -1;
        for (int k = 0; k < na; ++k) {
            int32_t e = anchors[(size_t)q * astride + k];
            if (e < 0 || e >= N) return -1;
        }
        for (int k = 0; k < nr; ++k) {
            int32_t r = rels[(size_t)q * rstride + k];
            if (r < 0 || r >= m->n_relations) return -1;
        }
    }
    set_threads(nthreads);
    double* states = (double*)malloc(sizeof(double) * (size_t)B * 2 * w);
    int* nst = (int*)malloc(sizeof(int) * (size_t)B);
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t q = 0; q < B; ++q) {
        nst[q] = kgo_query_states(m, sid[q], anchors + (size_t)q * astride,
                                  rels + (size_t)q * rstride, states + (size_t)q * 2 * w);
        if (margin) margin[q] = g_margin;
        if (nst[q] < 0) bad = 1;
    }
    if (!bad) score_terms(m, B, states, nst, 2, scores);
    free(states);
    free(nst);
    return bad ? -1 : 0;
}

/* ------------------------------------------------------------------ */
/* Query computation graphs                                            */
/* ------------------------------------------------------------------ */

/* A query computation graph (Eq. 2) is given as nodes in topological order,
 * KGO_NODE_WORDS int32 each: op, slot, in[0..3]. The ops follow Eq. 2's
 * mapping: an entity becomes a value node (op 0, anchor slot `slot`); a
 * relation becomes a projection of node in[0] (op 1, relation slot `slot`);
 * the connectives become f_and (op 2), f_or (op 3) over nodes in[0..] (two
 * to four, unused entries -1) and f_not of node in[0] (op 4). Inputs are
 * earlier nodes; the last node is the answer variable. */
#define KGO_OP_ANCHOR 0
#define KGO_OP_PROJECT 1
#define KGO_OP_AND 2
#define KGO_OP_OR 3
#define KGO_OP_NOT 4
#define KGO_NODE_WORDS 6
#define KGO_MAX_TERMS 16

/* Number of inputs of a node, or -1 if the node is malformed. */
static int node_inputs(const int32_t* g, int i)
{
    const int32_t* nd = g + (size_t)i * KGO_NODE_WORDS;
    int op = nd[0], k = 0;
    while (k < 4 && nd[2 + k] >= 0) ++k;
    for (int j = k; j < 4; ++j) if (nd[2 + j] != -1) return -1;
    for (int j = 0; j < k; ++j) if (nd[2 + j] >= i) return -1;   /* inputs are earlier nodes */
    switch (op) {
    case KGO_OP_ANCHOR: return (k == 0 && nd[1] >= 0) ? 0 : -1;
    case KGO_OP_PROJECT: return (k == 1 && nd[1] >= 0) ? 1 : -1;
    case KGO_OP_NOT: return k == 1 ? 1 : -1;
    case KGO_OP_AND:
    case KGO_OP_OR: return k >= 2 ? k : -1;
    }
    return -1;
}

/* Checks a graph and counts the anchor and relation slots it uses (largest
 * slot + 1) and the conjunctive terms of its answer. Returns 0, or -1 for a
 * malformed graph, a negation on a model without one, or more than
 * KGO_MAX_TERMS terms at any node. */
int kgo_graph_check(const kgo_model* m, const int32_t* g, int n, int* n_anchor_slots, int* n_rel_slots,
                    int* n_terms)
{
    if (n < 1 || n > 256) return -1;
    int* cnt = (int*)malloc(sizeof(int) * (size_t)n);
    int na = 0, nr = 0, ok = 1;
    for (int i = 0; i < n && ok; ++i) {
        const int32_t* nd = g + (size_t)i * KGO_NODE_WORDS;
        int k = node_inputs(g, i);
        if (k < 0) { ok = 0; break; }
        long c = 1;
        switch (nd[0]) {
        case KGO_OP_ANCHOR: if (nd[1] + 1 > na) na = nd[1] + 1; c = 1; break;
        case KGO_OP_PROJECT: if (nd[1] + 1 > nr) nr = nd[1] + 1; c = cnt[nd[2]]; break;
        case KGO_OP_NOT: if (!has_negation(m)) ok = 0; c = 1; break;
        case KGO_OP_OR: c = 0; for (int j = 0; j < k; ++j) c += cnt[nd[2 + j]]; break;
        case KGO_OP_AND: c = 1; for (int j = 0; j < k; ++j) c *= cnt[nd[2 + j]]; break;
        }
        if (c > KGO_MAX_TERMS) ok = 0;
        cnt[i] = (int)c;
    }
    if (ok) {
        *n_anchor_slots = na;
        *n_rel_slots = nr;
        *n_terms = cnt[n - 1];
    }
    free(cnt);
    return ok ? 0 : -1;
}

/* Evaluates one query's graph node by node. The value of each node is its
 * disjunctive normal form (Eq. 1): a list of conjunctive terms, each a query
 * state.
 *   entity:      one term, the anchor's embedding;
 *   projection:  each term projected;
 *   f_or:        the inputs' term lists concatenated;
 *   f_and:       one intersection per combination of one term from each
 *                input (conjunction distributes over disjunction), the
 *                first input's term varying slowest;
 *   f_not:       of a single term, its negation; of several terms, the
 *                intersection of their negations (De Morgan: the negation
 *                of a disjunction is the conjunction of the negations).
 * Writes the answer's terms to out (n_terms x w) and returns their number,
 * or -1 if the graph is rejected by kgo_graph_check. */
int kgo_graph_states(const kgo_model* m, const int32_t* g, int n, const int32_t* a, const int32_t* r,
                     double* out)
{
    int na, nr, nt;
    g_margin = INFINITY;
    if (kgo_graph_check(m, g, n, &na, &nr, &nt)) return -1;
    int w = kgo_state_width(m);
    int* cnt = (int*)calloc((size_t)n, sizeof(int));
    double** val = (double**)calloc((size_t)n, sizeof(double*));
    const double* br[KGO_MAX_TERMS];
    for (int i = 0; i < n; ++i) {
        const int32_t* nd = g + (size_t)i * KGO_NODE_WORDS;
        const int32_t* in = nd + 2;
        int k = node_inputs(g, i);
        int c = 0;
        switch (nd[0]) {
        case KGO_OP_ANCHOR:
            c = 1;
            val[i] = (double*)malloc(sizeof(double) * (size_t)w);
            kgo_anchor(m, a[nd[1]], val[i]);
            break;
        case KGO_OP_PROJECT:
            c = cnt[in[0]];
            val[i] = (double*)malloc(sizeof(double) * (size_t)c * w);
            for (int t = 0; t < c; ++t) kgo_project(m, val[in[0]] + (size_t)t * w, r[nd[1]], val[i] + (size_t)t * w);
            break;
        case KGO_OP_OR:
            for (int j = 0; j < k; ++j) c += cnt[in[j]];
            val[i] = (double*)malloc(sizeof(double) * (size_t)c * w);
            for (int j = 0, t0 = 0; j < k; t0 += cnt[in[j]], ++j)
                memcpy(val[i] + (size_t)t0 * w, val[in[j]], sizeof(double) * (size_t)cnt[in[j]] * w);
            break;
        case KGO_OP_AND:
            c = 1;
            for (int j = 0; j < k; ++j) c *= cnt[in[j]];
            val[i] = (double*)malloc(sizeof(double) * (size_t)c * w);
            for (int t = 0; t < c; ++t) {
                /* mixed-radix digits of t, last input fastest */
                int rest = t;
                for (int j = k - 1; j >= 0; --j) {
                    br[j] = val[in[j]] + (size_t)(rest % cnt[in[j]]) * w;
                    rest /= cnt[in[j]];
                }
                kgo_intersect(m, k, br, val[i] + (size_t)t * w);
            }
            break;
        case KGO_OP_NOT: {
            int ci = cnt[in[0]];
            c = 1;
            val[i] = (double*)malloc(sizeof(double) * (size_t)w);
            if (ci == 1) {
                kgo_negate(m, val[in[0]], val[i]);
            } else {
                double* neg = (double*)malloc(sizeof(double) * (size_t)ci * w);
                for (int t = 0; t < ci; ++t) {
                    kgo_negate(m, val[in[0]] + (size_t)t * w, neg + (size_t)t * w);
                    br[t] = neg + (size_t)t * w;
                }
                kgo_intersect(m, ci, br, val[i]);
                free(neg);
            }
            break;
        }
        }
        cnt[i] = c;
    }
    memcpy(out, val[n - 1], sizeof(double) * (size_t)cnt[n - 1] * w);
    int res = cnt[n - 1];
    for (int i = 0; i < n; ++i) free(val[i]);
    free(val);
    free(cnt);
    return res;
}

/* Scores of every entity for B queries sharing one graph: query q's anchor
 * slots are anchors[q*astride ..], its relation slots rels[q*rstride ..].
 * Returns 0, or -1 for a rejected graph or an id outside the tables. */
int kgo_graph_scores(const kgo_model* m, const int32_t* g, int n, int32_t B, const int32_t* anchors,
                     int32_t astride, const int32_t* rels, int32_t rstride, double* scores, double* margin,
                     int nthreads)
{
    int na, nr, nt;
    if (m->dim > KGO_MAX_DIM) return -1;
    if (kgo_graph_check(m, g, n, &na, &nr, &nt)) return -1;
    if (na > astride || nr > rstride) return -1;
    for (int32_t q = 0; q < B; ++q) {
        for (int k = 0; k < na; ++k) {
            int32_t e = anchors[(size_t)q * astride + k];
            if (e < 0 || e >= m->n_entities) return -1;
        }
        for (int k = 0; k < nr; ++k) {
            int32_t r = rels[(size_t)q * rstride + k];
            if (r < 0 || r >= m->n_relations) return -1;
        }
    }
    set_threads(nthreads);
    int w = kgo_state_width(m);
    double* states = (double*)malloc(sizeof(double) * (size_t)B * nt * w);
    int* nst = (int*)malloc(sizeof(int) * (size_t)B);
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t q = 0; q < B; ++q) {
        nst[q] = kgo_graph_states(m, g, n, anchors + (size_t)q * astride, rels + (size_t)q * rstride,
                                  states + (size_t)q * nt * w);
        if (margin) margin[q] = g_margin;
    }
    score_terms(m, B, states, nst, nt, scores);
    free(states);
    free(nst);
    return 0;
}

/* Ranking order: higher score first; equal scores by lower entity index. */
static int ranks_before(double sa, int64_t ia, double sb, int64_t ib)
{
    return sa > sb || (sa == sb && ia < ib);
}

/* Top-k of each row of scores [B x N]: a size-k heap whose root is the
 * weakest kept entry, then the kept entries in ranking order. */
int kgo_topk(const double* scores, int32_t B, int64_t N, int32_t k, int32_t* idx, double* val,
             int nthreads)
{
    if (k < 1 || k > N) return -1;
    set_threads(nthreads);
#pragma omp parallel
    {
        int64_t* hi = (int64_t*)malloc(sizeof(int64_t) * (size_t)k);
        double* hs = (double*)malloc(sizeof(double) * (size_t)k);
#pragma omp for schedule(dynamic, 1)
        for (int32_t q = 0; q < B; ++q) {
            const double* row = scores + (size_t)q * N;
            int n = 0;
            for (int64_t e = 0; e < N; ++e) {
                double s = row[e];
                if (n < k) {
                    /* sift up: the root holds the entry that ranks last */
                    int c = n++;
                    while (c > 0) {
                        int p = (c - 1) / 2;
                        if (!ranks_before(hs[p], hi[p], s, e)) break;
                        hs[c] = hs[p]; hi[c] = hi[p];
                        c = p;
                    }
                    hs[c] = s; hi[c] = e;
                } else if (ranks_before(s, e, hs[0], hi[0])) {
                    int c = 0;
                    for (;;) {
                        int l = 2 * c + 1, r = l + 1, worst = -1;
                        double ws = s; int64_t wi = e;
                        if (l < k && ranks_before(ws, wi, hs[l], hi[l])) { worst = l; ws = hs[l]; wi = hi[l]; }
                        if (r < k && ranks_before(ws, wi, hs[r], hi[r])) { worst = r; ws = hs[r]; wi = hi[r]; }
                        if (worst < 0) break;
                        hs[c] = hs[worst]; hi[c] = hi[worst];
                        c = worst;
                    }
                    hs[c] = s; hi[c] = e;
                }
            }
            /* pop the weakest into the last slot until empty */
            for (int t = k - 1; t >= 0; --t) {
                idx[(size_t)q * k + t] = (int32_t)hi[0];
                val[(size_t)q * k + t] = hs[0];
                double s = hs[t]; int64_t e = hi[t];
                int m2 = t, c = 0;
                if (m2 > 0) {
                    for (;;) {
                        int l = 2 * c + 1, r = l + 1, worst = -1;
                        double ws = s; int64_t wi = e;
                        if (l < m2 && ranks_before(ws, wi, hs[l], hi[l])) { worst = l; ws = hs[l]; wi = hi[l]; }
                        if (r < m2 && ranks_before(ws, wi, hs[r], hi[r])) { worst = r; ws = hs[r]; wi = hi[r]; }
                        if (worst < 0) break;
                        hs[c] = hs[worst]; hi[c] = hi[worst];
                        c = worst;
                    }
                    hs[c] = s; hi[c] = e;
                }
            }
        }
        free(hi);
        free(hs);
    }
    return 0;
}


/* Filtered ranks of answer entities and ranking metrics (the paper reports
 * MRR; Experiments). For query q with answer set A_q (ids[offsets[q] ..
 * offsets[q+1]), all distinct), the filtered rank of answer a is
 *   1 + #{ e in [0, N) : e not in A_q and e ranks before a },
 * "ranks before" being the ranking order above (higher score first, equal
 * scores by lower entity index), applied to the float32 scores as given.
 * Metrics per query over its hard answers H_q (hard[i] != 0; hard == NULL:
 * every answer is hard), in double precision in answer-list order:
 *   metrics[4q + 0] = mean over H_q of 1 / rank      (MRR)
 *   metrics[4q + j] = mean over H_q of [rank <= K_j]  (Hits@1, @3, @10)
 * A query without hard answers gets NaN metrics. Returns 0, or -1 for an
 * answer id outside [0, N) or a negative list length. */
int kgo_rank_answers(const float* scores, int32_t B, int64_t N, const int32_t* offsets, const int32_t* ids,
                     const int32_t* hard, int32_t* rank, double* metrics, int nthreads)
{
    static const int hits_k[3] = {1, 3, 10};
    for (int32_t q = 0; q < B; ++q) {
        if (offsets[q + 1] < offsets[q]) return -1;
        for (int32_t i = offsets[q]; i < offsets[q + 1]; ++i)
            if (ids[i] < 0 || ids[i] >= N) return -1;
    }
    set_threads(nthreads);
#pragma omp parallel
    {
        unsigned char* is_ans = (unsigned char*)calloc((size_t)N, 1);
#pragma omp for schedule(dynamic, 1)
        for (int32_t q = 0; q < B; ++q) {
            const float* row = scores + (size_t)q * N;
            const int32_t lo = offsets[q], hi = offsets[q + 1];
            for (int32_t i = lo; i < hi; ++i) is_ans[ids[i]] = 1;
            for (int32_t i = lo; i < hi; ++i) {
                const int64_t a = ids[i];
                int64_t before = 0;
                for (int64_t e = 0; e < N; ++e)
                    if (!is_ans[e] && ranks_before(row[e], e, row[a], a)) ++before;
                rank[i] = (int32_t)(1 + before);
            }
            double mrr = 0.0, hk[3] = {0.0, 0.0, 0.0};
            int64_t nh = 0;
            for (int32_t i = lo; i < hi; ++i) {
                if (hard && !hard[i]) continue;
                ++nh;
                mrr += 1.0 / (double)rank[i];
                for (int j = 0; j < 3; ++j) hk[j] += rank[i] <= hits_k[j] ? 1.0 : 0.0;
            }
            double* m = metrics + (size_t)4 * q;
            if (nh == 0) {
                m[0] = m[1] = m[2] = m[3] = NAN;
            } else {
                m[0] = mrr / (double)nh;
                for (int j = 0; j < 3; ++j) m[1 + j] = hk[j] / (double)nh;
            }
            for (int32_t i = lo; i < hi; ++i) is_ans[ids[i]] = 0;
        }
        free(is_ans);
    }
    return 0;
}
