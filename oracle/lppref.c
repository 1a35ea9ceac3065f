/*
 * lppref.c -- the fp64 CPU oracle for the LPP-SGD per-node step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code with the HIP library: its own layer
 * records, its own shape inference, its own loops.
 *
 * What it computes (paper "Scaling the Wild: Decentralizing Hogwild!-style
 * Shared-memory SGD", arXiv 2203.06638):
 *   - the model vector x in R^d as the concatenation of the CNN's parameter
 *     tensors in model order (Sec. 3, "Block partitions", eq. (partition));
 *   - the minibatch stochastic gradient of the mean softmax cross-entropy
 *     with respect to all of x, by the ordinary chain rule (Sec. 2, the
 *     block gradient is the restriction of this to a block);
 *   - the updater's lock-free block update x_i -= alpha * (direction)
 *     (Alg. 1, updater loop; Sec. 5 "minor iteration view", operator -|_i);
 *   - the averager's in-place update x += (mean of snapshots - own snapshot)
 *     (Alg. 1, averaging loop).
 *
 * Everything is double precision, NCHW, direct loops, no BLAS, no blocking.
 * OpenMP only splits independent output elements across threads; every
 * output element is summed by exactly one thread in a fixed order, so
 * results do not depend on the thread count.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ---- layer records (the oracle's own; mirrored by oracle/lppref.py) ---- */
enum { R_CONV = 0, R_BN = 1, R_RELU = 2, R_ADD = 3, R_MAXPOOL = 4, R_GAP = 5, R_LINEAR = 6, R_CONCAT = 7 };

typedef struct {
    int op;
    int in0, in1;            /* producer layer index; -1 = the image batch    */
    int cin, cout;           /* channels (conv, linear; bn uses cout)         */
    int k, stride, pad;      /* conv / maxpool window                         */
    int bias;                /* conv / linear have a bias vector              */
    long poff;               /* first index of this layer's params in x, or -1 */
} ref_layer;

typedef struct { int c, h, w; } shp;

static shp in_shape(const shp* S, int idx, shp img) { return idx < 0 ? img : S[idx]; }

/* Infer every layer's output shape; returns 0 on success. */
static int infer_shapes(const ref_layer* L, int nl, shp img, shp* S) {
    for (int l = 0; l < nl; ++l) {
        shp a = in_shape(S, L[l].in0, img);
        shp o = a;
        switch (L[l].op) {
        case R_CONV:
            if (a.c != L[l].cin) return -1;
            o.c = L[l].cout;
            o.h = (a.h + 2 * L[l].pad - L[l].k) / L[l].stride + 1;
            o.w = (a.w + 2 * L[l].pad - L[l].k) / L[l].stride + 1;
            break;
        case R_BN: case R_RELU: break;
        case R_ADD: {
            shp b = in_shape(S, L[l].in1, img);
            if (b.c != a.c || b.h != a.h || b.w != a.w) return -1;
            break;
        }
        case R_MAXPOOL:
            o.h = (a.h + 2 * L[l].pad - L[l].k) / L[l].stride + 1;
            o.w = (a.w + 2 * L[l].pad - L[l].k) / L[l].stride + 1;
            break;
        case R_CONCAT: {   /* channels of in0, then channels of in1 */
            shp b = in_shape(S, L[l].in1, img);
            if (b.h != a.h || b.w != a.w) return -1;
            o.c = a.c + b.c;
            break;
        }
        case R_GAP: o.h = 1; o.w = 1; break;
        case R_LINEAR:
            if (a.c * a.h * a.w != L[l].cin) return -1;
            o.c = L[l].cout; o.h = 1; o.w = 1;
            break;
        default: return -1;
        }
        S[l] = o;
    }
    return 0;
}

static long numel(shp s, int n) { return (long)n * s.c * s.h * s.w; }

/* Number of parameters a layer owns, from its record alone. */
static long layer_params(const ref_layer* l) {
    switch (l->op) {
    case R_CONV: return (long)l->cout * l->cin * l->k * l->k + (l->bias ? l->cout : 0);
    case R_BN: return 2L * l->cout;
    case R_LINEAR: return (long)l->cout * l->cin + (l->bias ? l->cout : 0);
    default: return 0;
    }
}

long ref_num_params(const ref_layer* L, int nl) {
    long d = 0;
    for (int l = 0; l < nl; ++l) d += layer_params(&L[l]);
    return d;
}

/* ---------------------------- forward pieces ---------------------------- */

/* Cross-correlation with zero padding: Y[n][k][p][q] = b[k] +
 * sum_{c,r,s} W[k][c][r][s] * X[n][c][p*st - pad + r][q*st - pad + s]. */
static void conv_fwd(const double* X, shp a, int N, const double* Wt, const double* b,
                     int K, int R, int st, int pad, double* Y, shp o) {
    #pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int k = 0; k < K; ++k)
            for (int p = 0; p < o.h; ++p)
                for (int q = 0; q < o.w; ++q) {
                    double acc = b ? b[k] : 0.0;
                    for (int c = 0; c < a.c; ++c)
                        for (int r = 0; r < R; ++r) {
                            int hi = p * st - pad + r;
                            if (hi < 0 || hi >= a.h) continue;
                            for (int s = 0; s < R; ++s) {
                                int wi = q * st - pad + s;
                                if (wi < 0 || wi >= a.w) continue;
                                acc += Wt[((long)(k * a.c + c) * R + r) * R + s] *
                                       X[(((long)n * a.c + c) * a.h + hi) * a.w + wi];
                            }
                        }
                    Y[(((long)n * K + k) * o.h + p) * o.w + q] = acc;
                }
}

/* Training-mode batch normalisation over (N,H,W) per channel with the biased
 * batch variance; keeps mean and 1/sqrt(var+eps) for the backward pass. */
static void bn_fwd(const double* X, shp a, int N, const double* gamma, const double* beta,
                   double eps, double* Y, double* mean, double* rstd) {
    long hw = (long)a.h * a.w, M = hw * N;
    #pragma omp parallel for schedule(static)
    for (int c = 0; c < a.c; ++c) {
        double s = 0.0;
        for (int n = 0; n < N; ++n)
            for (long e = 0; e < hw; ++e) s += X[((long)n * a.c + c) * hw + e];
        double mu = s / (double)M, v = 0.0;
        for (int n = 0; n < N; ++n)
            for (long e = 0; e < hw; ++e) {
                double t = X[((long)n * a.c + c) * hw + e] - mu;
                v += t * t;
            }
        v /= (double)M;
        double r = 1.0 / sqrt(v + eps);
        mean[c] = mu; rstd[c] = r;
        for (int n = 0; n < N; ++n)
            for (long e = 0; e < hw; ++e) {
                long i = ((long)n * a.c + c) * hw + e;
                Y[i] = gamma[c] * (X[i] - mu) * r + beta[c];
            }
    }
}

/* Max over the window; padding never wins (acts as -infinity). */
static void maxpool_fwd(const double* X, shp a, int N, int R, int st, int pad, double* Y, shp o) {
    #pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < a.c; ++c)
            for (int p = 0; p < o.h; ++p)
                for (int q = 0; q < o.w; ++q) {
                    double m = -INFINITY;
                    for (int r = 0; r < R; ++r)
                        for (int s = 0; s < R; ++s) {
                            int hi = p * st - pad + r, wi = q * st - pad + s;
                            if (hi < 0 || hi >= a.h || wi < 0 || wi >= a.w) continue;
                            double v = X[(((long)n * a.c + c) * a.h + hi) * a.w + wi];
                            if (v > m) m = v;
                        }
                    Y[(((long)n * a.c + c) * o.h + p) * o.w + q] = m;
                }
}

/* ---------------------------- backward pieces --------------------------- */

/* Adds this conv's contribution to dX (if wanted) and writes dW, db. */
static void conv_bwd(const double* X, shp a, int N, const double* Wt, int K, int R, int st, int pad,
                     const double* dY, shp o, double* dX, double* dW, double* db) {
    if (dW) {
        #pragma omp parallel for collapse(2) schedule(static)
        for (int k = 0; k < K; ++k)
            for (int c = 0; c < a.c; ++c)
                for (int r = 0; r < R; ++r)
                    for (int s = 0; s < R; ++s) {
                        double acc = 0.0;
                        for (int n = 0; n < N; ++n)
                            for (int p = 0; p < o.h; ++p) {
                                int hi = p * st - pad + r;
                                if (hi < 0 || hi >= a.h) continue;
                                for (int q = 0; q < o.w; ++q) {
                                    int wi = q * st - pad + s;
                                    if (wi < 0 || wi >= a.w) continue;
                                    acc += dY[(((long)n * K + k) * o.h + p) * o.w + q] *
                                           X[(((long)n * a.c + c) * a.h + hi) * a.w + wi];
                                }
                            }
                        dW[((long)(k * a.c + c) * R + r) * R + s] = acc;
                    }
    }
    if (db) {
        for (int k = 0; k < K; ++k) {
            double acc = 0.0;
            for (int n = 0; n < N; ++n)
                for (long e = 0; e < (long)o.h * o.w; ++e) acc += dY[((long)n * K + k) * o.h * o.w + e];
            db[k] = acc;
        }
    }
    if (dX) {
        #pragma omp parallel for schedule(static)
        for (int n = 0; n < N; ++n)
            for (int k = 0; k < K; ++k)
                for (int p = 0; p < o.h; ++p)
                    for (int q = 0; q < o.w; ++q) {
                        double g = dY[(((long)n * K + k) * o.h + p) * o.w + q];
                        for (int c = 0; c < a.c; ++c)
                            for (int r = 0; r < R; ++r) {
                                int hi = p * st - pad + r;
                                if (hi < 0 || hi >= a.h) continue;
                                for (int s = 0; s < R; ++s) {
                                    int wi = q * st - pad + s;
                                    if (wi < 0 || wi >= a.w) continue;
                                    dX[(((long)n * a.c + c) * a.h + hi) * a.w + wi] +=
                                        g * Wt[((long)(k * a.c + c) * R + r) * R + s];
                                }
                            }
                    }
    }
}

/* y = gamma * xhat + beta with xhat = (x - mean) * rstd.  Then
 * dgamma = sum dy*xhat, dbeta = sum dy,
 * dx = gamma * rstd / M * (M*dy - dbeta - xhat*dgamma). */
static void bn_bwd(const double* X, shp a, int N, const double* gamma, const double* mean,
                   const double* rstd, const double* dY, double* dX, double* dgamma, double* dbeta) {
    long hw = (long)a.h * a.w, M = hw * N;
    #pragma omp parallel for schedule(static)
    for (int c = 0; c < a.c; ++c) {
        double sdy = 0.0, sdyx = 0.0;
        for (int n = 0; n < N; ++n)
            for (long e = 0; e < hw; ++e) {
                long i = ((long)n * a.c + c) * hw + e;
                sdy += dY[i];
                sdyx += dY[i] * (X[i] - mean[c]) * rstd[c];
            }
        if (dgamma) dgamma[c] = sdyx;
        if (dbeta) dbeta[c] = sdy;
        if (dX) {
            double f = gamma[c] * rstd[c] / (double)M;
            for (int n = 0; n < N; ++n)
                for (long e = 0; e < hw; ++e) {
                    long i = ((long)n * a.c + c) * hw + e;
                    double xh = (X[i] - mean[c]) * rstd[c];
                    dX[i] += f * ((double)M * dY[i] - sdy - xh * sdyx);
                }
        }
    }
}

/* The gradient goes to the first maximal element of each window, scanning
 * rows then columns. */
static void maxpool_bwd(const double* X, shp a, int N, int R, int st, int pad,
                        const double* dY, shp o, double* dX) {
    #pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < a.c; ++c)
            for (int p = 0; p < o.h; ++p)
                for (int q = 0; q < o.w; ++q) {
                    double m = -INFINITY; long arg = -1;
                    for (int r = 0; r < R; ++r)
                        for (int s = 0; s < R; ++s) {
                            int hi = p * st - pad + r, wi = q * st - pad + s;
                            if (hi < 0 || hi >= a.h || wi < 0 || wi >= a.w) continue;
                            long i = (((long)n * a.c + c) * a.h + hi) * a.w + wi;
                            if (X[i] > m) { m = X[i]; arg = i; }
                        }
                    if (arg >= 0) dX[arg] += dY[(((long)n * a.c + c) * o.h + p) * o.w + q];
                }
}

/* ------------------------------ the model ------------------------------- */

/* ---------------- condition scales of the parameter gradients ----------------
 * For every parameter gradient, which is a sum of products, the sum of the
 * magnitudes of those products.  A sum of terms each known to relative
 * accuracy delta can only be computed to about delta times this scale, so
 * it is the right yardstick for a gradient entry whose terms cancel. */
static void conv_wscale(const double* X, shp a, int N, int K, int R, int st, int pad,
                        const double* dY, shp o, double* sW, double* sb) {
    #pragma omp parallel for collapse(2) schedule(static)
    for (int k = 0; k < K; ++k)
        for (int c = 0; c < a.c; ++c)
            for (int r = 0; r < R; ++r)
                for (int s = 0; s < R; ++s) {
                    double acc = 0.0;
                    for (int n = 0; n < N; ++n)
                        for (int p = 0; p < o.h; ++p) {
                            int hi = p * st - pad + r;
                            if (hi < 0 || hi >= a.h) continue;
                            for (int q = 0; q < o.w; ++q) {
                                int wi = q * st - pad + s;
                                if (wi < 0 || wi >= a.w) continue;
                                acc += fabs(dY[(((long)n * K + k) * o.h + p) * o.w + q] *
                                            X[(((long)n * a.c + c) * a.h + hi) * a.w + wi]);
                            }
                        }
                    sW[((long)(k * a.c + c) * R + r) * R + s] = acc;
                }
    if (sb)
        for (int k = 0; k < K; ++k) {
            double acc = 0.0;
            for (int n = 0; n < N; ++n)
                for (long e = 0; e < (long)o.h * o.w; ++e) acc += fabs(dY[((long)n * K + k) * o.h * o.w + e]);
            sb[k] = acc;
        }
}

static void bn_scale(const double* X, shp a, int N, const double* mean, const double* rstd,
                     const double* dY, double* sg, double* sb) {
    long hw = (long)a.h * a.w;
    for (int c = 0; c < a.c; ++c) {
        double s1 = 0.0, s2 = 0.0;
        for (int n = 0; n < N; ++n)
            for (long e = 0; e < hw; ++e) {
                long i = ((long)n * a.c + c) * hw + e;
                s1 += fabs(dY[i]);
                s2 += fabs(dY[i] * (X[i] - mean[c]) * rstd[c]);
            }
        sg[c] = s2;
        sb[c] = s1;
    }
}

/* Runs the forward pass, filling act[l] (and BN statistics) for every layer. */
static void run_forward(const ref_layer* L, int nl, int N, shp img, const shp* S, const double* x,
                        const double* images, double bn_eps, double** act, double** bmean, double** brstd) {
    for (int l = 0; l < nl; ++l) {
        const ref_layer* y = &L[l];
        shp a = in_shape(S, y->in0, img);
        const double* X0 = y->in0 < 0 ? images : act[y->in0];
        long n0 = numel(a, N);
        switch (y->op) {
        case R_CONV: {
            const double* Wt = x + y->poff;
            const double* b = y->bias ? Wt + (long)y->cout * y->cin * y->k * y->k : NULL;
            conv_fwd(X0, a, N, Wt, b, y->cout, y->k, y->stride, y->pad, act[l], S[l]);
            break;
        }
        case R_BN:
            bn_fwd(X0, a, N, x + y->poff, x + y->poff + y->cout, bn_eps, act[l], bmean[l], brstd[l]);
            break;
        case R_RELU:
            for (long i = 0; i < n0; ++i) act[l][i] = X0[i] > 0.0 ? X0[i] : 0.0;
            break;
        case R_ADD: {
            const double* X1 = y->in1 < 0 ? images : act[y->in1];
            for (long i = 0; i < n0; ++i) act[l][i] = X0[i] + X1[i];
            break;
        }
        case R_MAXPOOL:
            maxpool_fwd(X0, a, N, y->k, y->stride, y->pad, act[l], S[l]);
            break;
        case R_CONCAT: {
            shp b = in_shape(S, y->in1, img);
            const double* X1 = y->in1 < 0 ? images : act[y->in1];
            long na = (long)a.c * a.h * a.w, nb = (long)b.c * b.h * b.w;
            for (int n = 0; n < N; ++n) {
                memcpy(act[l] + n * (na + nb), X0 + n * na, sizeof(double) * (size_t)na);
                memcpy(act[l] + n * (na + nb) + na, X1 + n * nb, sizeof(double) * (size_t)nb);
            }
            break;
        }
        case R_GAP: {
            long hw = (long)a.h * a.w;
            for (long nc = 0; nc < (long)N * a.c; ++nc) {
                double s = 0.0;
                for (long e = 0; e < hw; ++e) s += X0[nc * hw + e];
                act[l][nc] = s / (double)hw;
            }
            break;
        }
        case R_LINEAR: {
            const double* Wt = x + y->poff;
            const double* b = y->bias ? Wt + (long)y->cout * y->cin : NULL;
            for (int n = 0; n < N; ++n)
                for (int o = 0; o < y->cout; ++o) {
                    double acc = b ? b[o] : 0.0;
                    for (int i = 0; i < y->cin; ++i) acc += Wt[(long)o * y->cin + i] * X0[(long)n * y->cin + i];
                    act[l][(long)n * y->cout + o] = acc;
                }
            break;
        }
        }
    }
}

/*
 * Forward, mean softmax cross-entropy and (if grad != NULL) the gradient of
 * the loss with respect to every parameter.
 *   x       : parameters, d doubles, layout given by each layer's poff
 *   images  : N x C x H x W doubles (NCHW)
 *   labels  : N ints in [0, n_classes)
 *   logits  : N x n_classes out (may be NULL)
 *   loss    : scalar out
 *   grad    : d doubles out (may be NULL: forward only)
 * The last layer's output is the logits.  Returns 0, or -1 on a bad model.
 */
static int forward_backward_impl(const ref_layer* L, int nl, int N, int C, int H, int W,
                                 const double* x, const double* images, const int* labels,
                                 double bn_eps, double* logits, double* loss, double* grad,
                                 int gl, double* gout, double* gscale) {
    shp img = { C, H, W };
    shp* S = (shp*)calloc((size_t)nl, sizeof(shp));
    if (!S || infer_shapes(L, nl, img, S)) { free(S); return -1; }
    double** act = (double**)calloc((size_t)nl, sizeof(double*));
    double** dact = (double**)calloc((size_t)nl, sizeof(double*));
    double** bmean = (double**)calloc((size_t)nl, sizeof(double*));
    double** brstd = (double**)calloc((size_t)nl, sizeof(double*));
    for (int l = 0; l < nl; ++l) {
        act[l] = (double*)calloc((size_t)numel(S[l], N), sizeof(double));
        if (L[l].op == R_BN) {
            bmean[l] = (double*)calloc((size_t)S[l].c, sizeof(double));
            brstd[l] = (double*)calloc((size_t)S[l].c, sizeof(double));
        }
    }
    run_forward(L, nl, N, img, S, x, images, bn_eps, act, bmean, brstd);

    /* loss: mean over the batch of logsumexp(z) - z[label] */
    int ncls = S[nl - 1].c * S[nl - 1].h * S[nl - 1].w;
    const double* Z = act[nl - 1];
    double* dZ = (double*)calloc((size_t)N * ncls, sizeof(double));
    double tot = 0.0;
    for (int n = 0; n < N; ++n) {
        double mx = Z[(long)n * ncls];
        for (int j = 1; j < ncls; ++j) if (Z[(long)n * ncls + j] > mx) mx = Z[(long)n * ncls + j];
        double se = 0.0;
        for (int j = 0; j < ncls; ++j) se += exp(Z[(long)n * ncls + j] - mx);
        double lse = mx + log(se);
        tot += lse - Z[(long)n * ncls + labels[n]];
        for (int j = 0; j < ncls; ++j)
            dZ[(long)n * ncls + j] = (exp(Z[(long)n * ncls + j] - lse) - (j == labels[n] ? 1.0 : 0.0)) / (double)N;
    }
    *loss = tot / (double)N;
    if (logits) memcpy(logits, Z, sizeof(double) * (size_t)N * ncls);

    if (grad) {
        long d = ref_num_params(L, nl);
        memset(grad, 0, sizeof(double) * (size_t)d);
        for (int l = 0; l < nl; ++l) dact[l] = (double*)calloc((size_t)numel(S[l], N), sizeof(double));
        memcpy(dact[nl - 1], dZ, sizeof(double) * (size_t)N * ncls);
        for (int l = nl - 1; l >= 0; --l) {
            const ref_layer* y = &L[l];
            shp a = in_shape(S, y->in0, img);
            const double* X0 = y->in0 < 0 ? images : act[y->in0];
            double* dX0 = y->in0 < 0 ? NULL : dact[y->in0];
            const double* dY = dact[l];
            long n0 = numel(a, N);
            switch (y->op) {
            case R_CONV: {
                const double* Wt = x + y->poff;
                double* dW = grad + y->poff;
                double* db = y->bias ? dW + (long)y->cout * y->cin * y->k * y->k : NULL;
                conv_bwd(X0, a, N, Wt, y->cout, y->k, y->stride, y->pad, dY, S[l], dX0, dW, db);
                if (gscale)
                    conv_wscale(X0, a, N, y->cout, y->k, y->stride, y->pad, dY, S[l], gscale + y->poff,
                                y->bias ? gscale + y->poff + (long)y->cout * y->cin * y->k * y->k : NULL);
                break;
            }
            case R_BN:
                bn_bwd(X0, a, N, x + y->poff, bmean[l], brstd[l], dY, dX0,
                       grad + y->poff, grad + y->poff + y->cout);
                if (gscale) bn_scale(X0, a, N, bmean[l], brstd[l], dY, gscale + y->poff, gscale + y->poff + y->cout);
                break;
            case R_RELU:
                if (dX0) for (long i = 0; i < n0; ++i) dX0[i] += X0[i] > 0.0 ? dY[i] : 0.0;
                break;
            case R_ADD: {
                double* dX1 = y->in1 < 0 ? NULL : dact[y->in1];
                if (dX0) for (long i = 0; i < n0; ++i) dX0[i] += dY[i];
                if (dX1) for (long i = 0; i < n0; ++i) dX1[i] += dY[i];
                break;
            }
            case R_MAXPOOL:
                if (dX0) maxpool_bwd(X0, a, N, y->k, y->stride, y->pad, dY, S[l], dX0);
                break;
            case R_CONCAT: {
                shp b = in_shape(S, y->in1, img);
                double* dX1 = y->in1 < 0 ? NULL : dact[y->in1];
                long na = (long)a.c * a.h * a.w, nb = (long)b.c * b.h * b.w;
                for (int n = 0; n < N; ++n) {
                    if (dX0) for (long i = 0; i < na; ++i) dX0[n * na + i] += dY[n * (na + nb) + i];
                    if (dX1) for (long i = 0; i < nb; ++i) dX1[n * nb + i] += dY[n * (na + nb) + na + i];
                }
                break;
            }
            case R_GAP: {
                long hw = (long)a.h * a.w;
                if (dX0)
                    for (long nc = 0; nc < (long)N * a.c; ++nc)
                        for (long e = 0; e < hw; ++e) dX0[nc * hw + e] += dY[nc] / (double)hw;
                break;
            }
            case R_LINEAR: {
                const double* Wt = x + y->poff;
                double* dW = grad + y->poff;
                for (int o = 0; o < y->cout; ++o) {
                    for (int i = 0; i < y->cin; ++i) {
                        double acc = 0.0;
                        for (int n = 0; n < N; ++n) acc += dY[(long)n * y->cout + o] * X0[(long)n * y->cin + i];
                        dW[(long)o * y->cin + i] = acc;
                    }
                    if (y->bias) {
                        double acc = 0.0;
                        for (int n = 0; n < N; ++n) acc += dY[(long)n * y->cout + o];
                        dW[(long)y->cout * y->cin + o] = acc;
                    }
                }
                if (dX0)
                    for (int n = 0; n < N; ++n)
                        for (int i = 0; i < y->cin; ++i) {
                            double acc = 0.0;
                            for (int o = 0; o < y->cout; ++o) acc += dY[(long)n * y->cout + o] * Wt[(long)o * y->cin + i];
                            dX0[(long)n * y->cin + i] += acc;
                        }
                if (gscale)
                    for (int o = 0; o < y->cout; ++o) {
                        for (int i = 0; i < y->cin; ++i) {
                            double acc = 0.0;
                            for (int n = 0; n < N; ++n) acc += fabs(dY[(long)n * y->cout + o] * X0[(long)n * y->cin + i]);
                            gscale[y->poff + (long)o * y->cin + i] = acc;
                        }
                        if (y->bias) {
                            double acc = 0.0;
                            for (int n = 0; n < N; ++n) acc += fabs(dY[(long)n * y->cout + o]);
                            gscale[y->poff + (long)y->cout * y->cin + o] = acc;
                        }
                    }
                break;
            }
            }
        }
        if (gout && gl >= 0 && gl < nl) memcpy(gout, dact[gl], sizeof(double) * (size_t)numel(S[gl], N));
        for (int l = 0; l < nl; ++l) free(dact[l]);
    }
    for (int l = 0; l < nl; ++l) { free(act[l]); free(bmean[l]); free(brstd[l]); }
    free(act); free(dact); free(bmean); free(brstd); free(S); free(dZ);
    return 0;
}

int ref_forward_backward(const ref_layer* L, int nl, int N, int C, int H, int W,
                         const double* x, const double* images, const int* labels,
                         double bn_eps, double* logits, double* loss, double* grad) {
    return forward_backward_impl(L, nl, N, C, H, W, x, images, labels, bn_eps, logits, loss, grad, -1, NULL, NULL);
}

/* Condition scale of every parameter gradient (see conv_wscale), d doubles;
 * the gradient itself goes to grad. */
int ref_grad_scale(const ref_layer* L, int nl, int N, int C, int H, int W,
                   const double* x, const double* images, const int* labels,
                   double bn_eps, double* grad, double* scale) {
    double loss;
    return forward_backward_impl(L, nl, N, C, H, W, x, images, labels, bn_eps, NULL, &loss, grad, -1, NULL, scale);
}

/* Gradient of the loss with respect to the output of layer `layer` (NCHW),
 * from the full backward pass. */
int ref_activation_grad(const ref_layer* L, int nl, int N, int C, int H, int W,
                        const double* x, const double* images, const int* labels,
                        double bn_eps, int layer, double* out) {
    long d = ref_num_params(L, nl);
    double* g = (double*)malloc(sizeof(double) * (size_t)(d > 0 ? d : 1));
    double loss;
    int rc = forward_backward_impl(L, nl, N, C, H, W, x, images, labels, bn_eps, NULL, &loss, g, layer, out, NULL);
    free(g);
    return rc;
}

/* Shapes of every layer output (c,h,w triples), for the tests. */
int ref_shapes(const ref_layer* L, int nl, int C, int H, int W, int* chw) {
    shp img = { C, H, W };
    shp* S = (shp*)calloc((size_t)nl, sizeof(shp));
    if (!S) return -1;
    int rc = infer_shapes(L, nl, img, S);
    for (int l = 0; l < nl && rc == 0; ++l) { chw[3 * l] = S[l].c; chw[3 * l + 1] = S[l].h; chw[3 * l + 2] = S[l].w; }
    free(S);
    return rc;
}

/* ------------------------- the optimiser steps -------------------------- */

/*
 * Block update (Alg. 1, updater's last step; Sec. 5, operator -|_i):
 * for e in [lo, hi):  with momentum,  m[e] = mu*m[e] + g[e] + wd*x[e];
 *                                     x[e] -= lr * m[e]
 *                     without (m == NULL): x[e] -= lr * (g[e] + wd*x[e]).
 * Indices outside [lo, hi) are not touched.  Block i of the paper, covering
 * the 1-indexed entries b_{i-1}+1 .. b_i, is lo = b_{i-1}, hi = b_i here.
 */
void ref_block_update(double* x, double* m, const double* g, long lo, long hi,
                      double lr, double mu, double wd) {
    for (long e = lo; e < hi; ++e) {
        double dir = g[e] + wd * x[e];
        if (m) { m[e] = mu * m[e] + dir; dir = m[e]; }
        x[e] -= lr * dir;
    }
}

/*
 * Averaging round over n replicas (Alg. 1, averaging loop): each replica's
 * snapshot v_k = x_k; vbar = (sum over k ascending of v_k) / n;
 * x_k += vbar - v_k.
 */
void ref_average(double* const* reps, int n, long d) {
    double* v = (double*)malloc(sizeof(double) * (size_t)n);
    for (long e = 0; e < d; ++e) {
        double s = 0.0;
        for (int k = 0; k < n; ++k) { v[k] = reps[k][e]; s += v[k]; }
        double vbar = s / (double)n;
        for (int k = 0; k < n; ++k) reps[k][e] += vbar - v[k];
    }
    free(v);
}

/*
 * One updater iteration on replica x (Alg. 1, updater loop) in the
 * zero-delay (sequential) schedule: snapshot v = x; gradient of the minibatch
 * loss at v; block update of x over [lo, hi).  grad_out (d doubles) receives
 * the gradient restricted to the block (zero outside), loss_out the loss.
 */
int ref_step(const ref_layer* L, int nl, int N, int C, int H, int W,
             double* x, double* m, const double* images, const int* labels,
             long lo, long hi, double lr, double mu, double wd, double bn_eps,
             double* grad_out, double* loss_out, double* logits_out) {
    long d = ref_num_params(L, nl);
    double* v = (double*)malloc(sizeof(double) * (size_t)d);
    double* g = (double*)malloc(sizeof(double) * (size_t)d);
    memcpy(v, x, sizeof(double) * (size_t)d);
    int rc = ref_forward_backward(L, nl, N, C, H, W, v, images, labels, bn_eps, logits_out, loss_out, g);
    if (rc == 0) {
        for (long e = 0; e < d; ++e) if (e < lo || e >= hi) g[e] = 0.0;
        ref_block_update(x, m, g, lo, hi, lr, mu, wd);
        if (grad_out) memcpy(grad_out, g, sizeof(double) * (size_t)d);
    }
    free(v); free(g);
    return rc;
}

/* Forward only; copies the output of layer `layer` (NCHW) into out. */
int ref_activation(const ref_layer* L, int nl, int N, int C, int H, int W, const double* x,
                   const double* images, double bn_eps, int layer, double* out) {
    shp img = { C, H, W };
    shp* S = (shp*)calloc((size_t)nl, sizeof(shp));
    if (!S || infer_shapes(L, nl, img, S) || layer < 0 || layer >= nl) { free(S); return -1; }
    double** act = (double**)calloc((size_t)nl, sizeof(double*));
    double** bmean = (double**)calloc((size_t)nl, sizeof(double*));
    double** brstd = (double**)calloc((size_t)nl, sizeof(double*));
    for (int l = 0; l < nl; ++l) {
        act[l] = (double*)calloc((size_t)numel(S[l], N), sizeof(double));
        if (L[l].op == R_BN) {
            bmean[l] = (double*)calloc((size_t)S[l].c, sizeof(double));
            brstd[l] = (double*)calloc((size_t)S[l].c, sizeof(double));
        }
    }
    run_forward(L, nl, N, img, S, x, images, bn_eps, act, bmean, brstd);
    memcpy(out, act[layer], sizeof(double) * (size_t)numel(S[layer], N));
    for (int l = 0; l < nl; ++l) { free(act[l]); free(bmean[l]); free(brstd[l]); }
    free(act); free(bmean); free(brstd); free(S);
    return 0;
}

/*
 * How far the forward pass at x stays from the method's non-smooth points:
 * the smallest |input| / max|input| over the inputs of every ReLU (per
 * layer), and the smallest (largest - second largest) / max|input| over the
 * windows of every max pool.  A gradient comparison between two precisions
 * is well posed only when this exceeds the precisions' disagreement on
 * those inputs; otherwise both mask / argmax decisions are valid.
 */
int ref_kink_margin(const ref_layer* L, int nl, int N, int C, int H, int W, const double* x,
                    const double* images, double bn_eps, double* margin) {
    shp img = { C, H, W };
    shp* S = (shp*)calloc((size_t)nl, sizeof(shp));
    if (!S || infer_shapes(L, nl, img, S)) { free(S); return -1; }
    double** act = (double**)calloc((size_t)nl, sizeof(double*));
    double** bmean = (double**)calloc((size_t)nl, sizeof(double*));
    double** brstd = (double**)calloc((size_t)nl, sizeof(double*));
    for (int l = 0; l < nl; ++l) {
        act[l] = (double*)calloc((size_t)numel(S[l], N), sizeof(double));
        if (L[l].op == R_BN) {
            bmean[l] = (double*)calloc((size_t)S[l].c, sizeof(double));
            brstd[l] = (double*)calloc((size_t)S[l].c, sizeof(double));
        }
    }
    run_forward(L, nl, N, img, S, x, images, bn_eps, act, bmean, brstd);
    double best = INFINITY;
    for (int l = 0; l < nl; ++l) {
        if (L[l].op != R_RELU && L[l].op != R_MAXPOOL) continue;
        shp a = in_shape(S, L[l].in0, img);
        const double* X = L[l].in0 < 0 ? images : act[L[l].in0];
        long n = numel(a, N);
        double mx = 0.0;
        for (long i = 0; i < n; ++i) if (fabs(X[i]) > mx) mx = fabs(X[i]);
        if (mx == 0.0) continue;
        if (L[l].op == R_RELU) {
            for (long i = 0; i < n; ++i) if (fabs(X[i]) / mx < best) best = fabs(X[i]) / mx;
        } else {
            shp o = S[l];
            int R = L[l].k, st = L[l].stride, pad = L[l].pad;
            for (int b = 0; b < N; ++b)
                for (int c = 0; c < a.c; ++c)
                    for (int p = 0; p < o.h; ++p)
                        for (int q = 0; q < o.w; ++q) {
                            double t1 = -INFINITY, t2 = -INFINITY;
                            for (int r = 0; r < R; ++r)
                                for (int s2 = 0; s2 < R; ++s2) {
                                    int hi = p * st - pad + r, wi = q * st - pad + s2;
                                    if (hi < 0 || hi >= a.h || wi < 0 || wi >= a.w) continue;
                                    double v = X[(((long)b * a.c + c) * a.h + hi) * a.w + wi];
                                    if (v > t1) { t2 = t1; t1 = v; } else if (v > t2) t2 = v;
                                }
                            if (t2 > -INFINITY && (t1 - t2) / mx < best) best = (t1 - t2) / mx;
                        }
        }
    }
    *margin = best;
    for (int l = 0; l < nl; ++l) { free(act[l]); free(bmean[l]); free(brstd[l]); }
    free(act); free(bmean); free(brstd); free(S);
    return 0;
}
