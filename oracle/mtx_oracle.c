/*
 * CPU ORACLE for the data-parallel synchronous SGD step -- TEST INFRASTRUCTURE ONLY.
 *
 * This file is the plain, slow, obviously-correct reference that the GPU library is checked
 * against.  Only the test-suite, the smoke check and the CPU-baseline leg of the benchmark may
 * load it.  It shares no code, header, table or helper with the GPU library and it never calls
 * into it.
 *
 * What it computes (paper: "User-transparent Distributed TensorFlow", arXiv 1704.04560):
 *   - Sec. III-A / III-E: data parallelism with synchronous replicas.  The global batch B is
 *     split into R equal shards; every replica holds the same weights and computes the gradient
 *     of the mean loss of its own shard.
 *   - Sec. II-B and Sec. III-D.2 (MPI_Allreduce operator): the replicas' gradients are combined
 *     by an all-reduce "for averaging gradients", layer by layer in a fixed order, so the applied
 *     gradient is (1/R) * sum_r g_r, which equals the full-batch mean gradient.
 *   - Sec. III-D.2 and Sec. III-E: the result is equivalent to the sequential SGD step.  The
 *     optimizer is the momentum method the paper lists among TensorFlow's optimizers (Sec. I):
 *     v <- mu*v + g, w <- w - lr*v (TensorFlow 1.0 MomentumOptimizer form); mu == 0 is plain SGD.
 *     The two other update rules Sec. I names, AdaGrad and Adam, follow the averaged gradient in
 *     orc_average_adagrad / orc_average_adam, each as defined in the work the paper cites.
 *   - Sec. III-D.1 (Broadcast operator): replicas start identical.  Here every replica reads the
 *     one weight vector, which is that property by construction.
 *   - Fig. 1 (AlexNet: convolution + fully connected layers) and Sec. I (MLP / CNN): the layer
 *     types: fully connected, convolution (stride, zero padding, groups), max-pooling, ReLU, and a
 *     softmax cross-entropy loss (the paper trains 1000-class ImageNet classifiers, Table II).
 *   - Table II also lists ResNet-50 and InceptionV3, whose building blocks add two layer types:
 *     batch normalisation and the residual addition.  Batch normalisation (Ioffe and Szegedy)
 *     normalises every channel by the mean and the biased variance over the samples and
 *     positions of the replica's own shard (each replica sees only its shard, so these
 *     statistics are per shard), y = gamma * (x - mean) / sqrt(var + eps) + beta, eps = 1e-3
 *     (TensorFlow's default); its gradients follow from that definition by the chain rule.
 *     Because the statistics are per shard, the average of the replica gradients of a network
 *     with batch normalisation is not the full-batch gradient.  The residual addition sums the
 *     previous layer's output and the output of an earlier layer of the same shape (He et al.);
 *     its gradient reaches both.  Where the block changes the shape (ResNet-50's downsampling
 *     blocks), the shortcut is a projection: a 1x1 convolution of the given stride, with weights
 *     and bias, of the earlier layer's output (He et al., the projection shortcut); its output is
 *     a stored output like any convolution's, then added.
 *
 * The paper gives no formula for any of these; the code below is the textbook definition of
 * each, written as direct loops in double precision.  Readings taken where the paper is silent:
 *   - mean (not sum) reduction; shard loss = mean over the shard's samples;
 *   - momentum form v <- mu*v + g, w <- w - lr*v with v0 = 0; no weight decay, no Nesterov;
 *   - relu'(0) = 0; max-pool ties resolve to the first maximal element in row-major window
 *     order; pooling windows are "valid" (no padding);
 *   - Glorot-uniform weights U(-a, a), a = sqrt(6 / (fan_in + fan_out)), biases zero, drawn from
 *     a counter-based generator (first output of SplitMix64 seeded with seed ^ (layer << 32 | i));
 *   - storage precision: in "fp32" mode every stored tensor (activations, gradients) is rounded
 *     to float; in "bf16" mode the input, the weights used by the layers, every hidden-layer
 *     output, the loss gradient and every data-gradient are rounded to bfloat16 (round to nearest
 *     even) while logits, weight/bias gradients, averages and the update stay float.  All sums
 *     are carried out in double.  An "exact" mode rounds nothing before the float outputs; it
 *     exists so that the oracle itself can be pinned against finite differences and against
 *     double-precision autograd.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC mtx_oracle.c -lm (OpenMP only parallelises over
 * independent outputs; every individual sum is a sequential loop, so results do not depend on
 * the thread count).
 */
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_FC 0
#define ORC_CONV 1
#define ORC_MAXPOOL 2
#define ORC_BN 3  /* batch normalisation: params gamma[c] (as W) and beta[c] (as b) */
#define ORC_ADD 4 /* residual addition: k = index of the earlier layer whose output is added */
#define ORC_ADDP 5 /* residual addition through a projection: k = the earlier layer, whose output
                    * passes a 1x1 convolution of the given stride (weights W[out][c], bias b)
                    * before it is added */

#define ORC_BN_EPS 1e-3

#define ORC_OK 0
#define ORC_EINVAL -1
#define ORC_ENOMEM -2
#define ORC_EHINT -6 /* a decision hint lies outside the oracle's own error bound */

/* storage precision of the training step */
#define ORC_PREC_F32 0   /* every stored tensor rounded to float */
#define ORC_PREC_BF16 1  /* bfloat16 storage at the documented points, float elsewhere */
#define ORC_PREC_EXACT 2 /* nothing rounded until the float outputs (used to pin the oracle) */

typedef struct {
    int kind, out, k, stride, pad, groups, relu;
} orc_layer;

typedef struct {
    int kind, relu;
    int c, h, w;    /* input shape (per sample) */
    int oc, oh, ow; /* output shape (per sample) */
    int k, s, p, g;
    long w_off, w_len, b_off, b_len; /* offsets into the flat parameter vector */
} orc_geom;

/* ------------------------------------------------------------------------------------------ */
/* rounding                                                                                   */
/* ------------------------------------------------------------------------------------------ */

static double rnd_f32(double x) { return (double)(float)x; }
static double rnd_none(double x) { return x; }

/* Round a value to bfloat16 the way an fp32 accumulator is stored: first to float, then keep the
 * top 16 bits with round-to-nearest-even on the discarded half. */
static double rnd_bf16(double x)
{
    float f = (float)x;
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) { /* NaN stays NaN */
        u |= 0x00400000u;
        u &= 0xffff0000u;
    } else {
        u = (u + 0x7fffu + ((u >> 16) & 1u)) & 0xffff0000u;
    }
    memcpy(&f, &u, 4);
    return (double)f;
}

float orc_round_bf16(float x) { return (float)rnd_bf16((double)x); }

/* Number of threads the oracle's parallel loops use. */
int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------------------------ */
/* geometry                                                                                   */
/* ------------------------------------------------------------------------------------------ */

int orc_plan(int in_c, int in_h, int in_w, int n_layers, const orc_layer* L, orc_geom* G,
             long* n_params)
{
    int c = in_c, h = in_h, w = in_w;
    long off = 0;
    if (in_c < 1 || in_h < 1 || in_w < 1 || n_layers < 1 || !L) return ORC_EINVAL;
    for (int i = 0; i < n_layers; i++) {
        orc_geom* g = &G[i];
        memset(g, 0, sizeof *g);
        g->kind = L[i].kind;
        g->relu = L[i].relu ? 1 : 0;
        g->c = c; g->h = h; g->w = w;
        if (L[i].kind == ORC_CONV) {
            g->k = L[i].k; g->s = L[i].stride; g->p = L[i].pad; g->g = L[i].groups;
            if (g->k < 1 || g->s < 1 || g->p < 0 || g->g < 1 || L[i].out < 1) return ORC_EINVAL;
            if (c % g->g || L[i].out % g->g) return ORC_EINVAL;
            g->oc = L[i].out;
            g->oh = (h + 2 * g->p - g->k) / g->s + 1;
            g->ow = (w + 2 * g->p - g->k) / g->s + 1;
            if (h + 2 * g->p < g->k || w + 2 * g->p < g->k) return ORC_EINVAL;
            g->w_len = (long)g->oc * (c / g->g) * g->k * g->k;
            g->b_len = g->oc;
        } else if (L[i].kind == ORC_FC) {
            if (L[i].out < 1) return ORC_EINVAL;
            g->k = 1; g->s = 1; g->p = 0; g->g = 1;
            g->oc = L[i].out; g->oh = 1; g->ow = 1;
            g->w_len = (long)g->oc * c * h * w;
            g->b_len = g->oc;
        } else if (L[i].kind == ORC_MAXPOOL) {
            g->k = L[i].k; g->s = L[i].stride; g->p = 0; g->g = 1;
            if (g->k < 1 || g->s < 1 || h < g->k || w < g->k || g->k > 16) return ORC_EINVAL;
            if (g->relu) return ORC_EINVAL;
            g->oc = c;
            g->oh = (h - g->k) / g->s + 1;
            g->ow = (w - g->k) / g->s + 1;
        } else if (L[i].kind == ORC_BN) {
            if (L[i].out != 0 && L[i].out != c) return ORC_EINVAL;
            g->k = 1; g->s = 1; g->p = 0; g->g = 1;
            g->oc = c; g->oh = h; g->ow = w;
            g->w_len = c;
            g->b_len = c;
        } else if (L[i].kind == ORC_ADD || L[i].kind == ORC_ADDP) {
            /* the source is an earlier layer (not the previous one), of this layer's input shape
             * (plain addition) or of a shape that a 1x1 convolution of the given stride maps to
             * it (projection, out = this layer's channel count); no layer is the source of two
             * additions */
            int src = L[i].k;
            if (src < 0 || src > i - 2) return ORC_EINVAL;
            for (int j = src + 1; j < i; j++)
                if ((G[j].kind == ORC_ADD || G[j].kind == ORC_ADDP) && G[j].k == src)
                    return ORC_EINVAL;
            if (L[i].kind == ORC_ADD) {
                if (G[src].oc != c || G[src].oh != h || G[src].ow != w) return ORC_EINVAL;
                g->s = 1;
            } else {
                const int s = L[i].stride;
                if (s < 1 || L[i].out != c || L[i].pad != 0 || (L[i].groups != 0 && L[i].groups != 1))
                    return ORC_EINVAL;
                if ((G[src].oh - 1) / s + 1 != h || (G[src].ow - 1) / s + 1 != w) return ORC_EINVAL;
                g->s = s;
                g->w_len = (long)c * G[src].oc; /* W[out][c_src] */
                g->b_len = c;
            }
            g->k = src; g->p = 0; g->g = 1;
            g->oc = c; g->oh = h; g->ow = w;
        } else {
            return ORC_EINVAL;
        }
        g->w_off = off; off += g->w_len;
        g->b_off = off; off += g->b_len;
        c = g->oc; h = g->oh; w = g->ow;
    }
    /* the network ends in a fully connected layer that produces the class scores */
    if (L[n_layers - 1].kind != ORC_FC || L[n_layers - 1].relu) return ORC_EINVAL;
    if (n_params) *n_params = off;
    return ORC_OK;
}

int orc_param_count(int in_c, int in_h, int in_w, int n_layers, const orc_layer* L, long* n)
{
    orc_geom* G = (orc_geom*)calloc((size_t)n_layers, sizeof(orc_geom));
    if (!G) return ORC_ENOMEM;
    int rc = orc_plan(in_c, in_h, in_w, n_layers, L, G, n);
    free(G);
    return rc;
}

/* ------------------------------------------------------------------------------------------ */
/* layers in double precision (textbook definitions)                                          */
/* ------------------------------------------------------------------------------------------ */

/* Convolution, NCHW, weights [oc][c/g][k][k], zero padding p, stride s, g groups.
 * y[n][o][i][j] = b[o] + sum_{c' , u, v} W[o][c'][u][v] * x[n][grp*c/g + c'][i*s - p + u][j*s - p + v]
 * Every output's sum is taken in ascending (c', u, v) order over the taps inside the image; a
 * whole output row is carried along at once (one running sum per column). */
void orc_conv_fwd(int N, int C, int H, int W, int OC, int K, int S, int P, int Gr,
                  const double* x, const double* w, const double* b, double* y)
{
    int OH = (H + 2 * P - K) / S + 1, OW = (W + 2 * P - K) / S + 1;
    int cg = C / Gr, og = OC / Gr;
#pragma omp parallel
    {
        double* row = (double*)malloc(sizeof(double) * (size_t)OW);
#pragma omp for collapse(2) schedule(static)
        for (int n = 0; n < N; n++)
            for (int o = 0; o < OC; o++) {
                if (!row) continue;
                int grp = o / og;
                for (int i = 0; i < OH; i++) {
                    for (int j = 0; j < OW; j++) row[j] = b ? b[o] : 0.0;
                    for (int cc = 0; cc < cg; cc++)
                        for (int u = 0; u < K; u++) {
                            int hi = i * S - P + u;
                            if (hi < 0 || hi >= H) continue;
                            const double* xr = x + (((long)n * C + grp * cg + cc) * H + hi) * W;
                            for (int v = 0; v < K; v++) {
                                const double wv = w[(((long)o * cg + cc) * K + u) * K + v];
                                /* columns j whose tap j*S - P + v lies inside the row */
                                int j0 = P - v > 0 ? (P - v + S - 1) / S : 0;
                                int j1 = (W - 1 + P - v) >= 0 ? (W - 1 + P - v) / S + 1 : 0;
                                if (j1 > OW) j1 = OW;
                                for (int j = j0; j < j1; j++) row[j] += wv * xr[j * S - P + v];
                            }
                        }
                    for (int j = 0; j < OW; j++) y[(((long)n * OC + o) * OH + i) * OW + j] = row[j];
                }
            }
        free(row);
    }
}

/* Gradients of the convolution: dW = sum over samples and output positions of dy times the
 * input patch, db = sum of dy, dx = adjoint of the forward index map (dx may be NULL).
 * dW[o][c'][u][v] sums over (n, i, j) in ascending order (the K sums of one kernel row are
 * carried along together); dx[n][c][h][w] gathers sum_{o in the group, i, j} dy[n][o][i][j] *
 * W[o][c'][h - i*s + p][w - j*s + p] in ascending (o, i, j) order over the taps that exist. */
void orc_conv_bwd(int N, int C, int H, int W, int OC, int K, int S, int P, int Gr,
                  const double* x, const double* w, const double* dy, double* dx, double* dw,
                  double* db)
{
    int OH = (H + 2 * P - K) / S + 1, OW = (W + 2 * P - K) / S + 1;
    int cg = C / Gr, og = OC / Gr;
#pragma omp parallel
    {
        double* acc = (double*)malloc(sizeof(double) * (size_t)K);
#pragma omp for schedule(static)
        for (int o = 0; o < OC; o++) {
            if (!acc) continue;
            int grp = o / og;
            double sb = 0.0;
            for (int n = 0; n < N; n++)
                for (int i = 0; i < OH; i++)
                    for (int j = 0; j < OW; j++) sb += dy[(((long)n * OC + o) * OH + i) * OW + j];
            if (db) db[o] = sb;
            for (int cc = 0; cc < cg; cc++)
                for (int u = 0; u < K; u++) {
                    for (int v = 0; v < K; v++) acc[v] = 0.0;
                    for (int n = 0; n < N; n++)
                        for (int i = 0; i < OH; i++) {
                            int hi = i * S - P + u;
                            if (hi < 0 || hi >= H) continue;
                            const double* dyr = dy + (((long)n * OC + o) * OH + i) * OW;
                            const double* xr = x + (((long)n * C + grp * cg + cc) * H + hi) * W;
                            for (int j = 0; j < OW; j++) {
                                const double d = dyr[j];
                                for (int v = 0; v < K; v++) {
                                    int wi = j * S - P + v;
                                    if (wi < 0 || wi >= W) continue;
                                    acc[v] += d * xr[wi];
                                }
                            }
                        }
                    for (int v = 0; v < K; v++) dw[(((long)o * cg + cc) * K + u) * K + v] = acc[v];
                }
        }
        free(acc);
    }
    if (!dx) return;
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; n++)
        for (int c = 0; c < C; c++) {
            int grp = c / cg, cc = c % cg;
            for (int hi = 0; hi < H; hi++)
                for (int wi = 0; wi < W; wi++) {
                    /* outputs whose window covers (hi, wi): u = hi + p - i*s in [0, K) */
                    int i0 = hi + P - K + 1 > 0 ? (hi + P - K + 1 + S - 1) / S : 0;
                    int i1 = (hi + P) / S + 1;
                    int j0 = wi + P - K + 1 > 0 ? (wi + P - K + 1 + S - 1) / S : 0;
                    int j1 = (wi + P) / S + 1;
                    if (i1 > OH) i1 = OH;
                    if (j1 > OW) j1 = OW;
                    double a = 0.0;
                    for (int o = grp * og; o < (grp + 1) * og; o++)
                        for (int i = i0; i < i1; i++) {
                            int u = hi + P - i * S;
                            for (int j = j0; j < j1; j++) {
                                int v = wi + P - j * S;
                                a += dy[(((long)n * OC + o) * OH + i) * OW + j] *
                                     w[(((long)o * cg + cc) * K + u) * K + v];
                            }
                        }
                    dx[(((long)n * C + c) * H + hi) * W + wi] = a;
                }
        }
}

/* Fully connected: y[n][o] = b[o] + sum_i W[o][i] x[n][i], W stored [out][in]. */
void orc_fc_fwd(int N, int IN, int OUT, const double* x, const double* w, const double* b,
                double* y)
{
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; n++)
        for (int o = 0; o < OUT; o++) {
            double acc = b ? b[o] : 0.0;
            for (int i = 0; i < IN; i++) acc += w[(long)o * IN + i] * x[(long)n * IN + i];
            y[(long)n * OUT + o] = acc;
        }
}

/* dW[o][i] = sum_n dy[n][o] x[n][i]; db[o] = sum_n dy[n][o]; dx[n][i] = sum_o dy[n][o] W[o][i].
 * Each sum runs in ascending order of its index (n, resp. o); a whole row of dW (resp. a chunk of
 * a row of dx) is carried along at once. */
void orc_fc_bwd(int N, int IN, int OUT, const double* x, const double* w, const double* dy,
                double* dx, double* dw, double* db)
{
#pragma omp parallel for schedule(static)
    for (int o = 0; o < OUT; o++) {
        double sb = 0.0;
        for (int n = 0; n < N; n++) sb += dy[(long)n * OUT + o];
        if (db) db[o] = sb;
        double* dwo = dw + (long)o * IN;
        for (int i = 0; i < IN; i++) dwo[i] = 0.0;
        for (int n = 0; n < N; n++) {
            const double d = dy[(long)n * OUT + o];
            const double* xn = x + (long)n * IN;
            for (int i = 0; i < IN; i++) dwo[i] += d * xn[i];
        }
    }
    if (!dx) return;
    const int CH = 256, nch = (IN + CH - 1) / CH;
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; n++)
        for (int ch = 0; ch < nch; ch++) {
            const int i0 = ch * CH, i1 = i0 + CH < IN ? i0 + CH : IN;
            double* dxn = dx + (long)n * IN;
            for (int i = i0; i < i1; i++) dxn[i] = 0.0;
            for (int o = 0; o < OUT; o++) {
                const double d = dy[(long)n * OUT + o];
                const double* wo = w + (long)o * IN;
                for (int i = i0; i < i1; i++) dxn[i] += d * wo[i];
            }
        }
}

/* Max-pooling over valid K x K windows with stride S.  argmax = u*K + v of the first maximal
 * element in row-major window order (strict '>' keeps the earliest). */
void orc_maxpool_fwd(int N, int C, int H, int W, int K, int S, const double* x, double* y,
                     int32_t* argmax)
{
    int OH = (H - K) / S + 1, OW = (W - K) / S + 1;
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; n++)
        for (int c = 0; c < C; c++)
            for (int i = 0; i < OH; i++)
                for (int j = 0; j < OW; j++) {
                    const double* xp = x + ((long)n * C + c) * H * W;
                    double best = xp[(long)(i * S) * W + j * S];
                    int bi = 0;
                    for (int u = 0; u < K; u++)
                        for (int v = 0; v < K; v++) {
                            double t = xp[(long)(i * S + u) * W + j * S + v];
                            if (t > best) { best = t; bi = u * K + v; }
                        }
                    long o = (((long)n * C + c) * OH + i) * OW + j;
                    y[o] = best;
                    argmax[o] = bi;
                }
}

/* dx[argmax position] += dy (windows may overlap when S < K). */
void orc_maxpool_bwd(int N, int C, int H, int W, int K, int S, const int32_t* argmax,
                     const double* dy, double* dx)
{
    int OH = (H - K) / S + 1, OW = (W - K) / S + 1;
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; n++)
        for (int c = 0; c < C; c++) {
            double* dxp = dx + ((long)n * C + c) * H * W;
            for (long t = 0; t < (long)H * W; t++) dxp[t] = 0.0;
            for (int i = 0; i < OH; i++)
                for (int j = 0; j < OW; j++) {
                    long o = (((long)n * C + c) * OH + i) * OW + j;
                    int u = argmax[o] / K, v = argmax[o] % K;
                    dxp[(long)(i * S + u) * W + j * S + v] += dy[o];
                }
        }
}

/* Batch normalisation of one shard, NCHW with N samples: for every channel the mean and the
 * biased variance over (n, h, w), inv = 1 / sqrt(var + eps), y = gamma (x - mean) inv + beta.
 * mean and inv are returned for the backward pass. */
void orc_bn_fwd(int N, int C, int HW, const double* x, const double* gamma, const double* beta,
                double* y, double* mean, double* inv)
{
    const double M = (double)N * HW;
#pragma omp parallel for schedule(static)
    for (int c = 0; c < C; c++) {
        double s = 0.0;
        for (int n = 0; n < N; n++)
            for (int t = 0; t < HW; t++) s += x[((long)n * C + c) * HW + t];
        const double m = s / M;
        double v = 0.0;
        for (int n = 0; n < N; n++)
            for (int t = 0; t < HW; t++) {
                const double d = x[((long)n * C + c) * HW + t] - m;
                v += d * d;
            }
        const double iv = 1.0 / sqrt(v / M + ORC_BN_EPS);
        mean[c] = m;
        inv[c] = iv;
        for (int n = 0; n < N; n++)
            for (int t = 0; t < HW; t++) {
                const long o = ((long)n * C + c) * HW + t;
                y[o] = gamma[c] * (x[o] - m) * iv + beta[c];
            }
    }
}

/* Gradients of batch normalisation with the statistics of the same shard (the chain rule through
 * mean and variance): with xhat = (x - mean) inv and M = N*H*W,
 * dgamma = sum dy xhat, dbeta = sum dy, dx = gamma inv (dy - dbeta / M - xhat dgamma / M). */
void orc_bn_bwd(int N, int C, int HW, const double* x, const double* gamma, const double* mean,
                const double* inv, const double* dy, double* dx, double* dgamma, double* dbeta)
{
    const double M = (double)N * HW;
#pragma omp parallel for schedule(static)
    for (int c = 0; c < C; c++) {
        double sd = 0.0, sdx = 0.0;
        for (int n = 0; n < N; n++)
            for (int t = 0; t < HW; t++) {
                const long o = ((long)n * C + c) * HW + t;
                sd += dy[o];
                sdx += dy[o] * (x[o] - mean[c]) * inv[c];
            }
        dgamma[c] = sdx;
        dbeta[c] = sd;
        if (!dx) continue;
        for (int n = 0; n < N; n++)
            for (int t = 0; t < HW; t++) {
                const long o = ((long)n * C + c) * HW + t;
                const double xh = (x[o] - mean[c]) * inv[c];
                dx[o] = gamma[c] * inv[c] * (dy[o] - sd / M - xh * sdx / M);
            }
    }
}

/* Softmax cross-entropy per sample: loss[n] = logsumexp(z[n]) - z[n][y[n]];
 * dz[n][c] = (softmax(z[n])[c] - [c == y[n]]) * scale.  logsumexp subtracts the row maximum. */
void orc_softmax_xent(int N, int NC, const double* z, const int32_t* y, double scale,
                      double* loss, double* dz)
{
    for (int n = 0; n < N; n++) {
        const double* zn = z + (long)n * NC;
        double m = zn[0];
        for (int c = 1; c < NC; c++)
            if (zn[c] > m) m = zn[c];
        double s = 0.0;
        for (int c = 0; c < NC; c++) s += exp(zn[c] - m);
        double lse = m + log(s);
        int yn = y[n];
        loss[n] = (yn >= 0 && yn < NC) ? lse - zn[yn] : NAN;
        if (dz)
            for (int c = 0; c < NC; c++)
                dz[(long)n * NC + c] = (exp(zn[c] - lse) - (c == yn ? 1.0 : 0.0)) * scale;
    }
}

/* ------------------------------------------------------------------------------------------ */
/* weight initialisation                                                                      */
/* ------------------------------------------------------------------------------------------ */

/* First output of a SplitMix64 generator whose state is `key` (Steele, Lea & Flood, OOPSLA 2014;
 * constants of Vigna's public-domain splitmix64.c). */
static uint64_t splitmix64_first(uint64_t key)
{
    uint64_t z = key + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* The generator on its own, for checking it against the published reference outputs. */
uint64_t orc_splitmix64_first(uint64_t key) { return splitmix64_first(key); }

int orc_init_glorot(int in_c, int in_h, int in_w, int n_layers, const orc_layer* L,
                    uint64_t seed, float* w)
{
    orc_geom* G = (orc_geom*)calloc((size_t)n_layers, sizeof(orc_geom));
    long P;
    if (!G) return ORC_ENOMEM;
    int rc = orc_plan(in_c, in_h, in_w, n_layers, L, G, &P);
    if (rc) { free(G); return rc; }
    for (int l = 0; l < n_layers; l++) {
        orc_geom* g = &G[l];
        if (g->kind == ORC_MAXPOOL || g->kind == ORC_ADD) continue;
        if (g->kind == ORC_BN) { /* gamma = 1, beta = 0: the identity at the start */
            for (long i = 0; i < g->w_len; i++) w[g->w_off + i] = 1.0f;
            for (long i = 0; i < g->b_len; i++) w[g->b_off + i] = 0.0f;
            continue;
        }
        double fan_in, fan_out;
        if (g->kind == ORC_CONV) {
            fan_in = (double)(g->c / g->g) * g->k * g->k;
            fan_out = (double)g->oc * g->k * g->k;
        } else if (g->kind == ORC_ADDP) { /* a 1x1 convolution of the source's channels */
            fan_in = (double)G[g->k].oc;
            fan_out = (double)g->oc;
        } else {
            fan_in = (double)g->c * g->h * g->w;
            fan_out = (double)g->oc;
        }
        double a = sqrt(6.0 / (fan_in + fan_out));
        for (long i = 0; i < g->w_len; i++) {
            uint64_t hsh = splitmix64_first(seed ^ (((uint64_t)l << 32) | (uint64_t)i));
            double u = (double)(hsh >> 40) / 16777216.0;
            w[g->w_off + i] = (float)(a * (2.0 * u - 1.0));
        }
        for (long i = 0; i < g->b_len; i++) w[g->b_off + i] = 0.0f;
    }
    free(G);
    return ORC_OK;
}

/* ------------------------------------------------------------------------------------------ */
/* the training step                                                                           */
/* ------------------------------------------------------------------------------------------ */

static long act_size(const orc_geom* g) { return (long)g->oc * g->oh * g->ow; }

/* gamma(n) of the standard floating-point summation error bound for unit roundoff 2^-24. */
static double gamma_f32(long n)
{
    double nu = (double)n * ldexp(1.0, -24);
    return nu / (1.0 - nu);
}

static void layer_fwd(const orc_geom* g, int N, const double* a, const double* w, const double* b,
                      double* z)
{
    if (g->kind == ORC_CONV)
        orc_conv_fwd(N, g->c, g->h, g->w, g->oc, g->k, g->s, g->p, g->g, a, w, b, z);
    else
        orc_fc_fwd(N, g->c * g->h * g->w, g->oc, a, w, b, z);
}

/* One synchronous data-parallel SGD/momentum step.  See the file header for the method.
 *   x [R*Nb][C][H][W], labels [R*Nb], w and v [P] (v may be NULL iff mu == 0).
 *   Outputs: loss (mean over the batch), optional per-shard losses, optional per-shard gradients
 *   grads[r*P + i], the averaged gradient gavg [P], optional updated w_new / v_new, optional
 *   stored activations of every layer for the whole batch (concatenated in layer order), the
 *   max-pool decisions (int32 window index, concatenated over pool layers) and the ReLU
 *   decisions (int8, concatenated over ReLU layers).
 *   pool_hint / relu_hint (optional, same layout, -1 = no hint) replace a decision by another one
 *   only where both are plausible outcomes of a float evaluation of the forward pass; any other
 *   hint makes the call fail with ORC_EHINT.  A hint is admitted when the gap it has to bridge
 *   is within BOTH of these limits:
 *     (1) the rigorous forward error bound of a float evaluation (propagated layer by layer);
 *     (2) a window that does not grow with depth: hint_rel times the scale of the layer's own
 *         values in this shard.  For a pooling window the gap is (oracle's maximum - hinted
 *         element) and the window is 2 * hint_rel * max|pool input| (each of the two elements
 *         may be off by hint_rel * max in an evaluation whose stored outputs agree with the
 *         oracle's to hint_rel of the tensor's maximum); for a ReLU the gap is |pre-activation|
 *         and the window is hint_rel * max(pre-activation, 0) (the layer's largest output).
 *   hint_rel must be positive when hints are given: it is the per-tensor tolerance to which the
 *   caller compares stored outputs, so a decision outside the window would also show up there. */
int orc_train_step(int in_c, int in_h, int in_w, int n_layers, const orc_layer* L, int R, int Nb,
                   int prec, const float* x, const int32_t* labels, const float* w,
                   const float* v, float lr, float mu, const int32_t* pool_hint,
                   const int8_t* relu_hint, double hint_rel, double* loss_out, float* shard_loss,
                   float* grads,
                   float* gavg, float* w_new, float* v_new, float* acts, int32_t* pool_argmax,
                   int8_t* relu_mask)
{
    if (R < 1 || Nb < 1 || !x || !labels || !w || !gavg || (!v && mu != 0.0f)) return ORC_EINVAL;
    orc_geom* G = (orc_geom*)calloc((size_t)n_layers, sizeof(orc_geom));
    if (!G) return ORC_ENOMEM;
    long P;
    int rc = orc_plan(in_c, in_h, in_w, n_layers, L, G, &P);
    if (rc) { free(G); return rc; }
    const int B = R * Nb;
    const long in_sz = (long)in_c * in_h * in_w;
    const int track = (pool_hint || relu_hint) ? 1 : 0; /* error bounds needed for hints */
    if (track && !(hint_rel > 0.0 && hint_rel < 1.0)) { free(G); return ORC_EINVAL; }
    if (prec < ORC_PREC_F32 || prec > ORC_PREC_EXACT) { free(G); return ORC_EINVAL; }
    const int bf16 = (prec == ORC_PREC_BF16);
    /* storage rounding of activations and data-gradients; final-layer outputs use `store32` */
    double (*store)(double) = bf16 ? rnd_bf16 : (prec == ORC_PREC_EXACT ? rnd_none : rnd_f32);
    double (*store32)(double) = (prec == ORC_PREC_EXACT) ? rnd_none : rnd_f32;

    /* per-layer offsets of the concatenated whole-batch output arrays */
    long* act_off = (long*)calloc((size_t)n_layers + 1, sizeof(long));
    long* pool_off = (long*)calloc((size_t)n_layers + 1, sizeof(long));
    long* relu_off = (long*)calloc((size_t)n_layers + 1, sizeof(long));
    double* wq = (double*)malloc(sizeof(double) * (size_t)P);
    double* wabs = track ? (double*)malloc(sizeof(double) * (size_t)P) : NULL;
    double* gsum = (double*)calloc((size_t)P, sizeof(double));
    double** a = (double**)calloc((size_t)n_layers + 1, sizeof(double*));  /* stored outputs */
    double** e = (double**)calloc((size_t)n_layers + 1, sizeof(double*));  /* error bounds */
    double** z = (double**)calloc((size_t)n_layers, sizeof(double*));      /* pre-activations */
    int32_t** am = (int32_t**)calloc((size_t)n_layers, sizeof(int32_t*));  /* pool argmax */
    double** bnm = (double**)calloc((size_t)n_layers, sizeof(double*));    /* BN mean */
    double** bni = (double**)calloc((size_t)n_layers, sizeof(double*));    /* BN 1/std */
    double** skipg = (double**)calloc((size_t)n_layers, sizeof(double*));  /* residual grads */
    double** proj = (double**)calloc((size_t)n_layers, sizeof(double*));   /* projection outputs */
    double* lossn = (double*)malloc(sizeof(double) * (size_t)Nb);
    double* dbuf = NULL;
    double* dbuf2 = NULL;
    double* gw = (double*)malloc(sizeof(double) * (size_t)P);
    if (!act_off || !pool_off || !relu_off || !wq || (track && !wabs) || !gsum || !a || !e || !z ||
        !am || !bnm || !bni || !skipg || !proj || !lossn || !gw) {
        rc = ORC_ENOMEM;
        goto done;
    }
    {
        long ao = 0, po = 0, ro = 0, maxact = in_sz;
        for (int l = 0; l < n_layers; l++) {
            act_off[l] = ao; ao += act_size(&G[l]) * B;
            pool_off[l] = po; if (G[l].kind == ORC_MAXPOOL) po += act_size(&G[l]) * B;
            relu_off[l] = ro; if (G[l].relu) ro += act_size(&G[l]) * B;
            if (act_size(&G[l]) > maxact) maxact = act_size(&G[l]);
        }
        a[0] = (double*)malloc(sizeof(double) * (size_t)(in_sz * Nb));
        e[0] = (double*)calloc((size_t)(in_sz * Nb), sizeof(double));
        for (int l = 0; l < n_layers; l++) {
            long sz = act_size(&G[l]) * Nb;
            a[l + 1] = (double*)malloc(sizeof(double) * (size_t)sz);
            z[l] = (double*)malloc(sizeof(double) * (size_t)sz);
            if (track) e[l + 1] = (double*)calloc((size_t)sz, sizeof(double));
            if (G[l].kind == ORC_MAXPOOL) am[l] = (int32_t*)malloc(sizeof(int32_t) * (size_t)sz);
            if (G[l].kind == ORC_BN) {
                bnm[l] = (double*)malloc(sizeof(double) * (size_t)G[l].c);
                bni[l] = (double*)malloc(sizeof(double) * (size_t)G[l].c);
            }
            if (G[l].kind == ORC_ADD || G[l].kind == ORC_ADDP) {
                const int src = G[l].k;
                skipg[src] = (double*)malloc(sizeof(double) * (size_t)(act_size(&G[src]) * Nb));
                if (!skipg[src]) { rc = ORC_ENOMEM; goto done; }
            }
            if (G[l].kind == ORC_ADDP) {
                proj[l] = (double*)malloc(sizeof(double) * (size_t)sz);
                if (!proj[l]) { rc = ORC_ENOMEM; goto done; }
            }
            if (!a[l + 1] || !z[l] || (track && !e[l + 1]) ||
                (G[l].kind == ORC_MAXPOOL && !am[l]) ||
                (G[l].kind == ORC_BN && (!bnm[l] || !bni[l]))) {
                rc = ORC_ENOMEM;
                goto done;
            }
        }
        dbuf = (double*)malloc(sizeof(double) * (size_t)(maxact * Nb));
        dbuf2 = (double*)malloc(sizeof(double) * (size_t)(maxact * Nb));
        if (!a[0] || !e[0] || !dbuf || !dbuf2) { rc = ORC_ENOMEM; goto done; }
    }

    /* weights as the layers use them: the float master weights, or their bfloat16 rounding */
    for (long i = 0; i < P; i++) {
        wq[i] = bf16 ? rnd_bf16((double)w[i]) : (double)w[i];
        if (track) wabs[i] = fabs(wq[i]);
    }
    /* biases are added in float by both sides; they are never rounded to bfloat16, and
     * neither are the batch-normalisation scales (elementwise float arithmetic, no product) */
    for (int l = 0; l < n_layers; l++) {
        for (long i = 0; i < G[l].b_len; i++) {
            wq[G[l].b_off + i] = (double)w[G[l].b_off + i];
            if (track) wabs[G[l].b_off + i] = fabs((double)w[G[l].b_off + i]);
        }
        if (G[l].kind == ORC_BN)
            for (long i = 0; i < G[l].w_len; i++) {
                wq[G[l].w_off + i] = (double)w[G[l].w_off + i];
                if (track) wabs[G[l].w_off + i] = fabs((double)w[G[l].w_off + i]);
            }
    }

    double loss_total = 0.0;
    for (int r = 0; r < R; r++) {
        /* ---- forward on shard r (rows r*Nb .. r*Nb+Nb-1 of the batch) ---- */
        for (long t = 0; t < in_sz * Nb; t++) a[0][t] = store((double)x[(long)r * Nb * in_sz + t]);
        for (int l = 0; l < n_layers; l++) {
            const orc_geom* g = &G[l];
            long sz = act_size(g) * Nb;
            const int last = (l == n_layers - 1);
            if (g->kind == ORC_MAXPOOL) {
                orc_maxpool_fwd(Nb, g->c, g->h, g->w, g->k, g->s, a[l], a[l + 1], am[l]);
                if (track)
                    for (long t = 0; t < sz; t++) {
                        /* bound of a window maximum: the largest bound inside the window */
                        long per = (long)g->oh * g->ow;
                        long nc = t / per, ij = t % per;
                        int i = (int)(ij / g->ow), j = (int)(ij % g->ow);
                        double m = 0.0;
                        for (int u = 0; u < g->k; u++)
                            for (int vv = 0; vv < g->k; vv++) {
                                double ev = e[l][nc * g->h * g->w + (long)(i * g->s + u) * g->w +
                                                 j * g->s + vv];
                                if (ev > m) m = ev;
                            }
                        e[l + 1][t] = m;
                    }
                if (pool_hint) {
                    const int32_t* hint = pool_hint + pool_off[l] + (long)r * sz;
                    long per = (long)g->oh * g->ow;
                    const long insz = (long)g->c * g->h * g->w * Nb;
                    double scale = 0.0; /* largest magnitude of this shard's pool input */
                    for (long t = 0; t < insz; t++)
                        if (fabs(a[l][t]) > scale) scale = fabs(a[l][t]);
                    const double window = 2.0 * hint_rel * scale;
                    for (long t = 0; t < sz; t++) {
                        int hv = hint[t];
                        if (hv < 0 || hv == am[l][t]) continue;
                        if (hv >= g->k * g->k) { rc = ORC_EHINT; goto done; }
                        long nc = t / per, ij = t % per;
                        int i = (int)(ij / g->ow), j = (int)(ij % g->ow);
                        int own = am[l][t];
                        long base = nc * g->h * g->w + (long)(i * g->s) * g->w + j * g->s;
                        long po = base + (long)(own / g->k) * g->w + own % g->k;
                        long ph = base + (long)(hv / g->k) * g->w + hv % g->k;
                        double lim = e[l][po] + e[l][ph];
                        if (window < lim) lim = window;
                        if (a[l][po] - a[l][ph] > lim) { rc = ORC_EHINT; goto done; }
                        am[l][t] = hv;
                        a[l + 1][t] = a[l][ph];
                    }
                }
            } else {
                const double us = ldexp(1.0, -24) + (bf16 && !last ? ldexp(1.0, -8) : ldexp(1.0, -24));
                if (g->kind == ORC_BN) {
                    const int HW = g->h * g->w;
                    orc_bn_fwd(Nb, g->c, HW, a[l], wq + g->w_off, wq + g->b_off, z[l], bnm[l],
                               bni[l]);
                    if (track)
                        for (int c = 0; c < g->c; c++) {
                            /* error of a float evaluation: a few roundings of each term, the
                             * input's own error, and its effect on the mean and the scale */
                            double emax = 0.0;
                            for (int n = 0; n < Nb; n++)
                                for (int t = 0; t < HW; t++) {
                                    const double ev = e[l][((long)n * g->c + c) * HW + t];
                                    if (ev > emax) emax = ev;
                                }
                            const double gm = fabs(wq[g->w_off + c]), iv = bni[l][c];
                            for (int n = 0; n < Nb; n++)
                                for (int t = 0; t < HW; t++) {
                                    const long o = ((long)n * g->c + c) * HW + t;
                                    const double xh = fabs((a[l][o] - bnm[l][c]) * iv);
                                    const double ez = 16.0 * ldexp(1.0, -24) *
                                                          (gm * xh + fabs(wq[g->b_off + c])) +
                                                      gm * iv * (e[l][o] + emax) +
                                                      2.0 * gm * xh * emax * iv;
                                    e[l + 1][o] = ez + 2.0 * us * (fabs(z[l][o]) + ez);
                                    dbuf2[o] = ez;
                                }
                        }
                } else if (g->kind == ORC_ADDP) {
                    /* the projection: a 1x1 convolution of stride s of the source's output, its
                     * result stored like a convolution's output, then added */
                    const orc_geom* gs = &G[g->k];
                    const orc_geom pg = {ORC_CONV, 0, gs->oc, gs->oh, gs->ow, g->oc, g->oh, g->ow,
                                         1, g->s, 0, 1, 0, 0, 0, 0};
                    const double* sa = a[g->k + 1];
                    layer_fwd(&pg, Nb, sa, wq + g->w_off, wq + g->b_off, proj[l]);
                    if (track) {
                        /* bound of the stored projection (as for a convolution), then of the sum */
                        const double gam = gamma_f32(2 * ((long)gs->oc + 1));
                        double* absa = dbuf;
                        const long ssz = act_size(gs) * Nb;
                        for (long t = 0; t < ssz; t++) absa[t] = fabs(sa[t]);
                        layer_fwd(&pg, Nb, absa, wabs + g->w_off, wabs + g->b_off, dbuf2);
                        double* ep = z[l]; /* scratch: z[l] is written below */
                        layer_fwd(&pg, Nb, e[g->k + 1], wabs + g->w_off, NULL, ep);
                        for (long t = 0; t < sz; t++) {
                            const double ev = gam * dbuf2[t] + ep[t];
                            dbuf2[t] = ev + us * (fabs(proj[l][t]) + ev); /* stored projection */
                        }
                    }
                    for (long t = 0; t < sz; t++) proj[l][t] = store(proj[l][t]);
                    for (long t = 0; t < sz; t++) z[l][t] = a[l][t] + proj[l][t];
                    if (track)
                        for (long t = 0; t < sz; t++) {
                            const double ez = e[l][t] + dbuf2[t] + ldexp(1.0, -24) * fabs(z[l][t]);
                            e[l + 1][t] = ez + 2.0 * us * (fabs(z[l][t]) + ez);
                            dbuf2[t] = ez;
                        }
                } else if (g->kind == ORC_ADD) {
                    const double* sa = a[g->k + 1];
                    for (long t = 0; t < sz; t++) z[l][t] = a[l][t] + sa[t];
                    if (track)
                        for (long t = 0; t < sz; t++) {
                            const double ez = e[l][t] + e[g->k + 1][t] + ldexp(1.0, -24) * fabs(z[l][t]);
                            e[l + 1][t] = ez + 2.0 * us * (fabs(z[l][t]) + ez);
                            dbuf2[t] = ez;
                        }
                } else {
                layer_fwd(g, Nb, a[l], wq + g->w_off, wq + g->b_off, z[l]);
                if (track) {
                    /* forward error bound of a float evaluation in any summation order:
                     * gamma(2(K+1)) * sum|w||a| + sum|w| e_in, then the storage rounding */
                    long Kacc = (g->kind == ORC_CONV) ? (long)(g->c / g->g) * g->k * g->k
                                                      : (long)g->c * g->h * g->w;
                    double gam = gamma_f32(2 * (Kacc + 1));
                    double* absa = dbuf;
                    long insz = (long)g->c * g->h * g->w * Nb;
                    for (long t = 0; t < insz; t++) absa[t] = fabs(a[l][t]);
                    layer_fwd(g, Nb, absa, wabs + g->w_off, wabs + g->b_off, e[l + 1]);
                    layer_fwd(g, Nb, e[l], wabs + g->w_off, NULL, dbuf2);
                    for (long t = 0; t < sz; t++) {
                        double ez = gam * e[l + 1][t] + dbuf2[t];
                        e[l + 1][t] = ez + 2.0 * us * (fabs(z[l][t]) + ez);
                        dbuf2[t] = ez;     /* bound of the pre-activation itself */
                    }
                }
                }
                double rwindow = 0.0; /* hint_rel times the layer's largest output here */
                if (g->relu && relu_hint) {
                    for (long t = 0; t < sz; t++)
                        if (z[l][t] > rwindow) rwindow = z[l][t];
                    rwindow *= hint_rel;
                }
                for (long t = 0; t < sz; t++) {
                    double zt = z[l][t];
                    int pass = 1;
                    if (g->relu) {
                        pass = zt > 0.0;
                        if (relu_hint) {
                            int8_t hv = relu_hint[relu_off[l] + (long)r * sz + t];
                            if (hv >= 0 && hv != pass) {
                                const double lim = dbuf2[t] < rwindow ? dbuf2[t] : rwindow;
                                if (fabs(zt) > lim) { rc = ORC_EHINT; goto done; }
                                pass = hv;
                            }
                        }
                    }
                    double out = pass ? zt : 0.0;
                    a[l + 1][t] = last ? store32(out) : store(out);
                    /* a hinted pass of a non-positive value stores a tiny value; keep the mask */
                    if (g->relu) z[l][t] = pass ? 1.0 : 0.0;
                }
            }
            /* export stored outputs and decisions of this shard */
            if (acts)
                for (long t = 0; t < sz; t++)
                    acts[act_off[l] + (long)r * sz + t] = (float)a[l + 1][t];
            if (pool_argmax && g->kind == ORC_MAXPOOL)
                for (long t = 0; t < sz; t++) pool_argmax[pool_off[l] + (long)r * sz + t] = am[l][t];
            if (relu_mask && g->relu)
                for (long t = 0; t < sz; t++)
                    relu_mask[relu_off[l] + (long)r * sz + t] = (int8_t)(z[l][t] > 0.0);
        }

        /* ---- loss: mean over the shard; gradient of the shard-mean loss ---- */
        const orc_geom* gl = &G[n_layers - 1];
        int NC = gl->oc;
        double* dcur = dbuf;
        orc_softmax_xent(Nb, NC, a[n_layers], labels + (long)r * Nb, 1.0 / Nb, lossn, dcur);
        double ls = 0.0;
        for (int n = 0; n < Nb; n++) ls += lossn[n];
        ls /= Nb;
        if (shard_loss) shard_loss[r] = (float)ls;
        loss_total += ls;
        for (long t = 0; t < (long)Nb * NC; t++) dcur[t] = store(dcur[t]);

        /* ---- backward in reverse layer order ---- */
        for (int l = n_layers - 1; l >= 0; l--) {
            const orc_geom* g = &G[l];
            long sz = act_size(g) * Nb;
            long insz = (long)g->c * g->h * g->w * Nb;
            double* dnext = (dcur == dbuf) ? dbuf2 : dbuf;
            /* a layer whose output a residual addition also read: its output gradient is the
             * sum of the two paths (each stored in the storage precision, the sum rounded) */
            if (skipg[l])
                for (long t = 0; t < sz; t++) dcur[t] = store(dcur[t] + skipg[l][t]);
            if (g->relu)
                for (long t = 0; t < sz; t++)
                    if (z[l][t] <= 0.0) dcur[t] = 0.0;
            if (g->kind == ORC_MAXPOOL) {
                orc_maxpool_bwd(Nb, g->c, g->h, g->w, g->k, g->s, am[l], dcur, dnext);
                for (long t = 0; t < insz; t++) dnext[t] = store(dnext[t]);
            } else if (g->kind == ORC_ADD) {
                /* the gradient reaches the previous layer and the source layer unchanged */
                for (long t = 0; t < sz; t++) skipg[g->k][t] = dcur[t];
                for (long t = 0; t < insz; t++) dnext[t] = dcur[t];
            } else if (g->kind == ORC_ADDP) {
                /* unchanged to the previous layer; through the projection to the source (its
                 * data gradient stored), and the projection's weight and bias gradients */
                const orc_geom* gs = &G[g->k];
                for (long t = 0; t < insz; t++) dnext[t] = dcur[t];
                orc_conv_bwd(Nb, gs->oc, gs->oh, gs->ow, g->oc, 1, g->s, 0, 1, a[g->k + 1],
                             wq + g->w_off, dcur, skipg[g->k], gw + g->w_off, gw + g->b_off);
                for (long t = 0; t < act_size(gs) * Nb; t++) skipg[g->k][t] = store(skipg[g->k][t]);
                for (long i = 0; i < g->w_len + g->b_len; i++) {
                    float gf = (float)gw[g->w_off + i];
                    if (grads) grads[(long)r * P + g->w_off + i] = gf;
                    gsum[g->w_off + i] += (double)gf;
                }
            } else if (g->kind == ORC_BN) {
                double* dx = (l > 0) ? dnext : NULL;
                orc_bn_bwd(Nb, g->c, g->h * g->w, a[l], wq + g->w_off, bnm[l], bni[l], dcur, dx,
                           gw + g->w_off, gw + g->b_off);
                if (dx)
                    for (long t = 0; t < insz; t++) dx[t] = store(dx[t]);
                for (long i = 0; i < g->w_len + g->b_len; i++) {
                    float gf = (float)gw[g->w_off + i];
                    if (grads) grads[(long)r * P + g->w_off + i] = gf;
                    gsum[g->w_off + i] += (double)gf;
                }
            } else {
                double* dx = (l > 0) ? dnext : NULL;
                if (g->kind == ORC_CONV)
                    orc_conv_bwd(Nb, g->c, g->h, g->w, g->oc, g->k, g->s, g->p, g->g, a[l],
                                 wq + g->w_off, dcur, dx, gw + g->w_off, gw + g->b_off);
                else
                    orc_fc_bwd(Nb, g->c * g->h * g->w, g->oc, a[l], wq + g->w_off, dcur, dx,
                               gw + g->w_off, gw + g->b_off);
                if (dx)
                    for (long t = 0; t < insz; t++) dx[t] = store(dx[t]);
                for (long i = 0; i < g->w_len + g->b_len; i++) {
                    float gf = (float)gw[g->w_off + i];
                    if (grads) grads[(long)r * P + g->w_off + i] = gf;
                    gsum[g->w_off + i] += (double)gf;
                }
            }
            dcur = dnext;
        }
    }

    /* ---- average of the R replica gradients (the all-reduce of Sec. III-D.2) ---- */
    for (long i = 0; i < P; i++) gavg[i] = (float)(gsum[i] / R);
    /* ---- momentum / SGD update ---- */
    for (long i = 0; i < P; i++) {
        double gi = (double)gavg[i];
        if (mu != 0.0f) {
            double vn = (double)(float)((double)mu * (double)v[i] + gi);
            if (v_new) v_new[i] = (float)vn;
            if (w_new) w_new[i] = (float)((double)w[i] - (double)lr * vn);
        } else {
            if (v_new) v_new[i] = v ? v[i] : 0.0f;
            if (w_new) w_new[i] = (float)((double)w[i] - (double)lr * gi);
        }
    }
    if (loss_out) *loss_out = loss_total / R;
    rc = ORC_OK;

done:
    if (a) for (int l = 0; l <= n_layers; l++) free(a[l]);
    if (e) for (int l = 0; l <= n_layers; l++) free(e[l]);
    if (z) for (int l = 0; l < n_layers; l++) free(z[l]);
    if (am) for (int l = 0; l < n_layers; l++) free(am[l]);
    if (bnm) for (int l = 0; l < n_layers; l++) free(bnm[l]);
    if (bni) for (int l = 0; l < n_layers; l++) free(bni[l]);
    if (skipg) for (int l = 0; l < n_layers; l++) free(skipg[l]);
    if (proj) for (int l = 0; l < n_layers; l++) free(proj[l]);
    free(a); free(e); free(z); free(am); free(bnm); free(bni); free(skipg); free(proj);
    free(act_off); free(pool_off); free(relu_off);
    free(wq); free(wabs); free(gsum); free(lossn); free(dbuf); free(dbuf2); free(gw); free(G);
    return rc;
}

/* Average of R gradient buffers (row stride ld) fused with the momentum update, as the last two
 * stages of the step above.  Exposed on its own for the gradient-average microbenchmark.
 * v / v_new may be NULL iff mu == 0; gavg and w_new may be NULL. */
int orc_average_update(const float* grads, int R, long n, long ld, float* w, float* v, float lr,
                       float mu, float* gavg)
{
    if (!grads || R < 1 || n < 1 || ld < n || (!v && mu != 0.0f)) return ORC_EINVAL;
    for (long i = 0; i < n; i++) {
        double s = 0.0;
        for (int r = 0; r < R; r++) s += (double)grads[(long)r * ld + i];
        float gi = (float)(s / R);
        if (gavg) gavg[i] = gi;
        if (!w) continue;
        if (mu != 0.0f) {
            double vn = (double)(float)((double)mu * (double)v[i] + (double)gi);
            v[i] = (float)vn;
            w[i] = (float)((double)w[i] - (double)lr * vn);
        } else {
            w[i] = (float)((double)w[i] - (double)lr * (double)gi);
        }
    }
    return ORC_OK;
}

/* The same average followed by the other update rules that Sec. I lists among TensorFlow's
 * gradient-descent improvements.  The paper gives no formula for them; each is the definition
 * in the work it cites.  Every state and weight is rounded to float once per step, as the
 * step stores them; the arithmetic in between is double.
 *
 * Adam (Kingma and Ba, cited in Sec. I; Algorithm 1 of that work), at step t >= 1:
 *   m <- b1*m + (1-b1)*g,  v <- b2*v + (1-b2)*g^2,
 *   w <- w - lr * (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps).
 * The constant eps is added to the square root of the bias-corrected second moment, as in
 * that algorithm (TensorFlow's own kernel adds it before the bias correction instead). */
int orc_average_adam(const float* grads, int R, long n, long ld, float* w, float* m, float* v,
                     float lr, float b1, float b2, float eps, long step, float* gavg)
{
    if (!grads || !w || !m || !v || R < 1 || n < 1 || ld < n || step < 1) return ORC_EINVAL;
    const double bc1 = 1.0 - pow((double)b1, (double)step);
    const double bc2 = 1.0 - pow((double)b2, (double)step);
    for (long i = 0; i < n; i++) {
        double s = 0.0;
        for (int r = 0; r < R; r++) s += (double)grads[(long)r * ld + i];
        const double g = (double)(float)(s / R);
        if (gavg) gavg[i] = (float)g;
        const double mi = (double)(float)((double)b1 * m[i] + (1.0 - (double)b1) * g);
        const double vi = (double)(float)((double)b2 * v[i] + (1.0 - (double)b2) * g * g);
        m[i] = (float)mi;
        v[i] = (float)vi;
        const double mhat = mi / bc1, vhat = vi / bc2;
        w[i] = (float)((double)w[i] - (double)lr * mhat / (sqrt(vhat) + (double)eps));
    }
    return ORC_OK;
}

/* AdaGrad (Duchi, Hazan and Singer, cited in Sec. I), diagonal form with the accumulated sum of
 * squared gradients G (its initial value is whatever acc holds, zero for a fresh start):
 *   G <- G + g^2,  w <- w - lr * g / (sqrt(G) + eps). */
int orc_average_adagrad(const float* grads, int R, long n, long ld, float* w, float* acc,
                        float lr, float eps, float* gavg)
{
    if (!grads || !w || !acc || R < 1 || n < 1 || ld < n) return ORC_EINVAL;
    for (long i = 0; i < n; i++) {
        double s = 0.0;
        for (int r = 0; r < R; r++) s += (double)grads[(long)r * ld + i];
        const double g = (double)(float)(s / R);
        if (gavg) gavg[i] = (float)g;
        const double G = (double)(float)((double)acc[i] + g * g);
        acc[i] = (float)G;
        w[i] = (float)((double)w[i] - (double)lr * g / (sqrt(G) + (double)eps));
    }
    return ORC_OK;
}
