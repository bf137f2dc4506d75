/*
 * hpacml_oracle.c -- CPU oracle for the surrogate-inference region of HPAC-ML
 * (arXiv 2407.18352).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke entry point and the
 * CPU-baseline leg of the benchmark may load this library.  The product path
 * (the HIP library) never calls, links or includes anything from here, and this
 * file includes nothing from the product.
 *
 * It is a plain, slow, scalar restatement of what the paper says the region
 * computes, in the paper's order:
 *   1. the tensor map sweeps a concrete index range and applies the functor at
 *      every point (Sec. III-B; grammar in Fig. 3);
 *   2. each right-hand-side slice of the functor is located relative to the
 *      sweep point (Sec. IV-A, Symbolic Shape Extraction / Resolution), wrapped
 *      as a view (Tensor Wrapping) and the views are flattened and concatenated
 *      into the left-hand-side feature vector (Tensor Composition);
 *   3. the model runs on the composed tensor (Sec. IV-B, inference);
 *   4. the output tensor is written back through a `from` map, which performs
 *      extraction, resolution and wrapping but no composition (Sec. IV-A, last
 *      paragraph);
 *   5. collect mode records the mapped values instead (Sec. III-A-2, IV-B);
 *   6. convolutional surrogates (the MiniWeather and ParticleFilter model
 *      spaces of Table IV: convolution, max-pool and fully connected layers)
 *      run on the composed tensor seen as images: the last two sweep
 *      dimensions are the image rows and columns, the features its channels.
 *
 * Arithmetic is fp64 with sequential summation.  Where the paper is silent the
 * readings are (each is listed in the design notes):
 *   - feature order: target-major, then slice order, then row-major over the
 *     slice's element counts;
 *   - batch order: row-major over the sweep (last dimension fastest);
 *   - boundaries: per dimension none / periodic / clamp;
 *   - symbolic expressions: `symbol + integer` only;
 *   - model: Linear layers with weight layout [out][in], per-layer activation
 *     identity or ReLU (hidden layers ReLU, output linear);
 *   - bf16 models: weights, gathered inputs and hidden activations rounded to
 *     bf16 (round to nearest even) after an fp32 rounding; biases and outputs
 *     stay fp32;
 *   - convolution: PyTorch's Conv2d definition (weights [out][in][kh][kw],
 *     cross-correlation), "same" padding split as floor((k-1)/2) before and
 *     the rest after, padding modes zeros / circular / replicate; max-pool
 *     without padding, NaN if any window value is NaN; a fully connected
 *     layer flattens its input image in [row][column][channel] order (the
 *     composed tensor's own order).
 *
 * Every function here is pinned by tests that do not re-type its formula:
 * brute-force numpy enumeration with np.pad wrap/edge, the paper's 5-point
 * example, one-hot weights, a float64 matmul, torch fp64 Linear stacks,
 * torch fp64 Conv2d/Conv3d with circular padding, batch-order invariance and
 * torch's own bf16 conversion over every fp32 bit pattern.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_MAX_RANK 4

enum { OR_BND_NONE = 0, OR_BND_PERIODIC = 1, OR_BND_CLAMP = 2 };
enum { OR_OK = 0, OR_ERR_RANGE = -1, OR_ERR_ARG = -2, OR_ERR_NOMEM = -3 };

/* A tensor map applied to concrete arrays: functor (slices), sweep, boundary
 * handling and the targets.  All targets share one index space (`extent`);
 * strides are per target, in elements. */
typedef struct {
    int32_t rank;
    int32_t n_slices;
    int32_t n_targets;
    int32_t pad_;
    const int32_t *lo;     /* [n_slices][4]: first element of slice relative to the symbol */
    const int32_t *count;  /* [n_slices][4]: elements of the slice per dimension */
    int64_t start[OR_MAX_RANK], stop[OR_MAX_RANK], step[OR_MAX_RANK];
    int32_t bnd[OR_MAX_RANK];
    int64_t extent[OR_MAX_RANK];
    void *const *data;     /* [n_targets] 32-bit element arrays */
    const int64_t *stride; /* [n_targets][4] */
} or_map;

/* A multilayer perceptron: layer l maps dims[l] -> dims[l+1] with
 * W[l] of shape [dims[l+1]][dims[l]] (row-major) and bias b[l]. */
typedef struct {
    int32_t n_layers;
    int32_t bf16;          /* 0: fp32 model, 1: bf16 weights/activations */
    const int32_t *dims;   /* [n_layers + 1] */
    const float *const *W; /* [n_layers] */
    const float *const *b; /* [n_layers] */
    const int32_t *act;    /* [n_layers]: 0 identity, 1 ReLU */
} or_model;

int or_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of later parallel loops (timing runs only; results do not depend on it). */
void or_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ---- bf16 round to nearest even ------------------------------------------
 * bf16 keeps the top 16 bits of an fp32 pattern.  Rounding to nearest even
 * adds half an ulp of the kept part (0x7FFF) plus the parity of the kept lsb,
 * then truncates.  NaNs map to a quiet NaN with the same sign. */
static uint16_t bf16_bits(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u)
        return (uint16_t)((u >> 16) | 0x0040u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

static float bf16_to_float(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* fp64 value -> fp32 (round to nearest even) -> bf16 (round to nearest even) */
static double quant_bf16(double v)
{
    return (double)bf16_to_float(bf16_bits((float)v));
}

void or_bf16_bits(const float *in, uint16_t *out, int64_t n)
{
    int64_t i;
#pragma omp parallel for schedule(static)
    for (i = 0; i < n; ++i)
        out[i] = bf16_bits(in[i]);
}

/* ---- sweep --------------------------------------------------------------
 * A concrete slice [start:stop:step] (stop exclusive) per dimension
 * (Sec. III-C, cs-specifier).  Points are numbered row-major. */
static int64_t sweep_len(const or_map *m, int d)
{
    int64_t span = m->stop[d] - m->start[d];
    if (span <= 0)
        return 0;
    return (span + m->step[d] - 1) / m->step[d];
}

int64_t or_map_points(const or_map *m)
{
    int64_t n = 1;
    for (int d = 0; d < m->rank; ++d)
        n *= sweep_len(m, d);
    return n;
}

int32_t or_map_features(const or_map *m)
{
    int64_t per = 0;
    for (int s = 0; s < m->n_slices; ++s) {
        int64_t e = 1;
        for (int d = 0; d < m->rank; ++d)
            e *= m->count[s * 4 + d];
        per += e;
    }
    return (int32_t)(per * m->n_targets);
}

void or_point_coords(const or_map *m, int64_t b, int64_t *p)
{
    for (int d = m->rank - 1; d >= 0; --d) {
        int64_t n = sweep_len(m, d);
        int64_t k = b % n;
        b /= n;
        p[d] = m->start[d] + k * m->step[d];
    }
}

/* Boundary handling of one coordinate (a reading: the paper only maps
 * interiors).  Returns 0 and the resolved coordinate, or OR_ERR_RANGE. */
static int resolve(int64_t x, int64_t n, int bnd, int64_t *q)
{
    if (x >= 0 && x < n) {
        *q = x;
        return OR_OK;
    }
    if (bnd == OR_BND_PERIODIC) {
        int64_t r = x % n;
        if (r < 0)
            r += n;
        *q = r;
        return OR_OK;
    }
    if (bnd == OR_BND_CLAMP) {
        *q = x < 0 ? 0 : n - 1;
        return OR_OK;
    }
    return OR_ERR_RANGE;
}

/* Elements touched by one sweep point, in feature order.
 * Extraction: slice s of the functor starts at p + lo[s] (its offset relative
 * to the sweep point).  Resolution: it spans count[s][d] elements per
 * dimension.  Wrapping: the element with slice-local index e sits at
 * p + lo[s] + e in target t.  Composition: flatten each slice row-major and
 * concatenate slices, target after target (Sec. IV-A). */
static int point_elements(const or_map *m, int64_t b, int32_t *tgt, int64_t *elem)
{
    int64_t p[OR_MAX_RANK];
    or_point_coords(m, b, p);
    int f = 0;
    for (int t = 0; t < m->n_targets; ++t) {
        for (int s = 0; s < m->n_slices; ++s) {
            const int32_t *lo = m->lo + 4 * s;
            const int32_t *cnt = m->count + 4 * s;
            int64_t total = 1;
            for (int d = 0; d < m->rank; ++d)
                total *= cnt[d];
            for (int64_t e = 0; e < total; ++e) {
                int64_t rem = e, idx = 0, ed[OR_MAX_RANK];
                for (int d = m->rank - 1; d >= 0; --d) {
                    ed[d] = rem % cnt[d];
                    rem /= cnt[d];
                }
                for (int d = 0; d < m->rank; ++d) {
                    int64_t q;
                    if (resolve(p[d] + lo[d] + ed[d], m->extent[d], m->bnd[d], &q) != OR_OK)
                        return OR_ERR_RANGE;
                    idx += q * m->stride[t * 4 + d];
                }
                tgt[f] = t;
                elem[f] = idx;
                ++f;
            }
        }
    }
    return f;
}

/* ---- gather (tensor composition) ----------------------------------------
 * X[r][f] for the listed sweep rows (all rows when rows == NULL), each value
 * promoted exactly from fp32 to fp64. */
int or_gather(const or_map *m, const int64_t *rows, int64_t n, double *X)
{
    int F = or_map_features(m);
    int err = OR_OK;
    int64_t r;
#pragma omp parallel
    {
        int32_t *tgt = malloc(sizeof(int32_t) * (F ? F : 1));
        int64_t *elem = malloc(sizeof(int64_t) * (F ? F : 1));
#pragma omp for schedule(static)
        for (r = 0; r < n; ++r) {
            int64_t b = rows ? rows[r] : r;
            if (point_elements(m, b, tgt, elem) < 0) {
#pragma omp atomic write
                err = OR_ERR_RANGE;
                continue;
            }
            for (int f = 0; f < F; ++f)
                X[r * F + f] = (double)((const float *)m->data[tgt[f]])[elem[f]];
        }
        free(tgt);
        free(elem);
    }
    return err;
}

/* ---- collect --------------------------------------------------------------
 * The record of a mapped region: the gathered values, copied as 32-bit
 * patterns into dst[r * ld + f] (Sec. III-A-2 Execution Control; Sec. IV-B). */
int or_collect(const or_map *m, const int64_t *rows, int64_t n, uint32_t *dst, int64_t ld)
{
    int F = or_map_features(m);
    int err = OR_OK;
    int64_t r;
    if (ld < F)
        return OR_ERR_ARG;
#pragma omp parallel
    {
        int32_t *tgt = malloc(sizeof(int32_t) * (F ? F : 1));
        int64_t *elem = malloc(sizeof(int64_t) * (F ? F : 1));
#pragma omp for schedule(static)
        for (r = 0; r < n; ++r) {
            int64_t b = rows ? rows[r] : r;
            if (point_elements(m, b, tgt, elem) < 0) {
#pragma omp atomic write
                err = OR_ERR_RANGE;
                continue;
            }
            for (int f = 0; f < F; ++f)
                dst[r * ld + f] = ((const uint32_t *)m->data[tgt[f]])[elem[f]];
        }
        free(tgt);
        free(elem);
    }
    return err;
}

/* ---- model ----------------------------------------------------------------
 * Weights as fp64, rounded to bf16 first for a bf16 model. */
static double *model_weights(const or_model *mdl, int64_t *woff, int64_t *boff)
{
    int64_t wtot = 0, btot = 0;
    for (int l = 0; l < mdl->n_layers; ++l) {
        woff[l] = wtot;
        boff[l] = btot;
        wtot += (int64_t)mdl->dims[l] * mdl->dims[l + 1];
        btot += mdl->dims[l + 1];
    }
    double *w = malloc(sizeof(double) * (size_t)(wtot + btot + 1));
    if (!w)
        return NULL;
    for (int l = 0; l < mdl->n_layers; ++l) {
        int64_t nw = (int64_t)mdl->dims[l] * mdl->dims[l + 1];
        for (int64_t i = 0; i < nw; ++i) {
            double v = (double)mdl->W[l][i];
            w[woff[l] + i] = mdl->bf16 ? quant_bf16(v) : v;
        }
        for (int64_t o = 0; o < mdl->dims[l + 1]; ++o)
            w[wtot + boff[l] + o] = (double)mdl->b[l][o]; /* biases stay fp32 */
        boff[l] += wtot;
    }
    return w;
}

/* One point through the network: per layer
 *   acc[o] = b[o] + sum_i W[o][i] * h[i]   (fp64, i ascending)
 *   h'[o]  = act(acc[o])
 * with the bf16 rounding points of a bf16 model; output rounded to fp32. */
static void mlp_point(const or_model *mdl, const double *w, const int64_t *woff, const int64_t *boff,
                      const double *x, double *h0, double *h1, float *y)
{
    int L = mdl->n_layers;
    for (int i = 0; i < mdl->dims[0]; ++i)
        h0[i] = mdl->bf16 ? quant_bf16(x[i]) : x[i];
    double *hin = h0, *hout = h1;
    for (int l = 0; l < L; ++l) {
        int K = mdl->dims[l], N = mdl->dims[l + 1];
        const double *W = w + woff[l];
        const double *bias = w + boff[l];
        for (int o = 0; o < N; ++o) {
            double acc = bias[o];
            for (int i = 0; i < K; ++i)
                acc += W[(int64_t)o * K + i] * hin[i];
            if (mdl->act[l] == 1)
                acc = acc > 0.0 ? acc : 0.0;
            if (mdl->bf16 && l < L - 1)
                acc = quant_bf16(acc);
            hout[o] = acc;
        }
        double *t = hin;
        hin = hout;
        hout = t;
    }
    for (int g = 0; g < mdl->dims[L]; ++g)
        y[g] = (float)hin[g];
}

static int max_width(const or_model *mdl)
{
    int mw = 1;
    for (int l = 0; l <= mdl->n_layers; ++l)
        if (mdl->dims[l] > mw)
            mw = mdl->dims[l];
    return mw;
}

/* Model on an already composed input tensor X[n][dims[0]] -> Y[n][dims[L]]. */
int or_mlp(const or_model *mdl, const double *X, int64_t n, float *Y)
{
    int64_t woff[64], boff[64];
    if (mdl->n_layers < 1 || mdl->n_layers > 64)
        return OR_ERR_ARG;
    double *w = model_weights(mdl, woff, boff);
    if (!w)
        return OR_ERR_NOMEM;
    int mw = max_width(mdl), Fin = mdl->dims[0], Fout = mdl->dims[mdl->n_layers];
    int64_t r;
#pragma omp parallel
    {
        double *h0 = malloc(sizeof(double) * mw), *h1 = malloc(sizeof(double) * mw);
#pragma omp for schedule(static)
        for (r = 0; r < n; ++r)
            mlp_point(mdl, w, woff, boff, X + r * Fin, h0, h1, Y + r * Fout);
        free(h0);
        free(h1);
    }
    free(w);
    return OR_OK;
}

/* Inference for the listed sweep rows (all when rows == NULL): gather through
 * the `to` map, then the model.  Writes Y[r][dims[L]] and nothing else, so the
 * caller can take every gather before any scatter (the region reads its inputs
 * before writing its outputs, Sec. III-A-2 Steps 1-2 before 5-6). */
int or_infer_rows(const or_map *in, const or_model *mdl, const int64_t *rows, int64_t n, float *Y)
{
    int64_t woff[64], boff[64];
    int F = or_map_features(in);
    if (mdl->n_layers < 1 || mdl->n_layers > 64 || F != mdl->dims[0])
        return OR_ERR_ARG;
    double *w = model_weights(mdl, woff, boff);
    if (!w)
        return OR_ERR_NOMEM;
    int mw = max_width(mdl), Fout = mdl->dims[mdl->n_layers];
    int err = OR_OK;
    int64_t r;
#pragma omp parallel
    {
        double *h0 = malloc(sizeof(double) * mw), *h1 = malloc(sizeof(double) * mw);
        double *x = malloc(sizeof(double) * (F ? F : 1));
        int32_t *tgt = malloc(sizeof(int32_t) * (F ? F : 1));
        int64_t *elem = malloc(sizeof(int64_t) * (F ? F : 1));
#pragma omp for schedule(static)
        for (r = 0; r < n; ++r) {
            int64_t b = rows ? rows[r] : r;
            if (point_elements(in, b, tgt, elem) < 0) {
#pragma omp atomic write
                err = OR_ERR_RANGE;
                continue;
            }
            for (int f = 0; f < F; ++f)
                x[f] = (double)((const float *)in->data[tgt[f]])[elem[f]];
            mlp_point(mdl, w, woff, boff, x, h0, h1, Y + r * Fout);
        }
        free(h0);
        free(h1);
        free(x);
        free(tgt);
        free(elem);
    }
    free(w);
    return err;
}

/* `from` map: the output tensor is written into the wrapped views of the
 * application arrays (Sec. IV-A, last paragraph).  Row r of Y goes to sweep
 * point rows[r]; feature g to the g-th element that point addresses. */
int or_scatter(const or_map *m, const int64_t *rows, int64_t n, const float *Y)
{
    int F = or_map_features(m);
    int32_t *tgt = malloc(sizeof(int32_t) * (F ? F : 1));
    int64_t *elem = malloc(sizeof(int64_t) * (F ? F : 1));
    int err = OR_OK;
    for (int64_t r = 0; r < n && err == OR_OK; ++r) {
        int64_t b = rows ? rows[r] : r;
        if (point_elements(m, b, tgt, elem) < 0) {
            err = OR_ERR_RANGE;
            break;
        }
        for (int g = 0; g < F; ++g)
            ((float *)m->data[tgt[g]])[elem[g]] = Y[r * F + g];
    }
    free(tgt);
    free(elem);
    return err;
}

/* ---- convolutional surrogates ---------------------------------------------
 * The composed tensor X[S][H][W][C0] (sweep order: leading sweep dimensions
 * number the S images, the last two are the rows and columns, the features
 * are the channels) passes through the layers in order. */
enum { OR_CONV2D = 0, OR_MAXPOOL2D = 1, OR_LINEAR = 2 };
enum { OR_PAD_VALID = 0, OR_PAD_SAME = 1 };
enum { OR_PM_ZEROS = 0, OR_PM_CIRCULAR = 1, OR_PM_REPLICATE = 2 };

typedef struct {
    int32_t kind;
    int32_t out_channels;  /* conv: output channels; linear: outputs */
    int32_t kh, kw;        /* window */
    int32_t sh, sw;        /* steps */
    int32_t padding;       /* conv: valid / same */
    int32_t pad_mode;      /* conv with same padding */
    int32_t act;           /* 0 identity, 1 ReLU */
    int32_t pad_;
    const float *W;        /* conv [out][in][kh][kw]; linear [out][in]; pool NULL */
    const float *b;        /* [out]; pool NULL */
} or_layer;

/* Image shape after every layer: shape[3l..3l+2] = (rows, columns, channels)
 * of layer l's input, l = 0..L (entry L is the output). */
int or_cnn_shapes(int32_t C0, int32_t H, int32_t W, int32_t L, const or_layer *ly, int32_t *shape)
{
    if (C0 < 1 || H < 1 || W < 1 || L < 1)
        return OR_ERR_ARG;
    int32_t h = H, w = W, c = C0;
    int flat = 0;
    shape[0] = h, shape[1] = w, shape[2] = c;
    for (int l = 0; l < L; ++l) {
        const or_layer *y = &ly[l];
        if (y->kind == OR_LINEAR) {
            c = y->out_channels;
            h = w = 1;
            flat = 1;
        } else {
            if (flat || y->kh < 1 || y->kw < 1 || y->sh < 1 || y->sw < 1)
                return OR_ERR_ARG;
            if (y->kind == OR_CONV2D && y->padding == OR_PAD_SAME) {
                if (y->sh != 1 || y->sw != 1)
                    return OR_ERR_ARG;
            } else {
                if (y->kh > h || y->kw > w)
                    return OR_ERR_ARG;
                h = (h - y->kh) / y->sh + 1;
                w = (w - y->kw) / y->sw + 1;
            }
            if (y->kind == OR_CONV2D)
                c = y->out_channels;
        }
        if (c < 1)
            return OR_ERR_ARG;
        shape[3 * (l + 1)] = h, shape[3 * (l + 1) + 1] = w, shape[3 * (l + 1) + 2] = c;
    }
    return OR_OK;
}

/* Input row or column q of a same-padded convolution, q possibly outside
 * [0, n): its index inside, or -1 for a zero (zeros mode). */
static int64_t pad_index(int64_t q, int64_t n, int mode)
{
    if (q >= 0 && q < n)
        return q;
    if (mode == OR_PM_CIRCULAR)
        return ((q % n) + n) % n;
    if (mode == OR_PM_REPLICATE)
        return q < 0 ? 0 : n - 1;
    return -1;
}

/* One layer on S images in[S][h][w][c] -> out[S][h2][w2][c2]. */
static void cnn_layer(const or_layer *y, const double *in, int64_t S, int h, int w, int c, double *out,
                      int h2, int w2, int c2)
{
    int64_t n_out = S * h2 * w2;
    int64_t i;
#pragma omp parallel for schedule(static)
    for (i = 0; i < n_out; ++i) {
        int64_t s = i / ((int64_t)h2 * w2);
        int oy = (int)(i / w2 % h2), ox = (int)(i % w2);
        const double *img = in + s * h * w * c;
        double *o = out + i * c2;
        if (y->kind == OR_CONV2D) {
            /* out[co] = b[co] + sum over ci, ky, kx of W[co][ci][ky][kx] * in[y0 + ky][x0 + kx][ci] */
            int same = y->padding == OR_PAD_SAME;
            int64_t y0 = (int64_t)oy * y->sh - (same ? (y->kh - 1) / 2 : 0);
            int64_t x0 = (int64_t)ox * y->sw - (same ? (y->kw - 1) / 2 : 0);
            for (int co = 0; co < c2; ++co) {
                double acc = (double)y->b[co];
                for (int ci = 0; ci < c; ++ci)
                    for (int ky = 0; ky < y->kh; ++ky) {
                        int64_t r = same ? pad_index(y0 + ky, h, y->pad_mode) : y0 + ky;
                        for (int kx = 0; kx < y->kw; ++kx) {
                            int64_t q = same ? pad_index(x0 + kx, w, y->pad_mode) : x0 + kx;
                            double v = (r < 0 || q < 0) ? 0.0 : img[(r * w + q) * c + ci];
                            acc += (double)y->W[(((int64_t)co * c + ci) * y->kh + ky) * y->kw + kx] * v;
                        }
                    }
                o[co] = y->act == 1 ? (acc > 0.0 ? acc : 0.0) : acc;
            }
        } else if (y->kind == OR_MAXPOOL2D) {
            /* the largest window value; a NaN anywhere in the window wins */
            const double *win = img + ((int64_t)oy * y->sh * w + (int64_t)ox * y->sw) * c;
            for (int ch = 0; ch < c2; ++ch) {
                double m = win[ch];
                for (int ky = 0; ky < y->kh; ++ky)
                    for (int kx = 0; kx < y->kw; ++kx) {
                        double v = win[((int64_t)ky * w + kx) * c + ch];
                        if (!isnan(m) && (isnan(v) || v > m))
                            m = v;
                    }
                o[ch] = y->act == 1 ? (m > 0.0 ? m : 0.0) : m;
            }
        } else {
            /* the image flattened in [row][column][channel] order */
            int64_t n_in = (int64_t)h * w * c;
            for (int oo = 0; oo < c2; ++oo) {
                double acc = (double)y->b[oo];
                for (int64_t k = 0; k < n_in; ++k)
                    acc += (double)y->W[(int64_t)oo * n_in + k] * img[k];
                o[oo] = y->act == 1 ? (acc > 0.0 ? acc : 0.0) : acc;
            }
        }
    }
}

/* The whole stack on X[S][H][W][C0] (fp64) -> Y[S][H'][W'][C'] rounded to fp32. */
int or_cnn(int32_t C0, int32_t H, int32_t W, int32_t L, const or_layer *ly, const double *X, int64_t S,
           float *Y)
{
    int32_t shape[3 * 65];
    if (L > 64)
        return OR_ERR_ARG;
    int rc = or_cnn_shapes(C0, H, W, L, ly, shape);
    if (rc != OR_OK)
        return rc;
    int64_t big = 0;
    for (int l = 0; l <= L; ++l) {
        int64_t n = (int64_t)shape[3 * l] * shape[3 * l + 1] * shape[3 * l + 2];
        big = n > big ? n : big;
    }
    double *a = malloc(sizeof(double) * (size_t)(S * big + 1));
    double *bb = malloc(sizeof(double) * (size_t)(S * big + 1));
    if (!a || !bb) {
        free(a);
        free(bb);
        return OR_ERR_NOMEM;
    }
    memcpy(a, X, sizeof(double) * (size_t)(S * H * W * C0));
    for (int l = 0; l < L; ++l) {
        const int32_t *si = shape + 3 * l, *so = shape + 3 * (l + 1);
        cnn_layer(&ly[l], a, S, si[0], si[1], si[2], bb, so[0], so[1], so[2]);
        double *t = a;
        a = bb;
        bb = t;
    }
    int64_t n = S * (int64_t)shape[3 * L] * shape[3 * L + 1] * shape[3 * L + 2];
    for (int64_t i = 0; i < n; ++i)
        Y[i] = (float)a[i];
    free(a);
    free(bb);
    return OR_OK;
}
