/*
 * hpacml.h -- C ABI of an MI355X (gfx950) library for HPAC-ML's
 * surrogate-inference region (arXiv 2407.18352).
 *
 * A region replaces an annotated scientific kernel by a neural-network
 * surrogate.  Its inputs are described by a tensor functor (a per-point access
 * pattern with symbolic indices, Sec. III-B, Fig. 2) applied by a tensor map to
 * concrete application arrays over a concrete index sweep (Sec. III-C, Fig. 3);
 * the map turns the arrays into a dense [points x features] tensor
 * (Sec. IV-A: extraction, resolution, wrapping, composition).  The model runs
 * on that tensor and a `from` map writes its outputs back into application
 * arrays (Sec. IV-A, last paragraph; Sec. IV-B).  Collect mode records the
 * mapped values instead of running the model (Sec. III-A-2, Sec. IV-B).
 *
 * Every pointer to application data is a DEVICE pointer on the current HIP
 * device.  The stream argument is a hipStream_t passed as void* (NULL = the
 * null stream).  No function throws; every failure is reported as a status,
 * and every check is done on the host before anything is enqueued, so a call
 * that fails writes nothing.  `*out` handles are set to NULL on failure.
 *
 * Thread safety: maps and models are immutable after creation, except for
 * buffers allocated on first need and reused: a `to` map's snapshot record
 * (inferences whose outputs overlap their inputs) and a model's workspace
 * (the layer-by-layer paths of convolutional models and of multilayer
 * perceptrons outside the fused kernels).  Concurrent infer and collect
 * calls with the same handles on different streams are allowed, except that
 * calls using one of those buffers must not overlap in time.  A region is
 * used from one thread at a time, and its accurate path must not call
 * functions of the same region.
 */
#ifndef HPACML_H
#define HPACML_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HPACML_ABI_VERSION 2
#define HPACML_MAX_RANK 4         /* spatial dimensions of a functor / sweep */
#define HPACML_MAX_SLICES 64      /* right-hand-side slices per functor */
#define HPACML_MAX_TARGETS 64     /* arrays per map */
#define HPACML_MAX_FEATURES 256   /* features per point of one map */
#define HPACML_MAX_LAYERS 8       /* layers per model */
#define HPACML_MAX_WIDTH 4096     /* width of any layer */
#define HPACML_MAX_CNN_WIDTH 65536 /* channels of a convolutional layer, inputs of a LINEAR layer */

typedef enum {
    HPACML_OK = 0,
    HPACML_E_INVAL = 1,       /* NULL or malformed argument, non-device pointer */
    HPACML_E_SHAPE = 2,       /* feature / point counts do not agree */
    HPACML_E_RANGE = 3,       /* an access leaves an array without a boundary mode */
    HPACML_E_ALIAS = 4,       /* outputs or records that could write one element twice */
    HPACML_E_UNSUPPORTED = 5, /* valid request outside this library's limits */
    HPACML_E_NOMEM = 6,       /* device or host allocation failed */
    HPACML_E_DEVICE = 7       /* HIP runtime error (launch, copy, no device) */
} hpacml_status;

/* direction of a tensor map (Sec. III-C, direction-specifier) */
enum { HPACML_TO = 0, HPACML_FROM = 1 };
/* per-dimension handling of accesses outside [0, extent); the paper maps only
 * interiors, so NONE makes such an access an error (HPACML_E_RANGE) */
enum { HPACML_BND_NONE = 0, HPACML_BND_PERIODIC = 1, HPACML_BND_CLAMP = 2 };
/* element / compute types */
enum { HPACML_F32 = 0, HPACML_BF16 = 1 };
/* per-layer activation */
enum { HPACML_ACT_IDENTITY = 0, HPACML_ACT_RELU = 1 };

/* One right-hand-side slice of a tensor functor (Sec. III-B; Sec. IV-A,
 * Symbolic Shape Extraction).  In dimension d the slice covers the symbol's
 * value s_d plus lo[d], lo[d]+1, ..., lo[d]+count[d]-1.  Example: the slice
 * [i, j-1:j+2] is lo = {0, -1}, count = {1, 3}.  Entries at d >= rank are
 * ignored.  count[d] >= 1. */
typedef struct {
    int32_t lo[HPACML_MAX_RANK];
    int32_t count[HPACML_MAX_RANK];
} hpacml_slice;

/* A tensor functor [s_0, ..., s_{rank-1}, 0:n_features] = (slices...).
 * Applied to T targets, each target contributes every slice's elements;
 * features are ordered target-major, then slice order, then row-major over
 * the slice's counts (Sec. IV-A, Tensor Composition: flatten, then
 * concatenate).  n_features must equal T * sum over slices of prod(count). */
typedef struct {
    int32_t rank;                 /* 1..HPACML_MAX_RANK */
    int32_t n_slices;             /* 1..HPACML_MAX_SLICES */
    const hpacml_slice *slices;   /* [n_slices], read during the call only */
    int32_t n_features;
} hpacml_functor;

/* An application array, borrowed: the library keeps the pointer, never a copy
 * (Sec. IV-A, Tensor Wrapping).  extent and stride are in elements; element
 * (x_0, ..., x_{rank-1}) is data[sum_d x_d * stride[d]].  Strides may be any
 * non-negative values (views).  All targets of one map share extents. */
typedef struct {
    void *data;                   /* device pointer */
    int32_t dtype;                /* HPACML_F32 only */
    int32_t reserved;             /* must be 0 */
    int64_t extent[HPACML_MAX_RANK];
    int64_t stride[HPACML_MAX_RANK];
} hpacml_array;

/* The concrete slice of a map target, per dimension [start:stop:step], stop
 * exclusive, step >= 1 (Sec. III-C, cs-specifier: [1:N] is 1..N-1).  The sweep
 * has prod_d ceil((stop-start)/step) points, numbered row-major (last dimension
 * fastest); that number is the point's row in the composed tensor.
 * 0 <= start <= stop <= extent. */
typedef struct {
    int64_t start[HPACML_MAX_RANK];
    int64_t stop[HPACML_MAX_RANK];
    int64_t step[HPACML_MAX_RANK];
} hpacml_sweep;

typedef struct hpacml_map_s hpacml_map;
typedef struct hpacml_model_s hpacml_model;

/* Checks a map description without touching any device: functor shape,
 * feature count, sweep bounds, boundary modes and every access of every sweep
 * point against the extents.  On success writes the number of points and
 * features (either output pointer may be NULL).  Returns the status
 * hpacml_map_create would return for the same arguments, except for checks of
 * the data pointers themselves (device residency).
 *   f, targets, sweep, bnd: read during the call only.
 *   dir: HPACML_TO or HPACML_FROM.  A FROM map must use one slice with one
 *        element per dimension (each point writes one element per target);
 *        otherwise HPACML_E_UNSUPPORTED.  CLAMP with a nonzero offset on a FROM
 *        map is HPACML_E_INVAL (two points would write one element).  A FROM
 *        map whose strides could send two sweep points to one element of a
 *        target (a zero stride over a swept dimension, or strides that fold
 *        the sweep onto itself) is HPACML_E_ALIAS: the swept dimensions,
 *        taken by increasing stride, must each have a stride larger than the
 *        element distance the finer ones can span.
 *   bnd: [rank] boundary modes. */
hpacml_status hpacml_map_validate(const hpacml_functor *f, int32_t dir,
                                  const hpacml_array *targets, int32_t n_targets,
                                  const hpacml_sweep *sweep, const int32_t *bnd,
                                  int64_t *n_points, int32_t *n_features);

/* Creates a tensor map (Sec. III-C, `tensor map(to|from: functor(targets))`):
 * validates as hpacml_map_validate, checks that every target pointer is device
 * memory (HPACML_E_INVAL otherwise), builds the access plan (Sec. IV-A
 * extraction + resolution + wrapping, done once per map) and uploads it.  May
 * synchronise the device.  The caller keeps the arrays alive while work that
 * uses the map is in flight. */
hpacml_status hpacml_map_create(const hpacml_functor *f, int32_t dir,
                                const hpacml_array *targets, int32_t n_targets,
                                const hpacml_sweep *sweep, const int32_t *bnd,
                                hpacml_map **out);

/* Points (rows) and features (columns) of the map's tensor. */
hpacml_status hpacml_map_shape(const hpacml_map *m, int64_t *n_points, int32_t *n_features);

/* Frees a map.  NULL-safe.  Synchronise streams that use it first. */
void hpacml_map_destroy(hpacml_map *m);

/* Checks a model description without touching any device (same status as
 * hpacml_model_create would return for these arguments). */
hpacml_status hpacml_model_validate(int32_t n_layers, const int32_t *dims,
                                    const int32_t *act, int32_t compute);

/* Creates a multilayer perceptron (the surrogate; the paper's models are
 * TorchScript Linear/ReLU stacks, Sec. IV-B).  Layer l maps dims[l] inputs to
 * dims[l+1] outputs: y = act[l](W[l] x + b[l]).
 *   n_layers: 1..HPACML_MAX_LAYERS; dims: [n_layers+1], each 1..HPACML_MAX_WIDTH,
 *             dims[0] <= HPACML_MAX_FEATURES.
 *   W[l]: HOST fp32 [dims[l+1]][dims[l]] row-major (PyTorch Linear layout).
 *   b[l]: HOST fp32 [dims[l+1]].
 *   act:  [n_layers] HPACML_ACT_*.
 *   compute: HPACML_F32 (fp32 everywhere) or HPACML_BF16 (weights, gathered
 *            inputs and hidden activations rounded to bf16, nearest-even;
 *            fp32 accumulation; fp32 biases and outputs).
 * The weights are copied (and converted) into library-owned device memory;
 * the caller may free its host arrays on return.  Synchronises the device.
 * hpacml_infer runs the whole model in one fused kernel when both maps take
 * the library's 32-bit form and the model fits one of its MFMA kernels
 * (hidden widths up to 128 for fp32, up to 512 for bf16, with limits on
 * depth, input features and outputs per kernel; hidden layers narrower than
 * the kernel's width run zero-padded, which changes no result).  Any
 * other model or map runs layer by layer over chunks of points: a kernel
 * that gathers the inputs (and computes the first layer when the input width
 * is at most 12), one hipBLASLt matmul per further layer (bias and
 * activation applied to the fp32 accumulators in its epilogue; the same
 * rounding points), and a kernel that writes the outputs through the `from`
 * map (and computes the last layer when it has at most 8 outputs).  That
 * path uses a workspace the model owns (allocated on the first
 * such call, grown as needed, freed with the model): two activation buffers
 * of one chunk (about 1 GB each; the environment variable
 * HPACML_LAYERS_CHUNK_MB, read when the model is created, sets another size
 * from 1 MB to 64 GB),
 * the chunk's fp32 outputs and up to 64 MB of library scratch; calls that
 * share such a model must not overlap in time on different streams.  The
 * path is not meant for stream capture into a HIP graph (its first call
 * allocates, and the matmul library may clear its scratch with memsets).  Where the library has
 * no algorithm for a layer, a general fused VALU kernel runs instead. */
hpacml_status hpacml_model_create(int32_t n_layers, const int32_t *dims,
                                  const float *const *W, const float *const *b,
                                  const int32_t *act, int32_t compute,
                                  hpacml_model **out);

/* Frees a model.  NULL-safe.  Synchronise streams that use it first. */
void hpacml_model_destroy(hpacml_model *m);

/* ---- convolutional surrogates --------------------------------------------
 * The models the paper searches for image-shaped regions (Table IV:
 * MiniWeather's one or two convolution layers of 4-8 channels, ParticleFilter's
 * convolution, max-pool and fully connected layers) run on the composed input
 * tensor seen as S images: the last two sweep dimensions of the `to` map are
 * the image rows and columns (the counts must equal `height`, `width`), any
 * leading sweep dimensions number the images, and the map's features are the
 * channels.  The result, [S][rows'][columns'][channels'] in that order, is
 * written through the `from` map, whose points must number S * rows' *
 * columns' and whose features must equal channels'. */
enum { HPACML_LAYER_CONV2D = 0, HPACML_LAYER_MAXPOOL2D = 1, HPACML_LAYER_LINEAR = 2 };
/* convolution padding: VALID (none: the output shrinks by window - 1) or SAME
 * (the output keeps the input's size; floor((k-1)/2) rows/columns of padding
 * before, the rest after; stride must be 1) */
enum { HPACML_PAD_VALID = 0, HPACML_PAD_SAME = 1 };
/* what SAME padding reads outside the image: zeros, the opposite edge
 * (wrapping as often as needed), or the nearest edge element */
enum { HPACML_PADMODE_ZEROS = 0, HPACML_PADMODE_CIRCULAR = 1, HPACML_PADMODE_REPLICATE = 2 };

/* One layer of a convolutional model.
 *   CONV2D:    out[y][x][co] = b[co] + sum over ci, ky, kx of
 *              W[co][ci][ky][kx] * in[y*stride[0] + ky - pad_top][x*stride[1] + kx - pad_left][ci]
 *              (PyTorch Conv2d weights, cross-correlation); out_channels >= 1.
 *   MAXPOOL2D: out[y][x][c] = max over the kernel window at (y*stride[0], x*stride[1]),
 *              no padding, NaN when any window value is NaN; out_channels unused.
 *   LINEAR:    the image flattened in [row][column][channel] order, then
 *              out[o] = b[o] + sum_i W[o][i] in[i]; the result is a 1 x 1 image
 *              of out_channels channels.  Only LINEAR layers may follow a LINEAR.
 * `act` (HPACML_ACT_*) applies to every layer's output.  kernel and stride
 * entries are >= 1; VALID windows must fit the layer's input. */
typedef struct {
    int32_t kind;            /* HPACML_LAYER_* */
    int32_t out_channels;    /* CONV2D: output channels; LINEAR: outputs */
    int32_t kernel[2];       /* CONV2D / MAXPOOL2D window: rows, columns */
    int32_t stride[2];       /* CONV2D / MAXPOOL2D step: rows, columns */
    int32_t padding;         /* CONV2D: HPACML_PAD_* */
    int32_t pad_mode;        /* CONV2D with SAME: HPACML_PADMODE_* */
    int32_t act;             /* HPACML_ACT_* */
} hpacml_layer;

/* Checks a convolutional model description without touching any device.
 * in_channels: 1..HPACML_MAX_FEATURES; height, width >= 1; n_layers
 * 1..HPACML_MAX_LAYERS; every layer's channels (and a LINEAR layer's inputs)
 * <= HPACML_MAX_CNN_WIDTH.  On success writes the output image's rows, columns
 * and channels (out_shape[3], may be NULL).  Returns what hpacml_cnn_create
 * would return for the same arguments. */
hpacml_status hpacml_cnn_validate(int32_t in_channels, int32_t height, int32_t width, int32_t n_layers,
                                  const hpacml_layer *layers, int32_t *out_shape);

/* Number of weights and biases hpacml_cnn_create reads from W[l] and b[l]
 * for each layer of a convolutional model (w_counts[l], b_counts[l], both
 * [n_layers] arrays the caller owns; 0 and 0 for MAXPOOL2D).  Errors as
 * hpacml_cnn_validate; NULL count arrays: HPACML_E_INVAL.  No device work. */
hpacml_status hpacml_cnn_param_counts(int32_t in_channels, int32_t height, int32_t width, int32_t n_layers,
                                      const hpacml_layer *layers, int64_t *w_counts, int64_t *b_counts);

/* Creates a convolutional model for images of height x width x in_channels.
 *   layers: [n_layers], read during the call only.
 *   W[l], b[l]: HOST fp32 (CONV2D [out][in][kh][kw] and [out]; LINEAR
 *   [out][rows*columns*channels of its input] and [out]; MAXPOOL2D: NULL).
 *   compute: HPACML_F32.
 * Weights are copied to library-owned device memory.  hpacml_infer with such a
 * model either runs one fused kernel (convolution-only stacks of SAME, stride-1
 * layers of at most 16 channels whose padding modes are all CIRCULAR or none
 * CIRCULAR, on maps in the 32-bit form; when the `from` targets meet the `to`
 * targets, the inputs are first copied into the `to` map's snapshot record
 * and the kernel reads them there), or a layer-by-layer path through a
 * workspace that the model
 * owns (allocated on first need, grown as needed, freed with the model): two
 * tensors of S * (largest layer tensor) floats, plus the partial sums of fully
 * connected layers whose K is split over blocks (at most 32 * S * outputs
 * floats).  That path reads every input
 * before writing any output, so `from` targets may overlap `to` targets; calls
 * that share a model must not overlap in time on different streams.  Errors
 * as hpacml_cnn_validate, plus HPACML_E_NOMEM / HPACML_E_DEVICE. */
hpacml_status hpacml_cnn_create(int32_t in_channels, int32_t height, int32_t width, int32_t n_layers,
                                const hpacml_layer *layers, const float *const *W, const float *const *b,
                                int32_t compute, hpacml_model **out);

/* Inference mode of a region (Sec. III-C `ml(infer)`, Sec. IV-B): for every
 * sweep point, gather through `in` (a TO map), run the model, write the outputs
 * through `out` (a FROM map).  The result is that of gathering every point's
 * inputs before any output is written, also when `from` targets overlap `to`
 * targets (a region that updates its own fields in place):
 *   - where both maps address exactly the same element per point (same
 *     array and strides, zero offsets, same sweep), one fused pass;
 *   - any other overlap first copies the inputs, as hpacml_collect would,
 *     into a snapshot record of n_points * features(in) floats that the `in`
 *     map owns (allocated on first need, freed by hpacml_map_destroy), then
 *     runs the fused pass on that record.  Inferences that share an `in`
 *     map share its snapshot: such calls on different streams must not
 *     overlap in time.
 * Two `from` targets that can address one element are HPACML_E_ALIAS.
 * Requires
 * points(in) == points(out), features(in) == dims[0] and
 * features(out) == dims[n_layers] (HPACML_E_SHAPE).  Asynchronous on `stream`;
 * returns HPACML_E_DEVICE only for launch errors.  Zero points: HPACML_OK,
 * nothing launched. */
hpacml_status hpacml_infer(const hpacml_model *model, const hpacml_map *in,
                           const hpacml_map *out, void *stream);

/* Collect mode (Sec. III-A-2, Sec. IV-B): the values a map addresses, copied
 * bit for bit into dst[p * ld + f] for point p and feature f (a TO map records
 * a region's inputs; a FROM map, the outputs it addresses).  dst is a DEVICE
 * float buffer of n_points * ld elements; ld >= n_features.  Columns f >=
 * n_features are not written, so two calls with dst and dst + F_in record
 * input/output pairs in one buffer.  Asynchronous on `stream`. */
hpacml_status hpacml_collect(const hpacml_map *m, float *dst, int64_t ld, void *stream);

/* Collect mode for a region's two records at once (Sec. IV-B: the mapped
 * inputs and the outputs are stored as two datasets): the same result as
 * hpacml_collect(a, dst_a, ld_a) followed by hpacml_collect(b, dst_b, ld_b),
 * in one launch when both maps allow the library's 32-bit form (else two).
 * Each argument triple follows hpacml_collect's contract; in addition both
 * maps are on one device, neither record may overlap a target of either map,
 * and the two records must be disjoint: byte ranges that do not meet, or one
 * buffer of equal pitch with disjoint column ranges (dst_b = dst_a + F_a,
 * ld_a = ld_b >= F_a + F_b) -- anything else is HPACML_E_ALIAS.  Nothing is
 * enqueued when a check fails.  Asynchronous on `stream`. */
hpacml_status hpacml_collect_pair(const hpacml_map *a, float *dst_a, int64_t ld_a,
                                  const hpacml_map *b, float *dst_b, int64_t ld_b, void *stream);

/* ---- execution control and the collection sink ---------------------------
 * A region ties the `to` map, the `from` map and the model of one annotated
 * code block together with the `ml` clause's mode (Sec. III-C, Fig. 3:
 * `ml(infer | collect | predicated[:cond]) ... if(cond)`; Sec. IV-B):
 *   INFER      every invocation runs hpacml_infer;
 *   COLLECT    every invocation records the inputs through the `to` map, runs
 *              the accurate path (the region's original code), records the
 *              outputs through the `from` map and the accurate path's time;
 *   PREDICATED per invocation: `cond` nonzero -> INFER, zero -> COLLECT.
 * The `if` clause (`enabled` = 0) runs the accurate path alone: no inference,
 * no recording.  Records go to a sink of `capacity` samples in device memory
 * (one sample per collected invocation: inputs [points(in)][F_in], outputs
 * [points(out)][F_out], the accurate path's time), the datasets of one region
 * group in the paper's database (Sec. IV-B). */
enum { HPACML_MODE_INFER = 0, HPACML_MODE_COLLECT = 1, HPACML_MODE_PREDICATED = 2 };

/* The accurate path: the region's original code, which must enqueue its work
 * on `stream` (a hipStream_t) and return; called on the calling thread. */
typedef void (*hpacml_accurate_fn)(void *user, void *stream);

typedef struct hpacml_region_s hpacml_region;

/* Creates a region.  The maps and the model are borrowed (keep them alive
 * while the region is used); `in` is a TO map, `out` a FROM map, with the
 * shapes hpacml_infer requires of them and `model` (checked here: the status
 * hpacml_infer would return, without launching).  capacity >= 0 samples are
 * allocated up front on the current device (0 for INFER regions);
 * HPACML_E_NOMEM if they do not fit. */
hpacml_status hpacml_region_create(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out,
                                   int32_t mode, int64_t capacity, hpacml_region **region);

/* One invocation of the region on `stream`.  Collecting into a full sink
 * returns HPACML_E_RANGE before anything is enqueued or called; a collecting
 * invocation needs `accurate` (HPACML_E_INVAL when NULL), as does enabled == 0.
 * Asynchronous like hpacml_infer / hpacml_collect; the accurate path's time is
 * measured with events around the callback's work on `stream`. */
hpacml_status hpacml_region_run(hpacml_region *region, int32_t cond, int32_t enabled,
                                hpacml_accurate_fn accurate, void *user, void *stream);

/* Number of samples collected so far. */
hpacml_status hpacml_region_samples(const hpacml_region *region, int64_t *n_samples);

/* Copies the first n samples to HOST buffers (any may be NULL):
 * inputs [n][points(in)][F_in], outputs [n][points(out)][F_out], times_ms [n].
 * Waits until the records of those samples are complete, on whatever stream
 * each was collected (an event recorded after each sample's output record),
 * then copies.  n > samples collected: HPACML_E_RANGE. */
hpacml_status hpacml_region_read(const hpacml_region *region, int64_t n, float *inputs, float *outputs,
                                 float *times_ms);

/* Writes the collected samples as one region group of the database: the
 * directory `dir`/`name`/ with inputs.npy [n][points(in)][F_in], outputs.npy
 * [n][points(out)][F_out] and time.npy [n] (milliseconds), NumPy's .npy format
 * (float32, C order), the outer dimension numbering the samples.  Creates the
 * two directories if needed.  HPACML_E_INVAL for an unwritable path. */
hpacml_status hpacml_region_save(const hpacml_region *region, const char *dir, const char *name);

/* Forgets the collected samples (the sink is reused from sample 0). */
hpacml_status hpacml_region_reset(hpacml_region *region);

/* Frees a region and its sink (not its maps or model).  NULL-safe.
 * Synchronise the streams that use it first. */
void hpacml_region_destroy(hpacml_region *region);

/* ---- inference without allocation ---------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.
 *
 * hpacml_infer_noalloc computes exactly what hpacml_infer computes, with the
 * same kernels, and allocates nothing (no hipMalloc / hipFree, no host heap),
 * except where hpacml_infer runs a multilayer perceptron layer by layer (it
 * needs a workspace): there this entry point runs the general fused kernel,
 * which has the same rounding points and another summation order.
 * Where hpacml_infer would copy the inputs into the `to` map's snapshot
 * record first (outputs that may overwrite inputs other points still read),
 * this entry point puts that record in a fixed scratch array of
 * HPACML_NOALLOC_SCRATCH_BYTES per device, held until the process ends.
 *   HPACML_E_RANGE        the record (points x F_in x 4 bytes) is larger than
 *                         the scratch array; nothing is enqueued.
 *   HPACML_E_UNSUPPORTED  convolutional models, and in-place inferences whose
 *                         maps or model take the general kernel (they need
 *                         device tables of their own).
 * Other statuses as hpacml_infer.  Asynchronous on `stream`.  Every call on
 * one device shares that device's scratch array: calls that overlap on one
 * device (on different streams) race; calls ordered on one stream do not.
 * The array keeps the last call's record, and every call overwrites the part
 * it reads before reading it. */
#define HPACML_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
hpacml_status hpacml_infer_noalloc(const hpacml_model *model, const hpacml_map *in,
                                   const hpacml_map *out, void *stream);

/* Name of the kernel hpacml_infer would launch for these handles (a static
 * string, prefixed "snapshot+" when the inputs are copied first; the
 * layer-by-layer path is "mlp_layers_f32" / "mlp_layers_bf16"), or NULL when
 * the arguments are invalid.  Allocates no device buffer; for a model that
 * runs layer by layer it selects the matmul library's algorithms for this
 * point count (host work, cached with the model). */
const char *hpacml_infer_variant(const hpacml_model *model, const hpacml_map *in,
                                 const hpacml_map *out);

/* Static, human-readable text of a status. */
const char *hpacml_status_string(hpacml_status s);

/* HPACML_ABI_VERSION of the built library. */
int32_t hpacml_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* HPACML_H */
