/*
 * flexserve.h -- C ABI of the MI355X ensemble-inference library.
 *
 * The operation (FlexServe, Fig. 1 caption and Sec. 2.2): N image
 * classification models are loaded into one device memory; a request's batch
 * of images is transformed ONCE (bilinear resize + mean/std normalisation)
 * and that one tensor feeds every model; the batch size varies per request
 * (Sec. 2.3); the outputs of all models are returned together, per model
 * and per image, together with a combined result (Fig. 1 caption; Sec. 2.1
 * on combining ensemble outputs).
 *
 * Conventions for every entry point:
 *  - The caller owns every host buffer.  fs_ensemble_create deep-copies and
 *    converts the weights; the caller may free them when it returns.  The
 *    library owns all device memory of an ensemble until fs_destroy.
 *  - No exception, abort or print crosses the ABI.  Each failure returns a
 *    status and sets a message readable with fs_last_error.
 *  - Arguments are validated on the host before any device work; an invalid
 *    call leaves the handle usable.
 *  - Calls on one handle are serialised by an internal lock; distinct
 *    handles are independent.
 *  - Layouts are row-major.  Activations are NHWC.  Outputs are model-major:
 *    probs[i][b][c] is model i, image b, class c.
 */
#ifndef FLEXSERVE_H
#define FLEXSERVE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct fs_ensemble fs_ensemble; /* opaque */

typedef enum {
    FS_OK = 0,
    FS_ERR_INVALID = 1,     /* bad argument, descriptor or shape          */
    FS_ERR_OOM = 2,         /* device or pinned host allocation failed    */
    FS_ERR_DEVICE = 3,      /* no such device, or a HIP runtime failure   */
    FS_ERR_UNSUPPORTED = 4, /* well-formed but outside what is supported  */
    FS_ERR_INTERNAL = 5
} fs_status;

typedef enum { FS_F32 = 0, FS_BF16 = 1 } fs_precision; /* storage type of the whole ensemble */
typedef enum { FS_OP_CONV = 0, FS_OP_MAXPOOL = 1, FS_OP_GAP = 2, FS_OP_FC = 3 } fs_op;
/* How vote[b] combines the models' outputs for image b (Sec. 2.1: outputs
 * are combined according to the consumer's policy).
 *   FS_COMBINE_MEAN       the smallest class maximising sum_i probs[i][b][c]
 *                         (the argmax of the mean probability)
 *   FS_COMBINE_PLURALITY  the class that is top-1 of the most models; among
 *                         classes with equally many, the smallest
 *   FS_COMBINE_ANY        sensitivity policy for one designated class c*:
 *                         model i detects c* when its top-1 class is c*;
 *                         vote[b] = 1 when at least k models detect it,
 *                         else 0.  k = 1 is the maximum-sensitivity OR of
 *                         the models' binary outputs (Sec. 2.1); k = N the
 *                         AND.  Set with fs_set_combine. */
typedef enum { FS_COMBINE_MEAN = 0, FS_COMBINE_PLURALITY = 1, FS_COMBINE_ANY = 2 } fs_combine;

/* One layer, listed in topological order.  Layer outputs are referred to by
 * index; src = -1 is the shared transformed input batch (3 channels). */
typedef struct {
    int32_t op;            /* fs_op */
    int32_t src;           /* producer of the input, -1 = transformed batch */
    int32_t residual_src;  /* conv: layer added before the ReLU, or -1      */
    int32_t cin, cout;     /* conv/fc channels (fc: in/out features)        */
    int32_t kh, kw;        /* conv kernel, maxpool window                   */
    int32_t stride, pad;   /* conv / maxpool                                */
    int32_t relu;          /* conv/fc: apply max(0, .) after bias+residual  */
    int32_t flatten_nchw;  /* fc: the input map is flattened channel-major  */
    const float *weight;   /* conv [cout][kh][kw][cin]; fc [cout][cin]      */
    const float *bias;     /* [cout] or NULL (= 0)                          */
    const float *bn_scale; /* conv: [cout] or NULL; w' = w*scale            */
    const float *bn_shift; /* conv: [cout] or NULL; bias' = shift           */
} fs_layer;

typedef struct {
    int32_t num_layers;
    const fs_layer *layers;
    int32_t num_classes; /* cout of the last layer, equal for all models */
} fs_model_spec;

/* The single data transformation shared by every model (Fig. 1 caption):
 * bilinear resize (half-pixel centres, no antialias) to out_h x out_w, then
 * (v/255 - mean[c]) / std[c] per RGB channel. */
typedef struct {
    int32_t out_h, out_w;
    float mean[3];
    float std[3];
} fs_preprocess;

typedef struct {
    int32_t num_models;
    const fs_model_spec *models;
    fs_preprocess pre;
    int32_t precision;  /* fs_precision */
    int32_t combine;    /* fs_combine: MEAN or PLURALITY (ANY needs fs_set_combine) */
    int32_t max_batch;  /* largest batch one device pass handles (1..4096) */
    int32_t device;     /* HIP device ordinal */
} fs_ensemble_desc;

/* A host image: uint8 HWC RGB, h rows of row_stride bytes (>= 3*w),
 * 1 <= h, w <= 32768. */
typedef struct {
    const uint8_t *data;
    int32_t h, w, row_stride;
} fs_image;

/* A device-resident image: offset (bytes) into a packed uint8 buffer; the
 * caller guarantees 1 <= h, w <= 32768, row_stride >= 3*w and that all
 * h*row_stride bytes lie inside the buffer (the device path reads them
 * without a host-side check). */
typedef struct {
    uint64_t offset;
    int32_t h, w, row_stride, reserved;
} fs_image_desc;

/* Create an ensemble: validate every model, fold batch norm, convert and
 * pack the weights, plan every layer for max_batch, allocate one weight
 * arena and one activation workspace on `device`, upload.
 * Errors: FS_ERR_INVALID (NULL, inconsistent shapes, unequal class counts),
 * FS_ERR_UNSUPPORTED (channel counts the kernels do not handle),
 * FS_ERR_DEVICE (no such device), FS_ERR_OOM. *out is NULL on failure. */
fs_status fs_ensemble_create(const fs_ensemble_desc *desc, fs_ensemble **out);

/* A second handle on the same ensemble (Sec. 2.2: several server workers
 * serve one set of models): it shares src's device weights (no copy; they
 * are freed with the last handle that uses them) and the plan, and has its
 * own activation workspace, stream, lock, recorded graphs and combine
 * policy, so calls on the two handles run concurrently.  src is not
 * modified.  Errors: FS_ERR_INVALID (NULL), FS_ERR_DEVICE, FS_ERR_OOM; *out
 * is NULL on failure. */
fs_status fs_ensemble_share(fs_ensemble *src, fs_ensemble **out);

/* Ensemble inference over a batch of B host images of any sizes (Sec. 2.3),
 * synchronous.  B == 0 is a no-op.  B > max_batch is processed in chunks.
 *   probs      [N][B][C] fp32, required
 *   mean_probs [B][C]    fp32, optional (NULL)
 *   vote       [B]       int32, required: the combined result of the current
 *                         policy (fs_combine; by default the smallest c
 *                         maximising sum_i probs[i][b][c])
 *   top1       [N][B]    int32, optional: smallest c maximising model i's logits
 *   logits     [N][B][C] fp32, optional */
fs_status fs_infer(fs_ensemble *e, const fs_image *imgs, int32_t B,
                   float *probs, float *mean_probs, int32_t *vote, int32_t *top1,
                   float *logits);

/* The same pass on device-resident data, asynchronous on `stream`
 * (a hipStream_t; NULL = the ensemble's own stream).  d_pixels holds the
 * packed uint8 images, d_desc[B] their descriptors; every output is a
 * device pointer with the layout of fs_infer (optional ones may be NULL).
 * Requires 1 <= B <= max_batch.  Nothing is copied to or from the host.
 * The passes of one handle share its workspace, so they never overlap: a
 * call on another stream than the handle's previous pass (fs_infer's
 * included) makes its stream wait, on the device, for that pass to end.
 * For passes that run concurrently use handles from fs_ensemble_share. */
fs_status fs_infer_device(fs_ensemble *e, const uint8_t *d_pixels,
                          const fs_image_desc *d_desc, int32_t B,
                          float *d_probs, float *d_mean_probs, int32_t *d_vote,
                          int32_t *d_top1, float *d_logits, void *stream);

/* HIP graphs for the pass (off by default).  With enable = 1, fs_infer and
 * fs_infer_device record the pass's kernel launches the first time a batch
 * size meets a set of buffers on a stream and replay them with one launch
 * from then on (one graph per exact batch size).  Off, every kernel is
 * launched from the host; the host then stays far ahead of the device
 * (25 launches against a pass of 0.27 ms or more for three ResNet-18s), and
 * replay measured 0.7-2 % slower per pass at every batch size from 1 to 32,
 * so graphs are for callers that need one launch per pass.  The pass runs
 * eagerly while the profiler is on and on the legacy default stream.
 * enable = 0 drops the recorded passes.  Synchronises the ensemble's
 * stream.  FS_ERR_INVALID for a NULL handle. */
fs_status fs_graphs_enable(fs_ensemble *e, int32_t enable);

/* Combine policy of the following fs_infer / fs_infer_device calls
 * (fs_combine).  positive_class (0 <= c* < num_classes) and min_votes
 * (1 <= k <= num_models) are read for FS_COMBINE_ANY only.  probs, mean and
 * top1 do not depend on the policy.  Synchronises the ensemble's stream and
 * drops its recorded graphs.  FS_ERR_INVALID for a NULL handle, an unknown
 * policy or parameters out of range; FS_ERR_UNSUPPORTED for PLURALITY with
 * more than 64 models. */
fs_status fs_set_combine(fs_ensemble *e, int32_t policy, int32_t positive_class, int32_t min_votes);

void fs_destroy(fs_ensemble *e); /* NULL-safe; waits for outstanding work */

/* Request coalescing (Sec. 2.3: batches of any size per request).  A
 * batcher serves fs_batcher_infer calls from any number of threads with one
 * worker thread per handle in handles[0..n_handles) (1..16 handles of one
 * ensemble: the first and handles shared from it with fs_ensemble_share).
 * One worker at a time gathers: it takes queued requests whole, in arrival
 * order, up to max_batch images per pass (a larger request runs alone,
 * chunked by fs_infer), waiting up to max_wait_us after the first for
 * others to arrive, and runs them as one fs_infer on its handle while the
 * next worker gathers.  fs_batcher_infer has the arguments and output
 * layout of fs_infer for its own B images and blocks until they are done;
 * the caller's buffers must stay valid until it returns.  Each image's
 * result is that of fs_infer on the same images in a batch of the pass's
 * size.  The handles must outlive the batcher and may still be used
 * directly.  FS_ERR_INVALID for NULL, n_handles outside 1..16, a negative
 * wait, or handles whose models, classes, max_batch or weights differ.
 * Errors are returned per call; their message is fs_batcher_last_error() of
 * the calling thread. */
typedef struct fs_batcher fs_batcher;
fs_status fs_batcher_create(fs_ensemble *const *handles, int32_t n_handles, int32_t max_wait_us,
                            fs_batcher **out);
fs_status fs_batcher_infer(fs_batcher *b, const fs_image *imgs, int32_t B, float *probs,
                           float *mean_probs, int32_t *vote, int32_t *top1, float *logits);
/* Passes run, requests served and images served so far. */
fs_status fs_batcher_stats(fs_batcher *b, int64_t *passes, int64_t *requests, int64_t *images);
const char *fs_batcher_last_error(void);
/* NULL-safe.  Serves the queued requests first, then returns once every
 * caller whose request was served has left fs_batcher_infer; no
 * fs_batcher_infer call may begin once fs_batcher_destroy has begun. */
void fs_batcher_destroy(fs_batcher *b);

/* Last error message of handle e, or of this thread's last failed create
 * when e is NULL.  Valid until the next call on the same handle/thread. */
const char *fs_last_error(const fs_ensemble *e);

typedef struct {
    int32_t num_models, num_classes, max_batch, precision;
    int32_t num_groups;          /* launches per layer are shared by a group */
    int32_t launches_per_pass;   /* kernel launches of one device pass at max_batch */
    int64_t weight_bytes;        /* device weight arena */
    int64_t workspace_bytes;     /* device activations + scratch */
    double flops_per_image;      /* 2 * multiply-accumulates of all models */
} fs_info;
fs_status fs_query(const fs_ensemble *e, fs_info *info);

/* Per-kernel-class timing with HIP events on the launch stream.  While
 * enabled, every launch of fs_infer/fs_infer_device is bracketed by two
 * events.  fs_profile_read synchronises the stream and returns, per class,
 * the launch count, summed event time and algorithmic FLOP/bytes. */
typedef struct {
    char name[32];
    int64_t launches;
    double total_ms;
    double flops;
    double bytes;
} fs_kernel_stat;
fs_status fs_profile_enable(fs_ensemble *e, int32_t enable); /* (re)starts, clearing */
fs_status fs_profile_read(fs_ensemble *e, fs_kernel_stat *stats, int32_t max_stats,
                          int32_t *n_stats);

/* The individual launches recorded since fs_profile_enable, in order (up to
 * max_out): kernel class and variant, group/layer of the plan (-1 outside
 * the layer list), GEMM shape M x N x K of conv/fc, models per launch Z, event
 * time and algorithmic FLOP/bytes.  Synchronises like fs_profile_read. */
typedef struct {
    char kclass[16];
    char kernel[32];
    int32_t group, layer, M, N, K, Z;
    double ms;
    double flops;
    double bytes;
} fs_launch_stat;
fs_status fs_profile_launches(fs_ensemble *e, fs_launch_stat *out, int32_t max_out,
                              int32_t *n_out);

/* The tile tuner's record: one text line per timed candidate (batch
 * bucket, group, layer, GEMM shape M N K, models Z, K split, tile name, mean
 * time of one launch in us) and one "choice" line per timed layer (its
 * shape key and the tile kept), for every bucket planned so far.  Tiles
 * come from a committed table of such choices per layer shape and batch
 * bucket; only layers the table lacks are timed (environment FS_TUNE=1:
 * time every layer, FS_TUNE=3: time every layer with the table's tile kept
 * unless another wins by 3 %, FS_TUNE=0: never time, the shape rule
 * instead).  Copies at
 * most n - 1 bytes and a terminating zero into buf (when buf is not NULL and
 * n > 0); *needed (if not NULL) receives the full length + 1.
 * FS_ERR_INVALID for a NULL handle. */
fs_status fs_tuning_log(fs_ensemble *e, char *buf, int64_t n, int64_t *needed);

/* Host-side time of the phases of the handle's last fs_infer, in ms,
 * summed over its chunks: ms[0] copying the images into pinned staging
 * memory and issuing their upload, ms[1] issuing the device pass, ms[2]
 * issuing the result downloads, ms[3] waiting for the stream (the device
 * work that has not finished by then), ms[4] copying the results into the
 * caller's buffers.  FS_ERR_INVALID for NULL arguments. */
fs_status fs_infer_phases(fs_ensemble *e, double *ms);

/* ---- test-only: one image's stored layer outputs, for layer-by-layer
 * parity (each layer's stored input fed to a reference of that layer alone).
 * fs_debug_capture(e, image) arms the following passes of e: after every
 * layer's launch, the stored output of image `image` of that layer, for
 * every model, is copied into a capture buffer of the handle (allocated
 * here), as is the image's transformed input; those passes run without
 * graphs.  image = -1 disarms and frees the buffer.  FS_ERR_INVALID when
 * image is outside -1..max_batch-1.
 * fs_debug_layer(e, model, layer, out, n) copies, widened to fp32, what the
 * last pass captured of model `model`'s layer `layer` (index in its
 * fs_model_spec) into out: n = H*W*C floats in NHWC order (features for an
 * FC or average pool, fp32 logits for the last layer); layer = -1 gives the
 * transformed input, n = out_h*out_w*3.  FS_ERR_UNSUPPORTED for a layer
 * whose output is never stored (a conv whose max pool or average pool is
 * fused into its launch; the pooled tensor is stored under the pool's
 * index) or that the last pass did not capture (image >= its B).
 * Synchronises the handle's passes. */
fs_status fs_debug_capture(fs_ensemble *e, int32_t image);
fs_status fs_debug_layer(fs_ensemble *e, int32_t model, int32_t layer, float *out, int64_t n);

/* ---- single-kernel entry points on host tensors (synchronous; for parity
 * tests).  precision selects fp32 or bf16 storage; in bf16 the inputs must
 * already be bf16-representable and outputs are returned widened to fp32. */

/* The shared transformation of B host images.  layout 0: out
 * [B][out_h][out_w][4] (channel 3 is zero padding); layout 1 (bf16, even
 * sizes): the space-to-depth form [B][out_h/2][out_w/2][16] whose channel
 * (sy*2 + sx)*3 + c holds pixel (2Y + sy, 2X + sx), channel c (12..15 zero). */
fs_status fs_test_preprocess(const fs_image *imgs, int32_t B, int32_t out_h, int32_t out_w,
                             const float mean[3], const float std_[3], int32_t precision,
                             int32_t layout, float *out, int32_t device);

/* Convolution with fused epilogue: out = relu?(conv(in, w) + bias + res).
 * in [B][H][W][Cin], w [Cout][kh][kw][Cin], bias [Cout] or NULL,
 * res [B][Ho][Wo][Cout] or NULL, out [B][Ho][Wo][Cout].  tile = -1 picks
 * the tile the planner would, otherwise forces tile configuration `tile`. */
fs_status fs_test_conv(const float *in, int32_t B, int32_t H, int32_t W, int32_t Cin,
                       const float *w, const float *bias, const float *res, int32_t Cout,
                       int32_t kh, int32_t kw, int32_t stride, int32_t pad, int32_t relu,
                       int32_t precision, int32_t tile, float *out, int32_t device);

/* The ResNet stem as the ensemble runs it in bf16: conv 7x7 / stride 2 /
 * pad 3 from 3 channels to 64 (in its space-to-depth form), + bias, ReLU,
 * bf16 rounding, then max pool 3x3 / stride 2 / pad 1 (He et al., the
 * ResNet stem; the paper's models are such CNNs, Sec. 2.2), in one kernel.
 * in [B][H][W][3] (H, W even), w [64][7][7][3], bias [64] or NULL,
 * out [B][Hp][Wp][64] with Ho = H/2, Hp = (Ho - 1)/2 + 1 (likewise W).
 * FS_ERR_UNSUPPORTED when the shape is not one the fused kernel takes
 * (conv output wider than 112). */
fs_status fs_test_stem_pool(const float *in, int32_t B, int32_t H, int32_t W, const float *w,
                            const float *bias, float *out, int32_t device);

fs_status fs_test_maxpool(const float *in, int32_t B, int32_t H, int32_t W, int32_t C,
                          int32_t k, int32_t stride, int32_t pad, int32_t precision,
                          float *out, int32_t device);

fs_status fs_test_gap(const float *in, int32_t B, int32_t H, int32_t W, int32_t C,
                      int32_t precision, float *out, int32_t device);

/* out [B][N] = relu?(in [B][K] . w[N][K]^T + bias); out_precision selects
 * an fp32 (final logits) or a storage-type output. */
fs_status fs_test_fc(const float *in, int32_t B, int32_t K, const float *w, const float *bias,
                     int32_t N, int32_t relu, int32_t precision, int32_t out_storage,
                     float *out, int32_t device);

/* Softmax per (model, image) row of logits [N][B][C] and the combination:
 * probs [N][B][C], mean [B][C] (optional), vote [B], top1 [N][B] (optional). */
fs_status fs_test_softmax_combine(const float *logits, int32_t N, int32_t B, int32_t C,
                                  float *probs, float *mean, int32_t *vote, int32_t *top1,
                                  int32_t device);
/* The same with a combine policy and its parameters (see fs_set_combine). */
fs_status fs_test_softmax_combine_policy(const float *logits, int32_t N, int32_t B, int32_t C,
                                         int32_t policy, int32_t positive_class, int32_t min_votes,
                                         float *probs, float *mean, int32_t *vote, int32_t *top1,
                                         int32_t device);

/* Measurement of one convolution layer shape: Z models' weights, one
 * shared input filled with a constant, `iters` back-to-back launches of tile
 * configuration `tile` (-1 = the planner's choice, reported in *tile_used),
 * timed with HIP events; *avg_ms is the mean time of one launch.  Used to
 * choose and evidence tile configurations per batch size. */
fs_status fs_bench_conv(int32_t B, int32_t H, int32_t W, int32_t Cin, int32_t Cout, int32_t kh,
                        int32_t kw, int32_t stride, int32_t pad, int32_t relu, int32_t residual,
                        int32_t precision, int32_t tile, int32_t Z, int32_t iters, double *avg_ms,
                        int32_t *tile_used, int32_t device);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): one bf16
 * convolution on device-resident tensors, computed by the kernels and the
 * tile and split-K rule fs_test_conv uses with tile = -1 (same bits).  It
 * calls no allocating routine: the split-K partial sums go to a
 * library-static device array of FS_NOALLOC_SCRATCH_BYTES per GPU (each GPU
 * the library runs on holds it until the process ends).  Every call on one
 * GPU shares that array, so calls that overlap on one GPU (concurrent
 * streams, several threads) race; calls issued on one stream are ordered.
 * Runs on the current device, asynchronously on `stream` (a hipStream_t,
 * NULL = the null stream).
 *   d_in   [B][H][W][Cin] bf16, Cin a multiple of 64
 *   d_w    [Cout][kh][kw][Cin] bf16, Cout a multiple of 8
 *   d_bias [Cout] fp32, required
 *   d_res  [B][Ho][Wo][Cout] bf16 added before the ReLU, or NULL
 *   d_out  [B][Ho][Wo][Cout] bf16 = bf16(relu?(conv + bias + res))
 * FS_ERR_INVALID for NULL or inconsistent arguments; FS_ERR_UNSUPPORTED
 * for channel counts outside the above, tensors of 2 GiB or more, or a
 * shape whose partial sums exceed the scratch array. */
#define FS_NOALLOC_SCRATCH_BYTES (16 << 20)
fs_status fs_conv_bf16_device_noalloc(const void *d_in, int32_t B, int32_t H, int32_t W, int32_t Cin,
                                      const void *d_w, const float *d_bias, const void *d_res,
                                      int32_t Cout, int32_t kh, int32_t kw, int32_t stride,
                                      int32_t pad, int32_t relu, void *d_out, void *stream);

/* Number of conv tile configurations fs_test_conv accepts (0..n-1) for a
 * precision, and the name of tile t (NULL when out of range). */
int32_t fs_conv_num_tiles(int32_t precision);
const char *fs_conv_tile_name(int32_t precision, int32_t tile);

#ifdef __cplusplus
}
#endif
#endif /* FLEXSERVE_H */
