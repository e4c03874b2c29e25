/*
 * sscater.h -- C ABI of the MI355X (gfx950) delta-scatter convolution library.
 *
 * The library keeps, per handle, the persistent state of a stack of 3x3
 * convolution layers over a bird's-eye-view pillar grid and advances it one
 * sliding-window stride at a time, touching only the cells that changed.
 * This is the SSCATeR method (arXiv 2512.08557):
 *
 *   - input change map: a grid cell is "changed" when its pillar feature
 *     vector differs from the previous window (Sec. III-B; Alg. 1, PFN part).
 *     Here the comparison is bitwise on the stored feature vectors; a missing
 *     pillar is an all-zero vector.
 *   - delta scatter: each changed input site scatters
 *     (I_curr - I_prev) x W[m,n] into the persistent output at
 *     (i - m + floor(k/2), j - n + floor(k/2))  (Eq. 2, Sec. III-D; it fuses
 *     the deconvolution of Eq. 1 with the convolution).  For stride 2 the
 *     target is the downsampled site ((i-m+1)/2, (j-n+1)/2) when integral.
 *   - change-map propagation: every output site touched by that scatter is
 *     marked changed, including sites that the ReLU sends to zero, and for
 *     stride 2 the downsampled sites under a changed site
 *     (Alg. 1, backbone part; Sec. III-D, ReLU paragraph).  The next layer's
 *     input delta at a marked site is phi(Z_new) - phi(Z_old).
 *
 * The result after every stride equals recomputing each layer's convolution
 * from scratch on the whole window (abstract; Sec. IV-G), up to floating-point
 * summation order.
 *
 * Conventions
 *   - grid: H rows by W columns, cell index p = r*W + c; all maps are NHWC
 *     (a cell's channels are contiguous).
 *   - each layer: 3x3 kernel, zero padding 1, stride 1 or 2, output extent
 *     (n - 1)/stride + 1 per axis; weights OIHW; no bias; optional ReLU.
 *   - dtype SSCATER_F32: fp32 features, weights, maps and accumulation.
 *     dtype SSCATER_BF16: bf16 features, weights and layer outputs (round to
 *     nearest even), fp32 accumulation and fp32 pre-activation maps.
 *   - all device pointers are HIP device memory of the calling process.
 *
 * Streams: a handle is used with one HIP stream at a time (pass the
 * hipStream_t as a void*, NULL = the null stream).  Calls only enqueue work on
 * that stream and return; the exceptions, which synchronise the stream, are
 * sscater_changed and sscater_stats.  Different handles are independent and
 * may run concurrently on different streams.
 *
 * Errors: every call returns 0 or a negative SSCATER_E_* code, never throws.
 * Device-side input faults (a cell index outside the grid, a duplicate
 * index within one stride, a list passed as sorted that does not increase,
 * or in points mode a pillar over its point capacity) set a sticky flag
 * reported as SSCATER_E_DEVICE by
 * the next call that finds it set after the offending stride has executed;
 * sscater_reset clears it.
 */
#ifndef SSCATER_H
#define SSCATER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SSCATER_MAX_LAYERS 32
#define SSCATER_MAX_UPSAMPLERS 4

enum {
    SSCATER_OK = 0,
    SSCATER_E_INVALID_ARG = -1,   /* null pointer, unsupported shape, broken layer chain, bad index */
    SSCATER_E_OUT_OF_MEMORY = -2, /* device or host allocation failed */
    SSCATER_E_HIP = -3,           /* HIP runtime error (text via sscater_strerror) */
    SSCATER_E_OVERFLOW = -4,      /* more pillars than max_pillars: no sampling, the stride is refused */
    SSCATER_E_DEVICE = -5,        /* sticky device-side input fault (see above) */
    SSCATER_E_SCRATCH = -6        /* the grid is larger than the fixed scratch of an allocation-free call */
};

typedef enum { SSCATER_F32 = 0, SSCATER_BF16 = 1 } sscater_dtype;

/* Input grid: H rows, W columns, each below 32768 and H*W at most 2^30.
 * C0 is the pillar feature width (C0 * element size a power of two between 16
 * and 1024 bytes).  max_pillars bounds the pillar count of one stride (the
 * paper's pillar budget P with an assertion instead of random sampling,
 * Sec. III-B). */
typedef struct {
    int32_t H, W, C0, max_pillars;
    int32_t dtype; /* sscater_dtype */
} sscater_grid;

/* One convolution layer.  k must be 3 and pad 1; stride 1 or 2; relu 0 or 1.
 * cin must equal the previous layer's cout (C0 for the first layer). */
typedef struct {
    int32_t cin, cout, k, stride, pad, relu;
} sscater_layer;

/* One upsampler of the neck (Sec. III-B, backbone paragraph: every block is
 * upsampled and the results are concatenated; Alg. 1, deconvolution branch):
 * a transposed convolution with kernel = stride (1, 2 or 4, no padding) on the
 * output Y of backbone layer src_layer (1-based), then ReLU if relu = 1.
 * Output cell (s*i + a, s*j + b) takes exactly input cell (i, j) times
 * W[:, :, a, b].  All upsamplers of a handle must map onto one grid; their
 * outputs are concatenated along the channels in order (the neck map). */
typedef struct {
    int32_t src_layer, cout, stride, relu;
} sscater_upsampler;

/* One stride's pillars (the full occupied set of the window).
 *   idx   : device int32[count], cell indices r*W + c, unique within the call;
 *           NULL with count == H*W selects dense mode: feats is then the whole
 *           [H][W][C0] canvas.  NULL with count == 0 is an empty window (every
 *           pillar vanished); feats may then be NULL too.
 *   feats : device [count][C0] in the grid dtype (fp32, or bf16 bit patterns).
 * Both buffers must stay valid until the stream has executed the step. */
typedef struct {
    const int32_t* idx;
    const void* feats;
    int32_t count;
} sscater_pillars;

/* Points mode: the incremental pillar feature net in front of the layers
 * (Sec. III-B; Alg. 1, PFN part).  The handle keeps, per grid cell (pillar),
 * a queue of the points of the last `window` strides:
 *   x_min, y_min : metric position of the grid corner; cell (r, c) holds the
 *                  points with c = floor((x - x_min) * inv_res) and
 *                  r = floor((y - y_min) * inv_res), inv_res = 1/res rounded to
 *                  float32 and every operation in float32; points with
 *                  0 <= those < W (resp. H) are in the grid, all others
 *                  (NaN included) are ignored;
 *   res          : pillar edge (same unit as the points), > 0;
 *   max_points   : N, points a pillar may hold at once (1..128; the paper's
 *                  100).  More is a device-side input fault (SSCATER_E_DEVICE,
 *                  no sampling);
 *   window       : strides a point stays in the window (1..64; 10 strides of
 *                  10 ms = 100 ms);
 *   max_new_points : most points one stride may bring (sizes the queues'
 *                  bookkeeping; a larger stride is refused with
 *                  SSCATER_E_OVERFLOW).
 * A pillar's features are max over its points of ReLU(w . d), d the point's
 * D = 9 decorated values (x, y, z, intensity, x and y offsets from the pillar
 * centre, x, y and z offsets from the mean of the pillar's points) and w the
 * caller's [C0][9] weights (batch norm folded in, no bias).  A pillar is
 * changed when a point enters or leaves it (event based, Alg. 1). */
typedef struct {
    float x_min, y_min, res;
    int32_t max_points, window, max_new_points;
} sscater_pfn;

/* Counters of the last stride and running totals since create/reset. */
typedef struct {
    int32_t n_layers;
    int32_t pillars;                        /* pillar count of the last stride (points mode: its points) */
    int64_t steps;                          /* strides since create/reset */
    int64_t active[SSCATER_MAX_LAYERS + 1]; /* |A_l| of the last stride, l = 0..L */
    int64_t pairs[SSCATER_MAX_LAYERS + 1];  /* (input cell, output cell) pairs of layer l = 1..L */
    int64_t active_total[SSCATER_MAX_LAYERS + 1]; /* sums over all strides since create/reset */
    int64_t pairs_total[SSCATER_MAX_LAYERS + 1];
    double flops;                           /* algorithmic flops of the last stride: sum over layers and
                                               upsamplers of 2*cin*cout*pairs */
    double bytes;                           /* algorithmic HBM bytes of the last stride */
    int32_t n_ups;                          /* upsamplers of the neck */
    int64_t up_pairs[SSCATER_MAX_UPSAMPLERS]; /* (input cell, output cell) pairs of upsampler u in the last
                                                 stride: stride^2 per changed source cell */
} sscater_stats_t;

typedef struct sscater* sscater_t;

/* Create a handle on the current HIP device.
 *   grid, layers[n_layers] : shapes as above (1 <= n_layers <= SSCATER_MAX_LAYERS).
 *   weights[l] : host pointer to layer l's OIHW weights [cout][cin][3][3] in the
 *                grid dtype; copied and repacked, so the caller may free them
 *                on return.
 * All state (input canvas, per-layer pre-activation maps, change lists, change
 * stamps, delta buffers) is allocated here, sized for the worst case; no later
 * call allocates.  The maps start at zero (an empty window). */
int sscater_create(const sscater_grid* grid, const sscater_layer* layers, int32_t n_layers,
                   const void* const* weights, sscater_t* out);

/* sscater_create with a neck: n_ups (0..SSCATER_MAX_UPSAMPLERS) upsamplers
 * ups[u] with host weights up_weights[u] laid out [cin][cout][s][s] (the
 * PyTorch ConvTranspose2d layout) in the grid dtype, copied and repacked.  The
 * neck map is layer n_layers + 1 for sscater_read and sscater_changed; its
 * change set is the union of the upsampled change sets of the source layers.
 * Errors as sscater_create, plus SSCATER_E_INVALID_ARG for a source layer out
 * of range, an unsupported (cin, cout, stride) or upsamplers that do not share
 * one output grid. */
int sscater_create_neck(const sscater_grid* grid, const sscater_layer* layers, int32_t n_layers,
                        const void* const* weights, const sscater_upsampler* ups, int32_t n_ups,
                        const void* const* up_weights, sscater_t* out);

/* A handle over a batch of `batch` independent images of one grid (several
 * sensor streams advanced together by one launch chain): as sscater_create,
 * with cell index b * H * W + r * W + c for image b (pillar indices, change
 * lists and maps alike; every map is [batch][H_l][W_l][C_l]); no convolution
 * neighbourhood crosses an image boundary, so each image's results equal those
 * of a handle of its own.  max_pillars bounds the pillars of all images
 * together; H * W * batch at most 2^30.  No neck.  Errors as sscater_create,
 * plus SSCATER_E_INVALID_ARG for batch < 1. */
int sscater_create_batched(const sscater_grid* grid, int32_t batch, const sscater_layer* layers, int32_t n_layers,
                           const void* const* weights, sscater_t* out);

/* A handle in points mode (see sscater_pfn): layers and weights as for
 * sscater_create, C0 <= 64, pfn_weights the host [C0][9] fp32 weights of the
 * pointwise linear layer (copied).  Strides are then given as points with
 * sscater_step_points; sscater_step is refused.  Layer 0 (sscater_read,
 * sscater_changed) is the pseudo-image built by the feature net and its
 * event-based change set.  Errors as sscater_create, plus
 * SSCATER_E_INVALID_ARG for a bad sscater_pfn or C0 > 64. */
int sscater_create_pfn(const sscater_grid* grid, const sscater_layer* layers, int32_t n_layers,
                       const void* const* weights, const sscater_pfn* pfn, const float* pfn_weights,
                       sscater_t* out);

/* Advance a points-mode handle by one stride (Alg. 1): points is device
 * float[n_points][4] = (x, y, z, intensity) of the new stride (NULL when
 * n_points is 0), valid until the stream has executed the step.  The points
 * of the stride `window` strides back leave their pillars, the new ones are
 * queued, every pillar that lost or gained a point gets its features
 * recomputed from its queue, and the layers follow as in sscater_step.  The
 * first `window` strides after create/reset build the first full window.
 * SSCATER_E_OVERFLOW when n_points > max_new_points.  Asynchronous. */
int sscater_step_points(sscater_t h, const float* points, int32_t n_points, void* stream);

/* A sparse backbone (Sec. III-E; the submanifold operator of Sec. II-B):
 * layers and weights as for sscater_create, plus submanifold[n_layers] (host,
 * 0 or 1 per layer).  The input is a sparse tensor whose active sites are the
 * stride's pillars (whatever their values); a regular layer
 * (submanifold[l] = 0) is a sparse convolution whose active output sites are
 * those with an active input site in their receptive field, a submanifold
 * layer (submanifold[l] = 1, stride 1) keeps its input's active sites; every
 * output is phi(conv) at its active sites and zero elsewhere.  Layer 1 must
 * be regular.  A changed set: A_0 gains the pillars that appeared or
 * vanished; A_l holds the sites of the receptive-field rule over A_{l-1} that
 * are active now or were in the previous stride (sscater_changed), while
 * sscater_stats counts each layer's work list (all sites of the rule, whose
 * maps are kept current so that a site joining the active set holds its
 * value).  Dense-mode steps are refused.  The stride counter behind the
 * active sets is 31 bits wide.  Errors as sscater_create, plus
 * SSCATER_E_INVALID_ARG for a null submanifold array, a submanifold first
 * layer or a submanifold layer with stride 2. */
int sscater_create_sparse(const sscater_grid* grid, const sscater_layer* layers, int32_t n_layers,
                          const void* const* weights, const int32_t* submanifold, sscater_t* out);

/* Advance by one stride (Alg. 1): detect the changed input cells, then for
 * each layer scatter the deltas into the persistent maps (Eq. 2) and build the
 * next layer's change list.  The first step after create/reset is the full
 * pass.  A stride whose input equals the previous one bit for bit changes
 * nothing.  Asynchronous on `stream`. */
int sscater_step(sscater_t h, const sscater_pillars* pillars, void* stream);

/* sscater_step for a pillar list whose cell indices increase strictly (the
 * row-major order a pillar scatter produces).  Same results as sscater_step;
 * the change detection of Alg. 1 (which cells gained, lost or changed a
 * pillar against the previous stride) then runs as one launch that merges
 * the new list with the previous one chunk by chunk, instead of a pass over
 * each list.  A stride that follows a dense stride or an sscater_step call
 * (whose list may come in any order) takes the two passes.  A list that does
 * not increase is a device-side input fault (SSCATER_E_DEVICE; the stride's
 * results are then undefined).  Dense mode (idx NULL) is accepted and
 * behaves as in sscater_step.  Asynchronous. */
int sscater_step_sorted(sscater_t h, const sscater_pillars* pillars, void* stream);

/* Write layer `layer`'s output map into dst (device, NHWC, grid dtype): the
 * maps the method keeps between passes and updates in place (Sec. III-D: the
 * previous output is kept and only the delta contributions are added; the
 * abstract and Sec. IV-G: the kept maps equal recomputation).
 * layer 0 = the input canvas, layer l = 1..L = phi(Z_l) (bf16-rounded for the
 * bf16 dtype), layer L + 1 = the neck map (each upsampler's phi over its
 * channels) when the handle has a neck.  dst_bytes must be at least
 * H_l*W_l*C_l*sizeof(dtype).  Asynchronous on `stream`. */
int sscater_read(sscater_t h, int32_t layer, void* dst, size_t dst_bytes, void* stream);

/* Return to the empty window: zero the canvas and maps, forget the change
 * lists and clear the sticky device error, so the next step is again the
 * initial full pass of Alg. 1 (the first window is built from nothing before
 * the strides start; Sec. III-B).  The stream is synchronised first, so a
 * device fault of a stride still in flight cannot outlive the reset; the
 * clears themselves are enqueued on `stream`. */
int sscater_reset(sscater_t h, void* stream);

/* Free everything.  The caller must make sure no work of the handle is still
 * pending on any stream. */
int sscater_destroy(sscater_t h);

/* Test / metrics extension: the last stride's change map of layer `layer`
 * (Alg. 1: the per-layer map of sites changed by the convolution or the
 * ReLU, and for stride 2 the downsampled sites under a changed site) as a
 * list of cell indices A_layer (0 <= layer <= L, or L + 1 for the neck),
 * sorted row-major into the HOST buffer dst[cap].  dst is host memory, not
 * device memory: the call exists for tests and metrics, it must sort the
 * device's unordered list segments, and every caller reads the result on
 * the host, so it synchronises `stream`, copies the segments down and sorts
 * there.  The list length goes to *count_host (also when it exceeds cap, in
 * which case only cap entries are written).  Errors: SSCATER_E_INVALID_ARG
 * for a null handle or count_host, a layer out of range, cap < 0 or a null
 * dst with cap > 0; SSCATER_E_DEVICE when the sticky flag is set. */
int sscater_changed(sscater_t h, int32_t layer, int32_t* dst, int32_t cap, int32_t* count_host,
                    void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * list as sscater_changed (the last stride's A_layer, sorted row-major), built
 * on the device into the caller's DEVICE buffer dst[cap], with its length
 * written to the DEVICE int *count (also when it exceeds cap, in which case
 * only cap entries are written).  Asynchronous on `stream`: the call enqueues
 * three kernels and returns; nothing is synchronised, allocated or freed, so
 * the call can be captured into a graph.  The kernels keep per-block counts
 * in a fixed device array of the library (256 KB per GPU, held until the
 * process ends), which limits the layer's grid to 64 Mi cells (whole batch);
 * a larger grid is refused with SSCATER_E_SCRATCH before anything is
 * enqueued.  Calls that overlap on one GPU (concurrent streams or threads)
 * share that array and race: order them on one stream.  Errors:
 * SSCATER_E_INVALID_ARG for a null handle or count, a layer out of range,
 * cap < 0 or a null dst with cap > 0; SSCATER_E_DEVICE when the sticky flag
 * is set; SSCATER_E_HIP for a launch failure. */
int sscater_changed_noalloc(sscater_t h, int32_t layer, int32_t* dst, int32_t cap, int32_t* count, void* stream);

/* Test / metrics extension: counters of the last stride and totals into the
 * host struct *out: |A_l| per layer (the sizes of Alg. 1's change maps), the
 * (changed input, in-grid tap) pairs each layer contracted (Eq. 2's scatter
 * terms; 2 * cin * cout flops each), and the stride's algorithmic flops and
 * HBM bytes.  Synchronises `stream`.  Errors: SSCATER_E_INVALID_ARG for a
 * null handle or out; SSCATER_E_DEVICE when the sticky flag is set (the
 * counters are still written). */
int sscater_stats(sscater_t h, sscater_stats_t* out, void* stream);

/* Metrics extension: per-kernel timing of every launch of sscater_step (and
 * sscater_step_points) while enabled, with a pair of HIP events that the
 * kernel's own dispatch stamps at its start and end (hipExtLaunchKernel), so
 * the figure is the kernel's execution time without the event packets' cost.
 * Slots: 0 = input change detection (present pillars; points mode: the pillar
 * queue update), 1 = vanished pillars (points mode: the feature net),
 * 1 + l = layer l (l = 1..L; for a wide stride-1 layer that runs in two
 * launches, its tap sum), L + 2 + u = upsampler u of the neck, and
 * L + 1 + n_ups + l = the contraction launch of layer l when it has one, so
 * 2L + 2 + n_ups slots in all.  Enable it only for runs that measure
 * kernels. */
int sscater_profile(sscater_t h, int32_t enable);

/* Sum of the timed launch durations per slot (milliseconds) and the number of
 * launches per slot since the previous read, into host arrays of
 * n >= 2L + 2 + n_ups entries; clears the record.  Synchronises `stream`. */
int sscater_profile_read(sscater_t h, double* ms, int64_t* launches, int32_t n, void* stream);

/* Static text for an error code; for SSCATER_E_HIP the last HIP error text of
 * the calling thread's most recent failing call. */
const char* sscater_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* SSCATER_H */
