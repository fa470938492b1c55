/*
 * donerf.h - C ABI of the DONeRF per-ray inference library for MI355X (gfx950).
 *
 * The library renders camera images with DONeRF (Neff et al., "DONeRF: Towards
 * Real-Time Rendering of Compact Neural Radiance Fields using Depth Oracle
 * Networks", EGSR 2021).  For every pixel ray (Sec. 4, Eq. 1) it
 *   1. moves the ray origin onto the sphere around the view cell (Sec. 5.2),
 *   2. evaluates the depth-oracle network once on the encoded unified origin
 *      and direction (or on the paper's unencoded input: unified origin,
 *      direction and one position per class centre, Sec. 5.2), giving one
 *      score per logarithmic depth class (Sec. 5.1, Eq. 3 discretisation),
 *   3. keeps the N best-scoring classes and places one sample at the centre
 *      of each (Eq. 1 with the class centre as depth),
 *   4. warps each sample towards the view cell (Eq. 4-5) and encodes it,
 *   5. evaluates the shading network at the N samples, with the encoded ray
 *      direction fed again into its last layer (App. D), and
 *   6. alpha-composites the N samples front to back over a black background.
 * Both networks have 8 linear layers of 256 units with ReLU (App. D).
 *
 * Conventions
 *   - All functions return a donerf_status; 0 is success.
 *   - Every argument is validated before any HIP call, so invalid arguments
 *     are reported without touching the GPU.
 *   - Pointers documented as "host" are read during the call only; pointers
 *     documented as "device" must be device memory of the current HIP device
 *     and are accessed asynchronously on the handle's stream.
 *   - A handle is not reentrant: one render in flight per handle at a time.
 *   - The message of the most recent failure in the calling thread is kept in
 *     donerf_last_error().
 */
#ifndef DONERF_H
#define DONERF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct donerf_handle donerf_t;

typedef enum donerf_status {
    DONERF_OK = 0,
    DONERF_E_INVALID_ARG = -1, /* NULL pointer, size or enum out of range    */
    DONERF_E_SIZE = -2,        /* weight count does not match the config     */
    DONERF_E_NONFINITE = -3,   /* NaN or Inf in weights, poses or config     */
    DONERF_E_DEVICE = -4,      /* no HIP device, or the device is not gfx950 */
    DONERF_E_NOMEM = -5,       /* device or host allocation failed           */
    DONERF_E_HIP = -6,         /* a HIP call failed; see donerf_last_error() */
    DONERF_E_UNSUPPORTED = -7  /* valid request the library does not handle */
} donerf_status;

typedef enum donerf_precision {
    DONERF_FP32 = 0, /* fp32 weights, features and activations, fp32 MFMA    */
    DONERF_BF16 = 1, /* bf16 weights, features and hidden activations (RNE),
                        fp32 accumulation, fp32 scores, heads, compositing;
                        sine, cosine, exp and reciprocal of the encoding and
                        compositing from the hardware instructions           */
    DONERF_FP8 = 2   /* the lower bit width Sec. 6.1 leaves as headroom: the
                        six hidden layers of each network in OCP E4M3 (weights
                        W 2^s rounded to nearest even with the largest s that
                        keeps max|W| 2^s <= 448, one s per layer; their inputs
                        clamped to [0, 448] after ReLU and rounded to E4M3);
                        the first layers and heads as in DONERF_BF16, fp32
                        accumulation throughout                               */
} donerf_precision;

typedef enum donerf_select {
    DONERF_SELECT_TOPN = 0,         /* one sample at the centre of each of the N
                                       highest-scoring classes; its width is
                                       the class width                          */
    DONERF_SELECT_TOPN_SOFTMAX = 1, /* the scores filtered by a softmax: the
                                       selection ranks the raw scores exactly
                                       as DONERF_SELECT_TOPN (the softmax is
                                       monotone; in fp32 it can also map
                                       distinct scores to equal values, so it
                                       is not ranked itself); the softmax only
                                       transforms the scores a debug render
                                       dumps                                   */
    DONERF_SELECT_CDF = 2           /* Sec. 5.1, Fig. 7: the class values
                                       sigmoid(score) as a piecewise-constant
                                       PDF over the classes (uniform in the
                                       coordinate of Eq. 3), its CDF inverted at
                                       u_i = (i + 0.5)/N; sample i's width is the
                                       depth extent of the slice [i/N, (i+1)/N].
                                       fp32 arithmetic; above 128 classes the
                                       depth head runs twice (class sums, then
                                       the values the targets fall in)       */
} donerf_select;

typedef enum donerf_depth_input {
    DONERF_DEPTH_ENCODED = 0,  /* encode(unified origin / d_max, 10) and encode(r, 4):
                                  90 inputs (layout below)                      */
    DONERF_DEPTH_POSITIONS = 1 /* Sec. 5.2, App. D: unified origin / d_max, r and
                                  one position (x_k - c) / d_max per class
                                  centre, x_k = o + c_k r from the camera origin,
                                  unencoded: 6 + 3 n_bins inputs in the order
                                  [origin xyz, r xyz, x_0 xyz, ..., x_{B-1} xyz].
                                  The first layer's weights are folded at create
                                  into 9 columns (the positions are affine in the
                                  ray) and evaluated in fp32 in both precisions;
                                  its inputs are not rounded to bf16           */
} donerf_depth_input;

/* Maximum number of samples per ray a handle can be created for. */
#define DONERF_MAX_SAMPLES 16

typedef struct donerf_cfg {
    float near_dist;   /* d_min > 0: nearest sample depth along the ray (Eq. 1) */
    float far_dist;    /* d_max > d_min: farthest depth; also the normalisation
                          of Eq. 2 and the warp scale of Eq. 5                 */
    int32_t n_bins;    /* B: number of logarithmic depth classes (Eq. 3);
                          the library supports 64, 128, 192 and 256          */
    int32_t n_max;     /* largest N a render may request, 1..16, n_max <= B   */
    float fov_x_deg;   /* horizontal field of view of the pinhole camera, in
                          degrees, 0 < fov < 180                               */
    float centre[3];   /* view-cell centre c (Eq. 2, Eq. 4)                    */
    float radius;      /* radius > 0 of the unification sphere (Sec. 5.2)      */
    int32_t precision; /* donerf_precision                                     */
    int32_t select;    /* donerf_select                                        */
    int32_t depth_input; /* donerf_depth_input                                 */
} donerf_cfg;

/*
 * Number of fp32 values in the weight blob for B depth classes and the given
 * donerf_depth_input, or 0 if B is not positive or depth_input is unknown.
 *
 * Blob layout (host, fp32): depth network layers 0..7, then shading network
 * layers 0..7; each layer is W[out][in] row-major followed by b[out].
 *   depth  : 90 (or 6 + 3 B) -> 256, 6 x (256 -> 256), 256 -> B
 *   shading: 63 -> 256, 6 x (256 -> 256), (256 + 27) -> 4
 * Depth layer 0 reads the encoding of the unified origin divided by d_max
 * (63 values) followed by the encoding of the direction (27 values).  The
 * encoding of v with L frequencies is [v, sin(2^0 pi v), cos(2^0 pi v), ...,
 * sin(2^(L-1) pi v), cos(2^(L-1) pi v)], each block over x, y, z; L = 10 for
 * positions, 4 for directions.  Shading layer 0 reads the encoding of the
 * warped sample (63); shading layer 7 reads the 256 hidden values followed by
 * the direction encoding (27) and outputs (r, g, b, sigma) before activation.
 */
size_t donerf_weight_count(int32_t n_bins, int32_t depth_input);

/*
 * Create a renderer on the current HIP device.
 *   cfg       host, read during the call
 *   weights   host fp32 blob of n_weights values (layout above); the library
 *             converts and copies it to the device, so the caller may free it
 *             on return
 *   out       receives the handle; set to NULL on failure
 * Errors: E_INVALID_ARG (NULL, cfg ranges), E_UNSUPPORTED (n_bins not in the
 * supported set), E_SIZE (n_weights !=
 * donerf_weight_count(cfg->n_bins, cfg->depth_input)),
 * E_NONFINITE (NaN/Inf in cfg or weights), E_DEVICE (no device or not
 * gfx950), E_NOMEM, E_HIP.
 */
int donerf_create(const donerf_cfg* cfg, const float* weights, size_t n_weights,
                  donerf_t** out);

/* Release the handle and its device memory.  NULL is allowed. */
void donerf_destroy(donerf_t* h);

/*
 * Bind the HIP stream (a hipStream_t passed as void*) on which the handle's
 * work is enqueued.  NULL selects the null stream (the default).
 */
int donerf_set_stream(donerf_t* h, void* stream);

/*
 * Render P camera images of H x W pixels with N samples per ray.
 *   cam_poses  host, P x 12 fp32: camera-to-world 3x4 row-major [R | o] per
 *              image; the camera looks down its -z axis, +y is up; pixel
 *              (i, j), i along the width and j downwards, is the ray through
 *              the pixel centre
 *   N          samples per ray, 1 <= N <= cfg.n_max (and <= B)
 *   out_rgb    device, P x H x W x 3 fp32, row-major, caller-owned
 *   out_depth  device, P x H x W fp32 (sum of sample weight x sample depth),
 *              or NULL to skip
 * The work is enqueued on the handle's stream; results are valid once the
 * stream has been synchronised.  No allocation, no host synchronisation.
 * The call issues kernel launches only (the poses travel in the launch
 * arguments; no memset or copy), so it can be captured into a HIP graph on
 * the handle's stream and replayed; a replay renders the poses, sizes and
 * buffers of the captured call.  Calls on one handle share its scratch
 * buffer for the split tail: do not let two of them overlap on different
 * streams.
 * Errors: E_INVALID_ARG (NULL handle/poses/out_rgb, P, H, W < 1, N out of
 * range, P*H*W >= 2^31, H*W > 2^24), E_NONFINITE (pose), E_HIP (launch
 * failed).
 */
int donerf_render(donerf_t* h, const float* cam_poses, int32_t P, int32_t H, int32_t W,
                  int32_t N, float* out_rgb, float* out_depth);

/*
 * donerf_render for callers that cannot allocate device memory at all (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and results, with the split tail's partial
 * results kept in a static device array of the library instead of the
 * handle's buffer.  The array holds 5 x 256 x 256 floats (1.25 MiB) on every
 * device the library runs on, until the process ends; its address is looked
 * up when a handle is created, so this call makes no HIP call other than its
 * kernel launches and allocates nothing.  Every call on one device shares that
 * device's array (no contents need clearing: each launch writes every part it
 * reads back), so calls that overlap on one device, on any handles or
 * streams, race and must not be issued.
 * Arguments and errors as donerf_render, plus E_UNSUPPORTED when a launch's
 * split tail needs more than the array holds (only on devices with more than
 * 256 compute units) and E_HIP when the array's address could not be looked
 * up at create.
 */
int donerf_render_static_scratch(donerf_t* h, const float* cam_poses, int32_t P, int32_t H, int32_t W,
                                 int32_t N, float* out_rgb, float* out_depth);

/*
 * donerf_render with optional per-ray intermediate outputs, for testing.
 *   out_bins     device, P x H x W x N int32: the class of each sample in sample
 *                (= depth) order, or NULL
 *   out_scores   device, P x H x W x B fp32: depth-network scores, or NULL;
 *                with DONERF_SELECT_TOPN_SOFTMAX the softmax probabilities
 *   out_samples  device, P x H x W x N x 2 fp32: depth and width of each
 *                sample, or NULL
 * Same errors as donerf_render.
 */
int donerf_render_debug(donerf_t* h, const float* cam_poses, int32_t P, int32_t H,
                        int32_t W, int32_t N, float* out_rgb, float* out_depth,
                        int32_t* out_bins, float* out_scores, float* out_samples);

/*
 * Run the device top-N selection on given scores, for testing.
 *   scores   device, rays x B fp32
 *   out_idx  device, rays x N int32: the N classes with the highest scores,
 *            ties broken towards the lower class index, +0 and -0 equal,
 *            NaN below every number, written in ascending class order
 * Errors: E_INVALID_ARG (NULL, rays < 1, N out of range), E_HIP.
 */
int donerf_debug_topn(donerf_t* h, const float* scores, int32_t rays, int32_t N,
                      int32_t* out_idx);

/*
 * Measured ceiling of the matrix cores, for the roofline of donerf_render:
 * a register-fed MFMA loop in the handle's precision (BF16: 32 x 32 x 16
 * bf16; FP8: 32 x 32 x 64 E4M3; FP32: 32 x 32 x 2 fp32), on the handle's
 * stream.  workgroups x 4 waves each run four independent accumulator chains
 * of `iters` steps on seeded random register operands drawn like the
 * render's: A uniform in [-1, 1) like weights, B the positive part of such
 * values like ReLU activations (no memory traffic, no dependence stalls).
 *   workgroups  1..2^20 (a few per compute unit fill the device)
 *   iters       1..2^24 steps per chain
 *   sink        device, workgroups x 256 fp32, caller-owned: one sum of
 *               accumulators per thread, written so the work is kept
 *   flop        host, may be NULL: the launch's FLOP (2 per multiply-add)
 * Time the launch with events on the handle's stream.
 * Errors: E_INVALID_ARG (NULL handle or sink, sizes out of range), E_HIP.
 */
int donerf_debug_mfma_peak(donerf_t* h, int32_t workgroups, int32_t iters, float* sink, double* flop);

/*
 * Training targets of the depth oracle (Sec. 5.1) for P depth maps, on the
 * handle's depth classes and stream:
 *   Eq. 6  C(z) = 1 for the class z with b_z <= d < b_{z+1} of the pixel's
 *          first-surface depth d (no class where d is outside [d_min, d_max)
 *          or not finite),
 *   Eq. 7  C^(z) = max over the offsets |i|, |j| <= floor(K/2) of
 *          C_{x+i,y+j}(z) minus sqrt(i^2 + j^2) / (sqrt(2) floor(K/2))
 *          (neighbours outside the image left out; K = 1 keeps C; an even
 *          K spans K + 1 pixels and gives the targets of K + 1),
 *   Eq. 8  C`(z) = min(sum_{|i| <= floor(Z/2)} C^(z + i) (floor(Z/2) + 1 - |i|)
 *          / (floor(Z/2) + 1), 1) (classes outside [0, B) left out).
 *   depth  device, P x H x W fp32: the distance from the camera to the first
 *          surface along each pixel's ray (Eq. 1's d), row-major
 *   K, Z   window sizes, 1..15 (the paper evaluates 1, 5 and 9 and uses
 *          K = Z = 5)
 *   out    device, P x H x W x B fp32, caller-owned; B = cfg.n_bins
 * Enqueued on the handle's stream; no allocation.
 * Errors: E_INVALID_ARG (NULL, P, H, W < 1, K or Z out of range, too many
 * pixels), E_HIP.
 */
int donerf_targets(donerf_t* h, const float* depth, int32_t P, int32_t H, int32_t W, int32_t K, int32_t Z,
                   float* out);

/*
 * Copy the handle's depth-class table to host memory: bounds (B + 1 values,
 * may be NULL), centres (B), widths (B).  Bounds b_k = d_min + (d_max - d_min
 * + 1)^(k/B) - 1 (the inverse of Eq. 3 on a uniform grid), centres at
 * (k + 0.5)/B, widths b_{k+1} - b_k; computed in fp64, stored as fp32.
 */
int donerf_debug_bins(const donerf_t* h, float* bounds, float* centres, float* widths);

/* Static description of a status code. */
const char* donerf_status_str(int status);

/* Message of the most recent failure in the calling thread ("" if none). */
const char* donerf_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DONERF_H */
