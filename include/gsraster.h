/*
 * gsraster -- differentiable tile-based Gaussian-splatting rasterizer with the
 * view-dependent appearance evaluated inside it, for AMD Instinct MI355X (gfx950).
 *
 * Method: "Compact Neural Appearance Models for Efficient Gaussian Splatting".
 *   Sec. 3.1     - a per-primitive preprocess projects each Gaussian, finds the
 *                  16x16-pixel tiles it overlaps and computes its colour; a
 *                  tile-based blend alpha-composites the Gaussians of each pixel
 *                  in depth order.
 *   eq. sh_color_eval - degree-3 spherical-harmonics colour, 48 fp32 per Gaussian.
 *   Sec. 4 and the appendix on the fused CUDA rasterizer - a per-Gaussian latent
 *                  (28 bytes) decoded by a small shared half-precision MLP, evaluated
 *                  only for Gaussians that survive culling, inside the preprocess;
 *                  the backward pass propagates the colour gradient through the
 *                  view direction into the means.
 * The rasterizer conventions the paper inherits from 3D Gaussian Splatting
 * without restating them (EWA projection with a 0.3 px^2 low-pass, 3-sigma tile
 * rectangle, alpha cap 0.99, skip below 1/255, stop when transmittance would
 * fall below 1e-4) are implemented as documented below.
 *
 * Conventions of every call:
 *  - All pointers in the structs are DEVICE pointers owned by the caller, unless
 *    a comment says "host". The library never allocates or frees device memory
 *    while rasterizing; scratch memory is the caller's `workspace`
 *    (size from gs_workspace_size), 256-byte aligned.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream) and
 *    is asynchronous unless a comment says the call synchronises.
 *  - Every call returns a gs_status. Arguments are validated on the host before
 *    any launch; on error nothing is enqueued and gs_last_error() (thread-local)
 *    describes the problem. A failed launch or an asynchronous device error
 *    reported by HIP surfaces as GS_ERR_DEVICE from the call that observes it.
 *  - Arrays named [k][n] are planar: element (c, i) is at c*n + i.
 *  - n must be below 2^31 and the number of (tile, Gaussian) pairs below 2^32.
 */
#ifndef GSRASTER_H
#define GSRASTER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gs_status {
    GS_OK = 0,
    GS_ERR_INVALID_ARG = 1,   /* bad pointer, size, enum value or camera */
    GS_ERR_CAPACITY = 2,      /* a caller buffer is too small; the needed size is reported */
    GS_ERR_DEVICE = 3,        /* HIP reported an error */
    GS_ERR_UNSUPPORTED = 4,   /* valid request the library does not implement */
} gs_status;

#define GS_TILE 16            /* tile edge in pixels (Sec. 3.1) */
#define GS_SH_COEFFS 48       /* degree-3 SH: 16 basis functions x RGB (eq. sh_color_eval) */
#define GS_LATENT_DIM 14      /* binary16 latent per Gaussian: 28 bytes */
#define GS_MLP_IN 17          /* decoder input: latent (14) then unit view direction (3) */
#define GS_MLP_HIDDEN 32
#define GS_MLP_OUT 3
#define GS_MLP_WEIGHTS 1664   /* 32*17 + 32*32 + 3*32 */

/* Pinhole camera. Host struct, passed by pointer. */
typedef struct gs_camera {
    float viewmat[12];        /* row-major 3x4 [R|t]: world -> camera, x right, y down, z forward */
    float campos[3];          /* camera centre in world coordinates (= -R^T t) */
    float fx, fy, cx, cy;     /* focal lengths and principal point, pixels */
    int32_t width, height;    /* image size, pixels (any size >= 1; edge tiles may be partial) */
    float near_plane;         /* Gaussians with camera z <= near_plane are culled (0.2 typical) */
    float bg[3];              /* background colour added with the final transmittance */
} gs_camera;

/* Geometry of n Gaussians (Sec. 3.1). Device arrays, fp32. */
typedef struct gs_gaussians {
    int64_t n;
    const float* means;           /* [3][n] world positions */
    const float* log_scales;      /* [3][n] scale = exp(log_scale) */
    const float* quats;           /* [4][n] rotation quaternion (w, x, y, z); need not be unit */
    const float* opacity_logits;  /* [n] opacity = 1 / (1 + exp(-logit)) */
} gs_gaussians;

enum {
    GS_APP_SH3 = 0,           /* eq. sh_color_eval: c = max(0, 0.5 + sum_k Y_k(d) sh_k) */
    GS_APP_LATENT_MLP = 1,    /* c = sigmoid(W3 relu(W2 relu(W1 [z, d]))), no biases */
    GS_APP_NEURAL = 2,        /* Sec. 4 (eq. mlp_input, eq. neural_color_eval, eq. common_appearance):
                                 c = max(0, c0 + tanh(W3 relu(W2 relu(W1 x))) + 0.5), no biases,
                                 x = (Y_0..15(d) with bands above sh_degree zero,
                                      sin f_0, cos f_0, ..., sin f_7, cos f_7) */
    GS_APP_NEURAL_FOLDED = 3, /* render only: NEURAL with its first layer folded (the paper's
                                 viewer, supplementary section on the WebGL implementation).
                                 The view-independent inputs Y_0, sin f_j, cos f_j times their
                                 17 columns of W1 are stored per Gaussian as 16 binary16
                                 pre-activations p (gs_neural_fold); per view only
                                 h1 = relu(p + W1[:, 1..15] Y_1..15(d)) is evaluated, the rest
                                 as NEURAL. gs_render_bwd rejects this kind. */
    GS_APP_NASG = 4,          /* eq. nasg with one lobe: c = max(0, c0 + G(d) tanh(amp) + 0.5), G the
                                 normalized anisotropic spherical Gaussian (unit integral over the
                                 sphere): frame from three raw angles (cos th = tanh r0, the half
                                 azimuth and half twist of cosines tanh r1, tanh r2), sharpness
                                 exp(clamp(r3, -8, 8)), anisotropy exp(clamp(r4, -8, 8));
                                 G = exp(2 lam (u^(1+psi) - 1)) u^psi / K, u = (d.z + 1)/2,
                                 psi = a (d.x)^2 / ((d.x)^2 + (d.y)^2),
                                 K = 2 pi (1 - exp(-2 lam)) / (lam sqrt(1 + a)) */
    GS_APP_NASGABOR = 5,      /* NASG times the carrier (1 + cos(omega d.x)) / 2,
                                 omega = 20 (tanh(r5) + 1) */
};

#define GS_NEURAL_FEATURES 8  /* binary16 features per Gaussian (16 B) beside a 12 B fp32 base colour */
#define GS_NEURAL_WEIGHTS 816 /* 16*32 + 16*16 + 3*16, the paper's default decoder */
#define GS_NEURAL_MAX_WEIGHTS 2144 /* 32*32 + 32*32 + 3*32: the 32-neuron configuration */

/* View-dependent appearance (Sec. 3.1 and 4). d is the unit vector from the camera
 * centre to the Gaussian's mean, in world coordinates. */
typedef struct gs_appearance {
    int32_t kind;             /* GS_APP_* */
    int32_t sh_degree;        /* SH3: bands 0..sh_degree are used (0..3). NEURAL: the active
                                 degree of the direction encoding (0..3); at 0 the residual
                                 is off and c = max(0, c0 + 0.5) (the paper's schedule) */
    const float* sh;          /* SH3: [48][n] fp32, row 3*k + c = basis k, channel c.
                                 Basis order l = 0..3, m = -l..l; real SH with the
                                 Condon-Shortley phase: band 1 = sqrt(3/(4 pi)) (-y, z, -x) */
    const uint16_t* latent;   /* LATENT_MLP: [14][n] binary16 bit patterns */
    const uint16_t* mlp_w;    /* LATENT_MLP: binary16 W1[32][17], W2[32][32], W3[3][32], row-major
                                 [out][in], concatenated (1664 values). The decoder sees d
                                 rounded to binary16 and accumulates in fp32.
                                 NEURAL: binary16 W1[16][32], W2[16][16], W3[3][16] (816 values;
                                 other neural_layers / neural_width: W1[W][32], L - 1 matrices
                                 [W][W], Wout[3][W]); the decoder's inputs and hidden activations are binary16,
                                 its sums fp32, tanh in fp32 */
    const float* base_color;  /* NEURAL: [3][n] fp32 base colour c0 */
    const uint16_t* features; /* NEURAL: [8][n] binary16 bit patterns */
    const uint16_t* preact;   /* NEURAL_FOLDED: [n][16] binary16 bit patterns, Gaussian-major
                                 (32 B per Gaussian), as gs_neural_fold writes them;
                                 base_color and mlp_w (the 816 NEURAL weights) as for NEURAL */
    const float* lobes;       /* NASG: [8][n] fp32 raw r0..r4 then the three raw amplitudes;
                                 NASGABOR: [9][n], the raw frequency r5 last. base_color [3][n]
                                 is c0; sh_degree 0 turns the lobe off (c = max(0, c0 + 0.5)),
                                 1..3 on (the paper's schedule) */
    int32_t sh_y0_folded;     /* SH3: 0 = eq. sh_color_eval as printed (DC times Y0); 1 = the
                                 paper's implementation (Sec. 3.1), Y0 folded into the stored DC
                                 coefficients: c = max(0, 0.5 + sh_0 + sum_{k>=1} Y_k(d) sh_k) */
    int32_t neural_layers;    /* NEURAL: hidden layers, 1..3 (0 = the paper's default, 2); the
                                 weights are W1[16][32], layers - 1 matrices [16][16], Wout[3][16]
                                 (the supplementary table of configurations) */
    int32_t neural_width;     /* NEURAL: neurons per hidden layer: 0 or 16, or 32 for the table's
                                 32-32-32-3 configuration (weights W1[32][32], W2[32][32],
                                 Wout[3][32]; other 32-neuron shapes: GS_ERR_UNSUPPORTED) */
    int32_t neural_raw16;     /* NEURAL: 1 = 16 raw binary16 features ([16][n]) as the 16 feature
                                 inputs instead of (sin f, cos f) of 8 (the table's F = 16) */
} gs_appearance;

/* Screen-space record of one Gaussian, written by gs_preprocess (64 bytes).
 * Only meaningful where tiles_touched[i] > 0 (other records are written as zeros).
 * power_min, ext_x and ext_y only let the blend skip work early: below
 * power_min the alpha is certainly under 1/255 (a margin of 1e-3 in power), and
 * every pixel centre where the power reaches power_min lies within ext_x / ext_y
 * of the mean (slightly enlarged bounding box of that ellipse). A Gaussian whose
 * opacity is below 1/255 gets power_min = +inf and negative extents. */
typedef struct gs_splat {
    float mean_x, mean_y;             /* projected mean, pixels */
    float conic_a, conic_b, conic_c;  /* inverse 2D covariance [[a, b], [b, c]] */
    float opacity;                    /* activated opacity */
    float color[3];                   /* view-dependent RGB */
    float power_min;                  /* -ln(255 opacity) - 1e-3 */
    float ext_x, ext_y;               /* half extents of the alpha >= 1/255 region, pixels */
    int16_t rect[4];                  /* tiles x0, y0, x1, y1 (half-open) */
    float depth;                      /* camera-space z (> near_plane) */
    float reserved;                   /* written as 0 */
} gs_splat;

/* Outputs of gs_preprocess; caller-allocated device arrays. */
typedef struct gs_preprocessed {
    gs_splat* splats;         /* [n] */
    uint32_t* tiles_touched;  /* [n] tiles of the rectangle; 0 = culled */
    uint32_t* depth_key;      /* [n] sort key: bit pattern of depth, 0xFFFFFFFF when culled */
    uint64_t* num_pairs;      /* [1] total tiles touched (number of pairs P) */
    float* color_jac;         /* optional, SH3 only (NULL: not written or read): [10][n] for the
                                 backward, meaningful for visible Gaussians. Row 3c + j: the
                                 derivative of colour channel c's sum 0.5 + sum_k Y_k(d) sh_k
                                 (eq. sh_color_eval before the clamp) by direction
                                 component d_j; row 9: bit c set where channel c is above zero
                                 (not clamped), stored as the bits of a u32. Given here and to
                                 gs_render_bwd, the backward takes the colour's view-direction
                                 term from these 40 bytes instead of re-reading the 192 bytes of
                                 coefficients. */
} gs_preprocessed;

/* Gradients, caller-allocated device arrays, OVERWRITTEN by gs_render_bwd
 * (not accumulated). Entries of culled Gaussians are set to zero. */
typedef struct gs_grads {
    float* dmeans;            /* [3][n] */
    float* dlog_scales;       /* [3][n] */
    float* dquats;            /* [4][n] */
    float* dopacity_logits;   /* [n] */
    float* dsh;               /* SH3: [48][n]; rows of bands above sh_degree are zero */
    float* dlatent;           /* LATENT_MLP: [14][n] fp32 */
    float* dmlp_w;            /* LATENT_MLP: [1664], NEURAL: [816] (as many as mlp_w holds for other
                                 configurations) fp32, same order as mlp_w */
    float* dmean2d;           /* optional (may be NULL): [2][n] screen-space mean gradient */
    float* dbase_color;       /* NEURAL, NASG, NASGABOR: [3][n] */
    float* dfeatures;         /* NEURAL: [8][n] fp32, [16][n] with neural_raw16 (the gradient
                                 passes the binary16 storage) */
    float* dlobes;            /* NASG: [8][n], NASGABOR: [9][n], rows as in gs_appearance.lobes */
} gs_grads;

/*
 * gs_preprocess -- Sec. 3.1 preprocess with the appearance fused in (the
 * appendix's fused rasterizer: colour only for Gaussians that survive culling).
 * Per Gaussian: scale = exp(log_scale), opacity = sigmoid(logit) (both taken
 * through fp64 and rounded once), unit quaternion -> R, Sigma = R S S^T R^T;
 * t = R_view mu + t_view, culled if t.z <= near_plane; Jacobian of the pinhole
 * projection at t with x/z and y/z clamped to 1.3x the half field of view;
 * Sigma2D = J R_view Sigma R_view^T J^T + 0.3 I, culled unless det > 0; conic;
 * r = ceil(3 sqrt(lambda_max)) with lambda_max = mid + sqrt(max(0.1, mid^2 - det));
 * rect = [floor((px - r)/16), ceil((px + r)/16)) per axis clamped to the grid,
 * culled if empty; colour from the appearance model. For SH3 with
 * out->color_jac non-NULL, also the colour's view-direction Jacobian and clamp
 * bits there (see gs_preprocessed), for gs_render_bwd.
 * The geometry is one fixed sequence of correctly rounded fp32 operations
 * (no fused multiply-add), so tile rectangles and depth keys are reproducible.
 * num_pairs_host: optional HOST pointer; if non-NULL the call synchronises the
 * stream and stores P there.
 * Errors: GS_ERR_INVALID_ARG for NULL arrays, n out of range, unknown kind,
 * sh_degree outside 0..3, non-positive image size or focal length.
 */
gs_status gs_preprocess(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app,
                        const gs_preprocessed* out, uint64_t* num_pairs_host,
                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * gs_preprocess_noalloc -- gs_preprocess for callers that cannot allocate
 * device memory or hand over a workspace (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation). Same arguments, results
 * and errors as gs_preprocess, without the workspace: its scratch (one tile
 * sum per preprocess workgroup, or per wave of a decoder's grid) is a static
 * device array of the
 * library, GS_NOALLOC_MAX_GAUSSIANS / 64 u32 (1 MiB), one per GPU, held until
 * the process ends; its address is looked up once per device, on the first
 * call with that device current. Calls no allocating routine.
 * Limits: n <= GS_NOALLOC_MAX_GAUSSIANS, else GS_ERR_CAPACITY with nothing
 * enqueued. Every call on one GPU uses that GPU's one array: calls that overlap
 * on one GPU (on different streams, or from different threads) race and must
 * be serialised by the caller. Nothing in it needs clearing between calls
 * (each call writes every slot it reads).
 */
#define GS_NOALLOC_MAX_GAUSSIANS (1 << 24)
gs_status gs_preprocess_noalloc(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app,
                                const gs_preprocessed* out, uint64_t* num_pairs_host, void* stream);

/*
 * gs_bin_sort -- the depth-sorted per-tile lists of Sec. 3.1. Produces, for the P
 * pairs (tile, Gaussian) of every Gaussian with tiles_touched > 0 and every
 * tile of its rectangle, the Gaussian indices sorted by (tile id, depth key,
 * Gaussian index), tile id = ty * ceil(width/16) + tx. tile_ranges[t] =
 * {first, one-past-last} position of tile t; an empty tile gets {s, s} with s
 * the number of pairs of lower tiles. The result is unique (bit-exact).
 * num_pairs: P as gs_preprocess returned it to the host (host mode), or
 *   GS_PAIRS_ON_DEVICE (device mode): the kernels then read P from
 *   pre->num_pairs on the device, so the call needs no synchronisation and no
 *   host read-back of P.
 * capacity: length of values and tile_ids. Host mode: GS_ERR_CAPACITY if
 *   num_pairs > capacity, nothing enqueued. Device mode: a P above capacity is
 *   found on the device; no pair is then written, every tile range comes out
 *   empty ({0, 0}: the image renders as background and the gradients as zero),
 *   and pre->num_pairs keeps the P needed, for the caller to compare with
 *   capacity when it next synchronises and to retry with a larger buffer.
 *   A host-mode num_pairs that disagrees with the preprocess's count is also
 *   found on the device when the lists need more than capacity; every range
 *   then comes out empty in the same way.
 * values: [capacity] u32 device; tile_ids: optional [capacity] u32 tile of each pair.
 * tile_ranges: [n_tiles][2] u32 device.
 * workspace: at least gs_workspace_size(n, width, height, capacity, ...) bytes
 *   for this camera's image size (the per-block buffers depend on it).
 * Method: the Gaussians are sorted by depth; each gets one entry per 4x4-tile
 *   block its rectangle meets, in that order; a stable sort by block id groups
 *   them; each block's 16 tile lists are then written by ordered compaction.
 */
#define GS_PAIRS_ON_DEVICE UINT64_MAX
gs_status gs_bin_sort(const gs_camera* cam, const gs_preprocessed* pre, int64_t n, uint64_t num_pairs,
                      uint64_t capacity, uint32_t* values, uint32_t* tile_ids, uint32_t* tile_ranges,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * gs_render_fwd -- Sec. 3.1 blend. One workgroup per 16x16 tile; per pixel, with
 * sample point (x + 0.5, y + 0.5) and T = 1, front to back over the tile's list:
 * power = -(a dx^2 + c dy^2)/2 - b dx dy (skip if > 0); alpha = min(0.99, o e^power)
 * (skip if < 1/255); stop, without blending, if T (1 - alpha) < 1e-4; otherwise
 * C += colour alpha T, T *= 1 - alpha. Finally C += T bg.
 * image: [3][H][W] fp32; final_T: [H][W] fp32; n_contrib: [H][W] u32 = 1 + the
 * list position (within the tile's range) of the last blended Gaussian, 0 if none.
 */
gs_status gs_render_fwd(const gs_camera* cam, const gs_preprocessed* pre, int64_t n, const uint32_t* values,
                        const uint32_t* tile_ranges, float* image, float* final_T, uint32_t* n_contrib,
                        void* stream);

/*
 * gs_render_work -- the work of the Sec. 3.1 blend, counted for measuring its
 * throughput (not needed to render). Walks every pixel's list with the same
 * fp32 decisions as gs_render_fwd and writes, summed over all pixels:
 *   counts[0] entries blended (alpha >= 1/255, composited before the stop);
 *   counts[1] entries up to the last blended one (the sum of n_contrib);
 *   counts[2] entries before the last blended one whose alpha >= 1/255 box meets
 *             the pixel's tile (those gs_render_bwd evaluates per pixel; it skips
 *             the others for the whole tile), blended ones included;
 *   counts[3] the same for gs_render_fwd: entries up to the one that stops the
 *             pixel (or the list's end);
 *   counts[4] entries the method visits in the forward, whatever the box:
 *             up to and including the one that stops the pixel, else the
 *             whole list (the per-pixel work of the Sec. 3.1 blend).
 * Arguments as for gs_render_fwd; counts: [5] u64 device, 8-byte aligned,
 * overwritten. Asynchronous on stream.
 */
gs_status gs_render_work(const gs_camera* cam, const gs_preprocessed* pre, int64_t n, const uint32_t* values,
                         const uint32_t* tile_ranges, uint64_t* counts, void* stream);

/*
 * gs_render_bwd -- gradients of L = sum(dL_dimage * image) with respect to every
 * Gaussian parameter, for the image that gs_render_fwd produced from the same
 * inputs (Sec. 4 fused backward; the colour gradient also reaches the means
 * through the view direction). Reverse blending per tile, then the derivative of
 * the preprocess per Gaussian; for LATENT_MLP also the decoder weights.
 * dL_dimage: [3][H][W] fp32 device. The pair-level accumulation uses float
 * atomics, so results vary in the last bits between runs.
 * pre: as gs_preprocess left it for this camera; for SH3, pre->color_jac must be
 *   NULL (the coefficients are read again) or the array that gs_preprocess
 *   filled (its Jacobian is used instead); either gives the same gradients up to
 *   rounding.
 * workspace: at least gs_workspace_size(n, width, height, ...) bytes for this
 *   camera's image size (it holds the per-Gaussian accumulators and an order
 *   of the tiles: images of up to 32768 tiles are walked longest list walk
 *   first, which evens out the work per SIMD; the order does not change what
 *   is computed).
 */
gs_status gs_render_bwd(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app,
                        const gs_preprocessed* pre, const uint32_t* values, const uint32_t* tile_ranges,
                        const float* final_T, const uint32_t* n_contrib, const float* dL_dimage,
                        const gs_grads* grads, void* workspace, size_t workspace_bytes, void* stream);

/*
 * gs_mlp_eval -- the latent decoder on its own (Sec. 4 neural appearance):
 * colours of `rows` decoder inputs, computed exactly as inside gs_preprocess.
 * x: [rows][17] binary16 device array, each row the 14 latent values followed
 * by the unit view direction; mlp_w as in gs_appearance; colors: [rows][3]
 * fp32 device array. rows must be in [0, 2^31).
 */
gs_status gs_mlp_eval(const uint16_t* x, int64_t rows, const uint16_t* mlp_w, float* colors, void* stream);

/*
 * gs_neural_fold -- first-layer folding of the neural decoder (the paper's viewer,
 * supplementary section on the WebGL implementation), done once per scene before
 * rendering with GS_APP_NEURAL_FOLDED:
 *   preact[i][r] = binary16( sum over k in {0, 16..31} of W1[r][k] x_k(i) ),
 * x_0 = Y_0 = 1/(2 sqrt(pi)), x_16+2j = sin f_j, x_17+2j = cos f_j of Gaussian
 * i's features, each input rounded to binary16 as the unfolded decoder sees it,
 * the sum in fp32, then rounded to nearest binary16.
 * features: [8][n] binary16 device array; mlp_w: the 816 NEURAL weights (device);
 * preact: [n][16] binary16 device array, caller-owned, overwritten.
 * n must be in [0, 2^31); n = 0 does nothing. Asynchronous on `stream`.
 */
gs_status gs_neural_fold(const uint16_t* features, const uint16_t* mlp_w, int64_t n, uint16_t* preact,
                         void* stream);

/*
 * gs_adam_step -- one Adam step (Kingma and Ba, Algorithm 1, with bias
 * correction) over several parameter tensors in a single launch: the fused
 * optimiser update of the paper's training pipeline (supplementary
 * implementation details: one learning rate per parameter channel; the decoder
 * weights kept and updated in fp32 with a half-precision copy made for the
 * passes; beta2 = 0.99 for the decoder weights; the update touches every
 * Gaussian, visible in the iteration or not -- the per-parameter traffic the
 * paper holds responsible for SH3's slower optimisation, Sec. 5).
 * Tensor k is planar [rows][n] fp32: param, exp_avg (m) and exp_avg_sq (v) are
 * updated in place, grad is read. Per element, with t = step and lr that of
 * the element's row:
 *   m = b1 m + (1 - b1) g,   v = b2 v + (1 - b2) g^2,
 *   param -= (lr / (1 - b1^t)) * m / (sqrt(v) / sqrt(1 - b2^t) + eps)
 * (Algorithm 1's update with the bias corrections moved onto the step size and
 * the denominator). param_half, when not NULL, receives the updated values
 * rounded to binary16 (to nearest even) -- the half copy the passes read.
 * lr is a HOST array of `rows` learning rates (the row index is the paper's
 * column index of its [n][channels] layout). beta2 is per tensor.
 * Limits: 1 <= count <= GS_ADAM_MAX_TENSORS, rows >= 1, sum of rows <=
 * GS_ADAM_MAX_ROWS, 0 <= n < 2^31 per tensor, step >= 1, 0 <= b1, b2 < 1,
 * eps > 0. Tensors must not overlap one another.
 */
#define GS_ADAM_MAX_TENSORS 8
#define GS_ADAM_MAX_ROWS 128
typedef struct gs_adam_tensor {
    float* param;             /* [rows][n] fp32, updated in place */
    const float* grad;        /* [rows][n] fp32 */
    float* exp_avg;           /* [rows][n] fp32 first moment, updated in place */
    float* exp_avg_sq;        /* [rows][n] fp32 second moment, updated in place */
    uint16_t* param_half;     /* [rows][n] binary16 copy of the result, or NULL */
    int64_t n;
    int32_t rows;
    float beta2;
    const float* lr;          /* HOST [rows] learning rates */
} gs_adam_tensor;
gs_status gs_adam_step(const gs_adam_tensor* tensors, int32_t count, float beta1, float eps, int64_t step,
                       void* stream);

/*
 * gs_render_bwd_adam -- gs_render_bwd followed by one gs_adam_step on the
 * Gaussians' own parameters, in one pass: the Adam step of the paper's training
 * pipeline (supplementary implementation details; Kingma and Ba, Algorithm 1)
 * is applied to each parameter element where its gradient is computed, with
 * the same fp32 operations as gs_adam_step, instead of the gradient being
 * written and read back (for SH3 that halves the bytes the backward and the
 * optimiser move together). SH3 appearance only: other kinds return
 * GS_ERR_UNSUPPORTED.
 * adam: GS_RENDER_ADAM_TENSORS tensors as gs_adam_step takes them, in the order
 *   means [3][n], log_scales [3][n], quats [4][n], opacity_logits [1][n], sh
 *   [48][n]. Each param must be the very array that g or app holds: the
 *   parameters are updated in place (each Gaussian's after its own backward has
 *   read them; no Gaussian reads another's). grad is ignored. Every element is
 *   stepped, those of culled Gaussians and of SH bands above sh_degree with a
 *   zero gradient, as gs_adam_step would step them. beta1, eps, step as for
 *   gs_adam_step (the step whose bias corrections apply, >= 1).
 * grads: every array may be NULL here; one that is not receives the gradient
 *   the update used (dmean2d as for gs_render_bwd).
 * pre->color_jac is not read: the update reads the coefficients anyway, so the
 *   forward before this call may be given color_jac = NULL.
 * Errors: as gs_render_bwd; GS_ERR_INVALID_ARG when a tensor's param, rows or n
 *   does not match, a moment or lr array is NULL, or a constant is out of range.
 */
#define GS_RENDER_ADAM_TENSORS 5
gs_status gs_render_bwd_adam(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app,
                             const gs_preprocessed* pre, const uint32_t* values, const uint32_t* tile_ranges,
                             const float* final_T, const uint32_t* n_contrib, const float* dL_dimage,
                             const gs_grads* grads, const gs_adam_tensor* adam, float beta1, float eps, int64_t step,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes needed by any call for these sizes (host only). */
gs_status gs_workspace_size(int64_t n, int32_t width, int32_t height, uint64_t capacity, int32_t kind,
                            size_t* bytes);

/* Kernel timing. A gs_timer is a caller-owned timing context holding its own
 * HIP events (created with the timer, on the current device, never while
 * rendering). While a timer is attached to a thread, every kernel the library
 * launches from that thread is bracketed by a pair of events on its stream.
 * gs_timer_read synchronises the recorded events and returns, per kernel id
 * (GS_KERNEL_*), the summed duration in ms and the launch count since the
 * last reset; `count` is the length of both host arrays. A timer is used by
 * one thread at a time; gs_timer_attach(NULL) detaches; destroying the timer
 * attached to the calling thread detaches it. The library keeps no other
 * state between calls than the calling thread's attached timer and error text. */
enum {
    GS_KERNEL_PREPROCESS = 0, GS_KERNEL_PAIR_COUNT, GS_KERNEL_DEPTH_SORT, GS_KERNEL_ENTRY_OFFSETS,
    GS_KERNEL_BLOCK_ENTRIES, GS_KERNEL_BLOCK_SORT, GS_KERNEL_TILE_LISTS, GS_KERNEL_BLEND_FWD,
    GS_KERNEL_BWD_PREP, GS_KERNEL_BLEND_BWD, GS_KERNEL_PREPROCESS_BWD, GS_KERNEL_MLP_REDUCE,
    GS_KERNEL_ADAM, GS_KERNEL_NEURAL_FOLD, GS_KERNEL_COUNT
};   /* GS_KERNEL_BWD_PREP: the backward's accumulator clear and its tile order */
typedef struct gs_timer gs_timer;
gs_status gs_timer_create(gs_timer** out);
gs_status gs_timer_destroy(gs_timer* timer);
gs_status gs_timer_attach(gs_timer* timer);
gs_status gs_timer_reset(gs_timer* timer);
gs_status gs_timer_read(gs_timer* timer, double* ms, int64_t* launches, int32_t count);
const char* gs_kernel_name(int32_t kernel_id);

const char* gs_last_error(void);
const char* gs_version(void);

#ifdef __cplusplus
}
#endif
#endif
