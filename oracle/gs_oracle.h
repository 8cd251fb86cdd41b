/*
 * CPU oracle for the tile-based differentiable Gaussian rasterizer with fused
 * SH3, latent+MLP or the paper's neural (base colour + feature) appearance.
 *
 * TEST INFRASTRUCTURE ONLY. This library defines what the GPU path must
 * compute; it is called by the test-suite, by the package's smoke check and by
 * the benchmark's CPU-baseline leg, and by nothing else. It shares no code,
 * header, table or constant with the HIP library.
 *
 * The method it follows (the paper's Sec. 3.1 and 4, plus the conventions the
 * paper inherits from 3D Gaussian Splatting, which it states only by citation):
 *   preprocess  - activation of scale/rotation/opacity, projection of the mean,
 *                 EWA 2D covariance with a 0.3 px low-pass, culling, tile
 *                 rectangle (Sec. 3.1 "preprocess kernel"); view-dependent
 *                 colour from SH (eq. sh_color_eval) or from a latent decoded
 *                 by a small MLP (Sec. 4 and the fused-implementation appendix);
 *   bin_sort    - list of (tile, Gaussian) pairs sorted by tile, then depth,
 *                 then index (Sec. 3.1 "depth-sorted order");
 *   render_fwd  - per-pixel front-to-back alpha compositing (Sec. 3.1 "blend");
 *   render_bwd  - exact derivative of render_fwd's output w.r.t. every input
 *                 parameter, chained through the preprocess (Sec. 4, fused
 *                 backward, including the colour gradient into the means).
 *
 * Two builds of every floating-point routine exist:
 *   *_f32 : quantities that decide integers (tile rectangles, sort keys,
 *           skip/stop decisions of the blend) are taken in fp32, the precision
 *           the GPU kernels take them in; sums of colours and all gradient
 *           arithmetic are done in fp64;
 *   *_f64 : everything in fp64 (used for finite-difference checks).
 * All arrays are host memory, planar ([channel][n]) and caller-allocated.
 */
#ifndef GS_ORACLE_H
#define GS_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct orc_camera {
    double viewmat[12];   /* row-major 3x4 [R|t], world -> camera (x right, y down, z forward) */
    double campos[3];     /* camera centre, world frame */
    double fx, fy, cx, cy;
    int32_t width, height;
    double near_plane;
    double bg[3];
} orc_camera;

enum { ORC_APP_SH3 = 0, ORC_APP_LATENT_MLP = 1, ORC_APP_NEURAL = 2, ORC_APP_NEURAL_FOLDED = 3, ORC_APP_NASG = 4,
       ORC_APP_NASGABOR = 5 };

/* flags written per Gaussian by the preprocess */
enum {
    ORC_VISIBLE = 1,
    ORC_CLAMP_X = 2,        /* guard band active on x in the Jacobian */
    ORC_CLAMP_Y = 4,
    ORC_COLOR_ZERO_R = 8,   /* SH colour pre-activation <= 0 for channel r/g/b */
    ORC_COLOR_ZERO_G = 16,
    ORC_COLOR_ZERO_B = 32,
};

typedef struct orc_appearance {
    int32_t kind;           /* ORC_APP_* */
    int32_t sh_degree;      /* 0..3; for NEURAL the active degree of the direction encoding */
    const double* sh;       /* [48][n] */
    const double* latent;   /* [14][n] values of binary16 numbers */
    const double* mlp_w;    /* values of binary16 numbers. LATENT_MLP: 1664, W1[32][17], W2[32][32],
                               W3[3][32]. NEURAL: 816, W1[16][32], W2[16][16], W3[3][16] */
    int32_t dir_exact;      /* 0: the decoder inputs derived from the view direction (and, for
                               NEURAL, the feature encodings) are rounded to binary16, as the
                               half-precision decoder sees them; 1: unrounded, for finite differences */
    int32_t half_act;       /* 1: the hidden activations are rounded to binary16 before they enter
                               the next layer (half-precision operands, Sec. 4 / fused appendix);
                               0: exact fp64 activations */
    const double* base_color; /* NEURAL: [3][n] base colour c0 */
    const double* features;   /* NEURAL: [8][n] values of binary16 numbers */
    const double* preact;     /* NEURAL_FOLDED: [16][n] first-layer pre-activations of the
                                 view-independent inputs (oracle.neural_fold); render only */
    const double* lobes;      /* NASG: [8][n] raw frame angles (3), sharpness, anisotropy and
                                 the three raw amplitudes; NASGABOR: [9][n], the frequency last.
                                 base_color is the base colour c0 of both */
    int32_t sh_y0_folded;     /* SH3: 1 = the constant degree-0 basis value Y0 is folded into the
                                 stored DC coefficients (the paper's implementation, Sec. 3.1):
                                 their basis value is 1 instead of Y0 */
    int32_t neural_layers;    /* NEURAL: hidden layers L (1..3; 0 = the paper's default, 2) */
    int32_t neural_width;     /* NEURAL: neurons per hidden layer W (16 or 32; 0 = 16) */
    int32_t neural_raw16;     /* NEURAL: 1 = 16 raw features as the 16 feature inputs instead of
                                 (sin f, cos f) of 8 (the table of configurations' F = 16) */
} orc_appearance;

/* Outputs of the preprocess. Entries of culled Gaussians are zero. */
typedef struct orc_pre {
    double* mean2d;         /* [2][n] */
    double* conic;          /* [3][n] (a, b, c) of the inverse 2D covariance */
    double* opacity;        /* [n] */
    double* color;          /* [3][n] */
    double* depth;          /* [n] */
    int32_t* rect;          /* [4][n] x0, y0, x1, y1 in tiles, half-open */
    int32_t* tiles;         /* [n] tiles touched, 0 when culled */
    int32_t* flags;         /* [n] ORC_* bits */
    uint64_t* mlp_mask;     /* [n] ReLU masks of the MLP's 64 hidden units, 0 for SH */
} orc_pre;

typedef struct orc_grads {
    double* dmeans;         /* [3][n] */
    double* dlog_scales;    /* [3][n] */
    double* dquats;         /* [4][n] */
    double* dopacity_logits;/* [n] */
    double* dsh;            /* [48][n] (SH3) or NULL */
    double* dlatent;        /* [14][n] (latent) or NULL */
    double* dmlp_w;         /* [1664] (latent), [816] (neural) or NULL */
    double* dmean2d;        /* [2][n] screen-space mean gradient, or NULL */
    double* dconic;         /* [3][n] or NULL */
    double* dopacity;       /* [n] or NULL (w.r.t. the activated opacity) */
    double* dcolor;         /* [3][n] or NULL */
    double* dbase_color;    /* [3][n] (neural) or NULL */
    double* dfeatures;      /* [8][n] (neural; [16][n] with 16 raw features) or NULL */
    double* dlobes;         /* [8][n] (NASG), [9][n] (NASGabor) or NULL */
    double* dmlp_w_abs;     /* like dmlp_w, or NULL: per weight, the sum over Gaussians of the
                               absolute values of the products whose sum is dmlp_w (the scale of
                               its rounding error when the products are formed in low precision) */
} orc_grads;

int orc_preprocess_f32(const orc_camera* cam, int64_t n, const double* means, const double* log_scales,
                       const double* quats, const double* opacity_logits, const orc_appearance* app,
                       const orc_pre* out);
int orc_preprocess_f64(const orc_camera* cam, int64_t n, const double* means, const double* log_scales,
                       const double* quats, const double* opacity_logits, const orc_appearance* app,
                       const orc_pre* out);

/* Pairs of every Gaussian with tiles > 0 and every tile of its rectangle, sorted
 * by (tile, depth, index). ranges[t] = [first, one-past-last) of tile t; an
 * empty tile gets [s, s) with s the number of pairs of smaller tiles.
 * Returns the number of pairs, or -1 if it exceeds capacity. */
int64_t orc_bin_sort(int64_t n, const int32_t* rect, const double* depth, const int32_t* tiles,
                     int32_t tiles_x, int32_t tiles_y, int64_t capacity, int32_t* values,
                     int32_t* tile_of, int64_t* ranges);

/* margin (nullable): per pixel, the smallest ratio, over its skip/stop/clamp
 * decisions, of the decision's relative distance from its threshold to a bound
 * on how far an fp32 evaluation in another operation order can move it (see
 * walk_pixel); above 1 every decision of the pixel is reproducible.
 * n_blended (nullable): per pixel, the number of entries composited.
 * n_walked (nullable): per pixel, the number of entries the blend visits: up
 * to and including the one that stops it, else the whole list. */
void orc_render_fwd_f32(const orc_camera* cam, int64_t n, const orc_pre* pre, const int64_t* ranges,
                        const int32_t* values, double* image, double* final_T, int32_t* n_contrib,
                        double* margin, int32_t* n_blended, int32_t* n_walked);
void orc_render_fwd_f64(const orc_camera* cam, int64_t n, const orc_pre* pre, const int64_t* ranges,
                        const int32_t* values, double* image, double* final_T, int32_t* n_contrib,
                        double* margin, int32_t* n_blended, int32_t* n_walked);

/* Gradients of sum(dL_dimage * image) w.r.t. all inputs; outputs overwritten. */
int orc_render_bwd_f32(const orc_camera* cam, int64_t n, const double* means, const double* log_scales,
                       const double* quats, const double* opacity_logits, const orc_appearance* app,
                       const orc_pre* pre, const int64_t* ranges, const int32_t* values,
                       const double* dL_dimage, const orc_grads* grads);
int orc_render_bwd_f64(const orc_camera* cam, int64_t n, const double* means, const double* log_scales,
                       const double* quats, const double* opacity_logits, const orc_appearance* app,
                       const orc_pre* pre, const int64_t* ranges, const int32_t* values,
                       const double* dL_dimage, const orc_grads* grads);

/* Threads of the OpenMP loops (results do not depend on them). */
void orc_set_threads(int32_t k);
int32_t orc_get_threads(void);

/* Real spherical harmonics of degree <= 3 (16 values) and their gradient
 * w.r.t. the direction components (16x3), built from the Legendre definition. */
void orc_sh_basis(const double d[3], double Y[16], double dY[48]);
/* The latent decoder on given inputs: x [rows][17] (binary16 values), out [rows][3]. */
void orc_mlp_eval(const double* x, int64_t rows, const double* w, double* out, int32_t half_act);
/* Round to the nearest binary16 value (ties to even), returned as a double. */
double orc_round_half(double x);

/* One NASG (gabor = 0) or NASGabor (gabor = 1) lobe kernel at unit direction v,
 * from its 5 (6) raw parameters (frame angles, sharpness, anisotropy[, frequency]);
 * see gs_oracle.c for the definition. _many evaluates m directions v[m][3]. */
double orc_lobe_eval(const double* raw, int32_t gabor, const double v[3]);
void orc_lobe_eval_many(const double* raw, int32_t gabor, int64_t m, const double* v, double* out);
/* the kernel value, its derivative w.r.t. the raw parameters (draw[5 or 6]) and w.r.t. v */
double orc_lobe_grad(const double* raw, int32_t gabor, const double v[3], double* draw, double dv[3]);

#ifdef __cplusplus
}
#endif
#endif
