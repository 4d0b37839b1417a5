/*
 * CPU oracle for the parallel-NeRF-inversion hot path (render -> robust loss
 * -> pose gradient, momentum step, Monte Carlo resampling).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or constant with the HIP implementation.
 *
 * Precision: every continuous quantity is computed in double.  The few places
 * where floating point decides an integer (which samples exist on a ray, their
 * distances t, the occupancy cell tested, the hash-grid cell of a point, and
 * whether a coordinate is clamped) are computed in float with a fixed operation
 * order and no contraction, exactly as the GPU path decides them, so that both
 * sides agree on every index.
 */
#ifndef PNERF_ORACLE_H
#define PNERF_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t width, height;
  float fx, fy, cx, cy;
} orc_intr;

typedef struct {
  int32_t L, F;                 /* levels, features per level (F = 2) */
  uint32_t T;                   /* entries per level (power of two) */
  const int32_t* level_res;     /* [L] grid resolution N_l */
  int32_t dense_coarse;         /* 1: levels with (N_l+1)^3 <= T index 1:1 */
  const double* table;          /* [L][T][F] */
  int32_t din;                  /* L*F */
  const double *wd1, *wd2;      /* [din][64], [64][16]    (out = in @ W) */
  const double *wc1, *wc2, *wc3;/* [32][64], [64][64], [64][3] */
  double density_bias;          /* sigma = exp(h0 + density_bias) */
  float aabb_min[3], aabb_max[3];
  int32_t march_mode;           /* 0: n_uniform midpoints in the AABB; 1: lattice */
  int32_t n_uniform;
  float step;                   /* lattice spacing */
  int32_t max_samples;          /* cap on kept lattice samples per ray */
  double t_stop;                /* stop after transmittance < t_stop (0 = off) */
  int32_t occ_res;              /* 0: no occupancy grid */
  const uint32_t* occ_bits;     /* R^3 bits, index x + R(y + Rz), LSB first */
  double bg[3];                 /* background colour */
  int32_t loss_type;            /* 0 Huber, 1 L1, 2 L2, 3 Log L1, 4 Relative L2, 5 MAPE,
                                   6 sMAPE, 7 Smooth L1 (see orc_pixel_loss) */
  double loss_param;            /* Huber / Smooth L1 threshold, relative losses' epsilon */
  int32_t sh_dir_grad;          /* 1: add the view-direction path to the torque */
} orc_field;

/* Hash-grid index of vertex (i,j,k) on level `level` (dense or spatial hash). */
uint32_t orc_grid_index(const orc_field* f, int32_t level, uint32_t i, uint32_t j, uint32_t k);

/* Ray of pixel `pix` for camera-to-world pose [3][4] (float decision path). */
void orc_ray_f32(const float pose[12], const orc_intr* in, int32_t pix, float o[3], float d[3]);

/* Samples of K*P rays (n_threads OpenMP threads over the rays).  Fills
 * ray_offset[K*P+1]; when the total fits in `capacity` also t[], lattice index
 * j[] and the per-ray spacing delta[K*P].  Returns 0, or 1 if the total exceeds
 * capacity (offsets still valid). */
int32_t orc_march(const orc_field* f, int32_t K, const float* poses, int32_t P,
                  const int32_t* pix, const orc_intr* in, int64_t* ray_offset,
                  float* t, int32_t* lattice_j, float* delta, int64_t capacity,
                  int32_t n_threads);

/* Columns of the per-sample output of orc_shade and orc_shade_ray_variant:
 *   0 sigma, 1..3 rgb, 4 dL/dh0, 5..7 dL/dz (z = pre-sigmoid colour),
 *   8..10 dL/dp (zeros past the ray's stop), 11 the smallest relative margin of
 *   the sample's ReLU decisions (|pre-activation| / sum of its terms'
 *   magnitudes, over density layer 1 and colour layers 1 and 2), 12 its ray's
 *   distance from the nearest jump of the loss derivative (INFINITY if none),
 *   13..15 its share of the torque, t d x dL/dp (+ d x its dL/dd through SH when
 *   the direction path is on), 16 its ray's stop-decision margin (relative
 *   distance of T_used and T_{used-1} from t_stop; INFINITY without a stop). */
#define ORC_SAMPLE_COLS 17

/* Shade the frozen sample set (ray_offset, t, delta) for poses given in double,
 * take the loss against `obs` [H][W][3] and its gradient w.r.t. each pose.
 * Outputs (each may be NULL): loss[K], dpose[K][6] = (rotation, translation),
 * rgb[K*P][3], ray_stop[K*P] (samples composited per ray), signature (hash of
 * every discrete decision), sample_out[S][ORC_SAMPLE_COLS] (see above).
 * sh_dirs: NULL, or [K*P][3] fixed directions fed to the SH encoding instead of
 * the ray direction (used to freeze that path). */
int32_t orc_shade(const orc_field* f, int32_t K, const double* poses, int32_t P,
                  const int32_t* pix, const float* obs, const orc_intr* in,
                  const int64_t* ray_offset, const float* t, const float* delta,
                  const double* sh_dirs, double* loss, double* dpose, double* rgb,
                  int32_t* ray_stop, uint64_t* signature, double* sample_out,
                  int32_t n_threads);

/* One ray (pixel `pix` of a hypothesis with pose [12] and P pixels, samples t[n]
 * at spacing delta) shaded with some of its threshold decisions taken the other
 * way: each of them has two valid outcomes when the compared value lies within
 * rounding of its threshold, and a float implementation may take either.
 *   relu_margin, relu_pattern: the ReLU units of sample i whose margin is below
 *     relu_margin are numbered b = 0, 1, ... (density layer 1, then colour
 *     layers 1 and 2, units in order); bit b of relu_pattern[i] flips that unit's
 *     mask in the backward pass (its forward value is within rounding of 0
 *     either way).  relu_pattern may be NULL.
 *   stop: -1 to test the transmittance as the field says, else the number of
 *     samples composited.
 *   loss_sign[c]: 0, or +1 / -1 to take channel c's loss derivative on that
 *     side of r = 0 (L1, Log L1, MAPE, sMAPE).
 * Outputs: sample_out [n][ORC_SAMPLE_COLS] (or NULL), near_out[n] (the number
 * of units below relu_margin per sample, or NULL), the ray's loss (already
 * divided by 3P), its (torque, force) g[6], colour and samples composited.
 * Returns 1 for an unsupported field. */
typedef struct {
  double relu_margin;
  const int32_t* relu_pattern; /* [n], or NULL: relu_pattern_all for every sample */
  int32_t relu_pattern_all;
  int32_t stop;
  int32_t loss_sign[3];
} orc_variant;
int32_t orc_shade_ray_variant(const orc_field* f, const double pose[12], int32_t P,
                              int32_t pix, const float* obs, const orc_intr* in, const float* t,
                              int32_t n, float delta, const orc_variant* var, double* sample_out,
                              int32_t* near_out, double* loss, double g[6], double rgb[3],
                              int32_t* stop);

/* Many rays at once (OpenMP over the jobs), each shaded like
 * orc_shade_ray_variant with the job's stop, loss signs and one ReLU pattern
 * for all its samples (each sample keeps the bits below its own count of near
 * units), the same relu_margin for all.  Job q reads its samples at t[t0..t0+n)
 * and pose poses[hyp] (double [12]); its per-sample rows go to
 * sample_out[out_row[q]..][ORC_SAMPLE_COLS] and near_out[out_row[q]..] (either
 * may be NULL), its loss to loss[q] and (torque, force) to g[q][6]. */
typedef struct {
  int32_t hyp, pix;
  int64_t t0;
  int32_t n;
  float delta;
  int32_t stop;
  int32_t loss_sign[3];
  int32_t relu_pattern;
} orc_ray_job;
int32_t orc_shade_ray_jobs(const orc_field* f, const double* poses, int32_t P, const float* obs,
                           const orc_intr* in, const float* t, double relu_margin, int32_t n_jobs,
                           const orc_ray_job* jobs, const int64_t* out_row, double* sample_out,
                           int32_t* near_out, double* loss, double* g, int32_t n_threads);

/* Pieces exposed for pinning. */
void orc_encode(const orc_field* f, const float x32[3], const double x64[3],
                const int32_t clamped[3], double* feat, double* jac /* [3][din] or NULL */);
void orc_sh16(const double d[3], double out[16], double grad[16][3]);
void orc_density_mlp(const orc_field* f, const double* feat, double h[16]);
void orc_color_mlp(const orc_field* f, const double xc[32], double rgb[3]);
void orc_composite(int32_t n, const double* sigma, const double* rgb, double delta,
                   const double bg[3], double t_stop, double C[3], double* trans,
                   double* weight, int32_t* n_used);
void orc_composite_grad(int32_t n, const double* sigma, const double* rgb, double delta,
                        const double bg[3], double t_stop, const double gC[3],
                        double* g_sigma, double* g_rgb);
void orc_exp_so3(const double w[3], double R[9]);
/* One channel of a pixel loss: value, d loss / d C, distance from the nearest
 * derivative jump (INFINITY if none). */
double orc_pixel_loss(int32_t type, double C, double y, double p, double* grad, double* kink);

/* Heavy-ball momentum step on SO(3) x T(3), in place. */
void orc_step_momentum(int32_t K, float* poses, float* momentum, const float* dpose,
                       float lr, float beta);

/* Adam on SO(3) x T(3), separate moments per subspace, in place.
 * state [K][16] = m[6], v[6], per-hypothesis step count, 3 zeros. */
typedef struct {
  float lr_rot, lr_trans, beta1, beta2, eps, decay_base;
  int32_t decay_steps;   /* 0: no decay */
  int32_t staircase;     /* 1: exponent floor(step / decay_steps) */
  int32_t second_moment; /* 0: per component; 1: squared norm per subspace */
  int32_t representation; /* 0: SO(3) x T(3); 1: coupled se(3) twist, T <- Exp(u) T */
} orc_adam;
void orc_step_adam(int32_t K, float* poses, float* state, const float* dpose, int32_t step,
                   const orc_adam* a);

/* Keep the lowest-loss hypotheses, redraw the rest around them, in place;
 * redrawn rows of the optimiser state ([K][state_dim]) restart at 0. */
void orc_resample(int32_t K, float* poses, float* state, int32_t state_dim, const float* loss,
                  float keep_frac, float sigma_rot, float sigma_trans, uint64_t seed,
                  uint32_t round_idx, int32_t* rank_out /* [K] or NULL */);
uint64_t orc_splitmix64_next(uint64_t* state);
void orc_normals6(uint64_t seed, uint32_t round_idx, uint32_t slot, double n[6]);

/* Occupancy bitfield: bit set iff sigma at the cell centre > threshold. */
void orc_build_occupancy(const orc_field* f, int32_t R, float threshold, uint32_t* bits,
                         int32_t n_threads);

#ifdef __cplusplus
}
#endif
#endif
