/*
 * pnerf.h -- C ABI of the MI355X (gfx950) hot path of parallel NeRF inversion
 * for pose estimation (Lin et al., "Parallel Inversion of Neural Radiance
 * Fields for Robust Pose Estimation", arXiv 2210.10108).
 *
 * Problem (Sec. III, iNeRF's formulation): the field Theta is trained and
 * frozen, intrinsics are known, and the camera pose T is updated iteratively to
 * minimise a photometric loss between the field's rendering and the observed
 * image.  This library evaluates, for K pose hypotheses at once (Sec. IV-B),
 * the loss and its gradient split into a rotation part (the torque of Eq. 3)
 * and a translation part (the force of Eq. 2), applies a momentum or Adam update
 * on SO(3) x T(3) (Sec. IV-A; setting of Sec. IV-D), and resamples hypotheses (Sec. IV-B).
 *
 * Conventions shared by every entry point
 *  - Poses are camera-to-world float32 [K][3][4] = [R | o], row major: o is the
 *    camera centre and the origin of every ray (Sec. IV-A).  Camera axes:
 *    x right, y down, z forward; pixel (u, v) has its centre at (u+0.5, v+0.5).
 *  - Pose gradients and momenta are float32 [K][6] = (w_x, w_y, w_z, t_x, t_y,
 *    t_z): w is the gradient w.r.t. a rotation Exp(w) R applied about the
 *    camera centre in world axes, t the gradient w.r.t. o.
 *  - Array arguments marked (device) are device pointers owned by the caller;
 *    they must stay valid until the work queued on `stream` has finished.
 *    Arguments marked (host) are read before the call returns.
 *  - `stream` is a hipStream_t (NULL = the default stream).  pnerf_step_momentum,
 *    pnerf_step_adam and pnerf_resample_hypotheses only enqueue work and
 *    return.  The calls that render (pnerf_render_loss_grad, pnerf_render,
 *    pnerf_march) synchronise the stream once per 2^21 rays: after counting
 *    every ray's samples they read the per-hypothesis sample counts back, size
 *    the workspace to them and cut the batch into chunks of whole hypotheses,
 *    then enqueue the rest and return.
 *    pnerf_create_field and pnerf_field_occupancy synchronise the stream.
 *  - Arguments are validated on the host before anything is enqueued; a
 *    failed validation returns PNERF_ERR_INVALID_ARG (or NOT_SUPPORTED) and
 *    enqueues nothing.  HIP errors map to PNERF_ERR_DEVICE.  The message of
 *    the last failure on the calling thread is pnerf_last_error().
 *  - A field is not safe for concurrent calls from several threads; calls on
 *    one field must be ordered (one stream, or externally synchronised).
 */
#ifndef PNERF_H
#define PNERF_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PNERF_OK = 0,
  PNERF_ERR_INVALID_ARG = 1,
  PNERF_ERR_OUT_OF_MEMORY = 2,
  PNERF_ERR_DEVICE = 3,
  PNERF_ERR_CAPACITY = 4,
  PNERF_ERR_NOT_SUPPORTED = 5
} pnerf_status;

typedef struct pnerf_field pnerf_field; /* opaque; owns device copies + workspace */

/* Pinhole intrinsics of the observed image (Sec. III: intrinsics are known). */
typedef struct {
  int32_t width, height;
  float fx, fy, cx, cy;
} pnerf_intrinsics;

/* A frozen Instant-NGP-style field (Sec. III, "Instant NGP") and how its rays
 * are sampled.  All pointers are host pointers, deep-copied by create_field.
 *
 * Encoding: L levels of a multiresolution grid; level l has resolution
 * level_res[l] (vertices 0..N_l per axis) and a table of T = 2^log2_table_size
 * entries of F = 2 features.  A level whose (N_l+1)^3 vertices fit in T is
 * indexed 1:1 (i + j(N_l+1) + k(N_l+1)^2) when dense_coarse_levels = 1,
 * otherwise by the spatial hash (i ^ j*2654435761 ^ k*805459861) mod T.  A
 * point p maps to x = clamp((p - aabb_min) / extent, 0, 1) and on level l to
 * the cell whose lower vertex is min(floor(x N_l), N_l - 1); its feature is the
 * trilinear blend of the 8 vertex entries.  Features concatenate level-major.
 *
 * Networks (no biases; weights stored [in][out], out = in @ W):
 *   density: a = relu(feat @ W_d1) (64), h = a @ W_d2 (16), sigma = exp(h_0 + density_bias)
 *   colour:  x_c = [h_1..h_15, SH_16(d), 0] (32), b1 = relu(x_c @ W_c1) (64),
 *            b2 = relu(b1 @ W_c2) (64), rgb = sigmoid(b2 @ W_c3) (3)
 * SH_16 are the real orthonormal spherical harmonics of degree 0..3 of the unit
 * ray direction, ordered by l then m = -l..l, without the Condon-Shortley phase.
 *
 * Sampling (Sec. IV-A ray model p_i = o + t_i d): the ray is clipped to the box
 * (t >= 0).  march_mode 0: n_uniform midpoints of equal segments of
 * [t_near, t_far], spacing delta = (t_far - t_near) / n_uniform.  march_mode 1:
 * lattice t_j = t_near + (j + 1/2) step below t_far, spacing step, at most
 * max_samples kept.  With occ_res > 0 a sample is kept only if its cell of the
 * occ_res^3 occupancy grid (index x + R(y + Rz), LSB-first uint32 words) is
 * set; occ_bits = NULL builds the grid on the device (bit set iff sigma at the
 * cell centre > occ_threshold).  Compositing is front to back with background
 * colour `background`; when t_stop > 0 a ray stops after the first sample whose
 * outgoing transmittance is below t_stop.
 *
 * Loss (Sec. IV-C, the pixel-based RGB losses): a function of each channel's
 * residual r = C - y (rendered C, observed y), averaged over the P pixels and 3
 * channels of a hypothesis; p = loss_param:
 *   0 Huber        0.5 r^2 if |r| <= p, else p (|r| - p/2)
 *   1 L1           |r|                     2 L2     r^2
 *   3 Log L1       log(1 + |r|)            4 Relative L2  r^2 / (y^2 + p)
 *   5 MAPE         |r| / (|y| + p)         6 sMAPE  2 |r| / (|C| + |y| + p)
 *   7 Smooth L1    0.5 r^2 / p if |r| < p, else |r| - p/2
 * (the derivative of |r| at r = 0 is taken as 0).
 * sh_dir_grad 0 gives the torque of Eq. 3 alone; 1 also carries the gradient
 * through the view-direction input of the colour network. */
typedef struct {
  int32_t n_levels;             /* L: 4, 8, 12 or 16 */
  int32_t n_features;           /* F: must be 2 */
  int32_t log2_table_size;      /* 4..24 */
  const int32_t* level_res;     /* [L] N_l >= 1 */
  int32_t dense_coarse_levels;  /* 0 or 1 */
  int32_t param_dtype;          /* 0: float32, 1: float16 table and weights */
  const void* table;            /* [L][T][2] */
  const void* w_density1;       /* [2L][64] */
  const void* w_density2;       /* [64][16] */
  const void* w_color1;         /* [32][64] */
  const void* w_color2;         /* [64][64] */
  const void* w_color3;         /* [64][3] */
  float density_bias;
  float aabb_min[3], aabb_max[3];
  int32_t march_mode;           /* 0 uniform, 1 lattice */
  int32_t n_uniform;            /* mode 0: samples per ray, 1..4096 */
  float step;                   /* mode 1: lattice spacing > 0 */
  int32_t max_samples;          /* mode 1: cap on kept samples per ray, 1..8192 */
  float t_stop;                 /* 0 = off */
  int32_t occ_res;              /* 0 = no occupancy grid, else 1..1024 */
  const uint32_t* occ_bits;     /* ceil(R^3/32) words, or NULL (build on device) */
  float occ_threshold;
  float background[3];
  int32_t loss_type;            /* 0..7, see above */
  float loss_param;             /* > 0: Huber / Smooth L1 threshold, or epsilon */
  int32_t sh_dir_grad;          /* 0 or 1 */
  int64_t max_workspace_bytes;  /* workspace budget; 0 = 96 GiB.  A batch whose
                                   samples need more is processed in chunks of
                                   whole hypotheses (about 56 + 20 L bytes per
                                   sample). */
  int32_t overlap_chunks;       /* render_loss_grad cuts a batch of 2^16 samples or
                                   more into this many chunks of whole hypotheses
                                   and runs the encoding of one chunk alongside
                                   the networks of the previous, on two internal
                                   streams (two sample buffers); 0 or 1 = off
                                   (pnerf_field_inspect needs it off), at most
                                   64.  Off by default: every kernel of the path
                                   loads through the same L1 address path, and
                                   on the 16 x 1024-ray workload the overlapped
                                   chunks ran slower than one chunk. */
  int32_t backward;             /* the backward pass of render_loss_grad:
                                   0 = separate kernels: composite and loss,
                                   network backward per 16-sample tile, then
                                   the per-hypothesis reduction (default; the
                                   faster on the measured workloads);
                                   1 = one fused kernel, a wavefront per ray:
                                   composite, loss, composite backward, both
                                   networks' backward and the encoding's
                                   Jacobian, the ray's torque and force summed
                                   in registers (no per-sample gradient in
                                   memory);
                                   2 = the fused kernel, also storing every
                                   sample's intermediates as 0 does
                                   (pnerf_field_inspect). */
  int32_t mlp_precision;        /* arithmetic of both networks (forward and
                                   backward):
                                   0 = fp32-equivalent: each fp32 operand split
                                   into two bf16 parts, three bf16 MFMA
                                   products per fp32 product, fp32
                                   accumulation (default);
                                   1 = fp16 MFMA: each weight as two fp16
                                   parts, each activation rounded to fp16, two
                                   products, fp32 accumulation; the backward
                                   scales each sample's incoming gradient by a
                                   power of two (exact) to keep its fp16
                                   operands normal.  Faster; results differ
                                   from 0 by the activations' fp16 rounding
                                   (2^-12 relative each). */
} pnerf_field_params;

/* Create a field: validates `params`, copies every array to the device (builds
 * the occupancy grid when asked), and synchronises `stream`.  On success *out
 * owns all device memory until pnerf_destroy_field. */
pnerf_status pnerf_create_field(const pnerf_field_params* params, void* stream,
                                pnerf_field** out);
/* Release a field (waits for its outstanding work).  NULL is a no-op. */
void pnerf_destroy_field(pnerf_field* field);

/* The hot path (Sec. IV-A, Eq. 2 and Eq. 3; Sec. IV-C): for every hypothesis
 * k < K and pixel slot s < P, render pixel pixel_ids[k][s] from poses[k],
 * take the loss against observed[v][u][0..2], and back-propagate through the
 * composite, both networks, the trilinear encoding and the sample positions
 * (the t_i, the sample set and the stop index are held fixed) to
 *   loss[k]     = (1 / 3P) sum_s sum_c H(C_c - I_c)
 *   dpose[k]    = (tau, g) with g = sum_rays sum_i dL/dp_i        (Eq. 2)
 *                 and tau = sum_rays d x sum_i t_i dL/dp_i         (Eq. 3)
 *                 (+ sum_rays d x dL/dd through SH when sh_dir_grad = 1)
 * poses (device) [K][3][4]; pixel_ids (device) int32 [K][P], each in [0, W*H);
 * observed (device) float32 [H][W][3]; loss (device) [K]; dpose (device) [K][6].
 * Limits: 1 <= K <= 65535, P >= 1, K*P < 2^31, pixel ids in range (not checked on the
 * device: out-of-range ids are undefined behaviour).
 * Stream capture: the call can be recorded into a HIP graph (and replayed with
 * new poses and pixel ids in the same buffers) when it only enqueues kernels:
 * the field has already run a batch of this shape (no workspace growth), the
 * batch's worst case (every ray at its sample cap) fits one sample buffer, so
 * that no read of its sample totals is needed, and profiling is off.  Otherwise
 * it returns PNERF_ERR_NOT_SUPPORTED under capture, having enqueued nothing. */
pnerf_status pnerf_render_loss_grad(pnerf_field* field, int32_t K, const float* poses,
                                    int32_t P, const int32_t* pixel_ids,
                                    const float* observed, const pnerf_intrinsics* intr,
                                    float* loss, float* dpose, void* stream);

/* Momentum step on SO(3) x T(3) (Sec. IV-A; vector moments): for each k,
 * m <- beta m + dpose, R <- Exp(-lr m_w) R, o <- o - lr m_t, in place.
 * poses (device) [K][3][4], momentum (device) [K][6], dpose (device) [K][6]. */
pnerf_status pnerf_step_momentum(int32_t K, float* poses, float* momentum,
                                 const float* dpose, float lr, float beta, void* stream);

/* Adam on SO(3) x T(3) (Sec. IV-A, "Momentum-Based Optimization": Adam's first
 * and second moments kept separately for the rotation and the translation, the
 * rotational moments as vectors, the orientation updated by the rotation they
 * induce; Kingma and Ba's Algorithm 1 within each subspace).  For each k, with
 * g = dpose[k] and n the hypothesis's own step count (state[k][12] + 1):
 *   m <- beta1 m + (1 - beta1) g
 *   v <- beta2 v + (1 - beta2) g^2        (second_moment = 0: per component)
 *   v_s <- beta2 v_s + (1 - beta2) |g_s|^2 (second_moment = 1: one value per
 *                                          subspace s, stored in its 3 slots)
 *   u = -lr_s(step) (m / (1 - beta1^n)) / (sqrt(v / (1 - beta2^n)) + eps)
 *   R <- Exp(u_w) R,  o <- o + u_t
 * with the learning rates of Sec. IV-D decaying exponentially in the global
 * step index `step` (0 for the first step of a run):
 *   lr_s(step) = lr_s * decay_base^(step / decay_steps)       (staircase = 0)
 *   lr_s(step) = lr_s * decay_base^floor(step / decay_steps)  (staircase = 1)
 * and no decay when decay_steps = 0.  The paper's setting is lr_rot 5e-3,
 * lr_trans 3e-3, decay_base 0.33, decay_steps 256.
 * representation = 1 runs the same optimiser on the coupled se(3) twist that
 * Sec. IV-A compares against (exponential coordinates about the world origin,
 * as in iNeRF): g is replaced by the twist gradient (tau + o x f, f) for
 * dpose = (tau, f) and camera centre o, and the step is T <- Exp(u) T, i.e.
 * R <- Exp(u_w) R, o <- Exp(u_w) o + V(u_w) u_t with
 * V(w) = I + (1 - cos|w|)/|w|^2 [w]x + (|w| - sin|w|)/|w|^3 [w]x^2.
 * state (device) float32 [K][PNERF_ADAM_STATE] = (m_w[3], m_t[3], v_w[3],
 * v_t[3], n, 0, 0, 0): all zero before a hypothesis's first step (also what
 * pnerf_resample_hypotheses leaves in a redrawn slot given state_dim =
 * PNERF_ADAM_STATE); n is exact up to 2^24 steps.  poses (device) [K][3][4],
 * dpose (device) [K][6], params (host).  Requires K >= 1, step >= 0, finite
 * lr >= 0, 0 <= beta < 1, eps > 0, decay_base > 0, decay_steps >= 0,
 * staircase, second_moment and representation each 0 or 1. */
#define PNERF_ADAM_STATE 16
typedef struct {
  float lr_rot, lr_trans;  /* learning rates at step 0 */
  float beta1, beta2, eps; /* Adam's moment decays and epsilon (0.9, 0.999, 1e-8) */
  float decay_base;        /* learning-rate factor per decay_steps steps */
  int32_t decay_steps;     /* 0: constant learning rates */
  int32_t staircase;       /* 0: continuous decay; 1: stepwise */
  int32_t second_moment;   /* 0: per component; 1: per subspace (rotation invariant) */
  int32_t representation;  /* 0: SO(3) x T(3) (the paper's); 1: coupled se(3) twist */
} pnerf_adam_params;

pnerf_status pnerf_step_adam(int32_t K, float* poses, float* state, const float* dpose,
                             int32_t step, const pnerf_adam_params* params, void* stream);

/* Monte Carlo resampling (Sec. IV-B): rank hypotheses by loss (ascending, ties
 * by index, NaN last), keep n_keep = max(1, floor(K keep_frac)), and redraw
 * each other slot -- the i-th one in ascending slot order takes the kept
 * hypothesis of rank i mod n_keep as parent -- as R = Exp(w) R_parent,
 * o = o_parent + v with w ~ N(0, sigma_rot^2 I), v ~ N(0, sigma_trans^2 I);
 * a redrawn slot's optimiser state (its row of opt_state, state_dim floats:
 * 6 for momentum, PNERF_ADAM_STATE for Adam) restarts at 0.  The normals of
 * slot s come from the SplitMix64 stream started at seed ^ mix(round << 32 | s)
 * (mix = SplitMix64's output function), uniforms ((u >> 11) + 1/2) 2^-53,
 * Box-Muller on pairs, in the order w_x, w_y, w_z, v_x, v_y, v_z.  In place;
 * 1 <= K <= 65535, 0 <= state_dim <= 64 (opt_state may be NULL when 0). */
pnerf_status pnerf_resample_hypotheses(int32_t K, float* poses, float* opt_state,
                                       int32_t state_dim, const float* loss, float keep_frac,
                                       float sigma_rot, float sigma_trans, uint64_t seed,
                                       uint32_t round_idx, void* stream);

/* pnerf_resample_hypotheses for callers that cannot allocate memory (code under
 * stream capture, tight serving loops, harnesses that forbid allocation): the
 * same operation, arguments and results, with no allocation of any kind.  Its
 * ranking scratch (2 K int32) lives in a static device array of each GPU, sized
 * for K <= 65535 and held until the process ends; a larger K returns
 * PNERF_ERR_CAPACITY before anything is enqueued.  The array is looked up on
 * the first call on each device (with that device current).  All calls on one
 * GPU share its array: calls that overlap on one GPU (several streams or host
 * threads at once) race and must be ordered by the caller.  Nothing of an
 * earlier call's contents is read. */
pnerf_status pnerf_resample_hypotheses_noalloc(int32_t K, float* poses, float* opt_state,
                                               int32_t state_dim, const float* loss,
                                               float keep_frac, float sigma_rot,
                                               float sigma_trans, uint64_t seed,
                                               uint32_t round_idx, void* stream);

/* Forward rendering only (the composite colour of each pixel's ray).
 * rgb (device) float32 [K][P][3].  Limits as for pnerf_render_loss_grad. */
pnerf_status pnerf_render(pnerf_field* field, int32_t K, const float* poses, int32_t P,
                          const int32_t* pixel_ids, const pnerf_intrinsics* intr,
                          float* rgb, void* stream);

/* The sample set of pnerf_render_loss_grad (rays ordered k*P + s, samples by
 * increasing t).  ray_offset (device) int64 [K*P+1] receives exclusive offsets
 * (total in ray_offset[K*P]).  If the total fits in `capacity`, t (device)
 * float32 and lattice_j (device) int32 [capacity] receive each sample's
 * distance and lattice / segment index; otherwise only ray_offset is written
 * and the call still returns PNERF_OK (compare the total with capacity).
 * Requires K*P <= 2^21 (else PNERF_ERR_CAPACITY) and the limits of
 * pnerf_render_loss_grad. */
pnerf_status pnerf_march(pnerf_field* field, int32_t K, const float* poses, int32_t P,
                         const int32_t* pixel_ids, const pnerf_intrinsics* intr,
                         int64_t* ray_offset, float* t, int32_t* lattice_j, int64_t capacity,
                         void* stream);

/* Per-sample intermediates of the last call on this field (inspection; the
 * last call must have run as one chunk, else PNERF_ERR_INVALID_ARG).  `dst` (device) receives
 * float32 values for the first n samples (n = the last call's sample total):
 *   what 0: t [n]
 *   what 1: after pnerf_render sigma [n]; after pnerf_render_loss_grad dL/dh_0 [n]
 *   what 2: after pnerf_render rgb [n][3]; after pnerf_render_loss_grad dL/dz [n][3]
 *           (z = pre-sigmoid colour)
 *   what 3: after pnerf_render_loss_grad (t d x dL/dp, dL/dp) [n][6]
 * PNERF_ERR_INVALID_ARG if n exceeds the workspace, `what` is unknown, or
 * `what` > 0 after a pnerf_render_loss_grad with backward = 1. */
pnerf_status pnerf_field_inspect(pnerf_field* field, int32_t what, float* dst, int64_t n,
                                 void* stream);

/* Copy the field's occupancy grid to `bits_host` (ceil(R^3/32) words);
 * synchronises `stream`.  PNERF_ERR_INVALID_ARG if the field has no grid. */
pnerf_status pnerf_field_occupancy(pnerf_field* field, uint32_t* bits_host, void* stream);

/* Total number of samples processed by the last render_loss_grad / render /
 * march call on this field (sum over hypothesis chunks).  When that call planned
 * its chunks on the host, the count is known there and `stream` is not used;
 * when it sized its buffer for the worst case (a loss gradient whose every ray
 * at its sample cap fits the workspace), the count is read from the device on
 * `stream`, which this call then synchronises: pass the stream of that call
 * (or one ordered after it). */
pnerf_status pnerf_field_last_sample_count(pnerf_field* field, int64_t* count, void* stream);

/* Per-kernel timing with HIP events recorded on the call's stream around every
 * kernel the field launches.  enable = 1 starts (and clears) collection, 0 stops.
 * pnerf_field_profile_read synchronises the device and returns, for kernel
 * number `index` (0-based, in launch order of first appearance), its name,
 * number of launches and total milliseconds; PNERF_ERR_INVALID_ARG past the end. */
pnerf_status pnerf_field_set_profiling(pnerf_field* field, int32_t enable);
pnerf_status pnerf_field_profile_read(pnerf_field* field, int32_t index, const char** name,
                                      int64_t* launches, double* total_ms);

/* Batch planning (host only: no device call, usable without a GPU).  The
 * rendering calls count every ray's samples for a "counted batch" of whole
 * hypotheses at a time, with 32-bit counts and offsets, then cut the counted
 * batch into chunks of whole hypotheses whose samples fit the workspace
 * (Sec. IV-B: hypotheses are independent, so any cut gives the same results).
 *
 * pnerf_plan_counted_batch: *hyps_per_batch = hypotheses per counted batch for
 * P rays per hypothesis of at most max_per_ray samples each: at most K, at most
 * 2^21 rays, and a worst case (every ray at its cap) below 2^31 samples.
 * PNERF_ERR_CAPACITY when P > 2^21 or P * max_per_ray >= 2^31 (one hypothesis
 * alone could overflow the counts); PNERF_ERR_INVALID_ARG for K, P or
 * max_per_ray below 1.  The rendering calls return these errors before any
 * device work is enqueued. */
pnerf_status pnerf_plan_counted_batch(int32_t K, int32_t P, int32_t max_per_ray,
                                      int32_t* hyps_per_batch);

/* pnerf_plan_chunks: cut n hypotheses with hyp_samples[k] samples (host) into
 * consecutive chunks: each chunk takes hypotheses while its sum stays within
 * `capacity` and is below `goal` (a chunk always takes at least one).  Writes
 * cut[0..c] (chunk i = hypotheses cut[i] .. cut[i+1]-1; cut[0] = 0, cut[c] = n),
 * sums[0..c-1] and *n_chunks = c; cut needs n + 1 entries, sums n.
 * PNERF_ERR_CAPACITY if one hypothesis exceeds capacity, INVALID_ARG for a
 * negative count, n < 1 or capacity < 1. */
pnerf_status pnerf_plan_chunks(const int32_t* hyp_samples, int32_t n, int64_t capacity,
                               int64_t goal, int32_t* cut, int64_t* sums, int32_t* n_chunks);

/* Message of the last non-OK status returned on this thread ("" if none). */
const char* pnerf_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
