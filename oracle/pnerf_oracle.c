/*
 * CPU oracle for the parallel-NeRF-inversion hot path.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path.  Shares no code with
 * the HIP implementation.  Plain loops, double precision for every continuous
 * quantity; float only where floating point decides an integer (sample
 * existence and placement, occupancy cell, hash-grid cell, clamping), written
 * with a fixed operation order and built with -ffp-contract=off.
 *
 * Paper: Lin et al., "Parallel Inversion of Neural Radiance Fields for Robust
 * Pose Estimation" (arXiv 2210.10108).  Section references are to that paper.
 */
#include "pnerf_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define HID 64
#define DOUT 16
#define CIN 32

/* ------------------------------------------------------------------ hashing */
/* Multiresolution hash encoding (Sec. III, "Instant NGP"): a vertex of a coarse
 * level whose full grid fits the table is stored 1:1; otherwise its index is
 * the xor of coordinate * prime (primes 1, 2654435761, 805459861) modulo T. */
uint32_t orc_grid_index(const orc_field* f, int32_t level, uint32_t i, uint32_t j,
                        uint32_t k) {
  uint64_t n1 = (uint64_t)f->level_res[level] + 1u;
  if (f->dense_coarse && n1 * n1 * n1 <= (uint64_t)f->T)
    return (uint32_t)((uint64_t)i + (uint64_t)j * n1 + (uint64_t)k * n1 * n1);
  uint32_t h = (i * 1u) ^ (j * 2654435761u) ^ (k * 805459861u);
  return h % f->T;
}

/* ------------------------------------------------------------- rays (float) */
/* A pixel's ray starts at the camera centre o (the translation of the pose) and
 * runs along the pixel's viewing direction d (Sec. IV-A, the ray model
 * p_i = o + t_i d).  Pinhole camera, OpenCV axes, pixel centres at +0.5. */
void orc_ray_f32(const float pose[12], const orc_intr* in, int32_t pix, float o[3],
                 float d[3]) {
  int32_t u = pix % in->width, v = pix / in->width;
  float xc = ((float)u + 0.5f - in->cx) / in->fx;
  float yc = ((float)v + 0.5f - in->cy) / in->fy;
  float dw[3];
  for (int a = 0; a < 3; ++a) {
    const float* row = pose + 4 * a;
    dw[a] = (row[0] * xc + row[1] * yc) + row[2];
    o[a] = row[3];
  }
  float n = sqrtf((dw[0] * dw[0] + dw[1] * dw[1]) + dw[2] * dw[2]);
  for (int a = 0; a < 3; ++a) d[a] = dw[a] / n;
}

/* Same ray in double for the continuous path. */
static void ray_f64(const double pose[12], const orc_intr* in, int32_t pix, double o[3],
                    double d[3]) {
  int32_t u = pix % in->width, v = pix / in->width;
  double xc = ((double)u + 0.5 - (double)in->cx) / (double)in->fx;
  double yc = ((double)v + 0.5 - (double)in->cy) / (double)in->fy;
  double dw[3], n = 0.0;
  for (int a = 0; a < 3; ++a) {
    const double* row = pose + 4 * a;
    dw[a] = row[0] * xc + row[1] * yc + row[2];
    o[a] = row[3];
    n += dw[a] * dw[a];
  }
  n = sqrt(n);
  for (int a = 0; a < 3; ++a) d[a] = dw[a] / n;
}

/* Slab test against the scene box; t_near is clipped at the camera (t >= 0). */
static int slab_f32(const orc_field* f, const float o[3], const float d[3], float* tn,
                    float* tf) {
  float t_entry = -INFINITY, t_exit = INFINITY;
  for (int a = 0; a < 3; ++a) {
    if (d[a] != 0.0f) {
      float t1 = (f->aabb_min[a] - o[a]) / d[a];
      float t2 = (f->aabb_max[a] - o[a]) / d[a];
      float lo = t1 < t2 ? t1 : t2, hi = t1 < t2 ? t2 : t1;
      if (lo > t_entry) t_entry = lo;
      if (hi < t_exit) t_exit = hi;
    } else if (o[a] < f->aabb_min[a] || o[a] > f->aabb_max[a]) {
      *tn = 0.0f;
      *tf = 0.0f;
      return 0;
    }
  }
  *tn = t_entry > 0.0f ? t_entry : 0.0f;
  *tf = t_exit;
  return *tf > *tn;
}

/* Occupancy test of the point o + t d (float decision path). */
static int occupied_f32(const orc_field* f, const float o[3], const float d[3], float t) {
  if (f->occ_res <= 0) return 1;
  int32_t R = f->occ_res;
  uint32_t c[3];
  for (int a = 0; a < 3; ++a) {
    float p = o[a] + t * d[a];
    float ext = f->aabb_max[a] - f->aabb_min[a];
    float s = (float)R / ext;
    float q = (p - f->aabb_min[a]) * s;
    int32_t ci = q < 0.0f ? 0 : (q >= (float)R ? R - 1 : (int32_t)q);
    c[a] = (uint32_t)ci;
  }
  uint64_t idx = (uint64_t)c[0] + (uint64_t)R * ((uint64_t)c[1] + (uint64_t)R * c[2]);
  return (int)((f->occ_bits[idx >> 5] >> (idx & 31u)) & 1u);
}

/* Samples of one ray, in order of increasing t.  Uniform mode: midpoints of
 * n_uniform equal segments of [t_near, t_far].  Lattice mode: points
 * t_near + (j + 1/2) step below t_far.  Either way a sample survives only if
 * its occupancy cell is set, and lattice mode keeps at most max_samples.
 * With t == NULL only counts.  Returns the number kept. */
static int32_t march_ray(const orc_field* f, const float o[3], const float d[3], float* t,
                         int32_t* jout, float* delta) {
  float tn, tf;
  int hit = slab_f32(f, o, d, &tn, &tf);
  int32_t kept = 0;
  if (f->march_mode == 0) {
    float dt = hit ? (tf - tn) / (float)f->n_uniform : 0.0f;
    if (delta) *delta = dt;
    if (!hit) return 0;
    for (int32_t j = 0; j < f->n_uniform; ++j) {
      float tj = tn + ((float)j + 0.5f) * dt;
      if (!occupied_f32(f, o, d, tj)) continue;
      if (t) {
        t[kept] = tj;
        jout[kept] = j;
      }
      ++kept;
    }
    return kept;
  }
  if (delta) *delta = f->step;
  if (!hit) return 0;
  for (int32_t j = 0; kept < f->max_samples; ++j) {
    float tj = tn + ((float)j + 0.5f) * f->step;
    if (!(tj < tf)) break;
    if (!occupied_f32(f, o, d, tj)) continue;
    if (t) {
      t[kept] = tj;
      jout[kept] = j;
    }
    ++kept;
  }
  return kept;
}

int32_t orc_march(const orc_field* f, int32_t K, const float* poses, int32_t P,
                  const int32_t* pix, const orc_intr* in, int64_t* ray_offset, float* t,
                  int32_t* lattice_j, float* delta, int64_t capacity, int32_t n_threads) {
  int64_t n_rays = (int64_t)K * P;
  if (n_threads < 1) n_threads = 1;
  /* rays are independent: count each ray's samples, then offsets in ray order */
  ray_offset[0] = 0;
#pragma omp parallel for schedule(dynamic, 64) num_threads(n_threads)
  for (int64_t r = 0; r < n_rays; ++r) {
    float o[3], d[3], dl;
    orc_ray_f32(poses + 12 * (r / P), in, pix[r], o, d);
    ray_offset[r + 1] = march_ray(f, o, d, NULL, NULL, &dl);
    if (delta) delta[r] = dl;
  }
  for (int64_t r = 0; r < n_rays; ++r) ray_offset[r + 1] += ray_offset[r];
  if (ray_offset[n_rays] > capacity) return 1;
  if (!t) return 0;
#pragma omp parallel for schedule(dynamic, 64) num_threads(n_threads)
  for (int64_t r = 0; r < n_rays; ++r) {
    float o[3], d[3];
    orc_ray_f32(poses + 12 * (r / P), in, pix[r], o, d);
    march_ray(f, o, d, t + ray_offset[r], lattice_j + ray_offset[r], NULL);
  }
  return 0;
}

/* ---------------------------------------------------------------- encoding */
/* Trilinear interpolation of the 8 vertex features of the cell containing the
 * point on every level, features concatenated level-major (Sec. III).  The
 * cell is chosen from the float position x32 (pos = x N_l, vertex grid
 * 0..N_l, lower corner clamped to N_l - 1); the interpolation weights use the
 * double position x64.  jac[a][q] = d feat[q] / d x_a, zero along clamped
 * components. */
void orc_encode(const orc_field* f, const float x32[3], const double x64[3],
                const int32_t clamped[3], double* feat, double* jac) {
  int32_t din = f->L * f->F;
  for (int32_t q = 0; q < din; ++q) feat[q] = 0.0;
  if (jac)
    for (int32_t q = 0; q < 3 * din; ++q) jac[q] = 0.0;
  for (int32_t l = 0; l < f->L; ++l) {
    int32_t N = f->level_res[l];
    int32_t i0[3];
    double w[3];
    for (int a = 0; a < 3; ++a) {
      float pos = x32[a] * (float)N;
      int32_t c = (int32_t)pos; /* pos >= 0: truncation is floor */
      if (c > N - 1) c = N - 1;
      i0[a] = c;
      w[a] = x64[a] * (double)N - (double)c;
    }
    for (int corner = 0; corner < 8; ++corner) {
      int b[3] = {corner & 1, (corner >> 1) & 1, (corner >> 2) & 1};
      uint32_t idx = orc_grid_index(f, l, (uint32_t)(i0[0] + b[0]), (uint32_t)(i0[1] + b[1]),
                                    (uint32_t)(i0[2] + b[2]));
      double wa[3], sa[3];
      for (int a = 0; a < 3; ++a) {
        wa[a] = b[a] ? w[a] : 1.0 - w[a];
        sa[a] = b[a] ? 1.0 : -1.0;
      }
      double weight = wa[0] * wa[1] * wa[2];
      const double* v = f->table + ((size_t)l * f->T + idx) * (size_t)f->F;
      for (int32_t q = 0; q < f->F; ++q) {
        feat[l * f->F + q] += weight * v[q];
        if (!jac) continue;
        double dw[3] = {sa[0] * wa[1] * wa[2], wa[0] * sa[1] * wa[2], wa[0] * wa[1] * sa[2]};
        for (int a = 0; a < 3; ++a)
          if (!clamped[a]) jac[a * din + l * f->F + q] += dw[a] * (double)N * v[q];
      }
    }
  }
}

/* ------------------------------------------------ spherical harmonics (view) */
/* Real orthonormal spherical harmonics of degree 0..3 (16 functions, ordered
 * by l then m = -l..l, no Condon-Shortley phase) of the view direction: the
 * direction input of the 5-D radiance field (Sec. III, "NeRF").  grad[q][a] is
 * the derivative of the polynomial w.r.t. d_a. */
void orc_sh16(const double d[3], double out[16], double grad[16][3]) {
  const double pi = 3.14159265358979323846;
  double x = d[0], y = d[1], z = d[2];
  double c0 = 0.5 * sqrt(1.0 / pi);
  double c1 = sqrt(3.0 / (4.0 * pi));
  double c2a = 0.5 * sqrt(15.0 / pi), c2b = 0.25 * sqrt(5.0 / pi), c2c = 0.25 * sqrt(15.0 / pi);
  double c3a = 0.25 * sqrt(35.0 / (2.0 * pi)), c3b = 0.5 * sqrt(105.0 / pi);
  double c3c = 0.25 * sqrt(21.0 / (2.0 * pi)), c3d = 0.25 * sqrt(7.0 / pi);
  double c3e = 0.25 * sqrt(105.0 / pi);
  double v[16] = {
      c0,
      c1 * y, c1 * z, c1 * x,
      c2a * x * y, c2a * y * z, c2b * (3.0 * z * z - 1.0), c2a * x * z, c2c * (x * x - y * y),
      c3a * y * (3.0 * x * x - y * y), c3b * x * y * z, c3c * y * (5.0 * z * z - 1.0),
      c3d * z * (5.0 * z * z - 3.0), c3c * x * (5.0 * z * z - 1.0), c3e * z * (x * x - y * y),
      c3a * x * (x * x - 3.0 * y * y)};
  double g[16][3] = {
      {0, 0, 0},
      {0, c1, 0}, {0, 0, c1}, {c1, 0, 0},
      {c2a * y, c2a * x, 0}, {0, c2a * z, c2a * y}, {0, 0, c2b * 6.0 * z}, {c2a * z, 0, c2a * x},
      {c2c * 2.0 * x, -c2c * 2.0 * y, 0},
      {c3a * 6.0 * x * y, c3a * (3.0 * x * x - 3.0 * y * y), 0},
      {c3b * y * z, c3b * x * z, c3b * x * y},
      {0, c3c * (5.0 * z * z - 1.0), c3c * 10.0 * y * z},
      {0, 0, c3d * (15.0 * z * z - 3.0)},
      {c3c * (5.0 * z * z - 1.0), 0, c3c * 10.0 * x * z},
      {c3e * 2.0 * x * z, -c3e * 2.0 * y * z, c3e * (x * x - y * y)},
      {c3a * (3.0 * x * x - 3.0 * y * y), -c3a * 6.0 * x * y, 0}};
  for (int q = 0; q < 16; ++q) {
    out[q] = v[q];
    if (grad)
      for (int a = 0; a < 3; ++a) grad[q][a] = g[q][a];
  }
}

/* ---------------------------------------------------------------- the MLPs */
/* Density network: h = W_d2^T relu(W_d1^T feat); sigma = exp(h_0 + bias);
 * h_1..h_15 feed the colour network. */
static void density_fwd(const orc_field* f, const double* feat, double a_pre[HID],
                        double h[DOUT]) {
  for (int j = 0; j < HID; ++j) {
    double s = 0.0;
    for (int i = 0; i < f->din; ++i) s += feat[i] * f->wd1[i * HID + j];
    a_pre[j] = s;
  }
  for (int o = 0; o < DOUT; ++o) {
    double s = 0.0;
    for (int j = 0; j < HID; ++j) s += (a_pre[j] > 0.0 ? a_pre[j] : 0.0) * f->wd2[j * DOUT + o];
    h[o] = s;
  }
}

void orc_density_mlp(const orc_field* f, const double* feat, double h[16]) {
  double a[HID];
  density_fwd(f, feat, a, h);
}

/* Colour network: rgb = sigmoid(W_c3^T relu(W_c2^T relu(W_c1^T x_c))). */
static void color_fwd(const orc_field* f, const double xc[CIN], double b1[HID], double b2[HID],
                      double rgb[3]) {
  for (int j = 0; j < HID; ++j) {
    double s = 0.0;
    for (int i = 0; i < CIN; ++i) s += xc[i] * f->wc1[i * HID + j];
    b1[j] = s;
  }
  for (int j = 0; j < HID; ++j) {
    double s = 0.0;
    for (int i = 0; i < HID; ++i) s += (b1[i] > 0.0 ? b1[i] : 0.0) * f->wc2[i * HID + j];
    b2[j] = s;
  }
  for (int c = 0; c < 3; ++c) {
    double s = 0.0;
    for (int i = 0; i < HID; ++i) s += (b2[i] > 0.0 ? b2[i] : 0.0) * f->wc3[i * 3 + c];
    rgb[c] = 1.0 / (1.0 + exp(-s));
  }
}

void orc_color_mlp(const orc_field* f, const double xc[32], double rgb[3]) {
  double b1[HID], b2[HID];
  color_fwd(f, xc, b1, b2, rgb);
}

/* --------------------------------------------------------------- composite */
/* Classic volume rendering (Sec. III, "NeRF"), front to back:
 * alpha_i = 1 - exp(-sigma_i delta), w_i = T_i alpha_i, T_{i+1} = T_i exp(-sigma_i delta),
 * C = sum_i w_i c_i + T_end bg.  With t_stop > 0, sample i is the last one
 * composited once T_{i+1} < t_stop.  trans[] holds T_0..T_{n_used}. */
void orc_composite(int32_t n, const double* sigma, const double* rgb, double delta,
                   const double bg[3], double t_stop, double C[3], double* trans,
                   double* weight, int32_t* n_used) {
  double T = 1.0;
  int32_t used = n;
  C[0] = C[1] = C[2] = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    double e = exp(-sigma[i] * delta);
    double w = T * (1.0 - e);
    trans[i] = T;
    weight[i] = w;
    for (int c = 0; c < 3; ++c) C[c] += w * rgb[3 * i + c];
    T *= e;
    if (t_stop > 0.0 && T < t_stop) {
      used = i + 1;
      break;
    }
  }
  trans[used] = T;
  for (int c = 0; c < 3; ++c) C[c] += T * bg[c];
  *n_used = used;
}

/* Backward of the composite: dC/dc_i = w_i and
 * dC/dsigma_i = delta (T_{i+1} c_i - S_i), S_i = sum_{j>i} w_j c_j + T_end bg. */
void orc_composite_grad(int32_t n, const double* sigma, const double* rgb, double delta,
                        const double bg[3], double t_stop, const double gC[3],
                        double* g_sigma, double* g_rgb) {
  double* trans = (double*)malloc(sizeof(double) * (size_t)(n + 1));
  double* weight = (double*)malloc(sizeof(double) * (size_t)(n + 1));
  double C[3];
  int32_t used;
  orc_composite(n, sigma, rgb, delta, bg, t_stop, C, trans, weight, &used);
  double S[3];
  for (int c = 0; c < 3; ++c) S[c] = trans[used] * bg[c];
  for (int32_t i = n - 1; i >= 0; --i) {
    if (i >= used) {
      g_sigma[i] = 0.0;
      for (int c = 0; c < 3; ++c) g_rgb[3 * i + c] = 0.0;
      continue;
    }
    double t_next = trans[i] * exp(-sigma[i] * delta);
    double gs = 0.0;
    for (int c = 0; c < 3; ++c) {
      gs += gC[c] * (t_next * rgb[3 * i + c] - S[c]);
      g_rgb[3 * i + c] = weight[i] * gC[c];
    }
    g_sigma[i] = delta * gs;
    for (int c = 0; c < 3; ++c) S[c] += weight[i] * rgb[3 * i + c];
  }
  free(trans);
  free(weight);
}

/* ------------------------------------------------------------------ loss */
/* Pixel-based RGB losses of one channel (Sec. IV-C), residual r = C - y of the
 * rendered value C against the observed y.  p is the loss parameter: the
 * threshold of Huber (0) and Smooth L1 (7), the epsilon of the relative losses
 * (4, 5, 6); unused by L1 (1), L2 (2) and Log L1 (3).  Returns the loss and
 * writes d loss / d C, a code of the branch taken (signature of the discrete
 * decision), and the distance of r (or C) from the nearest point where the
 * derivative jumps (INFINITY when there is none).
 *   0 Huber       0.5 r^2 (|r| <= p), p (|r| - p / 2)
 *   1 L1          |r|
 *   2 L2          r^2
 *   3 Log L1      log(1 + |r|)
 *   4 Relative L2 r^2 / (y^2 + p)
 *   5 MAPE        |r| / (|y| + p)
 *   6 sMAPE       2 |r| / (|C| + |y| + p)
 *   7 Smooth L1   0.5 r^2 / p (|r| < p), |r| - p / 2 */
static double pixel_loss(int type, double C, double y, double p, int force_sign, double* grad,
                         int* branch, double* kink) {
  const double r = C - y, ar = fabs(r);
  /* the sign of r in the derivative; force_sign = +1 / -1 takes the derivative
   * on that side of r = 0 (the other valid choice next to the jump) */
  const double sr = force_sign ? (double)force_sign : (r > 0.0 ? 1.0 : (r < 0.0 ? -1.0 : 0.0));
  *branch = r > 0.0 ? 1 : (r < 0.0 ? 2 : 0);
  *kink = INFINITY;
  switch (type) {
    case 0:
      if (ar <= p) {
        *grad = r;
        *branch = 0;
        return 0.5 * r * r;
      }
      *grad = p * sr;
      return p * (ar - 0.5 * p);
    case 1:
      *grad = sr;
      *kink = ar;
      return ar;
    case 2:
      *grad = 2.0 * r;
      *branch = 0;
      return r * r;
    case 3:
      *grad = sr / (1.0 + ar);
      *kink = ar;
      return log1p(ar);
    case 4: {
      const double den = y * y + p;
      *grad = 2.0 * r / den;
      *branch = 0;
      return r * r / den;
    }
    case 5: {
      const double den = fabs(y) + p;
      *grad = sr / den;
      *kink = ar;
      return ar / den;
    }
    case 6: {
      const double den = fabs(C) + fabs(y) + p;
      const double sc = C > 0.0 ? 1.0 : (C < 0.0 ? -1.0 : 0.0);
      *grad = 2.0 * sr / den - 2.0 * ar * sc / (den * den);
      *branch = 3 * *branch + (C > 0.0 ? 1 : (C < 0.0 ? 2 : 0));
      *kink = ar < fabs(C) ? ar : fabs(C);
      return 2.0 * ar / den;
    }
    default:  /* 7 */
      if (ar < p) {
        *grad = r / p;
        *branch = 0;
        return 0.5 * r * r / p;
      }
      /* C^1 at |r| = p: r / p and sign(r) meet, no jump of the derivative */
      *grad = sr;
      return ar - 0.5 * p;
  }
}

/* One channel's loss for testing: value, derivative and kink distance. */
double orc_pixel_loss(int32_t type, double C, double y, double p, double* grad, double* kink) {
  int br;
  return pixel_loss(type, C, y, p, 0, grad, &br, kink);
}

/* ------------------------------------------------------------- signature */
static uint64_t fnv(uint64_t h, int64_t v) {
  for (int b = 0; b < 8; ++b) {
    h ^= (uint64_t)((v >> (8 * b)) & 0xff);
    h *= 1099511628211ull;
  }
  return h;
}

/* ------------------------------------------------------------------ shade */
typedef struct {
  double feat[CIN];
  double jac[3 * CIN];
  double a_pre[HID], h[DOUT], b1[HID], b2[HID];
  double rgb[3], sigma;
  unsigned char flip[3][HID]; /* variant: ReLU backward masks taken the other way */
} sample_state;

/* Relative margin of one ReLU decision: |pre-activation| over the sum of its
 * terms' magnitudes (INFINITY when every term is zero). */
static double relu_margin(double pre, double magnitude) {
  return magnitude > 0.0 ? fabs(pre) / magnitude : INFINITY;
}

/* One ray: forward, loss, backward.  Returns per-ray loss, force G = sum_i
 * dL/dp_i and torque tau = d x sum_i t_i dL/dp_i (+ d x dL/dd through the SH
 * path when enabled) -- Eq. (2) and Eq. (3). */
static void shade_ray(const orc_field* f, const double pose64[12], const orc_intr* in,
                      int32_t pix, const float* obs, const float* ts, int32_t n, float delta32,
                      const double* sh_dir, int32_t P, const orc_variant* var, double* loss_out,
                      double g_out[6], double rgb_out[3], int32_t* stop_out, uint64_t* sig,
                      double* s_out, int32_t* near_out) {
  float pose32[12];
  for (int q = 0; q < 12; ++q) pose32[q] = (float)pose64[q];
  float o32[3], d32[3];
  orc_ray_f32(pose32, in, pix, o32, d32);
  double o[3], d[3];
  ray_f64(pose64, in, pix, o, d);
  const double* dsh = sh_dir ? sh_dir : d;
  double sh[16], shg[16][3];
  orc_sh16(dsh, sh, shg);
  double delta = (double)delta32;

  sample_state* st = (sample_state*)calloc((size_t)(n > 0 ? n : 1), sizeof(sample_state));
  double* sig_s = (double*)malloc(sizeof(double) * (size_t)(n + 1));
  double* rgb_s = (double*)malloc(sizeof(double) * 3 * (size_t)(n + 1));
  uint64_t h = 1469598103934665603ull;

  for (int32_t i = 0; i < n; ++i) {
    sample_state* s = st + i;
    float t32 = ts[i];
    double t = (double)t32;
    float x32[3];
    double x64[3];
    int32_t cl[3];
    for (int a = 0; a < 3; ++a) {
      float ext32 = f->aabb_max[a] - f->aabb_min[a];
      float inv32 = 1.0f / ext32;
      float p32 = o32[a] + t32 * d32[a];
      float xr = (p32 - f->aabb_min[a]) * inv32;
      double ext = (double)f->aabb_max[a] - (double)f->aabb_min[a];
      double xd = (o[a] + t * d[a] - (double)f->aabb_min[a]) / ext;
      if (xr < 0.0f) {
        x32[a] = 0.0f; x64[a] = 0.0; cl[a] = 1;
      } else if (xr > 1.0f) {
        x32[a] = 1.0f; x64[a] = 1.0; cl[a] = 1;
      } else {
        x32[a] = xr; x64[a] = xd; cl[a] = 0;
      }
      h = fnv(h, cl[a]);
    }
    orc_encode(f, x32, x64, cl, s->feat, s->jac);
    for (int32_t l = 0; l < f->L; ++l)
      for (int a = 0; a < 3; ++a) {
        float pos = x32[a] * (float)f->level_res[l];
        h = fnv(h, (int64_t)pos);
      }
    density_fwd(f, s->feat, s->a_pre, s->h);
    s->sigma = exp(s->h[0] + f->density_bias);
    double xc[CIN];
    for (int q = 0; q < 15; ++q) xc[q] = s->h[1 + q];
    for (int q = 0; q < 16; ++q) xc[15 + q] = sh[q];
    xc[31] = 0.0;
    color_fwd(f, xc, s->b1, s->b2, s->rgb);
    /* decision margins of the ReLUs (density layer 1, colour layers 1 and 2),
     * for comparing against float kernels; the smallest one is reported, and a
     * variant flips the backward mask of chosen units whose margin is below
     * var->relu_margin (numbered layer by layer, unit by unit) */
    double lm[3][HID];
    for (int j = 0; j < HID; ++j) {
      double m0 = 0.0, m1 = 0.0, m2 = 0.0;
      for (int q = 0; q < f->din; ++q) m0 += fabs(s->feat[q] * f->wd1[q * HID + j]);
      for (int q = 0; q < CIN; ++q) m1 += fabs(xc[q] * f->wc1[q * HID + j]);
      for (int q = 0; q < HID; ++q) m2 += fabs((s->b1[q] > 0.0 ? s->b1[q] : 0.0) * f->wc2[q * HID + j]);
      lm[0][j] = relu_margin(s->a_pre[j], m0);
      lm[1][j] = relu_margin(s->b1[j], m1);
      lm[2][j] = relu_margin(s->b2[j], m2);
    }
    double margin = INFINITY;
    int32_t near = 0;
    memset(s->flip, 0, sizeof(s->flip));
    for (int layer = 0; layer < 3; ++layer)
      for (int j = 0; j < HID; ++j) {
        if (lm[layer][j] < margin) margin = lm[layer][j];
        if (var && lm[layer][j] < var->relu_margin) {
          const int32_t pat = var->relu_pattern ? var->relu_pattern[i] : var->relu_pattern_all;
          if (near < 31 && ((pat >> near) & 1)) s->flip[layer][j] = 1;
          ++near;
        }
      }
    if (near_out) near_out[i] = near;
    for (int j = 0; j < HID; ++j) {
      h = fnv(h, s->a_pre[j] > 0.0);
      h = fnv(h, s->b1[j] > 0.0);
      h = fnv(h, s->b2[j] > 0.0);
    }
    sig_s[i] = s->sigma;
    for (int c = 0; c < 3; ++c) rgb_s[3 * i + c] = s->rgb[c];
    if (s_out) {
      double* so = s_out + ORC_SAMPLE_COLS * (size_t)i;
      for (int q = 0; q < ORC_SAMPLE_COLS; ++q) so[q] = 0.0;
      so[0] = s->sigma;
      for (int c = 0; c < 3; ++c) so[1 + c] = s->rgb[c];
      so[11] = margin;
    }
  }

  double* trans = (double*)malloc(sizeof(double) * (size_t)(n + 1));
  double* weight = (double*)malloc(sizeof(double) * (size_t)(n + 1));
  double C[3];
  int32_t used;
  /* a variant may composite a given number of samples instead of testing the
   * transmittance (the stop decision taken the other way) */
  const int forced = var && var->stop >= 0;
  const int32_t n_c = forced ? (var->stop < n ? var->stop : n) : n;
  const double t_stop = forced ? 0.0 : f->t_stop;
  orc_composite(n_c, sig_s, rgb_s, delta, f->bg, t_stop, C, trans, weight, &used);
  h = fnv(h, used);
  if (stop_out) *stop_out = used;
  if (rgb_out)
    for (int c = 0; c < 3; ++c) rgb_out[c] = C[c];

  /* loss: mean over the P pixels of the hypothesis and the 3 channels */
  const float* I = obs + 3 * (size_t)pix;
  double gC[3], L = 0.0, norm = 1.0 / (3.0 * (double)P);
  double kink = INFINITY;
  for (int c = 0; c < 3; ++c) {
    double g, km;
    int br;
    const int fs = var ? var->loss_sign[c] : 0;
    L += pixel_loss(f->loss_type, C[c], (double)I[c], f->loss_param, fs, &g, &br, &km) * norm;
    gC[c] = g * norm;
    h = fnv(h, br);
    if (km < kink) kink = km;
  }
  *loss_out = L;
  /* distance of the stop decision from its threshold, relative to it.  The
   * test T_{i+1} < t_stop runs after each sample i; the decisions next to the
   * crossing are T_used (the first below, when the ray stopped before its last
   * sample) and T_{used-1} (the last one at or above, tested when used >= 2). */
  double stop_margin = INFINITY;
  if (t_stop > 0.0 && used > 0) {
    if (used < n) stop_margin = fabs(trans[used] - t_stop) / t_stop;
    if (used >= 2) {
      const double mp = fabs(trans[used - 1] - t_stop) / t_stop;
      if (mp < stop_margin) stop_margin = mp;
    }
  }
  if (s_out)
    for (int32_t i = 0; i < n; ++i) {
      s_out[ORC_SAMPLE_COLS * (size_t)i + 12] = kink;
      s_out[ORC_SAMPLE_COLS * (size_t)i + 16] = stop_margin;
    }

  /* backward through the composite, then each sample's networks and encoding */
  double* g_sig = (double*)malloc(sizeof(double) * (size_t)(n + 1));
  double* g_rgb = (double*)malloc(sizeof(double) * 3 * (size_t)(n + 1));
  orc_composite_grad(n_c, sig_s, rgb_s, delta, f->bg, t_stop, gC, g_sig, g_rgb);
  for (int32_t i = n_c; i < n; ++i) {
    g_sig[i] = 0.0;
    for (int c = 0; c < 3; ++c) g_rgb[3 * i + c] = 0.0;
  }
  double G[3] = {0, 0, 0}, M[3] = {0, 0, 0}, gd[3] = {0, 0, 0};
  int32_t din = f->din;
  for (int32_t i = 0; i < used; ++i) {
    sample_state* s = st + i;
    double t = (double)ts[i];
    double gz[3], gb2[HID], gb1[HID], gxc[CIN], gh[DOUT], ga[HID], gf[CIN];
    for (int c = 0; c < 3; ++c) gz[c] = g_rgb[3 * i + c] * s->rgb[c] * (1.0 - s->rgb[c]);
    for (int j = 0; j < HID; ++j) {
      double acc = 0.0;
      for (int c = 0; c < 3; ++c) acc += f->wc3[j * 3 + c] * gz[c];
      gb2[j] = ((s->b2[j] > 0.0) != s->flip[2][j]) ? acc : 0.0;
    }
    for (int j = 0; j < HID; ++j) {
      double acc = 0.0;
      for (int k = 0; k < HID; ++k) acc += f->wc2[j * HID + k] * gb2[k];
      gb1[j] = ((s->b1[j] > 0.0) != s->flip[1][j]) ? acc : 0.0;
    }
    for (int q = 0; q < CIN; ++q) {
      double acc = 0.0;
      for (int j = 0; j < HID; ++j) acc += f->wc1[q * HID + j] * gb1[j];
      gxc[q] = acc;
    }
    gh[0] = g_sig[i] * s->sigma;
    for (int q = 0; q < 15; ++q) gh[1 + q] = gxc[q];
    for (int j = 0; j < HID; ++j) {
      double acc = 0.0;
      for (int o2 = 0; o2 < DOUT; ++o2) acc += f->wd2[j * DOUT + o2] * gh[o2];
      ga[j] = ((s->a_pre[j] > 0.0) != s->flip[0][j]) ? acc : 0.0;
    }
    for (int q = 0; q < din; ++q) {
      double acc = 0.0;
      for (int j = 0; j < HID; ++j) acc += f->wd1[q * HID + j] * ga[j];
      gf[q] = acc;
    }
    double gp[3];
    for (int a = 0; a < 3; ++a) {
      double gx = 0.0;
      for (int q = 0; q < din; ++q) gx += gf[q] * s->jac[a * din + q];
      double ext = (double)f->aabb_max[a] - (double)f->aabb_min[a];
      gp[a] = gx / ext;
    }
    if (s_out) {
      double* so = s_out + ORC_SAMPLE_COLS * (size_t)i;
      so[4] = gh[0];
      for (int c = 0; c < 3; ++c) {
        so[5 + c] = gz[c];
        so[8 + c] = gp[c];
      }
      /* this sample's share of the torque: t (d x gp) (+ d x gd_i on the SH path) */
      double m[3] = {t * gp[0], t * gp[1], t * gp[2]}, gdi[3] = {0, 0, 0};
      if (f->sh_dir_grad && !sh_dir)
        for (int q = 0; q < 16; ++q)
          for (int a = 0; a < 3; ++a) gdi[a] += gxc[15 + q] * shg[q][a];
      so[13] = d[1] * (m[2] + gdi[2]) - d[2] * (m[1] + gdi[1]);
      so[14] = d[2] * (m[0] + gdi[0]) - d[0] * (m[2] + gdi[2]);
      so[15] = d[0] * (m[1] + gdi[1]) - d[1] * (m[0] + gdi[0]);
    }
    for (int a = 0; a < 3; ++a) {
      G[a] += gp[a];
      M[a] += t * gp[a];
    }
    if (f->sh_dir_grad && !sh_dir)
      for (int q = 0; q < 16; ++q)
        for (int a = 0; a < 3; ++a) gd[a] += gxc[15 + q] * shg[q][a];
  }
  double tau[3] = {d[1] * M[2] - d[2] * M[1], d[2] * M[0] - d[0] * M[2],
                   d[0] * M[1] - d[1] * M[0]};
  if (f->sh_dir_grad && !sh_dir) {
    tau[0] += d[1] * gd[2] - d[2] * gd[1];
    tau[1] += d[2] * gd[0] - d[0] * gd[2];
    tau[2] += d[0] * gd[1] - d[1] * gd[0];
  }
  for (int a = 0; a < 3; ++a) {
    g_out[a] = tau[a];
    g_out[3 + a] = G[a];
  }
  *sig = h;
  free(st); free(sig_s); free(rgb_s); free(trans); free(weight); free(g_sig); free(g_rgb);
}

int32_t orc_shade(const orc_field* f, int32_t K, const double* poses, int32_t P,
                  const int32_t* pix, const float* obs, const orc_intr* in,
                  const int64_t* ray_offset, const float* t, const float* delta,
                  const double* sh_dirs, double* loss, double* dpose, double* rgb,
                  int32_t* ray_stop, uint64_t* signature, double* sample_out,
                  int32_t n_threads) {
  if (f->F != 2 || f->din != f->L * f->F || f->din > CIN || f->loss_type < 0 || f->loss_type > 7)
    return 1;
  int64_t n_rays = (int64_t)K * P;
  double* rl = (double*)malloc(sizeof(double) * (size_t)(n_rays + 1));
  double* rg = (double*)malloc(sizeof(double) * 6 * (size_t)(n_rays + 1));
  uint64_t* rs = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)(n_rays + 1));
  if (n_threads < 1) n_threads = 1;
#pragma omp parallel for schedule(dynamic, 16) num_threads(n_threads)
  for (int64_t r = 0; r < n_rays; ++r) {
    int64_t k = r / P;
    double c[3];
    int32_t used;
    shade_ray(f, poses + 12 * k, in, pix[r], obs, t + ray_offset[r],
              (int32_t)(ray_offset[r + 1] - ray_offset[r]), delta[r],
              sh_dirs ? sh_dirs + 3 * r : NULL, P, NULL, rl + r, rg + 6 * r, c, &used, rs + r,
              sample_out ? sample_out + ORC_SAMPLE_COLS * (size_t)ray_offset[r] : NULL, NULL);
    if (rgb)
      for (int q = 0; q < 3; ++q) rgb[3 * r + q] = c[q];
    if (ray_stop) ray_stop[r] = used;
  }
  /* "averaged over all pixels": the 1/(3P) already sits in dL/dC, so the
   * per-hypothesis result is the plain sum over its rays, in ray order */
  uint64_t h = 1469598103934665603ull;
  for (int32_t k = 0; k < K; ++k) {
    double L = 0.0, g[6] = {0, 0, 0, 0, 0, 0};
    for (int32_t s = 0; s < P; ++s) {
      int64_t r = (int64_t)k * P + s;
      L += rl[r];
      for (int q = 0; q < 6; ++q) g[q] += rg[6 * r + q];
      h = fnv(h, (int64_t)rs[r]);
    }
    if (loss) loss[k] = L;
    if (dpose)
      for (int q = 0; q < 6; ++q) dpose[6 * k + q] = g[q];
  }
  if (signature) *signature = h;
  free(rl); free(rg); free(rs);
  return 0;
}

int32_t orc_shade_ray_variant(const orc_field* f, const double pose[12], int32_t P,
                              int32_t pix, const float* obs, const orc_intr* in, const float* t,
                              int32_t n, float delta, const orc_variant* var, double* sample_out,
                              int32_t* near_out, double* loss, double g[6], double rgb[3],
                              int32_t* stop) {
  if (f->F != 2 || f->din != f->L * f->F || f->din > CIN || f->loss_type < 0 || f->loss_type > 7 ||
      n < 0 || P < 1 || !var)
    return 1;
  double c[3], gg[6], L;
  int32_t used;
  uint64_t h;
  shade_ray(f, pose, in, pix, obs, t, n, delta, NULL, P, var, &L, gg, c, &used, &h, sample_out,
            near_out);
  if (loss) *loss = L;
  if (g)
    for (int q = 0; q < 6; ++q) g[q] = gg[q];
  if (rgb)
    for (int q = 0; q < 3; ++q) rgb[q] = c[q];
  if (stop) *stop = used;
  return 0;
}

int32_t orc_shade_ray_jobs(const orc_field* f, const double* poses, int32_t P, const float* obs,
                           const orc_intr* in, const float* t, double relu_margin, int32_t n_jobs,
                           const orc_ray_job* jobs, const int64_t* out_row, double* sample_out,
                           int32_t* near_out, double* loss, double* g, int32_t n_threads) {
  if (f->F != 2 || f->din != f->L * f->F || f->din > CIN || f->loss_type < 0 || f->loss_type > 7 ||
      P < 1 || n_jobs < 0)
    return 1;
  if (n_threads < 1) n_threads = 1;
#pragma omp parallel for schedule(dynamic, 4) num_threads(n_threads)
  for (int32_t q = 0; q < n_jobs; ++q) {
    const orc_ray_job* jb = jobs + q;
    orc_variant var;
    var.relu_margin = relu_margin;
    var.relu_pattern = NULL;
    var.relu_pattern_all = jb->relu_pattern;
    var.stop = jb->stop;
    for (int c = 0; c < 3; ++c) var.loss_sign[c] = jb->loss_sign[c];
    double c3[3], gg[6], L;
    int32_t used;
    uint64_t h;
    shade_ray(f, poses + 12 * (size_t)jb->hyp, in, jb->pix, obs, t + jb->t0, jb->n, jb->delta, NULL,
              P, &var, &L, gg, c3, &used, &h,
              sample_out ? sample_out + ORC_SAMPLE_COLS * (size_t)out_row[q] : NULL,
              near_out ? near_out + out_row[q] : NULL);
    if (loss) loss[q] = L;
    if (g)
      for (int k = 0; k < 6; ++k) g[6 * (size_t)q + k] = gg[k];
  }
  return 0;
}

/* ------------------------------------------------------------- pose update */
/* Exponential map of so(3) (Rodrigues); second-order series for tiny angles. */
void orc_exp_so3(const double w[3], double R[9]) {
  double th = sqrt(w[0] * w[0] + w[1] * w[1] + w[2] * w[2]);
  double Wx[9] = {0, -w[2], w[1], w[2], 0, -w[0], -w[1], w[0], 0};
  double W2[9];
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j) {
      double s = 0.0;
      for (int k = 0; k < 3; ++k) s += Wx[3 * i + k] * Wx[3 * k + j];
      W2[3 * i + j] = s;
    }
  double A, B;
  if (th < 1e-4) {
    A = 1.0;
    B = 0.5;
  } else {
    A = sin(th) / th;
    B = (1.0 - cos(th)) / (th * th);
  }
  for (int i = 0; i < 9; ++i) R[i] = (i % 4 == 0 ? 1.0 : 0.0) + A * Wx[i] + B * W2[i];
}

/* Left-multiply the rotation by Exp(w) (about the camera centre, world axes)
 * and add v to the centre: the SO(3) x T(3) update of Sec. IV-A. */
static void apply_update(float* pose, const double w[3], const double v[3]) {
  double Rinc[9], R[9], Rn[9];
  orc_exp_so3(w, Rinc);
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j) R[3 * i + j] = (double)pose[4 * i + j];
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j) {
      double s = 0.0;
      for (int k = 0; k < 3; ++k) s += Rinc[3 * i + k] * R[3 * k + j];
      Rn[3 * i + j] = s;
    }
  for (int i = 0; i < 3; ++i) {
    for (int j = 0; j < 3; ++j) pose[4 * i + j] = (float)Rn[3 * i + j];
    pose[4 * i + 3] = (float)((double)pose[4 * i + 3] + v[i]);
  }
}

/* Momentum kept as vectors on both subspaces (Sec. IV-A, "Momentum-Based
 * Optimization"): heavy ball m <- beta m + g, step -lr m. */
void orc_step_momentum(int32_t K, float* poses, float* momentum, const float* dpose,
                       float lr, float beta) {
  for (int32_t k = 0; k < K; ++k) {
    double m[6], w[3], v[3];
    for (int q = 0; q < 6; ++q) {
      m[q] = (double)beta * (double)momentum[6 * k + q] + (double)dpose[6 * k + q];
      momentum[6 * k + q] = (float)m[q];
    }
    for (int a = 0; a < 3; ++a) {
      w[a] = -(double)lr * m[a];
      v[a] = -(double)lr * m[3 + a];
    }
    apply_update(poses + 12 * k, w, v);
  }
}

/* Learning rate at global step `step` under the exponential decay of Sec. IV-D
 * (base `decay_base` per `decay_steps` steps; continuous or stepwise). */
static double decayed_lr(double lr0, const orc_adam* a, int32_t step) {
  if (a->decay_steps <= 0) return lr0;
  double e = (double)step / (double)a->decay_steps;
  if (a->staircase) e = floor(e);
  return lr0 * pow((double)a->decay_base, e);
}

/* SE(3) exponential of the twist (w, v) (Lynch and Park, Modern Robotics,
 * Prop. 3.25): rotation Exp(w), translation V(w) v with
 * V = I + (1 - cos th)/th^2 [w]x + (th - sin th)/th^3 [w]x^2 (series for tiny th). */
static void exp_se3(const double w[3], const double v[3], double R[9], double t[3]) {
  orc_exp_so3(w, R);
  double th2 = w[0] * w[0] + w[1] * w[1] + w[2] * w[2], th = sqrt(th2);
  double B, C;
  if (th < 1e-4) {
    B = 0.5 - th2 / 24.0;
    C = 1.0 / 6.0 - th2 / 120.0;
  } else {
    B = (1.0 - cos(th)) / th2;
    C = (th - sin(th)) / (th2 * th);
  }
  double Wx[9] = {0, -w[2], w[1], w[2], 0, -w[0], -w[1], w[0], 0};
  double Wv[3], W2v[3];
  for (int i = 0; i < 3; ++i) Wv[i] = Wx[3 * i] * v[0] + Wx[3 * i + 1] * v[1] + Wx[3 * i + 2] * v[2];
  for (int i = 0; i < 3; ++i)
    W2v[i] = Wx[3 * i] * Wv[0] + Wx[3 * i + 1] * Wv[1] + Wx[3 * i + 2] * Wv[2];
  for (int i = 0; i < 3; ++i) t[i] = v[i] + B * Wv[i] + C * W2v[i];
}

/* T <- Exp(w, v) T for the twist (w, v) about the world origin: R <- E R,
 * o <- E o + V v. */
static void apply_twist(float* pose, const double w[3], const double v[3]) {
  double E[9], tv[3], R[9], o[3];
  exp_se3(w, v, E, tv);
  for (int i = 0; i < 3; ++i) {
    for (int j = 0; j < 3; ++j) R[3 * i + j] = (double)pose[4 * i + j];
    o[i] = (double)pose[4 * i + 3];
  }
  for (int i = 0; i < 3; ++i) {
    for (int j = 0; j < 3; ++j)
      pose[4 * i + j] = (float)(E[3 * i] * R[j] + E[3 * i + 1] * R[3 + j] + E[3 * i + 2] * R[6 + j]);
    pose[4 * i + 3] = (float)(E[3 * i] * o[0] + E[3 * i + 1] * o[1] + E[3 * i + 2] * o[2] + tv[i]);
  }
}

/* Adam (Kingma and Ba, ICLR 2015, Algorithm 1) applied independently on the two
 * subspaces SO(3) and T(3) (Sec. IV-A, "Momentum-Based Optimization"): the
 * first moments are vectors (the rotational one built from the torque), and the
 * bias-corrected step is applied as a rotation Exp(u_w) of the orientation and
 * a shift u_t of the camera centre.  The second moment is kept per component,
 * or (second_moment = 1) as one squared norm per subspace.  State row per
 * hypothesis: m[6], v[6], its own step count t, three zeros.
 * representation = 1 runs the same optimiser on the coupled se(3) twist that
 * Sec. IV-A compares against (exponential coordinates about the world origin,
 * as in iNeRF): the gradient w.r.t. the twist is (tau + o x g, g) for
 * dpose = (tau, g) and camera centre o, and the step is T <- Exp(u) T. */
void orc_step_adam(int32_t K, float* poses, float* state, const float* dpose, int32_t step,
                   const orc_adam* a) {
  const double b1 = (double)a->beta1, b2 = (double)a->beta2, eps = (double)a->eps;
  const double alpha[2] = {decayed_lr((double)a->lr_rot, a, step),
                           decayed_lr((double)a->lr_trans, a, step)};
  for (int32_t k = 0; k < K; ++k) {
    float* st = state + 16 * k;
    double G[6];
    for (int q = 0; q < 6; ++q) G[q] = (double)dpose[6 * k + q];
    if (a->representation == 1) {
      const double o[3] = {poses[12 * k + 3], poses[12 * k + 7], poses[12 * k + 11]};
      G[0] += o[1] * G[5] - o[2] * G[4];
      G[1] += o[2] * G[3] - o[0] * G[5];
      G[2] += o[0] * G[4] - o[1] * G[3];
    }
    double t = (double)st[12] + 1.0; /* t <- t + 1 */
    double u[6];
    for (int sub = 0; sub < 2; ++sub) {
      const double* g = G + 3 * sub;
      double m[3], v[3], sq = 0.0;
      for (int i = 0; i < 3; ++i) sq += g[i] * g[i];
      for (int i = 0; i < 3; ++i) {
        m[i] = b1 * (double)st[3 * sub + i] + (1.0 - b1) * g[i];
        if (a->second_moment)
          v[i] = b2 * (double)st[6 + 3 * sub] + (1.0 - b2) * sq;
        else
          v[i] = b2 * (double)st[6 + 3 * sub + i] + (1.0 - b2) * g[i] * g[i];
      }
      for (int i = 0; i < 3; ++i) {
        double m_hat = m[i] / (1.0 - pow(b1, t));
        double v_hat = v[i] / (1.0 - pow(b2, t));
        u[3 * sub + i] = -alpha[sub] * m_hat / (sqrt(v_hat) + eps);
        st[3 * sub + i] = (float)m[i];
        st[6 + 3 * sub + i] = (float)v[i];
      }
    }
    st[12] = (float)t;
    if (a->representation == 1)
      apply_twist(poses + 12 * k, u, u + 3);
    else
      apply_update(poses + 12 * k, u, u + 3);
  }
}

/* ------------------------------------------------------------- resampling */
/* SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): state += golden gamma, then
 * the output mix. */
static uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

uint64_t orc_splitmix64_next(uint64_t* state) {
  *state += 0x9E3779B97F4A7C15ull;
  return mix64(*state);
}

/* Six standard normals for (seed, round, slot): SplitMix64 stream started at
 * seed ^ mix64(round << 32 | slot), uniforms ((u >> 11) + 1/2) 2^-53, then
 * Box-Muller on consecutive pairs. */
void orc_normals6(uint64_t seed, uint32_t round_idx, uint32_t slot, double n[6]) {
  uint64_t state = seed ^ mix64(((uint64_t)round_idx << 32) | slot);
  double u[6];
  for (int q = 0; q < 6; ++q)
    u[q] = ((double)(orc_splitmix64_next(&state) >> 11) + 0.5) * (1.0 / 9007199254740992.0);
  const double two_pi = 6.28318530717958647692;
  for (int q = 0; q < 3; ++q) {
    double r = sqrt(-2.0 * log(u[2 * q]));
    n[2 * q] = r * cos(two_pi * u[2 * q + 1]);
    n[2 * q + 1] = r * sin(two_pi * u[2 * q + 1]);
  }
}

static int loss_before(float a, int32_t ia, float b, int32_t ib) {
  int na = isnan(a), nb = isnan(b);
  if (na != nb) return nb; /* NaN ranks last */
  if (!na && a != b) return a < b;
  return ia < ib;
}

/* Parallel Monte Carlo resampling (Sec. IV-B): rank hypotheses by loss, keep
 * the lowest-loss fraction, redraw every other one around a kept hypothesis
 * with a small random rotation and translation; a redrawn slot's optimiser
 * state (state_dim floats) restarts at 0.
 * The i-th redrawn slot (ascending index) takes the kept hypothesis of rank
 * i mod n_keep as its parent. */
void orc_resample(int32_t K, float* poses, float* state, int32_t state_dim, const float* loss,
                  float keep_frac, float sigma_rot, float sigma_trans, uint64_t seed,
                  uint32_t round_idx, int32_t* rank_out) {
  int32_t n_keep = (int32_t)floor((double)K * (double)keep_frac);
  if (n_keep < 1) n_keep = 1;
  if (n_keep > K) n_keep = K;
  int32_t* rank = (int32_t*)malloc(sizeof(int32_t) * (size_t)K);
  int32_t* by_rank = (int32_t*)malloc(sizeof(int32_t) * (size_t)K);
  for (int32_t i = 0; i < K; ++i) {
    int32_t r = 0;
    for (int32_t j = 0; j < K; ++j)
      if (j != i && loss_before(loss[j], j, loss[i], i)) ++r;
    rank[i] = r;
    by_rank[r] = i;
  }
  int32_t n_redrawn = 0;
  for (int32_t i = 0; i < K; ++i) {
    if (rank_out) rank_out[i] = rank[i];
    if (rank[i] < n_keep) continue;
    int32_t parent = by_rank[n_redrawn % n_keep];
    ++n_redrawn;
    double nz[6], w[3], v[3];
    orc_normals6(seed, round_idx, (uint32_t)i, nz);
    for (int a = 0; a < 3; ++a) {
      w[a] = (double)sigma_rot * nz[a];
      v[a] = (double)sigma_trans * nz[3 + a];
    }
    memcpy(poses + 12 * i, poses + 12 * parent, 12 * sizeof(float));
    apply_update(poses + 12 * i, w, v);
    for (int32_t q = 0; q < state_dim; ++q) state[(size_t)state_dim * i + q] = 0.0f;
  }
  free(rank);
  free(by_rank);
}

/* ---------------------------------------------------------------- occupancy */
void orc_build_occupancy(const orc_field* f, int32_t R, float threshold, uint32_t* bits,
                         int32_t n_threads) {
  size_t n = (size_t)R * R * R;
  memset(bits, 0, ((n + 31) / 32) * sizeof(uint32_t));
  if (n_threads < 1) n_threads = 1;
#pragma omp parallel for schedule(static) num_threads(n_threads)
  for (int32_t z = 0; z < R; ++z) {
    double feat[CIN], a[HID], h[DOUT];
    for (int32_t y = 0; y < R; ++y)
      for (int32_t x = 0; x < R; ++x) {
        int32_t c[3] = {x, y, z}, cl[3] = {0, 0, 0};
        float x32[3];
        double x64[3];
        for (int q = 0; q < 3; ++q) {
          float ext32 = f->aabb_max[q] - f->aabb_min[q];
          float cell = ext32 / (float)R;
          float p = f->aabb_min[q] + ((float)c[q] + 0.5f) * cell;
          float xr = (p - f->aabb_min[q]) * (1.0f / ext32);
          x32[q] = xr < 0.0f ? 0.0f : (xr > 1.0f ? 1.0f : xr);
          x64[q] = ((double)c[q] + 0.5) / (double)R;
        }
        orc_encode(f, x32, x64, cl, feat, NULL);
        density_fwd(f, feat, a, h);
        if (exp(h[0] + f->density_bias) > (double)threshold) {
          size_t idx = (size_t)x + (size_t)R * ((size_t)y + (size_t)R * z);
          /* each z-slab owns whole words only when R*R is a multiple of 32 */
#pragma omp atomic
          bits[idx >> 5] |= 1u << (idx & 31u);
        }
      }
  }
}
