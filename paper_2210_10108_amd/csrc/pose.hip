// Pose updates on SO(3) x T(3) (heavy-ball momentum; Adam with separate moments
// per subspace) and Monte Carlo hypothesis resampling.  All are tiny (one
// thread per hypothesis) and run in double precision; results are stored as
// float.
#include <mutex>

#include "pnerf_internal.h"

namespace pnerf {
namespace {

// Rodrigues: Exp(w) = I + A [w]x + B [w]x^2, series for small angles.
__device__ inline void exp_so3(const double w[3], double R[9]) {
  double th = sqrt(w[0] * w[0] + w[1] * w[1] + w[2] * w[2]);
  double A, B;
  if (th < 1e-4) {
    A = 1.0;
    B = 0.5;
  } else {
    A = sin(th) / th;
    B = (1.0 - cos(th)) / (th * th);
  }
  double W[9] = {0.0, -w[2], w[1], w[2], 0.0, -w[0], -w[1], w[0], 0.0};
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j) {
      double w2 = W[3 * i] * W[j] + W[3 * i + 1] * W[3 + j] + W[3 * i + 2] * W[6 + j];
      R[3 * i + j] = (i == j ? 1.0 : 0.0) + A * W[3 * i + j] + B * w2;
    }
}

// R <- Exp(w) R about the camera centre (world axes), o <- o + v.
__device__ inline void apply(float* pose, const double w[3], const double v[3]) {
  double E[9], R[9];
  exp_so3(w, E);
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j) R[3 * i + j] = (double)pose[4 * i + j];
  for (int i = 0; i < 3; ++i) {
    for (int j = 0; j < 3; ++j)
      pose[4 * i + j] =
          (float)(E[3 * i] * R[j] + E[3 * i + 1] * R[3 + j] + E[3 * i + 2] * R[6 + j]);
    pose[4 * i + 3] = (float)((double)pose[4 * i + 3] + v[i]);
  }
}

// SE(3) exponential applied on the left, about the world origin: R <- E R,
// o <- E o + V(w) v with E = Exp(w), V(w) = I + B [w]x + C [w]x^2,
// B = (1 - cos th)/th^2, C = (th - sin th)/th^3 (series for small th).
__device__ inline void apply_twist(float* pose, const double w[3], const double v[3]) {
  double E[9];
  exp_so3(w, E);
  const double th2 = w[0] * w[0] + w[1] * w[1] + w[2] * w[2], th = sqrt(th2);
  double B, C;
  if (th < 1e-4) {
    B = 0.5 - th2 / 24.0;
    C = 1.0 / 6.0 - th2 / 120.0;
  } else {
    B = (1.0 - cos(th)) / th2;
    C = (th - sin(th)) / (th2 * th);
  }
  const double wv[3] = {w[1] * v[2] - w[2] * v[1], w[2] * v[0] - w[0] * v[2],
                        w[0] * v[1] - w[1] * v[0]};
  const double wwv[3] = {w[1] * wv[2] - w[2] * wv[1], w[2] * wv[0] - w[0] * wv[2],
                         w[0] * wv[1] - w[1] * wv[0]};
  double R[9], o[3];
  for (int i = 0; i < 3; ++i) {
    for (int j = 0; j < 3; ++j) R[3 * i + j] = (double)pose[4 * i + j];
    o[i] = (double)pose[4 * i + 3];
  }
  for (int i = 0; i < 3; ++i) {
    for (int j = 0; j < 3; ++j)
      pose[4 * i + j] =
          (float)(E[3 * i] * R[j] + E[3 * i + 1] * R[3 + j] + E[3 * i + 2] * R[6 + j]);
    pose[4 * i + 3] = (float)(E[3 * i] * o[0] + E[3 * i + 1] * o[1] + E[3 * i + 2] * o[2] +
                              v[i] + B * wv[i] + C * wwv[i]);
  }
}

__global__ void k_step_momentum(int K, float* poses, float* mom, const float* dpose, float lr,
                                float beta) {
  int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= K) return;
  double m[6], w[3], v[3];
  for (int q = 0; q < 6; ++q) {
    m[q] = __dadd_rn(__dmul_rn((double)beta, (double)mom[6 * k + q]), (double)dpose[6 * k + q]);
    mom[6 * k + q] = (float)m[q];
  }
  for (int a = 0; a < 3; ++a) {
    w[a] = -(double)lr * m[a];
    v[a] = -(double)lr * m[3 + a];
  }
  float pose[12];
  for (int q = 0; q < 12; ++q) pose[q] = poses[12 * k + q];
  apply(pose, w, v);
  for (int q = 0; q < 12; ++q) poses[12 * k + q] = pose[q];
}

// Adam (Kingma and Ba, Algorithm 1) run separately on the rotation and the
// translation subspace.  State row: m[6], v[6], step count, 3 zero pads.
// twist: the coupled se(3) representation -- gradient (tau + o x f, f) for
// dpose = (tau, f), step T <- Exp(u) T.
__global__ void k_step_adam(int K, float* poses, float* state, const float* dpose, double lr_r,
                            double lr_t, double b1, double b2, double eps, int per_subspace,
                            int twist) {
  int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= K) return;
  float* st = state + (size_t)kAdamState * k;
  double G[6];
  for (int q = 0; q < 6; ++q) G[q] = (double)dpose[6 * k + q];
  if (twist) {
    const double o[3] = {poses[12 * k + 3], poses[12 * k + 7], poses[12 * k + 11]};
    const double tf[3] = {o[1] * G[5] - o[2] * G[4], o[2] * G[3] - o[0] * G[5],
                          o[0] * G[4] - o[1] * G[3]};
    for (int a = 0; a < 3; ++a) G[a] += tf[a];
  }
  double n = (double)st[12] + 1.0;
  double c1 = 1.0 - pow(b1, n), c2 = 1.0 - pow(b2, n);
  double u[6];
  for (int sub = 0; sub < 2; ++sub) {
    double g[3], m[3], v[3];
    for (int a = 0; a < 3; ++a) g[a] = G[3 * sub + a];
    for (int a = 0; a < 3; ++a) m[a] = b1 * (double)st[3 * sub + a] + (1.0 - b1) * g[a];
    if (per_subspace) {
      double gg = g[0] * g[0] + g[1] * g[1] + g[2] * g[2];
      double vs = b2 * (double)st[6 + 3 * sub] + (1.0 - b2) * gg;
      v[0] = v[1] = v[2] = vs;
    } else {
      for (int a = 0; a < 3; ++a) v[a] = b2 * (double)st[6 + 3 * sub + a] + (1.0 - b2) * g[a] * g[a];
    }
    double lr = sub == 0 ? lr_r : lr_t;
    for (int a = 0; a < 3; ++a) {
      u[3 * sub + a] = -lr * (m[a] / c1) / (sqrt(v[a] / c2) + eps);
      st[3 * sub + a] = (float)m[a];
      st[6 + 3 * sub + a] = (float)v[a];
    }
  }
  st[12] = (float)n;
  float pose[12];
  for (int q = 0; q < 12; ++q) pose[q] = poses[12 * k + q];
  if (twist)
    apply_twist(pose, u, u + 3);
  else
    apply(pose, u, u + 3);
  for (int q = 0; q < 12; ++q) poses[12 * k + q] = pose[q];
}

// ---------------------------------------------------------------- resample
// SplitMix64 output function and stream step (Steele, Lea, Flood 2014).
__device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ inline bool before(float a, int ia, float b, int ib) {
  bool na = isnan(a), nb = isnan(b);
  if (na != nb) return nb;
  if (!na && a != b) return a < b;
  return ia < ib;
}

constexpr int kRankBlock = 256;

// rank[i] = number of hypotheses ordered before i; by_rank[rank] = i.
__global__ __launch_bounds__(kRankBlock) void k_rank(int K, const float* loss, int32_t* rank,
                                                     int32_t* by_rank) {
  __shared__ float s_loss[kRankBlock];
  int i = blockIdx.x * kRankBlock + threadIdx.x;
  float li = i < K ? loss[i] : 0.0f;
  int r = 0;
  for (int j0 = 0; j0 < K; j0 += kRankBlock) {
    int j = j0 + threadIdx.x;
    s_loss[threadIdx.x] = j < K ? loss[j] : 0.0f;
    __syncthreads();
    int jn = K - j0 < kRankBlock ? K - j0 : kRankBlock;
    for (int q = 0; q < jn; ++q)
      if (j0 + q != i && before(s_loss[q], j0 + q, li, i)) ++r;
    __syncthreads();
  }
  if (i < K) {
    rank[i] = r;
    by_rank[r] = i;
  }
}

// Each discarded slot counts the discarded slots before it, picks its parent
// by rank, and redraws itself around the parent.
__global__ __launch_bounds__(kRankBlock) void k_redraw(int K, float* poses, float* opt,
                                                       int state_dim, const int32_t* rank,
                                                       const int32_t* by_rank, int n_keep,
                                                       float sr, float st, uint64_t seed,
                                                       uint32_t round) {
  __shared__ int32_t s_rank[kRankBlock];
  int i = blockIdx.x * kRankBlock + threadIdx.x;
  int ri = i < K ? rank[i] : 0;
  int before_i = 0;  // discarded slots with index < i
  for (int j0 = 0; j0 < K; j0 += kRankBlock) {
    int j = j0 + threadIdx.x;
    s_rank[threadIdx.x] = j < K ? rank[j] : 0;
    __syncthreads();
    int jn = K - j0 < kRankBlock ? K - j0 : kRankBlock;
    for (int q = 0; q < jn; ++q)
      if (j0 + q < i && s_rank[q] >= n_keep) ++before_i;
    __syncthreads();
  }
  if (i >= K || ri < n_keep) return;
  int parent = by_rank[before_i % n_keep];
  uint64_t state = seed ^ mix64(((uint64_t)round << 32) | (uint32_t)i);
  double u[6];
  for (int q = 0; q < 6; ++q) {
    state += 0x9E3779B97F4A7C15ull;
    u[q] = ((double)(mix64(state) >> 11) + 0.5) * (1.0 / 9007199254740992.0);
  }
  double nz[6];
  const double two_pi = 6.28318530717958647692;
  for (int q = 0; q < 3; ++q) {
    double r = sqrt(-2.0 * log(u[2 * q]));
    nz[2 * q] = r * cos(two_pi * u[2 * q + 1]);
    nz[2 * q + 1] = r * sin(two_pi * u[2 * q + 1]);
  }
  double w[3] = {sr * nz[0], sr * nz[1], sr * nz[2]};
  double v[3] = {st * nz[3], st * nz[4], st * nz[5]};
  float pose[12];
  for (int q = 0; q < 12; ++q) pose[q] = poses[12 * parent + q];
  apply(pose, w, v);
  for (int q = 0; q < 12; ++q) poses[12 * i + q] = pose[q];
  for (int q = 0; q < state_dim; ++q) opt[(size_t)state_dim * i + q] = 0.0f;
}

}  // namespace

hipError_t launch_step_momentum(int K, float* poses, float* mom, const float* dpose, float lr,
                                float beta, hipStream_t s) {
  hipLaunchKernelGGL(k_step_momentum, dim3((K + 63) / 64), dim3(64), 0, s, K, poses, mom, dpose,
                     lr, beta);
  return hipGetLastError();
}

hipError_t launch_step_adam(int K, float* poses, float* state, const float* dpose, double lr_r,
                            double lr_t, double b1, double b2, double eps, int per_subspace,
                            int twist, hipStream_t s) {
  hipLaunchKernelGGL(k_step_adam, dim3((K + 63) / 64), dim3(64), 0, s, K, poses, state, dpose,
                     lr_r, lr_t, b1, b2, eps, per_subspace, twist);
  return hipGetLastError();
}

// ------------------------------------------------ static resampling scratch
// The ranking scratch of pnerf_resample_hypotheses_noalloc: rank and by_rank
// of up to kMaxResampleK hypotheses, in a file-scope device array (512 KiB per
// GPU, held until the process ends).  Host code never passes the array's name
// to a kernel (on the host it is only a stand-in): it takes the device address
// from hipGetSymbolAddress, once per device, with that device current.
constexpr int kMaxResampleK = 65535;
static __device__ __align__(256) int32_t scratch[2 * kMaxResampleK];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int32_t* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t resample_scratch(int device, int32_t** ptr, int* max_k) {
  *max_k = kMaxResampleK;
  *ptr = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[device] = static_cast<int32_t*>(p);
  }
  *ptr = g_scratch_ptr[device];
  return hipSuccess;
}

hipError_t launch_resample(int K, float* poses, float* state, int state_dim, const float* loss,
                           int n_keep, float sr, float st, uint64_t seed, uint32_t round,
                           int32_t* scratch, hipStream_t s) {
  int nb = (K + kRankBlock - 1) / kRankBlock;
  int32_t* rank = scratch;
  int32_t* by_rank = scratch + K;
  hipLaunchKernelGGL(k_rank, dim3(nb), dim3(kRankBlock), 0, s, K, loss, rank, by_rank);
  hipLaunchKernelGGL(k_redraw, dim3(nb), dim3(kRankBlock), 0, s, K, poses, state, state_dim,
                     rank, by_rank, n_keep, sr, st, seed, round);
  return hipGetLastError();
}

}  // namespace pnerf
