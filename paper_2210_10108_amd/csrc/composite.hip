// Front-to-back compositing of each ray's samples (classic volume rendering),
// the robust photometric loss against the observed pixel, the backward pass of
// the composite, and the deterministic per-hypothesis reduction.
//
// One wavefront per ray; 64 samples per step.  Transmittance comes from a
// wavefront prefix sum of sigma*delta carried across steps; the backward pass
// re-sweeps the ray (keeping the first two steps from the forward sweep) and
// takes the colour still to come behind sample i as C - (prefix of w c up to i).
#include <algorithm>

#include "pnerf_internal.h"
#include "render_common.h"

namespace pnerf {
namespace {

constexpr int kBlock = 256;

template <int WITH_GRAD>
__global__ __launch_bounds__(kBlock) void k_composite(DevField f, DevBatch b, DevWork w,
                                                      float* rgb_out) {
  int lane = threadIdx.x & 63;
  int ray = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  if (ray >= b.n_rays) return;
  const int base = w.off[ray];
  const int n = w.off[ray + 1] - base;
  const float delta = w.rdelta[ray];
  // the observed pixel, loaded before the sweeps so that its two dependent
  // loads overlap them
  float y[3] = {0.f, 0.f, 0.f};
  if (WITH_GRAD) {
    int pix = b.pix[ray];
    const int n_pix = b.W * b.H;
    pix = pix < 0 ? 0 : (pix >= n_pix ? n_pix - 1 : pix);
    const float* I = b.obs + 3 * (size_t)pix;
#pragma unroll
    for (int q = 0; q < 3; ++q) y[q] = I[q];
  }

  // pass 1: colour, transmittance, stop index.  The first two steps' samples
  // are loaded together up front, and both steps are kept for pass 2, which
  // would compute them again from the same carry.
  float C[3] = {0.f, 0.f, 0.f};
  float carry = 0.0f;
  int n_used = n;
  const Raw r0 = load_raw(w, base, n, 0, lane), r1 = load_raw(w, base, n, 64, lane);
  Chunk first{}, second{};  // the ray's first two steps, reused by pass 2
  float first_incl = 0.0f, second_incl = 0.0f;
  for (int i0 = 0; i0 < n_used; i0 += 64) {
    float incl;
    const Raw r = i0 == 0 ? r0 : (i0 == 64 ? r1 : load_raw(w, base, n, i0, lane));
    Chunk ch = make_chunk(f, r, i0 + lane < n, delta, carry, incl);
    if (i0 == 0) {
      first = ch;
      first_incl = incl;
    } else if (i0 == 64) {
      second = ch;
      second_incl = incl;
    }
    uint64_t st = __ballot(ch.stop_here);
    int last = 63;
    if (st) {
      last = __ffsll((unsigned long long)st) - 1;
      n_used = i0 + last + 1;
    }
    bool use = ch.live && lane <= last;
#pragma unroll
    for (int q = 0; q < 3; ++q) C[q] += wave_sum(use ? ch.w * ch.c[q] : 0.0f);
    carry = lane_value(incl, last);
    if (st) break;
  }
  float T_end = __expf(-carry);
  for (int q = 0; q < 3; ++q) C[q] += T_end * f.bg[q];

  if (!WITH_GRAD) {
    if (lane < 3) rgb_out[3 * ray + lane] = C[lane];
    return;
  }

  // loss on the observed pixel: mean over the P pixels and 3 channels
  const float norm = 1.0f / (3.0f * (float)b.P);
  float gC[3], L = 0.0f;
  for (int q = 0; q < 3; ++q) {
    float gq;
    L += pixel_loss(f.loss_type, C[q], y[q], f.loss_param, gq);
    gC[q] = gq * norm;
  }
  if (lane == 0) w.ray_loss[ray] = L * norm;

  // pass 2: d loss / d sigma_i and d loss / d c_i, written over sigma and c as
  // d loss / d h_0 = g_sigma * sigma and d loss / d z = g_c * c (1 - c)
  float carry2 = 0.0f, pre[3] = {0.f, 0.f, 0.f};
  for (int i0 = 0; i0 < n; i0 += 64) {
    int i = i0 + lane;
    if (i0 >= n_used) {
      if (i < n) {
        w.sig[base + i] = 0.0f;
        w.cr[base + i] = 0.0f;
        w.cg[base + i] = 0.0f;
        w.cb[base + i] = 0.0f;
      }
      continue;
    }
    float incl = i0 == 0 ? first_incl : second_incl;
    Chunk ch = i0 == 0    ? first
               : i0 == 64 ? second
                          : step_chunk(f, w, base, n, i0, delta, carry2, lane, incl);
    bool use = ch.live && i < n_used;
    float gs = 0.0f, gz[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      float wc = use ? ch.w * ch.c[q] : 0.0f;
      float p = wave_incl_scan(wc) + pre[q];
      pre[q] = lane_value(p, 63);
      float S = C[q] - p;  // colour behind sample i (incl. background)
      gs += gC[q] * (ch.T_out * ch.c[q] - S);
      gz[q] = ch.w * gC[q] * ch.c[q] * (1.0f - ch.c[q]);
    }
    carry2 = lane_value(incl, 63);
    if (i < n) {
      w.sig[base + i] = use ? delta * gs * ch.sig : 0.0f;
      w.cr[base + i] = use ? gz[0] : 0.0f;
      w.cg[base + i] = use ? gz[1] : 0.0f;
      w.cb[base + i] = use ? gz[2] : 0.0f;
    }
  }
}

// Torque and force terms of one sample (Eq. 3 and Eq. 2 before the sums), as
// the MLP backward kernel left them in rows 0..5 of the feature array.
__device__ __forceinline__ void sample_terms(const DevField& f, const DevWork& w, int s,
                                             float out[6]) {
  (void)f;
#pragma unroll
  for (int q = 0; q < 6; ++q) out[q] = w.feat[(int64_t)q * w.cap + s];
}

// Per-hypothesis reduction in two fixed-order stages.  Block (j, k) sums part
// j of hypothesis k's rays (losses) and samples (torque and force terms): the
// ranges are cut into n_parts equal pieces, each summed by a strided loop, a
// wavefront scan and the four wavefronts' totals in order.  k_reduce_final adds the n_parts partials of each hypothesis in
// order.  Same inputs give the same bits.
__global__ __launch_bounds__(kBlock) void k_reduce_partial(DevField f, DevBatch b, DevWork w,
                                                           int n_parts, float* partial) {
  __shared__ float red[7][kBlock / 64];
  int j = blockIdx.x, k = blockIdx.y, tid = threadIdx.x;
  int r0 = k * b.P, nr = b.P;
  int s0 = w.off[r0], ns = w.off[r0 + nr] - s0;
  int ra = r0 + (int)((int64_t)nr * j / n_parts), rb = r0 + (int)((int64_t)nr * (j + 1) / n_parts);
  int sa = s0 + (int)((int64_t)ns * j / n_parts), sb = s0 + (int)((int64_t)ns * (j + 1) / n_parts);
  float acc[7] = {0, 0, 0, 0, 0, 0, 0};
  for (int r = ra + tid; r < rb; r += kBlock) acc[6] += w.ray_loss[r];
  for (int s = sa + tid; s < sb; s += kBlock) {
    float o[6];
    sample_terms(f, w, s, o);
#pragma unroll
    for (int q = 0; q < 6; ++q) acc[q] += o[q];
  }
  const int lane = tid & 63, wv = tid >> 6;
#pragma unroll
  for (int q = 0; q < 7; ++q) {
    const float v = wave_incl_scan(acc[q]);
    if (lane == 63) red[q][wv] = v;
  }
  __syncthreads();
  if (tid < 7) {
    float v = 0.0f;
    for (int u = 0; u < kBlock / 64; ++u) v += red[tid][u];
    partial[((size_t)k * n_parts + j) * 7 + tid] = v;
  }
}

// The same first stage over the fused backward's per-ray terms: block (j, k)
// sums part j of hypothesis k's rays, 7 values each.
__global__ __launch_bounds__(kBlock) void k_reduce_rays_partial(DevBatch b, DevWork w,
                                                                int n_parts, float* partial) {
  __shared__ float red[7][kBlock / 64];
  int j = blockIdx.x, k = blockIdx.y, tid = threadIdx.x;
  int r0 = k * b.P, nr = b.P;
  int ra = r0 + (int)((int64_t)nr * j / n_parts), rb = r0 + (int)((int64_t)nr * (j + 1) / n_parts);
  float acc[7] = {0, 0, 0, 0, 0, 0, 0};
  for (int r = ra + tid; r < rb; r += kBlock) {
    const float* v = w.ray_terms + (int64_t)7 * r;
#pragma unroll
    for (int q = 0; q < 7; ++q) acc[q] += v[q];
  }
  const int lane = tid & 63, wv = tid >> 6;
#pragma unroll
  for (int q = 0; q < 7; ++q) {
    const float v = wave_incl_scan(acc[q]);
    if (lane == 63) red[q][wv] = v;
  }
  __syncthreads();
  if (tid < 7) {
    float v = 0.0f;
    for (int u = 0; u < kBlock / 64; ++u) v += red[tid][u];
    partial[((size_t)k * n_parts + j) * 7 + tid] = v;
  }
}

// One wavefront per hypothesis: lane j holds partial j (n_parts <= 64), then a
// fixed butterfly adds them.
__global__ __launch_bounds__(64) void k_reduce_final(int K, int n_parts, const float* partial,
                                                     float* loss, float* dpose) {
  int k = blockIdx.x, lane = threadIdx.x;
  const float* p = partial + ((size_t)k * n_parts + lane) * 7;
#pragma unroll
  for (int q = 0; q < 7; ++q) {
    float v = lane < n_parts ? p[q] : 0.0f;
    v = wave_sum(v);
    if (lane == 0) {
      if (q < 6)
        dpose[6 * k + q] = v;
      else
        loss[k] = v;
    }
  }
}

// Copy per-sample intermediates out of the workspace (inspection only).
__global__ void k_inspect(DevField f, DevWork w, int what, float* dst, int64_t n) {
  const int64_t total = *w.total;
  for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < n;
       s += (int64_t)gridDim.x * blockDim.x) {
    if (s >= total) {  // past the last call's samples: nothing there
      const int width = what == 2 ? 3 : (what == 3 ? 6 : 1);
      for (int q = 0; q < width; ++q) dst[width * s + q] = 0.0f;
    } else if (what == 0) {
      dst[s] = w.t[s];
    } else if (what == 1) {
      dst[s] = w.sig[s];
    } else if (what == 2) {
      dst[3 * s] = w.cr[s];
      dst[3 * s + 1] = w.cg[s];
      dst[3 * s + 2] = w.cb[s];
    } else {
      float o[6];
      sample_terms(f, w, (int)s, o);
      for (int q = 0; q < 6; ++q) dst[6 * s + q] = o[q];
    }
  }
}

}  // namespace

hipError_t launch_inspect(const DevField& f, const DevBatch& b, const DevWork& w, int what,
                          float* dst, int64_t n, hipStream_t s) {
  (void)b;
  hipLaunchKernelGGL(k_inspect, dim3(1024), dim3(256), 0, s, f, w, what, dst, n);
  return hipGetLastError();
}

hipError_t launch_composite(const DevField& f, const DevBatch& b, const DevWork& w, int with_grad,
                            float* rgb_out, hipStream_t s) {
  int n_blocks = (b.n_rays + (kBlock / 64) - 1) / (kBlock / 64);
  if (with_grad)
    hipLaunchKernelGGL(k_composite<1>, dim3(n_blocks), dim3(kBlock), 0, s, f, b, w, rgb_out);
  else
    hipLaunchKernelGGL(k_composite<0>, dim3(n_blocks), dim3(kBlock), 0, s, f, b, w, rgb_out);
  return hipGetLastError();
}

// A fixed number of parts per hypothesis, so that a hypothesis's sums do not
// depend on how a batch is cut into chunks.
int reduce_parts(int K) {
  (void)K;
  return kReduceParts;
}

hipError_t launch_reduce(const DevField& f, const DevBatch& b, const DevWork& w, float* loss,
                         float* dpose, hipStream_t s) {
  int n_parts = reduce_parts(b.K);
  hipLaunchKernelGGL(k_reduce_partial, dim3(n_parts, b.K), dim3(kBlock), 0, s, f, b, w, n_parts,
                     w.partial);
  hipLaunchKernelGGL(k_reduce_final, dim3(b.K), dim3(64), 0, s, b.K, n_parts, w.partial, loss,
                     dpose);
  return hipGetLastError();
}

hipError_t launch_reduce_rays(const DevBatch& b, const DevWork& w, float* loss, float* dpose,
                              hipStream_t s) {
  // parts of at least 64 rays each, at most kReduceParts
  const int n_parts = std::max(1, std::min(kReduceParts, b.P / 64));
  hipLaunchKernelGGL(k_reduce_rays_partial, dim3(n_parts, b.K), dim3(kBlock), 0, s, b, w, n_parts,
                     w.partial);
  hipLaunchKernelGGL(k_reduce_final, dim3(b.K), dim3(64), 0, s, b.K, n_parts, w.partial, loss,
                     dpose);
  return hipGetLastError();
}

}  // namespace pnerf
