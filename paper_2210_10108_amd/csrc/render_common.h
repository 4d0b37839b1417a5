// Device helpers shared by the compositing kernels: the pixel-based RGB
// losses and one 64-sample step of a ray's front-to-back compositing
// (classic volume rendering: transmittance from a wavefront prefix sum of
// sigma * delta carried across steps).
#pragma once
#include "pnerf_internal.h"

namespace pnerf {
namespace {

// Sum over the wavefront, in every lane.
__device__ __forceinline__ float wave_sum(float x) { return lane_value(wave_incl_scan(x), 63); }

// Pixel-based RGB loss of one channel (Sec. IV-C): r = C - y; returns the
// loss and writes d loss / d C.  p: threshold of Huber (0) and Smooth L1 (7),
// epsilon of Relative L2 (4), MAPE (5) and sMAPE (6).
//   0 Huber 0.5 r^2 (|r| <= p) or p (|r| - p/2)   1 L1 |r|        2 L2 r^2
//   3 Log L1 log(1 + |r|)   4 Relative L2 r^2 / (y^2 + p)   5 MAPE |r| / (|y| + p)
//   6 sMAPE 2|r| / (|C| + |y| + p)   7 Smooth L1 0.5 r^2 / p (|r| < p) or |r| - p/2
__device__ __forceinline__ float pixel_loss(int type, float C, float y, float p, float& grad) {
  const float r = C - y, ar = fabsf(r), sr = r > 0.0f ? 1.0f : (r < 0.0f ? -1.0f : 0.0f);
  switch (type) {
    case 0:
      if (ar <= p) {
        grad = r;
        return 0.5f * r * r;
      }
      grad = p * sr;
      return p * (ar - 0.5f * p);
    case 1:
      grad = sr;
      return ar;
    case 2:
      grad = 2.0f * r;
      return r * r;
    case 3:
      grad = sr / (1.0f + ar);
      return log1pf(ar);
    case 4: {
      const float den = y * y + p;
      grad = 2.0f * r / den;
      return r * r / den;
    }
    case 5: {
      const float den = fabsf(y) + p;
      grad = sr / den;
      return ar / den;
    }
    case 6: {
      const float den = fabsf(C) + fabsf(y) + p;
      const float sc = C > 0.0f ? 1.0f : (C < 0.0f ? -1.0f : 0.0f);
      grad = 2.0f * sr / den - 2.0f * ar * sc / (den * den);
      return 2.0f * ar / den;
    }
    default:
      if (ar < p) {
        grad = r / p;
        return 0.5f * r * r / p;
      }
      grad = sr;
      return ar - 0.5f * p;
  }
}

struct Chunk {
  bool live;        // sample exists and is composited
  float sig, tau, T_in, T_out, w, c[3];
  bool stop_here;
};

// One lane's sample of a 64-sample step: density and colour (zero past the
// ray's end).
struct Raw {
  float sig, c[3];
};

__device__ __forceinline__ Raw load_raw(const DevWork& w, int base, int n, int i0, int lane) {
  Raw r;
  const int i = i0 + lane;
  const bool valid = i < n;
  r.sig = valid ? w.sig[base + i] : 0.0f;
  r.c[0] = valid ? w.cr[base + i] : 0.0f;
  r.c[1] = valid ? w.cg[base + i] : 0.0f;
  r.c[2] = valid ? w.cb[base + i] : 0.0f;
  return r;
}

// Evaluate one 64-sample step of a ray: transmittance in and out, weight.
__device__ inline Chunk make_chunk(const DevField& f, const Raw& r, bool valid, float delta,
                                   float carry, float& incl_out) {
  Chunk ch;
  ch.sig = r.sig;
#pragma unroll
  for (int q = 0; q < 3; ++q) ch.c[q] = r.c[q];
  ch.tau = ch.sig * delta;
  float incl = wave_incl_scan(ch.tau) + carry;
  incl_out = incl;
  ch.T_in = __expf(-(incl - ch.tau));
  ch.T_out = __expf(-incl);
  float alpha = -expm1f(-ch.tau);
  ch.w = valid ? ch.T_in * alpha : 0.0f;
  ch.live = valid;
  ch.stop_here = valid && f.t_stop > 0.0f && ch.T_out < f.t_stop;
  return ch;
}

__device__ inline Chunk step_chunk(const DevField& f, const DevWork& w, int base, int n, int i0,
                                   float delta, float carry, int lane, float& incl_out) {
  return make_chunk(f, load_raw(w, base, n, i0, lane), i0 + lane < n, delta, carry, incl_out);
}

}  // namespace
}  // namespace pnerf
