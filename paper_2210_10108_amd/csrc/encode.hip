// Multiresolution hash encoding of the samples (Sec. III, Instant NGP): the
// gather of every level's 8 vertex features, their trilinear blend, and the
// blend's derivative with respect to the sample position (the table is frozen,
// so the backward pass needs nothing else from it: the MLP backward kernel
// contracts this Jacobian with d loss / d feature, and nothing is re-gathered
// or scattered).
//
// Work split: the levels are partitioned into NG groups of two levels each,
// and block b works on group b % NG.  Workgroups are dispatched round-robin
// over the XCDs, so every XCD (own 4 MB L2) serves the same one or two level
// groups for the whole launch and its L2 holds only those levels' tables.  One
// thread handles one sample of its group; blocks are persistent and stride
// over the compacted sample array.
//
// Features are stored SoA, row p = (l % 4) * 2 LPG + (l / 4) * 2 + q for
// feature q of level l (the order in which the MLP kernels feed them to MFMA),
// row stride = the workspace sample capacity.  The Jacobian d feature /
// d pos of every level (pos = x N_l: bounded by the table's value
// differences, zero along clamped components) is stored SoA in fp16 (rounding
// below 2^-11 of each entry), row ((l % 4) LPG + l / 4) * 6 + 3 q + a, so that
// lane group l % 4 of the MLP backward kernel reads one contiguous block of
// rows; that kernel applies N_l and 1 / extent in fp32.
#include "pnerf_internal.h"

namespace pnerf {
namespace {

constexpr int kBlock = 256;
constexpr uint32_t kPrime1 = 2654435761u, kPrime2 = 805459861u;

struct Pos {
  float x[3];        // normalised, clamped position in [0,1]^3 (decides cells)
  float dx[3];       // exact normalised position minus x (0 where clamped)
  uint32_t clamped;  // bit a set: component a was clamped
};

// Error-free transformation of a float sum: a + b = s + return value.
__device__ __forceinline__ float two_sum_err(float a, float b, float s) {
  float bb = __fsub_rn(s, a);
  return __fadd_rn(__fsub_rn(a, __fsub_rn(s, bb)), __fsub_rn(b, bb));
}

// Sample position p = o + t d and x = (p - min) / extent.  The float chain
// (separately rounded, never fused) decides cells and clamping; the rounding
// errors of each step are recovered exactly (TwoSum / FMA) together with the
// float direction's own error, so that dx carries x's exact value to first
// order and interpolation weights are accurate to float precision.
__device__ inline Pos sample_pos(const DevField& f, const DevBatch& b, const DevWork& w, int s) {
  Pos ps;
  int ray = w.sray[s];
  const float* pose = b.poses + 12 * (ray / b.P);
  const float o[3] = {pose[3], pose[7], pose[11]};
  const float d[3] = {w.rdx[ray], w.rdy[ray], w.rdz[ray]};
  const float de[3] = {w.rex[ray], w.rey[ray], w.rez[ray]};
  const float t = w.t[s];
  ps.clamped = 0;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    float td = __fmul_rn(t, d[a]);
    float e_td = fmaf(t, d[a], -td) + t * de[a];
    float p = __fadd_rn(o[a], td);
    float e_p = two_sum_err(o[a], td, p);
    float q = __fsub_rn(p, f.mn[a]);
    float e_q = two_sum_err(p, -f.mn[a], q);
    float xr = __fmul_rn(q, f.inv_ext[a]);
    float e_x = fmaf(q, f.inv_ext[a], -xr);
    float dx = e_x + (e_td + e_p + e_q) * f.inv_ext[a] - xr * f.inv_ext_err[a];
    if (!(xr >= 0.0f)) {  // below the box (or NaN from a non-finite pose)
      ps.x[a] = 0.0f;
      ps.dx[a] = 0.0f;
      ps.clamped |= 1u << a;
    } else if (xr > 1.0f) {
      ps.x[a] = 1.0f;
      ps.dx[a] = 0.0f;
      ps.clamped |= 1u << a;
    } else {
      ps.x[a] = xr;
      ps.dx[a] = dx;
    }
  }
  return ps;
}

// Cell of one level and the 8 corner table indices (in vertex units).
struct Cell {
  float w[3];
  uint32_t idx[8];
};

// The cell comes from the float product x N (as a reference implementation in
// float decides it); the weights add back that product's rounding error and
// N dx, the part of the position float cannot hold.
__device__ __forceinline__ void make_cell(const DevField& f, int l, const float x[3],
                                          const float dx[3], Cell& c) {
  const int N = f.res[l];
  const uint32_t n1 = f.n1[l];
  const bool dense = f.dense[l] != 0;
  uint32_t i0[3];
  const float Nf = (float)N;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    float pos = __fmul_rn(x[a], Nf);
    int ci = (int)pos;
    ci = ci < N - 1 ? ci : N - 1;
    i0[a] = (uint32_t)ci;
    c.w[a] = (__fsub_rn(pos, (float)ci) + fmaf(x[a], Nf, -pos)) + Nf * dx[a];
  }
  const uint32_t mask = f.T - 1u;
  const uint32_t sy = dense ? n1 : kPrime1;
  const uint32_t sz = dense ? n1 * n1 : kPrime2;
  const uint32_t y0 = i0[1] * sy, y1 = y0 + sy;
  const uint32_t z0 = i0[2] * sz, z1 = z0 + sz;
  const uint32_t base = (uint32_t)l * f.T;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    uint32_t xi = i0[0] + (k & 1);
    uint32_t yi = (k & 2) ? y1 : y0;
    uint32_t zi = (k & 4) ? z1 : z0;
    uint32_t h = dense ? (xi + yi + zi) : ((xi ^ yi ^ zi) & mask);
    c.idx[k] = base + h;
  }
}

template <bool F16>
__device__ __forceinline__ float2 vertex(const DevField& f, uint32_t idx) {
  if (F16) {
    __half2 v = reinterpret_cast<const __half2*>(f.table16)[idx];
    return __half22float2(v);
  }
  return reinterpret_cast<const float2*>(f.table32)[idx];
}

// Feature (2 values) of level l at position x -- blend of the 8 vertices --
// and, when jac != nullptr, its derivative with respect to the level's grid
// coordinate (jac[3 q + a] = d feature_q / d pos_a, pos = x N).
template <bool F16>
__device__ __forceinline__ float2 level_feature(const DevField& f, int l, const float x[3],
                                                const float dx[3], float* jac) {
  Cell c;
  make_cell(f, l, x, dx, c);
  float2 v[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) v[k] = vertex<F16>(f, c.idx[k]);
  const float wx = c.w[0], wy = c.w[1], wz = c.w[2];
  const float ux = 1.0f - wx, uy = 1.0f - wy, uz = 1.0f - wz;
  float2 r;
  r.x = uz * (uy * (ux * v[0].x + wx * v[1].x) + wy * (ux * v[2].x + wx * v[3].x)) +
        wz * (uy * (ux * v[4].x + wx * v[5].x) + wy * (ux * v[6].x + wx * v[7].x));
  r.y = uz * (uy * (ux * v[0].y + wx * v[1].y) + wy * (ux * v[2].y + wx * v[3].y)) +
        wz * (uy * (ux * v[4].y + wx * v[5].y) + wy * (ux * v[6].y + wx * v[7].y));
  if (jac) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      float t[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) t[k] = q ? v[k].y : v[k].x;
      jac[3 * q + 0] = uy * uz * (t[1] - t[0]) + wy * uz * (t[3] - t[2]) +
                       uy * wz * (t[5] - t[4]) + wy * wz * (t[7] - t[6]);
      jac[3 * q + 1] = ux * uz * (t[2] - t[0]) + wx * uz * (t[3] - t[1]) +
                       ux * wz * (t[6] - t[4]) + wx * wz * (t[7] - t[5]);
      jac[3 * q + 2] = ux * uy * (t[4] - t[0]) + wx * uy * (t[5] - t[1]) +
                       ux * wy * (t[6] - t[2]) + wx * wy * (t[7] - t[3]);
    }
  }
  return r;
}

__device__ __forceinline__ int feat_row(const DevField& f, int l, int q) {
  return (l & 3) * 2 * f.lpg + (l >> 2) * 2 + q;
}

__device__ __forceinline__ int jac_row(const DevField& f, int l, int q, int a) {
  return ((l & 3) * f.lpg + (l >> 2)) * 6 + 3 * q + a;
}

// ------------------------------------------------------------------ forward
// One thread: both levels of its group for one sample (the position is
// computed once).  Features and Jacobian rows are streamed out with
// non-temporal stores so that they do not displace the level tables from L2.
// GRAD: also store the Jacobian rows.
template <bool F16, bool GRAD>
__global__ __launch_bounds__(kBlock) void k_encode(DevField f, DevBatch b, DevWork w) {
  const int S = *w.total;
  const int grp = blockIdx.x % f.n_groups;
  const int stride = gridDim.x / f.n_groups;
  const int64_t cap = w.cap;
  for (int sb = blockIdx.x / f.n_groups; sb * kBlock < S; sb += stride) {
    const int s = sb * kBlock + threadIdx.x;
    if (s >= S) break;
    Pos ps = sample_pos(f, b, w, s);
#pragma unroll
    for (int li = 0; li < 2; ++li) {
      const int l = f.grp_lv[grp][li];
      float* r0 = w.feat + (int64_t)feat_row(f, l, 0) * cap;
      float* r1 = w.feat + (int64_t)feat_row(f, l, 1) * cap;
      __half* jr = w.jac + (int64_t)jac_row(f, l, 0, 0) * cap;
      float jac[6];
      float2 a = level_feature<F16>(f, l, ps.x, ps.dx, GRAD ? jac : nullptr);
      __builtin_nontemporal_store(a.x, r0 + s);
      __builtin_nontemporal_store(a.y, r1 + s);
      if (GRAD) {
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int c = 0; c < 3; ++c) {
            const float v = (ps.clamped >> c) & 1u ? 0.0f : jac[3 * q + c];
            __builtin_nontemporal_store(__half_as_ushort(__float2half_rn(v)),
                                        reinterpret_cast<unsigned short*>(jr) +
                                            (int64_t)(3 * q + c) * cap + s);
          }
      }
    }
  }
}

// ---------------------------------------------------------------- occupancy
// Occupancy grid: bit set iff the density at the cell centre exceeds `thr`.
// One thread per cell (linear index x + R(y + Rz)), plain FMA arithmetic; run
// once at field creation.
template <bool F16>
__global__ __launch_bounds__(kBlock) void k_occupancy(DevField f, uint32_t* bits, int R,
                                                      float thr) {
  __shared__ float s_w1[2 * kMaxLevels * kHidden];
  __shared__ float s_w2[kHidden];
  const int din = 2 * f.L;
  for (int i = threadIdx.x; i < din * kHidden; i += kBlock) s_w1[i] = f.wd1[i];
  if (threadIdx.x < kHidden) s_w2[threadIdx.x] = f.wd2[threadIdx.x * 16];
  __syncthreads();
  const int64_t n = (int64_t)R * R * R;
  const int64_t lin = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  bool occ = false;
  if (lin < n) {
    const int ci[3] = {(int)(lin % R), (int)((lin / R) % R), (int)(lin / ((int64_t)R * R))};
    float x[3];
    const float dx[3] = {0.0f, 0.0f, 0.0f};
    for (int a = 0; a < 3; ++a) {
      float ext = __fsub_rn(f.mx[a], f.mn[a]);
      float cell = __fdiv_rn(ext, (float)R);
      float p = __fadd_rn(f.mn[a], __fmul_rn(__fadd_rn((float)ci[a], 0.5f), cell));
      float xr = __fmul_rn(__fsub_rn(p, f.mn[a]), f.inv_ext[a]);
      x[a] = xr < 0.0f ? 0.0f : (xr > 1.0f ? 1.0f : xr);
    }
    float feat[2 * kMaxLevels];
    for (int l = 0; l < f.L; ++l) {
      float2 v = level_feature<F16>(f, l, x, dx, nullptr);
      feat[2 * l] = v.x;
      feat[2 * l + 1] = v.y;
    }
    float h0 = 0.0f;
    for (int j = 0; j < kHidden; ++j) {
      float a = 0.0f;
      for (int i = 0; i < din; ++i) a += feat[i] * s_w1[i * kHidden + j];
      h0 += (a > 0.0f ? a : 0.0f) * s_w2[j];
    }
    occ = __expf(h0 + f.density_bias) > thr;
  }
  const uint64_t bal = __ballot(occ);
  const int lane = threadIdx.x & 63;
  const int64_t word = (lin - lane) / 32 + (lane == 32 ? 1 : 0);
  const int64_t n_words = (n + 31) / 32;
  if ((lane == 0 || lane == 32) && word < n_words)
    bits[word] = lane == 0 ? (uint32_t)(bal & 0xFFFFFFFFu) : (uint32_t)(bal >> 32);
}

}  // namespace

int encode_blocks(const DevField& f, int n_cu, int per_cu) {
  // per_cu resident blocks of 256 threads per CU, rounded to a multiple of the
  // group count and of 8 (XCDs) so that each block keeps its group's XCD
  int unit = 8;
  while (unit % f.n_groups) unit += 8;
  int want = n_cu * per_cu;
  return ((want + unit - 1) / unit) * unit;
}

hipError_t launch_encode(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                         int with_grad, hipStream_t s) {
  if (f.f16) {
    if (with_grad)
      hipLaunchKernelGGL((k_encode<true, true>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w);
    else
      hipLaunchKernelGGL((k_encode<true, false>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w);
  } else {
    if (with_grad)
      hipLaunchKernelGGL((k_encode<false, true>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w);
    else
      hipLaunchKernelGGL((k_encode<false, false>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w);
  }
  return hipGetLastError();
}

hipError_t launch_occupancy(const DevField& f, uint32_t* bits, int R, float thr, hipStream_t s) {
  const int64_t n = (int64_t)R * R * R;
  const int64_t nb = (n + kBlock - 1) / kBlock;
  if (f.f16)
    hipLaunchKernelGGL(k_occupancy<true>, dim3((unsigned)nb), dim3(kBlock), 0, s, f, bits, R, thr);
  else
    hipLaunchKernelGGL(k_occupancy<false>, dim3((unsigned)nb), dim3(kBlock), 0, s, f, bits, R, thr);
  return hipGetLastError();
}

}  // namespace pnerf
