// Per-sample forward and backward of the frozen field: multiresolution hash
// encoding (gather), density and colour networks on MFMA, and -- backward --
// the input gradient through both networks and the trilinear interpolation to
// the sample position, folded into each sample's force and torque terms of
// Eq. 2 and Eq. 3.
//
// Work unit: one wavefront takes a tile of 64 consecutive compacted samples,
// as four 16-sample column tiles of v_mfma_f32_16x16x4_f32.  The batch (sample)
// dimension is the MFMA N dimension, so every layer's output rows (C layout:
// lane holds rows 4*(lane/16)+i of column lane%16) are directly the next
// layer's B operand once the K order is permuted; the permutation is baked into
// the weight tiles built at field creation, which each workgroup stages in LDS.
// Lane group g = lane/16 encodes levels g, g+4, g+8, g+12 of its column's
// sample, which is again exactly the B layout of the first layer.
#include "pnerf_internal.h"

namespace pnerf {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;  // 4 wavefronts
constexpr uint32_t kPrime1 = 2654435761u, kPrime2 = 805459861u;

__device__ __forceinline__ floatx4 mfma(float a, float b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

struct LevelLds {
  int32_t res[kMaxLevels];
  uint32_t n1[kMaxLevels];
  uint32_t dense[kMaxLevels];
};

struct Sample {
  float o[3], d[3], t;
  float x[3];       // normalised, clamped position in [0,1]^3 (decides cells)
  float dx[3];      // exact normalised position minus x (0 where clamped)
  uint32_t clamped; // bit a set: component a was clamped
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
__device__ inline void load_sample(const DevField& f, const DevBatch& b, const DevWork& w, int s,
                                   Sample& sm) {
  int ray = w.sray[s];
  const float* pose = b.poses + 12 * (ray / b.P);
  sm.o[0] = pose[3];
  sm.o[1] = pose[7];
  sm.o[2] = pose[11];
  sm.d[0] = w.rdx[ray];
  sm.d[1] = w.rdy[ray];
  sm.d[2] = w.rdz[ray];
  const float de[3] = {w.rex[ray], w.rey[ray], w.rez[ray]};
  sm.t = w.t[s];
  sm.clamped = 0;
  for (int a = 0; a < 3; ++a) {
    float td = __fmul_rn(sm.t, sm.d[a]);
    float e_td = fmaf(sm.t, sm.d[a], -td) + sm.t * de[a];
    float p = __fadd_rn(sm.o[a], td);
    float e_p = two_sum_err(sm.o[a], td, p);
    float q = __fsub_rn(p, f.mn[a]);
    float e_q = two_sum_err(p, -f.mn[a], q);
    float xr = __fmul_rn(q, f.inv_ext[a]);
    float e_x = fmaf(q, f.inv_ext[a], -xr);
    float dx = e_x + (e_td + e_p + e_q) * f.inv_ext[a] - xr * f.inv_ext_err[a];
    if (xr < 0.0f) {
      sm.x[a] = 0.0f;
      sm.dx[a] = 0.0f;
      sm.clamped |= 1u << a;
    } else if (xr > 1.0f) {
      sm.x[a] = 1.0f;
      sm.dx[a] = 0.0f;
      sm.clamped |= 1u << a;
    } else {
      sm.x[a] = xr;
      sm.dx[a] = dx;
    }
  }
}

// Cell of one level and the 8 corner table offsets (in float2 units).
struct Cell {
  float w[3];
  uint32_t idx[8];
};

// The cell comes from the float product x N (as a reference implementation in
// float decides it); the weights add back that product's rounding error and
// N dx, the part of the position float cannot hold.
__device__ __forceinline__ void make_cell(const LevelLds& lv, uint32_t T, int l, const float x[3],
                                          const float dx[3], Cell& c) {
  int N = lv.res[l];
  uint32_t n1 = lv.n1[l];
  bool dense = lv.dense[l] != 0;
  uint32_t i0[3];
  const float Nf = (float)N;
  for (int a = 0; a < 3; ++a) {
    float pos = __fmul_rn(x[a], Nf);
    int ci = (int)pos;
    ci = ci < N - 1 ? ci : N - 1;
    i0[a] = (uint32_t)ci;
    c.w[a] = (__fsub_rn(pos, (float)ci) + fmaf(x[a], Nf, -pos)) + Nf * dx[a];
  }
  uint32_t mask = T - 1u;
  uint32_t sy = dense ? n1 : kPrime1;
  uint32_t sz = dense ? n1 * n1 : kPrime2;
  uint32_t y0 = i0[1] * sy, y1 = y0 + sy;
  uint32_t z0 = i0[2] * sz, z1 = z0 + sz;
  uint32_t base = (uint32_t)l * T;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    uint32_t xi = i0[0] + (k & 1);
    uint32_t yi = (k & 2) ? y1 : y0;
    uint32_t zi = (k & 4) ? z1 : z0;
    uint32_t h = dense ? (xi + yi + zi) : ((xi ^ yi ^ zi) & mask);
    c.idx[k] = base + h;
  }
}

__device__ __forceinline__ float corner_w(const Cell& c, int k) {
  float wx = (k & 1) ? c.w[0] : 1.0f - c.w[0];
  float wy = (k & 2) ? c.w[1] : 1.0f - c.w[1];
  float wz = (k & 4) ? c.w[2] : 1.0f - c.w[2];
  return wx * wy * wz;
}

// Real SH of degree 0..3, the 4 functions 4g..4g+3 (no Condon-Shortley phase).
__device__ inline void sh4(const float d[3], int g, float out[4]) {
  const float x = d[0], y = d[1], z = d[2];
  const float C0 = 0.28209479177387814f, C1 = 0.4886025119029199f;
  const float C2a = 1.0925484305920792f, C2b = 0.31539156525252005f, C2c = 0.5462742152960396f;
  const float C3a = 0.5900435899266435f, C3b = 2.890611442640554f, C3c = 0.4570457994644658f;
  const float C3d = 0.3731763325901154f, C3e = 1.445305721320277f;
  float v[16];
  v[0] = C0;
  v[1] = C1 * y;
  v[2] = C1 * z;
  v[3] = C1 * x;
  v[4] = C2a * x * y;
  v[5] = C2a * y * z;
  v[6] = C2b * (3.0f * z * z - 1.0f);
  v[7] = C2a * x * z;
  v[8] = C2c * (x * x - y * y);
  v[9] = C3a * y * (3.0f * x * x - y * y);
  v[10] = C3b * x * y * z;
  v[11] = C3c * y * (5.0f * z * z - 1.0f);
  v[12] = C3d * z * (5.0f * z * z - 3.0f);
  v[13] = C3c * x * (5.0f * z * z - 1.0f);
  v[14] = C3e * z * (x * x - y * y);
  v[15] = C3a * x * (x * x - 3.0f * y * y);
#pragma unroll
  for (int i = 0; i < 4; ++i)
    out[i] = g == 0 ? v[i] : (g == 1 ? v[4 + i] : (g == 2 ? v[8 + i] : v[12 + i]));
}

// Gradient of SH functions 4g..4g+3 w.r.t. the direction, contracted with gs.
__device__ inline void sh4_vjp(const float d[3], int g, const float gs[4], float gd[3]) {
  const float x = d[0], y = d[1], z = d[2];
  const float C1 = 0.4886025119029199f;
  const float C2a = 1.0925484305920792f, C2b = 0.31539156525252005f, C2c = 0.5462742152960396f;
  const float C3a = 0.5900435899266435f, C3b = 2.890611442640554f, C3c = 0.4570457994644658f;
  const float C3d = 0.3731763325901154f, C3e = 1.445305721320277f;
  float G[4][3];
  if (g == 0) {  // Y_0, Y_1 (y), Y_2 (z), Y_3 (x)
    G[0][0] = 0.f; G[0][1] = 0.f; G[0][2] = 0.f;
    G[1][0] = 0.f; G[1][1] = C1;  G[1][2] = 0.f;
    G[2][0] = 0.f; G[2][1] = 0.f; G[2][2] = C1;
    G[3][0] = C1;  G[3][1] = 0.f; G[3][2] = 0.f;
  } else if (g == 1) {  // xy, yz, 3z^2-1, xz
    G[0][0] = C2a * y; G[0][1] = C2a * x; G[0][2] = 0.f;
    G[1][0] = 0.f;     G[1][1] = C2a * z; G[1][2] = C2a * y;
    G[2][0] = 0.f;     G[2][1] = 0.f;     G[2][2] = 6.0f * C2b * z;
    G[3][0] = C2a * z; G[3][1] = 0.f;     G[3][2] = C2a * x;
  } else if (g == 2) {  // x^2-y^2, y(3x^2-y^2), xyz, y(5z^2-1)
    G[0][0] = 2.0f * C2c * x;     G[0][1] = -2.0f * C2c * y;                    G[0][2] = 0.f;
    G[1][0] = 6.0f * C3a * x * y; G[1][1] = C3a * (3.0f * x * x - 3.0f * y * y); G[1][2] = 0.f;
    G[2][0] = C3b * y * z;        G[2][1] = C3b * x * z;                         G[2][2] = C3b * x * y;
    G[3][0] = 0.f;                G[3][1] = C3c * (5.0f * z * z - 1.0f);         G[3][2] = 10.0f * C3c * y * z;
  } else {  // z(5z^2-3), x(5z^2-1), z(x^2-y^2), x(x^2-3y^2)
    G[0][0] = 0.f;                                G[0][1] = 0.f;                 G[0][2] = C3d * (15.0f * z * z - 3.0f);
    G[1][0] = C3c * (5.0f * z * z - 1.0f);        G[1][1] = 0.f;                 G[1][2] = 10.0f * C3c * x * z;
    G[2][0] = 2.0f * C3e * x * z;                 G[2][1] = -2.0f * C3e * y * z; G[2][2] = C3e * (x * x - y * y);
    G[3][0] = C3a * (3.0f * x * x - 3.0f * y * y); G[3][1] = -6.0f * C3a * x * y; G[3][2] = 0.f;
  }
#pragma unroll
  for (int a = 0; a < 3; ++a) gd[a] = gs[0] * G[0][a] + gs[1] * G[1][a] + gs[2] * G[2][a] + gs[3] * G[3][a];
}

__device__ __forceinline__ float wA(const float* lds, int kstep_unit, int lane) {
  return lds[kstep_unit * 64 + lane];
}

__device__ inline void stage(float* lds, const float* src, int n, LevelLds& lv, const DevField& f) {
  for (int i = threadIdx.x; i < n; i += kBlock) lds[i] = src[i];
  if (threadIdx.x < kMaxLevels) {
    lv.res[threadIdx.x] = f.res[threadIdx.x];
    lv.n1[threadIdx.x] = f.n1[threadIdx.x];
    lv.dense[threadIdx.x] = f.dense[threadIdx.x];
  }
  __syncthreads();
}

// ------------------------------------------------------------------ forward
// GRAD = false (forward rendering only) skips the ReLU masks the backward
// pass needs; it is a separate kernel so that profiles keep the two apart.
template <int LPG, bool GRAD>
__global__ __launch_bounds__(kBlock) void k_shade_fwd(DevField f, DevBatch b, DevWork w) {
  constexpr int KD = 2 * LPG;  // density-layer K steps
  __shared__ float lds[fwd_tile_floats(LPG)];
  __shared__ LevelLds lv;
  stage(lds, f.wfwd, fwd_tile_floats(LPG), lv, f);

  const int S = *w.total;
  const int n_tiles = (S + kTile - 1) / kTile;
  const int lane = threadIdx.x & 63, g = lane >> 4, col = lane & 15;
  const int wave = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  const int n_waves = gridDim.x * (kBlock / 64);
  const float* D1 = lds + 64 * fwd_off_d1(LPG);
  const float* D2 = lds + 64 * fwd_off_d2(LPG);
  const float* C1 = lds + 64 * fwd_off_c1(LPG);
  const float* C2 = lds + 64 * fwd_off_c2(LPG);
  const float* C3 = lds + 64 * fwd_off_c3(LPG);

  for (int tile = wave; tile < n_tiles; tile += n_waves) {
    float feat[4][KD];
    float shv[4][4];
    int sidx[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      int s = tile * kTile + nt * 16 + col;
      sidx[nt] = s;
      Sample sm;
      load_sample(f, b, w, s < S ? s : S - 1, sm);
      sh4(sm.d, g, shv[nt]);
#pragma unroll
      for (int j = 0; j < LPG; ++j) {
        Cell c;
        make_cell(lv, f.T, 4 * j + g, sm.x, sm.dx, c);
        float2 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = reinterpret_cast<const float2*>(f.table32)[c.idx[k]];
        float a0 = 0.f, a1 = 0.f;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          float cw = corner_w(c, k);
          a0 += cw * v[k].x;
          a1 += cw * v[k].y;
        }
        feat[nt][2 * j] = a0;
        feat[nt][2 * j + 1] = a1;
      }
    }
    // density layer 1: a = relu(W_d1^T feat), 4 row tiles of 16 hidden units
    floatx4 acc[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) acc[m][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KD; ++ks)
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        float a = wA(D1, m * KD + ks, lane);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) acc[m][nt] = mfma(a, feat[nt][ks], acc[m][nt]);
      }
    uint32_t mk_a[4] = {0, 0, 0, 0}, mk_b1[4] = {0, 0, 0, 0}, mk_b2[4] = {0, 0, 0, 0};
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = acc[m][nt][i];
          bool on = v > 0.0f;
          acc[m][nt][i] = on ? v : 0.0f;
          mk_a[nt] |= (on ? 1u : 0u) << (4 * m + i);
        }
    // density layer 2: h = W_d2^T a (16 outputs)
    floatx4 h[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) h[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a = wA(D2, 4 * m + i, lane);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) h[nt] = mfma(a, acc[m][nt][i], h[nt]);
      }
    // colour layer 1 on [h (h_0 row has zero weights), SH_16]
    floatx4 b1[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) b1[m][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        float a = wA(C1, m * 8 + i, lane);
        float a2 = wA(C1, m * 8 + 4 + i, lane);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          b1[m][nt] = mfma(a, h[nt][i], b1[m][nt]);
          b1[m][nt] = mfma(a2, shv[nt][i], b1[m][nt]);
        }
      }
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = b1[m][nt][i];
          bool on = v > 0.0f;
          b1[m][nt][i] = on ? v : 0.0f;
          mk_b1[nt] |= (on ? 1u : 0u) << (4 * m + i);
        }
    // colour layer 2
    floatx4 b2[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) b2[m][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mp = 0; mp < 4; ++mp)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          float a = wA(C2, m * 16 + 4 * mp + i, lane);
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) b2[m][nt] = mfma(a, b1[mp][nt][i], b2[m][nt]);
        }
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = b2[m][nt][i];
          bool on = v > 0.0f;
          b2[m][nt][i] = on ? v : 0.0f;
          mk_b2[nt] |= (on ? 1u : 0u) << (4 * m + i);
        }
    // colour layer 3 (3 outputs in rows 0..2)
    floatx4 z[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) z[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mp = 0; mp < 4; ++mp)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a = wA(C3, 4 * mp + i, lane);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) z[nt] = mfma(a, b2[mp][nt][i], z[nt]);
      }
    // outputs: rows 0..3 live in lane group 0
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      int s = sidx[nt];
      if (g == 0 && s < S) {
        w.sig[s] = __expf(h[nt][0] + f.density_bias);
        w.cr[s] = 1.0f / (1.0f + __expf(-z[nt][0]));
        w.cg[s] = 1.0f / (1.0f + __expf(-z[nt][1]));
        w.cb[s] = 1.0f / (1.0f + __expf(-z[nt][2]));
      }
    }
    if (GRAD) {
      uint32_t* mw = w.masks + (size_t)tile * kMaskWords * 64 + lane;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) mw[nt * 64] = mk_a[nt] | (mk_b1[nt] << 16);
      mw[4 * 64] = mk_b2[0] | (mk_b2[1] << 16);
      mw[5 * 64] = mk_b2[2] | (mk_b2[3] << 16);
    }
  }
}

// ----------------------------------------------------------------- backward
template <int LPG>
__global__ __launch_bounds__(kBlock) void k_shade_bwd(DevField f, DevBatch b, DevWork w) {
  constexpr int MD = (LPG + 1) / 2;  // row tiles of the first-layer input gradient
  __shared__ float lds[bwd_tile_floats(LPG)];
  __shared__ LevelLds lv;
  stage(lds, f.wbwd, bwd_tile_floats(LPG), lv, f);

  const int S = *w.total;
  const int n_tiles = (S + kTile - 1) / kTile;
  const int lane = threadIdx.x & 63, g = lane >> 4, col = lane & 15;
  const int wave = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  const int n_waves = gridDim.x * (kBlock / 64);
  const float* C3 = lds + 64 * bwd_off_c3(LPG);
  const float* C2 = lds + 64 * bwd_off_c2(LPG);
  const float* C1 = lds + 64 * bwd_off_c1(LPG);
  const float* D2 = lds + 64 * bwd_off_d2(LPG);
  const float* D1 = lds + 64 * bwd_off_d1(LPG);
  const bool dir_grad = f.sh_dir_grad != 0;

  for (int tile = wave; tile < n_tiles; tile += n_waves) {
    uint32_t* mw = w.masks + (size_t)tile * kMaskWords * 64 + lane;
    uint32_t mk_a[4], mk_b1[4], mk_b2[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      uint32_t v = mw[nt * 64];
      mk_a[nt] = v & 0xFFFFu;
      mk_b1[nt] = v >> 16;
    }
    {
      uint32_t v4 = mw[4 * 64], v5 = mw[5 * 64];
      mk_b2[0] = v4 & 0xFFFFu;
      mk_b2[1] = v4 >> 16;
      mk_b2[2] = v5 & 0xFFFFu;
      mk_b2[3] = v5 >> 16;
    }
    float gzv[4], gh0[4];
    int sidx[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      int s = tile * kTile + nt * 16 + col;
      sidx[nt] = s;
      int sc = s < S ? s : S - 1;
      const float* src = g == 0 ? w.cr : (g == 1 ? w.cg : w.cb);
      gzv[nt] = g < 3 && s < S ? src[sc] : 0.0f;
      gh0[nt] = g == 0 && s < S ? w.sig[sc] : 0.0f;
    }
    // colour layer 3 transposed: gb2 = W_c3 gz (one K step: channels in lane groups)
    floatx4 gb2[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      float a = wA(C3, m, lane);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        gb2[m][nt] = mfma(a, gzv[nt], floatx4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (!((mk_b2[nt] >> (4 * m + i)) & 1u)) gb2[m][nt][i] = 0.0f;
      }
    }
    // colour layer 2 transposed
    floatx4 gb1[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) gb1[m][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mp = 0; mp < 4; ++mp)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          float a = wA(C2, m * 16 + 4 * mp + i, lane);
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) gb1[m][nt] = mfma(a, gb2[mp][nt][i], gb1[m][nt]);
        }
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (!((mk_b1[nt] >> (4 * m + i)) & 1u)) gb1[m][nt][i] = 0.0f;
    // colour layer 1 transposed: rows = h index (row 0 has zero weights); optional SH rows
    floatx4 gh[4], gsh[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      gh[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
      gsh[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int mp = 0; mp < 4; ++mp)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a = wA(C1, 4 * mp + i, lane);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) gh[nt] = mfma(a, gb1[mp][nt][i], gh[nt]);
      }
    if (dir_grad) {
#pragma unroll
      for (int mp = 0; mp < 4; ++mp)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float a = wA(C1, 16 + 4 * mp + i, lane);
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) gsh[nt] = mfma(a, gb1[mp][nt][i], gsh[nt]);
        }
    }
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) gh[nt][0] += gh0[nt];  // d loss / d h_0 (zero off group 0)
    // density layer 2 transposed: ga = W_d2 gh, masked
    floatx4 ga[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) ga[m][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a = wA(D2, m * 4 + i, lane);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) ga[m][nt] = mfma(a, gh[nt][i], ga[m][nt]);
      }
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (!((mk_a[nt] >> (4 * m + i)) & 1u)) ga[m][nt][i] = 0.0f;
    }
    // density layer 1 transposed: gf rows permuted so lane group g gets its levels
    floatx4 gf[MD][4];
#pragma unroll
    for (int m = 0; m < MD; ++m)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) gf[m][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mp = 0; mp < 4; ++mp)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int m = 0; m < MD; ++m) {
          float a = wA(D1, m * 16 + 4 * mp + i, lane);
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) gf[m][nt] = mfma(a, ga[mp][nt][i], gf[m][nt]);
        }
    // trilinear backward to the position, then force / torque of this sample
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      int s = sidx[nt];
      Sample sm;
      load_sample(f, b, w, s < S ? s : S - 1, sm);
      float gx[3] = {0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < LPG; ++j) {
        int l = 4 * j + g;
        Cell c;
        make_cell(lv, f.T, l, sm.x, sm.dx, c);
        float2 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = reinterpret_cast<const float2*>(f.table32)[c.idx[k]];
        float g0 = gf[j / 2][nt][2 * (j % 2)], g1 = gf[j / 2][nt][2 * (j % 2) + 1];
        float dt[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) dt[k] = g0 * v[k].x + g1 * v[k].y;
        float wx = c.w[0], wy = c.w[1], wz = c.w[2];
        float ux = 1.f - wx, uy = 1.f - wy, uz = 1.f - wz;
        float ddx = uy * uz * (dt[1] - dt[0]) + wy * uz * (dt[3] - dt[2]) +
                    uy * wz * (dt[5] - dt[4]) + wy * wz * (dt[7] - dt[6]);
        float ddy = ux * uz * (dt[2] - dt[0]) + wx * uz * (dt[3] - dt[1]) +
                    ux * wz * (dt[6] - dt[4]) + wx * wz * (dt[7] - dt[5]);
        float ddz = ux * uy * (dt[4] - dt[0]) + wx * uy * (dt[5] - dt[1]) +
                    ux * wy * (dt[6] - dt[2]) + wx * wy * (dt[7] - dt[3]);
        float N = (float)lv.res[l];
        gx[0] += N * ddx;
        gx[1] += N * ddy;
        gx[2] += N * ddz;
      }
      float gd[3] = {0.f, 0.f, 0.f};
      if (dir_grad) {
        float gs[4] = {gsh[nt][0], gsh[nt][1], gsh[nt][2], gsh[nt][3]};
        sh4_vjp(sm.d, g, gs, gd);
      }
#pragma unroll
      for (int a = 0; a < 3; ++a) {
        gx[a] += __shfl_xor(gx[a], 16);
        gx[a] += __shfl_xor(gx[a], 32);
        gd[a] += __shfl_xor(gd[a], 16);
        gd[a] += __shfl_xor(gd[a], 32);
      }
      float gp[3];
#pragma unroll
      for (int a = 0; a < 3; ++a) gp[a] = (sm.clamped >> a) & 1u ? 0.0f : gx[a] * f.inv_ext[a];
      // torque t (d x gp) + d x gd, force gp
      float m3[3] = {sm.t * gp[0], sm.t * gp[1], sm.t * gp[2]};
      float out[6];
      out[0] = sm.d[1] * m3[2] - sm.d[2] * m3[1] + (sm.d[1] * gd[2] - sm.d[2] * gd[1]);
      out[1] = sm.d[2] * m3[0] - sm.d[0] * m3[2] + (sm.d[2] * gd[0] - sm.d[0] * gd[2]);
      out[2] = sm.d[0] * m3[1] - sm.d[1] * m3[0] + (sm.d[0] * gd[1] - sm.d[1] * gd[0]);
      out[3] = gp[0];
      out[4] = gp[1];
      out[5] = gp[2];
      float* ow = reinterpret_cast<float*>(w.masks) + (size_t)tile * kMaskWords * 64 + nt * 16 + col;
      if (s < S) {
        // lane group g stores outputs g and g + 4
        float o1 = g == 0 ? out[0] : (g == 1 ? out[1] : (g == 2 ? out[2] : out[3]));
        ow[g * 64] = o1;
        if (g < 2) ow[(g + 4) * 64] = g == 0 ? out[4] : out[5];
      }
    }
  }
}


// ---------------------------------------------------------------- occupancy
// Occupancy grid: bit set iff the density at the cell centre exceeds `thr`.
// One thread per cell (linear index x + R(y + Rz)), plain FMA arithmetic; run
// once at field creation.
__global__ __launch_bounds__(kBlock) void k_occupancy(DevField f, uint32_t* bits, int R,
                                                      float thr) {
  __shared__ float s_w1[32 * kHidden];
  __shared__ float s_w2[kHidden];
  __shared__ LevelLds lv;
  int din = 2 * f.L;
  for (int i = threadIdx.x; i < din * kHidden; i += kBlock) s_w1[i] = f.wd1[i];
  if (threadIdx.x < kHidden) s_w2[threadIdx.x] = f.wd2[threadIdx.x * 16];
  if (threadIdx.x < kMaxLevels) {
    lv.res[threadIdx.x] = f.res[threadIdx.x];
    lv.n1[threadIdx.x] = f.n1[threadIdx.x];
    lv.dense[threadIdx.x] = f.dense[threadIdx.x];
  }
  __syncthreads();
  int64_t n = (int64_t)R * R * R;
  int64_t lin = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  bool occ = false;
  if (lin < n) {
    int ci[3] = {(int)(lin % R), (int)((lin / R) % R), (int)(lin / ((int64_t)R * R))};
    float x[3], dx[3] = {0.0f, 0.0f, 0.0f};
    {
      for (int a = 0; a < 3; ++a) {
        float ext = __fsub_rn(f.mx[a], f.mn[a]);
        float cell = __fdiv_rn(ext, (float)R);
        float p = __fadd_rn(f.mn[a], __fmul_rn(__fadd_rn((float)ci[a], 0.5f), cell));
        float xr = __fmul_rn(__fsub_rn(p, f.mn[a]), f.inv_ext[a]);
        x[a] = xr < 0.0f ? 0.0f : (xr > 1.0f ? 1.0f : xr);
      }
    }
    float feat[32];
    for (int l = 0; l < f.L; ++l) {
      Cell c;
      make_cell(lv, f.T, l, x, dx, c);
      float a0 = 0.f, a1 = 0.f;
      for (int k = 0; k < 8; ++k) {
        float2 v = reinterpret_cast<const float2*>(f.table32)[c.idx[k]];
        float cw = corner_w(c, k);
        a0 += cw * v.x;
        a1 += cw * v.y;
      }
      feat[2 * l] = a0;
      feat[2 * l + 1] = a1;
    }
    float h0 = 0.0f;
    for (int j = 0; j < kHidden; ++j) {
      float a = 0.0f;
      for (int i = 0; i < din; ++i) a += feat[i] * s_w1[i * kHidden + j];
      h0 += (a > 0.0f ? a : 0.0f) * s_w2[j];
    }
    occ = __expf(h0 + f.density_bias) > thr;
  }
  uint64_t bal = __ballot(occ);
  int lane = threadIdx.x & 63;
  int64_t word = (lin - lane) / 32 + (lane == 32 ? 1 : 0);
  int64_t n_words = (n + 31) / 32;
  if ((lane == 0 || lane == 32) && word < n_words)
    bits[word] = lane == 0 ? (uint32_t)(bal & 0xFFFFFFFFu) : (uint32_t)(bal >> 32);
}

}  // namespace

int shade_fwd_blocks_per_cu(int lpg) {
  int n = 0;
  hipError_t e = hipErrorInvalidValue;
  switch (lpg) {
    case 1: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_shade_fwd<1, true>, kBlock, 0); break;
    case 2: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_shade_fwd<2, true>, kBlock, 0); break;
    case 3: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_shade_fwd<3, true>, kBlock, 0); break;
    case 4: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_shade_fwd<4, true>, kBlock, 0); break;
  }
  return e == hipSuccess && n > 0 ? n : 1;
}

int shade_bwd_blocks_per_cu(int lpg) {
  int n = 0;
  hipError_t e = hipErrorInvalidValue;
  switch (lpg) {
    case 1: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_shade_bwd<1>, kBlock, 0); break;
    case 2: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_shade_bwd<2>, kBlock, 0); break;
    case 3: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_shade_bwd<3>, kBlock, 0); break;
    case 4: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_shade_bwd<4>, kBlock, 0); break;
  }
  return e == hipSuccess && n > 0 ? n : 1;
}

template <bool GRAD>
void launch_fwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                hipStream_t s) {
  switch (f.lpg) {
    case 1: hipLaunchKernelGGL((k_shade_fwd<1, GRAD>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 2: hipLaunchKernelGGL((k_shade_fwd<2, GRAD>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 3: hipLaunchKernelGGL((k_shade_fwd<3, GRAD>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 4: hipLaunchKernelGGL((k_shade_fwd<4, GRAD>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
  }
}

hipError_t launch_shade_fwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                            int with_grad, hipStream_t s) {
  if (f.lpg < 1 || f.lpg > 4) return hipErrorInvalidValue;
  if (with_grad)
    launch_fwd<true>(f, b, w, n_blocks, s);
  else
    launch_fwd<false>(f, b, w, n_blocks, s);
  return hipGetLastError();
}

hipError_t launch_occupancy(const DevField& f, uint32_t* bits, int R, float thr, hipStream_t s) {
  int64_t n = (int64_t)R * R * R;
  int64_t nb = (n + kBlock - 1) / kBlock;
  hipLaunchKernelGGL(k_occupancy, dim3((unsigned)nb), dim3(kBlock), 0, s, f, bits, R, thr);
  return hipGetLastError();
}

hipError_t launch_shade_bwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                            hipStream_t s) {
  switch (f.lpg) {
    case 1: hipLaunchKernelGGL(k_shade_bwd<1>, dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 2: hipLaunchKernelGGL(k_shade_bwd<2>, dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 3: hipLaunchKernelGGL(k_shade_bwd<3>, dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 4: hipLaunchKernelGGL(k_shade_bwd<4>, dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace pnerf
