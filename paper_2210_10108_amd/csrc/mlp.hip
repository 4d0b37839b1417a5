// Density and colour networks of the frozen field on MFMA (Sec. III: the
// field's small MLPs), forward and -- backward -- the input gradient through
// both networks to d loss / d feature, then through the encoding's stored
// Jacobian to d loss / d p of every sample (and, on the view-direction path,
// through the SH input to d loss / d direction), ending in each sample's force
// and torque terms of Eq. 2 and Eq. 3.
//
// Arithmetic (mlp_precision 0): every fp32 operand x is split into bf16 parts
// x = hi + lo + r (|r| <= 2^-17 |x|), and each product is accumulated in fp32
// as hi*hi + hi*lo + lo*hi by v_mfma_f32_16x16x32_bf16 (the dropped lo*lo and
// r terms are about 2^-16 of the product).  The weights are split once at
// field creation; fp16-stored weights split exactly.  Activations are split
// two at a time (split2): two packed converts and two bf16 dot products per
// pair.  mlp_precision 1: each weight as two fp16 parts w = hi + lo (split
// once at field creation, |w - hi - lo| <= 2^-22 |w|), each activation
// rounded to fp16, and two v_mfma_f32_16x16x32_f16 products hi*x + lo*x per
// fp32 product, accumulated in fp32: the activation's rounding (2^-12) is the
// only error of note, and one packed convert per pair replaces the split.  The
// backward networks scale each sample's incoming gradient by a power of two
// that puts its largest component in [16, 32), so that the fp16 operands stay
// normal, and scale the result back (both exact).
//
// Work unit: one wavefront takes a tile of NT * 16 consecutive compacted
// samples, as NT 16-sample column tiles.  The batch (sample) dimension is the MFMA N
// dimension.  A layer's accumulators hold (C layout) rows 4*(lane/16)+i of
// column lane%16 of each 16-row tile; two such tiles are exactly one 32-deep
// K step of the next layer's B operand (lane group g holds K positions
// 8g..8g+7), once the K order -- hidden unit 16(2s + j/4) + 4g + j%4 at
// position j of step s -- is baked into the weight tiles built at field
// creation, which each workgroup stages in LDS (hi and lo parts).
// Lane group g reads the features of levels g, g+4, g+8, g+12 of its column's
// sample (rows 2 LPG g .. of the SoA feature array): the first layer's B
// operand.
#include <algorithm>

#include "pnerf_internal.h"
#include "render_common.h"

namespace pnerf {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr int kBlock = 512;  // 8 wavefronts: one LDS copy of the weight units serves 8 waves
constexpr int kFwdNT = 1;    // 16-sample column tiles per wavefront, forward
constexpr int kBwdNT = 1;    // and backward (68 registers without the SH direction path: 7 wavefronts per SIMD)

struct Split {
  bf16x8 hi, lo;
};

// The bf16 pairs (-1, 0) and (0, -1).  They come from the field as data: an
// inline constant for this instruction's packed bf16 operand is not read the
// way the compiler encodes it (-1.0 lands in the upper half), so the kernels
// never let it become one.
struct SplitK {
  bf16x2 m0, m1;
};

__device__ __forceinline__ SplitK split_k(const DevField& f) {
  return {__builtin_bit_cast(bf16x2, f.bf16_neg1[0]), __builtin_bit_cast(bf16x2, f.bf16_neg1[1])};
}

// A pair x0, x1 as x = hi + lo (+ a remainder below 2^-17 |x|), both parts
// rounded to nearest: hi by one packed convert; x - hi, exact in fp32, by one
// bf16 dot product each (hi . (-1, 0) + x0, hi . (0, -1) + x1); lo by one
// more packed convert.
__device__ __forceinline__ void split2(float x0, float x1, const SplitK& k, uint32_t& hi,
                                       uint32_t& lo) {
  const bf16x2 h = {(__bf16)x0, (__bf16)x1};
  const float l0 = __builtin_amdgcn_fdot2_f32_bf16(h, k.m0, x0, false);
  const float l1 = __builtin_amdgcn_fdot2_f32_bf16(h, k.m1, x1, false);
  const bf16x2 l = {(__bf16)l0, (__bf16)l1};
  hi = __builtin_bit_cast(uint32_t, h);
  lo = __builtin_bit_cast(uint32_t, l);
}

__device__ __forceinline__ Split split8(const float v[8], const SplitK& k) {
  u32x4 hw, lw;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    uint32_t h, l;
    split2(v[2 * p], v[2 * p + 1], k, h, l);
    hw[p] = h;
    lw[p] = l;
  }
  Split s;
  s.hi = __builtin_bit_cast(bf16x8, hw);
  s.lo = __builtin_bit_cast(bf16x8, lw);
  return s;
}

// c += A B for split operands (small terms first).  The wave's issue
// priority is raised while it issues the products, so that a wave with MFMA
// work ready goes ahead of the waves splitting their next operands on the
// vector ALU and the two pipes overlap (the networks' kernels ran 3-5% faster
// on the 2^21-entry workload).
__device__ __forceinline__ floatx4 mfma3(const Split& a, const Split& b, floatx4 c) {
  __builtin_amdgcn_s_setprio(1);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.lo, b.hi, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.hi, b.lo, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.hi, b.hi, c, 0, 0, 0);
  __builtin_amdgcn_s_setprio(0);
  return c;
}

// A operand of weight unit u (hi and lo parts, 16 bytes per lane each).
__device__ __forceinline__ Split load_unit(const WeightUnit* lds, int u, int lane) {
  Split s;
  s.hi = __builtin_bit_cast(bf16x8, lds[u].hi[lane]);
  s.lo = __builtin_bit_cast(bf16x8, lds[u].lo[lane]);
  return s;
}

// The B operand of one K step from two accumulator tiles (rows of tile t0 at
// positions 0..3, of tile t1 at 4..7) for a ReLU layer: relu(t0), relu(t1) and, when
// MASK, its mask bits.  Position v of the K step is value pair p = v / 2:
// the pair's bits are at shift + p (even v) and shift + p + 16 (odd v) of mk.
// max(bits, 0) as a signed integer is the ReLU (every non-positive float, -0
// included, has a bit pattern <= 0); a unit counts as active when its hi part
// is nonzero, which differs from x > 0 only for positive values below
// 2^-133.  Both halves of the packed hi are then below 0x8000, so adding
// 0x7FFF to each sets its top bit exactly when it is nonzero, without a carry
// into the other half.
template <bool MASK>
__device__ __forceinline__ Split relu_pack2(const floatx4& t0, const floatx4& t1, const SplitK& k,
                                            uint32_t& mk, int shift) {
  float v[8] = {t0[0], t0[1], t0[2], t0[3], t1[0], t1[1], t1[2], t1[3]};
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = __int_as_float(max(__float_as_int(v[i]), 0));
  u32x4 hw, lw;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    uint32_t h, l;
    split2(v[2 * p], v[2 * p + 1], k, h, l);
    hw[p] = h;
    lw[p] = l;
    if (MASK) {
      const uint32_t top = h + 0x7FFF7FFFu;  // bits 15 and 31: the halves are nonzero
      mk |= (top >> (15 - shift - p)) & (0x00010001u << (shift + p));
    }
  }
  Split s;
  s.hi = __builtin_bit_cast(bf16x8, hw);
  s.lo = __builtin_bit_cast(bf16x8, lw);
  return s;
}

// Copy n_units weight units of `words` 16-byte words each to LDS.
__device__ inline void stage(void* lds, const void* src, int n_units, int words) {
  const uint4* s = reinterpret_cast<const uint4*>(src);
  uint4* d = reinterpret_cast<uint4*>(lds);
  for (int i = threadIdx.x; i < n_units * words; i += kBlock) d[i] = s[i];
}

// An fp16 B operand of a K step (8 values per lane), and an fp16 A operand
// as two parts.
struct Half8 {
  f16x8 v;
};
struct Half8x2 {
  f16x8 hi, lo;
};

__device__ __forceinline__ uint32_t half2_rn(float x0, float x1) {
  const f16x2 h = {(_Float16)x0, (_Float16)x1};
  return __builtin_bit_cast(uint32_t, h);
}

// The two arithmetics behind one interface: the B operand type of a K step
// (Op), the A operand (AOp, weights), and pack (8 values), relu_pack (relu of
// two accumulator tiles, with their mask bits when MASK), mma (c += A B) and
// load (A operand of a weight unit staged in LDS).
template <bool H>
struct Arith;

template <>
struct Arith<false> {
  using Op = Split;
  using AOp = Split;
  using Unit = WeightUnit;
  static constexpr int kWords = 128;  // 16-byte words per staged unit (hi and lo)
  __device__ static __forceinline__ Op pack(const float v[8], const SplitK& k) {
    return split8(v, k);
  }
  template <bool MASK>
  __device__ static __forceinline__ Op relu_pack(const floatx4& t0, const floatx4& t1,
                                                 const SplitK& k, uint32_t& mk, int shift) {
    return relu_pack2<MASK>(t0, t1, k, mk, shift);
  }
  __device__ static __forceinline__ floatx4 mma(const AOp& a, const Op& b, floatx4 c) {
    return mfma3(a, b, c);
  }
  __device__ static __forceinline__ AOp load(const Unit* lds, int u, int lane) {
    return load_unit(lds, u, lane);
  }
  __device__ static __forceinline__ const Unit* fwd(const DevField& f) { return f.wfwd; }
  __device__ static __forceinline__ const Unit* bwd(const DevField& f) { return f.wbwd; }
};

template <>
struct Arith<true> {
  using Op = Half8;
  using AOp = Half8x2;
  using Unit = WeightUnit;  // fp16 hi and lo parts
  static constexpr int kWords = 128;
  __device__ static __forceinline__ Op pack(const float v[8], const SplitK&) {
    u32x4 w;
#pragma unroll
    for (int p = 0; p < 4; ++p) w[p] = half2_rn(v[2 * p], v[2 * p + 1]);
    return {__builtin_bit_cast(f16x8, w)};
  }
  // relu as in relu_pack2; a unit counts as active when its fp16 value is
  // nonzero (positive values below 2^-25 round to zero and count as off),
  // found by the same carry-free add: both halves are below 0x8000
  template <bool MASK>
  __device__ static __forceinline__ Op relu_pack(const floatx4& t0, const floatx4& t1,
                                                 const SplitK&, uint32_t& mk, int shift) {
    float v[8] = {t0[0], t0[1], t0[2], t0[3], t1[0], t1[1], t1[2], t1[3]};
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = __int_as_float(max(__float_as_int(v[i]), 0));
    u32x4 w;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t h = half2_rn(v[2 * p], v[2 * p + 1]);
      w[p] = h;
      if (MASK) {
        const uint32_t top = h + 0x7FFF7FFFu;
        mk |= (top >> (15 - shift - p)) & (0x00010001u << (shift + p));
      }
    }
    return {__builtin_bit_cast(f16x8, w)};
  }
  __device__ static __forceinline__ floatx4 mma(const AOp& a, const Op& b, floatx4 c) {
    __builtin_amdgcn_s_setprio(1);  // as in mfma3
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(a.lo, b.v, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(a.hi, b.v, c, 0, 0, 0);
    __builtin_amdgcn_s_setprio(0);
    return c;
  }
  __device__ static __forceinline__ AOp load(const Unit* lds, int u, int lane) {
    return {__builtin_bit_cast(f16x8, lds[u].hi[lane]), __builtin_bit_cast(f16x8, lds[u].lo[lane])};
  }
  __device__ static __forceinline__ const Unit* fwd(const DevField& f) { return f.hfwd; }
  __device__ static __forceinline__ const Unit* bwd(const DevField& f) { return f.hbwd; }
};

// Unit ray direction of sample s.
__device__ __forceinline__ void sample_dir(const DevWork& w, int s, float d[3]) {
  int ray = w.sray[s];
  d[0] = w.rdx[ray];
  d[1] = w.rdy[ray];
  d[2] = w.rdz[ray];
}

// Mask bits of a ReLU layer's 16 values t[m][i] of one column tile (unit
// 16m + 4g + i): value v = 4m + i is K position v % 8 of K step v / 8, so its
// bit is base + 4 (v / 8) + (v % 8) / 2, plus 16 for odd v (see relu_pack2).
__device__ __forceinline__ void apply_mask(floatx4 (&t)[4], uint32_t mk, int base) {
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = 4 * m + i;
      const int bit = base + 4 * (v / 8) + (v % 8) / 2 + 16 * (v & 1);
      if (!((mk >> bit) & 1u)) t[m][i] = 0.0f;
    }
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

// ------------------------------------------------------------------ forward
// GRAD = false (forward rendering only) skips the ReLU masks the backward
// pass needs; it is a separate kernel so that profiles keep the two apart.
template <int LPG, bool GRAD, bool H>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void k_mlp_fwd(DevField f, DevBatch b, DevWork w) {
  using A = Arith<H>;
  using Op = typename A::Op;
  constexpr int KD = 2 * LPG;  // features per lane group
  constexpr int NT = kFwdNT, TS = 16 * NT;
  __shared__ typename A::Unit lds[kFwdUnits];
  stage(lds, A::fwd(f), kFwdUnits, A::kWords);
  __syncthreads();

  const int S = *w.total;
  const int n_tiles = (S + TS - 1) / TS;
  const int lane = threadIdx.x & 63, g = lane >> 4, col = lane & 15;
  const int wave = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  const int n_waves = gridDim.x * (kBlock / 64);
  const float* frow = w.feat + (int64_t)(g * KD) * w.cap;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  const SplitK sk = split_k(f);

  for (int tile = wave; tile < n_tiles; tile += n_waves) {
    // the weight units are re-read from LDS every tile (hoisted, they would
    // take ~160 registers and spill)
    asm volatile("" ::: "memory");
    Op xf[NT];
    float shv[NT][4];
    int sidx[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int s = tile * TS + nt * 16 + col;
      sidx[nt] = s;
      const int sc = s < S ? s : S - 1;
      float v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = j < KD ? frow[(int64_t)j * w.cap + sc] : 0.0f;
      xf[nt] = A::pack(v, sk);
      // SH functions 4g..4g+3 of the sample's ray (sh16, stored per ray)
      const float4 sh = reinterpret_cast<const float4*>(w.rsh)[4 * w.sray[sc] + g];
      shv[nt][0] = sh.x;
      shv[nt][1] = sh.y;
      shv[nt][2] = sh.z;
      shv[nt][3] = sh.w;
    }
    // density layer 1: a = relu(W_d1^T feat), 4 row tiles of 16 hidden units
    floatx4 acc[NT][4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const typename A::AOp a = A::load(lds, kFD1 + m, lane);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[nt][m] = A::mma(a, xf[nt], zero);
    }
    // mask words: layer a at base 0 and colour layer 1 at base 8 of word 0,
    // colour layer 2 at base 0 of word 1 (bit layout: relu_pack2)
    uint32_t mw0[NT], mw1[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) mw0[nt] = mw1[nt] = 0u;
    // density layer 2: h = W_d2^T relu(a) (16 outputs)
    floatx4 h[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) h[nt] = zero;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const typename A::AOp a = A::load(lds, kFD2 + s2, lane);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        h[nt] = A::mma(a, A::template relu_pack<GRAD>(acc[nt][2 * s2], acc[nt][2 * s2 + 1], sk,
                                                      mw0[nt], 4 * s2),
                       h[nt]);
    }
    // colour layer 1 on [h (h_0 has zero weights), SH_16]
    floatx4 b1[NT][4];
    {
      Op xc[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const float v[8] = {h[nt][0], h[nt][1], h[nt][2], h[nt][3],
                            shv[nt][0], shv[nt][1], shv[nt][2], shv[nt][3]};
        xc[nt] = A::pack(v, sk);
      }
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const typename A::AOp a = A::load(lds, kFC1 + m, lane);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) b1[nt][m] = A::mma(a, xc[nt], zero);
      }
    }
    // colour layer 2 on relu(b1)
    floatx4 b2[NT][4];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int m = 0; m < 4; ++m) b2[nt][m] = zero;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      Op x[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        x[nt] = A::template relu_pack<GRAD>(b1[nt][2 * s2], b1[nt][2 * s2 + 1], sk, mw0[nt],
                                            8 + 4 * s2);
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const typename A::AOp a = A::load(lds, kFC2 + 2 * m + s2, lane);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) b2[nt][m] = A::mma(a, x[nt], b2[nt][m]);
      }
    }
    // colour layer 3 on relu(b2) (3 outputs in rows 0..2)
    floatx4 z[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) z[nt] = zero;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const typename A::AOp a = A::load(lds, kFC3 + s2, lane);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        z[nt] = A::mma(a, A::template relu_pack<GRAD>(b2[nt][2 * s2], b2[nt][2 * s2 + 1], sk,
                                                      mw1[nt], 4 * s2),
                       z[nt]);
    }
    // outputs: rows 0..3 live in lane group 0
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int s = sidx[nt];
      if (g == 0 && s < S) {
        // sigmoid with the hardware reciprocal (1 ulp)
        w.sig[s] = __expf(h[nt][0] + f.density_bias);
        w.cr[s] = __builtin_amdgcn_rcpf(1.0f + __expf(-z[nt][0]));
        w.cg[s] = __builtin_amdgcn_rcpf(1.0f + __expf(-z[nt][1]));
        w.cb[s] = __builtin_amdgcn_rcpf(1.0f + __expf(-z[nt][2]));
      }
    }
    if (GRAD) {
      // two words per lane per 16-sample column tile
      uint32_t* mw = w.masks + (size_t)tile * NT * 2 * 64 + lane;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        mw[(2 * nt) * 64] = mw0[nt];
        mw[(2 * nt + 1) * 64] = mw1[nt];
      }
    }
  }
}

// ----------------------------------------------------------------- backward
// The backward networks for one 16-sample column tile: lane (g, col) holds
// the sample of column col.  In: z = d loss / d z of that sample (zero when it
// has none), gh0 = d loss / d h_0 of that sample (in every lane group), the
// sample's two ReLU mask words as the forward kernel stored them for this lane
// group, and sc = the sample whose Jacobian records are read (any valid sample
// when the column is empty).  Out: d loss / d p of the sample, gx (in every
// lane group, after the sums over the groups), and on the direction path the
// term d loss / d d through the SH input, gd (likewise summed).
template <int LPG, bool DIR, bool H>
__device__ __forceinline__ void bwd_tile(const DevField& f, const DevWork& w,
                                         const typename Arith<H>::Unit* lds, const float* s_c3,
                                         const SplitK& sk, int lane, const float zin[3],
                                         float gh0in, uint32_t mw0, uint32_t mw1, int sc,
                                         const float d[3], float gx[3], float gd[3]) {
  using A = Arith<H>;
  using Op = typename A::Op;
  constexpr int MD = (LPG + 1) / 2;  // row tiles of d loss / d feature
  const int g = lane >> 4;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  // fp16 operands: the sample's gradient scaled by 2^k, its largest component
  // (biased exponent ex) into [16, 32); k is kept within +-100
  float scale = 1.0f, unscale = 1.0f;
  if (H) {
    const float m = fmaxf(fmaxf(fabsf(zin[0]), fabsf(zin[1])), fmaxf(fabsf(zin[2]), fabsf(gh0in)));
    const int ex = (__float_as_int(m) >> 23) & 0xFF;
    const int k = min(max(131 - ex, -100), 100);
    scale = __int_as_float((127 + k) << 23);
    unscale = __int_as_float((127 - k) << 23);
  }
  const float z[3] = {zin[0] * scale, zin[1] * scale, zin[2] * scale};
  const float gh0 = g == 0 ? gh0in * scale : 0.0f;
  // colour layer 3 transposed, in fp32 on the vector ALUs: gb2 = W_c3 gz
  // (rows 16m + 4g + i of this lane), masked by layer 2's ReLU
  floatx4 gb2[4];
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float* c3 = s_c3 + 3 * (16 * m + 4 * g + i);
      gb2[m][i] = c3[0] * z[0] + c3[1] * z[1] + c3[2] * z[2];
    }
  apply_mask(gb2, mw1, 0);
  // colour layer 2 transposed
  floatx4 gb1[4] = {zero, zero, zero, zero};
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
    const float v[8] = {gb2[2 * s2][0], gb2[2 * s2][1], gb2[2 * s2][2], gb2[2 * s2][3],
                        gb2[2 * s2 + 1][0], gb2[2 * s2 + 1][1], gb2[2 * s2 + 1][2], gb2[2 * s2 + 1][3]};
    const Op x = A::pack(v, sk);
#pragma unroll
    for (int m = 0; m < 4; ++m) gb1[m] = A::mma(A::load(lds, kBC2 + 2 * m + s2, lane), x, gb1[m]);
  }
  apply_mask(gb1, mw0, 8);
  // colour layer 1 transposed: rows = h index (row 0 has zero weights); SH rows
  floatx4 gh = zero, gsh = zero;
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
    const float v[8] = {gb1[2 * s2][0], gb1[2 * s2][1], gb1[2 * s2][2], gb1[2 * s2][3],
                        gb1[2 * s2 + 1][0], gb1[2 * s2 + 1][1], gb1[2 * s2 + 1][2], gb1[2 * s2 + 1][3]};
    const Op x = A::pack(v, sk);
    gh = A::mma(A::load(lds, kBC1 + s2, lane), x, gh);
    if (DIR) gsh = A::mma(A::load(lds, kBSH + s2, lane), x, gsh);
  }
  gh[0] += gh0;  // d loss / d h_0 (zero off group 0)
  // density layer 2 transposed: ga = W_d2 gh (one K step, upper half zero), masked
  floatx4 ga[4];
  {
    const float v[8] = {gh[0], gh[1], gh[2], gh[3], 0.f, 0.f, 0.f, 0.f};
    const Op x = A::pack(v, sk);
#pragma unroll
    for (int m = 0; m < 4; ++m) ga[m] = A::mma(A::load(lds, kBD2 + m, lane), x, zero);
  }
  apply_mask(ga, mw0, 0);
  // density layer 1 transposed: row 4g + i of tile mm = feature i % 2 of
  // level 4 (2 mm + i / 2) + g, so lane group g gets its own levels
  floatx4 gf[MD];
#pragma unroll
  for (int mm = 0; mm < MD; ++mm) gf[mm] = zero;
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
    const float v[8] = {ga[2 * s2][0], ga[2 * s2][1], ga[2 * s2][2], ga[2 * s2][3],
                        ga[2 * s2 + 1][0], ga[2 * s2 + 1][1], ga[2 * s2 + 1][2], ga[2 * s2 + 1][3]};
    const Op x = A::pack(v, sk);
#pragma unroll
    for (int mm = 0; mm < MD; ++mm)
      gf[mm] = A::mma(A::load(lds, kBD1 + 2 * mm + s2, lane), x, gf[mm]);
  }
  // d loss / d p = sum over the lane group's levels 4j + g of d loss / d
  // feature times the stored Jacobian, then over the 4 groups.  This lane
  // group's Jacobian records of the sample (level 4j + g at record j): six
  // fp16 values d feature_q / d pos_a at 3 q + a
  const uint32_t* jp = reinterpret_cast<const uint32_t*>(w.jac) +
                       (((int64_t)(sc >> 5) * 4 + g) * (6 * LPG * 32) + (sc & 31) * 6) / 2;
  gx[0] = gx[1] = gx[2] = 0.f;
#pragma unroll
  for (int j = 0; j < LPG; ++j) {
    // level 4j + g: d loss / d pos_l = sum_q gf * J, then times N_l
    const uint32_t* rec = jp + j * (32 * 6 / 2);
    // read once: non-temporal, so that they do not displace cached data
    const uint32_t r[3] = {__builtin_nontemporal_load(rec), __builtin_nontemporal_load(rec + 1),
                           __builtin_nontemporal_load(rec + 2)};
    float J[6];
#pragma unroll
    for (int k = 0; k < 6; ++k)
      J[k] = __half2float(__ushort_as_half((unsigned short)(r[k / 2] >> (16 * (k % 2)))));
    float gl[3] = {0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const float gq = gf[j / 2][2 * (j % 2) + q];
#pragma unroll
      for (int a = 0; a < 3; ++a) gl[a] += gq * J[3 * q + a];
    }
    const float N = (float)f.res[4 * j + g];
#pragma unroll
    for (int a = 0; a < 3; ++a) gx[a] += N * gl[a];
  }
  gd[0] = gd[1] = gd[2] = 0.f;
  if (DIR) {
    const float gs[4] = {gsh[0], gsh[1], gsh[2], gsh[3]};
    sh4_vjp(d, g, gs, gd);
  }
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    gx[a] += __shfl_xor(gx[a], 16);
    gx[a] += __shfl_xor(gx[a], 32);
    gx[a] *= f.inv_ext[a] * unscale;  // d pos / d p = N_l / extent (N_l applied above)
    gd[a] += __shfl_xor(gd[a], 16);
    gd[a] += __shfl_xor(gd[a], 32);
    gd[a] *= unscale;
  }
}

// The backward kernel of the separate-kernel path: one 16-sample column tile
// per wavefront, reading d loss / d h_0 and d loss / d z from the composite
// kernel, and storing each sample's torque and force terms for the
// reduction.  DIR: the SH direction path (sh_dir_grad) is on; without it the
// SH rows of colour layer 1 are not staged, and four blocks fit a CU's LDS.
template <int LPG, bool DIR, bool H>
__global__ __launch_bounds__(kBlock) void k_mlp_bwd(DevField f, DevBatch b, DevWork w) {
  static_assert(kBwdNT == 1, "one column tile per wavefront");
  using A = Arith<H>;
  constexpr int NU = DIR ? kBwdUnits : kBSH;  // staged weight units
  __shared__ typename A::Unit lds[NU];
  __shared__ float s_c3[64 * 3];
  stage(lds, A::bwd(f), NU, A::kWords);
  for (int i = threadIdx.x; i < 64 * 3; i += kBlock) s_c3[i] = f.wc3[i];
  __syncthreads();

  const int S = *w.total;
  const int n_tiles = (S + 15) / 16;
  const int lane = threadIdx.x & 63, g = lane >> 4, col = lane & 15;
  const int wave = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  const int n_waves = gridDim.x * (kBlock / 64);
  const SplitK sk = split_k(f);

  for (int tile = wave; tile < n_tiles; tile += n_waves) {
    // the weight units are re-read from LDS every tile: hoisted out of the
    // loop they would pin ~150 registers and cap occupancy at 1 wave/SIMD
    asm volatile("" ::: "memory");
    const uint32_t* mw = w.masks + (size_t)tile * 2 * 64 + lane;
    // word 0: density layer 1 (base 0) and colour layer 1 (base 8); word 1:
    // colour layer 2 (base 0)
    const uint32_t mw0 = mw[0], mw1 = mw[64];
    const int s = tile * 16 + col;
    const int sc = s < S ? s : S - 1;
    const bool ok = s < S;
    const float z[3] = {ok ? w.cr[sc] : 0.0f, ok ? w.cg[sc] : 0.0f, ok ? w.cb[sc] : 0.0f};
    const float gh0 = ok ? w.sig[sc] : 0.0f;
    float d[3];
    sample_dir(w, sc, d);
    float gx[3], gd[3];
    bwd_tile<LPG, DIR, H>(f, w, lds, s_c3, sk, lane, z, gh0, mw0, mw1, sc, d, gx, gd);
    // the sample's terms: force dL/dp, torque d x (t dL/dp + dL/dd)
    if (ok && g < 2) {
      const float t = w.t[s];
      const float m[3] = {t * gx[0] + gd[0], t * gx[1] + gd[1], t * gx[2] + gd[2]};
      // lane group 0 stores the torque, group 1 the force
      float o0, o1, o2;
      if (g == 0) {
        o0 = d[1] * m[2] - d[2] * m[1];
        o1 = d[2] * m[0] - d[0] * m[2];
        o2 = d[0] * m[1] - d[1] * m[0];
      } else {
        o0 = gx[0];
        o1 = gx[1];
        o2 = gx[2];
      }
      float* out = w.feat + (int64_t)(3 * g) * w.cap;  // feature rows are free by now
      out[s] = o0;
      out[w.cap + s] = o1;
      out[2 * w.cap + s] = o2;
    }
  }
}

// The fused backward kernel: one wavefront per ray, persistent over rays.
// It composites the ray front to back and takes the loss on its pixel
// (classic volume rendering), sweeps the composite backward in 64-sample
// steps, and runs every step's samples, 16 at a time, through the backward
// networks and the encoding's Jacobian: d loss / d h_0 and d loss / d z pass
// from the composite lanes to the network columns by cross-lane reads, and the
// ray's sums M = sum_i (t_i d loss / d p_i + d loss / d d_i) and
// G = sum_i d loss / d p_i stay in registers, so that the ray's torque
// (Eq. 3) is one cross product d x M.  Each ray leaves 7 floats -- torque,
// force (Eq. 2), loss -- for the per-hypothesis reduction; no per-sample
// gradient goes to memory.  KEEP also stores every sample's d loss / d h_0,
// d loss / d z and (torque, force) terms as the separate kernels do
// (inspection).
template <int LPG, bool DIR, bool KEEP, bool H>
__global__ __launch_bounds__(kBlock) void k_ray_bwd(DevField f, DevBatch b, DevWork w) {
  using A = Arith<H>;
  constexpr int NU = DIR ? kBwdUnits : kBSH;
  __shared__ typename A::Unit lds[NU];
  __shared__ float s_c3[64 * 3];
  stage(lds, A::bwd(f), NU, A::kWords);
  for (int i = threadIdx.x; i < 64 * 3; i += kBlock) s_c3[i] = f.wc3[i];
  __syncthreads();

  const int lane = threadIdx.x & 63, g = lane >> 4, col = lane & 15;
  const int wave = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  const int n_waves = gridDim.x * (kBlock / 64);
  const SplitK sk = split_k(f);
  const float norm = 1.0f / (3.0f * (float)b.P);
  const int n_pix = b.W * b.H;

  for (int ray = wave; ray < b.n_rays; ray += n_waves) {
    const int base = w.off[ray];
    const int n = w.off[ray + 1] - base;
    const float delta = w.rdelta[ray];
    int pix = b.pix[ray];
    pix = pix < 0 ? 0 : (pix >= n_pix ? n_pix - 1 : pix);
    const float* I = b.obs + 3 * (size_t)pix;
    const float y[3] = {I[0], I[1], I[2]};

    // pass 1: colour and stop index
    float C[3] = {0.f, 0.f, 0.f};
    float carry = 0.0f;
    int n_used = n;
    for (int i0 = 0; i0 < n_used; i0 += 64) {
      float incl;
      const Chunk ch = step_chunk(f, w, base, n, i0, delta, carry, lane, incl);
      const uint64_t st = __ballot(ch.stop_here);
      int last = 63;
      if (st) {
        last = __ffsll((unsigned long long)st) - 1;
        n_used = i0 + last + 1;
      }
      const bool use = ch.live && lane <= last;
#pragma unroll
      for (int q = 0; q < 3; ++q) C[q] += wave_sum(use ? ch.w * ch.c[q] : 0.0f);
      carry = lane_value(incl, last);
      if (st) break;
    }
    const float T_end = __expf(-carry);
    float gC[3], L = 0.0f;
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      C[q] += T_end * f.bg[q];
      float gq;
      L += pixel_loss(f.loss_type, C[q], y[q], f.loss_param, gq);
      gC[q] = gq * norm;
    }

    // pass 2: the composite backward, step by step, and the networks
    const float d[3] = {w.rdx[ray], w.rdy[ray], w.rdz[ray]};
    float R[3] = {C[0], C[1], C[2]};  // colour behind the step (background included)
    float carry2 = 0.0f;
    float M[3] = {0.f, 0.f, 0.f}, G[3] = {0.f, 0.f, 0.f};  // this column's share of the sums
    for (int i0 = 0; i0 < n_used; i0 += 64) {
      float incl;
      const Chunk ch = step_chunk(f, w, base, n, i0, delta, carry2, lane, incl);
      const int i = i0 + lane;
      const bool use = ch.live && i < n_used;
      float gs = 0.0f, gz[3];
#pragma unroll
      for (int q = 0; q < 3; ++q) {
        const float wc = use ? ch.w * ch.c[q] : 0.0f;
        const float p = wave_incl_scan(wc);
        const float S = R[q] - p;  // colour behind sample i
        R[q] -= lane_value(p, 63);
        gs += gC[q] * (ch.T_out * ch.c[q] - S);
        gz[q] = use ? ch.w * gC[q] * ch.c[q] * (1.0f - ch.c[q]) : 0.0f;
      }
      carry2 = lane_value(incl, 63);
      const float gh0 = use ? delta * gs * ch.sig : 0.0f;
      if (KEEP && i < n) {
        w.sig[base + i] = gh0;
        w.cr[base + i] = gz[0];
        w.cg[base + i] = gz[1];
        w.cb[base + i] = gz[2];
      }
      // the step's samples through the networks, 16 columns at a time
      const int n_step = min(64, n_used - i0);
      for (int c0 = 0; c0 < n_step; c0 += 16) {
        // the weight units are re-read from LDS every tile (see k_mlp_bwd)
        asm volatile("" ::: "memory");
        const int src = c0 + col;  // composite lane of this column's sample
        const bool ok = src < n_step;
        const int s = base + i0 + (ok ? src : 0);
        // lanes past the ray's used samples hold zero gradients
        const float z[3] = {__shfl(gz[0], src), __shfl(gz[1], src), __shfl(gz[2], src)};
        const float gh = __shfl(gh0, src);
        // the sample's mask words, where the forward kernel's column tile of
        // 16 compacted samples left them for this lane group
        const uint32_t* mw = w.masks + (size_t)(s >> 4) * 2 * 64 + 16 * g + (s & 15);
        float gx[3], gd[3];
        bwd_tile<LPG, DIR, H>(f, w, lds, s_c3, sk, lane, z, gh, mw[0], mw[64], s, d, gx, gd);
        const float t = w.t[s];
        if (ok) {
#pragma unroll
          for (int a = 0; a < 3; ++a) {
            M[a] += t * gx[a] + gd[a];
            G[a] += gx[a];
          }
        }
        if (KEEP && ok && g < 2) {
          const float m[3] = {t * gx[0] + gd[0], t * gx[1] + gd[1], t * gx[2] + gd[2]};
          const float o[3] = {g == 0 ? d[1] * m[2] - d[2] * m[1] : gx[0],
                              g == 0 ? d[2] * m[0] - d[0] * m[2] : gx[1],
                              g == 0 ? d[0] * m[1] - d[1] * m[0] : gx[2]};
          float* out = w.feat + (int64_t)(3 * g) * w.cap;
#pragma unroll
          for (int a = 0; a < 3; ++a) out[a * w.cap + s] = o[a];
        }
      }
    }
    if (KEEP) {  // samples after the stop: zero gradient
      for (int i = n_used + lane; i < n; i += 64) {
        w.sig[base + i] = 0.0f;
        w.cr[base + i] = 0.0f;
        w.cg[base + i] = 0.0f;
        w.cb[base + i] = 0.0f;
#pragma unroll
        for (int q = 0; q < 6; ++q) w.feat[(int64_t)q * w.cap + base + i] = 0.0f;
      }
    }
    // the ray's sums over the 16 columns (fixed butterfly), then the torque
#pragma unroll
    for (int a = 0; a < 3; ++a) {
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        M[a] += __shfl_xor(M[a], o);
        G[a] += __shfl_xor(G[a], o);
      }
    }
    const float tq[3] = {d[1] * M[2] - d[2] * M[1], d[2] * M[0] - d[0] * M[2],
                         d[0] * M[1] - d[1] * M[0]};
    const float v = lane == 0 ? tq[0] : lane == 1 ? tq[1] : lane == 2 ? tq[2]
                  : lane == 3 ? G[0]  : lane == 4 ? G[1]  : lane == 5 ? G[2] : L * norm;
    if (lane < 7) w.ray_terms[(int64_t)7 * ray + lane] = v;
  }
}

}  // namespace

namespace {
// Resident blocks per CU of a kernel (1 if the query fails).
template <class K>
int blocks_per_cu(K kernel) {
  int n = 0;
  const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kBlock, 0);
  return e == hipSuccess && n > 0 ? n : 1;
}

template <bool H>
int fwd_per_cu(int lpg) {
  switch (lpg) {
    case 1: return blocks_per_cu(k_mlp_fwd<1, true, H>);
    case 2: return blocks_per_cu(k_mlp_fwd<2, true, H>);
    case 3: return blocks_per_cu(k_mlp_fwd<3, true, H>);
    default: return blocks_per_cu(k_mlp_fwd<4, true, H>);
  }
}

template <bool DIR, bool H>
int bwd_per_cu(int lpg) {
  switch (lpg) {
    case 1: return blocks_per_cu(k_mlp_bwd<1, DIR, H>);
    case 2: return blocks_per_cu(k_mlp_bwd<2, DIR, H>);
    case 3: return blocks_per_cu(k_mlp_bwd<3, DIR, H>);
    default: return blocks_per_cu(k_mlp_bwd<4, DIR, H>);
  }
}

template <bool DIR, bool H>
int ray_per_cu(int lpg) {
  switch (lpg) {
    case 1: return blocks_per_cu(k_ray_bwd<1, DIR, false, H>);
    case 2: return blocks_per_cu(k_ray_bwd<2, DIR, false, H>);
    case 3: return blocks_per_cu(k_ray_bwd<3, DIR, false, H>);
    default: return blocks_per_cu(k_ray_bwd<4, DIR, false, H>);
  }
}
}  // namespace

int mlp_fwd_blocks_per_cu(int lpg, int f16) {
  return f16 ? fwd_per_cu<true>(lpg) : fwd_per_cu<false>(lpg);
}

int mlp_bwd_blocks_per_cu(int lpg, int sh_dir_grad, int f16) {
  if (sh_dir_grad) return f16 ? bwd_per_cu<true, true>(lpg) : bwd_per_cu<true, false>(lpg);
  return f16 ? bwd_per_cu<false, true>(lpg) : bwd_per_cu<false, false>(lpg);
}

int ray_bwd_blocks_per_cu(int lpg, int sh_dir_grad, int f16) {
  if (sh_dir_grad) return f16 ? ray_per_cu<true, true>(lpg) : ray_per_cu<true, false>(lpg);
  return f16 ? ray_per_cu<false, true>(lpg) : ray_per_cu<false, false>(lpg);
}

namespace {
template <bool GRAD, bool H>
void launch_fwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                hipStream_t s) {
  switch (f.lpg) {
    case 1: hipLaunchKernelGGL((k_mlp_fwd<1, GRAD, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 2: hipLaunchKernelGGL((k_mlp_fwd<2, GRAD, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 3: hipLaunchKernelGGL((k_mlp_fwd<3, GRAD, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 4: hipLaunchKernelGGL((k_mlp_fwd<4, GRAD, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
  }
}

template <bool DIR, bool H>
hipError_t launch_bwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                      hipStream_t s) {
  switch (f.lpg) {
    case 1: hipLaunchKernelGGL((k_mlp_bwd<1, DIR, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 2: hipLaunchKernelGGL((k_mlp_bwd<2, DIR, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 3: hipLaunchKernelGGL((k_mlp_bwd<3, DIR, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 4: hipLaunchKernelGGL((k_mlp_bwd<4, DIR, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <bool DIR, bool KEEP, bool H>
hipError_t launch_ray(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                      hipStream_t s) {
  switch (f.lpg) {
    case 1: hipLaunchKernelGGL((k_ray_bwd<1, DIR, KEEP, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 2: hipLaunchKernelGGL((k_ray_bwd<2, DIR, KEEP, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 3: hipLaunchKernelGGL((k_ray_bwd<3, DIR, KEEP, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    case 4: hipLaunchKernelGGL((k_ray_bwd<4, DIR, KEEP, H>), dim3(n_blocks), dim3(kBlock), 0, s, f, b, w); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <bool H>
hipError_t launch_ray_h(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                        int keep, hipStream_t s) {
  if (f.sh_dir_grad)
    return keep ? launch_ray<true, true, H>(f, b, w, n_blocks, s)
                : launch_ray<true, false, H>(f, b, w, n_blocks, s);
  return keep ? launch_ray<false, true, H>(f, b, w, n_blocks, s)
              : launch_ray<false, false, H>(f, b, w, n_blocks, s);
}
}  // namespace

hipError_t launch_mlp_fwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                          int with_grad, hipStream_t s) {
  if (f.lpg < 1 || f.lpg > 4) return hipErrorInvalidValue;
  if (f.mlp_f16) {
    if (with_grad)
      launch_fwd<true, true>(f, b, w, n_blocks, s);
    else
      launch_fwd<false, true>(f, b, w, n_blocks, s);
  } else {
    if (with_grad)
      launch_fwd<true, false>(f, b, w, n_blocks, s);
    else
      launch_fwd<false, false>(f, b, w, n_blocks, s);
  }
  return hipGetLastError();
}

hipError_t launch_mlp_bwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                          hipStream_t s) {
  if (f.mlp_f16)
    return f.sh_dir_grad ? launch_bwd<true, true>(f, b, w, n_blocks, s)
                         : launch_bwd<false, true>(f, b, w, n_blocks, s);
  return f.sh_dir_grad ? launch_bwd<true, false>(f, b, w, n_blocks, s)
                       : launch_bwd<false, false>(f, b, w, n_blocks, s);
}

hipError_t launch_ray_bwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                          int keep, hipStream_t s) {
  // no more workgroups than the rays need (8 rays each)
  const int need = (b.n_rays + kBlock / 64 - 1) / (kBlock / 64);
  n_blocks = std::max(1, std::min(n_blocks, need));
  return f.mlp_f16 ? launch_ray_h<true>(f, b, w, n_blocks, keep, s)
                   : launch_ray_h<false>(f, b, w, n_blocks, keep, s);
}

}  // namespace pnerf
