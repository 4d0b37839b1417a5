// Multiresolution hash encoding of the samples (Sec. III, Instant NGP): the
// gather of every level's 8 vertex features, their trilinear blend, and the
// blend's derivative with respect to the sample position (the table is frozen,
// so the backward pass needs nothing else from it: the MLP backward kernel
// contracts this Jacobian with d loss / d feature, and nothing is re-gathered
// or scattered).
//
// Work split: one level at a time per work item (see k_encode): every XCD
// (own 4 MB L2) works on one level table at a time, its home levels first.
//
// Two adjacent lanes handle one sample: lane side 0 gathers the four vertices
// at the cell's lower x, side 1 the four at x + 1.  The two x neighbours of a
// vertex nearly always share a cache line: a dense level stores them side by
// side, and the spatial hash (x ^ y' ^ z') of x and x + 1 differs only in the
// bits that the carry of x + 1 flips, the lowest bit for even x.  Each gather
// instruction so touches about half as many lines as with one lane per sample,
// and the gather's cost follows the lines, not the instructions.  Each lane
// blends its half; one lane-pair exchange completes the sums.
//
// Features are stored SoA, row p = (l % 4) * 2 LPG + (l / 4) * 2 + q for
// feature q of level l (the order in which the MLP kernels feed them to MFMA),
// row stride = the workspace sample capacity.  The Jacobian d feature /
// d pos of every level (pos = x N_l: bounded by the table's value
// differences, zero along clamped components) is stored in fp16 (rounding
// below 2^-11 of each entry), as one 12-byte record per sample and level (the
// six values d feature_q / d pos_a at 3 q + a), grouped in blocks of 32
// samples: block b, lane group g = l % 4, level l / 4 of the group, sample
// s % 32, at ((4 b + g) LPG 32 + (l / 4) 32 + s % 32) 6 halves.  The MLP
// backward kernel reads each of its samples' records of a lane group with one
// 12-byte load per level, and the 32 records of one level and block fill 3
// whole cache lines, so no line is written from two XCDs.  That kernel applies
// N_l and 1 / extent in fp32.
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

// The position held by lane ODD of each lane pair, in both lanes of the pair
// (DPP quad_perm [0,0,2,2] or [1,1,3,3]; all lanes active).
template <int ODD>
__device__ __forceinline__ float from_pair_lane(float v) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(v), ODD ? 0xF5 : 0xA0, 0xF, 0xF, false));
}

template <int ODD>
__device__ __forceinline__ Pos pos_from_pair_lane(const Pos& p) {
  auto bc = from_pair_lane<ODD>;
  Pos r;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    r.x[a] = bc(p.x[a]);
    r.dx[a] = bc(p.dx[a]);
  }
  r.clamped = (uint32_t)__float_as_int(bc(__int_as_float((int)p.clamped)));
  return r;
}

// Cell of one level: lower corner, interpolation weights, and the table index
// of corner k (bit 0: x + 1, bit 1: y + 1, bit 2: z + 1).
struct Cell {
  float w[3];
  uint32_t i0[3];
};

// The cell comes from the float product x N (as a reference implementation in
// float decides it); the weights add back that product's rounding error and
// N dx, the part of the position float cannot hold.
__device__ __forceinline__ void make_cell(const DevField& f, int l, const float x[3],
                                          const float dx[3], Cell& c) {
  const int N = f.res[l];
  const float Nf = (float)N;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    float pos = __fmul_rn(x[a], Nf);
    int ci = (int)pos;
    ci = ci < N - 1 ? ci : N - 1;
    c.i0[a] = (uint32_t)ci;
    c.w[a] = (__fsub_rn(pos, (float)ci) + fmaf(x[a], Nf, -pos)) + Nf * dx[a];
  }
}

// KIND: 0 the level's kind read from the field, 1 dense, 2 hashed.
template <int KIND>
__device__ __forceinline__ uint32_t corner_index(const DevField& f, int l, const Cell& c, int k) {
  const bool dense = KIND == 0 ? f.dense[l] != 0 : KIND == 1;
  const uint32_t n1 = f.n1[l];
  const uint32_t sy = dense ? n1 : kPrime1;
  const uint32_t sz = dense ? n1 * n1 : kPrime2;
  const uint32_t xi = c.i0[0] + (k & 1);
  const uint32_t yi = (c.i0[1] + ((k >> 1) & 1)) * sy;
  const uint32_t zi = (c.i0[2] + ((k >> 2) & 1)) * sz;
  const uint32_t h = dense ? (xi + yi + zi) : ((xi ^ yi ^ zi) & (f.T - 1u));
  return (uint32_t)l * f.T + h;
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
  for (int k = 0; k < 8; ++k) v[k] = vertex<F16>(f, corner_index<0>(f, l, c, k));
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

// One lane's half of level l: the four corners with x offset `side`, blended
// with that side's x weight.  p = (feature_0, feature_1, then when GRAD the
// half of d feature_q / d pos_a at 2 + 3 q + a).  The halves of the two lanes
// of a pair add up to the whole cell's values.  KIND: see corner_index.
template <bool F16, bool GRAD, int KIND>
__device__ __forceinline__ void half_cell(const DevField& f, int l, const float x[3],
                                          const float dx[3], int side, float p[8]) {
  Cell c;
  make_cell(f, l, x, dx, c);
  float2 v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = vertex<F16>(f, corner_index<KIND>(f, l, c, 2 * j + side));
  const float wx = c.w[0], wy = c.w[1], wz = c.w[2];
  const float ux = 1.0f - wx, uy = 1.0f - wy, uz = 1.0f - wz;
  const float sx = side ? wx : ux;       // this side's x weight
  const float sgn = side ? 1.0f : -1.0f; // its derivative along x
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    float t[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) t[j] = q ? v[j].y : v[j].x;
    // corners j: bit 0 = y + 1, bit 1 = z + 1
    const float ty0 = uz * t[0] + wz * t[2], ty1 = uz * t[1] + wz * t[3];
    p[q] = sx * (uy * ty0 + wy * ty1);
    if (GRAD) {
      p[2 + 3 * q + 0] = sgn * (uy * ty0 + wy * ty1);
      p[2 + 3 * q + 1] = sx * (ty1 - ty0);
      p[2 + 3 * q + 2] = sx * (uy * (t[2] - t[0]) + wy * (t[3] - t[1]));
    }
  }
}

__device__ __forceinline__ int feat_row(const DevField& f, int l, int q) {
  return (l & 3) * 2 * f.lpg + (l >> 2) * 2 + q;
}

// Index (in 32-bit words) of the Jacobian record of level l and sample s: six
// fp16 values d feature_q / d pos_a at 3 q + a, three words.
__device__ __forceinline__ int64_t jac_record(const DevField& f, int l, int64_t s) {
  const int kg = 6 * f.lpg * 32;  // halves of one lane group's share of a 32-sample block
  return (((s >> 5) * 4 + (l & 3)) * (int64_t)kg + ((l >> 2) * 32 + (s & 31)) * 6) / 2;
}

__device__ __forceinline__ uint32_t pack_half2(float lo, float hi) {
  return (uint32_t)__half_as_ushort(__float2half_rn(lo)) |
         ((uint32_t)__half_as_ushort(__float2half_rn(hi)) << 16);
}

// ------------------------------------------------------------------ forward
// Work items: kItem consecutive samples of one level, taken from that level's
// queue (a counter of the items handed out) by one atomic per block.  Queue q
// serves level q_level[q], hashed levels first.  Workgroups are dispatched
// round-robin over the XCDs, so block b runs on XCD b % 8: it starts on its
// home queues x, x + 8, ... (x = b % 8), one level at a time, so that each
// XCD's L2 holds one level table at a time, and once those are drained it
// takes what is left on every other queue in turn.  No XCD idles while
// another still has work, and blocks that find no free slot at launch and
// start late only take what is left.  The next item is claimed before the
// current one is gathered, hiding the atomic's latency.
constexpr int kXcds = 8;
constexpr int kPerPair = 4;                      // samples per lane pair and item
constexpr int kItem = kBlock / 2 * kPerPair;     // samples per work item
static_assert((kBlock / 2) % 32 == 0, "a lane-pair step must span whole 32-sample Jacobian blocks");

__device__ __forceinline__ uint32_t take_item(uint32_t* queue, int q) {
  return __hip_atomic_fetch_add(queue + q * kQueueStride, 1u, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
}

// A lane pair's share of level l for the sample at ps: lane side q keeps
// feature q and its Jacobian row, adding the partner's half of those to its
// own, and hands over its half of the other feature; it stores feature q at fo
// (the sample's entry of feature row q).  GRAD: lane side 0 also takes the
// partner's Jacobian row and stores the sample's whole record at jr.  Outputs
// are streamed out with non-temporal stores so that they do not displace the
// level tables from L2.
template <bool F16, bool GRAD, int KIND>
__device__ __forceinline__ void encode_level(const DevField& f, int l, const Pos& ps, int side,
                                             float* fo, uint32_t* jr) {
  float p[8];
  half_cell<F16, GRAD, KIND>(f, l, ps.x, ps.dx, side, p);
  const float keep = side ? p[1] : p[0];
  const float give = side ? p[0] : p[1];
  __builtin_nontemporal_store(keep + lane_pair_swap(give), fo);
  if (GRAD) {
    float v[3], o[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      const float jk = side ? p[5 + a] : p[2 + a];
      const float jg = side ? p[2 + a] : p[5 + a];
      v[a] = jk + lane_pair_swap(jg);
      v[a] = (ps.clamped >> a) & 1u ? 0.0f : v[a];
    }
#pragma unroll
    for (int a = 0; a < 3; ++a) o[a] = lane_pair_swap(v[a]);  // side 0: feature 1's row
    if (side == 0) {
      __builtin_nontemporal_store(pack_half2(v[0], v[1]), jr);
      __builtin_nontemporal_store(pack_half2(v[2], o[0]), jr + 1);
      __builtin_nontemporal_store(pack_half2(o[1], o[2]), jr + 2);
    }
  }
}

template <bool F16, bool GRAD>
__global__ __launch_bounds__(kBlock) void k_encode(DevField f, DevBatch b, DevWork w) {
  __shared__ uint32_t s_item[2];
  const int S = *w.total;
  const uint32_t n_items = (uint32_t)((S + kItem - 1) / kItem);
  const int NQ = f.L;
  const int side = threadIdx.x & 1;
  const int home = (int)(blockIdx.x % kXcds) < NQ ? (int)(blockIdx.x % kXcds) : (int)(blockIdx.x % NQ);
  int q = home;
  int visit = 0;  // 0: on the home queues; v > 0: on queue (home + v) % NQ
  int buf = 0;
  if (threadIdx.x == 0) s_item[buf] = take_item(w.queue, q);
  __syncthreads();
  uint32_t item = s_item[buf];
  // control flow below is uniform over the block: item, q and visit follow
  // from the same shared words for every thread
  while (true) {
    if (item >= n_items) {  // queue q is drained: the next home queue, else the others in turn
      if (visit == 0 && q + kXcds < NQ) {
        q += kXcds;
      } else {
        if (visit == NQ) break;
        ++visit;
        q = (home + visit) % NQ;
      }
      buf ^= 1;
      if (threadIdx.x == 0) s_item[buf] = take_item(w.queue, q);
      __syncthreads();
      item = s_item[buf];
      continue;
    }
    uint32_t next = 0;
    if (threadIdx.x == 0) next = take_item(w.queue, q);
    const int l = f.q_level[q];
    // the pair's kPerPair samples s0 + j kBlock / 2.  The bounds test makes each
    // sample a block of code of its own, so a wavefront gathers its samples one
    // after the other (4 loads in flight) and the 7-8 resident wavefronts per
    // SIMD overlap each other's waits; issuing all 16 loads at once doubles the
    // registers, halves the resident wavefronts and is slower, since the CU's
    // L1 already holds as many L2 misses in flight as it can.  Positions: lane
    // side computes samples 2 k + side and both lanes take each from the lane
    // that computed it (all lanes active); an odd last one both lanes compute.
    const int s0 = (int)item * kItem + (threadIdx.x >> 1);
    Pos ps[kPerPair];
#pragma unroll
    for (int k = 0; k < kPerPair / 2; ++k) {
      const int sm = s0 + (2 * k + side) * (kBlock / 2);
      const Pos mine = sample_pos(f, b, w, sm < S ? sm : S - 1);
      ps[2 * k] = pos_from_pair_lane<0>(mine);
      ps[2 * k + 1] = pos_from_pair_lane<1>(mine);
    }
    if (kPerPair & 1) {
      const int sl = s0 + (kPerPair - 1) * (kBlock / 2);
      ps[kPerPair - 1] = sample_pos(f, b, w, sl < S ? sl : S - 1);
    }
    // output entries of sample s0; sample j is kBlock / 2 entries further along
    // the feature row and kBlock / 64 Jacobian blocks further (kBlock / 2 is a
    // multiple of 32)
    float* fo = w.feat + (int64_t)feat_row(f, l, side) * w.cap + s0;
    uint32_t* jo = reinterpret_cast<uint32_t*>(w.jac) + jac_record(f, l, s0);
    const int64_t jstep = (int64_t)(kBlock / 64) * 4 * (6 * f.lpg * 32) / 2;  // words
    // the level's kind is uniform over the item: one branch, no per-lane selects
    if (f.dense[l]) {
#pragma unroll
      for (int j = 0; j < kPerPair; ++j)  // pairs leave together
        if (s0 + j * (kBlock / 2) < S)
          encode_level<F16, GRAD, 1>(f, l, ps[j], side, fo + j * (kBlock / 2), jo + j * jstep);
    } else {
#pragma unroll
      for (int j = 0; j < kPerPair; ++j)
        if (s0 + j * (kBlock / 2) < S)
          encode_level<F16, GRAD, 2>(f, l, ps[j], side, fo + j * (kBlock / 2), jo + j * jstep);
    }
    buf ^= 1;
    if (threadIdx.x == 0) s_item[buf] = next;
    __syncthreads();
    item = s_item[buf];
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
  // per_cu blocks of 256 threads per CU (the work queues balance whatever is
  // resident)
  (void)f;
  return n_cu * per_cu;
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
