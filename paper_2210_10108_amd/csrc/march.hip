// Ray generation, box clipping, sample placement with occupancy skipping, and
// deterministic compaction (count -> scan -> write) into SoA sample buffers.
//
// Every floating-point step that decides an integer (which samples exist, their
// distance t, the occupancy cell) is written as separate IEEE round-to-nearest
// operations (__fadd_rn, __fmul_rn, __fdiv_rn, sqrtf; the library is built with
// -ffp-contract=on and correctly rounded division and square root, so none of
// them is fused), and the sample set is reproducible bit for bit by any
// implementation following the same operation order.
#include "pnerf_internal.h"

namespace pnerf {
namespace {

constexpr int kRayBlock = 256;     // 4 wavefronts
constexpr int kRaysPerWave = 4;    // rays marched by one wavefront
constexpr int kScanBlock = 256;    // rays per block of the offset scan

struct RayGeom {
  float o[3], d[3], tn, tf, delta;
  float de[3];  // exact direction minus d (for compensated sample positions)
  int hit;
};

// Pixel -> ray (Sec. IV-A: the ray origin is the camera centre) and its
// clip against the scene box.
__device__ inline RayGeom make_ray(const DevField& f, const DevBatch& b, int ray) {
  RayGeom g;
  const float* pose = b.poses + 12 * (ray / b.P);
  int pix = b.pix[ray];
  const int n_pix = b.W * b.H;
  pix = pix < 0 ? 0 : (pix >= n_pix ? n_pix - 1 : pix);  // out-of-range ids are clamped
  int u = pix % b.W, v = pix / b.W;
  float xc = __fdiv_rn(__fsub_rn(__fadd_rn((float)u, 0.5f), b.cx), b.fx);
  float yc = __fdiv_rn(__fsub_rn(__fadd_rn((float)v, 0.5f), b.cy), b.fy);
  float dw[3];
  for (int a = 0; a < 3; ++a) {
    dw[a] = __fadd_rn(__fadd_rn(__fmul_rn(pose[4 * a], xc), __fmul_rn(pose[4 * a + 1], yc)),
                      pose[4 * a + 2]);
    g.o[a] = pose[4 * a + 3];
  }
  float n = sqrtf(__fadd_rn(__fadd_rn(__fmul_rn(dw[0], dw[0]), __fmul_rn(dw[1], dw[1])),
                                 __fmul_rn(dw[2], dw[2])));
  for (int a = 0; a < 3; ++a) g.d[a] = __fdiv_rn(dw[a], n);
  {
    // the same direction in double: its difference from d lets the shading
    // kernels place samples more precisely than float allows (decisions above
    // stay on the float values)
    double xd = ((double)u + 0.5 - (double)b.cx) / (double)b.fx;
    double yd = ((double)v + 0.5 - (double)b.cy) / (double)b.fy;
    double e[3], nn = 0.0;
    for (int a = 0; a < 3; ++a) {
      e[a] = (double)pose[4 * a] * xd + (double)pose[4 * a + 1] * yd + (double)pose[4 * a + 2];
      nn += e[a] * e[a];
    }
    nn = sqrt(nn);
    for (int a = 0; a < 3; ++a) g.de[a] = (float)(e[a] / nn - (double)g.d[a]);
  }
  float t_entry = -INFINITY, t_exit = INFINITY;
  bool empty = false;
  for (int a = 0; a < 3; ++a) {
    if (g.d[a] != 0.0f) {
      float t1 = __fdiv_rn(__fsub_rn(f.mn[a], g.o[a]), g.d[a]);
      float t2 = __fdiv_rn(__fsub_rn(f.mx[a], g.o[a]), g.d[a]);
      float lo = t1 < t2 ? t1 : t2, hi = t1 < t2 ? t2 : t1;
      if (lo > t_entry) t_entry = lo;
      if (hi < t_exit) t_exit = hi;
    } else if (g.o[a] < f.mn[a] || g.o[a] > f.mx[a]) {
      empty = true;
    }
  }
  if (empty) {
    g.tn = 0.0f;
    g.tf = 0.0f;
    g.hit = 0;
  } else {
    g.tn = t_entry > 0.0f ? t_entry : 0.0f;
    g.tf = t_exit;
    g.hit = g.tf > g.tn;
  }
  if (f.march_mode == 0)
    g.delta = g.hit ? __fdiv_rn(__fsub_rn(g.tf, g.tn), (float)f.n_uniform) : 0.0f;
  else
    g.delta = f.step;
  return g;
}

__device__ inline float sample_t(const DevField& f, float tn, float delta, int j) {
  float s = f.march_mode == 0 ? delta : f.step;
  return __fadd_rn(tn, __fmul_rn(__fadd_rn((float)j, 0.5f), s));
}

__device__ inline bool occupied(const DevField& f, const float o[3], const float d[3], float t) {
  if (f.occ_res <= 0) return true;
  int R = f.occ_res;
  uint32_t c[3];
  for (int a = 0; a < 3; ++a) {
    float p = __fadd_rn(o[a], __fmul_rn(t, d[a]));
    float ext = __fsub_rn(f.mx[a], f.mn[a]);
    float sc = __fdiv_rn((float)R, ext);
    float q = __fmul_rn(__fsub_rn(p, f.mn[a]), sc);
    int ci = !(q >= 0.0f) ? 0 : (q >= (float)R ? R - 1 : (int)q);  // NaN -> cell 0
    c[a] = (uint32_t)ci;
  }
  uint64_t idx = (uint64_t)c[0] + (uint64_t)R * ((uint64_t)c[1] + (uint64_t)R * c[2]);
  return (f.occ[idx >> 5] >> (idx & 31u)) & 1u;
}

// One wavefront marches one ray, 64 candidate samples per step: each lane
// tests one candidate, a ballot compacts the kept ones in order.
template <bool EMIT>
__device__ inline int march_wave(const DevField& f, const RayGeom& g, int lane, int cap,
                                 float* t_out, int32_t* j_out, int32_t* ray_out, int ray) {
  if (!g.hit) return 0;
  int kept = 0;
  int limit = f.march_mode == 0 ? f.n_uniform : f.max_samples;
  if (limit > cap) limit = cap;
  for (int j0 = 0;; j0 += 64) {
    int j = j0 + lane;
    float t = sample_t(f, g.tn, g.delta, j);
    bool valid = f.march_mode == 0 ? (j < f.n_uniform) : (t < g.tf);
    bool occ = valid && occupied(f, g.o, g.d, t);
    uint64_t bal = __ballot(occ);
    int rank = __popcll(bal & ((1ull << lane) - 1ull));
    if (EMIT && occ && kept + rank < limit) {
      t_out[kept + rank] = t;
      if (j_out) j_out[kept + rank] = j;
      ray_out[kept + rank] = ray;
    }
    int n = __popcll(bal);
    kept = kept + n < limit ? kept + n : limit;
    bool last_valid = __shfl(valid ? 1 : 0, 63) != 0;
    if (kept >= limit || !last_valid || j0 + 64 >= kMaxLatticeCandidates + 64) break;
  }
  return kept;
}

// Exclusive scan of one value per thread over a block of kScanBlock threads
// (shuffles within each wavefront, the wavefront totals in LDS, fixed order);
// returns the thread's exclusive prefix and sets *block_total.
__device__ inline int block_exclusive_scan(int c, int* s_wave, int* block_total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int inc = c;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int x = __shfl_up(inc, d);
    if (lane >= d) inc += x;
  }
  if (lane == 63) s_wave[wv] = inc;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int v = 0; v < kScanBlock / 64; ++v) {
    const int x = s_wave[v];
    before += v < wv ? x : 0;
    total += x;
  }
  *block_total = total;
  return before + inc - c;
}

// One thread per ray: ray generation and box clip, stored for the kernels
// that follow (their float values decide the samples, so they are computed
// once), and the SH basis of the ray's direction for the colour network.  Without an occupancy grid a uniform-mode ray keeps all its
// candidates, so its count is known here; SCAN then also takes the first
// level of the offset scan (as k_scan_local does).
template <bool SCAN>
__global__ __launch_bounds__(kRayBlock) void k_ray_setup(DevField f, DevBatch b, DevWork w) {
  static_assert(!SCAN || kRayBlock == kScanBlock, "one scan block per workgroup");
  const int ray = blockIdx.x * kRayBlock + threadIdx.x;
  int c = 0;
  if (ray < b.n_rays) {
    const RayGeom g = make_ray(f, b, ray);
    w.rdx[ray] = g.d[0];
    w.rdy[ray] = g.d[1];
    w.rdz[ray] = g.d[2];
    w.rex[ray] = g.de[0];
    w.rey[ray] = g.de[1];
    w.rez[ray] = g.de[2];
    float sh[16];
    sh16(g.d, sh);
    float4* o = reinterpret_cast<float4*>(w.rsh + (size_t)16 * ray);
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = make_float4(sh[4 * q], sh[4 * q + 1], sh[4 * q + 2], sh[4 * q + 3]);
    w.rtn[ray] = g.tn;
    w.rtf[ray] = g.tf;
    w.rdelta[ray] = g.delta;
    if (SCAN) {
      c = g.hit ? (f.n_uniform < f.max_per_ray ? f.n_uniform : f.max_per_ray) : 0;
      w.count[ray] = c;
    }
  }
  if (SCAN) {
    __shared__ int s_wave[kScanBlock / 64];
    int total;
    const int e = block_exclusive_scan(c, s_wave, &total);
    if (ray < b.n_rays) w.off[ray] = e;
    if (threadIdx.x == 0) w.blocksum[blockIdx.x] = total;
  }
}

// The stored geometry of a ray (hit = the clip left an interval).
__device__ inline RayGeom stored_ray(const DevBatch& b, const DevWork& w, int ray) {
  RayGeom g;
  const float* pose = b.poses + 12 * (ray / b.P);
  g.o[0] = pose[3];
  g.o[1] = pose[7];
  g.o[2] = pose[11];
  g.d[0] = w.rdx[ray];
  g.d[1] = w.rdy[ray];
  g.d[2] = w.rdz[ray];
  g.tn = w.rtn[ray];
  g.tf = w.rtf[ray];
  g.delta = w.rdelta[ray];
  g.hit = g.tf > g.tn;
  return g;
}

// Rays of one wavefront: kRaysPerWave consecutive rays, marched one after the
// other with all 64 lanes testing candidates; lane 0 stores the ray's count.
// (Not launched when k_ray_setup already knows the counts.)
__global__ __launch_bounds__(kRayBlock) void k_ray_count(DevField f, DevBatch b, DevWork w) {
  int lane = threadIdx.x & 63;
  int wave = blockIdx.x * (kRayBlock / 64) + (threadIdx.x >> 6);
  for (int q = 0; q < kRaysPerWave; ++q) {
    int ray = wave * kRaysPerWave + q;
    if (ray >= b.n_rays) break;
    const RayGeom g = stored_ray(b, w, ray);
    int n = march_wave<false>(f, g, lane, f.max_per_ray, nullptr, nullptr, nullptr, ray);
    if (lane == 0) w.count[ray] = n;
  }
}

// Exclusive scan of the counts of each block of kScanBlock rays: off[ray] =
// offset inside the block, blocksum = the block's total.
__global__ __launch_bounds__(kScanBlock) void k_scan_local(DevBatch b, DevWork w) {
  __shared__ int s_wave[kScanBlock / 64];
  const int ray = blockIdx.x * kScanBlock + threadIdx.x;
  const int c = ray < b.n_rays ? w.count[ray] : 0;
  int total;
  const int e = block_exclusive_scan(c, s_wave, &total);
  if (ray < b.n_rays) w.off[ray] = e;
  if (threadIdx.x == 0) w.blocksum[blockIdx.x] = total;
}

// Second level, in one workgroup: exclusive scan of the block totals
// (n_blocks <= kMaxScanBlocks, kPer per thread; shuffles within wavefronts,
// the wavefront totals in LDS), the batch's sample total, and the samples of
// every hypothesis -- the difference of the exclusive offsets at its first
// ray and past its last -- which the host reads to size and plan the chunks.
__global__ __launch_bounds__(1024) void k_scan_finish(DevBatch b, DevWork w, int n_blocks) {
  constexpr int kPer = kMaxScanBlocks / 1024;
  __shared__ int s_wave[1024 / 64];
  __shared__ int s_bs[kMaxScanBlocks];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int v[kPer], acc = 0;
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int i = tid * kPer + q;
    v[q] = i < n_blocks ? w.blocksum[i] : 0;
    acc += v[q];
  }
  int inc = acc;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int x = __shfl_up(inc, d);
    if (lane >= d) inc += x;
  }
  if (lane == 63) s_wave[wv] = inc;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int u = 0; u < 1024 / 64; ++u) {
    const int x = s_wave[u];
    before += u < wv ? x : 0;
    total += x;
  }
  int run = before + inc - acc;  // exclusive prefix of this thread's blocks
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int i = tid * kPer + q;
    if (i < n_blocks) {
      w.blocksum[i] = run;
      s_bs[i] = run;
    }
    run += v[q];
  }
  if (tid == 0) *w.total = total;
  __syncthreads();
  auto excl = [&](int r) { return r < b.n_rays ? s_bs[r / kScanBlock] + w.off[r] : total; };
  for (int k = tid; k < b.K; k += 1024) w.hyp_total[k] = excl((k + 1) * b.P) - excl(k * b.P);
}

// Second march of the rays of one sample chunk (rays ray_base .. of the counted
// batch `wb`), writing their kept samples into the chunk's sample arrays at
// offset (exclusive offset in the counted batch) - sample_base, and the chunk's
// ray offsets into wc.off (wc's per-ray arrays start at the chunk's first ray).
// chunk_total < 0: the chunk is the whole counted batch, whose total the scan
// left on the device.  RAW: the scan stopped at the raw sums of its
// raw_blocks (<= 64) blocks, and every wavefront scans them itself (then the
// chunk is the whole counted batch, and block 0 also stores its total).
template <bool RAW>
__global__ __launch_bounds__(kRayBlock) void k_ray_write(DevField f, DevBatch b, DevWork wb,
                                                         DevWork wc, int ray_base,
                                                         int sample_base, int chunk_total,
                                                         int raw_blocks, int32_t* j_out) {
  int lane = threadIdx.x & 63;
  int wave = blockIdx.x * (kRayBlock / 64) + (threadIdx.x >> 6);
  int raw_excl = 0, raw_total = 0;  // RAW: lane i holds the exclusive prefix of block i
  if (RAW) {
    const int v = lane < raw_blocks ? wb.blocksum[lane] : 0;
    int inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int x = __shfl_up(inc, d);
      if (lane >= d) inc += x;
    }
    raw_excl = inc - v;
    raw_total = __shfl(inc, 63);
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const int total = RAW ? raw_total : (chunk_total >= 0 ? chunk_total : *wb.total);
    *wc.total = total;
    wc.off[b.n_rays] = total;
    if (RAW) *wb.total = total;  // the counted batch's total (read back on demand)
  }
  // the encoding of this chunk, next on the stream, starts from empty work queues
  if (blockIdx.x == 0 && threadIdx.x < kMaxLevels) wc.queue[threadIdx.x * kQueueStride] = 0u;
  // every load the wavefront's rays need is issued before the first is
  // marched (a ray past the end loads the last ray's values and is skipped);
  // each wavefront reads only its own rays' offsets, which it then overwrites
  int off[kRaysPerWave], cnt[kRaysPerWave];
  RayGeom geo[kRaysPerWave];
#pragma unroll
  for (int q = 0; q < kRaysPerWave; ++q) {
    const int ray = wave * kRaysPerWave + q;
    const int rc = ray < b.n_rays ? ray : b.n_rays - 1;
    const int rb = ray_base + rc;
    const int before = RAW ? __shfl(raw_excl, rb / kScanBlock) : wb.blocksum[rb / kScanBlock];
    off[q] = before + wb.off[rb] - sample_base;
    cnt[q] = wc.count[rc];
    geo[q] = stored_ray(b, wc, rc);
  }
#pragma unroll
  for (int q = 0; q < kRaysPerWave; ++q) {
    const int ray = wave * kRaysPerWave + q;
    if (ray >= b.n_rays) break;
    const int o = off[q], n = cnt[q];
    if (lane == 0) wc.off[ray] = o;
    if (n == 0) continue;
    march_wave<true>(f, geo[q], lane, n, wc.t + o, j_out ? j_out + o : nullptr, wc.sray + o, ray);
  }
}

}  // namespace

hipError_t launch_march_count(const DevField& f, const DevBatch& b, const DevWork& w, bool raw_ok,
                              int* raw_blocks, hipStream_t s) {
  const int n_scan = (b.n_rays + kScanBlock - 1) / kScanBlock;
  if (n_scan > kMaxScanBlocks) return hipErrorInvalidValue;
  const int n_setup = (b.n_rays + kRayBlock - 1) / kRayBlock;
  *raw_blocks = 0;
  if (f.march_mode == 0 && f.occ_res <= 0) {
    // counts known at set-up: the first scan level runs in the same kernel
    hipLaunchKernelGGL(k_ray_setup<true>, dim3(n_setup), dim3(kRayBlock), 0, s, f, b, w);
    if (raw_ok && n_scan <= kMaxRawScanBlocks) {  // the write pass scans the block sums
      *raw_blocks = n_scan;
      return hipGetLastError();
    }
  } else {
    hipLaunchKernelGGL(k_ray_setup<false>, dim3(n_setup), dim3(kRayBlock), 0, s, f, b, w);
    const int rays_per_block = kRaysPerWave * (kRayBlock / 64);
    const int n_march = (b.n_rays + rays_per_block - 1) / rays_per_block;
    hipLaunchKernelGGL(k_ray_count, dim3(n_march), dim3(kRayBlock), 0, s, f, b, w);
    hipLaunchKernelGGL(k_scan_local, dim3(n_scan), dim3(kScanBlock), 0, s, b, w);
  }
  hipLaunchKernelGGL(k_scan_finish, dim3(1), dim3(1024), 0, s, b, w, n_scan);
  return hipGetLastError();
}

hipError_t launch_march_write(const DevField& f, const DevBatch& b, const DevWork& wb,
                              const DevWork& wc, int ray_base, int sample_base, int chunk_total,
                              int raw_blocks, int32_t* lattice_j_out, hipStream_t s) {
  int rays_per_block = kRaysPerWave * (kRayBlock / 64);
  int n_march = (b.n_rays + rays_per_block - 1) / rays_per_block;
  if (raw_blocks > kMaxRawScanBlocks || (raw_blocks > 0 && (ray_base != 0 || sample_base != 0)))
    return hipErrorInvalidValue;
  if (raw_blocks > 0)
    hipLaunchKernelGGL(k_ray_write<true>, dim3(n_march), dim3(kRayBlock), 0, s, f, b, wb, wc,
                       ray_base, sample_base, chunk_total, raw_blocks, lattice_j_out);
  else
    hipLaunchKernelGGL(k_ray_write<false>, dim3(n_march), dim3(kRayBlock), 0, s, f, b, wb, wc,
                       ray_base, sample_base, chunk_total, 0, lattice_j_out);
  return hipGetLastError();
}

__global__ void k_offsets_i64(const int32_t* off, int64_t* out, int n, int64_t base) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = base + off[i];
}

// Copy t and lattice index of n samples.
__global__ void k_copy_samples(const float* t, const int32_t* j, float* t_out, int32_t* j_out,
                               int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    t_out[i] = t[i];
    j_out[i] = j[i];
  }
}

hipError_t launch_copy_samples(const float* t, const int32_t* j, float* t_out, int32_t* j_out,
                               int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(k_copy_samples, dim3(1024), dim3(256), 0, s, t, j, t_out, j_out, n);
  return hipGetLastError();
}

hipError_t launch_offsets_i64(const int32_t* off, int64_t* out, int n, int64_t base,
                              hipStream_t s) {
  hipLaunchKernelGGL(k_offsets_i64, dim3((n + 255) / 256), dim3(256), 0, s, off, out, n, base);
  return hipGetLastError();
}

}  // namespace pnerf
