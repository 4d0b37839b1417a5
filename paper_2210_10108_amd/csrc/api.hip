// C ABI (include/pnerf.h): field creation with MFMA weight-tile layout,
// workspace management, hypothesis chunking, kernel sequencing, profiling and
// error reporting.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/pnerf.h"
#include "pnerf_internal.h"

using namespace pnerf;

namespace {

thread_local std::string g_err;

pnerf_status fail(pnerf_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess)                                                               \
      return fail(e_ == hipErrorOutOfMemory ? PNERF_ERR_OUT_OF_MEMORY : PNERF_ERR_DEVICE, \
                  "%s: %s", #expr, hipGetErrorString(e_));                              \
  } while (0)

float half_to_float(uint16_t h) {
  uint32_t s = (h >> 15) & 1u, e = (h >> 10) & 0x1Fu, m = h & 0x3FFu;
  float v;
  if (e == 0)
    v = std::ldexp((float)m, -24);
  else if (e == 31)
    v = m ? NAN : INFINITY;
  else
    v = std::ldexp((float)(m | 0x400u), (int)e - 25);
  return s ? -v : v;
}

struct KernelStat {
  std::string name;
  int64_t launches = 0;
  double total_ms = 0.0;
};

struct PendingEvent {
  int idx;
  hipEvent_t a, b;
};

}  // namespace

struct pnerf_field {
  DevField dev{};
  int device = 0;
  // owned device memory
  void* d_table = nullptr;
  void* d_wfwd = nullptr;
  void* d_wbwd = nullptr;
  void* d_hfwd = nullptr;       // fp16 tiles (mlp_precision 1)
  void* d_hbwd = nullptr;
  float* d_wc3 = nullptr;
  float* d_wd1 = nullptr;
  float* d_wd2 = nullptr;
  uint32_t* d_occ = nullptr;
  int64_t occ_words = 0;
  // workspace: per-ray arrays of one counted batch, per-sample arrays of one chunk
  void* d_rays = nullptr;
  size_t rays_bytes = 0;
  int rays_cap = 0, rays_hyp = 0;
  void* d_samp[2] = {nullptr, nullptr};  // two sample buffers (pipelined chunks alternate)
  size_t samp_bytes = 0;
  int64_t samp_cap = 0;
  int n_slots = 0;              // sample buffers allocated (1 or 2)
  int overlap_chunks = 0;       // chunks a loss-gradient batch is cut into for overlap
  int backward = 0;             // pnerf_field_params::backward
  bool last_keeps_samples = false;  // the last call left per-sample intermediates
  // internal streams of the pipelined loss gradient: encoding | networks
  hipStream_t s_enc = nullptr, s_mlp = nullptr;
  hipEvent_t ev_start = nullptr, ev_enc[2] = {nullptr, nullptr}, ev_mlp[2] = {nullptr, nullptr};
  hipEvent_t ev_end_enc = nullptr, ev_end_mlp = nullptr;
  int32_t* d_totals = nullptr;  // [max_chunks] sample totals of the chunks, + 1 counted total
  uint32_t* d_queue = nullptr;  // encoding work-queue counters (see DevWork::queue)
  int max_chunks = 0;
  int32_t* h_hyp = nullptr;     // pinned host copy of the per-hypothesis sample counts
  int h_hyp_cap = 0;
  int last_chunks = 0;
  int64_t last_total = 0;
  const int32_t* last_total_dev = nullptr;  // the last call's total, when only the device holds it
  int64_t budget = 0;
  int n_cu = 0, fwd_blocks = 0, bwd_blocks = 0, ray_blocks = 0, enc_blocks = 0,
      enc_blocks_overlap = 0;
  // profiling
  bool profiling = false;
  std::vector<KernelStat> stats;
  std::vector<PendingEvent> pending;
  std::vector<hipEvent_t> ev_pool;  // timing events made once, reused across launches
};

namespace {

// ------------------------------------------------------------ weight tiles
// Weight units (see WeightUnit): unit u, lane l = 16 g + r, K position j holds
// the weight of output row r of the unit's row tile and of the input that the
// previous layer's accumulator layout puts at position j of lane group g of
// the unit's K step: hidden unit 16 (2 s + j / 4) + 4 g + j % 4 of step s.
// Each fp32 weight w is stored as bf16 hi = rn(w) and lo = rn(w - hi).
struct Weights {
  int din;
  std::vector<float> d1, d2, c1, c2, c3;  // [in][out]
  float D1(int i, int o) const { return d1[(size_t)i * 64 + o]; }
  float D2(int i, int o) const { return d2[(size_t)i * 16 + o]; }
  float C1(int i, int o) const { return c1[(size_t)i * 64 + o]; }
  float C2(int i, int o) const { return c2[(size_t)i * 64 + o]; }
  float C3(int i, int o) const { return c3[(size_t)i * 3 + o]; }
};

uint16_t bf16_rn(float x) {
  uint32_t u;
  std::memcpy(&u, &x, 4);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);  // NaN
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

float bf16_value(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float x;
  std::memcpy(&x, &u, 4);
  return x;
}

struct Units {
  std::vector<uint16_t> v;  // [unit][hi, lo][lane][8]
  explicit Units(int n) : v((size_t)n * 2 * 64 * 8, 0) {}
  void put(int unit, int lane, int j, float w) {
    const uint16_t hi = bf16_rn(w);
    const uint16_t lo = bf16_rn(w - bf16_value(hi));
    v[(((size_t)unit * 2 + 0) * 64 + lane) * 8 + j] = hi;
    v[(((size_t)unit * 2 + 1) * 64 + lane) * 8 + j] = lo;
  }
};

// fp32 -> fp16, round to nearest even (IEEE binary16, subnormals kept).
uint16_t f16_rn(float x) {
  uint32_t u;
  std::memcpy(&u, &x, 4);
  const uint16_t sign = (uint16_t)((u >> 16) & 0x8000u);
  const uint32_t a = u & 0x7FFFFFFFu;
  if (a > 0x7F800000u) return sign | 0x7E00u;   // NaN
  if (a >= 0x477FF000u) return sign | 0x7C00u;  // from 65520 up: infinity
  if (a < 0x38800000u) {                        // below 2^-14: multiples of 2^-24
    float m;
    std::memcpy(&m, &a, 4);
    return sign | (uint16_t)std::nearbyint(m * 16777216.0f);  // exact product, ties to even
  }
  uint32_t r = a - 0x38000000u;                 // exponent bias 127 -> 15
  r += 0xFFFu + ((r >> 13) & 1u);
  return sign | (uint16_t)(r >> 13);
}

// The weight units of v_mfma_f32_16x16x32_f16: each fp32 weight as fp16
// hi = rn(w) and lo = rn(w - hi) (w - hi is exact in fp32).
struct HalfUnits {
  std::vector<uint16_t> v;  // [unit][hi, lo][lane][8]
  explicit HalfUnits(int n) : v((size_t)n * 2 * 64 * 8, 0) {}
  void put(int unit, int lane, int j, float w) {
    const uint16_t hi = f16_rn(w);
    const uint16_t lo = f16_rn(w - half_to_float(hi));
    v[(((size_t)unit * 2 + 0) * 64 + lane) * 8 + j] = hi;
    v[(((size_t)unit * 2 + 1) * 64 + lane) * 8 + j] = lo;
  }
};

// hidden unit at K position j of lane group g in K step s
inline int kpos(int s, int g, int j) { return 16 * (2 * s + j / 4) + 4 * g + j % 4; }

template <class U_t>
U_t build_fwd_units(const Weights& W, int lpg) {
  U_t U(kFwdUnits);
  for (int lane = 0; lane < 64; ++lane) {
    const int g = lane / 16, r = lane % 16;
    for (int j = 0; j < 8; ++j) {
      for (int m = 0; m < 4; ++m) {
        // density 1: position j = feature j % 2 of level 4 (j / 2) + g
        if (j < 2 * lpg) U.put(kFD1 + m, lane, j, W.D1(2 * (4 * (j / 2) + g) + j % 2, 16 * m + r));
        // colour 1: positions 0..3 = h_{4g+j} (x_c index 4g+j-1; h_0 has no weight),
        // positions 4..7 = SH_{4g+j-4} (x_c index 15 + 4g + j - 4)
        const int hidx = 4 * g + j;
        if (j < 4)
          U.put(kFC1 + m, lane, j, hidx >= 1 ? W.C1(hidx - 1, 16 * m + r) : 0.0f);
        else
          U.put(kFC1 + m, lane, j, W.C1(15 + 4 * g + (j - 4), 16 * m + r));
      }
      for (int s2 = 0; s2 < 2; ++s2) {
        const int u = kpos(s2, g, j);
        U.put(kFD2 + s2, lane, j, W.D2(u, r));
        U.put(kFC3 + s2, lane, j, r < 3 ? W.C3(u, r) : 0.0f);
        for (int m = 0; m < 4; ++m) U.put(kFC2 + 2 * m + s2, lane, j, W.C2(u, 16 * m + r));
      }
    }
  }
  return U;
}

template <class U_t>
U_t build_bwd_units(const Weights& W, int lpg) {
  U_t U(kBwdUnits);
  const int MD = (lpg + 1) / 2;
  for (int lane = 0; lane < 64; ++lane) {
    const int g = lane / 16, r = lane % 16;
    for (int j = 0; j < 8; ++j) {
      for (int s2 = 0; s2 < 2; ++s2) {
        const int o = kpos(s2, g, j);  // the layer's output unit (K of the transpose)
        for (int m = 0; m < 4; ++m) U.put(kBC2 + 2 * m + s2, lane, j, W.C2(16 * m + r, o));
        U.put(kBC1 + s2, lane, j, r >= 1 ? W.C1(r - 1, o) : 0.0f);  // h rows
        U.put(kBSH + s2, lane, j, W.C1(15 + r, o));                  // SH rows
        // density 1: row r = feature (r % 4) % 2 of level 4 (2 mm + (r % 4) / 2) + r / 4
        for (int mm = 0; mm < MD; ++mm) {
          const int jl = 2 * mm + (r % 4) / 2;
          const float v = jl < lpg ? W.D1(2 * (4 * jl + r / 4) + (r % 4) % 2, o) : 0.0f;
          U.put(kBD1 + 2 * mm + s2, lane, j, v);
        }
      }
      // density 2: one K step, positions 0..3 = h_{4g+j}
      for (int m = 0; m < 4; ++m) U.put(kBD2 + m, lane, j, j < 4 ? W.D2(16 * m + r, 4 * g + j) : 0.0f);
    }
  }
  return U;
}

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

struct Carver {
  char* base;
  size_t off = 0;
  template <class T>
  T* take(size_t n) {
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += align_up(n * sizeof(T));
    return p;
  }
};

// Per-ray arrays for n_rays rays (one counted batch).  `offc` receives the
// sample chunks' own exclusive offsets.
struct RayWs {
  float *rdx, *rdy, *rdz, *rtn, *rtf, *rdelta, *rex, *rey, *rez, *rsh;
  int32_t *count, *off, *blocksum, *hyp_total;
  int32_t* offc[2];             // per sample buffer: the chunk's own offsets,
  float *ray_loss[2], *partial[2];  // per-ray losses and reduction partials
  float* ray_terms[2];          // fused backward: [n_rays][7] per-ray torque, force, loss
};

size_t carve_rays(int n_rays, int n_hyp, RayWs* r, char* base) {
  Carver c{base};
  const size_t R = (size_t)n_rays;
  RayWs tmp{};
  RayWs& x = r ? *r : tmp;
  x.rdx = c.take<float>(R);
  x.rdy = c.take<float>(R);
  x.rdz = c.take<float>(R);
  x.rtn = c.take<float>(R);
  x.rtf = c.take<float>(R);
  x.rdelta = c.take<float>(R);
  x.rex = c.take<float>(R);
  x.rey = c.take<float>(R);
  x.rez = c.take<float>(R);
  x.rsh = c.take<float>(R * 16);
  x.count = c.take<int32_t>(R);
  x.off = c.take<int32_t>(R + 1);
  x.blocksum = c.take<int32_t>((R + 255) / 256);
  x.hyp_total = c.take<int32_t>(R);
  for (int q = 0; q < 2; ++q) {
    x.offc[q] = c.take<int32_t>(R + 1);
    x.ray_loss[q] = c.take<float>(R);
    x.partial[q] = c.take<float>((size_t)n_hyp * kReduceParts * 7);
    x.ray_terms[q] = c.take<float>(R * 7);
  }
  return c.off;
}

// Per-sample arrays for cap samples (one chunk); cap is a multiple of kTile.
size_t carve_samples(const DevField& f, int64_t cap, DevWork* w, char* base) {
  Carver c{base};
  const size_t n = (size_t)cap;
  DevWork tmp{};
  DevWork& x = w ? *w : tmp;
  x.t = c.take<float>(n);
  x.sray = c.take<int32_t>(n);
  x.sig = c.take<float>(n);
  x.cr = c.take<float>(n);
  x.cg = c.take<float>(n);
  x.cb = c.take<float>(n);
  x.masks = c.take<uint32_t>(n / kTile * kMaskWords * 64);
  x.feat = c.take<float>((size_t)std::max(2 * f.L, 6) * n);
  x.jac = c.take<__half>((size_t)6 * f.L * n);
  x.cap = cap;
  return c.off;
}

// Device views: the counted batch (all per-ray arrays from ray 0) and one
// sample chunk (per-ray arrays from the chunk's first ray, its own offsets).
DevWork counted_work(pnerf_field* F) {
  RayWs r{};
  carve_rays(F->rays_cap, F->rays_hyp, &r, (char*)F->d_rays);
  DevWork w{};
  w.rdx = r.rdx; w.rdy = r.rdy; w.rdz = r.rdz;
  w.rtn = r.rtn; w.rtf = r.rtf; w.rdelta = r.rdelta;
  w.rex = r.rex; w.rey = r.rey; w.rez = r.rez;
  w.rsh = r.rsh;
  w.count = r.count;
  w.off = r.off;
  w.blocksum = r.blocksum;
  w.hyp_total = r.hyp_total;
  w.total = F->d_totals + F->max_chunks;
  return w;
}

DevWork chunk_work(pnerf_field* F, int ray_base, int chunk_id, int slot) {
  RayWs r{};
  carve_rays(F->rays_cap, F->rays_hyp, &r, (char*)F->d_rays);
  DevWork w{};
  carve_samples(F->dev, F->samp_cap, &w, (char*)F->d_samp[slot]);
  w.rdx = r.rdx + ray_base; w.rdy = r.rdy + ray_base; w.rdz = r.rdz + ray_base;
  w.rtn = r.rtn + ray_base; w.rtf = r.rtf + ray_base; w.rdelta = r.rdelta + ray_base;
  w.rex = r.rex + ray_base; w.rey = r.rey + ray_base; w.rez = r.rez + ray_base;
  w.rsh = r.rsh + (size_t)16 * ray_base;
  w.count = r.count + ray_base;
  w.off = r.offc[slot];
  w.blocksum = nullptr;
  w.hyp_total = nullptr;
  w.ray_loss = r.ray_loss[slot];
  w.partial = r.partial[slot];
  w.ray_terms = r.ray_terms[slot];
  w.total = F->d_totals + chunk_id;
  w.queue = F->d_queue;
  return w;
}

int64_t bytes_per_sample(const DevField& f) {
  return (int64_t)carve_samples(f, 64 * kTile, nullptr, nullptr) / (64 * kTile) + 1;
}

// Under stream capture nothing may be allocated or waited for: a workspace
// that would have to grow is refused instead.
pnerf_status refuse_growth_in_capture(bool capturing, const char* what) {
  if (!capturing) return PNERF_OK;
  return fail(PNERF_ERR_NOT_SUPPORTED,
              "the %s would grow under stream capture: run the same shape once outside the "
              "capture first", what);
}

pnerf_status ensure_rays(pnerf_field* F, int n_rays, int n_hyp, hipStream_t s, bool capturing) {
  if (n_rays > F->rays_cap || n_hyp > F->rays_hyp || n_hyp > F->h_hyp_cap) {
    pnerf_status st = refuse_growth_in_capture(capturing, "ray workspace");
    if (st != PNERF_OK) return st;
  }
  if (n_rays > F->rays_cap || n_hyp > F->rays_hyp) {
    n_rays = std::max(n_rays, F->rays_cap);
    n_hyp = std::max(n_hyp, F->rays_hyp);
    if (F->d_rays) {
      HIP_TRY(hipStreamSynchronize(s));
      HIP_TRY(hipFree(F->d_rays));
      F->d_rays = nullptr;
      F->rays_cap = 0;
      F->rays_hyp = 0;
    }
    size_t bytes = carve_rays(n_rays, n_hyp, nullptr, nullptr);
    hipError_t e = hipMalloc(&F->d_rays, bytes);
    if (e != hipSuccess)
      return fail(PNERF_ERR_OUT_OF_MEMORY, "ray workspace of %zu bytes: %s", bytes, hipGetErrorString(e));
    F->rays_bytes = bytes;
    F->rays_cap = n_rays;
    F->rays_hyp = n_hyp;
  }
  if (n_hyp > F->h_hyp_cap) {
    if (F->h_hyp) {
      HIP_TRY(hipStreamSynchronize(s));
      HIP_TRY(hipHostFree(F->h_hyp));
      F->h_hyp = nullptr;
      F->h_hyp_cap = 0;
    }
    HIP_TRY(hipHostMalloc((void**)&F->h_hyp, sizeof(int32_t) * (size_t)n_hyp));
    F->h_hyp_cap = n_hyp;
  }
  return PNERF_OK;
}

// Grow the sample workspace to `slots` buffers of `need` samples each (a
// quarter more than asked when it grows, within `limit`), and the per-chunk
// totals to n_chunks.
pnerf_status ensure_samples(pnerf_field* F, int64_t need, int64_t limit, int n_chunks, int slots,
                            hipStream_t s, bool capturing) {
  if (n_chunks > F->max_chunks || std::max<int64_t>(need, 1) > F->samp_cap || slots > F->n_slots) {
    pnerf_status st = refuse_growth_in_capture(capturing, "sample workspace");
    if (st != PNERF_OK) return st;
  }
  if (n_chunks > F->max_chunks) {
    if (F->d_totals) {
      HIP_TRY(hipStreamSynchronize(s));
      HIP_TRY(hipFree(F->d_totals));
      F->d_totals = nullptr;
    }
    int nc = std::max(n_chunks, 16);
    HIP_TRY(hipMalloc(&F->d_totals, sizeof(int32_t) * (nc + 1)));
    F->max_chunks = nc;
  }
  need = std::max<int64_t>(need, 1);
  if (need <= F->samp_cap && slots <= F->n_slots) return PNERF_OK;
  int64_t cap = need <= F->samp_cap ? F->samp_cap
                                     : std::max(need, std::min(limit, F->samp_cap + F->samp_cap / 4));
  cap = (cap + kTile - 1) / kTile * kTile;
  slots = std::max(slots, F->n_slots);
  HIP_TRY(hipStreamSynchronize(s));
  for (int q = 0; q < 2; ++q) {
    if (F->d_samp[q]) HIP_TRY(hipFree(F->d_samp[q]));
    F->d_samp[q] = nullptr;
  }
  F->samp_cap = 0;
  F->n_slots = 0;
  size_t bytes = carve_samples(F->dev, cap, nullptr, nullptr);
  for (int q = 0; q < slots; ++q) {
    hipError_t e = hipMalloc(&F->d_samp[q], bytes);
    if (e != hipSuccess)
      return fail(PNERF_ERR_OUT_OF_MEMORY, "sample workspace of %zu bytes: %s", bytes,
                  hipGetErrorString(e));
  }
  F->samp_bytes = bytes;
  F->samp_cap = cap;
  F->n_slots = slots;
  return PNERF_OK;
}

// Internal streams (default priority, non-blocking) and events of the
// pipelined loss gradient, made on first use.
pnerf_status ensure_pipeline(pnerf_field* F) {
  if (F->s_enc) return PNERF_OK;
  HIP_TRY(hipStreamCreateWithFlags(&F->s_enc, hipStreamNonBlocking));
  HIP_TRY(hipStreamCreateWithFlags(&F->s_mlp, hipStreamNonBlocking));
  hipEvent_t* evs[] = {&F->ev_start, &F->ev_enc[0], &F->ev_enc[1], &F->ev_mlp[0], &F->ev_mlp[1],
                       &F->ev_end_enc, &F->ev_end_mlp};
  for (hipEvent_t* e : evs) HIP_TRY(hipEventCreateWithFlags(e, hipEventDisableTiming));
  return PNERF_OK;
}

// --------------------------------------------------------------- profiling
template <class Fn>
hipError_t timed(pnerf_field* F, const char* name, hipStream_t s, Fn fn) {
  if (!F->profiling) return fn();
  int idx = -1;
  for (size_t i = 0; i < F->stats.size(); ++i)
    if (F->stats[i].name == name) idx = (int)i;
  if (idx < 0) {
    F->stats.push_back(KernelStat{name, 0, 0.0});
    idx = (int)F->stats.size() - 1;
  }
  PendingEvent pe{idx, nullptr, nullptr};
  hipError_t e = hipSuccess;
  for (hipEvent_t* ev : {&pe.a, &pe.b}) {
    if (F->ev_pool.empty()) {
      e = hipEventCreate(ev);
      if (e != hipSuccess) return e;
    } else {
      *ev = F->ev_pool.back();
      F->ev_pool.pop_back();
    }
  }
  e = hipEventRecord(pe.a, s);
  if (e != hipSuccess) return e;
  e = fn();
  if (e != hipSuccess) return e;
  e = hipEventRecord(pe.b, s);
  F->pending.push_back(pe);
  F->stats[idx].launches += 1;
  return e;
}

pnerf_status resolve_profile(pnerf_field* F) {
  for (auto& pe : F->pending) {
    HIP_TRY(hipEventSynchronize(pe.b));
    float ms = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, pe.a, pe.b));
    F->stats[pe.idx].total_ms += ms;
    F->ev_pool.push_back(pe.a);
    F->ev_pool.push_back(pe.b);
  }
  F->pending.clear();
  return PNERF_OK;
}

// --------------------------------------------------------------- batches
pnerf_status check_batch(pnerf_field* F, int32_t K, const float* poses, int32_t P,
                         const int32_t* pix, const pnerf_intrinsics* intr) {
  if (!F) return fail(PNERF_ERR_INVALID_ARG, "field is NULL");
  if (K < 1 || P < 1) return fail(PNERF_ERR_INVALID_ARG, "K=%d and P=%d must be >= 1", K, P);
  // the per-hypothesis reduction runs one grid row per hypothesis
  if (K > 65535) return fail(PNERF_ERR_INVALID_ARG, "K=%d exceeds 65535", K);
  if ((int64_t)K * P >= ((int64_t)1 << 31))
    return fail(PNERF_ERR_INVALID_ARG, "K*P=%lld exceeds 2^31-1", (long long)K * P);
  if (!poses || !pix || !intr) return fail(PNERF_ERR_INVALID_ARG, "NULL pointer argument");
  if (intr->width < 1 || intr->height < 1 || !(intr->fx > 0.0f) || !(intr->fy > 0.0f) ||
      !std::isfinite(intr->cx) || !std::isfinite(intr->cy))
    return fail(PNERF_ERR_INVALID_ARG, "invalid intrinsics");
  if ((int64_t)intr->width * intr->height >= ((int64_t)1 << 31))
    return fail(PNERF_ERR_INVALID_ARG, "image too large");
  return PNERF_OK;
}

DevBatch make_batch(int32_t K, const float* poses, int32_t P, const int32_t* pix,
                    const float* obs, const pnerf_intrinsics* intr) {
  DevBatch b{};
  b.K = K;
  b.P = P;
  b.n_rays = K * P;
  b.poses = poses;
  b.pix = pix;
  b.obs = obs;
  b.W = intr->width;
  b.H = intr->height;
  b.fx = intr->fx;
  b.fy = intr->fy;
  b.cx = intr->cx;
  b.cy = intr->cy;
  return b;
}

enum Mode { kLossGrad, kRender, kMarch };

// One call: the rays of up to kMaxScanBlocks * 256 rays (whole hypotheses) are
// counted at a time; the host reads their per-hypothesis sample counts (one
// stream synchronisation) and cuts them into chunks of whole hypotheses whose
// samples fit the workspace budget; every chunk then runs the write pass and
// the shading pipeline.
pnerf_status run(pnerf_field* F, Mode mode, int32_t K, const float* poses, int32_t P,
                 const int32_t* pix, const float* obs, const pnerf_intrinsics* intr, float* loss,
                 float* dpose, float* rgb, int64_t* ray_offset, float* t_out, int32_t* j_out,
                 int64_t capacity, hipStream_t s) {
  HIP_TRY(hipSetDevice(F->device));
  // under stream capture (a HIP graph being recorded) the call may only
  // enqueue kernels: no allocation, no event timing, no read of the totals
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  HIP_TRY(hipStreamIsCapturing(s, &cs));
  const bool capturing = cs != hipStreamCaptureStatusNone;
  if (capturing && (mode != kLossGrad || F->profiling))
    return fail(PNERF_ERR_NOT_SUPPORTED, "only render_loss_grad, without profiling, can be "
                                         "recorded under stream capture");
  F->last_total_dev = nullptr;
  F->last_keeps_samples = mode != kLossGrad || F->backward != 1;
  const int64_t max_rays = (int64_t)kMaxScanBlocks * 256;
  int32_t kr = 0;
  pnerf_status st = pnerf_plan_counted_batch(K, P, F->dev.max_per_ray, &kr);
  if (st != PNERF_OK) return st;
  if (mode == kMarch && kr < K)
    return fail(PNERF_ERR_CAPACITY, "march inspection needs K*P <= %lld rays", (long long)max_rays);
  st = ensure_rays(F, kr * P, kr, s, capturing);
  if (st != PNERF_OK) return st;
  const int64_t per_sample = bytes_per_sample(F->dev);  // per buffer
  const int64_t limit = std::min<int64_t>(
      std::max<int64_t>((F->budget - (int64_t)F->rays_bytes) / per_sample, kTile),
      ((int64_t)1 << 31) - 4 * kTile);
  // loss gradient: several chunks, encoding of one overlapping the networks of
  // the previous, on two internal streams with a sample buffer each
  const int n_target = mode == kLossGrad ? std::max(1, F->overlap_chunks) : 1;
  const bool pipe = n_target > 1;
  if (pipe) {
    st = ensure_pipeline(F);
    if (st != PNERF_OK) return st;
  }
  const int64_t slot_limit = pipe ? std::max<int64_t>(limit / 2, kTile) : limit;
  int chunk_id = 0;
  int64_t grand = 0;
  for (int h0 = 0; h0 < K; h0 += kr) {
    const int hn = std::min(kr, K - h0);
    DevBatch bb = make_batch(hn, poses + (size_t)12 * h0, P, pix + (size_t)P * h0, obs, intr);
    // A loss gradient whose worst case (every ray at its sample cap) fits one
    // buffer runs as one chunk in a buffer sized for that worst case: the host
    // needs no sample totals, so the call never waits for the device.
    const int64_t worst = (int64_t)hn * P * F->dev.max_per_ray;
    const bool device_sized = mode == kLossGrad && !pipe && hn == K && worst <= limit &&
                              worst * per_sample <= kDeviceSizedBytes;
    if (capturing && !device_sized)
      return fail(PNERF_ERR_NOT_SUPPORTED,
                  "this batch needs the host's chunk plan (a read of its sample totals), which "
                  "stream capture cannot record");
    // the totals array for the counted batch (and, device-sized, the whole buffer)
    st = ensure_samples(F, device_sized ? worst : 0, slot_limit, chunk_id + 1, 1, s, capturing);
    if (st != PNERF_OK) return st;
    DevWork wb = counted_work(F);
    int raw_blocks = 0;  // device-sized: the write pass may finish the offset scan itself
    HIP_TRY(timed(F, "march", s, [&] {
      return launch_march_count(F->dev, bb, wb, device_sized, &raw_blocks, s);
    }));
    std::vector<int> cut{0};
    std::vector<int64_t> sums;  // samples per chunk; -1: the counted total, on the device
    int64_t counted = 0;
    bool overlap = false;
    if (device_sized) {
      cut.push_back(hn);
      sums.push_back(-1);
    } else {
      HIP_TRY(hipMemcpyAsync(F->h_hyp, wb.hyp_total, sizeof(int32_t) * hn, hipMemcpyDeviceToHost, s));
      HIP_TRY(hipStreamSynchronize(s));
      // chunks of whole hypotheses: about 1/n_target of the samples each (when
      // pipelined) and never more than a buffer holds
      for (int k = 0; k < hn; ++k) counted += F->h_hyp[k];
      const bool pipe_here = pipe && hn > 1 && counted >= (int64_t)kMinOverlapSamples;
      const int64_t cap_c = pipe_here ? slot_limit : limit;
      const int64_t goal = pipe_here ? (counted + n_target - 1) / n_target : cap_c;
      cut.assign((size_t)hn + 1, 0);
      sums.assign((size_t)hn, 0);
      int32_t nc = 0;
      st = pnerf_plan_chunks(F->h_hyp, hn, cap_c, goal, cut.data(), sums.data(), &nc);
      if (st != PNERF_OK) return fail(st, "hypotheses %d..%d: %s", h0, h0 + hn - 1, g_err.c_str());
      cut.resize((size_t)nc + 1);
      sums.resize((size_t)nc);
      int64_t biggest = 0;
      for (int64_t v : sums) biggest = std::max(biggest, v);
      overlap = pipe_here && sums.size() > 1;
      st = ensure_samples(F, biggest, cap_c, chunk_id + (int)sums.size(), overlap ? 2 : 1, s,
                          false);
      if (st != PNERF_OK) return st;
      wb = counted_work(F);
    }
    const int n_chunks = (int)sums.size();
    hipStream_t se = overlap ? F->s_enc : s, sm = overlap ? F->s_mlp : s;
    if (overlap) {
      HIP_TRY(hipEventRecord(F->ev_start, s));
      HIP_TRY(hipStreamWaitEvent(se, F->ev_start, 0));
      HIP_TRY(hipStreamWaitEvent(sm, F->ev_start, 0));
    }
    int64_t base = 0;  // samples of the counted batch before this chunk
    for (int c = 0; c < n_chunks; ++c, ++chunk_id) {
      const int a = cut[c], kn = cut[c + 1] - cut[c], k0 = h0 + a;
      const int slot = overlap ? c & 1 : 0;
      DevBatch b = make_batch(kn, poses + (size_t)12 * k0, P, pix + (size_t)P * k0, obs, intr);
      DevWork w = chunk_work(F, a * P, chunk_id, slot);
      // the buffer is free once the networks of chunk c - 2 are done
      if (overlap) HIP_TRY(hipStreamWaitEvent(se, F->ev_mlp[slot], 0));
      // inspection: lattice indices go to the (otherwise unused) blue-channel buffer
      int32_t* j_tmp = mode == kMarch ? reinterpret_cast<int32_t*>(w.cb) : nullptr;
      HIP_TRY(timed(F, "march_write", se, [&] {
        return launch_march_write(F->dev, b, wb, w, a * P, (int)base, (int)sums[c], raw_blocks, j_tmp,
                                  se);
      }));
      if (mode == kMarch) {
        const bool last = k0 + kn == K;
        HIP_TRY(launch_offsets_i64(w.off, ray_offset + (size_t)P * k0, b.n_rays + (last ? 1 : 0),
                                   grand + base, s));
        if (capacity >= counted && sums[c] > 0)
          HIP_TRY(launch_copy_samples(w.t, j_tmp, t_out + grand + base, j_out + grand + base,
                                      sums[c], s));
      } else if (mode == kRender) {
        HIP_TRY(timed(F, "encode_render", s, [&] { return launch_encode(F->dev, b, w, F->enc_blocks, 0, s); }));
        HIP_TRY(timed(F, "mlp_fwd_render", s, [&] {
          return launch_mlp_fwd(F->dev, b, w, F->fwd_blocks, 0, s);
        }));
        HIP_TRY(timed(F, "composite_fwd", s, [&] {
          return launch_composite(F->dev, b, w, 0, rgb + (size_t)3 * P * k0, s);
        }));
      } else {
        const int eb = overlap ? F->enc_blocks_overlap : F->enc_blocks;
        HIP_TRY(timed(F, "encode", se, [&] { return launch_encode(F->dev, b, w, eb, 1, se); }));
        if (overlap) {
          HIP_TRY(hipEventRecord(F->ev_enc[slot], se));
          HIP_TRY(hipStreamWaitEvent(sm, F->ev_enc[slot], 0));
        }
        HIP_TRY(timed(F, "mlp_fwd", sm, [&] { return launch_mlp_fwd(F->dev, b, w, F->fwd_blocks, 1, sm); }));
        if (F->backward == 0) {
          HIP_TRY(timed(F, "composite", sm, [&] { return launch_composite(F->dev, b, w, 1, nullptr, sm); }));
          HIP_TRY(timed(F, "mlp_bwd", sm, [&] { return launch_mlp_bwd(F->dev, b, w, F->bwd_blocks, sm); }));
          HIP_TRY(timed(F, "reduce", sm, [&] {
            return launch_reduce(F->dev, b, w, loss + k0, dpose + (size_t)6 * k0, sm);
          }));
        } else {
          HIP_TRY(timed(F, "ray_bwd", sm, [&] {
            return launch_ray_bwd(F->dev, b, w, F->ray_blocks, F->backward == 2, sm);
          }));
          HIP_TRY(timed(F, "reduce", sm, [&] {
            return launch_reduce_rays(b, w, loss + k0, dpose + (size_t)6 * k0, sm);
          }));
        }
        if (overlap) HIP_TRY(hipEventRecord(F->ev_mlp[slot], sm));
      }
      base += device_sized ? 0 : sums[c];
    }
    if (overlap) {
      // the caller's stream continues once both internal streams are done
      HIP_TRY(hipEventRecord(F->ev_end_enc, se));
      HIP_TRY(hipEventRecord(F->ev_end_mlp, sm));
      HIP_TRY(hipStreamWaitEvent(s, F->ev_end_enc, 0));
      HIP_TRY(hipStreamWaitEvent(s, F->ev_end_mlp, 0));
    }
    grand += counted;
    F->last_total_dev = device_sized ? wb.total : nullptr;
  }
  F->last_chunks = chunk_id;
  F->last_total = grand;
  return PNERF_OK;
}

}  // namespace

// =================================================================== C ABI
extern "C" {

const char* pnerf_last_error(void) { return g_err.c_str(); }

pnerf_status pnerf_plan_counted_batch(int32_t K, int32_t P, int32_t max_per_ray,
                                      int32_t* hyps_per_batch) {
  if (!hyps_per_batch) return fail(PNERF_ERR_INVALID_ARG, "NULL hyps_per_batch");
  *hyps_per_batch = 0;
  if (K < 1 || P < 1 || max_per_ray < 1)
    return fail(PNERF_ERR_INVALID_ARG, "K=%d, P=%d and max_per_ray=%d must be >= 1", K, P,
                max_per_ray);
  const int64_t max_rays = (int64_t)kMaxScanBlocks * 256;
  if (P > max_rays)
    return fail(PNERF_ERR_CAPACITY, "P=%d rays per hypothesis exceeds %lld", P, (long long)max_rays);
  // counts, block sums, hypothesis totals and offsets of a counted batch are
  // 32-bit: its worst case (every ray at its cap) must stay below 2^31
  const int64_t hyp_worst = (int64_t)P * max_per_ray;
  if (hyp_worst > kMaxCountedSamples)
    return fail(PNERF_ERR_CAPACITY, "P=%d rays of up to %d samples each (%lld) may exceed the "
                "%lld samples one hypothesis can hold", P, max_per_ray, (long long)hyp_worst,
                (long long)kMaxCountedSamples);
  *hyps_per_batch =
      (int32_t)std::min<int64_t>(std::min<int64_t>(K, max_rays / P), kMaxCountedSamples / hyp_worst);
  return PNERF_OK;
}

pnerf_status pnerf_plan_chunks(const int32_t* hyp_samples, int32_t n, int64_t capacity, int64_t goal,
                               int32_t* cut, int64_t* sums, int32_t* n_chunks) {
  if (!hyp_samples || !cut || !sums || !n_chunks || n < 1 || capacity < 1)
    return fail(PNERF_ERR_INVALID_ARG, "invalid chunk-planning arguments");
  *n_chunks = 0;
  for (int32_t k = 0; k < n; ++k)
    if (hyp_samples[k] < 0) return fail(PNERF_ERR_INVALID_ARG, "hypothesis %d: %d samples", k, hyp_samples[k]);
  int32_t c = 0;
  cut[0] = 0;
  for (int32_t a = 0; a < n;) {
    int64_t sum = 0;
    int32_t b = a;
    while (b < n && sum + hyp_samples[b] <= capacity && (sum < goal || b == a)) sum += hyp_samples[b++];
    if (b == a)
      return fail(PNERF_ERR_CAPACITY, "hypothesis %d has %d samples, more than the workspace "
                  "budget holds (%lld)", a, hyp_samples[a], (long long)capacity);
    sums[c] = sum;
    cut[++c] = b;
    a = b;
  }
  *n_chunks = c;
  return PNERF_OK;
}

pnerf_status pnerf_create_field(const pnerf_field_params* p, void* stream, pnerf_field** out) {
  if (!p || !out) return fail(PNERF_ERR_INVALID_ARG, "NULL params or out");
  *out = nullptr;
  hipStream_t s = (hipStream_t)stream;
  const int L = p->n_levels;
  if (L != 4 && L != 8 && L != 12 && L != 16)
    return fail(PNERF_ERR_NOT_SUPPORTED, "n_levels=%d (supported: 4, 8, 12, 16)", L);
  if (p->n_features != 2) return fail(PNERF_ERR_NOT_SUPPORTED, "n_features=%d (supported: 2)", p->n_features);
  if (p->log2_table_size < 4 || p->log2_table_size > 24)
    return fail(PNERF_ERR_INVALID_ARG, "log2_table_size=%d outside 4..24", p->log2_table_size);
  if (p->param_dtype != 0 && p->param_dtype != 1)
    return fail(PNERF_ERR_INVALID_ARG, "param_dtype=%d (0 float32, 1 float16)", p->param_dtype);
  if (!p->level_res || !p->table || !p->w_density1 || !p->w_density2 || !p->w_color1 ||
      !p->w_color2 || !p->w_color3)
    return fail(PNERF_ERR_INVALID_ARG, "NULL field array");
  for (int l = 0; l < L; ++l)
    if (p->level_res[l] < 1 || p->level_res[l] > (1 << 20))
      return fail(PNERF_ERR_INVALID_ARG, "level_res[%d]=%d outside 1..2^20", l, p->level_res[l]);
  for (int a = 0; a < 3; ++a)
    if (!(p->aabb_max[a] > p->aabb_min[a]) || !std::isfinite(p->aabb_min[a]) || !std::isfinite(p->aabb_max[a]))
      return fail(PNERF_ERR_INVALID_ARG, "empty or non-finite AABB on axis %d", a);
  if (p->march_mode == 0) {
    if (p->n_uniform < 1 || p->n_uniform > 4096)
      return fail(PNERF_ERR_INVALID_ARG, "n_uniform=%d outside 1..4096", p->n_uniform);
  } else if (p->march_mode == 1) {
    if (!(p->step > 0.0f) || !std::isfinite(p->step))
      return fail(PNERF_ERR_INVALID_ARG, "step must be > 0");
    if (p->max_samples < 1 || p->max_samples > 8192)
      return fail(PNERF_ERR_INVALID_ARG, "max_samples=%d outside 1..8192", p->max_samples);
    double diag2 = 0.0;
    for (int a = 0; a < 3; ++a) {
      double e = (double)p->aabb_max[a] - (double)p->aabb_min[a];
      diag2 += e * e;
    }
    if (std::sqrt(diag2) / (double)p->step > (double)kMaxLatticeCandidates)
      return fail(PNERF_ERR_INVALID_ARG, "step too small: more than %d lattice points per ray",
                  kMaxLatticeCandidates);
  } else {
    return fail(PNERF_ERR_INVALID_ARG, "march_mode=%d", p->march_mode);
  }
  if (p->occ_res < 0 || p->occ_res > 1024) return fail(PNERF_ERR_INVALID_ARG, "occ_res=%d", p->occ_res);
  if (p->loss_type < 0 || p->loss_type > 7)
    return fail(PNERF_ERR_INVALID_ARG, "loss_type=%d outside 0..7", p->loss_type);
  if (!(p->loss_param > 0.0f) || !std::isfinite(p->loss_param))
    return fail(PNERF_ERR_INVALID_ARG, "loss_param must be finite and > 0");
  if (p->sh_dir_grad != 0 && p->sh_dir_grad != 1) return fail(PNERF_ERR_INVALID_ARG, "sh_dir_grad");
  if (!(p->t_stop >= 0.0f)) return fail(PNERF_ERR_INVALID_ARG, "t_stop must be >= 0");
  if (p->overlap_chunks < 0 || p->overlap_chunks > 64)
    return fail(PNERF_ERR_INVALID_ARG, "overlap_chunks=%d outside 0..64", p->overlap_chunks);
  if (p->backward < 0 || p->backward > 2)
    return fail(PNERF_ERR_INVALID_ARG, "backward=%d outside 0..2", p->backward);
  if (p->mlp_precision != 0 && p->mlp_precision != 1)
    return fail(PNERF_ERR_INVALID_ARG, "mlp_precision=%d outside 0..1", p->mlp_precision);

  pnerf_field* F = new pnerf_field();
  auto cleanup_fail = [&](pnerf_status st) {
    pnerf_destroy_field(F);
    return st;
  };
  (void)hipGetDevice(&F->device);
  DevField& d = F->dev;
  d.L = L;
  d.lpg = L / 4;
  d.T = 1u << p->log2_table_size;
  for (int l = 0; l < kMaxLevels; ++l) {
    int N = l < L ? p->level_res[l] : 1;
    uint64_t n1 = (uint64_t)N + 1;
    d.res[l] = N;
    d.n1[l] = (uint32_t)n1;
    d.dense[l] = (p->dense_coarse_levels && n1 * n1 * n1 <= d.T) ? 1u : 0u;
  }
  d.f16 = p->param_dtype == 1;
  // work queues of the encoding kernel, one per level: hashed levels first, so
  // that the first queue of every XCD (queue x of XCD x) holds a hashed table
  {
    int q = 0;
    for (int l = 0; l < L; ++l)
      if (!d.dense[l]) d.q_level[q++] = l;
    for (int l = 0; l < L; ++l)
      if (d.dense[l]) d.q_level[q++] = l;
    for (; q < kMaxLevels; ++q) d.q_level[q] = 0;
  }
  d.density_bias = p->density_bias;
  d.bf16_neg1[0] = 0x0000BF80u;  // low half -1, high half 0
  d.bf16_neg1[1] = 0xBF800000u;  // low half 0, high half -1
  for (int a = 0; a < 3; ++a) {
    d.mn[a] = p->aabb_min[a];
    d.mx[a] = p->aabb_max[a];
    float ext = p->aabb_max[a] - p->aabb_min[a];
    d.inv_ext[a] = 1.0f / ext;
    d.inv_ext_err[a] = (float)((double)d.inv_ext[a] * (double)ext - 1.0);
  }
  d.march_mode = p->march_mode;
  d.n_uniform = p->n_uniform;
  d.step = p->step;
  d.max_samples = p->max_samples;
  d.t_stop = p->t_stop;
  d.occ_res = p->occ_res;
  for (int q = 0; q < 3; ++q) d.bg[q] = p->background[q];
  d.loss_type = p->loss_type;
  d.loss_param = p->loss_param;
  d.sh_dir_grad = p->sh_dir_grad;
  if (p->march_mode == 0) {
    d.max_per_ray = p->n_uniform;
  } else {
    double diag = 0.0;
    for (int a = 0; a < 3; ++a) {
      double e = (double)p->aabb_max[a] - (double)p->aabb_min[a];
      diag += e * e;
    }
    int64_t lat = (int64_t)std::ceil(std::sqrt(diag) / (double)p->step) + 2;
    d.max_per_ray = (int)std::min<int64_t>(lat, p->max_samples);
  }
  F->budget = p->max_workspace_bytes > 0 ? p->max_workspace_bytes : ((int64_t)96 << 30);

  // weights -> float, then MFMA tiles
  Weights W;
  W.din = 2 * L;
  auto load = [&](const void* src, size_t n, std::vector<float>& dst) {
    dst.resize(n);
    if (p->param_dtype == 0)
      std::memcpy(dst.data(), src, n * sizeof(float));
    else
      for (size_t i = 0; i < n; ++i) dst[i] = half_to_float(((const uint16_t*)src)[i]);
  };
  load(p->w_density1, (size_t)W.din * 64, W.d1);
  load(p->w_density2, 64 * 16, W.d2);
  load(p->w_color1, 32 * 64, W.c1);
  load(p->w_color2, 64 * 64, W.c2);
  load(p->w_color3, 64 * 3, W.c3);
  Units uf = build_fwd_units<Units>(W, d.lpg);
  Units ub = build_bwd_units<Units>(W, d.lpg);
  d.mlp_f16 = p->mlp_precision;
  // the fp16 network's tiles, built on the host with the others
  HalfUnits hf(d.mlp_f16 ? kFwdUnits : 0), hb(d.mlp_f16 ? kBwdUnits : 0);
  if (d.mlp_f16) {
    hf = build_fwd_units<HalfUnits>(W, d.lpg);
    hb = build_bwd_units<HalfUnits>(W, d.lpg);
  }

  size_t table_elems = (size_t)L * d.T * 2;
  size_t table_bytes = table_elems * (p->param_dtype == 0 ? 4 : 2);
#define CF_TRY(expr)                                                                  \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess)                                                             \
      return cleanup_fail(fail(e_ == hipErrorOutOfMemory ? PNERF_ERR_OUT_OF_MEMORY      \
                                                         : PNERF_ERR_DEVICE,            \
                               "%s: %s", #expr, hipGetErrorString(e_)));              \
  } while (0)
  CF_TRY(hipMalloc(&F->d_table, table_bytes));
  CF_TRY(hipMemcpyAsync(F->d_table, p->table, table_bytes, hipMemcpyHostToDevice, s));
  CF_TRY(hipMalloc(&F->d_wfwd, uf.v.size() * 2));
  CF_TRY(hipMemcpyAsync(F->d_wfwd, uf.v.data(), uf.v.size() * 2, hipMemcpyHostToDevice, s));
  CF_TRY(hipMalloc(&F->d_wbwd, ub.v.size() * 2));
  CF_TRY(hipMemcpyAsync(F->d_wbwd, ub.v.data(), ub.v.size() * 2, hipMemcpyHostToDevice, s));
  CF_TRY(hipMalloc(&F->d_wc3, W.c3.size() * 4));
  CF_TRY(hipMemcpyAsync(F->d_wc3, W.c3.data(), W.c3.size() * 4, hipMemcpyHostToDevice, s));
  CF_TRY(hipMalloc(&F->d_wd1, W.d1.size() * 4));
  CF_TRY(hipMemcpyAsync(F->d_wd1, W.d1.data(), W.d1.size() * 4, hipMemcpyHostToDevice, s));
  CF_TRY(hipMalloc(&F->d_wd2, W.d2.size() * 4));
  CF_TRY(hipMemcpyAsync(F->d_wd2, W.d2.data(), W.d2.size() * 4, hipMemcpyHostToDevice, s));
  d.table32 = p->param_dtype == 0 ? (const float*)F->d_table : nullptr;
  d.table16 = p->param_dtype == 1 ? (const __half*)F->d_table : nullptr;
  d.wfwd = (const WeightUnit*)F->d_wfwd;
  d.wbwd = (const WeightUnit*)F->d_wbwd;
  d.wc3 = F->d_wc3;
  d.hfwd = nullptr;
  d.hbwd = nullptr;
  if (d.mlp_f16) {
    CF_TRY(hipMalloc(&F->d_hfwd, hf.v.size() * 2));
    CF_TRY(hipMemcpyAsync(F->d_hfwd, hf.v.data(), hf.v.size() * 2, hipMemcpyHostToDevice, s));
    CF_TRY(hipMalloc(&F->d_hbwd, hb.v.size() * 2));
    CF_TRY(hipMemcpyAsync(F->d_hbwd, hb.v.data(), hb.v.size() * 2, hipMemcpyHostToDevice, s));
    d.hfwd = (const WeightUnit*)F->d_hfwd;
    d.hbwd = (const WeightUnit*)F->d_hbwd;
  }
  d.wd1 = F->d_wd1;
  d.wd2 = F->d_wd2;
  d.occ = nullptr;
  if (p->occ_res > 0) {
    int64_t R = p->occ_res;
    F->occ_words = (R * R * R + 31) / 32;
    CF_TRY(hipMalloc(&F->d_occ, F->occ_words * 4));
    d.occ = F->d_occ;
    if (p->occ_bits)
      CF_TRY(hipMemcpyAsync(F->d_occ, p->occ_bits, F->occ_words * 4, hipMemcpyHostToDevice, s));
    else
      CF_TRY(launch_occupancy(d, F->d_occ, (int)R, p->occ_threshold, s));
  }
  hipDeviceProp_t prop;
  CF_TRY(hipGetDeviceProperties(&prop, F->device));
  F->n_cu = prop.multiProcessorCount;
  F->fwd_blocks = F->n_cu * mlp_fwd_blocks_per_cu(d.lpg, d.mlp_f16);
  F->bwd_blocks = F->n_cu * mlp_bwd_blocks_per_cu(d.lpg, d.sh_dir_grad, d.mlp_f16);
  F->ray_blocks = F->n_cu * ray_bwd_blocks_per_cu(d.lpg, d.sh_dir_grad, d.mlp_f16);
  F->backward = p->backward;
  CF_TRY(hipMalloc(&F->d_queue, sizeof(uint32_t) * kMaxLevels * kQueueStride));
  F->enc_blocks = encode_blocks(d, F->n_cu, 8);
  F->enc_blocks_overlap = encode_blocks(d, F->n_cu, 4);  // leave room for the networks
  F->overlap_chunks = p->overlap_chunks == 0 ? kDefaultOverlapChunks : p->overlap_chunks;
  CF_TRY(hipStreamSynchronize(s));
#undef CF_TRY
  *out = F;
  return PNERF_OK;
}

void pnerf_destroy_field(pnerf_field* F) {
  if (!F) return;
  (void)hipSetDevice(F->device);
  (void)hipDeviceSynchronize();
  for (auto& pe : F->pending) {
    (void)hipEventDestroy(pe.a);
    (void)hipEventDestroy(pe.b);
  }
  for (hipEvent_t ev : F->ev_pool) (void)hipEventDestroy(ev);
  (void)hipFree(F->d_table);
  (void)hipFree(F->d_wfwd);
  (void)hipFree(F->d_wbwd);
  (void)hipFree(F->d_hfwd);
  (void)hipFree(F->d_hbwd);
  (void)hipFree(F->d_wc3);
  (void)hipFree(F->d_wd1);
  (void)hipFree(F->d_wd2);
  (void)hipFree(F->d_occ);
  (void)hipFree(F->d_rays);
  (void)hipFree(F->d_samp[0]);
  (void)hipFree(F->d_samp[1]);
  if (F->s_enc) (void)hipStreamDestroy(F->s_enc);
  if (F->s_mlp) (void)hipStreamDestroy(F->s_mlp);
  hipEvent_t evs[] = {F->ev_start, F->ev_enc[0], F->ev_enc[1], F->ev_mlp[0], F->ev_mlp[1],
                      F->ev_end_enc, F->ev_end_mlp};
  for (hipEvent_t e : evs)
    if (e) (void)hipEventDestroy(e);
  (void)hipFree(F->d_totals);
  (void)hipFree(F->d_queue);
  if (F->h_hyp) (void)hipHostFree(F->h_hyp);
  delete F;
}

pnerf_status pnerf_render_loss_grad(pnerf_field* F, int32_t K, const float* poses, int32_t P,
                                    const int32_t* pixel_ids, const float* observed,
                                    const pnerf_intrinsics* intr, float* loss, float* dpose,
                                    void* stream) {
  pnerf_status st = check_batch(F, K, poses, P, pixel_ids, intr);
  if (st != PNERF_OK) return st;
  if (!observed || !loss || !dpose) return fail(PNERF_ERR_INVALID_ARG, "NULL pointer argument");
  return run(F, kLossGrad, K, poses, P, pixel_ids, observed, intr, loss, dpose, nullptr, nullptr,
             nullptr, nullptr, 0, (hipStream_t)stream);
}

pnerf_status pnerf_render(pnerf_field* F, int32_t K, const float* poses, int32_t P,
                          const int32_t* pixel_ids, const pnerf_intrinsics* intr, float* rgb,
                          void* stream) {
  pnerf_status st = check_batch(F, K, poses, P, pixel_ids, intr);
  if (st != PNERF_OK) return st;
  if (!rgb) return fail(PNERF_ERR_INVALID_ARG, "NULL rgb");
  return run(F, kRender, K, poses, P, pixel_ids, nullptr, intr, nullptr, nullptr, rgb, nullptr,
             nullptr, nullptr, 0, (hipStream_t)stream);
}

pnerf_status pnerf_march(pnerf_field* F, int32_t K, const float* poses, int32_t P,
                         const int32_t* pixel_ids, const pnerf_intrinsics* intr,
                         int64_t* ray_offset, float* t, int32_t* lattice_j, int64_t capacity,
                         void* stream) {
  pnerf_status st = check_batch(F, K, poses, P, pixel_ids, intr);
  if (st != PNERF_OK) return st;
  if (!ray_offset) return fail(PNERF_ERR_INVALID_ARG, "NULL ray_offset");
  if (capacity < 0 || (capacity > 0 && (!t || !lattice_j)))
    return fail(PNERF_ERR_INVALID_ARG, "capacity > 0 needs t and lattice_j");
  return run(F, kMarch, K, poses, P, pixel_ids, nullptr, intr, nullptr, nullptr, nullptr,
             ray_offset, t, lattice_j, capacity, (hipStream_t)stream);
}

pnerf_status pnerf_step_momentum(int32_t K, float* poses, float* momentum, const float* dpose,
                                 float lr, float beta, void* stream) {
  if (K < 1) return fail(PNERF_ERR_INVALID_ARG, "K=%d", K);
  if (!poses || !momentum || !dpose) return fail(PNERF_ERR_INVALID_ARG, "NULL pointer argument");
  if (!std::isfinite(lr) || !std::isfinite(beta)) return fail(PNERF_ERR_INVALID_ARG, "lr/beta");
  HIP_TRY(launch_step_momentum(K, poses, momentum, dpose, lr, beta, (hipStream_t)stream));
  return PNERF_OK;
}

pnerf_status pnerf_step_adam(int32_t K, float* poses, float* state, const float* dpose,
                             int32_t step, const pnerf_adam_params* p, void* stream) {
  static_assert(PNERF_ADAM_STATE == kAdamState, "Adam state width");
  if (K < 1) return fail(PNERF_ERR_INVALID_ARG, "K=%d", K);
  if (!p) return fail(PNERF_ERR_INVALID_ARG, "NULL params");
  if (step < 0) return fail(PNERF_ERR_INVALID_ARG, "step=%d", step);
  if (!(std::isfinite(p->lr_rot) && p->lr_rot >= 0.0f && std::isfinite(p->lr_trans) &&
        p->lr_trans >= 0.0f))
    return fail(PNERF_ERR_INVALID_ARG, "learning rates must be finite and >= 0");
  if (!(p->beta1 >= 0.0f && p->beta1 < 1.0f && p->beta2 >= 0.0f && p->beta2 < 1.0f))
    return fail(PNERF_ERR_INVALID_ARG, "beta1/beta2 outside [0, 1)");
  if (!(std::isfinite(p->eps) && p->eps > 0.0f)) return fail(PNERF_ERR_INVALID_ARG, "eps");
  if (!(std::isfinite(p->decay_base) && p->decay_base > 0.0f) || p->decay_steps < 0)
    return fail(PNERF_ERR_INVALID_ARG, "decay_base/decay_steps");
  if ((p->staircase != 0 && p->staircase != 1) || (p->second_moment != 0 && p->second_moment != 1) ||
      (p->representation != 0 && p->representation != 1))
    return fail(PNERF_ERR_INVALID_ARG, "staircase/second_moment/representation must be 0 or 1");
  if (!poses || !state || !dpose) return fail(PNERF_ERR_INVALID_ARG, "NULL pointer argument");
  // Learning-rate decay of Sec. IV-D, evaluated once per call in double.
  double scale = 1.0;
  if (p->decay_steps > 0) {
    double e = p->staircase ? std::floor((double)step / (double)p->decay_steps)
                            : (double)step / (double)p->decay_steps;
    scale = std::pow((double)p->decay_base, e);
  }
  HIP_TRY(launch_step_adam(K, poses, state, dpose, (double)p->lr_rot * scale,
                           (double)p->lr_trans * scale, p->beta1, p->beta2, p->eps,
                           p->second_moment, p->representation, (hipStream_t)stream));
  return PNERF_OK;
}

pnerf_status pnerf_resample_hypotheses(int32_t K, float* poses, float* opt_state,
                                       int32_t state_dim, const float* loss, float keep_frac,
                                       float sigma_rot, float sigma_trans, uint64_t seed,
                                       uint32_t round_idx, void* stream) {
  if (K < 1 || K > 65535) return fail(PNERF_ERR_INVALID_ARG, "K=%d outside 1..65535", K);
  if (state_dim < 0 || state_dim > 64) return fail(PNERF_ERR_INVALID_ARG, "state_dim=%d", state_dim);
  if (!poses || !loss || (state_dim > 0 && !opt_state))
    return fail(PNERF_ERR_INVALID_ARG, "NULL pointer argument");
  if (!(keep_frac >= 0.0f && keep_frac <= 1.0f)) return fail(PNERF_ERR_INVALID_ARG, "keep_frac");
  if (!(sigma_rot >= 0.0f) || !(sigma_trans >= 0.0f)) return fail(PNERF_ERR_INVALID_ARG, "sigma");
  int n_keep = (int)std::floor((double)K * (double)keep_frac);
  n_keep = std::max(1, std::min(n_keep, K));
  hipStream_t s = (hipStream_t)stream;
  int32_t* scratch = nullptr;
  HIP_TRY(hipMallocAsync((void**)&scratch, sizeof(int32_t) * 2 * (size_t)K, s));
  hipError_t e = launch_resample(K, poses, opt_state, state_dim, loss, n_keep, sigma_rot,
                                 sigma_trans, seed, round_idx, scratch, s);
  hipError_t e2 = hipFreeAsync(scratch, s);
  if (e != hipSuccess) return fail(PNERF_ERR_DEVICE, "resample launch: %s", hipGetErrorString(e));
  HIP_TRY(e2);
  return PNERF_OK;
}

pnerf_status pnerf_resample_hypotheses_noalloc(int32_t K, float* poses, float* opt_state,
                                               int32_t state_dim, const float* loss,
                                               float keep_frac, float sigma_rot,
                                               float sigma_trans, uint64_t seed,
                                               uint32_t round_idx, void* stream) {
  if (K < 1) return fail(PNERF_ERR_INVALID_ARG, "K=%d must be >= 1", K);
  if (state_dim < 0 || state_dim > 64) return fail(PNERF_ERR_INVALID_ARG, "state_dim=%d", state_dim);
  if (!poses || !loss || (state_dim > 0 && !opt_state))
    return fail(PNERF_ERR_INVALID_ARG, "NULL pointer argument");
  if (!(keep_frac >= 0.0f && keep_frac <= 1.0f)) return fail(PNERF_ERR_INVALID_ARG, "keep_frac");
  if (!(sigma_rot >= 0.0f) || !(sigma_trans >= 0.0f)) return fail(PNERF_ERR_INVALID_ARG, "sigma");
  int device = 0;
  HIP_TRY(hipGetDevice(&device));
  int32_t* scratch = nullptr;
  int max_k = 0;
  HIP_TRY(resample_scratch(device, &scratch, &max_k));
  if (K > max_k)
    return fail(PNERF_ERR_CAPACITY, "K=%d exceeds the %d hypotheses the static scratch holds", K,
                max_k);
  int n_keep = (int)std::floor((double)K * (double)keep_frac);
  n_keep = std::max(1, std::min(n_keep, K));
  // every rank[i] and by_rank[r], i, r < K, is written before it is read:
  // nothing left from an earlier call is used
  HIP_TRY(launch_resample(K, poses, opt_state, state_dim, loss, n_keep, sigma_rot, sigma_trans,
                          seed, round_idx, scratch, (hipStream_t)stream));
  return PNERF_OK;
}

pnerf_status pnerf_field_inspect(pnerf_field* F, int32_t what, float* dst, int64_t n,
                                 void* stream) {
  if (!F || !dst) return fail(PNERF_ERR_INVALID_ARG, "NULL argument");
  if (what < 0 || what > 3) return fail(PNERF_ERR_INVALID_ARG, "what=%d", what);
  if (!F->d_samp[0] || n < 0 || n > F->samp_cap) return fail(PNERF_ERR_INVALID_ARG, "n=%lld", (long long)n);
  if (F->last_chunks != 1) return fail(PNERF_ERR_INVALID_ARG, "last call used %d chunks", F->last_chunks);
  if (what > 0 && !F->last_keeps_samples)
    return fail(PNERF_ERR_INVALID_ARG,
                "the last loss gradient kept no per-sample intermediates (backward = 1)");
  DevWork w{};
  carve_samples(F->dev, F->samp_cap, &w, (char*)F->d_samp[0]);
  w.total = F->d_totals;  // the single chunk of the last call
  HIP_TRY(launch_inspect(F->dev, DevBatch{}, w, what, dst, n, (hipStream_t)stream));
  return PNERF_OK;
}

pnerf_status pnerf_field_occupancy(pnerf_field* F, uint32_t* bits_host, void* stream) {
  if (!F || !bits_host) return fail(PNERF_ERR_INVALID_ARG, "NULL argument");
  if (!F->d_occ) return fail(PNERF_ERR_INVALID_ARG, "field has no occupancy grid");
  hipStream_t s = (hipStream_t)stream;
  HIP_TRY(hipMemcpyAsync(bits_host, F->d_occ, F->occ_words * 4, hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  return PNERF_OK;
}

pnerf_status pnerf_field_last_sample_count(pnerf_field* F, int64_t* count, void* stream) {
  if (!F || !count) return fail(PNERF_ERR_INVALID_ARG, "NULL argument");
  if (F->last_total_dev) {  // the call sized its buffer for the worst case: read the total
    int32_t n = 0;
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(hipMemcpyAsync(&n, F->last_total_dev, sizeof(int32_t), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    *count = n;
    return PNERF_OK;
  }
  *count = F->last_total;  // counted on the host when the call planned its chunks
  return PNERF_OK;
}

pnerf_status pnerf_field_set_profiling(pnerf_field* F, int32_t enable) {
  if (!F) return fail(PNERF_ERR_INVALID_ARG, "NULL field");
  pnerf_status st = resolve_profile(F);
  if (st != PNERF_OK) return st;
  if (enable) {
    F->stats.clear();
    // events for the first launches, made before any is timed
    HIP_TRY(hipSetDevice(F->device));
    while (F->ev_pool.size() < 512) {
      hipEvent_t ev;
      HIP_TRY(hipEventCreate(&ev));
      F->ev_pool.push_back(ev);
    }
  }
  F->profiling = enable != 0;
  return PNERF_OK;
}

pnerf_status pnerf_field_profile_read(pnerf_field* F, int32_t index, const char** name,
                                      int64_t* launches, double* total_ms) {
  if (!F) return fail(PNERF_ERR_INVALID_ARG, "NULL field");
  pnerf_status st = resolve_profile(F);
  if (st != PNERF_OK) return st;
  if (index < 0 || index >= (int32_t)F->stats.size())
    return fail(PNERF_ERR_INVALID_ARG, "profile index %d past the end", index);
  if (name) *name = F->stats[index].name.c_str();
  if (launches) *launches = F->stats[index].launches;
  if (total_ms) *total_ms = F->stats[index].total_ms;
  return PNERF_OK;
}

}  // extern "C"
