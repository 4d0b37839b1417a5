// Internal declarations of the HIP implementation (gfx950 / CDNA4).
// Device-side views of a field, of one batch chunk and of its workspace, plus
// the host launchers each kernel source file exports.
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

namespace pnerf {

constexpr int kMaxLevels = 16;
constexpr int kHidden = 64;
constexpr int kTile = 64;          // granule of the per-sample capacity (a multiple of every kernel's tile)
constexpr int kMaskWords = 8;      // ReLU-mask words per lane per 64 samples (2 per 16-sample column)
constexpr int kQueueStride = 32;   // uint32 words between the encoding's work-queue counters (one cache line)
constexpr int kMaxLatticeCandidates = 1 << 20;  // bound on lattice points tested per ray
constexpr int kMaxScanBlocks = 8192;  // offset scan: at most 8192 x 256 rays per counted batch
constexpr int kMaxRawScanBlocks = 64;  // block sums the write pass may scan itself (one wavefront)
constexpr int64_t kMaxCountedSamples = ((int64_t)1 << 31) - 1;  // int32 counts of a counted batch
constexpr int kDefaultOverlapChunks = 1;   // loss-gradient chunks pipelined over two streams (1 = off)
constexpr int kMinOverlapSamples = 1 << 16;  // smaller batches run as one chunk
constexpr int64_t kDeviceSizedBytes = (int64_t)16 << 30;  // worst-case sample buffer a loss
                                                           // gradient may allocate to skip the
                                                           // host's read of the sample totals
constexpr int kReduceParts = 64;      // parts per hypothesis of the reduction (lanes of one wave)
constexpr int kAdamState = 16;        // Adam state floats per hypothesis: m[6], v[6], n, 3 pads

// A operand of one (row tile, K step) of v_mfma_f32_16x16x32_bf16: 8 bf16
// values per lane, as a high part and the low part of the fp32 weight (for
// v_mfma_f32_16x16x32_f16 the two parts are fp16).  Lane
// l = 16 g + r supplies row r and K positions 8g .. 8g+7.
struct alignas(16) WeightUnit {
  uint4 hi[64];
  uint4 lo[64];
};

// unit indices of the forward tiles: density layer 1 (4 row tiles), layer 2
// (2 K steps), colour layer 1 (4 row tiles), layer 2 (4 x 2), layer 3 (2 K steps)
constexpr int kFD1 = 0, kFD2 = 4, kFC1 = 6, kFC2 = 10, kFC3 = 18, kFwdUnits = 20;
// backward (transposed layers): colour 2 (4 x 2), colour 1 h rows (2 K steps),
// density 2 (4 row tiles), density 1 (up to 2 row tiles x 2 K steps), then
// colour 1 SH rows (2 K steps; staged only when the direction path is on)
constexpr int kBC2 = 0, kBC1 = 8, kBD2 = 10, kBD1 = 14, kBSH = 18, kBwdUnits = 20;

// ---------------------------------------------------- wavefront primitives
// Cross-lane data movement through DPP (data-parallel primitives of the
// vector ALU) instead of the LDS crossbar that __shfl goes through.

// Real spherical harmonics of degree 0..3 (16 functions, no Condon-Shortley
// phase) of the unit direction d: the colour network's view-direction input.
__device__ inline void sh16(const float d[3], float v[16]) {
  const float x = d[0], y = d[1], z = d[2];
  const float C0 = 0.28209479177387814f, C1 = 0.4886025119029199f;
  const float C2a = 1.0925484305920792f, C2b = 0.31539156525252005f, C2c = 0.5462742152960396f;
  const float C3a = 0.5900435899266435f, C3b = 2.890611442640554f, C3c = 0.4570457994644658f;
  const float C3d = 0.3731763325901154f, C3e = 1.445305721320277f;
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
}

// The value of the partner lane (lane ^ 1).  Both lanes must be active.
__device__ __forceinline__ float lane_pair_swap(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1 /* quad_perm
                                                    [1,0,3,2] */, 0xF, 0xF, false));
}

// Inclusive prefix sum over the 64 lanes of a wavefront, all lanes active:
// shifts by 1, 2, 4, 8 within each row of 16, then the last lane of row 0 (2)
// into row 1 (3), and of row 1 into rows 2 and 3.  Fixed order.
__device__ __forceinline__ float wave_incl_scan(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x111, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x112, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x114, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x118, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x142, 0xA, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x143, 0xC, 0xF, false));
  return x;
}

// x of lane `lane` (uniform across the wavefront) in every lane.
__device__ __forceinline__ float lane_value(float x, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), lane));
}

struct DevField {
  int32_t L, lpg;               // levels, levels per lane group (L / 4)
  uint32_t T;                   // table entries per level (power of two)
  int32_t res[kMaxLevels];
  uint32_t dense[kMaxLevels];   // 1: vertex index i + j n1 + k n1^2
  uint32_t n1[kMaxLevels];      // res + 1
  int32_t f16;                  // table stored as fp16
  int32_t q_level[kMaxLevels];  // level served by encoding work queue q (hashed levels first)
  const float* table32;         // [L][T][2]
  const __half* table16;        // [L][T][2]
  const WeightUnit* wfwd;       // forward A-operand tiles [kFwdUnits]
  const WeightUnit* wbwd;       // backward A-operand tiles [kBwdUnits]
  const WeightUnit* hfwd;       // the same tiles for v_mfma_f32_16x16x32_f16: fp16 hi
  const WeightUnit* hbwd;       // and lo parts (mlp_precision 1)
  int32_t mlp_f16;              // network arithmetic: 0 split bf16 (3 products), 1 fp16
  const float* wc3;             // W_c3 [64][3] (fp32, transposed colour layer 3)
  const float* wd1;             // plain W_d1 [2L][64] and W_d2 [64][16] (occupancy build)
  const float* wd2;
  float density_bias;
  uint32_t bf16_neg1[2];        // bf16 pairs (-1, 0) and (0, -1): the MLP kernels' split
                                // multipliers, read as data (see split2 in mlp.hip)
  float mn[3], mx[3], inv_ext[3];
  float inv_ext_err[3];         // inv_ext * extent - 1 (relative rounding of the reciprocal)
  int32_t march_mode, n_uniform;
  float step;
  int32_t max_samples;
  float t_stop;
  int32_t occ_res;
  const uint32_t* occ;
  float bg[3];
  int32_t loss_type;
  float loss_param;
  int32_t sh_dir_grad;
  int32_t max_per_ray;          // hard cap on kept samples per ray (buffer bound)
};

struct DevBatch {
  int32_t K, P, n_rays;         // hypotheses, pixels per hypothesis, K*P (this chunk)
  const float* poses;           // [K][12]
  const int32_t* pix;           // [K][P]
  const float* obs;             // [H][W][3]
  int32_t W, H;
  float fx, fy, cx, cy;
};

struct DevWork {
  // per ray (SoA)
  float *rdx, *rdy, *rdz, *rtn, *rtf, *rdelta;
  float *rex, *rey, *rez;       // direction correction: exact unit direction - (rdx, rdy, rdz)
  float* rsh;                   // [n_rays][16] SH basis of each ray's direction (sh16)
  int32_t* count;               // kept samples per ray
  int32_t* off;                 // counted batch: offset inside each 256-ray block;
                                // sample chunk: [n_rays + 1] exclusive offsets
  int32_t* blocksum;            // per 256-ray block (exclusive, after the scan)
  int32_t* hyp_total;           // [K] samples of every hypothesis of the counted batch
  int32_t* total;               // device scalar: samples of the counted batch / the chunk
  float* ray_loss;              // [n_rays]
  float* partial;               // [K][parts][7] per-hypothesis partial sums
  float* ray_terms;             // [n_rays][7] fused backward: each ray's torque, force, loss
  // per sample
  float* t;
  int32_t* sray;                // ray of each sample
  float* sig;                   // sigma (forward) -> d loss / d h0 (after composite)
  float *cr, *cg, *cb;          // colour (forward) -> d loss / d z (after composite)
  uint32_t* masks;              // [column tiles of 16][2][64] ReLU masks
  float* feat;                  // [2L][cap] features; after the backward rows 0..5 = torque, force
  __half* jac;                  // [6L][cap] d feature / d pos: 12-byte records per sample and
                                // level in 32-sample blocks (jac_record in encode.hip)
  int64_t cap;                  // sample capacity (row stride of feat and jac)
  uint32_t* queue;              // [kMaxLevels * kQueueStride] encoding work-queue counters
                                // (word q * kQueueStride: items of queue q taken), zeroed by
                                // k_ray_write before every encoding of the chunk
};

// ---- launchers (all enqueue on `s`, no synchronisation)
// raw_ok: the caller lets the write pass scan up to kMaxRawScanBlocks raw block
// sums itself; returns (in *raw_blocks) how many it left raw (0: scanned here)
hipError_t launch_march_count(const DevField& f, const DevBatch& b, const DevWork& w, bool raw_ok,
                              int* raw_blocks, hipStream_t s);
hipError_t launch_march_write(const DevField& f, const DevBatch& b, const DevWork& wb,
                              const DevWork& wc, int ray_base, int sample_base, int chunk_total,
                              int raw_blocks, int32_t* lattice_j_out, hipStream_t s);
hipError_t launch_encode(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                         int with_grad, hipStream_t s);
hipError_t launch_mlp_fwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                          int with_grad, hipStream_t s);
hipError_t launch_composite(const DevField& f, const DevBatch& b, const DevWork& w, int with_grad,
                            float* rgb_out, hipStream_t s);
hipError_t launch_mlp_bwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                          hipStream_t s);
hipError_t launch_reduce(const DevField& f, const DevBatch& b, const DevWork& w, float* loss,
                         float* dpose, hipStream_t s);
// The fused per-ray backward (composite, loss, network backward, each ray's
// torque and force) and the per-hypothesis sums of its per-ray terms.  keep:
// also store the per-sample intermediates the separate kernels leave.
hipError_t launch_ray_bwd(const DevField& f, const DevBatch& b, const DevWork& w, int n_blocks,
                          int keep, hipStream_t s);
hipError_t launch_reduce_rays(const DevBatch& b, const DevWork& w, float* loss, float* dpose,
                              hipStream_t s);
hipError_t launch_occupancy(const DevField& f, uint32_t* bits, int R, float thr, hipStream_t s);
hipError_t launch_copy_samples(const float* t, const int32_t* j, float* t_out, int32_t* j_out,
                               int64_t n, hipStream_t s);
hipError_t launch_inspect(const DevField& f, const DevBatch& b, const DevWork& w, int what,
                          float* dst, int64_t n, hipStream_t s);
hipError_t launch_offsets_i64(const int32_t* off, int64_t* out, int n, int64_t base, hipStream_t s);
hipError_t launch_step_momentum(int K, float* poses, float* mom, const float* dpose, float lr,
                                float beta, hipStream_t s);
hipError_t launch_step_adam(int K, float* poses, float* state, const float* dpose, double lr_r,
                            double lr_t, double b1, double b2, double eps, int per_subspace,
                            int twist, hipStream_t s);
hipError_t launch_resample(int K, float* poses, float* state, int state_dim, const float* loss,
                           int n_keep, float sr, float st, uint64_t seed, uint32_t round,
                           int32_t* scratch, hipStream_t s);

// The device address of the static resampling scratch on `device` (which must
// be current): 2 * max_k int32 words, looked up once per device.
hipError_t resample_scratch(int device, int32_t** ptr, int* max_k);

int reduce_parts(int K);
int mlp_fwd_blocks_per_cu(int lpg, int f16);
int mlp_bwd_blocks_per_cu(int lpg, int sh_dir_grad, int f16);
int ray_bwd_blocks_per_cu(int lpg, int sh_dir_grad, int f16);
int encode_blocks(const DevField& f, int n_cu, int per_cu);

}  // namespace pnerf
