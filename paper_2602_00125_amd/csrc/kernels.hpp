// Kernel entry points of libminitensor_hip (device code in *.hip files).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

#include "gemm_params.hpp"

namespace mt {

// GEMM tile configurations: register-staged tiles (BM x BN; BK = 16 fp32 /
// 32 bf16; 4 waves per block), a register-staged 256x256 tile with 8 waves
// and BK = 32 fp32 / 64 bf16, and tiles whose operands stream straight into
// an LDS ring (gemm_dma.hpp).
enum GemmCfg {
  kCfg256x256 = 0,
  kCfg256x128 = 1,
  kCfg128x256 = 2,
  kCfg128x128 = 3,
  kCfg64x64 = 4,
  kCfg256x256x64w8 = 5,
  kCfgDma256x256 = 6,    // 256x256, 8 waves, BK = 32 / 64, 2-stage ring (128 KB), 1 block per CU
  kCfgDma256x256w4 = 7,  // the same with 4 waves (128x128 per wave)
  kCfgDma256x128 = 8,    // 256x128, 4 waves, BK = 16 / 32, 3-stage ring (72 KB), 2 blocks per CU
  kCfgDma128x256 = 9,    // 128x256, likewise
  kCfgDma128x128 = 10,   // 128x128, 4 waves, BK = 32 / 64, 2-stage ring (64 KB), 2 blocks per CU
  kCfgDma128x128w8 = 11, // the same tile with 8 waves (fp32: 64x32 each; bf16: 32x64)
  kCfgDma128x128k64 = 12, // fp32 only: 128x128, 8 waves of 64x32, BK = 64, 2-stage ring (128 KB), 1 block per CU
  // fp32 operands without 16-byte aligned rows (4-byte lanes), tiles shaped
  // for dimensions just past a multiple of 128 or 256 (every wave 64x96):
  kCfgDma256x192 = 13,   // 8 waves, BK = 16, 4-stage ring (112 KB), 1 block per CU
  kCfgDma256x96 = 14,    // 4 waves, BK = 16, 3-stage ring (66 KB), 2 blocks per CU; B K-contiguous
  kCfgDma64x384 = 15,    // 4 waves, BK = 16, 2-stage ring (56 KB), 2 blocks per CU
  kNumGemmCfg = 16
};
int gemm_tile_m(int cfg);
int gemm_tile_n(int cfg);
int gemm_tile_k(int cfg, bool bf16);

// fp32 operands. vec: 16-byte loads/stores (the host has checked that every
// contiguous extent, pitch, batch stride and base allows them); else 4-byte.
hipError_t gemm_f32(const GemmParams& p, bool a_kc, bool b_kc, bool vec, int cfg,
                    hipStream_t stream);
// Convolution products with an operand gathered by the loads (p.cg): mode 1
// the forward (A = unfolded input, NT; K a multiple of 32), mode 2 the weight
// gradient (B = unfolded input, TN), mode 3 the input gradient of a stride-1
// convolution (A = dY unfolded over the mirrored taps, B = the weights tap by
// tap, NN; K a multiple of 32), mode 4 one sub-pixel phase of a strided
// convolution's input gradient (no split: its rows go straight to dx). fp32, 16-byte loads and stores, on the
// DMA tiles 256x256 (cfg 6) and 128x128 (cfg 10, 11) only.
hipError_t gemm_f32_conv(const GemmParams& p, int mode, int cfg, hipStream_t stream);
// The same products of modes 1 and 3 on the 256x256 tile in stream-K order
// over `blocks` blocks (p.partial: sk_max_segments x M x N floats, pitch N,
// p.partial_stride = M N), then the fixed-order sum of the cut tiles.
hipError_t gemm_f32_conv_sk(const GemmParams& p, int mode, int blocks, hipStream_t stream);
int64_t sk_max_segments(int64_t tiles, int64_t ks, int64_t blocks);
// All sub-pixel phases of a strided input gradient (mode 4) in one launch on
// the 256x256 tile: phase k computes tiles tile0[k] .. tile0[k+1]-1.
hipError_t gemm_f32_conv_phases(const GemmParams& p, const ConvPhases& tab, hipStream_t stream);
bool gemm_conv_cfg(int cfg);
// bf16 operands (fp32 accumulation, bias and output). vec: 16-byte loads
// (8 elements) and 16-byte stores; else 2-byte loads and 4-byte stores.
hipError_t gemm_bf16(const GemmParams& p, bool a_kc, bool b_kc, bool vec, int cfg,
                     hipStream_t stream);

// Split-K finish: C[m][n] (+)= sum_s partial[s][m][n] (+ bias[n]), s ascending.
// With cs_part (the runs' column sums of A, splits x M floats), also
// cs_out[m] (+)= sum_s cs_part[s][m], s ascending (in the same launch where
// the 16-byte form runs).
hipError_t splitk_finish(const float* partial, int splits, int64_t M, int64_t N, float* c,
                         int64_t ldc, const float* bias, bool accumulate, hipStream_t stream,
                         const float* cs_part = nullptr, float* cs_out = nullptr);

// Column sums over the outer axis of a row-major [M][N] matrix with row pitch
// ld: out[n] (+)= sum_m x[m][n]. x is f32 or bf16 (is_bf16). With ws (room for
// `parts` x N floats) the rows are split into `parts` slices summed in a
// second, fixed-order pass; parts == 1 needs no workspace.
hipError_t colsum(const void* x, bool is_bf16, int64_t M, int64_t N, int64_t ld, float* out,
                  bool accumulate, float* ws, int parts, hipStream_t stream);
int colsum_parts(int64_t M, int64_t N);

// Sum of a strided tensor over some of its axes into a contiguous output.
struct ReducePlan {
  int32_t nkeep, nred;
  int64_t keep_shape[8], keep_stride[8];
  int64_t red_shape[8], red_stride[8];
  int64_t keep_count, red_count;
};
hipError_t reduce_strided(const float* x, const ReducePlan& plan, float* out, bool accumulate,
                          float* ws, int parts, hipStream_t stream);
int reduce_parts(const ReducePlan& plan);

// out[i] = value (i < n), a small fill kernel (used instead of hipMemsetAsync).
hipError_t fill_f32(float* out, int64_t n, float value, hipStream_t stream);

// out[n] (+)= sum_p ws[p][n] over p = 0 .. parts-1 in order (second pass of
// the row-sliced column sums).
hipError_t parts_finish(const float* ws, int parts, int64_t N, float* out, bool accumulate,
                        hipStream_t stream);

// Pullback of H = act(Z) for row-major [M][N] matrices with row pitches:
// dz (+)= dh * act'(z) (dh and dz f32, or both bf16: dz rounded to nearest
// even), and, when db is given, db[n] (+)= sum_m dh * act'(z) of the fp32
// terms. ws: room for `parts` x N floats (row slices, fixed-order second
// pass); parts = 1 needs none.
hipError_t act_bwd(int act, const float* z, int64_t ldz, const void* dh, int64_t ldh, void* dz,
                   int64_t ldd, bool is_bf16, int64_t M, int64_t N, bool acc_dz, float* db,
                   bool acc_db, float* ws, int parts, hipStream_t stream);

// Mean squared error over n contiguous fp32 elements: *loss = sum (p - t)^2 / n
// (nullable), dp = 2 (p - t) / n (nullable). ws: room for `parts` floats
// (block partials added in order by a second pass); parts = 1 needs none.
hipError_t mse(const float* p, const float* t, int64_t n, float* dp, float* loss, float* ws,
               int parts, hipStream_t stream);
int mse_parts(int64_t n);

// Geometry of a 2-D convolution (Sec. 3.3 Eq. (6)) in its unfolded form:
// rows m = (n, i, j) over the output pixels, columns k over the taps.
struct ConvGeom {
  int32_t N, C, H, W, CO, KH, KW, sh, sw, ph, pw, HO, WO;
  int32_t korder_uvc;  // 1: column k = (u, v, c), c fastest; 0: k = (c, u, v)
  int32_t dx_vec;      // fold: dx channels contiguous and 16-byte aligned pixels
  int64_t Kc, Kcp;     // columns of the unfolded matrix, and its row pitch (a multiple of 4)
  int64_t xs[4];       // element strides of x (n, c, h, w)
  int64_t ds[4];       // element strides of dx (n, c, h, w)
};
// col[m][k] = x at tap k of output pixel m (0 outside the image; columns
// Kc .. Kcp-1 are 0). col: 16-byte aligned, N HO WO rows of pitch Kcp.
hipError_t conv_unfold(const float* x, const ConvGeom& g, float* col, hipStream_t stream);
// dx (+)= the fold of dcol (rows of pitch Kcp) onto the image.
hipError_t conv_fold(const float* dcol, const ConvGeom& g, float* dx, bool accumulate,
                     hipStream_t stream);

// Up to kOptMaxTensors contiguous fp32 parameter tensors updated in one launch.
constexpr int kOptMaxTensors = 32;
struct OptBatch {
  int32_t n;
  float* param[kOptMaxTensors];
  const float* grad[kOptMaxTensors];
  float* state1[kOptMaxTensors];  // SGD velocity, Adam first moment, RMSprop average
  float* state2[kOptMaxTensors];  // Adam second moment
  int64_t numel[kOptMaxTensors];
  int64_t block_start[kOptMaxTensors + 1];  // filled by the launcher
  int8_t vec[kOptMaxTensors];               // every pointer of the tensor 16-byte aligned
};
hipError_t sgd_step(const OptBatch& b, float lr, float momentum, float weight_decay,
                    hipStream_t stream);
hipError_t adam_step(const OptBatch& b, float lr, float beta1, float beta2, float eps,
                     float inv_bc1, float inv_bc2, hipStream_t stream);
hipError_t rmsprop_step(const OptBatch& b, float lr, float alpha, float eps, hipStream_t stream);

}  // namespace mt
