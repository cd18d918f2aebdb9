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
  kNumGemmCfg = 10
};
int gemm_tile_m(int cfg);
int gemm_tile_n(int cfg);
int gemm_tile_k(int cfg, bool bf16);

// fp32 operands. vec: 16-byte loads/stores (the host has checked that every
// contiguous extent, pitch, batch stride and base allows them); else 4-byte.
hipError_t gemm_f32(const GemmParams& p, bool a_kc, bool b_kc, bool vec, int cfg,
                    hipStream_t stream);
// bf16 operands (fp32 accumulation, bias and output). vec: 16-byte loads
// (8 elements) and 16-byte stores; else 2-byte loads and 4-byte stores.
hipError_t gemm_bf16(const GemmParams& p, bool a_kc, bool b_kc, bool vec, int cfg,
                     hipStream_t stream);

// Split-K finish: C[m][n] (+)= sum_s partial[s][m][n] (+ bias[n]), s ascending.
hipError_t splitk_finish(const float* partial, int splits, int64_t M, int64_t N, float* c,
                         int64_t ldc, const float* bias, bool accumulate, hipStream_t stream);

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

}  // namespace mt
