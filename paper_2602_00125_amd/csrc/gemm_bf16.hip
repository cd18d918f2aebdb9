// bf16 instantiations of the matrix-core GEMM (see gemm_kernel.hpp):
// v_mfma_f32_32x32x16_bf16 (exact bf16 products, fp32 accumulation), BK = 32,
// 16-byte (VEC = 8) or 2-byte (VEC = 1) loads; fp32 bias and output.
#include "gemm_dma.hpp"
#include "gemm_kernel.hpp"
#include "kernels.hpp"

namespace mt {

template <bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int VEC, int WPE>
static hipError_t launch_bf16(const GemmParams& p, hipStream_t stream) {
  GemmParams q = p;
  q.tiles_m = (int32_t)((p.M + BM - 1) / BM);
  q.tiles_n = (int32_t)((p.N + BN - 1) / BN);
  const int64_t blocks = (int64_t)q.tiles_m * q.tiles_n * p.keep_count * p.splits;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((gemm::gemm_kernel<__bf16, A_KC, B_KC, BM, BN, BK, WGM, WGN, VEC, WPE>),
                     dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, stream, q);
  return hipGetLastError();
}

template <bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int NS, int WPE>
static hipError_t launch_dma(const GemmParams& p, hipStream_t stream) {
  GemmParams q = p;
  q.tiles_m = (int32_t)((p.M + BM - 1) / BM);
  q.tiles_n = (int32_t)((p.N + BN - 1) / BN);
  const int64_t blocks = (int64_t)q.tiles_m * q.tiles_n * p.keep_count * p.splits;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  // the per-load K-tail test only where K is not a whole number of stages
  if (p.K % BK != 0)
    hipLaunchKernelGGL((gemm::gemm_dma_kernel<__bf16, A_KC, B_KC, BM, BN, BK, WGM, WGN, NS, 1, 1, true, WPE>),
                       dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, stream, q);
  else
    hipLaunchKernelGGL((gemm::gemm_dma_kernel<__bf16, A_KC, B_KC, BM, BN, BK, WGM, WGN, NS, 1, 1, false, WPE>),
                       dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, stream, q);
  return hipGetLastError();
}

template <bool A_KC, bool B_KC, int VEC>
static hipError_t launch_layout(const GemmParams& p, int cfg, hipStream_t stream) {
  if constexpr (VEC == 1) {
    // element-load kernels exist up to 128x128 (larger tiles would spill staging registers)
    if (cfg == kCfg64x64) return launch_bf16<A_KC, B_KC, 64, 64, 32, 2, 2, 1, 4>(p, stream);
    return launch_bf16<A_KC, B_KC, 128, 128, 32, 2, 2, 1, 2>(p, stream);
  } else {
    switch (cfg) {
      case kCfg256x256: return launch_bf16<A_KC, B_KC, 256, 256, 32, 2, 2, VEC, 1>(p, stream);
      case kCfg256x256x64w8: return launch_bf16<A_KC, B_KC, 256, 256, 64, 2, 4, VEC, 2>(p, stream);
      case kCfgDma256x256: return launch_dma<A_KC, B_KC, 256, 256, 64, 2, 4, 2, 2>(p, stream);
      case kCfgDma256x256w4: return launch_dma<A_KC, B_KC, 256, 256, 64, 2, 2, 2, 1>(p, stream);
      case kCfgDma256x128: return launch_dma<A_KC, B_KC, 256, 128, 32, 2, 2, 3, 2>(p, stream);
      case kCfgDma128x256: return launch_dma<A_KC, B_KC, 128, 256, 32, 2, 2, 3, 2>(p, stream);
      case kCfg256x128: return launch_bf16<A_KC, B_KC, 256, 128, 32, 2, 2, VEC, 2>(p, stream);
      case kCfg128x256: return launch_bf16<A_KC, B_KC, 128, 256, 32, 2, 2, VEC, 2>(p, stream);
      case kCfg128x128: return launch_bf16<A_KC, B_KC, 128, 128, 32, 2, 2, VEC, 2>(p, stream);
      default: return launch_bf16<A_KC, B_KC, 64, 64, 32, 2, 2, VEC, 4>(p, stream);
    }
  }
}

hipError_t gemm_bf16(const GemmParams& p, bool a_kc, bool b_kc, bool vec, int cfg,
                     hipStream_t stream) {
  if (vec) {
    if (a_kc && b_kc) return launch_layout<true, true, 8>(p, cfg, stream);
    if (a_kc && !b_kc) return launch_layout<true, false, 8>(p, cfg, stream);
    if (!a_kc && b_kc) return launch_layout<false, true, 8>(p, cfg, stream);
    return launch_layout<false, false, 8>(p, cfg, stream);
  }
  if (a_kc && b_kc) return launch_layout<true, true, 1>(p, cfg, stream);
  if (a_kc && !b_kc) return launch_layout<true, false, 1>(p, cfg, stream);
  if (!a_kc && b_kc) return launch_layout<false, true, 1>(p, cfg, stream);
  return launch_layout<false, false, 1>(p, cfg, stream);
}

}  // namespace mt
