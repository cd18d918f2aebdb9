// bf16 instantiations of the matrix-core GEMM (see gemm_kernel.hpp):
// v_mfma_f32_32x32x16_bf16 (exact bf16 products, fp32 accumulation), BK = 32,
// 16-byte (VEC = 8) or 2-byte (VEC = 1) loads; fp32 bias and output.
#include "gemm_dma.hpp"
#include "gemm_kernel.hpp"
#include "kernels.hpp"

namespace mt {

template <bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int VEC, int WPE,
          bool EPI = false>
static hipError_t launch_bf16(const GemmParams& p, hipStream_t stream) {
  GemmParams q = p;
  q.tiles_m = (int32_t)((p.M + BM - 1) / BM);
  q.tiles_n = (int32_t)((p.N + BN - 1) / BN);
  const int64_t blocks = (int64_t)q.tiles_m * q.tiles_n * p.keep_count * p.splits;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((gemm::gemm_kernel<__bf16, A_KC, B_KC, BM, BN, BK, WGM, WGN, VEC, WPE, EPI>),
                     dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, stream, q);
  return hipGetLastError();
}

template <bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int NS, int WPE,
          bool EPI = false>
static hipError_t launch_dma(const GemmParams& p, hipStream_t stream) {
  GemmParams q = p;
  q.tiles_m = (int32_t)((p.M + BM - 1) / BM);
  q.tiles_n = (int32_t)((p.N + BN - 1) / BN);
  const int64_t blocks = (int64_t)q.tiles_m * q.tiles_n * p.keep_count * p.splits;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  // persistent grid (host decides: plain product, more tiles than CUs)
  if constexpr (BM == 256 && BN == 256 && !EPI) {
    if (p.persist > 0 && p.K % BK == 0 && blocks > p.persist) {
      // products with a K-contiguous A take the ring of five half-slots (the
      // A and B tiles of a stage loaded in different halves of the stage
      // before: forward +2%, dX +0.3% against the two-stage ring); the TN
      // product keeps the two-stage ring (3% slower on the half-slots)
      constexpr int NSP = A_KC ? 5 : NS;
      hipLaunchKernelGGL((gemm::gemm_dma_kernel<__bf16, A_KC, B_KC, BM, BN, BK, WGM, WGN, NSP, 1, 1, false, WPE,
                                                false, 16, true, true>),
                         dim3((unsigned)p.persist), dim3(WGM * WGN * 64), 0, stream, q);
      return hipGetLastError();
    }
  }
  // the per-load K-tail test only where K is not a whole number of stages
  if (p.K % BK != 0)
    hipLaunchKernelGGL((gemm::gemm_dma_kernel<__bf16, A_KC, B_KC, BM, BN, BK, WGM, WGN, NS, 1, 1, true, WPE, EPI>),
                       dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, stream, q);
  else
    hipLaunchKernelGGL((gemm::gemm_dma_kernel<__bf16, A_KC, B_KC, BM, BN, BK, WGM, WGN, NS, 1, 1, false, WPE, EPI>),
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
      case kCfgDma128x128: return launch_dma<A_KC, B_KC, 128, 128, 64, 2, 2, 2, 2>(p, stream);
      case kCfgDma128x128w8: return launch_dma<A_KC, B_KC, 128, 128, 64, 4, 2, 2, 4>(p, stream);
      case kCfg256x128: return launch_bf16<A_KC, B_KC, 256, 128, 32, 2, 2, VEC, 2>(p, stream);
      case kCfg128x256: return launch_bf16<A_KC, B_KC, 128, 256, 32, 2, 2, VEC, 2>(p, stream);
      case kCfg128x128: return launch_bf16<A_KC, B_KC, 128, 128, 32, 2, 2, VEC, 2>(p, stream);
      default: return launch_bf16<A_KC, B_KC, 64, 64, 32, 2, 2, VEC, 4>(p, stream);
    }
  }
}

// The dense layer followed by a nonlinearity (z / act set): the forward
// layout only, on the 256x256 or 128x128 DMA tiles or the 128x128 / 64x64
// register-staged tiles.
static hipError_t launch_epi(const GemmParams& p, bool vec, int cfg, hipStream_t stream) {
  if (vec) {
    if (cfg == kCfgDma128x128)
      return launch_dma<true, true, 128, 128, 64, 2, 2, 2, 2, true>(p, stream);
    if (cfg == kCfgDma256x256)
      return launch_dma<true, true, 256, 256, 64, 2, 4, 2, 2, true>(p, stream);
    if (cfg == kCfg128x128) return launch_bf16<true, true, 128, 128, 32, 2, 2, 8, 2, true>(p, stream);
    return launch_bf16<true, true, 64, 64, 32, 2, 2, 8, 4, true>(p, stream);
  }
  if (cfg == kCfg128x128) return launch_bf16<true, true, 128, 128, 32, 2, 2, 1, 2, true>(p, stream);
  return launch_bf16<true, true, 64, 64, 32, 2, 2, 1, 4, true>(p, stream);
}

hipError_t gemm_bf16(const GemmParams& p, bool a_kc, bool b_kc, bool vec, int cfg,
                     hipStream_t stream) {
  if (p.act || p.z) {
    if (!a_kc || !b_kc) return hipErrorInvalidValue;
    return launch_epi(p, vec, cfg, stream);
  }
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
