// fp32 instantiations of the matrix-core GEMM (see gemm_kernel.hpp):
// v_mfma_f32_32x32x2_f32, BK = 16, 16-byte (VEC = 4) or 4-byte (VEC = 1) loads.
#include "gemm_dma.hpp"
#include "gemm_kernel.hpp"
#include "kernels.hpp"

namespace mt {

template <bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int VEC, int WPE,
          bool EPI = false>
static hipError_t launch_f32(const GemmParams& p, hipStream_t stream) {
  GemmParams q = p;
  q.tiles_m = (int32_t)((p.M + BM - 1) / BM);
  q.tiles_n = (int32_t)((p.N + BN - 1) / BN);
  const int64_t blocks = (int64_t)q.tiles_m * q.tiles_n * p.keep_count * p.splits;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((gemm::gemm_kernel<float, A_KC, B_KC, BM, BN, BK, WGM, WGN, VEC, WPE, EPI>),
                     dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, stream, q);
  return hipGetLastError();
}

template <bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int NS, int WPE,
          bool EPI = false, int LANE = 16, bool VEC_C = true>
static hipError_t launch_dma(const GemmParams& p, hipStream_t stream) {
  GemmParams q = p;
  q.tiles_m = (int32_t)((p.M + BM - 1) / BM);
  q.tiles_n = (int32_t)((p.N + BN - 1) / BN);
  const int64_t blocks = (int64_t)q.tiles_m * q.tiles_n * p.keep_count * p.splits;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  // persistent grid (host decides: plain product of whole tiles, more tiles than CUs)
  if constexpr (BM == 256 && BN == 256 && !EPI && LANE == 16 && VEC_C) {
    if (p.persist > 0 && p.K % BK == 0 && blocks > p.persist) {
      hipLaunchKernelGGL((gemm::gemm_dma_kernel<float, A_KC, B_KC, BM, BN, BK, WGM, WGN, NS, 1, 1, false, WPE,
                                                false, 16, true, true>),
                         dim3((unsigned)p.persist), dim3(WGM * WGN * 64), 0, stream, q);
      return hipGetLastError();
    }
  }
  // the per-load K-tail test only where K is not a whole number of stages
  if (p.K % BK != 0)
    hipLaunchKernelGGL((gemm::gemm_dma_kernel<float, A_KC, B_KC, BM, BN, BK, WGM, WGN, NS, 1, 1, true, WPE, EPI, LANE, VEC_C>),
                       dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, stream, q);
  else
    hipLaunchKernelGGL((gemm::gemm_dma_kernel<float, A_KC, B_KC, BM, BN, BK, WGM, WGN, NS, 1, 1, false, WPE, EPI, LANE, VEC_C>),
                       dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, stream, q);
  return hipGetLastError();
}

template <bool A_KC, bool B_KC, int VEC>
static hipError_t launch_layout(const GemmParams& p, int cfg, hipStream_t stream) {
  if constexpr (VEC == 1) {
    // operands or output without 16-byte aligned rows: the DMA tiles with
    // 4-byte lanes and element stores, or the element-load register-staged
    // kernels up to 128x128 (larger tiles would spill staging registers)
    switch (cfg) {
      case kCfgDma256x256: return launch_dma<A_KC, B_KC, 256, 256, 32, 2, 4, 2, 2, false, 4, false>(p, stream);
      case kCfgDma256x128: return launch_dma<A_KC, B_KC, 256, 128, 16, 2, 2, 3, 2, false, 4, false>(p, stream);
      case kCfgDma128x256: return launch_dma<A_KC, B_KC, 128, 256, 16, 2, 2, 3, 2, false, 4, false>(p, stream);
      case kCfgDma128x128: return launch_dma<A_KC, B_KC, 128, 128, 32, 2, 2, 2, 2, false, 4, false>(p, stream);
      case kCfgDma256x192: return launch_dma<A_KC, B_KC, 256, 192, 16, 4, 2, 4, 2, false, 4, false>(p, stream);
      case kCfgDma256x96:
        // an N-contiguous B would need 384-byte LDS rows, which the swizzle cannot serve
        if constexpr (B_KC) return launch_dma<A_KC, B_KC, 256, 96, 16, 4, 1, 3, 2, false, 4, false>(p, stream);
        else return hipErrorInvalidValue;
      case kCfgDma64x384: return launch_dma<A_KC, B_KC, 64, 384, 16, 1, 4, 2, 2, false, 4, false>(p, stream);
      case kCfg64x64: return launch_f32<A_KC, B_KC, 64, 64, 16, 2, 2, 1, 4>(p, stream);
      default: return launch_f32<A_KC, B_KC, 128, 128, 16, 2, 2, 1, 2>(p, stream);
    }
  } else {
    switch (cfg) {
      case kCfgDma256x256: return launch_dma<A_KC, B_KC, 256, 256, 32, 2, 4, 2, 2>(p, stream);
      case kCfgDma256x256w4: return launch_dma<A_KC, B_KC, 256, 256, 32, 2, 2, 2, 1>(p, stream);
      case kCfgDma256x128: return launch_dma<A_KC, B_KC, 256, 128, 16, 2, 2, 3, 2>(p, stream);
      case kCfgDma128x256: return launch_dma<A_KC, B_KC, 128, 256, 16, 2, 2, 3, 2>(p, stream);
      case kCfgDma128x128: return launch_dma<A_KC, B_KC, 128, 128, 32, 2, 2, 2, 2>(p, stream);
      case kCfgDma128x128w8: return launch_dma<A_KC, B_KC, 128, 128, 32, 2, 4, 2, 4>(p, stream);
      case kCfgDma128x128k64: return launch_dma<A_KC, B_KC, 128, 128, 64, 2, 4, 2, 2>(p, stream);
      case kCfg256x256: return launch_f32<A_KC, B_KC, 256, 256, 16, 2, 2, VEC, 1>(p, stream);
      case kCfg256x256x64w8: return launch_f32<A_KC, B_KC, 256, 256, 32, 2, 4, VEC, 2>(p, stream);
      case kCfg256x128: return launch_f32<A_KC, B_KC, 256, 128, 16, 2, 2, VEC, 2>(p, stream);
      case kCfg128x256: return launch_f32<A_KC, B_KC, 128, 256, 16, 2, 2, VEC, 2>(p, stream);
      case kCfg128x128: return launch_f32<A_KC, B_KC, 128, 128, 16, 2, 2, VEC, 2>(p, stream);
      default: return launch_f32<A_KC, B_KC, 64, 64, 16, 2, 2, VEC, 4>(p, stream);
    }
  }
}

int gemm_tile_m(int cfg) {
  switch (cfg) {
    case kCfg256x256: case kCfg256x128: case kCfg256x256x64w8: case kCfgDma256x256:
    case kCfgDma256x256w4: case kCfgDma256x128: case kCfgDma256x192: case kCfgDma256x96: return 256;
    case kCfg128x256: case kCfg128x128: case kCfgDma128x256: case kCfgDma128x128:
    case kCfgDma128x128w8: case kCfgDma128x128k64: return 128;
    default: return 64;
  }
}
int gemm_tile_n(int cfg) {
  switch (cfg) {
    case kCfg256x256: case kCfg128x256: case kCfg256x256x64w8: case kCfgDma256x256:
    case kCfgDma256x256w4: case kCfgDma128x256: return 256;
    case kCfg256x128: case kCfg128x128: case kCfgDma256x128: case kCfgDma128x128:
    case kCfgDma128x128w8: case kCfgDma128x128k64: return 128;
    case kCfgDma256x192: return 192;
    case kCfgDma256x96: return 96;
    case kCfgDma64x384: return 384;
    default: return 64;
  }
}
int gemm_tile_k(int cfg, bool bf16) {
  if (cfg == kCfgDma128x128k64) return 64;
  if (cfg == kCfg256x256x64w8) return bf16 ? 64 : 32;
  if (cfg == kCfgDma256x256 || cfg == kCfgDma256x256w4 || cfg == kCfgDma128x128 ||
      cfg == kCfgDma128x128w8)
    return bf16 ? 64 : 32;
  return bf16 ? 32 : 16;
}

// The dense layer followed by a nonlinearity (z / act set): the forward
// layout only, on the 256x256 or 128x128 DMA tiles or the 128x128 / 64x64
// register-staged tiles.
static hipError_t launch_epi(const GemmParams& p, bool vec, int cfg, hipStream_t stream) {
  if (vec) {
    if (cfg == kCfgDma128x128)
      return launch_dma<true, true, 128, 128, 32, 2, 2, 2, 2, true>(p, stream);
    if (cfg == kCfgDma256x256)
      return launch_dma<true, true, 256, 256, 32, 2, 4, 2, 2, true>(p, stream);
    if (cfg == kCfg128x128) return launch_f32<true, true, 128, 128, 16, 2, 2, 4, 2, true>(p, stream);
    return launch_f32<true, true, 64, 64, 16, 2, 2, 4, 4, true>(p, stream);
  }
  if (cfg == kCfg128x128) return launch_f32<true, true, 128, 128, 16, 2, 2, 1, 2, true>(p, stream);
  return launch_f32<true, true, 64, 64, 16, 2, 2, 1, 4, true>(p, stream);
}

template <int MODE, int BM, int BN, int BK, int WGM, int WGN, int NS, int WPE>
static hipError_t launch_conv(const GemmParams& p, hipStream_t stream) {
  GemmParams q = p;
  q.tiles_m = (int32_t)((p.M + BM - 1) / BM);
  q.tiles_n = (int32_t)((p.N + BN - 1) / BN);
  const int64_t blocks = (int64_t)q.tiles_m * q.tiles_n * p.keep_count * p.splits;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  if (p.K % BK != 0) {
    // the forward's and the input gradient's stages are whole channel groups of one tap
    if constexpr (MODE != 2) return hipErrorInvalidValue;
    else
      hipLaunchKernelGGL((gemm::conv_dma_kernel<MODE, BM, BN, BK, WGM, WGN, NS, true, WPE>),
                         dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, stream, q);
  } else {
    hipLaunchKernelGGL((gemm::conv_dma_kernel<MODE, BM, BN, BK, WGM, WGN, NS, false, WPE>),
                       dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, stream, q);
  }
  return hipGetLastError();
}

template <int MODE>
static hipError_t conv_cfg(const GemmParams& p, int cfg, hipStream_t stream) {
  switch (cfg) {
    case kCfgDma256x256: return launch_conv<MODE, 256, 256, 32, 2, 4, 2, 2>(p, stream);
    case kCfgDma128x128: return launch_conv<MODE, 128, 128, 32, 2, 2, 2, 2>(p, stream);
    case kCfgDma128x128w8: return launch_conv<MODE, 128, 128, 32, 2, 4, 2, 4>(p, stream);
    default: return hipErrorInvalidValue;
  }
}

// Sum of the segments of every tile the stream-K product cut: C = sum over
// slots s < n(t) of partial[s] (+ bias, + C), slots in order; tiles computed
// whole were written by the product. A lane per 4 consecutive columns. The
// lane's row and its tile's segment count take integer divisions; where the
// sizes allow (NARROW: M N / 4 and the stage count times G below 2^32) they
// are 32-bit ones, a fraction of the instructions of 64-bit division.
template <int BM, int BN, bool NARROW>
__global__ __launch_bounds__(256) void sk_finish_kernel(const GemmParams p, int64_t G) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  const int64_t n4 = p.N / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= p.M * n4) return;
  const int64_t ks = (p.K + 31) / 32;
  const int64_t U = (int64_t)p.tiles_m * p.tiles_n * ks;
  int64_t m, n;
  gemm::SkSeg sg;
  if constexpr (NARROW) {
    const uint32_t q = (uint32_t)i / (uint32_t)n4;
    m = q;
    n = ((uint32_t)i - q * (uint32_t)n4) * 4;
    const uint32_t t = (uint32_t)(m / BM) * (uint32_t)p.tiles_n + (uint32_t)(n / BN);
    const uint32_t g = (uint32_t)G, u = (uint32_t)U, L = t * (uint32_t)ks;
    // sk_count(X) = ceil(X G / U) in 32 bits (X G <= U G < 2^32)
    auto cnt = [&](uint32_t X) { return (X * g + u - 1) / u; };
    sg.n = (int)(cnt(L + (uint32_t)ks) - cnt(L + 1) + 1);
  } else {
    m = i / n4;
    n = (i - m * n4) * 4;
    const int64_t t = (m / BM) * p.tiles_n + n / BN;
    sg = gemm::sk_segment(t, 0, ks, G, U);
  }
  if (sg.n <= 1) return;
  const float* src = p.partial + m * p.N + n;
  f32x4 v = *(const f32x4*)src;
  for (int s = 1; s < sg.n; ++s) v += *(const f32x4*)(src + s * p.partial_stride);
  float* c = p.c + m * p.ldc + n;
  if (p.bias) v += *(const f32x4*)(p.bias + n);
  if (p.accumulate) v += *(const f32x4*)c;
  *(f32x4*)c = v;
}

// Stream-K launch of the gathered forward / input-gradient product on the
// 256x256 tile: G blocks, then the finish. The host has sized p.partial for
// the most segments any tile gets (sk_max_segments).
hipError_t gemm_f32_conv_sk(const GemmParams& p, int mode, int blocks, hipStream_t stream) {
  GemmParams q = p;
  q.tiles_m = (int32_t)((p.M + 255) / 256);
  q.tiles_n = (int32_t)((p.N + 255) / 256);
  if (p.M <= 0 || p.N <= 0 || blocks <= 0 || p.K % 32 != 0 || p.N % 4 != 0)
    return hipErrorInvalidValue;
  if (mode == 1)
    hipLaunchKernelGGL((gemm::conv_dma_sk_kernel<1, 256, 256, 32, 2, 4, 2, 2>), dim3(blocks),
                       dim3(512), 0, stream, q);
  else if (mode == 3)
    hipLaunchKernelGGL((gemm::conv_dma_sk_kernel<3, 256, 256, 32, 2, 4, 2, 2>), dim3(blocks),
                       dim3(512), 0, stream, q);
  else
    return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t groups = p.M * (p.N / 4);
  if ((groups + 255) / 256 > 0x7fffffff) return hipErrorInvalidConfiguration;
  const int64_t units = (int64_t)q.tiles_m * q.tiles_n * (p.K / 32);
  const dim3 grid((unsigned)((groups + 255) / 256));
  if (groups < (int64_t(1) << 32) && units * blocks + units < (int64_t(1) << 32))
    hipLaunchKernelGGL((sk_finish_kernel<256, 256, true>), grid, dim3(256), 0, stream, q, (int64_t)blocks);
  else
    hipLaunchKernelGGL((sk_finish_kernel<256, 256, false>), grid, dim3(256), 0, stream, q, (int64_t)blocks);
  return hipGetLastError();
}

// Every sub-pixel phase of a strided input gradient in one grid on the
// 256x256 tile (p: the shared description, N = C; tab: the phases, their
// tile counts summed in tile0).
hipError_t gemm_f32_conv_phases(const GemmParams& p, const ConvPhases& tab, hipStream_t stream) {
  if (tab.n <= 0 || tab.n > kMaxConvPhases || p.N % 4 != 0) return hipErrorInvalidValue;
  for (int k = 0; k < tab.n; ++k)
    if (tab.ph[k].K % 32 != 0 || tab.ph[k].M <= 0) return hipErrorInvalidValue;
  GemmParams q = p;
  q.tiles_n = (int32_t)((p.N + 255) / 256);
  q.splits = 1;
  const int64_t blocks = tab.tile0[tab.n];
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((gemm::conv_dgrad_phases_kernel<256, 256, 32, 2, 4, 2, 2>), dim3((unsigned)blocks),
                     dim3(512), 0, stream, q, tab);
  return hipGetLastError();
}

int64_t sk_max_segments(int64_t tiles, int64_t ks, int64_t blocks) {
  const int64_t U = tiles * ks;
  int64_t most = 1;
  for (int64_t t = 0; t < tiles; ++t) {
    const int64_t n = gemm::sk_segment(t, 0, ks, blocks, U).n;
    if (n > most) most = n;
  }
  return most;
}

bool gemm_conv_cfg(int cfg) {
  return cfg == kCfgDma256x256 || cfg == kCfgDma128x128 || cfg == kCfgDma128x128w8;
}

hipError_t gemm_f32_conv(const GemmParams& p, int mode, int cfg, hipStream_t stream) {
  if (mode == 1) return conv_cfg<1>(p, cfg, stream);
  if (mode == 2) return conv_cfg<2>(p, cfg, stream);
  if (mode == 3) return conv_cfg<3>(p, cfg, stream);
  if (mode == 4) return conv_cfg<4>(p, cfg, stream);
  return hipErrorInvalidValue;
}

hipError_t gemm_f32(const GemmParams& p, bool a_kc, bool b_kc, bool vec, int cfg,
                    hipStream_t stream) {
  if (p.act || p.z) {
    if (!a_kc || !b_kc) return hipErrorInvalidValue;
    return launch_epi(p, vec, cfg, stream);
  }
  if (vec) {
    if (a_kc && b_kc) return launch_layout<true, true, 4>(p, cfg, stream);
    if (a_kc && !b_kc) return launch_layout<true, false, 4>(p, cfg, stream);
    if (!a_kc && b_kc) return launch_layout<false, true, 4>(p, cfg, stream);
    return launch_layout<false, false, 4>(p, cfg, stream);
  }
  if (a_kc && b_kc) return launch_layout<true, true, 1>(p, cfg, stream);
  if (a_kc && !b_kc) return launch_layout<true, false, 1>(p, cfg, stream);
  if (!a_kc && b_kc) return launch_layout<false, true, 1>(p, cfg, stream);
  return launch_layout<false, false, 1>(p, cfg, stream);
}

}  // namespace mt
