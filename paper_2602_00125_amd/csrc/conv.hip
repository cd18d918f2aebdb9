// Convolution (MiniTensor Sec. 3.3 Eq. (6)) as matrix products on the GEMM
// core, gfx950: the HBM-bound index work of the unfolded ("im2col") form.
//
// With the output pixels m = (n, i, j) as rows and the taps k of one output
// channel as columns, Eq. (6) is the dense product Y[m][co] = sum_k
// U[m][k] Wf[co][k] + b[co], where U is the unfolded input
//   U[m][k] = x[n][c][i sh + u - ph][j sw + v - pw]  (0 outside the image)
// and Wf the weights flattened to [CO][C KH KW] in their own memory order:
// k = (c, u, v) for weights stored [CO][C][KH][KW], k = (u, v, c) for
// channels-last weights [CO][KH][KW][C]. The pullbacks are the same products
// as the dense layer's (Eq. (4)): dWf = dY^T U and dU = dY Wf, and the input
// gradient folds dU back onto the image, each input element summing the
// unfolded entries that read it:
//   dx[n][c][h][x] = sum over taps (u, v) with h = i sh + u - ph, x = j sw + v - pw
//                    (i, j inside the output) of dU[(n, i, j)][k(c, u, v)].
//
// unfold_kernel: one block row per output pixel m (decoded once per block),
// each lane writes 4 consecutive k of U with one 16-byte store; channels-last
// x with k = (u, v, c) reads 4 channels with one 16-byte load.
// fold_kernel: a lane per input element (or 4 channels of one), summing the
// taps in a fixed (u, v) order: a gather, so no atomics and bit-identical
// reruns.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace mt {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// tap (c, u, v) of column k in the unfolded matrix
__device__ __forceinline__ void decode_k(const ConvGeom& g, int64_t k, int& c, int& u, int& v) {
  if (g.korder_uvc) {
    c = (int)(k % g.C);
    const int64_t uv = k / g.C;
    u = (int)(uv / g.KW);
    v = (int)(uv % g.KW);
  } else {
    v = (int)(k % g.KW);
    const int64_t cu = k / g.KW;
    u = (int)(cu % g.KH);
    c = (int)(cu / g.KH);
  }
}

// FAST: k = (u, v, c), x channels contiguous and 16-byte aligned, C % 4 == 0.
template <bool FAST>
__global__ __launch_bounds__(256) void unfold_kernel(const float* x, const ConvGeom g, float* col) {
  const int64_t m = blockIdx.x;
  const int64_t k0 = ((int64_t)blockIdx.y * 256 + threadIdx.x) * 4;
  if (k0 >= g.Kcp) return;
  const int j = (int)(m % g.WO);
  const int64_t t = m / g.WO;
  const int i = (int)(t % g.HO);
  const int64_t n = t / g.HO;
  const float* xn = x + n * g.xs[0];
  const int hb = i * g.sh - g.ph, wb = j * g.sw - g.pw;
  f32x4 out = {0.f, 0.f, 0.f, 0.f};
  if (FAST) {
    if (k0 < g.Kc) {
      int c, u, v;
      decode_k(g, k0, c, u, v);
      const int h = hb + u, w = wb + v;
      if (h >= 0 && h < g.H && w >= 0 && w < g.W)
        out = *(const f32x4*)(xn + (int64_t)h * g.xs[2] + (int64_t)w * g.xs[3] + c);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t k = k0 + e;
      if (k >= g.Kc) break;
      int c, u, v;
      decode_k(g, k, c, u, v);
      const int h = hb + u, w = wb + v;
      if (h >= 0 && h < g.H && w >= 0 && w < g.W)
        out[e] = xn[c * g.xs[1] + (int64_t)h * g.xs[2] + (int64_t)w * g.xs[3]];
    }
  }
  *(f32x4*)(col + m * g.Kcp + k0) = out;
}

// Sum over the taps reading input element (n, c, h, w); FAST: 4 channels at
// once (k = (u, v, c), C % 4 == 0).
template <bool FAST>
__device__ __forceinline__ f32x4 fold_sum(const float* dcol, const ConvGeom& g, int64_t n, int c,
                                          int h, int w) {
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
  for (int u = 0; u < g.KH; ++u) {
    const int ti = h + g.ph - u;
    if (ti < 0 || ti % g.sh) continue;
    const int i = ti / g.sh;
    if (i >= g.HO) continue;
    for (int v = 0; v < g.KW; ++v) {
      const int tj = w + g.pw - v;
      if (tj < 0 || tj % g.sw) continue;
      const int j = tj / g.sw;
      if (j >= g.WO) continue;
      const float* row = dcol + ((n * g.HO + i) * g.WO + j) * g.Kcp;
      if (FAST) {
        s += *(const f32x4*)(row + (int64_t)(u * g.KW + v) * g.C + c);
      } else {
        const int64_t k = g.korder_uvc ? (int64_t)(u * g.KW + v) * g.C + c
                                       : ((int64_t)c * g.KH + u) * g.KW + v;
        s[0] += row[k];
      }
    }
  }
  return s;
}

// grid.x: input pixels (n, h, w); grid.y: channel groups of 256 (x4 when FAST)
template <bool FAST>
__global__ __launch_bounds__(256) void fold_kernel(const float* dcol, const ConvGeom g, float* dx,
                                                   int accumulate) {
  const int64_t p = blockIdx.x;
  const int per = FAST ? 4 : 1;
  const int c0 = (int)(((int64_t)blockIdx.y * 256 + threadIdx.x) * per);
  if (c0 >= g.C) return;
  const int w = (int)(p % g.W);
  const int64_t t = p / g.W;
  const int h = (int)(t % g.H);
  const int64_t n = t / g.H;
  const f32x4 s = fold_sum<FAST>(dcol, g, n, c0, h, w);
  float* d = dx + n * g.ds[0] + (int64_t)h * g.ds[2] + (int64_t)w * g.ds[3];
  if (FAST && g.dx_vec) {
    f32x4* q = (f32x4*)(d + c0);
    *q = accumulate ? *q + s : s;
  } else {
#pragma unroll
    for (int e = 0; e < per; ++e) {
      float* q = d + (int64_t)(c0 + e) * g.ds[1];
      *q = accumulate ? *q + s[e] : s[e];
    }
  }
}

}  // namespace

hipError_t conv_unfold(const float* x, const ConvGeom& g, float* col, hipStream_t stream) {
  const int64_t M = (int64_t)g.N * g.HO * g.WO;
  if (M <= 0 || g.Kcp <= 0) return hipSuccess;
  const int64_t ky = (g.Kcp + 1023) / 1024;
  if (M > 0x7fffffff || ky > 65535) return hipErrorInvalidConfiguration;
  const bool fast = g.korder_uvc && g.xs[1] == 1 && g.C % 4 == 0 && (uintptr_t)x % 16 == 0 &&
                    g.xs[0] % 4 == 0 && g.xs[2] % 4 == 0 && g.xs[3] % 4 == 0;
  if (fast)
    hipLaunchKernelGGL(unfold_kernel<true>, dim3((unsigned)M, (unsigned)ky), dim3(256), 0, stream, x,
                       g, col);
  else
    hipLaunchKernelGGL(unfold_kernel<false>, dim3((unsigned)M, (unsigned)ky), dim3(256), 0, stream,
                       x, g, col);
  return hipGetLastError();
}

hipError_t conv_fold(const float* dcol, const ConvGeom& g, float* dx, bool accumulate,
                     hipStream_t stream) {
  const int64_t P = (int64_t)g.N * g.H * g.W;
  if (P <= 0 || g.C <= 0) return hipSuccess;
  const bool fast = g.korder_uvc && g.C % 4 == 0 && g.Kcp % 4 == 0;
  const int per = fast ? 4 : 1;
  const int64_t cy = (g.C + 256 * per - 1) / (256 * per);
  if (P > 0x7fffffff || cy > 65535) return hipErrorInvalidConfiguration;
  if (fast)
    hipLaunchKernelGGL(fold_kernel<true>, dim3((unsigned)P, (unsigned)cy), dim3(256), 0, stream, dcol,
                       g, dx, (int)accumulate);
  else
    hipLaunchKernelGGL(fold_kernel<false>, dim3((unsigned)P, (unsigned)cy), dim3(256), 0, stream,
                       dcol, g, dx, (int)accumulate);
  return hipGetLastError();
}

}  // namespace mt
