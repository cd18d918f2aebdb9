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
// unfold_kernel: a block per 8 output pixels (decoded once per block); a
// lane decodes the taps of its groups of 4 columns once and writes them in
// all 8 rows with 16-byte stores; channels-last x with k = (u, v, c) reads 4
// channels with one 16-byte load.
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

// Block b fills rows m = b R .. b R + R - 1 of the unfolded matrix. Each
// lane takes the column groups k4 = tid, tid + 256, ... (4 columns, one
// 16-byte store each), decodes their tap once, and writes that group in all
// R rows; the rows' pixel origins are decoded once per block (uniform).
// FAST: k = (u, v, c), x channels contiguous and 16-byte aligned, C % 4 == 0.
constexpr int kUnfoldRows = 8;

template <bool FAST>
__global__ __launch_bounds__(256) void unfold_kernel(const float* x, const ConvGeom g, float* col,
                                                     int64_t M) {
  const int64_t m0 = (int64_t)blockIdx.x * kUnfoldRows;
  const int64_t Kcp4 = g.Kcp / 4;
  int64_t nb[kUnfoldRows];  // x offset of image n
  int hb[kUnfoldRows], wb[kUnfoldRows];
#pragma unroll
  for (int r = 0; r < kUnfoldRows; ++r) {
    const int64_t m = m0 + r < M ? m0 + r : M - 1;
    const int j = (int)(m % g.WO);
    const int64_t t = m / g.WO;
    hb[r] = (int)(t % g.HO) * g.sh - g.ph;
    wb[r] = j * g.sw - g.pw;
    nb[r] = (t / g.HO) * g.xs[0];
  }
  const int rows = M - m0 < kUnfoldRows ? (int)(M - m0) : kUnfoldRows;
  for (int64_t k4 = threadIdx.x; k4 < Kcp4; k4 += 256) {
    const int64_t k0 = 4 * k4;
    if (FAST) {
      int c = 0, u = 0, v = 0;
      const bool live = k0 < g.Kc;
      if (live) decode_k(g, k0, c, u, v);
      f32x4 vals[kUnfoldRows];
#pragma unroll
      for (int r = 0; r < kUnfoldRows; ++r) {
        const int h = hb[r] + u, w = wb[r] + v;
        vals[r] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (live && r < rows && h >= 0 && h < g.H && w >= 0 && w < g.W)
          vals[r] = *(const f32x4*)(x + nb[r] + (int64_t)h * g.xs[2] + (int64_t)w * g.xs[3] + c);
      }
#pragma unroll
      for (int r = 0; r < kUnfoldRows; ++r)
        if (r < rows) *(f32x4*)(col + (m0 + r) * g.Kcp + k0) = vals[r];
    } else {
      int cs[4], us[4], vs[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        cs[e] = -1;
        if (k0 + e < g.Kc) decode_k(g, k0 + e, cs[e], us[e], vs[e]);
      }
      for (int r = 0; r < rows; ++r) {
        f32x4 out = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (cs[e] < 0) continue;
          const int h = hb[r] + us[e], w = wb[r] + vs[e];
          if (h >= 0 && h < g.H && w >= 0 && w < g.W)
            out[e] = x[nb[r] + cs[e] * g.xs[1] + (int64_t)h * g.xs[2] + (int64_t)w * g.xs[3]];
        }
        *(f32x4*)(col + (m0 + r) * g.Kcp + k0) = out;
      }
    }
  }
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
  const int64_t blocks = (M + kUnfoldRows - 1) / kUnfoldRows;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  const bool fast = g.korder_uvc && g.xs[1] == 1 && g.C % 4 == 0 && (uintptr_t)x % 16 == 0 &&
                    g.xs[0] % 4 == 0 && g.xs[2] % 4 == 0 && g.xs[3] % 4 == 0;
  if (fast)
    hipLaunchKernelGGL(unfold_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, x, g, col,
                       M);
  else
    hipLaunchKernelGGL(unfold_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, x, g, col,
                       M);
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
