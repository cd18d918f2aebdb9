// HBM-bound reductions of the backward pass, gfx950.
//
// * colsum: db[n] = sum_m dY[m][n], the add pullback through the broadcast
//   bias (MiniTensor Sec. 3.2 add pullback with the Sec. 3.1 broadcasting
//   rule; Sec. 3.3 Eq. (5)). The summed axis is the outer (strided) one, so
//   lanes run along the contiguous n (16-byte loads, 4 columns a lane) and
//   the sixteen waves of a block take interleaved rows with four loads in
//   flight per lane (64 KB per CU in flight keeps HBM busy); their partial
//   sums are combined through LDS in a fixed order. M is cut into row slices
//   so that about one block runs per CU; slice sums go to a workspace and
//   are added by a second pass in slice order: no atomics, bit-identical
//   reruns.
// * reduce_strided: the same add pullback for any broadcast (the gradient of
//   an operand that was expanded along some axes). When the innermost axis
//   of the gradient is kept, a thread per output walks the summed axes
//   (coalesced along the kept axis). When the innermost axis is summed, a
//   wave per output strides over it and the 64 lane sums are combined with
//   DPP row operations (quad_perm, row_half_mirror, row_mirror) and a final
//   fixed-order sum of the four row results.
// * splitk_finish: fixed-order sum of split-K partial tiles.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace mt {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(unsigned short v) {
  return __uint_as_float((unsigned)v << 16);
}

template <bool BF16>
__device__ __forceinline__ f32x4 load4(const void* base, int64_t idx) {
  if constexpr (BF16) {
    const u16x4 v = *(const u16x4*)((const unsigned short*)base + idx);
    return f32x4{bf16_to_f32(v[0]), bf16_to_f32(v[1]), bf16_to_f32(v[2]), bf16_to_f32(v[3])};
  } else {
    return *(const f32x4*)((const float*)base + idx);
  }
}
template <bool BF16>
__device__ __forceinline__ float load1(const void* base, int64_t idx) {
  if constexpr (BF16) return bf16_to_f32(((const unsigned short*)base)[idx]);
  else return ((const float*)base)[idx];
}

// grid: (ceil(N / (64*VEC)), parts). Block = WAVES wave64s; wave w sums rows
// r0 + w, r0 + w + WAVES, ... of its slice for 64*VEC columns, four rows in
// flight per lane; the WAVES partial sums meet in LDS in wave order.
template <bool BF16, int VEC, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void colsum_kernel(const void* x, int64_t M, int64_t N,
                                                            int64_t ld, float* out, int accumulate,
                                                            float* ws, int64_t rows_per_part) {
  __shared__ f32x4 red[WAVES][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t n = ((int64_t)blockIdx.x * 64 + lane) * VEC;
  const int64_t r0 = (int64_t)blockIdx.y * rows_per_part;
  const int64_t r1 = (r0 + rows_per_part) < M ? (r0 + rows_per_part) : M;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (n < N) {
    if (VEC == 4) {
      int64_t m = r0 + wave;
      for (; m + 3 * WAVES < r1; m += 4 * WAVES) {
        const f32x4 a = load4<BF16>(x, m * ld + n);
        const f32x4 b = load4<BF16>(x, (m + WAVES) * ld + n);
        const f32x4 c = load4<BF16>(x, (m + 2 * WAVES) * ld + n);
        const f32x4 d = load4<BF16>(x, (m + 3 * WAVES) * ld + n);
        acc += a;
        acc += b;
        acc += c;
        acc += d;
      }
      for (; m < r1; m += WAVES) acc += load4<BF16>(x, m * ld + n);
    } else {
      for (int64_t m = r0 + wave; m < r1; m += WAVES) acc[0] += load1<BF16>(x, m * ld + n);
    }
  }
  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0 && n < N) {
    f32x4 s = red[0][lane];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) s += red[w][lane];
    if (gridDim.y > 1) {
      float* dst = ws + (int64_t)blockIdx.y * N;
      for (int e = 0; e < VEC; ++e)
        if (n + e < N) dst[n + e] = s[e];
    } else {
      for (int e = 0; e < VEC; ++e)
        if (n + e < N) out[n + e] = accumulate ? out[n + e] + s[e] : s[e];
    }
  }
}

// out[n] (+)= sum_p ws[p][n], p ascending. The loads go out sixteen at a
// time ahead of their adds: with few columns (one block for 256 of them)
// and many parts the kernel is bound by load latency, which a load at a
// time per add left exposed (a 256-channel convolution's db: 17.6 us).
__global__ __launch_bounds__(256) void parts_finish_kernel(const float* ws, int parts, int64_t N,
                                                           float* out, int accumulate) {
  const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (n >= N) return;
  constexpr int U = 16;
  float s = 0.f;
  int p = 0;
  for (; p + U <= parts; p += U) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = ws[(int64_t)(p + u) * N + n];
#pragma unroll
    for (int u = 0; u < U; ++u) s += v[u];
  }
  for (; p < parts; ++p) s += ws[(int64_t)p * N + n];
  out[n] = accumulate ? out[n] + s : s;
}

__global__ __launch_bounds__(256) void splitk_finish_kernel(const float* partial, int splits, int64_t M,
                                                            int64_t N, float* c, int64_t ldc,
                                                            const float* bias, int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= M * N) return;
  const int64_t m = i / N, n = i % N;
  float s = 0.f;
  for (int p = 0; p < splits; ++p) s += partial[(int64_t)p * M * N + i];
  if (bias) s += bias[n];
  float* dst = c + m * ldc + n;
  *dst = accumulate ? *dst + s : s;
}

// The element sums above, four consecutive elements of the flattened M x N
// partial a lane (M N a multiple of 4 and the partial 16-byte aligned, so
// every run's slice is): one 16-byte load per run instead of four 4-byte
// ones, the stores one element at a time along C's rows (odd pitches). Each
// element is summed in the same order as above.
__global__ __launch_bounds__(256) void splitk_finish_flat4_kernel(const float* partial, int splits,
                                                                  int64_t M, int64_t N, float* c,
                                                                  int64_t ldc, const float* bias,
                                                                  int accumulate) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  const int64_t MN = M * N;
  if (i >= MN) return;
  float4 s = {0.f, 0.f, 0.f, 0.f};
  for (int p = 0; p < splits; ++p) {
    const float4 v = *(const float4*)(partial + (int64_t)p * MN + i);
    s.x += v.x;
    s.y += v.y;
    s.z += v.z;
    s.w += v.w;
  }
  int64_t m = i / N, n = i - m * N;
  const float e[4] = {s.x, s.y, s.z, s.w};
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    float x = e[u];
    if (bias) x += bias[n];
    float* dst = c + m * ldc + n;
    *dst = accumulate ? *dst + x : x;
    if (++n == N) {
      n = 0;
      ++m;
    }
  }
}

// The same sums four columns a lane with 16-byte accesses (N, ldc and every
// base a multiple of 4 floats): blockIdx.x covers 1024 columns, blockIdx.y
// strides over the rows. Each element is summed in the same order as above.
// With cs_part, one more column of blocks adds the runs' column sums of A
// (M of them) in run order, as parts_finish_kernel does, saving its launch.
__global__ __launch_bounds__(256) void splitk_finish4_kernel(const float* partial, int splits,
                                                             int64_t M, int64_t N, float* c,
                                                             int64_t ldc, const float* bias,
                                                             int accumulate, const float* cs_part,
                                                             float* cs_out) {
  if (cs_part && blockIdx.x == gridDim.x - 1) {
    const int64_t k = (int64_t)blockIdx.y * 256 + threadIdx.x;
    if (k >= M) return;
    float s = 0.f;
    for (int q = 0; q < splits; ++q) s += cs_part[(int64_t)q * M + k];
    cs_out[k] = accumulate ? cs_out[k] + s : s;
    return;
  }
  const int64_t n = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (n >= N) return;
  const int64_t MN = M * N;
  float4 bb = {0.f, 0.f, 0.f, 0.f};
  if (bias) bb = *(const float4*)(bias + n);
  for (int64_t m = blockIdx.y; m < M; m += gridDim.y) {
    const float* src = partial + m * N + n;
    float4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int p = 0; p < splits; ++p) {
      const float4 v = *(const float4*)(src + (int64_t)p * MN);
      s.x += v.x;
      s.y += v.y;
      s.z += v.z;
      s.w += v.w;
    }
    if (bias) {
      s.x += bb.x;
      s.y += bb.y;
      s.z += bb.z;
      s.w += bb.w;
    }
    float4* dst = (float4*)(c + m * ldc + n);
    if (accumulate) {
      const float4 d = *dst;
      s.x = d.x + s.x;
      s.y = d.y + s.y;
      s.z = d.z + s.z;
      s.w = d.w + s.w;
    }
    *dst = s;
  }
}

__global__ __launch_bounds__(256) void fill_kernel(float* out, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) out[i] = v;
}

__device__ __forceinline__ int64_t decode(int64_t flat, int nd, const int64_t* shape,
                                          const int64_t* stride) {
  int64_t off = 0;
  for (int d = nd - 1; d >= 0; --d) {
    const int64_t i = flat % shape[d];
    flat /= shape[d];
    off += i * stride[d];
  }
  return off;
}

// Thread per output element; summed index range [r0, r1) of part blockIdx.y.
__global__ __launch_bounds__(256) void reduce_outer_kernel(const float* x, const ReducePlan plan,
                                                           float* out, int accumulate, float* ws,
                                                           int64_t red_per_part) {
  const int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (o >= plan.keep_count) return;
  const int64_t base = decode(o, plan.nkeep, plan.keep_shape, plan.keep_stride);
  const int64_t r0 = (int64_t)blockIdx.y * red_per_part;
  const int64_t r1 = (r0 + red_per_part) < plan.red_count ? (r0 + red_per_part) : plan.red_count;
  float s = 0.f;
  for (int64_t r = r0; r < r1; ++r) s += x[base + decode(r, plan.nred, plan.red_shape, plan.red_stride)];
  if (gridDim.y > 1) ws[(int64_t)blockIdx.y * plan.keep_count + o] = s;
  else out[o] = accumulate ? out[o] + s : s;
}

// DPP butterfly inside each row of 16 lanes, then the 4 row sums in order.
__device__ __forceinline__ float wave_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));  // quad_perm [1,0,3,2]
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));  // quad_perm [2,3,0,1]
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false)); // row_half_mirror
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false)); // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return ((r0 + r1) + r2) + r3;
}

// Wave per output element: the innermost summed axis (stride red_stride[last])
// is spread over the lanes; outer summed axes are walked in order.
__global__ __launch_bounds__(256) void reduce_inner_kernel(const float* x, const ReducePlan plan,
                                                           float* out, int accumulate) {
  const int lane = threadIdx.x & 63;
  const int64_t o = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (o >= plan.keep_count) return;  // wave-uniform
  const int64_t base = decode(o, plan.nkeep, plan.keep_shape, plan.keep_stride);
  const int last = plan.nred - 1;
  const int64_t inner = plan.red_shape[last], istride = plan.red_stride[last];
  const int64_t outer = plan.red_count / inner;
  float s = 0.f;
  for (int64_t r = 0; r < outer; ++r) {
    const int64_t ob = base + decode(r, last, plan.red_shape, plan.red_stride);
    for (int64_t i = lane; i < inner; i += 64) s += x[ob + i * istride];
  }
  s = wave_sum(s);
  if (lane == 0) out[o] = accumulate ? out[o] + s : s;
}

}  // namespace

constexpr int kColsumWaves = 16;

int colsum_parts(int64_t M, int64_t N) {
  // one block per CU: (columns / 256) x parts ~ 256 blocks, slices of at
  // least 256 rows
  const int64_t col_blocks = (N + 255) / 256;
  int64_t parts = 256 / (col_blocks > 0 ? col_blocks : 1);
  const int64_t max_parts = M / 256;
  if (parts > max_parts) parts = max_parts;
  if (parts < 1) parts = 1;
  if (parts > 256) parts = 256;
  return (int)parts;
}

hipError_t colsum(const void* x, bool is_bf16, int64_t M, int64_t N, int64_t ld, float* out,
                  bool accumulate, float* ws, int parts, hipStream_t stream) {
  if (N <= 0) return hipSuccess;
  if (!ws) parts = 1;
  const bool vec = (N % 4 == 0) && (ld % 4 == 0) &&
                   ((uintptr_t)x % (is_bf16 ? 8 : 16) == 0);
  const int V = vec ? 4 : 1;
  const int64_t rows_per_part = M > 0 ? (M + parts - 1) / parts : 0;
  dim3 grid((unsigned)((N + 64 * V - 1) / (64 * V)), (unsigned)parts);
  dim3 block(kColsumWaves * 64);
  if (vec) {
    if (is_bf16)
      hipLaunchKernelGGL((colsum_kernel<true, 4, kColsumWaves>), grid, block, 0, stream, x, M, N, ld,
                         out, (int)accumulate, ws, rows_per_part);
    else
      hipLaunchKernelGGL((colsum_kernel<false, 4, kColsumWaves>), grid, block, 0, stream, x, M, N, ld,
                         out, (int)accumulate, ws, rows_per_part);
  } else {
    if (is_bf16)
      hipLaunchKernelGGL((colsum_kernel<true, 1, kColsumWaves>), grid, block, 0, stream, x, M, N, ld,
                         out, (int)accumulate, ws, rows_per_part);
    else
      hipLaunchKernelGGL((colsum_kernel<false, 1, kColsumWaves>), grid, block, 0, stream, x, M, N, ld,
                         out, (int)accumulate, ws, rows_per_part);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || parts == 1) return e;
  hipLaunchKernelGGL(parts_finish_kernel, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, stream,
                     ws, parts, N, out, (int)accumulate);
  return hipGetLastError();
}

int reduce_parts(const ReducePlan& plan) {
  if (plan.nred == 0 || plan.keep_count == 0) return 1;
  // split long sums when there are too few outputs to fill the chip
  const int64_t blocks = (plan.keep_count + 255) / 256;
  if (blocks >= 1024 || plan.red_count < 256) return 1;
  int64_t parts = 1024 / blocks;
  if (parts > plan.red_count / 64) parts = plan.red_count / 64;
  if (parts < 1) parts = 1;
  return (int)parts;
}

hipError_t reduce_strided(const float* x, const ReducePlan& plan, float* out, bool accumulate,
                          float* ws, int parts, hipStream_t stream) {
  if (plan.keep_count <= 0) return hipSuccess;
  const bool inner = plan.nred > 0 && plan.red_stride[plan.nred - 1] == 1 &&
                     (plan.nkeep == 0 || plan.keep_stride[plan.nkeep - 1] != 1);
  if (inner) {
    hipLaunchKernelGGL(reduce_inner_kernel, dim3((unsigned)((plan.keep_count + 3) / 4)), dim3(256),
                       0, stream, x, plan, out, (int)accumulate);
    return hipGetLastError();
  }
  if (!ws) parts = 1;
  const int64_t per = plan.red_count > 0 ? (plan.red_count + parts - 1) / parts : 0;
  hipLaunchKernelGGL(reduce_outer_kernel, dim3((unsigned)((plan.keep_count + 255) / 256), parts),
                     dim3(256), 0, stream, x, plan, out, (int)accumulate, ws, per);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || parts == 1) return e;
  hipLaunchKernelGGL(parts_finish_kernel, dim3((unsigned)((plan.keep_count + 255) / 256)),
                     dim3(256), 0, stream, ws, parts, plan.keep_count, out, (int)accumulate);
  return hipGetLastError();
}

hipError_t splitk_finish(const float* partial, int splits, int64_t M, int64_t N, float* c,
                         int64_t ldc, const float* bias, bool accumulate, hipStream_t stream,
                         const float* cs_part, float* cs_out) {
  const int64_t n = M * N;
  if (n <= 0) return hipSuccess;
  auto a16 = [](const void* q) { return ((uintptr_t)q & 15) == 0; };
  if (N % 4 == 0 && ldc % 4 == 0 && a16(partial) && a16(c) && (!bias || a16(bias))) {
    const int64_t rows = M < 65535 ? M : 65535;
    // the column sums' blocks (one per 256 of them) fit in the grid's rows
    const bool fold = cs_part && cs_out && (M + 255) / 256 <= rows;
    hipLaunchKernelGGL(splitk_finish4_kernel,
                       dim3((unsigned)((N / 4 + 255) / 256 + (fold ? 1 : 0)), (unsigned)rows), dim3(256),
                       0, stream, partial, splits, M, N, c, ldc, bias, (int)accumulate,
                       fold ? cs_part : nullptr, fold ? cs_out : nullptr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || fold || !cs_part) return e;
    return parts_finish(cs_part, splits, M, cs_out, accumulate, stream);
  }
  if (n % 4 == 0 && a16(partial))
    hipLaunchKernelGGL(splitk_finish_flat4_kernel, dim3((unsigned)((n / 4 + 255) / 256)), dim3(256), 0,
                       stream, partial, splits, M, N, c, ldc, bias, (int)accumulate);
  else
    hipLaunchKernelGGL(splitk_finish_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream,
                       partial, splits, M, N, c, ldc, bias, (int)accumulate);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !cs_part) return e;
  return parts_finish(cs_part, splits, M, cs_out, accumulate, stream);
}

hipError_t parts_finish(const float* ws, int parts, int64_t N, float* out, bool accumulate,
                        hipStream_t stream) {
  if (N <= 0) return hipSuccess;
  hipLaunchKernelGGL(parts_finish_kernel, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, stream,
                     ws, parts, N, out, (int)accumulate);
  return hipGetLastError();
}

hipError_t fill_f32(float* out, int64_t n, float value, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, out, n,
                     value);
  return hipGetLastError();
}

}  // namespace mt
