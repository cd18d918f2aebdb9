// HBM-bound kernels of the training step around the dense layer, gfx950.
//
// * act_bwd: the pullback of H = act(Z) (MiniTensor Sec. 3.3 nonlinearities,
//   chain rule of Sec. 3.2): dZ = dH * act'(Z) elementwise, with the bias
//   gradient db = 1^T dZ (add pullback through the broadcast bias) summed in
//   the same pass, so dZ is read from HBM by the GEMMs only. Layout and
//   reduction order follow colsum: lanes run along the contiguous n (four
//   columns per lane, 16-byte loads), the sixteen waves of a block take
//   interleaved rows, partial sums meet in LDS in wave order, row slices go
//   to a workspace that a second pass adds in slice order (deterministic).
// * mse: L = (1/N) sum (P - T)^2 and dP = 2 (P - T) / N (Sec. 3.3 losses):
//   each block sums its grid-stride share in a fixed order and writes one
//   partial; a one-block pass adds the partials in order.
// * optimizer steps (Sec. 3.3 Eq. (9), Eq. (10), RMSprop): several parameter
//   tensors in one launch; each block finds its tensor in a prefix table of
//   block counts and updates a contiguous chunk of it in place, 16-byte
//   accesses where every pointer of the tensor allows them.
#include <hip/hip_runtime.h>

#include "act.hpp"
#include "kernels.hpp"

namespace mt {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(unsigned short v) {
  return __uint_as_float((unsigned)v << 16);
}

// fp32 -> bf16, round to nearest even (a NaN stays a quiet NaN)
__device__ __forceinline__ unsigned short f32_to_bf16(float f) {
  const unsigned u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (unsigned short)((u >> 16) | 0x40);
  return (unsigned short)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

template <bool BF16>
__device__ __forceinline__ f32x4 ld4(const void* base, int64_t idx) {
  if constexpr (BF16) {
    const u16x4 v = *(const u16x4*)((const unsigned short*)base + idx);
    return f32x4{bf16_to_f32(v[0]), bf16_to_f32(v[1]), bf16_to_f32(v[2]), bf16_to_f32(v[3])};
  } else {
    return *(const f32x4*)((const float*)base + idx);
  }
}
template <bool BF16>
__device__ __forceinline__ void st4(void* base, int64_t idx, f32x4 v) {
  if constexpr (BF16) {
    *(u16x4*)((unsigned short*)base + idx) =
        u16x4{f32_to_bf16(v[0]), f32_to_bf16(v[1]), f32_to_bf16(v[2]), f32_to_bf16(v[3])};
  } else {
    *(f32x4*)((float*)base + idx) = v;
  }
}
template <bool BF16>
__device__ __forceinline__ float ld1(const void* base, int64_t idx) {
  if constexpr (BF16) return bf16_to_f32(((const unsigned short*)base)[idx]);
  else return ((const float*)base)[idx];
}
template <bool BF16>
__device__ __forceinline__ void st1(void* base, int64_t idx, float v) {
  if constexpr (BF16) ((unsigned short*)base)[idx] = f32_to_bf16(v);
  else ((float*)base)[idx] = v;
}

// dz[m][n] (+)= dh[m][n] * act'(z[m][n]); column sums of the new terms.
// grid: (ceil(N / (64 VEC)), parts); block: WAVES wave64s.
template <bool BF16, int VEC, int WAVES, bool DB>
__global__ __launch_bounds__(WAVES * 64) void act_bwd_kernel(
    int act, const float* z, int64_t ldz, const void* dh, int64_t ldh, void* dz, int64_t ldd,
    int64_t M, int64_t N, int acc_dz, float* db, int acc_db, float* ws, int64_t rows_per_part) {
  __shared__ f32x4 red[DB ? WAVES : 1][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t n = ((int64_t)blockIdx.x * 64 + lane) * VEC;
  const int64_t r0 = (int64_t)blockIdx.y * rows_per_part;
  const int64_t r1 = (r0 + rows_per_part) < M ? (r0 + rows_per_part) : M;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (n < N) {
    if constexpr (VEC == 4) {
      auto one = [&](int64_t m) {
        const f32x4 zz = *(const f32x4*)(z + m * ldz + n);
        const f32x4 g = ld4<BF16>(dh, m * ldh + n);
        f32x4 d;
#pragma unroll
        for (int e = 0; e < 4; ++e) d[e] = g[e] * act_grad(act, zz[e]);
        if (DB) acc += d;
        if (acc_dz) d += ld4<BF16>(dz, m * ldd + n);
        st4<BF16>(dz, m * ldd + n, d);
      };
      int64_t m = r0 + wave;
      // two rows in flight per lane (the loads of both issue before either's math)
      for (; m + WAVES < r1; m += 2 * WAVES) {
        one(m);
        one(m + WAVES);
      }
      for (; m < r1; m += WAVES) one(m);
    } else {
      for (int64_t m = r0 + wave; m < r1; m += WAVES) {
        float d = ld1<BF16>(dh, m * ldh + n) * act_grad(act, z[m * ldz + n]);
        if (DB) acc[0] += d;
        if (acc_dz) d += ld1<BF16>(dz, m * ldd + n);
        st1<BF16>(dz, m * ldd + n, d);
      }
    }
  }
  if constexpr (DB) {
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
          if (n + e < N) db[n + e] = acc_db ? db[n + e] + s[e] : s[e];
      }
    }
  }
}

// ---- mean squared error

constexpr int kMseThreads = 256;

// Block b sums (p - t)^2 over elements i = (b * 256 + tid) * 4 + 0..3 and then
// every (grid * 256 * 4) further, in that order per thread; the 256 thread
// sums are added by a fixed tree in LDS. dp = 2 (p - t) / N on the way.
template <int VEC>
__global__ __launch_bounds__(kMseThreads) void mse_kernel(const float* p, const float* t, int64_t n,
                                                          float inv_n, float* dp, float* partial,
                                                          float* loss) {
  __shared__ float red[kMseThreads];
  const int tid = threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * kMseThreads * VEC;
  float s = 0.f;
  for (int64_t i = ((int64_t)blockIdx.x * kMseThreads + tid) * VEC; i < n; i += stride) {
    if (VEC == 4 && i + 4 <= n) {
      const f32x4 a = *(const f32x4*)(p + i), b = *(const f32x4*)(t + i);
      const f32x4 d = a - b;
      s += d[0] * d[0];
      s += d[1] * d[1];
      s += d[2] * d[2];
      s += d[3] * d[3];
      if (dp) *(f32x4*)(dp + i) = d * (2.f * inv_n);
    } else {
      for (int e = 0; e < VEC && i + e < n; ++e) {
        const float d = p[i + e] - t[i + e];
        s += d * d;
        if (dp) dp[i + e] = d * (2.f * inv_n);
      }
    }
  }
  red[tid] = s;
  __syncthreads();
  for (int w = kMseThreads / 2; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  if (tid == 0) {
    if (partial) partial[blockIdx.x] = red[0];
    else if (loss) *loss = red[0] * inv_n;
  }
}

// loss = (sum of the partials in block order) / N, one block.
__global__ __launch_bounds__(kMseThreads) void mse_finish_kernel(const float* partial, int parts,
                                                                 float inv_n, float* loss) {
  __shared__ float red[kMseThreads];
  const int tid = threadIdx.x;
  float s = 0.f;
  for (int i = tid; i < parts; i += kMseThreads) s += partial[i];
  red[tid] = s;
  __syncthreads();
  for (int w = kMseThreads / 2; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  if (tid == 0 && loss) *loss = red[0] * inv_n;
}

// ---- optimizer steps

constexpr int kOptThreads = 256;
constexpr int kOptPerThread = 16;  // elements per thread per block (4 x 16 bytes)
constexpr int64_t kOptChunk = (int64_t)kOptThreads * kOptPerThread;

__device__ __forceinline__ int find_tensor(const OptBatch& b, int64_t blk) {
  int t = 0;
  while (t + 1 < b.n && b.block_start[t + 1] <= blk) ++t;
  return t;
}

struct SgdOp {
  float lr, mu, wd;
  __device__ __forceinline__ void operator()(float& th, float g, float& v, float&) const {
    v = mu * v + (g + wd * th);
    th = th - lr * v;
  }
};
struct AdamOp {
  float lr, b1, b2, eps, inv_bc1, inv_bc2;
  __device__ __forceinline__ void operator()(float& th, float g, float& m, float& v) const {
    m = b1 * m + (1.f - b1) * g;
    v = b2 * v + (1.f - b2) * (g * g);
    const float mhat = m * inv_bc1;
    const float vhat = v * inv_bc2;
    th = th - lr * (mhat / (sqrtf(vhat) + eps));
  }
};
struct RmspropOp {
  float lr, alpha, eps;
  __device__ __forceinline__ void operator()(float& th, float g, float& v, float&) const {
    v = alpha * v + (1.f - alpha) * (g * g);
    th = th - lr * (g / sqrtf(v + eps));
  }
};

// Block blk updates elements [c0, c0 + kOptChunk) of its tensor: lane i takes
// the 16-byte groups i, i + 256, ... (coalesced), or single elements when
// the tensor's pointers do not all allow 16-byte access.
template <typename Op, bool TWO_STATES>
__global__ __launch_bounds__(kOptThreads) void opt_kernel(const OptBatch b, const Op op) {
  const int64_t blk = blockIdx.x;
  const int t = find_tensor(b, blk);
  const int64_t c0 = (blk - b.block_start[t]) * kOptChunk;
  const int64_t n = b.numel[t];
  float* th = b.param[t];
  const float* g = b.grad[t];
  float* s1 = b.state1[t];
  float* s2 = TWO_STATES ? b.state2[t] : nullptr;
  const bool vec = b.vec[t] != 0;
  const int tid = threadIdx.x;
  if (vec && c0 + kOptChunk <= n) {
    // every load of the thread's groups goes out before the first store (the
    // compiler cannot move a load past a store to a pointer it may alias)
    constexpr int G = kOptPerThread / 4;
    f32x4 p4[G], g4[G], a4[G], b4[G];
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const int64_t i = c0 + ((int64_t)j * kOptThreads + tid) * 4;
      p4[j] = *(const f32x4*)(th + i);
      g4[j] = *(const f32x4*)(g + i);
      a4[j] = *(const f32x4*)(s1 + i);
      b4[j] = TWO_STATES ? *(const f32x4*)(s2 + i) : f32x4{};
    }
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const int64_t i = c0 + ((int64_t)j * kOptThreads + tid) * 4;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float pe = p4[j][e], ae = a4[j][e], be = b4[j][e];
        op(pe, g4[j][e], ae, be);
        p4[j][e] = pe;
        a4[j][e] = ae;
        b4[j][e] = be;
      }
      *(f32x4*)(th + i) = p4[j];
      *(f32x4*)(s1 + i) = a4[j];
      if (TWO_STATES) *(f32x4*)(s2 + i) = b4[j];
    }
  } else {
    for (int j = 0; j < kOptPerThread; ++j) {
      const int64_t i = c0 + (int64_t)j * kOptThreads + tid;
      if (i >= n) break;
      float pe = th[i], ae = s1[i], be = TWO_STATES ? s2[i] : 0.f;
      op(pe, g[i], ae, be);
      th[i] = pe;
      s1[i] = ae;
      if (TWO_STATES) s2[i] = be;
    }
  }
}

template <typename Op, bool TWO>
hipError_t launch_opt(OptBatch b, const Op& op, hipStream_t stream) {
  int64_t blocks = 0;
  for (int i = 0; i < b.n; ++i) {
    b.block_start[i] = blocks;
    blocks += (b.numel[i] + kOptChunk - 1) / kOptChunk;
  }
  for (int i = b.n; i <= kOptMaxTensors; ++i) b.block_start[i] = blocks;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((opt_kernel<Op, TWO>), dim3((unsigned)blocks), dim3(kOptThreads), 0, stream,
                     b, op);
  return hipGetLastError();
}

}  // namespace

constexpr int kActBwdWaves = 16;

hipError_t act_bwd(int act, const float* z, int64_t ldz, const void* dh, int64_t ldh, void* dz,
                   int64_t ldd, bool is_bf16, int64_t M, int64_t N, bool acc_dz, float* db,
                   bool acc_db, float* ws, int parts, hipStream_t stream) {
  if (M <= 0 || N <= 0) {
    // no rows: db is a sum of nothing
    if (db && N > 0 && !acc_db) return fill_f32(db, N, 0.f, stream);
    return hipSuccess;
  }
  if (!db || !ws) parts = 1;
  const int es = is_bf16 ? 2 : 4;
  const bool vec = N % 4 == 0 && ldz % 4 == 0 && ldh % 4 == 0 && ldd % 4 == 0 &&
                   (uintptr_t)z % 16 == 0 && (uintptr_t)dh % (4 * es) == 0 &&
                   (uintptr_t)dz % (4 * es) == 0;
  const int64_t rows_per_part = (M + parts - 1) / parts;
  const int V = vec ? 4 : 1;
  dim3 grid((unsigned)((N + 64 * V - 1) / (64 * V)), (unsigned)parts);
  dim3 block(kActBwdWaves * 64);
#define MT_ACT_BWD(BF, VV, DBF)                                                                   \
  hipLaunchKernelGGL((act_bwd_kernel<BF, VV, kActBwdWaves, DBF>), grid, block, 0, stream, act, z, \
                     ldz, dh, ldh, dz, ldd, M, N, (int)acc_dz, db, (int)acc_db, ws, rows_per_part)
  if (vec) {
    if (is_bf16) { if (db) MT_ACT_BWD(true, 4, true); else MT_ACT_BWD(true, 4, false); }
    else { if (db) MT_ACT_BWD(false, 4, true); else MT_ACT_BWD(false, 4, false); }
  } else {
    if (is_bf16) { if (db) MT_ACT_BWD(true, 1, true); else MT_ACT_BWD(true, 1, false); }
    else { if (db) MT_ACT_BWD(false, 1, true); else MT_ACT_BWD(false, 1, false); }
  }
#undef MT_ACT_BWD
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !db || parts == 1) return e;
  return parts_finish(ws, parts, N, db, acc_db, stream);
}

int mse_parts(int64_t n) {
  // ~ one block per CU with 64 KB of loads each at least
  int64_t parts = (n + 16383) / 16384;
  if (parts > 1024) parts = 1024;
  if (parts < 1) parts = 1;
  return (int)parts;
}

hipError_t mse(const float* p, const float* t, int64_t n, float* dp, float* loss, float* ws,
               int parts, hipStream_t stream) {
  if (n <= 0) {
    if (loss) return fill_f32(loss, 1, 0.f, stream);
    return hipSuccess;
  }
  if (!ws) parts = 1;
  const float inv_n = (float)(1.0 / (double)n);
  const bool vec = (uintptr_t)p % 16 == 0 && (uintptr_t)t % 16 == 0 &&
                   (!dp || (uintptr_t)dp % 16 == 0);
  if (vec)
    hipLaunchKernelGGL((mse_kernel<4>), dim3((unsigned)parts), dim3(kMseThreads), 0, stream, p, t, n,
                       inv_n, dp, parts > 1 ? ws : nullptr, loss);
  else
    hipLaunchKernelGGL((mse_kernel<1>), dim3((unsigned)parts), dim3(kMseThreads), 0, stream, p, t, n,
                       inv_n, dp, parts > 1 ? ws : nullptr, loss);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || parts == 1) return e;
  hipLaunchKernelGGL(mse_finish_kernel, dim3(1), dim3(kMseThreads), 0, stream, ws, parts, inv_n,
                     loss);
  return hipGetLastError();
}

hipError_t sgd_step(const OptBatch& b, float lr, float momentum, float weight_decay,
                    hipStream_t stream) {
  return launch_opt<SgdOp, false>(b, SgdOp{lr, momentum, weight_decay}, stream);
}

hipError_t adam_step(const OptBatch& b, float lr, float beta1, float beta2, float eps,
                     float inv_bc1, float inv_bc2, hipStream_t stream) {
  return launch_opt<AdamOp, true>(b, AdamOp{lr, beta1, beta2, eps, inv_bc1, inv_bc2}, stream);
}

hipError_t rmsprop_step(const OptBatch& b, float lr, float alpha, float eps, hipStream_t stream) {
  return launch_opt<RmspropOp, false>(b, RmspropOp{lr, alpha, eps}, stream);
}

}  // namespace mt
