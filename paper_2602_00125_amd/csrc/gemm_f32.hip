// fp32 GEMM on CDNA4 matrix cores (v_mfma_f32_32x32x2_f32), gfx950 only.
//
// Computes the three products of the dense layer and of the broadcasting
// matmul (MiniTensor Sec. 3.1 Eq. (1), Sec. 3.2 Eq. (4), Sec. 3.3 Eq. (5)):
//   C[m][n] = sum_k A[m][k] B[k][n]   (+ bias[n]) (+ C[m][n] when accumulating)
// with either operand stored K-contiguous or M/N-contiguous, so one template
// covers Y = X W^T (both K-contiguous), dX = dY W (A K-contiguous, B
// N-contiguous) and dW = dY^T X (both M/N-contiguous).
//
// Block: 256 threads = 4 wave64s in a WGM x WGN grid; each wave owns a
// (BM/WGM) x (BN/WGN) sub-tile made of 32x32 MFMA tiles held in
// accumulator registers. Per K-stage of BK:
//   global -> registers (buffer_load_dwordx4; out-of-range rows and the K
//   tail read as zero through the buffer's range check) for stage s+1 is
//   issued before the MFMAs of stage s, and written to the other half of a
//   double-buffered LDS tile afterwards: one barrier per stage.
// LDS layout follows the global layout of each operand:
//   K-contiguous operand: [BMN][BK+4] floats; a lane reads 4 consecutive k
//   with one ds_read_b128 (the +4 pad puts 8/16 consecutive rows on disjoint
//   banks).
//   M/N-contiguous operand: [BK][BMN+8] floats; a lane reads one float per
//   MFMA step, 32 consecutive lanes on consecutive banks.
// Within a group of 8 k, MFMA step j (0..3) takes k = 8g + 4h + j for lane
// half h, the same on both operands, so the contraction is unchanged.
// The MFMA's row operand is the B tile (n) and its column operand the A tile
// (m): each lane then holds 4 consecutive n of one output row per register
// quad, which the epilogue stores with one 16-byte store (bias added there).
#include <hip/hip_runtime.h>

#include "gemm_params.hpp"
#include "kernels.hpp"

namespace mt {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Offset beyond any buffer's num_records: the hardware returns zeros.
constexpr uint32_t kOOB = 0x80000000u;
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit data format

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff,
                                           kRsrcWord3);
}

template <int VEC>
struct VecT;
template <>
struct VecT<4> {
  using T = f32x4;
  static __device__ __forceinline__ T load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
  }
};
template <>
struct VecT<1> {
  using T = float;
  static __device__ __forceinline__ T load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
  }
};

// One operand's BMN x BK tile: global -> registers -> LDS.
template <bool KC, int BMN, int BK, int VEC>
struct Tile {
  static constexpr int PITCH = KC ? BK + 4 : BMN + 8;  // floats per LDS row
  static constexpr int ROWS = KC ? BMN : BK;
  static constexpr int COLS = KC ? BK : BMN;           // contiguous extent
  static constexpr int SIZE = ROWS * PITCH;            // floats per stage
  static constexpr int VPR = COLS / VEC;               // vectors per row
  static constexpr int PER_THREAD = ROWS * VPR / 256;
  static_assert((ROWS * VPR) % 256 == 0, "tile must split evenly over 256 threads");
  using V = typename VecT<VEC>::T;

  uint32_t off[PER_THREAD];
  int row[PER_THREAD], col[PER_THREAD];
  V reg[PER_THREAD];

  __device__ __forceinline__ void init(int tid, int64_t ld) {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * 256;
      row[i] = c / VPR;
      col[i] = (c % VPR) * VEC;
      off[i] = (uint32_t)(((int64_t)row[i] * ld + col[i]) * 4);
    }
  }
  // base: element (row 0, col 0) of this stage's tile; rows_left/cols_left:
  // how many rows / contiguous elements from there are inside the matrix.
  __device__ __forceinline__ void load(const float* base, int64_t rows_left, int64_t cols_left) {
    const __amdgpu_buffer_rsrc_t r = make_rsrc(base);
    const int rl = rows_left < ROWS ? (int)rows_left : ROWS;
    const int cl = cols_left < COLS ? (int)cols_left : COLS;
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const bool ok = row[i] < rl && col[i] < cl;
      reg[i] = VecT<VEC>::load(r, ok ? off[i] : kOOB);
    }
  }
  __device__ __forceinline__ void store(float* lds) const {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) *(V*)&lds[row[i] * PITCH + col[i]] = reg[i];
  }
};

__device__ __forceinline__ int64_t xcd_remap(int64_t bid, int64_t nb) {
  // Workgroups are dispatched round-robin over the 8 XCDs (block i -> XCD
  // i % 8). Renumber so that consecutive logical ids sit on one XCD and
  // neighbouring tiles share that XCD's L2.
  const int64_t per = nb / 8, rem = nb % 8, x = bid % 8;
  return x * per + (x < rem ? x : rem) + bid / 8;
}

template <bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int VEC, int WAVES_PER_EU>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_f32_kernel(const GemmParams p) {
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  static_assert(WGM * WGN == 4, "4 waves per block");
  static_assert(TM * 32 == WTM && TN * 32 == WTN && BK % 8 == 0, "tile shape");
  using TA = Tile<A_KC, BM, BK, VEC>;
  using TB = Tile<B_KC, BN, BK, VEC>;
  __shared__ __attribute__((aligned(16))) float lds[2 * (TA::SIZE + TB::SIZE)];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int l32 = lane & 31, h = lane >> 5;

  // ---- block -> (split, batch, tile)
  const int64_t tiles = (int64_t)p.tiles_m * p.tiles_n;
  int64_t logical = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t t = logical % tiles;
  logical /= tiles;
  const int64_t batch = logical % p.keep_count;
  const int split = (int)(logical / p.keep_count);
  int tm_idx, tn_idx;
  {
    const int64_t width = (int64_t)p.group_m * p.tiles_n;
    const int64_t gid = t / width;
    const int64_t first = gid * p.group_m;
    const int64_t gsz = (p.tiles_m - first) < p.group_m ? (p.tiles_m - first) : p.group_m;
    tm_idx = (int)(first + (t % width) % gsz);
    tn_idx = (int)((t % width) / gsz);
  }
  const int64_t m0 = (int64_t)tm_idx * BM, n0 = (int64_t)tn_idx * BN;

  int64_t a_off = 0, b_off = 0, c_off = 0;
  {
    int64_t rem = batch;
    for (int d = p.nkeep - 1; d >= 0; --d) {
      const int64_t i = rem % p.keep_shape[d];
      rem /= p.keep_shape[d];
      a_off += i * p.keep_sa[d];
      b_off += i * p.keep_sb[d];
      c_off += i * p.keep_sc[d];
    }
  }
  const float* A = (const float*)p.a + a_off;
  const float* B = (const float*)p.b + b_off;

  const int64_t k_begin = (int64_t)split * p.k_per_split;
  const int64_t k_end = (k_begin + p.k_per_split) < p.K ? (k_begin + p.k_per_split) : p.K;
  const int64_t KS = k_end > k_begin ? (k_end - k_begin + BK - 1) / BK : 0;
  const int64_t S = KS * p.red_count;

  TA ta;
  TB tb;
  ta.init(tid, p.lda);
  tb.init(tid, p.ldb);

  // stage cursor (reduction index r, k tile kt) with r's operand offsets
  int64_t cur_r = 0, cur_kt = 0, ra_off = 0, rb_off = 0;
  auto red_offsets = [&](int64_t r) {
    ra_off = 0;
    rb_off = 0;
    for (int d = p.nred - 1; d >= 0; --d) {
      const int64_t i = r % p.red_shape[d];
      r /= p.red_shape[d];
      ra_off += i * p.red_sa[d];
      rb_off += i * p.red_sb[d];
    }
  };
  auto load_stage = [&]() {
    const int64_t k0 = k_begin + cur_kt * BK;
    const float* Ar = A + ra_off;
    const float* Br = B + rb_off;
    if (A_KC) ta.load(Ar + m0 * p.lda + k0, p.M - m0, k_end - k0);
    else ta.load(Ar + k0 * p.lda + m0, k_end - k0, p.M - m0);
    if (B_KC) tb.load(Br + n0 * p.ldb + k0, p.N - n0, k_end - k0);
    else tb.load(Br + k0 * p.ldb + n0, k_end - k0, p.N - n0);
  };
  auto advance = [&]() {
    if (++cur_kt == KS) {
      cur_kt = 0;
      ++cur_r;
      if (cur_r < p.red_count) red_offsets(cur_r);
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};

  if (S > 0) {
    if (p.nred > 0) red_offsets(0);
    load_stage();
    advance();
    ta.store(lds);
    tb.store(lds + TA::SIZE);
    __syncthreads();
  }
  for (int64_t s = 0; s < S; ++s) {
    const int cur = (int)(s & 1);
    const bool more = s + 1 < S;
    if (more) {
      load_stage();
      advance();
    }
    const float* As = lds + cur * (TA::SIZE + TB::SIZE);
    const float* Bs = As + TA::SIZE;
#pragma unroll
    for (int g = 0; g < BK / 8; ++g) {
      float af[4][TM], bf[4][TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int mm = wm * WTM + i * 32 + l32;
        if (A_KC) {
          const f32x4 v = *(const f32x4*)&As[mm * TA::PITCH + 8 * g + 4 * h];
          af[0][i] = v[0];
          af[1][i] = v[1];
          af[2][i] = v[2];
          af[3][i] = v[3];
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) af[j][i] = As[(8 * g + 4 * h + j) * TA::PITCH + mm];
        }
      }
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int nn = wn * WTN + i * 32 + l32;
        if (B_KC) {
          const f32x4 v = *(const f32x4*)&Bs[nn * TB::PITCH + 8 * g + 4 * h];
          bf[0][i] = v[0];
          bf[1][i] = v[1];
          bf[2][i] = v[2];
          bf[3][i] = v[3];
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) bf[j][i] = Bs[(8 * g + 4 * h + j) * TB::PITCH + nn];
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int q = 0; q < TN; ++q)
            acc[i][q] = __builtin_amdgcn_mfma_f32_32x32x2f32(bf[j][q], af[j][i], acc[i][q], 0, 0, 0);
    }
    if (more) {
      float* nxt = lds + (cur ^ 1) * (TA::SIZE + TB::SIZE);
      ta.store(nxt);
      tb.store(nxt + TA::SIZE);
    }
    __syncthreads();
  }

  // ---- epilogue: lane holds C[m][n0' + 8g + 4h + 0..3] in acc regs 4g..4g+3
  const bool to_partial = p.splits > 1;
  float* C = to_partial ? p.partial + (int64_t)split * p.partial_stride : p.c + c_off;
  const int64_t ldc = to_partial ? p.N : p.ldc;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int64_t m = m0 + wm * WTM + i * 32 + l32;
    if (m >= p.M) continue;
    float* crow = C + m * ldc;
#pragma unroll
    for (int q = 0; q < TN; ++q) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t n = n0 + wn * WTN + q * 32 + 8 * g + 4 * h;
        f32x4 v = {acc[i][q][4 * g + 0], acc[i][q][4 * g + 1], acc[i][q][4 * g + 2],
                   acc[i][q][4 * g + 3]};
        if (VEC == 4) {
          // N % 4 == 0, ldc % 4 == 0 and 16-byte aligned C / bias (host-checked)
          if (n >= p.N) continue;
          if (!to_partial) {
            if (p.bias) v += *(const f32x4*)&p.bias[n];
            if (p.accumulate) v += *(const f32x4*)&crow[n];
          }
          *(f32x4*)&crow[n] = v;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (n + e >= p.N) continue;
            float x = v[e];
            if (!to_partial) {
              if (p.bias) x += p.bias[n + e];
              if (p.accumulate) x += crow[n + e];
            }
            crow[n + e] = x;
          }
        }
      }
    }
  }
}

}  // namespace

// ---------------------------------------------------------------- configs --

template <bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int VEC, int WPE>
static hipError_t launch_cfg(const GemmParams& p, hipStream_t stream) {
  GemmParams q = p;
  q.tiles_m = (int32_t)((p.M + BM - 1) / BM);
  q.tiles_n = (int32_t)((p.N + BN - 1) / BN);
  const int64_t blocks = (int64_t)q.tiles_m * q.tiles_n * p.keep_count * p.splits;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((gemm_f32_kernel<A_KC, B_KC, BM, BN, BK, WGM, WGN, VEC, WPE>),
                     dim3((unsigned)blocks), dim3(256), 0, stream, q);
  return hipGetLastError();
}

template <bool A_KC, bool B_KC, int VEC>
static hipError_t launch_layout(const GemmParams& p, int cfg, hipStream_t stream) {
  switch (cfg) {
    case kCfg256x256:
      return launch_cfg<A_KC, B_KC, 256, 256, 16, 2, 2, VEC, 1>(p, stream);
    case kCfg256x128:
      return launch_cfg<A_KC, B_KC, 256, 128, 16, 2, 2, VEC, 2>(p, stream);
    case kCfg128x256:
      return launch_cfg<A_KC, B_KC, 128, 256, 16, 2, 2, VEC, 2>(p, stream);
    case kCfg128x128:
      return launch_cfg<A_KC, B_KC, 128, 128, 16, 2, 2, VEC, 2>(p, stream);
    default:
      return launch_cfg<A_KC, B_KC, 64, 64, 16, 2, 2, VEC, 4>(p, stream);
  }
}

int gemm_tile_m(int cfg) {
  switch (cfg) {
    case kCfg256x256: case kCfg256x128: return 256;
    case kCfg128x256: case kCfg128x128: return 128;
    default: return 64;
  }
}
int gemm_tile_n(int cfg) {
  switch (cfg) {
    case kCfg256x256: case kCfg128x256: return 256;
    case kCfg256x128: case kCfg128x128: return 128;
    default: return 64;
  }
}
int gemm_tile_k(int) { return 16; }

hipError_t gemm_f32(const GemmParams& p, bool a_kc, bool b_kc, bool vec4, int cfg,
                    hipStream_t stream) {
  if (vec4) {
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
