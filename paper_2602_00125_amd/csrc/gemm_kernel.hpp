// GEMM kernel template on CDNA4 matrix cores, gfx950 only. Instantiated by
// gemm_f32.hip (fp32 operands, v_mfma_f32_32x32x2_f32) and gemm_bf16.hip
// (bf16 operands, v_mfma_f32_32x32x16_bf16); fp32 accumulation and output.
//
// Computes the products of the dense layer and of the broadcasting matmul
// (MiniTensor Sec. 3.1 Eq. (1), Sec. 3.2 Eq. (4), Sec. 3.3 Eq. (5)):
//   C[m][n] = sum_k A[m][k] B[k][n]   (+ bias[n]) (+ C[m][n] when accumulating)
// with either operand stored K-contiguous or M/N-contiguous, so one template
// covers Y = X W^T (both K-contiguous), dX = dY W (A K-contiguous, B
// N-contiguous) and dW = dY^T X (both M/N-contiguous).
//
// Block: 4 or 8 wave64s in a WGM x WGN grid; each wave owns a
// (BM/WGM) x (BN/WGN) sub-tile made of 32x32 MFMA tiles held in accumulator
// registers. Per K-stage of BK:
//   global -> registers (16-byte buffer_load_dwordx4; out-of-range rows and
//   the K tail read as zero through the buffer's range check) for stage s+1
//   is issued before the MFMAs of stage s, and written to the other half of
//   a double-buffered LDS tile afterwards: one barrier per stage.
// LDS layout follows the global layout of each operand:
//   K-contiguous operand: [BMN][BK + 16 bytes]; a lane fetches 16 bytes of
//   consecutive k with one ds_read_b128 (the pad puts 8/16 consecutive rows
//   on disjoint banks).
//   M/N-contiguous operand: [BK][BMN + 8 elements]; consecutive lanes read
//   consecutive m/n, i.e. consecutive banks.
// fp32: within a group of 8 k, MFMA step j (0..3) takes k = 8g + 4h + j for
// lane half h on both operands, so one ds_read_b128 feeds 4 steps.
// bf16: one MFMA step covers 16 k; lane half h supplies k = 16s + 8h + 0..7
// (one ds_read_b128 from a K-contiguous tile, two transposing
// ds_read_b64_tr_b16 from an M/N-contiguous one).
// The MFMA's row operand is the B tile (n) and its column operand the A tile
// (m): each lane then holds 4 consecutive n of one output row per register
// quad, which the epilogue stores with one 16-byte store (bias added there).
#pragma once
#include <hip/hip_runtime.h>

#include "act.hpp"
#include "gemm_params.hpp"

namespace mt {
namespace gemm {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

// Offset beyond any buffer's num_records: the hardware returns zeros.
constexpr uint32_t kOOB = 0x80000000u;
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit data format

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff,
                                           kRsrcWord3);
}

// A chunk of VEC elements of ESIZE bytes moved by one load / one LDS store.
template <int BYTES>
struct Chunk;
template <>
struct Chunk<16> {
  using T = i32x4;
  static __device__ __forceinline__ T load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  }
};
template <>
struct Chunk<4> {
  using T = int;
  static __device__ __forceinline__ T load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
  }
};
template <>
struct Chunk<2> {
  using T = unsigned short;
  static __device__ __forceinline__ T load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(unsigned short, __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0));
  }
};

// One operand's BMN x BK tile: global -> registers -> LDS. Sizes in elements
// of ESIZE bytes; LDS addressed in bytes.
template <int ESIZE, bool KC, int BMN, int BK, int VEC, int NT>
struct Tile {
  // K-contiguous rows: +16 bytes (an odd multiple of 16 bytes between rows
  // keeps 16-byte reads of consecutive rows conflict-free). M/N-contiguous
  // rows: fp32 +8 elements; bf16 +MT_BF16_MC_PAD elements (rows 64 bytes
  // apart modulo 256: the 4 rows x 2 column halves that two 16-lane groups
  // of ds_read_b64_tr_b16 read together fall on disjoint banks).
#ifndef MT_BF16_MC_PAD
#define MT_BF16_MC_PAD 32
#endif
  static constexpr int PAD = KC ? 16 / ESIZE : (ESIZE == 2 ? MT_BF16_MC_PAD : 8);  // elements
  static constexpr int PITCH = (KC ? BK : BMN) + PAD;       // elements per LDS row
  static constexpr int ROWS = KC ? BMN : BK;
  static constexpr int COLS = KC ? BK : BMN;                // contiguous extent
  static constexpr int BYTES = ROWS * PITCH * ESIZE;        // per stage
  static constexpr int VPR = COLS / VEC;                    // chunks per row
  static constexpr int PER_THREAD = ROWS * VPR / NT;
  static_assert((ROWS * VPR) % NT == 0, "tile must split evenly over the block's threads");
  static_assert((PITCH * ESIZE) % 16 == 0, "LDS rows stay 16-byte aligned");
  using C = Chunk<VEC * ESIZE>;
  using V = typename C::T;

  uint32_t off[PER_THREAD];
  int row[PER_THREAD], col[PER_THREAD];
  V reg[PER_THREAD];

  __device__ __forceinline__ void init(int tid, int64_t ld) {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * NT;
      row[i] = c / VPR;
      col[i] = (c % VPR) * VEC;
      off[i] = (uint32_t)(((int64_t)row[i] * ld + col[i]) * ESIZE);
    }
  }
  // base: element (row 0, col 0) of this stage's tile; rows_left/cols_left:
  // how many rows / contiguous elements from there are inside the matrix.
  __device__ __forceinline__ void load(const char* base, int64_t rows_left, int64_t cols_left) {
    const __amdgpu_buffer_rsrc_t r = make_rsrc(base);
    const int rl = rows_left < ROWS ? (int)rows_left : ROWS;
    const int cl = cols_left < COLS ? (int)cols_left : COLS;
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const bool ok = row[i] < rl && col[i] < cl;
      reg[i] = C::load(r, ok ? off[i] : kOOB);
    }
  }
  __device__ __forceinline__ void store(char* lds) const {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) *(V*)&lds[(row[i] * PITCH + col[i]) * ESIZE] = reg[i];
  }
};

__device__ __forceinline__ int64_t xcd_remap(int64_t bid, int64_t nb) {
  // Workgroups are dispatched round-robin over the 8 XCDs (block i -> XCD
  // i % 8). Renumber so that consecutive logical ids sit on one XCD and
  // neighbouring tiles share that XCD's L2.
  const int64_t per = nb / 8, rem = nb % 8, x = bid % 8;
  return x * per + (x < rem ? x : rem) + bid / 8;
}

// MFMA work on one LDS stage. fp32 and bf16 specialisations.
template <typename T, bool A_KC, bool B_KC, int TM, int TN, int BK, int PA, int PB>
struct Mma;

template <bool A_KC, bool B_KC, int TM, int TN, int BK, int PA, int PB>
struct Mma<float, A_KC, B_KC, TM, TN, BK, PA, PB> {
  static __device__ __forceinline__ void run(const float* As, const float* Bs, int am, int bn,
                                             int l32, int h, f32x16 (&acc)[TM][TN]) {
#pragma unroll
    for (int g = 0; g < BK / 8; ++g) {
      float af[4][TM], bf[4][TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int mm = am + i * 32 + l32;
        if (A_KC) {
          const f32x4 v = *(const f32x4*)&As[mm * PA + 8 * g + 4 * h];
          af[0][i] = v[0];
          af[1][i] = v[1];
          af[2][i] = v[2];
          af[3][i] = v[3];
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) af[j][i] = As[(8 * g + 4 * h + j) * PA + mm];
        }
      }
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int nn = bn + i * 32 + l32;
        if (B_KC) {
          const f32x4 v = *(const f32x4*)&Bs[nn * PB + 8 * g + 4 * h];
          bf[0][i] = v[0];
          bf[1][i] = v[1];
          bf[2][i] = v[2];
          bf[3][i] = v[3];
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) bf[j][i] = Bs[(8 * g + 4 * h + j) * PB + nn];
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
  }
};

template <bool A_KC, bool B_KC, int TM, int TN, int BK, int PA, int PB>
struct Mma<__bf16, A_KC, B_KC, TM, TN, BK, PA, PB> {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  // 8 consecutive k (k0 .. k0+7) of row/column mn for this lane.
  // K-contiguous tile [mn][k]: one 16-byte read.
  // M/N-contiguous tile [k][mn]: two ds_read_b64_tr_b16. Within each group of
  // 16 lanes, lane i of the group receives element i % 4 of the 8-byte
  // chunks addressed by lanes i/4, 4 + i/4, 8 + i/4, 12 + i/4 of the group.
  // Lane s of a group therefore addresses row k + s/4, columns
  // c0 + 4 (s % 4) .. +3, where c0 is the group's first column, and lane i
  // receives column c0 + i at rows k .. k+3.
  static __device__ __forceinline__ u16x8 frag_kc(const unsigned short* S, int P, int mn, int k0) {
    return *(const u16x8*)&S[mn * P + k0];
  }
  static __device__ __forceinline__ u16x8 frag_mc(const unsigned short* S, int P, int col0, int k0,
                                                  int lane) {
    const int g = lane >> 4, s = lane & 15;
    const int row = k0 + (s >> 2);
    const int col = col0 + 16 * (g & 1) + 4 * (s & 3);
    const unsigned short* p0 = &S[row * P + col];
    const unsigned short* p1 = p0 + 4 * P;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(const void*)p0);
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(const void*)p1);
    u16x8 v;
    v[0] = lo[0]; v[1] = lo[1]; v[2] = lo[2]; v[3] = lo[3];
    v[4] = hi[0]; v[5] = hi[1]; v[6] = hi[2]; v[7] = hi[3];
    return v;
  }
  static __device__ __forceinline__ void run(const unsigned short* As, const unsigned short* Bs,
                                             int am, int bn, int l32, int h,
                                             f32x16 (&acc)[TM][TN]) {
    const int lane = l32 + 32 * h;
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      const int k0 = 16 * s + 8 * h;
      u16x8 af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = A_KC ? frag_kc(As, PA, am + i * 32 + l32, k0) : frag_mc(As, PA, am + i * 32, k0, lane);
#pragma unroll
      for (int i = 0; i < TN; ++i)
        bf[i] = B_KC ? frag_kc(Bs, PB, bn + i * 32 + l32, k0) : frag_mc(Bs, PB, bn + i * 32, k0, lane);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int q = 0; q < TN; ++q)
          acc[i][q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, bf[q]),
                                                               __builtin_bit_cast(bf16x8, af[i]),
                                                               acc[i][q], 0, 0, 0);
    }
  }
};

template <typename T> struct LdsElem { using type = T; };
template <> struct LdsElem<__bf16> { using type = unsigned short; };

// Epilogue of the dense layer followed by a nonlinearity (Sec. 3.3 Eq. (5),
// "Nonlinearities"): z = acc + b[n] is stored when p.z is set and act(z) goes
// to C. No batch, split or accumulation (the host guarantees it). The lane
// holds C[m0l + 32 i][n0l + 32 q + 8 g + 0..3] in acc[i][q][4g .. 4g+3]. One
// copy per nonlinearity: the switch is taken once per block, outside the
// unrolled stores.
template <int ACT, int TM, int TN, bool VEC_C>
__device__ __forceinline__ void act_store(const GemmParams& p, const f32x16 (&acc)[TM][TN],
                                          int64_t m0l, int64_t n0l) {
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int64_t m = m0l + i * 32;
    if (m >= p.M) continue;
    float* crow = p.c + m * p.ldc;
    float* zrow = p.z ? p.z + m * p.ldz : nullptr;
#pragma unroll
    for (int q = 0; q < TN; ++q) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t n = n0l + q * 32 + 8 * g;
        f32x4 v = {acc[i][q][4 * g + 0], acc[i][q][4 * g + 1], acc[i][q][4 * g + 2],
                   acc[i][q][4 * g + 3]};
        if (VEC_C) {
          if (n >= p.N) continue;
          if (p.bias) v += *(const f32x4*)&p.bias[n];
          if (zrow) *(f32x4*)&zrow[n] = v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = act_apply_t<ACT>(v[e]);
          *(f32x4*)&crow[n] = v;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (n + e >= p.N) continue;
            float x = v[e];
            if (p.bias) x += p.bias[n + e];
            if (zrow) zrow[n + e] = x;
            crow[n + e] = act_apply_t<ACT>(x);
          }
        }
      }
    }
  }
}

template <int TM, int TN, bool VEC_C>
__device__ __forceinline__ void act_epilogue(const GemmParams& p, const f32x16 (&acc)[TM][TN],
                                             int64_t m0l, int64_t n0l) {
  switch (p.act) {
    case kActRelu: act_store<kActRelu, TM, TN, VEC_C>(p, acc, m0l, n0l); break;
    case kActSigmoid: act_store<kActSigmoid, TM, TN, VEC_C>(p, acc, m0l, n0l); break;
    case kActTanh: act_store<kActTanh, TM, TN, VEC_C>(p, acc, m0l, n0l); break;
    case kActGelu: act_store<kActGelu, TM, TN, VEC_C>(p, acc, m0l, n0l); break;
    default: act_store<kActNone, TM, TN, VEC_C>(p, acc, m0l, n0l); break;
  }
}

// EPI: the dense-layer-with-nonlinearity epilogue (act_epilogue) instead of
// the plain one; instantiated only for the forward layout and a few tiles.
template <typename T, bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int VEC,
          int WAVES_PER_EU, bool EPI = false>
__global__ __launch_bounds__(WGM * WGN * 64)
__attribute__((amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_kernel(const GemmParams p) {
  constexpr int ES = (int)sizeof(T);
  constexpr int NT = WGM * WGN * 64;  // threads per block
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  static_assert(WGM * WGN == 4 || WGM * WGN == 8, "4 or 8 waves per block");
  static_assert(TM * 32 == WTM && TN * 32 == WTN && BK % 16 == 0, "tile shape");
  using TA = Tile<ES, A_KC, BM, BK, VEC, NT>;
  using TB = Tile<ES, B_KC, BN, BK, VEC, NT>;
  using E = typename LdsElem<T>::type;
  __shared__ __attribute__((aligned(16))) char lds[2 * (TA::BYTES + TB::BYTES)];

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
  const char* A = (const char*)p.a + a_off * ES;
  const char* B = (const char*)p.b + b_off * ES;

  const int64_t KS = (p.K + BK - 1) / BK;  // k tiles per summed batch index
  const int64_t S_all = KS * p.red_count;
  const int64_t st0 = (int64_t)split * p.stages_per_split;
  const int64_t st1 = (st0 + p.stages_per_split) < S_all ? (st0 + p.stages_per_split) : S_all;
  const int64_t S = st1 > st0 ? st1 - st0 : 0;

  TA ta;
  TB tb;
  ta.init(tid, p.lda);
  tb.init(tid, p.ldb);

  // stage cursor (summed batch index r, k tile kt) with r's operand offsets
  int64_t cur_r = KS > 0 ? st0 / KS : 0, cur_kt = KS > 0 ? st0 % KS : 0;
  int64_t ra_off = 0, rb_off = 0;
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
    const int64_t k0 = cur_kt * BK;
    const char* Ar = A + ra_off * ES;
    const char* Br = B + rb_off * ES;
    if (A_KC) ta.load(Ar + (m0 * p.lda + k0) * ES, p.M - m0, p.K - k0);
    else ta.load(Ar + (k0 * p.lda + m0) * ES, p.K - k0, p.M - m0);
    if (B_KC) tb.load(Br + (n0 * p.ldb + k0) * ES, p.N - n0, p.K - k0);
    else tb.load(Br + (k0 * p.ldb + n0) * ES, p.K - k0, p.N - n0);
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
    if (p.nred > 0) red_offsets(cur_r);
    load_stage();
    advance();
    ta.store(lds);
    tb.store(lds + TA::BYTES);
    __syncthreads();
  }
  for (int64_t s = 0; s < S; ++s) {
    const int cur = (int)(s & 1);
    const bool more = s + 1 < S;
    if (more) {
      load_stage();
      advance();
    }
    const E* As = (const E*)(lds + cur * (TA::BYTES + TB::BYTES));
    const E* Bs = (const E*)(lds + cur * (TA::BYTES + TB::BYTES) + TA::BYTES);
    Mma<T, A_KC, B_KC, TM, TN, BK, TA::PITCH, TB::PITCH>::run(As, Bs, wm * WTM, wn * WTN, l32, h,
                                                             acc);
    if (more) {
      char* nxt = lds + (cur ^ 1) * (TA::BYTES + TB::BYTES);
      ta.store(nxt);
      tb.store(nxt + TA::BYTES);
    }
    __syncthreads();
  }

  // ---- epilogue: lane holds C[m][n0' + 8g + 4h + 0..3] in acc regs 4g..4g+3
  if constexpr (EPI) {
    act_epilogue<TM, TN, (VEC > 1)>(p, acc, m0 + wm * WTM + l32, n0 + wn * WTN + 4 * h);
    return;
  }
  const bool to_partial = p.splits > 1;
  float* C = to_partial ? p.partial + (int64_t)split * p.partial_stride + batch * p.M * p.N
                        : p.c + c_off;
  const int64_t ldc = to_partial ? p.N : p.ldc;
  constexpr bool VEC_C = VEC > 1;  // host guarantees N % 4 == 0 and aligned C / bias then
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
        if (VEC_C) {
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

}  // namespace gemm
}  // namespace mt
