// Matrix-core GEMM whose operand tiles travel from HBM straight into LDS
// (buffer_load_dwordx4 ... lds), gfx950 only. Same contract and epilogue as
// gemm_kernel.hpp (MiniTensor Sec. 3.1 Eq. (1), Sec. 3.2 Eq. (4), Sec. 3.3
// Eq. (5)); used for 16-byte-aligned operands of large products.
//
// Why: the loads write LDS themselves, so no staging registers and no
// ds_write instructions sit between HBM and the fragments. Tiles are
// 256x256 with BK = 32 (fp32) or 64 (bf16), i.e. 64 KB per stage, and the
// ring holds NS = 2 stages (128 KB of the 160 KB LDS): one stage is ~3 us of
// fp32 or ~1 us of bf16 matrix work at 256x256, long enough for its
// successor's loads to land, and the per-stage costs (barrier, first
// fragment reads, load issue) are paid half as often as with BK = 16 / 32
// in a deeper ring. The kernel accepts rings of 2 to 5 stages.
//
// LDS layout: each operand tile is stored without padding, in rows of
// 16-byte chunks. The chunk index is XOR-swizzled with a function of the row
// so that fragment reads hit distinct banks:
//   K-contiguous tile, 64-byte rows:  chunk ^ (((r >> 1) & 3) ^ ((r >> 3) & 1))
//   K-contiguous tile, 128-byte rows: chunk ^ ((r & 7) ^ ((r >> 3) & 1))
//     (16 consecutive rows read at one chunk land on 16 distinct 16-byte bank
//     slots of a 256-byte window, and 8 consecutive rows on 8 slots of 128 B)
//   M/N-contiguous bf16 tile (rows of >= 256 bytes): chunk ^ (4 * (r & 3))
//     (the 4 rows x 4 chunks that two 16-lane groups of ds_read_b64_tr_b16
//     read together land on 16 distinct slots)
//   M/N-contiguous fp32 tile: chunk ^ (8 * ((r >> 2) & 1)) (the two rows a
//     4-byte read takes at once, k and k+4, fall in opposite 128-byte halves)
// A DMA instruction writes 64 lanes x 16 bytes to 1 KB of consecutive LDS
// (lane i at base + 16 i); each lane therefore loads the global chunk that
// the swizzle places at its LDS slot.
//
// Pipeline per stage s: wait until this wave's loads of stage s have landed
// (s_waitcnt vmcnt with the NS-2 younger stages still in flight), barrier
// (every wave's loads of stage s landed; every wave finished reading stage
// s-1), then the k-steps of stage s, each k-step's fragments read from LDS
// while the previous k-step's MFMAs run. The loads of stage s+NS-1 (into
// the slot of stage s-1) go out one at a time between chunks of MFMAs. In
// the last NS-1 stages those loads are empty (all out of range, zeros into
// a dead slot), so the stage loop has no branches. The barrier is a bare
// s_barrier: a release fence would make every wave wait for all loads in
// flight, younger stages included.
#pragma once
#include <hip/hip_runtime.h>

#include "gemm_kernel.hpp"
#include "gemm_params.hpp"

namespace mt {
namespace gemm {

// One 16-byte-per-lane load from a buffer straight into LDS: lane i's bytes
// land at lds_byte + 16 i. Issued as assembly so that the compiler's wait
// insertion, which cannot tell the LDS bytes these loads write from the ones
// the MFMA fragments read, does not wait for every load in flight before
// each LDS read; the kernel waits for exactly the stage it reads instead.
// An LDS-DMA load that reads M0 right after a scalar write of M0 needs one
// wait state in between (the s_nop).
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t lds_byte) {
  __asm__ __volatile__("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                       :
                       : "s"(lds_byte), "v"(voff), "s"(r)
                       : "memory", "m0");
}

// The 4-byte form, for operands whose rows are not 16-byte aligned (odd
// pitches): lane i's 4 bytes land at lds_byte + 4 i.
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t lds_byte) {
  __asm__ __volatile__("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                       :
                       : "s"(lds_byte), "v"(voff), "s"(r)
                       : "memory", "m0");
}

// The same address in every lane, taken from lane 0: the compiler may keep a
// wave-uniform 64-bit offset in vector registers (after a 64-bit division),
// and the LDS-DMA load takes its buffer descriptor in scalar registers only.
__device__ __forceinline__ const char* uniform_ptr(const char* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const char*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ int64_t uniform_i64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ uint32_t lds_byte_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// s_waitcnt with only vmcnt limited (expcnt and lgkmcnt at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <int ES, bool KC, int BMN, int BK>
struct DmaTile {
  static constexpr int RB = KC ? BK * ES : BMN * ES;  // bytes per LDS row
  static constexpr int ROWS = KC ? BMN : BK;
  static constexpr int BYTES = ROWS * RB;
  static constexpr int BLOCKS = BYTES / 1024;          // 1 KB DMA blocks per stage
  static constexpr int EPC = 16 / ES;                   // elements per 16-byte chunk
  static_assert(BYTES % 1024 == 0, "tile must be whole 1 KB blocks");
  static_assert(!KC || RB == 64 || RB == 128, "K-contiguous rows of 64 or 128 bytes");
  static_assert(KC || RB >= 256, "M/N-contiguous rows of at least 256 bytes");

  static __device__ __forceinline__ int swz(int r) {
    if constexpr (KC) {
      if constexpr (RB == 64) return ((r >> 1) & 3) ^ ((r >> 3) & 1);
      else return (r & 7) ^ ((r >> 3) & 1);
    } else if constexpr (ES == 2) {
      return 4 * (r & 3);
    } else {
      // fp32 4-byte reads: lanes 0-31 read row k, lanes 32-63 row k+4, the
      // same 32 columns; rows k and k+4 go to opposite 128-byte halves
      return 8 * ((r >> 2) & 1);
    }
  }
  // byte address in the tile of element (row r, contiguous index c)
  static __device__ __forceinline__ int addr(int r, int c) {
    return r * RB + (((c / EPC) ^ swz(r)) * 16) + (c % EPC) * ES;
  }
};

// Per-lane DMA plan of one operand: the wave issues JB instructions per
// stage, each moving 64 lanes x LANE bytes (16: one chunk a lane; 4: one
// element a lane, for operands without 16-byte aligned rows).
template <int ES, bool KC, int BMN, int BK, int NW, int LANE = 16>
struct DmaLoader {
  using T = DmaTile<ES, KC, BMN, BK>;
  static_assert(LANE == 16 || LANE == 4, "16- or 4-byte lanes");
  static constexpr int IB = 64 * LANE;  // bytes per instruction
  static constexpr int JB = T::BYTES / IB / NW;
  static_assert(T::BYTES % (IB * NW) == 0, "instructions split evenly over the waves");
  // byte offset of the lane's chunk from the stage's tile origin in global
  // memory, or kOOB (reads zero) where its m / n lies past the matrix edge
  uint32_t off[JB];
  // the chunk's k within the stage (its column if K-contiguous, else its row);
  // with 4-byte lanes (4x the instructions) packed four to a register (k < 256)
  static constexpr int KXN = LANE == 16 ? JB : (JB + 3) / 4;
  uint32_t kx[KXN];
  __device__ __forceinline__ int kx_of(int j) const {
    if constexpr (LANE == 16) return (int)kx[j];
    else return (int)((kx[j >> 2] >> (8 * (j & 3))) & 0xffu);
  }

  // mn_left: rows of A (columns of B) from the block's tile origin on
  __device__ __forceinline__ void init(int wave, int lane, int64_t ld, int64_t mn_left) {
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const int b = wave + NW * j;
      const int byte = IB * b + LANE * lane;
      const int r = byte / T::RB;
      const int pchunk = (byte % T::RB) / 16;
      const int c = (pchunk ^ T::swz(r)) * T::EPC + (byte % 16) / ES;
      const int mn = KC ? r : c;
      const uint32_t k_in_stage = (uint32_t)(KC ? c : r);
      if constexpr (LANE == 16) {
        kx[j] = k_in_stage;
      } else {
        static_assert(BK <= 256, "packed k fits 8 bits");
        if ((j & 3) == 0) kx[j >> 2] = 0;
        kx[j >> 2] |= k_in_stage << (8 * (j & 3));
      }
      off[j] = mn < mn_left ? (uint32_t)(((int64_t)r * ld + c) * ES) : kOOB;
    }
  }
  // What one stage's loads of this operand need, computed once per stage:
  // the buffer descriptor, the k left in range (BK for a whole stage), the
  // LDS origin.
  struct Plan {
    __amdgpu_buffer_rsrc_t r;
    int kl;
    uint32_t lds0;
  };
  // base: the stage's tile origin in global memory; lds: the tile's LDS
  // origin. A stage that is not live (past the last) gets a descriptor of
  // zero records: all its loads read zero without touching memory.
  __device__ __forceinline__ Plan plan(const char* base, int64_t k_left, char* lds,
                                       bool live) const {
    Plan q;
    q.r = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), (short)0,
                                            live ? 0x7fffffff : 0, kRsrcWord3);
    q.kl = !live ? 0 : k_left < BK ? (int)k_left : BK;
    q.lds0 = lds_byte_addr(lds);
    return q;
  }
  // The j-th of this wave's JB loads of the stage. KTAIL (K not a multiple
  // of BK): chunks past the K tail read as zero; otherwise every stage is
  // whole and the per-lane test is left out (vector instructions between
  // the MFMAs cost matrix throughput).
  template <bool KTAIL>
  __device__ __forceinline__ void issue_one(const Plan& q, int j, int wave) const {
    const uint32_t o = KTAIL ? (kx_of(j) < q.kl ? off[j] : kOOB) : off[j];
    if constexpr (LANE == 16) dma16(q.r, o, q.lds0 + IB * (wave + NW * j));
    else dma4(q.r, o, q.lds0 + IB * (wave + NW * j));
  }
};

// Fragment loads and MFMAs of one k-step, split so that the next k-step's
// fragments load while the current k-step multiplies, and the MFMAs in
// chunks between which the kernel places its loads.
template <typename T, bool A_KC, bool B_KC, int TM, int TN, int BK, int BM, int BN>
struct DmaMma;

// fp32: a k-step is a group of 8 k; within it, MFMA step j (0..3) takes
// k = 8g + 4h + j for lane half h (one 16-byte read of a K-contiguous tile
// feeds 4 steps).
template <bool A_KC, bool B_KC, int TM, int TN, int BK, int BM, int BN>
struct DmaMma<float, A_KC, B_KC, TM, TN, BK, BM, BN> {
  static constexpr int KSTEPS = BK / 8;
  struct Frags {
    float a[4][TM], b[4][TN];
  };
  template <bool KC, int BMN, int N>
  static __device__ __forceinline__ void frag(const char* S, int mn0, int g, int lane,
                                              float (&f)[4][N], int i) {
    using Tl = DmaTile<4, KC, BMN, BK>;
    const int h = lane >> 5, mn = mn0 + (lane & 31);
    if constexpr (KC) {
      const f32x4 v = *(const f32x4*)(S + Tl::addr(mn, 8 * g + 4 * h));
      f[0][i] = v[0];
      f[1][i] = v[1];
      f[2][i] = v[2];
      f[3][i] = v[3];
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) f[j][i] = *(const float*)(S + Tl::addr(8 * g + 4 * h + j, mn));
    }
  }
  static __device__ __forceinline__ void load(const char* As, const char* Bs, int am, int bn,
                                              int lane, int g, Frags& f) {
#pragma unroll
    for (int i = 0; i < TM; ++i) frag<A_KC, BM, TM>(As, am + i * 32, g, lane, f.a, i);
#pragma unroll
    for (int i = 0; i < TN; ++i) frag<B_KC, BN, TN>(Bs, bn + i * 32, g, lane, f.b, i);
  }
  // a k-step's MFMAs in 4 chunks: chunk j is MFMA step j of every tile
  static constexpr int CHUNKS = 4;
  static __device__ __forceinline__ void compute_chunk(const Frags& f, f32x16 (&acc)[TM][TN],
                                                       int j) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int q = 0; q < TN; ++q)
        acc[i][q] = __builtin_amdgcn_mfma_f32_32x32x2f32(f.b[j][q], f.a[j][i], acc[i][q], 0, 0, 0);
  }
};

// bf16: a k-step covers 16 k; lane half h supplies k = 16s + 8h + 0..7.
template <bool A_KC, bool B_KC, int TM, int TN, int BK, int BM, int BN>
struct DmaMma<__bf16, A_KC, B_KC, TM, TN, BK, BM, BN> {
  static constexpr int KSTEPS = BK / 16;
  struct Frags {
    u16x8 a[TM], b[TN];
  };
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  template <bool KC, int BMN>
  static __device__ __forceinline__ u16x8 frag(const char* S, int mn0, int k0, int lane) {
    using Tl = DmaTile<2, KC, BMN, BK>;
    if constexpr (KC) {
      const int mn = mn0 + (lane & 31);
      return *(const u16x8*)(S + Tl::addr(mn, k0));
    } else {
      // ds_read_b64_tr_b16: lane s of each 16-lane group addresses row
      // k0 + s/4, columns c0 + 4 (s % 4); lane i then receives column c0 + i
      // at rows k0 .. k0+3 (second read: rows k0+4 .. k0+7)
      const int g = lane >> 4, s = lane & 15;
      const int col = mn0 + 16 * (g & 1) + 4 * (s & 3);
      const int r = k0 + (s >> 2);
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_s16x4*)(const void*)(S + Tl::addr(r, col)));
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_s16x4*)(const void*)(S + Tl::addr(r + 4, col)));
      u16x8 v;
      v[0] = lo[0]; v[1] = lo[1]; v[2] = lo[2]; v[3] = lo[3];
      v[4] = hi[0]; v[5] = hi[1]; v[6] = hi[2]; v[7] = hi[3];
      return v;
    }
  }
  static __device__ __forceinline__ void load(const char* As, const char* Bs, int am, int bn,
                                              int lane, int ks, Frags& f) {
    const int k0 = 16 * ks + 8 * (lane >> 5);
#pragma unroll
    for (int i = 0; i < TM; ++i) f.a[i] = frag<A_KC, BM>(As, am + i * 32, k0, lane);
#pragma unroll
    for (int i = 0; i < TN; ++i) f.b[i] = frag<B_KC, BN>(Bs, bn + i * 32, k0, lane);
  }
  // a k-step's MFMAs in TM chunks: chunk i is row i of the wave's tiles
  static constexpr int CHUNKS = TM;
  static __device__ __forceinline__ void compute_chunk(const Frags& f, f32x16 (&acc)[TM][TN],
                                                       int i) {
#pragma unroll
    for (int q = 0; q < TN; ++q)
      acc[i][q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, f.b[q]),
                                                           __builtin_bit_cast(bf16x8, f.a[i]),
                                                           acc[i][q], 0, 0, 0);
  }
};

template <typename T, bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int NS,
          int DMA_G0, int DMA_GS, bool KTAIL,
          int WAVES_PER_EU, bool EPI = false, int DMA_LANE = 16, bool VEC_C = true>
__global__ __launch_bounds__(WGM * WGN * 64)
__attribute__((amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_dma_kernel(const GemmParams p) {
  constexpr int ES = (int)sizeof(T);
  constexpr int NW = WGM * WGN;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  static_assert(NS >= 2 && NS <= 5, "a ring of two to five stages");
  using LA = DmaLoader<ES, A_KC, BM, BK, NW, DMA_LANE>;
  using LB = DmaLoader<ES, B_KC, BN, BK, NW, DMA_LANE>;
  constexpr int A_BYTES = LA::T::BYTES, B_BYTES = LB::T::BYTES;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int L = LA::JB + LB::JB;  // DMA instructions per wave per stage
  __shared__ __attribute__((aligned(1024))) char lds[NS * STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (LDS DMA base)
  const int wm = wave / WGN, wn = wave % WGN;
  const int l32 = lane & 31, h = lane >> 5;

  // ---- block -> (split, batch, tile), as in gemm_kernel
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

  const int64_t KS = (p.K + BK - 1) / BK;
  const int64_t S_all = KS * p.red_count;
  const int64_t st0 = (int64_t)split * p.stages_per_split;
  const int64_t st1 = (st0 + p.stages_per_split) < S_all ? (st0 + p.stages_per_split) : S_all;
  const int S = st1 > st0 ? (int)(st1 - st0) : 0;

  LA la;
  LB lb;
  la.init(wave, lane, p.lda, p.M - m0);
  lb.init(wave, lane, p.ldb, p.N - n0);

  // issue cursor: (summed batch index r, k tile kt) of the next stage to
  // load, wave-uniform (scalar registers)
  int64_t cur_r = uniform_i64(KS > 0 ? st0 / KS : 0);
  int64_t cur_kt = uniform_i64(KS > 0 ? st0 % KS : 0);
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
  if (S > 0 && p.nred > 0) red_offsets(cur_r);
  // tile origins of the next stage to load, advanced by one K-stage per
  // load; recomputed only where the summed batch index moves on
  const int64_t a_step = (A_KC ? (int64_t)BK : (int64_t)BK * p.lda) * ES;
  const int64_t b_step = (B_KC ? (int64_t)BK : (int64_t)BK * p.ldb) * ES;
  const char* a_nxt = A;
  const char* b_nxt = B;
  int64_t k_left = 0;
  auto seek = [&]() {
    const int64_t k0 = cur_kt * BK;
    a_nxt = uniform_ptr(A + (ra_off + (A_KC ? m0 * p.lda + k0 : k0 * p.lda + m0)) * ES);
    b_nxt = uniform_ptr(B + (rb_off + (B_KC ? n0 * p.ldb + k0 : k0 * p.ldb + n0)) * ES);
    k_left = uniform_i64(p.K - k0);
  };
  // K-stage rotation (p.krot): the sequence starts at stage rot and wraps to
  // stage 0 once, where the tile origins are sought again
  bool wrap_pending = false;
  if (p.krot && p.splits == 1 && p.red_count == 1 && KS > 1) {
    const int64_t rot = ((int64_t)(blockIdx.x & 7) * KS) >> 3;
    if (rot > 0) {
      cur_kt = uniform_i64(rot);
      wrap_pending = true;
    }
  }
  if (S > 0) seek();
  // plans of the next stage's loads (into LDS slot `slot`); advances the cursor
  typename LA::Plan pa;
  typename LB::Plan pb;
  // Stages past the last (planned while the final NS-1 stages compute) load
  // nothing: every chunk is out of range and reads zero into a slot no wave
  // reads again, so the loop issues the same loads in every stage, unbranched.
  int planned = 0;
  auto plan_next = [&](int slot) {
    char* dst = lds + slot * STAGE;
    const bool live = planned < S;
    ++planned;
    pa = la.plan(a_nxt, k_left, dst, live);
    pb = lb.plan(b_nxt, k_left, dst + A_BYTES, live);
    if (++cur_kt == KS) {
      cur_kt = 0;
      if (wrap_pending) {
        wrap_pending = false;
        seek();
      } else {
        ++cur_r;
        if (cur_r < p.red_count) {
          red_offsets(cur_r);
          seek();
        }
      }
    } else {
      a_nxt += a_step;
      b_nxt += b_step;
      k_left -= BK;
    }
  };
  // the j-th (of L) load of the planned stage: A's first, then B's
  auto issue_one = [&](int j) {
    if (j < LA::JB) la.template issue_one<KTAIL>(pa, j, wave);
    else lb.template issue_one<KTAIL>(pb, j - LA::JB, wave);
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};

  using Mma = DmaMma<T, A_KC, B_KC, TM, TN, BK, BM, BN>;
  typename Mma::Frags cur, nxt;
  const int am = wm * WTM, bn = wn * WTN;

  // prologue: stages 0 .. NS-2 in flight
#pragma unroll
  for (int q = 0; q < NS - 1; ++q) {
    plan_next(q);
#pragma unroll
    for (int j = 0; j < L; ++j) issue_one(j);
  }

  constexpr int CHUNKS = Mma::CHUNKS;
  static_assert(DMA_G0 >= 0 && DMA_GS >= 1 && DMA_G0 < Mma::KSTEPS * CHUNKS, "issue points");
  // issue points: chunks DMA_G0, DMA_G0 + DMA_GS, ... of the stage; PER loads at each
  constexpr int POINTS = (Mma::KSTEPS * CHUNKS - DMA_G0 + DMA_GS - 1) / DMA_GS;
  constexpr int PER = (L + POINTS - 1) / POINTS;
  // one stage; the loads of stage s+NS-1 go out during it
  auto run_stage = [&](int s) {
    // stages 0 .. s+NS-2 have been issued: this wave's loads of stage s have
    // landed once at most NS-2 later stages (of L loads each) are in flight;
    // the barrier then makes every wave's loads visible and frees the slot
    // stage s-1 used
    wait_vmcnt<(NS - 2) * L>();
    __builtin_amdgcn_s_barrier();
    __asm__ __volatile__("" ::: "memory");
    const char* st = lds + (s % NS) * STAGE;
    Mma::load(st, st + A_BYTES, am, bn, lane, 0, cur);
#pragma unroll
    for (int ks = 0; ks < Mma::KSTEPS; ++ks) {
      if (ks + 1 < Mma::KSTEPS) Mma::load(st, st + A_BYTES, am, bn, lane, ks + 1, nxt);
#pragma unroll
      for (int c = 0; c < CHUNKS; ++c) {
        Mma::compute_chunk(cur, acc, c);
        // the next stage's L loads go out PER at a time after every
        // DMA_GS-th chunk of MFMAs from chunk DMA_G0 on, so that no wave
        // stalls on a burst of loads the memory pipeline cannot take at once
        const int g = ks * CHUNKS + c;
        if (g >= DMA_G0 && (g - DMA_G0) % DMA_GS == 0 && (g - DMA_G0) / DMA_GS * PER < L) {
          if (g == DMA_G0) plan_next((s + NS - 1) % NS);
          const int j0 = (g - DMA_G0) / DMA_GS * PER;
#pragma unroll
          for (int j = j0; j < j0 + PER && j < L; ++j) issue_one(j);
        }
        // keep each chunk's MFMAs and loads where they are: left to itself
        // the scheduler gathers the loads into bursts again
        __builtin_amdgcn_sched_barrier(0);
      }
      cur = nxt;
    }
    __asm__ __volatile__("" ::: "memory");
  };
  for (int s = 0; s < S; ++s) run_stage(s);
  // the empty loads of the stages past the last land before the wave ends
  wait_vmcnt<0>();

  // ---- epilogue (as in gemm_kernel): lane holds C[m][n0' + 8g + 4h + 0..3]
  if constexpr (EPI) {
    act_epilogue<TM, TN, true>(p, acc, m0 + wm * WTM + l32, n0 + wn * WTN + 4 * h);
    return;
  }
  const bool to_partial = p.splits > 1;
  float* C = to_partial ? p.partial + (int64_t)split * p.partial_stride + batch * p.M * p.N
                        : p.c + c_off;
  const int64_t ldc = to_partial ? p.N : p.ldc;
  if constexpr (!VEC_C) {
    // Rows of C not 16-byte aligned (odd pitch or N): each wave stages 32
    // rows of its tile at a time in its own slice of the (now idle) ring,
    // then writes them back a row at a time, 64 lanes on 64 consecutive
    // columns: one contiguous 256-byte store per row segment instead of
    // scattered 4-byte stores. Row pitch WTN + 4 floats offsets consecutive
    // rows by 16 bytes in the LDS banks.
    constexpr int SP = WTN + 4;
    static_assert(NW * 32 * SP * 4 <= NS * STAGE, "staging fits in the ring");
    __syncthreads();  // every wave has finished reading the ring
    float* stg = (float*)(lds + wave * 32 * SP * 4);
    const int64_t mb = m0 + wm * WTM, nb = n0 + wn * WTN;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int q = 0; q < TN; ++q)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          *(f32x4*)&stg[l32 * SP + q * 32 + 8 * g + 4 * h] =
              f32x4{acc[i][q][4 * g + 0], acc[i][q][4 * g + 1], acc[i][q][4 * g + 2],
                    acc[i][q][4 * g + 3]};
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes done
      __builtin_amdgcn_wave_barrier();
#pragma unroll 4
      for (int r = 0; r < 32; ++r) {
        const int64_t m = mb + i * 32 + r;
        if (m >= p.M) break;
        float* crow = C + m * ldc;
#pragma unroll
        for (int cb = 0; cb < WTN; cb += 64) {
          const int64_t n = nb + cb + lane;
          if (n >= p.N) continue;
          float x = stg[r * SP + cb + lane];
          if (!to_partial) {
            if (p.bias) x += p.bias[n];
            if (p.accumulate) x += crow[n];
          }
          crow[n] = x;
        }
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the next slab overwrites
      __builtin_amdgcn_wave_barrier();
    }
    return;
  }
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
        if constexpr (!VEC_C) {
          // rows of C not 16-byte aligned (odd pitch or N): element stores
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (n + e >= p.N) continue;
            float x = acc[i][q][4 * g + e];
            if (!to_partial) {
              if (p.bias) x += p.bias[n + e];
              if (p.accumulate) x += crow[n + e];
            }
            crow[n + e] = x;
          }
          continue;
        }
        if (n >= p.N) continue;
        f32x4 v = {acc[i][q][4 * g + 0], acc[i][q][4 * g + 1], acc[i][q][4 * g + 2],
                   acc[i][q][4 * g + 3]};
        if (!to_partial) {
          if (p.bias) v += *(const f32x4*)&p.bias[n];
          if (p.accumulate) v += *(const f32x4*)&crow[n];
        }
        *(f32x4*)&crow[n] = v;
      }
    }
  }
}

}  // namespace gemm
}  // namespace mt
