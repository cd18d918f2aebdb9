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

#include <type_traits>

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
  static_assert(!KC || RB == 64 || RB == 128 || RB == 256, "K-contiguous rows of 64 to 256 bytes");
  static_assert(KC || RB % 256 == 0, "M/N-contiguous rows of whole 256-byte groups (the swizzle "
                                     "moves chunks within them)");

  static __device__ __forceinline__ int swz(int r) {
    if constexpr (KC) {
      if constexpr (RB == 64) return ((r >> 1) & 3) ^ ((r >> 3) & 1);
      else if constexpr (RB == 128) return (r & 7) ^ ((r >> 3) & 1);
      // 256-byte rows: 16 consecutive rows put one chunk in 16 distinct
      // 16-byte slots of the 256-byte window
      else return r & 15;
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

// q = n / d for n < 2^31 from the host's (mag, shift) of d.
__device__ __forceinline__ uint32_t fast_div(uint32_t n, uint32_t mag, int shift) {
  return (uint32_t)(((uint64_t)n * mag) >> shift);
}

// Convolution, forward product: A is the unfolded input U (rows m = output
// pixels, K-contiguous), gathered from the image. A stage covers BK channels
// of one tap (u, v) (C is a multiple of BK), so a lane's 16-byte chunk is 4
// consecutive channels of one input pixel: contiguous in channels-last x.
// Per lane and load the pixel's window origin is decoded once per block; per
// stage the tap moves, and a chunk whose input pixel falls in the padding (or
// whose row lies past the last pixel) reads zero.
template <int BM, int BK, int NW>
struct ConvGatherA {
  using T = DmaTile<4, true, BM, BK>;
  static constexpr int IB = 1024;
  static constexpr int JB = T::BYTES / IB / NW;
  static_assert(T::BYTES % (IB * NW) == 0, "instructions split evenly over the waves");
  static constexpr int32_t kFar = -(1 << 30);  // window origin of rows past the last pixel
  int32_t base[JB];  // element offset of the chunk at tap (0, 0), channel group 0
  int32_t hb[JB], wb[JB];  // input row / column of the window's tap (0, 0)

  __device__ __forceinline__ void init(int wave, int lane, const ConvGather& g, int64_t m0,
                                       int64_t M) {
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const int byte = IB * (wave + NW * j) + 16 * lane;
      const int r = byte / T::RB;
      const int c = (((byte % T::RB) / 16) ^ T::swz(r)) * 4;
      const int64_t m = m0 + r;
      if (m < M) {
        const uint32_t t = fast_div((uint32_t)m, g.wo_mag, g.wo_shift);
        const int32_t jj = (int32_t)((uint32_t)m - t * (uint32_t)g.WO);
        const uint32_t n = fast_div(t, g.ho_mag, g.ho_shift);
        const int32_t i = (int32_t)(t - n * (uint32_t)g.HO);
        hb[j] = i * g.sh - g.ph;
        wb[j] = jj * g.sw - g.pw;
        base[j] = (int32_t)n * g.xs0 + hb[j] * g.xs2 + wb[j] * g.xs3 + c;
      } else {
        hb[j] = kFar;
        wb[j] = 0;
        base[j] = 0;
      }
    }
  }
  struct Plan {
    __amdgpu_buffer_rsrc_t r;
    int32_t toff;  // element offset of tap (u, v), channel c0
    int32_t u, v;
    uint32_t lds0;
  };
  __device__ __forceinline__ Plan plan(const ConvGather& g, bool live, int u, int v, int c0,
                                       char* lds) const {
    Plan q;
    q.r = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(g.x), (short)0,
                                            live ? (int)g.x_bytes : 0, kRsrcWord3);
    q.toff = u * g.xs2 + v * g.xs3 + c0;
    q.u = u;
    q.v = v;
    q.lds0 = lds_byte_addr(lds);
    return q;
  }
  __device__ __forceinline__ void issue_one(const Plan& q, int j, int wave,
                                            const ConvGather& g) const {
    const int32_t h = hb[j] + q.u, w = wb[j] + q.v;
    const bool ok = (uint32_t)h < (uint32_t)g.H && (uint32_t)w < (uint32_t)g.W;
    const uint32_t o = ok ? (uint32_t)(base[j] + q.toff) * 4u : kOOB;
    dma16(q.r, o, q.lds0 + IB * (wave + NW * j));
  }
};

// Convolution, weight gradient: B is U again, now with the pixels m as the
// contraction (tile rows, BK per stage) and the unfolded columns k as tile
// columns. A lane's chunk keeps its column, so its tap (u, v) and channel are
// decoded once per block (C % 4 == 0 keeps a chunk inside one tap); per
// stage its row's pixel is decoded (two divisions by multiplication, on the
// scalar unit where a load covers one row).
template <int BN, int BK, int NW>
struct ConvGatherB {
  using T = DmaTile<4, false, BN, BK>;
  static constexpr int IB = 1024;
  static constexpr int JB = T::BYTES / IB / NW;
  static_assert(T::BYTES % (IB * NW) == 0, "instructions split evenly over the waves");
  // tap row of columns past the last: beyond any input row (H + ph < 2^14)
  static constexpr int32_t kFarTap = 0x7fff;
  uint32_t ch[JB];  // channel of the chunk's first column
  uint32_t uv[JB];  // tap u | v << 16
  uint32_t rr[JB];  // row (pixel) within the stage

  __device__ __forceinline__ void init(int wave, int lane, const ConvGather& g, int64_t n0,
                                       int64_t N) {
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const int byte = IB * (wave + NW * j) + 16 * lane;
      const int r = byte / T::RB;
      const int c = (((byte % T::RB) / 16) ^ T::swz(r)) * 4;
      const int64_t col = n0 + c;
      // rows of 1 KB or more: one row per instruction, the same in every
      // lane, so the pixel decode below runs on the scalar unit
      rr[j] = T::RB >= IB ? (uint32_t)__builtin_amdgcn_readfirstlane(IB * (wave + NW * j) / T::RB)
                          : (uint32_t)r;
      if (col < N) {
        const uint32_t tap = (uint32_t)col / (uint32_t)g.C;
        const uint32_t u = tap / (uint32_t)g.KW;
        ch[j] = (uint32_t)col - tap * (uint32_t)g.C;
        uv[j] = u | ((tap - u * (uint32_t)g.KW) << 16);
      } else {
        ch[j] = 0;
        uv[j] = (uint32_t)kFarTap;
      }
    }
  }
  struct Plan {
    __amdgpu_buffer_rsrc_t r;
    uint32_t m0;    // first pixel of the stage
    uint32_t mlim;  // number of pixels (the contraction length)
    uint32_t lds0;
  };
  __device__ __forceinline__ Plan plan(const ConvGather& g, bool live, uint32_t m0, uint32_t mlim,
                                       char* lds) const {
    Plan q;
    q.r = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(g.x), (short)0,
                                            live ? (int)g.x_bytes : 0, kRsrcWord3);
    q.m0 = m0;
    q.mlim = mlim;
    q.lds0 = lds_byte_addr(lds);
    return q;
  }
  __device__ __forceinline__ void issue_one(const Plan& q, int j, int wave,
                                            const ConvGather& g) const {
    const uint32_t m = q.m0 + rr[j];
    const uint32_t t = fast_div(m, g.wo_mag, g.wo_shift);
    const uint32_t jj = m - t * (uint32_t)g.WO;
    const uint32_t n = fast_div(t, g.ho_mag, g.ho_shift);
    const uint32_t i = t - n * (uint32_t)g.HO;
    const uint32_t h = i * (uint32_t)g.sh - (uint32_t)g.ph + (uv[j] & 0xffffu);
    const uint32_t w = jj * (uint32_t)g.sw - (uint32_t)g.pw + (uv[j] >> 16);
    const bool ok = m < q.mlim && h < (uint32_t)g.H && w < (uint32_t)g.W;
    const uint32_t o =
        ok ? (n * (uint32_t)g.xs0 + h * (uint32_t)g.xs2 + w * (uint32_t)g.xs3 + ch[j]) * 4u : kOOB;
    dma16(q.r, o, q.lds0 + IB * (wave + NW * j));
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
  // An M-contiguous A (TN products) is read TM consecutive rows at a time:
  // tile i's row r is the wave's row TM r + i (ROW_PERM), so one TM-wide read
  // of LDS row k feeds all TM tiles instead of TM 4-byte reads; the epilogue
  // writes tile i's row r to that row.
  static constexpr bool ROW_PERM = !A_KC && (TM == 2 || TM == 4);
  typedef float f32xTM __attribute__((ext_vector_type(TM == 4 ? 4 : 2)));
  static __device__ __forceinline__ void load(const char* As, const char* Bs, int am, int bn,
                                              int lane, int g, Frags& f) {
    if constexpr (ROW_PERM) {
      using Tl = DmaTile<4, false, BM, BK>;
      const int h = lane >> 5, c = am + TM * (lane & 31);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32xTM v = *(const f32xTM*)(As + Tl::addr(8 * g + 4 * h + j, c));
#pragma unroll
        for (int i = 0; i < TM; ++i) f.a[j][i] = v[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i) frag<A_KC, BM, TM>(As, am + i * 32, g, lane, f.a, i);
    }
#pragma unroll
    for (int i = 0; i < TN; ++i) frag<B_KC, BN, TN>(Bs, bn + i * 32, g, lane, f.b, i);
  }
  // Column sums of an M-contiguous A over the k-step's 4 MFMA steps: tile
  // i's value goes to the lane's column (see a_col), lane half h holding k
  // = 8g + 4h + j.
  static __device__ __forceinline__ void colsum(const Frags& f, float (&cs)[TM]) {
#pragma unroll
    for (int i = 0; i < TM; ++i) cs[i] += (f.a[0][i] + f.a[1][i]) + (f.a[2][i] + f.a[3][i]);
  }
  // the column of A (from the wave's first) whose values tile i holds in this lane
  static __device__ __forceinline__ int a_col(int lane, int i) {
    return ROW_PERM ? TM * (lane & 31) + i : 32 * i + (lane & 31);
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
  static constexpr bool ROW_PERM = false;
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
  // Column sums of an M-contiguous A over the k-step: lane L of tile i
  // holds 8 consecutive k of column 32 i + (L & 31), summed in pairs by
  // v_dot2_f32_bf16 against (1, 1) (exact products, fp32 sums).
  static __device__ __forceinline__ void colsum(const Frags& f, float (&cs)[TM]) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 one = __builtin_bit_cast(bf16x2, (uint32_t)0x3f803f80u);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      float s = cs[i];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        // elements 2e and 2e+1, packed as they sit in one register
        const uint32_t pair = (uint32_t)f.a[i][2 * e] | ((uint32_t)f.a[i][2 * e + 1] << 16);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pair), one, s, false);
      }
      cs[i] = s;
    }
  }
  static __device__ __forceinline__ int a_col(int lane, int i) { return 32 * i + (lane & 31); }
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

// PERSIST: the grid holds one block per CU and block b computes the tiles
// the plain grid's blocks b, b + gridDim.x, ... would (plain products only).
template <typename T, bool A_KC, bool B_KC, int BM, int BN, int BK, int WGM, int WGN, int NS,
          int DMA_G0, int DMA_GS, bool KTAIL,
          int WAVES_PER_EU, bool EPI = false, int DMA_LANE = 16, bool VEC_C = true,
          bool PERSIST = false>
__global__ __launch_bounds__(WGM * WGN * 64)
__attribute__((amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_dma_kernel(const GemmParams p) {
  constexpr int CONV = 0;
  constexpr bool SK = false, sk_part = false;
  constexpr int64_t sk_t = 0, sk_ka = 0, sk_kb = 0;
  constexpr int sk_slot = 0;
#include "gemm_dma_body.inc"
}

// The convolution products with an operand gathered by the loads: CONV_ 1 the
// forward (y = U Wf^T + b, NT), 2 the weight gradient (dW = dY^T U, TN), 3
// the input gradient of a stride-1 convolution (dx = V W, NN, V gathered from
// dY: V[(n, h, w)][(u, v, co)] = dY[n][h + ph - u][w + pw - v][co]), 4 one
// sub-pixel phase of a strided convolution's input gradient.
template <int CONV_, int BM, int BN, int BK, int WGM, int WGN, int NS, bool KTAIL, int WAVES_PER_EU>
__global__ __launch_bounds__(WGM * WGN * 64)
__attribute__((amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void conv_dma_kernel(const GemmParams p) {
  using T = float;
  constexpr bool A_KC = CONV_ != 2, B_KC = CONV_ == 1, EPI = false, VEC_C = true;  // CONV_ 1..4
  constexpr int DMA_G0 = 1, DMA_GS = 1, DMA_LANE = 16, CONV = CONV_;
  constexpr bool SK = false, sk_part = false;
  constexpr int64_t sk_t = 0, sk_ka = 0, sk_kb = 0;
  constexpr int sk_slot = 0;
  constexpr bool PERSIST = false;
#include "gemm_dma_body.inc"
}

// Stream-K schedule of the U = T KS K-stages of T tiles (tile-major, KS
// stages each) over G blocks: block b takes stages [b U / G, (b+1) U / G).
// A tile cut by block boundaries is summed in segments; sk_count(X) counts
// the boundaries floor(b U / G) (b >= 0) below X, for X >= 1. With U >= G
// the boundaries are distinct, so segments and boundaries match one to one.
__host__ __device__ inline int64_t sk_count(int64_t X, int64_t G, int64_t U) {
  return (X * G + U - 1) / U;
}
struct SkSeg {
  int n;     // segments of the tile
  int slot;  // index of the segment that starts at stage ka of the tile
};
__host__ __device__ inline SkSeg sk_segment(int64_t t, int64_t ka, int64_t KS, int64_t G,
                                            int64_t U) {
  const int64_t L = t * KS;
  const int64_t c0 = sk_count(L + 1, G, U);
  return {(int)(sk_count(L + KS, G, U) - c0 + 1), (int)(sk_count(L + ka + 1, G, U) - c0)};
}

// The stream-K form of the gathered forward (CONV_ 1) and input-gradient
// (CONV_ 3) products, for grids that would leave a partial last wave of
// tiles: every block (one per CU) computes its share of stages tile by tile;
// a tile computed whole is written with its bias, the segments of a cut
// tile go to partial slot `segment index` (p.partial, M x N each) and
// sk_finish adds them in slot order. No block waits on another.
template <int CONV_, int BM, int BN, int BK, int WGM, int WGN, int NS, int WAVES_PER_EU>
__global__ __launch_bounds__(WGM * WGN * 64)
__attribute__((amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void conv_dma_sk_kernel(const GemmParams p) {
  static_assert(CONV_ == 1 || CONV_ == 3, "stream-K: the gathered NT / NN products");
  using T = float;
  constexpr bool A_KC = true, B_KC = CONV_ == 1, EPI = false, VEC_C = true, KTAIL = false;
  constexpr int DMA_G0 = 1, DMA_GS = 1, DMA_LANE = 16, CONV = CONV_;
  constexpr bool SK = true;
  const int64_t ks_all = (p.K + BK - 1) / BK;
  const int64_t U = (int64_t)p.tiles_m * p.tiles_n * ks_all, G = gridDim.x;
  const int64_t u_end = ((int64_t)blockIdx.x + 1) * U / G;
  for (int64_t u = (int64_t)blockIdx.x * U / G; u < u_end;) {
    const int64_t sk_t = u / ks_all;
    const int64_t sk_ka = u - sk_t * ks_all;
    const int64_t sk_kb = (u_end - sk_t * ks_all) < ks_all ? (u_end - sk_t * ks_all) : ks_all;
    const SkSeg seg = sk_segment(sk_t, sk_ka, ks_all, G, U);
    const bool sk_part = seg.n > 1;
    const int sk_slot = seg.slot;
  constexpr bool PERSIST = false;
#include "gemm_dma_body.inc"
    u = sk_t * ks_all + sk_kb;
    __syncthreads();  // the next segment's loads reuse the ring
  }
}

// All sub-pixel phases of a strided input gradient in one grid (phases in
// the order of the table, longest contraction first, so that the longest
// tiles start first): the block finds its phase, rewrites the phase's fields
// of the description and computes one whole tile of it.
template <int BM, int BN, int BK, int WGM, int WGN, int NS, int WAVES_PER_EU>
__global__ __launch_bounds__(WGM * WGN * 64)
__attribute__((amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void conv_dgrad_phases_kernel(const GemmParams p0, const ConvPhases tab) {
  using T = float;
  constexpr bool A_KC = true, B_KC = false, EPI = false, VEC_C = true, KTAIL = false;
  constexpr int DMA_G0 = 1, DMA_GS = 1, DMA_LANE = 16, CONV = 4;
  constexpr bool SK = true, sk_part = false;
  constexpr int sk_slot = 0;
  int k = 0;
  while (k + 1 < tab.n && (int32_t)blockIdx.x >= tab.tile0[k + 1]) ++k;
  const ConvPhase& f = tab.ph[k];
  GemmParams p = p0;
  p.M = f.M;
  p.K = f.K;
  p.tiles_m = f.tiles_m;
  p.cg.u0 = f.u0;
  p.cg.v0 = f.v0;
  p.cg.ph = f.ph;
  p.cg.pw = f.pw;
  p.cg.HO = f.rows;
  p.cg.WO = f.cols;
  p.cg.KW = f.kw;
  p.cg.h0 = f.h0;
  p.cg.w0 = f.w0;
  p.cg.wo_mag = f.wo_mag;
  p.cg.ho_mag = f.ho_mag;
  p.cg.wo_shift = f.wo_shift;
  p.cg.ho_shift = f.ho_shift;
  const int64_t sk_t = (int64_t)blockIdx.x - tab.tile0[k];
  const int64_t sk_ka = 0, sk_kb = (f.K + BK - 1) / BK;
  constexpr bool PERSIST = false;
#include "gemm_dma_body.inc"
}

}  // namespace gemm
}  // namespace mt
