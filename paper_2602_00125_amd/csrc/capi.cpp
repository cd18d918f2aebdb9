// C-ABI of libminitensor_hip: argument validation, shape planning and kernel
// dispatch (the convolution's planning lives in conv_host.cpp). Declarations
// and their contracts: include/minitensor_hip.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/minitensor_hip.h"
#include "act.hpp"
#include "gemm_params.hpp"
#include "host.hpp"
#include "kernels.hpp"
#include "shape.hpp"

namespace mt::host {

thread_local std::string g_err;

// Knobs for tests and tuning (mt_debug_set): -1 / 0 = automatic.
std::atomic<int> g_force_cfg{-1};
std::atomic<int> g_force_vec1{0};
std::atomic<int> g_force_splits{0};
std::atomic<int> g_force_parts{0};
std::atomic<int> g_krot{1};  // K-stage rotation per XCD in the DMA kernel (measured: bf16 NT +2%, others neutral)
std::atomic<int> g_conv_gather{1};  // convolution products gather the image where the layout allows
std::atomic<int> g_stream_k{1};     // gathered 256x256 convolution products: 0 never, 1 on a ragged last wave, 2 always
std::atomic<int> g_sk_blocks{0};    // stream-K blocks (0: one per CU, 256)
std::atomic<int> g_persist{1};      // plain products on the 256x256 DMA tiles: one block per CU walking its tiles
std::atomic<int> g_phase_grid{1};   // strided input gradient: 0 a launch per phase, 1 one grid when large, 2 always

mt_status fail(mt_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

size_t elem_size(int32_t dt) { return dt == MT_BF16 ? 2 : 4; }

mt_status check_tensor(const mt_tensor* t, const char* name, int min_nd, int max_nd) {
  if (!t) return fail(MT_ERR_NULL, std::string(name) + ": null tensor descriptor");
  if (t->ndim < min_nd || t->ndim > max_nd)
    return fail(MT_ERR_NDIM, std::string(name) + ": rank " + std::to_string(t->ndim) +
                                 " outside " + std::to_string(min_nd) + ".." +
                                 std::to_string(max_nd));
  if (t->dtype != MT_F32 && t->dtype != MT_BF16)
    return fail(MT_ERR_DTYPE, std::string(name) + ": unknown dtype " + std::to_string(t->dtype));
  int64_t n = 1;
  for (int i = 0; i < t->ndim; ++i) {
    if (t->shape[i] < 0) return fail(MT_ERR_SHAPE, std::string(name) + ": negative size");
    if (t->stride[i] < 0) return fail(MT_ERR_LAYOUT, std::string(name) + ": negative stride");
    n *= t->shape[i];
  }
  if (n > 0 && !t->data) return fail(MT_ERR_NULL, std::string(name) + ": null data pointer");
  return MT_OK;
}

int64_t numel(const mt_tensor* t) {
  int64_t n = 1;
  for (int i = 0; i < t->ndim; ++i) n *= t->shape[i];
  return n;
}

// [lo, hi) byte range touched by a view; empty views touch nothing.
void byte_range(const mt_tensor* t, uintptr_t* lo, uintptr_t* hi) {
  const int64_t span = mt::span_elems(t->ndim, t->shape, t->stride);
  *lo = (uintptr_t)t->data;
  *hi = *lo + (uintptr_t)span * elem_size(t->dtype);
}

bool overlaps(const mt_tensor* a, const mt_tensor* b) {
  if (!a || !b || numel(a) == 0 || numel(b) == 0) return false;
  uintptr_t alo, ahi, blo, bhi;
  byte_range(a, &alo, &ahi);
  byte_range(b, &blo, &bhi);
  return alo < bhi && blo < ahi;
}

bool is_row_major(const mt_tensor* t) {
  int64_t expect = 1;
  for (int i = t->ndim - 1; i >= 0; --i) {
    if (t->shape[i] != 1 && t->stride[i] != expect) return false;
    expect *= t->shape[i];
  }
  return true;
}

mt_status hip_status(hipError_t e) {
  if (e == hipSuccess) return MT_OK;
  return fail(MT_ERR_HIP, std::string("HIP: ") + hipGetErrorString(e));
}


// Tile configuration: 128x256 / 256x128 blocks run two per CU (one wave per
// SIMD each), which hides one block's barrier behind the other's matrix-core
// work (measured faster than 256x256 on 8192^3). Smaller problems take
// 128x128 when split-K can fill the chip, else 64x64.
// K-stages of the 256x256 DMA tile per split-K run below which a run is too
// short to amortise its prologue and epilogue
constexpr int64_t kDmaMinRunStages = 32;

int choose_cfg_aligned(int64_t M, int64_t N, int64_t batch, int64_t stages, bool can_split,
                       bool bf16, bool a_kc, bool b_kc, bool vec, int64_t K, int64_t red);

// Tile choice. fp32 products whose operands or output lack 16-byte aligned
// rows run on the DMA tiles with 4-byte lanes; below ~4 waves of 256x256
// tiles the tile that wastes least on the matrix edges wins (measured on the
// 16x1x509x257 @ 1x8x257x383 products: 256x128 for 509 x 383 and 509 x 257
// outputs, 128x128 for 257 x 383).
int choose_cfg(int64_t M, int64_t N, int64_t batch, int64_t stages, bool can_split, bool bf16,
               bool a_kc, bool b_kc, bool vec, int64_t K, int64_t red) {
  if (const int fc = g_force_cfg; fc >= 0) return fc;
  const int c = choose_cfg_aligned(M, N, batch, stages, can_split, bf16, a_kc, b_kc, vec, K, red);
  if (vec || bf16 || c == mt::kCfg64x64) return c;
  if (cdiv(M, 256) * cdiv(N, 256) * batch >= 1024) return mt::kCfgDma256x256;
  // Each candidate tile is scored by the share of its work that is useful:
  // the output it covers inside the matrix, the K it covers inside the
  // contraction, and how full its last round of blocks is (a product that
  // will be split along K fills its round with the split). The tiles shaped
  // for sizes just past a multiple of 128 (96- and 192-wide, 64-row) stand in
  // for 128-wide tiles that would cover a third too much (measured on the
  // 16x1x509x257 @ 1x8x257x383 products).
  struct Cand {
    int cfg, bm, bn, bk, per_cu;
  };
  const Cand cands[] = {{mt::kCfgDma256x128, 256, 128, 16, 2}, {mt::kCfgDma128x256, 128, 256, 16, 2},
                        {mt::kCfgDma128x128, 128, 128, 32, 2}, {mt::kCfgDma256x192, 256, 192, 16, 1},
                        {mt::kCfgDma256x96, 256, 96, 16, 2},   {mt::kCfgDma64x384, 64, 384, 16, 2}};
  int best = mt::kCfgDma128x128;
  double best_score = -1.0;
  for (const Cand& t : cands) {
    if (t.cfg == mt::kCfgDma256x96 && !b_kc) continue;  // its B tile must be K-contiguous
    const int64_t blocks = cdiv(M, t.bm) * cdiv(N, t.bn) * batch;
    const int64_t slots = 256 * t.per_cu;
    const double used = (double)(M * N) / (double)(cdiv(M, t.bm) * t.bm * cdiv(N, t.bn) * t.bn);
    const double kuse = K > 0 ? (double)K / (double)(cdiv(K, t.bk) * t.bk) : 1.0;
    const bool split_fills = can_split && blocks < slots && stages >= 16;
    const double fill = split_fills ? 1.0 : (double)blocks / (double)(cdiv(blocks, slots) * slots);
    // the new tiles win only by a clear margin over the 128-multiple ones
    const double score = used * kuse * fill * (t.cfg >= mt::kCfgDma256x192 ? 0.95 : 1.0);
    if (score > best_score) {
      best_score = score;
      best = t.cfg;
    }
  }
  return best;
}

int choose_cfg_aligned(int64_t M, int64_t N, int64_t batch, int64_t stages, bool can_split,
                       bool bf16, bool a_kc, bool b_kc, bool vec, int64_t K, int64_t red) {
  auto tiles = [&](int64_t bm, int64_t bn) { return cdiv(M, bm) * cdiv(N, bn) * batch; };
  // share of a tile grid's output that lies inside the matrix
  auto used = [&](int64_t bm, int64_t bn) {
    return (double)(M * N) / (double)(cdiv(M, bm) * bm * cdiv(N, bn) * bn);
  };
  // fp32 products of fewer than ~4 waves of 256x256 tiles on which that tile
  // computes far more than the matrix (e.g. 384 columns as 512) take the
  // smaller tiles below instead (measured on 16 x 8 products of 509 x 384 x
  // 260 and on the gradients of both operands summed over the broadcast axes:
  // 135, 197 and 164 us against 175, 262 and 267 on 256x256)
  const bool wide_waste = !bf16 && M > 0 && N > 0 && tiles(256, 256) < 1024 && used(256, 256) < 0.85;
  // Large products (measured on 8192^3 fp32 and 16384x8192x8192 bf16, all
  // three layouts): the 256x256 tile whose operands stream straight into a
  // two-stage LDS ring, one block of 8 waves per CU, once there are enough
  // tiles to fill every CU.
  // bf16 with both operands K-contiguous (the forward layout) takes the
  // 4-wave form, 128x128 accumulators per wave (measured on 16384 x 8192 x
  // 8192: NT 1.889 -> 1.810 ms; NN 1.809 -> 1.828 and TN 1.788 -> 1.858 ms,
  // so those keep 8 waves)
  if (tiles(256, 256) >= 256 && !wide_waste)
    return bf16 && a_kc && b_kc ? mt::kCfgDma256x256w4 : mt::kCfgDma256x256;
  // A few such tiles over a long contraction (e.g. the weight gradient of a
  // convolution, K = every output pixel): the same tile, its K-stages split
  // into runs that fill the chip once, each run at least kDmaMinRunStages long
  if (can_split && (vec || !bf16) && !wide_waste) {
    const int64_t t = tiles(256, 256);
    const int64_t dma_stages = cdiv(K, bf16 ? 64 : 32) * red;
    if (t > 0 && 256 / t >= 2 && dma_stages / (256 / t) >= kDmaMinRunStages)
      return mt::kCfgDma256x256;
  }
  if (tiles(128, 256) >= 512) return N >= M ? mt::kCfg128x256 : mt::kCfg256x128;
  // mid-size products: the 128x128 tile streamed into an LDS ring, two blocks
  // per CU (measured on 4096 x 1024 x 1024: 96-106 TFLOP/s fp32 against 88-93
  // for the register-staged 128x128 tile); fp32 with 16-byte loads takes its
  // 8-wave form (98-114: one block per CU still has two waves per SIMD), bf16
  // the 4-wave form (the 8-wave one is 3% slower on dX and dW there)
  const int mid = vec ? (bf16 ? mt::kCfgDma128x128 : mt::kCfgDma128x128w8)
                      : (bf16 ? mt::kCfg128x128 : mt::kCfgDma128x128);
  // up to one tile per CU, fp32 with 16-byte loads: the 8-wave form at BK =
  // 64 (one block per CU, half as many stages and barriers; on 4096 x 1024 x
  // 1024: Y +1%, dX +2%, dW +5% split four ways against eight)
  const int small = vec && !bf16 ? mt::kCfgDma128x128k64 : mid;
  const int64_t t128 = tiles(128, 128);
  if (t128 >= 128) return t128 <= 256 ? small : mid;
  if (can_split && t128 * std::min<int64_t>(16, stages / 8) >= 256) {
    // the BK = 64 form only where runs of at least 8 of its stages fill the CUs
    const int64_t runs = t128 > 0 ? std::min<int64_t>(256 / t128, cdiv(K, 64) * red / 8) : 0;
    return t128 * runs >= 256 ? small : mid;
  }
  return mt::kCfg64x64;
}

// Split-K runs for a grid of `blocks` tiles over `stages` K-stages: below
// two blocks per CU, aim for ~512 blocks in all, with at least 8 stages per
// run and at most 16 runs.
int choose_splits(int64_t blocks, int64_t stages, int cfg) {
  if (const int fs = g_force_splits; fs > 0) return (int)std::min<int64_t>(fs, std::max<int64_t>(stages, 1));
  if (cfg == mt::kCfgDma256x256 || cfg == mt::kCfgDma128x128k64 || cfg == mt::kCfgDma256x192) {
    // one block per CU: runs that together fill the 256 CUs once, each at
    // least 1024 (256x256) or 512 (128x128 at BK = 64) deep in K
    if (blocks >= 256) return 1;
    const int64_t min_run = cfg == mt::kCfgDma128x128k64 ? 8 : kDmaMinRunStages;
    int64_t s = std::min<int64_t>(256 / blocks, stages / min_run);
    return s < 1 ? 1 : (int)s;
  }
  if (blocks >= 512) return 1;
  // the 128x128 DMA tiles with a block on every CU already keep the matrix
  // cores as busy as two blocks per CU do, so a split only adds its finish
  // (measured on 4096 x 1024 x 1024, dX unsplit: 121 TFLOP/s against 103-105
  // in two runs)
  if ((cfg == mt::kCfgDma128x128 || cfg == mt::kCfgDma128x128w8) && blocks >= 256) return 1;
  // two blocks per CU: at most 512 blocks, so that the grid stays one wave
  int64_t s = 512 / blocks;
  s = std::min<int64_t>(s, stages / 8);
  s = std::min<int64_t>(s, 16);
  return s < 1 ? 1 : (int)s;
}

// Tiles that carry the dense-layer-with-nonlinearity epilogue: the 256x256
// DMA tile for large products, else the 128x128 DMA tile (register-staged
// for unaligned operands) or 64x64 (a forced cfg outside these maps to the
// nearest of them).
int choose_epi_cfg(int64_t M, int64_t N, bool vec) {
  auto tiles = [&](int64_t bm, int64_t bn) { return cdiv(M, bm) * cdiv(N, bn); };
  if (const int fc = g_force_cfg; fc >= 0) {
    if ((fc == mt::kCfgDma256x256 || fc == mt::kCfgDma128x128) && vec) return fc;
    if (fc == mt::kCfg64x64) return fc;
    return mt::kCfg128x128;
  }
  if (vec && tiles(256, 256) >= 256) return mt::kCfgDma256x256;
  if (tiles(128, 128) >= 128) return vec ? mt::kCfgDma128x128 : mt::kCfg128x128;
  return mt::kCfg64x64;
}

// compute units of the current device (0 if the query fails)
int cu_count() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return cus;
}

void init_params(mt::GemmParams* p) {
  std::memset(p, 0, sizeof(*p));
  p->keep_count = 1;
  p->red_count = 1;
  p->group_m = 4;
  p->splits = 1;
  p->krot = g_krot;
}


// Whether an operand allows 16-byte loads: `per` elements per vector (4 fp32,
// 8 bf16) must divide its contiguous extent, its pitch and every batch
// stride, and its base must be 16-byte aligned.
bool vec_ok_operand(const void* base, int64_t rows_other, int64_t contig_extent, int64_t ld,
                    const int64_t* bstrides, int nb, int per) {
  if (!aligned16(base) || contig_extent % per != 0) return false;
  if (rows_other > 1 && ld % per != 0) return false;
  for (int i = 0; i < nb; ++i)
    if (bstrides[i] % per != 0) return false;
  return true;
}

int vec_elems(bool bf16) { return bf16 ? 8 : 4; }

// Whether the launcher runs tile configuration cfg on the DMA-ring kernel
// (gemm_f32.hip / gemm_bf16.hip): bf16 only with 16-byte loads, fp32 with
// 4-byte lanes on 256x256, 256x128, 128x256, the 4-wave 128x128 and the
// 256x192, 256x96 and 64x384 tiles.
bool dma_kernel(int cfg, bool vec, bool bf16) {
  if (cfg < mt::kCfgDma256x256) return false;
  if (vec) return true;
  return !bf16 && (cfg == mt::kCfgDma256x256 || cfg == mt::kCfgDma256x128 ||
                   cfg == mt::kCfgDma128x256 || cfg == mt::kCfgDma128x128 ||
                   cfg == mt::kCfgDma256x192 || cfg == mt::kCfgDma256x96 ||
                   cfg == mt::kCfgDma64x384);
}

// Byte offset of the split runs' column sums of A in the workspace: after
// the partial tiles, 256-byte aligned.
size_t colsum_part_offset(size_t tiles_bytes) { return (tiles_bytes + 255) & ~(size_t)255; }

// Resolves the tile configuration, vector width and split-K of a product.
// Returns the workspace bytes the split needs (0 = no split). With
// ws_bytes < that, the product runs unsplit.
size_t plan_gemm(GemmCall& g, bool may_split) {
  mt::GemmParams& p = g.p;
  if (g_force_vec1) g.vec = false;
  const int64_t stages_guess = cdiv(p.K, g.bf16 ? 32 : 16) * p.red_count;
  if (g.cfg < 0)
    g.cfg = choose_cfg(p.M, p.N, p.keep_count, stages_guess, may_split, g.bf16, g.a_kc, g.b_kc,
                       g.vec, p.K, p.red_count);
  // the gathering convolution kernels exist on the DMA tiles 256x256 and 128x128
  if (g.conv && !mt::gemm_conv_cfg(g.cfg)) g.cfg = mt::kCfgDma128x128w8;
  // the BK = 64 128x128 tile exists for fp32 with 16-byte lanes only
  if (g.cfg == mt::kCfgDma128x128k64 && (g.bf16 || !g.vec))
    g.cfg = g.bf16 ? mt::kCfgDma128x128 : mt::kCfgDma128x128w8;
  // the 256x192, 256x96 and 64x384 tiles exist for fp32 with 4-byte lanes
  // only, 256x96 with a K-contiguous B only
  if ((g.cfg == mt::kCfgDma256x192 || g.cfg == mt::kCfgDma256x96 || g.cfg == mt::kCfgDma64x384) &&
      (g.vec || g.bf16))
    g.cfg = g.bf16 ? mt::kCfgDma128x128 : mt::kCfgDma256x128;
  if (g.cfg == mt::kCfgDma256x96 && !g.b_kc) g.cfg = mt::kCfgDma256x128;
  // operands or output without 16-byte aligned rows: fp32 keeps the DMA tiles
  // (4-byte lanes, element stores) and maps the register-staged tiles above
  // 128x128 to them; the element-load register-staged kernels stop at 128x128
  if (!g.vec) {
    if (g.cfg == mt::kCfgDma128x128w8) g.cfg = mt::kCfgDma128x128;  // 4-byte lanes: 4 waves
    const bool dma = g.cfg == mt::kCfgDma256x256 || g.cfg == mt::kCfgDma256x128 ||
                     g.cfg == mt::kCfgDma128x256 || g.cfg == mt::kCfgDma128x128 ||
                     g.cfg == mt::kCfgDma256x192 || g.cfg == mt::kCfgDma256x96 ||
                     g.cfg == mt::kCfgDma64x384;
    if (!g.bf16 && (dma || g.cfg == mt::kCfg256x128 || g.cfg == mt::kCfg128x256)) {
      if (g.cfg == mt::kCfg256x128) g.cfg = mt::kCfgDma256x128;
      if (g.cfg == mt::kCfg128x256) g.cfg = mt::kCfgDma128x256;
    } else if (g.cfg != mt::kCfg64x64) {
      g.cfg = mt::kCfg128x128;
    }
  }
  // the column sums of A fold into the DMA kernels of plain TN products and
  // of the convolution's weight gradient only
  if (p.colsum && (g.a_kc || (g.conv && g.conv != 2) || p.nred > 0 || p.keep_count != 1 ||
                   !dma_kernel(g.cfg, g.vec, g.bf16)))
    p.colsum = nullptr;
  p.colsum_part = nullptr;
  const int64_t stages = cdiv(p.K, mt::gemm_tile_k(g.cfg, g.bf16)) * p.red_count;
  p.splits = 1;
  p.stages_per_split = stages > 0 ? stages : 1;
  p.partial = nullptr;
  p.partial_stride = 0;
  g.sk = 0;
  if (!may_split || p.M == 0 || p.N == 0 || p.keep_count == 0 || stages == 0) return 0;
  // The gathered forward / input-gradient products on the 256x256 tile (one
  // block per CU) whose tiles leave CUs idle: stream-K, every CU taking an
  // equal share of the tile-major K-stages; cut tiles are summed by a finish
  // pass
  const int stream_k = g_stream_k;
  if ((g.conv == 1 || g.conv == 3) && g.cfg == mt::kCfgDma256x256 && stream_k) {
    const int sk_blocks = g_sk_blocks;
    const int64_t G = sk_blocks > 0 ? sk_blocks : 256;
    const int64_t T = cdiv(p.M, 256) * cdiv(p.N, 256);
    // more tiles than CUs with a last wave under 90% full, or fewer tiles
    // than CUs (a split by whole runs leaves CUs idle) with at least 16
    // stages per block
    const bool ragged = (T > G && (double)T / (double)(cdiv(T, G) * G) < 0.9 &&
                         T * stages >= G * kDmaMinRunStages) ||
                        (T < G && T * stages >= G * 16);
    // (at least one stage per block keeps the block boundaries distinct)
    if ((stream_k == 2 && T * stages >= G) || ragged) {
      g.sk = (int)G;
      p.partial_stride = p.M * p.N;
      return (size_t)mt::sk_max_segments(T, stages, G) * p.M * p.N * sizeof(float);
    }
  }
  const int64_t blocks = cdiv(p.M, mt::gemm_tile_m(g.cfg)) * cdiv(p.N, mt::gemm_tile_n(g.cfg)) *
                         p.keep_count;
  const int want = choose_splits(blocks, stages, g.cfg);
  if (want <= 1) return 0;
  const int64_t per = cdiv(stages, want);
  const int64_t splits = cdiv(stages, per);
  if (splits <= 1) return 0;
  p.splits = (int32_t)splits;
  p.stages_per_split = per;
  p.partial_stride = p.keep_count * p.M * p.N;
  const size_t tiles_bytes = (size_t)splits * p.partial_stride * sizeof(float);
  // the runs' column sums of A follow the partial tiles
  return p.colsum ? colsum_part_offset(tiles_bytes) + (size_t)splits * p.M * sizeof(float)
                  : tiles_bytes;
}

mt_status launch_gemm(GemmCall& g, hipStream_t stream, void* ws, size_t ws_bytes) {
  mt::GemmParams& p = g.p;
  if (p.M == 0 || p.N == 0 || p.keep_count == 0) return MT_OK;
  const size_t need = plan_gemm(g, ws != nullptr);
  if (g.sk && need > ws_bytes) g.sk = 0;  // no room for the partial tiles: one tile per block
  if (g.sk) {
    p.partial = (float*)ws;
  } else if (need > 0 && need <= ws_bytes) {
    p.partial = (float*)ws;
    if (p.colsum)
      p.colsum_part = (float*)((char*)ws + colsum_part_offset((size_t)p.splits * p.partial_stride *
                                                              sizeof(float)));
  } else {
    p.splits = 1;
    const int64_t stages = cdiv(p.K, mt::gemm_tile_k(g.cfg, g.bf16)) * p.red_count;
    p.stages_per_split = stages > 0 ? stages : 1;
  }
  // 32-bit buffer offsets: one tile's rows times the row pitch must stay below 2 GiB
  const int64_t es = g.bf16 ? 2 : 4;
  const int64_t rows_a = g.a_kc ? mt::gemm_tile_m(g.cfg) : mt::gemm_tile_k(g.cfg, g.bf16);
  const int64_t rows_b = g.b_kc ? mt::gemm_tile_n(g.cfg) : mt::gemm_tile_k(g.cfg, g.bf16);
  if (rows_a * p.lda * es >= (int64_t)1 << 31 || rows_b * p.ldb * es >= (int64_t)1 << 31)
    return fail(MT_ERR_LAYOUT, "row pitch too large for 32-bit tile offsets");
  (void)hipGetLastError();  // clear a stale error so the launch check is ours
  // plain products (column sums of A included) on the one-block-per-CU DMA
  // tiles with more tiles than CUs and whole tiles only (M, N multiples of
  // 256): a persistent grid, whose blocks run their tiles back to back so
  // that each tile's first loads overlap the previous tile's last stage and
  // its stores overlap the next tile's work. fp32 TN products (dW) stay on
  // the plain grid: 0.5% slower persistent at 8192^3, with db or without
  // (bf16 dW + db: 1.1% faster persistent)
  p.persist = 0;
  if (g_persist && !g.conv && !g.sk && g.vec && p.splits == 1 && p.keep_count == 1 &&
      p.red_count == 1 && !p.z && p.act == 0 && !p.accumulate && (g.bf16 || g.a_kc) &&
      (g.cfg == mt::kCfgDma256x256 || g.cfg == mt::kCfgDma256x256w4)) {
    const int cus = cu_count() & ~7;
    if (cus >= 8 && p.M % 256 == 0 && p.N % 256 == 0 && (p.M / 256) * (p.N / 256) > cus)
      p.persist = cus;
  }
  if (g.sk) return hip_status(mt::gemm_f32_conv_sk(p, g.conv, g.sk, stream));
  hipError_t e = g.conv   ? mt::gemm_f32_conv(p, g.conv, g.cfg, stream)
                 : g.bf16 ? mt::gemm_bf16(p, g.a_kc, g.b_kc, g.vec, g.cfg, stream)
                          : mt::gemm_f32(p, g.a_kc, g.b_kc, g.vec, g.cfg, stream);
  if (e != hipSuccess) return hip_status(e);
  if (p.splits > 1) {
    // batch elements of C are contiguous M x N blocks when batched (mt_matmul)
    // the column sums (unbatched products only) are added by the same finish
    e = mt::splitk_finish(p.partial, p.splits, p.keep_count * p.M, p.N, p.c, p.ldc, p.bias,
                          p.accumulate != 0, stream, p.colsum ? p.colsum_part : nullptr, p.colsum);
    if (e != hipSuccess) return hip_status(e);
  }
  return MT_OK;
}

mt_status check_matrix(const mt_tensor* t, const char* name) {
  mt_status s = check_tensor(t, name, 2, 2);
  if (s) return s;
  if (t->shape[1] > 1 && t->stride[1] != 1)
    return fail(MT_ERR_LAYOUT, std::string(name) + ": inner dim must be contiguous (stride 1)");
  return MT_OK;
}

int64_t pitch(const mt_tensor* t) {
  return t->shape[0] > 1 ? t->stride[0] : (t->shape[1] > 0 ? t->shape[1] : 1);
}

mt_status check_out_matrix(const mt_tensor* t, const char* name) {
  mt_status s = check_matrix(t, name);
  if (s) return s;
  if (t->dtype != MT_F32) return fail(MT_ERR_DTYPE, std::string(name) + ": outputs are f32");
  if (t->shape[0] > 1 && t->stride[0] < t->shape[1])
    return fail(MT_ERR_LAYOUT, std::string(name) + ": rows overlap (row pitch < columns)");
  return MT_OK;
}

mt_status check_vector(const mt_tensor* t, const char* name, int64_t n) {
  mt_status s = check_tensor(t, name, 1, 1);
  if (s) return s;
  if (t->dtype != MT_F32) return fail(MT_ERR_DTYPE, std::string(name) + ": must be f32");
  if (t->shape[0] != n)
    return fail(MT_ERR_SHAPE, std::string(name) + ": length " + std::to_string(t->shape[0]) +
                                  ", expected " + std::to_string(n));
  if (n > 1 && t->stride[0] != 1) return fail(MT_ERR_LAYOUT, std::string(name) + ": must be contiguous");
  return MT_OK;
}

mt_status linear_bwd_impl(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                          const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db,
                          uint32_t flags, void* ws, size_t ws_bytes, hipStream_t stream,
                          size_t* ws_query) {
  if (flags & ~MT_ACCUMULATE) return fail(MT_ERR_INVALID, "mt_linear_bwd: unknown flags");
  mt_status s = check_matrix(dy, "dy");
  if (s) return s;
  const int64_t M = dy->shape[0], N = dy->shape[1];
  const int32_t dt = dy->dtype;
  int64_t K = -1;
  if (dw) {
    if ((s = check_matrix(x, "x"))) return s;
    if (x->dtype != dt) return fail(MT_ERR_DTYPE, "x and dy must share a dtype");
    if (x->shape[0] != M) return fail(MT_ERR_SHAPE, "x rows must equal dy rows");
    K = x->shape[1];
  }
  if (dx) {
    if ((s = check_matrix(w, "w"))) return s;
    if (w->dtype != dt) return fail(MT_ERR_DTYPE, "w and dy must share a dtype");
    if (w->shape[0] != N) return fail(MT_ERR_SHAPE, "w rows must equal dy columns");
    if (K >= 0 && w->shape[1] != K) return fail(MT_ERR_SHAPE, "w and x disagree on K");
    K = w->shape[1];
  }
  if (dx) {
    if ((s = check_out_matrix(dx, "dx"))) return s;
    if (dx->shape[0] != M || dx->shape[1] != K) return fail(MT_ERR_SHAPE, "dx must be [M, K]");
  }
  if (dw) {
    if ((s = check_out_matrix(dw, "dw"))) return s;
    if (dw->shape[0] != N || dw->shape[1] != K) return fail(MT_ERR_SHAPE, "dw must be [N, K]");
  }
  if (db && (s = check_vector(db, "db", N))) return s;
  const bool bf = dt == MT_BF16;
  const int per = vec_elems(bf);
  // inputs actually read: dy always, x for dw, w for dx
  const mt_tensor* ins[3] = {dy, dw ? x : nullptr, dx ? w : nullptr};
  const mt_tensor* outs[3] = {dx, dw, db};
  for (int i = 0; i < 3; ++i) {
    if (!outs[i]) continue;
    for (int j = 0; j < 3; ++j)
      if (overlaps(outs[i], ins[j])) return fail(MT_ERR_ALIAS, "an output overlaps an input");
    for (int j = i + 1; j < 3; ++j)
      if (overlaps(outs[i], outs[j])) return fail(MT_ERR_ALIAS, "outputs overlap");
  }
  const bool acc = (flags & MT_ACCUMULATE) != 0;

  // workspace needs (used in turn on the stream, so the size is the max):
  // dx / dw split-K partials and db row-slice sums
  GemmCall gdx{}, gdw{};
  size_t need_dx = 0, need_dw = 0, need_db = 0;
  bool fold_db = false;
  if (dx && M > 0 && K > 0) {
    init_params(&gdx.p);
    gdx.p.a = dy->data;
    gdx.p.b = w->data;
    gdx.p.c = (float*)dx->data;
    gdx.p.M = M;
    gdx.p.N = K;
    gdx.p.K = N;
    gdx.p.lda = pitch(dy);
    gdx.p.ldb = pitch(w);
    gdx.p.ldc = pitch(dx);
    gdx.p.accumulate = acc;
    gdx.a_kc = true;
    gdx.b_kc = false;
    gdx.bf16 = bf;
    gdx.vec = vec_ok_operand(dy->data, M, N, gdx.p.lda, nullptr, 0, per) &&
              vec_ok_operand(w->data, N, K, gdx.p.ldb, nullptr, 0, per) && aligned16(dx->data) &&
              K % 4 == 0 && gdx.p.ldc % 4 == 0;
    gdx.cfg = -1;
    GemmCall probe = gdx;
    need_dx = plan_gemm(probe, true);
  }
  if (dw && N > 0 && K > 0) {
    init_params(&gdw.p);
    gdw.p.a = dy->data;
    gdw.p.b = x->data;
    gdw.p.c = (float*)dw->data;
    gdw.p.M = N;
    gdw.p.N = K;
    gdw.p.K = M;
    gdw.p.lda = pitch(dy);
    gdw.p.ldb = pitch(x);
    gdw.p.ldc = pitch(dw);
    gdw.p.accumulate = acc;
    gdw.a_kc = false;
    gdw.b_kc = false;
    gdw.bf16 = bf;
    gdw.vec = vec_ok_operand(dy->data, M, N, gdw.p.lda, nullptr, 0, per) &&
              vec_ok_operand(x->data, M, K, gdw.p.ldb, nullptr, 0, per) &&
              aligned16(dw->data) && K % 4 == 0 && gdw.p.ldc % 4 == 0;
    gdw.cfg = -1;
    // db = 1^T dY is the column sum of A = dY^T: folded into the dW product
    // where its kernel allows (no second pass over dY)
    // (whether it does is settled by the plan of the launch, below: without
    // a workspace the product may take a tile that cannot)
    gdw.p.colsum = db ? (float*)db->data : nullptr;
    GemmCall probe = gdw;
    need_dw = plan_gemm(probe, true);
    fold_db = probe.p.colsum != nullptr;
  }
  int parts = 1;
  if (db && N > 0) {
    const int fp = g_force_parts;
    parts = fp > 0 ? fp : mt::colsum_parts(M, N);
    if (parts > 1 && !fold_db) need_db = (size_t)parts * N * sizeof(float);
  }
  if (ws_query) {
    *ws_query = std::max(need_dx, std::max(need_dw, need_db));
    return MT_OK;
  }
  if (ws && ((uintptr_t)ws & 255))
    return fail(MT_ERR_WORKSPACE, "workspace must be 256-byte aligned");

  if (dx && M > 0 && K > 0) {
    if ((s = launch_gemm(gdx, stream, ws, ws_bytes))) return s;
  }
  fold_db = false;
  if (dw && N > 0 && K > 0) {
    if ((s = launch_gemm(gdw, stream, ws, ws_bytes))) return s;
    fold_db = gdw.p.colsum != nullptr;  // the product summed db itself
  }
  if (db && N > 0 && !fold_db) {
    (void)hipGetLastError();
    const bool room = ws_bytes >= (size_t)parts * N * sizeof(float);
    float* wsp = (ws && parts > 1 && room) ? (float*)ws : nullptr;
    hipError_t e = mt::colsum(dy->data, bf, M, N, pitch(dy), (float*)db->data, acc,
                              wsp, parts, stream);
    if (e != hipSuccess) return hip_status(e);
  }
  return MT_OK;
}

mt_status matmul_impl(const mt_tensor* a, const mt_tensor* b, const mt_tensor* c, uint32_t flags,
                      void* ws, size_t ws_bytes, hipStream_t stream, size_t* ws_query) {
  if (flags & ~(MT_ACCUMULATE | MT_REDUCE_INTO)) return fail(MT_ERR_INVALID, "mt_matmul: unknown flags");
  mt_status s;
  if ((s = check_tensor(a, "a", 1, MT_MAX_DIMS))) return s;
  if ((s = check_tensor(b, "b", 1, MT_MAX_DIMS))) return s;
  if ((s = check_tensor(c, "c", 0, MT_MAX_DIMS))) return s;
  if (a->dtype != b->dtype) return fail(MT_ERR_DTYPE, "a and b must share a dtype");
  if (c->dtype != MT_F32) return fail(MT_ERR_DTYPE, "c must be f32");
  mt::MatmulPlan pl;
  std::string err;
  if ((s = mt::plan_matmul_shapes(a->ndim, a->shape, a->stride, b->ndim, b->shape, b->stride, &pl,
                                  &err)))
    return fail(s, "mt_matmul: " + err);
  if (!is_row_major(c)) return fail(MT_ERR_LAYOUT, "c must be row-major contiguous");
  // match c against the result shape (exact, or summed over batch dims)
  const int nmat = pl.nout - pl.nbatch;  // result dims after the batch dims (0..2)
  if (c->ndim < nmat || c->ndim > pl.nout) return fail(MT_ERR_SHAPE, "c has the wrong rank");
  for (int i = 0; i < nmat; ++i)
    if (c->shape[c->ndim - nmat + i] != pl.out[pl.nbatch + i])
      return fail(MT_ERR_SHAPE, "c matrix dims do not match the product");
  const bool reduce_into = (flags & MT_REDUCE_INTO) != 0;
  const int cb = c->ndim - nmat;  // c batch rank
  if (!reduce_into && cb != pl.nbatch) return fail(MT_ERR_SHAPE, "c has the wrong rank (no MT_REDUCE_INTO)");
  mt::GemmParams p;
  init_params(&p);
  int64_t c_batch_stride[MT_MAX_DIMS];
  {
    int64_t st = 1;
    for (int i = c->ndim - 1; i >= 0; --i) {
      if (i < cb) c_batch_stride[i] = st;
      st *= c->shape[i];
    }
  }
  for (int d = 0; d < pl.nbatch; ++d) {
    const int ci = d - (pl.nbatch - cb);
    const int64_t cd = ci >= 0 ? c->shape[ci] : 1;
    if (cd == pl.batch[d]) {
      if (cd == 1) continue;
      p.keep_shape[p.nkeep] = cd;
      p.keep_sa[p.nkeep] = pl.sa[d];
      p.keep_sb[p.nkeep] = pl.sb[d];
      p.keep_sc[p.nkeep] = c_batch_stride[ci];
      ++p.nkeep;
    } else if (cd == 1 && reduce_into) {
      p.red_shape[p.nred] = pl.batch[d];
      p.red_sa[p.nred] = pl.sa[d];
      p.red_sb[p.nred] = pl.sb[d];
      ++p.nred;
    } else {
      return fail(MT_ERR_SHAPE, "c batch dims do not match the product");
    }
  }
  if (overlaps(c, a) || overlaps(c, b)) return fail(MT_ERR_ALIAS, "c overlaps an input");
  for (int i = 0; i < p.nkeep; ++i) p.keep_count *= p.keep_shape[i];
  for (int i = 0; i < p.nred; ++i) p.red_count *= p.red_shape[i];
  if (pl.M == 0 || pl.N == 0 || p.keep_count == 0) {
    if (ws_query) *ws_query = 0;
    return MT_OK;
  }
  GemmCall g{};
  g.p = p;
  bool a_kc, b_kc;
  int64_t lda, ldb;
  if (!mt::operand_layout(pl.a, true, &a_kc, &lda))
    return fail(MT_ERR_LAYOUT, "a: neither matrix dim is contiguous");
  if (!mt::operand_layout(pl.b, false, &b_kc, &ldb))
    return fail(MT_ERR_LAYOUT, "b: neither matrix dim is contiguous");
  g.p.a = a->data;
  g.p.b = b->data;
  g.p.c = (float*)c->data;
  g.p.M = pl.M;
  g.p.N = pl.N;
  g.p.K = pl.K;
  g.p.lda = lda;
  g.p.ldb = ldb;
  g.p.ldc = pl.N;
  g.p.accumulate = (flags & MT_ACCUMULATE) != 0;
  if (p.red_count == 0) g.p.K = 0;  // an empty summed batch contributes nothing
  g.a_kc = a_kc;
  g.b_kc = b_kc;
  g.bf16 = a->dtype == MT_BF16;
  const int per = vec_elems(g.bf16);
  int64_t sa_all[2 * MT_MAX_DIMS], sb_all[2 * MT_MAX_DIMS];
  int na = 0;
  for (int i = 0; i < p.nkeep; ++i) { sa_all[na] = p.keep_sa[i]; sb_all[na++] = p.keep_sb[i]; }
  for (int i = 0; i < p.nred; ++i) { sa_all[na] = p.red_sa[i]; sb_all[na++] = p.red_sb[i]; }
  g.vec = vec_ok_operand(a->data, a_kc ? pl.M : pl.K, a_kc ? pl.K : pl.M, lda, sa_all, na, per) &&
          vec_ok_operand(b->data, b_kc ? pl.N : pl.K, b_kc ? pl.K : pl.N, ldb, sb_all, na, per) &&
          aligned16(c->data) && pl.N % 4 == 0;
  g.cfg = -1;
  if (ws_query) {
    GemmCall probe = g;
    *ws_query = plan_gemm(probe, true);
    return MT_OK;
  }
  if (ws && ((uintptr_t)ws & 255)) return fail(MT_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return launch_gemm(g, stream, ws, ws_bytes);
}

mt_status reduce_impl(const mt_tensor* go, const mt_tensor* gi, uint32_t flags, void* ws,
                      size_t ws_bytes, hipStream_t stream, size_t* ws_query) {
  if (flags & ~MT_ACCUMULATE) return fail(MT_ERR_INVALID, "mt_reduce_broadcast_grad: unknown flags");
  mt_status s;
  if ((s = check_tensor(go, "grad_out", 0, MT_MAX_DIMS))) return s;
  if ((s = check_tensor(gi, "grad_in", 0, MT_MAX_DIMS))) return s;
  if (go->dtype != MT_F32 || gi->dtype != MT_F32)
    return fail(MT_ERR_DTYPE, "grad_out and grad_in must be f32");
  if (!is_row_major(gi)) return fail(MT_ERR_LAYOUT, "grad_in must be row-major contiguous");
  mt::ReducePlan plan;
  std::string err;
  if ((s = mt::plan_reduce(go->ndim, go->shape, go->stride, gi->ndim, gi->shape, &plan, &err)))
    return fail(s, "mt_reduce_broadcast_grad: " + err);
  const int fp = g_force_parts;
  const int parts = fp > 0 ? fp : mt::reduce_parts(plan);
  const size_t need = parts > 1 ? (size_t)parts * plan.keep_count * sizeof(float) : 0;
  if (ws_query) {
    *ws_query = need;
    return MT_OK;
  }
  if (overlaps(go, gi)) return fail(MT_ERR_ALIAS, "grad_in overlaps grad_out");
  if (ws && ((uintptr_t)ws & 255)) return fail(MT_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  (void)hipGetLastError();
  float* wsp = (ws && need && ws_bytes >= need) ? (float*)ws : nullptr;
  return hip_status(mt::reduce_strided((const float*)go->data, plan, (float*)gi->data,
                                       (flags & MT_ACCUMULATE) != 0, wsp, wsp ? parts : 1, stream));
}

mt_status linear_fwd_impl(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b, int32_t act,
                          const mt_tensor* z, const mt_tensor* y, hipStream_t stream) {
  {
    mt_status s;
    if ((s = check_matrix(x, "x")) || (s = check_matrix(w, "w")) ||
        (s = check_out_matrix(y, "y")))
      return s;
    if (x->dtype != w->dtype) return fail(MT_ERR_DTYPE, "x and w must share a dtype");
    const int64_t M = x->shape[0], K = x->shape[1], N = w->shape[0];
    if (w->shape[1] != K) return fail(MT_ERR_SHAPE, "w must be [N, K] with x [M, K]");
    if (y->shape[0] != M || y->shape[1] != N) return fail(MT_ERR_SHAPE, "y must be [M, N]");
    if (b && (s = check_vector(b, "b", N))) return s;
    if (act < 0 || act >= mt::kNumAct) return fail(MT_ERR_INVALID, "unknown activation");
    if (z) {
      if ((s = check_out_matrix(z, "z"))) return s;
      if (z->shape[0] != M || z->shape[1] != N) return fail(MT_ERR_SHAPE, "z must be [M, N]");
      if (overlaps(z, x) || overlaps(z, w) || overlaps(z, b) || overlaps(z, y))
        return fail(MT_ERR_ALIAS, "z overlaps an input or y");
    }
    const bool bf = x->dtype == MT_BF16;
    const int per = vec_elems(bf);
    if (overlaps(y, x) || overlaps(y, w) || overlaps(y, b))
      return fail(MT_ERR_ALIAS, "y overlaps an input");
    if (M == 0 || N == 0) return MT_OK;
    GemmCall g{};
    init_params(&g.p);
    g.p.a = x->data;
    g.p.b = w->data;
    g.p.c = (float*)y->data;
    g.p.bias = (b && N > 0) ? (const float*)b->data : nullptr;
    g.p.M = M;
    g.p.N = N;
    g.p.K = K;
    g.p.lda = pitch(x);
    g.p.ldb = pitch(w);
    g.p.ldc = pitch(y);
    g.a_kc = true;
    g.b_kc = true;
    g.bf16 = bf;
    g.vec = vec_ok_operand(x->data, M, K, g.p.lda, nullptr, 0, per) &&
            vec_ok_operand(w->data, N, K, g.p.ldb, nullptr, 0, per) && aligned16(y->data) &&
            N % 4 == 0 && g.p.ldc % 4 == 0 && (!g.p.bias || aligned16(g.p.bias)) &&
            (!z || (aligned16(z->data) && pitch(z) % 4 == 0));
    g.cfg = -1;
    if (act != mt::kActNone || z) {
      g.p.act = act;
      g.p.z = z ? (float*)z->data : nullptr;
      g.p.ldz = z ? pitch(z) : 0;
      g.cfg = choose_epi_cfg(M, N, g.vec);
    }
    return launch_gemm(g, stream, nullptr, 0);
  }
}



// ------------------------------------------------------------- act_bwd
mt_status act_bwd_impl(int32_t act, const mt_tensor* z, const mt_tensor* dy, const mt_tensor* dz,
                       const mt_tensor* db, uint32_t flags, void* ws, size_t ws_bytes,
                       hipStream_t stream, size_t* ws_query) {
  if (flags & ~MT_ACCUMULATE) return fail(MT_ERR_INVALID, "mt_act_bwd: unknown flags");
  if (act < 0 || act >= mt::kNumAct) return fail(MT_ERR_INVALID, "unknown activation");
  mt_status s;
  if ((s = check_matrix(z, "z")) || (s = check_matrix(dy, "dy")) || (s = check_matrix(dz, "dz")))
    return s;
  if (z->dtype != MT_F32) return fail(MT_ERR_DTYPE, "z (the saved pre-activation) must be f32");
  if (dz->dtype != dy->dtype) return fail(MT_ERR_DTYPE, "dz must have dy's dtype");
  const int64_t M = z->shape[0], N = z->shape[1];
  if (dy->shape[0] != M || dy->shape[1] != N || dz->shape[0] != M || dz->shape[1] != N)
    return fail(MT_ERR_SHAPE, "z, dy and dz must share one [M, N] shape");
  if (dz->shape[0] > 1 && dz->stride[0] < dz->shape[1])
    return fail(MT_ERR_LAYOUT, "dz: rows overlap (row pitch < columns)");
  if (db && (s = check_vector(db, "db", N))) return s;
  if (overlaps(dz, z) || overlaps(dz, dy) || overlaps(db, z) || overlaps(db, dy) ||
      overlaps(db, dz))
    return fail(MT_ERR_ALIAS, "an output overlaps an input or the other output");
  int parts = 1;
  if (const int fp = g_force_parts; db && M > 0 && N > 0) parts = fp > 0 ? fp : mt::colsum_parts(M, N);
  const size_t need = parts > 1 ? (size_t)parts * N * sizeof(float) : 0;
  if (ws_query) {
    *ws_query = need;
    return MT_OK;
  }
  if (ws && ((uintptr_t)ws & 255)) return fail(MT_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  float* wsp = (ws && need && ws_bytes >= need) ? (float*)ws : nullptr;
  const bool acc = (flags & MT_ACCUMULATE) != 0;
  (void)hipGetLastError();
  return hip_status(mt::act_bwd(act, (const float*)z->data, pitch(z), dy->data, pitch(dy),
                                dz->data, pitch(dz), dy->dtype == MT_BF16, M, N, acc,
                                db ? (float*)db->data : nullptr, acc, wsp, wsp ? parts : 1,
                                stream));
}

// ----------------------------------------------------------------- mse
mt_status check_dense_f32(const mt_tensor* t, const char* name) {
  mt_status s = check_tensor(t, name, 0, MT_MAX_DIMS);
  if (s) return s;
  if (t->dtype != MT_F32) return fail(MT_ERR_DTYPE, std::string(name) + ": must be f32");
  if (!is_row_major(t)) return fail(MT_ERR_LAYOUT, std::string(name) + ": must be contiguous");
  return MT_OK;
}

bool same_shape(const mt_tensor* a, const mt_tensor* b) {
  if (a->ndim != b->ndim) return false;
  for (int i = 0; i < a->ndim; ++i)
    if (a->shape[i] != b->shape[i]) return false;
  return true;
}

mt_status mse_impl(const mt_tensor* pred, const mt_tensor* target, const mt_tensor* loss,
                   const mt_tensor* dpred, void* ws, size_t ws_bytes, hipStream_t stream,
                   size_t* ws_query) {
  mt_status s;
  if ((s = check_dense_f32(pred, "pred")) || (s = check_dense_f32(target, "target"))) return s;
  if (!same_shape(pred, target)) return fail(MT_ERR_SHAPE, "pred and target shapes differ");
  const int64_t n = numel(pred);
  const int parts = mt::mse_parts(n);
  const size_t need = parts > 1 ? (size_t)parts * sizeof(float) : 0;
  if (ws_query) {
    *ws_query = need;
    return MT_OK;
  }
  if (!loss && !dpred) return fail(MT_ERR_NULL, "mt_mse_loss: neither loss nor dpred given");
  if (loss) {
    if ((s = check_dense_f32(loss, "loss"))) return s;
    if (numel(loss) != 1) return fail(MT_ERR_SHAPE, "loss must hold exactly one element");
  }
  if (dpred) {
    if ((s = check_dense_f32(dpred, "dpred"))) return s;
    if (!same_shape(dpred, pred)) return fail(MT_ERR_SHAPE, "dpred must have pred's shape");
  }
  if (overlaps(loss, pred) || overlaps(loss, target) || overlaps(dpred, pred) ||
      overlaps(dpred, target) || overlaps(loss, dpred))
    return fail(MT_ERR_ALIAS, "an output overlaps an input or the other output");
  if (ws && ((uintptr_t)ws & 255)) return fail(MT_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  float* wsp = (ws && need && ws_bytes >= need) ? (float*)ws : nullptr;
  (void)hipGetLastError();
  return hip_status(mt::mse((const float*)pred->data, (const float*)target->data, n,
                            dpred ? (float*)dpred->data : nullptr,
                            loss ? (float*)loss->data : nullptr, wsp, wsp ? parts : 1, stream));
}

// ---------------------------------------------------------- optimizers
// Validates n (param, grad, state...) tuples of contiguous f32 tensors of one
// shape each, with no output overlapping anything else, and packs them into
// launches of up to kOptMaxTensors tensors.
mt_status plan_opt(int32_t n, const mt_tensor* params, const mt_tensor* grads,
                   const mt_tensor* st1, const mt_tensor* st2, const char* who,
                   std::vector<mt::OptBatch>* out) {
  if (n < 0) return fail(MT_ERR_INVALID, std::string(who) + ": negative tensor count");
  if (n > 0 && (!params || !grads || !st1)) return fail(MT_ERR_NULL, std::string(who) + ": null array");
  const std::string w(who);
  std::vector<const mt_tensor*> outs;  // every tensor written
  for (int32_t i = 0; i < n; ++i) {
    const mt_tensor* ts[4] = {&params[i], &grads[i], &st1[i], st2 ? &st2[i] : nullptr};
    const char* names[4] = {"param", "grad", "state", "state2"};
    for (int j = 0; j < 4; ++j) {
      if (!ts[j]) continue;
      mt_status s = check_dense_f32(ts[j], (w + ": " + names[j] + " " + std::to_string(i)).c_str());
      if (s) return s;
      if (!same_shape(ts[j], ts[0]))
        return fail(MT_ERR_SHAPE, w + ": tensor " + std::to_string(i) + " has mismatched shapes");
    }
    outs.push_back(ts[0]);
    outs.push_back(ts[2]);
    if (ts[3]) outs.push_back(ts[3]);
  }
  // outputs overlap no output and no gradient
  for (size_t a = 0; a < outs.size(); ++a) {
    for (size_t b = a + 1; b < outs.size(); ++b)
      if (overlaps(outs[a], outs[b])) return fail(MT_ERR_ALIAS, w + ": updated tensors overlap");
    for (int32_t i = 0; i < n; ++i)
      if (overlaps(outs[a], &grads[i]))
        return fail(MT_ERR_ALIAS, w + ": an updated tensor overlaps a gradient");
  }
  mt::OptBatch cur{};
  for (int32_t i = 0; i < n; ++i) {
    const int64_t cnt = numel(&params[i]);
    if (cnt == 0) continue;
    if (cur.n == mt::kOptMaxTensors) {
      out->push_back(cur);
      cur = mt::OptBatch{};
    }
    const int k = cur.n++;
    cur.param[k] = (float*)params[i].data;
    cur.grad[k] = (const float*)grads[i].data;
    cur.state1[k] = (float*)st1[i].data;
    cur.state2[k] = st2 ? (float*)st2[i].data : nullptr;
    cur.numel[k] = cnt;
    cur.vec[k] = aligned16(params[i].data) && aligned16(grads[i].data) && aligned16(st1[i].data) &&
                 (!st2 || aligned16(st2[i].data));
  }
  if (cur.n > 0) out->push_back(cur);
  return MT_OK;
}


}  // namespace mt::host

using namespace mt::host;

extern "C" {

mt_status mt_linear_fwd(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b,
                        const mt_tensor* y, void* stream) {
  try {
    return linear_fwd_impl(x, w, b, mt::kActNone, nullptr, y, (hipStream_t)stream);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_linear_act_fwd(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b,
                            int32_t act, const mt_tensor* z, const mt_tensor* y, void* stream) {
  try {
    return linear_fwd_impl(x, w, b, act, z, y, (hipStream_t)stream);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_act_bwd(int32_t act, const mt_tensor* z, const mt_tensor* dy, const mt_tensor* dz,
                     const mt_tensor* db, uint32_t flags, void* ws, size_t ws_bytes,
                     void* stream) {
  try {
    return act_bwd_impl(act, z, dy, dz, db, flags, ws, ws_bytes, (hipStream_t)stream, nullptr);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_act_bwd_workspace(int32_t act, const mt_tensor* z, const mt_tensor* dy,
                               const mt_tensor* dz, const mt_tensor* db, size_t* bytes) {
  try {
    if (!bytes) return fail(MT_ERR_NULL, "bytes is null");
    return act_bwd_impl(act, z, dy, dz, db, 0, nullptr, 0, nullptr, bytes);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_mse_loss(const mt_tensor* pred, const mt_tensor* target, const mt_tensor* loss,
                      const mt_tensor* dpred, void* ws, size_t ws_bytes, void* stream) {
  try {
    return mse_impl(pred, target, loss, dpred, ws, ws_bytes, (hipStream_t)stream, nullptr);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_mse_loss_workspace(const mt_tensor* pred, const mt_tensor* target, size_t* bytes) {
  try {
    if (!bytes) return fail(MT_ERR_NULL, "bytes is null");
    return mse_impl(pred, target, nullptr, nullptr, nullptr, 0, nullptr, bytes);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_sgd_step(int32_t n, const mt_tensor* params, const mt_tensor* grads,
                      const mt_tensor* velocity, float lr, float momentum, float weight_decay,
                      void* stream) {
  try {
    if (!std::isfinite(lr) || !std::isfinite(momentum) || !std::isfinite(weight_decay))
      return fail(MT_ERR_INVALID, "mt_sgd_step: lr, momentum and weight_decay must be finite");
    std::vector<mt::OptBatch> batches;
    mt_status s = plan_opt(n, params, grads, velocity, nullptr, "mt_sgd_step", &batches);
    if (s) return s;
    (void)hipGetLastError();
    for (const auto& b : batches)
      if ((s = hip_status(mt::sgd_step(b, lr, momentum, weight_decay, (hipStream_t)stream))))
        return s;
    return MT_OK;
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_adam_step(int32_t n, const mt_tensor* params, const mt_tensor* grads,
                       const mt_tensor* exp_avg, const mt_tensor* exp_avg_sq, float lr, float beta1,
                       float beta2, float eps, int64_t step, void* stream) {
  try {
    if (!std::isfinite(lr) || !(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f) ||
        !(eps >= 0.f) || !std::isfinite(eps))
      return fail(MT_ERR_INVALID, "mt_adam_step: needs finite lr, 0 <= beta < 1, finite eps >= 0");
    if (step < 1) return fail(MT_ERR_INVALID, "mt_adam_step: step counts from 1");
    std::vector<mt::OptBatch> batches;
    mt_status s = plan_opt(n, params, grads, exp_avg, exp_avg_sq, "mt_adam_step", &batches);
    if (s) return s;
    // bias corrections 1 / (1 - beta^t) in double, then rounded once
    const double bc1 = 1.0 - std::pow((double)beta1, (double)step);
    const double bc2 = 1.0 - std::pow((double)beta2, (double)step);
    const float inv_bc1 = (float)(1.0 / bc1), inv_bc2 = (float)(1.0 / bc2);
    if (!std::isfinite(inv_bc1) || !std::isfinite(inv_bc2))
      return fail(MT_ERR_INVALID, "mt_adam_step: bias correction 1 - beta^step underflows to 0");
    (void)hipGetLastError();
    for (const auto& b : batches)
      if ((s = hip_status(mt::adam_step(b, lr, beta1, beta2, eps, inv_bc1, inv_bc2,
                                        (hipStream_t)stream))))
        return s;
    return MT_OK;
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_rmsprop_step(int32_t n, const mt_tensor* params, const mt_tensor* grads,
                          const mt_tensor* sq_avg, float lr, float alpha, float eps, void* stream) {
  try {
    if (!std::isfinite(lr) || !(alpha >= 0.f && alpha <= 1.f) || !(eps >= 0.f) ||
        !std::isfinite(eps))
      return fail(MT_ERR_INVALID, "mt_rmsprop_step: needs finite lr, 0 <= alpha <= 1, finite eps >= 0");
    std::vector<mt::OptBatch> batches;
    mt_status s = plan_opt(n, params, grads, sq_avg, nullptr, "mt_rmsprop_step", &batches);
    if (s) return s;
    (void)hipGetLastError();
    for (const auto& b : batches)
      if ((s = hip_status(mt::rmsprop_step(b, lr, alpha, eps, (hipStream_t)stream)))) return s;
    return MT_OK;
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_linear_bwd(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                        const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db,
                        uint32_t flags, void* ws, size_t ws_bytes, void* stream) {
  try {
    return linear_bwd_impl(x, w, dy, dx, dw, db, flags, ws, ws_bytes, (hipStream_t)stream, nullptr);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_linear_bwd_workspace(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                                  const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db,
                                  size_t* bytes) {
  try {
    if (!bytes) return fail(MT_ERR_NULL, "bytes is null");
    return linear_bwd_impl(x, w, dy, dx, dw, db, 0, nullptr, 0, nullptr, bytes);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_matmul(const mt_tensor* a, const mt_tensor* b, const mt_tensor* c, uint32_t flags,
                    void* ws, size_t ws_bytes, void* stream) {
  try {
    return matmul_impl(a, b, c, flags, ws, ws_bytes, (hipStream_t)stream, nullptr);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_matmul_workspace(const mt_tensor* a, const mt_tensor* b, const mt_tensor* c,
                              uint32_t flags, size_t* bytes) {
  try {
    if (!bytes) return fail(MT_ERR_NULL, "bytes is null");
    return matmul_impl(a, b, c, flags, nullptr, 0, nullptr, bytes);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_reduce_broadcast_grad(const mt_tensor* grad_out, const mt_tensor* grad_in,
                                   uint32_t flags, void* ws, size_t ws_bytes, void* stream) {
  try {
    return reduce_impl(grad_out, grad_in, flags, ws, ws_bytes, (hipStream_t)stream, nullptr);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_reduce_broadcast_grad_workspace(const mt_tensor* grad_out, const mt_tensor* grad_in,
                                             size_t* bytes) {
  try {
    if (!bytes) return fail(MT_ERR_NULL, "bytes is null");
    return reduce_impl(grad_out, grad_in, 0, nullptr, 0, nullptr, bytes);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}


size_t mt_workspace_bytes(int32_t op, const mt_tensor* const* args, int32_t nargs) {
  try {
    static const int32_t want[] = {3, 3, 4, 6, 2, 2};
    if (op < 0 || op > MT_OP_MSE_LOSS) {
      fail(MT_ERR_INVALID, "mt_workspace_bytes: unknown op");
      return SIZE_MAX;
    }
    if (!args || nargs != want[op]) {
      fail(MT_ERR_INVALID, "mt_workspace_bytes: wrong argument count for this op");
      return SIZE_MAX;
    }
    size_t n = 0;
    mt_status s = MT_OK;
    switch (op) {
      case MT_OP_MATMUL: s = matmul_impl(args[0], args[1], args[2], 0, nullptr, 0, nullptr, &n); break;
      case MT_OP_MATMUL_REDUCE_INTO:
        s = matmul_impl(args[0], args[1], args[2], MT_REDUCE_INTO, nullptr, 0, nullptr, &n);
        break;
      case MT_OP_LINEAR_FWD:
        if (!args[0] || !args[1] || !args[3]) s = fail(MT_ERR_NULL, "x, w and y are required");
        break;
      case MT_OP_LINEAR_BWD:
        s = linear_bwd_impl(args[0], args[1], args[2], args[3], args[4], args[5], 0, nullptr, 0,
                            nullptr, &n);
        break;
      case MT_OP_REDUCE_BROADCAST_GRAD:
        s = reduce_impl(args[0], args[1], 0, nullptr, 0, nullptr, &n);
        break;
      case MT_OP_MSE_LOSS: s = mse_impl(args[0], args[1], nullptr, nullptr, nullptr, 0, nullptr, &n); break;
    }
    return s == MT_OK ? n : SIZE_MAX;
  } catch (...) {
    fail(MT_ERR_INVALID, "internal error");
    return SIZE_MAX;
  }
}

mt_status mt_conv2d_fwd(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b,
                        const mt_tensor* y, int32_t stride_h, int32_t stride_w, int32_t pad_h,
                        int32_t pad_w, void* ws, size_t ws_bytes, void* stream) {
  try {
    return conv_fwd_impl(x, w, b, y, stride_h, stride_w, pad_h, pad_w, ws, ws_bytes,
                         (hipStream_t)stream, nullptr);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_conv2d_fwd_workspace(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b,
                                  const mt_tensor* y, int32_t stride_h, int32_t stride_w,
                                  int32_t pad_h, int32_t pad_w, size_t* bytes) {
  try {
    if (!bytes) return fail(MT_ERR_NULL, "bytes is null");
    return conv_fwd_impl(x, w, b, y, stride_h, stride_w, pad_h, pad_w, nullptr, 0, nullptr, bytes);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_conv2d_bwd(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                        const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db,
                        int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                        uint32_t flags, void* ws, size_t ws_bytes, void* stream) {
  try {
    return conv_bwd_impl(x, w, dy, dx, dw, db, stride_h, stride_w, pad_h, pad_w, flags, ws,
                         ws_bytes, (hipStream_t)stream, nullptr);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_conv2d_bwd_workspace(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                                  const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db,
                                  int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                  size_t* bytes) {
  try {
    if (!bytes) return fail(MT_ERR_NULL, "bytes is null");
    return conv_bwd_impl(x, w, dy, dx, dw, db, stride_h, stride_w, pad_h, pad_w, 0, nullptr, 0,
                         nullptr, bytes);
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_broadcast_shape(int32_t na, const int64_t* a, int32_t nb, const int64_t* b,
                             int32_t* nout, int64_t* out) {
  try {
    if (!nout || !out) return fail(MT_ERR_NULL, "null output");
    std::string err;
    int n = 0;
    mt_status s = mt::broadcast_shapes(na, a, nb, b, &n, out, &err);
    if (s) return fail(s, err);
    *nout = n;
    return MT_OK;
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

mt_status mt_matmul_shape(int32_t na, const int64_t* a, int32_t nb, const int64_t* b,
                          int32_t* nout, int64_t* out) {
  try {
    if (!nout || !out || (na > 0 && !a) || (nb > 0 && !b)) return fail(MT_ERR_NULL, "null pointer");
    mt::MatmulPlan pl;
    std::string err;
    mt_status s = mt::plan_matmul_shapes(na, a, nullptr, nb, b, nullptr, &pl, &err);
    if (s) return fail(s, err);
    *nout = pl.nout;
    for (int i = 0; i < pl.nout; ++i) out[i] = pl.out[i];
    return MT_OK;
  } catch (...) {
    return fail(MT_ERR_INVALID, "internal error");
  }
}

const char* mt_status_str(mt_status s) {
  switch (s) {
    case MT_OK: return "ok";
    case MT_ERR_NULL: return "null pointer";
    case MT_ERR_NDIM: return "bad rank";
    case MT_ERR_SHAPE: return "shape mismatch";
    case MT_ERR_DTYPE: return "unsupported dtype";
    case MT_ERR_LAYOUT: return "unsupported layout";
    case MT_ERR_ALIAS: return "output overlaps input";
    case MT_ERR_WORKSPACE: return "bad workspace";
    case MT_ERR_HIP: return "HIP runtime error";
    case MT_ERR_INVALID: return "invalid argument";
  }
  return "unknown status";
}

const char* mt_last_error(void) { return g_err.c_str(); }

int mt_debug_set(const char* key, int64_t value) {
  if (!key) return -1;
  if (!std::strcmp(key, "cfg")) {
    if (value < -1 || value >= mt::kNumGemmCfg) return -2;
    g_force_cfg = (int)value;
  } else if (!std::strcmp(key, "vec1")) {
    if (value < 0 || value > 1) return -2;
    g_force_vec1 = (int)value;
  } else if (!std::strcmp(key, "krot")) {
    if (value < 0 || value > 1) return -2;
    g_krot = (int)value;
  } else if (!std::strcmp(key, "conv_gather")) {
    if (value < 0 || value > 1) return -2;
    g_conv_gather = (int)value;
  } else if (!std::strcmp(key, "stream_k")) {
    if (value < 0 || value > 2) return -2;
    g_stream_k = (int)value;
  } else if (!std::strcmp(key, "persist")) {
    if (value < 0 || value > 1) return -2;
    g_persist = (int)value;
  } else if (!std::strcmp(key, "phase_grid")) {
    if (value < 0 || value > 2) return -2;
    g_phase_grid = (int)value;
  } else if (!std::strcmp(key, "sk_blocks")) {
    if (value < 0 || value > 65535) return -2;
    g_sk_blocks = (int)value;
  } else if (!std::strcmp(key, "splits") || !std::strcmp(key, "parts")) {
    if (value < 0 || value > 4096) return -2;
    (key[0] == 's' ? g_force_splits : g_force_parts) = (int)value;
  } else {
    return -1;
  }
  return 0;
}

}  // extern "C"
