// Launch description shared by the host dispatch and the GEMM kernels.
//
// C[beta][m][n] (+)= sum_r sum_k A[beta, r][m][k] * B[beta, r][k][n] (+ bias[n])
//
// beta runs over the kept batch elements of the output, r over batch axes that
// are summed into the output (the gradient of a broadcast operand); both are
// decoded from flat indices with the per-dim sizes and element strides below.
// An operand is "K-contiguous" when its k index has stride 1, otherwise its
// m (for A) or n (for B) index has stride 1; `lda`/`ldb` is the stride of the
// other matrix index. C is row-major with row pitch `ldc`.
#pragma once
#include <cstdint>

namespace mt {

constexpr int kMaxBatchDims = 6;

// A convolution operand that the GEMM loads gather from the image instead of
// reading an unfolded matrix (MiniTensor Sec. 3.3 Eq. (6)): x is stored
// channels-last (c has stride 1), the unfolded columns run k = (u, v, c) with
// c fastest, and output pixel m = (n, i, j) reads input pixel
// (n, i sh - ph + u, j sw - pw + v), zero outside the image. Divisions by WO
// and HO use q = (m * mag) >> shift, exact for m < 2^31.
struct ConvGather {
  const float* x;
  uint32_t x_bytes;  // bytes from x that the loads may read (buffer bound)
  int32_t C, H, W, KW;
  int32_t sh, sw, ph, pw;
  int32_t HO, WO;
  int32_t xs0, xs2, xs3;  // element strides of x over n, h, w
  uint32_t wo_mag, ho_mag;
  int32_t wo_shift, ho_shift;
  // one sub-pixel phase of a strided input gradient (CONV 4): the phase's
  // taps are (u0 + su t, v0 + sv r) of the weight's KH x wKW; its rows, in
  // HO x WO order per image, are the dx pixels (h0 + sh i, w0 + sw j) of an
  // eH x eW image
  int32_t u0, v0, su, sv, wKW;
  int32_t eH, eW, h0, w0, esh, esw;
};

// The sub-pixel phases of one strided input gradient, launched as one grid:
// phase k owns blocks tile0[k] .. tile0[k+1]-1 (one tile each) and replaces
// these fields of the launch description (the rest is shared).
constexpr int kMaxConvPhases = 16;
struct ConvPhase {
  int64_t M, K;
  int32_t tiles_m;
  int32_t u0, v0, ph, pw, rows, cols, kw, h0, w0;
  uint32_t wo_mag, ho_mag;
  int32_t wo_shift, ho_shift;
};
struct ConvPhases {
  int32_t n;
  int32_t tile0[kMaxConvPhases + 1];
  ConvPhase ph[kMaxConvPhases];
};

struct GemmParams {
  const void* a;
  const void* b;
  float* c;
  const float* bias;  // nullable, length N, contiguous
  int64_t M, N, K;
  int64_t lda, ldb, ldc;
  // kept batch dims (output batch elements), outermost first
  int32_t nkeep;
  int32_t nred;
  int64_t keep_shape[kMaxBatchDims];
  int64_t keep_sa[kMaxBatchDims], keep_sb[kMaxBatchDims], keep_sc[kMaxBatchDims];
  // summed batch dims
  int64_t red_shape[kMaxBatchDims];
  int64_t red_sa[kMaxBatchDims], red_sb[kMaxBatchDims];
  int64_t keep_count;  // product of keep_shape (1 if none)
  int64_t red_count;   // product of red_shape (1 if none)
  int32_t tiles_m, tiles_n;
  int32_t accumulate;  // C += result
  int32_t group_m;     // tile-order group height (L2 reuse)
  // split-K: the sequence of K-stages (every summed batch index r times every
  // BK-wide k tile, r outermost) is cut into `splits` runs of
  // `stages_per_split` stages; run s writes its partial tile of batch
  // element beta to partial + s * partial_stride + beta * M * N (row-major,
  // pitch N), and a second pass adds the runs in order
  int32_t splits;
  int64_t stages_per_split;
  float* partial;
  int64_t partial_stride;
  // epilogue of the dense layer followed by a nonlinearity (no batch, no
  // split, no accumulation): z (nullable, row pitch ldz) receives the biased
  // product, C receives act(that) (act: an ActKind, 0 = none)
  float* z;
  int64_t ldz;
  int32_t act;
  // DMA kernel, plain products (no split, no summed batch axes): blocks on
  // XCD x start their K loop at stage x * KS / 8 and wrap around, so that the
  // eight XCDs stream different columns of the operands at any one time
  int32_t krot;
  // convolution kernels only: the gathered operand (A of the forward product,
  // B of the weight gradient); every other kernel ignores it
  ConvGather cg;
  // DMA kernels with an M-contiguous A (TN products), no batch: the column
  // sums of A over k, sum_k A[m][k], formed from the fragments the product
  // already reads (the dense layer's db = 1^T dY, with A = dY^T). Unsplit,
  // colsum[m] (+)= the sum (p.accumulate); split-K run s writes its sum to
  // colsum_part[s * M + m] and the host adds the runs in order. Null: off.
  float* colsum;
  float* colsum_part;
  // DMA kernels, plain products of whole 256x256 tiles (no batch, split,
  // activation or accumulation, M and N multiples of 256; column sums of A
  // allowed):
  // the size of a persistent grid (one block per CU, each walking the tiles
  // of the plain grid's blocks b, b + persist, ...); 0: the plain grid
  int32_t persist;
};

}  // namespace mt
