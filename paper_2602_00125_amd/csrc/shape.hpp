// Host-side shape bookkeeping (integer only, exact): the broadcasting rule of
// MiniTensor Sec. 3.1 applied to matmul batch dims, operand layouts, and the
// plans that fold broadcast-gradient sums into a product or a reduction.
#pragma once
#include <cstdint>
#include <string>

#include "../../include/minitensor_hip.h"
#include "gemm_params.hpp"
#include "kernels.hpp"

namespace mt {

// Broadcast of two shapes: right-aligned, each pair equal or one of them 1.
mt_status broadcast_shapes(int na, const int64_t* a, int nb, const int64_t* b, int* nout,
                           int64_t* out, std::string* err);

// One matrix operand after 1-D promotion: rows x cols with strides.
struct MatView {
  int64_t rows, cols;
  int64_t srow, scol;
};

// A broadcasting matmul resolved to batch dims and operand layouts.
struct MatmulPlan {
  int64_t M = 0, N = 0, K = 0;
  // batch dims of the result (broadcast of the operands' batch dims), with
  // each operand's element stride along them (0 where it is broadcast)
  int nbatch = 0;
  int64_t batch[MT_MAX_DIMS] = {0};
  int64_t sa[MT_MAX_DIMS] = {0}, sb[MT_MAX_DIMS] = {0};
  MatView a{}, b{};   // A: M x K, B: K x N (strides in elements)
  int nout = 0;       // result rank and shape
  int64_t out[MT_MAX_DIMS] = {0};
  bool a_vec_dims = true, b_vec_dims = true;  // 1-D promotions drop a result dim
};

mt_status plan_matmul_shapes(int na, const int64_t* ashape, const int64_t* astride, int nb,
                             const int64_t* bshape, const int64_t* bstride, MatmulPlan* p,
                             std::string* err);

// Operand layout of an M x K (is_a) or K x N matrix for the GEMM kernels:
// kc = contraction index contiguous; ld = stride of the other index.
// Returns false when neither matrix dim is contiguous.
bool operand_layout(const MatView& v, bool is_a, bool* kc, int64_t* ld);

// Reduction plan of a strided tensor onto `in_shape` (left-padded with ones,
// dims equal or 1). Size-1 dims are dropped, adjacent dims merged where the
// strides allow.
mt_status plan_reduce(int nout, const int64_t* oshape, const int64_t* ostride, int nin,
                      const int64_t* ishape, ReducePlan* plan, std::string* err);

// Bytes spanned by a strided view (0 for an empty one); negative strides are
// rejected by the caller.
int64_t span_elems(int n, const int64_t* shape, const int64_t* stride);

}  // namespace mt
