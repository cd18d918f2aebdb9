// Host-side shape bookkeeping for libminitensor_hip (integer only).
#include "shape.hpp"

#include <cstdio>

namespace mt {

static std::string dims_str(int n, const int64_t* d) {
  std::string s = "[";
  for (int i = 0; i < n; ++i) {
    if (i) s += ", ";
    s += std::to_string(d[i]);
  }
  return s + "]";
}

mt_status broadcast_shapes(int na, const int64_t* a, int nb, const int64_t* b, int* nout,
                           int64_t* out, std::string* err) {
  if (na < 0 || nb < 0 || na > MT_MAX_DIMS || nb > MT_MAX_DIMS) {
    if (err) *err = "rank outside 0.." + std::to_string(MT_MAX_DIMS);
    return MT_ERR_NDIM;
  }
  if ((na && !a) || (nb && !b)) {
    if (err) *err = "null shape array";
    return MT_ERR_NULL;
  }
  const int n = na > nb ? na : nb;
  int64_t tmp[MT_MAX_DIMS];
  for (int i = 0; i < n; ++i) {
    const int64_t x = i < na ? a[na - 1 - i] : 1;
    const int64_t y = i < nb ? b[nb - 1 - i] : 1;
    if (x < 0 || y < 0) {
      if (err) *err = "negative size";
      return MT_ERR_SHAPE;
    }
    if (x != y && x != 1 && y != 1) {
      if (err)
        *err = "shapes " + dims_str(na, a) + " and " + dims_str(nb, b) + " do not broadcast";
      return MT_ERR_SHAPE;
    }
    tmp[n - 1 - i] = (x == 1) ? y : x;
  }
  for (int i = 0; i < n; ++i) out[i] = tmp[i];
  *nout = n;
  return MT_OK;
}

mt_status plan_matmul_shapes(int na, const int64_t* ashape, const int64_t* astride, int nb,
                             const int64_t* bshape, const int64_t* bstride, MatmulPlan* p,
                             std::string* err) {
  if (na < 1 || nb < 1 || na > MT_MAX_DIMS || nb > MT_MAX_DIMS) {
    if (err) *err = "matmul operands need rank 1.." + std::to_string(MT_MAX_DIMS);
    return MT_ERR_NDIM;
  }
  for (int i = 0; i < na; ++i)
    if (ashape[i] < 0) { if (err) *err = "negative size"; return MT_ERR_SHAPE; }
  for (int i = 0; i < nb; ++i)
    if (bshape[i] < 0) { if (err) *err = "negative size"; return MT_ERR_SHAPE; }
  // promote 1-D operands: a [K] -> [1, K]; b [K] -> [K, 1]
  if (na == 1) {
    p->a = MatView{1, ashape[0], ashape[0] * (astride ? astride[0] : 1), astride ? astride[0] : 1};
    p->a_vec_dims = false;
  } else {
    p->a = MatView{ashape[na - 2], ashape[na - 1], astride ? astride[na - 2] : ashape[na - 1],
                   astride ? astride[na - 1] : 1};
  }
  if (nb == 1) {
    p->b = MatView{bshape[0], 1, bstride ? bstride[0] : 1, 1};
    p->b_vec_dims = false;
  } else {
    p->b = MatView{bshape[nb - 2], bshape[nb - 1], bstride ? bstride[nb - 2] : bshape[nb - 1],
                   bstride ? bstride[nb - 1] : 1};
  }
  p->M = p->a.rows;
  p->K = p->a.cols;
  if (p->b.rows != p->K) {
    if (err)
      *err = "matmul contraction mismatch: " + dims_str(na, ashape) + " @ " + dims_str(nb, bshape);
    return MT_ERR_SHAPE;
  }
  p->N = p->b.cols;
  const int ba = na > 2 ? na - 2 : 0, bb = nb > 2 ? nb - 2 : 0;
  std::string e;
  mt_status st = broadcast_shapes(ba, ashape, bb, bshape, &p->nbatch, p->batch, &e);
  if (st != MT_OK) {
    if (err) *err = "matmul batch dims: " + e;
    return st;
  }
  for (int i = 0; i < p->nbatch; ++i) {
    const int ia = i - (p->nbatch - ba), ib = i - (p->nbatch - bb);
    const int64_t da = ia >= 0 ? ashape[ia] : 1, db = ib >= 0 ? bshape[ib] : 1;
    p->sa[i] = (ia >= 0 && da != 1) ? (astride ? astride[ia] : 0) : 0;
    p->sb[i] = (ib >= 0 && db != 1) ? (bstride ? bstride[ib] : 0) : 0;
  }
  int n = 0;
  for (int i = 0; i < p->nbatch; ++i) p->out[n++] = p->batch[i];
  if (na != 1) p->out[n++] = p->M;
  if (nb != 1) p->out[n++] = p->N;
  p->nout = n;
  return MT_OK;
}

bool operand_layout(const MatView& v, bool is_a, bool* kc, int64_t* ld) {
  // A: rows = m, cols = k.  B: rows = k, cols = n.
  const bool row_major = v.scol == 1 || v.cols <= 1;
  const bool col_major = v.srow == 1 || v.rows <= 1;
  // prefer the layout whose contiguous index has extent > 1
  bool use_row;
  if (row_major && col_major) use_row = v.cols >= v.rows;
  else if (row_major) use_row = true;
  else if (col_major) use_row = false;
  else return false;
  if (use_row) {
    // contiguous along cols: A -> k contiguous (kc); B -> n contiguous
    *kc = is_a;
    *ld = v.rows <= 1 ? (v.cols > 0 ? v.cols : 1) : v.srow;
  } else {
    *kc = !is_a;
    *ld = v.cols <= 1 ? (v.rows > 0 ? v.rows : 1) : v.scol;
  }
  return true;
}

int64_t span_elems(int n, const int64_t* shape, const int64_t* stride) {
  int64_t hi = 0;
  for (int i = 0; i < n; ++i) {
    if (shape[i] == 0) return 0;
    hi += (shape[i] - 1) * stride[i];
  }
  return hi + 1;
}

mt_status plan_reduce(int nout, const int64_t* oshape, const int64_t* ostride, int nin,
                      const int64_t* ishape, ReducePlan* plan, std::string* err) {
  if (nout < 0 || nout > MT_MAX_DIMS || nin < 0 || nin > nout) {
    if (err) *err = "grad_in rank must be <= grad_out rank <= " + std::to_string(MT_MAX_DIMS);
    return MT_ERR_NDIM;
  }
  const int pad = nout - nin;
  // collect kept / reduced dims (size-1 output dims carry nothing)
  int64_t ks[MT_MAX_DIMS], kst[MT_MAX_DIMS], rs[MT_MAX_DIMS], rst[MT_MAX_DIMS];
  int nk = 0, nr = 0;
  int64_t kc = 1, rc = 1;
  for (int d = 0; d < nout; ++d) {
    const int64_t in = d < pad ? 1 : ishape[d - pad];
    if (in != oshape[d] && in != 1) {
      if (err)
        *err = "grad_in " + dims_str(nin, ishape) + " is not a broadcast source of grad_out " +
               dims_str(nout, oshape);
      return MT_ERR_SHAPE;
    }
    if (oshape[d] == 1) continue;
    if (in == 1) {
      rs[nr] = oshape[d];
      rst[nr++] = ostride[d];
      rc *= oshape[d];
    } else {
      ks[nk] = oshape[d];
      kst[nk++] = ostride[d];
      kc *= oshape[d];
    }
  }
  // merge adjacent dims that walk memory as one
  auto merge = [](int64_t* s, int64_t* st, int& n) {
    int w = 0;
    for (int i = 0; i < n; ++i) {
      if (w > 0 && st[w - 1] == s[i] * st[i]) {
        s[w - 1] *= s[i];
        st[w - 1] = st[i];
      } else {
        s[w] = s[i];
        st[w] = st[i];
        ++w;
      }
    }
    n = w;
  };
  merge(ks, kst, nk);
  merge(rs, rst, nr);
  plan->nkeep = nk;
  plan->nred = nr;
  for (int i = 0; i < nk; ++i) { plan->keep_shape[i] = ks[i]; plan->keep_stride[i] = kst[i]; }
  for (int i = 0; i < nr; ++i) { plan->red_shape[i] = rs[i]; plan->red_stride[i] = rst[i]; }
  plan->keep_count = kc;
  plan->red_count = rc;
  for (int d = 0; d < nout; ++d)
    if (oshape[d] == 0) { plan->keep_count = 0; plan->red_count = 0; }
  // an empty grad_out sums nothing: every grad_in element is 0
  if (plan->red_count == 0) {
    int64_t cnt = 1;
    for (int d = 0; d < nin; ++d) cnt *= ishape[d];
    plan->keep_count = cnt;
    plan->nkeep = 0;
    plan->nred = 0;
  }
  return MT_OK;
}

}  // namespace mt
