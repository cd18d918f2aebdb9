// Plain, slow fp64 CPU oracle for the dense layer and broadcasting matmul.
//
// TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the bench's
// CPU-baseline leg may load this library. The GPU library never includes,
// links or calls anything from here, and this file shares no code with it
// (its broadcast-shape logic is its own as well).
//
// What it computes (MiniTensor paper):
//   * Sec. 3.1, Eq. (1):     Y = X W^T                          (matmul)
//   * Sec. 3.3, Eq. (5):     Dense(x; W, b) = x W^T + 1 b^T      (linear)
//   * Sec. 3.2, Eq. (4):     Xbar += Ybar W,  Wbar += Ybar^T X   (pullbacks)
//   * Sec. 3.3, Eq. (6):     2-D convolution with stride and zero padding,
//                            and its pullbacks to the input, weights, bias
//   * Sec. 3.2, add pullback: xbar += zbar, ybar += zbar; with the
//     broadcasting rule of Sec. 3.1 this gives db = 1^T dY and, for
//     broadcast batch axes, a sum of the gradient over those axes.
//   * Sec. 3.1 broadcasting: shapes are aligned after left-padding with
//     singleton dims; a dim of size one is virtually expanded.
//
// Every value is accumulated in fp64 in ascending order of the summed index
// (for broadcast gradients: ascending flat index of the output batch, then
// the contraction index). Next to every output element the oracle returns
// S = sum |a_i * b_i| over exactly the products (and added terms) that the
// element sums; parity tolerances are stated relative to S.
//
// Parallelism is over output rows only (OpenMP), so every element's
// summation order is independent of the thread count: results are
// deterministic.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <vector>

namespace {

constexpr int kMaxDims = 8;

// Error codes returned by the shape helpers (0 = ok).
enum { OR_OK = 0, OR_ERR_NDIM = 1, OR_ERR_SHAPE = 2 };

// Broadcasting (Sec. 3.1): align the two shapes on the right, pad the shorter
// one with leading ones; each aligned pair must be equal or contain a 1.
int broadcast_dims(int na, const int64_t* a, int nb, const int64_t* b, int* nout, int64_t* out) {
  if (na < 0 || nb < 0 || na > kMaxDims || nb > kMaxDims) return OR_ERR_NDIM;
  int n = na > nb ? na : nb;
  for (int i = 0; i < n; ++i) {
    // i counts from the right
    int64_t da = (i < na) ? a[na - 1 - i] : 1;
    int64_t db = (i < nb) ? b[nb - 1 - i] : 1;
    if (da < 0 || db < 0) return OR_ERR_SHAPE;
    int64_t d;
    if (da == db) d = da;
    else if (da == 1) d = db;
    else if (db == 1) d = da;
    else return OR_ERR_SHAPE;
    out[n - 1 - i] = d;
  }
  *nout = n;
  return OR_OK;
}

int64_t prod(const int64_t* s, int n) {
  int64_t p = 1;
  for (int i = 0; i < n; ++i) p *= s[i];
  return p;
}

// matmul operands promoted to >= 2-D (a 1-D left operand gets a leading 1,
// a 1-D right operand a trailing 1), their batch shape broadcast.
struct MatmulPlan {
  int nbatch = 0;
  int64_t batch[kMaxDims] = {0};
  // per operand: batch dims left-padded to nbatch (size-1 dims stay 1)
  int64_t abatch[kMaxDims] = {0}, bbatch[kMaxDims] = {0};
  int64_t M = 0, K = 0, N = 0;
  int nout = 0;
  int64_t out[kMaxDims] = {0};
};

int plan_matmul(int na, const int64_t* a, int nb, const int64_t* b, MatmulPlan* p) {
  if (na < 1 || nb < 1 || na > kMaxDims || nb > kMaxDims) return OR_ERR_NDIM;
  for (int i = 0; i < na; ++i) if (a[i] < 0) return OR_ERR_SHAPE;
  for (int i = 0; i < nb; ++i) if (b[i] < 0) return OR_ERR_SHAPE;
  int64_t pa[kMaxDims + 1] = {0}, pb[kMaxDims + 1] = {0};
  int npa = 0, npb = 0;
  if (na == 1) { pa[0] = 1; pa[1] = a[0]; npa = 2; }
  else { for (int i = 0; i < na; ++i) pa[i] = a[i]; npa = na; }
  if (nb == 1) { pb[0] = b[0]; pb[1] = 1; npb = 2; }
  else { for (int i = 0; i < nb; ++i) pb[i] = b[i]; npb = nb; }
  p->M = pa[npa - 2];
  p->K = pa[npa - 1];
  if (pb[npb - 2] != p->K) return OR_ERR_SHAPE;
  p->N = pb[npb - 1];
  int r = broadcast_dims(npa - 2, pa, npb - 2, pb, &p->nbatch, p->batch);
  if (r) return r;
  for (int i = 0; i < p->nbatch; ++i) {
    int ia = i - (p->nbatch - (npa - 2));
    int ib = i - (p->nbatch - (npb - 2));
    p->abatch[i] = ia >= 0 ? pa[ia] : 1;
    p->bbatch[i] = ib >= 0 ? pb[ib] : 1;
  }
  // output shape: batch, then M unless A was 1-D, then N unless B was 1-D
  int n = 0;
  for (int i = 0; i < p->nbatch; ++i) p->out[n++] = p->batch[i];
  if (na != 1) p->out[n++] = p->M;
  if (nb != 1) p->out[n++] = p->N;
  if (n > kMaxDims) return OR_ERR_NDIM;
  p->nout = n;
  return OR_OK;
}

// Flat batch index of an operand for output batch multi-index `idx`: a
// broadcast (size-1) dim always reads index 0.
int64_t operand_batch_offset(const MatmulPlan& p, const int64_t* opbatch, const int64_t* idx) {
  int64_t off = 0;
  for (int i = 0; i < p.nbatch; ++i) off = off * opbatch[i] + (opbatch[i] == 1 ? 0 : idx[i]);
  return off;
}

void unflatten(int64_t flat, int n, const int64_t* shape, int64_t* idx) {
  for (int i = n - 1; i >= 0; --i) {
    idx[i] = shape[i] ? flat % shape[i] : 0;
    flat = shape[i] ? flat / shape[i] : 0;
  }
}

}  // namespace

namespace {

// ------------------------------------------------------------ convolution
//
// Sec. 3.3 Eq. (6), 2-D convolution with stride (sh, sw) and zero padding
// (ph, pw), batched over n, all indices 0-based, tensors in NCHW order:
//   y[n][c][i][j] = sum_{c'} sum_{u} sum_{v} w[c][c'][u][v] x[n][c'][i sh + u - ph][j sw + v - pw]
//                   (+ b[c]), x read as 0 outside the image;
//   Ho = (H + 2 ph - KH) / sh + 1, Wo = (W + 2 pw - KW) / sw + 1.
// Pullbacks (the matmul pullbacks of Eq. (4) through the linear map of
// Eq. (6)): each term w x of some y is charged to both factors,
//   dx[n][c'][h][x]  = sum over (c, u, v) with h = i sh + u - ph, x = j sw + v - pw
//                      of dy[n][c][i][j] w[c][c'][u][v],
//   dw[c][c'][u][v]  = sum over (n, i, j) of dy[n][c][i][j] x[n][c'][i sh + u - ph][j sw + v - pw],
//   db[c]            = sum over (n, i, j) of dy[n][c][i][j].
// Each element is one fp64 sum in the order of the indices as written
// (outermost first), with S = sum of |term| beside it.

struct ConvDims {
  int64_t N, C, H, W, CO, KH, KW, sh, sw, ph, pw, HO, WO;
};

ConvDims conv_dims(const int64_t* d) {
  ConvDims c;
  c.N = d[0]; c.C = d[1]; c.H = d[2]; c.W = d[3]; c.CO = d[4]; c.KH = d[5]; c.KW = d[6];
  c.sh = d[7]; c.sw = d[8]; c.ph = d[9]; c.pw = d[10];
  c.HO = (c.H + 2 * c.ph - c.KH) / c.sh + 1;
  c.WO = (c.W + 2 * c.pw - c.KW) / c.sw + 1;
  return c;
}

void conv_y_elem(const ConvDims& c, const double* x, const double* w, const double* b,
                 int64_t n, int64_t co, int64_t i, int64_t j, double* out, double* S) {
  double acc = 0.0, s = 0.0;
  for (int64_t ci = 0; ci < c.C; ++ci)
    for (int64_t u = 0; u < c.KH; ++u)
      for (int64_t v = 0; v < c.KW; ++v) {
        const int64_t h = i * c.sh + u - c.ph, xx = j * c.sw + v - c.pw;
        if (h < 0 || h >= c.H || xx < 0 || xx >= c.W) continue;
        const double p = w[((co * c.C + ci) * c.KH + u) * c.KW + v] *
                         x[((n * c.C + ci) * c.H + h) * c.W + xx];
        acc += p;
        s += std::fabs(p);
      }
  if (b) {
    acc += b[co];
    s += std::fabs(b[co]);
  }
  *out = acc;
  *S = s;
}

void conv_dx_elem(const ConvDims& c, const double* dy, const double* w, int64_t n, int64_t ci,
                  int64_t h, int64_t xx, double* out, double* S) {
  double acc = 0.0, s = 0.0;
  for (int64_t co = 0; co < c.CO; ++co)
    for (int64_t u = 0; u < c.KH; ++u)
      for (int64_t v = 0; v < c.KW; ++v) {
        const int64_t ti = h + c.ph - u, tj = xx + c.pw - v;   // = i sh, j sw
        if (ti < 0 || tj < 0 || ti % c.sh || tj % c.sw) continue;
        const int64_t i = ti / c.sh, j = tj / c.sw;
        if (i >= c.HO || j >= c.WO) continue;
        const double p = dy[((n * c.CO + co) * c.HO + i) * c.WO + j] *
                         w[((co * c.C + ci) * c.KH + u) * c.KW + v];
        acc += p;
        s += std::fabs(p);
      }
  *out = acc;
  *S = s;
}

void conv_dw_elem(const ConvDims& c, const double* dy, const double* x, int64_t co, int64_t ci,
                  int64_t u, int64_t v, double* out, double* S) {
  double acc = 0.0, s = 0.0;
  for (int64_t n = 0; n < c.N; ++n)
    for (int64_t i = 0; i < c.HO; ++i)
      for (int64_t j = 0; j < c.WO; ++j) {
        const int64_t h = i * c.sh + u - c.ph, xx = j * c.sw + v - c.pw;
        if (h < 0 || h >= c.H || xx < 0 || xx >= c.W) continue;
        const double p = dy[((n * c.CO + co) * c.HO + i) * c.WO + j] *
                         x[((n * c.C + ci) * c.H + h) * c.W + xx];
        acc += p;
        s += std::fabs(p);
      }
  *out = acc;
  *S = s;
}

void unflat4(int64_t f, int64_t d1, int64_t d2, int64_t d3, int64_t* a, int64_t* b_, int64_t* c_,
             int64_t* e) {
  *e = f % d3;
  f /= d3;
  *c_ = f % d2;
  f /= d2;
  *b_ = f % d1;
  *a = f / d1;
}

}  // namespace

extern "C" {

// ---------------------------------------------------------------- shapes --

// Sec. 3.1 broadcasting rule. Returns 0, or 1 (bad rank) / 2 (incompatible).
int or_broadcast_shape(int na, const int64_t* a, int nb, const int64_t* b, int* nout, int64_t* out) {
  return broadcast_dims(na, a, nb, b, nout, out);
}

// Output shape of a broadcasting matmul (Eq. (1) batched per Sec. 3.1).
int or_matmul_shape(int na, const int64_t* a, int nb, const int64_t* b, int* nout, int64_t* out) {
  MatmulPlan p;
  int r = plan_matmul(na, a, nb, b, &p);
  if (r) return r;
  *nout = p.nout;
  for (int i = 0; i < p.nout; ++i) out[i] = p.out[i];
  return OR_OK;
}

// ---------------------------------------------------------------- linear --

// Eq. (5): Y[m,n] = sum_k X[m,k] W[n,k] + b[n]; b may be null (Eq. (1)).
// X[M,K], W[N,K], b[N], Y[M,N], S[M,N]; all row-major fp64.
void or_linear_fwd(int64_t M, int64_t N, int64_t K, const double* X, const double* W,
                   const double* b, double* Y, double* S) {
#pragma omp parallel for schedule(static)
  for (int64_t m = 0; m < M; ++m) {
    for (int64_t n = 0; n < N; ++n) {
      double acc = 0.0, s = 0.0;
      for (int64_t k = 0; k < K; ++k) {
        double p = X[m * K + k] * W[n * K + k];
        acc += p;
        s += std::fabs(p);
      }
      if (b) {
        acc += b[n];
        s += std::fabs(b[n]);
      }
      Y[m * N + n] = acc;
      S[m * N + n] = s;
    }
  }
}

// Eq. (4), first pullback: dX[m,k] = sum_n dY[m,n] W[n,k].
void or_linear_bwd_dx(int64_t M, int64_t N, int64_t K, const double* dY, const double* W,
                      double* dX, double* S) {
#pragma omp parallel for schedule(static)
  for (int64_t m = 0; m < M; ++m) {
    double* acc = dX + m * K;
    double* s = S + m * K;
    for (int64_t k = 0; k < K; ++k) { acc[k] = 0.0; s[k] = 0.0; }
    // n ascending for every (m,k); the k loop only walks independent outputs
    for (int64_t n = 0; n < N; ++n) {
      double g = dY[m * N + n];
      for (int64_t k = 0; k < K; ++k) {
        double p = g * W[n * K + k];
        acc[k] += p;
        s[k] += std::fabs(p);
      }
    }
  }
}

// Eq. (4), second pullback: dW[n,k] = sum_m dY[m,n] X[m,k].
void or_linear_bwd_dw(int64_t M, int64_t N, int64_t K, const double* dY, const double* X,
                      double* dW, double* S) {
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    double* acc = dW + n * K;
    double* s = S + n * K;
    for (int64_t k = 0; k < K; ++k) { acc[k] = 0.0; s[k] = 0.0; }
    for (int64_t m = 0; m < M; ++m) {
      double g = dY[m * N + n];
      for (int64_t k = 0; k < K; ++k) {
        double p = g * X[m * K + k];
        acc[k] += p;
        s[k] += std::fabs(p);
      }
    }
  }
}

// Add pullback (Sec. 3.2) through the broadcast bias (Sec. 3.1):
// db[n] = sum_m dY[m,n], S[n] = sum_m |dY[m,n]|.
void or_linear_bwd_db(int64_t M, int64_t N, const double* dY, double* db, double* S) {
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    double acc = 0.0, s = 0.0;
    for (int64_t m = 0; m < M; ++m) {
      acc += dY[m * N + n];
      s += std::fabs(dY[m * N + n]);
    }
    db[n] = acc;
    S[n] = s;
  }
}

// Sampled forms: the same sums for P given output positions (r[i], c[i]).
// Y at (m, n); dX at (m, k); dW at (n, k).
void or_linear_fwd_at(int64_t M, int64_t N, int64_t K, const double* X, const double* W,
                      const double* b, int64_t P, const int64_t* r, const int64_t* c,
                      double* out, double* S) {
  (void)M;
  (void)N;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < P; ++i) {
    int64_t m = r[i], n = c[i];
    double acc = 0.0, s = 0.0;
    for (int64_t k = 0; k < K; ++k) {
      double p = X[m * K + k] * W[n * K + k];
      acc += p;
      s += std::fabs(p);
    }
    if (b) {
      acc += b[n];
      s += std::fabs(b[n]);
    }
    out[i] = acc;
    S[i] = s;
  }
}

void or_linear_bwd_dx_at(int64_t M, int64_t N, int64_t K, const double* dY, const double* W,
                         int64_t P, const int64_t* r, const int64_t* c, double* out, double* S) {
  (void)M;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < P; ++i) {
    int64_t m = r[i], k = c[i];
    double acc = 0.0, s = 0.0;
    for (int64_t n = 0; n < N; ++n) {
      double p = dY[m * N + n] * W[n * K + k];
      acc += p;
      s += std::fabs(p);
    }
    out[i] = acc;
    S[i] = s;
  }
}

void or_linear_bwd_dw_at(int64_t M, int64_t N, int64_t K, const double* dY, const double* X,
                         int64_t P, const int64_t* r, const int64_t* c, double* out, double* S) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < P; ++i) {
    int64_t n = r[i], k = c[i];
    double acc = 0.0, s = 0.0;
    for (int64_t m = 0; m < M; ++m) {
      double p = dY[m * N + n] * X[m * K + k];
      acc += p;
      s += std::fabs(p);
    }
    out[i] = acc;
    S[i] = s;
  }
}

// ------------------------------------------------- broadcasting matmul --

// Eq. (1) per batch element with the Sec. 3.1 broadcasting of batch dims:
// C[beta, m, n] = sum_k A[beta_A, m, k] B[beta_B, k, n], where beta_A and
// beta_B read index 0 along their size-1 (broadcast) dims. Operands are
// contiguous row-major of the given shapes (1-D operands promoted as in
// NumPy/PyTorch matmul). C and S have the matmul output shape.
int or_matmul(int na, const int64_t* ashape, const double* A, int nb, const int64_t* bshape,
              const double* B, double* C, double* S) {
  MatmulPlan p;
  int r = plan_matmul(na, ashape, nb, bshape, &p);
  if (r) return r;
  const int64_t nbatch = prod(p.batch, p.nbatch);
  const int64_t M = p.M, N = p.N, K = p.K;
  const int64_t rows = nbatch * M;
#pragma omp parallel for schedule(static)
  for (int64_t row = 0; row < rows; ++row) {
    int64_t bi = row / (M ? M : 1), m = row % (M ? M : 1);
    int64_t idx[kMaxDims];
    unflatten(bi, p.nbatch, p.batch, idx);
    const double* a = A + operand_batch_offset(p, p.abatch, idx) * M * K;
    const double* bb = B + operand_batch_offset(p, p.bbatch, idx) * K * N;
    double* acc = C + (bi * M + m) * N;
    double* s = S + (bi * M + m) * N;
    for (int64_t n = 0; n < N; ++n) { acc[n] = 0.0; s[n] = 0.0; }
    // k ascending for every (m, n); the n loop only walks independent outputs
    for (int64_t k = 0; k < K; ++k) {
      double av = a[m * K + k];
      for (int64_t n = 0; n < N; ++n) {
        double prd = av * bb[k * N + n];
        acc[n] += prd;
        s[n] += std::fabs(prd);
      }
    }
  }
  return OR_OK;
}

// Pullbacks of the broadcasting matmul: Eq. (4) per batch element, then the
// add pullback summed over every output batch element that reads the same
// operand batch (Sec. 3.1 broadcasting, Sec. 3.2):
//   dA[alpha, m, k] = sum_{beta -> alpha} sum_n dC[beta, m, n] B[beta_B, k, n]
//   dB[alpha, k, n] = sum_{beta -> alpha} sum_m A[beta_A, m, k] dC[beta, m, n]
// dA has A's shape, dB has B's shape; either may be null to skip it.
int or_matmul_bwd(int na, const int64_t* ashape, const double* A, int nb, const int64_t* bshape,
                  const double* B, const double* dC, double* dA, double* SA, double* dB,
                  double* SB) {
  MatmulPlan p;
  int r = plan_matmul(na, ashape, nb, bshape, &p);
  if (r) return r;
  const int64_t nbatch = prod(p.batch, p.nbatch);
  const int64_t nabatch = prod(p.abatch, p.nbatch);
  const int64_t nbbatch = prod(p.bbatch, p.nbatch);
  const int64_t M = p.M, N = p.N, K = p.K;
  // map every output batch to its operand batches
  std::vector<int64_t> amap(nbatch), bmap(nbatch);
  for (int64_t bi = 0; bi < nbatch; ++bi) {
    int64_t idx[kMaxDims];
    unflatten(bi, p.nbatch, p.batch, idx);
    amap[bi] = operand_batch_offset(p, p.abatch, idx);
    bmap[bi] = operand_batch_offset(p, p.bbatch, idx);
  }
  if (dA) {
#pragma omp parallel for schedule(static)
    for (int64_t row = 0; row < nabatch * M; ++row) {
      int64_t ai = row / (M ? M : 1), m = row % (M ? M : 1);
      for (int64_t k = 0; k < K; ++k) {
        double acc = 0.0, s = 0.0;
        for (int64_t bi = 0; bi < nbatch; ++bi) {
          if (amap[bi] != ai) continue;
          const double* g = dC + (bi * M + m) * N;
          const double* bb = B + bmap[bi] * K * N + k * N;
          for (int64_t n = 0; n < N; ++n) {
            double prd = g[n] * bb[n];
            acc += prd;
            s += std::fabs(prd);
          }
        }
        dA[(ai * M + m) * K + k] = acc;
        SA[(ai * M + m) * K + k] = s;
      }
    }
  }
  if (dB) {
#pragma omp parallel for schedule(static)
    for (int64_t row = 0; row < nbbatch * K; ++row) {
      int64_t bj = row / (K ? K : 1), k = row % (K ? K : 1);
      double* acc = dB + (bj * K + k) * N;
      double* s = SB + (bj * K + k) * N;
      for (int64_t n = 0; n < N; ++n) { acc[n] = 0.0; s[n] = 0.0; }
      // per (k, n): output batches ascending, then m ascending
      for (int64_t bi = 0; bi < nbatch; ++bi) {
        if (bmap[bi] != bj) continue;
        const double* a = A + amap[bi] * M * K;
        const double* g = dC + bi * M * N;
        for (int64_t m = 0; m < M; ++m) {
          double av = a[m * K + k];
          for (int64_t n = 0; n < N; ++n) {
            double prd = av * g[m * N + n];
            acc[n] += prd;
            s[n] += std::fabs(prd);
          }
        }
      }
    }
  }
  return OR_OK;
}

// Gradient of a broadcast (Sec. 3.1 + add pullback of Sec. 3.2):
// g_in[alpha] = sum over every g_out element whose index maps to alpha,
// where g_in's shape, left-padded with ones, is g_out's shape with some dims
// set to 1. Leading padded dims are summed away; size-1 dims of g_in are
// summed and kept. Ascending flat order of g_out. S = sum |g_out| per output.
int or_reduce_broadcast(int nout_dims, const int64_t* oshape, const double* gout, int nin_dims,
                        const int64_t* ishape, double* gin, double* S) {
  if (nout_dims < 0 || nout_dims > kMaxDims || nin_dims < 0 || nin_dims > nout_dims)
    return OR_ERR_NDIM;
  int64_t pin[kMaxDims];
  int pad = nout_dims - nin_dims;
  for (int i = 0; i < nout_dims; ++i) {
    pin[i] = i < pad ? 1 : ishape[i - pad];
    if (pin[i] != oshape[i] && pin[i] != 1) return OR_ERR_SHAPE;
  }
  const int64_t nin = prod(pin, nout_dims);
  const int64_t nall = prod(oshape, nout_dims);
  for (int64_t j = 0; j < nin; ++j) { gin[j] = 0.0; S[j] = 0.0; }
  // one sequential walk over g_out in ascending flat order
  int64_t idx[kMaxDims];
  for (int64_t f = 0; f < nall; ++f) {
    unflatten(f, nout_dims, oshape, idx);
    int64_t j = 0;
    for (int d = 0; d < nout_dims; ++d) j = j * pin[d] + (pin[d] == 1 ? 0 : idx[d]);
    gin[j] += gout[f];
    S[j] += std::fabs(gout[f]);
  }
  return OR_OK;
}


// dims = {N, C, H, W, CO, KH, KW, sh, sw, ph, pw}; every tensor NCHW-contiguous fp64.
void or_conv2d_fwd(const int64_t* dims, const double* x, const double* w, const double* b,
                   double* y, double* S) {
  const ConvDims c = conv_dims(dims);
  const int64_t rows = c.N * c.CO;
#pragma omp parallel for schedule(dynamic)
  for (int64_t r = 0; r < rows; ++r) {
    const int64_t n = r / c.CO, co = r % c.CO;
    for (int64_t i = 0; i < c.HO; ++i)
      for (int64_t j = 0; j < c.WO; ++j) {
        const int64_t f = ((n * c.CO + co) * c.HO + i) * c.WO + j;
        conv_y_elem(c, x, w, b, n, co, i, j, &y[f], &S[f]);
      }
  }
}

void or_conv2d_bwd_dx(const int64_t* dims, const double* dy, const double* w, double* dx,
                      double* S) {
  const ConvDims c = conv_dims(dims);
  const int64_t rows = c.N * c.C;
#pragma omp parallel for schedule(dynamic)
  for (int64_t r = 0; r < rows; ++r) {
    const int64_t n = r / c.C, ci = r % c.C;
    for (int64_t h = 0; h < c.H; ++h)
      for (int64_t xx = 0; xx < c.W; ++xx) {
        const int64_t f = ((n * c.C + ci) * c.H + h) * c.W + xx;
        conv_dx_elem(c, dy, w, n, ci, h, xx, &dx[f], &S[f]);
      }
  }
}

void or_conv2d_bwd_dw(const int64_t* dims, const double* dy, const double* x, double* dw,
                      double* S) {
  const ConvDims c = conv_dims(dims);
  const int64_t rows = c.CO * c.C;
#pragma omp parallel for schedule(dynamic)
  for (int64_t r = 0; r < rows; ++r) {
    const int64_t co = r / c.C, ci = r % c.C;
    for (int64_t u = 0; u < c.KH; ++u)
      for (int64_t v = 0; v < c.KW; ++v) {
        const int64_t f = ((co * c.C + ci) * c.KH + u) * c.KW + v;
        conv_dw_elem(c, dy, x, co, ci, u, v, &dw[f], &S[f]);
      }
  }
}

void or_conv2d_bwd_db(const int64_t* dims, const double* dy, double* db, double* S) {
  const ConvDims c = conv_dims(dims);
  for (int64_t co = 0; co < c.CO; ++co) {
    double acc = 0.0, s = 0.0;
    for (int64_t n = 0; n < c.N; ++n)
      for (int64_t i = 0; i < c.HO; ++i)
        for (int64_t j = 0; j < c.WO; ++j) {
          const double g = dy[((n * c.CO + co) * c.HO + i) * c.WO + j];
          acc += g;
          s += std::fabs(g);
        }
    db[co] = acc;
    S[co] = s;
  }
}

// Sampled elements: flat NCHW indices into y / dx / dw.
void or_conv2d_fwd_at(const int64_t* dims, const double* x, const double* w, const double* b,
                      int64_t cnt, const int64_t* flat, double* out, double* S) {
  const ConvDims c = conv_dims(dims);
#pragma omp parallel for schedule(dynamic)
  for (int64_t t = 0; t < cnt; ++t) {
    int64_t n, co, i, j;
    unflat4(flat[t], c.CO, c.HO, c.WO, &n, &co, &i, &j);
    conv_y_elem(c, x, w, b, n, co, i, j, &out[t], &S[t]);
  }
}

void or_conv2d_bwd_dx_at(const int64_t* dims, const double* dy, const double* w, int64_t cnt,
                         const int64_t* flat, double* out, double* S) {
  const ConvDims c = conv_dims(dims);
#pragma omp parallel for schedule(dynamic)
  for (int64_t t = 0; t < cnt; ++t) {
    int64_t n, ci, h, xx;
    unflat4(flat[t], c.C, c.H, c.W, &n, &ci, &h, &xx);
    conv_dx_elem(c, dy, w, n, ci, h, xx, &out[t], &S[t]);
  }
}

void or_conv2d_bwd_dw_at(const int64_t* dims, const double* dy, const double* x, int64_t cnt,
                         const int64_t* flat, double* out, double* S) {
  const ConvDims c = conv_dims(dims);
#pragma omp parallel for schedule(dynamic)
  for (int64_t t = 0; t < cnt; ++t) {
    int64_t co, ci, u, v;
    unflat4(flat[t], c.C, c.KH, c.KW, &co, &ci, &u, &v);
    conv_dw_elem(c, dy, x, co, ci, u, v, &out[t], &S[t]);
  }
}

}  // extern "C"

#ifdef _OPENMP
#include <omp.h>
#endif
extern "C" int or_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
