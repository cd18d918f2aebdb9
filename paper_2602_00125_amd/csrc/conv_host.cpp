// Host side of the convolution (MiniTensor Sec. 3.3 Eq. (6)): geometry and
// layout checks, the choice between products that gather their image
// operand and the unfolded path, the workspace plan, and the launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/minitensor_hip.h"
#include "gemm_params.hpp"
#include "host.hpp"
#include "kernels.hpp"

namespace mt::host {
namespace {

// ---------------------------------------------------------- convolution
struct ConvPlan {
  mt::ConvGeom g;
  int64_t M;         // output pixels N HO WO (rows of the unfolded matrix)
  int64_t wpitch;    // row pitch of the flattened weights [CO][Kc]
  size_t col_bytes;  // the unfolded matrix in the workspace, rounded up to 256
};

// dims `perm` (innermost first) of t form one dense row-major block
bool dense_block(const mt_tensor* t, const int* perm, int n) {
  int64_t expect = 1;
  for (int i = 0; i < n; ++i) {
    const int d = perm[i];
    if (t->shape[d] != 1 && t->stride[d] != expect) return false;
    expect *= t->shape[d];
  }
  return true;
}

// [N][C][H][W] stored channels-last: C fastest, then W, H, N, no gaps
bool channels_last(const mt_tensor* t) {
  static const int perm[4] = {1, 3, 2, 0};
  return dense_block(t, perm, 4);
}

mt_status conv_plan(const mt_tensor* x, const mt_tensor* w, int32_t sh, int32_t sw, int32_t ph,
                    int32_t pw, ConvPlan* cp) {
  mt_status s;
  if ((s = check_tensor(x, "x", 4, 4)) || (s = check_tensor(w, "w", 4, 4))) return s;
  if (x->dtype != MT_F32 || w->dtype != MT_F32)
    return fail(MT_ERR_DTYPE, "convolution: x and w must be f32");
  if (sh < 1 || sw < 1 || ph < 0 || pw < 0)
    return fail(MT_ERR_INVALID, "convolution: stride >= 1 and padding >= 0 required");
  const int64_t N = x->shape[0], C = x->shape[1], H = x->shape[2], W = x->shape[3];
  const int64_t CO = w->shape[0], KH = w->shape[2], KW = w->shape[3];
  if (w->shape[1] != C) return fail(MT_ERR_SHAPE, "convolution: w[1] must equal x's channels");
  if (C < 1 || H < 1 || W < 1 || CO < 1 || KH < 1 || KW < 1)
    return fail(MT_ERR_SHAPE, "convolution: every size but the batch must be >= 1");
  const int64_t lim = (int64_t)1 << 30;
  if (N >= lim || C >= lim || H >= lim || W >= lim || CO >= lim || KH >= lim || KW >= lim ||
      ph >= lim / 4 || pw >= lim / 4)
    return fail(MT_ERR_SHAPE, "convolution: a size exceeds 2^30");
  if (H + 2 * ph < KH || W + 2 * pw < KW)
    return fail(MT_ERR_SHAPE, "convolution: the kernel is larger than the padded image");
  const int64_t HO = (H + 2 * ph - KH) / sh + 1, WO = (W + 2 * pw - KW) / sw + 1;
  static const int uvc[3] = {1, 3, 2};  // c fastest, then v, u
  static const int cuv[3] = {3, 2, 1};  // v fastest, then u, c
  int korder;
  if (dense_block(w, cuv, 3)) korder = 0;
  else if (dense_block(w, uvc, 3)) korder = 1;
  else
    return fail(MT_ERR_LAYOUT, "w: the taps of one output channel must be contiguous, "
                               "[CO][C][KH][KW] or channels-last [CO][KH][KW][C]");
  const int64_t Kc = C * KH * KW;
  mt::ConvGeom& g = cp->g;
  std::memset(&g, 0, sizeof(g));
  g.N = (int32_t)N; g.C = (int32_t)C; g.H = (int32_t)H; g.W = (int32_t)W;
  g.CO = (int32_t)CO; g.KH = (int32_t)KH; g.KW = (int32_t)KW;
  g.sh = sh; g.sw = sw; g.ph = ph; g.pw = pw;
  g.HO = (int32_t)HO; g.WO = (int32_t)WO;
  g.korder_uvc = korder;
  g.Kc = Kc;
  g.Kcp = (Kc + 3) / 4 * 4;
  for (int d = 0; d < 4; ++d) g.xs[d] = x->stride[d];
  cp->M = N * HO * WO;
  cp->wpitch = CO > 1 ? w->stride[0] : Kc;
  if (cp->wpitch < Kc) return fail(MT_ERR_LAYOUT, "w: output channels overlap");
  const int64_t bytes = cp->M * g.Kcp * 4;
  cp->col_bytes = (size_t)((bytes + 255) / 256 * 256);
  return MT_OK;
}

// (mag, shift) with n / d = (n * mag) >> shift for every n < 2^31: shift =
// 31 + ceil(log2 d), mag = ceil(2^shift / d), which stays below 2^32.
void fast_div_params(int64_t d, uint32_t* mag, int32_t* shift) {
  int l = 0;
  while (((int64_t)1 << l) < d) ++l;
  const int s = 31 + l;
  *mag = (uint32_t)((((uint64_t)1 << s) + (uint64_t)d - 1) / (uint64_t)d);
  *shift = s;
}

// Whether a convolution product may gather the image in its loads instead of
// reading the unfolded matrix (mode 1: the forward, whose K-stages are whole
// groups of 32 channels of one tap; mode 2: the weight gradient, 4-channel
// chunks), and the description the kernels take. Needs channels-last x and
// weights (k = (u, v, c)), 16-byte aligned pixels, 32-bit offsets into x.
bool conv_gather(const ConvPlan& cp, const mt_tensor* x, int mode, mt::ConvGather* cg) {
  const mt::ConvGeom& g = cp.g;
  if (!g_conv_gather || g_force_vec1 || !g.korder_uvc || g.xs[1] != 1) return false;
  if (g.C % (mode == 1 ? 32 : 4) != 0) return false;
  if (!aligned16(x->data) || g.xs[0] % 4 || g.xs[2] % 4 || g.xs[3] % 4) return false;
  const int64_t lim = (int64_t)1 << 14;
  if (g.H >= lim || g.W >= lim || g.KH >= lim || g.KW >= lim || g.ph >= lim || g.pw >= lim)
    return false;
  const int64_t ext = (int64_t)(g.N - 1) * g.xs[0] + (int64_t)(g.H - 1) * g.xs[2] +
                      (int64_t)(g.W - 1) * g.xs[3] + g.C;
  if (ext + (int64_t)g.ph * g.xs[2] + (int64_t)g.pw * g.xs[3] >= ((int64_t)1 << 29)) return false;
  if (cp.M >= ((int64_t)1 << 31) - 64) return false;
  std::memset(cg, 0, sizeof(*cg));
  cg->x = (const float*)x->data;
  cg->x_bytes = (uint32_t)(ext * 4);
  cg->C = g.C; cg->H = g.H; cg->W = g.W; cg->KW = g.KW;
  cg->sh = g.sh; cg->sw = g.sw; cg->ph = g.ph; cg->pw = g.pw;
  cg->HO = g.HO; cg->WO = g.WO;
  cg->xs0 = (int32_t)g.xs[0]; cg->xs2 = (int32_t)g.xs[2]; cg->xs3 = (int32_t)g.xs[3];
  fast_div_params(g.WO, &cg->wo_mag, &cg->wo_shift);
  fast_div_params(g.HO, &cg->ho_mag, &cg->ho_shift);
  return true;
}

// Whether the input gradient may be computed by products gathering dy
// (channels-last dy, w and dx, CO a multiple of 32, 16-byte aligned rows,
// sizes within the gather's 32-bit offsets).
bool dgrad_gather_layout_ok(const ConvPlan& cp, const mt_tensor* dy, const mt_tensor* w,
                            const mt_tensor* dx) {
  const mt::ConvGeom& g = cp.g;
  if (!g_conv_gather || g_force_vec1 || !g.korder_uvc) return false;
  if (g.CO % 32 != 0 || g.C % 4 != 0 || !channels_last(dx) || !aligned16(dx->data)) return false;
  if (!aligned16(dy->data) || !aligned16(w->data) || cp.wpitch % 4 != 0) return false;
  const int64_t lim = (int64_t)1 << 14;
  if (g.H >= lim || g.W >= lim || g.HO >= lim || g.WO >= lim || g.KH >= lim || g.KW >= lim ||
      g.ph >= lim || g.pw >= lim)
    return false;
  const int64_t ys0 = dy->stride[0], ys2 = dy->stride[2], ys3 = dy->stride[3];
  if (ys0 % 4 || ys2 % 4 || ys3 % 4) return false;
  if ((int64_t)g.N * ys0 + (int64_t)(g.H + g.ph + 1) * ys2 + (int64_t)(g.W + g.pw + 1) * ys3 +
          g.CO >= ((int64_t)1 << 29))
    return false;
  return (int64_t)g.N * g.H * g.W < ((int64_t)1 << 31) - 64;
}

// The gathered description of dy for the input-gradient products, with the
// roles of the forward's fields turned round: the gathered image is dy (CO
// channels, HO x WO), the rows decode over rows x cols pixels per image and
// the window origin of row (i, j) is (i - ph', j - pw'), taps entering with a
// minus sign. For a stride-1 convolution rows x cols = H x W and ph' = -ph.
void dgrad_cg(const ConvPlan& cp, const mt_tensor* dy, int64_t rows, int64_t cols, int64_t ph_,
              int64_t pw_, int64_t taps_w, mt::ConvGather* cg) {
  const mt::ConvGeom& g = cp.g;
  const int64_t ys0 = dy->stride[0], ys2 = dy->stride[2], ys3 = dy->stride[3];
  std::memset(cg, 0, sizeof(*cg));
  cg->x = (const float*)dy->data;
  cg->x_bytes = (uint32_t)(((int64_t)(g.N - 1) * ys0 + (int64_t)(g.HO - 1) * ys2 +
                            (int64_t)(g.WO - 1) * ys3 + g.CO) * 4);
  cg->C = g.CO; cg->H = g.HO; cg->W = g.WO; cg->KW = (int32_t)taps_w;
  cg->sh = 1; cg->sw = 1; cg->ph = (int32_t)ph_; cg->pw = (int32_t)pw_;
  cg->HO = (int32_t)rows; cg->WO = (int32_t)cols;
  cg->xs0 = (int32_t)ys0; cg->xs2 = (int32_t)ys2; cg->xs3 = (int32_t)ys3;
  fast_div_params(cols, &cg->wo_mag, &cg->wo_shift);
  fast_div_params(rows, &cg->ho_mag, &cg->ho_shift);
}

// Whether the input gradient of a stride-1 convolution may run as one product
// gathering dy (dx = V W with V[(n, h, w)][(u, v, co)] = dY[n][h + ph - u][w + pw - v][co]
// and W read tap by tap) instead of dU = dY Wf and the fold.
bool conv_dgrad_gather(const ConvPlan& cp, const mt_tensor* dy, const mt_tensor* w,
                       const mt_tensor* dx, mt::ConvGather* cg) {
  const mt::ConvGeom& g = cp.g;
  if (g.sh != 1 || g.sw != 1 || !dgrad_gather_layout_ok(cp, dy, w, dx)) return false;
  dgrad_cg(cp, dy, g.H, g.W, -g.ph, -g.pw, g.KW, cg);
  return true;
}

// One sub-pixel phase (a, b) of a strided input gradient: the dx pixels with
// (h + ph) % sh == a and (w + pw) % sw == b, i.e. h = a - ph + sh i'. Only the
// taps u = a + sh t, v = b + sw r reach them, from dY row i' - t, column
// j' - r: a stride-1 gathered product over those taps. Returns false when the
// phase holds no pixel.
struct DgradPhase {
  mt::ConvGather cg;
  int64_t M, K;
};
bool dgrad_phase(const ConvPlan& cp, const mt_tensor* dy, int a, int b, DgradPhase* ph) {
  const mt::ConvGeom& g = cp.g;
  auto first = [](int64_t pad, int64_t r, int64_t s) { return pad > r ? (pad - r + s - 1) / s : 0; };
  const int64_t i0 = first(g.ph, a, g.sh), j0 = first(g.pw, b, g.sw);
  // pixels: a - ph + sh i' < H
  const int64_t i_end = (g.H - a + g.ph + g.sh - 1) / g.sh, j_end = (g.W - b + g.pw + g.sw - 1) / g.sw;
  const int64_t rows = i_end - i0, cols = j_end - j0;
  if (rows <= 0 || cols <= 0) return false;
  const int64_t th = (g.KH - a + g.sh - 1) / g.sh, tw = (g.KW - b + g.sw - 1) / g.sw;
  dgrad_cg(cp, dy, rows, cols, -i0, -j0, tw, &ph->cg);
  ph->cg.u0 = a; ph->cg.v0 = b; ph->cg.su = g.sh; ph->cg.sv = g.sw; ph->cg.wKW = g.KW;
  ph->cg.eH = g.H; ph->cg.eW = g.W; ph->cg.esh = g.sh; ph->cg.esw = g.sw;
  ph->cg.h0 = (int32_t)(a - g.ph + g.sh * i0);
  ph->cg.w0 = (int32_t)(b - g.pw + g.sw * j0);
  ph->M = (int64_t)g.N * rows * cols;
  ph->K = th * tw * g.CO;
  return true;
}

mt_status check_act4(const mt_tensor* t, const char* name, int64_t N, int64_t C, int64_t H,
                     int64_t W) {
  mt_status s = check_tensor(t, name, 4, 4);
  if (s) return s;
  if (t->dtype != MT_F32) return fail(MT_ERR_DTYPE, std::string(name) + ": must be f32");
  if (t->shape[0] != N || t->shape[1] != C || t->shape[2] != H || t->shape[3] != W)
    return fail(MT_ERR_SHAPE, std::string(name) + ": wrong shape");
  return MT_OK;
}

}  // namespace

mt_status conv_fwd_impl(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b,
                        const mt_tensor* y, int32_t sh, int32_t sw, int32_t ph, int32_t pw,
                        void* ws, size_t ws_bytes, hipStream_t stream, size_t* ws_query) {
  ConvPlan cp;
  mt_status s = conv_plan(x, w, sh, sw, ph, pw, &cp);
  if (s) return s;
  const mt::ConvGeom& g = cp.g;
  if ((s = check_act4(y, "y", g.N, g.CO, g.HO, g.WO))) return s;
  if (!channels_last(y)) return fail(MT_ERR_LAYOUT, "y must be channels-last contiguous");
  if (b && (s = check_vector(b, "b", g.CO))) return s;
  if (overlaps(y, x) || overlaps(y, w) || overlaps(y, b))
    return fail(MT_ERR_ALIAS, "y overlaps an input");
  GemmCall gc{};
  init_params(&gc.p);
  gc.p.b = w->data;
  gc.p.c = (float*)y->data;
  gc.p.bias = b ? (const float*)b->data : nullptr;
  gc.p.M = cp.M;
  gc.p.N = g.CO;
  gc.p.K = g.Kc;
  gc.p.lda = g.Kcp;
  gc.p.ldb = cp.wpitch;
  gc.p.ldc = g.CO;
  gc.a_kc = true;
  gc.b_kc = true;
  gc.bf16 = false;
  gc.vec = g.Kc % 4 == 0 && vec_ok_operand(w->data, g.CO, g.Kc, cp.wpitch, nullptr, 0, 4) &&
           aligned16(y->data) && g.CO % 4 == 0 && (!gc.p.bias || aligned16(gc.p.bias));
  gc.cfg = -1;
  // the product reads the image itself where it can, else the unfolded input
  // in the workspace
  const bool gather = gc.vec && conv_gather(cp, x, 1, &gc.p.cg);
  if (gather) {
    gc.conv = 1;
    gc.p.a = x->data;
    gc.p.lda = 0;
  }
  // the workspace: the unfolded input (if the product does not gather), then
  // split-K or stream-K partial tiles (optional: without them one tile per
  // block over the whole contraction)
  const size_t col_need = gather ? 0 : cp.col_bytes;
  if (ws_query) {
    GemmCall probe = gc;
    *ws_query = col_need + plan_gemm(probe, true);
    return MT_OK;
  }
  if (cp.M == 0) return MT_OK;
  if (ws && ((uintptr_t)ws & 255)) return fail(MT_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (!gather && (!ws || ws_bytes < cp.col_bytes))
    return fail(MT_ERR_WORKSPACE, "convolution: needs a 256-byte aligned workspace of "
                                  "mt_conv2d_fwd_workspace bytes (the unfolded input)");
  char* rest = ws ? (char*)ws + col_need : nullptr;
  const size_t rest_bytes = ws && ws_bytes > col_need ? ws_bytes - col_need : 0;
  if (!gather) {
    (void)hipGetLastError();
    if ((s = hip_status(mt::conv_unfold((const float*)x->data, g, (float*)ws, stream)))) return s;
    gc.p.a = ws;
  }
  return launch_gemm(gc, stream, rest_bytes ? rest : nullptr, rest_bytes);
}

mt_status conv_bwd_impl(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                        const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db, int32_t sh,
                        int32_t sw, int32_t ph, int32_t pw, uint32_t flags, void* ws,
                        size_t ws_bytes, hipStream_t stream, size_t* ws_query) {
  if (flags & ~(MT_ACCUMULATE | MT_CONV_REUSE_UNFOLD))
    return fail(MT_ERR_INVALID, "mt_conv2d_bwd: unknown flags");
  ConvPlan cp;
  mt_status s = conv_plan(x, w, sh, sw, ph, pw, &cp);
  if (s) return s;
  mt::ConvGeom& g = cp.g;
  if ((s = check_act4(dy, "dy", g.N, g.CO, g.HO, g.WO))) return s;
  if (!channels_last(dy)) return fail(MT_ERR_LAYOUT, "dy must be channels-last contiguous");
  if (dx) {
    if ((s = check_act4(dx, "dx", g.N, g.C, g.H, g.W))) return s;
    if (!channels_last(dx) && !is_row_major(dx))
      return fail(MT_ERR_LAYOUT, "dx must be contiguous, channels-last or [N][C][H][W]");
    for (int d = 0; d < 4; ++d) g.ds[d] = dx->stride[d];
    g.dx_vec = (g.C == 1 || dx->stride[1] == 1) && aligned16(dx->data) && dx->stride[0] % 4 == 0 &&
               dx->stride[2] % 4 == 0 && dx->stride[3] % 4 == 0;
  }
  if (dw) {
    s = check_tensor(dw, "dw", 4, 4);
    if (s) return s;
    if (dw->dtype != MT_F32) return fail(MT_ERR_DTYPE, "dw must be f32");
    for (int d = 0; d < 4; ++d)
      if (dw->shape[d] != w->shape[d]) return fail(MT_ERR_SHAPE, "dw must have w's shape");
    static const int uvc[3] = {1, 3, 2};
    static const int cuv[3] = {3, 2, 1};
    if (!dense_block(dw, g.korder_uvc ? uvc : cuv, 3))
      return fail(MT_ERR_LAYOUT, "dw must store the taps in w's order");
    if (g.CO > 1 && dw->stride[0] < g.Kc) return fail(MT_ERR_LAYOUT, "dw: output channels overlap");
  }
  if (db && (s = check_vector(db, "db", g.CO))) return s;
  const mt_tensor* ins[3] = {x, w, dy};
  const mt_tensor* outs[3] = {dx, dw, db};
  for (int i = 0; i < 3; ++i) {
    if (!outs[i]) continue;
    for (int j = 0; j < 3; ++j)
      if (overlaps(outs[i], ins[j])) return fail(MT_ERR_ALIAS, "an output overlaps an input");
    for (int j = i + 1; j < 3; ++j)
      if (overlaps(outs[i], outs[j])) return fail(MT_ERR_ALIAS, "outputs overlap");
  }
  const bool acc = (flags & MT_ACCUMULATE) != 0;
  const int64_t dwpitch = dw ? (g.CO > 1 ? dw->stride[0] : g.Kc) : 0;
  // dW = dY^T U (U unfolded into the workspace), split over the pixels when its
  // few output tiles under-fill the GPU; partial tiles go after U
  GemmCall gdw{};
  size_t need_dw = 0;
  bool fold_db = false;
  if (dw) {
    init_params(&gdw.p);
    gdw.p.a = dy->data;
    gdw.p.b = ws;  // U, set again at launch
    gdw.p.c = (float*)dw->data;
    gdw.p.M = g.CO;
    gdw.p.N = g.Kc;
    gdw.p.K = cp.M;
    gdw.p.lda = g.CO;
    gdw.p.ldb = g.Kcp;
    gdw.p.ldc = dwpitch;
    gdw.p.accumulate = acc;
    gdw.a_kc = false;
    gdw.b_kc = false;
    gdw.bf16 = false;
    gdw.vec = g.CO % 4 == 0 && g.Kc % 4 == 0 && aligned16(dy->data) && aligned16(dw->data) &&
              dwpitch % 4 == 0;
    gdw.cfg = -1;
    if (gdw.vec && conv_gather(cp, x, 2, &gdw.p.cg)) {
      gdw.conv = 2;
      gdw.p.b = x->data;
      gdw.p.ldb = 0;
    }
    // db = the column sums of dY^T, A of this product: folded into it where
    // its kernel allows (no second pass over dY); the plan settles whether
    gdw.p.colsum = db ? (float*)db->data : nullptr;
    GemmCall probe = gdw;
    need_dw = plan_gemm(probe, true);
    fold_db = probe.p.colsum != nullptr;
  }
  int parts = 1;
  size_t need_db = 0;
  if (db && cp.M > 0) {
    const int fp = g_force_parts;
    parts = fp > 0 ? fp : mt::colsum_parts(cp.M, g.CO);
    if (parts > 1 && !fold_db) need_db = (size_t)parts * g.CO * sizeof(float);
  }
  // dx = V W in one product where dy can be gathered (V: dy over the
  // mirrored taps), its rows the input pixels
  GemmCall gdxg{};
  const bool dx_gather = dx && conv_dgrad_gather(cp, dy, w, dx, &gdxg.p.cg);
  // strided: one gathered product per sub-pixel phase, where every phase has
  // taps (KH >= sh, KW >= sw)
  const bool dx_phased = dx && !dx_gather && (g.sh > 1 || g.sw > 1) && g.KH >= g.sh &&
                         g.KW >= g.sw && dgrad_gather_layout_ok(cp, dy, w, dx);
  size_t need_dx = 0;
  if (dx_gather) {
    const mt::ConvGather dcg = gdxg.p.cg;
    init_params(&gdxg.p);
    gdxg.p.cg = dcg;
    gdxg.p.a = dy->data;
    gdxg.p.b = w->data;
    gdxg.p.c = (float*)dx->data;
    gdxg.p.M = (int64_t)g.N * g.H * g.W;
    gdxg.p.N = g.C;
    gdxg.p.K = (int64_t)g.KH * g.KW * g.CO;  // k = (u, v, co)
    gdxg.p.lda = 0;
    gdxg.p.ldb = cp.wpitch;
    gdxg.p.ldc = g.C;
    gdxg.p.accumulate = acc;
    gdxg.a_kc = true;
    gdxg.b_kc = false;
    gdxg.bf16 = false;
    gdxg.vec = true;
    gdxg.cfg = -1;
    gdxg.conv = 3;
    GemmCall probe = gdxg;
    need_dx = plan_gemm(probe, true);
  }
  // the unfolded matrix (U for an unfolded dW, then dU for an unfolded dx)
  // heads the workspace; split or stream-K partials follow (the products run
  // one after another and share them)
  const size_t col_need = ((dx && !dx_gather && !dx_phased) || (dw && !gdw.conv)) ? cp.col_bytes : 0;
  const size_t need = col_need + std::max(std::max(need_dw, need_db), need_dx);
  if (ws_query) {
    *ws_query = need;
    return MT_OK;
  }
  if (col_need && cp.M > 0 && (!ws || ws_bytes < col_need || ((uintptr_t)ws & 255)))
    return fail(MT_ERR_WORKSPACE, "convolution: needs a 256-byte aligned workspace of "
                                  "mt_conv2d_bwd_workspace bytes (the unfolded input)");
  if (ws && ((uintptr_t)ws & 255)) return fail(MT_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  float* col = (float*)ws;
  char* rest = ws ? (char*)ws + col_need : nullptr;
  const size_t rest_bytes = ws && ws_bytes > col_need ? ws_bytes - col_need : 0;
  (void)hipGetLastError();
  if (dw && !gdw.conv) {
    // MT_CONV_REUSE_UNFOLD: the forward left the unfolded input at the start
    // of ws, unless that forward gathered the image (then nothing is there)
    mt::ConvGather unused;
    const bool reuse = (flags & MT_CONV_REUSE_UNFOLD) && !conv_gather(cp, x, 1, &unused);
    if (cp.M > 0 && !reuse &&
        (s = hip_status(mt::conv_unfold((const float*)x->data, g, col, stream))))
      return s;
    gdw.p.b = col;
    if ((s = launch_gemm(gdw, stream, rest_bytes ? rest : nullptr, rest_bytes))) return s;
  } else if (dw) {
    if ((s = launch_gemm(gdw, stream, rest_bytes ? rest : nullptr, rest_bytes))) return s;
  }
  // the product summed db itself (it ran: dW is not empty, and its kernel
  // kept the column sums)
  fold_db = dw && gdw.p.colsum != nullptr && gdw.p.M > 0 && gdw.p.N > 0;
  if (db && !fold_db) {
    (void)hipGetLastError();
    float* wsp = (rest && parts > 1 && rest_bytes >= need_db) ? (float*)rest : nullptr;
    if ((s = hip_status(mt::colsum(dy->data, false, cp.M, g.CO, g.CO, (float*)db->data, acc, wsp,
                                   parts, stream))))
      return s;
  }
  if (dx && dx_gather && cp.M > 0) {
    if ((s = launch_gemm(gdxg, stream, rest_bytes ? rest : nullptr, rest_bytes))) return s;
  } else if (dx && dx_phased && cp.M > 0) {
    // the phases holding pixels, longest contraction first
    std::vector<DgradPhase> phases;
    for (int a = 0; a < g.sh; ++a)
      for (int bb = 0; bb < g.sw; ++bb) {
        DgradPhase ph;
        if (dgrad_phase(cp, dy, a, bb, &ph)) phases.push_back(ph);
      }
    std::stable_sort(phases.begin(), phases.end(),
                     [](const DgradPhase& l, const DgradPhase& r) { return l.K > r.K; });
    int64_t rows = 0;
    for (const DgradPhase& ph : phases) rows += ph.M;
    // one grid of 256x256 tiles where that tile fits the channels (measured at
    // 32 x 256 x 56 x 56, 3x3, stride 2: dx 0.308 ms against 0.355 for a launch
    // per phase; with 128 channels half of every tile would idle: 0.28 against 0.20)
    const double used = (double)g.C / (double)(cdiv(g.C, 256) * 256);
    const int pg = g_phase_grid;
    const bool one_grid = pg == 2 || (pg == 1 && rows >= 256 * 64 && used >= 0.9);
    if (one_grid && !phases.empty() && (int)phases.size() <= mt::kMaxConvPhases && g.C % 4 == 0) {
      // one grid of 256x256 tiles: every phase's tiles run side by side
      mt::ConvPhases tab;
      std::memset(&tab, 0, sizeof(tab));
      tab.n = (int32_t)phases.size();
      for (int k = 0; k < tab.n; ++k) {
        const DgradPhase& ph = phases[k];
        mt::ConvPhase& f = tab.ph[k];
        f.M = ph.M;
        f.K = ph.K;
        f.tiles_m = (int32_t)cdiv(ph.M, 256);
        f.u0 = ph.cg.u0; f.v0 = ph.cg.v0; f.ph = ph.cg.ph; f.pw = ph.cg.pw;
        f.rows = ph.cg.HO; f.cols = ph.cg.WO; f.kw = ph.cg.KW; f.h0 = ph.cg.h0; f.w0 = ph.cg.w0;
        f.wo_mag = ph.cg.wo_mag; f.ho_mag = ph.cg.ho_mag;
        f.wo_shift = ph.cg.wo_shift; f.ho_shift = ph.cg.ho_shift;
        tab.tile0[k + 1] = tab.tile0[k] + f.tiles_m * (int32_t)cdiv(g.C, 256);
      }
      mt::GemmParams p;
      init_params(&p);
      p.cg = phases[0].cg;
      p.a = dy->data;
      p.b = w->data;
      p.c = (float*)dx->data;
      p.M = phases[0].M;
      p.N = g.C;
      p.K = phases[0].K;
      p.ldb = cp.wpitch;
      p.ldc = g.C;
      p.accumulate = acc;
      (void)hipGetLastError();
      if ((s = hip_status(mt::gemm_f32_conv_phases(p, tab, stream)))) return s;
    } else {
      for (const DgradPhase& ph : phases) {
        GemmCall gp{};
        init_params(&gp.p);
        gp.p.cg = ph.cg;
        gp.p.a = dy->data;
        gp.p.b = w->data;
        gp.p.c = (float*)dx->data;
        gp.p.M = ph.M;
        gp.p.N = g.C;
        gp.p.K = ph.K;
        gp.p.lda = 0;
        gp.p.ldb = cp.wpitch;
        gp.p.ldc = g.C;
        gp.p.accumulate = acc;
        gp.a_kc = true;
        gp.b_kc = false;
        gp.bf16 = false;
        gp.vec = true;
        gp.cfg = -1;
        gp.conv = 4;
        // no split: the phase's rows land directly in dx
        if ((s = launch_gemm(gp, stream, nullptr, 0))) return s;
      }
    }
  } else if (dx && cp.M > 0) {
    // dU = dY Wf into the workspace (U is no longer needed), then the fold
    GemmCall gdx{};
    init_params(&gdx.p);
    gdx.p.a = dy->data;
    gdx.p.b = w->data;
    gdx.p.c = col;
    gdx.p.M = cp.M;
    gdx.p.N = g.Kc;
    gdx.p.K = g.CO;
    gdx.p.lda = g.CO;
    gdx.p.ldb = cp.wpitch;
    gdx.p.ldc = g.Kcp;
    gdx.a_kc = true;
    gdx.b_kc = false;
    gdx.bf16 = false;
    gdx.vec = g.CO % 4 == 0 && aligned16(dy->data) &&
              vec_ok_operand(w->data, g.CO, g.Kc, cp.wpitch, nullptr, 0, 4) && g.Kc % 4 == 0;
    gdx.cfg = -1;
    if ((s = launch_gemm(gdx, stream, nullptr, 0))) return s;
    (void)hipGetLastError();
    if ((s = hip_status(mt::conv_fold(col, g, (float*)dx->data, acc, stream)))) return s;
  }
  return MT_OK;
}


}  // namespace mt::host
