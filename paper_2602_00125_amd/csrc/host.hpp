// Host-side pieces shared by the C-ABI translation units (capi.cpp and
// conv_host.cpp): error recording, tensor checks, the product planner and
// launcher, and the test / tuning knobs. Internal: not part of the ABI.
#pragma once
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <string>

#include "../../include/minitensor_hip.h"
#include "gemm_params.hpp"

namespace mt::host {

// knobs set by mt_debug_set (-1 / 0 = automatic); atomics, read once per use
extern std::atomic<int> g_force_cfg, g_force_vec1, g_force_splits, g_force_parts, g_krot;
extern std::atomic<int> g_conv_gather, g_stream_k, g_sk_blocks, g_phase_grid, g_persist;

// records the message for mt_last_error() and returns s
mt_status fail(mt_status s, const std::string& msg);
mt_status hip_status(hipError_t e);
mt_status check_tensor(const mt_tensor* t, const char* name, int min_nd, int max_nd);
mt_status check_vector(const mt_tensor* t, const char* name, int64_t n);
bool overlaps(const mt_tensor* a, const mt_tensor* b);
bool is_row_major(const mt_tensor* t);
bool vec_ok_operand(const void* base, int64_t rows_other, int64_t contig_extent, int64_t ld,
                    const int64_t* bstrides, int nb, int per);

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }
inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// One matrix product as the planner sees it: launch description, operand
// layouts, vector width, tile configuration (-1 = choose), gathered operand.
struct GemmCall {
  mt::GemmParams p;
  bool a_kc, b_kc;
  bool vec;   // 16-byte operand loads and output stores
  bool bf16;  // bf16 operands (else fp32)
  int cfg;
  int conv;   // 1 / 2 / 3: the convolution product gathering an operand (p.cg), else 0
  int sk;     // stream-K blocks (conv 1 and 3 on the 256x256 tile), else 0
};


void init_params(mt::GemmParams* p);
// resolves tile, vector width, split-K / stream-K; returns the workspace the
// split needs (0 = none)
size_t plan_gemm(GemmCall& g, bool may_split);
// plans and launches (split partials in ws if it is large enough), then the
// split's finish
mt_status launch_gemm(GemmCall& g, hipStream_t stream, void* ws, size_t ws_bytes);

// the convolution entry points' bodies (conv_host.cpp); ws_query non-null:
// validate and report the workspace size only
mt_status conv_fwd_impl(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b,
                        const mt_tensor* y, int32_t sh, int32_t sw, int32_t ph, int32_t pw,
                        void* ws, size_t ws_bytes, hipStream_t stream, size_t* ws_query);
mt_status conv_bwd_impl(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                        const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db, int32_t sh,
                        int32_t sw, int32_t ph, int32_t pw, uint32_t flags, void* ws,
                        size_t ws_bytes, hipStream_t stream, size_t* ws_query);

}  // namespace mt::host
