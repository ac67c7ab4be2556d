// capi.hip -- the extern "C" compute entry points declared in include/attn_jvp.h.
//
// Every argument and the mask layout are validated on the host (validate.cpp) before
// any HIP call; the derived query-group table and tile order travel to the kernels by
// value.  Errors are reported by return code plus a thread-local message.
#include <hip/hip_runtime.h>

#include <string>

#include "attn_jvp.h"
#include "kernels.hpp"
#include "validate.hpp"

namespace {

int launch(attn::Pass pass, int dtype, int D, const attn::AttnArgs& args, void* stream) {
  const hipError_t e = dtype == ATTN_DTYPE_BF16
                           ? attn::launch_mfma_bf16(args, D, pass, (hipStream_t)stream)
                           : attn::launch_mfma_f32(args, D, pass, (hipStream_t)stream);
  if (e != hipSuccess) return attn::set_error(ATTN_ERR_HIP, std::string("HIP launch failed: ") + hipGetErrorString(e));
  return ATTN_OK;
}

}  // namespace

extern "C" {

int attn_jvp_fwd(int dtype, int B, int H, int L, int D, const void* Q, const void* K, const void* V,
                 const void* dQ, const void* dK, const void* dV, const attn_chunk_layout* layout,
                 float softmax_scale, void* O, void* dO, float* LSE, void* stream) {
  attn::AttnArgs args;
  const int rc = attn::prepare(attn::Pass::kJvp, dtype, B, H, L, D, Q, K, V, dQ, dK, dV, layout, softmax_scale,
                               O, dO, LSE, &args);
  if (rc != ATTN_OK) return rc;
  return launch(attn::Pass::kJvp, dtype, D, args, stream);
}

int attn_jvp_fwd_zero_clean(int dtype, int B, int H, int L, int D, const void* Q, const void* K,
                            const void* V, const void* dQn, const void* dKn, const void* dVn,
                            const attn_chunk_layout* layout, float softmax_scale, void* O, void* dOn,
                            float* LSE, void* stream) {
  attn::AttnArgs args;
  const int rc = attn::prepare(attn::Pass::kJvpZeroClean, dtype, B, H, L, D, Q, K, V, dQn, dKn, dVn, layout,
                               softmax_scale, O, dOn, LSE, &args);
  if (rc != ATTN_OK) return rc;
  return launch(attn::Pass::kJvpZeroClean, dtype, D, args, stream);
}

int attn_fwd(int dtype, int B, int H, int L, int D, const void* Q, const void* K, const void* V,
             const attn_chunk_layout* layout, float softmax_scale, void* O, float* LSE, void* stream) {
  attn::AttnArgs args;
  const int rc = attn::prepare(attn::Pass::kFwd, dtype, B, H, L, D, Q, K, V, nullptr, nullptr, nullptr, layout,
                               softmax_scale, O, nullptr, LSE, &args);
  if (rc != ATTN_OK) return rc;
  return launch(attn::Pass::kFwd, dtype, D, args, stream);
}

int attn_bwd(int dtype, int B, int H, int L, int D, const void* Q, const void* K, const void* V, const void* O,
             const void* gO, const float* LSE, const attn_chunk_layout* layout, float softmax_scale, void* gQ,
             void* gK, void* gV, float* Delta, void* stream) {
  attn::BwdArgs qa, ka;
  const int rc = attn::prepare_bwd(dtype, B, H, L, D, Q, K, V, O, gO, LSE, layout, softmax_scale, gQ, gK, gV,
                                   Delta, &qa, &ka);
  if (rc != ATTN_OK) return rc;
  const hipError_t e = dtype == ATTN_DTYPE_BF16 ? attn::launch_bwd_mfma_bf16(qa, ka, D, (hipStream_t)stream)
                                                : attn::launch_bwd_mfma_f32(qa, ka, D, (hipStream_t)stream);
  if (e != hipSuccess) return attn::set_error(ATTN_ERR_HIP, std::string("HIP launch failed: ") + hipGetErrorString(e));
  return ATTN_OK;
}

}  // extern "C"
