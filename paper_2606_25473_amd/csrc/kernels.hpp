// kernels.hpp -- kernel launch interface used by the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>

#include "args.hpp"

namespace attn {

hipError_t launch_mfma_bf16(const AttnArgs& a, int D, Pass pass, hipStream_t stream);
hipError_t launch_mfma_f32(const AttnArgs& a, int D, Pass pass, hipStream_t stream);

// The backward is two launches on one stream: the query-tile pass (gQ and Delta, with
// `qa` holding the query-tile order) and then the key-tile pass (gK and gV, with `ka`
// holding the key-tile order), which reads Delta.
hipError_t launch_bwd_mfma_bf16(const BwdArgs& qa, const BwdArgs& ka, int D, hipStream_t stream);
hipError_t launch_bwd_mfma_f32(const BwdArgs& qa, const BwdArgs& ka, int D, hipStream_t stream);

}  // namespace attn
