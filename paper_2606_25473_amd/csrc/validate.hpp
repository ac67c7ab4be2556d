// validate.hpp -- argument validation of the compute entry points (plain C++, no HIP).
//
// Every pointer, size, alignment, overlap and layout check of the C ABI runs here,
// before any HIP call; on success the launch arguments are filled.  Kept free of HIP
// so that it can be built and exercised on the host alone (sanitizer tests).
#pragma once

#include <string>

#include "args.hpp"
#include "attn_jvp.h"

namespace attn {

// Record `msg` as this thread's last error message and return `code`.
int set_error(int code, const std::string& msg);
const char* last_error_message();

// Validation of attn_jvp_fwd / attn_jvp_fwd_zero_clean / attn_fwd (by `pass`).
int prepare(Pass pass, int dtype, int B, int H, int L, int D, const void* Q, const void* K, const void* V,
            const void* dQ, const void* dK, const void* dV, const attn_chunk_layout* layout,
            float softmax_scale, void* O, void* dO, float* LSE, AttnArgs* args);

// Validation of attn_bwd: `qa` gets the query-group table, `ka` the key-group table.
int prepare_bwd(int dtype, int B, int H, int L, int D, const void* Q, const void* K, const void* V,
                const void* O, const void* gO, const float* LSE, const attn_chunk_layout* layout,
                float softmax_scale, void* gQ, void* gK, void* gV, float* Delta, BwdArgs* qa, BwdArgs* ka);

}  // namespace attn
