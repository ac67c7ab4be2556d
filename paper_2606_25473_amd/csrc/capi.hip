// capi.hip -- the extern "C" entry points declared in include/attn_jvp.h.
//
// Every argument and the chunk layout are validated on the host before any
// HIP call; the derived query-group table and tile order travel to the kernel
// by value.  Errors are reported by return code plus a thread-local message.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "attn_jvp.h"
#include "kernels.hpp"
#include "layout.hpp"

namespace {

thread_local std::string g_last_error;

int fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

struct Span {
  uintptr_t lo, hi;
  const char* name;
};

bool overlap(const Span& x, const Span& y) { return x.lo < y.hi && y.lo < x.hi; }

// Size limits of the kernels (after the positivity checks): the bf16 kernels address a
// head with 32-bit byte offsets and launch one work-group per tile of at least 128 rows
// or keys and (batch, head) along x; the fp32 kernels launch one grid row per (batch,
// head) along y.
int check_sizes(int dtype, int B, int H, int L, int D) {
  const int64_t bh = (int64_t)B * H;
  if (bh > (int64_t)1 << 20) return fail(ATTN_ERR_INVALID, "B * H too large");
  if (dtype == ATTN_DTYPE_BF16) {
    if ((int64_t)L * D > (int64_t)1 << 31)
      return fail(ATTN_ERR_INVALID, "bf16 needs L * D <= 2^31 (32-bit offsets within a head), got L = " +
                                        std::to_string(L) + ", D = " + std::to_string(D));
    if (((int64_t)L + 127) / 128 * bh > INT32_MAX)
      return fail(ATTN_ERR_INVALID, "too many work-groups for one launch: ceil(L / 128) * B * H > 2^31 - 1");
  } else if (bh > 65535) {
    return fail(ATTN_ERR_INVALID, "fp32 needs B * H <= 65535, got " + std::to_string(bh));
  }
  return ATTN_OK;
}

int elem_size(int dtype) { return dtype == ATTN_DTYPE_F32 ? 4 : dtype == ATTN_DTYPE_BF16 ? 2 : 0; }

// Shared validation of the compute entry points; fills the launch arguments.
// kJvpZeroClean: teacher-forcing layouts only; the tangents (and dO) hold the noisy
// half, rows [L/2, L), of every (batch, head).
int prepare(attn::Pass pass, int dtype, int B, int H, int L, int D, const void* Q, const void* K,
            const void* V, const void* dQ, const void* dK, const void* dV,
            const attn_chunk_layout* layout, float softmax_scale, void* O, void* dO, float* LSE,
            attn::AttnArgs* args) {
  const bool jvp = pass != attn::Pass::kFwd;
  const bool zc = pass == attn::Pass::kJvpZeroClean;
  if (dtype != ATTN_DTYPE_F32 && dtype != ATTN_DTYPE_BF16)
    return fail(ATTN_ERR_UNSUPPORTED, "unsupported dtype " + std::to_string(dtype));
  if (D != 64 && D != 128)
    return fail(ATTN_ERR_UNSUPPORTED, "unsupported head_dim " + std::to_string(D) + " (built: 64, 128)");
  if (B <= 0 || H <= 0 || L <= 0)
    return fail(ATTN_ERR_INVALID, "B, H and L must be positive (B=" + std::to_string(B) +
                                      ", H=" + std::to_string(H) + ", L=" + std::to_string(L) + ")");
  if (const int rc = check_sizes(dtype, B, H, L, D)) return rc;
  if (!Q || !K || !V || !O || !LSE) return fail(ATTN_ERR_INVALID, "NULL tensor pointer");
  if (jvp && (!dQ || !dK || !dV || !dO)) return fail(ATTN_ERR_INVALID, "NULL tangent pointer");
  if (!layout) return fail(ATTN_ERR_INVALID, "layout is NULL");
  if (zc && layout->kind != ATTN_MASK_TEACHER_FORCING)
    return fail(ATTN_ERR_INVALID, "the zero-clean-tangent JVP needs a teacher-forcing layout");
  const int t0 = zc ? L / 2 : 0;
  const int es = elem_size(dtype);
  const uintptr_t tbytes = (uintptr_t)B * H * L * D * es;
  const uintptr_t gbytes = (uintptr_t)B * H * (L - t0) * D * es;  // tangents and dO
  const uintptr_t lbytes = (uintptr_t)B * H * L * sizeof(float);
  const uintptr_t align = dtype == ATTN_DTYPE_BF16 ? 16 : 4;
  const void* ins[6] = {Q, K, V, dQ, dK, dV};
  const char* in_names[6] = {"Q", "K", "V", "dQ", "dK", "dV"};
  const int nin = jvp ? 6 : 3;
  for (int i = 0; i < nin; ++i)
    if ((uintptr_t)ins[i] % align)
      return fail(ATTN_ERR_INVALID, std::string(in_names[i]) + " is not " + std::to_string(align) +
                                        "-byte aligned");
  if ((uintptr_t)O % align || (jvp && (uintptr_t)dO % align) || (uintptr_t)LSE % 4)
    return fail(ATTN_ERR_INVALID, "output pointer misaligned");
  Span outs[3] = {{(uintptr_t)O, (uintptr_t)O + tbytes, "O"},
                  {(uintptr_t)LSE, (uintptr_t)LSE + lbytes, "LSE"},
                  {(uintptr_t)dO, (uintptr_t)dO + gbytes, "dO"}};
  const int nout = jvp ? 3 : 2;
  for (int i = 0; i < nout; ++i) {
    for (int j = i + 1; j < nout; ++j)
      if (overlap(outs[i], outs[j]))
        return fail(ATTN_ERR_INVALID, std::string("outputs ") + outs[i].name + " and " + outs[j].name + " overlap");
    for (int k = 0; k < nin; ++k) {
      const Span in = {(uintptr_t)ins[k], (uintptr_t)ins[k] + (k < 3 ? tbytes : gbytes), in_names[k]};
      if (overlap(outs[i], in))
        return fail(ATTN_ERR_INVALID, std::string("output ") + outs[i].name + " overlaps input " + in.name);
    }
  }
  std::string err;
  if (!attn::build_groups(layout, L, &args->gt, &err)) return fail(ATTN_ERR_INVALID, err);
  args->Q = Q; args->K = K; args->V = V;
  args->dQ = dQ; args->dK = dK; args->dV = dV;
  args->O = O; args->dO = dO; args->LSE = LSE;
  args->B = B; args->H = H; args->L = L;
  args->t0 = t0;
  args->scale = softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf((float)D);
  // the forward-only bf16 kernel takes 128-row tiles, the JVP kernels 256-row tiles
  const int br = (pass == attn::Pass::kFwd && dtype == ATTN_DTYPE_BF16) ? attn::kMfmaBrFwd : attn::kMfmaBr;
  args->order = zc ? attn::make_tile_order_zero_clean(args->gt, L, attn::kMfmaBr, attn::kMfmaBc, t0)
                   : attn::make_tile_order(layout, L, br);
  return ATTN_OK;
}

int launch(attn::Pass pass, int dtype, int D, const attn::AttnArgs& args, void* stream) {
  const hipError_t e = dtype == ATTN_DTYPE_BF16
                           ? attn::launch_mfma_bf16(args, D, pass, (hipStream_t)stream)
                           : attn::launch_simt_f32(args, D, pass, (hipStream_t)stream);
  if (e != hipSuccess) return fail(ATTN_ERR_HIP, std::string("HIP launch failed: ") + hipGetErrorString(e));
  return ATTN_OK;
}

int prepare_bwd(int dtype, int B, int H, int L, int D, const void* Q, const void* K, const void* V,
                const void* O, const void* gO, const float* LSE, const attn_chunk_layout* layout,
                float softmax_scale, void* gQ, void* gK, void* gV, float* Delta, attn::BwdArgs* qa,
                attn::BwdArgs* ka) {
  if (dtype != ATTN_DTYPE_F32 && dtype != ATTN_DTYPE_BF16)
    return fail(ATTN_ERR_UNSUPPORTED, "unsupported dtype " + std::to_string(dtype));
  if (D != 64 && D != 128)
    return fail(ATTN_ERR_UNSUPPORTED, "unsupported head_dim " + std::to_string(D) + " (built: 64, 128)");
  if (B <= 0 || H <= 0 || L <= 0)
    return fail(ATTN_ERR_INVALID, "B, H and L must be positive (B=" + std::to_string(B) +
                                      ", H=" + std::to_string(H) + ", L=" + std::to_string(L) + ")");
  if (const int rc = check_sizes(dtype, B, H, L, D)) return rc;
  const void* ins[6] = {Q, K, V, O, gO, LSE};
  const char* in_names[6] = {"Q", "K", "V", "O", "gO", "LSE"};
  void* outs[4] = {gQ, gK, gV, Delta};
  const char* out_names[4] = {"gQ", "gK", "gV", "Delta"};
  for (int i = 0; i < 6; ++i)
    if (!ins[i]) return fail(ATTN_ERR_INVALID, std::string("NULL pointer ") + in_names[i]);
  for (int i = 0; i < 4; ++i)
    if (!outs[i]) return fail(ATTN_ERR_INVALID, std::string("NULL pointer ") + out_names[i]);
  const uintptr_t tbytes = (uintptr_t)B * H * L * D * elem_size(dtype);
  const uintptr_t lbytes = (uintptr_t)B * H * L * sizeof(float);
  const uintptr_t align = dtype == ATTN_DTYPE_BF16 ? 16 : 4;
  for (int i = 0; i < 6; ++i)
    if ((uintptr_t)ins[i] % (i < 5 ? align : 4))
      return fail(ATTN_ERR_INVALID, std::string(in_names[i]) + " is misaligned");
  for (int i = 0; i < 4; ++i)
    if ((uintptr_t)outs[i] % (i < 3 ? align : 4))
      return fail(ATTN_ERR_INVALID, std::string(out_names[i]) + " is misaligned");
  for (int i = 0; i < 4; ++i) {
    const Span o = {(uintptr_t)outs[i], (uintptr_t)outs[i] + (i < 3 ? tbytes : lbytes), out_names[i]};
    for (int j = i + 1; j < 4; ++j) {
      const Span p = {(uintptr_t)outs[j], (uintptr_t)outs[j] + (j < 3 ? tbytes : lbytes), out_names[j]};
      if (overlap(o, p))
        return fail(ATTN_ERR_INVALID, std::string("outputs ") + o.name + " and " + p.name + " overlap");
    }
    for (int k = 0; k < 6; ++k) {
      const Span in = {(uintptr_t)ins[k], (uintptr_t)ins[k] + (k < 5 ? tbytes : lbytes), in_names[k]};
      if (overlap(o, in))
        return fail(ATTN_ERR_INVALID, std::string("output ") + o.name + " overlaps input " + in.name);
    }
  }
  std::string err;
  if (!attn::build_groups(layout, L, &qa->gt, &err)) return fail(ATTN_ERR_INVALID, err);
  if (!attn::transpose_groups(qa->gt, L, &ka->gt, &err)) return fail(ATTN_ERR_UNSUPPORTED, err);
  qa->Q = ka->Q = Q; qa->K = ka->K = K; qa->V = ka->V = V;
  qa->O = ka->O = O; qa->gO = ka->gO = gO; qa->LSE = ka->LSE = LSE;
  qa->gQ = ka->gQ = gQ; qa->gK = ka->gK = gK; qa->gV = ka->gV = gV; qa->Delta = ka->Delta = Delta;
  qa->B = ka->B = B; qa->H = ka->H = H; qa->L = ka->L = L;
  qa->scale = ka->scale = softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf((float)D);
  qa->order = attn::make_tile_order(layout, L, attn::kMfmaBr);
  // key tiles: for the built-in layouts the work per key tile falls with the key index
  // (earlier keys are seen by more queries), so the natural order is heaviest first
  ka->order = attn::TileOrder{};
  ka->order.mode = 0;
  ka->order.nt = (L + attn::kBwdKeysPerTile - 1) / attn::kBwdKeysPerTile;
  ka->order.split = ka->order.nt;
  ka->order.first = -1;
  return ATTN_OK;
}

}  // namespace

extern "C" {

int attn_jvp_fwd(int dtype, int B, int H, int L, int D, const void* Q, const void* K, const void* V,
                 const void* dQ, const void* dK, const void* dV, const attn_chunk_layout* layout,
                 float softmax_scale, void* O, void* dO, float* LSE, void* stream) {
  attn::AttnArgs args;
  const int rc = prepare(attn::Pass::kJvp, dtype, B, H, L, D, Q, K, V, dQ, dK, dV, layout, softmax_scale,
                         O, dO, LSE, &args);
  if (rc != ATTN_OK) return rc;
  return launch(attn::Pass::kJvp, dtype, D, args, stream);
}

int attn_jvp_fwd_zero_clean(int dtype, int B, int H, int L, int D, const void* Q, const void* K,
                            const void* V, const void* dQn, const void* dKn, const void* dVn,
                            const attn_chunk_layout* layout, float softmax_scale, void* O, void* dOn,
                            float* LSE, void* stream) {
  attn::AttnArgs args;
  const int rc = prepare(attn::Pass::kJvpZeroClean, dtype, B, H, L, D, Q, K, V, dQn, dKn, dVn, layout,
                         softmax_scale, O, dOn, LSE, &args);
  if (rc != ATTN_OK) return rc;
  return launch(attn::Pass::kJvpZeroClean, dtype, D, args, stream);
}

int attn_fwd(int dtype, int B, int H, int L, int D, const void* Q, const void* K, const void* V,
             const attn_chunk_layout* layout, float softmax_scale, void* O, float* LSE, void* stream) {
  attn::AttnArgs args;
  const int rc = prepare(attn::Pass::kFwd, dtype, B, H, L, D, Q, K, V, nullptr, nullptr, nullptr, layout,
                         softmax_scale, O, nullptr, LSE, &args);
  if (rc != ATTN_OK) return rc;
  return launch(attn::Pass::kFwd, dtype, D, args, stream);
}

int attn_bwd(int dtype, int B, int H, int L, int D, const void* Q, const void* K, const void* V, const void* O,
             const void* gO, const float* LSE, const attn_chunk_layout* layout, float softmax_scale, void* gQ,
             void* gK, void* gV, float* Delta, void* stream) {
  attn::BwdArgs qa, ka;
  const int rc = prepare_bwd(dtype, B, H, L, D, Q, K, V, O, gO, LSE, layout, softmax_scale, gQ, gK, gV, Delta,
                             &qa, &ka);
  if (rc != ATTN_OK) return rc;
  const hipError_t e = dtype == ATTN_DTYPE_BF16 ? attn::launch_bwd_mfma_bf16(qa, ka, D, (hipStream_t)stream)
                                                : attn::launch_bwd_simt_f32(qa, ka, D, (hipStream_t)stream);
  if (e != hipSuccess) return fail(ATTN_ERR_HIP, std::string("HIP launch failed: ") + hipGetErrorString(e));
  return ATTN_OK;
}

int attn_key_groups(const attn_chunk_layout* layout, int L, int32_t* out, int max_groups) {
  attn::GroupTable gt, kt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) return fail(ATTN_ERR_INVALID, err), -1;
  if (!attn::transpose_groups(gt, L, &kt, &err)) return fail(ATTN_ERR_UNSUPPORTED, err), -1;
  if (!out || max_groups < kt.n) return fail(ATTN_ERR_INVALID, "output buffer too small"), -1;
  for (int g = 0; g < kt.n; ++g) {
    int32_t* r = out + 6 * g;
    r[0] = attn::group_q_begin(kt, g);
    r[1] = kt.q_end[g];
    r[2] = kt.a0[g]; r[3] = kt.a1[g];
    r[4] = kt.b0[g]; r[5] = kt.b1[g];
  }
  return kt.n;
}

int64_t attn_count_unmasked_pairs(const attn_chunk_layout* layout, int L) {
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) {
    fail(ATTN_ERR_INVALID, err);
    return -1;
  }
  return attn::count_pairs(gt);
}

int64_t attn_count_computed_pairs(const attn_chunk_layout* layout, int L, int D) {
  if (D != 64 && D != 128) {
    fail(ATTN_ERR_UNSUPPORTED, "unsupported head_dim " + std::to_string(D));
    return -1;
  }
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) {
    fail(ATTN_ERR_INVALID, err);
    return -1;
  }
  return attn::count_computed_pairs(gt, L, attn::kMfmaBr, attn::kMfmaBc);
}

int attn_query_groups(const attn_chunk_layout* layout, int L, int32_t* out, int max_groups) {
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) return fail(ATTN_ERR_INVALID, err), -1;
  if (!out || max_groups < gt.n) return fail(ATTN_ERR_INVALID, "output buffer too small"), -1;
  for (int g = 0; g < gt.n; ++g) {
    int32_t* r = out + 6 * g;
    r[0] = attn::group_q_begin(gt, g);
    r[1] = gt.q_end[g];
    r[2] = gt.a0[g]; r[3] = gt.a1[g];
    r[4] = gt.b0[g]; r[5] = gt.b1[g];
  }
  return gt.n;
}

void attn_tile_shape(int* rows_per_tile, int* keys_per_block) {
  if (rows_per_tile) *rows_per_tile = attn::kMfmaBr;
  if (keys_per_block) *keys_per_block = attn::kMfmaBc;
}

int attn_tile_plan(const attn_chunk_layout* layout, int L, int qtile, int32_t* blocks, int32_t* full, int cap) {
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) return fail(ATTN_ERR_INVALID, err), -1;
  const int br = attn::kMfmaBr, bc = attn::kMfmaBc;
  if (qtile < 0 || (int64_t)qtile * br >= L) return fail(ATTN_ERR_INVALID, "query tile out of range"), -1;
  const int q0 = qtile * br;
  const int q1 = q0 + br < L ? q0 + br : L;
  const attn::TilePlan p = attn::plan_tile(gt, q0, q1, bc);
  const int nb = attn::plan_num_blocks(p);
  if (!blocks || !full || cap < nb) return fail(ATTN_ERR_INVALID, "output buffer too small"), -1;
  for (int i = 0; i < nb; ++i) {
    blocks[i] = attn::plan_block(p, i);
    full[i] = attn::block_is_full(p, blocks[i] * bc, bc, L) ? 1 : 0;
  }
  return nb;
}

int attn_tile_order(const attn_chunk_layout* layout, int L, int zero_clean, int32_t* order, int cap) {
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) return fail(ATTN_ERR_INVALID, err), -1;
  if (zero_clean && layout->kind != ATTN_MASK_TEACHER_FORCING)
    return fail(ATTN_ERR_INVALID, "the zero-clean-tangent JVP needs a teacher-forcing layout"), -1;
  const attn::TileOrder o =
      zero_clean ? attn::make_tile_order_zero_clean(gt, L, attn::kMfmaBr, attn::kMfmaBc, L / 2)
                 : attn::make_tile_order(layout, L, attn::kMfmaBr);
  if (!order || cap < o.nt) return fail(ATTN_ERR_INVALID, "output buffer too small"), -1;
  for (int t = 0; t < o.nt; ++t) order[t] = attn::tile_of(o, t);
  return o.nt;
}

const char* attn_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
