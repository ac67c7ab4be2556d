// validate.cpp -- argument validation of the compute entry points (plain C++17, no HIP).
#include "validate.hpp"

#include <cmath>
#include <cstdint>
#include <string>

#include "layout.hpp"

namespace attn {

namespace {

thread_local std::string g_last_error;

int fail(int code, const std::string& msg) { return set_error(code, msg); }

struct Span {
  uintptr_t lo, hi;
  const char* name;
};

bool overlap(const Span& x, const Span& y) { return x.lo < y.hi && y.lo < x.hi; }

// Size limits of the kernels (after the positivity checks): the kernels address a head with
// 32-bit byte offsets and launch one work-group per tile of at least 128 rows or keys and
// (batch, head), in one grid dimension.
int check_sizes(int dtype, int B, int H, int L, int D) {
  const int64_t bh = (int64_t)B * H;
  if (bh > (int64_t)1 << 20) return fail(ATTN_ERR_INVALID, "B * H too large");
  // the kernels address a head with 32-bit byte offsets: 4 GiB per tensor and head
  const int64_t max_ld = dtype == ATTN_DTYPE_BF16 ? (int64_t)1 << 31 : (int64_t)1 << 30;
  if ((int64_t)L * D > max_ld)
    return fail(ATTN_ERR_INVALID, std::string(dtype == ATTN_DTYPE_BF16 ? "bf16 needs L * D <= 2^31" : "fp32 needs L * D <= 2^30") +
                                      " (32-bit offsets within a head), got L = " + std::to_string(L) +
                                      ", D = " + std::to_string(D));
  if (((int64_t)L + 127) / 128 * bh > INT32_MAX)
    return fail(ATTN_ERR_INVALID, "too many work-groups for one launch: ceil(L / 128) * B * H > 2^31 - 1");
  return ATTN_OK;
}

int elem_size(int dtype) { return dtype == ATTN_DTYPE_F32 ? 4 : dtype == ATTN_DTYPE_BF16 ? 2 : 0; }

}  // namespace

// Shared validation of the compute entry points; fills the launch arguments.
// kJvpZeroClean: teacher-forcing layouts only; the tangents (and dO) hold the noisy
// half, rows [L/2, L), of every (batch, head).
int prepare(Pass pass, int dtype, int B, int H, int L, int D, const void* Q, const void* K,
            const void* V, const void* dQ, const void* dK, const void* dV,
            const attn_chunk_layout* layout, float softmax_scale, void* O, void* dO, float* LSE,
            AttnArgs* args) {
  const bool jvp = pass != Pass::kFwd;
  const bool zc = pass == Pass::kJvpZeroClean;
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
  const uintptr_t align = 16;  // the kernels move tensor rows in 16-byte pieces
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
  if (!build_groups(layout, L, &args->gt, &err)) return fail(ATTN_ERR_INVALID, err);
  args->Q = Q; args->K = K; args->V = V;
  args->dQ = dQ; args->dK = dK; args->dV = dV;
  args->O = O; args->dO = dO; args->LSE = LSE;
  args->B = B; args->H = H; args->L = L;
  args->t0 = t0;
  args->scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt((float)D);
  // the bf16 forward-only kernel takes 128-row tiles, the bf16 JVP kernels 256-row tiles, the
  // fp32 kernels 128-row tiles
  if (dtype == ATTN_DTYPE_F32) {
    args->order = make_tile_order(layout, L, kF32Br);
  } else {
    const int br = pass == Pass::kFwd ? kMfmaBrFwd : kMfmaBr;
    args->order = zc ? make_tile_order_zero_clean(args->gt, L, kMfmaBr, kMfmaBc, t0)
                     : make_tile_order(layout, L, br);
  }
  return ATTN_OK;
}

int prepare_bwd(int dtype, int B, int H, int L, int D, const void* Q, const void* K, const void* V,
                const void* O, const void* gO, const float* LSE, const attn_chunk_layout* layout,
                float softmax_scale, void* gQ, void* gK, void* gV, float* Delta, BwdArgs* qa,
                BwdArgs* ka) {
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
  const uintptr_t align = 16;  // the kernels move tensor rows in 16-byte pieces
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
  if (!build_groups(layout, L, &qa->gt, &err)) return fail(ATTN_ERR_INVALID, err);
  ka->gt = qa->gt;  // the key-tile pass plans its tiles over the same query-group table
  qa->Q = ka->Q = Q; qa->K = ka->K = K; qa->V = ka->V = V;
  qa->O = ka->O = O; qa->gO = ka->gO = gO; qa->LSE = ka->LSE = LSE;
  qa->gQ = ka->gQ = gQ; qa->gK = ka->gK = gK; qa->gV = ka->gV = gV; qa->Delta = ka->Delta = Delta;
  qa->B = ka->B = B; qa->H = ka->H = H; qa->L = ka->L = L;
  qa->scale = ka->scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt((float)D);
  qa->order = make_tile_order(layout, L, dtype == ATTN_DTYPE_F32 ? kF32Br : kMfmaBr);
  // key tiles: for the built-in layouts the work per key tile falls with the key index
  // (earlier keys are seen by more queries), so the natural order is heaviest first
  ka->order = TileOrder{};
  ka->order.mode = 0;
  ka->order.nt = (L + kBwdKeysPerTile - 1) / kBwdKeysPerTile;
  ka->order.split = ka->order.nt;
  ka->order.first = -1;
  return ATTN_OK;
}

int set_error(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

const char* last_error_message() { return g_last_error.c_str(); }

}  // namespace attn
