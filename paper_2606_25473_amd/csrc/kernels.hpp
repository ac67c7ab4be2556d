// kernels.hpp -- kernel launch interface used by the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>

#include "schedule.hpp"

namespace attn {

// Arguments of one attention launch.  Everything the kernels need travels by
// value in the kernel arguments: the library holds no device memory.
struct AttnArgs {
  const void* Q;
  const void* K;
  const void* V;
  const void* dQ;   // tangents: unused by the forward-only kernels
  const void* dK;
  const void* dV;
  void* O;
  void* dO;
  float* LSE;
  int B, H, L;
  int t0;           // tangent rows are [t0, L) (dQ, dK, dV, dO hold L - t0 rows per head)
  float scale;      // softmax scale s applied to scores and score tangents
  GroupTable gt;
  TileOrder order;
};

// Arguments of one backward launch (reverse mode: gradients from the cotangent gO).
// `gt` is the query-group table for the query-tile kernels (gQ, Delta) and the
// transposed key-group table for the key-tile kernels (gK, gV).
struct BwdArgs {
  const void* Q;
  const void* K;
  const void* V;
  const void* O;
  const void* gO;
  const float* LSE;
  void* gQ;
  void* gK;
  void* gV;
  float* Delta;     // rowsum(gO o O): written by the query-tile pass, read by the key-tile pass
  int B, H, L;
  float scale;
  GroupTable gt;
  TileOrder order;
};

// bf16 MFMA kernels: query tiles of kMfmaBr rows (8 waves x 32 rows) for the JVP kernels,
// kMfmaBrFwd rows (4 waves) for the forward-only kernel; key blocks of kMfmaBc keys.
constexpr int kMfmaBr = 256;
constexpr int kMfmaBrFwd = 128;
constexpr int kMfmaBc = 32;

// fp32 exact-path kernels: one wave per query row.
constexpr int kSimtRowsPerBlock = 4;

// What a launch computes: the primal only, the JVP with tangents on every row (t0 = 0),
// or the JVP whose tangents are zero on rows [0, t0) and stored for rows [t0, L) only.
enum class Pass { kFwd, kJvp, kJvpZeroClean };

hipError_t launch_mfma_bf16(const AttnArgs& a, int D, Pass pass, hipStream_t stream);
hipError_t launch_simt_f32(const AttnArgs& a, int D, Pass pass, hipStream_t stream);

// bf16 backward: key tiles of kBwdKeysPerTile keys, query blocks of kBwdRowsPerBlock rows.
constexpr int kBwdKeysPerTile = 128;
constexpr int kBwdRowsPerBlock = 64;

// The backward is two launches on one stream: the query-tile pass (gQ and Delta, with
// `qa` holding the query-group table) and then the key-tile pass (gK and gV, with `ka`
// holding the key-group table), which reads Delta.
hipError_t launch_bwd_mfma_bf16(const BwdArgs& qa, const BwdArgs& ka, int D, hipStream_t stream);
hipError_t launch_bwd_simt_f32(const BwdArgs& qa, const BwdArgs& ka, int D, hipStream_t stream);

}  // namespace attn
