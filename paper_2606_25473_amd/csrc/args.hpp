// args.hpp -- kernel launch arguments and tile shapes (plain C++, no HIP).
//
// Everything a kernel needs travels by value in its arguments: the library holds
// no device memory.  The host validation code (validate.cpp) fills these structs
// and the launchers (kernels.hpp) pass them on.
#pragma once

#include "schedule.hpp"

namespace attn {

// Arguments of one attention launch.
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
// `gt` is the query-group table (both passes); `order` the work-group order of the
// pass's tiles (query tiles, or key tiles).
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

// The kernel-argument block stays well inside the 4 KiB a launch may carry.
static_assert(sizeof(AttnArgs) <= 3584 && sizeof(BwdArgs) <= 3584, "kernel arguments too large");

// bf16 MFMA kernels: query tiles of kMfmaBr rows (8 waves x 32 rows) for the JVP kernels,
// kMfmaBrFwd rows (4 waves) for the forward-only kernel; key blocks of kMfmaBc keys.
constexpr int kMfmaBr = 256;
constexpr int kMfmaBrFwd = 128;
constexpr int kMfmaBc = 32;

// fp32 kernels (fp32 matrix cores): query tiles of kF32Br rows (8 waves x 16) for the
// forward, the JVP and the backward's query-tile pass; the key-tile pass takes the same
// kBwdKeysPerTile keys as the bf16 one (8 waves x 16).
constexpr int kF32Br = 128;

// What a launch computes: the primal only, the JVP with tangents on every row (t0 = 0),
// or the JVP whose tangents are zero on rows [0, t0) and stored for rows [t0, L) only.
enum class Pass { kFwd, kJvp, kJvpZeroClean };

// bf16 backward: key tiles of kBwdKeysPerTile keys, query blocks of kBwdRowsPerBlock rows.
constexpr int kBwdKeysPerTile = 128;
constexpr int kBwdRowsPerBlock = 64;

}  // namespace attn
