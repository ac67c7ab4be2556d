// attn_simt.hip -- fp32 masked attention forward + JVP, exact-path kernel.
//
// The fp32 entry points must meet a much tighter tolerance than bf16 matrix
// cores allow, so this kernel keeps every operand and product in fp32.  One
// wave owns one query row; lanes split head_dim (1 or 2 elements per lane) and
// the score and score tangent of each admissible key are reduced across the
// wave.  Keys are visited one at a time over the row's own key ranges (exact
// skipping), with the online recurrence of the paper's Algorithm 1 (App. B) at
// a block size of one key: running max m, normaliser l, accumulators O,
// T = A + B and r, epilogue O / l, LSE = m + ln l, dO = (T - r O) / l.
// When the tangents are zero below row t0 (and stored from row t0 on), rows
// below t0 skip the tangent work and keys below t0 skip their dK, dV terms.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace attn {
namespace {

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

template <int D, bool JVP>
__global__ __launch_bounds__(64 * kSimtRowsPerBlock) void attn_simt_kernel(const AttnArgs a) {
  constexpr int E = D / 64;  // elements per lane
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kSimtRowsPerBlock + (threadIdx.x >> 6);
  const int bh = blockIdx.y;
  const int L = a.L;
  if (row >= L) return;  // whole wave leaves; no barriers below

  // tangent rows are [t0, L) (t0 = 0 unless the rows below t0 carry zero tangents,
  // which are then neither stored nor read)
  const int t0 = a.t0;
  const size_t head = (size_t)bh * L * D;
  const size_t thead = (size_t)bh * (L - t0) * D;
  const float* Q = (const float*)a.Q + head;
  const float* K = (const float*)a.K + head;
  const float* V = (const float*)a.V + head;
  const float* dQ = (const float*)a.dQ + thead;  // tangent row x - t0 of sequence row x
  const float* dK = (const float*)a.dK + thead;
  const float* dV = (const float*)a.dV + thead;

  const int g = find_group(a.gt, row);
  const int r_first = a.gt.r_begin[g], r_last = a.gt.r_begin[g + 1];  // the group's key ranges
  const bool row_tan = JVP && row >= t0;

  float q[E], dq[E], o[E], t[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    q[e] = Q[(size_t)row * D + lane + 64 * e];
    dq[e] = row_tan ? dQ[(size_t)(row - t0) * D + lane + 64 * e] : 0.f;
    o[e] = 0.f;
    t[e] = 0.f;
  }
  float m = -INFINITY, l = 0.f, r = 0.f;
  const float sc = a.scale;

  for (int ri = r_first; ri < r_last; ++ri) {
    for (int k = a.gt.k[2 * ri]; k < a.gt.k[2 * ri + 1]; ++k) {
      const bool key_tan = JVP && k >= t0;  // uniform across the wave
      float s = 0.f, ds = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float kv = K[(size_t)k * D + lane + 64 * e];
        s += q[e] * kv;
        if (JVP) ds += dq[e] * kv + (key_tan ? q[e] * dK[(size_t)(k - t0) * D + lane + 64 * e] : 0.f);
      }
      s = wave_sum(s) * sc;
      if (JVP) ds = wave_sum(ds) * sc;
      const float mnew = fmaxf(m, s);
      const float alpha = expf(m - mnew);  // m = -inf on the first key gives 0
      const float p = expf(s - mnew);
      l = l * alpha + p;
      if (JVP) r = r * alpha + p * ds;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float vv = V[(size_t)k * D + lane + 64 * e];
        o[e] = o[e] * alpha + p * vv;
        if (JVP) t[e] = t[e] * alpha + (key_tan ? p * dV[(size_t)(k - t0) * D + lane + 64 * e] : 0.f) + p * ds * vv;
      }
      m = mnew;
    }
  }

  const float inv = l > 0.f ? 1.f / l : 0.f;
  float* O = (float*)a.O + head + (size_t)row * D;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const float on = o[e] * inv;
    O[lane + 64 * e] = on;
    if (row_tan) ((float*)a.dO + thead)[(size_t)(row - t0) * D + lane + 64 * e] = (t[e] - r * on) * inv;
  }
  if (lane == 0) a.LSE[(size_t)bh * L + row] = l > 0.f ? m + logf(l) : -INFINITY;
}

}  // namespace

hipError_t launch_simt_f32(const AttnArgs& a, int D, Pass pass, hipStream_t stream) {
  const dim3 grid((unsigned)((a.L + kSimtRowsPerBlock - 1) / kSimtRowsPerBlock), (unsigned)(a.B * a.H));
  const dim3 block(64 * kSimtRowsPerBlock);
  const bool jvp = pass != Pass::kFwd;  // a.t0 selects the rows that carry tangents
  if (D == 128) {
    if (jvp) hipLaunchKernelGGL((attn_simt_kernel<128, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_simt_kernel<128, false>), grid, block, 0, stream, a);
  } else {
    if (jvp) hipLaunchKernelGGL((attn_simt_kernel<64, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_simt_kernel<64, false>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace attn
