// attn_f32.hip -- fp32 masked attention forward + JVP on gfx950 matrix cores.
//
// The fp32 entry points keep every product and sum in fp32 (their bar is 1e-4 relative),
// so this path uses fp32 matrix instructions: fp32 operands, fp32 accumulation.  The
// recurrence is the paper's Algorithm 1 (App. B) as in the bf16 kernel: running max m,
// normaliser l, O, one tangent accumulator T = A + B and r = sum rowsum(P~ o dS), with the
// epilogue O / l, LSE = m + ln l, dO = (T - r O) / l; P~ and H~ stay fp32.
//
// One work-group of 8 waves (two per SIMD) owns a query tile of 128 rows, 16 per wave,
// and streams the key blocks of its plan (schedule.hpp) through LDS, 32 keys at a time, in
// two stages (block k+1 loads while block k is used).  The matrix instruction is
// v_mfma_f32_16x16x4_f32 (16 x 16 outputs, 4 contraction elements, one per 16-lane group
// g = l/16; lane l supplies A[l%16][g] and B[g][l%16] and holds D[4 g + j][l%16], j = 0..3).
// Scores are computed transposed, S^T = K Q^T and dS^T = dK Q^T + K dQ^T, per 16-key half
// kt of the block, so that a lane owns one query (l%16) and keys 16 kt + 4 g + j:
//   scores: step s (0 .. D/4-1) contracts d = g D/4 + s, so a lane keeps its query's
//           quarter row of Q (and dQ) as B operands in registers and reads 4 consecutive d
//           of its key row per 16-byte LDS read (4 steps);
//   output: step (kt, j) contracts key 16 kt + 4 g + j of group g -- the key of the lane's
//           own accumulator slot (kt, j), so P~^T and H~^T are B operands as they are;
//           O^T tile dt (D/16 of them) holds d = 4 m + dt%4 + 64 (dt/4) in its row m, so a
//           lane reads whole 16-byte chunks m and m + 16 of one V row.
// Per wave and block (D = 128): 64 (S) + 128 (dS) + 64 (O) + 128 (T) MFMAs of 2048 flop =
// 12 D flop per (query, key) pair.  Registers per wave: Q and dQ quarters (2 x D/4), O^T
// and T^T (2 x D/4), scores 16: two waves fit a SIMD.
//
// LDS rows of D floats are stored with their 16-byte chunks XOR-swizzled by the row's low
// four bits: the 16 lanes of a pass of a score-operand read (16 rows, one chunk) and of
// an output-operand read (one row, 16 chunks) then hit distinct banks.
//
// Zero clean tangents (t0 > 0, the TF-sCM case): the tangents hold rows [t0, L) only; key
// blocks below t0 get their tangent rows cleared in LDS and queries below t0 a zero dQ, so
// the result equals the dense JVP of the zero-padded tangents; dO is stored for rows >= t0.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "kernels.hpp"
#include "mfma_common.hpp"

namespace attn {
namespace {

using namespace dev;

constexpr int BC = 32;       // keys per block
constexpr int NW = 8;        // waves per work-group (two per SIMD)
constexpr int QW = 16;       // query rows per wave
constexpr int BR = QW * NW;  // query rows per work-group
constexpr float kLazyF = 8.0f;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) f32x4 lds_f32x4;

template <int D>
struct FGeo {
  static constexpr int ROWB = 4 * D;        // bytes per LDS row
  static constexpr int NCH = D / 4;         // 16-byte chunks per row
  static constexpr int TILEB = BC * ROWB;   // one K, V, dK or dV tile
  static constexpr int DT = D / 16;         // O^T / T^T tiles of 16 d
  static constexpr int QS = D / 4;          // score steps (Q quarter row per lane)
  static constexpr int IPT = TILEB / 1024;  // 1 KiB direct loads per tile
};

__device__ __forceinline__ int fswz(int row) { return row & 15; }

template <int D>
__device__ __forceinline__ unsigned foff(int row, int chunk) {
  return (unsigned)(row * FGeo<D>::ROWB + ((chunk ^ fswz(row)) << 4));
}

__device__ __forceinline__ f32x4 mfma16(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// value of lane l ^ 16 and l ^ 32 (row statistics: a query's keys lie in four lanes)
__device__ __forceinline__ float xor16(float x) { return __shfl_xor(x, 16, 64); }

template <int D, bool JVP>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_f32_kernel(const AttnArgs a) {
  using G = FGeo<D>;
  constexpr int TB = G::TILEB;
  constexpr int NT = JVP ? 4 : 2;   // tiles per stage: K, V (, dK, dV)
  constexpr int SB = NT * TB;
  __shared__ __attribute__((aligned(1024))) char stages[2 * SB];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int g = lane >> 4;      // contraction group of the lane
  const int c16 = lane & 15;
  const int L = a.L;
  const int t0 = a.t0;
  const int Lt = L - t0;

  const TileSlot sl = slot_of(blockIdx.x, a.B * a.H, a.order.nt, kHeadGroup);
  const int bh = sl.bh;
  const int qtile = tile_of(a.order, sl.pos);
  const size_t head = (size_t)bh * L * D;
  const size_t thead = (size_t)bh * Lt * D;
  const float* __restrict__ Qg = (const float*)a.Q + head;
  const float* __restrict__ Kg = (const float*)a.K + head;
  const float* __restrict__ Vg = (const float*)a.V + head;
  const float* __restrict__ dQg = (const float*)a.dQ + thead;
  const float* __restrict__ dKg = (const float*)a.dK + thead;
  const float* __restrict__ dVg = (const float*)a.dV + thead;

  const int q0 = qtile * BR;
  const int q1 = q0 + BR < L ? q0 + BR : L;
  const TilePlan plan = plan_tile(a.gt, q0, q1, BC);
  const int nblk = plan_num_blocks(plan);

  const int row = q0 + wave * QW + c16;
  const int wrow0 = imin(q0 + wave * QW, L - 1);
  const int wg0 = find_group(a.gt, wrow0), wg1 = find_group(a.gt, imin(wrow0 + QW - 1, L - 1));

  // Q (and dQ) quarter rows as B operands: lane l holds d = g D/4 + s, s = 0 .. D/4-1
  float qv[G::QS], dqv[JVP ? G::QS : 1];
  {
    const float* qp = Qg + (size_t)imin(row, L - 1) * D + g * G::QS;
#pragma unroll
    for (int s = 0; s < G::QS; s += 4) {
      const f32x4 v = *(const f32x4*)(qp + s);
#pragma unroll
      for (int e = 0; e < 4; ++e) qv[s + e] = v[e];
    }
    if constexpr (JVP) {
      const bool tan = row >= t0 && row < L;  // rows below t0 carry a zero tangent
      const float* dp = dQg + (size_t)(tan ? row - t0 : 0) * D + g * G::QS;
#pragma unroll
      for (int s = 0; s < G::QS; s += 4) {
        const f32x4 v = *(const f32x4*)(dp + s);
#pragma unroll
        for (int e = 0; e < 4; ++e) dqv[s + e] = tan ? v[e] : 0.f;
      }
    }
  }

  // global -> LDS: one 1 KiB direct load per wave instruction; lane l lands at byte 16 l,
  // i.e. physical row 16 l / ROWB, physical chunk p, and fetches the logical chunk
  // p ^ swizzle(row).  Rows past the end are clamped (finite data; masked or unstored).
  constexpr int RPI = 1024 / G::ROWB;
  const int dma_r = (lane * 16) / G::ROWB;
  const int dma_p = ((lane * 16) % G::ROWB) >> 4;
  auto dma_tile = [&](const float* src, int row0, int rmax, unsigned dst) {
#pragma unroll
    for (int j0 = 0; j0 < G::IPT; j0 += NW) {
      const int j = j0 + wave;
      if (G::IPT % NW == 0 || j < G::IPT) {
        const int rr = j * RPI + dma_r;
        const unsigned grow = (unsigned)imin(imax(row0 + rr, 0), rmax);
        const unsigned off = (grow * D + (unsigned)((dma_p ^ fswz(rr)) * 4)) * 4u;
        lds_load16(src, off, dst + (unsigned)(j * 1024));
      }
    }
  };
  const unsigned st_lds = __builtin_amdgcn_readfirstlane(lds_addr(stages));
  auto dma_block = [&](int kb, unsigned st) {
    const int k0 = kb * BC;
    dma_tile(Kg, k0, L - 1, st);
    dma_tile(Vg, k0, L - 1, st + TB);
    if constexpr (JVP) {
      dma_tile(dKg, k0 - t0, Lt - 1, st + 2 * TB);
      dma_tile(dVg, k0 - t0, Lt - 1, st + 3 * TB);
    }
  };

  f32x4 oacc[G::DT], tacc[JVP ? G::DT : 1];
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt) {
    oacc[dt] = f32x4{};
    if constexpr (JVP) tacc[dt] = f32x4{};
  }
  float m = -INFINITY, lsum = 0.f, rsum = 0.f;
  const float c2 = a.scale * kLog2e;
  const float sc = a.scale;

  if (nblk > 0) dma_block(plan_block(plan, 0), st_lds);
  __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0): also the Q / dQ loads above
  __syncthreads();

  for (int it = 0; it < nblk; ++it) {
    const unsigned cur = st_lds + (unsigned)((it & 1) * SB);
    if (it + 1 < nblk) dma_block(plan_block(plan, it + 1), st_lds + (unsigned)(((it + 1) & 1) * SB));
    const int k0 = plan_block(plan, it) * BC;
    if constexpr (JVP) {
      if (k0 < t0) {
        // keys below t0 carry a zero tangent: clear those rows of the dK, dV tiles
        const int nz = imin(t0 - k0, BC) * G::NCH;
        for (int c = tid; c < nz; c += 64 * NW) {
          *(lds_f32x4*)(uintptr_t)(cur + 2 * TB + 16 * c) = f32x4{};
          *(lds_f32x4*)(uintptr_t)(cur + 3 * TB + 16 * c) = f32x4{};
        }
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      }
    }

    // ---- scores and score tangents (transposed) of the two 16-key halves; 4 steps per
    // 16-byte operand read, each read one group ahead of its MFMAs (order pinned with
    // scheduling fences)
    f32x4 S[2] = {f32x4{}, f32x4{}}, dS[2] = {f32x4{}, f32x4{}};
    {
      constexpr int NU = G::QS / 4;  // reads per key half
      f32x4 kv[2][2], dkv[2][2];
      auto read = [&](int u) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const unsigned o = foff<D>(16 * kt + c16, g * (G::NCH / 4) + u);
          kv[u & 1][kt] = *(lds_f32x4*)(uintptr_t)(cur + o);
          if constexpr (JVP) dkv[u & 1][kt] = *(lds_f32x4*)(uintptr_t)(cur + 2 * TB + o);
        }
      };
      read(0);
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        if (u + 1 < NU) read(u + 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int kt = 0; kt < 2; ++kt) {
            S[kt] = mfma16(kv[u & 1][kt][e], qv[4 * u + e], S[kt]);
            if constexpr (JVP) {
              dS[kt] = mfma16(dkv[u & 1][kt][e], qv[4 * u + e], dS[kt]);
              dS[kt] = mfma16(kv[u & 1][kt][e], dqv[4 * u + e], dS[kt]);
            }
          }
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // ---- mask (blocks not admissible for every row of the tile); slot (kt, j) holds key
    // k0 + 16 kt + 4 g + j
    float sv[8], dsv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      sv[i] = S[i >> 2][i & 3];
      dsv[i] = JVP ? dS[i >> 2][i & 3] : 0.f;
    }
    if (!block_is_full(plan, k0, BC, L)) {
      const uint32_t bits = row_bits(a.gt, wg0, wg1, row, k0) >> (4 * g);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const bool ok = (bits >> (16 * (i >> 2) + (i & 3))) & 1u;
        sv[i] = ok ? sv[i] : -INFINITY;
        dsv[i] = ok ? dsv[i] : 0.f;
      }
    }

    // ---- online softmax; the reference max moves (and the accumulators are rescaled)
    // only when a row's block max exceeds it by more than kLazyF (log2 units)
    float mloc = sv[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mloc = fmaxf(mloc, sv[i]);
    mloc *= c2;
    if (__ballot(mloc > m + kLazyF) != 0) {
      float mx = fmaxf(mloc, xor16(mloc));
      mx = fmaxf(mx, xor32(mx));
      const bool up = mx > m + kLazyF;
      const float mnew = up ? mx : m;
      const float alpha = up ? __builtin_amdgcn_exp2f(m - mnew) : 1.f;
      lsum *= alpha;
      rsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < G::DT; ++dt) {
        oacc[dt] *= alpha;
        if constexpr (JVP) tacc[dt] *= alpha;
      }
      m = mnew;
    }
    const float mneg = m == -INFINITY ? 0.f : -m;
    float p[8], h[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      p[i] = __builtin_amdgcn_exp2f(fmaf(sv[i], c2, mneg));
      lsum += p[i];
      if constexpr (JVP) {
        h[i] = p[i] * (dsv[i] * sc);
        rsum += h[i];
      }
    }

    // ---- O^T += V^T P~^T ; T^T += dV^T P~^T + V^T H~^T, step (kt, j) = slot i = 4 kt + j;
    // the V (dV) row of a step is read one step ahead
    {
      constexpr int NCR = G::DT / 4;  // 16-byte reads per row and step (chunks m, m + 16)
      f32x4 vv[2][NCR], dvv[2][NCR];
      auto read = [&](int i) {
        const int key = 16 * (i >> 2) + 4 * g + (i & 3);
#pragma unroll
        for (int c = 0; c < NCR; ++c) {
          const unsigned o = foff<D>(key, c16 + 16 * c);
          vv[i & 1][c] = *(lds_f32x4*)(uintptr_t)(cur + TB + o);
          if constexpr (JVP) dvv[i & 1][c] = *(lds_f32x4*)(uintptr_t)(cur + 3 * TB + o);
        }
      };
      read(0);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if (i + 1 < 8) read(i + 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int dt = 0; dt < G::DT; ++dt) {
          const float v = vv[i & 1][dt >> 2][dt & 3];
          oacc[dt] = mfma16(v, p[i], oacc[dt]);
          if constexpr (JVP) {
            tacc[dt] = mfma16(dvv[i & 1][dt >> 2][dt & 3], p[i], tacc[dt]);
            tacc[dt] = mfma16(v, h[i], tacc[dt]);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // every own load of block it+1 landed, every LDS read of block it returned
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  }

  // ---- epilogue: lane holds query l%16; tile dt slot j holds d = 4 m + dt%4 + 64 (dt/4)
  // with m = 4 g + j
  float l_tot = lsum + xor16(lsum);
  l_tot += xor32(l_tot);
  float r_tot = 0.f;
  if constexpr (JVP) {
    r_tot = rsum + xor16(rsum);
    r_tot += xor32(r_tot);
  }
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (row < L) {
    float* Og = (float*)a.O + head + (size_t)row * D;
    float* dOg = (float*)a.dO + thead + (size_t)imax(row - t0, 0) * D;
    const bool store_do = JVP && row >= t0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int mrow = 4 * g + j;
#pragma unroll
      for (int c = 0; c < G::DT / 4; ++c) {
        f32x4 ov, dov;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          ov[e] = oacc[4 * c + e][j] * inv;
          if constexpr (JVP) dov[e] = (tacc[4 * c + e][j] - r_tot * ov[e]) * inv;
        }
        *(f32x4*)(Og + 4 * mrow + 64 * c) = ov;
        if constexpr (JVP) {
          if (store_do) *(f32x4*)(dOg + 4 * mrow + 64 * c) = dov;
        }
      }
    }
    if (g == 0) a.LSE[(size_t)bh * L + row] = l_tot > 0.f ? (m + __log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

}  // namespace

hipError_t launch_mfma_f32(const AttnArgs& a, int D, Pass pass, hipStream_t stream) {
  const dim3 grid((unsigned)(a.order.nt * a.B * a.H));
  const dim3 block(64 * NW);
  const bool jvp = pass != Pass::kFwd;  // a.t0 selects the rows that carry tangents
  if (D == 128) {
    if (jvp) hipLaunchKernelGGL((attn_f32_kernel<128, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_f32_kernel<128, false>), grid, block, 0, stream, a);
  } else {
    if (jvp) hipLaunchKernelGGL((attn_f32_kernel<64, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_f32_kernel<64, false>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace attn
