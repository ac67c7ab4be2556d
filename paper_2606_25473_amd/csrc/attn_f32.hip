// attn_f32.hip -- fp32 masked attention on gfx950 matrix cores: forward, JVP (dense and
// with zero clean tangents) and the two backward passes (after the forward kernel below).
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
// the host sizes the grids and tile orders with these
static_assert(BR == kF32Br && BR == kBwdKeysPerTile, "fp32 tiles must match the host's tile sizes");
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

// Rows [row0, row0 + 32) of a [rows, D] fp32 tensor (rows clamped to [0, rmax]: finite
// data that the kernels mask or never store) into the swizzled LDS tile at dst, by 1 KiB
// direct loads.  Lane l of a load lands at byte 16 l, i.e. physical row 16 l / ROWB and
// physical chunk p, and fetches the logical chunk p ^ swizzle(row).  Load j is issued by
// wave j % NW.
template <int D>
__device__ __forceinline__ void dma_tile(const float* src, int row0, int rmax, unsigned dst, int wave,
                                         int lane) {
  using G = FGeo<D>;
  constexpr int RPI = 1024 / G::ROWB;
  const int r = (lane * 16) / G::ROWB;
  const int p = ((lane * 16) % G::ROWB) >> 4;
#pragma unroll
  for (int j0 = 0; j0 < G::IPT; j0 += NW) {
    const int j = j0 + wave;
    if (G::IPT % NW == 0 || j < G::IPT) {
      const int rr = j * RPI + r;
      const unsigned grow = (unsigned)imin(imax(row0 + rr, 0), rmax);
      const unsigned off = (grow * D + (unsigned)((p ^ fswz(rr)) * 4)) * 4u;
      lds_load16(src, off, dst + (unsigned)(j * 1024));
    }
  }
}

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

  const unsigned st_lds = __builtin_amdgcn_readfirstlane(lds_addr(stages));
  auto dma_block = [&](int kb, unsigned st) {
    const int k0 = kb * BC;
    dma_tile<D>(Kg, k0, L - 1, st, wave, lane);
    dma_tile<D>(Vg, k0, L - 1, st + TB, wave, lane);
    if constexpr (JVP) {
      dma_tile<D>(dKg, k0 - t0, Lt - 1, st + 2 * TB, wave, lane);
      dma_tile<D>(dVg, k0 - t0, Lt - 1, st + 3 * TB, wave, lane);
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

// ---------------------------------------------------------------- backward
//
// Reverse mode for a cotangent gO of O, P recomputed from the saved LSE:
//   Delta = rowsum(gO o O), gP = gO V^T, gS = P o (gP - Delta),
//   gQ = s gS K, gK = s gS^T Q, gV = P^T gO,
// in two deterministic passes with the geometry of the forward (no atomics).

// Query-tile pass: a work-group owns 128 query rows (16 per wave), computes Delta for
// them, and streams the key blocks of its plan (K, V tiles): S^T = K Q^T and
// gP^T = V gO^T with the lane's quarter rows of Q and gO as B operands, then
// gQ^T += K^T gS^T with gS^T as B operand as it stands (the output pattern of the forward).
// 6 D flop per pair of matrix work.
template <int D>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_f32_bwd_dq_kernel(const BwdArgs a) {
  using G = FGeo<D>;
  constexpr int TB = G::TILEB;
  constexpr int SB = 2 * TB;  // stage: K, V tiles
  __shared__ __attribute__((aligned(1024))) char stages[2 * SB];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int g = lane >> 4;
  const int c16 = lane & 15;
  const int L = a.L;

  const TileSlot sl = slot_of(blockIdx.x, a.B * a.H, a.order.nt, kHeadGroup);
  const int bh = sl.bh;
  const int qtile = tile_of(a.order, sl.pos);
  const size_t head = (size_t)bh * L * D;
  const float* __restrict__ Qg = (const float*)a.Q + head;
  const float* __restrict__ Kg = (const float*)a.K + head;
  const float* __restrict__ Vg = (const float*)a.V + head;
  const float* __restrict__ Og = (const float*)a.O + head;
  const float* __restrict__ gOg = (const float*)a.gO + head;

  const int q0 = qtile * BR;
  const int q1 = q0 + BR < L ? q0 + BR : L;
  const TilePlan plan = plan_tile(a.gt, q0, q1, BC);
  const int nblk = plan_num_blocks(plan);

  const int row = q0 + wave * QW + c16;
  const int rowc = imin(row, L - 1);
  const int wrow0 = imin(q0 + wave * QW, L - 1);
  const int wg0 = find_group(a.gt, wrow0), wg1 = find_group(a.gt, imin(wrow0 + QW - 1, L - 1));

  // quarter rows d = g D/4 + s of Q and gO; Delta from the same quarters of gO and O
  float qv[G::QS], gov[G::QS];
  float dpart = 0.f;
  {
    const size_t o = (size_t)rowc * D + g * G::QS;
#pragma unroll
    for (int s = 0; s < G::QS; s += 4) {
      const f32x4 vq = *(const f32x4*)(Qg + o + s);
      const f32x4 vg = *(const f32x4*)(gOg + o + s);
      const f32x4 vo = *(const f32x4*)(Og + o + s);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        qv[s + e] = vq[e];
        gov[s + e] = vg[e];
        dpart = fmaf(vg[e], vo[e], dpart);
      }
    }
  }
  float delta = dpart + xor16(dpart);
  delta += xor32(delta);
  // LSE in log2 units.  A row without admissible keys has LSE = -inf: exp2 then gives
  // +inf, which the mask replaces by 0 (such a row makes no block of its tile full).
  const float lse2 = a.LSE[(size_t)bh * L + rowc] * kLog2e;
  const float c2 = a.scale * kLog2e;

  const unsigned st_lds = __builtin_amdgcn_readfirstlane(lds_addr(stages));
  auto dma_block = [&](int kb, unsigned st) {
    dma_tile<D>(Kg, kb * BC, L - 1, st, wave, lane);
    dma_tile<D>(Vg, kb * BC, L - 1, st + TB, wave, lane);
  };

  f32x4 gq[G::DT];
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt) gq[dt] = f32x4{};

  if (nblk > 0) dma_block(plan_block(plan, 0), st_lds);
  __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0): also the operand loads above
  __syncthreads();

  for (int it = 0; it < nblk; ++it) {
    const unsigned cur = st_lds + (unsigned)((it & 1) * SB);
    if (it + 1 < nblk) dma_block(plan_block(plan, it + 1), st_lds + (unsigned)(((it + 1) & 1) * SB));
    const int k0 = plan_block(plan, it) * BC;

    // S^T = K Q^T and gP^T = V gO^T per 16-key half; operands read one group ahead
    f32x4 S[2] = {f32x4{}, f32x4{}}, GP[2] = {f32x4{}, f32x4{}};
    {
      constexpr int NU = G::QS / 4;
      f32x4 kc[2][2], vc[2][2];
      auto read = [&](int u) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const unsigned o = foff<D>(16 * kt + c16, g * (G::NCH / 4) + u);
          kc[u & 1][kt] = *(lds_f32x4*)(uintptr_t)(cur + o);
          vc[u & 1][kt] = *(lds_f32x4*)(uintptr_t)(cur + TB + o);
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
            S[kt] = mfma16(kc[u & 1][kt][e], qv[4 * u + e], S[kt]);
            GP[kt] = mfma16(vc[u & 1][kt][e], gov[4 * u + e], GP[kt]);
          }
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // P and gS; slot i = 4 kt + j holds key k0 + 16 kt + 4 g + j
    float p[8], gs[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) p[i] = __builtin_amdgcn_exp2f(fmaf(S[i >> 2][i & 3], c2, -lse2));
    if (!block_is_full(plan, k0, BC, L)) {
      const uint32_t bits = row_bits(a.gt, wg0, wg1, row, k0) >> (4 * g);
#pragma unroll
      for (int i = 0; i < 8; ++i) p[i] = ((bits >> (16 * (i >> 2) + (i & 3))) & 1u) ? p[i] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) gs[i] = p[i] * (GP[i >> 2][i & 3] - delta);

    // gQ^T += K^T gS^T: step i contracts key 16 kt + 4 g + j of group g (the lane's slot i)
    {
      constexpr int NCR = G::DT / 4;
      f32x4 kr[2][NCR];
      auto read = [&](int i) {
        const int key = 16 * (i >> 2) + 4 * g + (i & 3);
#pragma unroll
        for (int c = 0; c < NCR; ++c) kr[i & 1][c] = *(lds_f32x4*)(uintptr_t)(cur + foff<D>(key, c16 + 16 * c));
      };
      read(0);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if (i + 1 < 8) read(i + 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int dt = 0; dt < G::DT; ++dt) gq[dt] = mfma16(kr[i & 1][dt >> 2][dt & 3], gs[i], gq[dt]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  }

  // gQ = s gQ^T^T: tile dt slot j holds d = 4 m + dt%4 + 64 (dt/4), m = 4 g + j
  if (row < L) {
    float* gQg = (float*)a.gQ + head + (size_t)row * D;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int c = 0; c < G::DT / 4; ++c) {
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = a.scale * gq[4 * c + e][j];
        *(f32x4*)(gQg + 4 * (4 * g + j) + 64 * c) = v;
      }
    if (g == 0) a.Delta[(size_t)bh * L + row] = delta;
  }
}

// Key-tile pass: a work-group owns 128 keys (16 per wave) and streams the 32-row query
// blocks of the groups that admit some of them (the query-group table's key-tile plan):
// Q, gO tiles and the blocks' LSE and Delta.  S = Q K^T and gP = gO V^T with the lane's
// quarter rows of K and V as B operands put one key in each lane (16 queries per half),
// so gV^T += gO^T P and gK^T += Q^T gS take P and gS as B operands as they stand.
// 8 D flop per pair of matrix work.
template <int D>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_f32_bwd_dkdv_kernel(const BwdArgs a) {
  using G = FGeo<D>;
  constexpr int TB = G::TILEB;
  constexpr int SB = 2 * TB + 2 * 256;  // stage: Q, gO tiles, LSE and Delta (64 floats each)
  static_assert(SB % 512 == 0, "stages start on whole LDS rows");
  __shared__ __attribute__((aligned(1024))) char stages[2 * SB];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int g = lane >> 4;
  const int c16 = lane & 15;
  const int L = a.L;

  const TileSlot sl = slot_of(blockIdx.x, a.B * a.H, a.order.nt, kHeadGroupWide);
  const int bh = sl.bh;
  const int ktile = tile_of(a.order, sl.pos);
  const size_t head = (size_t)bh * L * D;
  const float* __restrict__ Qg = (const float*)a.Q + head;
  const float* __restrict__ Kg = (const float*)a.K + head;
  const float* __restrict__ Vg = (const float*)a.V + head;
  const float* __restrict__ gOg = (const float*)a.gO + head;
  const float* __restrict__ LSEg = a.LSE + (size_t)bh * L;
  const float* __restrict__ Dg = a.Delta + (size_t)bh * L;

  const int k0 = ktile * BR;
  const int k1 = k0 + BR < L ? k0 + BR : L;
  const TilePlan plan = plan_key_tile(a.gt, k0, k1, BC);
  const int nblk = plan_num_blocks(plan);

  const int key = k0 + wave * QW + c16;
  const int keyc = imin(key, L - 1);
  float kv[G::QS], vv[G::QS];
  {
    const size_t o = (size_t)keyc * D + g * G::QS;
#pragma unroll
    for (int s = 0; s < G::QS; s += 4) {
      const f32x4 vk = *(const f32x4*)(Kg + o + s);
      const f32x4 vw = *(const f32x4*)(Vg + o + s);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        kv[s + e] = vk[e];
        vv[s + e] = vw[e];
      }
    }
  }
  const float c2 = a.scale * kLog2e;

  const unsigned st_lds = __builtin_amdgcn_readfirstlane(lds_addr(stages));
  auto dma_block = [&](int qb, unsigned st) {
    const int r0 = qb * BC;
    dma_tile<D>(Qg, r0, L - 1, st, wave, lane);
    dma_tile<D>(gOg, r0, L - 1, st + TB, wave, lane);
    // 64 values each (rows past the block: clamped, never read)
    const unsigned roff = (unsigned)imin(r0 + lane, L - 1) * 4u;
    if (wave == NW - 2) lds_load4(LSEg, roff, st + 2 * TB);
    if (wave == NW - 1) lds_load4(Dg, roff, st + 2 * TB + 256);
  };

  f32x4 gk[G::DT], gv[G::DT];
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt) {
    gk[dt] = f32x4{};
    gv[dt] = f32x4{};
  }

  if (nblk > 0) dma_block(plan_block(plan, 0), st_lds);
  __builtin_amdgcn_s_waitcnt(0xF70);
  __syncthreads();

  for (int it = 0; it < nblk; ++it) {
    const unsigned cur = st_lds + (unsigned)((it & 1) * SB);
    if (it + 1 < nblk) dma_block(plan_block(plan, it + 1), st_lds + (unsigned)(((it + 1) & 1) * SB));
    const int q0b = plan_block(plan, it) * BC;

    // S = Q K^T and gP = gO V^T per 16-row half qt: the lane holds rows 16 qt + 4 g + j
    // of its key
    f32x4 S[2] = {f32x4{}, f32x4{}}, GP[2] = {f32x4{}, f32x4{}};
    {
      constexpr int NU = G::QS / 4;
      f32x4 qc[2][2], gc[2][2];
      auto read = [&](int u) {
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
          const unsigned o = foff<D>(16 * qt + c16, g * (G::NCH / 4) + u);
          qc[u & 1][qt] = *(lds_f32x4*)(uintptr_t)(cur + o);
          gc[u & 1][qt] = *(lds_f32x4*)(uintptr_t)(cur + TB + o);
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
          for (int qt = 0; qt < 2; ++qt) {
            S[qt] = mfma16(qc[u & 1][qt][e], kv[4 * u + e], S[qt]);
            GP[qt] = mfma16(gc[u & 1][qt][e], vv[4 * u + e], GP[qt]);
          }
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // LSE and Delta of the lane's rows 16 qt + 4 g .. + 3; P and gS
    float p[8], gs[8];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      const f32x4 lv = *(lds_f32x4*)(uintptr_t)(cur + 2 * TB + 4 * (16 * qt + 4 * g));
      const f32x4 dv = *(lds_f32x4*)(uintptr_t)(cur + 2 * TB + 256 + 4 * (16 * qt + 4 * g));
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = 4 * qt + j;
        p[i] = __builtin_amdgcn_exp2f(fmaf(S[qt][j], c2, -lv[j] * kLog2e));
        gs[i] = dv[j];
      }
    }
    if (!block_is_full(plan, q0b, BC, L)) {  // rows without admissible keys end up here too
      const uint32_t bits = key_bits(a.gt, key, q0b, L) >> (4 * g);
#pragma unroll
      for (int i = 0; i < 8; ++i) p[i] = ((bits >> (16 * (i >> 2) + (i & 3))) & 1u) ? p[i] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) gs[i] = p[i] * (GP[i >> 2][i & 3] - gs[i]);

    // gV^T += gO^T P and gK^T += Q^T gS: step i contracts row 16 qt + 4 g + j of group g
    {
      constexpr int NCR = G::DT / 4;
      f32x4 gr[2][NCR], qr[2][NCR];
      auto read = [&](int i) {
        const int r = 16 * (i >> 2) + 4 * g + (i & 3);
#pragma unroll
        for (int c = 0; c < NCR; ++c) {
          const unsigned o = foff<D>(r, c16 + 16 * c);
          qr[i & 1][c] = *(lds_f32x4*)(uintptr_t)(cur + o);
          gr[i & 1][c] = *(lds_f32x4*)(uintptr_t)(cur + TB + o);
        }
      };
      read(0);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if (i + 1 < 8) read(i + 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int dt = 0; dt < G::DT; ++dt) {
          gv[dt] = mfma16(gr[i & 1][dt >> 2][dt & 3], p[i], gv[dt]);
          gk[dt] = mfma16(qr[i & 1][dt >> 2][dt & 3], gs[i], gk[dt]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  }

  if (key < L) {
    float* gKg = (float*)a.gK + head + (size_t)key * D;
    float* gVg = (float*)a.gV + head + (size_t)key * D;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int c = 0; c < G::DT / 4; ++c) {
        f32x4 vk, vw;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vk[e] = a.scale * gk[4 * c + e][j];
          vw[e] = gv[4 * c + e][j];
        }
        const int d = 4 * (4 * g + j) + 64 * c;
        *(f32x4*)(gKg + d) = vk;
        *(f32x4*)(gVg + d) = vw;
      }
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

hipError_t launch_bwd_mfma_f32(const BwdArgs& qa, const BwdArgs& ka, int D, hipStream_t stream) {
  const dim3 gq((unsigned)(qa.order.nt * qa.B * qa.H)), gk((unsigned)(ka.order.nt * ka.B * ka.H));
  const dim3 block(64 * NW);
  if (D == 128) {
    hipLaunchKernelGGL((attn_f32_bwd_dq_kernel<128>), gq, block, 0, stream, qa);
    hipLaunchKernelGGL((attn_f32_bwd_dkdv_kernel<128>), gk, block, 0, stream, ka);
  } else {
    hipLaunchKernelGGL((attn_f32_bwd_dq_kernel<64>), gq, block, 0, stream, qa);
    hipLaunchKernelGGL((attn_f32_bwd_dkdv_kernel<64>), gk, block, 0, stream, ka);
  }
  return hipGetLastError();
}

}  // namespace attn
