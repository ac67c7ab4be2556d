// attn_mfma.hip -- bf16 masked attention forward + JVP on gfx950 matrix cores.
//
// One work-group of 8 waves owns a query tile of 256 rows (32 per wave) of one
// (batch, head) and streams the key blocks of its plan (schedule.hpp) through
// LDS, 32 keys at a time, with the online-softmax recurrence of the paper's
// Algorithm 1 (App. B): running max m, normaliser l, the primal accumulator O,
// one fused tangent accumulator T = A + B (only their sum enters the
// epilogue) and r = sum rowsum(P~ o dS).  Epilogue: O <- O / l,
// LSE = m + ln l, dO = (T - r O) / l.
//
// Matrix-core formulation (v_mfma_f32_32x32x16_bf16, wave64).  Each wave
// computes the TRANSPOSED score block S^T = K Q^T (32 keys x 32 queries) so that
// a lane owns one query and 16 of the 32 keys:
//   lane l -> query l%32, keys 8*(i/4) + 4*(l/32) + i%4 for accumulator slot i.
// Row statistics then need one cross-lane step (lanes l and l^32), and the
// probabilities P~^T feed the next contraction directly as the B operand,
// provided the A operand (V^T, dV^T) lists keys in the same order.  V and dV
// are stored key-major in LDS; the transposed operand comes from
// ds_read_b64_tr_b16, which returns, in each 16-lane group, lane j <- element
// j%4 of the 8-byte word addressed by lane 4e + j/4 (e = result element).
//
// Contractions per wave and 32-key block (D = 128: 48 MFMAs of 32x32x16, one per
// 16 keys x 32 d x 32 queries):
//   S^T  = K Q^T                     8       (2D flop / pair)
//   dS^T = dK Q^T + K dQ^T          16       (4D)
//   O^T += V^T P~^T                  8       (2D)
//   T^T += dV^T P~^T + V^T H~^T     16       (4D)      H~ = P~ o dS
// = 12 D flop per (query, key) pair.
//
// Numerics: bf16 operands, fp32 accumulation; exp2 with log2(e) folded into the
// score scale only (dS stays in natural units); P~ and H~ are rounded to bf16
// (round-to-nearest-even) as MFMA operands while l and r accumulate the fp32
// values.  The running max is refreshed lazily: the accumulators are rescaled
// only when a row's block max exceeds the stored max by more than kLazy (in
// log2 units), so P~ <= 2^kLazy; the result is the same function, since O, T, l
// and r always share one reference max.
//
// Three kernels come from one body: the forward only (kFwd), the JVP (kJvp) and the
// JVP with zero tangents on the clean half of a teacher-forcing sequence
// (kZeroClean); the block loop runs in lockstep (4-wave forward) or ping-pong order
// (8-wave JVP kernels), as described at the loop.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "kernels.hpp"
#include "mfma_common.hpp"

namespace attn {
namespace {

using namespace dev;

constexpr int BC = kMfmaBc;
constexpr float kLazy = 8.0f;

template <int D>
struct Geo {
  static constexpr int NCH = D / 8;               // 16-byte chunks per row
  static constexpr int ROWB = D * 2;              // bytes per LDS row (bf16)
  static constexpr int TILEB = BC * ROWB;         // bytes per LDS tile of BC keys
  static constexpr int DT = D / 32;               // 32-wide d tiles of O^T / T^T
  static constexpr int KS = D / 16;               // 16-deep k steps of the score contraction
  static constexpr int IPT = TILEB / 1024;        // 1 KiB direct-load instructions per key tile
};

// Kernel variants.  kZeroClean is the JVP of a sequence whose rows below t0 carry
// zero tangents (the clean context of the teacher-forcing sCM objective, paper
// Sec. 3.1.2, packed input tangent [0^clean, t^noisy]).  Those rows and keys then
// contribute nothing to dS or dO, so
//  - a query tile wholly below t0 runs the forward body (its dO is zero);
//  - a key block wholly below t0 drops dK Q^T and dV^T P~^T (dK = dV = 0 there);
//  - the tangent tensors (and dO) hold the rows [t0, L) only.
// A key block or query tile that straddles t0 runs the full JVP step with the
// tangent rows below t0 cleared in LDS, so that every result equals the dense JVP
// of the zero-padded tangents.
enum { kFwd = 0, kJvp = 1, kZeroClean = 2 };

template <bool B>
struct Tag {
  static constexpr bool value = B;
};
template <int N>
struct IC {
  static constexpr int value = N;
};

// One work-group's query tile `qtile` of (batch, head) `bh`.  `stages` and `sdQ`
// are the work-group's LDS buffers (sized for the JVP bodies).
template <int D, int MODE, int NW>
__device__ __forceinline__ void tile_body(const AttnArgs& a, const int bh, const int qtile,
                                          char* const stages, char* const sdQ) {
  // NW waves per work-group, 32 query rows each
  constexpr int BR = 32 * NW;
  constexpr int NTHREADS = 64 * NW;
  constexpr bool JVP = MODE != kFwd;
  constexpr bool ZC = MODE == kZeroClean;
  using G = Geo<D>;
  constexpr int TB = G::TILEB;
  constexpr int TBJ = JVP ? G::TILEB : 0;       // tangent tiles exist only in the JVP bodies
  // Three pipeline stages (block k is read from stage k mod 3 while block k+2 streams
  // into stage (k+2) mod 3), each holding the K, V, dK, dV tiles of one key block.
  constexpr int SB = 2 * TB + 2 * TBJ;
  // (operand addresses below are formed by XOR of the in-tile offsets, which needs
  // tile bases aligned beyond the tile-row size)
  static_assert(SB % 1024 == 0 && TB % 1024 == 0, "LDS tiles must be 1 KiB aligned");

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
  const int lane = tid & 63;
  const int hh = lane >> 5;   // which half of the wave (key sub-block within S^T)
  const int L = a.L;
  // tangent rows are [t0, L): t0 = 0 for the dense JVP
  const int t0 = ZC ? a.t0 : 0;
  const int Lt = L - t0;

  const size_t head = (size_t)bh * L * D;
  const size_t thead = (size_t)bh * Lt * D;
  const bf16_t* __restrict__ Qg = (const bf16_t*)a.Q + head;
  const bf16_t* __restrict__ Kg = (const bf16_t*)a.K + head;
  const bf16_t* __restrict__ Vg = (const bf16_t*)a.V + head;
  const bf16_t* __restrict__ dQg = (const bf16_t*)a.dQ + thead;
  const bf16_t* __restrict__ dKg = (const bf16_t*)a.dK + thead;
  const bf16_t* __restrict__ dVg = (const bf16_t*)a.dV + thead;

  const int q0 = qtile * BR;
  const int q1 = q0 + BR < L ? q0 + BR : L;
  const TilePlan plan = plan_tile(a.gt, q0, q1, BC);
  const int nblk = plan_num_blocks(plan);
  // (kZeroClean) the plan visits key blocks in increasing key order: the first ntk of
  // them hold no key >= t0
  int ntk = 0;
  if constexpr (ZC) ntk = plan_blocks_below(plan, t0 / BC);

  // ---- this lane's query row, and the groups holding the wave's 32 rows (uniform: the
  // per-row mask of partial blocks is formed from their key ranges on the scalar unit)
  const int qrow = wave * 32 + (lane & 31);   // row within the tile
  const int row = q0 + qrow;
  const int wrow0 = imin(q0 + wave * 32, L - 1);
  const int wg0 = find_group(a.gt, wrow0), wg1 = find_group(a.gt, imin(wrow0 + 31, L - 1));

  // ---- Q^T as B operand in registers: lane l holds row l%32, d = 16 s + 8 (l/32) + 0..7
  bf16x8 qop[G::KS];
#pragma unroll
  for (int s = 0; s < G::KS; ++s) {
    // rows past the end are clamped to the last row (their outputs are not stored)
    qop[s] = *(const bf16x8*)(Qg + (size_t)min(row, L - 1) * D + 16 * s + 8 * hh);
  }

  // ---- global -> LDS staging: direct loads (global_load_lds_dwordx4).  One wave
  // instruction writes 64 lanes x 16 bytes = 1 KiB of consecutive LDS, i.e. 1024 / ROWB
  // rows; the XOR swizzle is realised by choosing which logical chunk each lane fetches.
  // Rows past the end of the sequence are clamped to the last row (finite data; masked
  // keys / unstored queries).
  constexpr int RPI = 1024 / G::ROWB;  // rows per instruction
  const int dma_r = (lane * 16) / G::ROWB;
  const int dma_phys = ((lane * 16) % G::ROWB) >> 4;
  // (uniform 64-bit base + 32-bit per-lane byte offset: one head is < 4 GiB)
  // LDS destinations are passed as byte addresses (uniform integers)
  auto dma_rows = [&](const bf16_t* src, int row0, int r, unsigned dst) {
    const int rr = r + dma_r;
    const unsigned grow = (unsigned)min(row0 + rr, L - 1);
    const unsigned off = (grow * D + (unsigned)((dma_phys ^ swz<D>(rr)) * 8)) * 2u;
    lds_load16(src, off, dst + (unsigned)(r * G::ROWB));
  };
  // tangent rows: sequence row x is tangent row x - t0; rows below t0 are clamped to
  // tangent row 0 (finite data, cleared in LDS before use)
  auto dma_rows_t = [&](const bf16_t* src, int row0, int r, unsigned dst) {
    if constexpr (!ZC) {
      dma_rows(src, row0, r, dst);
    } else {
      const int rr = r + dma_r;
      const unsigned grow = (unsigned)min(max(row0 + rr - t0, 0), Lt - 1);
      const unsigned off = (grow * D + (unsigned)((dma_phys ^ swz<D>(rr)) * 8)) * 2u;
      lds_load16(src, off, dst + (unsigned)(r * G::ROWB));
    }
  };
  // One key tile of BC rows: instruction j (rows j*RPI ...) is issued by loading wave j % NI.
  // The loading waves are all of them, except in the dense JVP, where the second half of the
  // work-group issues every load (in its ping-pong order the first half's step is the longer
  // path; measured 0.7 % faster there, and 2 % slower for the zero-clean kernel).
  constexpr int NI = (MODE == kJvp && NW == 8) ? NW / 2 : NW;
  const int lw = wave - (NW - NI);  // index among the loading waves (negative: issues none)
  auto dma_tile = [&](const bf16_t* src, int k0, unsigned dst) {
#pragma unroll
    for (int j0 = 0; j0 < G::IPT; j0 += NI) {
      const int j = j0 + lw;
      if (lw >= 0 && (G::IPT % NI == 0 || j < G::IPT)) dma_rows(src, k0, j * RPI, dst);
    }
  };
  auto dma_tile_t = [&](const bf16_t* src, int k0, unsigned dst) {
#pragma unroll
    for (int j0 = 0; j0 < G::IPT; j0 += NI) {
      const int j = j0 + lw;
      if (lw >= 0 && (G::IPT % NI == 0 || j < G::IPT)) dma_rows_t(src, k0, j * RPI, dst);
    }
  };
  // the K, V (and dK, dV) tiles of key block kb into the stage at LDS address st.  A
  // zero-clean block wholly below t0 loads no tangent tiles (its step does not read them;
  // the stage keeps an older block's).  The load count then depends on the block, which
  // only the ping-pong schedule allows: it waits for all loads at each barrier.
  auto dma_block = [&](int kb, unsigned st) {
    const int k0 = kb * BC;
    dma_tile(Kg, k0, st);
    dma_tile(Vg, k0, st + TB);
    if constexpr (JVP) {
      if (!ZC || k0 + BC > t0) {
        dma_tile_t(dKg, k0, st + 2 * TB);
        dma_tile_t(dVg, k0, st + 2 * TB + TBJ);
      }
    }
  };
  // clear the first nrows rows of an LDS tile (16 bytes per thread and pass)
  auto zero_rows = [&](char* base, int nrows) {
    const int n = nrows * (G::ROWB / 16);
    for (int c = tid; c < n; c += NTHREADS) *(u32x4*)(base + 16 * c) = u32x4{0u, 0u, 0u, 0u};
  };

  // Per-lane LDS offsets of the MFMA operand reads.  With the row swizzle, the offset of
  // chunk 2s + hh of a row is lds_off(row, hh) ^ (32 s), and the transposed V / dV read
  // for k step t (16 keys), key half p (+0 / +8) and d tile dt is at
  // 16 t ROWB + (trx[p] ^ (64 dt)) (lane l of a 16-lane group reads 8 bytes addressed for
  // lane 4e + l/4, e = result element).  Only these bases stay in registers; the per-step
  // offsets cost one XOR each.
  const int g16 = lane >> 4, s16 = lane & 15;
  const int tr_r = 4 * (g16 >> 1) + (s16 >> 2), tr_c = 2 * (g16 & 1) + ((s16 & 3) >> 1);
  const unsigned trx0 = lds_off<D>(tr_r, tr_c) + 8 * (s16 & 1);
  const unsigned trx1 = lds_off<D>(8 + tr_r, tr_c) + 8 * (s16 & 1);

  // ---- accumulators (O^T, T^T: lane holds query l%32, d = 32 dt + 8 (i/4) + 4 (l/32) + i%4)
  f32x16 oacc[G::DT], tacc[JVP ? G::DT : 1];
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt) {
    oacc[dt] = f32x16{};
    if constexpr (JVP) tacc[dt] = f32x16{};
  }
  float m = -INFINITY;  // running reference max (log2 units); equal in lanes l and l^32
  float lsum = 0.f;     // partial normaliser over this lane's keys
  float rsum = 0.f;     // partial sum of P~ o dS over this lane's keys
  float mpend = 0.f;    // block max that triggered a rescale
  const float c2 = a.scale * kLog2e;
  const float sc = a.scale;
  const int krow = lane & 31;
  const unsigned koff = lds_off<D>(krow, hh), dqoff = lds_off<D>(qrow, hh);
  // The 4-wave forward kernel runs its block loop unrolled over the three stages: stage
  // bases become instruction immediates and the per-step offsets stay in 16 registers, so
  // its LDS reads need no address arithmetic (the 8-wave kernels have no registers to spare
  // and form each offset with one XOR per step).
  constexpr bool STATIC = MODE == kFwd && NW == 4;
  // (JVP) the dQ operand offsets do not depend on the stage: 8 registers, no arithmetic
  unsigned dqoffs[JVP ? G::KS : 1];
  if constexpr (JVP) {
#pragma unroll
    for (int s = 0; s < G::KS; ++s) dqoffs[s] = lds_addr(sdQ) + (dqoff ^ (32u * s));
  }
  unsigned koffs[STATIC ? G::KS : 1], vtro[2][STATIC ? G::DT : 1];
  if constexpr (STATIC) {
#pragma unroll
    for (int s = 0; s < G::KS; ++s) koffs[s] = koff ^ (32u * s);
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt) {
      vtro[0][dt] = trx0 ^ (64u * dt);
      vtro[1][dt] = trx1 ^ (64u * dt);
    }
  }

  // Two schedules of the key-block loop, both with three LDS stages.
  //
  // Lockstep (the 4-wave forward kernel, whose three work-groups per CU interleave by
  // themselves): every wave passes the barrier of block k after both phases of block k.
  // Block k+2 streams into stage (k+2) mod 3 during iterations k and k+1 (two
  // iterations of latency hidden).
  //
  // Ping-pong (the 8-wave kernels: JVP, zero-clean JVP): the waves of the first half of
  // the work-group (one per SIMD) pass the
  // barrier of block k after its output phase, those of the second half after its
  // score phase, so that each SIMD runs one wave's score phase (MFMA, then the softmax
  // on the vector ALU) beside the other wave's output phase:
  //   interval k (from barrier k-1 to barrier k):  first half   S(k), O(k)
  //                                                 second half  O(k-1), S(k)
  // Stage k mod 3 is then read in intervals k and k+1, so block k+1 streams into stage
  // (k+1) mod 3 (whose block, k-2, was last read in interval k-1) during interval k
  // only.  The score phase runs at raised wave priority, so that its MFMAs go first and
  // its softmax overlaps the other wave's output MFMAs.
  constexpr bool PP = NW == 8;  // (two waves of a work-group per SIMD; prefetch distance 1, else 2)
  static_assert(!ZC || PP, "zero-clean load counts vary by block: only full waits are correct");
  const bool late = PP && wave >= NW / 2;
  // barrier of block k: every own load but those of the block one prefetch distance
  // ahead has landed (lockstep: N per wave; D = 128: one per tile and wave; D = 64:
  // waves 0..3 issue one, the others none), every LDS read has returned
  auto end_iteration = [&]() {
    constexpr int N = PP ? 0 : (JVP ? 4 : 2) * ((G::IPT + NW - 1) / NW);
    static_assert(N == 0 || N == 2 || N == 4, "vmcnt immediate below");
    if constexpr (N == 4) asm volatile("s_waitcnt vmcnt(4) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    else if constexpr (N == 2) asm volatile("s_waitcnt vmcnt(2) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  };

  // Output phase of a block: O^T += V^T P~^T ; T^T += dV^T P~^T + V^T H~^T, one (t, dt)
  // group of MFMAs at a time, its operands read OPF groups ahead (the order is pinned with
  // scheduling fences: left to itself the compiler waits on each read right before its
  // MFMA)
  auto ophase = [&](auto tk, auto am, const char* cV, const char* cdV, const bf16x8* pb, const bf16x8* hb) {
    constexpr bool TK = JVP && decltype(tk)::value;
    constexpr int C = decltype(am)::value;  // stage index known at compile time, or -1
    constexpr int OPF = JVP ? 1 : 2;
    constexpr int NG = 2 * G::DT;
    const unsigned vb0 = C >= 0 ? 0u : vreg_add(lds_addr(cV), trx0);
    const unsigned vb1 = C >= 0 ? 0u : vreg_add(lds_addr(cV), trx1);
    const unsigned dvo = (unsigned)(cdV - cV);
    bf16x8 vop[OPF + 1], dvop[OPF + 1];
    auto read = [&](int g) {
      const int t = g / G::DT, dt = g % G::DT, b = g % (OPF + 1);
      const unsigned o = 16u * t * G::ROWB;
      unsigned a0, a1;
      if constexpr (C >= 0) {
        a0 = lds_addr(stages) + (unsigned)(C * SB + TB) + vtro[0][dt];
        a1 = lds_addr(stages) + (unsigned)(C * SB + TB) + vtro[1][dt];
      } else {
        a0 = vb0 ^ (64u * dt);
        a1 = vb1 ^ (64u * dt);
      }
      vop[b] = cat(ld_tr_at(a0 + o), ld_tr_at(a1 + o));
      if constexpr (TK) dvop[b] = cat(ld_tr_at(a0 + o + dvo), ld_tr_at(a1 + o + dvo));
    };
#pragma unroll
    for (int g = 0; g < OPF; ++g) read(g);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (g + OPF < NG) read(g + OPF);
      __builtin_amdgcn_sched_barrier(0);
      const int t = g / G::DT, dt = g % G::DT, b = g % (OPF + 1);
      oacc[dt] = mfma(vop[b], pb[t], oacc[dt]);
      if constexpr (TK) tacc[dt] = mfma(dvop[b], pb[t], tacc[dt]);
      if constexpr (JVP) tacc[dt] = mfma(vop[b], hb[t], tacc[dt]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // One key block; TK: the block has tangent keys (dK, dV tiles are present).  Returns
  // true -- before touching any accumulator -- if some row's block max exceeds its
  // reference by more than kLazy; the caller then rescales and redoes the block.
  auto step = [&](auto tk, auto am, int it, const char* cK, const char* cV, const char* cdK, const char* cdV,
                  unsigned next_stage) -> bool {
    constexpr bool TK = JVP && decltype(tk)::value;
    constexpr int C = decltype(am)::value;  // stage index known at compile time, or -1
    // prefetch the block one prefetch distance ahead (redone, with the same data, when
    // the block is redone).
    // Lockstep: a fixed number of loads per iteration, indices past the end clamped (that
    // stage is never read).
    if constexpr (PP) {
      if (it + 1 < nblk) dma_block(plan_block(plan, it + 1), next_stage);
    } else {
      dma_block(plan_block(plan, min(it + 2, nblk - 1)), next_stage);
    }
    const int k0 = plan_block(plan, it) * BC;

    // ---- scores and score tangents (transposed): S^T = K Q^T, dS^T = dK Q^T + K dQ^T
    if constexpr (PP) __builtin_amdgcn_s_setprio(1);
    f32x16 S = f32x16{}, dS = f32x16{};
    // operand reads run SPF k steps ahead of the MFMAs that consume them (order pinned
    // with scheduling fences, as in the output phase)
    constexpr int SPF = JVP ? 1 : 2;
    const unsigned kb = C >= 0 ? 0u : vreg_add(lds_addr(cK), koff);
    const unsigned dko = (unsigned)(cdK - cK);
    bf16x8 kop[SPF + 1], dkop[SPF + 1], dqop[SPF + 1];
    auto read = [&](int s) {
      const int b = s % (SPF + 1);
      if constexpr (C >= 0) kop[b] = ld128_at(lds_addr(stages) + (unsigned)(C * SB) + koffs[s]);
      else kop[b] = ld128_at(kb ^ (32u * s));
      if constexpr (TK) dkop[b] = ld128_at((kb ^ (32u * s)) + dko);
      if constexpr (JVP) dqop[b] = ld128_at(dqoffs[s]);
    };
#pragma unroll
    for (int s = 0; s < SPF; ++s) read(s);
#pragma unroll
    for (int s = 0; s < G::KS; ++s) {
      if (s + SPF < G::KS) read(s + SPF);
      __builtin_amdgcn_sched_barrier(0);
      const int b = s % (SPF + 1);
      S = mfma(kop[b], qop[s], S);
      if constexpr (TK) dS = mfma(dkop[b], qop[s], dS);
      if constexpr (JVP) dS = mfma(kop[b], dqop[b], dS);
      __builtin_amdgcn_sched_barrier(0);
    }

    // ---- mask (only on blocks not admissible for every row of the tile): S = -inf, dS = 0
    float sv[16], dsv[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      sv[i] = S[i];
      dsv[i] = JVP ? dS[i] : 0.f;
    }
    if (!block_is_full(plan, k0, BC, L)) {
      // admitted keys of the block for this lane's row; the lane holds keys
      // k0 + 8 (i/4) + 4 hh + i%4
      const uint32_t bits = row_bits(a.gt, wg0, wg1, row, k0) >> (4 * hh);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const bool ok = (bits >> (8 * (i >> 2) + (i & 3))) & 1u;
        sv[i] = ok ? sv[i] : -INFINITY;
        dsv[i] = ok ? dsv[i] : 0.f;
      }
    }

    // ---- online softmax.  The scale is positive, so max(S) * c2 = max(S * c2).
    const float mloc = max16(sv) * c2;
    if (__ballot(mloc > m + kLazy) != 0) {
      mpend = mloc;
      return true;
    }
    const float mneg = m == -INFINITY ? 0.f : -m;
    float p[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      p[i] = __builtin_amdgcn_exp2f(fmaf(sv[i], c2, mneg));
      lsum += p[i];
    }
    bf16x8 pb[2], hb[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 8; ++j) pb[t][j] = (bf16_t)p[8 * t + j];
    if constexpr (JVP) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float hv = p[i] * (dsv[i] * sc);
        rsum += hv;
        hb[i >> 3][i & 7] = (bf16_t)hv;
      }
    }

    if constexpr (PP) __builtin_amdgcn_s_setprio(0);
    if (late) end_iteration();
    ophase(tk, am, cV, cdV, pb, hb);
    if (!late) end_iteration();
    return false;
  };

  // prologue: dQ of the query tile, then the first key blocks (one per unit of prefetch distance)
  const unsigned st_lds = __builtin_amdgcn_readfirstlane(lds_addr(stages));
  if constexpr (JVP) {
    const unsigned dq_lds = __builtin_amdgcn_readfirstlane(lds_addr(sdQ));
    constexpr int IPQ = BR * G::ROWB / 1024;  // 1 KiB direct loads of the dQ tile
#pragma unroll
    for (int j0 = 0; j0 < IPQ; j0 += NW) dma_rows_t(dQg, q0, (j0 + wave) * RPI, dq_lds);
  }
  if (nblk > 0) {
    dma_block(plan_block(plan, 0), st_lds);
    if constexpr (!PP) dma_block(plan_block(plan, min(1, nblk - 1)), st_lds + SB);
  }
  // vmcnt(0) through the builtin, so that the compiler also knows that the Q operand
  // loads above are complete and does not wait for them inside the loop
  __builtin_amdgcn_s_waitcnt(0xF70);
  __syncthreads();
  if constexpr (ZC) {
    if (q0 < t0) {  // the tile straddles t0: its rows below t0 have zero dQ
      zero_rows(sdQ, t0 - q0);
      __syncthreads();
    }
  }

  int it = 0;
  int cur = 0;       // stage of block it
  int cleared = -1;  // (kZeroClean) last block whose tangent rows below t0 were cleared
  for (;;) {
    bool rescale = false;
    if constexpr (ZC) {
      // key blocks below t0: no dK, dV terms
      while (it < ntk) {
        const int nxt = PP ? (cur == 2 ? 0 : cur + 1) : (cur == 0 ? 2 : cur - 1);  // its prefetch stage
        const char* cs = stages + cur * SB;
        rescale = step(Tag<false>{}, IC<-1>{}, it, cs, cs + TB, cs + 2 * TB, cs + 2 * TB + TBJ,
                       st_lds + (unsigned)(nxt * SB));
        if (rescale) break;
        ++it;
        cur = cur == 2 ? 0 : cur + 1;
      }
    }
    if constexpr (STATIC) {
      // three copies of the step, one per stage: block it is in stage it mod 3, block it+2
      // streams into stage (it+2) mod 3
      auto sstep = [&](auto am) -> bool {
        constexpr int C = decltype(am)::value;
        char* cs = stages + C * SB;
        return step(Tag<false>{}, am, it, cs, cs + TB, cs + 2 * TB, cs + 2 * TB + TBJ,
                    st_lds + (unsigned)(((C + 2) % 3) * SB));
      };
      while (it < nblk) {
        if (cur == 0) {
          rescale = sstep(IC<0>{});
          if (rescale) break;
          cur = 1;
          if (++it >= nblk) break;
        }
        if (cur == 1) {
          rescale = sstep(IC<1>{});
          if (rescale) break;
          cur = 2;
          if (++it >= nblk) break;
        }
        rescale = sstep(IC<2>{});
        if (rescale) break;
        cur = 0;
        ++it;
      }
    } else if (!rescale) {
      while (it < nblk) {
        const int nxt = PP ? (cur == 2 ? 0 : cur + 1) : (cur == 0 ? 2 : cur - 1);  // its prefetch stage
        char* cs = stages + cur * SB;
        if constexpr (ZC) {
          // a block straddling t0: clear the tangent rows of its keys below t0 (once per
          // block, so that every wave passes this barrier equally often)
          const int k0 = plan_block(plan, it) * BC;
          if (k0 < t0 && cleared != it) {
            zero_rows(cs + 2 * TB, t0 - k0);
            zero_rows(cs + 2 * TB + TBJ, t0 - k0);
            asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
            cleared = it;
          }
        }
        rescale = step(Tag<true>{}, IC<-1>{}, it, cs, cs + TB, cs + 2 * TB, cs + 2 * TB + TBJ,
                       st_lds + (unsigned)(nxt * SB));
        if (rescale) break;
        ++it;
        cur = cur == 2 ? 0 : cur + 1;
      }
    }
    if (!rescale) break;
    // Cold path: move the reference max of the rows that need it (lanes l and l^32 hold
    // the same query, so the new reference is their joint max), rescale O, T, l, r, and
    // redo block `it` (its S is recomputed; its stage still holds its K/V, and the
    // repeated prefetch rewrites stage (it+1) mod 3 with identical data).
    const float mx = fmaxf(mpend, xor32(mpend));
    const bool up = mx > m + kLazy;
    const float mnew = up ? mx : m;
    const float alpha = up ? __builtin_amdgcn_exp2f(m - mnew) : 1.f;
    lsum *= alpha;
    if constexpr (JVP) rsum *= alpha;
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt) {
      oacc[dt] *= alpha;
      if constexpr (JVP) tacc[dt] *= alpha;
    }
    m = mnew;
  }

  // ---- epilogue: combine the two half-waves' partial sums, normalise, store
  const float l_tot = lsum + xor32(lsum);
  const float r_tot = JVP ? rsum + xor32(rsum) : 0.f;
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (row < L) {
    bf16_t* Og = (bf16_t*)a.O + head + (size_t)row * D;
    bf16_t* dOg = (bf16_t*)a.dO + thead + (size_t)max(row - t0, 0) * D;
    const bool store_do = !ZC || row >= t0;  // dO of rows below t0 is zero and not stored
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = 32 * dt + 8 * q4 + 4 * hh;
        bf16x4 ov, dov;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float on = oacc[dt][4 * q4 + e] * inv;
          ov[e] = (bf16_t)on;
          if constexpr (JVP) dov[e] = (bf16_t)((tacc[dt][4 * q4 + e] - r_tot * on) * inv);
        }
        *(bf16x4*)(Og + d) = ov;
        if constexpr (JVP) {
          if (store_do) *(bf16x4*)(dOg + d) = dov;
        }
      }
    }
    if (hh == 0)
      a.LSE[(size_t)bh * L + row] = l_tot > 0.f ? (m + __log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

// NW = 8 (JVP and zero-clean: 256-row tiles, one work-group and two waves per SIMD per
// CU) or 4 (forward only: 128-row tiles and a smaller register footprint, so that three
// work-groups share a CU, three waves per SIMD, and interleave without any schedule).
template <int D, int MODE, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(NW == 8 ? 2 : 3, NW == 8 ? 2 : 3)))
void attn_mfma_kernel(const AttnArgs a) {
  constexpr bool JVP = MODE != kFwd;
  using G = Geo<D>;
  // LDS: three stages of K, V (+ dK, dV) tiles, and (JVP) the dQ tile of the query
  // tile, read back as an MFMA operand (keeps the per-wave register footprint within
  // two waves per SIMD).  D = 128 JVP: 3 x 32 KiB + 64 KiB = 160 KiB.
  constexpr int SB = JVP ? 4 * G::TILEB : 2 * G::TILEB;  // (the stage size tile_body uses)
  __shared__ __attribute__((aligned(1024))) char stages[3 * SB];
  __shared__ __attribute__((aligned(1024))) char sdQ[JVP ? 32 * NW * G::ROWB : 16];

  const TileSlot sl = slot_of(blockIdx.x, a.B * a.H, a.order.nt, MODE == kZeroClean ? kHeadGroupWide : kHeadGroup);
  const int bh = sl.bh;
  const int qtile = tile_of(a.order, sl.pos);
  if constexpr (MODE == kZeroClean) {
    if ((qtile + 1) * 32 * NW <= a.t0) {  // no tangent row in the tile: the primal only
      tile_body<D, kFwd, NW>(a, bh, qtile, stages, sdQ);
      return;
    }
  }
  tile_body<D, MODE, NW>(a, bh, qtile, stages, sdQ);
}

}  // namespace

hipError_t launch_mfma_bf16(const AttnArgs& a, int D, Pass pass, hipStream_t stream) {
  const dim3 grid((unsigned)(a.order.nt * a.B * a.H));
  constexpr int NJ = kMfmaBr / 32, NF = kMfmaBrFwd / 32;
  const dim3 block(64 * (pass == Pass::kFwd ? NF : NJ));
  if (D == 128) {
    if (pass == Pass::kJvp) hipLaunchKernelGGL((attn_mfma_kernel<128, kJvp, NJ>), grid, block, 0, stream, a);
    else if (pass == Pass::kJvpZeroClean)
      hipLaunchKernelGGL((attn_mfma_kernel<128, kZeroClean, NJ>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_mfma_kernel<128, kFwd, NF>), grid, block, 0, stream, a);
  } else {
    if (pass == Pass::kJvp) hipLaunchKernelGGL((attn_mfma_kernel<64, kJvp, NJ>), grid, block, 0, stream, a);
    else if (pass == Pass::kJvpZeroClean)
      hipLaunchKernelGGL((attn_mfma_kernel<64, kZeroClean, NJ>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_mfma_kernel<64, kFwd, NF>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace attn
