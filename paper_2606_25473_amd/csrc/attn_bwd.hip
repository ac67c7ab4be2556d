// attn_bwd.hip -- gradient of masked softmax attention (reverse mode) on gfx950.
//
// For a cotangent gO of O = softmax(s Q K^T + M) V (the paper's masked-attention
// equation, App. B), with P recomputed from the saved LSE (P = exp(s Q K^T - LSE) on
// admissible pairs, 0 elsewhere):
//   Delta = rowsum(gO o O),  gP = gO V^T,  gS = P o (gP - Delta),
//   gQ = s gS K,  gK = s gS^T Q,  gV = P^T gO.
// Two passes on one stream, neither with atomics (results are deterministic):
//  - query-tile pass: a work-group owns 256 query rows (8 waves x 32), computes Delta
//    for them, then streams the key blocks of its plan (the forward's query-group
//    plan) and accumulates gQ^T = K^T gS^T;
//  - key-tile pass: a work-group owns 128 keys (4 waves x 32) and two halves of each
//    64-row query block (waves 0..3 the first 32 rows, 4..7 the second), streams the
//    query blocks that see its keys (the query groups admitting any of them) through a
//    three-stage LDS ring (block it+2 loads while block it is used), and
//    accumulates gV^T = gO^T P and gK^T = Q^T gS; the two halves are summed at the end.
//    Each wave keeps the K operands of its 32 keys in registers (read once from LDS), so
//    the LDS holds only the V tile and the three stages.
// Matrix-core work: 6 D flop per (query, key) pair in the first pass, 8 D in the second
// (the scores S and gP are computed in both), against 10 D for a single pass that would
// need atomic gQ updates.
//
// The fp32 entry point runs the same two passes on fp32 matrix cores (attn_f32.hip).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "kernels.hpp"
#include "mfma_common.hpp"

namespace attn {
namespace {

using namespace dev;

template <int N>
struct IC {  // a compile-time count (or stage index) passed to a generic lambda
  static constexpr int value = N;
};

constexpr int NW = 8;  // waves per work-group in both bf16 passes
constexpr int NTHREADS = 64 * NW;

// ---------------------------------------------------------------- bf16, query-tile pass

constexpr int QBR = kMfmaBr;  // 256 query rows per work-group
constexpr int QBC = kMfmaBc;  // 32 keys per block

template <int D>
struct QGeo {
  static constexpr int ROWB = D * 2;            // bytes per LDS row (bf16)
  static constexpr int TILEB = QBC * ROWB;      // one K or V tile of a key block
  static constexpr int DT = D / 32;             // 32-wide d tiles of gQ^T
  static constexpr int KS = D / 16;             // 16-deep k steps over d
  static constexpr int IPT = TILEB / 1024;      // 1 KiB direct loads per tile
};

template <int D>
__global__ __launch_bounds__(NTHREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_bwd_dq_kernel(const BwdArgs a) {
  using G = QGeo<D>;
  constexpr int TB = G::TILEB;
  constexpr int SB = 2 * TB;  // stage: K and V tiles of one key block
  __shared__ __attribute__((aligned(1024))) char stages[3 * SB];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int hh = lane >> 5;
  const int L = a.L;

  const TileSlot sl = slot_of(blockIdx.x, a.B * a.H, a.order.nt, kHeadGroup);
  const int bh = sl.bh;
  const int qtile = tile_of(a.order, sl.pos);
  const size_t head = (size_t)bh * L * D;
  const bf16_t* __restrict__ Qg = (const bf16_t*)a.Q + head;
  const bf16_t* __restrict__ Kg = (const bf16_t*)a.K + head;
  const bf16_t* __restrict__ Vg = (const bf16_t*)a.V + head;
  const bf16_t* __restrict__ Og = (const bf16_t*)a.O + head;
  const bf16_t* __restrict__ gOg = (const bf16_t*)a.gO + head;

  const int q0 = qtile * QBR;
  const int q1 = q0 + QBR < L ? q0 + QBR : L;
  const TilePlan plan = plan_tile(a.gt, q0, q1, QBC);
  const int nblk = plan_num_blocks(plan);

  const int qrow = wave * 32 + (lane & 31);
  const int row = q0 + qrow;
  // groups holding the wave's 32 rows (uniform; partial blocks form the row's mask bits
  // from their key ranges)
  const int wrow0 = imin(q0 + wave * 32, L - 1);
  const int wg0 = find_group(a.gt, wrow0), wg1 = find_group(a.gt, imin(wrow0 + 31, L - 1));

  // Q^T and gO^T as B operands in registers (lane: row l%32, d = 16 s + 8 (l/32) + 0..7);
  // rows past the end are clamped to the last row (their results are not stored)
  const size_t rbase = (size_t)min(row, L - 1) * D;
  bf16x8 qop[G::KS], gop[G::KS];
  float dpart = 0.f;
#pragma unroll
  for (int s = 0; s < G::KS; ++s) {
    qop[s] = *(const bf16x8*)(Qg + rbase + 16 * s + 8 * hh);
    gop[s] = *(const bf16x8*)(gOg + rbase + 16 * s + 8 * hh);
    const bf16x8 ov = *(const bf16x8*)(Og + rbase + 16 * s + 8 * hh);
#pragma unroll
    for (int j = 0; j < 8; ++j) dpart = fmaf((float)gop[s][j], (float)ov[j], dpart);
  }
  // Delta of this row: the two half-waves hold complementary halves of d
  const float delta = dpart + xor32(dpart);
  const float lse = a.LSE[(size_t)bh * L + min(row, L - 1)];
  // a row without admissible keys has LSE = -inf; all its pairs are masked below
  const float lse2 = lse == -INFINITY ? 0.f : lse * kLog2e;
  if (row < L && hh == 0) a.Delta[(size_t)bh * L + row] = delta;

  constexpr int RPI = 1024 / G::ROWB;
  const int dma_r = (lane * 16) / G::ROWB;
  const int dma_phys = ((lane * 16) % G::ROWB) >> 4;
  auto dma_tile = [&](const bf16_t* src, int k0, unsigned dst) {
#pragma unroll
    for (int j0 = 0; j0 < G::IPT; j0 += NW) {
      const int j = j0 + wave;
      if (G::IPT % NW == 0 || j < G::IPT) {
        const int rr = j * RPI + dma_r;
        const unsigned grow = (unsigned)min(k0 + rr, L - 1);
        const unsigned off = (grow * D + (unsigned)((dma_phys ^ swz<D>(rr)) * 8)) * 2u;
        lds_load16(src, off, dst + (unsigned)(j * RPI * G::ROWB));
      }
    }
  };
  auto dma_block = [&](int kb, unsigned st) {
    dma_tile(Kg, kb * QBC, st);
    dma_tile(Vg, kb * QBC, st + TB);
  };

  static_assert(SB % 1024 == 0 && TB % 1024 == 0, "LDS tiles must be 1 KiB aligned");
  unsigned trx[2];
  tr_bases<D>(lane, trx);

  f32x16 gacc[G::DT];
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt) gacc[dt] = f32x16{};
  const float c2 = a.scale * kLog2e;
  const int krow = lane & 31;
  // Per-lane LDS offsets of the operand reads within a stage, kept in 16 registers: chunk
  // 2s + hh of the lane's key row (K and V reads of k step s) and the transposed K reads of
  // key half p and d tile dt.  The block loop is unrolled over the three stages, so the
  // stage base is an instruction immediate and the reads need no address arithmetic.
  const unsigned koff = lds_off<D>(krow, hh);
  unsigned koffs[G::KS], ktro[2][G::DT];
#pragma unroll
  for (int s = 0; s < G::KS; ++s) koffs[s] = koff ^ (32u * s);
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt) {
    ktro[0][dt] = trx[0] ^ (64u * dt);
    ktro[1][dt] = trx[1] ^ (64u * dt);
  }

  // wait for every load but this iteration's prefetch (2 per wave at D = 128; at D = 64
  // waves 0..3 issue one per tile and the others none), then synchronise
  auto end_iteration = []() { asm volatile("s_waitcnt vmcnt(2) lgkmcnt(0)\n\ts_barrier" ::: "memory"); };
  static_assert((G::IPT + NW - 1) / NW == 1, "one direct load per tile and wave");

  // block it is in stage C = it mod 3; block it+2 streams into stage (C + 2) mod 3
  auto step = [&](auto am, int it) {
    constexpr int C = decltype(am)::value;
    // (opaque to the compiler: otherwise it hoists offset + stage base out of the loop, one
    // register per offset and stage, instead of folding the base into each read's immediate)
#pragma unroll
    for (int s = 0; s < G::KS; ++s) asm volatile("" : "+v"(koffs[s]));
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt) asm volatile("" : "+v"(ktro[0][dt]), "+v"(ktro[1][dt]));
    const unsigned sbase = lds_addr(stages) + (unsigned)(C * SB);  // (a compile-time constant)
    dma_block(plan_block(plan, min(it + 2, nblk - 1)), lds_addr(stages) + (unsigned)(((C + 2) % 3) * SB));
    const int k0 = plan_block(plan, it) * QBC;
    // S^T = K Q^T and gP^T = V gO^T (lane: query l%32, keys 8 (i/4) + 4 (l/32) + i%4);
    // operand reads run SPF k steps ahead of their MFMAs (order pinned with scheduling
    // fences)
    f32x16 S = f32x16{}, GP = f32x16{};
    constexpr int SPF = 2;
    bf16x8 kop[SPF + 1], vop[SPF + 1];
    auto read = [&](int s) {
      const int b = s % (SPF + 1);
      kop[b] = ld128_at(sbase + koffs[s]);
      vop[b] = ld128_at(sbase + TB + koffs[s]);
    };
#pragma unroll
    for (int s = 0; s < SPF; ++s) read(s);
#pragma unroll
    for (int s = 0; s < G::KS; ++s) {
      if (s + SPF < G::KS) read(s + SPF);
      __builtin_amdgcn_sched_barrier(0);
      const int b = s % (SPF + 1);
      S = mfma(kop[b], qop[s], S);
      GP = mfma(vop[b], gop[s], GP);
      __builtin_amdgcn_sched_barrier(0);
    }
    // P^T = exp(S^T - LSE) on admissible pairs, gS^T = P^T o (gP^T - Delta)
    float p[16], gs[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) p[i] = __builtin_amdgcn_exp2f(fmaf(S[i], c2, -lse2));
    if (!block_is_full(plan, k0, QBC, L)) {  // one uniform branch around the whole mask
      // the lane holds keys k0 + 8 (i/4) + 4 hh + i%4
      const uint32_t bits = row_bits(a.gt, wg0, wg1, row, k0) >> (4 * hh);
#pragma unroll
      for (int i = 0; i < 16; ++i) p[i] = ((bits >> (8 * (i >> 2) + (i & 3))) & 1u) ? p[i] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) gs[i] = p[i] * (GP[i] - delta);
    // gQ^T += K^T gS^T (K^T from transposed LDS reads, gS^T from this lane's registers),
    // one (t, dt) MFMA at a time with its operand read OPF groups ahead
    bf16x8 gsb[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 8; ++j) gsb[t][j] = (bf16_t)gs[8 * t + j];
    constexpr int OPF = 2, NG = 2 * G::DT;
    bf16x8 kt[OPF + 1];
    auto read_t = [&](int g) {
      const int t = g / G::DT, dt = g % G::DT;
      const unsigned o = sbase + 16u * t * G::ROWB;
      kt[g % (OPF + 1)] = cat(ld_tr_at(o + ktro[0][dt]), ld_tr_at(o + ktro[1][dt]));
    };
#pragma unroll
    for (int g = 0; g < OPF; ++g) read_t(g);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (g + OPF < NG) read_t(g + OPF);
      __builtin_amdgcn_sched_barrier(0);
      gacc[g % G::DT] = mfma(kt[g % (OPF + 1)], gsb[g / G::DT], gacc[g % G::DT]);
      __builtin_amdgcn_sched_barrier(0);
    }
    end_iteration();
  };

  const unsigned st_lds = __builtin_amdgcn_readfirstlane(lds_addr(stages));
  if (nblk > 0) {
    dma_block(plan_block(plan, 0), st_lds);
    dma_block(plan_block(plan, min(1, nblk - 1)), st_lds + SB);
  }
  __builtin_amdgcn_s_waitcnt(0xF70);  // (builtin: also retires the operand loads above)
  __syncthreads();
  // (whole triples in a loop without early exits, then the remainder: written with an exit
  // after each step, the three copies made the register allocator spill)
  int it = 0;
  for (; it + 3 <= nblk; it += 3) {
    step(IC<0>{}, it);
    step(IC<1>{}, it + 1);
    step(IC<2>{}, it + 2);
  }
  if (it < nblk) step(IC<0>{}, it);
  if (it + 1 < nblk) step(IC<1>{}, it + 1);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the clamped tail prefetches

  if (row < L) {
    bf16_t* gQg = (bf16_t*)a.gQ + head + (size_t)row * D;
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        bf16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (bf16_t)(a.scale * gacc[dt][4 * q4 + e]);
        *(bf16x4*)(gQg + 32 * dt + 8 * q4 + 4 * hh) = v;
      }
  }
}

// ---------------------------------------------------------------- bf16, key-tile pass

constexpr int KT = kBwdKeysPerTile;   // 128 keys per work-group (4 key groups of 32)

constexpr int QB = kBwdRowsPerBlock;  // 64 query rows per block (2 halves of 32)

template <int D>
struct KGeo {
  static constexpr int ROWB = D * 2;
  static constexpr int KTB = KT * ROWB;         // K (or V) rows of the work-group's keys
  static constexpr int QTB = QB * ROWB;         // Q (or gO) rows of one query block
  static constexpr int SB = 2 * QTB + 2 * 4 * QB;  // stage: Q, gO, LSE, Delta of a block
  static constexpr int BYTES = KTB + 3 * SB;    // V tile, three query-block stages
  static constexpr int DT = D / 32;
  static constexpr int KS = D / 16;
  static constexpr int IPK = KTB / 1024;        // 1 KiB direct loads per key tile
  static constexpr int IPQ = QTB / 1024;        // ... per query block tensor
  static constexpr int NACC = 2 * DT * 16;      // accumulator floats per lane (gK^T, gV^T)
  static_assert(4 * 64 * NACC * 4 <= BYTES, "the half-sum exchange fits in LDS");
};

template <int D>
__global__ __launch_bounds__(NTHREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_bwd_dkdv_kernel(const BwdArgs a) {
  using G = KGeo<D>;
  __shared__ __attribute__((aligned(1024))) char lds[G::BYTES];
  char* const stages = lds + G::KTB;  // the K tile passes through stages 1-2 at the start

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int hh = lane >> 5;
  const int kw = wave & 3;   // which 32 keys of the tile
  const int qh = wave >> 2;  // which 32 rows of each query block
  const int L = a.L;

  const TileSlot sl = slot_of(blockIdx.x, a.B * a.H, a.order.nt, kHeadGroupWide);
  const int bh = sl.bh;
  const int ktile = tile_of(a.order, sl.pos);
  const size_t head = (size_t)bh * L * D;
  const bf16_t* __restrict__ Qg = (const bf16_t*)a.Q + head;
  const bf16_t* __restrict__ Kg = (const bf16_t*)a.K + head;
  const bf16_t* __restrict__ Vg = (const bf16_t*)a.V + head;
  const bf16_t* __restrict__ gOg = (const bf16_t*)a.gO + head;
  const float* __restrict__ LSEg = a.LSE + (size_t)bh * L;
  const float* __restrict__ Dg = a.Delta + (size_t)bh * L;

  // plan over the query-group table: the query blocks of the groups that admit some key
  // of the tile
  const int k0 = ktile * KT;
  const int k1 = k0 + KT < L ? k0 + KT : L;
  const TilePlan plan = plan_key_tile(a.gt, k0, k1, QB);
  const int nblk = plan_num_blocks(plan);

  const int krow = kw * 32 + (lane & 31);  // this lane's key within the tile
  const int key = k0 + krow;

  constexpr int RPI = 1024 / G::ROWB;
  const int dma_r = (lane * 16) / G::ROWB;
  const int dma_phys = ((lane * 16) % G::ROWB) >> 4;
  // n_instr 1 KiB loads of rows [row0, ...) of src into dst, instruction j by wave j % NW
  auto dma_rows = [&](const bf16_t* src, int row0, unsigned dst, auto n_instr) {
    constexpr int N = decltype(n_instr)::value;
#pragma unroll
    for (int j0 = 0; j0 < N; j0 += NW) {
      const int j = j0 + wave;
      if (N % NW == 0 || j < N) {
        const int rr = j * RPI + dma_r;
        const unsigned grow = (unsigned)min(row0 + rr, L - 1);
        const unsigned off = (grow * D + (unsigned)((dma_phys ^ swz<D>(rr)) * 8)) * 2u;
        lds_load16(src, off, dst + (unsigned)(j * RPI * G::ROWB));
      }
    }
  };
  // query block qb into the stage at LDS address st: Q and gO rows, LSE and Delta values
  auto dma_qblock = [&](int qb, unsigned st) {
    const int r0 = qb * QB;
    dma_rows(Qg, r0, st, IC<G::IPQ>{});
    dma_rows(gOg, r0, st + G::QTB, IC<G::IPQ>{});
    const unsigned roff = (unsigned)min(r0 + lane, L - 1) * 4u;
    if (wave == NW - 2) lds_load4(LSEg, roff, st + 2 * G::QTB);
    if (wave == NW - 1) lds_load4(Dg, roff, st + 2 * G::QTB + 4 * QB);
  };

  static_assert(G::SB % 256 == 0 && G::KTB % 1024 == 0, "XOR-formed offsets need row-aligned tiles");
  unsigned trx[2];
  tr_bases<D>(lane, trx);
  const int qoff = qh * 32 * G::ROWB;  // this wave's 32 rows within a query block tile
  // chunk 2s + hh of a row sits at the row's chunk-hh offset ^ (32 s)
  const unsigned qaoff = qoff + lds_off<D>(lane & 31, hh);
  const unsigned kboff = lds_off<D>(krow, hh);

  f32x16 gk[G::DT], gv[G::DT];
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt) {
    gk[dt] = f32x16{};
    gv[dt] = f32x16{};
  }
  const float c2 = a.scale * kLog2e;

  const unsigned lds_base = __builtin_amdgcn_readfirstlane(lds_addr(lds));
  const unsigned st_lds = lds_base + G::KTB;
  // K tile into the space of stages 1-2, V tile to its own place; each wave then keeps the
  // K operands of its 32 keys in registers for the whole kernel
  const unsigned k_lds = st_lds + G::SB;
  dma_rows(Kg, k0, k_lds, IC<G::IPK>{});
  dma_rows(Vg, k0, lds_base, IC<G::IPK>{});
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  bf16x8 kreg[G::KS];
#pragma unroll
  for (int s = 0; s < G::KS; ++s) kreg[s] = ld128_at((k_lds + kboff) ^ (32u * s));
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __syncthreads();
  if (nblk > 0) {
    dma_qblock(plan_block(plan, 0), st_lds);
    dma_qblock(plan_block(plan, min(1, nblk - 1)), st_lds + G::SB);
  }
  __builtin_amdgcn_s_waitcnt(0xF70);
  __syncthreads();
  // loads per wave and block: the Q and gO rows, plus LSE (wave NW-2) or Delta (NW-1)
  constexpr int LPB = 2 * ((G::IPQ + NW - 1) / NW);
  static_assert(LPB == 4 || LPB == 2, "vmcnt immediates below");
  const bool stat_wave = wave >= NW - 2;
  int cur = 0;

  for (int it = 0; it < nblk; ++it) {
    const char* cs = stages + cur * G::SB;
    // block it+2 into the stage of block it-1, last read before the barrier that ended
    // iteration it-1 (past the end: the last block again, never read)
    const int nx2 = cur == 0 ? 2 : cur - 1;
    dma_qblock(plan_block(plan, min(it + 2, nblk - 1)), st_lds + (unsigned)(nx2 * G::SB));
    const int q0b = plan_block(plan, it) * QB;

    // S = Q K^T and gP = gO V^T (lane: key l%32, rows 8 (i/4) + 4 (l/32) + i%4 of the
    // half); operand reads one k step ahead of their MFMAs (order pinned with fences)
    f32x16 S = f32x16{}, GP = f32x16{};
    const unsigned qa = vreg_add(lds_addr(cs), qaoff);
    const unsigned kb = vreg_add(lds_base, kboff, it);
    bf16x8 aq[2], ag[2], bv[2];
    auto read = [&](int s) {
      const unsigned x = 32u * s;
      aq[s & 1] = ld128_at(qa ^ x);
      ag[s & 1] = ld128_at((qa ^ x) + G::QTB);
      bv[s & 1] = ld128_at(kb ^ x);
    };
    read(0);
#pragma unroll
    for (int s = 0; s < G::KS; ++s) {
      if (s + 1 < G::KS) read(s + 1);
      __builtin_amdgcn_sched_barrier(0);
      S = mfma(aq[s & 1], kreg[s], S);
      GP = mfma(ag[s & 1], bv[s & 1], GP);
      __builtin_amdgcn_sched_barrier(0);
    }
    // LSE and Delta of the lane's 16 rows (4 runs of 4 consecutive rows).  A row without
    // admissible keys has LSE = -inf: exp2 then gives +inf, which the mask (such a row is
    // never in a full block) replaces by 0.
    const float* sl = (const float*)(cs + 2 * G::QTB);
    const float* sd = sl + QB;
    float p[16], dl[16];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float4 lv = *(const float4*)(sl + 32 * qh + 8 * c + 4 * hh);
      const float4 dv = *(const float4*)(sd + 32 * qh + 8 * c + 4 * hh);
      const float lsev[4] = {lv.x, lv.y, lv.z, lv.w};
      const float dlv[4] = {dv.x, dv.y, dv.z, dv.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        p[4 * c + e] = __builtin_amdgcn_exp2f(fmaf(S[4 * c + e], c2, -lsev[e] * kLog2e));
        dl[4 * c + e] = dlv[e];
      }
    }
    if (!block_is_full(plan, q0b, QB, L)) {  // one uniform branch around the whole mask
      // the lane holds queries q0b + 32 qh + 8 (i/4) + 4 hh + i%4
      const uint32_t bits = key_bits(a.gt, key, q0b + 32 * qh, L) >> (4 * hh);
#pragma unroll
      for (int i = 0; i < 16; ++i) p[i] = ((bits >> (8 * (i >> 2) + (i & 3))) & 1u) ? p[i] : 0.f;
    }
    float gs[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) gs[i] = p[i] * (GP[i] - dl[i]);
    // gV^T += gO^T P and gK^T += Q^T gS (transposed LDS reads of the block's rows), one
    // (t, dt) group at a time with its operands read one group ahead
    bf16x8 pb[2], gsb[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        pb[t][j] = (bf16_t)p[8 * t + j];
        gsb[t][j] = (bf16_t)gs[8 * t + j];
      }
    constexpr int NG = 2 * G::DT;
    const unsigned tb0 = vreg_add(lds_addr(cs + qoff), trx[0]), tb1 = vreg_add(lds_addr(cs + qoff), trx[1]);
    bf16x8 got[2], qt[2];
    auto read_t = [&](int g) {
      const int t = g / G::DT, dt = g % G::DT;
      const unsigned o = 16u * t * G::ROWB;
      const unsigned a0 = (tb0 ^ (64u * dt)) + o, a1 = (tb1 ^ (64u * dt)) + o;
      got[g & 1] = cat(ld_tr_at(a0 + G::QTB), ld_tr_at(a1 + G::QTB));
      qt[g & 1] = cat(ld_tr_at(a0), ld_tr_at(a1));
    };
    read_t(0);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (g + 1 < NG) read_t(g + 1);
      __builtin_amdgcn_sched_barrier(0);
      const int t = g / G::DT, dt = g % G::DT;
      gv[dt] = mfma(got[g & 1], pb[t], gv[dt]);
      gk[dt] = mfma(qt[g & 1], gsb[t], gk[dt]);
      __builtin_amdgcn_sched_barrier(0);
    }
    // every load but this iteration's (block it+2) has landed
    if constexpr (LPB == 4) {
      if (stat_wave) asm volatile("s_waitcnt vmcnt(5) lgkmcnt(0)\n\ts_barrier" ::: "memory");
      else asm volatile("s_waitcnt vmcnt(4) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    } else {
      if (stat_wave) asm volatile("s_waitcnt vmcnt(3) lgkmcnt(0)\n\ts_barrier" ::: "memory");
      else asm volatile("s_waitcnt vmcnt(2) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    }
    cur = cur == 2 ? 0 : cur + 1;
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // (the clamped tail loads)
  __syncthreads();

  // Sum the two row halves: waves 4..7 leave their partial gK^T, gV^T in LDS (every
  // stage is idle after the last barrier), waves 0..3 add them and store.
  float* red = (float*)lds + (size_t)kw * G::NACC * 64 + lane;
  if (qh == 1) {
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        red[(dt * 16 + i) * 64] = gk[dt][i];
        red[((G::DT + dt) * 16 + i) * 64] = gv[dt][i];
      }
  }
  __syncthreads();
  if (qh == 0 && key < L) {
    bf16_t* gKg = (bf16_t*)a.gK + head + (size_t)key * D;
    bf16_t* gVg = (bf16_t*)a.gV + head + (size_t)key * D;
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        bf16x4 kv, vv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = 4 * q4 + e;
          kv[e] = (bf16_t)(a.scale * (gk[dt][i] + red[(dt * 16 + i) * 64]));
          vv[e] = (bf16_t)(gv[dt][i] + red[((G::DT + dt) * 16 + i) * 64]);
        }
        const int d = 32 * dt + 8 * q4 + 4 * hh;
        *(bf16x4*)(gKg + d) = kv;
        *(bf16x4*)(gVg + d) = vv;
      }
  }
}

}  // namespace

hipError_t launch_bwd_mfma_bf16(const BwdArgs& qa, const BwdArgs& ka, int D, hipStream_t stream) {
  const dim3 gq((unsigned)(qa.order.nt * qa.B * qa.H)), gk((unsigned)(ka.order.nt * ka.B * ka.H));
  const dim3 block(NTHREADS);
  if (D == 128) {
    hipLaunchKernelGGL((attn_bwd_dq_kernel<128>), gq, block, 0, stream, qa);
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<128>), gk, block, 0, stream, ka);
  } else {
    hipLaunchKernelGGL((attn_bwd_dq_kernel<64>), gq, block, 0, stream, qa);
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<64>), gk, block, 0, stream, ka);
  }
  return hipGetLastError();
}

}  // namespace attn
