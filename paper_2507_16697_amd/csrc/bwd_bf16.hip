// Recompute backward of ring-chunked attention, dK/dV part at head size 128: bf16 MFMA with fp32
// accumulation (gfx950).  Head size 64 runs the two-waves-per-SIMD kernel in bwd_bf16_d64.hip.
//
// One workgroup = 4 waves (one per SIMD) = one K/V head and a tile of 128 keys inside one chunk
// (a key tile never straddles a chunk boundary).  With the merged log-sum-exp saved by the
// forward, every chunk's gradients are independent (arXiv 2507.16697 Sec. III-A: K/V chunk
// gradients computed per chunk), so the workgroup sweeps every query of every query head that
// shares the K/V head (G > 1 for grouped-query attention) once, in tiles of 64.  Wave w owns keys
// 32w .. 32w+31: their K and V rows stay in registers as MFMA B operands, and their fp32 dK^T,
// dV^T accumulate in registers.  Per 32-query block:
//   S   = Q K^T           A = Q rows (LDS),  B = K rows (registers)      -> lane = key
//   D-dP = D + dO (-V)^T  A = dO rows (LDS), B = -V rows (registers), accumulators start at D
//   P   = exp2(S*scale*log2e + nl_i),  -dS = P (D - dP)                   (fp32; nl_i = -lse_i*log2e
//                                                                        from the preprocess)
//   dV^T += dO^T P        A = dO^T by transposed LDS reads, B = P from registers
//   -dK^T += Q^T (-dS)    A = Q^T by transposed LDS reads,  B = -dS from registers
// (negating V and dK are exact, and let the matrix cores subtract D).
//
// With one wave per SIMD nothing hides a stall, so each wave runs a fixed schedule, software
// pipelined over 32-query blocks: phase 1 of block j issues the 16 S/dP products of block j+1, one
// at a time, each beside half of one of the P/dS elements 8..15 of block j; phase 2 issues the 16
// dV/dK products of block j, each beside half of one of the elements 0..7 of block j+1.  LDS
// operands are read 16 products ahead.  Every vector instruction then hides behind a matrix
// product.  Q, dO, nl and D rotate through a four-stage LDS ring filled by direct global->LDS
// loads three tiles ahead; one barrier per tile.  Rows past Nq in a head's last tile are clamped
// copies whose dO row and D are zeroed in LDS, so they add nothing; key lanes past the chunk end
// only feed their own dK/dV columns, which are not written.  dQ is computed by the
// query-stationary kernel in bwd_dq_bf16.hip, or, in store mode (kStore), from the -dS operands
// this kernel writes out (bwd_dq_ds.hip): 4 KiB per wave and tile, two 1 KiB global stores per
// 32-query block.
//
// Register files: the 128 dK^T/dV^T accumulators and the K/V fragments live in AGPRs (MFMA
// accumulator and operand registers), the S/dP accumulators, P/dS and the operands in flight in
// VGPRs.  The matrix products are inline assembly so that each operand sits in the file named
// for it.  The compiler does not track hazards through inline assembly, so the schedule keeps
// every MFMA result at least 20 wait states (issued instructions, or s_nop cycles) away from any
// other instruction that reads or moves it, and every vector write of an operand at least 2 wait
// states ahead of the product that reads it; the tests check both in the built code.

#include "ringx_device.h"
#include "ringx_kernels.h"

#include <algorithm>
#include <type_traits>

namespace ringx {
namespace {

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

template <int D>
struct DkvCfg {
  static constexpr int kThreads = 256;
  static constexpr int kWaves = 4;
  static constexpr int kBK = 128;                  // keys per workgroup (32 per wave)
  static constexpr int kBQ = 64;                   // queries per tile
  static constexpr int kRowBytes = 2 * D;          // Q, dO, K, V rows
  static constexpr int kChunks = D / 8;            // 16-byte chunks per row
  static constexpr int kDSteps = D / 16;
  static constexpr int kCT = D / 32;
  static constexpr int kQTile = kBQ * kRowBytes;   // bytes of one Q or dO tile
  static constexpr int kLoads = kQTile / (kThreads * 16);   // 16-byte loads per thread per tile
  // one stage of the ring: Q tile, dO tile, nl[kBQ], D[kBQ]
  static constexpr int kOffO = kQTile;
  static constexpr int kOffL = 2 * kQTile;
  static constexpr int kOffD = kOffL + kBQ * 4;
  static constexpr int kStage = kOffD + kBQ * 4;
  static constexpr int kStages = 4;
  static constexpr int kLds = kStages * kStage;
  // vector-memory operations one tile puts in flight per wave (waves 0 and 1 add nl / D)
  static constexpr int kTileOps = 2 * kLoads;
  static_assert(kLoads >= 1 && kQTile == kLoads * kThreads * 16, "whole tiles per load round");
};

// XOR swizzle of the 16-byte chunks of a row of `RB` bytes (as in the forward kernel): 16
// consecutive rows read at one chunk, and 4 consecutive rows read at 2 chunks by transposed
// reads, hit distinct banks.
template <int RB>
__device__ __forceinline__ int swz(int row) {
  if constexpr (RB == 256) return ((row & 3) << 2) | ((row >> 2) & 3);
  else return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
}
template <int RB>
__device__ __forceinline__ int toff(int row, int c) {
  return row * RB + ((c ^ swz<RB>(row)) << 4);
}
// byte offset of element `col` (2-byte units) of `row`
template <int RB>
__device__ __forceinline__ int eoff(int row, int col) {
  return toff<RB>(row, col >> 3) + (col & 7) * 2;
}

template <int D, bool kStore>
__global__ __launch_bounds__(256, 1) void bwd_dkdv_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const __bf16* __restrict__ dout, const float* __restrict__ nl,
    const float* __restrict__ delta, float* __restrict__ dk, float* __restrict__ dv, int BHkv,
    int H, int grp, int64_t Nq, int64_t Nk, int R, int tiles_per_chunk, float c2, float scale,
    int accumulate, char* __restrict__ ds) {
  using C = DkvCfg<D>;
  __shared__ __attribute__((aligned(1024))) char lds[C::kLds];
  const uint32_t lbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int n = lane & 31;
  const int g = lane >> 5;

  const uint32_t wg = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t per_bh = (int64_t)R * tiles_per_chunk;
  const int64_t bh = wg / per_bh;   // K/V head (of B * H / G)
  const int r = (int)((wg % per_bh) / tiles_per_chunk);
  const int tile = (int)(wg % tiles_per_chunk);
  if (bh >= BHkv) return;
  const int64_t lo = (int64_t)r * Nk / R;
  const int64_t hi = (int64_t)(r + 1) * Nk / R;
  const int64_t k0 = lo + (int64_t)tile * C::kBK;
  if (k0 >= hi) return;                         // uniform over the workgroup

  // the grp query heads sharing this K/V head are swept one after the other
  const int64_t qh0 = (bh / (H / grp)) * H + (bh % (H / grp)) * grp;
  // wave-uniform bases in SGPRs, so that the per-tile load addresses are scalar arithmetic
  const char* qb =
      static_cast<const char*>(uniform_ptr(reinterpret_cast<const char*>(q + qh0 * Nq * D)));
  const char* ob =
      static_cast<const char*>(uniform_ptr(reinterpret_cast<const char*>(dout + qh0 * Nq * D)));
  const float* nlb = static_cast<const float*>(uniform_ptr(nl + qh0 * Nq));
  const float* deltab = static_cast<const float*>(uniform_ptr(delta + qh0 * Nq));
  // query positions within a head are 32-bit (the library takes at most 2^31 - 128 queries
  // per head), so that the tile bookkeeping below stays scalar instructions
  const int nq = (int)Nq;
  const int nqt = (nq + C::kBQ - 1) / C::kBQ;
  const int ntiles = grp * nqt;
  const int tail = nq - (nqt - 1) * C::kBQ;   // valid rows of a head's last tile

  // Per-lane offsets of the tile loads: load round u covers rows 16 u + (wave * 64 + lane) / 16
  // (d = 128) at a swizzled 16-byte chunk, so the offsets of round u are those of round 0 plus u
  // times the round's bytes (the swizzle repeats every 16 rows).
  constexpr uint32_t kRound = C::kWaves * 64 * 16;
  static_assert(kRound % (16 * C::kRowBytes) == 0, "rounds keep the swizzle phase");
  const int row0 = (wave * 64 + lane) / C::kChunks;
  const uint32_t goff = row0 * C::kRowBytes +
                        (((wave * 64 + lane) % C::kChunks) ^ swz<C::kRowBytes>(row0)) * 16;
  const uint32_t wdst = (uint32_t)__builtin_amdgcn_readfirstlane(wave * 1024);
  // next tile to load: first row within its head, and its row in the grp * Nq rows of the heads
  int ld_r = 0;
  int64_t ld_row = 0;
  auto issue_next = [&](int stage) {
    const char* qs = qb + ld_row * C::kRowBytes;
    const char* os = ob + ld_row * C::kRowBytes;
    const uint32_t dst = lbase + stage * C::kStage + wdst;
    if (ld_r + C::kBQ <= nq) {
#pragma unroll
      for (int u = 0; u < C::kLoads; ++u) {
        load_lds16_s(qs + u * kRound, goff, dst + u * kRound);
        load_lds16_s(os + u * kRound, goff, dst + C::kOffO + u * kRound);
      }
      if (wave == 0) load_lds4_s(nlb + ld_row, 4 * lane, dst - wdst + C::kOffL);
      else if (wave == 1) load_lds4_s(deltab + ld_row, 4 * lane, dst - wdst + C::kOffD);
    } else {
      // a head's last tile: rows past Nq are clamped to Nq - 1
      cold_path();
      const int last = nq - 1 - ld_r;
#pragma unroll
      for (int u = 0; u < C::kLoads; ++u) {
        const int row = row0 + u * (kRound / C::kRowBytes);
        const uint32_t off = goff + u * kRound - (row > last ? (row - last) * C::kRowBytes : 0);
        load_lds16_s(qs, off, dst + u * kRound);
        load_lds16_s(os, off, dst + C::kOffO + u * kRound);
      }
      const uint32_t loff = 4 * min(lane, last);
      if (wave == 0) load_lds4_s(nlb + ld_row, loff, dst - wdst + C::kOffL);
      else if (wave == 1) load_lds4_s(deltab + ld_row, loff, dst - wdst + C::kOffD);
    }
    ld_r += C::kBQ;
    ld_row += C::kBQ;
    if (ld_r >= nq) {
      ld_row += nq - ld_r;   // next head
      ld_r = 0;
    }
  };
  // the first three query tiles in flight
#pragma unroll
  for (int s = 0; s < 3; ++s)
    if (s < ntiles) issue_next(s);

  // this wave's 32 keys: K and V rows as B operands (key n, dims 16s + 8g .. +8)
  const int64_t key = k0 + 32 * wave + n;
  const bool key_ok = key < hi;
  bf16x8 kf[C::kDSteps], vf[C::kDSteps];
  {
    const int64_t kr = key_ok ? key : hi - 1;
    const __bf16* kp = k + (bh * Nk + kr) * D + 8 * g;
    const __bf16* vp = v + (bh * Nk + kr) * D + 8 * g;
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) {
      kf[s] = *reinterpret_cast<const bf16x8*>(kp + 16 * s);
      // -V: the dP products then start from D and return D - dP (exact sign flips)
      vf[s] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(vp + 16 * s) ^ (u32x4)0x80008000u);
    }
    // the fragments are in AGPRs, two wait states before the first product that reads them
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) asm volatile("" : "+a"(kf[s]), "+a"(vf[s]));
    asm volatile("s_nop 2");
  }

  // per-lane LDS byte offsets (stage-relative)
  // S / dP: A = Q / dO rows (query 32b + n), chunk 2s + g
  int aoff[C::kDSteps];
#pragma unroll
  for (int s = 0; s < C::kDSteps; ++s) aoff[s] = toff<C::kRowBytes>(n, 2 * s + g);
  // transposed reads of Q / dO (rows = queries, cols = dims): 16-lane group G reads rows
  // j0 + (lane%16)/4 with j0 = 4g + 8h (+16 per query step), columns 32*ct + 16*(G&1) + 4*(lane%4);
  // lane i of the group receives rows j0..j0+3 of column 32*ct + 16*(G&1) + i.
  int qtoff[2][C::kCT];
  {
    const int G = lane >> 4;
    const int trr = (lane & 15) >> 2;
    const int trc = 16 * (G & 1) + 4 * (lane & 3);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ct = 0; ct < C::kCT; ++ct)
        qtoff[h][ct] = eoff<C::kRowBytes>(4 * g + 8 * h + trr, 32 * ct + trc);
  }

  f32x16 dvt[C::kCT], dkt[C::kCT];
#pragma unroll
  for (int c = 0; c < C::kCT; ++c) {
    dvt[c] = f32x16{};
    dkt[c] = f32x16{};
  }

  // Rows tail .. kBQ-1 of a head's last tile are clamped copies: a zero dO row and D make their
  // P dO and dS vanish.  Called between barriers on a stage that has landed.
  auto zero_tail = [&](int stage) {
    char* ot = lds + stage * C::kStage + C::kOffO;
    float* dd = reinterpret_cast<float*>(lds + stage * C::kStage + C::kOffD);
    for (int i = t; i < (C::kBQ - tail) * C::kChunks; i += C::kThreads)
      *reinterpret_cast<u32x4*>(ot + (tail + i / C::kChunks) * C::kRowBytes +
                                (i % C::kChunks) * 16) = u32x4{};
    if (t >= tail && t < C::kBQ) dd[t] = 0.f;
  };
  // position of the tile after the current one, within its head (first row)
  int nx_r = 0;

  wait_vmem<0>();
  __syncthreads();
  if (tail < C::kBQ && nqt == 1) {
    cold_path();
    zero_tail(0);
    __syncthreads();
  }

  constexpr int kM1 = 2 * C::kDSteps;   // S and dP products of one block (phase 1)
  constexpr int kM2 = 4 * C::kCT;       // dV and dK products of one block (phase 2)
  constexpr int kEl = 16 / kM1;         // P/dS elements per phase-1 product
  constexpr int kPf = 16;               // operand reads run this many products ahead
  static_assert(kM1 >= kPf && kM2 >= kPf && kEl * kM1 == 16, "pipeline shape");

  // operand reads, by product index:
  // phase 1 product i: S (i even) or dP (i odd), k-step i/2, of the block at (st, blk)
  auto read_a = [&](int i, int st, int blk) -> bf16x8 {
    const char* base = lds + st + ((i & 1) ? C::kOffO : 0) + 32 * blk * C::kRowBytes;
    return *reinterpret_cast<const bf16x8*>(base + aoff[i >> 1]);
  };
  // phase 2 product i: dV (i even, dO^T) or dK (i odd, Q^T), pair i/2 = (ks, c)
  auto read_t = [&](int i, int st, int blk) -> bf16x8 {
    const int p = i >> 1, ks = p / C::kCT, c = p % C::kCT;
    const char* base = lds + st + ((i & 1) ? 0 : C::kOffO) + (32 * blk + 16 * ks) * C::kRowBytes;
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + qtoff[0][c]));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + qtoff[1][c]));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  auto read_l = [&](int rq, int st, int blk, f32x4& l4) {
    const float* cl =
        reinterpret_cast<const float*>(lds + st + C::kOffL) + 32 * blk + 8 * rq + 4 * g;
    l4 = *reinterpret_cast<const f32x4*>(cl);
  };
  // D of a block in accumulator order (element 4 rq + x is query 8 rq + 4 g + x)
  auto read_d = [&](int st, int blk) -> f32x16 {
    const float* cd = reinterpret_cast<const float*>(lds + st + C::kOffD) + 32 * blk + 4 * g;
    const f32x4 d0 = *reinterpret_cast<const f32x4*>(cd);
    const f32x4 d1 = *reinterpret_cast<const f32x4*>(cd + 8);
    const f32x4 d2 = *reinterpret_cast<const f32x4*>(cd + 16);
    const f32x4 d3 = *reinterpret_cast<const f32x4*>(cd + 24);
    return __builtin_shufflevector(__builtin_shufflevector(d0, d1, 0, 1, 2, 3, 4, 5, 6, 7),
                                   __builtin_shufflevector(d2, d3, 0, 1, 2, 3, 4, 5, 6, 7), 0, 1,
                                   2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
  };

  bf16x8 abuf[kM1];                 // phase-1 A operands in flight (indexed by product)
  bf16x8 tbuf[kM2];                 // phase-2 A operands in flight
  f32x4 lbuf[4];                    // nl of 4-query groups rq of the blocks in flight
  f32x16 dblk;                      // D of the block whose dP products come next

  // P and dS of score element e of a block, in two halves of about equal issue cost: the
  // exponential (reads S), then dS and the packing (reads dP).  pw, sw collect the packed pairs.
  float pe[16], dse[16];
  auto elem_exp = [&](const f32x16& cs, int e) {
    float se = cs[e];
    asm volatile("" : "+v"(se));
    pe[e] = fast_exp2(__builtin_fmaf(se, c2, lbuf[e >> 2][e & 3]));
  };
  auto elem_ds = [&](const f32x16& cp, int e, u32x4& pw, u32x4& sw) {
    float dpe = cp[e];                        // D - dP
    asm volatile("" : "+v"(dpe));
    dse[e] = pe[e] * dpe;                     // -dS
    if (e & 1) {
      uint32_t a2 = pack_bf16x2(pe[e - 1], pe[e]), b2 = pack_bf16x2(dse[e - 1], dse[e]);
      asm volatile("" : "+v"(a2), "+v"(b2));
      pw[(e & 7) >> 1] = a2;
      sw[(e & 7) >> 1] = b2;
    }
  };

  // Phase 1 of block j at (st, blk), scores (cs, cp): the S/dP products of block j+1 (at
  // (st_n, blk_n)) into (ns, np), each beside half of one of the score elements 8..15 of block j
  // (into pf1, sf1).  The last kPf slots start this block's phase-2 reads; nl and D of block j+1's
  // first two query groups are read on the way.
  auto phase1 = [&](const f32x16& cs, const f32x16& cp, f32x16& ns, f32x16& np, bf16x8& pf1,
                    bf16x8& sf1, int st, int blk, int st_n, int blk_n) {
    u32x4 pw, sw;
#pragma unroll
    for (int i = 0; i < kM1; ++i) {
      if (i + kPf < kM1) abuf[i + kPf] = read_a(i + kPf, st_n, blk_n);
      else tbuf[i + kPf - kM1] = read_t(i + kPf - kM1, st, blk);
      if (i == 1 || i == 3) read_l(i >> 1, st_n, blk_n, lbuf[i >> 1]);
      f32x16& acc = (i & 1) ? np : ns;
      const bf16x8 bop = (i & 1) ? vf[i >> 1] : kf[i >> 1];
      if (i == 0) mfma_first_v(acc, abuf[i], bop);
      else if (i == 1) mfma_first_vc(acc, abuf[i], bop, dblk);
      else mfma_acc_v(acc, abuf[i], bop);
#pragma unroll
      for (int u = 0; u < kEl; ++u) {
        const int h = i * kEl + u;            // half-element index 0 .. 15
        const int e = 8 + (h >> 1);
        if (h & 1) elem_ds(cp, e, pw, sw);
        else elem_exp(cs, e);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    pf1 = __builtin_bit_cast(bf16x8, pw);
    sf1 = __builtin_bit_cast(bf16x8, sw);
  };
  // Phase 2 of block j at (st, blk): its dV/dK products with (pf, sf), each beside half of one of
  // the score elements 0..7 of block j+1 (scores (ns, np), into pfn0, sfn0), starting two products
  // late so that the S/dP products just issued have finished.  The last kPf slots start the reads
  // of the next phase 1 (A operands of block j+2 at (st_a, blk_a)); nl and D of block j+1's last
  // two query groups (at (st_n, blk_n)) are read on the way.
  auto phase2 = [&](const bf16x8 (&pf)[2], const bf16x8 (&sf)[2], const f32x16& ns,
                    const f32x16& np, bf16x8& pfn0, bf16x8& sfn0, int st, int blk, int st_n,
                    int blk_n, int st_a, int blk_a) {
    u32x4 pw, sw;
    constexpr int kH = 16 / kM2;              // half-elements per product
#pragma unroll
    for (int i = 0; i < kM2; ++i) {
      if (i + kPf < kM2) {
        tbuf[i + kPf] = read_t(i + kPf, st, blk);
      } else {
        const int k2 = i + kPf - kM2;
        abuf[k2] = read_a(k2, st_a, blk_a);
        if (k2 == 1) dblk = read_d(st_a, blk_a);
      }
      if (i == 1 || i == 3) read_l(2 + (i >> 1), st_n, blk_n, lbuf[2 + (i >> 1)]);
      const int c = (i >> 1) % C::kCT, ks = (i >> 1) / C::kCT;
      if (i & 1) mfma_acc_a(dkt[c], tbuf[i], sf[ks]);
      else mfma_acc_a(dvt[c], tbuf[i], pf[ks]);
#pragma unroll
      for (int u = 0; u < kH; ++u) {
        const int h = i * kH + u - 2;         // half-element index, two products late
        if (h >= 0) {
          const int e = h >> 1;
          if (h & 1) elem_ds(np, e, pw, sw);
          else elem_exp(ns, e);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    elem_exp(ns, 7);
    elem_ds(np, 7, pw, sw);
    pfn0 = __builtin_bit_cast(bf16x8, pw);
    sfn0 = __builtin_bit_cast(bf16x8, sw);
  };

  // Block 0 of every tile lives in (sa, pa, pfa, sfa), block 1 in (sb, pb, pfb, sfb).
  // Prologue: scores of block 0 of tile 0, its elements 0..7, and the reads of its phase 1.
  f32x16 sa, pa, sb, pb;
  bf16x8 pfa[2], sfa[2], pfb[2], sfb[2];
  dblk = read_d(0, 0);
#pragma unroll
  for (int i = 0; i < kM1; ++i) {
    f32x16& acc = (i & 1) ? pa : sa;
    const bf16x8 aop = read_a(i, 0, 0);
    const bf16x8 bop = (i & 1) ? vf[i >> 1] : kf[i >> 1];
    if (i == 0) mfma_first_v(acc, aop, bop);
    else if (i == 1) mfma_first_vc(acc, aop, bop, dblk);
    else mfma_acc_v(acc, aop, bop);
  }
#pragma unroll
  for (int rq = 0; rq < 4; ++rq) read_l(rq, 0, 0, lbuf[rq]);
  // the vector ALU reads these scores next: their products have left the matrix cores by then
  asm volatile("s_nop 15\n\ts_nop 15" : "+v"(sa), "+v"(pa));
  {
    u32x4 pw, sw;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      elem_exp(sa, e);
      elem_ds(pa, e, pw, sw);
    }
    pfa[0] = __builtin_bit_cast(bf16x8, pw);
    sfa[0] = __builtin_bit_cast(bf16x8, sw);
  }
#pragma unroll
  for (int k2 = 0; k2 < kPf; ++k2) abuf[k2] = read_a(k2, 0, 1);
  dblk = read_d(0, 1);
  __builtin_amdgcn_sched_barrier(0);

  // Store mode: the -dS operands of each tile's two 32-query blocks (B operands of the dK
  // products: lane = key n, queries 16 ks + 4 g + (m & 3) + 8 (m >> 2) of the block in element m
  // of sf[ks]) go to the stored-dS layout (ds_unit_offset), each 16-byte fragment at 16 * lane of
  // its 1 KiB half-unit: block 0 of tile it once its dK products are issued, block 1 at the top
  // of tile it+1 (its registers live until then), 4 KiB per wave and tile.  ds_w: this wave's key
  // block in query group 0 of the first query head; ds_t: the current tile's units relative to
  // it (query head st_j of the group, query tile st_qt of that head).
  // (Offsets stay integers added to the kernel argument, so that the compiler keeps the stores
  // global stores; a pointer rebuilt from integers would become a flat store, which also counts
  // against the LDS wait counter.)
  int64_t ds_w = 0, ds_t = 0, ds_head = 0, ds_grp = 0;
  int st_j = 0, st_qt = 0;
  if constexpr (kStore) {
    const int64_t nqg = (Nq + 127) / 128;
    const int64_t nkb = 4 * (int64_t)R * tiles_per_chunk;
    const int64_t kb = ((int64_t)r * tiles_per_chunk + tile) * 4 + wave;
    ds_w = ds_unit_offset(qh0, 0, kb, 0, nqg, nkb);
    ds_grp = 4 * kDsUnitBytes;
    ds_head = nkb * nqg * ds_grp;
  }
  auto ds_store = [&](int64_t off, const bf16x8& x) {
    *reinterpret_cast<u32x4*>(ds + (ds_w + off) + 16 * lane) = __builtin_bit_cast(u32x4, x);
  };

  for (int it = 0; it < ntiles; ++it) {
    const int st_cur = (int)(it & 3) * C::kStage;
    const int st_nxt = (int)((it + 1) & 3) * C::kStage;
    // tile it+1 landed (tile it+2 may stay in flight); every wave is done with tile it-1.  In
    // store mode the stores issued after tile it+1's loads also count: block 0 of tile it-2
    // (it >= 2), block 1 of tile it-2 (it >= 2) and block 0 of tile it-1 (it >= 1), two each.
    if (it + 2 < ntiles) {
      if (!kStore || it == 0) {
        if (wave < 2) wait_vmem<C::kTileOps + 1>();
        else wait_vmem<C::kTileOps>();
      } else if (it == 1) {
        if (wave < 2) wait_vmem<C::kTileOps + 3>();
        else wait_vmem<C::kTileOps + 2>();
      } else {
        if (wave < 2) wait_vmem<C::kTileOps + 7>();
        else wait_vmem<C::kTileOps + 6>();
      }
    } else {
      wait_vmem<0>();
    }
    __syncthreads();
    nx_r += C::kBQ;
    if (nx_r >= nq) nx_r = 0;
    if (it + 1 < ntiles && nx_r + C::kBQ > nq) {
      cold_path();
      zero_tail((int)((it + 1) & 3));
      __syncthreads();
    }
    if constexpr (kStore) {
      if (it > 0) {
        ds_store(ds_t + kDsUnitBytes, sfb[0]);
        ds_store(ds_t + kDsUnitBytes + 1024, sfb[1]);
      }
      // units of tile it: query group st_qt / 2 of head st_j, blocks 2 (st_qt % 2) + 0, 1
      ds_t = st_j * ds_head + (st_qt >> 1) * ds_grp + (st_qt & 1) * 2 * kDsUnitBytes;
      if (++st_qt == nqt) {
        st_qt = 0;
        ++st_j;
      }
    }
    if (it + 3 < ntiles) issue_next((int)((it + 3) & 3));
    __builtin_amdgcn_sched_barrier(0);

    // block 0 of tile it; block 1 of tile it next; then block 0 of tile it+1 (a stale stage after
    // the last tile, whose results are not used)
    phase1(sa, pa, sb, pb, pfa[1], sfa[1], st_cur, 0, st_cur, 1);
    phase2(pfa, sfa, sb, pb, pfb[0], sfb[0], st_cur, 0, st_cur, 1, st_nxt, 0);
    if constexpr (kStore) {
      ds_store(ds_t, sfa[0]);
      ds_store(ds_t + 1024, sfa[1]);
    }
    phase1(sb, pb, sa, pa, pfb[1], sfb[1], st_cur, 1, st_nxt, 0);
    phase2(pfb, sfb, sa, pa, pfa[0], sfa[0], st_cur, 1, st_nxt, 0, st_nxt, 1);
    // after the last products, before any code at the loop exit reads or moves the accumulators
    if (it + 1 == ntiles) asm volatile("s_nop 15\n\ts_nop 15");
  }
  if constexpr (kStore) {
    ds_store(ds_t + kDsUnitBytes, sfb[0]);
    ds_store(ds_t + kDsUnitBytes + 1024, sfb[1]);
  }

  if (key_ok) {
    float* dkr = dk + (bh * Nk + key) * D;
    float* dvr = dv + (bh * Nk + key) * D;
#pragma unroll
    for (int c = 0; c < C::kCT; ++c)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int col = c * 32 + 8 * rq + 4 * g;
        // the dK^T accumulators hold sums of -dS products
        f32x4 kv = {dkt[c][4 * rq] * -scale, dkt[c][4 * rq + 1] * -scale,
                    dkt[c][4 * rq + 2] * -scale, dkt[c][4 * rq + 3] * -scale};
        f32x4 vv = {dvt[c][4 * rq], dvt[c][4 * rq + 1], dvt[c][4 * rq + 2], dvt[c][4 * rq + 3]};
        if (accumulate) {
          kv += *reinterpret_cast<const f32x4*>(dkr + col);
          vv += *reinterpret_cast<const f32x4*>(dvr + col);
        }
        *reinterpret_cast<f32x4*>(dkr + col) = kv;
        *reinterpret_cast<f32x4*>(dvr + col) = vv;
      }
  }
}

template <int D, bool kStore>
hipError_t launch(const BwdArgs& a) {
  using C = DkvCfg<D>;
  const int64_t max_chunk = (a.Nk + a.R - 1) / a.R;
  const int64_t tpc = (max_chunk + C::kBK - 1) / C::kBK;
  static_assert(C::kBK == 128, "stored-dS layout: 128-key tiles");
  const int64_t bhkv = a.BH / a.G;
  // About 16 rounds of 256 workgroups per launch (two K/V heads at the 8-way ring share; store
  // mode: the caller's slab).  The workgroups of an XCD sweep a head's queries together, each tile
  // fetched from HBM once per XCD and round only while they stay in step; over the 128 rounds of a
  // whole-tensor launch they drift apart and fetch 25-76 GB instead of the 20 GB of launches that
  // each end after 16 rounds, at the same speed.
  const int64_t per_launch = kStore ? bhkv : std::max<int64_t>(1, 4096 / (a.R * tpc));
  for (int64_t h0 = 0; h0 < bhkv; h0 += per_launch) {
    const int64_t nh = bhkv - h0 < per_launch ? bhkv - h0 : per_launch;
    // K/V head m serves query heads m G .. m G + G - 1: one launch is a batch of nh K/V heads
    // with G query heads each
    const int64_t q0 = h0 * a.G;
    const int64_t nwg = nh * a.R * tpc;
    hipLaunchKernelGGL((bwd_dkdv_kernel<D, kStore>), dim3((uint32_t)nwg), dim3(C::kThreads), 0,
                       a.stream, (const __bf16*)a.q + q0 * a.Nq * D,
                       (const __bf16*)a.k + h0 * a.Nk * D, (const __bf16*)a.v + h0 * a.Nk * D,
                       (const __bf16*)a.dout + q0 * a.Nq * D, a.nl + q0 * a.Nq,
                       a.delta + q0 * a.Nq, a.dk + h0 * a.Nk * D, a.dv + h0 * a.Nk * D, (int)nh,
                       (int)a.G, (int)a.G, a.Nq, a.Nk, (int)a.R, (int)tpc, a.scale * kLog2e,
                       a.scale, a.accumulate_dkv ? 1 : 0, a.ds);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

hipError_t launch_bwd_dkdv_bf16(const BwdArgs& a) {
  if (a.d == 128) return a.ds ? launch<128, true>(a) : launch<128, false>(a);
  return launch_bwd_dkdv_bf16_d64(a);
}

}  // namespace ringx
