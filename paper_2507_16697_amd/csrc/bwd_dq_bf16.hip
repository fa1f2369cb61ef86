// Recompute backward of ring-chunked attention, dQ part at head size 128: bf16 MFMA with fp32
// accumulation (gfx950).  Head size 64 runs the two-waves-per-SIMD kernel in bwd_dq_bf16_d64.hip.
//
// Query-stationary, like the forward: one workgroup = 4 waves (one per SIMD) = one (b, h) and 256
// queries, 64 per wave as two 32-query blocks.  The key/value sequence is streamed chunk by chunk
// (ring steps, arXiv 2507.16697 Sec. III-A) in tiles of 64 keys that never straddle a chunk,
// through a four-stage LDS ring filled by direct global->LDS loads three tiles ahead.  dQ
// accumulates over every tile of every chunk in fp32 registers and is written once, so it needs no
// atomics (the paper's "gradient for Q accumulated over N steps").  Per 32-key block ("unit") and
// query block, with lane = query n and g = lane / 32:
//   S^T  = K Q^T      A = K rows (LDS),  B = Q^T from registers
//   dP^T - D = V dO^T - D   A = V rows (LDS), B = dO^T from registers, accumulators start at -D
//   P^T  = exp2(S^T * scale*log2e - lse_q*log2e),  dS^T = P^T (dP^T - D_q)   (lse_q, D_q are
//          per-lane scalars because each lane holds one query; -D_q fills a 16-register block
//          per query block that starts every dP^T chain, so the subtraction rides on the
//          matrix cores)
//   dQ^T += K^T dS^T  A = K^T by transposed reads of the row-major K tile, B = dS^T from the
//          registers (keys 4g..4g+3, 8+4g..8+4g+3 of each 16-key step, as in the forward)
// Every LDS operand feeds the products of both query blocks, so a wave reads half a KiB of LDS per
// matrix product.
//
// One wave per SIMD, so each wave runs a fixed schedule, software pipelined over units: phase 1 of
// unit u issues the 32 S/dP products of unit u+1, beside the P/dS arithmetic of three of the four
// 8-element groups of unit u; phase 2 issues the 16 dQ products of unit u, beside the first group
// of unit u+1 (started a few products late, so that the S/dP products just issued have
// finished).  A product slot carries at most one element (fma, exp, multiply, half a pack; the
// subtraction of D rides on the products): one hides behind the 32-cycle product, two do not.
// LDS operands are read 10 products ahead.  Key rows past the end of a chunk (last tile of a
// chunk) are clamped copies of its last key; in the units that hold them (a branch outside the
// product schedule, between the phases) their scores are set to -inf once the S^T products have
// finished, so P and dS are exactly 0 there whatever the row's lse.
//
// Register files: Q/dO fragments (128) and the dQ^T accumulators (128) in AGPRs, the S/dP
// accumulators of two units, dS^T and the operands in flight in VGPRs; the products are the
// inline-assembly forms of ringx_device.h, whose hazard rules this schedule keeps (checked by the
// tests in the built code).

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

template <int D>
struct DqCfg {
  static constexpr int kThreads = 256;
  static constexpr int kWaves = 4;
  static constexpr int kQW = 64;                   // queries per wave (two 32-query blocks)
  static constexpr int kBQ = kWaves * kQW;         // queries per workgroup
  static constexpr int kBK = 64;                   // keys per tile (two units)
  static constexpr int kRowBytes = D * 2;
  static constexpr int kChunks = D / 8;
  static constexpr int kTile = kBK * kRowBytes;    // bytes of one K or V tile
  static constexpr int kDSteps = D / 16;
  static constexpr int kCT = D / 32;
  static constexpr int kLoads = kTile / (kThreads * 16);   // 16-byte loads per thread per tile
  static constexpr int kStage = 2 * kTile;         // K tile, then V tile
  static constexpr int kStages = 4;
  static constexpr int kLds = kStages * kStage;
  static constexpr int kTileOps = 2 * kLoads;      // vector-memory operations per wave per tile
  static_assert(kLoads >= 1 && kTile == kLoads * kThreads * 16, "whole tiles per load round");
};

template <int D>
__device__ __forceinline__ int swz(int row) {
  if constexpr (D == 128) return ((row & 3) << 2) | ((row >> 2) & 3);
  else return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
}
template <int D>
__device__ __forceinline__ int tile_off(int row, int c) {
  return row * (D * 2) + ((c ^ swz<D>(row)) << 4);
}

template <int D>
__global__ __launch_bounds__(256, 1) void bwd_dq_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const __bf16* __restrict__ dout, const float* __restrict__ lse,
    const float* __restrict__ delta, float* __restrict__ dq, int BH, int H, int grp, int64_t Nq,
    int64_t Nk, int R, float c2, float scale, int accumulate) {
  using C = DqCfg<D>;
  __shared__ __attribute__((aligned(1024))) char lds[C::kLds];
  const uint32_t lbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int n = lane & 31;
  const int g = lane >> 5;

  const int64_t nqt = (Nq + C::kBQ - 1) / C::kBQ;
  const uint32_t wg = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t bh = wg / nqt;
  const int64_t q0 = (wg % nqt) * C::kBQ + wave * C::kQW;
  if (bh >= BH) return;

  const int64_t kvh = kv_head(bh, H, grp);
  // wave-uniform bases in SGPRs, so that the per-tile load addresses are scalar arithmetic
  const char* kb =
      static_cast<const char*>(uniform_ptr(reinterpret_cast<const char*>(k + kvh * Nk * D)));
  const char* vb =
      static_cast<const char*>(uniform_ptr(reinterpret_cast<const char*>(v + kvh * Nk * D)));

  // Tiles: chunk r covers keys [r Nk / R, (r+1) Nk / R), cut into 64-key tiles from its start.
  // ld_t: the next tile to load; nx_t: the tile after the one being computed (32-bit positions
  // walked without divisions, so that the loop's bookkeeping stays scalar).
  const uint32_t nk = (uint32_t)Nk;
  ChunkWalk ld_w{nk, nk / (uint32_t)R, nk % (uint32_t)R, 0, (uint32_t)R};
  ChunkWalk nx_w = ld_w;
  KeyTile ld_t = ld_w.first();
  KeyTile nx_t = nx_w.first();
  int ntiles = 0;
  for (int r = 0; r < R; ++r) {
    const int64_t lo = (int64_t)r * Nk / R, hi = (int64_t)(r + 1) * Nk / R;
    ntiles += (int)((hi - lo + C::kBK - 1) / C::kBK);
  }

  // per-lane offsets of the tile loads: round u covers rows 16 u + (wave * 64 + lane) / 16 at a
  // swizzled chunk, so round u's offsets are round 0's plus u rounds (the swizzle repeats every 16
  // rows)
  constexpr uint32_t kRound = C::kWaves * 64 * 16;
  static_assert(kRound % (16 * C::kRowBytes) == 0, "rounds keep the swizzle phase");
  const int row0 = (wave * 64 + lane) / C::kChunks;
  const uint32_t goff =
      row0 * C::kRowBytes + (((wave * 64 + lane) % C::kChunks) ^ swz<D>(row0)) * 16;
  const uint32_t wdst = (uint32_t)__builtin_amdgcn_readfirstlane(wave * 1024);
  auto issue_next = [&](int stage) {
    const char* ks = kb + (uint64_t)ld_t.start * C::kRowBytes;
    const char* vs = vb + (uint64_t)ld_t.start * C::kRowBytes;
    const uint32_t dst = lbase + stage * C::kStage + wdst;
    if (ld_t.start + C::kBK <= ld_t.hi) {
#pragma unroll
      for (int u = 0; u < C::kLoads; ++u) {
        load_lds16_s(ks + u * kRound, goff, dst + u * kRound);
        load_lds16_s(vs + u * kRound, goff, dst + C::kTile + u * kRound);
      }
    } else {
      // the last tile of a chunk: rows past its end are clamped to the chunk's last key
      cold_path();
      const int last = (int)(ld_t.hi - 1 - ld_t.start);
#pragma unroll
      for (int u = 0; u < C::kLoads; ++u) {
        const int row = row0 + u * (kRound / C::kRowBytes);
        const uint32_t off = goff + u * kRound - (row > last ? (row - last) * C::kRowBytes : 0);
        load_lds16_s(ks, off, dst + u * kRound);
        load_lds16_s(vs, off, dst + C::kTile + u * kRound);
      }
    }
    ld_t = ld_w.next<C::kBK>(ld_t);
  };

#pragma unroll
  for (int s = 0; s < 3; ++s)
    if (s < ntiles) issue_next(s);

  // this lane's two queries: Q and dO fragments (B operands, in AGPRs), -lse*log2e and D
  bf16x8 qf[2][C::kDSteps], of[2][C::kDSteps];
  float nl[2], dd[2];
  bool q_ok[2];
  int64_t qrow[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    int64_t qi = q0 + 32 * b + n;
    q_ok[b] = qi < Nq;
    qi = q_ok[b] ? qi : Nq - 1;
    qrow[b] = qi;
    const __bf16* qr = q + (bh * Nq + qi) * D;
    const __bf16* orow = dout + (bh * Nq + qi) * D;
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) {
      qf[b][s] = *reinterpret_cast<const bf16x8*>(qr + s * 16 + g * 8);
      of[b][s] = *reinterpret_cast<const bf16x8*>(orow + s * 16 + g * 8);
    }
    nl[b] = -lse[bh * Nq + qi] * kLog2e;
    dd[b] = delta[bh * Nq + qi];
  }
  // -D of each query block as the start of its dP^T chains (the lane's query is the same for all
  // 16 accumulators), so that the products return dP - D
  f32x16 negd[2];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int e = 0; e < 16; ++e) negd[b][e] = -dd[b];
  // the fragments are in AGPRs and -D in VGPRs, two wait states before the first product that
  // reads them
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) asm volatile("" : "+a"(qf[b][s]), "+a"(of[b][s]));
  asm volatile("" : "+v"(negd[0]), "+v"(negd[1]));
  asm volatile("s_nop 2");

  // per-lane LDS offsets: K/V rows (A operands of S^T, dP^T) and transposed K (A of dQ^T)
  int koff[C::kDSteps];
#pragma unroll
  for (int s = 0; s < C::kDSteps; ++s) koff[s] = tile_off<D>(n, 2 * s + g);
  int toff[2][C::kCT];
  {
    const int G = lane >> 4;
    const int rr = (lane & 15) >> 2;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ct = 0; ct < C::kCT; ++ct) {
        const int row = 4 * g + 8 * h + rr;
        const int col = 32 * ct + 16 * (G & 1) + 4 * (lane & 3);
        toff[h][ct] = tile_off<D>(row, col >> 3) + (col & 7) * 2;
      }
  }

  f32x16 dqacc[2][C::kCT];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int c = 0; c < C::kCT; ++c) dqacc[b][c] = f32x16{};

  // keys of the tile being computed (cur_valid) and of the next one (nx_valid) that lie inside
  // their chunk: 64 except in the last tile of a chunk
  int cur_valid = (int)min<uint32_t>(C::kBK, nx_t.hi - nx_t.start);
  int nx_valid = C::kBK;

  wait_vmem<0>();
  __syncthreads();

  constexpr int kM1 = 4 * C::kDSteps;   // S and dP products of one unit, both query blocks
  constexpr int kM2 = 4 * C::kCT;       // dQ products of one unit, both query blocks
  constexpr int kPf = 10;               // operand reads run this many products ahead
  constexpr int kLate = 4;              // phase 2 starts its arithmetic this many products late
  static_assert(kM1 >= kPf && kM2 >= kPf && kM2 - kLate >= 8, "pipeline shape");

  // LDS operands.  Phase 1 product i: S (i % 4 < 2) or dP, query block i % 2, k-step i / 4; its
  // A operand (K or V rows of the unit's 32 keys) is shared by products 2j and 2j+1.
  auto read_a = [&](int i, int st, int kbk) -> bf16x8 {
    const char* base = lds + st + ((i & 2) ? C::kTile : 0) + 32 * kbk * C::kRowBytes;
    return *reinterpret_cast<const bf16x8*>(base + koff[i >> 2]);
  };
  // Phase 2 product j: query block j % 2, pair j / 2 = (ks, c); A = K^T of the unit's keys
  // 16 ks .. 16 ks + 15
  auto read_t = [&](int j, int st, int kbk) -> bf16x8 {
    const int p = j >> 1, ks = p / C::kCT, c = p % C::kCT;
    const char* base = lds + st + (32 * kbk + 16 * ks) * C::kRowBytes;
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + toff[0][c]));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + toff[1][c]));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };

  bf16x8 abuf[kM1 / 2];             // phase-1 A operands in flight (one per product pair)
  bf16x8 tbuf[kM2 / 2];             // phase-2 A operands in flight

  // P/dS of score element k (0 .. 31) of a unit: group k / 8 = (query block b, k-step ks), element
  // 8 ks + k % 8 of b's accumulators.  Pairs are packed as dS^T B operands after their second
  // element.
  float dse[2][16];
  auto elem = [&](const f32x16 (&sc)[2], const f32x16 (&dp)[2], int k, u32x4 (&sw)[2][2]) {
    const int grp_i = k >> 3, e8 = k & 7;
    const int b = grp_i & 1, ks = grp_i >> 1;
    const int e = 8 * ks + e8;
    float se = sc[b][e], de = dp[b][e];   // de = dP - D
    asm volatile("" : "+v"(se), "+v"(de));
    const float pe = fast_exp2(__builtin_fmaf(se, c2, nl[b]));
    dse[b][e] = pe * de;
    if (e8 & 1) {
      uint32_t a2 = pack_bf16x2(dse[b][e - 1], dse[b][e]);
      asm volatile("" : "+v"(a2));
      sw[b][ks][e8 >> 1] = a2;
    }
  };

  // Phase 1 of unit u (stage st, key block kbk; scores sc, dp) computes the S/dP of unit u+1 (at
  // (st_n, kbk_n)) into (nsc, ndp), beside elements 8 .. 31 of unit u (groups 1..3) into sw, at
  // most one per product; its last kPf slots start unit u's phase-2 reads.
  auto phase1 = [&](const f32x16 (&sc)[2], const f32x16 (&dp)[2], f32x16 (&nsc)[2],
                    f32x16 (&ndp)[2], u32x4 (&sw)[2][2], int st, int kbk, int st_n, int kbk_n) {
    constexpr int kE = 24;            // elements carried by this phase
#pragma unroll
    for (int i = 0; i < kM1; ++i) {
      if (((i + kPf) & 1) == 0) {
        if (i + kPf < kM1) abuf[(i + kPf) >> 1] = read_a(i + kPf, st_n, kbk_n);
        else tbuf[(i + kPf - kM1) >> 1] = read_t(i + kPf - kM1, st, kbk);
      }
      const int s = i >> 2, b = i & 1;
      const bool is_dp = (i & 2) != 0;
      f32x16& acc = is_dp ? ndp[b] : nsc[b];
      const bf16x8 bop = is_dp ? of[b][s] : qf[b][s];
      if (s == 0 && is_dp) mfma_first_vc(acc, abuf[i >> 1], bop, negd[b]);
      else if (s == 0) mfma_first_v(acc, abuf[i >> 1], bop);
      else mfma_acc_v(acc, abuf[i >> 1], bop);
#pragma unroll
      for (int e = (i * kE) / kM1; e < ((i + 1) * kE) / kM1; ++e) elem(sc, dp, 8 + e, sw);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Phase 2 of unit u (stage st, key block kbk): its dQ products with B operands sf, beside
  // elements 0 .. 7 of unit u+1 (group 0, scores nsc/ndp) into nsw, from product kLate on;
  // its last kPf slots start the reads of unit u+1's phase 1 (A operands of unit u+2 at
  // (st_a, kbk_a)).
  auto phase2 = [&](const bf16x8 (&sf)[2][2], const f32x16 (&nsc)[2], const f32x16 (&ndp)[2],
                    u32x4 (&nsw)[2][2], int st, int kbk, int st_a, int kbk_a) {
    constexpr int kSlots = kM2 - kLate;
#pragma unroll
    for (int j = 0; j < kM2; ++j) {
      if (((j + kPf) & 1) == 0) {
        if (j + kPf < kM2) tbuf[(j + kPf) >> 1] = read_t(j + kPf, st, kbk);
        else abuf[(j + kPf - kM2) >> 1] = read_a(j + kPf - kM2, st_a, kbk_a);
      }
      const int p = j >> 1, ks = p / C::kCT, c = p % C::kCT, b = j & 1;
      mfma_acc_a(dqacc[b][c], tbuf[j >> 1], sf[b][ks]);
      if (j >= kLate) {
        const int i2 = j - kLate;
#pragma unroll
        for (int e = (i2 * 8) / kSlots; e < ((i2 + 1) * 8) / kSlots; ++e) elem(nsc, ndp, e, nsw);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Scores of key rows nvalid .. 31 of a unit (S^T rows 8 (e / 4) + 4 g + e % 4) to -inf, so
  // that P = 0 and dS = 0 for keys past the end of a chunk.  Cold: only the last tile of a chunk
  // whose length is not a multiple of 64 gets here.  The wait lets the S^T products finish.
  auto mask_rows = [&](f32x16 (&sc)[2], int nvalid) {
    cold_path();
    asm volatile("s_nop 15\n\ts_nop 15" : "+v"(sc[0]), "+v"(sc[1]));
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (8 * (e >> 2) + 4 * g + (e & 3) >= nvalid) sc[b][e] = -INFINITY;
  };

  // Unit 0 of every tile lives in (sa, pa, swa), unit 1 in (sb, pb, swb).
  f32x16 sa[2], pa[2], sb[2], pb[2];
  u32x4 swa[2][2], swb[2][2];
  auto as_bf16 = [](const u32x4 (&w)[2][2], bf16x8 (&f)[2][2]) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) f[b][ks] = __builtin_bit_cast(bf16x8, w[b][ks]);
  };

  // prologue: scores of unit 0 (tile 0, key block 0), its group 0, the reads of its phase 1
#pragma unroll
  for (int i = 0; i < kM1; ++i) {
    const int s = i >> 2, b = i & 1;
    const bool is_dp = (i & 2) != 0;
    f32x16& acc = is_dp ? pa[b] : sa[b];
    const bf16x8 aop = read_a(i, 0, 0);
    const bf16x8 bop = is_dp ? of[b][s] : qf[b][s];
    if (s == 0 && is_dp) mfma_first_vc(acc, aop, bop, negd[b]);
    else if (s == 0) mfma_first_v(acc, aop, bop);
    else mfma_acc_v(acc, aop, bop);
  }
  asm volatile("s_nop 15\n\ts_nop 15" : "+v"(sa[0]), "+v"(sa[1]), "+v"(pa[0]), "+v"(pa[1]));
  if (cur_valid < 32) mask_rows(sa, cur_valid);
#pragma unroll
  for (int e = 0; e < 8; ++e) elem(sa, pa, e, swa);
#pragma unroll
  for (int i = 0; i < kPf; i += 2) abuf[i >> 1] = read_a(i, 0, 1);
  __builtin_amdgcn_sched_barrier(0);

  for (int it = 0; it < ntiles; ++it) {
    const int st_cur = (it & 3) * C::kStage;
    const int st_nxt = ((it + 1) & 3) * C::kStage;
    // tile it+1 landed (tile it+2 may stay in flight); every wave is done with tile it-1
    if (it + 2 < ntiles) wait_vmem<C::kTileOps>();
    else wait_vmem<0>();
    __syncthreads();
    nx_t = nx_w.next<C::kBK>(nx_t);
    if (it + 1 < ntiles) nx_valid = (int)min<uint32_t>(C::kBK, nx_t.hi - nx_t.start);
    if (it + 3 < ntiles) issue_next((it + 3) & 3);
    __builtin_amdgcn_sched_barrier(0);

    bf16x8 sf[2][2];
    // unit 0 of tile it (next: unit 1 of tile it; then unit 0 of tile it+1, a stale stage after
    // the last tile, whose results are not used)
    phase1(sa, pa, sb, pb, swa, st_cur, 0, st_cur, 1);
    if (cur_valid < C::kBK) mask_rows(sb, cur_valid - 32);
    as_bf16(swa, sf);
    phase2(sf, sb, pb, swb, st_cur, 0, st_nxt, 0);
    phase1(sb, pb, sa, pa, swb, st_cur, 1, st_nxt, 0);
    if (nx_valid < 32) mask_rows(sa, nx_valid);
    as_bf16(swb, sf);
    phase2(sf, sa, pa, swa, st_cur, 1, st_nxt, 1);
    cur_valid = nx_valid;
    // after the last products, before any code at the loop exit reads or moves the accumulators
    if (it + 1 == ntiles) asm volatile("s_nop 15\n\ts_nop 15");
  }

#pragma unroll
  for (int b = 0; b < 2; ++b) {
    if (!q_ok[b]) continue;
    float* dqr = dq + (bh * Nq + qrow[b]) * D;
#pragma unroll
    for (int c = 0; c < C::kCT; ++c)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        f32x4 val = {dqacc[b][c][4 * rq] * scale, dqacc[b][c][4 * rq + 1] * scale,
                     dqacc[b][c][4 * rq + 2] * scale, dqacc[b][c][4 * rq + 3] * scale};
        f32x4* dst = reinterpret_cast<f32x4*>(dqr + c * 32 + 8 * rq + 4 * g);
        if (accumulate) val += *dst;
        *dst = val;
      }
  }
}

template <int D>
hipError_t launch(const BwdArgs& a) {
  using C = DqCfg<D>;
  const int64_t nqt = (a.Nq + C::kBQ - 1) / C::kBQ;
  const int64_t nwg = nqt * a.BH;
  hipLaunchKernelGGL((bwd_dq_kernel<D>), dim3((uint32_t)nwg), dim3(C::kThreads), 0, a.stream,
                     (const __bf16*)a.q, (const __bf16*)a.k, (const __bf16*)a.v,
                     (const __bf16*)a.dout, a.lse, a.delta, a.dq, (int)a.BH, (int)a.H, (int)a.G,
                     a.Nq, a.Nk, (int)a.R, a.scale * kLog2e, a.scale, a.accumulate_dq ? 1 : 0);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd_dq_bf16(const BwdArgs& a) {
  if (a.d == 128) return launch<128>(a);
  return launch_bwd_dq_bf16_d64(a);
}

}  // namespace ringx
