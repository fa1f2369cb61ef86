// Ring-chunked attention forward, bf16 storage, bf16 MFMA with fp32 accumulation (gfx950).
//
// One workgroup = 8 waves (two per SIMD) = one (b, h) and a tile of 256 queries (32 per wave), so
// that each K/V tile brought into LDS serves 256 queries.  The key/value
// sequence is visited as R chunks (ring steps, arXiv 2507.16697 Sec. III-A), streamed through LDS
// in tiles of 64 keys that never straddle a chunk boundary.  K and V tiles are double buffered
// (the on-chip analogue of the paper's ping-pong buffers) and filled by direct global->LDS loads:
// while tile j is processed, the K tile j+2 and the V tile j+1 are in flight.
//
// Each wave is software pipelined over key tiles: the MFMAs of S_{j+1} = K_{j+1} Q^T are
// interleaved with the exponentials and row sums of tile j, so that the matrix cores and the
// vector ALU work at the same time (the other wave of the SIMD runs its O += V^T P^T products
// meanwhile).  Per wave, with g = lane / 32 and n = lane % 32:
//   S^T = K Q^T   A = K rows from LDS (key n, 8 dims), B = Q^T from registers (query n, 8 dims)
//                 -> lane holds query n and keys 8*(r/4) + 4g + r%4 of each 32-key block;
//   O^T += V^T P^T A = V^T read from the row-major V tile with ds_read_b64_tr_b16 (4 keys per
//                 read), B = P^T straight from the S^T registers (keys 4g..4g+3, 8+4g..8+4g+3).
// LDS tiles are row-major with the 16-byte chunks of each row XOR-swizzled by the row index, so
// that both the 16-byte K reads (16 rows, one chunk) and the transposed V reads (4 rows x 2
// chunks per 16 lanes) hit distinct banks.
//
// Softmax statistics are fp32 in the exp2 domain (t = scale*log2(e)*q.k).  Eqs. (2)-(3) hold for
// any per-row reference m, not only the running maximum, so no row maximum is taken per tile: a
// tile's probabilities exp2(t - m) are formed against the current m, and only when a lane's sum
// of them reaches 2^32 (or is not finite, as on the first tile, whose m is still -inf) is the tile
// redone with m moved to its row maximum and the accumulators rescaled.  A lane's sum bounds each
// of its terms, so every probability stays below 2^32: bf16 and fp32 keep the same relative
// precision at any magnitude, and a row sum or output accumulator of at most 2^32 per key stays
// far inside the fp32 range for any realistic V.  At the end of chunk r the
// wave forms the chunk's log-sum-exp loc_lse_r from the chunk's own row sum and folds it into the
// merged lse by Eq. (5).  The output numerator is kept unnormalised: Eq. (5)'s term
// exp(loc_lse_r - M) loc_out_r equals exp(m - M) times the chunk's unnormalised accumulator, so
// one accumulator holds the running sum of all chunk terms and the final division by the Eq. (5)
// denominator is a multiplication by 2^(m - lse).  MODE kPartials instead writes every chunk's
// (loc_out_r, loc_lse_r) and restarts the accumulator; MODE kStep (one chunk, R = 1) merges the
// chunk's result into a running fp32 (acc_out, acc_lse) by Eq. (5), one ring step at a time.

#include "ringx_device.h"
#include "ringx_kernels.h"

#include <type_traits>

namespace ringx {
namespace {

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr float kGuard = 4294967296.0f;   // 2^32: bound on a lane's probability sum

template <int D>
struct FwdCfg {
  static constexpr int kThreads = 512;
  static constexpr int kWaves = 8;
  static constexpr int kQW = 32;                  // queries per wave
  static constexpr int kBQ = kWaves * kQW;        // queries per workgroup
  static constexpr int kBK = 64;                  // keys per tile
  static constexpr int kRowBytes = D * 2;
  static constexpr int kChunks = D / 8;           // 16-byte chunks per row
  static constexpr int kTileBytes = kBK * kRowBytes;   // 16 KiB (d=128), 8 KiB (d=64)
  static constexpr int kKTiles = kBK / 32;        // 32-key blocks per tile
  static constexpr int kDSteps = D / 16;          // MFMA k-steps over the head dim
  static constexpr int kKSteps = kBK / 16;        // MFMA k-steps over the keys
  static constexpr int kCT = D / 32;              // 32-dim blocks of the output
  // Only waves 0..3, one on each SIMD, issue the tile loads: while a wave waits for the CU's load
  // path to take its loads, the other wave of its SIMD keeps the matrix core busy (2% faster at
  // d = 128 and 5% at d = 64 than all eight waves issuing at once; two loader waves: 1% and 3%).
  static constexpr int kLoaders = 4;
  static constexpr int kLoads = kTileBytes / (kLoaders * 64 * 16);   // 16-byte loads per loader lane
};

// Swizzled 16-byte chunk of (row, logical chunk c) inside a row-major tile.
template <int D>
__device__ __forceinline__ int swz(int row) {
  if constexpr (D == 128) return ((row & 3) << 2) | ((row >> 2) & 3);
  else return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
}
template <int D>
__device__ __forceinline__ int tile_off(int row, int c) {   // byte offset
  return row * (D * 2) + ((c ^ swz<D>(row)) << 4);
}


// Per-lane byte offsets (from the tile's first row) of this lane's direct loads: 16-byte slot
// `slot` of the swizzled tile holds logical chunk (slot % chunks) ^ swz(row) of row slot / chunks.
template <int D>
__device__ __forceinline__ void load_offsets(int (&goff)[FwdCfg<D>::kLoads],
                                             int (&grow)[FwdCfg<D>::kLoads], int wave, int lane) {
  using C = FwdCfg<D>;
#pragma unroll
  for (int u = 0; u < C::kLoads; ++u) {
    const int slot = (u * C::kLoaders + (wave % C::kLoaders)) * 64 + lane;
    const int row = slot / C::kChunks;
    const int c = (slot % C::kChunks) ^ swz<D>(row);
    grow[u] = row;
    goff[u] = row * C::kRowBytes + c * 16;
  }
}

// Issue the direct loads of one K or V tile starting at key `start` into the LDS buffer at
// `dst`; rows at or past `hi` (only in the last tile of a chunk) are clamped to hi - 1.
// `wdst` is the loader wave's first 1 KiB slot (wave * 1024, an SGPR).
template <int D>
__device__ __forceinline__ void issue_tile(const char* __restrict__ base, uint32_t dst,
                                           uint32_t start, uint32_t hi,
                                           const int (&goff)[FwdCfg<D>::kLoads],
                                           const int (&grow)[FwdCfg<D>::kLoads], int wave,
                                           uint32_t wdst) {
  using C = FwdCfg<D>;
  if (wave >= C::kLoaders) return;
  const char* src = base + (uint64_t)start * C::kRowBytes;
  if (start + C::kBK <= hi) {
#pragma unroll
    for (int u = 0; u < C::kLoads; ++u)
      load_lds16_s(src, (uint32_t)goff[u], dst + wdst + u * C::kLoaders * 1024);
  } else {
    cold_path();
    const int last = (int)(hi - 1 - start);
#pragma unroll
    for (int u = 0; u < C::kLoads; ++u) {
      const int off = grow[u] <= last ? goff[u] : goff[u] - (grow[u] - last) * C::kRowBytes;
      load_lds16_s(src, (uint32_t)off, dst + wdst + u * C::kLoaders * 1024);
    }
  }
}

template <int D, int MODE>
__global__ __launch_bounds__(512, 1) void fwd_bf16_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    __bf16* __restrict__ out, float* __restrict__ lse, float* __restrict__ part_out,
    float* __restrict__ part_lse, float* __restrict__ acc_out, float* __restrict__ acc_lse,
    int first, int BH, int H, int grp, int64_t Nq, int64_t Nk, int R, float c2) {
  using C = FwdCfg<D>;
  constexpr bool kPartials = MODE == (int)FwdMode::kPartials;
  constexpr bool kStep = MODE == (int)FwdMode::kStep;
  __shared__ __attribute__((aligned(1024))) char lds_k[2 * C::kTileBytes];
  __shared__ __attribute__((aligned(1024))) char lds_v[2 * C::kTileBytes];

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

  const __bf16* qb = q + bh * Nq * D;
  const int64_t kvh = kv_head(bh, H, grp);
  // wave-uniform bases in SGPRs, so that the per-tile load addresses are scalar arithmetic
  const char* kb =
      static_cast<const char*>(uniform_ptr(reinterpret_cast<const char*>(k + kvh * Nk * D)));
  const char* vb =
      static_cast<const char*>(uniform_ptr(reinterpret_cast<const char*>(v + kvh * Nk * D)));
  int goff[C::kLoads], grow[C::kLoads];
  load_offsets<D>(goff, grow, wave, lane);

  const uint32_t nk = (uint32_t)Nk;
  ChunkWalk walk{nk, nk / (uint32_t)R, nk % (uint32_t)R, 0, (uint32_t)R};
  uint32_t wdst = (uint32_t)__builtin_amdgcn_readfirstlane(wave * 1024);
  KeyTile t0 = walk.first();
  KeyTile t1 = walk.next<C::kBK>(t0);
  KeyTile t2 = walk.next<C::kBK>(t1);
  int r0 = 0;   // chunk of t0

  // LDS byte addresses of the two K and two V buffers
  const uint32_t lk = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_k;
  const uint32_t lv = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_v;

  // K_0, V_0 and K_1 in flight while Q is loaded
  issue_tile<D>(kb, lk, t0.start, t0.hi, goff, grow, wave, wdst);
  issue_tile<D>(vb, lv, t0.start, t0.hi, goff, grow, wave, wdst);
  if (t1.start < nk)
    issue_tile<D>(kb, lk + C::kTileBytes, t1.start, t1.hi, goff, grow, wave, wdst);

  // Q fragments (B operand of S^T = K Q^T): query n of this wave, dims 16*ks + 8g .. +8.
  bf16x8 qf[C::kDSteps];
  {
    int64_t qi = q0 + n;
    qi = qi < Nq ? qi : Nq - 1;
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s)
      qf[s] = *reinterpret_cast<const bf16x8*>(qb + qi * D + s * 16 + g * 8);
  }

  // per-lane LDS byte offsets (tile-relative)
  int koff[C::kDSteps];   // K fragment of 32-key block 0 at k-step s (block kt adds kt*32 rows)
#pragma unroll
  for (int s = 0; s < C::kDSteps; ++s) koff[s] = tile_off<D>(n, 2 * s + g);
  // V^T fragments via transposed reads: for 16-lane group G, rows j0 + (lane%16)/4 with
  // j0 = 16*ks + 4g (+8 for the second half), columns 32*ct + 16*(G%2) + 4*(lane%4).
  int voff[2][C::kCT];
  {
    const int G = lane >> 4;
    const int rr = (lane & 15) >> 2;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ct = 0; ct < C::kCT; ++ct) {
        const int row = 4 * g + 8 * h + rr;
        const int col = 32 * ct + 16 * (G & 1) + 4 * (lane & 3);
        voff[h][ct] = tile_off<D>(row, col >> 3) + (col & 7) * 2;
      }
  }

  f32x16 oacc[C::kCT];
#pragma unroll
  for (int c = 0; c < C::kCT; ++c) oacc[c] = f32x16{};
  float m2 = -INFINITY;     // reference max of the row (exp2 domain)
  float lc = 0.f;           // this lane's share of the chunk's row sum, relative to m2
  float lse2m = -INFINITY;  // merged log2-sum-exp over finished chunks (Eq. (5))

  wait_vmem_all();
  __syncthreads();

  // S_0
  f32x16 sa[C::kKTiles], sb[C::kKTiles];
#pragma unroll
  for (int kt = 0; kt < C::kKTiles; ++kt) sa[kt] = f32x16{};
#pragma unroll
  for (int s = 0; s < C::kDSteps; ++s)
#pragma unroll
    for (int kt = 0; kt < C::kKTiles; ++kt)
      sa[kt] = mfma32(*reinterpret_cast<const bf16x8*>(lds_k + koff[s] + kt * 32 * C::kRowBytes),
                      qf[s], sa[kt]);

  // One pipelined iteration for tile t0 (scores in `cur`); parity P selects the buffers: K_{j+1}
  // is read from K buffer 1-P, V_j from V buffer P; K_{j+2} lands in K buffer P, V_{j+1} in V
  // buffer 1-P.  Returns true after the last tile.
  auto step = [&](f32x16 (&cur)[C::kKTiles], f32x16 (&nxt)[C::kKTiles], auto parity) -> bool {
    constexpr int P = decltype(parity)::value;
    // K_{j+1} and V_j landed (issued one iteration ago); every wave is done with K_j, V_{j-1}
    wait_vmem_all();
    __syncthreads();
    // wdst counts as redefined here, so that the load slots' addresses are formed at each use
    // (scalar adds) instead of being held in registers across the loop
    asm volatile("" : "+s"(wdst));
    if (t2.start < nk)
      issue_tile<D>(kb, lk + P * C::kTileBytes, t2.start, t2.hi, goff, grow, wave, wdst);
    if (t1.start < nk)
      issue_tile<D>(vb, lv + (1 - P) * C::kTileBytes, t1.start, t1.hi, goff, grow, wave, wdst);
    // The vector work of this half (exponentials, row sums) is the longer chain; it issues ahead
    // of the other wave's matrix products on the SIMD, which fill the gaps (priority drops again
    // for the P V half).
    __builtin_amdgcn_s_setprio(1);

    // last tile of a chunk: keys past the chunk end (clamped copies of its last key) add nothing
    const int nvalid = (int)min<uint32_t>(C::kBK, t0.hi - t0.start);
    if (nvalid < C::kBK) {
      cold_path();
      const int thr = nvalid - 4 * g;   // key 4g + off is past the end iff off >= thr
#pragma unroll
      for (int kt = 0; kt < C::kKTiles; ++kt)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr)
          if (kt * 32 + 8 * (rr >> 2) + (rr & 3) >= thr) cur[kt][rr] = -INFINITY;
    }
    // S_{j+1} = K_{j+1} Q^T on the matrix cores, P_j = exp2(t - m) on the vector ALU
    const char* kbuf = lds_k + (1 - P) * C::kTileBytes;
#pragma unroll
    for (int kt = 0; kt < C::kKTiles; ++kt) nxt[kt] = f32x16{};
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s)
#pragma unroll
      for (int kt = 0; kt < C::kKTiles; ++kt)
        nxt[kt] = mfma32(*reinterpret_cast<const bf16x8*>(kbuf + koff[s] + kt * 32 * C::kRowBytes),
                         qf[s], nxt[kt]);
    bf16x8 pf[C::kKSteps];
    float la = 0.f, lb = 0.f;
#pragma unroll
    for (int kt = 0; kt < C::kKTiles; ++kt)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = fast_exp2(__builtin_fmaf(cur[kt][8 * h + 2 * e], c2, -m2));
          const float p1 = fast_exp2(__builtin_fmaf(cur[kt][8 * h + 2 * e + 1], c2, -m2));
          la += p0;
          lb += p1;
          w[e] = pack_bf16x2(p0, p1);
        }
        pf[2 * kt + h] = __builtin_bit_cast(bf16x8, w);
      }
    // at d = 128, four vector-ALU instructions (and, with them, two exponentials) beside each of
    // the 16 S products spread the tile's exponentials evenly over them (seven per product
    // front-loaded them onto the first nine and ran 1.5% slower; three and five were 0.3% and
    // 1.1% slower); d = 64 has half as many products for the same vector work and takes eight
    // per product (2-4% faster than seven, nine or ten)
    constexpr int kValuPerProduct = D == 128 ? 4 : 8;
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int i = 0; i < C::kDSteps * C::kKTiles; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, kValuPerProduct, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    // the reference m moves only when a probability of the tile could reach 2^32: the rare tile
    // that fails the check is redone against its row maximum
    if (__builtin_amdgcn_ballot_w64(!(la + lb < kGuard))) {
      cold_path();
      float ma = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < C::kKTiles; ++kt)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) ma = fmaxf(ma, cur[kt][rr]);
      const float mnew = fmaxf(m2, max_halves(ma) * c2);
      const float alpha = fast_exp2(m2 - mnew);
      m2 = mnew;
      lc *= alpha;
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) oacc[c] *= alpha;
      la = 0.f;
      lb = 0.f;
#pragma unroll
      for (int kt = 0; kt < C::kKTiles; ++kt)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          u32x4 w;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float p0 = fast_exp2(__builtin_fmaf(cur[kt][8 * h + 2 * e], c2, -m2));
            const float p1 = fast_exp2(__builtin_fmaf(cur[kt][8 * h + 2 * e + 1], c2, -m2));
            la += p0;
            lb += p1;
            w[e] = pack_bf16x2(p0, p1);
          }
          pf[2 * kt + h] = __builtin_bit_cast(bf16x8, w);
        }
    }
    lc += la + lb;

    __builtin_amdgcn_s_setprio(0);
    // O += V_j^T P_j on the matrix cores
    const char* vbuf = lds_v + P * C::kTileBytes;
#pragma unroll
    for (int s = 0; s < C::kKSteps; ++s)
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) {
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (lds_bf16x4*)(vbuf + voff[0][c] + s * 16 * C::kRowBytes));
        const bf16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (lds_bf16x4*)(vbuf + voff[1][c] + s * 16 * C::kRowBytes));
        oacc[c] = mfma32(__builtin_shufflevector(lo, hi4, 0, 1, 2, 3, 4, 5, 6, 7), pf[s], oacc[c]);
      }
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int i = 0; i < C::kKSteps * C::kCT; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_barrier(0);

    if (t0.start + C::kBK >= t0.hi) {
      // end of chunk r0: loc_lse_r from the chunk's own row sum
      const float lrow = sum_halves(lc);
      const float lse2r = m2 + fast_log2(lrow);
      if constexpr (kStep) {
        // Eq. (5) with the running result: out_acc <- (out_acc a + loc_out b) / (a + b)
        const int64_t qi = q0 + n;
        if (qi < Nq) {
          const int64_t row = bh * Nq + qi;
          float* ao = acc_out + row * D;
          const float inv = 1.0f / lrow;
          float wa = 0.f, wb = inv;
          float lnew = lse2r;
          if (!first) {
            const float lold = acc_lse[row] * kLog2e;
            const float M = fmaxf(lold, lse2r);
            const float a = fast_exp2(lold - M);
            const float b = fast_exp2(lse2r - M);
            const float den = a + b;
            wa = a / den;
            wb = b * inv / den;
            lnew = M + fast_log2(den);
          }
#pragma unroll
          for (int c = 0; c < C::kCT; ++c)
#pragma unroll
            for (int rq = 0; rq < 4; ++rq) {
              f32x4* dst = reinterpret_cast<f32x4*>(ao + c * 32 + 8 * rq + 4 * g);
              const f32x4 prev = first ? f32x4{} : *dst;
              f32x4 val;
#pragma unroll
              for (int e = 0; e < 4; ++e) val[e] = prev[e] * wa + oacc[c][4 * rq + e] * wb;
              *dst = val;
            }
          if (g == 0) acc_lse[row] = lnew * kLn2;
        }
#pragma unroll
        for (int c = 0; c < C::kCT; ++c) oacc[c] = f32x16{};
        m2 = -INFINITY;
      } else if constexpr (kPartials) {
        const int64_t qi = q0 + n;
        if (qi < Nq) {
          const float inv = 1.0f / lrow;
          const int64_t row = ((int64_t)r0 * BH + bh) * Nq + qi;
          float* po = part_out + row * D;
#pragma unroll
          for (int c = 0; c < C::kCT; ++c)
#pragma unroll
            for (int rq = 0; rq < 4; ++rq) {
              f32x4 val = {oacc[c][4 * rq] * inv, oacc[c][4 * rq + 1] * inv,
                           oacc[c][4 * rq + 2] * inv, oacc[c][4 * rq + 3] * inv};
              *reinterpret_cast<f32x4*>(po + c * 32 + 8 * rq + 4 * g) = val;
            }
          if (g == 0) part_lse[row] = lse2r * kLn2;
        }
#pragma unroll
        for (int c = 0; c < C::kCT; ++c) oacc[c] = f32x16{};
        m2 = -INFINITY;
      } else {
        // Eq. (5) on the log-sum-exps; the numerator terms already share the reference m2
        const float M = fmaxf(lse2m, lse2r);
        lse2m = M + fast_log2(fast_exp2(lse2m - M) + fast_exp2(lse2r - M));
      }
      lc = 0.f;
      ++r0;
    }
    t0 = t1;
    t1 = t2;
    t2 = walk.next<C::kBK>(t2);
    return t0.start >= nk;
  };

  while (true) {
    if (step(sa, sb, std::integral_constant<int, 0>{})) break;
    if (step(sb, sa, std::integral_constant<int, 1>{})) break;
  }

  if constexpr (MODE == (int)FwdMode::kFused) {
    const int64_t qi = q0 + n;
    if (qi < Nq) {
      // out = numerator / Eq. (5) denominator = oacc * 2^(m - lse)
      const float f = fast_exp2(m2 - lse2m);
      __bf16* ob = out + (bh * Nq + qi) * D;
#pragma unroll
      for (int c = 0; c < C::kCT; ++c)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          u32x2 w;
          w[0] = pack_bf16x2(oacc[c][4 * rq] * f, oacc[c][4 * rq + 1] * f);
          w[1] = pack_bf16x2(oacc[c][4 * rq + 2] * f, oacc[c][4 * rq + 3] * f);
          *reinterpret_cast<u32x2*>(ob + c * 32 + 8 * rq + 4 * g) = w;
        }
      if (g == 0) lse[bh * Nq + qi] = lse2m * kLn2;
    }
  }
}

template <int D, int MODE>
hipError_t launch(const FwdArgs& a) {
  using C = FwdCfg<D>;
  const int64_t nqt = (a.Nq + C::kBQ - 1) / C::kBQ;
  const int64_t nwg = nqt * a.BH;
  hipLaunchKernelGGL((fwd_bf16_kernel<D, MODE>), dim3((uint32_t)nwg), dim3(C::kThreads), 0,
                     a.stream, (const __bf16*)a.q, (const __bf16*)a.k, (const __bf16*)a.v,
                     (__bf16*)a.out, a.lse, a.part_out, a.part_lse, a.acc_out, a.acc_lse,
                     a.first ? 1 : 0, (int)a.BH, (int)a.H, (int)a.G, a.Nq, a.Nk, (int)a.R,
                     a.scale * kLog2e);
  return hipGetLastError();
}

template <int D>
hipError_t launch_mode(const FwdArgs& a, FwdMode mode) {
  switch (mode) {
    case FwdMode::kPartials: return launch<D, (int)FwdMode::kPartials>(a);
    case FwdMode::kStep: return launch<D, (int)FwdMode::kStep>(a);
    default: return launch<D, (int)FwdMode::kFused>(a);
  }
}

}  // namespace

int64_t fwd_bf16_workgroups(int64_t BH, int64_t Nq, int64_t d) {
  (void)d;
  const int64_t bq = FwdCfg<128>::kBQ;
  static_assert(FwdCfg<128>::kBQ == FwdCfg<64>::kBQ, "one query tile size");
  return BH * ((Nq + bq - 1) / bq);
}

hipError_t launch_fwd_bf16(const FwdArgs& a, FwdMode mode) {
  return a.d == 128 ? launch_mode<128>(a, mode) : launch_mode<64>(a, mode);
}

}  // namespace ringx
