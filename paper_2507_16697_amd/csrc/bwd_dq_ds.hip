// dQ of ring-chunked attention from stored dS, head size 128 (gfx950).
//
// The key-stationary dK/dV kernel (bwd_bf16.hip, store mode) already forms every dS_ij of the
// backward as the bf16 operand of its dK product; in store mode it also writes them to a workspace.
// This kernel then needs no recomputation: dQ_i = scale sum_j dS_ij k_j over the keys of every
// chunk (arXiv 2507.16697 Sec. III-A: the gradient of Q accumulated over the N ring steps) is one
// matrix product per query block, streamed from HBM.  The step executes 7U of matrix products
// instead of the 9U of the recompute path (U = 2 B H Nq Nk d), at the price of writing and reading
// B H Nq Nk bf16 values; this pass is bound by HBM bandwidth (about 2 bytes of dS per 256 flops).
//
// Stored layout (shared with the writer; ds_unit_offset in ringx_kernels.h): per query head j of
// the slab, 32-key block kb of the padded key axis (chunk r, 128-key tile t, block w ->
// kb = 4 (r tpc + t) + w), 128-query group qg and 32-query block qs of the group, one 2 KiB unit;
// within a unit, half h (16 queries) at 1024 h, then 16-byte chunks (32 gw + key) holding -dS of
// that key for queries 16 h + 4 gw + (m & 3) + 8 (m >> 2), m = 0..7.  The four units of one key
// block and one group are 8 KiB in a row; a 64-key tile of a group is two of them.
//
// One workgroup = 4 waves (one per SIMD) = one query head and 128 queries, 32 per wave, and two
// workgroups per CU.  Tiles of 64 keys (that tile's 16 KiB of dS and the 16 KiB of its K rows) are
// double buffered in LDS (64 KiB per workgroup), loaded by direct global->LDS loads one tile
// ahead: the two workgroups of a CU, with their own barriers, cover each other's load latency.
// (One workgroup per CU with a five-stage ring four tiles ahead streamed 15% slower, and with dS
// staged through registers eight tiles ahead 25% slower.)  Per 16-key step a wave reads its dS^T fragment (lane = query, 8 keys) and the four K^T fragments (lane = head
// dimension) by transposed LDS reads and issues four products into its dQ^T accumulators:
//   dQ^T (128 x 32) += K^T (128 x 16) dS^T (16 x 32)
// The dS chunks are XOR-swizzled in LDS (bits 2-3 of the chunk index by its half and gw), so that
// each transposed read touches every bank pair once.  Key rows past the end of a chunk (its last
// tile) are zeroed in LDS: their stored dS are finite but belong to no key.

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

struct DqsCfg {
  static constexpr int D = 128;
  static constexpr int kThreads = 256;
  static constexpr int kWaves = 4;
  static constexpr int kBQ = 128;                  // queries per workgroup (32 per wave)
  static constexpr int kBK = 64;                   // keys per tile
  static constexpr int kRowBytes = 2 * D;
  static constexpr int kChunks = D / 8;            // 16-byte chunks per K row
  static constexpr int kTile = kBK * kRowBytes;    // bytes of one K tile (16 KiB)
  static constexpr int kDsTile = kBK * kBQ * 2;    // bytes of one dS tile (16 KiB)
  static constexpr int kStage = kDsTile + kTile;
  static constexpr int kStages = 2;                // double buffer: loads run one tile ahead
  static constexpr int kLds = kStages * kStage;
  static constexpr int kLoads = kTile / (kThreads * 16);     // K loads per thread per tile
  static constexpr int kDsLoads = kDsTile / (kThreads * 16); // dS loads per thread per tile
  static constexpr int kCT = D / 32;
  static_assert(kTile == kLoads * kThreads * 16 && kDsTile == kDsLoads * kThreads * 16, "loads");
  static_assert(kDsTile == 8 * kDsUnitBytes, "a tile is two key blocks of four units");
};

__device__ __forceinline__ int swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }
__device__ __forceinline__ int tile_off(int row, int c) {
  return row * DqsCfg::kRowBytes + ((c ^ swz(row)) << 4);
}
// LDS position of 16-byte dS chunk c of a tile (an involution: bits 2-3 XOR bits 5-6)
__device__ __forceinline__ int ds_pos(int c) { return c ^ (((c >> 5) & 3) << 2); }

__global__ __launch_bounds__(256, 2) void bwd_dq_ds_kernel(
    const char* __restrict__ ds, const __bf16* __restrict__ k, float* __restrict__ dq, int nh,
    int grp, int64_t Nq, int64_t Nk, int R, int tpc, float neg_scale) {
  using C = DqsCfg;
  constexpr int D = C::D;
  __shared__ __attribute__((aligned(1024))) char lds[C::kLds];
  const uint32_t lbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int n = lane & 31;
  const int g = lane >> 5;

  const int64_t nqg = (Nq + C::kBQ - 1) / C::kBQ;
  const uint32_t wg = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t j = wg / nqg;          // query head within the slab
  const int64_t qg = wg % nqg;
  if (j >= nh) return;
  const int64_t nkb = 4 * (int64_t)R * tpc;

  const char* kbase = static_cast<const char*>(
      uniform_ptr(reinterpret_cast<const char*>(k + (j / grp) * Nk * D)));
  const char* dsbase = static_cast<const char*>(
      uniform_ptr(ds + ds_unit_offset(j, qg, 0, 0, nqg, nkb)));
  const int64_t kbstride = nqg * 4 * kDsUnitBytes;   // bytes from one key block to the next

  // tiles: chunk r holds keys [r Nk / R, (r+1) Nk / R), cut into 64-key tiles from its start;
  // its dS tiles sit at key-block pairs r * 2 tpc + 0, 1, ...
  int ntiles = 0;
  for (int r = 0; r < R; ++r) {
    const int64_t lo = (int64_t)r * Nk / R, hi = (int64_t)(r + 1) * Nk / R;
    ntiles += (int)((hi - lo + C::kBK - 1) / C::kBK);
  }
  // the next tile to load (ld_k, its chunk ld_r and key-block pair ld_pair = ld_r 2 tpc + its
  // tile within the chunk) and the tile being computed (cu_k): 32-bit positions walked without
  // divisions, so that the loop's bookkeeping stays scalar
  const uint32_t nk = (uint32_t)Nk;
  ChunkWalk ld_w{nk, nk / (uint32_t)R, nk % (uint32_t)R, 0, (uint32_t)R};
  ChunkWalk cu_w = ld_w;
  KeyTile ld_k = ld_w.first();
  KeyTile cu_k = cu_w.first();
  int ld_r = 0, ld_pair = 0;

  // K loads: round u covers rows 16 u + (wave * 64 + lane) / 16 at a swizzled chunk
  constexpr uint32_t kRound = C::kWaves * 64 * 16;
  static_assert(kRound % (16 * C::kRowBytes) == 0, "rounds keep the swizzle phase");
  const int row0 = (wave * 64 + lane) / C::kChunks;
  const uint32_t goff =
      row0 * C::kRowBytes + (((wave * 64 + lane) % C::kChunks) ^ swz(row0)) * 16;
  // dS loads: LDS chunk position P = 64 (4 u + wave) + lane receives stored chunk ds_pos(P),
  // which lies in the same 1 KiB half-unit
  const uint32_t dsoff = (uint32_t)(ds_pos(64 * wave + lane) - 64 * wave) * 16;
  static_assert(C::kDsLoads == 4 && kRound == 2 * kDsUnitBytes, "two rounds per key block");
  const uint32_t wdst = (uint32_t)__builtin_amdgcn_readfirstlane(wave * 1024);
  auto issue_next = [&](int stage) {
    const char* kt = kbase + (uint64_t)ld_k.start * C::kRowBytes;
    // key blocks 2 p and 2 p + 1 of the pair p = ld_pair; round u takes half u % 2 of block
    // u / 2's 8 KiB
    const char* dt = dsbase + (int64_t)ld_pair * 2 * kbstride;
    const uint32_t dst = lbase + stage * C::kStage + wdst;
#pragma unroll
    for (int u = 0; u < C::kDsLoads; ++u)
      load_lds16_s(dt + (u >> 1) * kbstride + (u & 1) * kRound + wave * 1024, dsoff,
                   dst + u * kRound);
    if (ld_k.start + C::kBK <= ld_k.hi) {
#pragma unroll
      for (int u = 0; u < C::kLoads; ++u)
        load_lds16_s(kt + u * kRound, goff, dst + C::kDsTile + u * kRound);
    } else {
      // the last tile of a chunk: rows past its end are clamped to the chunk's last key (and
      // zeroed once landed)
      cold_path();
      const int last = (int)(ld_k.hi - 1 - ld_k.start);
#pragma unroll
      for (int u = 0; u < C::kLoads; ++u) {
        const int row = row0 + u * (kRound / C::kRowBytes);
        const uint32_t off = goff + u * kRound - (row > last ? (row - last) * C::kRowBytes : 0);
        load_lds16_s(kt, off, dst + C::kDsTile + u * kRound);
      }
    }
    if (ld_k.start + C::kBK < ld_k.hi) {
      ++ld_pair;
    } else {
      ++ld_r;
      ld_pair = ld_r * 2 * tpc;
    }
    ld_k = ld_w.next<C::kBK>(ld_k);
  };

#pragma unroll
  for (int s = 0; s < C::kStages - 1; ++s)
    if (s < ntiles) issue_next(s);

  // transposed-read offsets.  K^T (A operand, lane = head dimension 32 c + n): rows (keys)
  // 16 s + 4 g + 8 h + (lane % 16) / 4, as in the other kernels.
  int toff[2][C::kCT];
  {
    const int G = lane >> 4;
    const int rr = (lane & 15) >> 2;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) {
        const int row = 4 * g + 8 * h + rr;
        const int col = 32 * c + 16 * (G & 1) + 4 * (lane & 3);
        toff[h][c] = tile_off(row, col >> 3) + (col & 7) * 2;
      }
  }
  // dS^T (B operand, lane = query): 16-lane group G reads half G & 1 of this wave's unit, keys
  // 4 (G >> 1) + 8 h + (lane % 16) / 4 (+16 per key step), gw = (lane % 4) / 2, the 8-byte half
  // lane % 2 of the chunk; lane i of the group receives the four keys of query
  // 16 (G & 1) + 4 (i >> 3) + 8 ((i >> 2) & 1) + (i & 3).
  int doff[2];
  {
    const int G = lane >> 4;
    const int e = (lane & 15) >> 2, p = lane & 3;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int key = 4 * (G >> 1) + 8 * h + e;
      const int c = 128 * wave + 64 * (G & 1) + 32 * (p >> 1) + key;
      doff[h] = ds_pos(c) * 16 + 8 * (p & 1);
    }
  }

  f32x16 acc[C::kCT];
#pragma unroll
  for (int c = 0; c < C::kCT; ++c) acc[c] = f32x16{};

  for (int it = 0; it < ntiles; ++it) {
    const int st = (it % C::kStages) * C::kStage;
    // tile it landed; every wave is done with tile it-1
    static_assert(C::kStages == 2, "nothing is in flight beyond the next tile");
    wait_vmem<0>();
    __syncthreads();
    const int valid = (int)min<uint32_t>(C::kBK, cu_k.hi - cu_k.start);
    if (valid < C::kBK) {
      // rows valid .. 63 of the K tile belong to no key
      cold_path();
      char* kt = lds + st + C::kDsTile;
      for (int i = t; i < (C::kBK - valid) * C::kChunks; i += C::kThreads)
        *reinterpret_cast<u32x4*>(kt + (valid + i / C::kChunks) * C::kRowBytes +
                                  (i % C::kChunks) * 16) = u32x4{};
      __syncthreads();
    }
    if (it + C::kStages - 1 < ntiles) issue_next((it + C::kStages - 1) % C::kStages);
    cu_k = cu_w.next<C::kBK>(cu_k);

    const char* dsl = lds + st;
    const char* kl = lds + st + C::kDsTile;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      // key step s: keys 16 s .. 16 s + 15 of the tile = key block s / 2, keys 16 (s % 2) ..
      const char* db = dsl + (s >> 1) * 8192 + (s & 1) * 256;
      const bf16x4 b0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(db + doff[0]));
      const bf16x4 b1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(db + doff[1]));
      const bf16x8 bop = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
      const char* kb = kl + 16 * s * C::kRowBytes;
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) {
        const bf16x4 a0 =
            __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(kb + toff[0][c]));
        const bf16x4 a1 =
            __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(kb + toff[1][c]));
        acc[c] = mfma32(__builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7), bop, acc[c]);
      }
    }
  }

  // column n of the accumulators is query 16 (n >> 4) + 4 ((n >> 3) & 1) + 8 ((n >> 2) & 1) +
  // (n & 3) of this wave's block; rows are head dimensions 32 c + 8 (r / 4) + 4 g + r % 4
  const int qn = 16 * (n >> 4) + 4 * ((n >> 3) & 1) + 8 * ((n >> 2) & 1) + (n & 3);
  const int64_t qi = qg * C::kBQ + 32 * wave + qn;
  if (qi < Nq) {
    float* row = dq + (j * Nq + qi) * D;
#pragma unroll
    for (int c = 0; c < C::kCT; ++c)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const f32x4 x = {acc[c][4 * rq] * neg_scale, acc[c][4 * rq + 1] * neg_scale,
                         acc[c][4 * rq + 2] * neg_scale, acc[c][4 * rq + 3] * neg_scale};
        *reinterpret_cast<f32x4*>(row + 32 * c + 8 * rq + 4 * g) = x;
      }
  }
}

}  // namespace

hipError_t launch_bwd_dq_ds(const DsArgs& a) {
  using C = DqsCfg;
  const int64_t nqg = (a.Nq + C::kBQ - 1) / C::kBQ;
  const int64_t nwg = a.nh * nqg;
  hipLaunchKernelGGL(bwd_dq_ds_kernel, dim3((uint32_t)nwg), dim3(C::kThreads), 0, a.stream,
                     static_cast<const char*>(a.ds), static_cast<const __bf16*>(a.k), a.dq,
                     (int)a.nh, (int)a.G, a.Nq, a.Nk, (int)a.R, (int)a.tpc, -a.scale);
  return hipGetLastError();
}

}  // namespace ringx
