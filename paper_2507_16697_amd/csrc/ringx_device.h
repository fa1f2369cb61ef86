// Device-side helpers shared by the libringx kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ringx {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// v_mfma_f32_32x32x16_bf16.  Operand layout for lane l (g = l / 32, n = l % 32):
//   A (32 x 16): row n, k = 8g .. 8g+7      B (16 x 32): column n, k = 8g .. 8g+7
//   C (32 x 32): column n, rows 8*(r/4) + 4g + (r%4) for accumulator r = 0..15
__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// fp32 pair -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 x = {lo, hi};
  bf16x2 y = __builtin_convertvector(x, bf16x2);
  return __builtin_bit_cast(uint32_t, y);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// x[l] + x[l ^ 32] and max(x[l], x[l ^ 32]) for every lane l, through v_permlane32_swap.  The
// swap of two copies of x returns, for lanes below 32, (x[l], x[l + 32]) and for the others
// (x[l - 32], x[l]): each result alone holds the lane's own value on one half of the wave, so the
// two are always combined.
__device__ __forceinline__ float sum_halves(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float max_halves(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// The chunked key sequence walked one tile of BK keys at a time, without divisions: chunk r is
// [floor(r Nk / R), floor((r + 1) Nk / R)), which holds Nk / R keys plus one whenever the running
// sum of the remainders Nk mod R passes a multiple of R.  Key positions are 32-bit (the library
// takes at most 2^31 keys per head), so that the walk and its tests stay scalar instructions.
struct KeyTile {
  uint32_t start, hi;   // first key of the tile, end of its chunk; start >= Nk: no tile
};

struct ChunkWalk {
  uint32_t Nk, q_sz, rem, racc;   // Nk, Nk / R, Nk mod R, running remainder
  uint32_t R;
  __device__ KeyTile first() {
    racc = rem;
    const uint32_t extra = racc >= R ? 1u : 0u;
    racc -= extra * R;
    return {0, q_sz + extra};
  }
  template <int BK>
  __device__ KeyTile next(const KeyTile& t) {
    if (t.start + BK < t.hi) return {t.start + BK, t.hi};
    if (t.hi >= Nk) return {Nk, Nk};
    racc += rem;
    const uint32_t extra = racc >= R ? 1u : 0u;
    racc -= extra * R;
    return {t.hi, t.hi + q_sz + extra};
  }
};

// K/V head serving query head `bh` (of B*H): query heads come in consecutive groups of `grp` per
// K/V head (grouped-query attention; grp = 1 is plain multi-head attention).
__device__ __forceinline__ int64_t kv_head(int64_t bh, int H, int grp) {
  return (bh / H) * (H / grp) + (bh % H) / grp;
}

// Logical workgroup id so that the workgroups resident on one XCD work on the same (b, h) slice.
// The hardware hands consecutive workgroup ids to the 8 XCDs round robin; this groups id w's
// XCD (w % 8) onto a contiguous range of logical ids.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t w, uint32_t n) {
  constexpr uint32_t kXcd = 8;
  const uint32_t per = n / kXcd;           // full rounds
  const uint32_t full = per * kXcd;
  if (w >= full) return w;                 // ragged last round keeps its id
  return (w % kXcd) * per + w / kXcd;
}

// One 16-byte direct global->LDS load per lane (global_load_lds_dwordx4): the LDS destination is
// lds_base + 16 * lane.  Issued through inline asm so that the compiler does not serialise later
// LDS reads of other buffers behind it.  The asm sets m0, which the compiler never uses in these
// kernels (a build test checks the generated code); an LDS DMA that reads m0 right after a scalar
// write of it needs one wait state on this chip family, hence the s_nop (the compiler's hazard
// recognizer does not look inside inline asm).  Callers publish the data with wait_vmem_all()
// followed by a workgroup barrier.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void load_lds16(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(lds_base), "v"(gptr)
               : "memory", "m0");
}
// Same with 4 bytes per lane: LDS destination = lds_base + 4 * lane.
__device__ __forceinline__ void load_lds4(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, off"
               :
               : "s"(lds_base), "v"(gptr)
               : "memory", "m0");
}
// A wave-uniform pointer in SGPRs (free when the compiler already holds it there).
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t x = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return reinterpret_cast<const void*>(((uint64_t)hi << 32) | lo);
}
// The same loads with a uniform 64-bit base (the callers' base is the same for every lane) in
// SGPRs and a per-lane 32-bit offset: the scalar-base form, no per-lane 64-bit address arithmetic.
__device__ __forceinline__ void load_lds16_s(const void* base, uint32_t off, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(lds_base), "v"(off), "s"(uniform_ptr(base))
               : "memory", "m0");
}
__device__ __forceinline__ void load_lds4_s(const void* base, uint32_t off, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, %2"
               :
               : "s"(lds_base), "v"(off), "s"(uniform_ptr(base))
               : "memory", "m0");
}

// v_mfma_f32_32x32x16_bf16 as inline assembly that names the register file of every operand ("a":
// AGPRs, the matrix cores' accumulation/operand registers; "v": VGPRs), for kernels that need
// more than the 256 VGPRs of one wave.  Volatile, so they keep the order the kernel gives them.
// The compiler inserts no wait states around inline assembly: a kernel using these keeps every
// result away from its next reader, and every vector write away from the product reading it
// (tests/test_build_isa.py checks the built code).
// acc += A B, accumulator in AGPRs
__device__ __forceinline__ void mfma_acc_a(f32x16& acc, bf16x8 a, bf16x8 b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// acc = A B (first product of a chain), accumulator in VGPRs, B in AGPRs
__device__ __forceinline__ void mfma_first_v(f32x16& acc, bf16x8 a, bf16x8 b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(acc) : "v"(a), "a"(b));
}
// acc = A B + c (first product of a chain that starts from c)
__device__ __forceinline__ void mfma_first_vc(f32x16& acc, bf16x8 a, bf16x8 b, const f32x16& c) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %3" : "=&v"(acc) : "v"(a), "a"(b), "v"(c));
}
// acc += A B, accumulator in VGPRs, B in AGPRs
__device__ __forceinline__ void mfma_acc_v(f32x16& acc, bf16x8 a, bf16x8 b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(a), "a"(b));
}
#pragma clang diagnostic pop

// s_waitcnt vmcnt(n) (expcnt and lgkmcnt left alone), n < 64.
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Keeps a rarely taken branch a branch: an empty volatile asm statement has side effects, so the
// compiler cannot speculate the branch body into straight-line selects executed on every tile.
__device__ __forceinline__ void cold_path() { asm volatile(""); }

// s_waitcnt vmcnt(0): every vector memory load of this wave (including direct LDS loads) done.
__device__ __forceinline__ void wait_vmem_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

}  // namespace ringx
