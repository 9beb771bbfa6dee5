// Shared device helpers for the gfx950 kernels: vector types, bf16 packing,
// MFMA wrappers, cross-lane reductions and the RoPE angle generator.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace prc {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kWave = 64;

// ---------------------------------------------------------------- bf16 ----
__device__ __forceinline__ float bf_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

// Round two floats to bf16 (round to nearest even, v_cvt_pk_bf16_f32) and pack.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ i16x4 as_i16x4(u32x2 v) { return __builtin_bit_cast(i16x4, v); }

// ---------------------------------------------------------------- loads ---
// 16-byte and 8-byte loads that return zero when `ok` is false, so masked
// rows never touch memory.
__device__ __forceinline__ u32x4 ld16(const uint16_t* p, bool ok) {
  u32x4 z = {0u, 0u, 0u, 0u};
  return ok ? *reinterpret_cast<const u32x4*>(p) : z;
}
__device__ __forceinline__ u32x2 ld8(const uint16_t* p, bool ok) {
  u32x2 z = {0u, 0u};
  return ok ? *reinterpret_cast<const u32x2*>(p) : z;
}

// ------------------------------------------------------- buffer loads ----
typedef int i32x4 __attribute__((ext_vector_type(4)));
// Raw buffer resource over `bytes` bytes from `base` (stride 0): loads at
// offsets at or past `bytes` return zeros.
__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, int32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  return i32x4{(int)(uint32_t)b, (int)(uint32_t)(b >> 32), bytes, 0x00020000};
}
// Direct global->LDS load of 16 bytes per lane: lane i's data lands at
// lds + 16 i.  Issued through inline assembly so that the compiler does not
// treat every later LDS read as dependent on it; the caller waits with
// s_waitcnt vmcnt before publishing the data (barrier) and reading it.
__device__ __forceinline__ void lds_dma16(i32x4 rsrc, const void* lds, int32_t voff, int32_t soff) {
  const uint32_t m = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)lds);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds" ::"s"(m), "v"(voff), "s"(rsrc),
               "s"(soff)
               : "memory", "m0");
}

// ---------------------------------------------------------------- MFMA ----
// 16x16x32 bf16: lane l holds A[m = l%16][k = (l/16)*8 + 0..7],
// B[k = (l/16)*8 + 0..7][n = l%16]; C[m = (l/16)*4 + i][n = l%16].
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// 16x16x16 bf16: lane l holds A[m = l%16][k = (l/16)*4 + 0..3],
// B[k = (l/16)*4 + 0..3][n = l%16]; C[m = (l/16)*4 + i][n = l%16].
__device__ __forceinline__ f32x4 mfma16x16x16(i16x4 a, i16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}
// 32x32x16 bf16: lane l holds A[m = l%32][k = (l/32)*8 + 0..7],
// B[k = (l/32)*8 + 0..7][n = l%32]; C[m = (j/4)*8 + (l/32)*4 + j%4][n = l%32].
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// ------------------------------------------------------- lane exchange ----
__device__ __forceinline__ float shfl_xor(float v, int mask) {
  return __shfl_xor(v, mask, kWave);
}
// Reductions over the 16 lanes that share l/16.
__device__ __forceinline__ float max16(float v) {
  v = fmaxf(v, shfl_xor(v, 1));
  v = fmaxf(v, shfl_xor(v, 2));
  v = fmaxf(v, shfl_xor(v, 4));
  v = fmaxf(v, shfl_xor(v, 8));
  return v;
}
__device__ __forceinline__ float sum16(float v) {
  v += shfl_xor(v, 1);
  v += shfl_xor(v, 2);
  v += shfl_xor(v, 4);
  v += shfl_xor(v, 8);
  return v;
}
// Combine lane l with lane l ^ 16 through v_permlane16_swap (no LDS trip):
// with both operands x, the two results hold rows (0,1) and (2,3) of x in
// swapped order, so combining them pairs every lane with its l ^ 16.
__device__ __forceinline__ float max_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
// Combine lane l with lane l ^ 32 through v_permlane32_swap (no LDS trip).
__device__ __forceinline__ float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float readlane_f(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ----------------------------------------------------------- paged walk ----
// Walks one request's rows of the block tables of paged caches in token
// order, one tile of `step` tokens at a time (step divides the block size,
// so no tile straddles two blocks).  A block's table entries are fetched
// once, with vector loads, when the walk enters the block -- a tile before
// they are used: scalar loads share their wait counter with LDS traffic, so
// every LDS wait in between would wait on them.  Entries are clamped into
// the pools, and table indexes past the row read as 0.  All state is
// wave-uniform except the fetched entries.
struct PageWalk {
  __amdgpu_buffer_rsrc_t kvt, lrt;
  int blk, kv_nblk, lr_nblk;
  int q, rem;         // block of the next tile and its first row there
  int32_t ekv, elr;   // table entries of block q

  __device__ __forceinline__ void fetch() {
    ekv = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(kvt, q * 4, 0, 0);
    elr = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(lrt, q * 4, 0, 0);
  }
  // Start at token t_first (a multiple of step); t_end bounds the walk.
  __device__ __forceinline__ void start(const int32_t* kv_tbl, const int32_t* lr_tbl, int max_blk, int blk_,
                                        int kvn, int lrn, int64_t t_first, int64_t t_end) {
    kvt = __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(kv_tbl), (short)0, max_blk * 4, 0x00020000);
    lrt = __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(lr_tbl), (short)0, max_blk * 4, 0x00020000);
    blk = blk_;
    kv_nblk = kvn;
    lr_nblk = lrn;
    q = (int)(t_first / blk_);
    rem = (int)(t_first - (int64_t)q * blk_);
    ekv = elr = 0;
    if (t_first < t_end) fetch();
  }
  // Pool rows (base, LR) of the next tile's first token; then step on.
  __device__ __forceinline__ void next(int step, int64_t t_end, int64_t& kv_row, int64_t& lr_row) {
    int32_t ek = __builtin_amdgcn_readfirstlane(ekv), el = __builtin_amdgcn_readfirstlane(elr);
    ek = ek < 0 ? 0 : (ek >= kv_nblk ? kv_nblk - 1 : ek);
    el = el < 0 ? 0 : (el >= lr_nblk ? lr_nblk - 1 : el);
    kv_row = (int64_t)ek * blk + rem;
    lr_row = (int64_t)el * blk + rem;
    rem += step;
    if (rem == blk) {
      rem = 0;
      ++q;
      if ((int64_t)q * blk < t_end) fetch();
    }
  }
};

// ---------------------------------------------------------------- RoPE ----
// cos/sin of the angle pos * omega_j, where w2pi = omega_j / (2 pi) in fp64.
// The angle is formed in fp64 revolutions, reduced to [0, 1) in fp64, and only
// then rounded to fp32 for the hardware sin/cos (which take revolutions).  The
// fp32 error stays near 1e-7 at every position below 2^31.
__device__ __forceinline__ void rope_cs(int pos, double w2pi, float& c, float& s) {
  double rev = (double)pos * w2pi;
  rev -= __builtin_floor(rev);
  float f = (float)rev;
  c = __builtin_amdgcn_cosf(f);
  s = __builtin_amdgcn_sinf(f);
}

}  // namespace prc
