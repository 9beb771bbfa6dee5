// On-chip rebuild of an agent's keys/values from the shared base cache and the
// agent's LR cache (Eq. 1; App. D.2: the key-side term is expanded from rank r
// and then rotated):
//     K[t] = K_base[t] + RoPE(L_k[t] B_k, t),     V[t] = V_base[t] + L_v[t] B_v.
//
// Register layout shared by every kernel that rebuilds (decode, prefill,
// materialise).  A wave handles 16 tokens of one KV head; lane l holds token
// l%16 and, with q = l/16, the head dims
//     [q*QPG, (q+1)*QPG)  and  [HALF + q*QPG, HALF + (q+1)*QPG),   QPG = d/8,
// so both elements of every RoPE pair (j, j + d/2) sit in the same lane.
// These dims are kept as D/32 "chunks" of 8 consecutive bf16 (u32x4):
// chunk kk starts at chunk_dim(kk, q).
//
// The rank-r expansion is E^T = B^T L^T on 16x16 MFMAs, one 16x16 output per
// 16-dim block.  Row m of block blk is head dim blk_dim(blk, m), which makes
// result row 4q+i of block blk land on element (blk&1)*4+i of chunk blk>>1 --
// the chunk layout above.  Blocks blk < D/32 cover the low RoPE half and
// pair with block blk + D/32.
#pragma once

#include <type_traits>

#include "common.hpp"

namespace prc {

// Number of 16-wide rank chunks (r = 8 pads to 16).  The value side's
// P L_v product is laid out in these.
constexpr int RCH(int r) { return r < 16 ? 1 : r / 16; }

// Rank chunks of the expansion E^T = B^T L^T.  Ranks 32 and 64 use 32-wide
// chunks on the full-rate 16x16x32 MFMA (lane l holds ranks c*32 + (l/16)*8
// .. +7, one 16-byte fragment); ranks 8 and 16 one 16-wide chunk on 16x16x16
// (ranks (l/16)*4 .. +3; rank 8 pads to 16).  Both give the same 16x16 result
// layout, so only the operand fragments differ.
template <int R>
struct Ex {
  static constexpr bool WIDE = R >= 32;
  static constexpr int K = WIDE ? 32 : 16;    // ranks per chunk
  static constexpr int NC = WIDE ? R / 32 : 1;
  static constexpr int PER = K / 4;           // ranks per lane and chunk
  typedef typename std::conditional<WIDE, u32x4, u32x2>::type Frag;
  static __device__ __forceinline__ int rank0(int c, int q) { return c * K + q * PER; }
  static __device__ __forceinline__ f32x4 mma(Frag a, Frag b, f32x4 acc) {
    if constexpr (WIDE)
      return mfma16x16x32(as_bf16x8(a), as_bf16x8(b), acc);
    else
      return mfma16x16x16(as_i16x4(a), as_i16x4(b), acc);
  }
  // PER consecutive bf16 at p (zeros when !ok).
  static __device__ __forceinline__ Frag load(const uint16_t* p, bool ok) {
    if constexpr (WIDE)
      return ld16(p, ok);
    else
      return ld8(p, ok);
  }
  // PER bf16 at p, p + ld, p + 2 ld, ... (consecutive ranks of one column of
  // an up-projection stored rank-major, [r, ld]); zeros when !ok.
  static __device__ __forceinline__ Frag gather(const uint16_t* p, int64_t ld, bool ok) {
    Frag f;
#pragma unroll
    for (int i = 0; i < PER / 2; ++i)
      f[i] = ok ? (uint32_t)p[2 * i * ld] | ((uint32_t)p[(2 * i + 1) * ld] << 16) : 0u;
    return f;
  }
};

template <int D, int R>
struct Rb {
  static constexpr int HALF = D / 2;
  static constexpr int NB = D / 32;    // 16-dim blocks per RoPE half
  static constexpr int NBLK = D / 16;  // 16-dim blocks
  static constexpr int NCH = D / 32;   // 8-dim chunks per lane
  static constexpr int QPG = D / 8;    // dims per lane group per half
  static constexpr int RC = R < 16 ? 1 : R / 16;  // 16-wide rank chunks
};

// First head dim of chunk kk for lane group q.
template <int D>
__device__ __forceinline__ int chunk_dim(int kk, int q) {
  constexpr int HALF = D / 2, NB = D / 32, QPG = D / 8;
  return ((2 * kk) / NB) * HALF + q * QPG + ((2 * kk) % NB) * 4;
}

// Head dim of row m in 16-dim block blk.
template <int D>
__device__ __forceinline__ int blk_dim(int blk, int m) {
  constexpr int HALF = D / 2, NB = D / 32, QPG = D / 8;
  return (blk / NB) * HALF + (m >> 2) * QPG + (blk % NB) * 4 + (m & 3);
}

// B^T fragments (A operand of the expansion) of one KV head.  The
// up-projection is stored as in Eq. 1, B [r, n_kv*d] (row j = rank j), with
// row stride ldb = n_kv*d; `bhead` points at the head's first column of rank
// 0, B[0][g*d].  A lane gathers its PER ranks of one column.
template <int D, int R>
__device__ __forceinline__ void load_bt_frags(typename Ex<R>::Frag (&f)[D / 16][Ex<R>::NC], const uint16_t* bhead,
                                              int64_t ldb, bool ok, int lane) {
  using E = Ex<R>;
  const int c16 = lane & 15, q = lane >> 4;
#pragma unroll
  for (int blk = 0; blk < D / 16; ++blk) {
    const int dim = blk_dim<D>(blk, c16);
#pragma unroll
    for (int c = 0; c < E::NC; ++c) {
      const int r0 = E::rank0(c, q);
      const bool v = ok && r0 < R;
      f[blk][c] = E::gather(v ? bhead + (int64_t)r0 * ldb + dim : nullptr, ldb, v);
    }
  }
}

// The same fragments as load_bt_frags, for kernels whose workgroups are
// short-lived (decode splits): the head's up-projection rows are read with
// coalesced 16-byte loads, 16 ranks at a time, and staged through a
// wave-private LDS area of at least 16 x (D + 16) bf16, from which they come
// back transposed through ds_read_b64_tr_b16 (lane j of each 16-lane group
// points at 4 consecutive bf16; lane i receives element i%4 of lanes i/4,
// i/4+4, i/4+8, i/4+12).  A source lane s of group q points at rank row
// 4q + s/4 (within a 16-rank chunk) and head dims blk_dim(blk, 4 (s%4)) .. + 3,
// so lane i receives ranks 4q .. 4q + 3 of dim blk_dim(blk, i), the
// expansion's A fragment.  Split in two so that the loads can be issued at
// the very start of a kernel and their latency hidden behind its other set-up.
template <int D, int R>
struct BtStage {
  static constexpr int NCH = (R + 15) / 16;       // 16-rank chunks (rank 8: one, upper rows zero)
  static constexpr int PPL = 16 * (D / 8) / 64;   // 16-byte pieces per lane and chunk
  u32x4 raw[NCH][PPL];

  __device__ __forceinline__ void issue(const uint16_t* bhead, int64_t ldb, bool ok, int lane) {
#pragma unroll
    for (int rc = 0; rc < NCH; ++rc)
#pragma unroll
      for (int i = 0; i < PPL; ++i) {
        const int p = lane + 64 * i, row = p / (D / 8), col = (p % (D / 8)) * 8, rank = 16 * rc + row;
        raw[rc][i] = ld16(bhead + (int64_t)(rank < R ? rank : 0) * ldb + col, ok && rank < R);
      }
  }

  __device__ __forceinline__ void finish(typename Ex<R>::Frag (&f)[D / 16][Ex<R>::NC], uint16_t* stage,
                                         int lane) const {
    typedef short v4s __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) v4s* lds_v4s;
    constexpr int ROW = D + 16;  // stage row stride (bf16)
    const int q = lane >> 4, s = lane & 15;
#pragma unroll
    for (int rc = 0; rc < NCH; ++rc) {
#pragma unroll
      for (int i = 0; i < PPL; ++i) {
        const int p = lane + 64 * i, row = p / (D / 8), col = (p % (D / 8)) * 8;
        *reinterpret_cast<u32x4*>(stage + row * ROW + col) = raw[rc][i];
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int blk = 0; blk < D / 16; ++blk) {
        const int dim = blk_dim<D>(blk, 4 * (s & 3));
        if constexpr (!Ex<R>::WIDE) {
          // Ranks 4q .. 4q + 3 of the one chunk.
          f[blk][0] = __builtin_bit_cast(
              u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(stage + (4 * q + (s >> 2)) * ROW + dim)));
        } else {
          // 32-rank chunk rc / 2 holds ranks 8q .. 8q + 7 for lane group q:
          // rows 8 (q % 2) + 0..7 of 16-rank chunk 2 (rc / 2) + q / 2.
          const int r0 = 8 * (q & 1) + (s >> 2);
          const u32x2 lo =
              __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(stage + r0 * ROW + dim)));
          const u32x2 hi = __builtin_bit_cast(
              u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(stage + (r0 + 4) * ROW + dim)));
          if ((q >> 1) == (rc & 1)) f[blk][rc >> 1] = u32x4{lo[0], lo[1], hi[0], hi[1]};
        }
      }
      // This chunk's reads are done before the next chunk overwrites the stage.
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
      __builtin_amdgcn_wave_barrier();
    }
  }
};

// One LR row as the B operand of the expansion (k = rank index).
template <int R>
__device__ __forceinline__ void load_lr_frag(typename Ex<R>::Frag (&l)[Ex<R>::NC], const uint16_t* lrow, bool ok,
                                             int lane) {
  using E = Ex<R>;
  const int q = lane >> 4;
#pragma unroll
  for (int c = 0; c < E::NC; ++c) {
    const int r0 = E::rank0(c, q);
    const bool v = ok && r0 < R;
    l[c] = E::load(v ? lrow + r0 : nullptr, v);
  }
}

// Base row of this lane's token in chunk layout.
template <int D>
__device__ __forceinline__ void load_chunks(u32x4 (&x)[D / 32], const uint16_t* head_row, bool ok, int lane) {
  const int q = lane >> 4;
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) x[kk] = ld16(head_row + chunk_dim<D>(kk, q), ok);
}

template <int D>
__device__ __forceinline__ void store_chunks(uint16_t* head_row, const u32x4 (&x)[D / 32], int lane) {
  const int q = lane >> 4;
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) *reinterpret_cast<u32x4*>(head_row + chunk_dim<D>(kk, q)) = x[kk];
}

__device__ __forceinline__ float chunk_get(const u32x4& c, int el) {
  const uint32_t u = c[el >> 1];
  return (el & 1) ? bf_hi(u) : bf_lo(u);
}

// x += L B (value side), rounded back to bf16.
template <int D, int R>
__device__ __forceinline__ void add_expansion(u32x4 (&x)[D / 32], const typename Ex<R>::Frag (&bf)[D / 16][Ex<R>::NC],
                                              const typename Ex<R>::Frag (&l)[Ex<R>::NC]) {
#pragma unroll
  for (int blk = 0; blk < D / 16; ++blk) {
    f32x4 e = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < Ex<R>::NC; ++c) e = Ex<R>::mma(bf[blk][c], l[c], e);
    const int kk = blk >> 1, w0 = (blk & 1) * 2;
    float v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = chunk_get(x[kk], (blk & 1) * 4 + i) + e[i];
    x[kk][w0] = pack_bf16(v[0], v[1]);
    x[kk][w0 + 1] = pack_bf16(v[2], v[3]);
  }
}

// x += RoPE(L B) (key side), rounded back to bf16.  c[blk][i], s[blk][i] are
// cos/sin of the token's angle at frequency q*QPG + blk*4 + i.
template <int D, int R>
__device__ __forceinline__ void add_rotated_expansion(u32x4 (&x)[D / 32],
                                                      const typename Ex<R>::Frag (&bf)[D / 16][Ex<R>::NC],
                                                      const typename Ex<R>::Frag (&l)[Ex<R>::NC],
                                                      const float (&c)[D / 32][4], const float (&s)[D / 32][4]) {
  constexpr int NB = D / 32;
#pragma unroll
  for (int blk = 0; blk < NB; ++blk) {
    f32x4 elo = {0.f, 0.f, 0.f, 0.f}, ehi = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int rc = 0; rc < Ex<R>::NC; ++rc) {
      elo = Ex<R>::mma(bf[blk][rc], l[rc], elo);
      ehi = Ex<R>::mma(bf[blk + NB][rc], l[rc], ehi);
    }
    const int klo = blk >> 1, khi = (blk + NB) >> 1, w0 = (blk & 1) * 2;
    float vlo[4], vhi[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int el = (blk & 1) * 4 + i;
      vlo[i] = chunk_get(x[klo], el) + elo[i] * c[blk][i] - ehi[i] * s[blk][i];
      vhi[i] = chunk_get(x[khi], el) + ehi[i] * c[blk][i] + elo[i] * s[blk][i];
    }
    x[klo][w0] = pack_bf16(vlo[0], vlo[1]);
    x[klo][w0 + 1] = pack_bf16(vlo[2], vlo[3]);
    x[khi][w0] = pack_bf16(vhi[0], vhi[1]);
    x[khi][w0 + 1] = pack_bf16(vhi[2], vhi[3]);
  }
}

}  // namespace prc
