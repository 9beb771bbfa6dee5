// LR-shared attention, prefill (many query tokens per request), gfx950.
//
// Causal flash attention of a chunk of new query tokens over the shared base
// cache plus the current agent's LR cache (Sec. 3.1, reuse step).
//   keys:   each KV tile is rebuilt in LDS, K = K_base + RoPE(L_k B_k), with
//           the rank-r expansion before RoPE (App. D.2);
//   values: rank 8 uses associativity (App. D.2),
//           O = P V_base + (P L_v) B_v: V_base and L_v go to LDS unchanged in
//           value, P L_v is accumulated beside P V_base and B_v is applied
//           once in the epilogue.  Ranks 16 to 64 rebuild V = V_base + L_v B_v
//           in the tile (bf16, like K): with 256 query rows per workgroup that
//           is half the flops of P L_v, needs no (P L_v)^T accumulator, and
//           the expansion rides on the MFMA that transposes V anyway.
//
// Work split: one workgroup of 8 waves per (request, KV head, 256 query rows).
// A query row is a (token, q head of the GQA group) pair, so the group's heads
// share every rebuilt tile.  Every wave both builds and attends:
//   build   wave w rebuilds 16 tokens (w % 4) x half of the RoPE pair blocks
//           (w / 4) of the next KV tile: E^T = B_k^T L_k^T on 16x16 MFMAs
//           (lane l: token l%16, both halves of each pair in the same lane),
//           RoPE by angle addition (exact per-tile base angle in LDS,
//           per-lane offset angles in LDS, or at rank 16 as fp16 pairs in
//           registers), + base, bf16 into LDS.  It also transposes a
//           32-token block of V_base (and, at rank 8, of L_v) on
//           the MFMA against a shifted identity, which writes them to LDS
//           directly in the PV A-fragment layout; from rank 32 the transpose
//           accumulates onto L_v B_v of the same block.  Its global loads for
//           the tile after next are in flight meanwhile;
//   attend  over 32 query rows (lanes l and l^32 share row l%32), in two
//           halves of 32 tokens:
//     scores  S^T = K Q^T on 32x32x16 MFMAs, so softmax statistics are per
//             lane; causal mask only on halves that cross it;
//     softmax online, exp2 domain, lazily rescaled; where the registers
//             allow it (plain and values-only kernels, tile-cache kernels
//             up to rank 32) Q is pre-scaled once and the main loop's score
//             MFMAs start from a block holding minus the reference maximum;
//     PV      O^T += V^T P^T (and, below rank 32, (P L_v)^T += L_v^T P^T) on
//             32x32x16 MFMAs,
//             one conflict-free 16-byte LDS read per A fragment; P is
//             already in the B operand layout.
// LDS instructions, not bytes, bound the tile rate here (each costs the CU
// about 4 cycles whatever its width), hence the fragment layouts above and
// the register-resident identities and small-rank B_k fragments (in LDS in
// the tile-cache kernels, which rebuild a few tiles per wave).  Large
// contiguous calls share rebuilt tiles between the row-tile workgroups of a
// KV head through a tile cache in the workspace (see below).  Tiles
// below every row's causal limit run a straight-line main loop (scores, then
// one block of exponentials, PV and the next tile's build); tiles that cross
// a limit run a per-half loop in which the two waves sharing a SIMD take
// build and attend in opposite order.  LDS is double-buffered with one
// barrier per tile.
#include "common.hpp"
#include "kernels.hpp"
#include "rebuild.hpp"

namespace prc {
namespace {

constexpr int TKV = 64;              // KV tokens per tile
constexpr int NW = 8;                // waves per workgroup
constexpr int NTHR = 64 * NW;
constexpr int WROWS = 32;            // query rows per wave
constexpr int BROWS = NW * WROWS;    // query rows per workgroup
constexpr float kRescaleLog2 = 8.f;  // lazy-rescale threshold (log2 domain)
// Value side of rank r: V = V_base + L_v B_v rebuilt in the tile, or
// associativity with (P L_v) accumulated beside P V_base.
constexpr bool rebuilds_v(int rank) { return rank >= 16; }

template <int D, int R, bool TCN = false>
struct Pre {
  static_assert(D == 64 || D == 128, "head dims 64 and 128");
  static constexpr int HALF = D / 2;
  static constexpr int NB = D / 32;          // 16-dim blocks per RoPE half
  static constexpr int NBW = NB / 2;         // low blocks rebuilt per wave
  static constexpr int SEG = 4 * NBW;        // contiguous dims per lane and half
  static constexpr int QPG = D / 8;          // dims per lane group per half
  static constexpr int RC = RCH(R);          // 16-wide rank chunks (value side)
  static constexpr int NC = Ex<R>::NC;       // rank chunks of the key expansion
  static constexpr int RB = (R + 31) / 32;   // 32-row blocks of (P L_v)^T
  static constexpr int NKQ = D / 16;         // 32x32x16 k-chunks over d
  static constexpr int NDB = D / 32;         // 32-dim blocks of O^T
  static constexpr int K_ROW = D + 8;        // bf16 per K row in LDS
  // V^T is kept in LDS as ready-made PV A fragments: fragment (m, db) holds,
  // for lane l, dims 32 db + l%32 at the 8 tokens of 16-token chunk m in P's
  // k order.  The tile is 2 x (D/16) half blocks of 32 tokens x 16 dims; each
  // wave transposes NHB of them.
  static constexpr int NHB = D / 64;         // half blocks per wave (8 waves)
  // L_v^T likewise, fragment (m, rb) for ranks 32 rb + l%32: waves
  // 0 .. 2 RB - 1 each transpose 32 tokens x 32 ranks, in NLP 16-rank halves.
  static constexpr int NLP = R >= 32 ? 2 : 1;
  // B_k^T fragments of small ranks stay in registers, larger ones in LDS;
  // the tile-cache instantiation (TCN) rebuilds a few tiles per wave only and
  // keeps them in LDS at every rank, freeing registers for the main loop.
  static constexpr bool BK_REG = R <= 16 && !TCN;
  // The per-lane offset angles of the rebuild stay in registers where the
  // register budget allows it (rank 16, V rebuilt in the tile), else in LDS.
  static constexpr bool OCS_REG = R == 16 && !TCN;
};

// SEG consecutive bf16 of one row.
template <int SEG>
struct Seg {
  uint32_t w[SEG / 2];
};
template <int SEG>
__device__ __forceinline__ Seg<SEG> ld_seg(const uint16_t* p, bool ok) {
  Seg<SEG> s;
  if constexpr (SEG == 8) {
    const u32x4 v = ld16(p, ok);
#pragma unroll
    for (int i = 0; i < 4; ++i) s.w[i] = v[i];
  } else {
    const u32x2 v = ld8(p, ok);
    s.w[0] = v[0];
    s.w[1] = v[1];
  }
  return s;
}
template <int SEG>
__device__ __forceinline__ void st_seg(uint16_t* p, const Seg<SEG>& s) {
  if constexpr (SEG == 8) {
    const u32x4 v = {s.w[0], s.w[1], s.w[2], s.w[3]};
    *reinterpret_cast<u32x4*>(p) = v;
  } else {
    const u32x2 v = {s.w[0], s.w[1]};
    *reinterpret_cast<u32x2*>(p) = v;
  }
}
template <int SEG>
__device__ __forceinline__ float seg_get(const Seg<SEG>& s, int e) {
  return (e & 1) ? bf_hi(s.w[e >> 1]) : bf_lo(s.w[e >> 1]);
}

// Two floats as an fp16 pair (low half first), rounded to nearest.
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)lo) | ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)hi) << 16);
}

// acc + both bf16 halves of w, in one dot-product instruction.  The row sums
// then add up the same bf16-rounded P that the PV product weights the values
// with.
__device__ __forceinline__ float sum2_bf16(uint32_t w, float acc) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, acc, false);
}

// Buffer resource over `bytes` bytes from `base`: loads at offsets at or past
// the end return zeros (raw buffer, stride 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const uint16_t* base, int32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), (short)0, bytes, 0x00020000);
}
__device__ __forceinline__ u32x4 buf_ld16(__amdgpu_buffer_rsrc_t r, int32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ u32x2 buf_ld8(__amdgpu_buffer_rsrc_t r, int32_t off) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}
// 16-byte store at device scope (sc1): written through to the memory side,
// where workgroups on other XCDs read it.
__device__ __forceinline__ void buf_st16_dev(u32x4 v, __amdgpu_buffer_rsrc_t r, int32_t off) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 16);
}

// Global data one wave stages for one KV tile.
template <int D, int R>
struct Unit {
  Seg<Pre<D, R>::SEG> klo, khi;   // K_base of the lane's rebuild token, both halves
  typename Ex<R>::Frag lk[Ex<R>::NC];  // L_k row of that token (expansion B operand)
  u32x4 v[Pre<D, R>::NHB];        // V_base half blocks (32 tokens x 16 dims, A layout)
  u32x4 lv[Pre<D, R>::NLP];       // L_v half blocks (32 tokens x 16 ranks, A layout)
  // Ranks >= 32: L_v of the V half blocks' 32 tokens, all ranks in 16-rank
  // chunks (A layout), for V = V_base + L_v B_v rebuilt on chip.
  u32x4 lvv[R >= 32 ? R / 16 : 1];
};

// PAGED: the caches are pools reached through block tables (a separate
// instantiation, so the contiguous kernel carries none of the walk's state).
// TCON: the instantiation that shares rebuilt tiles through the workspace
// tile cache (launched only when the call has one).
template <int D, int R, bool LK, bool LV, bool PAGED, bool TCON = false>
__global__ void __launch_bounds__(NTHR)
lrsa_prefill_kernel(const AttnArgs a) {
  using C = Pre<D, R, TCON && LK && D == 128 && !PAGED>;
  // Value side: rank 8 keeps associativity, P V_base + (P L_v) B_v, with the
  // softmax row sums in a spare row of (P L_v)^T.  From rank 16 on the
  // tile's V = V_base + L_v B_v is rebuilt on chip instead: per 64-token
  // tile a workgroup then spends 2 * 64 * d * r flop on the expansion rather
  // than 2 * 256 * 64 * r on P L_v, and needs no (P L_v)^T accumulator.
  constexpr bool VREB = LV && rebuilds_v(R);
  constexpr bool LVA = LV && !VREB;
  constexpr int NRB = LVA ? Pre<D, R>::RB : 1;
  constexpr bool ones_sum = LVA && R < 32;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][TKV * C::K_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][TKV * D];  // V^T fragments
  __shared__ __attribute__((aligned(16))) uint16_t lv_lds[LVA ? 2 : 1][LVA ? TKV * 32 * C::RB : 8];  // L_v^T fragments
  __shared__ __attribute__((aligned(16))) float2 base_cs[2][C::HALF];
  // cos/sin of each build lane's in-tile offset at its SEG frequencies,
  // [wave][pair of frequencies][lane] (one 16-byte read per pair), where
  // they are not kept in registers.
  __shared__ __attribute__((aligned(16))) f32x4 off_cs[LK && !C::OCS_REG ? NW : 1][C::SEG / 2][64];
  // cos/sin of each build lane's in-tile offset at its SEG frequencies,
  // [wave][pair of frequencies][lane] (one 16-byte read per pair).
  // B_k^T fragments of this KV head for ranks > 16, [RoPE half ph][block i]
  // [lane][rank chunk]: each lane's NC 16-byte fragments are contiguous.
  __shared__ __attribute__((aligned(16))) typename Ex<R>::Frag bk_lds[LK && !C::BK_REG ? 2 * 2 * C::NBW * 64 * C::NC : 1];
  // Rank-64 k+v with the tile cache: the B_v fragments of the value rebuild
  // wait in LDS (one copy per 32-dim block), since the rebuild runs for a
  // few tiles per wave only and their 16 VGPRs made the main loop spill.
  constexpr bool BV_LDS = TCON && LK && LV && R == 64 && D == 128 && !PAGED;
  __shared__ __attribute__((aligned(16))) u32x4 bv_lds[BV_LDS ? C::NDB * (R / 16) * 64 : 1];
  __shared__ int s_maxpos, s_minpos;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // Heaviest row tiles (latest positions, most keys) are dispatched first.
  // Grid: (row tile, KV head x KV split, request).
  const int nsp = a.pf_splits > 1 ? a.pf_splits : 1;
  const int rtile = gridDim.x - 1 - blockIdx.x, b = blockIdx.z;
  const int g = (int)blockIdx.y / nsp, split = (int)blockIdx.y - g * nsp;
  const int G = a.group;
  const int n_rows = a.n_tok * G;

  if (tid == 0) {
    s_maxpos = -1;
    s_minpos = INT32_MAX;
  }
  if constexpr (LK && !C::BK_REG) {
    // B_k [r, n_kv*d] (Eq. 1 orientation): rank j of head dim c at bh[j*ldb + c].
    const uint16_t* bh = a.Bk + (int64_t)b * a.b_stride + (int64_t)g * D;
    const int64_t ldb = (int64_t)a.n_kv * D;
    for (int e = tid; e < 2 * 2 * C::NBW * 64 * C::NC; e += NTHR) {
      const int c = e % C::NC, l = (e / C::NC) % 64, i = (e / (C::NC * 64)) % (2 * C::NBW);
      const int phe = e / (C::NC * 64 * 2 * C::NBW);
      const int blk = phe * C::NBW + (i % C::NBW) + (i / C::NBW) * C::NB;
      // Ranks > 16 use 32-wide chunks: 8 ranks per lane, one 16-byte fragment.
      const int r0 = Ex<R>::rank0(c, l >> 4);
      bk_lds[e] = Ex<R>::gather(bh + (int64_t)(r0 < R ? r0 : 0) * ldb + blk_dim<D>(blk, l & 15), ldb, r0 < R);
    }
  }
  int64_t kvl = a.kv_len[b];
  kvl = kvl < 0 ? 0 : (kvl > a.s_cap ? a.s_cap : kvl);

  // This lane's query row (the same row for lanes l and l^32).
  const int l32 = lane & 31, h32 = lane >> 5;
  const int row = rtile * BROWS + w * WROWS + l32;
  const bool row_ok = row < n_rows;
  const int qi = row_ok ? row / G : 0, hh = row_ok ? row - qi * G : 0;
  const int pos = row_ok ? a.positions[(int64_t)b * a.n_tok + qi] : -1;
  const int64_t last = (int64_t)pos < kvl - 1 ? (int64_t)pos : kvl - 1;  // last visible key

  __syncthreads();
  if (row_ok && last >= 0) atomicMax(&s_maxpos, (int)last);
  if (row_ok) atomicMin(&s_minpos, (int)(last < 0 ? -1 : last));
  __syncthreads();
  const int64_t kv_hi = (int64_t)s_maxpos + 1;  // keys [0, kv_hi) are needed
  const int n_tiles = (int)((kv_hi + TKV - 1) / TKV);
  // Tiles [0, n_full) lie wholly at or below every row's last visible key:
  // no row needs a mask there and every wave attends them.  Rank 64 with key
  // LR keeps the per-half loop for all tiles when it rebuilds every tile:
  // with it the straight-line main loop needs more registers than there are
  // (16 spilled against 4).  With the tile cache the rebuild (and its
  // spills) runs for a few tiles per wave only, and the main loop wins
  // (32k: 2.91 -> 2.56 ms; 64k, 2048 queries: 3.56 -> 3.24 ms).
  constexpr bool kMainLoop = R < 64 || (VREB && !LK) || (TCON && LK && D == 128 && !PAGED);
  const int n_full_raw = s_minpos < 0 ? 0 : (int)(((int64_t)s_minpos + 1) / TKV);
  const int n_full = !kMainLoop ? 0 : (n_full_raw < n_tiles ? n_full_raw : n_tiles);
  // This workgroup's tiles: all of them, or its split's share.
  const int t_lo = nsp > 1 ? (split * a.pf_split_tiles < n_tiles ? split * a.pf_split_tiles : n_tiles) : 0;
  const int t_hi = nsp > 1 ? (t_lo + a.pf_split_tiles < n_tiles ? t_lo + a.pf_split_tiles : n_tiles) : n_tiles;

  const int64_t row_el = (int64_t)a.n_kv * D;
  // This request's caches (or pools, paged through its rows of the block
  // tables).
  PageWalk walk;
  if constexpr (PAGED)
    walk.start(a.kv_tbl + (int64_t)b * a.max_blk, a.lr_tbl + (int64_t)b * a.max_blk, a.max_blk, a.blk, a.kv_nblk,
               a.lr_nblk, (int64_t)t_lo * TKV, kv_hi);
  const uint16_t* Kb = a.Kb + (int64_t)b * a.kv_stride + (int64_t)g * D;
  const uint16_t* Vb = a.Vb + (int64_t)b * a.kv_stride + (int64_t)g * D;
  const uint16_t* Lk = LK ? a.Lk + (int64_t)b * a.l_stride : nullptr;
  const uint16_t* Lv = LV ? a.Lv + (int64_t)b * a.l_stride : nullptr;

  // ---- tile cache -------------------------------------------------------------
  // Every full tile (all 64 rows below kv_hi) that a wave rebuilds is also
  // stored, as the wave's 4 KB part of the tile in LDS layout, to this
  // (request, KV head)'s slot of the workspace, and its flag is set once the
  // stores have completed.  A wave that finds the flag of its part set loads
  // the part instead of the raw rows and writes it to LDS unchanged: the
  // bytes are those the rebuild would produce.  No wave ever waits for a
  // flag, so there is no ordering between workgroups to deadlock on.  The
  // workgroups of a KV head walk their unmasked tiles from staggered
  // starting points, so each tile is mostly rebuilt once.  Flags are read
  // and data written at device scope (other XCDs' L2s are not coherent);
  // the data is read through L2, which holds no line of a part before its
  // flag was seen set (the flags are cleared by a kernel before this one).
  // Taken with LR on the keys (at rank 8 the L_v^T fragments, kept in
  // associativity form, are not part of a cached tile), and with LR on the
  // values only from rank 32
  // (at rank 64 the value rebuild alone costs 28% over plain attention; at
  // rank 16 there is too little to save).
  constexpr bool TC = TCON && (LK || (LV && R >= 32)) && D == 128 && !PAGED;
  constexpr bool tc_on = TC;
  // Q is scaled by log2(e)/sqrt(d) once (rounded to bf16) and the main
  // loop's score MFMAs start from a register block that holds minus the
  // reference maximum, so the exponentials read the scores directly.  It
  // needs 16 more VGPRs: taken by the tile-cache kernels up to rank 32 (their
  // build state lives in LDS) and by the kernels without key LR, not by the
  // others (they would spill).
  constexpr bool MSC = D == 128 && ((TC && R <= 32) || (!TCON && !LK));
  const float qscale = MSC ? 1.f : a.scale_log2;
  const int64_t tc_slot = ((int64_t)b * a.n_kv + g) * a.tc_tiles;  // first tile of the slot
  // Buffer resources over the slot's flags and data; empty (loads read 0)
  // when the cache is off, so that every path issues the same loads and the
  // compiler's load counting stays exact.  Offset INT32_MIN is out of range:
  // no access.  The stores of a built part and its flag are issued only
  // after a build, under a wave-uniform branch.
  const __amdgpu_buffer_rsrc_t tc_frsrc = __builtin_amdgcn_make_buffer_rsrc(
      tc_on ? a.tc_flags + tc_slot * NW : nullptr, (short)0, tc_on ? a.tc_tiles * NW * 4 : 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t tc_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      tc_on ? a.tc_data + tc_slot * NW * 1024 : nullptr, (short)0, tc_on ? a.tc_tiles * NW * 4096 : 0, 0x00020000);
  auto tc_off = [&](int T, int c) { return (T * NW + w) * 4096 + (c * 64 + lane) * 16; };

  // ---- build role: 16 tokens x SEG pair dims, 8 V rows, 8 L_v rows --------
  const int q = lane >> 4, c16 = lane & 15;
  const int tg = w & 3, ph = w >> 2;
  const int blk0 = ph * C::NBW;                    // first low 16-dim block
  const int lo_dim0 = q * C::QPG + blk0 * 4;       // first low dim of this lane
  const int delta = 16 * tg + c16;                 // rebuild token within a tile
  // V half blocks of this wave: token block vtb, dim block vdb, 16-dim halves
  // vp0 .. vp0 + NHB - 1 of it.
  const int vtb = w & 1, vdb = (w >> 1) % C::NDB, vp0 = C::NHB == 2 ? 0 : w / (2 * C::NDB);
  // Shifted identities (B operands): half p moves column 16p + k of a 16-wide
  // chunk to output column 16p + k, so the 32x32x16 product of a half block
  // of V or L_v rows (A operand: lane l = token l%32, columns (l/32)*8 + 0..7)
  // lands transposed, lane = column, in exactly the PV fragment order (exact
  // in bf16).
  u32x4 vid[2];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int i0 = (lane & 31) - 16 * p - (lane >> 5) * 8 - 2 * c;  // element index of the 1
      vid[p][c] = (i0 == 0 ? 0x3F80u : 0u) | (i0 == 1 ? 0x3F800000u : 0u);
    }
  // L_v half blocks of this wave (waves < 2 RB): tokens 32 ltb.., ranks 32 lrb..
  const int ltb = w & 1, lrb = w >> 1;
  const bool lv_wave = LVA && w < 2 * C::RB;
  // B_k^T fragment (16x16x16 A operand) of low block i (i < NBW) or of its
  // RoPE partner (i >= NBW), rank chunk rc: lane = dim row, 4 ranks from q*4.
  const uint16_t* bhead = LK ? a.Bk + (int64_t)b * a.b_stride + (int64_t)g * D : nullptr;
  const int64_t ldb = (int64_t)a.n_kv * D;  // row stride of the [r, n_kv*d] up-projections
  using Frag = typename Ex<R>::Frag;
  Frag bkr[C::BK_REG && LK ? 2 * C::NBW : 1][C::NC];
  if constexpr (C::BK_REG && LK) {
#pragma unroll
    for (int i = 0; i < 2 * C::NBW; ++i) {
      const int blk = blk0 + (i % C::NBW) + (i / C::NBW) * C::NB;
#pragma unroll
      for (int c = 0; c < C::NC; ++c) {
        const int r0 = Ex<R>::rank0(c, q);
        bkr[i][c] = Ex<R>::gather(bhead + (int64_t)(r0 < R ? r0 : 0) * ldb + blk_dim<D>(blk, c16), ldb, r0 < R);
      }
    }
  }
  // The NC fragments of block set i (registers, or 16-byte LDS reads).
  auto bk_set = [&](int i, Frag (&f)[C::NC]) {
    if constexpr (C::BK_REG) {
#pragma unroll
      for (int c = 0; c < C::NC; ++c) f[c] = bkr[i][c];
    } else {
      const typename Ex<R>::Frag* p = bk_lds + ((ph * 2 * C::NBW + i) * 64 + lane) * C::NC;
#pragma unroll
      for (int c = 0; c < C::NC; ++c) f[c] = p[c];
    }
  };
  // cos/sin of this build lane's in-tile offset angle at each of its SEG
  // frequencies: in registers as one fp16 pair per frequency (their fp16
  // rounding moves the rebuilt LR term by under 2^-11 of itself, far below
  // the bf16 rounding of the rebuilt key), or in LDS as fp32.
  uint32_t ocs[LK && C::OCS_REG ? C::SEG : 1];
  if constexpr (LK) {
#pragma unroll
    for (int e = 0; e < C::SEG; e += 2) {
      float c0, s0, c1, s1;
      rope_cs(delta, a.w2pi[lo_dim0 + e], c0, s0);
      rope_cs(delta, a.w2pi[lo_dim0 + e + 1], c1, s1);
      if constexpr (C::OCS_REG) {
        ocs[e] = pack_f16x2(c0, s0);
        ocs[e + 1] = pack_f16x2(c1, s1);
      } else {
        off_cs[w][e / 2][lane] = f32x4{c0, s0, c1, s1};
      }
    }
  }
  // Per-lane byte offsets of the staged data within a tile (constant); the
  // tile itself is addressed by buffer resources built per tile, whose
  // range check returns zeros for rows at or beyond kv_hi.
  const int32_t offk = delta * (int32_t)(row_el * 2) + lo_dim0 * 2;
  const int32_t offlk = delta * R * 2 + Ex<R>::rank0(0, q) * 2;
  int32_t offv[C::NHB];
#pragma unroll
  for (int hb = 0; hb < C::NHB; ++hb)
    offv[hb] = (32 * vtb + (lane & 31)) * (int32_t)(row_el * 2) + (32 * vdb + 16 * (vp0 + hb) + (lane >> 5) * 8) * 2;
  int32_t offlv[C::NLP];
#pragma unroll
  for (int p = 0; p < C::NLP; ++p) {
    const int r0 = 32 * lrb + 16 * p + (lane >> 5) * 8;
    offlv[p] = r0 < R ? (32 * ltb + (lane & 31)) * R * 2 + r0 * 2 : INT32_MIN;
  }
  // Ranks >= 32: L_v of the V block's tokens (A operand: lane = token l%32,
  // ranks 16 kc + (l/32)*8 ..) and B_v of its 32 dims (B operand: lane =
  // dim column l%32, same ranks), so that the expansion lands in the layout
  // of the V transpose.
  int32_t offlvv[VREB ? R / 16 : 1];
  u32x4 bvf[VREB && !BV_LDS ? R / 16 : 1];
  if constexpr (VREB) {
    const uint16_t* bvp = a.Bv + (int64_t)b * a.b_stride + (int64_t)g * D + 32 * vdb + (lane & 31);
#pragma unroll
    for (int kc = 0; kc < R / 16; ++kc) {
      offlvv[kc] = (32 * vtb + (lane & 31)) * R * 2 + (16 * kc + (lane >> 5) * 8) * 2;
      const u32x4 f = Ex<32>::gather(bvp + (int64_t)(16 * kc + (lane >> 5) * 8) * ldb, ldb, true);
      if constexpr (BV_LDS) {
        if ((w & 1) == 0) bv_lds[(vdb * (R / 16) + kc) * 64 + lane] = f;  // visible after the prologue's barrier
      } else {
        bvf[kc] = f;
      }
    }
  }
  // Tiles are loaded in token order, so paged caches are walked with them.
  // `cached`: the tile's part comes from the tile cache instead (its K and V
  // loads are pointed there, the L_k / L_v loads at empty resources).
  auto load_unit = [&](Unit<D, R>& u, int64_t t0, bool cached, int T) {
    // Valid rows of this tile; a tile at or past kv_hi gets empty resources
    // (its loads return zeros).
    const int64_t left = kv_hi - t0;
    const int rows_all = (int)(left < TKV ? (left > 0 ? left : 0) : TKV);
    const int rows = cached ? 0 : rows_all;
    const int32_t kv_bytes = rows > 0 ? (rows - 1) * (int32_t)(row_el * 2) + D * 2 : 0;
    int64_t kr = t0, lr = t0;  // cache rows of the tile's first token
    if constexpr (PAGED) walk.next(TKV, kv_hi, kr, lr);
    const auto rk = cached ? tc_rsrc : make_rsrc(Kb + kr * row_el, kv_bytes);
    const auto rv = cached ? tc_rsrc : make_rsrc(Vb + kr * row_el, kv_bytes);
    if constexpr (C::SEG == 8) {
      const u32x4 lo = buf_ld16(rk, cached ? tc_off(T, 0) : offk);
      const u32x4 hi = buf_ld16(rk, cached ? tc_off(T, 1) : offk + C::HALF * 2);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        u.klo.w[i] = lo[i];
        u.khi.w[i] = hi[i];
      }
    } else {
      const u32x2 lo = buf_ld8(rk, offk), hi = buf_ld8(rk, offk + C::HALF * 2);
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        u.klo.w[i] = lo[i];
        u.khi.w[i] = hi[i];
      }
    }
    if constexpr (LK) {
      const auto rl = make_rsrc(Lk + lr * R, rows * R * 2);
#pragma unroll
      for (int c = 0; c < C::NC; ++c) {
        if constexpr (Ex<R>::WIDE)
          u.lk[c] = buf_ld16(rl, offlk + c * 64);
        else
          u.lk[c] = Ex<R>::rank0(c, q) < R ? buf_ld8(rl, offlk) : u32x2{0u, 0u};
      }
    }
#pragma unroll
    for (int hb = 0; hb < C::NHB; ++hb) u.v[hb] = buf_ld16(rv, cached ? tc_off(T, 2 + hb) : offv[hb]);
    if constexpr (LVA) {
      // L_v^T fragments are not cached: their rows are loaded either way.
      const auto rl = make_rsrc(Lv + lr * R, rows_all * R * 2);
#pragma unroll
      for (int p = 0; p < C::NLP; ++p) u.lv[p] = lv_wave ? buf_ld16(rl, offlv[p]) : u32x4{0u, 0u, 0u, 0u};
    }
    if constexpr (VREB) {
      const auto rl = make_rsrc(Lv + lr * R, rows * R * 2);
#pragma unroll
      for (int kc = 0; kc < R / 16; ++kc) u.lvv[kc] = buf_ld16(rl, offlvv[kc]);
    }
  };
  // Tile-cache state of this wave: whether u holds a cached part (and of
  // which tile), and the tile whose part was stored but not yet flagged.
  bool u_cached = false;
  int u_tile = 0, pub_tile = -1;
  uint32_t fl_next = 0;  // flag of the tile fetched next (read a fetch ahead)
  auto publish = [&]() {
    // Only after a build (a few tiles per wave): vmcnt(0), so the part's
    // stores, issued a tile ago, have completed; then the flag, at device
    // scope, from every lane (same address, same value).  An unconditional
    // wait here drained the loads in flight on every tile and cost 2-4%.
    if (pub_tile >= 0) {
      __builtin_amdgcn_s_waitcnt(0x0F70);
      __builtin_amdgcn_raw_buffer_store_b32(1u, tc_frsrc, (pub_tile * NW + w) * 4, 0, 16);
      pub_tile = -1;
    }
  };
  auto rebuild = [&](const Unit<D, R>& u, int buf) {
    if constexpr (TC) publish();  // the previous part: its stores were issued a tile ago
    Seg<C::SEG> lo = u.klo, hi = u.khi;
    // With the cache, a cached part skips the rebuild: u holds the K rows of
    // this lane's token and its two V^T fragments as the rebuild makes them.
    const bool compute = !(TC && u_cached);
    u32x4 fv[2] = {u.v[0], u.v[C::NHB - 1]};
    if (compute) {
      if constexpr (LK) {
#pragma unroll
        for (int i = 0; i < C::NBW; ++i) {
          f32x4 elo = {0.f, 0.f, 0.f, 0.f}, ehi = {0.f, 0.f, 0.f, 0.f};
          Frag fl[C::NC], fh[C::NC];
          bk_set(i, fl);
          bk_set(C::NBW + i, fh);
#pragma unroll
          for (int c = 0; c < C::NC; ++c) {
            elo = Ex<R>::mma(fl[c], u.lk[c], elo);
            ehi = Ex<R>::mma(fh[c], u.lk[c], ehi);
          }
          float vlo[4], vhi[4];
          float cd[4], sd[4];
          if constexpr (C::OCS_REG) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              cd[j] = (float)__builtin_bit_cast(_Float16, (uint16_t)(ocs[4 * i + j] & 0xFFFFu));
              sd[j] = (float)__builtin_bit_cast(_Float16, (uint16_t)(ocs[4 * i + j] >> 16));
            }
          } else {
            const f32x4 od0 = off_cs[w][2 * i][lane], od1 = off_cs[w][2 * i + 1][lane];
            cd[0] = od0[0], cd[1] = od0[2], cd[2] = od1[0], cd[3] = od1[2];
            sd[0] = od0[1], sd[1] = od0[3], sd[2] = od1[1], sd[3] = od1[3];
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int e = 4 * i + j;
            const float2 bc = base_cs[buf][lo_dim0 + e];
            const float c = bc.x * cd[j] - bc.y * sd[j];
            const float s = bc.y * cd[j] + bc.x * sd[j];
            vlo[j] = seg_get(u.klo, e) + elo[j] * c - ehi[j] * s;
            vhi[j] = seg_get(u.khi, e) + ehi[j] * c + elo[j] * s;
          }
          lo.w[2 * i] = pack_bf16(vlo[0], vlo[1]);
          lo.w[2 * i + 1] = pack_bf16(vlo[2], vlo[3]);
          hi.w[2 * i] = pack_bf16(vhi[0], vhi[1]);
          hi.w[2 * i + 1] = pack_bf16(vhi[2], vhi[3]);
        }
      }
      // Transpose the V half blocks on the MFMA into fragments (2 vtb, vdb)
      // and (2 vtb + 1, vdb); from rank 16 on the transpose accumulates onto
      // L_v B_v of the same tokens and dims.
      f32x16 t;
#pragma unroll
      for (int j = 0; j < 16; ++j) t[j] = 0.f;
      if constexpr (VREB) {
#pragma unroll
        for (int kc = 0; kc < R / 16; ++kc) {
          u32x4 bv;
          if constexpr (BV_LDS)
            bv = bv_lds[(vdb * (R / 16) + kc) * 64 + lane];
          else
            bv = bvf[kc];
          t = mfma32x32x16(as_bf16x8(u.lvv[kc]), as_bf16x8(bv), t);
        }
      }
#pragma unroll
      for (int hb = 0; hb < C::NHB; ++hb) t = mfma32x32x16(as_bf16x8(u.v[hb]), as_bf16x8(vid[vp0 + hb]), t);
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int c = 0; c < 4; ++c) fv[hf][c] = pack_bf16(t[8 * hf + 2 * c], t[8 * hf + 2 * c + 1]);
    }
    st_seg<C::SEG>(k_lds[buf] + delta * C::K_ROW + lo_dim0, lo);
    st_seg<C::SEG>(k_lds[buf] + delta * C::K_ROW + C::HALF + lo_dim0, hi);
    // With one half block per wave (d = 64) the wave owns only its 16 dims
    // of each fragment; the other half's lanes are written by another wave.
    if (C::NHB == 2 || (lane & 31) / 16 == vp0) {
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
        *reinterpret_cast<u32x4*>(v_lds[buf] + (((2 * vtb + hf) * C::NDB + vdb) * 64 + lane) * 8) = fv[hf];
    }
    if constexpr (TC) {
      // A full tile rebuilt here goes to the cache too (flagged at the next
      // build).  The branch is wave-uniform; every wait on these stores is
      // the one in publish().
      const bool store_part = compute && tc_on && (u_tile + 1) * TKV <= kv_hi;
      if (store_part) {
        buf_st16_dev(u32x4{lo.w[0], lo.w[1], lo.w[2], lo.w[3]}, tc_rsrc, tc_off(u_tile, 0));
        buf_st16_dev(u32x4{hi.w[0], hi.w[1], hi.w[2], hi.w[3]}, tc_rsrc, tc_off(u_tile, 1));
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) buf_st16_dev(fv[hf], tc_rsrc, tc_off(u_tile, 2 + hf));
        pub_tile = u_tile;
      }
    }
    if (LVA && lv_wave) {
      // L_v^T fragments (2 ltb + hf, lrb).  With rank < 32, rank row `rank`
      // holds ones: the (P L_v)^T product then carries the softmax row sums in
      // its spare row for free.
      f32x16 t;
#pragma unroll
      for (int j = 0; j < 16; ++j) t[j] = 0.f;
#pragma unroll
      for (int p = 0; p < C::NLP; ++p) t = mfma32x32x16(as_bf16x8(u.lv[p]), as_bf16x8(vid[p]), t);
      const bool ones = ones_sum && (lane & 31) == R;
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        u32x4 f;
#pragma unroll
        for (int c = 0; c < 4; ++c) f[c] = ones ? 0x3F803F80u : pack_bf16(t[8 * hf + 2 * c], t[8 * hf + 2 * c + 1]);
        *reinterpret_cast<u32x4*>(lv_lds[buf] + (((2 * ltb + hf) * C::RB + lrb) * 64 + lane) * 8) = f;
      }
    }
  };
  // RoPE of each tile's first token, exact in fp64, by the last wave.  Its
  // lane's frequency is read once, outside the tile loop (a load in the loop
  // would make the compiler wait for the tile loads in flight).
  const double w2pi_lane = a.w2pi[lane < C::HALF ? lane : 0];
  auto base_angles = [&](int64_t t0, int buf) {
    if constexpr (LK) {
      if (w == NW - 1 && lane < C::HALF) {
        float c, s;
        rope_cs((int)t0, w2pi_lane, c, s);
        base_cs[buf][lane] = make_float2(c, s);
      }
    }
  };

  // ---- attend role ----------------------------------------------------------
  // Wave bounds: skip tiles no row of this wave sees; mask only tiles that
  // reach past some row's last visible key.
  int wave_last = (int)last, wave_first = row_ok ? (int)last : INT32_MAX;
#pragma unroll
  for (int x = 1; x < 64; x <<= 1) {
    const int o1 = __shfl_xor(wave_last, x, 64), o2 = __shfl_xor(wave_first, x, 64);
    wave_last = o1 > wave_last ? o1 : wave_last;
    wave_first = o2 < wave_first ? o2 : wave_first;
  }
  // Q^T as the B operand of S^T = K Q^T: lane col = row l%32,
  // k = (l/32)*8 + 0..7 within each 16-dim chunk.
  bf16x8 qf[C::NKQ];
  {
    const uint16_t* qp = a.Q + (((int64_t)b * a.n_tok + qi) * a.n_q + (int64_t)g * G + hh) * D;
#pragma unroll
    for (int kk = 0; kk < C::NKQ; ++kk) qf[kk] = as_bf16x8(ld16(qp + kk * 16 + h32 * 8, row_ok));
    if constexpr (MSC) {
#pragma unroll
      for (int kk = 0; kk < C::NKQ; ++kk) {
        u32x4 w = __builtin_bit_cast(u32x4, qf[kk]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float lo = __uint_as_float(w[i] << 16) * a.scale_log2, hi = __uint_as_float(w[i] & 0xFFFF0000u) * a.scale_log2;
          w[i] = pack_bf16(lo, hi);
        }
        qf[kk] = as_bf16x8(w);
      }
    }
  }
  // Let these one-time loads (Q, B_k) land before the tile loop: across the
  // loop's back edge the compiler could not tell them from the tile loads in
  // flight and would wait for all of those at the first score MFMA.
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  f32x16 acc[C::NDB];   // O^T: lane col = row l%32
  f32x16 accl[NRB];     // (P L_v)^T
#pragma unroll
  for (int db = 0; db < C::NDB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[db][j] = 0.f;
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int j = 0; j < 16; ++j) accl[rb][j] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 negm;  // MSC: minus the reference maximum (0 while there is none)
#pragma unroll
  for (int j = 0; j < 16; ++j) negm[j] = 0.f;


  // The two waves of a SIMD (w and w + 4, or w and w ^ 1, depending on how the
  // workgroup is laid out) take the two jobs in opposite order.
  const bool build_first = ((w >> 2) ^ w) & 1;

  // Tiles are walked as a sequence k = t_lo .. t_hi - 1, LDS buffer k & 1.
  // With the tile cache the unmasked tiles of this workgroup's range are
  // walked from a starting point staggered over the row tiles of the KV
  // head (the online softmax does not depend on the order), the rest in
  // order.
  // The starting points are shared by groups of row tiles that run on one
  // XCD (workgroup i runs on XCD i % 8, so row tiles r, r + 8, r + 16, ...):
  // a group walks nearly in step, so one memory-side read of a cached part
  // serves its workgroups through L2.  Groups of four from 32 row tiles on,
  // of two from 16 (32k rank 16: 2.318 -> 2.263 ms; 64k rank 64: 3.304 ->
  // 3.125 ms; groups of eight measured slower, and with 8 row tiles, one per
  // XCD, grouping only adds rebuilds).  Member m of a group starts kMemberLag
  // tiles after member m - 1 rather than at the same tile: members that
  // start together all rebuild every tile of the group's own stretch, while
  // a few tiles of lag let the later members find most of them published
  // and still keep the group's reads close enough to share L2 (32k rank 16:
  // no lag 2.239 ms, lags 1, 2, 3: 2.207, 2.197, 2.194 ms on one box; lags 3,
  // 5, 8: 2.150, 2.182, 2.268 ms on another; rank 64 2.429 -> 2.353 ms).
  constexpr int kMemberLag = 3;
  const int r_end = tc_on ? (n_full_raw < t_hi ? n_full_raw : t_hi) : t_lo;  // rotated steps [t_lo, r_end)
  const int n_rot = r_end > t_lo ? r_end - t_lo : 0;
  const int gsz = gridDim.x >= 32 ? 4 : (gridDim.x >= 16 ? 2 : 1);
  const int ngrp = (int)((gridDim.x + 8 * gsz - 1) / (8 * gsz)) * 8;  // > every group index
  const int grp = (rtile / (8 * gsz)) * 8 + rtile % 8;
  const int member = (rtile / 8) % gsz;
  const int rot =
      n_rot > 0 ? (int)((((int64_t)grp * n_rot) / ngrp + (int64_t)member * kMemberLag) % n_rot) : 0;
  auto tile_at = [&](int k) {
    if (k >= t_lo + n_rot) return k;
    const int t = k + rot;
    return t >= t_lo + n_rot ? t - n_rot : t;
  };
  // Loads of sequence step k into u: its cached part if the flag read one
  // fetch earlier says it is published, else the raw rows.  The flag of the
  // next step's tile is read here for the next fetch.
  Unit<D, R> u;
  auto fetch = [&](int k) {
    const int T = tile_at(k);
    bool cached = false;
    if constexpr (TC) {
      cached = tc_on && __builtin_amdgcn_readfirstlane(fl_next) != 0;
      u_cached = cached;
      u_tile = T;
      const int Tn = tile_at(k + 1);
      fl_next = __builtin_amdgcn_raw_buffer_load_b32(tc_frsrc, Tn < n_tiles ? (Tn * NW + w) * 4 : INT32_MIN, 0, 16);
    }
    load_unit(u, (int64_t)T * TKV, cached, T);
  };

  // Prologue: the first tile into its LDS buffer (tile parity), the next in
  // flight.
  if (t_lo < t_hi) {
    fetch(t_lo);
    base_angles((int64_t)tile_at(t_lo) * TKV, t_lo & 1);
  }
  __syncthreads();
  if (t_lo < t_hi) rebuild(u, t_lo & 1);
  if (t_lo + 1 < t_hi) {
    fetch(t_lo + 1);
    base_angles((int64_t)tile_at(t_lo + 1) * TKV, (t_lo + 1) & 1);
  }
  __syncthreads();

  // Main loop, tiles that need no mask: the scores of both halves, one
  // maximum and one (rare) rescale per tile, then a single straight-line
  // block that holds the exponentials and PV of both halves and the build of
  // the next tile, so that the compiler can interleave the build's vector
  // work and transposes with the PV MFMAs.  A wave raises its issue
  // priority while it attends, so that when the two waves of a SIMD are in
  // different parts of the tile the one with the MFMA-heavy work issues
  // first.  With LR keys (a heavier build) the two waves also take the
  // build and the attention in opposite order, as in the per-half loop
  // (not over paged caches, where it measured slower).
  int tile = t_lo;  // sequence step (the tile itself is tile_at(tile))
  const int main_end = n_full < t_hi ? n_full : t_hi;
  if constexpr (kMainLoop)
  for (; tile < main_end; ++tile) {
    const int buf = tile & 1;
    const bool build_now = LK && !PAGED && build_first;
    if (build_now) {
      rebuild(u, buf ^ 1);
      fetch(tile + 2);
    }
    __builtin_amdgcn_s_setprio(1);
    bf16x8 kf[C::NKQ];
    auto k_frag = [&](int tb, int kk) {
      return as_bf16x8(*reinterpret_cast<const u32x4*>(k_lds[buf] + (tb * 32 + l32) * C::K_ROW + h32 * 8 + kk * 16));
    };
    f32x16 sh[2];
#pragma unroll
    for (int kk = 0; kk < C::NKQ; ++kk) kf[kk] = k_frag(0, kk);
    f32x16 zinit;
#pragma unroll
    for (int j = 0; j < 16; ++j) zinit[j] = 0.f;
    sh[0] = mfma32x32x16(kf[0], qf[0], MSC ? negm : zinit);
    kf[0] = k_frag(1, 0);
#pragma unroll
    for (int kk = 1; kk < C::NKQ; ++kk) {
      sh[0] = mfma32x32x16(kf[kk], qf[kk], sh[0]);
      kf[kk] = k_frag(1, kk);
    }
    sh[1] = mfma32x32x16(kf[0], qf[0], MSC ? negm : zinit);
#pragma unroll
    for (int kk = 1; kk < C::NKQ; ++kk) sh[1] = mfma32x32x16(kf[kk], qf[kk], sh[1]);
    float mx = fmaxf(sh[0][0], sh[0][1]);
#pragma unroll
    for (int j = 2; j < 16; ++j) mx = fmaxf(mx, sh[0][j]);
#pragma unroll
    for (int j = 0; j < 16; ++j) mx = fmaxf(mx, sh[1][j]);
    // MSC: the scores are relative to the reference ms0 (0 before the first
    // maximum is known).
    const float ms0 = (m_run == -INFINITY) ? 0.f : m_run;
    mx = MSC ? max_xor32(mx) + ms0 : max_xor32(mx) * a.scale_log2;
    if (__ballot(mx > m_run + kRescaleLog2)) {
      const float mn = fmaxf(m_run, mx);
      const float alpha = fast_exp2(m_run - (mn == -INFINITY ? 0.f : mn));
#pragma unroll
      for (int db = 0; db < C::NDB; ++db) acc[db] *= alpha;
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) accl[rb] *= alpha;
      l_run *= alpha;
      m_run = mn;
      if constexpr (MSC) {
        const float shift = (mn == -INFINITY ? 0.f : mn) - ms0;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          sh[0][j] -= shift;
          sh[1][j] -= shift;
          negm[j] = -(mn == -INFINITY ? 0.f : mn);
        }
      }
    }
    const float ms = (m_run == -INFINITY) ? 0.f : m_run;
    float ls = 0.f;
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const uint16_t* vt = v_lds[buf];
      const uint16_t* lvt = lv_lds[buf];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        bf16x8 vf[C::NDB], lvf[NRB];
#pragma unroll
        for (int db = 0; db < C::NDB; ++db)
          vf[db] = as_bf16x8(*reinterpret_cast<const u32x4*>(vt + (((2 * tb + hf) * C::NDB + db) * 64 + lane) * 8));
        if constexpr (LVA) {
#pragma unroll
          for (int rb = 0; rb < C::RB; ++rb)
            lvf[rb] = as_bf16x8(*reinterpret_cast<const u32x4*>(lvt + (((2 * tb + hf) * C::RB + rb) * 64 + lane) * 8));
        }
        u32x4 pw;  // bf16 P of this 16-token chunk
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const float p0 = MSC ? fast_exp2(sh[tb][hf * 8 + 2 * c]) : fast_exp2(__builtin_fmaf(sh[tb][hf * 8 + 2 * c], a.scale_log2, -ms));
          const float p1 = MSC ? fast_exp2(sh[tb][hf * 8 + 2 * c + 1]) : fast_exp2(__builtin_fmaf(sh[tb][hf * 8 + 2 * c + 1], a.scale_log2, -ms));
          pw[c] = pack_bf16(p0, p1);
          if constexpr (!ones_sum) ls = sum2_bf16(pw[c], ls);
        }
        const bf16x8 pb = as_bf16x8(pw);
#pragma unroll
        for (int db = 0; db < C::NDB; ++db) acc[db] = mfma32x32x16(vf[db], pb, acc[db]);
        if constexpr (LVA) {
#pragma unroll
          for (int rb = 0; rb < C::RB; ++rb) accl[rb] = mfma32x32x16(lvf[rb], pb, accl[rb]);
        }
      }
    }
    if constexpr (!ones_sum) l_run += ls;
    __builtin_amdgcn_s_setprio(0);
    // Build tile + 1 and start the loads of tile + 2 (past the last tile this
    // writes a buffer no wave reads again and loads nothing).
    if (!build_now) {
      rebuild(u, buf ^ 1);
      fetch(tile + 2);
    }
    base_angles((int64_t)tile_at(tile + 2) * TKV, buf);
    __syncthreads();  // tile + 1 in LDS; tile consumed by every wave
  }

  // Tiles that cross some row's causal limit.
  for (; tile < t_hi; ++tile) {
    const int buf = tile & 1;
    const int64_t t0 = (int64_t)tile_at(tile) * TKV;
    // Build step + 1 (its data arrived during the previous step) and start
    // the loads of step + 2.
    auto build = [&]() {
      if (tile + 1 < t_hi) rebuild(u, buf ^ 1);
      if (tile + 2 < t_hi) fetch(tile + 2);
    };
    if (build_first) build();
    if (t0 <= (int64_t)wave_last) {
      // K fragments (A operand of S^T = K Q^T) of one half.
      bf16x8 kf[C::NKQ];
      auto k_frag = [&](int tb, int kk) {
        return as_bf16x8(*reinterpret_cast<const u32x4*>(k_lds[buf] + (tb * 32 + l32) * C::K_ROW + h32 * 8 + kk * 16));
      };
      // Scores of the first half.  Each second-half K fragment is read as
      // soon as the first half's MFMA has taken its register (harmless when
      // that half is unused).
      f32x16 s, s_next;
#pragma unroll
      for (int kk = 0; kk < C::NKQ; ++kk) kf[kk] = k_frag(0, kk);
#pragma unroll
      for (int j = 0; j < 16; ++j) s[j] = 0.f;
#pragma unroll
      for (int kk = 0; kk < C::NKQ; ++kk) {
        s = mfma32x32x16(kf[kk], qf[kk], s);
        kf[kk] = k_frag(1, kk);
      }
      // The tile is consumed as two 32-token halves, each with its own online
      // softmax update.  Per half: mask and row maximum, the (rare) rescale,
      // then one straight-line block in which the exponentials run beside
      // MFMAs: the second half's scores during the first half's softmax, and
      // each 16-token chunk's PV beside the next chunk's exponentials.
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        const int64_t th = t0 + tb * 32;  // first token of this half
        if (th > (int64_t)wave_last) break;
        if (tb == 1) s = s_next;
        if (th + 31 > (int64_t)wave_first) {  // this half crosses some row's causal limit
          // Positions fit in 32 bits (s_cap < 2^31): key t is masked iff t > last.
          const int rel = (int)last - (int)th - h32 * 4;  // last - (first token of this lane)
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if ((j >> 2) * 8 + (j & 3) > rel) s[j] = -INFINITY;
        }
        float mx = s[0];
#pragma unroll
        for (int j = 1; j < 16; ++j) mx = fmaxf(mx, s[j]);
        mx = max_xor32(mx) * qscale;
        // Lazy rescale: the reference maximum m_run only moves when some row's
        // maximum exceeds it by more than 2^8, so P stays below 256 and the
        // accumulators are rescaled a handful of times per row.
        if (__ballot(mx > m_run + kRescaleLog2)) {
          const float mn = fmaxf(m_run, mx);
          const float alpha = fast_exp2(m_run - (mn == -INFINITY ? 0.f : mn));
#pragma unroll
          for (int db = 0; db < C::NDB; ++db) acc[db] *= alpha;
#pragma unroll
          for (int rb = 0; rb < NRB; ++rb) accl[rb] *= alpha;
          l_run *= alpha;
          m_run = mn;
        }
        const float ms = (m_run == -INFINITY) ? 0.f : m_run;
        // PV A fragments of this half.
        const uint16_t* vt = v_lds[buf];
        const uint16_t* lvt = lv_lds[buf];
        bf16x8 vf[2][C::NDB], lvf[2][NRB];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
#pragma unroll
          for (int db = 0; db < C::NDB; ++db)
            vf[hf][db] = as_bf16x8(*reinterpret_cast<const u32x4*>(vt + (((2 * tb + hf) * C::NDB + db) * 64 + lane) * 8));
          if constexpr (LVA) {
#pragma unroll
            for (int rb = 0; rb < C::RB; ++rb)
              lvf[hf][rb] = as_bf16x8(*reinterpret_cast<const u32x4*>(lvt + (((2 * tb + hf) * C::RB + rb) * 64 + lane) * 8));
          }
        }
        if (tb == 0) {
#pragma unroll
          for (int j = 0; j < 16; ++j) s_next[j] = 0.f;
#pragma unroll
          for (int kk = 0; kk < C::NKQ; ++kk) s_next = mfma32x32x16(kf[kk], qf[kk], s_next);
        }
        float ls0 = 0.f, ls1 = 0.f;
        u32x4 pw[2];  // bf16 P of this half, one per 16-token chunk
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const float p0 = fast_exp2(__builtin_fmaf(s[hf * 8 + 2 * c], qscale, -ms));
            const float p1 = fast_exp2(__builtin_fmaf(s[hf * 8 + 2 * c + 1], qscale, -ms));
            pw[hf][c] = pack_bf16(p0, p1);
            if constexpr (!ones_sum) {
              if (c & 1) ls1 = sum2_bf16(pw[hf][c], ls1);
              else ls0 = sum2_bf16(pw[hf][c], ls0);
            }
          }
        if constexpr (!ones_sum) l_run += ls0 + ls1;
        // O^T[dims x rows] += V^T[dims x 16 tok] P^T[16 tok x rows] for the two
        // 16-token chunks of this half; (P L_v)^T likewise with L_v^T.
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const bf16x8 pb = as_bf16x8(pw[hf]);
#pragma unroll
          for (int db = 0; db < C::NDB; ++db) acc[db] = mfma32x32x16(vf[hf][db], pb, acc[db]);
          if constexpr (LVA) {
#pragma unroll
            for (int rb = 0; rb < C::RB; ++rb) accl[rb] = mfma32x32x16(lvf[hf][rb], pb, accl[rb]);
          }
        }
      }
    }
    if (!build_first) build();
    if (tile + 2 < t_hi) base_angles((int64_t)tile_at(tile + 2) * TKV, buf);
    __syncthreads();  // tile + 1 in LDS; tile consumed by every wave
  }

  if constexpr (TC) publish();  // the last part this wave stored

  // Row sum: from the ones row of (P L_v)^T (row R: register 4 (R/8) + R%4 of
  // block 0 in lanes (R%8)/4*32 .. +31), else from the per-lane partial sums.
  float l_tot;
  if constexpr (ones_sum) {
    constexpr int jr = 4 * ((R % 32) / 8) + (R % 4);
    l_tot = __shfl(accl[0][jr], l32 + 32 * ((R % 8) / 4), 64);
  } else {
    l_tot = sum_xor32(l_run);
  }
  if (nsp > 1) {
    // ---- split epilogue: this split's partial (m, l, O^T, (P L_v)^T) for
    // the merge, which applies B_v and 1/l.
    if (!row_ok) return;
    constexpr int PS = 4 + D + R;
    const int64_t orow = ((int64_t)b * a.n_tok + qi) * a.n_q + (int64_t)g * G + hh;
    float* wsp = a.ws + (orow * nsp + split) * PS;
    if (h32 == 0) {
      wsp[0] = m_run;
      wsp[1] = l_tot;
    }
#pragma unroll
    for (int db = 0; db < C::NDB; ++db)
#pragma unroll
      for (int jg = 0; jg < 4; ++jg)
        *reinterpret_cast<f32x4*>(wsp + 4 + db * 32 + jg * 8 + h32 * 4) =
            f32x4{acc[db][jg * 4], acc[db][jg * 4 + 1], acc[db][jg * 4 + 2], acc[db][jg * 4 + 3]};
    if constexpr (LVA) {
#pragma unroll
      for (int rb = 0; rb < C::RB; ++rb)
#pragma unroll
        for (int jg = 0; jg < 4; ++jg) {
          const int rk = rb * 32 + jg * 8 + h32 * 4;
          if (rk < R)
            *reinterpret_cast<f32x4*>(wsp + 4 + D + rk) =
                f32x4{accl[rb][jg * 4], accl[rb][jg * 4 + 1], accl[rb][jg * 4 + 2], accl[rb][jg * 4 + 3]};
        }
    }
    return;
  }

  // ---- epilogue: O^T += B_v^T (P L_v)^T, then O = acc / l, lse -------------
  if constexpr (LVA) {
    // (P L_v)^T registers of rank chunk jc (16 ranks) are the B operand in
    // the same k order as P; split into bf16 hi + lo to keep fp32 accuracy.
#pragma unroll
    for (int jc = 0; jc < C::RC; ++jc) {
      const int rb = jc >> 1, j0 = 8 * (jc & 1);
      u32x4 hi, lo;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float x0 = accl[rb][j0 + 2 * c], x1 = accl[rb][j0 + 2 * c + 1];
        hi[c] = pack_bf16(x0, x1);
        lo[c] = pack_bf16(x0 - bf_lo(hi[c]), x1 - bf_hi(hi[c]));
      }
      const int r0 = 16 * jc + 4 * h32;
#pragma unroll
      for (int db = 0; db < C::NDB; ++db) {
        const int dim = db * 32 + l32;
        const uint16_t* bv = a.Bv + (int64_t)b * a.b_stride + (int64_t)g * D + dim;
        const u32x2 b0 = Ex<R>::gather(bv + (int64_t)(r0 < R ? r0 : 0) * ldb, ldb, r0 < R);
        const u32x2 b1 = Ex<R>::gather(bv + (int64_t)(r0 + 8 < R ? r0 + 8 : 0) * ldb, ldb, r0 + 8 < R);
        const u32x4 bw = {b0[0], b0[1], b1[0], b1[1]};
        acc[db] = mfma32x32x16(as_bf16x8(bw), as_bf16x8(hi), acc[db]);
        acc[db] = mfma32x32x16(as_bf16x8(bw), as_bf16x8(lo), acc[db]);
      }
    }
  }
  if (!row_ok) return;
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  uint16_t* op = a.O + (((int64_t)b * a.n_tok + qi) * a.n_q + (int64_t)g * G + hh) * D;
#pragma unroll
  for (int db = 0; db < C::NDB; ++db)
#pragma unroll
    for (int jg = 0; jg < 4; ++jg) {
      const int dim = db * 32 + jg * 8 + h32 * 4;
      u32x2 o;
      o[0] = pack_bf16(acc[db][jg * 4 + 0] * inv, acc[db][jg * 4 + 1] * inv);
      o[1] = pack_bf16(acc[db][jg * 4 + 2] * inv, acc[db][jg * 4 + 3] * inv);
      *reinterpret_cast<u32x2*>(op + dim) = o;
    }
  if (a.lse != nullptr && h32 == 0)
    a.lse[((int64_t)b * a.n_tok + qi) * a.n_q + (int64_t)g * G + hh] =
        l_tot > 0.f ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
}

template <int D, int R, bool LK, bool LV>
hipError_t launch_t(const AttnArgs& a, hipStream_t st) {
  const int n_rows = a.n_tok * a.group;
  const int tiles = (n_rows + BROWS - 1) / BROWS;
  const int nsp = a.pf_splits > 1 ? a.pf_splits : 1;
  const dim3 grid(tiles, a.n_kv * nsp, a.batch);
  if (a.kv_tbl != nullptr)
    hipLaunchKernelGGL((lrsa_prefill_kernel<D, R, LK, LV, true>), grid, dim3(NTHR), 0, st, a);
  else if constexpr ((LK || (LV && R >= 32)) && D == 128) {
    if (a.tc_data != nullptr)
      hipLaunchKernelGGL((lrsa_prefill_kernel<D, R, LK, LV, false, true>), grid, dim3(NTHR), 0, st, a);
    else
      hipLaunchKernelGGL((lrsa_prefill_kernel<D, R, LK, LV, false>), grid, dim3(NTHR), 0, st, a);
  } else {
    hipLaunchKernelGGL((lrsa_prefill_kernel<D, R, LK, LV, false>), grid, dim3(NTHR), 0, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nsp == 1) return e;
  AttnArgs m = a;
  m.n_splits = nsp;
  // The partials are laid out for the rank this kernel was built with (a
  // call without LR runs the rank-8 build whatever dims.rank says).
  m.rank = R;
  // With V rebuilt in the tile B_v is already inside it: the partials carry
  // no (P L_v) part for the merge to expand.
  if (LV && rebuilds_v(R)) m.Lv = nullptr;
  return launch_split_merge(m, st);
}

template <int D, int R>
hipError_t launch_lr(const AttnArgs& a, hipStream_t st) {
  const bool lk = a.Lk != nullptr, lv = a.Lv != nullptr;
  if (lk && lv) return launch_t<D, R, true, true>(a, st);
  if (lk) return launch_t<D, R, true, false>(a, st);
  if (lv) return launch_t<D, R, false, true>(a, st);
  return launch_t<D, 8, false, false>(a, st);  // no LR: the rank is irrelevant
}

template <int D>
hipError_t launch_r(const AttnArgs& a, hipStream_t st) {
  switch (a.rank) {
    case 8: return launch_lr<D, 8>(a, st);
    case 16: return launch_lr<D, 16>(a, st);
    case 32: return launch_lr<D, 32>(a, st);
    case 64: return launch_lr<D, 64>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

void prefill_plan(int n_tok, int group, int n_kv, int batch, int64_t s_cap, int cus, int* splits,
                  int* split_tiles) {
  // Units of work without a split: (row tile, KV head, request), one
  // workgroup per CU at a time.  Splitting the KV tiles ns ways gives
  // units * ns workgroups of 1/ns the work, so the time per CU goes as
  // ceil(units * ns / CUs) / ns.  Take the ns in 1..8 (splits at least 8
  // tiles long) that minimises it, the smallest on ties, and split only when
  // that model gains at least a tenth over one pass: every split adds fp32
  // partials to write and merge, which a gain of a few per cent does not pay.
  const int64_t n_cu = cus > 0 ? cus : 1;
  const int64_t rows = (int64_t)n_tok * group;
  const int64_t units = ((rows + BROWS - 1) / BROWS) * n_kv * (batch > 0 ? batch : 1);
  const int64_t tiles = (s_cap + TKV - 1) / TKV;
  const double one_pass = (double)((units + n_cu - 1) / n_cu);
  int64_t best = 1;
  double best_cost = one_pass;
  for (int64_t ns = 2; ns <= 8 && ns <= tiles / 8; ++ns) {
    const double cost = (double)((units * ns + n_cu - 1) / n_cu) / (double)ns;
    if (cost < best_cost - 1e-9) {
      best = ns;
      best_cost = cost;
    }
  }
  *splits = 1;
  *split_tiles = (int)(tiles > 0 ? tiles : 1);
  if (best < 2 || best_cost > 0.9 * one_pass) return;
  const int64_t st = (tiles + best - 1) / best;
  *splits = (int)((tiles + st - 1) / st);
  *split_tiles = (int)st;
}

size_t prefill_workspace_bytes(int batch, int n_tok, int n_q, int splits, int head_dim, int rank) {
  if (splits <= 1) return 0;
  return (size_t)batch * n_tok * n_q * splits * (4 + head_dim + rank) * sizeof(float);
}

bool prefill_uses_tile_cache(int n_tok, int group, int head_dim, int rank, bool has_lk, bool has_lv, bool paged) {
  const int64_t row_tiles = ((int64_t)n_tok * group + BROWS - 1) / BROWS;
  return (has_lk || (has_lv && rank >= 32)) && !paged && head_dim == 128 && rank >= 8 && row_tiles >= 8;
}

namespace {
int64_t tc_slot_tiles(int64_t s_cap) { return (s_cap + TKV - 1) / TKV; }
}  // namespace

size_t prefill_tile_cache_flag_bytes(int batch, int n_kv, int64_t s_cap) {
  const size_t flags = (size_t)batch * n_kv * tc_slot_tiles(s_cap) * NW * sizeof(uint32_t);
  return (flags + 255) / 256 * 256;
}

size_t prefill_tile_cache_bytes(int batch, int n_kv, int64_t s_cap) {
  // Flags, then 32 KB of rebuilt K and V^T per tile.  A slot is addressed
  // with 32-bit offsets, so it must stay under 2 GB (s_cap < 4M tokens).
  if (tc_slot_tiles(s_cap) * NW * 4096 >= ((int64_t)1 << 31)) return 0;
  return prefill_tile_cache_flag_bytes(batch, n_kv, s_cap) +
         (size_t)batch * n_kv * tc_slot_tiles(s_cap) * NW * 4096;
}

namespace {
// Clears the tile cache's flags (a kernel, not a memset, so that the call can
// be captured into a graph).
__global__ void __launch_bounds__(256) tc_clear_kernel(uint32_t* flags, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) flags[i] = 0u;
}
}  // namespace

hipError_t launch_prefill(const AttnArgs& a, hipStream_t st) {
  if (a.tc_data != nullptr) {
    const int64_t n = (int64_t)a.batch * a.n_kv * a.tc_tiles * NW;
    const int64_t blocks = (n + 255) / 256;
    hipLaunchKernelGGL(tc_clear_kernel, dim3((unsigned)(blocks < 1024 ? blocks : 1024)), dim3(256), 0, st, a.tc_flags, n);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  }
  if (a.head_dim == 64) return launch_r<64>(a, st);
  if (a.head_dim == 128) return launch_r<128>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace prc
