// LR-shared attention, decode (one query token per request), gfx950.
//
// Reuse step of PreLRShared (Sec. 3.1): the current agent attends over the
// shared base cache plus its own rank-r LR cache.  Keys are rebuilt on chip,
// K = K_base + RoPE(L_k B_k), with the rank-r expansion done before RoPE
// (App. D.2).  Values use the associativity of App. D.2:
//     P (V_base + L_v B_v) = P V_base + (P L_v) B_v,
// so only an r-wide accumulator is carried per head and B_v is applied once,
// in the merge.
//
// Work split (flash-decoding): one workgroup per (request, KV-range split,
// group of up to 8 KV heads); one wavefront per KV head.  The waves of a
// workgroup walk the same tokens, so the RoPE cos/sin table of each 32-token
// tile is built once in LDS for all heads, and the per-token LR rows are read
// through shared L1 lines.  A second kernel merges the split partials with
// log-sum-exp weights.
//
// Per 16-token sub-block, each wave (lane l: query head l%16 of the group,
// q = l/16):
//   1. scores S^T = K Q^T on 16x16x32 MFMAs in two parts: the raw bf16
//      K_base rows (no rounding) plus bf16(RoPE(E)), where E^T = B_k^T L_k^T
//      comes from 16x16 MFMAs (16x16x32 over 32-rank chunks for ranks 32 and
//      64, 16x16x16 below) whose result layout holds both halves of every
//      RoPE pair in one lane;
//   2. online softmax per head (lane l%16), exp2 domain, lazily rescaled;
//   3. O^T += V^T P^T and (P L_v)^T += L_v^T P^T on 16x16x16 MFMAs.  V and
//      L_v rows pass through a wave-private LDS tile and come back through
//      the transposing LDS read (ds_read_b64_tr_b16), so P, already in B
//      operand layout, needs no shuffles and the softmax rescale is a
//      per-lane scalar.
// The loads of the next sub-block (the next two in the 4-wave rank-64
// kernel) are in flight while the current one is consumed.  The contiguous
// rank-64 kernel at d = 128 sends its V rows straight to LDS (direct
// global->LDS loads into a two-buffer ring) instead of through registers.
#include "common.hpp"
#include "kernels.hpp"
#include "rebuild.hpp"

namespace prc {
namespace {

constexpr int TK = 32;        // tokens per KV tile (one LDS table, one barrier)
constexpr int NSB = TK / 16;  // 16-token sub-blocks per tile
constexpr float kRescaleLog2 = 8.f;  // lazy-rescale threshold (log2 domain)
// Waves per workgroup (one KV head each).  Rank 64 keeps its B_k^T
// fragments (64 VGPRs) in registers; with V staged in registers that needs
// one wave per SIMD (the whole register file, architected plus accumulation
// registers) to avoid spilling.
constexpr int dec_waves(int rank) { return rank >= 64 ? 4 : 8; }
// Sub-blocks whose loads are in flight ahead of the one being consumed.  With
// one wave per SIMD (rank 64) no other wave hides a wave's load latency, and
// the whole register file leaves room for one more staged sub-block; at two
// waves per SIMD the extra stage spills and loses.
constexpr int dec_prefetch(int rank) { return rank >= 64 ? 2 : 1; }
// Contiguous rank-64 decode at d = 128 instead stages its V rows by direct
// global->LDS loads, which frees the registers the V stages take: with one
// sub-block in flight it then fits in 256 registers (251), so it runs 8-wave
// workgroups, two waves per SIMD, like the lower ranks (64k, 8 requests:
// 467 -> 440 us).  Paged caches keep the 4-wave form (their walk issues
// block-table loads between the stages, which the fixed load count of the
// V wait below does not cover).
constexpr bool dec_vdma(int d, int rank, bool paged) { return d == 128 && rank == 64 && !paged; }
constexpr int dec_nw(int d, int rank, bool paged) { return dec_vdma(d, rank, paged) ? 8 : dec_waves(rank); }
constexpr int gcd_c(int a, int b) { return b == 0 ? a : gcd_c(b, a % b); }

template <int D, int R, bool VD = false>
struct Dec {
  static constexpr int NW = VD ? 8 : dec_waves(R);  // waves per workgroup (KV heads)
  static constexpr int NT = NW * 64;         // threads per workgroup
  static constexpr int HALF = D / 2;
  static constexpr int NB = D / 32;           // 16-dim blocks per RoPE half
  static constexpr int NBLK = D / 16;         // 16-dim blocks
  static constexpr int NCH = D / 32;          // 8-dim chunks per lane
  static constexpr int QPG = D / 8;           // dims per lane group per half
  static constexpr int RC = RCH(R);           // 16-wide rank chunks
  // float2 per table row.  A lane reads row l%16 at frequencies from
  // (l/16)*QPG; with an odd row length (d = 128) the 32 lanes of each
  // half-wave pass then cover all 64 banks once.
  static constexpr int CS_ROW = D == 128 ? HALF + 1 : HALF + 2;
  static constexpr int EPT = TK * HALF / NT;  // table entries per thread
  // Row strides of the tiles read with ds_read_b64_tr_b16: the two 16-lane
  // groups serviced together read 8 consecutive rows of 32 bytes, which land
  // on disjoint banks when the stride is an odd multiple of 8 dwords mod 64.
  static constexpr int V_ROW = D + 16;                          // 72 / 40 dwords
  static constexpr int LV_ROW = RC == 1 ? 16 : (RC == 2 ? 48 : 80);  // 8 / 24 / 40 dwords
  static constexpr int LPR = D / 8;           // lanes per V row (16 bytes each)
  static constexpr int RPL = 64 / LPR;        // V rows per wave load
  static constexpr int NVL = 16 / RPL;        // V loads per sub-block
  static constexpr int PS = 4 + D + R;        // floats per split partial
  static constexpr int PF = VD ? 1 : dec_prefetch(R);  // sub-blocks loaded ahead
  static constexpr int NST = PF + 1;          // staged sub-blocks (a ring)
  static constexpr int TPR = NST / gcd_c(NST, NSB);  // tiles per whole number of turns of the ring
  // Direct-to-LDS V staging: a stage is the 16 V rows at the padded row
  // stride V_ROW, written by NVD 1 KB loads (lane i of load k lands at byte
  // 1024 k + 16 i; lanes that fall in a row's padding or past the last row
  // load nothing).  VST: bf16 per stage buffer.
  static constexpr int NVD = (16 * V_ROW * 2 + 1023) / 1024;
  static constexpr int VST = NVD * 512;
};

// Transposing LDS read: lane j of each 16-lane group points at 4 consecutive
// bf16; lane i receives element i%4 of lanes i/4, i/4+4, i/4+8, i/4+12.
__device__ __forceinline__ i16x4 lds_read_tr(const uint16_t* p) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((v4s __attribute__((address_space(3)))*)(p));
  return __builtin_bit_cast(i16x4, v);
}

template <int D, int R>
struct Stage {
  u32x4 kb[D / 32];                         // K_base chunks of token l%16
  typename Ex<R>::Frag lk[Ex<R>::NC];       // L_k row fragments of token l%16 (expansion B operand)
  u32x4 v[Dec<D, R>::NVL];                  // V rows, natural layout
  u32x2 lv[RCH(R)];                         // L_v row fragment of token l%16
};

// Buffer resource over `bytes` bytes from `base` (raw, stride 0): loads at
// offsets at or past the end return zeros.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const uint16_t* base, int32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), (short)0, bytes, 0x00020000);
}

// Per-lane byte offsets of one 16-token sub-block's data (constant over the
// kernel): the sub-block itself is addressed by resources built per
// sub-block, whose range check zero-fills tokens at or past the split end.
// The loads are branch-free, so the compiler can keep the next sub-block's
// loads in flight while the current one is consumed.
template <int D, int R>
struct StageOffsets {
  int32_t kb[D / 32], lk[Ex<R>::NC], lr[RCH(R)], v[Dec<D, R>::NVL], vd[Dec<D, R>::NVD];
};

template <int D, int R, bool VD>
__device__ __forceinline__ StageOffsets<D, R> stage_offsets(int64_t row, int lane) {
  using C = Dec<D, R>;
  StageOffsets<D, R> o;
  const int c16 = lane & 15, q = lane >> 4;
#pragma unroll
  for (int kk = 0; kk < C::NCH; ++kk) o.kb[kk] = c16 * (int32_t)(row * 2) + chunk_dim<D>(kk, q) * 2;
#pragma unroll
  for (int rc = 0; rc < C::RC; ++rc) {
    const int r0 = rc * 16 + q * 4;
    o.lr[rc] = r0 < R ? c16 * R * 2 + r0 * 2 : INT32_MIN;  // ranks past r read as zeros
  }
#pragma unroll
  for (int c = 0; c < Ex<R>::NC; ++c) {
    const int r0 = Ex<R>::rank0(c, q);
    o.lk[c] = r0 < R ? c16 * R * 2 + r0 * 2 : INT32_MIN;
  }
  const int vrow = lane / C::LPR, vdim = (lane % C::LPR) * 8;
  if constexpr (VD) {
#pragma unroll
    for (int k = 0; k < C::NVD; ++k) {
      const int byte = 1024 * k + 16 * lane, t = byte / (2 * C::V_ROW), in_row = byte % (2 * C::V_ROW);
      o.vd[k] = (t < 16 && in_row < 2 * D) ? t * (int32_t)(row * 2) + in_row : INT32_MIN;
    }
  } else {
#pragma unroll
    for (int iv = 0; iv < C::NVL; ++iv) o.v[iv] = (vrow + C::RPL * iv) * (int32_t)(row * 2) + vdim * 2;
  }
  return o;
}

// One expansion fragment of an LR row through a buffer resource.
template <int R>
__device__ __forceinline__ typename Ex<R>::Frag lr_frag_load(__amdgpu_buffer_rsrc_t r, int32_t off) {
  if constexpr (Ex<R>::WIDE)
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
  else
    return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}

// VD: V goes straight to the stage buffer `vdst` in LDS (its rows at stride
// V_ROW), issued after the stage's other loads.
template <int D, int R, bool VD>
__device__ __forceinline__ void stage_load(Stage<D, R>& s, const StageOffsets<D, R>& o, const uint16_t* Kb,
                                           const uint16_t* Vb, const uint16_t* Lk, const uint16_t* Lv,
                                           int64_t kv_row, int64_t lr_row, int64_t row, int64_t t0,
                                           int64_t t_end, uint16_t* vdst) {
  using C = Dec<D, R>;
  // Valid tokens of the sub-block (none past the end: every load reads zeros).
  const int64_t n = t_end - t0 < 0 ? 0 : (t_end - t0 < 16 ? t_end - t0 : 16);
  const int32_t kv_bytes = n > 0 ? (int32_t)((n - 1) * row * 2 + D * 2) : 0;
  // kv_row / lr_row: cache rows of token t0 (t0 itself unless paged).
  const auto rk = make_rsrc(Kb + kv_row * row, kv_bytes);
  const auto rv = make_rsrc(Vb + kv_row * row, kv_bytes);
  // Absent LR caches get empty resources (loads read zeros, touch nothing).
  const auto rlk = make_rsrc(Lk != nullptr ? Lk + lr_row * R : Kb, Lk != nullptr ? (int32_t)(n * R * 2) : 0);
  const auto rlv = make_rsrc(Lv != nullptr ? Lv + lr_row * R : Kb, Lv != nullptr ? (int32_t)(n * R * 2) : 0);
#pragma unroll
  for (int kk = 0; kk < C::NCH; ++kk)
    s.kb[kk] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, o.kb[kk], 0, 0));
#pragma unroll
  for (int c = 0; c < Ex<R>::NC; ++c) s.lk[c] = lr_frag_load<R>(rlk, o.lk[c]);
#pragma unroll
  for (int rc = 0; rc < C::RC; ++rc)
    s.lv[rc] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rlv, o.lr[rc], 0, 0));
  if constexpr (VD) {
#pragma unroll
    for (int k = 0; k < C::NVD; ++k)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (__attribute__((address_space(3))) void*)(vdst + 512 * k), 16,
                                               o.vd[k], 0, 0, 0);
  } else {
#pragma unroll
    for (int iv = 0; iv < C::NVL; ++iv)
      s.v[iv] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, o.v[iv], 0, 0));
  }
}

// s_waitcnt with vmcnt(n) and no wait on the other counters.
constexpr int vmcnt_imm(int n) { return (n & 0xF) | ((n >> 4) << 14) | 0x0F70; }
// Vector memory instructions one VD stage issues (K_base chunks, L_k
// fragments, L_v fragments, then the direct V loads).
template <int D, int R>
constexpr int kStageLoads = D / 32 + Ex<R>::NC + RCH(R) + Dec<D, R>::NVD;

// PAGED: the caches are pools reached through block tables (a separate
// instantiation, so the contiguous kernel carries none of the walk's state).
template <int D, int R, bool PAGED>
__global__ void __launch_bounds__(dec_nw(D, R, PAGED) * 64, dec_nw(D, R, PAGED) / 4)
lrsa_decode_kernel(const AttnArgs a) {
  constexpr bool VD = dec_vdma(D, R, PAGED);
  using C = Dec<D, R, VD>;
  constexpr int NW = C::NW, NT = C::NT;
  __shared__ float2 cs_lds[2][TK * C::CS_ROW];
  __shared__ float2 base_lds[2][C::HALF];
  // Per wave: the V tile written from registers, or (VD) the two V stage
  // buffers the direct loads fill, as separate arrays so that the compiler
  // can tell the LDS reads of one from the direct loads into the other.
  static_assert(!VD || C::NST == 2, "two V stage buffers");
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[NW][VD ? C::VST : 16 * C::V_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds1[VD ? NW : 1][VD ? C::VST : 8];
  __shared__ __attribute__((aligned(16))) uint16_t lv_lds[NW][16 * C::LV_ROW];

  // The wave index is made visibly wave-uniform, so that everything derived
  // from it (the KV head and its buffer resources) lives in scalar registers.
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int split = blockIdx.x, b = blockIdx.z;
  const int g = blockIdx.y * NW + w;
  const bool active = g < a.n_kv;
  const int G = a.group;
  const int q = lane >> 4, c16 = lane & 15;
  const bool has_lk = a.Lk != nullptr, has_lv = a.Lv != nullptr;
  // The up-projection rows go out first: their latency hides behind the rest
  // of the set-up (a split of a small batch covers only a few tiles).
  BtStage<D, R> bts;
  bts.issue(has_lk ? a.Bk + (int64_t)b * a.b_stride + (int64_t)g * D : nullptr, (int64_t)a.n_kv * D,
            has_lk && active, lane);

  // Keys this request may see: t < kv_len (clamped into the buffer) and
  // t <= position of its query token.
  int64_t kvl = a.kv_len[b];
  kvl = kvl < 0 ? 0 : (kvl > a.s_cap ? a.s_cap : kvl);
  const int64_t pos = a.positions[(int64_t)b * a.n_tok];
  int64_t vis = pos + 1 < kvl ? pos + 1 : kvl;
  if (vis < 0) vis = 0;
  const int64_t t_begin = (int64_t)split * a.split_tiles * TK;
  int64_t t_end = t_begin + (int64_t)a.split_tiles * TK;
  if (t_end > vis) t_end = vis;
  const int n_tiles = t_end > t_begin ? (int)((t_end - t_begin + TK - 1) / TK) : 0;

  // RoPE table entries this thread builds every tile, by angle addition from
  // the exact base angle of the tile and exact per-entry offset angles.
  float cdl[C::EPT], sdl[C::EPT];
  int ej[C::EPT], eidx[C::EPT];
#pragma unroll
  for (int k = 0; k < C::EPT; ++k) {
    const int e = tid + NT * k, tok = e / C::HALF;
    ej[k] = e - tok * C::HALF;
    eidx[k] = tok * C::CS_ROW + ej[k];
    cdl[k] = 1.f;
    sdl[k] = 0.f;
    if (has_lk) rope_cs(tok, a.w2pi[ej[k]], cdl[k], sdl[k]);
  }
  // This thread's frequency for the per-tile base angles, read once.
  const double w2pi_t = a.w2pi[tid < C::HALF ? tid : 0];
  if (has_lk && tid < C::HALF && n_tiles > 0) {
    float c, s;
    rope_cs((int)t_begin, a.w2pi[tid], c, s);
    base_lds[0][tid] = make_float2(c, s);
  }
  // L_v tile columns past the rank stay zero (rank 8 pads to 16).
  for (int i = lane; i < 16 * C::LV_ROW; i += 64) lv_lds[w][i] = 0;

  const int64_t row = (int64_t)a.n_kv * D;  // elements between tokens
  // This request's caches (or pools, paged through its rows of the block
  // tables).
  const uint16_t* Kb = a.Kb + (int64_t)b * a.kv_stride + (int64_t)g * D;
  const uint16_t* Vb = a.Vb + (int64_t)b * a.kv_stride + (int64_t)g * D;
  const uint16_t* Lk = has_lk ? a.Lk + (int64_t)b * a.l_stride : nullptr;
  const uint16_t* Lv = has_lv ? a.Lv + (int64_t)b * a.l_stride : nullptr;
  const int64_t t_end_w = active ? t_end : t_begin;  // inactive waves load nothing

  // Q^T of the group as the B operand (cols = q heads, zero past G).
  bf16x8 qf[C::NCH];
  {
    const bool ok = active && c16 < G;
    const uint16_t* qp = a.Q + ((int64_t)b * a.n_tok * a.n_q + (int64_t)g * G + c16) * D;
#pragma unroll
    for (int kk = 0; kk < C::NCH; ++kk) qf[kk] = as_bf16x8(ld16(qp + chunk_dim<D>(kk, q), ok));
  }
  typename Ex<R>::Frag bkf[C::NBLK][Ex<R>::NC];
  bts.finish(bkf, v_lds[w], lane);
  if constexpr (VD) {
    // The stage buffers start as zeros (finite rows for tokens past the end,
    // whatever the direct loads do at out-of-range offsets), written before
    // the first direct load is issued.
    for (int i = lane; i < C::VST / 8; i += 64) {
      *reinterpret_cast<u32x4*>(v_lds[w] + 8 * i) = u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(v_lds1[VD ? w : 0] + 8 * i) = u32x4{0u, 0u, 0u, 0u};
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  }

  float m_run = -INFINITY, l_part = 0.f;
  f32x4 acc[C::NBLK];   // O^T: dims blk*16 + 4q + i, head l%16
  f32x4 accl[C::RC];    // (P L_v)^T: rank rc*16 + 4q + i, head l%16
#pragma unroll
  for (int blk = 0; blk < C::NBLK; ++blk) acc[blk] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int rc = 0; rc < C::RC; ++rc) accl[rc] = f32x4{0.f, 0.f, 0.f, 0.f};

  uint16_t* vl = v_lds[w];
  uint16_t* lvl = lv_lds[w];
  const int vrow = lane / C::LPR, vdim = (lane % C::LPR) * 8;
  // Transposing-read addresses: lane j of group l/16 reads row
  // 4*(l/16) + (j/4), columns 4*(j%4) .. +3 of a 16-column block.
  const int tr_row = 4 * q + (c16 >> 2), tr_col = 4 * (c16 & 3);

  const StageOffsets<D, R> so = stage_offsets<D, R, VD>(row, lane);
  Stage<D, R> st[C::NST];
  // Sub-blocks are loaded in token order, so paged caches are walked with them.
  PageWalk walk;
  if constexpr (PAGED)
    walk.start(a.kv_tbl + (int64_t)b * a.max_blk, a.lr_tbl + (int64_t)b * a.max_blk, a.max_blk, a.blk, a.kv_nblk,
               a.lr_nblk, t_begin, t_end_w);
  // Stage `slot` of the ring (VD: also its V buffer in LDS).
  auto load = [&](Stage<D, R>& s, int64_t t, int slot) {
    int64_t kr = t, lr = t;
    if constexpr (PAGED) walk.next(16, t_end_w, kr, lr);
    stage_load<D, R, VD>(s, so, Kb, Vb, Lk, Lv, kr, lr, row, t, t_end_w, slot == 0 ? vl : v_lds1[VD ? w : 0]);
  };
#pragma unroll
  for (int p = 0; p < C::PF; ++p) load(st[p], t_begin + 16 * p, p);

  __syncthreads();  // base angles of the first tile, zeroed L_v tiles

  // RoPE table of tile k (from its base angles in base_lds[k & 1]) into
  // cs_lds[k & 1], and the base angles of tile k + 1 into base_lds[(k + 1) & 1].
  // Tile 0's here; each later one while the tile before it runs, beside that
  // tile's first loads, so that the barrier at the head of a tile has no
  // table work in front of it.
  auto build_table = [&](int k) {
    float2* csk = cs_lds[k & 1];
    const float2* base = base_lds[k & 1];
#pragma unroll
    for (int e = 0; e < C::EPT; ++e) {
      const float2 bc = base[ej[e]];
      csk[eidx[e]] = make_float2(bc.x * cdl[e] - bc.y * sdl[e], bc.y * cdl[e] + bc.x * sdl[e]);
    }
    if (tid < C::HALF && k + 1 < n_tiles) {
      float c, sn;
      rope_cs((int)(t_begin + (int64_t)(k + 1) * TK), w2pi_t, c, sn);
      base_lds[(k + 1) & 1][tid] = make_float2(c, sn);
    }
  };
  if (has_lk && n_tiles > 0) build_table(0);

  // The tile loop is unrolled by the tiles of one turn of the stage ring, so
  // that every stage index is a constant.  Inside it every path issues the
  // same loads (inactive waves and sub-blocks past the split end load zeros
  // and compute on them), and the only early exit leaves the loop for good:
  // the compiler's load counting then sees the same loads in flight on every
  // path and waits for no stage before it is needed.
  for (int tile0 = 0; tile0 < n_tiles; tile0 += C::TPR)
#pragma unroll
  for (int tt = 0; tt < C::TPR; ++tt) {
    const int tile = tile0 + tt;
    if (tile >= n_tiles) goto tiles_done;  // uniform over the workgroup
    const int64_t t0 = t_begin + (int64_t)tile * TK;
    float2* cs = cs_lds[tile & 1];
    __syncthreads();  // this tile's table and the next tile's base angles are
                      // ready, and every wave is done with the previous tile
                      // (whose table buffer the next table goes into).

#pragma unroll
    for (int sb = 0; sb < NSB; ++sb) {
      const int cslot = (tt * NSB + sb) % C::NST, nslot = (tt * NSB + sb + C::PF) % C::NST;
      Stage<D, R>& cur = st[cslot];
      Stage<D, R>& nxt = st[nslot];
      // A sub-block past the split end (only in its last tile) holds zeros
      // and no visible key: all its weights are exactly 0 and the running
      // maximum does not move, so it changes nothing.
      const int64_t ts = t0 + sb * 16;
      // Issue the loads of the sub-block PF ahead before consuming this one
      // (past the split end they read zeros and touch no memory).
      load(nxt, ts + 16 * C::PF, nslot);
      // Keep the loads ahead of this sub-block's work: the scheduler would
      // otherwise sink them to shorten their registers' live ranges, and the
      // wait for this stage would then also wait for the next one.
      __builtin_amdgcn_sched_barrier(0);
      // The next tile's table, while this sub-block's data is still landing.
      if (sb == 0 && has_lk && tile + 1 < n_tiles) build_table(tile + 1);

      // ---- V and L_v rows into the wave's LDS tile ------------------------
      if constexpr (!VD) {
#pragma unroll
        for (int iv = 0; iv < C::NVL; ++iv)
          *reinterpret_cast<u32x4*>(vl + (vrow + C::RPL * iv) * C::V_ROW + vdim) = cur.v[iv];
      }
      if (has_lv) {
#pragma unroll
        for (int rc = 0; rc < C::RC; ++rc)
          if (rc * 16 + q * 4 < R) *reinterpret_cast<u32x2*>(lvl + c16 * C::LV_ROW + rc * 16 + q * 4) = cur.lv[rc];
      }

      // ---- scores S^T = K_base Q^T + bf16(RoPE(E)) Q^T --------------------
      f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < C::NCH; ++kk) sc = mfma16x16x32(as_bf16x8(cur.kb[kk]), qf[kk], sc);
      if (has_lk) {
        const float2* csr = cs + (sb * 16 + c16) * C::CS_ROW + q * C::QPG;
        u32x4 ek[C::NCH];
#pragma unroll
        for (int blk = 0; blk < C::NB; ++blk) {
          f32x4 elo = {0.f, 0.f, 0.f, 0.f}, ehi = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < Ex<R>::NC; ++c) {
            elo = Ex<R>::mma(bkf[blk][c], cur.lk[c], elo);
            ehi = Ex<R>::mma(bkf[blk + C::NB][c], cur.lk[c], ehi);
          }
          float rlo[4], rhi[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float2 r = csr[blk * 4 + i];
            rlo[i] = elo[i] * r.x - ehi[i] * r.y;
            rhi[i] = ehi[i] * r.x + elo[i] * r.y;
          }
          const int klo = blk >> 1, khi = (blk + C::NB) >> 1, w0 = (blk & 1) * 2;
          ek[klo][w0] = pack_bf16(rlo[0], rlo[1]);
          ek[klo][w0 + 1] = pack_bf16(rlo[2], rlo[3]);
          ek[khi][w0] = pack_bf16(rhi[0], rhi[1]);
          ek[khi][w0 + 1] = pack_bf16(rhi[2], rhi[3]);
        }
#pragma unroll
        for (int kk = 0; kk < C::NCH; ++kk) sc = mfma16x16x32(as_bf16x8(ek[kk]), qf[kk], sc);
      }

      // ---- online softmax: lane l%16 is a head, 4 tokens per lane ---------
      float s2[4];
      float mx = -INFINITY;
      const int64_t left = t_end - ts;  // visible tokens from ts on
      const int n_vis = left < 0 ? 0 : (left < 16 ? (int)left : 16);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s2[i] = (q * 4 + i < n_vis) ? sc[i] * a.scale_log2 : -INFINITY;
        mx = fmaxf(mx, s2[i]);
      }
      mx = max_xor32(max_xor16(mx));
      // Lazy rescale: a head's reference maximum m_run only moves when a
      // score exceeds it by more than 2^8 (P stays below 256), so the
      // accumulators are rescaled a few times per split, not per sub-block.
      if (__ballot(mx > m_run + kRescaleLog2)) {
        const float mn = fmaxf(m_run, mx);
        const float alpha = fast_exp2(m_run - (mn == -INFINITY ? 0.f : mn));
#pragma unroll
        for (int blk = 0; blk < C::NBLK; ++blk) acc[blk] *= alpha;
#pragma unroll
        for (int rc = 0; rc < C::RC; ++rc) accl[rc] *= alpha;
        l_part *= alpha;
        m_run = mn;
      }
      const float ms = (m_run == -INFINITY) ? 0.f : m_run;
      float p[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) p[i] = fast_exp2(s2[i] - ms);
      l_part += (p[0] + p[1]) + (p[2] + p[3]);
      u32x2 pw;
      pw[0] = pack_bf16(p[0], p[1]);
      pw[1] = pack_bf16(p[2], p[3]);
      const i16x4 pb = as_i16x4(pw);
      __builtin_amdgcn_wave_barrier();

      // ---- O^T += V^T P^T, (P L_v)^T += L_v^T P^T -----------------------
      const uint16_t* vcur = vl;
      if constexpr (VD) {
        // This stage's direct V loads have landed once at most the loads of
        // the next stage, issued after them, are still in flight (the
        // counter drains in issue order; the sched barrier keeps the LDS
        // reads below the wait).
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(kStageLoads<D, R>));
        __builtin_amdgcn_sched_barrier(0);
        vcur = cslot == 0 ? vl : v_lds1[VD ? w : 0];
      }
#pragma unroll
      for (int blk = 0; blk < C::NBLK; ++blk)
        acc[blk] = mfma16x16x16(lds_read_tr(vcur + tr_row * C::V_ROW + blk * 16 + tr_col), pb, acc[blk]);
      if (has_lv) {
#pragma unroll
        for (int rc = 0; rc < C::RC; ++rc)
          accl[rc] = mfma16x16x16(lds_read_tr(lvl + tr_row * C::LV_ROW + rc * 16 + tr_col), pb, accl[rc]);
      }
      __builtin_amdgcn_wave_barrier();
    }
  }

tiles_done:
  // Direct loads past the split end may still be in flight: let them land
  // before the wave (and with the last wave, the workgroup's LDS) retires.
  if constexpr (VD) __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  if (!active) return;
  // One partial per (request, q head, split): lane l%16 is the head; lanes
  // l, l^16, l^32, l^48 share it and hold different dims of O^T.
  l_part += shfl_xor(l_part, 16);
  l_part += shfl_xor(l_part, 32);
  if (c16 >= G) return;
  const int64_t hstride = (int64_t)a.n_splits * C::PS;
  float* wsb = a.ws + ((int64_t)b * a.n_q + (int64_t)g * G + c16) * hstride + (int64_t)split * C::PS;
  if (q == 0) {
    wsb[0] = m_run;
    wsb[1] = l_part;
  }
#pragma unroll
  for (int blk = 0; blk < C::NBLK; ++blk)
    *reinterpret_cast<f32x4*>(wsb + 4 + blk * 16 + q * 4) = acc[blk];
  if (has_lv) {
#pragma unroll
    for (int rc = 0; rc < C::RC; ++rc)
      if (rc * 16 + q * 4 < R) *reinterpret_cast<f32x4*>(wsb + 4 + D + rc * 16 + q * 4) = accl[rc];
  }
}

// Merge the split partials of one (request, query token, q head):
// log-sum-exp weights, then the deferred up-projection
// O += (sum_s w_s P_s L_v) B_v, then 1/l.  Decode has one query token per
// request; a split prefill has n_tok.
// A row's partials are n_splits x (d + r) fp32 beside their maxima and sums.
// Thread t owns float4 column t % NV of those d + r accumulators for the
// splits congruent to t / NV modulo the number of such groups, so a
// workgroup keeps one independent 16-byte load per thread and split group
// in flight; the groups' sums then meet in LDS.  Rows with many splits
// (small decode batches) take 16-wave workgroups, rows with few 4-wave ones.
template <int D, int R, int MW>
__global__ void __launch_bounds__(64 * MW)
lrsa_merge_kernel(const AttnArgs a) {
  constexpr int PS = 4 + D + R, NT = 64 * MW;
  constexpr int NV = (D + R) / 4;  // float4 columns of the accumulators
  constexpr int NG = NT / NV;      // split groups
  __shared__ float red[NG][D + R];
  __shared__ float red_w[MW][2];
  __shared__ float fin[D + R];
  const int h = blockIdx.x, bi = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int b = bi / a.n_tok;  // bi = request * n_tok + query token
  const int g = h / a.group;
  const bool has_lv = a.Lv != nullptr;
  const int ns = a.n_splits;
  const int64_t orow = (int64_t)bi * a.n_q + h;  // (request, token, head) row of O
  const float* base = a.ws + orow * (int64_t)ns * PS;

  // Global maximum over the splits.
  float M = -INFINITY;
  for (int s = tid; s < ns; s += NT) M = fmaxf(M, base[(int64_t)s * PS]);
#pragma unroll
  for (int x = 1; x < 64; x <<= 1) M = fmaxf(M, shfl_xor(M, x));
  if (lane == 0) red_w[w][0] = M;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MW; ++i) M = fmaxf(M, red_w[i][0]);
  const float Ms = (M == -INFINITY) ? 0.f : M;

  // Row sum L = sum_s w_s l_s.
  float L = 0.f;
  for (int s = tid; s < ns; s += NT) {
    const float* p = base + (int64_t)s * PS;
    L += fast_exp2(p[0] - Ms) * p[1];
  }
#pragma unroll
  for (int x = 1; x < 64; x <<= 1) L += shfl_xor(L, x);

  // Weighted accumulators (d of P V, r of P L_v), one float4 column per thread.
  const int grp = tid / NV, v = tid - grp * NV;
  const int nv_used = has_lv ? NV : D / 4;
  if (grp < NG && v < nv_used) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int s = grp; s < ns; s += NG) {
      const float* p = base + (int64_t)s * PS;
      const float wgt = fast_exp2(p[0] - Ms);
      const f32x4 x = *reinterpret_cast<const f32x4*>(p + 4 + 4 * v);
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] += wgt * x[c];
    }
    *reinterpret_cast<f32x4*>(&red[grp][4 * v]) = acc;
  }
  if (lane == 0) red_w[w][1] = L;
  __syncthreads();
  for (int c = tid; c < D + R; c += NT) {
    float t = 0.f;
    if (c < D || has_lv)
      for (int i = 0; i < NG; ++i) t += red[i][c];
    fin[c] = t;
  }
  L = 0.f;
#pragma unroll
  for (int i = 0; i < MW; ++i) L += red_w[i][1];
  __syncthreads();

  // O = (acc + (sum_s w_s P_s L_v) B_v) / L, one head dim per thread.
  const float inv = L > 0.f ? 1.f / L : 0.f;
  uint16_t* o = a.O + orow * D;
  for (int dim = tid; dim < D; dim += NT) {
    float sum = fin[dim];
    if (has_lv) {
      // B_v [r, n_kv*d]: rank j of this head dim, coalesced over the threads.
      const int64_t ldb = (int64_t)a.n_kv * D;
      const uint16_t* bv = a.Bv + (int64_t)b * a.b_stride + (int64_t)g * D + dim;
#pragma unroll 8
      for (int j = 0; j < R; ++j) sum += fin[D + j] * __uint_as_float((uint32_t)bv[j * ldb] << 16);
    }
    const uint32_t pk = pack_bf16(sum * inv, 0.f);
    o[dim] = (uint16_t)(pk & 0xffffu);
  }
  if (a.lse != nullptr && tid == 0)
    a.lse[orow] = L > 0.f ? (M + __log2f(L)) * kLn2 : -INFINITY;
}

// ---------------------------------------------------------------------------
// Decode over one base cache shared by every request (kv_req_stride == 0):
// several agents' queries over the same trajectory, each with its own LR
// plane, up-projections, query and position.  One workgroup per (split, KV
// head, group of NW requests); wave w serves request group*NW + w.  Each
// 64-token step of the head's K_base/V_base rows is read from memory once,
// staged in LDS, and used by every wave: base bytes are paid once for all
// agents, and only the agents' LR rows (a few per cent of the base bytes)
// are read per request.  One barrier per step; within a step each wave runs
// the per-request kernel's 16-token sub-block work four times.  The partials
// go to the same workspace and the same merge.
template <int D, int R>
__global__ void __launch_bounds__(dec_waves(R) * 64, dec_waves(R) / 4)
lrsa_decode_shared_kernel(const AttnArgs a) {
  using C = Dec<D, R>;
  constexpr int NW = C::NW, NT = C::NT;
  constexpr int SB = 16;                    // tokens per sub-block
  constexpr int NSS = 4;                    // sub-blocks per step
  constexpr int STEP = SB * NSS;            // tokens per step (one barrier)
  constexpr int K_ROW = D + 8;              // conflict-free 16-byte row reads
  constexpr int EPS = SB * C::HALF / NT;    // RoPE table entries per thread per sub-block
  constexpr int CPR = D / 8;                // 16-byte chunks per base row
  constexpr int NBC = 2 * STEP * CPR;       // base chunks (K rows, then V rows) per step
  constexpr int NCK = (NBC + NT - 1) / NT;  // base chunks per thread per step
  static_assert(EPS >= 1 && SB * C::HALF % NT == 0 && NSS * C::HALF <= NT, "step sizes");
  __shared__ float2 cs_lds[2][NSS][SB * C::CS_ROW];
  __shared__ float2 base_lds[2][NSS][C::HALF];
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][STEP * K_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][STEP * C::V_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t lv_lds[NW][16 * C::LV_ROW];

  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int split = blockIdx.x, g = blockIdx.y;
  const int b = blockIdx.z * NW + w;
  const bool active = b < a.batch;
  const int G = a.group;
  const int q = lane >> 4, c16 = lane & 15;
  const bool has_lk = a.Lk != nullptr, has_lv = a.Lv != nullptr;
  const int64_t t_begin = (int64_t)split * a.split_tiles * TK;
  const int64_t t_cap = t_begin + (int64_t)a.split_tiles * TK;
  // The up-projection rows go out first (see the per-request kernel).
  BtStage<D, R> bts;
  bts.issue(has_lk && active ? a.Bk + (int64_t)b * a.b_stride + (int64_t)g * D : nullptr, (int64_t)a.n_kv * D,
            has_lk && active, lane);

  // Keys request r may see: t < min(kv_len, position + 1), within the split.
  auto req_end = [&](int r) -> int64_t {
    int64_t kvl = a.kv_len[r];
    kvl = kvl < 0 ? 0 : (kvl > a.s_cap ? a.s_cap : kvl);
    const int64_t pos = a.positions[(int64_t)r * a.n_tok];
    int64_t vis = pos + 1 < kvl ? pos + 1 : kvl;
    if (vis < t_begin) vis = t_begin;
    return vis < t_cap ? vis : t_cap;
  };
  const int64_t t_end = active ? req_end(b) : t_begin;
  // The workgroup walks up to the furthest end among its requests.
  int64_t t_end_wg = t_begin;
  for (int r = blockIdx.z * NW; r < blockIdx.z * NW + NW && r < a.batch; ++r) {
    const int64_t e = req_end(r);
    t_end_wg = e > t_end_wg ? e : t_end_wg;
  }
  const int n_steps = __builtin_amdgcn_readfirstlane((int)((t_end_wg - t_begin + STEP - 1) / STEP));

  // RoPE table entries of this thread within a sub-block (token, frequency j),
  // and the sub-block base angle it computes (sub-block tid / HALF, j).
  float cdl[EPS], sdl[EPS];
  int ej[EPS], eidx[EPS];
#pragma unroll
  for (int k = 0; k < EPS; ++k) {
    const int e = tid + NT * k, tok = e / C::HALF;
    ej[k] = e - tok * C::HALF;
    eidx[k] = tok * C::CS_ROW + ej[k];
    cdl[k] = 1.f;
    sdl[k] = 0.f;
    if (has_lk) rope_cs(tok, a.w2pi[ej[k]], cdl[k], sdl[k]);
  }
  const int bsb = tid / C::HALF, bj = tid % C::HALF;  // base angle this thread computes
  const bool base_thread = has_lk && tid < NSS * C::HALF;
  const double w2pi_t = a.w2pi[bj];
  auto base_angles = [&](int64_t t0s, int buf) {
    if (base_thread) {
      float c, s;
      rope_cs((int)(t0s + bsb * SB), w2pi_t, c, s);
      base_lds[buf][bsb][bj] = make_float2(c, s);
    }
  };
  if (n_steps > 0) base_angles(t_begin, 0);
  for (int i = lane; i < 16 * C::LV_ROW; i += 64) lv_lds[w][i] = 0;

  const int64_t row = (int64_t)a.n_kv * D;
  const uint16_t* Kb = a.Kb + (int64_t)g * D;
  const uint16_t* Vb = a.Vb + (int64_t)g * D;
  const uint16_t* Lk = has_lk && active ? a.Lk + (int64_t)b * a.l_stride : nullptr;
  const uint16_t* Lv = has_lv && active ? a.Lv + (int64_t)b * a.l_stride : nullptr;

  // Base chunks of a step: chunk c < STEP*CPR is K row c / CPR, else V.
  int32_t boff[NCK];
#pragma unroll
  for (int k = 0; k < NCK; ++k) {
    const int c = (tid + NT * k) % (STEP * CPR);
    boff[k] = tid + NT * k < NBC ? (c / CPR) * (int32_t)(row * 2) + (c % CPR) * 16 : INT32_MIN;
  }
  auto base_load = [&](u32x4 (&r)[NCK], int64_t t0) {
    const int64_t n = t_end_wg - t0 < 0 ? 0 : (t_end_wg - t0 < STEP ? t_end_wg - t0 : STEP);
    const int32_t bytes = n > 0 ? (int32_t)((n - 1) * row * 2 + D * 2) : 0;
    const auto rk = make_rsrc(Kb + t0 * row, bytes), rv = make_rsrc(Vb + t0 * row, bytes);
#pragma unroll
    for (int k = 0; k < NCK; ++k) {
      const bool isk = (tid + NT * k) < STEP * CPR;
      r[k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(isk ? rk : rv, boff[k], 0, 0));
    }
  };
  auto base_store = [&](const u32x4 (&r)[NCK], int buf) {
#pragma unroll
    for (int k = 0; k < NCK; ++k) {
      const int c = tid + NT * k, cc = c % (STEP * CPR), tok = cc / CPR, col = (cc % CPR) * 8;
      if (c < STEP * CPR)
        *reinterpret_cast<u32x4*>(k_lds[buf] + tok * K_ROW + col) = r[k];
      else if (c < NBC)
        *reinterpret_cast<u32x4*>(v_lds[buf] + tok * C::V_ROW + col) = r[k];
    }
  };
  // This wave's LR rows of a sub-block (rank chunks of token l%16), zero past
  // its end.
  struct LrStage {
    typename Ex<R>::Frag lk[Ex<R>::NC];
    u32x2 lv[C::RC];
  };
  int32_t lroff[C::RC], lkoff[Ex<R>::NC];
#pragma unroll
  for (int rc = 0; rc < C::RC; ++rc) {
    const int r0 = rc * 16 + q * 4;
    lroff[rc] = r0 < R ? c16 * R * 2 + r0 * 2 : INT32_MIN;
  }
#pragma unroll
  for (int c = 0; c < Ex<R>::NC; ++c) {
    const int r0 = Ex<R>::rank0(c, q);
    lkoff[c] = r0 < R ? c16 * R * 2 + r0 * 2 : INT32_MIN;
  }
  auto lr_load = [&](LrStage& s, int64_t t0) {
    const int64_t n = t_end - t0 < 0 ? 0 : (t_end - t0 < SB ? t_end - t0 : SB);
    const auto rlk = make_rsrc(Lk != nullptr ? Lk + t0 * R : Kb, Lk != nullptr ? (int32_t)(n * R * 2) : 0);
    const auto rlv = make_rsrc(Lv != nullptr ? Lv + t0 * R : Kb, Lv != nullptr ? (int32_t)(n * R * 2) : 0);
#pragma unroll
    for (int c = 0; c < Ex<R>::NC; ++c) s.lk[c] = lr_frag_load<R>(rlk, lkoff[c]);
#pragma unroll
    for (int rc = 0; rc < C::RC; ++rc)
      s.lv[rc] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rlv, lroff[rc], 0, 0));
  };

  bf16x8 qf[C::NCH];
  {
    const bool ok = active && c16 < G;
    const uint16_t* qp = a.Q + ((int64_t)(active ? b : 0) * a.n_tok * a.n_q + (int64_t)g * G + c16) * D;
#pragma unroll
    for (int kk = 0; kk < C::NCH; ++kk) qf[kk] = as_bf16x8(ld16(qp + chunk_dim<D>(kk, q), ok));
  }
  typename Ex<R>::Frag bkf[C::NBLK][Ex<R>::NC];
  // Staged through this wave's share of the (not yet used) V tiles.
  bts.finish(bkf, &v_lds[0][0] + w * 16 * C::V_ROW, lane);

  float m_run = -INFINITY, l_part = 0.f;
  f32x4 acc[C::NBLK];
  f32x4 accl[C::RC];
#pragma unroll
  for (int blk = 0; blk < C::NBLK; ++blk) acc[blk] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int rc = 0; rc < C::RC; ++rc) accl[rc] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint16_t* lvl = lv_lds[w];
  const int tr_row = 4 * q + (c16 >> 2), tr_col = 4 * (c16 & 3);

  // The base rows of the next step are in flight during a step; the wave's
  // LR rows run two sub-blocks ahead in a ring of NSS (static indices).
  u32x4 breg[NCK];
  LrStage lr[NSS];
  base_load(breg, t_begin);
  lr_load(lr[0], t_begin);
  lr_load(lr[1], t_begin + SB);
  __syncthreads();  // base angles of the first step, zeroed L_v tiles

  for (int step = 0; step < n_steps; ++step) {
    const int buf = step & 1;
    const int64_t t0s = t_begin + (int64_t)step * STEP;
    // ---- stage this step (tables, base rows) and start the next one -------
    if (has_lk) {
#pragma unroll
      for (int sb = 0; sb < NSS; ++sb) {
        const float2* base = base_lds[buf][sb];
        float2* cs = cs_lds[buf][sb];
#pragma unroll
        for (int k = 0; k < EPS; ++k) {
          const float2 bc = base[ej[k]];
          cs[eidx[k]] = make_float2(bc.x * cdl[k] - bc.y * sdl[k], bc.y * cdl[k] + bc.x * sdl[k]);
        }
      }
      if (step + 1 < n_steps) base_angles(t0s + STEP, buf ^ 1);
    }
    base_store(breg, buf);
    base_load(breg, t0s + STEP);
    __syncthreads();  // step's tables and base rows visible; double buffers
                      // keep the previous step's intact for slower waves
    const uint16_t* kt = k_lds[buf];
    const uint16_t* vt = v_lds[buf];
#pragma unroll
    for (int sb = 0; sb < NSS; ++sb) {
      const int64_t ts = t0s + sb * SB;
      lr_load(lr[(sb + 2) % NSS], ts + 2 * SB);
      if (!active || ts >= t_end) continue;
      const LrStage& cur = lr[sb];
        if (has_lv) {
#pragma unroll
          for (int rc = 0; rc < C::RC; ++rc)
            if (rc * 16 + q * 4 < R) *reinterpret_cast<u32x2*>(lvl + c16 * C::LV_ROW + rc * 16 + q * 4) = cur.lv[rc];
        }
        // ---- scores S^T = K_base Q^T + bf16(RoPE(E)) Q^T --------------------
        f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < C::NCH; ++kk)
          sc = mfma16x16x32(as_bf16x8(*reinterpret_cast<const u32x4*>(kt + (sb * SB + c16) * K_ROW + chunk_dim<D>(kk, q))),
                            qf[kk], sc);
        if (has_lk) {
          const float2* csr = cs_lds[buf][sb] + c16 * C::CS_ROW + q * C::QPG;
          u32x4 ek[C::NCH];
#pragma unroll
          for (int blk = 0; blk < C::NB; ++blk) {
            f32x4 elo = {0.f, 0.f, 0.f, 0.f}, ehi = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < Ex<R>::NC; ++c) {
              elo = Ex<R>::mma(bkf[blk][c], cur.lk[c], elo);
              ehi = Ex<R>::mma(bkf[blk + C::NB][c], cur.lk[c], ehi);
            }
            float rlo[4], rhi[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float2 r = csr[blk * 4 + i];
              rlo[i] = elo[i] * r.x - ehi[i] * r.y;
              rhi[i] = ehi[i] * r.x + elo[i] * r.y;
            }
            const int klo = blk >> 1, khi = (blk + C::NB) >> 1, w0 = (blk & 1) * 2;
            ek[klo][w0] = pack_bf16(rlo[0], rlo[1]);
            ek[klo][w0 + 1] = pack_bf16(rlo[2], rlo[3]);
            ek[khi][w0] = pack_bf16(rhi[0], rhi[1]);
            ek[khi][w0 + 1] = pack_bf16(rhi[2], rhi[3]);
          }
#pragma unroll
          for (int kk = 0; kk < C::NCH; ++kk) sc = mfma16x16x32(as_bf16x8(ek[kk]), qf[kk], sc);
        }
        // ---- online softmax: lane l%16 is a head, 4 tokens per lane ---------
        float s2[4];
        float mx = -INFINITY;
        const int64_t left = t_end - ts;  // visible tokens from ts on
        const int n_vis = left < 0 ? 0 : (left < 16 ? (int)left : 16);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          s2[i] = (q * 4 + i < n_vis) ? sc[i] * a.scale_log2 : -INFINITY;
          mx = fmaxf(mx, s2[i]);
        }
        mx = max_xor32(max_xor16(mx));
        if (__ballot(mx > m_run + kRescaleLog2)) {  // lazy rescale, as above
          const float mn = fmaxf(m_run, mx);
          const float alpha = fast_exp2(m_run - (mn == -INFINITY ? 0.f : mn));
#pragma unroll
          for (int blk = 0; blk < C::NBLK; ++blk) acc[blk] *= alpha;
#pragma unroll
          for (int rc = 0; rc < C::RC; ++rc) accl[rc] *= alpha;
          l_part *= alpha;
          m_run = mn;
        }
        const float ms = (m_run == -INFINITY) ? 0.f : m_run;
        float p[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] = fast_exp2(s2[i] - ms);
        l_part += (p[0] + p[1]) + (p[2] + p[3]);
        u32x2 pw;
        pw[0] = pack_bf16(p[0], p[1]);
        pw[1] = pack_bf16(p[2], p[3]);
        const i16x4 pb = as_i16x4(pw);
        __builtin_amdgcn_wave_barrier();
        // ---- O^T += V^T P^T, (P L_v)^T += L_v^T P^T -----------------------
#pragma unroll
        for (int blk = 0; blk < C::NBLK; ++blk)
          acc[blk] = mfma16x16x16(lds_read_tr(vt + (sb * SB + tr_row) * C::V_ROW + blk * 16 + tr_col), pb, acc[blk]);
        if (has_lv) {
#pragma unroll
          for (int rc = 0; rc < C::RC; ++rc)
            accl[rc] = mfma16x16x16(lds_read_tr(lvl + tr_row * C::LV_ROW + rc * 16 + tr_col), pb, accl[rc]);
        }
        __builtin_amdgcn_wave_barrier();
    }
  }

  if (!active) return;
  l_part += shfl_xor(l_part, 16);
  l_part += shfl_xor(l_part, 32);
  if (c16 >= G) return;
  const int64_t hstride = (int64_t)a.n_splits * C::PS;
  float* wsb = a.ws + ((int64_t)b * a.n_q + (int64_t)g * G + c16) * hstride + (int64_t)split * C::PS;
  if (q == 0) {
    wsb[0] = m_run;
    wsb[1] = l_part;
  }
#pragma unroll
  for (int blk = 0; blk < C::NBLK; ++blk)
    *reinterpret_cast<f32x4*>(wsb + 4 + blk * 16 + q * 4) = acc[blk];
  if (has_lv) {
#pragma unroll
    for (int rc = 0; rc < C::RC; ++rc)
      if (rc * 16 + q * 4 < R) *reinterpret_cast<f32x4*>(wsb + 4 + D + rc * 16 + q * 4) = accl[rc];
  }
}

// The same merge for rows with at most 16 splits (split prefill, longer
// decode splits): one wave per row and four rows per workgroup.  Lane s < ns
// reads split s's maximum and sum; lane v < (d + r)/4 owns float4 column v of
// the accumulators and folds every split into it (all loads of the row in
// flight at once); the row's (d + r) sums then pass through LDS for the
// B_v product.
constexpr int MR_ROWS = 4;

template <int D, int R>
__global__ void __launch_bounds__(64 * MR_ROWS) lrsa_merge_rows_kernel(const AttnArgs a, int64_t n_rows) {
  constexpr int PS = 4 + D + R, NV = (D + R) / 4;
  static_assert(NV <= 64, "one lane per float4 column");
  __shared__ __attribute__((aligned(16))) float fin[MR_ROWS][D + R];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t orow = (int64_t)blockIdx.x * MR_ROWS + w;  // (request, token, head) row of O
  if (orow >= n_rows) return;
  const int ns = a.n_splits;
  const int h = (int)(orow % a.n_q);
  const int b = (int)(orow / a.n_q / a.n_tok);
  const int g = h / a.group;
  const bool has_lv = a.Lv != nullptr;
  const float* base = a.ws + orow * (int64_t)ns * PS;

  const float m_s = lane < ns ? base[(int64_t)lane * PS] : -INFINITY;
  const float l_s = lane < ns ? base[(int64_t)lane * PS + 1] : 0.f;
  float M = m_s;
#pragma unroll
  for (int x = 1; x < 64; x <<= 1) M = fmaxf(M, shfl_xor(M, x));
  const float Ms = (M == -INFINITY) ? 0.f : M;
  const float w_s = lane < ns ? fast_exp2(m_s - Ms) : 0.f;
  float L = w_s * l_s;
#pragma unroll
  for (int x = 1; x < 64; x <<= 1) L += shfl_xor(L, x);

  const int nv_used = has_lv ? NV : D / 4;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  const int v = lane < nv_used ? lane : 0;
#pragma unroll 4
  for (int s = 0; s < ns; ++s) {
    const float wgt = __shfl(w_s, s, 64);
    const f32x4 x = *reinterpret_cast<const f32x4*>(base + (int64_t)s * PS + 4 + 4 * v);
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] += wgt * x[c];
  }
  if (lane < nv_used) *reinterpret_cast<f32x4*>(&fin[w][4 * lane]) = acc;
  __builtin_amdgcn_wave_barrier();

  const float inv = L > 0.f ? 1.f / L : 0.f;
  uint16_t* o = a.O + orow * D;
#pragma unroll
  for (int dd = 0; dd < D / 64; ++dd) {
    const int dim = lane + 64 * dd;
    float sum = fin[w][dim];
    if (has_lv) {
      const int64_t ldb = (int64_t)a.n_kv * D;
      const uint16_t* bv = a.Bv + (int64_t)b * a.b_stride + (int64_t)g * D + dim;
#pragma unroll 8
      for (int j = 0; j < R; ++j) sum += fin[w][D + j] * __uint_as_float((uint32_t)bv[j * ldb] << 16);
    }
    const uint32_t pk = pack_bf16(sum * inv, 0.f);
    o[dim] = (uint16_t)(pk & 0xffffu);
  }
  if (a.lse != nullptr && lane == 0)
    a.lse[orow] = L > 0.f ? (M + __log2f(L)) * kLn2 : -INFINITY;
}

template <int D, int R>
hipError_t launch_merge_t(const AttnArgs& a, hipStream_t st) {
  if (a.n_splits <= 16) {
    const int64_t n_rows = (int64_t)a.batch * a.n_tok * a.n_q;
    hipLaunchKernelGGL((lrsa_merge_rows_kernel<D, R>), dim3((unsigned)((n_rows + MR_ROWS - 1) / MR_ROWS)),
                       dim3(64 * MR_ROWS), 0, st, a, n_rows);
    return hipGetLastError();
  }
  const dim3 grid(a.n_q, a.batch * a.n_tok);
  if (a.n_splits > 64)
    hipLaunchKernelGGL((lrsa_merge_kernel<D, R, 16>), grid, dim3(64 * 16), 0, st, a);
  else
    hipLaunchKernelGGL((lrsa_merge_kernel<D, R, 4>), grid, dim3(64 * 4), 0, st, a);
  return hipGetLastError();
}

template <int D, int R>
hipError_t launch_t(const AttnArgs& a, hipStream_t st) {
  if (a.kv_tbl != nullptr) {
    constexpr int nw = dec_nw(D, R, true);
    const dim3 grid(a.n_splits, (a.n_kv + nw - 1) / nw, a.batch);
    hipLaunchKernelGGL((lrsa_decode_kernel<D, R, true>), grid, dim3(64 * nw), 0, st, a);
  } else {
    constexpr int nw = dec_nw(D, R, false);
    const dim3 grid(a.n_splits, (a.n_kv + nw - 1) / nw, a.batch);
    hipLaunchKernelGGL((lrsa_decode_kernel<D, R, false>), grid, dim3(64 * nw), 0, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_merge_t<D, R>(a, st);
}

template <int D, int R>
hipError_t launch_shared_t(const AttnArgs& a, hipStream_t st) {
  using C = Dec<D, R>;
  const int rg = (a.batch + C::NW - 1) / C::NW;
  hipLaunchKernelGGL((lrsa_decode_shared_kernel<D, R>), dim3(a.n_splits, a.n_kv, rg), dim3(C::NT), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_merge_t<D, R>(a, st);
}

template <int D>
hipError_t launch_merge_r(const AttnArgs& a, hipStream_t st) {
  switch (a.rank) {
    case 8: return launch_merge_t<D, 8>(a, st);
    case 16: return launch_merge_t<D, 16>(a, st);
    case 32: return launch_merge_t<D, 32>(a, st);
    case 64: return launch_merge_t<D, 64>(a, st);
    default: return hipErrorInvalidValue;
  }
}

template <int D>
hipError_t launch_r(const AttnArgs& a, hipStream_t st, bool shared) {
  switch (a.rank) {
    case 8: return shared ? launch_shared_t<D, 8>(a, st) : launch_t<D, 8>(a, st);
    case 16: return shared ? launch_shared_t<D, 16>(a, st) : launch_t<D, 16>(a, st);
    case 32: return shared ? launch_shared_t<D, 32>(a, st) : launch_t<D, 32>(a, st);
    case 64: return shared ? launch_shared_t<D, 64>(a, st) : launch_t<D, 64>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int decode_tile_tokens() { return TK; }

bool decode_shares_base(int batch, int64_t kv_req_stride) { return batch > 1 && kv_req_stride == 0; }

void decode_plan(int64_t s_cap, int batch, int n_kv, int head_dim, int rank, bool shared_base, bool paged, int cus,
                 int* n_splits, int* split_tiles) {
  const int64_t tiles = (s_cap + TK - 1) / TK;
  const int nw = dec_waves(rank);
  const int64_t nb = batch > 0 ? batch : 1;
  // Workgroups per split: (request, group of nw KV heads) for the per-request
  // kernel, (KV head, group of nw requests) when the base cache is shared.
  const int64_t groups = shared_base ? (int64_t)n_kv * ((nb + nw - 1) / nw) : nb * ((n_kv + nw - 1) / nw);
  // Splits for a target of `rounds` 8-wave workgroups per CU.
  auto plan = [&](int64_t rounds, int64_t* ns_out, int64_t* st_out) {
    const int64_t target_wgs = rounds * (cus > 0 ? cus : 1) * 8 / nw;
    int64_t ns = (target_wgs + groups - 1) / groups;
    if (ns < 1) ns = 1;
    if (ns > tiles) ns = tiles > 0 ? tiles : 1;
    int64_t st = (tiles + ns - 1) / ns;
    if (st < 1) st = 1;
    ns = (tiles + st - 1) / st;
    *ns_out = ns < 1 ? 1 : ns;
    *st_out = st;
  };
  // About two rounds of one workgroup per CU (measured best for large
  // batches) while splits stay at least 8 tiles long; otherwise one round:
  // small batches then get longer splits, each CU at most one workgroup,
  // and half the partials to merge (batch 1 at 36k: 46 -> 38 us per call).
  // The rank-64 kernel that stages V by direct global->LDS loads holds its
  // workgroup's whole register file per CU and keeps one sub-block in flight
  // per wave: one round of longer splits measured faster there (64k, 8
  // requests: 426 -> 419 us; two, three and four rounds 426, 442, 446 us).
  int64_t ns, st;
  plan(2, &ns, &st);
  if (st < 8 || (!shared_base && dec_vdma(head_dim, rank, paged))) plan(1, &ns, &st);
  *n_splits = (int)ns;
  *split_tiles = (int)st;
}

size_t decode_workspace_bytes(int batch, int n_q, int n_splits, int head_dim, int rank) {
  return (size_t)batch * n_q * n_splits * (4 + head_dim + rank) * sizeof(float);
}

hipError_t launch_split_merge(const AttnArgs& a, hipStream_t st) {
  if (a.head_dim == 64) return launch_merge_r<64>(a, st);
  if (a.head_dim == 128) return launch_merge_r<128>(a, st);
  return hipErrorInvalidValue;
}

hipError_t launch_decode(const AttnArgs& a, hipStream_t st) {
  // Paged caches go through the per-request kernel (requests may share some
  // blocks and not others).
  const bool shared = a.kv_tbl == nullptr && decode_shares_base(a.batch, a.kv_stride);
  if (a.head_dim == 64) return launch_r<64>(a, st, shared);
  if (a.head_dim == 128) return launch_r<128>(a, st, shared);
  return hipErrorInvalidValue;
}

}  // namespace prc
