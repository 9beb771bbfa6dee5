// LR-shared attention, prefill (many query tokens per request), gfx950.
//
// Causal flash attention of a chunk of new query tokens over the shared base
// cache plus the current agent's LR cache (Sec. 3.1, reuse step).
//   keys:   each KV tile is rebuilt in LDS, K = K_base + RoPE(L_k B_k), with
//           the rank-r expansion before RoPE (App. D.2);
//   values: associativity (App. D.2), O = P V_base + (P L_v) B_v: V_base and
//           L_v tiles go to LDS unchanged, P L_v is accumulated beside P V_base
//           and B_v is applied once in the epilogue.
//
// Work split: one workgroup per (request, KV head, 32 * NCONS query rows).  A
// query row is a (token, q head of the GQA group) pair, so the group's heads
// share every rebuilt tile.  The workgroup's NCONS + 4 waves specialise:
//   producers (last 4 waves) load KV tile k+2 from HBM while rebuilding tile k+1
//             into LDS: E^T = B_k^T L_k^T on 16x16x16 MFMAs (lane l: token
//             l%16, both RoPE halves of each pair in the same lane), RoPE by
//             angle addition (exact per-tile base angle in LDS, exact per-lane
//             offsets in registers), + base, bf16, stored as K[tok][dim];
//             V_base and L_v rows are stored as they are;
//   consumers (first NCONS waves, 32 rows each) attend over tile k, in two
//             halves of 32 tokens:
//     scores  S^T = K Q^T on 32x32x16 MFMAs: lane l holds row l%32 and 32 of
//             the tile's tokens, so softmax statistics are per lane;
//     softmax online, exp2 domain, running max shared by lanes l and l^32;
//             the causal mask is applied only on tiles that cross it;
//     PV      O^T += V^T P^T and (P L_v)^T += L_v^T P^T on 32x32x16 MFMAs;
//             V^T and L_v^T come from row-major LDS tiles through the
//             transposing LDS read, P is already in the B operand layout,
//             and the softmax rescale is a per-lane scalar.
// LDS is double-buffered with one barrier per tile; producers and consumers
// share each SIMD, so the rebuild's vector work overlaps the MFMAs, and with
// 8 consumers each rebuilt tile serves 256 query rows.
#include "common.hpp"
#include "kernels.hpp"
#include "rebuild.hpp"

namespace prc {
namespace {

constexpr int TKV = 64;      // KV tokens per tile
constexpr int NPROD = 4;     // producer waves (16 rebuilt tokens each)
constexpr int WROWS = 32;    // query rows per consumer wave

template <int D, int R>
struct Pre {
  // Consumer waves (32 query rows each).  Eight fit three workgroup-waves per
  // SIMD within the register file; the widest accumulators (d = 128 with
  // rank >= 32) need the registers of two per SIMD, so they take four.
  static constexpr int NCONS = (D == 128 && R >= 32) ? 4 : 8;
  static constexpr int NTHR = 64 * (NCONS + NPROD);
  static constexpr int BROWS = NCONS * WROWS;
  static constexpr int HALF = D / 2;
  static constexpr int NB = D / 32;          // 16-dim blocks per RoPE half
  static constexpr int NBLK = D / 16;
  static constexpr int NCH = D / 32;         // 8-dim chunks per lane (rebuild)
  static constexpr int QPG = D / 8;          // dims per lane group per half
  static constexpr int RC = RCH(R);          // 16-wide rank chunks
  static constexpr int RB = (R + 31) / 32;   // 32-row blocks of (P L_v)^T
  static constexpr int NKQ = D / 16;         // 32x32x16 k-chunks over d
  static constexpr int NDB = D / 32;         // 32-dim blocks of O^T
  static constexpr int K_ROW = D + 8;        // bf16 per K row in LDS
  // Row strides of the tiles read with ds_read_b64_tr_b16: the two 16-lane
  // groups serviced together read the same 4 rows at column offsets 8 dwords
  // apart, which land on disjoint banks when the stride is 16 or 48 dwords
  // mod 64.
  static constexpr int V_ROW = D + 32;                   // 80 / 48 dwords
  static constexpr int LV_ROW = RB == 1 ? 32 : 96;       // 16 / 48 dwords
  static constexpr int LPR = D / 8;          // lanes per V row (16 bytes each)
  static constexpr int RPL = 64 / LPR;       // V rows per wave load
  static constexpr int NVL = 16 / RPL;       // V loads per wave per tile
};

__device__ __forceinline__ i16x4 lds_read_tr(const uint16_t* p) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((v4s __attribute__((address_space(3)))*)(p));
  return __builtin_bit_cast(i16x4, v);
}

// 32x32x16 A operand [32 rows x 16 tokens] from a row-major [token][col] LDS
// tile, in the token order of the P fragments: k = 8h + i is token
// 16m + 4h + i (i < 4) or 16m + 8 + 4h + (i - 4) (i >= 4), h = l/32.
__device__ __forceinline__ bf16x8 lds_tr_a32(const uint16_t* tile, int row_stride, int m, int col0, int lane) {
  const int gg = lane >> 4, j = lane & 15, h = lane >> 5;
  const uint16_t* p = tile + (16 * m + 4 * h + (j >> 2)) * row_stride + col0 + 16 * (gg & 1) + 4 * (j & 3);
  const i16x4 lo = lds_read_tr(p);
  const i16x4 hi = lds_read_tr(p + 8 * row_stride);
  typedef short v8s __attribute__((ext_vector_type(8)));
  v8s v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

template <int D, int R>
struct TileRegs {
  u32x4 kb[D / 32];          // K_base chunks of this lane's rebuild token
  u32x2 lk[RCH(R)];          // L_k fragment of that token
  u32x4 v[Pre<D, R>::NVL];   // V_base rows of the wave's 16 tokens
  u32x2 lv[RCH(R)];          // L_v fragment of this lane's rebuild token
};

template <int D, int R>
__device__ __forceinline__ void tile_load(TileRegs<D, R>& x, const uint16_t* Kb, const uint16_t* Vb,
                                          const uint16_t* Lk, const uint16_t* Lv, int64_t row_el, int64_t t0w,
                                          int64_t kv_hi, int lane) {
  using C = Pre<D, R>;
  const int64_t t = t0w + (lane & 15);
  const bool ok = t < kv_hi;
  load_chunks<D>(x.kb, Kb + t * row_el, ok, lane);
  if (Lk != nullptr) load_lr_frag<R>(x.lk, Lk + t * R, ok, lane);
  if (Lv != nullptr) load_lr_frag<R>(x.lv, Lv + t * R, ok, lane);
  const int vrow = lane / C::LPR, vdim = (lane % C::LPR) * 8;
#pragma unroll
  for (int iv = 0; iv < C::NVL; ++iv) {
    const int64_t tv = t0w + vrow + C::RPL * iv;
    x.v[iv] = ld16(Vb + tv * row_el + vdim, tv < kv_hi);
  }
}

template <int D, int R>
__global__ void __launch_bounds__((Pre<D, R>::NTHR))
lrsa_prefill_kernel(const AttnArgs a) {
  using C = Pre<D, R>;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][TKV * C::K_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][TKV * C::V_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t lv_lds[2][TKV * C::LV_ROW];
  __shared__ float2 base_cs[2][C::HALF];
  __shared__ int s_maxpos;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // Heaviest row tiles (latest positions, most keys) are dispatched first.
  const int rtile = gridDim.x - 1 - blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int G = a.group;
  const int n_rows = a.n_tok * G;
  const bool consumer = w < C::NCONS;
  const bool has_lk = a.Lk != nullptr, has_lv = a.Lv != nullptr;

  if (tid == 0) s_maxpos = -1;
  // L_v columns past the rank stay zero in both buffers.
  for (int i = tid; i < 2 * TKV * C::LV_ROW; i += C::NTHR) (&lv_lds[0][0])[i] = 0;

  int64_t kvl = a.kv_len[b];
  kvl = kvl < 0 ? 0 : (kvl > a.s_cap ? a.s_cap : kvl);

  // Consumer lane's query row (the same row for lanes l and l^32).
  const int l32 = lane & 31, h32 = lane >> 5;
  const int row = rtile * C::BROWS + w * WROWS + l32;
  const bool row_ok = consumer && row < n_rows;
  const int qi = row_ok ? row / G : 0, hh = row_ok ? row - qi * G : 0;
  const int pos = row_ok ? a.positions[(int64_t)b * a.n_tok + qi] : -1;
  const int64_t last = (int64_t)pos < kvl - 1 ? (int64_t)pos : kvl - 1;  // last visible key

  __syncthreads();
  if (row_ok && last >= 0) atomicMax(&s_maxpos, (int)last);
  __syncthreads();
  const int64_t kv_hi = (int64_t)s_maxpos + 1;  // keys [0, kv_hi) are needed
  const int n_tiles = (int)((kv_hi + TKV - 1) / TKV);

  const int64_t row_el = (int64_t)a.n_kv * D;
  const uint16_t* Kb = a.Kb + (int64_t)b * a.kv_stride + (int64_t)g * D;
  const uint16_t* Vb = a.Vb + (int64_t)b * a.kv_stride + (int64_t)g * D;
  const uint16_t* Lk = has_lk ? a.Lk + (int64_t)b * a.l_stride : nullptr;
  const uint16_t* Lv = has_lv ? a.Lv + (int64_t)b * a.l_stride : nullptr;

  if (!consumer) {
    // ======================= producer waves ================================
    const int pw_ = w - C::NCONS;            // 0..3: tokens 16*pw_ .. +15 of a tile
    const int ptid = tid - 64 * C::NCONS;    // 0..255
    const int q = lane >> 4, c16 = lane & 15;
    const int delta = pw_ * 16 + c16;      // this lane's rebuild token in a tile
    const int vrow = lane / C::LPR, vdim = (lane % C::LPR) * 8;
    i16x4 bkf[C::NBLK][C::RC];
    load_bt_frags<D, R>(bkf, has_lk ? a.Bk + (int64_t)b * a.b_stride + (int64_t)g * D * R : nullptr, has_lk,
                        lane);
    // RoPE offsets of token `delta` for this lane's D/8 frequencies, exact in
    // fp64 once per kernel.
    float cd[C::NB][4], sd[C::NB][4];
#pragma unroll
    for (int blk = 0; blk < C::NB; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        cd[blk][i] = 1.f;
        sd[blk][i] = 0.f;
        if (has_lk) rope_cs(delta, a.w2pi[q * C::QPG + blk * 4 + i], cd[blk][i], sd[blk][i]);
      }
    auto rebuild = [&](const TileRegs<D, R>& x, int buf) {
      u32x4 kb[C::NCH];
#pragma unroll
      for (int kk = 0; kk < C::NCH; ++kk) kb[kk] = x.kb[kk];
      if (has_lk) {
        float cc[C::NB][4], ss[C::NB][4];
#pragma unroll
        for (int blk = 0; blk < C::NB; ++blk)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float2 bc = base_cs[buf][q * C::QPG + blk * 4 + i];
            cc[blk][i] = bc.x * cd[blk][i] - bc.y * sd[blk][i];
            ss[blk][i] = bc.y * cd[blk][i] + bc.x * sd[blk][i];
          }
        add_rotated_expansion<D, R>(kb, bkf, x.lk, cc, ss);
      }
      store_chunks<D>(k_lds[buf] + delta * C::K_ROW, kb, lane);
#pragma unroll
      for (int iv = 0; iv < C::NVL; ++iv)
        *reinterpret_cast<u32x4*>(v_lds[buf] + (pw_ * 16 + vrow + C::RPL * iv) * C::V_ROW + vdim) = x.v[iv];
      if (has_lv) {
#pragma unroll
        for (int rc = 0; rc < C::RC; ++rc)
          if (rc * 16 + q * 4 < R)
            *reinterpret_cast<u32x2*>(lv_lds[buf] + delta * C::LV_ROW + rc * 16 + q * 4) = x.lv[rc];
      }
    };
    auto base_angles = [&](int64_t t0, int buf) {
      if (has_lk && ptid < C::HALF) {
        float c, s;
        rope_cs((int)t0, a.w2pi[ptid], c, s);
        base_cs[buf][ptid] = make_float2(c, s);
      }
    };
    // Prologue: tile 0 into LDS buffer 0, tile 1 in flight.
    TileRegs<D, R> x;
    if (n_tiles > 0) {
      tile_load<D, R>(x, Kb, Vb, Lk, Lv, row_el, pw_ * 16, kv_hi, lane);
      base_angles(0, 0);
    }
    __syncthreads();  // [P1] base angles of tile 0
    if (n_tiles > 0) rebuild(x, 0);
    if (n_tiles > 1) {
      tile_load<D, R>(x, Kb, Vb, Lk, Lv, row_el, TKV + pw_ * 16, kv_hi, lane);
      base_angles(TKV, 1);
    }
    __syncthreads();  // [P2] tile 0 in LDS
    for (int tile = 0; tile < n_tiles; ++tile) {
      const int buf = tile & 1;
      const int64_t t0 = (int64_t)tile * TKV;
      if (tile + 1 < n_tiles) rebuild(x, buf ^ 1);
      if (tile + 2 < n_tiles) {
        tile_load<D, R>(x, Kb, Vb, Lk, Lv, row_el, t0 + 2 * TKV + pw_ * 16, kv_hi, lane);
        base_angles(t0 + 2 * TKV, buf);
      }
      __syncthreads();  // [T] tile+1 in LDS; tile consumed
    }
    return;
  }

  // ========================= consumer waves ================================
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
  }
  f32x16 acc[C::NDB];   // O^T: lane col = row l%32
  f32x16 accl[C::RB];   // (P L_v)^T
#pragma unroll
  for (int db = 0; db < C::NDB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[db][j] = 0.f;
#pragma unroll
  for (int rb = 0; rb < C::RB; ++rb)
#pragma unroll
    for (int j = 0; j < 16; ++j) accl[rb][j] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  __syncthreads();  // [P1]
  __syncthreads();  // [P2]
  for (int tile = 0; tile < n_tiles; ++tile) {
    const int buf = tile & 1;
    const int64_t t0 = (int64_t)tile * TKV;
    // The tile is consumed as two 32-token halves, each with its own online
    // softmax update (half the live score and P registers of a whole tile).
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const int64_t th = t0 + tb * 32;  // first token of this half
      if (th > (int64_t)wave_last) break;
      const uint16_t* kl = k_lds[buf] + (tb * 32 + l32) * C::K_ROW + h32 * 8;
      f32x16 s;
#pragma unroll
      for (int j = 0; j < 16; ++j) s[j] = 0.f;
#pragma unroll
      for (int kk = 0; kk < C::NKQ; ++kk)
        s = mfma32x32x16(as_bf16x8(*reinterpret_cast<const u32x4*>(kl + kk * 16)), qf[kk], s);
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
      mx = fmaxf(mx, shfl_xor(mx, 32)) * a.scale_log2;
      const float mn = fmaxf(m_run, mx);
      const float ms = (mn == -INFINITY) ? 0.f : mn;
      const float alpha = fast_exp2(m_run - ms);
      m_run = mn;
      float ls0 = 0.f, ls1 = 0.f;
      u32x4 pw[2];  // bf16 P of this half, one per 16-token chunk
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const float p0 = fast_exp2(__builtin_fmaf(s[hf * 8 + 2 * c], a.scale_log2, -ms));
          const float p1 = fast_exp2(__builtin_fmaf(s[hf * 8 + 2 * c + 1], a.scale_log2, -ms));
          ls0 += p0;
          ls1 += p1;
          pw[hf][c] = pack_bf16(p0, p1);
        }
      l_run = l_run * alpha + (ls0 + ls1);
      if (__ballot(alpha != 1.f)) {
#pragma unroll
        for (int db = 0; db < C::NDB; ++db) acc[db] *= alpha;
#pragma unroll
        for (int rb = 0; rb < C::RB; ++rb) accl[rb] *= alpha;
      }
      // O^T[dims x rows] += V^T[dims x 16 tok] P^T[16 tok x rows] for the two
      // 16-token chunks of this half; (P L_v)^T likewise with L_v^T.
      const uint16_t* vt = v_lds[buf];
      const uint16_t* lvt = lv_lds[buf];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const int m = 2 * tb + hf;
        const bf16x8 pb = as_bf16x8(pw[hf]);
#pragma unroll
        for (int db = 0; db < C::NDB; ++db)
          acc[db] = mfma32x32x16(lds_tr_a32(vt, C::V_ROW, m, db * 32, lane), pb, acc[db]);
        if (has_lv) {
#pragma unroll
          for (int rb = 0; rb < C::RB; ++rb)
            accl[rb] = mfma32x32x16(lds_tr_a32(lvt, C::LV_ROW, m, rb * 32, lane), pb, accl[rb]);
        }
      }
    }
    __syncthreads();  // [T]
  }

  // ---- epilogue: O^T += B_v^T (P L_v)^T, then O = acc / l, lse -------------
  if (has_lv) {
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
        const uint16_t* bv = a.Bv + (int64_t)b * a.b_stride + ((int64_t)g * D + dim) * R;
        const u32x2 b0 = ld8(bv + r0, r0 < R);
        const u32x2 b1 = ld8(bv + r0 + 8, r0 + 8 < R);
        const u32x4 bw = {b0[0], b0[1], b1[0], b1[1]};
        acc[db] = mfma32x32x16(as_bf16x8(bw), as_bf16x8(hi), acc[db]);
        acc[db] = mfma32x32x16(as_bf16x8(bw), as_bf16x8(lo), acc[db]);
      }
    }
  }
  const float l_tot = l_run + shfl_xor(l_run, 32);
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

template <int D, int R>
hipError_t launch_t(const AttnArgs& a, hipStream_t st) {
  const int n_rows = a.n_tok * a.group;
  using C = Pre<D, R>;
  const int tiles = (n_rows + C::BROWS - 1) / C::BROWS;
  hipLaunchKernelGGL((lrsa_prefill_kernel<D, R>), dim3(tiles, a.n_kv, a.batch), dim3(C::NTHR), 0, st, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_r(const AttnArgs& a, hipStream_t st) {
  switch (a.rank) {
    case 8: return launch_t<D, 8>(a, st);
    case 16: return launch_t<D, 16>(a, st);
    case 32: return launch_t<D, 32>(a, st);
    case 64: return launch_t<D, 64>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_prefill(const AttnArgs& a, hipStream_t st) {
  if (a.head_dim == 64) return launch_r<64>(a, st);
  if (a.head_dim == 128) return launch_r<128>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace prc
