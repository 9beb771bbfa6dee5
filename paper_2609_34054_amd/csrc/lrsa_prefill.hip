// LR-shared attention, prefill (many query tokens per request), gfx950.
//
// Causal flash attention of a chunk of new query tokens over the shared base
// cache plus the current agent's LR cache (Sec. 3.1, reuse step).  Each KV
// tile is rebuilt in LDS before use (App. D.2 order: rank-r expansion, then
// RoPE on the key side):
//     K_tile = K_base + RoPE(L_k B_k),   V_tile = V_base + L_v B_v.
//
// Work split: one workgroup (4 waves) per (request, KV head, 128 query rows).
// A query row is a (token, q head of the GQA group) pair, so the group's
// heads share every rebuilt tile.  Each wave owns 32 rows.
//
// Per 64-token KV tile:
//   rebuild   wave w rebuilds tokens 16w..16w+15: E^T = B^T L^T with 16x16x16
//             MFMAs (lane l: token l%16, both RoPE halves of 16 pairs), RoPE
//             by angle addition (exact per-tile base angle in LDS, exact
//             per-lane offset angles in registers), + base, bf16, stored as
//             K[tok][dim] and V^T[dim][tok] in LDS;
//   scores    S^T = K Q^T with 32x32x16 MFMAs: lane l holds row l%32 and 32
//             of the tile's tokens, so softmax statistics are per lane;
//   softmax   online, exp2 domain, running max shared by lanes l and l^32;
//   PV        O^T += V^T P^T with 32x32x16 MFMAs; P is already in the B
//             operand layout, O^T keeps one row per lane, so the rescale by
//             the softmax correction is a per-lane scalar.
#include "common.hpp"
#include "kernels.hpp"
#include "rebuild.hpp"

namespace prc {
namespace {

constexpr int TKV = 64;      // KV tokens per tile
constexpr int NWAVE = 4;     // waves per workgroup
constexpr int WROWS = 32;    // query rows per wave
constexpr int BROWS = NWAVE * WROWS;

template <int D, int R>
struct Pre {
  static constexpr int HALF = D / 2;
  static constexpr int NB = D / 32;        // 16-dim blocks per RoPE half
  static constexpr int NBLK = D / 16;
  static constexpr int QPG = HALF / 4;     // dims per lane group per half
  static constexpr int RC = R < 16 ? 1 : R / 16;
  static constexpr int NKQ = D / 16;       // 32x32x16 k-chunks over d
  static constexpr int NDB = D / 32;       // 32-dim blocks of O^T
  static constexpr int K_ROW = D + 8;      // bf16 per K row in LDS (padded)
  static constexpr int VT_ROW = TKV + 8;   // bf16 per V^T row in LDS (padded)
};

template <int D, int R>
__global__ void __launch_bounds__(256)
lrsa_prefill_kernel(const AttnArgs a) {
  using C = Pre<D, R>;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[TKV * C::K_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t vt_lds[D * C::VT_ROW];
  __shared__ float2 base_cs[C::HALF];
  __shared__ double w_lds[C::HALF];
  __shared__ int s_maxpos;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int rtile = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int G = a.group;
  const int n_rows = a.n_tok * G;
  const int q = lane >> 4, c16 = lane & 15;
  const int l32 = lane & 31, h32 = lane >> 5;
  const bool has_lk = a.Lk != nullptr, has_lv = a.Lv != nullptr;

  for (int j = tid; j < C::HALF; j += blockDim.x) w_lds[j] = a.w2pi[j];
  if (tid == 0) s_maxpos = -1;

  int64_t kvl = a.kv_len[b];
  kvl = kvl < 0 ? 0 : (kvl > a.s_cap ? a.s_cap : kvl);

  // This lane's query row (the same row for lanes l and l^32).
  const int row = rtile * BROWS + w * WROWS + l32;
  const bool row_ok = row < n_rows;
  const int qi = row_ok ? row / G : 0, hh = row_ok ? row - qi * G : 0;
  const int pos = row_ok ? a.positions[(int64_t)b * a.n_tok + qi] : -1;
  // Last key this row may see.
  const int64_t last = (int64_t)pos < kvl - 1 ? (int64_t)pos : kvl - 1;

  __syncthreads();
  if (row_ok && last >= 0) atomicMax(&s_maxpos, (int)last);
  // Wave-level bound, to skip tiles no row of this wave can see.
  int wave_last = (int)last;
#pragma unroll
  for (int x = 1; x < 64; x <<= 1) {
    const int o = __shfl_xor(wave_last, x, 64);
    wave_last = o > wave_last ? o : wave_last;
  }

  // Q^T as the B operand of S^T = K Q^T: lane col = row l%32,
  // k = (l/32)*8 + 0..7 within each 16-dim chunk.
  bf16x8 qf[C::NKQ];
  {
    const uint16_t* qp = a.Q + (((int64_t)b * a.n_tok + qi) * a.n_q + (int64_t)g * G + hh) * D;
#pragma unroll
    for (int kk = 0; kk < C::NKQ; ++kk) qf[kk] = as_bf16x8(ld16(qp + kk * 16 + h32 * 8, row_ok));
  }

  // Expansion operands B^T of this KV head (A operand of 16x16x16).
  i16x4 bkf[C::NBLK][C::RC], bvf[C::NBLK][C::RC];
  {
    const int64_t off = (int64_t)b * a.b_stride + (int64_t)g * D * R;
    load_bt_frags<D, R>(bkf, has_lk ? a.Bk + off : nullptr, has_lk, lane);
    load_bt_frags<D, R>(bvf, has_lv ? a.Bv + off : nullptr, has_lv, lane);
  }

  __syncthreads();  // w_lds, s_maxpos ready
  const int64_t kv_hi = (int64_t)s_maxpos + 1;  // keys [0, kv_hi) are needed

  // RoPE offsets of this lane's rebuild token (tile offset 16w + l%16) for its
  // 16 (or 8) frequencies, exact in fp64 once per kernel.
  const int delta = w * 16 + c16;
  float cd[C::NB][4], sd[C::NB][4];
#pragma unroll
  for (int blk = 0; blk < C::NB; ++blk)
#pragma unroll
    for (int i = 0; i < 4; ++i) rope_cs(delta, w_lds[q * C::QPG + blk * 4 + i], cd[blk][i], sd[blk][i]);

  const int64_t row_el = (int64_t)a.n_kv * D;
  const uint16_t* Kb = a.Kb + (int64_t)b * a.kv_stride + (int64_t)g * D;
  const uint16_t* Vb = a.Vb + (int64_t)b * a.kv_stride + (int64_t)g * D;
  const uint16_t* Lk = has_lk ? a.Lk + (int64_t)b * a.l_stride : nullptr;
  const uint16_t* Lv = has_lv ? a.Lv + (int64_t)b * a.l_stride : nullptr;

  f32x16 acc[C::NDB];
#pragma unroll
  for (int db = 0; db < C::NDB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[db][j] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  for (int64_t t0 = 0; t0 < kv_hi; t0 += TKV) {
    // ---- exact base angles of this tile --------------------------------
    if (has_lk && tid < C::HALF) {
      float c, s;
      rope_cs((int)t0, w_lds[tid], c, s);
      base_cs[tid] = make_float2(c, s);
    }
    __syncthreads();

    // ---- rebuild 16 tokens per wave ------------------------------------
    {
      const int64_t t = t0 + delta;
      const bool ok = t < kv_hi;
      u32x4 kb[Rb<D, R>::NCH], vb[Rb<D, R>::NCH];
      load_chunks<D>(kb, Kb + t * row_el, ok, lane);
      load_chunks<D>(vb, Vb + t * row_el, ok, lane);
      if (has_lk) {
        u32x2 lk[C::RC];
        load_lr_frag<R>(lk, Lk + t * R, ok, lane);
        // Angle addition: (t0 + delta) * omega from the exact tile base and
        // the exact per-lane offset.
        float cc[C::NB][4], ss[C::NB][4];
#pragma unroll
        for (int blk = 0; blk < C::NB; ++blk)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float2 bc = base_cs[q * C::QPG + blk * 4 + i];
            cc[blk][i] = bc.x * cd[blk][i] - bc.y * sd[blk][i];
            ss[blk][i] = bc.y * cd[blk][i] + bc.x * sd[blk][i];
          }
        add_rotated_expansion<D, R>(kb, bkf, lk, cc, ss);
      }
      store_chunks<D>(k_lds + delta * C::K_ROW, kb, lane);
      if (has_lv) {
        u32x2 lv[C::RC];
        load_lr_frag<R>(lv, Lv + t * R, ok, lane);
        add_expansion<D, R>(vb, bvf, lv);
      }
      // V stored transposed, V^T[dim][token], for the PV operand.
#pragma unroll
      for (int kk = 0; kk < Rb<D, R>::NCH; ++kk) {
        const int d0 = chunk_dim<D>(kk, q);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t u = vb[kk][e >> 1];
          vt_lds[(d0 + e) * C::VT_ROW + delta] = (uint16_t)((e & 1) ? (u >> 16) : (u & 0xffffu));
        }
      }
    }
    __syncthreads();

    // ---- scores, softmax and PV for this wave's 32 rows ----------------
    if (t0 <= (int64_t)wave_last) {
      f32x16 s[2];
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
#pragma unroll
        for (int j = 0; j < 16; ++j) s[tb][j] = 0.f;
        const uint16_t* kr = k_lds + (tb * 32 + l32) * C::K_ROW + h32 * 8;
#pragma unroll
        for (int kk = 0; kk < C::NKQ; ++kk) {
          const bf16x8 kfrag = as_bf16x8(*reinterpret_cast<const u32x4*>(kr + kk * 16));
          s[tb] = mfma32x32x16(kfrag, qf[kk], s[tb]);
        }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int64_t t = t0 + tb * 32 + (j >> 2) * 8 + h32 * 4 + (j & 3);
          const float v = t <= last ? s[tb][j] * a.scale_log2 : -INFINITY;
          s[tb][j] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, shfl_xor(mx, 32));
      const float mn = fmaxf(m_run, mx);
      const float ms = (mn == -INFINITY) ? 0.f : mn;
      const float alpha = fast_exp2(m_run - ms);
      m_run = mn;
      float ls = 0.f;
      u32x4 pw[2][2];  // bf16 P: [token block][half of its 16 registers]
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const float p0 = fast_exp2(s[tb][hf * 8 + 2 * c] - ms);
            const float p1 = fast_exp2(s[tb][hf * 8 + 2 * c + 1] - ms);
            ls += p0 + p1;
            pw[tb][hf][c] = pack_bf16(p0, p1);
          }
      l_run = l_run * alpha + ls;
#pragma unroll
      for (int db = 0; db < C::NDB; ++db)
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[db][j] *= alpha;
      // O^T[dims x rows] += V^T[dims x 16 tok] P^T[16 tok x rows], 4 chunks.
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const bf16x8 pb = as_bf16x8(pw[m >> 1][m & 1]);
#pragma unroll
        for (int db = 0; db < C::NDB; ++db) {
          const uint16_t* vr = vt_lds + (db * 32 + l32) * C::VT_ROW + m * 16 + h32 * 4;
          const u32x2 lo = *reinterpret_cast<const u32x2*>(vr);
          const u32x2 hi = *reinterpret_cast<const u32x2*>(vr + 8);
          const u32x4 va = {lo[0], lo[1], hi[0], hi[1]};
          acc[db] = mfma32x32x16(as_bf16x8(va), pb, acc[db]);
        }
      }
    }
    __syncthreads();
  }

  // ---- epilogue: O = acc / l, lse -----------------------------------------
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
  const int tiles = (n_rows + BROWS - 1) / BROWS;
  hipLaunchKernelGGL((lrsa_prefill_kernel<D, R>), dim3(tiles, a.n_kv, a.batch), dim3(64 * NWAVE), 0,
                     st, a);
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
