// LR-shared attention, decode (one query token per request), gfx950.
//
// Reuse step of PreLRShared (Sec. 3.1): the current agent attends over the
// shared base cache plus its own rank-r LR cache.  Keys are rebuilt on chip,
// K = K_base + RoPE(L_k B_k), with the rank-r expansion done before RoPE
// (App. D.2).  Values use the associativity of App. D.2:
//     P (V_base + L_v B_v) = P V_base + (P L_v) B_v,
// so only an r-wide accumulator is carried per head and B_v is applied once.
//
// Work split (flash-decoding): one workgroup per (request, KV-range split,
// group of up to 8 KV heads); one wavefront per KV head.  Each wave keeps the
// whole GQA group of its KV head in one 16-row MFMA tile.  The waves of a
// workgroup walk the same tokens, so the RoPE cos/sin table of each KV tile is
// built once in LDS and shared by all 8 heads.  The LR rows are per token and
// shared by all heads, so they are read through the same L1 lines.  A second
// kernel merges the split partials with log-sum-exp weights.
//
// Per 16-token sub-block, each wave:
//   1. loads L_k rows and expands E^T = B_k^T L_k^T with 16x16x16 MFMAs;
//      lane l then holds token l%16 and 32 head dims, both RoPE halves of
//      every pair in the same lane;
//   2. rotates E at the token's position, adds K_base and rounds to bf16;
//      the result is already the B operand of the QK^T MFMA;
//   3. computes S = Q K^T with 16x16x32 MFMAs (rows = q heads of the group).
//   4. updates the online softmax (exp2, per-head running max and sum);
//   5. passes P through a wave-private LDS block, then runs P V_base and
//      P L_v on the vector ALUs (fp32 P), reading V in its natural layout.
#include "common.hpp"
#include "kernels.hpp"
#include "rebuild.hpp"

namespace prc {
namespace {

constexpr int TK = 32;        // tokens per KV tile (one LDS table, one barrier)
constexpr int NSB = TK / 16;  // 16-token sub-blocks per tile
constexpr int MAXW = 8;       // waves (KV heads) per workgroup

template <int D, int R, int GM>
struct Dec {
  static constexpr int HALF = D / 2;
  static constexpr int NB = D / 32;           // 16-dim blocks per RoPE half
  static constexpr int NBLK = D / 16;         // 16-dim blocks
  static constexpr int QPG = HALF / 4;        // dims per lane group per half
  static constexpr int NKK = D / 32;          // 16x16x32 k-chunks over d
  static constexpr int RC = R < 16 ? 1 : R / 16;  // 16-wide rank chunks
  static constexpr int CS_ROW = HALF + 2;     // float2 per table row (padded)
  static constexpr int PG = GM <= 4 ? 4 : 8;  // floats per token row of P
  static constexpr int LPR = D / 8;           // lanes per V row (8 dims each)
  static constexpr int RPL = 64 / LPR;        // V rows per wave load
  static constexpr int NVL = 16 / RPL;        // V loads per sub-block
  static constexpr int PS = 4 + D + R;        // floats per split partial
  static constexpr int LRG = 64 / R;          // token groups of the P L_v layout
  static constexpr int LTK = 16 / LRG;        // P L_v tokens per lane per sub-block
};

template <int D, int R, int GM>
__global__ void __launch_bounds__(512)
lrsa_decode_kernel(const AttnArgs a) {
  using C = Dec<D, R, GM>;
  __shared__ float2 cs_lds[2][TK * C::CS_ROW];
  __shared__ __attribute__((aligned(16))) float p_lds[MAXW][16 * C::PG];
  __shared__ double w_lds[C::HALF];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nthreads = blockDim.x;
  const int split = blockIdx.x, b = blockIdx.z;
  const int g = blockIdx.y * MAXW + w;
  const bool active = g < a.n_kv;
  const int G = a.group;
  const int q = lane >> 4, c16 = lane & 15;
  const bool has_lk = a.Lk != nullptr, has_lv = a.Lv != nullptr;

  for (int j = tid; j < C::HALF; j += nthreads) w_lds[j] = a.w2pi[j];

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

  const int64_t row = (int64_t)a.n_kv * D;  // elements between tokens
  const uint16_t* Kb = a.Kb + (int64_t)b * a.kv_stride + (int64_t)g * D;
  const uint16_t* Vb = a.Vb + (int64_t)b * a.kv_stride + (int64_t)g * D;
  const uint16_t* Lk = has_lk ? a.Lk + (int64_t)b * a.l_stride : nullptr;
  const uint16_t* Lv = has_lv ? a.Lv + (int64_t)b * a.l_stride : nullptr;

  // Q of the group as the A operand (rows = q heads, zero rows past G).
  bf16x8 qf[C::NKK];
  {
    const bool ok = active && c16 < G;
    const uint16_t* qp = a.Q + ((int64_t)b * a.n_tok * a.n_q + (int64_t)g * G + c16) * D;
#pragma unroll
    for (int kk = 0; kk < C::NKK; ++kk) qf[kk] = as_bf16x8(ld16(qp + chunk_dim<D>(kk, q), ok));
  }
  // B_k^T of this KV head as the A operand of the expansion.
  i16x4 bkf[C::NBLK][C::RC];
  load_bt_frags<D, R>(bkf, has_lk ? a.Bk + (int64_t)b * a.b_stride + (int64_t)g * D * R : nullptr,
                      has_lk && active, lane);

  float m_run[4], l_run[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { m_run[i] = -INFINITY; l_run[i] = 0.f; }
  float acc[GM][8];
  float accl[GM];  // value-side LR accumulator: lane holds rank index lane % R
#pragma unroll
  for (int h = 0; h < GM; ++h) {
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[h][c] = 0.f;
    accl[h] = 0.f;
  }
  const int lr_j = lane % R, lr_g = lane / R;  // rank index, token group
  const int vrow0 = lane / C::LPR, vdim0 = (lane % C::LPR) * 8;
  float* pl = p_lds[w];

  __syncthreads();  // w_lds ready

  for (int tile = 0; tile < n_tiles; ++tile) {
    const int64_t t0 = t_begin + (int64_t)tile * TK;
    float2* cs = cs_lds[tile & 1];
    if (has_lk) {
      for (int e = tid; e < TK * C::HALF; e += nthreads) {
        const int tok = e / C::HALF, j = e - tok * C::HALF;
        float c, s;
        rope_cs((int)(t0 + tok), w_lds[j], c, s);
        cs[tok * C::CS_ROW + j] = make_float2(c, s);
      }
    }
    __syncthreads();  // table of this tile ready; double buffering keeps the
                      // previous tile's table intact for slower waves.
    if (!active) continue;

#pragma unroll 1
    for (int sb = 0; sb < NSB; ++sb) {
      // ---- 1-3: rebuild K for 16 tokens and score them -------------------
      const int64_t t = t0 + sb * 16 + c16;
      const bool ok = t < t_end;
      u32x4 kb[C::NKK];
      load_chunks<D>(kb, Kb + t * row, ok, lane);
      bf16x8 kf[C::NKK];
      if (has_lk) {
        u32x2 lk[C::RC];
        load_lr_frag<R>(lk, Lk + t * R, ok, lane);
        const float2* csr = cs + (sb * 16 + c16) * C::CS_ROW + q * C::QPG;
        float cc[C::NB][4], ss[C::NB][4];
#pragma unroll
        for (int blk = 0; blk < C::NB; ++blk)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float2 r = csr[blk * 4 + i];
            cc[blk][i] = r.x;
            ss[blk][i] = r.y;
          }
        add_rotated_expansion<D, R>(kb, bkf, lk, cc, ss);
      }
#pragma unroll
      for (int kk = 0; kk < C::NKK; ++kk) kf[kk] = as_bf16x8(kb[kk]);
      f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < C::NKK; ++kk) sc = mfma16x16x32(qf[kk], kf[kk], sc);

      // ---- online softmax over these 16 tokens ---------------------------
      // Lanes of group q hold q heads 4q..4q+3, one token per lane.
      float alpha[4], p[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float s2 = ok ? sc[i] * a.scale_log2 : -INFINITY;
        const float mx = max16(s2);
        const float mn = fmaxf(m_run[i], mx);
        const float ms = (mn == -INFINITY) ? 0.f : mn;
        alpha[i] = fast_exp2(m_run[i] - ms);
        p[i] = fast_exp2(s2 - ms);
        l_run[i] = l_run[i] * alpha[i] + p[i];
        m_run[i] = mn;
      }
      if (q * 4 < G)
        *reinterpret_cast<float4*>(&pl[c16 * C::PG + q * 4]) = make_float4(p[0], p[1], p[2], p[3]);
      __builtin_amdgcn_wave_barrier();
      float al[GM];
#pragma unroll
      for (int h = 0; h < GM; ++h) al[h] = readlane_f(alpha[h & 3], (h >> 2) * 16);

      // ---- P V_base on the vector ALUs, V in its natural layout ----------
#pragma unroll
      for (int h = 0; h < GM; ++h)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[h][c] *= al[h];
#pragma unroll
      for (int iv = 0; iv < C::NVL; ++iv) {
        const int tok = vrow0 + C::RPL * iv;
        const int64_t tv = t0 + sb * 16 + tok;
        const u32x4 v = ld16(Vb + tv * row + vdim0, tv < t_end);
        float vf[8];
#pragma unroll
        for (int c = 0; c < 4; ++c) { vf[2 * c] = bf_lo(v[c]); vf[2 * c + 1] = bf_hi(v[c]); }
        const float* pr = pl + tok * C::PG;
#pragma unroll
        for (int h = 0; h < GM; ++h) {
          const float ph = pr[h];
#pragma unroll
          for (int c = 0; c < 8; ++c) acc[h][c] += ph * vf[c];
        }
      }
      // ---- P L_v (value-side LR accumulator) ------------------------------
      // Lane l owns rank index l % R and the tokens congruent to l / R modulo
      // 64 / R, so each load instruction reads 64 consecutive bf16.
      if (has_lv) {
#pragma unroll
        for (int h = 0; h < GM; ++h) accl[h] *= al[h];
#pragma unroll
        for (int k = 0; k < C::LTK; ++k) {
          const int tok = lr_g + C::LRG * k;
          const int64_t tl = t0 + sb * 16 + tok;
          const float lv = tl < t_end ? __uint_as_float((uint32_t)Lv[tl * R + lr_j] << 16) : 0.f;
          const float* pr = pl + tok * C::PG;
#pragma unroll
          for (int h = 0; h < GM; ++h) accl[h] += pr[h] * lv;
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
    __builtin_amdgcn_wave_barrier();
  }

  if (!active) return;
  // Cross-lane reductions, then one partial per (request, q head, split).
#pragma unroll
  for (int i = 0; i < 4; ++i) l_run[i] = sum16(l_run[i]);
#pragma unroll
  for (int h = 0; h < GM; ++h)
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
      for (int x = C::LPR; x < 64; x <<= 1) acc[h][c] += shfl_xor(acc[h][c], x);
  if (has_lv) {
#pragma unroll
    for (int h = 0; h < GM; ++h)
#pragma unroll
      for (int x = R; x < 64; x <<= 1) accl[h] += shfl_xor(accl[h], x);
  }
  const int64_t hstride = (int64_t)a.n_splits * C::PS;
  float* wsb = a.ws + ((int64_t)b * a.n_q + (int64_t)g * G) * hstride + (int64_t)split * C::PS;
  if (c16 == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int hh = q * 4 + i;
      if (hh < G) {
        wsb[hh * hstride + 0] = m_run[i];
        wsb[hh * hstride + 1] = l_run[i];
      }
    }
  }
  if (lane < C::LPR) {
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      if (h < G) {
        float* dst = wsb + h * hstride + 4 + vdim0;
        *reinterpret_cast<float4*>(dst) = make_float4(acc[h][0], acc[h][1], acc[h][2], acc[h][3]);
        *reinterpret_cast<float4*>(dst + 4) = make_float4(acc[h][4], acc[h][5], acc[h][6], acc[h][7]);
      }
    }
  }
  if (has_lv && lane < R) {
#pragma unroll
    for (int h = 0; h < GM; ++h)
      if (h < G) wsb[h * hstride + 4 + D + lr_j] = accl[h];
  }
}

// Merge the split partials of one (request, q head): log-sum-exp weights,
// then the deferred up-projection O += (sum_s w_s P_s L_v) B_v, then 1/l.
template <int D, int R>
__global__ void __launch_bounds__(64)
lrsa_merge_kernel(const AttnArgs a) {
  constexpr int PS = 4 + D + R, DPL = D / 64;
  __shared__ float accl_s[64];
  const int h = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
  const int g = h / a.group;
  const bool has_lv = a.Lv != nullptr;
  const float* base = a.ws + ((int64_t)b * a.n_q + h) * (int64_t)a.n_splits * PS;

  float M = -INFINITY;
  for (int s = lane; s < a.n_splits; s += 64) M = fmaxf(M, base[(int64_t)s * PS]);
#pragma unroll
  for (int x = 1; x < 64; x <<= 1) M = fmaxf(M, shfl_xor(M, x));
  const float Ms = (M == -INFINITY) ? 0.f : M;

  float L = 0.f, accl = 0.f, acc[DPL];
#pragma unroll
  for (int dd = 0; dd < DPL; ++dd) acc[dd] = 0.f;
  for (int s = 0; s < a.n_splits; ++s) {
    const float* p = base + (int64_t)s * PS;
    const float wgt = fast_exp2(p[0] - Ms);
    L += wgt * p[1];
#pragma unroll
    for (int dd = 0; dd < DPL; ++dd) acc[dd] += wgt * p[4 + lane + 64 * dd];
    if (has_lv && lane < R) accl += wgt * p[4 + D + lane];
  }
  if (has_lv) {
    if (lane < R) accl_s[lane] = accl;
    __syncthreads();
#pragma unroll
    for (int dd = 0; dd < DPL; ++dd) {
      const int dim = lane + 64 * dd;
      const uint16_t* bv = a.Bv + (int64_t)b * a.b_stride + ((int64_t)g * D + dim) * R;
      float sum = 0.f;
#pragma unroll
      for (int j = 0; j < R; j += 8) {
        const u32x4 u = *reinterpret_cast<const u32x4*>(bv + j);
#pragma unroll
        for (int c = 0; c < 4; ++c) sum += accl_s[j + 2 * c] * bf_lo(u[c]) + accl_s[j + 2 * c + 1] * bf_hi(u[c]);
      }
      acc[dd] += sum;
    }
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  uint16_t* o = a.O + ((int64_t)b * a.n_tok * a.n_q + h) * D;
#pragma unroll
  for (int dd = 0; dd < DPL; ++dd) {
    const uint32_t pk = pack_bf16(acc[dd] * inv, 0.f);
    o[lane + 64 * dd] = (uint16_t)(pk & 0xffffu);
  }
  if (a.lse != nullptr && lane == 0)
    a.lse[(int64_t)b * a.n_tok * a.n_q + h] = L > 0.f ? (M + __log2f(L)) * kLn2 : -INFINITY;
}

template <int D, int R, int GM>
hipError_t launch_t(const AttnArgs& a, hipStream_t st) {
  const int hg = (a.n_kv + MAXW - 1) / MAXW;
  const int waves = a.n_kv < MAXW ? a.n_kv : MAXW;
  hipLaunchKernelGGL((lrsa_decode_kernel<D, R, GM>), dim3(a.n_splits, hg, a.batch), dim3(64 * waves),
                     0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((lrsa_merge_kernel<D, R>), dim3(a.n_q, a.batch), dim3(64), 0, st, a);
  return hipGetLastError();
}

template <int D, int R>
hipError_t launch_g(const AttnArgs& a, hipStream_t st) {
  if (a.group == 1) return launch_t<D, R, 1>(a, st);
  if (a.group <= 4) return launch_t<D, R, 4>(a, st);
  return launch_t<D, R, 8>(a, st);
}

template <int D>
hipError_t launch_r(const AttnArgs& a, hipStream_t st) {
  switch (a.rank) {
    case 8: return launch_g<D, 8>(a, st);
    case 16: return launch_g<D, 16>(a, st);
    case 32: return launch_g<D, 32>(a, st);
    case 64: return launch_g<D, 64>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int decode_tile_tokens() { return TK; }

void decode_plan(int64_t s_cap, int batch, int n_kv, int* n_splits, int* split_tiles) {
  const int64_t tiles = (s_cap + TK - 1) / TK;
  const int64_t hg = (n_kv + MAXW - 1) / MAXW;
  const int64_t groups = (int64_t)(batch > 0 ? batch : 1) * hg;
  const int64_t target_wgs = 1024;  // about four workgroups per CU
  int64_t ns = (target_wgs + groups - 1) / groups;
  if (ns < 1) ns = 1;
  if (ns > tiles) ns = tiles > 0 ? tiles : 1;
  int64_t st = (tiles + ns - 1) / ns;
  if (st < 1) st = 1;
  ns = (tiles + st - 1) / st;
  if (ns < 1) ns = 1;
  *n_splits = (int)ns;
  *split_tiles = (int)st;
}

size_t decode_workspace_bytes(int batch, int n_q, int n_splits, int head_dim, int rank) {
  return (size_t)batch * n_q * n_splits * (4 + head_dim + rank) * sizeof(float);
}

hipError_t launch_decode(const AttnArgs& a, hipStream_t st) {
  if (a.head_dim == 64) return launch_r<64>(a, st);
  if (a.head_dim == 128) return launch_r<128>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace prc
