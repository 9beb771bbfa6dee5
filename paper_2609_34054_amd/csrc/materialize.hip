// Reference point: materialise each request's full per-agent K/V, gfx950.
//
//     K_full[t] = K_base[t] + RoPE(L_k[t] B_k, t),    V_full[t] = V_base[t] + L_v[t] B_v
//
// These are the keys and values an agent that keeps its own full KV cache
// would hold (NonShared/BaseShared, Sec. 3.1).  Plain attention over them (an
// lr_shared_attention call with no LR cache) is the "materialise, then
// attend" path that the fused kernels avoid.
//
// One workgroup per (64 tokens, group of up to 8 KV heads, request); one wave
// per KV head, which loads its head's up-projection fragments once and then
// rebuilds the 64 tokens 16 at a time.  The 64 x d/2 RoPE table of the tile is
// built once in LDS and shared by the waves; the rebuild itself is the same
// on-chip code the attention kernels use.
#include "common.hpp"
#include "kernels.hpp"
#include "rebuild.hpp"

namespace prc {
namespace {

constexpr int MT = 64;    // tokens per workgroup
constexpr int SBT = 16;   // tokens per rebuild step of a wave
constexpr int MAXW = 8;   // KV heads per workgroup

template <int D, int R>
__global__ void __launch_bounds__(512)
materialize_kernel(const AttnArgs a) {
  constexpr int HALF = D / 2, NB = D / 32, QPG = D / 8, CS_ROW = HALF + 2;
  __shared__ float2 cs_lds[MT * CS_ROW];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c16 = lane & 15, q = lane >> 4;
  const int b = blockIdx.z, g = blockIdx.y * MAXW + w;
  const int64_t t0 = (int64_t)blockIdx.x * MT;
  const bool has_lk = a.Lk != nullptr, has_lv = a.Lv != nullptr;

  int64_t kvl = a.kv_len[b];
  kvl = kvl < 0 ? 0 : (kvl > a.s_cap ? a.s_cap : kvl);
  if (t0 >= kvl) return;  // uniform over the workgroup

  if (has_lk) {
    for (int e = tid; e < MT * HALF; e += blockDim.x) {
      const int tok = e / HALF, j = e - tok * HALF;
      float c, s;
      rope_cs((int)(t0 + tok), a.w2pi[j], c, s);
      cs_lds[tok * CS_ROW + j] = make_float2(c, s);
    }
  }
  __syncthreads();
  if (g >= a.n_kv) return;

  // Up-projections [r, n_kv*d] (Eq. 1 orientation): this head's columns.
  const int64_t boff = (int64_t)b * a.b_stride + (int64_t)g * D, ldb = (int64_t)a.n_kv * D;
  typename Ex<R>::Frag bk[D / 16][Ex<R>::NC], bv[D / 16][Ex<R>::NC];
  if (has_lk) load_bt_frags<D, R>(bk, a.Bk + boff, ldb, true, lane);
  if (has_lv) load_bt_frags<D, R>(bv, a.Bv + boff, ldb, true, lane);

  for (int sb = 0; sb < MT / SBT; ++sb) {
    const int64_t t = t0 + sb * SBT + c16;
    if (t0 + sb * SBT >= kvl) break;  // uniform over the wave
    const bool ok = t < kvl;
    const int64_t in_off = (int64_t)b * a.kv_stride + (t * a.n_kv + g) * D;
    const int64_t out_off = ((int64_t)b * a.s_cap * a.n_kv + t * a.n_kv + g) * D;
    u32x4 x[D / 32];
    load_chunks<D>(x, a.Kb + in_off, ok, lane);
    if (has_lk) {
      typename Ex<R>::Frag l[Ex<R>::NC];
      load_lr_frag<R>(l, a.Lk + (int64_t)b * a.l_stride + t * R, ok, lane);
      const float2* csr = cs_lds + (sb * SBT + c16) * CS_ROW + q * QPG;
      float cc[NB][4], ss[NB][4];
#pragma unroll
      for (int blk = 0; blk < NB; ++blk)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          cc[blk][i] = csr[blk * 4 + i].x;
          ss[blk][i] = csr[blk * 4 + i].y;
        }
      add_rotated_expansion<D, R>(x, bk, l, cc, ss);
    }
    if (ok) store_chunks<D>(a.Kout + out_off, x, lane);

    load_chunks<D>(x, a.Vb + in_off, ok, lane);
    if (has_lv) {
      typename Ex<R>::Frag l[Ex<R>::NC];
      load_lr_frag<R>(l, a.Lv + (int64_t)b * a.l_stride + t * R, ok, lane);
      add_expansion<D, R>(x, bv, l);
    }
    if (ok) store_chunks<D>(a.Vout + out_off, x, lane);
  }
}

template <int D, int R>
hipError_t launch_t(const AttnArgs& a, hipStream_t st) {
  const int hg = (a.n_kv + MAXW - 1) / MAXW;
  const int waves = a.n_kv < MAXW ? a.n_kv : MAXW;
  const dim3 grid((unsigned)((a.s_cap + MT - 1) / MT), hg, a.batch);
  hipLaunchKernelGGL((materialize_kernel<D, R>), grid, dim3(64 * waves), 0, st, a);
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

hipError_t launch_materialize(const AttnArgs& a, hipStream_t st) {
  if (a.head_dim == 64) return launch_r<64>(a, st);
  if (a.head_dim == 128) return launch_r<128>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace prc
