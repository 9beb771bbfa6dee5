// LR-cache precompute GEMM (PreLRShared, Sec. 3.1, Fig. 1 A1-A3), gfx950.
//
// When a segment of T hidden states is first processed, every agent's LoRA
// down-projection is applied to it at once:
//     L[p][a][tok_offset + t][j] = sum_k X[t][k] * A_rows[(p*N + a)*r + j][k]
// i.e. one GEMM  X[T x d_in] . A_stack[d_in x n_cols]  whose n_cols = n_proj*N*r
// output columns are scattered into per-agent planes [s_cap][r].
//
// Both operands are contiguous along d_in (A is stored as rows), so MFMA
// fragments are read straight from global memory in operand layout.  The
// kernel computes the transposed product C^T = A_rows . X^T with 16x16x32 bf16
// MFMAs: the result layout gives each lane 4 consecutive output columns of one
// token, i.e. 4 consecutive rank entries of one plane row (an 8-byte store).
//
// Workgroup tile: 64 columns x 64 tokens.  Each of the 4 waves computes the
// whole tile over a quarter of d_in (16 MFMAs per 8 fragment loads, loads of
// the next k-step in flight), and the partial tiles are summed through LDS.
// Block order is XCD-aware: the column tiles that share rows of X run on the
// same XCD, so X is fetched into each L2 once.
#include "common.hpp"
#include "kernels.hpp"

namespace prc {
namespace {

constexpr int TC = 64;  // output columns per workgroup
constexpr int TT = 64;  // tokens per workgroup
constexpr int KS = 32;  // k per MFMA
constexpr int NXCD = 8; // XCDs of an MI355X

struct Frag {
  u32x4 a[4];  // A rows: columns 16i + l%16, k chunk (l/16)*8
  u32x4 x[4];  // X rows: tokens 16j + l%16, same k chunk
};

__global__ void __launch_bounds__(256)
precompute_kernel(const PrecomputeArgs a, int n_ct, int n_tt) {
  __shared__ __attribute__((aligned(16))) float red[3][TC * TT];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c16 = lane & 15, q = lane >> 4;
  // XCD-aware tile order: workgroup L runs on XCD L % 8; consecutive slots of
  // one XCD walk the column tiles of one token tile.
  const int L = blockIdx.x, xcd = L % NXCD, slot = L / NXCD;
  const int ct = slot % n_ct;
  const int tt = (slot / n_ct) * NXCD + xcd;
  if (tt >= n_tt) return;  // padding of the grid (uniform over the workgroup)
  const int col0 = ct * TC;
  const int64_t tok0 = (int64_t)tt * TT;

  const uint16_t* ap[4];
  const uint16_t* xp[4];
  bool aok[4], xok[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = col0 + i * 16 + c16;
    aok[i] = c < a.n_cols;
    ap[i] = a.A + (int64_t)(aok[i] ? c : 0) * a.d_in + q * 8;
    const int64_t t = tok0 + i * 16 + c16;
    xok[i] = t < a.T;
    xp[i] = a.X + (xok[i] ? t : 0) * a.ld_x + q * 8;
  }
  // This wave's share of d_in, in whole k-steps of 32.
  const int64_t nk = (a.d_in + KS - 1) / KS;
  const int64_t k_begin = (nk * w / 4) * KS, k_end = (nk * (w + 1) / 4) * KS;

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load = [&](Frag& f, int64_t k0) {
    const bool kok = k0 + q * 8 < a.d_in;  // d_in is a multiple of 8
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f.a[i] = ld16(ap[i] + k0, aok[i] && kok);
      f.x[i] = ld16(xp[i] + k0, xok[i] && kok);
    }
  };
  auto mma = [&](const Frag& f) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x32(as_bf16x8(f.a[i]), as_bf16x8(f.x[j]), acc[i][j]);
  };

  Frag f0, f1;
  int64_t k0 = k_begin;
  if (k0 < k_end) load(f0, k0);
  for (; k0 + 2 * KS <= k_end; k0 += 2 * KS) {
    load(f1, k0 + KS);
    mma(f0);
    if (k0 + 2 * KS < k_end) load(f0, k0 + 2 * KS);
    mma(f1);
  }
  if (k0 < k_end) mma(f0);

  // Sum the 4 partial tiles: waves 1-3 park theirs in LDS, wave 0 adds them.
  // acc[i][j][e]: column col0 + 16i + 4q + e, token tok0 + 16j + l%16.
  if (w > 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<f32x4*>(&red[w - 1][((i * 4 + j) * 64 + lane) * 4]) = acc[i][j];
  }
  __syncthreads();
  if (w > 0) return;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = col0 + i * 16 + q * 4;
    const int plane = c / a.rank, jr = c - plane * a.rank;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f32x4 v = acc[i][j];
#pragma unroll
      for (int p = 0; p < 3; ++p) v += *reinterpret_cast<const f32x4*>(&red[p][((i * 4 + j) * 64 + lane) * 4]);
      const int64_t t = tok0 + j * 16 + c16;
      if (c >= a.n_cols || t >= a.T) continue;
      u32x2 o;
      o[0] = pack_bf16(v[0], v[1]);
      o[1] = pack_bf16(v[2], v[3]);
      *reinterpret_cast<u32x2*>(a.L + ((int64_t)plane * a.s_cap + a.tok_offset + t) * a.rank + jr) = o;
    }
  }
}

}  // namespace

hipError_t launch_precompute(const PrecomputeArgs& a, hipStream_t st) {
  const int n_ct = (a.n_cols + TC - 1) / TC;
  const int n_tt = (int)((a.T + TT - 1) / TT);
  const int groups = (n_tt + NXCD - 1) / NXCD;  // token tiles per XCD
  const int grid = groups * NXCD * n_ct;
  hipLaunchKernelGGL(precompute_kernel, dim3(grid), dim3(256), 0, st, a, n_ct, n_tt);
  return hipGetLastError();
}

}  // namespace prc
