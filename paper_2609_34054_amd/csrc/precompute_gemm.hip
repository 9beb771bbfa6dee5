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
// Workgroup tile: 64 columns x 64 tokens, 4 waves of 32 x 32.  Each wave
// double-issues two 32-wide k-steps per iteration.
#include "common.hpp"
#include "kernels.hpp"

namespace prc {
namespace {

constexpr int TC = 64;  // output columns per workgroup
constexpr int TT = 64;  // tokens per workgroup
constexpr int KS = 32;  // k per MFMA

__global__ void __launch_bounds__(256)
precompute_kernel(const PrecomputeArgs a) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c16 = lane & 15, q = lane >> 4;
  const int col0 = blockIdx.y * TC + (w >> 1) * 32;
  const int64_t tok0 = (int64_t)blockIdx.x * TT + (w & 1) * 32;

  // Operand rows this lane feeds: A rows (columns of the product) and X rows.
  const uint16_t* ap[2];
  const uint16_t* xp[2];
  bool aok[2], xok[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = col0 + i * 16 + c16;
    aok[i] = c < a.n_cols;
    ap[i] = a.A + (int64_t)(aok[i] ? c : 0) * a.d_in + q * 8;
    const int64_t t = tok0 + i * 16 + c16;
    xok[i] = t < a.T;
    xp[i] = a.X + (xok[i] ? t : 0) * a.ld_x + q * 8;
  }

  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // k chunk [k0 + q*8, +8) of this lane is valid iff k0 + q*8 < d_in
  // (d_in is a multiple of 8).
  int64_t k0 = 0;
  for (; k0 + 2 * KS <= a.d_in; k0 += 2 * KS) {
    u32x4 av[2][2], xv[2][2];
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        av[s][i] = ld16(ap[i] + k0 + s * KS, aok[i]);
        xv[s][i] = ld16(xp[i] + k0 + s * KS, xok[i]);
      }
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = mfma16x16x32(as_bf16x8(av[s][i]), as_bf16x8(xv[s][j]), acc[i][j]);
  }
  for (; k0 < a.d_in; k0 += KS) {
    const bool kok = k0 + q * 8 < a.d_in;
    u32x4 av[2], xv[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      av[i] = ld16(ap[i] + k0, aok[i] && kok);
      xv[i] = ld16(xp[i] + k0, xok[i] && kok);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = mfma16x16x32(as_bf16x8(av[i]), as_bf16x8(xv[j]), acc[i][j]);
  }

  // acc[i][j][e]: column col0 + 16i + 4q + e, token tok0 + 16j + l%16.
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = col0 + i * 16 + q * 4;
    if (c >= a.n_cols) continue;
    const int plane = c / a.rank, jr = c - plane * a.rank;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t t = tok0 + j * 16 + c16;
      if (t >= a.T) continue;
      u32x2 o;
      o[0] = pack_bf16(acc[i][j][0], acc[i][j][1]);
      o[1] = pack_bf16(acc[i][j][2], acc[i][j][3]);
      *reinterpret_cast<u32x2*>(a.L + ((int64_t)plane * a.s_cap + a.tok_offset + t) * a.rank + jr) = o;
    }
  }
}

}  // namespace

hipError_t launch_precompute(const PrecomputeArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((a.T + TT - 1) / TT), (unsigned)((a.n_cols + TC - 1) / TC));
  hipLaunchKernelGGL(precompute_kernel, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace prc
