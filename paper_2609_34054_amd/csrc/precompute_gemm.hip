// LR-cache precompute GEMM (PreLRShared, Sec. 3.1, Fig. 1 A1-A3), gfx950.
//
// When a segment of T hidden states is first processed, every agent's LoRA
// down-projection is applied to it at once:
//     L[p][a][tok_offset + t][j] = sum_k X[t][k] * A_rows[(p*N + a)*r + j][k]
// i.e. one GEMM  X[T x d_in] . A_stack[d_in x n_cols]  whose n_cols = n_proj*N*r
// output columns are scattered into per-agent planes [s_cap][r].
//
// The kernel computes the transposed product C^T = A_rows . X^T, so both
// operands are rows contiguous along d_in.  Workgroup tile: 64 columns x 64
// tokens, 4 waves, each owning a 32 x 32 quadrant on 32x32x16 MFMAs.  The
// operand tiles are staged in LDS, 64 k (128 bytes per row) per stage, in a
// ring of NST stages filled by direct global->LDS buffer loads: every load
// instruction brings 8 whole 128-byte rows, so the texture path sees full
// cache lines and no VGPRs are spent on staging.  Inside a stage each row's
// eight 16-byte chunks are XOR-swizzled by the row index so that the MFMA
// fragment reads are free of bank conflicts.  Rows past the matrix and k past
// d_in read as zeros (buffer range check / out-of-range offsets).  The result
// layout gives each lane 4 consecutive output columns of one token: 4
// consecutive rank entries of one plane row, one 8-byte store.
// Block order is XCD-aware: the column tiles that share rows of X run on the
// same XCD, so X is fetched into each L2 once.
#include "common.hpp"
#include "kernels.hpp"

namespace prc {
namespace {

constexpr int TC = 64;   // output columns per workgroup
constexpr int TT = 64;   // tokens per workgroup
constexpr int KST = 128;        // k per stage (256 bytes of a row)
constexpr int CPW = KST / 8;    // 16-byte chunks per row and stage
constexpr int RPI = 64 / CPW;   // rows per load instruction (1 KB)
constexpr int NI = 16 / RPI;    // load instructions per operand, wave and stage
constexpr int NST = 4;          // stages in the LDS ring
constexpr int AHEAD = NST - 2;  // stages in flight beyond the one awaited
constexpr int NXCD = 8;  // XCDs of an MI355X

// Physical 16-byte chunk of logical chunk c in row r of a stage tile.  A row
// of a stage spans all 64 banks (256 bytes); the XOR with r % 16 makes the 16
// rows read together by one fragment load hit distinct banks.
__device__ __forceinline__ int swz(int r, int c) { return c ^ (r & 15); }
static_assert(CPW == 16, "swizzle written for 256-byte stage rows");

// s_waitcnt vmcnt(n) for a wave-uniform n in {0, 4, ..., 24}, other
// counters not waited on.  gfx9 encoding: vmcnt bits [3:0] and [15:14],
// expcnt [6:4] = 7, lgkmcnt [11:8] = 15.  The immediate must be a constant,
// so the cases are spelled out.
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
__device__ __forceinline__ void wait_vmcnt_le(int n) {
  static_assert(2 * NI * AHEAD <= 24 && (2 * NI) % 4 == 0, "vmcnt cases");
  switch (n) {
    case 24: __builtin_amdgcn_s_waitcnt(vmcnt_imm(24)); break;
    case 20: __builtin_amdgcn_s_waitcnt(vmcnt_imm(20)); break;
    case 16: __builtin_amdgcn_s_waitcnt(vmcnt_imm(16)); break;
    case 12: __builtin_amdgcn_s_waitcnt(vmcnt_imm(12)); break;
    case 8: __builtin_amdgcn_s_waitcnt(vmcnt_imm(8)); break;
    case 4: __builtin_amdgcn_s_waitcnt(vmcnt_imm(4)); break;
    default: __builtin_amdgcn_s_waitcnt(vmcnt_imm(0)); break;
  }
}

__global__ void __launch_bounds__(512) precompute_kernel(const PrecomputeArgs a, int n_ct, int n_tt) {
  // [stage][A tile, X tile][64 rows x 128 bytes]
  __shared__ __attribute__((aligned(1024))) uint16_t tiles[NST][2][64 * KST];
  // Waves 0-3 compute, waves 4-7 fill the LDS ring: issuing a stage's loads
  // costs about as long as computing one, and the two now overlap.
  const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool producer = wv >= 4;
  const int w = wv & 3;
  // XCD-aware tile order: workgroup L runs on XCD L % 8; consecutive slots of
  // one XCD walk the column tiles of one token tile.
  const int L = blockIdx.x, xcd = L % NXCD, slot = L / NXCD;
  const int ct = slot % n_ct;
  const int tt = (slot / n_ct) * NXCD + xcd;
  if (tt >= n_tt) return;  // padding of the grid (uniform over the workgroup)
  const int col0 = ct * TC;
  const int64_t tok0 = (int64_t)tt * TT;
  const int cols = a.n_cols - col0 < TC ? a.n_cols - col0 : TC;          // valid rows of the A tile
  const int toks = (int)(a.T - tok0 < TT ? a.T - tok0 : (int64_t)TT);    // valid rows of the X tile

  // Buffer resources over the valid rows of each operand tile (k included).
  const i32x4 ra = buffer_rsrc(a.A + (int64_t)col0 * a.d_in, (int32_t)((cols - 1) * a.d_in * 2 + a.d_in * 2));
  const i32x4 rx = buffer_rsrc(a.X + tok0 * a.ld_x, (int32_t)((toks - 1) * a.ld_x * 2 + a.d_in * 2));

  // Loader: each producer wave fills 16 of the 64 rows of both tiles per
  // stage, NI instructions per tile, each writing 1 KB (RPI rows) at
  // consecutive lane positions.  Lane i of instruction j holds physical chunk
  // i % CPW of row 16 w + RPI j + i / CPW, i.e. logical chunk swz(row, i % CPW).
  int32_t offa[NI], offx[NI], kch[NI];
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const int row = 16 * w + RPI * j + lane / CPW;
    const int c = swz(row, lane % CPW);
    kch[j] = c * 8;  // first k of this lane's chunk within a stage
    offa[j] = row * (int32_t)(a.d_in * 2) + c * 16;
    offx[j] = row * (int32_t)(a.ld_x * 2) + c * 16;
  }
  const int nstage = (int)((a.d_in + KST - 1) / KST);
  // Each token tile walks the k stages from its own starting point (the
  // column tiles that share its X rows use the same one), so that at any
  // moment the workgroups read rows at different k offsets: with row strides
  // that are multiples of 4 KB, equal offsets would all hit the same few L2
  // channels.
  const int rot = (int)(((int64_t)tt * nstage) / n_tt);
  auto issue = [&](int s) {
    const int sl = s % NST;
    const int ks = s + rot < nstage ? s + rot : s + rot - nstage;
    const int32_t k0 = ks * KST;
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      // Chunks wholly past d_in (d_in is a multiple of 8) read as zeros.
      const bool kok = k0 + kch[j] < a.d_in;
      const int32_t oa = kok ? offa[j] : INT32_MIN, ox = kok ? offx[j] : INT32_MIN;
      lds_dma16(ra, &tiles[sl][0][(16 * w + RPI * j) * KST], oa, k0 * 2);
      lds_dma16(rx, &tiles[sl][1][(16 * w + RPI * j) * KST], ox, k0 * 2);
    }
  };

  // Compute: wave w owns columns 32 (w & 1) .. +31 and tokens 32 (w >> 1) .. +31.
  // 32x32x16 fragments: lane l holds row l % 32, k = (l / 32) * 8 + 0..7.
  const int l32 = lane & 31, h = lane >> 5;
  const int ra_row = 32 * (w & 1) + l32, rx_row = 32 * (w >> 1) + l32;
  f32x16 acc;
#pragma unroll
  for (int j = 0; j < 16; ++j) acc[j] = 0.f;

  if (producer) {
    // Stage s + AHEAD goes into the slot of stage s - 2, which the compute
    // waves finished before the previous barrier, so it is issued before
    // waiting for stage s: issuing overlaps the wait.
#pragma unroll
    for (int s = 0; s < AHEAD; ++s)
      if (s < nstage) issue(s);
    for (int s = 0; s < nstage; ++s) {
      if (s + AHEAD < nstage) issue(s + AHEAD);
      // Stage s has landed once at most the loads of the stages after it (up
      // to AHEAD of them, 2 NI instructions each) are still in flight.
      const int ahead = nstage - 1 - s < AHEAD ? nstage - 1 - s : AHEAD;
      wait_vmcnt_le(2 * NI * ahead);
      __syncthreads();  // stage s visible to all waves
    }
    return;
  }
  for (int s = 0; s < nstage; ++s) {
    __syncthreads();  // stage s visible to all waves; stage s - 1 consumed by all
    const uint16_t* ta = tiles[s % NST][0] + ra_row * KST;
    const uint16_t* tx = tiles[s % NST][1] + rx_row * KST;
#pragma unroll
    for (int kk = 0; kk < KST / 16; ++kk) {
      const int c = 2 * kk + h;  // logical chunk of this lane's 8 k
      const u32x4 fa = *reinterpret_cast<const u32x4*>(ta + swz(ra_row, c) * 8);
      const u32x4 fx = *reinterpret_cast<const u32x4*>(tx + swz(rx_row, c) * 8);
      acc = mfma32x32x16(as_bf16x8(fa), as_bf16x8(fx), acc);
    }
  }

  // acc[j]: column 32 (w & 1) + (j / 4) * 8 + h * 4 + j % 4, token 32 (w >> 1) + l32.
  const int64_t t = tok0 + 32 * (w >> 1) + l32;
  if (t >= a.T) return;
#pragma unroll
  for (int jg = 0; jg < 4; ++jg) {
    const int c = col0 + 32 * (w & 1) + jg * 8 + h * 4;
    if (c >= a.n_cols) continue;
    const int plane = c / a.rank, jr = c - plane * a.rank;
    u32x2 o;
    o[0] = pack_bf16(acc[4 * jg + 0], acc[4 * jg + 1]);
    o[1] = pack_bf16(acc[4 * jg + 2], acc[4 * jg + 3]);
    *reinterpret_cast<u32x2*>(a.L + ((int64_t)plane * a.s_cap + a.tok_offset + t) * a.rank + jr) = o;
  }
}

}  // namespace

hipError_t launch_precompute(const PrecomputeArgs& a, hipStream_t st) {
  const int n_ct = (a.n_cols + TC - 1) / TC;
  const int n_tt = (int)((a.T + TT - 1) / TT);
  const int groups = (n_tt + NXCD - 1) / NXCD;  // token tiles per XCD
  const int grid = groups * NXCD * n_ct;
  hipLaunchKernelGGL(precompute_kernel, dim3(grid), dim3(512), 0, st, a, n_ct, n_tt);
  return hipGetLastError();
}

}  // namespace prc
