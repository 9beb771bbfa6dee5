// LR-cache precompute GEMM (PreLRShared, Sec. 3.1, Fig. 1 A1-A3), optionally
// joined with the base K/V projection of the same segment, gfx950.
//
// When a segment of T hidden states is first processed, every agent's LoRA
// down-projection is applied to it at once:
//     L[p][a][tok_offset + t][j] = sum_k X[t][k] * A_rows[(p*N + a)*r + j][k]
// i.e. one GEMM  X[T x d_in] . A_stack[d_in x n_cols]  whose n_cols = n_proj*N*r
// output columns are scattered into per-agent planes [s_cap][r].  With the
// base projection joined (Sec. 2.2 base cache), the same GEMM also produces
// K_base = RoPE(X W_k) and V_base = X W_v: X is read once for all of it.
//
// The kernel computes the transposed product C^T = rows . X^T, so both
// operands are rows contiguous along d_in.  Workgroup tile: TB columns x TB
// tokens (TB = 64 for the narrow LR-only GEMM, 128 for the wide joined one),
// 4 compute waves, each owning a TB/2 x TB/2 quarter on 32x32x16 MFMAs, and
// 8 loader waves (the per-CU load rate from L2 needs about 8 issuing waves).
// The operand tiles are staged in LDS, 32 KB per stage, in a ring of NST
// stages filled by direct global->LDS buffer loads: every load instruction
// brings whole 128- or 256-byte rows, so the texture path sees full cache
// lines and no VGPRs are spent on staging.  Inside a stage each row's 16-byte
// chunks are XOR-swizzled by the row index so that the MFMA fragment reads are
// free of bank conflicts.  Rows past the matrix and k past d_in read as zeros
// (buffer range check / out-of-range offsets).  The result layout gives each
// lane 4 consecutive output columns of one token: one 8-byte store.
// Block order is XCD-aware: the column tiles that share rows of X run on the
// same XCD, so X is fetched into each L2 once.
#include "common.hpp"
#include "kernels.hpp"

namespace prc {
namespace {

constexpr int NPW = 8;          // loader waves
constexpr int NCW = 4;          // compute waves
constexpr int NST = 4;          // stages in the LDS ring
constexpr int AHEAD = NST - 2;  // stages in flight beyond the one awaited
constexpr int NXCD = 8;         // XCDs of an MI355X

template <int TB>
struct Tile {
  static constexpr int KST = TB == 64 ? 128 : 64;  // k per stage: 2 x TB x KST x 2 B = 32 KB
  static constexpr int CPW = KST / 8;              // 16-byte chunks per row and stage
  static constexpr int RPI = 64 / CPW;             // rows per load instruction (1 KB)
  static constexpr int RPW = TB / NPW;             // rows of each tile per loader wave
  static constexpr int NI = RPW / RPI;             // load instructions per tile, wave and stage
  static constexpr int QB = TB / 64;               // 32x32 blocks per compute wave and dimension
  // Physical 16-byte chunk of logical chunk c in row r of a stage tile: the
  // 16 rows read together by one fragment load hit distinct banks (a 256-byte
  // row spans all 64 banks; two 128-byte rows share them).
  static __device__ __forceinline__ int swz(int r, int c) { return CPW == 16 ? c ^ (r & 15) : c ^ ((r >> 1) & 7); }
};

// s_waitcnt vmcnt(n) for a wave-uniform n in {0, 4, ..., 24}, other
// counters not waited on.  gfx9 encoding: vmcnt bits [3:0] and [15:14],
// expcnt [6:4] = 7, lgkmcnt [11:8] = 15.  The immediate must be a constant,
// so the cases are spelled out.
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
__device__ __forceinline__ void wait_vmcnt_le(int n) {
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

template <int TB>
__global__ void __launch_bounds__((NCW + NPW) * 64) precompute_kernel(const PrecomputeArgs a, int n_ct, int n_tt) {
  using C = Tile<TB>;
  constexpr int KST = C::KST, CPW = C::CPW, RPI = C::RPI, RPW = C::RPW, NI = C::NI, QB = C::QB;
  static_assert(2 * NI * AHEAD <= 24 && (2 * NI) % 4 == 0 && NI >= 1, "vmcnt cases");
  // [stage][weight tile, X tile][TB rows x KST]
  __shared__ __attribute__((aligned(1024))) uint16_t tiles[NST][2][TB * KST];
  // Waves 0..NCW-1 compute, the others fill the LDS ring, so loading and
  // computing overlap.
  const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool producer = wv >= NCW;
  const int w = producer ? wv - NCW : wv;
  // XCD-aware tile order: workgroup L runs on XCD L % 8; consecutive slots of
  // one XCD walk the column tiles of one token tile.
  const int L = blockIdx.x, xcd = L % NXCD, slot = L / NXCD;
  const int ct = slot % n_ct;
  const int tt = (slot / n_ct) * NXCD + xcd;
  if (tt >= n_tt) return;  // padding of the grid (uniform over the workgroup)
  const int col0 = ct * TB;
  const int64_t tok0 = (int64_t)tt * TB;
  // Column regions (tiles never straddle them: nkv is a multiple of TB):
  // keys, values, then LR columns.
  const int region = col0 < a.nkv ? 0 : (col0 < 2 * a.nkv ? 1 : 2);
  const int lcol0 = col0 - 2 * a.nkv;  // first LR column of an LR tile
  const int cols = region < 2 ? TB : (a.n_cols - lcol0 < TB ? a.n_cols - lcol0 : TB);  // valid weight rows
  const int toks = (int)(a.T - tok0 < TB ? a.T - tok0 : (int64_t)TB);  // valid rows of the X tile

  // Buffer resources over the valid rows of each operand tile (k included).
  // Key and value tiles read rows of W: a value tile rows col0 - nkv ..; a
  // key tile reorders the rows of its head so that every RoPE pair (dims j,
  // j + d/2) lands in one lane of the result: local column e of a head
  // (32-column block e / 32) holds dim (e / 32) * 16 + e % 16 + (e % 32 >= 16 ? d / 2 : 0).
  const i32x4 ra = region == 2
      ? buffer_rsrc(a.A + (int64_t)lcol0 * a.d_in, (int32_t)((cols - 1) * a.d_in * 2 + a.d_in * 2))
      : buffer_rsrc(a.W, (int32_t)(2 * a.nkv * a.d_in * 2));
  auto weight_row = [&](int row) -> int {  // row of the resource for local tile row `row`
    if (region == 2) return row;
    if (region == 1) return col0 + row;
    const int vc = col0 + row, hd = vc / a.head_dim, e = vc - hd * a.head_dim;
    return hd * a.head_dim + (e / 32) * 16 + (e % 16) + ((e % 32) / 16) * (a.head_dim / 2);
  };
  const i32x4 rx = buffer_rsrc(a.X + tok0 * a.ld_x, (int32_t)((toks - 1) * a.ld_x * 2 + a.d_in * 2));

  // Loader: each loader wave fills RPW of the TB rows of both tiles per
  // stage, NI instructions per tile, each writing 1 KB (RPI rows) at
  // consecutive lane positions.  Lane i of instruction j holds physical chunk
  // i % CPW of row RPW w + RPI j + i / CPW, i.e. logical chunk swz(row, i % CPW).
  int32_t offa[NI], offx[NI], kch[NI];
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const int row = RPW * w + RPI * j + lane / CPW;
    const int c = C::swz(row, lane % CPW);
    kch[j] = c * 8;  // first k of this lane's chunk within a stage
    offa[j] = weight_row(row) * (int32_t)(a.d_in * 2) + c * 16;
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
      lds_dma16(ra, &tiles[sl][0][(RPW * w + RPI * j) * KST], oa, k0 * 2);
      lds_dma16(rx, &tiles[sl][1][(RPW * w + RPI * j) * KST], ox, k0 * 2);
    }
  };

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

  // Compute: wave w owns columns (TB/2)(w & 1) .. and tokens (TB/2)(w >> 1) ..,
  // QB x QB blocks of 32 x 32.  32x32x16 fragments: lane l holds row l % 32,
  // k = (l / 32) * 8 + 0..7.
  const int l32 = lane & 31, h = lane >> 5;
  const int ra_row0 = (TB / 2) * (w & 1) + l32, rx_row0 = (TB / 2) * (w >> 1) + l32;
  // Cache row of each of the lane's tokens: its position tok_offset + t, or
  // its row in the paged pools.  The table is read here, so that its latency
  // hides behind the first stage's loads.
  int64_t srow[QB];
#pragma unroll
  for (int bt = 0; bt < QB; ++bt) {
    const int64_t t = tok0 + (TB / 2) * (w >> 1) + 32 * bt + l32;
    const int p = (int)(a.tok_offset + t);  // positions stay below 2^31
    srow[bt] = p;
    if (a.tbl != nullptr && t < a.T) {
      const int q = p / a.blk;
      int32_t e = a.tbl[q];
      e = e < 0 ? 0 : (e >= a.nblk ? a.nblk - 1 : e);
      srow[bt] = (int64_t)e * a.blk + (p - q * a.blk);
    }
  }
  f32x16 acc[QB][QB];
#pragma unroll
  for (int bc = 0; bc < QB; ++bc)
#pragma unroll
    for (int bt = 0; bt < QB; ++bt)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[bc][bt][j] = 0.f;
  for (int s = 0; s < nstage; ++s) {
    __syncthreads();  // stage s visible to all waves; stage s - 1 consumed by all
    const uint16_t* ta = tiles[s % NST][0];
    const uint16_t* tx = tiles[s % NST][1];
#pragma unroll
    for (int kk = 0; kk < KST / 16; ++kk) {
      const int c = 2 * kk + h;  // logical chunk of this lane's 8 k
      bf16x8 fa[QB], fx[QB];
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        const int ar = ra_row0 + 32 * b, xr = rx_row0 + 32 * b;
        fa[b] = as_bf16x8(*reinterpret_cast<const u32x4*>(ta + ar * KST + C::swz(ar, c) * 8));
        fx[b] = as_bf16x8(*reinterpret_cast<const u32x4*>(tx + xr * KST + C::swz(xr, c) * 8));
      }
#pragma unroll
      for (int bc = 0; bc < QB; ++bc)
#pragma unroll
        for (int bt = 0; bt < QB; ++bt) acc[bc][bt] = mfma32x32x16(fa[bc], fx[bt], acc[bc][bt]);
    }
  }

  // acc[bc][bt][j]: column (TB/2)(w & 1) + 32 bc + (j / 4) * 8 + h * 4 + j % 4,
  // token (TB/2)(w >> 1) + 32 bt + l32.
#pragma unroll
  for (int bt = 0; bt < QB; ++bt) {
    const int64_t t = tok0 + (TB / 2) * (w >> 1) + 32 * bt + l32;
    if (t >= a.T) continue;
    const int64_t trow = a.tok_offset + t;  // absolute position of the token
    const int64_t row = srow[bt];           // its cache row
#pragma unroll
    for (int bc = 0; bc < QB; ++bc) {
      const f32x16& r = acc[bc][bt];
      const int cb = col0 + (TB / 2) * (w & 1) + 32 * bc;  // first column of this 32-column block
      if (region == 0) {
        // Keys: registers j and j + 8 hold dims j0 + i and j0 + i + d/2 of one
        // head (the row order above); rotate-half RoPE at position trow.
#pragma unroll
        for (int jg = 0; jg < 2; ++jg) {
          const int vc = cb + jg * 8 + h * 4;
          const int hd = vc / a.head_dim, e = vc - hd * a.head_dim;
          const int j0 = (e / 32) * 16 + (e % 16);
          float lo[4], hi[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float cs, sn;
            rope_cs((int)trow, a.w2pi[j0 + i], cs, sn);
            const float x = r[4 * jg + i], y = r[4 * jg + 8 + i];
            lo[i] = x * cs - y * sn;
            hi[i] = y * cs + x * sn;
          }
          uint16_t* kp = a.Kout + row * a.nkv + hd * a.head_dim + j0;
          *reinterpret_cast<u32x2*>(kp) = u32x2{pack_bf16(lo[0], lo[1]), pack_bf16(lo[2], lo[3])};
          *reinterpret_cast<u32x2*>(kp + a.head_dim / 2) = u32x2{pack_bf16(hi[0], hi[1]), pack_bf16(hi[2], hi[3])};
        }
        continue;
      }
#pragma unroll
      for (int jg = 0; jg < 4; ++jg) {
        const int c = cb + jg * 8 + h * 4;
        u32x2 o;
        o[0] = pack_bf16(r[4 * jg + 0], r[4 * jg + 1]);
        o[1] = pack_bf16(r[4 * jg + 2], r[4 * jg + 3]);
        if (region == 1) {
          *reinterpret_cast<u32x2*>(a.Vout + row * a.nkv + (c - a.nkv)) = o;
        } else {
          const int lc = c - 2 * a.nkv;
          if (lc >= a.n_cols) continue;
          const int plane = lc / a.rank, jr = lc - plane * a.rank;
          *reinterpret_cast<u32x2*>(a.L + ((int64_t)plane * a.s_cap + row) * a.rank + jr) = o;
        }
      }
    }
  }
}

template <int TB>
hipError_t launch_tb(const PrecomputeArgs& a, hipStream_t st) {
  const int n_ct = 2 * a.nkv / TB + (a.n_cols + TB - 1) / TB;
  const int n_tt = (int)((a.T + TB - 1) / TB);
  const int groups = (n_tt + NXCD - 1) / NXCD;  // token tiles per XCD
  const int grid = groups * NXCD * n_ct;
  hipLaunchKernelGGL((precompute_kernel<TB>), dim3(grid), dim3((NCW + NPW) * 64), 0, st, a, n_ct, n_tt);
  return hipGetLastError();
}

// A handful of rows (the K/V and LR rows of newly decoded tokens) is a
// matrix-vector product: one workgroup per output column streams that
// column's row of W_rows or A_rows (contiguous along d_in; 4 waves x 64 lanes
// x 16 bytes = 4096 elements per step, so a 4096-wide row is one load per
// lane) against the T <= GV_T rows of X, which every workgroup reads from L2,
// then reduces over lanes and waves.  Key workgroups take the two rows of one
// RoPE pair (dims j and j + d/2 of a head) and rotate them at the token's
// position.  This spreads the weights over thousands of workgroups instead
// of the few tiles the GEMM would have, and keeps a whole row's loads in
// flight at once (the rows are usually cold in the decode loop).
constexpr int GV_T = 4;
constexpr int GV_W = 4;  // waves per column

__global__ void __launch_bounds__(64 * GV_W) project_gemv_kernel(const PrecomputeArgs a) {
  __shared__ float red[GV_W][2][GV_T];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int u = blockIdx.x;
  const int n_pair = a.nkv / 2;  // key RoPE pairs (nkv = n_kv * head_dim, 0 without K/V)
  const int half = a.head_dim / 2;
  // Region of this workgroup: 0 keys (a pair of rows), 1 values, 2 LR.
  int region, hd = 0, j = 0, c = 0;
  const uint16_t* r0;
  const uint16_t* r1 = nullptr;
  if (u < n_pair) {
    region = 0;
    hd = u / half;
    j = u - hd * half;
    r0 = a.W + (int64_t)(hd * a.head_dim + j) * a.d_in;
    r1 = r0 + (int64_t)half * a.d_in;
  } else if (u < n_pair + a.nkv) {
    region = 1;
    c = u - n_pair;
    r0 = a.W + (int64_t)(a.nkv + c) * a.d_in;
  } else {
    region = 2;
    c = u - n_pair - a.nkv;
    r0 = a.A + (int64_t)c * a.d_in;
  }
  const int T = (int)a.T;
  float acc0[GV_T] = {0.f, 0.f, 0.f, 0.f}, acc1[GV_T] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 2
  for (int64_t k = (int64_t)tid * 8; k < a.d_in; k += 64 * GV_W * 8) {
    const u32x4 av = *reinterpret_cast<const u32x4*>(r0 + k);
    const bool pair = region == 0;  // uniform over the workgroup
    u32x4 bv = {0u, 0u, 0u, 0u};
    if (pair) bv = *reinterpret_cast<const u32x4*>(r1 + k);
#pragma unroll
    for (int t = 0; t < GV_T; ++t) {
      if (t < T) {
        const u32x4 xv = *reinterpret_cast<const u32x4*>(a.X + t * a.ld_x + k);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc0[t] += bf_lo(av[e]) * bf_lo(xv[e]) + bf_hi(av[e]) * bf_hi(xv[e]);
        if (pair) {
#pragma unroll
          for (int e = 0; e < 4; ++e) acc1[t] += bf_lo(bv[e]) * bf_lo(xv[e]) + bf_hi(bv[e]) * bf_hi(xv[e]);
        }
      }
    }
  }
#pragma unroll
  for (int t = 0; t < GV_T; ++t) {
#pragma unroll
    for (int x = 1; x < 64; x <<= 1) {
      acc0[t] += shfl_xor(acc0[t], x);
      acc1[t] += shfl_xor(acc1[t], x);
    }
    if (lane == 0) {
      red[w][0][t] = acc0[t];
      red[w][1][t] = acc1[t];
    }
  }
  __syncthreads();
  if (tid < T) {
    float x = 0.f, y = 0.f;
#pragma unroll
    for (int i = 0; i < GV_W; ++i) {
      x += red[i][0][tid];
      y += red[i][1][tid];
    }
    const int64_t row = a.tok_offset + tid;  // absolute position and cache row
    if (region == 0) {
      float cs, sn;
      rope_cs((int)row, a.w2pi[j], cs, sn);
      uint16_t* kp = a.Kout + row * a.nkv + hd * a.head_dim + j;
      kp[0] = (uint16_t)(pack_bf16(x * cs - y * sn, 0.f) & 0xffffu);
      kp[half] = (uint16_t)(pack_bf16(y * cs + x * sn, 0.f) & 0xffffu);
    } else if (region == 1) {
      a.Vout[row * a.nkv + c] = (uint16_t)(pack_bf16(x, 0.f) & 0xffffu);
    } else {
      const int64_t plane = c / a.rank, jr = c - plane * a.rank;
      a.L[(plane * a.s_cap + row) * a.rank + jr] = (uint16_t)(pack_bf16(x, 0.f) & 0xffffu);
    }
  }
}

}  // namespace

hipError_t launch_precompute(const PrecomputeArgs& a, hipStream_t st) {
  if (a.tbl == nullptr && a.T <= GV_T) {
    hipLaunchKernelGGL(project_gemv_kernel, dim3(a.nkv / 2 + a.nkv + a.n_cols), dim3(64 * GV_W), 0, st, a);
    return hipGetLastError();
  }
  // 128-wide tiles halve the bytes loaded per MFMA but need enough of them to
  // fill the 256 CUs; the K/V boundary must fall on a tile edge.
  const int64_t wide = (int64_t)((2 * a.nkv + a.n_cols + 127) / 128) * ((a.T + 127) / 128);
  if (a.nkv % 128 == 0 && wide >= 256) return launch_tb<128>(a, st);
  return launch_tb<64>(a, st);
}

}  // namespace prc
