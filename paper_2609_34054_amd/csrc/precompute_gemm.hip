// LR-cache precompute GEMM (PreLRShared, Sec. 3.1, Fig. 1 A1-A3), optionally
// joined with the base K/V projection of the same segment, gfx950.
//
// When a segment of T hidden states is first processed, every agent's LoRA
// down-projection is applied to it at once:
//     L[p][a][tok_offset + t][j] = sum_k X[t][k] * A_stack[k][(p*N + a)*r + j]
// i.e. one GEMM  X[T x d_in] . A_stack[d_in x n_cols]  whose n_cols = n_proj*N*r
// output columns are scattered into per-agent planes [s_cap][r].  With the
// base projection joined (Sec. 2.2 base cache), the same GEMM also produces
// K_base = RoPE(X W_k) and V_base = X W_v: X is read once for all of it.
// The weights come in the orientation of Eq. 1, [d_in, d_out] row-major.
//
// The kernel computes the transposed product C^T = W^T X^T.  X tiles are
// staged in LDS k-contiguous, so each lane's B fragment (8 consecutive k of
// one token) is one 16-byte read.  Weight tiles are staged as they lie in
// memory, k rows of output columns, and the A fragments (8 consecutive k of
// one column) come out of the transposing LDS read ds_read_b64_tr_b16 (two
// per fragment).  A workgroup owns TB columns x TB tokens and has 4 compute
// waves, each accumulating a 64 x 64 block on 32x32x16 MFMAs (four 16-byte
// fragment reads per four MFMAs), and 8 loader waves filling a 4-stage ring of
// 32 KB stages with direct global->LDS buffer loads.  For the narrow LR-only
// GEMM (TB = 64) the four compute waves split every stage's k steps between
// them and sum their 64 x 64 partials through LDS at the end, in a fixed
// order; for the wide joined GEMM (TB = 128) each owns a quarter of the tile.
// Inside a stage, 16-byte chunks are XOR-swizzled by row so that both kinds
// of fragment read are free of bank conflicts; with direct-to-LDS loads the
// swizzle is applied by choosing which global chunk each lane fetches.
// Tokens past T, k past d_in and LR columns past n_cols read as zeros.  The
// result layout gives each lane 4 consecutive output columns of one token: one
// 8-byte store.  Block order is XCD-aware: the column tiles that share rows of
// X run on the same XCD, so X is fetched into each L2 once.
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
  static constexpr bool SPLITK = TB == 64;        // compute waves split k (narrow GEMM)
  static constexpr int KST = TB == 64 ? 128 : 64;  // k per stage: 2 x TB x KST x 2 B = 32 KB
  // X tile: TB token rows of KST k (XCPR 16-byte chunks per row).
  static constexpr int XCPR = KST / 8;
  static constexpr int XRPI = 64 / XCPR;           // rows per load instruction (1 KB)
  static constexpr int XRPW = TB / NPW;            // rows per loader wave
  static constexpr int NIX = XRPW / XRPI;          // X load instructions per wave and stage
  // Weight tile: KST k rows of TB columns (WCPR chunks per row).
  static constexpr int WCPR = TB / 8;
  static constexpr int WRPI = 64 / WCPR;
  static constexpr int WRPW = KST / NPW;
  static constexpr int NIW = WRPW / WRPI;
  // Physical chunk of logical chunk c in row r.  X rows: the 16 rows one
  // fragment read touches hit distinct banks.  Weight rows: the 4 k rows x 64
  // bytes a half-wave of transposing reads touches hit distinct banks.
  static __device__ __forceinline__ int swx(int r, int c) { return XCPR == 16 ? c ^ (r & 15) : c ^ ((r >> 1) & 7); }
  static __device__ __forceinline__ int sww(int r, int c) {
    return WCPR == 8 ? c ^ (((r >> 1) & 1) << 2) : c ^ ((r & 3) << 2);
  }
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

// Transposing LDS read of 4 bf16 per lane: lane j of each 16-lane group
// points at 4 consecutive bf16; lane i receives element i%4 of lanes i/4,
// i/4+4, i/4+8, i/4+12 of its group.
__device__ __forceinline__ u32x2 lds_read_tr(const uint16_t* p) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((v4s __attribute__((address_space(3)))*)(p));
  return __builtin_bit_cast(u32x2, v);
}

// First W column (within the [d_in, 2 nkv] key/value weights) of the 8
// output columns starting at key column vc (a multiple of 8).  Key tiles
// permute the columns of each head so that every RoPE pair (dims j and
// j + d/2) lands in one lane of the result: local column e of a head (32-column
// block e / 32) holds dim (e / 32) * 16 + e % 16 + (e % 32 >= 16 ? d / 2 : 0).
__device__ __forceinline__ int key_wcol(int vc, int head_dim) {
  const int hd = vc / head_dim, e = vc - hd * head_dim;
  return hd * head_dim + (e / 32) * 16 + (e % 16) + ((e % 32) / 16) * (head_dim / 2);
}

// Writes one 32 x 32 block of C^T in the 32x32x16 result layout: r[j] is
// output column cb + (j / 4) * 8 + h * 4 + j % 4 of token t (h = lane / 32).
// Keys are rotated at the token's position as they are written; every token
// goes to its cache row (its position, or its row in the paged pools).
__device__ __forceinline__ void store_block(const PrecomputeArgs& a, const f32x16& r, int region, int cb, int64_t t,
                                            int h) {
  if (t >= a.T) return;
  const int64_t trow = a.tok_offset + t;  // absolute position of the token
  int64_t row = trow;
  if (a.tbl != nullptr) {
    const int q = (int)(trow / a.blk);
    int32_t e = a.tbl[q];
    e = e < 0 ? 0 : (e >= a.nblk ? a.nblk - 1 : e);
    row = (int64_t)e * a.blk + (trow - (int64_t)q * a.blk);
  }
  if (region == 0) {
    // Keys: registers j and j + 8 hold dims j0 + i and j0 + i + d/2 of one
    // head (the column order of key tiles); rotate-half RoPE at position trow.
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
    return;
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

template <int TB>
__global__ void __launch_bounds__((NCW + NPW) * 64) precompute_kernel(const PrecomputeArgs a, int n_ct, int n_tt) {
  using C = Tile<TB>;
  constexpr int KST = C::KST;
  static_assert((C::NIX + C::NIW) * AHEAD <= 24 && (C::NIX + C::NIW) % 2 == 0 && C::NIX >= 1 && C::NIW >= 1,
                "vmcnt cases");
  static_assert(NST * 2 * TB * KST * 2 >= NCW * 4 * 16 * 64 * 4, "ring holds the split-k partials");
  static_assert(!C::SPLITK || (KST / 16) % NCW == 0, "k steps per stage split evenly");
  // [stage][X tile, weight tile][TB x KST]
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
  const int cols = region < 2 ? TB : (a.n_cols - lcol0 < TB ? a.n_cols - lcol0 : TB);  // valid columns
  const int toks = (int)(a.T - tok0 < TB ? a.T - tok0 : (int64_t)TB);  // valid rows of the X tile
  const int64_t ldw = region < 2 ? 2 * (int64_t)a.nkv : (int64_t)a.n_cols;  // weight row stride (elements)
  const i32x4 rw = buffer_rsrc(region < 2 ? a.W : a.A, (int32_t)(a.d_in * ldw * 2));
  const i32x4 rx = buffer_rsrc(a.X + tok0 * a.ld_x, (int32_t)((toks - 1) * a.ld_x * 2 + a.d_in * 2));

  // Loader: each instruction writes 1 KB (whole rows) at consecutive LDS
  // positions.  Lane i of an X instruction holds physical chunk i % XCPR of
  // token row XRPW w + XRPI j + i / XCPR, i.e. logical chunk swx(row, i % XCPR);
  // lane i of a weight instruction physical chunk i % WCPR of k row
  // WRPW w + WRPI j + i / WCPR.
  int32_t offx[C::NIX], kch[C::NIX], offw[C::NIW], krow[C::NIW];
#pragma unroll
  for (int j = 0; j < C::NIX; ++j) {
    const int row = C::XRPW * w + C::XRPI * j + lane / C::XCPR;
    const int c = C::swx(row, lane % C::XCPR);
    kch[j] = c * 8;  // first k of this lane's chunk within a stage
    offx[j] = row * (int32_t)(a.ld_x * 2) + c * 16;
  }
#pragma unroll
  for (int j = 0; j < C::NIW; ++j) {
    const int row = C::WRPW * w + C::WRPI * j + lane / C::WCPR;
    const int c = C::sww(row, lane % C::WCPR);
    int wcol;
    if (region == 0) wcol = key_wcol(col0 + 8 * c, a.head_dim);
    else if (region == 1) wcol = col0 + 8 * c;  // W_v columns follow W_k's
    else wcol = lcol0 + 8 * c;
    krow[j] = row;
    offw[j] = 8 * c < cols ? row * (int32_t)(ldw * 2) + wcol * 2 : INT32_MIN;  // LR columns past n_cols: zeros
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
    for (int j = 0; j < C::NIX; ++j) {
      // Chunks wholly past d_in (d_in is a multiple of 8) read as zeros.
      const int32_t ox = k0 + kch[j] < a.d_in ? offx[j] : INT32_MIN;
      lds_dma16(rx, &tiles[sl][0][(C::XRPW * w + C::XRPI * j) * KST], ox, k0 * 2);
    }
#pragma unroll
    for (int j = 0; j < C::NIW; ++j) {
      // k rows past d_in read as zeros; the whole offset is range-checked.
      const int32_t ow =
          (k0 + krow[j] < a.d_in && offw[j] != INT32_MIN) ? offw[j] + k0 * (int32_t)(ldw * 2) : INT32_MIN;
      lds_dma16(rw, &tiles[sl][1][(C::WRPW * w + C::WRPI * j) * TB], ow, 0);
    }
  };

  f32x16 acc[2][2];
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
      // to AHEAD of them, NIX + NIW instructions each) are still in flight.
      const int ahead = nstage - 1 - s < AHEAD ? nstage - 1 - s : AHEAD;
      wait_vmcnt_le((C::NIX + C::NIW) * ahead);
      __syncthreads();  // stage s visible to all waves
    }
  } else {
    // Compute: a 64 x 64 block of columns cw0 .. and tokens tw0 ..
    // (split k: the whole tile, k steps kk with kk % 4 == w).
    const int l32 = lane & 31, h = lane >> 5, grp = lane >> 4, i16 = lane & 15;
    const int cw0 = C::SPLITK ? 0 : 64 * (w & 1), tw0 = C::SPLITK ? 0 : 64 * (w >> 1);
#pragma unroll
    for (int bc = 0; bc < 2; ++bc)
#pragma unroll
      for (int bt = 0; bt < 2; ++bt)
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[bc][bt][j] = 0.f;
    // Transposing-read address of this lane within a k16 step: k row
    // 8 (grp / 2) + i16 / 4 (+4 for the second read), columns
    // (grp % 2) * 16 + 4 (i16 % 4) .. + 3 of each 32-column block.
    const int tr_k = 8 * (grp >> 1) + (i16 >> 2);
    const int tr_c = (grp & 1) * 16 + 4 * (i16 & 3);
    auto wfrag = [&](const uint16_t* tw, int kr, int col) {
      const int ch = col >> 3;
      return tw + kr * TB + C::sww(kr, ch) * 8 + (col & 7);
    };
    constexpr int KK = KST / 16;
    for (int s = 0; s < nstage; ++s) {
      __syncthreads();  // stage s visible to all waves; stage s - 1 consumed by all
      const uint16_t* tx = tiles[s % NST][0];
      const uint16_t* tw = tiles[s % NST][1];
#pragma unroll
      for (int ki = 0; ki < (C::SPLITK ? KK / NCW : KK); ++ki) {
        const int kk = C::SPLITK ? ki * NCW + w : ki;
        bf16x8 fa[2], fx[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int kr = 16 * kk + tr_k, col = cw0 + 32 * b + tr_c;
          const u32x2 lo = lds_read_tr(wfrag(tw, kr, col)), hi = lds_read_tr(wfrag(tw, kr + 4, col));
          fa[b] = as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]});
          const int xr = tw0 + 32 * b + l32, c = 2 * kk + h;
          fx[b] = as_bf16x8(*reinterpret_cast<const u32x4*>(tx + xr * KST + C::swx(xr, c) * 8));
        }
#pragma unroll
        for (int bc = 0; bc < 2; ++bc)
#pragma unroll
          for (int bt = 0; bt < 2; ++bt) acc[bc][bt] = mfma32x32x16(fa[bc], fx[bt], acc[bc][bt]);
      }
    }
  }

  // Which 32 x 32 blocks this wave writes: split k sums the four waves'
  // partials through LDS (the ring is free once every wave is past the last
  // stage) in a fixed order, and wave w writes block (w & 1, w >> 1).
  if constexpr (C::SPLITK) {
    float* part = reinterpret_cast<float*>(&tiles[0][0][0]);  // [wave][bc][bt][16][64]
    __syncthreads();  // every wave is past the last stage
    if (!producer) {
#pragma unroll
      for (int bc = 0; bc < 2; ++bc)
#pragma unroll
        for (int bt = 0; bt < 2; ++bt)
#pragma unroll
          for (int j = 0; j < 16; ++j) part[(((w * 2 + bc) * 2 + bt) * 16 + j) * 64 + lane] = acc[bc][bt][j];
    }
    __syncthreads();
    if (producer) return;
    const int bc = w & 1, bt = w >> 1;
    f32x16 sum;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      float v = 0.f;
#pragma unroll
      for (int ww = 0; ww < NCW; ++ww) v += part[(((ww * 2 + bc) * 2 + bt) * 16 + j) * 64 + lane];
      sum[j] = v;
    }
    acc[0][0] = sum;
  } else {
    if (producer) return;
  }

  // acc[bc][bt][j]: column cw + 32 bc + (j / 4) * 8 + h * 4 + j % 4, token
  // tw + 32 bt + l32 (split k: the one block acc[0][0] at (32 (w & 1), 32 (w >> 1))).
  const int l32 = lane & 31, h = lane >> 5;
  const int cw = C::SPLITK ? 32 * (w & 1) : 64 * (w & 1), tw = C::SPLITK ? 32 * (w >> 1) : 64 * (w >> 1);
  constexpr int NBLK = C::SPLITK ? 1 : 2;
#pragma unroll
  for (int bt = 0; bt < NBLK; ++bt)
#pragma unroll
    for (int bc = 0; bc < NBLK; ++bc)
      store_block(a, acc[bc][bt], region, col0 + cw + 32 * bc, tok0 + tw + 32 * bt + l32, h);
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
// matrix-vector product.  One workgroup per 8 output columns (a key
// workgroup: 8 dims of a head and their RoPE partners d/2 further on), so the
// weights are spread over many workgroups.  Thread t takes the k rows
// 8t .. 8t + 7 (+ 4096 per round, so a 4096-wide hidden state is one round
// with all of a thread's loads in flight at once): one 16-byte load of each
// of the T <= GV_T rows of X, and one 16-byte load (8 columns) of each weight
// row.  The partial sums are reduced over the lanes by shuffles and over the
// waves in LDS.
constexpr int GV_T = 4;
constexpr int GV_W = 8;  // waves per workgroup

__global__ void __launch_bounds__(64 * GV_W) project_gemv_kernel(const PrecomputeArgs a, int n_units) {
  __shared__ float red[GV_W][2][GV_T][8];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // The 8 workgroups whose columns share 128-byte lines of the weight rows run
  // on one XCD (workgroup L runs on XCD L % 8), so each line is fetched into
  // one L2 only.
  const int L = blockIdx.x, slot = L / NXCD;
  const int u = 8 * ((slot / 8) * NXCD + L % NXCD) + slot % 8;
  if (u >= n_units) return;
  const int half = a.head_dim / 2;
  const int n_pair = a.nkv / 16;  // key workgroups (8 pair columns each)
  const int n_val = a.nkv / 8;
  // Region of this workgroup: 0 keys (dims j0 .. j0+7 and their partners), 1
  // values, 2 LR.
  int region, c0;
  const uint16_t* w0;
  const uint16_t* w1 = nullptr;
  int64_t ldw;
  if (u < n_pair) {
    region = 0;
    const int hd = (u * 8) / half, j0 = u * 8 - hd * half;
    c0 = hd * a.head_dim + j0;  // first dim (column of W_k) of the low half
    ldw = 2 * (int64_t)a.nkv;
    w0 = a.W + c0;
    w1 = w0 + half;
  } else if (u < n_pair + n_val) {
    region = 1;
    c0 = (u - n_pair) * 8;
    ldw = 2 * (int64_t)a.nkv;
    w0 = a.W + a.nkv + c0;
  } else {
    region = 2;
    c0 = (u - n_pair - n_val) * 8;
    ldw = a.n_cols;
    w0 = a.A + c0;
  }
  const int T = (int)a.T;
  float acc0[GV_T][8], acc1[GV_T][8];
#pragma unroll
  for (int t = 0; t < GV_T; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc0[t][e] = acc1[t][e] = 0.f;
  for (int64_t k0 = (int64_t)tid * 8; k0 < a.d_in; k0 += 64 * GV_W * 8) {
    float x[GV_T][8];
#pragma unroll
    for (int t = 0; t < GV_T; ++t) {
      const u32x4 xv = ld16(a.X + t * a.ld_x + k0, t < T);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[t][2 * e] = bf_lo(xv[e]);
        x[t][2 * e + 1] = bf_hi(xv[e]);
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t k = k0 + i;  // d_in is a multiple of 8: k < d_in
      const u32x4 wv = *reinterpret_cast<const u32x4*>(w0 + k * ldw);
      float wf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        wf[2 * e] = bf_lo(wv[e]);
        wf[2 * e + 1] = bf_hi(wv[e]);
      }
#pragma unroll
      for (int t = 0; t < GV_T; ++t)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc0[t][e] += x[t][i] * wf[e];
      if (region == 0) {  // uniform over the workgroup
        const u32x4 wv1 = *reinterpret_cast<const u32x4*>(w1 + k * ldw);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          wf[2 * e] = bf_lo(wv1[e]);
          wf[2 * e + 1] = bf_hi(wv1[e]);
        }
#pragma unroll
        for (int t = 0; t < GV_T; ++t)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc1[t][e] += x[t][i] * wf[e];
      }
    }
  }
  // Sum each of the 32 (token, column) partials over the wave's lanes with a
  // transposing reduction: every step hands half of a lane's values to its
  // partner and adds the half it keeps, so after five steps lane l holds one
  // value, index (l >> 1) & 31, summed over the 32 lanes that share lane bit 0
  // (32 shuffles instead of 6 per value).
  auto reduce = [&](float (&acc)[GV_T][8]) -> float {
    float v[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) v[i] = acc[i / 8][i % 8];
#pragma unroll
    for (int st = 0; st < 5; ++st) {
      const int m = 32 >> st, half = 16 >> st;
      const bool up = (lane & m) != 0;
#pragma unroll
      for (int i = 0; i < half; ++i) {
        const float send = up ? v[i] : v[i + half];
        const float keep = up ? v[i + half] : v[i];
        v[i] = keep + shfl_xor(send, m);
      }
    }
    return v[0] + shfl_xor(v[0], 1);
  };
  static_assert(GV_T * 8 == 32, "32 partials per lane");
  const float r0 = reduce(acc0);
  const float r1 = region == 0 ? reduce(acc1) : 0.f;  // uniform over the workgroup
  if ((lane & 1) == 0) {
    const int vi = (lane >> 1) & 31;
    red[w][0][vi / 8][vi % 8] = r0;
    red[w][1][vi / 8][vi % 8] = r1;
  }
  __syncthreads();
  if (tid >= T * 8) return;
  const int t = tid / 8, e = tid % 8;
  float x = 0.f, y = 0.f;
#pragma unroll
  for (int i = 0; i < GV_W; ++i) {
    x += red[i][0][t][e];
    y += red[i][1][t][e];
  }
  const int64_t row = a.tok_offset + t;  // absolute position and cache row
  if (region == 0) {
    const int hd = c0 / a.head_dim, j = c0 - hd * a.head_dim + e;
    float cs, sn;
    rope_cs((int)row, a.w2pi[j], cs, sn);
    uint16_t* kp = a.Kout + row * a.nkv + hd * a.head_dim + j;
    kp[0] = (uint16_t)(pack_bf16(x * cs - y * sn, 0.f) & 0xffffu);
    kp[half] = (uint16_t)(pack_bf16(y * cs + x * sn, 0.f) & 0xffffu);
  } else if (region == 1) {
    a.Vout[row * a.nkv + c0 + e] = (uint16_t)(pack_bf16(x, 0.f) & 0xffffu);
  } else {
    const int c = c0 + e;
    const int64_t plane = c / a.rank, jr = c - plane * a.rank;
    a.L[(plane * a.s_cap + row) * a.rank + jr] = (uint16_t)(pack_bf16(x, 0.f) & 0xffffu);
  }
}

}  // namespace

hipError_t launch_precompute(const PrecomputeArgs& a, hipStream_t st) {
  if (a.tbl == nullptr && a.T <= GV_T) {
    const int units = a.nkv / 16 + a.nkv / 8 + a.n_cols / 8;
    hipLaunchKernelGGL(project_gemv_kernel, dim3(64 * ((units + 63) / 64)), dim3(64 * GV_W), 0, st, a, units);
    return hipGetLastError();
  }
  // 128-wide tiles halve the bytes loaded per MFMA but need enough of them to
  // fill the CUs; the K/V boundary must fall on a tile edge.
  const int64_t wide = (int64_t)((2 * a.nkv + a.n_cols + 127) / 128) * ((a.T + 127) / 128);
  if (a.nkv % 128 == 0 && wide >= 256) return launch_tb<128>(a, st);
  return launch_tb<64>(a, st);
}

}  // namespace prc
