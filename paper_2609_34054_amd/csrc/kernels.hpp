// Internal interface between the C ABI layer (abi.cpp) and the kernel files.
// Everything here runs after host-side validation has passed.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace prc {

constexpr int kMaxHalfDim = 64;  // head_dim <= 128

// Arguments of one attention (or materialise) launch.  Strides are in
// elements; `kv_stride` etc. may be 0 (all requests share one buffer).
struct AttnArgs {
  const uint16_t* Q;
  const uint16_t* Kb;
  const uint16_t* Vb;
  const uint16_t* Lk;   // nullptr: key projection not adapted
  const uint16_t* Lv;   // nullptr: value projection not adapted
  const uint16_t* Bk;   // [n_kv*d, r] per request
  const uint16_t* Bv;
  const int32_t* positions;
  const int32_t* kv_len;
  uint16_t* O;
  float* lse;
  float* ws;            // decode split partials
  uint16_t* Kout;       // materialise outputs
  uint16_t* Vout;
  // Paged caches (block tables): token t of request b sits at row t % blk of
  // block kv_tbl[b * max_blk + t / blk] of request b's base pools (Kb, Vb +
  // b * kv_stride: [kv_nblk, blk, n_kv, d]) and of block lr_tbl[...] of its
  // LR pools (Lk, Lv + b * l_stride: [lr_nblk, blk, r]).  Table entries are
  // clamped into the pools.  kv_tbl == nullptr: contiguous caches.
  const int32_t* kv_tbl;
  const int32_t* lr_tbl;
  int32_t blk;          // tokens per block (a multiple of 64)
  int32_t max_blk;      // table entries per request
  int32_t kv_nblk;      // blocks per base pool
  int32_t lr_nblk;      // blocks per LR pool
  int64_t s_cap;
  int64_t kv_stride;
  int64_t l_stride;
  int64_t b_stride;
  int32_t batch;
  int32_t n_tok;
  int32_t n_q;
  int32_t n_kv;
  int32_t group;        // n_q / n_kv
  int32_t head_dim;
  int32_t rank;
  int32_t n_splits;     // decode: KV splits per request
  int32_t split_tiles;  // decode: KV tiles per split
  int32_t pf_splits;    // prefill: KV splits per row tile (1: none)
  int32_t pf_split_tiles;  // prefill: 64-token KV tiles per split
  // Prefill tile cache in the workspace (tc_data == nullptr: off).  The
  // rebuilt K rows and V^T fragments of a full 64-token tile, in the LDS
  // layout, in eight 4 KB parts (one per wave), [request][KV head][tile][part],
  // beside one flag per part that turns nonzero once the part is published.
  uint32_t* tc_flags;
  uint32_t* tc_data;
  int32_t tc_tiles;     // tiles per (request, KV head) slot
  float scale_log2;     // softmax scale * log2(e)
  double w2pi[kMaxHalfDim];  // RoPE omega_j / (2 pi), fp64
};

// Decode (one query token per request): split-KV partials + merge.
int decode_tile_tokens();
// A decode batch whose requests all read one base cache (request stride 0)
// runs the shared-base kernel: each base tile is read once for all of them.
bool decode_shares_base(int batch, int64_t kv_req_stride);
// `cus`: compute units of the device the call runs on; `paged`: the caches
// are block pools (the plan follows the kernel form the call takes).
void decode_plan(int64_t s_cap, int batch, int n_kv, int head_dim, int rank, bool shared_base, bool paged, int cus,
                 int* n_splits, int* split_tiles);
size_t decode_workspace_bytes(int batch, int n_q, int n_splits, int head_dim, int rank);
hipError_t launch_decode(const AttnArgs& a, hipStream_t stream);

// Log-sum-exp merge of split partials ws[((b n_tok + i) n_q + h) n_splits
// + s][4 + d + r] into O (and lse), with the deferred B_v up-projection.
hipError_t launch_split_merge(const AttnArgs& a, hipStream_t stream);

// Prefill (several query tokens per request): causal flash attention.  A
// call with too few (row tile, KV head, request) units to fill the GPU is
// also split over the KV tiles, each split writing partials for the merge.
void prefill_plan(int n_tok, int group, int n_kv, int batch, int64_t s_cap, int cus, int* splits,
                  int* split_tiles);
size_t prefill_workspace_bytes(int batch, int n_tok, int n_q, int splits, int head_dim, int rank);
// Whether a prefill call shares rebuilt tiles through the workspace tile
// cache: contiguous caches, d = 128, rank >= 16 with LR on the keys, and
// enough row-tile workgroups per KV head (at least 16) for the reuse to pay
// for the cache's writes (measured: gains at ranks 16, 32 and 64 with k LR,
// a loss with LR on v only).  A split call keeps its partials first in the
// workspace, the cache after them (256-byte aligned).  tile_cache_bytes: its
// size (flags, then data).
bool prefill_uses_tile_cache(int n_tok, int group, int head_dim, int rank, bool has_lk, bool has_lv, bool paged);
size_t prefill_tile_cache_bytes(int batch, int n_kv, int64_t s_cap);
size_t prefill_tile_cache_flag_bytes(int batch, int n_kv, int64_t s_cap);
hipError_t launch_prefill(const AttnArgs& a, hipStream_t stream);

// Reference point: write the full per-agent K/V.
hipError_t launch_materialize(const AttnArgs& a, hipStream_t stream);

// LR-cache precompute GEMM.
// One GEMM over a segment of hidden states X: output columns
// [0, nkv) are keys (W rows, RoPE applied at position tok_offset + t),
// [nkv, 2 nkv) values (W rows), then n_cols LR columns (A rows).  nkv = 0 is
// the LR precompute alone.
struct PrecomputeArgs {
  const uint16_t* X;
  const uint16_t* A;    // [d_in, n_cols] (A_stack, Eq. 1 orientation)
  uint16_t* L;          // [n_cols / r][s_cap][r]
  const uint16_t* W;    // [d_in, 2 nkv]: W_k columns, then W_v columns (nkv > 0)
  uint16_t* Kout;       // [s_cap, nkv] (tokens x (head, dim))
  uint16_t* Vout;
  int64_t T;
  int64_t d_in;
  int64_t ld_x;
  int64_t s_cap;
  int64_t tok_offset;
  int32_t n_cols;
  int32_t rank;
  int32_t nkv;          // n_kv * head_dim, a multiple of 64 (or 0)
  int32_t head_dim;
  // Paged output (tbl != nullptr): token p = tok_offset + t is written to row
  // tbl[p / blk] * blk + p % blk of every pool (s_cap = nblk * blk rows per
  // LR plane); the table entry is clamped into [0, nblk).
  const int32_t* tbl;
  int32_t blk;
  int32_t nblk;
  double w2pi[kMaxHalfDim];  // RoPE omega_j / (2 pi), fp64
};
hipError_t launch_precompute(const PrecomputeArgs& a, hipStream_t stream);

// Measurement helper: stream `bytes` (a multiple of 16) from src with `grid`
// workgroups, one XOR word per workgroup to sink.
hipError_t launch_stream_read(const void* src, int64_t bytes, uint32_t* sink, int grid, hipStream_t stream);

// Checked build: the first kv_len outside [1, s_cap] or query position
// outside [0, kv_len[b]) (positions may be null), written to `result` as
// {kind, request, token, value} with kind 0 for none, 1 kv_len, 2 position.
// `result` is the per-device array whose address device_checks_result gives.
hipError_t device_checks_result(int32_t** ptr);
hipError_t launch_device_checks(const int32_t* positions, const int32_t* kv_len, int batch, int n_tok, int64_t s_cap,
                                int32_t* result, hipStream_t st);

}  // namespace prc
