/*
 * precache.h -- C ABI of the PreLRShared hot path on MI355X (gfx950).
 *
 * PReCache's PreLRShared design (Sec. 3.1) lets N LoRA agents share one base
 * KV cache.  Each agent i keeps a compact low-rank (LR) cache X A_i of r
 * numbers per token (Sec. 2.2).  The LR caches of all agents are built once,
 * when a context segment is first processed (the precompute).  Any agent can
 * then attend over the shared base cache plus its own LR cache without
 * re-processing the trajectory.  By Eq. 1 the keys and values an agent sees are
 *     K = K_base + RoPE(L_k B_k),      V = V_base + L_v B_v,
 * where RoPE is applied after the rank-r expansion (App. D.2).
 *
 * General conventions (every entry point):
 *   - Tensor arguments are DEVICE pointers owned by the caller.  The library
 *     never frees, retains or reallocates them.  bf16 data is passed as
 *     uint16_t storage (IEEE bfloat16 bit patterns).
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = the
 *     device's default stream).  No call synchronises, and no call allocates
 *     device memory.
 *   - Every call first validates its arguments on the host, before any HIP
 *     call is made.  A failed check returns a non-zero prc_status and launches
 *     nothing; prc_last_error() then gives a thread-local message naming the
 *     argument.  A call that passes every check and has work to do then
 *     requires the current HIP device to be a gfx950 (PRC_EDEVICE otherwise,
 *     nothing launched).  HIP launch failures return PRC_ELAUNCH.
 *   - Row-major layouts throughout; "[a, b, c]" lists dimensions from
 *     outermost to innermost; the innermost dimension is contiguous.
 *   - All bf16 pointers must be 16-byte aligned, and every row stride given
 *     in elements must keep rows 16-byte aligned.  int32 and fp32 pointers
 *     must be 4-byte aligned.
 *   - Values that live in device memory (positions, kv_len) cannot be checked
 *     by the host.  Kernels clamp kv_len[b] into [0, s_cap], so no access ever
 *     leaves the caller's buffers.  The checked build of the library checks
 *     them on the device (see prc_device_checks).
 *
 * Orientation of the weights.  Every weight matrix is passed in the
 * orientation of Eq. 1 (Sec. 2.1), Y = X (W0 + A B) with row vectors: frozen
 * projections W [d_in, d_out], down-projections A [d_in, r] (stacked side by
 * side for all agents: A_stack [d_in, n_proj*N*r]) and up-projections
 * B [r, d_out], all row-major.  A caller holding PEFT-style transposed
 * storage ([d_out, d_in], [r, d_in], [d_out, r]) transposes it once, when the
 * adapters are loaded.
 */
#ifndef PRECACHE_H
#define PRECACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum prc_status {
  PRC_OK = 0,
  PRC_EINVAL = 1,       /* null pointer, negative size, non-finite scalar     */
  PRC_ESHAPE = 2,       /* inconsistent sizes or strides                      */
  PRC_EALIGN = 3,       /* pointer or stride breaks the alignment rules       */
  PRC_EUNSUPPORTED = 4, /* head_dim, rank or GQA group outside the set built  */
  PRC_EWORKSPACE = 5,   /* workspace null or smaller than the size query      */
  PRC_ELAUNCH = 6,      /* a HIP launch reported an error                     */
  PRC_EDEVICE = 7,      /* no usable gfx950 device is current                 */
  PRC_EDEVDATA = 8      /* checked build: kv_len or a position out of range   */
} prc_status;

/* Thread-local message describing the last non-OK status on this thread. */
const char* prc_last_error(void);
/* Static name of a status code. */
const char* prc_status_string(prc_status s);
/* Library version string, e.g. "0.1.0". */
const char* prc_version(void);
/* 1 in the checked build (libprecache_checked.so), 0 in the release build
 * (libprecache.so).  The two export the same entry points; the checked one
 * also verifies, on the device, before launching an attention or
 * materialise call, that 1 <= kv_len[b] <= s_cap and 0 <= positions[b][i] <
 * kv_len[b] (Sec. 2.2: every query sees a non-empty causal prefix of the
 * cache).  It reads the verdict back, so each such call waits for its stream
 * (not usable under graph capture), and on a violation it launches nothing,
 * returns PRC_EDEVDATA and names the first offender (lowest request, then
 * lowest token; a kv_len fault before a position fault) in prc_last_error(). */
int prc_device_checks(void);

/*
 * precompute_lr_cache -- the LR-cache precompute of Sec. 3.1 (Fig. 1 A1-A3).
 *
 * For a newly processed segment of T hidden states, apply EVERY agent's LoRA
 * down-projection, for every adapted projection, in one batched GEMM
 * X . [A_1 | ... | A_N]:
 *     L[p][a][tok_offset + t][j] = sum_k X[t][k] * A_stack[k][(p*N + a)*r + j]
 * This is X A_k of Sec. 2.2 for all agents k at once.
 *
 *   X        [T, d_in] bf16, row stride ld_x (elements, >= d_in).  These are
 *            the hidden states that feed k_proj/v_proj.
 *   A_stack  [d_in, n_proj*N*r] bf16, contiguous.  Columns
 *            [(p*N + a)*r, (p*N + a + 1)*r) hold agent a's down-projection
 *            A [d_in, r] for projection p (p = 0: k_proj, p = 1: v_proj when
 *            n_proj = 2).
 *   L_out    [n_proj, N, s_cap, r] bf16, contiguous.  Rows
 *            [tok_offset, tok_offset + T) of every plane are overwritten;
 *            nothing else is touched.
 * Arithmetic: bf16 inputs, fp32 accumulation, round-to-nearest-even to bf16.
 * Requires d_in % 8 == 0, ld_x % 8 == 0, d_in <= ld_x < 2^23 and
 * (d_in + 128) * n_proj*N*r < 2^30 (PRC_EUNSUPPORTED otherwise), r in
 * {8, 16, 32, 64}, 1 <= s_cap < 2^31, 0 <= tok_offset and tok_offset + T <=
 * s_cap.  T == 0 is a no-op.
 */
prc_status precompute_lr_cache(const uint16_t* X, int64_t T, int64_t d_in, int64_t ld_x,
                               const uint16_t* A_stack, int32_t n_proj, int32_t n_agents,
                               int32_t rank, uint16_t* L_out, int64_t s_cap,
                               int64_t tok_offset, void* stream);

/*
 * project_kv_and_lr_cache -- the base projection of a newly processed segment
 * joined with the LR-cache precompute (Sec. 2.2 base cache X W0 with RoPE on
 * the key side; Sec. 3.1 LR precompute X A_k for every agent), as one GEMM
 * over the segment's hidden states, so X is read once for all of it:
 *     K_base[tok_offset + t][h][:] = RoPE(X[t] . W_k[:, h*d:(h+1)*d], tok_offset + t)
 *     V_base[tok_offset + t][h][:] = X[t] . W_v[:, h*d:(h+1)*d]
 *     L[p][a][tok_offset + t][j]  = X[t] . A_stack[:, (p*N + a)*r + j]
 * RoPE is the rotate-half form with omega_j = rope_theta^(-2j/d), each token
 * at its absolute position tok_offset + t (KV token t sits at position t).
 *
 *   X        [T, d_in] bf16, row stride ld_x, as for precompute_lr_cache.
 *   W        [d_in, 2*n_kv*d] bf16, contiguous: [W_k | W_v], the key
 *            projection's n_kv*d columns, then the value projection's.
 *   A_stack  as for precompute_lr_cache.
 *   K_base, V_base  [s_cap, n_kv, d] bf16, contiguous (one request's base
 *            cache); rows [tok_offset, tok_offset + T) are overwritten.
 *   L_out    [n_proj, N, s_cap, r] bf16, contiguous; the same rows of every
 *            plane are overwritten.  Nothing else is touched.
 *   n_proj * n_agents == 0 computes the base cache alone; A_stack and L_out
 *            may then be NULL and rank is ignored.
 * Arithmetic: bf16 inputs, fp32 accumulation, RoPE in fp32 with angles
 * reduced in fp64, round-to-nearest-even to bf16.  Requires d in {64, 128},
 * the precompute_lr_cache limits, 2*n_kv*d*(d_in + 128) < 2^29 and
 * s_cap < 2^31 (PRC_EUNSUPPORTED / PRC_EINVAL otherwise).  T == 0 is a no-op.
 */
prc_status project_kv_and_lr_cache(const uint16_t* X, int64_t T, int64_t d_in, int64_t ld_x,
                                   const uint16_t* W, int32_t n_kv_heads, int32_t head_dim,
                                   const uint16_t* A_stack, int32_t n_proj, int32_t n_agents,
                                   int32_t rank, double rope_theta, uint16_t* K_base,
                                   uint16_t* V_base, uint16_t* L_out, int64_t s_cap,
                                   int64_t tok_offset, void* stream);

/*
 * project_kv_and_lr_cache_paged -- project_kv_and_lr_cache writing into paged
 * caches (the block-table layout of the paged-KV serving setup, Sec. 4.1 and
 * App. C.2), so that a trajectory's cache grows one segment (or prefill
 * chunk) at a time without a contiguous reservation of s_cap tokens, and
 * trajectories can share blocks.  The trajectory's tokens are cut
 * into blocks of block_size tokens: token p (its absolute position) lives at
 * row p % block_size of pool block block_table[p / block_size].  The values
 * written are those of project_kv_and_lr_cache (RoPE still at position p).
 *
 *   block_table  [max_blocks] int32, DEVICE memory: the trajectory's blocks.
 *                Entries are clamped into [0, n_blocks), so no write leaves
 *                the pools; a wrong entry writes a wrong block of them.
 *   K_pool, V_pool  [n_blocks, block_size, n_kv, d] bf16, contiguous.
 *   L_pool   [n_proj, N, n_blocks, block_size, r] bf16, contiguous: each
 *            agent's LR plane is a pool indexed by the same block ids as the
 *            base pools.
 *   n_kv_heads == 0 writes the LR planes alone (W, K_pool, V_pool may be
 *            NULL; head_dim and rope_theta are ignored); n_proj * n_agents == 0
 *            the base pools alone.
 * Requires block_size a positive multiple of 64, max_blocks and n_blocks >= 1,
 * their products with block_size below 2^31, and tok_offset + T <=
 * max_blocks * block_size; other limits as for project_kv_and_lr_cache.
 * Rows of the pools not addressed by [tok_offset, tok_offset + T) are not
 * touched.
 */
prc_status project_kv_and_lr_cache_paged(const uint16_t* X, int64_t T, int64_t d_in, int64_t ld_x,
                                         const uint16_t* W, int32_t n_kv_heads, int32_t head_dim,
                                         const uint16_t* A_stack, int32_t n_proj, int32_t n_agents,
                                         int32_t rank, double rope_theta, uint16_t* K_pool,
                                         uint16_t* V_pool, uint16_t* L_pool, const int32_t* block_table,
                                         int32_t block_size, int32_t max_blocks, int32_t n_blocks,
                                         int64_t tok_offset, void* stream);

/* Dimensions of one LR-shared attention call (a batch of B requests). */
typedef struct lrsa_dims {
  int32_t batch;        /* B >= 0 requests                                     */
  int32_t n_tok;        /* query tokens per request (1 = decode)               */
  int32_t n_q_heads;    /* query heads                                         */
  int32_t n_kv_heads;   /* KV heads; n_q_heads / n_kv_heads in 1..8            */
  int32_t head_dim;     /* d in {64, 128}                                      */
  int32_t rank;         /* r in {8, 16, 32, 64}; ignored when no LR is given   */
  int64_t s_cap;        /* token capacity of each request's caches             */
  int64_t kv_req_stride;/* elements between requests in K_base/V_base
                           (>= s_cap*n_kv*d, or 0: all requests share one)     */
  int64_t l_req_stride; /* elements between requests' LR planes (0: shared)    */
  int64_t b_req_stride; /* elements between requests' up-projections (0: shared) */
  float softmax_scale;  /* <= 0 selects 1/sqrt(head_dim)                       */
  float reserved0;      /* must be 0                                           */
  double rope_theta;    /* RoPE base, > 0                                      */
} lrsa_dims;

/*
 * lr_shared_attention -- attention of an agent over the shared base cache plus
 * its own LR cache (Sec. 3.1, reuse step; value-side reordering of App. D.2).
 *
 * For request b, query token i and query head h (KV head g = h / (n_q/n_kv)):
 *     K[t] = K_base[t][g] + RoPE(L_k[t] . B_k[:, g*d:(g+1)*d], t)
 *     V[t] = V_base[t][g] + L_v[t] . B_v[:, g*d:(g+1)*d]
 *     O[b][i][h] = softmax_t( scale * Q[b][i][h] . K[t] ) . V[t]
 * over the keys t with t < kv_len[b] and t <= positions[b][i].  KV token t sits
 * at absolute position t.  RoPE is rotate-half: element j pairs with j + d/2,
 * at angle t * theta^(-2j/d).  The full per-agent K/V is never written to
 * memory: each KV tile is rebuilt on chip.
 *
 *   Q          [B, n_tok, n_q, d] bf16, already rotated at positions[b][i].
 *   K_base     [B, s_cap, n_kv, d] bf16 (request stride kv_req_stride), already
 *              rotated at each token's position.
 *   V_base     same layout as K_base.
 *   L_k, L_v   [B, s_cap, r] bf16 (request stride l_req_stride): each request's
 *              agent plane of the LR cache.  NULL = that projection is not
 *              adapted.  The QV setting of the paper passes L_k = NULL.
 *   B_k, B_v   [B, r, n_kv*d] bf16 (request stride b_req_stride): each request's
 *              agent up-projection B of Eq. 1 (row j: rank j, all KV heads'
 *              columns; head g owns columns [g*d, (g+1)*d)).  Must be NULL
 *              exactly when the matching L is NULL.
 *   positions  [B, n_tok] int32, absolute query positions.
 *   kv_len     [B] int32, number of valid cache rows per request (device memory).
 *   O          [B, n_tok, n_q, d] bf16 output.
 *   lse        [B, n_tok, n_q] fp32 natural-log log-sum-exp of the scaled scores,
 *              or NULL.  A row that sees no key gets O = 0 and lse = -inf.
 *   workspace  device scratch of at least lr_shared_attention_workspace_size(dims)
 *              bytes (NULL allowed when the size is 0): the split partials of
 *              decode (n_tok == 1), and of a prefill whose units of work (256
 *              query rows x KV head x request) fill the device's CUs so
 *              unevenly that splitting the KV tiles 2-8 ways shortens the
 *              modelled time (rounds of one unit per CU) by at least 10%.
 *              For a prefill of rank 8, 16, 32 or 64 with at least 8 row
 *              tiles (256 query rows each) per KV head, d = 128 and
 *              contiguous caches, the size also covers an optional tile
 *              cache (after the partials, 256-byte aligned): with
 *              L_k given (or L_v alone at rank 32 or 64) and a 256-byte
 *              aligned workspace of at least that
 *              size, each rebuilt 64-token K/V tile is shared between the
 *              row tiles of its KV head through it; otherwise every row tile
 *              rebuilds every tile (the result then differs only by the
 *              order in which tiles are summed).  Its size is 32 bytes of
 *              flags per tile, request and KV head (rounded up to 256), then
 *              32 KB per tile: about the size of the agent's K and V over
 *              s_cap, held only during the call.
 *              Contents need no initialisation; calls that share a workspace
 *              must be ordered on one stream.
 * Arithmetic: bf16 inputs; fp32 accumulation and softmax; rebuilt K tiles are
 * rounded to bf16 before the QK^T contraction; output rounded to bf16.
 */
prc_status lr_shared_attention(const lrsa_dims* dims, const uint16_t* Q,
                               const uint16_t* K_base, const uint16_t* V_base,
                               const uint16_t* L_k, const uint16_t* L_v,
                               const uint16_t* B_k, const uint16_t* B_v,
                               const int32_t* positions, const int32_t* kv_len,
                               uint16_t* O, float* lse, void* workspace,
                               size_t workspace_bytes, void* stream);

/* Workspace bytes lr_shared_attention needs for `dims` (0 when none, or when
 * dims is invalid; validation errors are reported by the call itself). */
size_t lr_shared_attention_workspace_size(const lrsa_dims* dims);

/*
 * lr_shared_attention_noalloc -- lr_shared_attention for callers that cannot
 * allocate device memory or hand in a workspace: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, output, arithmetic and errors as lr_shared_attention, minus the
 * workspace: the split partials go to a static device array of
 * PRC_NOALLOC_WORKSPACE_BYTES that the library holds on each device it runs
 * on until the process ends (its device address is fetched on the first call
 * made with that device current).  The call allocates nothing.
 *   - A call whose partials (lr_shared_attention_workspace_size(dims)) exceed
 *     PRC_NOALLOC_WORKSPACE_BYTES returns PRC_EWORKSPACE and launches nothing.
 *   - Every call on one device shares that device's array.  No part of it
 *     needs to start at zero (each split writes all of its partial before the
 *     merge reads it), but calls that overlap on one device, on different
 *     streams or from different threads, race on it: order them on one stream.
 */
#define PRC_NOALLOC_WORKSPACE_BYTES (32u << 20)
prc_status lr_shared_attention_noalloc(const lrsa_dims* dims, const uint16_t* Q,
                                       const uint16_t* K_base, const uint16_t* V_base,
                                       const uint16_t* L_k, const uint16_t* L_v,
                                       const uint16_t* B_k, const uint16_t* B_v,
                                       const int32_t* positions, const int32_t* kv_len,
                                       uint16_t* O, float* lse, void* stream);

/* Block tables of a paged lr_shared_attention_paged call. */
typedef struct lrsa_paging {
  const int32_t* kv_block_table; /* [B, max_blocks] int32, DEVICE memory: row b
                                    lists request b's blocks of the base pools */
  const int32_t* lr_block_table; /* [B, max_blocks] int32, DEVICE memory, for the
                                    LR pools; NULL: the same as kv_block_table */
  int32_t block_size;  /* tokens per block, a positive multiple of 64          */
  int32_t max_blocks;  /* entries per table row; s_cap = max_blocks*block_size */
  int32_t n_kv_blocks; /* blocks in (each request's) base pools, >= 1          */
  int32_t n_lr_blocks; /* blocks in each LR pool, >= 1 when an L is given      */
} lrsa_paging;

/*
 * lr_shared_attention_paged -- lr_shared_attention over paged caches (the
 * block-table layout of the paged-KV serving setup of Sec. 4.1 and App. C.2,
 * with chunked prefill: the n_tok
 * queries of a chunk attend over every earlier token plus the chunk itself,
 * once the chunk has been written with project_kv_and_lr_cache_paged).
 * Computes exactly what lr_shared_attention computes (bit for bit, given the
 * same cache contents) with token t of request b read from row
 * t % block_size of block kv_block_table[b][t / block_size] (base) and
 * lr_block_table[b][t / block_size] (LR).
 *
 *   K_pool, V_pool  [n_kv_blocks, block_size, n_kv, d] bf16; request b's pool
 *              starts kv_req_stride * b elements in (normally 0: one pool
 *              shared by all requests, so agents of one trajectory list the
 *              same blocks).
 *   L_k, L_v   [n_lr_blocks, block_size, r] bf16 pools; request b's starts
 *              l_req_stride * b elements in (e.g. its agent's plane of the
 *              L_pool written by project_kv_and_lr_cache_paged).
 *   dims.s_cap must equal max_blocks * block_size; strides, when non-zero,
 *   must cover one request's pools.  Table entries are clamped into the
 *   pools, so no read leaves them.  Other arguments, the output and the
 *   arithmetic as for lr_shared_attention.  Decode (n_tok == 1) needs the
 *   workspace given by lr_shared_attention_paged_workspace_size.
 */
prc_status lr_shared_attention_paged(const lrsa_dims* dims, const lrsa_paging* paging,
                                     const uint16_t* Q, const uint16_t* K_pool,
                                     const uint16_t* V_pool, const uint16_t* L_k,
                                     const uint16_t* L_v, const uint16_t* B_k,
                                     const uint16_t* B_v, const int32_t* positions,
                                     const int32_t* kv_len, uint16_t* O, float* lse,
                                     void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes lr_shared_attention_paged needs for `dims` (0 as for
 * lr_shared_attention_workspace_size). */
size_t lr_shared_attention_paged_workspace_size(const lrsa_dims* dims);

/*
 * materialize_agent_kv -- the reference point: write out each request's full
 * per-agent K/V (the keys and values NonShared/BaseShared agents would hold,
 * Sec. 3.1) so that a plain attention call (L_k = L_v = NULL) can consume them.
 *     K_full[b][t][g] = K_base[b][t][g] + RoPE(L_k[b][t] . B_k[b][:, g*d:(g+1)*d], t)
 *     V_full[b][t][g] = V_base[b][t][g] + L_v[b][t] . B_v[b][:, g*d:(g+1)*d]
 * for t < kv_len[b].  Rows t >= kv_len[b] of K_full/V_full are not written.
 *   K_full, V_full  [B, s_cap, n_kv, d] bf16, contiguous (request stride
 *                   s_cap*n_kv*d), and must not alias the inputs.
 * Other arguments (B_k, B_v as [B, r, n_kv*d]) as in lr_shared_attention
 * (n_tok, softmax_scale ignored).  No output byte may lie in any input's
 * extent (PRC_EINVAL).  A NULL L_k (or L_v) copies K_base (or V_base)
 * unchanged.
 */
prc_status materialize_agent_kv(const lrsa_dims* dims, const uint16_t* K_base,
                                const uint16_t* V_base, const uint16_t* L_k,
                                const uint16_t* L_v, const uint16_t* B_k,
                                const uint16_t* B_v, const int32_t* kv_len,
                                uint16_t* K_full, uint16_t* V_full, void* stream);

/*
 * prc_stream_read -- measurement helper, not part of the hot path: reads
 * `bytes` bytes of device memory at `src` with 16-byte loads from `grid`
 * workgroups of 256 threads (grid-stride) and writes one XOR word per
 * workgroup to `sink` [grid] uint32 (device memory), so the reads cannot be
 * elided.  Timing it over a buffer far larger than the 256 MB Infinity Cache
 * gives the device's achievable HBM read rate, the measured ceiling the
 * bandwidth-bound kernels are compared with.  Requires bytes a positive
 * multiple of 16 (at most 2^40), src 16-byte and sink 4-byte aligned,
 * 1 <= grid <= 2^20.
 */
prc_status prc_stream_read(const void* src, size_t bytes, uint32_t* sink, int32_t grid, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PRECACHE_H */
