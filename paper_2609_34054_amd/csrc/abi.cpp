// C ABI of the PreLRShared hot path: host-side validation and dispatch.
//
// Every argument check runs on the host before any HIP call, so each error
// status can be produced (and tested) without a GPU.  The semantics of each
// entry point are documented in include/precache.h.
#include "precache.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "kernels.hpp"

#define PRC_API extern "C" __attribute__((visibility("default")))

// 1 in libprecache_checked.so: device-resident kv_len and positions are
// checked before each attention or materialise call.
#ifndef PRC_DEVICE_CHECKS
#define PRC_DEVICE_CHECKS 0
#endif

namespace {

thread_local std::string g_err;

prc_status fail(prc_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

prc_status ok() {
  g_err.clear();
  return PRC_OK;
}

bool aligned(const void* p, size_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }
bool rank_ok(int64_t r) { return r == 8 || r == 16 || r == 32 || r == 64; }

// The current device, probed once per device: the kernels are built for
// gfx950 only, and the split plans size themselves to its compute units.
struct DeviceInfo {
  bool probed = false;
  bool gfx950 = false;
  int cus = 0;
};
constexpr int kMaxDevices = 64;
DeviceInfo g_dev[kMaxDevices];
std::mutex g_dev_mu;
// Plans made where no device is visible (a workspace query on a host without
// a GPU) assume the 256 CUs of an MI355X.
constexpr int kDefaultCUs = 256;

const DeviceInfo* current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> lk(g_dev_mu);
  DeviceInfo& d = g_dev[dev];
  if (!d.probed) {
    hipDeviceProp_t p;
    if (hipGetDeviceProperties(&p, dev) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    d.gfx950 = std::strncmp(p.gcnArchName, "gfx950", 6) == 0;
    d.cus = p.multiProcessorCount;
    d.probed = true;
  }
  return &d;
}

int plan_cus() {
  const DeviceInfo* d = current_device();
  return d != nullptr && d->cus > 0 ? d->cus : kDefaultCUs;
}

// Checked right before a launch, after every argument check.
prc_status device_ready(int* cus) {
  const DeviceInfo* d = current_device();
  if (d == nullptr) return fail(PRC_EDEVICE, "no HIP device is current");
  if (!d->gfx950) return fail(PRC_EDEVICE, "the current device is not a gfx950 (MI355X)");
  *cus = d->cus > 0 ? d->cus : kDefaultCUs;
  return PRC_OK;
}

prc_status launch_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(PRC_ELAUNCH, "%s: HIP launch failed: %s", what, hipGetErrorString(e));
  return ok();
}

#if PRC_DEVICE_CHECKS
// Checked build: before a call's kernels run, check the device-resident
// kv_len and positions and read the verdict back (the call then waits for the
// stream).  A failed check launches nothing and returns PRC_EDEVDATA.
int32_t* g_check_ptr[kMaxDevices];

prc_status device_data_check(const char* who, const int32_t* positions, const int32_t* kv_len, int batch, int n_tok,
                             int64_t s_cap, hipStream_t st) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return fail(PRC_EDEVICE, "no HIP device is current");
  }
  int32_t* res = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_dev_mu);
    if (g_check_ptr[dev] == nullptr) {
      int32_t* p = nullptr;
      const hipError_t e = prc::device_checks_result(&p);
      if (e != hipSuccess || p == nullptr) {
        (void)hipGetLastError();
        return fail(PRC_EDEVICE, "%s: device check array unavailable: %s", who, hipGetErrorString(e));
      }
      g_check_ptr[dev] = p;
    }
    res = g_check_ptr[dev];
  }
  hipError_t e = prc::launch_device_checks(positions, kv_len, batch, n_tok, s_cap, res, st);
  int32_t h[4] = {0, 0, 0, 0};
  if (e == hipSuccess) e = hipMemcpyAsync(h, res, sizeof(h), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail(PRC_ELAUNCH, "%s: device check failed: %s", who, hipGetErrorString(e));
  if (h[0] == 1)
    return fail(PRC_EDEVDATA, "%s: kv_len[%d]=%d outside [1, s_cap=%lld]", who, h[1], h[3], (long long)s_cap);
  if (h[0] == 2)
    return fail(PRC_EDEVDATA, "%s: positions[%d][%d]=%d outside [0, kv_len[%d])", who, h[1], h[2], h[3], h[1]);
  return PRC_OK;
}
#endif

// Validated view of an attention/materialise call.
struct Checked {
  prc::AttnArgs a;
  bool empty;
};

prc_status check_attention(const lrsa_dims* dims, const uint16_t* Q, const uint16_t* K_base,
                           const uint16_t* V_base, const uint16_t* L_k, const uint16_t* L_v,
                           const uint16_t* B_k, const uint16_t* B_v, const int32_t* positions,
                           const int32_t* kv_len, bool need_q, const lrsa_paging* pg, Checked* out) {
  if (dims == nullptr) return fail(PRC_EINVAL, "dims is NULL");
  const lrsa_dims& d = *dims;
  if (d.batch < 0 || d.batch > 65535) return fail(PRC_EINVAL, "batch=%d outside [0, 65535]", d.batch);
  if (d.n_tok < 0) return fail(PRC_EINVAL, "n_tok=%d is negative", d.n_tok);
  if (d.n_q_heads < 1 || d.n_kv_heads < 1 || d.n_kv_heads > 65535)
    return fail(PRC_EINVAL, "n_q_heads=%d, n_kv_heads=%d must be positive", d.n_q_heads, d.n_kv_heads);
  if (d.n_q_heads % d.n_kv_heads != 0)
    return fail(PRC_ESHAPE, "n_q_heads=%d is not a multiple of n_kv_heads=%d", d.n_q_heads, d.n_kv_heads);
  const int group = d.n_q_heads / d.n_kv_heads;
  if (group > 8) return fail(PRC_EUNSUPPORTED, "GQA group n_q/n_kv=%d > 8 is not built", group);
  if (d.head_dim != 64 && d.head_dim != 128)
    return fail(PRC_EUNSUPPORTED, "head_dim=%d (built: 64, 128)", d.head_dim);
  if (d.s_cap < 1 || d.s_cap > INT32_MAX) return fail(PRC_EINVAL, "s_cap=%lld outside [1, 2^31-1]", (long long)d.s_cap);
  if ((int64_t)d.n_tok * group > INT32_MAX / 2) return fail(PRC_EINVAL, "n_tok * group too large");
  if (!(d.rope_theta > 0.0) || !std::isfinite(d.rope_theta))
    return fail(PRC_EINVAL, "rope_theta=%g must be positive and finite", d.rope_theta);
  if (!std::isfinite(d.softmax_scale)) return fail(PRC_EINVAL, "softmax_scale is not finite");
  if (d.reserved0 != 0.f) return fail(PRC_EINVAL, "reserved0 must be 0");
  if ((L_k == nullptr) != (B_k == nullptr))
    return fail(PRC_EINVAL, "L_k and B_k must both be given or both be NULL");
  if ((L_v == nullptr) != (B_v == nullptr))
    return fail(PRC_EINVAL, "L_v and B_v must both be given or both be NULL");
  const bool has_lr = L_k != nullptr || L_v != nullptr;
  if (has_lr && !rank_ok(d.rank)) return fail(PRC_EUNSUPPORTED, "rank=%d (built: 8, 16, 32, 64)", d.rank);
  const int64_t dd = d.head_dim, r = has_lr ? d.rank : 8;
  // Elements of one request's base and LR caches (paged: of its pools).
  int64_t kv_need = d.s_cap * d.n_kv_heads * dd, l_need = d.s_cap * r;
  if (pg != nullptr) {
    const lrsa_paging& p = *pg;
    if (p.block_size < 64 || p.block_size % 64)
      return fail(PRC_EUNSUPPORTED, "block_size=%d must be a positive multiple of 64", p.block_size);
    if (p.max_blocks < 1 || p.n_kv_blocks < 1 || (has_lr && p.n_lr_blocks < 1))
      return fail(PRC_EINVAL, "max_blocks=%d, n_kv_blocks=%d, n_lr_blocks=%d must be positive", p.max_blocks,
                  p.n_kv_blocks, p.n_lr_blocks);
    if ((int64_t)p.max_blocks * p.block_size != d.s_cap)
      return fail(PRC_ESHAPE, "s_cap=%lld must equal max_blocks*block_size=%lld", (long long)d.s_cap,
                  (long long)p.max_blocks * p.block_size);
    kv_need = (int64_t)p.n_kv_blocks * p.block_size * d.n_kv_heads * dd;
    l_need = (int64_t)p.n_lr_blocks * p.block_size * r;
  }
  if (d.kv_req_stride != 0 && d.kv_req_stride < kv_need && d.batch > 1)
    return fail(PRC_ESHAPE, "kv_req_stride=%lld < %lld elements of one request's base cache",
                (long long)d.kv_req_stride, (long long)kv_need);
  if (d.kv_req_stride < 0 || d.l_req_stride < 0 || d.b_req_stride < 0)
    return fail(PRC_EINVAL, "request strides must be >= 0");
  if (has_lr && d.l_req_stride != 0 && d.l_req_stride < l_need && d.batch > 1)
    return fail(PRC_ESHAPE, "l_req_stride=%lld < %lld elements of one request's LR cache", (long long)d.l_req_stride,
                (long long)l_need);
  if (has_lr && d.b_req_stride != 0 && d.b_req_stride < d.n_kv_heads * dd * r && d.batch > 1)
    return fail(PRC_ESHAPE, "b_req_stride=%lld < n_kv*d*rank", (long long)d.b_req_stride);
  if (d.kv_req_stride % 8 || d.l_req_stride % 8 || d.b_req_stride % 8)
    return fail(PRC_EALIGN, "request strides must be multiples of 8 elements (16 bytes)");

  out->empty = d.batch == 0 || (need_q && d.n_tok == 0);
  if (out->empty) return ok();
  if (need_q && Q == nullptr) return fail(PRC_EINVAL, "Q is NULL");
  if (K_base == nullptr || V_base == nullptr) return fail(PRC_EINVAL, "K_base/V_base is NULL");
  if (kv_len == nullptr) return fail(PRC_EINVAL, "kv_len is NULL");
  if (need_q && positions == nullptr) return fail(PRC_EINVAL, "positions is NULL");
  const void* bf[] = {Q, K_base, V_base, L_k, L_v, B_k, B_v};
  const char* names[] = {"Q", "K_base", "V_base", "L_k", "L_v", "B_k", "B_v"};
  for (int i = 0; i < 7; ++i)
    if (bf[i] != nullptr && !aligned(bf[i], 16)) return fail(PRC_EALIGN, "%s is not 16-byte aligned", names[i]);
  if (!aligned(kv_len, 4) || (positions != nullptr && !aligned(positions, 4)))
    return fail(PRC_EALIGN, "positions/kv_len are not 4-byte aligned");
  if (pg != nullptr) {
    if (pg->kv_block_table == nullptr) return fail(PRC_EINVAL, "kv_block_table is NULL");
    if (!aligned(pg->kv_block_table, 4) || (pg->lr_block_table != nullptr && !aligned(pg->lr_block_table, 4)))
      return fail(PRC_EALIGN, "block tables are not 4-byte aligned");
  }

  prc::AttnArgs& a = out->a;
  a = prc::AttnArgs{};
  a.Q = Q;
  a.Kb = K_base;
  a.Vb = V_base;
  a.Lk = L_k;
  a.Lv = L_v;
  a.Bk = B_k;
  a.Bv = B_v;
  a.positions = positions;
  a.kv_len = kv_len;
  a.s_cap = d.s_cap;
  a.kv_stride = d.kv_req_stride;
  a.l_stride = d.l_req_stride;
  a.b_stride = d.b_req_stride;
  a.batch = d.batch;
  a.n_tok = d.n_tok;
  a.n_q = d.n_q_heads;
  a.n_kv = d.n_kv_heads;
  a.group = group;
  a.head_dim = d.head_dim;
  a.rank = (int32_t)r;
  if (pg != nullptr) {
    a.kv_tbl = pg->kv_block_table;
    a.lr_tbl = pg->lr_block_table != nullptr ? pg->lr_block_table : pg->kv_block_table;
    a.blk = pg->block_size;
    a.max_blk = pg->max_blocks;
    a.kv_nblk = pg->n_kv_blocks;
    a.lr_nblk = has_lr ? pg->n_lr_blocks : 1;
  }
  const double scale = d.softmax_scale > 0.f ? (double)d.softmax_scale : 1.0 / std::sqrt((double)d.head_dim);
  a.scale_log2 = (float)(scale * 1.4426950408889634);
  // RoPE frequencies omega_j = theta^(-2j/d), passed as revolutions per
  // position, omega_j / (2 pi), in fp64.
  for (int j = 0; j < d.head_dim / 2; ++j)
    a.w2pi[j] = std::pow(d.rope_theta, -2.0 * j / (double)d.head_dim) / (2.0 * M_PI);
  return ok();
}

}  // namespace

PRC_API const char* prc_last_error(void) { return g_err.c_str(); }

PRC_API const char* prc_status_string(prc_status s) {
  switch (s) {
    case PRC_OK: return "PRC_OK";
    case PRC_EINVAL: return "PRC_EINVAL";
    case PRC_ESHAPE: return "PRC_ESHAPE";
    case PRC_EALIGN: return "PRC_EALIGN";
    case PRC_EUNSUPPORTED: return "PRC_EUNSUPPORTED";
    case PRC_EWORKSPACE: return "PRC_EWORKSPACE";
    case PRC_ELAUNCH: return "PRC_ELAUNCH";
    case PRC_EDEVICE: return "PRC_EDEVICE";
    case PRC_EDEVDATA: return "PRC_EDEVDATA";
  }
  return "PRC_UNKNOWN";
}

PRC_API const char* prc_version(void) { return "0.1.0"; }

PRC_API int prc_device_checks(void) { return PRC_DEVICE_CHECKS; }

PRC_API prc_status precompute_lr_cache(const uint16_t* X, int64_t T, int64_t d_in, int64_t ld_x,
                                       const uint16_t* A_stack, int32_t n_proj, int32_t n_agents,
                                       int32_t rank, uint16_t* L_out, int64_t s_cap, int64_t tok_offset,
                                       void* stream) {
  if (T < 0) return fail(PRC_EINVAL, "T=%lld is negative", (long long)T);
  if (d_in < 1 || d_in % 8) return fail(PRC_EUNSUPPORTED, "d_in=%lld must be a positive multiple of 8", (long long)d_in);
  if (ld_x < d_in) return fail(PRC_ESHAPE, "ld_x=%lld < d_in=%lld", (long long)ld_x, (long long)d_in);
  if (ld_x % 8) return fail(PRC_EALIGN, "ld_x=%lld is not a multiple of 8 elements", (long long)ld_x);
  // Tiles of up to 128 rows are addressed with 32-bit byte offsets.
  if (ld_x >= (1LL << 23)) return fail(PRC_EUNSUPPORTED, "ld_x=%lld must be below 2^23", (long long)ld_x);
  if (n_proj < 1 || n_agents < 1) return fail(PRC_EINVAL, "n_proj=%d, n_agents=%d must be positive", n_proj, n_agents);
  if (!rank_ok(rank)) return fail(PRC_EUNSUPPORTED, "rank=%d (built: 8, 16, 32, 64)", rank);
  const int64_t n_cols = (int64_t)n_proj * n_agents * rank;
  if (n_cols > 65535LL * 64) return fail(PRC_EINVAL, "n_proj*n_agents*rank=%lld too large", (long long)n_cols);
  // A_stack is addressed with 32-bit byte offsets (a stage reads up to 128 k rows past d_in).
  if ((d_in + 128) * n_cols * 2 >= (1LL << 31))
    return fail(PRC_EUNSUPPORTED, "d_in*n_cols=%lld weights are too many", (long long)(d_in * n_cols));
  if (s_cap < 1 || s_cap > INT32_MAX)
    return fail(PRC_EINVAL, "s_cap=%lld must be in [1, 2^31)", (long long)s_cap);
  if (tok_offset < 0 || tok_offset + T > s_cap)
    return fail(PRC_ESHAPE, "rows [%lld, %lld) fall outside s_cap=%lld", (long long)tok_offset,
                (long long)(tok_offset + T), (long long)s_cap);
  if (T == 0) return ok();
  if (T > (int64_t)INT32_MAX * 64) return fail(PRC_EINVAL, "T too large");
  if (X == nullptr || A_stack == nullptr || L_out == nullptr) return fail(PRC_EINVAL, "X/A_stack/L_out is NULL");
  if (!aligned(X, 16) || !aligned(A_stack, 16) || !aligned(L_out, 16))
    return fail(PRC_EALIGN, "X/A_stack/L_out must be 16-byte aligned");
  prc::PrecomputeArgs a{};
  a.X = X;
  a.A = A_stack;
  a.L = L_out;
  a.T = T;
  a.d_in = d_in;
  a.ld_x = ld_x;
  a.s_cap = s_cap;
  a.tok_offset = tok_offset;
  a.n_cols = (int32_t)n_cols;
  a.rank = rank;
  int cus = 0;
  if (prc_status ds = device_ready(&cus)) return ds;
  return launch_status(prc::launch_precompute(a, static_cast<hipStream_t>(stream)), "precompute_lr_cache");
}

namespace {

// Shared body of the contiguous and paged projection entry points.  Paged:
// the caches are pools of n_blocks blocks of blk tokens and
// s_cap is the trajectory's logical capacity max_blocks * blk.
prc_status project_impl(const char* who, const uint16_t* X, int64_t T, int64_t d_in, int64_t ld_x,
                        const uint16_t* W, int32_t n_kv_heads, int32_t head_dim, const uint16_t* A_stack,
                        int32_t n_proj, int32_t n_agents, int32_t rank, double rope_theta, uint16_t* K_base,
                        uint16_t* V_base, uint16_t* L_out, int64_t s_cap, int64_t tok_offset, bool paged,
                        const int32_t* tbl, int32_t blk, int32_t n_blocks, hipStream_t stream) {
  if (T < 0) return fail(PRC_EINVAL, "T=%lld is negative", (long long)T);
  if (d_in < 1 || d_in % 8) return fail(PRC_EUNSUPPORTED, "d_in=%lld must be a positive multiple of 8", (long long)d_in);
  if (ld_x < d_in) return fail(PRC_ESHAPE, "ld_x=%lld < d_in=%lld", (long long)ld_x, (long long)d_in);
  if (ld_x % 8) return fail(PRC_EALIGN, "ld_x=%lld is not a multiple of 8 elements", (long long)ld_x);
  if (ld_x >= (1LL << 23)) return fail(PRC_EUNSUPPORTED, "ld_x=%lld must be below 2^23", (long long)ld_x);
  // Paged calls may leave out the base projection (n_kv_heads == 0).
  const bool with_base = n_kv_heads != 0 || !paged;
  if (with_base && head_dim != 64 && head_dim != 128)
    return fail(PRC_EUNSUPPORTED, "head_dim=%d (built: 64, 128)", head_dim);
  if (n_kv_heads < 0 || (!paged && n_kv_heads < 1))
    return fail(PRC_EINVAL, "n_kv_heads=%d must be positive", n_kv_heads);
  const int64_t nkv = with_base ? (int64_t)n_kv_heads * head_dim : 0;
  // The weights are addressed with 32-bit byte offsets (a stage reads up to
  // 128 k rows past d_in).
  if (2 * nkv * (d_in + 128) * 2 >= (1LL << 31))
    return fail(PRC_EUNSUPPORTED, "2*n_kv*head_dim*d_in=%lld weights are too many", (long long)(2 * nkv * d_in));
  // n_proj * n_agents == 0: the base projection alone (no LR planes).
  if (n_proj < 0 || n_agents < 0) return fail(PRC_EINVAL, "n_proj=%d, n_agents=%d must not be negative", n_proj, n_agents);
  const bool with_lr = n_proj > 0 && n_agents > 0;
  if (!with_base && !with_lr) return fail(PRC_EINVAL, "neither the base projection nor an LR plane is asked for");
  if (with_lr && !rank_ok(rank)) return fail(PRC_EUNSUPPORTED, "rank=%d (built: 8, 16, 32, 64)", rank);
  const int64_t n_cols = with_lr ? (int64_t)n_proj * n_agents * rank : 0;
  if (2 * nkv + n_cols > 65535LL * 64) return fail(PRC_EINVAL, "too many output columns");
  if ((d_in + 128) * n_cols * 2 >= (1LL << 31))
    return fail(PRC_EUNSUPPORTED, "d_in*n_cols=%lld weights are too many", (long long)(d_in * n_cols));
  if (with_base && !(rope_theta > 0.0)) return fail(PRC_EINVAL, "rope_theta must be positive");
  if (s_cap < 1 || s_cap > INT32_MAX) return fail(PRC_EINVAL, "s_cap=%lld must be in [1, 2^31)", (long long)s_cap);
  if (tok_offset < 0 || tok_offset + T > s_cap)
    return fail(PRC_ESHAPE, "rows [%lld, %lld) fall outside s_cap=%lld", (long long)tok_offset,
                (long long)(tok_offset + T), (long long)s_cap);
  if (T == 0) return ok();
  if (X == nullptr || (with_base && (W == nullptr || K_base == nullptr || V_base == nullptr)) ||
      (with_lr && (A_stack == nullptr || L_out == nullptr)))
    return fail(PRC_EINVAL, "X/W/A_stack/K_base/V_base/L_out is NULL");
  if (!aligned(X, 16) || (with_base && (!aligned(W, 16) || !aligned(K_base, 16) || !aligned(V_base, 16))) ||
      (with_lr && (!aligned(A_stack, 16) || !aligned(L_out, 16))))
    return fail(PRC_EALIGN, "X/W/A_stack/K_base/V_base/L_out must be 16-byte aligned");
  if (paged && tbl == nullptr) return fail(PRC_EINVAL, "block_table is NULL");
  if (paged && !aligned(tbl, 4)) return fail(PRC_EALIGN, "block_table is not 4-byte aligned");
  prc::PrecomputeArgs a{};
  a.X = X;
  a.A = A_stack;
  a.L = L_out;
  a.W = W;
  a.Kout = K_base;
  a.Vout = V_base;
  a.T = T;
  a.d_in = d_in;
  a.ld_x = ld_x;
  a.s_cap = paged ? (int64_t)n_blocks * blk : s_cap;
  a.tok_offset = tok_offset;
  a.n_cols = (int32_t)n_cols;
  a.rank = with_lr ? rank : 8;
  a.nkv = (int32_t)nkv;
  a.head_dim = with_base ? head_dim : 64;
  a.tbl = paged ? tbl : nullptr;
  a.blk = blk;
  a.nblk = n_blocks;
  if (with_base)
    for (int j = 0; j < head_dim / 2; ++j)
      a.w2pi[j] = std::pow(rope_theta, -2.0 * j / (double)head_dim) / (2.0 * M_PI);
  int cus = 0;
  if (prc_status ds = device_ready(&cus)) return ds;
  return launch_status(prc::launch_precompute(a, stream), who);
}

}  // namespace

PRC_API prc_status project_kv_and_lr_cache(const uint16_t* X, int64_t T, int64_t d_in, int64_t ld_x,
                                           const uint16_t* W, int32_t n_kv_heads, int32_t head_dim,
                                           const uint16_t* A_stack, int32_t n_proj, int32_t n_agents,
                                           int32_t rank, double rope_theta, uint16_t* K_base, uint16_t* V_base,
                                           uint16_t* L_out, int64_t s_cap, int64_t tok_offset, void* stream) {
  return project_impl("project_kv_and_lr_cache", X, T, d_in, ld_x, W, n_kv_heads, head_dim, A_stack, n_proj,
                      n_agents, rank, rope_theta, K_base, V_base, L_out, s_cap, tok_offset, false, nullptr, 0, 0,
                      static_cast<hipStream_t>(stream));
}

PRC_API prc_status project_kv_and_lr_cache_paged(const uint16_t* X, int64_t T, int64_t d_in, int64_t ld_x,
                                                 const uint16_t* W, int32_t n_kv_heads, int32_t head_dim,
                                                 const uint16_t* A_stack, int32_t n_proj, int32_t n_agents,
                                                 int32_t rank, double rope_theta, uint16_t* K_pool,
                                                 uint16_t* V_pool, uint16_t* L_pool, const int32_t* block_table,
                                                 int32_t block_size, int32_t max_blocks, int32_t n_blocks,
                                                 int64_t tok_offset, void* stream) {
  if (block_size < 64 || block_size % 64)
    return fail(PRC_EUNSUPPORTED, "block_size=%d must be a positive multiple of 64", block_size);
  if (max_blocks < 1 || n_blocks < 1)
    return fail(PRC_EINVAL, "max_blocks=%d, n_blocks=%d must be positive", max_blocks, n_blocks);
  if ((int64_t)max_blocks * block_size > INT32_MAX || (int64_t)n_blocks * block_size > INT32_MAX)
    return fail(PRC_EINVAL, "max_blocks or n_blocks times block_size reaches 2^31 tokens");
  return project_impl("project_kv_and_lr_cache_paged", X, T, d_in, ld_x, W, n_kv_heads, head_dim, A_stack,
                      n_proj, n_agents, rank, rope_theta, K_pool, V_pool, L_pool,
                      (int64_t)max_blocks * block_size, tok_offset, true, block_table, block_size,
                      n_blocks, static_cast<hipStream_t>(stream));
}

namespace {

size_t workspace_size(const lrsa_dims* dims, bool paged, bool tile_cache = true) {
  if (dims == nullptr || dims->n_tok < 1 || dims->batch < 1 || dims->n_kv_heads < 1 || dims->s_cap < 1 ||
      dims->n_q_heads < dims->n_kv_heads)
    return 0;
  const int r = rank_ok(dims->rank) ? dims->rank : 8;
  if (dims->n_tok > 1) {
    // Prefill: partials of a split over the KV tiles, when the call is too
    // small to fill the GPU otherwise; then, for calls with enough row tiles
    // per KV head with an LR rank, the tile cache (room is asked for whenever
    // the rank is one of those, since dims do not say whether the call
    // brings L_k).
    int splits = 1, split_tiles = 0;
    const int group = dims->n_q_heads / dims->n_kv_heads;
    prc::prefill_plan(dims->n_tok, group, dims->n_kv_heads, dims->batch, dims->s_cap, plan_cus(), &splits,
                      &split_tiles);
    const size_t parts =
        prc::prefill_workspace_bytes(dims->batch, dims->n_tok, dims->n_q_heads, splits, dims->head_dim, r);
    if (tile_cache && !paged && rank_ok(dims->rank) &&
        prc::prefill_uses_tile_cache(dims->n_tok, group, dims->head_dim, dims->rank, true, true, paged)) {
      const size_t cache = prc::prefill_tile_cache_bytes(dims->batch, dims->n_kv_heads, dims->s_cap);
      if (cache > 0) return (parts + 255) / 256 * 256 + cache;
    }
    return parts;
  }
  int n_splits = 0, split_tiles = 0;
  // Paged caches always take the per-request decode kernel.
  const bool shared = !paged && prc::decode_shares_base(dims->batch, dims->kv_req_stride);
  prc::decode_plan(dims->s_cap, dims->batch, dims->n_kv_heads, dims->head_dim, r, shared, paged, plan_cus(), &n_splits,
                   &split_tiles);
  return prc::decode_workspace_bytes(dims->batch, dims->n_q_heads, n_splits, dims->head_dim, r);
}

prc_status attention_impl(const char* who, const lrsa_dims* dims, const lrsa_paging* pg, const uint16_t* Q,
                          const uint16_t* K_base, const uint16_t* V_base, const uint16_t* L_k, const uint16_t* L_v,
                          const uint16_t* B_k, const uint16_t* B_v, const int32_t* positions, const int32_t* kv_len,
                          uint16_t* O, float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  Checked c;
  prc_status s = check_attention(dims, Q, K_base, V_base, L_k, L_v, B_k, B_v, positions, kv_len, true, pg, &c);
  if (s != PRC_OK || c.empty) return s;
  if (O == nullptr) return fail(PRC_EINVAL, "O is NULL");
  if (!aligned(O, 16)) return fail(PRC_EALIGN, "O is not 16-byte aligned");
  if (lse != nullptr && !aligned(lse, 4)) return fail(PRC_EALIGN, "lse is not 4-byte aligned");
  prc::AttnArgs& a = c.a;
  a.O = O;
  a.lse = lse;
  // A rank outside the built set is only legal without LR; keep the size
  // query and the launch on the same effective rank.
  if (!rank_ok(dims->rank)) a.rank = 8;
  else a.rank = dims->rank;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char what[96];
  if (dims->n_tok == 1) {
    const size_t need = workspace_size(dims, pg != nullptr);
    if (workspace == nullptr || workspace_bytes < need)
      return fail(PRC_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace == nullptr ? 0 : workspace_bytes,
                  need);
    if (!aligned(workspace, 16)) return fail(PRC_EALIGN, "workspace is not 16-byte aligned");
    int cus = 0;
    if (prc_status ds = device_ready(&cus)) return ds;
#if PRC_DEVICE_CHECKS
    if (prc_status dc = device_data_check(who, positions, kv_len, a.batch, a.n_tok, a.s_cap, st)) return dc;
#endif
    prc::decode_plan(a.s_cap, a.batch, a.n_kv, a.head_dim, a.rank,
                     pg == nullptr && prc::decode_shares_base(a.batch, a.kv_stride), pg != nullptr, cus, &a.n_splits,
                     &a.split_tiles);
    a.ws = static_cast<float*>(workspace);
    snprintf(what, sizeof(what), "%s (decode)", who);
    return launch_status(prc::launch_decode(a, st), what);
  }
  const int plan_cu = plan_cus();
  prc::prefill_plan(a.n_tok, a.group, a.n_kv, a.batch, a.s_cap, plan_cu, &a.pf_splits, &a.pf_split_tiles);
  // Split partials first (required when the plan splits), then the tile
  // cache, taken when the workspace has room for it (a smaller or absent
  // workspace only means every workgroup rebuilds every tile).
  const size_t parts = prc::prefill_workspace_bytes(a.batch, a.n_tok, a.n_q, a.pf_splits, a.head_dim, a.rank);
  if (a.pf_splits > 1) {
    if (workspace == nullptr || workspace_bytes < parts)
      return fail(PRC_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace == nullptr ? 0 : workspace_bytes,
                  parts);
    if (!aligned(workspace, 16)) return fail(PRC_EALIGN, "workspace is not 16-byte aligned");
    a.ws = static_cast<float*>(workspace);
  }
  if (prc::prefill_uses_tile_cache(a.n_tok, a.group, a.head_dim, a.rank, L_k != nullptr, L_v != nullptr,
                                   pg != nullptr)) {
    const size_t off = (parts + 255) / 256 * 256;
    const size_t need = prc::prefill_tile_cache_bytes(a.batch, a.n_kv, a.s_cap);
    if (need > 0 && workspace != nullptr && workspace_bytes >= off + need && aligned(workspace, 256)) {
      const size_t fb = prc::prefill_tile_cache_flag_bytes(a.batch, a.n_kv, a.s_cap);
      char* base = static_cast<char*>(workspace) + off;
      a.tc_flags = reinterpret_cast<uint32_t*>(base);
      a.tc_data = reinterpret_cast<uint32_t*>(base + fb);
      a.tc_tiles = (int32_t)((a.s_cap + 63) / 64);
    }
  }
  int cus = 0;
  if (prc_status ds = device_ready(&cus)) return ds;
#if PRC_DEVICE_CHECKS
  if (prc_status dc = device_data_check(who, positions, kv_len, a.batch, a.n_tok, a.s_cap, st)) return dc;
#endif
  snprintf(what, sizeof(what), "%s (prefill)", who);
  return launch_status(prc::launch_prefill(a, st), what);
}

}  // namespace

namespace {

// Split partials of lr_shared_attention_noalloc: one array per device, held
// until the process ends.  Host code never passes `scratch` itself to a
// kernel or a copy (in host code its name is only a stand-in); it uses the
// device address fetched once per device below.
constexpr size_t kStaticWsBytes = (size_t)PRC_NOALLOC_WORKSPACE_BYTES;
static __device__ __align__(256) float scratch[kStaticWsBytes / sizeof(float)];
void* g_scratch_ptr[kMaxDevices];

// Device address of this device's `scratch`, fetched on the first call made
// with the device current.
prc_status static_workspace(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return fail(PRC_EDEVICE, "no HIP device is current");
  }
  std::lock_guard<std::mutex> lk(g_dev_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return fail(PRC_EDEVICE, "static workspace unavailable on device %d: %s", dev, hipGetErrorString(e));
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return PRC_OK;
}

}  // namespace

PRC_API size_t lr_shared_attention_workspace_size(const lrsa_dims* dims) { return workspace_size(dims, false); }

PRC_API prc_status lr_shared_attention_noalloc(const lrsa_dims* dims, const uint16_t* Q, const uint16_t* K_base,
                                               const uint16_t* V_base, const uint16_t* L_k, const uint16_t* L_v,
                                               const uint16_t* B_k, const uint16_t* B_v, const int32_t* positions,
                                               const int32_t* kv_len, uint16_t* O, float* lse, void* stream) {
  Checked c;
  prc_status s = check_attention(dims, Q, K_base, V_base, L_k, L_v, B_k, B_v, positions, kv_len, true, nullptr, &c);
  if (s != PRC_OK || c.empty) return s;
  // The split partials must fit; the tile cache is used when it fits too.
  const size_t need = workspace_size(dims, false, false);
  if (need > kStaticWsBytes)
    return fail(PRC_EWORKSPACE, "the call needs %zu bytes of split partials, above the %zu-byte static workspace",
                need, kStaticWsBytes);
  void* ws = nullptr;
  if (need > 0) {
    int cus = 0;
    if (prc_status ds = device_ready(&cus)) return ds;
    if (prc_status ss = static_workspace(&ws)) return ss;
  }
  return attention_impl("lr_shared_attention_noalloc", dims, nullptr, Q, K_base, V_base, L_k, L_v, B_k, B_v,
                        positions, kv_len, O, lse, ws, need > 0 ? kStaticWsBytes : 0, stream);
}

PRC_API size_t lr_shared_attention_paged_workspace_size(const lrsa_dims* dims) { return workspace_size(dims, true); }

PRC_API prc_status lr_shared_attention(const lrsa_dims* dims, const uint16_t* Q, const uint16_t* K_base,
                                       const uint16_t* V_base, const uint16_t* L_k, const uint16_t* L_v,
                                       const uint16_t* B_k, const uint16_t* B_v, const int32_t* positions,
                                       const int32_t* kv_len, uint16_t* O, float* lse, void* workspace,
                                       size_t workspace_bytes, void* stream) {
  return attention_impl("lr_shared_attention", dims, nullptr, Q, K_base, V_base, L_k, L_v, B_k, B_v, positions,
                        kv_len, O, lse, workspace, workspace_bytes, stream);
}

PRC_API prc_status lr_shared_attention_paged(const lrsa_dims* dims, const lrsa_paging* paging, const uint16_t* Q,
                                             const uint16_t* K_pool, const uint16_t* V_pool, const uint16_t* L_k,
                                             const uint16_t* L_v, const uint16_t* B_k, const uint16_t* B_v,
                                             const int32_t* positions, const int32_t* kv_len, uint16_t* O,
                                             float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  if (paging == nullptr) return fail(PRC_EINVAL, "paging is NULL");
  return attention_impl("lr_shared_attention_paged", dims, paging, Q, K_pool, V_pool, L_k, L_v, B_k, B_v, positions,
                        kv_len, O, lse, workspace, workspace_bytes, stream);
}

PRC_API prc_status materialize_agent_kv(const lrsa_dims* dims, const uint16_t* K_base, const uint16_t* V_base,
                                        const uint16_t* L_k, const uint16_t* L_v, const uint16_t* B_k,
                                        const uint16_t* B_v, const int32_t* kv_len, uint16_t* K_full,
                                        uint16_t* V_full, void* stream) {
  Checked c;
  prc_status s = check_attention(dims, nullptr, K_base, V_base, L_k, L_v, B_k, B_v, nullptr, kv_len, false, nullptr, &c);
  if (s != PRC_OK || c.empty) return s;
  if (K_full == nullptr || V_full == nullptr) return fail(PRC_EINVAL, "K_full/V_full is NULL");
  if (!aligned(K_full, 16) || !aligned(V_full, 16)) return fail(PRC_EALIGN, "K_full/V_full not 16-byte aligned");
  // Outputs must not overlap any input.  Each output spans batch * s_cap
  // rows; each input its requests' extents (a request stride of 0 means one
  // buffer for all).
  const int64_t nkvd = (int64_t)dims->n_kv_heads * dims->head_dim;
  const int64_t r = c.a.rank;
  const int64_t nb = dims->batch;
  auto extent = [&](int64_t stride, int64_t per_req) -> uintptr_t {
    const int64_t reqs = stride == 0 ? 1 : nb;
    return (uintptr_t)(((reqs - 1) * stride + per_req) * 2);
  };
  const uintptr_t out_bytes = (uintptr_t)nb * dims->s_cap * nkvd * 2;
  struct Span {
    const void* p;
    uintptr_t bytes;
  } ins[] = {{K_base, extent(dims->kv_req_stride, dims->s_cap * nkvd)},
             {V_base, extent(dims->kv_req_stride, dims->s_cap * nkvd)},
             {L_k, extent(dims->l_req_stride, dims->s_cap * r)},
             {L_v, extent(dims->l_req_stride, dims->s_cap * r)},
             {B_k, extent(dims->b_req_stride, nkvd * r)},
             {B_v, extent(dims->b_req_stride, nkvd * r)}};
  auto overlap = [](uintptr_t a0, uintptr_t an, uintptr_t b0, uintptr_t bn) { return a0 < b0 + bn && b0 < a0 + an; };
  for (const void* o : {static_cast<const void*>(K_full), static_cast<const void*>(V_full)}) {
    const uintptr_t o0 = reinterpret_cast<uintptr_t>(o);
    for (const Span& in : ins)
      if (in.p != nullptr && overlap(o0, out_bytes, reinterpret_cast<uintptr_t>(in.p), in.bytes))
        return fail(PRC_EINVAL, "K_full/V_full overlap an input");
  }
  if (overlap(reinterpret_cast<uintptr_t>(K_full), out_bytes, reinterpret_cast<uintptr_t>(V_full), out_bytes))
    return fail(PRC_EINVAL, "K_full and V_full overlap");
  int cus = 0;
  if (prc_status ds = device_ready(&cus)) return ds;
#if PRC_DEVICE_CHECKS
  if (prc_status dc = device_data_check("materialize_agent_kv", nullptr, kv_len, c.a.batch, 0, c.a.s_cap,
                                        static_cast<hipStream_t>(stream)))
    return dc;
#endif
  c.a.Kout = K_full;
  c.a.Vout = V_full;
  return launch_status(prc::launch_materialize(c.a, static_cast<hipStream_t>(stream)), "materialize_agent_kv");
}

PRC_API prc_status prc_stream_read(const void* src, size_t bytes, uint32_t* sink, int32_t grid, void* stream) {
  if (src == nullptr || sink == nullptr) return fail(PRC_EINVAL, "src/sink is NULL");
  if (bytes == 0 || bytes % 16 || bytes > ((size_t)1 << 40)) return fail(PRC_EINVAL, "bytes=%zu must be a positive multiple of 16", bytes);
  if (!aligned(src, 16) || !aligned(sink, 4)) return fail(PRC_EALIGN, "src must be 16-byte and sink 4-byte aligned");
  if (grid < 1 || grid > (1 << 20)) return fail(PRC_EINVAL, "grid=%d outside [1, 2^20]", grid);
  int cus = 0;
  if (prc_status ds = device_ready(&cus)) return ds;
  return launch_status(prc::launch_stream_read(src, (int64_t)bytes, sink, grid, static_cast<hipStream_t>(stream)),
                       "prc_stream_read");
}
