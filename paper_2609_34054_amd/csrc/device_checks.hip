// Checks of the values the host cannot see, for the checked build of the
// library (libprecache_checked.so): kv_len[b] must lie in [1, s_cap] and every
// query position in [0, kv_len[b]) (the causal prefix of Sec. 2.2 is then
// never empty and never reaches past the cache).  The release build trusts
// these values; its kernels only clamp kv_len into [0, s_cap].
//
// One workgroup walks all requests and query tokens and records the first
// offender in a fixed order (requests first, then tokens), so the report does
// not depend on scheduling.  The result goes to a small per-device array that
// the host reads back before it launches the call's kernels.
#include "common.hpp"
#include "kernels.hpp"

namespace prc {
namespace {

constexpr int DC_THREADS = 256;

// result[0]: 0 all valid, 1 kv_len out of range, 2 position out of range;
// result[1]: request; result[2]: query token; result[3]: the offending value.
static __device__ __align__(16) int32_t check_result[4];

__global__ void __launch_bounds__(DC_THREADS)
device_checks_kernel(const int32_t* positions, const int32_t* kv_len, int batch, int n_tok, int64_t s_cap,
                     int32_t* result) {
  // First offender as one linear key: kv_len faults of request b sort before
  // every position fault, position faults by (b, i).
  __shared__ long long first;
  if (threadIdx.x == 0) first = LLONG_MAX;
  __syncthreads();
  const long long per_req = (long long)n_tok + 1;
  for (int b = threadIdx.x; b < batch; b += DC_THREADS) {
    const int32_t k = kv_len[b];
    if (k < 1 || (int64_t)k > s_cap) atomicMin(&first, (long long)b * per_req);
  }
  if (positions != nullptr) {
    const long long n = (long long)batch * n_tok;
    for (long long e = threadIdx.x; e < n; e += DC_THREADS) {
      const int b = (int)(e / n_tok), i = (int)(e - (long long)b * n_tok);
      const int32_t p = positions[e], k = kv_len[b];
      if (p < 0 || p >= k) atomicMin(&first, (long long)b * per_req + 1 + i);
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t out[4] = {0, 0, 0, 0};
    if (first != LLONG_MAX) {
      const int b = (int)(first / per_req), j = (int)(first - (long long)b * per_req);
      out[0] = j == 0 ? 1 : 2;
      out[1] = b;
      out[2] = j == 0 ? 0 : j - 1;
      out[3] = j == 0 ? kv_len[b] : positions[(long long)b * n_tok + (j - 1)];
    }
    *reinterpret_cast<i32x4*>(result) = i32x4{out[0], out[1], out[2], out[3]};
  }
}

}  // namespace

hipError_t device_checks_result(int32_t** ptr) {
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(check_result));
  *ptr = static_cast<int32_t*>(p);
  return e;
}

hipError_t launch_device_checks(const int32_t* positions, const int32_t* kv_len, int batch, int n_tok, int64_t s_cap,
                                int32_t* result, hipStream_t st) {
  hipLaunchKernelGGL(device_checks_kernel, dim3(1), dim3(DC_THREADS), 0, st, positions, kv_len, batch, n_tok, s_cap,
                     result);
  return hipGetLastError();
}

}  // namespace prc
