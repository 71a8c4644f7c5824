// EW-side partial-batch trigger (§5.2).
//
// The EW's receive buffer holds the token rows of A attention workers (AWs)
// as consecutive chunks. One block of 1024 threads, thread a owning AW a,
// polls the per-AW "delivered" flags with system-scope loads (the flags may
// live in device memory or in host memory that the transport writes while
// the kernel waits) until every live AW has delivered, or the delivered rows
// of live AWs reach the minimum batch, or the poll budget (the probing
// window) is spent. Every poll is a block-wide vote, so all threads take the
// same decision at the same poll; the loop ends after at most spin_limit
// polls. The batch is then the rows of the AWs that were live and had
// delivered at that poll; token_valid marks them.
#include "tg_device.h"
#include "tg_launch.h"

namespace tg {
namespace {

constexpr int kBlock = 1024;

__device__ __forceinline__ uint32_t load_flag(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__global__ __launch_bounds__(kBlock) void batch_trigger_kernel(
    const uint32_t* delivered, const uint8_t* __restrict__ aw_alive,
    const int32_t* __restrict__ chunk_rows, int A, int T, int min_rows, long long spin_limit,
    uint8_t* __restrict__ token_valid, int32_t* __restrict__ status) {
  __shared__ int rows_sum;
  const int a = threadIdx.x;
  const bool live = a < A && aw_alive[a];
  int lo = 0, hi = 0;
  if (a < A) {
    lo = min(max(chunk_rows[a], 0), T);
    hi = min(max(chunk_rows[a + 1], lo), T);
  }
  long long polls = 0;
  int reason = 2, rows = 0;
  bool got = false;
  for (;;) {
    if (a == 0) rows_sum = 0;
    got = live && load_flag(delivered + a) != 0;
    const int pending = __syncthreads_count(live && !got);
    if (got && hi > lo) atomicAdd(&rows_sum, hi - lo);
    __syncthreads();
    rows = rows_sum;
    ++polls;
    __syncthreads();  // every thread has read rows_sum before the next reset
    if (pending == 0) {
      reason = 0;
      break;
    }
    if (rows >= min_rows) {
      reason = 1;
      break;
    }
    if (polls >= spin_limit) break;
    __builtin_amdgcn_s_sleep(127);
  }
  __shared__ int lo_s[kBlock], hi_s[kBlock];
  lo_s[a] = got ? lo : 0;
  hi_s[a] = got ? hi : 0;  // empty range for AWs outside the batch
  const int n_aws = __syncthreads_count(got);
  for (int t = a; t < T; t += kBlock) token_valid[t] = 0;
  __syncthreads();
  for (int b = 0; b < A; ++b)
    for (int t = lo_s[b] + a; t < hi_s[b]; t += kBlock) token_valid[t] = 1;
  if (a == 0) {
    status[0] = reason;
    status[1] = rows;
    status[2] = n_aws;
    status[3] = (int)min(polls, (long long)0x7fffffff);
  }
}

}  // namespace

hipError_t launch_batch_trigger(const uint32_t* delivered, const uint8_t* aw_alive,
                                const int32_t* chunk_rows, int A, int T, int min_rows,
                                long long spin_limit, uint8_t* token_valid, int32_t* status,
                                hipStream_t stream) {
  hipLaunchKernelGGL(batch_trigger_kernel, dim3(1), dim3(kBlock), 0, stream, delivered, aw_alive,
                     chunk_rows, A, T, min_rows, spin_limit, token_valid, status);
  return hipGetLastError();
}

}  // namespace tg
