// Incremental KV-segment checkpoint and request-level restoration (§6.1,
// §6.2), with host memory in the role of the checkpoint store.
//
// Two ways to copy: a kernel over an arbitrary list of segments, on a
// bounded number of workgroups; and, for segments at a constant stride (one
// decode step of a [layer][request][position] region), one strided copy on
// the copy engine, which leaves the compute units to the forward.
//
// The KV region and the store have the same layout, so a segment's offset
// in the region is its offset in the store. A checkpoint call copies a batch
// of segments (one block per segment at a time, 16-byte loads and stores
// straight into host-visible memory), writes one log record per segment,
// makes its writes visible system-wide, and then, in a second kernel that
// starts only after every copy has finished, publishes the commit record:
// the sequence number after the batch's last, so every number below it has
// landed. Restoration copies back only the segments numbered below the
// commit record.
#include "tg.h"
#include "tg_device.h"
#include "tg_launch.h"

namespace tg {
namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ bool seg_ok(uint64_t off, uint64_t bytes, uint64_t limit) {
  return (off % 16 == 0) && (bytes % 16 == 0) && off <= limit && bytes <= limit - off;
}

__global__ __launch_bounds__(kBlock) void ckpt_copy_kernel(
    const uint4* __restrict__ kv, uint64_t kv_bytes, const uint64_t* __restrict__ seg_off,
    const uint32_t* __restrict__ seg_bytes, int n, uint64_t first_seq, uint4* store,
    tg_ckpt_record* log, int log_cap) {
  for (int i = blockIdx.x; i < n; i += gridDim.x) {
    const uint64_t o = seg_off[i];
    const uint32_t b = seg_bytes[i];
    const bool ok = seg_ok(o, b, kv_bytes);
    if (ok) {
      const uint64_t base = o / 16;
      for (uint32_t c = threadIdx.x; c < b / 16; c += kBlock) store[base + c] = kv[base + c];
    }
    // The log is a ring of log_cap records: of a batch longer than the ring
    // only the last log_cap records are kept, so no two writes collide.
    if (threadIdx.x == 0 && i >= n - log_cap) {
      tg_ckpt_record r;
      r.seq = first_seq + (uint64_t)i;
      r.offset = o;
      r.bytes = ok ? b : 0;  // 0: rejected (misaligned or outside the region)
      log[r.seq % (uint64_t)log_cap] = r;
    }
  }
  __threadfence_system();
}

__global__ void ckpt_commit_kernel(uint64_t* commit, uint64_t seq) {
  __threadfence_system();
  __hip_atomic_store(commit, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Records of a strided batch (segment i at first_offset + i * pitch), then,
// after every record, the commit record; one block.
__global__ __launch_bounds__(kBlock) void ckpt_log_commit_kernel(
    uint64_t first_offset, uint64_t pitch, uint32_t seg_bytes, int n, uint64_t first_seq,
    tg_ckpt_record* log, int log_cap, uint64_t* commit) {
  for (int i = max(0, n - log_cap) + threadIdx.x; i < n; i += kBlock) {
    tg_ckpt_record r;
    r.seq = first_seq + (uint64_t)i;
    r.offset = first_offset + (uint64_t)i * pitch;
    r.bytes = seg_bytes;
    log[r.seq % (uint64_t)log_cap] = r;
  }
  __threadfence_system();
  __syncthreads();
  if (commit && threadIdx.x == 0)
    __hip_atomic_store(commit, first_seq + (uint64_t)n, __ATOMIC_RELEASE,
                       __HIP_MEMORY_SCOPE_SYSTEM);
}

__global__ __launch_bounds__(kBlock) void kv_restore_kernel(
    const uint4* store, uint64_t store_bytes, const uint64_t* commit,
    const uint64_t* __restrict__ seq, const uint64_t* __restrict__ src,
    const uint64_t* __restrict__ dst, const uint32_t* __restrict__ bytes, int n,
    uint4* __restrict__ kv, uint64_t kv_bytes, uint8_t* __restrict__ status) {
  const uint64_t committed = __hip_atomic_load(commit, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM);
  for (int i = blockIdx.x; i < n; i += gridDim.x) {
    const uint32_t b = bytes[i];
    uint8_t st;
    if (!seg_ok(src[i], b, store_bytes) || !seg_ok(dst[i], b, kv_bytes)) {
      st = 2;
    } else if (seq[i] >= committed) {
      st = 0;  // not committed: its bytes may be incomplete
    } else {
      st = 1;
      const uint64_t s0 = src[i] / 16, d0 = dst[i] / 16;
      for (uint32_t c = threadIdx.x; c < b / 16; c += kBlock) kv[d0 + c] = store[s0 + c];
    }
    if (threadIdx.x == 0) status[i] = st;
  }
}

int grid_for(int n, int max_blocks) { return n < max_blocks ? n : max_blocks; }

}  // namespace

hipError_t launch_kv_checkpoint(const void* kv, size_t kv_bytes, const uint64_t* seg_off,
                                const uint32_t* seg_bytes, int n, uint64_t first_seq, void* store,
                                tg_ckpt_record* log, int log_cap, uint64_t* commit, int max_blocks,
                                hipStream_t stream) {
  if (n > 0)
    hipLaunchKernelGGL(ckpt_copy_kernel, dim3(grid_for(n, max_blocks)), dim3(kBlock), 0, stream,
                       static_cast<const uint4*>(kv), (uint64_t)kv_bytes, seg_off, seg_bytes, n,
                       first_seq, static_cast<uint4*>(store), log, log_cap);
  if (commit && n > 0)
    hipLaunchKernelGGL(ckpt_commit_kernel, dim3(1), dim3(1), 0, stream, commit,
                       first_seq + (uint64_t)n);
  return hipGetLastError();
}

hipError_t launch_kv_checkpoint_strided(const void* kv, uint64_t first_offset, uint64_t pitch,
                                        uint32_t seg_bytes, int n, uint64_t first_seq,
                                        void* store, tg_ckpt_record* log, int log_cap,
                                        uint64_t* commit, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  // One strided copy by the copy engine: no compute unit is used. The store
  // has the region's layout, so source and destination share the pitch.
  hipError_t e = hipMemcpy2DAsync(static_cast<char*>(store) + first_offset, pitch,
                                  static_cast<const char*>(kv) + first_offset, pitch, seg_bytes, n,
                                  hipMemcpyDefault, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(ckpt_log_commit_kernel, dim3(1), dim3(kBlock), 0, stream, first_offset, pitch,
                     seg_bytes, n, first_seq, log, log_cap, commit);
  return hipGetLastError();
}

hipError_t launch_kv_restore(const void* store, size_t store_bytes, const uint64_t* commit,
                             const uint64_t* seq, const uint64_t* src, const uint64_t* dst,
                             const uint32_t* bytes, int n, void* kv, size_t kv_bytes,
                             uint8_t* status, hipStream_t stream) {
  if (n > 0)
    hipLaunchKernelGGL(kv_restore_kernel, dim3(grid_for(n, 4096)), dim3(kBlock), 0, stream,
                       static_cast<const uint4*>(store), (uint64_t)store_bytes, commit, seq, src,
                       dst, bytes, n, static_cast<uint4*>(kv), (uint64_t)kv_bytes, status);
  return hipGetLastError();
}

}  // namespace tg
