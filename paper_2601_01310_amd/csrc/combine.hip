// Gate-weighted combine (§2.1): out[t] = bf16(sum_j w[t,j] * y[pair_row[t,j]])
// in float32, in rank order j = 0..k-1, skipping pairs not routed here; and
// the merge step of a replay (§5.1), which re-forms the same sum for the
// tokens whose pairs were recomputed on another slot.
// One block per token; threads own 8-element (16-byte) column chunks, so a
// token's k rows are read and its output row written fully coalesced.
#include "tg_device.h"
#include "tg_launch.h"

namespace tg {
namespace {

constexpr int kMaxBlock = 1024;

// rows[j] >= 0: y row; rows[j] <= -2: row -rows[j]-2 of y2; -1: no output.
__device__ __forceinline__ void combine_row(const uint4* __restrict__ y,
                                            const uint4* __restrict__ y2, const int* rows,
                                            const float* ws, int t, int k, int nch,
                                            uint4* __restrict__ out) {
  for (int c = threadIdx.x; c < nch; c += blockDim.x) {
    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
    for (int j = 0; j < k; ++j) {
      const int r = rows[j];
      if (r == -1) continue;
      const float wj = ws[j];
      const uint4 v = (r >= 0) ? y[(size_t)r * nch + c] : y2[(size_t)(-r - 2) * nch + c];
      const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] = fmaf(wj, __uint_as_float(u[i] << 16), acc[2 * i]);
        acc[2 * i + 1] = fmaf(wj, __uint_as_float(u[i] & 0xffff0000u), acc[2 * i + 1]);
      }
    }
    uint4 o;
    o.x = pack_bf16x2(acc[0], acc[1]);
    o.y = pack_bf16x2(acc[2], acc[3]);
    o.z = pack_bf16x2(acc[4], acc[5]);
    o.w = pack_bf16x2(acc[6], acc[7]);
    out[(size_t)t * nch + c] = o;
  }
}

__global__ __launch_bounds__(kMaxBlock) void combine_kernel(const uint4* __restrict__ y,
                                                         const int32_t* __restrict__ pair_row,
                                                         const float* __restrict__ w, int T, int k,
                                                         int nch, uint4* __restrict__ out) {
  __shared__ int rows[32];
  __shared__ float ws[32];
  const int t = blockIdx.x;
  if (threadIdx.x < k) {
    const int r = pair_row[(size_t)t * k + threadIdx.x];
    rows[threadIdx.x] = r < 0 ? -1 : r;
    ws[threadIdx.x] = w[(size_t)t * k + threadIdx.x];
  }
  __syncthreads();
  combine_row(y, nullptr, rows, ws, t, k, nch, out);
}

// One block per token; tokens whose pairs all keep their first-pass result
// return at once.
__global__ __launch_bounds__(kMaxBlock) void recombine_kernel(
    const uint4* __restrict__ y, const int32_t* __restrict__ pair_row,
    const int32_t* __restrict__ prior, const uint8_t* __restrict__ alive, int S,
    const uint4* __restrict__ y2, const int32_t* __restrict__ replay_row,
    const float* __restrict__ w, int T, int k, int nch, uint4* __restrict__ out) {
  __shared__ int rows[32];
  __shared__ float ws[32];
  __shared__ int changed;
  const int t = blockIdx.x;
  if (threadIdx.x == 0) changed = 0;
  __syncthreads();
  if (threadIdx.x < k) {
    const size_t p = (size_t)t * k + threadIdx.x;
    const int rr = replay_row[p];
    const int ps = prior[p];
    int r = -1;
    if (rr >= 0) {
      r = -rr - 2;
      atomicOr(&changed, 1);
    } else if (ps >= 0 && ps < S) {
      if (alive[ps]) r = pair_row[p];
      else atomicOr(&changed, 1);  // lost: its output leaves the sum
    }
    rows[threadIdx.x] = r;
    ws[threadIdx.x] = w[p];
  }
  __syncthreads();
  if (!changed) return;
  combine_row(y, y2, rows, ws, t, k, nch, out);
}

}  // namespace

// Threads per block. Few tokens (a decode step): one thread per 16-byte
// chunk of a row, in whole waves, so each block issues all its loads at
// once. Many tokens: 256 threads looping over the chunks, which keeps more
// blocks resident per CU.
static int combine_block(int T, int d) {
  if (T > 2048) return 256;
  const int nch = d / 8;
  const int b = (nch + kWave - 1) / kWave * kWave;
  return b < kMaxBlock ? b : kMaxBlock;
}

hipError_t launch_combine(const uint16_t* y, const int32_t* pair_row, const float* w, int T, int k,
                          int d, uint16_t* out, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  hipLaunchKernelGGL(combine_kernel, dim3(T), dim3(combine_block(T, d)), 0, stream,
                     reinterpret_cast<const uint4*>(y), pair_row, w, T, k, d / 8,
                     reinterpret_cast<uint4*>(out));
  return hipGetLastError();
}

hipError_t launch_recombine(const uint16_t* y, const int32_t* pair_row, const int32_t* prior_slot,
                            const uint8_t* alive, int S, const uint16_t* y2,
                            const int32_t* replay_row, const float* w, int T, int k, int d,
                            uint16_t* out, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  hipLaunchKernelGGL(recombine_kernel, dim3(T), dim3(combine_block(T, d)), 0, stream,
                     reinterpret_cast<const uint4*>(y), pair_row, prior_slot, alive, S,
                     reinterpret_cast<const uint4*>(y2), replay_row, w, T, k, d / 8,
                     reinterpret_cast<uint4*>(out));
  return hipGetLastError();
}

}  // namespace tg
