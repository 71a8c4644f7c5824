// Gate-weighted combine (§2.1): out[t] = bf16(sum_j w[t,j] * y[pair_row[t,j]])
// in float32, in rank order j = 0..k-1, skipping pairs not routed here; and
// the merge step of a replay (§5.1), which re-forms the same sum for the
// tokens whose pairs were recomputed on another slot.
// One block per token; threads own 8-element (16-byte) column chunks, so a
// token's rows are read and its output row written fully coalesced.
#include "tg_device.h"
#include "tg_launch.h"

namespace tg {
namespace {

constexpr int kMaxBlock = 1024;

// The token's nv contributing pairs, in rank order: rows[j] >= 0 is a row
// of y, rows[j] <= -2 row -rows[j]-2 of y2. Each thread takes kU column
// chunks at once and issues all their loads before the first FMA, so a
// block keeps kU * nv 16-byte loads per thread in flight (kU = 4 for many
// tokens; 1 for few, where one thread per chunk is the better shape).
template <int kU>
__device__ __forceinline__ void combine_row(const uint4* __restrict__ y,
                                            const uint4* __restrict__ y2, const int* rows,
                                            const float* ws, int nv, int t, int nch,
                                            uint4* __restrict__ out) {
  for (int c0 = threadIdx.x; c0 < nch; c0 += blockDim.x * kU) {
    float acc[kU][8];
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[u][i] = 0.0f;
    for (int j = 0; j < nv; ++j) {
      const int r = rows[j];
      const float wj = ws[j];
      const uint4* src = (r >= 0) ? y + (size_t)r * nch : y2 + (size_t)(-r - 2) * nch;
      uint4 v[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int c = c0 + u * blockDim.x;
        v[u] = (c < nch) ? src[c] : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const uint32_t uu[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[u][2 * i] = fmaf(wj, __uint_as_float(uu[i] << 16), acc[u][2 * i]);
          acc[u][2 * i + 1] = fmaf(wj, __uint_as_float(uu[i] & 0xffff0000u), acc[u][2 * i + 1]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int c = c0 + u * blockDim.x;
      if (c < nch) {
        uint4 o;
        o.x = pack_bf16x2(acc[u][0], acc[u][1]);
        o.y = pack_bf16x2(acc[u][2], acc[u][3]);
        o.z = pack_bf16x2(acc[u][4], acc[u][5]);
        o.w = pack_bf16x2(acc[u][6], acc[u][7]);
        out[(size_t)t * nch + c] = o;
      }
    }
  }
}

// Keeps the entries of rows_in / ws_in (k <= 32, in LDS) that are not -1,
// in order; returns their number (every thread gets it).
__device__ __forceinline__ int compact_rows(const int* rows_in, const float* ws_in, int k,
                                            int* rows, float* ws) {
  int nv = 0;
  for (int j = 0; j < k; ++j) {
    if (rows_in[j] != -1) {
      rows[nv] = rows_in[j];
      ws[nv] = ws_in[j];
      ++nv;
    }
  }
  return nv;
}

template <int kU>
__global__ __launch_bounds__(kMaxBlock) void combine_kernel(const uint4* __restrict__ y,
                                                         const int32_t* __restrict__ pair_row,
                                                         const float* __restrict__ w, int T, int k,
                                                         int nch, uint4* __restrict__ out) {
  __shared__ int rows_in[32], rows[32];
  __shared__ float ws_in[32], ws[32];
  __shared__ int nv_s;
  const int t = blockIdx.x;
  if (threadIdx.x < k) {
    const int r = pair_row[(size_t)t * k + threadIdx.x];
    rows_in[threadIdx.x] = r < 0 ? -1 : r;
    ws_in[threadIdx.x] = w[(size_t)t * k + threadIdx.x];
  }
  __syncthreads();
  if (threadIdx.x == 0) nv_s = compact_rows(rows_in, ws_in, k, rows, ws);
  __syncthreads();
  combine_row<kU>(y, nullptr, rows, ws, nv_s, t, nch, out);
}

// One block per token; tokens whose pairs all keep their first-pass result
// return at once.
template <int kU>
__global__ __launch_bounds__(kMaxBlock) void recombine_kernel(
    const uint4* __restrict__ y, const int32_t* __restrict__ pair_row,
    const int32_t* __restrict__ prior, const uint8_t* __restrict__ alive, int S,
    const uint4* __restrict__ y2, const int32_t* __restrict__ replay_row,
    const float* __restrict__ w, int T, int k, int nch, uint4* __restrict__ out) {
  __shared__ int rows_in[32], rows[32];
  __shared__ float ws_in[32], ws[32];
  __shared__ int changed, nv_s;
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
    rows_in[threadIdx.x] = r;
    ws_in[threadIdx.x] = w[p];
  }
  __syncthreads();
  if (!changed) return;
  if (threadIdx.x == 0) nv_s = compact_rows(rows_in, ws_in, k, rows, ws);
  __syncthreads();
  combine_row<kU>(y, y2, rows, ws, nv_s, t, nch, out);
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
  hipLaunchKernelGGL(T > 2048 ? combine_kernel<4> : combine_kernel<1>, dim3(T),
                     dim3(combine_block(T, d)), 0, stream,
                     reinterpret_cast<const uint4*>(y), pair_row, w, T, k, d / 8,
                     reinterpret_cast<uint4*>(out));
  return hipGetLastError();
}

hipError_t launch_recombine(const uint16_t* y, const int32_t* pair_row, const int32_t* prior_slot,
                            const uint8_t* alive, int S, const uint16_t* y2,
                            const int32_t* replay_row, const float* w, int T, int k, int d,
                            uint16_t* out, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  hipLaunchKernelGGL(T > 2048 ? recombine_kernel<4> : recombine_kernel<1>, dim3(T),
                     dim3(combine_block(T, d)), 0, stream,
                     reinterpret_cast<const uint4*>(y), pair_row, prior_slot, alive, S,
                     reinterpret_cast<const uint4*>(y2), replay_row, w, T, k, d / 8,
                     reinterpret_cast<uint4*>(out));
  return hipGetLastError();
}

}  // namespace tg
