// Gating (§2.1): gate logits, top-k selection and renormalised gate weights.
//
// One wave per token. In weight mode each lane accumulates its stride of the
// hidden dimension in float64 for 8 experts at a time (bf16*bf16 products
// are exact in float64), a butterfly reduction gives every lane the full
// sums, and the float64 sum is rounded once to float32. Top-k runs as k
// rounds of a wave arg-max over the float32 logits (larger first, ties to
// the lower expert id); lane 0 then forms the weights in rank order.
#include "tg_device.h"
#include "tg_launch.h"

namespace tg {
namespace {

constexpr int kTokPerBlock = 4;  // waves per block
constexpr int kMaxEPerLane = 16; // E <= 1024

__device__ __forceinline__ bool better(float v, int id, float bv, int bid) {
  return v > bv || (v == bv && id < bid);
}

// Top-k over the logits held in `lg` (LDS, E floats) by one wave, writing
// ids and weights for token t.
__device__ void wave_topk(const float* lg, int E, int k, int t, int32_t* ids, float* w,
                          float* top_v /*LDS, k floats*/, int* top_id /*LDS, k ints*/) {
  const int lane = lane_id();
  float v[kMaxEPerLane];
  uint32_t taken = 0;
  const int nq = (E + kWave - 1) / kWave;
#pragma unroll
  for (int q = 0; q < kMaxEPerLane; ++q) {
    const int e = lane + q * kWave;
    v[q] = (q < nq && e < E) ? lg[e] : 0.0f;
  }
  for (int j = 0; j < k; ++j) {
    float bv = -__builtin_inff();
    int bid = 0x7fffffff;
#pragma unroll
    for (int q = 0; q < kMaxEPerLane; ++q) {
      const int e = lane + q * kWave;
      if (q < nq && e < E && !(taken & (1u << q)) && better(v[q], e, bv, bid)) {
        bv = v[q];
        bid = e;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float ov = __shfl_xor(bv, off);
      const int oid = __shfl_xor(bid, off);
      if (better(ov, oid, bv, bid)) {
        bv = ov;
        bid = oid;
      }
    }
    if ((bid % kWave) == lane) taken |= 1u << (bid / kWave);
    if (lane == 0) {
      top_v[j] = bv;
      top_id[j] = bid;
    }
  }
  __builtin_amdgcn_wave_barrier();
  if (lane == 0) {
    const float v0 = top_v[0];
    float z = 0.0f;
    for (int j = 0; j < k; ++j) z += expf(top_v[j] - v0);
    for (int j = 0; j < k; ++j) {
      ids[(size_t)t * k + j] = top_id[j];
      w[(size_t)t * k + j] = expf(top_v[j] - v0) / z;
    }
  }
}

__global__ __launch_bounds__(256) void gate_weights_topk_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg, int T, int d, int E, int k,
    float* __restrict__ logits_out, int32_t* __restrict__ ids, float* __restrict__ w) {
  extern __shared__ float smem[];  // [kTokPerBlock][E] logits + [kTokPerBlock][32] top values/ids
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int t = blockIdx.x * kTokPerBlock + wave;
  float* lg = smem + wave * E;
  float* top_v = smem + kTokPerBlock * E + wave * 64;
  int* top_id = reinterpret_cast<int*>(top_v + 32);
  if (t >= T) return;  // whole wave leaves together; no block barrier below
  const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)t * d);
  const int nchunk = d / 8;
  for (int e0 = 0; e0 < E; e0 += 8) {
    double acc[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = 0.0;
    for (int c = lane; c < nchunk; c += kWave) {
      const uint4 xv = xr[c];
      const uint32_t xs[4] = {xv.x, xv.y, xv.z, xv.w};
      double xd[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        xd[2 * i] = (double)__uint_as_float(xs[i] << 16);
        xd[2 * i + 1] = (double)__uint_as_float(xs[i] & 0xffff0000u);
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int e = e0 + q;
        if (e < E) {
          const uint4 wv = reinterpret_cast<const uint4*>(wg + (size_t)e * d)[c];
          const uint32_t ws[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            acc[q] = fma(xd[2 * i], (double)__uint_as_float(ws[i] << 16), acc[q]);
            acc[q] = fma(xd[2 * i + 1], (double)__uint_as_float(ws[i] & 0xffff0000u), acc[q]);
          }
        }
      }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) acc[q] += __shfl_xor(acc[q], off);
    }
    if (lane == 0) {
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (e0 + q < E) lg[e0 + q] = (float)acc[q];
    }
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  if (logits_out) {
    for (int e = lane; e < E; e += kWave) logits_out[(size_t)t * E + e] = lg[e];
  }
  wave_topk(lg, E, k, t, ids, w, top_v, top_id);
}

__global__ __launch_bounds__(256) void logits_topk_kernel(const float* __restrict__ logits, int T,
                                                          int E, int k, int32_t* __restrict__ ids,
                                                          float* __restrict__ w) {
  extern __shared__ float smem[];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int t = blockIdx.x * kTokPerBlock + wave;
  float* lg = smem + wave * E;
  float* top_v = smem + kTokPerBlock * E + wave * 64;
  int* top_id = reinterpret_cast<int*>(top_v + 32);
  if (t >= T) return;
  for (int e = lane; e < E; e += kWave) lg[e] = logits[(size_t)t * E + e];
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  wave_topk(lg, E, k, t, ids, w, top_v, top_id);
}

}  // namespace

hipError_t launch_gate_topk(const uint16_t* x, const uint16_t* wg, const float* logits_in, int T,
                            int d, int E, int k, float* logits_out, int32_t* ids, float* w,
                            hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const dim3 grid((T + kTokPerBlock - 1) / kTokPerBlock);
  const size_t lds = (size_t)kTokPerBlock * (E + 64) * sizeof(float);
  if (logits_in) {
    hipLaunchKernelGGL(logits_topk_kernel, grid, dim3(256), lds, stream, logits_in, T, E, k, ids, w);
  } else {
    hipLaunchKernelGGL(gate_weights_topk_kernel, grid, dim3(256), lds, stream, x, wg, T, d, E, k,
                       logits_out, ids, w);
  }
  return hipGetLastError();
}

}  // namespace tg
