// Gating (§2.1): gate logits, top-k selection and renormalised gate weights.
//
// One wave per token at a time. In weight mode each lane accumulates its
// stride of the hidden dimension in float64 for 8 experts at a time
// (bf16*bf16 products are exact in float64), a butterfly reduction gives
// every lane the full sums, and the float64 sum is rounded once to float32.
// When the gate matrix fits (E*d*2 <= 96 KB) a block of 16 waves (16
// tokens) stages it in LDS once, so the matrix is read from memory once per
// 16 tokens instead of once per token. Top-k runs as k rounds of a wave
// arg-max over the float32 logits (larger first, ties to the lower expert
// id); lane j keeps the j-th winner, the k exponentials are formed in
// parallel and summed in rank order.
#include "tg_device.h"
#include "tg_launch.h"

namespace tg {
namespace {

constexpr int kWaves = 4;          // waves per block (unstaged kernels)
constexpr int kMaxEPerLane = 16;   // E <= 1024
constexpr int kStagedWaves = 16;   // waves (= tokens) per block when the gate matrix is staged
constexpr int kStageElems = 48 * 1024;  // 96 KB of bf16
constexpr int kStagedMaxE = kStageElems / 256;  // staged only when E * d fits, d >= 256

__device__ __forceinline__ bool better(float v, int id, float bv, int bid) {
  return v > bv || (v == bv && id < bid);
}

// Top-k over the logits held in `lg` (LDS, E floats) by one wave; writes
// ids and weights of token t.
__device__ void wave_topk(const float* lg, int E, int k, int t, int32_t* __restrict__ ids,
                          float* __restrict__ w) {
  const int lane = lane_id();
  float v[kMaxEPerLane];
  uint32_t taken = 0;
  const int nq = (E + kWave - 1) / kWave;
#pragma unroll
  for (int q = 0; q < kMaxEPerLane; ++q) {
    const int e = lane + q * kWave;
    v[q] = (q < nq && e < E) ? lg[e] : 0.0f;
  }
  float my_v = 0.0f;
  int my_id = 0;
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
    if (lane == j) {
      my_v = bv;
      my_id = bid;
    }
  }
  // w_j = exp(l_j - l_0) / sum_{j'<k} exp(l_j' - l_0), the sum in rank order.
  const float v0 = __shfl(my_v, 0);
  const float ex = (lane < k) ? expf(my_v - v0) : 0.0f;
  float z = 0.0f;
  for (int j = 0; j < k; ++j) z += __shfl(ex, j);
  if (lane < k) {
    ids[(size_t)t * k + lane] = my_id;
    w[(size_t)t * k + lane] = ex / z;
  }
}

// float64 logits of token t for experts e0..e0+7 against a gate matrix
// (global or LDS), written to lg by lane 0 after a butterfly reduction.
template <typename WgPtr>
__device__ __forceinline__ void logits8(const uint4* __restrict__ xr, WgPtr wg, int d, int E,
                                        int e0, float* lg) {
  const int lane = lane_id();
  const int nchunk = d / 8;
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

// Weight mode, one token per wave. STAGED: a block of 16 waves first
// copies the gate matrix to LDS; otherwise 4 waves read it from global
// memory.
template <bool STAGED>
__global__ __launch_bounds__(STAGED ? 64 * kStagedWaves : 64 * kWaves) void gate_weights_topk_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg, int T, int d, int E, int k,
    float* __restrict__ logits_out, int32_t* __restrict__ ids, float* __restrict__ w) {
  constexpr int NW = STAGED ? kStagedWaves : kWaves;
  constexpr int LG = STAGED ? kStagedMaxE : 1024;
  __shared__ __attribute__((aligned(16))) uint16_t wg_s[STAGED ? kStageElems : 8];
  __shared__ float lg_s[NW][LG];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  float* lg = lg_s[wave];
  if (STAGED) {
    const int n16 = E * d / 8;
    for (int i = threadIdx.x; i < n16; i += 64 * NW)
      reinterpret_cast<uint4*>(wg_s)[i] = reinterpret_cast<const uint4*>(wg)[i];
    __syncthreads();
  }
  const int t = blockIdx.x * NW + wave;
  if (t < T) {
    const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)t * d);
    for (int e0 = 0; e0 < E; e0 += 8) {
      if (STAGED)
        logits8(xr, static_cast<const uint16_t*>(wg_s), d, E, e0, lg);
      else
        logits8(xr, wg, d, E, e0, lg);
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    if (logits_out) {
      for (int e = lane; e < E; e += kWave) logits_out[(size_t)t * E + e] = lg[e];
    }
    wave_topk(lg, E, k, t, ids, w);
  }
}

__global__ __launch_bounds__(256) void logits_topk_kernel(const float* __restrict__ logits, int T,
                                                          int E, int k, int32_t* __restrict__ ids,
                                                          float* __restrict__ w) {
  __shared__ float lg_s[kWaves][1024];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int t = blockIdx.x * kWaves + wave;
  float* lg = lg_s[wave];
  if (t >= T) return;
  for (int e = lane; e < E; e += kWave) lg[e] = logits[(size_t)t * E + e];
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  wave_topk(lg, E, k, t, ids, w);
}

}  // namespace

hipError_t launch_gate_topk(const uint16_t* x, const uint16_t* wg, const float* logits_in, int T,
                            int d, int E, int k, float* logits_out, int32_t* ids, float* w,
                            hipStream_t stream) {
  if (T == 0) return hipSuccess;
  if (logits_in) {
    hipLaunchKernelGGL(logits_topk_kernel, dim3((T + kWaves - 1) / kWaves), dim3(256), 0, stream,
                       logits_in, T, E, k, ids, w);
  } else if ((long)E * d <= kStageElems && E <= kStagedMaxE) {
    hipLaunchKernelGGL(gate_weights_topk_kernel<true>, dim3((T + kStagedWaves - 1) / kStagedWaves),
                       dim3(64 * kStagedWaves), 0, stream, x, wg, T, d, E, k, logits_out, ids, w);
  } else {
    hipLaunchKernelGGL(gate_weights_topk_kernel<false>, dim3((T + kWaves - 1) / kWaves), dim3(256),
                       0, stream, x, wg, T, d, E, k, logits_out, ids, w);
  }
  return hipGetLastError();
}

}  // namespace tg
