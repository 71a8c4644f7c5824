// Gating (§2.1): gate logits, top-k selection and renormalised gate weights.
//
// One wave per token at a time. In weight mode each lane accumulates its
// stride of the hidden dimension in float64 for 8 experts at a time
// (bf16*bf16 products are exact in float64), a DPP reduction gives every
// lane the full sums, and the float64 sum is rounded once to float32.
// When the gate matrix fits (E*d*2 <= 96 KB) a block of 16 waves (16
// tokens) stages it in LDS once, so the matrix is read from memory once per
// 16 tokens instead of once per token; up to E*d*4 = 128 KB it is staged
// widened to float32, which takes the unpacking out of the dot product (the
// loop is bound by the vector ALU). Top-k runs as k rounds of a wave
// arg-max over the float32 logits (larger first, ties to the lower expert
// id), the cross-lane step in DPP row operations and lane reads; lane j
// keeps the j-th winner, the k exponentials are formed in parallel and
// summed in rank order.
#include "tg_device.h"
#include "tg_launch.h"

namespace tg {
namespace {

constexpr int kWaves = 4;          // waves per block (unstaged kernels)
constexpr int kStagedWaves = 16;   // waves (= tokens) per block when the gate matrix is staged
constexpr int kStageElems = 48 * 1024;  // 96 KB of bf16
constexpr int kStageElemsF32 = 32 * 1024;  // 128 KB of float32
constexpr int kStageBytes = 128 * 1024;
constexpr int kStagedMaxE = kStageElems / 256;  // staged only when E * d fits, d >= 256

__device__ __forceinline__ bool better(float v, int id, float bv, int bid) {
  return v > bv || (v == bv && id < bid);
}

// Arg-max of (v, id) over the 16 lanes of each DPP row: xor 1, xor 2
// (quad permutes), then half-row and row mirrors; afterwards every lane of a
// row holds the row's best.
__device__ __forceinline__ void row_best(float& bv, int& bid) {
#define TG_DPP_STEP(ctrl)                                                                 \
  do {                                                                                    \
    const float ov = __int_as_float(                                                      \
        __builtin_amdgcn_update_dpp(0, __float_as_int(bv), ctrl, 0xF, 0xF, false));       \
    const int oid = __builtin_amdgcn_update_dpp(0, bid, ctrl, 0xF, 0xF, false);           \
    if (better(ov, oid, bv, bid)) {                                                       \
      bv = ov;                                                                            \
      bid = oid;                                                                          \
    }                                                                                     \
  } while (0)
  TG_DPP_STEP(0xB1);   // quad_perm [1,0,3,2]
  TG_DPP_STEP(0x4E);   // quad_perm [2,3,0,1]
  TG_DPP_STEP(0x141);  // row_half_mirror
  TG_DPP_STEP(0x140);  // row_mirror
#undef TG_DPP_STEP
}

// Top-k over the logits held in `lg` (LDS, E <= 64 * NQ floats) by one
// wave; writes ids and weights of token t. Each round takes the best
// remaining candidate of every lane, reduces the rows with DPP and the four
// rows with lane reads, so no round goes through LDS.
template <int NQ>
__device__ void wave_topk(const float* lg, int E, int k, int t, int32_t* __restrict__ ids,
                          float* __restrict__ w) {
  const int lane = lane_id();
  float v[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int e = lane + q * kWave;
    v[q] = (e < E) ? lg[e] : 0.0f;
  }
  uint32_t taken = 0;
  float my_v = 0.0f;
  int my_id = 0;
  for (int j = 0; j < k; ++j) {
    float bv = -__builtin_inff();
    int bid = 0x7fffffff;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int e = lane + q * kWave;
      if (e < E && !(taken & (1u << q)) && better(v[q], e, bv, bid)) {
        bv = v[q];
        bid = e;
      }
    }
    row_best(bv, bid);
    float gv = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bv), 0));
    int gid = __builtin_amdgcn_readlane(bid, 0);
#pragma unroll
    for (int r = 1; r < 4; ++r) {
      const float rv = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bv), 16 * r));
      const int rid = __builtin_amdgcn_readlane(bid, 16 * r);
      if (better(rv, rid, gv, gid)) {
        gv = rv;
        gid = rid;
      }
    }
    if ((gid & (kWave - 1)) == lane) taken |= 1u << (gid / kWave);
    if (lane == j) {
      my_v = gv;
      my_id = gid;
    }
  }
  // w_j = exp(l_j - l_0) / sum_{j'<k} exp(l_j' - l_0), the sum in rank order.
  const float v0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_v), 0));
  const float ex = (lane < k) ? expf(my_v - v0) : 0.0f;
  float z = 0.0f;
  for (int j = 0; j < k; ++j) z += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ex), j));
  if (lane < k) {
    ids[(size_t)t * k + lane] = my_id;
    w[(size_t)t * k + lane] = ex / z;
  }
}

// wave_topk for the smallest NQ that covers E.
__device__ __forceinline__ void wave_topk_any(const float* lg, int E, int k, int t,
                                              int32_t* __restrict__ ids, float* __restrict__ w) {
  if (E <= 64) wave_topk<1>(lg, E, k, t, ids, w);
  else if (E <= 128) wave_topk<2>(lg, E, k, t, ids, w);
  else if (E <= 256) wave_topk<4>(lg, E, k, t, ids, w);
  else if (E <= 512) wave_topk<8>(lg, E, k, t, ids, w);
  else wave_topk<16>(lg, E, k, t, ids, w);
}

// Sum over the wave of a float64 held per lane, the same on every lane, in
// a fixed order: DPP row steps (xor 1, xor 2, half-row mirror, row mirror)
// give each 16-lane row its sum, then the four row sums are added.
__device__ __forceinline__ double wave_sum_f64(double v) {
#define TG_DPP_ADD(ctrl)                                                                     \
  do {                                                                                       \
    const int lo = __builtin_amdgcn_update_dpp(0, (int)__double2loint(v), ctrl, 0xF, 0xF,     \
                                               false);                                       \
    const int hi = __builtin_amdgcn_update_dpp(0, (int)__double2hiint(v), ctrl, 0xF, 0xF,     \
                                               false);                                       \
    v += __hiloint2double(hi, lo);                                                           \
  } while (0)
  TG_DPP_ADD(0xB1);
  TG_DPP_ADD(0x4E);
  TG_DPP_ADD(0x141);
  TG_DPP_ADD(0x140);
#undef TG_DPP_ADD
  double total = 0.0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int lo = __builtin_amdgcn_readlane((int)__double2loint(v), 16 * r);
    const int hi = __builtin_amdgcn_readlane((int)__double2hiint(v), 16 * r);
    total += __hiloint2double(hi, lo);
  }
  return total;
}

// float64 logits of token t for experts e0..e0+7 against a gate matrix
// (global or LDS), written to lg by lane 0 after a wave reduction.
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
    const double sum = wave_sum_f64(acc[q]);
    if (lane == 0 && e0 + q < E) lg[e0 + q] = (float)sum;
  }
}

// The same against a gate matrix staged in LDS as float32 (two float4 per
// chunk of 8), which saves the unpacking of every weight; the products and
// their order are those of logits8.
__device__ __forceinline__ void logits8_f32(const uint4* __restrict__ xr, const float* wg, int d,
                                            int E, int e0, float* lg) {
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
        const float4* wr = reinterpret_cast<const float4*>(wg + (size_t)e * d) + 2 * c;
        const float4 w0 = wr[0], w1 = wr[1];
        const float wf[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[q] = fma(xd[i], (double)wf[i], acc[q]);
      }
    }
  }
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const double sum = wave_sum_f64(acc[q]);
    if (lane == 0 && e0 + q < E) lg[e0 + q] = (float)sum;
  }
}

// Weight mode, one token per wave. STAGE 0: 4 waves read the gate matrix
// from global memory; otherwise a block of 16 waves first copies it to LDS,
// as bf16 (STAGE 1) or, when it fits in 128 KB that way, widened to float32
// (STAGE 2).
template <int STAGE>
__global__ __launch_bounds__(STAGE ? 64 * kStagedWaves : 64 * kWaves) void gate_weights_topk_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg, int T, int d, int E, int k,
    float* __restrict__ logits_out, int32_t* __restrict__ ids, float* __restrict__ w) {
  constexpr int NW = STAGE ? kStagedWaves : kWaves;
  constexpr int LG = STAGE ? kStagedMaxE : 1024;
  __shared__ __attribute__((aligned(16))) uint32_t wg_s[STAGE ? kStageBytes / 4 : 4];
  __shared__ float lg_s[NW][LG];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  float* lg = lg_s[wave];
  if (STAGE) {
    const int n16 = E * d / 8;
    for (int i = threadIdx.x; i < n16; i += 64 * NW) {
      const uint4 v = reinterpret_cast<const uint4*>(wg)[i];
      if (STAGE == 1) {
        reinterpret_cast<uint4*>(wg_s)[i] = v;
      } else {
        const uint32_t m = 0xffff0000u;
        reinterpret_cast<uint4*>(wg_s)[2 * i] = make_uint4(v.x << 16, v.x & m, v.y << 16, v.y & m);
        reinterpret_cast<uint4*>(wg_s)[2 * i + 1] =
            make_uint4(v.z << 16, v.z & m, v.w << 16, v.w & m);
      }
    }
    __syncthreads();
  }
  const int t = blockIdx.x * NW + wave;
  if (t < T) {
    const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)t * d);
    for (int e0 = 0; e0 < E; e0 += 8) {
      if (STAGE == 2)
        logits8_f32(xr, reinterpret_cast<const float*>(wg_s), d, E, e0, lg);
      else if (STAGE == 1)
        logits8(xr, reinterpret_cast<const uint16_t*>(wg_s), d, E, e0, lg);
      else
        logits8(xr, wg, d, E, e0, lg);
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    if (logits_out) {
      for (int e = lane; e < E; e += kWave) logits_out[(size_t)t * E + e] = lg[e];
    }
    wave_topk_any(lg, E, k, t, ids, w);
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
  wave_topk_any(lg, E, k, t, ids, w);
}

// Logits mode for E <= 256 and k <= 16: four tokens per wave, one 16-lane
// DPP row per token. Lane l of a row holds the candidates l, l + 16, ... of
// its token in registers as 64-bit keys: the float32 logit in an order-
// preserving encoding (-0 taken as +0) above the complement of the expert
// id, so a larger key is a larger logit or, on equal logits, a lower id, and
// no two keys are equal. Round j takes every lane's largest key below the
// previous winner's and reduces the row with the four DPP row steps, so
// every lane of the row knows each round's winner (no lane reads, no LDS).
// Lane j keeps the j-th winner; every lane sums the k exponentials in rank
// order, the same sum as the one-token-per-wave kernel.
constexpr int kRowTokens = 4;  // tokens per wave

__device__ __forceinline__ uint64_t topk_key(float v, int e) {
  uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (0xffffffffu - (uint32_t)e);
}

__device__ __forceinline__ float key_value(uint64_t key) {
  const uint32_t u = (uint32_t)(key >> 32);
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7fffffffu) : ~u);
}

__device__ __forceinline__ uint64_t row_max_key(uint64_t k) {
#define TG_DPP_MAX(ctrl)                                                                  \
  do {                                                                                    \
    const uint32_t lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)k, ctrl, 0xF, 0xF,   \
                                                    false);                               \
    const uint32_t hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(k >> 32), ctrl,     \
                                                    0xF, 0xF, false);                     \
    const uint64_t o = ((uint64_t)hi << 32) | lo;                                         \
    k = o > k ? o : k;                                                                    \
  } while (0)
  TG_DPP_MAX(0xB1);   // quad_perm [1,0,3,2]
  TG_DPP_MAX(0x4E);   // quad_perm [2,3,0,1]
  TG_DPP_MAX(0x141);  // row_half_mirror
  TG_DPP_MAX(0x140);  // row_mirror
#undef TG_DPP_MAX
  return k;
}

template <int NQ>
__global__ __launch_bounds__(256) void logits_topk_rows_kernel(const float* __restrict__ logits,
                                                               int T, int E, int k,
                                                               int32_t* __restrict__ ids,
                                                               float* __restrict__ w) {
  const int lane = lane_id();
  const int l16 = lane & 15;
  const int t = (blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave) * kRowTokens + (lane >> 4);
  const bool on = t < T;
  uint64_t key[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int e = l16 + 16 * q;
    key[q] = (on && e < E) ? topk_key(logits[(size_t)t * E + e], e) : 0;  // 0: no candidate
  }
  uint64_t thr = ~0ull;
  float my_v = 0.0f, v0 = 0.0f, z = 0.0f;
  int my_id = 0;
  for (int j = 0; j < k; ++j) {
    uint64_t best = 0;
#pragma unroll
    for (int q = 0; q < NQ; ++q) best = (key[q] < thr && key[q] > best) ? key[q] : best;
    best = row_max_key(best);  // every lane of the row: this round's winner
    thr = best;
    const float bv = key_value(best);
    if (j == 0) v0 = bv;
    const float ex = expf(bv - v0);
    z += ex;
    if (l16 == j) {
      my_v = ex;
      my_id = (int)(0xffffffffu - (uint32_t)best);
    }
  }
  if (on && l16 < k) {
    ids[(size_t)t * k + l16] = my_id;
    w[(size_t)t * k + l16] = my_v / z;
  }
}

}  // namespace

hipError_t launch_gate_topk(const uint16_t* x, const uint16_t* wg, const float* logits_in, int T,
                            int d, int E, int k, float* logits_out, int32_t* ids, float* w,
                            hipStream_t stream) {
  if (T == 0) return hipSuccess;
  if (logits_in && E <= 256 && k <= 16 && T >= 4096) {
    const int per_block = 4 * kRowTokens;  // 4 waves of 4 tokens
    const dim3 grid((T + per_block - 1) / per_block);
    if (E <= 64)
      hipLaunchKernelGGL(logits_topk_rows_kernel<4>, grid, dim3(256), 0, stream, logits_in, T, E, k,
                         ids, w);
    else if (E <= 128)
      hipLaunchKernelGGL(logits_topk_rows_kernel<8>, grid, dim3(256), 0, stream, logits_in, T, E, k,
                         ids, w);
    else
      hipLaunchKernelGGL(logits_topk_rows_kernel<16>, grid, dim3(256), 0, stream, logits_in, T, E,
                         k, ids, w);
  } else if (logits_in) {
    hipLaunchKernelGGL(logits_topk_kernel, dim3((T + kWaves - 1) / kWaves), dim3(256), 0, stream,
                       logits_in, T, E, k, ids, w);
  } else if ((long)E * d <= kStageElemsF32 && E <= kStagedMaxE) {
    hipLaunchKernelGGL(gate_weights_topk_kernel<2>, dim3((T + kStagedWaves - 1) / kStagedWaves),
                       dim3(64 * kStagedWaves), 0, stream, x, wg, T, d, E, k, logits_out, ids, w);
  } else if ((long)E * d <= kStageElems && E <= kStagedMaxE) {
    hipLaunchKernelGGL(gate_weights_topk_kernel<1>, dim3((T + kStagedWaves - 1) / kStagedWaves),
                       dim3(64 * kStagedWaves), 0, stream, x, wg, T, d, E, k, logits_out, ids, w);
  } else {
    hipLaunchKernelGGL(gate_weights_topk_kernel<0>, dim3((T + kWaves - 1) / kWaves), dim3(256),
                       0, stream, x, wg, T, d, E, k, logits_out, ids, w);
  }
  return hipGetLastError();
}

}  // namespace tg
