// Grouped expert GEMMs on MFMA (bf16 operands, float32 accumulation).
//
// The expert FFN (§2.1) of every slot runs in one launch per projection:
//   GEMM1  h = bf16(silu(x W1^T) * (x W3^T))   (gate and up fused, SwiGLU)
//   GEMM2  y = bf16(h W2^T)
// Rows of slot s are rows offsets[s] .. offsets[s+1]-1 of the activation
// matrix. Both operands are K-contiguous ("TN"): activations [rows, K] and
// weights [N, K], so every MFMA fragment is one 16-byte LDS read.
//
// Tiling (gfx950, wave64): a block of 4 waves computes a BM x BNW tile of
// (rows x weight rows) with BK = 64 K-steps; waves form a 2x2 grid and each
// issues v_mfma_f32_32x32x16_bf16 on 32x32 sub-blocks. Tiles are staged
// through LDS with two buffers (the next K-step's global loads are in flight
// while the current one is multiplied) and an XOR swizzle of the 16-byte
// chunks so that fragment reads are bank-conflict free. For GEMM1 the
// weight tile holds BNW/2 gate rows and the matching BNW/2 up rows, so g and
// u of one output element land in the same lane and register and the
// SwiGLU epilogue needs no data exchange. Results are staged through LDS and
// written as 16-byte row segments.
//
// Every output element is one fixed sequence of MFMA accumulations over K
// in increasing order, independent of the row's position, its tile or the
// other rows of its group; a row therefore gives identical bits in any slot
// holding the same weights (shadow failover, §5.3).
#include "tg_device.h"
#include "tg_launch.h"

namespace tg {
namespace {

constexpr int kThreads = 256;
constexpr int kBK = 64;  // K per stage: 8 chunks of 8 bf16 per row

__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Maps the global m-tile index to (slot, first row, valid rows). Wave 0
// scans ceil(count/BM) over the slots 64 at a time.
template <int BM>
__device__ __forceinline__ bool find_tile(const int32_t* __restrict__ offsets, int S, int mt,
                                          int* sh /*LDS: slot,row0,rows*/) {
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    int acc = 0;
    bool found = false;
    for (int base = 0; base < S && !found; base += kWave) {
      const int s = base + lane;
      int cnt = 0, o = 0;
      if (s < S) {
        o = offsets[s];
        cnt = offsets[s + 1] - o;
      }
      const int nt = (cnt + BM - 1) / BM;
      int incl = nt;
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) {
        const int v = __shfl_up(incl, off);
        if (lane >= off) incl += v;
      }
      const int excl = incl - nt;
      const bool mine = (mt >= acc + excl) && (mt < acc + incl);
      const uint64_t b = __ballot(mine);
      if (b) {
        found = true;
        if (mine) {
          const int local = mt - acc - excl;
          sh[0] = s;
          sh[1] = o + local * BM;
          sh[2] = min(BM, cnt - local * BM);
        }
      }
      acc += __shfl(incl, kWave - 1);
    }
    if (lane == 0 && !found) sh[0] = -1;
  }
  __syncthreads();
  return sh[0] >= 0;
}

template <int BM, int BNW, bool SWIGLU>
__global__ __launch_bounds__(kThreads) void grouped_gemm_kernel(
    const uint16_t* __restrict__ A, const int32_t* __restrict__ offsets, int S,
    const uint16_t* __restrict__ B, int K, int NW, int I, uint16_t* __restrict__ C, int ldc) {
  constexpr int MB = BM / 64;    // 32-row MFMA blocks per wave (2 wave rows)
  constexpr int NB = BNW / 64;   // 32-col MFMA blocks per wave (2 wave cols)
  constexpr int A_CH = BM * 8 / kThreads;   // 16-byte chunks per thread per stage
  constexpr int B_CH = BNW * 8 / kThreads;
  constexpr int BN_OUT = SWIGLU ? BNW / 2 : BNW;
  constexpr int CP = BN_OUT + 8;  // padded LDS pitch of the output tile (elements)
  static_assert(BM % 64 == 0 && BNW % 64 == 0, "tile");
  static_assert(!SWIGLU || NB % 2 == 0, "gate/up halves");
  static_assert(BM * CP <= 2 * (BM + BNW) * kBK, "epilogue fits in the stage buffers");

  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (BM + BNW) * kBK];
  __shared__ int tile[4];
  if (!find_tile<BM>(offsets, S, blockIdx.x, tile)) return;
  const int slot = tile[0], row0 = tile[1], rows = tile[2];
  const int nt = blockIdx.y;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Global source rows of this thread's chunks (fixed over K).
  const uint16_t* a_src[A_CH];
  int a_dst[A_CH];
#pragma unroll
  for (int i = 0; i < A_CH; ++i) {
    const int q = tid + kThreads * i;
    const int r = q >> 3, c = q & 7;
    const int gr = row0 + min(r, rows - 1);  // tail rows re-read the last valid row
    a_src[i] = A + (size_t)gr * K + c * 8;
    a_dst[i] = r * kBK + ((c ^ swz(r)) << 3);
  }
  const uint16_t* Bslot = B + (size_t)slot * NW * K;
  const uint16_t* b_src[B_CH];
  int b_dst[B_CH];
#pragma unroll
  for (int i = 0; i < B_CH; ++i) {
    const int q = tid + kThreads * i;
    const int r = q >> 3, c = q & 7;
    int wr;
    if (SWIGLU)
      wr = (r < BNW / 2) ? nt * (BNW / 2) + r : I + nt * (BNW / 2) + (r - BNW / 2);
    else
      wr = nt * BNW + r;
    b_src[i] = Bslot + (size_t)wr * K + c * 8;
    b_dst[i] = r * kBK + ((c ^ swz(r)) << 3);
  }

  // Fragment read offsets (elements) for k16 sub-step 0; sub-step kk adds 2*kk chunks.
  int a_row[MB], b_row[NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) a_row[mb] = wm * (BM / 2) + mb * 32 + (lane & 31);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (SWIGLU)
      b_row[nb] = (nb < NB / 2) ? wn * (BNW / 4) + nb * 32 + (lane & 31)
                                : BNW / 2 + wn * (BNW / 4) + (nb - NB / 2) * 32 + (lane & 31);
    else
      b_row[nb] = wn * (BNW / 2) + nb * 32 + (lane & 31);
  }
  const int khalf = lane >> 5;

  f32x16 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.0f;

  uint4 ra[A_CH], rb[B_CH];
#define TG_GLOAD(k0)                                                                        \
  do {                                                                                      \
    _Pragma("unroll") for (int i = 0; i < A_CH; ++i) ra[i] =                                \
        *reinterpret_cast<const uint4*>(a_src[i] + (k0));                                   \
    _Pragma("unroll") for (int i = 0; i < B_CH; ++i) rb[i] =                                \
        *reinterpret_cast<const uint4*>(b_src[i] + (k0));                                   \
  } while (0)
#define TG_SSTORE(buf)                                                                      \
  do {                                                                                      \
    _Pragma("unroll") for (int i = 0; i < A_CH; ++i)                                        \
        *reinterpret_cast<uint4*>(smem + (buf) * (BM * kBK) + a_dst[i]) = ra[i];            \
    _Pragma("unroll") for (int i = 0; i < B_CH; ++i)                                        \
        *reinterpret_cast<uint4*>(smem + 2 * BM * kBK + (buf) * (BNW * kBK) + b_dst[i]) =   \
            rb[i];                                                                          \
  } while (0)

  const int nk = K / kBK;
  TG_GLOAD(0);
  TG_SSTORE(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) TG_GLOAD((kt + 1) * kBK);
    const uint16_t* as = smem + cur * (BM * kBK);
    const uint16_t* bs = smem + 2 * BM * kBK + cur * (BNW * kBK);
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int ch = 2 * kk + khalf;
      bf16x8 af[MB], bfr[NB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        af[mb] = *reinterpret_cast<const bf16x8*>(as + a_row[mb] * kBK +
                                                  ((ch ^ swz(a_row[mb])) << 3));
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        bfr[nb] = *reinterpret_cast<const bf16x8*>(bs + b_row[nb] * kBK +
                                                   ((ch ^ swz(b_row[nb])) << 3));
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb], bfr[nb], acc[mb][nb], 0, 0, 0);
    }
    if (kt + 1 < nk) TG_SSTORE(cur ^ 1);
    __syncthreads();
  }
#undef TG_GLOAD
#undef TG_SSTORE

  // Epilogue: accumulators -> bf16 tile in LDS -> 16-byte row segments.
  // MFMA 32x32 output: lane l, register r holds row 8*(r/4) + 4*(l/32) + r%4,
  // column l%32 of its block.
  uint16_t* Cs = smem;
  const int mrow = 4 * (lane >> 5);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    if (SWIGLU) {
#pragma unroll
      for (int nb = 0; nb < NB / 2; ++nb) {
        const int col = wn * (BNW / 4) + nb * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float g = acc[mb][nb][r];
          const float u = acc[mb][nb + NB / 2][r];
          const float hv = g / (1.0f + __expf(-g)) * u;
          const int m = wm * (BM / 2) + mb * 32 + 8 * (r >> 2) + mrow + (r & 3);
          Cs[m * CP + col] = f32_to_bf16(hv);
        }
      }
    } else {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int col = wn * (BNW / 2) + nb * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = wm * (BM / 2) + mb * 32 + 8 * (r >> 2) + mrow + (r & 3);
          Cs[m * CP + col] = f32_to_bf16(acc[mb][nb][r]);
        }
      }
    }
  }
  __syncthreads();
  constexpr int CPR = BN_OUT / 8;  // 16-byte chunks per output row
  for (int q = tid; q < BM * CPR; q += kThreads) {
    const int r = q / CPR, c = q - r * CPR;
    if (r < rows) {
      *reinterpret_cast<uint4*>(C + (size_t)(row0 + r) * ldc + nt * BN_OUT + c * 8) =
          *reinterpret_cast<const uint4*>(Cs + r * CP + c * 8);
    }
  }
}

constexpr int kBM = 128;
constexpr int kBNW = 256;

}  // namespace

hipError_t launch_ffn_gateup(const uint16_t* x_perm, const int32_t* offsets, int S, int max_rows,
                             const uint16_t* w13, int d, int I, uint16_t* h, hipStream_t stream) {
  if (max_rows == 0) return hipSuccess;
  const int mtiles = (max_rows + kBM - 1) / kBM + S;  // bound on sum_s ceil(count_s / BM)
  hipLaunchKernelGGL((grouped_gemm_kernel<kBM, kBNW, true>), dim3(mtiles, (2 * I) / kBNW),
                     dim3(kThreads), 0, stream, x_perm, offsets, S, w13, d, 2 * I, I, h, I);
  return hipGetLastError();
}

hipError_t launch_ffn_down(const uint16_t* h, const int32_t* offsets, int S, int max_rows,
                           const uint16_t* w2, int d, int I, uint16_t* y, hipStream_t stream) {
  if (max_rows == 0) return hipSuccess;
  const int mtiles = (max_rows + kBM - 1) / kBM + S;
  hipLaunchKernelGGL((grouped_gemm_kernel<kBM, kBNW, false>), dim3(mtiles, d / kBNW),
                     dim3(kThreads), 0, stream, h, offsets, S, w2, I, d, 0, y, d);
  return hipGetLastError();
}

hipError_t launch_expert_ffn(const uint16_t* x_perm, const int32_t* offsets, int S, int max_rows,
                             const uint16_t* w13, const uint16_t* w2, int d, int I, uint16_t* h,
                             uint16_t* y, hipStream_t stream) {
  hipError_t e = launch_ffn_gateup(x_perm, offsets, S, max_rows, w13, d, I, h, stream);
  if (e != hipSuccess) return e;
  return launch_ffn_down(h, offsets, S, max_rows, w2, d, I, y, stream);
}

}  // namespace tg
