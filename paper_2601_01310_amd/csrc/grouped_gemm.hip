// Grouped expert GEMMs on MFMA (bf16 operands, float32 accumulation).
//
// The expert FFN (§2.1) of every slot runs in one launch per projection:
//   GEMM1  h = bf16(silu(x W1^T) * (x W3^T))   (gate and up fused, SwiGLU)
//   GEMM2  y = bf16(h W2^T)
// Rows of slot s are rows offsets[s] .. offsets[s+1]-1 of the activation
// matrix. Both operands are K-contiguous: activations [rows, K] and weights
// [N, K], so every MFMA fragment is one 16-byte LDS read.
//
// Tiling (gfx950, wave64): a block computes a BM x BN tile of (activation
// rows x weight rows) in BK-deep K stages with WM x WN waves; each wave
// issues v_mfma_f32_32x32x16_bf16 on 32x32 sub-blocks with the weight
// fragment as the first operand, so a lane's accumulators hold four
// consecutive output columns of one row (packed 8-byte epilogue writes).
//
// Staging: both tiles go global -> LDS with buffer loads that write LDS
// directly (no register staging), in a ring of stage buffers refilled as
// each stage's closing barrier releases one (weights are first touched in
// HBM, so they are requested several stages ahead); at 256 x 256 x 64 the
// stage buffers fill the 160 KB of LDS. Each 16-byte chunk sits at an
// XOR-swizzled position within its row so that fragment reads of
// consecutive rows hit distinct banks; a lane fetches whichever global chunk
// the swizzle assigns to its LDS position. The K loop has no branches: each
// stage ends with one block barrier after which the freed buffers are
// refilled, and the next stage's first fragments are read while the stage's
// last MFMAs run. Rows past the end of a group read as zeros through the
// buffer range check and are never stored; waves whose rows all lie past the
// end skip their MFMAs. Likewise a slot's last weight panel may be partial
// (I or d not a multiple of the panel width): its rows past the slot's
// weights read as zeros and its columns past the output width are never
// stored.
//
// For GEMM1 the weight tile holds BN/2 gate rows and the matching BN/2 up
// rows and every wave owns equal numbers of both, so g and u of one output
// element land in the same lane and register and the SwiGLU epilogue needs
// no data exchange.
//
// Tile shapes: one persistent kernel (one block per CU) runs every launch
// in one of two shapes, chosen on the device from the slot counts, so that
// the host never reads them: 256 x 256 tiles with 4 waves (one per SIMD,
// 128 x 128 each) for batches that fill the MFMA units, walked with the DMA
// pipeline running on across tiles (the gate/up results written straight
// from the accumulators, the down projection's staged in LDS and written as
// whole 128-byte lines); or 32-row tiles with 4 waves (32 x 256 in the gate/up
// projection, 32 x 128 in the down projection), where a launch mostly
// streams weights (decode steps, a single small expert batch) and a 256-row
// tile would stage and multiply mostly zero rows (results staged through
// each wave's own LDS region and written as 16-byte row segments). The
// 32-row shape runs when its rounds of tiles over the grid cost less, at
// about two thirds of a 256-row round each; in the down projection, whose
// partial last round of 256 x 256 tiles runs as 128 x 128 quarter tiles
// (keeping the CUs busy with few tiles), when no slot holds more than 32
// rows or the 32-row tiles fit in one round. All shapes give identical
// bits, so the choice never changes a result.
//
// Tile order: the tiles of one launch are enumerated slot by slot, then by
// weight panel (n), then by row block (m), so consecutive tiles share a
// weight panel; each of the 8 XCDs (blocks are dealt to XCDs round robin)
// takes one contiguous range of that order, keeping a panel in one L2. With
// a schedule area (the fused forward and the replay have one), all but the
// last three rounds of each range (at least two) are dealt statically and
// the rest are claimed from a per-XCD counter, blocks of an XCD that has run out taking tiles
// from the other XCDs' counters, and the pieces of a spilled last round are
// claimed from one more counter; the standalone FFN entry point, and 32-row
// tiles everywhere, deal every tile statically. Which block runs a tile
// never changes its bits.
//
// Every output element is one fixed sequence of MFMA accumulations over K
// in increasing order, independent of the row's position, its tile or the
// other rows of its group; a row therefore gives identical bits in any slot
// holding the same weights (shadow failover, §5.3).
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "tg_device.h"
#include "tg_launch.h"

namespace tg {
namespace {

constexpr int kXcds = 8;
constexpr int kDynRounds = 3;  // last rounds of each XCD's range that are claimed, not dealt

// XOR swizzle of the 16-byte chunks of a staged row (CH chunks per row);
// fragment reads of 8 or 16 consecutive rows hit distinct banks.
template <int CH>
__device__ __forceinline__ int swz(int r) {
  if (CH == 8) return (r & 7) ^ ((r >> 3) & 1);
  return ((r >> 1) ^ (r >> 3)) & 3;
}

#define TG_WAIT_VM(n) \
  __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (((n) >> 4) << 14) | (0x7 << 4) | (0xF << 8))

__device__ __forceinline__ void block_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

typedef __attribute__((address_space(3))) uint16_t lds_u16;
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// SwiGLU of one output element: silu(g) * u = g / (1 + e^-g) * u, with the
// reciprocal from the hardware approximation (about 1 ulp in float32, far
// below the bf16 rounding of h). Every kernel's epilogue uses this one
// expression, so all tile shapes give the same bits.
__device__ __forceinline__ float swiglu(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}

// One 16-byte global -> LDS transfer per lane; the wave's 64 chunks land at
// consecutive 16-byte positions starting at the (wave-uniform) `lds` row.
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t rsrc, lds_u16* lds, int voffset,
                                           int soffset) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)lds, 16,
                                           voffset, soffset, 0, 0);
#endif
}

// Raw buffer resource over [base, base + bytes); loads beyond it return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Resource over the weight rows b_row0 .. end of slot `slot` (NW rows of K
// elements per slot); empty when b_row0 lies past the slot's last row.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t weight_rsrc(const uint16_t* B, int slot, int NW,
                                                              size_t b_row0, int K) {
  const size_t end = (size_t)(slot + 1) * NW;
  const size_t bytes = b_row0 < end ? (end - b_row0) * K * 2 : 0;
  return make_rsrc(B + b_row0 * K, (uint32_t)min((size_t)0x7fffffff, bytes));
}

struct TileInfo {
  int slot, row0, rows, nt;
};

// Row-block counts of one launch at both tile heights, and its largest slot
// (every lane gets the results).
struct Census {
  int full, small, max_rows;  // 256-row tiles, 32-row tiles (times NTx), largest count
};
__device__ __forceinline__ Census census(const int32_t* __restrict__ offsets, int S, int NTx) {
  const int lane = lane_id();
  int full = 0, small = 0, mx = 0;
  for (int base = 0; base < S; base += kWave) {
    const int s = base + lane;
    const int cnt = (s < S) ? offsets[s + 1] - offsets[s] : 0;
    int f = (cnt + 255) / 256, q = (cnt + 31) / 32, m = cnt;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      f += __shfl_xor(f, off);
      q += __shfl_xor(q, off);
      m = max(m, __shfl_xor(m, off));
    }
    full += f;
    small += q;
    mx = max(mx, m);
  }
  return {__builtin_amdgcn_readfirstlane(full) * NTx,
          __builtin_amdgcn_readfirstlane(small) * NTx, __builtin_amdgcn_readfirstlane(mx)};
}

// Tile L of BMx-row tiles in the order slot, panel, row block:
// its slot, first row, row count, panel and row-block index.
__device__ __forceinline__ bool find_tile(const int32_t* __restrict__ offsets, int S, int BMx,
                                          int NTx, int L, TileInfo* t, int* m_out) {
  const int lane = lane_id();
  int acc = 0;  // tiles before this group of slots
  for (int base = 0; base < S; base += kWave) {
    const int s = base + lane;
    int o = 0, cnt = 0;
    if (s < S) {
      o = offsets[s];
      cnt = offsets[s + 1] - o;
    }
    const int mt = (cnt + BMx - 1) / BMx;
    const int tiles = mt * NTx;
    int incl = tiles;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int v = __shfl_up(incl, off);
      if (lane >= off) incl += v;
    }
    const int excl = incl - tiles;
    const uint64_t owner = __ballot(L >= acc + excl && L < acc + incl);
    if (owner) {
      const int src = __builtin_ctzll(owner);
      const int local = L - acc - __shfl(excl, src);
      const int m_t = __shfl(mt, src);
      const int n = local / m_t, m = local - n * m_t;
      t->slot = __builtin_amdgcn_readfirstlane(base + src);
      t->row0 = __builtin_amdgcn_readfirstlane(__shfl(o, src));  // slot's first row
      t->rows = __builtin_amdgcn_readfirstlane(__shfl(cnt, src));  // slot's row count
      t->nt = __builtin_amdgcn_readfirstlane(n);
      *m_out = __builtin_amdgcn_readfirstlane(m);
      return true;
    }
    acc += __shfl(incl, kWave - 1);
  }
  return false;
}

// Both operands stream through one ring of NBUF stage buffers: stage j
// sits in buffer j % NBUF, and the buffer that stage kt releases at its
// closing barrier takes stage kt + NBUF, so NBUF - 1 stages are in flight
// while one is multiplied. A and B of a stage are issued together: the wait
// for stage kt + 1 (vector loads complete in issue order) then leaves the
// NBUF - 2 younger stages in flight instead of draining them.
//
// GATHER: the activation rows are not pre-permuted; row r of the grouped
// matrix is row perm[r] / kq of A (the token of routed pair perm[r]), read
// in place through a buffer resource over all A_rows rows of A.
template <int BM, int BN, int BK, int WM, int WN, bool SWIGLU, bool GATHER, int NBUF>
__device__ __forceinline__ void gemm_tile(uint16_t* smem, const TileInfo& tile,
                                          const uint16_t* __restrict__ A,
                                          const uint16_t* __restrict__ B, int K, int NW, int I,
                                          uint16_t* __restrict__ C, int ldc,
                                          const int32_t* __restrict__ perm, int kq, int A_rows) {
  constexpr int NWAVE = WM * WN;
  constexpr int MB = BM / WM / 32;          // 32-row blocks per wave
  constexpr int NB = BN / WN / 32;          // 32-col blocks per wave
  constexpr int CH = BK / 8;                // 16-byte chunks per staged row
  constexpr int RPI = 64 / CH;              // rows per load instruction (64 lanes x 16 B)
  constexpr int AI = BM / NWAVE / RPI;      // A load instructions per wave per stage
  constexpr int BI = BN / NWAVE / RPI;      // B load instructions per wave per stage
  constexpr int A_ST = BM * BK, B_ST = BN * BK;  // elements per stage buffer
  constexpr int WOUT = SWIGLU ? BN / 2 / WN : BN / WN;  // output columns per wave
  constexpr int WP = WOUT + 8;
  static_assert(MB >= 1 && NB >= 1 && AI >= 1 && BI >= 1 && (BK == 32 || BK == 64), "tile");
  static_assert(!SWIGLU || NB % 2 == 0, "gate/up halves");
  static_assert(NBUF >= 2 && (NBUF - 2) * (AI + BI) <= 63, "ring depth within the wait count");
  static_assert(NWAVE * 32 * WP <= NBUF * (A_ST + B_ST), "epilogue fits in the stage buffers");

  const int slot = tile.slot, row0 = tile.row0, rows = tile.rows, nt = tile.nt;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;

  // Direct-to-LDS staging: load instruction i of this wave fills RPI
  // consecutive staged rows (1 KB); lane l writes chunk position l % CH of
  // row l / CH, so it fetches the global chunk that the swizzle puts there.
  const size_t b_row0 = (size_t)slot * NW + (SWIGLU ? nt * (BN / 2) : nt * BN);
  // Rows past the group's end read as zeros (their results are never stored).
  const __amdgpu_buffer_rsrc_t a_rsrc =
      GATHER ? make_rsrc(A, (uint32_t)A_rows * K * 2)
             : make_rsrc(A + (size_t)row0 * K, (uint32_t)rows * K * 2);
  const __amdgpu_buffer_rsrc_t b_rsrc = weight_rsrc(B, slot, NW, b_row0, K);
  int a_off[AI], b_off[BI];  // byte offsets
#pragma unroll
  for (int i = 0; i < AI; ++i) {
    const int r = wave * (BM / NWAVE) + i * RPI + lane / CH;
    const int c = (lane % CH) ^ swz<CH>(r);
    if (GATHER) {
      // rows past the group's end get an offset beyond the resource: zeros
      a_off[i] = (r < rows) ? ((perm[row0 + r] / kq) * K + c * 8) * 2 : (int)0x80000000u;
    } else {
      a_off[i] = (r * K + c * 8) * 2;
    }
  }
#pragma unroll
  for (int i = 0; i < BI; ++i) {
    const int r = wave * (BN / NWAVE) + i * RPI + lane / CH;
    const int c = (lane % CH) ^ swz<CH>(r);
    const int wr = (SWIGLU && r >= BN / 2) ? I - BN / 2 + r : r;  // up rows follow gate rows
    b_off[i] = (wr * K + c * 8) * 2;
  }
  lds_u16* const smem3 = (lds_u16*)smem;
  const int a_lds = wave * (BM / NWAVE) * BK;
  const int b_lds = NBUF * A_ST + wave * (BN / NWAVE) * BK;
#define TG_ISSUE_A(k0, buf)                                                        \
  do {                                                                             \
    _Pragma("unroll") for (int i = 0; i < AI; ++i)                                 \
        load_lds16(a_rsrc, smem3 + (buf) * A_ST + a_lds + i * RPI * BK, a_off[i],   \
                   (k0) * 2);                                                      \
  } while (0)
#define TG_ISSUE_B(k0, buf)                                                        \
  do {                                                                             \
    _Pragma("unroll") for (int i = 0; i < BI; ++i)                                 \
        load_lds16(b_rsrc, smem3 + (buf) * B_ST + b_lds + i * RPI * BK, b_off[i],   \
                   (k0) * 2);                                                      \
  } while (0)

  // LDS element offsets of this lane's fragments for k16 sub-step kk.
  const int khalf = lane >> 5;
  const int xrow = wm * (BM / WM) + (lane & 31);
  const int wrow = (SWIGLU ? wn * (BN / 2 / WN) : wn * (BN / WN)) + (lane & 31);
  int xoff[BK / 16], woff[BK / 16];
#pragma unroll
  for (int kk = 0; kk < BK / 16; ++kk) {
    xoff[kk] = xrow * BK + (((2 * kk + khalf) ^ swz<CH>(xrow)) << 3);
    woff[kk] = NBUF * A_ST + wrow * BK + (((2 * kk + khalf) ^ swz<CH>(wrow)) << 3);
  }
  // Weight rows of block nb relative to wrow (gate blocks, then up blocks).
  auto wblk = [](int nb) constexpr {
    return SWIGLU ? ((nb < NB / 2) ? nb * 32 : BN / 2 + (nb - NB / 2) * 32) : nb * 32;
  };

  f32x16 acc[NB][MB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[nb][mb][r] = 0.0f;

  const int nk = K / BK;
  constexpr int KK = BK / 16;          // k16 sub-steps per stage
  static_assert(KK % 2 == 0, "fragment double buffering alternates within a stage");
  bf16x8 xf[2][MB], wf[2][NB];
#define TG_FRAGS(abuf, bbuf, kk, dst)                                                  \
  do {                                                                                 \
    _Pragma("unroll") for (int mb = 0; mb < MB; ++mb) xf[dst][mb] =                    \
        *reinterpret_cast<const bf16x8*>(smem + (abuf) * A_ST + xoff[kk] +             \
                                         mb * 32 * BK);                                \
    _Pragma("unroll") for (int nb = 0; nb < NB; ++nb) wf[dst][nb] =                    \
        *reinterpret_cast<const bf16x8*>(smem + (bbuf) * B_ST + woff[kk] +             \
                                         wblk(nb) * BK);                               \
  } while (0)
#define TG_MFMAS(src)                                                                  \
  do {                                                                                 \
    _Pragma("unroll") for (int nb = 0; nb < NB; ++nb)                                  \
        _Pragma("unroll") for (int mb = 0; mb < MB; ++mb) acc[nb][mb] =                \
            __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[src][nb], xf[src][mb],          \
                                                    acc[nb][mb], 0, 0, 0);             \
  } while (0)

  // Prologue: stages 0 .. NBUF-1 in flight (indices past the end re-load the
  // last stage, so every wait counts the same loads); stage 0 visible; its
  // first fragments loaded.
#pragma unroll
  for (int j = 0; j < NBUF; ++j) {
    const int k0 = min(j, nk - 1) * BK;
    TG_ISSUE_A(k0, j);
    TG_ISSUE_B(k0, j);
  }
  TG_WAIT_VM((NBUF - 1) * (AI + BI));
  block_barrier();
  TG_FRAGS(0, 0, 0, 0);

  // Branch-free K loop: every iteration waits, synchronises and refills one
  // stage buffer, so each sub-step is one straight-line region. A wave whose
  // rows all lie past the group's end (in the tail tile of a slot) skips the
  // fragment reads and MFMAs but keeps its loads and barriers.
  if (wm * (BM / WM) < rows) {
    for (int kt = 0; kt < nk; ++kt) {
      const int cb = kt % NBUF;
#pragma unroll
      for (int kk = 0; kk < KK - 1; ++kk) {
        TG_FRAGS(cb, cb, kk + 1, (kk + 1) & 1);
        TG_MFMAS(kk & 1);
      }
      // Last sub-step: once every wave holds its fragments of stage kt and
      // stage kt+1 has landed, stage kt's buffer takes stage kt + NBUF, and
      // the next stage's first fragments are read while the last MFMAs run.
      TG_WAIT_VM((NBUF - 2) * (AI + BI));
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
      block_barrier();
      const int k0 = min(kt + NBUF, nk - 1) * BK;
      TG_ISSUE_A(k0, cb);
      TG_ISSUE_B(k0, cb);
      TG_FRAGS((kt + 1) % NBUF, (kt + 1) % NBUF, 0, 0);
      TG_MFMAS((KK - 1) & 1);
    }
  } else {
    for (int kt = 0; kt < nk; ++kt) {
      TG_WAIT_VM((NBUF - 2) * (AI + BI));
      block_barrier();
      const int k0 = min(kt + NBUF, nk - 1) * BK;
      TG_ISSUE_A(k0, kt % NBUF);
      TG_ISSUE_B(k0, kt % NBUF);
    }
  }
  TG_WAIT_VM(0);
#undef TG_FRAGS
#undef TG_MFMAS
#undef TG_ISSUE_A
#undef TG_ISSUE_B
  __syncthreads();

  // Epilogue. acc[nb][mb] register r of lane l holds row mb*32 + l%32 and
  // column nb*32 + 8*(r/4) + 4*(l/32) + r%4 of the wave's sub-tile. Each wave
  // stages one 32-row block at a time in its own LDS region (8-byte writes)
  // and stores it as 16-byte row segments.
  uint16_t* region = smem + wave * (32 * WP);
  const int colbase = SWIGLU ? nt * (BN / 2) + wn * WOUT : nt * BN + wn * WOUT;
  constexpr int CPR = WOUT / 8;  // 16-byte chunks per wave row
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int mm = lane & 31;
#pragma unroll
    for (int nb = 0; nb < (SWIGLU ? NB / 2 : NB); ++nb) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * q + e;
          if (SWIGLU) {
            const float g = acc[nb][mb][r];
            const float u = acc[nb + NB / 2][mb][r];
            v[e] = swiglu(g, u);
          } else {
            v[e] = acc[nb][mb][r];
          }
        }
        const int col = nb * 32 + 8 * q + 4 * (lane >> 5);
        uint2 pk;
        pk.x = pack_bf16x2(v[0], v[1]);
        pk.y = pack_bf16x2(v[2], v[3]);
        *reinterpret_cast<uint2*>(region + mm * WP + col) = pk;
      }
    }
    // The region is this wave's own: LDS completes a wave's accesses in
    // order, so only the compiler must keep the reads after the writes.
    __builtin_amdgcn_s_waitcnt(0xc07f);
    asm volatile("" ::: "memory");
    const int mbase = wm * (BM / WM) + mb * 32;
#pragma unroll
    for (int i = 0; i < (32 * CPR + kWave - 1) / kWave; ++i) {
      const int q = lane + kWave * i;
      const int r = q / CPR, c = q - r * CPR;
      if (q < 32 * CPR && mbase + r < rows && colbase + c * 8 < ldc) {
        *reinterpret_cast<uint4*>(C + (size_t)(row0 + mbase + r) * ldc + colbase + c * 8) =
            *reinterpret_cast<const uint4*>(region + r * WP + c * 8);
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    asm volatile("" ::: "memory");
  }
}

// Persistent kernel with one wave per SIMD: 4 waves, 256 x 256 tiles. A
// tile with more than 128 rows runs in full mode: waves (wm, wn) of a 2 x 2
// grid each compute 128 x 128 (4 x 4 blocks of 32 x 32), so each fragment
// read from LDS feeds four MFMAs instead of two; that halves the LDS read
// traffic of a 16-wave shape, and under the power limit the clock stays
// higher. The last row block of a slot is usually partial: with at most 128
// rows the tile runs in half mode (every wave rows 0-127 and a quarter of the
// columns, 4 x 2 blocks), with at most 64 rows in quarter mode (rows 0-63,
// 2 x 2 blocks), so its cost follows its rows instead of a full tile's.
// The 32 x 32 blocks stay aligned in every mode, so each output element gets
// the same MFMA sequence, hence the same bits.
//
// With a single wave per SIMD no other wave covers a gap in the instruction
// stream, so the order within a stage of four k16 sub-steps is fixed
// explicitly:
//   sub-steps 0-2: the MFMAs with the next sub-step's fragment reads and a
//               quarter of the stage's DMA loads among them (A in sub-steps
//               0 and 1, B in sub-step 2);
//   sub-step 3: half of its MFMAs with the last quarter of the loads, then
//               the wait and the block barrier while they run, then the next
//               stage's first fragments interleaved with the other half.
// During stage g (counted on across tiles) A of stage g+1 and B of stage g+2
// are loaded into the buffers that stage g-1 released at the previous
// barrier; at the end of stage g only B of stage g+2 may still be in flight.
// Loads past the last stage of the walk re-load that stage into released
// buffers, so every wait counts the same number of loads.
template <bool SWIGLU, bool GATHER, bool TAIL>
__global__ __launch_bounds__(256) void grouped_gemm_persistent4_kernel(
    const uint16_t* __restrict__ A, const int32_t* __restrict__ offsets, int S,
    const uint16_t* __restrict__ B, int K, int NW, int I, uint16_t* __restrict__ C, int ldc,
    int NT, const int32_t* __restrict__ perm, int kq, uint32_t kq_magic, int kq_shift,
    int A_rows, int32_t* __restrict__ claims,
    int policy) {
  constexpr int BM = 256, BN = 256, BK = 64, NWAVE = 4;
  constexpr int CH = BK / 8;                            // 16-byte chunks per staged row
  constexpr int RPI = 64 / CH;                          // staged rows per load instruction
  constexpr int RW = BM / NWAVE;                        // staged A rows per wave
  constexpr int AI = RW / RPI, BI = BN / NWAVE / RPI;   // load instructions per stage
  constexpr int A_ST = BM * BK, B_ST = BN * BK;
  constexpr int KK = BK / 16;
  static_assert(KK == 4 && AI == 8 && BI == 8, "schedule assumes this shape");
  static_assert(!(TAIL && GATHER), "quarter tiles read pre-permuted rows");
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * A_ST + 3 * B_ST];

  const int per_xcd_blocks = gridDim.x / kXcds;
  const int x = blockIdx.x % kXcds, c = blockIdx.x / kXcds;
  const int G = gridDim.x;
  const Census cs = census(offsets, S, NT);
  bool small_tiles = policy == kTilesSmall;
  if (policy == kTilesAuto) {
    // Gate/up: rounds of tiles over the grid at each height; a 32-row round
    // costs about two thirds of a 256-row round (it streams the same weight
    // panel with an eighth of the MFMA work). Down (TAIL, 32 x 128 tiles, two
    // per 256-column panel): 32-row tiles when no slot exceeds 32 rows, or
    // when they fit in one round; otherwise the 256-row walk, whose partial
    // last round splits into quarters, is faster (measured on single expert
    // batches: a Mixtral expert's down projection of 64 to 256 rows takes
    // 88 us in one round of 32-row tiles against 107-139 us in 256-row
    // tiles, and 170 against 139 us at 512 rows, two rounds).
    const int rs = (cs.small + G - 1) / G, rf = (cs.full + G - 1) / G;
    small_tiles = TAIL ? (cs.max_rows <= 32 || 2 * cs.small <= G) : 2 * rs < 3 * rf;
  }
  if (small_tiles) {
    // 32 x 256 tiles (gate/up) or 32 x 128 tiles (down), each XCD walking
    // one contiguous range of them. These launches stream weights; the down
    // projection's narrower tiles split its panels finely enough to even out
    // the blocks' shares (32 slots of d = 7168: 1792 tiles, 7 per block,
    // instead of 896, 3 or 4 per block), and their smaller stages leave room
    // for a deeper ring.
    constexpr int NS = SWIGLU ? 1 : 2;  // tiles per 256-column panel
    const int n_small = cs.small * NS;
    const int per_s = (n_small + kXcds - 1) / kXcds;
    const int hi_s = min(x * per_s + per_s, n_small);
    for (int q = x * per_s + c; q < hi_s; q += per_xcd_blocks) {
      TileInfo t;
      int m;
      if (!find_tile(offsets, S, 32, NT * NS, q, &t, &m)) break;
      t.row0 += m * 32;
      t.rows = min(32, t.rows - m * 32);
      if constexpr (SWIGLU)
        gemm_tile<32, BN, BK, 1, 4, SWIGLU, GATHER, 4>(smem, t, A, B, K, NW, I, C, ldc, perm, kq,
                                                      A_rows);
      else
        gemm_tile<32, BN / 2, BK, 1, 4, SWIGLU, GATHER, 8>(smem, t, A, B, K, NW, I, C, ldc, perm,
                                                          kq, A_rows);
      __syncthreads();
    }
    return;
  }
  const int total = cs.full;
  const int rem = TAIL ? total % (int)gridDim.x : 0;
  const bool tail = rem > 0 && 2 * rem <= (int)gridDim.x;
  const int n_head = tail ? total - rem : total;
  const int per = (n_head + kXcds - 1) / kXcds;
  const int lo = x * per, hi = min(lo + per, n_head);
  int L = lo + c;
  if (L < hi) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;

    // Dynamic schedule (claims != nullptr; claims[0..8] are zero at
    // launch). The first R rounds of each XCD's range are dealt statically
    // (tile lo + jP + c is the block's tile j), R being all but the last
    // three rounds and at least 2: blocks that start the same round together
    // stream the same weight panels close together in time, so they share
    // them in L2. Every later tile of XCD x's range is claimed from counter
    // claims[x], position v giving tile lo_x + RP + v. A block whose own
    // range is used up claims from the XCD with the most tiles left, so that
    // XCDs that run ahead take work from those behind; every tile still runs
    // exactly once, and its bits do not depend on where it runs. Tile j of a
    // block is claimed by thread 0 when the block starts its tile j - 2 (a
    // static tile needs no claim; a block whose static tiles pass its range's
    // end claims instead); when tile j - 2 ends, wave 0 resolves the claim
    // and hands tile j to the other waves through LDS, at the switch that
    // makes it the next tile. The claim is a plain memory instruction issued
    // by every thread, with an out-of-range offset where it must do nothing
    // (the resource is empty without a schedule), and its result is read
    // only after the tile's last stage, whose wait has covered it: no branch
    // or loop makes the compiler wait for it inside the K loop, so the DMA
    // pipeline never drains for the schedule.
    const bool dyn = claims != nullptr;
    const int P = per_xcd_blocks;
    constexpr int kOut = (int)0x80000000u;  // an offset past any resource: no access
    constexpr int kCoherent = 16;           // sc1: the device-coherent copy
    const __amdgpu_buffer_rsrc_t cl_rsrc = make_rsrc(claims, dyn ? kXcds * 4 : 0);
    auto range_lo = [&](int xx) { return xx * per; };
    auto range_hi = [&](int xx) { return min(xx * per + per, n_head); };
    int cl_x = x, cl_v = 0;        // thread 0: the counter claimed from, its last value
    int cl_last = -1;              // wave 0: the block's latest known tile (-1: none left)
    // Read right after the last stage, whose wait has covered the claim, so
    // that nothing later waits for it: thread 0's claim.
    int cl_got = 0;
    // Tile j + 2's claim, issued when tile j starts (thread 0 only).
    const int R = max(2, (per + P - 1) / P - kDynRounds);  // static rounds
    auto static_tile = [&](int j) { return j < R && lo + j * P + c < hi; };
    auto claim_issue = [&](int j) {
      cl_v = __builtin_amdgcn_raw_ptr_buffer_atomic_add_i32(
          1, cl_rsrc, (tid == 0 && cl_last >= 0 && !static_tile(j + 2)) ? cl_x * 4 : kOut, 0, 0);
    };
    // When tile j ends: tile j + 2, static or from the claim (wave 0).
    auto claim_resolve = [&](int jn) -> int {
      int t = -1;
      if (cl_last >= 0 && static_tile(jn)) {
        t = lo + jn * P + c;
      } else if (cl_last >= 0) {
        t = range_lo(cl_x) + R * P + cl_got;
        if (t >= range_hi(cl_x)) {  // this range is used up: take from the fullest one
          t = -1;
          for (int tries = 0; tries < kXcds; ++tries) {
            const int cv = (int)__builtin_amdgcn_raw_buffer_load_b32(
                cl_rsrc, lane < kXcds ? lane * 4 : kOut, 0, kCoherent);
            int left = lane < kXcds ? range_hi(lane) - (range_lo(lane) + R * P + cv) : 0;
            int bx = lane;
#pragma unroll
            for (int off = 4; off >= 1; off >>= 1) {
              const int ol = __shfl_xor(left, off), ox = __shfl_xor(bx, off);
              if (ol > left || (ol == left && ox < bx)) {
                left = ol;
                bx = ox;
              }
            }
            left = __shfl(left, 0);
            bx = __shfl(bx, 0);
            if (left <= 0) break;
            cl_x = bx;
            const int v = __shfl(__builtin_amdgcn_raw_ptr_buffer_atomic_add_i32(
                                     1, cl_rsrc, lane == 0 ? cl_x * 4 : kOut, 0, 0),
                                 0);
            if (range_lo(cl_x) + R * P + v < range_hi(cl_x)) {
              t = range_lo(cl_x) + R * P + v;
              break;
            }
          }
        }
      }
      cl_last = t;
      return t;
    };

    int s_cur = 0, before = 0, pos = 0, c_nt = 0, c_m = 0;
    int o_cur = offsets[0];
    int cnt_cur = offsets[1] - o_cur;
    int mt_cur = (cnt_cur + BM - 1) / BM;
    auto seek = [&](int Lq, int& slot, int& row0, int& rows, int& nt) {
      if (Lq < pos) {  // a stolen tile before the cursor: walk again from slot 0
        s_cur = 0;
        before = 0;
        pos = 0;
        c_nt = 0;
        c_m = 0;
        o_cur = offsets[0];
        cnt_cur = offsets[1] - o_cur;
        mt_cur = (cnt_cur + BM - 1) / BM;
      }
      while (Lq >= before + mt_cur * NT) {
        before += mt_cur * NT;
        ++s_cur;
        o_cur = offsets[s_cur];
        cnt_cur = offsets[s_cur + 1] - o_cur;
        mt_cur = (cnt_cur + BM - 1) / BM;
        pos = before;
        c_nt = 0;
        c_m = 0;
      }
      for (c_m += Lq - pos; c_m >= mt_cur; c_m -= mt_cur) ++c_nt;
      pos = Lq;
      slot = s_cur;
      nt = c_nt;
      row0 = o_cur + c_m * BM;
      rows = min(BM, cnt_cur - c_m * BM);
    };
    auto b_of = [&](int slot, int nt) {
      const size_t b_row0 = (size_t)slot * NW + (SWIGLU ? nt * (BN / 2) : nt * BN);
      return weight_rsrc(B, slot, NW, b_row0, K);
    };
    auto a_of = [&](int row0, int rows) {
      return GATHER ? make_rsrc(A, (uint32_t)A_rows * K * 2)
                    : make_rsrc(A + (size_t)row0 * K, (uint32_t)rows * K * 2);
    };
    // Byte offsets of this lane's A chunks for a tile. GATHER: the RPI rows of
    // each load instruction come in by scalar loads of perm (clamped to the
    // tile's last row), pair index / kq by multiply-high with the host's
    // magic number, and each lane picks its row; rows past the end read as
    // zeros.
    auto a_offsets = [&](int row0, int rows, int* a_off) {
#pragma unroll
      for (int i = 0; i < AI; ++i) {
        const int r = wave * RW + i * RPI + lane / CH;
        const int cc = ((lane % CH) ^ swz<CH>(r)) * 8;
        if (GATHER) {
          int t = 0;
#pragma unroll
          for (int j = 0; j < RPI; ++j) {
            const uint32_t pj = (uint32_t)perm[row0 + min(wave * RW + i * RPI + j, rows - 1)];
            const int tj = (int)(kq_shift ? __umulhi(pj, kq_magic) >> (kq_shift - 1) : pj);
            t = (lane / CH == j) ? tj : t;
          }
          a_off[i] = (r < rows) ? (t * K + cc) * 2 : (int)0x80000000u;
        } else {
          a_off[i] = (r * K + cc) * 2;
        }
      }
    };

    int b_off[BI];
#pragma unroll
    for (int i = 0; i < BI; ++i) {
      const int r = wave * (BN / NWAVE) + i * RPI + lane / CH;
      const int wr = (SWIGLU && r >= BN / 2) ? I - BN / 2 + r : r;
      b_off[i] = (wr * K + ((lane % CH) ^ swz<CH>(r)) * 8) * 2;
    }
    lds_u16* const smem3 = (lds_u16*)smem;
    const int a_lds = wave * RW * BK;
    const int b_lds = 2 * A_ST + wave * (BN / NWAVE) * BK;
    const int khalf = lane >> 5;
    const int nk = K / BK;  // at least 2 (checked by the launcher)

#define TG_ISSUE_A(rs, offs, k0, buf, i0, i1)                                              \
  do {                                                                                     \
    _Pragma("unroll") for (int i = (i0); i < (i1); ++i)                                    \
        load_lds16(rs, smem3 + (buf) * A_ST + a_lds + i * RPI * BK, offs[i], (k0) * 2);    \
  } while (0)
#define TG_ISSUE_B(rs, k0, buf, i0, i1)                                                    \
  do {                                                                                     \
    _Pragma("unroll") for (int i = (i0); i < (i1); ++i)                                    \
        load_lds16(rs, smem3 + (buf) * B_ST + b_lds + i * RPI * BK, b_off[i], (k0) * 2);   \
  } while (0)
#define TG_FRAGS(abuf, bbuf, kk, dst)                                                      \
  do {                                                                                     \
    _Pragma("unroll") for (int mb = 0; mb < MBm; ++mb) xf[dst][mb] =                       \
        *reinterpret_cast<const bf16x8*>(smem + (abuf) * A_ST + xoff[kk] + mb * 32 * BK);  \
    _Pragma("unroll") for (int nb = 0; nb < NBm; ++nb) wf[dst][nb] =                       \
        *reinterpret_cast<const bf16x8*>(smem + (bbuf) * B_ST + woff[kk] + wblk(nb) * BK); \
  } while (0)
#define TG_MFMAS(src, lo_, hi_)                                                            \
  do {                                                                                     \
    _Pragma("unroll") for (int q = (lo_); q < (hi_); ++q) acc[q / MBm][q % MBm] =          \
        __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[src][q / MBm], xf[src][q % MBm],        \
                                                acc[q / MBm][q % MBm], 0, 0, 0);           \
  } while (0)
#define TG_SG(mask, n) __builtin_amdgcn_sched_group_barrier(mask, n, 0)
#define TG_DM TG_SG(0x100, 1); TG_SG(0x008, 1)
    // Scheduling groups: 0x008 MFMA, 0x010 VMEM, 0x100 DS read. In sub-steps
    // 0-2 the fragment reads of the next sub-step are spread over the first
    // MFMAs and the sub-step's 4 DMA loads over the rest, so that neither the
    // LDS queue nor the load path (about 16 cycles per 1 KB load) backs up
    // far enough to stall the wave's instruction stream. The fragment reads
    // come before the loads: the compiler keeps every LDS read ahead of the
    // DMA writes that follow it in program order (it cannot tell that they
    // touch other buffers).
#define TG_PATTERN_LOADS                                                                   \
  do {                                                                                     \
    if constexpr (M == 0) {                                                                \
      _Pragma("unroll") for (int i = 0; i < 8; ++i) { TG_DM; }                             \
      _Pragma("unroll") for (int i = 0; i < 4; ++i) { TG_SG(0x010, 1); TG_SG(0x008, 2); }  \
    } else if constexpr (M == 1) {                                                         \
      _Pragma("unroll") for (int i = 0; i < 6; ++i) { TG_DM; }                             \
      _Pragma("unroll") for (int i = 0; i < 2; ++i) { TG_SG(0x010, 1); TG_SG(0x008, 1); }  \
      TG_SG(0x010, 2);                                                                     \
    } else {                                                                               \
      _Pragma("unroll") for (int i = 0; i < 4; ++i) { TG_DM; }                             \
      TG_SG(0x010, 4);                                                                     \
    }                                                                                      \
  } while (0)
    // Sub-step 3 before the barrier: half of the MFMAs with the last 4 loads.
#define TG_PATTERN_PRE                                                                     \
  do {                                                                                     \
    if constexpr (M == 0) {                                                                \
      _Pragma("unroll") for (int i = 0; i < 4; ++i) {                                      \
        TG_SG(0x008, 1); TG_SG(0x010, 1); TG_SG(0x008, 1);                                 \
      }                                                                                    \
    } else if constexpr (M == 1) {                                                         \
      _Pragma("unroll") for (int i = 0; i < 4; ++i) { TG_SG(0x008, 1); TG_SG(0x010, 1); }  \
    } else {                                                                               \
      _Pragma("unroll") for (int i = 0; i < 2; ++i) { TG_SG(0x008, 1); TG_SG(0x010, 2); }  \
    }                                                                                      \
  } while (0)
    // After the barrier: the next stage's first fragment reads with the
    // other half of the MFMAs.
#define TG_PATTERN_POST                                                                    \
  do {                                                                                     \
    _Pragma("unroll") for (int i = 0; i < NQ / 2; ++i) { TG_DM; }                          \
    if constexpr (ND > NQ / 2) TG_SG(0x100, ND - NQ / 2);                                  \
  } while (0)

    // A of stage kt+1 and B of stage kt+2 go into the buffers released at
    // the previous barrier: this tile's, else the next tile's, else (no next
    // tile) this tile's last stage again. Without a next tile its operands
    // (a_n, b_n, a_off_n) are the current tile's, so a load past the end of
    // this tile may always take them. A of stage kt+1 lies in this tile in
    // every stage but the last (LAST, known to the compiler).
#define TG_TARGETS(kt, LAST)                                                               \
  const bool cb = (kt) + 2 < nk;                                                           \
  const int ka = !(LAST) ? (kt) + 1 : (has_n ? 0 : nk - 1);                                \
  const int kb = cb ? (kt) + 2 : (has_n ? (kt) + 2 - nk : nk - 1);                         \
  const __amdgpu_buffer_rsrc_t ra = !(LAST) ? a_cur : a_n;                                 \
  const __amdgpu_buffer_rsrc_t rb = cb ? b_cur : b_n;                                      \
  int offa[AI];                                                                            \
  _Pragma("unroll") for (int i = 0; i < AI; ++i) offa[i] = !(LAST) ? a_off[i] : a_off_n[i]; \
  const int abn = ab ^ 1, bbn = (bb == 0) ? 2 : bb - 1

    int slot, row0, rows, nt;
    seek(L, slot, row0, rows, nt);
    __amdgpu_buffer_rsrc_t a_cur = a_of(row0, rows), b_cur = b_of(slot, nt);
    int a_off[AI], a_off_n[AI];
    a_offsets(row0, rows, a_off);
    int Ln = L + per_xcd_blocks;
    bool has_n = Ln < hi;
    if (dyn) cl_last = has_n ? Ln : -1;  // tile 1
    int tj = 0;  // index of the current tile in this block's sequence
    int slot_n = slot, row0_n = row0, rows_n = rows, nt_n = nt;
    if (has_n) seek(Ln, slot_n, row0_n, rows_n, nt_n);
    __amdgpu_buffer_rsrc_t a_n = a_of(row0_n, rows_n), b_n = b_of(slot_n, nt_n);
    a_offsets(row0_n, rows_n, a_off_n);
    int ab = 0, bb = 0;  // buffers of the current stage

    // One tile in mode M (0 full, 1 half, 2 quarter): its K loop and epilogue.
    // The tile's stage 0 has landed and is visible (previous barrier).
    auto run_tile = [&](auto mode) __attribute__((always_inline)) {
      constexpr int M = decltype(mode)::value;
      constexpr int MBm = (M == 2) ? 2 : 4;  // 32-row blocks per wave
      constexpr int NBm = (M == 0) ? 4 : 2;  // 32-column blocks per wave
      constexpr int NQ = MBm * NBm;          // MFMAs per sub-step
      constexpr int ND = MBm + NBm;          // fragment reads per sub-step
      const int rbase = (M == 0) ? wm * 128 : 0;
      const int cw = (M == 0) ? (SWIGLU ? wn * 64 : wn * 128) : (SWIGLU ? wave * 32 : wave * 64);
      const int xrow = rbase + (lane & 31), wrow = cw + (lane & 31);
      int xoff[KK], woff[KK];
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        xoff[kk] = xrow * BK + (((2 * kk + khalf) ^ swz<CH>(xrow)) << 3);
        woff[kk] = 2 * A_ST + wrow * BK + (((2 * kk + khalf) ^ swz<CH>(wrow)) << 3);
      }
      // Weight rows of block nb relative to wrow (gate blocks, then up blocks).
      auto wblk = [](int nb) constexpr {
        return SWIGLU ? ((nb < NBm / 2) ? nb * 32 : BN / 2 + (nb - NBm / 2) * 32) : nb * 32;
      };
      bf16x8 xf[2][MBm], wf[2][NBm];
      f32x16 acc[NBm][MBm];
#pragma unroll
      for (int nb = 0; nb < NBm; ++nb)
#pragma unroll
        for (int mb = 0; mb < MBm; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[nb][mb][r] = 0.0f;
      // One stage; the last stage of the tile reads no fragments after its
      // barrier (the next tile may run in another mode).
#define TG_STAGE(kt, LAST)                                                                 \
  do {                                                                                     \
    TG_TARGETS(kt, LAST);                                                                  \
    TG_FRAGS(ab, bb, 1, 1);                                                                \
    TG_ISSUE_A(ra, offa, ka * BK, abn, 0, AI / 2);                                        \
    TG_MFMAS(0, 0, NQ);                                                                    \
    TG_PATTERN_LOADS;                                                                      \
    __builtin_amdgcn_sched_barrier(0);                                                     \
    TG_FRAGS(ab, bb, 2, 0);                                                                \
    TG_ISSUE_A(ra, offa, ka * BK, abn, AI / 2, AI);                                        \
    TG_MFMAS(1, 0, NQ);                                                                    \
    TG_PATTERN_LOADS;                                                                      \
    __builtin_amdgcn_sched_barrier(0);                                                     \
    TG_FRAGS(ab, bb, 3, 1);                                                                \
    TG_ISSUE_B(rb, kb * BK, bbn, 0, BI / 2);                                               \
    TG_MFMAS(0, 0, NQ);                                                                    \
    TG_PATTERN_LOADS;                                                                      \
    __builtin_amdgcn_sched_barrier(0);                                                     \
    __builtin_amdgcn_s_waitcnt(0xc07f); /* lgkmcnt(0): this stage's buffers are read */    \
    TG_ISSUE_B(rb, kb * BK, bbn, BI / 2, BI);                                              \
    TG_MFMAS(1, 0, NQ / 2);                                                                \
    TG_PATTERN_PRE;                                                                        \
    __builtin_amdgcn_sched_barrier(0);                                                     \
    TG_WAIT_VM(BI);                                                                        \
    block_barrier();                                                                       \
    ab ^= 1;                                                                               \
    bb = (bb == 2) ? 0 : bb + 1;                                                           \
    if constexpr (!(LAST)) {                                                               \
      TG_FRAGS(ab, bb, 0, 0);                                                              \
      TG_MFMAS(1, NQ / 2, NQ);                                                             \
      TG_PATTERN_POST;                                                                     \
    } else {                                                                               \
      TG_MFMAS(1, NQ / 2, NQ);                                                             \
    }                                                                                      \
    __builtin_amdgcn_sched_barrier(0);                                                     \
  } while (0)
      TG_FRAGS(ab, bb, 0, 0);
      for (int kt = 0; kt < nk - 1; ++kt) TG_STAGE(kt, false);  // nk >= 2
      TG_STAGE(nk - 1, true);
      cl_got = __builtin_amdgcn_readfirstlane(cl_v);  // thread 0's claim in wave 0
#undef TG_STAGE
      // acc[nb][mb] register r of lane l: row mb*32 + l%32, column
      // nb*32 + 8*(r/4) + 4*(l/32) + r%4 of the wave's sub-tile; SwiGLU pairs
      // gate block nb with up block nb + NBm/2.
      const int colbase = SWIGLU ? nt * (BN / 2) + cw : nt * BN + cw;
      if constexpr (SWIGLU) {
#pragma unroll
        for (int mb = 0; mb < MBm; ++mb) {
          const int r = rbase + mb * 32 + (lane & 31);
          uint16_t* crow = C + (size_t)(row0 + r) * ldc + colbase + 4 * (lane >> 5);
#pragma unroll
          for (int nb = 0; nb < NBm / 2; ++nb) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              float v[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const int rr = 4 * q + e;
                v[e] = swiglu(acc[nb][mb][rr], acc[nb + NBm / 2][mb][rr]);
              }
              uint2 pk;
              pk.x = pack_bf16x2(v[0], v[1]);
              pk.y = pack_bf16x2(v[2], v[3]);
              if (r < rows && colbase + 4 * (lane >> 5) + nb * 32 + 8 * q < ldc)
                *reinterpret_cast<uint2*>(crow + nb * 32 + 8 * q) = pk;
            }
          }
        }
      } else {
        // The down projection's rows leave as whole 128-byte lines: each
        // 32-row by 64-column block of the wave's sub-tile is staged in the
        // wave's own quarter of the A buffer that the last stage released
        // (the part that only this wave's next A loads refill, issued after
        // these reads; rows padded by 16 bytes against bank conflicts) and
        // read back as 16-byte pieces of whole rows, eight rows per store.
        // Straight from the accumulators each store would put 16 bytes into
        // each of 32 rows; staged, the DeepSeek-sized down GEMM runs 7-8 %
        // faster; the gate/up GEMM's output gains nothing from the same
        // staging, so it keeps its direct stores. The stores go through a resource
        // over the tile's rows, so rows past its end are dropped by the
        // hardware's range check.
        constexpr int PITCH = 64 + 8;  // staged row pitch (elements)
        static_assert(32 * PITCH <= A_ST / NWAVE, "staging fits in the wave's quarter");
        lds_u16* const region = smem3 + (ab ^ 1) * A_ST + wave * (A_ST / NWAVE);
        lds_u16* const wbase = region + (lane & 31) * PITCH + 4 * (lane >> 5);
        lds_u16* const rbase_l = region + (lane >> 3) * PITCH + (lane & 7) * 8;
        const __amdgpu_buffer_rsrc_t c_rsrc =
            make_rsrc(C + (size_t)row0 * ldc, (uint32_t)rows * ldc * 2);
#pragma unroll
        for (int hb = 0; hb < NBm / 2; ++hb) {
          const int col = colbase + hb * 64 + (lane & 7) * 8;
          const int voff0 = col < ldc ? ((rbase + (lane >> 3)) * ldc + col) * 2 : kOut;
#pragma unroll
          for (int mb = 0; mb < MBm; ++mb) {
#pragma unroll
            for (int n2 = 0; n2 < 2; ++n2) {
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const f32x16& a = acc[2 * hb + n2][mb];
                const u32x2 pk = {pack_bf16x2(a[4 * q], a[4 * q + 1]),
                                  pack_bf16x2(a[4 * q + 2], a[4 * q + 3])};
                *reinterpret_cast<__attribute__((address_space(3))) u32x2*>(
                    wbase + n2 * 32 + 8 * q) = pk;
              }
            }
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const u32x4 v = *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(
                  rbase_l + i * 8 * PITCH);
              const int voff = voff0 == kOut ? kOut : voff0 + (mb * 32 + i * 8) * ldc * 2;
              __builtin_amdgcn_raw_buffer_store_b128(v, c_rsrc, voff, 0, 0);
            }
          }
        }
      }
    };

    // Prologue: A and B of stage 0, B of stage 1; stage 0 visible.
    TG_ISSUE_A(a_cur, a_off, 0, 0, 0, AI);
    TG_ISSUE_B(b_cur, 0, 0, 0, BI);
    TG_ISSUE_B(b_cur, BK, 1, 0, BI);
    TG_WAIT_VM(BI);
    block_barrier();

    for (;;) {
      claim_issue(tj);  // no effect without a schedule or when no tile is left
      if (rows > 128) run_tile(std::integral_constant<int, 0>{});
      else if (rows > 64) run_tile(std::integral_constant<int, 1>{});
      else run_tile(std::integral_constant<int, 2>{});
      if (!has_n) break;
      // Tile tj + 2 becomes the next tile at this switch. With a schedule
      // wave 0 resolves it and hands it to the other waves through the A
      // stage buffer that the last stage released (the next tile's first
      // stage refills it only after the second barrier).
      int t2;
      if (dyn) {
        int* const rec = reinterpret_cast<int*>(smem + (ab ^ 1) * A_ST);
        if (wave == 0) {
          const int t = claim_resolve(tj + 2);
          if (lane == 0) *rec = t;
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the record is written
        block_barrier();
        t2 = __builtin_amdgcn_readfirstlane(*rec);
        __builtin_amdgcn_s_waitcnt(0xc07f);  // and read by every wave
        block_barrier();
      } else {
        t2 = Ln + per_xcd_blocks < hi ? Ln + per_xcd_blocks : -1;
      }
      row0 = row0_n;
      rows = rows_n;
      nt = nt_n;
      a_cur = a_n;
      b_cur = b_n;
#pragma unroll
      for (int i = 0; i < AI; ++i) a_off[i] = a_off_n[i];
      Ln = t2;
      has_n = Ln >= 0;
      ++tj;
      if (has_n) {
        seek(Ln, slot_n, row0_n, rows_n, nt_n);
        a_n = a_of(row0_n, rows_n);
        b_n = b_of(slot_n, nt_n);
        a_offsets(row0_n, rows_n, a_off_n);
      }
    }
    TG_WAIT_VM(0);  // no LDS write may land after the walk
#undef TG_TARGETS
#undef TG_PATTERN_POST
#undef TG_PATTERN_PRE
#undef TG_PATTERN_LOADS
#undef TG_DM
#undef TG_SG
#undef TG_FRAGS
#undef TG_MFMAS
#undef TG_ISSUE_A
#undef TG_ISSUE_B
  }
  if constexpr (TAIL) {
    if (!tail) return;
    __syncthreads();
    // The spilled tiles run as 128-column halves of their upper and lower
    // 128 rows: pieces 0 .. 2 rem - 1 are the upper halves of every spilled
    // tile (two column halves each), pieces 2 rem .. 4 rem - 1 the lower
    // halves, which are empty for tiles of at most 128 rows. With a schedule
    // area the pieces are claimed from a counter (claims[8]), so that blocks
    // whose walk held cheap partial tiles, and end it early, take more of
    // them; without one they are dealt round robin over the grid. Each piece
    // runs at the height its rows need, with as many stage buffers as that
    // height leaves room for in LDS: with a long K a piece is bound by the
    // latency of its weight stream, not by its MFMAs.
    const int npieces = 4 * rem;
    int* const piece_ctr = claims ? claims + kXcds : nullptr;
    // Thread 0 claims the next piece; the block reads it through LDS, whose
    // stage buffers are free between pieces.
    auto next_piece = [&](int prev) {
      if (!piece_ctr) return prev < 0 ? (int)blockIdx.x : prev + G;
      __syncthreads();
      if (threadIdx.x == 0) reinterpret_cast<int*>(smem)[0] = atomicAdd(piece_ctr, 1);
      __syncthreads();
      const int v = reinterpret_cast<const int*>(smem)[0];
      __syncthreads();  // every wave has read it before the next piece's loads land
      return v;
    };
    for (int p = next_piece(-1); p < npieces; p = next_piece(p)) {
      const int half = p / (2 * rem), r = p - half * (2 * rem);
      TileInfo t;
      int m;
      if (!find_tile(offsets, S, BM, NT, n_head + r / 2, &t, &m)) break;
      m = 2 * m + half;
      t.nt = 2 * t.nt + (r & 1);
      const int rows = min(BM / 2, t.rows - m * (BM / 2));
      // A piece past a partial last panel has no output column to store.
      const int col0 = t.nt * (SWIGLU ? BN / 4 : BN / 2);
      if (rows > 0 && col0 < ldc) {
        t.row0 += m * (BM / 2);
        t.rows = rows;
        if (rows <= 32)
          gemm_tile<32, BN / 2, BK, 1, 4, SWIGLU, GATHER, 8>(smem, t, A, B, K, NW, I, C, ldc, perm,
                                                            1, A_rows);
        else if (rows <= 64)
          gemm_tile<64, BN / 2, BK, 2, 2, SWIGLU, GATHER, 6>(smem, t, A, B, K, NW, I, C, ldc, perm,
                                                            1, A_rows);
        else
          gemm_tile<BM / 2, BN / 2, BK, 2, 2, SWIGLU, GATHER, 5>(smem, t, A, B, K, NW, I, C, ldc,
                                                              perm, 1, A_rows);
        __syncthreads();
      }
    }
  }
}

int cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    return 256;
  return n;
}

std::atomic<int> g_tile_policy{kTilesAuto};

// Launch of the 4-wave persistent kernel: one block per CU (a multiple of
// 8); K of at least 2 stages (d and I are multiples of 64, at least 128).
template <bool SWIGLU, bool GATHER, bool TAIL>
hipError_t launch_persistent4(const uint16_t* A, const int32_t* offsets, int S, const uint16_t* B,
                              int K, int NW, int I, uint16_t* C, int ldc, int NT,
                              hipStream_t stream, const int32_t* perm, int kq, int A_rows,
                              const GemmSched* sched) {
  int l = 0;
  while ((1 << l) < kq) ++l;
  const uint32_t m = (uint32_t)((((uint64_t)1 << (31 + l)) + (uint64_t)kq - 1) / (uint64_t)kq);
  const int grid = std::max(kXcds, cu_count() / kXcds * kXcds);  // a multiple of 8, never 0
  const bool dyn = sched && sched->claims;
  hipLaunchKernelGGL((grouped_gemm_persistent4_kernel<SWIGLU, GATHER, TAIL>), dim3(grid), dim3(256),
                     0, stream, A, offsets, S, B, K, NW, I, C, ldc, NT, perm, kq, m, l, A_rows,
                     dyn ? sched->claims : nullptr,
                     g_tile_policy.load(std::memory_order_relaxed));
  return hipGetLastError();
}

constexpr int kBN = 256;

// Weight panels per slot: gate/up panels hold kBN / 2 output columns (as
// many gate as up rows), down panels kBN. A last, partial panel (I or d not
// a multiple of the panel width) reads zeros past the slot's weight rows and
// stores only the columns below the output width.
int panels_gateup(int I) { return (I + kBN / 2 - 1) / (kBN / 2); }
int panels_down(int d) { return (d + kBN - 1) / kBN; }

}  // namespace

void set_tile_policy(int policy) { g_tile_policy.store(policy, std::memory_order_relaxed); }

hipError_t launch_ffn_gateup(const uint16_t* x_perm, const int32_t* offsets, int S, int max_rows,
                             const uint16_t* w13, int d, int I, uint16_t* h, hipStream_t stream,
                             const GemmSched* sched) {
  if (max_rows == 0) return hipSuccess;
  return launch_persistent4<true, false, false>(x_perm, offsets, S, w13, d, 2 * I, I, h, I,
                                                panels_gateup(I), stream, nullptr, 1, 0, sched);
}

hipError_t launch_ffn_gateup_gather(const uint16_t* x, int T, const int32_t* perm, int k,
                                    const int32_t* offsets, int S, int max_rows,
                                    const uint16_t* w13, int d, int I, uint16_t* h,
                                    hipStream_t stream, const GemmSched* sched) {
  if (max_rows == 0) return hipSuccess;
  return launch_persistent4<true, true, false>(x, offsets, S, w13, d, 2 * I, I, h, I,
                                               panels_gateup(I), stream, perm, k, T, sched);
}

hipError_t launch_ffn_down(const uint16_t* h, const int32_t* offsets, int S, int max_rows,
                           const uint16_t* w2, int d, int I, uint16_t* y, hipStream_t stream,
                           const GemmSched* sched) {
  if (max_rows == 0) return hipSuccess;
  return launch_persistent4<false, false, true>(h, offsets, S, w2, I, d, 0, y, d, panels_down(d),
                                                stream, nullptr, 1, 0, sched);
}

hipError_t launch_expert_ffn(const uint16_t* x_perm, const int32_t* offsets, int S, int max_rows,
                             const uint16_t* w13, const uint16_t* w2, int d, int I, uint16_t* h,
                             uint16_t* y, hipStream_t stream) {
  hipError_t e = launch_ffn_gateup(x_perm, offsets, S, max_rows, w13, d, I, h, stream);
  if (e != hipSuccess) return e;
  return launch_ffn_down(h, offsets, S, max_rows, w2, d, I, y, stream);
}

}  // namespace tg
