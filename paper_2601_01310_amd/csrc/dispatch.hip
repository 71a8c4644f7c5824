// ERT remap with failure mask, per-slot counts, deterministic permutation and
// the activation gather (§4.2, §5.1, §5.3; per-expert batching, §2.2.1).
//
// Three passes over the routed pairs, all integer and free of ordering races:
//   1. remap_count: per pair, the first live candidate slot of its expert;
//      per chunk of pairs, an S-wide histogram and an unserved count
//      (integer LDS atomics: the totals do not depend on their order).
//      Pairs of tokens outside the batch (token_valid[t] == 0, the partial
//      batch of §5.2) get slot -2 and are not counted. In replay mode (§5.1)
//      a pair keeps its first-pass slot while that slot is alive and is
//      otherwise given its first live candidate now, to be recomputed;
//   2. scan: per-slot totals, exclusive slot offsets, and the position of
//      every (chunk, slot) within its slot in chunk order (the histograms
//      are slot-major, so one wave scans one slot's chunks). When S times
//      the number of chunks is at most 1024, each scatter block does this
//      for itself from the whole histogram instead, and the launch is saved;
//   3. scatter: each wave walks an equal share of a chunk in pair order and
//      ranks the pairs of each group of 64 by slot: one ballot per bit of
//      the slot index gives every lane the lanes that share its slot, so the
//      rank costs the same for any mix of slots, and rows follow
//      (slot, token, rank).
// Up to 4096 pairs, one block runs all three passes (the batch of a decode
// step fits, and two launches are saved; past that the three grids are
// faster, as each group of 1024 pairs costs the one block about 1.7 us).
// The gather then copies one activation row per routed pair with 16-byte
// loads and stores (rows are contiguous in source and destination, so the
// copy is fully coalesced without staging).
#include "tg_device.h"
#include "tg_launch.h"

namespace tg {
namespace {

constexpr int kMaxS = 1024;
constexpr int kBlock = 256;
constexpr int kFusedScanHist = 1024;  // S * nchunks up to which scatter scans by itself

// Slot of a pair of expert e: the first live ERT candidate of e.
// REPLAY: -1 also when the first pass's slot pr is still alive (its result
// stands). *unserved: the expert lists a local candidate, none alive.
template <bool REPLAY>
__device__ __forceinline__ int resolve_expert(int e, int pr, const int32_t* __restrict__ ert,
                                              int E, int R, const uint8_t* __restrict__ alive,
                                              int S, bool* unserved) {
  int slot = -1;
  bool listed = false;
  if (e >= 0 && e < E) {
    for (int r = 0; r < R; ++r) {
      const int c = ert[(size_t)e * R + r];
      if (c >= 0 && c < S) {
        listed = true;
        if (alive[c]) {
          slot = c;
          break;
        }
      }
    }
  }
  *unserved = slot < 0 && listed;
  if (REPLAY && pr >= 0 && pr < S && alive[pr]) slot = -1;  // first-pass result stands
  return slot;
}

// Slot that pair p is computed on: the first live ERT candidate of its
// expert; -2 for a token outside the batch. REPLAY: -1 also when the first
// pass's slot prior[p] is still alive (its result stands) or the token was
// outside the batch. *unserved: the expert lists a local candidate, none
// alive.
template <bool REPLAY>
__device__ __forceinline__ int resolve_pair(int p, const int32_t* __restrict__ ids, int k,
                                            const int32_t* __restrict__ ert, int E, int R,
                                            const uint8_t* __restrict__ alive, int S,
                                            const uint8_t* __restrict__ token_valid,
                                            const int32_t* __restrict__ prior, bool* unserved) {
  *unserved = false;
  int pr = 0;
  if (REPLAY) {
    pr = prior[p];
    if (pr == -2) return -1;
  } else if (token_valid && !token_valid[p / k]) {
    return -2;
  }
  return resolve_expert<REPLAY>(ids[p], pr, ert, E, R, alive, S, unserved);
}

// Lanes of the wave that hold a routed pair (s >= 0) on the same slot as
// this lane: start from the routed lanes and keep, for every bit of the slot
// index (sbits bits), the lanes that agree with this lane on that bit. The
// cost is the same for any mix of slots. 0 on lanes with s < 0.
__device__ __forceinline__ uint64_t same_slot_lanes(int s, int sbits) {
  uint64_t eq = __ballot(s >= 0);
  for (int b = 0; b < sbits; ++b) {
    const bool bit = (s >> b) & 1;
    const uint64_t mb = __ballot(bit);
    eq &= bit ? mb : ~mb;
  }
  return s >= 0 ? eq : 0;
}

// REPLAY: `prior` holds the first pass's slot of every pair; out_slot gets
// the slot the pair is recomputed on, or -1 when its first-pass result still
// stands (slot alive), it is outside the batch (-2), or no candidate is live.
template <bool REPLAY>
__global__ __launch_bounds__(kBlock) void remap_count_kernel(
    const int32_t* __restrict__ ids, int npairs, int k, const int32_t* __restrict__ ert, int E,
    int R, const uint8_t* __restrict__ alive, int S, const uint8_t* __restrict__ token_valid,
    const int32_t* __restrict__ prior, int32_t* __restrict__ out_slot, int32_t* __restrict__ hist,
    int32_t* __restrict__ unserved_chunk, int chunk, uint32_t* __restrict__ zero, int zero_words) {
  __shared__ int h[kMaxS];
  __shared__ int nu;
  for (int s = threadIdx.x; s < S; s += kBlock) h[s] = 0;
  if (threadIdx.x == 0) nu = 0;
  __syncthreads();
  const int base = blockIdx.x * chunk;
  for (int i = threadIdx.x; i < chunk; i += kBlock) {
    const int p = base + i;
    if (p >= npairs) break;
    bool unserved;
    const int slot =
        resolve_pair<REPLAY>(p, ids, k, ert, E, R, alive, S, token_valid, prior, &unserved);
    out_slot[p] = slot;
    if (unserved) atomicAdd(&nu, 1);
    if (slot >= 0) atomicAdd(&h[slot], 1);
  }
  __syncthreads();
  for (int s = threadIdx.x; s < S; s += kBlock) hist[(size_t)s * gridDim.x + blockIdx.x] = h[s];
  if (threadIdx.x == 0) unserved_chunk[blockIdx.x] = nu;
  // The GEMMs' schedule area of this call starts at zero.
  if (zero && blockIdx.x == 0)
    for (int i = threadIdx.x; i < zero_words; i += kBlock) zero[i] = 0;
}

// One block of 1024 threads (16 waves). hist[s * nchunks + c] holds the
// pairs of chunk c on slot s (nchunks <= 4 * 64). Wave w takes slots w,
// w + 16, ...: lane l sums chunks 4l .. 4l+3, a wave scan gives every chunk
// its exclusive position within the slot (written back in place, the
// scatter adds the slot offset), and the slot totals go through a block
// scan (wave scans and the waves' totals) to the exclusive slot offsets.
__global__ __launch_bounds__(1024) void scan_kernel(int32_t* __restrict__ hist,
                                                    const int32_t* __restrict__ unserved_chunk,
                                                    int nchunks, int S, int32_t* __restrict__ counts,
                                                    int32_t* __restrict__ offsets,
                                                    int32_t* __restrict__ n_unserved,
                                                    int32_t* __restrict__ total_out) {
  __shared__ int tot[1024];
  __shared__ int wsum[1024 / kWave];
  __shared__ int nu;
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = lane_id();
  if (tid == 0) nu = 0;
  for (int s = wave; s < S; s += 1024 / kWave) {
    int32_t* hs = hist + (size_t)s * nchunks;
    int v[4], sum = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 4 * lane + i;
      v[i] = (c < nchunks) ? hs[c] : 0;
      sum += v[i];
    }
    int incl = sum;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int t = __shfl_up(incl, off);
      if (lane >= off) incl += t;
    }
    int run = incl - sum;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 4 * lane + i;
      if (c < nchunks) hs[c] = run;
      run += v[i];
    }
    if (lane == kWave - 1) tot[s] = incl;
  }
  int part = 0;
  for (int c = tid; c < nchunks; c += 1024) part += unserved_chunk[c];
  __syncthreads();
  if (part) atomicAdd(&nu, part);
  // Inclusive scan over the slot totals: a wave scan per 64 slots, then the
  // totals of the waves before.
  const int total = (tid < S) ? tot[tid] : 0;
  int incl = total;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int t = __shfl_up(incl, off);
    if (lane >= off) incl += t;
  }
  if (lane == kWave - 1) wsum[wave] = incl;
  __syncthreads();
  for (int w = 0; w < wave; ++w) incl += wsum[w];
  if (tid < S) {
    counts[tid] = total;
    offsets[tid] = incl - total;
  }
  if (tid == S - 1) {
    offsets[S] = incl;
    if (total_out) total_out[0] = incl;
  }
  if (tid == 0) n_unserved[0] = nu;
}

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// SCAN false: hist[s * nchunks + c] is the position of chunk c's first pair
// within slot s and offsets the slot offsets (both from scan_kernel).
// SCAN true: hist holds the per-chunk counts of remap_count, and every block
// derives what it needs itself (its chunk's position in each slot and the
// slot offsets, from all of hist; for small S * nchunks this is cheaper
// than a launch); block 0 also writes counts, offsets, the unserved count
// and the total. sbits: bits of the largest slot index.
template <bool SCAN>
__global__ __launch_bounds__(kBlock) void scatter_kernel(
    const int32_t* __restrict__ pair_slot, int npairs, int S, int nchunks, int sbits,
    const int32_t* __restrict__ hist, const int32_t* __restrict__ unserved_chunk,
    int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ n_unserved, int32_t* __restrict__ total_out,
    int32_t* __restrict__ perm, int32_t* __restrict__ pair_row, int chunk) {
  constexpr int kWaves = kBlock / kWave;
  __shared__ int cnt[kWaves][kMaxS];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  // The chunk's pairs are split evenly (in multiples of 64) over the waves.
  const int c0 = blockIdx.x * chunk;
  const int n_c = min(chunk, npairs - c0);
  const int span = ((n_c + kWaves * kWave - 1) / (kWaves * kWave)) * kWave;
  const int p0 = c0 + wave * span;
  const int p1 = min(c0 + n_c, p0 + span);
  __shared__ int base[SCAN ? kMaxS : 1];  // first row of this chunk's pairs on each slot
  __shared__ int tot[SCAN ? kMaxS : 1];
  __shared__ int wsum[kWaves];
  for (int i = threadIdx.x; i < kWaves * kMaxS; i += kBlock) (&cnt[0][0])[i] = 0;
  constexpr int kPer = SCAN ? kFusedScanHist / kBlock : 1;
  int hv[kPer];
  if (SCAN) {
    // Thread i loads histogram entries i, i + 256, ... (all loads at once),
    // and the slot totals and this chunk's positions are summed in LDS
    // (integer atomics: the sums do not depend on their order).
    const int nh = S * nchunks;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int j = threadIdx.x + q * kBlock;
      hv[q] = j < nh ? hist[j] : 0;
    }
    for (int s = threadIdx.x; s < S; s += kBlock) {
      tot[s] = 0;
      base[s] = 0;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int j = threadIdx.x + q * kBlock;
      if (hv[q]) {
        const int s = j / nchunks, c = j - s * nchunks;
        atomicAdd(&tot[s], hv[q]);
        if (c < (int)blockIdx.x) atomicAdd(&base[s], hv[q]);
      }
    }
  }
  __syncthreads();
  if (SCAN) {
    // Exclusive scan of the slot totals: thread i holds slots 4i .. 4i+3.
    int v[4], sum = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int s = 4 * threadIdx.x + j;
      v[j] = s < S ? tot[s] : 0;
      sum += v[j];
    }
    int incl = sum;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int t = __shfl_up(incl, off);
      if (lane >= off) incl += t;
    }
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    for (int w = 0; w < wave; ++w) incl += wsum[w];
    int run = incl - sum;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int s = 4 * threadIdx.x + j;
      if (s < S) {
        base[s] += run;
        if (blockIdx.x == 0) {
          counts[s] = v[j];
          offsets[s] = run;
        }
      }
      run += v[j];
    }
    if (blockIdx.x == 0) {
      if (threadIdx.x == kBlock - 1) {
        offsets[S] = run;  // the last thread's run is the grand total
        if (total_out) total_out[0] = run;
      }
      if (wave == 0) {
        int nu = 0;
        for (int c = lane; c < nchunks; c += kWave) nu += unserved_chunk[c];
        nu = wave_sum_int(nu);
        if (lane == 0) n_unserved[0] = nu;
      }
    }
  }
  for (int p = p0 + lane; p < p1; p += kWave) {
    const int s = pair_slot[p];
    if (s >= 0) atomicAdd(&cnt[wave][s], 1);
  }
  __syncthreads();
  for (int s = threadIdx.x; s < S; s += kBlock) {
    int run = SCAN ? base[s] : offsets[s] + hist[(size_t)s * nchunks + blockIdx.x];
    for (int w = 0; w < kWaves; ++w) {
      const int v = cnt[w][s];
      cnt[w][s] = run;
      run += v;
    }
  }
  __syncthreads();
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int g = p0; g < p1; g += kWave) {
    const int p = g + lane;
    int s = -1;
    if (p < p1) {
      s = pair_slot[p];
      if (s < 0) pair_row[p] = -1;
    }
    if (!__ballot(s >= 0)) continue;  // uniform
    const uint64_t eq = same_slot_lanes(s, sbits);
    if (s >= 0) {
      const int row = cnt[wave][s] + __builtin_popcountll(eq & lt);
      perm[row] = p;
      pair_row[p] = row;
      // The slot's lowest lane advances the slot's next row (every lane's
      // read above precedes this write in the wave's LDS order).
      if (!(eq & lt)) cnt[wave][s] = row + __builtin_popcountll(eq);
    }
  }
}

// All three passes in one block of 1024 threads, for at most kSmallPairs
// pairs; thread i takes pairs i, i + 1024, ... The ERT and the liveness mask
// are first copied to LDS while the pairs' expert ids load, so resolving a
// pair costs one memory latency. Each wave counts its pairs per slot with
// same_slot_lanes (one LDS add per distinct slot), a wave scan with one
// barrier gives the slot offsets, and the pairs are then ranked 1024 at a
// time in pair order (wave w holds pairs 64w .. 64w+63 of the group) exactly
// as scatter_kernel does, so rows follow (slot, token, rank).
constexpr int kOneBlock = 1024;
constexpr int kSmallPairs = 4096;
constexpr int kSmallPer = kSmallPairs / kOneBlock;
constexpr int kMaxErt = 1024 * 16;  // E * R entries staged in LDS (E <= 1024, R <= 16)

template <bool REPLAY>
__global__ __launch_bounds__(kOneBlock) void dispatch_one_block_kernel(
    const int32_t* __restrict__ ids, int npairs, int k, const int32_t* __restrict__ ert, int E,
    int R, const uint8_t* __restrict__ alive, int S, int sbits,
    const uint8_t* __restrict__ token_valid, const int32_t* __restrict__ prior,
    int32_t* __restrict__ out_slot, int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ perm, int32_t* __restrict__ pair_row, int32_t* __restrict__ n_unserved,
    int32_t* __restrict__ total_out, uint32_t* __restrict__ zero, int zero_words) {
  constexpr int kWaves = kOneBlock / kWave;
  // cnt[w][s]: pairs of wave w on slot s in the current group of 1024, then
  // their first row; 0 wherever wave w has no pair on s.
  __shared__ int cnt[kWaves][kMaxS];
  __shared__ int run[kMaxS];
  __shared__ int ert_s[kMaxErt];
  __shared__ uint8_t alive_s[kMaxS];
  __shared__ int wsum[kWaves];
  __shared__ int nu;
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = lane_id();
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

  // Loads that do not depend on one another: the pairs' ids (and first-pass
  // slots or batch flags), the ERT and the mask. Raw values only, so no load
  // waits for another.
  // Every lane loads (indices past the end read the last pair, and their
  // values are never used), so no load sits in a divergent branch.
  int e_of[kSmallPer], f_of[kSmallPer];
  if (npairs > 0) {
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
      const int p = min(tid + i * kOneBlock, npairs - 1);
      e_of[i] = ids[p];
      f_of[i] = REPLAY ? prior[p] : 1;
    }
    if (!REPLAY && token_valid) {
#pragma unroll
      for (int i = 0; i < kSmallPer; ++i)
        f_of[i] = token_valid[min(tid + i * kOneBlock, npairs - 1) / k];
    }
  }
  for (int j = tid; j < E * R; j += kOneBlock) ert_s[j] = ert[j];
  for (int j = tid; j < S; j += kOneBlock) {
    alive_s[j] = alive[j];
    run[j] = 0;
  }
  for (int j = tid; j < kWaves * S; j += kOneBlock) cnt[j / S][j % S] = 0;
  if (tid == 0) nu = 0;
  __syncthreads();

  // Global stores wait until the end: on this chip a wait for a load also
  // waits for every earlier store, so stores issued here would stall the
  // passes below.
  int my_slot[kSmallPer];
  uint64_t my_eq[kSmallPer];
#pragma unroll
  for (int i = 0; i < kSmallPer; ++i) {
    my_slot[i] = -1;
    my_eq[i] = 0;
    if (i * kOneBlock >= npairs) continue;  // uniform
    const int p = tid + i * kOneBlock;
    bool unserved = false;
    int s = -1;
    if (p < npairs) {
      if (REPLAY ? f_of[i] != -2 : f_of[i] != 0)
        s = resolve_expert<REPLAY>(e_of[i], REPLAY ? f_of[i] : 0, ert_s, E, R, alive_s, S,
                                   &unserved);
      else
        s = REPLAY ? -1 : -2;
    }
    const int n_un = __builtin_popcountll(__ballot(unserved));
    if (lane == 0 && n_un) atomicAdd(&nu, n_un);
    const uint64_t eq = same_slot_lanes(s, sbits);
    if (s >= 0 && !(eq & lt)) atomicAdd(&run[s], __builtin_popcountll(eq));
    my_slot[i] = s;
    my_eq[i] = eq;
  }
  __syncthreads();

  // Exclusive scan of the slot totals: a wave scan per 64 slots, then the
  // totals of the waves before.
  const int total = (tid < S) ? run[tid] : 0;
  int incl = total;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int t = __shfl_up(incl, off);
    if (lane >= off) incl += t;
  }
  if (lane == kWave - 1) wsum[wave] = incl;
  __syncthreads();
  for (int w = 0; w < wave; ++w) incl += wsum[w];
  if (tid < S) run[tid] = incl - total;  // next row of the slot

  int my_row[kSmallPer];
#pragma unroll
  for (int i = 0; i < kSmallPer; ++i) my_row[i] = -1;
#pragma unroll
  for (int i = 0; i < kSmallPer; ++i) {
    if (i * kOneBlock >= npairs) break;  // uniform
    const int s = my_slot[i];
    const uint64_t eq = my_eq[i];
    const bool lead = s >= 0 && !(eq & lt);
    if (lead) cnt[wave][s] = __builtin_popcountll(eq);
    __syncthreads();
    // Thread q turns slot q's per-wave counts into first rows (all reads
    // first, so they are in flight together; absent waves keep 0).
    if (tid < S) {
      int v[kWaves];
#pragma unroll
      for (int w = 0; w < kWaves; ++w) v[w] = cnt[w][tid];
      int r = run[tid];
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        cnt[w][tid] = v[w] ? r : 0;
        r += v[w];
      }
      run[tid] = r;
    }
    __syncthreads();
    if (s >= 0) my_row[i] = cnt[wave][s] + __builtin_popcountll(eq & lt);
    // Every lane's read above precedes this write in the wave's LDS order.
    if (lead) cnt[wave][s] = 0;
  }

  if (tid < S) {
    counts[tid] = total;
    offsets[tid] = incl - total;
  }
  if (tid == S - 1) {
    offsets[S] = incl;
    if (total_out) total_out[0] = incl;
  }
  if (tid == 0) n_unserved[0] = nu;
#pragma unroll
  for (int i = 0; i < kSmallPer; ++i) {
    const int p = tid + i * kOneBlock;
    if (p < npairs) {
      out_slot[p] = my_slot[i];
      pair_row[p] = my_row[i];
      if (my_row[i] >= 0) perm[my_row[i]] = p;
    }
  }
  // The GEMMs' schedule area of this call starts at zero.
  if (zero)
    for (int j = tid; j < zero_words; j += kOneBlock) zero[j] = 0;
}

__global__ __launch_bounds__(kBlock) void gather_kernel(const uint4* __restrict__ x,
                                                        const int32_t* __restrict__ perm,
                                                        const int32_t* __restrict__ offsets, int S,
                                                        int k, int nch, uint4* __restrict__ x_perm) {
  const int P = offsets[S];
  const long total = (long)P * nch;
  for (long q = (long)blockIdx.x * kBlock + threadIdx.x; q < total; q += (long)gridDim.x * kBlock) {
    const int r = (int)(q / nch);
    const int c = (int)(q - (long)r * nch);
    const int t = perm[r] / k;
    x_perm[q] = x[(size_t)t * nch + c];
  }
}

}  // namespace

int dispatch_chunk(long npairs) {
  const long per = (npairs + kDispatchChunks - 1) / kDispatchChunks;
  const long c = (per + 255) / 256 * 256;
  return (int)(c < 256 ? 256 : c);
}

size_t dispatch_workspace_bytes(int T, int k, int S) {
  const size_t npairs = (size_t)T * k;
  const int chunk = dispatch_chunk((long)npairs);
  const size_t nchunks = (npairs + chunk - 1) / chunk;
  const size_t hist = nchunks * (size_t)S * sizeof(int32_t);
  return ((hist + 255) & ~(size_t)255) + ((nchunks * sizeof(int32_t) + 255) & ~(size_t)255) + 256;
}

namespace {

hipError_t remap_dispatch(bool replay, const int32_t* ids, int T, int k, const int32_t* ert, int E,
                          int R, const uint8_t* alive, int S, const uint8_t* token_valid,
                          const int32_t* prior, const uint16_t* x, int d, int32_t* pair_slot,
                          int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* pair_row,
                          uint16_t* x_perm, int32_t* n_unserved, int32_t* total_out, void* ws,
                          hipStream_t stream, void* sched_area) {
  uint32_t* const zero = static_cast<uint32_t*>(sched_area);
  const int zero_words = sched_area ? (int)(kSchedBytes / 4) : 0;
  const int npairs = T * k;
  const int chunk = dispatch_chunk(npairs);
  const int nchunks = (npairs + chunk - 1) / chunk;
  const size_t hist_bytes = ((size_t)nchunks * S * sizeof(int32_t) + 255) & ~(size_t)255;
  int32_t* hist = static_cast<int32_t*>(ws);
  int32_t* unserved_chunk = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + hist_bytes);
  const int sbits = (S > 1) ? 32 - __builtin_clz((unsigned)(S - 1)) : 0;
  if (npairs <= kSmallPairs) {
    if (replay)
      hipLaunchKernelGGL(dispatch_one_block_kernel<true>, dim3(1), dim3(kOneBlock), 0, stream, ids,
                         npairs, k, ert, E, R, alive, S, sbits, nullptr, prior, pair_slot, counts,
                         offsets, perm, pair_row, n_unserved, total_out, zero, zero_words);
    else
      hipLaunchKernelGGL(dispatch_one_block_kernel<false>, dim3(1), dim3(kOneBlock), 0, stream,
                         ids, npairs, k, ert, E, R, alive, S, sbits, token_valid, nullptr,
                         pair_slot, counts, offsets, perm, pair_row, n_unserved, total_out, zero,
                         zero_words);
    if (x_perm && npairs > 0) {
      const int nch = d / 8;
      const long maxq = (long)npairs * nch;
      const long blocks = (maxq + kBlock - 1) / kBlock;
      const int grid = (int)(blocks < 8192 ? blocks : 8192);
      hipLaunchKernelGGL(gather_kernel, dim3(grid), dim3(kBlock), 0, stream,
                         reinterpret_cast<const uint4*>(x), perm, offsets, S, k, nch,
                         reinterpret_cast<uint4*>(x_perm));
    }
    return hipGetLastError();
  }
  if (nchunks > 0) {
    if (replay)
      hipLaunchKernelGGL(remap_count_kernel<true>, dim3(nchunks), dim3(kBlock), 0, stream, ids,
                         npairs, k, ert, E, R, alive, S, nullptr, prior, pair_slot, hist,
                         unserved_chunk, chunk, zero, zero_words);
    else
      hipLaunchKernelGGL(remap_count_kernel<false>, dim3(nchunks), dim3(kBlock), 0, stream, ids,
                         npairs, k, ert, E, R, alive, S, token_valid, nullptr, pair_slot, hist,
                         unserved_chunk, chunk, zero, zero_words);
  }
  // A small histogram is scanned by every scatter block (one launch less).
  const bool fused_scan = nchunks > 0 && (long)S * nchunks <= (long)kFusedScanHist;
  if (!fused_scan)
    hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(1024), 0, stream, hist, unserved_chunk, nchunks,
                       S, counts, offsets, n_unserved, total_out);
  if (nchunks > 0) {
    if (fused_scan)
      hipLaunchKernelGGL(scatter_kernel<true>, dim3(nchunks), dim3(kBlock), 0, stream, pair_slot,
                         npairs, S, nchunks, sbits, hist, unserved_chunk, counts, offsets,
                         n_unserved, total_out, perm, pair_row, chunk);
    else
      hipLaunchKernelGGL(scatter_kernel<false>, dim3(nchunks), dim3(kBlock), 0, stream, pair_slot,
                         npairs, S, nchunks, sbits, hist, unserved_chunk, counts, offsets,
                         n_unserved, total_out, perm, pair_row, chunk);
    if (x_perm) {
      const int nch = d / 8;
      const long maxq = (long)npairs * nch;
      const long blocks = (maxq + kBlock - 1) / kBlock;
      const int grid = (int)(blocks < 8192 ? blocks : 8192);
      hipLaunchKernelGGL(gather_kernel, dim3(grid), dim3(kBlock), 0, stream,
                         reinterpret_cast<const uint4*>(x), perm, offsets, S, k, nch,
                         reinterpret_cast<uint4*>(x_perm));
    }
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_remap_dispatch(const int32_t* ids, int T, int k, const int32_t* ert, int E, int R,
                                 const uint8_t* alive, int S, const uint16_t* x, int d,
                                 int32_t* pair_slot, int32_t* counts, int32_t* offsets,
                                 int32_t* perm, int32_t* pair_row, uint16_t* x_perm,
                                 int32_t* n_unserved, void* ws, hipStream_t stream,
                                 const uint8_t* token_valid, void* sched_area) {
  return remap_dispatch(false, ids, T, k, ert, E, R, alive, S, token_valid, nullptr, x, d,
                        pair_slot, counts, offsets, perm, pair_row, x_perm, n_unserved, nullptr,
                        ws, stream, sched_area);
}

hipError_t launch_replay_dispatch(const int32_t* ids, int T, int k, const int32_t* ert, int E,
                                  int R, const uint8_t* alive, int S, const int32_t* prior_slot,
                                  const uint16_t* x, int d, int32_t* replay_slot, int32_t* counts,
                                  int32_t* offsets, int32_t* perm, int32_t* replay_row,
                                  uint16_t* x_perm, int32_t* n_unserved, int32_t* n_replayed,
                                  void* ws, hipStream_t stream, void* sched_area) {
  return remap_dispatch(true, ids, T, k, ert, E, R, alive, S, nullptr, prior_slot, x, d,
                        replay_slot, counts, offsets, perm, replay_row, x_perm, n_unserved,
                        n_replayed, ws, stream, sched_area);
}

}  // namespace tg
