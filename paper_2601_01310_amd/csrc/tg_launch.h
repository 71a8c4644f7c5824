// Internal launchers of the libtg kernels. Arguments are validated by the
// C-ABI layer (tg_api.cpp) before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "tg.h"

namespace tg {

// C-ABI internals (tg_api.cpp) shared with the no-allocation forward
// (noalloc.hip): argument validation with the workspace size it implies,
// the checked forward on a given workspace, and the thread-local error
// detail that tg_last_error() reports.
tg_status ew_check(const tg_ew_args* a, size_t* ws_bytes);
tg_status ew_forward(const tg_ew_args* a, void* ws, size_t ws_bytes, void* stream,
                     void* const* events);
tg_status set_error(tg_status s, const char* fmt, ...);

// Work area of the dynamic tile schedule of the two grouped GEMMs of one
// forward (or replay): per GEMM, 16 claim counters (one per XCD for the
// tile walk, then one for the pieces of a spilled last round; the rest
// unused). The dispatch of the same call zeroes the whole area before the
// GEMMs run.
struct GemmSched {
  int32_t* claims;
};
constexpr size_t kSchedBytes = 2 * 16 * sizeof(int32_t);
// Carves the two GEMMs' schedules out of a kSchedBytes area (base may be null).
inline void sched_carve(void* base, GemmSched* gateup, GemmSched* down) {
  char* b = static_cast<char*>(base);
  gateup->claims = b ? reinterpret_cast<int32_t*>(b) : nullptr;
  down->claims = b ? reinterpret_cast<int32_t*>(b + 64) : nullptr;
}

hipError_t launch_gate_topk(const uint16_t* x, const uint16_t* wg, const float* logits_in, int T,
                            int d, int E, int k, float* logits_out, int32_t* ids, float* w,
                            hipStream_t stream);

// Pairs are processed in at most kDispatchChunks chunks (each a multiple of
// 256 pairs, at least 256); the workspace holds one S-wide histogram and one
// unserved count per chunk.
constexpr int kDispatchChunks = 256;
int dispatch_chunk(long npairs);
size_t dispatch_workspace_bytes(int T, int k, int S);
// token_valid (optional, [T]): pairs of tokens with 0 get pair_slot -2 and
// are neither batched nor counted as unserved.
hipError_t launch_remap_dispatch(const int32_t* ids, int T, int k, const int32_t* ert, int E, int R,
                                 const uint8_t* alive, int S, const uint16_t* x, int d,
                                 int32_t* pair_slot, int32_t* counts, int32_t* offsets,
                                 int32_t* perm, int32_t* pair_row, uint16_t* x_perm,
                                 int32_t* n_unserved, void* ws, hipStream_t stream,
                                 const uint8_t* token_valid = nullptr, void* sched_area = nullptr);
// Replay batching: pairs whose first-pass slot (prior_slot) is no longer
// alive, or that had no live candidate, go to their first live candidate now
// (replay_slot; -1 for every other pair) and are batched by (slot, token,
// rank) into rows replay_row; n_replayed = number of such rows. Same
// workspace as launch_remap_dispatch.
hipError_t launch_replay_dispatch(const int32_t* ids, int T, int k, const int32_t* ert, int E,
                                  int R, const uint8_t* alive, int S, const int32_t* prior_slot,
                                  const uint16_t* x, int d, int32_t* replay_slot, int32_t* counts,
                                  int32_t* offsets, int32_t* perm, int32_t* replay_row,
                                  uint16_t* x_perm, int32_t* n_unserved, int32_t* n_replayed,
                                  void* ws, hipStream_t stream, void* sched_area = nullptr);

// Tile height of the grouped GEMMs: chosen per launch on the device (auto)
// or forced; every choice gives the same bits.
enum TilePolicy { kTilesAuto = 0, kTilesSmall = 1, kTilesFull = 2 };
void set_tile_policy(int policy);

// sched (optional): the GEMM's dynamic-schedule area, zeroed before the
// launch; without it the tiles are dealt statically. Both give the same bits.
hipError_t launch_ffn_gateup(const uint16_t* x_perm, const int32_t* offsets, int S, int max_rows,
                             const uint16_t* w13, int d, int I, uint16_t* h, hipStream_t stream,
                             const GemmSched* sched = nullptr);
// Same as launch_ffn_gateup with the activation rows gathered in place:
// grouped row r is row perm[r] / k of x [T, d] (requires T * d * 2 < 2^31).
hipError_t launch_ffn_gateup_gather(const uint16_t* x, int T, const int32_t* perm, int k,
                                    const int32_t* offsets, int S, int max_rows,
                                    const uint16_t* w13, int d, int I, uint16_t* h,
                                    hipStream_t stream, const GemmSched* sched = nullptr);
hipError_t launch_ffn_down(const uint16_t* h, const int32_t* offsets, int S, int max_rows,
                           const uint16_t* w2, int d, int I, uint16_t* y, hipStream_t stream,
                           const GemmSched* sched = nullptr);
hipError_t launch_expert_ffn(const uint16_t* x_perm, const int32_t* offsets, int S, int max_rows,
                             const uint16_t* w13, const uint16_t* w2, int d, int I, uint16_t* h,
                             uint16_t* y, hipStream_t stream);

hipError_t launch_combine(const uint16_t* y, const int32_t* pair_row, const float* w, int T, int k,
                          int d, uint16_t* out, hipStream_t stream);
// Re-forms out[t] for every token with a replayed pair or a pair whose
// first-pass slot has failed with no live candidate left; other rows of out
// are left as they are. A pair's output comes from y2[replay_row] when it was
// replayed, from y[pair_row] when its first-pass slot is still alive, and is
// absent otherwise. Same float32 rank-order sum as launch_combine.
hipError_t launch_recombine(const uint16_t* y, const int32_t* pair_row, const int32_t* prior_slot,
                            const uint8_t* alive, int S, const uint16_t* y2,
                            const int32_t* replay_row, const float* w, int T, int k, int d,
                            uint16_t* out, hipStream_t stream);

// Partial-batch trigger (one block): waits until every live AW has
// delivered, or the delivered rows of live AWs reach min_rows, or spin_limit
// polls have passed; then marks the rows of the delivered live AWs in
// token_valid [T] and writes status [4].
hipError_t launch_batch_trigger(const uint32_t* delivered, const uint8_t* aw_alive,
                                const int32_t* chunk_rows, int A, int T, int min_rows,
                                long long spin_limit, uint8_t* token_valid, int32_t* status,
                                hipStream_t stream);

// KV-segment checkpoint / restoration (one block per segment; the commit
// record is written by a second kernel after the copies).
hipError_t launch_kv_checkpoint(const void* kv, size_t kv_bytes, const uint64_t* seg_off,
                                const uint32_t* seg_bytes, int n, uint64_t first_seq, void* store,
                                tg_ckpt_record* log, int log_cap, uint64_t* commit, int max_blocks,
                                hipStream_t stream);
// Strided batch: segment i at first_offset + i * pitch (validated by the
// caller); copy engine for the bytes, one kernel for the records and commit.
hipError_t launch_kv_checkpoint_strided(const void* kv, uint64_t first_offset, uint64_t pitch,
                                        uint32_t seg_bytes, int n, uint64_t first_seq,
                                        void* store, tg_ckpt_record* log, int log_cap,
                                        uint64_t* commit, hipStream_t stream);
hipError_t launch_kv_restore(const void* store, size_t store_bytes, const uint64_t* commit,
                             const uint64_t* seq, const uint64_t* src, const uint64_t* dst,
                             const uint32_t* bytes, int n, void* kv, size_t kv_bytes,
                             uint8_t* status, hipStream_t stream);

}  // namespace tg
