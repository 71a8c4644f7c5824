/*
 * tg.h -- C ABI of libtg.so: the expert-worker (EW) forward of Tarragon
 * (arXiv 2601.01310) on one MI355X (gfx950).
 *
 * An MoE layer's gating network picks the top-k experts of each token and
 * the layer output is the gate-weighted sum of those experts' outputs (§2.1).
 * Experts are stateless functions of their input (§2.1), so an expert may be
 * served by any replica holding its weights: the expert routing table (ERT)
 * maps a logical expert to one or more candidate locations, including
 * pre-loaded "shadow" replicas (§4.2, §5.3), and a failed location is masked
 * by rerouting to the next healthy candidate (§5.1). On this EW a location
 * is a physical expert *slot* on the GPU.
 *
 * Conventions for every entry point:
 *   - All tensor pointers are DEVICE pointers to dense row-major arrays.
 *     bf16 values travel as uint16_t bit patterns.
 *   - The caller owns every buffer; the library allocates nothing and keeps
 *     no state between calls. (The exceptions: tg_ew_forward_noalloc takes
 *     its workspace from a scratch area the library holds per GPU, and
 *     tg_set_gemm_tile_policy sets a process-wide measurement knob.)
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = default stream)
 *     and is asynchronous: no call synchronises with the host. Data-dependent
 *     sizes (per-slot counts) stay on the device.
 *   - Arguments are validated on the host before anything is enqueued; a
 *     rejected call enqueues nothing and returns a TG_ERR_* code, with
 *     detail in tg_last_error(). A failed launch returns TG_ERR_HIP.
 *   - Calls are reentrant; concurrent calls must not share output or
 *     workspace buffers.
 *   - Shape limits: 1 <= k <= min(E, 32), E <= 1024, 1 <= S <= 1024,
 *     1 <= R <= 16, d and I multiples of 64 and at least 128,
 *     T * k < 2^31, and one slot's weights under 2 GiB
 *     (4 * I * d < 2^31 bytes). T may be 0. Other shapes return
 *     TG_ERR_UNSUPPORTED.
 */
#ifndef TG_H_
#define TG_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TG_OK = 0,
  TG_ERR_NULL_ARG = 1,    /* a required pointer is NULL */
  TG_ERR_BAD_DIM = 2,     /* a size is negative/zero where it must be positive, or k > E */
  TG_ERR_UNSUPPORTED = 3, /* valid but outside the shape limits above */
  TG_ERR_WORKSPACE = 4,   /* workspace pointer NULL or smaller than required */
  TG_ERR_HIP = 5          /* the HIP runtime reported an error (see tg_last_error) */
} tg_status;

/* Name of a status code (static string). */
const char* tg_status_string(tg_status s);

/* Detail of the calling thread's last failed call ("" if none). */
const char* tg_last_error(void);

/*
 * Gating (§2.1): logits, top-k experts and renormalised gate weights.
 *
 * Either x [T,d] bf16 and w_gate [E,d] bf16 are given (logits_in NULL), and
 * logit l[t,e] = sum_i x[t,i]*w_gate[e,i] is accumulated in float64 and
 * rounded once to float32; or logits_in [T,E] float32 is given (x, w_gate
 * NULL). topk_ids[t, 0..k-1] are the k largest float32 logits, larger first,
 * equal logits ordered by lower expert id. topk_w[t,j] =
 * exp(l_j - l_0) / sum_{j'<k} exp(l_j' - l_0) in float32, which equals the
 * softmax over all E renormalised over the chosen k. logits_out [T,E] is
 * written when non-NULL. Logits must be finite.
 */
tg_status tg_gate_topk(const uint16_t* x, const uint16_t* w_gate, const float* logits_in,
                       int T, int d, int E, int k,
                       float* logits_out, int32_t* topk_ids, float* topk_w,
                       void* stream);

/*
 * ERT remap with failure mask, per-slot batching and dispatch (§4.2, §5.1,
 * §5.3; the EW batches the tokens of each expert, §2.2.1).
 *
 * ert [E,R] int32 lists candidate slots of each logical expert in priority
 * order (primary first); entries outside [0,S) are ignored (-1 = none).
 * slot_alive [S] uint8 (0 = failed). Outputs:
 *   pair_slot [T,k]   first live candidate of topk_ids[t,j], or -1;
 *   n_unserved [1]    pairs whose expert has a valid local candidate but
 *                     none alive (to be replayed elsewhere);
 *   slot_counts [S], slot_offsets [S+1]  per-slot pair counts and their
 *                     exclusive prefix sum; P = slot_offsets[S];
 *   perm [T*k]        rows 0..P-1: flat pair index t*k+j in (slot, token,
 *                     rank) order; rows >= P are not written;
 *   pair_row [T,k]    row of pair (t,j) in that order, or -1;
 *   x_perm [T*k, d]   rows 0..P-1: x[perm[r] / k] (bf16); may be NULL to
 *                     skip the gather.
 * x may be NULL iff x_perm is NULL. ws must hold
 * tg_remap_dispatch_workspace(T,k,S) bytes (256-byte aligned).
 */
size_t tg_remap_dispatch_workspace(int T, int k, int S);
tg_status tg_remap_dispatch(const int32_t* topk_ids, int T, int k,
                            const int32_t* ert, int E, int R,
                            const uint8_t* slot_alive, int S,
                            const uint16_t* x, int d,
                            int32_t* pair_slot, int32_t* slot_counts, int32_t* slot_offsets,
                            int32_t* perm, int32_t* pair_row, uint16_t* x_perm,
                            int32_t* n_unserved, void* ws, size_t ws_bytes, void* stream);

/*
 * Grouped SwiGLU expert FFN over per-slot row groups (the stateless expert
 * of §2.1; SwiGLU form, no biases).
 *
 * Rows slot_offsets[s] .. slot_offsets[s+1]-1 of x_perm [max_rows, d] bf16
 * belong to slot s (slot_offsets is a device array, P = slot_offsets[S] <=
 * max_rows). For each such row x:
 *   g = x W1_s^T, u = x W3_s^T (float32 accumulation),
 *   h = bf16(silu(g) * u)      -> h [max_rows, I]
 *   y = bf16(h W2_s^T)         -> y [max_rows, d] (float32 accumulation)
 * w13 [S, 2I, d] bf16 holds W1_s (rows 0..I-1) and W3_s (rows I..2I-1);
 * w2 [S, d, I] bf16. Rows >= P of h and y are not written. A row's result
 * does not depend on its position or on the other rows.
 */
tg_status tg_expert_ffn_grouped(const uint16_t* x_perm, const int32_t* slot_offsets, int S,
                                int max_rows, const uint16_t* w13, const uint16_t* w2,
                                int d, int I, uint16_t* h, uint16_t* y, void* stream);

/*
 * Tile height of the grouped expert GEMMs (the FFN of §2.1, in
 * tg_expert_ffn_grouped, tg_ew_forward and tg_ew_replay), for measurements
 * and tests; not needed in normal use.
 *
 *   TG_TILES_AUTO  (default) each GEMM launch chooses on the device from
 *                  the slot counts: 32-row tiles for batches whose slots
 *                  hold few rows (decode steps, a single small expert
 *                  batch), 256-row tiles otherwise;
 *   TG_TILES_SMALL every tile 32 rows;
 *   TG_TILES_FULL  every tile 256 rows (partial last rounds of the down
 *                  projection still split into 128 x 128 quarters).
 *
 * Every choice gives identical bits. The setting is process-wide and read
 * when a launch is enqueued. Returns TG_ERR_BAD_DIM for any other value.
 */
#define TG_TILES_AUTO 0
#define TG_TILES_SMALL 1
#define TG_TILES_FULL 2
tg_status tg_set_gemm_tile_policy(int policy);

/*
 * Gate-weighted combine (§2.1): out[t] = bf16(sum_j topk_w[t,j] * y[pair_row[t,j]])
 * over j = 0..k-1 with pair_row >= 0, float32, in rank order; a token with
 * no routed pair gets +0. On one expert-parallel share this is the share's
 * partial sum with the global weights.
 */
tg_status tg_combine(const uint16_t* y, const int32_t* pair_row, const float* topk_w,
                     int T, int k, int d, uint16_t* out, void* stream);

/*
 * The whole EW forward: gating -> remap/dispatch -> grouped FFN -> combine,
 * enqueued on one stream with no host synchronisation.
 *
 * Gating input is either (x, w_gate) or logits_in (see tg_gate_topk).
 * Optional outputs (NULL = kept in the workspace only): topk_ids, topk_w,
 * pair_slot, slot_counts, slot_offsets, pair_row, n_unserved, and y, the
 * per-pair expert outputs [T*k, d] bf16 in pair_row order (keep topk_ids,
 * topk_w, pair_slot, pair_row and y to replay failed pairs later with
 * tg_ew_replay). out is required. The workspace holds every other
 * intermediate (h, and y when not given, sized for T*k rows).
 *
 * token_valid [T] uint8 (optional): the EW-side partial batch (§5.2). Tokens
 * with 0 are not part of this batch: their pairs get pair_slot -2 and
 * pair_row -1, are not counted in n_unserved, and their out rows are +0.
 * The other tokens' results do not depend on the mask.
 */
typedef struct {
  int T, d, E, k, I, S, R;
  const uint16_t* x;          /* [T,d] bf16, required */
  const uint16_t* w_gate;     /* [E,d] bf16, or NULL with logits_in */
  const float* logits_in;     /* [T,E] float32, or NULL with w_gate */
  const int32_t* ert;         /* [E,R] */
  const uint8_t* slot_alive;  /* [S] */
  const uint16_t* w13;        /* [S,2I,d] bf16 */
  const uint16_t* w2;         /* [S,d,I] bf16 */
  uint16_t* out;              /* [T,d] bf16, required */
  int32_t* topk_ids;          /* [T,k] or NULL */
  float* topk_w;              /* [T,k] or NULL */
  int32_t* pair_slot;         /* [T,k] or NULL */
  int32_t* slot_counts;       /* [S] or NULL */
  int32_t* slot_offsets;      /* [S+1] or NULL */
  int32_t* pair_row;          /* [T,k] or NULL */
  int32_t* n_unserved;        /* [1] or NULL */
  uint16_t* y;                /* [T*k,d] bf16 or NULL */
  const uint8_t* token_valid; /* [T] or NULL (all tokens in the batch) */
} tg_ew_args;

size_t tg_ew_forward_workspace(const tg_ew_args* a);
tg_status tg_ew_forward(const tg_ew_args* a, void* ws, size_t ws_bytes, void* stream);

/*
 * tg_ew_forward with per-stage timing marks: events[0..5] (hipEvent_t
 * handles created by the caller; n_events must be 6) are recorded on
 * `stream` before gating, before remap/dispatch, before the gate/up GEMM,
 * before the down GEMM, before the combine, and after the combine. The
 * computation is identical to tg_ew_forward.
 */
tg_status tg_ew_forward_timed(const tg_ew_args* a, void* ws, size_t ws_bytes, void* stream,
                              void* const* events, int n_events);

/*
 * tg_ew_forward without a caller workspace, for callers that cannot
 * allocate device memory: code under HIP graph capture, serving loops and
 * harnesses that must not call the allocator. It computes what tg_ew_forward
 * computes, with the same kernels in the same order, and allocates nothing:
 * its workspace is a scratch area of TG_NOALLOC_SCRATCH_BYTES that the
 * library holds on each GPU it runs on, until the process ends.
 *
 * A batch whose tg_ew_forward_workspace(a) exceeds TG_NOALLOC_SCRATCH_BYTES
 * is rejected with TG_ERR_WORKSPACE before anything is enqueued (a caller
 * buffer in a->y keeps the per-pair outputs out of the scratch area; 64 MiB
 * covers, e.g., a decode step of 432 tokens at DeepSeek-V3 expert shapes).
 * The first call on a device resolves that device's scratch address, which
 * may load the library's device code there: make it outside graph capture.
 * All calls on one GPU share its scratch area, which keeps the last call's
 * contents (nothing in it has to start at zero): calls that may overlap on
 * one GPU (streams with no ordering between them, concurrent host threads)
 * race and must be serialised by the caller.
 */
#define TG_NOALLOC_SCRATCH_BYTES (64u * 1024u * 1024u)
tg_status tg_ew_forward_noalloc(const tg_ew_args* a, void* stream);

/*
 * Replay of failed pairs (§5.1): after a forward, slots may fail (or be
 * restored) before its result is used. Experts are stateless and
 * deterministic, so a pair whose slot has failed is recomputed on the next
 * live candidate of its expert from the same token row and merged into the
 * output, without recomputing anything else.
 *
 * Inputs are the first pass's x, topk_ids, topk_w, pair_slot, pair_row and
 * y (tg_ew_args fields), the ERT, the weights and the CURRENT slot_alive.
 * A pair is replayed when its first-pass slot is no longer alive, or when it
 * had no live local candidate, and its expert now has one; it is computed on
 * the first live candidate. A pair whose first-pass slot failed and that has
 * no live candidate left is dropped (the remaining weights are not
 * renormalised). Every token with a replayed or dropped pair gets its out
 * row re-formed (same float32 rank-order sum as tg_combine); other rows of
 * out are not touched. When every candidate slot of an expert holds the same
 * weights, out afterwards equals, bit for bit, what tg_ew_forward gives with
 * the current slot_alive.
 *
 * Outputs: out [T,d] (in/out), and optionally replay_slot [T,k] (slot of
 * each replayed pair, else -1), n_replayed [1], n_unserved [1] (pairs whose
 * expert has local candidates, none alive now; as tg_ew_forward counts
 * them). Pairs with pair_slot -2 (outside the batch) are never replayed.
 */
typedef struct {
  int T, d, E, k, I, S, R;
  const uint16_t* x;          /* [T,d] bf16, the first pass's token rows */
  const int32_t* ert;         /* [E,R] */
  const uint8_t* slot_alive;  /* [S], current */
  const uint16_t* w13;        /* [S,2I,d] bf16 */
  const uint16_t* w2;         /* [S,d,I] bf16 */
  const int32_t* topk_ids;    /* [T,k], first pass */
  const float* topk_w;        /* [T,k], first pass */
  const int32_t* pair_slot;   /* [T,k], first pass */
  const int32_t* pair_row;    /* [T,k], first pass */
  const uint16_t* y;          /* [T*k,d] bf16, first pass */
  uint16_t* out;              /* [T,d] bf16, in/out */
  int32_t* replay_slot;       /* [T,k] or NULL */
  int32_t* n_replayed;        /* [1] or NULL */
  int32_t* n_unserved;        /* [1] or NULL */
} tg_replay_args;

size_t tg_ew_replay_workspace(const tg_replay_args* a);
tg_status tg_ew_replay(const tg_replay_args* a, void* ws, size_t ws_bytes, void* stream);

/*
 * EW-side partial-batch trigger (§5.2): start the layer's expert work once
 * a sufficient subset of attention workers (AWs) has delivered its tokens.
 *
 * The batch buffer x [T,d] holds the rows of A AWs as chunks: AW a's rows
 * are chunk_rows[a] .. chunk_rows[a+1]-1 (chunk_rows [A+1] int32, device,
 * non-decreasing; rows outside [0,T) are ignored, rows in no chunk are never
 * in the batch). delivered [A] uint32 is nonzero once AW a's chunk has
 * arrived; it may be device memory or host-visible memory that the
 * transport writes while the trigger waits (read with system-scope loads).
 * aw_alive [A] uint8 is 0 for AWs known to have failed.
 *
 * One kernel on `stream` polls delivered[] until (i) every AW with
 * aw_alive[a] != 0 has delivered, or (ii) the rows of the live AWs that
 * have delivered reach min_rows, or (iii) spin_limit polls (each followed by
 * a short sleep, about 4 us) have passed: the probing window, after which
 * live AWs that have not delivered are left out of this batch (treated as
 * failed for this layer). It then writes token_valid [T] (1 for the rows of
 * live AWs that had delivered at the deciding poll, else 0), ready to pass
 * as tg_ew_args.token_valid to a forward enqueued after it, and status [4]
 * int32 = {condition met (0, 1 or 2 for i, ii, iii), rows in the batch,
 * AWs in the batch, polls made}. The kernel always ends after at most
 * spin_limit polls. Limits: 1 <= A <= 1024, spin_limit >= 1.
 */
tg_status tg_batch_trigger(const uint32_t* delivered, const uint8_t* aw_alive,
                           const int32_t* chunk_rows, int A, int T, int min_rows,
                           long long spin_limit, uint8_t* token_valid, int32_t* status,
                           void* stream);

/*
 * Incremental KV-segment checkpoint (§6.1) and request-level restoration
 * (§6.2), on one GPU: host-visible memory (pinned host memory, or any
 * memory the GPU can write) plays the checkpoint store.
 *
 * The store has the KV region's layout: a segment at byte offset o of the
 * KV region is stored at byte offset o of the store (both buffers
 * kv_bytes long and 16-byte aligned). tg_kv_checkpoint copies n segments
 * (seg_offset [n] uint64 byte offsets, seg_bytes [n] uint32 lengths, device
 * arrays; both multiples of 16 and inside the region) from the device KV
 * region to the store, tags segment i with sequence number first_seq + i,
 * writes its record {seq, offset, bytes} to log[seq % log_cap] (bytes 0 when
 * the segment was rejected as misaligned or out of range; the log is a ring,
 * so it keeps the last log_cap records), and, once every
 * copy and record has landed, stores first_seq + n into *commit (the
 * "log + commit record" of §6.1: every sequence number below the commit
 * record has landed; 0 = nothing committed; commit may be NULL to leave the
 * batch uncommitted). Calls on one stream commit in order; the caller gives
 * consecutive, increasing sequence numbers across calls. The copy runs on
 * at most max_blocks workgroups (0 = 16), so that it can proceed on a
 * second stream beside the caller's compute (the gaps of §6.1) while taking
 * few CUs from it.
 *
 * tg_kv_restore copies n committed segments from the store back into a
 * device KV region (src [n] store offsets, dst [n] offsets in kv_dst, bytes
 * [n], seq [n] their sequence numbers): a segment whose seq is not below
 * the commit record read at the start of the kernel is skipped. status [n]
 * uint8: 1 restored, 0 not committed, 2 misaligned or out of range.
 */
typedef struct {
  uint64_t seq;
  uint64_t offset;
  uint64_t bytes;
} tg_ckpt_record;

tg_status tg_kv_checkpoint(const void* kv, size_t kv_bytes, const uint64_t* seg_offset,
                           const uint32_t* seg_bytes, int n, uint64_t first_seq, void* store,
                           tg_ckpt_record* log, int log_cap, uint64_t* commit, int max_blocks,
                           void* stream);
/*
 * tg_kv_checkpoint for n segments at a constant stride: segment i is at
 * byte offset first_offset + i * pitch and is seg_bytes long (one decode
 * step of a [layer][request][position][segment] region is such a batch).
 * The bytes move by one strided copy on the GPU's copy engine, so no
 * compute unit is taken from concurrent work; the records and the commit
 * record follow in one small kernel, after the copy in stream order.
 * Offsets, pitch and seg_bytes must be multiples of 16 with seg_bytes <=
 * pitch, and the batch must lie inside the region (checked on the host:
 * TG_ERR_BAD_DIM otherwise).
 */
tg_status tg_kv_checkpoint_strided(const void* kv, size_t kv_bytes, uint64_t first_offset,
                                   uint64_t pitch, uint32_t seg_bytes, int n, uint64_t first_seq,
                                   void* store, tg_ckpt_record* log, int log_cap,
                                   uint64_t* commit, void* stream);
tg_status tg_kv_restore(const void* store, size_t store_bytes, const uint64_t* commit,
                        const uint64_t* seq, const uint64_t* src, const uint64_t* dst,
                        const uint32_t* bytes, int n, void* kv_dst, size_t kv_bytes,
                        uint8_t* status, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TG_H_ */
