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
 *     no state between calls.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = default stream)
 *     and is asynchronous: no call synchronises with the host. Data-dependent
 *     sizes (per-slot counts) stay on the device.
 *   - Arguments are validated on the host before anything is enqueued; a
 *     rejected call enqueues nothing and returns a TG_ERR_* code, with
 *     detail in tg_last_error(). A failed launch returns TG_ERR_HIP.
 *   - Calls are reentrant; concurrent calls must not share output or
 *     workspace buffers.
 *   - Shape limits: 1 <= k <= min(E, 32), E <= 1024, 1 <= S <= 1024,
 *     1 <= R <= 16, d % 256 == 0, I % 128 == 0, T * k < 2^31, and one
 *     slot's weights under 2 GiB (4 * I * d < 2^31 bytes). T may be 0.
 *     Other shapes return TG_ERR_UNSUPPORTED.
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
 * pair_slot, slot_counts, slot_offsets, pair_row, n_unserved. out is
 * required. The workspace holds every intermediate, including the permuted
 * activations, h and y sized for T*k rows.
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

#ifdef __cplusplus
}
#endif

#endif /* TG_H_ */
