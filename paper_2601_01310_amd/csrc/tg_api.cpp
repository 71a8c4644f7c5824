// C ABI of libtg.so: argument validation, workspace layout and launch order.
// Nothing here computes on the data; every step runs in the HIP kernels.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <string>

#include "tg.h"
#include "tg_launch.h"

namespace {

thread_local std::string g_last_error;

tg_status vfail(tg_status s, const char* fmt, va_list ap) {
  char buf[512];
  vsnprintf(buf, sizeof(buf), fmt, ap);
  g_last_error = buf;
  return s;
}

tg_status fail(tg_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vfail(s, fmt, ap);
  va_end(ap);
  return s;
}

tg_status ok() {
  g_last_error.clear();
  return TG_OK;
}

tg_status hip_status(hipError_t e, const char* where) {
  if (e != hipSuccess) return fail(TG_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
  return ok();
}

constexpr int kMaxK = 32, kMaxE = 1024, kMaxS = 1024, kMaxR = 16, kMaxAws = 1024;

tg_status check_gate_dims(int T, int E, int k) {
  if (T < 0) return fail(TG_ERR_BAD_DIM, "T=%d must be >= 0", T);
  if (E <= 0 || k <= 0) return fail(TG_ERR_BAD_DIM, "E=%d and k=%d must be > 0", E, k);
  if (k > E) return fail(TG_ERR_BAD_DIM, "k=%d exceeds E=%d", k, E);
  if (k > kMaxK) return fail(TG_ERR_UNSUPPORTED, "k=%d exceeds %d", k, kMaxK);
  if (E > kMaxE) return fail(TG_ERR_UNSUPPORTED, "E=%d exceeds %d", E, kMaxE);
  if ((long long)T * k >= (1LL << 31)) return fail(TG_ERR_UNSUPPORTED, "T*k >= 2^31");
  return TG_OK;
}

// Hidden and intermediate sizes: multiples of 64 (the GEMMs' K stage), at
// least 128 (two K stages).
tg_status check_hidden(int d, const char* name) {
  if (d <= 0) return fail(TG_ERR_BAD_DIM, "%s=%d must be > 0", name, d);
  if (d % 64 || d < 128)
    return fail(TG_ERR_UNSUPPORTED, "%s=%d is not a multiple of 64 of at least 128", name, d);
  return TG_OK;
}

tg_status check_inter(int I) {
  if (I <= 0) return fail(TG_ERR_BAD_DIM, "I=%d must be > 0", I);
  if (I % 64 || I < 128)
    return fail(TG_ERR_UNSUPPORTED, "I=%d is not a multiple of 64 of at least 128", I);
  return TG_OK;
}

// One slot's gate/up weights are addressed with 32-bit byte offsets.
tg_status check_ffn(int d, int I) {
  tg_status st = check_hidden(d, "d");
  if (st != TG_OK) return st;
  if ((st = check_inter(I)) != TG_OK) return st;
  if (4LL * I * d >= (1LL << 31))
    return fail(TG_ERR_UNSUPPORTED, "one slot's weights (4*I*d = %lld bytes) reach 2 GiB",
                4LL * I * d);
  return TG_OK;
}

tg_status check_slots(int S, int R) {
  if (S <= 0 || R <= 0) return fail(TG_ERR_BAD_DIM, "S=%d and R=%d must be > 0", S, R);
  if (S > kMaxS) return fail(TG_ERR_UNSUPPORTED, "S=%d exceeds %d", S, kMaxS);
  if (R > kMaxR) return fail(TG_ERR_UNSUPPORTED, "R=%d exceeds %d", R, kMaxR);
  return TG_OK;
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// Carves the tg_ew_forward workspace; with base == nullptr only sizes it.
struct EwLayout {
  int32_t* ids;
  float* w;
  int32_t* pair_slot;
  int32_t* counts;
  int32_t* offsets;
  int32_t* pair_row;
  int32_t* n_unserved;
  int32_t* perm;
  void* dispatch_ws;
  uint16_t* x_perm;
  uint16_t* h;
  uint16_t* y;
  void* sched;
  size_t bytes;
};

EwLayout ew_layout(const tg_ew_args* a, char* base) {
  EwLayout L{};
  size_t off = 0;
  const size_t np = (size_t)a->T * a->k;
  auto take = [&](size_t bytes) -> char* {
    char* p = base ? base + off : nullptr;
    off += align256(bytes);
    return p;
  };
  L.ids = reinterpret_cast<int32_t*>(take(np * 4));
  L.w = reinterpret_cast<float*>(take(np * 4));
  L.pair_slot = reinterpret_cast<int32_t*>(take(np * 4));
  L.counts = reinterpret_cast<int32_t*>(take((size_t)a->S * 4));
  L.offsets = reinterpret_cast<int32_t*>(take(((size_t)a->S + 1) * 4));
  L.pair_row = reinterpret_cast<int32_t*>(take(np * 4));
  L.n_unserved = reinterpret_cast<int32_t*>(take(4));
  L.perm = reinterpret_cast<int32_t*>(take(np * 4));
  L.dispatch_ws = take(tg::dispatch_workspace_bytes(a->T, a->k, a->S));
  // The permuted copy of x is only needed when x is too large to be read in
  // place (see tg_ew_forward).
  const bool in_place = 2LL * a->T * a->d < (1LL << 31);
  L.x_perm = reinterpret_cast<uint16_t*>(take(in_place ? 0 : np * a->d * 2));
  L.h = reinterpret_cast<uint16_t*>(take(np * a->I * 2));
  L.y = reinterpret_cast<uint16_t*>(take(a->y ? 0 : np * a->d * 2));
  if (a->y) L.y = a->y;
  L.sched = take(tg::kSchedBytes);
  L.bytes = off;
  return L;
}

// Carves the tg_ew_replay workspace; with base == nullptr only sizes it.
struct ReplayLayout {
  int32_t* replay_slot;
  int32_t* counts;
  int32_t* offsets;
  int32_t* replay_row;
  int32_t* perm;
  int32_t* n_replayed;
  int32_t* n_unserved;
  void* dispatch_ws;
  uint16_t* x_perm;
  uint16_t* h;
  uint16_t* y2;
  void* sched;
  size_t bytes;
};

ReplayLayout replay_layout(const tg_replay_args* a, char* base) {
  ReplayLayout L{};
  size_t off = 0;
  const size_t np = (size_t)a->T * a->k;
  auto take = [&](size_t bytes) -> char* {
    char* p = base ? base + off : nullptr;
    off += align256(bytes);
    return p;
  };
  L.replay_slot = reinterpret_cast<int32_t*>(take(np * 4));
  L.counts = reinterpret_cast<int32_t*>(take((size_t)a->S * 4));
  L.offsets = reinterpret_cast<int32_t*>(take(((size_t)a->S + 1) * 4));
  L.replay_row = reinterpret_cast<int32_t*>(take(np * 4));
  L.perm = reinterpret_cast<int32_t*>(take(np * 4));
  L.n_replayed = reinterpret_cast<int32_t*>(take(4));
  L.n_unserved = reinterpret_cast<int32_t*>(take(4));
  L.dispatch_ws = take(tg::dispatch_workspace_bytes(a->T, a->k, a->S));
  const bool in_place = 2LL * a->T * a->d < (1LL << 31);
  L.x_perm = reinterpret_cast<uint16_t*>(take(in_place ? 0 : np * a->d * 2));
  L.h = reinterpret_cast<uint16_t*>(take(np * a->I * 2));
  L.y2 = reinterpret_cast<uint16_t*>(take(np * a->d * 2));
  L.sched = take(tg::kSchedBytes);
  L.bytes = off;
  return L;
}

tg_status check_ew(const tg_ew_args* a) {
  if (!a) return fail(TG_ERR_NULL_ARG, "args is NULL");
  tg_status st = check_gate_dims(a->T, a->E, a->k);
  if (st != TG_OK) return st;
  if ((st = check_ffn(a->d, a->I)) != TG_OK) return st;
  if ((st = check_slots(a->S, a->R)) != TG_OK) return st;
  if (!a->x || !a->ert || !a->slot_alive || !a->w13 || !a->w2 || !a->out)
    return fail(TG_ERR_NULL_ARG, "a required pointer is NULL");
  if ((a->w_gate == nullptr) == (a->logits_in == nullptr))
    return fail(TG_ERR_NULL_ARG, "give exactly one of w_gate and logits_in");
  return TG_OK;
}

}  // namespace

namespace tg {

tg_status ew_forward(const tg_ew_args* a, void* ws, size_t ws_bytes, void* stream,
                     void* const* events) {
  tg_status st = check_ew(a);
  if (st != TG_OK) return st;
  const size_t need = ew_layout(a, nullptr).bytes;
  if (!ws || ws_bytes < need)
    return fail(TG_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  if (reinterpret_cast<uintptr_t>(ws) & 255)
    return fail(TG_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  EwLayout L = ew_layout(a, static_cast<char*>(ws));
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* ids = a->topk_ids ? a->topk_ids : L.ids;
  float* w = a->topk_w ? a->topk_w : L.w;
  int32_t* pair_slot = a->pair_slot ? a->pair_slot : L.pair_slot;
  int32_t* counts = a->slot_counts ? a->slot_counts : L.counts;
  int32_t* offsets = a->slot_offsets ? a->slot_offsets : L.offsets;
  int32_t* pair_row = a->pair_row ? a->pair_row : L.pair_row;
  int32_t* n_unserved = a->n_unserved ? a->n_unserved : L.n_unserved;
  const int max_rows = a->T * a->k;
  hipError_t e = hipSuccess;
  auto mark = [&](int i) {
    if (events && e == hipSuccess) e = hipEventRecord(static_cast<hipEvent_t>(events[i]), s);
  };
  mark(0);
  if (e == hipSuccess)
    e = tg::launch_gate_topk(a->w_gate ? a->x : nullptr, a->w_gate, a->logits_in, a->T, a->d, a->E,
                             a->k, nullptr, ids, w, s);
  mark(1);
  // The gate/up GEMM reads the token rows in place through perm when x is
  // addressable with 32-bit byte offsets; otherwise they are gathered first.
  const bool in_place = 2LL * a->T * a->d < (1LL << 31);
  if (e == hipSuccess)
    e = tg::launch_remap_dispatch(ids, a->T, a->k, a->ert, a->E, a->R, a->slot_alive, a->S,
                                  in_place ? nullptr : a->x, a->d, pair_slot, counts, offsets,
                                  L.perm, pair_row, in_place ? nullptr : L.x_perm, n_unserved,
                                  L.dispatch_ws, s, a->token_valid, L.sched);
  mark(2);
  // The dispatch has zeroed the GEMMs' dynamic-schedule area.
  tg::GemmSched sched_gu, sched_dn;
  tg::sched_carve(L.sched, &sched_gu, &sched_dn);
  if (e == hipSuccess)
    e = in_place ? tg::launch_ffn_gateup_gather(a->x, a->T, L.perm, a->k, offsets, a->S, max_rows,
                                                a->w13, a->d, a->I, L.h, s, &sched_gu)
                 : tg::launch_ffn_gateup(L.x_perm, offsets, a->S, max_rows, a->w13, a->d, a->I,
                                         L.h, s, &sched_gu);
  mark(3);
  if (e == hipSuccess)
    e = tg::launch_ffn_down(L.h, offsets, a->S, max_rows, a->w2, a->d, a->I, L.y, s, &sched_dn);
  mark(4);
  if (e == hipSuccess) e = tg::launch_combine(L.y, pair_row, w, a->T, a->k, a->d, a->out, s);
  mark(5);
  return hip_status(e, "tg_ew_forward");
}

tg_status ew_check(const tg_ew_args* a, size_t* ws_bytes) {
  const tg_status st = check_ew(a);
  if (st == TG_OK) *ws_bytes = ew_layout(a, nullptr).bytes;
  return st;
}

tg_status set_error(tg_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vfail(s, fmt, ap);
  va_end(ap);
  return s;
}

}  // namespace tg

extern "C" {

const char* tg_status_string(tg_status s) {
  switch (s) {
    case TG_OK: return "TG_OK";
    case TG_ERR_NULL_ARG: return "TG_ERR_NULL_ARG";
    case TG_ERR_BAD_DIM: return "TG_ERR_BAD_DIM";
    case TG_ERR_UNSUPPORTED: return "TG_ERR_UNSUPPORTED";
    case TG_ERR_WORKSPACE: return "TG_ERR_WORKSPACE";
    case TG_ERR_HIP: return "TG_ERR_HIP";
  }
  return "TG_ERR_UNKNOWN";
}

const char* tg_last_error(void) { return g_last_error.c_str(); }

tg_status tg_gate_topk(const uint16_t* x, const uint16_t* w_gate, const float* logits_in, int T,
                       int d, int E, int k, float* logits_out, int32_t* topk_ids, float* topk_w,
                       void* stream) {
  tg_status st = check_gate_dims(T, E, k);
  if (st != TG_OK) return st;
  const bool weights_mode = (x != nullptr || w_gate != nullptr);
  if (weights_mode) {
    if (!x || !w_gate || logits_in)
      return fail(TG_ERR_NULL_ARG, "give either x and w_gate, or logits_in");
    if ((st = check_hidden(d, "d")) != TG_OK) return st;
  } else if (!logits_in) {
    return fail(TG_ERR_NULL_ARG, "give either x and w_gate, or logits_in");
  }
  if (!topk_ids || !topk_w) return fail(TG_ERR_NULL_ARG, "topk_ids and topk_w are required");
  return hip_status(tg::launch_gate_topk(x, w_gate, logits_in, T, d, E, k,
                                         weights_mode ? logits_out : nullptr, topk_ids, topk_w,
                                         static_cast<hipStream_t>(stream)),
                    "tg_gate_topk");
}

size_t tg_remap_dispatch_workspace(int T, int k, int S) {
  if (T < 0 || k <= 0 || S <= 0) return 0;
  return tg::dispatch_workspace_bytes(T, k, S);
}

tg_status tg_remap_dispatch(const int32_t* topk_ids, int T, int k, const int32_t* ert, int E,
                            int R, const uint8_t* slot_alive, int S, const uint16_t* x, int d,
                            int32_t* pair_slot, int32_t* slot_counts, int32_t* slot_offsets,
                            int32_t* perm, int32_t* pair_row, uint16_t* x_perm,
                            int32_t* n_unserved, void* ws, size_t ws_bytes, void* stream) {
  tg_status st = check_gate_dims(T, E, k);
  if (st != TG_OK) return st;
  if ((st = check_slots(S, R)) != TG_OK) return st;
  if (!topk_ids || !ert || !slot_alive || !pair_slot || !slot_counts || !slot_offsets || !perm ||
      !pair_row || !n_unserved)
    return fail(TG_ERR_NULL_ARG, "a required pointer is NULL");
  if ((x == nullptr) != (x_perm == nullptr))
    return fail(TG_ERR_NULL_ARG, "x and x_perm must both be given or both be NULL");
  if (x_perm && (st = check_hidden(d, "d")) != TG_OK) return st;
  const size_t need = tg::dispatch_workspace_bytes(T, k, S);
  if (!ws || ws_bytes < need)
    return fail(TG_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  if (reinterpret_cast<uintptr_t>(ws) & 255)
    return fail(TG_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return hip_status(tg::launch_remap_dispatch(topk_ids, T, k, ert, E, R, slot_alive, S, x, d,
                                              pair_slot, slot_counts, slot_offsets, perm, pair_row,
                                              x_perm, n_unserved, ws,
                                              static_cast<hipStream_t>(stream)),
                    "tg_remap_dispatch");
}

tg_status tg_expert_ffn_grouped(const uint16_t* x_perm, const int32_t* slot_offsets, int S,
                                int max_rows, const uint16_t* w13, const uint16_t* w2, int d,
                                int I, uint16_t* h, uint16_t* y, void* stream) {
  tg_status st;
  if (S <= 0) return fail(TG_ERR_BAD_DIM, "S=%d must be > 0", S);
  if (S > kMaxS) return fail(TG_ERR_UNSUPPORTED, "S=%d exceeds %d", S, kMaxS);
  if (max_rows < 0) return fail(TG_ERR_BAD_DIM, "max_rows=%d must be >= 0", max_rows);
  if ((st = check_ffn(d, I)) != TG_OK) return st;
  if (!x_perm || !slot_offsets || !w13 || !w2 || !h || !y)
    return fail(TG_ERR_NULL_ARG, "a required pointer is NULL");
  return hip_status(tg::launch_expert_ffn(x_perm, slot_offsets, S, max_rows, w13, w2, d, I, h, y,
                                          static_cast<hipStream_t>(stream)),
                    "tg_expert_ffn_grouped");
}

tg_status tg_set_gemm_tile_policy(int policy) {
  if (policy != TG_TILES_AUTO && policy != TG_TILES_SMALL && policy != TG_TILES_FULL)
    return fail(TG_ERR_BAD_DIM, "tile policy %d is not one of 0, 1, 2", policy);
  tg::set_tile_policy(policy);
  return TG_OK;
}

tg_status tg_combine(const uint16_t* y, const int32_t* pair_row, const float* topk_w, int T, int k,
                     int d, uint16_t* out, void* stream) {
  tg_status st;
  if (T < 0 || k <= 0) return fail(TG_ERR_BAD_DIM, "T=%d >= 0 and k=%d > 0 required", T, k);
  if (k > kMaxK) return fail(TG_ERR_UNSUPPORTED, "k=%d exceeds %d", k, kMaxK);
  if ((st = check_hidden(d, "d")) != TG_OK) return st;
  if (!y || !pair_row || !topk_w || !out) return fail(TG_ERR_NULL_ARG, "a required pointer is NULL");
  return hip_status(
      tg::launch_combine(y, pair_row, topk_w, T, k, d, out, static_cast<hipStream_t>(stream)),
      "tg_combine");
}

size_t tg_ew_forward_workspace(const tg_ew_args* a) {
  if (check_ew(a) != TG_OK) return 0;
  return ew_layout(a, nullptr).bytes;
}

tg_status tg_ew_forward(const tg_ew_args* a, void* ws, size_t ws_bytes, void* stream) {
  return tg::ew_forward(a, ws, ws_bytes, stream, nullptr);
}

tg_status tg_ew_forward_timed(const tg_ew_args* a, void* ws, size_t ws_bytes, void* stream,
                              void* const* events, int n_events) {
  if (!events) return fail(TG_ERR_NULL_ARG, "events is NULL");
  if (n_events != 6) return fail(TG_ERR_BAD_DIM, "n_events=%d, 6 required", n_events);
  for (int i = 0; i < 6; ++i)
    if (!events[i]) return fail(TG_ERR_NULL_ARG, "events[%d] is NULL", i);
  return tg::ew_forward(a, ws, ws_bytes, stream, events);
}

static tg_status check_replay(const tg_replay_args* a) {
  if (!a) return fail(TG_ERR_NULL_ARG, "args is NULL");
  tg_status st = check_gate_dims(a->T, a->E, a->k);
  if (st != TG_OK) return st;
  if ((st = check_ffn(a->d, a->I)) != TG_OK) return st;
  if ((st = check_slots(a->S, a->R)) != TG_OK) return st;
  if (!a->x || !a->ert || !a->slot_alive || !a->w13 || !a->w2 || !a->topk_ids || !a->topk_w ||
      !a->pair_slot || !a->pair_row || !a->y || !a->out)
    return fail(TG_ERR_NULL_ARG, "a required pointer is NULL");
  return TG_OK;
}

size_t tg_ew_replay_workspace(const tg_replay_args* a) {
  if (check_replay(a) != TG_OK) return 0;
  return replay_layout(a, nullptr).bytes;
}

tg_status tg_ew_replay(const tg_replay_args* a, void* ws, size_t ws_bytes, void* stream) {
  tg_status st = check_replay(a);
  if (st != TG_OK) return st;
  const size_t need = replay_layout(a, nullptr).bytes;
  if (!ws || ws_bytes < need)
    return fail(TG_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  if (reinterpret_cast<uintptr_t>(ws) & 255)
    return fail(TG_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  ReplayLayout L = replay_layout(a, static_cast<char*>(ws));
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* replay_slot = a->replay_slot ? a->replay_slot : L.replay_slot;
  int32_t* n_replayed = a->n_replayed ? a->n_replayed : L.n_replayed;
  int32_t* n_unserved = a->n_unserved ? a->n_unserved : L.n_unserved;
  const int max_rows = a->T * a->k;
  const bool in_place = 2LL * a->T * a->d < (1LL << 31);
  hipError_t e = tg::launch_replay_dispatch(
      a->topk_ids, a->T, a->k, a->ert, a->E, a->R, a->slot_alive, a->S, a->pair_slot,
      in_place ? nullptr : a->x, a->d, replay_slot, L.counts, L.offsets, L.perm, L.replay_row,
      in_place ? nullptr : L.x_perm, n_unserved, n_replayed, L.dispatch_ws, s, L.sched);
  tg::GemmSched sched_gu, sched_dn;
  tg::sched_carve(L.sched, &sched_gu, &sched_dn);
  if (e == hipSuccess)
    e = in_place ? tg::launch_ffn_gateup_gather(a->x, a->T, L.perm, a->k, L.offsets, a->S,
                                                max_rows, a->w13, a->d, a->I, L.h, s, &sched_gu)
                 : tg::launch_ffn_gateup(L.x_perm, L.offsets, a->S, max_rows, a->w13, a->d, a->I,
                                         L.h, s, &sched_gu);
  if (e == hipSuccess)
    e = tg::launch_ffn_down(L.h, L.offsets, a->S, max_rows, a->w2, a->d, a->I, L.y2, s,
                            &sched_dn);
  if (e == hipSuccess)
    e = tg::launch_recombine(a->y, a->pair_row, a->pair_slot, a->slot_alive, a->S, L.y2,
                             L.replay_row, a->topk_w, a->T, a->k, a->d, a->out, s);
  return hip_status(e, "tg_ew_replay");
}

tg_status tg_batch_trigger(const uint32_t* delivered, const uint8_t* aw_alive,
                           const int32_t* chunk_rows, int A, int T, int min_rows,
                           long long spin_limit, uint8_t* token_valid, int32_t* status,
                           void* stream) {
  if (A <= 0 || T < 0 || min_rows < 0 || spin_limit < 1)
    return fail(TG_ERR_BAD_DIM, "A=%d > 0, T=%d >= 0, min_rows=%d >= 0, spin_limit=%lld >= 1",
                A, T, min_rows, spin_limit);
  if (A > kMaxAws) return fail(TG_ERR_UNSUPPORTED, "A=%d exceeds %d", A, kMaxAws);
  if (!delivered || !aw_alive || !chunk_rows || !status || (T > 0 && !token_valid))
    return fail(TG_ERR_NULL_ARG, "a required pointer is NULL");
  return hip_status(tg::launch_batch_trigger(delivered, aw_alive, chunk_rows, A, T, min_rows,
                                             spin_limit, token_valid, status,
                                             static_cast<hipStream_t>(stream)),
                    "tg_batch_trigger");
}

// Blocks a checkpoint copy occupies by default: enough to keep the host
// link busy while leaving nearly every CU to concurrent compute.
constexpr int kCkptBlocks = 16;

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

tg_status tg_kv_checkpoint(const void* kv, size_t kv_bytes, const uint64_t* seg_offset,
                           const uint32_t* seg_bytes, int n, uint64_t first_seq, void* store,
                           tg_ckpt_record* log, int log_cap, uint64_t* commit, int max_blocks,
                           void* stream) {
  if (n < 0) return fail(TG_ERR_BAD_DIM, "n=%d must be >= 0", n);
  if (max_blocks < 0) return fail(TG_ERR_BAD_DIM, "max_blocks=%d must be >= 0", max_blocks);
  if (n > 0 && log_cap <= 0) return fail(TG_ERR_BAD_DIM, "log_cap=%d must be > 0", log_cap);
  if (!kv || !store || (n > 0 && (!seg_offset || !seg_bytes || !log)))
    return fail(TG_ERR_NULL_ARG, "a required pointer is NULL");
  if (!aligned16(kv) || !aligned16(store) || !aligned16(log))
    return fail(TG_ERR_UNSUPPORTED, "kv, store and log must be 16-byte aligned");
  return hip_status(tg::launch_kv_checkpoint(kv, kv_bytes, seg_offset, seg_bytes, n, first_seq,
                                             store, log, log_cap, commit,
                                             max_blocks ? max_blocks : kCkptBlocks,
                                             static_cast<hipStream_t>(stream)),
                    "tg_kv_checkpoint");
}

tg_status tg_kv_checkpoint_strided(const void* kv, size_t kv_bytes, uint64_t first_offset,
                                   uint64_t pitch, uint32_t seg_bytes, int n, uint64_t first_seq,
                                   void* store, tg_ckpt_record* log, int log_cap,
                                   uint64_t* commit, void* stream) {
  if (n < 0) return fail(TG_ERR_BAD_DIM, "n=%d must be >= 0", n);
  if (n > 0 && log_cap <= 0) return fail(TG_ERR_BAD_DIM, "log_cap=%d must be > 0", log_cap);
  if (!kv || !store || (n > 0 && !log)) return fail(TG_ERR_NULL_ARG, "a required pointer is NULL");
  if (!aligned16(kv) || !aligned16(store) || !aligned16(log))
    return fail(TG_ERR_UNSUPPORTED, "kv, store and log must be 16-byte aligned");
  if (n > 0) {
    if (first_offset % 16 || pitch % 16 || seg_bytes % 16 || seg_bytes == 0 || pitch < seg_bytes)
      return fail(TG_ERR_BAD_DIM, "offsets, pitch and segment size must be multiples of 16, "
                  "with seg_bytes <= pitch");
    const unsigned __int128 end =
        (unsigned __int128)first_offset + (unsigned __int128)(n - 1) * pitch + seg_bytes;
    if (end > kv_bytes)
      return fail(TG_ERR_BAD_DIM, "the last segment ends past the region (%zu bytes)", kv_bytes);
  }
  return hip_status(tg::launch_kv_checkpoint_strided(kv, first_offset, pitch, seg_bytes, n,
                                                     first_seq, store, log, log_cap, commit,
                                                     static_cast<hipStream_t>(stream)),
                    "tg_kv_checkpoint_strided");
}

tg_status tg_kv_restore(const void* store, size_t store_bytes, const uint64_t* commit,
                        const uint64_t* seq, const uint64_t* src, const uint64_t* dst,
                        const uint32_t* bytes, int n, void* kv_dst, size_t kv_bytes,
                        uint8_t* status, void* stream) {
  if (n < 0) return fail(TG_ERR_BAD_DIM, "n=%d must be >= 0", n);
  if (!store || !commit || !kv_dst ||
      (n > 0 && (!seq || !src || !dst || !bytes || !status)))
    return fail(TG_ERR_NULL_ARG, "a required pointer is NULL");
  if (!aligned16(store) || !aligned16(kv_dst))
    return fail(TG_ERR_UNSUPPORTED, "store and kv_dst must be 16-byte aligned");
  return hip_status(tg::launch_kv_restore(store, store_bytes, commit, seq, src, dst, bytes, n,
                                          kv_dst, kv_bytes, status,
                                          static_cast<hipStream_t>(stream)),
                    "tg_kv_restore");
}

}  // extern "C"
