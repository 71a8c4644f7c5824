"""ctypes binding of libtg.so (the C ABI declared in ``include/tg.h``).

The functions below carry the C names and marshal torch tensors (device
memory owned by the caller) into raw pointers; every step of the forward
runs in the library's HIP kernels. The binding refuses to run without the
built library: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtg.so")
_lib = None

TG_OK, TG_ERR_NULL_ARG, TG_ERR_BAD_DIM, TG_ERR_UNSUPPORTED, TG_ERR_WORKSPACE, TG_ERR_HIP = range(6)

EXPORTS = [
    "tg_status_string", "tg_last_error", "tg_gate_topk", "tg_remap_dispatch_workspace",
    "tg_remap_dispatch", "tg_expert_ffn_grouped", "tg_set_gemm_tile_policy", "tg_combine",
    "tg_ew_forward_workspace", "tg_ew_forward", "tg_ew_forward_timed", "tg_ew_forward_noalloc",
    "tg_ew_replay_workspace", "tg_ew_replay", "tg_batch_trigger", "tg_kv_checkpoint",
    "tg_kv_checkpoint_strided", "tg_kv_restore",
]


class TgError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = load()
        name = lib.tg_status_string(status).decode()
        detail = lib.tg_last_error().decode()
        super().__init__(f"{where}: {name}: {detail}")
        self.status = status


class EwArgs(ctypes.Structure):
    """Mirror of ``tg_ew_args``."""
    _fields_ = [(n, ctypes.c_int) for n in ("T", "d", "E", "k", "I", "S", "R")] + [
        (n, ctypes.c_void_p) for n in (
            "x", "w_gate", "logits_in", "ert", "slot_alive", "w13", "w2", "out", "topk_ids",
            "topk_w", "pair_slot", "slot_counts", "slot_offsets", "pair_row", "n_unserved", "y",
            "token_valid")
    ]


class ReplayArgs(ctypes.Structure):
    """Mirror of ``tg_replay_args``."""
    _fields_ = [(n, ctypes.c_int) for n in ("T", "d", "E", "k", "I", "S", "R")] + [
        (n, ctypes.c_void_p) for n in (
            "x", "ert", "slot_alive", "w13", "w2", "topk_ids", "topk_w", "pair_slot", "pair_row",
            "y", "out", "replay_slot", "n_replayed", "n_unserved")
    ]


def load(path: Optional[str] = None):
    """Loads libtg.so (built in-tree by ``paper_2601_01310_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or _LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2601_01310_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.tg_status_string.restype = ctypes.c_char_p
    lib.tg_status_string.argtypes = [i]
    lib.tg_last_error.restype = ctypes.c_char_p
    lib.tg_last_error.argtypes = []
    lib.tg_gate_topk.restype = i
    lib.tg_gate_topk.argtypes = [vp, vp, vp, i, i, i, i, vp, vp, vp, vp]
    lib.tg_remap_dispatch_workspace.restype = sz
    lib.tg_remap_dispatch_workspace.argtypes = [i, i, i]
    lib.tg_remap_dispatch.restype = i
    lib.tg_remap_dispatch.argtypes = [vp, i, i, vp, i, i, vp, i, vp, i, vp, vp, vp, vp, vp, vp, vp,
                                      vp, sz, vp]
    lib.tg_expert_ffn_grouped.restype = i
    lib.tg_expert_ffn_grouped.argtypes = [vp, vp, i, i, vp, vp, i, i, vp, vp, vp]
    lib.tg_set_gemm_tile_policy.argtypes = [i]
    lib.tg_set_gemm_tile_policy.restype = i
    lib.tg_combine.restype = i
    lib.tg_combine.argtypes = [vp, vp, vp, i, i, i, vp, vp]
    lib.tg_ew_forward_workspace.restype = sz
    lib.tg_ew_forward_workspace.argtypes = [ctypes.POINTER(EwArgs)]
    lib.tg_ew_forward.restype = i
    lib.tg_ew_forward.argtypes = [ctypes.POINTER(EwArgs), vp, sz, vp]
    lib.tg_ew_forward_timed.restype = i
    lib.tg_ew_forward_timed.argtypes = [ctypes.POINTER(EwArgs), vp, sz, vp,
                                        ctypes.POINTER(ctypes.c_void_p), i]
    lib.tg_ew_forward_noalloc.restype = i
    lib.tg_ew_forward_noalloc.argtypes = [ctypes.POINTER(EwArgs), vp]
    lib.tg_ew_replay_workspace.restype = sz
    lib.tg_ew_replay_workspace.argtypes = [ctypes.POINTER(ReplayArgs)]
    lib.tg_ew_replay.restype = i
    lib.tg_ew_replay.argtypes = [ctypes.POINTER(ReplayArgs), vp, sz, vp]
    lib.tg_batch_trigger.restype = i
    lib.tg_batch_trigger.argtypes = [vp, vp, vp, i, i, i, ctypes.c_longlong, vp, vp, vp]
    u64 = ctypes.c_uint64
    lib.tg_kv_checkpoint.restype = i
    lib.tg_kv_checkpoint.argtypes = [vp, sz, vp, vp, i, u64, vp, vp, i, vp, i, vp]
    lib.tg_kv_checkpoint_strided.restype = i
    lib.tg_kv_checkpoint_strided.argtypes = [vp, sz, u64, u64, ctypes.c_uint32, i, u64, vp, vp, i,
                                             vp, vp]
    lib.tg_kv_restore.restype = i
    lib.tg_kv_restore.argtypes = [vp, sz, vp, vp, vp, vp, vp, i, vp, sz, vp, vp]
    _lib = lib
    return lib


def _p(t) -> Optional[int]:
    """Tensor (or None, or an int address) -> raw pointer."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if t.device.type != "cuda":
        raise ValueError("libtg takes device tensors only")
    if not t.is_contiguous():
        raise ValueError("libtg takes contiguous tensors only")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int, where: str):
    if status != TG_OK:
        raise TgError(status, where)


def tg_gate_topk(x, w_gate, logits_in, T, d, E, k, logits_out, topk_ids, topk_w, stream=None):
    _check(load().tg_gate_topk(_p(x), _p(w_gate), _p(logits_in), T, d, E, k, _p(logits_out),
                               _p(topk_ids), _p(topk_w), _stream(stream)), "tg_gate_topk")


def tg_remap_dispatch_workspace(T, k, S) -> int:
    return int(load().tg_remap_dispatch_workspace(T, k, S))


def tg_remap_dispatch(topk_ids, T, k, ert, E, R, slot_alive, S, x, d, pair_slot, slot_counts,
                      slot_offsets, perm, pair_row, x_perm, n_unserved, ws, ws_bytes, stream=None):
    _check(load().tg_remap_dispatch(_p(topk_ids), T, k, _p(ert), E, R, _p(slot_alive), S, _p(x), d,
                                    _p(pair_slot), _p(slot_counts), _p(slot_offsets), _p(perm),
                                    _p(pair_row), _p(x_perm), _p(n_unserved), _p(ws), ws_bytes,
                                    _stream(stream)), "tg_remap_dispatch")


def tg_expert_ffn_grouped(x_perm, slot_offsets, S, max_rows, w13, w2, d, I, h, y, stream=None):
    _check(load().tg_expert_ffn_grouped(_p(x_perm), _p(slot_offsets), S, max_rows, _p(w13), _p(w2),
                                        d, I, _p(h), _p(y), _stream(stream)),
           "tg_expert_ffn_grouped")


TILES_AUTO, TILES_SMALL, TILES_FULL = 0, 1, 2


def tg_set_gemm_tile_policy(policy):
    _check(load().tg_set_gemm_tile_policy(policy), "tg_set_gemm_tile_policy")


class tile_policy:
    """Context manager: the grouped GEMMs' tile height forced for a block."""

    def __init__(self, policy):
        self.policy = policy

    def __enter__(self):
        tg_set_gemm_tile_policy(self.policy)
        return self

    def __exit__(self, *exc):
        tg_set_gemm_tile_policy(TILES_AUTO)


def tg_combine(y, pair_row, topk_w, T, k, d, out, stream=None):
    _check(load().tg_combine(_p(y), _p(pair_row), _p(topk_w), T, k, d, _p(out), _stream(stream)),
           "tg_combine")


def make_ew_args(T, d, E, k, I, S, R, x, w_gate, logits_in, ert, slot_alive, w13, w2, out,
                 topk_ids=None, topk_w=None, pair_slot=None, slot_counts=None, slot_offsets=None,
                 pair_row=None, n_unserved=None, y=None, token_valid=None) -> EwArgs:
    a = EwArgs()
    a.T, a.d, a.E, a.k, a.I, a.S, a.R = T, d, E, k, I, S, R
    for name, v in dict(x=x, w_gate=w_gate, logits_in=logits_in, ert=ert, slot_alive=slot_alive,
                        w13=w13, w2=w2, out=out, topk_ids=topk_ids, topk_w=topk_w,
                        pair_slot=pair_slot, slot_counts=slot_counts, slot_offsets=slot_offsets,
                        pair_row=pair_row, n_unserved=n_unserved, y=y,
                        token_valid=token_valid).items():
        setattr(a, name, _p(v))
    return a


def make_replay_args(T, d, E, k, I, S, R, x, ert, slot_alive, w13, w2, topk_ids, topk_w,
                     pair_slot, pair_row, y, out, replay_slot=None, n_replayed=None,
                     n_unserved=None) -> ReplayArgs:
    a = ReplayArgs()
    a.T, a.d, a.E, a.k, a.I, a.S, a.R = T, d, E, k, I, S, R
    for name, v in dict(x=x, ert=ert, slot_alive=slot_alive, w13=w13, w2=w2, topk_ids=topk_ids,
                        topk_w=topk_w, pair_slot=pair_slot, pair_row=pair_row, y=y, out=out,
                        replay_slot=replay_slot, n_replayed=n_replayed,
                        n_unserved=n_unserved).items():
        setattr(a, name, _p(v))
    return a


def tg_ew_forward_workspace(args: EwArgs) -> int:
    return int(load().tg_ew_forward_workspace(ctypes.byref(args)))


def tg_ew_forward(args: EwArgs, ws, ws_bytes, stream=None):
    _check(load().tg_ew_forward(ctypes.byref(args), _p(ws), ws_bytes, _stream(stream)),
           "tg_ew_forward")


# Bytes of the library's own scratch area behind tg_ew_forward_noalloc
# (TG_NOALLOC_SCRATCH_BYTES in tg.h).
NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024


def tg_ew_forward_noalloc(args: EwArgs, stream=None):
    _check(load().tg_ew_forward_noalloc(ctypes.byref(args), _stream(stream)),
           "tg_ew_forward_noalloc")


def tg_ew_forward_timed(args: EwArgs, ws, ws_bytes, events, stream=None):
    """``events``: six hipEvent_t handles (ints)."""
    arr = (ctypes.c_void_p * len(events))(*events)
    _check(load().tg_ew_forward_timed(ctypes.byref(args), _p(ws), ws_bytes, _stream(stream), arr,
                                      len(events)), "tg_ew_forward_timed")


def tg_batch_trigger(delivered, aw_alive, chunk_rows, A, T, min_rows, spin_limit, token_valid,
                     status, stream=None):
    """``delivered`` may be a device tensor or a pinned host tensor (its
    device-visible address is passed)."""
    _check(load().tg_batch_trigger(_flag_ptr(delivered), _p(aw_alive), _p(chunk_rows), A, T,
                                   min_rows, spin_limit, _p(token_valid), _p(status),
                                   _stream(stream)), "tg_batch_trigger")


def tg_kv_checkpoint(kv, kv_bytes, seg_offset, seg_bytes, n, first_seq, store, log, log_cap,
                     commit, stream=None, max_blocks=0):
    """``store``, ``log`` ([log_cap, 3] uint64) and ``commit`` ([1] uint64)
    may be pinned host tensors or device tensors; ``commit`` may be None."""
    _check(load().tg_kv_checkpoint(_p(kv), kv_bytes, _p(seg_offset), _p(seg_bytes), n, first_seq,
                                   _flag_ptr(store), _flag_ptr(log), log_cap,
                                   None if commit is None else _flag_ptr(commit), max_blocks,
                                   _stream(stream)), "tg_kv_checkpoint")


def tg_kv_checkpoint_strided(kv, kv_bytes, first_offset, pitch, seg_bytes, n, first_seq, store,
                             log, log_cap, commit, stream=None):
    _check(load().tg_kv_checkpoint_strided(_p(kv), kv_bytes, first_offset, pitch, seg_bytes, n,
                                           first_seq, _flag_ptr(store), _flag_ptr(log), log_cap,
                                           None if commit is None else _flag_ptr(commit),
                                           _stream(stream)), "tg_kv_checkpoint_strided")


def tg_kv_restore(store, store_bytes, commit, seq, src, dst, nbytes, n, kv_dst, kv_bytes, status,
                  stream=None):
    _check(load().tg_kv_restore(_flag_ptr(store), store_bytes, _flag_ptr(commit), _p(seq), _p(src),
                                _p(dst), _p(nbytes), n, _p(kv_dst), kv_bytes, _p(status),
                                _stream(stream)), "tg_kv_restore")


def _flag_ptr(t):
    """Device tensors as usual; a pinned host tensor is passed by its address,
    which the GPU can use directly."""
    if isinstance(t, torch.Tensor) and t.device.type == "cpu":
        if not t.is_pinned() or not t.is_contiguous():
            raise ValueError("host buffers must be contiguous pinned tensors")
        return t.data_ptr()  # pinned host memory is mapped at the same address on the device
    return _p(t)


def tg_ew_replay_workspace(args: ReplayArgs) -> int:
    return int(load().tg_ew_replay_workspace(ctypes.byref(args)))


def tg_ew_replay(args: ReplayArgs, ws, ws_bytes, stream=None):
    _check(load().tg_ew_replay(ctypes.byref(args), _p(ws), ws_bytes, _stream(stream)),
           "tg_ew_replay")


# ----------------------------------------------------------------------------
# Convenience wrappers: allocate outputs with torch, then call the C ABI.
# ----------------------------------------------------------------------------


def workspace(nbytes: int, device) -> torch.Tensor:
    """A 256-byte aligned device buffer (torch's caching allocator aligns to 512)."""
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


class EwForward:
    """Holds the outputs and workspace of one workload shape so repeated calls
    allocate nothing (the timed loop of the benchmark reuses one of these).

    ``keep_y`` keeps the per-pair expert outputs in ``self.y`` so that failed
    pairs can be replayed afterwards (``replay``); ``token_valid`` ([T] uint8)
    restricts the batch to the tokens marked 1."""

    def __init__(self, wl, alive=None, keep_y=False, token_valid=None):
        dev = wl.x.device
        T, k, S = wl.T, wl.k, wl.S
        self.wl = wl
        self.alive = wl.alive if alive is None else alive
        self.out = torch.empty((T, wl.d), dtype=torch.bfloat16, device=dev)
        self.topk_ids = torch.empty((T, k), dtype=torch.int32, device=dev)
        self.topk_w = torch.empty((T, k), dtype=torch.float32, device=dev)
        self.pair_slot = torch.empty((T, k), dtype=torch.int32, device=dev)
        self.slot_counts = torch.empty((S,), dtype=torch.int32, device=dev)
        self.slot_offsets = torch.empty((S + 1,), dtype=torch.int32, device=dev)
        self.pair_row = torch.empty((T, k), dtype=torch.int32, device=dev)
        self.n_unserved = torch.empty((1,), dtype=torch.int32, device=dev)
        self.y = (torch.empty((max(T * k, 1), wl.d), dtype=torch.bfloat16, device=dev)
                  if keep_y else None)
        self.token_valid = token_valid
        self.args = make_ew_args(
            T, wl.d, wl.E, k, wl.I, S, wl.R, wl.x, wl.wg, wl.logits, wl.ert, self.alive, wl.w13,
            wl.w2, self.out, self.topk_ids, self.topk_w, self.pair_slot, self.slot_counts,
            self.slot_offsets, self.pair_row, self.n_unserved, self.y, token_valid)
        self.ws_bytes = tg_ew_forward_workspace(self.args)
        if self.ws_bytes == 0:
            raise TgError(load().tg_ew_forward(ctypes.byref(self.args), None, 0, None), "workspace")
        self.ws = workspace(self.ws_bytes, dev)
        self._replay = None

    def __call__(self, stream=None):
        tg_ew_forward(self.args, self.ws, self.ws_bytes, stream)
        return self.out

    def set_alive(self, alive):
        self.alive = alive
        self.args.slot_alive = _p(alive)

    def replay(self, alive, stream=None):
        """Replays the pairs of the last forward whose slots are not alive in
        ``alive`` (needs ``keep_y``); updates ``self.out`` in place and
        returns (replay_slot, n_replayed, n_unserved) device tensors."""
        if self.y is None:
            raise ValueError("construct EwForward with keep_y=True to replay")
        wl, dev = self.wl, self.out.device
        if self._replay is None:
            r = dict(replay_slot=torch.empty((wl.T, wl.k), dtype=torch.int32, device=dev),
                     n_replayed=torch.empty((1,), dtype=torch.int32, device=dev),
                     n_unserved=torch.empty((1,), dtype=torch.int32, device=dev))
            r["args"] = make_replay_args(
                wl.T, wl.d, wl.E, wl.k, wl.I, wl.S, wl.R, wl.x, wl.ert, alive, wl.w13, wl.w2,
                self.topk_ids, self.topk_w, self.pair_slot, self.pair_row, self.y, self.out,
                r["replay_slot"], r["n_replayed"], r["n_unserved"])
            r["ws_bytes"] = tg_ew_replay_workspace(r["args"])
            r["ws"] = workspace(r["ws_bytes"], dev)
            self._replay = r
        r = self._replay
        r["alive"] = alive
        r["args"].slot_alive = _p(alive)
        tg_ew_replay(r["args"], r["ws"], r["ws_bytes"], stream)
        return r["replay_slot"], r["n_replayed"], r["n_unserved"]
