"""CPU oracle for the incremental KV-segment checkpoint and the
request-level restoration of Tarragon (arXiv 2601.01310, §6.1, §6.2).

TEST INFRASTRUCTURE ONLY: imported by the tests, never by the product path;
it shares no code with the HIP path. Buffers are numpy uint8 arrays.

§6.1: the attention worker's KV cache is one contiguous region and the
checkpoint store keeps a bucket of the same layout, so a segment's offset in
the region is its offset in the store. Each new per-token, per-layer segment
is written to the store asynchronously, tagged with a monotonically
increasing sequence number; because such writes may land in any order, a
commit record (the "async log + commit record" design) says up to which
sequence number the store is complete: here it holds the number after the
last committed one (0 = nothing committed). §6.2: restoring a request copies its
committed segments into a fresh region of another worker's KV cache.
"""
from __future__ import annotations

import numpy as np


def _ok(off: int, nbytes: int, limit: int) -> bool:
    return off % 16 == 0 and nbytes % 16 == 0 and off <= limit and nbytes <= limit - off


def checkpoint(kv, store, log, log_cap, commit, seg_offset, seg_bytes, first_seq,
               write_commit=True):
    """Copies segment i (kv[off:off+len]) to store[off:off+len] with sequence
    number first_seq + i, records {seq, offset, bytes} at log[seq % log_cap]
    (bytes 0 for a rejected segment), then sets the commit record past the
    batch's last sequence number. Returns the new (store, log, commit)."""
    store = np.array(store, dtype=np.uint8, copy=True)
    log = np.array(log, dtype=np.uint64, copy=True)
    n = len(seg_offset)
    for i in range(n):
        off, nb = int(seg_offset[i]), int(seg_bytes[i])
        seq = first_seq + i
        ok = _ok(off, nb, kv.size)
        if ok:
            store[off:off + nb] = kv[off:off + nb]
        log[seq % log_cap] = (seq, off, nb if ok else 0)
    if write_commit and n:
        commit = first_seq + n
    return store, log, commit


def restore(store, commit, seq, src, dst, seg_bytes, kv_dst):
    """Copies each committed segment (seq < commit) from the store to its
    place in the destination KV region; returns (kv_dst, status) with status
    1 restored, 0 not committed, 2 misaligned or out of range."""
    kv_dst = np.array(kv_dst, dtype=np.uint8, copy=True)
    status = np.zeros(len(seq), dtype=np.uint8)
    for i in range(len(seq)):
        nb = int(seg_bytes[i])
        if not (_ok(int(src[i]), nb, store.size) and _ok(int(dst[i]), nb, kv_dst.size)):
            status[i] = 2
        elif int(seq[i]) >= commit:
            status[i] = 0
        else:
            kv_dst[int(dst[i]):int(dst[i]) + nb] = store[int(src[i]):int(src[i]) + nb]
            status[i] = 1
    return kv_dst, status


def segment_bytes(n_kv_heads: int, hidden: int, n_heads: int, elem_bytes: int) -> int:
    """Bytes of one token's KV segment of one layer, C = 2 H_kv (N/H_attn)
    S_elem (App. C): keys and values of every KV head."""
    return 2 * n_kv_heads * (hidden // n_heads) * elem_bytes


def expert_traffic_bytes(top_k: int, hidden: int, elem_bytes: int) -> int:
    """Per-token, per-layer AW-EW traffic, V = 2 top_k N S_elem (App. C):
    the token's row to each chosen expert and the outputs back."""
    return 2 * top_k * hidden * elem_bytes
