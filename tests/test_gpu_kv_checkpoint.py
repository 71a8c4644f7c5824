"""Incremental KV-segment checkpoint and request-level restoration (§6.1,
§6.2) on the GPU, byte for byte against the oracle, with pinned host memory
as the checkpoint store."""
import numpy as np
import pytest
import torch

from oracle import kv_checkpoint as K
from paper_2601_01310_amd import synth, tg
from tests._util import u16

pytestmark = pytest.mark.gpu
DEV = "cuda"

# Mixtral-8x7B segment: 8 KV heads x 128 x bf16, keys and values (App. C).
SEG = K.segment_bytes(8, 4096, 32, 2)


def _layout(layers, requests, max_len):
    """Byte offset of (layer, request, position) in a region laid out
    [layer][request][position][segment]."""
    def off(l, r, p):
        return ((l * requests + r) * max_len + p) * SEG
    return off, layers * requests * max_len * SEG


def _step_segments(off, layers, requests, pos):
    o = [off(l, r, pos) for r in range(requests) for l in range(layers)]
    return np.array(o, dtype=np.uint64), np.full(len(o), SEG, dtype=np.uint32)


def _host(nbytes, dtype=torch.uint8, fill=0):
    t = torch.empty(nbytes, dtype=dtype, pin_memory=True)
    t.fill_(fill)
    return t


def test_checkpoint_steps_then_restore_one_request():
    print("[gpu] kv checkpoint round trip", flush=True)
    layers, requests, max_len = 4, 16, 8
    off, size = _layout(layers, requests, max_len)
    g = torch.Generator(device=DEV)
    g.manual_seed(3)
    kv = torch.randint(0, 256, (size,), dtype=torch.uint8, device=DEV, generator=g)
    store = _host(size, fill=0xEE)
    log_cap = 256
    log = _host(log_cap * 3, dtype=torch.int64)
    commit = _host(1, dtype=torch.int64, fill=0)
    np_store = np.full(size, 0xEE, dtype=np.uint8)
    np_log = np.zeros((log_cap, 3), dtype=np.uint64)
    np_commit = 0
    kv_np = kv.cpu().numpy()
    seq = 0
    per_req = {}
    for pos in range(5):  # five decode steps
        o, b = _step_segments(off, layers, requests, pos)
        tg.tg_kv_checkpoint(kv, size, torch.from_numpy(o.view(np.int64)).to(DEV),
                            torch.from_numpy(b.view(np.int32)).to(DEV), len(o), seq, store, log,
                            log_cap, commit)
        np_store, np_log, np_commit = K.checkpoint(kv_np, np_store, np_log, log_cap, np_commit, o,
                                                   b, seq)
        for i, oi in enumerate(o.tolist()):
            r = (i // layers)
            per_req.setdefault(r, []).append((seq + i, oi))
        seq += len(o)
    torch.cuda.synchronize()
    assert np.array_equal(store.numpy(), np_store)
    assert np.array_equal(log.numpy().view(np.uint64).reshape(log_cap, 3), np_log)
    assert int(commit[0]) == np_commit == seq
    # restore request 5 into a fresh, compact region of another KV cache
    segs = per_req[5]
    sq = np.array([s for s, _ in segs], dtype=np.uint64)
    src = np.array([o for _, o in segs], dtype=np.uint64)
    dst = np.arange(len(segs), dtype=np.uint64) * SEG
    nb = np.full(len(segs), SEG, dtype=np.uint32)
    kv2 = torch.zeros(len(segs) * SEG, dtype=torch.uint8, device=DEV)
    status = torch.empty(len(segs), dtype=torch.uint8, device=DEV)
    tg.tg_kv_restore(store, size, commit, *(torch.from_numpy(a.view(np.int64)).to(DEV)
                                            for a in (sq, src, dst)),
                     torch.from_numpy(nb.view(np.int32)).to(DEV), len(segs), kv2, kv2.numel(),
                     status)
    torch.cuda.synchronize()
    want, st = K.restore(np_store, np_commit, sq, src, dst, nb, np.zeros(kv2.numel(), np.uint8))
    assert (status.cpu().numpy() == 1).all() and (st == 1).all()
    assert np.array_equal(kv2.cpu().numpy(), want)


def test_uncommitted_and_rejected_segments():
    size = 1 << 16
    kv = torch.randint(0, 256, (size,), dtype=torch.uint8, device=DEV)
    store = _host(size)
    log = _host(8 * 3, dtype=torch.int64)
    commit = _host(1, dtype=torch.int64, fill=0)
    o = np.array([0, 4096, 8, size - 16], dtype=np.uint64)
    b = np.array([4096, 4096, 16, 32], dtype=np.uint32)  # the last two are rejected
    tg.tg_kv_checkpoint(kv, size, torch.from_numpy(o.view(np.int64)).to(DEV),
                        torch.from_numpy(b.view(np.int32)).to(DEV), 4, 0, store, log, 8, commit)
    # a second batch that never commits (the worker fails before its commit record)
    o2 = np.array([8192], dtype=np.uint64)
    b2 = np.array([4096], dtype=np.uint32)
    tg.tg_kv_checkpoint(kv, size, torch.from_numpy(o2.view(np.int64)).to(DEV),
                        torch.from_numpy(b2.view(np.int32)).to(DEV), 1, 4, store, log, 8, None)
    torch.cuda.synchronize()
    assert int(commit[0]) == 4
    lg = log.numpy().view(np.uint64).reshape(8, 3)
    assert lg[:5, 2].tolist() == [4096, 4096, 0, 0, 4096]
    assert np.array_equal(store.numpy()[8192:12288], kv.cpu().numpy()[8192:12288])
    sq = torch.tensor([0, 4, 1], dtype=torch.int64, device=DEV)
    src = torch.tensor([0, 8192, 4096], dtype=torch.int64, device=DEV)
    dst = torch.tensor([0, 4096, 8192 + 8], dtype=torch.int64, device=DEV)
    nb = torch.tensor([4096, 4096, 4096], dtype=torch.int32, device=DEV)
    kv2 = torch.zeros(3 * 4096, dtype=torch.uint8, device=DEV)
    status = torch.empty(3, dtype=torch.uint8, device=DEV)
    tg.tg_kv_restore(store, size, commit, sq, src, dst, nb, 3, kv2, kv2.numel(), status)
    torch.cuda.synchronize()
    assert status.cpu().tolist() == [1, 0, 2]
    assert torch.equal(kv2[:4096], kv[:4096]) and not kv2[4096:].any()


def test_checkpoint_alongside_the_forward_changes_neither():
    """A checkpoint stream running while the EW forward runs on another
    stream: the forward's output is bit-identical to a forward alone and the
    store holds the segments."""
    print("[gpu] kv checkpoint alongside the forward", flush=True)
    wl = synth.make("tiny", device=DEV)
    f = tg.EwForward(wl)
    f()
    torch.cuda.synchronize()
    alone = u16(f.out)
    layers, requests, max_len = 32, 64, 4
    off, size = _layout(layers, requests, max_len)
    kv = torch.randint(0, 256, (size,), dtype=torch.uint8, device=DEV)
    store = _host(size)
    log = _host(4096 * 3, dtype=torch.int64)
    commit = _host(1, dtype=torch.int64, fill=0)
    o, b = _step_segments(off, layers, requests, 1)
    od, bd = torch.from_numpy(o.view(np.int64)).to(DEV), torch.from_numpy(b.view(np.int32)).to(DEV)
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        tg.tg_kv_checkpoint(kv, size, od, bd, len(o), 0, store, log, 4096, commit, stream=side)
    f()
    torch.cuda.synchronize()
    assert np.array_equal(u16(f.out), alone)
    assert int(commit[0]) == len(o)
    s, k = store.numpy(), kv.cpu().numpy()
    for oi in o.tolist()[::97]:
        assert np.array_equal(s[oi:oi + SEG], k[oi:oi + SEG])


def test_strided_checkpoint_on_the_copy_engine_matches_the_oracle():
    """One decode step of a [layer][request][position] region is a strided
    batch; the copy-engine path must leave the same store, log and commit
    record as the oracle, and a restore from it must round-trip."""
    layers, requests, max_len, pos = 8, 16, 6, 3
    off, size = _layout(layers, requests, max_len)
    kv = torch.randint(0, 256, (size,), dtype=torch.uint8, device=DEV)
    store = _host(size, fill=0x5A)
    log_cap = 64
    log = _host(log_cap * 3, dtype=torch.int64)
    commit = _host(1, dtype=torch.int64, fill=0)
    n = layers * requests
    first, pitch = off(0, 0, pos), max_len * SEG
    assert all(off(l, r, pos) == first + (l * requests + r) * pitch
               for l in range(layers) for r in range(requests))
    tg.tg_kv_checkpoint_strided(kv, size, first, pitch, SEG, n, 1000, store, log, log_cap, commit)
    torch.cuda.synchronize()
    o = np.array([first + i * pitch for i in range(n)], dtype=np.uint64)
    b = np.full(n, SEG, dtype=np.uint32)
    np_store, np_log, np_commit = K.checkpoint(kv.cpu().numpy(), np.full(size, 0x5A, np.uint8),
                                               np.zeros((log_cap, 3), np.uint64), log_cap, 0, o,
                                               b, 1000)
    assert np.array_equal(store.numpy(), np_store)
    assert np.array_equal(log.numpy().view(np.uint64).reshape(log_cap, 3), np_log)
    assert int(commit[0]) == np_commit == 1000 + n
    sq = torch.arange(1000, 1000 + n, dtype=torch.int64, device=DEV)
    src = torch.from_numpy(o.view(np.int64)).to(DEV)
    dst = torch.arange(n, dtype=torch.int64, device=DEV) * SEG
    nb = torch.full((n,), SEG, dtype=torch.int32, device=DEV)
    kv2 = torch.zeros(n * SEG, dtype=torch.uint8, device=DEV)
    status = torch.empty(n, dtype=torch.uint8, device=DEV)
    tg.tg_kv_restore(store, size, commit, sq, src, dst, nb, n, kv2, kv2.numel(), status)
    torch.cuda.synchronize()
    assert (status == 1).all()
    want = kv.view(layers * requests, max_len, SEG)[:, pos].reshape(-1)
    assert torch.equal(kv2, want)
