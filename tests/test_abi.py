"""The C ABI loads, exports every symbol its header declares, and rejects bad
arguments on the host before anything reaches the GPU (CPU-only tests)."""
import ctypes
import os
import re

import pytest

from paper_2601_01310_amd import tg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tg.h")

# Bogus but non-NULL addresses: every call below fails validation, so none is
# ever dereferenced or handed to the HIP runtime.
P = 0x1000


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(tg._LIB_PATH):
        from paper_2601_01310_amd import build
        build.build()
    return tg.load()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tg_[a-z_]+)\s*\(", src)))


def test_header_declares_the_documented_entry_points():
    names = declared_functions()
    assert set(names) == set(tg.EXPORTS), names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    assert lib.tg_status_string(0) == b"TG_OK"
    assert lib.tg_status_string(4) == b"TG_ERR_WORKSPACE"
    assert lib.tg_status_string(99) == b"TG_ERR_UNKNOWN"


def test_tile_policy_accepts_the_three_settings_only(lib):
    for bad in (-1, 3, 1 << 20):
        assert lib.tg_set_gemm_tile_policy(bad) == tg.TG_ERR_BAD_DIM
    assert b"tile policy" in lib.tg_last_error()
    for good in (tg.TILES_SMALL, tg.TILES_FULL, tg.TILES_AUTO):  # ends on the default
        assert lib.tg_set_gemm_tile_policy(good) == tg.TG_OK


def _gate(lib, **kw):
    a = dict(x=P, w_gate=P, logits_in=None, T=4, d=256, E=8, k=2, logits_out=None, ids=P, w=P)
    a.update(kw)
    return lib.tg_gate_topk(a["x"], a["w_gate"], a["logits_in"], a["T"], a["d"], a["E"], a["k"],
                            a["logits_out"], a["ids"], a["w"], None)


def test_gate_topk_rejects_bad_arguments(lib):
    assert _gate(lib, k=9) == tg.TG_ERR_BAD_DIM            # k > E
    assert _gate(lib, k=0) == tg.TG_ERR_BAD_DIM
    assert _gate(lib, T=-1) == tg.TG_ERR_BAD_DIM
    assert _gate(lib, E=2000, k=2) == tg.TG_ERR_UNSUPPORTED
    assert _gate(lib, E=64, k=33) == tg.TG_ERR_UNSUPPORTED
    assert _gate(lib, d=200) == tg.TG_ERR_UNSUPPORTED
    assert _gate(lib, ids=None) == tg.TG_ERR_NULL_ARG
    assert _gate(lib, w_gate=None) == tg.TG_ERR_NULL_ARG    # x without w_gate
    assert _gate(lib, logits_in=P) == tg.TG_ERR_NULL_ARG    # both modes at once
    assert _gate(lib, x=None, w_gate=None) == tg.TG_ERR_NULL_ARG
    assert b"k=9" in (_gate(lib, k=9) and lib.tg_last_error())


def _dispatch(lib, **kw):
    a = dict(ids=P, T=16, k=2, ert=P, E=8, R=2, alive=P, S=10, x=P, d=256, ps=P, cnt=P, off=P,
             perm=P, pr=P, xp=P, nu=P, ws=P, wsb=1 << 20)
    a.update(kw)
    return lib.tg_remap_dispatch(a["ids"], a["T"], a["k"], a["ert"], a["E"], a["R"], a["alive"],
                                 a["S"], a["x"], a["d"], a["ps"], a["cnt"], a["off"], a["perm"],
                                 a["pr"], a["xp"], a["nu"], a["ws"], a["wsb"], None)


def test_remap_dispatch_rejects_bad_arguments(lib):
    need = lib.tg_remap_dispatch_workspace(16, 2, 10)
    assert need > 0
    assert _dispatch(lib, wsb=need - 1) == tg.TG_ERR_WORKSPACE
    assert _dispatch(lib, ws=None) == tg.TG_ERR_WORKSPACE
    assert _dispatch(lib, ws=P + 8) == tg.TG_ERR_WORKSPACE  # misaligned
    assert _dispatch(lib, S=0) == tg.TG_ERR_BAD_DIM
    assert _dispatch(lib, S=1025) == tg.TG_ERR_UNSUPPORTED
    assert _dispatch(lib, R=17) == tg.TG_ERR_UNSUPPORTED
    assert _dispatch(lib, perm=None) == tg.TG_ERR_NULL_ARG
    assert _dispatch(lib, x=None) == tg.TG_ERR_NULL_ARG     # x_perm without x
    assert _dispatch(lib, d=300) == tg.TG_ERR_UNSUPPORTED
    assert lib.tg_remap_dispatch_workspace(-1, 2, 10) == 0


def test_workspace_grows_with_pairs(lib):
    small = lib.tg_remap_dispatch_workspace(64, 2, 10)
    big = lib.tg_remap_dispatch_workspace(1 << 20, 8, 40)
    assert big > small > 0


def _ffn(lib, **kw):
    a = dict(xp=P, off=P, S=10, rows=128, w13=P, w2=P, d=256, I=512, h=P, y=P)
    a.update(kw)
    return lib.tg_expert_ffn_grouped(a["xp"], a["off"], a["S"], a["rows"], a["w13"], a["w2"],
                                     a["d"], a["I"], a["h"], a["y"], None)


def test_expert_ffn_rejects_bad_arguments(lib):
    assert _ffn(lib, I=100) == tg.TG_ERR_UNSUPPORTED
    assert _ffn(lib, I=0) == tg.TG_ERR_BAD_DIM
    assert _ffn(lib, d=96) == tg.TG_ERR_UNSUPPORTED   # not a multiple of 64
    assert _ffn(lib, d=64) == tg.TG_ERR_UNSUPPORTED   # fewer than two K stages
    assert _ffn(lib, I=64) == tg.TG_ERR_UNSUPPORTED
    assert _ffn(lib, rows=-1) == tg.TG_ERR_BAD_DIM
    assert _ffn(lib, S=0) == tg.TG_ERR_BAD_DIM
    assert _ffn(lib, h=None) == tg.TG_ERR_NULL_ARG
    assert _ffn(lib, d=16384, I=32768) == tg.TG_ERR_UNSUPPORTED  # 2 GiB per slot


def test_combine_rejects_bad_arguments(lib):
    assert lib.tg_combine(P, P, P, 4, 0, 256, P, None) == tg.TG_ERR_BAD_DIM
    assert lib.tg_combine(P, P, P, 4, 40, 256, P, None) == tg.TG_ERR_UNSUPPORTED
    assert lib.tg_combine(P, P, P, 4, 2, 100, P, None) == tg.TG_ERR_UNSUPPORTED
    assert lib.tg_combine(None, P, P, 4, 2, 256, P, None) == tg.TG_ERR_NULL_ARG


def test_ew_forward_rejects_bad_arguments(lib):
    a = tg.EwArgs()
    a.T, a.d, a.E, a.k, a.I, a.S, a.R = 8, 256, 8, 2, 512, 10, 2
    for n in ("x", "w_gate", "ert", "slot_alive", "w13", "w2", "out"):
        setattr(a, n, P)
    need = lib.tg_ew_forward_workspace(ctypes.byref(a))
    assert need > 0
    assert lib.tg_ew_forward(ctypes.byref(a), P, need - 1, None) == tg.TG_ERR_WORKSPACE
    a.logits_in = P  # both gating inputs
    assert lib.tg_ew_forward(ctypes.byref(a), P, need, None) == tg.TG_ERR_NULL_ARG
    assert lib.tg_ew_forward_workspace(ctypes.byref(a)) == 0
    a.logits_in = None
    a.out = None
    assert lib.tg_ew_forward(ctypes.byref(a), P, need, None) == tg.TG_ERR_NULL_ARG
    a.out = P
    a.k = 9
    assert lib.tg_ew_forward(ctypes.byref(a), P, need, None) == tg.TG_ERR_BAD_DIM
    assert lib.tg_ew_forward(None, P, need, None) == tg.TG_ERR_NULL_ARG


def test_ew_replay_rejects_bad_arguments(lib):
    a = tg.ReplayArgs()
    a.T, a.d, a.E, a.k, a.I, a.S, a.R = 8, 256, 8, 2, 512, 10, 2
    for n in ("x", "ert", "slot_alive", "w13", "w2", "topk_ids", "topk_w", "pair_slot",
              "pair_row", "y", "out"):
        setattr(a, n, P)
    need = lib.tg_ew_replay_workspace(ctypes.byref(a))
    assert need > 0
    assert lib.tg_ew_replay(ctypes.byref(a), P, need - 1, None) == tg.TG_ERR_WORKSPACE
    assert lib.tg_ew_replay(ctypes.byref(a), P + 16, need, None) == tg.TG_ERR_WORKSPACE
    a.y = None  # the first pass's per-pair outputs are required
    assert lib.tg_ew_replay(ctypes.byref(a), P, need, None) == tg.TG_ERR_NULL_ARG
    assert lib.tg_ew_replay_workspace(ctypes.byref(a)) == 0
    a.y = P
    a.k = 9
    assert lib.tg_ew_replay(ctypes.byref(a), P, need, None) == tg.TG_ERR_BAD_DIM
    a.k, a.I = 2, 100
    assert lib.tg_ew_replay(ctypes.byref(a), P, need, None) == tg.TG_ERR_UNSUPPORTED
    assert lib.tg_ew_replay(None, P, need, None) == tg.TG_ERR_NULL_ARG


def test_kept_outputs_shrink_the_forward_workspace(lib):
    a = tg.EwArgs()
    a.T, a.d, a.E, a.k, a.I, a.S, a.R = 64, 256, 8, 2, 512, 10, 2
    for n in ("x", "w_gate", "ert", "slot_alive", "w13", "w2", "out"):
        setattr(a, n, P)
    need = lib.tg_ew_forward_workspace(ctypes.byref(a))
    a.y = P  # per-pair outputs in a caller buffer instead of the workspace
    assert lib.tg_ew_forward_workspace(ctypes.byref(a)) == need - 64 * 2 * 256 * 2


def test_batch_trigger_rejects_bad_arguments(lib):
    def call(**kw):
        a = dict(d=P, al=P, cr=P, A=4, T=64, m=16, spin=10, tv=P, st=P)
        a.update(kw)
        return lib.tg_batch_trigger(a["d"], a["al"], a["cr"], a["A"], a["T"], a["m"], a["spin"],
                                    a["tv"], a["st"], None)
    assert call(A=0) == tg.TG_ERR_BAD_DIM
    assert call(T=-1) == tg.TG_ERR_BAD_DIM
    assert call(m=-1) == tg.TG_ERR_BAD_DIM
    assert call(spin=0) == tg.TG_ERR_BAD_DIM
    assert call(A=1025) == tg.TG_ERR_UNSUPPORTED
    assert call(d=None) == tg.TG_ERR_NULL_ARG
    assert call(tv=None) == tg.TG_ERR_NULL_ARG
    assert call(st=None) == tg.TG_ERR_NULL_ARG


def test_kv_checkpoint_entry_points_reject_bad_arguments(lib):
    A = 0x10000  # 16-byte aligned bogus addresses
    assert lib.tg_kv_checkpoint(A, 1 << 20, A, A, -1, 0, A, A, 8, None, 0, None) == tg.TG_ERR_BAD_DIM
    assert lib.tg_kv_checkpoint(A, 1 << 20, A, A, 4, 0, A, A, 0, None, 0, None) == tg.TG_ERR_BAD_DIM
    assert lib.tg_kv_checkpoint(A, 1 << 20, A, A, 4, 0, A, A, 8, None, -1, None) == tg.TG_ERR_BAD_DIM
    assert lib.tg_kv_checkpoint(A, 1 << 20, None, A, 4, 0, A, A, 8, None, 0, None) == tg.TG_ERR_NULL_ARG
    assert lib.tg_kv_checkpoint(A + 8, 1 << 20, A, A, 4, 0, A, A, 8, None, 0, None) == \
        tg.TG_ERR_UNSUPPORTED
    s = lib.tg_kv_checkpoint_strided
    assert s(A, 1 << 20, 0, 4096, 4096, 257, 0, A, A, 8, None, None) == tg.TG_ERR_BAD_DIM  # past end
    assert s(A, 1 << 20, 8, 4096, 4096, 4, 0, A, A, 8, None, None) == tg.TG_ERR_BAD_DIM   # misaligned
    assert s(A, 1 << 20, 0, 2048, 4096, 4, 0, A, A, 8, None, None) == tg.TG_ERR_BAD_DIM   # overlap
    assert s(A, 1 << 20, 0, 4096, 4096, 4, 0, A, None, 8, None, None) == tg.TG_ERR_NULL_ARG
    r = lib.tg_kv_restore
    assert r(A, 1 << 20, None, A, A, A, A, 4, A, 1 << 20, A, None) == tg.TG_ERR_NULL_ARG
    assert r(A, 1 << 20, A, A, A, A, A, -1, A, 1 << 20, A, None) == tg.TG_ERR_BAD_DIM
    assert r(A, 1 << 20, A, A, A, A, A, 4, A + 4, 1 << 20, A, None) == tg.TG_ERR_UNSUPPORTED


def test_binding_refuses_host_tensors(lib):
    import torch
    with pytest.raises(ValueError):
        tg.tg_combine(torch.zeros(4), None, None, 1, 1, 256, None, stream=0)


def test_readme_c_example_compiles_against_the_header(tmp_path):
    """The C function in README.md is valid C against include/tg.h."""
    import re
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    text = open(os.path.join(ROOT, "README.md")).read()
    blocks = re.findall(r"```c\n(.*?)```", text, flags=re.S)
    assert blocks, "README.md has no C example"
    src = tmp_path / "example.c"
    src.write_text(blocks[0])
    r = subprocess.run([cc, "-std=c11", "-Wall", "-Werror", "-fsyntax-only",
                        f"-I{os.path.join(ROOT, 'include')}", str(src)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
