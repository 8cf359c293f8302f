"""The C-ABI library loads, exports every declared entry point and rejects bad
arguments on the host, before any HIP call (runs without a GPU)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dllm_rps.h")
LIB = os.path.join(ROOT, "paper_2608_11742_amd", "libdllm_rps.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libdllm_rps.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:[\w\s\*]+?)\b(\w+)\s*\(", text, flags=re.M)) - {"if", "for"})


@pytest.fixture(scope="module")
def abi():
    from paper_2608_11742_amd import _abi
    return _abi, _abi.load()


def test_every_declared_symbol_is_exported(abi):
    _, lib = abi
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    from paper_2608_11742_amd._abi import SIGNATURES
    assert set(SIGNATURES) == set(names)


def test_version_and_strings(abi):
    _abi, lib = abi
    assert lib.dllm_abi_version() == 1
    assert lib.dllm_status_string(4) == b"workspace too small"


def test_struct_layouts_match_header_sizes(abi):
    _abi, _ = abi
    assert C.sizeof(_abi.RpsPlan) == 4 * (2 + 3 * 16 + 5 * 16)
    assert C.sizeof(_abi.RpsDecision) == 32
    assert C.sizeof(_abi.StatsC) == 6 * 8 + 8
    assert C.sizeof(_abi.ModelDesc) == 11 * 4


def _err(lib):
    return lib.dllm_last_error().decode()


def _desc(_abi, **kw):
    d = dict(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ffn=1024, vocab=1024, mask_id=1023,
             rope_base=10000.0, rms_eps=1e-5, dtype=_abi.DLLM_F32, max_pos=128)
    d.update(kw)
    return _abi.ModelDesc(**d)


def _weights(_abi, L=2, null_layer=None):
    fake = C.c_void_p(0x1000)
    arr = (C.c_void_p * L)(*([fake] * L))
    if null_layer is not None:
        arr[null_layer] = None
    p = C.cast(arr, C.POINTER(C.c_void_p))
    return _abi.Weights(fake, fake, p, p, p, p), arr


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, 2), ("d_model", 320, 2), ("d_model", 8448, 2), ("d_ffn", 1000, 2), ("dtype", 7, 3),
    ("mask_id", 1024, 1), ("n_layers", 0, 2), ("rms_eps", 0.0, 1),
])
def test_model_create_rejects_bad_desc(abi, field, value, status):
    _abi, lib = abi
    w, keep = _weights(_abi)
    kw = {field: value}
    if field == "d_model":
        kw["n_heads"] = value // 64
    h = C.c_void_p()
    assert lib.dllm_model_create(C.byref(_desc(_abi, **kw)), C.byref(w), C.byref(h)) == status
    assert _err(lib)


def test_model_create_rejects_null_weights(abi):
    _abi, lib = abi
    w, keep = _weights(_abi, null_layer=1)
    h = C.c_void_p()
    assert lib.dllm_model_create(C.byref(_desc(_abi)), C.byref(w), C.byref(h)) == 1
    assert "layer 1" in _err(lib)
    assert lib.dllm_model_create(None, C.byref(w), C.byref(h)) == 1


def _stats(_abi, k=16, null=False):
    fake = 0x2000
    return _abi.StatsC(None if null else fake, fake, fake, fake, fake, fake, k)


def test_vocab_entropy_topk_validation(abi):
    _abi, lib = abi
    fake = C.c_void_p(0x3000)
    st = _stats(_abi)
    need = lib.vocab_entropy_topk_workspace_bytes(64, 1024)
    assert need > 0
    call = lambda **kw: lib.vocab_entropy_topk(
        kw.get("h", fake), fake, kw.get("R", 64), kw.get("d", 256), 1024, kw.get("dt", 0), None, 1.0,
        kw.get("mask", 1023), C.byref(kw.get("st", st)), fake, kw.get("ws", need), None)
    assert call(h=None) == 1
    assert call(st=_stats(_abi, null=True)) == 1
    assert call(st=_stats(_abi, k=17)) == 1
    assert call(dt=5) == 3
    assert call(R=0) == 2
    assert call(d=100) == 2                 # not a multiple of the 32-element fp32 stage
    assert call(dt=1, d=96) == 2            # nor of the 64-element bf16 stage
    assert call(mask=1024) == 1
    assert call(ws=need - 1) == 4
    assert "workspace" in _err(lib)


def test_scheduler_validation(abi):
    _abi, lib = abi
    fake = C.c_void_p(0x4000)
    st = _stats(_abi)
    prm = _abi.RpsParams(1, 10, 0.9, 25.0, 75.0, 2, 0.0, 4, 16)
    assert lib.rps_select_pivots(C.byref(st), fake, 0, C.byref(prm), fake, None) == 2
    assert lib.rps_select_pivots(C.byref(st), fake, 2000, C.byref(prm), fake, None) == 2
    bad = _abi.RpsParams(1, 17, 0.9, 25.0, 75.0, 2, 0.0, 4, 16)
    assert lib.rps_select_pivots(C.byref(st), fake, 32, C.byref(bad), fake, None) == 1
    bad = _abi.RpsParams(1, 10, 0.9, 75.0, 25.0, 2, 0.0, 4, 16)
    assert lib.rps_select_pivots(C.byref(st), fake, 32, C.byref(bad), fake, None) == 1
    bad = _abi.RpsParams(1, 10, 0.9, 25.0, 75.0, 2, 0.0, 4, 17)
    assert lib.rps_select_pivots(C.byref(st), fake, 32, C.byref(bad), fake, None) == 1
    assert lib.rps_build_branches(fake, 64, fake, 0, 18, fake, None) == 2
    assert lib.rps_lookahead_score(C.byref(st), C.byref(st), 2, 32, fake, None, 0.0, None, None, fake, None) == 1
    assert lib.rps_lookahead_score(C.byref(st), C.byref(st), 0, 32, fake, None, -1.0, None, None, fake, None) == 1
    assert lib.rps_commit(fake, 64, fake, 0, C.byref(st), None, None, 0, None, 0.9, fake, fake, fake, None) == 2
    st8 = _stats(_abi, k=8)
    assert lib.rps_commit(fake, 64, fake, 32, C.byref(st), fake, C.byref(st8), 0, None, 0.9, fake, fake, fake,
                          None) == 1
    # baseline scheduler commit: rule outside the enum, k < 1, |M| out of range, NULL arguments
    assert lib.sched_commit(fake, 64, fake, 32, C.byref(st), 2, 1, fake, fake, fake, None) == 1
    assert lib.sched_commit(fake, 64, fake, 32, C.byref(st), _abi.SCHED_LOW_ENTROPY, 0, fake, fake, fake, None) == 1
    assert lib.sched_commit(fake, 64, fake, 0, C.byref(st), _abi.SCHED_TOP_CONFIDENCE, 1, fake, fake, fake, None) == 2
    assert lib.sched_commit(fake, 64, fake, 2000, C.byref(st), 0, 1, fake, fake, fake, None) == 2
    assert lib.sched_commit(None, 64, fake, 32, C.byref(st), 0, 1, fake, fake, fake, None) == 1
    # packed lookahead tokens: block outside the sequence, capacity beyond RPS_MAX_BRANCH, NULL arguments
    assert lib.rps_build_packed(fake, 64, fake, 48, 32, 4, fake, None) == 2
    assert lib.rps_build_packed(fake, 64, fake, -1, 8, 4, fake, None) == 2
    assert lib.rps_build_packed(fake, 64, fake, 0, 8, _abi.RPS_MAX_BRANCH + 1, fake, None) == 2
    assert lib.rps_build_packed(fake, 64, None, 0, 8, 4, fake, None) == 1
    # packed forward without a model
    assert lib.dllm_forward_packed(None, fake, 64, 0, 8, 2, 0, None, fake, 4, None, 1.0, None, C.byref(st), fake, 1 << 20,
                                   None) == 1
    assert lib.dllm_workspace_bytes_packed(None, 64, 8, 2, 4) == 0


def test_model_create_without_device_reports_hip_error(abi):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    _abi, lib = abi
    w, keep = _weights(_abi)
    h = C.c_void_p()
    assert lib.dllm_model_create(C.byref(_desc(_abi)), C.byref(w), C.byref(h)) == 5
    assert "hipMalloc" in _err(lib)


def test_mfma_ceiling_rejects_null_output(abi):
    _abi, lib = abi
    assert lib.dllm_mfma_ceiling(1, None, None) == 1   # DLLM_EINVAL, before any device call
    assert "NULL" in _err(lib)
