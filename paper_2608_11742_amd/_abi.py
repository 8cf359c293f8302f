"""ctypes mirror of include/dllm_rps.h and the loader of libdllm_rps.so.

The library is required: there is no fallback.  Importing this module fails
with ImportError if the in-tree shared object has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdllm_rps.so")

DLLM_MAX_TOPK = 16
RPS_MAX_PIVOTS = 16
RPS_MAX_BRANCH = 16
RPS_MAX_MASKED = 1024

DLLM_F32, DLLM_BF16 = 0, 1
RPS_PIVOT_PAPER, RPS_PIVOT_BAND = 0, 1
DLLM_PROF_CLASSES = 10
PROF_NAMES = ("embed", "rmsnorm", "gemm_qkv", "attention", "gemm_o", "gemm_gateup", "gemm_down", "lmhead",
              "lmhead_merge", "other")

STATUS = {0: "DLLM_OK", 1: "DLLM_EINVAL", 2: "DLLM_ESHAPE", 3: "DLLM_EDTYPE", 4: "DLLM_ENOMEM",
          5: "DLLM_EHIP", 6: "DLLM_EUNSUPPORTED"}

i32, f32, vp, sz = C.c_int32, C.c_float, C.c_void_p, C.c_size_t


class ModelDesc(C.Structure):
    _fields_ = [("n_layers", i32), ("d_model", i32), ("n_heads", i32), ("head_dim", i32), ("d_ffn", i32),
                ("vocab", i32), ("mask_id", i32), ("rope_base", f32), ("rms_eps", f32), ("dtype", i32),
                ("max_pos", i32)]


class Weights(C.Structure):
    _fields_ = [("emb", vp), ("lm_head", vp), ("wqkv", C.POINTER(vp)), ("wo", C.POINTER(vp)),
                ("wgu", C.POINTER(vp)), ("wdown", C.POINTER(vp))]


class StatsC(C.Structure):
    _fields_ = [("H", vp), ("lse", vp), ("lmax", vp), ("argmax", vp), ("topk_id", vp), ("topk_logit", vp),
                ("k", i32)]


class KvCache(C.Structure):
    _fields_ = [("k", vp), ("vt", vp), ("len", i32), ("cap", i32)]


class Probe(C.Structure):
    _fields_ = [("row", vp), ("token", vp), ("logit", vp), ("n", i32)]


class RpsParams(C.Structure):
    _fields_ = [("mode", i32), ("k_max", i32), ("tau_pivot", f32), ("pct_lo", f32), ("pct_hi", f32),
                ("n_pivots", i32), ("r", f32), ("n_cand", i32), ("max_branch", i32)]


class RpsPlan(C.Structure):
    _fields_ = [("n_pivots", i32), ("n_branch", i32), ("pivot_row", i32 * RPS_MAX_PIVOTS),
                ("pivot_pos", i32 * RPS_MAX_PIVOTS), ("n_cand", i32 * RPS_MAX_PIVOTS),
                ("br_pivot", i32 * RPS_MAX_BRANCH), ("br_row", i32 * RPS_MAX_BRANCH),
                ("br_pos", i32 * RPS_MAX_BRANCH), ("br_token", i32 * RPS_MAX_BRANCH),
                ("br_logp", f32 * RPS_MAX_BRANCH)]


class RpsDecision(C.Structure):
    _fields_ = [("commit", i32), ("branch", i32), ("pivot_row", i32), ("pivot_pos", i32), ("token", i32),
                ("delta", f32), ("second_delta", f32), ("n_masked", i32)]


# name -> (restype, argtypes); the same names as the C ABI
SIGNATURES = {
    "dllm_abi_version": (i32, []),
    "dllm_last_error": (C.c_char_p, []),
    "dllm_status_string": (C.c_char_p, [i32]),
    "dllm_model_create": (i32, [C.POINTER(ModelDesc), C.POINTER(Weights), C.POINTER(vp)]),
    "dllm_model_destroy": (None, [vp]),
    "dllm_workspace_bytes": (sz, [vp, i32, i32, i32]),
    "dllm_workspace_bytes_packed": (sz, [vp, i32, i32, i32, i32]),
    "dllm_forward": (i32, [vp, vp, i32, i32, i32, C.POINTER(KvCache), C.POINTER(KvCache), vp, i32, vp, f32,
                           C.POINTER(Probe), C.POINTER(StatsC), vp, sz, vp]),
    "dllm_forward_packed": (i32, [vp, vp, i32, i32, i32, i32, i32, C.POINTER(KvCache), vp, i32, vp, f32,
                                  C.POINTER(Probe), C.POINTER(StatsC), vp, sz, vp]),
    "vocab_entropy_topk_workspace_bytes": (sz, [i32, i32]),
    "vocab_entropy_topk": (i32, [vp, vp, i32, i32, i32, i32, vp, f32, i32, C.POINTER(StatsC), vp, sz, vp]),
    "vocab_entropy_topk_noalloc": (i32, [vp, vp, i32, i32, i32, i32, vp, f32, i32, C.POINTER(StatsC), vp]),
    "dllm_profile_begin": (i32, [vp, i32]),
    "dllm_profile_begin_classes": (i32, [vp, i32, C.c_uint32]),
    "dllm_profile_end": (i32, [vp, C.POINTER(f32), C.POINTER(i32)]),
    "dllm_mfma_ceiling": (i32, [i32, C.POINTER(f32), vp]),
    "rps_select_pivots": (i32, [C.POINTER(StatsC), vp, i32, C.POINTER(RpsParams), vp, vp]),
    "rps_build_branches": (i32, [vp, i32, vp, i32, i32, vp, vp]),
    "rps_build_packed": (i32, [vp, i32, vp, i32, i32, i32, vp, vp]),
    "rps_lookahead_score": (i32, [C.POINTER(StatsC), C.POINTER(StatsC), i32, i32, vp, vp, f32, vp, vp, vp, vp]),
    "rps_commit": (i32, [vp, i32, vp, i32, C.POINTER(StatsC), vp, C.POINTER(StatsC), i32, C.POINTER(StatsC), f32,
                         vp, vp, vp, vp]),
    "sched_commit": (i32, [vp, i32, vp, i32, C.POINTER(StatsC), i32, i32, vp, vp, vp, vp]),
}

SCHED_TOP_CONFIDENCE, SCHED_LOW_ENTROPY = 0, 1


def load(path: str = LIB_PATH):
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: the HIP library must be built first "
                          "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = C.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


class DllmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status
