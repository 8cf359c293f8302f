"""Python binding of libdllm_rps: argument marshalling only.

Every function has the name of the C entry point it calls and takes torch
tensors (device memory) instead of raw pointers.  Torch provides device
memory and the current stream; every step of the computation runs in the
library's HIP kernels.  A non-zero status raises DllmError with the
library's message.
"""
from __future__ import annotations

import ctypes as C

import torch

from . import _abi
from ._abi import (DllmError, ModelDesc, Weights, StatsC, KvCache, Probe, RpsParams, RpsPlan, RpsDecision,
                   DLLM_F32, DLLM_BF16, RPS_PIVOT_PAPER, RPS_PIVOT_BAND, DLLM_MAX_TOPK, RPS_MAX_BRANCH)

_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        _LIB = _abi.load()
    return _LIB


def _check(status: int):
    if status != 0:
        raise DllmError(status, lib().dllm_last_error().decode())


def _p(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return C.c_void_p(stream.cuda_stream)
    return C.c_void_p(stream)


# ---------------------------------------------------------------- device buffers

class Stats:
    """Per-position statistics of R rows in device memory (dllm_stats)."""

    def __init__(self, R: int, k: int = DLLM_MAX_TOPK, device="cuda", _views=None):
        if _views is not None:
            self.H, self.lse, self.lmax, self.argmax, self.topk_id, self.topk_logit = _views
        else:
            f = dict(dtype=torch.float32, device=device)
            i = dict(dtype=torch.int32, device=device)
            self.H = torch.empty(R, **f)
            self.lse = torch.empty(R, **f)
            self.lmax = torch.empty(R, **f)
            self.argmax = torch.empty(R, **i)
            self.topk_id = torch.empty(R, k, **i)
            self.topk_logit = torch.empty(R, k, **f)
        self.k = self.topk_id.shape[1]

    @property
    def R(self) -> int:
        return self.H.shape[0]

    def rows(self, start: int, n: int) -> "Stats":
        sl = slice(start, start + n)
        return Stats(0, _views=(self.H[sl], self.lse[sl], self.lmax[sl], self.argmax[sl], self.topk_id[sl],
                                self.topk_logit[sl]))

    def c(self) -> StatsC:
        return StatsC(self.H.data_ptr(), self.lse.data_ptr(), self.lmax.data_ptr(), self.argmax.data_ptr(),
                      self.topk_id.data_ptr(), self.topk_logit.data_ptr(), self.k)

    def fill_(self, value: float):
        for t in (self.H, self.lse, self.lmax, self.topk_logit):
            t.fill_(value)
        self.argmax.fill_(-1)
        self.topk_id.fill_(-1)
        return self

    def numpy(self) -> dict:
        return {n: getattr(self, n).cpu().numpy() for n in ("H", "lse", "lmax", "argmax", "topk_id", "topk_logit")}


def new_plan(device="cuda"):
    return torch.zeros(C.sizeof(RpsPlan), dtype=torch.uint8, device=device)


def new_decision(device="cuda"):
    return torch.zeros(C.sizeof(RpsDecision), dtype=torch.uint8, device=device)


def read_plan(t) -> RpsPlan:
    return RpsPlan.from_buffer_copy(t.cpu().numpy().tobytes())


def read_decision(t) -> RpsDecision:
    return RpsDecision.from_buffer_copy(t.cpu().numpy().tobytes())


def plan_field_ptr(plan, name: str) -> int:
    """Device address of an array field of a device-resident rps_plan."""
    return plan.data_ptr() + getattr(RpsPlan, name).offset


def params(mode="band", k_max=10, tau_pivot=0.9, pct_lo=25.0, pct_hi=75.0, n_pivots=1, r=0.1, n_cand=10,
           max_branch=RPS_MAX_BRANCH) -> RpsParams:
    m = RPS_PIVOT_BAND if mode == "band" else RPS_PIVOT_PAPER
    return RpsParams(m, k_max, tau_pivot, pct_lo, pct_hi, n_pivots, r, n_cand, max_branch)


# ---------------------------------------------------------------- model

def dllm_model_create(desc: ModelDesc, weights: dict):
    """weights: emb, lm_head, wqkv, wo, wgu, wdown (lists of per-layer device tensors)."""
    L = desc.n_layers
    arrs = {}
    for name in ("wqkv", "wo", "wgu", "wdown"):
        a = (C.c_void_p * L)(*[w.data_ptr() for w in weights[name]])
        arrs[name] = a
    w = Weights(weights["emb"].data_ptr(), weights["lm_head"].data_ptr(),
                C.cast(arrs["wqkv"], C.POINTER(C.c_void_p)), C.cast(arrs["wo"], C.POINTER(C.c_void_p)),
                C.cast(arrs["wgu"], C.POINTER(C.c_void_p)), C.cast(arrs["wdown"], C.POINTER(C.c_void_p)))
    handle = C.c_void_p()
    _check(lib().dllm_model_create(C.byref(desc), C.byref(w), C.byref(handle)))
    return handle


def dllm_model_destroy(handle):
    lib().dllm_model_destroy(handle)


def dllm_profile_begin(handle, max_launches: int = 20000, classes=None):
    """classes: optional iterable of kernel-class names (PROF_NAMES) to bracket; default all."""
    if classes is None:
        _check(lib().dllm_profile_begin(handle, max_launches))
        return
    mask = 0
    for name in classes:
        mask |= 1 << _abi.PROF_NAMES.index(name)
    _check(lib().dllm_profile_begin_classes(handle, max_launches, mask))


def dllm_profile_end(handle) -> dict:
    """{kernel class: (total ms, launches)} of the launches since dllm_profile_begin."""
    ms = (C.c_float * _abi.DLLM_PROF_CLASSES)()
    n = (C.c_int32 * _abi.DLLM_PROF_CLASSES)()
    _check(lib().dllm_profile_end(handle, ms, n))
    return {name: (float(ms[i]), int(n[i])) for i, name in enumerate(_abi.PROF_NAMES)}


def dllm_mfma_ceiling(random_operands: bool = True, stream=None) -> float:
    """Sustained bf16 MFMA rate of the device on a register-only loop, TFLOP/s
    (random_operands: different random operands at every instruction)."""
    out = C.c_float(0.0)
    _check(lib().dllm_mfma_ceiling(1 if random_operands else 0, C.byref(out), _stream(stream)))
    return float(out.value)


def dllm_workspace_bytes(handle, batch: int, seq: int, n_lm_pos: int) -> int:
    return lib().dllm_workspace_bytes(handle, batch, seq, n_lm_pos)


def dllm_workspace_bytes_packed(handle, shared_len: int, block_len: int, n_branch: int, n_lm_pos: int) -> int:
    return lib().dllm_workspace_bytes_packed(handle, shared_len, block_len, n_branch, n_lm_pos)


def dllm_forward(handle, tokens, lm_pos, out: Stats, ws, pos_offset: int = 0, row_scale=None, scale: float = 1.0,
                 kv_prefix: KvCache | None = None, kv_out: KvCache | None = None, probe: Probe | None = None,
                 n_lm_pos: int | None = None, stream=None):
    batch, seq = tokens.shape
    n_lm = lm_pos.shape[0] if n_lm_pos is None else n_lm_pos
    _check(lib().dllm_forward(handle, _p(tokens), batch, seq, pos_offset,
                              None if kv_prefix is None else C.byref(kv_prefix),
                              None if kv_out is None else C.byref(kv_out), _p(lm_pos), n_lm, _p(row_scale),
                              scale, None if probe is None else C.byref(probe), C.byref(out.c()), _p(ws),
                              ws.numel() * ws.element_size(), _stream(stream)))


def dllm_forward_packed(handle, tokens, shared_len: int, block_start: int, block_len: int, n_branch: int, lm_pos,
                        out: Stats, ws, pos_offset: int = 0, kv_prefix: KvCache | None = None, row_scale=None,
                        scale: float = 1.0, probe: Probe | None = None, n_lm_pos: int | None = None, stream=None):
    """Packed lookahead forward: tokens [shared_len + n_branch * block_len] (one
    sequence); out receives (1 + n_branch) * n_lm_pos rows (shared, then each branch)."""
    n_lm = lm_pos.shape[0] if n_lm_pos is None else n_lm_pos
    _check(lib().dllm_forward_packed(handle, _p(tokens), shared_len, block_start, block_len, n_branch, pos_offset,
                                     None if kv_prefix is None else C.byref(kv_prefix), _p(lm_pos), n_lm,
                                     _p(row_scale), scale, None if probe is None else C.byref(probe),
                                     C.byref(out.c()), _p(ws), ws.numel() * ws.element_size(), _stream(stream)))


def vocab_entropy_topk_workspace_bytes(R: int, vocab: int) -> int:
    return lib().vocab_entropy_topk_workspace_bytes(R, vocab)


def vocab_entropy_topk(hidden, w_lm, out: Stats, ws, row_scale=None, scale: float = 1.0, mask_id: int = -1,
                       stream=None):
    R, d = hidden.shape
    V = w_lm.shape[0]
    dt = DLLM_BF16 if hidden.dtype == torch.bfloat16 else DLLM_F32
    _check(lib().vocab_entropy_topk(_p(hidden), _p(w_lm), R, d, V, dt, _p(row_scale), scale, mask_id,
                                    C.byref(out.c()), _p(ws), ws.numel() * ws.element_size(), _stream(stream)))


def vocab_entropy_topk_noalloc(hidden, w_lm, out: Stats, row_scale=None, scale: float = 1.0, mask_id: int = -1,
                               stream=None):
    R, d = hidden.shape
    V = w_lm.shape[0]
    dt = DLLM_BF16 if hidden.dtype == torch.bfloat16 else DLLM_F32
    _check(lib().vocab_entropy_topk_noalloc(_p(hidden), _p(w_lm), R, d, V, dt, _p(row_scale), scale, mask_id,
                                            C.byref(out.c()), _stream(stream)))


# ---------------------------------------------------------------- scheduler

def rps_select_pivots(base: Stats, m_pos, n_m: int, prm: RpsParams, plan, stream=None):
    _check(lib().rps_select_pivots(C.byref(base.c()), _p(m_pos), n_m, C.byref(prm), _p(plan), _stream(stream)))


def rps_build_branches(tokens, plan, anchor_first: bool, capacity: int, out, stream=None):
    _check(lib().rps_build_branches(_p(tokens), tokens.shape[-1], _p(plan), int(anchor_first), capacity, _p(out),
                                    _stream(stream)))


def rps_build_packed(tokens, plan, block_start: int, block_len: int, capacity: int, out, stream=None):
    """out[seq + capacity * block_len]: tokens, then one block copy per branch slot."""
    _check(lib().rps_build_packed(_p(tokens), tokens.shape[-1], _p(plan), block_start, block_len, capacity, _p(out),
                                  _stream(stream)))


def rps_lookahead_score(anchor: Stats, branches: Stats, branch_offset: int, n_m: int, plan, lam: float, dec,
                        anchor_logit=None, scores=None, deltas=None, stream=None):
    _check(lib().rps_lookahead_score(C.byref(anchor.c()), C.byref(branches.c()), branch_offset, n_m, _p(plan),
                                     _p(anchor_logit), lam, _p(scores), _p(deltas), _p(dec), _stream(stream)))


def rps_commit(tokens, m_pos, n_m: int, base: Stats, tau: float, n_m_out, committed, n_committed, dec=None,
               branches: Stats | None = None, branch_offset: int = 0, anchor: Stats | None = None, stream=None):
    _check(lib().rps_commit(_p(tokens), tokens.shape[-1], _p(m_pos), n_m, C.byref(base.c()), _p(dec),
                            None if branches is None else C.byref(branches.c()), branch_offset,
                            None if anchor is None else C.byref(anchor.c()), tau, _p(n_m_out), _p(committed),
                            _p(n_committed), _stream(stream)))


def sched_commit(tokens, m_pos, n_m: int, stats: Stats, rule: int, k: int, n_m_out, committed, n_committed,
                 stream=None):
    """Baseline scheduler commit (Eq. 2, top-k by confidence or by lowest entropy)."""
    _check(lib().sched_commit(_p(tokens), tokens.shape[-1], _p(m_pos), n_m, C.byref(stats.c()), rule, k,
                              _p(n_m_out), _p(committed), _p(n_committed), _stream(stream)))
