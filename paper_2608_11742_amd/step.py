"""Drivers that sequence the library calls of one RPS step and of the full
RPS decode (Algorithm 1).  All arithmetic runs in libdllm_rps; the host only
reads back |M| (and, in the decode loop, the plan's branch count) to size
the next launch.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

from . import binding as B
from . import _abi
from ._abi import Probe, KvCache


class RpsStep:
    """Batched lookahead step over one sequence whose anchor is the current
    statistics (the carried distributions): pivots and candidates from
    `base`, a lookahead forward over `capacity` branch sequences, Eq. 4
    scoring against `base`, then commit and carry-over.

    tokens: [seq] int32 device; m_pos: [n_m] int32 device (ascending masked
    positions); base: statistics of the n_m rows.  All three are updated in place.
    """

    def __init__(self, model, tokens, m_pos, base: B.Stats, prm, lam: float = 0.0, capacity: int = 16,
                 row_scale=None, scale: float = 1.0, kv_prefix: KvCache | None = None, pos_offset: int = 0):
        self.model, self.tokens, self.m_pos, self.base = model, tokens, m_pos, base
        self.prm, self.lam, self.capacity = prm, lam, capacity
        self.row_scale, self.scale, self.kv_prefix, self.pos_offset = row_scale, scale, kv_prefix, pos_offset
        self.n_m = int(m_pos.shape[0])
        dev = tokens.device
        self.plan = B.new_plan(dev)
        self.dec = B.new_decision(dev)
        self.branch_tokens = torch.empty(capacity, tokens.shape[0], dtype=torch.int32, device=dev)
        self.branch_stats = B.Stats(capacity * self.n_m, base.k, device=dev)
        self.scores = torch.zeros(16, dtype=torch.float32, device=dev)
        self.deltas = torch.zeros(16, dtype=torch.float32, device=dev)
        self.n_m_out = torch.zeros(1, dtype=torch.int32, device=dev)
        self.committed = torch.zeros(self.n_m, dtype=torch.int32, device=dev)
        self.n_committed = torch.zeros(1, dtype=torch.int32, device=dev)
        model.workspace(capacity, tokens.shape[0], self.n_m)   # sized once for the largest step

    def launch(self, stream=None):
        """Enqueue one step (no host synchronisation)."""
        n = self.n_m
        B.rps_select_pivots(self.base, self.m_pos, n, self.prm, self.plan, stream)
        B.rps_build_branches(self.tokens, self.plan, False, self.capacity, self.branch_tokens, stream)
        self.model.forward(self.branch_tokens, self.m_pos, out=self.branch_stats, n_lm_pos=n,
                           row_scale=self.row_scale, scale=self.scale, pos_offset=self.pos_offset,
                           kv_prefix=self.kv_prefix, stream=stream)
        B.rps_lookahead_score(self.base, self.branch_stats, 0, n, self.plan, self.lam, self.dec,
                              scores=self.scores, deltas=self.deltas, stream=stream)
        B.rps_commit(self.tokens, self.m_pos, n, self.base, -1.0, self.n_m_out, self.committed, self.n_committed,
                     dec=self.dec, branches=self.branch_stats, branch_offset=0, anchor=None, stream=stream)

    def run(self, stream=None) -> int:
        """One step; returns the new |M| (synchronises on it)."""
        if self.n_m <= 1:
            return self.n_m
        self.launch(stream)
        self.n_m = int(self.n_m_out.item())
        return self.n_m


@dataclass
class DecodeStats:
    nfe: int = 0
    normal: int = 0
    lookahead: int = 0
    commits_conf: int = 0
    commits_pivot: int = 0
    abstains: int = 0
    normal_ms: float = 0.0
    lookahead_ms: float = 0.0
    trace: list = field(default_factory=list)


class _BlockView:
    """Where the forwards of one block run.  Without a prefix cache: the whole
    sequence, absolute positions.  With the prefix cache (Fast-dLLM's, which
    the paper combines RPS with; Section 5.3): the full forward that opens the
    block writes every layer's keys and values into the cache, and the later
    forwards of the block run on the block and the masked suffix only, at
    positions relative to the block start, attending to the cached prefix."""

    def __init__(self, model, tokens, row_scale, scale, prefix_cache: bool):
        self.model, self.tokens, self.row_scale, self.scale = model, tokens, row_scale, scale
        self.S = tokens.shape[0]
        self.kv = None
        if prefix_cache:
            k, vt, cap = model.new_kv_cache(self.S)
            self._kv_buf = (k, vt)
            self.kv = KvCache(k.data_ptr(), vt.data_ptr(), 0, cap)
        self.b0 = 0

    def open(self, b0: int, block: int, out, n: int, probe=None):
        """Full forward over the sequence at the block opening; returns the
        block's masked positions in the view's coordinates."""
        dev = self.tokens.device
        m_abs = torch.arange(b0, b0 + block, dtype=torch.int32, device=dev)
        self.b0 = b0
        if self.kv is None:
            self.model.forward(self.tokens[None], m_abs, out=out, n_lm_pos=n, row_scale=self.row_scale,
                               scale=self.scale, probe=probe)
            return m_abs
        self.kv.len = 0
        self.model.forward(self.tokens[None], m_abs, out=out, n_lm_pos=n, row_scale=self.row_scale,
                           scale=self.scale, probe=probe, kv_out=self.kv)
        self.kv.len = b0
        return torch.arange(0, block, dtype=torch.int32, device=dev)

    @property
    def seq(self):
        """The token sequence the block's later forwards and commits work on."""
        return self.tokens if self.kv is None else self.tokens[self.b0:]

    @property
    def offset(self) -> int:
        return 0 if self.kv is None else self.b0

    def forward_packed(self, tok, block: int, nb: int, m_pos, out, n: int, probe=None):
        """Packed lookahead [seq || nb copies of the block] (tok: the packed tokens)."""
        L = self.seq.shape[0]
        if self.kv is None:
            self.model.forward_packed(tok, L, self.b0, block, nb, m_pos, out=out, n_lm_pos=n,
                                      row_scale=self.row_scale, scale=self.scale, probe=probe)
            return
        rs = None if self.row_scale is None else self.row_scale[self.b0:]
        self.model.forward_packed(tok, L, 0, block, nb, m_pos, out=out, n_lm_pos=n, row_scale=rs, scale=self.scale,
                                  pos_offset=self.b0, kv_prefix=self.kv if self.b0 > 0 else None, probe=probe)

    def forward(self, tok, m_pos, out, n: int, probe=None):
        if self.kv is None:
            self.model.forward(tok, m_pos, out=out, n_lm_pos=n, row_scale=self.row_scale, scale=self.scale,
                               probe=probe)
            return
        rs = None if self.row_scale is None else self.row_scale[self.b0:]
        self.model.forward(tok, m_pos, out=out, n_lm_pos=n, row_scale=rs, scale=self.scale, probe=probe,
                           pos_offset=self.b0, kv_prefix=self.kv if self.b0 > 0 else None)


def rps_decode(model, prompt, gen_len: int, block: int, prm, lam: float, tau: float, capacity: int = 16,
               row_scale=None, scale: float = 1.0, k: int = 16, timing: bool = False, record: bool = False,
               packed: bool = False, prefix_cache: bool = False):
    """Algorithm 1 on the GPU.  prompt: [P] int32 device.  Returns (tokens, DecodeStats).

    row_scale: optional [P + gen_len] per-position logit scales (device float32).
    record: keep a trace of every decision, ("commit", positions),
    ("skip",) and ("lookahead", pivot, token or -1), at the cost of one more
    read-back per standard commit.
    packed: run each lookahead as one packed sequence [x || block copies] with
    the branch-isolating mask (dllm_forward_packed) instead of a batch of
    1 + n full sequences; block must then be a power of two.
    prefix_cache: refresh a prefix KV cache at every block opening and run the
    block's later forwards (normal and lookahead) on the block and the masked
    suffix only (see _BlockView); with packed, the packed sequence is [block +
    suffix || block copies] over the cached prefix.
    """
    if prm.max_branch > capacity - 1:
        raise ValueError("prm.max_branch must leave slot 0 of the lookahead batch to the anchor")
    dev = prompt.device
    P = prompt.shape[0]
    S = P + gen_len
    mask_id = model.shape.mask_id
    tokens = torch.cat([prompt.to(torch.int32), torch.full((gen_len,), mask_id, dtype=torch.int32, device=dev)])
    st = DecodeStats()
    base = B.Stats(block, k, device=dev)
    branch = B.Stats(capacity * block, k, device=dev)
    plan = B.new_plan(dev)
    dec = B.new_decision(dev)
    bt_buf = torch.empty(capacity * S, dtype=torch.int32, device=dev)
    pk = torch.empty(S + (capacity - 1) * block, dtype=torch.int32, device=dev) if packed else None
    anchor_logit = torch.empty(16, dtype=torch.float32, device=dev)
    n_m_out = torch.zeros(1, dtype=torch.int32, device=dev)
    committed = torch.zeros(block, dtype=torch.int32, device=dev)
    n_committed = torch.zeros(1, dtype=torch.int32, device=dev)
    if packed:
        model.workspace(1, S, block)
        model.workspace_packed(S, block, capacity - 1, block)
    else:
        model.workspace(capacity, S, block)
    view = _BlockView(model, tokens, row_scale, scale, prefix_cache)
    ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) if timing else None

    def timed(kind, fn):
        if ev:
            ev[0].record()
        r = fn()
        st.nfe += 1
        if kind == "normal":
            st.normal += 1
        else:
            st.lookahead += 1
        if ev:
            ev[1].record()
            ev[1].synchronize()
            ms = ev[0].elapsed_time(ev[1])
            if kind == "normal":
                st.normal_ms += ms
            else:
                st.lookahead_ms += ms
        return r

    for b in range(gen_len // block):
        b0 = P + b * block
        n_m = block
        m_pos = timed("normal", lambda: view.open(b0, block, base, n_m))   # block-opening forward
        seq, off = view.seq, view.offset
        L = seq.shape[0]
        bt = bt_buf[:capacity * L].view(capacity, L)
        while n_m > 0:
            B.rps_commit(seq, m_pos, n_m, base, tau, n_m_out, committed, n_committed)   # standard commit
            n_new = int(n_m_out.item())
            st.commits_conf += n_m - n_new
            if record:
                st.trace.append(("commit", sorted(int(c) + off for c in committed[:n_m - n_new].tolist())))
            n_m = n_new
            if n_m == 0:
                break
            B.rps_select_pivots(base, m_pos, n_m, prm, plan)
            nb = B.read_plan(plan).n_branch
            if nb == 0:                                                  # skip rules: normal forward
                timed("normal", lambda: view.forward(seq[None], m_pos, base, n_m))
                st.trace.append(("skip",))
                continue
            probe = Probe(B.plan_field_ptr(plan, "br_row"), B.plan_field_ptr(plan, "br_token"),
                          anchor_logit.data_ptr(), nb)
            if packed:
                B.rps_build_packed(seq, plan, b0 - off, block, nb, pk)
                timed("lookahead", lambda: view.forward_packed(pk[:L + nb * block], block, nb, m_pos, branch, n_m,
                                                               probe=probe))
            else:
                B.rps_build_branches(seq, plan, True, 1 + nb, bt)
                timed("lookahead", lambda: view.forward(bt[:1 + nb], m_pos, branch, n_m, probe=probe))
            anchor = branch.rows(0, n_m)
            B.rps_lookahead_score(anchor, branch, 1, n_m, plan, lam, dec, anchor_logit=anchor_logit)
            B.rps_commit(seq, m_pos, n_m, base, -1.0, n_m_out, committed, n_committed, dec=dec,
                         branches=branch, branch_offset=1, anchor=anchor)
            n_new = int(n_m_out.item())
            if record:
                d = B.read_decision(dec)
                st.trace.append(("lookahead", d.pivot_pos + off, d.token if d.commit else -1))
            if n_new < n_m:
                st.commits_pivot += 1
            else:
                st.abstains += 1
            n_m = n_new
    return tokens, st


_SCHED_RULES = {"confidence": _abi.SCHED_TOP_CONFIDENCE, "entropy": _abi.SCHED_LOW_ENTROPY}


def baseline_decode(model, prompt, gen_len: int, block: int, rule: str, k: int = 1, tau: float = 0.9,
                    row_scale=None, scale: float = 1.0, topk: int = 16, timing: bool = False,
                    record: bool = False, prefix_cache: bool = False):
    """The semi-autoregressive baselines of Section 3 (Eq. 1 and 2) on the GPU.

    Blocks left to right; every step is one forward over the sequence and one
    commit of S with greedy tokens: the k most confident masked positions
    (rule "confidence"; k = 1 is the Default decoder), the k lowest-entropy
    ones (rule "entropy", sched_commit), or every position with P^max >= tau
    and else the most confident one (rule "threshold", rps_commit without a
    lookahead decision: the Confidence baseline).  Returns (tokens, DecodeStats);
    record keeps ("commit", positions) per step.  prefix_cache: as in
    rps_decode; a block's first step is its full opening forward.
    """
    if rule not in ("confidence", "entropy", "threshold"):
        raise ValueError(f"unknown rule {rule!r}")
    dev = prompt.device
    P = prompt.shape[0]
    S = P + gen_len
    mask_id = model.shape.mask_id
    tokens = torch.cat([prompt.to(torch.int32), torch.full((gen_len,), mask_id, dtype=torch.int32, device=dev)])
    st = DecodeStats()
    base = B.Stats(block, topk, device=dev)
    n_m_out = torch.zeros(1, dtype=torch.int32, device=dev)
    committed = torch.zeros(block, dtype=torch.int32, device=dev)
    n_committed = torch.zeros(1, dtype=torch.int32, device=dev)
    model.workspace(1, S, block)
    view = _BlockView(model, tokens, row_scale, scale, prefix_cache)
    ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) if timing else None
    for b in range(gen_len // block):
        b0 = P + b * block
        n_m = block
        m_pos = None
        while n_m > 0:
            if ev:
                ev[0].record()
            if m_pos is None:
                m_pos = view.open(b0, block, base, n_m)
                seq, off = view.seq, view.offset
            else:
                view.forward(seq[None], m_pos, base, n_m)
            st.nfe += 1
            st.normal += 1
            if ev:
                ev[1].record()
                ev[1].synchronize()
                st.normal_ms += ev[0].elapsed_time(ev[1])
            if rule == "threshold":
                B.rps_commit(seq, m_pos, n_m, base, tau, n_m_out, committed, n_committed)
            else:
                B.sched_commit(seq, m_pos, n_m, base, _SCHED_RULES[rule], k, n_m_out, committed, n_committed)
            n_new = int(n_m_out.item())
            st.commits_conf += n_m - n_new
            if record:
                st.trace.append(("commit", sorted(int(c) + off for c in committed[:n_m - n_new].tolist())))
            n_m = n_new
    return tokens, st
