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


def rps_decode(model, prompt, gen_len: int, block: int, prm, lam: float, tau: float, capacity: int = 16,
               row_scale=None, scale: float = 1.0, k: int = 16, timing: bool = False, record: bool = False,
               packed: bool = False):
    """Algorithm 1 on the GPU.  prompt: [P] int32 device.  Returns (tokens, DecodeStats).

    row_scale: optional [P + gen_len] per-position logit scales (device float32).
    record: keep a trace of every decision, ("commit", positions),
    ("skip",) and ("lookahead", pivot, token or -1), at the cost of one more
    read-back per standard commit.
    packed: run each lookahead as one packed sequence [x || block copies] with
    the branch-isolating mask (dllm_forward_packed) instead of a batch of
    1 + n full sequences; block must then be a power of two.
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
    bt = torch.empty(capacity, S, dtype=torch.int32, device=dev)
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
    ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) if timing else None

    def fwd(tok, n, out, probe=None, kind="normal", nb=0):
        if ev:
            ev[0].record()
        if kind == "packed":
            model.forward_packed(tok, S, b0, block, nb, m_pos, out=out, n_lm_pos=n,
                                 row_scale=row_scale, scale=scale, probe=probe)
        else:
            model.forward(tok, m_pos, out=out, n_lm_pos=n, row_scale=row_scale, scale=scale, probe=probe)
        st.nfe += 1
        if kind == "normal":
            st.normal += 1
        else:
            st.lookahead += 1
            kind = "lookahead"
        if ev:
            ev[1].record()
            ev[1].synchronize()
            ms = ev[0].elapsed_time(ev[1])
            if kind == "normal":
                st.normal_ms += ms
            else:
                st.lookahead_ms += ms

    for b in range(gen_len // block):
        b0 = P + b * block
        m_pos = torch.arange(b0, b0 + block, dtype=torch.int32, device=dev)
        n_m = block
        fwd(tokens[None], n_m, base)                                     # block-opening forward
        while n_m > 0:
            B.rps_commit(tokens, m_pos, n_m, base, tau, n_m_out, committed, n_committed)   # standard commit
            n_new = int(n_m_out.item())
            st.commits_conf += n_m - n_new
            if record:
                st.trace.append(("commit", sorted(committed[:n_m - n_new].tolist())))
            n_m = n_new
            if n_m == 0:
                break
            B.rps_select_pivots(base, m_pos, n_m, prm, plan)
            nb = B.read_plan(plan).n_branch
            if nb == 0:                                                  # skip rules: normal forward
                fwd(tokens[None], n_m, base)
                st.trace.append(("skip",))
                continue
            probe = Probe(B.plan_field_ptr(plan, "br_row"), B.plan_field_ptr(plan, "br_token"),
                          anchor_logit.data_ptr(), nb)
            if packed:
                B.rps_build_packed(tokens, plan, b0, block, nb, pk)
                fwd(pk[:S + nb * block], n_m, branch, probe=probe, kind="packed", nb=nb)
            else:
                B.rps_build_branches(tokens, plan, True, 1 + nb, bt)
                fwd(bt[:1 + nb], n_m, branch, probe=probe, kind="lookahead")
            anchor = branch.rows(0, n_m)
            B.rps_lookahead_score(anchor, branch, 1, n_m, plan, lam, dec, anchor_logit=anchor_logit)
            B.rps_commit(tokens, m_pos, n_m, base, -1.0, n_m_out, committed, n_committed, dec=dec,
                         branches=branch, branch_offset=1, anchor=anchor)
            n_new = int(n_m_out.item())
            if record:
                d = B.read_decision(dec)
                st.trace.append(("lookahead", d.pivot_pos, d.token if d.commit else -1))
            if n_new < n_m:
                st.commits_pivot += 1
            else:
                st.abstains += 1
            n_m = n_new
    return tokens, st


_SCHED_RULES = {"confidence": _abi.SCHED_TOP_CONFIDENCE, "entropy": _abi.SCHED_LOW_ENTROPY}


def baseline_decode(model, prompt, gen_len: int, block: int, rule: str, k: int = 1, tau: float = 0.9,
                    row_scale=None, scale: float = 1.0, topk: int = 16, timing: bool = False,
                    record: bool = False):
    """The semi-autoregressive baselines of Section 3 (Eq. 1 and 2) on the GPU.

    Blocks left to right; every step is one forward over the sequence and one
    commit of S with greedy tokens: the k most confident masked positions
    (rule "confidence"; k = 1 is the Default decoder), the k lowest-entropy
    ones (rule "entropy", sched_commit), or every position with P^max >= tau
    and else the most confident one (rule "threshold", rps_commit without a
    lookahead decision: the Confidence baseline).  Returns (tokens, DecodeStats);
    record keeps ("commit", positions) per step.
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
    ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) if timing else None
    for b in range(gen_len // block):
        m_pos = torch.arange(P + b * block, P + (b + 1) * block, dtype=torch.int32, device=dev)
        n_m = block
        while n_m > 0:
            if ev:
                ev[0].record()
            model.forward(tokens[None], m_pos, out=base, n_lm_pos=n_m, row_scale=row_scale, scale=scale)
            st.nfe += 1
            st.normal += 1
            if ev:
                ev[1].record()
                ev[1].synchronize()
                st.normal_ms += ev[0].elapsed_time(ev[1])
            if rule == "threshold":
                B.rps_commit(tokens, m_pos, n_m, base, tau, n_m_out, committed, n_committed)
            else:
                B.sched_commit(tokens, m_pos, n_m, base, _SCHED_RULES[rule], k, n_m_out, committed, n_committed)
            n_new = int(n_m_out.item())
            st.commits_conf += n_m - n_new
            if record:
                st.trace.append(("commit", sorted(committed[:n_m - n_new].tolist())))
            n_m = n_new
    return tokens, st

