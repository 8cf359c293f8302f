"""Oracle of the RPS decoding loop (Algorithm 1, Appendix A).

``forward(batch_tokens, m_pos)`` is any model: it returns, for every sequence
of the batch, (Stats over rows m_pos, log p of requested tokens at rows).
The loop itself only follows Algorithm 1:

  for each block b (left to right):
      block-opening forward; M <- masked positions of block b
      while M is not empty:
          standard (confidence-aware) commit of S, fallback to the most
          confident position; M <- M minus S; stop the block if M is empty
          pivot selection (Eq. 3); if infeasible: normal forward, continue
          candidate set; if at most one real candidate: normal forward, continue
          lookahead forward over [anchor, branch_1, ..., branch_n]
          Eq. 4 decision; commit c* at i* and carry the winner's
          distributions, or abstain and carry the anchor's

Every forward is counted (NFE), split into normal and lookahead passes as in
the paper's speedup decomposition (Table 4).  The trace records every
decision with its margin (distance of the deciding value from its boundary):
("commit", positions, margin), ("skip", margin), ("lookahead", pivot, token
or -1 for abstain, margin).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import rps


@dataclass
class DecodeResult:
    tokens: np.ndarray
    nfe: int = 0
    normal: int = 0
    lookahead: int = 0
    commits_conf: int = 0
    commits_pivot: int = 0
    abstains: int = 0
    trace: list = field(default_factory=list)


def rps_decode(forward, prompt, gen_len: int, block: int, mask_id: int, prm: rps.Params,
               lam: float, tau: float, capacity: int = 16, max_iters: int = 100000,
               lookahead=None, block_forward=None) -> DecodeResult:
    """lookahead: optional model for the lookahead forward,
    ``lookahead(batch_tokens, m_pos, probe, block_start, block_len)`` with the
    return of ``forward`` (e.g. a packed forward, which may use that every
    branch differs from the anchor inside the current block only).
    block_forward: optional ``block_forward(tokens, block_start)``, called at
    every block opening, that returns the model used for every later forward
    of that block (e.g. a prefix-cached model built from the opening state),
    or a pair (that model, a lookahead model as ``lookahead`` above) when the
    lookahead of the block has a model of its own (packed over the cache)."""
    import dataclasses
    if lookahead is not None and block_forward is not None:
        raise ValueError("pass the lookahead of a block model through block_forward")
    prm = dataclasses.replace(prm, max_branch=min(prm.max_branch, capacity - 1))   # slot 0: anchor
    prompt = np.asarray(prompt, dtype=np.int64)
    P = len(prompt)
    tokens = np.concatenate([prompt, np.full(gen_len, mask_id, dtype=np.int64)])
    res = DecodeResult(tokens=tokens)
    iters = 0
    for b in range(gen_len // block):
        m_pos = np.arange(P + b * block, P + (b + 1) * block)
        m_pos = m_pos[tokens[m_pos] == mask_id]
        stats = forward(tokens[None, :], m_pos, None)[0][0]
        res.nfe += 1
        res.normal += 1
        fb = None if block_forward is None else block_forward(tokens.copy(), P + b * block)
        fwd_b, look_b = fb if isinstance(fb, tuple) else (fb or forward, lookahead)
        state = rps.State(tokens, m_pos, stats)
        while len(state.m_pos) > 0:
            iters += 1
            assert iters <= max_iters
            committed, cmargin = rps.apply_confidence_commit(state, tau, mask_id)
            res.commits_conf += len(committed)
            res.trace.append(("commit", sorted(int(c) for c in committed), cmargin))
            if len(state.m_pos) == 0:
                break
            plan = rps.select_pivots(state.stats, state.m_pos, prm)
            plan.pivots = plan.pivots[:1]
            brs = plan.branches()
            if not brs:
                state.stats = fwd_b(state.tokens[None, :], state.m_pos, None)[0][0]
                res.nfe += 1
                res.normal += 1
                res.trace.append(("skip", plan.empty_margin))
                continue
            pv = plan.pivots[0]
            batch = rps.branch_tokens(state.tokens, plan, with_anchor=True)
            probe = [(pv.row, t) for t in pv.tokens]
            if look_b is None:
                outs = fwd_b(batch, state.m_pos, probe)
            else:
                outs = look_b(batch, state.m_pos, probe, P + b * block, block)
            res.nfe += 1
            res.lookahead += 1
            anchor, anchor_probe = outs[0]
            branch_stats = [o[0] for o in outs[1:]]
            dec = rps.score(anchor, branch_stats, plan, lam, anchor_logp=anchor_probe)
            pmargin = min(pv.feas_margin, pv.rank_margin, pv.cand_margin, plan.empty_margin)
            res.trace.append(("lookahead", pv.pos, dec.token if dec.commit else -1,
                              min(dec.margin_sum, pmargin)))
            if dec.commit:
                res.commits_pivot += 1
            else:
                res.abstains += 1
            rps.apply_decision(state, dec, branch_stats, anchor)
        tokens = state.tokens
    res.tokens = tokens
    return res


def baseline_decode(forward, prompt, gen_len: int, block: int, mask_id: int, rule: str, k: int = 1,
                    tau: float = 0.9, max_iters: int = 100000, block_forward=None) -> DecodeResult:
    """The semi-autoregressive baselines of Section 3 (Eq. 1 and 2): blocks
    left to right; inside a block every step is one forward over the current
    sequence and a commit of S with greedy tokens, where S is the k most
    confident masked positions (rule "confidence"; k = 1 is the Default
    decoder), the k lowest-entropy ones (rule "entropy"), or every position
    with P^max >= tau and else the most confident one (rule "threshold", the
    Confidence baseline of Fast-dLLM).  Trace: ("commit", positions, margin).
    block_forward: as in ``rps_decode``; the block's first step is the full
    forward, every later step uses the model it returns."""
    prompt = np.asarray(prompt, dtype=np.int64)
    P = len(prompt)
    tokens = np.concatenate([prompt, np.full(gen_len, mask_id, dtype=np.int64)])
    res = DecodeResult(tokens=tokens)
    iters = 0
    for b in range(gen_len // block):
        m_pos = np.arange(P + b * block, P + (b + 1) * block)
        m_pos = m_pos[tokens[m_pos] == mask_id]
        fwd_b = None
        while len(m_pos) > 0:
            iters += 1
            assert iters <= max_iters
            stats = (forward if fwd_b is None else fwd_b)(tokens[None, :], m_pos, None)[0][0]
            if fwd_b is None:
                fb = forward if block_forward is None else block_forward(tokens.copy(), P + b * block)
                fwd_b = fb[0] if isinstance(fb, tuple) else fb
            res.nfe += 1
            res.normal += 1
            state = rps.State(tokens, m_pos, stats)
            if rule == "threshold":
                committed, margin = rps.apply_confidence_commit(state, tau, mask_id)
            else:
                committed, margin = rps.apply_topk_commit(state, rule, k, mask_id)
            res.commits_conf += len(committed)
            res.trace.append(("commit", sorted(int(c) for c in committed), margin))
            tokens, m_pos = state.tokens, state.m_pos
    res.tokens = tokens
    return res


def model_forward(weights, shape, topk: int = 16, scales=None, scale: float = 1.0,
                  mirror: bool = False):
    """Forward callback for ``rps_decode`` backed by the oracle transformer.

    scales: optional per-absolute-position logit scale array (indexed by position).
    """
    from .model import forward_logits
    from .stats import softmax_stats

    def fwd(batch, m_pos, probe):
        rs = None if scales is None else np.asarray(scales)[np.asarray(m_pos)]
        logits = forward_logits(batch, weights, shape, m_pos, mirror=mirror, row_scale=rs, scale=scale)
        out = []
        for b in range(logits.shape[0]):
            st = softmax_stats(logits[b], topk)
            pl = None if probe is None else [float(logits[b][row, tok] - st.lse[row]) for row, tok in probe]
            out.append((st, pl))
        return out
    return fwd


def model_packed_lookahead(weights, shape, topk: int = 16, scales=None, scale: float = 1.0,
                           mirror: bool = False):
    """Lookahead callback for ``rps_decode`` that evaluates the anchor and its
    branches as one packed sequence [x || x_b^(c_1) || ...] with the
    branch-isolating mask (Section 4.1, lookahead scoring; Algorithm 1)."""
    from .model import packed_logits
    from .stats import softmax_stats

    def fwd(batch, m_pos, probe, block_start, block_len):
        batch = np.asarray(batch)
        S, b0, B = batch.shape[1], block_start, block_len
        outside = np.ones(S, dtype=bool)
        outside[b0:b0 + B] = False
        assert np.all(batch[1:, outside] == batch[0, outside]), "branches differ from the anchor outside the block"
        tokens = np.concatenate([batch[0]] + [row[b0:b0 + B] for row in batch[1:]])
        rs = None if scales is None else np.asarray(scales)[np.asarray(m_pos)]
        logits = packed_logits(tokens, weights, shape, S, b0, B, batch.shape[0] - 1, m_pos, mirror=mirror,
                               row_scale=rs, scale=scale)
        out = []
        for c in range(logits.shape[0]):
            st = softmax_stats(logits[c], topk)
            pl = None if probe is None else [float(logits[c][row, tok] - st.lse[row]) for row, tok in probe]
            out.append((st, pl))
        return out
    return fwd



def model_prefix_cached(weights, shape, topk: int = 16, scales=None, scale: float = 1.0,
                        mirror: bool = False, packed: bool = False):
    """Block-forward factory for ``rps_decode`` and ``baseline_decode``: the
    prefix cache the paper combines RPS with (Fast-dLLM's; Section 5.3, KV caching).

    Reading: at a block opening the full forward over the whole sequence also
    yields the per-layer keys and values of every position before the block;
    they are kept, and every later forward of the block runs on the positions
    from the block start to the end of the sequence (the block and the masked
    suffix), attending to those cached keys and values plus its own.  Cached
    rows do not see commits made after the block opened (the approximation).
    packed: the factory returns (forward, lookahead), the lookahead being the
    packed sequence [block + suffix || branch blocks] over the same cache.
    """
    from .model import hidden, lm_logits, packed_logits
    from .stats import softmax_stats

    def stats_of(logits, probe):
        st = softmax_stats(logits, topk)
        pl = None if probe is None else [float(logits[row, tok] - st.lse[row]) for row, tok in probe]
        return st, pl

    def open_block(tokens, block_start):
        kv = []
        hidden(np.asarray(tokens), weights, shape, mirror=mirror, collect=kv)
        ctx = [(k[:, :block_start], v[:, :block_start]) for k, v in kv] if block_start > 0 else None

        def fwd(batch, m_pos, probe):
            m_pos = np.asarray(m_pos)
            rel = m_pos - block_start
            assert np.all(rel >= 0), "LM rows must lie at or after the block start"
            rs = None if scales is None else np.asarray(scales)[m_pos]
            out = []
            for toks in np.asarray(batch):
                h = hidden(toks[block_start:], weights, shape, pos_offset=block_start, mirror=mirror, prefix_kv=ctx)
                out.append(stats_of(lm_logits(h[rel], weights, shape, row_scale=rs, scale=scale), probe))
            return out

        def look(batch, m_pos, probe, b0, B):
            assert b0 == block_start
            batch = np.asarray(batch)
            tail = batch[0, b0:]
            assert np.all(batch[1:, b0 + B:] == tail[B:]), "branches differ from the anchor outside the block"
            tokens = np.concatenate([tail] + [row[b0:b0 + B] for row in batch[1:]])
            m_pos = np.asarray(m_pos)
            rs = None if scales is None else np.asarray(scales)[m_pos]
            logits = packed_logits(tokens, weights, shape, len(tail), 0, B, batch.shape[0] - 1, m_pos - b0,
                                   pos_offset=b0, mirror=mirror, row_scale=rs, scale=scale, prefix_kv=ctx)
            return [stats_of(logits[c], probe) for c in range(logits.shape[0])]

        return (fwd, look) if packed else fwd
    return open_block


# ------------------------------------------------------------ teacher forcing

@dataclass
class ForcedEvent:
    """One decision of a followed trajectory: the oracle's own decision at
    that point (made on the followed state) next to the one applied."""
    kind: str                 # "commit", "skip" or "lookahead"
    oracle: tuple             # the oracle's decision: ("commit", positions), ("skip",) or
                              # ("lookahead", pivot, token or -1)
    applied: tuple            # the followed (applied) decision, same form
    margin: float             # the oracle's decision margin
    token_rows: list = field(default_factory=list)   # (position, oracle argmax, applied token, argmax margin)


def _commit_forced(state: rps.State, positions, tokens):
    """Commit the given positions with the given tokens (the followed
    trajectory's standard commit)."""
    pos = np.asarray(sorted(positions), dtype=np.int64)
    rows = np.nonzero(np.isin(state.m_pos, pos))[0]
    assert rows.size == pos.size, "followed commit names positions outside M"
    state.tokens[pos] = np.asarray([tokens[p] for p in pos], dtype=state.tokens.dtype)
    keep = np.setdiff1d(np.arange(len(state.m_pos)), rows)
    state.m_pos = state.m_pos[keep]
    state.stats = state.stats.rows(keep)


def rps_decode_follow(forward, prompt, gen_len: int, block: int, mask_id: int, prm: rps.Params, lam: float,
                      tau: float, follow, final_tokens, capacity: int = 16, lookahead=None, block_forward=None):
    """Algorithm 1 along a given trajectory (teacher forcing).

    follow: the decisions of another implementation in order, ("commit",
    positions), ("skip",) and ("lookahead", pivot, token or -1);
    final_tokens: its final sequence (the token a commit wrote at each
    position).  At every decision point the oracle makes its own decision on
    the current state (the followed trajectory so far, with the oracle's own
    forwards and carried distributions), records it with its margin, then
    applies the followed decision, so that a near-tie does not change the
    states that later decisions are made on.  Returns the list of
    ForcedEvent."""
    import dataclasses
    prm = dataclasses.replace(prm, max_branch=min(prm.max_branch, capacity - 1))
    prompt = np.asarray(prompt, dtype=np.int64)
    final_tokens = np.asarray(final_tokens, dtype=np.int64)
    P = len(prompt)
    tokens = np.concatenate([prompt, np.full(gen_len, mask_id, dtype=np.int64)])
    follow = list(follow)
    events = []
    it = iter(follow)
    for b in range(gen_len // block):
        m_pos = np.arange(P + b * block, P + (b + 1) * block)
        m_pos = m_pos[tokens[m_pos] == mask_id]
        stats = forward(tokens[None, :], m_pos, None)[0][0]
        fb = None if block_forward is None else block_forward(tokens.copy(), P + b * block)
        fwd_b, look_b = fb if isinstance(fb, tuple) else (fb or forward, lookahead)
        state = rps.State(tokens, m_pos, stats)
        while len(state.m_pos) > 0:
            ev = next(it)
            assert ev[0] == "commit", f"followed trajectory: expected a standard commit, got {ev}"
            rows, toks, cmargin = rps.confidence_commit(state.stats, tau)
            own = ("commit", tuple(sorted(int(state.m_pos[r]) for r in rows)))
            applied = ("commit", tuple(sorted(int(p) for p in ev[1])))
            # greedy tokens (Eq. 1) at the positions both sides commit
            both = set(own[1]) & set(applied[1])
            trow = [(int(state.m_pos[r]), int(state.stats.argmax[r]), int(final_tokens[state.m_pos[r]]),
                     float(state.stats.argmax_margin[r]) if state.stats.argmax_margin is not None else np.inf)
                    for r in range(len(state.m_pos)) if int(state.m_pos[r]) in both]
            events.append(ForcedEvent("commit", own, applied, cmargin, trow))
            _commit_forced(state, applied[1], final_tokens)
            if len(state.m_pos) == 0:
                break
            ev = next(it)
            plan = rps.select_pivots(state.stats, state.m_pos, prm)
            plan.pivots = plan.pivots[:1]
            brs = plan.branches()
            if brs:
                pv = plan.pivots[0]
                batch = rps.branch_tokens(state.tokens, plan, with_anchor=True)
                probe = [(pv.row, t) for t in pv.tokens]
                outs = fwd_b(batch, state.m_pos, probe) if look_b is None else \
                    look_b(batch, state.m_pos, probe, P + b * block, block)
                anchor, anchor_probe = outs[0]
                branch_stats = [o[0] for o in outs[1:]]
                dec = rps.score(anchor, branch_stats, plan, lam, anchor_logp=anchor_probe)
                pmargin = min(pv.feas_margin, pv.rank_margin, pv.cand_margin, plan.empty_margin)
                own = ("lookahead", pv.pos, dec.token if dec.commit else -1)
                margin = min(dec.margin_sum, pmargin)
            else:
                own, margin = ("skip",), plan.empty_margin
            applied = tuple(ev)
            events.append(ForcedEvent(own[0], own, applied, margin))
            if applied[0] == "skip":
                state.stats = fwd_b(state.tokens[None, :], state.m_pos, None)[0][0]
                continue
            assert applied[0] == "lookahead", applied
            _, piv, tok = applied
            prow = int(np.nonzero(state.m_pos == piv)[0][0])
            # the followed lookahead's anchor and, on a commit, its winning
            # branch, evaluated by the oracle as one lookahead batch
            fplan = rps.Plan([rps.Pivot(row=prow, pos=int(piv), tokens=[int(tok)] if tok >= 0 else [],
                                        logp=[0.0] if tok >= 0 else [])])
            fbatch = rps.branch_tokens(state.tokens, fplan, with_anchor=True)
            if tok >= 0 and brs and plan.pivots[0].pos == piv and int(tok) in plan.pivots[0].tokens:
                win = branch_stats[plan.pivots[0].tokens.index(int(tok))]
            elif tok < 0 and brs:
                pass                                 # the anchor of the oracle's own lookahead
            else:
                fouts = fwd_b(fbatch, state.m_pos, None) if look_b is None else \
                    look_b(fbatch, state.m_pos, None, P + b * block, block)
                anchor = fouts[0][0]
                win = fouts[1][0] if tok >= 0 else None
            if tok >= 0:
                state.tokens[piv] = tok
                keep = np.array([j for j in range(len(state.m_pos)) if j != prow], dtype=np.int64)
                state.m_pos = state.m_pos[keep]
                state.stats = win.rows(keep)
            else:
                state.stats = anchor.rows(np.arange(len(anchor)))
        tokens = state.tokens
    assert next(it, None) is None, "followed trajectory has more decisions than the oracle's loop"
    return events


def baseline_decode_follow(forward, prompt, gen_len: int, block: int, mask_id: int, rule: str, k: int, tau: float,
                           follow, final_tokens, block_forward=None):
    """The baseline schedulers (Eq. 2) along a given trajectory of
    ("commit", positions) steps: each step the oracle makes its own commit on
    the followed state, records it with its margin, and applies the followed
    commit.  Returns the list of ForcedEvent."""
    prompt = np.asarray(prompt, dtype=np.int64)
    final_tokens = np.asarray(final_tokens, dtype=np.int64)
    P = len(prompt)
    tokens = np.concatenate([prompt, np.full(gen_len, mask_id, dtype=np.int64)])
    it = iter(list(follow))
    events = []
    for b in range(gen_len // block):
        m_pos = np.arange(P + b * block, P + (b + 1) * block)
        m_pos = m_pos[tokens[m_pos] == mask_id]
        fwd_b = None
        while len(m_pos) > 0:
            stats = (forward if fwd_b is None else fwd_b)(tokens[None, :], m_pos, None)[0][0]
            if fwd_b is None:
                fb = forward if block_forward is None else block_forward(tokens.copy(), P + b * block)
                fwd_b = fb[0] if isinstance(fb, tuple) else fb
            state = rps.State(tokens, m_pos, stats)
            if rule == "threshold":
                rows, _, margin = rps.confidence_commit(stats, tau)
            else:
                rows, _, margin = rps.topk_commit(stats, rule, k)
            own = ("commit", tuple(sorted(int(m_pos[r]) for r in rows)))
            ev = next(it)
            applied = ("commit", tuple(sorted(int(p) for p in ev[1])))
            both = set(own[1]) & set(applied[1])
            trow = [(int(m_pos[r]), int(stats.argmax[r]), int(final_tokens[m_pos[r]]),
                     float(stats.argmax_margin[r]) if stats.argmax_margin is not None else np.inf)
                    for r in range(len(m_pos)) if int(m_pos[r]) in both]
            events.append(ForcedEvent("commit", own, applied, margin, trow))
            _commit_forced(state, applied[1], final_tokens)
            tokens, m_pos = state.tokens, state.m_pos
    assert next(it, None) is None, "followed trajectory has more steps than the oracle's loop"
    return events
