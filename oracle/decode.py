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
