"""Pins of the oracle decoding loop (Algorithm 1)."""
import json
import os

import numpy as np
import pytest

import synth
from oracle import rps
from oracle.decode import rps_decode, model_forward, model_packed_lookahead, model_prefix_cached
from oracle.stats import softmax_stats

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def scripted_model(vocab, scale_of_pos, seed=0):
    """A deterministic stand-in model: logits are a hash of (sequence, position)."""
    def fwd(batch, m_pos, probe):
        out = []
        for toks in batch:
            key = hash((tuple(int(t) for t in toks), seed)) % (2 ** 32)
            rng = np.random.default_rng(key)
            logits = rng.normal(0, 1, (len(m_pos), vocab)) * np.array([scale_of_pos(p) for p in m_pos])[:, None]
            logits[:, vocab - 1] = -np.inf
            st = softmax_stats(logits, 16)
            pl = None if probe is None else [float(logits[r, t] - st.lse[r]) for r, t in probe]
            out.append((st, pl))
        return out
    return fwd


def test_default_decoder_takes_one_forward_per_token():
    g = json.load(open(os.path.join(GOLDEN, "default_decoder_nfe.json")))
    V = 50
    fwd = scripted_model(V, lambda p: 1.0)
    prompt = np.arange(8)
    # confidence threshold above 1 and an unreachable pivot mass: one commit per forward
    res = rps_decode(fwd, prompt, g["gen_len"], g["block"], V - 1,
                     rps.Params(mode="paper", tau_pivot=2.0), lam=0.1, tau=2.0)
    assert res.nfe == g["nfe"]
    assert res.lookahead == 0
    assert np.all(res.tokens[8:] != V - 1)


def _check_trace(res, prompt_len, gen_len, block, mask_id):
    assert np.all(res.tokens[prompt_len:] != mask_id)
    assert res.commits_conf + res.commits_pivot == gen_len


def test_monotone_commits_and_termination_scripted():
    V = 40
    fwd = scripted_model(V, lambda p: 1.0 + 7.0 * ((p * 2654435761) % 97) / 97.0)
    prompt = np.arange(6)
    res = rps_decode(fwd, prompt, 48, 16, V - 1,
                     rps.Params(mode="paper", tau_pivot=0.5, k_max=5, r=0.1, n_cand=5), lam=0.2, tau=0.9)
    _check_trace(res, 6, 48, 16, V - 1)
    assert res.lookahead > 0


class RecordingModel:
    """Wraps a forward callback and records every sequence it sees."""

    def __init__(self, fwd):
        self.fwd = fwd
        self.seen = []

    def __call__(self, batch, m_pos, probe):
        self.seen.append((np.array(batch[0]), np.array(m_pos)))
        return self.fwd(batch, m_pos, probe)


def test_tiny_model_decode_invariants():
    shape = synth.TINY
    w = synth.model_weights_np(shape, seed=0, dtype="f32")
    P, G, B = 16, 32, 16
    prompt = synth.tokens_np(1, "prompt", P, shape.vocab - 1)
    scales = synth.position_scales_np(2, np.arange(P + G), 2.6, 16.0)
    rec = RecordingModel(model_forward(w, shape, scales=scales))
    prm = rps.Params(mode="paper", k_max=10, tau_pivot=0.9, r=0.1, n_cand=10)
    res = rps_decode(rec, prompt, G, B, shape.mask_id, prm, lam=0.1, tau=0.9)
    _check_trace(res, P, G, B, shape.mask_id)
    # masked count never increases; committed tokens never change; prompt untouched
    prev = None
    for toks, m_pos in rec.seen:
        assert np.array_equal(toks[:P], prompt)
        masked = toks[P:] == shape.mask_id
        if prev is not None:
            assert masked.sum() <= prev[0].sum()
            committed = ~prev[0]
            assert np.array_equal(toks[P:][committed], prev[1][committed])
        prev = (masked, toks[P:])
    # every iteration commits at least one position: at most B forwards per block
    assert res.nfe <= G
    assert res.nfe == res.normal + res.lookahead
    assert res.lookahead + res.abstains >= 0


def test_packed_lookahead_one_layer_takes_the_unpacked_decisions():
    # With one layer the packed forward equals the batch of full branch
    # sequences (up to summation order), so Algorithm 1 takes the same path.
    shape = synth.ModelShape(n_layers=1, d_model=64, n_heads=4, head_dim=16, d_ffn=96, vocab=101)
    w = synth.model_weights_np(shape, seed=4, dtype="f32")
    P, G, B = 8, 32, 16
    prompt = synth.tokens_np(3, "prompt", P, shape.vocab - 1)
    scales = synth.position_scales_np(4, np.arange(P + G), 2.6, 16.0)
    prm = rps.Params(mode="paper", k_max=8, tau_pivot=0.5, r=0.05, n_cand=8)
    fwd = model_forward(w, shape, scales=scales)
    a = rps_decode(fwd, prompt, G, B, shape.mask_id, prm, lam=0.1, tau=0.9)
    b = rps_decode(fwd, prompt, G, B, shape.mask_id, prm, lam=0.1, tau=0.9,
                   lookahead=model_packed_lookahead(w, shape, scales=scales))
    assert a.lookahead > 0
    assert np.array_equal(a.tokens, b.tokens)
    assert [t[:-1] for t in a.trace] == [t[:-1] for t in b.trace]          # decisions; margins last
    for ta, tb in zip(a.trace, b.trace):
        assert ta[-1] == tb[-1] or abs(ta[-1] - tb[-1]) < 1e-9   # margins agree to rounding


def test_packed_lookahead_decode_invariants():
    shape = synth.TINY
    w = synth.model_weights_np(shape, seed=0, dtype="f32")
    P, G, B = 16, 32, 16
    prompt = synth.tokens_np(1, "prompt", P, shape.vocab - 1)
    scales = synth.position_scales_np(2, np.arange(P + G), 2.6, 16.0)
    prm = rps.Params(mode="paper", k_max=10, tau_pivot=0.9, r=0.1, n_cand=10)
    res = rps_decode(model_forward(w, shape, scales=scales), prompt, G, B, shape.mask_id, prm, lam=0.1, tau=0.9,
                     lookahead=model_packed_lookahead(w, shape, scales=scales))
    _check_trace(res, P, G, B, shape.mask_id)
    assert res.nfe == res.normal + res.lookahead and res.nfe <= G


def test_prefix_cached_forward_on_the_opening_tokens_is_the_full_forward():
    # The cache holds the full forward's own keys and values, so a cached
    # forward over unchanged tokens reproduces the full forward at any depth.
    shape = synth.ModelShape(n_layers=2, d_model=64, n_heads=4, head_dim=16, d_ffn=96, vocab=101)
    w = synth.model_weights_np(shape, seed=5, dtype="f32")
    toks = synth.tokens_np(6, "t", 40, shape.vocab - 1)
    toks[24:] = shape.mask_id
    m_pos = np.arange(24, 32)
    full = model_forward(w, shape)(toks[None], m_pos, [(1, 7)])
    cached = model_prefix_cached(w, shape)(toks, 24)(toks[None], m_pos, [(1, 7)])
    assert np.allclose(full[0][0].H, cached[0][0].H, atol=1e-10)
    assert np.allclose(full[0][0].lse, cached[0][0].lse, atol=1e-10)
    assert np.array_equal(full[0][0].topk_id, cached[0][0].topk_id)
    assert abs(full[0][1][0] - cached[0][1][0]) < 1e-10
    # after a commit inside the block the cached rows are stale: outputs differ
    t2 = toks.copy()
    t2[24] = 5
    a = model_forward(w, shape)(t2[None], m_pos[1:], None)[0][0]
    b = model_prefix_cached(w, shape)(toks, 24)(t2[None], m_pos[1:], None)[0][0]
    assert not np.allclose(a.H, b.H, atol=1e-8)


@pytest.mark.parametrize("decoder", ["rps", "confidence", "threshold"])
def test_prefix_cache_with_one_layer_changes_nothing(decoder):
    # With one layer every cached key and value depends on its own token and
    # position only, so the cache is exact and the decode takes the same path.
    shape = synth.ModelShape(n_layers=1, d_model=64, n_heads=4, head_dim=16, d_ffn=96, vocab=101)
    w = synth.model_weights_np(shape, seed=7, dtype="f32")
    P, G, B = 8, 48, 16
    prompt = synth.tokens_np(8, "prompt", P, shape.vocab - 1)
    scales = synth.position_scales_np(9, np.arange(P + G), 2.6, 16.0)
    fwd = model_forward(w, shape, scales=scales)
    cache = model_prefix_cached(w, shape, scales=scales)
    if decoder == "rps":
        prm = rps.Params(mode="paper", k_max=8, tau_pivot=0.5, r=0.05, n_cand=8)
        a = rps_decode(fwd, prompt, G, B, shape.mask_id, prm, lam=0.1, tau=0.9)
        b = rps_decode(fwd, prompt, G, B, shape.mask_id, prm, lam=0.1, tau=0.9, block_forward=cache)
        assert a.lookahead > 0
    else:
        from oracle.decode import baseline_decode
        k, tau = (2, 0.0) if decoder == "confidence" else (1, 0.6)
        a = baseline_decode(fwd, prompt, G, B, shape.mask_id, decoder, k, tau=tau)
        b = baseline_decode(fwd, prompt, G, B, shape.mask_id, decoder, k, tau=tau, block_forward=cache)
    assert np.array_equal(a.tokens, b.tokens) and a.nfe == b.nfe
    assert [t[:-1] for t in a.trace] == [t[:-1] for t in b.trace]


def test_prefix_cached_decode_invariants():
    shape = synth.TINY
    w = synth.model_weights_np(shape, seed=0, dtype="f32")
    P, G, B = 16, 64, 32
    prompt = synth.tokens_np(1, "prompt", P, shape.vocab - 1)
    scales = synth.position_scales_np(2, np.arange(P + G), 2.6, 16.0)
    prm = rps.Params(mode="paper", k_max=10, tau_pivot=0.9, r=0.1, n_cand=10)
    res = rps_decode(model_forward(w, shape, scales=scales), prompt, G, B, shape.mask_id, prm, lam=0.1, tau=0.9,
                     block_forward=model_prefix_cached(w, shape, scales=scales))
    _check_trace(res, P, G, B, shape.mask_id)
    assert res.nfe == res.normal + res.lookahead and res.nfe <= G


def test_packed_lookahead_over_the_cache_with_one_layer_is_exact():
    # one layer: the cache and the packing are both exact, so the packed cached
    # decode takes the plain decode's path
    shape = synth.ModelShape(n_layers=1, d_model=64, n_heads=4, head_dim=16, d_ffn=96, vocab=101)
    w = synth.model_weights_np(shape, seed=4, dtype="f32")
    P, G, B = 8, 32, 16
    prompt = synth.tokens_np(3, "prompt", P, shape.vocab - 1)
    scales = synth.position_scales_np(4, np.arange(P + G), 2.6, 16.0)
    prm = rps.Params(mode="paper", k_max=8, tau_pivot=0.5, r=0.05, n_cand=8)
    fwd = model_forward(w, shape, scales=scales)
    a = rps_decode(fwd, prompt, G, B, shape.mask_id, prm, lam=0.1, tau=0.9)
    b = rps_decode(fwd, prompt, G, B, shape.mask_id, prm, lam=0.1, tau=0.9,
                   block_forward=model_prefix_cached(w, shape, scales=scales, packed=True))
    assert a.lookahead > 0
    assert np.array_equal(a.tokens, b.tokens)
    assert [t[:-1] for t in a.trace] == [t[:-1] for t in b.trace]


def test_packed_lookahead_over_the_cache_decode_invariants():
    shape = synth.TINY
    w = synth.model_weights_np(shape, seed=0, dtype="f32")
    P, G, B = 16, 64, 32
    prompt = synth.tokens_np(1, "prompt", P, shape.vocab - 1)
    scales = synth.position_scales_np(2, np.arange(P + G), 2.6, 16.0)
    prm = rps.Params(mode="paper", k_max=10, tau_pivot=0.9, r=0.1, n_cand=10)
    res = rps_decode(model_forward(w, shape, scales=scales), prompt, G, B, shape.mask_id, prm, lam=0.1, tau=0.9,
                     block_forward=model_prefix_cached(w, shape, scales=scales, packed=True))
    _check_trace(res, P, G, B, shape.mask_id)
    assert res.nfe == res.normal + res.lookahead and res.nfe <= G


# ------------------------------------------------------------ teacher forcing

from oracle.decode import rps_decode_follow, baseline_decode, baseline_decode_follow  # noqa: E402

_F_SHAPE = synth.ModelShape(n_layers=2, d_model=64, n_heads=4, head_dim=16, d_ffn=96, vocab=101)


def _own_key(e):
    return ("commit", tuple(e[1])) if e[0] == "commit" else tuple(e[:-1])


@pytest.mark.parametrize("variant", ["plain", "packed", "prefix_cache"])
def test_following_its_own_trajectory_reproduces_every_decision(variant):
    w = synth.model_weights_np(_F_SHAPE, seed=7, dtype="f32")
    P, G, B = 8, 32, 16
    prompt = synth.tokens_np(8, "prompt", P, _F_SHAPE.vocab - 1)
    scales = synth.position_scales_np(9, np.arange(P + G), 2.6, 16.0)
    prm = rps.Params(mode="paper", k_max=8, tau_pivot=0.5, r=0.05, n_cand=8)
    fwd = model_forward(w, _F_SHAPE, scales=scales)
    kw = {}
    if variant == "packed":
        kw["lookahead"] = model_packed_lookahead(w, _F_SHAPE, scales=scales)
    elif variant == "prefix_cache":
        kw["block_forward"] = model_prefix_cached(w, _F_SHAPE, scales=scales)
    res = rps_decode(fwd, prompt, G, B, _F_SHAPE.mask_id, prm, lam=0.1, tau=0.9, **kw)
    follow = [("commit", t[1]) if t[0] == "commit" else (("skip",) if t[0] == "skip" else tuple(t[:-1]))
              for t in res.trace]
    ev = rps_decode_follow(fwd, prompt, G, B, _F_SHAPE.mask_id, prm, 0.1, 0.9, follow, res.tokens, **kw)
    assert res.lookahead > 0
    assert len(ev) == len(res.trace)
    for e, t in zip(ev, res.trace):
        assert e.oracle == e.applied
        assert e.oracle == _own_key(t)
        assert e.margin == t[-1]
        assert all(own == app for _, own, app, _ in e.token_rows)


def test_following_another_trajectory_records_the_differences():
    # a valid trajectory of a differently scaled model, followed with the
    # original: the follower takes every step of it (its own decision may
    # differ, the applied one is the other's) and finishes the sequence
    w = synth.model_weights_np(_F_SHAPE, seed=7, dtype="f32")
    P, G, B = 8, 32, 16
    prompt = synth.tokens_np(8, "prompt", P, _F_SHAPE.vocab - 1)
    scales = synth.position_scales_np(9, np.arange(P + G), 2.6, 16.0)
    prm = rps.Params(mode="paper", k_max=8, tau_pivot=0.5, r=0.05, n_cand=8)
    other = rps_decode(model_forward(w, _F_SHAPE, scales=scales * 1.3), prompt, G, B, _F_SHAPE.mask_id, prm,
                       lam=0.1, tau=0.9)
    follow = [("commit", t[1]) if t[0] == "commit" else (("skip",) if t[0] == "skip" else tuple(t[:-1]))
              for t in other.trace]
    fwd = model_forward(w, _F_SHAPE, scales=scales)
    ev = rps_decode_follow(fwd, prompt, G, B, _F_SHAPE.mask_id, prm, 0.1, 0.9, follow, other.tokens)
    assert len(ev) == len(other.trace)
    assert [e.applied for e in ev] == [("commit", tuple(f[1])) if f[0] == "commit" else tuple(f) for f in follow]
    assert any(e.oracle != e.applied for e in ev)
    # the first decision is made on the same state by both and differs only if the models disagree
    own = rps_decode(fwd, prompt, G, B, _F_SHAPE.mask_id, prm, lam=0.1, tau=0.9)
    assert ev[0].oracle == _own_key(own.trace[0])


@pytest.mark.parametrize("rule,k,tau", [("confidence", 2, 0.0), ("entropy", 3, 0.0), ("threshold", 1, 0.6)])
def test_baseline_following_its_own_trajectory(rule, k, tau):
    w = synth.model_weights_np(_F_SHAPE, seed=7, dtype="f32")
    P, G, B = 8, 32, 16
    prompt = synth.tokens_np(8, "prompt", P, _F_SHAPE.vocab - 1)
    scales = synth.position_scales_np(9, np.arange(P + G), 2.6, 16.0)
    fwd = model_forward(w, _F_SHAPE, scales=scales)
    res = baseline_decode(fwd, prompt, G, B, _F_SHAPE.mask_id, rule, k, tau=tau)
    ev = baseline_decode_follow(fwd, prompt, G, B, _F_SHAPE.mask_id, rule, k, tau,
                                [("commit", t[1]) for t in res.trace], res.tokens)
    assert len(ev) == len(res.trace)
    for e, t in zip(ev, res.trace):
        assert e.oracle == e.applied == ("commit", tuple(t[1])) and e.margin == t[2]
