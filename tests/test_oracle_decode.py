"""Pins of the oracle decoding loop (Algorithm 1)."""
import json
import os

import numpy as np
import pytest

import synth
from oracle import rps
from oracle.decode import rps_decode, model_forward, model_packed_lookahead
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
