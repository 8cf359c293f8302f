"""Pins of the oracle's baseline schedulers (Section 3, Eq. 1 and 2): the
Default decoder's NFE printed in Table 1, the closed-form step count of the
top-k rules, brute-force ranking of every committed set from the raw logits,
planted ties, and the threshold rule against Algorithm 1 with pivots off."""
import json
import math
import os

import numpy as np
import pytest
from scipy.special import softmax
from scipy.stats import entropy

from oracle import rps
from oracle.decode import baseline_decode, rps_decode
from oracle.stats import softmax_stats

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def scripted(vocab, scale_of_pos, seed=0, log=None):
    """Deterministic stand-in model: logits are a hash of (sequence, position);
    `log` collects (tokens, m_pos, logits) of every call."""
    def fwd(batch, m_pos, probe):
        out = []
        for toks in batch:
            key = hash((tuple(int(t) for t in toks), seed)) % (2 ** 32)
            rng = np.random.default_rng(key)
            logits = rng.normal(0, 1, (len(m_pos), vocab)) * np.array([scale_of_pos(p) for p in m_pos])[:, None]
            logits[:, vocab - 1] = -np.inf
            if log is not None:
                log.append((np.array(toks), np.array(m_pos), logits.copy()))
            out.append((softmax_stats(logits, 16), None))
        return out
    return fwd


def test_default_decoder_nfe_matches_table_1():
    """k = 1 highest-confidence decoding commits one token per forward: NFE = L
    (Table 1, Default, NFE 256.0 at generation length 256)."""
    g = json.load(open(os.path.join(GOLDEN, "default_decoder_nfe.json")))
    V = 50
    res = baseline_decode(scripted(V, lambda p: 1.0), np.arange(8), g["gen_len"], g["block"], V - 1, "confidence", 1)
    assert res.nfe == g["nfe"]
    assert np.all(res.tokens[8:] != V - 1)


@pytest.mark.parametrize("rule", ["confidence", "entropy"])
@pytest.mark.parametrize("k", [1, 2, 3, 5, 16, 40])
def test_topk_step_count_closed_form(rule, k):
    """Each step commits min(k, |M|) positions, so a block of B takes ceil(B / k) forwards."""
    V, L, Bk = 30, 48, 16
    res = baseline_decode(scripted(V, lambda p: 0.5 + (p % 7) / 3), np.arange(5), L, Bk, V - 1, rule, k)
    assert res.nfe == (L // Bk) * math.ceil(Bk / k)
    assert all(len(t[1]) == min(k, Bk - (i % math.ceil(Bk / k)) * k) for i, t in enumerate(res.trace))


@pytest.mark.parametrize("rule,k", [("confidence", 3), ("entropy", 4), ("threshold", 0)])
def test_every_commit_is_the_brute_force_selection(rule, k):
    """Rank the masked positions of every step from the raw logits with scipy
    (max softmax probability, Shannon entropy) and check the committed set."""
    V, tau = 40, 0.35
    log = []
    scale = lambda p: [0.3, 1.0, 2.5, 4.0][p % 4]   # a spread of confidences, some above tau
    res = baseline_decode(scripted(V, scale, seed=3, log=log), np.arange(6), 32, 16, V - 1, rule, k, tau=tau)
    assert len(log) == res.nfe
    for (toks, m_pos, logits), (_, committed, _) in zip(log, res.trace):
        p = softmax(logits, axis=1)
        conf = p.max(axis=1)
        if rule == "threshold":
            want = [int(m_pos[j]) for j in range(len(m_pos)) if conf[j] >= tau]
            if not want:
                want = [int(m_pos[min(range(len(m_pos)), key=lambda j: (-conf[j], m_pos[j]))])]
        else:
            key = conf if rule == "confidence" else -entropy(p, axis=1)
            ranked = sorted(range(len(m_pos)), key=lambda j: (-key[j], m_pos[j]))
            want = [int(m_pos[j]) for j in ranked[:k]]
        assert committed == sorted(want)
        # committed tokens are the greedy predictions (Eq. 1)
        for pos in committed:
            j = int(np.nonzero(m_pos == pos)[0][0])
            assert res.tokens[pos] == int(np.argmax(logits[j]))


def test_ties_go_to_the_lower_position():
    """Identical distributions at every masked position: the k lowest positions commit first."""
    lse = np.full(6, 2.0)
    st = rps.Stats(H=np.full(6, 1.5), lse=lse, lmax=np.full(6, 1.0), argmax=np.arange(6),
                   topk_id=np.zeros((6, 16), dtype=np.int64), topk_logit=np.zeros((6, 16)))
    for rule in ("confidence", "entropy"):
        rows, toks, margin = rps.topk_commit(st, rule, 2)
        assert list(rows) == [0, 1] and margin == 0.0


def test_threshold_rule_is_algorithm_1_without_pivots():
    """The confidence-threshold baseline and Algorithm 1 with an unreachable
    pivot mass take the same commits and forwards."""
    V = 40
    fwd = scripted(V, lambda p: [0.5, 3.0, 6.0][p % 3], seed=7)
    a = baseline_decode(fwd, np.arange(6), 32, 16, V - 1, "threshold", tau=0.6)
    b = rps_decode(fwd, np.arange(6), 32, 16, V - 1, rps.Params(mode="paper", tau_pivot=2.0), lam=0.1, tau=0.6)
    assert a.nfe == b.nfe
    assert np.array_equal(a.tokens, b.tokens)
    assert [t[:2] for t in a.trace] == [t[:2] for t in b.trace if t[0] == "commit"]
