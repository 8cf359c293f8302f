"""Pins of the oracle scheduler: planted distributions, brute force, Propositions 1 and 2."""
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats

import synth
from oracle import model as om
from oracle import rps
from oracle.stats import softmax_stats, confidence

V = 64
MASK = V - 1


def planted(rows):
    """Stats of rows given as {token: probability} dicts (remaining mass spread uniformly)."""
    logits = np.full((len(rows), V), -np.inf)
    for i, row in enumerate(rows):
        rest = 1.0 - sum(row.values())
        free = [v for v in range(V - 1) if v not in row]
        for v in free:
            logits[i, v] = math.log(rest / len(free)) if rest > 0 else -np.inf
        for v, p in row.items():
            logits[i, v] = math.log(p)
    return softmax_stats(logits, 16)


# ------------------------------------------------------------ standard commit

def dyadic(rows, k=16):
    """Stats built directly from exact probabilities (lse = 0, logit = log p):
    every p used here is a dyadic rational whose exp(log p) round-trips exactly,
    so a value placed on a threshold sits exactly on it."""
    n = len(rows)
    tid = np.zeros((n, k), dtype=np.int64)
    tl = np.full((n, k), -np.inf)
    for i, row in enumerate(rows):
        items = sorted(row.items(), key=lambda kv: (-kv[1], kv[0]))
        for j, (v, p) in enumerate(items):
            assert math.exp(math.log(p)) == p, p
            tid[i, j], tl[i, j] = v, math.log(p)
        for j in range(len(items), k):
            tid[i, j] = 40 + j                          # tokens of no mass (p = 0)
    z = np.zeros(n)
    return rps.Stats(H=z.copy(), lse=z, lmax=tl[:, 0].copy(), argmax=tid[:, 0].copy(), topk_id=tid, topk_logit=tl)


def test_confidence_commit_threshold_inclusive():
    # rows 0 and 2 sit exactly on tau = 0.5; a strict ">" would commit only the
    # fallback row (one row) instead of both
    st = dyadic([{1: 0.5, 9: 0.25}, {2: 0.375, 9: 0.25}, {3: 0.5, 9: 0.375}, {4: 0.25}])
    assert np.all(confidence(st)[[0, 2]] == 0.5)
    rows, toks, margin = rps.confidence_commit(st, 0.5)
    assert rows.tolist() == [0, 2] and toks.tolist() == [1, 3]
    assert margin == 0.0
    rows, _, _ = rps.confidence_commit(st, 0.75)        # nothing reaches 0.75: fallback, lower row
    assert rows.tolist() == [0]


def test_confidence_commit_fallback_picks_most_confident_lowest_row():
    st = planted([{1: 0.3}, {2: 0.6}, {3: 0.6}, {4: 0.2}])
    rows, toks, _ = rps.confidence_commit(st, 0.9)
    assert rows.tolist() == [1] and toks.tolist() == [2]


# ------------------------------------------------------------ pivot selection

def test_percentile_matches_numpy_linear():
    x = np.random.default_rng(0).normal(size=37)
    for q in (0, 25, 50, 75, 100, 12.5):
        assert math.isclose(rps.percentile_linear(x, q), float(np.percentile(x, q)), rel_tol=0, abs_tol=1e-12)


def test_full_support_truncation_is_full_entropy():
    rng = np.random.default_rng(1)
    logits = rng.normal(0, 2, (5, 20))
    st = softmax_stats(logits, 20)
    mu, htr = rps.truncated(st, 20)
    assert np.allclose(mu, 1.0)
    assert np.allclose(htr, st.H)


def test_no_feasible_pivot_skips():
    st = planted([{1: 0.3, 2: 0.2}] * 5)            # top-10 mass far below 0.9
    plan = rps.select_pivots(st, np.arange(10, 15), rps.Params(mode="paper", tau_pivot=0.9))
    assert plan.pivots == []


def test_single_candidate_skips():
    # feasible (mass >= 0.9) but the runner-up is below r * P^max
    st = planted([{5: 0.95, 6: 0.04}, {7: 0.97, 8: 0.02}])
    plan = rps.select_pivots(st, np.array([3, 4]), rps.Params(mode="paper", tau_pivot=0.9, r=0.1))
    assert plan.pivots == []


def test_pivot_is_max_truncated_entropy_among_feasible():
    st = planted([
        {1: 0.99},                          # feasible, nearly determined
        {2: 0.5, 3: 0.45},                  # feasible, mid entropy  <- pivot
        {4: 0.3, 5: 0.3},                   # infeasible (mass 0.6 + spread)
        {6: 0.8, 7: 0.15},                  # feasible, lower truncated entropy
    ])
    plan = rps.select_pivots(st, np.array([10, 11, 12, 13]), rps.Params(mode="paper", tau_pivot=0.9, r=0.1))
    assert len(plan.pivots) == 1
    pv = plan.pivots[0]
    assert (pv.row, pv.pos) == (1, 11)
    assert pv.tokens == [2, 3]
    assert np.allclose(pv.logp, [math.log(0.5), math.log(0.45)])


def test_candidate_ratio_and_cap():
    st = planted([{1: 0.5, 2: 0.2, 3: 0.06, 4: 0.049, 5: 0.04, 6: 0.04, 7: 0.04}])
    pv = rps.select_pivots(st, np.array([9]), rps.Params(mode="paper", tau_pivot=0.0))
    assert pv.pivots == []                                  # |M| = 1: no pivot search
    st2 = softmax_stats(np.vstack([st_logits_row(st), st_logits_row(st)]), 16)
    plan = rps.select_pivots(st2, np.array([8, 9]), rps.Params(mode="paper", tau_pivot=0.0, r=0.1, n_cand=10))
    assert plan.pivots[0].tokens == [1, 2, 3]               # 0.049 / 0.5 < 0.1
    plan = rps.select_pivots(st2, np.array([8, 9]), rps.Params(mode="paper", tau_pivot=0.0, r=0.0, n_cand=2))
    assert plan.pivots[0].tokens == [1, 2]


def st_logits_row(st):
    row = np.full(V, -np.inf)
    row[st.topk_id[0]] = st.topk_logit[0]
    # remaining tokens share the rest of the mass uniformly
    rest = 1.0 - np.exp(st.topk_logit[0] - st.lse[0]).sum()
    free = [v for v in range(V - 1) if v not in st.topk_id[0]]
    row[free] = math.log(rest / len(free)) + st.lse[0]
    return row


def test_band_mode_picks_mid_entropy_rows():
    rng = np.random.default_rng(2)
    scales = np.linspace(0.2, 6.0, 21)                      # entropy decreases with scale
    logits = rng.normal(0, 1, (21, V)) * scales[:, None]
    logits[:, MASK] = -np.inf
    st = softmax_stats(logits, 16)
    m_pos = np.arange(100, 121)
    prm = rps.Params(mode="band", k_max=10, pct_lo=25, pct_hi=75, n_pivots=3, r=0.0, n_cand=4)
    plan = rps.select_pivots(st, m_pos, prm)
    # expectation from the logits alone: scipy entropies and probabilities,
    # numpy percentiles, and a plain loop over each row's 10 most probable tokens
    p = scipy.special.softmax(logits, axis=1)
    H = scipy.stats.entropy(p, axis=1)
    lo, hi = np.percentile(H, 25), np.percentile(H, 75)
    htr = []
    for j in range(21):
        top = sorted(range(V), key=lambda v: (-p[j, v], v))[:10]
        htr.append(sum(-p[j, v] * math.log(p[j, v]) for v in top))
    band = [j for j in range(21) if lo <= H[j] <= hi]
    expect = sorted(band, key=lambda j: (-htr[j], m_pos[j]))[:3]
    assert [p.row for p in plan.pivots] == expect
    assert all(len(p.tokens) == 4 for p in plan.pivots)
    assert all(p.tokens == st.topk_id[p.row, :4].tolist() for p in plan.pivots)


# Row A keeps mass 0.9 on its top two tokens (0.5, 0.4); row B puts all its mass
# on two tokens (0.5, 0.5).  Eq. 3's objective as printed (p not renormalised
# over T_i) ranks A first: 0.5 ln 2 + 0.4 ln 2.5 = 0.7131 > ln 2.  Renormalised
# over T_i, A would be (5/9, 4/9) with entropy 0.6870 < ln 2, and B would win.
ROW_A = {3: 0.5, 4: 0.4}
ROW_B = {5: 0.5, 6: 0.5}


def _unnormalised_vs_renormalised():
    def h(ps):
        return -sum(q * math.log(q) for q in ps)
    a, b = [0.5, 0.4], [0.5, 0.5]
    un = (h(a), h(b))
    re_ = (h([q / sum(a) for q in a]), h([q / sum(b) for q in b]))
    assert un[0] > un[1] + 0.01 and re_[0] < re_[1] - 0.005     # the two readings disagree
    return un


@pytest.mark.parametrize("mode", ["paper", "band"])
def test_truncated_entropy_is_not_renormalised(mode):
    _unnormalised_vs_renormalised()
    st = planted([ROW_B, ROW_A])
    prm = rps.Params(mode=mode, k_max=2, tau_pivot=0.85, pct_lo=0, pct_hi=100, n_pivots=1, r=0.1)
    plan = rps.select_pivots(st, np.array([20, 21]), prm)
    assert [pv.pos for pv in plan.pivots] == [21]
    assert plan.pivots[0].tokens == [3, 4]


def test_pivot_mass_threshold_inclusive():
    # row 0: top-2 mass 0.5 + 0.25 = 0.75 = tau_pivot exactly; row 1: 0.5 + 0.375
    # is feasible too but has the lower truncated entropy; row 2: 0.25 + 0.25
    st = dyadic([{1: 0.5, 2: 0.25}, {3: 0.5, 4: 0.375}, {5: 0.25, 6: 0.25, 7: 0.25}])
    prm = rps.Params(mode="paper", k_max=2, tau_pivot=0.75, r=0.1)
    mu, _ = rps.truncated(st, 2)
    assert mu[0] == 0.75
    plan = rps.select_pivots(st, np.array([7, 8, 9]), prm)
    # truncated entropies: row 0: 0.5 ln 2 + 0.25 ln 4 = ln 2 = 0.693;
    # row 1: 0.5 ln 2 + 0.375 ln(8/3) = 0.714  -> row 1 ranks first, row 0 second
    assert [pv.row for pv in plan.pivots] == [1]
    prm2 = rps.Params(mode="paper", k_max=2, tau_pivot=0.75, r=0.1, n_pivots=2)
    plan2 = rps.select_pivots(st, np.array([7, 8, 9]), prm2)
    assert [pv.row for pv in plan2.pivots] == [1, 0]
    assert plan2.pivots[1].feas_margin == 0.0
    # alone with an infeasible row, the boundary row is still the pivot
    plan3 = rps.select_pivots(st.rows([0, 2]), np.array([7, 9]), prm)
    assert [pv.pos for pv in plan3.pivots] == [7]


def test_candidate_ratio_threshold_inclusive():
    # p(v) / P^max = 0.25 / 0.5 = r exactly keeps the runner-up; a strict ">"
    # would leave a single candidate and skip the pivot
    st = dyadic([{1: 0.5, 2: 0.25, 3: 0.125 + 0.0625}, {4: 0.25, 5: 0.25}])
    plan = rps.select_pivots(st, np.array([4, 5]), rps.Params(mode="paper", k_max=2, tau_pivot=0.5, r=0.5))
    assert len(plan.pivots) == 1 and plan.pivots[0].tokens == [1, 2]
    assert plan.pivots[0].cand_margin == 0.0
    plan = rps.select_pivots(st, np.array([4, 5]), rps.Params(mode="paper", k_max=2, tau_pivot=0.5, r=0.5 + 2 ** -20))
    assert plan.pivots == []


# ------------------------------------------------------------ lookahead scoring

def _stats_from_H(H):
    """Stats whose rows have the given entropies (only H is used by Eq. 4)."""
    n = len(H)
    z = np.zeros(n)
    return rps.Stats(H=np.asarray(H, float), lse=z, lmax=z, argmax=z.astype(int),
                     topk_id=np.zeros((n, 1), int), topk_logit=np.zeros((n, 1)))


def test_lambda_zero_single_pivot_is_argmin_mean_entropy():
    anchor = _stats_from_H([2.0, 5.0, 3.0, 1.0])
    plan = rps.Plan([rps.Pivot(row=1, pos=7, tokens=[10, 11, 12], logp=[-0.5, -1.0, -2.0])])
    branches = [_stats_from_H([1.9, 0.0, 2.9, 1.0]),        # mean 1.9333
                _stats_from_H([1.0, 0.0, 2.0, 1.0]),        # mean 1.3333  <- best
                _stats_from_H([2.5, 0.0, 3.5, 1.5])]        # worse than anchor (2.0)
    dec = rps.score(anchor, branches, plan, lam=0.0)
    assert dec.commit and dec.branch == 1 and dec.token == 11 and dec.pivot_pos == 7
    assert math.isclose(dec.delta, 2.0 - 4.0 / 3.0)


def test_abstain_when_no_candidate_beats_mask_and_on_exact_tie():
    anchor = _stats_from_H([1.0, 9.0, 1.0])
    plan = rps.Plan([rps.Pivot(row=1, pos=3, tokens=[4, 5], logp=[-0.1, -0.2])])
    worse = [_stats_from_H([1.5, 0.0, 1.5]), _stats_from_H([1.0, 0.0, 1.0])]   # second ties [MASK]
    dec = rps.score(anchor, worse, plan, lam=0.0)
    assert not dec.commit


def test_large_lambda_always_abstains():
    # a_[MASK] = P^max >= p_anchor(c) for every c, so lambda -> inf favours abstaining
    rng = np.random.default_rng(3)
    logits = rng.normal(0, 2, (6, V))
    logits[:, MASK] = -np.inf
    anchor = softmax_stats(logits, 16)
    plan = rps.Plan([rps.Pivot(row=2, pos=2, tokens=anchor.topk_id[2, 1:4].tolist(),
                               logp=(anchor.topk_logit[2, 1:4] - anchor.lse[2]).tolist())])
    branches = [softmax_stats(logits * 3.0, 16) for _ in range(3)]   # much lower entropy
    assert rps.score(anchor, branches, plan, lam=0.0).commit
    assert not rps.score(anchor, branches, plan, lam=1e6).commit


def test_proposition2_lagrangian_and_pairwise_margin():
    rng = np.random.default_rng(4)
    for _ in range(200):
        n = rng.integers(2, 8)
        Hbar = rng.uniform(0, 5, n)
        a = rng.uniform(1e-4, 1, n)
        lam = rng.uniform(0, 1)
        S = -Hbar + lam * np.log(a)
        assert np.argmax(S) == np.argmin(Hbar - lam * np.log(a))
        for c in range(n):
            for d in range(n):
                lhs = S[c] >= S[d]
                rhs = Hbar[d] - Hbar[c] >= lam * math.log(a[d] / a[c])
                if abs((Hbar[d] - Hbar[c]) - lam * math.log(a[d] / a[c])) > 1e-12:
                    assert lhs == rhs


def binary_entropy(t):
    return -t * math.log(t) - (1 - t) * math.log(1 - t)


def prop1_holds(logits, tau):
    st = softmax_stats(logits, 1)
    n = len(st)
    N = int((confidence(st) >= tau).sum())
    Hbar = st.H.mean()
    return N >= max(0, n - math.floor(n * Hbar / binary_entropy(tau)))


def test_proposition1_bound_on_random_distributions():
    rng = np.random.default_rng(5)
    for _ in range(300):
        n = rng.integers(1, 30)
        logits = rng.normal(0, rng.uniform(0.1, 12), (n, 40))
        tau = rng.uniform(0.5, 0.999)
        assert prop1_holds(logits, tau)


def test_proposition1_is_tight_for_two_point_rows():
    # every row at confidence exactly tau with all remaining mass on one token
    tau = 0.8
    logits = np.full((5, 10), -np.inf)
    logits[:, 0] = math.log(tau)
    logits[:, 1] = math.log(1 - tau)
    st = softmax_stats(logits, 1)
    n = 5
    # Hbar = h(tau): the bound gives n - n = 0, and all 5 rows are eligible
    assert math.isclose(st.H.mean(), binary_entropy(tau), rel_tol=1e-12)
    assert prop1_holds(logits, tau)


# ------------------------------------------------------------ brute force

def _tiny_setup(seed_prompt=1):
    shape = synth.TINY
    w = synth.model_weights_np(shape, seed=0, dtype="f32")
    P, G = 32, 32
    toks = np.concatenate([synth.tokens_np(seed_prompt, "prompt", P, shape.vocab - 1),
                           np.full(G, shape.mask_id, dtype=np.int32)]).astype(np.int64)
    return shape, w, toks, np.arange(P, P + G)


def test_brute_force_every_pivot_candidate_pair_matches_score():
    shape, w, toks, m_pos = _tiny_setup()
    scale = 4.0
    base_logits = om.forward_logits(toks[None], w, shape, m_pos, scale=scale)[0]
    base = softmax_stats(base_logits, 16)
    prm = rps.Params(mode="band", k_max=10, n_pivots=2, r=0.0, n_cand=4)
    plan = rps.select_pivots(base, m_pos, prm)
    assert len(plan.pivots) == 2
    batch = rps.branch_tokens(toks, plan)
    lg = om.forward_logits(batch, w, shape, m_pos, scale=scale)
    branch_stats = [softmax_stats(l, 16) for l in lg]
    dec = rps.score(base, branch_stats, plan, lam=0.3)

    # brute force: every pair as its own batch-1 forward, Eq. 4 from scipy entropies
    H_anchor = scipy.stats.entropy(scipy.special.softmax(base_logits, axis=1), axis=1)
    n = len(m_pos) - 1
    best, best_val = None, -np.inf
    for b, (pi, row, pos, tok, _) in enumerate(plan.branches()):
        t = toks.copy()
        t[pos] = tok
        l1 = om.forward_logits(t[None], w, shape, m_pos, scale=scale)[0]
        Hb = scipy.stats.entropy(scipy.special.softmax(l1, axis=1), axis=1)
        log_a = base_logits[row, tok] - scipy.special.logsumexp(base_logits[row])
        S = -(Hb.sum() - Hb[row]) / n + 0.3 * log_a
        S_mask = -(H_anchor.sum() - H_anchor[row]) / n + 0.3 * (base_logits[row].max() - scipy.special.logsumexp(base_logits[row]))
        assert math.isclose(dec.scores[b], S, abs_tol=1e-10)
        assert math.isclose(dec.deltas[b], S - S_mask, abs_tol=1e-10)
        if S - S_mask > best_val:
            best, best_val = b, S - S_mask
    assert dec.branch == best
    assert dec.commit == (best_val > 0)


def test_every_oracle_branch_satisfies_proposition1():
    shape, w, toks, m_pos = _tiny_setup(seed_prompt=3)
    base = softmax_stats(om.forward_logits(toks[None], w, shape, m_pos, scale=8.0)[0], 16)
    plan = rps.select_pivots(base, m_pos, rps.Params(mode="band", n_pivots=2, r=0.0, n_cand=4))
    lg = om.forward_logits(rps.branch_tokens(toks, plan), w, shape, m_pos, scale=8.0)
    for (pi, row, pos, tok, _), l in zip(plan.branches(), lg):
        rest = np.delete(l, row, axis=0)
        for tau in (0.5, 0.7, 0.9):
            assert prop1_holds(rest, tau)


def test_commit_and_carry_over():
    shape, w, toks, m_pos = _tiny_setup()
    base = softmax_stats(om.forward_logits(toks[None], w, shape, m_pos, scale=4.0)[0], 16)
    plan = rps.select_pivots(base, m_pos, rps.Params(mode="band", n_pivots=2, r=0.0, n_cand=4))
    lg = om.forward_logits(rps.branch_tokens(toks, plan), w, shape, m_pos, scale=4.0)
    bst = [softmax_stats(l, 16) for l in lg]
    dec = rps.score(base, bst, plan, lam=0.0)
    st = rps.State(toks.copy(), m_pos.copy(), base)
    committed = rps.apply_decision(st, dec, bst, base)
    if dec.commit:
        assert committed == [dec.pivot_pos]
        assert st.tokens[dec.pivot_pos] == dec.token
        assert dec.pivot_pos not in st.m_pos and len(st.m_pos) == len(m_pos) - 1
        keep = [j for j in range(len(m_pos)) if j != dec.pivot_row]
        assert np.array_equal(st.stats.H, bst[dec.branch].H[keep])
    else:
        assert committed == [] and np.array_equal(st.m_pos, m_pos)


def test_branch_capacity_truncates_then_drops():
    rng = np.random.default_rng(9)
    logits = rng.normal(0, 1, (12, V))
    logits[:, MASK] = -np.inf
    st = softmax_stats(logits, 16)
    prm = rps.Params(mode="band", pct_lo=0, pct_hi=100, n_pivots=4, r=0.0, n_cand=4, max_branch=9)
    plan = rps.select_pivots(st, np.arange(12), prm)
    # 4 + 4 fit, the third pivot keeps 1 candidate and is dropped, the fourth has none
    assert [len(p.tokens) for p in plan.pivots] == [4, 4]
    assert len(plan.branches()) == 8


def test_band_edges_inclusive():
    # with 5 rows the 25th and 75th percentiles (linear interpolation) are the
    # 2nd and 4th order statistics exactly, so those two rows lie on the band's
    # edges and stay feasible; a strict band would leave only the median row
    rows = [{1: 0.5, 2: 0.25}, {3: 0.5, 4: 0.375}, {5: 0.25, 6: 0.25}, {7: 0.75, 8: 0.0625}, {9: 0.5, 10: 0.5}]
    st = dyadic(rows)
    st.H[:] = [4.0, 1.0, 3.0, 2.0, 5.0]          # edges: H = 2 (row 3) and H = 4 (row 0)
    assert rps.percentile_linear(st.H, 25) == 2.0 and rps.percentile_linear(st.H, 75) == 4.0
    prm = rps.Params(mode="band", k_max=2, pct_lo=25, pct_hi=75, n_pivots=3, r=0.0, n_cand=2)
    plan = rps.select_pivots(st, np.arange(30, 35), prm)
    # truncated entropies: row 0 ln 2 = 0.693, row 2 0.693 (0.25 ln 4 x 2), row 3
    # 0.75 ln(4/3) + 0.0625 ln 16 = 0.389; ties go to the lower position
    assert sorted(pv.row for pv in plan.pivots) == [0, 2, 3]
    assert [pv.row for pv in plan.pivots] == [0, 2, 3]
    assert min(pv.feas_margin for pv in plan.pivots) == 0.0
