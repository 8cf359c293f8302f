"""Oracle for the RPS scheduler (Section 3 Decoding, Section 4.1, Appendix A).

State of one decoding step: the token sequence, the ordered list of masked
positions M of the current block, and the statistics of the current
predictive distributions at those positions (row j <-> position M[j]).

Readings taken where the paper is silent (stated once here, used below):
  * thresholds are inclusive everywhere (the paper writes >=);
  * position ties (confidence fallback, pivot ranking) go to the lower
    position; token ties go to the lower token id;
  * Eq. 4 ties between a candidate and [MASK] go to [MASK] (abstain);
  * with |M| <= 1 after the standard commit no pivot search is made, since
    Eq. 4 divides by |M| - 1;
  * multi-pivot steps (several pivots, as in the percentile-band workloads)
    score each (pivot, candidate) pair by its Eq. 4 margin over the same
    pivot's [MASK] branch and commit the pair with the largest margin if that
    margin is positive; with one pivot this is exactly Eq. 4;
  * band mode replaces the mass filter of Eq. 3 by "full entropy within the
    [pct_lo, pct_hi] percentiles of H over M" (percentiles by linear
    interpolation between order statistics, Hyndman-Fan definition 7) and
    keeps Eq. 3's truncated-entropy objective for ranking.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from .stats import Stats, confidence


@dataclass
class Params:
    mode: str = "paper"       # "paper": mass filter of Eq. 3; "band": percentile band
    k_max: int = 10
    tau_pivot: float = 0.9
    pct_lo: float = 25.0
    pct_hi: float = 75.0
    n_pivots: int = 1
    r: float = 0.1
    n_cand: int = 10
    max_branch: int = 16      # lookahead capacity: branches beyond it are dropped


@dataclass
class Pivot:
    row: int                  # index j into M
    pos: int                  # absolute position M[j]
    tokens: list              # candidate tokens (rank order)
    logp: list                # anchor log-probabilities of the candidates
    # decision margins (distance from the deciding boundary)
    feas_margin: float = math.inf
    rank_margin: float = math.inf
    cand_margin: float = math.inf


@dataclass
class Plan:
    pivots: list = field(default_factory=list)
    # decision margin of an empty plan (distance of the nearest row from feasibility)
    empty_margin: float = math.inf

    def branches(self):
        """(pivot index, pivot row, pivot pos, token, anchor logp) in pivot-major, rank order."""
        out = []
        for pi, pv in enumerate(self.pivots):
            for t, lp in zip(pv.tokens, pv.logp):
                out.append((pi, pv.row, pv.pos, int(t), float(lp)))
        return out


# ------------------------------------------------------------ standard commit

def confidence_commit(st: Stats, tau: float):
    """Rows committed by the confidence-aware rule (Eq. 2, third case, and Algorithm 1).

    S = {i in M : P_i^max >= tau}; if S is empty it is the single most
    confident row.  Returns (rows, tokens, margin) with tokens = argmax
    (Eq. 1) and margin = min |P^max - tau| (or the fallback's confidence gap).
    """
    pmax = confidence(st)
    rows = np.nonzero(pmax >= tau)[0]
    if rows.size == 0:
        order = np.lexsort((np.arange(len(pmax)), -pmax))
        rows = order[:1]
        gap = pmax[order[0]] - pmax[order[1]] if len(pmax) > 1 else math.inf
        margin = min(float(np.min(np.abs(pmax - tau))), float(gap))
    else:
        margin = float(np.min(np.abs(pmax - tau)))
    return rows, st.argmax[rows], margin


def top_k_rows(values: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest values of a score, lower index first on ties."""
    return np.lexsort((np.arange(len(values)), -values))[:k]


def topk_commit(st: Stats, rule: str, k: int):
    """Rows committed by the top-k rules of Eq. 2: the k rows of highest
    confidence (first case; ranked by log P^max = lmax - lse, the same order
    as P^max) or of lowest entropy (second case; ranked by -H), the lower row
    (= lower position) first on ties.  Returns (rows ascending, tokens =
    argmax (Eq. 1), margin = gap between the k-th and (k+1)-th ranked keys)."""
    if rule == "confidence":
        key = np.asarray(st.lmax, dtype=np.float64) - np.asarray(st.lse, dtype=np.float64)
    elif rule == "entropy":
        key = -np.asarray(st.H, dtype=np.float64)
    else:
        raise ValueError(rule)
    order = np.lexsort((np.arange(len(key)), -key))
    k = min(k, len(key))
    margin = float(key[order[k - 1]] - key[order[k]]) if k < len(key) else math.inf
    rows = np.sort(order[:k])
    return rows, st.argmax[rows], margin


# ------------------------------------------------------------ pivot selection

def truncated(st: Stats, k_max: int):
    """Eq. 3 quantities: mu_i = sum_{v in T_i} p_i(v) and -sum_{v in T_i} p_i(v) log p_i(v).

    T_i is the top-k_max support; p is not renormalised on T_i.
    """
    logp = st.topk_logit[:, :k_max] - st.lse[:, None]
    p = np.exp(logp)
    return p.sum(axis=1), -(p * logp).sum(axis=1)


def percentile_linear(values: np.ndarray, q: float) -> float:
    """q-th percentile (0..100) by linear interpolation between order statistics."""
    s = np.sort(np.asarray(values, dtype=np.float64))
    idx = q / 100.0 * (len(s) - 1)
    lo = int(math.floor(idx))
    hi = min(lo + 1, len(s) - 1)
    return float(s[lo] + (idx - lo) * (s[hi] - s[lo]))


def select_pivots(st: Stats, m_pos, prm: Params) -> Plan:
    """Pivot selection (Eq. 3) and adaptive candidate sets (Section 4.1).

    Returns an empty plan when no pivot is feasible or when the chosen
    pivot has at most one real candidate (both skip rules of Algorithm 1).
    Candidates beyond the lookahead capacity (max_branch branches in total)
    are dropped before that check.
    """
    m_pos = np.asarray(m_pos)
    n = len(m_pos)
    if n <= 1:
        return Plan()
    mu, htr = truncated(st, prm.k_max)
    if prm.mode == "paper":
        feas = mu >= prm.tau_pivot
        feas_margin = np.abs(mu - prm.tau_pivot)
    elif prm.mode == "band":
        lo = percentile_linear(st.H, prm.pct_lo)
        hi = percentile_linear(st.H, prm.pct_hi)
        feas = (st.H >= lo) & (st.H <= hi)
        feas_margin = np.minimum(np.abs(st.H - lo), np.abs(st.H - hi))
    else:
        raise ValueError(prm.mode)
    cand_rows = np.nonzero(feas)[0]
    if cand_rows.size == 0:
        return Plan(empty_margin=float(np.min(feas_margin)))
    # rank feasible rows by truncated entropy, larger first, then lower position
    order = cand_rows[np.lexsort((m_pos[cand_rows], -htr[cand_rows]))]
    chosen = order[:prm.n_pivots]
    plan = Plan()
    used = 0
    for rank, j in enumerate(chosen):
        nxt = [htr[order[rank + 1]]] if rank + 1 < len(order) else []
        prv = [htr[order[rank - 1]]] if rank > 0 else []
        rank_margin = min([abs(htr[j] - x) for x in nxt + prv] + [math.inf])
        # candidate set: v in T_{i*} with p(v) >= r * P^max, in rank order, capped
        logp = st.topk_logit[j, :prm.k_max] - st.lse[j]
        p = np.exp(logp)
        pmax = math.exp(st.lmax[j] - st.lse[j])
        ratio = p / pmax
        keep = [k for k in range(len(p)) if ratio[k] >= prm.r][:prm.n_cand]
        keep = keep[:max(0, prm.max_branch - used)]
        cand_margin = float(np.min(np.abs(ratio - prm.r))) if prm.r > 0 else math.inf
        pv = Pivot(row=int(j), pos=int(m_pos[j]),
                   tokens=[int(st.topk_id[j, k]) for k in keep],
                   logp=[float(logp[k]) for k in keep],
                   feas_margin=float(feas_margin[j]), rank_margin=float(rank_margin),
                   cand_margin=cand_margin)
        if len(pv.tokens) > 1:
            plan.pivots.append(pv)
            used += len(pv.tokens)
    return plan


def branch_tokens(tokens: np.ndarray, plan: Plan, with_anchor: bool = False) -> np.ndarray:
    """Lookahead batch: one copy of the sequence per (pivot, candidate), pivot := candidate.

    with_anchor puts the unchanged sequence (pivot still [MASK]) first.
    """
    rows = [np.array(tokens, copy=True)] if with_anchor else []
    for _, _, pos, tok, _ in plan.branches():
        t = np.array(tokens, copy=True)
        t[pos] = tok
        rows.append(t)
    return np.stack(rows) if rows else np.zeros((0, len(tokens)), dtype=np.asarray(tokens).dtype)


# ------------------------------------------------------------ lookahead scoring

@dataclass
class Decision:
    commit: bool
    branch: int               # winning branch (index into plan.branches()), -1 if none
    pivot_row: int
    pivot_pos: int
    token: int
    delta: float              # best Eq. 4 margin over the pivot's [MASK] branch
    scores: np.ndarray        # Eq. 4 score of every branch
    deltas: np.ndarray        # margin of every branch over its pivot's [MASK] score
    mask_scores: np.ndarray   # Eq. 4 score of [MASK] per pivot
    margin_sum: float = math.inf   # decision margin on the summed-entropy scale


def eq4_score(H_rows: np.ndarray, pivot_row: int, log_a: float, lam: float) -> float:
    """Eq. 4: -(1/(|M|-1)) sum_{i in M minus pivot} H(p_i^c) + lambda * log a_c."""
    n = len(H_rows) - 1
    rest = np.delete(H_rows, pivot_row)
    return -rest.sum() / n + lam * log_a


def score(anchor: Stats, branch_stats, plan: Plan, lam: float, anchor_logp=None) -> Decision:
    """Eq. 4 over every branch, [MASK] per pivot, and the commit/abstain decision.

    anchor: statistics of the anchor branch (pivot kept masked); its P^max at a
    pivot is the plausibility of [MASK].  branch_stats: one Stats per branch,
    rows aligned with M.  anchor_logp: log p_anchor(c) per branch; defaults
    to the plan's values (when the anchor is the distribution the plan came from).
    """
    brs = plan.branches()
    nb = len(brs)
    if nb == 0:
        return Decision(False, -1, -1, -1, -1, 0.0, np.zeros(0), np.zeros(0), np.zeros(0))
    n = len(anchor) - 1
    mask_scores = np.zeros(len(plan.pivots))
    for pi, pv in enumerate(plan.pivots):
        log_amask = anchor.lmax[pv.row] - anchor.lse[pv.row]         # log P^max_anchor
        mask_scores[pi] = eq4_score(anchor.H, pv.row, log_amask, lam)
    scores = np.zeros(nb)
    deltas = np.zeros(nb)
    for b, (pi, row, pos, tok, lp) in enumerate(brs):
        log_a = lp if anchor_logp is None else anchor_logp[b]
        scores[b] = eq4_score(branch_stats[b].H, row, log_a, lam)
        deltas[b] = scores[b] - mask_scores[pi]
    best = int(np.lexsort((np.arange(nb), -deltas))[0])
    others = np.delete(deltas, best)
    gap = deltas[best] - others.max() if others.size else math.inf
    commit = bool(deltas[best] > 0.0)
    _, row, pos, tok, _ = brs[best]
    margin_sum = n * min(abs(deltas[best]), gap)
    return Decision(commit, best, row, pos, tok, float(deltas[best]), scores, deltas,
                    mask_scores, float(margin_sum))


# ------------------------------------------------------------ commit / carry-over

@dataclass
class State:
    tokens: np.ndarray        # [S] current sequence
    m_pos: np.ndarray         # masked positions of the current block, ascending
    stats: Stats              # current distributions, rows aligned with m_pos

    def copy(self) -> "State":
        return State(self.tokens.copy(), self.m_pos.copy(), self.stats.rows(np.arange(len(self.stats))))


def apply_confidence_commit(state: State, tau: float, mask_id: int):
    """Commit S (Eq. 2, third case) with greedy tokens (Eq. 1); returns committed positions."""
    rows, toks, margin = confidence_commit(state.stats, tau)
    assert np.all(toks != mask_id)
    state.tokens[state.m_pos[rows]] = toks
    keep = np.setdiff1d(np.arange(len(state.m_pos)), rows)
    committed = state.m_pos[rows].copy()
    state.m_pos = state.m_pos[keep]
    state.stats = state.stats.rows(keep)
    return committed, margin


def apply_topk_commit(state: State, rule: str, k: int, mask_id: int):
    """Commit the top-k rule's rows (Eq. 2, first or second case) with greedy
    tokens (Eq. 1); returns (committed positions ascending, margin)."""
    rows, toks, margin = topk_commit(state.stats, rule, k)
    assert np.all(toks != mask_id)
    state.tokens[state.m_pos[rows]] = toks
    keep = np.setdiff1d(np.arange(len(state.m_pos)), rows)
    committed = state.m_pos[rows].copy()
    state.m_pos = state.m_pos[keep]
    state.stats = state.stats.rows(keep)
    return committed, margin


def apply_decision(state: State, dec: Decision, branch_stats, anchor: Stats):
    """Commit c* at i* or abstain; carry the winner's (or the anchor's) distributions."""
    if dec.commit:
        state.tokens[dec.pivot_pos] = dec.token
        keep = np.array([j for j in range(len(state.m_pos)) if j != dec.pivot_row], dtype=np.int64)
        state.m_pos = state.m_pos[keep]
        state.stats = branch_stats[dec.branch].rows(keep)
        return [dec.pivot_pos]
    state.stats = anchor.rows(np.arange(len(anchor)))
    return []
