"""Oracle per-position predictive statistics (Section 3, Notation).

For each row of logits the oracle computes, over the vocabulary without
[MASK] (whose logit is -inf, so p([MASK]) = 0):

  lmax   the largest logit,
  lse    log sum_v exp(logit_v),
  p      p_v = exp(logit_v - lse),
  H      the entropy -sum_v p_v log p_v in nats (natural log: the paper's
         binary-entropy bound h(tau) <= log 2 in Appendix B fixes the base),
  P^max  the confidence max_v p_v = exp(lmax - lse),
  argmax the token with the largest logit, the lowest id on ties,
  top-K  token ids ordered by logit descending, lower id first on ties, and
         their logits.

Decision margins (the distance of a float value from the boundary that
decides an integer output) are returned alongside, so tests can exclude
near-ties.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class Stats:
    """Statistics of R rows; topk arrays are [R, K]."""
    H: np.ndarray
    lse: np.ndarray
    lmax: np.ndarray
    argmax: np.ndarray
    topk_id: np.ndarray
    topk_logit: np.ndarray
    argmax_margin: np.ndarray | None = None   # logit gap top-1 vs top-2
    topk_margin: np.ndarray | None = None     # logit gap at rank K vs rank K+1

    @property
    def K(self) -> int:
        return self.topk_id.shape[1]

    def __len__(self) -> int:
        return self.H.shape[0]

    def rows(self, idx) -> "Stats":
        idx = np.asarray(idx, dtype=np.int64)
        pick = lambda a: None if a is None else a[idx]
        return Stats(self.H[idx], self.lse[idx], self.lmax[idx], self.argmax[idx],
                     self.topk_id[idx], self.topk_logit[idx],
                     pick(self.argmax_margin), pick(self.topk_margin))

    @staticmethod
    def concat(parts) -> "Stats":
        cat = lambda name: np.concatenate([getattr(p, name) for p in parts])
        opt = lambda name: None if any(getattr(p, name) is None for p in parts) else cat(name)
        return Stats(cat("H"), cat("lse"), cat("lmax"), cat("argmax"), cat("topk_id"),
                     cat("topk_logit"), opt("argmax_margin"), opt("topk_margin"))


def entropy_from_logits(logits: np.ndarray) -> np.ndarray:
    """H(p) = -sum_v p_v log p_v for p = softmax(logits) per row (terms with p_v = 0 are 0)."""
    logits = np.asarray(logits, dtype=np.float64)
    lse = log_sum_exp(logits)
    logp = logits - lse[:, None]
    p = np.exp(logp)
    terms = np.where(p > 0.0, p * np.where(p > 0.0, logp, 0.0), 0.0)
    return -terms.sum(axis=1)


def log_sum_exp(logits: np.ndarray) -> np.ndarray:
    m = logits.max(axis=1)
    return m + np.log(np.exp(logits - m[:, None]).sum(axis=1))


def top_order(row: np.ndarray, n: int) -> np.ndarray:
    """Indices of the n largest entries of a row, larger value first and the
    lower index first on ties.  Every entry at least as large as the n-th
    largest value is a candidate (so all entries tied with it are), and the
    candidates are sorted by (-value, index)."""
    V = row.shape[0]
    if n >= V:
        return np.lexsort((np.arange(V), -row))[:n]
    thr = np.partition(row, V - n)[V - n]          # the n-th largest value
    cand = np.nonzero(row >= thr)[0]
    return cand[np.lexsort((cand, -row[cand]))][:n]


def softmax_stats(logits: np.ndarray, topk: int) -> Stats:
    """Statistics of each row of logits ([R, V], -inf marks excluded tokens).

    Rows are processed 16 at a time: every row's statistics depend on that
    row alone, and small blocks keep the temporaries in reused heap memory."""
    logits = np.asarray(logits, dtype=np.float64)
    if logits.shape[0] > 16:
        return Stats.concat([_stats_block(logits[i:i + 16], topk) for i in range(0, logits.shape[0], 16)])
    return _stats_block(logits, topk)


def _stats_block(logits: np.ndarray, topk: int) -> Stats:
    R, V = logits.shape
    lmax = logits.max(axis=1)
    lse = log_sum_exp(logits)
    H = entropy_from_logits(logits)
    # order: larger logit first, then smaller token id; only the first
    # topk + 1 ranks are needed
    order = np.stack([top_order(row, min(V, max(topk + 1, 2))) for row in logits])
    top = order[:, :topk]
    top_logit = np.take_along_axis(logits, top, axis=1)
    nxt = np.take_along_axis(logits, order[:, 1:2], axis=1)[:, 0]
    kth1 = np.take_along_axis(logits, order[:, topk:topk + 1], axis=1)[:, 0] if topk < V else np.full(R, -np.inf)
    with np.errstate(invalid="ignore"):          # -inf minus -inf where rows have < 2 finite logits
        am, km = lmax - nxt, top_logit[:, -1] - kth1
    return Stats(H=H, lse=lse, lmax=lmax, argmax=top[:, 0].astype(np.int64),
                 topk_id=top.astype(np.int64), topk_logit=top_logit,
                 argmax_margin=np.nan_to_num(am, nan=np.inf), topk_margin=np.nan_to_num(km, nan=np.inf))


def confidence(st: Stats) -> np.ndarray:
    """P^max = max_v p_v = exp(lmax - lse)."""
    return np.exp(st.lmax - st.lse)
