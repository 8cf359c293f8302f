"""Comparison helpers for GPU-vs-oracle parity tests (imported by the GPU tests)."""
from __future__ import annotations

import numpy as np

MARGIN = 1e-3   # integer decisions must agree wherever the oracle's margin exceeds this


def dev():
    import torch
    return torch.device("cuda:0")


def determined_ranks(ref_logits: np.ndarray, kth_margin: np.ndarray, margin: float) -> np.ndarray:
    """[R, K] mask of top-K ranks whose token is fixed by a gap > margin to both neighbours."""
    R, K = ref_logits.shape
    gaps = np.empty((R, K))
    gaps[:, :K - 1] = ref_logits[:, :K - 1] - ref_logits[:, 1:]
    gaps[:, K - 1] = kth_margin
    left = np.concatenate([np.full((R, 1), np.inf), gaps[:, :K - 1]], axis=1)
    return (gaps > margin) & (left > margin)


def compare_stats(got: dict, ref, tol: float, k: int | None = None, margin=MARGIN, label: str = "",
                  logit_tol: float | None = None):
    """Float fields within tol (max-abs); argmax and top-k ids equal where determined.

    logit_tol (default tol) bounds the individual logits (lmax, top-k
    logits); entropies and log-partition values keep tol.

    margin="auto" (end-to-end bf16 comparisons, where the inputs of the LM head
    already differ by rounding-order effects amplified through the layers):
    decisions are compared where the oracle's margin exceeds
    max(1e-3, 2 x the observed max-abs logit error); kernel-level comparisons
    on identical inputs use the fixed 1e-3.
    """
    k = k or ref.topk_id.shape[1]
    logit_tol = tol if logit_tol is None else logit_tol
    report = {}
    for name in ("H", "lse", "lmax"):
        err = float(np.max(np.abs(got[name].astype(np.float64) - getattr(ref, name))))
        report[name] = err
        bound = logit_tol if name == "lmax" else tol
        assert err <= bound, f"{label} {name}: max-abs error {err:.3e} > {bound:.1e}"
    # the r-th largest logit is defined even where tied tokens swap ranks
    tl_err = float(np.max(np.abs(got["topk_logit"][:, :k] - ref.topk_logit[:, :k])))
    report["topk_logit"] = tl_err
    assert tl_err <= logit_tol, f"{label} topk_logit: max-abs error {tl_err:.3e} > {logit_tol:.1e}"
    if margin == "auto":
        margin = max(MARGIN, 2.0 * max(tl_err, report["lmax"]))
    report["margin"] = margin
    am = ref.argmax_margin > margin
    bad = np.nonzero(am & (got["argmax"] != ref.argmax))[0]
    assert bad.size == 0, f"{label} argmax mismatch at rows {bad[:8]}"
    det = determined_ranks(ref.topk_logit[:, :k], ref.topk_margin if k == ref.topk_id.shape[1]
                           else ref.topk_logit[:, k - 1] - ref.topk_logit[:, k], margin)
    mism = det & (got["topk_id"][:, :k] != ref.topk_id[:, :k])
    assert not mism.any(), f"{label} top-k id mismatch at rows {np.nonzero(mism.any(1))[0][:8]}"
    report["excluded_argmax"] = int((~am).sum())
    report["excluded_topk"] = int((~det).sum())
    return report
