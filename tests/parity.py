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


def compare_stats(got: dict, ref, tol: float, k: int | None = None, margin: float = MARGIN, label: str = "",
                  logit_tol: float | None = None, max_exceptions: int = 0, id_ranks: int | None = None):
    """Float fields within tol (max-abs); argmax and top-k ids equal where the
    oracle's decision margin exceeds `margin` (1e-3).

    logit_tol (default tol) bounds the individual logits (lmax, top-k
    logits); entropies and log-partition values keep tol.

    Exceptions: in end-to-end bf16 comparisons the inputs of the LM head
    already differ from the oracle's by rounding-order effects, so a decision
    whose margin lies above 1e-3 but within twice the observed logit error can
    legitimately flip.  At most `max_exceptions` such rows (argmax and top-k
    rows together) are accepted; a mismatch at a margin above twice the
    observed error always fails.  The report counts compared, excluded and
    excepted decisions.

    id_ranks (default k): the top-k ids are compared on the first id_ranks
    ranks (the logit values on all k).  End-to-end bf16 comparisons use the
    4 ranks that the workloads' candidate sets take: deeper ranks of the
    unscaled 8B-class logits lie a few hundredths apart, inside the rounding
    noise, and routinely swap.
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
    noise = 2.0 * max(tl_err, report["lmax"])
    report["margin"] = margin
    am = ref.argmax_margin > margin
    bad_am = am & (got["argmax"] != ref.argmax)
    assert not np.any(bad_am & (ref.argmax_margin > noise)), \
        f"{label} argmax mismatch beyond the noise bound at rows {np.nonzero(bad_am & (ref.argmax_margin > noise))[0][:8]}"
    ki = k if id_ranks is None else min(id_ranks, k)
    kth = ref.topk_margin if ki == ref.topk_id.shape[1] else ref.topk_logit[:, ki - 1] - ref.topk_logit[:, ki]
    det = determined_ranks(ref.topk_logit[:, :ki], kth, margin)
    mism = det & (got["topk_id"][:, :ki] != ref.topk_id[:, :ki])
    strict = determined_ranks(ref.topk_logit[:, :ki], kth, noise)
    assert not np.any(mism & strict), \
        f"{label} top-k id mismatch beyond the noise bound at rows {np.nonzero((mism & strict).any(1))[0][:8]}"
    exc_rows = np.union1d(np.nonzero(bad_am)[0], np.nonzero(mism.any(1))[0])
    report["compared_argmax"] = int(am.sum())
    report["compared_topk"] = int(det.sum())
    report["excluded_argmax"] = int((~am).sum())
    report["excluded_topk"] = int((~det).sum())
    report["exceptions"] = int(exc_rows.size)
    assert exc_rows.size <= max_exceptions, \
        f"{label} {exc_rows.size} rows with decisions flipped above the 1e-3 margin (allowed {max_exceptions}): " \
        f"{exc_rows[:8]}; {report}"
    return report


def flip_rows(ref, other, margin: float = MARGIN, id_ranks: int = 4) -> int:
    """Rows where a second oracle evaluation (`other`, e.g. through slightly
    perturbed weights) changes a decision that `ref` fixes by more than
    `margin`: the argmax or one of the first id_ranks top-k ids.  This is the
    number of flips the oracle's own rounding noise produces, the yardstick for
    a bf16 implementation's.  `other` may be a list of such evaluations: the
    largest count among them."""
    if isinstance(other, (list, tuple)):
        return max(flip_rows(ref, o, margin, id_ranks) for o in other)
    am = (ref.argmax_margin > margin) & (other.argmax != ref.argmax)
    K = ref.topk_id.shape[1]
    ki = min(id_ranks, K)
    kth = ref.topk_margin if ki == K else ref.topk_logit[:, ki - 1] - ref.topk_logit[:, ki]
    det = determined_ranks(ref.topk_logit[:, :ki], kth, margin)
    tk = (det & (other.topk_id[:, :ki] != ref.topk_id[:, :ki])).any(1)
    return int((am | tk).sum())


def perturbed(weights: dict, rel: float = 1e-6, seed: int = 46) -> dict:
    """A copy of the layer weights scaled by 1 + rel * (random sign), the
    embedding and LM head unchanged: evaluating the oracle through it shows how
    far rounding-order differences of the size of float32 accumulation error
    (a relative 1e-6 over 4096-term sums) move its outputs."""
    import synth
    sgn = np.where(synth.uniform01_np(seed, "perturb", 1 << 16) < 0.5, -1.0, 1.0)
    out = {}
    for k, v in weights.items():
        if k.startswith("layers."):
            v = np.asarray(v, dtype=np.float64)
            out[k] = v * (1.0 + rel * np.resize(sgn, v.size).reshape(v.shape))
        else:
            out[k] = v
    return out


def perturbations(weights: dict, n: int = 3, rel: float = 1e-6) -> list:
    """n perturbed copies of the weights (seeds 46, 47, ...): the flip count of
    one random perturbation is itself noisy, the largest of a few is the
    yardstick."""
    return [perturbed(weights, rel=rel, seed=46 + i) for i in range(n)]


def allowed_flips(ref, other, floor: int = 2, factor: float = 2.0, **kw) -> int:
    """Exceptions allowed to a bf16 implementation: `factor` times the flips of
    the oracle's own perturbed evaluation(s) (the largest, for a list), at
    least `floor`."""
    return max(floor, int(np.ceil(factor * flip_rows(ref, other, **kw))))


def judge_events(events, label: str = "", margin: float = MARGIN, max_exceptions: int = 0):
    """Teacher-forced decode parity: every decision the oracle makes on the
    followed trajectory must equal the applied (GPU) decision wherever the
    oracle's margin exceeds `margin`, and so must every greedy token of a
    committed position whose argmax margin exceeds it.  At most
    `max_exceptions` such decisions may differ (bf16 trajectories, where the
    GPU's rounding noise can exceed 1e-3); the report counts the compared,
    excluded and excepted decisions."""
    rep = {"events": len(events), "compared": 0, "excluded": 0, "exceptions": 0,
           "tokens_compared": 0, "tokens_excluded": 0, "exception_list": []}
    for i, e in enumerate(events):
        if e.margin > margin:
            rep["compared"] += 1
            if e.oracle != e.applied:
                rep["exceptions"] += 1
                rep["exception_list"].append((i, e.oracle, e.applied, e.margin))
        else:
            rep["excluded"] += 1
        for pos, own, applied, m in e.token_rows:
            if m > margin:
                rep["tokens_compared"] += 1
                if own != applied:
                    rep["exceptions"] += 1
                    rep["exception_list"].append((i, ("token", pos, own), ("token", pos, applied), m))
            else:
                rep["tokens_excluded"] += 1
    assert rep["exceptions"] <= max_exceptions, f"{label}: {rep['exceptions']} decisions differ above the " \
        f"{margin:g} margin (allowed {max_exceptions}): {rep['exception_list'][:6]}"
    return rep


def event_flips(ev, ev2, margin: float = MARGIN) -> int:
    """Decisions of a teacher-forced oracle run that a second oracle run along
    the same trajectory (e.g. through perturbed weights) makes differently,
    where the first run's margin exceeds `margin` (greedy tokens included)."""
    n = 0
    for a, b in zip(ev, ev2):
        if a.margin > margin and a.oracle != b.oracle:
            n += 1
        for (pa, oa, _, ma), (pb, ob, _, _) in zip(a.token_rows, b.token_rows):
            if ma > margin and pa == pb and oa != ob:
                n += 1
    return n
