"""Oracle parity of the benchmark's own step at full depth: the 32-layer 8B-shape
RPS lookahead step (16 branch sequences x 512 tokens, statistics on 16 x 256
masked rows, band pivots, Eq. 4 with lambda = 0) against the mirror oracle.

The oracle evaluates the base sequence, every branch sequence of the GPU's
plan and one perturbed copy of the base (for its own rounding-order noise
floor) through all 32 layers in float64, one layer at a time (the layer's
weights upcast from the device's bf16 values).  The work is split over
several tests that share the state of the layer walk, so that each finishes
in about a minute.  Compared:
  * the base statistics (all 256 masked rows) and every branch's statistics
    (16 x 256 rows): entropies and log-partition values within 2e-2, logits
    within max(2e-2, 1.5 x the oracle's noise floor), argmax and top-4 ids
    where the oracle's margin exceeds 1e-3, with at most twice as many flips
    as the oracle's own perturbed evaluation of the base makes (reported);
  * the plan: the oracle's pivots and candidates from its own base statistics
    against the GPU's, wherever the band-edge and rank margins exceed 1e-3;
  * the decision: the oracle's Eq. 4 scores of the GPU's branches against the
    GPU's, on the summed-entropy scale (winning branch and commit) where its
    margin exceeds 1e-3.
"""
import numpy as np
import pytest
import torch

import synth
from synth import workloads as W
from oracle import model as om
from oracle import rps as orps
from oracle.stats import softmax_stats
from tests.parity import compare_stats, MARGIN, allowed_flips, flip_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
B8 = synth.B8
WL = W.WORKLOADS["b8_rps_step_bf16"]
NB = WL.n_pivots * WL.n_cand          # 16 branch sequences
STATE = {}


@pytest.fixture(scope="module")
def gpu_step():
    """The benchmark's step on the GPU, with everything the comparisons read."""
    import paper_2608_11742_amd as P
    w = synth.model_weights_torch(B8, seed=W.SEED_WEIGHTS, dtype="bf16", device=DEV)
    model = P.Model(B8, w, dtype="bf16", max_pos=512)
    prompt = synth.tokens_torch(W.SEED_PROMPT, "prompt", WL.prompt_len, B8.vocab - 1, device=DEV)
    tokens = torch.cat([prompt, torch.full((WL.gen_len,), B8.mask_id, dtype=torch.int32, device=DEV)])
    m_pos = torch.arange(WL.prompt_len, WL.seq, dtype=torch.int32, device=DEV)
    base = model.forward(tokens[None], m_pos)
    res = {"tokens": tokens.cpu().numpy().astype(np.int64), "m_pos": m_pos.cpu().numpy().astype(np.int64),
           "base": base.numpy()}
    prm = P.params(mode=WL.pivot_mode, k_max=WL.k_max, n_pivots=WL.n_pivots, r=WL.r, n_cand=WL.n_cand,
                   max_branch=WL.capacity)
    stp = P.RpsStep(model, tokens, m_pos, base, prm, lam=WL.lam, capacity=WL.capacity)
    stp.run()
    torch.cuda.synchronize()
    res["plan"] = P.read_plan(stp.plan)
    res["dec"] = P.read_decision(stp.dec)
    res["deltas"] = stp.deltas.cpu().numpy()[:NB].astype(np.float64)
    res["branch_tokens"] = stp.branch_tokens.cpu().numpy().astype(np.int64)
    res["branch"] = stp.branch_stats.numpy()
    # the base sequence evaluated inside the 16-sequence batch (slot 0), for
    # the batch-1 versus in-batch summation-order offset
    inb = res["branch_tokens"].copy()
    inb[0] = res["tokens"]
    m_fresh = torch.from_numpy(res["m_pos"].astype(np.int32)).to(DEV)   # the step compacted m_pos in place
    res["in_batch"] = model.forward(torch.from_numpy(inb.astype(np.int32)).to(DEV), m_fresh).numpy()
    torch.cuda.synchronize()
    yield P, w, res
    model.close()


def _layer_weights(w, l):
    return {f"layers.{l}.{n}": w[f"layers.{l}.{n}"].double().cpu().numpy() for n in synth.WEIGHT_NAMES}


def test_full_step_gpu_runs(gpu_step):
    P, w, res = gpu_step
    plan = res["plan"]
    assert plan.n_pivots == WL.n_pivots and plan.n_branch == NB
    # sequences of the oracle's walk: the base, its perturbed copy, the GPU's 16 branches
    seqs = np.concatenate([res["tokens"][None], res["tokens"][None], res["branch_tokens"][:NB]])
    x = w["emb"][torch.from_numpy(seqs).to(DEV)].double().cpu().numpy()
    STATE.update(seqs=seqs, x=x, done=0)


def _walk(w, upto):
    """Advance the oracle's layer walk of every sequence to layer `upto`."""
    assert STATE.get("done") is not None, "the GPU step must run first"
    pos = np.arange(WL.seq)
    sgn = np.where(synth.uniform01_np(45, "perturb", 1 << 16) < 0.5, -1.0, 1.0)
    for l in range(STATE["done"], upto):
        wl = _layer_weights(w, l)
        # sequence 1 is the base through weights perturbed by a relative 1e-6
        # (random signs): the oracle's own rounding-order noise floor
        wp = {k: v * (1.0 + 1e-6 * np.resize(sgn, v.size).reshape(v.shape)) for k, v in wl.items()}
        x = STATE["x"]
        for s in range(x.shape[0]):
            x[s] = om.layer(x[s], wp if s == 1 else wl, l, B8, pos, mirror=True)
        STATE["done"] = l + 1


@pytest.mark.parametrize("upto", [8, 16, 24, 32])
def test_full_step_oracle_layers(gpu_step, upto):
    _walk(gpu_step[1], upto)
    assert STATE["done"] == upto


def test_full_step_oracle_lm_head(gpu_step):
    P, w, res = gpu_step
    assert STATE["done"] == B8.n_layers
    lm = {"lm_head": w["lm_head"].double().cpu().numpy()}
    rows = res["m_pos"]
    stats = []
    for s in range(STATE["x"].shape[0]):
        h = om.bf16_round(om.rmsnorm(STATE["x"][s][rows], B8.rms_eps))
        stats.append(softmax_stats(om.lm_logits(h, lm, B8, scale=WL.logit_scale), WL.topk))
    STATE["stats"] = stats
    del STATE["x"]


def _logit_tol():
    """Individual logits: max(2e-2, 1.5 x the oracle's own spread), the spread
    measured on the base's 256 rows (the branch comparisons take their
    maximum over 16 times as many rows).  After 32 random layers the oracle
    moves its own logits by ~6e-2 under a relative 1e-6 weight perturbation,
    so 2e-2 lies below its noise floor; entropies and log-partition values
    keep 2e-2."""
    a, b = STATE["stats"][0], STATE["stats"][1]
    spread = max(float(np.max(np.abs(a.lmax - b.lmax))), float(np.max(np.abs(a.topk_logit - b.topk_logit))))
    return spread, max(2e-2, 1.5 * spread)


def test_full_step_base_stats_and_plan(gpu_step):
    P, w, res = gpu_step
    ref = STATE["stats"][0]
    spread, ltol = _logit_tol()
    own = flip_rows(ref, STATE["stats"][1])
    print(f"\nbase: oracle noise floor {spread:.3e}, logit bound {ltol:.3e}, oracle's own flips {own}")
    rep = compare_stats(res["base"], ref, 2e-2, logit_tol=ltol, label="full-depth base",
                        max_exceptions=allowed_flips(ref, STATE["stats"][1]), id_ranks=4)
    print(f"base: {rep}")
    # the oracle's plan from its own base statistics
    prm = orps.Params(mode=WL.pivot_mode, k_max=WL.k_max, n_pivots=WL.n_pivots, r=WL.r, n_cand=WL.n_cand,
                      max_branch=WL.capacity)
    plan = orps.select_pivots(ref, res["m_pos"], prm)
    gp = res["plan"]
    gpu_pivots = [gp.pivot_pos[i] for i in range(gp.n_pivots)]
    # a pivot whose band-edge and rank margins both exceed 1e-3 must be chosen,
    # and the chosen ones keep their relative order; a pivot the oracle places
    # within the margin may be missing, and for each such one the GPU may take
    # the next row of the ranking instead
    det = [pv.pos for pv in plan.pivots if min(pv.feas_margin, pv.rank_margin) > MARGIN]
    undet = [pv.pos for pv in plan.pivots if min(pv.feas_margin, pv.rank_margin) <= MARGIN]
    missing = [p for p in det if p not in gpu_pivots]
    assert not missing, f"determined pivots {missing} missing: oracle {[p.pos for p in plan.pivots]}, gpu {gpu_pivots}"
    assert [p for p in gpu_pivots if p in det] == det, f"order: oracle {det}, gpu {gpu_pivots}"
    extra = [p for p in gpu_pivots if p not in [pv.pos for pv in plan.pivots]]
    assert len(extra) <= len(undet), f"gpu pivots {extra} beyond the oracle's {len(undet)} undetermined ones"
    compared, excluded = len(det), len(undet)
    print(f"plan: oracle pivots {[p.pos for p in plan.pivots]}, gpu {gpu_pivots}; "
          f"{compared} determined and chosen, {excluded} within the 1e-3 margin, gpu's others {extra}")
    STATE["plan_report"] = (compared, excluded)


def test_full_step_branch_stats(gpu_step):
    P, w, res = gpu_step
    spread, ltol = _logit_tol()
    n = len(res["m_pos"])
    exc = 0
    worst = {}
    # the oracle's own flips on the base (256 rows) set the per-branch allowance
    allowed = allowed_flips(STATE["stats"][0], STATE["stats"][1])
    for b in range(NB):
        got = {k: v[b * n:(b + 1) * n] for k, v in res["branch"].items()}
        rep = compare_stats(got, STATE["stats"][2 + b], 2e-2, logit_tol=ltol, label=f"full-depth branch {b}",
                            max_exceptions=allowed, id_ranks=4)
        exc += rep["exceptions"]
        for k in ("H", "lse", "lmax", "topk_logit"):
            worst[k] = max(worst.get(k, 0.0), rep[k])
    print(f"\nbranches: worst errors {worst}, decision exceptions {exc} over {NB} x {n} rows "
          f"(allowed {allowed} per branch)")


def test_full_step_decision(gpu_step):
    """Eq. 4 on the oracle's statistics of the GPU's branches, against the
    oracle's base as the anchor: winning branch and commit."""
    P, w, res = gpu_step
    gp = res["plan"]
    pivots = []
    for i in range(gp.n_pivots):
        bs = [b for b in range(gp.n_branch) if gp.br_pivot[b] == i]
        pivots.append(orps.Pivot(row=gp.pivot_row[i], pos=gp.pivot_pos[i], tokens=[gp.br_token[b] for b in bs],
                                 logp=[float(gp.br_logp[b]) for b in bs]))
    plan = orps.Plan(pivots)
    assert len(plan.branches()) == NB
    anchor = STATE["stats"][0]
    dec = orps.score(anchor, STATE["stats"][2:], plan, WL.lam)
    n = len(res["m_pos"]) - 1
    gd = res["dec"]
    gap = np.abs(n * (dec.deltas - res["deltas"]))
    print(f"\ndecision: oracle branch {dec.branch} commit {dec.commit} margin(summed) {dec.margin_sum:.3e}; "
          f"gpu branch {gd.branch} commit {bool(gd.commit)}; summed-scale delta error max {gap.max():.3e}")
    same = gd.branch == dec.branch and bool(gd.commit) == dec.commit
    if dec.margin_sum > MARGIN and not same:
        # only a decision within the GPU's own summed-scale error may differ
        assert dec.margin_sum <= 2.0 * gap.max(), "decision differs above the noise bound"
        print("decision differs within the summed-scale noise bound (one reported exception)")
    STATE["decision_margin"] = dec.margin_sum


def test_full_step_batch_order_offset(gpu_step):
    """The step's anchor is the batch-1 forward (split-K projections at 512
    rows) while its branches run in the 16-sequence batch (no split-K): the
    same sequence evaluated both ways differs only by summation order.  Its
    entropy offset, summed over the masked rows (the scale of Eq. 4's
    decisions), is reported and bounded."""
    P, w, res = gpu_step
    d = res["in_batch"]["H"][:len(res["m_pos"])].astype(np.float64) - res["base"]["H"].astype(np.float64)
    print(f"\nbatch-1 vs in-batch: max |dH| {np.abs(d).max():.3e}, summed dH {d.sum():.3e}, "
          f"summed |dH| {np.abs(d).sum():.3e}")
    assert np.abs(d).max() < 2e-2
