"""GPU parity at the 8B-class shapes, in the launch configuration the benchmark
times (16 sequences x 512 tokens, LM head on 16 x 256 rows), checked on
sampled outputs the oracle can compute, and by properties that hold at any size."""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from synth import workloads as W
from oracle import model as om
from oracle import rps as orps
from oracle.stats import softmax_stats
from tests.parity import compare_stats, MARGIN, perturbed, perturbations, allowed_flips, flip_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
B8 = synth.B8


@pytest.fixture(scope="module")
def P():
    import paper_2608_11742_amd as P
    return P


@pytest.fixture(scope="module")
def lm_head():
    return synth.weight_torch(W.SEED_WEIGHTS, "lm_head", (B8.vocab, B8.d_model), dtype="bf16", device=DEV)


@pytest.mark.parametrize("R", [1, 16, 31, 32, 128, 129, 4000, 4096])
def test_lm_head_stats_full_shape(P, lm_head, R):
    """vocab_entropy_topk with the 8B LM head (d 4096, V 126464).  Up to 129
    rows (one or two 128-row tiles over all vocabulary slices, the multi-wave
    merge of a decode's block forwards) every row is compared; at the step's
    4096 (and a ragged 4000) rows, 24 sampled rows."""
    h = synth.weight_torch(21, "hidden", (R, B8.d_model), std=1.0, dtype="bf16", device=DEV)
    rs = torch.from_numpy((0.5 + 3 * synth.uniform01_np(22, "rs", R)).astype(np.float32)).to(DEV)
    out = P.Stats(R, 16, device=DEV)
    ws = torch.empty(P.vocab_entropy_topk_workspace_bytes(R, B8.vocab), dtype=torch.uint8, device=DEV)
    P.vocab_entropy_topk(h, lm_head, out, ws, row_scale=rs, scale=1.0, mask_id=B8.mask_id)
    torch.cuda.synchronize()
    if R <= 256:
        rows = np.arange(R)
    else:
        rows = np.unique(np.concatenate([[0, 1, 127, 128, R - 1], synth.tokens_np(23, "rows", 19, R)]))
    hn = h[torch.from_numpy(rows).to(DEV)].float().cpu().numpy().astype(np.float64)
    wn = lm_head.float().cpu().numpy().astype(np.float64)
    logits = rs.cpu().numpy()[rows].astype(np.float64)[:, None] * (hn @ wn.T)
    logits[:, B8.mask_id] = -np.inf
    ref = softmax_stats(logits, 16)
    got = {k: v[rows] for k, v in out.numpy().items()}
    print(compare_stats(got, ref, 1e-3, label=f"lm head R={R}"))


@pytest.fixture(scope="module")
def b8_two_layer(P, lm_head):
    shape = dataclasses.replace(B8, n_layers=2)
    w = synth.model_weights_torch(shape, seed=W.SEED_WEIGHTS, dtype="bf16", device=DEV, layers=range(2))
    m = P.Model(shape, w, dtype="bf16", max_pos=512)
    yield shape, w, m
    m.close()


def _branch_batch(shape, n_branch=16, P_=256, G=256):
    prompt = synth.tokens_np(W.SEED_PROMPT, "prompt", P_, shape.vocab - 1)
    toks = np.concatenate([prompt, np.full(G, shape.mask_id, np.int32)])
    batch = np.repeat(toks[None], n_branch, axis=0)
    piv = P_ + synth.tokens_np(31, "piv", n_branch, G)
    cand = synth.tokens_np(32, "cand", n_branch, shape.vocab - 1)
    batch[np.arange(n_branch), piv] = cand
    return batch, np.arange(P_, P_ + G, dtype=np.int32)


def test_two_layer_8b_width_forward_in_bench_launch_config(P, b8_two_layer):
    """16 x 512 batch (M = 8192 GEMM rows) through 2 layers of 8B width; sequence 5
    against the mirror oracle on 32 sampled masked rows, at the unscaled logits
    of the 8B workloads (scale 1)."""
    shape, w, model = b8_two_layer
    batch, m_pos = _branch_batch(shape)
    out = model.forward(torch.from_numpy(batch).to(DEV), torch.from_numpy(m_pos).to(DEV), scale=1.0)
    torch.cuda.synchronize()
    b = 5
    w_np = {k: v.double().cpu().numpy() for k, v in w.items()}
    sample = np.unique(np.concatenate([[0, 255], synth.tokens_np(33, "s", 30, 256)]))

    def oracle(wts):
        h = om.hidden(batch[b], wts, shape, mirror=True)[m_pos[sample]]
        return softmax_stats(om.lm_logits(h, wts, shape, scale=1.0), 16)
    ref, ref2 = oracle(w_np), [oracle(wp) for wp in perturbations(w_np)]
    got = {k: v[b * 256 + sample] for k, v in out.numpy().items()}
    # individual logits: max(2e-2, 1.25 x the oracle's own spread under
    # relative 1e-6 weight perturbations, the largest of three), as for the
    # cached step below; entropies and log-partition values keep 2e-2
    spread = max(max(float(np.max(np.abs(ref.lmax - r.lmax))), float(np.max(np.abs(ref.topk_logit - r.topk_logit))))
                 for r in ref2)
    rep = compare_stats(got, ref, 2e-2, label="2-layer 8B width", logit_tol=max(2e-2, 1.25 * spread),
                        max_exceptions=allowed_flips(ref, ref2), id_ranks=4)
    print(f"oracle noise floor {spread:.3e}, oracle's own flips {flip_rows(ref, ref2)}", rep)


def test_batch_invariance(P, b8_two_layer):
    """A branch's statistics do not depend on the other sequences of its batch:
    replacing every other sequence of the 16 x 512 batch (same launch shape)
    leaves branches 0 and 9 bit-identical."""
    shape, w, model = b8_two_layer
    batch, m_pos = _branch_batch(shape)
    m_dev = torch.from_numpy(m_pos).to(DEV)
    full = model.forward(torch.from_numpy(batch).to(DEV), m_dev).numpy()
    for b in (0, 9):
        other = synth.tokens_np(40 + b, "other", batch.size, shape.vocab - 1).reshape(batch.shape)
        other[b] = batch[b]
        one = model.forward(torch.from_numpy(other).to(DEV), m_dev).numpy()
        sl = slice(b * 256, (b + 1) * 256)
        for k in ("H", "lse", "lmax", "argmax", "topk_id", "topk_logit"):
            assert np.array_equal(full[k][sl], one[k][sl]), k


@pytest.fixture(scope="module")
def b8_full(P):
    w = synth.model_weights_torch(B8, seed=W.SEED_WEIGHTS, dtype="bf16", device=DEV)
    m = P.Model(B8, w, dtype="bf16", max_pos=512)
    yield w, m
    m.close()


def test_full_step_properties(P, b8_full):
    """One 32-layer RPS lookahead step (the benchmark's workload): plan, branches,
    decision and commit are consistent with their definitions."""
    w, model = b8_full
    wl = W.WORKLOADS["b8_rps_step_bf16"]
    prompt = synth.tokens_torch(W.SEED_PROMPT, "prompt", wl.prompt_len, B8.vocab - 1, device=DEV)
    tokens = torch.cat([prompt, torch.full((wl.gen_len,), B8.mask_id, dtype=torch.int32, device=DEV)])
    m_pos = torch.arange(wl.prompt_len, wl.seq, dtype=torch.int32, device=DEV)
    base = model.forward(tokens[None], m_pos)
    b0 = base.numpy()
    t0 = tokens.cpu().numpy()
    prm = P.params(mode="band", k_max=10, n_pivots=4, r=0.0, n_cand=4, max_branch=16)
    stp = P.RpsStep(model, tokens, m_pos, base, prm, lam=0.0, capacity=16)
    stp.run()
    torch.cuda.synchronize()
    plan = P.read_plan(stp.plan)
    assert plan.n_pivots == 4 and plan.n_branch == 16
    # pivots lie in the entropy band and are the feasible rows of largest truncated entropy
    H = b0["H"].astype(np.float64)
    lo, hi = np.percentile(H, 25), np.percentile(H, 75)
    lp = b0["topk_logit"][:, :10].astype(np.float64) - b0["lse"][:, None]
    htr = -(np.exp(lp) * lp).sum(1)
    order = [j for j in np.lexsort((np.arange(256), -htr)) if lo <= H[j] <= hi]
    rows = [plan.pivot_row[i] for i in range(4)]
    gaps = np.abs(np.diff(np.sort(htr)))
    if gaps.min() > 1e-6:
        assert rows == order[:4]
    for b in range(16):
        j = plan.br_row[b]
        assert plan.br_token[b] == b0["topk_id"][j, b % 4]
    bt = stp.branch_tokens.cpu().numpy()
    for b in range(16):
        e = t0.copy()
        e[plan.br_pos[b]] = plan.br_token[b]
        assert np.array_equal(bt[b], e)
    # the decision is the largest margin; commit iff positive
    dec = P.read_decision(stp.dec)
    deltas = stp.deltas.cpu().numpy()
    assert dec.branch == int(np.argmax(deltas))
    assert bool(dec.commit) == bool(deltas.max() > 0)
    # every branch statistic is finite and the entropies are below log(V - 1)
    bs = stp.branch_stats.numpy()
    assert np.all(np.isfinite(bs["H"])) and np.all(bs["H"] <= np.log(B8.vocab - 1) + 1e-3)
    # commit / carry-over
    t1 = stp.tokens.cpu().numpy()
    if dec.commit:
        assert t1[dec.pivot_pos] == dec.token and stp.n_m == 255
        keep = [j for j in range(256) if j != dec.pivot_row]
        assert np.array_equal(stp.base.H.cpu().numpy()[:255], bs["H"][dec.branch * 256:(dec.branch + 1) * 256][keep])
    else:
        assert np.array_equal(t1, t0) and stp.n_m == 256


def test_cached_step_two_layer_8b_width(P, b8_two_layer):
    """KV-cached lookahead (1024 cached prefix positions, 16 branch blocks of 32):
    branch 7 against the mirror oracle with the oracle's own prefix cache, in
    the batch, alone (the batch-1 anchor forward's launches) and in a ragged
    batch of 10 blocks."""
    from paper_2608_11742_amd._abi import KvCache
    shape, w, model = b8_two_layer
    Pn, Bk, nb = 1024, 32, 16
    model_p = P.Model(shape, w, dtype="bf16", max_pos=Pn + Bk)
    prefix = synth.tokens_np(41, "prefix", Pn, shape.vocab - 1)
    k, vt, cap = model_p.new_kv_cache(Pn)
    kv = KvCache(k.data_ptr(), vt.data_ptr(), 0, cap)
    model_p.forward(torch.from_numpy(prefix).to(DEV)[None], torch.zeros(1, dtype=torch.int32, device=DEV), kv_out=kv)
    kv.len = Pn
    blocks = np.full((nb, Bk), shape.mask_id, dtype=np.int32)
    blocks[np.arange(nb), synth.tokens_np(42, "piv", nb, Bk)] = synth.tokens_np(43, "tok", nb, shape.vocab - 1)
    lm = np.arange(Bk, dtype=np.int32)
    out = model_p.forward(torch.from_numpy(blocks).to(DEV), torch.from_numpy(lm).to(DEV), pos_offset=Pn,
                          kv_prefix=kv, scale=1.0)
    torch.cuda.synchronize()
    w_np = {kk: v.double().cpu().numpy() for kk, v in w.items()}
    b = 7

    def oracle_stats(wts):
        kv_ = om.prefix_cache(prefix, wts, shape, mirror=True)
        h = om.hidden(blocks[b], wts, shape, pos_offset=Pn, mirror=True, prefix_kv=kv_)
        return softmax_stats(om.lm_logits(h, wts, shape, scale=1.0), 16)
    ref = oracle_stats(w_np)
    got = {kk: v[b * Bk:(b + 1) * Bk] for kk, v in out.numpy().items()}
    # The oracle's own rounding-order noise floor on this model: the same
    # mirror oracle with every layer weight perturbed by a relative 1e-6
    # (random signs; the size of float32 accumulation error over 4096 terms)
    # moves individual logits by `spread`, since two random layers over 1056
    # keys amplify flips of bf16 rounding decisions.  Individual logits (lmax,
    # top-k logits) are held to max(2e-2, 1.25 x spread); entropies and
    # log-partition values keep 2e-2.
    # three perturbations (32 rows give few flips each): the largest spread
    # and flip count set the bounds
    others = [oracle_stats(wp) for wp in perturbations(w_np)]
    spread = max(max(float(np.max(np.abs(ref.lmax - o.lmax))), float(np.max(np.abs(ref.topk_logit - o.topk_logit))))
                 for o in others)
    logit_tol = max(2e-2, 1.25 * spread)
    own = max(flip_rows(ref, o) for o in others)
    rep = compare_stats(got, ref, 2e-2, label="cached step 2-layer 8B width", logit_tol=logit_tol,
                        max_exceptions=max(2, 2 * own), id_ranks=4)
    print(f"oracle noise floor {spread:.3e}, logit bound {logit_tol:.3e}, oracle's own flips {own}", rep)
    # the same block alone (batch 1, the step's anchor form): 32 workgroups of
    # the 32-query attention layout, so each head's 17 key tiles are split
    # over workgroups and merged, and the 32-row projections
    out1 = model_p.forward(torch.from_numpy(blocks[b:b + 1]).to(DEV), torch.from_numpy(lm).to(DEV), pos_offset=Pn,
                           kv_prefix=kv, scale=1.0)
    torch.cuda.synchronize()
    rep1 = compare_stats(out1.numpy(), ref, 2e-2, label="cached block alone 2-layer 8B width", logit_tol=logit_tol,
                         max_exceptions=max(2, 2 * own), id_ranks=4)
    print(rep1)
    # the same block in a ragged batch of 10 (320 rows per projection: QKV
    # split-K parts on 256 x 192 tiles with a partial second row tile, O in 4
    # and down in 8 K parts, gate/up on 256 x 192 tiles)
    out10 = model_p.forward(torch.from_numpy(blocks[:10]).to(DEV), torch.from_numpy(lm).to(DEV), pos_offset=Pn,
                            kv_prefix=kv, scale=1.0)
    torch.cuda.synchronize()
    got10 = {kk: v[b * Bk:(b + 1) * Bk] for kk, v in out10.numpy().items()}
    rep10 = compare_stats(got10, ref, 2e-2, label="cached block in a batch of 10, 2-layer 8B width",
                          logit_tol=logit_tol, max_exceptions=max(2, 2 * own), id_ranks=4)
    print(rep10)
    model_p.close()
