"""GPU parity of the full RPS decode (Algorithm 1): the GPU loop and the oracle
loop make the same decisions, step by step, on the same model and inputs."""
import numpy as np
import pytest
import torch

import synth
from oracle import rps as orps
from oracle.decode import rps_decode as oracle_decode, baseline_decode as oracle_baseline, model_forward
from oracle.decode import rps_decode_follow, baseline_decode_follow
from tests.parity import MARGIN, judge_events, perturbed, event_flips

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def tiny():
    import paper_2608_11742_amd as P
    shape = synth.TINY
    w_np = synth.model_weights_np(shape, seed=0, dtype="f32")
    m = P.Model(shape, {k: torch.from_numpy(v).to(DEV) for k, v in w_np.items()}, dtype="f32", max_pos=256)
    yield P, shape, w_np, m
    m.close()


def _event_key(e):
    return e[:-1] if e[0] in ("commit", "lookahead", "skip") else e


@pytest.mark.parametrize("tau_pivot,lam,seed", [(0.9, 0.1, 1), (0.6, 0.3, 2), (0.75, 0.0, 3)])
def test_decode_trajectory_matches_oracle(tiny, tau_pivot, lam, seed):
    P, shape, w_np, model = tiny
    Pl, G, B = 16, 64, 32
    prompt = synth.tokens_np(seed, "prompt", Pl, shape.vocab - 1)
    scales = synth.position_scales_np(seed + 10, np.arange(Pl + G), 2.6, 16.0)
    prm = P.params(mode="paper", k_max=10, tau_pivot=tau_pivot, n_pivots=1, r=0.1, n_cand=10, max_branch=15)
    toks, st = P.rps_decode(model, torch.from_numpy(prompt).to(DEV), G, B, prm, lam, 0.9, capacity=16,
                            row_scale=torch.from_numpy(scales).to(DEV), record=True)
    got = toks.cpu().numpy()
    prm_o = orps.Params(mode="paper", k_max=10, tau_pivot=tau_pivot, r=0.1, n_cand=10)
    fwd = model_forward(w_np, shape, scales=scales)
    # teacher forcing: the oracle decides on every state of the GPU's trajectory
    ev = rps_decode_follow(fwd, prompt, G, B, shape.mask_id, prm_o, lam, 0.9, st.trace, got, capacity=16)
    rep = judge_events(ev, label=f"decode f32 seed {seed}")
    assert rep["compared"] >= 0.8 * rep["events"] and rep["compared"] >= 10, rep
    # the free-running oracle from the same start, while no near-tie intervenes
    ref = oracle_decode(fwd, prompt, G, B, shape.mask_id, prm_o, lam, 0.9, capacity=16)
    if all(tuple(g) == tuple(_event_key(o)) for g, o in zip(st.trace, ref.trace)):
        assert len(st.trace) == len(ref.trace) and np.array_equal(got, ref.tokens)
        assert st.nfe == ref.nfe and st.lookahead == ref.lookahead
    assert np.all(got[Pl:] != shape.mask_id)
    print(f"nfe {st.nfe} (lookahead {st.lookahead}), pivot commits {st.commits_pivot}, abstains {st.abstains}; "
          f"{rep['compared']} of {rep['events']} decisions compared, {rep['tokens_compared']} tokens")


@pytest.mark.parametrize("rule,k,tau,seed", [("confidence", 1, 0.0, 4), ("confidence", 3, 0.0, 5),
                                             ("entropy", 2, 0.0, 6), ("threshold", 0, 0.5, 7)])
def test_baseline_trajectory_matches_oracle(tiny, rule, k, tau, seed):
    """The GPU baseline schedulers (Eq. 2: top-k by confidence or by lowest
    entropy, confidence threshold) commit the same positions, step by step, as
    the oracle; a divergence is accepted only on a step whose ranking the oracle
    itself places within the near-tie margin."""
    P, shape, w_np, model = tiny
    Pl, G, B = 16, 64, 32
    prompt = synth.tokens_np(seed, "prompt", Pl, shape.vocab - 1)
    scales = synth.position_scales_np(seed + 10, np.arange(Pl + G), 2.6, 16.0)
    toks, st = P.baseline_decode(model, torch.from_numpy(prompt).to(DEV), G, B, rule, k=max(k, 1), tau=tau,
                                 row_scale=torch.from_numpy(scales).to(DEV), record=True)
    got = toks.cpu().numpy()
    fwd = model_forward(w_np, shape, scales=scales)
    ev = baseline_decode_follow(fwd, prompt, G, B, shape.mask_id, rule, max(k, 1), tau, st.trace, got)
    rep = judge_events(ev, label=f"{rule} k={k}")
    assert rep["compared"] >= 0.8 * rep["events"], rep
    if rule != "threshold":
        assert st.nfe == (G // B) * -(-B // k)
    assert np.all(got[Pl:] != shape.mask_id)
    print(f"{rule} k={k} tau={tau}: nfe {st.nfe}; {rep['compared']} of {rep['events']} steps compared, "
          f"{rep['tokens_compared']} tokens")


@pytest.mark.parametrize("tau_pivot,lam,seed", [(0.9, 0.1, 11), (0.6, 0.3, 12)])
def test_prefix_cached_decode_trajectory_matches_oracle(tiny, tau_pivot, lam, seed):
    """Algorithm 1 with the prefix cache refreshed at every block opening: the
    GPU loop (cache written by the opening forward, later forwards over the
    block and suffix) takes the oracle's decisions."""
    from oracle.decode import model_prefix_cached
    P, shape, w_np, model = tiny
    Pl, G, B = 16, 96, 32
    prompt = synth.tokens_np(seed, "prompt", Pl, shape.vocab - 1)
    scales = synth.position_scales_np(seed + 10, np.arange(Pl + G), 2.6, 16.0)
    prm = P.params(mode="paper", k_max=10, tau_pivot=tau_pivot, n_pivots=1, r=0.1, n_cand=10, max_branch=15)
    toks, st = P.rps_decode(model, torch.from_numpy(prompt).to(DEV), G, B, prm, lam, 0.9, capacity=16,
                            row_scale=torch.from_numpy(scales).to(DEV), record=True, prefix_cache=True)
    got = toks.cpu().numpy()
    prm_o = orps.Params(mode="paper", k_max=10, tau_pivot=tau_pivot, r=0.1, n_cand=10)
    ev = rps_decode_follow(model_forward(w_np, shape, scales=scales), prompt, G, B, shape.mask_id, prm_o, lam,
                           0.9, st.trace, got, capacity=16,
                           block_forward=model_prefix_cached(w_np, shape, scales=scales))
    rep = judge_events(ev, label=f"prefix-cached decode seed {seed}")
    assert rep["compared"] >= 0.8 * rep["events"] and rep["compared"] >= 10, rep
    assert np.all(got[Pl:] != shape.mask_id)
    print(f"prefix cache: nfe {st.nfe} (lookahead {st.lookahead}), pivot commits {st.commits_pivot}, "
          f"abstains {st.abstains}; {rep['compared']} of {rep['events']} decisions compared")


@pytest.mark.parametrize("rule,k,tau,seed", [("confidence", 2, 0.0, 13), ("threshold", 0, 0.5, 14)])
def test_prefix_cached_baseline_matches_oracle(tiny, rule, k, tau, seed):
    from oracle.decode import model_prefix_cached
    P, shape, w_np, model = tiny
    Pl, G, B = 16, 96, 32
    prompt = synth.tokens_np(seed, "prompt", Pl, shape.vocab - 1)
    scales = synth.position_scales_np(seed + 10, np.arange(Pl + G), 2.6, 16.0)
    toks, st = P.baseline_decode(model, torch.from_numpy(prompt).to(DEV), G, B, rule, k=max(k, 1), tau=tau,
                                 row_scale=torch.from_numpy(scales).to(DEV), record=True, prefix_cache=True)
    got = toks.cpu().numpy()
    ev = baseline_decode_follow(model_forward(w_np, shape, scales=scales), prompt, G, B, shape.mask_id, rule,
                                max(k, 1), tau, st.trace, got,
                                block_forward=model_prefix_cached(w_np, shape, scales=scales))
    rep = judge_events(ev, label=f"prefix-cached {rule}")
    assert rep["compared"] >= 0.8 * rep["events"], rep
    assert np.all(got[Pl:] != shape.mask_id)
    print(f"prefix cache {rule} k={k}: nfe {st.nfe}; {rep['compared']} of {rep['events']} steps compared")


# 2 layers of a 512 residual with the 8B workloads' vocabulary (126464): every
# later forward of a block puts at most 32 rows per sequence through the LM
# head, i.e. the 128-row tiles, the full set of vocabulary slices and the
# multi-wave merge of the 8B decode
DECODE_BF16 = synth.ModelShape(n_layers=2, d_model=512, n_heads=4, head_dim=128, d_ffn=1536, vocab=126464)


@pytest.fixture(scope="module")
def decode_bf16():
    import paper_2608_11742_amd as P
    shape = DECODE_BF16
    w = synth.model_weights_torch(shape, seed=0, dtype="bf16", device=DEV)
    m = P.Model(shape, w, dtype="bf16", max_pos=256)
    w_np = {k: v.double().cpu().numpy() for k, v in w.items()}
    yield P, shape, w_np, m
    m.close()


@pytest.mark.parametrize("packed,prefix_cache,seed", [(False, False, 21), (True, True, 22)])
def test_bf16_8b_vocab_decode_teacher_forced(decode_bf16, packed, prefix_cache, seed):
    """Algorithm 1 in bf16 with the 8B vocabulary against the mirror oracle,
    teacher-forced: the oracle decides on every state of the GPU's trajectory.
    The per-position logit scales are those of the 8B decode workload times
    sqrt(4096 / 512), so that the logits (and the entropies, ~0.5-6 nats) have
    the 8B model's spread."""
    from oracle.decode import model_packed_lookahead, model_prefix_cached
    P, shape, w_np, model = decode_bf16
    Pl, G, B = 32, 64, 32
    prompt = synth.tokens_np(seed, "prompt", Pl, shape.vocab - 1)
    f = float(np.sqrt(4096 / shape.d_model))
    scales = synth.position_scales_np(seed + 10, np.arange(Pl + G), 2.6 * f, 16.0 * f)
    prm = P.params(mode="paper", k_max=10, tau_pivot=0.9, n_pivots=1, r=0.1, n_cand=10, max_branch=15)
    toks, st = P.rps_decode(model, torch.from_numpy(prompt).to(DEV), G, B, prm, 0.1, 0.9, capacity=16,
                            row_scale=torch.from_numpy(scales).to(DEV), record=True, packed=packed,
                            prefix_cache=prefix_cache)
    got = toks.cpu().numpy()
    assert np.all(got[Pl:] != shape.mask_id)
    prm_o = orps.Params(mode="paper", k_max=10, tau_pivot=0.9, r=0.1, n_cand=10)
    def follow(wts):
        kw = {}
        if prefix_cache:
            kw["block_forward"] = model_prefix_cached(wts, shape, scales=scales, mirror=True, packed=packed)
        elif packed:
            kw["lookahead"] = model_packed_lookahead(wts, shape, scales=scales, mirror=True)
        return rps_decode_follow(model_forward(wts, shape, scales=scales, mirror=True), prompt, G, B,
                                 shape.mask_id, prm_o, 0.1, 0.9, st.trace, got, capacity=16, **kw)
    ev = follow(w_np)
    # the oracle's own flips along the same trajectory through weights
    # perturbed by a relative 1e-6: the yardstick for the GPU's bf16 noise
    own = event_flips(ev, follow(perturbed(w_np)))
    rep = judge_events(ev, label=f"bf16 8B-vocab decode packed={packed} cache={prefix_cache}",
                       max_exceptions=max(3, 2 * own))
    print(f"bf16 8B vocab packed={packed} cache={prefix_cache}: nfe {st.nfe} (lookahead {st.lookahead}), "
          f"pivot commits {st.commits_pivot}, abstains {st.abstains}; {rep['compared']} of {rep['events']} "
          f"decisions compared ({rep['excluded']} near-ties), {rep['tokens_compared']} tokens compared, "
          f"oracle's own flips {own}, exceptions {rep['exception_list']}")
    assert st.lookahead >= 3, "the workload must exercise the lookahead"
    assert rep["compared"] >= 0.7 * rep["events"] and rep["compared"] >= 10, rep
