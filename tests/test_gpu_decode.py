"""GPU parity of the full RPS decode (Algorithm 1): the GPU loop and the oracle
loop make the same decisions, step by step, on the same model and inputs."""
import numpy as np
import pytest
import torch

import synth
from oracle import rps as orps
from oracle.decode import rps_decode as oracle_decode, baseline_decode as oracle_baseline, model_forward
from tests.parity import MARGIN

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
    ref = oracle_decode(model_forward(w_np, shape, scales=scales), prompt, G, B, shape.mask_id,
                        orps.Params(mode="paper", k_max=10, tau_pivot=tau_pivot, r=0.1, n_cand=10), lam, 0.9,
                        capacity=16)
    excluded = None
    for i, (g, o) in enumerate(zip(st.trace, ref.trace)):
        if tuple(g) != tuple(_event_key(o)):
            # the first divergence must sit on a decision the oracle itself calls a near-tie
            assert o[-1] <= MARGIN, f"event {i}: gpu {g} vs oracle {o}"
            excluded = i
            break
    if excluded is None:
        assert len(st.trace) == len(ref.trace)
        assert np.array_equal(got, ref.tokens)
        assert st.nfe == ref.nfe and st.lookahead == ref.lookahead
    assert np.all(got[Pl:] != shape.mask_id)
    print(f"nfe {st.nfe} (lookahead {st.lookahead}), pivot commits {st.commits_pivot}, "
          f"abstains {st.abstains}, first excluded event {excluded}")


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
    ref = oracle_baseline(model_forward(w_np, shape, scales=scales), prompt, G, B, shape.mask_id, rule, max(k, 1),
                          tau=tau)
    excluded = None
    for i, (g, o) in enumerate(zip(st.trace, ref.trace)):
        if tuple(g) != tuple(o[:2]):
            assert o[2] <= MARGIN, f"step {i}: gpu {g} vs oracle {o}"
            excluded = i
            break
    if excluded is None:
        assert len(st.trace) == len(ref.trace) and st.nfe == ref.nfe
        assert np.array_equal(got, ref.tokens)
    if rule != "threshold":
        assert st.nfe == (G // B) * -(-B // k)
    assert np.all(got[Pl:] != shape.mask_id)
    print(f"{rule} k={k} tau={tau}: nfe {st.nfe}, first excluded step {excluded}")



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
    ref = oracle_decode(model_forward(w_np, shape, scales=scales), prompt, G, B, shape.mask_id,
                        orps.Params(mode="paper", k_max=10, tau_pivot=tau_pivot, r=0.1, n_cand=10), lam, 0.9,
                        capacity=16, block_forward=model_prefix_cached(w_np, shape, scales=scales))
    excluded = None
    for i, (g, o) in enumerate(zip(st.trace, ref.trace)):
        if tuple(g) != tuple(_event_key(o)):
            assert o[-1] <= MARGIN, f"event {i}: gpu {g} vs oracle {o}"
            excluded = i
            break
    if excluded is None:
        assert len(st.trace) == len(ref.trace)
        assert np.array_equal(got, ref.tokens)
        assert st.nfe == ref.nfe and st.lookahead == ref.lookahead
    assert np.all(got[Pl:] != shape.mask_id)
    print(f"prefix cache: nfe {st.nfe} (lookahead {st.lookahead}), pivot commits {st.commits_pivot}, "
          f"abstains {st.abstains}, first excluded event {excluded}")


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
    ref = oracle_baseline(model_forward(w_np, shape, scales=scales), prompt, G, B, shape.mask_id, rule, max(k, 1),
                          tau=tau, block_forward=model_prefix_cached(w_np, shape, scales=scales))
    excluded = None
    for i, (g, o) in enumerate(zip(st.trace, ref.trace)):
        if tuple(g) != tuple(o[:2]):
            assert o[2] <= MARGIN, f"step {i}: gpu {g} vs oracle {o}"
            excluded = i
            break
    if excluded is None:
        assert len(st.trace) == len(ref.trace) and st.nfe == ref.nfe
        assert np.array_equal(got, ref.tokens)
    assert np.all(got[Pl:] != shape.mask_id)
    print(f"prefix cache {rule} k={k}: nfe {st.nfe}, first excluded step {excluded}")
