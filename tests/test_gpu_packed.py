"""GPU parity of the packed lookahead (Section 4.1, lookahead scoring;
Algorithm 1's x_ahead = [x || x_b^(c_1) || ...]): dllm_forward_packed and
rps_build_packed against the oracle's packed forward, and the full RPS decode
with packed lookaheads against the oracle loop with the same packing."""
import numpy as np
import pytest
import torch

import synth
from synth import ModelShape
from oracle import model as om
from oracle import rps as orps
from oracle.decode import rps_decode as oracle_decode, model_forward, model_packed_lookahead
from oracle.stats import softmax_stats
from tests.parity import compare_stats, perturbed, perturbations, allowed_flips, flip_rows, MARGIN

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
SMALL_BF16 = ModelShape(n_layers=2, d_model=512, n_heads=4, head_dim=128, d_ffn=1536, vocab=3000)


@pytest.fixture(scope="module")
def P():
    import paper_2608_11742_amd as P
    return P


@pytest.fixture(scope="module")
def tiny(P):
    shape = synth.TINY
    w_np = synth.model_weights_np(shape, seed=0, dtype="f32")
    m = P.Model(shape, {k: torch.from_numpy(v).to(DEV) for k, v in w_np.items()}, dtype="f32", max_pos=256)
    yield shape, w_np, m
    m.close()


@pytest.fixture(scope="module")
def small_bf16(P):
    shape = SMALL_BF16
    w_np = synth.model_weights_np(shape, seed=0, dtype="bf16")
    w = {k: torch.from_numpy(v).to(DEV).to(torch.bfloat16).contiguous() for k, v in w_np.items()}
    m = P.Model(shape, w, dtype="bf16", max_pos=512)
    yield shape, w_np, m
    m.close()


def _packed_case(shape, S, b0, B, n, seed):
    """Shared sequence with its block masked past a few committed tokens, and
    n branches that each fill one block position with a token."""
    shared = synth.tokens_np(seed, "shared", S, shape.vocab - 1)
    shared[b0 + min(3, B - 1):b0 + B] = shape.mask_id
    fill = synth.tokens_np(seed + 1, "fill", n, shape.vocab - 1)
    piv = b0 + (synth.tokens_np(seed + 2, "piv", n, B) % B)
    blocks = []
    for c in range(n):
        blk = shared[b0:b0 + B].copy()
        blk[piv[c] - b0] = fill[c]
        blocks.append(blk)
    return shared, np.concatenate([shared] + blocks)


def _lm_pos(S, b0, B):
    """Positions before, inside (every other one, and the block's ends) and after the block."""
    inside = list(range(b0, b0 + B, 2)) + [b0 + B - 1]
    out = sorted(set([0, max(b0 - 1, 0), min(b0 + B, S - 1), S - 1] + inside))
    return np.array(out, dtype=np.int32)


@pytest.mark.parametrize("S,b0,B,n", [(100, 52, 32, 3), (200, 128, 64, 15), (77, 0, 8, 9), (160, 32, 128, 2),
                                      (48, 32, 16, 1), (90, 58, 32, 0), (128, 0, 64, 3)])
def test_packed_forward_tiny_f32(P, tiny, S, b0, B, n):
    shape, w_np, model = tiny
    shared, packed = _packed_case(shape, S, b0, B, n, seed=S + B + n)
    lm_pos = _lm_pos(S, b0, B)
    scales = (1.0 + 6.0 * synth.uniform01_np(S, "s", S)).astype(np.float32)
    out = model.forward_packed(torch.from_numpy(packed).to(DEV), S, b0, B, n, torch.from_numpy(lm_pos).to(DEV),
                               row_scale=torch.from_numpy(scales).to(DEV), scale=2.0, pos_offset=3)
    torch.cuda.synchronize()
    logits = om.packed_logits(packed, w_np, shape, S, b0, B, n, lm_pos, pos_offset=3, row_scale=scales[lm_pos],
                              scale=2.0)
    ref = softmax_stats(logits.reshape(-1, shape.vocab), 16)
    print(compare_stats(out.numpy(), ref, 1e-4, label=f"packed f32 S{S} b0{b0} B{B} n{n}"))


def test_packed_forward_probe(P, tiny):
    from paper_2608_11742_amd._abi import Probe
    shape, w_np, model = tiny
    S, b0, B, n = 96, 32, 32, 4
    shared, packed = _packed_case(shape, S, b0, B, n, seed=21)
    lm_pos = np.arange(b0, b0 + B, dtype=np.int32)
    # probe rows index the LM-head rows: anchor rows first, then branch rows
    rows = np.array([0, 5, 31, B + 4, 3 * B + 30], dtype=np.int32)
    tk = np.array([3, 1000, 17, 9, 500], dtype=np.int32)
    pl = torch.zeros(len(rows), dtype=torch.float32, device=DEV)
    rows_d, tk_d = torch.from_numpy(rows).to(DEV), torch.from_numpy(tk).to(DEV)
    model.forward_packed(torch.from_numpy(packed).to(DEV), S, b0, B, n, torch.from_numpy(lm_pos).to(DEV),
                         scale=1.5, probe=Probe(rows_d.data_ptr(), tk_d.data_ptr(), pl.data_ptr(), len(rows)))
    torch.cuda.synchronize()
    logits = om.packed_logits(packed, w_np, shape, S, b0, B, n, lm_pos, scale=1.5).reshape(-1, shape.vocab)
    assert np.allclose(pl.cpu().numpy(), logits[rows, tk], atol=1e-4)


@pytest.mark.parametrize("S,b0,B,n", [(136, 64, 32, 5), (256, 192, 64, 15)])
def test_packed_forward_small_bf16_against_mirror(P, small_bf16, S, b0, B, n):
    shape, w_np, model = small_bf16
    shared, packed = _packed_case(shape, S, b0, B, n, seed=7 + n)
    lm_pos = np.arange(b0, b0 + B, dtype=np.int32)
    out = model.forward_packed(torch.from_numpy(packed).to(DEV), S, b0, B, n, torch.from_numpy(lm_pos).to(DEV),
                               scale=3.0)
    torch.cuda.synchronize()
    ref, *ref2 = [softmax_stats(om.packed_logits(packed, w, shape, S, b0, B, n, lm_pos, scale=3.0,
                                                mirror=True).reshape(-1, shape.vocab), 16)
                 for w in (w_np, *perturbations(w_np))]
    print(compare_stats(out.numpy(), ref, 2e-2, max_exceptions=allowed_flips(ref, ref2), id_ranks=4,
                        label=f"packed bf16 S{S} B{B} n{n}"), "oracle's own flips", flip_rows(ref, ref2))


def test_packed_forward_rejects_bad_shapes(P, tiny):
    shape, w_np, model = tiny
    t = torch.zeros(200, dtype=torch.int32, device=DEV)
    lm = torch.zeros(4, dtype=torch.int32, device=DEV)
    for S, b0, B, n in [(100, 52, 24, 3), (100, 90, 16, 2), (100, -1, 8, 2)]:
        with pytest.raises(RuntimeError):
            model.forward_packed(t[:S + n * B], S, b0, B, n, lm)


def test_build_packed(P):
    S, b0, B = 100, 36, 64
    toks = synth.tokens_np(9, "t", S, 299)
    toks[b0:] = 299
    m_pos = np.arange(b0, b0 + B, dtype=np.int32)
    rng = np.random.default_rng(5)
    logits = (rng.normal(0, 1, (B, 300)) * 3.0).astype(np.float32).astype(np.float64)
    logits[:, 299] = -np.inf
    ref = softmax_stats(logits, 16)
    st = P.Stats(B, 16, device=DEV)
    for name in ("H", "lse", "lmax", "argmax", "topk_id", "topk_logit"):
        dst = getattr(st, name)
        dst.copy_(torch.from_numpy(np.asarray(getattr(ref, name))).to(dst.dtype))
    plan = P.new_plan(DEV)
    P.rps_select_pivots(st, torch.from_numpy(m_pos).to(DEV), B, P.params(mode="band", n_pivots=3, r=0.0, n_cand=4),
                        plan)
    got_plan = P.read_plan(plan)
    cap = 13
    out = torch.full((S + cap * B,), -7, dtype=torch.int32, device=DEV)
    P.rps_build_packed(torch.from_numpy(toks).to(DEV), plan, b0, B, cap, out)
    o = out.cpu().numpy()
    assert got_plan.n_branch > 0
    assert np.array_equal(o[:S], toks)
    for c in range(cap):
        e = toks[b0:b0 + B].copy()
        if c < got_plan.n_branch:
            e[got_plan.br_pos[c] - b0] = got_plan.br_token[c]
        assert np.array_equal(o[S + c * B:S + (c + 1) * B], e)


def _event_key(e):
    return e[:-1] if e[0] in ("commit", "lookahead", "skip") else e


@pytest.mark.parametrize("tau_pivot,lam,seed", [(0.9, 0.1, 1), (0.6, 0.3, 2)])
def test_packed_decode_trajectory_matches_oracle(P, tiny, tau_pivot, lam, seed):
    shape, w_np, model = tiny
    Pl, G, B = 16, 64, 32
    prompt = synth.tokens_np(seed, "prompt", Pl, shape.vocab - 1)
    scales = synth.position_scales_np(seed + 10, np.arange(Pl + G), 2.6, 16.0)
    prm = P.params(mode="paper", k_max=10, tau_pivot=tau_pivot, n_pivots=1, r=0.1, n_cand=10, max_branch=15)
    toks, st = P.rps_decode(model, torch.from_numpy(prompt).to(DEV), G, B, prm, lam, 0.9, capacity=16,
                            row_scale=torch.from_numpy(scales).to(DEV), record=True, packed=True)
    got = toks.cpu().numpy()
    oprm = orps.Params(mode="paper", k_max=10, tau_pivot=tau_pivot, r=0.1, n_cand=10)
    ref = oracle_decode(model_forward(w_np, shape, scales=scales), prompt, G, B, shape.mask_id, oprm, lam, 0.9,
                        capacity=16, lookahead=model_packed_lookahead(w_np, shape, scales=scales))
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
    assert st.lookahead > 0
    print(f"packed: nfe {st.nfe} (lookahead {st.lookahead}), pivot commits {st.commits_pivot}, "
          f"abstains {st.abstains}, first excluded event {excluded}")


@pytest.mark.parametrize("Pn,S,B,n", [(40, 96, 32, 4), (77, 64, 64, 3), (130, 32, 32, 10)])
def test_packed_forward_over_a_prefix_tiny_f32(P, tiny, Pn, S, B, n):
    """The packed lookahead of a cached block: [block + suffix || block copies]
    (block_start 0) attending to a cached prefix, against the oracle."""
    from paper_2608_11742_amd._abi import KvCache
    shape, w_np, model = tiny
    prefix = synth.tokens_np(Pn, "prefix", Pn, shape.vocab - 1)
    k, vt, cap = model.new_kv_cache(Pn)
    kvc = KvCache(k.data_ptr(), vt.data_ptr(), 0, cap)
    model.forward(torch.from_numpy(prefix).to(DEV)[None], torch.arange(1, dtype=torch.int32, device=DEV),
                  kv_out=kvc)
    kvc.len = Pn
    shared, packed = _packed_case(shape, S, 0, B, n, seed=Pn + S)
    lm_pos = _lm_pos(S, 0, B)
    scales = (1.0 + 6.0 * synth.uniform01_np(Pn + 1, "s", S)).astype(np.float32)
    out = model.forward_packed(torch.from_numpy(packed).to(DEV), S, 0, B, n, torch.from_numpy(lm_pos).to(DEV),
                               row_scale=torch.from_numpy(scales).to(DEV), scale=2.0, pos_offset=Pn, kv_prefix=kvc)
    torch.cuda.synchronize()
    kv = om.prefix_cache(prefix, w_np, shape)
    logits = om.packed_logits(packed, w_np, shape, S, 0, B, n, lm_pos, pos_offset=Pn, row_scale=scales[lm_pos],
                              scale=2.0, prefix_kv=kv)
    ref = softmax_stats(logits.reshape(-1, shape.vocab), 16)
    print(compare_stats(out.numpy(), ref, 1e-4, label=f"packed over prefix {Pn}: S{S} B{B} n{n}"))


@pytest.mark.parametrize("tau_pivot,lam,seed", [(0.9, 0.1, 21), (0.6, 0.3, 22)])
def test_packed_cached_decode_trajectory_matches_oracle(P, tiny, tau_pivot, lam, seed):
    from oracle.decode import model_prefix_cached
    shape, w_np, model = tiny
    Pl, G, B = 16, 96, 32
    prompt = synth.tokens_np(seed, "prompt", Pl, shape.vocab - 1)
    scales = synth.position_scales_np(seed + 10, np.arange(Pl + G), 2.6, 16.0)
    prm = P.params(mode="paper", k_max=10, tau_pivot=tau_pivot, n_pivots=1, r=0.1, n_cand=10, max_branch=15)
    toks, st = P.rps_decode(model, torch.from_numpy(prompt).to(DEV), G, B, prm, lam, 0.9, capacity=16,
                            row_scale=torch.from_numpy(scales).to(DEV), record=True, packed=True, prefix_cache=True)
    got = toks.cpu().numpy()
    oprm = orps.Params(mode="paper", k_max=10, tau_pivot=tau_pivot, r=0.1, n_cand=10)
    ref = oracle_decode(model_forward(w_np, shape, scales=scales), prompt, G, B, shape.mask_id, oprm, lam, 0.9,
                        capacity=16, block_forward=model_prefix_cached(w_np, shape, scales=scales, packed=True))
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
    assert st.lookahead > 0
    print(f"packed + prefix cache: nfe {st.nfe} (lookahead {st.lookahead}), pivot commits {st.commits_pivot}, "
          f"abstains {st.abstains}, first excluded event {excluded}")
