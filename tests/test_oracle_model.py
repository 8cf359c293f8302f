"""Pins of the oracle transformer against library routines and invariants."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import model as om
from synth import ModelShape

SMALL = ModelShape(n_layers=2, d_model=64, n_heads=4, head_dim=16, d_ffn=96, vocab=101)


def _weights(shape, seed=0):
    return synth.model_weights_np(shape, seed=seed, dtype="f32")


def test_rmsnorm_matches_torch():
    x = np.random.default_rng(0).normal(0, 2, (5, 64))
    ref = F.rms_norm(torch.from_numpy(x), (64,), eps=1e-5).numpy()
    assert np.allclose(om.rmsnorm(x, 1e-5), ref, atol=1e-12)


def test_silu_matches_torch():
    x = np.linspace(-20, 20, 101)
    assert np.allclose(om.silu(x), F.silu(torch.from_numpy(x)).numpy(), atol=1e-14)


def test_attention_matches_torch_sdpa():
    rng = np.random.default_rng(1)
    q, k, v = (rng.normal(0, 1, (3, n, 16)) for n in (7, 11, 11))
    ref = F.scaled_dot_product_attention(*(torch.from_numpy(t) for t in (q, k, v))).numpy()
    assert np.allclose(om.attention(q, k, v), ref, atol=1e-12)


def test_attention_key_permutation_invariance_and_query_equivariance():
    rng = np.random.default_rng(2)
    q, k, v = (rng.normal(0, 1, (2, 13, 16)) for _ in range(3))
    pk = rng.permutation(13)
    assert np.allclose(om.attention(q, k[:, pk], v[:, pk]), om.attention(q, k, v), atol=1e-12)
    pq = rng.permutation(13)
    assert np.allclose(om.attention(q[:, pq], k, v), om.attention(q, k, v)[:, pq], atol=1e-12)


def test_rope_relative_position_and_norm():
    rng = np.random.default_rng(3)
    hd = 16
    q = rng.normal(0, 1, (1, 1, hd))
    k = rng.normal(0, 1, (1, 1, hd))
    dots = {}
    for m, n in [(3, 1), (10, 8), (102, 100), (7, 9), (0, 2)]:
        qm = om.rope(q, np.array([m]), 10000.0)
        kn = om.rope(k, np.array([n]), 10000.0)
        dots.setdefault(m - n, []).append(float((qm * kn).sum()))
    for vals in dots.values():
        assert np.allclose(vals, vals[0], atol=1e-10)
    # rotation preserves norms and is the identity at position 0
    r = om.rope(q, np.array([37]), 10000.0)
    assert np.isclose(np.linalg.norm(r), np.linalg.norm(q))
    assert np.allclose(om.rope(q, np.array([0]), 10000.0), q)


def test_rope_pairs_rotate_half():
    # the first frequency is 1 rad per position and pairs (j, j + hd/2)
    u = np.zeros((1, 1, 8))
    u[0, 0, 0] = 1.0
    r = om.rope(u, np.array([1]), 10000.0)[0, 0]
    assert np.isclose(r[0], math.cos(1.0)) and np.isclose(r[4], math.sin(1.0))
    assert np.allclose(np.delete(r, [0, 4]), 0.0)


def test_bf16_round_matches_torch_on_float32_values():
    x = synth.weight_np(5, "r", (10000,), std=10.0, dtype="f32")
    ours = om.bf16_round(x.astype(np.float64))
    theirs = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, theirs)
    # ties go to even: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7
    assert om.bf16_round(np.array([1.0 + 2 ** -8]))[0] == 1.0
    assert om.bf16_round(np.array([1.0 + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6


def test_f16_round_matches_torch_and_saturates():
    """The mirror's binary16 rounding of attention values: torch's float16
    conversion (round to nearest even) on values inside the finite range,
    including subnormals, and saturation to +-65504 beyond it."""
    x = np.concatenate([synth.weight_np(6, "r", (10000,), std=10.0, dtype="f32"),
                        synth.weight_np(7, "r", (2000,), std=1e-5, dtype="f32")]).astype(np.float64)
    ours = om.f16_round(x)
    theirs = torch.from_numpy(x).to(torch.float16).to(torch.float64).numpy()
    assert np.array_equal(ours, theirs)
    # ties go to even: 1 + 2^-11 lies halfway between 1 and 1 + 2^-10
    assert om.f16_round(np.array([1.0 + 2 ** -11]))[0] == 1.0
    assert om.f16_round(np.array([1.0 + 3 * 2 ** -11]))[0] == 1.0 + 2 ** -9
    # smallest subnormal, and beyond the finite range
    assert om.f16_round(np.array([2.0 ** -24]))[0] == 2.0 ** -24
    assert list(om.f16_round(np.array([65504.0, 70000.0, -1e9]))) == [65504.0, 65504.0, -65504.0]


def test_degenerate_weights_reduce_to_embedding_lookup():
    w = _weights(SMALL)
    for l in range(SMALL.n_layers):
        w[f"layers.{l}.wo"] = np.zeros_like(w[f"layers.{l}.wo"])
        w[f"layers.{l}.wdown"] = np.zeros_like(w[f"layers.{l}.wdown"])
    toks = np.array([[3, 9, 27, 81, 0, 5]])
    logits = om.forward_logits(toks, w, SMALL, lm_pos=[1, 4], scale=2.0)
    emb = w["emb"].astype(np.float64)[toks[0, [1, 4]]]
    h = emb / np.sqrt((emb ** 2).mean(1, keepdims=True) + SMALL.rms_eps)
    ref = 2.0 * h @ w["lm_head"].astype(np.float64).T
    ref[:, SMALL.mask_id] = -np.inf
    assert np.allclose(logits[0], ref, atol=1e-12)


def test_forward_is_non_causal_and_batch_independent():
    w = _weights(SMALL)
    rng = np.random.default_rng(4)
    toks = rng.integers(0, SMALL.vocab - 1, (2, 9))
    a = om.forward_logits(toks, w, SMALL, lm_pos=[0])
    t2 = toks.copy()
    t2[:, -1] = (t2[:, -1] + 1) % (SMALL.vocab - 1)
    b = om.forward_logits(t2, w, SMALL, lm_pos=[0])
    assert not np.allclose(a, b)                        # position 0 sees the last token
    single = om.forward_logits(toks[1:], w, SMALL, lm_pos=[0])
    assert np.allclose(a[1:], single)


def test_one_layer_cached_prefix_equals_full_forward():
    # With one layer the prefix keys/values only depend on the embeddings, so
    # attending to a cached prefix is exactly the full-sequence forward.
    shape = ModelShape(n_layers=1, d_model=64, n_heads=4, head_dim=16, d_ffn=96, vocab=101)
    w = _weights(shape)
    rng = np.random.default_rng(5)
    toks = rng.integers(0, shape.vocab - 1, 12)
    full = om.forward_logits(toks[None], w, shape, lm_pos=np.arange(8, 12))
    kv = om.prefix_cache(toks[:8], w, shape)
    h = om.hidden(toks[8:], w, shape, pos_offset=8, prefix_kv=kv)
    cached = om.lm_logits(h, w, shape)
    assert np.allclose(full[0], cached, atol=1e-12)


def test_position_offset_shifts_rope_only():
    # the same tokens at a shifted offset give the same outputs (relative positions
    # are all that attention sees when every position shifts together)
    w = _weights(SMALL)
    toks = np.random.default_rng(6).integers(0, SMALL.vocab - 1, 10)
    a = om.hidden(toks, w, SMALL, pos_offset=0)
    b = om.hidden(toks, w, SMALL, pos_offset=57)
    assert np.allclose(a, b, atol=1e-9)


def _torch_layer(x, w, l, shape, pos):
    """One layer from torch library routines: F.linear ([out, in] weights),
    F.rms_norm, scaled_dot_product_attention and rotary embedding written as a
    complex rotation of (u_j, u_{j+hd/2}) pairs."""
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    d, H, hd, Fd = shape.d_model, shape.n_heads, shape.head_dim, shape.d_ffn
    x = t(x)
    a = F.rms_norm(x, (d,), eps=shape.rms_eps)
    q, k, v = F.linear(a, t(w[f"layers.{l}.wqkv"])).split(d, dim=-1)
    half = hd // 2
    freqs = shape.rope_base ** (-torch.arange(half, dtype=torch.float64) * 2 / hd)
    rot = torch.polar(torch.ones(len(pos), half, dtype=torch.float64), t(pos)[:, None] * freqs[None])

    def rope(u):
        u = u.view(-1, H, hd)
        z = torch.complex(u[..., :half], u[..., half:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1).transpose(0, 1)      # [H, S, hd]
    o = F.scaled_dot_product_attention(rope(q), rope(k), v.view(-1, H, hd).transpose(0, 1))
    x = x + F.linear(o.transpose(0, 1).reshape(-1, d), t(w[f"layers.{l}.wo"]))
    b = F.rms_norm(x, (d,), eps=shape.rms_eps)
    g, u = F.linear(b, t(w[f"layers.{l}.wgu"])).split(Fd, dim=-1)
    return (x + F.linear(F.silu(g) * u, t(w[f"layers.{l}.wdown"]))).numpy()


def test_layer_matches_torch_composition():
    w = _weights(SMALL, seed=3)
    rng = np.random.default_rng(7)
    x = rng.normal(0, 1, (11, SMALL.d_model))
    pos = np.arange(5, 16)
    ours = om.layer(x, w, 1, SMALL, pos)
    ref = _torch_layer(x, w, 1, SMALL, pos)
    assert np.allclose(ours, ref, atol=1e-10)
