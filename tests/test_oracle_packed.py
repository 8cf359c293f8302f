"""Pins of the oracle's packed lookahead forward (Section 4.1, lookahead
scoring; Algorithm 1's x_ahead = [x || x_b^(c_1) || ... ]): the masked
attention against torch's SDPA, the branch-isolating mask's invariants, and
the packed forward against forwards that need no mask at all (the plain
forward of the shared sequence, the independent forward of each branch with
one layer, the prefix-cache forward of each branch at any depth)."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import model as om
from synth import ModelShape

ONE = ModelShape(n_layers=1, d_model=64, n_heads=4, head_dim=16, d_ffn=96, vocab=101)
TWO = ModelShape(n_layers=2, d_model=64, n_heads=4, head_dim=16, d_ffn=96, vocab=101)


def _weights(shape, seed=0):
    return synth.model_weights_np(shape, seed=seed, dtype="f32")


def _case(shape, S=14, b0=6, B=4, n=3, seed=0):
    """Shared sequence with its block masked, and n branches that fill one
    pivot of the block with different tokens."""
    rng = np.random.default_rng(seed)
    shared = rng.integers(0, shape.vocab - 1, S)
    shared[b0:b0 + B] = shape.mask_id
    branches = []
    for c in range(n):
        blk = shared[b0:b0 + B].copy()
        blk[1] = rng.integers(0, shape.vocab - 1)
        branches.append(blk)
    return shared, branches, np.concatenate([shared] + branches)


def test_masked_attention_matches_torch_sdpa():
    rng = np.random.default_rng(1)
    q, k, v = (rng.normal(0, 1, (3, n, 16)) for n in (7, 11, 11))
    mask = rng.random((7, 11)) < 0.6
    mask[:, 0] = True                                   # every query keeps a key
    ref = F.scaled_dot_product_attention(*(torch.from_numpy(t) for t in (q, k, v)),
                                         attn_mask=torch.from_numpy(mask)).numpy()
    assert np.allclose(om.attention(q, k, v, mask), ref, atol=1e-12)


@pytest.mark.parametrize("S,b0,B,n", [(6, 2, 2, 2), (13, 0, 4, 3), (16, 8, 8, 1), (9, 5, 4, 0)])
def test_mask_isolates_branches_and_keeps_the_key_count(S, b0, B, n):
    pos, mask = om.packed_layout(S, b0, B, n, pos_offset=3)
    T = S + n * B
    assert mask.shape == (T, T) and pos.shape == (T,)
    assert np.all(np.diag(mask))                        # every row sees itself
    # every row attends to exactly S keys: as many as in an unpacked forward
    assert np.all(mask.sum(axis=1) == S)
    assert not mask[:S, S:].any()                       # the anchor never sees a branch
    for c in range(n):
        r = slice(S + c * B, S + (c + 1) * B)
        assert np.array_equal(pos[r], 3 + np.arange(b0, b0 + B))
        assert not mask[r, b0:b0 + B].any()            # a branch hides the block it replaces
        others = np.ones(T, dtype=bool)
        others[:S] = False
        others[r] = False
        assert not mask[r][:, others].any()             # ... and every other branch


def test_no_branch_is_the_plain_forward():
    w = _weights(TWO)
    shared, _, _ = _case(TWO)
    h = om.packed_hidden(shared, w, TWO, 14, 6, 4, 0, pos_offset=2)
    assert np.allclose(h, om.hidden(shared, w, TWO, pos_offset=2), atol=1e-12)


@pytest.mark.parametrize("mirror", [False, True])
def test_shared_rows_are_the_anchor_forward_at_any_depth(mirror):
    w = _weights(TWO, seed=1)
    shared, _, packed = _case(TWO, seed=1)
    h = om.packed_hidden(packed, w, TWO, 14, 6, 4, 3, mirror=mirror)
    ref = om.hidden(shared, w, TWO, mirror=mirror)
    # mirror=True rounds to bfloat16: identical arithmetic gives identical roundings
    assert np.allclose(h[:14], ref, atol=1e-12)


def test_one_layer_branch_rows_are_the_independent_forward():
    # With one layer every key and value is a function of its own token and
    # position, so a branch row sees exactly what the same row sees in the full
    # sequence with the block replaced.
    w = _weights(ONE, seed=2)
    shared, branches, packed = _case(ONE, seed=2)
    h = om.packed_hidden(packed, w, ONE, 14, 6, 4, 3, pos_offset=5)
    for c, blk in enumerate(branches):
        seq = shared.copy()
        seq[6:10] = blk
        ref = om.hidden(seq, w, ONE, pos_offset=5)
        assert np.allclose(h[14 + 4 * c:14 + 4 * (c + 1)], ref[6:10], atol=1e-12)


def test_branch_rows_are_the_block_forward_over_the_anchor_cache():
    # At any depth a branch's rows equal a forward of its block alone that
    # attends, in every layer, to the anchor's cached keys and values outside
    # the block: the prefix-cache path of the oracle, which uses no mask.
    w = _weights(TWO, seed=3)
    shared, branches, packed = _case(TWO, S=15, b0=5, B=4, seed=3)
    h = om.packed_hidden(packed, w, TWO, 15, 5, 4, 3)
    kv = []
    om.hidden(shared, w, TWO, collect=kv)
    keep = np.r_[0:5, 9:15]
    ctx = [(k[:, keep], v[:, keep]) for k, v in kv]
    for c, blk in enumerate(branches):
        ref = om.hidden(blk, w, TWO, pos_offset=5, prefix_kv=ctx)
        assert np.allclose(h[15 + 4 * c:15 + 4 * (c + 1)], ref, atol=1e-12)


def test_two_layers_differ_from_the_independent_forward():
    # the packing approximation is real beyond one layer: the shared rows keep
    # the anchor's block in their second-layer keys
    w = _weights(TWO, seed=4)
    shared, branches, packed = _case(TWO, seed=4)
    h = om.packed_hidden(packed, w, TWO, 14, 6, 4, 3)
    seq = shared.copy()
    seq[6:10] = branches[0]
    assert not np.allclose(h[14:18], om.hidden(seq, w, TWO)[6:10], atol=1e-6)


def test_branches_are_permutation_equivariant_and_independent():
    w = _weights(TWO, seed=5)
    shared, branches, packed = _case(TWO, n=3, seed=5)
    h = om.packed_hidden(packed, w, TWO, 14, 6, 4, 3)
    perm = [2, 0, 1]
    hp = om.packed_hidden(np.concatenate([shared] + [branches[i] for i in perm]), w, TWO, 14, 6, 4, 3)
    for j, i in enumerate(perm):
        assert np.allclose(hp[14 + 4 * j:18 + 4 * j], h[14 + 4 * i:18 + 4 * i], atol=1e-12)
    changed = [branches[0], branches[1].copy(), branches[2]]
    changed[1][3] = (changed[1][3] + 7) % (TWO.vocab - 1)
    hc = om.packed_hidden(np.concatenate([shared] + changed), w, TWO, 14, 6, 4, 3)
    assert np.allclose(hc[:18], h[:18], atol=1e-12) and np.allclose(hc[22:], h[22:], atol=1e-12)


def test_packed_logits_rows():
    w = _weights(TWO, seed=6)
    shared, branches, packed = _case(TWO, seed=6)
    lm_pos = np.array([2, 6, 7, 9, 13])
    rs = np.linspace(0.5, 2.0, 14)
    lg = om.packed_logits(packed, w, TWO, 14, 6, 4, 3, lm_pos, row_scale=rs[lm_pos], scale=1.3)
    assert lg.shape == (4, 5, TWO.vocab)
    anchor = om.forward_logits(shared[None], w, TWO, lm_pos, row_scale=rs[lm_pos], scale=1.3)[0]
    assert np.allclose(lg[0], anchor, atol=1e-10)
    h = om.packed_hidden(packed, w, TWO, 14, 6, 4, 3)
    for c in range(3):
        assert np.allclose(lg[1 + c][[0, 4]], anchor[[0, 4]], atol=1e-10)    # outside the block: shared rows
        ref = om.lm_logits(h[14 + 4 * c + np.array([0, 1, 3])], w, TWO, row_scale=rs[[6, 7, 9]], scale=1.3)
        assert np.allclose(lg[1 + c][1:4], ref, atol=1e-10)


def _prefix(shape, w, n=9, seed=11):
    toks = np.random.default_rng(seed).integers(0, shape.vocab - 1, n)
    kv = []
    om.hidden(toks, w, shape, collect=kv)
    return toks, kv


def test_packed_over_a_prefix_without_branches_is_the_cached_forward():
    w = _weights(TWO, seed=7)
    _, kv = _prefix(TWO, w)
    shared, _, _ = _case(TWO, seed=7)
    h = om.packed_hidden(shared, w, TWO, 14, 0, 4, 0, pos_offset=9, prefix_kv=kv)
    ref = om.hidden(shared, w, TWO, pos_offset=9, prefix_kv=kv)
    assert np.allclose(h, ref, atol=1e-12)


def test_packed_over_a_prefix_matches_the_cached_forwards():
    # shared rows: the cached forward of the shared sequence; branch rows: the
    # block alone over the prefix plus the anchor's keys outside the block
    w = _weights(TWO, seed=8)
    _, kv = _prefix(TWO, w)
    shared, branches, packed = _case(TWO, S=14, b0=0, B=4, seed=8)
    h = om.packed_hidden(packed, w, TWO, 14, 0, 4, 3, pos_offset=9, prefix_kv=kv)
    anchor = []
    ref = om.hidden(shared, w, TWO, pos_offset=9, prefix_kv=kv, collect=anchor)
    assert np.allclose(h[:14], ref, atol=1e-12)
    ctx = [(np.concatenate([pk, ak[:, 4:]], axis=1), np.concatenate([pv, av[:, 4:]], axis=1))
           for (pk, pv), (ak, av) in zip(kv, anchor)]
    for c, blk in enumerate(branches):
        hb = om.hidden(blk, w, TWO, pos_offset=9, prefix_kv=ctx)
        assert np.allclose(h[14 + 4 * c:18 + 4 * c], hb, atol=1e-12)
