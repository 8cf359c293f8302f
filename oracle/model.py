"""Oracle forward pass of the masked-diffusion transformer, float64.

The paper treats the dLLM as a black box that returns p_i = p_theta(. | y, x)
for every masked position in one forward pass over [y || x] (Section 3,
Notation).  The architecture used here is a LLaMA-style bidirectional
transformer: pre-RMSNorm (unit gain), rotate-half RoPE, full non-causal
softmax attention, SwiGLU feed-forward, untied embedding and LM head, no biases.

Every operation is its textbook definition written out once; matrix products
use numpy's matmul in float64.

``mirror=True`` rounds values at the points where the GPU contract stores
16-bit values: to bfloat16 (nearest-even) the inputs of every projection
(normed activations, attention output, SwiGLU output), Q and K after RoPE and
the final normed hidden state; to IEEE binary16 (nearest-even, saturated to
+-65504) the attention values V.  Everything else stays float64.
"""
from __future__ import annotations

import numpy as np


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value (ties to even), kept as float64."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    b = x.view(np.uint64)
    drop = np.uint64(45)                      # float64 keeps 52 mantissa bits, bfloat16 keeps 7
    half = np.uint64((1 << 44) - 1)
    lsb = (b >> drop) & np.uint64(1)
    with np.errstate(over="ignore"):
        r = ((b + half + lsb) >> drop) << drop
    return r.view(np.float64)


F16_MAX = 65504.0


def f16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest IEEE binary16 value (ties to even)
    after saturating them to the finite range +-65504, kept as float64."""
    x = np.clip(np.asarray(x, dtype=np.float64), -F16_MAX, F16_MAX)
    return x.astype(np.float16).astype(np.float64)


def rmsnorm(x: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) over the last axis (gain 1)."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def rope(u: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half rotary embedding.

    u: [..., S, hd]; pos: [S] absolute position ids.  For j < hd/2 the pair
    (u_j, u_{j+hd/2}) is rotated by the angle pos * base^(-2j/hd).
    """
    hd = u.shape[-1]
    half = hd // 2
    theta = base ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = pos.astype(np.float64)[:, None] * theta[None, :]
    c, s = np.cos(ang), np.sin(ang)
    u1, u2 = u[..., :half], u[..., half:]
    return np.concatenate([u1 * c - u2 * s, u1 * s + u2 * c], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, mask: np.ndarray | None = None) -> np.ndarray:
    """Non-causal softmax attention: softmax(q k^T / sqrt(hd)) v over all keys.

    q: [H, Sq, hd], k, v: [H, Sk, hd] -> [H, Sq, hd].  mask: optional boolean
    [Sq, Sk]; a query attends only to the keys where it is True (every row
    needs at least one).
    """
    hd = q.shape[-1]
    s = q @ np.swapaxes(k, -1, -2) / np.sqrt(hd)
    if mask is not None:
        s = np.where(mask[None], s, -np.inf)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    return p @ v


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def _w(weights, name) -> np.ndarray:
    return np.asarray(weights[name], dtype=np.float64)


def layer(x, weights, l, shape, pos, mirror=False, prefix_kv=None, collect=None, mask=None):
    """One transformer layer on one sequence.

    x: [S, d] residual stream; pos: [S] position ids.  prefix_kv: optional
    (k, v) of a cached prefix, each [H, P, hd] (post-RoPE); the S block
    positions then attend to the prefix keys followed by their own keys.
    collect: optional list that receives this layer's (k, v), each [H, S, hd].
    mask: optional boolean attention mask over the keys, [S, S], or
    [S, P + S] with a prefix.
    """
    R = bf16_round if mirror else (lambda t: t)
    RV = f16_round if mirror else (lambda t: t)
    S, d = x.shape
    H, hd = shape.n_heads, shape.head_dim
    a = R(rmsnorm(x, shape.rms_eps))
    qkv = a @ _w(weights, f"layers.{l}.wqkv").T                   # [S, 3d]
    q = qkv[:, 0 * d:1 * d].reshape(S, H, hd).transpose(1, 0, 2)  # [H, S, hd]
    k = qkv[:, 1 * d:2 * d].reshape(S, H, hd).transpose(1, 0, 2)
    v = qkv[:, 2 * d:3 * d].reshape(S, H, hd).transpose(1, 0, 2)
    q = R(rope(q, pos, shape.rope_base))
    k = R(rope(k, pos, shape.rope_base))
    v = RV(v)
    if collect is not None:
        collect.append((k, v))
    if prefix_kv is not None:
        kk = np.concatenate([prefix_kv[0], k], axis=1)
        vv = np.concatenate([prefix_kv[1], v], axis=1)
    else:
        kk, vv = k, v
    o = attention(q, kk, vv, mask).transpose(1, 0, 2).reshape(S, d)
    o = R(o)
    x = x + o @ _w(weights, f"layers.{l}.wo").T
    b = R(rmsnorm(x, shape.rms_eps))
    gu = b @ _w(weights, f"layers.{l}.wgu").T                     # [S, 2F]
    F = shape.d_ffn
    f = R(silu(gu[:, :F]) * gu[:, F:])
    return x + f @ _w(weights, f"layers.{l}.wdown").T


def hidden(tokens, weights, shape, pos_offset=0, mirror=False, prefix_kv=None, collect=None):
    """Final normed hidden states of one sequence.

    tokens: [S] int; positions are pos_offset + t.  prefix_kv: optional list
    (one entry per layer) of cached (k, v).  collect: optional list that
    receives per-layer (k, v).
    """
    tokens = np.asarray(tokens, dtype=np.int64)
    pos = pos_offset + np.arange(tokens.shape[0])
    x = _w(weights, "emb")[tokens]
    for l in range(shape.n_layers):
        x = layer(x, weights, l, shape, pos, mirror=mirror,
                  prefix_kv=None if prefix_kv is None else prefix_kv[l], collect=collect)
    h = rmsnorm(x, shape.rms_eps)
    return bf16_round(h) if mirror else h


def lm_logits(h, weights, shape, row_scale=None, scale=1.0):
    """Scaled LM-head logits with the [MASK] logit removed (set to -inf).

    h: [R, d].  logits = scale * row_scale_r * (h W_lm^T).
    """
    logits = h @ _w(weights, "lm_head").T
    s = np.full(h.shape[0], float(scale)) if row_scale is None else float(scale) * np.asarray(row_scale, np.float64)
    logits = logits * s[:, None]
    logits[:, shape.mask_id] = -np.inf
    return logits


def forward_logits(tokens_batch, weights, shape, lm_pos, pos_offset=0, mirror=False,
                   prefix_kv=None, row_scale=None, scale=1.0):
    """Logits at positions lm_pos of every sequence in the batch.

    tokens_batch: [B, S].  Returns [B, len(lm_pos), V] (float64).
    row_scale: optional per-position scale, indexed like lm_pos.
    """
    out = []
    for tokens in np.asarray(tokens_batch):
        h = hidden(tokens, weights, shape, pos_offset=pos_offset, mirror=mirror, prefix_kv=prefix_kv)
        out.append(lm_logits(h[np.asarray(lm_pos)], weights, shape, row_scale=row_scale, scale=scale))
    return np.stack(out)


def packed_layout(shared_len: int, block_start: int, block_len: int, n_branch: int, pos_offset: int = 0):
    """Position ids and attention mask of a packed lookahead sequence
    x_ahead = [x || x_b^(c_1) || ... || x_b^(c_n)] (Section 4.1, lookahead
    scoring; Algorithm 1).

    Rows 0 .. S-1 are the shared sequence x (the anchor); branch c occupies
    rows S + c*B .. S + (c+1)*B - 1 and stands in for the block b =
    block_start .. block_start+B-1 of x, so its rows take the block's position
    ids.  The mask isolates the branches: a shared row sees every shared row;
    a branch row sees the shared rows outside block b and the rows of its own
    branch.  Returns (pos [T], mask [T, T]) with T = S + n*B.
    """
    S, b0, B = shared_len, block_start, block_len
    T = S + n_branch * B
    grp = np.full(T, -1)                      # -1: shared row, c: branch c
    pos = pos_offset + np.arange(T)
    for c in range(n_branch):
        rows = slice(S + c * B, S + (c + 1) * B)
        grp[rows] = c
        pos[rows] = pos_offset + b0 + np.arange(B)
    in_block = np.zeros(T, dtype=bool)
    in_block[b0:b0 + B] = True
    mask = np.zeros((T, T), dtype=bool)
    for r in range(T):
        if grp[r] < 0:
            mask[r] = grp < 0
        else:
            mask[r] = ((grp < 0) & ~in_block) | (grp == grp[r])
    return pos, mask


def packed_hidden(tokens, weights, shape, shared_len, block_start, block_len, n_branch, pos_offset=0,
                  mirror=False, prefix_kv=None):
    """Final normed hidden states of every row of a packed lookahead sequence
    (tokens [S + n*B]); layout and mask of ``packed_layout``.  prefix_kv:
    optional per-layer cached (k, v) of positions before pos_offset, visible
    to every row (the prefix cache; the packed rows then start at pos_offset)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    pos, mask = packed_layout(shared_len, block_start, block_len, n_branch, pos_offset)
    assert tokens.shape[0] == pos.shape[0]
    x = _w(weights, "emb")[tokens]
    for l in range(shape.n_layers):
        if prefix_kv is None:
            x = layer(x, weights, l, shape, pos, mirror=mirror, mask=mask)
        else:
            P = prefix_kv[l][0].shape[1]
            full = np.concatenate([np.ones((mask.shape[0], P), dtype=bool), mask], axis=1)
            x = layer(x, weights, l, shape, pos, mirror=mirror, prefix_kv=prefix_kv[l], mask=full)
    h = rmsnorm(x, shape.rms_eps)
    return bf16_round(h) if mirror else h


def packed_logits(tokens, weights, shape, shared_len, block_start, block_len, n_branch, lm_pos, pos_offset=0,
                  mirror=False, row_scale=None, scale=1.0, prefix_kv=None):
    """Logits of a packed lookahead forward at positions lm_pos of the shared
    sequence, for the anchor and then for every branch: [1 + n, len(lm_pos), V].
    A branch reads its own row where the position lies in the block, else the
    shared row.  row_scale: optional per-position scale indexed like lm_pos."""
    S, b0, B = shared_len, block_start, block_len
    h = packed_hidden(tokens, weights, shape, S, b0, B, n_branch, pos_offset, mirror, prefix_kv=prefix_kv)
    lm_pos = np.asarray(lm_pos, dtype=np.int64)
    out = []
    for c in range(-1, n_branch):
        rows = np.array([S + c * B + (p - b0) if c >= 0 and b0 <= p < b0 + B else p for p in lm_pos],
                        dtype=np.int64)
        out.append(lm_logits(h[rows], weights, shape, row_scale=row_scale, scale=scale))
    return np.stack(out)


def prefix_cache(tokens, weights, shape, mirror=False):
    """Post-RoPE per-layer (k, v) of a prefix forward pass, each [H, P, hd]."""
    kv = []
    hidden(tokens, weights, shape, mirror=mirror, collect=kv)
    return kv
