"""Model handle: weights in HBM, the library handle and a reusable workspace."""
from __future__ import annotations

import torch

from . import binding as B
from ._abi import ModelDesc, KvCache, DLLM_BF16, DLLM_F32


class Model:
    """A bidirectional masked-diffusion transformer held by libdllm_rps.

    shape: any object with n_layers, d_model, n_heads, head_dim, d_ffn, vocab,
    mask_id, rope_base and rms_eps.  weights: {"emb", "lm_head",
    "layers.{l}.wqkv", "layers.{l}.wo", "layers.{l}.wgu", "layers.{l}.wdown"}
    device tensors of the model dtype ([out][in] layout).
    """

    def __init__(self, shape, weights: dict, dtype: str = "bf16", max_pos: int = 4096):
        if dtype not in ("bf16", "f32"):
            raise ValueError(dtype)
        self.shape = shape
        self.dtype = dtype
        self.torch_dtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.device = weights["emb"].device
        L = shape.n_layers
        self._w = {"emb": weights["emb"], "lm_head": weights["lm_head"]}
        for name in ("wqkv", "wo", "wgu", "wdown"):
            self._w[name] = [weights[f"layers.{l}.{name}"] for l in range(L)]
        for t in [self._w["emb"], self._w["lm_head"]] + sum((self._w[n] for n in ("wqkv", "wo", "wgu", "wdown")), []):
            if t.dtype != self.torch_dtype or not t.is_contiguous() or t.device != self.device:
                raise ValueError("weights must be contiguous device tensors of the model dtype")
        self.desc = ModelDesc(L, shape.d_model, shape.n_heads, shape.head_dim, shape.d_ffn, shape.vocab,
                              shape.mask_id, shape.rope_base, shape.rms_eps,
                              DLLM_BF16 if dtype == "bf16" else DLLM_F32, max_pos)
        self.handle = B.dllm_model_create(self.desc, self._w)
        self._ws = None

    def close(self):
        if self.handle is not None:
            B.dllm_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _reserve(self, need: int):
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        return self._ws

    def workspace(self, batch: int, seq: int, n_lm_pos: int):
        return self._reserve(B.dllm_workspace_bytes(self.handle, batch, seq, n_lm_pos))

    def workspace_packed(self, shared_len: int, block_len: int, n_branch: int, n_lm_pos: int):
        return self._reserve(B.dllm_workspace_bytes_packed(self.handle, shared_len, block_len, n_branch, n_lm_pos))

    def new_kv_cache(self, cap: int):
        """Device buffers for a prefix cache of `cap` positions (cap rounded up to 8).

        Keys in the model's dtype; values (transposed) in IEEE float16 for
        bf16 models, float32 for fp32 models."""
        cap = (cap + 7) // 8 * 8
        s = self.shape
        k = torch.empty(s.n_layers, s.n_heads, cap, s.head_dim, dtype=self.torch_dtype, device=self.device)
        v_dtype = torch.float16 if self.torch_dtype == torch.bfloat16 else self.torch_dtype
        vt = torch.empty(s.n_layers, s.n_heads, s.head_dim, cap, dtype=v_dtype, device=self.device)
        return k, vt, cap

    def forward(self, tokens, lm_pos, out: B.Stats | None = None, n_lm_pos: int | None = None, row_scale=None,
                scale: float = 1.0, pos_offset: int = 0, kv_prefix: KvCache | None = None,
                kv_out: KvCache | None = None, probe=None, k: int = 16, stream=None) -> B.Stats:
        if tokens.dim() == 1:
            tokens = tokens[None]
        n = lm_pos.shape[0] if n_lm_pos is None else n_lm_pos
        if out is None:
            out = B.Stats(tokens.shape[0] * n, k, device=self.device)
        ws = self.workspace(tokens.shape[0], tokens.shape[1], n)
        B.dllm_forward(self.handle, tokens, lm_pos, out, ws, pos_offset=pos_offset, row_scale=row_scale, scale=scale,
                       kv_prefix=kv_prefix, kv_out=kv_out, probe=probe, n_lm_pos=n, stream=stream)
        return out

    def forward_packed(self, tokens, shared_len: int, block_start: int, block_len: int, n_branch: int, lm_pos,
                       out: B.Stats | None = None, n_lm_pos: int | None = None, row_scale=None, scale: float = 1.0,
                       pos_offset: int = 0, kv_prefix: KvCache | None = None, probe=None, k: int = 16,
                       stream=None) -> B.Stats:
        """Packed lookahead forward over [shared || n_branch block copies] (one
        sequence, branch-isolating mask); returns (1 + n_branch) * n_lm_pos rows."""
        n = lm_pos.shape[0] if n_lm_pos is None else n_lm_pos
        if out is None:
            out = B.Stats((1 + n_branch) * n, k, device=self.device)
        ws = self.workspace_packed(shared_len, block_len, n_branch, n)
        B.dllm_forward_packed(self.handle, tokens, shared_len, block_start, block_len, n_branch, lm_pos, out, ws,
                              pos_offset=pos_offset, kv_prefix=kv_prefix, row_scale=row_scale, scale=scale,
                              probe=probe, n_lm_pos=n, stream=stream)
        return out
