"""The allocation-free LM head (vocab_entropy_topk_noalloc, partial statistics
in the library's device scratch) against the workspace entry point
(vocab_entropy_topk) through the C ABI: two calls in a row, the second on a
smaller input, and the size limit."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _case(R, d, V, seed):
    h = synth.weight_torch(seed, "h", (R, d), std=1.0, dtype="bf16", device=DEV)
    w = synth.weight_torch(seed + 1, "w", (V, d), dtype="bf16", device=DEV)
    rs = torch.from_numpy((0.5 + 3 * synth.uniform01_np(seed + 2, "rs", R)).astype(np.float32)).to(DEV)
    return h, w, rs


def test_noalloc_matches_the_workspace_entry_point_on_consecutive_calls():
    import paper_2608_11742_amd as P
    # the 8B vocabulary at 300 rows (two 256-row tiles), then fewer rows and a
    # smaller ragged vocabulary (one 128-row tile, more partials per row):
    # the second call must not see the first call's partials
    for R, d, V, seed in [(300, 512, 126464, 60), (37, 256, 30011, 63)]:
        h, w, rs = _case(R, d, V, seed)
        ref = P.Stats(R, 16, device=DEV)
        ws = torch.empty(P.vocab_entropy_topk_workspace_bytes(R, V), dtype=torch.uint8, device=DEV)
        P.vocab_entropy_topk(h, w, ref, ws, row_scale=rs, scale=1.0, mask_id=V - 1)
        got = P.Stats(R, 16, device=DEV)
        got.fill_(float("nan"))
        P.vocab_entropy_topk_noalloc(h, w, got, row_scale=rs, scale=1.0, mask_id=V - 1)
        torch.cuda.synchronize()
        a, b = ref.numpy(), got.numpy()
        for k in ("H", "lse", "lmax", "argmax", "topk_id", "topk_logit"):
            assert np.array_equal(a[k], b[k]), (R, V, k)
        assert np.all(np.isfinite(b["H"]))


def test_noalloc_rejects_inputs_beyond_its_scratch():
    import paper_2608_11742_amd as P
    R, d, V = 262144, 64, 300          # 2 partials of 140 bytes per row: 73 MB > 48 MiB
    h = torch.zeros(R, d, dtype=torch.bfloat16, device=DEV)
    w = torch.zeros(V, d, dtype=torch.bfloat16, device=DEV)
    assert P.vocab_entropy_topk_workspace_bytes(R, V) > (48 << 20)
    out = P.Stats(R, 16, device=DEV)
    with pytest.raises(RuntimeError, match="scratch"):
        P.vocab_entropy_topk_noalloc(h, w, out, mask_id=V - 1)
