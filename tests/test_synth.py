"""The seeded input generators: both backends agree bit for bit."""
import numpy as np
import pytest
import torch

import synth
from synth import inputs as si


def test_splitmix_reference_values():
    # SplitMix64 seeded with 0: first outputs of the published generator
    r = si.counter_u64_np(0, 0, 3)
    assert [int(x) for x in r] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_fnv1a64_reference_values():
    assert si.fnv1a64("") == 0xCBF29CE484222325
    assert si.fnv1a64("a") == 0xAF63DC4C8601EC8C


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_numpy_and_torch_backends_identical(dtype):
    a = si.weight_np(7, "layers.3.wqkv", (96, 80), dtype=dtype)
    b = si.weight_torch(7, "layers.3.wqkv", (96, 80), dtype=dtype, chunk=1000).float().numpy()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    ta = si.tokens_np(1, "prompt", 1000, 1023)
    tb = si.tokens_torch(1, "prompt", 1000, 1023).numpy()
    assert np.array_equal(ta, tb)


def test_bf16_rounding_matches_torch():
    x = si.weight_np(3, "x", (4096,), std=3.0, dtype="f32")
    ours = si.f32_to_bf16_bits(x)
    theirs = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, theirs)


def test_weight_distribution():
    w = si.weight_np(0, "w", (512, 512), dtype="f32").astype(np.float64)
    assert abs(w.mean()) < 2e-4
    assert abs(w.std() - 0.02) < 2e-4
    assert np.abs(w).max() <= 0.02 * 3.47          # Irwin-Hall(4) support is +-sqrt(12) sigma


def test_tokens_uniform_and_exclude_mask():
    t = si.tokens_np(1, "prompt", 200000, 1023)
    assert t.min() == 0 and t.max() == 1022
    counts = np.bincount(t, minlength=1023)
    assert counts.std() / counts.mean() < 0.1


def test_workloads_consistent():
    for w in synth.WORKLOADS.values():
        assert w.n_cand <= w.k_max <= w.topk <= 16
        assert w.model.d_model == w.model.n_heads * w.model.head_dim
        assert w.gen_len % w.block == 0
