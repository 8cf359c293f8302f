"""MI355X (gfx950) library for one batched denoising step of Ripple-Pivot
Search over a bidirectional masked-diffusion transformer.

The compute runs in libdllm_rps.so (hand-written HIP, C ABI declared in
include/dllm_rps.h); this package marshals torch tensors into that ABI.
Importing the package loads the library and fails if it is not built.
"""
from . import binding  # noqa: F401
from .binding import (  # noqa: F401
    Stats, dllm_model_create, dllm_model_destroy, dllm_workspace_bytes, dllm_forward, dllm_forward_packed,
    vocab_entropy_topk, vocab_entropy_topk_noalloc, vocab_entropy_topk_workspace_bytes, rps_select_pivots, rps_build_branches, rps_build_packed,
    dllm_workspace_bytes_packed,
    rps_lookahead_score, rps_commit, sched_commit, params, new_plan, new_decision, read_plan, read_decision, lib,
    dllm_profile_begin, dllm_profile_end, dllm_mfma_ceiling,
)
from .model import Model  # noqa: F401
from .step import RpsStep, rps_decode, baseline_decode  # noqa: F401

lib()  # fail loudly here if the HIP library is missing
