"""Shared helpers for the GPU tests: device placement, tolerances, case announcements."""
import sys

import numpy as np
import torch

# Tolerances vs the fp64 oracle: fp32 max-abs 1e-5; bf16 |d| <= 2e-2 + 1e-2 |oracle|.
F32_ATOL = 1e-5
BF16_ATOL, BF16_RTOL = 2e-2, 1e-2
LSE_BF16_ATOL = 2e-2


def announce(msg: str) -> None:
    """Name the case on stderr before a GPU step, so a hang or fault is attributable."""
    print(f"[gpu-case] {msg}", file=sys.stderr, flush=True)


def to_dev(a: dict, keys=("q", "k_live", "v_live", "k_cache", "v_cache", "seed_idx", "n_seed")):
    return [a[k].cuda() for k in keys]


def check_attn(out_gpu, lse_gpu, out_ref, lse_ref, dtype, where=""):
    o = out_gpu.double().cpu().numpy().reshape(out_ref.shape)
    err = np.abs(o - out_ref)
    if dtype == torch.float32:
        assert err.max() <= F32_ATOL, f"{where}: out max-abs {err.max():.3e}"
    else:
        bad = err > BF16_ATOL + BF16_RTOL * np.abs(out_ref)
        assert not bad.any(), f"{where}: {bad.sum()} out elements off; max-abs {err.max():.3e}"
    if lse_gpu is not None and lse_ref is not None:
        l = lse_gpu.double().cpu().numpy().reshape(lse_ref.shape)
        le = np.abs(l - lse_ref).max()
        tol = F32_ATOL if dtype == torch.float32 else LSE_BF16_ATOL
        assert le <= tol, f"{where}: lse max-abs {le:.3e}"
    return float(err.max())
