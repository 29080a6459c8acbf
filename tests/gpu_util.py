"""Shared helpers for the GPU tests (not collected)."""
import sys

import numpy as np
import pytest
import torch


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2405_00263_amd as P  # raises if the library is missing
    return P


def note(msg: str):
    """Name the case before a GPU step so a crash log shows it."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def to_np(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def seeded(shape, seed, scale=1.0, dtype=torch.float32, device="cuda"):
    g = torch.Generator(device=device).manual_seed(seed)
    return (torch.randn(shape, generator=g, device=device) * scale).to(dtype)


def mask_words(mask_bool: np.ndarray) -> np.ndarray:
    T = mask_bool.shape[0]
    W = (T + 63) // 64
    out = np.zeros((T, W), dtype=np.uint64)
    for i in range(T):
        for j in np.nonzero(mask_bool[i])[0]:
            out[i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    return out
