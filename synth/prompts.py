"""Uniform-random prompt tokens (stand-in for the paper's internal dialogues)."""
import torch

from .configs import CloverConfig


def make_prompt_lengths(c: CloverConfig, seed: int = 2):
    lo, hi = c.prompt_len
    g = torch.Generator().manual_seed(seed * 7_777 + 3)
    return [int(x) for x in torch.randint(lo, hi + 1, (c.batch,), generator=g)]


def make_prompt(c: CloverConfig, seq: int = 0, n: int = None, seed: int = 1):
    if n is None:
        n = c.prompt_len[0]
    g = torch.Generator().manual_seed(seed * 1_000_033 + seq * 131 + 7)
    return [int(x) for x in torch.randint(0, c.vocab, (n,), generator=g)]
