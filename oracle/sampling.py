"""Sampled targets for speculative sampling (oracle side; test infrastructure only).

The paper evaluates greedy decoding and mentions a tree sampling algorithm without
describing it (Sec. 4.1).  The reading taken here keeps acceptance lossless for any
candidate tree: at every tree node the target draws its own next token from
softmax(logits / temperature), and the walk of greedy acceptance (Sec. 2.1) follows the
child carrying that token.  Every emitted token is then a sample of the target model
given the tokens before it, so speculative sampling emits what sampling the target
token by token would, in distribution.

The draw is Gumbel-max: argmax_v (logit_v / temperature + G_v) with independent standard
Gumbel variables G_v = -log(-log(U_v)), which is an exact sample of the softmax.  The
uniforms come from the counter-based generator Philox4x32-10 (Salmon, Moraes, Dror and
Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011), one draw per counter
(vocab id, tree node, step of the sequence, sequence slot) under the key (seed, domain),
so the GPU draws the same numbers without sharing any code with this module.
"""
import numpy as np

_M0, _M1 = np.uint64(0xD2511F53), np.uint64(0xCD9E8D57)
_W0, _W1 = 0x9E3779B9, 0xBB67AE85
_MASK = np.uint64(0xFFFFFFFF)

DOMAIN_VERIFY = 0   # targets of the tree nodes in a speculate-and-verify step
DOMAIN_PREFILL = 1  # the first token after the prompt


def philox4x32_10_w0(c0, c1, c2, c3, k0: int, k1: int) -> np.ndarray:
    """First output word of Philox4x32-10 for the (broadcast) counters and the key."""
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) & _MASK for c in (c0, c1, c2, c3))
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    for r in range(10):
        ka, kb = np.uint64((k0 + r * _W0) & 0xFFFFFFFF), np.uint64((k1 + r * _W1) & 0xFFFFFFFF)
        p0 = _M0 * c0
        p1 = _M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK
        c0, c1, c2, c3 = hi1 ^ c1 ^ ka, lo1, hi0 ^ c3 ^ kb, lo0
    return c0.astype(np.uint32)


def uniform_from_bits(x) -> np.ndarray:
    """U = (m + 1/2) / 2^23 with m the top 23 bits of each 32-bit word.

    m + 1/2 needs at most 24 significant bits, so the sum and the scaling are exact in
    float32, and U runs over the midpoints 2^-24, 3 * 2^-24, ..., 1 - 2^-24: strictly
    inside (0, 1), which keeps both logarithms of the Gumbel transform finite.  (With
    the top 24 bits the sum m + 1/2 would need 25 bits and round, up to 1.0 for the
    largest words.)"""
    return ((np.asarray(x, dtype=np.uint32) >> np.uint32(9)).astype(np.float32) + np.float32(0.5)) \
        * np.float32(2.0 ** -23)


def gumbel_from_bits(x) -> np.ndarray:
    u = uniform_from_bits(x)
    return -np.log(-np.log(u))  # float32 throughout


def gumbel_scores(logits, temperature: float, seed: int, domain: int, step, slot, node) -> np.ndarray:
    """float32 logit / temperature + Gumbel noise of every vocab entry (last axis) of one draw,
    or of one draw per leading row when step, slot or node are arrays over the rows."""
    lg = np.asarray(logits, dtype=np.float32)
    v = np.arange(lg.shape[-1], dtype=np.uint64)
    col = (lambda a: np.asarray(a, dtype=np.uint64).reshape(-1, 1)) if lg.ndim == 2 else np.asarray
    x = philox4x32_10_w0(v, col(node), col(step), col(slot), seed & 0xFFFFFFFF, domain)
    inv = np.float32(1.0) / np.float32(temperature)  # the reciprocal in float32, as the GPU takes it
    return lg * inv + gumbel_from_bits(x)


def sample_token(logits, temperature: float, seed: int, domain: int, step: int, slot: int,
                 node: int) -> int:
    """The target's sampled token for one draw (lowest id on an exact tie)."""
    return int(np.argmax(gumbel_scores(logits, temperature, seed, domain, step, slot, node)))


def sample_tokens(logits, temperature: float, seed: int, domain: int, step, slot, node) -> np.ndarray:
    """One draw per row of logits [rows, V]; step, slot and node broadcast over the rows."""
    return np.argmax(gumbel_scores(logits, temperature, seed, domain, step, slot, node), axis=-1)
