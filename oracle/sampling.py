"""Counter-based seeded sampling -- oracle, test infrastructure only.

Rollout draws each response token from softmax(logits / T).  The draw is made
order-independent with the Gumbel-max construction: token = argmax_v
(logits_v / T + g_v), g_v = -ln(-ln u_v), with u_v from the Philox4x64-10
counter-based generator (Salmon, Moraes, Dror, Shaw, "Parallel random numbers:
as easy as 1, 2, 3", SC'11), keyed by (seed, seq_id) and counted by
(position, v // 8, 0, 0).  Each 256-bit block gives eight 32-bit words (the
low half of each 64-bit output first); word w maps to
u = ((w >> 9) + 0.5) * 2^-23, exactly representable in fp32 (24 significant
bits), so u lies in [2^-24, 1 - 2^-24].

Temperature 0 is greedy argmax.  Ties go to the lowest vocabulary index.
The logits/T + g sum and the argmax are taken in fp32, the precision of the
kernel, since that arithmetic decides an integer.

RL training needs the log-probability of each sampled token under the
distribution it was drawn from: log softmax(logits / T)[token], computed here
in fp64.  For greedy decoding (T = 0) the reported value is taken at T = 1.
A response that stops at an end-of-sequence token is the forced-length
response cut after the first occurrence of that token: tokens are keyed by
position, so stopping changes nothing before it.
"""
from __future__ import annotations

import numpy as np

_M0 = np.uint64(0xD2E7470EE14C6C93)
_M1 = np.uint64(0xCA5A826395121157)
_W0 = np.uint64(0x9E3779B97F4A7C15)
_W1 = np.uint64(0xBB67AE8584CAA73B)
_LO32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo64(a: np.ndarray, b: np.uint64):
    """Full 128-bit product of uint64 arrays, from 32-bit limbs: (hi, lo)."""
    a_lo, a_hi = a & _LO32, a >> _S32
    b_lo, b_hi = b & _LO32, b >> _S32
    p00 = a_lo * b_lo
    p01 = a_lo * b_hi
    p10 = a_hi * b_lo
    p11 = a_hi * b_hi
    mid = (p00 >> _S32) + (p01 & _LO32) + (p10 & _LO32)
    hi = p11 + (p01 >> _S32) + (p10 >> _S32) + (mid >> _S32)
    lo = a * b
    return hi, lo


def philox4x64_10(counter: np.ndarray, key) -> np.ndarray:
    """Philox4x64 with 10 rounds.

    counter: uint64 [..., 4]; key: (k0, k1).  Returns uint64 [..., 4].
    Each round: (hi0, lo0) = M0 * x0, (hi1, lo1) = M1 * x2,
    x = (hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0); then the key is bumped by
    the Weyl constants.
    """
    with np.errstate(over="ignore"):
        x = np.array(counter, dtype=np.uint64, copy=True)
        x0, x1, x2, x3 = x[..., 0], x[..., 1], x[..., 2], x[..., 3]
        k0, k1 = np.uint64(key[0]), np.uint64(key[1])
        for _ in range(10):
            hi0, lo0 = _mulhilo64(x0, _M0)
            hi1, lo1 = _mulhilo64(x2, _M1)
            x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
            k0 = k0 + _W0
            k1 = k1 + _W1
    return np.stack([x0, x1, x2, x3], axis=-1)


def uniforms(seed: int, seq_id: int, pos: int, vocab: int) -> np.ndarray:
    """u_v in (0, 1) as float32 for v < vocab."""
    groups = (vocab + 7) // 8
    ctr = np.zeros((groups, 4), np.uint64)
    ctr[:, 0] = np.uint64(pos)
    ctr[:, 1] = np.arange(groups, dtype=np.uint64)
    out = philox4x64_10(ctr, (np.uint64(seed), np.uint64(seq_id)))       # [groups, 4]
    words = np.empty((groups, 8), np.uint64)
    words[:, 0::2] = out & _LO32
    words[:, 1::2] = out >> _S32
    w = words.reshape(-1)[:vocab]
    return (((w >> np.uint64(9)).astype(np.float32) + np.float32(0.5))
            * np.float32(2.0 ** -23)).astype(np.float32)


def gumbel(seed: int, seq_id: int, pos: int, vocab: int) -> np.ndarray:
    """g_v = -ln(-ln u_v) in float32."""
    u = uniforms(seed, seq_id, pos, vocab)
    return (-np.log(-np.log(u))).astype(np.float32)


def scores(logits: np.ndarray, temperature: float, seed: int, seq_id: int, pos: int) -> np.ndarray:
    """The fp32 quantity whose argmax is the token: logits (T = 0) or logits/T + g."""
    l32 = np.asarray(logits).astype(np.float32)
    if temperature == 0.0:
        return l32
    inv_t = np.float32(1.0) / np.float32(temperature)
    return (l32 * inv_t + gumbel(seed, seq_id, pos, l32.shape[-1])).astype(np.float32)


def sample(logits: np.ndarray, temperature: float, seed: int, seq_id: int, pos: int) -> int:
    """Token at absolute position ``pos``; lowest index wins ties (np.argmax)."""
    return int(np.argmax(scores(logits, temperature, seed, seq_id, pos)))


def logprob(logits: np.ndarray, temperature: float, token: int) -> float:
    """log softmax(logits / T)[token] in fp64 (T = 1 when T = 0)."""
    t = 1.0 if temperature == 0.0 else float(temperature)
    s = np.asarray(logits, np.float64) / t
    m = float(np.max(s))
    return float(s[token] - (m + np.log(np.sum(np.exp(s - m)))))


def stop_at(tokens, eos: int):
    """The response up to and including the first ``eos`` (all of it if there is none)."""
    tokens = list(tokens)
    return tokens[:tokens.index(eos) + 1] if eos in tokens else tokens


def top2_gap(s: np.ndarray) -> float:
    """Difference between the largest and second largest score."""
    part = np.partition(np.asarray(s, np.float64), -2)
    return float(part[-1] - part[-2])


def sampler(temperature: float, seed: int, seq_id: int):
    """A ``sample_fn(logits, pos)`` closure for oracle.model.generate."""
    return lambda logits, pos: sample(logits, temperature, seed, seq_id, pos)
