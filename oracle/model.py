"""Qwen2.5 decoder forward in fp64 -- oracle, test infrastructure only.

The paper runs rollout with Qwen2.5 models (section 6, "Models") but writes no
model equations; this module is the standard Qwen2.5 decoder written out
directly from its definition:

  x_i = E[t_i]
  per layer:  h = RMSNorm(x) ; q,k,v = W h + b ; RoPE(q, k) at position i ;
              causal GQA softmax attention ; x += W_o a ;
              h2 = RMSNorm(x) ; x += W_down (silu(W_gate h2) * (W_up h2))
  logits = W_lm RMSNorm(x)   (W_lm = E when embeddings are tied)

Weights are given in [out, in] layout, so a projection is ``h @ W.T``.
RoPE pairs dimension d with d + hd/2 ("rotate half"), with frequencies
theta^(-2d/hd) and angles computed in fp64.  Query head h reads KV head
h // (n_q / n_kv).  No padding: positions are 0-based and contiguous.

Every function takes an optional ``rnd``: a rounding applied where a
reduced-precision implementation stores a GEMM or attention input (the
normalised activations, q after RoPE, the K/V cache, the softmax
probabilities, the attention output, silu(gate)*up).  ``rnd=None`` is the
plain fp64 definition; ``rnd=bf16_round`` is a diagnostic that separates
the error of bf16 storage from everything else.
"""
from __future__ import annotations

import numpy as np


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even), returned as fp64.

    fp64 -> fp32 first (a bf16 value is an fp32 with 16 zero low bits), then
    the low 16 bits are rounded to nearest even.
    """
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def _id(x):
    return x


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def rope_cos_sin(positions: np.ndarray, head_dim: int, theta: float):
    """cos/sin of angle pos * theta^(-2d/hd), d < hd/2, in fp64. Shapes [n, hd/2]."""
    d = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = theta ** (-2.0 * d / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(u: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate pairs (d, d + hd/2) of u [n, heads, hd] by the per-row angles."""
    half = u.shape[-1] // 2
    u1, u2 = u[..., :half], u[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([u1 * c - u2 * s, u2 * c + u1 * s], axis=-1)


def softmax(s: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: np.ndarray,
              k_pos: np.ndarray, rnd=None) -> np.ndarray:
    """Causal GQA attention.

    q [nq_tok, n_q, hd], k/v [nk_tok, n_kv, hd]; query at position q_pos[i]
    attends to keys with k_pos <= q_pos[i].  Returns [nq_tok, n_q, hd].
    With ``rnd`` the normalised probabilities are rounded before P @ V.
    """
    n_q, n_kv, hd = q.shape[1], k.shape[1], q.shape[2]
    group = n_q // n_kv
    out = np.empty_like(q)
    mask = k_pos[None, :] <= q_pos[:, None]                    # [nq_tok, nk_tok]
    for h in range(n_q):
        kh = h // group
        s = q[:, h, :] @ k[:, kh, :].T / np.sqrt(hd)           # [nq_tok, nk_tok]
        s = np.where(mask, s, -np.inf)
        if rnd is None:
            out[:, h, :] = softmax(s, axis=-1) @ v[:, kh, :]
        else:
            e = np.exp(s - np.max(s, axis=-1, keepdims=True))
            out[:, h, :] = (rnd(e) @ v[:, kh, :]) / np.sum(e, axis=-1, keepdims=True)
    return out


def _qkv(layer, h, shape):
    """q, k, v before RoPE (the bias is part of the projection)."""
    hd = shape.head_dim
    q = (h @ layer["wq"].T + layer["bq"]).reshape(-1, shape.n_q, hd)
    k = (h @ layer["wk"].T + layer["bk"]).reshape(-1, shape.n_kv, hd)
    v = (h @ layer["wv"].T + layer["bv"]).reshape(-1, shape.n_kv, hd)
    return q, k, v


def _mlp(layer, x, shape, r=_id):
    h2 = r(rmsnorm(x, layer["mlp_norm"], shape.eps))
    return r(silu(h2 @ layer["w_gate"].T) * (h2 @ layer["w_up"].T)) @ layer["w_down"].T


def lm_head(w, x, shape, rnd=None) -> np.ndarray:
    r = rnd or _id
    hf = r(rmsnorm(x, w["final_norm"], shape.eps))
    wl = w["embed"] if w["lm_head"] is None else w["lm_head"]
    return hf @ wl.T


def forward_full(w: dict, shape, tokens, rnd=None) -> np.ndarray:
    """Brute-force causal forward over a whole sequence: logits [n, V] for every position."""
    r = rnd or _id
    tokens = np.asarray(tokens)
    n = len(tokens)
    pos = np.arange(n)
    cos, sin = rope_cos_sin(pos, shape.head_dim, shape.theta)
    x = w["embed"][tokens].astype(np.float64)
    for layer in w["layers"]:
        h = r(rmsnorm(x, layer["attn_norm"], shape.eps))
        q, k, v = _qkv(layer, h, shape)
        q, k, v = r(apply_rope(q, cos, sin)), r(apply_rope(k, cos, sin)), r(v)
        a = r(attention(q, k, v, pos, pos, rnd).reshape(n, -1))
        x = x + a @ layer["wo"].T
        x = x + _mlp(layer, x, shape, r)
    return lm_head(w, x, shape, rnd)


class KVState:
    """Incremental decoding state of one sequence: post-RoPE K and V per layer."""

    def __init__(self, shape, rnd=None):
        self.shape = shape
        self.rnd = rnd
        self.k = [np.zeros((0, shape.n_kv, shape.head_dim)) for _ in range(shape.layers)]
        self.v = [np.zeros((0, shape.n_kv, shape.head_dim)) for _ in range(shape.layers)]
        self.length = 0

    def step(self, w: dict, tokens) -> np.ndarray:
        """Append tokens at positions length.. and return their logits [n, V]."""
        shape = self.shape
        r = self.rnd or _id
        tokens = np.asarray(tokens)
        n = len(tokens)
        pos = np.arange(self.length, self.length + n)
        cos, sin = rope_cos_sin(pos, shape.head_dim, shape.theta)
        x = w["embed"][tokens].astype(np.float64)
        for li, layer in enumerate(w["layers"]):
            h = r(rmsnorm(x, layer["attn_norm"], shape.eps))
            q, k, v = _qkv(layer, h, shape)
            q, k, v = r(apply_rope(q, cos, sin)), r(apply_rope(k, cos, sin)), r(v)
            self.k[li] = np.concatenate([self.k[li], k])
            self.v[li] = np.concatenate([self.v[li], v])
            kpos = np.arange(self.length + n)
            a = r(attention(q, self.k[li], self.v[li], pos, kpos, self.rnd).reshape(n, -1))
            x = x + a @ layer["wo"].T
            x = x + _mlp(layer, x, shape, r)
        self.length += n
        return lm_head(w, x, shape, self.rnd)


def generate(w: dict, shape, prompt, n_new: int, sample_fn, rnd=None) -> tuple:
    """Rollout of one sequence: prefill the prompt, then n_new - 1 decode steps.

    ``n_new`` counts every generated token, the one sampled from the prefill
    logits included; the KV of the last generated token is never needed.
    ``sample_fn(logits_row, pos)`` returns the token at absolute position pos.
    Returns (tokens [n_new], logits [n_new, V]) where logits[j] produced tokens[j].
    """
    st = KVState(shape, rnd)
    logits = st.step(w, prompt)[-1]
    p = len(prompt)
    toks, rows = [], []
    for j in range(n_new):
        t = int(sample_fn(logits, p + j))
        toks.append(t)
        rows.append(logits)
        if j + 1 < n_new:
            logits = st.step(w, [t])[-1]
    return np.array(toks, np.int32), np.array(rows)


def teacher_forced_logits(w: dict, shape, prompt, response, rnd=None) -> np.ndarray:
    """Logits that predict response[j] given prompt + response[:j], rows j = 0..L-1."""
    seq = np.concatenate([np.asarray(prompt), np.asarray(response)[:-1]])
    return forward_full(w, shape, seq, rnd)[len(prompt) - 1:]


def decode_step_batch(w: dict, states, tokens) -> np.ndarray:
    """One decode step for several sequences at once: logits [B, V].

    Sequence b appends tokens[b] at its own position states[b].length.  Every
    projection, norm and MLP acts on each row independently, so they run on
    the whole batch as [B, H] products; RoPE uses each row's position and the
    attention of row b reads only its own cache.  Row b equals
    ``states[b].step(w, [tokens[b]])[-1]`` (the definition, batched).
    """
    shape = states[0].shape
    rnd = states[0].rnd
    r = rnd or _id
    tokens = np.asarray(tokens)
    pos = np.array([st.length for st in states])
    cos, sin = rope_cos_sin(pos, shape.head_dim, shape.theta)
    x = w["embed"][tokens].astype(np.float64)
    for li, layer in enumerate(w["layers"]):
        h = r(rmsnorm(x, layer["attn_norm"], shape.eps))
        q, k, v = _qkv(layer, h, shape)
        q, k, v = r(apply_rope(q, cos, sin)), r(apply_rope(k, cos, sin)), r(v)
        a = np.empty_like(q)
        for b, st in enumerate(states):
            st.k[li] = np.concatenate([st.k[li], k[b:b + 1]])
            st.v[li] = np.concatenate([st.v[li], v[b:b + 1]])
            a[b] = attention(q[b:b + 1], st.k[li], st.v[li], pos[b:b + 1], np.arange(pos[b] + 1), rnd)[0]
        x = x + r(a.reshape(len(states), -1)) @ layer["wo"].T
        x = x + _mlp(layer, x, shape, r)
    for st in states:
        st.length += 1
    return lm_head(w, x, shape, rnd)
