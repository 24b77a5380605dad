"""Model shapes, random weights and rollout workloads (all seeded, synthetic).

The paper trains Qwen2.5 models (section 6, "Models") and characterises
rollout by its long-tailed response lengths (section 2.2: P75 between 755 and
1.1k tokens, maxima up to 16k).  Real checkpoints and datasets are not used;
the shapes below are the Qwen2.5 sizes and the length draws reproduce the
long-tail structure with lognormal distributions clamped to a range.

Weights: every tensor has its own torch generator seeded from
(weight seed, tensor index), values N(0, 0.02) rounded once to the storage
dtype (round-to-nearest-even for bf16).  Norm gains are 1.  The q/k/v biases
are drawn like the weights so that a dropped bias is visible.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    layers: int
    hidden: int
    n_q: int
    n_kv: int
    head_dim: int
    inter: int
    vocab: int
    tied: bool
    dtype: str  # "f32" or "bf16": storage and GEMM-input type
    eps: float = 1e-6
    theta: float = 1e6

    @property
    def group(self) -> int:
        return self.n_q // self.n_kv

    @property
    def qkv_out(self) -> int:
        return (self.n_q + 2 * self.n_kv) * self.head_dim

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def kv_bytes_per_token(self) -> int:
        return self.layers * 2 * self.n_kv * self.head_dim * self.elem_bytes

    def decode_weight_bytes(self) -> int:
        """Bytes of weights one decode step must read once (all layers + LM head)."""
        h, i, hd = self.hidden, self.inter, self.head_dim
        per_layer = (h * self.qkv_out + self.qkv_out + self.n_q * hd * h + 3 * h * i + 2 * h)
        return (self.layers * per_layer + self.vocab * h + h) * self.elem_bytes

    def params_nonembed(self) -> int:
        h, i, hd = self.hidden, self.inter, self.head_dim
        return self.layers * (h * self.qkv_out + self.n_q * hd * h + 3 * h * i)


SHAPES: Dict[str, ModelShape] = {
    "tiny": ModelShape("tiny", 2, 256, 4, 2, 64, 688, 2048, False, "f32"),
    "qwen2.5-0.5b": ModelShape("qwen2.5-0.5b", 24, 896, 14, 2, 64, 4864, 151936, True, "bf16"),
    "qwen2.5-7b": ModelShape("qwen2.5-7b", 28, 3584, 28, 4, 128, 18944, 152064, False, "bf16"),
    "qwen2.5-32b": ModelShape("qwen2.5-32b", 64, 5120, 40, 8, 128, 27648, 152064, False, "bf16"),
}


def truncated(shape: ModelShape, layers: int, vocab: Optional[int] = None) -> ModelShape:
    """Same per-layer shapes with fewer layers (and optionally a smaller vocabulary)."""
    return dataclasses.replace(shape, name=f"{shape.name}-L{layers}", layers=layers,
                               vocab=shape.vocab if vocab is None else vocab)


LAYER_TENSORS = ("wq", "bq", "wk", "bk", "wv", "bv", "wo", "w_gate", "w_up", "w_down")


def tensor_names(shape: ModelShape) -> List[str]:
    names = ["embed"]
    for l in range(shape.layers):
        names += [f"layers.{l}.{t}" for t in LAYER_TENSORS]
    names.append("lm_head")
    return names


def _tensor_shape(shape: ModelShape, t: str):
    h, i, hd = shape.hidden, shape.inter, shape.head_dim
    return {
        "wq": (shape.n_q * hd, h), "bq": (shape.n_q * hd,),
        "wk": (shape.n_kv * hd, h), "bk": (shape.n_kv * hd,),
        "wv": (shape.n_kv * hd, h), "bv": (shape.n_kv * hd,),
        "wo": (h, shape.n_q * hd),
        "w_gate": (i, h), "w_up": (i, h), "w_down": (h, i),
    }[t]


def _randn(dims, seed: int, index: int, device, dtype) -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1_000_003 + index)
    t = torch.randn(dims, generator=g, device=device, dtype=torch.float32)
    t.mul_(0.02)
    return t.to(dtype)


def make_weights(shape: ModelShape, seed: int = 0, device="cpu") -> dict:
    """Random Qwen2.5-layout weights ([out, in] row-major) on `device`.

    Returns {"embed", "final_norm", "lm_head" (None when tied), "layers": [dict]}.
    Values differ between a CPU and a GPU generator for the same seed; a test
    that needs identical weights on both sides copies one to the other.
    """
    dtype = torch.float32 if shape.dtype == "f32" else torch.bfloat16
    h = shape.hidden
    w = {"embed": _randn((shape.vocab, h), seed, 0, device, dtype),
         "final_norm": torch.ones(h, device=device, dtype=dtype), "layers": []}
    idx = 1
    for _ in range(shape.layers):
        layer = {"attn_norm": torch.ones(h, device=device, dtype=dtype),
                 "mlp_norm": torch.ones(h, device=device, dtype=dtype)}
        for t in LAYER_TENSORS:
            layer[t] = _randn(_tensor_shape(shape, t), seed, idx, device, dtype)
            idx += 1
        w["layers"].append(layer)
    w["lm_head"] = None if shape.tied else _randn((shape.vocab, h), seed, idx, device, dtype)
    return w


def weights_to_numpy(w: dict, dtype=np.float64) -> dict:
    """Host copy of a weight dict, upcast (exactly) to `dtype`."""
    def cv(t):
        return None if t is None else t.detach().to("cpu", torch.float32).numpy().astype(dtype)
    return {"embed": cv(w["embed"]), "final_norm": cv(w["final_norm"]),
            "lm_head": cv(w["lm_head"]),
            "layers": [{k: cv(v) for k, v in layer.items()} for layer in w["layers"]]}


@dataclasses.dataclass
class Workload:
    """A batch of rollout sequences: prompt ids (CSR), forced response lengths."""
    name: str
    shape: ModelShape
    seq_ids: np.ndarray         # int64 [n], unique
    prompt_tokens: np.ndarray   # int32 [sum p]
    prompt_offsets: np.ndarray  # int64 [n+1]
    max_new: np.ndarray         # int32 [n], counts every generated token
    prompt_group: np.ndarray    # int32 [n], sequences of one GRPO prompt share ids
    temperature: float
    sample_seed: int
    round_id: Optional[np.ndarray] = None  # int32 [n] when the rounds are given

    @property
    def n(self) -> int:
        return len(self.seq_ids)

    def prompt(self, i: int) -> np.ndarray:
        return self.prompt_tokens[self.prompt_offsets[i]:self.prompt_offsets[i + 1]]

    def prompt_lens(self) -> np.ndarray:
        return np.diff(self.prompt_offsets).astype(np.int64)

    def subset(self, idx) -> "Workload":
        idx = np.asarray(idx)
        prompts = [self.prompt(int(i)) for i in idx]
        offs = np.zeros(len(idx) + 1, np.int64)
        offs[1:] = np.cumsum([len(p) for p in prompts])
        return dataclasses.replace(
            self, seq_ids=self.seq_ids[idx].copy(),
            prompt_tokens=np.concatenate(prompts).astype(np.int32) if prompts else np.zeros(0, np.int32),
            prompt_offsets=offs, max_new=self.max_new[idx].copy(),
            prompt_group=self.prompt_group[idx].copy(),
            round_id=None if self.round_id is None else self.round_id[idx].copy())


def _lognormal_lengths(rng, n, median, sigma, lo, hi) -> np.ndarray:
    z = rng.standard_normal(n)
    return np.clip(np.rint(median * np.exp(sigma * z)), lo, hi).astype(np.int32)


def _build(name, shape, rng, n_prompts, per_prompt, p_lo, p_hi, len_spec, temperature,
           sample_seed, id_base=0, fixed_len=None) -> Workload:
    plen = rng.integers(p_lo, p_hi + 1, size=n_prompts)
    prompts = [rng.integers(0, shape.vocab, size=int(p)).astype(np.int32) for p in plen]
    n = n_prompts * per_prompt
    if fixed_len is not None:
        max_new = np.full(n, fixed_len, np.int32)
    else:
        max_new = _lognormal_lengths(rng, n, *len_spec)
    group = np.repeat(np.arange(n_prompts, dtype=np.int32), per_prompt)
    seq_prompts = [prompts[g] for g in group]
    offs = np.zeros(n + 1, np.int64)
    offs[1:] = np.cumsum([len(p) for p in seq_prompts])
    return Workload(name, shape, np.arange(id_base, id_base + n, dtype=np.int64),
                    np.concatenate(seq_prompts).astype(np.int32), offs, max_new, group,
                    temperature, sample_seed)


def make_workload(name: str, shape: Optional[ModelShape] = None) -> Workload:
    """Seeded workloads at the shapes of the paper's models.

    tiny      8 prompts x 32 ids, exactly 64 new tokens each, greedy
    0.5b      32 prompts x 8 responses, prompts U[64,512], LogN(512, 0.8) in [32,4096]
    7b-short  512 sequences, prompts U[128,1024], LogN(768, 0.4) in [64,2048]
    7b-long   64 sequences, prompts U[128,1024], LogN(4096, 1.0) in [512,16384]
    7b-mixed  the 512 + 64 sequences above in one batch (round ids 0 / 1 given)
    32b       96 sequences, prompts U[256,1024], LogN(2048, 0.9) in [64,8192]
    """
    if name == "tiny":
        s = shape or SHAPES["tiny"]
        rng = np.random.Generator(np.random.Philox(101))
        return _build(name, s, rng, 8, 1, 32, 32, None, 0.0, 0, fixed_len=64)
    if name == "0.5b":
        s = shape or SHAPES["qwen2.5-0.5b"]
        rng = np.random.Generator(np.random.Philox(102))
        return _build(name, s, rng, 32, 8, 64, 512, (512, 0.8, 32, 4096), 1.0, 202)
    if name == "7b-short":
        s = shape or SHAPES["qwen2.5-7b"]
        rng = np.random.Generator(np.random.Philox(103))
        return _build(name, s, rng, 512, 1, 128, 1024, (768, 0.4, 64, 2048), 1.0, 203)
    if name == "7b-long":
        s = shape or SHAPES["qwen2.5-7b"]
        rng = np.random.Generator(np.random.Philox(104))
        return _build(name, s, rng, 64, 1, 128, 1024, (4096, 1.0, 512, 16384), 1.0, 203,
                      id_base=512)
    if name == "7b-mixed":
        a, b = make_workload("7b-short", shape), make_workload("7b-long", shape)
        offs = np.concatenate([a.prompt_offsets, a.prompt_offsets[-1] + b.prompt_offsets[1:]])
        return Workload("7b-mixed", a.shape, np.concatenate([a.seq_ids, b.seq_ids]),
                        np.concatenate([a.prompt_tokens, b.prompt_tokens]), offs,
                        np.concatenate([a.max_new, b.max_new]),
                        np.concatenate([a.prompt_group, b.prompt_group + a.n]),
                        1.0, 203,
                        round_id=np.concatenate([np.zeros(a.n, np.int32), np.ones(b.n, np.int32)]))
    if name == "32b":
        s = shape or SHAPES["qwen2.5-32b"]
        rng = np.random.Generator(np.random.Philox(105))
        return _build(name, s, rng, 96, 1, 256, 1024, (2048, 0.9, 64, 8192), 1.0, 205)
    raise KeyError(name)


WORKLOADS = ("tiny", "0.5b", "7b-short", "7b-long", "7b-mixed", "32b")


@dataclasses.dataclass
class RLBatch:
    """Prompts of consecutive RL steps, each with r_spec candidate responses.

    Response r of prompt p is sequence ``seq_ids[p, r]`` with forced length
    ``max_new[p, r]``.  Prompt ids are stored once per prompt (CSR)."""
    name: str
    shape: ModelShape
    seq_ids: np.ndarray         # int64 [n_prompts, r_spec], unique
    prompt_tokens: np.ndarray   # int32 [sum p]
    prompt_offsets: np.ndarray  # int64 [n_prompts + 1]
    max_new: np.ndarray         # int32 [n_prompts, r_spec]
    temperature: float
    sample_seed: int

    @property
    def n_prompts(self) -> int:
        return self.seq_ids.shape[0]

    @property
    def r_spec(self) -> int:
        return self.seq_ids.shape[1]

    def sequences(self, prompts, responses: int) -> Workload:
        """The first `responses` responses of the given prompts, one sequence each (prompt-major)."""
        prompts = [int(p) for p in prompts]
        idx = [(p, r) for p in prompts for r in range(responses)]
        seq_prompts = [self.prompt_tokens[self.prompt_offsets[p]:self.prompt_offsets[p + 1]] for p, _ in idx]
        offs = np.zeros(len(idx) + 1, np.int64)
        offs[1:] = np.cumsum([len(t) for t in seq_prompts])
        return Workload(self.name, self.shape, np.array([self.seq_ids[p, r] for p, r in idx], np.int64),
                        np.concatenate(seq_prompts).astype(np.int32), offs,
                        np.array([self.max_new[p, r] for p, r in idx], np.int32),
                        np.array([p for p, _ in idx], np.int32), self.temperature, self.sample_seed)


def make_rl_batch(shape: ModelShape, n_prompts: int, r_spec: int, *, p_lo: int, p_hi: int, median: float,
                  sigma_p: float, sigma_r: float, lo: int, hi: int, seed: int, sample_seed: int = 0,
                  temperature: float = 1.0, name: str = "rl") -> RLBatch:
    """Prompt-correlated long-tail lengths: log L = log median + sigma_p z_p + sigma_r z_pr, clamped to [lo, hi].

    z_p is one standard normal draw per prompt (its difficulty: hard prompts give
    long responses across the board, as the paper observes in section 6.3) and
    z_pr one per response.  Prompt lengths are U[p_lo, p_hi], ids U[0, vocab).
    Response r's draws come from a stream of their own, so the first r
    responses of every prompt are the same whatever r_spec is."""
    rng = np.random.Generator(np.random.Philox(seed))
    plen = rng.integers(p_lo, p_hi + 1, size=n_prompts)
    prompts = [rng.integers(0, shape.vocab, size=int(p)).astype(np.int32) for p in plen]
    z_p = rng.standard_normal(n_prompts)[:, None]
    z_pr = np.stack([np.random.Generator(np.random.Philox(key=np.array([seed, 1 + r], np.uint64)))
                     .standard_normal(n_prompts) for r in range(r_spec)], axis=1).reshape(n_prompts, r_spec)
    lens = np.clip(np.rint(median * np.exp(sigma_p * z_p + sigma_r * z_pr)), lo, hi).astype(np.int32)
    offs = np.zeros(n_prompts + 1, np.int64)
    offs[1:] = np.cumsum(plen)
    ids = np.arange(n_prompts * r_spec, dtype=np.int64).reshape(n_prompts, r_spec)
    return RLBatch(name, shape, ids, np.concatenate(prompts).astype(np.int32) if prompts else np.zeros(0, np.int32),
                   offs, lens, temperature, sample_seed)
