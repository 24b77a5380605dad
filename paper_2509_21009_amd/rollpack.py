"""Python binding of librollpack.so (include/rollpack.h).

Argument marshalling only: every step of rollout runs inside the HIP library.
PyTorch provides the device memory (weights, KV pool, scratch workspace) and
the stream.  Importing this module does not load the library; the first call
does, and raises if it was not built -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librollpack.so")

RP_DTYPE_F32, RP_DTYPE_BF16 = 0, 1
STATUS = {0: "RP_OK", 1: "RP_ERR_INVALID_ARG", 2: "RP_ERR_OUT_OF_PAGES", 3: "RP_ERR_DUPLICATE_ID",
          4: "RP_ERR_UNKNOWN_ID", 5: "RP_ERR_BAD_STATE", 6: "RP_ERR_HIP", 7: "RP_ERR_CAPACITY"}


class RpModelConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("intermediate", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float),
                ("tied_embeddings", ctypes.c_int32), ("dtype", ctypes.c_int32)]


_LAYER_FIELDS = ("attn_norm", "wq", "bq", "wk", "bk", "wv", "bv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")


class RpLayerWeights(ctypes.Structure):
    _fields_ = [(f, ctypes.c_void_p) for f in _LAYER_FIELDS]


class RpWeights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
                ("layers", ctypes.POINTER(RpLayerWeights))]


class RpEngineLimits(ctypes.Structure):
    _fields_ = [("max_seqs", ctypes.c_int32), ("max_prefill_tokens", ctypes.c_int32),
                ("max_context", ctypes.c_int32), ("page_tokens", ctypes.c_int32), ("kv_pages", ctypes.c_int64)]


class RpRoundStats(ctypes.Structure):
    _fields_ = [("round_id", ctypes.c_int32), ("n_seqs", ctypes.c_int32), ("decode_steps", ctypes.c_int32),
                ("kind", ctypes.c_int32), ("prompt_tokens", ctypes.c_int64),
                ("generated_tokens", ctypes.c_int64), ("peak_pages", ctypes.c_int64),
                ("makespan_ms", ctypes.c_double), ("prefill_ms", ctypes.c_double),
                ("decode_ms", ctypes.c_double), ("slot_idle", ctypes.c_double), ("idle_slot_s", ctypes.c_double),
                ("preemptions", ctypes.c_int64), ("recomputed_tokens", ctypes.c_int64)]

    def as_dict(self) -> dict:
        return {f: getattr(self, f) for f, _ in self._fields_}


KERNEL_CLASSES = ("embed_norm", "add_norm", "gemm_qkv", "rope_append", "attn", "attn_merge", "gemm_o",
                  "gemm_gate_up", "gemm_down", "gemm_lm_head", "sample")


class RpTailParams(ctypes.Structure):
    _fields_ = [("P0", ctypes.c_int32), ("R0", ctypes.c_int32), ("r_spec", ctypes.c_int32),
                ("eta_p", ctypes.c_float), ("eta_r", ctypes.c_float)]


SCHEDULE_NONE, SCHEDULE_ROUNDS, SCHEDULE_TAIL_BATCHING = 0, 1, 2


class RpKernelStats(ctypes.Structure):
    _fields_ = [("kernel_class", ctypes.c_int32), ("phase", ctypes.c_int32), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("bytes", ctypes.c_double), ("flops", ctypes.c_double)]

    def as_dict(self) -> dict:
        return {"kernel": KERNEL_CLASSES[self.kernel_class], "phase": ("prefill", "decode")[self.phase],
                "launches": self.launches, "total_ms": self.total_ms, "bytes": self.bytes, "flops": self.flops}


class RpStepRecord(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("round_id", ctypes.c_int32), ("rows", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("sum_ctx", ctypes.c_int64), ("ms", ctypes.c_double),
                ("end_ms", ctypes.c_double)]


class RollpackError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


_P = ctypes.c_void_p
_I32P = ctypes.POINTER(ctypes.c_int32)
_I64P = ctypes.POINTER(ctypes.c_int64)
_F32P = ctypes.POINTER(ctypes.c_float)
_SZP = ctypes.POINTER(ctypes.c_size_t)

# name -> (restype, argtypes), in the order of include/rollpack.h
SIGNATURES = {
    "rp_workspace_size": (ctypes.c_int, [ctypes.POINTER(RpModelConfig), ctypes.POINTER(RpEngineLimits), _SZP, _SZP]),
    "rp_kv_bytes_per_token": (ctypes.c_int, [ctypes.POINTER(RpModelConfig), _SZP]),
    "rp_engine_create": (ctypes.c_int, [ctypes.POINTER(RpModelConfig), ctypes.POINTER(RpWeights),
                                        ctypes.POINTER(RpEngineLimits), _P, ctypes.c_size_t, _P, ctypes.c_size_t,
                                        _P, ctypes.POINTER(_P)]),
    "rp_engine_destroy": (None, [_P]),
    "rp_packed_weights_bytes": (ctypes.c_int, [ctypes.POINTER(RpModelConfig), _SZP]),
    "rp_engine_set_packed_weights": (ctypes.c_int, [_P, _P, ctypes.c_size_t]),
    "rp_prefill": (ctypes.c_int, [_P, ctypes.c_int32, _I64P, _I32P, _I64P, _I32P, ctypes.c_uint64, ctypes.c_float,
                                  _P, _I32P]),
    "rp_decode_step": (ctypes.c_int, [_P, _I32P, _P, _I64P, _I32P]),
    "rp_free_finished": (ctypes.c_int, [_P, _I64P, ctypes.c_int32, _I32P]),
    "rp_abort": (ctypes.c_int, [_P, ctypes.c_int32, _I64P]),
    "rp_get_tokens": (ctypes.c_int, [_P, ctypes.c_int64, _I32P, ctypes.c_int32, _I32P]),
    "rp_get_logprobs": (ctypes.c_int, [_P, ctypes.c_int64, _F32P, ctypes.c_int32, _I32P]),
    "rp_set_eos": (ctypes.c_int, [_P, ctypes.c_int32]),
    "rp_rollout_generate": (ctypes.c_int, [_P, ctypes.c_int32, _I64P, _I32P, _I64P, _I32P, ctypes.c_uint64,
                                           ctypes.c_float, _I32P, _I32P, _F32P, _I32P, ctypes.POINTER(RpRoundStats),
                                           ctypes.c_int32, _I32P]),
    "rp_generate": (ctypes.c_int, [ctypes.POINTER(RpModelConfig), ctypes.POINTER(RpWeights),
                                   ctypes.POINTER(RpEngineLimits), _P, ctypes.c_size_t, _P, ctypes.c_size_t, _P,
                                   ctypes.c_int32, _I64P, _I32P, _I64P, _I32P, ctypes.c_uint64, ctypes.c_float,
                                   ctypes.c_int32, _I32P, ctypes.POINTER(RpTailParams), _I32P, _F32P, _I32P, _I32P,
                                   ctypes.POINTER(RpRoundStats), ctypes.c_int32, _I32P]),
    "rp_generate_static": (ctypes.c_int, [ctypes.POINTER(RpModelConfig), ctypes.POINTER(RpWeights),
                                          ctypes.POINTER(RpEngineLimits), _P, ctypes.c_int32, _I64P, _I32P, _I64P,
                                          _I32P, ctypes.c_uint64, ctypes.c_float, ctypes.c_int32, _I32P,
                                          ctypes.POINTER(RpTailParams), _I32P, _F32P, _I32P, _I32P,
                                          ctypes.POINTER(RpRoundStats), ctypes.c_int32, _I32P]),
    "rp_rollout_tail_batched": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32, _I64P, _I32P, _I64P, _I32P,
                                               ctypes.c_uint64, ctypes.c_float, ctypes.c_int32, ctypes.c_int32,
                                               ctypes.c_float, ctypes.c_float, _I32P, _F32P, _I32P, _I32P, _I32P,
                                               ctypes.POINTER(RpRoundStats), ctypes.c_int32, _I32P]),
    "rp_plan_tail_batching": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, _I32P, ctypes.c_int32, ctypes.c_int32,
                                             ctypes.c_float, ctypes.c_float, ctypes.c_int32, ctypes.c_int32, _I32P, _I32P, _I32P,
                                             _I32P, _I32P, _I32P, _I32P, _I32P]),
    "rp_set_kv_policy": (ctypes.c_int, [_P, ctypes.c_int32]),
    "rp_kv_status": (ctypes.c_int, [_P, _I64P, _I32P, _I32P, _I64P, _I64P]),
    "rp_step_trace_enable": (ctypes.c_int, [_P, ctypes.c_int32]),
    "rp_step_trace_read": (ctypes.c_int, [_P, ctypes.POINTER(RpStepRecord), ctypes.c_int32, _I32P]),
    "rp_profile_enable": (ctypes.c_int, [_P, ctypes.c_uint32]),
    "rp_profile_every": (ctypes.c_int, [_P, ctypes.c_int32]),
    "rp_profile_read": (ctypes.c_int, [_P, ctypes.POINTER(RpKernelStats), ctypes.c_int32, _I32P]),
    "rp_stream_read_gbs": (ctypes.c_int, [_P, ctypes.c_size_t, ctypes.c_int32, _P, ctypes.POINTER(ctypes.c_double)]),
    "rp_last_error": (ctypes.c_char_p, []),
}

_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load librollpack.so once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                               "(there is no fallback implementation)")
        lib = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(status: int):
    if status != 0:
        raise RollpackError(status, load_library().rp_last_error().decode())


def _arr(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ctypes.POINTER(np.ctypeslib.as_ctypes_type(dtype)))


def _opt(a, dtype):
    if a is None:
        return None, None
    return _arr(a, dtype)


# ---- thin wrappers with the C names -------------------------------------------------

def rp_workspace_size(cfg: RpModelConfig, limits: RpEngineLimits):
    kv, sc = ctypes.c_size_t(), ctypes.c_size_t()
    _check(load_library().rp_workspace_size(ctypes.byref(cfg), ctypes.byref(limits), ctypes.byref(kv), ctypes.byref(sc)))
    return kv.value, sc.value


def rp_kv_bytes_per_token(cfg: RpModelConfig) -> int:
    b = ctypes.c_size_t()
    _check(load_library().rp_kv_bytes_per_token(ctypes.byref(cfg), ctypes.byref(b)))
    return b.value


def rp_engine_create(cfg, weights: RpWeights, limits, kv_ptr: int, kv_bytes: int, scratch_ptr: int,
                     scratch_bytes: int, stream_ptr: int) -> int:
    out = _P()
    _check(load_library().rp_engine_create(ctypes.byref(cfg), ctypes.byref(weights), ctypes.byref(limits), kv_ptr,
                                           kv_bytes, scratch_ptr, scratch_bytes, stream_ptr, ctypes.byref(out)))
    return out.value


def rp_engine_destroy(eng: int) -> None:
    load_library().rp_engine_destroy(eng)


def rp_packed_weights_bytes(cfg: RpModelConfig) -> int:
    b = ctypes.c_size_t()
    _check(load_library().rp_packed_weights_bytes(ctypes.byref(cfg), ctypes.byref(b)))
    return b.value


def rp_engine_set_packed_weights(eng: int, ptr: Optional[int], nbytes: int) -> None:
    _check(load_library().rp_engine_set_packed_weights(eng, ptr, nbytes))


def rp_prefill(eng: int, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed: int, temperature: float,
               logits_out_ptr: Optional[int] = None, want_first_tokens: bool = False):
    ids, ids_p = _arr(seq_ids, np.int64)
    toks, toks_p = _arr(prompt_tokens, np.int32)
    offs, offs_p = _arr(prompt_offsets, np.int64)
    mn, mn_p = _arr(max_new_tokens, np.int32)
    first = np.zeros(len(ids), np.int32) if want_first_tokens else None
    first_p = first.ctypes.data_as(_I32P) if first is not None else None
    _check(load_library().rp_prefill(eng, len(ids), ids_p, toks_p, offs_p, mn_p, ctypes.c_uint64(seed),
                                     ctypes.c_float(temperature), logits_out_ptr, first_p))
    return first


def rp_decode_step(eng: int, forced_tokens=None, logits_out_ptr: Optional[int] = None, max_rows: int = 0):
    f, f_p = _opt(forced_tokens, np.int32)
    rows = np.zeros(max(max_rows, 1), np.int64)
    n = ctypes.c_int32()
    _check(load_library().rp_decode_step(eng, f_p, logits_out_ptr, rows.ctypes.data_as(_I64P) if max_rows else None,
                                         ctypes.byref(n)))
    return n.value, rows[:n.value] if max_rows else None


def rp_free_finished(eng: int, cap: int = 4096) -> np.ndarray:
    out = np.zeros(max(cap, 1), np.int64)
    n = ctypes.c_int32()
    _check(load_library().rp_free_finished(eng, out.ctypes.data_as(_I64P), cap, ctypes.byref(n)))
    return out[:n.value]


def rp_abort(eng: int, seq_ids) -> None:
    ids, ids_p = _arr(seq_ids, np.int64)
    _check(load_library().rp_abort(eng, len(ids), ids_p))


def rp_get_tokens(eng: int, seq_id: int, cap: int) -> np.ndarray:
    out = np.zeros(max(cap, 1), np.int32)
    n = ctypes.c_int32()
    _check(load_library().rp_get_tokens(eng, seq_id, out.ctypes.data_as(_I32P), cap, ctypes.byref(n)))
    return out[:min(n.value, cap)]


def rp_rollout_generate(eng: int, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed: int,
                        temperature: float, round_ids=None, max_stats: int = 16, details: bool = False):
    """Returns (tokens, stats); with details=True (tokens, logprobs, lengths, stats)."""
    ids, ids_p = _arr(seq_ids, np.int64)
    toks, toks_p = _arr(prompt_tokens, np.int32)
    offs, offs_p = _arr(prompt_offsets, np.int64)
    mn, mn_p = _arr(max_new_tokens, np.int32)
    rid, rid_p = _opt(round_ids, np.int32)
    resp = np.zeros(int(mn.sum()), np.int32)
    logp = np.zeros(int(mn.sum()), np.float32) if details else None
    lens = np.zeros(len(ids), np.int32) if details else None
    stats = (RpRoundStats * max_stats)()
    nr = ctypes.c_int32()
    _check(load_library().rp_rollout_generate(eng, len(ids), ids_p, toks_p, offs_p, mn_p, ctypes.c_uint64(seed),
                                              ctypes.c_float(temperature), rid_p, resp.ctypes.data_as(_I32P),
                                              None if logp is None else logp.ctypes.data_as(_F32P),
                                              None if lens is None else lens.ctypes.data_as(_I32P), stats,
                                              max_stats, ctypes.byref(nr)))
    st = [stats[i].as_dict() for i in range(min(nr.value, max_stats))]
    return (resp, logp, lens, st) if details else (resp, st)


def _generate_args(seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, schedule_mode, round_ids, tail):
    ids, ids_p = _arr(seq_ids, np.int64)
    toks, toks_p = _arr(prompt_tokens, np.int32)
    offs, offs_p = _arr(prompt_offsets, np.int64)
    mn, mn_p = _arr(max_new_tokens, np.int32)
    rid, rid_p = _opt(round_ids, np.int32)
    tp = None if tail is None else ctypes.byref(tail)
    keep = (ids, toks, offs, mn, rid)
    return keep, [len(ids), ids_p, toks_p, offs_p, mn_p], rid_p, tp


def _generate_outputs(n, total, max_stats):
    resp = np.zeros(max(total, 1), np.int32)
    logp = np.zeros(max(total, 1), np.float32)
    lens = np.zeros(n, np.int32)
    kept = np.zeros(n, np.int32)
    stats = (RpRoundStats * max(max_stats, 1))()
    return resp, logp, lens, kept, stats


def rp_generate(cfg: RpModelConfig, weights: RpWeights, limits: RpEngineLimits, kv_ptr: int, kv_bytes: int,
                scratch_ptr: int, scratch_bytes: int, stream_ptr: int, seq_ids, prompt_tokens, prompt_offsets,
                max_new_tokens, seed: int, temperature: float, schedule_mode: int = SCHEDULE_NONE, round_ids=None,
                tail: Optional[RpTailParams] = None, max_stats: int = 64):
    """One-shot rollout.  Returns (tokens, logprobs, lengths, kept (bool), round stats)."""
    keep, head, rid_p, tp = _generate_args(seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, schedule_mode,
                                           round_ids, tail)
    n, total = head[0], int(keep[3].sum())
    resp, logp, lens, kept, stats = _generate_outputs(n, total, max_stats)
    nr = ctypes.c_int32()
    _check(load_library().rp_generate(ctypes.byref(cfg), ctypes.byref(weights), ctypes.byref(limits), kv_ptr, kv_bytes,
                                      scratch_ptr, scratch_bytes, stream_ptr, *head, ctypes.c_uint64(seed),
                                      ctypes.c_float(temperature), schedule_mode, rid_p, tp,
                                      resp.ctypes.data_as(_I32P), logp.ctypes.data_as(_F32P),
                                      lens.ctypes.data_as(_I32P), kept.ctypes.data_as(_I32P), stats, max_stats,
                                      ctypes.byref(nr)))
    return resp[:total], logp[:total], lens, kept.astype(bool), [stats[i].as_dict() for i in range(min(nr.value, max_stats))]


def rp_generate_static(cfg: RpModelConfig, weights: RpWeights, limits: RpEngineLimits, stream_ptr: int, seq_ids,
                       prompt_tokens, prompt_offsets, max_new_tokens, seed: int, temperature: float,
                       schedule_mode: int = SCHEDULE_NONE, round_ids=None, tail: Optional[RpTailParams] = None,
                       max_stats: int = 64):
    """rp_generate over the library's static workspace.  Returns what rp_generate returns."""
    keep, head, rid_p, tp = _generate_args(seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, schedule_mode,
                                           round_ids, tail)
    n, total = head[0], int(keep[3].sum())
    resp, logp, lens, kept, stats = _generate_outputs(n, total, max_stats)
    nr = ctypes.c_int32()
    _check(load_library().rp_generate_static(ctypes.byref(cfg), ctypes.byref(weights), ctypes.byref(limits),
                                             stream_ptr, *head, ctypes.c_uint64(seed), ctypes.c_float(temperature),
                                             schedule_mode, rid_p, tp, resp.ctypes.data_as(_I32P),
                                             logp.ctypes.data_as(_F32P), lens.ctypes.data_as(_I32P),
                                             kept.ctypes.data_as(_I32P), stats, max_stats, ctypes.byref(nr)))
    return resp[:total], logp[:total], lens, kept.astype(bool), [stats[i].as_dict() for i in range(min(nr.value, max_stats))]


def rp_get_logprobs(eng: int, seq_id: int, cap: int) -> np.ndarray:
    out = np.zeros(max(cap, 1), np.float32)
    n = ctypes.c_int32()
    _check(load_library().rp_get_logprobs(eng, seq_id, out.ctypes.data_as(_F32P), cap, ctypes.byref(n)))
    return out[:min(n.value, cap)]


def rp_set_eos(eng: int, eos_token: int) -> None:
    _check(load_library().rp_set_eos(eng, eos_token))


def rp_rollout_tail_batched(eng: int, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed: int,
                            temperature: float, P0: int, R0: int, eta: float, eta_r: Optional[float] = None,
                            max_stats: int = 0, logprobs: bool = False):
    """seq_ids, max_new_tokens: [n_prompts, r_spec]; prompt CSR over prompts.  eta is the prompt
    speculation factor and, unless eta_r is given, the response factor too.

    Returns (resp_tokens, resp_len [n, r_spec], accept_round [n], kept [n, r_spec] bool, round stats),
    and the log-probabilities last when logprobs=True."""
    ids = np.ascontiguousarray(seq_ids, np.int64)
    n, r_spec = ids.shape
    toks, toks_p = _arr(prompt_tokens, np.int32)
    offs, offs_p = _arr(prompt_offsets, np.int64)
    mn = np.ascontiguousarray(max_new_tokens, np.int32)
    assert mn.shape == ids.shape and len(offs) == n + 1
    max_stats = max_stats or 2 * n + 2
    resp = np.zeros(max(int(mn.sum()), 1), np.int32)
    logp = np.zeros(max(int(mn.sum()), 1), np.float32) if logprobs else None
    glen = np.zeros((n, r_spec), np.int32)
    acc = np.zeros(n, np.int32)
    kept = np.zeros((n, r_spec), np.int32)
    stats = (RpRoundStats * max_stats)()
    nr = ctypes.c_int32()
    P = lambda a: a.ctypes.data_as(_I32P)  # noqa: E731
    _check(load_library().rp_rollout_tail_batched(eng, n, r_spec, ids.ctypes.data_as(_I64P), toks_p, offs_p, P(mn),
                                                  ctypes.c_uint64(seed), ctypes.c_float(temperature), P0, R0,
                                                  ctypes.c_float(eta), ctypes.c_float(eta if eta_r is None else eta_r),
                                                  P(resp), None if logp is None else logp.ctypes.data_as(_F32P),
                                                  P(glen), P(acc), P(kept), stats, max_stats, ctypes.byref(nr)))
    out = (resp, glen, acc, kept.astype(bool), [stats[i].as_dict() for i in range(min(nr.value, max_stats))])
    return out + (logp,) if logprobs else out


def rp_plan_tail_batching(lens, P0: int, R0: int, eta: float, eta_r: Optional[float] = None):
    """lens: int array [n_prompts, r_spec].  Returns a list of round dicts and per-prompt arrays.
    eta is the prompt speculation factor and, unless eta_r is given, the response factor too."""
    lens = np.ascontiguousarray(lens, np.int32)
    n, r_spec = lens.shape
    max_rounds = 2 * n + 2
    cap = n * (n + 2) + 8
    kind = np.zeros(max_rounds, np.int32)
    rtime = np.zeros(max_rounds, np.int32)
    loff = np.zeros(max_rounds + 1, np.int32)
    lp = np.zeros(max(cap, 1), np.int32)
    run = np.zeros(max(cap, 1) * r_spec, np.int32)
    acc = np.zeros(max(n, 1), np.int32)
    kept = np.zeros(max(n * r_spec, 1), np.int32)
    nr = ctypes.c_int32()
    P = lambda a: a.ctypes.data_as(_I32P)  # noqa: E731
    _check(load_library().rp_plan_tail_batching(n, r_spec, P(lens), P0, R0, ctypes.c_float(eta),
                                                ctypes.c_float(eta if eta_r is None else eta_r), max_rounds, cap,
                                                P(kind), P(rtime), P(loff), P(lp), P(run), P(acc), P(kept),
                                                ctypes.byref(nr)))
    rounds = []
    for k in range(nr.value):
        launched = lp[loff[k]:loff[k + 1]].tolist()
        steps = run[loff[k] * r_spec:loff[k + 1] * r_spec].reshape(-1, r_spec)
        rounds.append({"kind": "long" if kind[k] else "short", "time": int(rtime[k]), "launched": launched,
                       "run": {(p, r): int(steps[i, r]) for i, p in enumerate(launched) for r in range(r_spec)}})
    return rounds, acc[:n].copy(), kept[:n * r_spec].reshape(n, r_spec).astype(bool)


KV_RESERVE, KV_ON_DEMAND = 0, 1


def rp_set_kv_policy(eng: int, policy: int) -> None:
    _check(load_library().rp_set_kv_policy(eng, policy))


def rp_kv_status(eng: int) -> dict:
    f, p, rt = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    r, w = ctypes.c_int32(), ctypes.c_int32()
    _check(load_library().rp_kv_status(eng, ctypes.byref(f), ctypes.byref(r), ctypes.byref(w), ctypes.byref(p),
                                       ctypes.byref(rt)))
    return {"free_pages": f.value, "running": r.value, "waiting": w.value, "preemptions": p.value,
            "recomputed_tokens": rt.value}


def rp_step_trace_enable(eng: int, cap: int) -> None:
    _check(load_library().rp_step_trace_enable(eng, cap))


def rp_step_trace_read(eng: int, cap: int) -> np.ndarray:
    """Structured array of the recorded steps: kind, round_id, rows, sum_ctx, ms, end_ms."""
    out = (RpStepRecord * max(cap, 1))()
    n = ctypes.c_int32()
    _check(load_library().rp_step_trace_read(eng, out, cap, ctypes.byref(n)))
    rec = np.zeros(n.value, dtype=[("kind", np.int32), ("round_id", np.int32), ("rows", np.int32),
                                   ("sum_ctx", np.int64), ("ms", np.float64), ("end_ms", np.float64)])
    for i in range(n.value):
        r = out[i]
        rec[i] = (r.kind, r.round_id, r.rows, r.sum_ctx, r.ms, r.end_ms)
    return rec


def rp_profile_enable(eng: int, classes) -> None:
    """classes: iterable of names from KERNEL_CLASSES (empty stops profiling)."""
    mask = 0
    for c in classes:
        mask |= 1 << KERNEL_CLASSES.index(c)
    _check(load_library().rp_profile_enable(eng, mask))


def rp_profile_every(eng: int, every: int) -> None:
    """Time one launch in `every` of each selected class (1: all)."""
    _check(load_library().rp_profile_every(eng, every))


def rp_profile_read(eng: int, cap: int = 64):
    out = (RpKernelStats * cap)()
    n = ctypes.c_int32()
    _check(load_library().rp_profile_read(eng, out, cap, ctypes.byref(n)))
    return [out[i].as_dict() for i in range(n.value)]


def rp_stream_read_gbs(buf, reps: int = 5) -> float:
    """HBM read ceiling in GB/s: the fastest of `reps` streaming reads of the device tensor `buf`
    (contiguous; use more than 256 MB so that the last-level cache does not hold it)."""
    import torch
    gbs = ctypes.c_double()
    stream = torch.cuda.current_stream(buf.device).cuda_stream
    _check(load_library().rp_stream_read_gbs(ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(),
                                             reps, ctypes.c_void_p(stream), ctypes.byref(gbs)))
    return gbs.value


def rp_last_error() -> str:
    return load_library().rp_last_error().decode()


# ---- convenience owner of the device buffers ----------------------------------------

def model_config(shape) -> RpModelConfig:
    """RpModelConfig from any object with the Qwen2.5 shape attributes."""
    return RpModelConfig(shape.layers, shape.hidden, shape.n_q, shape.n_kv, shape.head_dim, shape.inter,
                         shape.vocab, shape.eps, shape.theta, 1 if shape.tied else 0,
                         RP_DTYPE_BF16 if shape.dtype == "bf16" else RP_DTYPE_F32)


class Engine:
    """An engine over torch-allocated workspaces on the current CUDA (HIP) device.

    weights: dict with "embed", "final_norm", "lm_head" (None if tied) and
    "layers" (list of dicts with the rp_layer_weights field names), all
    contiguous device tensors of the model dtype.  The dict is kept alive.
    pack_weights: for a bf16 model, also allocate the packed copy of the
    weights that the decode GEMMs stream (rp_engine_set_packed_weights).
    """

    def __init__(self, shape, weights: dict, max_seqs: int, max_prefill_tokens: int, max_context: int,
                 kv_pages: int, stream=None, pack_weights: bool = True):
        import torch
        self.torch = torch
        self.shape = shape
        self.cfg = model_config(shape)
        self.limits = RpEngineLimits(max_seqs, max_prefill_tokens, max_context, 64, kv_pages)
        kv_bytes, sc_bytes = rp_workspace_size(self.cfg, self.limits)
        dev = weights["embed"].device
        self.kv = torch.empty(kv_bytes, dtype=torch.uint8, device=dev)
        self.scratch = torch.empty(sc_bytes, dtype=torch.uint8, device=dev)
        self.weights = weights
        self._w, self._layers = weights_struct(shape, weights)
        self.stream = stream if stream is not None else torch.cuda.current_stream(dev)
        self.handle = rp_engine_create(self.cfg, self._w, self.limits, self.kv.data_ptr(), kv_bytes,
                                       self.scratch.data_ptr(), sc_bytes, self.stream.cuda_stream)
        self.max_seqs = max_seqs
        self.packed = None
        if pack_weights and shape.dtype == "bf16":
            nbytes = rp_packed_weights_bytes(self.cfg)
            self.packed = torch.empty(nbytes, dtype=torch.uint8, device=dev)
            rp_engine_set_packed_weights(self.handle, self.packed.data_ptr(), nbytes)

    def close(self):
        if getattr(self, "handle", None):
            rp_engine_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prefill(self, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed=0, temperature=0.0,
                logits: bool = False, first_tokens: bool = False):
        torch = self.torch
        out = None
        if logits:
            out = torch.empty((len(seq_ids), self.shape.vocab), dtype=torch.float32, device=self.kv.device)
        first = rp_prefill(self.handle, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed, temperature,
                           None if out is None else out.data_ptr(), first_tokens)
        return out, first

    def decode_step(self, forced_tokens=None, logits: bool = False):
        torch = self.torch
        out = None
        if logits:
            out = torch.empty((self.max_seqs, self.shape.vocab), dtype=torch.float32, device=self.kv.device)
        n, rows = rp_decode_step(self.handle, forced_tokens, None if out is None else out.data_ptr(), self.max_seqs)
        return n, rows, (None if out is None else out[:n])

    def free_finished(self):
        return rp_free_finished(self.handle, self.max_seqs)

    def abort(self, seq_ids):
        rp_abort(self.handle, seq_ids)

    def get_tokens(self, seq_id: int, cap: int):
        return rp_get_tokens(self.handle, seq_id, cap)

    def get_logprobs(self, seq_id: int, cap: int):
        return rp_get_logprobs(self.handle, seq_id, cap)

    def set_eos(self, eos_token: int):
        rp_set_eos(self.handle, eos_token)

    def set_kv_policy(self, policy: int):
        rp_set_kv_policy(self.handle, policy)

    def kv_status(self) -> dict:
        return rp_kv_status(self.handle)

    def step_trace(self, cap: int):
        rp_step_trace_enable(self.handle, cap)

    def step_trace_read(self, cap: int = 1 << 20):
        return rp_step_trace_read(self.handle, cap)

    def profile(self, classes, every: int = 1):
        rp_profile_every(self.handle, every)
        rp_profile_enable(self.handle, classes)

    def profile_read(self):
        return rp_profile_read(self.handle)

    def rollout(self, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed, temperature, round_ids=None,
                details: bool = False):
        return rp_rollout_generate(self.handle, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed,
                                   temperature, round_ids, details=details)


    def rollout_tail_batched(self, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed, temperature,
                             P0: int, R0: int, eta: float, eta_r: Optional[float] = None):
        return rp_rollout_tail_batched(self.handle, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed,
                                       temperature, P0, R0, eta, eta_r)


def weights_struct(shape, weights: dict):
    """(RpWeights, its layer array) pointing at the device tensors of `weights`; keep both alive."""
    dev = weights["embed"].device
    layers = (RpLayerWeights * shape.layers)()
    for i, L in enumerate(weights["layers"]):
        for f in _LAYER_FIELDS:
            t = L[f]
            assert t.is_contiguous() and t.device == dev
            setattr(layers[i], f, t.data_ptr())
    lm = weights.get("lm_head")
    w = RpWeights(weights["embed"].data_ptr(), weights["final_norm"].data_ptr(),
                  None if lm is None else lm.data_ptr(), layers)
    return w, layers


def generate(shape, weights: dict, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed: int,
             temperature: float, *, limits: RpEngineLimits, schedule_mode: int = SCHEDULE_NONE, round_ids=None,
             tail: Optional[RpTailParams] = None, stream=None):
    """rp_generate with workspaces allocated here from torch (freed when the call returns)."""
    import torch
    cfg = model_config(shape)
    kv_bytes, sc_bytes = rp_workspace_size(cfg, limits)
    dev = weights["embed"].device
    kv = torch.empty(kv_bytes, dtype=torch.uint8, device=dev)
    scratch = torch.empty(sc_bytes, dtype=torch.uint8, device=dev)
    w, layers = weights_struct(shape, weights)
    stream = stream if stream is not None else torch.cuda.current_stream(dev)
    return rp_generate(cfg, w, limits, kv.data_ptr(), kv_bytes, scratch.data_ptr(), sc_bytes, stream.cuda_stream,
                       seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed, temperature, schedule_mode,
                       round_ids, tail)


def weights_for_engine(w: dict) -> dict:
    """Contiguous tensors keyed by the rp_layer_weights names (a shallow copy)."""
    out = {"embed": w["embed"].contiguous(), "final_norm": w["final_norm"].contiguous(),
           "lm_head": None if w.get("lm_head") is None else w["lm_head"].contiguous(),
           "layers": [{f: L[f].contiguous() for f in _LAYER_FIELDS} for L in w["layers"]]}
    return out


def exported_names() -> Sequence[str]:
    return list(SIGNATURES)
