"""Shared helpers of the GPU parity tests (imported by tests marked gpu)."""
from __future__ import annotations

import dataclasses
import os
import sys

import numpy as np

from oracle import model as om
from oracle import sampling as osm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def rp():
    from paper_2509_21009_amd import rollpack
    if not os.path.exists(rollpack.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    rollpack.load_library()
    return rollpack


def to_device(w: dict, dev) -> dict:
    return {"embed": w["embed"].to(dev), "final_norm": w["final_norm"].to(dev),
            "lm_head": None if w["lm_head"] is None else w["lm_head"].to(dev),
            "layers": [{k: v.to(dev).contiguous() for k, v in L.items()} for L in w["layers"]]}


@dataclasses.dataclass
class ParityResult:
    max_rel_err: float
    positions: int
    greedy_agree: int
    id_checked: int
    id_mismatch: int
    worst: tuple


ORACLE_CHUNK = 2048


def oracle_rollout(w64, shape, prompt, n_new, temperature, seed, seq_id, rnd=None):
    """oracle.model.generate with the seeded sampler, the prompt prefilled in pieces of
    ORACLE_CHUNK tokens (KVState.step is incremental: pieces equal one whole step up to the
    order of fp64 sums, and bound the [queries, keys] score matrices of long prompts)."""
    sample_fn = osm.sampler(temperature, seed, seq_id)
    if len(prompt) <= ORACLE_CHUNK:
        return om.generate(w64, shape, prompt, n_new, sample_fn, rnd)
    st = om.KVState(shape, rnd)
    for o in range(0, len(prompt), ORACLE_CHUNK):
        logits = st.step(w64, prompt[o:o + ORACLE_CHUNK])[-1]
    p = len(prompt)
    toks, rows = [], []
    for j in range(n_new):
        t = int(sample_fn(logits, p + j))
        toks.append(t)
        rows.append(logits)
        if j + 1 < n_new:
            logits = st.step(w64, [t])[-1]
    return np.array(toks, np.int32), np.array(rows)


def teacher_forced_parity(eng, shape, w64, wl, n_new, tol, temperature, seed, rnd=None, check=None):
    """Prefill + (n_new - 1) teacher-forced decode steps on the GPU vs the oracle.

    Per position r: e_r = max|l_gpu - l_ref| / max|l_ref|; the GPU's sampled
    id must equal the oracle's wherever the oracle's top-2 score gap exceeds
    tol * max|l_ref| / T (T = 1 for greedy).  With `check` (sequence indices),
    every sequence runs on the GPU but only those are compared; the others are
    forced with seeded random tokens.
    """
    import torch
    n = wl.n
    idx = list(range(n)) if check is None else list(check)
    refs = {i: oracle_rollout(w64, shape, wl.prompt(i), n_new, temperature, seed, int(wl.seq_ids[i]), rnd)
            for i in idx}
    forced = np.random.default_rng(1234).integers(0, shape.vocab, size=(n, n_new)).astype(np.int32)
    for i in idx:
        forced[i] = refs[i][0]
    max_new = np.full(n, n_new, np.int32)
    logits0, _ = eng.prefill(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, max_new, seed, temperature,
                             logits=True)
    gpu_log = [logits0.cpu().numpy().astype(np.float64)]
    for j in range(1, n_new):
        b, rows, lg = eng.decode_step(forced_tokens=forced[:, j - 1], logits=True)
        assert b == n and np.array_equal(rows, wl.seq_ids)
        gpu_log.append(lg.cpu().numpy()[idx].astype(np.float64))
    torch.cuda.synchronize()
    gpu_log[0] = gpu_log[0][idx]
    gpu_log = np.stack(gpu_log, axis=1)               # [len(idx), n_new, V]
    gpu_tok = np.stack([eng.get_tokens(int(wl.seq_ids[i]), n_new) for i in idx])
    ref_tok = np.stack([refs[i][0] for i in idx])      # [len(idx), n_new]
    ref_log = np.stack([refs[i][1] for i in idx])      # [len(idx), n_new, V]
    freed = eng.free_finished()
    assert sorted(freed.tolist()) == sorted(wl.seq_ids.tolist())
    err = np.max(np.abs(gpu_log - ref_log), axis=-1) / np.max(np.abs(ref_log), axis=-1)
    agree = int(np.sum(np.argmax(gpu_log, -1) == np.argmax(ref_log, -1)))
    checked = mism = 0
    t_eff = temperature if temperature > 0 else 1.0
    for k, i in enumerate(idx):
        for j in range(n_new):
            pos = len(wl.prompt(i)) + j
            s = osm.scores(ref_log[k, j], temperature, seed, int(wl.seq_ids[i]), pos)
            tau = tol * np.max(np.abs(ref_log[k, j])) / t_eff
            if osm.top2_gap(s) > tau:
                checked += 1
                if gpu_tok[k, j] != ref_tok[k, j]:
                    mism += 1
    worst = np.unravel_index(np.argmax(err), err.shape)
    return ParityResult(float(err.max()), int(err.size), agree, checked, mism, tuple(int(v) for v in worst))
