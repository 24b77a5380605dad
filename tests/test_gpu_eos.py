"""Per-token log-probabilities and end-of-sequence stopping on the GPU.

Log-probabilities are checked against the oracle's fp64 definition, applied
to the logits the same step produced on the GPU (this isolates the sampler's
log-sum-exp over the vocabulary) and, for the fp32 model, to the oracle's own
logits.  A response that stops at the end-of-sequence token must equal the
forced-length response cut after the first occurrence of that token
(tokens are keyed by position), with the same log-probabilities, through the
round runner, the step API, tail-batched rounds and preemption.
"""

import numpy as np
import pytest

from oracle import model as om
from oracle import sampling as osm
from tests.gpu_helpers import log, rp, to_device
from workloads import SHAPES, make_rl_batch, make_weights, make_workload, truncated, weights_to_numpy  # noqa: F401

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def tiny():
    s = SHAPES["tiny"]
    w = make_weights(s, seed=0, device="cpu")
    return s, to_device(w, DEV), weights_to_numpy(w)


def _engine(shape, wdev, max_seqs, max_prefill, max_ctx, pages):
    R = rp()
    return R.Engine(shape, R.weights_for_engine(wdev), max_seqs=max_seqs, max_prefill_tokens=max_prefill,
                    max_context=max_ctx, kv_pages=pages)


def _teacher_forced_logprobs(eng, wl, n_new, temperature, seed, forced):
    """GPU logits, sampled tokens and reported log-probabilities over n_new positions."""
    n = wl.n
    lg0, _ = eng.prefill(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, np.full(n, n_new, np.int32), seed,
                         temperature, logits=True)
    logits = [lg0.cpu().numpy().astype(np.float64)]
    for j in range(1, n_new):
        _, _, lg = eng.decode_step(forced_tokens=forced[:, j - 1], logits=True)
        logits.append(lg.cpu().numpy().astype(np.float64))
    logits = np.stack(logits, axis=1)
    toks = np.stack([eng.get_tokens(int(i), n_new) for i in wl.seq_ids])
    lps = np.stack([eng.get_logprobs(int(i), n_new) for i in wl.seq_ids])
    eng.free_finished()
    return logits, toks, lps


@pytest.mark.parametrize("temperature", [0.0, 0.8, 1.0])
def test_logprobs_tiny_fp32(tiny, temperature):
    s, wd, w64 = tiny
    wl = make_workload("tiny")
    refs = [om.generate(w64, s, wl.prompt(i), 16, lambda l, pos: int(np.argmax(l))) for i in range(wl.n)]
    forced = np.stack([r[0] for r in refs])
    eng = _engine(s, wd, 8, 256, 128, 32)
    logits, toks, lps = _teacher_forced_logprobs(eng, wl, 16, temperature, 3, forced)
    eng.close()
    own = np.array([[osm.logprob(logits[i, j], temperature, toks[i, j]) for j in range(16)] for i in range(wl.n)])
    ref = np.array([[osm.logprob(refs[i][1][j], temperature, toks[i, j]) for j in range(16)] for i in range(wl.n)])
    e_own, e_ref = np.abs(lps - own).max(), np.abs(lps - ref).max()
    log(f"tiny T={temperature}: |logprob - oracle(GPU logits)| {e_own:.2e}, |logprob - oracle| {e_ref:.2e}")
    assert e_own <= 1e-4 and e_ref <= 1e-3
    assert (lps <= 0).all()


def test_logprobs_full_vocabulary_bf16():
    """A 0.5B-shape layer with the real 151,936-entry vocabulary: the log-sum-exp runs over 75 chunks."""
    s = truncated(SHAPES["qwen2.5-0.5b"], 1)
    wd = make_weights(s, seed=3, device=DEV)
    wl = make_workload("0.5b", s).subset([0, 9, 40])
    rng = np.random.default_rng(2)
    forced = rng.integers(0, s.vocab, size=(wl.n, 6)).astype(np.int32)
    max_ctx = int(wl.prompt_lens().max()) + 8
    eng = _engine(s, wd, 4, 1024, max_ctx, 4 * (max_ctx // 64 + 2))
    logits, toks, lps = _teacher_forced_logprobs(eng, wl, 6, 1.0, wl.sample_seed, forced)
    eng.close()
    own = np.array([[osm.logprob(logits[i, j], 1.0, toks[i, j]) for j in range(6)] for i in range(wl.n)])
    err = np.abs(lps - own).max()
    log(f"0.5B vocabulary: |logprob - oracle(GPU logits)| {err:.2e}")
    assert err <= 1e-4


def _eos_token(full, mn):
    """A token that occurs in the middle of some responses and never in others."""
    counts = {}
    off = np.concatenate([[0], np.cumsum(mn)])
    for i in range(len(mn)):
        for t in set(full[off[i]:off[i + 1]].tolist()):
            counts[t] = counts.get(t, 0) + 1
    # the token present in the most responses, but not all
    return max((c, t) for t, c in counts.items() if c < len(mn))[1]


def test_eos_rollout_equals_cut_forced_rollout(tiny):
    s, wd, _ = tiny
    wl = make_workload("tiny")
    mn = np.array([64, 40, 64, 17, 64, 52, 30, 64], np.int32)
    eng = _engine(s, wd, 8, 256, 128, 32)
    full, flp, flen, _ = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, mn, 7, 1.0, details=True)
    eos = _eos_token(full, mn)
    eng.set_eos(eos)
    got, glp, glen, st = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, mn, 7, 1.0, details=True)
    with pytest.raises(rp().RollpackError):
        eng.set_eos(s.vocab)
    eng.close()
    assert np.array_equal(flen, mn)
    off = np.concatenate([[0], np.cumsum(mn)])
    stopped = 0
    for i in range(wl.n):
        want = osm.stop_at(full[off[i]:off[i + 1]], eos)
        assert glen[i] == len(want), (i, glen[i], len(want))
        assert got[off[i]:off[i] + glen[i]].tolist() == want
        assert np.array_equal(glp[off[i]:off[i] + glen[i]], flp[off[i]:off[i] + glen[i]])
        stopped += glen[i] < mn[i]
    log(f"eos {eos}: {stopped} of {wl.n} responses stopped early; {st[0]['decode_steps']} steps")
    assert 0 < stopped < wl.n
    assert st[0]["generated_tokens"] == int(glen.sum())


def test_eos_step_api(tiny):
    """prefill / decode_step / get_tokens / get_logprobs / free_finished with an end-of-sequence token."""
    s, wd, _ = tiny
    R = rp()
    wl = make_workload("tiny")
    mn = np.full(wl.n, 48, np.int32)
    eng = _engine(s, wd, 8, 256, 128, 32)
    full, flp, _, _ = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, mn, 5, 1.0, details=True)
    eos = _eos_token(full, mn)
    eng.set_eos(eos)
    eng.prefill(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, mn, 5, 1.0)
    with pytest.raises(R.RollpackError) as e:
        eng.set_eos(-1)                       # not while sequences are live
    assert e.value.status == 5
    steps = 0
    while eng.decode_step()[0] > 0:
        steps += 1
        assert steps < 60
    for k, i in enumerate(wl.seq_ids):
        want = osm.stop_at(full[k * 48:(k + 1) * 48], eos)
        assert eng.get_tokens(int(i), 64).tolist() == want, k
        assert np.array_equal(eng.get_logprobs(int(i), 64), flp[k * 48:k * 48 + len(want)])
    assert sorted(eng.free_finished().tolist()) == sorted(wl.seq_ids.tolist())
    eng.close()


def test_eos_in_tail_batched_and_preempted_rounds(tiny):
    s, wd, _ = tiny
    R = rp()
    b = make_rl_batch(s, 6, 3, p_lo=50, p_hi=60, median=40, sigma_p=0.5, sigma_r=0.5, lo=8, hi=64, seed=51)
    u = b.sequences(range(6), 3)
    eng = _engine(s, wd, 32, 512, 128, 64)
    full, _ = eng.rollout(u.seq_ids, u.prompt_tokens, u.prompt_offsets, u.max_new, b.sample_seed, 1.0)
    eos = _eos_token(full, u.max_new)
    eng.set_eos(eos)
    cut, _, clen, _ = eng.rollout(u.seq_ids, u.prompt_tokens, u.prompt_offsets, u.max_new, b.sample_seed, 1.0,
                                  details=True)
    resp, glen, acc, kept, stats = eng.rollout_tail_batched(b.seq_ids, b.prompt_tokens, b.prompt_offsets, b.max_new,
                                                            b.sample_seed, 1.0, 2, 2, 1.5)
    eng.close()
    off = np.concatenate([[0], np.cumsum(u.max_new)])
    for i in range(u.n):
        p, r = divmod(i, 3)
        want = osm.stop_at(full[off[i]:off[i + 1]], eos)
        assert clen[i] == len(want) and cut[off[i]:off[i] + clen[i]].tolist() == want
        g = glen[p, r]
        assert resp[off[i]:off[i] + g].tolist() == want[:g], (p, r)
        if kept[p, r]:
            assert g == len(want)
    assert (acc >= 0).all() and (kept.sum(axis=1) == 2).all()
    # the same stopping under KV pressure, with preemption and recompute
    eng = _engine(s, wd, 32, 512, 128, 11)
    eng.set_kv_policy(R.KV_ON_DEMAND)
    eng.set_eos(eos)
    got, _, plen, st = eng.rollout(u.seq_ids, u.prompt_tokens, u.prompt_offsets, u.max_new, b.sample_seed, 1.0,
                                   details=True)
    eng.close()
    log(f"eos under pressure: {st[0]['preemptions']} preemptions")
    assert np.array_equal(plen, clen)
    for i in range(u.n):
        assert np.array_equal(got[off[i]:off[i] + plen[i]], cut[off[i]:off[i] + plen[i]])
