"""KV pressure on the GPU: on-demand pages, preemption and resume by recompute.

Under RP_KV_ON_DEMAND a pool smaller than the batch's total need forces the
engine to preempt running sequences and later recompute their KV from their
tokens (a prefill of prompt + generated tokens, cut into pieces when longer
than one prefill chunk).  Tokens are keyed by (seed, sequence id, position),
so the result must equal an unpressured run: exactly for the fp32 model,
whose kernels reduce every output in a fixed order whatever the batch and
whichever path (prefill or decode) computed the KV.  The bf16 prefill of a
prompt cut into pieces is checked against the oracle.
"""
import dataclasses

import numpy as np
import pytest

from tests.gpu_helpers import log, rp, teacher_forced_parity, to_device
from workloads import SHAPES, make_weights, truncated, weights_to_numpy
from workloads.gen import Workload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def tiny():
    s = SHAPES["tiny"]
    return s, to_device(make_weights(s, seed=0, device="cpu"), DEV)


def _engine(shape, wdev, max_seqs, max_prefill, max_ctx, pages):
    R = rp()
    return R.Engine(shape, R.weights_for_engine(wdev), max_seqs=max_seqs, max_prefill_tokens=max_prefill,
                    max_context=max_ctx, kv_pages=pages)


def _batch(shape, n, seed, p_rng=(20, 40), new_rng=(40, 88)):
    rng = np.random.default_rng(seed)
    plen = rng.integers(p_rng[0], p_rng[1] + 1, size=n)
    prompts = [rng.integers(0, shape.vocab, size=int(p)).astype(np.int32) for p in plen]
    offs = np.zeros(n + 1, np.int64)
    offs[1:] = np.cumsum(plen)
    mn = rng.integers(new_rng[0], new_rng[1] + 1, size=n).astype(np.int32)
    return np.arange(500, 500 + n, dtype=np.int64), np.concatenate(prompts), offs, mn


@pytest.mark.parametrize("pages,max_prefill", [(14, 48), (10, 512), (26, 48)])
def test_preempted_rollout_equals_unpressured(tiny, pages, max_prefill):
    s, wd = tiny
    R = rp()
    ids, toks, offs, mn = _batch(s, 12, 3)
    need = int(np.sum((np.diff(offs) + mn - 1 + 63) // 64))
    log(f"preemption: 12 sequences needing {need} pages in a pool of {pages}, prefill chunk {max_prefill}")
    ref_eng = _engine(s, wd, 16, 512, 128, need)
    ref, _ = ref_eng.rollout(ids, toks, offs, mn, 9, 1.0)
    ref_eng.close()
    eng = _engine(s, wd, 16, max_prefill, 128, pages)
    eng.set_kv_policy(R.KV_ON_DEMAND)
    got, st = eng.rollout(ids, toks, offs, mn, 9, 1.0)
    status = eng.kv_status()
    eng.close()
    log(f"  {st[0]['preemptions']} preemptions, {st[0]['recomputed_tokens']} tokens recomputed, "
        f"{st[0]['decode_steps']} steps")
    assert np.array_equal(got, ref)
    assert st[0]["generated_tokens"] == int(mn.sum())
    if pages < need:
        assert st[0]["preemptions"] > 0 and st[0]["recomputed_tokens"] > 0
    assert st[0]["peak_pages"] <= pages
    assert status["running"] == 0 and status["waiting"] == 0 and status["free_pages"] == pages


def test_step_api_under_pressure(tiny):
    """prefill / decode_step / get_tokens / abort / free_finished with sequences preempted between steps."""
    s, wd = tiny
    R = rp()
    ids, toks, offs, mn = _batch(s, 8, 4, p_rng=(50, 60), new_rng=(60, 60))
    ref_eng = _engine(s, wd, 8, 512, 128, 16)
    ref, _ = ref_eng.rollout(ids, toks, offs, mn, 2, 1.0)
    ref_eng.close()
    eng = _engine(s, wd, 8, 512, 128, 10)
    with pytest.raises(R.RollpackError):            # no such policy
        eng.set_kv_policy(7)
    eng.set_kv_policy(R.KV_ON_DEMAND)
    eng.prefill(ids, toks, offs, mn, 2, 1.0)        # 8 one-page prompts
    with pytest.raises(R.RollpackError) as e:
        eng.set_kv_policy(R.KV_RESERVE)              # not while sequences are live
    assert e.value.status == 5
    with pytest.raises(R.RollpackError):            # teacher forcing needs reserved pages
        eng.decode_step(forced_tokens=np.zeros(8, np.int32))
    saw_waiting = aborted = None
    out = {}
    for _ in range(200):
        n, rows, _ = eng.decode_step()
        st = eng.kv_status()
        if st["waiting"] and saw_waiting is None:
            saw_waiting = st
            # the latest arrival is preempted first; it still answers get_tokens; abort it
            victim = int(ids[-1])
            assert victim not in rows.tolist()
            part = eng.get_tokens(victim, 128)
            assert 0 < len(part) < 60
            assert np.array_equal(part, ref[(victim - 500) * 60:(victim - 500) * 60 + len(part)])
            eng.abort(np.array([victim], np.int64))
            aborted = victim
        for i in ids:
            i = int(i)
            if i != aborted and i not in out:
                try:
                    t = eng.get_tokens(i, 128)
                except R.RollpackError:
                    continue
                if len(t) == 60:
                    out[i] = t
        eng.free_finished()
        st = eng.kv_status()
        if n == 0 and st["waiting"] == 0 and st["running"] == 0:
            break
    status = eng.kv_status()
    eng.close()
    assert saw_waiting is not None and status["preemptions"] > 0
    assert status["running"] == 0 and status["waiting"] == 0 and status["free_pages"] == 10
    for i, t in out.items():
        assert np.array_equal(t, ref[(i - 500) * 60:(i - 500 + 1) * 60]), i
    assert len(out) == 7


def test_tail_batched_race_under_pressure(tiny):
    """A short round whose responses are preempted still accepts P0 prompts with R0 finished responses;
    every token equals the unpressured run's."""
    s, wd = tiny
    R = rp()
    from workloads import make_rl_batch
    b = make_rl_batch(s, 6, 3, p_lo=50, p_hi=60, median=40, sigma_p=0.5, sigma_r=0.5, lo=8, hi=64, seed=41)
    ref_eng = _engine(s, wd, 32, 512, 128, 64)
    u = b.sequences(range(6), 3)
    full, _ = ref_eng.rollout(u.seq_ids, u.prompt_tokens, u.prompt_offsets, u.max_new, b.sample_seed, 1.0)
    ref_eng.close()
    eng = _engine(s, wd, 32, 512, 128, 11)
    eng.set_kv_policy(R.KV_ON_DEMAND)
    resp, glen, acc, kept, stats = eng.rollout_tail_batched(b.seq_ids, b.prompt_tokens, b.prompt_offsets, b.max_new,
                                                            b.sample_seed, 1.0, 2, 2, 1.5)
    eng.close()
    log(f"race under pressure: {[(st['kind'], st['decode_steps'], st['preemptions']) for st in stats]}")
    assert sum(st["preemptions"] for st in stats) > 0
    assert (acc >= 0).all() and (kept.sum(axis=1) == 2).all()
    off = np.concatenate([[0], np.cumsum(b.max_new.reshape(-1))])
    for i in range(u.n):
        p, r = divmod(i, 3)
        g = glen[p, r]
        assert np.array_equal(resp[off[i]:off[i] + g], full[off[i]:off[i] + g]), (p, r)
        if kept[p, r]:
            assert g == b.max_new[p, r]


def test_bf16_prompt_cut_into_prefill_pieces():
    """Prompts of 300 and 200 tokens prefilled in pieces of at most 128 (the later pieces attend to
    keys an earlier chunk wrote), then teacher-forced decode, against the oracle."""
    s = dataclasses.replace(truncated(SHAPES["qwen2.5-0.5b"], 1, vocab=2048), tied=False)
    wd = make_weights(s, seed=8, device=DEV)
    w64 = weights_to_numpy(wd)
    rng = np.random.default_rng(12)
    plen = [300, 17, 200]
    prompts = [rng.integers(0, s.vocab, size=p).astype(np.int32) for p in plen]
    offs = np.zeros(4, np.int64)
    offs[1:] = np.cumsum(plen)
    wl = Workload("pieces", s, np.array([3, 4, 5], np.int64), np.concatenate(prompts), offs,
                  np.full(3, 6, np.int32), np.arange(3, dtype=np.int32), 1.0, 11)
    eng = _engine(s, wd, 4, 128, 320, 20)
    r = teacher_forced_parity(eng, s, w64, wl, 6, 2e-2, 1.0, 11)
    eng.close()
    log(f"prefill pieces: {r}")
    assert r.max_rel_err <= 2e-2 and r.id_mismatch == 0, r


def test_pressured_rollout_matches_the_oracle(tiny):
    """Preemption by recompute against the oracle itself (not only against an unpressured
    GPU run): with a pool of 12 pages for 12 sequences that need 24, every sequence's seeded
    T = 1 tokens equal oracle.model.generate with the oracle's sampler up to the first
    position whose top-2 score margin is within 1e-4 of the logits' scale (after a near-tie
    the two fp32/fp64 paths may legitimately diverge)."""
    from oracle import model as om
    from oracle import sampling as osm
    from workloads import weights_to_numpy
    s, wd = tiny
    R = rp()
    w64 = weights_to_numpy({k: v for k, v in wd.items()})
    ids, toks, offs, mn = _batch(s, 12, 3)
    eng = _engine(s, wd, 16, 48, 128, 12)
    eng.set_kv_policy(R.KV_ON_DEMAND)
    got, st = eng.rollout(ids, toks, offs, mn, 9, 1.0)
    eng.close()
    log(f"pressured vs oracle: {st[0]['preemptions']} preemptions, {st[0]['recomputed_tokens']} tokens recomputed")
    assert st[0]["preemptions"] > 0
    resp_off = np.concatenate([[0], np.cumsum(mn)])
    full = 0
    for i in range(12):
        ref, logits = om.generate(w64, s, toks[offs[i]:offs[i + 1]], int(mn[i]), osm.sampler(1.0, 9, int(ids[i])))
        mine = got[resp_off[i]:resp_off[i + 1]]
        p = int(offs[i + 1] - offs[i])
        for j in range(int(mn[i])):
            sc = osm.scores(logits[j], 1.0, 9, int(ids[i]), p + j)
            if osm.top2_gap(sc) <= 1e-4 * np.max(np.abs(logits[j])):
                break
            assert mine[j] == ref[j], (i, j)
        else:
            full += 1
    log(f"pressured vs oracle: {full}/12 sequences identical over all their tokens")
    assert full >= 10
