"""GPU: the one-shot rp_generate (the problem statement's form, section 2.1)
against the engine calls it is made of, in its three schedule modes.

rp_generate creates an engine over the caller's workspaces, runs one rollout
call and destroys the engine; its tokens and log-probabilities must equal,
bit for bit, those of rp_rollout_generate / rp_rollout_tail_batched on an
engine with the same inputs (the same kernels run on the same data).  The
engine calls themselves are checked against the oracle in the other GPU
tests.
"""
import numpy as np
import pytest

from tests.gpu_helpers import log, rp, to_device
from workloads import SHAPES, make_weights, make_workload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def tiny():
    s = SHAPES["tiny"]
    return s, rp().weights_for_engine(to_device(make_weights(s, seed=0, device="cpu"), DEV))


def _limits(R, max_seqs=16, max_prefill=256, max_ctx=128, pages=64):
    return R.RpEngineLimits(max_seqs, max_prefill, max_ctx, 64, pages)


@pytest.mark.parametrize("mode", ["none", "rounds"])
def test_generate_equals_engine_rollout(tiny, mode):
    s, wd = tiny
    R = rp()
    wl = make_workload("tiny")
    max_new = np.array([64, 3, 17, 64, 1, 40, 9, 64], np.int32)
    rounds = np.array([1, 0, 1, 0, 0, 1, 1, 0], np.int32) if mode == "rounds" else None
    log(f"rp_generate mode={mode}")
    toks, logp, lens, kept, st = R.generate(
        s, wd, wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, max_new, 7, 0.8, limits=_limits(R),
        schedule_mode=R.SCHEDULE_ROUNDS if rounds is not None else R.SCHEDULE_NONE, round_ids=rounds)
    eng = R.Engine(s, wd, max_seqs=16, max_prefill_tokens=256, max_context=128, kv_pages=64)
    ref, ref_logp, ref_lens, ref_st = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, max_new, 7, 0.8,
                                                  rounds, details=True)
    eng.close()
    assert np.array_equal(toks, ref) and np.array_equal(logp, ref_logp)
    assert np.array_equal(lens, max_new) and np.array_equal(ref_lens, max_new) and kept.all()
    assert len(st) == len(ref_st) == (2 if rounds is not None else 1)
    for a, b in zip(st, ref_st):
        assert (a["round_id"], a["n_seqs"], a["decode_steps"], a["generated_tokens"]) == \
               (b["round_id"], b["n_seqs"], b["decode_steps"], b["generated_tokens"])


def test_generate_tail_batching_equals_engine_call(tiny):
    s, wd = tiny
    R = rp()
    n_prompts, r_spec, P0, R0 = 6, 3, 2, 2
    rng = np.random.default_rng(5)
    lens = rng.integers(2, 60, size=(n_prompts, r_spec)).astype(np.int32)
    plen = rng.integers(3, 30, size=n_prompts)
    ptoks = rng.integers(0, s.vocab, size=int(plen.sum())).astype(np.int32)
    poffs = np.concatenate([[0], np.cumsum(plen)]).astype(np.int64)
    ids = np.arange(100, 100 + n_prompts * r_spec, dtype=np.int64).reshape(n_prompts, r_spec)
    tail = R.RpTailParams(P0, R0, r_spec, 1.5, 1.5)
    log("rp_generate tail batching")
    toks, logp, glen, kept, st = R.generate(s, wd, ids.ravel(), ptoks, poffs, lens.ravel(), 3, 1.0,
                                            limits=_limits(R, max_seqs=24, pages=96),
                                            schedule_mode=R.SCHEDULE_TAIL_BATCHING, tail=tail)
    eng = R.Engine(s, wd, max_seqs=24, max_prefill_tokens=256, max_context=128, kv_pages=96)
    r_toks, r_glen, _, r_kept, r_st, r_logp = R.rp_rollout_tail_batched(
        eng.handle, ids, ptoks, poffs, lens, 3, 1.0, P0, R0, 1.5, 1.5, logprobs=True)
    eng.close()
    assert np.array_equal(glen, r_glen.ravel()) and np.array_equal(kept, r_kept.ravel())
    off = np.concatenate([[0], np.cumsum(lens.ravel())])
    for i in range(n_prompts * r_spec):
        a, b = off[i], off[i] + glen[i]
        assert np.array_equal(toks[a:b], r_toks[a:b]) and np.array_equal(logp[a:b], r_logp[a:b]), i
    assert [x["kind"] for x in st] == [x["kind"] for x in r_st]
    assert kept.reshape(n_prompts, r_spec).sum(1).tolist() == [R0] * n_prompts


def test_generate_rejects_mode_mismatches(tiny):
    s, wd = tiny
    R = rp()
    wl = make_workload("tiny").subset([0, 1])
    mn = np.array([4, 4], np.int32)
    for mode, rounds, tail in [(R.SCHEDULE_ROUNDS, None, None), (R.SCHEDULE_NONE, np.array([0, 1], np.int32), None),
                               (R.SCHEDULE_TAIL_BATCHING, None, None), (7, None, None)]:
        with pytest.raises(R.RollpackError) as e:
            R.generate(s, wd, wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, mn, 0, 0.0, limits=_limits(R),
                       schedule_mode=mode, round_ids=rounds, tail=tail)
        assert e.value.status == 1
