"""GPU: rp_generate_static, the entry point that allocates nothing, against
rp_generate (the same call over caller workspaces).

Two calls in a row, the second with a smaller input, for the tiny fp32
model and for a one-layer bf16 model of the 0.5B layer shape (which uses the
split-K partial, decode-split and sampler scratch of the bf16 path): tokens,
log-probabilities, lengths and round counts equal bit for bit, since the same
kernels run on the same inputs and the engine clears what must start at zero.
Limits beyond the static array are refused before anything runs.
"""
import numpy as np
import pytest

from tests.gpu_helpers import log, rp, to_device
from workloads import SHAPES, make_weights, make_workload, truncated

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")
STATIC_BYTES = 64 << 20


def _both(R, shape, wd, limits, ids, toks, offs, max_new, seed, temp, mode, rounds=None):
    a = R.generate(shape, wd, ids, toks, offs, max_new, seed, temp, limits=limits, schedule_mode=mode,
                   round_ids=rounds)
    w, layers = R.weights_struct(shape, wd)
    stream = torch.cuda.current_stream(DEV).cuda_stream
    b = R.rp_generate_static(R.model_config(shape), w, limits, stream, ids, toks, offs, max_new, seed, temp,
                             mode, rounds)
    torch.cuda.synchronize()
    return a, b


def _same(a, b):
    assert np.array_equal(a[0], b[0]), "tokens differ"
    assert np.array_equal(a[1], b[1]), "log-probabilities differ"
    assert np.array_equal(a[2], b[2]) and np.array_equal(a[3], b[3])
    assert [(x["round_id"], x["n_seqs"], x["decode_steps"], x["generated_tokens"]) for x in a[4]] == \
           [(x["round_id"], x["n_seqs"], x["decode_steps"], x["generated_tokens"]) for x in b[4]]


def test_static_entry_matches_generate_tiny_twice():
    R = rp()
    s = SHAPES["tiny"]
    wd = R.weights_for_engine(to_device(make_weights(s, seed=0, device="cpu"), DEV))
    wl = make_workload("tiny")
    lim = R.RpEngineLimits(8, 256, 128, 64, 32)
    kv, sc = R.rp_workspace_size(R.model_config(s), lim)
    assert kv + sc <= STATIC_BYTES
    log("no-alloc tiny: call 1, 8 sequences")
    mn = np.array([64, 5, 64, 33, 1, 64, 12, 64], np.int32)
    a, b = _both(R, s, wd, lim, wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, mn, 0, 0.0, R.SCHEDULE_NONE)
    _same(a, b)
    log("no-alloc tiny: call 2, 3 sequences, two rounds, T = 1")
    sub = wl.subset([2, 5, 7])
    a, b = _both(R, s, wd, R.RpEngineLimits(4, 64, 128, 64, 8), sub.seq_ids, sub.prompt_tokens, sub.prompt_offsets,
                 np.array([20, 7, 30], np.int32), 9, 1.0, R.SCHEDULE_ROUNDS, np.array([1, 0, 1], np.int32))
    _same(a, b)


def test_static_entry_matches_generate_bf16_twice():
    R = rp()
    s = truncated(SHAPES["qwen2.5-0.5b"], 1, vocab=4096)
    wd = R.weights_for_engine(to_device(make_weights(s, seed=1, device="cpu"), DEV))
    wl = make_workload("0.5b", s).subset(list(range(6)))
    plens = wl.prompt_lens()
    mn = np.array([48, 9, 48, 30, 1, 48], np.int32)
    lim = R.RpEngineLimits(8, 1024, int(plens.max()) + 64, 64, 64)
    kv, sc = R.rp_workspace_size(R.model_config(s), lim)
    log(f"no-alloc bf16: workspace {kv + sc} bytes; call 1, 6 sequences")
    assert kv + sc <= STATIC_BYTES
    a, b = _both(R, s, wd, lim, wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, mn, 202, 1.0, R.SCHEDULE_NONE)
    _same(a, b)
    log("no-alloc bf16: call 2, 2 sequences")
    sub = wl.subset([1, 4])
    a, b = _both(R, s, wd, R.RpEngineLimits(2, 256, int(plens.max()) + 64, 64, 24), sub.seq_ids, sub.prompt_tokens,
                 sub.prompt_offsets, np.array([25, 3], np.int32), 202, 1.0, R.SCHEDULE_NONE)
    _same(a, b)


def test_static_entry_refuses_limits_beyond_the_array():
    R = rp()
    s = SHAPES["tiny"]
    wd = R.weights_for_engine(to_device(make_weights(s, seed=0, device="cpu"), DEV))
    wl = make_workload("tiny").subset([0])
    big = R.RpEngineLimits(8, 256, 4096, 64, 40000)
    kv, sc = R.rp_workspace_size(R.model_config(s), big)
    assert kv + sc > STATIC_BYTES
    w, layers = R.weights_struct(s, wd)
    with pytest.raises(R.RollpackError) as e:
        R.rp_generate_static(R.model_config(s), w, big, torch.cuda.current_stream(DEV).cuda_stream, wl.seq_ids,
                             wl.prompt_tokens, wl.prompt_offsets, np.array([4], np.int32), 0, 0.0)
    assert e.value.status == 7 and "static workspace" in R.rp_last_error()
