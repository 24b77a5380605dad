"""GPU: the round metrics recomputed from their definition.

The bubble of section 2.2 is measured per sequence slot: a sequence that
finishes at f_i idles until its round ends at T, so
    idle_slot_s = sum_i (T - f_i)      slot_idle = idle_slot_s / (N T)
with T the round's makespan.  The per-step trace gives, for every step, its
end time from the round's start (end_ms); a sequence of max_new = L finishes
at the end of the step that produced its last token: the prefill chunk for
L = 1, else decode step L - 1.  Those, and the makespan, recompute both
metrics; the engine's own figures must agree to within the event timing
resolution (a few microseconds per departure).  The same trace also fixes
prefill_ms (the end of the last prefill chunk) and the decode-step count.
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


def _check_round(st, rec, max_new):
    T = st["makespan_ms"]
    pre = rec[rec["kind"] == 1]
    dec = rec[rec["kind"] == 0]
    assert len(pre) >= 1 and len(dec) == int(max_new.max()) - 1 == st["decode_steps"]
    assert np.all(rec["end_ms"] > 0) and np.all(np.diff(rec["end_ms"]) > 0)
    assert np.all(dec["rows"] == [int(np.sum(max_new > j)) for j in range(1, int(max_new.max()))])
    f = np.where(max_new == 1, pre["end_ms"][-1], dec["end_ms"][np.maximum(max_new, 2) - 2])
    idle_ref = float(np.sum(T - f)) * 1e-3
    slot_ref = idle_ref / (len(max_new) * T * 1e-3)
    log(f"  makespan {T:.3f} ms, idle {st['idle_slot_s']:.6f} s (recomputed {idle_ref:.6f}), "
        f"slot_idle {st['slot_idle']:.5f} (recomputed {slot_ref:.5f})")
    tol_s = len(max_new) * 20e-6 + 1e-3 * idle_ref
    assert abs(st["idle_slot_s"] - idle_ref) <= tol_s
    assert abs(st["slot_idle"] - slot_ref) <= tol_s / (len(max_new) * T * 1e-3)
    assert abs(st["prefill_ms"] - pre["end_ms"][-1]) <= 0.02 + 1e-3 * st["prefill_ms"]
    assert T >= dec["end_ms"][-1] and T - dec["end_ms"][-1] <= 0.05 * T + 1.0


@pytest.mark.parametrize("model", ["tiny", "0.5b-L2"])
def test_idle_metrics_from_step_trace(model):
    R = rp()
    if model == "tiny":
        s = SHAPES["tiny"]
        wd = to_device(make_weights(s, seed=0, device="cpu"), DEV)
        wl = make_workload("tiny")
        max_new = np.array([64, 5, 64, 33, 1, 64, 12, 40], np.int32)
        temp = 0.0
    else:
        s = truncated(SHAPES["qwen2.5-0.5b"], 2)
        wd = make_weights(s, seed=0, device=DEV)
        wl = make_workload("0.5b", s).subset(list(range(0, 256, 8)))
        max_new = np.minimum(wl.max_new, 300).astype(np.int32)
        max_new[3] = 1
        temp = 1.0
    plens = wl.prompt_lens()
    eng = R.Engine(s, R.weights_for_engine(wd), max_seqs=wl.n, max_prefill_tokens=int(plens.sum()),
                   max_context=int((plens + max_new).max()), kv_pages=int(np.sum((plens + max_new + 63) // 64)))
    eng.step_trace(1 << 16)
    log(f"{model}: rollout of {wl.n} sequences with the step trace on")
    _, stats = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, max_new, 5, temp)
    rec = eng.step_trace_read()
    eng.close()
    assert len(stats) == 1 and np.all(rec["round_id"] == 0)
    _check_round(stats[0], rec, max_new)


def test_idle_metrics_per_round_of_a_two_round_rollout():
    R = rp()
    s = SHAPES["tiny"]
    wd = to_device(make_weights(s, seed=0, device="cpu"), DEV)
    wl = make_workload("tiny")
    max_new = np.array([64, 5, 50, 33, 1, 64, 12, 40], np.int32)
    rounds = np.array([0, 1, 0, 1, 1, 0, 1, 0], np.int32)
    eng = R.Engine(s, R.weights_for_engine(wd), max_seqs=8, max_prefill_tokens=256, max_context=128, kv_pages=16)
    eng.step_trace(1 << 16)
    _, stats = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, max_new, 5, 0.0, rounds)
    rec = eng.step_trace_read()
    eng.close()
    assert [x["round_id"] for x in stats] == [0, 1]
    for r, st in enumerate(stats):
        log(f"round {r}:")
        _check_round(st, rec[rec["round_id"] == r], max_new[rounds == r])
