"""Host-only replica simulation: step-model fit, replica clocks, and Algorithm 1's trigger."""
import numpy as np
import pytest

from paper_2509_21009_amd.replica_sim import StepModel, simulate


def test_fit_recovers_a_linear_step_model():
    rng = np.random.default_rng(0)
    rows = rng.integers(1, 65, 400)
    ctx = rows * rng.integers(100, 9000, 400)
    dec = np.stack([np.zeros(400), np.zeros(400), rows, ctx, 1.5 + 0.02 * rows + 3e-6 * ctx], 1)
    tok = rng.integers(100, 16000, 50)
    pre = np.stack([np.ones(50), np.zeros(50), tok, tok * (tok + 1) / 2, 0.3 + 1e-4 * tok + 2e-9 * tok * (tok + 1) / 2], 1)
    m = StepModel.fit(np.concatenate([dec, pre]))
    assert np.allclose(m.decode, [1.5, 0.02, 3e-6], rtol=1e-6, atol=1e-9)
    assert np.allclose(m.prefill, [0.3, 1e-4, 2e-9], rtol=1e-6, atol=1e-12)


def test_replica_clock_closed_forms():
    lens = [5, 1, 9, 3]
    prompts = [10, 20, 30, 40]
    const = StepModel([2.0, 0.0, 0.0], [0.0, 0.0, 0.0])
    r = simulate(prompts, lens, 1, const)
    assert r["step_ms"] == pytest.approx(2.0 * (max(lens) - 1))      # one step per token after the first
    per_row = StepModel([0.0, 1.0, 0.0], [0.0, 0.0, 0.0])
    r = simulate(prompts, lens, 1, per_row)
    assert r["step_ms"] == pytest.approx(sum(l - 1 for l in lens))    # sum over steps of live rows
    per_ctx = StepModel([0.0, 0.0, 1.0], [0.0, 0.0, 0.0])
    r = simulate([7], [4], 1, per_ctx)
    assert r["step_ms"] == pytest.approx(8 + 9 + 10)                  # contexts p + 1, p + 2, p + 3


def test_barrier_and_idle_across_replicas():
    m = StepModel([1.0, 0.0, 0.0], [0.0, 0.0, 0.0])
    lens = [10, 2, 2, 2]                                               # replica 0 holds the long one
    r = simulate([5] * 4, lens, 4, m)
    assert r["step_ms"] == pytest.approx(9.0)
    assert r["idle_gpu_s"] == pytest.approx(3 * (9.0 - 1.0) / 1e3)
    same = simulate([5] * 4, [6] * 4, 4, m)
    assert same["idle_gpu_s"] == 0.0 and same["replica_idle_frac"] == 0.0


def _trainer(cap_gb, hist):
    return {"history": hist, "kv_bytes_per_token": 1000, "kv_capacity": cap_gb * 1e9, "lo": 0.2, "hi": 0.5,
            "delta": 0.05}


def test_scale_down_fires_inside_the_window_and_frees_half():
    m = StepModel([1.0, 0.0, 0.0], [0.0, 0.0, 0.0])
    rng = np.random.default_rng(3)
    lens = rng.integers(2, 200, 64)
    r = simulate([10] * 64, lens, 8, m, trainer=_trainer(1e9, lens))
    assert r["scaled"] is not None
    assert 0.2 <= r["scaled"]["completed"] <= 0.5 and r["scaled"]["freed"] == 4
    assert r["checks"][-1]["scaled"] and all(0.2 <= c["completed"] <= 0.5 for c in r["checks"])
    assert r["train_gpu_s"] > 0
    # every request still ends: the rollout finishes no earlier than the longest request
    assert r["step_ms"] >= max(lens) - 1


def test_scale_down_refused_when_projected_kv_exceeds_memory():
    m = StepModel([1.0, 0.0, 0.0], [0.0, 0.0, 0.0])
    lens = np.arange(2, 66)
    r = simulate([10] * 64, lens, 8, m, trainer=_trainer(1e-6, lens))
    assert r["scaled"] is None and r["checks"] and not any(c["scaled"] for c in r["checks"])
    # checks at least 5% of new completions apart
    fr = [c["completed"] for c in r["checks"]]
    assert all(b - a >= 0.05 - 1e-9 for a, b in zip(fr, fr[1:]))
