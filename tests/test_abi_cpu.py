"""CPU checks of the C-ABI library: it loads, exports every declared symbol,
its host-only calls behave, and the host C++ passes its sanitizer build."""
import math
import os
import re
import subprocess

import numpy as np
import pytest

from oracle import schedule as osch
from paper_2509_21009_amd import rollpack as rp
from workloads import SHAPES, make_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rollpack.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(rp.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return rp.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rp_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("rp_prefill", "rp_decode_step", "rp_free_finished", "rp_rollout_generate", "rp_generate",
                     "rp_abort", "rp_engine_create", "rp_workspace_size", "rp_plan_tail_batching", "rp_last_error"):
        assert required in names


def declaration_comments():
    """{function name: the comment block right before its declaration}."""
    text = open(HEADER).read()
    out = {}
    for m in re.finditer(r"/\*((?:(?!\*/).)*)\*/\s*(?:typedef[^;]*;\s*)*(?:rp_status|void|const char\*)\s+(rp_[a-z_]+)\s*\(",
                         text, flags=re.S):
        out[m.group(2)] = re.sub(r"\s+", " ", re.sub(r"\n\s*\*", " ", m.group(1)))
    return out


def test_core_declarations_cite_the_paper():
    """Each entry point of the boundary says which passage defines it: section 2.1 (rollout:
    prefill, decode, generate), section 3 (tail batching), section 5 (add / abort), section 4.x
    (KV pressure, profiling), or Algorithm 1; the allocation-free variant names its callers."""
    comments = declaration_comments()
    infra = {"rp_last_error", "rp_engine_destroy"}
    missing = [n for n in declared_functions() if n not in infra and n not in comments]
    assert not missing, missing
    uncited = [n for n, c in comments.items() if n not in infra and
               not re.search(r"section \d|Algorithm 1|cannot allocate", c)]
    assert not uncited, uncited
    for name, cites in {"rp_prefill": "section 2.1", "rp_decode_step": "section 2.1", "rp_generate": "section 2.1",
                        "rp_rollout_generate": "section 2.1", "rp_abort": "section 5",
                        "rp_rollout_tail_batched": "section 3", "rp_plan_tail_batching": "section 3",
                        "rp_free_finished": "Algorithm 1"}.items():
        assert cites in comments[name], (name, cites)


def test_library_exports_every_declared_symbol(lib):
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    out = subprocess.run(["nm", "-D", "--defined-only", rp.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (rp_\w+)", out))
    assert set(declared_functions()) <= exported
    assert set(rp.SIGNATURES) == set(declared_functions())


def test_workspace_size_and_kv_bytes(lib):
    s = SHAPES["qwen2.5-7b"]
    cfg = rp.model_config(s)
    assert rp.rp_kv_bytes_per_token(cfg) == s.kv_bytes_per_token() == 57344
    lim = rp.RpEngineLimits(64, 4096, 17408, 64, 1000)
    kv, sc = rp.rp_workspace_size(cfg, lim)
    assert kv == 1000 * 64 * 57344 and kv % 256 == 0 and sc % 256 == 0 and sc > 0
    lim2 = rp.RpEngineLimits(64, 4096, 17408, 64, 2000)
    assert rp.rp_workspace_size(cfg, lim2)[0] == 2 * kv


def test_packed_weights_bytes(lib):
    """The packed copy holds every projection and the LM head once (for these shapes every
    tensor is already a multiple of 256 bytes); the fp32 model has none."""
    for name in ("qwen2.5-7b", "qwen2.5-0.5b", "qwen2.5-32b"):
        s = SHAPES[name]
        per_layer = s.hidden * s.qkv_out + s.n_q * s.head_dim * s.hidden + 3 * s.hidden * s.inter
        assert rp.rp_packed_weights_bytes(rp.model_config(s)) == 2 * (s.layers * per_layer + s.vocab * s.hidden)
    assert rp.rp_packed_weights_bytes(rp.model_config(SHAPES["tiny"])) == 0


@pytest.mark.parametrize("field,value", [("head_dim", 96), ("n_kv_heads", 3), ("hidden", 100), ("vocab", 1000)])
def test_invalid_configs_are_rejected(lib, field, value):
    import dataclasses
    cfg = rp.model_config(dataclasses.replace(SHAPES["qwen2.5-0.5b"], **{
        {"head_dim": "head_dim", "n_kv_heads": "n_kv", "hidden": "hidden", "vocab": "vocab"}[field]: value}))
    with pytest.raises(rp.RollpackError) as e:
        rp.rp_workspace_size(cfg, rp.RpEngineLimits(8, 128, 256, 64, 16))
    assert e.value.status == 1 and rp.rp_last_error()


@pytest.mark.parametrize("lim", [(0, 128, 256, 64, 16), (8, 128, 256, 32, 16), (8, 128, 1, 64, 16),
                                 (8, 128, 256, 64, 0), (8, 128, 70000, 64, 16)])
def test_invalid_limits_are_rejected(lib, lim):
    with pytest.raises(rp.RollpackError) as e:
        rp.rp_workspace_size(rp.model_config(SHAPES["tiny"]), rp.RpEngineLimits(*lim))
    assert e.value.status == 1


def test_engine_create_rejects_bad_workspaces_without_gpu(lib):
    s = SHAPES["tiny"]
    cfg = rp.model_config(s)
    lim = rp.RpEngineLimits(4, 64, 128, 64, 8)
    layers = (rp.RpLayerWeights * s.layers)()
    w = rp.RpWeights(None, None, None, layers)
    with pytest.raises(rp.RollpackError) as e:
        rp.rp_engine_create(cfg, w, lim, 0, 0, 0, 0, 0)
    assert e.value.status == 1


def test_null_engine_calls_fail_cleanly(lib):
    n = rp.ctypes.c_int32()
    assert lib.rp_decode_step(None, None, None, None, rp.ctypes.byref(n)) == 1
    assert "null engine" in rp.rp_last_error()


def _lens(seed, n, r_spec):
    rng = np.random.default_rng(seed)
    return np.clip(np.rint(300 * np.exp(0.9 * rng.standard_normal((n, r_spec)))), 1, 8000).astype(np.int32)


@pytest.mark.parametrize("seed", range(16))
def test_tail_batching_plan_matches_oracle(lib, seed):
    rng = np.random.default_rng(seed)
    P0, R0 = int(rng.integers(1, 11)), int(rng.integers(1, 11))
    eta_p, eta_r = (float(rng.choice([1.0, 1.1, 1.25, 1.5])) for _ in range(2))
    r_spec = osch.spec_count(eta_r, R0)
    n = int(rng.integers(0, 60))
    lens = _lens(seed, n, r_spec)
    ours, acc, kept = rp.rp_plan_tail_batching(lens.reshape(n, r_spec), P0, R0, eta_p, eta_r)
    ref = osch.plan_tail_batching(lens.tolist(), P0, R0, eta_p, eta_r)
    assert len(ours) == len(ref)
    for a, b in zip(ours, ref):
        assert a["kind"] == b["kind"] and a["time"] == b["time"]
        assert a["launched"] == sorted(b["launched"])
        for (p, r), t in a["run"].items():
            assert t == b["run"].get((p, r), 0)
    for k, b in enumerate(ref):
        for p in b["accepted"]:
            assert acc[p] == k
            assert sorted(np.flatnonzero(kept[p]).tolist()) == b["kept"][p]


def test_tail_batching_rejects_bad_arguments(lib):
    with pytest.raises(rp.RollpackError):
        rp.rp_plan_tail_batching(np.ones((3, 2), np.int32), 0, 2, 1.0)
    with pytest.raises(rp.RollpackError):
        rp.rp_plan_tail_batching(np.ones((3, 2), np.int32), 1, 2, 1.25)   # r_spec must be ceil(1.25*2)=3


def test_host_cpp_under_sanitizers(tmp_path):
    csrc = os.path.join(ROOT, "paper_2509_21009_amd", "csrc")
    exe = tmp_path / "test_host"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           f"-I{csrc}", os.path.join(ROOT, "tests", "cpp", "test_host.cpp"), os.path.join(csrc, "tail_batch.cpp"),
           "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1"})
    assert r.returncode == 0, r.stderr
    assert "host tests passed" in r.stdout


def test_workload_shapes_follow_the_configs():
    w = make_workload("7b-long")
    assert w.n == 64 and w.max_new.min() >= 512 and w.max_new.max() <= 16384
    pl = w.prompt_lens()
    assert pl.min() >= 128 and pl.max() <= 1024
    m = make_workload("7b-mixed")
    assert m.n == 576 and set(m.round_id.tolist()) == {0, 1} and len(set(m.seq_ids.tolist())) == 576
    c2 = make_workload("0.5b")
    assert c2.n == 256 and len(set(c2.prompt_group.tolist())) == 32


def test_rl_batch_lengths_are_prompt_correlated():
    from workloads import SHAPES, make_rl_batch
    s = SHAPES["qwen2.5-0.5b"]
    kw = dict(p_lo=64, p_hi=512, median=512, lo=32, hi=4096, seed=7)
    a = make_rl_batch(s, 200, 10, sigma_p=0.6, sigma_r=0.53, **kw)
    b = make_rl_batch(s, 200, 10, sigma_p=0.6, sigma_r=0.53, **kw)
    assert np.array_equal(a.max_new, b.max_new) and np.array_equal(a.prompt_tokens, b.prompt_tokens)
    assert a.max_new.min() >= 32 and a.max_new.max() <= 4096
    assert len(set(a.seq_ids.reshape(-1).tolist())) == 2000
    same = make_rl_batch(s, 50, 4, sigma_p=0.6, sigma_r=0.0, **kw)      # no per-response spread
    assert (same.max_new == same.max_new[:, :1]).all()
    wider = make_rl_batch(s, 200, 12, sigma_p=0.6, sigma_r=0.53, **kw)  # more responses, same first ten
    assert np.array_equal(wider.max_new[:, :10], a.max_new) and np.array_equal(wider.prompt_tokens, a.prompt_tokens)
    # log-length variance splits into a between-prompt part (~sigma_p^2) and a within part (~sigma_r^2)
    lg = np.log(make_rl_batch(s, 2000, 10, sigma_p=0.6, sigma_r=0.53, p_lo=64, p_hi=512, median=512, lo=1,
                              hi=10**7, seed=8).max_new)
    within = lg.var(axis=1, ddof=1).mean()
    between = lg.mean(axis=1).var(ddof=1) - within / 10
    assert abs(within - 0.53 ** 2) < 0.03 and abs(between - 0.6 ** 2) < 0.05
    # sequences(): prompt-major, each response with its own prompt's ids
    w = a.sequences([3, 5], 2)
    assert w.seq_ids.tolist() == [30, 31, 50, 51] and w.max_new.tolist() == [a.max_new[3, 0], a.max_new[3, 1],
                                                                             a.max_new[5, 0], a.max_new[5, 1]]
    assert np.array_equal(w.prompt(2), a.prompt_tokens[a.prompt_offsets[5]:a.prompt_offsets[6]])


def test_tail_batched_rollout_rejects_null_engine(lib):
    with pytest.raises(rp.RollpackError) as e:
        rp.rp_rollout_tail_batched(None, np.zeros((2, 2), np.int64), np.arange(4, dtype=np.int32),
                                   np.array([0, 2, 4], np.int64), np.ones((2, 2), np.int32), 0, 1.0, 1, 2, 1.0)
    assert e.value.status == 1


def test_bench_reports_counter_traffic_only_for_the_measured_kernel(tmp_path):
    """roofline.traffic comes from a calibrated counter record and is dropped when the workload
    or kernel differs or the deep kernel's source no longer matches the recorded hash."""
    import json
    import bench
    from paper_2509_21009_amd.counter_traffic import COMMON, SOURCE, deep_source_digest
    rec = {"kernel": "gemm_gate_up", "workload": "7b-long", "source": SOURCE,
           "source_sha256_deep": deep_source_digest(ROOT), "traffic_bytes_per_launch": 123456}
    path = tmp_path / "rec.json"
    path.write_text(json.dumps(rec))
    assert bench.measured_traffic("gemm_gate_up", "7b-long", str(path)) == 123456
    assert bench.measured_traffic("gemm_gate_up", "7b-short", str(path)) is None
    assert bench.measured_traffic("gemm_down", "7b-long", str(path)) is None
    path.write_text(json.dumps(dict(rec, source_sha256_deep="0" * 64)))
    assert bench.measured_traffic("gemm_gate_up", "7b-long", str(path)) is None
    assert bench.measured_traffic("gemm_gate_up", "7b-long", str(tmp_path / "missing.json")) is None
    # the digest covers the deep kernel and its plan, not the rest of the GEMM source
    root = tmp_path / "tree"
    for rel in (SOURCE, COMMON):
        (root / rel).parent.mkdir(parents=True, exist_ok=True)
        (root / rel).write_text(open(os.path.join(ROOT, rel)).read())
    base = deep_source_digest(str(root))
    assert base == deep_source_digest(ROOT)
    gemm = (root / SOURCE).read_text()
    (root / SOURCE).write_text(gemm.replace("constexpr int kGBN = 256", "constexpr int kGBN = 256  /* edit */"))
    assert deep_source_digest(str(root)) == base
    (root / SOURCE).write_text(gemm.replace("const int K = a.K, KU = K / 64;", "const int K = a.K, KU = K / 64;  // edit"))
    assert deep_source_digest(str(root)) != base
    # the committed record names the kernel bench.py reports by default
    committed = json.load(open(bench.TRAFFIC_RECORD))
    assert committed["kernel"] == "gemm_gate_up" and committed["workload"] == "7b-long"
