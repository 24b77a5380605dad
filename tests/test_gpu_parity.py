"""GPU parity: the HIP rollout path through the C ABI vs the CPU oracle.

Bars (written here, from the rollout contract): teacher-forced logits with
max relative error <= 1e-4 (fp32 model) or <= 2e-2 (bf16 model); sampled ids
identical wherever the oracle's top-2 score margin exceeds that tolerance;
greedy agreement >= 99.5% over the positions of the fp32 model and reported
for the others.  Shapes are the paper's Qwen2.5 sizes, truncated in depth
where the fp64 oracle would be too slow; they span several GEMM and KV-page
tiles and ragged tails.
"""
import dataclasses

import numpy as np
import pytest

from tests.gpu_helpers import log, rp, teacher_forced_parity, to_device
from workloads import SHAPES, make_weights, make_workload, truncated, weights_to_numpy
from oracle import model as om

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


def _engine(shape, wdev, max_seqs, max_prefill, max_ctx, pages):
    R = rp()
    return R.Engine(shape, R.weights_for_engine(wdev), max_seqs=max_seqs, max_prefill_tokens=max_prefill,
                    max_context=max_ctx, kv_pages=pages)


@pytest.fixture(scope="module")
def tiny():
    s = SHAPES["tiny"]
    w = make_weights(s, seed=0, device="cpu")
    return s, to_device(w, DEV), weights_to_numpy(w)


def test_tiny_fp32_teacher_forced(tiny):
    s, wd, w64 = tiny
    wl = make_workload("tiny")
    log(f"tiny fp32 teacher-forced: n={wl.n} new=64")
    eng = _engine(s, wd, 8, 256, 128, 32)
    r = teacher_forced_parity(eng, s, w64, wl, 64, 1e-4, 0.0, 0)
    eng.close()
    log(str(r))
    assert r.max_rel_err <= 1e-4, r
    assert r.id_mismatch == 0, r
    assert r.greedy_agree >= 0.995 * r.positions, r


def test_tiny_fp32_free_running_rollout(tiny):
    """rp_rollout_generate greedy tokens equal the oracle's up to the first low-margin position."""
    s, wd, w64 = tiny
    wl = make_workload("tiny")
    eng = _engine(s, wd, 8, 256, 128, 32)
    resp, stats = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, wl.max_new, 0, 0.0)
    eng.close()
    assert stats[0]["generated_tokens"] == 8 * 64 and stats[0]["decode_steps"] == 63
    full_match = 0
    for i in range(wl.n):
        toks, logits = om.generate(w64, s, wl.prompt(i), 64, lambda l, pos: int(np.argmax(l)))
        got = resp[i * 64:(i + 1) * 64]
        for j in range(64):
            srt = np.sort(logits[j])
            if srt[-1] - srt[-2] <= 1e-4 * np.max(np.abs(logits[j])):
                break                                  # a near-tie: later tokens may legitimately differ
            assert got[j] == toks[j], (i, j)
        else:
            full_match += 1
    log(f"free-running: {full_match}/{wl.n} sequences identical over all 64 tokens")


CASES = [
    # name, shape, layers, workload, rows, n_new, temperature
    ("0.5b-L2", "qwen2.5-0.5b", 2, "0.5b", [0, 9, 17, 250], 16, 1.0),
    ("7b-L2", "qwen2.5-7b", 2, "7b-long", [1, 5, 33], 16, 1.0),
    ("32b-L1", "qwen2.5-32b", 1, "32b", [3, 40], 8, 1.0),
]


@pytest.mark.parametrize("name,shape_name,layers,wl_name,rows,n_new,temp", CASES, ids=[c[0] for c in CASES])
def test_bf16_teacher_forced(name, shape_name, layers, wl_name, rows, n_new, temp):
    s = truncated(SHAPES[shape_name], layers)
    log(f"{name}: generating weights on GPU")
    wd = make_weights(s, seed=0, device=DEV)
    w64 = weights_to_numpy(wd)
    wl = make_workload(wl_name, s).subset(rows)
    max_ctx = int(wl.prompt_lens().max()) + n_new + 64
    eng = _engine(s, wd, 8, 4096, max_ctx, 8 * (max_ctx // 64 + 2))
    log(f"{name}: teacher-forced parity, prompts {wl.prompt_lens().tolist()}")
    r = teacher_forced_parity(eng, s, w64, wl, n_new, 2e-2, temp, wl.sample_seed)
    eng.close()
    log(f"{name}: {r}")
    assert r.max_rel_err <= 2e-2, r
    assert r.id_mismatch == 0, r


def test_bf16_against_rounding_oracle():
    """The oracle rounds to bf16 where the kernels store GEMM/attention inputs.  What remains is
    accumulation order and the online softmax (probabilities rounded against each page's running
    maximum instead of the final one), whose small differences flip later bf16 roundings, so the
    logits still differ by a few 1e-3; greedy agreement over 256 positions must reach 99.5%."""
    from oracle import model as om
    s = truncated(SHAPES["qwen2.5-0.5b"], 2)
    wd = make_weights(s, seed=4, device=DEV)
    w64 = weights_to_numpy(wd)
    wl = make_workload("0.5b", s).subset([0, 8, 16, 24, 40, 64, 100, 200])
    max_ctx = int(wl.prompt_lens().max()) + 32 + 64
    eng = _engine(s, wd, 8, 4096, max_ctx, 8 * (max_ctx // 64 + 2))
    r = teacher_forced_parity(eng, s, w64, wl, 32, 1e-2, 0.0, 0, rnd=om.bf16_round)
    eng.close()
    log(f"rounding oracle: {r}")
    assert r.max_rel_err <= 1e-2, r
    assert r.id_mismatch == 0, r
    assert r.greedy_agree >= 0.995 * r.positions, r


@pytest.mark.parametrize("model,layers,vocab,batches", [
    ("qwen2.5-0.5b", 1, 4096, (1, 17, 40, 64, 80)),
    ("qwen2.5-7b", 1, 8192, (2, 24, 40, 64)),
])
def test_bf16_decode_batch_shapes(model, layers, vocab, batches):
    """Decode GEMM regimes by live rows: 1-16, 17-32, 33-48, 49-64 (weight streaming: one
    to four 16-row activation tiles) and 80 (LDS-tiled MFMA).  The 0.5B layer (K = 896 and
    4864) runs the small-matrix kernels; the 7B layer (K = 3584 and 18944, LM head 8192 x 3584)
    runs the deep-pipelined ones with their K splits and ragged last blocks."""
    base = truncated(SHAPES[model], layers, vocab=vocab)
    wd = make_weights(base, seed=1, device=DEV)
    w64 = weights_to_numpy(wd)
    rng = np.random.default_rng(5)
    for B in batches:
        plen = rng.integers(1, 24, size=B)
        prompts = [rng.integers(0, base.vocab, size=int(p)).astype(np.int32) for p in plen]
        offs = np.zeros(B + 1, np.int64)
        offs[1:] = np.cumsum(plen)
        from workloads.gen import Workload
        wl = Workload("batch", base, np.arange(100, 100 + B, dtype=np.int64), np.concatenate(prompts), offs,
                      np.full(B, 3, np.int32), np.arange(B, dtype=np.int32), 1.0, 77)
        eng = _engine(base, wd, 96, 4096, 64, 2 * 96)
        log(f"{model}: decode batch B={B}")
        r = teacher_forced_parity(eng, base, w64, wl, 3, 2e-2, 1.0, 77)
        eng.close()
        log(f"B={B}: {r}")
        assert r.max_rel_err <= 2e-2 and r.id_mismatch == 0, (B, r)


@pytest.mark.parametrize("model,batches", [("qwen2.5-7b", (100, 200, 300)), ("qwen2.5-32b", (160, 300))])
def test_bf16_large_decode_batches(model, batches):
    """Decode batches above 64 rows run the LDS-tiled MFMA GEMM, whose plan picks a block tile
    (128 or 256 activation rows x 128 or 256 weight rows) and a K split per product: at the 7B
    layer 100 and 300 rows take 128-row activation tiles, 200 rows 256-row ones; the 32B layer
    at 160 and 300 rows takes yet other pairs (256 x 128 q/k/v split 4, 256 x 256 down split 12,
    128 x 256 q/k/v and o).  Every row runs on the GPU; three per batch (first, middle, last: the
    ragged last block tile) are compared with the oracle."""
    base = truncated(SHAPES[model], 1, vocab=8192)
    wd = make_weights(base, seed=2, device=DEV)
    w64 = weights_to_numpy(wd)
    rng = np.random.default_rng(6)
    from workloads.gen import Workload
    for B in batches:
        plen = rng.integers(1, 24, size=B)
        prompts = [rng.integers(0, base.vocab, size=int(p)).astype(np.int32) for p in plen]
        offs = np.zeros(B + 1, np.int64)
        offs[1:] = np.cumsum(plen)
        wl = Workload("batch", base, np.arange(1000, 1000 + B, dtype=np.int64), np.concatenate(prompts), offs,
                      np.full(B, 3, np.int32), np.arange(B, dtype=np.int32), 1.0, 78)
        eng = _engine(base, wd, 320, 8192, 64, 2 * 320)
        log(f"{model} layer: decode batch B={B}")
        r = teacher_forced_parity(eng, base, w64, wl, 3, 2e-2, 1.0, 78, check=[0, B // 2, B - 1])
        eng.close()
        log(f"B={B}: {r}")
        assert r.max_rel_err <= 2e-2 and r.id_mismatch == 0, (B, r)


def test_long_context_many_splits():
    """One 4150-token row beside two short ones: its decode context spans 65 pages, so the
    split-context attention runs 65 work items for that row and the merge walks two chunks
    of 64 splits; the short rows are single-split items written without a merge."""
    s = truncated(SHAPES["qwen2.5-0.5b"], 1, vocab=2048)
    s = dataclasses.replace(s, tied=False)
    wd = make_weights(s, seed=6, device=DEV)
    w64 = weights_to_numpy(wd)
    rng = np.random.default_rng(21)
    plen = [4150, 17, 40]
    prompts = [rng.integers(0, s.vocab, size=p).astype(np.int32) for p in plen]
    offs = np.zeros(4, np.int64)
    offs[1:] = np.cumsum(plen)
    from workloads.gen import Workload
    wl = Workload("long", s, np.array([7, 8, 9], np.int64), np.concatenate(prompts), offs,
                  np.full(3, 4, np.int32), np.arange(3, dtype=np.int32), 1.0, 5)
    eng = _engine(s, wd, 4, 4200, 4224, 3 * 67)
    r = teacher_forced_parity(eng, s, w64, wl, 4, 2e-2, 1.0, 5)
    eng.close()
    log(f"long context: {r}")
    assert r.max_rel_err <= 2e-2 and r.id_mismatch == 0, r


@pytest.mark.parametrize("plen,kernel", [
    ([450, 300, 200, 100, 64, 30, 10, 3], "one-wave merge, up to 8 splits"),
    ([3800, 1900, 700, 300, 130, 65, 20, 5], "one-wave merge, up to 64 splits"),
    ([4150, 1900, 700, 300, 130, 65, 20, 5], "1024-thread merge (a row of 65 splits)"),
])
def test_split_merge_kernels_at_eight_rows(plen, kernel):
    """Eight decode rows of one-page to 65-page contexts, one split per page: single-split rows
    are written by the decode kernel, the others are merged, from eight rows up by the one-wave
    kernel while no row has more than 64 splits, else by the 1024-thread kernel.  Three rows
    (the longest, a middle one, a single-split one) are compared with the oracle."""
    s = truncated(SHAPES["qwen2.5-0.5b"], 1, vocab=2048)
    s = dataclasses.replace(s, tied=False)
    wd = make_weights(s, seed=8, device=DEV)
    w64 = weights_to_numpy(wd)
    rng = np.random.default_rng(22)
    prompts = [rng.integers(0, s.vocab, size=p).astype(np.int32) for p in plen]
    offs = np.zeros(len(plen) + 1, np.int64)
    offs[1:] = np.cumsum(plen)
    from workloads.gen import Workload
    n = len(plen)
    wl = Workload("merge", s, np.arange(40, 40 + n, dtype=np.int64), np.concatenate(prompts), offs,
                  np.full(n, 3, np.int32), np.arange(n, dtype=np.int32), 1.0, 6)
    log(f"split merge at 8 rows: {kernel}")
    eng = _engine(s, wd, n, 4200, 4224, n * 67)
    r = teacher_forced_parity(eng, s, w64, wl, 3, 2e-2, 1.0, 6, check=[0, 2, n - 1])
    eng.close()
    log(f"{kernel}: {r}")
    assert r.max_rel_err <= 2e-2 and r.id_mismatch == 0, r


def test_page_boundaries_chunked_prefill_and_short_sequences():
    """Prompts of 1, 63, 64, 65 and 130 tokens, max_new 1 and 70 (decode crosses pages),
    prefill split into chunks of at most 140 tokens."""
    s = truncated(SHAPES["qwen2.5-0.5b"], 1, vocab=2048)
    s = dataclasses.replace(s, tied=False)
    wd = make_weights(s, seed=2, device=DEV)
    w64 = weights_to_numpy(wd)
    rng = np.random.default_rng(9)
    plen = [1, 63, 64, 65, 130]
    prompts = [rng.integers(0, s.vocab, size=p).astype(np.int32) for p in plen]
    offs = np.zeros(6, np.int64)
    offs[1:] = np.cumsum(plen)
    from workloads.gen import Workload
    wl = Workload("pages", s, np.arange(5, dtype=np.int64) + 1000, np.concatenate(prompts), offs,
                  np.full(5, 70, np.int32), np.arange(5, dtype=np.int32), 0.0, 0)
    eng = _engine(s, wd, 8, 140, 256, 40)
    r = teacher_forced_parity(eng, s, w64, wl, 70, 2e-2, 0.0, 0)
    log(f"pages: {r}")
    assert r.max_rel_err <= 2e-2 and r.id_mismatch == 0, r
    # max_new = 1: the prefill token is the whole response
    resp, st = eng.rollout(np.array([7, 8], np.int64), np.concatenate(prompts[:2]), offs[:3], np.array([1, 1], np.int32),
                           0, 0.0)
    eng.close()
    for i in range(2):
        ref = int(np.argmax(om.forward_full(w64, s, prompts[i])[-1]))
        assert resp[i] == ref
    assert st[0]["decode_steps"] == 0


def test_rollout_is_deterministic_and_frees_pages(tiny):
    s, wd, _ = tiny
    wl = make_workload("tiny")
    mn = np.array([5, 64, 1, 30, 64, 2, 17, 40], np.int32)
    eng = _engine(s, wd, 8, 256, 128, 32)
    a, sa = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, mn, 3, 1.0)
    b, sb = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, mn, 3, 1.0)
    eng.close()
    assert np.array_equal(a, b)
    assert sa[0]["decode_steps"] == 63 and sa[0]["generated_tokens"] == int(mn.sum())
    assert 0.0 < sa[0]["slot_idle"] < 1.0


def test_engine_errors_leave_state_unchanged(tiny):
    s, wd, _ = tiny
    R = rp()
    eng = _engine(s, wd, 4, 64, 128, 3)
    p = np.arange(10, dtype=np.int32)
    eng.prefill(np.array([1], np.int64), p, np.array([0, 10], np.int64), np.array([20], np.int32))
    with pytest.raises(R.RollpackError) as e:
        eng.prefill(np.array([1], np.int64), p, np.array([0, 10], np.int64), np.array([20], np.int32))
    assert e.value.status == 3                                # duplicate id
    with pytest.raises(R.RollpackError) as e:                 # 10 + 120 - 1 > 128 context
        eng.prefill(np.array([2], np.int64), p, np.array([0, 10], np.int64), np.array([120], np.int32))
    assert e.value.status == 7
    with pytest.raises(R.RollpackError) as e:                 # 2 x 2 pages wanted, 2 of 3 free
        eng.prefill(np.array([2, 3], np.int64), np.concatenate([p, p]), np.array([0, 10, 20], np.int64),
                    np.array([60, 60], np.int32))
    assert e.value.status == 2
    with pytest.raises(R.RollpackError) as e:
        eng.abort(np.array([99], np.int64))
    assert e.value.status == 4
    n, rows, _ = eng.decode_step()
    assert n == 1 and rows.tolist() == [1]
    eng.abort(np.array([1], np.int64))
    assert eng.decode_step()[0] == 0
    eng.prefill(np.array([2, 3], np.int64), np.concatenate([p, p]), np.array([0, 10, 20], np.int64),
                np.array([50, 50], np.int32))                 # the pages came back
    eng.close()


def test_profile_sampling(tiny):
    """rp_profile_every: one launch in N of a class is timed, from the first, per phase."""
    s, wd, _ = tiny
    R = rp()
    wl = make_workload("tiny")
    counts = {}
    for every in (1, 3):
        eng = _engine(s, wd, 8, 256, 128, 32)
        eng.profile(["attn", "gemm_gate_up", "sample"], every=every)
        toks, _ = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, wl.max_new, 0, 0.0)
        counts[every] = {(r["kernel"], r["phase"]): r for r in eng.profile_read()}
        counts[every]["toks"] = toks
        with pytest.raises(R.RollpackError):
            eng.profile(["attn"], every=0)
        eng.close()
    assert np.array_equal(counts[1]["toks"], counts[3]["toks"])
    # sampling launches two kernels: its events run from the first one's start to the last one's end
    for key in [("attn", "decode"), ("gemm_gate_up", "decode"), ("gemm_gate_up", "prefill"), ("sample", "decode")]:
        full, part = counts[1][key], counts[3][key]
        assert part["launches"] == (full["launches"] + 2) // 3, key
        assert part["total_ms"] > 0 and part["bytes"] > 0


def test_stream_read_ceiling():
    """rp_stream_read_gbs: a read-only streaming pass over a 1 GiB buffer reports a plausible HBM
    rate, leaves the buffer unchanged, and rejects buffers under 1 MiB."""
    R = rp()
    x = torch.arange(1 << 28, dtype=torch.int32, device=DEV)
    before = int(x[::4096].sum().item())
    gbs = R.rp_stream_read_gbs(x, 3)
    log(f"stream read: {gbs:.0f} GB/s")
    assert 1000.0 < gbs < 8000.0
    assert int(x[::4096].sum().item()) == before
    with pytest.raises(R.RollpackError):
        R.rp_stream_read_gbs(torch.zeros(1024, dtype=torch.int32, device=DEV), 1)



def test_packed_weights_give_identical_logits():
    """The decode GEMMs read a packed copy of the weights when the engine has one
    (rp_engine_set_packed_weights); every lane loads the same MFMA operand as from the
    row-major matrix, so prefill and teacher-forced decode logits must be bitwise equal with
    and without it, over the deep kernel's regimes (1-4 activation tiles, K-split down and
    q/k/v projections, a ragged LM head of 8,320 rows) at the 7B layer shape."""
    R = rp()
    s = truncated(SHAPES["qwen2.5-7b"], 2, vocab=8320)
    wd = make_weights(s, seed=2, device=DEV)
    rng = np.random.default_rng(9)
    for B in (1, 17, 40, 64):
        plen = rng.integers(1, 40, size=B)
        toks = rng.integers(0, s.vocab, size=int(plen.sum())).astype(np.int32)
        offs = np.concatenate([[0], np.cumsum(plen)]).astype(np.int64)
        ids = np.arange(10, 10 + B, dtype=np.int64)
        forced = rng.integers(0, s.vocab, size=(3, B)).astype(np.int32)
        out = []
        for pack in (True, False):
            eng = R.Engine(s, R.weights_for_engine(wd), max_seqs=64, max_prefill_tokens=4096, max_context=64,
                           kv_pages=2 * 64, pack_weights=pack)
            assert (eng.packed is not None) == pack
            lg0, _ = eng.prefill(ids, toks, offs, np.full(B, 4, np.int32), 3, 1.0, logits=True)
            rows = [lg0.cpu().numpy()]
            for j in range(3):
                _, _, lg = eng.decode_step(forced_tokens=forced[j], logits=True)
                rows.append(lg.cpu().numpy())
            out.append(np.stack(rows))
            eng.close()
        log(f"packed vs row-major weights, B={B}: identical={np.array_equal(out[0], out[1])}")
        assert np.array_equal(out[0], out[1]), B
