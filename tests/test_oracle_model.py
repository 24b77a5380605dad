"""Pins of the decoder oracle against things other than itself (CPU only).

* an installed library: transformers' Qwen2 causal LM with the same weights;
* brute force: full causal recompute vs incremental KV-cache decoding;
* closed forms and invariants: RoPE is a rotation (norm kept, identity at
  position 0, the 2-D rotation matrix for hd = 2), softmax rows sum to 1,
  RMSNorm output has unit RMS, single-key attention returns V, uniform
  scores return the mean of V, and GQA equals MHA with K/V heads repeated
  per group (consecutive grouping).
"""
import numpy as np
import pytest
import torch

from oracle import model as om
from oracle import sampling as osm
from workloads import SHAPES, make_weights, make_workload, truncated, weights_to_numpy


@pytest.fixture(scope="module")
def tiny():
    s = SHAPES["tiny"]
    return s, weights_to_numpy(make_weights(s, seed=0))


def _hf_model(shape, w64):
    from transformers import Qwen2Config, Qwen2ForCausalLM
    cfg = Qwen2Config(hidden_size=shape.hidden, intermediate_size=shape.inter,
                      num_attention_heads=shape.n_q, num_key_value_heads=shape.n_kv,
                      num_hidden_layers=shape.layers, vocab_size=shape.vocab,
                      rms_norm_eps=shape.eps, rope_theta=shape.theta,
                      tie_word_embeddings=shape.tied, max_position_embeddings=4096,
                      attn_implementation="eager")
    m = Qwen2ForCausalLM(cfg).double().eval()
    sd = {"model.embed_tokens.weight": w64["embed"], "model.norm.weight": w64["final_norm"]}
    for l, L in enumerate(w64["layers"]):
        p = f"model.layers.{l}."
        sd.update({p + "input_layernorm.weight": L["attn_norm"],
                   p + "post_attention_layernorm.weight": L["mlp_norm"],
                   p + "self_attn.q_proj.weight": L["wq"], p + "self_attn.q_proj.bias": L["bq"],
                   p + "self_attn.k_proj.weight": L["wk"], p + "self_attn.k_proj.bias": L["bk"],
                   p + "self_attn.v_proj.weight": L["wv"], p + "self_attn.v_proj.bias": L["bv"],
                   p + "self_attn.o_proj.weight": L["wo"],
                   p + "mlp.gate_proj.weight": L["w_gate"], p + "mlp.up_proj.weight": L["w_up"],
                   p + "mlp.down_proj.weight": L["w_down"]})
    sd["lm_head.weight"] = w64["embed"] if shape.tied else w64["lm_head"]
    sd = {k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in sd.items()}
    missing, unexpected = m.load_state_dict(sd, strict=False)
    assert not unexpected, unexpected
    assert all("rotary" in k for k in missing), missing
    return m


@pytest.mark.parametrize("tied,n_kv", [(False, 2), (True, 1), (False, 4)])
def test_forward_matches_transformers_qwen2(tied, n_kv):
    """The whole forward (bias, GQA map, RoPE pairing/theta, tying) against transformers."""
    import dataclasses
    s = dataclasses.replace(SHAPES["tiny"], tied=tied, n_kv=n_kv, vocab=512)
    w = weights_to_numpy(make_weights(s, seed=3))
    rng = np.random.default_rng(7)
    toks = rng.integers(0, s.vocab, size=48)
    ours = om.forward_full(w, s, toks)
    with torch.no_grad():
        ref = _hf_model(s, w)(torch.from_numpy(toks)[None]).logits[0].numpy()
    # transformers computes RoPE angles in fp32: ~1e-7 * position radians of error.
    err = np.max(np.abs(ours - ref)) / np.max(np.abs(ref))
    assert err < 2e-5, err


def test_incremental_equals_full_recompute(tiny):
    s, w = tiny
    wl = make_workload("tiny")
    prompt = wl.prompt(0)
    toks, rows = om.generate(w, s, prompt, 12, lambda l, pos: int(np.argmax(l)))
    full = om.forward_full(w, s, np.concatenate([prompt, toks[:-1]]))[len(prompt) - 1:]
    assert np.max(np.abs(full - rows)) / np.max(np.abs(full)) < 1e-12
    assert np.array_equal(np.argmax(full, axis=-1), toks)
    tf = om.teacher_forced_logits(w, s, prompt, toks)
    assert np.max(np.abs(tf - rows)) < 1e-12


def test_chunked_incremental_equals_full(tiny):
    s, w = tiny
    rng = np.random.default_rng(1)
    toks = rng.integers(0, s.vocab, size=40)
    st = om.KVState(s)
    parts = [st.step(w, toks[:17]), st.step(w, toks[17:18]), st.step(w, toks[18:])]
    inc = np.concatenate(parts)
    full = om.forward_full(w, s, toks)
    assert np.max(np.abs(inc - full)) < 1e-12


def test_rope_is_a_rotation():
    rng = np.random.default_rng(0)
    u = rng.standard_normal((50, 3, 128))
    pos = rng.integers(0, 20000, size=50)
    cos, sin = om.rope_cos_sin(pos, 128, 1e6)
    r = om.apply_rope(u, cos, sin)
    assert np.allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(u, axis=-1), rtol=1e-13)
    c0, s0 = om.rope_cos_sin(np.zeros(50), 128, 1e6)
    assert np.array_equal(om.apply_rope(u, c0, s0), u)
    # hd = 2: one pair rotated by angle = pos (frequency theta^0 = 1)
    v = rng.standard_normal((4, 1, 2))
    p = np.array([0.0, 1.0, 2.5, 7.0])
    c, s_ = om.rope_cos_sin(p, 2, 1e6)
    rot = om.apply_rope(v, c, s_)
    for i, a in enumerate(p):
        m = np.array([[np.cos(a), -np.sin(a)], [np.sin(a), np.cos(a)]])
        assert np.allclose(rot[i, 0], m @ v[i, 0], atol=1e-14)
    # relative property: <R(m)q, R(n)k> depends only on m - n
    q, k = rng.standard_normal((1, 1, 64)), rng.standard_normal((1, 1, 64))
    def dot(m, n):
        cm, sm = om.rope_cos_sin([m], 64, 1e4)
        cn, sn = om.rope_cos_sin([n], 64, 1e4)
        return float(np.sum(om.apply_rope(q, cm, sm) * om.apply_rope(k, cn, sn)))
    assert abs(dot(10, 3) - dot(107, 100)) < 1e-10


def test_softmax_rows_sum_to_one():
    rng = np.random.default_rng(2)
    s = rng.standard_normal((20, 300)) * 30
    assert np.allclose(om.softmax(s).sum(-1), 1.0, atol=1e-12)


def test_rmsnorm_unit_rms():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 256)) * 7 + 3
    y = om.rmsnorm(x, np.ones(256), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, -1)), 1.0, atol=1e-13)
    g = rng.standard_normal(256)
    assert np.allclose(om.rmsnorm(x, g, 0.0), y * g)


def test_silu_limits():
    assert om.silu(np.array(0.0)) == 0.0
    assert abs(om.silu(np.array(40.0)) - 40.0) < 1e-12
    assert abs(om.silu(np.array(-40.0))) < 1e-12
    from scipy.special import expit
    z = np.linspace(-8, 8, 101)
    assert np.allclose(om.silu(z), z * expit(z), atol=1e-15)


def test_attention_special_cases():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((1, 4, 16))
    k = rng.standard_normal((1, 2, 16))
    v = rng.standard_normal((1, 2, 16))
    out = om.attention(q, k, v, np.array([0]), np.array([0]))
    assert np.allclose(out[0], v[0][[0, 0, 1, 1]])           # single key returns V
    k5, v5 = rng.standard_normal((5, 2, 16)), rng.standard_normal((5, 2, 16))
    out = om.attention(np.zeros((1, 4, 16)), k5, v5, np.array([4]), np.arange(5))
    assert np.allclose(out[0, 3], v5[:, 1].mean(0))           # uniform scores: mean of V
    out = om.attention(np.zeros((1, 4, 16)), k5, v5, np.array([2]), np.arange(5))
    assert np.allclose(out[0, 0], v5[:3, 0].mean(0))          # causal: keys 0..2 only


def test_gqa_equals_mha_with_repeated_heads(tiny):
    """Query head h reads KV head h // group: repeat K/V weights per group -> MHA."""
    import dataclasses
    s, w = tiny
    g = s.group
    mha = dataclasses.replace(s, n_kv=s.n_q)
    w2 = {"embed": w["embed"], "final_norm": w["final_norm"], "lm_head": w["lm_head"], "layers": []}
    hd = s.head_dim
    for L in w["layers"]:
        L2 = dict(L)
        for t in ("wk", "wv"):
            L2[t] = np.repeat(L[t].reshape(s.n_kv, hd, -1), g, axis=0).reshape(s.n_q * hd, -1)
        for t in ("bk", "bv"):
            L2[t] = np.repeat(L[t].reshape(s.n_kv, hd), g, axis=0).reshape(-1)
        w2["layers"].append(L2)
    toks = np.random.default_rng(5).integers(0, s.vocab, size=20)
    assert np.allclose(om.forward_full(w, s, toks), om.forward_full(w2, mha, toks), atol=1e-12)


def test_generate_with_sampler_is_reproducible(tiny):
    s, w = tiny
    prompt = make_workload("tiny").prompt(1)
    a, _ = om.generate(w, s, prompt, 6, osm.sampler(1.0, 9, 3))
    b, _ = om.generate(w, s, prompt, 6, osm.sampler(1.0, 9, 3))
    c, _ = om.generate(w, s, prompt, 6, osm.sampler(1.0, 9, 4))
    assert np.array_equal(a, b) and not np.array_equal(a, c)


def test_bf16_round_matches_torch():
    """The diagnostic rounding equals torch's fp32 -> bfloat16 conversion (round to nearest even)."""
    rng = np.random.default_rng(11)
    x = np.concatenate([rng.standard_normal(10000) * 10.0 ** rng.integers(-6, 6, 10000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38, -2.5e-38]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(om.bf16_round(x), ref)


def test_rounding_diagnostic_reduces_to_plain_oracle(tiny):
    """rnd=None and rnd=identity give the plain fp64 forward; bf16 rounding stays close to it."""
    s, w = tiny
    toks = np.random.default_rng(12).integers(0, s.vocab, size=30)
    plain = om.forward_full(w, s, toks)
    ident = om.forward_full(w, s, toks, rnd=lambda v: v)      # same maths, P normalised after P @ V
    assert np.max(np.abs(ident - plain)) < 1e-12
    rounded = om.forward_full(w, s, toks, rnd=om.bf16_round)
    err = np.max(np.abs(rounded - plain)) / np.max(np.abs(plain))
    assert 1e-6 < err < 5e-2
    st = om.KVState(s, om.bf16_round)
    inc = np.concatenate([st.step(w, toks[:20]), st.step(w, toks[20:21]), st.step(w, toks[21:])])
    assert np.max(np.abs(inc - rounded)) < 1e-10


def test_truncated_shape_keeps_layer_dims():
    s = truncated(SHAPES["qwen2.5-7b"], 2)
    assert s.layers == 2 and s.hidden == 3584 and s.group == 7


def test_batched_decode_step_equals_per_sequence_steps(tiny):
    """decode_step_batch against brute force: each row recomputed from scratch
    over its whole sequence (prompts of different lengths, so rows sit at
    different positions and attend to different cache lengths)."""
    s, w = tiny
    rng = np.random.default_rng(11)
    prompts = [rng.integers(0, s.vocab, size=n) for n in (5, 17, 33, 1)]
    states = [om.KVState(s) for _ in prompts]
    for st, p in zip(states, prompts):
        st.step(w, p)
    seqs = [list(p) for p in prompts]
    for _ in range(3):
        nxt = rng.integers(0, s.vocab, size=len(prompts))
        got = om.decode_step_batch(w, states, nxt)
        for b in range(len(prompts)):
            seqs[b].append(int(nxt[b]))
            ref = om.forward_full(w, s, np.array(seqs[b]))[-1]
            assert np.max(np.abs(got[b] - ref)) / np.max(np.abs(ref)) < 1e-12
    assert [st.length for st in states] == [len(q) for q in seqs]
