"""Whole-step pins of the oracle (CPU only).

The oracle's incremental paged decode, fed one token at a time from an empty
cache, must reproduce the logits of an independent full-sequence causal
forward of the same architecture in the ``transformers`` library (Qwen3:
RMSNorm, per-head QK-RMSNorm, rotate-half RoPE, GQA, SwiGLU) -- a library
special case that exercises every layer step, the KV append slots and the
RoPE positions.  Further invariants: page-permutation invariance of a whole
step, the zero-block special case and determinism.
"""
import contextlib

import numpy as np
import pytest
import torch

from oracle import decoder as od
from oracle.bf16 import round_bf16
from paper_2604_07725_amd.synth import ModelShape

SHAPE = ModelShape(n_layers=2, hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=32, ffn=96,
                   vocab=97, rope_theta=1.0e4)


def _weights(shape, rng, scale=0.2):
    H, F, V = shape.hidden, shape.ffn, shape.vocab
    layers = []
    for _ in range(shape.n_layers):
        layers.append({
            "attn_norm": 1 + 0.1 * rng.standard_normal(H),
            "w_qkv": scale * rng.standard_normal((shape.qkv_dim, H)),
            "q_norm": 1 + 0.1 * rng.standard_normal(shape.head_dim),
            "k_norm": 1 + 0.1 * rng.standard_normal(shape.head_dim),
            "w_o": scale * rng.standard_normal((H, shape.q_dim)),
            "ffn_norm": 1 + 0.1 * rng.standard_normal(H),
            "w_gate_up": scale * rng.standard_normal((2 * F, H)),
            "w_down": scale * rng.standard_normal((H, F)),
        })
    return {"embed": rng.standard_normal((V, H)), "lm_head": scale * rng.standard_normal((V, H)),
            "final_norm": 1 + 0.1 * rng.standard_normal(H), "layers": layers}


def _hf_model(shape, w):
    from transformers import Qwen3Config, Qwen3ForCausalLM
    cfg = Qwen3Config(vocab_size=shape.vocab, hidden_size=shape.hidden,
                      intermediate_size=shape.ffn, num_hidden_layers=shape.n_layers,
                      num_attention_heads=shape.n_q_heads, num_key_value_heads=shape.n_kv_heads,
                      head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
                      rope_parameters={"rope_theta": shape.rope_theta, "rope_type": "default"},
                      max_position_embeddings=256, tie_word_embeddings=False,
                      attention_bias=False, hidden_act="silu")
    cfg._attn_implementation = "eager"
    m = Qwen3ForCausalLM(cfg).to(torch.float64).eval()
    T = lambda a: torch.from_numpy(np.asarray(a, np.float64))  # noqa: E731
    qd, kd = shape.q_dim, shape.kv_dim
    F = shape.ffn
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(T(w["embed"]))
        m.lm_head.weight.copy_(T(w["lm_head"]))
        m.model.norm.weight.copy_(T(w["final_norm"]))
        for l, lw in enumerate(w["layers"]):
            layer = m.model.layers[l]
            layer.input_layernorm.weight.copy_(T(lw["attn_norm"]))
            layer.post_attention_layernorm.weight.copy_(T(lw["ffn_norm"]))
            a = layer.self_attn
            a.q_proj.weight.copy_(T(lw["w_qkv"][:qd]))
            a.k_proj.weight.copy_(T(lw["w_qkv"][qd:qd + kd]))
            a.v_proj.weight.copy_(T(lw["w_qkv"][qd + kd:]))
            a.o_proj.weight.copy_(T(lw["w_o"]))
            a.q_norm.weight.copy_(T(lw["q_norm"]))
            a.k_norm.weight.copy_(T(lw["k_norm"]))
            layer.mlp.gate_proj.weight.copy_(T(lw["w_gate_up"][:F]))
            layer.mlp.up_proj.weight.copy_(T(lw["w_gate_up"][F:]))
            layer.mlp.down_proj.weight.copy_(T(lw["w_down"]))
    return m


def _empty_pools(shape, n_pages):
    return [np.zeros((n_pages, shape.n_kv_heads, 2, 16 * shape.head_dim))
            for _ in range(shape.n_layers)]


def test_incremental_paged_decode_equals_transformers_causal_forward():
    rng = np.random.default_rng(7)
    w = _weights(SHAPE, rng)
    N, T = 2, 37                      # crosses two page boundaries
    seqs = rng.integers(0, SHAPE.vocab, size=(N, T))
    pages_per = (T + 15) // 16
    perm = rng.permutation(N * pages_per)
    pt = perm.reshape(N, pages_per)
    kvp = _empty_pools(SHAPE, N * pages_per)
    oracle_logits = np.empty((N, T, SHAPE.vocab))
    for t in range(T):
        out = od.decode_step(SHAPE, w, kvp, pt, seqs[:, t], np.full(N, t), np.arange(N),
                             seed=1, temperature=1.0, mirror=False)
        oracle_logits[:, t] = out["logits"]
    m = _hf_model(SHAPE, w)
    with torch.no_grad():
        ref = m(input_ids=torch.from_numpy(seqs)).logits.numpy()
    # transformers keeps its RMSNorm and RoPE tables in float32; the bound
    # covers that, while any structural slip gives O(0.1) differences
    err = np.abs(oracle_logits - ref).max()
    assert err < 2e-5 * np.abs(ref).max(), err


def test_whole_step_invariant_under_page_permutation_and_deterministic():
    rng = np.random.default_rng(8)
    w = _weights(SHAPE, rng)
    N = 3
    lens = np.array([5, 33, 20])
    need = (lens + 1 + 15) // 16
    P = int(need.sum())
    kvp = [rng.standard_normal((P, 2, 2, 16 * 32)) for _ in range(2)]
    pt = np.full((N, need.max()), -1)
    c = 0
    for i in range(N):
        pt[i, :need[i]] = np.arange(c, c + need[i])
        c += need[i]
    perm = rng.permutation(P)
    kvp2 = []
    for l in range(2):
        a = np.empty_like(kvp[l]); a[perm] = kvp[l]; kvp2.append(a)
    pt2 = np.where(pt >= 0, perm[np.maximum(pt, 0)], -1)
    toks = np.array([1, 50, 96])
    args = dict(tokens=toks, positions=lens, uids=np.array([10, 11, 12]), seed=3, temperature=1.0)
    a = od.decode_step(SHAPE, w, [k.copy() for k in kvp], pt, **args)
    b = od.decode_step(SHAPE, w, kvp2, pt2, **args)
    c2 = od.decode_step(SHAPE, w, [k.copy() for k in kvp], pt, **args)
    np.testing.assert_array_equal(a["logits"], b["logits"])
    np.testing.assert_array_equal(a["ids"], b["ids"])
    np.testing.assert_array_equal(a["logits"], c2["logits"])


def test_zero_blocks_reduce_to_embedding_head():
    """With W_o = 0 and W_down = 0 each layer leaves x unchanged, so the logits
    are RMSNorm(E[t]) * g_final . W_lm^T, whatever the KV cache holds."""
    rng = np.random.default_rng(9)
    w = _weights(SHAPE, rng)
    for lw in w["layers"]:
        lw["w_o"] = np.zeros_like(lw["w_o"])
        lw["w_down"] = np.zeros_like(lw["w_down"])
    kvp = _empty_pools(SHAPE, 4)
    for k in kvp:
        k[:] = rng.standard_normal(k.shape)
    pt = np.array([[0, 1], [2, 3]])
    toks = np.array([3, 40])
    out = od.decode_step(SHAPE, w, kvp, pt, toks, np.array([20, 7]), np.array([0, 1]), 0, 1.0,
                         mirror=False)
    x = w["embed"][toks]
    hf = x / np.sqrt((x * x).mean(-1, keepdims=True) + SHAPE.rms_eps) * w["final_norm"]
    np.testing.assert_allclose(out["logits"], hf @ w["lm_head"].T, rtol=1e-12, atol=1e-12)


def test_mirror_rounds_only_storage_points():
    """mirror=True differs from the pure definition only by bf16 storage rounding:
    small but non-zero relative change of the logits."""
    rng = np.random.default_rng(10)
    w = _weights(SHAPE, rng)
    kvp = _empty_pools(SHAPE, 4)
    for k in kvp:
        k[:] = rng.standard_normal(k.shape)
    pt = np.array([[0, 1], [2, 3]])
    args = dict(tokens=np.array([3, 40]), positions=np.array([20, 7]), uids=np.array([0, 1]),
                seed=0, temperature=1.0)
    a = od.decode_step(SHAPE, w, [k.copy() for k in kvp], pt, mirror=False, **args)
    b = od.decode_step(SHAPE, w, [k.copy() for k in kvp], pt, mirror=True, **args)
    rel = np.abs(a["logits"] - b["logits"]).max() / np.abs(a["logits"]).max()
    assert 1e-5 < rel < 5e-2, rel


# ------------------------------------------------------------------ bf16 storage points
# The GPU path stores h, q and k (after RoPE), v, the attention output o, h2,
# the SwiGLU product a and the final normed row in bf16, keeps the residual
# stream and the logits in fp32, and computes everything else in fp32; the
# oracle's mirror mode rounds at exactly those points.  The pin: the
# transformers Qwen3 causal forward, run in float64 throughout (torch's
# library rms_norm for every norm, a float64 RoPE table, SDPA attention) with
# rounding hooks at those points only, must give the oracle's logits exactly,
# while leaving out any single bf16 point moves them by ~1e-3.
STORAGE_POINTS = ("h", "qk", "v", "o", "h2", "a", "hf", "x32", "logits32")


def _bf16_t(t):
    return t.to(torch.bfloat16).to(torch.float64)


def _f32_t(t):
    return t.to(torch.float32).to(torch.float64)


@contextlib.contextmanager
def _float64_with_storage_rounding(m, shape, points):
    import torch.nn.functional as Fn
    import transformers.models.qwen3.modeling_qwen3 as mq
    hooks, saved = [], []
    norms = [m.model.norm] + [n for l in m.model.layers for n in
                              (l.input_layernorm, l.post_attention_layernorm,
                               l.self_attn.q_norm, l.self_attn.k_norm)]
    for n in norms:          # the library norm in float64 instead of its fp32 path
        saved.append((n, n.forward))
        n.forward = lambda x, n=n: Fn.rms_norm(x, (x.shape[-1],), n.weight, n.variance_epsilon)
    rot = m.model.rotary_emb
    old_inv, old_float, old_rope = rot.inv_freq, torch.Tensor.float, mq.apply_rotary_pos_emb
    d = shape.head_dim
    rot.inv_freq = 1.0 / (shape.rope_theta ** (torch.arange(0, d, 2, dtype=torch.float64) / d))
    torch.Tensor.float = lambda self: self.to(torch.float64)   # its cos / sin in float64
    impl = m.config._attn_implementation
    m.config._attn_implementation = "sdpa"                     # float64 softmax
    if "qk" in points:
        def rope(q, k, cos, sin, *a, **kw):
            qe, ke = old_rope(q, k, cos, sin, *a, **kw)
            return _bf16_t(qe), _bf16_t(ke)
        mq.apply_rotary_pos_emb = rope
    out_hook = lambda mod, inp, out: _bf16_t(out)                          # noqa: E731
    in_hook = lambda mod, inp: (_bf16_t(inp[0]),) + tuple(inp[1:])        # noqa: E731
    for layer in m.model.layers:
        res = {}
        keep = lambda mod, inp, res=res: res.__setitem__("x", inp[0])     # noqa: E731
        # fp32 residual: a branch output b becomes f32(x + b) - x (exact in
        # float64), so the layer's own x + b is f32(x + b)
        fix = lambda mod, inp, out, res=res: _f32_t(res["x"] + out) - res["x"]  # noqa: E731
        if "x32" in points:
            hooks += [layer.input_layernorm.register_forward_pre_hook(keep),
                      layer.post_attention_layernorm.register_forward_pre_hook(keep)]
        if "h" in points:
            hooks.append(layer.input_layernorm.register_forward_hook(out_hook))
        if "v" in points:
            hooks.append(layer.self_attn.v_proj.register_forward_hook(out_hook))
        if "o" in points:
            hooks.append(layer.self_attn.o_proj.register_forward_pre_hook(in_hook))
        if "x32" in points:
            hooks.append(layer.self_attn.o_proj.register_forward_hook(fix))
        if "h2" in points:
            hooks.append(layer.post_attention_layernorm.register_forward_hook(out_hook))
        if "a" in points:
            hooks.append(layer.mlp.down_proj.register_forward_pre_hook(in_hook))
        if "x32" in points:
            hooks.append(layer.mlp.down_proj.register_forward_hook(fix))
    if "hf" in points:
        hooks.append(m.model.norm.register_forward_hook(out_hook))
    if "logits32" in points:
        hooks.append(m.lm_head.register_forward_hook(lambda mod, inp, out: _f32_t(out)))
    try:
        yield
    finally:
        for h in hooks:
            h.remove()
        for n, f in saved:
            n.forward = f
        rot.inv_freq = old_inv
        torch.Tensor.float = old_float
        mq.apply_rotary_pos_emb = old_rope
        m.config._attn_implementation = impl


def _hf64_logits(m, shape, seqs, points):
    with _float64_with_storage_rounding(m, shape, points), torch.no_grad():
        return m(input_ids=torch.from_numpy(np.asarray(seqs))).logits.numpy()


def _bf16_weights(shape, rng):
    w = _weights(shape, rng)
    return {k: ([{kk: round_bf16(vv) for kk, vv in lw.items()} for lw in v] if k == "layers"
                else round_bf16(v)) for k, v in w.items()}


@pytest.mark.parametrize("seed", [0, 1])
def test_mirror_storage_points_equal_transformers_with_bf16_hooks(seed):
    """The oracle's mirrored decode (token by token from an empty paged cache)
    equals the hooked float64 transformers forward exactly; without any one of
    its bf16 points (or the fp32 logits) the forward differs, so every point
    is in the oracle, and none is added elsewhere."""
    rng = np.random.default_rng(100 + seed)
    w = _bf16_weights(SHAPE, rng)
    N, T = 2, 37
    seqs = rng.integers(0, SHAPE.vocab, size=(N, T))
    pt = rng.permutation(N * 3).reshape(N, 3)
    kvp = _empty_pools(SHAPE, N * 3)
    oracle_logits = np.empty((N, T, SHAPE.vocab))
    for t in range(T):
        out = od.decode_step(SHAPE, w, kvp, pt, seqs[:, t], np.full(N, t), np.arange(N),
                             seed=1, temperature=1.0, mirror=True)
        oracle_logits[:, t] = out["logits"]
    m = _hf_model(SHAPE, w)
    scale = np.abs(oracle_logits).max()
    err = np.abs(_hf64_logits(m, SHAPE, seqs, STORAGE_POINTS) - oracle_logits).max() / scale
    assert err <= 1e-12, err
    for p in STORAGE_POINTS:
        if p == "x32":
            continue    # below the fp32 logits' resolution at this size (no flip it decides)
        off = np.abs(_hf64_logits(m, SHAPE, seqs, [q for q in STORAGE_POINTS if q != p])
                      - oracle_logits).max() / scale
        assert off > (1e-9 if p == "logits32" else 1e-4), (p, off)
    # and the pure definition: no rounding anywhere equals mirror=False exactly
    kvp = _empty_pools(SHAPE, N * 3)
    pure = np.empty_like(oracle_logits)
    for t in range(T):
        pure[:, t] = od.decode_step(SHAPE, w, kvp, pt, seqs[:, t], np.full(N, t), np.arange(N),
                                    seed=1, temperature=1.0, mirror=False)["logits"]
    err = np.abs(_hf64_logits(m, SHAPE, seqs, ()) - pure).max() / scale
    assert err <= 1e-12, err


def test_prefill_mirror_storage_points_equal_transformers_with_bf16_hooks():
    """The same pin for the prefill (every token of two sequences through each
    layer at once, the confidence engine's forward)."""
    rng = np.random.default_rng(21)
    w = _bf16_weights(SHAPE, rng)
    lens = [37, 20]
    seqs = [rng.integers(0, SHAPE.vocab, size=n) for n in lens]
    starts = np.array([0, lens[0], lens[0] + lens[1]])
    pt = np.array([[3, 0, 4], [1, 2, -1]])
    x = od.prefill_forward(SHAPE, w, _empty_pools(SHAPE, 5), pt, np.concatenate(seqs), starts,
                           mirror=True)
    logits = od.lm_logits(SHAPE, w["final_norm"], w["lm_head"], x, mirror=True)
    m = _hf_model(SHAPE, w)
    for s in range(2):
        ref = _hf64_logits(m, SHAPE, seqs[s][None], STORAGE_POINTS)[0]
        err = np.abs(logits[starts[s]:starts[s + 1]] - ref).max() / np.abs(ref).max()
        assert err <= 1e-12, (s, err)


# ------------------------------------------------------------------ prefill (confidence engine)
def test_prefill_forward_equals_transformers_and_incremental_decode():
    """The batched prefill (two sequences back to back, every token through the
    layer at once) reproduces the transformers causal forward's logits of each
    sequence, and the oracle's own token-by-token decode."""
    rng = np.random.default_rng(11)
    w = _weights(SHAPE, rng)
    lens = [37, 20]
    seqs = [rng.integers(0, SHAPE.vocab, size=n) for n in lens]
    starts = np.array([0, lens[0], lens[0] + lens[1]])
    need = [(n + 15) // 16 for n in lens]
    perm = rng.permutation(sum(need))
    pt = np.full((2, max(need)), -1)
    pt[0, :need[0]] = perm[:need[0]]
    pt[1, :need[1]] = perm[need[0]:]
    kvp = _empty_pools(SHAPE, sum(need))
    x = od.prefill_forward(SHAPE, w, kvp, pt, np.concatenate(seqs), starts, mirror=False)
    logits = od.lm_logits(SHAPE, w["final_norm"], w["lm_head"], x, mirror=False)
    m = _hf_model(SHAPE, w)
    for s in range(2):
        with torch.no_grad():
            ref = m(input_ids=torch.from_numpy(seqs[s][None])).logits.numpy()[0]
        err = np.abs(logits[starts[s]:starts[s + 1]] - ref).max()
        assert err < 2e-5 * np.abs(ref).max(), err
    # token-by-token decode of sequence 1 from an empty cache
    kvp2 = _empty_pools(SHAPE, sum(need))
    for t in range(lens[1]):
        out = od.decode_step(SHAPE, w, kvp2, pt[1:2], seqs[1][t:t + 1], np.array([t]),
                             np.array([0]), seed=1, temperature=1.0, mirror=False)
        np.testing.assert_allclose(out["logits"][0], logits[starts[1] + t], rtol=0,
                                   atol=1e-10 * np.abs(logits).max())


def test_prefill_with_cached_prefix_equals_full_prefill():
    """A sequence whose first p0 tokens are already cached (start_pos = p0)
    gives the same hidden states for the rest as prefilling it whole."""
    rng = np.random.default_rng(12)
    w = _weights(SHAPE, rng)
    n, p0 = 41, 18
    toks = rng.integers(0, SHAPE.vocab, size=n)
    pt = rng.permutation(3)[None]
    kvp = _empty_pools(SHAPE, 3)
    full = od.prefill_forward(SHAPE, w, kvp, pt, toks, [0, n], mirror=False)
    kvp2 = _empty_pools(SHAPE, 3)
    od.prefill_forward(SHAPE, w, kvp2, pt, toks[:p0], [0, p0], mirror=False)
    tail = od.prefill_forward(SHAPE, w, kvp2, pt, toks[p0:], [0, n - p0], start_pos=[p0],
                              mirror=False)
    np.testing.assert_allclose(tail, full[p0:], rtol=0, atol=1e-12 * np.abs(full).max())


def test_prefill_confidence_per_sequence_means_and_batch_independence():
    """C of a sequence is the mean of Eq. 1's c over its scored rows, computed
    the same whether the sequence is scored alone or in a batch; a sequence
    without scored rows gets 0."""
    rng = np.random.default_rng(13)
    w = _weights(SHAPE, rng)
    lens = [30, 25, 9]
    toks = rng.integers(0, SHAPE.vocab, size=sum(lens))
    starts = np.concatenate([[0], np.cumsum(lens)])
    pt = np.arange(6).reshape(3, 2)
    rows = np.array([3, 10, 29, 31, 40, 54])   # none in the third sequence
    conf, c, logits = od.prefill_confidence(SHAPE, w, _empty_pools(SHAPE, 6), pt, toks, starts,
                                            rows, 5, mirror=False)
    np.testing.assert_allclose(c, od.token_confidence(logits, 5))
    np.testing.assert_allclose(conf[:2], [c[:3].mean(), c[3:].mean()])
    assert conf[2] == 0.0
    alone, c1, _ = od.prefill_confidence(SHAPE, w, _empty_pools(SHAPE, 6), pt[1:2],
                                         toks[starts[1]:starts[2]], [0, lens[1]],
                                         rows[3:] - starts[1], 5, mirror=False)
    np.testing.assert_allclose(alone[0], conf[1], rtol=1e-12)
