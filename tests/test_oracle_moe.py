"""Pins of the oracle's mixture-of-experts FFN (CPU only).

The MoE layer follows the Qwen3-MoE layout the paper's own scoring and
aggregation models use: a router, the top-k experts of each token, a softmax
over the selected router logits (the router probabilities of the selected
experts renormalised), SwiGLU experts.  Pins: the ``transformers`` Qwen3-MoE
causal forward (an independent library implementation), the closed form with
identical experts (the dense SwiGLU FFN), brute force with every expert
selected, and the routing rule's ties and normalisation.
"""
import numpy as np
import torch

from oracle import decoder as od
from paper_2604_07725_amd.synth import ModelShape

SHAPE = ModelShape(n_layers=2, hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=32, ffn=0,
                   vocab=97, rope_theta=1.0e4, n_experts=8, top_k=3, expert_ffn=24)
RNG = np.random.default_rng(21)


def _weights(shape, rng, scale=0.2):
    H, E, Fe, V = shape.hidden, shape.n_experts, shape.expert_ffn, shape.vocab
    layers = []
    for _ in range(shape.n_layers):
        layers.append({
            "attn_norm": 1 + 0.1 * rng.standard_normal(H),
            "w_qkv": scale * rng.standard_normal((shape.qkv_dim, H)),
            "q_norm": 1 + 0.1 * rng.standard_normal(shape.head_dim),
            "k_norm": 1 + 0.1 * rng.standard_normal(shape.head_dim),
            "w_o": scale * rng.standard_normal((H, shape.q_dim)),
            "ffn_norm": 1 + 0.1 * rng.standard_normal(H),
            "w_router": rng.standard_normal((E, H)),
            "w_expert_gate_up": scale * rng.standard_normal((E, 2 * Fe, H)),
            "w_expert_down": scale * rng.standard_normal((E, H, Fe)),
        })
    return {"embed": rng.standard_normal((V, H)), "lm_head": scale * rng.standard_normal((V, H)),
            "final_norm": 1 + 0.1 * rng.standard_normal(H), "layers": layers}


def test_route_picks_largest_with_low_index_ties_and_normalises():
    logits = np.array([[0.5, 2.0, 2.0, -1.0, 2.0, 0.1]])
    sel, w, gap = od.moe_route(logits, 2)
    assert sel.tolist() == [[1, 2]]                 # three-way tie at 2.0: lowest indices first
    np.testing.assert_allclose(w, [[0.5, 0.5]])
    assert gap[0] == 0.0
    z = RNG.standard_normal((5, 9))
    sel, w, _ = od.moe_route(z, 4)
    p = np.exp(z - z.max(-1, keepdims=True))
    p /= p.sum(-1, keepdims=True)                   # router softmax over all experts
    for t in range(5):
        top = np.argsort(-p[t])[:4]
        assert sorted(sel[t].tolist()) == sorted(top.tolist())
        np.testing.assert_allclose(w[t], p[t, sel[t]] / p[t, sel[t]].sum(), rtol=1e-12)
        np.testing.assert_allclose(w[t].sum(), 1.0, rtol=1e-14)


def test_identical_experts_reduce_to_the_dense_ffn():
    lw = _weights(SHAPE, RNG)["layers"][0]
    lw["w_expert_gate_up"][:] = lw["w_expert_gate_up"][0]
    lw["w_expert_down"][:] = lw["w_expert_down"][0]
    h2 = RNG.standard_normal((6, SHAPE.hidden))
    out, _ = od.moe_ffn(SHAPE, lw, h2, mirror=False)
    Fe = SHAPE.expert_ffn
    gu = h2 @ lw["w_expert_gate_up"][0].T
    dense = (od.silu(gu[:, :Fe]) * gu[:, Fe:]) @ lw["w_expert_down"][0].T
    np.testing.assert_allclose(out, dense, rtol=1e-12, atol=1e-12)


def test_all_experts_selected_is_the_softmax_weighted_sum():
    import dataclasses
    shape = dataclasses.replace(SHAPE, top_k=SHAPE.n_experts)
    lw = _weights(shape, RNG)["layers"][0]
    h2 = RNG.standard_normal((3, shape.hidden))
    out, _ = od.moe_ffn(shape, lw, h2, mirror=False)
    Fe = shape.expert_ffn
    for t in range(3):
        z = h2[t] @ lw["w_router"].T
        p = np.exp(z - z.max())
        p /= p.sum()
        ref = np.zeros(shape.hidden)
        for e in range(shape.n_experts):
            gu = h2[t] @ lw["w_expert_gate_up"][e].T
            ref += p[e] * ((od.silu(gu[:Fe]) * gu[Fe:]) @ lw["w_expert_down"][e].T)
        np.testing.assert_allclose(out[t], ref, rtol=1e-11, atol=1e-12)


def _hf_moe_model(shape, w):
    from transformers import Qwen3MoeConfig, Qwen3MoeForCausalLM
    cfg = Qwen3MoeConfig(vocab_size=shape.vocab, hidden_size=shape.hidden,
                         intermediate_size=4 * shape.hidden,
                         moe_intermediate_size=shape.expert_ffn,
                         num_experts=shape.n_experts, num_experts_per_tok=shape.top_k,
                         norm_topk_prob=True, decoder_sparse_step=1, mlp_only_layers=[],
                         num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_q_heads,
                         num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                         rms_norm_eps=shape.rms_eps,
                         rope_parameters={"rope_theta": shape.rope_theta, "rope_type": "default"},
                         max_position_embeddings=256, tie_word_embeddings=False,
                         attention_bias=False, hidden_act="silu")
    cfg._attn_implementation = "eager"
    cfg._experts_implementation = "eager"    # the per-expert loop (float64 capable)
    m = Qwen3MoeForCausalLM(cfg).to(torch.float64).eval()
    T = lambda a: torch.from_numpy(np.asarray(a, np.float64))  # noqa: E731
    qd, kd = shape.q_dim, shape.kv_dim
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
            layer.mlp.gate.weight.copy_(T(lw["w_router"]))
            layer.mlp.experts.gate_up_proj.copy_(T(lw["w_expert_gate_up"]))
            layer.mlp.experts.down_proj.copy_(T(lw["w_expert_down"]))
    return m


def test_moe_prefill_equals_transformers_qwen3_moe():
    """The oracle's MoE decoder (prefill over one sequence, no bf16 mirroring)
    reproduces the transformers Qwen3-MoE causal forward with normalised top-k
    routing; the margins of the routing choices are reported so a tie cannot
    pass silently."""
    w = _weights(SHAPE, RNG)
    n = 29
    toks = RNG.integers(0, SHAPE.vocab, size=n)
    pt = RNG.permutation(2)[None]
    kvp = [np.zeros((2, SHAPE.n_kv_heads, 2, 16 * SHAPE.head_dim)) for _ in range(2)]
    row, pos = od.prefill_index([0, n])
    x = np.asarray(w["embed"][toks], np.float64)
    stats = {}
    for l in range(SHAPE.n_layers):
        x = od.decoder_layer(SHAPE, w["layers"][l], x, pos, kvp[l], pt[row], mirror=False,
                             stats=stats)
    logits = od.lm_logits(SHAPE, w["final_norm"], w["lm_head"], x, mirror=False)
    assert stats["route_gap"] > 1e-6        # no routing tie that rounding could flip
    m = _hf_moe_model(SHAPE, w)
    with torch.no_grad():
        ref = m(input_ids=torch.from_numpy(toks[None])).logits.numpy()[0]
    err = np.abs(logits - ref).max()
    assert err < 2e-5 * np.abs(ref).max(), err
