"""GPU parity of the mixture-of-experts decode path against the oracle,
through the C ABI: the MoE FFN alone (routing, weights, expert outputs) and
whole decode steps of MoE models.

Routing decisions are taken on fp32 router logits on both sides; an expert
choice is compared exactly wherever the oracle's float64 gap between the k-th
and (k+1)-th logit exceeds ROUTE_GAP (a choice that close could flip on
rounding).  The FFN test checks near-tie tokens for a valid choice instead;
the step tests check that their inputs have none.
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import decoder as od
from paper_2604_07725_amd import synth
from tests.gpu_helpers import (check_ids, poisoned, say, subset_host_state,
                               tile_activations_host)

pytestmark = pytest.mark.gpu

ROUTE_GAP = 1e-5


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_07725_amd import device_inputs, sevo
    sevo.lib()
    return sevo, device_inputs


def _model(S, shape, seed, max_position=1024):
    sevo, di = S
    tensors = di.device_weights(shape, seed)
    return sevo.sevo_init_model(shape, tensors, max_position=max_position)


@pytest.mark.parametrize("shape_name,n", [("tiny", 1), ("tiny", 37), ("tiny", 100), ("tiny", 2000),
                                          ("moe30b", 64), ("moe30b", 300)])
def test_moe_ffn_matches_oracle(S, shape_name, n):
    """One layer's MoE FFN on random normed inputs: selected experts (exact),
    routing weights, and the sum of the per-slot partials against the oracle
    on the same bf16 inputs.  The partials start as NaN, so a (token, slot)
    the expert lists miss fails; n = 2000 spans several expert row tiles and
    several chunks of the assignment planner."""
    sevo, _ = S
    shape = synth.TINY_MOE if shape_name == "tiny" else dataclasses.replace(
        synth.MOE_30B_A3B, n_layers=1)
    seed = 41 + n
    say(f"moe ffn {shape_name} n={n}")
    model = _model(S, shape, seed)
    key = synth.tensor_key(seed, 60, 0)
    h_vals = synth.host_values(synth.TensorSpec((n, shape.hidden), key, 1.0)).reshape(
        n, shape.hidden)
    bits = (np.ascontiguousarray(h_vals, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    ht = torch.from_numpy(tile_activations_host(bits).view(np.int16)).cuda().view(torch.bfloat16)
    part = torch.full((shape.top_k, n, shape.hidden), float("nan"), device="cuda")
    ex, wt, part = sevo.sevo_moe_ffn(model, 0, ht, n, partials=part)
    torch.cuda.synchronize()
    g_ex = ex.cpu().numpy().astype(np.int64)
    g_wt = wt.cpu().numpy().astype(np.float64)
    g_out = part.double().sum(0).cpu().numpy()   # slot order is the sum order on the GPU too
    assert np.isfinite(g_out).all(), "a (token, slot) partial was never written"
    model.close()
    lw = synth.host_weights(shape, seed, lazy=True)["layers"][0]
    logits = od._f32(h_vals.astype(np.float64) @ np.asarray(lw["w_router"], np.float64).T)
    sel, w, gap = od.moe_route(logits, shape.top_k)
    exact = gap > ROUTE_GAP
    say(f"  smallest routing gap {gap.min():.2e}; {int((~exact).sum())} near-tie tokens")
    assert exact.mean() > 0.9
    np.testing.assert_array_equal(g_ex[exact], sel[exact])
    np.testing.assert_allclose(g_wt[exact], w[exact], rtol=2e-5, atol=1e-6)
    for t in np.nonzero(~exact)[0]:
        # a near tie: k distinct experts, each within the gap of the k-th largest logit
        assert len(set(g_ex[t].tolist())) == shape.top_k
        kth = np.sort(logits[t])[::-1][shape.top_k - 1]
        assert logits[t, g_ex[t]].min() >= kth - ROUTE_GAP
    ref, _ = od.moe_ffn(shape, lw, h_vals.astype(np.float64))
    err = np.abs(g_out[exact] - ref[exact]).max() / np.abs(ref).max()
    say(f"  expert output max rel err {err:.2e}")
    # one bf16 rounding of the SwiGLU product (mirrored) and fp32 sums
    assert err <= 2e-3


def test_tiny_moe_step_sequence_matches_oracle(S):
    """Three decode steps of the tiny MoE workload (2 layers, 64 experts,
    top-4): logits, ids and log-probs against the oracle."""
    sevo, di = S
    w = synth.WORKLOADS["tiny_moe_step"]
    shape = w.shape
    steps = 3
    say("tiny MoE step sequence")
    pop = synth.workload_population(w, extra_tokens=steps)
    model = _model(S, shape, w.seed, max_position=int(pop.lengths.max()) + steps + 1)
    kvp = di.device_pools(shape, w.seed, pop.n_pages)
    d = di.device_population(pop)
    hw = synth.host_weights(shape, w.seed)
    hkv = [p.astype(np.float64) for p in synth.host_pools(shape, w.seed, pop.n_pages)]
    toks = pop.tokens.astype(np.int64)
    pos = pop.lengths.astype(np.int64)
    pos_d = d["lengths"].clone()
    ws_bytes = sevo.sevo_step_workspace_bytes(model, pop.n, pop.max_pages)
    for step in range(steps):
        ids, lps, logits = sevo.sevo_decode_step(
            model, torch.from_numpy(toks.astype(np.int32)).cuda(), pos_d, d["page_table"], kvp,
            d["uids"], 7, 1.0, keep_logits=True, workspace=poisoned(ws_bytes))  # NaN scratch
        torch.cuda.synchronize()
        stats, det = {}, {}
        ref = od.decode_step(shape, hw, hkv, pop.page_table, toks, pos, pop.uids, 7, 1.0,
                             stats=stats, details=det)
        assert stats["route_gap"] > ROUTE_GAP, "test input has a routing near-tie"
        err = np.abs(logits.double().cpu().numpy() - ref["logits"]).max()
        say(f"  step {step}: logit max abs err {err:.2e}; route gap {stats['route_gap']:.2e}")
        assert err <= 1e-2       # the tiny-model end-to-end bar of the dense step
        check_ids(ids.cpu().numpy(), lps.cpu().numpy(), ref["ids"], ref["lps"], ref["gaps"],
                  det, label=f"step {step}")
        toks = ref["ids"]
        pos = pos + 1
        pos_d += 1
    model.close()


def test_moe30b_step_reduced_depth(S):
    """The 30B-A3B-class MoE model at its real widths (hidden 2048, 32/4 heads,
    128 experts, top-8, expert FFN 768, vocab 151936), full population and
    contexts of the benchmark, 2 layers: logits and log-probs of sampled
    candidates against the oracle on those candidates alone."""
    sevo, di = S
    w = synth.WORKLOADS["moe30b_pop64_agg4"]
    shape = dataclasses.replace(w.shape, n_layers=2)
    say("MoE 30B-A3B widths at 2 layers")
    pop = synth.workload_population(w, extra_tokens=1)
    model = _model(S, shape, w.seed, max_position=int(pop.lengths.max()) + 2)
    kvp = di.device_pools(shape, w.seed, pop.n_pages)
    d = di.device_population(pop)
    ids, lps, logits = sevo.sevo_decode_step(model, d["tokens"], d["lengths"], d["page_table"],
                                             kvp, d["uids"], 77, 1.0, keep_logits=True)
    torch.cuda.synchronize()
    idx = sorted({int(np.argmin(pop.lengths)), int(np.argmax(pop.lengths)), 1})
    g_logits = logits.double().cpu().numpy()[idx]
    g_lps = lps.cpu().numpy()[idx]
    model.close()
    del kvp
    torch.cuda.empty_cache()
    # the oracle runs on the sampled candidates alone: candidates do not
    # interact, routing included (each token routes on its own)
    hkv, pt = subset_host_state(shape, w.seed, pop, idx, shape.n_layers)
    hw = synth.host_weights(shape, w.seed, lazy=True)
    hw = {"embed": hw["embed"], "final_norm": hw["final_norm"], "layers": hw["layers"],
          "lm_head": hw["lm_head"][0:shape.vocab]}
    stats = {}
    ref = od.decode_step(shape, hw, hkv, pt, pop.tokens[idx], pop.lengths[idx], pop.uids[idx],
                         77, 1.0, stats=stats)
    err = np.abs(g_logits - ref["logits"]).max()
    lp_err = np.abs(g_lps - ref["lps"]).max()
    say(f"  candidates {idx}: logit err {err:.2e}, lp err {lp_err:.2e}, route gap "
        f"{stats['route_gap']:.2e}")
    assert stats["route_gap"] > ROUTE_GAP, "test input has a routing near-tie"
    # the full-width end-to-end bars of the dense step (bf16 storage flips)
    assert err <= 6e-2
    assert lp_err <= 2.5e-2


def test_moe_entry_points_reject_bad_arguments(S):
    """Error paths: the MoE FFN of a dense model (UNSUPPORTED), a layer out of
    range and more than 2^30 expert entries (INVALID_ARGUMENT), and the
    confidence engine with a negative moe_chunk (INVALID_ARGUMENT)."""
    import ctypes as C
    sevo, di = S
    dense = _model(S, synth.TINY, 1)
    moe = _model(S, synth.TINY_MOE, 1)
    L = sevo.lib()
    buf = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    p = C.c_void_p(buf.data_ptr())
    args = lambda m, layer, n: (m.handle, layer, p, n, p, p, p, p, buf.numel(), None)  # noqa: E731
    assert L.sevo_moe_ffn(*args(dense, 0, 4)) == sevo.UNSUPPORTED
    assert L.sevo_moe_ffn(*args(moe, 2, 4)) == sevo.INVALID_ARGUMENT
    assert L.sevo_moe_ffn(*args(moe, -1, 4)) == sevo.INVALID_ARGUMENT
    assert L.sevo_moe_ffn(*args(moe, 0, (1 << 30) // 4 + 1)) == sevo.INVALID_ARGUMENT
    assert L.sevo_moe_ffn(*args(moe, 0, 0)) == sevo.OK
    # the engine on the MoE model with a negative chunk
    toks = torch.zeros(32, dtype=torch.int32, device="cuda")
    ss = torch.tensor([0, 32], dtype=torch.int32, device="cuda")
    pt = torch.arange(2, dtype=torch.int32, device="cuda")[None]
    pool = torch.zeros(2, 2, 2, 16 * 64, dtype=torch.bfloat16, device="cuda")
    rows = torch.arange(32, dtype=torch.int32, device="cuda")
    b = sevo.PrefillBuffers(moe, toks, ss, pt, pool, rows, 20, 32, moe_chunk=-1)
    assert L.sevo_prefill_confidence(moe.handle, C.byref(b.args), None) == sevo.INVALID_ARGUMENT
    b.args.moe_chunk = 16
    assert L.sevo_prefill_confidence(moe.handle, C.byref(b.args), None) == sevo.OK
    torch.cuda.synchronize()
    assert np.isfinite(b.out_conf.cpu().numpy()).all()
    dense.close()
    moe.close()
