"""GPU parity of the prefill path (the confidence engine's scoring pass)
against the CPU oracle, through the C ABI.

Inputs come from the seeded generator (device twin on the GPU, host twin for
the oracle); sizes span several 64-token query blocks and 64-key blocks with
ragged tails, cached-prefix offsets and every supported GQA group.
"""
import numpy as np
import pytest
import torch

from oracle import decoder as od
from paper_2604_07725_amd import synth
from tests.gpu_helpers import ATTN_REL_TOL, attn_rel_err, make_population, say, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_07725_amd import device_inputs, sevo
    sevo.lib()
    return sevo, device_inputs


def _shape(hq, hkv, d):
    return synth.ModelShape(n_layers=1, hidden=hq * d, n_q_heads=hq, n_kv_heads=hkv, head_dim=d,
                            ffn=128, vocab=256)


PREFILL_ATTN_CASES = [
    # (hq, hkv, d), sequence lengths, cached-prefix positions
    ((32, 8, 128), [1, 63, 64, 65, 200], [0, 0, 17, 5, 300]),
    ((4, 2, 64), [130, 7], [0, 40]),
    ((64, 8, 128), [100], [0]),
    ((8, 8, 64), [77, 33], [3, 0]),
    ((32, 8, 128), [1000], [0]),
]


@pytest.mark.parametrize("dims,lens,starts", PREFILL_ATTN_CASES)
def test_attn_prefill_matches_oracle(S, dims, lens, starts):
    sevo, di = S
    shape = _shape(*dims)
    say(f"attn prefill {dims} lens={lens} start={starts}")
    lens = np.asarray(lens, np.int64)
    starts = np.asarray(starts, np.int64)
    keys = starts + lens
    seed = int(keys.sum()) % 1000 + 7
    pop = make_population(keys, shuffle=True, seed=seed)
    kvp = di.device_pools(shape, seed, pop.n_pages, layers=[0])[0]
    T = int(lens.sum())
    q = di.device_q(shape, seed, T)
    seq_starts = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    out = sevo.sevo_attn_prefill(q, kvp, torch.from_numpy(pop.page_table.astype(np.int32)).cuda(),
                                 torch.from_numpy(seq_starts).cuda(), int(lens.max()),
                                 start_pos=torch.from_numpy(starts.astype(np.int32)).cuda())
    torch.cuda.synchronize()
    got = to_np(out)
    qh = synth.host_values(synth.q_spec(shape, seed, T)).reshape(T, shape.n_q_heads,
                                                                  shape.head_dim)
    spec = synth.kv_spec(shape, seed, 0, pop.n_pages)
    pool = synth.pool_pages(spec, np.arange(pop.n_pages))
    ref = od.prefill_attention(qh, pool, pop.page_table, seq_starts, starts,
                               shape.head_dim ** -0.5)
    for s in range(len(lens)):
        a, b = seq_starts[s], seq_starts[s + 1]
        err = attn_rel_err(got[a:b], ref[a:b])
        say(f"  seq {s}: len {lens[s]} start {starts[s]} rel err {err:.2e}")
        # bf16 probabilities in the P V product: a few 1e-3 at most
        assert err <= min(ATTN_REL_TOL, 8e-3), f"seq {s}: {err}"


@pytest.mark.parametrize("hq,hkv", [(32, 8), (32, 4)])
def test_attn_prefill_full_size_sampled(S, hq, hkv):
    """The prefill attention at the engine benchmark's size and launch shape
    (one 40960-token sequence, d = 128, the 8B and 30B-A3B head layouts) on
    sampled query rows, each computed by the oracle over its keys 0..t."""
    sevo, di = S
    T, d = 40960, 128
    shape = _shape(hq, hkv, d)
    seed = 91 + hkv
    say(f"attn prefill full size {hq}/{hkv} x {d}, {T} tokens")
    pop = make_population([T], shuffle=True, seed=seed)
    kvp = di.device_pools(shape, seed, pop.n_pages, layers=[0])[0]
    q = di.device_q(shape, seed, T)
    pt = torch.from_numpy(pop.page_table.astype(np.int32)).cuda()
    ss = torch.tensor([0, T], dtype=torch.int32, device="cuda")
    out = sevo.sevo_attn_prefill(q, kvp, pt, ss, T)
    rows = [0, 1, 63, 64, 4095, 20011, 40958, 40959]
    got = to_np(out[rows])
    del kvp, q, out
    torch.cuda.empty_cache()
    pool = synth.pool_pages(synth.kv_spec(shape, seed, 0, pop.n_pages), np.arange(pop.n_pages))
    K, V = od.gather_kv(pool, pop.page_table[0], T)
    qspec = synth.q_spec(shape, seed, T)
    for i, t in enumerate(rows):
        qt = synth.host_values(qspec, offset=t * hq * d, count=hq * d).reshape(hq, d)
        ref = od.attention_dense(qt, K[:, :t + 1], V[:, :t + 1], d ** -0.5)
        err = attn_rel_err(got[i], ref)
        say(f"  row {t}: rel err {err:.2e}")
        assert err <= min(ATTN_REL_TOL, 8e-3), f"row {t}: {err}"


def test_attn_prefill_page_permutation_bit_exact(S):
    """The result depends only on the logical key order: moving the pages to
    other physical slots gives identical bits."""
    sevo, di = S
    shape = _shape(32, 8, 128)
    lens = np.array([150, 70])
    say("attn prefill page permutation")
    pop = make_population(lens, shuffle=True, seed=5)
    kvp = di.device_pools(shape, 5, pop.n_pages, layers=[0])[0]
    perm = np.random.default_rng(1).permutation(pop.n_pages)
    kvp2 = torch.empty_like(kvp)
    kvp2[torch.from_numpy(perm).cuda()] = kvp
    pt2 = np.where(pop.page_table >= 0, perm[np.maximum(pop.page_table, 0)], -1)
    q = di.device_q(shape, 5, int(lens.sum()))
    ss = torch.tensor([0, 150, 220], dtype=torch.int32, device="cuda")
    o1 = sevo.sevo_attn_prefill(q, kvp, torch.from_numpy(pop.page_table.astype(np.int32)).cuda(),
                                ss, 150)
    o2 = sevo.sevo_attn_prefill(q, kvp2, torch.from_numpy(pt2.astype(np.int32)).cuda(), ss, 150)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))


@pytest.mark.parametrize("dims", [(32, 8, 128), (32, 4, 128), (8, 2, 64)])
def test_attn_prefill_ignores_slots_past_the_last_key(S, dims):
    """Slots of a sequence's last page past its last key may hold anything:
    NaN patterns written there (K and V tiles, every kv head) leave the
    output bit-identical."""
    sevo, di = S
    shape = _shape(*dims)
    d = shape.head_dim
    lens = np.array([37, 100, 16, 250])
    say(f"attn prefill with NaN past the last key {dims}")
    pop = make_population(lens, shuffle=True, seed=21)
    kvp = di.device_pools(shape, 21, pop.n_pages, layers=[0])[0]
    q = di.device_q(shape, 21, int(lens.sum()))
    ss = torch.from_numpy(np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)).cuda()
    pt = torch.from_numpy(pop.page_table.astype(np.int32)).cuda()
    o1 = sevo.sevo_attn_prefill(q, kvp, pt, ss, int(lens.max()))
    pool = kvp.view(torch.int16).cpu().numpy().copy()   # [P][hkv][2][16 d]
    e = np.arange(d)
    for i, n in enumerate(lens):
        if n % 16 == 0:
            continue
        page = pop.page_table[i, n // 16]
        for slot in range(n % 16, 16):
            pool[page, :, 0, ((e // 32) * 16 + slot) * 32 + e % 32] = np.int16(0x7FC0)  # K
            pool[page, :, 1, e * 16 + slot] = np.int16(0x7FC0)                          # V
    kvp_nan = torch.from_numpy(pool).cuda().view(torch.bfloat16)
    o2 = sevo.sevo_attn_prefill(q, kvp_nan, pt, ss, int(lens.max()))
    torch.cuda.synchronize()
    assert torch.isfinite(o2.float()).all()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))


# ------------------------------------------------------------------ confidence engine
def _token_major(pool, d):
    """K and V of every (page, head, slot) of a pool [P, hkv, 2, 16 d] as
    [P, hkv, 16, d] arrays (tile offsets of the documented layout)."""
    s = np.arange(16)[:, None]
    e = np.arange(d)[None, :]
    return (pool[:, :, 0, :][:, :, ((e // 32) * 16 + s) * 32 + e % 32],
            pool[:, :, 1, :][:, :, e * 16 + s])


def _engine_case(S, shape, seed, lens, scored, conf_k, starts=None, moe_chunk=0):
    """Run the confidence engine on the GPU; returns its outputs and the inputs
    the oracle needs (host side)."""
    sevo, di = S
    lens = np.asarray(lens, np.int64)
    starts = np.zeros(len(lens), np.int64) if starts is None else np.asarray(starts, np.int64)
    pop = make_population(starts + lens, shuffle=True, seed=seed)
    rng = np.random.default_rng(seed)
    toks = rng.integers(0, shape.vocab, size=int(lens.sum())).astype(np.int32)
    seq_starts = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    tensors = di.device_weights(shape, seed)
    model = sevo.sevo_init_model(shape, tensors, max_position=int((starts + lens).max()) + 1)
    kvp = di.device_pools(shape, seed, pop.n_pages)
    buf = sevo.PrefillBuffers(model, torch.from_numpy(toks).cuda(),
                              torch.from_numpy(seq_starts).cuda(),
                              torch.from_numpy(pop.page_table.astype(np.int32)).cuda(), kvp,
                              torch.from_numpy(np.asarray(scored, np.int32)).cuda(), conf_k,
                              int(lens.max()),
                              start_pos=torch.from_numpy(starts.astype(np.int32)).cuda(),
                              moe_chunk=moe_chunk)
    conf = buf.run()
    torch.cuda.synchronize()
    out = (conf.cpu().numpy().astype(np.float64),
           buf.out_row_conf[:len(scored)].cpu().numpy().astype(np.float64),
           [p.double().cpu().numpy() for p in kvp])
    model.close()
    return out, pop, toks, seq_starts, starts


def test_prefill_confidence_full_size_batch_invariance(S):
    """The dense 8B engine at the benchmark's size (36 layers, 40960 tokens as
    sequences of 24576 and 16384, every row scored): each row's c equals, bit
    for bit, its value with the sequence run alone, and so does each C (rows
    of different sequences never interact; a property at any size), all
    finite, and C is the mean of its sequence's c."""
    sevo, di = S
    shape = synth.DENSE_8B
    lens = [24576, 16384]
    seed = 17
    say(f"prefill confidence full size, dense 8B, sequences {lens}")
    pop = make_population(lens, shuffle=True, seed=seed)
    rng = np.random.default_rng(seed)
    toks = [rng.integers(0, shape.vocab, size=n).astype(np.int32) for n in lens]
    model = sevo.sevo_init_model(shape, di.device_weights(shape, seed),
                                 max_position=max(lens) + 1)
    # every slot the prefill reads it writes first; later slots may hold anything
    kvp = [torch.empty(pop.n_pages, shape.n_kv_heads, 2, 16 * shape.head_dim,
                       dtype=torch.bfloat16, device="cuda") for _ in range(shape.n_layers)]

    def run(seqs):
        t = np.concatenate([toks[i] for i in seqs])
        ss = np.concatenate([[0], np.cumsum([lens[i] for i in seqs])]).astype(np.int32)
        pt = np.ascontiguousarray(pop.page_table[seqs]).astype(np.int32)
        buf = sevo.PrefillBuffers(model, torch.from_numpy(t).cuda(), torch.from_numpy(ss).cuda(),
                                  torch.from_numpy(pt).cuda(), kvp,
                                  torch.arange(len(t), dtype=torch.int32, device="cuda"), 20,
                                  max(lens[i] for i in seqs))
        conf = buf.run()
        torch.cuda.synchronize()
        return conf.cpu().numpy(), buf.out_row_conf[:len(t)].cpu().numpy()

    c01, r01 = run([0, 1])
    c0, r0 = run([0])
    c1, r1 = run([1])
    model.close()
    say(f"  C = {c01}, alone {c0} {c1}")
    assert np.isfinite(r01).all() and np.isfinite(c01).all()
    np.testing.assert_array_equal(r01[:lens[0]], r0)
    np.testing.assert_array_equal(r01[lens[0]:], r1)
    np.testing.assert_array_equal(c01, np.concatenate([c0, c1]))
    np.testing.assert_allclose(c01, [r0.astype(np.float64).mean(), r1.astype(np.float64).mean()],
                               rtol=1e-5)


def test_prefill_confidence_tiny_matches_oracle(S):
    """Two sequences of the tiny model through the whole engine: per-row c
    (Eq. 1), per-sequence C (Eq. 2) and every appended K/V slot against the
    oracle's prefill."""
    shape = synth.WORKLOADS["tiny_step"].shape
    lens = [300, 170]
    scored = list(range(40, 300)) + list(range(320, 470))
    say("prefill confidence (tiny model)")
    (g_conf, g_row, g_pools), pop, toks, seq_starts, starts = _engine_case(
        S, shape, 3, lens, scored, 20)
    hw = synth.host_weights(shape, 3)
    hkv = [p.astype(np.float64) for p in synth.host_pools(shape, 3, pop.n_pages)]
    conf, c, _ = od.prefill_confidence(shape, hw, hkv, pop.page_table, toks, seq_starts, scored,
                                       20)
    row_err = np.abs(g_row - c).max()
    say(f"  row c max err {row_err:.2e} (c in [{c.min():.3f}, {c.max():.3f}]); C {g_conf} vs "
        f"{conf}")
    # logits of the tiny model hold to 1e-2 end to end (bf16 storage flips, as
    # for the decode step); c = logsumexp - mean top-K follows them
    assert row_err <= 2e-2
    assert np.abs(g_conf - conf).max() <= 1e-2
    # every key / value the prefill appended, within one bf16 rounding step
    for l in range(shape.n_layers):
        gk, gv = _token_major(g_pools[l], shape.head_dim)
        hk, hv = _token_major(hkv[l], shape.head_dim)
        written = np.zeros(gk.shape[:3], bool)
        for s, n in enumerate(lens):
            for p in range(n):
                written[pop.page_table[s, p // 16], :, p % 16] = True
        spec = synth.kv_spec(shape, 3, l, pop.n_pages)
        k0, v0 = _token_major(synth.host_values(spec).reshape(spec.shape), shape.head_dim)
        np.testing.assert_array_equal(gk[~written], k0[~written])
        np.testing.assert_array_equal(gv[~written], v0[~written])
        for name, g, h in (("k", gk[written], hk[written]), ("v", gv[written], hv[written])):
            # g, h: [slots, d].  A value is one bf16 rounding step from the
            # oracle's, except where an upstream bf16 storage point (the
            # normed input h of the projection) rounded the other way: that
            # moves a whole vector by about one step of its largest entry
            d = np.abs(g - h)
            step = 2.0 ** -7 * np.abs(h) + 1e-6
            vec = 2.0 ** -7 * np.abs(h).max(axis=-1, keepdims=True)
            frac = float(np.mean(d <= step))
            say(f"  layer {l} {name}: {frac:.5f} within one rounding step, worst "
                f"{(d / (step + vec)).max():.2f} of the vector-scale bound")
            assert np.all(d <= step + vec)
            assert frac >= 0.99


def test_prefill_confidence_full_width_reduced_depth(S):
    """The 8B-class widths (hidden 4096, 32/8 x 128 heads, FFN 12288, vocab
    151936) at 2 layers, two sequences of 400 and 200 tokens (the large-M GEMM
    and several query / key blocks), 32 scored rows spread over both."""
    import dataclasses
    shape = dataclasses.replace(synth.DENSE_8B, n_layers=2)
    lens = [400, 200]
    scored = sorted(set(np.linspace(0, 599, 32).astype(int).tolist()))
    say("prefill confidence (8B widths, 2 layers)")
    (g_conf, g_row, _), pop, toks, seq_starts, starts = _engine_case(S, shape, 4, lens, scored, 20)
    torch.cuda.empty_cache()
    hw = synth.host_weights(shape, 4, lazy=True)
    hw = {"embed": hw["embed"], "final_norm": hw["final_norm"], "layers": hw["layers"],
          "lm_head": hw["lm_head"][0:shape.vocab]}
    hkv = [p.astype(np.float64) for p in synth.host_pools(shape, 4, pop.n_pages)]
    conf, c, _ = od.prefill_confidence(shape, hw, hkv, pop.page_table, toks, seq_starts, scored,
                                       20)
    row_err = np.abs(g_row - c).max()
    say(f"  row c max err {row_err:.2e} (c in [{c.min():.3f}, {c.max():.3f}]); C {g_conf} vs "
        f"{conf}")
    # the full-width end-to-end bar of the decode step (bf16 storage flips)
    assert row_err <= 6e-2
    assert np.abs(g_conf - conf).max() <= 3e-2


@pytest.mark.parametrize("lens,moe_chunk", [([300, 170], 0), ([300, 170], 64),
                                            ([400, 300], 0), ([400, 300], 512),
                                            ([1500, 700], 0)])
def test_prefill_confidence_tiny_moe_matches_oracle(S, lens, moe_chunk):
    """The tiny MoE model (2 layers, 64 experts of FFN 64, top-4) through the
    whole engine: per-row c, per-sequence C against the oracle's prefill.  The
    expert FFN runs in one chunk or in several (the last one partial); 470
    tokens take the decode expert kernels, 700 tokens (>= 32 entries per
    expert) the grouped large-M GEMMs, and 512 + 188 one of each; 2200 tokens
    (8800 entries) plan their lists in 1024-entry chunks (three launches).  The
    inputs have no routing choice closer than 1e-5."""
    shape = synth.TINY_MOE
    seed = 9
    T = sum(lens)
    scored = list(range(40, lens[0])) + list(range(lens[0] + 20, T))
    say(f"prefill confidence (tiny MoE, {lens}, chunk {moe_chunk})")
    (g_conf, g_row, _), pop, toks, seq_starts, starts = _engine_case(
        S, shape, seed, lens, scored, 20, moe_chunk=moe_chunk)
    hw = synth.host_weights(shape, seed)
    hkv = [p.astype(np.float64) for p in synth.host_pools(shape, seed, pop.n_pages)]
    stats = {}
    conf, c, _ = od.prefill_confidence(shape, hw, hkv, pop.page_table, toks, seq_starts, scored,
                                       20, stats=stats)
    row_err = np.abs(g_row - c).max()
    say(f"  row c max err {row_err:.2e}; C {g_conf} vs {conf}; route gap {stats['route_gap']:.2e}")
    assert stats["route_gap"] > 1e-5, "test input has a routing near-tie"
    assert row_err <= 2e-2
    assert np.abs(g_conf - conf).max() <= 1e-2


@pytest.mark.parametrize("moe_chunk", [0, 256])
def test_prefill_confidence_moe30b_reduced_depth(S, moe_chunk):
    """The 30B-A3B-class MoE widths (hidden 2048, 32/4 heads, 128 experts of
    FFN 768, top-8, vocab 151936) at 2 layers, two sequences of 400 and 200
    tokens, 32 scored rows; the expert FFN in one chunk (37.5 entries per
    expert: the grouped large-M GEMMs) or in 256-token chunks (the decode
    expert kernels)."""
    import dataclasses
    shape = dataclasses.replace(synth.MOE_30B_A3B, n_layers=2)
    lens = [400, 200]
    scored = sorted(set(np.linspace(0, 599, 32).astype(int).tolist()))
    say("prefill confidence (30B-A3B widths, 2 layers)")
    (g_conf, g_row, _), pop, toks, seq_starts, starts = _engine_case(
        S, shape, 10, lens, scored, 20, moe_chunk=moe_chunk)
    torch.cuda.empty_cache()
    hw = synth.host_weights(shape, 10, lazy=True)
    hw = {"embed": hw["embed"], "final_norm": hw["final_norm"], "layers": hw["layers"],
          "lm_head": hw["lm_head"][0:shape.vocab]}
    hkv = [p.astype(np.float64) for p in synth.host_pools(shape, 10, pop.n_pages)]
    stats = {}
    conf, c, _ = od.prefill_confidence(shape, hw, hkv, pop.page_table, toks, seq_starts, scored,
                                       20, stats=stats)
    row_err = np.abs(g_row - c).max()
    say(f"  row c max err {row_err:.2e}; C {g_conf} vs {conf}; route gap {stats['route_gap']:.2e}")
    assert stats["route_gap"] > 1e-5, "test input has a routing near-tie"
    assert row_err <= 6e-2
    assert np.abs(g_conf - conf).max() <= 3e-2


@pytest.mark.parametrize("dims", [(32, 8, 128), (8, 2, 64)])
def test_attn_prefill_absent_pages_contribute_no_keys(S, dims):
    """A page id outside the pool contributes no keys, as in decode: keys
    48..63 of sequence 0 (an id past the pool) and keys 0..15 of sequence 1 (a
    negative id) are left out of every row's softmax; rows 0..15 of sequence 1
    then see no key at all and give o = 0."""
    sevo, di = S
    shape = _shape(*dims)
    hq, d = shape.n_q_heads, shape.head_dim
    lens = np.array([150, 70])
    say(f"attn prefill with absent pages {dims}")
    pop = make_population(lens, shuffle=True, seed=23)
    bad = pop.page_table.copy()
    bad[0, 3] = pop.n_pages + 1000
    bad[1, 0] = -5
    kvp = di.device_pools(shape, 23, pop.n_pages, layers=[0])[0]
    T = int(lens.sum())
    q = di.device_q(shape, 23, T)
    ss = np.array([0, 150, 220], np.int32)
    out = sevo.sevo_attn_prefill(q, kvp, torch.from_numpy(bad.astype(np.int32)).cuda(),
                                 torch.from_numpy(ss).cuda(), int(lens.max()))
    torch.cuda.synchronize()
    got = to_np(out)
    assert np.isfinite(got).all()
    qh = synth.host_values(synth.q_spec(shape, 23, T)).reshape(T, hq, d)
    pool = synth.pool_pages(synth.kv_spec(shape, 23, 0, pop.n_pages), np.arange(pop.n_pages))
    worst = 0.0
    for s, drop in ((0, range(48, 64)), (1, range(0, 16))):
        K, V = od.gather_kv(pool, pop.page_table[s], int(lens[s]))
        for t in range(int(lens[s])):
            keep = np.array([u for u in range(t + 1) if u not in drop], np.int64)
            row = got[ss[s] + t]
            if keep.size == 0:
                assert np.all(row == 0), (s, t)
                continue
            ref = od.attention_dense(qh[ss[s] + t], K[:, keep], V[:, keep], d ** -0.5)
            worst = max(worst, attn_rel_err(row, ref))
    say(f"  worst rel err {worst:.2e}")
    assert worst <= min(ATTN_REL_TOL, 8e-3)


def test_prefill_confidence_rejects_a_short_max_seq_len(S):
    """max_seq_len below the mean sequence length (0 with tokens present
    included) is rejected before any launch."""
    sevo, di = S
    shape = synth.WORKLOADS["tiny_step"].shape
    pop = make_population([40, 30], seed=1)
    model = sevo.sevo_init_model(shape, di.device_weights(shape, 1), max_position=64)
    kvp = di.device_pools(shape, 1, pop.n_pages)
    toks = torch.zeros(70, dtype=torch.int32, device="cuda")
    ss = torch.tensor([0, 40, 70], dtype=torch.int32, device="cuda")
    pt = torch.from_numpy(pop.page_table.astype(np.int32)).cuda()
    rows = torch.arange(70, dtype=torch.int32, device="cuda")
    for bound in (0, 34):
        buf = sevo.PrefillBuffers(model, toks, ss, pt, kvp, rows, 20, bound)
        with pytest.raises(sevo.SevoError) as e:
            buf.run()
        assert e.value.status == sevo.INVALID_ARGUMENT and "max_seq_len" in str(e.value)
    sevo.PrefillBuffers(model, toks, ss, pt, kvp, rows, 20, 40).run()
    torch.cuda.synchronize()
    model.close()


def test_prefill_confidence_moe_chunk_keeps_gathered_rows_below_2gib(S):
    """A MoE model whose expert rows are wide (top-16 of 64 experts with FFN
    4096: 128 KB of SwiGLU rows per token) at 40000 tokens: the default chunk
    (65536 tokens, which would put 5.2 GB of gathered rows behind one 32-bit
    buffer descriptor) is lowered to 16368 tokens; every row's c and each C
    equal, bit for bit, the run in 4096-token chunks, and all are finite."""
    sevo, di = S
    shape = synth.ModelShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                             ffn=0, vocab=4096, n_experts=64, top_k=16, expert_ffn=4096)
    T = 40000
    say(f"prefill confidence MoE chunk bound: {T} tokens, top-16 of 64 experts x 4096")
    pop = make_population([T], seed=31)
    rng = np.random.default_rng(31)
    toks = torch.from_numpy(rng.integers(0, shape.vocab, size=T).astype(np.int32)).cuda()
    model = sevo.sevo_init_model(shape, di.device_weights(shape, 31), max_position=T + 1)
    kvp = di.device_pools(shape, 31, pop.n_pages)
    ss = torch.tensor([0, T], dtype=torch.int32, device="cuda")
    pt = torch.from_numpy(pop.page_table.astype(np.int32)).cuda()
    rows = torch.arange(T, dtype=torch.int32, device="cuda")
    out = []
    for chunk in (0, 4096):
        buf = sevo.PrefillBuffers(model, toks, ss, pt, kvp, rows, 20, T, moe_chunk=chunk)
        conf = buf.run()
        torch.cuda.synchronize()
        out.append((conf.cpu().numpy(), buf.out_row_conf[:T].cpu().numpy()))
        del buf
        torch.cuda.empty_cache()
    model.close()
    say(f"  C {out[0][0]} vs {out[1][0]}")
    assert np.isfinite(out[0][1]).all()
    np.testing.assert_array_equal(out[0][0], out[1][0])
    np.testing.assert_array_equal(out[0][1], out[1][1])
