"""GPU parity of each decode-step kernel against the CPU oracle, through the C ABI.

Sizes: small cases span several tiles and ragged tails; the attention and
sampler cases at the full workload sizes run in the same launch
configuration the benchmark uses and are checked on sampled candidates.
"""
import numpy as np
import pytest
import torch

from oracle import decoder as od
from oracle.bf16 import round_bf16
from paper_2604_07725_amd import synth
from tests.gpu_helpers import (ATTN_REL_TOL, attn_rel_err, bf16_bits, check_ids,
                               host_candidate_kv, make_population, pack_weight_host, poisoned, say,
                               tile_activations_host, to_np, untile_activations_host)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_07725_amd import device_inputs, sevo
    sevo.lib()
    return sevo, device_inputs


# ------------------------------------------------------------------ generator
@pytest.mark.parametrize("count,offset,std,mean", [(1000003, 0, 1.0, None),
                                                   (4096, 12345678901, 0.02, None),
                                                   (777, 5, 0.02, 1.0), (3, 0, 1.0, None)])
def test_device_fill_equals_host_generator(S, count, offset, std, mean):
    sevo, _ = S
    key = synth.tensor_key(9, 30, 4)
    say(f"fill count={count} offset={offset}")
    t = torch.empty(count, dtype=torch.bfloat16, device="cuda")
    sevo.sevo_fill_normal_bf16(t, key, offset, std, mean)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bf16_bits(t), synth.fill_bf16_bits(count, key, offset, std, mean))


# ------------------------------------------------------------------ KV layout
def _fused_from_plain(kp, vp):
    """Host form of the fused pool from plain pools [P][hkv][16][d] (uint16
    bit patterns), through the K and V tile offsets of the layout."""
    P, hkv, slots, d = kp.shape
    fused = np.zeros((P, hkv, 2, slots * d), np.uint16)
    s, e = np.meshgrid(np.arange(slots), np.arange(d), indexing="ij")
    fused[:, :, 0][:, :, od.k_tile_offset(s, e)] = kp
    fused[:, :, 1][:, :, od.v_tile_offset(s, e)] = vp
    return fused


@pytest.mark.parametrize("pages,hkv,d", [(1, 1, 64), (37, 2, 64), (37, 8, 128), (5000, 4, 128)])
def test_pack_kv_bit_exact(S, pages, hkv, d):
    """Plain K and V pools to the fused pool: every element moved bit for bit
    to its place in the K (32-dim blocks) and V (dim-major) tiles."""
    sevo, _ = S
    say(f"pack_kv pages={pages} hkv={hkv} d={d}")
    rng = np.random.default_rng([pages, hkv, d])
    kp = rng.integers(0, 1 << 16, size=(pages, hkv, 16, d), dtype=np.uint16)
    vp = rng.integers(0, 1 << 16, size=(pages, hkv, 16, d), dtype=np.uint16)
    kd = torch.from_numpy(kp.view(np.int16)).cuda().view(torch.bfloat16)
    vd = torch.from_numpy(vp.view(np.int16)).cuda().view(torch.bfloat16)
    out = torch.full((pages, hkv, 2, 16 * d), float("nan"), dtype=torch.bfloat16, device="cuda")
    sevo.sevo_pack_kv(kd, vd, out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bf16_bits(out), _fused_from_plain(kp, vp))


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (16, 2, 64)])
def test_attention_over_packed_plain_pools(S, hq, hkv, d):
    """A cache kept in the plain layout (separate K and V pools, slot-major
    rows), packed once, gives the oracle's attention over the candidates' keys."""
    sevo, _ = S
    lengths = [700, 1, 333, 1024, 65]
    pop = make_population(lengths, seed=hq + d)
    rng = np.random.default_rng([hq, hkv, d, 7])
    kp = round_bf16(rng.standard_normal((pop.n_pages, hkv, 16, d))).astype(np.float32)
    vp = round_bf16(rng.standard_normal((pop.n_pages, hkv, 16, d))).astype(np.float32)
    q = round_bf16(rng.standard_normal((pop.n, hq, d))).astype(np.float32)
    say(f"attention over packed plain pools hq={hq} hkv={hkv} d={d}")
    kd = torch.from_numpy(kp).to(torch.bfloat16).cuda()
    vd = torch.from_numpy(vp).to(torch.bfloat16).cuda()
    kv = sevo.sevo_pack_kv(kd, vd)
    out = sevo.sevo_attn_decode(torch.from_numpy(q).to(torch.bfloat16).cuda(), kv,
                                torch.from_numpy(pop.page_table).cuda(),
                                torch.from_numpy(pop.lengths).cuda())
    torch.cuda.synchronize()
    o = to_np(out)
    for i, n in enumerate(lengths):
        pages = pop.page_table[i, :(n + 15) // 16]
        K = kp[pages].transpose(1, 0, 2, 3).reshape(hkv, -1, d)[:, :n].astype(np.float64)
        V = vp[pages].transpose(1, 0, 2, 3).reshape(hkv, -1, d)[:, :n].astype(np.float64)
        ref = od.attention_dense(q[i].astype(np.float64), K, V, d ** -0.5)
        assert attn_rel_err(o[i], ref) <= min(ATTN_REL_TOL, 8e-3), i


# ------------------------------------------------------------------ attention
def _attn_case(S, shape, lengths, seed, num_splits=0, shuffle=True, pt_override=None):
    sevo, di = S
    pop = make_population(lengths, shuffle=shuffle, seed=seed)
    pt = pop.page_table if pt_override is None else pt_override
    kvp = di.device_pools(shape, seed, pop.n_pages, layers=[0])[0]
    q = di.device_q(shape, seed, pop.n)
    lens = torch.from_numpy(pop.lengths.astype(np.int32)).cuda()
    ptd = torch.from_numpy(pt.astype(np.int32)).cuda()
    ws = poisoned(sevo.sevo_attn_workspace_bytes(pop.n, shape.n_q_heads, shape.n_kv_heads,
                                                 shape.head_dim, pt.shape[1], num_splits))
    out = sevo.sevo_attn_decode(q, kvp, ptd, lens, num_splits=num_splits, workspace=ws)
    torch.cuda.synchronize()
    return pop, q, kvp, ptd, lens, out


def _oracle_attn(shape, seed, pop, i, n_keys=None):
    n_keys = int(pop.lengths[i]) if n_keys is None else n_keys
    qh = synth.host_values(synth.q_spec(shape, seed, pop.n)).reshape(pop.n, shape.n_q_heads,
                                                                      shape.head_dim)
    K, V = host_candidate_kv(shape, seed, 0, pop, i, n_keys, pop.n_pages)
    return od.attention_dense(qh[i], K, V, shape.head_dim ** -0.5)


ATTN_SMALL = [
    # (hq, hkv, d, lengths, splits)
    (4, 2, 64, [300, 256, 512, 401], 0),
    (32, 8, 128, [1, 15, 16, 17, 31, 33, 1000, 257], 0),
    (32, 8, 128, [1, 15, 16, 17, 31, 33, 1000, 257], 1),
    (32, 8, 128, [700, 2000, 64, 129], 7),
    (8, 8, 128, [100, 37], 0),
    (16, 8, 64, [90, 300], 3),
    (64, 8, 128, [500, 33], 0),
    (8, 1, 128, [1000, 5], 2),
    # 8 query heads per kv head: the matrix-core variant (every partial-page
    # count, split counts, both head sizes)
    (32, 4, 128, [1, 15, 16, 17, 31, 33, 1000, 257], 0),
    (32, 4, 128, [1, 15, 16, 17, 31, 33, 1000, 257], 1),
    (32, 4, 128, [700, 2000, 64, 129], 7),
    (16, 2, 64, [1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15, 16, 500], 0),
]


@pytest.mark.parametrize("hq,hkv,d,lengths,splits", ATTN_SMALL)
def test_attention_small_matches_oracle(S, hq, hkv, d, lengths, splits):
    shape = synth.ModelShape(1, 256, hq, hkv, d, 256, 256)
    say(f"attention hq={hq} hkv={hkv} d={d} lens={lengths} splits={splits}")
    pop, q, kvp, pt, lens, out = _attn_case(S, shape, lengths, seed=11, num_splits=splits)
    o = to_np(out)
    for i in range(pop.n):
        ref = _oracle_attn(shape, 11, pop, i)
        e = attn_rel_err(o[i], ref)
        assert e <= ATTN_REL_TOL, (i, e)
        # the bf16 output rounding alone is 2^-9 relative: the kernel is far tighter
        assert e <= 8e-3, (i, e)


@pytest.mark.parametrize("hq,hkv", [(32, 8), (32, 4)])
def test_attention_page_permutation_and_determinism_bit_exact(S, hq, hkv):
    sevo, di = S
    shape = synth.ModelShape(1, 256, hq, hkv, 128, 256, 256)
    lengths = [900, 33, 1600, 17]
    say("attention permutation / determinism")
    pop, q, kvp, pt, lens, out1 = _attn_case(S, shape, lengths, seed=5, shuffle=False)
    out2 = sevo.sevo_attn_decode(q, kvp, pt, lens)
    # physically permute the pages and the page table the same way
    perm = torch.randperm(pop.n_pages, generator=torch.Generator().manual_seed(3))
    kvp2 = torch.empty_like(kvp)
    kvp2[perm.cuda()] = kvp
    pt_np = pop.page_table.copy()
    pt_np[pt_np >= 0] = perm.numpy()[pt_np[pt_np >= 0]]
    out3 = sevo.sevo_attn_decode(q, kvp2, torch.from_numpy(pt_np).cuda(), lens)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bf16_bits(out1), bf16_bits(out2))
    np.testing.assert_array_equal(bf16_bits(out1), bf16_bits(out3))


@pytest.mark.parametrize("hq,hkv", [(32, 8), (32, 4)])
def test_attention_ignores_slots_past_the_last_key(S, hq, hkv):
    """Slots of a candidate's last page past its last key may hold anything:
    NaN patterns written there (K and V tiles, every kv head) leave the output
    bit-identical."""
    sevo, di = S
    d = 128
    shape = synth.ModelShape(1, 256, hq, hkv, d, 256, 256)
    lengths = [17, 5, 300, 31, 64]
    say(f"attention with NaN past the last key hq={hq} hkv={hkv}")
    pop, q, kvp, pt, lens, out1 = _attn_case(S, shape, lengths, seed=13)
    pool = kvp.view(torch.int16).cpu().numpy().copy()   # [P][hkv][2][16 d]
    e = np.arange(d)
    for i, n in enumerate(lengths):
        if n % 16 == 0:
            continue
        page = pop.page_table[i, n // 16]
        for slot in range(n % 16, 16):
            pool[page, :, 0, ((e // 32) * 16 + slot) * 32 + e % 32] = np.int16(0x7FC0)  # K
            pool[page, :, 1, e * 16 + slot] = np.int16(0x7FC0)                          # V
    kvp_nan = torch.from_numpy(pool).cuda().view(torch.bfloat16)
    out2 = sevo.sevo_attn_decode(q, kvp_nan, pt, lens)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bf16_bits(out1), bf16_bits(out2))
    assert np.isfinite(to_np(out2)).all()


@pytest.mark.parametrize("hq,hkv", [(32, 8), (32, 4)])
def test_attention_split_count_changes_only_rounding(S, hq, hkv):
    sevo, di = S
    shape = synth.ModelShape(1, 256, hq, hkv, 128, 256, 256)
    say("attention split counts")
    pop, q, kvp, pt, lens, out1 = _attn_case(S, shape, [3000, 2500, 100], seed=6,
                                             num_splits=1)
    for s in (2, 5, 16, 0):
        o = sevo.sevo_attn_decode(q, kvp, pt, lens, num_splits=s)
        torch.cuda.synchronize()
        d = np.abs(to_np(o) - to_np(out1)).max() / np.abs(to_np(out1)).max()
        assert d < 4e-3, (s, d)


@pytest.mark.parametrize("hq,hkv", [(16, 4), (32, 4)])
def test_attention_out_of_range_page_ids_are_skipped(S, hq, hkv):
    """A page id outside the pool contributes no keys and is never read."""
    sevo, di = S
    shape = synth.ModelShape(1, 256, hq, hkv, 128, 256, 256)
    lengths = [200, 100]
    pop = make_population(lengths, seed=8)
    bad = pop.page_table.copy()
    bad[0, 3] = pop.n_pages + 1000      # keys 48..63 of candidate 0
    bad[1, 0] = -7                      # keys 0..15 of candidate 1
    say("attention bad page ids")
    _, q, kvp, pt, lens, out = _attn_case(S, shape, lengths, seed=8, pt_override=bad)
    o = to_np(out)
    qh = synth.host_values(synth.q_spec(shape, 8, 2)).reshape(2, hq, 128)
    for i, drop in ((0, range(48, 64)), (1, range(0, 16))):
        K, V = host_candidate_kv(shape, 8, 0, pop, i, int(pop.lengths[i]), pop.n_pages)
        keep = np.array([t for t in range(int(pop.lengths[i])) if t not in drop])
        ref = od.attention_dense(qh[i], K[:, keep], V[:, keep], 128 ** -0.5)
        assert attn_rel_err(o[i], ref) <= 8e-3


@pytest.mark.parametrize("hq,hkv", [(32, 8), (32, 4)])
def test_attention_zero_length_candidate_gives_zero(S, hq, hkv):
    """A candidate with no cached keys yields o = 0 and never disturbs the others."""
    shape = synth.ModelShape(1, 256, hq, hkv, 128, 256, 256)
    say("attention with a zero-length candidate")
    pop, q, kvp, pt, lens, out = _attn_case(S, shape, [0, 40, 0, 300], seed=12)
    o = to_np(out)
    assert np.all(o[0] == 0) and np.all(o[2] == 0)
    for i in (1, 3):
        assert attn_rel_err(o[i], _oracle_attn(shape, 12, pop, i)) <= 8e-3


@pytest.mark.parametrize("workload,sample", [("attn_pop16_agg4", [0, 5, 11, 15]),
                                             ("dense8b_pop64_agg4", None),
                                             ("dense8b_pop16_agg8", None),
                                             ("moe30b_pop64_agg4", None)])
def test_attention_full_size_sampled(S, workload, sample):
    """Full-size pools and the benchmark's launch configuration (auto splits);
    the oracle checks sampled candidates (all heads), including the shortest
    and the longest context."""
    sevo, di = S
    w = synth.WORKLOADS[workload]
    shape = w.shape
    pop = synth.workload_population(w)
    say(f"attention full size {workload}: N={pop.n} pages={pop.n_pages}")
    kvp = di.device_pools(shape, w.seed, pop.n_pages, layers=[0])[0]
    q = di.device_q(shape, w.seed, pop.n)
    lens = torch.from_numpy(pop.lengths.astype(np.int32)).cuda()
    pt = torch.from_numpy(pop.page_table).cuda()
    out = sevo.sevo_attn_decode(q, kvp, pt, lens)
    torch.cuda.synchronize()
    o = to_np(out)
    if sample is None:
        sample = sorted({int(np.argmin(pop.lengths)), int(np.argmax(pop.lengths)), 7})
    qh = synth.host_values(synth.q_spec(shape, w.seed, pop.n)).reshape(pop.n, shape.n_q_heads,
                                                                      shape.head_dim)
    for i in sample:
        K, V = host_candidate_kv(shape, w.seed, 0, pop, i, int(pop.lengths[i]), pop.n_pages)
        ref = od.attention_dense(qh[i], K, V, shape.head_dim ** -0.5)
        e = attn_rel_err(o[i], ref)
        say(f"  candidate {i} len {pop.lengths[i]} rel err {e:.2e}")
        assert e <= ATTN_REL_TOL
        assert e <= 8e-3
    assert np.isfinite(o).all()


# ------------------------------------------------------------------ sampler
def _logits(n, vocab, ld, seed, std=1.28):
    key = synth.tensor_key(seed, 40)
    host = synth.fill_values(n * vocab, key, 0, std).reshape(n, vocab).astype(np.float32)
    dev = torch.zeros(n, ld, dtype=torch.float32, device="cuda")
    dev[:, :vocab] = torch.from_numpy(host).cuda()
    return host, dev


@pytest.mark.parametrize("n,vocab,ld,temp", [(64, 151936, 151936, 1.0), (64, 151936, 151936, 0.7),
                                             (16, 151936, 151936, 0.0), (4, 4093, 4096, 1.0),
                                             (3, 5, 8, 1.0), (2, 4096, 4096, 1.3)])
def test_logprob_sample_matches_oracle(S, n, vocab, ld, temp):
    sevo, _ = S
    say(f"sampler n={n} vocab={vocab} T={temp}")
    host, dev = _logits(n, vocab, ld, seed=vocab + n)
    seed = 0x1234_5678_9ABC
    uids = np.arange(n, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15) + np.uint64(17)
    pos = (np.arange(n) * 977 + 5).astype(np.int32)
    ids, lps = sevo.sevo_logprob_sample(dev[:, :vocab] if ld == vocab else dev.as_strided(
        (n, vocab), (ld, 1)), temp, seed, torch.from_numpy(uids.view(np.int64)).cuda(),
        torch.from_numpy(pos).cuda(), workspace=poisoned(sevo.sevo_sample_workspace_bytes(n, vocab)))
    torch.cuda.synchronize()
    det = {}
    rid, rlp, gaps = od.logprob_sample(host.astype(np.float64), temp, seed, uids, pos,
                                       details=det)
    err, n_exact = check_ids(ids.cpu().numpy(), lps.cpu().numpy(), rid, rlp, gaps, det,
                             label=f"T={temp}")
    say(f"  lp max err {err:.2e}, {n_exact}/{n} decisions with gap > 1e-3")
    assert (ids.cpu().numpy() >= 0).all() and (ids.cpu().numpy() < vocab).all()


def test_logprob_sample_is_keyed_by_uid_and_position(S):
    """Permuting the population permutes the draws (noise is not keyed by slot)."""
    sevo, _ = S
    host, dev = _logits(8, 4096, 4096, seed=3)
    uids = np.arange(8, dtype=np.int64) + 100
    pos = np.arange(8, dtype=np.int32) * 3
    a, la = sevo.sevo_logprob_sample(dev, 1.0, 7, torch.from_numpy(uids).cuda(),
                                     torch.from_numpy(pos).cuda())
    perm = np.array([3, 1, 7, 0, 2, 6, 5, 4])
    b, lb = sevo.sevo_logprob_sample(dev[perm], 1.0, 7, torch.from_numpy(uids[perm]).cuda(),
                                     torch.from_numpy(pos[perm]).cuda())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(a.cpu().numpy()[perm], b.cpu().numpy())
    np.testing.assert_array_equal(la.cpu().numpy()[perm], lb.cpu().numpy())


@pytest.mark.parametrize("n,vocab,ld,temp,k", [(64, 151936, 151936, 1.0, 20),
                                               (64, 151936, 151936, 0.7, 32),
                                               (16, 151936, 151936, 0.0, 1),
                                               (4, 4093, 4096, 1.3, 8), (3, 40, 40, 1.0, 32),
                                               (5, 9000, 9000, 1.0, 5)])
def test_self_confidence_matches_oracle(S, n, vocab, ld, temp, k):
    """Per-token confidence (Eq. 1) fused in the sampler, on identical logits:
    c = -(1/K) sum of the K largest log-probabilities at T = 1, whatever T;
    the running sum adds it; ids and log-probs are unchanged by it."""
    sevo, _ = S
    say(f"confidence n={n} vocab={vocab} T={temp} K={k}")
    host, dev = _logits(n, vocab, ld, 7)
    uid = torch.from_numpy(np.arange(n, dtype=np.int64) * 977 + 5).cuda()
    pos = torch.from_numpy(np.arange(n, dtype=np.int32) + 100).cuda()
    base = np.linspace(-1.0, 1.0, n).astype(np.float32)
    acc = torch.from_numpy(base.copy()).cuda()
    ids, lps, conf = sevo.sevo_logprob_sample(dev, temp, 31, uid, pos, vocab=vocab, conf_topk=k,
                                              conf_sum=acc)
    ids0, lps0 = sevo.sevo_logprob_sample(dev, temp, 31, uid, pos, vocab=vocab)
    torch.cuda.synchronize()
    ref = od.token_confidence(host.astype(np.float64), k)
    got = conf.cpu().numpy().astype(np.float64)
    err = np.abs(got - ref).max()
    say(f"  max |c - c_ref| {err:.2e} (c in [{ref.min():.3f}, {ref.max():.3f}])")
    assert err <= 2e-4
    np.testing.assert_allclose(acc.cpu().numpy(), base + conf.cpu().numpy(), rtol=0, atol=1e-6)
    np.testing.assert_array_equal(ids.cpu().numpy(), ids0.cpu().numpy())
    np.testing.assert_array_equal(lps.cpu().numpy(), lps0.cpu().numpy())


@pytest.mark.parametrize("n,vocab,ld,temp,top_k,top_p,min_p,conf", [
    (64, 151936, 151936, 0.7, 20, 0.8, 0.0, 0),     # instruct rows of the table
    (64, 151936, 151936, 0.6, 20, 0.95, 0.0, 20),   # thinking rows, with confidence
    (16, 151936, 151936, 1.0, 20, 0.95, 0.0, 0),
    (16, 151936, 151936, 0.0, 20, 0.8, 0.0, 0),     # greedy
    (8, 4093, 4096, 1.0, 32, 1.0, 0.1, 32),         # min-p
    (3, 40, 40, 1.3, 5, 0.5, 0.2, 3),
    (4, 9000, 9000, 2.0, 1, 1.0, 0.0, 0)])
def test_truncated_sampling_matches_oracle(S, n, vocab, ld, temp, top_k, top_p, min_p, conf):
    """Top-k with min-p and top-p inside the top-k set, on identical logits."""
    sevo, _ = S
    say(f"truncated sampling n={n} V={vocab} T={temp} k={top_k} p={top_p} min_p={min_p}")
    host, dev = _logits(n, vocab, ld, 11, std=2.0)
    uid = torch.from_numpy(np.arange(n, dtype=np.int64) * 7919 + 3).cuda()
    pos = torch.from_numpy(np.arange(n, dtype=np.int32) * 13 + 2).cuda()
    out = sevo.sevo_logprob_sample(dev, temp, 99, uid, pos, vocab=vocab, top_k=top_k,
                                   top_p=top_p, min_p=min_p, conf_topk=conf)
    torch.cuda.synchronize()
    ids, lps = out[0].cpu().numpy(), out[1].cpu().numpy()
    det = {}
    rid, rlp, gap = od.truncated_logprob_sample(host, temp, 99, np.arange(n) * 7919 + 3,
                                                np.arange(n) * 13 + 2, top_k, top_p, min_p,
                                                details=det)
    # ids exact where the gap among the kept entries exceeds 1e-3; a near tie
    # must pick a kept entry within 1e-3 of the largest perturbed value; lp of
    # the GPU's own token under the truncated distribution
    lp_err, n_exact = check_ids(ids, lps, rid, rlp, gap, det, label="truncated")
    say(f"  ids equal {np.mean(ids == rid):.3f}, lp err {lp_err:.2e}, {n_exact}/{n} exact")
    if conf:
        ref = od.token_confidence(host.astype(np.float64), conf)
        assert np.abs(out[2].cpu().numpy() - ref).max() <= 2e-4


def test_truncated_sampling_tied_logits_use_index_order(S):
    """Equal logits at the top-k boundary: the lower vocabulary indices are kept."""
    sevo, _ = S
    n, vocab = 2, 5000
    dev = torch.zeros(n, vocab, dtype=torch.float32, device="cuda")
    dev[:, 100:140] = 3.0            # 40 tied maxima: top-8 keeps indices 100..107
    uid = torch.arange(n, dtype=torch.int64, device="cuda") + 5
    seen = set()
    for seed in range(40):
        ids, lps = sevo.sevo_logprob_sample(dev, 1.0, seed, uid, torch.zeros(n, dtype=torch.int32,
                                                                             device="cuda"),
                                            top_k=8)
        seen |= set(ids.cpu().numpy().tolist())
        np.testing.assert_allclose(lps.cpu().numpy(), np.log(1 / 8), atol=1e-6)
    assert seen <= set(range(100, 108)) and len(seen) > 4


def test_self_confidence_ties_and_uniform(S):
    """Uniform logits give c = log V exactly; many equal maxima count once each."""
    sevo, _ = S
    n, vocab = 3, 10000
    dev = torch.zeros(n, vocab, dtype=torch.float32, device="cuda")
    dev[1, 123:163] = 2.5            # 40 tied maxima
    dev[2, ::1000] = 4.0             # 10 tied maxima, K = 16 also takes 6 zeros
    uid = torch.arange(n, dtype=torch.int64, device="cuda")
    pos = torch.zeros(n, dtype=torch.int32, device="cuda")
    _, _, conf = sevo.sevo_logprob_sample(dev, 1.0, 1, uid, pos, conf_topk=16)
    torch.cuda.synchronize()
    ref = od.token_confidence(dev.double().cpu().numpy(), 16)
    np.testing.assert_allclose(conf.cpu().numpy(), ref, rtol=0, atol=2e-5)
    assert abs(float(conf[0]) - np.log(vocab)) < 2e-5


def test_group_confidence_matches_oracle(S):
    sevo, _ = S
    rng = np.random.default_rng(3)
    n, M, K = 64, 16, 4
    csum = rng.uniform(1, 50, n).astype(np.float32)
    cnt = rng.integers(1, 500, n).astype(np.int32)
    groups = np.stack([rng.choice(n, K, replace=False) for _ in range(M)]).astype(np.int32)
    gc = sevo.sevo_group_confidence(torch.from_numpy(csum).cuda(), torch.from_numpy(cnt).cuda(),
                                    torch.from_numpy(groups).cuda())
    torch.cuda.synchronize()
    ref = od.group_confidence(od.candidate_confidence(csum, cnt), groups)
    np.testing.assert_allclose(gc.cpu().numpy(), ref, rtol=2e-6)


# ------------------------------------------------------------------ linear
LINEAR_CASES = [
    # m, n_out, k, mode, k_splits, x_tiled
    (4, 512, 256, 0, 0, 0), (4, 256, 256, 1, 0, 1), (4, 2048, 256, 2, 0, 0),
    (4, 256, 1024, 1, 0, 0), (17, 128, 1024, 0, 3, 1), (33, 192, 512, 1, 0, 0),
    (64, 256, 4096, 0, 1, 1), (64, 6144, 4096, 0, 0, 1), (64, 4096, 12288, 1, 0, 1),
    (64, 24576, 4096, 2, 0, 1), (16, 4096, 4096, 1, 0, 0), (100, 128, 256, 0, 2, 1),
    # k not a multiple of 128: per-wave step counts differ, short tails
    (5, 128, 96, 0, 0, 0), (20, 256, 160, 1, 0, 1), (3, 128, 32, 2, 0, 1), (40, 192, 352, 0, 2, 0),
    # m >= 256 with k % 64 == 0: the large-M kernel (256 x 256 tiles, 64-k
    # stages); one exact tile, ragged m and n tails, row-major X, prefill shapes
    (256, 256, 64, 0, 0, 1), (300, 320, 128, 0, 0, 1), (777, 448, 192, 1, 0, 0),
    (513, 640, 256, 2, 0, 1), (1024, 6144, 4096, 0, 0, 1), (1000, 4096, 12288, 1, 0, 1),
    (600, 2048, 1024, 2, 0, 0), (255, 128, 64, 0, 0, 1),
]


def _linear_inputs(sevo, m, n_out, k, mode):
    x = torch.empty(m, k, dtype=torch.bfloat16, device="cuda")
    w = torch.empty(n_out, k, dtype=torch.bfloat16, device="cuda")
    kx, kw = synth.tensor_key(m, 50, k), synth.tensor_key(n_out, 51, k)
    sevo.sevo_fill_normal_bf16(x, kx, 0, 1.0)
    sevo.sevo_fill_normal_bf16(w, kw, 0, 0.02)
    wp = sevo.sevo_pack_weight(w, sevo.PACK_GATE_UP if mode == 2 else sevo.PACK_PLAIN)
    xh = synth.host_values(synth.TensorSpec((m, k), kx, 1.0)).reshape(m, k)
    wh = synth.host_values(synth.TensorSpec((n_out, k), kw, 0.02)).reshape(n_out, k)
    return x, w, wp, xh, wh


@pytest.mark.parametrize("n_out,k,mode,xt", [(24576, 4096, 2, 1), (6144, 4096, 0, 0)])
def test_linear_large_m_full_size_sampled(S, n_out, k, mode, xt):
    """The large-M GEMM at the confidence engine's size (M = 40960 tokens: the
    whole tile grid and its XCD-aware order): gate/up + SwiGLU on tiled
    activations and the QKV store on row-major ones, on sampled rows against
    float64 products of those rows."""
    sevo, _ = S
    m = 40960
    say(f"linear full size m={m} n={n_out} k={k} mode={mode} x_tiled={xt}")
    x = torch.empty(m, k, dtype=torch.bfloat16, device="cuda")
    w = torch.empty(n_out, k, dtype=torch.bfloat16, device="cuda")
    kx, kw = synth.tensor_key(m, 53, k), synth.tensor_key(n_out, 54, k)
    sevo.sevo_fill_normal_bf16(x, kx, 0, 1.0)
    sevo.sevo_fill_normal_bf16(w, kw, 0, 0.02)
    wp = sevo.sevo_pack_weight(w, sevo.PACK_GATE_UP if mode == 2 else sevo.PACK_PLAIN)
    del w
    if xt:
        xb = tile_activations_host(bf16_bits(x).reshape(m, k))
        x = torch.from_numpy(xb.view(np.int16)).cuda().view(torch.bfloat16)
    out = sevo.sevo_linear(x, wp, mode=mode, x_tiled=bool(xt), m=m)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 255, 256, 12345, 20479, 40703, 40959])
    if mode == 2:
        got = to_np(out)[rows]
    else:
        got = out[torch.from_numpy(rows).cuda()].double().cpu().numpy()
    del x, wp, out
    torch.cuda.empty_cache()
    wh = synth.host_values(synth.TensorSpec((n_out, k), kw, 0.02)).reshape(n_out, k)
    xspec = synth.TensorSpec((m, k), kx, 1.0)
    xh = np.stack([synth.host_values(xspec, offset=int(r) * k, count=k) for r in rows])
    y = xh.astype(np.float64) @ wh.astype(np.float64).T
    if mode == 2:
        F = n_out // 2
        ref = od.silu(y[:, :F]) * y[:, F:]
        assert np.all(np.abs(got - ref) <= 2 ** -8 * np.abs(ref) + 1e-4 * np.abs(ref).max())
    else:
        scale = np.sqrt(k) * 0.02
        np.testing.assert_allclose(got, y, rtol=0, atol=2e-5 * scale + 1e-6 * np.abs(y).max())


@pytest.mark.parametrize("m,n_out,k,mode,ks,xt", LINEAR_CASES)
def test_linear_matches_float64_matmul(S, m, n_out, k, mode, ks, xt):
    sevo, _ = S
    say(f"linear m={m} n={n_out} k={k} mode={mode} ks={ks} x_tiled={xt}")
    x, _, wp, xh, wh = _linear_inputs(sevo, m, n_out, k, mode)
    if xt:
        xb = tile_activations_host(bf16_bits(x).reshape(m, k))
        x = torch.from_numpy(xb.view(np.int16)).cuda().view(torch.bfloat16)
    kw = dict(k_splits=ks, x_tiled=bool(xt), m=m)
    y = xh.astype(np.float64) @ wh.astype(np.float64).T
    if mode == 2:
        out = sevo.sevo_linear(x, wp, mode=2, **kw)
        torch.cuda.synchronize()
        F = n_out // 2
        ref = od.silu(y[:, :F]) * y[:, F:]
        got = to_np(out)
        # one bf16 rounding of the product plus fp32 accumulation error
        assert np.all(np.abs(got - ref) <= 2 ** -8 * np.abs(ref) + 1e-4 * np.abs(ref).max())
        return
    if mode == 1:
        base = synth.host_values(synth.TensorSpec((m, n_out), synth.tensor_key(1, 52), 1.0))
        base = base.reshape(m, n_out).astype(np.float32)
        out = torch.from_numpy(base.copy()).cuda()
        sevo.sevo_linear(x, wp, mode=1, out=out, **kw)
        ref = base.astype(np.float64) + y
    else:
        out = sevo.sevo_linear(x, wp, mode=0, **kw)
        ref = y
    torch.cuda.synchronize()
    got = out.double().cpu().numpy()
    scale = np.sqrt(k) * 0.02
    np.testing.assert_allclose(got, ref, rtol=0, atol=2e-5 * scale + 1e-6 * np.abs(ref).max())


# one shape per instantiated skinny kernel: (M tile rows, 16-row weight blocks
# per workgroup, SwiGLU pairs or not), found by running the planner over n_out;
# every one leaves a ragged last workgroup (row blocks past the matrix)
ROW_BLOCK_CASES = [
    # m, n_out, mode, row blocks the plan must pick
    (16, 128, 0, 2), (16, 128, 2, 2), (16, 8256, 0, 3), (16, 12352, 0, 4), (16, 8320, 2, 4),
    (16, 16448, 0, 5), (16, 20544, 0, 6), (16, 16512, 2, 6), (16, 24640, 0, 8),
    (16, 24704, 2, 8), (16, 32832, 0, 10), (16, 32896, 2, 10), (16, 41024, 0, 12),
    (16, 41088, 2, 12), (16, 49216, 0, 14), (16, 49280, 2, 14), (16, 57408, 0, 16),
    (16, 57472, 2, 16),
    (24, 128, 0, 2), (24, 128, 2, 2), (24, 8256, 0, 3), (24, 12352, 0, 4), (24, 8320, 2, 4),
    (24, 16448, 0, 5), (24, 20544, 0, 6), (24, 16512, 2, 6), (24, 24640, 0, 8),
    (24, 24704, 2, 8), (24, 32832, 0, 10), (24, 32896, 2, 10), (24, 41024, 0, 12),
    (24, 41088, 2, 12),
    (64, 128, 0, 3), (64, 12352, 0, 4), (64, 128, 2, 4), (64, 16448, 0, 5), (64, 20544, 0, 6),
    (64, 16512, 2, 6), (64, 24640, 0, 8), (64, 24704, 2, 8),
]


@pytest.mark.parametrize("m,n_out,mode,rb", ROW_BLOCK_CASES)
def test_linear_every_row_block_kernel(S, m, n_out, mode, rb):
    """Each (M tile, row blocks, epilogue) instance of the skinny kernel against
    a float64 product, every output column (k = 256, one split); every third
    case takes a row-major X."""
    sevo, _ = S
    k = 256
    assert sevo.sevo_linear_plan(m, n_out, k, 0, mode)[2] == rb
    xt = ROW_BLOCK_CASES.index((m, n_out, mode, rb)) % 3 != 0
    say(f"linear row blocks {rb} m={m} n={n_out} mode={mode} x_tiled={xt}")
    x, _, wp, xh, wh = _linear_inputs(sevo, m, n_out, k, mode)
    if xt:
        xb = tile_activations_host(bf16_bits(x).reshape(m, k))
        x = torch.from_numpy(xb.view(np.int16)).cuda().view(torch.bfloat16)
    out = sevo.sevo_linear(x, wp, mode=mode, x_tiled=xt, m=m)
    torch.cuda.synchronize()
    y = xh.astype(np.float64) @ wh.astype(np.float64).T
    if mode == 2:
        F = n_out // 2
        ref = od.silu(y[:, :F]) * y[:, F:]
        got = to_np(out)
        assert np.all(np.abs(got - ref) <= 2 ** -8 * np.abs(ref) + 1e-4 * np.abs(ref).max())
    else:
        got = out.double().cpu().numpy()
        np.testing.assert_allclose(got, y, rtol=0, atol=2e-5 * np.sqrt(k) * 0.02 + 1e-6 * np.abs(y).max())


@pytest.mark.parametrize("n_out,k,gate_up", [(64, 32, False), (192, 160, False),
                                             (4096, 4096, False), (256, 96, True),
                                             (24576, 4096, True)])
def test_pack_weight_bit_exact(S, n_out, k, gate_up):
    sevo, _ = S
    say(f"pack n={n_out} k={k} gate_up={gate_up}")
    w = torch.empty(n_out, k, dtype=torch.bfloat16, device="cuda")
    kw = synth.tensor_key(n_out, 53, k)
    sevo.sevo_fill_normal_bf16(w, kw, 0, 0.02)
    wp = sevo.sevo_pack_weight(w, sevo.PACK_GATE_UP if gate_up else sevo.PACK_PLAIN)
    wh = synth.host_values(synth.TensorSpec((n_out, k), kw, 0.02)).reshape(n_out, k)
    torch.cuda.synchronize()
    # bf16 bit patterns (the host values are exactly representable in bf16)
    bits = (np.ascontiguousarray(wh, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    np.testing.assert_array_equal(bf16_bits(wp).reshape(n_out, k), pack_weight_host(bits, gate_up))


@pytest.mark.parametrize("m", [37, 600])
def test_swiglu_tiled_output_and_tiled_chain(S, m):
    """SwiGLU written in the tiled layout equals the row-major result, and feeds
    the next projection as a tiled input (the decode step's FFN chain; m = 600
    takes the large-M kernel)."""
    sevo, _ = S
    F2, H = 512, 256
    say(f"swiglu tiled chain m={m}")
    x, _, wp, _, _ = _linear_inputs(sevo, m, F2, H, 2)
    a_row = sevo.sevo_linear(x, wp, mode=2)
    a_til = sevo.sevo_linear(x, wp, mode=2, out_tiled=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(untile_activations_host(bf16_bits(a_til), m, F2 // 2),
                                  bf16_bits(a_row))
    wd = torch.empty(H, F2 // 2, dtype=torch.bfloat16, device="cuda")
    sevo.sevo_fill_normal_bf16(wd, synth.tensor_key(9, 54), 0, 0.02)
    wdp = sevo.sevo_pack_weight(wd)
    y_row = sevo.sevo_linear(a_row, wdp, mode=0, k_splits=1)
    y_til = sevo.sevo_linear(a_til, wdp, mode=0, k_splits=1, x_tiled=True, m=m)
    torch.cuda.synchronize()
    # same operands, same kernel schedule: identical sums
    np.testing.assert_array_equal(y_row.cpu().numpy(), y_til.cpu().numpy())


# ------------------------------------------------------------------ norm / embed / rope
@pytest.mark.parametrize("rows,cols,n_part", [(600, 4096, 1), (600, 2048, 1), (530, 5120, 1),
                                                (600, 4096, 0), (100, 4096, 3), (37, 256, 16)])
def test_add_rmsnorm_matches_oracle_and_forms_agree(S, rows, cols, n_part):
    """Residual update + RMSNorm: x written back equal to the fp32 sum in
    partial order, the normed rows against the oracle; from 512 rows with at
    most one partial the many-row form runs, and the same rows in slices of
    192 (the 1024-thread form) must give identical bits."""
    sevo, _ = S
    say(f"add_rmsnorm rows={rows} cols={cols} partials={n_part}")
    g = torch.Generator(device="cuda")
    g.manual_seed(rows * 7 + cols + n_part)
    x0 = torch.randn(rows, cols, device="cuda", generator=g) * 2.0
    parts = (torch.randn(n_part, rows, cols, device="cuda", generator=g) if n_part else None)
    gain = (1.0 + 0.02 * torch.randn(cols, device="cuda", generator=g)).to(torch.bfloat16)
    x = x0.clone()
    out = sevo.sevo_add_rmsnorm(x, parts, gain, 1e-6)
    torch.cuda.synchronize()
    ref_x = x0.cpu().numpy()
    for s_ in range(n_part):
        ref_x = ref_x + parts[s_].cpu().numpy()        # float32, in partial order
    np.testing.assert_array_equal(x.cpu().numpy(), ref_x)
    got = untile_activations_host(to_np(out), rows, cols)
    ref = od.rms_norm(ref_x.astype(np.float64), to_np(gain), 1e-6)
    assert np.all(np.abs(got - ref) <= 2 ** -8 * np.abs(ref) + 1e-6)
    if rows >= 512 and n_part <= 1:
        xb = x0.clone()
        outb = torch.zeros_like(out)
        for a in range(0, rows, 192):
            b = min(rows, a + 192)
            pb = parts[:, a:b].contiguous() if n_part else None
            nb = -(-(b - a) // 16) * 16 * cols
            sevo.sevo_add_rmsnorm(xb[a:b], pb, gain, 1e-6, out=outb[a * cols:a * cols + nb])
        torch.cuda.synchronize()
        assert torch.equal(x, xb)
        assert torch.equal(out.view(torch.int16), outb.view(torch.int16))


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (64, 8, 128), (4, 2, 64)])
def test_qk_norm_rope_append_forms_agree(S, hq, hkv, d):
    """The per-token form of QK-norm + RoPE + append (from 256 tokens) against
    the per-(token, head) form (the same tokens in calls of 100): q and the
    whole KV pool identical bit for bit, and every appended slot written."""
    sevo, di = S
    say(f"qk_norm_rope_append forms {hq}/{hkv}x{d}")
    shape = synth.ModelShape(1, 512, hq, hkv, d, 256, 256)
    n = 300
    lens = np.random.default_rng(3).integers(1, 200, size=n)
    pop = make_population(lens, shuffle=True, seed=4, extra=1)
    model = sevo.sevo_init_model(shape, di.device_weights(shape, 5), max_position=256)
    g = torch.Generator(device="cuda")
    g.manual_seed(hq + d)
    qkv = torch.randn(n, (hq + 2 * hkv) * d, device="cuda", generator=g)
    pos = torch.from_numpy(pop.lengths.astype(np.int32)).cuda()
    pt = torch.from_numpy(pop.page_table).cuda()
    pool0 = torch.full((pop.n_pages, hkv, 2, 16 * d), float("nan"), dtype=torch.bfloat16,
                       device="cuda")
    pool_a = pool0.clone()
    q_a = sevo.sevo_qk_norm_rope_append(model, 0, qkv, pos, pt, pool_a)
    pool_b = pool0.clone()
    q_b = torch.empty_like(q_a)
    for a in range(0, n, 100):
        b = min(n, a + 100)
        sevo.sevo_qk_norm_rope_append(model, 0, qkv[a:b], pos[a:b], pt[a:b], pool_b, q_out=q_b[a:b])
    torch.cuda.synchronize()
    model.close()
    assert torch.isfinite(q_a.float()).all()
    assert torch.equal(q_a.view(torch.int16), q_b.view(torch.int16))
    assert torch.equal(pool_a.view(torch.int16), pool_b.view(torch.int16))
    # each token's slot: finite K and V in its page, the rest of the pool untouched
    written = int(torch.isfinite(pool_a.float()).sum())
    assert written == n * hkv * 2 * d


def test_rmsnorm_and_embed_match_oracle(S):
    sevo, _ = S
    say("rmsnorm / embed")
    V, H, n = 1000, 4096, 64
    emb = torch.empty(V, H, dtype=torch.bfloat16, device="cuda")
    ke = synth.tensor_key(2, 60)
    sevo.sevo_fill_normal_bf16(emb, ke, 0, 0.5)
    toks = np.array(list(range(0, V, 16))[:n], np.int32)
    toks[3] = V + 5            # out of range -> zero row
    x = sevo.sevo_embed(emb, torch.from_numpy(toks).cuda())
    eh = synth.host_values(synth.TensorSpec((V, H), ke, 0.5)).reshape(V, H)
    torch.cuda.synchronize()
    xr = eh[np.clip(toks, 0, V - 1)].astype(np.float64)
    xr[3] = 0.0
    np.testing.assert_array_equal(x.double().cpu().numpy(), xr)
    xs = (x * 7.5 + 0.25).contiguous()
    g = torch.empty(H, dtype=torch.bfloat16, device="cuda")
    kg = synth.tensor_key(2, 61)
    sevo.sevo_fill_normal_bf16(g, kg, 0, 0.02, 1.0)
    h = sevo.sevo_rmsnorm(xs, g, 1e-6)
    torch.cuda.synchronize()
    gh = synth.host_values(synth.TensorSpec((H,), kg, 0.02, 1.0)).astype(np.float64)
    ref = od.rms_norm(xs.double().cpu().numpy(), gh, 1e-6)
    got = to_np(h)
    assert np.all(np.abs(got - ref) <= 2 ** -8 * np.abs(ref) + 1e-6)
    # mostly equal to the oracle's own bf16 rounding of the same value
    assert np.mean(got == round_bf16(ref)) > 0.99


# ------------------------------------------------------------------ read probe
@pytest.mark.parametrize("grid", [1, 7, 256, 4096])
def test_read_probe_reads_every_byte_once(S, grid):
    """The streaming-read microbenchmark reads each 16-byte word exactly once:
    the XOR of its per-workgroup words equals the XOR of the whole buffer
    (sequential), of all pages (a permutation) and of the listed pages only
    (ids outside the buffer skipped)."""
    sevo, di = S
    n_pages = 77
    rng = np.random.default_rng(grid)
    host = rng.integers(0, 2 ** 32, size=(n_pages, 512, 4), dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(grid * 16, dtype=torch.uint8, device="cuda")

    def xor_sink():
        torch.cuda.synchronize()
        return np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32).reshape(grid, 4), axis=0)

    whole = np.bitwise_xor.reduce(host.reshape(-1, 4), axis=0)
    sevo.sevo_hbm_read_probe(buf, None, grid, sink)
    np.testing.assert_array_equal(xor_sink(), whole)
    order = rng.permutation(n_pages).astype(np.int32)
    sevo.sevo_hbm_read_probe(buf, torch.from_numpy(order).cuda(), grid, sink)
    np.testing.assert_array_equal(xor_sink(), whole)
    order[[3, 40]] = [-1, n_pages + 5]     # two pages skipped
    sevo.sevo_hbm_read_probe(buf, torch.from_numpy(order).cuda(), grid, sink)
    listed = order[(order >= 0) & (order < n_pages)]
    np.testing.assert_array_equal(
        xor_sink(), np.bitwise_xor.reduce(host[listed].reshape(-1, 4), axis=0))
