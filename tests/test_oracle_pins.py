"""Pins of the CPU oracle against things other than itself (CPU only).

Each test ties one oracle function to a closed form, an invariant, a library
routine it reduces to, or brute force on tiny inputs, chosen so that a
plausible slip (dropped term, wrong sign or index, transposed operand) fails.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import decoder as od
from oracle.philox import philox4x32_10, sampler_bits, uniform01, gumbel_noise

RNG = np.random.default_rng(1234)


# ---------------------------------------------------------------- bf16 storage
def test_bf16_matches_torch_conversion():
    x = np.concatenate([RNG.standard_normal(20000) * s for s in (1e-3, 1.0, 37.0, 1e4)])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.round_bf16(x), ref)


def test_bf16_ties_to_even_by_hand():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to the even mantissa (1)
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: ties to 1 + 2^-6
    vals = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20, -(1 + 2 ** -8)])
    want = np.array([1.0, 1 + 2 ** -6, 1 + 2 ** -7, -1.0])
    np.testing.assert_array_equal(oracle.round_bf16(vals), want)


# ---------------------------------------------------------------- Philox / noise
def _philox_bigint(ctr, key):
    """Independent scalar Philox4x32-10 on Python ints (published definition)."""
    c = list(ctr)
    k0, k1 = key
    mask = 0xFFFFFFFF
    for r in range(10):
        if r:
            k0 = (k0 + 0x9E3779B9) & mask
            k1 = (k1 + 0xBB67AE85) & mask
        p0 = 0xD2511F53 * c[0]
        p1 = 0xCD9E8D57 * c[2]
        c = [((p1 >> 32) ^ c[1] ^ k0) & mask, p1 & mask, ((p0 >> 32) ^ c[3] ^ k1) & mask,
             p0 & mask]
    return c


def test_philox_vectorised_equals_bigint():
    ctrs = RNG.integers(0, 2 ** 32, size=(200, 4), dtype=np.uint64)
    keys = RNG.integers(0, 2 ** 32, size=(200, 2), dtype=np.uint64)
    ctrs[0] = [0xFFFFFFFF] * 4
    keys[0] = [0xFFFFFFFF] * 2
    ctrs[1] = [0] * 4
    keys[1] = [0] * 2
    out = philox4x32_10(ctrs[:, 0], ctrs[:, 1], ctrs[:, 2], ctrs[:, 3], keys[:, 0], keys[:, 1])
    for i in range(200):
        want = _philox_bigint([int(v) for v in ctrs[i]], (int(keys[i, 0]), int(keys[i, 1])))
        assert [int(o[i]) for o in out] == want


def test_uniform_is_exact_fp32_and_open_interval():
    b = np.array([0, 511, 512, 0xFFFFFFFF, 0x80000000], np.uint64)
    u = uniform01(b)
    assert u[0] == 0.5 * 2 ** -23 and u[1] == u[0]
    assert u[2] == 1.5 * 2 ** -23
    assert u[3] == 1 - 0.5 * 2 ** -23 and u[3] < 1.0
    assert np.all(u.astype(np.float32).astype(np.float64) == u)


def test_philox_uniformity_and_independence():
    v = np.arange(1 << 18, dtype=np.uint64)
    bits = sampler_bits(v, position=12345, uid=0xDEADBEEF12345, seed=77)
    u = uniform01(bits)
    # chi-square over 256 bins (df = 255): mean 255, sd ~22.6; 6 sd bound
    counts = np.bincount((u * 256).astype(np.int64), minlength=256)
    expected = len(u) / 256
    chi2 = float(((counts - expected) ** 2 / expected).sum())
    assert chi2 < 255 + 6 * math.sqrt(2 * 255), chi2
    # the four words of one Philox call and neighbouring counters are uncorrelated
    corr = np.corrcoef(u[:-1], u[1:])[0, 1]
    assert abs(corr) < 6 / math.sqrt(len(u))
    # each bit position is fair
    for k in (0, 9, 17, 31):
        frac = float(((bits >> np.uint64(k)) & np.uint64(1)).mean())
        assert abs(frac - 0.5) < 6 * 0.5 / math.sqrt(len(u))


def test_gumbel_moments_closed_form():
    # Standard Gumbel: mean = Euler-Mascheroni gamma, variance = pi^2 / 6
    g = np.concatenate([gumbel_noise(1 << 16, p, uid=99, seed=5) for p in range(8)])
    n = len(g)
    assert abs(g.mean() - 0.5772156649) < 6 * math.sqrt(math.pi ** 2 / 6 / n)
    assert abs(g.var() - math.pi ** 2 / 6) < 0.05


def test_noise_keyed_by_uid_and_position_not_order():
    a = gumbel_noise(64, 7, uid=11, seed=3)
    b = gumbel_noise(64, 8, uid=11, seed=3)
    c = gumbel_noise(64, 7, uid=12, seed=3)
    d = gumbel_noise(64, 7, uid=11, seed=4)
    assert not np.allclose(a, b) and not np.allclose(a, c) and not np.allclose(a, d)
    np.testing.assert_array_equal(a, gumbel_noise(64, 7, uid=11, seed=3))


# ---------------------------------------------------------------- sampler
def test_gumbel_max_with_zero_noise_is_argmax_lowest_tie():
    logits = np.array([[0.5, 2.0, 2.0, -1.0], [3.0, -1.0, 3.0, 3.0], [-5, -5, -5, -4.5]])
    ids, lps, _ = od.logprob_sample(logits, 1.0, 0, [0, 0, 0], [0, 0, 0],
                                    noise=np.zeros_like(logits))
    assert ids.tolist() == [1, 0, 3]
    ref = torch.log_softmax(torch.from_numpy(logits), dim=-1).numpy()
    np.testing.assert_allclose(lps, ref[np.arange(3), ids], rtol=0, atol=1e-14)


def test_greedy_temperature_zero():
    logits = RNG.standard_normal((5, 50))
    ids, lps, _ = od.logprob_sample(logits, 0.0, 1, np.arange(5), np.arange(5))
    np.testing.assert_array_equal(ids, logits.argmax(axis=1))
    ref = torch.log_softmax(torch.from_numpy(logits), dim=-1).numpy()
    np.testing.assert_allclose(lps, ref[np.arange(5), ids], atol=1e-14)


def test_gumbel_max_frequencies_equal_softmax():
    """Gumbel-max with the Philox noise samples softmax(logits / T) exactly."""
    V, T = 8, 0.7
    logits = np.array([1.0, 0.0, -0.5, 2.0, 0.3, -2.0, 1.5, 0.9])
    p = torch.softmax(torch.tensor(logits / T), 0).numpy()
    n = 200000
    pos = np.arange(n)
    # one Philox call gives 4 words, so V=8 -> counters (0|1, pos, uid, 0)
    v = np.arange(V, dtype=np.uint64)
    k0, k1 = np.uint64(31), np.uint64(0)
    out = [philox4x32_10(np.uint64(c), pos.astype(np.uint64), np.uint64(5), np.uint64(0), k0, k1)
           for c in (0, 1)]
    words = np.stack([out[int(vi) >> 2][int(vi) & 3] for vi in v], axis=1)   # [n, V]
    G = -np.log(-np.log(uniform01(words)))
    ids = np.argmax(logits / T + G, axis=1)
    # the same draws through logprob_sample (spot check of its noise path)
    ids_ls, _, _ = od.logprob_sample(np.tile(logits, (16, 1)), T, 31, [5] * 16, pos[:16])
    np.testing.assert_array_equal(ids_ls, ids[:16])
    counts = np.bincount(ids, minlength=V)
    chi2 = float(((counts - n * p) ** 2 / (n * p)).sum())
    assert chi2 < 7 + 6 * math.sqrt(14), (chi2, counts / n, p)


def test_temperature_scaling_consistency():
    logits = RNG.standard_normal((3, 40)) * 3
    a = od.logprob_sample(logits, 2.0, 9, [1, 2, 3], [4, 5, 6])
    b = od.logprob_sample(logits / 2.0, 1.0, 9, [1, 2, 3], [4, 5, 6])
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_allclose(a[1], b[1], atol=1e-13)


def test_log_softmax_matches_torch_and_normalises():
    z = RNG.standard_normal((4, 1000)) * 5
    lp = od.log_softmax(z)
    np.testing.assert_allclose(lp, torch.log_softmax(torch.from_numpy(z), -1).numpy(),
                               atol=1e-12)
    np.testing.assert_allclose(np.log(np.exp(lp).sum(-1)), 0.0, atol=1e-12)


# ---------------------------------------------------------------- RMSNorm, RoPE, SiLU
def test_rms_norm_unit_gain_and_torch():
    x = RNG.standard_normal((6, 256)) * 4
    y = od.rms_norm(x, np.ones(256), 1e-6)
    np.testing.assert_allclose(np.sqrt((y ** 2).mean(-1)), 1.0, rtol=1e-6)
    g = 1 + 0.1 * RNG.standard_normal(256)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (256,), torch.from_numpy(g), 1e-6)
    np.testing.assert_allclose(od.rms_norm(x, g, 1e-6), ref.numpy(), rtol=1e-12)


def test_silu_matches_torch():
    z = RNG.standard_normal(1000) * 6
    np.testing.assert_allclose(od.silu(z), torch.nn.functional.silu(torch.from_numpy(z)).numpy(),
                               rtol=1e-13)


def test_rope_identity_at_zero_and_pair_norms():
    u = RNG.standard_normal((3, 64))
    np.testing.assert_array_equal(od.rope_rotate(u, 0, 1e6), u)
    r = od.rope_rotate(u, 777, 1e6)
    np.testing.assert_allclose(r[:, :32] ** 2 + r[:, 32:] ** 2, u[:, :32] ** 2 + u[:, 32:] ** 2,
                               rtol=1e-12)


def test_rope_relative_position():
    q = RNG.standard_normal(128)
    k = RNG.standard_normal(128)
    for m, n in [(3, 10), (1000, 65000), (5, 5)]:
        lhs = od.rope_rotate(q, m, 1e6) @ od.rope_rotate(k, n, 1e6)
        rhs = q @ od.rope_rotate(k, n - m, 1e6)
        assert abs(lhs - rhs) < 1e-9 * (1 + abs(lhs))


def test_rope_equals_complex_rotation():
    """Rotate-half RoPE = multiplying z_m = u_m + i u_{m+d/2} by e^{i p theta^(-2m/d)}."""
    d, p, theta = 64, 4242, 1e6
    u = RNG.standard_normal(d)
    z = u[: d // 2] + 1j * u[d // 2:]
    ang = p * theta ** (-2.0 * np.arange(d // 2) / d)
    w = z * np.exp(1j * ang)
    np.testing.assert_allclose(od.rope_rotate(u, p, theta), np.concatenate([w.real, w.imag]),
                               atol=1e-12)


def test_rope_per_candidate_positions_broadcast():
    u = RNG.standard_normal((3, 4, 16))
    pos = np.array([0, 5, 900])
    r = od.rope_rotate(u, pos[:, None], 1e4)
    for i in range(3):
        np.testing.assert_allclose(r[i], od.rope_rotate(u[i], pos[i], 1e4), atol=0)


# ---------------------------------------------------------------- attention
def _sdpa(q, K, V, scale):
    """torch SDPA (float64) as the library special case; q [hq,d], K/V [hkv,L,d]."""
    hq, hkv = q.shape[0], K.shape[0]
    g = hq // hkv
    Kr = torch.from_numpy(K).repeat_interleave(g, dim=0)
    Vr = torch.from_numpy(V).repeat_interleave(g, dim=0)
    o = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[:, None, :], Kr, Vr, scale=scale)
    return o[:, 0, :].numpy()


@pytest.mark.parametrize("hq,hkv,L,d", [(4, 2, 37, 64), (32, 8, 300, 128), (8, 8, 5, 16),
                                        (64, 8, 100, 128), (6, 1, 17, 8)])
def test_attention_matches_sdpa(hq, hkv, L, d):
    q = RNG.standard_normal((hq, d))
    K = RNG.standard_normal((hkv, L, d))
    V = RNG.standard_normal((hkv, L, d))
    np.testing.assert_allclose(od.attention_dense(q, K, V, d ** -0.5), _sdpa(q, K, V, d ** -0.5),
                               atol=1e-12)


def test_attention_brute_force_loops():
    hq, hkv, L, d = 4, 2, 6, 8
    q = RNG.standard_normal((hq, d))
    K = RNG.standard_normal((hkv, L, d))
    V = RNG.standard_normal((hkv, L, d))
    out = od.attention_dense(q, K, V, 0.3)
    for j in range(hq):
        c = j // 2
        s = [sum(q[j, e] * K[c, t, e] for e in range(d)) * 0.3 for t in range(L)]
        w = [math.exp(x) for x in s]
        tot = sum(w)
        for e in range(d):
            assert abs(out[j, e] - sum(w[t] * V[c, t, e] for t in range(L)) / tot) < 1e-12


def test_attention_special_cases():
    d = 16
    V = RNG.standard_normal((2, 9, d))
    K = RNG.standard_normal((2, 9, d))
    q = RNG.standard_normal((4, d))
    # single key returns V
    o = od.attention_dense(q, K[:, :1], V[:, :1], 0.25)
    np.testing.assert_allclose(o, np.repeat(V[:, 0], 2, axis=0), atol=0)
    # all-equal scores (q = 0) return the mean of V
    o = od.attention_dense(np.zeros((4, d)), K, V, 0.25)
    np.testing.assert_allclose(o, np.repeat(V.mean(axis=1), 2, axis=0), atol=1e-14)
    # one dominant key returns its value
    K2 = K.copy()
    K2[:, 4] = 1e3 * q[::2] / np.linalg.norm(q[::2], axis=1, keepdims=True)
    o = od.attention_dense(q[::2].repeat(2, axis=0), K2, V, 1.0)
    np.testing.assert_allclose(o, np.repeat(V[:, 4], 2, axis=0), atol=1e-10)


def test_attention_rows_sum_to_one_and_shift_invariant():
    d = 32
    q = RNG.standard_normal((2, d))
    K = RNG.standard_normal((1, 50, d))
    ones = np.ones((1, 50, d))
    np.testing.assert_allclose(od.attention_dense(q, K, ones, 0.2), 1.0, atol=1e-14)
    # adding a constant vector to all keys along q shifts every score equally
    Kp = K + 3.0 * q[0][None, None, :]
    V = RNG.standard_normal((1, 50, d))
    np.testing.assert_allclose(od.attention_dense(q[:1], Kp, V, 0.2),
                               od.attention_dense(q[:1], K, V, 0.2), atol=1e-12)


def test_gqa_with_equal_heads_is_mha():
    d, L = 32, 40
    q = RNG.standard_normal((4, d))
    K = RNG.standard_normal((4, L, d))
    V = RNG.standard_normal((4, L, d))
    o = od.attention_dense(q, K, V, d ** -0.5)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[:, None], torch.from_numpy(K), torch.from_numpy(V), scale=d ** -0.5)
    np.testing.assert_allclose(o, ref[:, 0].numpy(), atol=1e-12)
    # GQA equals MHA on repeat_interleave'd K, V
    K2, V2 = K[:2], V[:2]
    np.testing.assert_allclose(od.attention_dense(q, K2, V2, 0.1),
                               od.attention_dense(q, np.repeat(K2, 2, 0), np.repeat(V2, 2, 0), 0.1),
                               atol=0)


@pytest.mark.parametrize("L,S", [(1, 1), (17, 4), (300, 1), (300, 7), (300, 32), (4096, 16)])
def test_split_equals_unsplit(L, S):
    d = 64
    q = RNG.standard_normal((4, d))
    K = RNG.standard_normal((2, L, d))
    V = RNG.standard_normal((2, L, d))
    bounds = od.split_bounds(L, S)
    assert bounds[0][0] == 0 and bounds[-1][1] == L
    assert all(b[0] % 16 == 0 for b in bounds if b[1] > b[0])
    np.testing.assert_allclose(od.attention_split(q, K, V, 0.125, bounds),
                               od.attention_dense(q, K, V, 0.125), atol=1e-12)


def _random_pool(n_pages, hkv, d):
    return RNG.standard_normal((n_pages, hkv, 2, 16 * d))


def test_gather_layout_by_hand():
    kvp = _random_pool(5, 2, 64)
    pages = np.array([3, 0, 4])
    K, V = od.gather_kv(kvp, pages, 35)
    assert K.shape == (2, 35, 64) and V.shape == (2, 35, 64)
    # key 20 lives in logical page 1 -> physical 0, slot 4; dim 40 is in dim
    # block 1 at offset 8: K tile position (1 * 16 + 4) * 32 + 8
    assert K[1, 20, 40] == kvp[0, 1, 0, (1 * 16 + 4) * 32 + 8]
    # V tile is dim-major: dim 40, slot 4 at 40 * 16 + 4
    assert V[1, 20, 40] == kvp[0, 1, 1, 40 * 16 + 4]
    # key 34: logical page 2 -> physical 4, slot 2; dim 3 in block 0
    assert K[0, 34, 3] == kvp[4, 0, 0, 2 * 32 + 3]
    np.testing.assert_array_equal(V[0, 0], kvp[3, 0, 1, np.arange(64) * 16])
    # one K row of a slot is two 32-dim runs of the tile
    np.testing.assert_array_equal(K[1, 20], np.concatenate([kvp[0, 1, 0, 4 * 32:5 * 32],
                                                           kvp[0, 1, 0, 20 * 32:21 * 32]]))


def test_paging_invariant_under_physical_permutation():
    N, hq, hkv, d = 3, 4, 2, 32
    lens = np.array([16, 45, 70])
    need = (lens + 15) // 16
    P = int(need.sum())
    kvp = _random_pool(P, hkv, d)
    pt_id = np.full((N, need.max()), -1)
    c = 0
    for i in range(N):
        pt_id[i, : need[i]] = np.arange(c, c + need[i])
        c += need[i]
    perm = RNG.permutation(P)          # logical page L now lives at physical perm[L]
    kvp2 = np.empty_like(kvp)
    kvp2[perm] = kvp
    pt2 = np.where(pt_id >= 0, perm[np.maximum(pt_id, 0)], -1)
    q = RNG.standard_normal((N, hq, d))
    a = od.paged_attention(q, kvp, pt_id, lens, 0.25)
    b = od.paged_attention(q, kvp2, pt2, lens, 0.25)
    np.testing.assert_array_equal(a, b)


# ---------------------------------------------------------------- prefill attention
def _seq_pool(lengths, hkv, d):
    """Pool with the pages of each sequence (lengths = keys) randomly placed."""
    need = [(n + 15) // 16 for n in lengths]
    P = sum(need)
    kvp = _random_pool(P, hkv, d)
    perm = RNG.permutation(P)
    pt = np.full((len(lengths), max(need)), -1)
    c = 0
    for i, n in enumerate(need):
        pt[i, :n] = perm[c:c + n]
        c += n
    return kvp, pt


@pytest.mark.parametrize("hq,hkv,d", [(4, 2, 32), (8, 8, 32), (8, 1, 64)])
def test_prefill_attention_is_causal_sdpa(hq, hkv, d):
    """Each sequence from position 0 equals torch's causal SDPA (float64) on its
    gathered keys, GQA by repeat-interleave: the library special case."""
    lens = [1, 17, 40]
    kvp, pt = _seq_pool(lens, hkv, d)
    starts = np.concatenate([[0], np.cumsum(lens)])
    q = RNG.standard_normal((starts[-1], hq, d))
    out = od.prefill_attention(q, kvp, pt, starts, None, 0.2)
    for s, n in enumerate(lens):
        K, V = od.gather_kv(kvp, pt[s], n)
        g = hq // hkv
        Kr = torch.from_numpy(K).repeat_interleave(g, dim=0)
        Vr = torch.from_numpy(V).repeat_interleave(g, dim=0)
        qs = torch.from_numpy(q[starts[s]:starts[s + 1]]).transpose(0, 1)   # [hq, n, d]
        ref = torch.nn.functional.scaled_dot_product_attention(qs, Kr, Vr, is_causal=True,
                                                               scale=0.2)
        np.testing.assert_allclose(out[starts[s]:starts[s + 1]], ref.transpose(0, 1).numpy(),
                                   atol=1e-12)


def test_prefill_attention_rows_are_decode_steps_and_prefix_offsets():
    """Row t of a prefill is the decode attention over keys 0..pos(t); a sequence
    that starts at position p0 equals the tail rows of a prefill from 0 over the
    same keys."""
    hq, hkv, d = 4, 2, 32
    n_all, p0 = 45, 29
    kvp, pt = _seq_pool([n_all], hkv, d)
    q = RNG.standard_normal((n_all, hq, d))
    full = od.prefill_attention(q, kvp, pt, [0, n_all], None, 0.3)
    for t in (0, 15, 16, 44):
        dec = od.paged_attention(q[t:t + 1], kvp, pt, [t + 1], 0.3)
        np.testing.assert_allclose(full[t], dec[0], atol=1e-13)
    tail = od.prefill_attention(q[p0:], kvp, pt, [0, n_all - p0], [p0], 0.3)
    np.testing.assert_allclose(tail, full[p0:], atol=1e-13)


def test_append_writes_exactly_one_slot():
    kvp = _random_pool(6, 2, 64)
    kv0 = kvp.copy()
    pt = np.array([[5, 1], [0, 3]])
    pos = np.array([17, 9])
    k = RNG.standard_normal((2, 2, 64))
    v = RNG.standard_normal((2, 2, 64))
    od.append_kv(kvp, pt, pos, k, v)
    changed = np.argwhere(kvp != kv0)                 # [page, head, K|V, position]
    assert int(len(changed)) == 2 * 2 * 2 * 64
    assert sorted(set(map(tuple, changed[:, :2].tolist()))) == [(0, 0), (0, 1), (1, 0), (1, 1)]
    K, V = od.gather_kv(kvp, pt[0], 18)               # candidate 0, key 17: page 1, slot 1
    np.testing.assert_array_equal(K[:, 17], k[0])
    np.testing.assert_array_equal(V[:, 17], v[0])
    K, V = od.gather_kv(kvp, pt[1], 10)               # candidate 1, key 9: page 0, slot 9
    np.testing.assert_array_equal(K[:, 9], k[1])
    np.testing.assert_array_equal(V[:, 9], v[1])
    # K values sit at the slot's tile positions, V values at the dim-major ones
    np.testing.assert_array_equal(kvp[1, 0, 0, (np.arange(64) // 32 * 16 + 1) * 32 + np.arange(64) % 32],
                                  k[0, 0])
    np.testing.assert_array_equal(kvp[0, 1, 1, np.arange(64) * 16 + 9], v[1, 1])


# ---------------------------------------------------------------- confidence (Eq. 1, 2)
def test_token_confidence_uniform_is_log_vocab():
    for V, k in ((7, 1), (7, 7), (4096, 20)):
        c = od.token_confidence(np.full((2, V), 3.25), k)
        np.testing.assert_allclose(c, math.log(V), rtol=0, atol=1e-12)


def test_token_confidence_all_tokens_is_lse_minus_mean():
    z = RNG.standard_normal((3, 50)) * 2
    lse = np.log(np.exp(z).sum(-1))
    np.testing.assert_allclose(od.token_confidence(z, 50), lse - z.mean(-1), atol=1e-12)


def test_token_confidence_dominant_token_and_brute_force():
    z = np.zeros((1, 10))
    z[0, 3] = 1000.0
    assert abs(od.token_confidence(z, 1)[0]) < 1e-12        # log p(top) = 0
    np.testing.assert_allclose(od.token_confidence(z, 2), [500.0 + 0.5 * math.log(1.0)],
                               atol=1e-9)
    z = RNG.standard_normal((4, 9))
    for k in (1, 3, 9):
        for i in range(4):
            p = [math.exp(v) for v in z[i]]
            s = sum(p)
            lps = sorted((math.log(v / s) for v in p), reverse=True)
            want = -sum(lps[:k]) / k
            assert abs(od.token_confidence(z[i:i + 1], k)[0] - want) < 1e-12


def test_token_confidence_shift_and_permutation_invariant():
    z = RNG.standard_normal((2, 64))
    c = od.token_confidence(z, 5)
    np.testing.assert_allclose(od.token_confidence(z + 17.5, 5), c, atol=1e-12)
    np.testing.assert_allclose(od.token_confidence(z[:, RNG.permutation(64)], 5), c, atol=1e-12)


def test_candidate_and_group_confidence_by_hand():
    C = od.candidate_confidence([6.0, 9.0, 2.0, 8.0], [3, 3, 1, 4])
    np.testing.assert_allclose(C, [2.0, 3.0, 2.0, 2.0])
    np.testing.assert_allclose(od.group_confidence(C, [[0, 1], [2, 3], [1, 3]]), [2.5, 2.0, 2.5])


# ---------------------------------------------------------------- truncated sampling
def test_truncated_with_everything_kept_is_the_plain_sampler():
    z = RNG.standard_normal((6, 300)) * 2
    uids = np.arange(6) + 40
    pos = np.arange(6) + 7
    for T in (1.0, 0.7, 0.0):
        a = od.logprob_sample(z, T, 3, uids, pos)
        b = od.truncated_logprob_sample(z, T, 3, uids, pos, top_k=300)
        np.testing.assert_array_equal(a[0], b[0])
        np.testing.assert_allclose(a[1], b[1], atol=1e-12)


def test_truncated_top1_is_greedy_with_zero_logprob():
    z = np.array([[0.5, 2.0, 2.0, -1.0], [3.0, 1.0, 0.0, 3.0]])
    ids, lps, _ = od.truncated_logprob_sample(z, 1.0, 5, [1, 2], [0, 0], top_k=1)
    assert list(ids) == [1, 0] and np.all(lps == 0.0)


def test_truncated_top_p_and_min_p_boundaries_by_hand():
    p = np.array([0.5, 0.3, 0.15, 0.05])
    z = np.log(p)[None, :]
    def kept(**kw):
        seen = set()
        for s in range(400):
            ids, lps, _ = od.truncated_logprob_sample(z, 1.0, s, [9], [0], top_k=4, **kw)
            seen.add(int(ids[0]))
        return seen
    assert kept(top_p=0.79) == {0, 1}           # cumulative before token 2 is 0.8: not below
    assert kept(top_p=0.81) == {0, 1, 2}
    assert kept(min_p=0.31) == {0, 1}           # 0.15 < 0.31 * 0.5
    assert kept(min_p=0.29) == {0, 1, 2}
    # the log-prob is renormalised over the kept set
    ids, lps, _ = od.truncated_logprob_sample(z, 1.0, 0, [9], [0], top_k=4, top_p=0.79)
    assert abs(lps[0] - np.log(p[ids[0]] / 0.8)) < 1e-12


def test_truncated_frequencies_match_renormalised_softmax():
    V = 10
    z = np.array([[1.2, 0.3, 2.0, -0.5, 1.9, 0.0, -3.0, 1.0, 0.9, 0.2]])
    T, k, top_p, min_p = 0.8, 5, 0.9, 0.05
    order = np.lexsort((np.arange(V), -z[0]))[:k]
    w = np.exp(z[0][order] / T)
    w = w / w.sum()
    keep = w >= min_p * w.max()
    cum, kp = 0.0, []
    tot = w[keep].sum()
    for j in range(k):
        if keep[j] and cum < top_p * tot:
            kp.append(j)
            cum += w[j]
    probs = np.zeros(V)
    probs[order[kp]] = w[kp] / w[kp].sum()
    n = 6000
    counts = np.zeros(V)
    for u in range(n):
        ids, _, _ = od.truncated_logprob_sample(z, T, 77, [u], [3], top_k=k, top_p=top_p,
                                                min_p=min_p)
        counts[ids[0]] += 1
    assert np.all(counts[probs == 0] == 0)
    m = probs > 0
    chi2 = np.sum((counts[m] - n * probs[m]) ** 2 / (n * probs[m]))
    assert chi2 < 25.0, (chi2, counts, probs)        # df <= 4: p ~ 1e-4


def test_truncated_set_does_not_depend_on_temperature():
    z = RNG.standard_normal((1, 64))
    sets = []
    for T in (0.3, 1.0, 2.5):
        seen = set()
        for s in range(200):
            ids, _, _ = od.truncated_logprob_sample(z, T, s, [1], [0], top_k=3)
            seen.add(int(ids[0]))
        sets.append(seen)
    top3 = set(np.argsort(-z[0])[:3].tolist())
    assert all(s <= top3 for s in sets)
