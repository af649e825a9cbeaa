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
