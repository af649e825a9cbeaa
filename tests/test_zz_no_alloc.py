"""The attention entry point that allocates nothing (sevo_attn_decode_noalloc):
its split partials live in the library's fixed device scratch, and its output
must equal sevo_attn_decode's, bit for bit, call after call."""
import ctypes as C

import numpy as np
import pytest
import torch

from oracle import decoder as od
from paper_2604_07725_amd import synth
from tests.gpu_helpers import attn_rel_err, bf16_bits, host_candidate_kv, make_population, say, to_np


def test_noalloc_rejects_partials_beyond_the_scratch():
    """Partials larger than the fixed scratch are refused before any launch
    (a host check: no GPU needed)."""
    from paper_2604_07725_amd import sevo
    fake = 1 << 20            # never dereferenced: the size check fails first
    # 2048 candidates x 32 heads x 1 split x (128 + 2) x 4 bytes = 34 MB > 32 MiB
    a = sevo.AttnArgs(n=2048, n_q_heads=32, n_kv_heads=8, head_dim=128, page_size=16,
                      max_pages=4, num_splits=1, num_pages=4, q=fake, kv_pool=fake,
                      page_table=fake, seq_lens=fake, scale=0.088, out=fake)
    assert sevo.lib().sevo_attn_decode_noalloc(C.byref(a), None) == sevo.WORKSPACE_TOO_SMALL
    assert b"scratch" in sevo.lib().sevo_last_error()
    a.n = 0
    assert sevo.lib().sevo_attn_decode_noalloc(C.byref(a), None) == sevo.OK


@pytest.mark.gpu
def test_noalloc_attention_equals_the_workspace_attention():
    """Calls in a row -- a population of 6, then a smaller one of 2 (the
    scratch still holds the first call's partials), then 8 query heads per kv
    head -- each bit-identical to sevo_attn_decode with a workspace of its
    own, and within the attention bar of the oracle."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_07725_amd import device_inputs as di
    from paper_2604_07725_amd import sevo
    sevo.lib()
    for call, (hq, hkv, lengths, splits) in enumerate([
            (32, 8, [3000, 17, 1600, 900, 1, 4100], 0),
            (32, 8, [40, 5], 0),
            (32, 4, [2500, 700, 33], 5)]):
        shape = synth.ModelShape(1, 256, hq, hkv, 128, 256, 256)
        seed = 40 + call
        say(f"no-alloc attention call {call}: {hq}/{hkv} heads, lengths {lengths}")
        pop = make_population(lengths, seed=seed)
        kvp = di.device_pools(shape, seed, pop.n_pages, layers=[0])[0]
        q = di.device_q(shape, seed, pop.n)
        pt = torch.from_numpy(pop.page_table).cuda()
        lens = torch.from_numpy(pop.lengths).cuda()
        out = torch.empty_like(q)
        sevo.sevo_attn_decode_noalloc(q, kvp, pt, lens, out, num_splits=splits)
        ref = sevo.sevo_attn_decode(q, kvp, pt, lens, num_splits=splits)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(bf16_bits(out), bf16_bits(ref))
        i = int(np.argmax(pop.lengths))
        qh = synth.host_values(synth.q_spec(shape, seed, pop.n)).reshape(pop.n, hq, 128)
        K, V = host_candidate_kv(shape, seed, 0, pop, i, int(pop.lengths[i]), pop.n_pages)
        e = attn_rel_err(to_np(out)[i], od.attention_dense(qh[i], K, V, 128 ** -0.5))
        say(f"  bit-identical; candidate {i} rel err {e:.2e}")
        assert e <= 8e-3
