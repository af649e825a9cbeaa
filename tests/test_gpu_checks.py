"""GPU checks of the paging validator, the sampler's counter-based noise at
scale, and the sampler on rows without a comparable logit."""
import numpy as np
import pytest
import torch

from oracle import philox
from tests.gpu_helpers import make_population, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_07725_amd import sevo
    sevo.lib()
    return sevo


def _validate(sevo, pt, lengths, num_pages):
    try:
        sevo.sevo_validate_paging(torch.from_numpy(np.ascontiguousarray(pt, np.int32)).cuda(),
                                  torch.from_numpy(np.asarray(lengths, np.int32)).cuda(),
                                  num_pages)
        return sevo.OK, ""
    except sevo.SevoError as e:
        return e.status, str(e)


def test_validate_paging_finds_each_kind_of_bad_table(S):
    """A valid table passes; an id outside the pool, a physical page used twice,
    a missing page for a needed slot (the slot a decode step appends: lengths =
    positions + 1) and a length beyond the table each give BAD_PAGE_TABLE."""
    sevo = S
    pop = make_population([40, 16, 1, 100], seed=4, extra=1)
    P = pop.n_pages
    pos = pop.lengths.astype(np.int64)
    say("validate paging")
    assert _validate(sevo, pop.page_table, pos + 1, P)[0] == sevo.OK
    assert _validate(sevo, pop.page_table, np.zeros(4), P)[0] == sevo.OK
    cases = []
    bad = pop.page_table.copy()
    bad[0, 1] = P                                   # outside [0, num_pages)
    cases.append(("out of range", bad, pos + 1))
    bad = pop.page_table.copy()
    bad[0, 2] = -3
    cases.append(("negative id", bad, pos + 1))
    bad = pop.page_table.copy()
    bad[3, 5] = bad[2, 0]                           # one physical page twice
    cases.append(("duplicate", bad, pos + 1))
    bad = pop.page_table.copy()
    bad[1, 1] = -1                                  # 16 cached keys: slot 16 needs page 1
    cases.append(("missing append page", bad, pos + 1))
    cases.append(("length beyond the table", pop.page_table,
                  np.array([40, 16, 1, 16 * pop.max_pages + 1])))
    cases.append(("negative length", pop.page_table, np.array([40, -1, 1, 100])))
    for name, pt, lens in cases:
        status, msg = _validate(sevo, pt, lens, P)
        say(f"  {name}: {msg}")
        assert status == sevo.BAD_PAGE_TABLE, name
    # the append page of candidate 1 is only needed once its slot 16 is appended
    bad = pop.page_table.copy()
    bad[1, 1] = -1
    assert _validate(sevo, bad, pos, P)[0] == sevo.OK


@pytest.mark.parametrize("n,vocab", [(1 << 20, 4), (16384, 8192)])
def test_sampler_noise_at_scale_matches_philox(S, n, vocab):
    """Zero logits at T = 1: the sample is the argmax of the Philox-driven noise
    (its 23-bit uniform, ties to the lowest index), so every id checks the
    Philox4x32-10 words of its row against the oracle's integer Philox.
    1M (uid, position) pairs x 4 words, and 16K pairs x 8192 words: 1.4e8
    words in all.  Ids are exact wherever the oracle's top two uniforms differ
    by 2 or more 23-bit steps (the fp32 Gumbel map keeps their order);
    elsewhere the GPU's id must hold one of the two largest."""
    sevo = S
    say(f"sampler noise at scale: n={n} vocab={vocab}")
    rng = np.random.default_rng(n + vocab)
    uids = rng.integers(0, 2 ** 63 - 1, size=n, dtype=np.int64).astype(np.uint64)
    pos = rng.integers(0, 2 ** 31 - 1, size=n).astype(np.int32)
    seed = 0xDEADBEEF12345
    logits = torch.zeros(n, vocab, dtype=torch.float32, device="cuda")
    ids, lps = sevo.sevo_logprob_sample(logits, 1.0, seed, torch.from_numpy(uids.view(np.int64))
                                        .cuda(), torch.from_numpy(pos).cuda())
    torch.cuda.synchronize()
    g_ids = ids.cpu().numpy().astype(np.int64)
    np.testing.assert_allclose(lps.cpu().numpy(), -np.log(vocab), rtol=0, atol=2e-6)
    del logits
    ref = np.empty(n, np.int64)
    top2 = np.empty((n, 2), np.int64)
    rows = max(1, (1 << 22) // vocab)
    blocks = np.arange(vocab // 4, dtype=np.uint64)            # counter word 0 = v >> 2
    for a in range(0, n, rows):
        b = min(n, a + rows)
        out = philox.philox4x32_10(blocks[None, :], pos[a:b, None].astype(np.uint64),
                                   (uids[a:b, None] & np.uint64(0xFFFFFFFF)),
                                   uids[a:b, None] >> np.uint64(32), seed & 0xFFFFFFFF,
                                   seed >> 32)
        # word v & 3 of block v >> 2 drives token v
        u = np.stack(out, axis=-1).reshape(b - a, vocab) >> np.uint64(9)   # 23-bit uniforms
        ref[a:b] = np.argmax(u, axis=1)                       # first maximum
        srt = np.sort(u, axis=1)
        top2[a:b] = srt[:, -2:].astype(np.int64)
        ok = (u[np.arange(b - a), g_ids[a:b]] >= srt[:, -2])
        assert ok.all(), "a GPU id outside the two largest uniforms"
    exact = top2[:, 1] - top2[:, 0] >= 2
    bad = np.nonzero(exact & (g_ids != ref))[0]
    say(f"  {exact.mean():.6f} of rows decided by >= 2 steps; mismatches {bad.size}")
    assert bad.size == 0, bad[:10]


def test_sampler_row_of_nan_logits_gives_no_token(S):
    """A row whose logits are all NaN has no comparable perturbed value: id -1,
    log-prob NaN, for full-vocabulary and truncated sampling; other rows are
    unaffected."""
    sevo = S
    n, vocab = 3, 5000
    logits = torch.randn(n, vocab, generator=torch.Generator().manual_seed(2)).cuda()
    logits[1] = float("nan")
    uid = torch.arange(n, dtype=torch.int64, device="cuda") + 9
    pos = torch.arange(n, dtype=torch.int32, device="cuda")
    for kw in ({}, {"top_k": 20, "top_p": 0.9}):
        for temp in (1.0, 0.0, 0.7):
            ids, lps = sevo.sevo_logprob_sample(logits, temp, 5, uid, pos, **kw)
            clean, _ = sevo.sevo_logprob_sample(logits[[0, 2]].contiguous(), temp, 5, uid[[0, 2]],
                                                pos[[0, 2]], **kw)
            torch.cuda.synchronize()
            assert int(ids[1]) == -1 and np.isnan(float(lps[1])), (kw, temp)
            assert ids[[0, 2]].tolist() == clean.tolist()
