"""Shared set-up for the GPU parity tests: device inputs, host oracle inputs,
and the comparison rules of the decode path.

Inputs on both sides come from the seeded generator (device twin on the GPU,
host twin for the oracle); no oracle input or expected value is read back from
the HIP path.
"""
import sys

import numpy as np
import torch

from oracle import decoder as od
from paper_2604_07725_amd import synth

ATTN_REL_TOL = 2e-2   # attention: max|o - o_ref| / max|o_ref|, per candidate
LP_ABS_TOL = 3e-3     # log-probabilities, absolute
GAP_EXACT = 1e-3      # ids bit-exact where the top-2 perturbed-logit gap exceeds this


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def make_population(lengths, shuffle=True, seed=0, extra=0, vocab=4096):
    lengths = np.asarray(lengths, np.int64)
    return synth.make_population(len(lengths), lengths, vocab, seed, extra, shuffle)


def host_candidate_kv(shape, seed, layer, pop, i, n_keys, n_pages_total):
    """Logical K, V [hkv, n_keys, d] of candidate i regenerated on the host."""
    kspec, vspec = synth.kv_specs(shape, seed, layer, n_pages_total)
    pages = pop.page_table[i, : (n_keys + 15) // 16]
    kp = synth.pool_pages(kspec, pages)
    vp = synth.pool_pages(vspec, pages)
    return od.gather_kv(kp, vp, np.arange(len(pages)), n_keys)


def attn_rel_err(o, ref):
    return float(np.abs(o - ref).max() / max(np.abs(ref).max(), 1e-30))


def check_ids(gpu_ids, gpu_lps, ref_ids, ref_lps, ref_gaps, pert=None, label=""):
    """ids bit-exact where the gap exceeds GAP_EXACT, log-probs within LP_ABS_TOL."""
    gpu_ids = np.asarray(gpu_ids, np.int64)
    exact = ref_gaps > GAP_EXACT
    bad = np.nonzero(exact & (gpu_ids != ref_ids))[0]
    assert bad.size == 0, f"{label}: ids differ at {bad[:8]} (gaps {ref_gaps[bad[:8]]})"
    if pert is not None:
        for i in np.nonzero(~exact)[0]:
            top = pert[i].max()
            assert pert[i][gpu_ids[i]] >= top - GAP_EXACT, f"{label}: invalid near-tie id"
    lp_err = np.abs(np.asarray(gpu_lps, np.float64) - ref_lps)
    # compare the log-prob of the GPU's own id when a near-tie made it differ
    assert lp_err[exact].max(initial=0.0) <= LP_ABS_TOL, f"{label}: lp err {lp_err.max()}"
    return float(lp_err.max(initial=0.0)), int(exact.sum())
