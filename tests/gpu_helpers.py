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
    spec = synth.kv_spec(shape, seed, layer, n_pages_total)
    pages = pop.page_table[i, : (n_keys + 15) // 16]
    pool = synth.pool_pages(spec, pages)
    return od.gather_kv(pool, np.arange(len(pages)), n_keys)


def subset_host_state(shape, seed, pop, idx, layers):
    """Host KV pools holding only the pages of candidates ``idx`` (the slot the
    step appends included), compacted, with a matching page table."""
    need = (pop.lengths[idx].astype(np.int64) + pop.extra_tokens + 15) // 16
    pt = np.full((len(idx), int(need.max())), -1, np.int64)
    kvp = [np.empty((int(need.sum()), shape.n_kv_heads, 2, 16 * shape.head_dim))
           for _ in range(layers)]
    c = 0
    for j, i in enumerate(idx):
        pages = pop.page_table[i, :need[j]]
        for l in range(layers):
            kvp[l][c:c + need[j]] = synth.pool_pages(synth.kv_spec(shape, seed, l, pop.n_pages),
                                                      pages)
        pt[j, :need[j]] = np.arange(c, c + need[j])
        c += need[j]
    return kvp, pt


def poisoned(nbytes: int, device="cuda") -> torch.Tensor:
    """A workspace whose every byte is 0xFF: NaN as fp32 and as bf16, -1 as an
    int32, so a kernel that reads scratch it did not write shows it."""
    return torch.full((max(int(nbytes), 256),), 255, dtype=torch.uint8, device=device)


def attn_rel_err(o, ref):
    return float(np.abs(o - ref).max() / max(np.abs(ref).max(), 1e-30))


def check_ids(gpu_ids, gpu_lps, ref_ids, ref_lps, ref_gaps, details, label=""):
    """The sampler's bars against the oracle: ids bit-exact where the oracle's
    top-2 perturbed-value gap exceeds GAP_EXACT; elsewhere (a near tie) the GPU's
    id must be a valid pick, its perturbed value within GAP_EXACT of the
    oracle's largest.  Log-probs within LP_ABS_TOL of the oracle's log-prob of
    the same token.  ``details`` is what the oracle sampler put in its
    ``details`` dict ("pert", "logp" [N, V])."""
    gpu_ids = np.asarray(gpu_ids, np.int64)
    pert, logp = details["pert"], details["logp"]
    exact = ref_gaps > GAP_EXACT
    bad = np.nonzero(exact & (gpu_ids != ref_ids))[0]
    assert bad.size == 0, f"{label}: ids differ at {bad[:8]} (gaps {ref_gaps[bad[:8]]})"
    assert np.all((gpu_ids >= 0) & (gpu_ids < pert.shape[1])), f"{label}: id out of range"
    rows = np.arange(len(gpu_ids))
    slack = pert.max(axis=1) - pert[rows, gpu_ids]
    assert np.all(slack <= GAP_EXACT), f"{label}: invalid pick (slack {slack.max():.2e})"
    lp_err = np.abs(np.asarray(gpu_lps, np.float64) - logp[rows, gpu_ids])
    assert np.all(np.abs(ref_lps[gpu_ids == ref_ids] - logp[rows, gpu_ids][gpu_ids == ref_ids])
                  <= 1e-12)
    assert lp_err.max(initial=0.0) <= LP_ABS_TOL, f"{label}: lp err {lp_err.max()}"
    return float(lp_err.max(initial=0.0)), int(exact.sum())


# ---- GEMM operand layouts, written out from their definition in include/sevo.h
def packed_weight_offsets(n_out: int, k: int) -> np.ndarray:
    """Flat offset of every element (r, c) of W [n_out][k] in the packed layout."""
    r = np.arange(n_out)[:, None]
    c = np.arange(k)[None, :]
    return ((((r // 64) * (k // 32) + c // 32) * 4 + (r // 16) % 4) * 512
            + (16 * ((c // 8) % 4) + r % 16) * 8 + c % 8)


def gate_up_row_order(n_out: int) -> np.ndarray:
    """Logical row order of a SEVO_PACK_GATE_UP weight: per superblock s the gate
    rows 32s..32s+31, then the up rows n_out/2 + 32s.."""
    F = n_out // 2
    order = []
    for s in range(n_out // 64):
        order += list(range(32 * s, 32 * s + 32)) + list(range(F + 32 * s, F + 32 * s + 32))
    return np.array(order)


def pack_weight_host(w: np.ndarray, gate_up: bool = False) -> np.ndarray:
    n_out, k = w.shape
    if gate_up:
        w = w[gate_up_row_order(n_out)]
    out = np.empty(n_out * k, w.dtype)
    out[packed_weight_offsets(n_out, k).ravel()] = w.ravel()
    return out.reshape(n_out, k)


def act_tile_offsets(m: int, k: int) -> np.ndarray:
    r = np.arange(m)[:, None]
    c = np.arange(k)[None, :]
    return ((r // 16) * (k // 32) + c // 32) * 512 + (16 * ((c // 8) % 4) + r % 16) * 8 + c % 8


def tile_activations_host(x: np.ndarray) -> np.ndarray:
    """x [m][k] -> flat tiled buffer of ceil(m/16)*16 rows (padding rows zero)."""
    m, k = x.shape
    out = np.zeros(-(-m // 16) * 16 * k, x.dtype)
    out[act_tile_offsets(m, k).ravel()] = x.ravel()
    return out


def untile_activations_host(t: np.ndarray, m: int, k: int) -> np.ndarray:
    return np.asarray(t).reshape(-1)[act_tile_offsets(m, k)]
