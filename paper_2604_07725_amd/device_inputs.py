"""Synthetic inputs materialised in device memory.

The tensors are filled on the GPU by ``sevo_fill_normal_bf16`` (the device
twin of the seeded generator in ``synth``), so every value equals what the
host generator gives for the same tensor key and element index.  Population
metadata (lengths, page tables, tokens, uids) is drawn on the host and copied.
"""
from __future__ import annotations

import numpy as np
import torch

from . import synth
from .sevo import PACKED_WEIGHTS, sevo_fill_normal_bf16, sevo_pack_weight


def _filled(spec: synth.TensorSpec, device) -> torch.Tensor:
    t = torch.empty(spec.shape, dtype=torch.bfloat16, device=device)
    sevo_fill_normal_bf16(t, spec.key, 0, spec.std, spec.mean)
    return t


def device_weights(shape: synth.ModelShape, seed: int, device="cuda") -> dict:
    """The model's weights as the library takes them: projection matrices are
    generated row-major (the generator's element order) into a scratch tensor
    and packed; the rest stay row-major."""
    scratch = {}

    def make(name, spec):
        if name not in PACKED_WEIGHTS:
            return _filled(spec, device)
        n = 1
        for d in spec.shape:
            n *= d
        buf = scratch.get("buf")
        if buf is None or buf.numel() < n:
            buf = scratch["buf"] = torch.empty(n, dtype=torch.bfloat16, device=device)
        src = buf[:n].view(spec.shape)
        sevo_fill_normal_bf16(src, spec.key, 0, spec.std, spec.mean)
        if len(spec.shape) == 3:   # one matrix per expert, each packed on its own
            dst = torch.empty(spec.shape, dtype=torch.bfloat16, device=device)
            for e in range(spec.shape[0]):
                sevo_pack_weight(src[e], PACKED_WEIGHTS[name], dst=dst[e])
            return dst
        return sevo_pack_weight(src, PACKED_WEIGHTS[name])

    g = synth.global_specs(shape, seed)
    out = {k: make(k, s) for k, s in g.items()}
    out["layers"] = [{k: make(k, s) for k, s in synth.layer_specs(shape, seed, l).items()}
                     for l in range(shape.n_layers)]
    return out


def device_pools(shape: synth.ModelShape, seed: int, n_pages: int, device="cuda",
                 layers=None) -> list:
    """One KV pool per layer, [P][hkv][2][16 d] bf16."""
    return [_filled(synth.kv_spec(shape, seed, l, n_pages), device)
            for l in (range(shape.n_layers) if layers is None else layers)]


def device_q(shape: synth.ModelShape, seed: int, n: int, device="cuda") -> torch.Tensor:
    return _filled(synth.q_spec(shape, seed, n), device)


def device_population(pop: synth.Population, device="cuda") -> dict:
    return {
        "lengths": torch.from_numpy(pop.lengths.astype(np.int32)).to(device),
        "page_table": torch.from_numpy(pop.page_table.astype(np.int32)).to(device),
        "tokens": torch.from_numpy(pop.tokens.astype(np.int32)).to(device),
        "uids": torch.from_numpy(pop.uids.view(np.int64)).to(device),
    }
