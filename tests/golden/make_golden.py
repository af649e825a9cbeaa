"""Writes the oracle's expected outputs for the tiny decode-step workload.

The paper prints no worked numeric example for the decode path, so the stored
values here are the oracle's own (inputs from the seeded generator, outputs
from oracle/ only).  They guard the oracle against silent drift: a change to
its arithmetic must regenerate this file and say why in its commit message.

Usage: python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import decoder as od  # noqa: E402
from paper_2604_07725_amd import synth  # noqa: E402

SEED_SAMPLE = 1234


def tiny_step_expected():
    w = synth.WORKLOADS["tiny_step"]
    shape = w.shape
    pop = synth.workload_population(w, extra_tokens=1)
    weights = synth.host_weights(shape, w.seed)
    kvp = [p.astype(np.float64) for p in synth.host_pools(shape, w.seed, pop.n_pages)]
    out = od.decode_step(shape, weights, kvp, pop.page_table, pop.tokens, pop.lengths,
                         pop.uids, SEED_SAMPLE, 1.0, mirror=True)
    return {
        "workload": "tiny_step", "sample_seed": SEED_SAMPLE, "temperature": 1.0,
        "ids": out["ids"].tolist(), "lps": out["lps"].tolist(), "gaps": out["gaps"].tolist(),
        "logits_first8": out["logits"][:, :8].tolist(),
        "logits_sum": out["logits"].sum(axis=1).tolist(),
    }


if __name__ == "__main__":
    data = tiny_step_expected()
    with open(os.path.join(HERE, "tiny_step_oracle.json"), "w") as f:
        json.dump(data, f, indent=1)
    print("wrote tiny_step_oracle.json", data["ids"])
