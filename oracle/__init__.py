"""CPU oracle for the population decode step — TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously-correct numpy code for what one decode step of a
population of candidates computes: a pre-norm GQA decoder layer stack over
per-candidate paged KV caches, a full-vocabulary log-softmax and a Gumbel-max
categorical sample with a counter-based RNG.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The product path (the C-ABI library and its Python binding)
never imports, links or calls it, and shares no code with it: the only module
both sides use is the seeded input generator, which holds none of the
method's arithmetic.

Precision: attention in float64; everything else in float64 too (a superset
of the fp32 the decode path needs); bf16 *storage* points of the GPU path are
mirrored with round-to-nearest-even (``mirror=True``) so that parity measures
the kernels rather than the storage format.  ``mirror=False`` gives the pure
definition.

Pins (checked by ``tests/test_oracle_*.py`` on the CPU): see each module.
Every function is pinned.  The paper prints no worked numeric example for
this path, so each pin is a closed form, an invariant, a library special
case or a brute force rather than a value printed in the paper.
"""
from .bf16 import round_bf16, bf16_bits_to_f32
from .philox import philox4x32_10, uniform01, gumbel_noise
from . import decoder
from .decoder import (rms_norm, rope_rotate, attention_dense, attention_split, gather_kv,
                      paged_attention, append_kv, decoder_layer, logprob_sample,
                      decode_step, silu, log_softmax)

__all__ = [
    "round_bf16", "bf16_bits_to_f32", "philox4x32_10", "uniform01", "gumbel_noise",
    "decoder", "rms_norm", "rope_rotate", "attention_dense", "attention_split", "gather_kv",
    "paged_attention", "append_kv", "decoder_layer", "logprob_sample", "decode_step", "silu",
    "log_softmax",
]
