"""Seeded synthetic inputs for the population decode step.

This module only *generates inputs*: model shapes, population recipes, context
lengths, shuffled page tables, token ids, candidate uids and bf16 tensors of
random values.  It holds none of the decode step's arithmetic, so both the HIP
path (via its device twin ``sevo_fill_normal_bf16``) and the CPU oracle may use
it.

Value generator (counter based, identical on host and device):
    r   = SplitMix64 finaliser of (key + (e + 1) * 0x9E3779B97F4A7C15)
          (Steele, Lea & Flood, OOPSLA 2014)
    s   = sum of the four 16-bit fields of r         (Irwin-Hall with n = 4)
    val = fp32(s - 131070) * mul [+ add], each operation rounded once
    bf16 = round-to-nearest-even of val
``mul = std / sqrt((2**32 - 1) / 3)`` rounded to fp32, so ``val`` has mean
``add`` and standard deviation ``std``; its support is +-3.46 std.  The
Irwin-Hall sum stands in for the Gaussian draws that the workloads specify
(weights N(0, 0.02), KV N(0, 1)) because it is exactly reproducible with
integer arithmetic and one fp32 rounding on any device.

Workload recipes follow the population shapes of the paper's method section
(N candidates, aggregation prompts of K concatenated candidates) and the
generation lengths of its hyper-parameter table; token content is random
because only shapes and lengths decide decode cost.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass, field

import numpy as np

GOLDEN = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB
_MASK64 = (1 << 64) - 1
IH_STD = math.sqrt((2.0 ** 32 - 1.0) / 3.0)  # std of the 4-field sum
IH_MEAN = 131070

PAGE_SIZE = 16


def mix64(z: int) -> int:
    """SplitMix64 finaliser on a Python int (mod 2**64)."""
    z &= _MASK64
    z = ((z ^ (z >> 30)) * _M1) & _MASK64
    z = ((z ^ (z >> 27)) * _M2) & _MASK64
    return z ^ (z >> 31)


def tensor_key(seed: int, kind: int, layer: int = 0) -> int:
    """Key of one synthetic tensor: kind and layer select a stream per seed."""
    return mix64(mix64(seed * 0x100000001B3 + 0x5E70) ^ ((kind << 32) | (layer & 0xFFFFFFFF)))


def ih_mul(std: float) -> np.float32:
    return np.float32(std / IH_STD)


# ---------------------------------------------------------------- host generator
_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(os.path.dirname(__file__), "libsynth_host.so")
        if not os.path.exists(path):
            raise RuntimeError(
                f"{path} is missing: run __graft_entry__.build() to compile the host generator")
        lib = ctypes.CDLL(path)
        for name, ptr_t in (("synth_fill_bf16", ctypes.c_void_p),
                            ("synth_fill_bf16_as_f32", ctypes.c_void_p)):
            fn = getattr(lib, name)
            fn.argtypes = [ptr_t, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int64,
                           ctypes.c_float, ctypes.c_float, ctypes.c_int]
            fn.restype = None
        lib.synth_fill_pages_as_f32.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                                ctypes.c_int64, ctypes.c_uint64, ctypes.c_float,
                                                ctypes.c_float, ctypes.c_int]
        lib.synth_fill_pages_as_f32.restype = None
        lib.synth_mix64.argtypes = [ctypes.c_uint64]
        lib.synth_mix64.restype = ctypes.c_uint64
        _LIB = lib
    return _LIB


def fill_bf16_bits(count: int, key: int, offset: int = 0, std: float = 1.0,
                   mean: float | None = None) -> np.ndarray:
    """uint16 bf16 bit patterns of elements [offset, offset + count)."""
    out = np.empty(count, np.uint16)
    if count:
        _lib().synth_fill_bf16(out.ctypes.data, count, key, offset, float(ih_mul(std)),
                               0.0 if mean is None else float(mean), 0 if mean is None else 1)
    return out


def fill_values(count: int, key: int, offset: int = 0, std: float = 1.0,
                mean: float | None = None) -> np.ndarray:
    """The same elements as fp32 values (each exactly a bf16 value)."""
    out = np.empty(count, np.float32)
    if count:
        _lib().synth_fill_bf16_as_f32(out.ctypes.data, count, key, offset, float(ih_mul(std)),
                                      0.0 if mean is None else float(mean),
                                      0 if mean is None else 1)
    return out


def fill_bf16_bits_numpy(count: int, key: int, offset: int = 0, std: float = 1.0,
                         mean: float | None = None) -> np.ndarray:
    """Pure-numpy twin of :func:`fill_bf16_bits` (slow; for cross-checks)."""
    with np.errstate(over="ignore"):
        e = np.arange(offset + 1, offset + count + 1, dtype=np.uint64)
        z = np.uint64(key) + e * np.uint64(GOLDEN)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(_M1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(_M2)
        r = z ^ (z >> np.uint64(31))
    m = np.uint64(0xFFFF)
    s = ((r & m) + ((r >> np.uint64(16)) & m) + ((r >> np.uint64(32)) & m)
         + (r >> np.uint64(48))).astype(np.int64) - IH_MEAN
    v = s.astype(np.float32) * ih_mul(std)
    if mean is not None:
        v = v + np.float32(mean)
    b = v.view(np.uint32).astype(np.uint64)
    b = b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))
    return ((b >> np.uint64(16)) & np.uint64(0xFFFF)).astype(np.uint16)


def bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------- model shapes
@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rope_theta: float = 1.0e6
    rms_eps: float = 1.0e-6
    qk_norm: bool = True
    page_size: int = PAGE_SIZE
    # mixture-of-experts FFN (0 experts = the dense SwiGLU FFN of size ffn)
    n_experts: int = 0
    top_k: int = 0
    expert_ffn: int = 0

    @property
    def is_moe(self) -> bool:
        return self.n_experts > 0

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def qkv_dim(self) -> int:
        return self.q_dim + 2 * self.kv_dim

    def layer_weight_elems(self, active_experts: float | None = None) -> int:
        """bf16 weight elements of one layer a decode step reads; a MoE layer
        reads the router and the experts its tokens select (all experts if
        active_experts is None)."""
        H = self.hidden
        attn = self.qkv_dim * H + H * self.q_dim
        if self.is_moe:
            e = self.n_experts if active_experts is None else active_experts
            return attn + self.n_experts * H + e * 3 * self.expert_ffn * H
        return attn + 2 * self.ffn * H + H * self.ffn

    def weight_bytes(self, active_experts: float | None = None) -> int:
        """Bytes of bf16 weights one decode step streams (layers + LM head)."""
        return int(2 * (self.n_layers * self.layer_weight_elems(active_experts)
                        + self.vocab * self.hidden))

    def stored_weight_bytes(self) -> int:
        return self.weight_bytes(None)


TINY = ModelShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                  ffn=1024, vocab=4096)
DENSE_8B = ModelShape(n_layers=36, hidden=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                      ffn=12288, vocab=151936)
DENSE_32B = ModelShape(n_layers=64, hidden=5120, n_q_heads=64, n_kv_heads=8, head_dim=128,
                       ffn=25600, vocab=151936)
# mixture-of-experts decoders (Qwen3-MoE layout: router, top-k of the experts,
# softmax over the selected logits, SwiGLU experts)
TINY_MOE = ModelShape(n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=0,
                      vocab=4096, n_experts=64, top_k=4, expert_ffn=64)
MOE_30B_A3B = ModelShape(n_layers=48, hidden=2048, n_q_heads=32, n_kv_heads=4, head_dim=128,
                         ffn=0, vocab=151936, n_experts=128, top_k=8, expert_ffn=768)


# ---------------------------------------------------------------- workloads
@dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    n: int                 # population size N (decode batch)
    lengths: str           # length recipe, see draw_lengths
    seed: int
    attention_only: bool = False
    steps: int = 1
    num_splits: int = 0    # 0 = library picks
    aggregation_k: int | None = 4   # candidates concatenated per context (None: no recipe)


WORKLOADS = {
    w.name: w for w in [
        # 1 layer, d=256, 4/2 heads x 64, FFN 1024, V 4096, N=4, p ~ U{256..512}
        Workload("tiny_step", TINY, 4, "u256_512", seed=0, aggregation_k=None),
        # attention only, 32/8 heads x 128, N=16, p = sum of 4 x U{2048..4096}
        Workload("attn_pop16_agg4", ModelShape(1, 4096, 32, 8, 128, 12288, 151936), 16,
                 "agg4_u2048_4096", seed=1, attention_only=True),
        # 8B-class dense decoder, N=64, p ~ U{16384..32768}
        Workload("dense8b_pop64_agg4", DENSE_8B, 64, "u16384_32768", seed=2, steps=16),
        # 8B-class, N=16, K=8 x 8k, +-10%
        Workload("dense8b_pop16_agg8", DENSE_8B, 16, "agg8_8k_pm10", seed=3, steps=128,
                 aggregation_k=8),
        # 32B-class, N=16, p = 16384
        Workload("dense32b_pop16_agg4", DENSE_32B, 16, "const16384", seed=4, steps=64),
        # tiny MoE decoder (2 layers, 64 experts, top-4), N=4, p ~ U{256..512}
        Workload("tiny_moe_step", TINY_MOE, 4, "u256_512", seed=5, aggregation_k=None),
        # 30B-A3B-class MoE decoder (48 layers, 128 experts, top-8), N=64,
        # p ~ U{16384..32768}
        Workload("moe30b_pop64_agg4", MOE_30B_A3B, 64, "u16384_32768", seed=6, steps=16),
    ]
}


def draw_lengths(recipe: str, n: int, rng: np.random.Generator) -> np.ndarray:
    """Cached-token counts per candidate (int64)."""
    if recipe == "u256_512":
        return rng.integers(256, 512, size=n, endpoint=True)
    if recipe == "agg4_u2048_4096":
        return rng.integers(2048, 4096, size=(n, 4), endpoint=True).sum(axis=1)
    if recipe == "u16384_32768":
        return rng.integers(16384, 32768, size=n, endpoint=True)
    if recipe == "agg8_8k_pm10":
        return np.floor(65536.0 * rng.uniform(0.9, 1.1, size=n)).astype(np.int64)
    if recipe == "const16384":
        return np.full(n, 16384, np.int64)
    if recipe.startswith("const"):
        return np.full(n, int(recipe[5:]), np.int64)
    raise ValueError(f"unknown length recipe {recipe!r}")


@dataclass
class Population:
    """Host-side description of a population and its paged KV layout."""
    lengths: np.ndarray        # int32 [N]: tokens already cached (p_i)
    page_table: np.ndarray     # int32 [N, max_pages]; -1 = unused entry
    n_pages: int               # physical pages per layer pool
    tokens: np.ndarray         # int32 [N]: the input token of the first step
    uids: np.ndarray           # uint64 [N]
    extra_tokens: int = 0      # slots reserved per candidate beyond lengths
    meta: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return int(self.lengths.shape[0])

    @property
    def max_pages(self) -> int:
        return int(self.page_table.shape[1])

    def pages_of(self, i: int, n_keys: int) -> np.ndarray:
        return self.page_table[i, : (n_keys + PAGE_SIZE - 1) // PAGE_SIZE]


def make_population(n: int, lengths: np.ndarray, vocab: int, seed: int,
                    extra_tokens: int, shuffle: bool = True,
                    rng: np.random.Generator | None = None) -> Population:
    """Page tables with room for ``lengths + extra_tokens`` keys per candidate.

    Physical pages are a random permutation of 0..P-1 (``shuffle``) or the
    identity, assigned candidate by candidate in logical order.
    """
    if rng is None:
        rng = np.random.Generator(np.random.PCG64(seed))
    lengths = np.asarray(lengths, np.int64)
    need = (lengths + extra_tokens + PAGE_SIZE - 1) // PAGE_SIZE
    need = np.maximum(need, 1)
    total = int(need.sum())
    max_pages = int(need.max())
    perm = rng.permutation(total) if shuffle else np.arange(total)
    pt = np.full((n, max_pages), -1, np.int32)
    cur = 0
    for i in range(n):
        k = int(need[i])
        pt[i, :k] = perm[cur:cur + k]
        cur += k
    tokens = rng.integers(0, vocab, size=n).astype(np.int32)
    uids = rng.integers(0, 2 ** 63 - 1, size=n, dtype=np.int64).astype(np.uint64)
    return Population(lengths.astype(np.int32), pt, total, tokens, uids, extra_tokens)


def workload_population(w: Workload, extra_tokens: int = 0, shuffle: bool = True,
                        n: int | None = None) -> Population:
    """Draw order: lengths, page permutation, token ids, uids (seeded by w.seed)."""
    rng = np.random.Generator(np.random.PCG64(w.seed))
    nn = w.n if n is None else n
    lengths = draw_lengths(w.lengths, nn, rng)
    return make_population(nn, lengths, w.shape.vocab, w.seed, extra_tokens, shuffle, rng)


# ---------------------------------------------------------------- tensor kinds
K_EMBED, K_LMHEAD, K_FINAL_NORM = 1, 2, 3
K_ATTN_NORM, K_WQKV, K_QNORM, K_KNORM, K_WO, K_FFN_NORM, K_WGU, K_WDOWN = range(10, 18)
K_KVPOOL, K_Q = 30, 32
K_WROUTER, K_WEGU, K_WEDOWN = 18, 19, 20

WEIGHT_STD = 0.02
GAIN_STD = 0.02


@dataclass(frozen=True)
class TensorSpec:
    """One synthetic tensor: element count, key, distribution."""
    shape: tuple
    key: int
    std: float
    mean: float | None = None

    @property
    def count(self) -> int:
        return int(np.prod(self.shape))


def layer_specs(shape: ModelShape, seed: int, layer: int) -> dict:
    H, F, D = shape.hidden, shape.ffn, shape.head_dim
    k = lambda kind: tensor_key(seed, kind, layer)  # noqa: E731
    specs = {
        "attn_norm": TensorSpec((H,), k(K_ATTN_NORM), GAIN_STD, 1.0),
        "w_qkv": TensorSpec((shape.qkv_dim, H), k(K_WQKV), WEIGHT_STD),
        "q_norm": TensorSpec((D,), k(K_QNORM), GAIN_STD, 1.0),
        "k_norm": TensorSpec((D,), k(K_KNORM), GAIN_STD, 1.0),
        "w_o": TensorSpec((H, shape.q_dim), k(K_WO), WEIGHT_STD),
        "ffn_norm": TensorSpec((H,), k(K_FFN_NORM), GAIN_STD, 1.0),
    }
    if shape.is_moe:
        E, Fe = shape.n_experts, shape.expert_ffn
        specs["w_router"] = TensorSpec((E, H), k(K_WROUTER), WEIGHT_STD)
        # expert e's gate (rows 0..Fe-1) and up (rows Fe..2Fe-1) projections,
        # then its down projection, each expert's matrix contiguous
        specs["w_expert_gate_up"] = TensorSpec((E, 2 * Fe, H), k(K_WEGU), WEIGHT_STD)
        specs["w_expert_down"] = TensorSpec((E, H, Fe), k(K_WEDOWN), WEIGHT_STD)
    else:
        specs["w_gate_up"] = TensorSpec((2 * F, H), k(K_WGU), WEIGHT_STD)
        specs["w_down"] = TensorSpec((H, F), k(K_WDOWN), WEIGHT_STD)
    return specs


def global_specs(shape: ModelShape, seed: int) -> dict:
    H, V = shape.hidden, shape.vocab
    return {
        "embed": TensorSpec((V, H), tensor_key(seed, K_EMBED), WEIGHT_STD),
        "lm_head": TensorSpec((V, H), tensor_key(seed, K_LMHEAD), WEIGHT_STD),
        "final_norm": TensorSpec((H,), tensor_key(seed, K_FINAL_NORM), GAIN_STD, 1.0),
    }


def kv_spec(shape: ModelShape, seed: int, layer: int, n_pages: int) -> TensorSpec:
    """The layer's KV pool [P][hkv][2][16 d] (K tile, then V tile), N(0, 1)."""
    return TensorSpec((n_pages, shape.n_kv_heads, 2, PAGE_SIZE * shape.head_dim),
                      tensor_key(seed, K_KVPOOL, layer), 1.0)


def q_spec(shape: ModelShape, seed: int, n: int) -> TensorSpec:
    return TensorSpec((n, shape.n_q_heads, shape.head_dim), tensor_key(seed, K_Q), 1.0)


def host_values(spec: TensorSpec, offset: int = 0, count: int | None = None) -> np.ndarray:
    """fp32 values (bf16-exact) of a spec, optionally a flat slice of it."""
    c = spec.count - offset if count is None else count
    return fill_values(c, spec.key, offset, spec.std, spec.mean)


def host_bits(spec: TensorSpec) -> np.ndarray:
    return fill_bf16_bits(spec.count, spec.key, 0, spec.std, spec.mean).reshape(spec.shape)


def pool_pages(spec: TensorSpec, pages: np.ndarray) -> np.ndarray:
    """Values of selected physical pages of a KV pool spec -> [len(pages), ...]."""
    per_page = int(np.prod(spec.shape[1:]))
    pages = np.ascontiguousarray(pages, np.int64)
    if pages.size and (pages.min() < 0 or pages.max() >= spec.shape[0]):
        raise IndexError("page id outside the pool")
    out = np.empty((len(pages),) + tuple(spec.shape[1:]), np.float32)
    if len(pages):
        _lib().synth_fill_pages_as_f32(out.ctypes.data, pages.ctypes.data, len(pages), per_page,
                                       spec.key, float(ih_mul(spec.std)),
                                       0.0 if spec.mean is None else float(spec.mean),
                                       0 if spec.mean is None else 1)
    return out


# ---------------------------------------------------------------- host views
class _LazyRows:
    """Row-indexable view of a [rows, cols] spec, generated on demand."""

    def __init__(self, spec: TensorSpec):
        self.spec = spec
        self.shape = spec.shape

    def __getitem__(self, idx):
        cols = self.spec.shape[1]
        if isinstance(idx, slice):
            start, stop, step = idx.indices(self.spec.shape[0])
            assert step == 1
            return host_values(self.spec, start * cols, (stop - start) * cols).reshape(-1, cols)
        rows = np.atleast_1d(np.asarray(idx, np.int64))
        out = np.stack([host_values(self.spec, int(r) * cols, cols) for r in rows])
        return out if np.ndim(idx) else out[0]


class _LazyLayers:
    def __init__(self, shape: ModelShape, seed: int):
        self.shape, self.seed = shape, seed

    def __len__(self):
        return self.shape.n_layers

    def __getitem__(self, l):
        if not 0 <= l < self.shape.n_layers:
            raise IndexError(l)
        return {k: host_values(s).reshape(s.shape) for k, s in
                layer_specs(self.shape, self.seed, l).items()}


def host_weights(shape: ModelShape, seed: int, lazy: bool = False) -> dict:
    """Host fp32 copies (bf16-exact) of the synthetic weights of a model.

    ``lazy`` generates each layer when it is indexed and embedding / LM-head
    rows on demand, so 8B/32B-class models can be walked layer by layer.
    """
    g = global_specs(shape, seed)
    if lazy:
        return {"embed": _LazyRows(g["embed"]), "lm_head": _LazyRows(g["lm_head"]),
                "final_norm": host_values(g["final_norm"]),
                "layers": _LazyLayers(shape, seed)}
    layers = _LazyLayers(shape, seed)
    return {"embed": host_values(g["embed"]).reshape(g["embed"].shape),
            "lm_head": host_values(g["lm_head"]).reshape(g["lm_head"].shape),
            "final_norm": host_values(g["final_norm"]),
            "layers": [layers[l] for l in range(shape.n_layers)]}


def host_pools(shape: ModelShape, seed: int, n_pages: int, layers=None) -> list:
    """Full host KV pools (fp32 values) for the given layers."""
    out = []
    for l in (range(shape.n_layers) if layers is None else layers):
        spec = kv_spec(shape, seed, l, n_pages)
        out.append(host_values(spec).reshape(spec.shape))
    return out
