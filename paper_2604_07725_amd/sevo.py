"""Thin Python binding of libsevo.so (argument marshalling only).

Every function here packs torch tensors into the C structs of
``include/sevo.h`` and calls the same-named C entry point; all arithmetic of
the decode step runs in the HIP kernels of the library.  PyTorch provides
device memory and the current stream.  There is no fallback: a missing or
unloadable library raises.
"""
from __future__ import annotations

import ctypes as C
import os
import re

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# SEVO_LIBRARY selects another build of the same library (the host-sanitized
# checking build); the default is the in-tree libsevo.so
LIB_PATH = os.environ.get("SEVO_LIBRARY") or os.path.join(_HERE, "libsevo.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "sevo.h")

OK, INVALID_ARGUMENT, UNSUPPORTED, WORKSPACE_TOO_SMALL, OUT_OF_MEMORY, HIP, BAD_PAGE_TABLE = range(7)
LINEAR_STORE, LINEAR_ADD, LINEAR_SWIGLU = 0, 1, 2
LINEAR_X_TILED, LINEAR_OUT_TILED = 1, 2
PACK_PLAIN, PACK_GATE_UP = 0, 1
# projection weights held in the packed layout, and how each is packed
PACKED_WEIGHTS = {"w_qkv": PACK_PLAIN, "w_o": PACK_PLAIN, "w_gate_up": PACK_GATE_UP,
                  "w_down": PACK_PLAIN, "lm_head": PACK_PLAIN, "w_router": PACK_PLAIN,
                  "w_expert_gate_up": PACK_GATE_UP, "w_expert_down": PACK_PLAIN}
PAGE_SIZE = 16
NOALLOC_SCRATCH_BYTES = 32 << 20   # SEVO_NOALLOC_SCRATCH_BYTES
PROF_KINDS = ["attn_split", "attn_combine", "qkv", "attn_out", "gate_up", "down", "lm_head",
              "norm", "rope_append", "sample", "embed", "attn_prefill", "moe_route",
              "moe_experts"]   # SEVO_PROF_* order

vp = C.c_void_p
i32 = C.c_int32
i64 = C.c_int64
u64 = C.c_uint64
f32 = C.c_float
sz = C.c_size_t


class ModelConfig(C.Structure):
    _fields_ = [("n_layers", i32), ("hidden", i32), ("n_q_heads", i32), ("n_kv_heads", i32),
                ("head_dim", i32), ("ffn", i32), ("vocab", i32), ("page_size", i32),
                ("max_position", i32), ("qk_norm", i32), ("rope_theta", f32), ("rms_eps", f32),
                ("n_experts", i32), ("n_experts_active", i32), ("expert_ffn", i32)]


class Weights(C.Structure):
    _fields_ = [("embed", vp), ("lm_head", vp), ("final_norm", vp),
                ("attn_norm", C.POINTER(vp)), ("w_qkv", C.POINTER(vp)), ("q_norm", C.POINTER(vp)),
                ("k_norm", C.POINTER(vp)), ("w_o", C.POINTER(vp)), ("ffn_norm", C.POINTER(vp)),
                ("w_gate_up", C.POINTER(vp)), ("w_down", C.POINTER(vp)),
                ("w_router", C.POINTER(vp)), ("w_expert_gate_up", C.POINTER(vp)),
                ("w_expert_down", C.POINTER(vp))]


class AttnArgs(C.Structure):
    _fields_ = [("n", i32), ("n_q_heads", i32), ("n_kv_heads", i32), ("head_dim", i32),
                ("page_size", i32), ("max_pages", i32), ("num_splits", i32), ("num_pages", i64),
                ("q", vp), ("kv_pool", vp), ("page_table", vp), ("seq_lens", vp),
                ("scale", f32), ("out", vp), ("workspace", vp), ("workspace_bytes", sz)]


class PrefillAttnArgs(C.Structure):
    _fields_ = [("n_seqs", i32), ("total_tokens", i32), ("max_seq_len", i32),
                ("n_q_heads", i32), ("n_kv_heads", i32), ("head_dim", i32), ("page_size", i32),
                ("max_pages", i32), ("num_pages", i64), ("q", vp), ("kv_pool", vp),
                ("page_table", vp), ("seq_starts", vp), ("start_pos", vp), ("scale", f32),
                ("out", vp)]


class PrefillArgs(C.Structure):
    _fields_ = [("n_seqs", i32), ("total_tokens", i32), ("max_seq_len", i32), ("tokens", vp),
                ("seq_starts", vp), ("start_pos", vp), ("page_table", vp), ("max_pages", i32),
                ("num_pages", i64), ("kv_pools", C.POINTER(vp)), ("conf_topk", i32),
                ("n_scored", i32), ("scored_rows", vp), ("out_conf", vp), ("out_row_conf", vp),
                ("workspace", vp), ("workspace_bytes", sz), ("moe_chunk", i32)]


class SampleArgs(C.Structure):
    _fields_ = [("logits", vp), ("n", i32), ("vocab", i32), ("ld", i64), ("temperature", f32),
                ("seed", u64), ("cand_uid", vp), ("positions", vp), ("out_tokens", vp),
                ("out_logprobs", vp), ("top_k", i32), ("top_p", f32), ("min_p", f32),
                ("conf_topk", i32), ("out_conf", vp), ("conf_sum", vp), ("workspace", vp),
                ("workspace_bytes", sz)]


class StepArgs(C.Structure):
    _fields_ = [("n", i32), ("tokens", vp), ("positions", vp), ("page_table", vp),
                ("max_pages", i32), ("num_pages", i64), ("kv_pools", C.POINTER(vp)),
                ("cand_uid", vp), ("seed", u64),
                ("temperature", f32), ("num_splits", i32), ("out_tokens", vp),
                ("out_logprobs", vp), ("out_logits", vp), ("top_k", i32), ("top_p", f32),
                ("min_p", f32), ("conf_topk", i32), ("out_conf", vp), ("conf_sum", vp),
                ("workspace", vp), ("workspace_bytes", sz), ("out_hidden", vp)]


class LinearArgs(C.Structure):
    _fields_ = [("m", i32), ("n_out", i32), ("k", i32), ("ldx", i32), ("mode", i32),
                ("k_splits", i32), ("flags", i32), ("x", vp), ("w", vp), ("out", vp),
                ("workspace", vp), ("workspace_bytes", sz)]


_SIGS = {
    "sevo_status_string": ([i32], C.c_char_p),
    "sevo_last_error": ([], C.c_char_p),
    "sevo_version": ([], C.c_char_p),
    "sevo_init_model": ([C.POINTER(ModelConfig), C.POINTER(Weights), C.POINTER(vp)], i32),
    "sevo_free_model": ([vp], None),
    "sevo_attn_decode": ([C.POINTER(AttnArgs), vp], i32),
    "sevo_attn_decode_noalloc": ([C.POINTER(AttnArgs), vp], i32),
    "sevo_attn_plan_splits": ([i32, i32, i32], i32),
    "sevo_attn_workspace_bytes": ([i32, i32, i32, i32, i32, i32], sz),
    "sevo_attn_prefill": ([C.POINTER(PrefillAttnArgs), vp], i32),
    "sevo_logprob_sample": ([C.POINTER(SampleArgs), vp], i32),
    "sevo_sample_workspace_bytes": ([i32, i32], sz),
    "sevo_group_confidence": ([vp, vp, vp, i32, i32, vp, vp], i32),
    "sevo_decode_step": ([vp, C.POINTER(StepArgs), vp], i32),
    "sevo_step_workspace_bytes": ([vp, i32, i32, i32], sz),
    "sevo_prefill_confidence": ([vp, C.POINTER(PrefillArgs), vp], i32),
    "sevo_moe_ffn": ([vp, i32, vp, i32, vp, vp, vp, vp, sz, vp], i32),
    "sevo_moe_workspace_bytes": ([vp, i32], sz),
    "sevo_hbm_read_probe": ([vp, sz, vp, i32, vp, vp], i32),
    "sevo_prefill_workspace_bytes": ([vp, i32, i32], sz),
    "sevo_embed": ([vp, vp, i32, i32, i32, vp, vp], i32),
    "sevo_rmsnorm": ([vp, vp, i32, i32, f32, vp, vp], i32),
    "sevo_add_rmsnorm": ([vp, vp, i32, vp, i32, i32, f32, vp, vp], i32),
    "sevo_linear": ([C.POINTER(LinearArgs), vp], i32),
    "sevo_linear_workspace_bytes": ([i32, i32, i32, i32], sz),
    "sevo_linear_plan": ([i32, i32, i32, i32, i32, C.POINTER(i32)], i32),
    "sevo_pack_weight": ([vp, vp, i32, i32, i32, vp], i32),
    "sevo_pack_kv": ([vp, vp, i64, i32, i32, vp, vp], i32),
    "sevo_qk_norm_rope_append": ([vp, i32, vp, i32, vp, vp, i32, i64, vp, vp, vp], i32),
    "sevo_fill_normal_bf16": ([vp, i64, u64, i64, f32, f32, i32, vp], i32),
    "sevo_validate_paging": ([vp, vp, i32, i32, i64, vp], i32),
    "sevo_profile_begin": ([i32, C.c_uint32], i32),
    "sevo_profile_end": ([C.POINTER(f32), C.POINTER(i32)], i32),
}

_lib = None


class SevoError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"sevo status {status}: {msg}")
        self.status = status


def lib():
    """Load libsevo.so (raises if it is missing: there is no fallback path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} not built: run __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def header_functions() -> list[str]:
    """Names of every function declared in include/sevo.h."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sevo_[a-z0-9_]+)\s*\(", text)))


def _check(status: int) -> None:
    if status != OK:
        raise SevoError(status, lib().sevo_last_error().decode())


def _stream(stream):
    if stream is None:
        return vp(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return vp(stream.cuda_stream)
    return vp(stream)


def _p(t):
    return None if t is None else vp(t.data_ptr())


def _workspace(nbytes: int, device, ws=None):
    if ws is not None:
        return ws
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


# ------------------------------------------------------------------ attention
def sevo_attn_plan_splits(n: int, n_kv_heads: int, max_pages: int) -> int:
    return int(lib().sevo_attn_plan_splits(n, n_kv_heads, max_pages))


def sevo_attn_workspace_bytes(n, n_q_heads, n_kv_heads, head_dim, max_pages, num_splits=0) -> int:
    return int(lib().sevo_attn_workspace_bytes(n, n_q_heads, n_kv_heads, head_dim, max_pages,
                                               num_splits))


def sevo_attn_decode(q, kv_pool, page_table, seq_lens, out=None, scale=None,
                     num_splits=0, workspace=None, stream=None):
    """o = paged GQA decode attention.  q [n, hq, d] bf16; kv_pool in the paged
    layout [P, hkv, 2, 16 d]; page_table int32 [n, max_pages]; seq_lens int32 [n]."""
    n, hq, d = q.shape
    hkv = kv_pool.shape[1]
    max_pages = page_table.shape[1]
    if out is None:
        out = torch.empty_like(q)
    need = sevo_attn_workspace_bytes(n, hq, hkv, d, max_pages, num_splits)
    ws = _workspace(need, q.device, workspace)
    a = AttnArgs(n=n, n_q_heads=hq, n_kv_heads=hkv, head_dim=d, page_size=PAGE_SIZE,
                 max_pages=max_pages, num_splits=num_splits, num_pages=kv_pool.shape[0],
                 q=_p(q), kv_pool=_p(kv_pool), page_table=_p(page_table),
                 seq_lens=_p(seq_lens), scale=float(d ** -0.5 if scale is None else scale),
                 out=_p(out), workspace=_p(ws), workspace_bytes=ws.numel())
    _check(lib().sevo_attn_decode(C.byref(a), _stream(stream)))
    return out


def sevo_attn_decode_noalloc(q, kv_pool, page_table, seq_lens, out, scale=None, num_splits=0,
                             stream=None):
    """The same attention with the split partials in the library's fixed device
    scratch (no workspace; ``out`` must be given, so nothing is allocated)."""
    n, hq, d = q.shape
    a = AttnArgs(n=n, n_q_heads=hq, n_kv_heads=kv_pool.shape[1], head_dim=d,
                 page_size=PAGE_SIZE, max_pages=page_table.shape[1], num_splits=num_splits,
                 num_pages=kv_pool.shape[0], q=_p(q), kv_pool=_p(kv_pool),
                 page_table=_p(page_table), seq_lens=_p(seq_lens),
                 scale=float(d ** -0.5 if scale is None else scale), out=_p(out), workspace=None,
                 workspace_bytes=0)
    _check(lib().sevo_attn_decode_noalloc(C.byref(a), _stream(stream)))
    return out


# ------------------------------------------------------------------ prefill
def sevo_attn_prefill(q, kv_pool, page_table, seq_starts, max_seq_len, start_pos=None, out=None,
                      scale=None, stream=None):
    """Causal GQA prefill attention.  q [T, hq, d] bf16 (sequences back to back);
    kv_pool [P, hkv, 2, 16 d]; page_table int32 [n_seqs, max_pages]; seq_starts
    int32 [n_seqs + 1] and start_pos int32 [n_seqs] (or None) on the device;
    max_seq_len: host bound of the sequence lengths."""
    T, hq, d = q.shape
    hkv = kv_pool.shape[1]
    n_seqs, max_pages = page_table.shape
    if out is None:
        out = torch.empty_like(q)
    a = PrefillAttnArgs(n_seqs=n_seqs, total_tokens=T, max_seq_len=int(max_seq_len),
                        n_q_heads=hq, n_kv_heads=hkv, head_dim=d, page_size=PAGE_SIZE,
                        max_pages=max_pages, num_pages=kv_pool.shape[0], q=_p(q),
                        kv_pool=_p(kv_pool), page_table=_p(page_table),
                        seq_starts=_p(seq_starts), start_pos=_p(start_pos),
                        scale=float(d ** -0.5 if scale is None else scale), out=_p(out))
    _check(lib().sevo_attn_prefill(C.byref(a), _stream(stream)))
    return out


# ------------------------------------------------------------------ sampling
def sevo_sample_workspace_bytes(n: int, vocab: int) -> int:
    return int(lib().sevo_sample_workspace_bytes(n, vocab))


def sevo_logprob_sample(logits, temperature, seed, cand_uid, positions, out_tokens=None,
                        out_logprobs=None, workspace=None, stream=None, vocab=None,
                        conf_topk=0, out_conf=None, conf_sum=None, top_k=0, top_p=1.0,
                        min_p=0.0):
    """(ids int32 [n], logprobs fp32 [n]) from fp32 logits [n, ld] (the first
    ``vocab`` columns, default all).  ``top_k`` > 0: truncated sampling with
    ``top_p`` / ``min_p`` inside the top-k set.  With ``conf_topk`` > 0 also the
    per-token self-confidence: returned as a third element (``out_conf``) and/or
    added to ``conf_sum``."""
    n = logits.shape[0]
    vocab = logits.shape[1] if vocab is None else vocab
    if conf_topk and out_conf is None:
        out_conf = torch.empty(n, dtype=torch.float32, device=logits.device)
    if out_tokens is None:
        out_tokens = torch.empty(n, dtype=torch.int32, device=logits.device)
    if out_logprobs is None:
        out_logprobs = torch.empty(n, dtype=torch.float32, device=logits.device)
    ws = _workspace(sevo_sample_workspace_bytes(n, vocab), logits.device, workspace)
    a = SampleArgs(logits=_p(logits), n=n, vocab=vocab, ld=logits.stride(0),
                   temperature=float(temperature), seed=int(seed), cand_uid=_p(cand_uid),
                   positions=_p(positions), out_tokens=_p(out_tokens),
                   out_logprobs=_p(out_logprobs), top_k=int(top_k), top_p=float(top_p),
                   min_p=float(min_p), conf_topk=int(conf_topk), out_conf=_p(out_conf),
                   conf_sum=_p(conf_sum), workspace=_p(ws), workspace_bytes=ws.numel())
    _check(lib().sevo_logprob_sample(C.byref(a), _stream(stream)))
    if conf_topk:
        return out_tokens, out_logprobs, out_conf
    return out_tokens, out_logprobs


def sevo_group_confidence(conf_sum, token_counts, groups, out=None, stream=None):
    """GC [n_groups] from per-candidate confidence sums, token counts (int32)
    and groups int32 [n_groups, K] of candidate indices."""
    n_groups, k = groups.shape
    if out is None:
        out = torch.empty(n_groups, dtype=torch.float32, device=conf_sum.device)
    _check(lib().sevo_group_confidence(_p(conf_sum), _p(token_counts), _p(groups), n_groups, k,
                                       _p(out), _stream(stream)))
    return out


# ------------------------------------------------------------------ sub-steps
def sevo_embed(embed, tokens, x=None, stream=None):
    n = tokens.shape[0]
    hidden = embed.shape[1]
    if x is None:
        x = torch.empty(n, hidden, dtype=torch.float32, device=embed.device)
    _check(lib().sevo_embed(_p(embed), _p(tokens), n, hidden, embed.shape[0], _p(x),
                            _stream(stream)))
    return x


def sevo_rmsnorm(x, gain, eps, out=None, stream=None):
    rows, cols = x.shape
    if out is None:
        out = torch.empty(rows, cols, dtype=torch.bfloat16, device=x.device)
    _check(lib().sevo_rmsnorm(_p(x), _p(gain), rows, cols, float(eps), _p(out), _stream(stream)))
    return out


def sevo_add_rmsnorm(x, partials, gain, eps, out=None, stream=None):
    """x fp32 [rows, cols] += the partials fp32 [S, rows, cols] (in s order; None
    for none), in place; returns RMSNorm(x) * gain as bf16 in the tiled
    activation layout (a flat buffer of ceil(rows / 16) * 16 rows)."""
    rows, cols = x.shape
    S = 0 if partials is None else partials.shape[0]
    if out is None:
        out = torch.zeros(-(-rows // 16) * 16 * cols, dtype=torch.bfloat16, device=x.device)
    _check(lib().sevo_add_rmsnorm(_p(x), _p(partials) if S else None, S, _p(gain), rows, cols,
                                  float(eps), _p(out), _stream(stream)))
    return out


def sevo_linear_workspace_bytes(m, n_out, k, k_splits=0) -> int:
    return int(lib().sevo_linear_workspace_bytes(m, n_out, k, k_splits))


def sevo_linear_plan(m, n_out, k, k_splits=0, mode=LINEAR_STORE):
    """(k splits, k per split, 16-row weight blocks per workgroup) of the skinny kernel."""
    plan = (C.c_int32 * 3)()
    _check(lib().sevo_linear_plan(m, n_out, k, k_splits, mode, plan))
    return tuple(int(v) for v in plan)


def sevo_linear(x, w, mode=LINEAR_STORE, out=None, k_splits=0, workspace=None, stream=None,
                m=None, x_tiled=False, out_tiled=False):
    """Y = x w^T (bf16 in, fp32 accumulate) with the STORE / ADD / SWIGLU epilogue.

    w [n_out, k] is in the packed weight layout (``sevo_pack_weight``).  x is
    row-major [m, k] (row stride from the tensor), or with ``x_tiled`` a buffer
    in the tiled activation layout, whose row count ``m`` must be given.
    ``out_tiled`` (SWIGLU only) writes the bf16 product in the tiled layout."""
    n_out, k = w.shape
    if x_tiled:
        if m is None:
            raise ValueError("x_tiled needs m")
        ldx = k
    else:
        m = x.shape[0]
        ldx = x.stride(0)
    if out is None:
        if mode == LINEAR_SWIGLU:
            rows = -(-m // 16) * 16 if out_tiled else m
            out = torch.empty(rows, n_out // 2, dtype=torch.bfloat16, device=x.device)
        else:
            out = torch.zeros(m, n_out, dtype=torch.float32, device=x.device)
    ws = _workspace(sevo_linear_workspace_bytes(m, n_out, k, k_splits), x.device, workspace)
    flags = (LINEAR_X_TILED if x_tiled else 0) | (LINEAR_OUT_TILED if out_tiled else 0)
    a = LinearArgs(m=m, n_out=n_out, k=k, ldx=ldx, mode=mode, k_splits=k_splits, flags=flags,
                   x=_p(x), w=_p(w), out=_p(out), workspace=_p(ws), workspace_bytes=ws.numel())
    _check(lib().sevo_linear(C.byref(a), _stream(stream)))
    return out


def sevo_pack_weight(src, kind=PACK_PLAIN, dst=None, stream=None):
    """Row-major bf16 [n_out, k] -> a new tensor of the same shape in the packed layout."""
    n_out, k = src.shape
    if dst is None:
        dst = torch.empty_like(src)
    _check(lib().sevo_pack_weight(_p(src), _p(dst), n_out, k, int(kind), _stream(stream)))
    return dst


def sevo_pack_kv(k_pool, v_pool, kv_pool=None, stream=None):
    """Plain K and V pools bf16 [pages, hkv, 16, d] -> the fused pool [pages, hkv, 2, 16 d]."""
    pages, hkv, slots, d = k_pool.shape
    if kv_pool is None:
        kv_pool = torch.empty(pages, hkv, 2, slots * d, dtype=k_pool.dtype, device=k_pool.device)
    _check(lib().sevo_pack_kv(_p(k_pool), _p(v_pool), pages, hkv, d, _p(kv_pool),
                              _stream(stream)))
    return kv_pool


def sevo_qk_norm_rope_append(model, layer, qkv, positions, page_table, kv_pool, q_out=None,
                             stream=None):
    n = qkv.shape[0]
    cfg = model.config
    if q_out is None:
        q_out = torch.empty(n, cfg.n_q_heads, cfg.head_dim, dtype=torch.bfloat16,
                            device=qkv.device)
    _check(lib().sevo_qk_norm_rope_append(model.handle, layer, _p(qkv), n, _p(positions),
                                          _p(page_table), page_table.shape[1], kv_pool.shape[0],
                                          _p(q_out), _p(kv_pool), _stream(stream)))
    return q_out


def sevo_fill_normal_bf16(dst, key, offset=0, std=1.0, mean=None, stream=None):
    """Device twin of the seeded input generator: fills a bf16 tensor."""
    from .synth import ih_mul
    _check(lib().sevo_fill_normal_bf16(_p(dst), dst.numel(), int(key), int(offset),
                                       float(ih_mul(std)), 0.0 if mean is None else float(mean),
                                       0 if mean is None else 1, _stream(stream)))
    return dst


def sevo_validate_paging(page_table, lengths, num_pages, stream=None):
    n, max_pages = page_table.shape
    _check(lib().sevo_validate_paging(_p(page_table), _p(lengths), n, max_pages, int(num_pages),
                                      _stream(stream)))


def sevo_profile_begin(max_launches: int, kinds=("attn_split", "attn_combine")) -> None:
    """Open a recording that times the launches of the named kinds (PROF_KINDS)."""
    mask = 0
    for k in kinds:
        mask |= 1 << PROF_KINDS.index(k)
    _check(lib().sevo_profile_begin(int(max_launches), mask))


def sevo_profile_end() -> dict:
    """{kind: (summed ms, launches)} of the recording, for kinds with launches."""
    n = len(PROF_KINDS)
    ms = (f32 * n)()
    cnt = (i32 * n)()
    _check(lib().sevo_profile_end(ms, cnt))
    return {k: (ms[i], cnt[i]) for i, k in enumerate(PROF_KINDS) if cnt[i]}


# ------------------------------------------------------------------ model + step
class Model:
    """A sevo_model handle plus the bf16 device weights it borrows."""

    def __init__(self, shape, tensors: dict, max_position: int):
        self.shape = shape
        self.tensors = tensors  # keeps the weights alive
        L = shape.n_layers
        self.config = ModelConfig(
            n_layers=L, hidden=shape.hidden, n_q_heads=shape.n_q_heads,
            n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim, ffn=shape.ffn,
            vocab=shape.vocab, page_size=PAGE_SIZE, max_position=int(max_position),
            qk_norm=1 if shape.qk_norm else 0, rope_theta=float(shape.rope_theta),
            rms_eps=float(shape.rms_eps), n_experts=int(shape.n_experts),
            n_experts_active=int(shape.top_k), expert_ffn=int(shape.expert_ffn))

        def table(name):
            arr = (vp * L)(*[t[name].data_ptr() if name in t else None
                             for t in tensors["layers"]])
            return arr

        ffn = (("w_router", "w_expert_gate_up", "w_expert_down") if shape.is_moe
               else ("w_gate_up", "w_down"))
        self._tables = {k: table(k) for k in ("attn_norm", "w_qkv", "q_norm", "k_norm", "w_o",
                                               "ffn_norm") + ffn}
        self.weights = Weights(embed=_p(tensors["embed"]), lm_head=_p(tensors["lm_head"]),
                               final_norm=_p(tensors["final_norm"]),
                               **{k: C.cast(v, C.POINTER(vp)) for k, v in self._tables.items()})
        h = vp()
        _check(lib().sevo_init_model(C.byref(self.config), C.byref(self.weights), C.byref(h)))
        self.handle = h

    def close(self):
        if self.handle:
            lib().sevo_free_model(self.handle)
            self.handle = vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def sevo_init_model(shape, tensors: dict, max_position: int) -> Model:
    return Model(shape, tensors, max_position)


def sevo_step_workspace_bytes(model: Model, n: int, max_pages: int, num_splits: int = 0) -> int:
    return int(lib().sevo_step_workspace_bytes(model.handle, n, max_pages, num_splits))


class StepBuffers:
    """Pre-built argument struct for repeated decode steps (no per-step allocation)."""

    def __init__(self, model: Model, tokens, positions, page_table, kv_pools, cand_uid,
                 seed, temperature, num_splits=0, keep_logits=False, workspace=None,
                 conf_topk=0, conf_sum=None, top_k=0, top_p=1.0, min_p=0.0,
                 keep_hidden=False):
        n = tokens.shape[0]
        dev = tokens.device
        self.model = model
        self.out_hidden = (torch.empty(model.shape.n_layers + 1, n, model.shape.hidden,
                                       dtype=torch.float32, device=dev) if keep_hidden else None)
        self.out_tokens = torch.empty(n, dtype=torch.int32, device=dev)
        self.out_logprobs = torch.empty(n, dtype=torch.float32, device=dev)
        self.out_logits = (torch.empty(n, model.shape.vocab, dtype=torch.float32, device=dev)
                           if keep_logits else None)
        self.out_conf = (torch.empty(n, dtype=torch.float32, device=dev) if conf_topk else None)
        self.conf_sum = conf_sum
        need = sevo_step_workspace_bytes(model, n, page_table.shape[1], num_splits)
        self.workspace = _workspace(need, dev, workspace)
        L = model.shape.n_layers
        self._kv = (vp * L)(*[p.data_ptr() for p in kv_pools])
        self.keep = (tokens, positions, page_table, kv_pools, cand_uid)
        self.args = StepArgs(
            n=n, tokens=_p(tokens), positions=_p(positions), page_table=_p(page_table),
            max_pages=page_table.shape[1], num_pages=kv_pools[0].shape[0],
            kv_pools=C.cast(self._kv, C.POINTER(vp)),
            cand_uid=_p(cand_uid), seed=int(seed), temperature=float(temperature),
            num_splits=num_splits, out_tokens=_p(self.out_tokens),
            out_logprobs=_p(self.out_logprobs), out_logits=_p(self.out_logits),
            top_k=int(top_k), top_p=float(top_p), min_p=float(min_p),
            conf_topk=int(conf_topk), out_conf=_p(self.out_conf), conf_sum=_p(conf_sum),
            workspace=_p(self.workspace), workspace_bytes=self.workspace.numel(),
            out_hidden=_p(self.out_hidden))

    def run(self, stream=None):
        _check(lib().sevo_decode_step(self.model.handle, C.byref(self.args), _stream(stream)))
        return self.out_tokens, self.out_logprobs


def sevo_decode_step(model: Model, tokens, positions, page_table, kv_pools, cand_uid,
                     seed, temperature=1.0, num_splits=0, keep_logits=False, stream=None,
                     conf_topk=0, conf_sum=None, top_k=0, top_p=1.0, min_p=0.0,
                     keep_hidden=False, workspace=None):
    """One decode step of the population; returns (ids, logprobs[, logits][, conf]
    [, hidden]), hidden = the residual stream entering each layer and after the
    last [n_layers + 1, n, hidden].  ``workspace``: a caller's uint8 device
    buffer of at least sevo_step_workspace_bytes (else one is allocated)."""
    b = StepBuffers(model, tokens, positions, page_table, kv_pools, cand_uid, seed,
                    temperature, num_splits, keep_logits, conf_topk=conf_topk, conf_sum=conf_sum,
                    top_k=top_k, top_p=top_p, min_p=min_p, keep_hidden=keep_hidden,
                    workspace=workspace)
    ids, lps = b.run(stream)
    out = (ids, lps) + ((b.out_logits,) if keep_logits else ()) + \
        ((b.out_conf,) if conf_topk else ()) + ((b.out_hidden,) if keep_hidden else ())
    return out


# ------------------------------------------------------------------ mixture of experts
def sevo_moe_ffn(model: Model, layer: int, h_tiled, n: int, stream=None, partials=None):
    """The MoE FFN of one layer on normed inputs in the tiled activation layout
    (n rows).  Returns (experts int32 [n, k], weights fp32 [n, k],
    partials fp32 [k, n, hidden]); ``partials`` may be given (written in full)."""
    shape = model.shape
    k = shape.top_k
    dev = h_tiled.device
    ex = torch.empty(n, k, dtype=torch.int32, device=dev)
    wt = torch.empty(n, k, dtype=torch.float32, device=dev)
    part = (torch.empty(k, n, shape.hidden, dtype=torch.float32, device=dev)
            if partials is None else partials)
    if (part.shape != (k, n, shape.hidden) or part.dtype != torch.float32
            or not part.is_contiguous()):
        raise ValueError("partials must be a contiguous fp32 [k, n, hidden] tensor")
    ws = _workspace(int(lib().sevo_moe_workspace_bytes(model.handle, n)), dev)
    _check(lib().sevo_moe_ffn(model.handle, int(layer), _p(h_tiled), int(n), _p(ex), _p(wt),
                              _p(part), _p(ws), ws.numel(), _stream(stream)))
    return ex, wt, part


# ------------------------------------------------------------------ read probe
def sevo_hbm_read_probe(buf, page_order=None, grid=32768, sink=None, stream=None):
    """Read every byte of the device tensor ``buf`` once (sequentially, or as
    8 KB pages in the int32 order ``page_order``); returns the sink tensor."""
    if sink is None:
        sink = torch.empty(grid * 16, dtype=torch.uint8, device=buf.device)
    nbytes = buf.numel() * buf.element_size()
    _check(lib().sevo_hbm_read_probe(_p(buf), nbytes, _p(page_order), int(grid), _p(sink),
                                     _stream(stream)))
    return sink


# ------------------------------------------------------------------ confidence engine
def sevo_prefill_workspace_bytes(model: Model, total_tokens: int, n_scored: int) -> int:
    return int(lib().sevo_prefill_workspace_bytes(model.handle, int(total_tokens), int(n_scored)))


class PrefillBuffers:
    """Argument struct and outputs of one confidence-engine call shape (the
    workspace is allocated once; ``run`` only enqueues kernels)."""

    def __init__(self, model: Model, tokens, seq_starts, page_table, kv_pools, scored_rows,
                 conf_topk, max_seq_len, start_pos=None, keep_row_conf=True, workspace=None,
                 moe_chunk=0):
        T = tokens.shape[0]
        n_seqs = seq_starts.shape[0] - 1
        dev = tokens.device
        R = 0 if scored_rows is None else scored_rows.shape[0]
        self.model = model
        self.out_conf = torch.empty(n_seqs, dtype=torch.float32, device=dev)
        self.out_row_conf = (torch.empty(max(R, 1), dtype=torch.float32, device=dev)
                             if keep_row_conf else None)
        need = sevo_prefill_workspace_bytes(model, max(T, 1), R)
        self.workspace = _workspace(need, dev, workspace)
        L = model.shape.n_layers
        if not isinstance(kv_pools, (list, tuple)):
            kv_pools = [kv_pools] * L
        self._kv = (vp * L)(*[p.data_ptr() for p in kv_pools])
        self.keep = (tokens, seq_starts, page_table, kv_pools, scored_rows, start_pos)
        self.args = PrefillArgs(
            n_seqs=n_seqs, total_tokens=T, max_seq_len=int(max_seq_len), tokens=_p(tokens),
            seq_starts=_p(seq_starts), start_pos=_p(start_pos), page_table=_p(page_table),
            max_pages=page_table.shape[1], num_pages=kv_pools[0].shape[0],
            kv_pools=C.cast(self._kv, C.POINTER(vp)), conf_topk=int(conf_topk), n_scored=R,
            scored_rows=_p(scored_rows), out_conf=_p(self.out_conf),
            out_row_conf=_p(self.out_row_conf), workspace=_p(self.workspace),
            workspace_bytes=self.workspace.numel(), moe_chunk=int(moe_chunk))

    def run(self, stream=None):
        _check(lib().sevo_prefill_confidence(self.model.handle, C.byref(self.args),
                                             _stream(stream)))
        return self.out_conf
