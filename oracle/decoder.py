"""One population decode step, written as its plain definition (test infrastructure).

What is computed is the step the method section repeats for every candidate
of a population during LLM aggregation: the assigned model reads the K
concatenated candidates of its group as context (already in the candidate's
KV cache) and produces the next token of the refined trajectory, together
with that token's log-probability under the model (the per-token
log-probabilities that the fitness signal, Eq. 1, consumes).  Algorithm 1's
aggregation line runs this step for the whole population at once.

The paper gives no architecture for the models it serves; the decoder below
is the pre-norm GQA transformer of the Qwen3 family that the workloads are
shaped after (RMSNorm, per-head QK-RMSNorm, rotate-half RoPE, SwiGLU FFN).
Sampling is exact full-vocabulary categorical sampling at temperature T (the
temperature-1, top-k off, top-p 1 row of the generation hyper-parameter
table), realised as Gumbel-max with counter-based noise (see philox.py).

Paged KV layout (one pool per layer; page size 16; head_dim a multiple of 32):
    pool [num_pages][n_kv_heads][2][16 head_dim]: per (page, head) the K tile,
    then the V tile.
    K tile: dims in blocks of 32, each block token-major -- element (slot s,
            dim e) at ((e // 32) * 16 + s) * 32 + e % 32
    V tile: dim-major -- element (s, e) at e * 16 + s
    logical key t of candidate i -> page page_table[i][t // 16], slot t % 16.

Everything here is float64.  bf16 storage points of the GPU path are mirrored
with round-to-nearest-even when ``mirror`` is true.
"""
from __future__ import annotations

import numpy as np

from .bf16 import round_bf16
from .philox import gumbel_noise

PAGE = 16


def _ident(x):
    return np.asarray(x, np.float64)


def _f32(x):
    return np.asarray(x, np.float64).astype(np.float32).astype(np.float64)


# ------------------------------------------------------------------ elementary ops
def rms_norm(x, gain, eps):
    """x / sqrt(mean(x^2) + eps) * gain over the last axis."""
    x = np.asarray(x, np.float64)
    inv = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * inv * np.asarray(gain, np.float64)


def rope_rotate(u, position, theta):
    """Rotate-half RoPE of the last axis (size d) at an integer position.

    For m < d/2 the pair (u[m], u[m + d/2]) is rotated by the angle
    position * theta^(-2m/d).  ``position`` may be a scalar or broadcast over
    the leading axes (``position`` broadcastable to ``u.shape[:-1]``).
    """
    u = np.asarray(u, np.float64)
    d = u.shape[-1]
    h = d // 2
    inv_freq = np.power(float(theta), -2.0 * np.arange(h, dtype=np.float64) / d)
    phi = np.asarray(position, np.float64)[..., None] * inv_freq
    c, s = np.cos(phi), np.sin(phi)
    a, b = u[..., :h], u[..., h:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(z):
    z = np.asarray(z, np.float64)
    return z / (1.0 + np.exp(-z))


def log_softmax(z):
    z = np.asarray(z, np.float64)
    m = np.max(z, axis=-1, keepdims=True)
    return z - (m + np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True)))


# ------------------------------------------------------------------ attention
def attention_dense(q, K, V, scale):
    """Decode attention of one candidate.

    q [hq, d]; K, V [hkv, L, d].  Query head j reads KV head j // (hq / hkv)
    (contiguous groups).  o_j = softmax(scale * K_c q_j) V_c.  Returns [hq, d].
    """
    q = np.asarray(q, np.float64)
    K = np.asarray(K, np.float64)
    V = np.asarray(V, np.float64)
    hq, d = q.shape
    hkv = K.shape[0]
    g = hq // hkv
    out = np.empty((hq, d))
    for j in range(hq):
        c = j // g
        s = (K[c] @ q[j]) * scale
        a = np.exp(s - s.max())
        a /= a.sum()
        out[j] = a @ V[c]
    return out


def split_bounds(n_keys, num_splits, page=PAGE):
    """Key ranges of a page-granular split: split s owns logical pages
    [s * ceil(P/S), (s + 1) * ceil(P/S)) of the candidate's P pages."""
    n_pages = -(-n_keys // page)
    per = -(-n_pages // num_splits)
    out = []
    for s in range(num_splits):
        lo = min(s * per * page, n_keys)
        hi = min((s + 1) * per * page, n_keys)
        out.append((lo, hi))
    return out


def attention_split(q, K, V, scale, bounds):
    """The same attention computed split-wise and combined.

    Each split s over keys [lo, hi) yields m_s = max score (-inf when empty),
    l_s = sum exp(score - m_s), acc_s = sum exp(score - m_s) V.  The combine
    takes m = max_s m_s and o = sum_s e^(m_s - m) acc_s / sum_s e^(m_s - m) l_s.
    """
    q = np.asarray(q, np.float64)
    hq, d = q.shape
    hkv = K.shape[0]
    g = hq // hkv
    out = np.empty((hq, d))
    for j in range(hq):
        c = j // g
        ms, ls, accs = [], [], []
        for lo, hi in bounds:
            if hi <= lo:
                ms.append(-np.inf)
                ls.append(0.0)
                accs.append(np.zeros(d))
                continue
            s = (np.asarray(K[c, lo:hi], np.float64) @ q[j]) * scale
            m = s.max()
            e = np.exp(s - m)
            ms.append(m)
            ls.append(e.sum())
            accs.append(e @ np.asarray(V[c, lo:hi], np.float64))
        m = max(ms)
        w = np.array([np.exp(mi - m) if np.isfinite(mi) else 0.0 for mi in ms])
        out[j] = sum(wi * a for wi, a in zip(w, accs)) / float(np.dot(w, ls))
    return out


def k_tile_offset(slot, dim):
    """Position of (slot, dim) inside a K tile (dims in blocks of 32, token-major)."""
    return ((dim // 32) * PAGE + slot) * 32 + dim % 32


def v_tile_offset(slot, dim):
    """Position of (slot, dim) inside a V tile (dim-major)."""
    return dim * PAGE + slot


def gather_kv(kv_pool, pages, n_keys):
    """Logical K, V [hkv, n_keys, d] of one candidate from its page list.

    Logical key t is slot t % 16 of physical page pages[t // 16].  The offsets
    of the tile layout are read as index decompositions: a K tile element
    (s, e) at ((e // 32) * 16 + s) * 32 + e % 32 is entry [e // 32][s][e % 32]
    of the tile viewed as [d / 32][16][32]; a V tile element (s, e) at
    e * 16 + s is entry [e][s] of the tile viewed as [d][16].
    """
    kv = np.asarray(kv_pool)
    hkv, d = kv.shape[1], kv.shape[3] // PAGE
    pg = np.asarray(pages, np.int64)[: -(-n_keys // PAGE)]
    tiles = kv[pg]                      # [n_pages][hkv][2][16 d], logical page order
    K = tiles[:, :, 0].reshape(len(pg), hkv, d // 32, PAGE, 32).transpose(1, 0, 3, 2, 4)
    V = tiles[:, :, 1].reshape(len(pg), hkv, d, PAGE).transpose(1, 0, 3, 2)
    K = K.reshape(hkv, len(pg) * PAGE, d)[:, :n_keys].astype(np.float64)
    V = V.reshape(hkv, len(pg) * PAGE, d)[:, :n_keys].astype(np.float64)
    return K, V


def paged_attention(q, kv_pool, page_table, seq_lens, scale):
    """Decode attention for a population: q [N, hq, d] -> [N, hq, d]."""
    q = np.asarray(q, np.float64)
    out = np.empty_like(q)
    for i in range(q.shape[0]):
        K, V = gather_kv(kv_pool, page_table[i], int(seq_lens[i]))
        out[i] = attention_dense(q[i], K, V, scale)
    return out


def prefill_attention(q, kv_pool, page_table, seq_starts, start_pos, scale):
    """Causal attention of a prefill batch (the scoring pass of the confidence
    engine): token t of sequence s sits at position start_pos[s] + t -
    seq_starts[s] and attends to the keys 0..that position of the sequence
    (page-table row s).  q [T, hq, d] -> [T, hq, d]."""
    q = np.asarray(q, np.float64)
    out = np.empty_like(q)
    for s in range(len(seq_starts) - 1):
        a, b = int(seq_starts[s]), int(seq_starts[s + 1])
        if b <= a:
            continue
        p0 = 0 if start_pos is None else int(start_pos[s])
        K, V = gather_kv(kv_pool, page_table[s], p0 + b - a)
        for t in range(a, b):
            n = p0 + (t - a) + 1
            out[t] = attention_dense(q[t], K[:, :n], V[:, :n], scale)
    return out


def append_kv(kv_pool, page_table, positions, k, v):
    """Write key/value number p_i of every candidate into its page slot."""
    d = np.asarray(k).shape[-1]
    e = np.arange(d)
    for i, p in enumerate(np.asarray(positions, np.int64)):
        page = int(page_table[i][p // PAGE])
        tiles = kv_pool[page]              # [hkv][2][16 d] view of the page
        tiles[:, 0, k_tile_offset(p % PAGE, e)] = k[i]
        tiles[:, 1, v_tile_offset(p % PAGE, e)] = v[i]


# ------------------------------------------------------------------ mixture of experts
def moe_route(logits, top_k, decision_dtype=np.float32):
    """Experts and weights of each token: the top_k largest router logits
    (value descending, ties to the lower expert index; the choice is taken in
    ``decision_dtype``, the kernel's fp32) and a softmax over the selected
    logits -- the router's softmax probabilities of the selected experts,
    renormalised to sum to one.  ``gap`` = the float64 k-th minus (k+1)-th
    largest logit, so a caller can tell choices rounding may flip.
    Returns sel int64 [N, k], w float64 [N, k], gap float64 [N]."""
    logits = np.asarray(logits, np.float64)
    N, E = logits.shape
    dec = logits.astype(decision_dtype).astype(np.float64)
    sel = np.empty((N, top_k), np.int64)
    w = np.empty((N, top_k))
    gap = np.empty(N)
    for t in range(N):
        order = np.lexsort((np.arange(E), -dec[t]))
        sel[t] = order[:top_k]
        z = logits[t, sel[t]]
        e = np.exp(z - z.max())
        w[t] = e / e.sum()
        srt = np.sort(logits[t])[::-1]
        gap[t] = srt[top_k - 1] - srt[top_k] if top_k < E else np.inf
    return sel, w, gap


def moe_ffn(shape, lw, h2, mirror=True):
    """The mixture-of-experts FFN on normed inputs h2 [N, H]:
    sum over the token's selected experts e of w_e * (silu(h2 W_g[e]^T) *
    (h2 W_u[e]^T)) W_d[e]^T.  Returns (out [N, H], routing gap [N])."""
    rb = round_bf16 if mirror else _ident
    keep32 = _f32 if mirror else _ident
    Fe = shape.expert_ffn
    h2 = np.asarray(h2, np.float64)
    logits = keep32(h2 @ np.asarray(lw["w_router"], np.float64).T)
    sel, w, gap = moe_route(logits, shape.top_k)
    wgu = lw["w_expert_gate_up"]
    wd = lw["w_expert_down"]
    # y[t, j] = w_{t,j} * expert sel[t, j] applied to h2[t]; an expert's
    # matrices are read once for all the rows routed to it
    y = np.zeros((h2.shape[0], shape.top_k, h2.shape[1]))
    for e in np.unique(sel):
        t, j = np.nonzero(sel == e)
        gu = h2[t] @ np.asarray(wgu[e], np.float64).T
        a = rb(silu(gu[:, :Fe]) * gu[:, Fe:])
        y[t, j] = w[t, j][:, None] * (a @ np.asarray(wd[e], np.float64).T)
    out = np.zeros_like(h2)
    for j in range(shape.top_k):      # the k slots, summed in slot order
        out += y[:, j]
    return out, gap


# ------------------------------------------------------------------ decoder
def decoder_layer(shape, lw, x, positions, kv_pool, page_table, mirror=True, stats=None):
    """One pre-norm GQA decoder layer for the population (updates x, appends KV).

    x [N, H] residual stream.  Steps: RMSNorm, QKV projection, per-head
    QK-RMSNorm, RoPE at p_i, append k and v as key p_i, attention over keys
    0..p_i, output projection + residual, RMSNorm, SwiGLU FFN (or the
    mixture of experts) + residual.  ``stats`` (a dict) collects the smallest
    routing gap of MoE layers under "route_gap".
    """
    rb = round_bf16 if mirror else _ident
    keep32 = _f32 if mirror else _ident
    N = x.shape[0]
    hq, hkv, D = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    F = shape.ffn
    eps = shape.rms_eps
    pos = np.asarray(positions, np.int64)

    h = rb(rms_norm(x, lw["attn_norm"], eps))
    qkv = h @ np.asarray(lw["w_qkv"], np.float64).T
    q = qkv[:, : hq * D].reshape(N, hq, D)
    k = qkv[:, hq * D: (hq + hkv) * D].reshape(N, hkv, D)
    v = qkv[:, (hq + hkv) * D:].reshape(N, hkv, D)
    if shape.qk_norm:
        q = rms_norm(q, lw["q_norm"], eps)
        k = rms_norm(k, lw["k_norm"], eps)
    q = rb(rope_rotate(q, pos[:, None], shape.rope_theta))
    k = rb(rope_rotate(k, pos[:, None], shape.rope_theta))
    v = rb(v)
    append_kv(kv_pool, page_table, pos, k, v)
    o = paged_attention(q, kv_pool, page_table, pos + 1, 1.0 / np.sqrt(D))
    o = rb(o).reshape(N, hq * D)
    x = keep32(x + o @ np.asarray(lw["w_o"], np.float64).T)
    h2 = rb(rms_norm(x, lw["ffn_norm"], eps))
    if shape.is_moe:
        y, gap = moe_ffn(shape, lw, h2, mirror)
        if stats is not None:
            stats["route_gap"] = min(stats.get("route_gap", np.inf), float(gap.min()))
        return keep32(x + y)
    gu = h2 @ np.asarray(lw["w_gate_up"], np.float64).T
    a = rb(silu(gu[:, :F]) * gu[:, F:])
    x = keep32(x + a @ np.asarray(lw["w_down"], np.float64).T)
    return x


def lm_logits(shape, final_norm, lm_head, x, mirror=True, chunk=16384):
    """logits = RMSNorm(x) * g_final . W_lm^T, computed in vocab chunks."""
    rb = round_bf16 if mirror else _ident
    hf = rb(rms_norm(x, final_norm, shape.rms_eps))
    V = lm_head.shape[0]
    out = np.empty((x.shape[0], V))
    for v0 in range(0, V, chunk):
        out[:, v0:v0 + chunk] = hf @ np.asarray(lm_head[v0:v0 + chunk], np.float64).T
    return _f32(out) if mirror else out


def logprob_sample(logits, temperature, seed, uids, positions, noise=None,
                   decision_dtype=np.float32, details=None):
    """Gumbel-max sample and its log-probability, per candidate.

    z = logits / T;  id = argmax_v (z_v + G_v) with ties to the lowest v;
    lp = log_softmax(z)[id].  T == 0 means greedy: id = argmax logits and lp
    from T = 1.  The argmax decision is taken in ``decision_dtype`` (the
    kernel's fp32); ``gap`` is the float64 top-1 minus top-2 perturbed value,
    so a caller can tell decisions that rounding may flip.
    ``noise`` [N, V] overrides the Philox noise (for pins).  ``details`` (a
    dict) receives "pert" [N, V], the float64 perturbed values the decision is
    taken on, and "logp" [N, V], log_softmax(z) of every vocabulary entry.
    Returns ids int64 [N], lps float64 [N], gaps float64 [N].
    """
    logits = np.asarray(logits, np.float64)
    N, V = logits.shape
    ids = np.empty(N, np.int64)
    lps = np.empty(N)
    gaps = np.empty(N)
    if details is not None:
        details["pert"] = np.empty((N, V))
        details["logp"] = np.empty((N, V))
    for i in range(N):
        if temperature == 0:
            z = logits[i]
            pert = z
            pert_dec = z.astype(decision_dtype)
        else:
            z = logits[i] / float(temperature)
            G = (gumbel_noise(V, int(positions[i]), int(uids[i]), int(seed)) if noise is None
                 else np.asarray(noise[i], np.float64))
            pert = z + G
            pert_dec = z.astype(decision_dtype) + G.astype(decision_dtype)
        ids[i] = int(np.argmax(pert_dec))          # first maximum = lowest index
        top2 = np.partition(pert, V - 2)[V - 2:] if V > 1 else np.array([-np.inf, pert[0]])
        gaps[i] = float(top2.max() - top2.min())
        lps[i] = log_softmax(z)[ids[i]]
        if details is not None:
            details["pert"][i] = pert
            details["logp"][i] = log_softmax(z)
    return ids, lps, gaps


def decode_step(shape, weights, kv_pools, page_table, tokens, positions, uids,
                seed, temperature, mirror=True, layers=None, stats=None, details=None):
    """One decode step for a population.

    weights: mapping with "embed" [V, H] (row-indexable), "lm_head" [V, H],
    "final_norm" [H] and "layers" (sequence of per-layer mappings with
    attn_norm, w_qkv, q_norm, k_norm, w_o, ffn_norm, w_gate_up, w_down).
    kv_pools: per-layer pools in the paged layout (float arrays, modified in
    place by the KV append).  positions p_i = keys already cached.
    ``details`` is handed to ``logprob_sample``.
    Returns dict(ids, lps, gaps, logits, x).
    """
    tokens = np.asarray(tokens, np.int64)
    x = np.asarray(weights["embed"][tokens], np.float64)
    n_layers = shape.n_layers if layers is None else layers
    for l in range(n_layers):
        x = decoder_layer(shape, weights["layers"][l], x, positions, kv_pools[l], page_table,
                          mirror, stats)
    logits = lm_logits(shape, weights["final_norm"], weights["lm_head"], x, mirror)
    ids, lps, gaps = logprob_sample(logits, temperature, seed, uids, positions, details=details)
    return {"ids": ids, "lps": lps, "gaps": gaps, "logits": logits, "x": x}


# ------------------------------------------------------------------ prefill (scoring pass)
def prefill_index(seq_starts, start_pos=None):
    """Sequence (page-table row) and position of every packed token."""
    seq_starts = np.asarray(seq_starts, np.int64)
    T = int(seq_starts[-1])
    row = np.empty(T, np.int64)
    pos = np.empty(T, np.int64)
    for s in range(len(seq_starts) - 1):
        a, b = int(seq_starts[s]), int(seq_starts[s + 1])
        p0 = 0 if start_pos is None else int(start_pos[s])
        row[a:b] = s
        pos[a:b] = p0 + np.arange(b - a)
    return row, pos


def prefill_forward(shape, weights, kv_pools, page_table, tokens, seq_starts, start_pos=None,
                    mirror=True, stats=None):
    """Residual stream after the last layer for every token of a prefill batch.

    Every token takes the decoder layer with its sequence's page-table row and
    its own position: all keys of a layer are appended before its attention,
    and token t attends keys 0..pos(t), which is causal attention over the
    sequence (plus any cached prefix).  kv_pools are modified in place.
    ``stats`` as in decoder_layer (the smallest routing gap of MoE layers).
    """
    tokens = np.asarray(tokens, np.int64)
    row, pos = prefill_index(seq_starts, start_pos)
    pt_rows = np.asarray(page_table)[row]
    x = np.asarray(weights["embed"][tokens], np.float64)
    for l in range(shape.n_layers):
        x = decoder_layer(shape, weights["layers"][l], x, pos, kv_pools[l], pt_rows, mirror,
                          stats)
    return x


def prefill_confidence(shape, weights, kv_pools, page_table, tokens, seq_starts, scored_rows,
                       k_l, start_pos=None, mirror=True, stats=None):
    """The confidence engine: c (Eq. 1) of the next-token distribution at each
    scored row, and per sequence C = mean of c over its scored rows (Eq. 2;
    0 without any).  Returns (conf [n_seqs], row_conf [len(scored_rows)], logits)."""
    x = prefill_forward(shape, weights, kv_pools, page_table, tokens, seq_starts, start_pos,
                        mirror, stats)
    rows = np.asarray(scored_rows, np.int64)
    logits = lm_logits(shape, weights["final_norm"], weights["lm_head"], x[rows], mirror)
    c = token_confidence(logits, k_l)
    seq_starts = np.asarray(seq_starts, np.int64)
    conf = np.zeros(len(seq_starts) - 1)
    for s in range(len(conf)):
        sel = (rows >= seq_starts[s]) & (rows < seq_starts[s + 1])
        if sel.any():
            conf[s] = c[sel].mean()
    return conf, c, logits


# ------------------------------------------------------------------ fitness signal
def token_confidence(logits, k_l):
    """Per-token confidence of Eq. 1 from the scoring model's logits.

    c = -(1/K_l) * sum of the K_l largest log-probabilities log p(v | prefix),
    where p is the model's own distribution (softmax of the logits at T = 1).
    logits [N, V] -> c [N].
    """
    lp = log_softmax(np.asarray(logits, np.float64))
    k_l = int(k_l)
    top = -np.sort(-lp, axis=-1)[:, :k_l]
    return -np.mean(top, axis=-1)


def candidate_confidence(token_conf_sum, n_tokens):
    """C(tau) of Eq. 2: the mean of c(i) over the trajectory's tokens."""
    return np.asarray(token_conf_sum, np.float64) / np.asarray(n_tokens, np.float64)


def group_confidence(cand_conf, groups):
    """GC(g) of Eq. 2: the mean of C(tau) over the K candidates of each group.
    groups [M, K] holds candidate indices."""
    cand_conf = np.asarray(cand_conf, np.float64)
    return cand_conf[np.asarray(groups, np.int64)].mean(axis=-1)


def truncated_logprob_sample(logits, temperature, seed, uids, positions, top_k, top_p=1.0,
                             min_p=0.0, decision_dtype=np.float32, details=None):
    """Top-k sampling with min-p and top-p applied inside the top-k set.

    The kept list is the top_k logits in (value desc, index asc) order -- a
    temperature does not change it.  With z = logit / T on that list, min-p
    keeps z_j >= z_0 + log(min_p) (a probability at least min_p times the
    largest); top-p then keeps, in list order, each entry whose preceding
    cumulative probability (renormalised over the min-p set) is below top_p.
    The token is the Gumbel-max over the kept entries with the same noise as
    ``logprob_sample``; lp = z_id - logsumexp(kept z).  T == 0 takes the first
    entry and evaluates the truncation and lp at T = 1.  Decisions in
    ``decision_dtype``; ``gap`` = float64 top-1 minus top-2 perturbed value
    among the kept entries (inf when one is kept).  ``details`` (a dict)
    receives "pert" and "logp" [N, V] as in ``logprob_sample``, over the kept
    entries (-inf at every other entry).
    Returns ids int64 [N], lps float64 [N], gaps float64 [N].
    """
    logits = np.asarray(logits, np.float64)
    N, V = logits.shape
    tdiv = 1.0 if temperature == 0 else float(temperature)
    ids = np.empty(N, np.int64)
    lps = np.empty(N)
    gaps = np.empty(N)
    if details is not None:
        details["pert"] = np.full((N, V), -np.inf)
        details["logp"] = np.full((N, V), -np.inf)
    for i in range(N):
        order = np.lexsort((np.arange(V), -logits[i]))[:int(top_k)]
        z = logits[i][order] / tdiv
        keep = np.ones(len(order), bool)
        if min_p > 0:
            keep &= z - z[0] >= np.log(min_p)
        if top_p < 1:
            p = np.exp(z - z[0]) * keep
            tot = p.sum()
            cum = 0.0
            for j in range(len(order)):
                if not keep[j]:
                    continue
                if cum < top_p * tot:
                    cum += p[j]
                else:
                    keep[j] = False
        kz, kv = z[keep], order[keep]
        if temperature == 0:
            pert = kz
            pert_dec = kz.astype(decision_dtype)
        else:
            G = gumbel_noise(V, int(positions[i]), int(uids[i]), int(seed))[kv]
            pert = kz + G
            pert_dec = kz.astype(decision_dtype) + G.astype(decision_dtype)
        best = np.lexsort((kv, -pert_dec.astype(np.float64)))[0]   # ties -> lowest vocab index
        ids[i] = int(kv[best])
        srt = np.sort(pert)[::-1]
        gaps[i] = float(srt[0] - srt[1]) if len(srt) > 1 else np.inf
        lse = kz.max() + np.log(np.sum(np.exp(kz - kz.max())))
        lps[i] = kz[best] - lse
        if details is not None:
            details["pert"][i, kv] = pert
            details["logp"][i, kv] = kz - lse
    return ids, lps, gaps
