"""C-ABI checks that need no GPU: symbols, struct layouts, host-side validation."""
import ctypes as C
import os
import subprocess
import tempfile

import pytest

from paper_2604_07725_amd import sevo

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_header_function():
    names = sevo.header_functions()
    assert len(names) >= 19
    L = sevo.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(sevo._SIGS), set(names) ^ set(sevo._SIGS)
    assert L.sevo_version().startswith(b"sevo")


_LAYOUT_C = r"""
#include <stdio.h>
#include <stddef.h>
#include "sevo.h"
#define P(T, f) printf(#T "." #f " %zu\n", offsetof(T, f));
#define S(T) printf(#T " %zu\n", sizeof(T));
int main(void) {
  S(sevo_model_config) P(sevo_model_config, rope_theta) P(sevo_model_config, rms_eps)
  P(sevo_model_config, n_experts) P(sevo_model_config, expert_ffn)
  S(sevo_weights) P(sevo_weights, w_down) P(sevo_weights, w_router)
  P(sevo_weights, w_expert_down)
  S(sevo_attn_args) P(sevo_attn_args, num_pages) P(sevo_attn_args, q) P(sevo_attn_args, scale)
  P(sevo_attn_args, out) P(sevo_attn_args, workspace_bytes)
  S(sevo_sample_args) P(sevo_sample_args, ld) P(sevo_sample_args, temperature)
  P(sevo_sample_args, seed) P(sevo_sample_args, top_k) P(sevo_sample_args, min_p)
  P(sevo_sample_args, conf_topk) P(sevo_sample_args, conf_sum)
  P(sevo_sample_args, workspace_bytes)
  S(sevo_step_args) P(sevo_step_args, max_pages) P(sevo_step_args, num_pages)
  P(sevo_step_args, kv_pools) P(sevo_step_args, seed) P(sevo_step_args, temperature)
  P(sevo_step_args, num_splits) P(sevo_step_args, out_logits) P(sevo_step_args, top_p)
  P(sevo_step_args, conf_topk)
  P(sevo_step_args, out_conf) P(sevo_step_args, workspace_bytes) P(sevo_step_args, out_hidden)
  S(sevo_linear_args) P(sevo_linear_args, flags) P(sevo_linear_args, x)
  P(sevo_linear_args, workspace_bytes)
  S(sevo_prefill_attn_args) P(sevo_prefill_attn_args, num_pages) P(sevo_prefill_attn_args, q)
  P(sevo_prefill_attn_args, start_pos) P(sevo_prefill_attn_args, scale)
  P(sevo_prefill_attn_args, out)
  S(sevo_prefill_args) P(sevo_prefill_args, tokens) P(sevo_prefill_args, max_pages)
  P(sevo_prefill_args, num_pages) P(sevo_prefill_args, kv_pools) P(sevo_prefill_args, conf_topk)
  P(sevo_prefill_args, scored_rows) P(sevo_prefill_args, out_row_conf)
  P(sevo_prefill_args, workspace_bytes) P(sevo_prefill_args, moe_chunk)
  return 0;
}
"""

_PY = {"sevo_model_config": sevo.ModelConfig, "sevo_weights": sevo.Weights,
       "sevo_attn_args": sevo.AttnArgs, "sevo_sample_args": sevo.SampleArgs,
       "sevo_step_args": sevo.StepArgs, "sevo_linear_args": sevo.LinearArgs,
       "sevo_prefill_attn_args": sevo.PrefillAttnArgs, "sevo_prefill_args": sevo.PrefillArgs}


def test_ctypes_structs_match_c_layout():
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "layout.c")
        exe = os.path.join(d, "layout")
        open(src, "w").write(_LAYOUT_C)
        subprocess.check_call(["gcc", "-I", os.path.join(ROOT, "include"), src, "-o", exe])
        out = subprocess.check_output([exe], text=True)
    for line in out.splitlines():
        key, val = line.split()
        val = int(val)
        if "." in key:
            t, f = key.split(".")
            assert getattr(_PY[t], f).offset == val, key
        else:
            assert C.sizeof(_PY[key]) == val, key


def _attn(**kw):
    base = dict(n=1, n_q_heads=4, n_kv_heads=2, head_dim=64, page_size=16, max_pages=4,
                num_splits=0, num_pages=4, scale=0.125)
    base.update(kw)
    return sevo.AttnArgs(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), sevo.UNSUPPORTED),
    (dict(page_size=8), sevo.UNSUPPORTED),
    (dict(n_q_heads=6, n_kv_heads=4), sevo.UNSUPPORTED),
    (dict(n_q_heads=32, n_kv_heads=2), sevo.UNSUPPORTED),
    (dict(max_pages=0), sevo.INVALID_ARGUMENT),
    (dict(num_pages=0), sevo.INVALID_ARGUMENT),
    (dict(num_splits=-1), sevo.INVALID_ARGUMENT),
    (dict(scale=0.0), sevo.INVALID_ARGUMENT),
    (dict(), sevo.INVALID_ARGUMENT),           # null pointers
])
def test_attention_rejects_bad_arguments(kw, status):
    a = _attn(**kw)
    assert sevo.lib().sevo_attn_decode(C.byref(a), None) == status
    assert sevo.lib().sevo_last_error()


def test_attention_workspace_too_small_is_reported_before_launch():
    fake = 1 << 20  # never dereferenced: the check fails first
    a = _attn(q=fake, kv_pool=fake, page_table=fake, seq_lens=fake, out=fake,
              workspace=fake, workspace_bytes=16)
    assert sevo.lib().sevo_attn_decode(C.byref(a), None) == sevo.WORKSPACE_TOO_SMALL
    assert b"workspace" in sevo.lib().sevo_last_error()


def test_zero_population_is_a_no_op():
    assert sevo.lib().sevo_attn_decode(C.byref(_attn(n=0)), None) == sevo.OK


def test_split_planning():
    L = sevo.lib()
    # enough workgroups for 256 CUs, at least 32 pages per split, at least one
    # split, and no split longer than 512 pages
    # fewest splits that fill whole rounds of 512 resident workgroups, at
    # least the 512-pages-per-split minimum, at most max_pages / 32
    assert L.sevo_attn_plan_splits(64, 8, 2037) == 4
    assert L.sevo_attn_plan_splits(64, 8, 2049) == 5      # the minimum rises to 5
    assert L.sevo_attn_plan_splits(64, 8, 1024) == 4      # 2 would be two ragged rounds
    assert L.sevo_attn_plan_splits(16, 8, 1024) == 4      # 2 would leave half a round
    assert L.sevo_attn_plan_splits(16, 8, 4470) == 12     # minimum 9, 12 fills 3 rounds
    assert L.sevo_attn_plan_splits(64, 4, 2040) == 8      # 4 would be two ragged rounds
    assert L.sevo_attn_plan_splits(64, 8, 4100) == 9
    assert L.sevo_attn_plan_splits(3, 5, 4000) == 35      # no whole-round count up to 2x
    assert L.sevo_attn_plan_splits(4, 2, 33) == 2         # capped: 32 pages per split
    assert L.sevo_attn_plan_splits(1, 1, 1) == 1
    ws = L.sevo_attn_workspace_bytes(64, 32, 8, 128, 2049, 0)
    assert ws >= 64 * 32 * 4 * 130 * 4


@pytest.mark.parametrize("temp", [-1.0, float("nan"), float("inf")])
def test_sampler_rejects_bad_temperature(temp):
    a = sevo.SampleArgs(logits=1 << 20, n=1, vocab=8, ld=8, temperature=temp)
    assert sevo.lib().sevo_logprob_sample(C.byref(a), None) == sevo.INVALID_ARGUMENT


def test_sampler_rejects_bad_ld_and_small_workspace():
    L = sevo.lib()
    a = sevo.SampleArgs(logits=1 << 20, n=1, vocab=8, ld=6, temperature=1.0, top_p=1.0)
    assert L.sevo_logprob_sample(C.byref(a), None) == sevo.INVALID_ARGUMENT
    f = 1 << 20
    a = sevo.SampleArgs(logits=f, n=2, vocab=8, ld=8, temperature=1.0, cand_uid=f, positions=f,
                        out_tokens=f, out_logprobs=f, workspace=f, workspace_bytes=1, top_p=1.0)
    assert L.sevo_logprob_sample(C.byref(a), None) == sevo.WORKSPACE_TOO_SMALL


@pytest.mark.parametrize("kw,status", [
    (dict(k=200, ldx=200), sevo.UNSUPPORTED),
    (dict(n_out=96), sevo.UNSUPPORTED),
    (dict(mode=3), sevo.INVALID_ARGUMENT),
    (dict(ldx=100), sevo.INVALID_ARGUMENT),
    (dict(flags=4), sevo.INVALID_ARGUMENT),
    (dict(flags=2, mode=0), sevo.INVALID_ARGUMENT),     # tiled output needs SWIGLU
])
def test_linear_rejects_bad_shapes(kw, status):
    base = dict(m=4, n_out=128, k=128, ldx=128, mode=0, k_splits=0)
    base.update(kw)
    a = sevo.LinearArgs(**base)
    assert sevo.lib().sevo_linear(C.byref(a), None) == status


def test_linear_plan_and_workspace():
    L = sevo.lib()
    # the fewest splits (each >= 1024 k) whose row-block count fits the
    # projection in one round of 256 workgroups: QKV 3 row blocks x 2 splits,
    # output / down 4 x 4; at M = 16 QKV 5 x 2, output / down 5 x 4
    assert L.sevo_linear_workspace_bytes(64, 6144, 4096, 0) == 2 * 64 * 6144 * 4
    assert L.sevo_linear_workspace_bytes(64, 4096, 4096, 0) == 4 * 64 * 4096 * 4
    assert L.sevo_linear_workspace_bytes(64, 4096, 12288, 0) == 4 * 64 * 4096 * 4
    assert L.sevo_linear_workspace_bytes(16, 10240, 5120, 0) == 2 * 16 * 10240 * 4
    assert L.sevo_linear_workspace_bytes(16, 5120, 8192, 0) == 4 * 16 * 5120 * 4
    assert L.sevo_linear_workspace_bytes(16, 5120, 25600, 0) == 4 * 16 * 5120 * 4
    # several rounds whatever the split: one split, no partials
    assert L.sevo_linear_workspace_bytes(64, 151936, 4096, 0) == 0
    assert L.sevo_linear_workspace_bytes(4, 512, 256, 0) == 0           # short k: one split


def test_linear_plans_of_the_decode_projections():
    """(splits, k per split, row blocks per workgroup) of the decode shapes:
    about one round of 256 workgroups each, the LM head many rounds."""
    plan = sevo.sevo_linear_plan
    # 8B-class, 64 candidates: QKV, output, gate/up (3 gate/up pairs), down, LM head
    assert plan(64, 6144, 4096) == (2, 2048, 3)
    assert plan(64, 4096, 4096) == (4, 1024, 4)
    assert plan(64, 24576, 4096, mode=sevo.LINEAR_SWIGLU) == (1, 4096, 6)
    assert plan(64, 4096, 12288) == (4, 3072, 4)
    assert plan(64, 151936, 4096, k_splits=1) == (1, 4096, 8)
    # 32B-class, 16 candidates (7 gate/up pairs: 229 workgroups)
    assert plan(16, 10240, 5120) == (2, 2560, 5)
    assert plan(16, 5120, 8192) == (4, 2048, 5)
    assert plan(16, 51200, 5120, mode=sevo.LINEAR_SWIGLU) == (1, 5120, 14)
    assert plan(16, 5120, 25600) == (4, 6400, 5)
    assert plan(16, 151936, 5120, k_splits=1) == (1, 5120, 10)
    # the caller's split count is kept
    assert plan(64, 6144, 4096, k_splits=3)[0] == 3


@pytest.mark.parametrize("args", [(0, 128, 256, 0, 0), (256, 128, 256, 0, 0), (4, 96, 256, 0, 0),
                                  (4, 128, 48, 0, 0), (4, 128, 256, -1, 0), (4, 128, 256, 0, 3)])
def test_linear_plan_rejects_bad_shapes(args):
    out = (C.c_int32 * 3)()
    assert sevo.lib().sevo_linear_plan(*args, out) == sevo.INVALID_ARGUMENT
    assert sevo.lib().sevo_linear_plan(4, 128, 256, 0, 0, None) == sevo.INVALID_ARGUMENT


@pytest.mark.parametrize("kw,status", [
    (dict(n_out=96), sevo.UNSUPPORTED),
    (dict(k=48), sevo.UNSUPPORTED),
    (dict(kind=2), sevo.INVALID_ARGUMENT),
    (dict(src=0), sevo.INVALID_ARGUMENT),
    (dict(dst=(1 << 20) + 4096), sevo.INVALID_ARGUMENT),                # overlapping buffers
])
def test_pack_weight_rejects_bad_arguments(kw, status):
    a = dict(src=1 << 20, dst=1 << 24, n_out=64, k=64, kind=0)
    a.update(kw)
    assert sevo.lib().sevo_pack_weight(a["src"], a["dst"], a["n_out"], a["k"], a["kind"],
                                       None) == status


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), sevo.UNSUPPORTED),
    (dict(n_kv_heads=0), sevo.INVALID_ARGUMENT),
    (dict(num_pages=-1), sevo.INVALID_ARGUMENT),
    (dict(k_pool=0), sevo.INVALID_ARGUMENT),
    (dict(v_pool=(1 << 22) + 8), sevo.INVALID_ARGUMENT),                 # misaligned
    (dict(kv_pool=(1 << 20) + 4096), sevo.INVALID_ARGUMENT),             # overlaps k_pool
    (dict(kv_pool=(1 << 22) - 8192), sevo.INVALID_ARGUMENT),             # overlaps v_pool
    (dict(num_pages=0, k_pool=0, v_pool=0, kv_pool=0), sevo.OK),         # nothing to move
])
def test_pack_kv_rejects_bad_arguments(kw, status):
    a = dict(k_pool=1 << 20, v_pool=1 << 22, num_pages=4, n_kv_heads=2, head_dim=64,
             kv_pool=1 << 24)
    a.update(kw)
    assert sevo.lib().sevo_pack_kv(a["k_pool"], a["v_pool"], a["num_pages"], a["n_kv_heads"],
                                   a["head_dim"], a["kv_pool"], None) == status


@pytest.mark.parametrize("kw,status", [
    (dict(rows=-1), sevo.INVALID_ARGUMENT),
    (dict(cols=4094), sevo.INVALID_ARGUMENT),
    (dict(n_partials=17), sevo.INVALID_ARGUMENT),
    (dict(n_partials=-1), sevo.INVALID_ARGUMENT),
    (dict(eps=0.0), sevo.INVALID_ARGUMENT),
    (dict(x=0), sevo.INVALID_ARGUMENT),
    (dict(x=(1 << 20) + 8), sevo.INVALID_ARGUMENT),                      # x not 16-byte aligned
    (dict(partials=0), sevo.INVALID_ARGUMENT),                           # partials needed
    (dict(gain=(1 << 22) + 2), sevo.INVALID_ARGUMENT),
    (dict(rows=0), sevo.OK),                                             # nothing to do
])
def test_add_rmsnorm_rejects_bad_arguments(kw, status):
    """Host-side validation of the residual add + RMSNorm sub-step (no launch)."""
    a = dict(x=1 << 20, partials=1 << 21, n_partials=2, gain=1 << 22, rows=4, cols=4096,
             eps=1e-6, out=1 << 23)
    a.update(kw)
    assert sevo.lib().sevo_add_rmsnorm(a["x"], a["partials"], a["n_partials"], a["gain"],
                                       a["rows"], a["cols"], a["eps"], a["out"], None) == status


def test_init_model_rejects_bad_config():
    cfg = sevo.ModelConfig(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                           ffn=1024, vocab=4096, page_size=16, max_position=1024, qk_norm=1,
                           rope_theta=1e6, rms_eps=1e-6)
    w = sevo.Weights()
    h = C.c_void_p()
    L = sevo.lib()
    assert L.sevo_init_model(C.byref(cfg), C.byref(w), C.byref(h)) == sevo.INVALID_ARGUMENT
    cfg.head_dim = 80
    assert L.sevo_init_model(C.byref(cfg), C.byref(w), C.byref(h)) == sevo.UNSUPPORTED
    cfg.head_dim = 64
    cfg.hidden = 200
    assert L.sevo_init_model(C.byref(cfg), C.byref(w), C.byref(h)) == sevo.UNSUPPORTED


def test_status_strings():
    L = sevo.lib()
    for s in range(7):
        assert L.sevo_status_string(s)
    assert L.sevo_status_string(99) == b"unknown status"


@pytest.mark.parametrize("kw,status", [
    (dict(conf_topk=33, out_conf=1 << 20), sevo.INVALID_ARGUMENT),
    (dict(conf_topk=-1, out_conf=1 << 20), sevo.INVALID_ARGUMENT),
    (dict(conf_topk=9, out_conf=1 << 20), sevo.INVALID_ARGUMENT),     # more than vocab
    (dict(conf_topk=4), sevo.INVALID_ARGUMENT),                       # no output
    (dict(top_k=33), sevo.INVALID_ARGUMENT),
    (dict(top_k=9), sevo.INVALID_ARGUMENT),                           # more than vocab
    (dict(top_k=4, top_p=0.0), sevo.INVALID_ARGUMENT),
    (dict(top_k=4, top_p=1.5), sevo.INVALID_ARGUMENT),
    (dict(top_k=4, min_p=-0.1), sevo.INVALID_ARGUMENT),
    (dict(top_p=0.9), sevo.UNSUPPORTED),                              # top-p without top-k
    (dict(min_p=0.1), sevo.UNSUPPORTED),
])
def test_sampler_rejects_bad_confidence_arguments(kw, status):
    f = 1 << 20
    a = dict(logits=f, n=2, vocab=8, ld=8, temperature=1.0, cand_uid=f, positions=f,
             out_tokens=f, out_logprobs=f, workspace=f, workspace_bytes=1 << 20, top_p=1.0)
    a.update(kw)
    assert sevo.lib().sevo_logprob_sample(C.byref(sevo.SampleArgs(**a)), None) == status


def test_group_confidence_rejects_bad_arguments():
    L = sevo.lib()
    f = 1 << 20
    assert L.sevo_group_confidence(f, f, f, -1, 4, f, None) == sevo.INVALID_ARGUMENT
    assert L.sevo_group_confidence(f, f, f, 3, 0, f, None) == sevo.INVALID_ARGUMENT
    assert L.sevo_group_confidence(None, f, f, 3, 4, f, None) == sevo.INVALID_ARGUMENT
    assert L.sevo_group_confidence(None, None, None, 0, 4, None, None) == sevo.OK


def test_profile_begin_rejects_bad_arguments():
    L = sevo.lib()
    assert L.sevo_profile_begin(0, 1) == sevo.INVALID_ARGUMENT
    assert L.sevo_profile_begin(8, 0) == sevo.INVALID_ARGUMENT
    assert L.sevo_profile_begin(8, 1 << len(sevo.PROF_KINDS)) == sevo.INVALID_ARGUMENT
    # ending without a recording returns empty totals
    import ctypes as CT
    ms = (CT.c_float * len(sevo.PROF_KINDS))()
    cnt = (CT.c_int32 * len(sevo.PROF_KINDS))()
    assert L.sevo_profile_end(ms, cnt) == sevo.OK and sum(cnt) == 0


def test_read_probe_rejects_bad_arguments():
    L = sevo.lib()
    f = 1 << 20
    assert L.sevo_hbm_read_probe(None, 1 << 20, None, 64, f, None) == sevo.INVALID_ARGUMENT
    assert L.sevo_hbm_read_probe(f + 4, 1 << 20, None, 64, f, None) == sevo.INVALID_ARGUMENT
    assert L.sevo_hbm_read_probe(f, 1 << 20, None, 64, None, None) == sevo.INVALID_ARGUMENT
    assert L.sevo_hbm_read_probe(f, 1 << 20, None, 0, f, None) == sevo.INVALID_ARGUMENT
    assert L.sevo_hbm_read_probe(f, 1 << 20, None, (1 << 20) + 1, f, None) == \
        sevo.INVALID_ARGUMENT
    assert L.sevo_hbm_read_probe(f, 8, None, 64, f, None) == sevo.INVALID_ARGUMENT
    assert L.sevo_hbm_read_probe(f, 4096, f, 64, f, None) == sevo.INVALID_ARGUMENT


@pytest.mark.parametrize("kw,ok", [
    (dict(max_seq_len=0), False),                              # tokens but no length bound
    (dict(max_seq_len=49), False),                             # below the mean (100 / 2)
    (dict(max_seq_len=-1), False),
    (dict(max_seq_len=50), True),                              # passes this check
])
def test_attn_prefill_rejects_a_short_max_seq_len(kw, ok):
    """max_seq_len sizes the grid: a bound below the mean sequence length
    would leave rows uncomputed, so it is rejected before any launch."""
    base = dict(n_seqs=2, total_tokens=100, max_seq_len=60, n_q_heads=4, n_kv_heads=2,
                head_dim=64, page_size=16, max_pages=8, num_pages=16, scale=0.125)
    base.update(kw)
    a = sevo.PrefillAttnArgs(**base)           # null pointers: the next check fails
    st = sevo.lib().sevo_attn_prefill(C.byref(a), None)
    assert st == sevo.INVALID_ARGUMENT
    msg = sevo.lib().sevo_last_error().decode()
    assert ("max_seq_len" in msg) != ok, msg
