"""GPU parity of the whole decode step (sevo_decode_step) against the oracle."""
import numpy as np
import pytest
import torch

from oracle import decoder as od
from paper_2604_07725_amd import synth
from tests.gpu_helpers import LP_ABS_TOL, bf16_bits, check_ids, say

pytestmark = pytest.mark.gpu

TINY_LOGIT_TOL = 1e-2


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_07725_amd import device_inputs, sevo
    sevo.lib()
    return sevo, device_inputs


def _setup(S, w, extra, n=None, shape=None):
    sevo, di = S
    shape = w.shape if shape is None else shape
    pop = synth.workload_population(w, extra_tokens=extra, n=n)
    tensors = di.device_weights(shape, w.seed)
    model = sevo.sevo_init_model(shape, tensors, max_position=int(pop.lengths.max()) + extra + 1)
    kp, vp = di.device_pools(shape, w.seed, pop.n_pages)
    d = di.device_population(pop)
    return pop, model, kp, vp, d


def test_tiny_step_sequence_matches_oracle(S):
    """Three consecutive steps of the tiny workload: logits, ids, log-probs and
    the appended KV slots against the oracle (which appends its own k, v)."""
    sevo, di = S
    w = synth.WORKLOADS["tiny_step"]
    shape = w.shape
    steps = 3
    say("tiny step sequence")
    pop, model, kp, vp, d = _setup(S, w, extra=steps)
    hw = synth.host_weights(shape, w.seed)
    hk, hv = synth.host_pools(shape, w.seed, pop.n_pages)
    hk = [k.astype(np.float64) for k in hk]
    hv = [v.astype(np.float64) for v in hv]
    seed, temp = 99, 1.0
    toks = pop.tokens.astype(np.int64)
    pos = pop.lengths.astype(np.int64)
    pos_d = d["lengths"].clone()
    for step in range(steps):
        ids, lps, logits = sevo.sevo_decode_step(model, torch.from_numpy(toks.astype(np.int32)).cuda(),
                                                 pos_d, d["page_table"], kp, vp, d["uids"], seed,
                                                 temp, keep_logits=True)
        torch.cuda.synchronize()
        ref = od.decode_step(shape, hw, hk, hv, pop.page_table, toks, pos, pop.uids, seed, temp)
        lg = logits.double().cpu().numpy()
        err = np.abs(lg - ref["logits"]).max()
        lp_err = np.abs(lps.cpu().numpy() - ref["lps"]).max()
        say(f"  step {step}: logit max abs err {err:.2e}, lp max err {lp_err:.2e}, ids "
            f"{ids.cpu().numpy().tolist()} vs {ref['ids'].tolist()} gaps {np.round(ref['gaps'], 4)}")
        # bf16 storage points round values that differ in the last fp32 bits
        # between any two correct implementations; in this tiny model (residual
        # stream ~0.05, one layer) a single 1-ulp flip moves logits by ~1e-3.
        # The oracle's own logits move by up to 6e-3 when its pre-rounding
        # values are perturbed by 1e-6 relative, so logits are held to 1e-2.
        assert err <= TINY_LOGIT_TOL
        check_ids(ids.cpu().numpy(), lps.cpu().numpy(), ref["ids"], ref["lps"], ref["gaps"],
                  label=f"step {step}")
        toks = ref["ids"]
        pos = pos + 1
        pos_d += 1
    # appended slots: close to the oracle's; every other slot untouched
    torch.cuda.synchronize()
    for l in range(shape.n_layers):
        def tok_major(a):   # [P, hkv, d/32, 16, 32] -> [P, hkv, 16, d]
            return np.transpose(a, (0, 1, 3, 2, 4)).reshape(a.shape[0], a.shape[1], 16, -1)
        gk = tok_major(kp[l].double().cpu().numpy())
        gv = vp[l].double().cpu().numpy()
        kspec, vspec = synth.kv_specs(shape, w.seed, l, pop.n_pages)
        k0 = tok_major(synth.host_values(kspec).reshape(kspec.shape))
        v0 = synth.host_values(vspec).reshape(vspec.shape)
        hkl = tok_major(hk[l])
        written = np.zeros(gk.shape[:3], bool)   # [page, head, slot]
        for i in range(pop.n):
            for p in range(int(pop.lengths[i]), int(pop.lengths[i]) + steps):
                written[pop.page_table[i, p // 16], :, p % 16] = True
        np.testing.assert_array_equal(gk[~written], k0[~written])
        np.testing.assert_array_equal(np.transpose(gv, (0, 1, 3, 2))[~written],
                                      np.transpose(v0, (0, 1, 3, 2))[~written])
        gkw, rkw = gk[written], hkl[written]
        gvw = np.transpose(gv, (0, 1, 3, 2))[written]
        rvw = np.transpose(hv[l], (0, 1, 3, 2))[written]
        say(f"  layer {l}: appended k max diff {np.abs(gkw - rkw).max():.2e}, "
            f"v {np.abs(gvw - rvw).max():.2e}; equal {np.mean(gkw == rkw):.3f} / "
            f"{np.mean(gvw == rvw):.3f}")
        # at most one bf16 rounding step apart (values rounded from fp32 vs fp64)
        assert np.all(np.abs(gkw - rkw) <= 2.0 ** -7 * np.abs(rkw) + 1e-6)
        assert np.all(np.abs(gvw - rvw) <= 2.0 ** -7 * np.abs(rvw) + 1e-6)
    model.close()


def test_tiny_step_deterministic_and_resumable(S):
    """Same state -> bit-identical outputs; 4 straight steps equal 2 + (re-init) 2."""
    sevo, di = S
    w = synth.WORKLOADS["tiny_step"]
    say("tiny step determinism / resume")

    def run(steps_a, steps_b):
        pop, model, kp, vp, d = _setup(S, w, extra=4)
        toks = torch.from_numpy(pop.tokens).cuda()
        pos = d["lengths"].clone()
        out = []
        for s in range(steps_a + steps_b):
            if s == steps_a and steps_b:
                # resume: a fresh model handle over the same device state
                model.close()
                model = sevo.sevo_init_model(w.shape, model.tensors, max_position=1024)
            ids, lps = sevo.sevo_decode_step(model, toks, pos, d["page_table"], kp, vp, d["uids"],
                                             1234, 1.0)
            torch.cuda.synchronize()
            out.append((ids.cpu().numpy().copy(), lps.cpu().numpy().copy()))
            toks = ids.clone()
            pos += 1
        model.close()
        return out, [bf16_bits(k) for k in kp]

    a, ka = run(4, 0)
    b, kb = run(2, 2)
    for (ia, la), (ib, lb) in zip(a, b):
        np.testing.assert_array_equal(ia, ib)
        np.testing.assert_array_equal(la, lb)
    for x, y in zip(ka, kb):
        np.testing.assert_array_equal(x, y)


def test_step_rejects_small_workspace_and_bad_temperature(S):
    sevo, di = S
    import ctypes as C
    w = synth.WORKLOADS["tiny_step"]
    pop, model, kp, vp, d = _setup(S, w, extra=1)
    b = sevo.StepBuffers(model, torch.from_numpy(pop.tokens).cuda(), d["lengths"],
                         d["page_table"], kp, vp, d["uids"], 1, 1.0)
    b.args.workspace_bytes = 1024
    assert sevo.lib().sevo_decode_step(model.handle, C.byref(b.args), None) == \
        sevo.WORKSPACE_TOO_SMALL
    b.args.workspace_bytes = b.workspace.numel()
    b.args.temperature = -1.0
    assert sevo.lib().sevo_decode_step(model.handle, C.byref(b.args), None) == \
        sevo.INVALID_ARGUMENT
    model.close()
