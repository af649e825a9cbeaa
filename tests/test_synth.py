"""The seeded input generator: host C twin vs numpy twin, statistics, recipes."""
import numpy as np

from paper_2604_07725_amd import synth


def test_c_generator_equals_numpy_twin():
    for kind, layer, off, std, mean in [(10, 0, 0, 0.02, None), (30, 5, 123456789, 1.0, None),
                                        (12, 3, 17, 0.02, 1.0)]:
        key = synth.tensor_key(3, kind, layer)
        a = synth.fill_bf16_bits(50000, key, off, std, mean)
        b = synth.fill_bf16_bits_numpy(50000, key, off, std, mean)
        np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(synth.bits_to_f32(a),
                                      synth.fill_values(50000, key, off, std, mean))


def test_generator_statistics():
    v = synth.fill_values(1 << 20, synth.tensor_key(0, 30, 0), 0, 1.0).astype(np.float64)
    assert abs(v.mean()) < 0.01 and abs(v.std() - 1.0) < 0.01
    assert np.abs(v).max() <= 3.47
    g = synth.fill_values(1 << 16, synth.tensor_key(0, 10, 0), 0, 0.02, 1.0).astype(np.float64)
    assert abs(g.mean() - 1.0) < 1e-3 and abs(g.std() - 0.02) < 1e-3


def test_slices_are_consistent():
    key = synth.tensor_key(1, 31, 2)
    full = synth.fill_values(10000, key)
    np.testing.assert_array_equal(full[4000:7000], synth.fill_values(3000, key, 4000))


def test_population_paging_invariants():
    w = synth.WORKLOADS["dense8b_pop64_agg4"]
    pop = synth.workload_population(w, extra_tokens=40)
    assert pop.n == 64
    assert pop.lengths.min() >= 16384 and pop.lengths.max() <= 32768
    used = pop.page_table[pop.page_table >= 0]
    # every physical page is used exactly once
    np.testing.assert_array_equal(np.sort(used), np.arange(pop.n_pages))
    need = (pop.lengths.astype(np.int64) + 40 + 15) // 16
    np.testing.assert_array_equal((pop.page_table >= 0).sum(1), need)


def test_length_recipes():
    rng = np.random.default_rng(0)
    a = synth.draw_lengths("agg4_u2048_4096", 1000, rng)
    assert a.min() >= 8192 and a.max() <= 16384 and abs(a.mean() - 12288) < 150
    b = synth.draw_lengths("agg8_8k_pm10", 1000, rng)
    assert b.min() >= int(65536 * 0.9) and b.max() <= int(65536 * 1.1)
    c = synth.draw_lengths("u256_512", 1000, rng)
    assert c.min() >= 256 and c.max() <= 512


def test_lazy_weights_match_eager():
    shape = synth.TINY
    eager = synth.host_weights(shape, 0)
    lazy = synth.host_weights(shape, 0, lazy=True)
    np.testing.assert_array_equal(eager["embed"][[5, 77]], lazy["embed"][[5, 77]])
    np.testing.assert_array_equal(eager["lm_head"][100:300], lazy["lm_head"][100:300])
    np.testing.assert_array_equal(eager["layers"][0]["w_qkv"], lazy["layers"][0]["w_qkv"])


def test_pool_pages_equal_the_pool_slices():
    """The batched page generator gives each selected page's elements of the
    whole pool (and rejects page ids outside it)."""
    import pytest
    spec = synth.kv_spec(synth.TINY, 3, 1, 40)
    full = synth.host_values(spec).reshape(spec.shape)
    pages = np.array([7, 0, 39, 7, 12])
    np.testing.assert_array_equal(synth.pool_pages(spec, pages), full[pages])
    assert synth.pool_pages(spec, np.array([], np.int64)).shape == (0,) + spec.shape[1:]
    with pytest.raises(IndexError):
        synth.pool_pages(spec, np.array([40]))
