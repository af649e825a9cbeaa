"""The GEMM operand layouts of include/sevo.h, as the tests write them out on the
host: each is a permutation of the elements, and every MFMA operand fragment
(16 rows x 32 columns) is one contiguous 1 KB block in the documented lane
order (run index 16 ((c / 8) % 4) + r % 16)."""
import numpy as np
import pytest

from tests.gpu_helpers import (act_tile_offsets, gate_up_row_order, pack_weight_host,
                               packed_weight_offsets, tile_activations_host,
                               untile_activations_host)


@pytest.mark.parametrize("n_out,k", [(64, 32), (192, 160), (128, 512)])
def test_packed_weight_is_a_permutation_with_contiguous_fragments(n_out, k):
    off = packed_weight_offsets(n_out, k)
    assert np.array_equal(np.sort(off.ravel()), np.arange(n_out * k))
    for r0 in range(0, n_out, 16):
        for c0 in range(0, k, 32):
            frag = off[r0:r0 + 16, c0:c0 + 32]
            base = frag.min()
            assert base % 512 == 0 and frag.max() == base + 511
            r, c = np.meshgrid(np.arange(16), np.arange(32), indexing="ij")
            np.testing.assert_array_equal(frag - base, (16 * (c // 8) + r) * 8 + c % 8)
    # the four fragments of a superblock step are adjacent
    assert off[16, 0] == off[0, 0] + 512
    if k >= 64:
        assert off[0, 32] == off[0, 0] + 2048


def test_gate_up_order_pairs_matching_rows():
    order = gate_up_row_order(256)
    assert np.array_equal(np.sort(order), np.arange(256))
    # superblock 1: gate rows 32..63 then up rows 160..191
    assert list(order[64:96]) == list(range(32, 64))
    assert list(order[96:128]) == list(range(160, 192))
    w = np.arange(256 * 32).reshape(256, 32)
    p = pack_weight_host(w, gate_up=True).ravel()
    assert p[packed_weight_offsets(256, 32)[96, 0]] == w[160, 0]


@pytest.mark.parametrize("m,k", [(1, 32), (17, 64), (64, 96)])
def test_tiled_activations_round_trip(m, k):
    off = act_tile_offsets(m, k)
    assert len(np.unique(off)) == m * k and off.max() < (-(-m // 16) * 16) * k
    x = np.random.default_rng(0).standard_normal((m, k))
    t = tile_activations_host(x)
    np.testing.assert_array_equal(untile_activations_host(t, m, k), x)
    # fragment (block 0, columns 0..31) is the first 1 KB block in lane order
    r, c = 3 % m, 13
    assert t[(16 * (c // 8) + r) * 8 + c % 8] == x[r, c]
