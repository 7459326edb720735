"""Pins of the oracle's bookkeeping and number formats against closed forms
and library routines (no GPU)."""
import math

import numpy as np
import pytest

import oracle
from paper_2308_04623_amd import workloads as W


# ---------------------------------------------------------------- tree info

def test_complete_binary_tree_closed_form():
    n = 31
    p = W.complete_binary_tree(n)
    depth, anc = oracle.tree_info(p)
    for i in range(n):
        assert depth[i] == int(math.floor(math.log2(i + 1)))
        for j in range(n):
            # j is an ancestor-or-self of i iff shifting (i+1) right by the
            # depth difference lands on (j+1)
            dd = depth[i] - int(math.floor(math.log2(j + 1)))
            want = dd >= 0 and ((i + 1) >> dd) == j + 1
            assert anc[i, j] == int(want), (i, j)


def test_chain_is_lower_triangular():
    n = 20
    depth, anc = oracle.tree_info(W.chain_tree(n))
    assert np.array_equal(depth, np.arange(n))
    assert np.array_equal(anc, np.tril(np.ones((n, n), dtype=np.uint8)))


@pytest.mark.parametrize("branching,n,counts", [
    ([4, 2, 2, 1], 32, {0: 1, 1: 4, 2: 8, 3: 16, 4: 3}),
    ([8, 4, 2, 2, 1], 256, {0: 1, 1: 8, 2: 32, 3: 64, 4: 128, 5: 23}),
])
def test_branching_tree_depth_histogram(branching, n, counts):
    p = W.branching_tree(branching, n)
    assert len(p) == n
    depth, _ = oracle.tree_info(p)
    vals, cnt = np.unique(depth, return_counts=True)
    assert dict(zip(vals.tolist(), cnt.tolist())) == counts


@pytest.mark.parametrize("parents", [[0, 0], [-1, 1], [-1, 0, 5], [-1, -1]])
def test_invalid_trees_rejected(parents):
    with pytest.raises(oracle.OracleError) as e:
        oracle.tree_info(parents)
    assert e.value.code == -2


# ---------------------------------------------------------------- bf16

def test_bf16_rounding_ties_and_double_rounding():
    one = 0x3F80
    assert oracle.round_bf16(1.0) == one
    assert oracle.round_bf16(1.0 + 2.0 ** -8) == one                   # tie -> even (down)
    assert oracle.round_bf16(1.0 + 3 * 2.0 ** -8) == one + 2           # tie -> even (up)
    assert oracle.round_bf16(1.0 + 2.0 ** -8 + 2.0 ** -40) == one + 1  # above the tie: no double rounding
    assert oracle.round_bf16(-2.5) == 0xC020
    assert oracle.round_bf16(0.0) == 0 and oracle.round_bf16(-0.0) == 0x8000
    assert oracle.round_bf16(3.0e38 * 10) == 0x7F80                    # overflow -> inf
    assert oracle.round_bf16(2.0 ** -133) == 0x0001                    # smallest subnormal
    assert oracle.round_bf16(2.0 ** -134) == 0x0000                    # tie -> even (zero)


def test_bf16_rounding_matches_float32_bit_trick():
    # for values already representable in float32 the result must equal the
    # classic float32 round-to-nearest-even bit trick
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(3000).astype(np.float32),
                        (g.standard_normal(1000) * 1e-30).astype(np.float32),
                        (g.standard_normal(1000) * 1e30).astype(np.float32)])
    want = W.f32_to_bf16_bits(x)
    got = np.array([oracle.round_bf16(float(v)) for v in x], dtype=np.uint16)
    assert np.array_equal(got, want)


# ---------------------------------------------------------------- Philox

@pytest.mark.parametrize("key,ctr", [([0, 0], [1, 0, 0, 0]), ([5, 7], [4, 0, 0, 0]),
                                     ([2 ** 64 - 1, 123456789], [99, 0, 0, 0]),
                                     ([17, 1], [2 ** 40 + 3, 0, 0, 0])])
def test_philox_matches_numpy(key, ctr):
    # numpy's Philox increments its 256-bit counter before producing a block
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                          counter=np.array([ctr[0] - 1] + ctr[1:], dtype=np.uint64))
    assert np.array_equal(oracle.philox4x64_10(key, ctr), bg.random_raw(4))


def test_uniform_definition():
    for seed, s, n in [(0, 0, 1), (3, 1, 17), (2 ** 63, 0, 255)]:
        raw = oracle.philox4x64_10([seed, s], [n, 0, 0, 0])[0]
        u = oracle.uniform(seed, s, n)
        assert u == float(int(raw) >> 11) * 2.0 ** -53
        assert 0.0 <= u < 1.0
