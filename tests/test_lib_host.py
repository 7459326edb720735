"""libssd host-side checks that need no GPU: the library loads, exports every
function include/ssd.h declares, and its host tree bookkeeping equals the
oracle's bit for bit."""
import os
import re

import numpy as np
import pytest

import oracle
from paper_2308_04623_amd import ssd
from paper_2308_04623_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions(name):
    txt = open(os.path.join(ROOT, "include", name)).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(ssd_[a-z_0-9]+)\s*\(", txt)))


@pytest.mark.parametrize("header,listed", [("ssd.h", "EXPORTS"), ("ssd_diag.h", "DIAG_EXPORTS")])
def test_library_exports_every_declared_function(header, listed):
    L = ssd.lib()
    names = _header_functions(header)
    assert len(names) >= 4
    for n in names:
        assert hasattr(L, n), n
    assert sorted(getattr(ssd, listed)) == names


def _random_tree(g, n):
    p = [-1] + [int(g.integers(0, i)) for i in range(1, n)]
    return np.array(p, dtype=np.int32)


@pytest.mark.parametrize("kind,n", [("binary", 15), ("binary", 255), ("chain", 70), ("branch", 256),
                                    ("random", 1), ("random", 65), ("random", 300), ("random", 1024)])
def test_tree_prep_matches_oracle(kind, n):
    g = np.random.default_rng(n)
    p = {"binary": lambda: W.complete_binary_tree(n), "chain": lambda: W.chain_tree(n),
         "branch": lambda: W.branching_tree([8, 4, 2, 2, 1], n), "random": lambda: _random_tree(g, n)}[kind]()
    depth, anc_bits = ssd.tree_prep(p)
    od, oanc = oracle.tree_info(p)
    assert np.array_equal(depth, od)
    bits = ((anc_bits[:, np.arange(n) // 64] >> (np.arange(n) % 64).astype(np.uint64)) & np.uint64(1))
    assert np.array_equal(bits.astype(np.uint8), oanc)


def test_validate_tree_errors():
    assert ssd.validate_tree([1, 2, 3], [-1, 0, 1], 10) == 2
    for toks, par, st in [([1, 2], [0, 0], ssd.E_INVALID_TREE), ([1, 2], [-1, 1], ssd.E_INVALID_TREE),
                          ([1, 2], [-1, 2], ssd.E_INVALID_TREE), ([1, 10], [-1, 0], ssd.E_INVALID_ARG),
                          ([-1, 2], [-1, 0], ssd.E_INVALID_ARG)]:
        with pytest.raises(ssd.SSDError) as e:
            ssd.validate_tree(toks, par, 10)
        assert e.value.status == st


def test_kv_bytes():
    c, t = ssd.kv_bytes(W.GPT2L, 1024, 64)
    assert c == 36 * 20 * 1024 * 64 * 2 and t == 36 * 20 * 64 * 64 * 2
    c, t = ssd.kv_bytes(W.TINY, 10, 3)
    assert c == 2 * 4 * 10 * 32 * 4 and t == 2 * 4 * 3 * 32 * 4
    with pytest.raises(ssd.SSDError):
        ssd.kv_bytes(W.TINY.with_(n_head=3), 10, 3)


# ---- the persistent pass's work split (host-only)

SHAPES = [(20, 1280, 5120, 50257), (4, 256, 1024, 2000), (12, 768, 3072, 50257), (25, 1600, 6400, 50257),
          (1, 64, 256, 100)]


@pytest.mark.parametrize("H,d,M,V", SHAPES)
@pytest.mark.parametrize("nt", [1, 2, 3, 4])
def test_fused_plan_covers_every_unit_once(H, d, M, V, nt):
    """Every weight row block of every stage is computed by exactly one
    workgroup of the XCD that owns it, and every LM-head row block once; XCD
    ranges tile the heads and hidden features.  The attention order is a
    permutation of the 32 ranks of an XCD that puts ranks with fewer QKV row
    blocks first; WPR's extra row blocks go to ranks with fewer FC ones."""
    tab, xh, xf = ssd.fused_plan(H, d, M, V, nt)
    assert xh[0] == 0 and xh[15] == H and xf[0] == 0 and xf[15] == M // 32
    assert all(xh[2 * x + 1] == xh[2 * x + 2] and xf[2 * x + 1] == xf[2 * x + 2] for x in range(7))
    assert all(xh[2 * x + 1] >= xh[2 * x] and xf[2 * x + 1] >= xf[2 * x] for x in range(8))
    rbd = d // 16
    for x in range(8):
        rows = tab[32 * x:32 * x + 32]
        heads = range(xh[2 * x], xh[2 * x + 1])

        def units(slot, cap):
            out = []
            for r in rows:
                assert 0 <= r[slot] <= cap
                out += list(r[slot + 1:slot + 1 + r[slot]])
            return sorted(out)

        pos = rows[:, 0]
        assert sorted(pos.tolist()) == list(range(32))
        by_pos = rows[np.argsort(pos)]
        assert all(by_pos[i, 9] <= by_pos[i + 1, 9] for i in range(31))
        if rows[:, 24].max() > rows[:, 24].min() and rows[:, 19].max() > rows[:, 19].min():
            extra_p = rows[:, 24] == rows[:, 24].max()
            assert rows[extra_p, 19].max() <= rows[~extra_p, 19].min()
        assert units(9, 4) == sorted(p * rbd + 4 * h + j for p in range(3) for h in heads for j in range(4))
        assert units(14, 4) == (list(range(rbd)) if len(heads) else [])
        assert units(19, 4) == list(range(2 * xf[2 * x], 2 * xf[2 * x + 1]))
        assert units(24, 4) == (list(range(rbd)) if xf[2 * x + 1] > xf[2 * x] else [])
        # each stage split into floor/ceil shares over the 32 ranks
        for slot in (9, 14, 19, 24):
            c = rows[:, slot]
            assert c.max() - c.min() <= 1
    head = sorted((int(r[29]), int(r[30])) for r in tab)
    assert head[0][0] == 0 and head[-1][1] == (V + 15) // 16
    assert all(head[i][1] == head[i + 1][0] for i in range(255))


def test_fused_plan_balances_gpt2l_xcds():
    """GPT-2-L: four XCDs own 3 heads and 576 hidden features, four own 2 heads
    and 704, so every XCD streams 4,915,200 bytes of weights per layer."""
    tab, xh, xf = ssd.fused_plan(20, 1280, 5120, 50257, 2)
    heads = [xh[2 * x + 1] - xh[2 * x] for x in range(8)]
    hidden = [32 * (xf[2 * x + 1] - xf[2 * x]) for x in range(8)]
    assert heads == [3, 3, 3, 3, 2, 2, 2, 2]
    assert hidden == [576] * 4 + [704] * 4
    per_xcd = [h * 4 * 64 * 1280 * 2 + f * 2 * 1280 * 2 for h, f in zip(heads, hidden)]
    assert per_xcd == [4915200] * 8


def test_fused_plan_rejects_other_head_dims():
    with pytest.raises(ssd.SSDError):
        ssd.fused_plan(4, 128, 512, 512, 1)  # head dimension 32


def test_host_uniform_equals_the_oracle_generator():
    """ssd_uniform (host, product code) against the oracle's Philox4x64-10
    uniform, itself pinned against numpy's Philox: bit for bit."""
    import oracle
    g = np.random.default_rng(1)
    for _ in range(2000):
        seed, stream, n = (int(x) for x in g.integers(0, 2 ** 63, 3))
        stream %= 4
        assert ssd.uniform(seed, stream, n) == oracle.uniform(seed, stream, n)
    for seed, stream, n in ((0, 0, 0), (2 ** 64 - 1, 2, 2 ** 64 - 1), (7, 2, 255)):
        assert ssd.uniform(seed, stream, n) == oracle.uniform(seed, stream, n)
