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


def _header_functions():
    txt = open(os.path.join(ROOT, "include", "ssd.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(ssd_[a-z_0-9]+)\s*\(", txt)))


def test_library_exports_every_declared_function():
    L = ssd.lib()
    names = _header_functions()
    assert len(names) >= 17
    for n in names:
        assert hasattr(L, n), n
    assert sorted(ssd.EXPORTS) == names


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


def test_gemm_path_switch_validates():
    with pytest.raises(ssd.SSDError):
        ssd.set_gemm_path(7)
    ssd.set_gemm_path(ssd.GEMM_AUTO)


def test_weight_prefetch_switch_validates():
    assert ssd.lib().ssd_set_weight_prefetch(2) != 0
    ssd.set_weight_prefetch(False)
    ssd.set_weight_prefetch(True)
