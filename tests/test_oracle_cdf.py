"""Pins of the oracle's CDF-first sampling mode (no GPU).

Sec. 4 suggests drawing the multinomial CDF samples first and assembling
the batch around them (e.g. keeping only draft ranks 5-10 when the draw is
0.99).  The reading taken (ssdref.h, SAMPLE_CDF): node u owns the uniform
U_u = uniform(seed, 2, u), known before the tree is built; the oracle's token
at u is the inverse CDF of its target at U_u (ascending token id); the walk
follows the child carrying it, and otherwise emits it.  A tree builder may
use U_u to choose u's children (here: the draft's inverse CDF at U_u and at
U_u +- 0.15), but a node's own index, token and presence never depend on its
own uniform.  Pinned by:

- Closed form: a lone root emits the inverse CDF of softmax(logits / T)
  (top-k restricted) at its uniform, with the helpers the other sampling
  pins use.
- Definition: on random trees, the path and extra token equal a loop
  written here from the rule, fed the same uniforms.
- Monte Carlo: over a Markov-table target on 6 tokens, the joint law of the
  first three emitted tokens with CDF-first trees equals the target's (full
  vocabulary and top-3); chi-square.
- Power check: a Python copy of the rule that reuses the parent's uniform at
  the child, or draws from the full vocabulary under top-k, fails it.
"""
import numpy as np
import pytest

import oracle
from paper_2308_04623_amd import workloads as W
from tests.test_oracle_accept import V6, _cdf_pick, _chi2_p, _markov_tables, _softmax
from tests.test_oracle_sampling_variants import topk_target

CDF = oracle.SAMPLE_CDF


@pytest.mark.parametrize("k,T", [(0, 1.0), (0, 0.6), (5, 1.0), (50, 1.3)])
def test_lone_root_is_inverse_cdf_of_target(k, T):
    g = np.random.default_rng(3 + k)
    V = 90
    lg = np.round(g.standard_normal((1, V)) * 2, 1).astype(np.float32)
    p = topk_target(lg[0], k, T)
    for s in range(400):
        path, nxt = oracle.tree_accept(CDF, [0], [-1], lg, None, T, s, top_k=k)
        assert path.tolist() == [0] and nxt == _cdf_pick(p, 1.0, oracle.uniform(s, 2, 0)), s


def _py_walk(toks, parents, p_rows, seed, mutant=None, p_full=None):
    """The rule, written out: x = inverse CDF of p_u at U_u; the first child
    (lowest index) with token x is followed, otherwise x is emitted."""
    u, path = 0, [0]
    while True:
        U = oracle.uniform(seed, 2, parents[u] if mutant == "parent_uniform" and u > 0 else u)
        p = p_full[u] if mutant == "full_vocab" else p_rows[u]
        x = _cdf_pick(p, 1.0, U)
        kids = [c for c in range(u + 1, len(toks)) if parents[c] == u and toks[c] == x]
        if not kids:
            return path, x
        path.append(kids[0])
        u = kids[0]


def test_random_trees_follow_the_definition():
    g = np.random.default_rng(8)
    V, n = 10, 24
    for s in range(300):
        par = np.array([-1] + [int(g.integers(0, i)) for i in range(1, n)], np.int32)
        toks = g.integers(0, V, n).astype(np.int32)   # duplicate siblings happen: the lowest index wins
        lg = (g.standard_normal((n, V)) * 1.2).astype(np.float32)
        k = int(s % 3) * 3
        rows = [topk_target(lg[i], k) for i in range(n)]
        want = _py_walk(toks, par, rows, s)
        path, nxt = oracle.tree_accept(CDF, toks, par, lg, None, 1.0, s, top_k=k)
        assert path.tolist() == want[0] and nxt == want[1], s


def test_argument_rules():
    lg = np.zeros((2, 4), np.float32)
    with pytest.raises(oracle.OracleError):          # no draft rows in this mode
        oracle.tree_accept(CDF, [0, 1], [-1, 0], lg, np.ones((2, 4), np.float32))
    with pytest.raises(oracle.OracleError):          # temperature must be positive
        oracle.tree_accept(CDF, [0, 1], [-1, 0], lg, None, 0.0)


# ---------------------------------------------------------------- Monte Carlo

def _cdf_first_tree(root_tok, q_tab, seed, branching=(3, 2), offsets=(0.0, 0.15, -0.15)):
    """CDF-first assembly: nodes get indices in breadth-first creation order;
    node u's children are the draft's inverse-CDF picks at U_u + offsets
    (wrapped into [0, 1), duplicates dropped, at most branching[depth])."""
    toks, parents, frontier = [root_tok], [-1], [0]
    for b in branching:
        nxt = []
        for u in frontier:
            U = oracle.uniform(seed, 2, u)
            q = q_tab[toks[u]].astype(np.float64)
            kids = []
            for o in offsets:
                x = _cdf_pick(q, q.sum(), (U + o) % 1.0)
                if x not in kids:
                    kids.append(x)
            for x in kids[:b]:
                toks.append(int(x))
                parents.append(u)
                nxt.append(len(toks) - 1)
        frontier = nxt
    return np.array(toks, np.int32), np.array(parents, np.int32)


def _mc_first3(trials, k, accept_fn):
    p_tab, q_tab = _markov_tables()
    logit_tab = np.log(p_tab).astype(np.float32)
    pk_tab = np.stack([topk_target(logit_tab[v], k) for v in range(V6)])
    pf_tab = np.stack([_softmax(logit_tab[v].astype(np.float64)) for v in range(V6)])
    counts = np.zeros((V6, V6, V6))
    x0, hits = 2, 0
    for t in range(trials):
        seq, step = [x0], 0
        while len(seq) < 4:
            seed = t * 8 + step
            toks, par = _cdf_first_tree(seq[-1], q_tab, seed)
            path, nxt = accept_fn(toks, par, logit_tab[toks], pk_tab[toks], pf_tab[toks], seed)
            hits += len(path) - 1
            seq += [int(toks[i]) for i in path[1:]] + [int(nxt)]
            step += 1
        counts[seq[1], seq[2], seq[3]] += 1
    want = np.einsum("a,ab,bc->abc", pk_tab[x0], pk_tab, pk_tab).ravel()
    return counts.ravel(), want * trials, hits


TRIALS = 20000


@pytest.mark.slow
@pytest.mark.parametrize("k", [0, 3])
def test_monte_carlo_cdf_first_trees_keep_the_target(k):
    fn = lambda toks, par, lg, pk, pf, seed: oracle.tree_accept(CDF, toks, par, lg, None, 1.0, seed, top_k=k)
    counts, exp, hits = _mc_first3(TRIALS, k, fn)
    nz = exp > 0
    assert counts[~nz].sum() == 0
    assert _chi2_p(counts[nz], exp[nz]) > 1e-3
    assert hits > TRIALS // 2          # the assembled trees are followed, not just the extra token


@pytest.mark.slow
@pytest.mark.parametrize("mutant,k", [("parent_uniform", 0), ("full_vocab", 3)])
def test_monte_carlo_detects_planted_cdf_mistakes(mutant, k):
    p_tab, q_tab = _markov_tables()
    logit_tab = np.log(p_tab).astype(np.float32)
    # the unmutated copy agrees with the oracle decision for decision
    for s in range(200):
        toks, par = _cdf_first_tree(int(s % V6), q_tab, s)
        pk = [topk_target(logit_tab[x], k) for x in toks]
        a = _py_walk(toks, par, pk, s)
        b = oracle.tree_accept(CDF, toks, par, logit_tab[toks], None, 1.0, s, top_k=k)
        assert a[0] == b[0].tolist() and a[1] == b[1], s
    fn = lambda toks, par, lg, pk, pf, seed: _py_walk(toks, par, pk, seed, mutant, pf)
    counts, exp, _ = _mc_first3(TRIALS, k, fn)
    nz = exp > 0
    bad = counts[~nz].sum() > 0 or _chi2_p(counts[nz], exp[nz]) < 1e-6
    assert bad, mutant


def test_cdf_pick_is_the_lone_root_draw():
    """ssdref_cdf_pick at a node's own uniform is the SAMPLE_CDF draw there
    (pinned above), for full-vocabulary targets."""
    g = np.random.default_rng(12)
    for s in range(200):
        V = int(g.integers(2, 300))
        T = float(g.choice([0.5, 1.0, 1.7]))
        lg = (g.standard_normal((1, V)) * 2).astype(np.float32)
        _, want = oracle.tree_accept(CDF, [0], [-1], lg, None, T, s)
        assert oracle.cdf_pick(lg[0], T, oracle.uniform(s, 2, 0)) == want, s
    with pytest.raises(oracle.OracleError):
        oracle.cdf_pick(np.zeros(4, np.float32), 1.0, 1.0)
