"""Pins of the oracle's accept/reject walk (no GPU).

- Greedy: hand-built logits with known answers; a chain accepts the longest
  prefix whose tokens equal the running argmax.
- Sampling on a chain equals a textbook speculative-sampling loop (Leviathan
  et al.) written here from its definition and fed the same uniforms.
- Distribution preservation (Sec. 2.3): Monte Carlo on a Markov-table target
  and draft over a 6-token vocabulary; the joint law of the first three
  emitted tokens must match the target's (chi-square), for trees whose
  siblings are drawn without replacement and independently.  Planted mistakes
  in a Python copy of the rule must fail the same test at the same trial count.
- The single-child acceptance probability equals sum_x min(p(x), q(x)).
"""
import numpy as np
import pytest

import oracle
from paper_2308_04623_amd import workloads as W

GREEDY, WOR, IID = oracle.GREEDY, oracle.SAMPLE_WOR, oracle.SAMPLE_IID


# ---------------------------------------------------------------- greedy

def _onehot_logits(n, V, argmaxes, base=0.0):
    lg = np.full((n, V), base, dtype=np.float32)
    for i, a in enumerate(argmaxes):
        lg[i, a] = 1.0
    return lg


def test_greedy_deepest_match():
    parents = [-1, 0, 0, 1, 2, 4]
    toks = [9, 3, 5, 7, 6, 2]
    # argmax per node: root->5, so node 2 (tok 5) matches; node 2 -> 6, node 4 matches;
    # node 4 -> 1, node 5 (tok 2) does not match
    lg = _onehot_logits(6, 10, [5, 0, 6, 0, 1, 8])
    path, nxt = oracle.tree_accept(GREEDY, toks, parents, lg)
    assert path.tolist() == [0, 2, 4] and nxt == 1


def test_greedy_ties_lowest_index_and_lowest_token():
    parents = [-1, 0, 0]
    toks = [1, 4, 4]                 # duplicate siblings: both match
    lg = np.zeros((3, 8), dtype=np.float32)
    lg[0, 4] = 2.0
    lg[1, [2, 6]] = 3.0              # tie between tokens 2 and 6 -> 2
    lg[2, 5] = 1.0
    path, nxt = oracle.tree_accept(GREEDY, toks, parents, lg)
    assert path.tolist() == [0, 1] and nxt == 2


def test_greedy_nothing_accepted():
    lg = _onehot_logits(3, 8, [7, 1, 1])
    path, nxt = oracle.tree_accept(GREEDY, [0, 1, 2], [-1, 0, 0], lg)
    assert path.tolist() == [0] and nxt == 7


def test_greedy_chain_longest_prefix():
    rng = np.random.default_rng(0)
    V, n = 16, 9
    for _ in range(50):
        lg = rng.standard_normal((n, V)).astype(np.float32)
        g = lg.argmax(1)
        toks = rng.integers(0, V, n).astype(np.int32)
        k = rng.integers(0, n)
        toks[1:k + 1] = g[:k]                # first k draft tokens agree
        path, nxt = oracle.tree_accept(GREEDY, toks, W.chain_tree(n), lg)
        acc = 0
        while acc + 1 < n and toks[acc + 1] == g[acc]:
            acc += 1
        assert path.tolist() == list(range(acc + 1)) and nxt == g[acc]


# ---------------------------------------------------------------- sampling: chain

def _softmax(x):
    e = np.exp(x - x.max())
    return e / e.sum()


def _cdf_pick(w, Z, U):
    c = 0.0
    last = 0
    for v, x in enumerate(w):
        c += x
        if x > 0:
            last = v
        if c > U * Z:
            return v
    return last


def _leviathan_chain(toks, p, q, seed):
    """Speculative sampling for a chain draft: token i+1 was proposed from
    q[i]; accept with prob min(1, p[i](x)/q[i](x)); on the first rejection
    resample from norm(max(p[i]-q[i], 0)); if all pass, sample p[last]."""
    n = len(toks)
    for i in range(n - 1):
        x = toks[i + 1]
        U = oracle.uniform(seed, 0, i + 1)
        if q[i][x] == 0 or U < p[i][x] / q[i][x]:
            continue
        r = np.maximum(p[i] - q[i] / q[i].sum(), 0)
        return list(range(i + 1)), _cdf_pick(r, r.sum(), oracle.uniform(seed, 1, i))
    return list(range(n)), _cdf_pick(p[n - 1], 1.0, oracle.uniform(seed, 1, n - 1))


def test_chain_sampling_equals_textbook_speculative_sampling():
    rng = np.random.default_rng(1)
    V, n = 12, 6
    for seed in range(300):
        lg = (rng.standard_normal((n, V)) * 1.5).astype(np.float32)
        p = [_softmax(lg[i].astype(np.float64)) for i in range(n)]
        q = rng.dirichlet(np.ones(V) * 0.5, size=n).astype(np.float32)
        toks = np.zeros(n, dtype=np.int32)
        for i in range(1, n):
            qi = q[i - 1].astype(np.float64)
            toks[i] = rng.choice(V, p=qi / qi.sum())
        qd = [q[i].astype(np.float64) for i in range(n)]
        want_path, want_next = _leviathan_chain(toks, p, qd, seed)
        for mode in (WOR, IID):
            path, nxt = oracle.tree_accept(mode, toks, W.chain_tree(n), lg, q, 1.0, seed)
            assert path.tolist() == want_path and nxt == want_next, (seed, mode)


# ---------------------------------------------------------------- sampling: Monte Carlo

V6 = 6


def _markov_tables():
    g = np.random.default_rng(7)
    p = g.dirichlet(np.ones(V6) * 2.0, size=V6)         # target p(next | prev)
    q = g.dirichlet(np.ones(V6) * 1.0, size=V6)         # draft q(next | prev)
    return p, q.astype(np.float32)


def _draw_children(g, q, k, wor):
    if not wor:
        w = q.astype(np.float64)
        return list(g.choice(V6, size=k, p=w / w.sum()))
    out, w = [], q.astype(np.float64).copy()
    for _ in range(k):
        x = g.choice(V6, p=w / w.sum())
        out.append(int(x))
        w[x] = 0.0
    return out


def _build_tree(g, root_tok, q_tab, branching, wor):
    toks, parents = [root_tok], [-1]
    frontier = [0]
    for b in branching:
        nxt = []
        for u in frontier:
            for x in _draw_children(g, q_tab[toks[u]], b, wor):
                toks.append(int(x))
                parents.append(u)
                nxt.append(len(toks) - 1)
        frontier = nxt
    return np.array(toks, dtype=np.int32), np.array(parents, dtype=np.int32)


def _py_accept(toks, parents, p_rows, q_rows, seed, wor, mutant):
    """Python copy of the rule with an optional planted mistake (power check)."""
    n = len(toks)
    u, path = 0, [0]
    while True:
        r = p_rows[u].copy()
        Z = 1.0
        qq = q_rows[u].astype(np.float64).copy()
        Zq = qq.sum()
        acc = -1
        for c in range(u + 1, n):
            if parents[c] != u:
                continue
            x = toks[c]
            U = oracle.uniform(seed, 0, c)
            if mutant == "ignore_q":
                ok = U < r[x] / Z
            else:
                ok = (r[x] > 0) if qq[x] == 0 else U < (r[x] / Z) / (qq[x] / Zq)
            if ok:
                acc = c
                break
            t = r / Z - qq / Zq
            r = t if mutant == "no_clamp" else np.maximum(t, 0.0)
            Z = r.sum()
            if wor and mutant != "keep_q":
                qq[x] = 0.0
                Zq = qq.sum()
        if acc < 0:
            break
        path.append(acc)
        u = acc
    U2 = oracle.uniform(seed, 1, u)
    w = np.maximum(r, 0) if mutant == "no_clamp" else r
    return path, _cdf_pick(w, w.sum() if mutant == "no_clamp" else Z, U2)


def _mc_first3(trials, wor, accept_fn, seed0=0):
    p_tab, q_tab = _markov_tables()
    logit_tab = np.log(p_tab).astype(np.float32)
    p_rows_tab = [_softmax(logit_tab[v].astype(np.float64)) for v in range(V6)]
    g = np.random.default_rng([11, int(wor)])
    counts = np.zeros((V6, V6, V6))
    x0 = 2
    for t in range(trials):
        seq = [x0]
        step = 0
        while len(seq) < 4:
            toks, parents = _build_tree(g, seq[-1], q_tab, [3, 2], wor)
            lg = logit_tab[toks]
            dp = q_tab[toks]
            path, nxt = accept_fn(toks, parents, lg, dp, [p_rows_tab[x] for x in toks], seed0 + t * 8 + step)
            seq += [int(toks[i]) for i in path[1:]] + [int(nxt)]
            step += 1
        counts[seq[1], seq[2], seq[3]] += 1
    want = np.einsum("a,ab,bc->abc", p_tab[x0], p_tab, p_tab)
    # the target is the table itself; logits were rounded to float32 on the way
    return counts.ravel(), want.ravel() * trials


def _chi2_p(counts, expected):
    from scipy.stats import chisquare
    return chisquare(counts, expected * counts.sum() / expected.sum()).pvalue


TRIALS = 20000


@pytest.mark.slow
@pytest.mark.parametrize("wor", [True, False])
def test_monte_carlo_preserves_target_distribution(wor):
    mode = WOR if wor else IID
    fn = lambda toks, par, lg, dp, prow, seed: oracle.tree_accept(mode, toks, par, lg, dp, 1.0, seed)
    counts, exp = _mc_first3(TRIALS, wor, fn)
    assert _chi2_p(counts, exp) > 1e-3


@pytest.mark.slow
@pytest.mark.parametrize("mutant,wor", [("ignore_q", True), ("keep_q", True), ("no_clamp", False)])
def test_monte_carlo_detects_planted_mistakes(mutant, wor):
    # the unmutated Python copy agrees with the oracle decision for decision
    p_tab, q_tab = _markov_tables()
    g = np.random.default_rng(5)
    logit_tab = np.log(p_tab).astype(np.float32)
    for s in range(200):
        toks, par = _build_tree(g, int(g.integers(V6)), q_tab, [3, 2], wor)
        prow = [_softmax(logit_tab[x].astype(np.float64)) for x in toks]
        a = _py_accept(toks, par, prow, q_tab[toks], s, wor, None)
        b = oracle.tree_accept(WOR if wor else IID, toks, par, logit_tab[toks], q_tab[toks], 1.0, s)
        assert a[0] == b[0].tolist() and a[1] == b[1]
    fn = lambda toks, par, lg, dp, prow, seed: _py_accept(toks, par, prow, dp, seed, wor, mutant)
    counts, exp = _mc_first3(TRIALS, wor, fn)
    assert _chi2_p(counts, exp) < 1e-6, mutant


def test_single_child_acceptance_rate():
    g = np.random.default_rng(3)
    V = 10
    lg = (g.standard_normal(V) * 1.2).astype(np.float32)
    p = _softmax(lg.astype(np.float64))
    q = g.dirichlet(np.ones(V)).astype(np.float32)
    qd = q.astype(np.float64)
    qd = qd / qd.sum()
    want = np.minimum(p, qd).sum()
    trials = 20000
    acc = 0
    for s in range(trials):
        x = g.choice(V, p=qd)
        path, _ = oracle.tree_accept(WOR, [0, x], [-1, 0], np.stack([lg, lg]), np.stack([q, q]), 1.0, s)
        acc += len(path) == 2
    sd = np.sqrt(want * (1 - want) / trials)
    assert abs(acc / trials - want) < 4 * sd


def test_leaf_root_samples_target():
    # a lone root: next token ~ softmax(logits / T); check the temperature too
    V = 5
    lg = np.array([[0.0, 1.0, 2.0, -1.0, 0.5]], dtype=np.float32)
    for T in (1.0, 0.5):
        p = _softmax(lg[0].astype(np.float64) / T)
        cnt = np.zeros(V)
        for s in range(20000):
            _, nxt = oracle.tree_accept(WOR, [0], [-1], lg, np.full((1, V), 0.2, np.float32), T, s)
            cnt[nxt] += 1
        assert _chi2_p(cnt, p) > 1e-3


def test_sampling_error_paths():
    lg = np.zeros((2, 4), dtype=np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.tree_accept(WOR, [0, 1], [-1, 0], lg, None)
    with pytest.raises(oracle.OracleError):
        oracle.tree_accept(WOR, [0, 1], [-1, 0], lg, np.ones((2, 4), np.float32), 0.0)
    with pytest.raises(oracle.OracleError):
        oracle.tree_accept(GREEDY, [0, 9], [-1, 0], lg)
