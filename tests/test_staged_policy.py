"""Staged speculation around the verification path (Sec. 3.2), on the CPU:
the draft^2 bigram table, the bigram tree, the oracle tree built from one
draft pass (hand-computed cases), and staged greedy decoding emitting exactly
the plain greedy sequence with the oracle as backend."""
import numpy as np
import pytest

import oracle
from paper_2308_04623_amd import staged as S
from paper_2308_04623_amd import workloads as W
from tests.helpers import OracleBackend, draft_weights, host_topk, oracle_prefill


def test_bigram_table_ranks_and_pads():
    src = [0, 0, 0, 0, 0, 1, 2]
    dst = [1, 1, 2, 3, 3, 5, 4]
    t = S.bigram_table(np.array(src), np.array(dst), vocab=6, k=3)
    # successor counts overall: 1:2, 3:2, 2:1, 4:1, 5:1, 0:0 -> ranking 1, 3, 2, 4, 5, 0
    assert t[0].tolist() == [1, 3, 2]      # counts 2, 2, 1: ties to the lower id
    assert t[1].tolist() == [5, 1, 3]      # own successor, then the global ranking
    assert t[2].tolist() == [4, 1, 3]
    assert t[3].tolist() == [1, 3, 2]      # never seen: the global ranking
    assert t[5].tolist() == [1, 3, 2]


def test_bigram_tree_shape():
    V = 1000
    succ = (np.arange(V)[:, None] * 7 + np.arange(8)[None, :] * 13) % V
    toks, par = S.bigram_tree(5, succ)
    assert len(toks) == 32
    depth = np.zeros(32, int)
    for i in range(1, 32):
        assert par[i] < i
        depth[i] = depth[par[i]] + 1
        j = list(np.where(par == par[i])[0]).index(i)   # rank among siblings
        assert toks[i] == succ[toks[par[i]]][j]
    # branching 4, 2, 1, 1, ... breadth first, cut at 32: 1 + 4 + 8 + 8 + 8 + 3
    assert np.bincount(depth).tolist() == [1, 4, 8, 8, 8, 3]


def _hand_case():
    # bigram tree: root -> (10, 11); 10 -> 12
    toks = np.array([7, 10, 11, 12], np.int32)
    par = np.array([-1, 0, 0, 1], np.int32)
    top_idx = np.array([[10, 20], [30, 12], [11, 40], [50, 51]], np.int32)
    top_val = np.array([[-0.1, -2.0], [-0.5, -1.0], [-0.3, -0.4], [-0.2, -0.3]], np.float32)
    lse = np.zeros(4, np.float32)
    return toks, par, top_idx, top_val, lse


def test_oracle_tree_hand_case():
    toks, par, top_idx, top_val, lse = _hand_case()
    t, p, n_end = S.oracle_tree(toks, par, top_idx, top_val, lse)
    # endorsed: root, node 1 (10 in root's top-2), node 3 (12 in node 1's top-2); node 2 (11) is not.
    # best first: 10 (-0.1), 30 (-0.6), 12 (-1.1), 50 (-1.3), 51 (-1.4), 20 (-2.0)
    assert n_end == 3
    assert t.tolist() == [7, 10, 30, 12, 50, 51, 20]
    assert p.tolist() == [-1, 0, 1, 1, 3, 3, 0]
    t4, p4, _ = S.oracle_tree(toks, par, top_idx, top_val, lse, cap=4)
    assert t4.tolist() == [7, 10, 30, 12] and p4.tolist() == [-1, 0, 1, 1]


def test_endorsed_subtree_hand_case():
    toks, par, top_idx, _, _ = _hand_case()
    keep, t, p = S.endorsed_subtree(toks, par, top_idx)
    # root, node 1 (10 in the root's top-2), node 3 (12 in node 1's top-2)
    assert keep.tolist() == [0, 1, 3] and t.tolist() == [7, 10, 12] and p.tolist() == [-1, 0, 1]
    keep1, _, _ = S.endorsed_subtree(toks, par, top_idx, top=1)   # 12 is node 1's second choice
    assert keep1.tolist() == [0, 1]


def test_endorsed_subtree_matches_oracle_tree_count():
    g = np.random.default_rng(2)
    for s in range(50):
        n = int(g.integers(1, 32))
        par = np.array([-1] + [int(g.integers(0, i)) for i in range(1, n)], np.int32)
        toks = g.integers(0, 6, n).astype(np.int32)
        top_idx = g.integers(0, 6, (n, 2)).astype(np.int32)
        keep, t, p = S.endorsed_subtree(toks, par, top_idx)
        _, _, n_end = S.oracle_tree(toks, par, top_idx, np.zeros((n, 2), np.float32), np.zeros(n, np.float32))
        assert len(keep) == n_end
        assert np.array_equal(t, toks[keep])
        assert all(p[i] < i and keep[p[i]] == par[keep[i]] for i in range(1, len(keep)))


def test_oracle_tree_uses_log_probabilities():
    toks, par, top_idx, top_val, lse = _hand_case()
    lse = np.array([0.0, 5.0, 0.0, 0.0], np.float32)   # node 1's children become unlikely
    t, p, _ = S.oracle_tree(toks, par, top_idx, top_val, lse, cap=4)
    assert t.tolist() == [7, 10, 20, 30] and p.tolist() == [-1, 0, 0, 1]


def test_host_topk_definition():
    lg = np.array([[1.0, 3.0, 3.0, 2.0], [0.0, 0.0, 0.0, 0.0]], np.float32)
    idx, val, lse = host_topk(lg, 3)
    assert idx.tolist() == [[1, 2, 3], [0, 1, 2]]
    assert val.tolist() == [[3.0, 3.0, 2.0], [0.0, 0.0, 0.0]]
    assert np.allclose(lse, np.log(np.exp(lg.astype(np.float64)).sum(1)))


def test_staged_greedy_equals_plain_greedy_on_the_oracle():
    cfg = W.TINY
    w = W.make_weights(cfg, 0, perturb_affine=True)
    m = oracle.Model(cfg, w)
    md = oracle.Model(cfg.with_(n_layer=1), draft_weights(w, 1))
    prompt = W.prefix_tokens(40, cfg.vocab, seed=5)
    n_new = 24

    def backend():
        kc, vc, _ = oracle_prefill(m, prompt[:-1], 160)
        return OracleBackend(m, md, kc, vc)

    b0 = backend()
    stream = S.bigram_stream(cfg.vocab, 1024, seed=4)
    preds = np.concatenate([b0.greedy_predictions(stream[s:s + 64]) for s in range(0, 1024, 64)])
    succ = S.bigram_table(stream, preds, cfg.vocab)
    plain = S.plain_greedy(b0, len(prompt) - 1, int(prompt[-1]), n_new)
    st = S.staged_greedy(backend(), len(prompt) - 1, int(prompt[-1]), n_new, succ)
    assert st.tokens == plain.tokens
    assert st.steps <= n_new and all(1 <= n <= S.MAX_ORACLE_NODES for n in st.oracle_nodes)


def test_cdf_first_tree_hand_case():
    """Breadth-first numbering, children from the picks at U_u + offsets
    (duplicates dropped), bigram matches expandable, others leaves, cap."""
    bt = np.array([5, 1, 2, 3], np.int32)
    bp = np.array([-1, 0, 0, 1], np.int32)
    picks = {(0, 0.5): 2, (0, 0.6): 9, (0, 0.4): 2, (2, 0.25): 7, (2, 0.35): 7, (2, 0.15): 8}
    us = {0: 0.5, 1: 0.25}
    pick = lambda rows, u: [picks[(r, round(x, 6))] for r, x in zip(rows, u)]
    t, p = S.cdf_first_tree(bt, bp, 0, lambda u: us[u], pick, offsets=(0.0, 0.1, -0.1))
    # root -> 2 (bigram node 2, expandable), 9 (leaf); node 1 (token 2) -> 7, 8
    assert t.tolist() == [5, 2, 9, 7, 8] and p.tolist() == [-1, 0, 0, 1, 1]
    t, p = S.cdf_first_tree(bt, bp, 0, lambda u: us[u], pick, offsets=(0.0, 0.1, -0.1), cap=4)
    assert t.tolist() == [5, 2, 9, 7]


@pytest.mark.slow
def test_cdf_first_trees_keep_the_target_exact():
    """The staged loop's CDF-first assembly with the oracle's SAMPLE_CDF walk:
    over a Markov-table target on 6 tokens (draft = another table), the
    joint law of the first three emitted tokens equals the target's
    (chi-square), and the trees are followed."""
    from tests.test_oracle_accept import V6, _cdf_pick, _chi2_p, _markov_tables
    p_tab, q_tab = _markov_tables()
    logit_tab = np.log(p_tab).astype(np.float32)
    succ = np.stack([np.lexsort((np.arange(V6), -q_tab[v].astype(np.float64))) for v in range(V6)]).astype(np.int32)
    trials, x0, hits = 12000, 2, 0
    counts = np.zeros((V6, V6, V6))
    for t in range(trials):
        seq, step = [x0], 0
        while len(seq) < 4:
            seed = t * 8 + step
            bt, bp = S.bigram_tree(seq[-1], succ, branch=(3, 2, 1), cap=12)
            pick = lambda rows, us: [_cdf_pick(q_tab[bt[r]].astype(np.float64), 1.0, U) for r, U in zip(rows, us)]
            ot, op = S.cdf_first_tree(bt, bp, seed, lambda u: oracle.uniform(seed, 2, u), pick, cap=16)
            path, nxt = oracle.tree_accept(oracle.SAMPLE_CDF, ot, op, logit_tab[ot], None, 1.0, seed)
            hits += len(path) - 1
            seq += [int(ot[i]) for i in path[1:]] + [int(nxt)]
            step += 1
        counts[seq[1], seq[2], seq[3]] += 1
    want = np.einsum("a,ab,bc->abc", p_tab[x0], p_tab, p_tab).ravel() * trials
    assert _chi2_p(counts.ravel(), want) > 1e-3
    assert hits > trials // 2
