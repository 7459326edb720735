"""Greedy speculative decoding with token trees emits exactly the plain greedy
sequence (the paper's claim that output quality is preserved, Sec. 1, 2.3),
checked on the oracle (no GPU)."""
import numpy as np

import oracle
from paper_2308_04623_amd import workloads as W
from tests.helpers import oracle_prefill

CFG = W.TINY
STEPS = 24


def _plain_greedy(m, prompt, n_new, max_ctx):
    kc, vc, _ = oracle_prefill(m, prompt[:-1], max_ctx)
    P, root = len(prompt) - 1, int(prompt[-1])
    kt, vt = m.kv(1), m.kv(1)
    out = []
    while len(out) < n_new:
        lg = oracle.tree_verify(m, kc, vc, P, [root], [-1], kt, vt)
        path, nxt = oracle.tree_accept(oracle.GREEDY, [root], [-1], lg)
        oracle.kv_commit(m, kc, vc, P, kt, vt, path)
        P += len(path)
        out.append(nxt)
        root = nxt
    return out


def _random_tree(g, root, truth, vocab, max_nodes=24):
    """Random tree whose nodes copy the true continuation with prob 0.6."""
    toks, parents, depth = [root], [-1], [0]
    i = 0
    while i < len(toks) and len(toks) < max_nodes:
        for _ in range(int(g.integers(0, 4))):
            if len(toks) >= max_nodes:
                break
            d = depth[i] + 1
            t = truth[d - 1] if (d - 1 < len(truth) and g.random() < 0.6) else int(g.integers(vocab))
            toks.append(t)
            parents.append(i)
            depth.append(d)
        i += 1
    return np.array(toks, np.int32), np.array(parents, np.int32)


def test_tree_speculative_greedy_equals_plain_greedy():
    w = W.make_weights(CFG, 0, perturb_affine=True)
    m = oracle.Model(CFG, w)
    prompt = W.prefix_tokens(40, CFG.vocab, seed=5)
    ref = _plain_greedy(m, prompt, STEPS, 128)

    kc, vc, _ = oracle_prefill(m, prompt[:-1], 128)
    P, root = len(prompt) - 1, int(prompt[-1])
    kt, vt = m.kv(32), m.kv(32)
    g = np.random.default_rng(9)
    out, steps, accepted = [], 0, 0
    while len(out) < STEPS:
        toks, parents = _random_tree(g, root, ref[len(out):], CFG.vocab)
        lg = oracle.tree_verify(m, kc, vc, P, toks, parents, kt, vt)
        path, nxt = oracle.tree_accept(oracle.GREEDY, toks, parents, lg)
        oracle.kv_commit(m, kc, vc, P, kt, vt, path)
        P += len(path)
        emitted = [int(toks[i]) for i in path[1:]] + [nxt]
        out += emitted
        accepted += len(path) - 1
        root = nxt
        steps += 1
    assert out[:STEPS] == ref
    assert steps < STEPS and accepted > 0     # speculation actually skipped steps
