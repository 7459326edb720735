"""Oracle-side helpers shared by the tests: prefill, sequential decoding,
staged loops.  Everything here calls the CPU oracle only."""
import numpy as np

import oracle


def oracle_prefill(m, tokens, max_ctx, chunk=64):
    """Build the KV cache of `tokens` with chain-shaped verify passes plus
    commits (the root of each chunk sits right after the cached prefix)."""
    kc, vc = m.kv(max_ctx), m.kv(max_ctx)
    kt, vt = m.kv(chunk), m.kv(chunk)
    P = 0
    logits = []
    toks = np.asarray(tokens, dtype=np.int32)
    while P < len(toks):
        c = toks[P:P + chunk]
        par = np.arange(-1, len(c) - 1, dtype=np.int32)
        lg = oracle.tree_verify(m, kc, vc, P, c, par, kt, vt)
        oracle.kv_commit(m, kc, vc, P, kt, vt, np.arange(len(c)))
        logits.append(lg)
        P += len(c)
    return kc, vc, np.concatenate(logits, 0)


def oracle_sequential_path_logits(m, kc, vc, P, tokens, path):
    """Decode the root->node path one token at a time (1-node trees plus
    commits) on a copy of the cache; returns the logits of the last token."""
    kc, vc = kc.copy(), vc.copy()
    kt, vt = m.kv(1), m.kv(1)
    lg = None
    for t, node in enumerate(path):
        lg = oracle.tree_verify(m, kc, vc, P + t, [tokens[node]], [-1], kt, vt)
        oracle.kv_commit(m, kc, vc, P + t, kt, vt, [0])
    return lg[0]


def root_path(parents, i):
    out = []
    while i != -1:
        out.append(int(i))
        i = int(parents[i])
    return out[::-1]
