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


def host_topk(logits, k):
    """Top-k per row (decreasing logit, lower id first on ties) and the row's
    log-sum-exp (float64), the definition ssd_topk follows."""
    lg = np.asarray(logits, np.float32)
    n, V = lg.shape
    idx = np.empty((n, k), np.int32)
    for r in range(n):
        order = np.lexsort((np.arange(V), -lg[r].astype(np.float64)))
        idx[r] = order[:k]
    val = np.take_along_axis(lg, idx, 1)
    m = lg.astype(np.float64).max(1, keepdims=True)
    lse = (m[:, 0] + np.log(np.exp(lg.astype(np.float64) - m).sum(1))).astype(np.float32)
    return idx, val, lse


class OracleBackend:
    """The staged loop's backend on the CPU oracle: the draft is an oracle
    model of the first layers reading the same cache arrays (a slice of the
    oracle's)."""

    def __init__(self, m, m_draft, kc, vc, max_nodes=64):
        self.m, self.md = m, m_draft
        self.kc, self.vc = kc, vc
        self.kt, self.vt = m.kv(max_nodes), m.kv(max_nodes)
        self.dkt, self.dvt = m_draft.kv(max_nodes), m_draft.kv(max_nodes)
        self.ld = m_draft.cfg.n_layer

    def draft_top(self, P, toks, par, k):
        lg = oracle.tree_verify(self.md, self.kc[:self.ld], self.vc[:self.ld], P, toks, par, self.dkt, self.dvt)
        return host_topk(lg, k)

    def oracle_step(self, P, toks, par):
        lg = oracle.tree_verify(self.m, self.kc, self.vc, P, toks, par, self.kt, self.vt)
        path, nxt = oracle.tree_accept(oracle.GREEDY, toks, par, lg)
        oracle.kv_commit(self.m, self.kc, self.vc, P, self.kt, self.vt, path)
        return path, nxt

    def greedy_predictions(self, window_tokens):
        n = len(window_tokens)
        kt, vt = self.md.kv(n), self.md.kv(n)
        lg = oracle.tree_verify(self.md, None, None, 0, window_tokens, np.arange(-1, n - 1, dtype=np.int32), kt, vt)
        return host_topk(lg, 1)[0][:, 0]


def draft_weights(w, n_layer):
    """The first n_layer blocks of a weight dict plus its embeddings and final LayerNorm."""
    out = dict(w)
    for k, v in w.items():
        if isinstance(v, (list, tuple)):
            out[k] = list(v[:n_layer])
    return out
