"""Staged speculative decoding around the tree-verification path (Sec. 3.2).

The paper stages the speculation: a draft model proposes a tree of tokens
(Sec. 3.1), and a still cheaper draft^2 model proposes the draft's own
candidates.  Here:
  - draft^2 is a bigram table, vocab x top-8 successors, counted from the
    draft's greedy predictions on a seeded uniform token stream (windows of
    256 tokens, teacher forced);
  - the draft is the oracle's first layers with its final LayerNorm and tied
    head (ssd_model_prefix_view), sharing the oracle's KV cache;
  - each step builds a bigram tree from the last emitted token, runs one
    draft verification over it, keeps ("endorses") the bigram nodes whose
    path agrees with the draft's top-2 at every parent, and hands the oracle
    the endorsed nodes plus the draft's top-2 children of each, best first by
    draft log-probability, at most 64 nodes;
  - the oracle verifies that tree, the greedy walk accepts a path, the path's
    K/V are committed.
Greedy acceptance makes the emitted sequence the oracle's greedy sequence
whatever the trees (Sec. 2.3), which the tests check against plain decoding.

CDF-first sampling (Sec. 4 suggests drawing the multinomial CDF samples
first and assembling the batch around them): every oracle-tree node u owns
the uniform U_u = ssd_uniform(seed, 2, u), read before the tree exists.  The
oracle's token at u will be the inverse CDF of its target at U_u
(SSD_ACCEPT_SAMPLE_CDF), so u's children are the draft's own inverse-CDF
picks at U_u and a few nearby uniforms: the tokens the oracle is likely to
draw there.  Nodes are numbered in breadth-first creation order and a node's
uniform only decides its children, which keeps every emitted token an exact
draw from the oracle's target.

The policy code here is pure host logic over small arrays; the model work
goes through a backend (the GPU library in this module, the CPU oracle in the
tests).
"""
from __future__ import annotations

import heapq
import time
from dataclasses import dataclass, field
from typing import List, Sequence, Tuple

import numpy as np

BRANCH = (4, 2, 1, 1, 1, 1)  # bigram tree: children per node at depth 0, 1, ...
DRAFT_TOP = 2                # endorsement and expansion width
BIGRAM_TOP = 8
MAX_BIGRAM_NODES = 32
MAX_ORACLE_NODES = 64
CDF_OFFSETS = (0.0, 0.05, -0.05)  # CDF-first children: the draft's picks at U_u + these


# ---------------------------------------------------------------- draft^2: bigram table

def bigram_table(src: np.ndarray, dst: np.ndarray, vocab: int, k: int = BIGRAM_TOP) -> np.ndarray:
    """succ[v][0..k) from (token, predicted next token) pairs: the k most
    frequent successors of v (count, then lower id), padded with the most
    frequent successors overall (same order) not already in the row."""
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    key = src * vocab + dst
    uk, cnt = np.unique(key, return_counts=True)
    a, b = uk // vocab, uk % vocab
    # global successor ranking
    gcnt = np.bincount(dst, minlength=vocab)
    glob = np.lexsort((np.arange(vocab), -gcnt))[: 4 * k]
    succ = np.empty((vocab, k), np.int32)
    # per-row ranking: sort pairs by (row, -count, successor id)
    order = np.lexsort((b, -cnt, a))
    a, b = a[order], b[order]
    starts = np.searchsorted(a, np.arange(vocab))
    ends = np.searchsorted(a, np.arange(vocab), side="right")
    for v in range(vocab):
        row = list(b[starts[v]:min(ends[v], starts[v] + k)])
        for gtok in glob:
            if len(row) >= k:
                break
            if gtok not in row:
                row.append(int(gtok))
        succ[v] = row[:k]
    return succ


def bigram_stream(vocab: int, n_tokens: int = 1 << 15, seed: int = 4) -> np.ndarray:
    return np.random.default_rng(seed).integers(0, vocab, n_tokens).astype(np.int32)


# ---------------------------------------------------------------- trees

def bigram_tree(root: int, succ: np.ndarray, branch: Sequence[int] = BRANCH,
                cap: int = MAX_BIGRAM_NODES) -> Tuple[np.ndarray, np.ndarray]:
    """Breadth-first tree from the root: a node at depth d gets the first
    branch[d] bigram successors of its token (the last entry repeats),
    truncated at cap nodes."""
    toks, par, dep = [int(root)], [-1], [0]
    i = 0
    while i < len(toks) and len(toks) < cap:
        b = branch[min(dep[i], len(branch) - 1)]
        for j in range(b):
            if len(toks) >= cap:
                break
            toks.append(int(succ[toks[i]][j]))
            par.append(i)
            dep.append(dep[i] + 1)
        i += 1
    return np.array(toks, np.int32), np.array(par, np.int32)


def oracle_tree(toks: np.ndarray, par: np.ndarray, top_idx: np.ndarray, top_val: np.ndarray, lse: np.ndarray,
                top: int = DRAFT_TOP, cap: int = MAX_ORACLE_NODES) -> Tuple[np.ndarray, np.ndarray, int]:
    """The oracle's tree from one draft pass over a bigram tree.

    top_idx/top_val/lse: the draft's top tokens, their logits and the row
    log-sum-exp at every bigram node.  A bigram node is endorsed when its
    parent is endorsed and its token is among the parent's `top` draft
    tokens (the root is endorsed).  Candidates: the root and the `top` draft
    children of every endorsed node, scored by cumulative draft
    log-probability; the best `cap` are kept (best first, earlier candidates
    first on ties), which keeps every kept node's parent.  Returns tokens,
    parents (topological order) and the number of endorsed nodes."""
    n = len(toks)
    endorsed = np.zeros(n, bool)
    endorsed[0] = True
    kids = [[] for _ in range(n)]
    for i in range(1, n):
        kids[par[i]].append(i)
        p = par[i]
        endorsed[i] = endorsed[p] and int(toks[i]) in set(int(t) for t in top_idx[p, :top])
    # candidates: (score, creation order, token, parent candidate, bigram node or -1)
    cand = [(0.0, 0, int(toks[0]), -1, 0)]
    heap = []  # (-score, order, candidate id)
    order = 1

    def expand(ci):
        nonlocal order
        score, _, _, _, b = cand[ci]
        if b < 0 or not endorsed[b]:
            return
        for j in range(top):
            t = int(top_idx[b, j])
            lp = float(top_val[b, j]) - float(lse[b])
            match = [k for k in kids[b] if int(toks[k]) == t and endorsed[k]]
            cand.append((score + lp, order, t, ci, match[0] if match else -1))
            heapq.heappush(heap, (-(score + lp), order, len(cand) - 1))
            order += 1

    kept = [0]
    expand(0)
    while heap and len(kept) < cap:
        _, _, ci = heapq.heappop(heap)
        kept.append(ci)
        expand(ci)
    # topological order = order of acceptance into `kept` (a parent is kept before its children)
    pos = {ci: i for i, ci in enumerate(kept)}
    t_out = np.array([cand[ci][2] for ci in kept], np.int32)
    p_out = np.array([-1 if cand[ci][3] < 0 else pos[cand[ci][3]] for ci in kept], np.int32)
    return t_out, p_out, int(endorsed.sum())


def endorsed_subtree(toks: np.ndarray, par: np.ndarray, top_idx: np.ndarray,
                     top: int = DRAFT_TOP) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """The bigram nodes the draft endorses (the root; a node whose parent is
    endorsed and whose token is among the parent's `top` draft tokens), in
    bigram order: their bigram indices, tokens and renumbered parents.  The
    draft ran on every one of them, so its work on them can be reused."""
    keep, pos = [0], {0: 0}
    for i in range(1, len(toks)):
        p = int(par[i])
        if p in pos and int(toks[i]) in set(int(t) for t in top_idx[p, :top]):
            pos[i] = len(keep)
            keep.append(i)
    k = np.array(keep, np.int32)
    return k, toks[k].astype(np.int32), np.array([-1] + [pos[int(par[i])] for i in keep[1:]], np.int32)


def cdf_first_tree(bt: np.ndarray, bp: np.ndarray, seed: int, uniform, pick, offsets: Sequence[float] = CDF_OFFSETS,
                   cap: int = MAX_ORACLE_NODES) -> Tuple[np.ndarray, np.ndarray]:
    """CDF-first oracle tree over a draft pass on the bigram tree (bt, bp).

    Oracle node u (numbered in breadth-first creation order) stands for a
    bigram node b(u) the draft ran on, or for a leaf.  A node with a bigram
    node gets as children the draft's picks at U_u + offsets (wrapped into
    [0, 1), duplicates dropped): uniform(u) gives U_u, pick(rows, us) the
    draft's inverse-CDF tokens of bigram rows at uniforms.  A child maps to
    the first bigram child of b(u) with its token, or is a leaf.  Levels are
    picked in one batch each; creation stops at cap nodes.  Returns tokens
    and parents."""
    kids = [[] for _ in range(len(bt))]
    for i in range(1, len(bt)):
        kids[int(bp[i])].append(i)
    toks, par, big = [int(bt[0])], [-1], [0]
    level = [0]
    while level and len(toks) < cap:
        rows, us, owner = [], [], []
        for u in level:
            if big[u] < 0:
                continue
            U = uniform(u)
            for o in offsets:
                rows.append(big[u])
                us.append((U + o) % 1.0)
                owner.append(u)
        picked = pick(rows, us) if rows else []
        nxt = []
        by_owner = {}
        for u, t in zip(owner, picked):
            lst = by_owner.setdefault(u, [])
            if int(t) not in lst:
                lst.append(int(t))
        for u in level:
            for t in by_owner.get(u, []):
                if len(toks) >= cap:
                    break
                match = [k for k in kids[big[u]] if int(bt[k]) == t]
                toks.append(t)
                par.append(u)
                big.append(match[0] if match else -1)
                nxt.append(len(toks) - 1)
        level = nxt
    return np.array(toks, np.int32), np.array(par, np.int32)


# ---------------------------------------------------------------- decoding loops

@dataclass
class DecodeStats:
    tokens: List[int] = field(default_factory=list)
    steps: int = 0
    accepted: List[int] = field(default_factory=list)   # tree tokens accepted per step
    oracle_nodes: List[int] = field(default_factory=list)
    endorsed: List[int] = field(default_factory=list)
    seconds: float = 0.0


def plain_greedy(backend, P: int, root: int, n_new: int) -> DecodeStats:
    """One-token steps: a single-node tree per step (Sec. 2.1)."""
    st = DecodeStats()
    t0 = time.perf_counter()
    while len(st.tokens) < n_new:
        path, nxt = backend.oracle_step(P, np.array([root], np.int32), np.array([-1], np.int32))
        P += len(path)
        st.tokens.append(nxt)
        st.steps += 1
        root = nxt
    st.seconds = time.perf_counter() - t0
    return st


def staged_greedy(backend, P: int, root: int, n_new: int, succ: np.ndarray) -> DecodeStats:
    """Staged speculation (Sec. 3.2) with greedy acceptance."""
    st = DecodeStats()
    t0 = time.perf_counter()
    while len(st.tokens) < n_new:
        bt, bp = bigram_tree(root, succ)
        top_idx, top_val, lse = backend.draft_top(P, bt, bp, DRAFT_TOP)
        ot, op, n_end = oracle_tree(bt, bp, top_idx, top_val, lse)
        path, nxt = backend.oracle_step(P, ot, op)
        P += len(path)
        emitted = [int(ot[i]) for i in path[1:]] + [int(nxt)]
        st.tokens += emitted
        st.steps += 1
        st.accepted.append(len(path) - 1)
        st.oracle_nodes.append(len(ot))
        st.endorsed.append(n_end)
        root = int(nxt)
    st.tokens = st.tokens[:n_new]
    st.seconds = time.perf_counter() - t0
    return st


def staged_greedy_reuse(backend, P: int, root: int, n_new: int, succ: np.ndarray) -> DecodeStats:
    """Staged speculation (Sec. 3.2) that reuses the draft's work, which the
    paper does not describe: with the draft being the oracle's first layers,
    the oracle verifies the subtree of the bigram tree the draft endorses,
    starting from the draft's residual stream and layer K/V (ssd_tree_reuse,
    ssd_tree_verify_from), so its pass skips the draft's layers for every
    node.  The price: no leaves past the endorsed nodes (the draft did not
    run on them).  Greedy acceptance keeps the emitted sequence the plain
    greedy one."""
    st = DecodeStats()
    t0 = time.perf_counter()
    while len(st.tokens) < n_new:
        bt, bp = bigram_tree(root, succ)
        top_idx, _, _ = backend.draft_top(P, bt, bp, DRAFT_TOP)
        keep, ot, op = endorsed_subtree(bt, bp, top_idx)
        path, nxt = backend.oracle_step_reuse(P, ot, op, keep)
        P += len(path)
        st.tokens += [int(ot[i]) for i in path[1:]] + [int(nxt)]
        st.steps += 1
        st.accepted.append(len(path) - 1)
        st.oracle_nodes.append(len(ot))
        st.endorsed.append(len(ot))
        root = int(nxt)
    st.tokens = st.tokens[:n_new]
    st.seconds = time.perf_counter() - t0
    return st


def plain_sample(backend, P: int, root: int, n_new: int, top_k: int, temperature: float = 1.0,
                 seed0: int = 0) -> DecodeStats:
    """One-token steps with sampling: the next token drawn from the oracle's
    top-k target (Sec. 4: top-k sampling with k = 50, T = 1)."""
    st = DecodeStats()
    t0 = time.perf_counter()
    while len(st.tokens) < n_new:
        path, nxt = backend.oracle_step(P, np.array([root], np.int32), np.array([-1], np.int32),
                                        sample=(top_k, temperature, seed0 + st.steps))
        P += len(path)
        st.tokens.append(nxt)
        st.steps += 1
        root = nxt
    st.seconds = time.perf_counter() - t0
    return st


def staged_sample(backend, P: int, root: int, n_new: int, succ: np.ndarray, top_k: int,
                  temperature: float = 1.0, seed0: int = 0) -> DecodeStats:
    """Staged speculation with sampling: the same trees as staged_greedy (the
    draft's top tokens, chosen rather than drawn), accepted by rejection
    sampling against the oracle's top-k target, so the emitted tokens follow
    that target exactly (Sec. 2.3)."""
    st = DecodeStats()
    t0 = time.perf_counter()
    while len(st.tokens) < n_new:
        bt, bp = bigram_tree(root, succ)
        top_idx, top_val, lse = backend.draft_top(P, bt, bp, DRAFT_TOP)
        ot, op, n_end = oracle_tree(bt, bp, top_idx, top_val, lse)
        path, nxt = backend.oracle_step(P, ot, op, sample=(top_k, temperature, seed0 + st.steps))
        P += len(path)
        st.tokens += [int(ot[i]) for i in path[1:]] + [int(nxt)]
        st.steps += 1
        st.accepted.append(len(path) - 1)
        st.oracle_nodes.append(len(ot))
        st.endorsed.append(n_end)
        root = int(nxt)
    st.tokens = st.tokens[:n_new]
    st.seconds = time.perf_counter() - t0
    return st


def staged_sample_cdf(backend, P: int, root: int, n_new: int, succ: np.ndarray, temperature: float = 1.0,
                      seed0: int = 0) -> DecodeStats:
    """Staged speculation with CDF-first sampling over the whole vocabulary:
    one draft pass over the bigram tree, the oracle tree assembled around
    each node's pre-drawn uniform from the draft's inverse-CDF picks, and the
    walk of SSD_ACCEPT_SAMPLE_CDF; every emitted token is an exact draw from
    the oracle's softmax(logits / temperature)."""
    st = DecodeStats()
    t0 = time.perf_counter()
    while len(st.tokens) < n_new:
        seed = seed0 + st.steps
        bt, bp = bigram_tree(root, succ)
        ot, op = backend.cdf_tree(P, bt, bp, seed, temperature)
        path, nxt = backend.oracle_step(P, ot, op, sample=(0, temperature, seed), cdf=True)
        P += len(path)
        st.tokens += [int(ot[i]) for i in path[1:]] + [int(nxt)]
        st.steps += 1
        st.accepted.append(len(path) - 1)
        st.oracle_nodes.append(len(ot))
        root = int(nxt)
    st.tokens = st.tokens[:n_new]
    st.seconds = time.perf_counter() - t0
    return st


# ---------------------------------------------------------------- GPU backend (libssd)

class GpuBackend:
    """Draft and oracle work through libssd: ssd_tree_verify, ssd_topk,
    ssd_tree_accept (greedy) and ssd_kv_commit.  The draft session binds the
    oracle session's cache (the draft's layers are the oracle's first ones),
    so the oracle's commit serves both."""

    def __init__(self, oracle_session, draft_session, record_gaps: bool = False):
        self.o, self.d = oracle_session, draft_session
        # per oracle step, the top-2 logit gap at the node whose argmax became
        # the next token (to tell precision ties from real divergences)
        self.gaps = [] if record_gaps else None
        self._errors = {id(s): s.error_count() for s in (self.o, self.d)}

    def _check_errors(self, session):
        """A pass that ended early, a float16 overflow or a skipped commit row
        leaves results undefined: stop rather than emit tokens from them."""
        n = session.error_count()
        if n != self._errors[id(session)]:
            raise RuntimeError(f"libssd session error counter grew from {self._errors[id(session)]} to {n}")

    def prefill(self, tokens: np.ndarray, P: int = 0) -> int:
        """Cache `tokens` after P cached ones, in chains of at most max_nodes
        (one verification + commit each); returns the new prefix length."""
        import torch
        tokens = np.asarray(tokens, np.int32)
        step = self.o.max_nodes
        for s in range(0, len(tokens), step):
            chunk = tokens[s:s + step]
            n = len(chunk)
            par = np.arange(-1, n - 1, dtype=np.int32)
            self.o.verify(P, chunk, par)
            path = torch.arange(n, dtype=torch.int32, device=self.o.model.device)
            plen = torch.tensor([n], dtype=torch.int32, device=self.o.model.device)
            self.o.commit(P, path, plen)
            P += n
        self._check_errors(self.o)
        return P

    def draft_top(self, P: int, toks: np.ndarray, par: np.ndarray, k: int):
        lg = self.d.verify(P, toks, par)
        idx, val, lse = self.d.topk(lg, k)
        self._check_errors(self.d)
        return idx.cpu().numpy(), val.cpu().numpy(), lse.cpu().numpy()

    def cdf_tree(self, P: int, bt: np.ndarray, bp: np.ndarray, seed: int, temperature: float):
        """One draft pass over the bigram tree, then the CDF-first oracle
        tree from its logits (ssd_uniform, ssd_cdf_pick)."""
        from . import ssd
        lg = self.d.verify(P, bt, bp)
        n = len(bt)

        def pick(rows, us):
            out = []
            for s0 in range(0, len(rows), 64):
                out += self.d.cdf_pick(lg, rows[s0:s0 + 64], us[s0:s0 + 64], temperature, n).cpu().tolist()
            return out
        ot, op = cdf_first_tree(bt, bp, seed, lambda u: ssd.uniform(seed, 2, u), pick)
        self._check_errors(self.d)
        return ot, op

    def oracle_step(self, P: int, toks: np.ndarray, par: np.ndarray, sample=None, cdf: bool = False):
        """Verify, accept and commit; greedy, or with sample = (top_k,
        temperature, seed) rejection sampling of children chosen by the
        draft (SSD_ACCEPT_SAMPLE_DET), or with cdf=True the CDF-first walk
        (SSD_ACCEPT_SAMPLE_CDF)."""
        from . import ssd
        if sample is None:
            lg, path, plen, nxt = self.o.verify_greedy(P, toks, par)
        else:
            top_k, temperature, seed = sample
            lg = self.o.verify(P, toks, par)
            path, plen, nxt = self.o.accept(toks, par, lg, mode=ssd.SAMPLE_CDF if cdf else ssd.SAMPLE_DET,
                                            temperature=temperature, seed=seed, top_k=top_k)
        self.o.commit(P, path, plen)
        self._check_errors(self.o)
        n = int(plen.item())
        p = path[:n].cpu().numpy().astype(np.int32)
        if self.gaps is not None:
            _, val, _ = self.o.topk(lg, 2)
            v = val[int(p[-1])].cpu().numpy()
            self.gaps.append(float(v[0] - v[1]))
        return p, int(nxt.item())

    def oracle_step_reuse(self, P: int, toks: np.ndarray, par: np.ndarray, draft_rows: np.ndarray):
        """Verify from the draft's last layer on (the draft's last pass ran on
        every node: draft_rows are their slots there), greedy accept, commit."""
        x = self.d.reuse_into(self.o, draft_rows)
        lg, path, plen, nxt = self.o.verify_from(P, toks, par, self.d.model.cfg.n_layer, x, greedy=True)
        self.o.commit(P, path, plen)
        self._check_errors(self.o)
        n = int(plen.item())
        return path[:n].cpu().numpy().astype(np.int32), int(nxt.item())

    def greedy_predictions(self, window_tokens: np.ndarray) -> np.ndarray:
        """The draft's greedy next token at every position of a window fed as
        a chain from an empty cache (teacher forcing)."""
        n = len(window_tokens)
        par = np.arange(-1, n - 1, dtype=np.int32)
        lg = self.d.verify(0, window_tokens, par)
        idx, _, _ = self.d.topk(lg, 1)
        self._check_errors(self.d)
        return idx[:, 0].cpu().numpy()


def build_bigram_gpu(backend: GpuBackend, vocab: int, n_tokens: int = 1 << 15, window: int = 256,
                     seed: int = 4) -> np.ndarray:
    stream = bigram_stream(vocab, n_tokens, seed)
    preds = np.concatenate([backend.greedy_predictions(stream[s:s + window]) for s in range(0, n_tokens, window)])
    return bigram_table(stream, preds, vocab)
