"""Seeded synthetic inputs: GPT-2-shaped random models, prefixes, token trees.

This module generates inputs only.  It holds none of the verification,
acceptance or commit arithmetic, and both the GPU library's tests and the CPU
oracle's tests draw their inputs from it.

The paper's experiments use trained GPT-2 weights and HumanEval prompts
(Sec. 4); neither is available, so random-init models of the same shape and
uniform random token streams stand in for them.

Parameter init: every matrix and embedding is N(0, 0.02) drawn in float32,
LayerNorm gain 1, LayerNorm bias 0, linear biases 0 (GPT-2's init without the
residual rescaling).  ``perturb_affine=True`` instead draws biases and LN
biases from N(0, 0.02) and LN gains from 1 + N(0, 0.02), so that parity tests
exercise every affine term.  bfloat16 models round the float32 draw to
nearest-even and store the bit patterns as uint16.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Sequence, Tuple

import numpy as np

LAYER_TENSORS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                 "ln2_g", "ln2_b", "w_fc", "b_fc", "w_pr", "b_pr")


@dataclasses.dataclass(frozen=True)
class GPT2Config:
    n_layer: int
    d_model: int
    n_head: int
    d_mlp: int
    vocab: int
    n_pos: int
    dtype: str = "f32"          # storage type of parameters and K/V: "f32" or "bf16"
    ln_eps: float = 1e-5

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_head

    def with_(self, **kw) -> "GPT2Config":
        return dataclasses.replace(self, **kw)


# 2-layer toy decoder: parity on every code path in seconds.
TINY = GPT2Config(n_layer=2, d_model=128, n_head=4, d_mlp=512, vocab=512, n_pos=256, dtype="f32")
# GPT-2-Large shape (36 x 1280, 20 heads of 64, MLP 5120, vocab 50257).  The
# learned-position table is extended past 1024 rows so that prefixes of 1024
# (and 2048) tokens plus a tree still have positions.
GPT2L = GPT2Config(n_layer=36, d_model=1280, n_head=20, d_mlp=5120, vocab=50257, n_pos=1024 + 256,
                   dtype="bf16")
GPT2L_LONG = GPT2L.with_(n_pos=2048 + 256)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest-even); returns uint16 bit patterns.
    (NaN inputs are not expected.)"""
    u = np.array(a, dtype=np.float32, copy=True).view(np.uint32)
    u += np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (u >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _tensor_shapes(cfg: GPT2Config) -> List[Tuple[str, int, Tuple[int, ...], str]]:
    """(name, layer, shape, kind) in the fixed enumeration order that fixes seeds."""
    d, m = cfg.d_model, cfg.d_mlp
    out = [("wte", -1, (cfg.vocab, d), "mat"), ("wpe", -1, (cfg.n_pos, d), "mat"),
           ("lnf_g", -1, (d,), "gain"), ("lnf_b", -1, (d,), "bias")]
    per = {"ln1_g": ((d,), "gain"), "ln1_b": ((d,), "bias"), "w_qkv": ((3 * d, d), "mat"),
           "b_qkv": ((3 * d,), "bias"), "w_o": ((d, d), "mat"), "b_o": ((d,), "bias"),
           "ln2_g": ((d,), "gain"), "ln2_b": ((d,), "bias"), "w_fc": ((m, d), "mat"),
           "b_fc": ((m,), "bias"), "w_pr": ((d, m), "mat"), "b_pr": ((d,), "bias")}
    for l in range(cfg.n_layer):
        for name in LAYER_TENSORS:
            shape, kind = per[name]
            out.append((name, l, shape, kind))
    return out


def make_weights(cfg: GPT2Config, seed: int = 0, perturb_affine: bool = False) -> Dict[str, object]:
    """Random GPT-2 parameters.  Matrices are [out][in] row-major.

    Returns a dict: 'wte', 'wpe', 'lnf_g', 'lnf_b' -> arrays; each name in
    LAYER_TENSORS -> list of n_layer arrays.  Arrays are float32 ("f32") or
    uint16 bfloat16 bit patterns ("bf16").  Tensor t uses
    numpy.random.default_rng([seed, t]) with t its index in the fixed
    enumeration (wte, wpe, lnf_g, lnf_b, then per layer the LAYER_TENSORS order).
    """
    out: Dict[str, object] = {name: [None] * cfg.n_layer for name in LAYER_TENSORS}

    def one(item):
        tid, (name, layer, shape, kind) = item
        if kind == "mat" or perturb_affine:
            g = np.random.default_rng([seed, tid])
            a = g.standard_normal(shape, dtype=np.float32)
            a *= np.float32(0.02)
            if kind == "gain":
                a += np.float32(1.0)
        elif kind == "gain":
            a = np.ones(shape, dtype=np.float32)
        else:
            a = np.zeros(shape, dtype=np.float32)
        if cfg.dtype == "bf16":
            a = f32_to_bf16_bits(a)
        return name, layer, a

    items = list(enumerate(_tensor_shapes(cfg)))
    workers = max(1, min(16, os.cpu_count() or 1))
    with ThreadPoolExecutor(workers) as ex:   # numpy's generators release the GIL
        for name, layer, a in ex.map(one, items):
            if layer < 0:
                out[name] = a
            else:
                out[name][layer] = a
    return out


def storage_dtype(cfg: GPT2Config):
    return np.float32 if cfg.dtype == "f32" else np.uint16


def kv_shape(cfg: GPT2Config, rows: int) -> Tuple[int, int, int, int]:
    """[n_layer][n_head][rows][head_dim], used for both the cache and the tree scratch."""
    return (cfg.n_layer, cfg.n_head, rows, cfg.head_dim)


def random_kv_cache(cfg: GPT2Config, max_ctx: int, prefix_len: int, seed: int,
                    sigma: float = 0.7) -> Tuple[np.ndarray, np.ndarray]:
    """Synthetic prefix cache: rows < prefix_len ~ N(0, sigma), the rest zero.

    sigma ~ 0.7 matches K/V of the random-init model (unit-variance LayerNorm
    output times N(0, 0.02) weights over 1280 inputs).  Stands in for a
    prefill when only the verification pass is under test."""
    k = np.zeros(kv_shape(cfg, max_ctx), dtype=np.float32)
    v = np.zeros_like(k)
    g = np.random.default_rng([seed, 101])
    k[:, :, :prefix_len, :] = g.standard_normal(k[:, :, :prefix_len, :].shape, dtype=np.float32) * sigma
    v[:, :, :prefix_len, :] = g.standard_normal(v[:, :, :prefix_len, :].shape, dtype=np.float32) * sigma
    if cfg.dtype == "bf16":
        return f32_to_bf16_bits(k), f32_to_bf16_bits(v)
    return k, v


def empty_kv(cfg: GPT2Config, rows: int) -> np.ndarray:
    return np.zeros(kv_shape(cfg, rows), dtype=storage_dtype(cfg))


# ----------------------------------------------------------------------------
# token trees: tokens[n] and parent_idx[n] with parent_idx[0] = -1 and
# parent_idx[i] < i (topological order)
# ----------------------------------------------------------------------------

def chain_tree(n: int) -> np.ndarray:
    return np.arange(-1, n - 1, dtype=np.int32)


def complete_binary_tree(n: int) -> np.ndarray:
    p = (np.arange(n, dtype=np.int32) - 1) // 2
    p[0] = -1
    return p.astype(np.int32)


def branching_tree(branching: Sequence[int], n_nodes: int) -> np.ndarray:
    """Breadth-first tree where every node at depth t gets branching[t] children
    (the last entry repeats), truncated at n_nodes."""
    parents = [-1]
    frontier = [0]
    depth = 0
    while len(parents) < n_nodes and frontier:
        b = branching[min(depth, len(branching) - 1)]
        nxt = []
        for u in frontier:
            for _ in range(b):
                if len(parents) >= n_nodes:
                    break
                parents.append(u)
                nxt.append(len(parents) - 1)
        frontier = nxt
        depth += 1
    return np.asarray(parents, dtype=np.int32)


def best_first_tree(n_nodes: int, seed: int = 3, fanout: int = 8, vocab: int = 50257
                    ) -> Tuple[np.ndarray, np.ndarray]:
    """Nested best-first tree: every node gets `fanout` distinct uniform
    candidate tokens with scores from a sorted Dirichlet(1,...,1); the frontier
    candidate with the highest cumulative log-score is expanded next (ties to
    the lower creation index).  Tree(n) is the first n nodes of one expansion.
    Returns (tokens[1:] of the chosen children..., parents); node 0's token is
    left to the caller (tokens[0] = -1 placeholder)."""
    tokens = [-1]
    parents = [-1]
    logscore = [0.0]
    cand: List[Tuple[float, int, int, int]] = []   # (-score, creation, parent, token)
    created = 0

    def add_children(u: int):
        nonlocal created
        g = np.random.default_rng([seed, u])
        toks = g.choice(vocab, size=fanout, replace=False)
        sc = np.sort(g.dirichlet(np.ones(fanout)))[::-1]
        for t, s in zip(toks, sc):
            cand.append((-(logscore[u] + float(np.log(s))), created, u, int(t)))
            created += 1

    add_children(0)
    while len(tokens) < n_nodes:
        cand.sort()
        negs, _, u, t = cand.pop(0)
        tokens.append(t)
        parents.append(u)
        logscore.append(-negs)
        add_children(len(tokens) - 1)
    return np.asarray(tokens, dtype=np.int32), np.asarray(parents, dtype=np.int32)


def tree_tokens(parents: np.ndarray, vocab: int, seed: int) -> np.ndarray:
    """Uniform node tokens (root included) from default_rng(seed)."""
    return np.random.default_rng(seed).integers(0, vocab, size=len(parents)).astype(np.int32)


def prefix_tokens(n: int, vocab: int, seed: int = 1) -> np.ndarray:
    return np.random.default_rng(seed).integers(0, vocab, size=n).astype(np.int32)
