"""ctypes binding of the plain CPU oracle (libssdref.so).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg.  The GPU library never imports it.

All arrays are numpy host arrays.  Parameters and K/V are float32 or uint16
(bfloat16 bit patterns) according to the model's storage type.
"""
from __future__ import annotations

import contextlib
import ctypes as C
import os
import subprocess
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libssdref.so")
_SRC = os.path.join(_HERE, "ssdref.c")

GCC_CMD = ["gcc", "-O3", "-std=c11", "-D_GNU_SOURCE", "-fopenmp", "-fPIC", "-shared",
           "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra", "-o", _SO, _SRC, "-lm"]

F32, BF16 = 0, 1
GREEDY, SAMPLE_WOR, SAMPLE_IID, SAMPLE_DET, SAMPLE_CDF = 0, 1, 2, 3, 4
_ERR = {-1: "invalid argument", -2: "invalid tree", -3: "capacity exceeded"}

LAYER_TENSORS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                 "ln2_g", "ln2_b", "w_fc", "b_fc", "w_pr", "b_pr")


def build() -> str:
    """Compile libssdref.so with gcc (always rebuilds)."""
    subprocess.run(GCC_CMD, check=True)
    return _SO


class OracleError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {_ERR.get(code, code)} ({code})")
        self.code = code


class _Config(C.Structure):
    _fields_ = [("n_layer", C.c_int32), ("d_model", C.c_int32), ("n_head", C.c_int32),
                ("d_mlp", C.c_int32), ("vocab", C.c_int32), ("n_pos", C.c_int32),
                ("dtype", C.c_int32), ("ln_eps", C.c_double)]


_PP = C.POINTER(C.c_void_p)


_I8P, _F32P = C.POINTER(C.c_int8), C.POINTER(C.c_float)
Q8_MATRICES = ("w_qkv", "w_o", "w_fc", "w_pr")


class _Q8(C.Structure):
    _fields_ = [(f"{n}_code", C.POINTER(_I8P)) for n in ("qkv", "o", "fc", "pr")] + \
               [(f"{n}_scale", C.POINTER(_F32P)) for n in ("qkv", "o", "fc", "pr")] + \
               [("head_code", _I8P), ("head_scale", _F32P)]


class _Weights(C.Structure):
    _fields_ = [("wte", C.c_void_p), ("wpe", C.c_void_p), ("lnf_g", C.c_void_p), ("lnf_b", C.c_void_p)] + \
               [(n, _PP) for n in LAYER_TENSORS] + [("q8", C.POINTER(_Q8))]


_lib = None


def _bind(L):
    i32p = C.POINTER(C.c_int32)
    L.ssdref_tree_info.argtypes = [i32p, C.c_int32, i32p, C.POINTER(C.c_uint8)]
    L.ssdref_tree_verify.argtypes = [C.POINTER(_Config), C.POINTER(_Weights), C.c_void_p, C.c_void_p,
                                     C.c_int32, C.c_int32, i32p, i32p, C.c_int32, C.c_void_p, C.c_void_p,
                                     C.c_int32, C.POINTER(C.c_float), C.c_int32]
    L.ssdref_kv_commit.argtypes = [C.POINTER(_Config), C.c_void_p, C.c_void_p, C.c_int32, C.c_int32,
                                   C.c_void_p, C.c_void_p, C.c_int32, i32p, C.c_int32]
    L.ssdref_tree_accept.argtypes = [C.c_int32, i32p, i32p, C.c_int32, C.c_int32, C.POINTER(C.c_float),
                                     C.POINTER(C.c_float), C.c_double, C.c_uint64, i32p, i32p, i32p]
    L.ssdref_tree_accept_k.argtypes = [C.c_int32, i32p, i32p, C.c_int32, C.c_int32, C.POINTER(C.c_float),
                                       C.POINTER(C.c_float), C.c_double, C.c_int32, C.c_uint64, i32p, i32p, i32p]
    L.ssdref_philox4x64_10.argtypes = [C.POINTER(C.c_uint64), C.POINTER(C.c_uint64), C.POINTER(C.c_uint64)]
    L.ssdref_philox4x64_10.restype = None
    L.ssdref_uniform.argtypes = [C.c_uint64, C.c_uint64, C.c_uint64]
    L.ssdref_uniform.restype = C.c_double
    L.ssdref_quantize_q8.argtypes = [C.POINTER(C.c_uint16), C.c_int32, C.c_int32, _I8P, _F32P]
    L.ssdref_cdf_pick.argtypes = [C.POINTER(C.c_float), C.c_int32, C.c_double, C.c_double]
    L.ssdref_cdf_pick.restype = C.c_int32
    L.ssdref_round_bf16.argtypes = [C.c_double]
    L.ssdref_round_bf16.restype = C.c_uint16
    return L


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        _lib = _bind(C.CDLL(_SO))
    return _lib


def build_variant(replacements: Sequence[Tuple[str, str]], out_dir: str) -> str:
    """Compiles a copy of ssdref.c with textual replacements (each must occur
    exactly once) into out_dir; returns the library path.  Used by the power
    checks of the pins, which plant a mistake in a copy and expect the pin to
    fail on it."""
    src = open(_SRC).read()
    for old, new in replacements:
        if src.count(old) != 1:
            raise ValueError(f"replacement target occurs {src.count(old)} times: {old!r}")
        src = src.replace(old, new)
    os.makedirs(out_dir, exist_ok=True)
    c_path = os.path.join(out_dir, "ssdref_variant.c")
    so_path = os.path.join(out_dir, "libssdref_variant.so")
    with open(c_path, "w") as f:
        f.write(src)
    cmd = [a for a in GCC_CMD]
    cmd[cmd.index(_SO)] = so_path
    cmd[cmd.index(_SRC)] = c_path
    subprocess.run(cmd + ["-I", _HERE], check=True)
    return so_path


@contextlib.contextmanager
def variant(so_path: str):
    """Oracle calls inside the block run on another build of ssdref.c."""
    global _lib
    prev = lib()
    _lib = _bind(C.CDLL(so_path))
    try:
        yield
    finally:
        _lib = prev


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a: np.ndarray, t=C.c_void_p):
    return a.ctypes.data_as(t) if t is not C.c_void_p else C.c_void_p(a.ctypes.data)


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(rc, what)


def quantize_q8(w_bits: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """8-bit codes (int8 [rows][cols]) and per-row scales (float32 [rows]) of
    a bfloat16 matrix, by ssdref_quantize_q8 (format in ssdref.h)."""
    w = np.ascontiguousarray(w_bits, dtype=np.uint16)
    rows, cols = w.shape
    codes = np.zeros((rows, cols), dtype=np.int8)
    scales = np.zeros(rows, dtype=np.float32)
    _check(lib().ssdref_quantize_q8(w.ctypes.data_as(C.POINTER(C.c_uint16)), rows, cols,
                                    codes.ctypes.data_as(_I8P), scales.ctypes.data_as(_F32P)), "quantize_q8")
    return codes, scales


class Model:
    """A GPT-2 model for the oracle: config fields plus host parameter arrays.
    q8=True (bfloat16 models): the four weight matrices of every layer and
    the LM head are used as their 8-bit copies (quantize_q8); the embedding
    keeps wte."""

    def __init__(self, cfg, weights: Dict[str, object], q8: bool = False):
        self.cfg = cfg
        self.dtype = F32 if cfg.dtype == "f32" else BF16
        self.np_dtype = np.float32 if self.dtype == F32 else np.uint16
        self._keep = []

        def arr(a):
            a = np.ascontiguousarray(a, dtype=self.np_dtype)
            self._keep.append(a)
            return C.c_void_p(a.ctypes.data)

        self._c = _Config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_pos,
                          self.dtype, float(cfg.ln_eps))
        fields = {"wte": arr(weights["wte"]), "wpe": arr(weights["wpe"]),
                  "lnf_g": arr(weights["lnf_g"]), "lnf_b": arr(weights["lnf_b"])}
        for n in LAYER_TENSORS:
            ptrs = (C.c_void_p * cfg.n_layer)(*[arr(a) for a in weights[n]])
            self._keep.append(ptrs)
            fields[n] = C.cast(ptrs, _PP)
        self.q8 = None
        if q8:
            if self.dtype != BF16:
                raise ValueError("8-bit weights are made from a bfloat16 model")
            self.q8 = {n: [quantize_q8(a) for a in weights[n]] for n in Q8_MATRICES}
            self.q8["head"] = quantize_q8(weights["wte"])
            qf = {}
            for n, short in zip(Q8_MATRICES, ("qkv", "o", "fc", "pr")):
                codes = (_I8P * cfg.n_layer)(*[c.ctypes.data_as(_I8P) for c, _ in self.q8[n]])
                scales = (_F32P * cfg.n_layer)(*[sc.ctypes.data_as(_F32P) for _, sc in self.q8[n]])
                self._keep += [codes, scales]
                qf[f"{short}_code"] = C.cast(codes, C.POINTER(_I8P))
                qf[f"{short}_scale"] = C.cast(scales, C.POINTER(_F32P))
            hc, hs = self.q8["head"]
            self._q8 = _Q8(head_code=hc.ctypes.data_as(_I8P), head_scale=hs.ctypes.data_as(_F32P), **qf)
            fields["q8"] = C.pointer(self._q8)
        self._w = _Weights(**fields)

    def kv(self, rows: int) -> np.ndarray:
        c = self.cfg
        return np.zeros((c.n_layer, c.n_head, rows, c.head_dim), dtype=self.np_dtype)


def tree_info(parent_idx: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
    """(depth[n], anc[n][n] as 0/1 uint8: anc[i][j] = j is i or an ancestor of i)."""
    p = _i32(parent_idx)
    n = len(p)
    depth = np.zeros(n, dtype=np.int32)
    anc = np.zeros((n, n), dtype=np.uint8)
    _check(lib().ssdref_tree_info(_ptr(p, C.POINTER(C.c_int32)), n, _ptr(depth, C.POINTER(C.c_int32)),
                                  _ptr(anc, C.POINTER(C.c_uint8))), "tree_info")
    return depth, anc


def tree_verify(model: Model, k_cache: Optional[np.ndarray], v_cache: Optional[np.ndarray], prefix_len: int,
                tokens: Sequence[int], parent_idx: Sequence[int], k_tree: np.ndarray, v_tree: np.ndarray,
                n_threads: int = 0) -> np.ndarray:
    """Returns logits[n][vocab] (float32); fills k_tree/v_tree rows 0..n-1."""
    cfg = model.cfg
    t, p = _i32(tokens), _i32(parent_idx)
    n = len(t)
    for a in (k_tree, v_tree):
        assert a.dtype == model.np_dtype and a.flags.c_contiguous
    max_nodes = k_tree.shape[2]
    if k_cache is None:
        max_ctx = 0
        kc = vc = C.c_void_p(0)
    else:
        assert k_cache.dtype == model.np_dtype and k_cache.flags.c_contiguous and v_cache.flags.c_contiguous
        max_ctx = k_cache.shape[2]
        kc, vc = _ptr(k_cache), _ptr(v_cache)
    logits = np.empty((n, cfg.vocab), dtype=np.float32)
    rc = lib().ssdref_tree_verify(C.byref(model._c), C.byref(model._w), kc, vc, max_ctx, prefix_len,
                                  _ptr(t, C.POINTER(C.c_int32)), _ptr(p, C.POINTER(C.c_int32)), n,
                                  _ptr(k_tree), _ptr(v_tree), max_nodes, _ptr(logits, C.POINTER(C.c_float)),
                                  n_threads)
    _check(rc, "tree_verify")
    return logits


def kv_commit(model: Model, k_cache: np.ndarray, v_cache: np.ndarray, prefix_len: int,
              k_tree: np.ndarray, v_tree: np.ndarray, path: Sequence[int]) -> None:
    pa = _i32(path)
    rc = lib().ssdref_kv_commit(C.byref(model._c), _ptr(k_cache), _ptr(v_cache), k_cache.shape[2], prefix_len,
                                _ptr(k_tree), _ptr(v_tree), k_tree.shape[2], _ptr(pa, C.POINTER(C.c_int32)),
                                len(pa))
    _check(rc, "kv_commit")


def tree_accept(mode: int, tokens: Sequence[int], parent_idx: Sequence[int], logits: np.ndarray,
                draft_probs: Optional[np.ndarray] = None, temperature: float = 1.0,
                seed: int = 0, top_k: int = 0) -> Tuple[np.ndarray, int]:
    """Returns (path root-first, next_token).  top_k > 0 restricts every
    sampling target to the row's top_k logits; mode SAMPLE_DET takes no
    draft_probs (children chosen, not drawn)."""
    t, p = _i32(tokens), _i32(parent_idx)
    n = len(t)
    lg = np.ascontiguousarray(logits, dtype=np.float32)
    vocab = lg.shape[1]
    dp = None if draft_probs is None else np.ascontiguousarray(draft_probs, dtype=np.float32)
    path = np.zeros(n, dtype=np.int32)
    plen = np.zeros(1, dtype=np.int32)
    nxt = np.zeros(1, dtype=np.int32)
    fp = C.POINTER(C.c_float)
    rc = lib().ssdref_tree_accept_k(mode, _ptr(t, C.POINTER(C.c_int32)), _ptr(p, C.POINTER(C.c_int32)), n, vocab,
                                    None if dp is None else _ptr(dp, fp), _ptr(lg, fp), float(temperature),
                                    int(top_k), C.c_uint64(seed), _ptr(path, C.POINTER(C.c_int32)),
                                    _ptr(plen, C.POINTER(C.c_int32)), _ptr(nxt, C.POINTER(C.c_int32)))
    _check(rc, "tree_accept")
    return path[:plen[0]].copy(), int(nxt[0])


def cdf_pick(row: np.ndarray, temperature: float, U: float) -> int:
    """ssdref_cdf_pick: the token drawn from softmax(row / T) at U by inverse
    CDF in ascending token id."""
    r = np.ascontiguousarray(row, dtype=np.float32)
    x = lib().ssdref_cdf_pick(r.ctypes.data_as(C.POINTER(C.c_float)), len(r), float(temperature), float(U))
    if x < 0:
        raise OracleError(-1, "cdf_pick")
    return int(x)


def philox4x64_10(key: Sequence[int], ctr: Sequence[int]) -> np.ndarray:
    k = np.asarray(key, dtype=np.uint64)
    c = np.asarray(ctr, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    u64p = C.POINTER(C.c_uint64)
    lib().ssdref_philox4x64_10(_ptr(k, u64p), _ptr(c, u64p), _ptr(out, u64p))
    return out


def uniform(seed: int, stream: int, n: int) -> float:
    return float(lib().ssdref_uniform(C.c_uint64(seed), C.c_uint64(stream), C.c_uint64(n)))


def round_bf16(x: float) -> int:
    return int(lib().ssdref_round_bf16(float(x)))
