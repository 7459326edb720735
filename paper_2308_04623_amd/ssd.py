"""ctypes binding of libssd (include/ssd.h): argument marshalling only.

Every step of the verification pass, the accept walk and the commit runs in
the library's HIP kernels; PyTorch supplies device memory and streams.  If
libssd.so has not been built this module raises on first use: there is no
CPU fallback.
"""
from __future__ import annotations

import contextlib
import ctypes as C
import os
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libssd.so")

OK, E_INVALID_ARG, E_INVALID_TREE, E_CAPACITY, E_DEVICE, E_UNSUPPORTED = 0, -1, -2, -3, -4, -5
F32, BF16 = 0, 1
GREEDY, SAMPLE_WOR, SAMPLE_IID, SAMPLE_DET, SAMPLE_CDF = 0, 1, 2, 3, 4
GEMM_AUTO, GEMM_VEC, GEMM_MFMA = 0, 1, 2

LAYER_TENSORS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                 "ln2_g", "ln2_b", "w_fc", "b_fc", "w_pr", "b_pr")

# every function include/ssd.h declares
EXPORTS = ("ssd_model_create", "ssd_model_create_q8", "ssd_model_destroy", "ssd_kv_bytes", "ssd_kv_create", "ssd_kv_destroy",
           "ssd_tree_verify", "ssd_tree_accept", "ssd_kv_commit", "ssd_kv_error_count",
           "ssd_graph_capture_verify", "ssd_graph_launch", "ssd_graph_destroy", "ssd_validate_tree",
           "ssd_tree_prep", "ssd_kv_set_options", "ssd_kv_get_options", "ssd_status_string", "ssd_last_error",
           "ssd_model_prefix_view", "ssd_topk", "ssd_tree_accept_noalloc", "ssd_tree_verify_greedy",
           "ssd_graph_capture_verify_greedy", "ssd_uniform", "ssd_cdf_pick", "ssd_tree_verify_from",
           "ssd_tree_reuse")
# and every function include/ssd_diag.h declares (measurement and diagnostics)
DIAG_EXPORTS = ("ssd_launch_gemm", "ssd_verify_path", "ssd_fused_plan", "ssd_kv_set_trace", "ssd_model_q8_matrix")


class SSDError(RuntimeError):
    def __init__(self, status: int, what: str, detail: str):
        super().__init__(f"{what} failed: status {status} ({detail})")
        self.status = status


class _Config(C.Structure):
    _fields_ = [("n_layer", C.c_int32), ("d_model", C.c_int32), ("n_head", C.c_int32), ("d_mlp", C.c_int32),
                ("vocab", C.c_int32), ("n_pos", C.c_int32), ("dtype", C.c_int32), ("ln_eps", C.c_float)]


_PP = C.POINTER(C.c_void_p)


class _Weights(C.Structure):
    _fields_ = [("wte", C.c_void_p), ("wpe", C.c_void_p), ("lnf_g", C.c_void_p), ("lnf_b", C.c_void_p)] + \
               [(n, _PP) for n in LAYER_TENSORS]


class _Options(C.Structure):
    _fields_ = [("pass_mode", C.c_int32), ("gemm_path", C.c_int32), ("weight_prefetch", C.c_int32)]


class _Tree(C.Structure):
    _fields_ = [("tokens", C.POINTER(C.c_int32)), ("parent_idx", C.POINTER(C.c_int32)), ("n_nodes", C.c_int32),
                ("vocab", C.c_int32), ("mode", C.c_int32), ("temperature", C.c_float), ("top_k", C.c_int32)]


_lib = None


def lib():
    """Load libssd.so (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        # torch first: libssd then binds to the HIP runtime torch has loaded
        # instead of bringing up a second one that sees no device
        import torch  # noqa: F401
        L = C.CDLL(LIB_PATH)
        i32p, vp = C.POINTER(C.c_int32), C.c_void_p
        sig = {
            "ssd_model_create": [C.POINTER(_Config), C.POINTER(_Weights), vp, C.POINTER(vp)],
            "ssd_model_create_q8": [C.POINTER(_Config), C.POINTER(_Weights), vp, C.POINTER(vp)],
            "ssd_model_q8_matrix": [vp, C.c_int32, C.c_int32, vp, vp],
            "ssd_model_destroy": [vp],
            "ssd_kv_bytes": [C.POINTER(_Config), C.c_int32, C.c_int32, C.POINTER(C.c_size_t),
                             C.POINTER(C.c_size_t)],
            "ssd_kv_create": [vp, C.c_int32, C.c_int32, vp, vp, vp, vp, C.POINTER(vp)],
            "ssd_kv_destroy": [vp],
            "ssd_tree_verify": [vp, vp, C.c_int32, i32p, i32p, C.c_int32, vp, vp],
            "ssd_tree_verify_greedy": [vp, vp, C.c_int32, i32p, i32p, C.c_int32, vp, vp, vp, vp, vp],
            "ssd_graph_capture_verify_greedy": [vp, vp, C.c_int32, i32p, i32p, C.c_int32, vp, vp, vp, vp, vp,
                                                C.POINTER(vp)],
            "ssd_tree_accept": [vp, C.POINTER(_Tree), vp, vp, C.c_uint64, vp, vp, vp, vp],
            "ssd_tree_accept_noalloc": [C.POINTER(_Tree), vp, vp, C.c_uint64, vp, vp, vp, vp],
            "ssd_kv_commit": [vp, C.c_int32, vp, vp, vp],
            "ssd_kv_error_count": [vp, vp, C.POINTER(C.c_uint32)],
            "ssd_graph_capture_verify": [vp, vp, C.c_int32, i32p, i32p, C.c_int32, vp, vp, C.POINTER(vp)],
            "ssd_graph_launch": [vp, vp],
            "ssd_graph_destroy": [vp],
            "ssd_validate_tree": [i32p, i32p, C.c_int32, C.c_int32, i32p],
            "ssd_tree_prep": [i32p, C.c_int32, i32p, C.POINTER(C.c_uint64)],
            "ssd_kv_set_options": [vp, C.POINTER(_Options)],
            "ssd_kv_get_options": [vp, C.POINTER(_Options)],
            "ssd_verify_path": [vp, vp, C.c_int32, C.POINTER(C.c_int32)],
            "ssd_fused_plan": [C.c_int32] * 5 + [vp, vp, vp],
            "ssd_kv_set_trace": [vp, vp],
            "ssd_launch_gemm": [vp, vp, C.c_int32, C.c_int32, C.c_int32, vp],
            "ssd_model_prefix_view": [vp, C.c_int32, C.POINTER(vp)],
            "ssd_topk": [vp, vp, C.c_int32, C.c_int32, vp, vp, vp, vp],
            "ssd_status_string": [C.c_int],
            "ssd_uniform": [C.c_uint64, C.c_uint64, C.c_uint64],
            "ssd_tree_verify_from": [vp, vp, C.c_int32, i32p, i32p, C.c_int32, C.c_int32, vp, vp, vp, vp, vp, vp],
            "ssd_tree_reuse": [vp, vp, C.c_int32, vp, vp, vp],
            "ssd_cdf_pick": [vp, vp, C.c_int32, C.c_int32, C.c_float, C.c_int32, vp, vp, vp, vp],
            "ssd_last_error": [],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = C.c_int
        for name in ("ssd_model_destroy", "ssd_kv_destroy", "ssd_graph_destroy"):
            getattr(L, name).restype = None
        L.ssd_status_string.restype = C.c_char_p
        L.ssd_uniform.restype = C.c_double
        L.ssd_last_error.restype = C.c_char_p
        _lib = L
    return _lib


def _check(status: int, what: str):
    if status != OK:
        raise SSDError(status, what, lib().ssd_last_error().decode())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.int32)


def _p32(a: np.ndarray):
    return a.ctypes.data_as(C.POINTER(C.c_int32))


# ---------------------------------------------------------------- host-only helpers

def validate_tree(tokens, parent_idx, vocab: int) -> int:
    t, p = _i32(tokens), _i32(parent_idx)
    md = C.c_int32(0)
    _check(lib().ssd_validate_tree(_p32(t), _p32(p), len(t), vocab, C.byref(md)), "ssd_validate_tree")
    return md.value


def tree_prep(parent_idx) -> Tuple[np.ndarray, np.ndarray]:
    """(depth[n], anc[n][ceil(n/64)] uint64 bitmask) as the library computes them."""
    p = _i32(parent_idx)
    n = len(p)
    depth = np.zeros(n, dtype=np.int32)
    anc = np.zeros((n, (n + 63) // 64), dtype=np.uint64)
    _check(lib().ssd_tree_prep(_p32(p), n, _p32(depth), anc.ctypes.data_as(C.POINTER(C.c_uint64))),
           "ssd_tree_prep")
    return depth, anc


PASS_AUTO, PASS_KERNELS, PASS_FUSED = 0, 1, 2


def fused_plan(n_head: int, d_model: int, d_mlp: int, vocab: int, n_tiles: int):
    """The persistent pass's work split (host-only): (tab [256][32], xh [16], xf [16])."""
    tab = np.zeros((256, 32), np.int32)
    xh = np.zeros(16, np.int32)
    xf = np.zeros(16, np.int32)
    _check(lib().ssd_fused_plan(n_head, d_model, d_mlp, vocab, n_tiles, tab.ctypes.data, xh.ctypes.data,
                                xf.ctypes.data), "ssd_fused_plan")
    return tab, xh, xf


def accept_noalloc(tokens, parent_idx, logits, out, mode: int = GREEDY, draft_probs=None,
                   temperature: float = 1.0, seed: int = 0, top_k: int = 0, stream=None):
    """ssd_tree_accept_noalloc: the accept walk without a session or any
    device allocation (n <= 256, vocab <= 65536).  out = (path[n],
    path_len[1], next_token[1]) device int32 tensors the caller allocated."""
    t, p = _i32(tokens), _i32(parent_idx)
    path, plen, nxt = out
    tree = _Tree(_p32(t), _p32(p), len(t), logits.shape[1], mode, float(temperature), int(top_k))
    dp = C.c_void_p(draft_probs.data_ptr()) if draft_probs is not None else C.c_void_p(0)
    _check(lib().ssd_tree_accept_noalloc(C.byref(tree), dp, C.c_void_p(logits.data_ptr()), C.c_uint64(seed),
                                         C.c_void_p(path.data_ptr()), C.c_void_p(plen.data_ptr()),
                                         C.c_void_p(nxt.data_ptr()), _stream(stream)), "ssd_tree_accept_noalloc")
    return path, plen, nxt


def uniform(seed: int, stream: int, counter: int) -> float:
    """ssd_uniform: the accept walk's uniform for (seed, stream, counter)."""
    return float(lib().ssd_uniform(seed, stream, counter))


def kv_bytes(cfg, max_ctx: int, max_nodes: int) -> Tuple[int, int]:
    c = _config(cfg)
    a, b = C.c_size_t(0), C.c_size_t(0)
    _check(lib().ssd_kv_bytes(C.byref(c), max_ctx, max_nodes, C.byref(a), C.byref(b)), "ssd_kv_bytes")
    return a.value, b.value


def _config(cfg) -> _Config:
    return _Config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_pos,
                   F32 if cfg.dtype == "f32" else BF16, float(cfg.ln_eps))


# ---------------------------------------------------------------- device objects

def _torch():
    import torch
    return torch


def _stream(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def storage_torch_dtype(cfg):
    torch = _torch()
    return torch.float32 if cfg.dtype == "f32" else torch.bfloat16


def to_device(a: np.ndarray, cfg, device="cuda"):
    """Host parameter/K-V array (float32, or uint16 bf16 bits) -> device tensor."""
    torch = _torch()
    if cfg.dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16)).to(device)
    return t.view(torch.bfloat16)


def to_host_bits(t) -> np.ndarray:
    """Device tensor -> host array in the oracle's representation."""
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


class Model:
    """A GPT-2 model resident on the GPU.  `weights` is the dict produced by
    workloads.make_weights (host arrays); they are uploaded once.  q8=True
    (bfloat16 models): ssd_model_create_q8, 8-bit weight matrices and LM
    head."""

    def __init__(self, cfg, weights: Dict[str, object], device="cuda", stream=None, q8: bool = False):
        self.cfg = cfg
        self.q8 = q8
        self.device = device
        self.tensors = {}
        ptr = lambda t: C.c_void_p(t.data_ptr())
        for k in ("wte", "wpe", "lnf_g", "lnf_b"):
            self.tensors[k] = to_device(weights[k], cfg, device)
        fields = {k: ptr(self.tensors[k]) for k in ("wte", "wpe", "lnf_g", "lnf_b")}
        self._arrays = []
        for n in LAYER_TENSORS:
            ts = [to_device(a, cfg, device) for a in weights[n]]
            self.tensors[n] = ts
            arr = (C.c_void_p * cfg.n_layer)(*[t.data_ptr() for t in ts])
            self._arrays.append(arr)
            fields[n] = C.cast(arr, _PP)
        self._cfg = _config(cfg)
        self._w = _Weights(**fields)
        h = C.c_void_p()
        create = lib().ssd_model_create_q8 if q8 else lib().ssd_model_create
        _check(create(C.byref(self._cfg), C.byref(self._w), _stream(stream), C.byref(h)),
               "ssd_model_create_q8" if q8 else "ssd_model_create")
        self.handle = h

    def q8_matrix(self, which: int, layer: int = 0):
        """(codes int8 [rows][cols], scales float32 [rows]) of one 8-bit
        matrix: which 0 W_qkv, 1 W_o, 2 W_fc, 3 W_pr, 4 the LM head."""
        c = self.cfg
        ok = 0 <= which <= 4   # (other ids go to the library, which refuses them)
        rows = [3 * c.d_model, c.d_model, c.d_mlp, c.d_model, c.vocab][which] if ok else 1
        cols = [c.d_model, c.d_model, c.d_model, c.d_mlp, c.d_model][which] if ok else 1
        codes = np.zeros((rows, cols), dtype=np.int8)
        scales = np.zeros(rows, dtype=np.float32)
        _check(lib().ssd_model_q8_matrix(self.handle, which, layer, C.c_void_p(codes.ctypes.data),
                                         C.c_void_p(scales.ctypes.data)), "ssd_model_q8_matrix")
        return codes, scales

    def prefix_view(self, n_layer: int) -> "ModelView":
        """Draft view: the first n_layer blocks with this model's final
        LayerNorm and tied head, sharing its device memory."""
        return ModelView(self, n_layer)

    def close(self):
        if getattr(self, "handle", None):
            lib().ssd_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class ModelView:
    """ssd_model_prefix_view of a Model (keeps the parent alive)."""

    def __init__(self, parent: Model, n_layer: int):
        self.parent = parent
        self.cfg = parent.cfg.with_(n_layer=n_layer)
        self.device = parent.device
        h = C.c_void_p()
        _check(lib().ssd_model_prefix_view(parent.handle, n_layer, C.byref(h)), "ssd_model_prefix_view")
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            lib().ssd_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Graph:
    def __init__(self, handle, keep):
        self.handle = handle
        self._keep = keep

    def launch(self, stream=None):
        _check(lib().ssd_graph_launch(self.handle, _stream(stream)), "ssd_graph_launch")

    def close(self):
        if getattr(self, "handle", None):
            lib().ssd_graph_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Session:
    """One decoding session: caller-owned K/V cache and tree scratch (torch
    tensors [L][H][rows][head_dim]) plus the library's workspaces."""

    def __init__(self, model: Model, max_ctx: int, max_nodes: int, k_cache=None, v_cache=None):
        torch = _torch()
        cfg = model.cfg
        self.model, self.max_ctx, self.max_nodes = model, max_ctx, max_nodes
        dt = storage_torch_dtype(cfg)
        shape = lambda r: (cfg.n_layer, cfg.n_head, r, cfg.head_dim)
        self.k_cache = k_cache if k_cache is not None else torch.zeros(shape(max_ctx), dtype=dt, device=model.device)
        self.v_cache = v_cache if v_cache is not None else torch.zeros(shape(max_ctx), dtype=dt, device=model.device)
        self.k_tree = torch.zeros(shape(max_nodes), dtype=dt, device=model.device)
        self.v_tree = torch.zeros(shape(max_nodes), dtype=dt, device=model.device)
        h = C.c_void_p()
        _check(lib().ssd_kv_create(model.handle, max_ctx, max_nodes, C.c_void_p(self.k_cache.data_ptr()),
                                   C.c_void_p(self.v_cache.data_ptr()), C.c_void_p(self.k_tree.data_ptr()),
                                   C.c_void_p(self.v_tree.data_ptr()), C.byref(h)), "ssd_kv_create")
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            lib().ssd_kv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def verify(self, prefix_len: int, tokens, parent_idx, logits=None, stream=None):
        torch = _torch()
        t, p = _i32(tokens), _i32(parent_idx)
        n = len(t)
        if logits is None:
            logits = torch.empty((n, self.model.cfg.vocab), dtype=torch.float32, device=self.model.device)
        _check(lib().ssd_tree_verify(self.model.handle, self.handle, prefix_len, _p32(t), _p32(p), n,
                                     C.c_void_p(logits.data_ptr()), _stream(stream)), "ssd_tree_verify")
        return logits

    def _accept_outs(self, n, out):
        torch = _torch()
        if out is not None:
            return out
        return (torch.zeros(n, dtype=torch.int32, device=self.model.device),
                torch.zeros(1, dtype=torch.int32, device=self.model.device),
                torch.zeros(1, dtype=torch.int32, device=self.model.device))

    def verify_greedy(self, prefix_len: int, tokens, parent_idx, logits=None, out=None, stream=None):
        """ssd_tree_verify_greedy: (logits, path, path_len, next_token)."""
        torch = _torch()
        t, p = _i32(tokens), _i32(parent_idx)
        n = len(t)
        if logits is None:
            logits = torch.empty((n, self.model.cfg.vocab), dtype=torch.float32, device=self.model.device)
        path, plen, nxt = self._accept_outs(n, out)
        _check(lib().ssd_tree_verify_greedy(self.model.handle, self.handle, prefix_len, _p32(t), _p32(p), n,
                                            C.c_void_p(logits.data_ptr()), C.c_void_p(path.data_ptr()),
                                            C.c_void_p(plen.data_ptr()), C.c_void_p(nxt.data_ptr()),
                                            _stream(stream)), "ssd_tree_verify_greedy")
        return logits, path, plen, nxt

    def capture_verify_greedy(self, prefix_len: int, tokens, parent_idx, logits, out, stream=None) -> Graph:
        """ssd_graph_capture_verify_greedy into logits and out = (path, path_len, next_token)."""
        t, p = _i32(tokens), _i32(parent_idx)
        path, plen, nxt = out
        h = C.c_void_p()
        _check(lib().ssd_graph_capture_verify_greedy(self.model.handle, self.handle, prefix_len, _p32(t), _p32(p),
                                                     len(t), C.c_void_p(logits.data_ptr()),
                                                     C.c_void_p(path.data_ptr()), C.c_void_p(plen.data_ptr()),
                                                     C.c_void_p(nxt.data_ptr()), _stream(stream), C.byref(h)),
               "ssd_graph_capture_verify_greedy")
        return Graph(h, (t, p, logits, out))

    def capture_verify(self, prefix_len: int, tokens, parent_idx, logits, stream=None) -> Graph:
        t, p = _i32(tokens), _i32(parent_idx)
        h = C.c_void_p()
        _check(lib().ssd_graph_capture_verify(self.model.handle, self.handle, prefix_len, _p32(t), _p32(p), len(t),
                                              C.c_void_p(logits.data_ptr()), _stream(stream), C.byref(h)),
               "ssd_graph_capture_verify")
        return Graph(h, (t, p, logits))

    def accept(self, tokens, parent_idx, logits, mode: int = GREEDY, draft_probs=None, temperature: float = 1.0,
               seed: int = 0, out=None, stream=None, top_k: int = 0):
        """Returns device int32 tensors (path[n], path_len[1], next_token[1])."""
        torch = _torch()
        t, p = _i32(tokens), _i32(parent_idx)
        n = len(t)
        if out is None:
            out = (torch.zeros(n, dtype=torch.int32, device=self.model.device),
                   torch.zeros(1, dtype=torch.int32, device=self.model.device),
                   torch.zeros(1, dtype=torch.int32, device=self.model.device))
        path, plen, nxt = out
        tree = _Tree(_p32(t), _p32(p), n, logits.shape[1], mode, float(temperature), int(top_k))
        dp = C.c_void_p(draft_probs.data_ptr()) if draft_probs is not None else C.c_void_p(0)
        _check(lib().ssd_tree_accept(self.handle, C.byref(tree), dp, C.c_void_p(logits.data_ptr()), C.c_uint64(seed),
                                     C.c_void_p(path.data_ptr()), C.c_void_p(plen.data_ptr()),
                                     C.c_void_p(nxt.data_ptr()), _stream(stream)), "ssd_tree_accept")
        return path, plen, nxt

    def commit(self, prefix_len: int, path, path_len, stream=None):
        _check(lib().ssd_kv_commit(self.handle, prefix_len, C.c_void_p(path.data_ptr()),
                                   C.c_void_p(path_len.data_ptr()), _stream(stream)), "ssd_kv_commit")

    def launch_gemm(self, which: int, layer: int, n_nodes: int, stream=None):
        """One weight GEMM of the pass on its own (measurement only)."""
        _check(lib().ssd_launch_gemm(self.model.handle, self.handle, which, layer, n_nodes, _stream(stream)),
               "ssd_launch_gemm")

    def topk(self, logits, k: int, n_rows: Optional[int] = None, stream=None):
        """Per-row top-k of logits[n][vocab] on the device: (idx int32 [n][k],
        val float32 [n][k], lse float32 [n])."""
        torch = _torch()
        n = logits.shape[0] if n_rows is None else n_rows
        idx = torch.empty((n, k), dtype=torch.int32, device=self.model.device)
        val = torch.empty((n, k), dtype=torch.float32, device=self.model.device)
        lse = torch.empty((n,), dtype=torch.float32, device=self.model.device)
        _check(lib().ssd_topk(self.handle, C.c_void_p(logits.data_ptr()), n, k, C.c_void_p(idx.data_ptr()),
                              C.c_void_p(val.data_ptr()), C.c_void_p(lse.data_ptr()), _stream(stream)), "ssd_topk")
        return idx, val, lse

    def verify_from(self, prefix_len: int, tokens, parent_idx, start_layer: int, x_in, logits=None, greedy=False,
                    stream=None):
        """ssd_tree_verify_from: logits, or with greedy=True (logits, path,
        path_len, next_token)."""
        torch = _torch()
        t, p = _i32(tokens), _i32(parent_idx)
        n = len(t)
        if logits is None:
            logits = torch.empty((n, self.model.cfg.vocab), dtype=torch.float32, device=self.model.device)
        outs = self._accept_outs(n, None) if greedy else None
        gp = [C.c_void_p(o.data_ptr()) for o in outs] if greedy else [C.c_void_p(0)] * 3
        _check(lib().ssd_tree_verify_from(self.model.handle, self.handle, prefix_len, _p32(t), _p32(p), n,
                                          start_layer, C.c_void_p(x_in.data_ptr() if x_in is not None else 0),
                                          C.c_void_p(logits.data_ptr()), *gp, _stream(stream)),
               "ssd_tree_verify_from")
        return (logits,) + tuple(outs) if greedy else logits

    def reuse_into(self, dst: "Session", src_rows, stream=None):
        """ssd_tree_reuse from this (draft) session into dst: returns the
        residual rows x [n][d_model] (device fp32) for dst.verify_from."""
        torch = _torch()
        r = _i32(src_rows)
        x = torch.empty((len(r), self.model.cfg.d_model), dtype=torch.float32, device=self.model.device)
        _check(lib().ssd_tree_reuse(self.handle, dst.handle, len(r), C.c_void_p(r.ctypes.data),
                                    C.c_void_p(x.data_ptr()), _stream(stream)), "ssd_tree_reuse")
        return x

    def cdf_pick(self, logits, rows, uniforms, temperature: float = 1.0, n_rows: Optional[int] = None,
                 stream=None):
        """ssd_cdf_pick: device int32 tokens, query q drawn from
        softmax(logits[rows[q]] / temperature) at uniforms[q] by inverse CDF
        (ascending token id)."""
        torch = _torch()
        r = _i32(rows)
        u = np.ascontiguousarray(uniforms, dtype=np.float64)
        n = logits.shape[0] if n_rows is None else n_rows
        out = torch.empty(len(r), dtype=torch.int32, device=self.model.device)
        _check(lib().ssd_cdf_pick(self.handle, C.c_void_p(logits.data_ptr()), n, int(logits.shape[1]),
                                  float(temperature), len(r),
                                  C.c_void_p(r.ctypes.data), C.c_void_p(u.ctypes.data), C.c_void_p(out.data_ptr()),
                                  _stream(stream)), "ssd_cdf_pick")
        return out

    def set_trace(self, buf=None):
        """Stage timestamps of the persistent pass into buf (device uint64/int64
        tensor of 256 * (n_layer + 1) * 24 words), or None to stop."""
        _check(lib().ssd_kv_set_trace(self.handle, C.c_void_p(buf.data_ptr() if buf is not None else 0)),
               "ssd_kv_set_trace")

    def verify_path(self, n: int) -> int:
        """PASS_KERNELS or PASS_FUSED: how a pass of n nodes would run now."""
        v = C.c_int32(0)
        _check(lib().ssd_verify_path(self.model.handle, self.handle, n, C.byref(v)), "ssd_verify_path")
        return v.value

    def get_options(self) -> Dict[str, int]:
        o = _Options()
        _check(lib().ssd_kv_get_options(self.handle, C.byref(o)), "ssd_kv_get_options")
        return {"pass_mode": o.pass_mode, "gemm_path": o.gemm_path, "weight_prefetch": o.weight_prefetch}

    def set_options(self, pass_mode: Optional[int] = None, gemm_path: Optional[int] = None,
                    weight_prefetch: Optional[int] = None):
        """This session's switches (ssd_kv_set_options); None keeps a value.
        pass_mode: PASS_AUTO / PASS_KERNELS / PASS_FUSED; gemm_path: GEMM_AUTO
        / GEMM_VEC / GEMM_MFMA; weight_prefetch: 0 or 1."""
        cur = self.get_options()
        for k, v in (("pass_mode", pass_mode), ("gemm_path", gemm_path), ("weight_prefetch", weight_prefetch)):
            if v is not None:
                cur[k] = int(v)
        o = _Options(cur["pass_mode"], cur["gemm_path"], cur["weight_prefetch"])
        _check(lib().ssd_kv_set_options(self.handle, C.byref(o)), "ssd_kv_set_options")

    @contextlib.contextmanager
    def options(self, **kw):
        """Switches set for the block, restored afterwards."""
        prev = self.get_options()
        self.set_options(**kw)
        try:
            yield self
        finally:
            self.set_options(**prev)

    def error_count(self, stream=None) -> int:
        c = C.c_uint32(0)
        _check(lib().ssd_kv_error_count(self.handle, _stream(stream), C.byref(c)), "ssd_kv_error_count")
        return c.value
