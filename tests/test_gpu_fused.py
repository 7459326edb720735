"""GPU parity of the persistent single-launch pass (bf16 models with head
dimension 64, at most 64 tree nodes) against the CPU oracle, through the C ABI.

The model is a small GPT-2-shaped decoder (3 layers, d 256, 4 heads of 64,
MLP 1024, vocab 2000) with perturbed affine terms, so the oracle runs in
seconds while the pass exercises every stage: XCDs without heads, ragged
node tiles (1, 15, 17, 33, 48, 64 nodes) and prefixes of 0, 64 and 200 rows
(200 is not a multiple of the 128-row attention chunk).

Bars: logits and tree K/V within 2e-2 max-abs of the oracle; a node's logits
bitwise independent of the rest of the tree, its slot and the tile count;
bitwise determinism and graph replay; greedy accept bit-exact on the GPU's
own logits."""
import numpy as np
import pytest

import oracle
from paper_2308_04623_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = 2e-2
SMALL = W.GPT2Config(n_layer=3, d_model=256, n_head=4, d_mlp=1024, vocab=2000, n_pos=512, dtype="bf16")


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


@pytest.fixture(scope="module")
def ssd(torch):
    from paper_2308_04623_amd import ssd as s
    s.lib()
    yield s


class Small:
    def __init__(self, ssd, cfg=SMALL, max_ctx=320, max_nodes=64, P=200):
        self.cfg = cfg
        self.w = W.make_weights(cfg, 0, perturb_affine=True)
        self.om = oracle.Model(cfg, self.w)
        self.P, self.max_ctx, self.max_nodes = P, max_ctx, max_nodes
        self.kc, self.vc = W.random_kv_cache(cfg, max_ctx, P, seed=3)
        self.m = ssd.Model(cfg, self.w)
        self.s = ssd.Session(self.m, max_ctx, max_nodes, ssd.to_device(self.kc, cfg), ssd.to_device(self.vc, cfg))

    def oracle_verify(self, toks, parents, P):
        kt, vt = self.om.kv(self.max_nodes), self.om.kv(self.max_nodes)
        lg = oracle.tree_verify(self.om, self.kc, self.vc, P, toks, parents, kt, vt)
        return lg, kt, vt


@pytest.fixture(scope="module")
def small(ssd):
    return Small(ssd)


def _rand_tree(seed, n):
    g = np.random.default_rng(seed)
    return np.array([-1] + [int(g.integers(max(0, i - 8), i)) for i in range(1, n)], np.int32)


TREES = {"single": np.array([-1], np.int32), "binary15": W.complete_binary_tree(15), "chain17": W.chain_tree(17),
         "branch32": W.branching_tree([4, 2, 2, 1], 32), "random33": _rand_tree(1, 33),
         "random48": _rand_tree(2, 48), "chain64": W.chain_tree(64), "random64": _rand_tree(3, 64)}


def _fused(ssd, *sessions):
    for s in sessions:
        s.set_options(pass_mode=ssd.PASS_FUSED)


def _auto(ssd, *sessions):
    for s in sessions:
        s.set_options(pass_mode=ssd.PASS_AUTO)


@pytest.mark.parametrize("name", list(TREES))
@pytest.mark.parametrize("P", [0, 64, 200])
def test_fused_verify_matches_oracle(small, ssd, torch, name, P):
    t = small
    par = TREES[name]
    toks = W.tree_tokens(par, t.cfg.vocab, seed=len(par) + P)
    print(f"fused verify {name} P={P}", flush=True)
    ref, kt, vt = t.oracle_verify(toks, par, P)
    before = t.s.error_count()
    _fused(ssd, t.s)
    try:
        lg = t.s.verify(P, toks, par)
        torch.cuda.synchronize()
    finally:
        _auto(ssd, t.s)
    assert t.s.error_count() == before
    got = lg.cpu().numpy()
    err = np.abs(got - ref).max()
    assert err < TOL, err
    n = len(par)
    for a, b in ((t.s.k_tree, kt), (t.s.v_tree, vt)):
        g = W.bf16_bits_to_f32(ssd.to_host_bits(a)[:, :, :n])
        assert np.abs(g - W.bf16_bits_to_f32(b[:, :, :n])).max() < TOL
    path, plen, nxt = t.s.accept(toks, par, lg)
    op, on = oracle.tree_accept(oracle.GREEDY, toks, par, got)
    assert path[:int(plen.item())].cpu().numpy().tolist() == op.tolist() and int(nxt.item()) == on


def test_fused_and_kernel_paths_agree(small, ssd, torch):
    t = small
    par = TREES["random48"]
    toks = W.tree_tokens(par, t.cfg.vocab, seed=11)
    ref, _, _ = t.oracle_verify(toks, par, t.P)
    out = {}
    for mode in (ssd.PASS_KERNELS, ssd.PASS_FUSED):
        with t.s.options(pass_mode=mode):
            out[mode] = t.s.verify(t.P, toks, par).cpu().numpy()
    assert np.abs(out[ssd.PASS_FUSED] - ref).max() < TOL
    assert np.abs(out[ssd.PASS_KERNELS] - ref).max() < TOL
    assert np.abs(out[ssd.PASS_FUSED] - out[ssd.PASS_KERNELS]).max() < TOL


def test_fused_determinism_and_graph_replay(small, ssd, torch):
    t = small
    par = TREES["random64"]
    toks = W.tree_tokens(par, t.cfg.vocab, seed=9)
    _fused(ssd, t.s)
    try:
        a = t.s.verify(t.P, toks, par).clone()
        b = t.s.verify(t.P, toks, par).clone()
        torch.cuda.synchronize()
        assert torch.equal(a, b)
        out = torch.zeros_like(a)
        g = t.s.capture_verify(t.P, toks, par, out)
        other = W.tree_tokens(TREES["binary15"], t.cfg.vocab, seed=1)
        for _ in range(3):
            out.zero_()
            g.launch()
            torch.cuda.synchronize()
            assert torch.equal(out, a)
            t.s.verify(t.P, other, TREES["binary15"])  # eager work between replays
            torch.cuda.synchronize()
        g.close()
    finally:
        _auto(ssd, t.s)
    assert t.s.error_count() == 0


def test_fused_node_independent_of_tree_slot_and_tiles(small, ssd, torch):
    """A node's logits depend only on its root path, bitwise: the same chain
    alone (1 tile), at other slots among decoys (1 tile), and spread over a
    3-tile tree."""
    t = small
    _fused(ssd, t.s)
    try:
        toks_a = np.array([5, 6, 7, 8], np.int32)
        lg_a = t.s.verify(t.P, toks_a, W.chain_tree(4)).clone()
        par_b = np.array([-1, 0, 0, 1, 2, 2, 3, 5, 4, 5], np.int32)
        toks_b = np.array([5, 100, 6, 101, 102, 7, 103, 104, 105, 8], np.int32)
        lg_b = t.s.verify(t.P, toks_b, par_b).clone()
        # 40 nodes: the chain at slots 0, 13, 27, 39, decoys elsewhere
        n = 40
        slots = [0, 13, 27, 39]
        par_c = np.zeros(n, np.int32)
        toks_c = np.full(n, 300, np.int32)
        par_c[0] = -1
        prev = 0
        for i in range(1, n):
            if i in slots:
                par_c[i] = prev
                prev = i
            else:
                par_c[i] = 0
                toks_c[i] = 300 + i
        toks_c[slots] = toks_a
        lg_c = t.s.verify(t.P, toks_c, par_c).clone()
        torch.cuda.synchronize()
    finally:
        _auto(ssd, t.s)
    for i, j in zip(range(4), [0, 2, 5, 9]):
        assert torch.equal(lg_a[i], lg_b[j]), (i, j)
    for i, j in zip(range(4), slots):
        assert torch.equal(lg_a[i], lg_c[j]), (i, j)


def test_fused_prefix_view_equals_truncated_model(small, ssd, torch):
    """A 2-layer view of the 3-layer model (shared session) gives bitwise the
    logits of a model built from those two layers alone."""
    t = small
    cfg2 = t.cfg.with_(n_layer=2)
    w2 = dict(t.w)
    for k in W.LAYER_TENSORS:
        w2[k] = t.w[k][:2]
    m2 = ssd.Model(cfg2, w2)
    s2 = ssd.Session(m2, t.max_ctx, t.max_nodes, ssd.to_device(t.kc[:2], cfg2), ssd.to_device(t.vc[:2], cfg2))
    view = t.m.prefix_view(2)
    par = TREES["branch32"]
    toks = W.tree_tokens(par, t.cfg.vocab, seed=4)
    _fused(ssd, t.s, s2)
    try:
        a = s2.verify(t.P, toks, par).clone()
        lg = torch.empty((len(par), t.cfg.vocab), dtype=torch.float32, device="cuda")
        from paper_2308_04623_amd.ssd import _check, _i32, _p32, _stream, lib
        import ctypes as C
        tt, pp = _i32(toks), _i32(par)
        _check(lib().ssd_tree_verify(view.handle, t.s.handle, t.P, _p32(tt), _p32(pp), len(tt),
                                     C.c_void_p(lg.data_ptr()), _stream(None)), "ssd_tree_verify")
        torch.cuda.synchronize()
    finally:
        _auto(ssd, t.s, s2)
    assert torch.equal(a, lg)
    om2 = oracle.Model(cfg2, w2)
    ref = oracle.tree_verify(om2, t.kc[:2], t.vc[:2], t.P, toks, par, om2.kv(t.max_nodes), om2.kv(t.max_nodes))
    assert np.abs(a.cpu().numpy() - ref).max() < TOL
    view.close()
    s2.close()
    m2.close()


def test_fused_only_mode_rejects_unsupported(small, ssd, torch):
    t = small
    par = W.chain_tree(65)
    s = ssd.Session(t.m, t.max_ctx, 65, ssd.to_device(t.kc, t.cfg), ssd.to_device(t.vc, t.cfg))
    _fused(ssd, s)
    with pytest.raises(ssd.SSDError) as e:
        s.verify(t.P, W.tree_tokens(par, t.cfg.vocab, seed=1), par)
    assert e.value.status == ssd.E_UNSUPPORTED
    s.close()


def test_fused_long_cache_matches_oracle(ssd, torch):
    """A 5000-row prefix: 20 prefix units per (head, tile), so every tile's
    parts are merged in several rounds and the tile counter wraps at 20."""
    P, max_ctx = 5000, 5120
    cfg = SMALL.with_(n_pos=max_ctx + 64)
    w = W.make_weights(cfg, 1, perturb_affine=True)
    om = oracle.Model(cfg, w)
    m = ssd.Model(cfg, w)
    kc, vc = W.random_kv_cache(cfg, max_ctx, P, seed=5)
    s = ssd.Session(m, max_ctx, 40, ssd.to_device(kc, cfg), ssd.to_device(vc, cfg))
    _fused(ssd, s)
    assert s.verify_path(33) == ssd.PASS_FUSED
    par = TREES["random33"]
    toks = W.tree_tokens(par, cfg.vocab, seed=8)
    got = s.verify(P, toks, par).cpu().numpy()
    again = s.verify(P, toks, par).cpu().numpy()
    assert s.error_count() == 0
    assert np.array_equal(got, again)
    ref = oracle.tree_verify(om, kc, vc, P, toks, par, om.kv(40), om.kv(40))
    assert np.abs(got - ref).max() < TOL
    s.close()
    m.close()


def test_fused_float16_overflow_is_counted(small, ssd, torch):
    """A LayerNorm output past float16's range (gain 1e5) is counted in the
    session's error counter by the persistent pass too."""
    t = small
    w = dict(t.w)
    w["ln1_g"] = [W.f32_to_bf16_bits(np.full(t.cfg.d_model, 1e5, np.float32))] + list(t.w["ln1_g"][1:])
    m = ssd.Model(t.cfg, w)
    s = ssd.Session(m, t.max_ctx, 16, ssd.to_device(t.kc, t.cfg), ssd.to_device(t.vc, t.cfg))
    _fused(ssd, s)
    assert s.verify_path(3) == ssd.PASS_FUSED
    s.verify(t.P, [1, 2, 3], [-1, 0, 0])
    assert s.error_count() > 0
    s.close()
    m.close()


@pytest.mark.parametrize("name", ["single", "binary15", "random33", "random64"])
@pytest.mark.parametrize("mode", ["fused", "kernels"])
def test_verify_greedy_equals_verify_then_accept(small, ssd, torch, name, mode):
    """ssd_tree_verify_greedy (the persistent pass's LM head leaves each
    workgroup's maximum per node, so the walk skips the logits) gives the
    logits and the greedy path of ssd_tree_verify + ssd_tree_accept, bit for
    bit, eagerly and from a captured graph; a vocabulary row duplicated at a
    far id makes exact ties across workgroups, which go to the lower id."""
    t = small
    w = dict(t.w)
    wte = t.w["wte"].copy()
    wte[1999] = wte[3]           # token 3 and token 1999 always have equal logits
    w["wte"] = wte
    m = ssd.Model(t.cfg, w)
    s = ssd.Session(m, t.max_ctx, t.max_nodes, ssd.to_device(t.kc, t.cfg), ssd.to_device(t.vc, t.cfg))
    s.set_options(pass_mode=ssd.PASS_FUSED if mode == "fused" else ssd.PASS_KERNELS)
    par = TREES[name]
    toks = W.tree_tokens(par, t.cfg.vocab, seed=21)
    for P in (0, t.P):
        lg_a = s.verify(P, toks, par).clone()
        pa, la, na = s.accept(toks, par, lg_a)
        lg_b, pb, lb, nb = s.verify_greedy(P, toks, par)
        torch.cuda.synchronize()
        assert torch.equal(lg_a, lg_b)
        n = int(la.item())
        assert int(lb.item()) == n and pa[:n].tolist() == pb[:n].tolist() and int(na.item()) == int(nb.item())
        host = lg_a.cpu().numpy()
        assert np.array_equal(host[:, 3], host[:, 1999])
        # graph replay of the same step
        lg_c = torch.zeros_like(lg_a)
        outs = s._accept_outs(len(par), None)
        g = s.capture_verify_greedy(P, toks, par, lg_c, outs)
        for _ in range(2):
            g.launch()
            torch.cuda.synchronize()
            assert torch.equal(lg_c, lg_a)
            assert int(outs[1].item()) == n and outs[0][:n].tolist() == pa[:n].tolist()
            assert int(outs[2].item()) == int(na.item())
        g.close()
    assert s.error_count() == 0
    s.close()
    m.close()
