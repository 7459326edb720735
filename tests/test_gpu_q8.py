"""GPU parity of the 8-bit weight models (ssd_model_create_q8) against the
oracle's 8-bit mode (oracle.Model(..., q8=True)) on the same seeded inputs.

Bars: the 8-bit codes and float32 scales bit-exact (the codes are integers
decided in float32 on both sides); logits and tree K/V within 2e-2 max-abs
(the bfloat16 models' bar: the same float16 activations and float32
accumulation, only the weights differ); greedy accept bit-exact on the GPU's
logits."""
import numpy as np
import pytest

import oracle
from paper_2308_04623_amd import workloads as W

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


@pytest.fixture(scope="module")
def ssd(torch):
    from paper_2308_04623_amd import ssd as s
    s.lib()
    return s


def special_rows(g, rows, cols):
    """bfloat16 rows that probe the quantizer's edges: all zeros, below the
    2^-100 floor, exact multiples of a power of two, one huge entry, ties
    of w * 127 / max near x.5, heavy tails."""
    x = g.standard_normal((rows, cols)).astype(np.float32) * 0.02
    x[0] = 0
    x[1] = 0
    x[1, 3] = 2.0 ** -101
    x[2] = g.integers(-127, 128, cols) * 2.0 ** -9
    x[2, 0] = 127 * 2.0 ** -9
    x[3, 5] = 300.0
    x[4] = (np.arange(cols) % 254 - 127 + 0.5) / 127.0   # near k + 1/2 on the 127 scale
    x[4, 0] = 1.0
    x[5] *= g.standard_t(1.5, cols).astype(np.float32)
    return W.f32_to_bf16_bits(x)


class Q8Tiny:
    def __init__(self, ssd, P=64, max_ctx=160, max_nodes=128):
        self.cfg = cfg = W.TINY.with_(dtype="bf16")
        self.w = W.make_weights(cfg, 0, perturb_affine=True)
        self.om = oracle.Model(cfg, self.w, q8=True)
        self.P, self.max_ctx, self.max_nodes = P, max_ctx, max_nodes
        self.kc, self.vc = W.random_kv_cache(cfg, max_ctx, P, seed=3)
        self.m = ssd.Model(cfg, self.w, q8=True)
        self.s = ssd.Session(self.m, max_ctx, max_nodes, ssd.to_device(self.kc, cfg), ssd.to_device(self.vc, cfg))

    def oracle_verify(self, toks, parents, P=None):
        P = self.P if P is None else P
        kt, vt = self.om.kv(self.max_nodes), self.om.kv(self.max_nodes)
        return oracle.tree_verify(self.om, self.kc, self.vc, P, toks, parents, kt, vt), kt, vt


@pytest.fixture(scope="module")
def tq(ssd):
    return Q8Tiny(ssd)


MATS = ["w_qkv", "w_o", "w_fc", "w_pr"]


def _codes_equal(m, om, cfg):
    for which, name in enumerate(MATS):
        for l in range(cfg.n_layer):
            codes, scales = m.q8_matrix(which, l)
            rc, rs = om.q8[name][l]
            assert np.array_equal(codes, rc), (name, l)
            assert np.array_equal(scales.view(np.uint32), rs.view(np.uint32)), (name, l)
    codes, scales = m.q8_matrix(4)
    rc, rs = om.q8["head"]
    assert np.array_equal(codes, rc) and np.array_equal(scales.view(np.uint32), rs.view(np.uint32))


def test_q8_codes_and_scales_bit_exact(tq, ssd):
    _codes_equal(tq.m, tq.om, tq.cfg)
    # the quantizer's edge rows (these weights only feed this check: rows
    # like the one at 300 put the activations far from the parity cases')
    cfg, w = tq.cfg, W.make_weights(tq.cfg, 1)
    g = np.random.default_rng(11)
    w["w_qkv"][0] = special_rows(g, 3 * cfg.d_model, cfg.d_model)
    w["w_pr"][1] = special_rows(g, cfg.d_model, cfg.d_mlp)
    w["wte"] = special_rows(g, cfg.vocab, cfg.d_model)
    m = ssd.Model(cfg, w, q8=True)
    _codes_equal(m, oracle.Model(cfg, w, q8=True), cfg)
    m.close()


def _trees():
    g = np.random.default_rng(5)
    rnd = lambda n: np.array([-1] + [int(g.integers(max(0, i - 8), i)) for i in range(1, n)], np.int32)
    return {"binary15": W.complete_binary_tree(15), "single": np.array([-1], np.int32),
            "chain17": W.chain_tree(17), "random100": rnd(100), "random128": rnd(128)}


TREES = _trees()


@pytest.mark.parametrize("gemm", ["vec", "mfma"])
@pytest.mark.parametrize("name", list(TREES))
@pytest.mark.parametrize("P", [0, 64])
def test_q8_tiny_verify(tq, ssd, torch, gemm, name, P):
    par = TREES[name]
    if gemm == "vec" and len(par) > 16:
        par = par[:16]
    toks = W.tree_tokens(par, tq.cfg.vocab, seed=7 + len(par))
    ref, kt, vt = tq.oracle_verify(toks, par, P)
    with tq.s.options(gemm_path=ssd.GEMM_VEC if gemm == "vec" else ssd.GEMM_MFMA):
        lg = tq.s.verify(P, toks, par)
        torch.cuda.synchronize()
    assert tq.s.error_count() == 0
    err = np.abs(lg.cpu().numpy() - ref).max()
    assert err < TOL, err
    n = len(par)
    kg = W.bf16_bits_to_f32(ssd.to_host_bits(tq.s.k_tree)[:, :, :n])
    assert np.abs(kg - W.bf16_bits_to_f32(kt[:, :, :n])).max() < TOL
    # greedy accept on the GPU's logits, bit-exact
    path, plen, nxt = tq.s.accept(toks, par, lg)
    op, on = oracle.tree_accept(oracle.GREEDY, toks, par, lg.cpu().numpy())
    assert path[:int(plen.item())].cpu().numpy().tolist() == op.tolist() and int(nxt.item()) == on


def test_q8_graph_replay_and_determinism(tq, ssd, torch):
    par = TREES["random100"]
    toks = W.tree_tokens(par, tq.cfg.vocab, seed=9)
    a = tq.s.verify(tq.P, toks, par).clone()
    b = tq.s.verify(tq.P, toks, par).clone()
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    out = torch.zeros_like(a)
    g = tq.s.capture_verify(tq.P, toks, par, out)
    other = W.tree_tokens(TREES["binary15"], tq.cfg.vocab, seed=1)
    for _ in range(3):
        out.zero_()
        g.launch()
        torch.cuda.synchronize()
        assert torch.equal(out, a)
        tq.s.verify(tq.P, other, TREES["binary15"])
        torch.cuda.synchronize()
    g.close()


def test_q8_prefix_view_is_the_first_layers(tq, ssd, torch):
    """The draft view of an 8-bit model runs the first layers' 8-bit
    matrices and the 8-bit head (the oracle's 8-bit model cut to one layer)."""
    cfg1 = tq.cfg.with_(n_layer=1)
    w1 = {k: (v[:1] if isinstance(v, list) else v) for k, v in tq.w.items()}
    om1 = oracle.Model(cfg1, w1, q8=True)
    view = tq.m.prefix_view(1)
    kc1, vc1 = tq.kc[:1].copy(), tq.vc[:1].copy()
    s1 = ssd.Session(view, tq.max_ctx, 32, ssd.to_device(kc1, cfg1), ssd.to_device(vc1, cfg1))
    par = TREES["binary15"]
    toks = W.tree_tokens(par, cfg1.vocab, seed=4)
    lg = s1.verify(tq.P, toks, par)
    torch.cuda.synchronize()
    ref = oracle.tree_verify(om1, kc1, vc1, tq.P, toks, par, om1.kv(32), om1.kv(32))
    assert np.abs(lg.cpu().numpy() - ref).max() < TOL
    s1.close()
    view.close()


def test_q8_error_paths(ssd, torch):
    f32 = W.TINY
    w = W.make_weights(f32, 0)
    with pytest.raises(ssd.SSDError) as e:
        ssd.Model(f32, w, q8=True)
    assert e.value.status == ssd.E_UNSUPPORTED
    # d_model 96 (head_dim 32) is a multiple of 32, not of 64
    odd = W.TINY.with_(dtype="bf16", d_model=96, n_head=3)
    with pytest.raises(ssd.SSDError) as e:
        ssd.Model(odd, W.make_weights(odd, 0), q8=True)
    assert e.value.status == ssd.E_UNSUPPORTED
    cfg = W.TINY.with_(dtype="bf16")
    wn = W.make_weights(cfg, 0)
    wn["w_fc"][1] = wn["w_fc"][1].copy()
    wn["w_fc"][1][7, 9] = 0x7FC0      # NaN
    with pytest.raises(ssd.SSDError) as e:
        ssd.Model(cfg, wn, q8=True)
    assert e.value.status == ssd.E_UNSUPPORTED
    m16 = ssd.Model(cfg, W.make_weights(cfg, 0))
    with pytest.raises(ssd.SSDError) as e:
        m16.q8_matrix(0, 0)
    assert e.value.status == ssd.E_INVALID_ARG
    m8 = ssd.Model(cfg, W.make_weights(cfg, 0), q8=True)
    for which, layer in ((5, 0), (-1, 0), (0, cfg.n_layer)):
        with pytest.raises(ssd.SSDError) as e:
            m8.q8_matrix(which, layer)
        assert e.value.status == ssd.E_INVALID_ARG
    m16.close()
    m8.close()


# ---- the persistent single-launch pass (head dimension 64, <= 64 nodes)

SMALL = W.GPT2Config(n_layer=3, d_model=256, n_head=4, d_mlp=1024, vocab=2000, n_pos=512, dtype="bf16")


class Q8Small:
    def __init__(self, ssd, P=200, max_ctx=320, max_nodes=64):
        self.cfg = cfg = SMALL
        self.w = W.make_weights(cfg, 0, perturb_affine=True)
        self.om = oracle.Model(cfg, self.w, q8=True)
        self.P, self.max_ctx, self.max_nodes = P, max_ctx, max_nodes
        self.kc, self.vc = W.random_kv_cache(cfg, max_ctx, P, seed=3)
        self.m = ssd.Model(cfg, self.w, q8=True)
        self.s = ssd.Session(self.m, max_ctx, max_nodes, ssd.to_device(self.kc, cfg), ssd.to_device(self.vc, cfg))

    def oracle_verify(self, toks, parents, P):
        kt, vt = self.om.kv(self.max_nodes), self.om.kv(self.max_nodes)
        return oracle.tree_verify(self.om, self.kc, self.vc, P, toks, parents, kt, vt), kt, vt


@pytest.fixture(scope="module")
def sq(ssd):
    return Q8Small(ssd)


def _rand_tree(seed, n):
    g = np.random.default_rng(seed)
    return np.array([-1] + [int(g.integers(max(0, i - 8), i)) for i in range(1, n)], np.int32)


FTREES = {"single": np.array([-1], np.int32), "binary15": W.complete_binary_tree(15), "chain17": W.chain_tree(17),
          "branch32": W.branching_tree([4, 2, 2, 1], 32), "random33": _rand_tree(1, 33),
          "random48": _rand_tree(2, 48), "random64": _rand_tree(3, 64)}


@pytest.mark.parametrize("name", list(FTREES))
@pytest.mark.parametrize("P", [0, 64, 200])
def test_q8_fused_verify_matches_oracle(sq, ssd, torch, name, P):
    par = FTREES[name]
    toks = W.tree_tokens(par, sq.cfg.vocab, seed=len(par) + P)
    print(f"8-bit fused verify {name} P={P}", flush=True)
    ref, kt, vt = sq.oracle_verify(toks, par, P)
    with sq.s.options(pass_mode=ssd.PASS_FUSED):
        assert sq.s.verify_path(len(par)) == ssd.PASS_FUSED
        lg = sq.s.verify(P, toks, par)
        torch.cuda.synchronize()
    assert sq.s.error_count() == 0
    got = lg.cpu().numpy()
    assert np.abs(got - ref).max() < TOL
    n = len(par)
    for a, b in ((sq.s.k_tree, kt), (sq.s.v_tree, vt)):
        g = W.bf16_bits_to_f32(ssd.to_host_bits(a)[:, :, :n])
        assert np.abs(g - W.bf16_bits_to_f32(b[:, :, :n])).max() < TOL
    path, plen, nxt = sq.s.accept(toks, par, lg)
    op, on = oracle.tree_accept(oracle.GREEDY, toks, par, got)
    assert path[:int(plen.item())].cpu().numpy().tolist() == op.tolist() and int(nxt.item()) == on


def test_q8_fused_replay_greedy_and_kernel_path(sq, ssd, torch):
    """The 8-bit persistent pass: bitwise repeatable eagerly and from a
    captured graph; its verify + greedy step equals verify then accept bit
    for bit; the per-sub-layer path agrees with it within the bar."""
    par = FTREES["random64"]
    toks = W.tree_tokens(par, sq.cfg.vocab, seed=9)
    ref, _, _ = sq.oracle_verify(toks, par, sq.P)
    with sq.s.options(pass_mode=ssd.PASS_FUSED):
        a = sq.s.verify(sq.P, toks, par).clone()
        b = sq.s.verify(sq.P, toks, par).clone()
        torch.cuda.synchronize()
        assert torch.equal(a, b)
        out = torch.zeros_like(a)
        g = sq.s.capture_verify(sq.P, toks, par, out)
        other = W.tree_tokens(FTREES["binary15"], sq.cfg.vocab, seed=1)
        for _ in range(3):
            out.zero_()
            g.launch()
            torch.cuda.synchronize()
            assert torch.equal(out, a)
            sq.s.verify(sq.P, other, FTREES["binary15"])
            torch.cuda.synchronize()
        g.close()
        pa, la, na = sq.s.accept(toks, par, a)
        lg_b, pb, lb, nb = sq.s.verify_greedy(sq.P, toks, par)
        torch.cuda.synchronize()
        assert torch.equal(a, lg_b)
        n = int(la.item())
        assert int(lb.item()) == n and pa[:n].tolist() == pb[:n].tolist() and int(na.item()) == int(nb.item())
    with sq.s.options(pass_mode=ssd.PASS_KERNELS):
        k = sq.s.verify(sq.P, toks, par).cpu().numpy()
    assert np.abs(k - ref).max() < TOL
    assert np.abs(a.cpu().numpy() - ref).max() < TOL
    assert sq.s.error_count() == 0
