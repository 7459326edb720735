"""GPU parity: libssd (HIP, through the C ABI) against the CPU oracle on the
same seeded inputs.

Bars: float32 models within 1e-4 max-abs on logits and K/V; bfloat16 models
within 2e-2 on logits; tree bookkeeping, accepted paths, greedy and sampled
tokens and committed cache rows bit-exact (accept is compared on identical
logits, the GPU's own copied to the host)."""
import numpy as np
import pytest

import oracle
from paper_2308_04623_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL_F32, TOL_BF16 = 1e-4, 2e-2


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


class Tiny:
    """TINY model on both sides, with a prefix cache."""

    def __init__(self, ssd, dtype="f32", max_ctx=160, max_nodes=128, P=64):
        self.cfg = cfg = W.TINY.with_(dtype=dtype)
        self.w = W.make_weights(cfg, 0, perturb_affine=True)
        self.om = oracle.Model(cfg, self.w)
        self.P, self.max_ctx, self.max_nodes = P, max_ctx, max_nodes
        self.kc, self.vc = W.random_kv_cache(cfg, max_ctx, P, seed=3)
        self.m = ssd.Model(cfg, self.w)
        self.s = ssd.Session(self.m, max_ctx, max_nodes, ssd.to_device(self.kc, cfg), ssd.to_device(self.vc, cfg))

    def oracle_verify(self, toks, parents, P=None):
        P = self.P if P is None else P
        kt, vt = self.om.kv(self.max_nodes), self.om.kv(self.max_nodes)
        lg = oracle.tree_verify(self.om, self.kc, self.vc, P, toks, parents, kt, vt)
        return lg, kt, vt


@pytest.fixture(scope="module")
def tiny32(ssd):
    return Tiny(ssd, "f32")


@pytest.fixture(scope="module")
def tiny16(ssd):
    return Tiny(ssd, "bf16")


def _trees():
    g = np.random.default_rng(5)
    rnd = lambda n: np.array([-1] + [int(g.integers(max(0, i - 8), i)) for i in range(1, n)], np.int32)
    return {"binary15": W.complete_binary_tree(15), "single": np.array([-1], np.int32),
            "chain17": W.chain_tree(17), "chain64": W.chain_tree(64), "branch32": W.branching_tree([4, 2, 2, 1], 32),
            "random100": rnd(100), "random128": rnd(128)}


TREES = _trees()


@pytest.mark.parametrize("name", list(TREES))
@pytest.mark.parametrize("P", [0, 64])
def test_tiny_f32_verify(tiny32, ssd, torch, name, P):
    t = tiny32
    par = TREES[name]
    toks = W.tree_tokens(par, t.cfg.vocab, seed=len(par))
    ref, kt, vt = t.oracle_verify(toks, par, P)
    lg = t.s.verify(P, toks, par)
    torch.cuda.synchronize()
    got = lg.cpu().numpy()
    assert np.abs(got - ref).max() < TOL_F32
    n = len(par)
    for a, b in ((t.s.k_tree, kt), (t.s.v_tree, vt)):
        assert np.abs(ssd.to_host_bits(a)[:, :, :n] - b[:, :, :n]).max() < TOL_F32
    # greedy accept on the GPU's own logits is bit-exact with the oracle's walk
    path, plen, nxt = t.s.accept(toks, par, lg)
    op, on = oracle.tree_accept(oracle.GREEDY, toks, par, got)
    assert path[:int(plen.item())].cpu().numpy().tolist() == op.tolist() and int(nxt.item()) == on


@pytest.mark.parametrize("gemm", ["vec", "mfma"])
@pytest.mark.parametrize("name", ["binary15", "single", "chain17", "random100"])
def test_tiny_bf16_verify(tiny16, ssd, torch, gemm, name):
    t = tiny16
    par = TREES[name]
    if gemm == "vec" and len(par) > 16:
        par = par[:16]
    t.s.set_options(gemm_path=ssd.GEMM_VEC if gemm == "vec" else ssd.GEMM_MFMA)
    try:
        toks = W.tree_tokens(par, t.cfg.vocab, seed=7)
        ref, kt, vt = t.oracle_verify(toks, par)
        lg = t.s.verify(t.P, toks, par)
        torch.cuda.synchronize()
    finally:
        t.s.set_options(gemm_path=ssd.GEMM_AUTO)
    assert np.abs(lg.cpu().numpy() - ref).max() < TOL_BF16
    n = len(par)
    kg = W.bf16_bits_to_f32(ssd.to_host_bits(t.s.k_tree)[:, :, :n])
    assert np.abs(kg - W.bf16_bits_to_f32(kt[:, :, :n])).max() < TOL_BF16


def test_determinism_and_graph_replay(tiny16, ssd, torch):
    t = tiny16
    par = TREES["random100"]
    toks = W.tree_tokens(par, t.cfg.vocab, seed=9)
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
        t.s.verify(t.P, other, TREES["binary15"])      # eager work between replays
        torch.cuda.synchronize()
    g.close()


@pytest.mark.parametrize("gemm", ["vec", "mfma"])
def test_node_result_independent_of_tree_and_slot(tiny16, ssd, torch, gemm):
    """A node's logits depend only on its root path, bitwise, whatever the
    other nodes and its index (one GEMM path pinned)."""
    t = tiny16
    t.s.set_options(gemm_path=ssd.GEMM_VEC if gemm == "vec" else ssd.GEMM_MFMA)
    try:
        toks_a = np.array([5, 6, 7, 8], np.int32)
        lg_a = t.s.verify(t.P, toks_a, W.chain_tree(4)).clone()
        # same chain at slots 0, 2, 5, 9 with decoy siblings
        par_b = np.array([-1, 0, 0, 1, 2, 2, 3, 5, 4, 5], np.int32)
        toks_b = np.array([5, 100, 6, 101, 102, 7, 103, 104, 105, 8], np.int32)
        lg_b = t.s.verify(t.P, toks_b, par_b).clone()
        torch.cuda.synchronize()
    finally:
        t.s.set_options(gemm_path=ssd.GEMM_AUTO)
    for i, j in zip([0, 1, 2, 3], [0, 2, 5, 9]):
        assert torch.equal(lg_a[i], lg_b[j]), (i, j)


def test_commit_bitwise_and_continue(tiny32, ssd, torch):
    t = tiny32
    par = TREES["binary15"]
    toks = W.tree_tokens(par, t.cfg.vocab, seed=2)
    lg = t.s.verify(t.P, toks, par)
    path = torch.tensor([0, 1, 4, 9, 0, 0], dtype=torch.int32, device="cuda")
    plen = torch.tensor([4], dtype=torch.int32, device="cuda")
    kc0 = ssd.to_host_bits(t.s.k_cache).copy()
    t.s.commit(t.P, path, plen)
    torch.cuda.synchronize()
    kc1, kt = ssd.to_host_bits(t.s.k_cache), ssd.to_host_bits(t.s.k_tree)
    for j, node in enumerate([0, 1, 4, 9]):
        assert np.array_equal(kc1[:, :, t.P + j], kt[:, :, node])
    assert np.array_equal(kc1[:, :, :t.P], kc0[:, :, :t.P])
    assert np.array_equal(kc1[:, :, t.P + 4:], kc0[:, :, t.P + 4:])
    # continuing from the committed cache matches the oracle doing the same
    ref_lg, okt, ovt = t.oracle_verify(toks, par)
    assert np.abs(lg.cpu().numpy() - ref_lg).max() < TOL_F32
    okc, ovc = t.kc.copy(), t.vc.copy()
    oracle.kv_commit(t.om, okc, ovc, t.P, okt, ovt, [0, 1, 4, 9])
    nxt = [int(toks[3])]
    want = oracle.tree_verify(t.om, okc, ovc, t.P + 4, nxt, [-1], t.om.kv(1), t.om.kv(1))
    got = t.s.verify(t.P + 4, nxt, [-1])
    torch.cuda.synchronize()
    assert np.abs(got.cpu().numpy() - want).max() < TOL_F32
    # commit rows past max_ctx are skipped and counted, never written
    before = t.s.error_count()
    far = torch.tensor([0, 1, 2], dtype=torch.int32, device="cuda")
    t.s.commit(t.max_ctx - 1, far, torch.tensor([3], dtype=torch.int32, device="cuda"))
    assert t.s.error_count() == before + 2
    # restore the cache for the other tests
    t.s.k_cache.copy_(ssd.to_device(t.kc, t.cfg))
    t.s.v_cache.copy_(ssd.to_device(t.vc, t.cfg))


def test_error_paths_enqueue_nothing(tiny32, ssd, torch):
    t = tiny32
    cases = [(dict(P=0, toks=[1, 2], par=[0, 0]), ssd.E_INVALID_TREE),
             (dict(P=0, toks=[1, 99999], par=[-1, 0]), ssd.E_INVALID_ARG),
             (dict(P=t.max_ctx + 1, toks=[1], par=[-1]), ssd.E_CAPACITY),
             (dict(P=0, toks=[1] * (t.max_nodes + 1), par=W.chain_tree(t.max_nodes + 1)), ssd.E_CAPACITY),
             (dict(P=t.cfg.n_pos - 1, toks=[1, 2], par=[-1, 0]), ssd.E_CAPACITY)]
    for c, st in cases:
        with pytest.raises(ssd.SSDError) as e:
            t.s.verify(c["P"], c["toks"], c["par"])
        assert e.value.status == st
    # a model of another shape on this session's buffers: refused on the host
    own = t.s.model
    for other_cfg in (t.cfg.with_(d_mlp=t.cfg.d_mlp // 2), t.cfg.with_(vocab=t.cfg.vocab + 32),
                      t.cfg.with_(n_layer=t.cfg.n_layer + 1)):
        t.s.model = ssd.Model(other_cfg, W.make_weights(other_cfg, 2))
        try:
            with pytest.raises(ssd.SSDError) as e:
                t.s.verify(0, [1, 2], [-1, 0])
            assert e.value.status == ssd.E_INVALID_ARG, other_cfg
        finally:
            t.s.model = own
    lg = torch.zeros((2, t.cfg.vocab), device="cuda")
    with pytest.raises(ssd.SSDError):
        t.s.accept([0, 1], [-1, 0], lg, mode=ssd.SAMPLE_WOR)             # no draft probs
    with pytest.raises(ssd.SSDError):
        t.s.accept([0, 1], [-1, 0], lg, mode=ssd.GREEDY, draft_probs=lg)  # greedy with draft probs


# ---------------------------------------------------------------- sampling accept

@pytest.fixture(scope="module")
def wide(ssd):
    """A small model whose vocabulary is GPT-2's, for accept-only tests."""
    cfg = W.TINY.with_(vocab=50257, n_layer=1)
    m = ssd.Model(cfg, W.make_weights(cfg, 1))
    return cfg, ssd.Session(m, 8, 256)


def _draft_tree(g, V, branching, n_max):
    par = W.branching_tree(branching, n_max)
    toks = g.integers(0, V, len(par)).astype(np.int32)
    return toks, par


@pytest.mark.parametrize("V", [512, 50257])
@pytest.mark.parametrize("mode", ["wor", "iid"])
def test_sampling_accept_bit_exact(wide, ssd, torch, V, mode):
    cfg, s = wide
    g = np.random.default_rng(V + len(mode))
    md = ssd.SAMPLE_WOR if mode == "wor" else ssd.SAMPLE_IID
    for trial in range(12):
        toks, par = _draft_tree(g, V, [4, 2, 2, 1], 32 if trial % 2 else 256)
        n = len(par)
        lg = (g.standard_normal((n, V)) * 2.0).astype(np.float32)
        q = g.dirichlet(np.ones(V) * 0.3, size=n).astype(np.float32)
        # make acceptance likely somewhere: copy target mass into the draft
        q = (0.5 * q + 0.5 * np.exp(lg - lg.max(1, keepdims=True)) /
             np.exp(lg - lg.max(1, keepdims=True)).sum(1, keepdims=True)).astype(np.float32)
        # children of the root: draw the top target tokens so paths get long
        for c in range(1, n):
            if g.random() < 0.7:
                toks[c] = int(np.argmax(lg[par[c]] + g.gumbel(size=V)))
        dlg, dq = torch.from_numpy(lg).cuda(), torch.from_numpy(q).cuda()
        path, plen, nxt = s.accept(toks, par, dlg, mode=md, draft_probs=dq, temperature=1.0, seed=trial)
        op, on = oracle.tree_accept(oracle.SAMPLE_WOR if mode == "wor" else oracle.SAMPLE_IID, toks, par, lg, q,
                                    1.0, trial)
        assert path[:int(plen.item())].cpu().numpy().tolist() == op.tolist(), trial
        assert int(nxt.item()) == on, trial


def test_greedy_accept_full_vocab_ties(wide, ssd, torch):
    cfg, s = wide
    V = 50257
    g = np.random.default_rng(1)
    n = 64
    par = W.branching_tree([4, 2, 2, 1], n)
    lg = g.integers(-3, 3, (n, V)).astype(np.float32)    # many exact ties
    am = np.array([np.flatnonzero(r == r.max())[0] for r in lg])
    toks = g.integers(0, V, n).astype(np.int32)
    for c in range(1, n):
        if g.random() < 0.8:
            toks[c] = am[par[c]]
    path, plen, nxt = s.accept(toks, par, torch.from_numpy(lg).cuda())
    op, on = oracle.tree_accept(oracle.GREEDY, toks, par, lg)
    assert path[:int(plen.item())].cpu().numpy().tolist() == op.tolist() and int(nxt.item()) == on


@pytest.mark.parametrize("T", [0.7, 1.5])
@pytest.mark.parametrize("mode", ["wor", "iid"])
def test_sampling_accept_temperature_and_zero_draft_entries(wide, ssd, torch, T, mode):
    """Temperatures other than 1, and draft rows that are exactly zero at
    tested tokens: such a child is accepted iff the residual target mass at
    its token is positive (tested both ways: tokens whose target probability
    underflows to 0 are rejected)."""
    cfg, s = wide
    V = 4096
    g = np.random.default_rng(int(T * 10) + len(mode))
    md = ssd.SAMPLE_WOR if mode == "wor" else ssd.SAMPLE_IID
    zero_hits = 0
    for trial in range(10):
        toks, par = _draft_tree(g, V, [3, 2, 2, 1], 40)
        n = len(par)
        lg = (g.standard_normal((n, V)) * 2.0).astype(np.float32)
        q = g.dirichlet(np.ones(V) * 0.3, size=n).astype(np.float32)
        for c in range(1, n):
            u = par[c]
            kind = g.random()
            if kind < 0.35:
                q[u, toks[c]] = 0.0                       # zero draft mass, positive target mass
                zero_hits += 1
            elif kind < 0.5:
                q[u, toks[c]] = 0.0                       # zero draft mass and zero target mass
                lg[u, toks[c]] = -1e30
                zero_hits += 1
        dlg, dq = torch.from_numpy(lg).cuda(), torch.from_numpy(q).cuda()
        path, plen, nxt = s.accept(toks, par, dlg, mode=md, draft_probs=dq, temperature=T, seed=100 + trial)
        op, on = oracle.tree_accept(oracle.SAMPLE_WOR if mode == "wor" else oracle.SAMPLE_IID, toks, par, lg, q,
                                    T, 100 + trial)
        assert path[:int(plen.item())].cpu().numpy().tolist() == op.tolist(), trial
        assert int(nxt.item()) == on, trial
    assert zero_hits > 20


@pytest.mark.parametrize("mode", ["wor", "iid"])
def test_sampling_accept_residual_mass_zero(wide, ssd, torch, mode):
    """A root whose target and draft are the same point mass: every child
    (a different token) is rejected, the residual becomes all zeros (Z = 0),
    and the extra token is drawn from the target itself (the point)."""
    cfg, s = wide
    V = 1000
    par = np.array([-1, 0, 0, 0, 1], np.int32)
    toks = np.array([5, 11, 12, 13, 14], np.int32)
    n = len(par)
    lg = np.full((n, V), -1e30, np.float32)
    lg[:, 7] = 0.0
    q = np.zeros((n, V), np.float32)
    q[:, 7] = 1.0
    md = ssd.SAMPLE_WOR if mode == "wor" else ssd.SAMPLE_IID
    for seed in range(3):
        path, plen, nxt = s.accept(toks, par, torch.from_numpy(lg).cuda(), mode=md,
                                   draft_probs=torch.from_numpy(q).cuda(), temperature=1.0, seed=seed)
        op, on = oracle.tree_accept(oracle.SAMPLE_WOR if mode == "wor" else oracle.SAMPLE_IID, toks, par, lg, q,
                                    1.0, seed)
        assert op.tolist() == [0] and on == 7
        assert path[:int(plen.item())].cpu().numpy().tolist() == [0] and int(nxt.item()) == 7


def test_session_options_validate_and_stay_per_session(tiny16, ssd, torch):
    t = tiny16
    default = {"pass_mode": ssd.PASS_AUTO, "gemm_path": ssd.GEMM_AUTO, "weight_prefetch": 1}
    assert t.s.get_options() == default
    for bad in (dict(pass_mode=3), dict(gemm_path=-1), dict(weight_prefetch=2)):
        with pytest.raises(ssd.SSDError) as e:
            t.s.set_options(**bad)
        assert e.value.status == ssd.E_INVALID_ARG
    assert t.s.get_options() == default
    other = ssd.Session(t.m, 16, 4)
    with t.s.options(pass_mode=ssd.PASS_KERNELS, gemm_path=ssd.GEMM_VEC, weight_prefetch=0):
        assert t.s.get_options() == {"pass_mode": 1, "gemm_path": 1, "weight_prefetch": 0}
        assert other.get_options() == default
    assert t.s.get_options() == default
    other.close()


def test_float16_range_is_checked(ssd, torch):
    """The matrix cores take float16 copies of bf16 weights and float16 GEMM
    inputs: a weight past 65504 is refused at model creation, and a GEMM
    input past it is counted in the session's error counter."""
    cfg = W.TINY.with_(dtype="bf16", n_layer=1)
    w = W.make_weights(cfg, 0)
    big = W.f32_to_bf16_bits(np.array([1e5], np.float32))[0]
    w2 = dict(w)
    w2["w_fc"] = [w["w_fc"][0].copy()]
    w2["w_fc"][0][3, 5] = big
    with pytest.raises(ssd.SSDError) as e:
        ssd.Model(cfg, w2)
    assert e.value.status == ssd.E_UNSUPPORTED
    w3 = dict(w)
    w3["ln1_g"] = [W.f32_to_bf16_bits(np.full(cfg.d_model, 1e5, np.float32))]
    m = ssd.Model(cfg, w3)
    s = ssd.Session(m, 16, 4)
    assert s.error_count() == 0
    s.verify(0, [1, 2], [-1, 0])
    assert s.error_count() > 0
    s.close()


@pytest.mark.slow
def test_attention_largest_prefix_chunk(ssd, torch):
    """The one-kernel-per-sub-layer attention at its largest chunk: 32 heads
    over a 2000-token prefix make the chunk 256 cache rows (8 per head), the
    most the split kernel stages; every logit of a 20-node tree against the
    oracle (2e-2), and the greedy walk on them."""
    cfg = W.GPT2Config(n_layer=1, d_model=2048, n_head=32, d_mlp=256, vocab=512, n_pos=2100, dtype="bf16")
    w = W.make_weights(cfg, 4, perturb_affine=True)
    P = 2000
    kc, vc = W.random_kv_cache(cfg, P + 32, P, seed=9)
    m = ssd.Model(cfg, w)
    s = ssd.Session(m, P + 32, 32, ssd.to_device(kc, cfg), ssd.to_device(vc, cfg))
    par = W.branching_tree([4, 2, 2, 1], 20)
    toks = W.tree_tokens(par, cfg.vocab, seed=3)
    with s.options(pass_mode=ssd.PASS_KERNELS):
        lg = s.verify(P, toks, par)
        path, plen, nxt = s.accept(toks, par, lg)
        torch.cuda.synchronize()
    assert s.error_count() == 0
    om = oracle.Model(cfg, w)
    ref = oracle.tree_verify(om, kc, vc, P, toks, par, om.kv(32), om.kv(32))
    got = lg.cpu().numpy()
    assert np.abs(got - ref).max() < 2e-2
    op, on = oracle.tree_accept(oracle.GREEDY, toks, par, got)
    assert path[:int(plen.item())].cpu().tolist() == op.tolist() and int(nxt.item()) == on
    s.close()
    m.close()


@pytest.mark.parametrize("V", [512, 50257])
@pytest.mark.parametrize("mode", ["wor", "iid", "det"])
@pytest.mark.parametrize("k", [1, 50])
def test_sampling_accept_topk_and_chosen_siblings_bit_exact(wide, ssd, torch, V, mode, k):
    """Top-k targets (Sec. 4's k = 50, T = 1; ties at the cut to the lower id,
    here made likely by rounding the logits) and siblings chosen rather than
    drawn (the draft's top tokens; no draft rows): path and extra token
    bit-exact against the oracle on identical logits."""
    cfg, s = wide
    g = np.random.default_rng(V + k + len(mode))
    md = {"wor": ssd.SAMPLE_WOR, "iid": ssd.SAMPLE_IID, "det": ssd.SAMPLE_DET}[mode]
    omd = {"wor": oracle.SAMPLE_WOR, "iid": oracle.SAMPLE_IID, "det": oracle.SAMPLE_DET}[mode]
    for trial in range(8):
        toks, par = _draft_tree(g, V, [4, 2, 2, 1], 32 if trial % 2 else 120)
        n = len(par)
        lg = np.round(g.standard_normal((n, V)) * 2.0, 1).astype(np.float32)
        q = g.dirichlet(np.ones(V) * 0.3, size=n).astype(np.float32)
        for c in range(1, n):
            if g.random() < 0.7:     # the target's top tokens, so paths get long
                toks[c] = int(np.lexsort((np.arange(V), -lg[par[c]]))[int(g.integers(0, min(k, 4)))])
        dlg = torch.from_numpy(lg).cuda()
        dq = None if mode == "det" else torch.from_numpy(q).cuda()
        path, plen, nxt = s.accept(toks, par, dlg, mode=md, draft_probs=dq, temperature=1.0, seed=trial, top_k=k)
        op, on = oracle.tree_accept(omd, toks, par, lg, None if mode == "det" else q, 1.0, trial, top_k=k)
        assert path[:int(plen.item())].cpu().numpy().tolist() == op.tolist(), trial
        assert int(nxt.item()) == on, trial
        if k == 1:   # the target is the argmax: every emitted token is one
            assert on == int(np.lexsort((np.arange(V), -lg[op[-1]]))[0])


from tests.test_oracle_sampling_variants import topk_target  # noqa: E402


def _cdf_pick_host(w, U):
    """Smallest id whose running sum (ascending id) exceeds U (else the last
    positive id): the test's own inverse CDF, for building trees."""
    c = np.cumsum(np.asarray(w, np.float64))
    i = int(np.searchsorted(c, U, side="right"))
    return i if i < len(w) else int(np.flatnonzero(np.asarray(w) > 0)[-1])


def _cdf_first_tree(lg_rows_for, V, seed, branching, n_max, ssd, offsets=(0.0, 0.1, -0.1)):
    """CDF-first assembly (breadth first, indices in creation order): node
    u's children are the inverse-CDF picks of a draft row at U_u + offsets,
    U_u = ssd_uniform(seed, 2, u) read on the host before the tree exists;
    the draft row of node u is lg_rows_for(u, token)."""
    toks, par, frontier = [int(lg_rows_for.root)], [-1], [0]
    for b in branching:
        nxt = []
        for u in frontier:
            q = lg_rows_for(u, toks[u])
            U = ssd.uniform(seed, 2, u)
            kids = []
            for o in offsets:
                x = _cdf_pick_host(q, (U + o) % 1.0)
                if x not in kids:
                    kids.append(x)
            for x in kids[:b]:
                if len(toks) < n_max:
                    toks.append(x)
                    par.append(u)
                    nxt.append(len(toks) - 1)
        frontier = nxt
    return np.array(toks, np.int32), np.array(par, np.int32)


@pytest.mark.parametrize("V", [512, 50257])
@pytest.mark.parametrize("k,T", [(0, 1.0), (50, 1.0), (0, 0.7)])
def test_sampling_accept_cdf_first_bit_exact(wide, ssd, torch, V, k, T):
    """CDF-first sampling (uniforms drawn before the tree is built, the
    oracle's token by inverse CDF at each node's uniform): trees assembled
    around the uniforms from a draft close to the target (so walks go deep),
    path and extra token bit-exact against the oracle on identical logits."""
    cfg, s = wide
    g = np.random.default_rng(V + k)
    deep = 0
    for trial in range(8):
        n_max = 40 if trial % 2 else 200
        lg = np.round(g.standard_normal((n_max, V)) * 2.0, 1).astype(np.float32)
        # node u's draft row: the target row u itself (even trials: the
        # draft's pick at U_u is the oracle's token but for rounding, so the
        # walks go deep) or the target of slightly perturbed logits
        noise = 0.0 if trial % 2 == 0 else 0.05
        dl = lg + (g.standard_normal(lg.shape) * noise).astype(np.float32)

        def rows(u, tok):
            return topk_target(dl[u], k, T)
        rows.root = int(g.integers(V))
        toks, par = _cdf_first_tree(rows, V, trial, [3, 2, 2, 2, 1, 1], n_max, ssd)
        n = len(par)
        dlg = torch.from_numpy(np.ascontiguousarray(lg[:n])).cuda()
        path, plen, nxt = s.accept(toks, par, dlg, mode=ssd.SAMPLE_CDF, temperature=T, seed=trial, top_k=k)
        op, on = oracle.tree_accept(oracle.SAMPLE_CDF, toks, par, lg[:n], None, T, trial, top_k=k)
        assert path[:int(plen.item())].cpu().numpy().tolist() == op.tolist(), trial
        assert int(nxt.item()) == on, trial
        deep += len(op) - 1
    assert s.error_count() == 0
    assert deep >= 8          # the walks follow the assembled trees
    # draft rows are refused in this mode
    with pytest.raises(ssd.SSDError):
        s.accept([0, 1], [-1, 0], dlg[:2], mode=ssd.SAMPLE_CDF, draft_probs=dlg[:2])


@pytest.mark.parametrize("V", [512, 50257])
@pytest.mark.parametrize("T", [1.0, 0.7])
def test_cdf_pick_bit_exact(wide, ssd, torch, V, T):
    """ssd_cdf_pick (the draft's inverse-CDF picks for CDF-first assembly)
    against the oracle's pick: 64 queries over 40 rows, tokens equal."""
    cfg, s = wide
    g = np.random.default_rng(V + int(T * 10))
    lg = np.round(g.standard_normal((40, V)) * 2.0, 1).astype(np.float32)
    rows = g.integers(0, 40, 64).astype(np.int32)
    us = g.random(64)
    us[:3] = [0.0, 0.999999999, 0.5]
    dlg = torch.from_numpy(lg).cuda()
    got = s.cdf_pick(dlg, rows, us, T).cpu().numpy()
    want = [oracle.cdf_pick(lg[r], T, u) for r, u in zip(rows, us)]
    assert got.tolist() == want
    for bad in (dict(rows=[40], us=[0.5]), dict(rows=[0], us=[1.0]), dict(rows=[0], us=[-0.1]),
                dict(rows=list(range(65)), us=[0.5] * 65)):
        with pytest.raises(ssd.SSDError):
            s.cdf_pick(dlg, np.array(bad["rows"]) % 65, bad["us"], T, n_rows=40)
