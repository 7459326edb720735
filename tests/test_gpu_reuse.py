"""The oracle pass reusing the draft's work (ssd_tree_reuse +
ssd_tree_verify_from), through the C ABI.  The draft is a layer prefix of
the oracle (ssd_model_prefix_view), so its residual stream after its last
layer and its layers' K/V are exactly what the oracle computes for the same
nodes; the oracle pass over an ancestor-closed subset of the draft's tree
may then start at the draft's last layer.

- The persistent pass (head dimension 64, <= 64 nodes): logits from layer
  start_layer equal the full pass over the subset bit for bit (a node's
  arithmetic depends only on its root path), and the oracle's within 2e-2.
- One kernel per sub-layer: the oracle's within 2e-2 and the full pass's
  within 1e-2 (the draft ran over a different node count, so its GEMM
  tiling may differ in the last bits).
- The greedy variant equals the pass then the greedy accept; error paths.
- Staged greedy decoding with reuse emits the plain greedy sequence: on the
  tiny float32 model the oracle's own, token for token.
- GPT-2-L at 32 nodes (4-layer draft): bitwise equal to the full pass.
- The 8-bit weight model (its own start-layer variant of the persistent
  pass): bitwise equal to the full pass, and the oracle's 8-bit mode within
  2e-2, on both paths.
"""
import numpy as np
import pytest

import oracle
from paper_2308_04623_amd import staged as S
from paper_2308_04623_amd import workloads as W
from tests.helpers import draft_weights

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
    return s


class Pair:
    """An oracle model, its first-layers draft view, and two sessions on one cache."""

    def __init__(self, ssd, cfg, n_draft, P=64, max_ctx=160, max_nodes=64, seed=0, q8=False):
        self.cfg, self.P, self.ld = cfg, P, n_draft
        self.w = W.make_weights(cfg, seed, perturb_affine=True)
        self.om = oracle.Model(cfg, self.w, q8=q8)
        self.kc, self.vc = W.random_kv_cache(cfg, max_ctx, P, seed=3)
        self.m = ssd.Model(cfg, self.w, q8=q8)
        self.view = self.m.prefix_view(n_draft)
        self.o = ssd.Session(self.m, max_ctx, max_nodes, ssd.to_device(self.kc, cfg), ssd.to_device(self.vc, cfg))
        self.d = ssd.Session(self.view, max_ctx, max_nodes, self.o.k_cache, self.o.v_cache)
        self.max_nodes = max_nodes

    def oracle_logits(self, toks, par):
        kt, vt = self.om.kv(self.max_nodes), self.om.kv(self.max_nodes)
        return oracle.tree_verify(self.om, self.kc, self.vc, self.P, toks, par, kt, vt)


@pytest.fixture(scope="module")
def small(ssd):
    return Pair(ssd, SMALL, 1)


@pytest.fixture(scope="module")
def small_q8(ssd):
    return Pair(ssd, SMALL, 1, q8=True)


@pytest.fixture(scope="module")
def tiny(ssd):
    return Pair(ssd, W.TINY.with_(dtype="bf16"), 1)


def _tree_and_subset(seed, n):
    g = np.random.default_rng(seed)
    par = np.array([-1] + [int(g.integers(max(0, i - 8), i)) for i in range(1, n)], np.int32)
    keep, pos = [0], {0: 0}
    for i in range(1, n):
        if int(par[i]) in pos and g.random() < 0.7:
            pos[i] = len(keep)
            keep.append(i)
    sub_par = np.array([-1] + [pos[int(par[i])] for i in keep[1:]], np.int32)
    return par, np.array(keep, np.int32), sub_par


def _run(pair, ssd, torch, mode, seed, n):
    par, keep, sub_par = _tree_and_subset(seed, n)
    toks = W.tree_tokens(par, pair.cfg.vocab, seed=seed)
    sub_toks = toks[keep]
    with pair.o.options(pass_mode=mode), pair.d.options(pass_mode=mode):
        pair.d.verify(pair.P, toks, par)
        x = pair.d.reuse_into(pair.o, keep)
        lg_r = pair.o.verify_from(pair.P, sub_toks, sub_par, pair.ld, x).clone()
        lg_g, path, plen, nxt = pair.o.verify_from(pair.P, sub_toks, sub_par, pair.ld, x, greedy=True)
        lg_f = pair.o.verify(pair.P, sub_toks, sub_par).clone()
        torch.cuda.synchronize()
    assert pair.o.error_count() == 0 and pair.d.error_count() == 0
    return sub_toks, sub_par, lg_r, lg_g, (path, plen, nxt), lg_f


@pytest.mark.parametrize("seed,n", [(1, 20), (2, 48), (3, 64)])
def test_reuse_persistent_pass_is_bitwise_the_full_pass(small, ssd, torch, seed, n):
    t, p, lg_r, lg_g, (path, plen, nxt), lg_f = _run(small, ssd, torch, ssd.PASS_FUSED, seed, n)
    assert torch.equal(lg_r, lg_f)
    assert torch.equal(lg_g, lg_r)
    got = lg_r.cpu().numpy()
    assert np.abs(got - small.oracle_logits(t, p)).max() < TOL
    op, on = oracle.tree_accept(oracle.GREEDY, t, p, got)
    assert path[:int(plen.item())].cpu().tolist() == op.tolist() and int(nxt.item()) == on


@pytest.mark.parametrize("pair_name", ["small", "tiny"])
def test_reuse_per_sub_layer_path(small, tiny, ssd, torch, pair_name):
    pair = small if pair_name == "small" else tiny
    t, p, lg_r, lg_g, (path, plen, nxt), lg_f = _run(pair, ssd, torch, ssd.PASS_KERNELS, 4, 40)
    got = lg_r.cpu().numpy()
    assert np.abs(got - pair.oracle_logits(t, p)).max() < TOL
    assert np.abs(got - lg_f.cpu().numpy()).max() < 1e-2
    assert torch.equal(lg_g, lg_r)
    op, on = oracle.tree_accept(oracle.GREEDY, t, p, got)
    assert path[:int(plen.item())].cpu().tolist() == op.tolist() and int(nxt.item()) == on


@pytest.mark.parametrize("mode", ["fused", "kernels"])
def test_reuse_q8_model(small_q8, ssd, torch, mode):
    pm = ssd.PASS_FUSED if mode == "fused" else ssd.PASS_KERNELS
    t, p, lg_r, lg_g, (path, plen, nxt), lg_f = _run(small_q8, ssd, torch, pm, 6, 44)
    if mode == "fused":
        assert torch.equal(lg_r, lg_f)
    else:
        assert np.abs(lg_r.cpu().numpy() - lg_f.cpu().numpy()).max() < 1e-2
    assert torch.equal(lg_g, lg_r)
    got = lg_r.cpu().numpy()
    assert np.abs(got - small_q8.oracle_logits(t, p)).max() < TOL
    op, on = oracle.tree_accept(oracle.GREEDY, t, p, got)
    assert path[:int(plen.item())].cpu().tolist() == op.tolist() and int(nxt.item()) == on


def test_reuse_error_paths(small, tiny, ssd, torch):
    pair = small
    par = W.chain_tree(4)
    toks = W.tree_tokens(par, pair.cfg.vocab, seed=1)
    pair.d.verify(pair.P, toks, par)
    x = pair.d.reuse_into(pair.o, [0, 1, 2, 3])
    for start, xi in ((3, x), (-1, x), (1, None)):
        with pytest.raises(ssd.SSDError) as e:
            pair.o.verify_from(pair.P, toks, par, start, xi)
        assert e.value.status == ssd.E_INVALID_ARG
    with pytest.raises(ssd.SSDError):
        pair.o.reuse_into(pair.o, [0])            # same session
    with pytest.raises(ssd.SSDError):
        pair.d.reuse_into(pair.o, [pair.max_nodes])   # row outside the source session
    with pytest.raises(ssd.SSDError):
        pair.d.reuse_into(pair.o, [0, 4])             # row outside the source's last pass (4 nodes)
    with pytest.raises(ssd.SSDError):
        pair.d.reuse_into(tiny.o, [0])            # another model's shape
    with pytest.raises(ssd.SSDError):
        pair.d.reuse_into(pair.o, list(range(257)))
    fresh = ssd.Session(pair.view, 160, 64, pair.o.k_cache, pair.o.v_cache)
    with pytest.raises(ssd.SSDError) as e:                  # no pass ran on the source yet
        fresh.reuse_into(pair.o, [0])
    assert e.value.status == ssd.E_INVALID_ARG
    fresh.close()


def test_staged_reuse_equals_oracle_plain_greedy_tiny_f32(ssd, torch):
    """Staged greedy decoding that reuses the draft's work, on the tiny
    float32 model: the emitted tokens are the oracle's own plain greedy
    sequence, every one (no tie escape), and trees are accepted."""
    from tests.helpers import oracle_prefill
    cfg = W.TINY
    w = W.make_weights(cfg, 0, perturb_affine=True)
    prompt = W.prefix_tokens(40, cfg.vocab, seed=5)
    n_new = 32
    om = oracle.Model(cfg, w)
    kc, vc, _ = oracle_prefill(om, prompt[:-1], 128)
    P, root = len(prompt) - 1, int(prompt[-1])
    kt, vt = om.kv(1), om.kv(1)
    ref = []
    while len(ref) < n_new:
        lg = oracle.tree_verify(om, kc, vc, P, [root], [-1], kt, vt)
        path, nxt = oracle.tree_accept(oracle.GREEDY, [root], [-1], lg)
        oracle.kv_commit(om, kc, vc, P, kt, vt, path)
        P += 1
        ref.append(nxt)
        root = nxt
    m = ssd.Model(cfg, w)
    view = m.prefix_view(1)
    o = ssd.Session(m, 128, 64)
    d = ssd.Session(view, 128, 64, o.k_cache, o.v_cache)
    b = S.GpuBackend(o, d)
    P0 = b.prefill(prompt[:-1])
    stream = S.bigram_stream(cfg.vocab, 2048, seed=4)
    preds = np.concatenate([b.greedy_predictions(stream[i:i + 64]) for i in range(0, 2048, 64)])
    succ = S.bigram_table(stream, preds, cfg.vocab)
    st = S.staged_greedy_reuse(b, P0, int(prompt[-1]), n_new, succ)
    assert st.tokens == ref
    assert sum(st.accepted) > 0
    assert o.error_count() == 0 and d.error_count() == 0


@pytest.mark.slow
def test_reuse_gpt2l_32_nodes_bitwise(ssd, torch):
    cfg = W.GPT2L
    w = W.make_weights(cfg, 0)
    m = ssd.Model(cfg, w)
    view = m.prefix_view(4)
    kc, vc = W.random_kv_cache(cfg, 576, 512, seed=3)
    o = ssd.Session(m, 576, 64, ssd.to_device(kc, cfg), ssd.to_device(vc, cfg))
    d = ssd.Session(view, 576, 64, o.k_cache, o.v_cache)
    toks, par = W.best_first_tree(48, seed=3, vocab=cfg.vocab)
    toks[0] = 17
    keep = np.arange(32, dtype=np.int32)            # a best-first tree's first nodes are ancestor-closed
    assert all(int(par[i]) < i for i in keep[1:])
    d.verify(512, toks, par)
    x = d.reuse_into(o, keep)
    lg_r = o.verify_from(512, toks[keep], par[keep], 4, x).clone()
    lg_f = o.verify(512, toks[keep], par[keep]).clone()
    torch.cuda.synchronize()
    assert o.verify_path(32) == ssd.PASS_FUSED
    assert torch.equal(lg_r, lg_f)
    assert o.error_count() == 0 and d.error_count() == 0
