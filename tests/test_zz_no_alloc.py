"""The allocation-free accept entry point (ssd_tree_accept_noalloc) against
ssd_tree_accept on the same device logits, through the C ABI: greedy and
every sampling mode, bit-exact paths and tokens, on two calls in a row
(the second with fewer nodes and a smaller vocabulary, so the shared
scratch holds a larger call's leftovers), plus its limits."""
import numpy as np
import pytest

from paper_2308_04623_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_2308_04623_amd import ssd
    assert torch.cuda.is_available()
    cfg = W.TINY.with_(vocab=50257, n_layer=1)
    m = ssd.Model(cfg, W.make_weights(cfg, 1))
    s = ssd.Session(m, 8, 256)
    return torch, ssd, s


def _outs(torch, n):
    return (torch.full((n,), -7, dtype=torch.int32, device="cuda"), torch.zeros(1, dtype=torch.int32, device="cuda"),
            torch.zeros(1, dtype=torch.int32, device="cuda"))


def _case(g, n, V, greedy_hint):
    par = W.branching_tree([4, 2, 2, 1], n)
    lg = (g.standard_normal((n, V)) * 2.0).astype(np.float32)
    q = g.dirichlet(np.ones(V) * 0.3, size=n).astype(np.float32)
    e = np.exp(lg - lg.max(1, keepdims=True))
    q = (0.5 * q + 0.5 * e / e.sum(1, keepdims=True)).astype(np.float32)
    toks = g.integers(0, V, n).astype(np.int32)
    for c in range(1, n):
        if g.random() < 0.7:
            toks[c] = int(np.argmax(lg[par[c]])) if greedy_hint else int(np.argmax(lg[par[c]] + g.gumbel(size=V)))
    return toks, par, lg, q


@pytest.mark.parametrize("mode", ["greedy", "wor", "iid", "det", "cdf"])
def test_noalloc_accept_equals_session_accept(env, mode):
    torch, ssd, s = env
    md = {"greedy": ssd.GREEDY, "wor": ssd.SAMPLE_WOR, "iid": ssd.SAMPLE_IID, "det": ssd.SAMPLE_DET,
          "cdf": ssd.SAMPLE_CDF}[mode]
    top_k = 50 if mode in ("det", "cdf") else 0
    g = np.random.default_rng(len(mode))
    for call, (n, V) in enumerate([(256, 50257), (24, 3000)]):
        print(f"noalloc {mode} call {call}: n={n} V={V}", flush=True)
        toks, par, lg, q = _case(g, n, V, mode == "greedy")
        dlg = torch.from_numpy(lg).cuda()
        dq = None if mode in ("greedy", "det", "cdf") else torch.from_numpy(q).cuda()
        a = s.accept(toks, par, dlg, mode=md, draft_probs=dq, temperature=1.0, seed=call, top_k=top_k)
        b = ssd.accept_noalloc(toks, par, dlg, _outs(torch, n), mode=md, draft_probs=dq, temperature=1.0, seed=call,
                               top_k=top_k)
        torch.cuda.synchronize()
        la, lb = int(a[1].item()), int(b[1].item())
        assert la == lb, (call, la, lb)
        assert a[0][:la].cpu().tolist() == b[0][:lb].cpu().tolist(), call
        assert int(a[2].item()) == int(b[2].item()), call


def test_noalloc_accept_limits(env):
    torch, ssd, s = env
    lg = torch.zeros((257, 10), device="cuda")
    par = W.chain_tree(257)
    with pytest.raises(ssd.SSDError) as e:
        ssd.accept_noalloc(np.zeros(257, np.int32), par, lg, _outs(torch, 257))
    assert e.value.status == ssd.E_CAPACITY
    wide = torch.zeros((2, 65537), device="cuda")
    with pytest.raises(ssd.SSDError) as e:
        ssd.accept_noalloc([0, 1], [-1, 0], wide, _outs(torch, 2))
    assert e.value.status == ssd.E_CAPACITY
    with pytest.raises(ssd.SSDError) as e:
        ssd.accept_noalloc([0, 1], [0, 0], torch.zeros((2, 10), device="cuda"), _outs(torch, 2))
    assert e.value.status == ssd.E_INVALID_TREE
