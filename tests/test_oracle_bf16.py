"""Pins of the oracle's bfloat16 storage mode (no GPU).

Sec. 3.1 keeps the batch's K/V apart and later appends the accepted rows to
the cache.  In a bfloat16 model every parameter and every K/V row is stored
in bfloat16, so the K/V a node produces are rounded to bfloat16 when they are
written, and every attention that reads them (the node's own included) sees
the rounded values.  These tests pin that mode against things other than the
oracle itself:

- Library routine: transformers' GPT2LMHeadModel in float64, loaded with the
  bfloat16 weights widened exactly (bits shifted into a float32 here), and a
  forward hook on each attention input projection that rounds its K and V
  thirds to bfloat16 (nearest-even, straight from float64) before attention
  reads them.
- Closed form: with W_q = 0 every score is equal, so attention returns the
  mean of the visible values; in bfloat16 mode those are rounded values.
- Power check: copies of the oracle with a planted mistake (a wrong widening
  shift, K/V rounded only after the node's own attention used them,
  truncation instead of nearest-even) must fail the library comparison.
"""
import numpy as np
import pytest

import oracle
from paper_2308_04623_amd import workloads as W
from tests.helpers import oracle_prefill, root_path

CFG = W.TINY.with_(dtype="bf16")
P = 48
TOL = 1e-5  # float64 on both sides; the oracle rounds logits to float32 at output


def widen(bits):
    """bfloat16 bit patterns -> float64, exactly (the pattern is the top half of a float32)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def round_bf16(x):
    """float64 -> float64 holding the nearest-even bfloat16 value, with one
    rounding: round to float32 first, then to bfloat16 on the bit pattern,
    except that a float32 result sitting exactly halfway between two bfloat16
    values which is not x itself was made a tie by the first rounding, so it
    goes towards x instead of to even."""
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)
    u = f.view(np.uint32)
    low = u & np.uint32(0xFFFF)
    hi = u >> np.uint32(16)
    fd = f.astype(np.float64)
    fake_tie = (low == 0x8000) & (fd != x)
    up_tie = np.where(fake_tie, np.abs(x) > np.abs(fd), (hi & np.uint32(1)) == 1)
    up = (low > 0x8000) | ((low == 0x8000) & up_tie)
    r = (hi + up.astype(np.uint32)) << np.uint32(16)
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def test_round_bf16_helper_against_exact_cases():
    one = 1.0
    assert round_bf16(one + 2.0 ** -8) == one                       # tie -> even (down)
    assert round_bf16(one + 3 * 2.0 ** -8) == one + 2 * 2.0 ** -7   # tie -> even (up)
    assert round_bf16(one + 2.0 ** -8 + 2.0 ** -40) == one + 2.0 ** -7  # just above the tie
    # the float32 rounding of this value lands exactly on the tie: single rounding goes down
    x = one + 2.0 ** -8 - 2.0 ** -30
    assert np.float32(x) == np.float32(one + 2.0 ** -8)
    assert round_bf16(x) == one
    assert round_bf16(-(one + 3 * 2.0 ** -8)) == -(one + 2 * 2.0 ** -7)
    # agrees with the oracle's own rounding on random values (both pinned here)
    g = np.random.default_rng(0)
    xs = g.standard_normal(2000) * 10.0 ** g.uniform(-6, 3, 2000)
    for v in xs[:300]:
        assert widen(oracle.round_bf16(float(v))) == round_bf16(v), v


def _hf_bf16(w, cfg):
    torch = pytest.importorskip("torch")
    tr = pytest.importorskip("transformers")
    hc = tr.GPT2Config(vocab_size=cfg.vocab, n_positions=cfg.n_pos, n_embd=cfg.d_model, n_layer=cfg.n_layer,
                       n_head=cfg.n_head, n_inner=cfg.d_mlp, activation_function="gelu_new",
                       layer_norm_epsilon=cfg.ln_eps, resid_pdrop=0.0, embd_pdrop=0.0, attn_pdrop=0.0,
                       tie_word_embeddings=True)
    hf = tr.GPT2LMHeadModel(hc)
    hf.config._attn_implementation = "eager"
    sd = {"transformer.wte.weight": w["wte"], "transformer.wpe.weight": w["wpe"],
          "transformer.ln_f.weight": w["lnf_g"], "transformer.ln_f.bias": w["lnf_b"]}
    for l in range(cfg.n_layer):
        pre = f"transformer.h.{l}."
        sd.update({pre + "ln_1.weight": w["ln1_g"][l], pre + "ln_1.bias": w["ln1_b"][l],
                   pre + "attn.c_attn.weight": np.asarray(w["w_qkv"][l]).T, pre + "attn.c_attn.bias": w["b_qkv"][l],
                   pre + "attn.c_proj.weight": np.asarray(w["w_o"][l]).T, pre + "attn.c_proj.bias": w["b_o"][l],
                   pre + "ln_2.weight": w["ln2_g"][l], pre + "ln_2.bias": w["ln2_b"][l],
                   pre + "mlp.c_fc.weight": np.asarray(w["w_fc"][l]).T, pre + "mlp.c_fc.bias": w["b_fc"][l],
                   pre + "mlp.c_proj.weight": np.asarray(w["w_pr"][l]).T, pre + "mlp.c_proj.bias": w["b_pr"][l]})
    sd = {k: torch.from_numpy(np.ascontiguousarray(widen(v))) for k, v in sd.items()}
    hf = hf.double()
    missing, unexpected = hf.load_state_dict(sd, strict=False)
    assert not unexpected
    hf.lm_head.weight = hf.transformer.wte.weight
    d = cfg.d_model

    def round_kv(_mod, _inp, out):
        a = out.detach().numpy().copy()
        a[..., d:] = round_bf16(a[..., d:])
        return torch.from_numpy(a)

    for blk in hf.transformer.h:
        blk.attn.c_attn.register_forward_hook(round_kv)
    return hf.eval()


def _hf_logits(hf, seq):
    import torch
    with torch.no_grad():
        return hf(torch.tensor(np.asarray(seq, dtype=np.int64))[None]).logits[0].numpy()


@pytest.fixture(scope="module")
def setup():
    w = W.make_weights(CFG, 0, perturb_affine=True)
    return w, _hf_bf16(w, CFG)


def _oracle_causal(m, seq):
    kt, vt = m.kv(len(seq)), m.kv(len(seq))
    return oracle.tree_verify(m, None, None, 0, seq, W.chain_tree(len(seq)), kt, vt)


def _oracle_tree_rows(m, prefix, toks, parents):
    kc, vc, _ = oracle_prefill(m, prefix, 96)
    kt, vt = m.kv(len(parents)), m.kv(len(parents))
    return oracle.tree_verify(m, kc, vc, len(prefix), toks, parents, kt, vt)


def test_bf16_causal_logits_match_transformers(setup):
    w, hf = setup
    m = oracle.Model(CFG, w)
    seq = W.prefix_tokens(40, CFG.vocab, seed=11)
    got = _oracle_causal(m, seq)
    ref = _hf_logits(hf, seq)
    err = np.abs(got - ref).max()
    assert err < TOL, err


def test_bf16_tree_rows_match_transformers_on_root_paths(setup):
    w, hf = setup
    m = oracle.Model(CFG, w)
    prefix = W.prefix_tokens(P, CFG.vocab, seed=1)
    parents = W.complete_binary_tree(15)
    toks = W.tree_tokens(parents, CFG.vocab, seed=2)
    lg = _oracle_tree_rows(m, prefix, toks, parents)
    for i in range(15):
        ref = _hf_logits(hf, np.concatenate([prefix, toks[root_path(parents, i)]]))[-1]
        assert np.abs(lg[i] - ref).max() < TOL, i


def test_bf16_uniform_attention_closed_form():
    """W_q = 0 and the MLP off: attention is the mean of the visible values,
    the tree's own values rounded to bfloat16 as produced, and the logits
    follow in closed form."""
    cfg = CFG.with_(n_layer=1)
    w = W.make_weights(cfg, 0, perturb_affine=True)
    d, H, dh = cfg.d_model, cfg.n_head, cfg.head_dim
    zero = np.uint16(0)
    w["w_qkv"][0][:d] = zero
    w["b_qkv"][0][:d] = zero
    w["w_fc"][0][:] = zero
    w["b_fc"][0][:] = zero
    w["b_pr"][0][:] = zero
    m = oracle.Model(cfg, w)
    Pp = 5
    kc, vc = W.random_kv_cache(cfg, 16, Pp, seed=3)
    parents = np.array([-1, 0, 0, 1, 3], dtype=np.int32)
    toks = np.array([7, 100, 200, 300, 400], dtype=np.int32)
    lg = oracle.tree_verify(m, kc, vc, Pp, toks, parents, m.kv(8), m.kv(8))

    def ln(x, g, b):
        mu = x.mean(-1, keepdims=True)
        var = ((x - mu) ** 2).mean(-1, keepdims=True)
        return (x - mu) / np.sqrt(var + cfg.ln_eps) * widen(g) + widen(b)

    depth = [0, 1, 1, 2, 3]
    emb = np.stack([widen(w["wte"][toks[i]]) + widen(w["wpe"][Pp + depth[i]]) for i in range(5)])
    a = ln(emb, w["ln1_g"][0], w["ln1_b"][0])
    v_tree = round_bf16(a @ widen(w["w_qkv"][0][2 * d:]).T + widen(w["b_qkv"][0][2 * d:]))
    for i in range(5):
        vis = root_path(parents, i)
        o = np.zeros(d)
        for h in range(H):
            vals = np.concatenate([widen(vc[0, h, :Pp]), v_tree[vis][:, h * dh:(h + 1) * dh]], 0)
            o[h * dh:(h + 1) * dh] = vals.mean(0)
        x = emb[i] + o @ widen(w["w_o"][0]).T + widen(w["b_o"][0])
        want = ln(x, w["lnf_g"], w["lnf_b"]) @ widen(w["wte"]).T
        assert np.abs(lg[i] - want).max() < 1e-5, i


# planted mistakes: each must make the library comparison fail
MUTANTS = {
    "widening_shift_15": [("uint32_t u = (uint32_t)h << 16;", "uint32_t u = (uint32_t)h << 15;")],
    "kv_rounded_after_own_use": [
        ("          for (int32_t j = 0; j < dh; ++j) dot += q[j] * ld(K, row * dh + j, dt);",
         "          const double *qi = qkv + (size_t)i * 3 * d + d + h * dh;\n"
         "          for (int32_t j = 0; j < dh; ++j)\n"
         "            dot += q[j] * (t == nk - 1 ? qi[j] : ld(K, row * dh + j, dt));"),
        ("            acc += s[t] * ld(Vs, row * dh + j, dt);",
         "            acc += s[t] * (t == nk - 1 ? qkv[(size_t)i * 3 * d + 2 * d + h * dh + j]\n"
         "                                         : ld(Vs, row * dh + j, dt));"),
    ],
    "truncating_rounding": [("double r = nearbyint(ldexp(ax, -q_exp));", "double r = trunc(ldexp(ax, -q_exp));")],
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_power_check_planted_mistakes_fail(setup, tmp_path, name):
    w, hf = setup
    so = oracle.build_variant(MUTANTS[name], str(tmp_path / name))
    seq = W.prefix_tokens(40, CFG.vocab, seed=11)
    ref = _hf_logits(hf, seq)
    with oracle.variant(so):
        m = oracle.Model(CFG, w)
        got = _oracle_causal(m, seq)
    err = np.abs(got - ref).max()
    assert err > 20 * TOL, (name, err)
