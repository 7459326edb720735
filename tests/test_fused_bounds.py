"""Host-side bounds check of the persistent pass's memory accesses (no GPU).

The persistent single-launch pass reads its work split from a plan table
(ssd_fused_plan, computed on the host) and derives every global and LDS
address from it, the model shape, the node count N, the prefix length P and
the session's capacities.  This test replays, for every workgroup and every
stage, the largest and smallest index each access can form (the same
expressions as the kernel's, written out per access) on the real plan
tables, and checks them against the sizes of the buffers the session
allocates, for the small test model, the GPT-2-L shape and GPT-2-sized
variants, N = 1..64 and prefixes 0 to 5000; it also checks that the ranks of
every XCD are dealt each of its attention units exactly once.  A plan or
layout change that lets any access leave its allocation fails here, on the
CPU, before a kernel runs.
"""
import numpy as np
import pytest

from paper_2308_04623_amd import ssd

# constants of the pass (ssd_internal.h / fused.hip)
XCD, RANKS, GROUPS, MAXN = 8, 32, 256, 64
ATT_ROWS, AREC, DH, PATH32 = 256, 68, 64, 32
PL_ATT, PL_QKV, PL_WO, PL_FC, PL_WPR, PL_HEAD = 0, 9, 14, 19, 24, 29
LDS_LIMIT = 160 * 1024
NTH, NWV, QW = 512, 8, 4
A_KV = 2 * ATT_ROWS * (DH + 8) * 2
A_RV = 2 * NWV * 32 * (DH + 8) * 2
A_REGION = max(A_KV, A_RV)
A_PART = NWV * 16 * AREC * 4
A_Q = NWV * 2 * DH * 4
WST = 16 * 1024
WST_FRAGS = (73728 + 34816 + 4096 - WST) // 1024
WO_FRAGS = 24
LW_SLOTS = 12
PLAN_STRIDE = 32


class Check:
    def __init__(self):
        self.bad = []

    def rng(self, what, lo, hi, size):
        """Indices lo..hi (inclusive) must lie in [0, size)."""
        if lo < 0 or hi >= size:
            self.bad.append(f"{what}: [{lo}, {hi}] outside [0, {size})")


def act_index(n, k, ld):
    """st_act / st_act4 element index (fragment order)."""
    f = (n >> 4) * ld + (k >> 5)
    return f * 512 + ((n & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7)


def lds_bytes(L):
    return A_REGION + A_PART + A_Q + 128 + PLAN_STRIDE * 4 + L * LW_SLOTS * 8 + WO_FRAGS * 1024


def check_pass(H, d, M, V, L, N, P, max_ctx, max_nodes, q8=False):
    """q8: 8-bit weights (fragments of 512 B, indexed in 8-byte lane slots
    like the float16 ones in 16-byte slots, followed by one float32 scale per
    row of the 16-row blocks; staged into LDS by two 4-byte copies each)."""
    c = Check()
    FB = 512 if q8 else 1024                        # fragment bytes
    nt = (N + 15) // 16
    NT = 1 if nt == 1 else 2 if nt == 2 else 4          # the kernel template serving nt tiles
    tab, xh, xf = ssd.fused_plan(H, d, M, V, nt)
    KCd, KCm, RBd = d // 32, M // 32, d // 16
    att_parts = (max_ctx + ATT_ROWS - 1) // ATT_ROWS + 1
    S = (P + ATT_ROWS - 1) // ATT_ROWS
    sizes = {
        "xr": XCD * MAXN * d, "q": MAXN * d, "act": XCD * MAXN * d, "fo": MAXN * d, "ff": MAXN * M,
        "apart": H * 4 * att_parts * 16 * AREC, "tile_ctr": H * 4, "xacc": 3 * MAXN * d,
        "logits": N * V, "kvt": L * H * max_nodes * DH, "kvc": L * H * max_ctx * DH,
        "w_qkv": (3 * d // 16) * KCd * 64, "w_o": RBd * KCd * 64, "w_fc": (M // 16) * KCd * 64,
        "w_pr": RBd * KCm * 64, "head": ((V + 15) // 16) * KCd * 64,
        "tree": 5 * max_nodes + max_nodes * PATH32 + max_nodes * (max_nodes + 1) // 2,
    }
    c.rng("LDS size", 0, lds_bytes(L) - 1, LDS_LIMIT + 1)
    c.rng("GEMM reduction below the staged weights", 0, (QW - 1) * 64 * 16 * 4 - 1 + 0, WST + 1)
    for x in range(XCD):
        act_base = x * MAXN * d
        kh0, kh1 = 2 * xh[2 * x], 2 * xh[2 * x + 1]
        kf0, kf1 = xf[2 * x], xf[2 * x + 1]
        nhx = xh[2 * x + 1] - xh[2 * x]
        n_attu = nhx * nt * (S + 1)
        dealt = []
        for r in range(RANKS):
            row = tab[x * RANKS + r]
            tag = f"x{x} r{r}"
            # LayerNorm rows r, r + 32 below N: x row, fixed-point sum row of
            # each buffer, this XCD's eighth of the columns cleared, act row
            for n in (r, r + RANKS):
                if n >= N:
                    continue
                c.rng(f"{tag} xr row", (x * MAXN + n) * d, (x * MAXN + n) * d + d - 1, sizes["xr"])
                for b in range(3):
                    c.rng(f"{tag} sum row", (b * MAXN + n) * d, (b * MAXN + n) * d + d - 1, sizes["xacc"])
                    c.rng(f"{tag} cleared columns", (b * MAXN + n) * d + x * (d // 8),
                          (b * MAXN + n) * d + (x + 1) * (d // 8) - 1, sizes["xacc"])
                c.rng(f"{tag} act row", act_base + act_index(n, 0, KCd), act_base + act_index(n, d - 4, KCd) + 3,
                      sizes["act"])
                # a pass from a later layer: the row of the given residual stream [N][d]
                c.rng(f"{tag} x_in row", n * d, n * d + d - 1, N * d)
            # GEMM tasks: weights of each row block, activation fragments of
            # every tile (and the 8-bit copies' row scales)
            for slot, wname, kc0, kc1, KC, actn, rows_out in (
                    (PL_QKV, "w_qkv", 0, KCd, KCd, "act", 3 * d), (PL_WO, "w_o", kh0, kh1, KCd, "fo", d),
                    (PL_FC, "w_fc", 0, KCd, KCd, "act", M), (PL_WPR, "w_pr", kf0, kf1, KCm, "ff", d)):
                nrb = row[slot]
                if nrb == 0:
                    continue
                rbs = row[slot + 1:slot + 1 + nrb]
                c.rng(f"{tag} {wname} row blocks", int(rbs.min()) * 16, int(rbs.max()) * 16 + 15, rows_out)
                if q8:
                    c.rng(f"{tag} {wname} scales", int(rbs.min()) * 16, int(rbs.max()) * 16 + 15,
                          sizes[wname] // (KC * 64) * 16)
                if kc1 > kc0:
                    c.rng(f"{tag} {wname} fragments", (int(rbs.min()) * KC + kc0) * 64,
                          (int(rbs.max()) * KC + kc1 - 1) * 64 + 63, sizes[wname])
                    base = act_base if actn == "act" else 0
                    c.rng(f"{tag} {actn} fragments", base + kc0 * 64 * 8,
                          base + ((NT - 1) * KC + kc1 - 1) * 512 + 511, sizes[actn])
                # epilogue outputs of every node
                o_lo, o_hi = int(rbs.min()) * 16, min(int(rbs.max()) * 16 + 15, rows_out - 1)
                if slot == PL_QKV:
                    for o in (o_lo, o_hi):
                        if o < d:
                            c.rng(f"{tag} q", o, (N - 1) * d + o, sizes["q"])
                        else:
                            h = ((o - d) % d) // DH
                            c.rng(f"{tag} k/v tree row", ((L - 1) * H + h) * max_nodes * DH,
                                  (((L - 1) * H + h) * max_nodes + N - 1) * DH + DH - 1, sizes["kvt"])
                elif slot in (PL_WO, PL_WPR):
                    for b in range(3):
                        c.rng(f"{tag} sum out", (b * MAXN) * d + o_lo, (b * MAXN + N - 1) * d + o_hi, sizes["xacc"])
                elif slot == PL_FC:
                    c.rng(f"{tag} ff out", act_index(0, o_lo, KCm), act_index(N - 1, o_hi, KCm), sizes["ff"])
            # staged weights in LDS
            n_wo, n_wpr = row[PL_WO], row[PL_WPR]
            # (the copies' sources, in 4-byte words: (rb KC + k) FB / 4 + lane
            # (+ 64 for the second half of an 8-bit fragment))
            if NT >= 2 and n_wo > 0 and n_wo * (kh1 - kh0) <= WO_FRAGS:
                ofs = A_REGION + A_PART + A_Q + 256 + L * LW_SLOTS * 8
                c.rng(f"{tag} staged W_o (LDS)", ofs, ofs + n_wo * (kh1 - kh0) * FB - 1, lds_bytes(L))
                rbs = row[PL_WO + 1:PL_WO + 1 + n_wo]
                c.rng(f"{tag} staged W_o sources", (int(rbs.min()) * KCd + kh0) * FB // 4,
                      (int(rbs.max()) * KCd + kh1 - 1) * FB // 4 + FB // 4 - 1, sizes["w_o"] * FB // 4 // 64)
            if NT >= 2 and n_wpr > 0 and n_wpr * (kf1 - kf0) <= WST_FRAGS:
                c.rng(f"{tag} staged W_pr (LDS)", WST, WST + n_wpr * (kf1 - kf0) * FB - 1,
                      A_REGION + A_PART + A_Q)
                rbs = row[PL_WPR + 1:PL_WPR + 1 + n_wpr]
                c.rng(f"{tag} staged W_pr sources", (int(rbs.min()) * KCm + kf0) * FB // 4,
                      (int(rbs.max()) * KCm + kf1 - 1) * FB // 4 + FB // 4 - 1, sizes["w_pr"] * FB // 4 // 64)
            # attention units dealt to this rank
            for u in range(row[PL_ATT], n_attu, RANKS):
                if n_attu <= RANKS:
                    hloc, rem = divmod(u, nt * (S + 1))
                    t, part = divmod(rem, S + 1)
                elif u < nhx * nt:
                    (hloc, t), part = divmod(u, nt), S
                else:
                    hloc, rem = divmod(u - nhx * nt, nt * S)
                    t, part = divmod(rem, S)
                h = xh[2 * x] + hloc
                dealt.append((hloc, t, part))
                c.rng(f"{tag} att head", h, h, H)
                rec = lambda j, nl: ((((h * 4 + t) * (S + 1) + j) * 16 + nl) * AREC)
                c.rng(f"{tag} part record", rec(part, 0), rec(part, 15) + AREC - 1, sizes["apart"])
                c.rng(f"{tag} tile counter", h * 4 + t, h * 4 + t, sizes["tile_ctr"])
                c.rng(f"{tag} merge parts", rec(0, 0), rec(S, 15) + AREC - 1, sizes["apart"])
                n_lo, n_hi = 16 * t, min(16 * t + 15, N - 1)
                c.rng(f"{tag} query rows", n_lo * d + h * DH, n_hi * d + h * DH + DH - 1, sizes["q"])
                c.rng(f"{tag} merged out", act_index(n_lo, h * DH, KCd), act_index(n_hi, h * DH + DH - 1, KCd),
                      sizes["fo"])
                if part < S:
                    cb = part * ATT_ROWS
                    nk = min(ATT_ROWS, P - cb)
                    c.rng(f"{tag} cache rows", cb, cb + nk - 1, P)
                    c.rng(f"{tag} cache K/V", (((L - 1) * H + h) * max_ctx + cb) * DH,
                          (((L - 1) * H + h) * max_ctx + cb + nk - 1) * DH + DH - 1, sizes["kvc"])
                else:
                    c.rng(f"{tag} root-path table", 5 * max_nodes + n_lo * PATH32,
                          5 * max_nodes + n_hi * PATH32 + PATH32 - 1, sizes["tree"])
            # LM head row blocks and logits
            hb0, hb1 = row[PL_HEAD], row[PL_HEAD + 1]
            if hb1 > hb0:
                c.rng(f"{tag} head fragments", hb0 * KCd * 64, (hb1 - 1) * KCd * 64 + KCd * 64 - 1, sizes["head"])
                if q8:
                    c.rng(f"{tag} head scales", hb0 * 16, (hb1 - 1) * 16 + 15, ((V + 15) // 16) * 16)
                c.rng(f"{tag} logits", hb0 * 16, (N - 1) * V + min(hb1 * 16, V) - 1, sizes["logits"])
        want = sorted((hl, tt, pp) for hl in range(nhx) for tt in range(nt) for pp in range(S + 1))
        if sorted(dealt) != want:
            c.bad.append(f"x{x}: attention units dealt {len(dealt)}, not each of {len(want)} once")
    return c.bad


SHAPES = {"small": (4, 256, 1024, 2000, 3), "gpt2l": (20, 1280, 5120, 50257, 36),
          "gpt2m": (16, 1024, 4096, 50257, 24), "gpt2xl": (25, 1600, 6400, 50257, 48)}


@pytest.mark.parametrize("q8", [False, True])
@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("P", [0, 64, 200, 512, 1500, 5000])
def test_persistent_pass_accesses_stay_in_bounds(shape, P, q8):
    H, d, M, V, L = SHAPES[shape]
    max_ctx, max_nodes = P + 128, 64
    bad = []
    for N in list(range(1, 18)) + [31, 32, 33, 47, 48, 49, 63, 64]:
        bad += [f"N={N}: {b}" for b in check_pass(H, d, M, V, L, N, P, max_ctx, max_nodes, q8)]
    assert not bad, bad[:10]


def test_checker_catches_a_planted_overrun():
    """Power check: a plan whose LM-head range runs one row block past the
    packed head must be reported."""
    H, d, M, V, L = SHAPES["small"]
    orig = ssd.fused_plan

    def bad_plan(*a):
        tab, xh, xf = orig(*a)
        tab = tab.copy()
        tab[255, PL_HEAD + 1] += 1
        return tab, xh, xf

    ssd.fused_plan = bad_plan
    try:
        bad = check_pass(H, d, M, V, L, 5, 64, 192, 64)
    finally:
        ssd.fused_plan = orig
    assert any("head fragments" in b for b in bad), bad
