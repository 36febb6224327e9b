"""GPU parity of CDF-mode selection (Section 8.1) against the oracle.

The cut of a CDF row is decided in floating point: the kernel sums float32
exponentials, the oracle float64 ones. Both decide on the mass a prefix
leaves out, compared with (1 - tau) of the row's total, and both keep every
block at tau = 1. What is unique is compared exactly:

* at tau = 1 every row keeps all n blocks, bit for bit;
* the kept set must be a prefix of the row's unique order (score descending,
  index ascending) together with the forced blocks;
* for tau < 1 the prefix length k must be a valid cut within the kernel's
  float32 error: left(k) <= (1 - tau) Z (1 + eps) and left(k-1) > (1 - tau) Z
  (1 - eps), where left(k) is the oracle's left-out mass after k blocks and
  eps bounds the relative error of float32 sums of n positive terms, each
  exp(x) rounded with an error that grows with |x| (the score's distance from
  the row maximum). Wherever the float64 left-out masses are farther than
  eps from the budget, the cut is therefore exactly the oracle's;
* sel lists the kept blocks ascending then -1, counts their number.

tau is handed to both sides as the same float32 value.
"""

import numpy as np
import pytest

import oracle as orc
import paper_2609_32197_amd as sp
from tests import _parity as P

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


def rel_eps(n, spread):
    # sum of n positive float32 terms: (n - 1) u of the sum; each term exp(x),
    # x = s - max rounded (|x| u) and scaled to base 2 (|x| u), exp itself a few
    # ulp; the budget (1 - tau) Z carries the same for Z plus one rounding.
    return 2.0 * (2 * n + 8 + 4 * spread) * U


def check_rows(scores, mask_words, sel, counts, tau, i0, glob):
    """Asserts the validity of every row; returns the fraction of rows whose cut
    is exactly the oracle's."""
    H, nq, n = scores.shape
    tau = float(np.float32(tau))
    mask = orc.words_to_mask(mask_words.view(np.uint64), n)
    exact = 0
    for h in range(H):
        for r in range(nq):
            forced = {i0 + r} | set(glob)
            kept = set(np.nonzero(mask[h, r])[0].tolist())
            row = scores[h, r]
            order, left, Z = orc.cdf_order_and_mass(row)
            k_or = orc.cdf_cut(left, Z, tau)
            idx = sorted(kept)
            assert counts[h, r] == len(idx)
            assert sel[h, r, :len(idx)].tolist() == idx
            assert (sel[h, r, len(idx):] == -1).all()
            if tau >= 1.0:
                assert kept == set(range(n)), f"row h={h} r={r}: tau = 1 must keep every block"
                exact += 1
                continue
            budget = (1.0 - tau) * Z
            e = rel_eps(n, float(row.max()) - float(row.min()))
            ok = False
            prefix = set(forced)
            for k in range(1, n + 1):
                prefix.add(int(order[k - 1]))
                if prefix == kept and left[k] <= budget * (1 + e) and \
                        (k == 1 or left[k - 1] > budget * (1 - e)):
                    ok = True
                    break
            assert ok, f"row h={h} r={r}: kept set is not a valid CDF cut (oracle keeps {k_or})"
            exact += kept == (set(order[:k_or].tolist()) | forced)
    return exact / (H * nq)


def run_cdf(scores, tau, i0, glob):
    H, nq, n = scores.shape
    g = P.geometry(H, n * 64, 64, 64, i0, i0 + nq, "f32")
    m, sel, cnt = sp.sparsp_cdf_mask(g, P.to_device(scores, "f32"), tau, glob)
    return m.cpu().numpy(), sel.cpu().numpy(), cnt.cpu().numpy()


@pytest.mark.parametrize("n,nq,i0,glob,spread", [
    (16, 16, 0, (), 1.0), (71, 30, 41, (), 3.0), (129, 7, 100, (5, 128), 0.5),
    (591, 12, 0, (), 2.0), (4096, 3, 4000, (), 1.5), (1, 1, 0, (), 1.0),
    (200, 8, 0, (), 30.0), (64, 4, 60, (1,), 80.0)])
@pytest.mark.parametrize("tau", [0.5, 0.85, 0.9, 0.95, 0.999, 1.0 - 2.0 ** -24, 1.0])
def test_cdf_mask_valid_against_oracle(gpu, n, nq, i0, glob, spread, tau):
    rng = np.random.default_rng(n + nq)
    H = 2
    scores = (rng.standard_normal((H, nq, n)) * spread).astype(np.float32)
    if n > 8:
        scores[0, 0, 3] = scores[0, 0, 7]  # a tie
    m, sel, cnt = run_cdf(scores, tau, i0, glob)
    frac = check_rows(scores, m, sel, cnt, tau, i0, glob)
    assert frac >= 0.9, f"only {frac:.3f} of the rows cut where the oracle does"


def test_cdf_peaked_rows_exact(gpu):
    # Rows whose trailing blocks carry far less mass than float32 (or float64)
    # resolves against the total. The left-out mass decides the cut, so each
    # trailing block still counts: tau = 1 keeps all of them, and a tau just
    # below 1 leaves out exactly the blocks whose mass fits the budget.
    rows = [
        [0.0] + [-40.0] * 7,                     # 7 x 4.2e-18 behind the top block
        [0.0, -10.0, -20.0, -30.0, -40.0, -50.0, -60.0, -70.0],
        [5.0, 5.0, -30.0, -30.0, 4.0, -100.0, -200.0, 0.0],  # ties, underflow in float32
    ]
    # row r is query block r, so block r is forced as its diagonal
    scores = np.array(rows, dtype=np.float32)[None]  # H = 1, nq = 3, n = 8
    want = {
        1.0: [list(range(8))] * 3,
        1.0 - 2.0 ** -24: [[0], [0, 1], [0, 1, 4, 7]],
        0.999: [[0], [0, 1], [0, 1, 4, 7]],
    }
    for tau, rows_want in want.items():
        m, sel, cnt = run_cdf(scores, tau, 0, ())
        mask = orc.words_to_mask(m.view(np.uint64), 8)
        o_mask, _, _ = orc.select_cdf(scores, float(np.float32(tau)), 0)
        for r in range(3):
            forced = {r}
            got = sorted(np.nonzero(mask[0, r])[0].tolist())
            assert got == sorted(set(rows_want[r]) | forced), (tau, r, got)
            assert got == np.nonzero(o_mask[0, r])[0].tolist(), (tau, r)
            assert cnt[0, r] == len(got)


def test_cdf_full_size_wan_share_and_attention(gpu):
    from workloads import get_workload, make_qkv
    wl = get_workload("wan-share")
    q, k, v = make_qkv(wl)
    g = P.geometry(wl.H, wl.L, wl.d, wl.block, wl.i0, wl.i1, wl.dtype)
    Qd, Kd, Vd = (P.to_device(x, wl.dtype) for x in (q, k, v))
    _, _, sc = sp.sparsp_block_scores(g, Qd, Kd)
    scores = sc.cpu().numpy()
    for tau in (0.85, 0.9, 0.95, 1.0):
        m, sel, cnt = sp.sparsp_cdf_mask(g, sc, tau)
        frac = check_rows(scores, m.cpu().numpy(), sel.cpu().numpy(), cnt.cpu().numpy(), tau,
                          wl.i0, ())
        assert frac >= 0.99, (tau, frac)
    m, sel, cnt = sp.sparsp_cdf_mask(g, sc, 0.9)
    # attention with the CDF selection (sel is n wide, padded with -1), every
    # row against the oracle over the GPU's own mask; the longest-first launch
    # of sparsp_row_order must give the same bits
    out = sp.sparsp_demand_union_gather(g, m, Kd, Vd)
    args = (g, Qd, sel, out["slot_of"], out["K_packed"], out["V_packed"], wl.softmax_scale)
    O, lse = sp.sparsp_block_sparse_attn(*args)
    order = sp.sparsp_row_order(g, cnt)
    O2, lse2 = sp.sparsp_block_sparse_attn(*args, row_order=order)
    torch = P.torch()
    assert torch.equal(O.view(torch.int16), O2.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), lse2.view(torch.int32))
    mask = orc.words_to_mask(m.cpu().numpy().view(np.uint64), g.n)
    worst = P.check_every_row(q, k, v, mask, O.float().cpu().numpy(), lse.cpu().numpy(), wl,
                              g.i0, g.nq, True, "cdf attention", 1e-4)
    print(f"\n[cdf attention] tau 0.9, {wl.H * g.nq} rows, max-abs {worst:.3g}")
