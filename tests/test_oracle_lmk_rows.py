"""Pins for the oracle's S+1 query rows (the LMK token as the last query row of
every chunk; Methodology, Model Architecture and Grouped Cross-Attention: the
queries of chunk t+1 are its S + 1 hidden states, the retrieved memories have S
rows).  Each test ties the Sq = S + 1 path to something other than itself: a
dense attention matrix built by loops, finite differences, the row-wise
independence of attention (the S-row and one-row problems it splits into), and
invariants of the softmax Jacobian.
"""

import math

import numpy as np
import pytest

from oracle import gca
from test_oracle_pins import _small_problem


def _lmk_problem(seed, **kw):
    """_small_problem plus one extra query/dout row per chunk (the LMK row)."""
    p, lq, lk, q, k, v, dout = _small_problem(seed, **kw)
    S = p["S"]
    B, H, L, d = q.shape
    nQ = L // S
    rng = np.random.default_rng(seed + 1000)
    qx = rng.standard_normal((B, H, nQ, 1, d))
    dx = rng.standard_normal((B, H, nQ, 1, d))
    q1 = np.concatenate([q.reshape(B, H, nQ, S, d), qx], axis=3).reshape(B, H, nQ * (S + 1), d)
    d1 = np.concatenate([dout.reshape(B, H, nQ, S, d), dx], axis=3).reshape(B, H, nQ * (S + 1), d)
    return dict(p, Sq=S + 1), lq, lk, q1, k, v, d1


def _split(x, S):
    """[B,H,nQ*(S+1),...] -> (the S token rows of every chunk, the LMK rows)."""
    B, H, L = x.shape[:3]
    nQ = L // (S + 1)
    y = x.reshape(B, H, nQ, S + 1, *x.shape[3:])
    return (y[:, :, :, :S].reshape(B, H, nQ * S, *x.shape[3:]),
            y[:, :, :, S:].reshape(B, H, nQ, *x.shape[3:]))


def test_lmk_rows_dense_matrix_cross_check():
    """O = A V with A built by pure-Python loops over all S+1 rows of every chunk
    (row i of chunk i // (S+1)); A's rows sum to 1 from chunk 2 on, 0 before."""
    p, lq, lk, q, k, v, _ = _lmk_problem(21, nC=6, k=2, H=1, S=3, d=4)
    f = gca.forward(p, lq, lk, q, k, v)
    S, Sq, sc = p["S"], p["Sq"], p["attn_scale"]
    Lq, Lk = q.shape[2], k.shape[2]
    A = np.zeros((Lq, Lk))
    for i in range(Lq):
        c = i // Sq
        if c == 0:
            continue
        for s, j in enumerate(f["idx"][0, 0, c - 1]):
            if j < 0:
                continue
            logits = [sc * sum(q[0, 0, i, x] * k[0, 0, j * S + m, x] for x in range(4))
                      for m in range(S)]
            mx = max(logits)
            den = math.fsum(math.exp(a - mx) for a in logits)
            for m in range(S):
                A[i, j * S + m] += f["w"][0, 0, c - 1, s] * math.exp(logits[m] - mx) / den
    np.testing.assert_allclose(A @ v[0, 0], f["out"][0, 0], atol=1e-12)
    rs = A.sum(1)
    assert np.allclose(rs[2 * Sq:], 1.0) and np.all(rs[:2 * Sq] == 0.0)
    assert f["out"].shape == q.shape and f["lse"].shape == q.shape[:3] + (p["topk"],)


def test_lmk_rows_split_into_row_problems():
    """Attention is row-wise: the S+1 forward equals the S-row forward on the token
    rows and a one-row-per-chunk forward on the LMK rows; dq splits the same way,
    and dk, dv, dw are the sums of the two problems' gradients."""
    p, lq, lk, q, k, v, dout = _lmk_problem(22, nC=7, k=3, H=2, S=4, d=5)
    S = p["S"]
    f = gca.forward(p, lq, lk, q, k, v)
    g = gca.backward(p, f, lq, lk, q, k, v, dout)
    qt, qx = _split(q, S)
    dt, dx = _split(dout, S)
    pt = dict(p, Sq=S)
    px = dict(p, Sq=1)
    ft = gca.forward(pt, lq, lk, qt, k, v)
    fx = gca.forward(px, lq, lk, qx, k, v)
    gt = gca.backward(pt, ft, lq, lk, qt, k, v, dt)
    gx = gca.backward(px, fx, lq, lk, qx, k, v, dx)
    ot, ox = _split(f["out"], S)
    lt, lx = _split(f["lse"], S)
    # (equal up to the rounding of products over a different number of rows)
    for got, want in ((ot, ft["out"]), (ox, fx["out"]), (lt, ft["lse"]), (lx, fx["lse"])):
        assert np.array_equal(np.isinf(got), np.isinf(want))
        fin = np.isfinite(want)
        np.testing.assert_allclose(got[fin], want[fin], rtol=0, atol=1e-13)
    qgt, qgx = _split(g["dq"], S)
    np.testing.assert_allclose(qgt, gt["dq"], atol=1e-13)
    np.testing.assert_allclose(qgx, gx["dq"], atol=1e-13)
    # (dsel and the landmark gradients follow from dw through Eq. 2 and Eq. 1)
    for name in ("dk", "dv", "dw"):
        np.testing.assert_allclose(g[name], gt[name] + gx[name], atol=1e-12, err_msg=name)
    # the LMK rows do change the score gradient (they carry D_s like any row)
    assert np.abs(gx["dw"]).max() > 1e-3


@pytest.mark.parametrize("variant", ["plain", "off_by_one", "per_head_retrieval"])
def test_lmk_rows_backward_finite_differences(variant):
    """Central differences in fp64 (h=1e-6) for q, k, v, lmk_q, lmk_k with S+1 rows."""
    kw = dict(Hr=2, D=8) if variant == "per_head_retrieval" else {}
    p, lq, lk, q, k, v, dout = _lmk_problem(23, nC=5, S=3, d=4, **kw)
    pp = dict(p, off_by_one=variant == "off_by_one")
    f = gca.forward(pp, lq, lk, q, k, v)
    g = gca.backward(pp, f, lq, lk, q, k, v, dout)

    def loss(lq_, lk_, q_, k_, v_):
        ff = gca.forward(pp, lq_, lk_, q_, k_, v_)
        assert np.array_equal(ff["idx"], f["idx"])
        return float((dout * ff["out"]).sum())

    args = [lq, lk, q, k, v]
    h = 1e-6
    for ai, name in enumerate(["dlmk_q", "dlmk_k", "dq", "dk", "dv"]):
        a = args[ai]
        num = np.zeros_like(a)
        for ix in np.ndindex(a.shape):
            ap, am = a.copy(), a.copy()
            ap[ix] += h
            am[ix] -= h
            A = list(args)
            A[ai] = ap
            lp = loss(*A)
            A[ai] = am
            num[ix] = (lp - loss(*A)) / (2 * h)
        err = np.abs(num - g[name]).max() / max(np.abs(num).max(), 1e-30)
        assert err < 1e-6, (name, err)


def test_lmk_rows_backward_invariants():
    """Per head, the token sum of dK is 0 (plain softmax) and the token sum of dV is
    the sum of dout over every row that has a retrieved set, LMK rows included."""
    p, lq, lk, q, k, v, dout = _lmk_problem(24, nC=9, k=3, H=2)
    f = gca.forward(p, lq, lk, q, k, v)
    g = gca.backward(p, f, lq, lk, q, k, v, dout)
    assert np.abs(g["dk"].sum(2)).max() < 1e-11
    Sq = p["Sq"]
    np.testing.assert_allclose(g["dv"].sum(2), dout[:, :, 2 * Sq:].sum(2), atol=1e-11)
    assert np.abs(g["dsel"].sum(-1)).max() < 1e-12
