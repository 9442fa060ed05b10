"""Pins for the CPU oracle: it is checked against things other than itself.

Each test ties one part of the oracle to an independent fact: a hand-derived
closed form (tests/golden), a brute-force definition written differently, a
library routine, an invariant of the mathematics, or finite differences.
"""

import itertools
import json
import math
import os

import numpy as np
import pytest

from gen import bf16, get_workload, inputs as gi
from oracle import gca, margins

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_closed_form.json")


def _ev(x):
    if isinstance(x, str):
        return float(eval(x, {"__builtins__": {}}, {"exp": math.exp, "log": math.log,
                                                    "inf": math.inf}))
    return float(x)


def _arr(a):
    return np.array([[_ev(x) for x in row] for row in a])


# ---------------------------------------------------------------- golden ----

def _golden_problem(case, g):
    S = g["S"]
    k = np.array([[_ev(x) for x in r] for r in g["k"]])
    v = np.array(g["v"], dtype=float)
    if case["mode"] == "causal":
        lq = np.array(g["lmk_q"], float)[None, None]
        q = np.array(g["q"], float)[None, None]
    else:
        lq = np.array(case["decode_lmk_q"], float)[None, None]
        q = np.array(case["decode_q"], float)[None, None]
    lk = np.array(g["lmk_k"], float)[None, None]
    p = dict(S=S, topk=case["topk"], score_scale=g["score_scale"],
             attn_scale=g["attn_scale"], mode=case["mode"])
    return p, lq, lk, q, k[None, None], v[None, None]


@pytest.mark.parametrize("ci", [0, 1, 2])
def test_golden_closed_form(ci):
    """Hand-derived tiny case (Eq. 1-3, Alg. 1): indices, weights, outputs, lse."""
    g = json.load(open(GOLDEN))
    case = g["cases"][ci]
    p, lq, lk, q, k, v = _golden_problem(case, g)
    f = gca.forward(p, lq, lk, q, k, v)
    np.testing.assert_array_equal(f["idx"][0, 0], np.array(case["idx"]))
    np.testing.assert_array_equal(f["sel"][0, 0], _arr(case["sel"]))
    np.testing.assert_allclose(f["w"][0, 0], _arr(case["w"]), rtol=0, atol=1e-14)
    np.testing.assert_allclose(f["out"][0, 0], _arr(case["out"]), rtol=0, atol=1e-12)
    for row, slot, val in case["lse_valid"]:
        assert abs(f["lse"][0, 0, row, slot] - _ev(val)) < 1e-12
    # every slot not listed is a pad or an unused row: -inf
    listed = {(r, s) for r, s, _ in case["lse_valid"]}
    for r in range(f["lse"].shape[2]):
        for s in range(f["lse"].shape[3]):
            if (r, s) not in listed:
                assert f["lse"][0, 0, r, s] == -np.inf


# ---------------------------------------------------------------- scores ----

def test_scores_brute_force_fsum():
    """Eq. 1 scores against a pure-Python triple loop with exact summation."""
    rng = np.random.default_rng(0)
    lq = rng.standard_normal((2, 1, 7, 5))
    lk = rng.standard_normal((2, 1, 7, 5))
    sc = 0.37
    r = gca.scores(lq, lk, sc, "causal")
    for b in range(2):
        for t in range(7):
            for j in range(7):
                if j < t:
                    ref = sc * math.fsum(lq[b, 0, t, x] * lk[b, 0, j, x] for x in range(5))
                    assert abs(r[b, 0, t, j] - ref) < 1e-12
                else:
                    assert r[b, 0, t, j] == -np.inf
    rd = gca.scores(lq[:, :, :1], lk, sc, "decode")
    assert np.all(np.isfinite(rd))


# ------------------------------------------------------------------ top-k ----

def _rank_definition(row, t, k):
    """j is chosen iff fewer than k candidates beat it (higher score, or equal and lower j)."""
    chosen = []
    for j in range(t):
        beats = sum(1 for jj in range(t)
                    if row[jj] > row[j] or (row[jj] == row[j] and jj < j))
        if beats < k:
            chosen.append(j)
    return chosen


def test_topk_rank_definition_with_ties():
    rng = np.random.default_rng(1)
    for trial in range(200):
        t = int(rng.integers(0, 12))
        k = int(rng.integers(1, 6))
        row = np.full(12, -np.inf)
        # small integer scores force many ties
        row[:t] = rng.integers(-3, 4, size=t).astype(float)
        idx, sel = gca.topk_row(row, k)
        ref = _rank_definition(row, t, k)
        assert list(idx[:len(ref)]) == ref
        assert np.all(idx[len(ref):] == -1)
        assert np.all(sel[len(ref):] == -np.inf)
        assert np.array_equal(sel[:len(ref)], row[ref])


def test_topk_subset_maximises_sum():
    """With distinct scores the top-k set is the k-subset of largest total score."""
    rng = np.random.default_rng(2)
    for trial in range(50):
        t, k = 8, 3
        row = np.full(9, -np.inf)
        row[:t] = rng.standard_normal(t)
        best = max(itertools.combinations(range(t), k), key=lambda c: sum(row[list(c)]))
        idx, _ = gca.topk_row(row, k)
        assert tuple(idx) == tuple(sorted(best))


def test_k_covers_all_history_and_chunk0_empty():
    """k >= number of past chunks: chunk t retrieves exactly [0, t); chunk 0 retrieves nothing."""
    rng = np.random.default_rng(3)
    nC = 9
    lq = rng.standard_normal((1, 1, nC, 4))
    lk = rng.standard_normal((1, 1, nC, 4))
    r = gca.scores(lq, lk, 0.5)
    idx, sel = gca.topk(r, nC)
    for t in range(nC):
        assert list(idx[0, 0, t, :t]) == list(range(t))
        assert np.all(idx[0, 0, t, t:] == -1)
    assert np.all(idx[0, 0, 0] == -1)


# ---------------------------------------------------------------- weights ----

def _small_problem(seed, B=1, H=2, d=8, S=4, nC=6, k=2, D=16, Hr=1, margin=0.1,
                   mode="causal"):
    rng = np.random.default_rng(seed)
    nQ = 1 if mode == "decode" else nC
    for _ in range(1000):
        lq = rng.standard_normal((B, Hr, nQ, D))
        lk = rng.standard_normal((B, Hr, nC, D))
        g = margins.row_gaps(lq, lk, 1 / math.sqrt(D), k, mode)
        if np.all(g >= margin):
            break
    else:
        raise RuntimeError("no margin")
    q = rng.standard_normal((B, H, nQ * S, d))
    kk = rng.standard_normal((B, H, nC * S, d))
    v = rng.standard_normal((B, H, nC * S, d))
    dout = rng.standard_normal((B, H, nQ * S, d))
    p = dict(S=S, topk=k, score_scale=1 / math.sqrt(D), attn_scale=1 / math.sqrt(d), mode=mode)
    return p, lq, lk, q, kk, v, dout


def test_weights_sum_and_key_shift_invariance():
    """Weights sum to 1 over valid slots; adding one vector to every landmark key
    shifts each row's scores by a constant, leaving idx, w and the output unchanged."""
    p, lq, lk, q, k, v, _ = _small_problem(4, nC=10, k=3)
    f = gca.forward(p, lq, lk, q, k, v)
    valid = f["idx"] >= 0
    s = f["w"].sum(-1)
    assert np.allclose(s[valid.any(-1)], 1.0, atol=1e-14)
    assert np.all(s[~valid.any(-1)] == 0.0)
    u = np.random.default_rng(5).standard_normal(lk.shape[-1]) * 0.01
    f2 = gca.forward(p, lq, lk + u, q, k, v)
    np.testing.assert_array_equal(f["idx"], f2["idx"])
    np.testing.assert_allclose(f["w"], f2["w"], atol=1e-12)
    np.testing.assert_allclose(f["out"], f2["out"], atol=1e-12)


# ------------------------------------------------------- cross attention ----

def test_k1_equals_library_attention():
    """k=1: w=1 and each chunk's output is textbook attention onto its one retrieved chunk
    (torch scaled_dot_product_attention in fp64 on the CPU)."""
    torch = pytest.importorskip("torch")
    p, lq, lk, q, k, v, _ = _small_problem(6, nC=7, k=1, H=3, S=8, d=16)
    f = gca.forward(p, lq, lk, q, k, v)
    S = p["S"]
    for h in range(3):
        for c in range(2, 7):
            j = int(f["idx"][0, 0, c - 1, 0])
            qt = torch.tensor(q[0, h, c * S:(c + 1) * S])[None, None]
            kt = torch.tensor(k[0, h, j * S:(j + 1) * S])[None, None]
            vt = torch.tensor(v[0, h, j * S:(j + 1) * S])[None, None]
            ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=p["attn_scale"])
            np.testing.assert_allclose(f["out"][0, h, c * S:(c + 1) * S], ref[0, 0].numpy(),
                                       atol=1e-12)
    assert np.all(f["out"][0, :, :2 * S] == 0.0)


def test_off_by_one_equals_softmax_with_zero_logit():
    """Eq. 3's softmax-off-by-one equals an ordinary softmax over the logits plus one
    extra logit fixed at 0, with that extra column dropped (scipy reference)."""
    from scipy.special import softmax, logsumexp
    rng = np.random.default_rng(7)
    qc = rng.standard_normal((5, 4)) * 3
    kc = rng.standard_normal((6, 4))
    vc = rng.standard_normal((6, 3))
    p, o, lse = gca.chunk_attention(qc, kc, vc, 0.5, off_by_one=True)
    a = 0.5 * qc @ kc.T
    aug = np.concatenate([np.zeros((5, 1)), a], axis=1)
    np.testing.assert_allclose(p, softmax(aug, axis=1)[:, 1:], atol=1e-14)
    np.testing.assert_allclose(lse, logsumexp(aug, axis=1), atol=1e-12)
    np.testing.assert_allclose(o, p @ vc, atol=1e-13)
    # very negative logits: the row can ignore every retrieved token
    p2, o2, _ = gca.chunk_attention(np.ones((5, 4)), -10 * np.ones((6, 4)), vc, 0.5,
                                    off_by_one=True)
    assert np.all(p2.sum(1) < 1e-7) and np.abs(o2).max() < 1e-7


def test_gca_differs_from_cca_and_is_linear_in_v():
    """GCA normalises each retrieved chunk separately and fuses with w; concatenating the
    chunks under one softmax (CCA) gives a different result.  The output is linear in V."""
    p, lq, lk, q, k, v, _ = _small_problem(8, nC=8, k=3)
    f = gca.forward(p, lq, lk, q, k, v)
    S, sc = p["S"], p["attn_scale"]
    c = 7
    rows = slice(c * S, (c + 1) * S)
    js = [int(j) for j in f["idx"][0, 0, c - 1] if j >= 0]
    kc = np.concatenate([k[0, 0, j * S:(j + 1) * S] for j in js])
    vc = np.concatenate([v[0, 0, j * S:(j + 1) * S] for j in js])
    a = sc * q[0, 0, rows] @ kc.T
    e = np.exp(a - a.max(1, keepdims=True))
    cca = (e / e.sum(1, keepdims=True)) @ vc
    assert np.abs(cca - f["out"][0, 0, rows]).max() > 1e-3
    f3 = gca.forward(p, lq, lk, q, k, 2.5 * v)
    np.testing.assert_allclose(f3["out"], 2.5 * f["out"], atol=1e-12)


def test_dense_matrix_cross_check():
    """O = A V with A[i, j*S+m] = w_s p_m built by pure-Python loops; A's rows sum to 1
    for chunks >= 2 and to 0 for chunks 0 and 1."""
    p, lq, lk, q, k, v, _ = _small_problem(9, nC=6, k=2, H=1, S=3, d=4)
    f = gca.forward(p, lq, lk, q, k, v)
    S, sc = p["S"], p["attn_scale"]
    L = q.shape[2]
    A = np.zeros((L, L))
    for i in range(L):
        c = i // S
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
    assert np.allclose(rs[2 * S:], 1.0) and np.all(rs[:2 * S] == 0.0)


def test_causality():
    """Perturbing anything of chunks > c leaves rows <= c unchanged; perturbing K/V of
    chunk c-1 leaves chunk c unchanged (its set lies in [0, c-2])."""
    p, lq, lk, q, k, v, _ = _small_problem(10, nC=8, k=2)
    f = gca.forward(p, lq, lk, q, k, v)
    S = p["S"]
    rng = np.random.default_rng(11)
    for c in range(1, 7):
        lq2, lk2, q2, k2, v2 = lq.copy(), lk.copy(), q.copy(), k.copy(), v.copy()
        lq2[:, :, c + 1:] += rng.standard_normal(lq2[:, :, c + 1:].shape)
        lk2[:, :, c + 1:] += rng.standard_normal(lk2[:, :, c + 1:].shape)
        for a in (q2, k2, v2):
            a[:, :, (c + 1) * S:] += rng.standard_normal(a[:, :, (c + 1) * S:].shape)
        k2[:, :, (c - 1) * S:c * S] += 1.0
        v2[:, :, (c - 1) * S:c * S] += 1.0
        f2 = gca.forward(p, lq2, lk2, q2, k2, v2)
        np.testing.assert_array_equal(f2["out"][:, :, :(c + 1) * S], f["out"][:, :, :(c + 1) * S])


# --------------------------------------------------------------- backward ----

def _loss_grads(p, lq, lk, q, k, v, dout, obo=False):
    p = dict(p, off_by_one=obo)
    f = gca.forward(p, lq, lk, q, k, v)
    return f, gca.backward(p, f, lq, lk, q, k, v, dout)


@pytest.mark.parametrize("variant", ["plain", "off_by_one", "per_head_retrieval", "decode"])
def test_backward_finite_differences(variant):
    """Central differences in fp64 (h=1e-6) for q, k, v, lmk_q, lmk_k."""
    kw = {}
    if variant == "per_head_retrieval":
        kw = dict(Hr=2, D=8)
    if variant == "decode":
        kw = dict(mode="decode", nC=7, k=3)
    p, lq, lk, q, k, v, dout = _small_problem(12, **kw)
    obo = variant == "off_by_one"
    f, g = _loss_grads(p, lq, lk, q, k, v, dout, obo)
    pp = dict(p, off_by_one=obo)

    def loss(lq_, lk_, q_, k_, v_):
        ff = gca.forward(pp, lq_, lk_, q_, k_, v_)
        assert np.array_equal(ff["idx"], f["idx"])
        return float((dout * ff["out"]).sum())

    args = [lq, lk, q, k, v]
    names = ["dlmk_q", "dlmk_k", "dq", "dk", "dv"]
    h = 1e-6
    for ai, name in enumerate(names):
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
            lm = loss(*A)
            num[ix] = (lp - lm) / (2 * h)
        scale = max(np.abs(num).max(), 1e-30)
        err = np.abs(num - g[name]).max() / scale
        assert err < 1e-6, (name, err)


def test_backward_invariants():
    """sum_s dsel = 0 per row, so sum_j dlmk_k = 0; with plain softmax sum over tokens of
    dK is 0 per head, and sum over tokens of dV equals sum of dout over rows with a set."""
    p, lq, lk, q, k, v, dout = _small_problem(13, nC=9, k=3, H=2)
    f, g = _loss_grads(p, lq, lk, q, k, v, dout)
    assert np.abs(g["dsel"].sum(-1)).max() < 1e-12
    assert np.abs(g["dlmk_k"].sum(2)).max() < 1e-12
    assert np.abs(g["dk"].sum(2)).max() < 1e-11
    S = p["S"]
    np.testing.assert_allclose(g["dv"].sum(2), dout[:, :, 2 * S:].sum(2), atol=1e-11)


# --------------------------------------------------- planted / generator ----

def test_planted_closed_form():
    """Planted keys 4*q_last make the last row's top-8 exactly the planted chunks,
    with equal scores and so weights 1/8 each."""
    w = get_workload("planted_1m_bf16", n_chunks=512, H=1)
    lq, lk = gi.draw_landmarks(w)
    pos = gi.plant_positions(w)
    r = gca.scores(gi.decode(w, lq), gi.decode(w, lk), w.score_scale, rows=[w.n_chunks - 1])
    idx, sel = gca.topk(r, 8)
    assert list(idx[0, 0, 0]) == list(pos)
    wt = gca.fusion_weights(sel)
    np.testing.assert_allclose(wt[0, 0, 0], np.full(8, 1 / 8), atol=1e-15)
    qn = gi.decode(w, lq)[0, 0, -1]
    assert np.allclose(sel[0, 0, 0], 4 * w.score_scale * (qn @ qn))


def test_margin_enforcement():
    w = get_workload("train_16k_bf16", B=2)
    inp, n = margins.checked_inputs(w, tokens=False)
    g = margins.row_gaps(gi.decode(w, inp["lmk_q"]), gi.decode(w, inp["lmk_k"]),
                         w.score_scale, w.topk, w.mode)
    assert n > 0 and np.all(g >= w.margin)


def test_bf16_codec():
    """Known patterns, and agreement with torch's round-to-nearest-even on fp32 inputs."""
    assert bf16.from_f64(np.array([1.0]))[0] == 0x3F80
    assert bf16.from_f64(np.array([-2.0]))[0] == 0xC000
    assert bf16.from_f64(np.array([0.0]))[0] == 0
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7 -> even (1.0); 1 + 3*2^-8 -> up
    assert bf16.from_f64(np.array([1 + 2 ** -8]))[0] == 0x3F80
    assert bf16.from_f64(np.array([1 + 3 * 2 ** -8]))[0] == 0x3F82
    torch = pytest.importorskip("torch")
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(bf16.from_f64(x.astype(np.float64)), ref)
    np.testing.assert_array_equal(bf16.to_f64(ref), torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).double().numpy())
