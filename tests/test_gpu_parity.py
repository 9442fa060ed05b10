"""GPU parity of every libgca entry point against the CPU oracle.

Inputs are seeded and margin-checked (the k-th and (k+1)-th landmark scores of
every row differ by >= 1e-3), so top-k indices must match bit-exactly; floating
outputs must match within max-abs-rel 1e-4 (fp32) or 2e-2 (bf16).  Shapes here
are small enough for the oracle to run in seconds while spanning several tiles
and ragged tails; the full workload sizes are in test_gpu_workloads.py.
"""

import math

import numpy as np
import pytest

from _helpers import TOL, decode_all, ensure_built, host64, max_abs_rel, oracle_params, problem_for, upload
from gen import get_workload, inputs as gi
from oracle import gca as og, margins

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ensure_built()
    return torch.device("cuda:0")


def _case(name, **kw):
    w = get_workload(name, **kw)
    inp, _ = margins.checked_inputs(w)
    return w, inp


def _check_forward(w, inp, f, off_by_one=False, tol=None):
    tol = tol or TOL[w.dtype]
    x = decode_all(w, inp)
    ref = og.forward(oracle_params(w, off_by_one), x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"])
    np.testing.assert_array_equal(f["idx"].cpu().numpy(), ref["idx"])
    assert max_abs_rel(host64(f["sel"]), ref["sel"]) <= tol
    if f.get("w") is not None:
        assert max_abs_rel(host64(f["w"]), ref["w"]) <= tol
    assert max_abs_rel(host64(f["out"]), ref["out"]) <= tol
    if f.get("lse") is not None:
        assert max_abs_rel(host64(f["lse"]), ref["lse"]) <= tol
    return ref


def test_tiny_fp32_forward(dev):
    """1,024 tokens, 16 chunks, top-2, fp32: the whole forward against the oracle."""
    from paper_2410_01651_amd import gca
    w, inp = _case("tiny_fp32_1k")
    t = upload(w, inp, dev)
    f = gca.forward(problem_for(w), t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    ref = _check_forward(w, inp, f)
    out = f["out"].cpu().numpy()
    assert np.all(out[:, :, :2 * w.S] == 0.0)          # chunks 0 and 1 retrieve nothing
    assert np.all(ref["idx"][0, 0, 0] == -1)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_stepwise_equals_forward(dev, dtype):
    """gca_chunk_scores -> gca_topk -> gca_grouped_xattn_fwd gives what gca_forward gives."""
    from paper_2410_01651_amd import gca
    w, inp = _case("train_16k_bf16", B=2, H=3, n_chunks=70, topk=5, dtype=dtype)
    t = upload(w, inp, dev)
    p = problem_for(w)
    sc = gca.chunk_scores(p, t["lmk_q"], t["lmk_k"])
    idx, sel = gca.topk(p, sc)
    out, lse, wt = gca.grouped_xattn_fwd(p, t["q"], t["k"], t["v"], idx, sel)
    f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    assert np.array_equal(idx.cpu().numpy(), f["idx"].cpu().numpy())
    assert np.array_equal(sel.cpu().numpy(), f["sel"].cpu().numpy())
    assert np.array_equal(host64(out), host64(f["out"]))
    assert np.array_equal(lse.cpu().numpy(), f["lse"].cpu().numpy())
    _check_forward(w, inp, dict(f, w=wt))
    x = decode_all(w, inp)
    rs = og.scores(x["lmk_q"], x["lmk_k"], w.score_scale)
    assert max_abs_rel(host64(sc), rs) <= TOL[dtype]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_topk_ties_to_lower_chunk(dev, dtype):
    """Score rows full of exact ties: the chosen set is decided by (score desc, chunk asc)."""
    import torch
    from paper_2410_01651_amd import gca
    rng = np.random.default_rng(5)
    for nC, k in ((16, 2), (100, 8), (300, 32), (1000, 17)):
        p = gca.problem(2, 1, nC, k, D=64, dtype=dtype)
        r = rng.integers(-4, 5, size=(2, 1, nC, nC)).astype(np.float32)
        r = np.where(np.arange(nC)[None, :] < np.arange(nC)[:, None], r, -np.inf).astype(np.float32)
        idx, sel = gca.topk(p, torch.from_numpy(r).to(dev))
        ri, rs = og.topk(r.astype(np.float64), k)
        np.testing.assert_array_equal(idx.cpu().numpy(), ri)
        np.testing.assert_array_equal(sel.cpu().numpy(), rs.astype(np.float32))


FUSED = [
    # split select (per-row lists of key-tile parts, then a merge)
    ("planted_1m_bf16", "fp32", dict(H=2, n_chunks=300)),
    ("planted_1m_bf16", "bf16", dict(H=2, n_chunks=300)),
    ("planted_1m_bf16", "bf16", dict(H=8, n_chunks=700, topk=12)),        # width 512, best-16 lists, 3 row blocks
    ("planted_1m_bf16", "bf16", dict(H=1, D=64, n_chunks=5000, topk=8)),  # 79 key tiles: 2 parts per class
    ("train_16k_bf16", "fp32", dict(B=2, H=4, n_chunks=1100, topk=3)),    # fp32 at width 256
    # one pass per 64-row block (outside the split form's register budget)
    ("planted_1m_bf16", "bf16", dict(H=2, n_chunks=300, topk=20)),
    ("planted_1m_bf16", "bf16", dict(H=16, n_chunks=200, topk=8)),        # width 1024
    ("planted_1m_bf16", "fp32", dict(H=8, n_chunks=300, topk=8)),         # fp32 at width 512
]


@pytest.mark.parametrize("name,dtype,kw", FUSED)
def test_fused_select_equals_oracle(dev, name, dtype, kw):
    """The causal select without the score matrix against the oracle and the
    materialised path."""
    from paper_2410_01651_amd import gca
    w, inp = _case(name, dtype=dtype, **kw)
    t = upload(w, inp, dev)
    fa = gca.forward(problem_for(w, flags=gca.FLAG_FUSED_TOPK), t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    fb = gca.forward(problem_for(w, flags=gca.FLAG_MATERIALIZE), t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    assert np.array_equal(fa["idx"].cpu().numpy(), fb["idx"].cpu().numpy())
    ref = _check_forward(w, inp, fa)
    if w.planted:           # the planted chunks are the last row's best (with k >= 8 of them)
        assert set(gi.plant_positions(w).tolist()) <= set(ref["idx"][0, 0, -1].tolist())


SWEEP = [
    # name, overrides, off_by_one
    ("train_16k_bf16", dict(B=1, H=2, n_chunks=1, topk=4), False),       # single chunk: all empty
    ("train_16k_bf16", dict(B=2, H=2, n_chunks=3, topk=8), False),       # k > history
    ("train_16k_bf16", dict(B=1, H=4, n_chunks=9, topk=1), False),       # k = 1
    ("train_16k_bf16", dict(B=1, H=4, Hr=4, D=64, n_chunks=33, topk=3), False),   # per-head retrieval
    ("train_16k_bf16", dict(B=2, H=2, n_chunks=65, topk=32), True),      # off-by-one, k = 32
    ("train_16k_bf16", dict(B=1, H=2, n_chunks=700, topk=3), False),     # 1,400 chunks: uneven streams
    # either side of the switch to the chip-wide window order (eight slices' K/V
    # above 256 MiB: more than 2,048 bf16 chunks per slice)
    ("train_16k_bf16", dict(B=1, H=1, n_chunks=2048, topk=2), False),
    ("train_16k_bf16", dict(B=1, H=1, n_chunks=2049, topk=2), False),
    ("tiny_fp32_1k", dict(B=2, H=3, n_chunks=37, topk=6, whole_reseed=False), True),
    ("tiny_fp32_1k", dict(B=1, H=2, Hr=2, D=128, n_chunks=20, topk=9, whole_reseed=False), False),
    ("decode_16m_bf16", dict(H=4, n_chunks=3000, device_kv=False), False),
    ("decode_16m_bf16", dict(H=2, n_chunks=500, topk=32, dtype="fp32", device_kv=False), True),
    ("decode_16m_bf16", dict(H=2, Hr=2, D=64, n_chunks=5, topk=8, device_kv=False), False),
    # decode scan ranges: a ragged last key group, 16 and 1 column blocks per key,
    # fp32 with 3 blocks per key, several retrieval rows
    ("decode_16m_bf16", dict(H=2, n_chunks=20001, device_kv=False), False),
    ("decode_16m_bf16", dict(H=2, D=1024, n_chunks=1001, topk=5, device_kv=False), True),
    ("decode_16m_bf16", dict(H=2, Hr=2, D=64, n_chunks=777, device_kv=False), False),
    ("decode_16m_bf16", dict(H=1, D=192, n_chunks=999, topk=3, dtype="fp32", device_kv=False), False),
    ("decode_16m_bf16", dict(B=3, H=2, n_chunks=4000, topk=16, device_kv=False), False),
    # D = 512: the query fragments live in registers
    ("decode_16m_bf16", dict(H=8, n_chunks=3001, device_kv=False), False),
    ("decode_16m_bf16", dict(H=8, n_chunks=2001, topk=5, dtype="fp32", device_kv=False), True),
]


@pytest.mark.parametrize("name,kw,obo", SWEEP)
def test_forward_sweep(dev, name, kw, obo):
    from paper_2410_01651_amd import gca
    w, inp = _case(name, **kw)
    t = upload(w, inp, dev)
    f = gca.forward(problem_for(w, off_by_one=obo), t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    _check_forward(w, inp, f, off_by_one=obo)


BWD = [
    ("tiny_fp32_1k", dict(B=1, H=2, n_chunks=16, topk=2), False),
    ("tiny_fp32_1k", dict(B=2, H=2, n_chunks=21, topk=4, whole_reseed=False), True),
    ("tiny_fp32_1k", dict(B=1, H=3, Hr=3, D=64, n_chunks=12, topk=3, whole_reseed=False), False),
    ("fwdbwd_64k_bf16", dict(B=2, H=3, n_chunks=40, topk=8), False),
    ("fwdbwd_64k_bf16", dict(B=1, H=2, n_chunks=70, topk=20), True),
    ("fwdbwd_64k_bf16", dict(B=1, H=2, Hr=2, D=128, n_chunks=33, topk=5), False),
    ("fwdbwd_64k_bf16", dict(B=1, H=2, n_chunks=700, topk=1), False),    # k = 1, uneven streams
    ("tiny_fp32_1k", dict(B=1, H=2, n_chunks=600, topk=1, whole_reseed=False), True),
    # slices long enough for the chip-wide window order of the query-chunk streams
    # (eight slices' K/V above 256 MiB), with partial windows and a slice boundary
    # inside a window
    ("tiny_fp32_1k", dict(B=1, H=1, n_chunks=1100, topk=2, whole_reseed=False), False),
    ("fwdbwd_64k_bf16", dict(B=1, H=2, n_chunks=2100, topk=4), False),
    ("decode_16m_bf16", dict(H=2, n_chunks=300, planted=0, backward=True, device_kv=False), False),
    ("decode_16m_bf16", dict(H=2, n_chunks=100, topk=4, planted=0, dtype="fp32", backward=True,
                             device_kv=False), False),
    # decode backward past the window-order threshold (one query chunk per head)
    ("decode_16m_bf16", dict(H=2, n_chunks=2500, topk=8, planted=0, backward=True, device_kv=False), False),
]


def _random_cases(n, seed=20241001):
    """n seeded random small configurations across the problem options."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        base = "tiny_fp32_1k" if rng.random() < 0.3 else "fwdbwd_64k_bf16"
        H = int(rng.integers(1, 5))
        per_head = bool(rng.random() < 0.3)
        kw = dict(B=int(rng.integers(1, 3)), H=H, n_chunks=int(rng.integers(1, 48)), topk=int(rng.integers(1, 17)),
                  lmk_row=bool(rng.random() < 0.3))
        if per_head:
            kw.update(Hr=H, D=int(rng.choice([64, 128, 192])))
        else:
            kw.update(D=int(rng.choice([64, 256, 512, 768, 1024])))
        if base == "tiny_fp32_1k":
            kw["whole_reseed"] = False
        if rng.random() < 0.3:
            kw["gumbel_seed"] = int(rng.integers(1, 2**31))
        out.append((f"r{i}", base, kw, bool(rng.random() < 0.4)))
    return out


@pytest.mark.parametrize("tag,name,kw,obo", _random_cases(40))
def test_random_sweep(dev, tag, name, kw, obo):
    """Seeded random small problems (batch, heads, shared or per-head retrieval,
    landmark width, k from 1 to 16 with chunk counts around and below it, S or S+1
    query rows, off-by-one, Gumbel top-k, fp32 or bf16): forward and every gradient
    against the oracle."""
    from paper_2410_01651_amd import gca
    w, inp = _case(name, **kw)
    if "dout" not in inp:
        inp["dout"] = gi.draw_slices(w, "dout", (w.B, w.H, w.Lq, w.d))
    t = upload(w, inp, dev)
    p = problem_for(w, off_by_one=obo)
    f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    ref = _check_forward(w, inp, f, off_by_one=obo)
    g = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"],
                              t["lmk_q"], t["lmk_k"])
    x = decode_all(w, inp)
    rb = og.backward(oracle_params(w, obo), ref, x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"], x["dout"])
    for key in ("dq", "dk", "dv", "dsel", "dlmk_q", "dlmk_k"):
        assert max_abs_rel(host64(g[key]), rb[key]) <= TOL[w.dtype], key


def _random_decode_cases(n, seed=20241002):
    """n seeded random decode problems (past chunks from 1 to 6,000; the K/V of
    the larger ones over fewer heads)."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        nc, B = int(rng.integers(1, 6001)), int(rng.integers(1, 3))
        # heads capped so that the drawn K/V cache stays small (B * H * nc <= 2,500)
        H = max(1, min(int(rng.integers(1, 9)), 2500 // (B * nc)))
        kw = dict(B=B, H=H, n_chunks=nc, topk=int(rng.integers(1, 33)),
                  planted=0, device_kv=False, dtype="fp32" if rng.random() < 0.3 else "bf16")
        if rng.random() < 0.3:
            kw.update(Hr=H, D=int(rng.choice([64, 128])))
        else:
            kw.update(D=int(rng.choice([64, 192, 512, 1024, 2048])))
        if rng.random() < 0.3:
            kw["gumbel_seed"] = int(rng.integers(1, 2**31))
        out.append((f"d{i}", kw, bool(rng.random() < 0.3)))
    return out


@pytest.mark.parametrize("tag,kw,obo", _random_decode_cases(24))
def test_random_decode_sweep(dev, tag, kw, obo):
    """Seeded random decode problems (batch, heads, shared or per-head retrieval,
    landmark width, k up to 32, past lengths from 1 chunk up, off-by-one, Gumbel
    top-k, fp32/bf16): the decode scan, merge and attention against the oracle."""
    from paper_2410_01651_amd import gca
    w, inp = _case("decode_16m_bf16", **kw)
    t = upload(w, inp, dev)
    f = gca.forward(problem_for(w, off_by_one=obo), t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    _check_forward(w, inp, f, off_by_one=obo)


@pytest.mark.parametrize("name,kw,obo", BWD)
def test_backward(dev, name, kw, obo):
    """dq, dk, dv, dsel and both landmark gradients against the oracle's chain rule."""
    from paper_2410_01651_amd import gca
    w, inp = _case(name, **kw)
    if "dout" not in inp:
        inp["dout"] = gi.draw_slices(w, "dout", (w.B, w.H, w.Lq, w.d))
    t = upload(w, inp, dev)
    p = problem_for(w, off_by_one=obo)
    f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    g = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"],
                              t["lmk_q"], t["lmk_k"])
    x = decode_all(w, inp)
    pp = oracle_params(w, obo)
    rf = og.forward(pp, x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"])
    np.testing.assert_array_equal(f["idx"].cpu().numpy(), rf["idx"])
    rb = og.backward(pp, rf, x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"], x["dout"])
    tol = TOL[w.dtype]
    for key in ("dq", "dk", "dv", "dsel", "dlmk_q", "dlmk_k"):
        e = max_abs_rel(host64(g[key]), rb[key])
        assert e <= tol, (key, e)
    # the score gradient sums to zero over each row's slots
    assert np.abs(host64(g["dsel"]).sum(-1)).max() <= 1e-5 * max(1.0, np.abs(rb["dsel"]).max())


def test_backward_saturated_weights(dev):
    """A planted chunk takes weight 1 - O(e^-85): the score gradient vanishes (in absolute
    terms) and the token gradients equal single-chunk attention's."""
    from paper_2410_01651_amd import gca
    w, inp = _case("decode_16m_bf16", H=2, n_chunks=300, backward=True, device_kv=False)
    t = upload(w, inp, dev)
    p = problem_for(w)
    f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    g = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"],
                              t["lmk_q"], t["lmk_k"])
    x = decode_all(w, inp)
    pp = oracle_params(w)
    rf = og.forward(pp, x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"])
    np.testing.assert_array_equal(f["idx"].cpu().numpy(), rf["idx"])
    assert int(gi.plant_positions(w)[0]) in list(rf["idx"][0, 0, 0])
    rb = og.backward(pp, rf, x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"], x["dout"])
    dw = max(1.0, np.abs(rb["dw"]).max())
    assert np.abs(rb["dsel"]).max() <= 1e-12 * dw          # w = 1 - O(e^-85): only rounding left
    assert np.abs(host64(g["dsel"])).max() <= 1e-5 * dw
    for key in ("dq", "dk", "dv"):
        assert max_abs_rel(host64(g[key]), rb[key]) <= TOL[w.dtype], key


@pytest.mark.parametrize("name,kw,obo", [("fwdbwd_64k_bf16", dict(B=1, H=2, n_chunks=24, topk=4), False),
                                         ("fwdbwd_64k_bf16", dict(B=1, H=2, n_chunks=24, topk=4), True),
                                         ("tiny_fp32_1k", dict(B=1, H=2, n_chunks=20, topk=3), False)])
def test_large_logits(dev, name, kw, obo):
    """Q and K scaled by 4 (exact in both dtypes: a power of two), so the attention
    logits reach tens of nats and each chunk's softmax is nearly one-hot: the
    shifted exponentials, the log-sum-exp and the backward's cancellations in
    dP - D stay finite and match the oracle."""
    from paper_2410_01651_amd import gca
    w, inp = _case(name, backward=True, **kw)
    for key in ("q", "k"):
        inp[key] = gi.encode(w, gi.decode(w, inp[key]) * 4.0)
    t = upload(w, inp, dev)
    p = problem_for(w, off_by_one=obo)
    f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    x = decode_all(w, inp)
    pp = oracle_params(w, obo)
    rf = og.forward(pp, x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"])
    np.testing.assert_array_equal(f["idx"].cpu().numpy(), rf["idx"])
    lse = rf["lse"][np.isfinite(rf["lse"])]
    assert lse.max() - lse.min() > 40.0  # the logits really are large
    tol = TOL[w.dtype]
    for key in ("out", "lse", "w"):
        assert max_abs_rel(host64(f[key]), rf[key]) <= tol, key
    g = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"],
                              t["lmk_q"], t["lmk_k"])
    rb = og.backward(pp, rf, x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"], x["dout"])
    for key in ("dq", "dk", "dv", "dsel", "dlmk_q", "dlmk_k"):
        e = max_abs_rel(host64(g[key]), rb[key])
        assert e <= tol, (key, e)


def test_backward_deterministic(dev):
    """No floating-point atomics: two backward passes are bit-identical."""
    from paper_2410_01651_amd import gca
    w, inp = _case("fwdbwd_64k_bf16", B=1, H=4, n_chunks=96, topk=8)
    t = upload(w, inp, dev)
    p = problem_for(w)
    f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    g1 = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"],
                               t["lmk_q"], t["lmk_k"])
    g2 = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"],
                               t["lmk_q"], t["lmk_k"])
    for key in g1:
        assert np.array_equal(host64(g1[key]), host64(g2[key])), key


@pytest.mark.parametrize("name,kw", [("fwdbwd_64k_bf16", dict(B=2, H=4, n_chunks=40, topk=8)),
                                     ("tiny_fp32_1k", dict(B=1, H=2, n_chunks=20, topk=3, whole_reseed=False)),
                                     ("fwdbwd_64k_bf16", dict(B=1, H=2, n_chunks=12, topk=4, D=8192))])
def test_landmark_gradients_one_at_a_time(dev, name, kw):
    """dlmk_q alone, dlmk_k alone and both (one launch whose dlmk_k blocks form
    dsel themselves) give the same bits for every output."""
    from paper_2410_01651_amd import gca
    w, inp = _case(name, **kw)
    if "dout" not in inp:
        inp["dout"] = gi.draw_slices(w, "dout", (w.B, w.H, w.Lq, w.d))
    t = upload(w, inp, dev)
    p = problem_for(w)
    f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    args = (p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"], t["lmk_q"], t["lmk_k"])
    both = gca.grouped_xattn_bwd(*args)
    only_q = gca.grouped_xattn_bwd(*args, landmark_grads=("dlmk_q",))
    only_k = gca.grouped_xattn_bwd(*args, landmark_grads=("dlmk_k",))
    assert "dlmk_k" not in only_q and "dlmk_q" not in only_k
    for part in (only_q, only_k):
        for key in part:
            assert np.array_equal(host64(part[key]), host64(both[key])), key


@pytest.mark.parametrize("name,kw,backward", [
    ("train_16k_bf16", dict(B=1, H=2, n_chunks=40, topk=8), True),
    ("train_16k_bf16", dict(B=1, H=2, n_chunks=30, topk=5, lmk_row=True), True),
    ("decode_16m_bf16", dict(H=2, n_chunks=3000, device_kv=False), False),
])
def test_graph_capture_replays(dev, name, kw, backward):
    """The path captured into a HIP graph (the library enqueues kernels only, no
    allocation or memset) and replayed three times, with eager work and a clear of
    every output between replays: each replay reproduces the eager call bit for bit."""
    import torch
    from paper_2410_01651_amd import gca
    w, inp = _case(name, **kw)
    if backward and "dout" not in inp:
        inp["dout"] = gi.draw_slices(w, "dout", (w.B, w.H, w.Lq, w.d))
    t = upload(w, inp, dev)
    p = problem_for(w)
    sh = gca.shapes(p)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    outs = {"out": torch.empty(sh.q, dtype=dt, device=dev), "idx": torch.empty(sh.rows, dtype=torch.int32, device=dev),
            "sel": torch.empty(sh.rows, dtype=torch.float32, device=dev),
            "lse": torch.empty(sh.lse, dtype=torch.float32, device=dev),
            "w": torch.empty(sh.rows, dtype=torch.float32, device=dev)}
    wsf, _ = gca.workspace(p, gca.OP_FORWARD, dev)
    grads = {}
    if backward:
        grads = {"dq": torch.empty(sh.q, dtype=dt, device=dev), "dk": torch.empty(sh.kv, dtype=dt, device=dev),
                 "dv": torch.empty(sh.kv, dtype=dt, device=dev),
                 "dsel": torch.empty(sh.rows, dtype=torch.float32, device=dev),
                 "dlmk_q": torch.empty(sh.lmk_q, dtype=torch.float32, device=dev),
                 "dlmk_k": torch.empty(sh.lmk_k, dtype=torch.float32, device=dev)}
        wsb, _ = gca.workspace(p, gca.OP_BACKWARD, dev)

    def step():
        gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"], ws=wsf, **outs)
        if backward:
            gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], outs["idx"], outs["sel"], outs["lse"], t["dout"],
                                  t["lmk_q"], t["lmk_k"], ws=wsb, grads=grads)

    every = dict(outs, **grads)
    step()
    torch.cuda.synchronize()
    eager = {k: v.clone() for k, v in every.items()}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        for v in every.values():
            v.fill_(-7)
        junk = (t["q"].float() * 3.0).sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in every.items():
            assert torch.equal(v, eager[k]), (rep, k)
        assert torch.isfinite(junk)
    del g


def test_xattn_only_entry_points(dev):
    """gca_grouped_xattn_fwd / _bwd driven with an index set chosen by the caller,
    including pad slots in the middle and an out-of-range index (treated as a pad)."""
    import torch
    from paper_2410_01651_amd import gca
    w = get_workload("tiny_fp32_1k", B=1, H=2, n_chunks=10, topk=4, whole_reseed=False)
    inp = gi.draw_tokens(w, with_dout=True)
    t = upload(w, inp, dev)
    p = problem_for(w)
    nC, k = w.n_chunks, w.topk
    idx = np.full((1, 1, nC, k), -1, np.int32)
    sel = np.full((1, 1, nC, k), -np.inf, np.float32)
    rng = np.random.default_rng(3)
    for r in range(1, nC):
        js = sorted(rng.choice(r, size=min(r, 3), replace=False))
        slots = [0, 2, 3][:len(js)]
        for s, j in zip(slots, js):
            idx[0, 0, r, s] = j
            sel[0, 0, r, s] = rng.standard_normal()
    idx[0, 0, 5, 1] = 10_000          # out of range -> pad
    ti, ts = torch.from_numpy(idx).to(dev), torch.from_numpy(sel).to(dev)
    out, lse, wt = gca.grouped_xattn_fwd(p, t["q"], t["k"], t["v"], ti, ts)
    x = decode_all(w, inp)
    idx_ref = np.where(idx >= nC, -1, idx)
    sel_ref = np.where(idx >= nC, -np.inf, sel).astype(np.float64)
    w_ref = og.fusion_weights(sel_ref)
    o_ref, l_ref = og.xattn_fwd(x["q"], x["k"], x["v"], idx_ref, w_ref, w.S, w.attn_scale)
    assert max_abs_rel(host64(out), o_ref) <= 1e-4
    assert max_abs_rel(host64(lse), l_ref) <= 1e-4
    assert max_abs_rel(host64(wt), w_ref) <= 1e-5
    g = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], ti, ts, lse, t["dout"], landmark_grads=False)
    dq, dk, dv, dw = og.xattn_bwd(x["q"], x["k"], x["v"], idx_ref, w_ref, x["dout"], w.S, w.attn_scale)
    for key, ref in (("dq", dq), ("dk", dk), ("dv", dv), ("dsel", og.dsel_from_dw(w_ref, dw))):
        assert max_abs_rel(host64(g[key]), ref) <= 1e-4, key


@pytest.mark.parametrize("name,lmk_row", [("tiny_fp32_1k", False), ("fwdbwd_64k_bf16", False),
                                          ("tiny_fp32_1k", True), ("fwdbwd_64k_bf16", True)])
def test_backward_hot_key_chunk(dev, name, lmk_row):
    """Every row retrieves chunk 0 (599 retrievers, more than one staged batch of the
    key-stationary pass's list) plus up to two other earlier chunks, from an index set
    chosen by the caller; forward and backward against the oracle.  With S+1 rows the
    LMK rows' staged contractions also cross those batch boundaries."""
    import torch
    from paper_2410_01651_amd import gca
    w = get_workload(name, B=1, H=2, n_chunks=600, topk=4, whole_reseed=False, lmk_row=lmk_row)
    inp = gi.draw_tokens(w, with_dout=True)
    t = upload(w, inp, dev)
    p = problem_for(w)
    nC, k = w.n_chunks, w.topk
    idx = np.full((1, 1, nC, k), -1, np.int32)
    sel = np.full((1, 1, nC, k), -np.inf, np.float32)
    rng = np.random.default_rng(5)
    for r in range(1, nC):
        idx[0, 0, r, 0] = 0
        sel[0, 0, r, 0] = rng.standard_normal()
        if r > 1:
            for s, j in zip((1, 2), sorted(rng.choice(np.arange(1, r), size=min(r - 1, 2), replace=False))):
                idx[0, 0, r, s] = j
                sel[0, 0, r, s] = rng.standard_normal()
    assert int((idx == 0).sum()) == nC - 1
    ti, ts = torch.from_numpy(idx).to(dev), torch.from_numpy(sel).to(dev)
    out, lse, wt = gca.grouped_xattn_fwd(p, t["q"], t["k"], t["v"], ti, ts)
    x = decode_all(w, inp)
    w_ref = og.fusion_weights(sel.astype(np.float64))
    sq = w.Sq if lmk_row else None
    o_ref, _ = og.xattn_fwd(x["q"], x["k"], x["v"], idx, w_ref, w.S, w.attn_scale, Sq=sq)
    assert max_abs_rel(host64(out), o_ref) <= TOL[w.dtype]
    g = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], ti, ts, lse, t["dout"], landmark_grads=False)
    dq, dk, dv, dw = og.xattn_bwd(x["q"], x["k"], x["v"], idx, w_ref, x["dout"], w.S, w.attn_scale, Sq=sq)
    for key, ref in (("dq", dq), ("dk", dk), ("dv", dv), ("dsel", og.dsel_from_dw(w_ref, dw))):
        assert max_abs_rel(host64(g[key]), ref) <= TOL[w.dtype], key


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_decode_xattn_only_entry_point(dev, dtype):
    """gca_grouped_xattn_fwd in decode mode with an index set chosen by the caller:
    pads between valid slots, an out-of-range index (a pad), and a row with no
    valid slot at all."""
    import torch
    from paper_2410_01651_amd import gca
    w = get_workload("decode_16m_bf16", B=2, H=2, Hr=2, D=64, n_chunks=30, topk=6, dtype=dtype, planted=0,
                     device_kv=False)
    inp = gi.draw_tokens(w)
    t = upload(w, inp, dev)
    p = problem_for(w)
    k = w.topk
    idx = np.full((2, 2, 1, k), -1, np.int32)
    sel = np.full((2, 2, 1, k), -np.inf, np.float32)
    rng = np.random.default_rng(11)
    for b, hr, slots in ((0, 0, [0, 2, 5]), (0, 1, [1, 2, 3, 4]), (1, 0, [3])):
        for s, j in zip(slots, sorted(rng.choice(w.n_chunks, size=len(slots), replace=False))):
            idx[b, hr, 0, s] = j
            sel[b, hr, 0, s] = rng.standard_normal()
    idx[0, 1, 0, 3] = 1000            # out of range -> pad
    # row (1, 1) keeps no valid slot
    ti, ts = torch.from_numpy(idx).to(dev), torch.from_numpy(sel).to(dev)
    out, lse, wt = gca.grouped_xattn_fwd(p, t["q"], t["k"], t["v"], ti, ts)
    x = decode_all(w, inp)
    idx_ref = np.where(idx >= w.n_chunks, -1, idx)
    sel_ref = np.where(idx >= w.n_chunks, -np.inf, sel).astype(np.float64)
    w_ref = og.fusion_weights(sel_ref)
    o_ref, l_ref = og.xattn_fwd(x["q"], x["k"], x["v"], idx_ref, w_ref, w.S, w.attn_scale, mode="decode")
    tol = TOL[dtype]
    assert max_abs_rel(host64(out), o_ref) <= tol
    assert max_abs_rel(host64(lse), l_ref) <= tol
    assert max_abs_rel(host64(wt), w_ref) <= 1e-5
    assert not np.any(host64(out)[1, 1])          # the empty row's output is zero


GUMBEL = [
    # name, overrides, problem flags: every selection path with Gumbel top-k
    ("train_16k_bf16", dict(B=2, H=2, n_chunks=70, topk=5, gumbel_seed=11), "materialize"),
    ("train_16k_bf16", dict(B=1, H=2, n_chunks=300, topk=8, gumbel_seed=12, dtype="fp32"), "fused"),
    ("planted_1m_bf16", dict(H=2, n_chunks=500, topk=8, gumbel_seed=13), "fused"),
    ("planted_1m_bf16", dict(H=2, n_chunks=600, topk=12, gumbel_seed=17), "fused"),
    ("decode_16m_bf16", dict(H=2, n_chunks=3001, topk=8, gumbel_seed=14, device_kv=False), None),
    ("decode_16m_bf16", dict(H=1, D=64, n_chunks=40000, topk=4, gumbel_seed=15, device_kv=False), None),
    ("decode_16m_bf16", dict(H=8, n_chunks=2500, topk=8, gumbel_seed=16, device_kv=False), None),
]


@pytest.mark.parametrize("name,kw,path", GUMBEL)
def test_gumbel_forward(dev, name, kw, path):
    """Gumbel top-k selection: the noisy ranking reproduces the oracle's indices
    exactly (margins enforced on the noisy scores) while sel, w and the outputs
    use the raw scores."""
    from paper_2410_01651_amd import gca
    w, inp = _case(name, **kw)
    t = upload(w, inp, dev)
    flags = {"materialize": gca.FLAG_MATERIALIZE, "fused": gca.FLAG_FUSED_TOPK, None: 0}[path]
    f = gca.forward(problem_for(w, flags=flags), t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    ref = _check_forward(w, inp, f)
    plain = og.topk(ref["scores"], w.topk)[0]
    assert not np.array_equal(plain, ref["idx"]), "the noise changed no selection"


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_gumbel_topk_entry_point(dev, dtype):
    """gca_topk with Gumbel selection over a score matrix: exact indices, and sel
    holds the raw matrix entries."""
    import torch
    from paper_2410_01651_amd import gca
    w, inp = _case("train_16k_bf16", B=1, H=2, n_chunks=200, topk=8, dtype=dtype, gumbel_seed=21)
    t = upload(w, inp, dev)
    p = problem_for(w)
    sc = gca.chunk_scores(p, t["lmk_q"], t["lmk_k"])
    idx, sel = gca.topk(p, sc)
    r = sc.double().cpu().numpy()
    ri, rs = og.topk(r, w.topk, gumbel_seed=w.gumbel_seed)
    np.testing.assert_array_equal(idx.cpu().numpy(), ri)
    np.testing.assert_array_equal(sel.cpu().numpy(), rs.astype(np.float32))


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_decode_host_kv(dev, dtype):
    """Decode with the K/V cache in pinned host memory (GCA_FLAG_HOST_KV): the
    attention (and its backward) reads the retrieved chunks over the host link and
    gives exactly what the device-resident cache gives; the oracle agrees;
    unpinned host tensors are refused."""
    import torch
    from paper_2410_01651_amd import gca
    w, inp = _case("decode_16m_bf16", H=2, n_chunks=3000, topk=8, dtype=dtype, device_kv=False)
    t = upload(w, inp, dev)
    kh = torch.empty(t["k"].shape, dtype=t["k"].dtype, pin_memory=True)
    vh = torch.empty(t["v"].shape, dtype=t["v"].dtype, pin_memory=True)
    kh.copy_(t["k"].cpu())
    vh.copy_(t["v"].cpu())
    f_dev = gca.forward(problem_for(w), t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    ph = problem_for(w, flags=gca.FLAG_HOST_KV)
    f_host = gca.forward(ph, t["lmk_q"], t["lmk_k"], t["q"], kh, vh)
    torch.cuda.synchronize()
    for key in ("idx", "sel", "w", "out", "lse"):
        assert torch.equal(f_dev[key], f_host[key]), key
    _check_forward(w, inp, f_host)
    out, lse, wt = gca.grouped_xattn_fwd(ph, t["q"], kh, vh, f_host["idx"], f_host["sel"])
    assert torch.equal(out, f_dev["out"]) and torch.equal(lse, f_dev["lse"])
    dout = torch.randn(t["q"].shape, device=dev).to(t["q"].dtype)
    g_dev = gca.grouped_xattn_bwd(problem_for(w), t["q"], t["k"], t["v"], f_dev["idx"], f_dev["sel"], f_dev["lse"],
                                  dout, t["lmk_q"], t["lmk_k"])
    g_host = gca.grouped_xattn_bwd(ph, t["q"], kh, vh, f_dev["idx"], f_dev["sel"], f_dev["lse"], dout,
                                   t["lmk_q"], t["lmk_k"])
    for key in ("dq", "dk", "dv", "dsel", "dlmk_q", "dlmk_k"):
        assert torch.equal(g_dev[key], g_host[key]), key
    with pytest.raises(gca.GcaError, match="pinned host memory"):
        gca.forward(ph, t["lmk_q"], t["lmk_k"], t["q"], t["k"].cpu(), t["v"].cpu())


def test_selection_reused_by_layers(dev):
    """One selection (gca_topk) serves several layers of a group: each layer runs
    gca_grouped_xattn_fwd / _bwd with its own q, k, v on the same idx / sel."""
    import torch
    from paper_2410_01651_amd import gca
    w, inp = _case("train_16k_bf16", B=1, H=2, n_chunks=40, topk=4)
    t = upload(w, inp, dev)
    p = problem_for(w)
    idx, sel = gca.topk(p, gca.chunk_scores(p, t["lmk_q"], t["lmk_k"]))
    x = decode_all(w, inp)
    ref = og.forward(oracle_params(w), x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"])
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
    for layer in range(1, 3):
        lw = get_workload("train_16k_bf16", B=1, H=2, n_chunks=40, topk=4, seed=100 + layer)
        tok = gi.draw_tokens(lw, with_dout=True)
        tt = upload(lw, tok, dev)
        out, lse, wt = gca.grouped_xattn_fwd(p, tt["q"], tt["k"], tt["v"], idx, sel)
        y = decode_all(lw, tok)
        o_ref, l_ref = og.xattn_fwd(y["q"], y["k"], y["v"], ref["idx"], ref["w"], w.S, w.attn_scale)
        assert max_abs_rel(host64(out), o_ref) <= TOL[w.dtype], layer
        g = gca.grouped_xattn_bwd(p, tt["q"], tt["k"], tt["v"], idx, sel, lse, tt["dout"], landmark_grads=False)
        dq, dk, dv, _ = og.xattn_bwd(y["q"], y["k"], y["v"], ref["idx"], ref["w"], y["dout"], w.S, w.attn_scale)
        for key, r in (("dq", dq), ("dk", dk), ("dv", dv)):
            assert max_abs_rel(host64(g[key]), r) <= TOL[w.dtype], (layer, key)


LMK = [
    # (workload, overrides, off_by_one): S+1 query rows per chunk (the LMK row)
    ("train_16k_bf16", dict(B=2, H=3, n_chunks=70, topk=5), False),
    ("train_16k_bf16", dict(B=2, H=3, n_chunks=70, topk=5, dtype="fp32"), False),
    ("train_16k_bf16", dict(B=1, H=4, n_chunks=40, topk=8), True),
    ("train_16k_bf16", dict(B=1, H=2, n_chunks=50, topk=12, Hr=2, D=128), False),  # k > 8, per-head retrieval
    ("train_16k_bf16", dict(B=1, H=2, n_chunks=20, topk=1), False),
    ("fwdbwd_64k_bf16", dict(B=1, H=4, n_chunks=96, topk=8), False),
    # edges: one chunk (everything empty), k above the history, k = 32 (unstaged
    # per-slot values), fp32 with off-by-one, uneven streams
    ("train_16k_bf16", dict(B=1, H=2, n_chunks=1, topk=4), False),
    ("train_16k_bf16", dict(B=2, H=2, n_chunks=3, topk=8), False),
    ("train_16k_bf16", dict(B=1, H=2, n_chunks=65, topk=32), True),
    ("tiny_fp32_1k", dict(B=2, H=3, n_chunks=37, topk=6, whole_reseed=False), True),
    ("fwdbwd_64k_bf16", dict(B=1, H=2, n_chunks=700, topk=3), False),
    ("fwdbwd_64k_bf16", dict(B=1, H=2, n_chunks=2100, topk=3), False),   # window stream order
    ("fwdbwd_64k_bf16", dict(B=1, H=1, n_chunks=2100, topk=12), True),   # window order, unstaged k, off-by-one
]


@pytest.mark.parametrize("name,kw,obo", LMK)
def test_lmk_rows_forward_backward(dev, name, kw, obo):
    """S+1 query rows per chunk (GCA_FLAG_LMK_ROW): out, lse, w and every gradient
    against the oracle; the LMK rows of chunks >= 2 are really attended."""
    from paper_2410_01651_amd import gca
    w, inp = _case(name, lmk_row=True, **kw)
    assert w.Sq == w.S + 1
    if "dout" not in inp:
        inp["dout"] = gi.draw_slices(w, "dout", (w.B, w.H, w.Lq, w.d))
    t = upload(w, inp, dev)
    p = problem_for(w, off_by_one=obo)
    f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    assert tuple(f["out"].shape) == (w.B, w.H, w.n_chunks * (w.S + 1), w.d)
    ref = _check_forward(w, inp, f, off_by_one=obo)
    lmk_out = host64(f["out"]).reshape(w.B, w.H, w.n_chunks, w.S + 1, w.d)[:, :, :, w.S]
    assert np.all(lmk_out[:, :, :2] == 0.0)
    if w.n_chunks > 2:
        assert np.abs(lmk_out[:, :, 2:]).min(axis=-1).max() > 0.0
    g = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"],
                              t["lmk_q"], t["lmk_k"])
    x = decode_all(w, inp)
    rb = og.backward(oracle_params(w, obo), ref, x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"], x["dout"])
    for key in ("dq", "dk", "dv", "dsel", "dlmk_q", "dlmk_k"):
        e = max_abs_rel(host64(g[key]), rb[key])
        assert e <= TOL[w.dtype], (key, e)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_max_landmark_width(dev, dtype):
    """The widest landmarks the library takes (D = 8192): the score matrix path and
    the one-pass select of the forward, the backward's landmark gradients, and a
    decode scan, against the oracle."""
    from paper_2410_01651_amd import gca
    w, inp = _case("fwdbwd_64k_bf16", B=1, H=2, D=8192, n_chunks=60, topk=4, dtype=dtype)
    t = upload(w, inp, dev)
    tol = TOL[w.dtype]
    x = decode_all(w, inp)
    pp = oracle_params(w)
    rf = og.forward(pp, x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"])
    rb = og.backward(pp, rf, x["lmk_q"], x["lmk_k"], x["q"], x["k"], x["v"], x["dout"])
    for flags in (gca.FLAG_MATERIALIZE, gca.FLAG_FUSED_TOPK):
        p = problem_for(w, flags=flags)
        f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
        np.testing.assert_array_equal(f["idx"].cpu().numpy(), rf["idx"])
        for key in ("sel", "w", "out", "lse"):
            assert max_abs_rel(host64(f[key]), rf[key]) <= tol, (flags, key)
    g = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"],
                              t["lmk_q"], t["lmk_k"])
    for key in ("dq", "dk", "dv", "dsel", "dlmk_q", "dlmk_k"):
        assert max_abs_rel(host64(g[key]), rb[key]) <= tol, key
    wd, ind = _case("decode_16m_bf16", H=2, D=8192, n_chunks=300, dtype=dtype, device_kv=False)
    td = upload(wd, ind, dev)
    fd = gca.forward(problem_for(wd), td["lmk_q"], td["lmk_k"], td["q"], td["k"], td["v"])
    _check_forward(wd, ind, fd)


def test_side_stream(dev):
    """The forward and backward enqueued on a side stream (the binding allocates
    their outputs and workspaces for that stream) give bit for bit what the
    default stream gives."""
    import torch
    from paper_2410_01651_amd import gca
    w, inp = _case("fwdbwd_64k_bf16", B=1, H=4, n_chunks=96, topk=8)
    t = upload(w, inp, dev)
    p = problem_for(w)
    f0 = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    g0 = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f0["idx"], f0["sel"], f0["lse"], t["dout"],
                               t["lmk_q"], t["lmk_k"])
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    f1 = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"], stream=side)
    g1 = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f1["idx"], f1["sel"], f1["lse"], t["dout"],
                               t["lmk_q"], t["lmk_k"], stream=side)
    side.synchronize()
    for key in ("out", "idx", "sel", "lse", "w"):
        assert torch.equal(f0[key], f1[key]), key
    for key in g0:
        assert torch.equal(g0[key], g1[key]), key


def test_concurrent_streams(dev):
    """Two different problems in flight at once on two streams (each call with its
    own workspace: the library keeps no per-call state of its own), interleaved
    launch by launch, give bit for bit what each gives alone."""
    import torch
    from paper_2410_01651_amd import gca
    cases = [_case("fwdbwd_64k_bf16", B=1, H=4, n_chunks=96, topk=8),
             _case("train_16k_bf16", B=2, H=3, n_chunks=70, topk=5, lmk_row=True)]
    probs, ts, alone = [], [], []
    for w, inp in cases:
        if "dout" not in inp:
            inp["dout"] = gi.draw_slices(w, "dout", (w.B, w.H, w.Lq, w.d))
        t = upload(w, inp, dev)
        p = problem_for(w)
        f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
        g = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"],
                                  t["lmk_q"], t["lmk_k"])
        probs.append(p)
        ts.append(t)
        alone.append(dict(f, **g))
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for rep in range(3):
        fs = [gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"], stream=s)
              for p, t, s in zip(probs, ts, streams)]
        gs = [gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"],
                                    t["lmk_q"], t["lmk_k"], stream=s)
              for p, t, f, s in zip(probs, ts, fs, streams)]
        for s in streams:
            s.synchronize()
        for ref, f, g in zip(alone, fs, gs):
            for key, v in dict(f, **g).items():
                assert torch.equal(v, ref[key]), (rep, key)


_DEBUG_SYNC_CHILD = r"""
import hashlib, sys
sys.path.insert(0, sys.argv[1])
sys.path.insert(0, sys.argv[1] + "/tests")
import torch
from _helpers import problem_for, upload
from gen import get_workload
from oracle import margins
from paper_2410_01651_amd import gca
w = get_workload("fwdbwd_64k_bf16", B=1, H=2, n_chunks=40, topk=4)
inp, _ = margins.checked_inputs(w)
t = upload(w, inp, torch.device("cuda:0"))
p = problem_for(w)
f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
g = gca.grouped_xattn_bwd(p, t["q"], t["k"], t["v"], f["idx"], f["sel"], f["lse"], t["dout"], t["lmk_q"], t["lmk_k"])
h = hashlib.sha256()
for d in (f, g):
    for key in sorted(d):
        h.update(d[key].cpu().contiguous().view(torch.uint8).numpy().tobytes())
print(h.hexdigest())
"""


def test_debug_sync_mode(dev):
    """GCA_DEBUG_SYNC=1 (every launch synchronised and checked) gives bit for bit
    the results of the ordinary mode, in a child process that reads it at load."""
    import os
    import subprocess
    import sys
    from _helpers import ROOT
    env = dict(os.environ)
    outs = []
    for mode in ("0", "1"):
        env["GCA_DEBUG_SYNC"] = mode
        r = subprocess.run([sys.executable, "-c", _DEBUG_SYNC_CHILD, ROOT], env=env, capture_output=True,
                           text=True, timeout=240)
        assert r.returncode == 0, r.stderr[-2000:]
        outs.append(r.stdout.strip().splitlines()[-1])
    assert outs[0] == outs[1]


def test_profile_hook(dev):
    """The per-kernel timing hook: kernels are timed in launch order up to the
    capacity, named, with positive durations, and the results do not change."""
    import ctypes
    import torch
    from paper_2410_01651_amd import gca
    w, inp = _case("tiny_fp32_1k")
    t = upload(w, inp, dev)
    p = problem_for(w)
    ref = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    ev = (ctypes.c_void_p * 4)()
    for i in range(4):
        assert hip.hipEventCreate(ctypes.byref(ev, i * ctypes.sizeof(ctypes.c_void_p))) == 0
    try:
        torch.cuda.synchronize()
        gca.profile_arm(ev, 4)                     # room for two kernels of the three
        f = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
        torch.cuda.synchronize()
        names = gca.profile_record()
        gca.profile_arm(None, 0)
        assert names == ["chunk_scores_kernel", "topk_kernel"]
        for i in range(2):
            ms = ctypes.c_float()
            assert hip.hipEventElapsedTime(ctypes.byref(ms), ev[2 * i], ev[2 * i + 1]) == 0
            assert ms.value > 0.0
        for key in ("out", "idx", "sel", "lse", "w"):
            assert torch.equal(f[key], ref[key]), key
        gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])  # disarmed: nothing recorded
        torch.cuda.synchronize()
        assert gca.profile_record() == []
    finally:
        gca.profile_arm(None, 0)
        for i in range(4):
            hip.hipEventDestroy(ctypes.c_void_p(ev[i]))
