"""gca_forward_noalloc through the C ABI: the same results as gca_forward on the
same inputs (the same kernels run, so bit for bit), on two calls in a row whose
second problem is smaller, for the decode scan, the materialised causal path
and the single-pass causal select; and the size limit is enforced before any
launch."""

import numpy as np
import pytest

from _helpers import ensure_built, problem_for, to_dev
from gen import get_workload, inputs as gi
from oracle import margins

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ensure_built()
    return torch.device("cuda:0")


def _inputs(w, dev):
    inp, _ = margins.checked_inputs(w, tokens=False)
    t = {"lmk_q": to_dev(w.dtype, inp["lmk_q"], dev), "lmk_k": to_dev(w.dtype, inp["lmk_k"], dev)}
    t.update(gi.device_tensors(w, ("q", "k", "v"), dev))
    return t


def _outputs(p, dev):
    import torch
    from paper_2410_01651_amd import gca
    sh = gca.shapes(p)
    dt = torch.bfloat16 if p.dtype == gca.GCA_BF16 else torch.float32
    # filled with garbage so that every element the call must write is checked
    return {"out": torch.full(sh.q, 7.0, dtype=dt, device=dev),
            "idx": torch.full(sh.rows, 12345, dtype=torch.int32, device=dev),
            "sel": torch.full(sh.rows, 3.0, dtype=torch.float32, device=dev),
            "lse": torch.full(sh.lse, 5.0, dtype=torch.float32, device=dev),
            "w": torch.full(sh.rows, 9.0, dtype=torch.float32, device=dev)}


def _same(a, b):
    import torch
    for key in ("out", "idx", "sel", "lse", "w"):
        x, y = a[key], b[key]
        if x.dtype == torch.bfloat16:
            x, y = x.view(torch.int16), y.view(torch.int16)
        assert torch.equal(x, y), key


CASES = [
    # (workload, first overrides, second (smaller) overrides, flags)
    ("decode_16m_bf16", dict(H=4, n_chunks=40_000), dict(H=2, n_chunks=5_000), 0),
    ("train_16k_bf16", dict(B=2, H=4, n_chunks=300), dict(B=1, H=2, n_chunks=90), 0),
    ("planted_1m_bf16", dict(H=2, n_chunks=2_000), dict(H=2, n_chunks=700), 1),
    ("tiny_fp32_1k", dict(B=2, H=2, n_chunks=80, topk=3), dict(B=1, H=1, n_chunks=16), 0),
    # S+1 query rows per chunk
    ("train_16k_bf16", dict(B=1, H=4, n_chunks=200, lmk_row=True), dict(B=1, H=2, n_chunks=70, lmk_row=True), 0),
]


@pytest.mark.parametrize("name,first,second,fused", CASES)
def test_noalloc_matches_forward(dev, name, first, second, fused):
    import torch
    from paper_2410_01651_amd import gca
    for n, kw in enumerate((first, second)):
        w = get_workload(name, **kw)
        flags = gca.FLAG_FUSED_TOPK if fused else 0
        p = problem_for(w, flags=flags)
        assert gca.workspace_size(p, gca.OP_FORWARD) <= gca.NOALLOC_SCRATCH_BYTES
        t = _inputs(w, dev)
        ref = gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"])
        o = _outputs(p, dev)
        gca.forward_noalloc(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"], **o)
        torch.cuda.synchronize()
        _same(o, ref)
        if w.planted:
            assert int(gi.plant_positions(w)[0]) in o["idx"].cpu().numpy().ravel().tolist(), n


def test_noalloc_rejects_too_large(dev):
    import torch
    from paper_2410_01651_amd import gca
    # a materialised 4,096 x 4,096 score matrix needs 64 MiB of workspace
    p = gca.problem(1, 1, 4096, 8, D=64, flags=gca.FLAG_MATERIALIZE)
    assert gca.workspace_size(p, gca.OP_FORWARD) > gca.NOALLOC_SCRATCH_BYTES
    sh = gca.shapes(p)
    bf = torch.bfloat16
    lq = torch.zeros(sh.lmk_q, dtype=bf, device=dev)
    lk = torch.zeros(sh.lmk_k, dtype=bf, device=dev)
    q = torch.zeros(sh.q, dtype=bf, device=dev)
    kv = torch.zeros(sh.kv, dtype=bf, device=dev)
    o = _outputs(p, dev)
    with pytest.raises(gca.GcaError) as e:
        gca.forward_noalloc(p, lq, lk, q, kv, kv, **o)
    assert e.value.status == gca.GCA_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert torch.all(o["idx"] == 12345)          # nothing was launched
