"""Shared test plumbing: device upload of generator outputs, the oracle's
problem dict, and the max-abs-rel error measure (per tensor:
max |x - ref| / max |ref|)."""

import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from gen import inputs as gi  # noqa: E402

TOL = {"fp32": 1e-4, "bf16": 2e-2}


def ensure_built():
    from paper_2410_01651_amd import build as b
    if not os.path.exists(b.OUT):
        b.build()


def to_dev(dtype, a, dev):
    import torch
    a = np.ascontiguousarray(a)
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(a.astype(np.float32)).to(dev)


def host64(t):
    """Exact fp64 copy of a device tensor (bf16 and fp32 widen exactly)."""
    return t.detach().float().cpu().double().numpy()


def max_abs_rel(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert x.shape == ref.shape, (x.shape, ref.shape)
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(x)), "non-finite pattern differs"
    if not fin.any():
        return 0.0
    scale = np.abs(ref[fin]).max()
    diff = np.abs(x[fin] - ref[fin]).max()
    return float(diff / scale) if scale > 0 else float(diff)


def _gumbel(w):
    return w.gumbel_seed if w.gumbel_seed >= 0 else None


def oracle_params(w, off_by_one=False):
    return dict(S=w.S, topk=w.topk, score_scale=w.score_scale, attn_scale=w.attn_scale,
                mode=w.mode, off_by_one=off_by_one, gumbel_seed=_gumbel(w), Sq=w.Sq)


def problem_for(w, off_by_one=False, flags=0):
    from paper_2410_01651_amd import gca
    return gca.problem(w.B, w.H, w.n_chunks, w.topk, D=w.Dl, Hr=w.Hr, dtype=w.dtype, mode=w.mode,
                       off_by_one=off_by_one, flags=flags, gumbel_seed=_gumbel(w), lmk_row=w.lmk_row)


def upload(w, inp, dev):
    return {k: to_dev(w.dtype, v, dev) for k, v in inp.items()}


def decode_all(w, inp):
    return {k: gi.decode(w, v) for k, v in inp.items()}
