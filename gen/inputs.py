"""Seeded input draws for the GCA workloads.

Every tensor is i.i.d. N(0,1), drawn in fp64 from
``PCG64(SeedSequence([seed, tensor_id, *slice]))`` and stored in the
workload's dtype: fp32 arrays for fp32 workloads, bf16 bit patterns (uint16,
rounded to nearest-even from fp64) for bf16 workloads.  Per-token tensors are
drawn one (batch, head) slice at a time so that any slice can be redrawn on its
own.

Layouts (row-major):

* landmark queries ``lmk_q``  [B, Hr, nQ, D]   (one per query chunk)
* landmark keys    ``lmk_k``  [B, Hr, nC, D]   (one per key chunk)
* ``q``                        [B, H, nQ*S, d]
* ``k``, ``v``                 [B, H, nC*S, d]
* upstream gradient ``dout``   [B, H, nQ*S, d]

Planted long-range targets: the planted key chunks get the landmark key
``4 * lmk_q[target row]`` (exact in bf16 and fp32), so that the target row's
top-k set is known in closed form.
"""

import numpy as np

from . import bf16 as _bf16
from .workloads import Workload

TENSOR_ID = {"lmk_q": 0, "lmk_k": 1, "q": 2, "k": 3, "v": 4, "dout": 5,
             "plant": 6, "row_redraw": 100}


def rng(seed: int, *sub: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *sub])))


def encode(w: Workload, x64: np.ndarray) -> np.ndarray:
    """Store fp64 draws in the workload dtype (fp32 array or bf16 bits)."""
    if w.dtype == "bf16":
        return _bf16.from_f64(x64)
    return x64.astype(np.float32)


def decode(w_or_dtype, arr: np.ndarray) -> np.ndarray:
    """Exact fp64 view of stored values."""
    dtype = w_or_dtype if isinstance(w_or_dtype, str) else w_or_dtype.dtype
    if dtype == "bf16":
        return _bf16.to_f64(arr)
    return np.asarray(arr, dtype=np.float64)


def _store_dtype(w: Workload):
    return np.uint16 if w.dtype == "bf16" else np.float32


def _attempt_sub(w: Workload, attempt: int):
    # whole-input reseeding keys every stream on the attempt number
    return (attempt,) if w.whole_reseed else ()


def draw_slices(w: Workload, name: str, shape, attempt: int = 0) -> np.ndarray:
    """Draw a [B, X, rows, cols] tensor one (b, x) slice at a time."""
    B, X, rows, cols = shape
    out = np.empty(shape, dtype=_store_dtype(w))
    tid = TENSOR_ID[name]
    for b in range(B):
        for x in range(X):
            g = rng(w.seed, tid, *_attempt_sub(w, attempt), b, x)
            out[b, x] = encode(w, g.standard_normal((rows, cols)))
    return out


def plant_positions(w: Workload) -> np.ndarray:
    """Distinct planted key-chunk positions, ascending (empty if none)."""
    if not w.planted:
        return np.zeros(0, dtype=np.int64)
    g = rng(w.seed, TENSOR_ID["plant"])
    hi = w.n_chunks if w.mode == "decode" else w.n_chunks - 1   # causal: < last row
    pos = g.choice(hi, size=w.planted, replace=False)
    return np.sort(pos.astype(np.int64))


def plant_target_row(w: Workload) -> int:
    return 0 if w.mode == "decode" else w.n_chunks - 1


def apply_plant(w: Workload, lmk_q: np.ndarray, lmk_k: np.ndarray) -> None:
    """Set the planted keys to 4x the target row's landmark query (in place)."""
    if not w.planted:
        return
    pos = plant_positions(w)
    t = plant_target_row(w)
    for b in range(lmk_q.shape[0]):
        for hr in range(lmk_q.shape[1]):
            scaled = encode(w, 4.0 * decode(w, lmk_q[b, hr, t]))
            lmk_k[b, hr, pos] = scaled[None, :]


def draw_landmarks(w: Workload, attempt: int = 0):
    """Landmark queries and keys, with planted targets applied."""
    nQ = w.n_query_chunks
    lmk_q = draw_slices(w, "lmk_q", (w.B, w.Hr, nQ, w.Dl), attempt)
    lmk_k = draw_slices(w, "lmk_k", (w.B, w.Hr, w.n_chunks, w.Dl), attempt)
    apply_plant(w, lmk_q, lmk_k)
    return lmk_q, lmk_k


def redraw_lmk_q_row(w: Workload, lmk_q: np.ndarray, lmk_k: np.ndarray,
                     b: int, hr: int, t: int, attempt: int) -> None:
    """Replace one landmark query row by a fresh draw (in place).

    The draw comes from ``SeedSequence([seed, 100, b, hr, t, attempt])``.  If
    the row is a planted target, its planted keys follow it.
    """
    g = rng(w.seed, TENSOR_ID["row_redraw"], b, hr, t, attempt)
    lmk_q[b, hr, t] = encode(w, g.standard_normal(w.Dl))
    if w.planted and t == plant_target_row(w):
        pos = plant_positions(w)
        lmk_k[b, hr, pos] = encode(w, 4.0 * decode(w, lmk_q[b, hr, t]))[None, :]


def draw_tokens(w: Workload, attempt: int = 0, with_dout: bool = None):
    """Per-token q, k, v (and dout for backward workloads) on the host."""
    out = {
        "q": draw_slices(w, "q", (w.B, w.H, w.Lq, w.d), attempt),
        "k": draw_slices(w, "k", (w.B, w.H, w.Lkv, w.d), attempt),
        "v": draw_slices(w, "v", (w.B, w.H, w.Lkv, w.d), attempt),
    }
    if with_dout is None:
        with_dout = w.backward
    if with_dout:
        out["dout"] = draw_slices(w, "dout", (w.B, w.H, w.Lq, w.d), attempt)
    return out


def draw_inputs(w: Workload, attempt: int = 0, tokens: bool = True):
    """All host-side inputs of a workload (no margin enforcement)."""
    lmk_q, lmk_k = draw_landmarks(w, attempt)
    inp = {"lmk_q": lmk_q, "lmk_k": lmk_k}
    if tokens and not w.device_kv:
        inp.update(draw_tokens(w, attempt))
    elif tokens:
        inp["q"] = draw_slices(w, "q", (w.B, w.H, w.Lq, w.d), attempt)
        if w.backward:
            inp["dout"] = draw_slices(w, "dout", (w.B, w.H, w.Lq, w.d), attempt)
    return inp


def device_tensors(w: Workload, names, device, torch_mod=None):
    """Per-token tensors drawn on the device, for workloads too large for the host.

    Each (b, h) slice of each named tensor (q and dout are [B,H,Lq,d], k and v
    [B,H,Lkv,d]) is i.i.d. N(0,1) from a torch device generator seeded with
    ``seed * 1_000_003 + tensor_id * 10_007 + b * 131 + h`` and stored in the
    workload dtype.  Tests read back only the slices they need.
    """
    import torch as _t
    torch = torch_mod or _t
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    out = {}
    for name in names:
        rows = w.Lq if name in ("q", "dout") else w.Lkv
        t = torch.empty((w.B, w.H, rows, w.d), dtype=dt, device=device)
        for b in range(w.B):
            for h in range(w.H):
                g = torch.Generator(device=device)
                g.manual_seed(w.seed * 1_000_003 + TENSOR_ID[name] * 10_007 + b * 131 + h)
                t[b, h].normal_(generator=g)
        out[name] = t
    return out


def device_kv(w: Workload, device, torch_mod=None):
    """The K/V cache of a workload drawn on the device (see device_tensors)."""
    return device_tensors(w, ("k", "v"), device, torch_mod)
