"""Python binding of libgca (ctypes; argument marshalling only).

Every function here forwards to the C entry point of the same name in
``include/gca.h``: it checks that the tensors are contiguous device tensors of
the expected dtype, allocates the outputs (and workspace) with torch, and passes
raw device pointers plus torch's current HIP stream.  All arithmetic runs in the
library's HIP kernels; nothing here computes.  A missing library raises.
"""

import ctypes
import math
import os
from dataclasses import dataclass

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgca.so")

EXPORTS = (
    "gca_chunk_scores",
    "gca_topk",
    "gca_grouped_xattn_fwd",
    "gca_grouped_xattn_bwd",
    "gca_forward",
    "gca_forward_noalloc",
    "gca_workspace_size",
    "gca_status_string",
    "gca_last_error",
    "gca_profile_arm",
    "gca_profile_count",
    "gca_profile_name",
)

GCA_OK, GCA_ERR_INVALID, GCA_ERR_UNSUPPORTED, GCA_ERR_WORKSPACE, GCA_ERR_HIP = range(5)
GCA_FP32, GCA_BF16 = 0, 1
GCA_CAUSAL, GCA_DECODE = 0, 1
FLAG_FUSED_TOPK, FLAG_MATERIALIZE, FLAG_GUMBEL, FLAG_HOST_KV, FLAG_LMK_ROW = 1, 2, 4, 8, 16
OP_FORWARD, OP_BACKWARD = 0, 1
NOALLOC_SCRATCH_BYTES = 16 << 20


class Problem(ctypes.Structure):
    """Mirror of ``gca_problem``."""

    _fields_ = [
        ("B", ctypes.c_int32),
        ("H", ctypes.c_int32),
        ("d", ctypes.c_int32),
        ("S", ctypes.c_int32),
        ("n_chunks", ctypes.c_int64),
        ("topk", ctypes.c_int32),
        ("Hr", ctypes.c_int32),
        ("D", ctypes.c_int32),
        ("score_scale", ctypes.c_float),
        ("attn_scale", ctypes.c_float),
        ("off_by_one", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("mode", ctypes.c_int32),
        ("flags", ctypes.c_uint32),
        ("gumbel_seed", ctypes.c_uint64),
    ]

    @property
    def n_query_chunks(self) -> int:
        return self.n_chunks if self.mode == GCA_CAUSAL else 1

    @property
    def query_rows(self) -> int:
        """Query rows per chunk: S, or S + 1 with the LMK row (GCA_FLAG_LMK_ROW)."""
        return self.S + 1 if self.flags & FLAG_LMK_ROW else self.S


class GcaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


_lib = None


def lib():
    """The loaded libgca (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libgca is not built ({LIB_PATH} missing); run "
                               "`python -m paper_2410_01651_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, P = ctypes.c_void_p, ctypes.POINTER(Problem)
        sig = {
            "gca_chunk_scores": [P, vp, vp, vp, vp],
            "gca_topk": [P, vp, vp, vp, vp],
            "gca_grouped_xattn_fwd": [P, vp, vp, vp, vp, vp, vp, vp, vp, vp],
            "gca_grouped_xattn_bwd": [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                      vp, ctypes.c_size_t, vp],
            "gca_forward": [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp],
            "gca_forward_noalloc": [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        L.gca_workspace_size.argtypes = [P, ctypes.c_int]
        L.gca_workspace_size.restype = ctypes.c_size_t
        L.gca_status_string.argtypes = [ctypes.c_int]
        L.gca_status_string.restype = ctypes.c_char_p
        L.gca_last_error.argtypes = []
        L.gca_last_error.restype = ctypes.c_char_p
        L.gca_profile_arm.argtypes = [ctypes.c_void_p, ctypes.c_int]
        L.gca_profile_arm.restype = None
        L.gca_profile_count.argtypes = []
        L.gca_profile_count.restype = ctypes.c_int
        L.gca_profile_name.argtypes = [ctypes.c_int]
        L.gca_profile_name.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != GCA_OK:
        L = lib()
        raise GcaError(status, f"{L.gca_status_string(status).decode()}: {L.gca_last_error().decode()}")


def problem(B, H, n_chunks, topk, D=None, Hr=1, d=64, S=64, score_scale=None, attn_scale=None,
            off_by_one=False, dtype="bf16", mode="causal", flags=0, gumbel_seed=None,
            lmk_row=False) -> Problem:
    """Build a ``gca_problem``; D defaults to H*d, scales to 1/sqrt(D) and 1/sqrt(d).
    A ``gumbel_seed`` turns on Gumbel top-k selection (GCA_FLAG_GUMBEL);
    ``lmk_row`` gives every query chunk S + 1 rows (GCA_FLAG_LMK_ROW)."""
    D = H * d if D is None else D
    if gumbel_seed is not None:
        flags |= FLAG_GUMBEL
    if lmk_row:
        flags |= FLAG_LMK_ROW
    return Problem(
        B=B, H=H, d=d, S=S, n_chunks=n_chunks, topk=topk, Hr=Hr, D=D,
        score_scale=1.0 / math.sqrt(D) if score_scale is None else score_scale,
        attn_scale=1.0 / math.sqrt(d) if attn_scale is None else attn_scale,
        off_by_one=int(bool(off_by_one)),
        dtype={"fp32": GCA_FP32, "bf16": GCA_BF16}[dtype] if isinstance(dtype, str) else dtype,
        mode={"causal": GCA_CAUSAL, "decode": GCA_DECODE}[mode] if isinstance(mode, str) else mode,
        flags=flags,
        gumbel_seed=0 if gumbel_seed is None else int(gumbel_seed),
    )


# ----------------------------------------------------------- marshalling ----

def _torch():
    import torch
    return torch


def _elem_dtype(p: Problem):
    torch = _torch()
    return torch.bfloat16 if p.dtype == GCA_BF16 else torch.float32


def _ptr(t, name, dtype=None, shape=None, host_ok=False):
    if t is None:
        return None
    # a host tensor (GCA_FLAG_HOST_KV) is checked by the library itself: it must
    # be pinned memory with a device mapping (torch's is_pinned() query costs far
    # more than the call it would guard)
    if not t.is_cuda and not host_ok:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _host_kv(p: Problem) -> bool:
    return bool(p.flags & FLAG_HOST_KV)


def _stream(stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _alloc_on(stream):
    """Context for allocating outputs and workspace that the kernels use on
    `stream`: torch's caching allocator then ties the blocks to that stream, so a
    temporary freed on return is not handed to other streams' work while the
    kernels may still run."""
    import contextlib
    if stream is None:
        return contextlib.nullcontext()
    return _torch().cuda.stream(stream)


@dataclass
class Shapes:
    lmk_q: tuple
    lmk_k: tuple
    q: tuple
    kv: tuple
    rows: tuple     # [B, Hr, nQ, topk]
    scores: tuple   # [B, Hr, nQ, nC]
    lse: tuple      # [B, H, Lq, topk]


def shapes(p: Problem) -> Shapes:
    nQ, nC = p.n_query_chunks, p.n_chunks
    return Shapes(
        lmk_q=(p.B, p.Hr, nQ, p.D), lmk_k=(p.B, p.Hr, nC, p.D),
        q=(p.B, p.H, nQ * p.query_rows, p.d), kv=(p.B, p.H, nC * p.S, p.d),
        rows=(p.B, p.Hr, nQ, p.topk), scores=(p.B, p.Hr, nQ, nC),
        lse=(p.B, p.H, nQ * p.query_rows, p.topk),
    )


def workspace_size(p: Problem, op: int) -> int:
    return int(lib().gca_workspace_size(ctypes.byref(p), op))


def workspace(p: Problem, op: int, device="cuda"):
    torch = _torch()
    n = workspace_size(p, op)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=device), n


# ------------------------------------------------------------ entry points ----

def chunk_scores(p: Problem, lmk_q, lmk_k, scores=None, stream=None):
    torch = _torch()
    sh, dt = shapes(p), _elem_dtype(p)
    with _alloc_on(stream):
        if scores is None:
            scores = torch.empty(sh.scores, dtype=torch.float32, device=lmk_q.device)
    _check(lib().gca_chunk_scores(ctypes.byref(p), _ptr(lmk_q, "lmk_q", dt, sh.lmk_q),
                                  _ptr(lmk_k, "lmk_k", dt, sh.lmk_k),
                                  _ptr(scores, "scores", torch.float32, sh.scores), _stream(stream)))
    return scores


def topk(p: Problem, scores, idx=None, sel=None, stream=None):
    torch = _torch()
    sh = shapes(p)
    with _alloc_on(stream):
        if idx is None:
            idx = torch.empty(sh.rows, dtype=torch.int32, device=scores.device)
        if sel is None:
            sel = torch.empty(sh.rows, dtype=torch.float32, device=scores.device)
    _check(lib().gca_topk(ctypes.byref(p), _ptr(scores, "scores", torch.float32, sh.scores),
                          _ptr(idx, "idx", torch.int32, sh.rows), _ptr(sel, "sel", torch.float32, sh.rows),
                          _stream(stream)))
    return idx, sel


def grouped_xattn_fwd(p: Problem, q, k, v, idx, sel, out=None, lse=None, w=None, want_lse=True,
                      want_w=True, stream=None):
    torch = _torch()
    sh, dt = shapes(p), _elem_dtype(p)
    dev = q.device
    with _alloc_on(stream):
        if out is None:
            out = torch.empty(sh.q, dtype=dt, device=dev)
        if lse is None and want_lse:
            lse = torch.empty(sh.lse, dtype=torch.float32, device=dev)
        if w is None and want_w:
            w = torch.empty(sh.rows, dtype=torch.float32, device=dev)
    _check(lib().gca_grouped_xattn_fwd(
        ctypes.byref(p), _ptr(q, "q", dt, sh.q),
        _ptr(k, "k", dt, sh.kv, _host_kv(p)), _ptr(v, "v", dt, sh.kv, _host_kv(p)),
        _ptr(idx, "idx", torch.int32, sh.rows), _ptr(sel, "sel", torch.float32, sh.rows),
        _ptr(out, "out", dt, sh.q), _ptr(lse, "lse", torch.float32, sh.lse),
        _ptr(w, "w", torch.float32, sh.rows), _stream(stream)))
    return out, lse, w


def grouped_xattn_bwd(p: Problem, q, k, v, idx, sel, lse, dout, lmk_q=None, lmk_k=None,
                      landmark_grads=True, ws=None, grads=None, stream=None):
    """Returns dict dq, dk, dv, dsel and (if landmark_grads) dlmk_q, dlmk_k.
    landmark_grads: True (both), False (neither), or a collection of the names
    "dlmk_q" / "dlmk_k" to request one of them."""
    torch = _torch()
    sh, dt = shapes(p), _elem_dtype(p)
    dev = q.device
    g = dict(grads or {})
    if landmark_grads is True:
        wanted = ("dlmk_q", "dlmk_k")
    elif not landmark_grads:
        wanted = ()
    else:
        wanted = tuple(landmark_grads)
        if not set(wanted) <= {"dlmk_q", "dlmk_k"}:
            raise ValueError(f"landmark_grads names must be dlmk_q / dlmk_k, got {wanted}")
    landmark_grads = bool(wanted)
    with _alloc_on(stream):
        for name, shape, gdt in (("dq", sh.q, dt), ("dk", sh.kv, dt), ("dv", sh.kv, dt),
                                 ("dsel", sh.rows, torch.float32)):
            if name not in g:
                g[name] = torch.empty(shape, dtype=gdt, device=dev)
        for name, shape in (("dlmk_q", sh.lmk_q), ("dlmk_k", sh.lmk_k)):
            if name in wanted and name not in g:
                g[name] = torch.empty(shape, dtype=torch.float32, device=dev)
        if ws is None:
            ws, nbytes = workspace(p, OP_BACKWARD, dev)
        else:
            nbytes = ws.numel()
    _check(lib().gca_grouped_xattn_bwd(
        ctypes.byref(p), _ptr(q, "q", dt, sh.q),
        _ptr(k, "k", dt, sh.kv, _host_kv(p)), _ptr(v, "v", dt, sh.kv, _host_kv(p)),
        _ptr(idx, "idx", torch.int32, sh.rows), _ptr(sel, "sel", torch.float32, sh.rows),
        _ptr(lse, "lse", torch.float32, sh.lse), _ptr(dout, "dout", dt, sh.q),
        _ptr(g["dq"], "dq", dt, sh.q), _ptr(g["dk"], "dk", dt, sh.kv), _ptr(g["dv"], "dv", dt, sh.kv),
        _ptr(g["dsel"], "dsel", torch.float32, sh.rows),
        _ptr(lmk_q, "lmk_q", dt, sh.lmk_q) if landmark_grads else None,
        _ptr(lmk_k, "lmk_k", dt, sh.lmk_k) if landmark_grads else None,
        _ptr(g.get("dlmk_q") if "dlmk_q" in wanted else None, "dlmk_q", torch.float32, sh.lmk_q),
        _ptr(g.get("dlmk_k") if "dlmk_k" in wanted else None, "dlmk_k", torch.float32, sh.lmk_k),
        _ptr(ws, "workspace"), ctypes.c_size_t(nbytes), _stream(stream)))
    return g


def forward(p: Problem, lmk_q, lmk_k, q, k, v, out=None, idx=None, sel=None, lse=None, w=None,
            want_lse=True, want_w=True, ws=None, stream=None):
    """The whole path; returns dict out, idx, sel, lse, w."""
    torch = _torch()
    sh, dt = shapes(p), _elem_dtype(p)
    dev = q.device
    with _alloc_on(stream):
        if out is None:
            out = torch.empty(sh.q, dtype=dt, device=dev)
        if idx is None:
            idx = torch.empty(sh.rows, dtype=torch.int32, device=dev)
        if sel is None:
            sel = torch.empty(sh.rows, dtype=torch.float32, device=dev)
        if lse is None and want_lse:
            lse = torch.empty(sh.lse, dtype=torch.float32, device=dev)
        if w is None and want_w:
            w = torch.empty(sh.rows, dtype=torch.float32, device=dev)
        if ws is None:
            ws, nbytes = workspace(p, OP_FORWARD, dev)
        else:
            nbytes = ws.numel()
    _check(lib().gca_forward(
        ctypes.byref(p), _ptr(lmk_q, "lmk_q", dt, sh.lmk_q), _ptr(lmk_k, "lmk_k", dt, sh.lmk_k),
        _ptr(q, "q", dt, sh.q),
        _ptr(k, "k", dt, sh.kv, _host_kv(p)), _ptr(v, "v", dt, sh.kv, _host_kv(p)),
        _ptr(out, "out", dt, sh.q), _ptr(idx, "idx", torch.int32, sh.rows),
        _ptr(sel, "sel", torch.float32, sh.rows), _ptr(lse, "lse", torch.float32, sh.lse),
        _ptr(w, "w", torch.float32, sh.rows), _ptr(ws, "workspace"), ctypes.c_size_t(nbytes),
        _stream(stream)))
    return {"out": out, "idx": idx, "sel": sel, "lse": lse, "w": w}


def forward_noalloc(p: Problem, lmk_q, lmk_k, q, k, v, out, idx, sel, lse=None, w=None, stream=None):
    """gca_forward_noalloc: the whole forward path into caller-provided outputs,
    with the library's own per-device scratch as workspace (nothing allocated)."""
    torch = _torch()
    sh, dt = shapes(p), _elem_dtype(p)
    _check(lib().gca_forward_noalloc(
        ctypes.byref(p), _ptr(lmk_q, "lmk_q", dt, sh.lmk_q), _ptr(lmk_k, "lmk_k", dt, sh.lmk_k),
        _ptr(q, "q", dt, sh.q),
        _ptr(k, "k", dt, sh.kv, _host_kv(p)), _ptr(v, "v", dt, sh.kv, _host_kv(p)),
        _ptr(out, "out", dt, sh.q), _ptr(idx, "idx", torch.int32, sh.rows),
        _ptr(sel, "sel", torch.float32, sh.rows), _ptr(lse, "lse", torch.float32, sh.lse),
        _ptr(w, "w", torch.float32, sh.rows), _stream(stream)))
    return {"out": out, "idx": idx, "sel": sel, "lse": lse, "w": w}


# ---------------------------------------------------------------- profiling ----

def profile_arm(event_array, capacity: int) -> None:
    """Arm the per-kernel event hook with a ctypes array of hipEvent_t (None disarms)."""
    lib().gca_profile_arm(event_array, capacity if event_array is not None else 0)


def profile_record():
    """Kernel names preceding each recorded event since arming."""
    L = lib()
    return [L.gca_profile_name(i).decode() for i in range(L.gca_profile_count())]
