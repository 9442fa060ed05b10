"""gca_forward_noalloc on the host: exported, and its argument checks (NULL
pointers, the scratch size limit) reject a call before anything is launched."""

import ctypes

import pytest

from _helpers import ensure_built


@pytest.fixture(scope="module")
def gca():
    ensure_built()
    from paper_2410_01651_amd import gca as g
    g.lib()
    return g


FAKE = ctypes.c_void_p(1 << 20)   # aligned, never dereferenced: validation fails first


def _call(gca, p, **override):
    args = dict(lmk_q=FAKE, lmk_k=FAKE, q=FAKE, k=FAKE, v=FAKE, out=FAKE, idx=FAKE, sel=FAKE, lse=None, w=None)
    args.update(override)
    L = gca.lib()
    st = L.gca_forward_noalloc(ctypes.byref(p), args["lmk_q"], args["lmk_k"], args["q"], args["k"], args["v"],
                               args["out"], args["idx"], args["sel"], args["lse"], args["w"], None)
    return st, L.gca_last_error().decode()


def test_scratch_size_matches_header(gca):
    import os
    import re
    from _helpers import ROOT
    text = open(os.path.join(ROOT, "include", "gca.h")).read()
    m = re.search(r"#define GCA_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == gca.NOALLOC_SCRATCH_BYTES


@pytest.mark.parametrize("arg", ["lmk_q", "lmk_k", "q", "k", "v", "out", "idx", "sel"])
def test_null_required_pointer(gca, arg):
    st, msg = _call(gca, gca.problem(1, 2, 64, 4), **{arg: None})
    assert st == gca.GCA_ERR_INVALID and arg in msg


def test_scratch_limit(gca):
    big = gca.problem(1, 1, 4096, 8, D=64, flags=gca.FLAG_MATERIALIZE)   # 64 MiB score matrix
    assert gca.workspace_size(big, gca.OP_FORWARD) > gca.NOALLOC_SCRATCH_BYTES
    st, msg = _call(gca, big)
    assert st == gca.GCA_ERR_UNSUPPORTED and "scratch" in msg
    bad = gca.problem(1, 1, 16, 2, d=32)
    st, _ = _call(gca, bad)
    assert st == gca.GCA_ERR_UNSUPPORTED
