"""Pins for the oracle's forward and backward against an independent statement of
Eq. 1-3 in PyTorch (fp64, CPU), differentiated by autograd: the selection is
taken with torch.topk, the fusion weights with torch.softmax over the selected
raw scores (Eq. 2), each retrieved chunk's attention written directly (Eq. 3, plain
or off-by-one softmax), and every gradient (q, k, v, the selected scores, both
landmark tensors) comes from the autograd graph rather than from the chain rule
the oracle writes out.  Seeded random small configurations cover both modes,
shared or per-head retrieval, S or S+1 query rows and k at, above and below the
history."""

import math

import numpy as np
import pytest
import torch

from oracle import gca, margins


def _config(seed):
    rng = np.random.default_rng(seed)
    mode = "decode" if rng.random() < 0.3 else "causal"
    H = int(rng.integers(1, 4))
    c = dict(B=int(rng.integers(1, 3)), H=H, Hr=H if rng.random() < 0.4 else 1, S=int(rng.integers(2, 5)),
             d=int(rng.choice([4, 8])), nC=int(rng.integers(2, 8)), k=int(rng.integers(1, 5)),
             D=int(rng.choice([8, 16])), obo=bool(rng.random() < 0.4), mode=mode)
    c["Sq"] = c["S"] + 1 if (mode == "causal" and rng.random() < 0.4) else c["S"]
    return c, rng


def _inputs(c, rng):
    B, H, Hr, S, Sq, d, nC, k, D = (c[x] for x in ("B", "H", "Hr", "S", "Sq", "d", "nC", "k", "D"))
    nQ = 1 if c["mode"] == "decode" else nC
    for _ in range(1000):
        lq = rng.standard_normal((B, Hr, nQ, D))
        lk = rng.standard_normal((B, Hr, nC, D))
        if np.all(margins.row_gaps(lq, lk, 1 / math.sqrt(D), k, c["mode"]) >= 0.05):
            break
    else:
        raise RuntimeError("no margin")
    q = rng.standard_normal((B, H, nQ * Sq, d))
    kk = rng.standard_normal((B, H, nC * S, d))
    v = rng.standard_normal((B, H, nC * S, d))
    dout = rng.standard_normal((B, H, nQ * Sq, d))
    return lq, lk, q, kk, v, dout


def _torch_gca(c, lq, lk, q, k, v, dout):
    """Eq. 1-3 in torch, differentiated by autograd."""
    T = lambda x: torch.tensor(x, dtype=torch.float64, requires_grad=True)
    lq_t, lk_t, q_t, k_t, v_t = T(lq), T(lk), T(q), T(k), T(v)
    B, H, Hr, S, Sq, nC, K = (c[x] for x in ("B", "H", "Hr", "S", "Sq", "nC", "k"))
    nQ = lq.shape[2]
    r = (lq_t @ lk_t.transpose(-1, -2)) / math.sqrt(c["D"])          # Eq. 1 scores
    chosen, sels = {}, {}
    for b in range(B):
        for hr in range(Hr):
            for t in range(nQ):
                ncand = t if c["mode"] == "causal" else nC           # causal: chunks j < t
                if ncand == 0:
                    continue
                top = torch.topk(r[b, hr, t, :ncand].detach(), min(K, ncand)).indices
                js = sorted(int(j) for j in top)
                sel = r[b, hr, t, js]
                sel.retain_grad()
                chosen[b, hr, t], sels[b, hr, t] = js, sel
    rows = []
    lse = {}
    for b in range(B):
        for h in range(H):
            hr = 0 if Hr == 1 else h
            for cq in range(nQ):
                t = cq - 1 if c["mode"] == "causal" else 0
                out_c = torch.zeros(Sq, q.shape[-1], dtype=torch.float64)
                if t >= 0 and (b, hr, t) in chosen:
                    w = torch.softmax(sels[b, hr, t], 0)                # Eq. 2 fusion weights
                    Qc = q_t[b, h, cq * Sq:(cq + 1) * Sq]
                    for s, j in enumerate(chosen[b, hr, t]):
                        logits = (Qc @ k_t[b, h, j * S:(j + 1) * S].T) / math.sqrt(c["d"])
                        if c["obo"]:                                     # Eq. 3, off-by-one
                            den = 1.0 + torch.exp(logits).sum(-1, keepdim=True)
                            P = torch.exp(logits) / den
                            lse[b, h, cq, s] = torch.log(den[:, 0])
                        else:
                            P = torch.softmax(logits, -1)
                            lse[b, h, cq, s] = torch.logsumexp(logits, -1)
                        out_c = out_c + w[s] * (P @ v_t[b, h, j * S:(j + 1) * S])
                rows.append(out_c)
    out = torch.stack(rows).reshape(B, H, nQ * Sq, -1)
    if out.requires_grad:                 # (no chunk retrieves anything: every gradient is zero)
        (out * torch.tensor(dout)).sum().backward()
    grad = lambda x: np.zeros(x.shape) if x.grad is None else x.grad.numpy()
    return dict(out=out.detach().numpy(), lse=lse, sels=sels, chosen=chosen, dq=grad(q_t), dk=grad(k_t),
                dv=grad(v_t), dlmk_q=grad(lq_t), dlmk_k=grad(lk_t))


@pytest.mark.parametrize("seed", range(24))
def test_oracle_matches_autograd(seed):
    c, rng = _config(seed)
    lq, lk, q, k, v, dout = _inputs(c, rng)
    p = dict(S=c["S"], topk=c["k"], score_scale=1 / math.sqrt(c["D"]), attn_scale=1 / math.sqrt(c["d"]),
             mode=c["mode"], off_by_one=c["obo"], Sq=c["Sq"])
    f = gca.forward(p, lq, lk, q, k, v)
    g = gca.backward(p, f, lq, lk, q, k, v, dout)
    ref = _torch_gca(c, lq, lk, q, k, v, dout)
    # the same selection, slot by slot
    for (b, hr, t), js in ref["chosen"].items():
        assert list(f["idx"][b, hr, t][:len(js)]) == js and np.all(f["idx"][b, hr, t][len(js):] == -1)
        sg = ref["sels"][b, hr, t].grad
        sg = np.zeros(len(js)) if sg is None else sg.numpy()
        np.testing.assert_allclose(g["dsel"][b, hr, t][:len(js)], sg, rtol=0, atol=1e-12)
    np.testing.assert_allclose(f["out"], ref["out"], rtol=0, atol=1e-12)
    for (b, h, cq, s), val in ref["lse"].items():
        np.testing.assert_allclose(f["lse"][b, h, cq * c["Sq"]:(cq + 1) * c["Sq"], s], val.detach().numpy(),
                                   rtol=0, atol=1e-12)
    for key in ("dq", "dk", "dv", "dlmk_q", "dlmk_k"):
        np.testing.assert_allclose(g[key], ref[key], rtol=0, atol=1e-11, err_msg=key)
