"""CPU oracle for Grouped Cross Attention (GCA) -- TEST INFRASTRUCTURE ONLY.

This module is the plain, slow, fp64 definition of what the GPU path computes.
It exists to check that path.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import or call it; the product path never
does, and it shares no code, tables or constants with the HIP kernels.

It follows the paper's definitions, not its tiled kernels:

* relevance scores and top-k retrieval: Eq. 1 (Methodology, Model
  Architecture, "Forward Pass");
* fusion weights and the per-chunk cross attention fused by them: Eq. 2 and
  Eq. 3 ("Grouped Cross-Attention");
* the backward pass: the chain rule through Eq. 2-3, with the quantities that
  Algorithm 2 (Appendix B, FlashGCA backward) names -- D = rowsum(dO o O'),
  dS = w P o (dP - D) and the gradient into the weights -- computed densely.

Readings where the paper is silent or ambiguous (all configurable):

* chunks are numbered from 0; chunk t retrieves among chunks [0, t) and its
  retrieved set feeds the tokens of chunk t+1 (causal mode).  In decode mode
  one new chunk's landmark scores all past chunks and its set feeds that same
  new chunk's tokens;
* top-k keeps the min(k, t) largest scores, ties to the lower chunk index, and
  reports the set in ascending chunk order, padded with index -1 / score -inf;
* the weights are a softmax over the valid slots only; an empty set gives an
  all-zero output row (chunks 0 and 1 in causal mode);
* the per-chunk softmax is the plain softmax of Algorithm 1 by default;
  ``off_by_one=True`` gives Eq. 3's softmax-off-by-one (denominator 1 + sum);
* Gumbel top-k (Training & Inference, an option): noise from a counter-based
  generator (gumbel_noise) is added to the scores for the selection only; sel,
  the weights and everything after use the raw scores;
* ``lse`` is the log of each (row, slot) softmax denominator, -inf for pads;
* one retrieval head shared by all heads (Hr = 1, as Eq. 1 yields one score per
  chunk pair) or one per head (Hr = H);
* query rows per chunk ``Sq``: S by default; S + 1 when every chunk carries its
  landmark (LMK) token as a last query row (Methodology, Model Architecture: the
  LMK token is inserted at the end of each chunk, and Grouped Cross-Attention
  takes the S + 1 hidden states of chunk t+1 as queries against the S-row
  memories C_k of the retrieved chunks).

Array layouts are row-major: lmk_q [B,Hr,nQ,D], lmk_k [B,Hr,nC,D],
q/dout [B,H,nQ*Sq,d], k/v [B,H,nC*S,d]; all inputs are taken as fp64.
"""

import numpy as np

from .philox import philox4x32_10

NEG_INF = -np.inf


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def retrieval_row(c: int, mode: str) -> int:
    """Which landmark row's retrieved set feeds query chunk c (Eq. 2: C_t feeds chunk t+1)."""
    return c - 1 if mode == "causal" else 0


def head_to_rhead(h: int, H: int, Hr: int) -> int:
    if Hr == 1:
        return 0
    if Hr == H:
        return h
    raise ValueError("Hr must be 1 or H")


# --------------------------------------------------------------------------
# Eq. 1: causal relevance scores and top-k
# --------------------------------------------------------------------------

def scores(lmk_q, lmk_k, score_scale, mode="causal", rows=None):
    """Relevance scores r[b, hr, t, j] = score_scale * <lmk_q[t], lmk_k[j]> (Eq. 1).

    Causal mode keeps only strictly earlier chunks j < t (Eq. 1 ranges over
    1..t-1); every other entry is -inf.  Decode mode scores every past chunk.
    ``rows`` restricts the computation to the listed query rows.
    """
    q = _f64(lmk_q)
    k = _f64(lmk_k)
    B, Hr, nQ, D = q.shape
    nC = k.shape[2]
    rows = np.arange(nQ) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.full((B, Hr, len(rows), nC), NEG_INF)
    for b in range(B):
        for hr in range(Hr):
            r = score_scale * (q[b, hr, rows] @ k[b, hr].T)
            if mode == "causal":
                j = np.arange(nC)[None, :]
                r = np.where(j < rows[:, None], r, NEG_INF)
            out[b, hr] = r
    return out


def gumbel_noise(seed, bhr, t, j):
    """Gumbel noise g = -ln(-ln u) of candidate chunk j for retrieval row t of
    (batch, retrieval head) bhr = b * Hr + hr (Gumbel top-k sampling, Training &
    Inference).  u is uniform in (0, 1) from the Philox4x32-10 generator: key =
    the 64-bit seed (low word, high word), counter = (j div 4, t, bhr, 0), output
    word j mod 4, whose top 24 bits x give u = (x + 1/2) / 2^24.  Broadcasts over
    array arguments."""
    j = np.asarray(j, dtype=np.int64)
    words = philox4x32_10(j >> 2, t, bhr, 0, seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    shape = np.broadcast_shapes(np.shape(words[0]), j.shape)
    sel = np.broadcast_to(j & 3, shape)
    x = np.select([sel == 0, sel == 1, sel == 2, sel == 3], [np.broadcast_to(w, shape) for w in words])
    u = ((x >> np.uint64(8)).astype(np.float64) + 0.5) / 2.0 ** 24
    return -np.log(-np.log(u))


def topk_row(r_row, k, noise_row=None):
    """Top-k of one score row (Eq. 1): indices ascending, ties to the lower index.

    Only finite entries are candidates.  With ``noise_row`` (Gumbel top-k) the
    candidates are ranked by score + noise, and sel still reports the raw score:
    the noise only decides membership.  Returns (idx[k] int32 padded with -1,
    sel[k] fp64 padded with -inf).
    """
    r_row = _f64(r_row)
    cand = np.nonzero(np.isfinite(r_row))[0]
    key = r_row[cand] if noise_row is None else r_row[cand] + _f64(noise_row)[cand]
    order = cand[np.lexsort((cand, -key))]               # (noisy) score desc, then j asc
    chosen = np.sort(order[:k])
    idx = np.full(k, -1, dtype=np.int32)
    sel = np.full(k, NEG_INF)
    idx[:len(chosen)] = chosen
    sel[:len(chosen)] = r_row[chosen]
    return idx, sel


def topk(r, k, gumbel_seed=None, rows=None, bhr0=0):
    """Row-wise top-k over a [B, Hr, nRows, nC] score array.  ``rows`` are the
    landmark rows the array holds (default 0..nRows-1); with ``gumbel_seed`` the
    selection is Gumbel top-k (noise from gumbel_noise), the array's first
    (batch, retrieval head) slice being slice ``bhr0`` of the problem."""
    B, Hr, n, nC = r.shape
    rows = np.arange(n) if rows is None else np.asarray(rows)
    idx = np.full((B, Hr, n, k), -1, dtype=np.int32)
    sel = np.full((B, Hr, n, k), NEG_INF)
    cols = np.arange(nC)
    for b in range(B):
        for hr in range(Hr):
            for i in range(n):
                noise = None if gumbel_seed is None else gumbel_noise(gumbel_seed, bhr0 + b * Hr + hr,
                                                                      int(rows[i]), cols)
                idx[b, hr, i], sel[b, hr, i] = topk_row(r[b, hr, i], k, noise)
    return idx, sel


# --------------------------------------------------------------------------
# Eq. 2: fusion weights
# --------------------------------------------------------------------------

def fusion_weights(sel):
    """w = softmax of the retrieved chunks' raw scores over valid slots (Eq. 2).

    Pad slots (score -inf) get weight 0; a row with no valid slot is all zero.
    """
    sel = _f64(sel)
    valid = np.isfinite(sel)
    m = np.where(valid, sel, NEG_INF).max(axis=-1, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    e = np.where(valid, np.exp(np.where(valid, sel, 0.0) - m), 0.0)
    s = e.sum(axis=-1, keepdims=True)
    return np.where(s > 0, e / np.where(s > 0, s, 1.0), 0.0)


# --------------------------------------------------------------------------
# Eq. 2-3: grouped cross attention
# --------------------------------------------------------------------------

def chunk_attention(qc, kc, vc, attn_scale, off_by_one=False):
    """Cross attention of one query chunk onto one retrieved chunk (Eq. 3, one head).

    Returns (P [Sq,Sk], O' = P V [Sq,d], lse [Sq]) with P the row softmax of
    attn_scale * qc kc^T; with ``off_by_one`` the denominator gains exp(0).
    """
    a = attn_scale * (qc @ kc.T)
    if off_by_one:
        m = np.maximum(a.max(axis=1, keepdims=True), 0.0)
        e = np.exp(a - m)
        l = np.exp(-m) + e.sum(axis=1, keepdims=True)
    else:
        m = a.max(axis=1, keepdims=True)
        e = np.exp(a - m)
        l = e.sum(axis=1, keepdims=True)
    p = e / l
    return p, p @ vc, (m + np.log(l))[:, 0]


def xattn_fwd(q, k, v, idx, w, S, attn_scale, mode="causal", off_by_one=False,
              chunks=None, heads=None, Sq=None):
    """Grouped cross attention forward (Eq. 2-3).

    For each head and query chunk c, every valid slot s of the retrieved set
    C_t (t = retrieval_row(c)) gives O'_s = CA(Q_c, chunk j_s) separately, and
    O_c = sum_s w[t, s] O'_s.  Returns (O [B,H,Lq,d], lse [B,H,Lq,k]); rows of
    chunks whose set is empty are 0 and their lse is -inf.  ``chunks`` /
    ``heads`` restrict the work to the listed query chunks / heads (other rows
    are left 0 / -inf).  Query chunk c is rows [c*Sq, (c+1)*Sq) of q (Sq = S
    unless given); key chunk j is rows [j*S, (j+1)*S) of k and v.
    """
    q, k, v, w = _f64(q), _f64(k), _f64(v), _f64(w)
    B, H, Lq, d = q.shape
    Hr, kk = idx.shape[1], idx.shape[-1]
    Sq = S if Sq is None else Sq
    nQ = Lq // Sq
    out = np.zeros((B, H, Lq, d))
    lse = np.full((B, H, Lq, kk), NEG_INF)
    chunks = range(nQ) if chunks is None else chunks
    heads = range(H) if heads is None else heads
    for b in range(B):
        for h in heads:
            hr = head_to_rhead(h, H, Hr)
            for c in chunks:
                t = retrieval_row(c, mode)
                if t < 0:
                    continue
                rows = slice(c * Sq, (c + 1) * Sq)
                for s in range(kk):
                    j = int(idx[b, hr, t, s])
                    if j < 0:
                        continue
                    cols = slice(j * S, (j + 1) * S)
                    _, o_s, lse_s = chunk_attention(q[b, h, rows], k[b, h, cols], v[b, h, cols],
                                                    attn_scale, off_by_one)
                    out[b, h, rows] += w[b, hr, t, s] * o_s
                    lse[b, h, rows, s] = lse_s
    return out, lse


def xattn_bwd(q, k, v, idx, w, dout, S, attn_scale, mode="causal", off_by_one=False,
              chunks=None, heads=None, Sq=None):
    """Backward of grouped cross attention (chain rule through Eq. 2-3).

    With L = sum(dout o O), for every (head, query chunk c, valid slot s):
    O'_s = P_s V_j, D_s = rowsum(dout_c o O'_s), dP_s = dout_c V_j^T,
    dS = w P_s o (dP_s - D_s) (the softmax Jacobian, which has the same form for
    softmax-off-by-one), dV_j += w P_s^T dout_c, dQ_c += attn_scale dS K_j,
    dK_j += attn_scale dS^T Q_c, and dL/dw[t, s] = sum over heads of the retrieval
    head and rows of D_s.  Returns (dq, dk, dv, dw [B,Hr,nQr,k]).  Query chunks
    have Sq rows (S unless given), key chunks S.
    """
    q, k, v, w, dout = _f64(q), _f64(k), _f64(v), _f64(w), _f64(dout)
    B, H, Lq, d = q.shape
    Hr, nQr, kk = idx.shape[1], idx.shape[2], idx.shape[-1]
    Sq = S if Sq is None else Sq
    nQ = Lq // Sq
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    dw = np.zeros((B, Hr, nQr, kk))
    chunks = range(nQ) if chunks is None else chunks
    heads = range(H) if heads is None else heads
    for b in range(B):
        for h in heads:
            hr = head_to_rhead(h, H, Hr)
            for c in chunks:
                t = retrieval_row(c, mode)
                if t < 0:
                    continue
                rows = slice(c * Sq, (c + 1) * Sq)
                qc, doc = q[b, h, rows], dout[b, h, rows]
                for s in range(kk):
                    j = int(idx[b, hr, t, s])
                    if j < 0:
                        continue
                    cols = slice(j * S, (j + 1) * S)
                    kc, vc = k[b, h, cols], v[b, h, cols]
                    p, o_s, _ = chunk_attention(qc, kc, vc, attn_scale, off_by_one)
                    ws = w[b, hr, t, s]
                    D = (doc * o_s).sum(axis=1, keepdims=True)
                    dP = doc @ vc.T
                    dS = ws * p * (dP - D)
                    dv[b, h, cols] += ws * (p.T @ doc)
                    dq[b, h, rows] += attn_scale * (dS @ kc)
                    dk[b, h, cols] += attn_scale * (dS.T @ qc)
                    dw[b, hr, t, s] += D.sum()
    return dq, dk, dv, dw


def dsel_from_dw(w, dw):
    """Gradient into the retrieved scores through the weight softmax (Eq. 2).

    dsel[s] = w[s] (dw[s] - sum_s' w[s'] dw[s']); pad slots (w = 0) get 0.
    """
    w, dw = _f64(w), _f64(dw)
    return w * (dw - (w * dw).sum(axis=-1, keepdims=True))


def landmark_grads(dsel, idx, lmk_q, lmk_k, score_scale):
    """Gradients into the landmark vectors through Eq. 1.

    r[t, j_s] = score_scale <lmk_q[t], lmk_k[j_s]>, so
    dlmk_q[t] = score_scale sum_s dsel[t,s] lmk_k[j_s] and
    dlmk_k[j] = score_scale sum over (t, s) with j_s = j of dsel[t,s] lmk_q[t].
    The indices are constants (the top-k choice carries no gradient).
    """
    dsel = _f64(dsel)
    lq, lk = _f64(lmk_q), _f64(lmk_k)
    B, Hr, nQ, kk = idx.shape
    dq = np.zeros_like(lq)
    dk = np.zeros_like(lk)
    for b in range(B):
        for hr in range(Hr):
            for t in range(nQ):
                for s in range(kk):
                    j = int(idx[b, hr, t, s])
                    if j < 0:
                        continue
                    dq[b, hr, t] += score_scale * dsel[b, hr, t, s] * lk[b, hr, j]
                    dk[b, hr, j] += score_scale * dsel[b, hr, t, s] * lq[b, hr, t]
    return dq, dk


# --------------------------------------------------------------------------
# Whole path
# --------------------------------------------------------------------------

def forward(p, lmk_q, lmk_k, q, k, v):
    """Scores -> top-k -> weights -> grouped cross attention (Eq. 1-3).

    ``p`` is a mapping with S, topk, score_scale, attn_scale, mode, off_by_one
    and optionally gumbel_seed (Gumbel top-k selection) and Sq (query rows per
    chunk, S + 1 with the LMK row).  Returns a dict with scores, idx, sel, w, out
    and lse.
    """
    r = scores(lmk_q, lmk_k, p["score_scale"], p["mode"])
    idx, sel = topk(r, p["topk"], p.get("gumbel_seed"))
    w = fusion_weights(sel)
    out, lse = xattn_fwd(q, k, v, idx, w, p["S"], p["attn_scale"], p["mode"],
                         p.get("off_by_one", False), Sq=p.get("Sq"))
    return {"scores": r, "idx": idx, "sel": sel, "w": w, "out": out, "lse": lse}


def backward(p, fwd, lmk_q, lmk_k, q, k, v, dout):
    """Gradients of sum(dout o out) into q, k, v, the scores and the landmarks."""
    dq, dk, dv, dw = xattn_bwd(q, k, v, fwd["idx"], fwd["w"], dout, p["S"],
                               p["attn_scale"], p["mode"], p.get("off_by_one", False),
                               Sq=p.get("Sq"))
    dsel = dsel_from_dw(fwd["w"], dw)
    dlq, dlk = landmark_grads(dsel, fwd["idx"], lmk_q, lmk_k, p["score_scale"])
    return {"dq": dq, "dk": dk, "dv": dv, "dw": dw, "dsel": dsel,
            "dlmk_q": dlq, "dlmk_k": dlk}
