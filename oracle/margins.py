"""Top-k margin enforcement for synthetic inputs -- TEST INFRASTRUCTURE ONLY.

The GPU accumulates landmark scores in fp32 while the oracle uses fp64, so a
row whose k-th and (k+1)-th best scores (Eq. 1) nearly tie could be ranked
differently by the two.  Inputs used for parity therefore keep a gap of at
least ``margin`` between the k-th and (k+1)-th score of every row that has
more than k candidates, measured in fp64 on the exact stored values (for Gumbel
top-k workloads, between the noisy scores that the selection ranks).

Two ways to restore the gap (the workload says which):

* whole-input reseeding: redraw every tensor with the next attempt number
  until every row passes (cheap for tiny inputs);
* row redraw: redraw only a failing row's landmark query, from its own seed
  stream, until that row passes.  Keys are fixed first and row t's scores
  depend only on lmk_q[t], so rows never disturb each other.  A planted
  target row is left as it is (its planted keys dominate by construction),
  except in decode mode where the single query and its planted key move
  together.
"""

import numpy as np

from gen import inputs as gi
from . import gca


def row_gaps(lmk_q64, lmk_k64, score_scale, k, mode, rows=None, gumbel_seed=None, bhr0=0):
    """fp64 gap between the k-th and (k+1)-th best score of each row (inf if <= k
    candidates).  With ``gumbel_seed`` the ranked values are score + Gumbel noise
    (the selection's key); ``bhr0`` is the (batch, retrieval head) index of the
    first slice, for the noise counters."""
    r = gca.scores(lmk_q64, lmk_k64, score_scale, mode, rows=rows)
    B, Hr, n, nC = r.shape
    rows_ = np.arange(n) if rows is None else np.asarray(rows)
    gaps = np.full((B, Hr, n), np.inf)
    for b in range(B):
        for hr in range(Hr):
            rb = r[b, hr]
            if gumbel_seed is not None:
                rb = rb + gca.gumbel_noise(gumbel_seed, bhr0 + b * Hr + hr, rows_[:, None], np.arange(nC)[None, :])
            if nC > k:
                # the k-th and (k+1)-th largest of each row (order statistics,
                # -inf last): a partial sort gives exactly what a full sort would
                part = -np.partition(-rb, [k - 1, k], axis=1)
                kth, nxt = part[:, k - 1], part[:, k]
                ok = np.isfinite(nxt)
                gaps[b, hr] = np.where(ok, kth - np.where(ok, nxt, 0.0), np.inf)
    return gaps


def _seed(w):
    return w.gumbel_seed if w.gumbel_seed >= 0 else None


def _failing_rows(w, lmk_q, lmk_k, block=2048):
    q64 = gi.decode(w, lmk_q)
    k64 = gi.decode(w, lmk_k)
    nQ = lmk_q.shape[2]
    bad = []
    for r0 in range(0, nQ, block):
        rows = np.arange(r0, min(nQ, r0 + block))
        g = row_gaps(q64, k64, w.score_scale, w.topk, w.mode, rows=rows, gumbel_seed=_seed(w))
        for b, hr, i in zip(*np.nonzero(g < w.margin)):
            bad.append((int(b), int(hr), int(rows[i])))
    return bad


def enforce(w, lmk_q, lmk_k, max_attempts=1000):
    """Redraw failing landmark-query rows in place until every margin holds."""
    target = gi.plant_target_row(w) if (w.planted and w.mode == "causal") else None
    pending = _failing_rows(w, lmk_q, lmk_k)
    keys64 = {}                                   # decoded key slices, one per (b, hr)
    plant = gi.plant_positions(w)
    for (b, hr, t) in pending:
        if t == target:
            raise RuntimeError("planted target row lost its margin")
        if (b, hr) not in keys64:
            keys64[(b, hr)] = gi.decode(w, lmk_k[b:b + 1, hr:hr + 1])
        k64 = keys64[(b, hr)]
        for attempt in range(1, max_attempts + 1):
            gi.redraw_lmk_q_row(w, lmk_q, lmk_k, b, hr, t, attempt)
            if w.planted and t == gi.plant_target_row(w):
                k64[0, 0, plant] = gi.decode(w, lmk_k[b, hr, plant])   # planted keys follow the row
            # row t's gap from its own query (a broadcast view stands in for the
            # other rows, which the gap of row t does not read)
            q_row = gi.decode(w, lmk_q[b, hr, t])
            q64 = np.broadcast_to(q_row, (1, 1, t + 1, q_row.shape[-1]))
            g = row_gaps(q64, k64, w.score_scale, w.topk, w.mode, rows=[t], gumbel_seed=_seed(w),
                         bhr0=b * w.Hr + hr)
            if g[0, 0, 0] >= w.margin:
                break
        else:
            raise RuntimeError(f"no margin after {max_attempts} redraws of row {t}")
    return len(pending)


def checked_inputs(w, tokens=True, max_attempts=200):
    """Workload inputs whose top-k is unambiguous (see module docstring).

    Returns (inputs dict, attempts or redrawn-row count).
    """
    if w.whole_reseed:
        for attempt in range(max_attempts):
            lq, lk = gi.draw_landmarks(w, attempt)
            if not _failing_rows(w, lq, lk):
                inp = gi.draw_inputs(w, attempt, tokens=tokens)
                return inp, attempt
        raise RuntimeError("no margin-satisfying draw found")
    inp = gi.draw_inputs(w, 0, tokens=tokens)
    n = enforce(w, inp["lmk_q"], inp["lmk_k"])
    return inp, n
