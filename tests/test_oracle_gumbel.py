"""Pins of the oracle's Gumbel top-k retrieval (Training & Inference, "Gumbel
Top-k sampling"): the counter-based generator against its published
known-answer values, the noise against the Gumbel distribution's closed-form
moments, and the selection against exact sampling without replacement."""

import json
import math
import os

import numpy as np

from oracle import gca as og
from oracle.philox import philox4x32_10

KAT = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.json")


def test_philox_known_answers():
    for v in json.load(open(KAT))["vectors"]:
        c = [int(x, 16) for x in v["counter"]]
        k = [int(x, 16) for x in v["key"]]
        out = philox4x32_10(*c, *k)
        assert [int(x) for x in out] == [int(x, 16) for x in v["out"]]


def test_gumbel_noise_moments():
    """Gumbel(0, 1): mean = Euler's constant, variance = pi^2 / 6, P(g <= 0) = 1/e."""
    g = og.gumbel_noise(12345, 3, np.arange(400)[:, None], np.arange(500)[None, :]).ravel()
    n = g.size
    assert abs(g.mean() - 0.5772156649) < 5 * math.sqrt(math.pi ** 2 / 6 / n)
    assert abs(g.var() - math.pi ** 2 / 6) < 0.03
    assert abs((g <= 0).mean() - math.exp(-1)) < 5 * math.sqrt(0.25 / n)


def test_gumbel_noise_independent_streams():
    """Different seeds, rows, (batch, head) slices and chunks draw different values;
    the same arguments draw the same value."""
    a = og.gumbel_noise(7, 0, 5, np.arange(64))
    assert np.array_equal(a, og.gumbel_noise(7, 0, 5, np.arange(64)))
    assert len(np.unique(a)) == 64
    for other in (og.gumbel_noise(8, 0, 5, np.arange(64)), og.gumbel_noise(7, 1, 5, np.arange(64)),
                  og.gumbel_noise(7, 0, 6, np.arange(64))):
        assert not np.any(other == a)
    assert abs(np.corrcoef(a, og.gumbel_noise(7, 0, 6, np.arange(64)))[0, 1]) < 0.5


def _inclusion_exact(r, k):
    """P(candidate in the sample) for k draws without replacement, p ~ exp(r):
    brute force over ordered draws."""
    p = np.exp(r - r.max())
    p /= p.sum()
    n = len(r)
    inc = np.zeros(n)

    def rec(chosen, prob):
        if len(chosen) == k:
            for c in chosen:
                inc[c] += prob
            return
        rest = 1.0 - sum(p[c] for c in chosen)
        for c in range(n):
            if c not in chosen:
                rec(chosen + [c], prob * p[c] / rest)
    rec([], 1.0)
    return inc


def test_gumbel_topk_samples_without_replacement():
    """Top-k of score + Gumbel noise is k draws without replacement with
    probabilities proportional to exp(score); the sel values stay the raw scores."""
    r = np.array([1.0, 0.2, -0.5, 0.9, 2.0])
    k, rows = 2, 20000
    rr = np.broadcast_to(r, (1, 1, rows, len(r))).copy()
    idx, sel = og.topk(rr, k, gumbel_seed=99)
    freq = np.array([(idx[0, 0] == c).any(axis=1).mean() for c in range(len(r))])
    exact = _inclusion_exact(r, k)
    assert np.all(np.abs(freq - exact) < 4.5 * np.sqrt(exact * (1 - exact) / rows))
    assert np.array_equal(sel[0, 0], r[idx[0, 0]])
    # without noise the selection is the deterministic top-k on every row
    idx0, _ = og.topk(rr[:, :, :3], k)
    assert np.all(idx0[0, 0] == np.array([0, 4]))


def test_gumbel_forward_keeps_raw_scores():
    """In the whole forward the noise moves membership only: sel = r[idx] and
    w = softmax(sel), on a causal problem where the noisy sets differ."""
    rng = np.random.default_rng(0)
    B, Hr, nC, D, S, d, k = 1, 1, 12, 8, 4, 4, 3
    lq, lk = rng.standard_normal((B, Hr, nC, D)), rng.standard_normal((B, Hr, nC, D))
    q, kk, v = (rng.standard_normal((B, 1, nC * S, d)) for _ in range(3))
    p = dict(S=S, topk=k, score_scale=1.0, attn_scale=0.5, mode="causal")
    plain = og.forward(p, lq, lk, q, kk, v)
    noisy = og.forward(dict(p, gumbel_seed=3), lq, lk, q, kk, v)
    assert not np.array_equal(plain["idx"], noisy["idx"])
    r = plain["scores"][0, 0]
    for t in range(nC):
        valid = noisy["idx"][0, 0, t] >= 0
        assert np.array_equal(noisy["sel"][0, 0, t][valid], r[t, noisy["idx"][0, 0, t][valid]])
    assert np.allclose(noisy["w"], og.fusion_weights(noisy["sel"]))
