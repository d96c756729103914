"""Pins of the oracle's GLA-prior read (Appendix "Gated Linear Attention (GLA)
Prior": RoPE, ReLU + eps features, decay envelope; eqs. gla-score-appendix
and gla-assoc).

None of these retypes ``fem_gla``: it is checked against a 50-digit
term-by-term evaluation (``oracle.brute``), against the float64 step-by-step
recurrence of the appendix's streaming form, against a closed form (equal
features and a scalar decay make the prior geometric), and RoPE against its
defining properties.  Planted mistakes must each fail a pin.
"""

import math

import numpy as np
import pytest

import oracle
from oracle import brute
from oracle import fem_oracle as fo


def head(fn, q, k, v, g, beta, **kw):
    return fn(q[None, None], k[None, None], v[None, None], g[None, None],
              np.asarray(beta)[None], **kw)[0, 0]


def rnd(seed, T, d, D, gscale=0.5):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((T, d)), rng.standard_normal((T, d)),
            2.0 * rng.standard_normal((T, D)), -gscale * rng.uniform(0, 1, (T, d)), rng)


# ---------------------------------------------------------------------------
# RoPE
# ---------------------------------------------------------------------------
def test_rope_properties():
    rng = np.random.default_rng(60)
    x, y = rng.standard_normal((5, 8)), rng.standard_normal((5, 8))
    pos = np.array([0, 1, 7, 100, 4095])
    np.testing.assert_allclose(fo.rope(x, np.zeros(5)), x, rtol=0, atol=0)
    np.testing.assert_allclose(np.linalg.norm(fo.rope(x, pos), axis=1), np.linalg.norm(x, axis=1),
                               rtol=1e-13)
    # relative position: <R_t x, R_i y> depends on t - i only
    a = np.sum(fo.rope(x, pos) * fo.rope(y, pos - 3), axis=1)
    b = np.sum(fo.rope(x, pos + 50) * fo.rope(y, pos + 47), axis=1)
    np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-10)
    # d = 4 by explicit rotation matrices: angles t and t / 100 on pairs (0,1), (2,3)
    t = 3.0
    z = np.array([[1.0, 2.0, 3.0, 4.0]])
    rot = lambda th: np.array([[math.cos(th), -math.sin(th)], [math.sin(th), math.cos(th)]])
    want = np.concatenate([rot(t) @ z[0, :2], rot(t / 100.0) @ z[0, 2:]])
    np.testing.assert_allclose(fo.rope(z, np.array([t]))[0], want, rtol=0, atol=1e-14)


# ---------------------------------------------------------------------------
# The read
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed,T,d,D", [(61, 9, 4, 2), (62, 12, 6, 3)])
def test_gla_brute_force(seed, T, d, D):
    q, k, v, g, rng = rnd(seed, T, d, D, gscale=2.5)  # decays down to e^-2.5 per step
    beta = np.exp(rng.uniform(np.log(0.1), np.log(8.0), D))
    want = np.array(brute.brute_fem_gla(q.tolist(), k.tolist(), v.tolist(), g.tolist(),
                                        beta.tolist(), fo.GLA_EPS, fo.GLA_ROPE_BASE),
                    dtype=np.float64)
    np.testing.assert_allclose(head(oracle.fem_gla, q, k, v, g, beta), want, rtol=0, atol=1e-11)


def test_gla_quadratic_matches_recurrence():
    q, k, v, g, rng = rnd(63, 90, 8, 5, gscale=1.0)
    beta = np.exp(rng.uniform(np.log(0.1), np.log(8.0), 5))
    a = head(oracle.fem_gla, q, k, v, g, beta, block=32)
    b = head(oracle.fem_gla_recurrent, q, k, v, g, beta)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-10)


def test_gla_geometric_prior_closed_form():
    """q = k = 0 gives equal features eps * 1; a scalar decay gamma in every
    channel then makes p_t(i) = w^(t-i) (1 - w) / (1 - w^(t+1)), w = e^gamma."""
    T, d, gamma = 40, 6, -0.3
    z = np.zeros((T, d))
    g = np.full((T, d), gamma)
    p = fo.gla_prior_rows(z, z, g, np.arange(T))
    w = math.exp(gamma)
    for t in (0, 1, 10, 39):
        i = np.arange(t + 1)
        want = w ** (t - i) * (1 - w) / (1 - w ** (t + 1))
        np.testing.assert_allclose(p[t, : t + 1], want, rtol=1e-12)
        assert (p[t, t + 1:] == 0).all()


def test_gla_no_decay_and_strong_decay():
    q, k, v, _, rng = rnd(64, 30, 4, 3)
    beta = np.array([0.5, 2.0, 6.0])
    zero = np.zeros((30, 4))
    # a decay far below any clip leaves the prior on the diagonal key alone:
    # every earlier key carries a factor e^{-200 (t - i)}, far below what the
    # features (>= d eps^2) and e^{beta (v_i - v_t)} (beta |v| < 50 here) can
    # make up, so F_t = v_t
    np.testing.assert_allclose(head(oracle.fem_gla, q, k, v, zero - 200.0, beta), v,
                               rtol=0, atol=1e-12)
    # without decay every causal entry is positive and rows sum to one
    p = fo.gla_prior_rows(q, k, zero, np.arange(30))
    assert (p[np.tril_indices(30)] > 0).all()
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=1e-13)


def test_gla_rows_subset():
    q, k, v, g, rng = rnd(65, 70, 8, 4)
    beta = np.array([0.3, 1.0, 3.0, 7.0])
    full = head(oracle.fem_gla, q, k, v, g, beta)
    rows = np.array([0, 3, 64, 69])
    np.testing.assert_allclose(head(oracle.fem_gla, q, k, v, g, beta, rows=rows), full[rows],
                               rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# Planted mistakes
# ---------------------------------------------------------------------------
def _gla_pins_pass(fn):
    fails = []
    q, k, v, g, rng = rnd(66, 10, 4, 2, gscale=1.5)
    beta = np.array([0.7, 4.0])
    want = np.array(brute.brute_fem_gla(q.tolist(), k.tolist(), v.tolist(), g.tolist(),
                                        beta.tolist(), fo.GLA_EPS, fo.GLA_ROPE_BASE, dps=30),
                    dtype=np.float64)
    if np.abs(head(fn, q, k, v, g, beta) - want).max() > 1e-9:
        fails.append("brute")
    T, d, gamma = 20, 4, -0.4
    z = np.zeros((T, d))
    zv = np.zeros((T, 1))
    zv[0] = 1.0
    # under the geometric prior the read of v = e_0 is (1/beta) log(1 + p_t(0)(e^beta - 1))
    o = head(fn, z, z, zv, np.full((T, d), gamma), np.array([1.0]))[:, 0]
    w = math.exp(gamma)
    t = np.arange(T)
    p0 = w ** t * (1 - w) / (1 - w ** (t + 1))
    if np.abs(o - np.log1p(p0 * (math.e - 1))).max() > 1e-10:
        fails.append("geometric")
    return fails


def _mutant(patch):
    def fn(*a, **kw):
        saved = {name: getattr(fo, name) for name in patch}
        try:
            for name, f in patch.items():
                setattr(fo, name, f)
            return fo.fem_gla(*a, **kw)
        finally:
            for name, f in saved.items():
                setattr(fo, name, f)
    return fn


_prior = fo.gla_prior_rows
_rope = fo.rope


def _prior_decay_from_i(q, k, g, rows):
    # exp(sum_{tau=i+2}^{t+1} g): the decay window shifted by one step
    n = int(rows.max()) + 1
    g2 = np.concatenate([g[1:n], np.zeros((1, g.shape[1]))])
    return _prior(q, k, np.concatenate([g2, g[n:]]), rows)


def _prior_decay_halved(q, k, g, rows):
    return _prior(q, k, 0.5 * g, rows)


def _rope_rotate_half(x, pos, base=fo.GLA_ROPE_BASE):
    d = x.shape[-1]
    h = d // 2
    theta = base ** (-2.0 * np.arange(h) / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * theta[None, :]
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x, dtype=np.float64)
    out[:, :h] = x[:, :h] * c - x[:, h:] * s
    out[:, h:] = x[:, :h] * s + x[:, h:] * c
    return out


def _features_no_relu(x, pos):
    return _rope(x, pos) + fo.GLA_EPS


@pytest.mark.parametrize("name,patch", [
    ("decay window shifted by one step", {"gla_prior_rows": _prior_decay_from_i}),
    ("decay rate halved", {"gla_prior_rows": _prior_decay_halved}),
    ("RoPE pairs (m, m + d/2)", {"rope": _rope_rotate_half}),
    ("ReLU left out", {"gla_features": _features_no_relu}),
])
def test_gla_pins_catch_planted_mistakes(name, patch):
    assert _gla_pins_pass(oracle.fem_gla) == []
    with np.errstate(all="ignore"):
        assert _gla_pins_pass(_mutant(patch)) != [], name
