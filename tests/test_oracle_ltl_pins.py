"""Pins of the oracle's two-level gated read (Sec. "Linearized Temperature
Learning" and "Two-Level Gated FEM": eqs. ltl, ltl-final, inner-gate-main,
fem-two-gates-main; Appendix "Monotonicity and hidden temperature").

The gated read is pinned through facts that do not retype it:
  * lam = 0 is the prior's expectation, i.e. causal softmax attention from
    PyTorch's library routine, and under a uniform prior the running mean;
  * lam = 1 is the free energy at beta_max, pinned by the reverse-KL identity
    (eq. revKL) and, under a uniform prior, by logcumsumexp;
  * the read is affine in lam and positively homogeneous in g, element-wise;
  * the sandwich mu <= F~ <= F(beta_max), and the hidden temperature of
    Proposition "Inner gate as hidden-temperature free energy": bisection over
    beta on the un-gated free energy recovers F~ at some beta* in [0, beta_max],
    increasing in lam, with the KL fraction of Appendix "KL-controlled
    interpretation of the gate".
``test_ltl_pins_catch_planted_mistakes`` plants slips into copies of the
oracle and checks that these pins reject each one.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from oracle import fem_oracle as fo


def head(fn, q, k, v, beta, lam, gate=None, **kw):
    g = None if gate is None else gate[None, None]
    return fn(q[None, None], k[None, None], v[None, None], np.asarray(beta)[None],
              lam[None, None], g, **kw)[0, 0]


def rnd(seed, T, d, D, scale=2.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((T, d)), rng.standard_normal((T, d)),
            scale * rng.standard_normal((T, D)), rng)


def sdpa_causal(q, k, v):
    """Causal softmax attention from PyTorch's library routine (float64)."""
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))[None, None]
    o = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=True)
    return o[0, 0].numpy()


def causal_alpha(q, k):
    T, d = q.shape
    s = torch.from_numpy(q @ k.T / math.sqrt(d))
    s = s.masked_fill(torch.triu(torch.ones(T, T, dtype=torch.bool), 1), float("-inf"))
    return torch.softmax(s, dim=1).numpy()


def free_energy_direct(p, v, beta):
    """F(beta) of one row and channel by a plain sum (beta = 0 is the mean)."""
    if beta == 0.0:
        return float(np.dot(p, v))
    x = beta * v
    c = x.max()
    return float((math.log(np.dot(p, np.exp(x - c))) + c) / beta)


# ---------------------------------------------------------------------------
# Endpoints
# ---------------------------------------------------------------------------
def test_lam0_is_causal_attention():
    q, k, v, rng = rnd(31, 80, 8, 5)
    bmax = np.exp(rng.uniform(np.log(0.1), np.log(8.0), 5))
    o = head(oracle.fem_softmax_ltl, q, k, v, bmax, np.zeros((80, 5)))
    np.testing.assert_allclose(o, sdpa_causal(q, k, v), rtol=0, atol=1e-12)


def test_lam1_is_reverse_kl_identity():
    q, k, v, rng = rnd(32, 64, 8, 4)
    bmax = np.array([0.1, 0.9, 3.0, 12.0])
    o = head(oracle.fem_softmax_ltl, q, k, v, bmax, np.ones((64, 4)))
    mu = sdpa_causal(q, k, v)
    alpha = causal_alpha(q, k)
    for t in (0, 1, 30, 63):
        p = alpha[t, : t + 1]
        for j in range(4):
            w = p * np.exp(bmax[j] * (v[: t + 1, j] - v[: t + 1, j].max()))
            post = w / w.sum()
            kl = float(np.sum(p * (np.log(p) - np.log(post))))
            assert abs(o[t, j] - (mu[t, j] + kl / bmax[j])) < 1e-10


def test_uniform_prior_closed_forms():
    """q = 0 makes p_t uniform over i <= t: mu is the running mean, F the
    running log-mean-exp (logcumsumexp minus log t)."""
    _, k, v, rng = rnd(33, 50, 6, 4)
    q = np.zeros_like(k)
    bmax = np.array([0.3, 1.0, 4.0, 9.0])
    n = np.arange(1, 51)[:, None]
    mean = np.cumsum(v, axis=0) / n
    lse = (np.logaddexp.accumulate(v * bmax, axis=0) - np.log(n)) / bmax
    np.testing.assert_allclose(head(oracle.fem_softmax_ltl, q, k, v, bmax, np.zeros((50, 4))),
                               mean, rtol=0, atol=1e-12)
    np.testing.assert_allclose(head(oracle.fem_softmax_ltl, q, k, v, bmax, np.ones((50, 4))),
                               lse, rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# Structure in lam and g
# ---------------------------------------------------------------------------
def test_affine_in_lam_and_homogeneous_in_gate():
    q, k, v, rng = rnd(34, 70, 8, 6)
    bmax = np.exp(rng.uniform(np.log(0.1), np.log(8.0), 6))
    f = lambda lam, g=None: head(oracle.fem_softmax_ltl, q, k, v, bmax, lam, g)
    o0, o1 = f(np.zeros((70, 6))), f(np.ones((70, 6)))
    lam = rng.uniform(0, 1, (70, 6))
    np.testing.assert_allclose(f(lam), o0 + lam * (o1 - o0), rtol=0, atol=1e-12)
    g = np.exp(rng.standard_normal((70, 6)))
    np.testing.assert_allclose(f(lam, g), g * f(lam), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(f(lam, np.ones((70, 6))), f(lam), rtol=0, atol=0)


def test_sandwich_and_hidden_temperature():
    q, k, v, rng = rnd(35, 40, 8, 3)
    bmax = np.array([0.5, 2.0, 7.0])
    alpha = causal_alpha(q, k)
    lams = np.linspace(0.0, 1.0, 6)
    mu = sdpa_causal(q, k, v)
    fmax = head(oracle.fem_softmax_ltl, q, k, v, bmax, np.ones((40, 3)))
    for t in (3, 17, 39):
        p = alpha[t, : t + 1]
        for j in range(3):
            vj = v[: t + 1, j]
            prev = -1.0
            for lam in lams:
                lm = np.full((40, 3), lam)
                o = head(oracle.fem_softmax_ltl, q, k, v, bmax, lm)[t, j]
                assert mu[t, j] - 1e-12 <= o <= fmax[t, j] + 1e-12
                lo, hi = 0.0, float(bmax[j])
                for _ in range(200):
                    mid = 0.5 * (lo + hi)
                    if free_energy_direct(p, vj, mid) < o:
                        lo = mid
                    else:
                        hi = mid
                bstar = 0.5 * (lo + hi)
                assert 0.0 <= bstar <= bmax[j]
                assert abs(free_energy_direct(p, vj, bstar) - o) < 1e-10
                assert bstar >= prev
                prev = bstar
                if 0.0 < lam < 1.0:
                    # F(beta*) - mu is lam times the achievable KL improvement
                    w = p * np.exp(bstar * (vj - vj.max()))
                    kl = float(np.sum(p * (np.log(p) - np.log(w / w.sum()))))
                    gain = fmax[t, j] - mu[t, j]
                    assert abs(kl / bstar - lam * gain) < 1e-9


def test_ltl_rows_subset_and_causality():
    q, k, v, rng = rnd(36, 90, 8, 4)
    bmax = np.exp(rng.uniform(np.log(0.1), np.log(8.0), 4))
    lam = rng.uniform(0, 1, (90, 4))
    g = np.exp(rng.standard_normal((90, 4)))
    full = head(oracle.fem_softmax_ltl, q, k, v, bmax, lam, g, block=16)
    rows = np.array([0, 5, 47, 89])
    sub = oracle.fem_softmax_ltl(q[None, None], k[None, None], v[None, None], bmax[None],
                                 lam[None, None], g[None, None], rows=rows)[0, 0]
    np.testing.assert_allclose(sub, full[rows], rtol=0, atol=1e-12)
    k2, v2 = k.copy(), v.copy()
    k2[50:] *= -2
    v2[50:] += 3
    o2 = head(oracle.fem_softmax_ltl, q, k2, v2, bmax, lam, g)
    np.testing.assert_allclose(o2[:50], full[:50], rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# Planted mistakes
# ---------------------------------------------------------------------------
def _ltl_pins_pass(fn):
    fails = []
    q, k, v, rng = rnd(41, 48, 8, 4)
    bmax = np.array([0.2, 1.0, 3.0, 9.0])
    z, one = np.zeros((48, 4)), np.ones((48, 4))
    o0 = head(fn, q, k, v, bmax, z)
    if np.abs(o0 - sdpa_causal(q, k, v)).max() > 1e-9:
        fails.append("lam0")
    o1 = head(fn, q, k, v, bmax, one)
    qz = np.zeros_like(q)
    n = np.arange(1, 49)[:, None]
    lse = (np.logaddexp.accumulate(v * bmax, axis=0) - np.log(n)) / bmax
    if np.abs(head(fn, qz, k, v, bmax, one) - lse).max() > 1e-9:
        fails.append("lam1")
    lam = rng.uniform(0, 1, (48, 4))
    if np.abs(head(fn, q, k, v, bmax, lam) - (o0 + lam * (o1 - o0))).max() > 1e-9:
        fails.append("affine")
    g = np.exp(rng.standard_normal((48, 4)))
    if np.abs(head(fn, q, k, v, bmax, lam, g) - g * head(fn, q, k, v, bmax, lam)).max() > 1e-9:
        fails.append("gate")
    return fails


def _mutant(patch):
    def fn(*a, **kw):
        saved = {name: getattr(fo, name) for name in patch}
        try:
            for name, f in patch.items():
                setattr(fo, name, f)
            return fo.fem_softmax_ltl(*a, **kw)
        finally:
            for name, f in saved.items():
                setattr(fo, name, f)
    return fn


_free_energy = fo.free_energy_read


def _ltl_lam_swapped(p, v, beta_max, lam, gate=None, logp=None):
    o = lam * (p @ v) + (1.0 - lam) * _free_energy(p, v, beta_max, logp=logp)
    return o if gate is None else gate * o


def _ltl_gate_on_fmax_only(p, v, beta_max, lam, gate=None, logp=None):
    f = _free_energy(p, v, beta_max, logp=logp)
    return (1.0 - lam) * (p @ v) + lam * (f if gate is None else gate * f)


def _ltl_half_beta(p, v, beta_max, lam, gate=None, logp=None):
    o = (1.0 - lam) * (p @ v) + lam * _free_energy(p, v, 0.5 * beta_max, logp=logp)
    return o if gate is None else gate * o


def _mean_uniform(p, v):
    w = (p > 0).astype(np.float64)
    return (w / w.sum(1, keepdims=True)) @ v


def _mean_summed(p, v):
    return (p > 0).astype(np.float64) @ v


@pytest.mark.parametrize("name,patch", [
    ("lam and 1 - lam swapped", {"ltl_read": _ltl_lam_swapped}),
    ("outer gate on the F branch only", {"ltl_read": _ltl_gate_on_fmax_only}),
    ("F taken at beta_max / 2", {"ltl_read": _ltl_half_beta}),
    ("mean ignores the prior", {"expectation_read": _mean_uniform}),
    ("support sum instead of mean", {"expectation_read": _mean_summed}),
])
def test_ltl_pins_catch_planted_mistakes(name, patch):
    assert _ltl_pins_pass(oracle.fem_softmax_ltl) == []
    assert _ltl_pins_pass(_mutant(patch)) != [], name
