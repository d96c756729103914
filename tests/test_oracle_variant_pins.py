"""Pins of the oracle's read variants: the encoder (unmasked) read and a value
width d_v different from d_qk.

The encoder read (encoder-only use removes the causal mask, Sec. "Empirical
Evaluation") is pinned by facts that do not retype it:
  * 50-digit term-by-term evaluation (``oracle.brute``);
  * row t equals the causal read's last row when q_t is the last query;
  * joint permutations of the (k_i, v_i) pairs leave every row unchanged;
  * under a uniform prior every row is the log-mean-exp of the whole column;
  * beta -> 0 gives unmasked softmax attention (torch SDPA, float64).
The decode step against a KV cache is pinned to the causal read's row t
(query t over the first t + 1 keys) and to the 50-digit evaluation.
d_v != d_qk (budget (i) of Sec. "Free Energy Mixer", d_v = d_qk / 2): the
score scale stays 1/sqrt(d_qk) and each value channel is read independently,
so the read of a value subset equals the read of the full width restricted to
that subset, and the 50-digit evaluation covers it directly.
"""

import math

import mpmath
import numpy as np
import pytest
import torch

import oracle
from oracle import brute
from oracle import fem_oracle as fo


def head(fn, q, k, v, beta, **kw):
    return fn(q[None, None], k[None, None], v[None, None], np.asarray(beta)[None], **kw)[0, 0]


def rnd(seed, T, d, D, scale=2.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((T, d)), rng.standard_normal((T, d)),
            scale * rng.standard_normal((T, D)), rng)


@pytest.mark.parametrize("seed,T,d,D", [(51, 13, 4, 3), (52, 20, 6, 2)])
def test_encoder_brute_force(seed, T, d, D):
    q, k, v, rng = rnd(seed, T, d, D)
    beta = np.exp(rng.uniform(np.log(0.05), np.log(16.0), D))
    want = np.array(brute.brute_fem_softmax_encoder(q.tolist(), k.tolist(), v.tolist(),
                                                    beta.tolist()), dtype=np.float64)
    np.testing.assert_allclose(head(oracle.fem_softmax_encoder, q, k, v, beta), want,
                               rtol=0, atol=1e-12)


def test_encoder_row_is_causal_last_row():
    q, k, v, rng = rnd(53, 40, 8, 5)
    beta = np.exp(rng.uniform(np.log(0.1), np.log(8.0), 5))
    enc = head(oracle.fem_softmax_encoder, q, k, v, beta)
    for t in (0, 7, 39):
        q2 = q.copy()
        q2[-1] = q[t]
        last = head(oracle.fem_softmax, q2, k, v, beta, rows=np.array([39]))[0]
        np.testing.assert_allclose(enc[t], last, rtol=0, atol=1e-12)


def test_encoder_key_permutation_invariance():
    q, k, v, rng = rnd(54, 33, 8, 4)
    beta = np.array([0.2, 1.0, 4.0, 12.0])
    perm = rng.permutation(33)
    a = head(oracle.fem_softmax_encoder, q, k, v, beta)
    b = head(oracle.fem_softmax_encoder, q, k[perm], v[perm], beta)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_encoder_uniform_prior_and_small_beta():
    _, k, v, rng = rnd(55, 30, 6, 4)
    beta = np.array([0.3, 1.0, 3.0, 9.0])
    u = head(oracle.fem_softmax_encoder, np.zeros_like(k), k, v, beta)
    want = (np.logaddexp.reduce(v * beta, axis=0) - math.log(30)) / beta
    np.testing.assert_allclose(u, np.broadcast_to(want, u.shape), rtol=0, atol=1e-12)
    q = rng.standard_normal(k.shape)
    small = head(oracle.fem_softmax_encoder, q, k, v, np.full(4, 1e-7))
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))[None, None]
    mu = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v))[0, 0].numpy()
    np.testing.assert_allclose(small, mu, rtol=0, atol=1e-5)


def test_value_width_half_of_key_width():
    q, k, v, rng = rnd(56, 15, 8, 4)
    beta = np.array([0.3, 1.5, 5.0, 0.8])
    for fn, bf in ((oracle.fem_softmax, brute.brute_fem_softmax),
                   (oracle.fem_softmax_encoder, brute.brute_fem_softmax_encoder)):
        want = np.array(bf(q.tolist(), k.tolist(), v.tolist(), beta.tolist()), dtype=np.float64)
        got = head(fn, q, k, v, beta)
        assert got.shape == (15, 4)
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)
        wide = np.concatenate([v, rng.standard_normal((15, 4))], axis=1)
        bw = np.concatenate([beta, [1.0, 2.0, 3.0, 4.0]])
        np.testing.assert_allclose(head(fn, q, k, wide, bw)[:, :4], got, rtol=0, atol=1e-12)


def _enc_pins_pass(fn):
    fails = []
    q, k, v, rng = rnd(57, 24, 6, 3)
    beta = np.array([0.5, 2.0, 8.0])
    want = np.array(brute.brute_fem_softmax_encoder(q.tolist(), k.tolist(), v.tolist(),
                                                    beta.tolist(), dps=30), dtype=np.float64)
    if np.abs(head(fn, q, k, v, beta) - want).max() > 1e-10:
        fails.append("brute")
    perm = rng.permutation(24)
    if np.abs(head(fn, q, k, v, beta) - head(fn, q, k[perm], v[perm], beta)).max() > 1e-10:
        fails.append("perm")
    return fails


def _mutant(patch):
    def fn(*a, **kw):
        saved = {name: getattr(fo, name) for name in patch}
        try:
            for name, f in patch.items():
                setattr(fo, name, f)
            return fo.fem_softmax_encoder(*a, **kw)
        finally:
            for name, f in saved.items():
                setattr(fo, name, f)
    return fn


_prior_all = fo.softmax_prior_all
_prior_causal = fo.softmax_prior_rows


def _prior_causal_left_in(q, k, rows):
    p = _prior_causal(q, k, rows)
    return np.pad(p, ((0, 0), (0, q.shape[0] - p.shape[1])))


def _prior_drops_last_key(q, k, rows):
    p = _prior_all(q, k, rows)
    p[:, -1] = 0.0
    return p / p.sum(axis=1, keepdims=True)


def _prior_sqrt_dv(q, k, rows):
    s = (q[rows] @ k.T) / math.sqrt(2 * q.shape[1])
    e = np.exp(s - s.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


@pytest.mark.parametrize("name,patch", [
    ("causal mask left in", {"softmax_prior_all": _prior_causal_left_in,
                             "softmax_logprior_all": lambda q, k, r: np.log(_prior_causal_left_in(q, k, r))}),
    ("last key dropped", {"softmax_prior_all": _prior_drops_last_key,
                          "softmax_logprior_all": lambda q, k, r: np.log(_prior_drops_last_key(q, k, r))}),
    ("wrong score scale", {"softmax_prior_all": _prior_sqrt_dv,
                           "softmax_logprior_all": lambda q, k, r: np.log(_prior_sqrt_dv(q, k, r))}),
])
def test_encoder_pins_catch_planted_mistakes(name, patch):
    assert _enc_pins_pass(oracle.fem_softmax_encoder) == []
    with np.errstate(divide="ignore"):
        assert _enc_pins_pass(_mutant(patch)) != [], name


# ---------------------------------------------------------------------------
# Decode step against a KV cache
# ---------------------------------------------------------------------------
def test_decode_is_causal_row():
    """The decode read of q_t over the first t+1 cached keys is row t of the
    causal read (whose own pins fix it)."""
    rng = np.random.default_rng(58)
    B, H, L, d, dv = 2, 3, 50, 8, 4
    q = rng.standard_normal((B, H, L, d))
    k = rng.standard_normal((B, H, L, d))
    v = 2 * rng.standard_normal((B, H, L, dv))
    beta = np.exp(rng.uniform(np.log(0.1), np.log(8.0), (H, dv)))
    full = oracle.fem_softmax(q, k, v, beta)
    for t in (0, 1, 31, 49):
        lens = np.array([t + 1, t + 1])
        got = oracle.fem_softmax_decode(q[:, :, t], k, v, lens, beta)
        np.testing.assert_allclose(got, full[:, :, t], rtol=0, atol=1e-12)
    lens = np.array([7, 50])
    got = oracle.fem_softmax_decode(q[:, :, 20], k, v, lens, beta)
    want0 = oracle.fem_softmax_encoder(q[0:1, :, 20:21], k[0:1, :, :7], v[0:1, :, :7], beta)[0, :, 0]
    np.testing.assert_allclose(got[0], want0, rtol=0, atol=1e-12)


def test_decode_brute_force():
    rng = np.random.default_rng(59)
    L, d, dv = 11, 4, 3
    q = rng.standard_normal((1, 1, d))
    k = rng.standard_normal((1, 1, L, d))
    v = 2 * rng.standard_normal((1, 1, L, dv))
    beta = np.array([[0.3, 2.0, 9.0]])
    n = 8
    # brute causal read with the query in the last row: its last row is the step
    qq = np.concatenate([np.zeros((n - 1, d)), q[0, 0][None]], axis=0)
    want = brute.brute_fem_softmax(qq.tolist(), k[0, 0, :n].tolist(), v[0, 0, :n].tolist(),
                                   beta[0].tolist())[-1]
    got = oracle.fem_softmax_decode(q, k, v, np.array([n]), beta)[0, 0]
    np.testing.assert_allclose(got, np.array(want, dtype=np.float64), rtol=0, atol=1e-12)
