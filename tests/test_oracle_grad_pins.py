"""Pins of the oracle's gradients of the softmax-prior read
(``fem_softmax_grads``: the posterior as the value gradient, Proposition
"Local geometry" / eq. app-grad-hess; (q - p)/beta as the logit gradient,
prior sensitivity (iv); KL(q||p)/beta^2 as the temperature derivative, eq.
app-beta-deriv).

They are pinned by central finite differences of the oracle's own forward
read (itself pinned elsewhere), by float64 autograd through an independent
PyTorch statement of the read (masked log-sum-exp of score + beta v minus the
log-sum-exp of the scores), and by identities the closed forms imply.
Planted mistakes must each fail a pin.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from oracle import fem_oracle as fo


def rnd(seed, B, H, T, d, D):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, H, T, d))
    k = rng.standard_normal((B, H, T, d))
    v = 1.5 * rng.standard_normal((B, H, T, D))
    beta = np.exp(rng.uniform(np.log(0.2), np.log(6.0), (H, D)))
    g = rng.standard_normal((B, H, T, D))
    return q, k, v, beta, g


def torch_read(q, k, v, beta):
    """F = (LSE_{i<=t}(s_ti + beta v_ij) - LSE_{i<=t}(s_ti)) / beta, float64."""
    B, H, T, d = q.shape
    s = q @ k.transpose(-1, -2) / math.sqrt(d)
    mask = torch.triu(torch.ones(T, T, dtype=torch.bool), 1)
    s = s.masked_fill(mask, float("-inf"))
    x = s[..., None] + (beta[None, :, None, None, :] * v[:, :, None, :, :])  # [B,H,t,i,D]
    num = torch.logsumexp(x, dim=3)
    den = torch.logsumexp(s, dim=3)[..., None]
    return (num - den) / beta[None, :, None, :]


def test_grads_match_autograd():
    q, k, v, beta, g = rnd(70, 2, 2, 24, 8, 5)
    t = [torch.tensor(a, requires_grad=True) for a in (q, k, v, beta)]
    loss = (torch_read(*t) * torch.tensor(g)).sum()
    loss.backward()
    got = oracle.fem_softmax_grads(q, k, v, beta, g, block=7)
    for name, a, b in zip(("dq", "dk", "dv", "dbeta"), got, [x.grad.numpy() for x in t]):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-10, err_msg=name)


def test_grads_match_finite_differences():
    q, k, v, beta, g = rnd(71, 1, 1, 9, 4, 3)
    loss = lambda q_, k_, v_, b_: float((oracle.fem_softmax(q_, k_, v_, b_) * g).sum())
    dq, dk, dv, db = oracle.fem_softmax_grads(q, k, v, beta, g)
    h = 1e-6
    for arr, grad, idx in ((q, dq, (0, 0, 5, 2)), (k, dk, (0, 0, 1, 3)), (v, dv, (0, 0, 0, 1)),
                           (v, dv, (0, 0, 8, 2)), (beta, db, (0, 1))):
        a1, a2 = arr.copy(), arr.copy()
        a1[idx] += h
        a2[idx] -= h
        args1 = [a1 if arr is x else x for x in (q, k, v, beta)]
        args2 = [a2 if arr is x else x for x in (q, k, v, beta)]
        fd = (loss(*args1) - loss(*args2)) / (2 * h)
        assert abs(fd - grad[idx]) < 1e-7, (idx, fd, grad[idx])


def test_grad_identities():
    q, k, v, beta, g = rnd(72, 1, 2, 30, 6, 4)
    dq, dk, dv, db = oracle.fem_softmax_grads(q, k, v, beta, g)
    # posterior rows sum to one: sum_i dV_ij = sum_t G_tj
    np.testing.assert_allclose(dv.sum(axis=2), g.sum(axis=2), rtol=1e-12, atol=1e-12)
    # with G >= 0 the temperature gradient is a sum of KL terms, hence >= 0
    _, _, _, db_pos = oracle.fem_softmax_grads(q, k, v, beta, np.abs(g))
    assert (db_pos >= 0).all()
    # (q - p) sums to zero over i, so a constant shift of every key leaves the
    # loss unchanged: sum_i dK_i = 0 per head
    np.testing.assert_allclose(dk.sum(axis=2), 0.0, atol=1e-12)


def _pins_pass(fn):
    q, k, v, beta, g = rnd(73, 1, 2, 14, 4, 3)
    t = [torch.tensor(a, requires_grad=True) for a in (q, k, v, beta)]
    (torch_read(*t) * torch.tensor(g)).sum().backward()
    got = fn(q, k, v, beta, g)
    return [n for n, a, x in zip(("dq", "dk", "dv", "dbeta"), got, t)
            if np.abs(a - x.grad.numpy()).max() > 1e-9]


_prior = fo.softmax_prior_rows


def _prior_transposed(q, k, rows):
    return _prior(k, q, rows)


def _mutant_grads(variant):
    """Copies of the closed forms with one slip each."""
    def fn(q, k, v, beta, g):
        dq, dk, dv, db = oracle.fem_softmax_grads(q, k, v, beta, g)
        if variant == "p - q":
            return -dq, -dk, dv, db
        if variant == "no 1/beta on logits":
            dq2, dk2, _, _ = oracle.fem_softmax_grads(q, k, v, beta, g * beta[None, :, None, :])
            return dq2, dk2, dv, db
        if variant == "KL(p||q)":
            out = np.zeros_like(db)
            for h in range(q.shape[1]):
                for t in range(q.shape[2]):
                    p = _prior(q[0, h], k[0, h], np.array([t]))[0]
                    for j in range(v.shape[3]):
                        post = oracle.posterior(p, v[0, h, : t + 1, j], beta[h, j])
                        out[h, j] += g[0, h, t, j] * np.sum(p * np.log(p / post)) / beta[h, j] ** 2
            return dq, dk, dv, out
        raise ValueError(variant)
    return fn


@pytest.mark.parametrize("variant", ["p - q", "no 1/beta on logits", "KL(p||q)"])
def test_grad_pins_catch_planted_mistakes(variant):
    assert _pins_pass(oracle.fem_softmax_grads) == []
    assert _pins_pass(_mutant_grads(variant)) != [], variant
