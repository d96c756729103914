"""Brute-force arbitrary-precision evaluation of the FEM read (test infrastructure).

Evaluates the definitions term by term with mpmath at a chosen number of
digits, with no shift, no matrix product and no vectorisation, for tiny
inputs (T up to a few dozen).  It pins the float64 oracle:

  s_{t,i} = q_t . k_i / sqrt(d)                     (Sec. 1, masked scores)
  alpha_{t,i} = exp(s_{t,i}) / sum_{r<=t} exp(s_{t,r})
                 (encoder read: every key r < T, since encoder-only use
                  removes the mask, Sec. "Empirical Evaluation")
  p_t(i) = <phi q_t, phi k_i> / sum_{r<=t} <phi q_t, phi k_r>, phi = elu + 1
  F_{t,j} = log( sum_{i<=t} p_t(i) exp(beta_j v_{i,j}) ) / beta_j
                                   (Sec. 2.3, eq. fem-free-energy-main)
"""

from __future__ import annotations

import mpmath


def _phi(x):
    return x + 1 if x > 0 else mpmath.e ** x


def brute_read(prior_rows, v, beta, dps=50):
    """prior_rows[t] = list of p_t(i) over the support (i <= t, or every i
    for the encoder read) as mpf; v: T x D; beta: D."""
    with mpmath.workdps(dps):
        T = len(v)
        D = len(v[0])
        out = []
        for t in range(T):
            row = []
            for j in range(D):
                b = mpmath.mpf(beta[j])
                acc = mpmath.mpf(0)
                for i in range(len(prior_rows[t])):
                    acc += prior_rows[t][i] * mpmath.exp(b * mpmath.mpf(v[i][j]))
                row.append(mpmath.log(acc) / b)
            out.append(row)
        return out


def brute_softmax_prior(q, k, dps=50, causal=True):
    with mpmath.workdps(dps):
        T = len(q)
        d = len(q[0])
        rows = []
        for t in range(T):
            s = []
            for i in range(t + 1 if causal else T):
                dot = mpmath.mpf(0)
                for c in range(d):
                    dot += mpmath.mpf(q[t][c]) * mpmath.mpf(k[i][c])
                s.append(mpmath.e ** (dot / mpmath.sqrt(d)))
            z = sum(s)
            rows.append([x / z for x in s])
        return rows


def brute_linear_prior(q, k, dps=50):
    with mpmath.workdps(dps):
        T = len(q)
        d = len(q[0])
        rows = []
        for t in range(T):
            s = []
            for i in range(t + 1):
                dot = mpmath.mpf(0)
                for c in range(d):
                    dot += _phi(mpmath.mpf(q[t][c])) * _phi(mpmath.mpf(k[i][c]))
                s.append(dot)
            z = sum(s)
            rows.append([x / z for x in s])
        return rows


def brute_fem_softmax(q, k, v, beta, dps=50):
    """One head: q, k: T x d; v: T x D; beta: D (nested lists or arrays)."""
    return brute_read(brute_softmax_prior(q, k, dps), v, beta, dps)


def brute_fem_softmax_encoder(q, k, v, beta, dps=50):
    """Encoder (unmasked) read of one head."""
    return brute_read(brute_softmax_prior(q, k, dps, causal=False), v, beta, dps)


def brute_fem_linear(q, k, v, beta, dps=50):
    return brute_read(brute_linear_prior(q, k, dps), v, beta, dps)


def brute_gla_prior(q, k, g, eps, base, dps=50):
    """GLA prior rows term by term: features ReLU(RoPE(x)) + eps, decay
    exp(sum_{tau=i+1}^{t} g_tau) per key channel (Appendix "Gated Linear
    Attention (GLA) Prior", eq. gla-score-appendix)."""
    with mpmath.workdps(dps):
        T = len(q)
        d = len(q[0])

        def feat(x, t):
            out = [mpmath.mpf(0)] * d
            for m in range(d // 2):
                ang = t * mpmath.power(mpmath.mpf(base), -mpmath.mpf(2 * m) / d)
                c, s = mpmath.cos(ang), mpmath.sin(ang)
                a, b = mpmath.mpf(x[2 * m]), mpmath.mpf(x[2 * m + 1])
                out[2 * m] = a * c - b * s
                out[2 * m + 1] = a * s + b * c
            return [max(u, 0) + mpmath.mpf(eps) for u in out]

        gg = [[mpmath.mpf(g[t][c]) for c in range(d)] for t in range(T)]
        rows = []
        for t in range(T):
            fq = feat(q[t], t)
            s = []
            for i in range(t + 1):
                fk = feat(k[i], i)
                tot = mpmath.mpf(0)
                for c in range(d):
                    dec = mpmath.exp(sum(gg[tau][c] for tau in range(i + 1, t + 1)))
                    tot += fq[c] * fk[c] * dec
                s.append(tot)
            z = sum(s)
            rows.append([x / z for x in s])
        return rows


def brute_fem_gla(q, k, v, g, beta, eps, base, dps=50):
    return brute_read(brute_gla_prior(q, k, g, eps, base, dps), v, beta, dps)
