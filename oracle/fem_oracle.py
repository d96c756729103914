"""Plain float64 oracle of the Free Energy Mixer (FEM) read.

TEST INFRASTRUCTURE.  This module is a slow, obviously-correct CPU statement of
what the HIP library computes.  It is used only by the tests, the smoke check
and the CPU-baseline leg of the benchmark; the product path never touches it.
It shares no code with the HIP path: the only thing the two sides share is the
seeded input generator, which holds none of the method's arithmetic.

What is computed (paper, Sec. 1 and Sec. 2.3; Appendix "Selection
distributions, support, and normalization"; Appendix "Parameterizations of the
Prior Selection", softmax prior):

  prior     p_t(i) = softmax over i <= t of  q_t . k_i / sqrt(d)      (softmax)
            p_t(i) = <phi(q_t), phi(k_i)> / sum_{r<=t} <phi(q_t), phi(k_r)>
                     with phi = elu + 1                                (linear)
            p_t(i) = softmax over every i < T                  (encoder: no mask)
            p_t(i) propto <q~_t, exp(G_t - G_i) k~_i>, q~ = ReLU(RoPE(q)) + eps,
                     G_t = sum_{tau<=t} g_tau                         (GLA)
  read      F_{t,j} = (1 / beta_j) * log sum_{i<=t} p_t(i) * exp(beta_j v_{i,j})
                                  (free-energy read, eq. fem-free-energy-main)
  gated     o_{t,j} = g_{t,j} * ((1 - lam_{t,j}) * mu_{t,j} + lam_{t,j} * F_{t,j}(beta_max))
            mu_{t,j} = sum_{i<=t} p_t(i) v_{i,j}
                                  (two-level gated read, eqs. ltl-final,
                                   inner-gate-main, fem-two-gates-main)

Indices are 0-based here; the causal support of row t is {0, ..., t}, diagonal
included.  The read is exact up to float64 rounding: the only numerical device
is the per-channel log-sum-exp shift of the paper's "Numerical stability"
paragraph (Appendix, two-level gated FEM), i.e. a constant c_j subtracted
inside the exponential and added back after the logarithm, which is an exact
identity for any constant.

Nothing here is blocked, fused or reordered beyond evaluating the rows of the
output independently (each row's formula is unchanged) and using a float64
matrix product for the sum over i.
"""

from __future__ import annotations

import math

import numpy as np

# Smallest per-(t, j) sum that the shifted matrix-product evaluation accepts;
# anything smaller is recomputed with a joint per-(t, j) log-sum-exp, which has
# no underflow at all.  float64's normal range ends near 2.2e-308.
_TINY = 1e-280


def elu_plus_one(x: np.ndarray) -> np.ndarray:
    """phi(x) = elu(x) + 1: x + 1 for x > 0, exp(x) for x <= 0.

    The paper leaves the nonnegative feature map of the linear prior open
    (Appendix "Selection distributions ..."); the oracle fixes phi = elu + 1.
    """
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0, x + 1.0, np.exp(np.minimum(x, 0.0)))


def softmax_prior_rows(q: np.ndarray, k: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """Causal softmax prior for the requested query rows.

    q: [T, d], k: [T, d] float64; rows: 1-D int array of query indices.
    Returns P with P[r, i] = p_{rows[r]}(i) for i < n, n = max(rows) + 1,
    and P[r, i] = 0 for i > rows[r] (causal mask, support {0..t}).
    Sec. 1 (masked scores s_{t,i} = q_t.k_i / sqrt d, -inf for i > t;
    alpha = softmax(s)).
    """
    d = q.shape[1]
    n = int(rows.max()) + 1
    s = (q[rows] @ k[:n].T) / math.sqrt(d)
    mask = np.arange(n)[None, :] <= rows[:, None]
    s = np.where(mask, s, -np.inf)
    s = s - s.max(axis=1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=1, keepdims=True)


def softmax_logprior_rows(q: np.ndarray, k: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """log p_t(i) of the causal softmax prior (-inf off the support)."""
    d = q.shape[1]
    n = int(rows.max()) + 1
    s = (q[rows] @ k[:n].T) / math.sqrt(d)
    mask = np.arange(n)[None, :] <= rows[:, None]
    s = np.where(mask, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    return s - (m + np.log(np.exp(s - m).sum(axis=1, keepdims=True)))


def softmax_prior_all(q: np.ndarray, k: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """Encoder (unmasked) softmax prior: p_t(i) = softmax_i(q_t.k_i / sqrt d)
    over every key i < T.  Encoder-only use removes the causal mask (opening of
    Sec. "Empirical Evaluation"); otherwise as softmax_prior_rows."""
    d = q.shape[1]
    s = (q[rows] @ k.T) / math.sqrt(d)
    s = s - s.max(axis=1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=1, keepdims=True)


def softmax_logprior_all(q: np.ndarray, k: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """log p_t(i) of the encoder softmax prior."""
    d = q.shape[1]
    s = (q[rows] @ k.T) / math.sqrt(d)
    m = s.max(axis=1, keepdims=True)
    return s - (m + np.log(np.exp(s - m).sum(axis=1, keepdims=True)))


def linear_prior_rows(q: np.ndarray, k: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """Causal linear-attention prior p_t(i) = <phi q_t, phi k_i> / sum_{r<=t} (...)

    Appendix "Selection distributions, support, and normalization" (linear
    attention) and the unified interface p_t(i) = s_t(i) / sum_{r<=t} s_t(r)
    (Appendix "Parameterizations of the Prior Selection").  No 1/sqrt(d)
    factor: the normalisation makes p invariant to any scaling of phi.
    """
    n = int(rows.max()) + 1
    a = elu_plus_one(q[rows]) @ elu_plus_one(k[:n]).T
    mask = np.arange(n)[None, :] <= rows[:, None]
    a = np.where(mask, a, 0.0)
    return a / a.sum(axis=1, keepdims=True)


def free_energy_read(p: np.ndarray, v: np.ndarray, beta: np.ndarray,
                     logp=None) -> np.ndarray:
    """F[r, j] = (1/beta_j) log sum_i p[r, i] exp(beta_j v[i, j]).

    p: [R, n] prior rows (zero off the support); v: [n, D]; beta: [D] > 0.
    Eq. fem-free-energy-main / eq. fem-fixed (Sec. 2.3), evaluated as
      G = p @ exp(beta*v - c),  F = (log G + c) / beta,
    with c_j = max_i beta_j v_{i,j} (the paper's per-channel LSE shift).
    Entries whose G would fall near float64 underflow are recomputed as a
    joint log-sum-exp of log p + beta v for that single (r, j).
    ``logp`` (an array shaped like p, or a function returning one) supplies
    exact log-probabilities for that fallback; if absent, log p is taken
    from p.
    """
    beta = np.asarray(beta, dtype=np.float64)
    x = v * beta[None, :]
    c = x.max(axis=0)
    g = p @ np.exp(x - c[None, :])
    with np.errstate(divide="ignore"):
        out = (np.log(g) + c[None, :]) / beta[None, :]
    bad = ~(g > _TINY)
    if bad.any():
        if callable(logp):
            logp = logp()
        if logp is None:
            with np.errstate(divide="ignore"):
                logp = np.log(p)
        for r, j in zip(*np.nonzero(bad)):
            w = logp[r] + x[:, j]
            w = w[np.isfinite(w)]
            mw = w.max()
            out[r, j] = (mw + math.log(np.exp(w - mw).sum())) / beta[j]
    return out


def expectation_read(p: np.ndarray, v: np.ndarray) -> np.ndarray:
    """mu[r, j] = sum_i p[r, i] v[i, j], the prior's expectation of the values.

    The expectation baseline of the linearized temperature learning (Sec.
    "Linearized Temperature Learning": mu_{t,j} = E_{i ~ p_t}[v_{i,j}]).
    """
    return p @ v


def ltl_read(p: np.ndarray, v: np.ndarray, beta_max: np.ndarray, lam: np.ndarray,
             gate=None, logp=None) -> np.ndarray:
    """Two-level gated read o = g * ((1 - lam) * mu + lam * F(beta_max)).

    Eq. ltl-final (one expectation and one log-sum-exp at beta_max per
    channel), eq. inner-gate-main (the inner temperature gate lam in [0, 1])
    and eq. fem-two-gates-main (the outer gate g > 0).  p: [R, n]; v: [n, D];
    beta_max: [D]; lam, gate: [R, D] (gate None means g = 1).
    """
    mu = expectation_read(p, v)
    fmax = free_energy_read(p, v, beta_max, logp=logp)
    o = (1.0 - lam) * mu + lam * fmax
    return o if gate is None else gate * o


def posterior(p_row: np.ndarray, v_col: np.ndarray, beta: float) -> np.ndarray:
    """Posterior selector q(i) proportional to p(i) exp(beta v_i) on the support.

    Eq. fem-posterior-main (Sec. 2.3).  Used by the tests to check the
    reverse-KL identity and the gradient identity of the read.
    """
    w = np.full(p_row.shape, -np.inf)
    sup = p_row > 0
    w[sup] = np.log(p_row[sup]) + beta * v_col[sup]
    w = w - w.max()
    e = np.exp(w)
    return e / e.sum()


def _as64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def _row_blocks(rows: np.ndarray, block: int):
    for s in range(0, len(rows), block):
        yield rows[s:s + block]


def fem_softmax(q, k, v, beta, rows=None, block: int = 512) -> np.ndarray:
    """FEM read with the causal softmax prior.

    q, k: [B, H, T, d]; v: [B, H, T, d_v]; beta: [H, d_v] (> 0), shared
    over batch and time.
    rows: optional 1-D array of query rows to evaluate (default: all T).
    Returns float64 [B, H, len(rows), d].
    """
    q, k, v, beta = _as64(q), _as64(k), _as64(v), _as64(beta)
    B, H, T, _ = q.shape
    dv = v.shape[3]
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.empty((B, H, len(rows), dv))
    for b in range(B):
        for h in range(H):
            pos = 0
            for rb in _row_blocks(rows, block):
                n = int(rb.max()) + 1
                p = softmax_prior_rows(q[b, h], k[b, h], rb)
                lp = (lambda qq=q[b, h], kk=k[b, h], rr=rb:
                      softmax_logprior_rows(qq, kk, rr))
                out[b, h, pos:pos + len(rb)] = free_energy_read(
                    p, v[b, h, :n], beta[h], logp=lp)
                pos += len(rb)
    return out


def fem_softmax_grads(q, k, v, beta, gout, block: int = 128):
    """Gradients of L = sum_{b,h,t,j} gout[b,h,t,j] F[b,h,t,j] for the causal
    softmax-prior read, from the paper's closed forms:
      dF_tj/dv_ij = q_tj(i)                 (posterior; Proposition "Local
                                              geometry", eq. app-grad-hess)
      dF_tj/db_ti = (q_tj(i) - p_t(i))/beta_j  (normalized logits b; prior
                                              sensitivity, Proposition (iv))
      dF_tj/dbeta_j = KL(q_tj || p_t)/beta_j^2   (eq. app-beta-deriv)
    with q_tj(i) = p_t(i) e^{beta_j v_ij} / sum_r p_t(r) e^{beta_j v_rj} and
    b_ti = q_t.k_i / sqrt d, so dQ = dB K / sqrt d and dK = dB^T Q / sqrt d.
    Returns float64 (dq, dk, dv, dbeta) shaped like q, k, v and beta [H, d_v]
    (dbeta summed over batch and time).
    """
    q, k, v, beta, gout = _as64(q), _as64(k), _as64(v), _as64(beta), _as64(gout)
    B, H, T, d = q.shape
    dv_ = v.shape[3]
    dq, dk, dvv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    dbeta = np.zeros((H, dv_))
    for b in range(B):
        for h in range(H):
            bt = beta[h]
            x = v[b, h] * bt[None, :]                       # beta v   [T, D]
            for r0 in range(0, T, block):
                rows = np.arange(r0, min(T, r0 + block))
                n = int(rows[-1]) + 1
                p = softmax_prior_rows(q[b, h], k[b, h], rows)   # [R, n]
                with np.errstate(divide="ignore"):
                    lp = np.log(p)
                # posterior q_tj(i) in log space, per channel: [R, n, D]
                w = lp[:, :, None] + x[None, :n, :]
                m = w.max(axis=1, keepdims=True)
                post = np.exp(w - m)
                post /= post.sum(axis=1, keepdims=True)
                g = gout[b, h, rows]                          # [R, D]
                dvv[b, h, :n] += np.einsum("rj,rij->ij", g, post)
                dB = np.einsum("rj,rij->ri", g / bt[None, :], post) - \
                    p * (g / bt[None, :]).sum(axis=1, keepdims=True)
                dq[b, h, rows] += dB @ k[b, h, :n] / math.sqrt(d)
                dk[b, h, :n] += dB.T @ q[b, h, rows] / math.sqrt(d)
                with np.errstate(divide="ignore", invalid="ignore"):
                    kl = np.where(post > 0, post * (np.log(post) - lp[:, :, None]), 0.0).sum(axis=1)
                dbeta[h] += (g * kl).sum(axis=0) / bt ** 2
    return dq, dk, dvv, dbeta


def fem_softmax_encoder(q, k, v, beta, rows=None, block: int = 512) -> np.ndarray:
    """FEM read with the unmasked (encoder) softmax prior: every query sees
    all T keys.  Shapes as fem_softmax (d_v may differ from d)."""
    q, k, v, beta = _as64(q), _as64(k), _as64(v), _as64(beta)
    B, H, T, _ = q.shape
    dv = v.shape[3]
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.empty((B, H, len(rows), dv))
    for b in range(B):
        for h in range(H):
            pos = 0
            for rb in _row_blocks(rows, block):
                p = softmax_prior_all(q[b, h], k[b, h], rb)
                lp = (lambda qq=q[b, h], kk=k[b, h], rr=rb:
                      softmax_logprior_all(qq, kk, rr))
                out[b, h, pos:pos + len(rb)] = free_energy_read(p, v[b, h], beta[h], logp=lp)
                pos += len(rb)
    return out


def fem_softmax_decode(q, kc, vc, lens, beta) -> np.ndarray:
    """One decoding step against a KV cache: the read of a single new query
    per (b, h) over the first lens[b] cached keys, which include the new
    token's own key and value (the autoregressive O(T) KV-cache setting of the
    softmax prior, Appendix "Parameterizations of the Prior Selection").

    q: [B, H, d]; kc: [B, H, L, d]; vc: [B, H, L, d_v]; lens: [B] ints in
    [1, L]; beta: [H, d_v].  Returns float64 [B, H, d_v].
    """
    q, kc, vc, beta = _as64(q), _as64(kc), _as64(vc), _as64(beta)
    B, H, _, _ = kc.shape
    out = np.empty((B, H, vc.shape[3]))
    for b in range(B):
        n = int(lens[b])
        for h in range(H):
            qq = q[b, h][None, :]
            kk = kc[b, h, :n]
            p = softmax_prior_all(qq, kk, np.array([0]))
            lp = (lambda qq=qq, kk=kk: softmax_logprior_all(qq, kk, np.array([0])))
            out[b, h] = free_energy_read(p, vc[b, h, :n], beta[h], logp=lp)[0]
    return out


def fem_softmax_ltl(q, k, v, beta_max, lam, gate=None, rows=None,
                    block: int = 512) -> np.ndarray:
    """Two-level gated FEM read with the causal softmax prior.

    q, k: [B, H, T, d]; v: [B, H, T, d_v]; beta_max: [H, d_v] (> 0);
    lam: [B, H, T, d_v] in [0, 1]; gate: [B, H, T, d_v] (> 0) or None (= 1).
    rows: optional query rows (default all T).  Returns float64
    [B, H, len(rows), d_v].
    """
    q, k, v, beta_max, lam = _as64(q), _as64(k), _as64(v), _as64(beta_max), _as64(lam)
    gate = None if gate is None else _as64(gate)
    B, H, T, _ = q.shape
    dv = v.shape[3]
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.empty((B, H, len(rows), dv))
    for b in range(B):
        for h in range(H):
            pos = 0
            for rb in _row_blocks(rows, block):
                n = int(rb.max()) + 1
                p = softmax_prior_rows(q[b, h], k[b, h], rb)
                lp = (lambda qq=q[b, h], kk=k[b, h], rr=rb:
                      softmax_logprior_rows(qq, kk, rr))
                g = None if gate is None else gate[b, h, rb]
                out[b, h, pos:pos + len(rb)] = ltl_read(
                    p, v[b, h, :n], beta_max[h], lam[b, h, rb], g, logp=lp)
                pos += len(rb)
    return out


# ---------------------------------------------------------------------------
# Gated linear attention (GLA) prior (Appendix "Gated Linear Attention (GLA)
# Prior": RoPE, then ReLU + eps features; decay envelope; eqs.
# gla-score-appendix and gla-assoc).
# ---------------------------------------------------------------------------
GLA_EPS = 1e-6          # the small positive constant of the feature map
GLA_ROPE_BASE = 10000.0  # RoPE frequency base


def rope(x: np.ndarray, pos: np.ndarray, base: float = GLA_ROPE_BASE) -> np.ndarray:
    """Rotary position embedding of rows x[r] at positions pos[r]: the pair of
    dimensions (2m, 2m+1) is rotated by the angle pos * base^(-2m/d)."""
    d = x.shape[-1]
    theta = base ** (-2.0 * np.arange(d // 2) / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * theta[None, :]
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x, dtype=np.float64)
    out[:, 0::2] = x[:, 0::2] * c - x[:, 1::2] * s
    out[:, 1::2] = x[:, 0::2] * s + x[:, 1::2] * c
    return out


def gla_features(x: np.ndarray, pos: np.ndarray) -> np.ndarray:
    """ReLU(RoPE(x)) + eps, the nonnegative GLA features."""
    return np.maximum(rope(x, pos), 0.0) + GLA_EPS


def gla_prior_rows(q: np.ndarray, k: np.ndarray, g: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """Causal GLA prior p_t(i) = s_t(i) / Z_t (eq. gla-score-appendix) with a
    per-key-channel decay: s_t(i) = sum_c q~_{t,c} k~_{i,c} exp(sum_{tau=i+1}^{t}
    g_{tau,c}) for i <= t, i.e. <D_t q~_t, D_i^{-1} k~_i> with the envelope D
    acting element-wise.  The log-decays g are used as given (the paper's
    decays have g <= 0; it clips the envelope in practice without saying
    where, so the definition itself carries no clip).  q, k, g: [T, d_k];
    returns [len(rows), max(rows)+1].
    """
    n = int(rows.max()) + 1
    fq = gla_features(q[rows], rows)
    fk = gla_features(k[:n], np.arange(n))
    G = np.cumsum(g[:n], axis=0)  # G_t = sum_{tau <= t} g_tau, the decays as given
    s = np.zeros((len(rows), n))
    step = max(1, (1 << 21) // (n * k.shape[1]))
    for a in range(0, len(rows), step):
        rr = rows[a:a + step]
        e = G[rr][:, None, :] - G[None, :, :]                     # [r, i, c]
        e = np.where(np.arange(n)[None, :, None] <= rr[:, None, None], e, -np.inf)
        s[a:a + step] = np.einsum("ric,ic,rc->ri", np.exp(e), fk, fq[a:a + step])
    return s / s.sum(axis=1, keepdims=True)


def fem_gla(q, k, v, g, beta, rows=None, block: int = 256) -> np.ndarray:
    """FEM read with the causal GLA prior: q, k, g: [B, H, T, d_k] (g the
    log-decays); v: [B, H, T, d_v]; beta: [H, d_v].  Float64 [B, H, R, d_v]."""
    q, k, v, g, beta = _as64(q), _as64(k), _as64(v), _as64(g), _as64(beta)
    B, H, T, _ = q.shape
    dv = v.shape[3]
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.empty((B, H, len(rows), dv))
    for b in range(B):
        for h in range(H):
            pos = 0
            for rb in _row_blocks(rows, block):
                n = int(rb.max()) + 1
                p = gla_prior_rows(q[b, h], k[b, h], g[b, h], rb)
                out[b, h, pos:pos + len(rb)] = free_energy_read(p, v[b, h, :n], beta[h])
                pos += len(rb)
    return out


def fem_gla_recurrent(q, k, v, g, beta) -> np.ndarray:
    """The GLA-prior read as a float64 recurrence over t (the streaming
    recurrences of the GLA appendix, with the constant value channel):
      S_t = diag(e^{g_t}) S_{t-1} + k~_t exp(beta v_t - c)^T,
      z_t = diag(e^{g_t}) z_{t-1} + k~_t,
      F_t = (log(q~_t^T S_t) - log(q~_t^T z_t) + c) / beta,
    one global per-channel shift c_j.  An independent cross-check of
    ``fem_gla`` on small T."""
    q, k, v, g, beta = _as64(q), _as64(k), _as64(v), _as64(g), _as64(beta)
    B, H, T, dk = q.shape
    dv = v.shape[3]
    out = np.empty((B, H, T, dv))
    pos = np.arange(T)
    for b in range(B):
        for h in range(H):
            x = v[b, h] * beta[h][None, :]
            c = x.max(axis=0)
            e = np.exp(x - c[None, :])
            fq = gla_features(q[b, h], pos)
            fk = gla_features(k[b, h], pos)
            a = np.exp(g[b, h])
            S = np.zeros((dk, dv))
            z = np.zeros(dk)
            for t in range(T):
                S = a[t][:, None] * S + np.outer(fk[t], e[t])
                z = a[t] * z + fk[t]
                out[b, h, t] = (np.log(fq[t] @ S) - np.log(fq[t] @ z) + c) / beta[h]
    return out


def fem_linear(q, k, v, beta, rows=None, block: int = 512) -> np.ndarray:
    """FEM read with the causal linear-attention prior (phi = elu + 1).

    Quadratic evaluation of the definition: the masked, row-normalised
    phi(Q) phi(K)^T, then the same free-energy read as the softmax case.
    q, k: [B, H, T, d_k]; v: [B, H, T, d_v]; beta: [H, d_v].
    """
    q, k, v, beta = _as64(q), _as64(k), _as64(v), _as64(beta)
    B, H, T, _ = q.shape
    dv = v.shape[3]
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.empty((B, H, len(rows), dv))
    for b in range(B):
        for h in range(H):
            pos = 0
            for rb in _row_blocks(rows, block):
                n = int(rb.max()) + 1
                p = linear_prior_rows(q[b, h], k[b, h], rb)
                out[b, h, pos:pos + len(rb)] = free_energy_read(p, v[b, h, :n], beta[h])
                pos += len(rb)
    return out


def fem_linear_recurrent(q, k, v, beta) -> np.ndarray:
    """The linear-prior read as a float64 recurrence over t.

    Streaming form of the linearisable prior (Appendix "Parameterizations of
    the Prior Selection", GLA prior with no decay; "Streaming compatibility":
    a constant channel appended to the values gives the normaliser):
      S_t = S_{t-1} + phi(k_t) exp(beta v_t - c)^T,   z_t = z_{t-1} + phi(k_t)
      F_t = (log(phi(q_t)^T S_t) - log(phi(q_t)^T z_t) + c) / beta
    with one global per-channel shift c_j = max_t beta_j v_{t,j}.  Used only as
    an independent cross-check of ``fem_linear`` on small T.
    """
    q, k, v, beta = _as64(q), _as64(k), _as64(v), _as64(beta)
    B, H, T, dk = q.shape
    dv = v.shape[3]
    out = np.empty((B, H, T, dv))
    for b in range(B):
        for h in range(H):
            x = v[b, h] * beta[h][None, :]
            c = x.max(axis=0)
            e = np.exp(x - c[None, :])
            fq = elu_plus_one(q[b, h])
            fk = elu_plus_one(k[b, h])
            S = np.zeros((dk, dv))
            z = np.zeros(dk)
            for t in range(T):
                S += np.outer(fk[t], e[t])
                z += fk[t]
                num = fq[t] @ S
                den = fq[t] @ z
                out[b, h, t] = (np.log(num) - np.log(den) + c) / beta[h]
    return out
