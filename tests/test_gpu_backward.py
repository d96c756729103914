"""GPU parity of the training pair fem_softmax_fwd_train / fem_softmax_bwd
(HIP, through the C ABI) against the float64 oracle's gradients.

Tolerances (written per check): lse within 1e-2 absolute (the forward sums
bf16-rounded probabilities, a relative 2^-9 per term); dQ, dK, dV element by
element within 2^-6 of the element's cancellation-free term magnitude M
(grad_scales: the sum of the absolute values of the terms the closed forms
add up; the posterior uses the forward's F, whose bf16 rounding moves beta F
by at most 2^-8, and dS enters the dQ / dK products in bf16, 2^-9; the
factor 4 covers their accumulation).  dbeta is the difference
(sum_i v dV - sum_t G F) / beta of two terms of size sum |G v| / beta, whose
products the matrix-core path forms from bf16 hi + lo parts (2^-16
relative each); its floor adds 2^-14 sum_{b,t} |G v| / beta per (h, j), which
matters only where dbeta itself is near zero (a single key: exactly zero).
Every case prints its name, shape and seed before touching the GPU.
"""

import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2602_07160_amd import inputs

pytestmark = pytest.mark.gpu

TOL = 2e-2
ATOL = 1e-4


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def run(fem, q, k, v, b, g):
    """Forward (training) and backward through the C ABI; returns numpy."""
    dev = torch.device("cuda:0")
    qd, kd, vd, bd, gd = (x.to(dev) for x in (q, k, v, b, g))
    out, lse = fem.fem_softmax_fwd_train(qd, kd, vd, bd)
    grads = fem.fem_softmax_bwd(qd, kd, vd, bd, out, lse, gd)
    torch.cuda.synchronize()
    return out.cpu().double().numpy(), lse.cpu().double().numpy(), \
        [x.cpu().double().numpy() for x in grads]


def lse_ref(q, k):
    qq, kk = q.double(), k.double()
    T, d = q.shape[2], q.shape[3]
    s = qq @ kk.transpose(-1, -2) / math.sqrt(d)
    s = s.masked_fill(torch.triu(torch.ones(T, T, dtype=torch.bool), 1), float("-inf"))
    return torch.logsumexp(s, dim=-1).numpy()


def dbeta_floor(v, b, g):
    """2^-14 sum_{b,t} |G v| / beta per (h, j): the rounding scale of dbeta."""
    gv = (np.abs(g.double().numpy()) * np.abs(v.double().numpy())).sum(axis=(0, 2))
    return 2.0 ** -14 * gv / b.double().numpy()


def grad_scales(q, k, v, b, g, jc=8):
    """Cancellation-free magnitudes of the gradients' terms, in float64 from
    the definitions: with the prior p_t(i), the posterior q_tj(i) and
    D_ti = sum_j |G_tj| / beta_j (q_tj(i) + p_t(i)) (a bound on |dS_ti|),
      M_V[i,j] = sum_t |G_tj| q_tj(i),
      M_Q[t,c] = sum_i D_ti |k_ic| / sqrt(d),   M_K[i,c] = sum_t D_ti |q_tc| / sqrt(d).
    Channels are taken jc at a time (the posterior is T x T per channel)."""
    qq, kk, vv = q.double(), k.double(), v.double()
    bb, gg = b.double(), g.double()
    B, H, T, d = qq.shape
    mask = torch.triu(torch.ones(T, T, dtype=torch.bool), 1)
    s = (qq @ kk.transpose(-1, -2) / math.sqrt(d)).masked_fill(mask, float("-inf"))
    logp = torch.log_softmax(s, dim=-1)                      # [B,H,T,T]
    p = logp.exp()
    MV = torch.zeros(B, H, T, d, dtype=torch.float64)
    D = p * (gg.abs() / bb[None, :, None, :]).sum(-1, keepdim=True)  # the p part of D
    for j0 in range(0, d, jc):
        x = logp[..., None] + (bb[None, :, None, None, j0:j0 + jc] * vv[:, :, None, :, j0:j0 + jc])
        post = torch.softmax(x, dim=3)                       # [B,H,t,i,jc]
        ga = gg[..., j0:j0 + jc].abs()                        # [B,H,t,jc]
        MV[..., j0:j0 + jc] = (post * ga[:, :, :, None, :]).sum(2)
        D += (post * (ga / bb[None, :, None, j0:j0 + jc])[:, :, :, None, :]).sum(-1)
    MQ = D @ kk.abs() / math.sqrt(d)
    MK = D.transpose(-1, -2) @ qq.abs() / math.sqrt(d)
    return MQ.numpy(), MK.numpy(), MV.numpy()


RTOL_M = 2.0 ** -6


def check_grads(got, want, what, floor_db, scales):
    """dQ, dK, dV element by element: |g - g_ref| <= 2^-6 M, M the element's
    cancellation-free term magnitude (grad_scales).  The largest single
    relative rounding in the terms is 2^-8 (the forward's bf16-rounded F
    enters the posterior; dS enters the dQ / dK products as bf16, 2^-9);
    2^-6 leaves a factor 4 for their accumulation (observed worst 3.8e-3).
    dbeta: 2e-2 of its scale plus the floor of dbeta_floor."""
    for n, (name, a, b) in enumerate(zip(("dq", "dk", "dv", "dbeta"), got, want)):
        assert np.isfinite(a).all(), f"{what} {name}: non-finite"
        err = np.abs(a - b)
        if name != "dbeta":
            m = scales[n]
            tol = RTOL_M * m + 1e-7 * m.max()
            big = m > 1e-7 * m.max()  # elements above the absolute floor
            ratio = float(np.max(err[big] / m[big])) if big.any() else 0.0
            say(f"{what} {name}: max err {err.max():.3e}, max err / M {ratio:.3e}"
                f" (tol {RTOL_M:.4f} M + 1e-7 max M)")
            assert (err <= tol).all(), f"{what} {name}: max err / M {np.max(err / (m + 1e-300))}"
        else:
            scale = np.abs(b).max()
            tol = TOL * scale + ATOL + floor_db
            say(f"{what} dbeta: max err {err.max():.3e}, scale {scale:.3e}")
            assert (err <= tol).all(), f"{what} dbeta: {err.max()} > {TOL} * {scale} + floor"


def draw(seed, B, H, T, d, **kw):
    q, k, v, b = inputs.draw(seed, B, H, T, d, dtype="bf16", **kw)
    g = torch.from_numpy(np.random.default_rng(seed + 1).standard_normal((B, H, T, d)).astype(np.float32))
    return q, k, v, b, g


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("T", [1, 33, 64, 65, 200])
def test_backward_shapes(fem, d, T):
    seed = 13000 + T + d
    say(f"backward B2 H2 T{T} d{d}, seed {seed}")
    q, k, v, b, g = draw(seed, 2, 2, T, d)
    out, lse, grads = run(fem, q, k, v, b, g)
    err = np.abs(lse - lse_ref(q, k)).max()
    say(f"lse: max err {err:.3e} (tol 1e-2)")
    assert err <= 1e-2
    want = oracle.fem_softmax_grads(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                    b.double().numpy(), g.double().numpy())
    check_grads(grads, want, f"T{T} d{d}", dbeta_floor(v, b, g), grad_scales(q, k, v, b, g))


def test_backward_forward_output_unchanged(fem):
    say("fem_softmax_fwd_train out == fem_softmax_fwd out: B1 H2 T300 d128, seed 13100")
    q, k, v, b, g = draw(13100, 1, 2, 300, 128)
    dev = torch.device("cuda:0")
    a = fem.fem_softmax_fwd(q.to(dev), k.to(dev), v.to(dev), b.to(dev))
    out, _, _ = run(fem, q, k, v, b, g)
    assert np.array_equal(a.cpu().double().numpy(), out)


@pytest.mark.parametrize("beta", [0.01, 1.0, 16.0])
def test_backward_beta_extremes(fem, beta):
    say(f"backward constant beta {beta}: B1 H2 T256 d64, seed 13200")
    q, k, v, _, g = draw(13200, 1, 2, 256, 64)
    b = torch.full((2, 64), beta)
    _, _, grads = run(fem, q, k, v, b, g)
    want = oracle.fem_softmax_grads(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                    b.double().numpy(), g.double().numpy())
    check_grads(grads, want, f"beta={beta}", dbeta_floor(v, b, g), grad_scales(q, k, v, b, g))


def test_backward_longer_sequence(fem):
    say("backward B1 H2 T1024 d128 (workload-3 recipe), seed 13300")
    q, k, v, b, g = draw(13300, 1, 2, 1024, 128)
    _, _, grads = run(fem, q, k, v, b, g)
    want = oracle.fem_softmax_grads(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                    b.double().numpy(), g.double().numpy())
    check_grads(grads, want, "T1024 d128", dbeta_floor(v, b, g), grad_scales(q, k, v, b, g))


@pytest.mark.parametrize("d,T", [(32, 700), (64, 1000)])
def test_backward_longer_small_d(fem, d, T):
    """Many tile pairs (pipelined passes, unmasked off-diagonal pairs, a
    ragged last tile) for the narrower head widths."""
    seed = 13600 + d
    say(f"backward B1 H2 T{T} d{d}, seed {seed}")
    q, k, v, b, g = draw(seed, 1, 2, T, d)
    _, _, grads = run(fem, q, k, v, b, g)
    want = oracle.fem_softmax_grads(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                    b.double().numpy(), g.double().numpy())
    check_grads(grads, want, f"T{T} d{d}", dbeta_floor(v, b, g), grad_scales(q, k, v, b, g))


def test_backward_deterministic(fem):
    say("backward determinism: B2 H2 T500 d64, seed 13400")
    q, k, v, b, g = draw(13400, 2, 2, 500, 64)
    a = run(fem, q, k, v, b, g)[2]
    c = run(fem, q, k, v, b, g)[2]
    for x, y in zip(a, c):
        assert np.array_equal(x, y)


def test_backward_exact_fallback(fem):
    """Values spread over [-5, 5] with beta = 16 give every channel a
    beta-scaled range (16 log2(e) 10 = 231) beyond the matrix-core form's
    fp32 bound, so the element-wise kernels take every channel."""
    say("backward fallback case: B1 H2 T300 d64, v in {-5, +5, N(0,1)}, beta 16, seed 13500")
    q, k, _, _, g = draw(13500, 1, 2, 300, 64)
    rng = np.random.default_rng(13501)
    v = rng.standard_normal((1, 2, 300, 64))
    v[:, :, ::7] = 5.0
    v[:, :, 3::11] = -5.0
    v = torch.from_numpy(v.astype(np.float32)).to(torch.bfloat16)
    b = torch.full((2, 64), 16.0)
    _, _, grads = run(fem, q, k, v, b, g)
    want = oracle.fem_softmax_grads(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                    b.double().numpy(), g.double().numpy())
    check_grads(grads, want, "fallback", dbeta_floor(v, b, g), grad_scales(q, k, v, b, g))


@pytest.mark.parametrize("d", [32, 64, 128])
def test_backward_some_wide_channels(fem, d):
    """A few channels per head get beta = 16 and values spread over [-5, 5]
    (range 231 in log2 units): the element-wise kernels take those channels
    only and add their part to the matrix-core dQ and dK; the other channels
    (beta log-uniform in [0.1, 8]) stay on the matrix cores."""
    seed = 13700 + d
    say(f"backward mixed wide channels: B2 H2 T333 d{d}, seed {seed}")
    q, k, v, b, g = draw(seed, 2, 2, 333, d)
    wide = {0: [3, 17], 1: [d - 1]}
    v = v.float().numpy().copy()
    b = b.clone()
    for h, chans in wide.items():
        for j in chans:
            v[:, h, ::7, j] = 5.0
            v[:, h, 3::11, j] = -5.0
            b[h, j] = 16.0
    v = torch.from_numpy(v).to(torch.bfloat16)
    _, _, grads = run(fem, q, k, v, b, g)
    want = oracle.fem_softmax_grads(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                    b.double().numpy(), g.double().numpy())
    check_grads(grads, want, f"mixed d{d}", dbeta_floor(v, b, g), grad_scales(q, k, v, b, g))
    # the wide channels' dV columns, against their own scale and element by
    # element against their term magnitude M_V
    mv = grad_scales(q, k, v, b, g)[2]
    for h, chans in wide.items():
        for j in chans:
            err = np.abs(grads[2][:, h, :, j] - want[2][:, h, :, j])
            scale = np.abs(want[2][:, h, :, j]).max()
            m = mv[:, h, :, j]
            big = m > 1e-7 * m.max()
            ratio = float((err[big] / m[big]).max())
            say(f"wide channel h{h} j{j} dv: max err {err.max():.3e}, scale {scale:.3e}, "
                f"max err / M {ratio:.3e}")
            assert err.max() <= TOL * scale + ATOL
            # the element-wise pass normalises its posterior (the forward's
            # rounded F would leave ~beta |F - F^| ~ 3e-4 of M here)
            assert ratio <= 2.0 ** -14, f"wide channel h{h} j{j}: dV err / M {ratio}"


def test_backward_guard_fallback(fem):
    """Output gradients of size 2^98 push W U = (G / beta) 2^{c - bl F} past
    2^124 (the matrix-core form's fp32 guard) on early rows, so the whole call
    is redone by the element-wise kernels; every gradient stays inside fp32."""
    say("backward guard fallback: B1 H2 T200 d64, beta 8, G * 2^98, seed 13800")
    q, k, v, _, g = draw(13800, 1, 2, 200, 64)
    b = torch.full((2, 64), 8.0)
    g = g * 2.0 ** 98
    _, _, grads = run(fem, q, k, v, b, g)
    want = oracle.fem_softmax_grads(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                    b.double().numpy(), g.double().numpy())
    check_grads(grads, want, "guard fallback", dbeta_floor(v, b, g), grad_scales(q, k, v, b, g))


def test_backward_wide_deterministic(fem):
    """The element-wise kernels that add the wide channels' part write with
    plain stores in a fixed order: two calls give the same bits."""
    say("backward wide-channel determinism: B1 H2 T257 d64, seed 13900")
    q, k, v, b, g = draw(13900, 1, 2, 257, 64)
    v = v.float().numpy().copy()
    v[:, 1, ::5, 9] = 5.0
    v[:, 1, 2::9, 9] = -5.0
    v = torch.from_numpy(v).to(torch.bfloat16)
    b = b.clone()
    b[1, 9] = 16.0
    a = run(fem, q, k, v, b, g)[2]
    c = run(fem, q, k, v, b, g)[2]
    for x, y in zip(a, c):
        assert np.array_equal(x, y)


def test_backward_wide_in_one_batch(fem):
    """beta = 16 on one channel of head 1; in batch 0 its values spread over
    [-5, 5] (wide), in batch 1 they are scaled to a range of ~2 (beta-scaled
    ~45, matrix cores), so dbeta of that channel adds the element-wise pass's
    partial sums of batch 0 to the matrix-core sums of batch 1."""
    say("backward wide in one batch: B2 H2 T300 d64, seed 14000")
    q, k, v, b, g = draw(14000, 2, 2, 300, 64)
    v = v.float().numpy().copy()
    v[0, 1, ::6, 20] = 5.0
    v[0, 1, 1::10, 20] = -5.0
    v[1, 1, :, 20] *= 0.3
    v = torch.from_numpy(v).to(torch.bfloat16)
    b = b.clone()
    b[1, 20] = 16.0
    _, _, grads = run(fem, q, k, v, b, g)
    want = oracle.fem_softmax_grads(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                    b.double().numpy(), g.double().numpy())
    check_grads(grads, want, "wide in batch 0 only", dbeta_floor(v, b, g), grad_scales(q, k, v, b, g))
    err = abs(grads[3][1, 20] - want[3][1, 20])
    say(f"dbeta[1, 20]: {grads[3][1, 20]:.6e} vs {want[3][1, 20]:.6e} (err {err:.3e})")
    assert err <= TOL * abs(want[3][1, 20]) + dbeta_floor(v, b, g)[1, 20] + ATOL
