"""GPU parity of fem_softmax_fwd (HIP, through the C ABI) against the float64 oracle.

Tolerances (max abs error, written per test): 1e-4 for fp32 inputs and 2e-2
for bf16 inputs.  Every case prints its name, shape and seed before touching
the GPU.
"""

import sys
import time

import numpy as np
import pytest
import torch

import oracle
from paper_2602_07160_amd import inputs

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-2
TOL_F32 = 1e-4


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def run(fem, q, k, v, beta):
    dev = torch.device("cuda:0")
    out = fem.fem_softmax_fwd(q.to(dev), k.to(dev), v.to(dev), beta.to(dev))
    torch.cuda.synchronize()
    return out.cpu().double().numpy()


def ref(q, k, v, beta, rows=None):
    return oracle.fem_softmax(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                              beta.double().numpy(), rows=rows)


def check(got, want, tol, what):
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - want).max()
    say(f"{what}: max abs err {err:.3e} (tol {tol})")
    assert err <= tol, f"{what}: max abs err {err} > {tol}"
    return err


# --------------------------------------------------------------------------
# the five workloads (softmax ones): full oracle where it is cheap, sampled
# rows at full size otherwise
# --------------------------------------------------------------------------
def test_workload1_fp32_full(fem):
    say("workload 1: fp32 B1 H1 T128 d32, seed 43")
    q, k, v, b = inputs.make_inputs(1)
    got = run(fem, q, k, v, b)
    t0 = time.perf_counter()
    want = ref(q, k, v, b)
    say(f"w1: oracle {time.perf_counter() - t0:.2f} s")
    check(got, want, TOL_F32, "w1")


def test_workload2_bf16_full(fem):
    say("workload 2: bf16 B4 H8 T1024 d64, seed 44")
    q, k, v, b = inputs.make_inputs(2)
    got = run(fem, q, k, v, b)
    t0 = time.perf_counter()
    want = ref(q, k, v, b)
    say(f"w2: oracle {time.perf_counter() - t0:.2f} s")
    check(got, want, TOL_BF16, "w2")


def _sampled_rows(T, rng, extra=12):
    fixed = [0, 1, 2, 31, 32, 63, 64, 65, 127, 255, 256, 257, T // 2, T - 2, T - 1]
    rows = set(x for x in fixed if 0 <= x < T)
    rows |= set(int(x) for x in rng.integers(0, T, extra))
    return np.array(sorted(rows))


def full_compare(got, q, k, v, b, tol, what, fn=None):
    """Every head and row of ``got`` against the oracle, head by head (the
    oracle is plain float64 numpy); prints progress so the run never goes
    quiet for long."""
    fn = oracle.fem_softmax if fn is None else fn
    B, H = got.shape[:2]
    worst = 0.0
    t_oracle = 0.0
    for bb in range(B):
        for hh in range(H):
            t0 = time.perf_counter()
            want = fn(q[bb:bb + 1, hh:hh + 1].double().numpy(), k[bb:bb + 1, hh:hh + 1].double().numpy(),
                      v[bb:bb + 1, hh:hh + 1].double().numpy(), b[hh:hh + 1].double().numpy())[0, 0]
            t_oracle += time.perf_counter() - t0
            g = got[bb, hh]
            assert np.isfinite(g).all(), f"{what} b{bb} h{hh}: non-finite output"
            err = float(np.abs(g - want).max())
            worst = max(worst, err)
            assert err <= tol, f"{what} b{bb} h{hh}: max abs err {err} > {tol}"
        say(f"{what}: batch {bb} done, worst max abs err so far {worst:.3e}")
    say(f"{what}: all {B * H} heads, every row: max abs err {worst:.3e} (tol {tol}); "
        f"oracle {t_oracle:.1f} s")
    return worst


def test_workload3_full_size_every_row(fem):
    say("workload 3: bf16 B8 H16 T4096 d128, seed 45, every head and row")
    q, k, v, b = inputs.make_inputs(3)
    got = run(fem, q, k, v, b)
    full_compare(got, q, k, v, b, TOL_BF16, "w3")


def test_workload3_reduced_full(fem):
    say("workload 3 recipe, reduced: B1 H2 T600 d128 (ragged), full oracle")
    q, k, v, b = inputs.make_inputs(3, B=1, H=2, T=600)
    check(run(fem, q, k, v, b), ref(q, k, v, b), TOL_BF16, "w3-reduced")


def test_workload4_full_size_every_row(fem):
    say("workload 4: bf16 B1 H8 T16384 d64 offset/clip, seed 46, every head and row")
    q, k, v, b = inputs.make_inputs(4)
    got = run(fem, q, k, v, b)
    full_compare(got, q, k, v, b, TOL_BF16, "w4")


def test_workload4_reduced_full(fem):
    say("workload 4 recipe, reduced: B1 H8 T2048 d64, full oracle")
    q, k, v, b = inputs.make_inputs(4, T=2048)
    check(run(fem, q, k, v, b), ref(q, k, v, b), TOL_BF16, "w4-reduced")


# --------------------------------------------------------------------------
# shapes: every supported d, ragged T, T=1, tile boundaries, many heads
# --------------------------------------------------------------------------
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("T", [1, 2, 31, 63, 64, 65, 255, 256, 257, 700])
def test_bf16_shapes(fem, d, T):
    say(f"bf16 shape B2 H3 T{T} d{d}, seed {1000 + T + d}")
    q, k, v, b = inputs.draw(1000 + T + d, 2, 3, T, d, dtype="bf16")
    check(run(fem, q, k, v, b), ref(q, k, v, b), TOL_BF16, f"T{T} d{d}")


@pytest.mark.parametrize("d", [1, 7, 32, 100, 256])
@pytest.mark.parametrize("T", [1, 5, 300])
def test_fp32_shapes(fem, d, T):
    say(f"fp32 shape B2 H2 T{T} d{d}")
    q, k, v, b = inputs.draw(2000 + T + d, 2, 2, T, d, dtype="f32", beta_lo=0.25, beta_hi=4.0)
    check(run(fem, q, k, v, b), ref(q, k, v, b), TOL_F32, f"fp32 T{T} d{d}")


# --------------------------------------------------------------------------
# numerics: small and large beta, peaked scores, equal scores, underflow
# --------------------------------------------------------------------------
@pytest.mark.parametrize("beta", [1e-3, 0.1, 1.0, 16.0, 64.0])
def test_bf16_beta_extremes(fem, beta):
    say(f"bf16 constant beta {beta}: B1 H2 T512 d64")
    q, k, v, _ = inputs.draw(3000, 1, 2, 512, 64, dtype="bf16")
    b = torch.full((2, 64), beta, dtype=torch.float32)
    check(run(fem, q, k, v, b), ref(q, k, v, b), TOL_BF16, f"beta={beta}")


# --------------------------------------------------------------------------
# channel split: a channel whose beta is at or above 0.5 takes E rounded to
# bf16 without the lo product (|dF| <= 2^-8 / beta); each workgroup orders its
# head's channels so that the small-beta ones fill the first column blocks.
# One head per pattern: every number of lo blocks, block boundaries (32 and
# 33 small channels), interleaved and reversed orders, beta exactly 0.5.
# --------------------------------------------------------------------------
LO_BETA = 0.5
SPLIT_PATTERNS = ["interleaved", "exactly32", "exactly33", "one_last", "none", "all", "reversed"]


def split_beta(d, seed):
    """[H, d] beta, one pattern per head; small = log-U[0.05, 0.1] (where a
    missing lo product would show: 2^-8 / 0.05 = 0.078), large = log-U[0.5, 8]
    with one channel at exactly 0.5."""
    rng = np.random.default_rng(seed)
    out = []
    for pat in SPLIT_PATTERNS:
        small = np.zeros(d, bool)
        if pat == "interleaved":
            small[::2] = True
        elif pat in ("exactly32", "exactly33"):
            small[rng.choice(d, min(d, 32 if pat == "exactly32" else 33), replace=False)] = True
        elif pat == "one_last":
            small[-1] = True
        elif pat == "all":
            small[:] = True
        elif pat == "reversed":
            small[d // 3:] = True
        lo = np.exp(rng.uniform(np.log(0.05), np.log(0.1), d))
        hi = np.exp(rng.uniform(np.log(LO_BETA), np.log(8.0), d))
        big = np.flatnonzero(~small)
        if big.size:
            hi[big[0]] = LO_BETA
        out.append(np.where(small, lo, hi))
    return torch.from_numpy(np.array(out, dtype=np.float32))


@pytest.mark.parametrize("d", [64, 128])
def test_bf16_channel_split(fem, d):
    say(f"channel split patterns {SPLIT_PATTERNS}: B1 H{len(SPLIT_PATTERNS)} T333 d{d}, seed {3100 + d}")
    H = len(SPLIT_PATTERNS)
    q, k, v, _ = inputs.draw(3100 + d, 1, H, 333, d, dtype="bf16")
    b = split_beta(d, 3200 + d)
    got = run(fem, q, k, v, b)
    want = ref(q, k, v, b)
    check(got, want, TOL_BF16, f"split d{d}")
    err = np.abs(got - want).max(axis=(0, 2))        # [H, d]
    bn = b.double().numpy()
    small = bn < LO_BETA
    # small beta: the lo product is there (a rounded E alone would be off by
    # up to 2^-8 / beta, several times this)
    assert err[small].max() <= 1e-2, f"small-beta channel error {err[small].max()}"
    # beta >= 0.5: within the rounding bound of E plus the other rounding
    bound = 2.0 ** -8 / bn + 5e-3
    worst = (err - bound)[~small].max()
    say(f"split d{d}: worst small-beta err {err[small].max():.3e}, worst slack vs 2^-8/beta bound {worst:.3e}")
    assert worst <= 0, "a channel with beta >= 0.5 exceeds its rounding bound"


def test_bf16_channel_split_variants(fem):
    """The reordered columns with the encoder read, bf16 output, d_v < d_qk and
    the gated read."""
    say("channel split variants: encoder / bf16 out / d_qk128 d_v64 / gated, B1 H7 T200, seed 3300")
    H = len(SPLIT_PATTERNS)
    dev = torch.device("cuda:0")
    q, k, v, _ = inputs.draw(3300, 1, H, 200, 128, dtype="bf16")
    b = split_beta(128, 3301)
    qd, kd, vd, bd = q.to(dev), k.to(dev), v.to(dev), b.to(dev)
    enc = fem.fem_softmax_fwd_ex(qd, kd, vd, bd, causal=False)
    o16 = fem.fem_softmax_fwd_ex(qd, kd, vd, bd, out_dtype=torch.bfloat16)
    o32 = fem.fem_softmax_fwd(qd, kd, vd, bd)
    v64, b64 = v[..., :64].contiguous(), b[:, :64].contiguous()
    half = fem.fem_softmax_fwd_ex(qd, kd, v64.to(dev), b64.to(dev))
    torch.cuda.synchronize()
    check(enc.cpu().double().numpy(),
          oracle.fem_softmax_encoder(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                     b.double().numpy()), TOL_BF16, "split encoder")
    assert torch.equal(o16.cpu(), o32.cpu().to(torch.bfloat16)), "bf16 output != RNE(fp32 output)"
    check(half.cpu().double().numpy(), ref(q, k, v64, b64), TOL_BF16, "split d_qk128 d_v64")
    lam, g = inputs.draw_gates(3302, 1, H, 200, 128)
    og = fem.fem_softmax_gated_fwd(qd, kd, vd, bd, lam.to(dev), g.to(dev))
    torch.cuda.synchronize()
    want = oracle.fem_softmax_ltl(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                  b.double().numpy(), lam.double().numpy(), g.double().numpy())
    errg = (np.abs(og.cpu().double().numpy() - want) / np.maximum(1.0, g.double().numpy())).max()
    say(f"split gated: max scaled err {errg:.3e}")
    assert errg <= TOL_BF16


def test_bf16_peaked_scores(fem):
    say("bf16 peaked scores q = 8 k_t: B1 H2 T384 d64")
    q, k, v, b = inputs.draw(3001, 1, 2, 384, 64, dtype="bf16")
    q = (8.0 * k.float()).to(torch.bfloat16)
    check(run(fem, q, k, v, b), ref(q, k, v, b), TOL_BF16, "peaked")


def test_bf16_equal_scores_is_logcumsumexp(fem):
    say("bf16 Q = 0 (uniform prior) vs torch.logcumsumexp: B2 H2 T300 d64")
    q, k, v, b = inputs.draw(3002, 2, 2, 300, 64, dtype="bf16")
    q = torch.zeros_like(q)
    got = run(fem, q, k, v, b)
    x = v.double() * b.double()[None, :, None, :]
    want = (torch.logcumsumexp(x, dim=2) - torch.log(torch.arange(1, 301, dtype=torch.float64))[:, None]) \
        / b.double()[None, :, None, :]
    check(got, want.numpy(), TOL_BF16, "uniform prior")


def test_bf16_first_tile_underflow(fem):
    """In-support values 160 nats below a masked value in the same tile: the
    shared column shift leaves rows 0..31 with an underflowed accumulator,
    which the exact per-(t, j) path must repair."""
    say("bf16 forced underflow: B1 H1 T128 d64, v=-5 then +5 at key 32, beta=16")
    q, k, _, _ = inputs.draw(3003, 1, 1, 128, 64, dtype="bf16")
    v = torch.full((1, 1, 128, 64), -5.0)
    v[:, :, 32] = 5.0
    v[:, :, 40:] = torch.randn(1, 1, 88, 64, generator=torch.Generator().manual_seed(0))
    v = v.to(torch.bfloat16)
    b = torch.full((1, 64), 16.0)
    got = run(fem, q, k, v, b)
    check(got, ref(q, k, v, b), TOL_BF16, "underflow repair")
    np.testing.assert_allclose(got[0, 0, :32], -5.0, atol=TOL_BF16)


@pytest.mark.parametrize("d,T", [(128, 256), (64, 300), (32, 200)])
def test_bf16_whole_rows_underflow(fem, d, T):
    """Every channel of every row before the block's last key underflows
    against that key's value (-5 everywhere, +5 at the last key, beta 16):
    the exact path repairs whole rows, a batch of channels per pass over the
    keys, and must agree with the oracle on every element."""
    say(f"bf16 whole-row underflow: B1 H2 T{T} d{d}, v=-5 then +5 at the last key, beta=16")
    q, k, _, _ = inputs.draw(3007, 1, 2, T, d, dtype="bf16")
    v = torch.full((1, 2, T, d), -5.0)
    v[:, :, T - 1] = 5.0
    v[:, 1, :, 1::2] = torch.randn(1, T, d // 2, generator=torch.Generator().manual_seed(1))
    v = v.to(torch.bfloat16)
    b = torch.full((2, d), 16.0)
    got = run(fem, q, k, v, b)
    check(got, ref(q, k, v, b), TOL_BF16, "whole-row underflow repair")
    np.testing.assert_allclose(got[0, 0, : T - 1], -5.0, atol=TOL_BF16)


def test_bf16_scale_law(fem):
    """F(beta; 2v) = 2 F(2beta; v); doubling is exact in bf16."""
    say("bf16 scale law a=2: B1 H2 T400 d128")
    q, k, v, b = inputs.draw(3004, 1, 2, 400, 128, dtype="bf16", beta_lo=0.1, beta_hi=4.0)
    lhs = run(fem, q, k, (2 * v.float()).to(torch.bfloat16), b)
    rhs = 2 * run(fem, q, k, v, 2 * b)
    check(lhs, rhs, 2 * TOL_BF16, "scale law")


def test_bf16_causality(fem):
    """Keys and values after t = 300 must not enter rows t <= 300.  Exactly,
    the perturbed run's rows <= 300 match the oracle of the unperturbed
    inputs.  In rounding, they may move: the column shift is shared by the
    256 rows of a workgroup, so a larger later value re-scales the earlier
    terms (and can send an element to the exact path), which changes the
    result by rounding only -- far below any leak of probability mass."""
    say("bf16 causality: perturb keys/values after t=300, B1 H2 T640 d64, seed 3005/77")
    q, k, v, b = inputs.draw(3005, 1, 2, 640, 64, dtype="bf16")
    a = run(fem, q, k, v, b)
    gen = torch.Generator().manual_seed(77)
    k2, v2 = k.clone(), v.clone()
    k2[:, :, 301:] = (3 * torch.randn(k2[:, :, 301:].shape, generator=gen)).to(torch.bfloat16)
    v2[:, :, 301:] = (3 * torch.randn(v2[:, :, 301:].shape, generator=gen)).to(torch.bfloat16)
    b2 = run(fem, q, k2, v2, b)
    want = ref(q, k, v, b, rows=np.arange(301))
    check(b2[:, :, :301], want, TOL_BF16, "perturbed run, rows <= 300")
    err = np.abs(a[:, :, :301] - b2[:, :, :301]).max()
    say(f"causality: rows <= 300 changed by {err:.3e}")
    assert err <= 2e-3
    assert np.abs(a[:, :, 301:] - b2[:, :, 301:]).max() > 1e-1


def test_bf16_deterministic(fem):
    say("bf16 determinism: two runs bit-identical, B2 H4 T1000 d128")
    q, k, v, b = inputs.draw(3006, 2, 4, 1000, 128, dtype="bf16")
    a = run(fem, q, k, v, b)
    c = run(fem, q, k, v, b)
    assert np.array_equal(a, c)


def test_nondefault_stream(fem):
    say("bf16 on a non-default stream: B1 H2 T500 d64")
    q, k, v, b = inputs.draw(3007, 1, 2, 500, 64, dtype="bf16")
    dev = torch.device("cuda:0")
    qd, kd, vd, bd = q.to(dev), k.to(dev), v.to(dev), b.to(dev)
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s):
        out = fem.fem_softmax_fwd(qd, kd, vd, bd)
    s.synchronize()
    check(out.cpu().double().numpy(), ref(q, k, v, b), TOL_BF16, "stream")


def test_binding_rejects_bad_arguments(fem):
    say("binding argument errors")
    dev = torch.device("cuda:0")
    q = torch.zeros(1, 1, 8, 48, dtype=torch.bfloat16, device=dev)
    b = torch.ones(1, 48, device=dev)
    with pytest.raises(fem.FemError) as e:
        fem.fem_softmax_fwd(q, q, q, b)
    assert e.value.status == 3
    q = torch.zeros(1, 1, 8, 64, dtype=torch.bfloat16, device=dev)
    with pytest.raises(ValueError):
        fem.fem_softmax_fwd(q, q, q, torch.ones(2, 64, device=dev))
    with pytest.raises(ValueError):
        fem.fem_softmax_fwd(q, q.transpose(2, 3).contiguous().transpose(2, 3), q,
                            torch.ones(1, 64, device=dev))
