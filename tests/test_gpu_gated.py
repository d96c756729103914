"""GPU parity of fem_softmax_gated_fwd (two-level gated read, HIP through the
C ABI) against the float64 oracle's fem_softmax_ltl.

Tolerance: the bf16 budget 2e-2 applies to the inner read
F~ = (1 - lam) mu + lam F(beta_max); the outer gate multiplies it, so the
check on o = g F~ is |o - o_ref| <= 2e-2 * max(1, g) element-wise.  Every
case prints its name, shape and seed before touching the GPU.
"""

import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2602_07160_amd import inputs

pytestmark = pytest.mark.gpu

TOL = 2e-2


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def run(fem, q, k, v, bmax, lam, gate):
    dev = torch.device("cuda:0")
    out = fem.fem_softmax_gated_fwd(q.to(dev), k.to(dev), v.to(dev), bmax.to(dev), lam.to(dev),
                                    None if gate is None else gate.to(dev))
    torch.cuda.synchronize()
    return out.cpu().double().numpy()


def ref(q, k, v, bmax, lam, gate, rows=None):
    n = lambda x: None if x is None else x.double().numpy()
    return oracle.fem_softmax_ltl(n(q), n(k), n(v), n(bmax), n(lam), n(gate), rows=rows)


def check(got, want, gate, what):
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    scale = 1.0 if gate is None else np.maximum(1.0, gate)
    err = (np.abs(got - want) / scale).max()
    say(f"{what}: max scaled err {err:.3e} (tol {TOL})")
    assert err <= TOL, f"{what}: max scaled err {err} > {TOL}"


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("T", [1, 63, 64, 65, 257, 700])
def test_gated_shapes(fem, d, T):
    say(f"gated bf16 B2 H3 T{T} d{d}, seeds {4000 + T + d}/{5000 + T + d}")
    q, k, v, b = inputs.draw(4000 + T + d, 2, 3, T, d, dtype="bf16")
    lam, g = inputs.draw_gates(5000 + T + d, 2, 3, T, d)
    check(run(fem, q, k, v, b, lam, g), ref(q, k, v, b, lam, g), g, f"T{T} d{d}")


@pytest.mark.parametrize("d", [64, 128])
def test_gated_no_outer_gate(fem, d):
    say(f"gated bf16 gate=NULL B1 H4 T500 d{d}")
    q, k, v, b = inputs.draw(4100 + d, 1, 4, 500, d, dtype="bf16")
    lam, _ = inputs.draw_gates(5100 + d, 1, 4, 500, d)
    check(run(fem, q, k, v, b, lam, None), ref(q, k, v, b, lam, None), None, f"no gate d{d}")


def test_gated_lambda_endpoints(fem):
    """lam = 0 is the expectation alone (torch SDPA in float64); lam = 1 with
    no outer gate is fem_softmax_fwd at beta_max."""
    say("gated lam=0 / lam=1: B2 H2 T400 d128")
    q, k, v, b = inputs.draw(4200, 2, 2, 400, 128, dtype="bf16")
    z, one = torch.zeros(2, 2, 400, 128), torch.ones(2, 2, 400, 128)
    mu = torch.nn.functional.scaled_dot_product_attention(q.double(), k.double(), v.double(),
                                                          is_causal=True).numpy()
    check(run(fem, q, k, v, b, z, None), mu, None, "lam=0 vs SDPA")
    dev = torch.device("cuda:0")
    f = fem.fem_softmax_fwd(q.to(dev), k.to(dev), v.to(dev), b.to(dev))
    torch.cuda.synchronize()
    got = run(fem, q, k, v, b, one, None)
    err = np.abs(got - f.cpu().double().numpy()).max()
    say(f"lam=1 vs fem_softmax_fwd: max abs diff {err:.3e}")
    assert err <= 1e-5


def test_gated_full_size_sampled(fem):
    say("gated workload 3 shape: bf16 B8 H16 T4096 d128, seed 45 (+ gates seed 145), sampled rows")
    q, k, v, b = inputs.make_inputs(3)
    lam, g = inputs.draw_gates(145, 8, 16, 4096, 128)
    got = run(fem, q, k, v, b, lam, g)
    rng = np.random.default_rng(2)
    rows = np.array(sorted(set([0, 1, 63, 64, 255, 256, 2047, 4094, 4095]) |
                           set(int(x) for x in rng.integers(0, 4096, 10))))
    for bb, hh in [(0, 0), (6, 11)]:
        sl = lambda x: x[bb:bb + 1, hh:hh + 1]
        want = ref(sl(q), sl(k), sl(v), b[hh:hh + 1], sl(lam), sl(g), rows=rows)[0, 0]
        check(got[bb, hh, rows], want, g[bb, hh, rows].numpy(), f"w3 gated b{bb} h{hh}")


def test_gated_underflow_repair(fem):
    """The forced-underflow case of the plain read: rows 0..31 take the exact
    path, which must combine its F with mu, lam and g like the fast path."""
    say("gated forced underflow: B1 H1 T128 d64, beta_max=16")
    q, k, _, _ = inputs.draw(3003, 1, 1, 128, 64, dtype="bf16")
    v = torch.full((1, 1, 128, 64), -5.0)
    v[:, :, 32] = 5.0
    v[:, :, 40:] = torch.randn(1, 1, 88, 64, generator=torch.Generator().manual_seed(0))
    v = v.to(torch.bfloat16)
    b = torch.full((1, 64), 16.0)
    lam, g = inputs.draw_gates(4300, 1, 1, 128, 64)
    got = run(fem, q, k, v, b, lam, g)
    check(got, ref(q, k, v, b, lam, g), g.numpy(), "gated underflow repair")
    np.testing.assert_allclose(got[0, 0, :32], -5.0 * g[0, 0, :32].numpy(), atol=TOL)


def test_gated_deterministic_and_stream(fem):
    say("gated determinism + non-default stream: B1 H2 T900 d128")
    q, k, v, b = inputs.draw(4400, 1, 2, 900, 128, dtype="bf16")
    lam, g = inputs.draw_gates(4401, 1, 2, 900, 128)
    a = run(fem, q, k, v, b, lam, g)
    dev = torch.device("cuda:0")
    args = [x.to(dev) for x in (q, k, v, b, lam, g)]
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s):
        out = fem.fem_softmax_gated_fwd(*args)
    s.synchronize()
    assert np.array_equal(a, out.cpu().double().numpy())


def test_gated_binding_rejects_bad_arguments(fem):
    say("gated binding argument errors")
    dev = torch.device("cuda:0")
    q = torch.zeros(1, 1, 8, 64, dtype=torch.bfloat16, device=dev)
    b = torch.ones(1, 64, device=dev)
    lam = torch.zeros(1, 1, 8, 64, device=dev)
    with pytest.raises(ValueError):
        fem.fem_softmax_gated_fwd(q, q, q, b, lam[..., :32])
    with pytest.raises(ValueError):
        fem.fem_softmax_gated_fwd(q.float(), q.float(), q.float(), b, lam)
    q48 = torch.zeros(1, 1, 8, 48, dtype=torch.bfloat16, device=dev)
    with pytest.raises(fem.FemError) as e:
        fem.fem_softmax_gated_fwd(q48, q48, q48, torch.ones(1, 48, device=dev),
                                  torch.zeros(1, 1, 8, 48, device=dev))
    assert e.value.status == 3
