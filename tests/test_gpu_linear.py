"""GPU parity of fem_linear_fwd (HIP chunked scan, through the C ABI) against
the float64 oracle.  Tolerance: max abs error <= 2e-2 (bf16 inputs)."""

import sys
import time

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


def run(fem, q, k, v, beta, chunk=64):
    dev = torch.device("cuda:0")
    out = fem.fem_linear_fwd(q.to(dev), k.to(dev), v.to(dev), beta.to(dev), chunk=chunk)
    torch.cuda.synchronize()
    return out.cpu().double().numpy()


def ref(q, k, v, beta, rows=None):
    return oracle.fem_linear(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                             beta.double().numpy(), rows=rows)


def check(got, want, tol, what):
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - want).max()
    say(f"{what}: max abs err {err:.3e} (tol {tol})")
    assert err <= tol, f"{what}: max abs err {err} > {tol}"


def test_workload5_full_size_every_row(fem):
    say("workload 5: linear bf16 B4 H16 T8192 d64 chunk 64, seed 47, every head and row")
    q, k, v, b = inputs.make_inputs(5)
    got = run(fem, q, k, v, b)
    worst = 0.0
    t_oracle = 0.0
    for bb in range(4):
        for hh in range(16):
            t0 = time.perf_counter()
            want = oracle.fem_linear(q[bb:bb + 1, hh:hh + 1].double().numpy(),
                                     k[bb:bb + 1, hh:hh + 1].double().numpy(),
                                     v[bb:bb + 1, hh:hh + 1].double().numpy(),
                                     b[hh:hh + 1].double().numpy())[0, 0]
            t_oracle += time.perf_counter() - t0
            assert np.isfinite(got[bb, hh]).all()
            err = float(np.abs(got[bb, hh] - want).max())
            worst = max(worst, err)
            assert err <= TOL, f"workload 5 b{bb} h{hh}: {err} > {TOL}"
        say(f"workload 5: batch {bb} done, worst max abs err so far {worst:.3e}")
    say(f"workload 5: all 64 heads, every row: max abs err {worst:.3e} (tol {TOL}); "
        f"oracle {t_oracle:.1f} s")


def test_workload5_reduced_full(fem):
    say("workload 5 recipe, reduced: B1 H3 T1300 (3 segments, ragged), full oracle")
    q, k, v, b = inputs.make_inputs(5, B=1, H=3, T=1300)
    check(run(fem, q, k, v, b), ref(q, k, v, b), TOL, "w5-reduced")


@pytest.mark.parametrize("T", [1, 2, 63, 64, 65, 511, 512, 513, 1025])
def test_linear_shapes(fem, T):
    say(f"linear shape B2 H2 T{T} d64")
    q, k, v, b = inputs.draw(4000 + T, 2, 2, T, 64, dtype="bf16", beta_lo=0.1, beta_hi=4.0)
    check(run(fem, q, k, v, b), ref(q, k, v, b), TOL, f"linear T{T}")


@pytest.mark.parametrize("beta", [1e-2, 0.1, 1.0, 16.0])
def test_linear_beta_extremes(fem, beta):
    say(f"linear constant beta {beta}: B1 H2 T700")
    q, k, v, _ = inputs.draw(4100, 1, 2, 700, 64, dtype="bf16")
    b = torch.full((2, 64), beta, dtype=torch.float32)
    check(run(fem, q, k, v, b), ref(q, k, v, b), TOL, f"linear beta={beta}")


def test_linear_equal_keys_is_logcumsumexp(fem):
    say("linear all keys equal (uniform prior) vs torch.logcumsumexp: B1 H2 T600")
    q, k, v, b = inputs.draw(4200, 1, 2, 600, 64, dtype="bf16")
    k = k[:, :, :1].expand(-1, -1, 600, -1).contiguous()
    got = run(fem, q, k, v, b)
    x = v.double() * b.double()[None, :, None, :]
    want = (torch.logcumsumexp(x, dim=2) - torch.log(torch.arange(1, 601, dtype=torch.float64))[:, None]) \
        / b.double()[None, :, None, :]
    check(got, want.numpy(), TOL, "linear uniform prior")


def test_linear_underflow_repair(fem):
    say("linear forced underflow: v=-5 then +5 at key 20 in the same chunk, beta=16, T200")
    q, k, _, _ = inputs.draw(4300, 1, 1, 200, 64, dtype="bf16")
    v = torch.full((1, 1, 200, 64), -5.0)
    v[:, :, 20] = 5.0
    v[:, :, 30:] = torch.randn(1, 1, 170, 64, generator=torch.Generator().manual_seed(1))
    v = v.to(torch.bfloat16)
    b = torch.full((1, 64), 16.0)
    got = run(fem, q, k, v, b)
    check(got, ref(q, k, v, b), TOL, "linear underflow repair")


def test_linear_segment_end_spike(fem):
    """Values far above the rest of their segment at its last key: the read
    of a segment shifts by the segment's own maximum, so every earlier row of
    those channels underflows and is recomputed exactly; rows of other
    channels and heads are unaffected."""
    say("linear spikes at segment ends: B2 H64 T1024 (4 segments of 256), beta=16 on 4 channels")
    q, k, v, b = inputs.draw(4350, 2, 64, 1024, 64, dtype="bf16", beta_lo=0.1, beta_hi=4.0)
    v = v.float()
    v[0, 0, :, :4] = -5.0
    v[0, 0, 255, :4] = 5.0
    v[0, 0, 767, :4] = 5.0
    v = v.to(torch.bfloat16)
    b[0, :4] = 16.0
    got = run(fem, q, k, v, b)
    for bb, hh in [(0, 0), (0, 1), (1, 0), (1, 63)]:
        want = ref(q[bb:bb + 1, hh:hh + 1], k[bb:bb + 1, hh:hh + 1], v[bb:bb + 1, hh:hh + 1],
                   b[hh:hh + 1])
        check(got[bb:bb + 1, hh:hh + 1], want, TOL, f"segment-end spikes (b={bb}, h={hh})")


def test_linear_one_segment_per_head(fem):
    """With B*H large enough that every head is one segment, the scan runs
    without segment states and raises its shift lazily chunk by chunk; a
    sample of heads is compared with the oracle over every row."""
    say("linear one segment per head: B4 H128 T700 d64 (no state pass), 4 heads checked")
    q, k, v, b = inputs.draw(4360, 4, 128, 700, 64, dtype="bf16", beta_lo=0.1, beta_hi=8.0)
    got = run(fem, q, k, v, b)
    for bb, hh in [(0, 0), (1, 37), (2, 90), (3, 127)]:
        want = ref(q[bb:bb + 1, hh:hh + 1], k[bb:bb + 1, hh:hh + 1], v[bb:bb + 1, hh:hh + 1],
                   b[hh:hh + 1])
        check(got[bb:bb + 1, hh:hh + 1], want, TOL, f"one segment per head (b={bb}, h={hh})")


def test_linear_deterministic(fem):
    say("linear determinism: B2 H2 T1500")
    q, k, v, b = inputs.draw(4400, 2, 2, 1500, 64, dtype="bf16")
    assert np.array_equal(run(fem, q, k, v, b), run(fem, q, k, v, b))


def test_linear_rejects_unsupported(fem):
    say("linear argument errors")
    dev = torch.device("cuda:0")
    q = torch.zeros(1, 1, 8, 64, dtype=torch.bfloat16, device=dev)
    b = torch.ones(1, 64, device=dev)
    for c in (8, 48, 256):
        with pytest.raises(fem.FemError) as e:
            fem.fem_linear_fwd(q, q, q, b, chunk=c)
        assert e.value.status == 3
    q32 = torch.zeros(1, 1, 8, 32, dtype=torch.bfloat16, device=dev)
    with pytest.raises(fem.FemError):
        fem.fem_linear_fwd(q32, q32, q32, torch.ones(1, 32, device=dev))


CHUNKS = (16, 32, 64, 128)


@pytest.mark.parametrize("chunk", CHUNKS)
@pytest.mark.parametrize("T", [1, 15, 16, 17, 31, 33, 64, 127, 129, 300, 1000])
def test_linear_chunks_small(fem, chunk, T):
    seed = 5100 + T + chunk
    say(f"linear chunk {chunk}: B2 H3 T{T} d64, seed {seed}")
    q, k, v, b = inputs.draw(seed, 2, 3, T, 64, dtype="bf16", beta_lo=0.1, beta_hi=4.0)
    check(run(fem, q, k, v, b, chunk=chunk), ref(q, k, v, b), TOL, f"linear chunk {chunk} T{T}")


def test_linear_chunk_invariance(fem):
    """The chunk only schedules the scan (the result is chunk-independent in
    exact arithmetic): every chunk length matches the oracle, and the four
    schedules agree with each other to the same budget, on a case with many
    segments, a ragged tail and both small and large beta."""
    say("linear chunk invariance: B2 H4 T3001 d64, chunks 16/32/64/128, seed 5201")
    q, k, v, b = inputs.draw(5201, 2, 4, 3001, 64, dtype="bf16", beta_lo=0.05, beta_hi=8.0)
    want = ref(q, k, v, b)
    got = {c: run(fem, q, k, v, b, chunk=c) for c in CHUNKS}
    for c in CHUNKS:
        check(got[c], want, TOL, f"chunk {c} vs oracle")
    for c in CHUNKS[1:]:
        d = np.abs(got[c] - got[CHUNKS[0]]).max()
        say(f"chunk {c} vs chunk {CHUNKS[0]}: max abs diff {d:.3e}")
        assert d <= TOL
    # the schedules differ: chunk 16 routes half of each tile's keys through
    # the state, chunk 128 through the masked product
    assert not np.array_equal(got[16], got[128])


@pytest.mark.parametrize("chunk", (16, 32, 128))
def test_workload5_other_chunks_sampled(fem, chunk):
    say(f"workload 5 at chunk {chunk}: B4 H16 T8192 d64, sampled rows")
    q, k, v, b = inputs.make_inputs(5)
    got = run(fem, q, k, v, b, chunk=chunk)
    rows = np.array([0, 1, 15, 16, 17, 31, 32, 127, 128, 4095, 4096, 8191])
    for bb, hh in [(0, 0), (3, 15)]:
        want = oracle.fem_linear(q[bb:bb + 1, hh:hh + 1].double().numpy(),
                                 k[bb:bb + 1, hh:hh + 1].double().numpy(),
                                 v[bb:bb + 1, hh:hh + 1].double().numpy(),
                                 b[hh:hh + 1].double().numpy(), rows=rows)
        check(got[bb:bb + 1, hh:hh + 1][:, :, rows], want, TOL,
              f"workload 5 chunk {chunk} (b={bb}, h={hh})")


def test_linear_caller_workspace(fem):
    """A caller-provided workspace gives the same bits as one the binding
    allocates; a short one is rejected before anything is launched."""
    say("linear caller workspace: B2 H4 T3000 (several segments)")
    dev = torch.device("cuda:0")
    q, k, v, b = inputs.draw(4401, 2, 4, 3000, 64, dtype="bf16")
    q, k, v, b = q.to(dev), k.to(dev), v.to(dev), b.to(dev)
    need = fem.workspace_bytes("linear", 2, 4, 3000, 64, 64, 64)
    assert need > 0
    ws = torch.full((need + 512,), 0xAB, dtype=torch.uint8, device=dev)  # dirty on purpose
    a = fem.fem_linear_fwd(q, k, v, b, ws=ws)
    c = fem.fem_linear_fwd(q, k, v, b)
    torch.cuda.synchronize()
    assert torch.equal(a, c)
    out = torch.full((2, 4, 3000, 64), 7.0, device=dev)
    with pytest.raises(fem.FemError) as e:
        fem.fem_linear_fwd(q, k, v, b, out=out, ws=ws[:need - 1])
    assert e.value.status == 6
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
