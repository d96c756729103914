"""GPU parity of fem_softmax_fwd_ex (HIP, through the C ABI): the encoder
(unmasked) read, d_v = d_qk / 2, and bf16 output, against the float64 oracle.

Tolerances: 2e-2 max abs for fp32 output (the bf16-input budget); for bf16
output 2e-2 + 2^-8 |o_ref| (the output rounding adds at most 2^-9 |o|), and
the bf16 output must equal the fp32 output rounded to nearest even, bit for
bit.  Every case prints its name, shape and seed before touching the GPU.
"""

import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2602_07160_amd import inputs

pytestmark = pytest.mark.gpu

TOL = 2e-2
PAIRS = [(32, 32), (64, 64), (128, 128), (64, 32), (128, 64)]


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def run(fem, q, k, v, b, causal=True, out_dtype=torch.float32):
    dev = torch.device("cuda:0")
    out = fem.fem_softmax_fwd_ex(q.to(dev), k.to(dev), v.to(dev), b.to(dev), causal=causal,
                                 out_dtype=out_dtype)
    torch.cuda.synchronize()
    return out.cpu()


def ref(q, k, v, b, causal=True, rows=None):
    fn = oracle.fem_softmax if causal else oracle.fem_softmax_encoder
    return fn(q.double().numpy(), k.double().numpy(), v.double().numpy(), b.double().numpy(),
              rows=rows)


def check(got, want, what, rel=0.0):
    got = got.double().numpy() if isinstance(got, torch.Tensor) else got
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = (np.abs(got - want) - rel * np.abs(want)).max()
    say(f"{what}: max err {err:.3e} (tol {TOL}{' + %.4g|ref|' % rel if rel else ''})")
    assert err <= TOL, f"{what}: {err} > {TOL}"


def draw(seed, B, H, T, dqk, dv):
    q, k, v, b = inputs.draw(seed, B, H, T, dqk, dv, dtype="bf16")
    return q, k, v, b


@pytest.mark.parametrize("dqk,dv", PAIRS)
@pytest.mark.parametrize("T", [1, 31, 64, 65, 257, 700])
def test_encoder_shapes(fem, dqk, dv, T):
    seed = 6000 + T + dqk + dv
    say(f"encoder bf16 B2 H3 T{T} d_qk{dqk} d_v{dv}, seed {seed}")
    q, k, v, b = draw(seed, 2, 3, T, dqk, dv)
    check(run(fem, q, k, v, b, causal=False), ref(q, k, v, b, causal=False),
          f"encoder T{T} {dqk}/{dv}")


@pytest.mark.parametrize("dqk,dv", [(64, 32), (128, 64)])
@pytest.mark.parametrize("T", [1, 65, 300, 700])
def test_causal_half_value_width(fem, dqk, dv, T):
    seed = 7000 + T + dqk
    say(f"causal bf16 B2 H3 T{T} d_qk{dqk} d_v{dv}, seed {seed}")
    q, k, v, b = draw(seed, 2, 3, T, dqk, dv)
    check(run(fem, q, k, v, b), ref(q, k, v, b), f"causal T{T} {dqk}/{dv}")


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("dqk,dv", [(64, 64), (128, 128), (128, 64)])
def test_bf16_output(fem, causal, dqk, dv):
    seed = 8000 + dqk + dv + int(causal)
    say(f"bf16 output, causal={causal}, B1 H4 T600 d_qk{dqk} d_v{dv}, seed {seed}")
    q, k, v, b = draw(seed, 1, 4, 600, dqk, dv)
    o16 = run(fem, q, k, v, b, causal=causal, out_dtype=torch.bfloat16)
    o32 = run(fem, q, k, v, b, causal=causal)
    assert o16.dtype == torch.bfloat16
    check(o16, ref(q, k, v, b, causal=causal), "bf16 out", rel=2.0 ** -8)
    assert torch.equal(o16, o32.to(torch.bfloat16)), "bf16 output != RNE(fp32 output)"


def test_default_flags_match_plain_entry(fem):
    say("fem_softmax_fwd_ex(causal, fp32) == fem_softmax_fwd: B2 H2 T500 d128, seed 8100")
    q, k, v, b = draw(8100, 2, 2, 500, 128, 128)
    dev = torch.device("cuda:0")
    a = fem.fem_softmax_fwd(q.to(dev), k.to(dev), v.to(dev), b.to(dev))
    torch.cuda.synchronize()
    assert torch.equal(a.cpu(), run(fem, q, k, v, b))


def test_encoder_large_sampled(fem):
    say("encoder bf16 B2 H4 T4096 d128, seed 8200, sampled rows")
    q, k, v, b = draw(8200, 2, 4, 4096, 128, 128)
    got = run(fem, q, k, v, b, causal=False).double().numpy()
    rows = np.array([0, 1, 255, 256, 1000, 2047, 4000, 4095])
    for bb, hh in [(0, 0), (1, 3)]:
        sl = lambda x: x[bb:bb + 1, hh:hh + 1]
        want = oracle.fem_softmax_encoder(sl(q).double().numpy(), sl(k).double().numpy(),
                                          sl(v).double().numpy(), b[hh:hh + 1].double().numpy(),
                                          rows=rows)[0, 0]
        check(got[bb, hh, rows], want, f"encoder T4096 b{bb} h{hh}")


def test_encoder_rows_permutation_invariant(fem):
    """Permuting the (k_i, v_i) pairs leaves every encoder row unchanged (up
    to rounding: the tiles see the keys in another order)."""
    say("encoder key permutation: B1 H2 T333 d64, seed 8300")
    q, k, v, b = draw(8300, 1, 2, 333, 64, 64)
    perm = torch.from_numpy(np.random.default_rng(5).permutation(333))
    a = run(fem, q, k, v, b, causal=False).double().numpy()
    c = run(fem, q, k[:, :, perm].contiguous(), v[:, :, perm].contiguous(), b,
            causal=False).double().numpy()
    err = np.abs(a - c).max()
    say(f"permutation: max diff {err:.3e}")
    assert err <= TOL
