"""GPU parity of fem_softmax_decode (one decoding step against a KV cache,
HIP through the C ABI) against the float64 oracle.

Tolerance: 2e-2 max abs (the bf16-input budget; the step itself computes in
fp32 with a per-channel joint log-sum-exp).  Every case prints its name,
shape and seed before touching the GPU.
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


def draw(seed, B, H, L, dqk, dv, **kw):
    q, k, v, b = inputs.draw(seed, B, H, L, dqk, dv, dtype="bf16", **kw)
    return q, k, v, b


def run(fem, q1, k, v, b, lens):
    dev = torch.device("cuda:0")
    ld = None if lens is None else torch.as_tensor(lens, dtype=torch.int32).to(dev)
    out = fem.fem_softmax_decode(q1.to(dev), k.to(dev), v.to(dev), b.to(dev), lens=ld)
    torch.cuda.synchronize()
    return out.cpu().double().numpy()


def ref(q1, k, v, b, lens):
    L = k.shape[2]
    lens = np.full(k.shape[0], L) if lens is None else np.asarray(lens)
    return oracle.fem_softmax_decode(q1.double().numpy(), k.double().numpy(),
                                     v.double().numpy(), lens, b.double().numpy())


def check(got, want, what):
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - want).max()
    say(f"{what}: max abs err {err:.3e} (tol {TOL})")
    assert err <= TOL, f"{what}: {err} > {TOL}"


@pytest.mark.parametrize("dqk,dv", PAIRS)
@pytest.mark.parametrize("L", [1, 63, 64, 65, 300, 2048])
def test_decode_shapes(fem, dqk, dv, L):
    seed = 9000 + L + dqk + dv
    say(f"decode B3 H2 L{L} d_qk{dqk} d_v{dv}, seed {seed}")
    q, k, v, b = draw(seed, 3, 2, L, dqk, dv)
    q1 = q[:, :, -1].contiguous()
    rng = np.random.default_rng(seed)
    lens = [L, 1, int(rng.integers(1, L + 1))]
    check(run(fem, q1, k, v, b, lens), ref(q1, k, v, b, lens), f"L{L} {dqk}/{dv} lens {lens}")


def test_decode_full_cache_default_lens(fem):
    say("decode lens=NULL: B2 H4 L777 d64, seed 9100")
    q, k, v, b = draw(9100, 2, 4, 777, 64, 64)
    q1 = q[:, :, 5].contiguous()
    check(run(fem, q1, k, v, b, None), ref(q1, k, v, b, None), "lens=NULL")


def test_decode_matches_causal_row(fem):
    """The step for query t over t+1 cached keys is row t of the causal read."""
    say("decode vs fem_softmax_fwd row t: B2 H2 T512 d128, seed 9200")
    q, k, v, b = draw(9200, 2, 2, 512, 128, 128)
    dev = torch.device("cuda:0")
    full = fem.fem_softmax_fwd(q.to(dev), k.to(dev), v.to(dev), b.to(dev))
    torch.cuda.synchronize()
    full = full.cpu().double().numpy()
    want = oracle.fem_softmax(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                              b.double().numpy(), rows=np.array([0, 100, 511]))
    for r, t in enumerate((0, 100, 511)):
        got = run(fem, q[:, :, t].contiguous(), k, v, b, [t + 1, t + 1])
        check(got, want[:, :, r], f"step t={t} vs oracle")
        err = np.abs(got - full[:, :, t]).max()
        say(f"step t={t} vs fem_softmax_fwd row: {err:.3e}")
        assert err <= 2 * TOL


def test_decode_invalid_lengths_give_nan(fem):
    say("decode lens 0 and L+1 -> NaN rows: B3 H2 L100 d64, seed 9300")
    q, k, v, b = draw(9300, 3, 2, 100, 64, 64)
    q1 = q[:, :, 0].contiguous()
    got = run(fem, q1, k, v, b, [0, 50, 101])
    assert np.isnan(got[0]).all() and np.isnan(got[2]).all()
    check(got[1:2], ref(q1[1:2], k[1:2], v[1:2], b, [50]), "valid row beside invalid ones")


@pytest.mark.parametrize("beta", [1e-3, 64.0])
def test_decode_beta_extremes(fem, beta):
    say(f"decode constant beta {beta}: B2 H2 L1000 d128, seed 9400")
    q, k, v, _ = draw(9400, 2, 2, 1000, 128, 128)
    b = torch.full((2, 128), beta)
    q1 = q[:, :, 3].contiguous()
    check(run(fem, q1, k, v, b, [1000, 613]), ref(q1, k, v, b, [1000, 613]), f"beta={beta}")


def test_decode_serving_shape(fem):
    say("decode B8 H16 L4096 d128, seed 9500, random lengths")
    q, k, v, b = draw(9500, 8, 16, 4096, 128, 128)
    q1 = q[:, :, 0].contiguous()
    lens = [4096, 1, 64, 65, 2000, 4095, 3000, 17]
    check(run(fem, q1, k, v, b, lens), ref(q1, k, v, b, lens), "serving shape")
