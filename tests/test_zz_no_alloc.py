"""GPU check of fem_softmax_decode_noalloc (the decoding step that keeps its
partial results in the library's fixed per-device array instead of a caller
workspace) against fem_softmax_decode, through the C ABI.

Two calls in a row, the second with a smaller problem, so the second reads
an array that still holds the first call's partials.  Both entry points run
the same kernels with the same split plan, so the outputs must be equal bit
for bit; a few rows are also checked against the float64 oracle (2e-2, the
bf16-input budget).  Every case prints its name and sizes before touching
the GPU.
"""

import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2602_07160_amd import inputs

pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def one_step(fem, seed, B, H, L, dqk, dv, lens):
    dev = torch.device("cuda:0")
    q, k, v, b = inputs.draw(seed, B, H, L, dqk, dv, dtype="bf16")
    q1 = q[:, :, -1].contiguous()
    ld = torch.as_tensor(lens, dtype=torch.int32).to(dev)
    args = (q1.to(dev), k.to(dev), v.to(dev), b.to(dev))
    got = fem.fem_softmax_decode_noalloc(*args, lens=ld)
    torch.cuda.synchronize()
    got = got.cpu()
    want = fem.fem_softmax_decode(*args, lens=ld)
    torch.cuda.synchronize()
    want = want.cpu()
    assert torch.isfinite(got).all()
    assert torch.equal(got, want), float((got - want).abs().max())
    # the oracle on the first and last sequences
    for bb in (0, B - 1):
        n = int(lens[bb])
        ref = oracle.fem_softmax_decode(q1[bb:bb + 1].double().numpy(),
                                        k[bb:bb + 1].double().numpy(),
                                        v[bb:bb + 1].double().numpy(), np.array([n]),
                                        b.double().numpy())
        err = float(np.abs(got[bb:bb + 1].double().numpy() - ref).max())
        say(f"  b={bb} len={n}: max abs err vs oracle {err:.3e}")
        assert err <= 2e-2


def test_noalloc_two_calls_second_smaller(fem):
    say("decode_noalloc call 1: B8 H16 L4096 d128, mixed lengths, seed 9901")
    rng = np.random.default_rng(9901)
    lens1 = np.concatenate([[4096, 1], rng.integers(1, 4097, 6)]).astype(np.int32)
    one_step(fem, 9901, 8, 16, 4096, 128, 128, lens1)
    say("decode_noalloc call 2: B2 H3 L300 d_qk64 d_v32, seed 9902")
    one_step(fem, 9902, 2, 3, 300, 64, 32, np.array([300, 77], dtype=np.int32))


def test_noalloc_rejects_oversize(fem):
    say("decode_noalloc size limit: B64 H128 L64 d128 needs more than 8 MiB of partials")
    dev = torch.device("cuda:0")
    B, H, L, d = 64, 128, 64, 128
    assert fem.workspace_bytes("decode", B, H, L, d, d) > 8 << 20
    q = torch.zeros(B, H, d, dtype=torch.bfloat16, device=dev)
    kc = torch.zeros(B, H, L, d, dtype=torch.bfloat16, device=dev)
    b = torch.ones(H, d, device=dev)
    out = torch.full((B, H, d), 3.0, device=dev)
    with pytest.raises(fem.FemError) as e:
        fem.fem_softmax_decode_noalloc(q, kc, kc, b, out=out)
    assert e.value.status == 6
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())
