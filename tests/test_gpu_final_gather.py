"""GPU parity of the final-stream gather that feeds the loss, eq. (hd_loss), and of its
adjoint, against the oracle.  Both are copies, so the bar is bit-exact: every output
word equals the oracle's, including the zeros the backward writes at the first n - 1
streams of every token (dh is filled with a NaN pattern beforehand)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_08186_amd as hd
from paper_2607_08186_amd import synth, workloads
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _h(seed, B, N, Dm, dtype):
    x = synth.normal(seed, (B, N, Dm), 1.0)
    return synth.to_bf16_bits(x) if dtype == "bf16" else x.astype(np.float32)


def _host(t, dtype):
    return G.bits(t) if dtype == "bf16" else t.cpu().numpy()


# B, L, n, Dm, dtype: row bytes multiple of 16, of 4 only, of 2 only; n = 1; one token
CASES = [(2, 37, 3, 40, "bf16"), (1, 100, 4, 13, "f32"), (3, 50, 2, 7, "bf16"),
         (1, 64, 1, 64, "bf16"), (1, 1, 5, 8, "f32"), (2, 300, 8, 128, "f32"),
         (1, 257, 4, 4096, "bf16")]


@pytest.mark.parametrize("B,L,n,Dm,dtype", CASES, ids=[str(c) for c in CASES])
def test_final_gather_bitexact(B, L, n, Dm, dtype):
    seed = synth.seed_for("final_gather", B, L, n, Dm, dtype)
    print(f"final_gather B={B} L={L} n={n} Dm={Dm} {dtype}", flush=True)
    h = _h(seed, B, n * L, Dm, dtype)
    out = hd.final_stream_gather(G.to_dev(h), n)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_host(out, dtype), oracle.final_gather(h, n))


@pytest.mark.parametrize("B,L,n,Dm,dtype", CASES, ids=[str(c) for c in CASES])
def test_final_gather_bwd_bitexact(B, L, n, Dm, dtype):
    seed = synth.seed_for("final_gather_bwd", B, L, n, Dm, dtype)
    print(f"final_gather_bwd B={B} L={L} n={n} Dm={Dm} {dtype}", flush=True)
    dout = _h(seed, B, L, Dm, dtype)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dh = torch.full((B, n * L, Dm), float("nan"), dtype=tdt, device=G.dev())
    hd.hd_final_stream_gather_bwd(G.to_dev(dout), dh, B, L, n, Dm)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_host(dh, dtype), oracle.final_gather_bwd(dout, n))


@pytest.mark.slow
def test_final_gather_stack_shape_roundtrip():
    """The 36-layer stack's loss input: B=1, L=4096 tokens, n=4 streams of width 4096
    (bf16): the gather equals the oracle's, and gathering the backward's output returns
    the upstream gradient unchanged."""
    s = workloads.QWEN8B.shape
    B, L, n, Dm = 1, s.L, s.n, workloads.STACK_DMODEL
    print(f"final_gather stack shape L={L} n={n} Dm={Dm}", flush=True)
    h = _h(synth.seed_for("final_gather_stack"), B, n * L, Dm, "bf16")
    th = G.to_dev(h)
    out = hd.final_stream_gather(th, n)
    dh = hd.final_stream_gather_backward(out, n)
    back = hd.final_stream_gather(dh, n)
    torch.cuda.synchronize()
    want = oracle.final_gather(h, n)
    np.testing.assert_array_equal(G.bits(out), want)
    np.testing.assert_array_equal(G.bits(back), want)
    np.testing.assert_array_equal(G.bits(dh), oracle.final_gather_bwd(want, n))
