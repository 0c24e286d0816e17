"""Helpers for the GPU tests: device transfer, running the HIP path, tolerances.

Tolerances (fixed by the acceptance bar of the hot path):
  bf16 runs: max |O - O_ref| <= 2e-2, max |lse - lse_ref| <= 2e-2, and for each of
             dQ, dK, dV: max |g - g_ref| / max |g_ref| <= 5e-2;
  fp32 runs: the same forms, each <= 1e-4.
"""
import numpy as np
import torch

import paper_2607_08186_amd as hd
from paper_2607_08186_amd import synth

TOL = {"bf16": dict(o=2e-2, lse=2e-2, grad=5e-2), "f32": dict(o=1e-4, lse=1e-4, grad=1e-4)}


def dev():
    return torch.device("cuda:0")


def to_dev(a):
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev())
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev())


def to_host64(t):
    if t.dtype == torch.bfloat16:
        bits = t.detach().cpu().view(torch.int16).numpy().view(np.uint16)
        return synth.bf16_bits_to_f32(bits).astype(np.float64)
    return t.detach().cpu().numpy().astype(np.float64)


def bits(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def run_sfa(ins, n, mode, scale, backward=True, window=None):
    """Forward (+ backward) through the C ABI; returns device tensors.  ``window`` is
    the window of a local layer (mode 2) and None otherwise."""
    q, k, v, do = (to_dev(ins[x]) for x in ("q", "k", "v", "dout"))
    o, lse = hd.sfa_forward(q, k, v, n=n, mode=mode, scale=scale, window=window)
    out = {"o": o, "lse": lse}
    if backward:
        dq, dk, dv = hd.sfa_backward(q, k, v, o, lse, do, n=n, mode=mode, scale=scale,
                                     window=window)
        out.update(dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    return out


def rel_err(a, ref):
    den = np.abs(ref).max()
    return np.abs(a - ref).max() / (den if den > 0 else 1.0)


def assert_close_fwd(o, lse, ro, rlse, dtype, what=""):
    t = TOL[dtype]
    eo = np.abs(o - ro).max()
    el = np.abs(lse - rlse).max()
    assert eo <= t["o"], f"{what} O max abs err {eo:.3e} > {t['o']}"
    assert el <= t["lse"], f"{what} lse max abs err {el:.3e} > {t['lse']}"
    return eo, el


def assert_close_grad(g, rg, dtype, name, what=""):
    e = rel_err(g, rg)
    assert e <= TOL[dtype]["grad"], f"{what} {name} rel err {e:.3e} > {TOL[dtype]['grad']}"
    return e
