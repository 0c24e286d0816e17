"""GPU parity of the bf16 backward in query bands (a workspace below the one-pass size).

The backward accepts any workspace from hd_sfa_bwd_min_workspace_bytes up.  Below the
one-pass size it sweeps the query rows in bands of whole 256-row units: each band's
dK/dV pass stores only that band's dS tiles and its dQ pass reads them back, and dK/dV
are carried between bands as fp32 partials.  Checked here:
  * element-wise against the fp64 oracle at the bf16 bar (max |g - g_ref| / max |g_ref|
    <= 5e-2 for dQ, dK, dV), with the smallest workspace and one between the smallest and
    the one-pass size, at sizes with several bands and ragged tails, for every layer
    type (intra-stream, full and local cross-stream, final-stream);
  * dQ bitwise equal to the one-pass run (it reads the same dS values) and dK/dV equal
    to it up to the fp32 summation order of the band partials;
  * the Qwen3-8B-like layer at full size in bands, against the one-pass run and on
    sampled rows and keys against the oracle.
The backward at the longest expanded length the boundary accepts, which only the banded
path can run, is in test_gpu_fullsize.py next to the forward at that length.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_08186_amd as hd
from paper_2607_08186_amd import synth, workloads
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

INTRA, MIX, LOCAL = 0, 1, 2
ULP_REL = 2.0 ** -7  # dK/dV of banded and one-pass runs: bf16 roundings of nearly equal sums


def _dkdv_launches():
    """dK/dV sweep launches (one per query band; a split-sweep combine is not one)."""
    return sum(n for name, n, _ in hd.hd_timing_collect()
               if name.startswith("sfa_dkdv") and "combine" not in name)


def _backward(q, k, v, o, lse, do, *, n, mode, scale, window, final, ws_bytes):
    """Backward with a workspace of ws_bytes (None: one pass); returns the gradients and
    the number of dK/dV launches (= query bands)."""
    hd.hd_timing_collect()
    hd.hd_timing_filter("sfa_dkdv")
    hd.hd_timing_enable(True)
    try:
        if final:
            out = hd.sfa_final_backward(q, k, v, o, lse, do, n=n, scale=scale,
                                        window=window or 0, workspace_bytes=ws_bytes)
        else:
            out = hd.sfa_backward(q, k, v, o, lse, do, n=n, mode=mode, scale=scale,
                                  window=window, workspace_bytes=ws_bytes)
        torch.cuda.synchronize()
        bands = _dkdv_launches()
    finally:
        hd.hd_timing_enable(False)
        hd.hd_timing_filter(None)
    return out, bands


def _sizes(B, L, n, Hq, Hkv, D, mode, window, final):
    if final:
        w = window or 0
        return (hd.hd_sfa_bwd_final_min_workspace_bytes(B, L, n, Hq, Hkv, D, w, hd.HD_DTYPE_BF16),
                hd.hd_sfa_bwd_final_workspace_bytes(B, L, n, Hq, Hkv, D, w, hd.HD_DTYPE_BF16))
    if mode == LOCAL:
        return (hd.hd_sfa_bwd_local_min_workspace_bytes(B, L, n, Hq, Hkv, D, window, hd.HD_DTYPE_BF16),
                hd.hd_sfa_bwd_local_workspace_bytes(B, L, n, Hq, Hkv, D, window, hd.HD_DTYPE_BF16))
    return (hd.hd_sfa_bwd_min_workspace_bytes(B, L, n, Hq, Hkv, D, mode, hd.HD_DTYPE_BF16),
            hd.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, mode, hd.HD_DTYPE_BF16))


def _same_as_one_pass(got, ref, what):
    gq, gk, gv = (G.bits(t) for t in got)
    rq, rk, rv = (G.bits(t) for t in ref)
    assert np.array_equal(gq, rq), f"{what}: dQ differs from the one-pass run"
    for name, a, b in (("dk", got[1], ref[1]), ("dv", got[2], ref[2])):
        e = G.rel_err(G.to_host64(a), G.to_host64(b))
        assert e <= ULP_REL, f"{what}: {name} differs from the one-pass run by {e:.3e}"


# B, L, n, Hq, Hkv, D, mode, window, final
# (shapes where the smallest workspace is below the one-pass size: the fp32 dK/dV
# partials, 8 bytes per key and head dim, must not outweigh the dS tiles)
CASES = [
    (1, 300, 4, 4, 2, 64, MIX, None, False),      # N=1200: five 256-row units, the last ragged
    (1, 2000, 2, 8, 1, 64, INTRA, None, False),   # 2000 rows per stream: eight units
    (2, 1100, 3, 4, 1, 128, INTRA, None, False),  # B=2, odd n, ragged units
    (1, 1000, 1, 8, 2, 32, MIX, None, False),     # n=1, D=32
    (1, 400, 3, 4, 1, 128, LOCAL, 200, False),    # window across key tiles
    (1, 500, 2, 8, 2, 64, LOCAL, 700, False),
    (1, 600, 3, 4, 1, 128, MIX, None, True),      # final-stream queries, 600 rows
    (1, 1400, 3, 8, 1, 64, LOCAL, 300, True),     # final-stream, local window
]


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_banded_backward_parity(case):
    B, L, n, Hq, Hkv, D, mode, window, final = case
    seed = synth.seed_for("banded", case)
    print(f"banded {case} seed={seed}", flush=True)
    scale = D ** -0.5
    N = n * L
    qrows = L if final else N
    to = synth.to_bf16_bits
    std = 2 ** -0.5
    ins = dict(q=to(synth.normal(seed, (B, qrows, Hq, D), std)),
               k=to(synth.normal(seed + 1, (B, N, Hkv, D), std)),
               v=to(synth.normal(seed + 2, (B, N, Hkv, D), std)),
               dout=to(synth.normal(seed + 3, (B, qrows, Hq, D), 1.0)))
    q, k, v, do = (G.to_dev(ins[x]) for x in ("q", "k", "v", "dout"))
    if final:
        o, lse = hd.sfa_final_forward(q, k, v, n=n, window=window or 0, scale=scale)
    else:
        o, lse = hd.sfa_forward(q, k, v, n=n, mode=mode, scale=scale, window=window)
    kw = dict(n=n, mode=mode, scale=scale, window=window, final=final)
    low, full = _sizes(B, L, n, Hq, Hkv, D, mode, window, final)
    assert 0 < low < full
    one, bands1 = _backward(q, k, v, o, lse, do, ws_bytes=None, **kw)
    assert bands1 == 1
    ref = oracle.sfa_bwd(ins["q"], ins["k"], ins["v"], ins["dout"], L=L, n=n,
                         mode=MIX if final and not window else mode, scale=scale,
                         window=window or 0, final=final)
    for ws in (low, (low + full) // 2 // 256 * 256):
        got, bands = _backward(q, k, v, o, lse, do, ws_bytes=ws, **kw)
        assert bands >= 2, f"workspace {ws} of {full}: {bands} band(s)"
        for name, g, r in zip(("dq", "dk", "dv"), got, ref):
            G.assert_close_grad(G.to_host64(g), r, "bf16", name, f"{case} ws={ws} bands={bands}")
        _same_as_one_pass(got, one, f"{case} ws={ws} bands={bands}")


@pytest.mark.slow
@pytest.mark.parametrize("mode", [INTRA, MIX], ids=["intra", "mix"])
def test_banded_backward_fullsize(mode):
    """The Qwen3-8B-like layer (B=1, L=4096, n=4, Hq=32, Hkv=8, D=128) with a workspace of
    a fifth of the way from the smallest to the one-pass size: dQ bitwise and dK/dV to
    the summation order equal to the one-pass run, and sampled dQ rows and dK/dV of the
    last keys (plus, intra-stream, the first keys of two streams) against the oracle."""
    wl = workloads.QWEN8B
    s = wl.shape
    seed = synth.seed_for(wl.name, mode, "banded")
    print(f"banded fullsize mode={mode} seed={seed}", flush=True)
    ins = synth.sfa_inputs(s.B, s.L, s.n, s.Hq, s.Hkv, s.D, seed=seed, dtype="bf16",
                           qkv_std=wl.qkv_std, dout_std=wl.dout_std, k_spike=wl.k_spike)
    q, k, v, do = (G.to_dev(ins[x]) for x in ("q", "k", "v", "dout"))
    o, lse = hd.sfa_forward(q, k, v, n=s.n, mode=mode, scale=s.scale)
    kw = dict(n=s.n, mode=mode, scale=s.scale, window=None, final=False)
    low, full = _sizes(s.B, s.L, s.n, s.Hq, s.Hkv, s.D, mode, None, False)
    ws = (low + (full - low) // 5) // 256 * 256
    one, _ = _backward(q, k, v, o, lse, do, ws_bytes=None, **kw)
    got, bands = _backward(q, k, v, o, lse, do, ws_bytes=ws, **kw)
    print(f"  {bands} bands with {ws / 2**30:.2f} GiB (one pass {full / 2**30:.2f} GiB)", flush=True)
    assert bands >= 3
    _same_as_one_pass(got, one, f"fullsize mode={mode}")

    rng = np.random.default_rng(seed & 0xFFFFFFFF)
    okw = dict(L=s.L, n=s.n, mode=mode, scale=s.scale)
    rows = {(0, 0, 0), (0, s.Hq - 1, s.N - 1), (0, 5, s.N // 2)}
    while len(rows) < 24:
        rows.add((0, int(rng.integers(s.Hq)), int(rng.integers(s.N))))
    rows = np.array(sorted(rows), dtype=np.int64)
    rdq = oracle.sfa_bwd_dq_rows(ins["q"], ins["k"], ins["v"], ins["dout"], rows, **okw)
    dq = G.to_host64(got[0])
    b, h, p = rows.T
    G.assert_close_grad(dq[b, p, h], rdq, "bf16", "dq", "banded fullsize")
    hk = int(rng.integers(s.Hkv))
    keys = {(0, hk, s.N - 1), (0, hk, s.N - 2), (0, hk, s.N - s.n - 1)}
    if mode == INTRA:  # the first key of streams 0 and n-1: every query of its stream sees it
        keys |= {(0, hk, 0), (0, hk, s.n - 1), (0, hk, 77 * s.n + 2)}
    keys = np.array(sorted(keys), dtype=np.int64)
    rdk, rdv = oracle.sfa_bwd_dkdv_rows(ins["q"], ins["k"], ins["v"], ins["dout"], keys, **okw)
    dk, dv = G.to_host64(got[1]), G.to_host64(got[2])
    b, h, j = keys.T
    G.assert_close_grad(dk[b, j, h], rdk, "bf16", "dk", "banded fullsize")
    G.assert_close_grad(dv[b, j, h], rdv, "bf16", "dv", "banded fullsize")
