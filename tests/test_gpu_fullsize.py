"""Full-size parity in the launch configuration the benchmark times.

At these sizes the oracle evaluates sampled rows one by one (forward rows, dQ rows,
and dK/dV rows of keys that only the last tokens see); properties that hold at any
size check the rest: the gradient sums of softmax attention (sum over keys of dV is the
group's summed dO; sum over keys of dK is zero), per stream for intra layers.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2607_08186_amd import synth, workloads
from tests import gpu_helpers as G

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

INTRA, MIX, LOCAL = 0, 1, 2
CASES = [workloads.QWEN8B, *workloads.SWEEP, workloads.FRONTIER]


def _sample_rows(rng, B, H, N, count):
    rows = {(0, 0, 0), (B - 1, H - 1, N - 1), (0, H - 1, N // 2), (B - 1, 0, 1)}
    while len(rows) < count:
        rows.add((int(rng.integers(B)), int(rng.integers(H)), int(rng.integers(N))))
    return np.array(sorted(rows), dtype=np.int64)


def _tail_key_rows(rng, B, Hkv, N, n, count):
    rows = set()
    last = range(max(0, N - 2 * n), N)  # keys of the last two tokens
    while len(rows) < count:
        rows.add((int(rng.integers(B)), int(rng.integers(Hkv)), int(rng.choice(list(last)))))
    return np.array(sorted(rows), dtype=np.int64)


@pytest.mark.parametrize("mode", [INTRA, MIX, LOCAL], ids=["intra", "mix", "local"])
@pytest.mark.parametrize("wl", CASES, ids=[w.name for w in CASES])
def test_fullsize_sampled(wl, mode):
    s = wl.shape
    seed = synth.seed_for(wl.name, mode, "parity")
    window = workloads.LOCAL_WINDOW if mode == LOCAL else None
    print(f"fullsize {wl.name} mode={mode} window={window} seed={seed}", flush=True)
    ins = synth.sfa_inputs(s.B, s.L, s.n, s.Hq, s.Hkv, s.D, seed=seed, dtype="bf16",
                           qkv_std=wl.qkv_std, dout_std=wl.dout_std, k_spike=wl.k_spike)
    got = G.run_sfa(ins, s.n, mode, s.scale, window=window)
    kw = dict(L=s.L, n=s.n, mode=mode, scale=s.scale, window=window or 0)
    rng = np.random.default_rng(seed & 0xFFFFFFFF)

    rows = _sample_rows(rng, s.B, s.Hq, s.N, 40)
    ro, rl = oracle.sfa_fwd_rows(ins["q"], ins["k"], ins["v"], rows, **kw)
    rdq = oracle.sfa_bwd_dq_rows(ins["q"], ins["k"], ins["v"], ins["dout"], rows, **kw)
    o = G.to_host64(got["o"])
    lse = G.to_host64(got["lse"])
    dq = G.to_host64(got["dq"])
    b, h, p = rows.T
    G.assert_close_fwd(o[b, p, h], lse[b, h, p], ro, rl, "bf16", wl.name)
    G.assert_close_grad(dq[b, p, h], rdq, "bf16", "dq", wl.name)

    krows = _tail_key_rows(rng, s.B, s.Hkv, s.N, s.n, 8)
    rdk, rdv = oracle.sfa_bwd_dkdv_rows(ins["q"], ins["k"], ins["v"], ins["dout"], krows, **kw)
    dk = G.to_host64(got["dk"])
    dv = G.to_host64(got["dv"])
    b, h, j = krows.T
    G.assert_close_grad(dk[b, j, h], rdk, "bf16", "dk", wl.name)
    G.assert_close_grad(dv[b, j, h], rdv, "bf16", "dv", wl.name)

    # gradient sums over all keys, per (b, kv-head) and per stream for intra
    dout = synth.bf16_bits_to_f32(ins["dout"]).astype(np.float64)
    Gq = s.Hq // s.Hkv
    groups = [slice(None)] if mode != INTRA else [slice(st, None, s.n) for st in range(s.n)]
    for sl in groups:
        want = dout[:, sl].reshape(s.B, -1, s.Hkv, Gq, s.D).sum(axis=(1, 3))
        got_v = dv[:, sl].sum(axis=1)
        scale_v = np.abs(dv[:, sl]).sum(axis=1)
        assert np.all(np.abs(got_v - want) <= 1e-2 * scale_v + 1e-3), "sum_j dV_j != sum dO"
        got_k = dk[:, sl].sum(axis=1)
        scale_k = np.abs(dk[:, sl]).sum(axis=1)
        assert np.all(np.abs(got_k) <= 1e-2 * scale_k + 1e-3), "sum_j dK_j != 0"
    assert np.all(np.isfinite(lse)) and np.all(np.isfinite(o))
