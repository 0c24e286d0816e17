"""GPU parity of the final-stream layers (only the final stream of each token carries a
query; keys and values over all n streams; full cross-stream mask, or a local window)
against the fp64 oracle, at sizes that span several tiles with ragged tails, plus
full-size sampled parity at the Qwen3-8B-like shape.  Tolerances as for the other bf16
layers: max |O - O_ref| and max |lse - lse_ref| <= 2e-2, and for each of dQ, dK, dV
max |g - g_ref| / max |g_ref| <= 5e-2."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2607_08186_amd as hd
from paper_2607_08186_amd import synth, workloads
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

MIX, LOCAL = 1, 2


def _inputs(seed, B, L, n, Hq, Hkv, D, std=2 ** -0.5):
    N = n * L
    to = synth.to_bf16_bits
    return dict(q=to(synth.normal(seed, (B, L, Hq, D), std)),
                k=to(synth.normal(seed + 1, (B, N, Hkv, D), std)),
                v=to(synth.normal(seed + 2, (B, N, Hkv, D), std)),
                dout=to(synth.normal(seed + 3, (B, L, Hq, D), 1.0)))


def _run(ins, n, window, scale):
    q, k, v, do = (G.to_dev(ins[x]) for x in ("q", "k", "v", "dout"))
    o, lse = hd.sfa_final_forward(q, k, v, n=n, window=window, scale=scale)
    dq, dk, dv = hd.sfa_final_backward(q, k, v, o, lse, do, n=n, window=window, scale=scale)
    torch.cuda.synchronize()
    return {name: G.to_host64(t) for name, t in
            dict(o=o, lse=lse, dq=dq, dk=dk, dv=dv).items()}


# B, L, n, Hq, Hkv, D, window (0: full cross-stream mask)
CASES = [
    (1, 200, 2, 4, 2, 64, 0),     # 200 final rows: one 256-row block, ragged
    (2, 130, 3, 2, 1, 128, 0),    # B=2, odd n
    (1, 64, 4, 8, 2, 32, 0),      # D=32, GQA 4
    (1, 97, 1, 2, 2, 128, 0),     # n=1: the full cross-stream layer itself
    (1, 40, 8, 4, 1, 64, 0),      # n=8
    (1, 1, 3, 2, 1, 128, 0),      # one token
    (1, 300, 2, 2, 2, 128, 0),    # two 256-row blocks
    (1, 300, 4, 2, 1, 128, 100),  # local window across key tiles
    (1, 257, 3, 4, 2, 64, 1),     # window 1: each query sees only its own key
    (2, 100, 2, 2, 1, 128, 37),
    (1, 150, 4, 2, 2, 128, 5000), # window >= n*L: the full mask
]


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_final_stream_parity(case):
    B, L, n, Hq, Hkv, D, w = case
    seed = synth.seed_for("final", case)
    print(f"final case={case} seed={seed}", flush=True)
    ins = _inputs(seed, B, L, n, Hq, Hkv, D)
    scale = 1.0 / math.sqrt(D)
    got = _run(ins, n, w, scale)
    kw = dict(L=L, n=n, mode=LOCAL if w else MIX, scale=scale, window=w, final=True)
    ro, rl = oracle.sfa_fwd(ins["q"], ins["k"], ins["v"], **kw)
    rdq, rdk, rdv = oracle.sfa_bwd(ins["q"], ins["k"], ins["v"], ins["dout"], **kw)
    G.assert_close_fwd(got["o"], got["lse"], ro, rl, "bf16", str(case))
    for name, ref in (("dq", rdq), ("dk", rdk), ("dv", rdv)):
        G.assert_close_grad(got[name], ref, "bf16", name, str(case))


def test_final_stream_unseen_keys_get_zero_gradient():
    """Window 1: only the final-stream keys are seen, so the keys of the other streams
    get exactly zero dK and dV."""
    B, L, n, Hq, Hkv, D = 1, 130, 4, 2, 1, 64
    ins = _inputs(synth.seed_for("final_unseen"), B, L, n, Hq, Hkv, D)
    got = _run(ins, n, 1, D ** -0.5)
    for name in ("dk", "dv"):
        other = np.delete(got[name], np.arange(n - 1, n * L, n), axis=1)
        assert np.all(other == 0), name


def test_final_stream_uniform_logit_probe():
    """q = 0: token t's query sees (t+1) n keys; lse = ln((t+1) n) and, with one-hot
    values v_j = e_(j mod D), O[d] counts the visible keys with j = d (mod D)."""
    L, n, D = 90, 3, 64
    N = n * L
    ins = dict(q=synth.to_bf16_bits(np.zeros((1, L, 1, D))),
               k=synth.to_bf16_bits(synth.normal(5, (1, N, 1, D))),
               v=np.zeros((1, N, 1, D)), dout=synth.to_bf16_bits(np.zeros((1, L, 1, D))))
    ins["v"][0, np.arange(N), 0, np.arange(N) % D] = 1.0
    ins["v"] = synth.to_bf16_bits(ins["v"])
    got = _run(ins, n, 0, 1.0)
    for t in range(L):
        vis = np.arange(t * n + n)
        assert abs(got["lse"][0, 0, t] - math.log(len(vis))) < 1e-5
        want = np.bincount(vis % D, minlength=D) / len(vis)
        np.testing.assert_array_equal(got["o"][0, t, 0] == 0, want == 0)
        np.testing.assert_allclose(got["o"][0, t, 0], want, atol=4e-3)


def test_final_stream_deterministic():
    B, L, n, Hq, Hkv, D = 1, 257, 3, 4, 1, 128
    ins = _inputs(synth.seed_for("final_det"), B, L, n, Hq, Hkv, D)
    a = _run(ins, n, 0, D ** -0.5)
    b = _run(ins, n, 0, D ** -0.5)
    for name in a:
        np.testing.assert_array_equal(a[name], b[name])


@pytest.mark.slow
@pytest.mark.parametrize("window", [0, workloads.LOCAL_WINDOW], ids=["full", "local"])
def test_final_stream_fullsize_sampled(window):
    """Qwen3-8B-like shape (L=4096 final-stream rows over N=16384 keys, Hq=32, Hkv=8,
    D=128): sampled rows against the oracle (dK/dV of keys across the whole sequence,
    the first key included, which every final-stream query sees), and the gradient sums (the keys'
    dV add up to the group's summed dO, their dK to zero) over every key."""
    s = workloads.QWEN8B.shape
    seed = synth.seed_for("final_full", window)
    print(f"final fullsize window={window} seed={seed}", flush=True)
    ins = _inputs(seed, s.B, s.L, s.n, s.Hq, s.Hkv, s.D)
    got = _run(ins, s.n, window, s.scale)
    kw = dict(L=s.L, n=s.n, mode=LOCAL if window else MIX, scale=s.scale, window=window,
              final=True)
    rng = np.random.default_rng(seed & 0xFFFFFFFF)
    rows = {(0, 0, 0), (0, s.Hq - 1, s.L - 1), (0, 3, s.L // 2)}
    while len(rows) < 40:
        rows.add((0, int(rng.integers(s.Hq)), int(rng.integers(s.L))))
    rows = np.array(sorted(rows), dtype=np.int64)
    ro, rl = oracle.sfa_fwd_rows(ins["q"], ins["k"], ins["v"], rows, **kw)
    rdq = oracle.sfa_bwd_dq_rows(ins["q"], ins["k"], ins["v"], ins["dout"], rows, **kw)
    b, h, t = rows.T
    G.assert_close_fwd(got["o"][b, t, h], got["lse"][b, h, t], ro, rl, "bf16", "final")
    G.assert_close_grad(got["dq"][b, t, h], rdq, "bf16", "dq", "final")
    # keys of one key/value head: near the start (seen by every final-stream query, or by
    # the whole first window), in the first 128-key block, in the middle block, and last
    hk = int(rng.integers(s.Hkv))
    heavy = [0, 1, int(rng.integers(2, 128)), s.N // 2 + int(rng.integers(128))]
    for what, keys in (("heavy keys", heavy), ("last keys", (s.N - 1, s.N - 2, s.N - s.n - 1, s.N - 7))):
        krows = np.array([(0, hk, j) for j in keys], dtype=np.int64)
        print(f"  dK/dV of {what}: {krows.tolist()}", flush=True)
        rdk, rdv = oracle.sfa_bwd_dkdv_rows(ins["q"], ins["k"], ins["v"], ins["dout"], krows,
                                            **kw)
        b, h, j = krows.T
        G.assert_close_grad(got["dk"][b, j, h], rdk, "bf16", "dk", f"final {what}")
        G.assert_close_grad(got["dv"][b, j, h], rdv, "bf16", "dv", f"final {what}")
    dout = synth.bf16_bits_to_f32(ins["dout"]).astype(np.float64)
    Gq = s.Hq // s.Hkv
    want = dout.reshape(s.B, s.L, s.Hkv, Gq, s.D).sum(axis=(1, 3))
    dv, dk = got["dv"], got["dk"]
    assert np.all(np.abs(dv.sum(axis=1) - want) <= 1e-2 * np.abs(dv).sum(axis=1) + 1e-3)
    assert np.all(np.abs(dk.sum(axis=1)) <= 1e-2 * np.abs(dk).sum(axis=1) + 1e-3)
