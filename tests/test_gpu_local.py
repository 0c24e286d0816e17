"""GPU parity of local cross-stream layers (Fig. "masks" panel (b)): the causal mask
over the expanded sequence restricted to a sliding window of w expanded positions,
p - w < p' <= p, through hd_sfa_fwd_local / hd_sfa_bwd_local, against the fp64
oracle on seeded inputs.

Windows cover the degenerate w = 1 (every row sees only itself), windows shorter than
the stream count, windows at and around the 64-row tile size, windows that end inside
a tile, and windows at least as long as the sequence (the full causal layer).
"""
import math

import numpy as np
import pytest

import oracle
from paper_2607_08186_amd import synth
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

MIX, LOCAL = 1, 2

# (B, L, n, Hq, Hkv, D), window
BF16_CASES = [
    ((1, 200, 2, 4, 2, 64), 1),
    ((1, 200, 2, 4, 2, 64), 3),      # shorter than a tile, ragged N=400
    ((1, 200, 2, 4, 2, 64), 64),
    ((1, 200, 2, 4, 2, 64), 65),
    ((2, 130, 3, 2, 1, 128), 100),   # B=2, odd n, window ends inside a tile
    ((2, 130, 3, 2, 1, 128), 127),
    ((1, 64, 4, 8, 2, 32), 200),     # D=32, GQA 4
    ((1, 300, 2, 2, 2, 128), 129),   # several key tiles per row tile
    ((1, 300, 2, 2, 2, 128), 333),
    ((1, 97, 1, 2, 2, 128), 50),     # n=1: a plain sliding-window causal layer
    ((1, 40, 8, 4, 1, 64), 7),       # n=8, window shorter than a token's streams
    ((1, 1, 3, 2, 1, 128), 2),       # a single token
    ((1, 150, 2, 2, 1, 64), 300),    # w == N: the full causal layer
    ((1, 150, 2, 2, 1, 64), 10000),  # w > N
]


def _case(shape, window, dtype, seed):
    B, L, n, Hq, Hkv, D = shape
    ins = synth.sfa_inputs(B, L, n, Hq, Hkv, D, seed=seed, dtype=dtype,
                           qkv_std=1.0 if dtype == "f32" else 2 ** -0.5)
    scale = 1.0 / math.sqrt(D)
    print(f"case shape={shape} window={window} dtype={dtype} seed={seed}", flush=True)
    got = G.run_sfa(ins, n, LOCAL, scale, window=window)
    kw = dict(L=L, n=n, mode=LOCAL, scale=scale, window=window)
    ro, rlse = oracle.sfa_fwd(ins["q"], ins["k"], ins["v"], **kw)
    rdq, rdk, rdv = oracle.sfa_bwd(ins["q"], ins["k"], ins["v"], ins["dout"], **kw)
    what = f"{shape} w={window}"
    G.assert_close_fwd(G.to_host64(got["o"]), G.to_host64(got["lse"]), ro, rlse, dtype, what)
    for name, ref in (("dq", rdq), ("dk", rdk), ("dv", rdv)):
        G.assert_close_grad(G.to_host64(got[name]), ref, dtype, name, what)


@pytest.mark.parametrize("shape,window", BF16_CASES, ids=[f"{s}-w{w}" for s, w in BF16_CASES])
def test_bf16_local_parity(shape, window):
    _case(shape, window, "bf16", seed=synth.seed_for("bf16-local", shape, window))


F32_CASES = [
    ((1, 64, 2, 2, 1, 32), 1),
    ((1, 64, 2, 2, 1, 32), 17),
    ((1, 37, 3, 4, 2, 64), 64),
    ((2, 70, 2, 2, 1, 128), 65),
    ((2, 70, 2, 2, 1, 128), 140),
    ((1, 1, 1, 1, 1, 32), 1),
]


@pytest.mark.parametrize("shape,window", F32_CASES, ids=[f"{s}-w{w}" for s, w in F32_CASES])
def test_f32_local_parity(shape, window):
    _case(shape, window, "f32", seed=synth.seed_for("f32-local", shape, window))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_window_covering_sequence_is_the_full_layer(dtype):
    """w >= N visits the same tiles with the same masks as the full cross-stream layer:
    outputs and gradients are bitwise those of hd_sfa_fwd / hd_sfa_bwd in MIX mode."""
    B, L, n, Hq, Hkv, D = 1, 190, 3, 4, 2, 128 if dtype == "bf16" else 64
    ins = synth.sfa_inputs(B, L, n, Hq, Hkv, D, seed=21, dtype=dtype)
    full = G.run_sfa(ins, n, MIX, D ** -0.5)
    for w in (n * L, n * L + 1, 1 << 30):
        loc = G.run_sfa(ins, n, LOCAL, D ** -0.5, window=w)
        for name in ("o", "lse", "dq", "dk", "dv"):
            assert loc[name].cpu().equal(full[name].cpu()), (w, name)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_window_one_copies_value(dtype):
    """w = 1: every row sees only its own key, so O = V of its group bit for bit and
    lse = scale q.k (one term)."""
    B, L, n, Hq, Hkv, D = 1, 100, 3, 4, 2, 64
    ins = synth.sfa_inputs(B, L, n, Hq, Hkv, D, seed=22, dtype=dtype)
    got = G.run_sfa(ins, n, LOCAL, D ** -0.5, backward=False, window=1)
    o = got["o"].cpu()
    v = G.to_dev(ins["v"]).cpu()
    for h in range(Hq):
        assert o[:, :, h].equal(v[:, :, h // 2]), h
    q = G.to_host64(G.to_dev(ins["q"]))
    k = G.to_host64(G.to_dev(ins["k"]))
    want = np.einsum("bphd,bphd->bhp", q, np.repeat(k, 2, axis=2)) * D ** -0.5
    tol = 1e-4 if dtype == "f32" else 2e-2
    assert np.abs(G.to_host64(got["lse"]) - want).max() <= tol


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("window", [1, 5, 64, 130])
def test_uniform_logit_window_probe(dtype, window):
    """Q = 0: lse_p = ln min(p+1, w) exactly; with one-hot V_j = e_(j mod D), O_p[d]
    counts the keys of the window with j = d (mod D), so the zero pattern of O names
    exactly which keys a row sees."""
    L, n, D = 80, 4, 64
    N = n * L
    q = np.zeros((1, N, 1, D))
    k = synth.normal(1, (1, N, 1, D))
    v = np.zeros((1, N, 1, D))
    v[0, np.arange(N), 0, np.arange(N) % D] = 1.0
    do = np.zeros((1, N, 1, D))
    conv = synth.to_bf16_bits if dtype == "bf16" else (lambda x: x.astype(np.float32))
    ins = {"q": conv(q), "k": conv(k), "v": conv(v), "dout": conv(do)}
    got = G.run_sfa(ins, n, LOCAL, 1.0, backward=False, window=window)
    o, lse = G.to_host64(got["o"]), G.to_host64(got["lse"])
    for p in range(N):
        vis = np.arange(max(0, p - window + 1), p + 1)
        want = np.bincount(vis % D, minlength=D) / len(vis)
        assert abs(lse[0, 0, p] - math.log(len(vis))) < 1e-5, p
        np.testing.assert_array_equal(o[0, p, 0] == 0, want == 0)
        np.testing.assert_allclose(o[0, p, 0], want, atol=4e-3 if dtype == "bf16" else 1e-6)


def test_keys_before_the_window_are_never_read():
    """Poison every key/value row older than the windows of the rows from P0 on (a
    multiple of 128, so no wave or workgroup mixes the two groups of rows): the
    outputs of rows >= P0, and dK/dV of keys >= P0 (which only those rows see), must
    not change by a single bit."""
    B, L, n, Hq, Hkv, D = 1, 320, 2, 2, 1, 128
    window, P0 = 100, 384
    ins = synth.sfa_inputs(B, L, n, Hq, Hkv, D, seed=23, dtype="bf16")
    base = G.run_sfa(ins, n, LOCAL, D ** -0.5, window=window)
    poisoned = dict(ins)
    cut = P0 - window + 1
    for name in ("k", "v"):
        arr = ins[name].copy()
        arr[:, :cut] = synth.to_bf16_bits(np.full(arr[:, :cut].shape, 3.0e4))
        poisoned[name] = arr
    got = G.run_sfa(poisoned, n, LOCAL, D ** -0.5, window=window)
    for name in ("o", "dq", "dk", "dv"):
        np.testing.assert_array_equal(G.bits(base[name])[:, P0:], G.bits(got[name])[:, P0:],
                                      err_msg=name)
    np.testing.assert_array_equal(base["lse"].cpu().numpy()[:, :, P0:],
                                  got["lse"].cpu().numpy()[:, :, P0:])


def test_local_deterministic():
    """No atomics: two runs give bitwise identical outputs."""
    B, L, n, Hq, Hkv, D = 1, 257, 3, 4, 1, 128
    ins = synth.sfa_inputs(B, L, n, Hq, Hkv, D, seed=24, dtype="bf16")
    a = G.run_sfa(ins, n, LOCAL, D ** -0.5, window=200)
    b = G.run_sfa(ins, n, LOCAL, D ** -0.5, window=200)
    for name in ("o", "lse", "dq", "dk", "dv"):
        assert a[name].cpu().equal(b[name].cpu()), name
