"""Full-size parity in the launch configuration the benchmark times.

At these sizes the oracle evaluates sampled rows one by one: forward rows, dQ rows,
and dK/dV rows of sampled keys.  The keys come from one key/value head and, where the
oracle's cost allows it (it forms every query row that sees a listed key, once for all
of them), span the whole sequence: the first key of a stream, which every query of the
stream sees, a key of the first 128-key block, one of the middle block, and the last
keys; elsewhere (the mixing layers at N >= 16384) the keys of the last tokens.
Properties that hold at any size check the rest: the gradient sums of softmax attention
(sum over keys of dV is the group's summed dO; sum over keys of dK is zero), per stream
for intra layers.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2607_08186_amd import synth, workloads
from tests import gpu_helpers as G

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

INTRA, MIX, LOCAL = 0, 1, 2
# The dQ launch picks its LDS ring by grid size: the n=1 sweep shapes (512 workgroups,
# two per CU on 256 CUs) take the one-workgroup-per-CU ring, the others the ring that
# puts two workgroups on a CU, so both are checked here at full size.
CASES = [workloads.QWEN8B, *workloads.SWEEP, workloads.FRONTIER]


def _sample_rows(rng, B, H, N, count):
    rows = {(0, 0, 0), (B - 1, H - 1, N - 1), (0, H - 1, N // 2), (B - 1, 0, 1)}
    while len(rows) < count:
        rows.add((int(rng.integers(B)), int(rng.integers(H)), int(rng.integers(N))))
    return np.array(sorted(rows), dtype=np.int64)


def _key_rows(rng, s, mode, window):
    """Sampled key rows (b, hk, j) of one key/value head, split into the keys that many
    queries see (compared together) and the last keys (compared together)."""
    b, hk = int(rng.integers(s.B)), int(rng.integers(s.Hkv))
    G = s.Hq // s.Hkv
    # oracle cost of a key near the start: every query row that sees it, each formed in
    # full (about 3D flop per visible pair)
    if mode == INTRA:
        heavy_cost = 2 * G * s.L * s.L / 2 * 3 * s.D      # two streams' first keys
    elif mode == LOCAL:
        w = min(window, s.N)
        heavy_cost = G * w * w * 3 * s.D
    else:
        heavy_cost = G * s.N * s.N / 2 * 3 * s.D
    tail = {(b, hk, int(j)) for j in (s.N - 1, s.N - 2, s.N - s.n - 1)}
    tail.add((b, hk, int(rng.integers(max(0, s.N - 2 * s.n), s.N))))
    heavy = set()
    if heavy_cost <= 6e10:
        if mode == INTRA:  # stream 0 and stream n-1: first key, one of the first 128 tokens,
            for st in {0, s.n - 1}:  # one of the middle block
                heavy |= {(b, hk, st), (b, hk, int(rng.integers(1, 128)) * s.n + st),
                          (b, hk, (s.L // 2 + int(rng.integers(128))) * s.n + st)}
        else:
            heavy |= {(b, hk, 0), (b, hk, 1), (b, hk, int(rng.integers(2, 128))),
                      (b, hk, s.N // 2 + int(rng.integers(128)))}
    return (np.array(sorted(heavy), dtype=np.int64).reshape(-1, 3),
            np.array(sorted(tail), dtype=np.int64))


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

    heavy, tail = _key_rows(rng, s, mode, window or 0)
    dk = G.to_host64(got["dk"])
    dv = G.to_host64(got["dv"])
    if wl is workloads.QWEN8B and mode != MIX:
        assert len(heavy), "the Qwen3-8B-like intra and local layers check keys near the start"
    for what, krows in (("heavy keys", heavy), ("last keys", tail)):
        if not len(krows):
            continue
        print(f"  dK/dV of {what}: {krows.tolist()}", flush=True)
        rdk, rdv = oracle.sfa_bwd_dkdv_rows(ins["q"], ins["k"], ins["v"], ins["dout"], krows,
                                            **kw)
        b, h, j = krows.T
        G.assert_close_grad(dk[b, j, h], rdk, "bf16", "dk", f"{wl.name} {what}")
        G.assert_close_grad(dv[b, j, h], rdv, "bf16", "dv", f"{wl.name} {what}")

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


_SLICE_LIMIT = {}


def _slice_limit_inputs(N, Hq, Hkv, D):
    """Seeded inputs of the slice-limit shape, drawn once for all tests here: q, k, v
    ~ N(0, 1/2) and dO ~ N(0, 1) from torch's seeded device generator (a host draw of
    10^9 normals takes minutes), rounded to bf16; the oracle reads host copies of the
    same tensors."""
    if not _SLICE_LIMIT:
        import torch

        seed = synth.seed_for("slice_limit")
        t = {name: synth.device_normal((1, N, h, D), std, seed + i, G.dev(), torch.bfloat16)
             for i, (name, h, std) in enumerate((("q", Hq, 2 ** -0.5), ("k", Hkv, 2 ** -0.5),
                                                 ("v", Hkv, 2 ** -0.5), ("dout", Hq, 1.0)))}
        _SLICE_LIMIT.update(seed=seed, dev=t, **{name: G.bits(x) for name, x in t.items()})
    return _SLICE_LIMIT


@pytest.mark.parametrize("mode", [INTRA, MIX], ids=["intra", "mix"])
def test_forward_at_the_slice_limit(mode):
    """q and o as large as the boundary accepts: B=1, L=32752, n=4 (N=131008), Hq=64,
    Hkv=8, D=128 puts 2146435072 bytes of q in the batch slice, just under the 2^31 bytes
    that the kernels' 32-bit buffer offsets address.  Sampled rows, among them the last
    rows of the sequence in the last head, against the oracle."""
    B, L, n, Hq, Hkv, D = 1, 32752, 4, 64, 8, 128
    N = n * L
    assert N * Hq * D * 2 < 2 ** 31 <= (N + 64) * Hq * D * 2
    print(f"slice limit mode={mode} N={N} Hq={Hq}: drawing inputs", flush=True)
    ins = _slice_limit_inputs(N, Hq, Hkv, D)
    seed, q, k, v = ins["seed"], ins["q"], ins["k"], ins["v"]
    print(f"slice limit mode={mode} seed={seed}: forward", flush=True)
    import paper_2607_08186_amd as hd
    import torch

    o, lse = hd.sfa_forward(*(ins["dev"][x] for x in "qkv"), n=n, mode=mode, scale=D ** -0.5)
    torch.cuda.synchronize()
    rng = np.random.default_rng((seed + mode) & 0xFFFFFFFF)
    rows = {(0, Hq - 1, N - 1), (0, 0, N - 1), (0, Hq - 1, N - 2), (0, 31, N - 5), (0, 0, 0)}
    while len(rows) < 24:
        rows.add((0, int(rng.integers(Hq)), int(rng.integers(N - 2048, N))))
    while len(rows) < 40:
        rows.add((0, int(rng.integers(Hq)), int(rng.integers(N))))
    rows = np.array(sorted(rows), dtype=np.int64)
    ro, rl = oracle.sfa_fwd_rows(q, k, v, rows, L=L, n=n, mode=mode, scale=D ** -0.5)
    b, h, p = (torch.as_tensor(x, device=o.device) for x in rows.T)
    oh = G.to_host64(o[b, p, h])
    lh = G.to_host64(lse[b, h, p])
    G.assert_close_fwd(oh, lh, ro, rl, "bf16", "slice limit")


@pytest.mark.parametrize("mode", [INTRA, MIX], ids=["intra", "mix"])
def test_backward_at_the_slice_limit(mode):
    """The backward at the same length.  Its one-pass dS workspace would be about 0.27 TB
    (intra-stream) or 1.1 TB (mixing), so it runs in query bands with a 24 GiB
    workspace.  Sampled dQ rows and dK/dV of the last keys (which only the last rows
    see, so the oracle can form them) against the oracle; the gradient sums over all
    keys (sum of dV = the group's summed dO, sum of dK = 0, per stream for intra)."""
    import paper_2607_08186_amd as hd
    import torch

    B, L, n, Hq, Hkv, D = 1, 32752, 4, 64, 8, 128
    N = n * L
    scale = D ** -0.5
    ws_bytes = 24 << 30
    low = hd.hd_sfa_bwd_min_workspace_bytes(B, L, n, Hq, Hkv, D, mode, hd.HD_DTYPE_BF16)
    full = hd.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, mode, hd.HD_DTYPE_BF16)
    assert low <= ws_bytes < full
    print(f"slice limit backward mode={mode}: drawing inputs", flush=True)
    ins = _slice_limit_inputs(N, Hq, Hkv, D)
    seed = ins["seed"]
    q, k, v, do = (ins["dev"][x] for x in ("q", "k", "v", "dout"))
    print(f"slice limit backward mode={mode} seed={seed}: forward + backward in bands",
          flush=True)
    o, lse = hd.sfa_forward(q, k, v, n=n, mode=mode, scale=scale)
    dq, dk, dv = hd.sfa_backward(q, k, v, o, lse, do, n=n, mode=mode, scale=scale,
                                 workspace_bytes=ws_bytes)
    torch.cuda.synchronize()
    del o, lse
    rng = np.random.default_rng((seed + 7 * mode) & 0xFFFFFFFF)
    rows = {(0, Hq - 1, N - 1), (0, 0, N - 1), (0, 17, N - 3), (0, 0, 0), (0, 40, 1)}
    while len(rows) < 16:
        rows.add((0, int(rng.integers(Hq)), int(rng.integers(N - 1024, N))))
    while len(rows) < 24:
        rows.add((0, int(rng.integers(Hq)), int(rng.integers(N))))
    rows = np.array(sorted(rows), dtype=np.int64)
    kw = dict(L=L, n=n, mode=mode, scale=scale)
    print(f"  oracle dQ rows: {len(rows)}", flush=True)
    rdq = oracle.sfa_bwd_dq_rows(ins["q"], ins["k"], ins["v"], ins["dout"], rows, **kw)
    b, h, p = (torch.as_tensor(x, device=dq.device) for x in rows.T)
    G.assert_close_grad(G.to_host64(dq[b, p, h]), rdq, "bf16", "dq", "slice limit backward")
    hk = int(rng.integers(Hkv))
    keys = np.array(sorted({(0, hk, N - 1), (0, hk, N - 2), (0, hk, N - n - 1),
                            (0, Hkv - 1 - hk, N - 3)}), dtype=np.int64)
    print(f"  oracle dK/dV keys: {keys.tolist()}", flush=True)
    rdk, rdv = oracle.sfa_bwd_dkdv_rows(ins["q"], ins["k"], ins["v"], ins["dout"], keys, **kw)
    b, h, j = (torch.as_tensor(x, device=dk.device) for x in keys.T)
    G.assert_close_grad(G.to_host64(dk[b, j, h]), rdk, "bf16", "dk", "slice limit backward")
    G.assert_close_grad(G.to_host64(dv[b, j, h]), rdv, "bf16", "dv", "slice limit backward")
    # gradient sums, in fp64 on the device
    Gq = Hq // Hkv
    dof = do.double()
    groups = [slice(None)] if mode != INTRA else [slice(st, None, n) for st in range(n)]
    for sl in groups:
        want = dof[:, sl].reshape(B, -1, Hkv, Gq, D).sum(dim=(1, 3))
        dvs, dks = dv[:, sl].double(), dk[:, sl].double()
        assert torch.all((dvs.sum(dim=1) - want).abs() <= 1e-2 * dvs.abs().sum(dim=1) + 1e-3), \
            "sum_j dV_j != sum dO"
        assert torch.all(dks.sum(dim=1).abs() <= 1e-2 * dks.abs().sum(dim=1) + 1e-3), "sum_j dK_j != 0"
    assert bool(torch.isfinite(dq).all()) and bool(torch.isfinite(dk).all())
