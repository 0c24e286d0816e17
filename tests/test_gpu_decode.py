"""GPU parity of the parallel-stream decode (the n streams of each sequence's new token
against its cached prefix) with the fp64 oracle.  bf16 tolerances as for the other
forward paths: max |O - O_ref| <= 2e-2 and max |lse - lse_ref| <= 2e-2."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_08186_amd as hd
from paper_2607_08186_amd import synth, workloads
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

INTRA, MIX, LOCAL = 0, 1, 2


def _inputs(seed, B, Lcap, n, Hq, Hkv, D, std=2 ** -0.5):
    to = synth.to_bf16_bits
    return dict(q=to(synth.normal(seed, (B, n, Hq, D), std)),
                k=to(synth.normal(seed + 1, (B, n * Lcap, Hkv, D), std)),
                v=to(synth.normal(seed + 2, (B, n * Lcap, Hkv, D), std)))


def _run(ins, ctx, mode, window, max_ctx=None):
    q, k, v = (G.to_dev(ins[x]) for x in ("q", "k", "v"))
    tctx = torch.from_numpy(np.asarray(ctx, dtype=np.int32)).to(G.dev())
    max_ctx = int(np.max(ctx)) if max_ctx is None else max_ctx
    o, lse = hd.sfa_decode(q, k, v, tctx, max_ctx=max_ctx, mode=mode, window=window,
                           scale=q.shape[-1] ** -0.5)
    torch.cuda.synchronize()
    return G.to_host64(o), G.to_host64(lse)


# B, Lcap, n, Hq, Hkv, D, mode, window, contexts (tokens before the new one)
CASES = [
    (3, 300, 4, 32, 8, 128, MIX, 0, [0, 299, 137]),     # ragged contexts, 16 query slots
    (2, 100, 4, 32, 8, 128, INTRA, 0, [57, 99]),
    (2, 200, 2, 8, 2, 64, LOCAL, 50, [199, 10]),
    (1, 513, 8, 64, 8, 128, MIX, 0, [512]),             # 64 query rows per group: 2 chunks
    (2, 64, 1, 4, 4, 32, MIX, 0, [63, 0]),              # n = 1, one head per group
    (1, 40, 3, 6, 2, 64, MIX, 0, [39]),                 # 9 query slots
    (4, 70, 4, 16, 2, 128, INTRA, 0, [0, 1, 2, 69]),
    (2, 90, 4, 8, 2, 128, LOCAL, 1, [89, 30]),          # window 1: each row sees only itself
    (1, 129, 2, 4, 1, 128, LOCAL, 200, [128]),          # window beyond the context
]


@pytest.mark.parametrize("case", CASES, ids=[str(c[:8]) + str(c[8]) for c in CASES])
def test_decode_parity(case):
    B, Lcap, n, Hq, Hkv, D, mode, w, ctx = case
    seed = synth.seed_for("decode", str(case))
    print(f"decode case={case} seed={seed}", flush=True)
    ins = _inputs(seed, B, Lcap, n, Hq, Hkv, D)
    o, lse = _run(ins, ctx, mode, w)
    ro, rl = oracle.sfa_decode(ins["q"], ins["k"], ins["v"], ctx, n=n, mode=mode,
                               scale=D ** -0.5, window=w)
    G.assert_close_fwd(o, lse, ro, rl, "bf16", str(case))


def test_decode_grid_bound_above_the_contexts():
    """max_ctx_tokens larger than every context: the extra cache chunks are skipped."""
    B, Lcap, n, Hq, Hkv, D = 2, 600, 4, 32, 8, 128
    ins = _inputs(synth.seed_for("decode_bound"), B, Lcap, n, Hq, Hkv, D)
    ctx = [100, 3]
    a = _run(ins, ctx, MIX, 0)
    b = _run(ins, ctx, MIX, 0, max_ctx=Lcap - 1)
    ro, rl = oracle.sfa_decode(ins["q"], ins["k"], ins["v"], ctx, n=n, mode=MIX, scale=D ** -0.5)
    G.assert_close_fwd(b[0], b[1], ro, rl, "bf16", "bound")
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


@pytest.mark.parametrize("mode,w", [(MIX, 0), (INTRA, 0), (LOCAL, 33)])
def test_decode_never_reads_past_the_new_token(mode, w):
    """Cache rows past ctx*n + n - 1 hold huge values: the outputs are unchanged."""
    B, Lcap, n, Hq, Hkv, D = 2, 200, 4, 8, 2, 128
    ins = _inputs(synth.seed_for("decode_poison", mode), B, Lcap, n, Hq, Hkv, D)
    ctx = [77, 150]
    base = _run(ins, ctx, mode, w)
    bad = dict(ins)
    for name in ("k", "v"):
        arr = ins[name].copy()
        for b in range(B):
            arr[b, (ctx[b] + 1) * n:] = synth.to_bf16_bits(np.full_like(
                arr[b, (ctx[b] + 1) * n:], 3.0e4, dtype=np.float64))
        bad[name] = arr
    got = _run(bad, ctx, mode, w)
    np.testing.assert_array_equal(base[0], got[0])
    np.testing.assert_array_equal(base[1], got[1])


def test_decode_intra_reads_only_its_stream():
    B, Lcap, n, Hq, Hkv, D = 1, 120, 4, 8, 2, 64
    ins = _inputs(synth.seed_for("decode_intra_poison"), B, Lcap, n, Hq, Hkv, D)
    ctx = [119]
    base = _run(ins, ctx, INTRA, 0)
    bad = dict(ins)
    for name in ("k", "v"):
        arr = ins[name].copy()
        arr[:, 2::n] = synth.to_bf16_bits(np.full_like(arr[:, 2::n], 3.0e4, dtype=np.float64))
        bad[name] = arr
    got = _run(bad, ctx, INTRA, 0)
    keep = [s for s in range(n) if s != 2]
    np.testing.assert_array_equal(base[0][:, keep], got[0][:, keep])
    np.testing.assert_array_equal(base[1][:, :, keep], got[1][:, :, keep])


@pytest.mark.slow
@pytest.mark.parametrize("mode", [MIX, INTRA], ids=["mix", "intra"])
def test_decode_fullsize_batch(mode):
    """16 sequences of up to 4096 tokens at the Qwen3-8B-like head layout (n=4, Hq=32,
    Hkv=8, D=128); three sequences checked against the oracle, all rows finite."""
    s = workloads.QWEN8B.shape
    B, Lcap = 16, s.L
    seed = synth.seed_for("decode_full", mode)
    ins = _inputs(seed, B, Lcap, s.n, s.Hq, s.Hkv, s.D)
    ctx = np.random.default_rng(seed).integers(1, Lcap, size=B)
    ctx[0], ctx[1] = Lcap - 1, 0
    print(f"decode fullsize mode={mode} seed={seed}", flush=True)
    o, lse = _run(ins, ctx, mode, 0)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    pick = [0, 1, 7]
    ro, rl = oracle.sfa_decode(ins["q"][pick], ins["k"][pick], ins["v"][pick], ctx[pick],
                               n=s.n, mode=mode, scale=s.scale)
    G.assert_close_fwd(o[pick], lse[pick], ro, rl, "bf16", "decode fullsize")


@pytest.mark.slow
@pytest.mark.parametrize("mode", [MIX, INTRA], ids=["mix", "intra"])
def test_decode_at_the_cache_slice_limit(mode):
    """Each sequence's cache as large as the boundary accepts: Lcap=262143 tokens of n=4
    streams at Hkv=8, D=128 is 2147475456 bytes per sequence for K (and for V), the
    largest below the 2^31 bytes that the kernels' 32-bit buffer offsets address; two sequences,
    so the second one's slice starts past 2 GiB.  Contexts at the capacity and mid-way,
    checked against the oracle.  The caches come from torch's seeded device generator
    (a host draw of 2 x 10^9 normals takes minutes); the oracle reads host copies."""
    B, Lcap, n, Hq, Hkv, D = 2, 262143, 4, 32, 8, 128
    assert n * Lcap * Hkv * D * 2 < 2 ** 31 <= n * (Lcap + 1) * Hkv * D * 2
    seed = synth.seed_for("decode_slice_limit", mode)
    print(f"decode slice limit mode={mode} Lcap={Lcap} seed={seed}", flush=True)
    dev = G.dev()
    q = synth.device_normal((B, n, Hq, D), 2 ** -0.5, seed, dev, torch.bfloat16)
    k = synth.device_normal((B, n * Lcap, Hkv, D), 2 ** -0.5, seed + 1, dev, torch.bfloat16)
    v = synth.device_normal((B, n * Lcap, Hkv, D), 2 ** -0.5, seed + 2, dev, torch.bfloat16)
    ctx = np.array([Lcap - 1, 100003], dtype=np.int32)
    o, lse = hd.sfa_decode(q, k, v, torch.from_numpy(ctx).to(dev), max_ctx=Lcap - 1, mode=mode,
                           window=0, scale=D ** -0.5)
    torch.cuda.synchronize()
    print("decode slice limit: oracle", flush=True)
    ro, rl = oracle.sfa_decode(G.bits(q), G.bits(k), G.bits(v), ctx, n=n, mode=mode,
                               scale=D ** -0.5)
    G.assert_close_fwd(G.to_host64(o), G.to_host64(lse), ro, rl, "bf16", "decode slice limit")
