"""The allocation-free parallel-stream decode (hd_sfa_decode_noalloc), through the C ABI,
against hd_sfa_decode with a caller workspace: the same kernels, so o and lse must agree
bit for bit.  Two calls in a row share the library's scratch, the second one smaller
than the first (its partials cover a prefix of what the first one left there), then a
local layer; each is compared with its own reference call."""
import numpy as np
import pytest
import torch

import paper_2607_08186_amd as hd
from paper_2607_08186_amd import synth
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

INTRA, MIX, LOCAL = 0, 1, 2


def _case(seed, B, Lcap, n, Hq, Hkv, D, mode, window, ctx):
    dev = G.dev()
    q = synth.device_normal((B, n, Hq, D), 2 ** -0.5, seed, dev, torch.bfloat16)
    k = synth.device_normal((B, n * Lcap, Hkv, D), 2 ** -0.5, seed + 1, dev, torch.bfloat16)
    v = synth.device_normal((B, n * Lcap, Hkv, D), 2 ** -0.5, seed + 2, dev, torch.bfloat16)
    tctx = torch.tensor(ctx, dtype=torch.int32, device=dev)
    max_ctx = int(max(ctx))
    scale = D ** -0.5
    o_ref, lse_ref = torch.empty_like(q), torch.empty((B, Hq, n), dtype=torch.float32, device=dev)
    need = hd.hd_sfa_decode_workspace_bytes(B, Lcap, n, Hq, Hkv, D, mode, window, max_ctx)
    assert 0 < need <= hd.hd_sfa_decode_noalloc_max_bytes()
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    hd.hd_sfa_decode(q, k, v, tctx, max_ctx, o_ref, lse_ref, B, Lcap, n, Hq, Hkv, D, mode, window,
                     scale, ws, need)
    o, lse = torch.empty_like(q), torch.empty_like(lse_ref)
    hd.hd_sfa_decode_noalloc(q, k, v, tctx, max_ctx, o, lse, B, Lcap, n, Hq, Hkv, D, mode, window,
                             scale)
    torch.cuda.synchronize()
    return (G.bits(o), lse.cpu().numpy()), (G.bits(o_ref), lse_ref.cpu().numpy())


def _check(got, ref, what):
    (o, lse), (o_ref, lse_ref) = got, ref
    assert np.array_equal(o, o_ref), f"{what}: o differs in {np.count_nonzero(o != o_ref)} places"
    assert np.array_equal(lse.view(np.uint32), lse_ref.view(np.uint32)), f"{what}: lse differs"


def test_noalloc_decode_matches_the_workspace_entry_point():
    # 1: the serving shape (16 sequences, up to 4096 tokens, full cross-stream layer):
    #    65 MiB of partials, about half the scratch
    ctx1 = [4095, 4000, 3333, 17, 0, 4095, 2048, 1, 4094, 1000, 3999, 2500, 100, 4095, 7, 512]
    print("noalloc call 1: B=16 Lcap=4096 n=4 MIX", flush=True)
    got, ref = _case(synth.seed_for("noalloc", 1), 16, 4096, 4, 32, 8, 128, MIX, 0, ctx1)
    _check(got, ref, "call 1")
    # 2: a smaller intra-stream call right after it (stale partials of call 1 remain)
    print("noalloc call 2: B=3 Lcap=700 n=2 INTRA", flush=True)
    got, ref = _case(synth.seed_for("noalloc", 2), 3, 700, 2, 8, 2, 64, INTRA, 0, [699, 5, 300])
    _check(got, ref, "call 2")
    # 3: a local layer at D=32
    print("noalloc call 3: B=2 Lcap=900 n=3 LOCAL w=100", flush=True)
    got, ref = _case(synth.seed_for("noalloc", 3), 2, 900, 3, 4, 1, 32, LOCAL, 100, [899, 40])
    _check(got, ref, "call 3")


def test_noalloc_decode_rejects_oversize():
    """Partials beyond the scratch: an error, nothing enqueued."""
    dev = G.dev()
    q = torch.zeros((32, 4, 32, 128), dtype=torch.bfloat16, device=dev)
    kc = torch.zeros((32, 4 * 4096, 8, 128), dtype=torch.bfloat16, device=dev)  # full size
    ctx = torch.zeros(32, dtype=torch.int32, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty((32, 32, 4), dtype=torch.float32, device=dev)
    need = hd.hd_sfa_decode_workspace_bytes(32, 4096, 4, 32, 8, 128, MIX, 0, 4095)
    assert need > hd.hd_sfa_decode_noalloc_max_bytes()
    with pytest.raises(hd.binding.HDError):
        hd.hd_sfa_decode_noalloc(q, kc, kc, ctx, 4095, o, lse, 32, 4096, 4, 32, 8, 128, MIX, 0,
                                 128 ** -0.5)
