"""ctypes binding of libhd.so: the C ABI of include/hd.h, argument marshalling only.

Each ``hd_*`` function here has the name and argument order of its C counterpart;
tensors stand in for device pointers (``torch.Tensor`` on the GPU; plain ints are
accepted as raw addresses).  All computation happens in the HIP kernels of libhd.so.
If the library is missing, every call raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhd.so")

HD_OK, HD_ERR_INVALID_ARG, HD_ERR_UNSUPPORTED, HD_ERR_HIP = 0, 1, 2, 3
HD_SFA_INTRA, HD_SFA_MIX, HD_SFA_LOCAL = 0, 1, 2
HD_DTYPE_BF16, HD_DTYPE_F32 = 0, 1

# every symbol include/hd.h declares
EXPORTS = ("hd_expand_embed", "hd_expand_embed_bwd_workspace_bytes", "hd_expand_embed_bwd",
           "hd_embed_grad_scatter_add", "hd_cyclic_replicate", "hd_sfa_fwd_final",
           "hd_sfa_bwd_final_workspace_bytes", "hd_sfa_bwd_final", "hd_sfa_decode_workspace_bytes",
           "hd_sfa_decode", "hd_sfa_decode_noalloc", "hd_sfa_decode_noalloc_max_bytes",
           "hd_final_stream_gather", "hd_final_stream_gather_bwd", "hd_sfa_fwd", "hd_sfa_fwd_local", "hd_sfa_bwd_workspace_bytes",
           "hd_sfa_bwd_local_workspace_bytes", "hd_sfa_bwd_min_workspace_bytes",
           "hd_sfa_bwd_local_min_workspace_bytes", "hd_sfa_bwd_final_min_workspace_bytes",
           "hd_sfa_bwd", "hd_sfa_bwd_local", "hd_status_str", "hd_last_error",
           "hd_timing_enable", "hd_timing_filter", "hd_timing_collect")


class HDError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"{_STATUS.get(status, status)}: {detail}")


_STATUS = {0: "HD_OK", 1: "HD_ERR_INVALID_ARG", 2: "HD_ERR_UNSUPPORTED", 3: "HD_ERR_HIP"}


class KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 64), ("launches", ctypes.c_int),
                ("total_ms", ctypes.c_double)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libhd.so (built in-tree by paper_2607_08186_amd.build); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                          "(there is no fallback implementation)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float
    sz = ctypes.c_size_t
    L.hd_expand_embed.argtypes = [vp, vp, vp, i32, i32, i32, i64, i32, i32, vp, vp]
    L.hd_sfa_fwd.argtypes = [vp, vp, vp, vp, vp] + [i32] * 7 + [f32, i32, vp]
    L.hd_sfa_bwd_workspace_bytes.argtypes = [i32] * 8
    L.hd_sfa_bwd_workspace_bytes.restype = sz
    L.hd_sfa_bwd_local_workspace_bytes.argtypes = [i32] * 8
    L.hd_sfa_bwd_local_workspace_bytes.restype = sz
    for f in (L.hd_sfa_bwd_min_workspace_bytes, L.hd_sfa_bwd_local_min_workspace_bytes,
              L.hd_sfa_bwd_final_min_workspace_bytes):
        f.argtypes = [i32] * 8
        f.restype = sz
    L.hd_sfa_bwd.argtypes = [vp] * 9 + [i32] * 7 + [f32, i32, vp, sz, vp]
    # the *_local variants take the window where the others take the mode
    L.hd_sfa_fwd_local.argtypes = L.hd_sfa_fwd.argtypes
    L.hd_sfa_bwd_local.argtypes = L.hd_sfa_bwd.argtypes
    L.hd_sfa_fwd_final.argtypes = L.hd_sfa_fwd.argtypes
    L.hd_sfa_bwd_final.argtypes = L.hd_sfa_bwd.argtypes
    L.hd_sfa_bwd_final_workspace_bytes.argtypes = [i32] * 8
    L.hd_sfa_bwd_final_workspace_bytes.restype = sz
    L.hd_sfa_decode_workspace_bytes.argtypes = [i32] * 9
    L.hd_sfa_decode_workspace_bytes.restype = sz
    L.hd_sfa_decode.argtypes = [vp, vp, vp, vp, i32, vp, vp] + [i32] * 8 + [f32, i32, vp, sz, vp]
    L.hd_sfa_decode_noalloc.argtypes = [vp, vp, vp, vp, i32, vp, vp] + [i32] * 8 + [f32, i32, vp]
    L.hd_sfa_decode_noalloc_max_bytes.argtypes = []
    L.hd_sfa_decode_noalloc_max_bytes.restype = sz
    L.hd_expand_embed_bwd_workspace_bytes.argtypes = [i32, i32]
    L.hd_expand_embed_bwd_workspace_bytes.restype = sz
    L.hd_expand_embed_bwd.argtypes = [vp, vp, i32, i32, i32, i64, i32, i32, vp, vp, vp, vp, sz, vp]
    L.hd_embed_grad_scatter_add.argtypes = [vp, vp, vp, i32, i32, i64, i32, vp, vp]
    L.hd_cyclic_replicate.argtypes = [vp, vp, i32, i32, i64, i32, i32, vp]
    L.hd_final_stream_gather.argtypes = [vp, vp] + [i32] * 5 + [vp]
    L.hd_final_stream_gather_bwd.argtypes = [vp, vp] + [i32] * 5 + [vp]
    for f in (L.hd_expand_embed, L.hd_expand_embed_bwd, L.hd_embed_grad_scatter_add,
              L.hd_cyclic_replicate, L.hd_final_stream_gather, L.hd_final_stream_gather_bwd,
              L.hd_sfa_fwd_final, L.hd_sfa_bwd_final, L.hd_sfa_decode, L.hd_sfa_decode_noalloc,
              L.hd_sfa_fwd,
              L.hd_sfa_fwd_local, L.hd_sfa_bwd,
              L.hd_sfa_bwd_local, L.hd_timing_enable, L.hd_timing_filter):
        f.restype = i32
    L.hd_status_str.argtypes = [i32]
    L.hd_status_str.restype = ctypes.c_char_p
    L.hd_last_error.argtypes = []
    L.hd_last_error.restype = ctypes.c_char_p
    L.hd_timing_enable.argtypes = [i32]
    L.hd_timing_filter.argtypes = [ctypes.c_char_p]
    L.hd_timing_collect.argtypes = [ctypes.POINTER(KernelTime), i32]
    L.hd_timing_collect.restype = i32
    _lib = L
    return L


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not x.is_cuda:
        raise ValueError("tensors passed to libhd must live on the GPU (device pointers)")
    if not x.is_contiguous():
        raise ValueError("tensors passed to libhd must be contiguous")
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _dtype_code(t, dtype):
    if dtype is not None:
        return int(dtype)
    import torch

    if t.dtype == torch.bfloat16:
        return HD_DTYPE_BF16
    if t.dtype == torch.float32:
        return HD_DTYPE_F32
    raise TypeError(f"unsupported tensor dtype {t.dtype}")


def _check(status: int):
    if status != HD_OK:
        raise HDError(status, lib().hd_last_error().decode())


def hd_expand_embed(ids, tables, out, B, L, n, V, Dm, dtype=None, bad_id_count=None,
                    stream=None):
    _check(lib().hd_expand_embed(_ptr(ids), _ptr(tables), _ptr(out), B, L, n, V, Dm,
                                 _dtype_code(tables, dtype), _ptr(bad_id_count),
                                 _stream(stream)))


def hd_expand_embed_bwd_workspace_bytes(B, L) -> int:
    return int(lib().hd_expand_embed_bwd_workspace_bytes(B, L))


def hd_expand_embed_bwd(ids, dout, B, L, n, V, Dm, uniq_ids, drows, num_uniq, workspace,
                        workspace_bytes, dtype=None, stream=None):
    _check(lib().hd_expand_embed_bwd(_ptr(ids), _ptr(dout), B, L, n, V, Dm,
                                     _dtype_code(dout, dtype), _ptr(uniq_ids), _ptr(drows),
                                     _ptr(num_uniq), _ptr(workspace), workspace_bytes,
                                     _stream(stream)))


def hd_embed_grad_scatter_add(uniq_ids, drows, num_uniq, max_rows, n, V, Dm, dtables,
                              stream=None):
    _check(lib().hd_embed_grad_scatter_add(_ptr(uniq_ids), _ptr(drows), _ptr(num_uniq), max_rows,
                                           n, V, Dm, _ptr(dtables), _stream(stream)))


def hd_cyclic_replicate(src, dst, n, m, V, Dm, dtype=None, stream=None):
    _check(lib().hd_cyclic_replicate(_ptr(src), _ptr(dst), n, m, V, Dm, _dtype_code(src, dtype),
                                     _stream(stream)))


def hd_final_stream_gather(h, out, B, L, n, Dm, dtype=None, stream=None):
    _check(lib().hd_final_stream_gather(_ptr(h), _ptr(out), B, L, n, Dm, _dtype_code(h, dtype),
                                        _stream(stream)))


def hd_final_stream_gather_bwd(dout, dh, B, L, n, Dm, dtype=None, stream=None):
    _check(lib().hd_final_stream_gather_bwd(_ptr(dout), _ptr(dh), B, L, n, Dm,
                                            _dtype_code(dout, dtype), _stream(stream)))


def hd_sfa_fwd(q, k, v, o, lse, B, L, n, Hq, Hkv, D, mode, scale, dtype=None, stream=None):
    _check(lib().hd_sfa_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, L, n, Hq, Hkv, D,
                            int(mode), float(scale), _dtype_code(q, dtype), _stream(stream)))


def hd_sfa_fwd_local(q, k, v, o, lse, B, L, n, Hq, Hkv, D, window, scale, dtype=None,
                     stream=None):
    _check(lib().hd_sfa_fwd_local(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, L, n, Hq,
                                  Hkv, D, int(window), float(scale), _dtype_code(q, dtype),
                                  _stream(stream)))


def hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, mode, dtype) -> int:
    return int(lib().hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, int(mode), int(dtype)))


def hd_sfa_bwd_min_workspace_bytes(B, L, n, Hq, Hkv, D, mode, dtype) -> int:
    return int(lib().hd_sfa_bwd_min_workspace_bytes(B, L, n, Hq, Hkv, D, int(mode), int(dtype)))


def hd_sfa_bwd_local_min_workspace_bytes(B, L, n, Hq, Hkv, D, window, dtype) -> int:
    return int(lib().hd_sfa_bwd_local_min_workspace_bytes(B, L, n, Hq, Hkv, D, int(window),
                                                          int(dtype)))


def hd_sfa_bwd_final_min_workspace_bytes(B, L, n, Hq, Hkv, D, window, dtype) -> int:
    return int(lib().hd_sfa_bwd_final_min_workspace_bytes(B, L, n, Hq, Hkv, D, int(window),
                                                          int(dtype)))


def hd_sfa_bwd_local_workspace_bytes(B, L, n, Hq, Hkv, D, window, dtype) -> int:
    return int(lib().hd_sfa_bwd_local_workspace_bytes(B, L, n, Hq, Hkv, D, int(window),
                                                      int(dtype)))


def hd_sfa_bwd(q, k, v, o, lse, dO, dq, dk, dv, B, L, n, Hq, Hkv, D, mode, scale, workspace,
               workspace_bytes, dtype=None, stream=None):
    _check(lib().hd_sfa_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(dO), _ptr(dq),
                            _ptr(dk), _ptr(dv), B, L, n, Hq, Hkv, D, int(mode), float(scale),
                            _dtype_code(q, dtype), _ptr(workspace), int(workspace_bytes),
                            _stream(stream)))


def hd_sfa_bwd_local(q, k, v, o, lse, dO, dq, dk, dv, B, L, n, Hq, Hkv, D, window, scale,
                     workspace, workspace_bytes, dtype=None, stream=None):
    _check(lib().hd_sfa_bwd_local(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(dO),
                                  _ptr(dq), _ptr(dk), _ptr(dv), B, L, n, Hq, Hkv, D, int(window),
                                  float(scale), _dtype_code(q, dtype), _ptr(workspace),
                                  int(workspace_bytes), _stream(stream)))


def hd_sfa_fwd_final(q, k, v, o, lse, B, L, n, Hq, Hkv, D, window, scale, dtype=None,
                     stream=None):
    _check(lib().hd_sfa_fwd_final(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, L, n, Hq,
                                  Hkv, D, int(window), float(scale), _dtype_code(q, dtype),
                                  _stream(stream)))


def hd_sfa_bwd_final_workspace_bytes(B, L, n, Hq, Hkv, D, window, dtype) -> int:
    return int(lib().hd_sfa_bwd_final_workspace_bytes(B, L, n, Hq, Hkv, D, int(window), int(dtype)))


def hd_sfa_bwd_final(q, k, v, o, lse, dO, dq, dk, dv, B, L, n, Hq, Hkv, D, window, scale,
                     workspace, workspace_bytes, dtype=None, stream=None):
    _check(lib().hd_sfa_bwd_final(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(dO),
                                  _ptr(dq), _ptr(dk), _ptr(dv), B, L, n, Hq, Hkv, D, int(window),
                                  float(scale), _dtype_code(q, dtype), _ptr(workspace),
                                  workspace_bytes, _stream(stream)))


def hd_sfa_decode_workspace_bytes(B, Lcap, n, Hq, Hkv, D, mode, window, max_ctx_tokens) -> int:
    return int(lib().hd_sfa_decode_workspace_bytes(B, Lcap, n, Hq, Hkv, D, int(mode), int(window),
                                                   int(max_ctx_tokens)))


def hd_sfa_decode(q, k_cache, v_cache, ctx_tokens, max_ctx_tokens, o, lse, B, Lcap, n, Hq, Hkv, D,
                  mode, window, scale, workspace, workspace_bytes, dtype=None, stream=None):
    _check(lib().hd_sfa_decode(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(ctx_tokens),
                               int(max_ctx_tokens), _ptr(o), _ptr(lse), B, Lcap, n, Hq, Hkv, D,
                               int(mode), int(window), float(scale), _dtype_code(q, dtype),
                               _ptr(workspace), workspace_bytes, _stream(stream)))


def hd_sfa_decode_noalloc(q, k_cache, v_cache, ctx_tokens, max_ctx_tokens, o, lse, B, Lcap, n,
                          Hq, Hkv, D, mode, window, scale, dtype=None, stream=None):
    _check(lib().hd_sfa_decode_noalloc(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(ctx_tokens),
                                       int(max_ctx_tokens), _ptr(o), _ptr(lse), B, Lcap, n, Hq,
                                       Hkv, D, int(mode), int(window), float(scale),
                                       _dtype_code(q, dtype), _stream(stream)))


def hd_sfa_decode_noalloc_max_bytes() -> int:
    return int(lib().hd_sfa_decode_noalloc_max_bytes())


def hd_timing_enable(enable: bool):
    _check(lib().hd_timing_enable(1 if enable else 0))


def hd_timing_filter(prefix: str | None = None):
    """Time only kernels whose timing name starts with `prefix` (None or "": all)."""
    _check(lib().hd_timing_filter(prefix.encode() if prefix else None))


def hd_timing_collect(max_entries: int = 64):
    """-> list of (kernel name, launches, total ms) accumulated since the last collect."""
    buf = (KernelTime * max_entries)()
    n = lib().hd_timing_collect(buf, max_entries)
    if n < 0:
        raise HDError(HD_ERR_HIP, lib().hd_last_error().decode())
    return [(buf[i].name.decode(), buf[i].launches, buf[i].total_ms) for i in range(n)]


# ---------------------------------------------------------------- conveniences
# Shape inference and output allocation through torch (device memory plumbing only).
# The softmax scale is a required argument, passed through unchanged.

def _shape(q, k, n):
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    if N % n:
        raise ValueError(f"expanded length {N} is not a multiple of n={n}")
    return B, N // n, Hq, Hkv, D


def sfa_forward(q, k, v, *, n, mode, scale, window=None, stream=None):
    """q [B][n*L][Hq][D], k/v [B][n*L][Hkv][D] -> (o, lse [B][Hq][n*L] fp32).
    ``window`` is required for, and only accepted with, mode HD_SFA_LOCAL."""
    import torch

    B, L, Hq, Hkv, D = _shape(q, k, n)
    o = torch.empty_like(q)
    lse = torch.empty((B, Hq, n * L), dtype=torch.float32, device=q.device)
    if _local(mode, window):
        hd_sfa_fwd_local(q, k, v, o, lse, B, L, n, Hq, Hkv, D, window, scale, stream=stream)
    else:
        hd_sfa_fwd(q, k, v, o, lse, B, L, n, Hq, Hkv, D, mode, scale, stream=stream)
    return o, lse


def _local(mode, window):
    if int(mode) == HD_SFA_LOCAL:
        if window is None:
            raise ValueError("mode HD_SFA_LOCAL needs a window")
        return True
    if window is not None:
        raise ValueError("a window is only meaningful with mode HD_SFA_LOCAL")
    return False


def sfa_backward(q, k, v, o, lse, dO, *, n, mode, scale, window=None, workspace=None,
                 workspace_bytes=None, stream=None):
    """-> (dq, dk, dv).  A workspace tensor (uint8, 256-byte aligned) may be passed in;
    otherwise one of ``workspace_bytes`` bytes is allocated (default: the one-pass
    size; anything down to the minimum size runs the backward in query bands)."""
    import torch

    B, L, Hq, Hkv, D = _shape(q, k, n)
    dtype = _dtype_code(q, None)
    if _local(mode, window):
        need = hd_sfa_bwd_local_workspace_bytes(B, L, n, Hq, Hkv, D, window, dtype)
    else:
        need = hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, mode, dtype)
    if workspace is None:
        workspace = torch.empty(need if workspace_bytes is None else int(workspace_bytes),
                                dtype=torch.uint8, device=q.device)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    if _local(mode, window):
        hd_sfa_bwd_local(q, k, v, o, lse, dO, dq, dk, dv, B, L, n, Hq, Hkv, D, window, scale,
                         workspace, workspace.numel(), stream=stream)
    else:
        hd_sfa_bwd(q, k, v, o, lse, dO, dq, dk, dv, B, L, n, Hq, Hkv, D, mode, scale, workspace,
                   workspace.numel(), stream=stream)
    return dq, dk, dv


def expand_embed(ids, tables, *, bad_id_count=None, stream=None):
    """ids [B][L] int32, tables [n][V][Dm] -> out [B][n*L][Dm]."""
    import torch

    B, L = ids.shape
    n, V, Dm = tables.shape
    out = torch.empty((B, n * L, Dm), dtype=tables.dtype, device=tables.device)
    hd_expand_embed(ids, tables, out, B, L, n, V, Dm, bad_id_count=bad_id_count, stream=stream)
    return out


def expand_embed_backward(ids, dout, V, *, stream=None):
    """Gradient of the expansion w.r.t. the tables, sparse: ids [B][L] int32, dout
    [B][n*L][Dm] -> (uniq_ids [B*L] int32, drows [n][B*L][Dm] fp32, num_uniq [1] int32),
    all device tensors; only the first num_uniq ids / rows are defined."""
    import torch

    B, L = ids.shape
    N, Dm = dout.shape[1], dout.shape[2]
    if N % L:
        raise ValueError("dout must be [B][n*L][Dm]")
    n = N // L
    dev = dout.device
    uniq = torch.empty(B * L, dtype=torch.int32, device=dev)
    drows = torch.empty((n, B * L, Dm), dtype=torch.float32, device=dev)
    num = torch.empty(1, dtype=torch.int32, device=dev)
    need = hd_expand_embed_bwd_workspace_bytes(B, L)
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    hd_expand_embed_bwd(ids, dout, B, L, n, V, Dm, uniq, drows, num, ws, need, stream=stream)
    return uniq, drows, num


def cyclic_replicate(tables, m, *, stream=None):
    """eq. (cyclic_init): tables [n][V][Dm] -> new [m][V][Dm] with table s = tables[s mod n]."""
    import torch

    n, V, Dm = tables.shape
    out = torch.empty((m, V, Dm), dtype=tables.dtype, device=tables.device)
    hd_cyclic_replicate(tables, out, n, m, V, Dm, stream=stream)
    return out


def final_stream_gather(h, n, *, stream=None):
    """eq. (hd_loss) input: h [B][n*L][Dm] -> new [B][L][Dm], row i = h[i*n + n - 1]."""
    import torch

    B, N, Dm = h.shape
    if N % n:
        raise ValueError("h must hold n*L expanded rows")
    out = torch.empty((B, N // n, Dm), dtype=h.dtype, device=h.device)
    hd_final_stream_gather(h, out, B, N // n, n, Dm, stream=stream)
    return out


def final_stream_gather_backward(dout, n, *, stream=None):
    """Adjoint: dout [B][L][Dm] -> new dh [B][n*L][Dm], zero off the final-stream rows."""
    import torch

    B, L, Dm = dout.shape
    dh = torch.empty((B, n * L, Dm), dtype=dout.dtype, device=dout.device)
    hd_final_stream_gather_bwd(dout, dh, B, L, n, Dm, stream=stream)
    return dh


def sfa_final_forward(q, k, v, *, n, scale, window=0, stream=None):
    """Final-stream layer: q [B][L][Hq][D] (final-stream rows), k/v [B][n*L][Hkv][D] ->
    (o [B][L][Hq][D], lse [B][Hq][L] fp32).  window 0: full cross-stream mask."""
    import torch

    B, L, Hq, D = q.shape
    Hkv = k.shape[2]
    if k.shape[1] != n * L:
        raise ValueError("k/v must hold n*L expanded rows")
    o = torch.empty_like(q)
    lse = torch.empty((B, Hq, L), dtype=torch.float32, device=q.device)
    hd_sfa_fwd_final(q, k, v, o, lse, B, L, n, Hq, Hkv, D, window, scale, stream=stream)
    return o, lse


def sfa_final_backward(q, k, v, o, lse, dO, *, n, scale, window=0, workspace=None,
                       workspace_bytes=None, stream=None):
    """-> (dq [B][L][Hq][D], dk, dv [B][n*L][Hkv][D]).  Workspace as for sfa_backward."""
    import torch

    B, L, Hq, D = q.shape
    Hkv = k.shape[2]
    need = hd_sfa_bwd_final_workspace_bytes(B, L, n, Hq, Hkv, D, window, _dtype_code(q, None))
    if workspace is None:
        workspace = torch.empty(need if workspace_bytes is None else int(workspace_bytes),
                                dtype=torch.uint8, device=q.device)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    hd_sfa_bwd_final(q, k, v, o, lse, dO, dq, dk, dv, B, L, n, Hq, Hkv, D, window, scale,
                     workspace, workspace.numel(), stream=stream)
    return dq, dk, dv


def sfa_decode(q, k_cache, v_cache, ctx_tokens, *, max_ctx, mode, scale, window=0,
               workspace=None, stream=None):
    """Parallel-stream decode: q [B][n][Hq][D] (the new token's n streams), caches
    [B][n*Lcap][Hkv][D], ctx_tokens [B] int32 (device) -> (o [B][n][Hq][D],
    lse [B][Hq][n] fp32)."""
    import torch

    B, n, Hq, D = q.shape
    Lcap = k_cache.shape[1] // n
    Hkv = k_cache.shape[2]
    need = hd_sfa_decode_workspace_bytes(B, Lcap, n, Hq, Hkv, D, mode, window, max_ctx)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    o = torch.empty_like(q)
    lse = torch.empty((B, Hq, n), dtype=torch.float32, device=q.device)
    hd_sfa_decode(q, k_cache, v_cache, ctx_tokens, max_ctx, o, lse, B, Lcap, n, Hq, Hkv, D, mode,
                  window, scale, workspace, workspace.numel(), stream=stream)
    return o, lse
