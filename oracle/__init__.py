"""Plain fp64 CPU oracle for the Hidden Decoding hot path -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and its
Python binding) never imports, links or calls it.

The arithmetic lives in ``sfa_oracle.c`` (fp64, explicit mask from the paper's
definitions: eq. (expansion), eq. (indices), eq. (mask_intra), the causal mask of
Fig. "masks"(a) and its sliding-window form of Fig. "masks"(b)).  This module only marshals numpy arrays through ctypes and
builds the shared object with gcc.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# HD_ORACLE_SRC / HD_ORACLE_LIB point the module at another build of the oracle (the
# mutation tests use them to check that the pins catch planted mistakes)
_SRC = os.environ.get("HD_ORACLE_SRC") or os.path.join(_HERE, "sfa_oracle.c")
_LIB = os.environ.get("HD_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

INTRA, MIX, LOCAL = 0, 1, 2
_F64, _F32, _BF16 = 0, 1, 2

_lib = None


def build() -> str:
    """Compile sfa_oracle.c into liboracle.so (plain gcc, no fast-math)."""
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-fPIC", "-shared", "-pthread",
           "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    i64, vp, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    dbl = ctypes.c_double
    dims = [i64] * 6 + [i32, i64, dbl, i32]  # B L n Hq Hkv D mode window scale nthreads
    lib.oracle_sfa_fwd.argtypes = [vp, vp, vp, i32, vp, vp] + dims
    lib.oracle_sfa_fwd_rows.argtypes = [vp, vp, vp, i32, vp, i64, vp, vp] + dims
    lib.oracle_sfa_bwd.argtypes = [vp, vp, vp, vp, i32, vp, vp, vp] + dims
    lib.oracle_sfa_bwd_dq_rows.argtypes = [vp, vp, vp, vp, i32, vp, i64, vp] + dims
    lib.oracle_sfa_bwd_dkdv_rows.argtypes = [vp, vp, vp, vp, i32, vp, i64, vp, vp] + dims
    for f in (lib.oracle_sfa_fwd, lib.oracle_sfa_fwd_rows, lib.oracle_sfa_bwd,
              lib.oracle_sfa_bwd_dq_rows, lib.oracle_sfa_bwd_dkdv_rows):
        f.restype = None
    lib.oracle_final_gather.argtypes = [vp, vp, i64, i64, i64, i64, i64]
    lib.oracle_final_gather.restype = None
    lib.oracle_final_gather_bwd.argtypes = [vp, vp, i64, i64, i64, i64, i64]
    lib.oracle_final_gather_bwd.restype = None
    lib.oracle_expand_embed.argtypes = [vp, vp, vp, i64, i64, i64, i64, i64, i64]
    lib.oracle_expand_embed.restype = i64
    lib.oracle_expand_embed_bwd.argtypes = [vp, vp, i32, vp, i64, i64, i64, i64, i64]
    lib.oracle_expand_embed_bwd.restype = None
    lib.oracle_expand_embed_bwd_rows.argtypes = [vp, vp, i32, vp, i64, vp, i64, i64, i64, i64,
                                                 i64]
    lib.oracle_expand_embed_bwd_rows.restype = None
    lib.oracle_cyclic_replicate.argtypes = [vp, vp, i64, i64, i64, i64, i64]
    lib.oracle_cyclic_replicate.restype = None
    lib.oracle_sfa_mask.argtypes = [vp, i64, i64, i32, i64]
    lib.oracle_sfa_mask.restype = None
    _lib = lib
    return lib


def default_threads() -> int:
    """Every thread this process may use: OMP_NUM_THREADS when set (shared GPU hosts
    set it to the CPU share of one GPU), else the CPUs of the affinity mask."""
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        return int(env)
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:
        return max(1, os.cpu_count() or 1)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float64:
        return _F64
    if a.dtype == np.float32:
        return _F32
    if a.dtype == np.uint16:  # bf16 bit patterns
        return _BF16
    raise TypeError(f"oracle inputs must be float64, float32 or uint16 (bf16 bits), got {a.dtype}")


def _prep(*arrays):
    out = [np.ascontiguousarray(a) for a in arrays]
    code = _dtype_code(out[0])
    for a in out[1:]:
        if _dtype_code(a) != code:
            raise TypeError("oracle inputs must share one dtype")
    return out, code


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check_window(mode, window):
    if int(mode) == LOCAL and int(window) < 1:
        raise ValueError("local mode needs a window of at least 1 expanded position")


FINAL = 4  # or-ed into the mode: queries at the final stream of each token only


def _dims(q, k, B, L, n, mode, scale, nthreads, window=0, final=False):
    N = n * L
    qrows = L if final else N
    if q.shape[:2] != (B, qrows) or k.shape[:2] != (B, N) or q.shape[3] != k.shape[3]:
        raise ValueError(f"q must be [B][{'L' if final else 'n*L'}][Hq][D] and k/v "
                         "[B][n*L][Hkv][D]")
    Hq, D, Hkv = q.shape[2], q.shape[3], k.shape[2]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    _check_window(mode, window)
    return (B, L, n, Hq, Hkv, D, int(mode) | (FINAL if final else 0), int(window), float(scale),
            int(nthreads or default_threads())), Hq, Hkv, D


def _final_rows(rows, n, final):
    """Query rows (b, hq, t) of a final-stream layer name expanded position t*n + n - 1."""
    rows = np.ascontiguousarray(rows, dtype=np.int64).reshape(-1, 3).copy()
    if final:
        rows[:, 2] = rows[:, 2] * n + n - 1
    return rows


def sfa_fwd(q, k, v, *, L, n, mode, scale, nthreads=None, window=0, final=False):
    """Full forward. Returns (o [B][N][Hq][D], lse [B][Hq][N]) in float64; with
    final=True, q and o are [B][L][Hq][D] (final-stream queries) and lse [B][Hq][L]."""
    (q, k, v), code = _prep(q, k, v)
    B = q.shape[0]
    dims, Hq, Hkv, D = _dims(q, k, B, L, n, mode, scale, nthreads, window, final)
    rows = L if final else n * L
    o = np.zeros((B, rows, Hq, D))
    lse = np.zeros((B, Hq, rows))
    _load().oracle_sfa_fwd(_ptr(q), _ptr(k), _ptr(v), code, _ptr(o), _ptr(lse), *dims)
    return o, lse


def sfa_fwd_rows(q, k, v, rows, *, L, n, mode, scale, nthreads=None, window=0, final=False):
    """Forward of listed rows; rows is int64 [R][3] of (b, hq, p) (p = t, the token,
    with final=True)."""
    (q, k, v), code = _prep(q, k, v)
    rows = _final_rows(rows, n, final)
    dims, Hq, Hkv, D = _dims(q, k, q.shape[0], L, n, mode, scale, nthreads, window, final)
    o = np.zeros((len(rows), D))
    lse = np.zeros(len(rows))
    _load().oracle_sfa_fwd_rows(_ptr(q), _ptr(k), _ptr(v), code, _ptr(rows), len(rows),
                                _ptr(o), _ptr(lse), *dims)
    return o, lse


def sfa_bwd(q, k, v, dout, *, L, n, mode, scale, nthreads=None, window=0, final=False):
    """Full backward from (q, k, v, dO). Returns (dq, dk, dv) in float64 (dq, like q
    and dO, [B][L][Hq][D] with final=True)."""
    (q, k, v, dout), code = _prep(q, k, v, dout)
    B = q.shape[0]
    dims, Hq, Hkv, D = _dims(q, k, B, L, n, mode, scale, nthreads, window, final)
    dq = np.zeros((B, L if final else n * L, Hq, D))
    dk = np.zeros((B, n * L, Hkv, D))
    dv = np.zeros((B, n * L, Hkv, D))
    _load().oracle_sfa_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(dout), code, _ptr(dq), _ptr(dk),
                           _ptr(dv), *dims)
    return dq, dk, dv


def sfa_bwd_dq_rows(q, k, v, dout, rows, *, L, n, mode, scale, nthreads=None, window=0,
                    final=False):
    """dQ of listed query rows (b, hq, p) ((b, hq, t) with final=True)."""
    (q, k, v, dout), code = _prep(q, k, v, dout)
    rows = _final_rows(rows, n, final)
    dims, Hq, Hkv, D = _dims(q, k, q.shape[0], L, n, mode, scale, nthreads, window, final)
    dq = np.zeros((len(rows), D))
    _load().oracle_sfa_bwd_dq_rows(_ptr(q), _ptr(k), _ptr(v), _ptr(dout), code, _ptr(rows),
                                   len(rows), _ptr(dq), *dims)
    return dq


def sfa_bwd_dkdv_rows(q, k, v, dout, rows, *, L, n, mode, scale, nthreads=None, window=0,
                      final=False):
    """dK, dV of listed key rows (b, hk, j), summed over the group's query heads."""
    (q, k, v, dout), code = _prep(q, k, v, dout)
    rows = np.ascontiguousarray(rows, dtype=np.int64).reshape(-1, 3)
    dims, Hq, Hkv, D = _dims(q, k, q.shape[0], L, n, mode, scale, nthreads, window, final)
    dk = np.zeros((len(rows), D))
    dv = np.zeros((len(rows), D))
    _load().oracle_sfa_bwd_dkdv_rows(_ptr(q), _ptr(k), _ptr(v), _ptr(dout), code, _ptr(rows),
                                     len(rows), _ptr(dk), _ptr(dv), *dims)
    return dk, dv


def expand_embed(ids, tables):
    """eq. (expansion): ids [B][L] int32, tables [n][V][Dm] (any dtype) -> (out, bad)."""
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    tables = np.ascontiguousarray(tables)
    B, L = ids.shape
    n, V, Dm = tables.shape
    out = np.empty((B, n * L, Dm), dtype=tables.dtype)
    bad = _load().oracle_expand_embed(_ptr(ids), _ptr(tables), _ptr(out), B, L, n, V, Dm,
                                      tables.dtype.itemsize)
    return out, int(bad)


def expand_embed_bwd(ids, dout, V):
    """Gradient of eq. (expansion) w.r.t. the tables: ids [B][L] int32, dout [B][n*L][Dm]
    (fp64, fp32 or bf16 bits) -> dense fp64 [n][V][Dm]."""
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    dout = np.ascontiguousarray(dout)
    B, L = ids.shape
    N, Dm = dout.shape[1], dout.shape[2]
    if dout.shape[0] != B or N % L:
        raise ValueError("dout must be [B][n*L][Dm]")
    n = N // L
    out = np.empty((n, V, Dm))
    _load().oracle_expand_embed_bwd(_ptr(ids), _ptr(dout), _dtype_code(dout), _ptr(out), B, L,
                                    n, V, Dm)
    return out


def expand_embed_bwd_rows(ids, dout, V, req):
    """The same gradient for the token ids listed in ``req`` only -> fp64 [len(req)][n][Dm]."""
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    dout = np.ascontiguousarray(dout)
    req = np.ascontiguousarray(req, dtype=np.int32).reshape(-1)
    B, L = ids.shape
    N, Dm = dout.shape[1], dout.shape[2]
    n = N // L
    out = np.empty((len(req), n, Dm))
    _load().oracle_expand_embed_bwd_rows(_ptr(ids), _ptr(dout), _dtype_code(dout), _ptr(req),
                                         len(req), _ptr(out), B, L, n, V, Dm)
    return out


def cyclic_replicate(tables, m):
    """eq. (cyclic_init): tables [n][V][Dm] -> [m][V][Dm] with table s = tables[s mod n]."""
    tables = np.ascontiguousarray(tables)
    n, V, Dm = tables.shape
    if m < n or m % n:
        raise ValueError("m must be a positive multiple of n")
    out = np.empty((m, V, Dm), dtype=tables.dtype)
    _load().oracle_cyclic_replicate(_ptr(tables), _ptr(out), n, m, V, Dm, tables.dtype.itemsize)
    return out


def final_gather(h, n):
    """eq. (hd_loss) input: h [B][n*L][Dm] (any dtype) -> [B][L][Dm], row i = h[i*n + n-1]."""
    h = np.ascontiguousarray(h)
    B, N, Dm = h.shape
    if N % n:
        raise ValueError("h must be [B][n*L][Dm]")
    L = N // n
    out = np.empty((B, L, Dm), dtype=h.dtype)
    _load().oracle_final_gather(_ptr(h), _ptr(out), B, L, n, Dm, h.dtype.itemsize)
    return out


def final_gather_bwd(dout, n):
    """Adjoint of final_gather: dout [B][L][Dm] -> dh [B][n*L][Dm], zero off the final rows."""
    dout = np.ascontiguousarray(dout)
    B, L, Dm = dout.shape
    dh = np.empty((B, n * L, Dm), dtype=dout.dtype)
    _load().oracle_final_gather_bwd(_ptr(dout), _ptr(dh), B, L, n, Dm, dout.dtype.itemsize)
    return dh


def sfa_mask(L, n, mode, window=0):
    """Explicit [N][N] 0/1 mask straight from the definitions."""
    _check_window(mode, window)
    N = n * L
    m = np.zeros((N, N), dtype=np.uint8)
    _load().oracle_sfa_mask(_ptr(m), L, n, int(mode), int(window))
    return m


def sfa_decode(q, kcache, vcache, ctx, *, n, mode, scale, window=0, nthreads=None):
    """Parallel-stream decode: the n streams of each sequence's new token attend to its
    cached prefix.  q [B][n][Hq][D] (stream s of the new token of sequence b),
    kcache/vcache [B][n*Lcap][Hkv][D] (expanded rows; the new token's own rows at
    ctx[b]*n + s are already in the cache), ctx [B] tokens before the new one.
    By definition this is the forward of the layer over the ctx[b] + 1 cached tokens,
    read at the last token's n rows: returns o [B][n][Hq][D], lse [B][Hq][n] (fp64)."""
    q = np.ascontiguousarray(q)
    B, n_, Hq, D = q.shape
    if n_ != n:
        raise ValueError("q must be [B][n][Hq][D]")
    o = np.zeros((B, n, Hq, D))
    lse = np.zeros((B, Hq, n))
    for b in range(B):
        c = int(ctx[b])
        L = c + 1
        qf = np.zeros((1, n * L, Hq, D), dtype=q.dtype)
        qf[0, c * n:(c + 1) * n] = q[b]
        rows = np.array([(0, h, c * n + s) for s in range(n) for h in range(Hq)], np.int64)
        ro, rl = sfa_fwd_rows(qf, np.ascontiguousarray(kcache[b:b + 1, :n * L]),
                              np.ascontiguousarray(vcache[b:b + 1, :n * L]), rows, L=L, n=n,
                              mode=mode, scale=scale, nthreads=nthreads, window=window)
        for i, (_, h, p) in enumerate(rows):
            o[b, p - c * n, h] = ro[i]
            lse[b, h, p - c * n] = rl[i]
    return o, lse
