"""Reference oracle for uncertainty-gated block-sparse prefill.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke``
and the CPU-baseline leg of ``bench.py``.  The product library never imports
or links it, and it imports nothing from the product package.

Thin numpy wrappers over ``libugbs_oracle.so`` (plain C, IEEE double; see
``ugbs_oracle.c`` for the paper sections each function follows).  bf16 arrays
are numpy ``uint16`` bit patterns.
"""
import ctypes
import os

import numpy as np

from . import build as _build

KMEAN, QUEST = 0, 1
BLOCK = 64

_lib = None


def lib():
    global _lib
    if _lib is None:
        # rebuilt when missing or older than its source, so a run never loads a stale oracle
        if (not os.path.exists(_build.LIB)
                or os.path.getmtime(_build.SRC) > os.path.getmtime(_build.LIB)):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int, ctypes.c_long, ctypes.c_double
        L.orc_block_meta.argtypes = [i32, i32, i32, i32, i32, P, P, i32]
        L.orc_tile_scores.argtypes = [i32, i32, i32, i32, i32, i32, P, P, i64, P, P, i32]
        L.orc_select.argtypes = [i32, i32, i32, i64, P, P, P, P]
        L.orc_route.argtypes = [i32, i32, i32, i32, i32, f64, P, P, P, P, P, P]
        L.orc_attend.argtypes = [i32, i32, i32, i32, f64, P, P, P, P, i32, i32, i64, P, P, i32]
        L.orc_row_roughness.argtypes = [i32, i32, i32, i32, i32, P, P, i64, P, P, i32]
        L.orc_row_roughness.restype = ctypes.c_int
        L.orc_row_scores.argtypes = [i32, i32, i32, i32, i32, P, P, i64, P, P, i32]
        L.orc_row_scores.restype = ctypes.c_int
        L.orc_bf16_round.argtypes = [f64]
        L.orc_bf16_round.restype = ctypes.c_uint16
        for f in ("orc_block_meta", "orc_tile_scores", "orc_select", "orc_route", "orc_attend"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def _c(a, dtype):
    a = np.ascontiguousarray(a)
    assert a.dtype == dtype, (a.dtype, dtype)
    return a


def default_threads():
    return max(1, os.cpu_count() or 1)


def bf16_round(x: float) -> int:
    return int(lib().orc_bf16_round(float(x)))


def meta_width(backbone):
    return 1 if backbone == KMEAN else 2


def block_meta(backbone, K, nthreads=None):
    """A.1: K [B,Hkv,N,d] bf16 bits -> meta [B,Hkv,N_B,w,d] bf16 bits (w=1 mean; w=2 min,max)."""
    K = _c(K, np.uint16)
    B, Hkv, N, d = K.shape
    NB = N // BLOCK
    meta = np.zeros((B, Hkv, NB, meta_width(backbone), d), np.uint16)
    rc = lib().orc_block_meta(backbone, B, Hkv, N, d, _ptr(K), _ptr(meta), nthreads or default_threads())
    assert rc == 0
    return meta


def all_units(B, H, T):
    b, h, t = np.meshgrid(np.arange(B), np.arange(H), np.arange(T), indexing="ij")
    return np.stack([b.ravel(), h.ravel(), t.ravel()], axis=1).astype(np.int32)


def tile_scores(backbone, Q, meta, Hkv, units=None, nthreads=None):
    """A.2-A.3: per unit (b,h,t) -> fp32 row over N_B blocks (-inf outside C(t) = 1..t-1).

    With ``units=None`` returns [B,H,T,N_B]; else [n_units, N_B]."""
    Q = _c(Q, np.uint16)
    meta = _c(meta, np.uint16)
    B, H, N, d = Q.shape
    NB = N // BLOCK
    full = units is None
    if full:
        units = all_units(B, H, NB)
    units = _c(units, np.int32)
    out = np.empty((units.shape[0], NB), np.float32)
    rc = lib().orc_tile_scores(backbone, B, H, Hkv, N, d, _ptr(Q), _ptr(meta), units.shape[0],
                               _ptr(units), _ptr(out), nthreads or default_threads())
    assert rc == 0
    return out.reshape(B, H, NB, NB) if full else out


def select(tile_score, k, t_of_row=None, rho=2):
    """A.4-A.6: tile_score [..., N_B] fp32 -> idx_sorted [..., rho k] int32, sigma [...] fp32.

    If ``t_of_row`` is None the second-to-last axis of a [B,H,T,N_B] array is t."""
    ts = _c(tile_score, np.float32)
    NB = ts.shape[-1]
    lead = ts.shape[:-1]
    if t_of_row is None:
        T = ts.shape[-2]
        t_of_row = np.broadcast_to(np.arange(T, dtype=np.int32), lead)
    t_of_row = _c(np.asarray(t_of_row, np.int32).reshape(-1), np.int32)
    rows = t_of_row.shape[0]
    W = rho * k
    idx = np.empty((rows, W), np.int32)
    sig = np.empty((rows,), np.float32)
    rc = lib().orc_select(NB, k, rho, rows, _ptr(t_of_row), _ptr(ts.reshape(rows, NB)), _ptr(idx),
                          _ptr(sig))
    assert rc == 0
    return idx.reshape(*lead, W), sig.reshape(lead)


def route(sigma, idx_sorted, k, q, rho=2):
    """A.7-A.9: sigma [B,H,T], idx_sorted [B,H,T,rho k] -> kv_idx, sigma_bar [B,T], tau [B], trigger [B,T]."""
    sigma = _c(sigma, np.float32)
    idx_sorted = _c(idx_sorted, np.int32)
    B, H, T = sigma.shape
    kv = np.empty_like(idx_sorted)
    sb = np.empty((B, T), np.float32)
    tau = np.empty((B,), np.float32)
    trig = np.empty((B, T), np.uint8)
    assert idx_sorted.shape[-1] == rho * k
    rc = lib().orc_route(B, H, T, k, rho, float(q), _ptr(sigma), _ptr(idx_sorted), _ptr(kv), _ptr(sb),
                         _ptr(tau), _ptr(trig))
    assert rc == 0
    return kv, sb, tau, trig


def attend(Q, K, V, kv_idx=None, scale=None, units=None, dense=False, nthreads=None):
    """A.10 / Eq. (Attn): exact softmax attention, fp64.

    kv_idx: [B,H,T,W] (units=None) or [n_units, W]; ignored if ``dense``.
    Returns [B,H,N,d] float64 (units=None) or [n_units, 64, d]."""
    Q, K, V = (_c(x, np.uint16) for x in (Q, K, V))
    B, H, N, d = Q.shape
    Hkv = K.shape[1]
    NB = N // BLOCK
    full = units is None
    if full:
        units = all_units(B, H, NB)
    units = _c(units, np.int32)
    n = units.shape[0]
    if dense:
        W = 1
        kv = np.zeros((n, 1), np.int32)
    else:
        kv = _c(np.asarray(kv_idx, np.int32).reshape(n, -1), np.int32)
        W = kv.shape[1]
    if scale is None or scale == 0:
        scale = 1.0 / np.sqrt(d)
    O = np.empty((n, BLOCK, d), np.float64)
    rc = lib().orc_attend(H, Hkv, N, d, float(scale), _ptr(Q), _ptr(K), _ptr(V), _ptr(kv), W,
                          1 if dense else 0, n, _ptr(units), _ptr(O), nthreads or default_threads())
    assert rc == 0
    if full:
        return O.reshape(B, H, NB * BLOCK, d)
    return O


def row_roughness(backbone, Q, meta, Hkv, units=None, nthreads=None):
    """Appendix D step 3: per unit (b, h, t), sum over candidate blocks of
    C(t) and the 63 adjacent row pairs of the tile of (s[r+1,b] - s[r,b])^2
    (per-row block scores, fp64).  Returns (sums [n_units] f64, terms [n_units])."""
    Q = _c(Q, np.uint16)
    meta = _c(meta, np.uint16)
    B, H, N, d = Q.shape
    T = N // BLOCK
    if units is None:
        units = all_units(B, H, T)
    units = _c(np.asarray(units, np.int32), np.int32)
    out = np.empty(units.shape[0], np.float64)
    rc = lib().orc_row_roughness(backbone, H, Hkv, N, d, _ptr(Q), _ptr(meta), units.shape[0],
                                 _ptr(units), _ptr(out), nthreads or default_threads())
    assert rc == 0
    terms = 63 * np.maximum(units[:, 2].astype(np.int64) - 1, 0)
    return out, terms


def row_scores(backbone, Q, meta, Hkv, units=None, nthreads=None):
    """A.2 per row: for each unit (b, h, t) the [64, N_B] fp32 scores of the
    tile's query rows against the candidate blocks C(t) (fp64, rounded to
    fp32; -inf elsewhere).  Returns [n_units, 64, N_B] ([B, H, T, 64, N_B]
    with units=None)."""
    Q = _c(Q, np.uint16)
    meta = _c(meta, np.uint16)
    B, H, N, d = Q.shape
    T = N // BLOCK
    full = units is None
    if full:
        units = all_units(B, H, T)
    units = _c(np.asarray(units, np.int32), np.int32)
    out = np.empty((units.shape[0], BLOCK, T), np.float32)
    rc = lib().orc_row_scores(backbone, H, Hkv, N, d, _ptr(Q), _ptr(meta), units.shape[0],
                              _ptr(units), _ptr(out), nthreads or default_threads())
    assert rc == 0
    return out.reshape(B, H, T, BLOCK, T) if full else out


def select_rows(rows, t_of_unit, k, rho=2, trig_of_unit=None):
    """Per-row selection scattered into a per-tile bitmap (the per-row variant
    the Limitations of Section 4 name; Section 3.2 describes the per-tile
    rule it refines).  For each unit with tile t and each of its 64 rows:
    the forced blocks F = [0] (t = 0) or [0, t] and the row's R best
    candidates of C(t) by (row score descending, lower block first, -0 ==
    +0), R = (trigger ? rho k : k) - |F|, all of C(t) when fewer; the tile's
    set is the union over its rows.

    rows [n_units, 64, N_B] fp32; returns [n_units, ceil(N_B / 32)] uint32
    words (bit b of word b // 32 set = block b attended)."""
    rows = np.asarray(rows, np.float32)
    n, R64, NB = rows.shape
    nw = (NB + 31) // 32
    out = np.zeros((n, nw), np.uint32)
    for u in range(n):
        t = int(t_of_unit[u])
        nf = 1 if t == 0 else 2
        nc = max(t - 1, 0)
        trig = bool(trig_of_unit[u]) if trig_of_unit is not None else False
        R = min((rho * k if trig else k) - nf, nc)
        keep = {0} | ({t} if t > 0 else set())
        for r in range(R64):
            cand = [(float(rows[u, r, b]) + 0.0, b) for b in range(1, t)]   # -0 -> +0
            cand.sort(key=lambda x: (-x[0], x[1]))
            keep |= {b for _, b in cand[:R]}
        for b in keep:
            out[u, b // 32] |= np.uint32(1 << (b % 32))
    return out


def bitmap_blocks(words, NB):
    """The attended blocks of one bitmap row, ascending."""
    return [b for b in range(NB) if (int(words[b // 32]) >> (b % 32)) & 1]


def population(T, k):
    """Tiles with more non-forced candidates than kept slots (quantile population)."""
    t = np.arange(T)
    nf = np.where(t == 0, 1, 2)
    nc = np.maximum(t - 1, 0)
    return nc > (k - nf)
