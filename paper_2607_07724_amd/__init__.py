"""Uncertainty-gated block-sparse causal prefill attention for MI355X (gfx950).

Thin ctypes binding over ``libugbs.so`` (the C ABI declared in
``include/ugbs.h``).  Each ``ugbs_*`` function here has the name of the C
entry point it calls and only marshals arguments: it checks that the torch
tensors have the shapes, dtypes and device the problem implies (the C ABI
receives bare pointers and cannot), passes ``data_ptr()`` values and the
current HIP stream, and raises :class:`UGBSError` on a non-zero status.
Every step of the method runs in the HIP kernels; there is no fallback.

PyTorch is used for device memory and streams only.
"""
from __future__ import annotations

import ctypes
import math
import os

__all__ = [
    "KMEAN", "QUEST", "BLOCK", "Problem", "UGBSError", "lib", "library_path",
    "ugbs_block_meta", "ugbs_score_select", "ugbs_route", "ugbs_attend",
    "ugbs_workspace_bytes", "ugbs_status_string", "ugbs_abi_version",
    "ugbs_attend_select", "prefill_fused", "ugbs_select_rows", "ugbs_attend_bitmap",
    "ugbs_noise_scale", "ugbs_bai_tiles", "ugbs_bai_heads", "BAI_TILE_FIELDS", "BAI_HEAD_FIELDS",
    "bai_tile_records", "bai_head_records", "ugbs_route_noalloc", "ROUTE_SCRATCH_BYTES",
    "ugbs_quest_scores_valu",
]

KMEAN, QUEST = 0, 1
BLOCK = 64
MAX_BLOCKS = 4096
MAX_BLOCKS_ROWS = 2048
MAX_KV_WIDTH = 4096
ROUTE_SCRATCH_BYTES = 1 << 20
_HERE = os.path.dirname(os.path.abspath(__file__))


def library_path() -> str:
    return os.path.join(_HERE, "libugbs.so")


class UGBSError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        msg = ugbs_status_string(status) if _lib is not None else str(status)
        super().__init__(f"{fn} failed with status {status}: {msg}")


class Problem(ctypes.Structure):
    """Mirror of ``ugbs_problem`` (include/ugbs.h)."""
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("seq_len", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block", ctypes.c_int32),
        ("k_budget", ctypes.c_int32),
        ("backbone", ctypes.c_int32),
        ("q", ctypes.c_double),
        ("softmax_scale", ctypes.c_float),
        ("rho", ctypes.c_int32),
    ]

    @classmethod
    def make(cls, B, H, Hkv, N, d, k, q, backbone=KMEAN, scale=0.0, block=BLOCK, rho=2):
        return cls(B, H, Hkv, N, d, block, k, backbone, float(q), float(scale), rho)

    @property
    def NB(self) -> int:
        return self.seq_len // BLOCK

    @property
    def T(self) -> int:
        return self.seq_len // BLOCK

    @property
    def W(self) -> int:
        return (self.rho or 2) * self.k_budget

    @property
    def meta_width(self) -> int:
        return 2 if self.backbone == QUEST else 1

    def __repr__(self):
        return (f"Problem(B={self.batch}, H={self.n_heads}, Hkv={self.n_kv_heads}, N={self.seq_len}, "
                f"d={self.head_dim}, k={self.k_budget}, q={self.q}, backbone={self.backbone})")


_lib = None


def lib():
    """Load libugbs.so; raise if it is missing (there is no CPU fallback)."""
    global _lib
    if _lib is None:
        path = library_path()
        if not os.path.exists(path):
            raise ImportError(f"{path} is not built; run paper_2607_07724_amd/build.py "
                              "(or __graft_entry__.build())")
        L = ctypes.CDLL(path)
        P = ctypes.c_void_p
        pp = ctypes.POINTER(Problem)
        L.ugbs_block_meta.argtypes = [pp, P, P, P]
        L.ugbs_score_select.argtypes = [pp, P, P, P, P, P, P, P, ctypes.c_size_t, P]
        L.ugbs_route.argtypes = [pp, P, P, P, P, P, P, P, ctypes.c_size_t, P]
        L.ugbs_route_noalloc.argtypes = [pp, P, P, P, P, P, P, P]
        L.ugbs_attend.argtypes = [pp, P, P, P, P, ctypes.c_int32, P, P]
        L.ugbs_workspace_bytes.argtypes = [pp]
        L.ugbs_workspace_bytes.restype = ctypes.c_size_t
        L.ugbs_status_string.argtypes = [ctypes.c_int]
        L.ugbs_status_string.restype = ctypes.c_char_p
        L.ugbs_abi_version.argtypes = []
        L.ugbs_attend_select.argtypes = [pp, P, P, P, P, P, P, ctypes.c_size_t, P, P]
        L.ugbs_select_rows.argtypes = [pp, P, P, P, P, P, P]
        L.ugbs_attend_bitmap.argtypes = [pp, P, P, P, P, P, P]
        L.ugbs_noise_scale.argtypes = [pp, P, P, P, P, P]
        L.ugbs_bai_tiles.argtypes = [pp, P, P, P, ctypes.c_int32, P, P]
        L.ugbs_bai_heads.argtypes = [pp, P, P, ctypes.c_int32, P, P]
        L.ugbs_quest_scores_valu.argtypes = [pp, P, P, P, P]
        for f in ("ugbs_block_meta", "ugbs_score_select", "ugbs_route", "ugbs_attend", "ugbs_abi_version",
                  "ugbs_attend_select", "ugbs_select_rows", "ugbs_attend_bitmap",
                  "ugbs_noise_scale", "ugbs_bai_tiles", "ugbs_bai_heads", "ugbs_route_noalloc",
                  "ugbs_quest_scores_valu"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def ugbs_status_string(status: int) -> str:
    return lib().ugbs_status_string(int(status)).decode()


def ugbs_abi_version() -> int:
    return int(lib().ugbs_abi_version())


def ugbs_workspace_bytes(p: Problem) -> int:
    return int(lib().ugbs_workspace_bytes(ctypes.byref(p)))


# ---------------------------------------------------------------- marshalling

def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(int(stream))
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(name, t, shape, dtypes, device=None):
    import torch
    if t is None:
        raise ValueError(f"{name} is required")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)} != expected {tuple(shape)}")
    if t.dtype not in dtypes:
        raise ValueError(f"{name}: dtype {t.dtype} not in {dtypes}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _opt(name, t, shape, dtypes, device):
    return None if t is None else _check(name, t, shape, dtypes, device)


def _bf16():
    import torch
    return (torch.bfloat16, torch.int16, torch.uint16)


def _raise(fn, st):
    if st != 0:
        raise UGBSError(fn, st)


def ugbs_block_meta(p: Problem, K, meta, stream=None):
    """Stage 1 (A.1): K [B,Hkv,N,d] bf16 -> meta [B,Hkv,N_B,d,(1|2)] bf16
    (Quest: per channel the pair (min, max))."""
    bf = _bf16()
    dev = K.device
    k = _check("K", K, (p.batch, p.n_kv_heads, p.seq_len, p.head_dim), bf)
    m = _check("meta", meta, (p.batch, p.n_kv_heads, p.NB, p.head_dim, p.meta_width), bf, dev)
    _raise("ugbs_block_meta", lib().ugbs_block_meta(ctypes.byref(p), k, m, _stream(stream)))


def ugbs_score_select(p: Problem, Q, meta, idx_sorted, sigma, scores_in=None, scores_out=None,
                      stream=None, workspace=None):
    """Stages 2-3 (A.2-A.6): -> idx_sorted [B,H,T,2k] int32 (or None: sigma
    only), sigma [B,H,T] fp32.  Without scores_in/scores_out the tile scores
    pass through `workspace` (>= ugbs_workspace_bytes(p) bytes)."""
    import torch
    bf = _bf16()
    dev = Q.device
    q = _check("Q", Q, (p.batch, p.n_heads, p.seq_len, p.head_dim), bf)
    m = _check("meta", meta, (p.batch, p.n_kv_heads, p.NB, p.head_dim, p.meta_width), bf, dev)
    si = _opt("scores_in", scores_in, (p.batch, p.n_heads, p.T, p.NB), (torch.float32,), dev)
    so = _opt("scores_out", scores_out, (p.batch, p.n_heads, p.T, p.NB), (torch.float32,), dev)
    ix = _opt("idx_sorted", idx_sorted, (p.batch, p.n_heads, p.T, p.W), (torch.int32,), dev)
    sg = _check("sigma", sigma, (p.batch, p.n_heads, p.T), (torch.float32,), dev)
    ws, nbytes = None, 0
    if workspace is not None:
        ws = _check("workspace", workspace, tuple(workspace.shape), (workspace.dtype,), dev)
        nbytes = workspace.numel() * workspace.element_size()
    _raise("ugbs_score_select",
           lib().ugbs_score_select(ctypes.byref(p), q, m, si, so, ix, sg, ws, nbytes, _stream(stream)))


def ugbs_quest_scores_valu(p: Problem, Q, meta, scores_out, stream=None):
    """Quest tile scores on the vector ALU (the literal per-channel form of
    Eq. (quest-score)): scores_out [B,H,T,N_B] fp32, -inf outside C(t)."""
    import torch
    bf = _bf16()
    dev = Q.device
    q = _check("Q", Q, (p.batch, p.n_heads, p.seq_len, p.head_dim), bf)
    m = _check("meta", meta, (p.batch, p.n_kv_heads, p.NB, p.head_dim, p.meta_width), bf, dev)
    so = _check("scores_out", scores_out, (p.batch, p.n_heads, p.T, p.NB), (torch.float32,), dev)
    _raise("ugbs_quest_scores_valu",
           lib().ugbs_quest_scores_valu(ctypes.byref(p), q, m, so, _stream(stream)))


def ugbs_route(p: Problem, sigma, idx_sorted, kv_idx, workspace, sigma_bar=None, tau=None,
               trigger=None, stream=None):
    """Stage 4 (A.7-A.9): sigma, idx_sorted -> kv_idx (may be idx_sorted itself);
    idx_sorted and kv_idx both None: statistics and trigger flags only."""
    import torch
    dev = sigma.device
    sg = _check("sigma", sigma, (p.batch, p.n_heads, p.T), (torch.float32,))
    if (idx_sorted is None) != (kv_idx is None):
        raise ValueError("idx_sorted and kv_idx are given together or not at all")
    ix = _opt("idx_sorted", idx_sorted, (p.batch, p.n_heads, p.T, p.W), (torch.int32,), dev)
    kv = _opt("kv_idx", kv_idx, (p.batch, p.n_heads, p.T, p.W), (torch.int32,), dev)
    need = ugbs_workspace_bytes(p)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace must hold >= {need} bytes")
    ws = _check("workspace", workspace, tuple(workspace.shape), (workspace.dtype,), dev)
    sb = _opt("sigma_bar", sigma_bar, (p.batch, p.T), (torch.float32,), dev)
    ta = _opt("tau", tau, (p.batch,), (torch.float32,), dev)
    tr = _opt("trigger", trigger, (p.batch, p.T), (torch.uint8,), dev)
    _raise("ugbs_route", lib().ugbs_route(ctypes.byref(p), sg, ix, kv, sb, ta, tr, ws,
                                          workspace.numel() * workspace.element_size(),
                                          _stream(stream)))


def ugbs_route_noalloc(p: Problem, sigma, idx_sorted, kv_idx, sigma_bar=None, tau=None, trigger=None,
                       stream=None):
    """Stage 4 without a workspace (for callers that cannot allocate): the
    route's sections live in the library's static per-GPU scratch; outputs
    equal ugbs_route's."""
    import torch
    dev = sigma.device
    sg = _check("sigma", sigma, (p.batch, p.n_heads, p.T), (torch.float32,))
    if (idx_sorted is None) != (kv_idx is None):
        raise ValueError("idx_sorted and kv_idx are given together or not at all")
    ix = _opt("idx_sorted", idx_sorted, (p.batch, p.n_heads, p.T, p.W), (torch.int32,), dev)
    kv = _opt("kv_idx", kv_idx, (p.batch, p.n_heads, p.T, p.W), (torch.int32,), dev)
    sb = _opt("sigma_bar", sigma_bar, (p.batch, p.T), (torch.float32,), dev)
    ta = _opt("tau", tau, (p.batch,), (torch.float32,), dev)
    tr = _opt("trigger", trigger, (p.batch, p.T), (torch.uint8,), dev)
    _raise("ugbs_route_noalloc", lib().ugbs_route_noalloc(ctypes.byref(p), sg, ix, kv, sb, ta, tr,
                                                          _stream(stream)))


def ugbs_attend(p: Problem, Q, K, V, kv_idx, O, stream=None):
    """Stage 5 (A.10): O [B,H,N,d] = softmax attention over the blocks in kv_idx [B,H,T,W]."""
    import torch
    bf = _bf16()
    dev = Q.device
    q = _check("Q", Q, (p.batch, p.n_heads, p.seq_len, p.head_dim), bf)
    k = _check("K", K, (p.batch, p.n_kv_heads, p.seq_len, p.head_dim), bf, dev)
    v = _check("V", V, (p.batch, p.n_kv_heads, p.seq_len, p.head_dim), bf, dev)
    if kv_idx.dim() != 4:
        raise ValueError("kv_idx must be [B,H,T,W]")
    width = int(kv_idx.shape[3])
    kv = _check("kv_idx", kv_idx, (p.batch, p.n_heads, p.T, width), (torch.int32,), dev)
    o = _check("O", O, (p.batch, p.n_heads, p.seq_len, p.head_dim), bf, dev)
    _raise("ugbs_attend", lib().ugbs_attend(ctypes.byref(p), q, k, v, kv, width, o, _stream(stream)))


def ugbs_attend_select(p: Problem, Q, K, V, O, workspace=None, scores=None, trigger=None,
                       stream=None):
    """Stage 5 with the selection in the attention kernel: the blocks of
    ugbs_route's kv_idx, chosen from the tile scores (`scores` [B,H,T,N_B]
    fp32, or the packed rows ugbs_score_select left in `workspace`) and the
    trigger flags (`trigger` [B,T] uint8, or ugbs_route's in `workspace`)."""
    import torch
    bf = _bf16()
    dev = Q.device
    q = _check("Q", Q, (p.batch, p.n_heads, p.seq_len, p.head_dim), bf)
    k = _check("K", K, (p.batch, p.n_kv_heads, p.seq_len, p.head_dim), bf, dev)
    v = _check("V", V, (p.batch, p.n_kv_heads, p.seq_len, p.head_dim), bf, dev)
    o = _check("O", O, (p.batch, p.n_heads, p.seq_len, p.head_dim), bf, dev)
    sc = _opt("scores", scores, (p.batch, p.n_heads, p.T, p.NB), (torch.float32,), dev)
    tr = _opt("trigger", trigger, (p.batch, p.T), (torch.uint8,), dev)
    ws, nbytes = None, 0
    if workspace is not None:
        ws = _check("workspace", workspace, tuple(workspace.shape), (workspace.dtype,), dev)
        nbytes = workspace.numel() * workspace.element_size()
    _raise("ugbs_attend_select", lib().ugbs_attend_select(ctypes.byref(p), q, k, v, sc, tr, ws, nbytes, o,
                                                          _stream(stream)))


def bitmap_words(p: Problem) -> int:
    return (p.NB + 31) // 32


def ugbs_select_rows(p: Problem, trigger, bitmap, Q=None, meta=None, row_scores=None, stream=None):
    """Per-row selection into tile bitmaps: bitmap [B,H,T,ceil(N_B/32)] int32
    (uint32 words) from the per-row scores of Q against meta (or `row_scores`
    [B,H,N,N_B] fp32) and the trigger flags [B,T] uint8."""
    import torch
    dev = bitmap.device
    bf = _bf16()
    tr = _check("trigger", trigger, (p.batch, p.T), (torch.uint8,), dev)
    bm = _check("bitmap", bitmap, (p.batch, p.n_heads, p.T, bitmap_words(p)), (torch.int32,), dev)
    q = _opt("Q", Q, (p.batch, p.n_heads, p.seq_len, p.head_dim), bf, dev)
    m = _opt("meta", meta, (p.batch, p.n_kv_heads, p.NB, p.head_dim, p.meta_width), bf, dev)
    rs = _opt("row_scores", row_scores, (p.batch, p.n_heads, p.seq_len, p.NB), (torch.float32,), dev)
    _raise("ugbs_select_rows", lib().ugbs_select_rows(ctypes.byref(p), q, m, rs, tr, bm, _stream(stream)))


def ugbs_attend_bitmap(p: Problem, Q, K, V, bitmap, O, stream=None):
    """Stage 5 over the blocks set in bitmap [B,H,T,ceil(N_B/32)] (int32 words)."""
    import torch
    bf = _bf16()
    dev = Q.device
    q = _check("Q", Q, (p.batch, p.n_heads, p.seq_len, p.head_dim), bf)
    k = _check("K", K, (p.batch, p.n_kv_heads, p.seq_len, p.head_dim), bf, dev)
    v = _check("V", V, (p.batch, p.n_kv_heads, p.seq_len, p.head_dim), bf, dev)
    bm = _check("bitmap", bitmap, (p.batch, p.n_heads, p.T, bitmap_words(p)), (torch.int32,), dev)
    o = _check("O", O, (p.batch, p.n_heads, p.seq_len, p.head_dim), bf, dev)
    _raise("ugbs_attend_bitmap", lib().ugbs_attend_bitmap(ctypes.byref(p), q, k, v, bm, o, _stream(stream)))


# ---------------------------------------------------------------- diagnostics

# Field layout of ugbs_bai_tile (32 bytes) and ugbs_bai_head (160 bytes).
BAI_TILE_FIELDS = [("g", "<f4"), ("G", "<f4"), ("r", "<f4"), ("sigma", "<f4"), ("delta2", "<f4"),
                   ("fail_k", "<i4"), ("fail_rk", "<i4"), ("valid", "<i4")]
BAI_HEAD_FIELDS = [("n_tiles", "<i4"), ("n_q", "<i4"), ("pad", "<i4", (2,))] + [
    (n, "<f8") for n in ("r_mean", "r_cv", "sigma_q", "gamma_q", "band_mass", "delta2_p05",
                         "delta2_p50", "pi2", "tau", "chi", "eps_bar", "vbar_gamma", "C_q", "bound",
                         "bound_band", "mc_err_k", "mc_err_rk", "mc_regret")]
BAI_TILE_BYTES, BAI_HEAD_BYTES = 32, 160


def _bytes_buf(name, t, n_bytes, dev):
    if t is None or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous device tensor")
    if t.numel() * t.element_size() != n_bytes:
        raise ValueError(f"{name} must hold exactly {n_bytes} bytes")
    if t.device != dev:
        raise ValueError(f"{name} is on {t.device}, expected {dev}")
    return ctypes.c_void_p(t.data_ptr())


def bai_tile_records(tiles):
    """Host copy of a ugbs_bai_tile buffer as a numpy structured array [..]."""
    import numpy as np
    raw = tiles.detach().cpu().contiguous().view(-1).numpy().view(np.uint8)
    return raw.view(np.dtype(BAI_TILE_FIELDS))


def bai_head_records(heads):
    """Host copy of a ugbs_bai_head buffer as a numpy structured array [..]."""
    import numpy as np
    raw = heads.detach().cpu().contiguous().view(-1).numpy().view(np.uint8)
    return raw.view(np.dtype(BAI_HEAD_FIELDS))


def ugbs_noise_scale(p: Problem, Q, meta, rough, tau, stream=None):
    """Appendix D step 3: rough [B,H,T] fp64 (per-tile sums of squared
    row-to-row score differences), tau [B,H] fp32."""
    import torch
    bf = _bf16()
    dev = Q.device
    q = _check("Q", Q, (p.batch, p.n_heads, p.seq_len, p.head_dim), bf)
    m = _check("meta", meta, (p.batch, p.n_kv_heads, p.NB, p.head_dim, p.meta_width), bf, dev)
    r = _check("rough", rough, (p.batch, p.n_heads, p.T), (torch.float64,), dev)
    ta = _check("tau", tau, (p.batch, p.n_heads), (torch.float32,), dev)
    _raise("ugbs_noise_scale", lib().ugbs_noise_scale(ctypes.byref(p), q, m, r, ta, _stream(stream)))


def ugbs_bai_tiles(p: Problem, scores, tiles, tau=None, z=None, stream=None):
    """Appendix D per-tile gaps and Monte Carlo failures.  scores [B,H,T,N_B]
    fp32 (scores_out layout); tau [B,H] fp32; z [N_B, n_samples] fp32
    (block-major); tiles: device buffer of B*H*T*32 bytes (ugbs_bai_tile
    records)."""
    import torch
    dev = scores.device
    sc = _check("scores", scores, (p.batch, p.n_heads, p.T, p.NB), (torch.float32,))
    ns = 0 if z is None else int(z.shape[1])
    zz = _opt("z", z, (p.NB, ns), (torch.float32,), dev)
    ta = _opt("tau", tau, (p.batch, p.n_heads), (torch.float32,), dev)
    tl = _bytes_buf("tiles", tiles, p.batch * p.n_heads * p.T * BAI_TILE_BYTES, dev)
    _raise("ugbs_bai_tiles", lib().ugbs_bai_tiles(ctypes.byref(p), sc, ta, zz, ns, tl, _stream(stream)))


def ugbs_bai_heads(p: Problem, tiles, tau, n_samples, heads, stream=None):
    """Appendix D per-head aggregates from the tile records; heads: device
    buffer of B*H*160 bytes (ugbs_bai_head records)."""
    import torch
    dev = tau.device
    ta = _check("tau", tau, (p.batch, p.n_heads), (torch.float32,))
    tl = _bytes_buf("tiles", tiles, p.batch * p.n_heads * p.T * BAI_TILE_BYTES, dev)
    hd = _bytes_buf("heads", heads, p.batch * p.n_heads * BAI_HEAD_BYTES, dev)
    _raise("ugbs_bai_heads", lib().ugbs_bai_heads(ctypes.byref(p), tl, ta, int(n_samples), hd,
                                                  _stream(stream)))


# ---------------------------------------------------------------- convenience

class Buffers:
    """Device buffers for one layer's pipeline (allocated by torch)."""

    def __init__(self, p: Problem, device="cuda"):
        import torch
        B, H, Hkv, T, NB, d = p.batch, p.n_heads, p.n_kv_heads, p.T, p.NB, p.head_dim
        self.meta = torch.empty((B, Hkv, NB, d, p.meta_width), dtype=torch.bfloat16, device=device)
        self.idx_sorted = torch.empty((B, H, T, p.W), dtype=torch.int32, device=device)
        self.sigma = torch.empty((B, H, T), dtype=torch.float32, device=device)
        self.kv_idx = torch.empty((B, H, T, p.W), dtype=torch.int32, device=device)
        self.sigma_bar = torch.empty((B, T), dtype=torch.float32, device=device)
        self.tau = torch.empty((B,), dtype=torch.float32, device=device)
        self.trigger = torch.empty((B, T), dtype=torch.uint8, device=device)
        nbytes = ugbs_workspace_bytes(p)
        self.workspace = torch.empty((max(nbytes, 256),), dtype=torch.uint8, device=device)


def prefill(p: Problem, Q, K, V, O, bufs: Buffers, stream=None, scores_in=None, scores_out=None):
    """Run the four stages in order on one stream: meta, score+select, route, attend."""
    ugbs_block_meta(p, K, bufs.meta, stream)
    ugbs_score_select(p, Q, bufs.meta, bufs.idx_sorted, bufs.sigma, scores_in, scores_out, stream,
                      workspace=bufs.workspace)
    ugbs_route(p, bufs.sigma, bufs.idx_sorted, bufs.kv_idx, bufs.workspace, bufs.sigma_bar,
               bufs.tau, bufs.trigger, stream)
    ugbs_attend(p, Q, K, V, bufs.kv_idx, O, stream)
    return O


def prefill_fused(p: Problem, Q, K, V, O, bufs: Buffers, stream=None):
    """The layer with the selection inside the attention kernel: meta,
    scores + sigma (no lists), route flags, attention."""
    ugbs_block_meta(p, K, bufs.meta, stream)
    ugbs_score_select(p, Q, bufs.meta, None, bufs.sigma, stream=stream, workspace=bufs.workspace)
    ugbs_route(p, bufs.sigma, None, None, bufs.workspace, bufs.sigma_bar, bufs.tau, bufs.trigger, stream)
    ugbs_attend_select(p, Q, K, V, O, workspace=bufs.workspace, stream=stream)
    return O


def default_scale(d: int) -> float:
    return 1.0 / math.sqrt(d)
