"""Thin Python binding of ``liblongstraw.so`` (argument marshalling only).

Torch tensors supply device memory and the stream; every step of the replay
path runs in the library's HIP kernels.  There is no fallback: if the library
is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_float, c_int32, c_int64, c_size_t, c_uint32, c_uint64, c_void_p

LIB_PATH = os.environ.get("LONGSTRAW_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "liblongstraw.so")

ABI_VERSION = 1
LS_BF16, LS_F32 = 0, 1
FLAG_CHECKED = 1
FLAG_ACCUMULATE_DQ = 4
FLAG_ACCUMULATE_DKV = 8
FLAG_BF16_NUMERATOR = 16
FLAG_PREP_READY = 32
STATUS = {0: "LS_OK", -1: "LS_ERR_INVALID_ARG", -2: "LS_ERR_UNSUPPORTED", -3: "LS_ERR_WORKSPACE",
          -4: "LS_ERR_ALIAS", -5: "LS_ERR_STALE", -6: "LS_ERR_PAGE_OOB", -7: "LS_ERR_HIP"}
EXPORTS = ["ls_abi_version", "ls_status_string", "ls_last_error", "ls_gather_kv", "ls_scatter_kv",
           "ls_prefix_attn_fwd", "ls_lse_merge", "ls_prefix_attn_bwd_workspace_size",
           "ls_prefix_attn_bwd", "ls_sparse_attn_workspace_size", "ls_sparse_attn_fwd",
           "ls_sparse_attn_bwd", "ls_dsa_index_scores", "ls_topk_select", "ls_hbm_read_probe",
           "ls_sparse_attn_fwd_noalloc"]


class AttnParams(ctypes.Structure):
    _fields_ = [("abi_version", c_int32), ("dtype", c_int32), ("n_q", c_int32),
                ("n_q_heads", c_int32), ("n_kv_heads", c_int32), ("head_dim", c_int32),
                ("head_dim_v", c_int32), ("page_size", c_int32), ("n_phys_pages", c_int64),
                ("n_logical_pages", c_int64), ("prefix_len", c_int64), ("q_pos0", c_int64),
                ("softmax_scale", c_float), ("flags", c_uint32), ("q", c_void_p),
                ("k_pool", c_void_p), ("v_pool", c_void_p), ("page_table", c_void_p),
                ("pool_epoch", c_uint64), ("expected_epoch", c_uint64)]


class DsaParams(ctypes.Structure):
    _fields_ = [("q_index", c_void_p), ("w_index", c_void_p), ("k_index_pool", c_void_p),
                ("page_table", c_void_p), ("n_phys_pages", c_int64), ("n_logical_pages", c_int64),
                ("n_q", c_int32), ("n_heads", c_int32), ("head_dim", c_int32),
                ("page_size", c_int32)]


class Split(ctypes.Structure):
    _fields_ = [("kv_begin", c_int64), ("kv_end", c_int64)]


class LongStrawError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status
        self.name = STATUS.get(status, str(status))


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FileNotFoundError(
            f"{path} not found: build it with `python -m paper_2607_14952_amd.build`")
    lib = ctypes.CDLL(path)
    P = POINTER(AttnParams)
    lib.ls_abi_version.restype = c_int32
    lib.ls_status_string.restype = ctypes.c_char_p
    lib.ls_status_string.argtypes = [c_int32]
    lib.ls_last_error.restype = ctypes.c_char_p
    lib.ls_gather_kv.restype = c_int32
    lib.ls_gather_kv.argtypes = [P, c_int64, c_int64, c_void_p, c_void_p, c_void_p]
    lib.ls_scatter_kv.restype = c_int32
    lib.ls_scatter_kv.argtypes = [P, c_int64, c_int64, c_void_p, c_void_p, c_void_p]
    lib.ls_prefix_attn_fwd.restype = c_int32
    lib.ls_prefix_attn_fwd.argtypes = [P, POINTER(Split), c_int32, c_void_p, c_void_p, c_void_p]
    lib.ls_lse_merge.restype = c_int32
    lib.ls_lse_merge.argtypes = [c_void_p, c_void_p, c_int32, c_int32, c_int32, c_int32, c_int32,
                                 c_void_p, c_void_p, c_uint32, c_void_p]
    lib.ls_prefix_attn_bwd_workspace_size.restype = c_size_t
    lib.ls_prefix_attn_bwd_workspace_size.argtypes = [P]
    lib.ls_prefix_attn_bwd.restype = c_int32
    lib.ls_prefix_attn_bwd.argtypes = [P, c_int64, c_int64, c_void_p, c_void_p, c_int32, c_void_p,
                                       c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
    lib.ls_sparse_attn_workspace_size.restype = c_size_t
    lib.ls_sparse_attn_workspace_size.argtypes = [P, c_int32, c_int32]
    lib.ls_sparse_attn_fwd.restype = c_int32
    lib.ls_sparse_attn_fwd.argtypes = [P, c_void_p, c_int32, c_void_p, c_void_p, c_void_p,
                                       c_size_t, c_void_p]
    lib.ls_sparse_attn_bwd.restype = c_int32
    lib.ls_sparse_attn_bwd.argtypes = [P, c_void_p, c_int32, c_void_p, c_void_p, c_int32, c_void_p,
                                       c_void_p, c_void_p, c_size_t, c_void_p]
    lib.ls_dsa_index_scores.restype = c_int32
    lib.ls_dsa_index_scores.argtypes = [POINTER(DsaParams), c_int64, c_int64, c_void_p, c_int64,
                                        c_void_p]
    lib.ls_topk_select.restype = c_int32
    lib.ls_topk_select.argtypes = [c_void_p, c_int64, c_void_p, c_int32, c_int64, c_int64, c_int32,
                                   c_void_p, c_void_p, c_int64, c_void_p]
    lib.ls_sparse_attn_fwd_noalloc.restype = c_int32
    lib.ls_sparse_attn_fwd_noalloc.argtypes = [P, c_void_p, c_int32, c_void_p, c_void_p, c_void_p]
    lib.ls_hbm_read_probe.restype = c_int32
    lib.ls_hbm_read_probe.argtypes = [c_void_p, c_size_t, c_void_p, c_void_p]
    if lib.ls_abi_version() != ABI_VERSION:
        raise RuntimeError("liblongstraw ABI version mismatch")
    _lib = lib
    return lib


def check(status: int) -> None:
    if status != 0:
        raise LongStrawError(status, load_library().ls_last_error().decode())


# ----------------------------------------------------------------- torch helpers
def _torch():
    import torch
    return torch


def _ptr(t, dtype=None, name="tensor", dense=True):
    """Device address of a tensor argument (None stays NULL), after checking
    that it lives on the GPU, has the expected dtype, and is contiguous
    (dense) or has unit stride in its last dimension (row-strided views whose
    leading stride is passed on).  The library itself cannot tell a host
    pointer from a device one."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (got device {t.device})")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if dense and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if not dense and t.dim() and t.stride(-1) != 1:
        raise ValueError(f"{name} must have unit stride in its last dimension")
    return t.data_ptr()


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return LS_BF16
    if t.dtype == torch.float32:
        return LS_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


class PagedKV:
    """A paged KV store: pools [n_phys, S, Hkv, D|Dv] and an int32 page table,
    all device tensors owned by the caller (read-only to the library)."""

    def __init__(self, k_pool, v_pool, page_table, epoch: int = 0):
        self.k_pool, self.v_pool, self.page_table = k_pool, v_pool, page_table
        self.epoch = epoch

    @property
    def page_size(self):
        return self.k_pool.shape[1]


def make_params(q, kv: PagedKV, *, n_q=None, n_q_heads=None, prefix_len: int, q_pos0: int,
                scale: float, flags: int = 0, expected_epoch=None) -> AttnParams:
    p = AttnParams()
    p.abi_version = ABI_VERSION
    p.dtype = _dtype_code(kv.k_pool)
    p.n_q = q.shape[0] if n_q is None else n_q
    p.n_q_heads = q.shape[1] if n_q_heads is None else n_q_heads
    p.n_kv_heads = kv.k_pool.shape[2]
    p.head_dim = kv.k_pool.shape[3]
    p.head_dim_v = kv.v_pool.shape[3]
    p.page_size = kv.k_pool.shape[1]
    p.n_phys_pages = kv.k_pool.shape[0]
    p.n_logical_pages = kv.page_table.shape[0]
    p.prefix_len = prefix_len
    p.q_pos0 = q_pos0
    p.softmax_scale = scale
    p.flags = flags
    torch = _torch()
    p.q = _ptr(q, kv.k_pool.dtype, "q")
    p.k_pool = _ptr(kv.k_pool, None, "k_pool")
    p.v_pool = _ptr(kv.v_pool, kv.k_pool.dtype, "v_pool")
    p.page_table = _ptr(kv.page_table, torch.int32, "page_table")
    p.pool_epoch = kv.epoch
    p.expected_epoch = kv.epoch if expected_epoch is None else expected_epoch
    return p


# ----------------------------------------------------------------- entry points
def gather_kv(kv: PagedKV, pos_begin: int, pos_end: int, *, flags: int = 0, k_out=None,
              v_out=None, stream=None):
    """ls_gather_kv: dense copies of logical positions [pos_begin, pos_end)."""
    torch = _torch()
    n = pos_end - pos_begin
    k = k_out if k_out is not None else torch.empty(
        (n,) + tuple(kv.k_pool.shape[2:]), dtype=kv.k_pool.dtype, device=kv.k_pool.device)
    v = v_out if v_out is not None else torch.empty(
        (n,) + tuple(kv.v_pool.shape[2:]), dtype=kv.v_pool.dtype, device=kv.v_pool.device)
    dummy_q = torch.empty((0, 1, 1), dtype=kv.k_pool.dtype, device=kv.k_pool.device)
    p = make_params(dummy_q, kv, n_q=0, n_q_heads=kv.k_pool.shape[2], prefix_len=0, q_pos0=0,
                    scale=1.0, flags=flags)
    p.q = None
    check(load_library().ls_gather_kv(ctypes.byref(p), pos_begin, pos_end,
                                      _ptr(k, kv.k_pool.dtype, "k_out"),
                                      _ptr(v, kv.v_pool.dtype, "v_out"), _stream(stream)))
    return k, v


def scatter_kv(kv: PagedKV, pos_begin: int, k_src, v_src, *, flags: int = 0, stream=None):
    """ls_scatter_kv: write dense rows into logical positions [pos_begin, pos_begin + n)
    of the paged store (the append step of a response branch)."""
    torch = _torch()
    n = k_src.shape[0]
    dummy_q = torch.empty((0, 1, 1), dtype=kv.k_pool.dtype, device=kv.k_pool.device)
    p = make_params(dummy_q, kv, n_q=0, n_q_heads=kv.k_pool.shape[2], prefix_len=0, q_pos0=0,
                    scale=1.0, flags=flags)
    p.q = None
    check(load_library().ls_scatter_kv(ctypes.byref(p), pos_begin, pos_begin + n,
                                       _ptr(k_src, kv.k_pool.dtype, "k_src"),
                                       _ptr(v_src, kv.v_pool.dtype, "v_src"), _stream(stream)))


def prefix_attn_fwd(q, kv: PagedKV, splits, *, prefix_len: int, q_pos0: int, scale: float,
                    flags: int = 0, out_part=None, lse_part=None, expected_epoch=None,
                    stream=None):
    """ls_prefix_attn_fwd: per-split normalized output [S, R, Hq, Dv] fp32 and
    log-normalizer [S, Hq, R] fp32."""
    torch = _torch()
    R, Hq = q.shape[0], q.shape[1]
    Dv = kv.v_pool.shape[3]
    n = len(splits)
    if out_part is None:
        out_part = torch.empty((n, R, Hq, Dv), dtype=torch.float32, device=q.device)
    if lse_part is None:
        lse_part = torch.empty((n, Hq, R), dtype=torch.float32, device=q.device)
    arr = (Split * n)(*[Split(int(b), int(e)) for b, e in splits])
    p = make_params(q, kv, prefix_len=prefix_len, q_pos0=q_pos0, scale=scale, flags=flags,
                    expected_epoch=expected_epoch)
    check(load_library().ls_prefix_attn_fwd(ctypes.byref(p), arr, n,
                                            _ptr(out_part, torch.float32, "out_part"),
                                            _ptr(lse_part, torch.float32, "lse_part"),
                                            _stream(stream)))
    return out_part, lse_part


def lse_merge(out_part, lse_part, *, out_dtype=None, out=None, lse=None, flags: int = 0,
              stream=None):
    """ls_lse_merge over the leading (split) dimension."""
    torch = _torch()
    n, R, H, Dv = out_part.shape
    out_dtype = torch.float32 if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((R, H, Dv), dtype=out_dtype, device=out_part.device)
    if lse is None:
        lse = torch.empty((H, R), dtype=torch.float32, device=out_part.device)
    check(load_library().ls_lse_merge(_ptr(out_part, torch.float32, "out_part"),
                                      _ptr(lse_part, torch.float32, "lse_part"), n, R, H, Dv,
                                      _dtype_code(out), _ptr(out, None, "out"),
                                      _ptr(lse, torch.float32, "lse"), flags, _stream(stream)))
    return out, lse


def bwd_workspace(q, kv: PagedKV, *, prefix_len: int, q_pos0: int):
    """Workspace for ls_prefix_attn_bwd calls with these rows, prefix_len and
    q_pos0 (also large enough for any call with a smaller q_pos0)."""
    torch = _torch()
    p = make_params(q, kv, prefix_len=prefix_len, q_pos0=q_pos0, scale=1.0)
    n = load_library().ls_prefix_attn_bwd_workspace_size(ctypes.byref(p))
    return torch.empty(max(n, 16), dtype=torch.uint8, device=q.device)


def prefix_attn_bwd(q, kv: PagedKV, d_out, out, lse, *, prefix_len: int, q_pos0: int,
                    scale: float, kv_begin: int = 0, kv_end=None, flags: int = 0, dq=None,
                    dk_resp=None, dv_resp=None, workspace=None, expected_epoch=None,
                    stream=None):
    """ls_prefix_attn_bwd: dq over keys [kv_begin, kv_end) and dK/dV of the
    response keys in that range (rows j - prefix_len of dk_resp / dv_resp)."""
    torch = _torch()
    R, Hq, D = q.shape
    Hkv, Dv = kv.k_pool.shape[2], kv.v_pool.shape[3]
    kv_len = q_pos0 + R
    kv_end = kv_len if kv_end is None else kv_end
    if dq is None:
        dq = torch.empty((R, Hq, D), dtype=torch.float32, device=q.device)
    if kv_end > prefix_len:
        n_resp = kv_len - prefix_len
        if dk_resp is None:
            dk_resp = torch.zeros((n_resp, Hkv, D), dtype=torch.float32, device=q.device)
        if dv_resp is None:
            dv_resp = torch.zeros((n_resp, Hkv, Dv), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = bwd_workspace(q, kv, prefix_len=prefix_len, q_pos0=q_pos0)
    p = make_params(q, kv, prefix_len=prefix_len, q_pos0=q_pos0, scale=scale, flags=flags,
                    expected_epoch=expected_epoch)
    f32 = torch.float32
    check(load_library().ls_prefix_attn_bwd(
        ctypes.byref(p), kv_begin, kv_end, _ptr(d_out, q.dtype, "d_out"), _ptr(out, None, "out"),
        _dtype_code(out), _ptr(lse, f32, "lse"), _ptr(dq, f32, "dq"),
        _ptr(dk_resp, f32, "dk_resp"), _ptr(dv_resp, f32, "dv_resp"),
        _ptr(workspace, None, "workspace"), workspace.numel() * workspace.element_size(),
        _stream(stream)))
    return dq, dk_resp, dv_resp


# ----------------------------------------------------------------- sparse latent replay
def _sparse_params(q, latent: PagedKV, *, prefix_len, q_pos0, scale, flags=0):
    p = make_params(q, latent, prefix_len=prefix_len, q_pos0=q_pos0, scale=scale, flags=flags)
    p.head_dim_v = 512
    return p


def sparse_workspace(q, latent: PagedKV, topk: int, *, prefix_len: int, q_pos0: int,
                     backward: bool):
    torch = _torch()
    p = _sparse_params(q, latent, prefix_len=prefix_len, q_pos0=q_pos0, scale=1.0)
    n = load_library().ls_sparse_attn_workspace_size(ctypes.byref(p), topk, int(backward))
    return torch.empty(max(n, 16), dtype=torch.uint8, device=q.device)


def sparse_attn_fwd(q, latent: PagedKV, idx, *, prefix_len: int, q_pos0: int, scale: float,
                    flags: int = 0, out=None, lse=None, workspace=None, stream=None):
    """ls_sparse_attn_fwd: out [R, H, 512] fp32, lse [H, R] fp32.  `latent` holds the
    latent pool as both k_pool and v_pool."""
    torch = _torch()
    R, H = q.shape[0], q.shape[1]
    topk = 0 if idx is None else idx.shape[1]
    if out is None:
        out = torch.empty((R, H, 512), dtype=torch.float32, device=q.device)
    if lse is None:
        lse = torch.empty((H, R), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = sparse_workspace(q, latent, topk, prefix_len=prefix_len, q_pos0=q_pos0,
                                     backward=False)
    p = _sparse_params(q, latent, prefix_len=prefix_len, q_pos0=q_pos0, scale=scale, flags=flags)
    check(load_library().ls_sparse_attn_fwd(ctypes.byref(p), _ptr(idx, torch.int32, "idx"), topk,
                                            _ptr(out, torch.float32, "out"),
                                            _ptr(lse, torch.float32, "lse"),
                                            _ptr(workspace, None, "workspace"),
                                            workspace.numel() * workspace.element_size(),
                                            _stream(stream)))
    return out, lse


def sparse_attn_fwd_noalloc(q, latent: PagedKV, idx, *, out, lse, prefix_len: int, q_pos0: int,
                            scale: float, flags: int = 0, stream=None):
    """ls_sparse_attn_fwd_noalloc: the sparse forward into caller-provided out
    [R, H, 512] and lse [H, R] (fp32), with no workspace; nothing is allocated
    here either."""
    torch = _torch()
    topk = 0 if idx is None else idx.shape[1]
    p = _sparse_params(q, latent, prefix_len=prefix_len, q_pos0=q_pos0, scale=scale, flags=flags)
    check(load_library().ls_sparse_attn_fwd_noalloc(ctypes.byref(p),
                                                    _ptr(idx, torch.int32, "idx"), topk,
                                                    _ptr(out, torch.float32, "out"),
                                                    _ptr(lse, torch.float32, "lse"),
                                                    _stream(stream)))
    return out, lse


def sparse_attn_bwd(q, latent: PagedKV, idx, d_out, out, lse, *, prefix_len: int, q_pos0: int,
                    scale: float, flags: int = 0, dq=None, workspace=None, stream=None):
    """ls_sparse_attn_bwd: dq [R, H, 576] fp32."""
    torch = _torch()
    R, H = q.shape[0], q.shape[1]
    topk = 0 if idx is None else idx.shape[1]
    if dq is None:
        dq = torch.empty((R, H, 576), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = sparse_workspace(q, latent, topk, prefix_len=prefix_len, q_pos0=q_pos0,
                                     backward=True)
    p = _sparse_params(q, latent, prefix_len=prefix_len, q_pos0=q_pos0, scale=scale, flags=flags)
    check(load_library().ls_sparse_attn_bwd(ctypes.byref(p), _ptr(idx, torch.int32, "idx"), topk,
                                            _ptr(d_out, torch.bfloat16, "d_out"),
                                            _ptr(out, None, "out"), _dtype_code(out),
                                            _ptr(lse, torch.float32, "lse"),
                                            _ptr(dq, torch.float32, "dq"),
                                            _ptr(workspace, None, "workspace"),
                                            workspace.numel() * workspace.element_size(),
                                            _stream(stream)))
    return dq


def dsa_index_scores(q_index, w_index, k_index_pool, page_table, *, pos_begin: int, pos_end: int,
                     scores=None, stream=None):
    """ls_dsa_index_scores: I [n_q, pos_end - pos_begin] fp32 (or into ``scores``,
    a [n_q, ld] view with ld a multiple of 4)."""
    torch = _torch()
    n_q, H, d = q_index.shape
    n = pos_end - pos_begin
    if scores is None:
        scores = torch.empty((n_q, max(4, n + (-n) % 4)), dtype=torch.float32,
                             device=q_index.device)
    p = DsaParams(_ptr(q_index, torch.bfloat16, "q_index"), _ptr(w_index, torch.float32, "w_index"),
                  _ptr(k_index_pool, torch.bfloat16, "k_index_pool"),
                  _ptr(page_table, torch.int32, "page_table"), k_index_pool.shape[0],
                  page_table.shape[0], n_q, H, d, k_index_pool.shape[1])
    check(load_library().ls_dsa_index_scores(ctypes.byref(p), pos_begin, pos_end,
                                             _ptr(scores, torch.float32, "scores", dense=False),
                                             scores.stride(0), _stream(stream)))
    return scores[:, :n]


def topk_select(scores, k: int, *, n: int | None = None, positions=None, pos_offset: int = 0,
                out_pos=None, out_scores=None, stream=None):
    """ls_topk_select over the rows of ``scores`` [rows, >= n] (row stride ld):
    positions [rows, k] int32 ascending and their scores [rows, k] (outputs may
    be column slices of wider arrays: their row stride is passed on)."""
    torch = _torch()
    rows = scores.shape[0]
    n = scores.shape[1] if n is None else n
    if out_pos is None:
        out_pos = torch.empty((rows, k), dtype=torch.int32, device=scores.device)
    if out_scores is None:
        out_scores = torch.empty((rows, k), dtype=torch.float32, device=scores.device)
    # the library takes one row stride for the two outputs and one for scores and positions
    if out_pos.stride(0) != out_scores.stride(0) or out_pos.stride(1) != 1 \
            or out_scores.stride(1) != 1:
        raise ValueError("topk_select: out_pos and out_scores must share one row stride and "
                         "have unit column stride")
    if positions is not None and positions.stride(0) != scores.stride(0):
        raise ValueError("topk_select: positions must have the row stride of scores")
    check(load_library().ls_topk_select(
        _ptr(scores, torch.float32, "scores", dense=False), scores.stride(0),
        _ptr(positions, torch.int32, "positions", dense=False), rows, n, pos_offset, k,
        _ptr(out_pos, torch.int32, "out_pos", dense=False),
        _ptr(out_scores, torch.float32, "out_scores", dense=False), out_pos.stride(0),
        _stream(stream)))
    return out_pos, out_scores


def hbm_read_probe(buf, out=None, *, stream=None):
    """Read every byte of ``buf`` once (ls_hbm_read_probe); returns the int32
    device word holding the XOR of its 32-bit words."""
    torch = _torch()
    if out is None:
        out = torch.zeros(1, dtype=torch.int32, device=buf.device)
    else:
        out.zero_()
    check(load_library().ls_hbm_read_probe(_ptr(buf, name="buf"), buf.numel() * buf.element_size(),
                                           _ptr(out, torch.int32, "out"), _stream(stream)))
    return out
