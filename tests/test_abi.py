"""C ABI of liblongstraw.so on the CPU: the library loads, exports every symbol
the header declares, and rejects bad arguments on the host before any launch."""
import ctypes
import os
import re

import pytest

from paper_2607_14952_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "longstraw.h")

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH),
                                reason="liblongstraw.so not built (run __graft_entry__.build())")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ls_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_symbols() == sorted(B.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(B.LIB_PATH)
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_only_ls_symbols_are_exported():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True,
                         text=True).stdout
    funcs = [l.split()[-1] for l in out.splitlines() if " T " in l]
    assert sorted(f for f in funcs if f.startswith("ls_")) == declared_symbols()
    assert all(f.startswith("ls_") or f.startswith("_") for f in funcs), funcs


def test_version_and_status_strings():
    lib = B.load_library()
    assert lib.ls_abi_version() == B.ABI_VERSION
    for code, name in B.STATUS.items():
        assert lib.ls_status_string(code).decode() == name


FAKE = 1 << 20   # 16-byte aligned addresses that are never dereferenced


def good_params(**kw):
    p = B.AttnParams()
    p.abi_version = B.ABI_VERSION
    p.dtype = B.LS_BF16
    p.n_q, p.n_q_heads, p.n_kv_heads = 64, 16, 2
    p.head_dim = p.head_dim_v = 256
    p.page_size = 256
    p.n_phys_pages = p.n_logical_pages = 64
    p.prefix_len = p.q_pos0 = 4096
    p.softmax_scale = 1 / 16
    p.flags = 0
    p.q = FAKE
    p.k_pool = FAKE * 64
    p.v_pool = FAKE * 128
    p.page_table = FAKE * 192
    p.pool_epoch = p.expected_epoch = 3
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def fwd(p, splits=((0, 4096), (4096, 4160)), out=FAKE * 256, lse=FAKE * 320):
    lib = B.load_library()
    arr = (B.Split * len(splits))(*[B.Split(b, e) for b, e in splits])
    return lib.ls_prefix_attn_fwd(ctypes.byref(p), arr, len(splits), out, lse, None)


@pytest.mark.parametrize("kw,status", [
    (dict(abi_version=99), -1),
    (dict(dtype=7), -2),
    (dict(n_q_heads=15), -1),
    (dict(head_dim=128, head_dim_v=128), -2),
    (dict(page_size=96), -2),
    (dict(page_size=0), -1),
    (dict(q_pos0=100), -1),                      # q_pos0 < prefix_len
    (dict(n_logical_pages=16), -1),              # kv_len beyond the logical store
    (dict(q=FAKE + 8), -1),                      # misaligned
    (dict(k_pool=0), -1),
    (dict(softmax_scale=-1.0), -1),
    (dict(expected_epoch=2), -5),                # stale pool
    (dict(n_q_heads=16 * 3, n_kv_heads=1), -2),  # bf16 group 48 does not divide 32
    (dict(n_q=1, n_q_heads=32768, n_kv_heads=32768), -2),  # pool rows of 2^24 bytes
])
def test_forward_rejects(kw, status):
    assert fwd(good_params(**kw)) == status
    assert B.load_library().ls_last_error()


@pytest.mark.parametrize("splits", [
    ((0, 4096), (4000, 4160)),      # overlapping
    ((4096, 4160), (0, 4096)),      # unsorted
    ((0, 0),),                      # empty
    ((0, 5000),),                   # beyond kv_len
    ((-4, 10),),
])
def test_forward_rejects_bad_splits(splits):
    assert fwd(good_params(), splits) == -1


def test_forward_rejects_aliased_outputs():
    assert fwd(good_params(), out=FAKE) == -4               # out_part over q
    assert fwd(good_params(), out=FAKE * 256, lse=FAKE * 256) == -4


def test_merge_rejects():
    lib = B.load_library()
    args = (FAKE, FAKE * 64, 4, 16, 16, 256, B.LS_BF16, FAKE * 128, FAKE * 192, 0, None)
    assert lib.ls_lse_merge(*args[:6], 5, *args[7:]) == -2                      # out dtype
    assert lib.ls_lse_merge(*args[:5], 254, *args[6:]) == -2                    # dv % 4
    assert lib.ls_lse_merge(*args[:9], 2, None) == -2                           # flags
    assert lib.ls_lse_merge(FAKE, FAKE * 64, 4, 16, 16, 256, B.LS_BF16, FAKE + 64,
                            FAKE * 192, 0, None) == -4                          # out inside part
    assert lib.ls_lse_merge(FAKE, FAKE * 64, 0, 16, 16, 256, B.LS_BF16, FAKE * 128,
                            FAKE * 192, 0, None) == -1


def test_backward_rejects():
    lib = B.load_library()
    p = good_params()
    need = lib.ls_prefix_attn_bwd_workspace_size(ctypes.byref(p))
    assert need >= 2 * 64 * 16 * 4
    base = dict(d_out=FAKE * 400, out=FAKE * 420, lse=FAKE * 440, dq=FAKE * 460,
                dk=FAKE * 480, dv=FAKE * 500, ws=FAKE * 520)

    def call(p=p, kb=0, ke=4160, out_dtype=B.LS_BF16, ws_bytes=need, **kw):
        a = dict(base, **kw)
        return lib.ls_prefix_attn_bwd(ctypes.byref(p), kb, ke, a["d_out"], a["out"], out_dtype,
                                      a["lse"], a["dq"], a["dk"], a["dv"], a["ws"], ws_bytes, None)

    assert call(ws_bytes=need - 4) == -3
    assert call(ws=None) == -3
    assert call(dk=None) == -1                    # range holds response keys
    assert call(ke=5000) == -1
    assert call(kb=10, ke=5) == -1
    assert call(out_dtype=9) == -2
    assert call(dq=FAKE * 420) == -4              # dq over out
    assert call(p=good_params(expected_epoch=9)) == -5


def test_gather_rejects():
    lib = B.load_library()
    p = good_params(n_q=0)
    assert lib.ls_gather_kv(ctypes.byref(p), 10, 5, FAKE * 300, FAKE * 400, None) == -1
    assert lib.ls_gather_kv(ctypes.byref(p), 0, 64 * 256 + 1, FAKE * 300, FAKE * 400, None) == -1
    assert lib.ls_gather_kv(ctypes.byref(p), 0, 16, FAKE * 64, FAKE * 400, None) == -4
    assert lib.ls_gather_kv(ctypes.byref(p), 0, 0, FAKE * 300, FAKE * 400, None) == 0


def test_scatter_rejects():
    lib = B.load_library()
    p = good_params(n_q=0)
    # source overlapping the K pool, bad ranges
    assert lib.ls_scatter_kv(ctypes.byref(p), 0, 16, FAKE * 64, FAKE * 400, None) == -4
    assert lib.ls_scatter_kv(ctypes.byref(p), 10, 5, FAKE * 300, FAKE * 400, None) == -1
    assert lib.ls_scatter_kv(ctypes.byref(p), 0, 64 * 256 + 1, FAKE * 300, FAKE * 400, None) == -1
    assert lib.ls_scatter_kv(ctypes.byref(p), 0, 0, FAKE * 300, FAKE * 400, None) == 0
    assert lib.ls_scatter_kv(ctypes.byref(p), 0, 16, 0, FAKE * 400, None) == -1


def _dsa_params(**kw):
    f = dict(q_index=FAKE, w_index=FAKE * 16, k_index_pool=FAKE * 32, page_table=FAKE * 64,
             n_phys_pages=256, n_logical_pages=256, n_q=64, n_heads=32, head_dim=128,
             page_size=64)
    f.update(kw)
    return B.DsaParams(**f)


@pytest.mark.parametrize("kw,rng,status", [
    (dict(head_dim=64), (0, 4096), -2),
    (dict(n_heads=12), (0, 4096), -2),
    (dict(page_size=16), (0, 4096), -2),
    (dict(), (16, 4096), -1),                  # pos_begin not a multiple of 32
    (dict(), (0, 256 * 64 + 1), -1),           # beyond the table
    (dict(), (4096, 0), -1),
])
def test_dsa_scores_rejects(kw, rng, status):
    lib = B.load_library()
    p = _dsa_params(**kw)
    assert lib.ls_dsa_index_scores(ctypes.byref(p), rng[0], rng[1], FAKE * 1024, 4096, None) == status
    assert lib.ls_last_error()


def test_dsa_scores_rejects_ld_and_alias():
    lib = B.load_library()
    p = _dsa_params()
    assert lib.ls_dsa_index_scores(ctypes.byref(p), 0, 4096, FAKE * 1024, 4095, None) == -1
    assert lib.ls_dsa_index_scores(ctypes.byref(p), 0, 4096, FAKE * 1024, 4094, None) == -1
    assert lib.ls_dsa_index_scores(ctypes.byref(p), 0, 4096, FAKE * 32, 4096, None) == -4


def test_topk_rejects():
    lib = B.load_library()
    ok = (FAKE, 1000, None, 4, 1000, 0, 16, FAKE * 64, FAKE * 96, 16, None)
    assert lib.ls_topk_select(*ok[:6], 0, *ok[7:]) == -1                         # k = 0
    assert lib.ls_topk_select(*ok[:9], 15, None) == -1                           # out_ld < k
    assert lib.ls_topk_select(FAKE, 999, None, 4, 1000, 0, 16, FAKE * 64, None, 16,
                              None) == -1                                       # ld < n
    assert lib.ls_topk_select(FAKE, 1000, None, 4, 1000, (1 << 31) - 10, 16, FAKE * 64, None,
                              16, None) == -1                                   # positions >= 2^31
    assert lib.ls_topk_select(FAKE, 1000, None, 4, 1000, 0, 16, FAKE + 64, None, 16, None) == -4
    assert lib.ls_topk_select(FAKE, 1000, None, 0, 1000, 0, 16, FAKE * 64, None, 16, None) == 0


# ------------------------------------------------------------ binding argument checks
class _FakeTensor:
    """Just enough of a tensor for the binding's pointer checks."""

    def __init__(self, dtype, cuda=True, contiguous=True, last_stride=1):
        self.dtype, self.is_cuda = dtype, cuda
        self._contig, self._last = contiguous, last_stride
        self.device = "cuda:0" if cuda else "cpu"

    def is_contiguous(self):
        return self._contig

    def dim(self):
        return 2

    def stride(self, i):
        return self._last if i == -1 else 64

    def data_ptr(self):
        return 0x1000


def test_binding_checks_device_dtype_and_layout():
    """A host tensor would reach a kernel as a host address, a wrong dtype would be
    reinterpreted and a strided tensor misread: the binding refuses all three before
    calling the library."""
    import torch
    f32 = torch.float32
    assert B._ptr(None) is None
    assert B._ptr(_FakeTensor(f32), f32, "x") == 0x1000
    with pytest.raises(ValueError, match="GPU tensor"):
        B._ptr(_FakeTensor(f32, cuda=False), f32, "x")
    with pytest.raises(TypeError, match="must be torch.float32"):
        B._ptr(_FakeTensor(torch.bfloat16), f32, "x")
    with pytest.raises(ValueError, match="contiguous"):
        B._ptr(_FakeTensor(f32, contiguous=False), f32, "x")
    # row-strided views: only the last dimension has to be unit-stride
    assert B._ptr(_FakeTensor(f32, contiguous=False), f32, "x", dense=False) == 0x1000
    with pytest.raises(ValueError, match="unit stride"):
        B._ptr(_FakeTensor(f32, contiguous=False, last_stride=2), f32, "x", dense=False)
    # through an entry point: host tensors are refused before anything is launched
    q = torch.zeros((4, 2, 64), dtype=f32)
    pool = torch.zeros((2, 64, 1, 64), dtype=f32)
    kv = B.PagedKV(pool, pool, torch.zeros(2, dtype=torch.int32))
    with pytest.raises(ValueError, match="GPU tensor"):
        B.prefix_attn_fwd(q, kv, [(0, 4)], prefix_len=0, q_pos0=0, scale=0.125)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.topk_select(torch.zeros((2, 8)), 3)
    # one row stride for both outputs, one for scores and positions
    wide = torch.zeros((2, 10), dtype=torch.int32)
    with pytest.raises(ValueError, match="share one row stride"):
        B.topk_select(torch.zeros((2, 8)), 3, out_pos=wide[:, :3],
                      out_scores=torch.zeros((2, 3)))
    with pytest.raises(ValueError, match="row stride of scores"):
        B.topk_select(torch.zeros((2, 8)), 3, positions=torch.zeros((2, 9), dtype=torch.int32))


def test_sparse_noalloc_rejects_on_the_host():
    """The allocation-free sparse forward refuses checked mode and calls whose
    key lists exceed its scratch array, before touching the GPU."""
    lib = B.load_library()
    p = good_params(head_dim=576, head_dim_v=512, n_kv_heads=1, n_q_heads=128, page_size=64,
                    n_phys_pages=4096, n_logical_pages=4096, prefix_len=65536, q_pos0=65536,
                    n_q=16)
    p.v_pool = p.k_pool
    idx, out, lse = FAKE * 512, FAKE * 576, FAKE * 1024
    p.flags = B.FLAG_CHECKED
    assert lib.ls_sparse_attn_fwd_noalloc(ctypes.byref(p), idx, 64, out, lse, None) == -2
    p.flags = 0
    # 16 rows x (64 selections + a window of 2^22 response positions) x 4 bytes > 64 MiB
    big = good_params(**{k: getattr(p, k) for k in ("head_dim", "head_dim_v", "n_kv_heads",
                                                     "n_q_heads", "page_size", "n_phys_pages",
                                                     "prefix_len", "n_q")})
    big.v_pool = big.k_pool
    big.q_pos0 = p.prefix_len + (1 << 22)
    big.n_logical_pages = (big.q_pos0 + 16) // 64 + 1
    assert lib.ls_sparse_attn_fwd_noalloc(ctypes.byref(big), idx, 64, out, lse, None) == -3
    assert b"scratch" in lib.ls_last_error()
