"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments synchronously (before any HIP call,
so these run on a machine without a device)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "losa.h")


@pytest.fixture(scope="module")
def L():
    from paper_2608_12032_amd import losa
    return losa


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(losa_\w+)\s*\(", text)))


def test_header_declares_the_three_entry_points():
    names = declared_functions()
    for n in ("losa_calibrate_mass", "losa_select_blocks", "losa_sparse_attn_fwd"):
        assert n in names


def test_library_exports_every_declared_symbol(L):
    lib = ctypes.CDLL(L.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in losa.h but not exported"
    assert set(declared_functions()) == set(L.EXPORTED)


def test_status_strings_and_version(L):
    for code, name in L.STATUS.items():
        assert L.lib.losa_status_string(code).decode() == name
    assert L.lib.losa_version() == 100


FAKE = 0x10000          # never dereferenced: every call below fails validation first
MIS = 0x10001           # misaligned


def _cal(L, q=FAKE, k=FAKE, dtype=1, B=1, H=2, N=1000, d=128, bq=128, bk=128, scale=0.1,
         mass=FAKE, lse=None, ws=None, wsb=0):
    return L.lib.losa_calibrate_mass(q, k, dtype, B, H, N, d, bq, bk, scale, mass, lse, ws, wsb,
                                     None)


def _sel(L, mass=FAKE, B=1, H=2, N=1000, bq=128, bk=128, tau=0.99, rp=FAKE, ci=FAKE, cap=10**6,
         ws=FAKE, wsb=10**7):
    return L.lib.losa_select_blocks(mass, B, H, N, bq, bk, tau, rp, ci, cap, ws, wsb, None)


def _fwd(L, q=FAKE, dtype=1, B=1, H=2, N=1000, d=128, bq=128, bk=128, rp=FAKE, ci=FAKE, cl=100,
         o=FAKE, ws=FAKE, wsb=10**9, scale=0.1):
    return L.lib.losa_sparse_attn_fwd(q, q, q, dtype, B, H, N, d, bq, bk, scale, rp, ci, cl, o,
                                      None, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), 1), (dict(mass=None), 1),
    (dict(B=0), 2), (dict(N=-5), 2), (dict(d=0), 2), (dict(bq=96), 2), (dict(bk=512), 2),
    (dict(scale=float("nan")), 2), (dict(q=MIS), 4), (dict(lse=MIS), 4),
    (dict(d=96), 5), (dict(bq=128, bk=64), 5), (dict(bq=32, bk=32), 5), (dict(dtype=7), 5),
    (dict(N=1 << 30, d=128), 2),
    # the optional bf16 workspace: aligned, and at least one head's share
    (dict(ws=MIS, wsb=10**9), 4), (dict(ws=FAKE, wsb=100), 6),
])
def test_calibrate_validation(L, kw, code):
    assert _cal(L, **kw) == code
    assert L.lib.losa_last_error().decode() != ""


@pytest.mark.parametrize("kw,code", [
    (dict(mass=None), 1), (dict(ws=None), 1), (dict(ci=None), 1),
    (dict(tau=0.0), 3), (dict(tau=-0.5), 3), (dict(tau=1.5), 3), (dict(tau=float("nan")), 3),
    (dict(cap=2 * 8 * 8 - 1), 6), (dict(wsb=10), 6), (dict(rp=MIS), 4),
    (dict(H=0), 2), (dict(bq=100), 2),
])
def test_select_validation(L, kw, code):
    assert _sel(L, **kw) == code


def test_select_capacity_is_checked_against_worst_case(L):
    # N=1000, block 128 -> N_pad 1024, n_q = n_k = 8, rows = B*H*n_q = 16
    assert _sel(L, cap=16 * 8 - 1) == 6
    ws_need = L.workspace_bytes(1, 0, 1, 2, 1000, 1, 128, 128)
    assert ws_need >= 16 * 4 + 16 * 8
    assert _sel(L, cap=16 * 8, wsb=ws_need - 1) == 6


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), 1), (dict(rp=None), 1), (dict(o=None), 1), (dict(ci=None), 1),
    (dict(cl=-1), 2), (dict(B=-1), 2), (dict(q=MIS), 4), (dict(o=MIS), 4), (dict(ws=MIS), 4),
    (dict(d=80), 5), (dict(bq=64, bk=128), 5), (dict(ws=None), 1), (dict(wsb=1), 6),
    # more than 4096 key blocks per head: beyond the per-row LDS flags (both dtypes)
    (dict(N=4097 * 128, d=64), 5), (dict(N=4097 * 128, d=64, dtype=0), 5),
])
def test_fwd_validation(L, kw, code):
    assert _fwd(L, **kw) == code


def _fwd_na(L, q=FAKE, dtype=1, B=1, H=2, N=1000, d=128, bq=128, bk=128, rp=FAKE, ci=FAKE,
            cl=100, o=FAKE, scale=0.1):
    return L.lib.losa_sparse_attn_fwd_noalloc(q, q, q, dtype, B, H, N, d, bq, bk, scale, rp, ci,
                                              cl, o, None, None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), 1), (dict(rp=None), 1), (dict(o=None), 1), (dict(ci=None), 1),
    (dict(cl=-1), 2), (dict(B=-1), 2), (dict(q=MIS), 4), (dict(d=80), 5),
    # scratch beyond the 128 MiB the library holds: the HunyuanVideo shape's V^T
    (dict(B=1, H=24, N=118800), 6), (dict(B=2, H=12, N=32760), 6),
])
def test_fwd_noalloc_validation(L, kw, code):
    assert _fwd_na(L, **kw) == code
    if code == 6:
        assert "scratch" in L.lib.losa_last_error().decode()


def test_fwd_noalloc_scratch_limit(L):
    # the Wan shape (96 MiB of V^T plus the dispatch order) fits; 16 more
    # heads of it do not
    fits = L.workspace_bytes(2, 1, 1, 12, 32760, 128, 128, 128)
    assert fits <= L.NOALLOC_SCRATCH_BYTES < L.workspace_bytes(2, 1, 1, 16, 32760, 128, 128, 128)
    assert _fwd_na(L, H=16, N=32760) == 6


def _topk(L, mass=FAKE, B=1, H=2, N=1000, bq=128, bk=32, k=5, rp=FAKE, ci=FAKE, cap=10**6,
          ws=FAKE, wsb=10**7):
    return L.lib.losa_select_blocks_topk(mass, B, H, N, bq, bk, k, rp, ci, cap, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(k=0), 2), (dict(k=-3), 2), (dict(mass=None), 1), (dict(ws=None), 1),
    (dict(cap=16 * 32 - 1), 6), (dict(wsb=10), 6), (dict(ci=MIS), 4), (dict(bq=100), 2),
])
def test_select_topk_validation(L, kw, code):
    # N=1000, blocks 128 x 32 -> N_pad 1024, rows 16, n_k 32
    assert _topk(L, **kw) == code


def _rec(L, mass=FAKE, B=1, H=2, N=1000, bq=128, bk=128, rp=FAKE, ci=FAKE, cl=100, rows=FAKE,
         heads=FAKE, ws=FAKE, wsb=10**6):
    return L.lib.losa_block_recall(mass, B, H, N, bq, bk, rp, ci, cl, rows, heads, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(mass=None), 1), (dict(rp=None), 1), (dict(ws=None), 1), (dict(ci=None), 1),
    (dict(cl=-1), 2), (dict(H=0), 2), (dict(rows=MIS), 4), (dict(heads=MIS), 4),
    (dict(wsb=16 * 16 - 1), 6), (dict(N=4097 * 128), 5),
])
def test_recall_validation(L, kw, code):
    assert _rec(L, **kw) == code


def _con(L, q=FAKE, dtype=1, B=1, H=2, N=1000, d=128, bq=128, bk=128, o=FAKE, mass=FAKE,
         lse=None, ws=FAKE, wsb=10**9, scale=0.1):
    return L.lib.losa_construct(q, q, q, dtype, B, H, N, d, bq, bk, scale, o, mass, lse, ws, wsb,
                                None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), 1), (dict(o=None), 1), (dict(mass=None), 1), (dict(ws=None), 1),
    (dict(B=0), 2), (dict(scale=0.0), 2), (dict(o=MIS), 4), (dict(lse=MIS), 4),
    (dict(d=96), 5), (dict(bq=128, bk=64), 5), (dict(wsb=100), 6),
])
def test_construct_validation(L, kw, code):
    assert _con(L, **kw) == code


def test_workspace_sizes(L):
    B, H, N, d = 1, 12, 32760, 128
    up = lambda x: (x + 255) // 256 * 256  # noqa: E731
    stat_head = 256 * 32768 * 4              # one fp32 per (query, key block) of a head
    one_cal = up(stat_head) + up(32768 * 4)  # statistics, lse
    assert L.workspace_bytes(0, 1, 1, 1, N, d, 128, 128) == one_cal
    assert L.workspace_bytes(0, 1, B, H, N, d, 128, 128) == H * one_cal
    assert L.workspace_bytes(0, 0, B, H, N, d, 128, 128) == 0
    # 32-key blocks: four times the statistics
    assert L.workspace_bytes(0, 1, 1, 1, N, d, 128, 32) == up(4 * stat_head) + up(32768 * 4)
    # the suggestion stops at 16 GiB worth of whole heads
    big = L.workspace_bytes(0, 1, 1, 600, N, d, 128, 128)
    assert big == (16 << 30) // one_cal * one_cal
    assert L.workspace_bytes(2, 1, B, H, N, d, 128, 128) == B * H * 32768 * d * 2 + B * H * 256 * 4
    assert L.workspace_bytes(2, 0, B, H, N, d, 128, 128) == 0
    rows, n_k = 12 * 256, 256
    assert L.workspace_bytes(1, 0, B, H, N, 1, 128, 128) == ((rows * 4 + 255) // 256) * 256 + rows * n_k
    assert L.workspace_bytes(3, 0, B, H, N, 1, 128, 128) == rows * 16
    one_con = one_cal + up(L.workspace_bytes(2, 1, 1, 1, N, d, 128, 128))  # + V^T and order
    assert L.workspace_bytes(4, 1, 1, 1, N, d, 128, 128) == one_con
    assert L.workspace_bytes(4, 1, B, H, N, d, 128, 128) == H * one_con
    assert L.workspace_bytes(4, 0, B, H, N, d, 128, 128) == 0
    assert L.workspace_bytes(5, 1, B, H, N, d, 128, 128) == 0
    assert L.workspace_bytes(2, 1, 0, H, N, d, 128, 128) == 0


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    import importlib
    import paper_2608_12032_amd.losa as mod
    monkeypatch.setattr(mod, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        mod._load()
