"""losa_sparse_attn_fwd_noalloc through the C ABI against losa_sparse_attn_fwd.

The no-alloc entry point runs the same kernels with the library's own scratch
array in place of the caller's workspace, so its output must equal the
workspace entry point's bitwise (stronger than the 2e-2 / 2e-3 output bars).
Two calls in a row on different shapes, the second smaller, check that the
shared scratch carries nothing from one call into the next; a graph capture
replayed between eager calls checks it under capture, where allocation is
not possible; the device's free memory is unchanged across calls.
"""
import ctypes

import numpy as np
import pytest
import torch

from oracle import losa_oracle as O
from paper_2608_12032_amd import workload as W

pytestmark = pytest.mark.gpu

SHAPES = [  # larger first, then smaller: the second call reuses the scratch
    W.WORKLOADS["wan"],                                                        # 96 MiB of scratch
    W.scaled(W.WORKLOADS["cog"], grid=(3, 10, 45), H=4, name="cog-small"),    # d = 64, ragged
    W.rectangular(W.scaled(W.WORKLOADS["wan"], grid=(4, 12, 30), H=3, name="wan-small")),
]


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2608_12032_amd import losa
    return losa


def say(msg):
    print(f"[gpu-noalloc] {msg}", flush=True)


def f64(x):
    return x.detach().float().cpu().numpy().astype(np.float64)


def _case(L, w):
    q, k, v = W.make_inputs(w, device="cuda")
    mass, _ = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk, want_lse=False)
    rp, ci = L.losa_select_blocks(mass, w.N, w.block, w.bk, w.tau)
    torch.cuda.synchronize()
    return q, k, v, rp, ci


def _noalloc_raw(L, w, q, k, v, rp, ci, o, lse):
    """The entry point called through ctypes directly (no binding logic)."""
    B, H, Np, d = q.shape
    st = L.lib.losa_sparse_attn_fwd_noalloc(
        ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
        ctypes.c_void_p(v.data_ptr()), L.LOSA_DTYPE_BF16, B, H, w.N, d, w.block, w.bk, w.scale,
        ctypes.c_void_p(rp.data_ptr()), ctypes.c_void_p(ci.data_ptr()), ci.numel(),
        ctypes.c_void_p(o.data_ptr()), ctypes.c_void_p(lse.data_ptr()),
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, L.lib.losa_last_error().decode()


def test_noalloc_equals_workspace_entry_point(L):
    for rnd in range(2):  # the whole sequence twice: the second pass allocates nothing
        for w in SHAPES:
            need = L.workspace_bytes(2, L.LOSA_DTYPE_BF16, w.B, w.H, w.N, w.d, w.block, w.bk)
            assert need <= L.NOALLOC_SCRATCH_BYTES
            say(f"round {rnd}: {w.name} H={w.H} N={w.N} d={w.d} blocks={w.block}x{w.bk}, "
                f"scratch {need / 2**20:.1f} MiB")
            q, k, v, rp, ci = _case(L, w)
            o_ref, l_ref = L.losa_sparse_attn_fwd(q, k, v, w.N, w.block, w.bk, rp, ci,
                                                  want_lse=True)
            o = torch.full_like(q, float("nan"))
            lse = torch.full_like(l_ref, float("nan"))
            torch.cuda.synchronize()
            free0 = torch.cuda.mem_get_info()[0]
            _noalloc_raw(L, w, q, k, v, rp, ci, o, lse)
            torch.cuda.synchronize()
            free1 = torch.cuda.mem_get_info()[0]
            assert torch.equal(o, o_ref), w.name
            assert torch.equal(lse, l_ref), w.name
            if rnd == 1:
                # outputs preallocated, scratch already reserved by the first
                # pass (loading the code on the device): the call takes no
                # device memory
                assert abs(free1 - free0) <= (1 << 20), (w.name, free0 - free1)
            # and the oracle on a few rows, so the equality is not of two wrong results
            rows = [0, w.n_blocks - 1, w.B * w.H * w.n_blocks - 1]
            rp_g = rp.cpu().numpy().astype(np.int64)
            ci_g = ci[:int(rp_g[-1])].cpu().numpy().astype(np.int64)
            ref, _ = O.sparse_attention(f64(q), f64(k), f64(v), w.N, w.block, w.bk, w.scale,
                                        rp_g, ci_g, rows_subset=rows)
            og = f64(o).reshape(-1, w.d)
            n_q = w.n_blocks
            for r in rows:
                base = (r // n_q) * w.N_pad + (r % n_q) * w.block
                hi = min((r % n_q + 1) * w.block, w.N) - (r % n_q) * w.block
                err = np.abs(og[base:base + hi] - ref.reshape(-1, w.d)[base:base + hi])
                assert err.max() <= 2e-2 and err.mean() <= 2e-3, (w.name, r)
            del q, k, v, o, o_ref


def test_noalloc_under_graph_capture(L):
    w = SHAPES[2]
    q, k, v, rp, ci = _case(L, w)
    o_ref = L.losa_sparse_attn_fwd(q, k, v, w.N, w.block, w.bk, rp, ci)
    o = torch.empty_like(q)
    lse = torch.empty((w.B, w.H, w.N_pad), dtype=torch.float32, device="cuda")
    L.losa_sparse_attn_fwd_noalloc(q, k, v, w.N, w.block, w.bk, rp, ci, out=o)  # first call
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    o.zero_()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            L.losa_sparse_attn_fwd_noalloc(q, k, v, w.N, w.block, w.bk, rp, ci, out=o,
                                           want_lse=True, lse=lse)
    torch.cuda.current_stream().wait_stream(s)
    other = SHAPES[1]
    for rep in range(3):
        o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o, o_ref), rep
        # eager no-alloc work of another shape between replays: the scratch is
        # rewritten, and the next replay must not depend on what it held
        q2, k2, v2, rp2, ci2 = _case(L, other)
        o2 = L.losa_sparse_attn_fwd_noalloc(q2, k2, v2, other.N, other.block, other.bk, rp2, ci2)
        o2_ref = L.losa_sparse_attn_fwd(q2, k2, v2, other.N, other.block, other.bk, rp2, ci2)
        torch.cuda.synchronize()
        assert torch.equal(o2, o2_ref), rep


def test_noalloc_rejects_shapes_beyond_the_scratch(L):
    w = W.WORKLOADS["hunyuan"]  # 697 MiB of V^T: more than the library holds
    need = L.workspace_bytes(2, L.LOSA_DTYPE_BF16, w.B, w.H, w.N, w.d, w.block, w.bk)
    assert need > L.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((1, 1, 16, 16), dtype=torch.bfloat16, device="cuda")  # never read
    p = ctypes.c_void_p(q.data_ptr())
    st = L.lib.losa_sparse_attn_fwd_noalloc(p, p, p, L.LOSA_DTYPE_BF16, w.B, w.H, w.N, w.d,
                                            w.block, w.bk, w.scale, p, p, 1, p, None, None)
    assert L.STATUS[st] == "LOSA_ERR_CAPACITY"
    assert "scratch" in L.lib.losa_last_error().decode()
