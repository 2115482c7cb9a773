"""The path under HIP graph capture.  No entry point allocates, synchronizes or
records a memset, and each launches only on the stream it is given, so one
whole LoSA cycle (construction step, selection, reuse-step forwards, and the
calibration with either scheme and the top-k rule beside them) can be
captured once and replayed.  Every replay, with eager work and
synchronizations between replays, must equal the eager run bitwise."""
import pytest
import torch

from paper_2608_12032_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2608_12032_amd import losa
    return losa


@pytest.mark.parametrize("block_k", [0, 32])
def test_losa_cycle_replays_from_a_hip_graph(L, block_k):
    w = W.scaled(W.WORKLOADS["wan"], grid=(4, 12, 30), H=3, name="wan-small")
    if block_k:
        w = W.rectangular(w, block_k)
    N, C, Ck, d = w.N, w.block, w.bk, w.d
    state = W.make_state(w, device="cuda")
    q0, k0, v0 = W.cast(state, w)
    steps = []
    for t in range(1, 4):
        W.drift_(state, w, t)
        steps.append(W.cast(state, w))
    dev = q0.device
    rows = w.B * w.H * w.n_blocks
    mass = torch.empty((w.B, w.H, w.n_blocks, w.n_kblocks), dtype=torch.float32, device=dev)
    o0 = torch.empty_like(q0)
    outs = [torch.empty_like(q0) for _ in steps]
    row_ptr = torch.empty(rows + 1, dtype=torch.int32, device=dev)
    col_idx = torch.empty(rows * w.n_kblocks, dtype=torch.int32, device=dev)
    ws_con = torch.empty(L.workspace_bytes(4, 1, w.B, w.H, N, d, C, Ck), dtype=torch.uint8,
                         device=dev)
    ws_sel = torch.empty(L.workspace_bytes(1, 0, w.B, w.H, N, 1, C, Ck), dtype=torch.uint8,
                         device=dev)
    ws_fwd = torch.empty(L.workspace_bytes(2, 1, w.B, w.H, N, d, C, Ck), dtype=torch.uint8,
                         device=dev)
    # the calibration (both schemes) and the top-k rule ride along
    mass1 = torch.empty_like(mass)
    mass2 = torch.empty_like(mass)
    lse1 = torch.empty((w.B, w.H, w.N_pad), dtype=torch.float32, device=dev)
    ws_cal = torch.empty(L.workspace_bytes(0, 1, w.B, w.H, N, d, C, Ck), dtype=torch.uint8,
                         device=dev)
    rk = torch.empty_like(row_ptr)
    ck = torch.empty_like(col_idx)

    def cycle():
        L.losa_construct(q0, k0, v0, N, C, Ck, out=o0, mass=mass, workspace=ws_con)
        L.losa_select_blocks(mass, N, C, Ck, w.tau, row_ptr=row_ptr, col_idx=col_idx,
                             workspace=ws_sel)
        for (q, k, v), o in zip(steps, outs):
            L.losa_sparse_attn_fwd(q, k, v, N, C, Ck, row_ptr, col_idx, out=o, workspace=ws_fwd)
        L.losa_calibrate_mass(q0, k0, N, C, Ck, mass=mass1, lse=lse1, workspace=ws_cal)
        L.losa_calibrate_mass(q0, k0, N, C, Ck, want_lse=False, mass=mass2, two_sweep=True)
        L.losa_select_blocks_topk(mass1, N, C, Ck, 3, row_ptr=rk, col_idx=ck, workspace=ws_sel)

    results = [o0, mass, row_ptr] + outs + [mass1, lse1, mass2, rk]
    cycle()
    torch.cuda.synchronize()
    nnz = int(row_ptr[-1].item())
    nnz_k = int(rk[-1].item())
    ref = [t.clone() for t in results] + [col_idx[:nnz].clone(), ck[:nnz_k].clone()]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        cycle()  # warm-up on the capture stream, as torch asks before capturing
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        cycle()
    torch.cuda.synchronize()

    scratch = torch.randn(1 << 20, device=dev)
    for rep in range(4):
        for t in results + [col_idx, ck]:
            t.zero_()                      # eager work between replays
        scratch.mul_(1.0001).add_(rep)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = [t for t in results] + [col_idx[:nnz], ck[:nnz_k]]
        for a, b in zip(ref, got):
            assert torch.equal(a, b), f"replay {rep} differs from the eager run"
