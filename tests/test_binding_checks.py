"""The Python binding rejects bad tensor arguments before any pointer reaches
the library (which cannot tell a host pointer, a wrong element type or a short
buffer from a valid one).  The host-tensor cases run on the CPU; the rest need
device tensors and are marked gpu (nothing is launched in them)."""
import pytest
import torch


@pytest.fixture(scope="module")
def L():
    from paper_2608_12032_amd import losa
    return losa


def test_host_tensors_are_rejected(L):
    q = torch.zeros((1, 2, 128, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="must live on"):
        L.losa_calibrate_mass(q, q, 100, 128)
    with pytest.raises(ValueError, match="must live on"):
        L.losa_sparse_attn_fwd(q, q, q, 100, 128, 128, torch.zeros(3, dtype=torch.int32),
                               torch.zeros(4, dtype=torch.int32))
    mass = torch.zeros((1, 2, 1, 1))
    with pytest.raises(ValueError, match="must live on"):
        L.losa_select_blocks(mass, 100, 128, 128, 0.99)


@pytest.mark.gpu
def test_device_argument_checks(L):
    dev = "cuda"
    B, H, N, d, C = 1, 2, 200, 128, 128
    Np = L.padded_len(N, C, C)
    q = torch.zeros((B, H, Np, d), dtype=torch.bfloat16, device=dev)
    n_q = Np // C
    rp = torch.zeros(B * H * n_q + 1, dtype=torch.int32, device=dev)
    ci = torch.zeros(B * H * n_q * n_q, dtype=torch.int32, device=dev)
    mass = torch.zeros((B, H, n_q, n_q), dtype=torch.float32, device=dev)
    cases = [
        # N_pad of q does not match N and the block sizes
        (lambda: L.losa_calibrate_mass(q, q, N + 128, C), ValueError, "N_pad"),
        # k of another dtype, v of another shape
        (lambda: L.losa_calibrate_mass(q, q.float(), N, C), TypeError, "k must be"),
        (lambda: L.losa_sparse_attn_fwd(q, q, q[:, :1].contiguous(), N, C, C, rp, ci),
         ValueError, "v must have shape"),
        # a non-contiguous operand
        (lambda: L.losa_sparse_attn_fwd(q, q.transpose(2, 3).contiguous().transpose(2, 3), q,
                                        N, C, C, rp, ci), ValueError, "contiguous"),
        # CSR of the wrong type or too short
        (lambda: L.losa_sparse_attn_fwd(q, q, q, N, C, C, rp.long(), ci), TypeError, "row_ptr"),
        (lambda: L.losa_sparse_attn_fwd(q, q, q, N, C, C, rp[:-1], ci), ValueError, "row_ptr"),
        # output buffers of the wrong shape / a short workspace
        (lambda: L.losa_sparse_attn_fwd(q, q, q, N, C, C, rp, ci, out=q[:, :1].contiguous()),
         ValueError, "out must have shape"),
        (lambda: L.losa_sparse_attn_fwd(q, q, q, N, C, C, rp, ci,
                                        workspace=torch.empty(16, dtype=torch.uint8, device=dev)),
         ValueError, "workspace holds"),
        (lambda: L.losa_calibrate_mass(q, q, N, C, mass=mass[:, :1].contiguous()), ValueError,
         "mass must have shape"),
        # masses whose shape does not match N and the block sizes
        (lambda: L.losa_select_blocks(mass, N + 256, C, C, 0.99), ValueError,
         "mass must have shape"),
        (lambda: L.losa_select_blocks(mass.double(), N, C, C, 0.99), TypeError, "mass must be"),
        (lambda: L.losa_block_recall(mass, N, C, C, rp[:1], ci), ValueError, "row_ptr"),
    ]
    for fn, exc, msg in cases:
        with pytest.raises(exc, match=msg):
            fn()
