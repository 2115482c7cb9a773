"""GPU parity at degenerate sequence lengths: N = 1, N shorter than one 32-key
sub-tile, shorter than one block, one key past a block boundary.  Every entry
point of the path on the same inputs, against the oracle on every row:
calibration (both bf16 schemes), selection at tau < 1 and tau = 1, the
sparse forward, the construction step, recall and the top-k rule.  Padding
rows of Q/K/V are zero; padding outputs must be 0 (O) and -inf (lse)."""
import numpy as np
import pytest
import torch

from oracle import compare as CMP
from oracle import losa_oracle as O

pytestmark = pytest.mark.gpu

MASS_TOL, LSE_TOL, REC_TOL = 1e-4, 1e-3, 1e-6
OUT_TOL = {"bf16": (2e-2, 2e-3), "f32": (1e-4, 1e-4)}

CASES = ([("bf16", 128, 128, 128, n) for n in (1, 5, 33, 96, 129)]
         + [("bf16", 128, 128, 32, n) for n in (1, 31, 65)]
         + [("bf16", 64, 64, 64, n) for n in (1, 63)]
         + [("bf16", 64, 128, 32, n) for n in (2, 160)]
         + [("f32", 64, 64, 64, n) for n in (1, 7, 100)]
         + [("f32", 128, 128, 32, n) for n in (1, 40)])


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2608_12032_amd import losa
    return losa


def f64(x):
    return x.detach().float().cpu().numpy().astype(np.float64)


def inputs(dtype, d, N, Cq, Ck, seed):
    B, H = 1, 2
    n_pad = O.padded_len(N, Cq, Ck)
    g = torch.Generator().manual_seed(seed)
    t = torch.randn((3, B, H, n_pad, d), generator=g) * 1.5
    t[:, :, :, N:] = 0
    t = t.to(torch.bfloat16 if dtype == "bf16" else torch.float32).cuda()
    return t[0].contiguous(), t[1].contiguous(), t[2].contiguous()


@pytest.mark.parametrize("dtype,d,Cq,Ck,N", CASES)
def test_short_sequence_every_entry_point(L, dtype, d, Cq, Ck, N):
    q, k, v = inputs(dtype, d, N, Cq, Ck, seed=1000 + N + d + Ck)
    scale = 1.0 / np.sqrt(d)
    print(f"[gpu-short] {dtype} d={d} blocks={Cq}x{Ck} N={N}", flush=True)
    qh, kh, vh = f64(q), f64(k), f64(v)
    m_ref, l_ref = O.block_masses(qh, kh, N, Cq, Ck, scale)
    n_q, n_k = m_ref.shape[2], m_ref.shape[3]
    R = m_ref.shape[0] * m_ref.shape[1] * n_q

    # calibration: every scheme against Eq. (1) and the row normaliser
    runs = [L.losa_calibrate_mass(q, k, N, Cq, Ck)]
    if dtype == "bf16":
        runs.append(L.losa_calibrate_mass(q, k, N, Cq, Ck, two_sweep=True))
    for mass, lse in runs:
        torch.cuda.synchronize()
        assert np.abs(f64(mass) - m_ref).max() <= MASS_TOL
        lg = f64(lse)
        assert np.abs(lg[:, :, :N] - l_ref[:, :, :N]).max() <= LSE_TOL
        assert np.all(np.isneginf(lg[:, :, N:]))
    mass = runs[0][0]
    mg = f64(mass)

    # selection at tau < 1 against the oracle's rule on its own masses; tau = 1
    for tau in (0.9, 1.0):
        rp, ci = L.losa_select_blocks(mass, N, Cq, Ck, tau)
        rp_g = rp.cpu().numpy().astype(np.int64)
        ci_g = ci[:rp_g[-1]].cpu().numpy().astype(np.int64)
        assert O.validate_csr(rp_g, ci_g, R, n_k, N, Cq, n_q) == []
        _, _, details = O.select_blocks(m_ref, N, Cq, Ck, float(np.float32(tau)))
        cmp = CMP.compare_selection(rp_g, ci_g, details, m_ref.reshape(R, n_k),
                                    float(np.float32(tau)))
        assert cmp["ok"], cmp

        # sparse forward on the GPU's CSR against Eq. (4) on the same CSR
        o, lo = L.losa_sparse_attn_fwd(q, k, v, N, Cq, Ck, rp, ci, want_lse=True)
        torch.cuda.synchronize()
        o_ref, lo_ref = O.sparse_attention(qh, kh, vh, N, Cq, Ck, scale, rp_g, ci_g)
        tmax, tmean = OUT_TOL[dtype]
        err = np.abs(f64(o)[:, :, :N] - o_ref[:, :, :N])
        assert err.max() <= tmax and err.mean() <= tmean, (tau, err.max(), err.mean())
        assert np.all(f64(o)[:, :, N:] == 0)
        assert np.abs(f64(lo)[:, :, :N] - lo_ref[:, :, :N]).max() <= LSE_TOL
        assert np.all(np.isneginf(f64(lo)[:, :, N:]))

        # recall of this support on the GPU's masses (Eq. (2))
        rr, rh = L.losa_block_recall(mass, N, Cq, Ck, rp, ci)
        torch.cuda.synchronize()
        assert np.abs(f64(rr) - O.recall_rows(mg, rp_g, ci_g)).max() <= REC_TOL
        assert np.abs(f64(rh) - O.recall_heads(mg, rp_g, ci_g, N, Cq)).max() <= REC_TOL

    # top-k with k = 1 on the GPU's masses: exact
    rp, ci = L.losa_select_blocks_topk(mass, N, Cq, Ck, 1)
    rp_g = rp.cpu().numpy().astype(np.int64)
    rp_o, ci_o, _ = O.select_blocks_topk(mg, N, Cq, Ck, 1)
    assert np.array_equal(rp_g, rp_o)
    assert np.array_equal(ci[:rp_g[-1]].cpu().numpy().astype(np.int64), ci_o)

    # construction step: dense output and masses
    o, m2, l2 = L.losa_construct(q, k, v, N, Cq, Ck, want_lse=True)
    torch.cuda.synchronize()
    od_ref, ld_ref = O.dense_attention(qh, kh, vh, N, scale)
    tmax, tmean = OUT_TOL[dtype]
    err = np.abs(f64(o)[:, :, :N] - od_ref[:, :, :N])
    assert err.max() <= tmax and err.mean() <= tmean
    assert np.all(f64(o)[:, :, N:] == 0)
    assert np.abs(f64(m2) - m_ref).max() <= MASS_TOL
    assert np.abs(f64(l2)[:, :, :N] - ld_ref[:, :, :N]).max() <= LSE_TOL
