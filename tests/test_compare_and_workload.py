"""Host-side tests: the selection comparison rule and the seeded input generator."""
import numpy as np
import pytest
import torch

from oracle import compare as CMP
from oracle import losa_oracle as O
from paper_2608_12032_amd import workload as W


def _check(got, m, tau):
    m = np.asarray(m, dtype=np.float64)
    sel = O.select_row(m, tau, m.size)
    rp = np.array([0, len(got)])
    return CMP.compare_selection(rp, np.array(sorted(got)), [sel], m.reshape(1, -1), tau)


def test_exact_selection_passes():
    m = [0.5, 0.3, 0.15, 0.05]
    assert _check([0, 1, 2], m, 0.9)["ok"]


def test_one_block_late_near_tau_is_exempt():
    # oracle: cum after 3 blocks = 0.9 + 3e-6 >= tau = 0.9 -> s = 3; a result
    # whose fp32 sum fell just short would also keep block 3
    m = np.array([0.5, 0.3, 0.1 + 3e-6, 0.1 - 3e-6])
    assert O.select_row(m, 0.9, 4).s == 3
    assert _check([0, 1, 2, 3], m, 0.9)["ok"]


def test_one_block_early_near_tau_is_exempt_only_if_mass_reaches():
    m = np.array([0.5, 0.3, 0.1 + 3e-6, 0.1 - 3e-6])
    # dropping block 2 leaves 0.8 < tau - eps: rejected
    assert not _check([0, 1], m, 0.9)["ok"]
    m2 = np.array([0.6, 0.3 - 4e-6, 4e-6 + 1e-7, 0.1 - 1e-7])
    sel = O.select_row(m2, 0.9, 4)
    assert sel.s == 3
    # keeping only {0, 1} reaches 0.9 - 4e-6 >= tau - 1e-5: exempt
    assert _check([0, 1], m2, 0.9)["ok"]


def test_wrong_block_far_from_tau_fails():
    m = [0.5, 0.3, 0.15, 0.05]
    r = _check([0, 1, 3], m, 0.9)
    assert not r["ok"]


def test_tau_one_allows_no_exemption():
    m = np.array([0.5, 0.3, 0.2 - 1e-9, 1e-9])
    assert not _check([0, 1, 2], m, 1.0)["ok"]
    assert _check([0, 1, 2, 3], m, 1.0)["ok"]


def test_near_tie_at_cut_is_exempt():
    m = np.array([0.5, 0.42, 0.04 + 2e-7, 0.04 - 2e-7])
    sel = O.select_row(m, 0.95, 4)
    assert sel.omega.tolist() == [0, 1, 2]
    assert _check([0, 1, 3], m, 0.95)["ok"]


def test_output_errors_over_valid_rows_only():
    a = np.zeros((1, 1, 8, 2))
    b = np.zeros((1, 1, 8, 2))
    b[0, 0, 7] = 5.0          # padding row: ignored
    b[0, 0, 0, 0] = 0.01
    mx, mean = CMP.output_errors(a, b, 7)
    assert mx == pytest.approx(0.01) and mean == pytest.approx(0.01 / 14)


# ----------------------------------------------------------------------------
# generator
# ----------------------------------------------------------------------------

def test_workload_shapes():
    want = {"tiny": (1024, 1024, 16), "wan": (32760, 32768, 256),
            "cog": (17550, 17664, 138), "hunyuan": (118800, 118912, 929)}
    for key, (N, Np, nb) in want.items():
        w = W.WORKLOADS[key]
        assert (w.N, w.N_pad, w.n_blocks) == (N, Np, nb)
    pts = W.sweep_points()
    assert len(pts) == 12 and {p.tau for p in pts} == {0.95, 0.99, 0.999, 1.0}
    assert all((p.N, p.N_pad) == (32760, 32768) for p in pts)


def test_generator_deterministic_and_padded():
    w = W.scaled(W.WORKLOADS["cog"], grid=(2, 6, 9), H=3)    # N = 108 -> N_pad = 128
    a = W.make_inputs(w)
    b = W.make_inputs(w)
    for x, y in zip(a, b):
        assert x.dtype == torch.bfloat16 and x.shape == (1, 3, 128, 64)
        assert torch.equal(x, y)
        assert torch.all(x[:, :, w.N:] == 0)
    al = W.head_alphas(w)
    assert torch.all((al >= 0.8) & (al <= 2.0))
    st = W.make_state(w)
    before = [x.clone() for x in st]
    W.drift_(st, w, 1)
    for x, y in zip(st, before):
        assert torch.all(x[:, :, w.N:] == 0)
        d = (x - y)[:, :, :w.N]
        assert 0.5 * w.sigma < d.std().item() < 2 * w.sigma


def test_tiny_inputs_are_fp32():
    q, k, v = W.make_inputs(W.WORKLOADS["tiny"])
    assert q.dtype == torch.float32 and q.shape == (1, 2, 1024, 64)
