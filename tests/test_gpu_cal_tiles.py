"""Calibration (Sec. 3.1, Eq. (1)) when a row's running max jumps inside a key block.

At d = 128 with 128-row query blocks the calibration streams keys in 64-key
tiles, so a 128-key block spans two tiles and its sums are carried from the
first to the second.  When the lazy running max is raised in the second tile,
the carried sum must move to the new reference with the row sum.  These cases
plant one key per head whose score exceeds every other key of the rows by
more than 26 (log2 units; the max is raised once a tile's probabilities sum
past 2^20), in the second half of a 128-key block, after a first half of ordinary
scores, so that a carried sum left at the old reference would count the first
half 2^26 times or more too heavily.  Controls: the same inputs with 32-key
blocks (two blocks per tile), and d = 64 (one tile per block).  Both schemes
(one sweep with statistics, two sweeps) against the oracle's masses and lse on
every row."""
import numpy as np
import pytest
import torch

from oracle import losa_oracle as O

pytestmark = pytest.mark.gpu

CASES = [  # (d, block_k, N, hot key per head)
    (128, 128, 600, (199, 451)),   # second halves of blocks 1 and 3
    (128, 128, 449, (71, 448)),    # block 0's second half; the ragged last block's only key in its second half
    (128, 32, 600, (199, 451)),
    (64, 128, 600, (199, 451)),
]


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2608_12032_amd import losa
    return losa


def f64(x):
    return x.detach().float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"d{c[0]}-bk{c[1]}-N{c[2]}")
def test_max_raised_in_second_tile_of_a_block(L, case):
    d, Ck, N, hot = case
    Cq, B, H = 128, 1, len(hot)
    print(f"[gpu-cal-tiles] d={d} blocks={Cq}x{Ck} N={N} hot keys {hot}", flush=True)
    rng = np.random.default_rng(9100 + CASES.index(case))
    Np = O.padded_len(N, Cq, Ck)
    q = 0.3 * rng.standard_normal((B, H, Np, d))
    k = 0.3 * rng.standard_normal((B, H, Np, d))
    u = np.full(d, 3.0 / np.sqrt(d))           # |u| = 3, shared by every query
    q += u
    for h, key in enumerate(hot):
        k[0, h, key] = 38.0 * u                # score ~ 38 * 9 * scale above the rest
    q[:, :, N:] = 0
    k[:, :, N:] = 0
    qt = torch.from_numpy(q).to(torch.bfloat16).cuda()
    kt = torch.from_numpy(k).to(torch.bfloat16).cuda()
    scale = 1.0 / np.sqrt(d)
    qh, kh = f64(qt), f64(kt)
    s = qh[:, :, :N] @ np.swapaxes(kh[:, :, :N], 2, 3) * scale
    for h, key in enumerate(hot):              # the planted key leads every row by > 20 in log2 units
        others = np.delete(s[0, h], key, axis=1).max(axis=1)
        assert np.all((s[0, h, :, key] - others) * np.log2(np.e) > 20.0)
    m_ref, l_ref = O.block_masses(qh, kh, N, Cq, Ck, scale)
    for two in (False, True):
        mass, lse = L.losa_calibrate_mass(qt, kt, N, Cq, Ck, two_sweep=two)
        torch.cuda.synchronize()
        e = np.abs(f64(mass) - m_ref).max()
        print(f"[gpu-cal-tiles]   two_sweep={two}: mass max-abs err {e:.3e}", flush=True)
        assert e <= 1e-4, ("mass", two, e)
        lg = f64(lse)
        assert np.abs(lg[:, :, :N] - l_ref[:, :, :N]).max() <= 1e-3, ("lse", two)
        sums = f64(mass).reshape(-1, Np // Ck).sum(axis=1)
        assert np.all(np.abs(sums - 1.0) < 1e-4)
