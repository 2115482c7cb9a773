"""Softmaxes at their extremes, every entry point against the oracle on every row.

* Uniform: Q = 0, so every valid key gets the same probability; block masses
  are key counts over N, every mass row is a tie (kept blocks: the smallest
  indices), and the output is the mean of V over the kept keys.
* Peaked: Q and K scaled so that score gaps reach hundreds (in log2 units);
  each row's softmax is one-hot up to fp32 underflow, which drives the lazy
  running max through its overflow branch (a first sub-tile sum of +inf) on
  almost every row, and the output is one V row.
* Large V: V scaled by 1,000; the output bound scales with it (half an ulp of
  the bf16 output plus P rounded to bf16 for P V, as derived for the random
  configurations).

Bounds derived from the arithmetic.  Scores are formed in fp32, so their
absolute rounding error grows with their size; with max|s| in the hundreds it
reaches 1e-5..1e-4, a relative error of the probabilities of that size.  The
output bound adds 2 max|v| max|s| 2^-20 (16 ulps of the largest score) to the
workloads' bounds; for scores of size 10 that term is below 1e-4.  The same
score rounding moves the block masses: a probability carries the relative
error of its score and of its row's lse, so a mass (at most 1) moves by at
most 2 * 16 ulps of the largest score, max|s| 2^-18.  Two blocks whose exact
masses are closer than twice that at the cut can trade places.  The selection
is therefore checked in two parts: exactly against Eq. (3) applied to the
masses the GPU computed, and against the oracle's selection on exact masses
under the workloads' rule (cumulative mass within 1e-5 of tau, near-ties
within 1e-6), where every row that rule does not accept must be a named
near-cut swap: the same number of blocks, one block traded for one other,
their exact masses within the bound above (fixed from the inputs before the
GPU runs), the kept mass still at least tau - 1e-5.
"""
import numpy as np
import pytest
import torch

from oracle import compare as CMP
from oracle import losa_oracle as O

pytestmark = pytest.mark.gpu

CASES = [  # (kind, dtype, d, Cq, Ck, N)
    ("uniform", "bf16", 128, 128, 128, 700), ("uniform", "bf16", 64, 128, 32, 517),
    ("uniform", "f32", 64, 64, 64, 300),
    ("peaked", "bf16", 128, 128, 128, 640), ("peaked", "bf16", 64, 128, 32, 389),
    ("peaked", "f32", 128, 64, 32, 250),
    ("large_v", "bf16", 128, 128, 128, 600), ("large_v", "f32", 64, 128, 128, 333),
]


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2608_12032_amd import losa
    return losa


def f64(x):
    return x.detach().float().cpu().numpy().astype(np.float64)


def selection_with_named_swaps(rp_g, ci_g, details, flat, tau, swap_bound):
    """The workloads' selection rule row by row; a row it rejects must be a
    near-cut swap within swap_bound.  Returns the swapped rows."""
    swaps = []
    for r, det in enumerate(details):
        got = ci_g[rp_g[r]:rp_g[r + 1]]
        cmp = CMP.compare_selection(np.array([0, got.size]), got, [det], flat[r:r + 1], tau)
        if cmp["ok"]:
            continue
        want = det.omega
        extra, missing = np.setdiff1d(got, want), np.setdiff1d(want, got)
        assert got.size == want.size and extra.size == 1 and missing.size == 1, (r, cmp)
        gap = abs(flat[r, extra[0]] - flat[r, missing[0]])
        assert gap <= swap_bound, ("swap beyond the rounding bound", r, gap, swap_bound)
        assert flat[r, got].sum() >= tau - 1e-5, (r, "kept mass")
        swaps.append((r, int(extra[0]), int(missing[0]), float(gap)))
    return swaps


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_extreme_softmax(L, case):
    kind, dtype, d, Cq, Ck, N = case
    B, H = 1, 2
    print(f"[gpu-extremes] {kind} {dtype} d={d} blocks={Cq}x{Ck} N={N}", flush=True)
    rng = np.random.default_rng(9000 + CASES.index(case))
    Np = O.padded_len(N, Cq, Ck)
    t = torch.from_numpy(rng.standard_normal((3, B, H, Np, d))).float()
    if kind == "uniform":
        t[0] = 0.0
    elif kind == "peaked":
        t[:2] *= 12.0
    else:
        t[2] *= 1000.0
    t[:, :, :, N:] = 0
    t = t.to(torch.bfloat16 if dtype == "bf16" else torch.float32).cuda()
    q, k, v = t[0].contiguous(), t[1].contiguous(), t[2].contiguous()
    scale = 1.0 / np.sqrt(d)
    qh, kh, vh = f64(q), f64(k), f64(v)
    n_q, n_k = Np // Cq, Np // Ck
    n_kv = O.num_valid_key_blocks(N, Ck)
    vmax = float(np.abs(vh).max())
    smax = float(np.abs(qh[:, :, :N] @ np.swapaxes(kh[:, :, :N], 2, 3)).max() * scale)
    score_term = 2.0 * vmax * smax * 2.0 ** -20
    mass_bound = max(1e-6, smax * 2.0 ** -18)  # what fp32 score rounding moves a mass by

    m_ref, l_ref = O.block_masses(qh, kh, N, Cq, Ck, scale)
    if kind == "uniform":  # the closed form: valid keys of block j over N
        counts = np.array([min(Ck, max(0, N - j * Ck)) for j in range(n_k)], np.float64)
        valid_q = np.array([i * Cq < N for i in range(n_q)])
        assert np.allclose(m_ref[:, :, valid_q], counts / N, atol=1e-12)
    for two in (False, True):
        mass, lse = L.losa_calibrate_mass(q, k, N, Cq, Ck, two_sweep=two)
        torch.cuda.synchronize()
        e = np.abs(f64(mass) - m_ref).max()
        assert e <= 1e-4, ("mass", two, e)
        lg = f64(lse)
        assert np.abs(lg[:, :, :N] - l_ref[:, :, :N]).max() <= 1e-3, ("lse", two)
        assert np.all(np.isneginf(lg[:, :, N:]))

    for tau in (0.5, 0.99):
        rp, ci = L.losa_select_blocks(mass, N, Cq, Ck, tau)
        torch.cuda.synchronize()
        rp_g = rp.cpu().numpy().astype(np.int64)
        ci_g = ci[:int(rp_g[-1])].cpu().numpy().astype(np.int64)
        t32 = float(np.float32(tau))
        valid = [(r % n_q) * Cq < N for r in range(B * H * n_q)]
        gflat = f64(mass).reshape(-1, n_k)
        for r in range(gflat.shape[0]):  # Eq. (3) on the masses the GPU selected from
            want = O.select_row(gflat[r], t32, n_kv, valid[r]).omega
            assert np.array_equal(ci_g[rp_g[r]:rp_g[r + 1]], want), (tau, r)
        flat = m_ref.reshape(-1, n_k)
        details = [O.select_row(flat[r], t32, n_kv, valid[r]) for r in range(flat.shape[0])]
        swaps = selection_with_named_swaps(rp_g, ci_g, details, flat, t32, 2 * mass_bound)
        print(f"[gpu-extremes]   tau={tau}: {len(swaps)} near-cut swaps {swaps[:4]}", flush=True)

        o, lo = L.losa_sparse_attn_fwd(q, k, v, N, Cq, Ck, rp, ci, want_lse=True)
        torch.cuda.synchronize()
        o_ref, lo_ref = O.sparse_attention(qh, kh, vh, N, Cq, Ck, scale, rp_g, ci_g)
        og = f64(o)
        err = np.abs(og[:, :, :N] - o_ref[:, :, :N])
        if dtype == "bf16":
            bound = (1e-2 * max(1.0, vmax / 4) + 2.0 ** -8 * (np.abs(o_ref[:, :, :N]) + vmax)
                     + score_term)
            assert np.all(err <= bound), (tau, float(err.max()))
        else:
            assert err.max() <= 1e-4 * max(1.0, vmax / 4) + score_term, (tau, float(err.max()))
        assert np.abs(f64(lo)[:, :, :N] - lo_ref[:, :, :N]).max() <= 1e-3
        assert np.all(og[:, :, N:] == 0)

    oc, mc = L.losa_construct(q, k, v, N, Cq, Ck)
    torch.cuda.synchronize()
    assert np.abs(f64(mc) - m_ref).max() <= 1e-4
    od_ref, _ = O.dense_attention(qh, kh, vh, N, scale)
    errc = np.abs(f64(oc)[:, :, :N] - od_ref[:, :, :N])
    if dtype == "bf16":
        assert np.all(errc <= 1e-2 * max(1.0, vmax / 4)
                      + 2.0 ** -8 * (np.abs(od_ref[:, :, :N]) + vmax) + score_term)
    else:
        assert errc.max() <= 1e-4 * max(1.0, vmax / 4) + score_term


@pytest.mark.parametrize("dtype,scale", [("bf16", 0.02), ("bf16", 1.0), ("f32", 0.02), ("f32", 0.5)])
def test_explicit_scale(L, dtype, scale):
    """A score scale other than 1/sqrt(d), passed through every entry point."""
    B, H, d, Cq, Ck, N = 1, 2, 64, 128, 32, 450
    print(f"[gpu-extremes] scale {scale} {dtype}", flush=True)
    rng = np.random.default_rng(9100 + int(scale * 100))
    Np = O.padded_len(N, Cq, Ck)
    t = torch.from_numpy(rng.standard_normal((3, B, H, Np, d))).float()
    t[:, :, :, N:] = 0
    t = t.to(torch.bfloat16 if dtype == "bf16" else torch.float32).cuda()
    q, k, v = t[0].contiguous(), t[1].contiguous(), t[2].contiguous()
    qh, kh, vh = f64(q), f64(k), f64(v)
    n_k = Np // Ck
    n_q = Np // Cq
    n_kv = O.num_valid_key_blocks(N, Ck)
    m_ref, l_ref = O.block_masses(qh, kh, N, Cq, Ck, scale)
    mass, lse = L.losa_calibrate_mass(q, k, N, Cq, Ck, scale=scale)
    torch.cuda.synchronize()
    assert np.abs(f64(mass) - m_ref).max() <= 1e-4
    assert np.abs(f64(lse)[:, :, :N] - l_ref[:, :, :N]).max() <= 1e-3
    rp, ci = L.losa_select_blocks(mass, N, Cq, Ck, 0.9)
    torch.cuda.synchronize()
    rp_g = rp.cpu().numpy().astype(np.int64)
    ci_g = ci[:int(rp_g[-1])].cpu().numpy().astype(np.int64)
    gflat = f64(mass).reshape(-1, n_k)
    t32 = float(np.float32(0.9))
    for r in range(gflat.shape[0]):
        want = O.select_row(gflat[r], t32, n_kv, (r % n_q) * Cq < N).omega
        assert np.array_equal(ci_g[rp_g[r]:rp_g[r + 1]], want)
    o, lo = L.losa_sparse_attn_fwd(q, k, v, N, Cq, Ck, rp, ci, scale=scale, want_lse=True)
    oc, mc = L.losa_construct(q, k, v, N, Cq, Ck, scale=scale)
    torch.cuda.synchronize()
    o_ref, lo_ref = O.sparse_attention(qh, kh, vh, N, Cq, Ck, scale, rp_g, ci_g)
    od_ref, _ = O.dense_attention(qh, kh, vh, N, scale)
    tol = (2e-2, 2e-3) if dtype == "bf16" else (1e-4, 1e-4)
    for got, ref in ((f64(o), o_ref), (f64(oc), od_ref)):
        err = np.abs(got[:, :, :N] - ref[:, :, :N])
        assert err.max() <= tol[0] and err.mean() <= tol[1]
    assert np.abs(f64(lo)[:, :, :N] - lo_ref[:, :, :N]).max() <= 1e-3
    assert np.abs(f64(mc) - m_ref).max() <= 1e-4
