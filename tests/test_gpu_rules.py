"""GPU parity of the selection-rule ablation and of recall tracking.

* losa_select_blocks_topk, the fixed-ratio top-k rule (Sec. 5, Table 2),
  against the oracle's select_blocks_topk on the same fp32 masses: the sets
  must be identical (same order, same tie rule, no floating point involved).
* losa_block_recall, Eq. (2) of a frozen support on the masses of a later
  step (Sec. 3.1, 3.3), against the oracle's recall_rows / recall_heads on the
  masses the GPU produced (tolerance 1e-6: fp64 sums returned as fp32) and on
  the oracle's own masses of the same inputs (1e-4, the mass tolerance).
"""
import numpy as np
import pytest
import torch

from oracle import losa_oracle as O
from paper_2608_12032_amd import workload as W

pytestmark = pytest.mark.gpu

REC_TOL = 1e-6
MASS_TOL = 1e-4


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2608_12032_amd import losa
    return losa


def say(msg):
    print(f"[gpu-rules] {msg}", flush=True)


def f64(x):
    return x.detach().float().cpu().numpy().astype(np.float64)


def host_csr(rp, ci):
    rp_h = rp.cpu().numpy().astype(np.int64)
    return rp_h, ci[:rp_h[-1]].cpu().numpy().astype(np.int64)


CASES = {
    "wan-small": W.scaled(W.WORKLOADS["wan"], grid=(4, 12, 30), H=3, name="wan-small"),
    "wan-small-c32": W.rectangular(W.scaled(W.WORKLOADS["wan"], grid=(4, 12, 30), H=3,
                                            name="wan-small")),
    "tiny": W.WORKLOADS["tiny"],
}


@pytest.mark.parametrize("key", list(CASES))
def test_topk_on_oracle_masses_is_exact(L, key):
    w = CASES[key]
    q, k, _ = W.make_inputs(w)
    m_ref, _ = O.block_masses(q.float().numpy(), k.float().numpy(), w.N, w.block, w.bk, w.scale)
    m32 = m_ref.astype(np.float32)
    # force exact ties inside some rows: equal masses must go to the smaller id
    m32.reshape(-1, w.n_kblocks)[::3, 1:4] = m32.reshape(-1, w.n_kblocks)[::3, 1:2]
    mdev = torch.from_numpy(m32).cuda()
    n_kv = O.num_valid_key_blocks(w.N, w.bk)
    for kk in sorted({1, 2, max(1, n_kv // 3), n_kv - 1, n_kv, n_kv + 5}):
        rp, ci = L.losa_select_blocks_topk(mdev, w.N, w.block, w.bk, kk)
        torch.cuda.synchronize()
        rp_g, ci_g = host_csr(rp, ci)
        rp_o, ci_o, _ = O.select_blocks_topk(m32.astype(np.float64), w.N, w.block, w.bk, kk)
        say(f"{key}: k={kk} nnz={rp_g[-1]}")
        assert np.array_equal(rp_g, rp_o) and np.array_equal(ci_g, ci_o), kk


@pytest.mark.parametrize("key", ["wan-small", "wan-small-c32"])
def test_rules_at_matched_coverage(L, key):
    # Table 2's comparison on synthetic inputs: the threshold rule and the
    # top-k rule with the same average coverage; recall of both on the same
    # masses, GPU against the oracle.  The threshold rule keeps >= tau per row.
    w = CASES[key]
    q, k, _ = W.make_inputs(w, device="cuda")
    mass, _ = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk, want_lse=False)
    rp_t, ci_t = L.losa_select_blocks(mass, w.N, w.block, w.bk, w.tau)
    torch.cuda.synchronize()
    rows = w.B * w.H * w.n_blocks
    kk = max(1, round(L.nnz(rp_t) / rows))
    rp_k, ci_k = L.losa_select_blocks_topk(mass, w.N, w.block, w.bk, kk)
    torch.cuda.synchronize()
    mg = f64(mass)
    res = {}
    for name, (rp, ci) in {"threshold": (rp_t, ci_t), "topk": (rp_k, ci_k)}.items():
        rr, rh = L.losa_block_recall(mass, w.N, w.block, w.bk, rp, ci)
        torch.cuda.synchronize()
        rp_h, ci_h = host_csr(rp, ci)
        want_r = O.recall_rows(mg, rp_h, ci_h)
        want_h = O.recall_heads(mg, rp_h, ci_h, w.N, w.block)
        assert np.abs(f64(rr) - want_r).max() <= REC_TOL
        assert np.abs(f64(rh) - want_h).max() <= REC_TOL
        res[name] = (rp_h[-1] / (rows * w.n_kblocks), float(want_h.mean()), float(want_h.min()))
    say(f"{key}: k={kk} (coverage, mean head recall, worst head recall) {res}")
    rp_h, ci_h = host_csr(rp_t, ci_t)
    valid = np.array([(r % w.n_blocks) * w.block < w.N for r in range(rows)])
    assert np.all(O.recall_rows(mg, rp_h, ci_h)[valid] >= np.float32(w.tau) - 1e-5)


@pytest.mark.parametrize("key", ["wan-small", "wan-small-c32", "tiny"])
def test_recall_of_frozen_support_across_drift(L, key):
    # construct at step 0, then recall of that support on the masses of the
    # drifted steps (the paper's frozen-pattern measurement), plus a support
    # with repeated and stray ids
    w = CASES[key]
    state = W.make_state(w, device="cuda")
    q, k, _ = W.cast(state, w)
    mass0, _ = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk, want_lse=False)
    rp, ci = L.losa_select_blocks(mass0, w.N, w.block, w.bk, w.tau)
    torch.cuda.synchronize()
    rp_h, ci_h = host_csr(rp, ci)
    rows = rp_h.size - 1
    rng = np.random.default_rng(5)
    dup = [np.concatenate([ci_h[rp_h[r]:rp_h[r + 1]],
                           rng.choice(w.n_kblocks, 3), [-2, w.n_kblocks + 1]]) for r in range(rows)]
    rp_d = np.concatenate([[0], np.cumsum([len(x) for x in dup])])
    ci_d = np.concatenate(dup)
    for step in range(1, 4):
        W.drift_(state, w, step)
        q, k, _ = W.cast(state, w)
        mass, _ = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk, want_lse=False)
        m_ref, _ = O.block_masses(f64(q), f64(k), w.N, w.block, w.bk, w.scale)
        mg = f64(mass)
        for rp_x, ci_x in ((rp_h, ci_h), (rp_d, ci_d)):
            rr, rh = L.losa_block_recall(mass, w.N, w.block, w.bk,
                                         torch.from_numpy(rp_x.astype(np.int32)).cuda(),
                                         torch.from_numpy(ci_x.astype(np.int32)).cuda())
            torch.cuda.synchronize()
            assert np.abs(f64(rr) - O.recall_rows(mg, rp_x, ci_x)).max() <= REC_TOL
            assert np.abs(f64(rh) - O.recall_heads(mg, rp_x, ci_x, w.N, w.block)).max() <= REC_TOL
            assert np.abs(f64(rh) - O.recall_heads(m_ref, rp_x, ci_x, w.N, w.block)).max() \
                <= MASS_TOL
        say(f"{key}: step {step} head recall {f64(rh).round(4).tolist()}")


def test_recall_full_size_wan(L):
    # every row of the Wan-shaped workload at the first reuse step
    w = W.WORKLOADS["wan"]
    state = W.make_state(w, device="cuda")
    q, k, _ = W.cast(state, w)
    mass0, _ = L.losa_calibrate_mass(q, k, w.N, w.block, want_lse=False)
    rp, ci = L.losa_select_blocks(mass0, w.N, w.block, w.block, w.tau)
    W.drift_(state, w, 1)
    q, k, _ = W.cast(state, w)
    del state
    mass1, _ = L.losa_calibrate_mass(q, k, w.N, w.block, want_lse=False)
    rr, rh = L.losa_block_recall(mass1, w.N, w.block, w.block, rp, ci)
    torch.cuda.synchronize()
    rp_h, ci_h = host_csr(rp, ci)
    mg = f64(mass1)
    assert np.abs(f64(rr) - O.recall_rows(mg, rp_h, ci_h)).max() <= REC_TOL
    want_h = O.recall_heads(mg, rp_h, ci_h, w.N, w.block)
    assert np.abs(f64(rh) - want_h).max() <= REC_TOL
    say(f"wan full: step-1 recall mean {want_h.mean():.4f} worst head {want_h.min():.4f}")


# ----------------------------------------------------------------------------
# the construction step: dense attention output + exact block masses
# ----------------------------------------------------------------------------

CONSTRUCT = dict(CASES, **{
    "cog-small": W.scaled(W.WORKLOADS["cog"], grid=(3, 10, 45), H=4, name="cog-small"),
    "tiny-c32": W.rectangular(W.WORKLOADS["tiny"]),
})
OUT_TOL = {"bf16": (2e-2, 2e-3), "f32": (1e-4, 1e-4)}


@pytest.mark.parametrize("key", list(CONSTRUCT))
def test_construct_matches_oracle_and_the_separate_calls(L, key):
    w = CONSTRUCT[key]
    q, k, v = W.make_inputs(w, device="cuda")
    o, mass, lse = L.losa_construct(q, k, v, w.N, w.block, w.bk, want_lse=True)
    o2, mass2 = L.losa_construct(q, k, v, w.N, w.block, w.bk)   # lse kept in the workspace
    m_cal, l_cal = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk)
    rp, ci = L.losa_select_blocks(m_cal, w.N, w.block, w.bk, 1.0)
    o_full = L.losa_sparse_attn_fwd(q, k, v, w.N, w.block, w.bk, rp, ci)
    torch.cuda.synchronize()
    qh, kh, vh = f64(q), f64(k), f64(v)
    o_ref, l_ref = O.dense_attention(qh, kh, vh, w.N, w.scale)
    m_ref, _ = O.block_masses(qh, kh, w.N, w.block, w.bk, w.scale)
    tmax, tmean = OUT_TOL[w.dtype]
    err = np.abs(f64(o)[:, :, :w.N] - o_ref[:, :, :w.N])
    say(f"construct {key}: out max {err.max():.2e} mean {err.mean():.2e}")
    assert err.max() <= tmax and err.mean() <= tmean
    assert np.all(f64(o)[:, :, w.N:] == 0)
    assert np.abs(f64(mass) - m_ref).max() <= MASS_TOL
    lg = f64(lse)
    assert np.abs(lg[:, :, :w.N] - l_ref[:, :, :w.N]).max() <= 1e-3
    assert np.all(np.isneginf(lg[:, :, w.N:]))
    # the same scores as the separate calls: O exactly the forward over the
    # full support; masses and lse to fp32 rounding (the forward's softmax
    # reference moves lazily, the calibration's at every tile)
    assert torch.equal(o, o_full) and torch.equal(o, o2) and torch.equal(mass, mass2)
    assert np.abs(f64(mass) - f64(m_cal)).max() <= 5e-6
    assert np.abs(lg[:, :, :w.N] - f64(l_cal)[:, :, :w.N]).max() <= 1e-5


BF16_CASES = [k for k in CONSTRUCT if CONSTRUCT[k].dtype == "bf16"]


@pytest.mark.parametrize("key", BF16_CASES)
def test_calibration_schemes_and_head_groups(L, key):
    """bf16 calibration: the one-sweep scheme (block statistics + reduction) and
    the two-sweep scheme both match the oracle and each other to fp32 rounding;
    a workspace that holds fewer heads than B*H (the call then works through
    groups of heads, the last one ragged) gives bitwise the same results, for
    the calibration and for the construction step."""
    w = CONSTRUCT[key]
    q, k, v = W.make_inputs(w, device="cuda")
    m1, l1 = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk)
    m2, l2 = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk, two_sweep=True)
    one = L.workspace_bytes(0, 1, 1, 1, w.N, w.d, w.block, w.bk)
    ws1 = torch.empty(one + 100, dtype=torch.uint8, device="cuda")        # one head at a time
    m3, l3 = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk, workspace=ws1)
    one_c = L.workspace_bytes(4, 1, 1, 1, w.N, w.d, w.block, w.bk)
    ws2 = torch.empty(2 * one_c, dtype=torch.uint8, device="cuda")        # two heads at a time
    o4, m4 = L.losa_construct(q, k, v, w.N, w.block, w.bk, workspace=ws2)
    o5, m5 = L.losa_construct(q, k, v, w.N, w.block, w.bk)
    torch.cuda.synchronize()
    assert torch.equal(m3, m1) and torch.equal(l3, l1)
    assert torch.equal(o4, o5) and torch.equal(m4, m5)
    m_ref, l_ref = O.block_masses(f64(q), f64(k), w.N, w.block, w.bk, w.scale)
    e1, e2 = np.abs(f64(m1) - m_ref).max(), np.abs(f64(m2) - m_ref).max()
    say(f"calibration {key}: one sweep {e1:.2e}, two sweeps {e2:.2e}")
    assert e1 <= MASS_TOL and e2 <= MASS_TOL
    assert np.abs(f64(m1) - f64(m2)).max() <= 5e-6
    n = w.N
    assert np.abs(f64(l1)[:, :, :n] - l_ref[:, :, :n]).max() <= 1e-3
    assert np.abs(f64(l1)[:, :, :n] - f64(l2)[:, :, :n]).max() <= 1e-5
    assert np.all(np.isneginf(f64(l1)[:, :, n:])) and np.all(np.isneginf(f64(l2)[:, :, n:]))


@pytest.mark.parametrize("key", ["wan", "cog", "hunyuan", "wan-c32"])
def test_construct_full_size_sampled(L, key):
    w = W.rectangular(W.WORKLOADS[key[:-4]]) if key.endswith("-c32") else W.WORKLOADS[key]
    q, k, v = W.make_inputs(w, device="cuda")
    o, mass = L.losa_construct(q, k, v, w.N, w.block, w.bk)
    torch.cuda.synchronize()
    n_q = w.n_blocks
    heads, blocks = (0, w.H - 1), (0, n_q // 2, n_q - 1)
    rows = [h * n_q + i for h in heads for i in blocks]
    qh, kh, vh = f64(q), f64(k), f64(v)
    m_ref, _ = O.block_masses(qh, kh, w.N, w.block, w.bk, w.scale, rows_subset=rows)
    n_kv = O.num_valid_key_blocks(w.N, w.bk)  # dense attention: every valid key block
    rp_full = np.arange(0, (w.H * n_q + 1) * n_kv, n_kv)
    ci_full = np.tile(np.arange(n_kv), w.H * n_q)
    o_ref, _ = O.sparse_attention(qh, kh, vh, w.N, w.block, w.bk, w.scale, rp_full, ci_full,
                                  rows_subset=rows)
    mg, og = f64(mass), f64(o)
    for r in rows:
        h, i = divmod(r, n_q)
        assert np.abs(mg[0, h, i] - m_ref[0, h, i]).max() <= MASS_TOL
        lo, hi = i * w.block, min((i + 1) * w.block, w.N)
        err = np.abs(og[0, h, lo:hi] - o_ref[0, h, lo:hi])
        assert err.max() <= 2e-2 and err.mean() <= 2e-3


def test_corrupt_masses_select_like_zeros(L):
    """Negative and NaN masses count as 0 in both selection rules (reading of
    the selection for corrupt inputs): the GPU's sets equal the oracle's."""
    w = CASES["wan-small"]
    q, k, _ = W.make_inputs(w, device="cuda")
    mass, _ = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk, want_lse=False)
    torch.cuda.synchronize()
    m = f64(mass)
    rng = np.random.default_rng(12)
    bad = rng.random(m.shape) < 0.2
    m[bad] = np.where(rng.random(bad.sum()) < 0.5, np.nan, -rng.random(bad.sum()))
    mt = torch.tensor(m, dtype=torch.float32, device="cuda")
    m32 = m.astype(np.float32).astype(np.float64)
    for tau in (0.5, 0.9, 0.99):
        rp, ci = L.losa_select_blocks(mt, w.N, w.block, w.bk, tau)
        rp_o, ci_o, _ = O.select_blocks(m32, w.N, w.block, w.bk, float(np.float32(tau)))
        rp_g, ci_g = host_csr(rp, ci)
        assert np.array_equal(rp_g, rp_o) and np.array_equal(ci_g, ci_o), tau
    for kk in (1, 7, 30):
        rp, ci = L.losa_select_blocks_topk(mt, w.N, w.block, w.bk, kk)
        rp_o, ci_o, _ = O.select_blocks_topk(m32, w.N, w.block, w.bk, kk)
        rp_g, ci_g = host_csr(rp, ci)
        assert np.array_equal(rp_g, rp_o) and np.array_equal(ci_g, ci_o), kk
