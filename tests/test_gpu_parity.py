"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Tolerances (from the target): block masses max-abs <= 1e-4; attention outputs
max-abs <= 2e-2 and mean-abs <= 2e-3 over valid rows (bf16); selected sets
exact except blocks the oracle's cumulative mass puts within 1e-5 of tau
(oracle.compare with tie = 0: only exact ties at the cut, whose order the
smaller-index rule fixes on both sides, count as ties).  Internal, tighter
checks: lse within 1e-3; fp32 outputs within 1e-4.

The oracle always receives the exact values the GPU received (bf16 and fp32
upcast exactly to fp64), copied back from the device.  Small cases are checked
element by element on every row; full-size workloads on sampled rows (first,
middle, ragged last query block of several heads) plus properties that hold at
any size.  Full-size rows: the fixed sample plus seeded random rows drawn
over every head.
"""
import math

import numpy as np
import pytest
import torch

from oracle import compare as CMP
from oracle import losa_oracle as O
from paper_2608_12032_amd import workload as W

pytestmark = pytest.mark.gpu

MASS_TOL = 1e-4
LSE_TOL = 1e-3
OUT_MAX, OUT_MEAN = 2e-2, 2e-3
F32_OUT_MAX = 1e-4


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2608_12032_amd import losa
    return losa


def say(msg):
    print(f"[gpu-parity] {msg}", flush=True)


def f64(x):
    return x.detach().float().cpu().numpy().astype(np.float64)


def tau32(t):
    return float(np.float32(t))


def sub_csr(rp, ci, rows):
    rp = np.asarray(rp, dtype=np.int64)
    ci = np.asarray(ci, dtype=np.int64)
    out_rp = [0]
    out_ci = []
    for r in rows:
        seg = ci[rp[r]:rp[r + 1]]
        out_ci.append(seg)
        out_rp.append(out_rp[-1] + seg.size)
    return np.array(out_rp), (np.concatenate(out_ci) if out_ci else np.zeros(0, np.int64))


def out_tol(w):
    return (F32_OUT_MAX, F32_OUT_MAX) if w.dtype == "f32" else (OUT_MAX, OUT_MEAN)


def sample_rows(w, extra=()):
    n_q = w.n_blocks
    heads = sorted({0, w.H - 1, w.H // 2})
    blocks = sorted({0, 1, n_q // 3, n_q // 2, n_q - 2, n_q - 1, *extra})
    return [(b * w.H + h) * n_q + i for b in range(w.B) for h in heads for i in blocks
            if 0 <= i < n_q]


def random_rows(w, per_head=0, total=0, seed=0):
    """Seeded random CSR rows on top of the fixed sample: per_head query blocks
    of every (b, h), or `total` rows drawn over the whole grid.  The dispatch
    order puts rows on every XCD and at every position of a chunk, so rows
    drawn anywhere reach parts of the launch the fixed sample does not."""
    rng = np.random.default_rng(60_000 + seed)
    n_q = w.n_blocks
    rows = set()
    if per_head:
        for bh in range(w.B * w.H):
            rows.update(bh * n_q + int(i) for i in rng.choice(n_q, size=min(per_head, n_q),
                                                              replace=False))
    if total:
        rows.update(int(r) for r in rng.choice(w.B * w.H * n_q, size=total, replace=False))
    return sorted(rows)


def run_case(L, w, tau, reuse=0, rows=None, label="", check_steps=None):
    """calibrate -> select -> sparse fwd (+ reuse steps), all checked against the oracle.

    The inputs drift through steps 1..reuse; the forward is checked at the steps
    in check_steps (default: every step)."""
    N, Cq, Ck, scale = w.N, w.block, w.bk, w.scale
    n_q, n_k = w.n_blocks, w.n_kblocks
    n_kv = O.num_valid_key_blocks(N, Ck)
    t32 = tau32(tau)
    say(f"{label}: generate {w.name} B={w.B} H={w.H} N={N} d={w.d} blocks={Cq}x{Ck} {w.dtype} "
        f"tau={tau}")
    state = W.make_state(w, device="cuda")
    q, k, v = W.cast(state, w)

    say(f"{label}: calibrate")
    mass, lse = L.losa_calibrate_mass(q, k, N, Cq, Ck)
    say(f"{label}: select")
    rp, ci = L.losa_select_blocks(mass, N, Cq, Ck, tau)
    say(f"{label}: sparse fwd step 0")
    o, lse_o = L.losa_sparse_attn_fwd(q, k, v, N, Cq, Ck, rp, ci, want_lse=True)
    torch.cuda.synchronize()
    say(f"{label}: oracle")

    qh, kh, vh = f64(q), f64(k), f64(v)
    mass_g, lse_g = f64(mass), f64(lse)
    rp_g = rp.cpu().numpy().astype(np.int64)
    nnz = int(rp_g[-1])
    ci_g = ci[:nnz].cpu().numpy().astype(np.int64)
    R = w.B * w.H * n_q
    assert O.validate_csr(rp_g, ci_g, R, n_k, N, Cq, n_q) == []

    # properties at any size: every row of masses sums to one; recall >= tau
    sums = mass_g.reshape(R, n_k).sum(axis=1)
    assert np.all(np.abs(sums - 1.0) < 1e-4), f"mass rows sum to {sums.min()}..{sums.max()}"
    if t32 < 1:
        assert O.recall(mass_g, rp_g, ci_g, N, Cq) >= t32 - 1e-5
    else:
        assert nnz == R * n_kv

    todo = list(range(R)) if rows is None else rows
    m_ref, l_ref = O.block_masses(qh, kh, N, Cq, Ck, scale, rows_subset=todo)
    flat_m_ref = m_ref.reshape(R, n_k)
    flat_m_g = mass_g.reshape(R, n_k)
    merr = np.abs(flat_m_g[todo] - flat_m_ref[todo]).max()
    say(f"{label}: mass max-abs err {merr:.3e}")
    assert merr <= MASS_TOL
    qrows = np.concatenate([np.arange(i * Cq, min((i + 1) * Cq, N)) + (r // n_q) * w.N_pad
                            for r in todo for i in [r % n_q]])
    lerr = np.abs(lse_g.reshape(-1)[qrows] - l_ref.reshape(-1)[qrows]).max()
    assert lerr <= LSE_TOL, f"lse err {lerr}"

    # selection: the GPU's rows against the oracle's selection on oracle masses
    details = [O.select_row(flat_m_ref[r], t32, n_kv, (r % n_q) * Cq < N) for r in todo]
    srp, sci = sub_csr(rp_g, ci_g, todo)
    cmp = CMP.compare_selection(srp, sci, details, flat_m_ref[todo], t32, tie=0.0)
    say(f"{label}: selection {cmp}")
    assert cmp["ok"], cmp

    # sparse forward with the GPU's CSR (isolates Eq. (4) from the selection)
    tmax, tmean = out_tol(w)
    check = set(range(reuse + 1)) if check_steps is None else set(check_steps)
    for step in range(reuse + 1):
        if step > 0:
            W.drift_(state, w, step)
            if step not in check:
                continue
            q, k, v = W.cast(state, w)
            say(f"{label}: sparse fwd reuse step {step}")
            o, lse_o = L.losa_sparse_attn_fwd(q, k, v, N, Cq, Ck, rp, ci, want_lse=True)
            torch.cuda.synchronize()
            qh, kh, vh = f64(q), f64(k), f64(v)
        o_ref, lo_ref = O.sparse_attention(qh, kh, vh, N, Cq, Ck, scale, rp_g, ci_g,
                                           rows_subset=todo)
        og = f64(o)
        err = np.abs(og.reshape(-1, w.d)[qrows] - o_ref.reshape(-1, w.d)[qrows])
        say(f"{label}: step {step} out max {err.max():.3e} mean {err.mean():.3e}")
        assert err.max() <= tmax and err.mean() <= tmean
        lo_err = np.abs(f64(lse_o).reshape(-1)[qrows] - lo_ref.reshape(-1)[qrows]).max()
        assert lo_err <= LSE_TOL
        # padding rows are zero, lse -inf
        og4 = og.reshape(w.B, w.H, w.N_pad, w.d)
        assert np.all(og4[:, :, N:] == 0)
        assert np.all(np.isneginf(f64(lse_o)[:, :, N:]))
    return dict(nnz=nnz, coverage=nnz / (R * n_k), exempt=cmp["exempt"])


# ----------------------------------------------------------------------------
# small cases: every row, several tiles, ragged tails
# ----------------------------------------------------------------------------

SMALL = {
    "tiny-f32": W.WORKLOADS["tiny"],
    "wan-bf16-d128-ragged": W.scaled(W.WORKLOADS["wan"], grid=(4, 12, 30), H=3, name="wan-small"),
    "cog-bf16-d64-ragged": W.scaled(W.WORKLOADS["cog"], grid=(3, 10, 45), H=4, name="cog-small"),
    "bf16-d128-blk64": W.scaled(W.Workload("b64", 1, 2, 128, "bf16", (3, 9, 25), 64, 0.99, 1.5,
                                           0.5, 0.02, 1, 77), name="bf16-d128-b64"),
    "bf16-d64-blk64": W.Workload("bf16-d64-b64", 2, 2, 64, "bf16", (2, 11, 23), 64, 0.95, 2.0,
                                 0.5, 0.02, 1, 78),
    "f32-d128-blk128": W.Workload("f32-d128-b128", 1, 2, 128, "f32", (2, 10, 25), 128, 0.99, 1.5,
                                  0.5, 0.02, 1, 79),
    "f32-d64-blk128": W.Workload("f32-d64-b128", 1, 3, 64, "f32", (2, 10, 19), 128, 0.9, 1.5,
                                 0.5, 0.02, 1, 80),
    # the paper's rectangular blocks (Sec. 5.1): 128-row query blocks, 32-key key blocks
    "wan-bf16-d128-r128c32": W.rectangular(W.scaled(W.WORKLOADS["wan"], grid=(4, 12, 30), H=3,
                                                    name="wan-small")),
    "cog-bf16-d64-r128c32": W.rectangular(W.scaled(W.WORKLOADS["cog"], grid=(3, 10, 45), H=4,
                                                   name="cog-small")),
    "bf16-d128-r64c32": W.rectangular(W.Workload("b64", 1, 2, 128, "bf16", (3, 9, 25), 64, 0.99,
                                                 1.5, 0.5, 0.02, 1, 81)),
    "tiny-f32-r64c32": W.rectangular(W.WORKLOADS["tiny"]),
    "f32-d128-r128c32": W.rectangular(W.Workload("f32-d128-b128", 1, 2, 128, "f32", (2, 10, 25),
                                                 128, 0.99, 1.5, 0.5, 0.02, 1, 82)),
}


@pytest.mark.parametrize("key", list(SMALL))
def test_small_pipeline_all_rows(L, key):
    w = SMALL[key]
    info = run_case(L, w, w.tau, reuse=min(w.reuse, 3), label=key)
    assert 0 < info["coverage"] <= 1


@pytest.mark.parametrize("key", ["wan-bf16-d128-ragged", "cog-bf16-d64-ragged", "tiny-f32",
                                 "wan-bf16-d128-r128c32", "tiny-f32-r64c32"])
def test_small_tau_one_is_dense(L, key):
    w = SMALL[key]
    q, k, v = W.make_inputs(w, device="cuda")
    mass, _ = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk, want_lse=False)
    rp, ci = L.losa_select_blocks(mass, w.N, w.block, w.bk, 1.0)
    o = L.losa_sparse_attn_fwd(q, k, v, w.N, w.block, w.bk, rp, ci)
    torch.cuda.synchronize()
    assert L.nnz(rp) == w.B * w.H * w.n_blocks * O.num_valid_key_blocks(w.N, w.bk)
    o_ref, _ = O.dense_attention(f64(q), f64(k), f64(v), w.N, w.scale)
    mx, mean = CMP.output_errors(f64(o), o_ref, w.N)
    tmax, tmean = out_tol(w)
    assert mx <= tmax and mean <= tmean, (mx, mean)


@pytest.mark.parametrize("key", ["wan-bf16-d128-ragged", "cog-bf16-d64-ragged", "tiny-f32",
                                 "wan-bf16-d128-r128c32"])
def test_select_on_oracle_masses(L, key):
    # the selection kernel alone, fed the oracle's masses (rounded to fp32 for
    # both sides), at several thresholds
    w = SMALL[key]
    q, k, _ = W.make_inputs(w)
    m_ref, _ = O.block_masses(q.float().numpy(), k.float().numpy(), w.N, w.block, w.bk, w.scale)
    m32 = m_ref.astype(np.float32)
    mdev = torch.from_numpy(m32).cuda()
    n_k = w.n_kblocks
    n_kv = O.num_valid_key_blocks(w.N, w.bk)
    for tau in (0.5, 0.9, 0.95, 0.99, 0.999, 1.0):
        rp, ci = L.losa_select_blocks(mdev, w.N, w.block, w.bk, tau)
        torch.cuda.synchronize()
        rp_g = rp.cpu().numpy().astype(np.int64)
        ci_g = ci[:rp_g[-1]].cpu().numpy().astype(np.int64)
        m64 = m32.astype(np.float64)
        details = [O.select_row(m64.reshape(-1, n_k)[r], tau32(tau), n_kv) for r in range(rp_g.size - 1)]
        cmp = CMP.compare_selection(rp_g, ci_g, details, m64, tau32(tau), tie=0.0)
        assert cmp["ok"], (tau, cmp)


def test_select_ties_go_to_smaller_index(L):
    # equal masses everywhere: the kept prefix is the smallest indices
    B, H, n, N = 1, 2, 8, 8 * 64
    m = torch.full((B, H, n, n), 1.0 / n, dtype=torch.float32, device="cuda")
    rp, ci = L.losa_select_blocks(m, N, 64, 64, 0.5)
    torch.cuda.synchronize()
    rp_h = rp.cpu().numpy()
    assert np.all(np.diff(rp_h) == 4)
    assert ci[:rp_h[-1]].cpu().numpy().reshape(-1, 4).tolist() == [[0, 1, 2, 3]] * (B * H * n)


@pytest.mark.parametrize("key", ["wan-bf16-d128-ragged", "wan-bf16-d128-r128c32"])
def test_fwd_edge_case_csr(L, key):
    # empty row, single-block row, descending order, out-of-range ids, full row
    # (with 32-key blocks the row lengths 1, 3, 2 and n_k also cover every
    # remainder of the stream padding to whole loop passes)
    w = SMALL[key]
    q, k, v = W.make_inputs(w, device="cuda")
    n_q, n_k = w.n_blocks, w.n_kblocks
    R = w.B * w.H * n_q
    rows = []
    for r in range(R):
        kind = r % 5
        if kind == 0:
            rows.append([])
        elif kind == 1:
            rows.append([r % n_k])
        elif kind == 2:
            rows.append(sorted({(r + 3) % n_k, (r + 7) % n_k, n_k - 1}, reverse=True))
        elif kind == 3:
            rows.append([-1, 0, n_k + 5, 2])
        else:
            rows.append(list(range(n_k)))
    rp = np.zeros(R + 1, np.int64)
    for r, seg in enumerate(rows):
        rp[r + 1] = rp[r] + len(seg)
    ci = np.array([j for seg in rows for j in seg], np.int64)
    rp_d = torch.from_numpy(rp.astype(np.int32)).cuda()
    ci_d = torch.from_numpy(ci.astype(np.int32)).cuda()
    o, lse = L.losa_sparse_attn_fwd(q, k, v, w.N, w.block, w.bk, rp_d, ci_d, want_lse=True)
    torch.cuda.synchronize()
    # ids outside [0, n_k) are ignored by contract: drop them for the oracle
    keep = (ci >= 0) & (ci < n_k)
    rp_clean = np.concatenate([[0], np.cumsum([np.sum(keep[rp[r]:rp[r + 1]]) for r in range(R)])])
    o_ref, l_ref = O.sparse_attention(f64(q), f64(k), f64(v), w.N, w.block, w.bk, w.scale,
                                      rp_clean, ci[keep])
    mx, mean = CMP.output_errors(f64(o), o_ref, w.N)
    assert mx <= OUT_MAX and mean <= OUT_MEAN, (mx, mean)
    lg = f64(lse)
    empty_rows = [r for r in range(R) if r % 5 == 0]
    for r in empty_rows:
        h, i = divmod(r, n_q)
        assert np.all(f64(o)[0, h, i * w.block:(i + 1) * w.block] == 0)
        assert np.all(np.isneginf(lg[0, h, i * w.block:(i + 1) * w.block]))
    valid = ~np.isneginf(l_ref)
    assert np.abs(lg[valid] - l_ref[valid]).max() <= LSE_TOL

    # a col_idx shorter than row_ptr claims: row bounds are clamped
    cut = int(rp[-1]) - 7
    o2 = L.losa_sparse_attn_fwd(q, k, v, w.N, w.block, w.bk, rp_d, ci_d[:cut])
    torch.cuda.synchronize()
    rp_cut = np.minimum(rp, cut)
    ci_cut = ci[:cut]
    keep = (ci_cut >= 0) & (ci_cut < n_k)
    rp_cut_clean = np.concatenate([[0], np.cumsum([np.sum(keep[rp_cut[r]:rp_cut[r + 1]])
                                                   for r in range(R)])])
    o_ref2, _ = O.sparse_attention(f64(q), f64(k), f64(v), w.N, w.block, w.bk, w.scale,
                                   rp_cut_clean, ci_cut[keep])
    mx, mean = CMP.output_errors(f64(o2), o_ref2, w.N)
    assert mx <= OUT_MAX and mean <= OUT_MEAN, (mx, mean)


@pytest.mark.parametrize("key", ["wan-bf16-d128-ragged", "bf16-d64-blk64", "f32-d128-blk128",
                                 "bf16-d128-r64c32", "f32-d128-r128c32"])
def test_fwd_repeated_ids_count_once(L, key):
    # K(q) of Eq. (4) is a set: an id listed twice (or more) must weigh its
    # keys once, exactly as the deduplicated row
    w = SMALL[key]
    q, k, v = W.make_inputs(w, device="cuda")
    n_q, n_k = w.n_blocks, w.n_kblocks
    R = w.B * w.H * n_q
    rng = np.random.default_rng(1234)
    rows, clean = [], []
    for r in range(R):
        base = rng.choice(n_k, size=int(rng.integers(1, n_k + 1)), replace=False)
        reps = rng.choice(base, size=int(rng.integers(1, 2 * n_k)), replace=True)
        seg = np.concatenate([base, reps, [-3, n_k]])
        rng.shuffle(seg)
        rows.append(seg)
        clean.append(np.sort(base))
    rp = np.concatenate([[0], np.cumsum([len(x) for x in rows])]).astype(np.int64)
    ci = np.concatenate(rows).astype(np.int64)
    rp_c = np.concatenate([[0], np.cumsum([len(x) for x in clean])]).astype(np.int64)
    ci_c = np.concatenate(clean).astype(np.int64)
    say(f"repeated ids {key}: {R} rows, {ci.size} entries, {ci_c.size} distinct")
    o, lse = L.losa_sparse_attn_fwd(q, k, v, w.N, w.block, w.bk,
                                    torch.from_numpy(rp.astype(np.int32)).cuda(),
                                    torch.from_numpy(ci.astype(np.int32)).cuda(), want_lse=True)
    torch.cuda.synchronize()
    o_ref, l_ref = O.sparse_attention(f64(q), f64(k), f64(v), w.N, w.block, w.bk, w.scale,
                                      rp_c, ci_c)
    tmax, tmean = out_tol(w)
    mx, mean = CMP.output_errors(f64(o), o_ref, w.N)
    assert mx <= tmax and mean <= tmean, (mx, mean)
    valid = ~np.isneginf(l_ref)
    assert np.abs(f64(lse)[valid] - l_ref[valid]).max() <= LSE_TOL


@pytest.mark.parametrize("key", ["wan-bf16-d128-ragged", "bf16-d64-blk64", "cog-bf16-d64-ragged",
                                 "cog-bf16-d64-r128c32"])
def test_fwd_writes_every_row_once(L, key):
    # the forward dispatches rows in a computed order (per-XCD, longest
    # first): every row of O and lse must be written, with the row count not
    # a multiple of 8 and rows of equal length; poison the outputs first
    w = SMALL[key]
    q, k, v = W.make_inputs(w, device="cuda")
    R = w.B * w.H * w.n_blocks
    say(f"every row {key}: {R} rows")
    mass, _ = L.losa_calibrate_mass(q, k, w.N, w.block, w.bk)
    rp, ci = L.losa_select_blocks(mass, w.N, w.block, w.bk, w.tau)
    o = torch.full_like(q, float("nan"))
    lse = torch.full((w.B, w.H, w.N_pad), float("nan"), dtype=torch.float32, device=q.device)
    L.losa_sparse_attn_fwd(q, k, v, w.N, w.block, w.bk, rp, ci, want_lse=True, out=o, lse=lse)
    torch.cuda.synchronize()
    assert not torch.isnan(o).any().item()
    assert not torch.isnan(lse).any().item()
    o_ref, _ = O.sparse_attention(f64(q), f64(k), f64(v), w.N, w.block, w.bk, w.scale,
                                  rp.cpu().numpy().astype(np.int64),
                                  ci[:L.nnz(rp)].cpu().numpy().astype(np.int64))
    mx, mean = CMP.output_errors(f64(o), o_ref, w.N)
    assert mx <= OUT_MAX and mean <= OUT_MEAN, (mx, mean)


@pytest.mark.parametrize("mag", [300.0, 1e38], ids=["x300", "near-max"])
@pytest.mark.parametrize("key", ["cog-bf16-d64-ragged", "wan-bf16-d128-r128c32", "f32-d64-blk128",
                                 "bf16-d128-blk64"])
def test_padding_contents_are_ignored(L, key, mag):
    """Rows n >= N of Q, K and V may hold any finite values: with large random
    values there (up to 1e38, near the largest bf16 and fp32 values, where a
    score against a padded key overflows to inf), every output agrees with the
    zero-padded run: padded keys are masked before the exponential, padded
    queries are read as 0 and never enter a mass.  Not bitwise: a padded query
    row shares its wave with valid rows, and its scores may trigger an earlier
    softmax rescale of the wave."""
    w = SMALL[key]
    N, Cq, Ck = w.N, w.block, w.bk
    assert N < w.N_pad
    q, k, v = W.make_inputs(w, device="cuda")
    gen = torch.Generator(device="cuda").manual_seed(5)
    qg, kg, vg = q.clone(), k.clone(), v.clone()
    for t in (qg, kg, vg):
        big = torch.randn(t[:, :, N:].shape, generator=gen, device="cuda").clamp_(-3, 3) * mag
        t[:, :, N:] = big.to(t.dtype)
        assert torch.isfinite(t).all().item()

    def run(q, k, v, fwd_csr=None):
        m1, l1 = L.losa_calibrate_mass(q, k, N, Cq, Ck)
        m2, _ = L.losa_calibrate_mass(q, k, N, Cq, Ck, two_sweep=True)
        rp, ci = L.losa_select_blocks(m1, N, Cq, Ck, w.tau)
        frp, fci = fwd_csr if fwd_csr is not None else (rp, ci)   # the forward on one support
        o, lo = L.losa_sparse_attn_fwd(q, k, v, N, Cq, Ck, frp, fci, want_lse=True)
        oc, mc = L.losa_construct(q, k, v, N, Cq, Ck)
        torch.cuda.synchronize()
        return [f64(x) for x in (m1, l1, m2, o, lo, oc, mc)], (rp, ci)

    ref, csr_ref = run(q, k, v)
    got, csr_got = run(qg, kg, vg, fwd_csr=csr_ref)
    csr_ref = (csr_ref[0], csr_ref[1][:L.nnz(csr_ref[0])])
    csr_got = (csr_got[0], csr_got[1][:L.nnz(csr_got[0])])
    tol = 1e-4 if w.dtype == "f32" else 1e-2
    for name, a, b, t in zip(("mass", "lse", "mass2", "o", "lse_o", "o_con", "mass_con"), ref, got,
                             (1e-6, 1e-5, 1e-6, tol, 1e-5, tol, 1e-6)):
        a, b = a.copy(), b.copy()
        if name.startswith("lse"):
            assert np.all(np.isneginf(b[:, :, N:])), name
            a, b = a[:, :, :N], b[:, :, :N]
        if name.startswith("o"):
            assert np.all(b[:, :, N:] == 0), name
        err = np.abs(a - b).max()
        say(f"padding {key}: {name} {err:.2e}")
        assert err <= t, (name, err)
    if not all(x.shape == y.shape and torch.equal(x, y) for x, y in zip(csr_ref, csr_got)):
        # a flip is allowed only for blocks within rounding of tau
        m = ref[0].reshape(-1, w.n_kblocks)
        details = [O.select_row(m[r], tau32(w.tau), O.num_valid_key_blocks(N, Ck),
                                (r % w.n_blocks) * Cq < N) for r in range(m.shape[0])]
        rp_g = csr_got[0].cpu().numpy().astype(np.int64)
        cmp = CMP.compare_selection(rp_g, csr_got[1].cpu().numpy().astype(np.int64), details, m,
                                    tau32(w.tau))
        assert cmp["ok"], cmp


@pytest.mark.parametrize("key", ["cog-bf16-d64-ragged", "wan-bf16-d128-r128c32"])
def test_deterministic(L, key):
    """Every entry point twice on the same inputs: bitwise equal results (no
    atomics, fixed reduction orders)."""
    w = SMALL[key]
    N, Cq, Ck = w.N, w.block, w.bk
    q, k, v = W.make_inputs(w, device="cuda")
    outs = []
    for _ in range(2):
        mass, lse = L.losa_calibrate_mass(q, k, N, Cq, Ck)
        mass2, lse2 = L.losa_calibrate_mass(q, k, N, Cq, Ck, two_sweep=True)
        rp, ci = L.losa_select_blocks(mass, N, Cq, Ck, w.tau)
        rk, ck = L.losa_select_blocks_topk(mass, N, Cq, Ck, 5)
        o, lo = L.losa_sparse_attn_fwd(q, k, v, N, Cq, Ck, rp, ci, want_lse=True)
        rr, rh = L.losa_block_recall(mass2, N, Cq, Ck, rp, ci)
        oc, mc, lc = L.losa_construct(q, k, v, N, Cq, Ck, want_lse=True)
        torch.cuda.synchronize()
        outs.append([t.clone() for t in (mass, lse, mass2, lse2, rp, ci[:L.nnz(rp)], rk,
                                         ck[:L.nnz(rk)], o, lo, rr, rh, oc, mc, lc)])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


# ----------------------------------------------------------------------------
# full-size workloads, sampled rows
# ----------------------------------------------------------------------------

# the frozen support is checked at the reuse steps of the measurement: Wan and
# CogVideoX shapes at steps 0, 1, 25, 49; HunyuanVideo at 0, 1, 49
FULL_STEPS = {"wan": (0, 1, 25, 49), "cog": (0, 1, 25, 49), "hunyuan": (0, 1, 49),
              "wan-c32": (0, 1, 49), "hunyuan-c32": (0, 1), "wan-b2": (0, 1),
              "cog-c32": (0, 1, 49)}


@pytest.mark.parametrize("key", ["wan", "cog", "hunyuan", "wan-c32", "hunyuan-c32", "wan-b2",
                                 "cog-c32"])
def test_full_size_sampled(L, key):
    # wan-b2: the Wan shape with a batch of two (the two classifier-free guidance
    # branches of a step are batch entries b = 0, 1, each with its own support)
    if key.endswith("-c32"):
        w = W.rectangular(W.WORKLOADS[key[:-4]])
    elif key.endswith("-b2"):
        w = W.scaled(W.WORKLOADS[key[:-3]], B=2, name="wan-b2")
    else:
        w = W.WORKLOADS[key]
    steps = FULL_STEPS[key]
    # the fixed sample, plus seeded random rows: every head x 8 query blocks at
    # the Wan and CogVideoX shapes, 64 rows over the whole HunyuanVideo grid,
    # 32 for the other variants
    extra = {"wan": dict(per_head=8), "cog": dict(per_head=8), "hunyuan": dict(total=64)}
    rows = sorted(set(sample_rows(w)) | set(random_rows(w, seed=len(key),
                                                        **extra.get(key, dict(total=32)))))
    info = run_case(L, w, w.tau, reuse=max(steps), rows=rows, label=f"full-{key}",
                    check_steps=steps)
    say(f"full-{key}: coverage {info['coverage']:.3f} nnz {info['nnz']}")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_max_key_blocks(L, dtype):
    """The largest supported key-block count per head, 4,096 (128 x 32 blocks,
    N = 130,975 padded to 131,072, ragged last block): every entry point of the
    pipeline at the limit, sampled rows against the oracle."""
    w = W.rectangular(W.Workload(f"maxnk-{dtype}", 1, 1, 64, dtype, (31, 65, 65), 128, 0.99,
                                 1.5, 0.5, 0.02, 0, 83))
    assert w.n_kblocks == 4096 and w.N < w.N_pad
    rows = sample_rows(w)
    info = run_case(L, w, w.tau, rows=rows, label=f"maxnk-{dtype}")
    say(f"maxnk-{dtype}: coverage {info['coverage']:.3f} nnz {info['nnz']}")
    # the construction step at the limit: masses, and the dense output through
    # the oracle's Eq. (4) over every valid key block (dense attention)
    q, k, v = W.make_inputs(w, device="cuda")
    o, mass = L.losa_construct(q, k, v, w.N, w.block, w.bk)
    torch.cuda.synchronize()
    qh, kh, vh = f64(q), f64(k), f64(v)
    n_q, n_k = w.n_blocks, w.n_kblocks
    n_kv = O.num_valid_key_blocks(w.N, w.bk)
    m_ref, _ = O.block_masses(qh, kh, w.N, w.block, w.bk, w.scale, rows_subset=rows)
    rp_full = np.arange(0, (n_q + 1) * n_kv, n_kv)
    ci_full = np.tile(np.arange(n_kv), n_q)
    o_ref, _ = O.sparse_attention(qh, kh, vh, w.N, w.block, w.bk, w.scale, rp_full, ci_full,
                                  rows_subset=rows)
    mg, og = f64(mass).reshape(-1, n_k), f64(o)
    tmax, tmean = out_tol(w)
    for r in rows:
        assert np.abs(mg[r] - m_ref.reshape(-1, n_k)[r]).max() <= MASS_TOL
        lo, hi = r * w.block, min((r + 1) * w.block, w.N)
        err = np.abs(og[0, 0, lo:hi] - o_ref[0, 0, lo:hi])
        assert err.max() <= tmax and err.mean() <= tmean
    # recall of the threshold support and the top-k rule at the limit, on the
    # construction step's masses (every row)
    rp, ci = L.losa_select_blocks(mass, w.N, w.block, w.bk, w.tau)
    rr, rh = L.losa_block_recall(mass, w.N, w.block, w.bk, rp, ci)
    kk = 1000
    rk, ck = L.losa_select_blocks_topk(mass, w.N, w.block, w.bk, kk)
    torch.cuda.synchronize()
    rp_g = rp.cpu().numpy().astype(np.int64)
    ci_g = ci[:int(rp_g[-1])].cpu().numpy().astype(np.int64)
    assert np.abs(f64(rr) - O.recall_rows(mg.reshape(mass.shape), rp_g, ci_g)).max() <= 1e-6
    rk_g = rk.cpu().numpy().astype(np.int64)
    ck_g = ck[:int(rk_g[-1])].cpu().numpy().astype(np.int64)
    for r in range(n_q):
        want = O.select_row_topk(mg[r], kk, n_kv, r * w.block < w.N).omega
        assert np.array_equal(ck_g[rk_g[r]:rk_g[r + 1]], want), r


@pytest.mark.parametrize("alpha", W.SWEEP_ALPHAS)
def test_density_sweep_sampled(L, alpha):
    pts = [p for p in W.sweep_points() if p.alpha == alpha]
    base = pts[0]
    state = W.make_state(base, device="cuda")
    q, k, v = W.cast(state, base)
    N, C = base.N, base.block
    say(f"sweep alpha={alpha}: calibrate")
    mass, _ = L.losa_calibrate_mass(q, k, N, C, want_lse=False)
    rows = sample_rows(base)
    n_q = base.n_blocks
    qh, kh, vh = f64(q), f64(k), f64(v)
    m_ref, _ = O.block_masses(qh, kh, N, C, C, base.scale, rows_subset=rows)
    flat = m_ref.reshape(-1, n_q)
    assert np.abs(f64(mass).reshape(-1, n_q)[rows] - flat[rows]).max() <= MASS_TOL
    prev_cov = 0.0
    for p in pts:
        rp, ci = L.losa_select_blocks(mass, N, C, C, p.tau)
        o = L.losa_sparse_attn_fwd(q, k, v, N, C, C, rp, ci)
        torch.cuda.synchronize()
        rp_g = rp.cpu().numpy().astype(np.int64)
        ci_g = ci[:rp_g[-1]].cpu().numpy().astype(np.int64)
        cov = rp_g[-1] / (rp_g.size - 1) / n_q
        say(f"sweep tau={p.tau} alpha={alpha}: coverage {cov:.3f}")
        assert cov >= prev_cov
        prev_cov = cov
        details = [O.select_row(flat[r], tau32(p.tau), n_q) for r in rows]
        srp, sci = sub_csr(rp_g, ci_g, rows)
        cmp = CMP.compare_selection(srp, sci, details, flat[rows], tau32(p.tau), tie=0.0)
        assert cmp["ok"], cmp
        if p.tau >= 1.0:
            ref, _ = O.sparse_attention(qh, kh, vh, N, C, C, base.scale,
                                        np.arange(rp_g.size) * n_q,
                                        np.tile(np.arange(n_q), rp_g.size - 1), rows_subset=rows)
        else:
            ref, _ = O.sparse_attention(qh, kh, vh, N, C, C, base.scale, rp_g, ci_g,
                                        rows_subset=rows)
        qrows = np.concatenate([np.arange(i * C, min((i + 1) * C, N)) + (r // n_q) * base.N_pad
                                for r in rows for i in [r % n_q]])
        err = np.abs(f64(o).reshape(-1, base.d)[qrows] - ref.reshape(-1, base.d)[qrows])
        assert err.max() <= OUT_MAX and err.mean() <= OUT_MEAN, (p.tau, err.max(), err.mean())
