"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

* a hand-worked example with exact rational answers (tests/golden),
* library special cases (torch's fp64 scaled-dot-product attention),
* closed forms (uniform attention when K = 0 or Q = 0; a dominating block),
* brute force on tiny inputs (full N x N probabilities; all key-block subsets;
  an explicit token-level mask),
* invariants the paper states (rows of A sum to one, so a query block's mass
  is R; recall >= theta at the construction step; the prefix is the shortest)
  and ones that follow from Eq. (4) (the |O_sparse - O_dense| bound).

Each ``check_*`` returns True when the pin holds; the mutation tests at the end
plant plausible mistakes in the oracle (on the CPU) and confirm that at least
one pin then fails.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import losa_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_worked_8tok.json")


def _rand_qkv(rng, B=1, H=2, N=37, Np=40, d=8, scale_qk=1.0):
    q = np.zeros((B, H, Np, d))
    k = np.zeros((B, H, Np, d))
    v = np.zeros((B, H, Np, d))
    q[:, :, :N] = rng.standard_normal((B, H, N, d)) * scale_qk
    k[:, :, :N] = rng.standard_normal((B, H, N, d)) * scale_qk
    v[:, :, :N] = rng.standard_normal((B, H, N, d))
    return q, k, v


def _full_csr(B, H, n_q, n_kv):
    rows = B * H * n_q
    row_ptr = np.arange(rows + 1) * n_kv
    col_idx = np.tile(np.arange(n_kv), rows)
    return row_ptr, col_idx


# ----------------------------------------------------------------------------
# hand-worked example
# ----------------------------------------------------------------------------

def _golden_inputs(g):
    Np, N = g["N_pad"], g["N"]
    q = np.zeros((1, 1, Np, 1))
    k = np.zeros((1, 1, Np, 1))
    v = np.zeros((1, 1, Np, 1))
    q[0, 0, :N, 0] = g["c"]
    k[0, 0, :N, 0] = np.log(np.array(g["w"], dtype=np.float64))
    v[0, 0, :N, 0] = np.arange(N)
    return q, k, v


def _fr(s):
    return float(Fraction(s))


def check_golden() -> bool:
    g = json.load(open(GOLDEN))
    q, k, v = _golden_inputs(g)
    N, R, C = g["N"], g["block_q"], g["block_k"]
    mbar, lse = O.block_masses(q, k, N, R, C, g["scale"])
    want = np.array([[_fr(x) for x in row] for row in g["mbar"]])
    if not np.allclose(mbar[0, 0], want, rtol=0, atol=1e-14):
        return False
    for sel in g["selections"]:
        rp, ci, _ = O.select_blocks(mbar, N, R, C, sel["tau"])
        if rp.tolist() != sel["row_ptr"] or ci.tolist() != sel["col_idx"]:
            return False
        o, l = O.sparse_attention(q, k, v, N, R, C, g["scale"], rp, ci)
        if not np.allclose(o[0, 0, :, 0], [_fr(x) for x in sel["o"]], rtol=0, atol=1e-13):
            return False
        if not np.allclose(np.exp(l[0, 0]), [_fr(x) for x in sel["lse_exp"]], rtol=1e-13, atol=0):
            return False
        if "recall" in sel:
            if abs(O.recall(mbar, rp, ci, N, R) - _fr(sel["recall"])) > 1e-14:
                return False
            if abs(O.coverage(rp, 1, 1, 4, 4) - _fr(sel["coverage"])) > 1e-15:
                return False
    o, l = O.dense_attention(q, k, v, N, g["scale"])
    if not np.allclose(o[0, 0, :, 0], [_fr(x) for x in g["dense"]["o"]], rtol=0, atol=1e-13):
        return False
    return bool(np.allclose(np.exp(l[0, 0]), [_fr(x) for x in g["dense"]["lse_exp"]],
                            rtol=1e-13, atol=0))


def test_hand_worked_example():
    assert check_golden()


# ----------------------------------------------------------------------------
# dense path: library special case
# ----------------------------------------------------------------------------

def check_dense_vs_sdpa(seed=0) -> bool:
    rng = np.random.default_rng(seed)
    N, Np, d = 37, 40, 8
    q, k, v = _rand_qkv(rng, N=N, Np=Np, d=d)
    scale = 1 / math.sqrt(d)
    o, lse = O.dense_attention(q, k, v, N, scale)
    qt, kt, vt = (torch.from_numpy(x[:, :, :N].copy()) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale).numpy()
    lse_ref = torch.logsumexp(scale * qt @ kt.transpose(-1, -2), dim=-1).numpy()
    return bool(np.allclose(o[:, :, :N], ref, rtol=0, atol=1e-12)
                and np.allclose(lse[:, :, :N], lse_ref, rtol=0, atol=1e-12)
                and np.all(o[:, :, N:] == 0) and np.all(np.isneginf(lse[:, :, N:])))


def check_sparse_full_equals_dense(seed=1, R=8, C=8) -> bool:
    rng = np.random.default_rng(seed)
    N, Np, d = 37, 40, 8
    q, k, v = _rand_qkv(rng, N=N, Np=Np, d=d)
    scale = 1 / math.sqrt(d)
    n_q, n_k = Np // R, Np // C
    mbar, _ = O.block_masses(q, k, N, R, C, scale)
    rp, ci, _ = O.select_blocks(mbar, N, R, C, 1.0)
    o_s, l_s = O.sparse_attention(q, k, v, N, R, C, scale, rp, ci)
    o_d, l_d = O.dense_attention(q, k, v, N, scale)
    return bool(rp[-1] == 1 * 2 * n_q * O.num_valid_key_blocks(N, C)
                and np.allclose(o_s, o_d, rtol=0, atol=1e-12)
                and np.allclose(l_s[:, :, :N], l_d[:, :, :N], rtol=0, atol=1e-12))


def test_dense_matches_torch_sdpa():
    assert check_dense_vs_sdpa()


@pytest.mark.parametrize("R,C", [(8, 8), (8, 4), (4, 8)])
def test_tau_one_reproduces_dense(R, C):
    assert check_sparse_full_equals_dense(R=R, C=C)


# ----------------------------------------------------------------------------
# block masses: invariants, closed forms, brute force
# ----------------------------------------------------------------------------

def check_masses_brute_force(seed=2, R=8, C=4) -> bool:
    rng = np.random.default_rng(seed)
    N, Np, d = 37, 40, 8
    q, k, _ = _rand_qkv(rng, N=N, Np=Np, d=d, scale_qk=1.5)
    scale = 1 / math.sqrt(d)
    mbar, lse = O.block_masses(q, k, N, R, C, scale)
    for b in range(q.shape[0]):
        for h in range(q.shape[1]):
            A = O.dense_probabilities(q, k, N, scale, b, h)          # [N, N]
            if not np.allclose(A.sum(axis=1), 1.0, rtol=0, atol=1e-12):
                return False
            for i in range(Np // R):
                rows = list(range(i * R, min((i + 1) * R, N)))
                for j in range(Np // C):
                    keys = [kk for kk in range(j * C, min((j + 1) * C, N))]
                    tot = sum(A[qq, kk] for qq in rows for kk in keys) if rows else 0.0
                    want = tot / len(rows) if rows else 0.0
                    if abs(mbar[b, h, i, j] - want) > 1e-13:
                        return False
    n_valid_q = O.ceil_div(N, R)
    return bool(np.allclose(mbar[:, :, :n_valid_q].sum(-1), 1.0, rtol=0, atol=1e-12))


def test_masses_match_brute_force_and_sum_to_one():
    assert check_masses_brute_force()


@pytest.mark.parametrize("zero", ["q", "k"])
def test_masses_uniform_closed_form(zero):
    # Q = 0 or K = 0 makes every score equal: A(q, k) = 1/N for every valid key,
    # so mbar(i, j) = |B_j intersect [0, N)| / N exactly.
    rng = np.random.default_rng(3)
    N, Np, d, R, C = 45, 48, 8, 8, 8
    q, k, _ = _rand_qkv(rng, N=N, Np=Np, d=d)
    if zero == "q":
        q[:] = 0
    else:
        k[:] = 0
    mbar, lse = O.block_masses(q, k, N, R, C, 0.3)
    want = np.array([len(O.valid_keys(j, C, N)) / N for j in range(Np // C)])
    assert np.allclose(mbar[0, :, :], want, rtol=0, atol=1e-15)
    assert np.allclose(lse[0, :, :N], math.log(N), rtol=0, atol=1e-13)


def test_dominating_block_takes_all_mass():
    # keys of block j* pushed along a direction u with q . u > 0: the block's
    # mass tends to one as the push grows.
    rng = np.random.default_rng(4)
    N, Np, d, R, C = 32, 32, 4, 8, 8
    q, k, _ = _rand_qkv(rng, N=N, Np=Np, d=d)
    q[:, :, :N] = np.abs(q[:, :, :N]) + 0.1
    u = np.ones(d) / 2
    prev = 0.0
    for lam in (1.0, 5.0, 25.0):
        kk = k.copy()
        kk[:, :, 2 * C:3 * C] += lam * u
        mbar, _ = O.block_masses(q, kk, N, R, C, 1.0)
        cur = float(mbar[:, :, :, 2].min())
        assert cur > prev
        prev = cur
    assert prev > 1 - 1e-6


# ----------------------------------------------------------------------------
# selection: brute force over subsets, invariants
# ----------------------------------------------------------------------------

def check_selection_brute_force(seed=5, trials=60) -> bool:
    rng = np.random.default_rng(seed)
    for t in range(trials):
        n_k = int(rng.integers(1, 11))
        m = rng.random(n_k) ** 3
        if t % 3 == 0:                  # force ties
            m = np.round(m * 4) / 4 + 0.01
        m = m / m.sum()
        tau = float(rng.choice([0.5, 0.8, 0.9, 0.95, 0.99]))
        sel = O.select_row(m, tau, n_k)
        best_by_size = {}
        for size in range(1, n_k + 1):
            best_by_size[size] = max(m[list(c)].sum() for c in itertools.combinations(range(n_k), size))
        s_brute = min(sz for sz, tot in best_by_size.items() if tot >= tau - 1e-15)
        if sel.s != s_brute:
            return False
        if abs(m[sel.omega].sum() - best_by_size[sel.s]) > 1e-15:
            return False
        # among equal-mass alternatives the smaller indices are kept
        thr = m[sel.order[sel.s - 1]]
        strictly = set(np.nonzero(m > thr)[0].tolist())
        ties = sorted(np.nonzero(m == thr)[0].tolist())
        want = sorted(strictly | set(ties[:sel.s - len(strictly)]))
        if sel.omega.tolist() != want:
            return False
    return True


def test_selection_is_shortest_prefix_brute_force():
    assert check_selection_brute_force()


def test_selection_nested_and_recall_at_least_tau():
    rng = np.random.default_rng(6)
    N, Np, d, R, C = 61, 64, 8, 8, 8
    q, k, _ = _rand_qkv(rng, N=N, Np=Np, d=d, scale_qk=1.3)
    mbar, _ = O.block_masses(q, k, N, R, C, 1 / math.sqrt(d))
    prev = None
    covs = []
    for tau in (0.5, 0.8, 0.9, 0.99, 0.999, 1.0):
        rp, ci, _ = O.select_blocks(mbar, N, R, C, tau)
        assert O.validate_csr(rp, ci, 2 * (Np // R), Np // C, N, R, Np // R) == []
        assert O.recall(mbar, rp, ci, N, R) >= tau - 1e-12
        sets = [set(ci[rp[r]:rp[r + 1]].tolist()) for r in range(len(rp) - 1)]
        if prev is not None:
            assert all(a <= b for a, b in zip(prev, sets))
        prev = sets
        covs.append(O.coverage(rp, 1, 2, Np // R, Np // C))
    assert covs == sorted(covs) and covs[-1] == 1.0


def check_corrupt_masses_count_as_zero(seed=11) -> bool:
    """Negative and NaN masses select exactly like zeros (both rules); the pin
    is the same row with those entries written as 0 by hand."""
    rng = np.random.default_rng(seed)
    ok = True
    for _ in range(20):
        n = int(rng.integers(3, 12))
        m = rng.dirichlet(np.ones(n))
        bad = rng.random(n) < 0.3
        if not bad.any():
            bad[0] = True
        corrupt = m.copy()
        corrupt[bad] = np.where(rng.random(bad.sum()) < 0.5, np.nan, -rng.random(bad.sum()))
        clean = m.copy()
        clean[bad] = 0.0
        for tau in (0.5, 0.9, 0.999):
            a, b = O.select_row(corrupt, tau, n), O.select_row(clean, tau, n)
            ok &= np.array_equal(a.omega, b.omega) and a.s == b.s
        for kk in (1, n // 2, n):
            a, b = O.select_row_topk(corrupt, kk, n), O.select_row_topk(clean, kk, n)
            ok &= np.array_equal(a.omega, b.omega)
    return bool(ok)


def test_corrupt_masses_count_as_zero():
    assert check_corrupt_masses_count_as_zero()


def test_padding_only_blocks_are_never_kept():
    # block_k smaller than the padding tail: key blocks made only of padding
    rng = np.random.default_rng(7)
    N, Np, d, R, C = 50, 64, 8, 16, 4   # key blocks 13..15 are all padding
    q, k, _ = _rand_qkv(rng, N=N, Np=Np, d=d)
    mbar, _ = O.block_masses(q, k, N, R, C, 0.4)
    assert np.all(mbar[..., 13:] == 0)
    for tau in (0.9, 1.0):
        rp, ci, _ = O.select_blocks(mbar, N, R, C, tau)
        assert ci.max() <= 12


# ----------------------------------------------------------------------------
# the fixed-ratio top-k rule (Table 2): brute force, link to Eq. (3), nesting
# ----------------------------------------------------------------------------

def check_topk_brute_force(seed=15, trials=40) -> bool:
    rng = np.random.default_rng(seed)
    for t in range(trials):
        n_k = int(rng.integers(1, 10))
        m = rng.random(n_k) ** 2
        if t % 2 == 0:                  # force ties
            m = np.round(m * 3) / 3 + 0.02
        m = m / m.sum()
        for k in range(1, n_k + 1):
            sel = O.select_row_topk(m, k, n_k)
            if sel.s != k or sel.omega.size != k:
                return False
            best = max(m[list(c)].sum() for c in itertools.combinations(range(n_k), k))
            if abs(m[sel.omega].sum() - best) > 1e-15:
                return False
            thr = m[sel.order[k - 1]]
            strictly = set(np.nonzero(m > thr)[0].tolist())
            ties = sorted(np.nonzero(m == thr)[0].tolist())
            if sel.omega.tolist() != sorted(strictly | set(ties[:k - len(strictly)])):
                return False
    return True


def test_topk_is_the_heaviest_k_subset_brute_force():
    assert check_topk_brute_force()


def test_topk_at_the_prefix_length_equals_the_threshold_rule():
    # both rules walk the same mass order: keeping the s of Eq. (3) blocks is
    # the threshold selection itself
    rng = np.random.default_rng(16)
    N, Np, d, R, C = 61, 64, 8, 8, 4
    q, k, _ = _rand_qkv(rng, N=N, Np=Np, d=d, scale_qk=1.3)
    mbar, _ = O.block_masses(q, k, N, R, C, 1 / math.sqrt(d))
    nkv = O.num_valid_key_blocks(N, C)
    for tau in (0.5, 0.9, 0.99):
        for row in mbar.reshape(-1, Np // C):
            sel = O.select_row(row, tau, nkv)
            assert O.select_row_topk(row, sel.s, nkv).omega.tolist() == sel.omega.tolist()


def test_topk_nested_clamped_and_padding_free():
    rng = np.random.default_rng(17)
    N, Np, d, R, C = 50, 64, 8, 16, 4   # key blocks 13..15 hold only padding
    q, k, _ = _rand_qkv(rng, N=N, Np=Np, d=d)
    mbar, _ = O.block_masses(q, k, N, R, C, 0.4)
    nkv = O.num_valid_key_blocks(N, C)
    prev = None
    for kk in range(1, Np // C + 3):
        rp, ci, _ = O.select_blocks_topk(mbar, N, R, C, kk)
        assert O.validate_csr(rp, ci, 2 * (Np // R), Np // C, N, R, Np // R) == []
        assert np.all(np.diff(rp) == min(kk, nkv))
        assert ci.max() < nkv
        sets = [set(ci[rp[r]:rp[r + 1]].tolist()) for r in range(len(rp) - 1)]
        if prev is not None:
            assert all(a <= b for a, b in zip(prev, sets))
        prev = sets
    assert all(st == set(range(nkv)) for st in prev)


# ----------------------------------------------------------------------------
# recall of a frozen support (Eq. (2)) per query block and per head
# ----------------------------------------------------------------------------

def check_recall_closed_form(seed=18) -> bool:
    # K = 0: every valid key gets probability 1/N, so M(i, j) = R_i |B_j ∩ [0,N)| / N
    # and a support's recall is the count of its distinct valid keys over N,
    # per query block and per head, exactly (duplicates and stray ids ignored)
    rng = np.random.default_rng(seed)
    N, Np, d, R, C = 45, 48, 4, 16, 8   # ragged last query and key block
    q, k, _ = _rand_qkv(rng, N=N, Np=Np, d=d)
    k[:] = 0.0
    mbar, _ = O.block_masses(q, k, N, R, C, 1.0)
    n_q, n_k = Np // R, Np // C
    rows, want = [], []
    for r in range(2 * n_q):
        js = rng.choice(n_k, size=int(rng.integers(1, n_k + 1)), replace=True)
        rows.append(np.concatenate([js, [-1, n_k + 2]]))
        want.append(sum(min(C, N - j * C) for j in set(js.tolist())) / N)
    rp = np.concatenate([[0], np.cumsum([len(x) for x in rows])])
    ci = np.concatenate(rows)
    got = O.recall_rows(mbar, rp, ci)
    if not np.allclose(got, want, rtol=0, atol=1e-12):
        return False
    Ri = np.array([min(R, N - i * R) for i in range(n_q)], dtype=float)
    heads = O.recall_heads(mbar, rp, ci, N, R)
    want_h = [(np.array(want[h * n_q:(h + 1) * n_q]) * Ri).sum() / N for h in range(2)]
    if not np.allclose(heads[0], want_h, rtol=0, atol=1e-12):
        return False
    # Eq. (2) over both heads at once: every head's queries carry N in total
    total = O.recall(mbar, rp, ci, N, R)
    return bool(abs(total - sum(want_h) / 2) <= 1e-12)


def test_recall_closed_form_uniform_attention():
    assert check_recall_closed_form()


def test_recall_weights_query_blocks_by_their_valid_rows():
    # two query blocks of one head, the second ragged with 1 valid row of 4:
    # Eq. (2) weights block recall by rows, 4 * 1.0 + 1 * 0.0 over 5 rows
    mbar = np.array([[[[0.5, 0.5], [0.25, 0.75]]]])
    rp = np.array([0, 2, 2])
    ci = np.array([0, 1])
    assert O.recall_rows(mbar, rp, ci).tolist() == [1.0, 0.0]
    assert O.recall_heads(mbar, rp, ci, 5, 4)[0, 0] == pytest.approx(0.8, abs=1e-15)
    assert O.recall(mbar, rp, ci, 5, 4) == pytest.approx(0.8, abs=1e-15)


def test_recall_full_support_one_and_at_least_tau_at_construction():
    rng = np.random.default_rng(19)
    N, Np, d, R, C = 61, 64, 8, 8, 4
    q, k, _ = _rand_qkv(rng, N=N, Np=Np, d=d, scale_qk=1.3)
    mbar, _ = O.block_masses(q, k, N, R, C, 1 / math.sqrt(d))
    rp, ci, _ = O.select_blocks(mbar, N, R, C, 1.0)
    assert np.allclose(O.recall_rows(mbar, rp, ci), 1.0, atol=1e-12)
    for tau in (0.5, 0.9, 0.99):
        rp, ci, _ = O.select_blocks(mbar, N, R, C, tau)
        assert np.all(O.recall_rows(mbar, rp, ci) >= tau - 1e-12)
        heads = O.recall_heads(mbar, rp, ci, N, R)
        assert np.all(heads >= tau - 1e-12)
        assert heads.mean() == pytest.approx(O.recall(mbar, rp, ci, N, R), abs=1e-12)


# ----------------------------------------------------------------------------
# Eq. (4): token-level brute force, special cases, error bound
# ----------------------------------------------------------------------------

def check_token_mask_equals_blockwise(seed=8, R=8, C=4, tau=0.8) -> bool:
    rng = np.random.default_rng(seed)
    N, Np, d = 37, 40, 8
    q, k, v = _rand_qkv(rng, N=N, Np=Np, d=d, scale_qk=1.4)
    scale = 1 / math.sqrt(d)
    mbar, _ = O.block_masses(q, k, N, R, C, scale)
    rp, ci, _ = O.select_blocks(mbar, N, R, C, tau)
    o_b, _ = O.sparse_attention(q, k, v, N, R, C, scale, rp, ci)
    o_t = O.token_mask_attention(q, k, v, N, R, C, scale, rp, ci)
    return bool(rp[-1] < 2 * (Np // R) * (Np // C) and np.allclose(o_b, o_t, rtol=0, atol=1e-12))


def check_out_of_range_ids_ignored(seed=9, R=8, C=4) -> bool:
    """A CSR with unordered, repeated and out-of-range ids (negative and >= n_k)
    against the token-level mask, which by construction only ever matches
    key blocks 0 .. n_kv-1."""
    rng = np.random.default_rng(seed)
    N, Np, d = 37, 40, 8
    q, k, v = _rand_qkv(rng, N=N, Np=Np, d=d, scale_qk=1.4)
    scale = 1 / math.sqrt(d)
    rows = q.shape[0] * q.shape[1] * (Np // R)
    n_k = Np // C
    lens = rng.integers(0, n_k + 4, size=rows)
    rp = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    ci = rng.integers(-3, n_k + 3, size=int(rp[-1])).astype(np.int64)
    if not ((ci < 0).any() and (ci >= n_k).any()):
        return False
    o_b, _ = O.sparse_attention(q, k, v, N, R, C, scale, rp, ci)
    o_t = O.token_mask_attention(q, k, v, N, R, C, scale, rp, ci)
    # and with the out-of-range ids removed beforehand
    keep = (ci >= 0) & (ci < n_k)
    rp2 = np.concatenate([[0], np.cumsum([keep[rp[i]:rp[i + 1]].sum() for i in range(rows)])])
    o_c, _ = O.sparse_attention(q, k, v, N, R, C, scale, rp2.astype(np.int64), ci[keep])
    return bool(np.allclose(o_b, o_t, rtol=0, atol=1e-12) and np.array_equal(o_b, o_c))


def test_out_of_range_ids_are_ignored():
    assert check_out_of_range_ids_ignored()


@pytest.mark.parametrize("R,C", [(8, 8), (8, 4), (4, 8)])
def test_token_mask_brute_force(R, C):
    assert check_token_mask_equals_blockwise(R=R, C=C)


def test_single_block_support_is_softmax_over_that_block():
    rng = np.random.default_rng(9)
    N, Np, d, R, C = 30, 32, 4, 8, 8
    q, k, v = _rand_qkv(rng, N=N, Np=Np, d=d)
    rows = 1 * 1 * (Np // R)
    rp = np.arange(rows + 1)
    ci = np.array([3, 0, 2, 1])
    o, _ = O.sparse_attention(q[:, :1], k[:, :1], v[:, :1], N, R, C, 0.5, rp, ci)
    for i, j in enumerate(ci):
        keys = O.valid_keys(j, C, N)
        for qq in O.valid_rows(i, R, N):
            s = 0.5 * k[0, 0, keys] @ q[0, 0, qq]
            p = np.exp(s - s.max())
            p /= p.sum()
            assert np.allclose(o[0, 0, qq], p @ v[0, 0, keys], rtol=0, atol=1e-13)


def test_output_invariant_to_order_within_row():
    rng = np.random.default_rng(10)
    N, Np, d, R, C = 40, 40, 8, 8, 8
    q, k, v = _rand_qkv(rng, N=N, Np=Np, d=d)
    mbar, _ = O.block_masses(q, k, N, R, C, 0.35)
    rp, ci, _ = O.select_blocks(mbar, N, R, C, 0.9)
    ci2 = ci.copy()
    for r in range(len(rp) - 1):
        ci2[rp[r]:rp[r + 1]] = ci2[rp[r]:rp[r + 1]][::-1]
    o1, _ = O.sparse_attention(q, k, v, N, R, C, 0.35, rp, ci)
    o2, _ = O.sparse_attention(q, k, v, N, R, C, 0.35, rp, ci2)
    assert np.allclose(o1, o2, rtol=0, atol=1e-14)


def test_sparse_dense_error_bound():
    # From Eq. (4): O_dense(q) = r_q O_sparse(q) + (1 - r_q) O_dropped(q), with
    # r_q the kept probability of row q, so |O_sparse - O_dense| <= 2 (1 - r_q) max|V|.
    rng = np.random.default_rng(11)
    N, Np, d, R, C = 61, 64, 8, 8, 8
    q, k, v = _rand_qkv(rng, N=N, Np=Np, d=d, scale_qk=1.3)
    scale = 1 / math.sqrt(d)
    mbar, _ = O.block_masses(q, k, N, R, C, scale)
    rp, ci, _ = O.select_blocks(mbar, N, R, C, 0.9)
    o_s, _ = O.sparse_attention(q, k, v, N, R, C, scale, rp, ci)
    o_d, _ = O.dense_attention(q, k, v, N, scale)
    n_q = Np // R
    for h in range(2):
        A = O.dense_probabilities(q, k, N, scale, 0, h)
        vmax = np.abs(v[0, h, :N]).max()
        for qq in range(N):
            r = h * n_q + qq // R
            kept = ci[rp[r]:rp[r + 1]]
            keymask = np.isin(np.arange(N) // C, kept)
            r_q = A[qq, keymask].sum()
            err = np.abs(o_s[0, h, qq] - o_d[0, h, qq]).max()
            assert err <= 2 * (1 - r_q) * vmax + 1e-12


def test_validate_csr_flags_corruption():
    rp = np.array([0, 2, 3])
    ci = np.array([0, 1, 1])
    assert O.validate_csr(rp, ci, 2, 4) == []
    assert O.validate_csr(np.array([0, 3, 2]), ci, 2, 4)
    assert O.validate_csr(rp, np.array([1, 0, 1]), 2, 4)
    assert O.validate_csr(rp, np.array([0, 4, 1]), 2, 4)
    assert O.validate_csr(np.array([1, 2, 3]), ci, 2, 4)


# ----------------------------------------------------------------------------
# mutation tests: plausible mistakes planted in the oracle must fail a pin
# ----------------------------------------------------------------------------

def _softmax_no_norm(S):
    m = S.max(axis=1, keepdims=True)
    e = np.exp(S - m)
    return e, (m + np.log(e.sum(axis=1, keepdims=True)))[:, 0]


def _softmax_wrong_axis(S):
    m = S.max(axis=0, keepdims=True)
    e = np.exp(S - m)
    l = e.sum(axis=0, keepdims=True)
    return e / l, (m + np.log(l))[0, :]


def _order_ties_high_first(mrow):
    idx = np.arange(mrow.size)
    return np.lexsort((-idx, -np.asarray(mrow)))


def _order_ascending(mrow):
    idx = np.arange(mrow.size)
    return np.lexsort((idx, np.asarray(mrow)))


def _select_row_strict(mrow, tau, n_k_valid, has_valid_rows=True):
    # ">" instead of ">=" and one block too many
    sel = _orig_select_row(mrow, tau, n_k_valid, has_valid_rows)
    if 0 < sel.s < n_k_valid and tau < 1:
        s = sel.s + 1
        sel = O.RowSelection(sel.order, sel.cum, s, np.sort(sel.order[:s]))
    return sel


def _sparse_v_is_k(q, k, v, *a, **kw):
    return _orig_sparse(q, k, k, *a, **kw)


def _sparse_no_scale(q, k, v, N, R, C, scale, rp, ci, rows_subset=None):
    return _orig_sparse(q, k, v, N, R, C, 1.0, rp, ci, rows_subset)


def _sparse_ids_wrap(q, k, v, N, R, C, scale, rp, ci, rows_subset=None):
    # a negative block id taken modulo n_k instead of being ignored
    ci = np.asarray(ci, dtype=np.int64)
    n_k = np.asarray(q).shape[2] // C
    return _orig_sparse(q, k, v, N, R, C, scale, rp, np.where(ci < 0, ci % n_k, ci), rows_subset)


def _clean_masses_kept_negative(mrow):
    # corrupt masses read as they are instead of as 0
    return np.asarray(mrow, dtype=np.float64)


def _masses_sum_not_mean(q, k, N, R, C, scale):
    mbar, lse = _orig_masses(q, k, N, R, C, scale)
    return mbar * R, lse


def _masses_include_padding(q, k, N, R, C, scale):
    Np = q.shape[2]
    return _orig_masses(q, k, Np, R, C, scale)


def _recall_rows_counts_duplicates(mbar, row_ptr, col_idx):
    mbar = np.asarray(mbar, dtype=np.float64)
    n_k = mbar.shape[-1]
    flat = mbar.reshape(-1, n_k)
    out = np.zeros(flat.shape[0])
    for r in range(flat.shape[0]):
        js = np.asarray(col_idx[row_ptr[r]:row_ptr[r + 1]])
        out[r] = flat[r, js[(js >= 0) & (js < n_k)]].sum()
    return out


def _recall_ids_wrap(mbar, row_ptr, col_idx, N, block_q):
    # a negative block id taken modulo n_k instead of being ignored
    n_k = np.asarray(mbar).shape[-1]
    ci = np.asarray(col_idx, dtype=np.int64)
    return _orig_recall(mbar, row_ptr, np.where(ci < 0, ci % n_k, ci), N, block_q)


def _recall_heads_unweighted(mbar, row_ptr, col_idx, N, block_q):
    B, H, n_q, _ = np.asarray(mbar).shape
    return O.recall_rows(mbar, row_ptr, col_idx).reshape(B, H, n_q).mean(axis=2)


def _topk_off_by_one(mrow, k, n_k_valid, has_valid_rows=True):
    return _orig_topk(mrow, max(k - 1, 0), n_k_valid, has_valid_rows)


_orig_sparse = O.sparse_attention
_orig_masses = O.block_masses
_orig_select_row = O.select_row
_orig_topk = O.select_row_topk
_orig_recall = O.recall

ALL_PINS = [check_golden, check_dense_vs_sdpa, check_sparse_full_equals_dense,
            check_masses_brute_force, check_selection_brute_force,
            check_token_mask_equals_blockwise, check_topk_brute_force,
            check_recall_closed_form, check_out_of_range_ids_ignored,
            check_corrupt_masses_count_as_zero]


def _some_pin_fails():
    for pin in ALL_PINS:
        try:
            if not pin():
                return True
        except Exception:
            return True
    return False


@pytest.mark.parametrize("attr,mutant", [
    ("row_softmax", _softmax_no_norm),
    ("row_softmax", _softmax_wrong_axis),
    ("mass_order", _order_ties_high_first),
    ("mass_order", _order_ascending),
    ("select_row", _select_row_strict),
    ("sparse_attention", _sparse_v_is_k),
    ("sparse_attention", _sparse_no_scale),
    ("sparse_attention", _sparse_ids_wrap),
    ("clean_masses", _clean_masses_kept_negative),
    ("block_masses", _masses_sum_not_mean),
    ("block_masses", _masses_include_padding),
    ("select_row_topk", _topk_off_by_one),
    ("recall_rows", _recall_rows_counts_duplicates),
    ("recall_heads", _recall_heads_unweighted),
    ("recall", _recall_ids_wrap),
])
def test_planted_mistake_is_caught(monkeypatch, attr, mutant):
    assert not _some_pin_fails(), "pins must hold for the unmodified oracle"
    monkeypatch.setattr(O, attr, mutant)
    assert _some_pin_fails(), f"mutant {mutant.__name__} of {attr} passed every pin"
