"""Plain fp64 CPU oracle for LoSA's attention hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  It shares no code
with the HIP path (``paper_2608_12032_amd``) and never imports it.

Every function writes out the paper's definitions directly, in float64, with a
library matmul / exp / sort as its only primitives and no blocking, fusion or
reordering beyond what the definition states:

* dense attention, A = row-softmax(Q K^T / sqrt(d))          -- Sec. 3.1
* block attention mass M(i, j)                                -- Sec. 3.1, Eq. (1)
* Recall(Omega) and Coverage(Omega)                           -- Sec. 3.1, Eq. (2)
* mass-ordered shortest prefix s and the set Omega            -- Sec. 4.1, Eq. (3)
* frozen-support (block-sparse) attention                     -- Sec. 4.2, Eq. (4)
* the fixed-ratio top-k rule of the selection ablation        -- Sec. 5, Table 2
* recall of a frozen support per query block and per head     -- Sec. 3.1, Eq. (2)

Readings taken where the paper is silent (each is also what the GPU path does):

* The mass of a query block is stored divided by its number of valid rows
  (``mbar = M / R_i``).  Each row of A sums to one, so a full block's masses sum
  to R and Eq. (3)'s test ``>= theta * R`` becomes ``mbar >= theta``.
* Token positions ``n >= N`` are padding: they never enter a softmax as keys,
  padding query rows are left out of every mass, and their outputs are zero
  with lse = -inf.  A query block with no valid row has an empty Omega.
* Ties in the mass order (Sec. 4.1 leaves them arbitrary) are broken by the
  smaller key-block index first.
* ``tau >= 1`` keeps every key block that holds at least one valid key, so the
  sparse path then equals dense attention.
* Omega is a set: within a CSR row the indices are kept ascending.

Parity pins for every function here live in ``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


# ----------------------------------------------------------------------------
# shapes
# ----------------------------------------------------------------------------

def ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def padded_len(N: int, block_q: int, block_k: int) -> int:
    """Padded sequence length: N rounded up to the larger block size."""
    L = max(block_q, block_k)
    return ceil_div(N, L) * L


def valid_rows(i: int, block_q: int, N: int) -> np.ndarray:
    """Token indices of query block B^Q_i that are < N (Sec. 3.1 partition)."""
    return np.arange(i * block_q, min((i + 1) * block_q, N))


def valid_keys(j: int, block_k: int, N: int) -> np.ndarray:
    """Token indices of key/value block B^K_j that are < N (Sec. 3.1 partition)."""
    return np.arange(j * block_k, min((j + 1) * block_k, N))


def num_valid_key_blocks(N: int, block_k: int) -> int:
    return ceil_div(N, block_k)


# ----------------------------------------------------------------------------
# dense attention and the row softmax (Sec. 3.1)
# ----------------------------------------------------------------------------

def row_softmax(S: np.ndarray):
    """Row-wise softmax of a score matrix; returns (A, lse) with lse natural-log."""
    m = S.max(axis=1, keepdims=True)
    e = np.exp(S - m)
    l = e.sum(axis=1, keepdims=True)
    return e / l, (m + np.log(l))[:, 0]


def dense_attention(q, k, v, N: int, scale: float):
    """A = softmax(scale * Q K^T) over the N valid keys, O = A V.

    q, k, v: [B, H, N_pad, d] (any float dtype; converted exactly to fp64).
    Returns (o [B,H,N_pad,d] fp64, lse [B,H,N_pad] fp64); padding rows: o = 0,
    lse = -inf.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, H, Np, d = q.shape
    o = np.zeros((B, H, Np, v.shape[-1]))
    lse = np.full((B, H, Np), -np.inf)
    for b in range(B):
        for h in range(H):
            S = scale * (q[b, h, :N] @ k[b, h, :N].T)
            A, l = row_softmax(S)
            o[b, h, :N] = A @ v[b, h, :N]
            lse[b, h, :N] = l
    return o, lse


def dense_probabilities(q, k, N: int, scale: float, b: int = 0, h: int = 0):
    """The full N x N probability matrix A of one head (tiny inputs only)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    S = scale * (q[b, h, :N] @ k[b, h, :N].T)
    return row_softmax(S)[0]


# ----------------------------------------------------------------------------
# block attention mass (Sec. 3.1, Eq. (1))
# ----------------------------------------------------------------------------

def block_masses(q, k, N: int, block_q: int, block_k: int, scale: float, rows_subset=None):
    """Exact block masses of the dense step.

    For each (b, h, i): A = softmax over all N valid keys of scale * q k^T for
    the valid rows q of B^Q_i; Mrow[q, j] = sum_{k in B^K_j, k < N} A[q, k];
    mbar[i, j] = mean over those rows of Mrow[q, j]  (= M(i, j) / R_i, Eq. (1)).

    Returns (mbar [B,H,n_q,n_k] fp64, lse [B,H,N_pad] fp64, natural log; -inf
    on padding rows).  A query block with no valid row gets an all-zero row.
    ``rows_subset``: optional iterable of rows r = (b*H + h)*n_q + i to compute
    (the others stay zero / -inf).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    B, H, Np, d = q.shape
    n_q, n_k = Np // block_q, Np // block_k
    mbar = np.zeros((B, H, n_q, n_k))
    lse = np.full((B, H, Np), -np.inf)
    todo = range(B * H * n_q) if rows_subset is None else rows_subset
    for r in todo:
        b, rem = divmod(int(r), H * n_q)
        h, i = divmod(rem, n_q)
        rows = valid_rows(i, block_q, N)
        if rows.size == 0:
            continue
        S = scale * (q[b, h, rows] @ k[b, h, :N].T)
        A, l = row_softmax(S)
        lse[b, h, rows] = l
        # per-row mass of every key block: sum the probabilities of its valid
        # keys (padding keys carry no probability)
        Apad = np.zeros((rows.size, n_k * block_k))
        Apad[:, :N] = A
        Mrow = Apad.reshape(rows.size, n_k, block_k).sum(axis=2)
        mbar[b, h, i] = Mrow.mean(axis=0)
    return mbar, lse


# ----------------------------------------------------------------------------
# shortest-prefix selection and CSR storage (Sec. 4.1, Eq. (3))
# ----------------------------------------------------------------------------

@dataclass
class RowSelection:
    order: np.ndarray   # pi: key-block ids by decreasing mass (ties: smaller id first)
    cum: np.ndarray     # cum[r] = sum of the first r+1 masses in that order (fp64)
    s: int              # prefix length kept
    omega: np.ndarray   # sorted ascending ids of the kept blocks


def mass_order(mrow: np.ndarray) -> np.ndarray:
    """pi: indices sorted by decreasing mass, ties by increasing index."""
    idx = np.arange(mrow.size)
    return np.lexsort((idx, -np.asarray(mrow, dtype=np.float64)))


def clean_masses(mrow) -> np.ndarray:
    """Masses as the selection reads them: a mass is a probability sum, so a
    negative or NaN entry (a corrupt input) counts as 0."""
    m = np.asarray(mrow, dtype=np.float64)
    return np.where(m > 0, m, 0.0)


def select_row(mrow, tau: float, n_k_valid: int, has_valid_rows: bool = True) -> RowSelection:
    """Eq. (3): the shortest prefix of the mass order whose sum reaches tau."""
    mrow = clean_masses(mrow)
    order = mass_order(mrow)
    cum = np.cumsum(mrow[order])
    if not has_valid_rows:
        s = 0
        omega = np.zeros(0, dtype=np.int64)
    elif tau >= 1.0:
        s = n_k_valid
        omega = np.arange(n_k_valid)
    else:
        hit = np.nonzero(cum >= tau)[0]
        if hit.size:
            s = max(int(hit[0]) + 1, 1)
            omega = np.sort(order[:s])
        else:
            # the masses never reach tau (they sum below it): keep every
            # block that holds a valid key, as for tau >= 1
            s = n_k_valid
            omega = np.arange(n_k_valid)
    return RowSelection(order=order, cum=cum, s=s, omega=omega.astype(np.int64))


def select_blocks(mbar, N: int, block_q: int, block_k: int, tau: float):
    """Apply Eq. (3) to every (b, h, i) row; emit Omega as CSR.

    Returns (row_ptr int64 [rows+1], col_idx int64 [nnz], details) where row
    r = (b*H + h)*n_q + i and details[r] is that row's RowSelection.
    """
    mbar = np.asarray(mbar, dtype=np.float64)
    B, H, n_q, n_k = mbar.shape
    nkv = num_valid_key_blocks(N, block_k)
    rows = B * H * n_q
    row_ptr = np.zeros(rows + 1, dtype=np.int64)
    cols = []
    details = []
    for b in range(B):
        for h in range(H):
            for i in range(n_q):
                r = (b * H + h) * n_q + i
                sel = select_row(mbar[b, h, i], tau, nkv, i * block_q < N)
                details.append(sel)
                cols.append(sel.omega)
                row_ptr[r + 1] = row_ptr[r] + sel.omega.size
    col_idx = np.concatenate(cols) if cols else np.zeros(0, dtype=np.int64)
    return row_ptr, col_idx.astype(np.int64), details


def select_row_topk(mrow, k: int, n_k_valid: int, has_valid_rows: bool = True) -> RowSelection:
    """Fixed-ratio top-k rule (the ablation of Table 2): the k largest masses of
    the row in the same order as Eq. (3)'s (ties: smaller index first), k
    clamped to the blocks that hold a valid key.  Padding-only blocks carry no
    mass and have the largest indices, so they never enter while k <= n_k_valid."""
    mrow = clean_masses(mrow)
    order = mass_order(mrow)
    cum = np.cumsum(mrow[order])
    s = min(int(k), n_k_valid) if has_valid_rows else 0
    return RowSelection(order=order, cum=cum, s=s, omega=np.sort(order[:s]).astype(np.int64))


def select_blocks_topk(mbar, N: int, block_q: int, block_k: int, k: int):
    """The top-k rule on every (b, h, i) row, emitted as CSR like select_blocks."""
    mbar = np.asarray(mbar, dtype=np.float64)
    B, H, n_q, n_k = mbar.shape
    nkv = num_valid_key_blocks(N, block_k)
    rows = B * H * n_q
    row_ptr = np.zeros(rows + 1, dtype=np.int64)
    cols, details = [], []
    for r in range(rows):
        b, rem = divmod(r, H * n_q)
        h, i = divmod(rem, n_q)
        sel = select_row_topk(mbar[b, h, i], k, nkv, i * block_q < N)
        details.append(sel)
        cols.append(sel.omega)
        row_ptr[r + 1] = row_ptr[r] + sel.omega.size
    col_idx = np.concatenate(cols) if cols else np.zeros(0, dtype=np.int64)
    return row_ptr, col_idx.astype(np.int64), details


def validate_csr(row_ptr, col_idx, rows: int, n_k: int, N: int | None = None,
                 block_q: int | None = None, n_q: int | None = None) -> list[str]:
    """Structural checks of a CSR block list; returns the problems found."""
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col_idx = np.asarray(col_idx, dtype=np.int64)
    errs = []
    if row_ptr.shape != (rows + 1,):
        return [f"row_ptr has shape {row_ptr.shape}, expected ({rows + 1},)"]
    if row_ptr[0] != 0:
        errs.append("row_ptr[0] != 0")
    if np.any(np.diff(row_ptr) < 0):
        errs.append("row_ptr not monotone")
    if row_ptr[-1] != col_idx.size:
        errs.append(f"row_ptr[-1]={row_ptr[-1]} != nnz={col_idx.size}")
    if col_idx.size and (col_idx.min() < 0 or col_idx.max() >= n_k):
        errs.append("col_idx out of range")
    for r in range(rows):
        seg = col_idx[row_ptr[r]:row_ptr[r + 1]]
        if seg.size > 1 and np.any(np.diff(seg) <= 0):
            errs.append(f"row {r}: indices not strictly ascending")
            break
        if N is not None and block_q is not None and n_q is not None:
            i = r % n_q
            if i * block_q < N and seg.size == 0:
                errs.append(f"row {r}: empty but has valid query rows")
                break
    return errs


# ----------------------------------------------------------------------------
# frozen-support attention (Sec. 4.2, Eq. (4))
# ----------------------------------------------------------------------------

def sparse_attention(q, k, v, N: int, block_q: int, block_k: int, scale: float,
                     row_ptr, col_idx, rows_subset=None):
    """Eq. (4): each query attends to the union of its block's retained key
    blocks, with the softmax renormalised over those keys only.

    A direct fp64 softmax over the gathered keys (no online rescaling).
    ``rows_subset``: optional iterable of CSR rows to compute (others stay 0).
    Returns (o [B,H,N_pad,d] fp64, lse [B,H,N_pad] fp64).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col_idx = np.asarray(col_idx, dtype=np.int64)
    B, H, Np, d = q.shape
    n_q, n_k = Np // block_q, Np // block_k
    o = np.zeros((B, H, Np, v.shape[-1]))
    lse = np.full((B, H, Np), -np.inf)
    todo = range(B * H * n_q) if rows_subset is None else rows_subset
    for r in todo:
        b, rem = divmod(int(r), H * n_q)
        h, i = divmod(rem, n_q)
        rows = valid_rows(i, block_q, N)
        if rows.size == 0:
            continue
        # Omega is a set of key blocks: repeated ids count once, and an id
        # outside [0, n_k) names no key block (it contributes no key)
        blocks = np.unique(col_idx[row_ptr[r]:row_ptr[r + 1]])
        blocks = blocks[(blocks >= 0) & (blocks < n_k)]
        keys = (np.concatenate([valid_keys(int(j), block_k, N) for j in blocks])
                if blocks.size else np.zeros(0, dtype=np.int64))
        if keys.size == 0:
            continue
        S = scale * (q[b, h, rows] @ k[b, h, keys].T)
        A, l = row_softmax(S)
        o[b, h, rows] = A @ v[b, h, keys]
        lse[b, h, rows] = l
    return o, lse


def token_mask_attention(q, k, v, N: int, block_q: int, block_k: int, scale: float,
                         row_ptr, col_idx):
    """Brute-force Eq. (4) through an explicit token-level mask (tiny N only).

    Builds the full N x N score matrix of each head, masks out every (q, k)
    whose key block is not in Omega of q's query block, then softmaxes.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col_idx = np.asarray(col_idx, dtype=np.int64)
    B, H, Np, d = q.shape
    n_q = Np // block_q
    o = np.zeros((B, H, Np, v.shape[-1]))
    tok = np.arange(N)
    for b in range(B):
        for h in range(H):
            S = scale * (q[b, h, :N] @ k[b, h, :N].T)
            mask = np.zeros((N, N), dtype=bool)
            for qi in range(N):
                r = (b * H + h) * n_q + qi // block_q
                kept = set(int(j) for j in col_idx[row_ptr[r]:row_ptr[r + 1]])
                mask[qi] = np.isin(tok // block_k, list(kept))
            for qi in range(N):
                if not mask[qi].any():
                    continue
                s = S[qi, mask[qi]]
                p = np.exp(s - s.max())
                p /= p.sum()
                o[b, h, qi] = p @ v[b, h, :N][mask[qi]]
    return o


# ----------------------------------------------------------------------------
# Recall and Coverage (Sec. 3.1, Eq. (2))
# ----------------------------------------------------------------------------

def coverage(row_ptr, B: int, H: int, n_q: int, n_k: int) -> float:
    """Coverage = mean over heads of sum_i |Omega_i| / (n_q n_k)."""
    nnz = int(np.asarray(row_ptr)[-1])
    return nnz / float(B * H * n_q * n_k)


def recall_rows(mbar, row_ptr, col_idx) -> np.ndarray:
    """Per query block: the retained share of its mass, sum over the distinct
    ids of Omega_r inside [0, n_k) of mbar(r, j).  Masses of a query block sum
    to one, so this is Eq. (2) restricted to that block."""
    mbar = np.asarray(mbar, dtype=np.float64)
    n_k = mbar.shape[-1]
    flat = mbar.reshape(-1, n_k)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col_idx = np.asarray(col_idx, dtype=np.int64)
    out = np.zeros(flat.shape[0])
    for r in range(flat.shape[0]):
        js = np.unique(col_idx[row_ptr[r]:row_ptr[r + 1]])
        js = js[(js >= 0) & (js < n_k)]
        out[r] = flat[r, js].sum()
    return out


def recall_heads(mbar, row_ptr, col_idx, N: int, block_q: int) -> np.ndarray:
    """Eq. (2) per (b, h): sum_i sum_{j in Omega_i} M(i, j) / sum_i sum_j M(i, j)
    with M(i, j) = R_i * mbar(i, j), R_i the valid rows of query block i
    (so the denominator is N).  Returns [B, H]."""
    mbar = np.asarray(mbar, dtype=np.float64)
    B, H, n_q, n_k = mbar.shape
    Ri = np.array([valid_rows(i, block_q, N).size for i in range(n_q)], dtype=np.float64)
    rec = recall_rows(mbar, row_ptr, col_idx).reshape(B, H, n_q)
    tot = (mbar * Ri[None, None, :, None]).sum(axis=(2, 3))
    return (rec * Ri[None, None, :]).sum(axis=2) / tot


def recall(mbar, row_ptr, col_idx, N: int, block_q: int) -> float:
    """Eq. (2) over all heads together, with M(i, j) = R_i * mbar(i, j) (R_i =
    valid rows of block i).  Omega_i is a set of key blocks: a repeated id
    counts once, and an id outside [0, n_k) names no block and is ignored."""
    mbar = np.asarray(mbar, dtype=np.float64)
    B, H, n_q, n_k = mbar.shape
    Ri = np.array([valid_rows(i, block_q, N).size for i in range(n_q)], dtype=np.float64)
    M = mbar * Ri[None, None, :, None]
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col_idx = np.asarray(col_idx, dtype=np.int64)
    kept = 0.0
    flat = M.reshape(B * H * n_q, n_k)
    for r in range(B * H * n_q):
        js = np.unique(col_idx[row_ptr[r]:row_ptr[r + 1]])
        js = js[(js >= 0) & (js < n_k)]
        kept += flat[r, js].sum()
    return kept / M.sum()
