"""Seeded random configurations against the oracle: batch and head counts,
lengths, head dims, block shapes, dtypes and thresholds drawn at random (a
fixed list of seeds, so every run checks the same cases), plus a random CSR
with repeated, unordered and out-of-range ids for the forward and the recall.
Every entry point is compared on every row.

Output tolerance.  The fixed bf16 bound (max 2e-2, mean 2e-3) is stated for
the workloads, whose outputs stay near unit size.  Here Q and K are scaled by
up to 3, so a softmax can be so peaked that an output is one V row of size 4
and more; its bf16 rounding alone then reaches 2^-8 |o| (half an ulp), and
rounding P to bf16 for P V adds up to 2^-9 max|v|.  The bound used here is
derived from that arithmetic, per element:
    |o - o_ref| <= 1e-2 + 2^-8 (|o_ref| + max|v|)   (bf16; fp32: 1e-4).
It is asserted on every element, and beside it the workloads' own bars: max-abs
2e-2 on every element whose exact output stays in the workloads' range
(|o_ref| <= 1, where half an output ulp is at most 2^-9), and mean-abs 2e-3
over all valid elements.  Only the few outputs above 1 are judged by the
arithmetic bound alone."""
import numpy as np
import pytest
import torch

from oracle import compare as CMP
from oracle import losa_oracle as O

pytestmark = pytest.mark.gpu

BLOCKS = [(64, 64), (128, 128), (128, 32), (64, 32)]
SEEDS = list(range(200))


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2608_12032_amd import losa
    return losa


def f64(x):
    return x.detach().float().cpu().numpy().astype(np.float64)


def draw(seed):
    rng = np.random.default_rng(7000 + seed)
    Cq, Ck = BLOCKS[rng.integers(len(BLOCKS))]
    return dict(B=int(rng.integers(1, 3)), H=int(rng.integers(1, 4)),
                N=int(rng.integers(1, 700)), d=int(rng.choice([64, 128])), Cq=Cq, Ck=Ck,
                dtype=str(rng.choice(["bf16", "f32"])),
                tau=float(rng.choice([0.1, 0.5, 0.9, 0.99, 0.999, 1.0])),
                spread=float(rng.uniform(0.5, 3.0)), rng=rng)


@pytest.mark.parametrize("seed", SEEDS)
def test_random_configuration(L, seed):
    c = draw(seed)
    B, H, N, d, Cq, Ck, dtype, tau, rng = (c[k] for k in ("B", "H", "N", "d", "Cq", "Ck",
                                                          "dtype", "tau", "rng"))
    print(f"[gpu-random] seed {seed}: B={B} H={H} N={N} d={d} blocks={Cq}x{Ck} {dtype} "
          f"tau={tau}", flush=True)
    Np = O.padded_len(N, Cq, Ck)
    # the spread shapes the softmax through Q and K; V stays N(0, 1) as in the
    # workloads, the scale the absolute output tolerances are stated for
    t = torch.from_numpy(rng.standard_normal((3, B, H, Np, d))).float()
    t[:2] *= c["spread"]
    t[:, :, :, N:] = 0
    t = t.to(torch.bfloat16 if dtype == "bf16" else torch.float32).cuda()
    q, k, v = t[0].contiguous(), t[1].contiguous(), t[2].contiguous()
    scale = 1.0 / np.sqrt(d)
    qh, kh, vh = f64(q), f64(k), f64(v)
    n_q, n_k = Np // Cq, Np // Ck
    R = B * H * n_q
    vmax = float(np.abs(vh).max())

    def close(o, o_ref):
        err = np.abs(o[:, :, :N] - o_ref[:, :, :N])
        if dtype == "bf16":
            mag = np.abs(o_ref[:, :, :N])
            bound = 1e-2 + 2.0 ** -8 * (mag + vmax)
            in_range = mag <= 1.0
            return bool(np.all(err <= bound) and err[in_range].max(initial=0.0) <= 2e-2
                        and err.mean() <= 2e-3), err
        return bool(err.max() <= 1e-4), err

    m_ref, l_ref = O.block_masses(qh, kh, N, Cq, Ck, scale)
    mass, lse = L.losa_calibrate_mass(q, k, N, Cq, Ck)
    torch.cuda.synchronize()
    assert np.abs(f64(mass) - m_ref).max() <= 1e-4
    assert np.abs(f64(lse)[:, :, :N] - l_ref[:, :, :N]).max() <= 1e-3

    t32 = float(np.float32(tau))
    rp, ci = L.losa_select_blocks(mass, N, Cq, Ck, tau)
    rp_g = rp.cpu().numpy().astype(np.int64)
    ci_g = ci[:rp_g[-1]].cpu().numpy().astype(np.int64)
    _, _, details = O.select_blocks(m_ref, N, Cq, Ck, t32)
    cmp = CMP.compare_selection(rp_g, ci_g, details, m_ref.reshape(R, n_k), t32)
    assert cmp["ok"], cmp

    # the forward and the recall on a random CSR: unordered, repeated and
    # out-of-range ids, empty rows
    lens = rng.integers(0, n_k + 3, size=R)
    ids = [rng.integers(-2, n_k + 2, size=n) for n in lens]
    rp_r = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    ci_r = np.concatenate(ids).astype(np.int64) if rp_r[-1] else np.zeros(0, np.int64)
    rp_t = torch.tensor(rp_r, dtype=torch.int32, device="cuda")
    ci_t = torch.tensor(ci_r if ci_r.size else np.zeros(1, np.int64), dtype=torch.int32,
                        device="cuda")
    o, lo = L.losa_sparse_attn_fwd(q, k, v, N, Cq, Ck, rp_t, ci_t, want_lse=True)
    rr, rh = L.losa_block_recall(mass, N, Cq, Ck, rp_t, ci_t)
    torch.cuda.synchronize()
    o_ref, lo_ref = O.sparse_attention(qh, kh, vh, N, Cq, Ck, scale, rp_r, ci_r)
    ok, err = close(f64(o), o_ref)
    assert ok, (err.max(), err.mean())
    assert np.all(f64(o)[:, :, N:] == 0)
    lg, lr = f64(lo)[:, :, :N], lo_ref[:, :, :N]
    fin = np.isfinite(lr)
    assert np.array_equal(np.isfinite(lg), fin)
    assert np.abs(lg[fin] - lr[fin]).max(initial=0.0) <= 1e-3
    mg = f64(mass)
    assert np.abs(f64(rr) - O.recall_rows(mg, rp_r, ci_r)).max() <= 1e-6
    assert np.abs(f64(rh) - O.recall_heads(mg, rp_r, ci_r, N, Cq)).max() <= 1e-6

    # top-k with a random k, on the GPU's masses: exact
    kk = int(rng.integers(1, n_k + 2))
    rp_k, ci_k = L.losa_select_blocks_topk(mass, N, Cq, Ck, kk)
    rpo, cio, _ = O.select_blocks_topk(mg, N, Cq, Ck, kk)
    rpk = rp_k.cpu().numpy().astype(np.int64)
    assert np.array_equal(rpk, rpo)
    assert np.array_equal(ci_k[:rpk[-1]].cpu().numpy().astype(np.int64), cio)

    # construction step
    oc, mc = L.losa_construct(q, k, v, N, Cq, Ck)
    torch.cuda.synchronize()
    od, _ = O.dense_attention(qh, kh, vh, N, scale)
    ok, err = close(f64(oc), od)
    assert ok, (err.max(), err.mean())
    assert np.abs(f64(mc) - m_ref).max() <= 1e-4
