"""Seeded synthetic Q/K/V with the shapes and locality of video-DiT self-attention.

The paper measures real video latents (Wan2.1, CogVideoX-style and HunyuanVideo
transformers); neither the models nor the prompts are available, so these
seeded tensors stand in for them.  The module holds no part of the attention
method itself: it only draws inputs.  Both the HIP path's tests/benchmark and
the CPU oracle consume exactly the tensors produced here.

Construction (frozen constants):

* Tokens form a T x Hg x Wg grid flattened frame-major, n = (t*Hg + h)*Wg + w.
* phi(n) in R^96 = [sin(w_f x), cos(w_f x)] for x in (t, h, w), f = 0..15,
  with w_f = 10000^(-f/16).
* One seeded projection W in R^(96 x d), entries N(0, PROJ_STD^2), shared by
  Q, K and all heads; E = phi W.
* Q_h = noise * Z_q + alpha_h * E,  K_h = noise * Z_k + alpha_h * E,
  V ~ N(0, 1); Z iid N(0, 1), independent per tensor and head.
* Padding rows n >= N are zero.  Tensors are drawn in fp32 and cast once
  (round-to-nearest-even) to the workload dtype.
* Reuse-step drift: X_t = X_{t-1} + sigma * Z_t for X in (Q, K, V), padding
  rows re-zeroed, then cast.
* Seeds: one base seed per workload; sub-seeds base+1 (W), base+2 (alpha),
  base+3 (Z_q), base+4 (Z_k), base+5 (V), base+100+t (drift of step t).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace

import torch

N_FREQ = 16
# 1.7 / sqrt(96): chosen once so that the Wan-shaped workload keeps ~60 % of its
# blocks at tau = 0.99 (about 40 % dropped); 1 / sqrt(96) kept ~95 %.
PROJ_STD = 1.7 / math.sqrt(96.0)


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    d: int
    dtype: str            # "f32" or "bf16"
    grid: tuple           # (T, Hg, Wg)
    block: int            # square blocks: query block R = key block C
    tau: float
    alpha: object         # float, or ("uniform", lo, hi) drawn per head
    noise: float
    sigma: float          # per-step drift std
    reuse: int            # reuse steps after the calibration step
    seed: int
    block_k: int = 0      # key block C when it differs from the query block (0: C = R)

    @property
    def N(self) -> int:
        T, Hg, Wg = self.grid
        return T * Hg * Wg

    @property
    def N_pad(self) -> int:
        return -(-self.N // self.block) * self.block

    @property
    def n_blocks(self) -> int:
        """Query blocks per head (n_q)."""
        return self.N_pad // self.block

    @property
    def bk(self) -> int:
        """Key block size C."""
        return self.block_k or self.block

    @property
    def n_kblocks(self) -> int:
        """Key blocks per head (n_k)."""
        return self.N_pad // self.bk

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)


WORKLOADS = {
    "tiny": Workload("tiny", B=1, H=2, d=64, dtype="f32", grid=(4, 16, 16), block=64,
                     tau=0.99, alpha=1.5, noise=0.5, sigma=0.05, reuse=3, seed=0),
    "wan": Workload("wan2.1-1.3b", B=1, H=12, d=128, dtype="bf16", grid=(21, 30, 52),
                    block=128, tau=0.99, alpha=1.5, noise=0.5, sigma=0.02, reuse=49,
                    seed=1000),
    "cog": Workload("cogvideox-5b", B=1, H=48, d=64, dtype="bf16", grid=(13, 30, 45),
                    block=128, tau=0.99, alpha=("uniform", 0.8, 2.0), noise=0.5,
                    sigma=0.02, reuse=49, seed=2000),
    "hunyuan": Workload("hunyuanvideo", B=1, H=24, d=128, dtype="bf16", grid=(33, 45, 80),
                        block=128, tau=0.99, alpha=1.5, noise=0.5, sigma=0.02, reuse=49,
                        seed=3000),
}

SWEEP_TAUS = (0.95, 0.99, 0.999, 1.0)
SWEEP_ALPHAS = (0.5, 1.5, 3.0)


def sweep_points():
    """Density sweep at the Wan shape: tau x locality weight."""
    base = replace(WORKLOADS["wan"], name="density-sweep", seed=4000, reuse=1)
    return [replace(base, tau=t, alpha=a, name=f"sweep-tau{t}-alpha{a}")
            for a in SWEEP_ALPHAS for t in SWEEP_TAUS]


def scaled(w: Workload, grid=None, H=None, B=None, name=None, block_k=None) -> Workload:
    """The same construction at a smaller grid / head count (parity cases)."""
    return replace(w, grid=grid or w.grid, H=H or w.H, B=B or w.B, name=name or w.name,
                   block_k=w.block_k if block_k is None else block_k)


def rectangular(w: Workload, block_k: int = 32) -> Workload:
    """The same inputs with the paper's rectangular blocks: query blocks of
    w.block rows, key blocks of block_k keys (Sec. 5.1 uses 128 x 32)."""
    return replace(w, block_k=block_k, name=f"{w.name}-c{block_k}")


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def positional_features(grid, device="cpu") -> torch.Tensor:
    """phi(n) for every grid token, frame-major order: [N, 96] fp32."""
    T, Hg, Wg = grid
    t = torch.arange(T, device=device, dtype=torch.float64)
    h = torch.arange(Hg, device=device, dtype=torch.float64)
    w = torch.arange(Wg, device=device, dtype=torch.float64)
    tt, hh, ww = torch.meshgrid(t, h, w, indexing="ij")
    coords = [tt.reshape(-1), hh.reshape(-1), ww.reshape(-1)]
    freqs = 10000.0 ** (-torch.arange(N_FREQ, device=device, dtype=torch.float64) / N_FREQ)
    feats = []
    for x in coords:
        ang = x[:, None] * freqs[None, :]
        feats.append(torch.sin(ang))
        feats.append(torch.cos(ang))
    return torch.cat(feats, dim=1).to(torch.float32)


def head_alphas(w: Workload, device="cpu") -> torch.Tensor:
    if isinstance(w.alpha, tuple):
        _, lo, hi = w.alpha
        u = torch.rand(w.H, generator=_gen("cpu", w.seed + 2), dtype=torch.float64)
        return (lo + (hi - lo) * u).to(torch.float32).to(device)
    return torch.full((w.H,), float(w.alpha), dtype=torch.float32, device=device)


def make_state(w: Workload, device="cpu"):
    """fp32 master tensors (Q, K, V), each [B, H, N_pad, d], padding rows zero."""
    N, Np, d = w.N, w.N_pad, w.d
    phi = positional_features(w.grid, device)
    W = torch.randn(96, d, generator=_gen(device, w.seed + 1), device=device) * PROJ_STD
    E = phi @ W                                                   # [N, d]
    alpha = head_alphas(w, device)                                # [H]
    shape = (w.B, w.H, Np, d)
    out = []
    for sub in (3, 4):
        Z = torch.randn(shape, generator=_gen(device, w.seed + sub), device=device)
        X = w.noise * Z
        X[:, :, :N] += alpha[None, :, None, None] * E[None, None]
        X[:, :, N:] = 0
        out.append(X)
    V = torch.randn(shape, generator=_gen(device, w.seed + 5), device=device)
    V[:, :, N:] = 0
    out.append(V)
    return tuple(out)


def drift_(state, w: Workload, step: int):
    """In-place reuse-step drift of the fp32 master tensors."""
    g = _gen(state[0].device, w.seed + 100 + step)
    for X in state:
        X.add_(torch.randn(X.shape, generator=g, device=X.device), alpha=w.sigma)
        X[:, :, w.N:] = 0
    return state


def cast(state, w: Workload):
    """Cast the master tensors once to the workload dtype (contiguous)."""
    return tuple(X.to(w.torch_dtype).contiguous() for X in state)


def make_inputs(w: Workload, device="cpu"):
    """Calibration-step inputs (Q, K, V) in the workload dtype."""
    return cast(make_state(w, device), w)
