"""Workload definitions and seeded generators.

Recipe (all tensors drawn in fp32, then rounded once to bf16, nearest-even):

* Weights W [out, in]:
  - "normal": N(0, std^2) entries;
  - "student_t": t(df) entries built as z / sqrt(chi2_df / df) with chi2_df a
    sum of df squared standard normals, then scaled to the stated std by
    std / sqrt(df / (df - 2));
  - optional outliers: round(p * out * in) positions drawn without
    replacement and multiplied by a factor.
* Activations X [tokens, in]: column j has std sigma_j = exp(N(0, s^2))
  (log-normal(0, s)); a few outlier channels, drawn without replacement,
  multiply sigma_j by a factor; x_tj = sigma_j * z_tj with z ~ N(0, 1).
* Global scale (a caller input of the search): the harness convention
  s_g = fp32(fp32(max |W|) / 2688), 2688 = 6 * 448, which maps the tensor's
  largest magnitude onto the largest E2M1 value times the largest E4M3 value.

Generation uses a torch.Generator on the requested device (CPU for the small
cases and the CPU tests, the GPU for the large tensors), seeded per tensor,
so a workload is reproducible on a given device.  Large activations are
generated in row chunks to bound the fp32 staging memory.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

_SEED_W = 1
_SEED_X = 2
_SEED_W_OUT = 3
_SEED_X_SIGMA = 4
_SEED_X_OUT = 5


@dataclass(frozen=True)
class Workload:
    name: str
    out: int
    inp: int
    tokens: int
    w_dist: str  # "normal" | "student_t"
    w_std: float
    w_df: int = 0
    w_outlier_frac: float = 0.0
    w_outlier_mult: float = 1.0
    x_log_sigma: float = 0.5
    x_outlier_channels: int = 0
    x_outlier_mult: float = 1.0
    window: int = 4
    seed: int = 0
    note: str = ""

    @property
    def weights(self) -> int:
        return self.out * self.inp

    @property
    def groups(self) -> int:
        return self.out * self.inp // 16


CONFIGS: dict[str, Workload] = {
    # 256x512 weights and 128x512 activations: small enough for the oracle to
    # finish in well under a second; spans several tiles of both kernels.
    "tiny": Workload("tiny", 256, 512, 128, "normal", 0.02,
                     w_outlier_frac=0.005, w_outlier_mult=10.0,
                     x_log_sigma=0.5, x_outlier_channels=4, x_outlier_mult=30.0,
                     window=4, seed=0),
    # A single 8B-class attention projection (q or o), 128 sequences x 2048.
    "attn_proj": Workload("attn_proj", 4096, 4096, 262144, "normal", 0.02,
                          w_outlier_frac=0.001, w_outlier_mult=8.0,
                          x_log_sigma=0.5, x_outlier_channels=8, x_outlier_mult=50.0,
                          window=4, seed=1,
                          note="log-normal spread of the channel std read as s=0.5"),
    # Llama-3-8B-shaped MLP down_proj (the headline workload).
    "down_proj": Workload("down_proj", 4096, 14336, 262144, "student_t", 0.015, w_df=4,
                          x_log_sigma=0.7, x_outlier_channels=16, x_outlier_mult=50.0,
                          window=4, seed=2,
                          note="'sparse outlier channels' read as 16 channels x50"),
    # 70B-class down_proj, heavy-tailed weights, window +-8.
    "down_proj_70b": Workload("down_proj_70b", 8192, 28672, 131072, "student_t", 0.01, w_df=3,
                              x_log_sigma=1.0, x_outlier_channels=16, x_outlier_mult=100.0,
                              window=8, seed=4),
}

# Full 8B-class decoder block: (name, out, in, activation tensor, weight kind).
BLOCK_LAYERS = [
    ("q_proj", 4096, 4096, "attn", "normal"),
    ("k_proj", 1024, 4096, "attn", "normal"),
    ("v_proj", 1024, 4096, "attn", "normal"),
    ("o_proj", 4096, 4096, "attn", "normal"),
    ("gate_proj", 14336, 4096, "mlp", "normal"),
    ("up_proj", 14336, 4096, "mlp", "normal"),
    ("down_proj", 4096, 14336, "down", "student_t"),
]


def block_workloads(window: int = 4, seed: int = 3) -> dict[str, Workload]:
    """Per-layer workloads of the decoder-block config.  Three shared
    calibration tensors of 262144 tokens: X_attn (q, k, v and o; o reuses it),
    X_mlp (gate, up) and X_down (down)."""
    out = {}
    for k, (name, m, n, xname, kind) in enumerate(BLOCK_LAYERS):
        if kind == "normal":
            wl = Workload(name, m, n, 262144, "normal", 0.02,
                          w_outlier_frac=0.001, w_outlier_mult=8.0,
                          x_log_sigma=0.5, x_outlier_channels=8, x_outlier_mult=50.0,
                          window=window, seed=seed * 100 + k)
        else:
            wl = Workload(name, m, n, 262144, "student_t", 0.015, w_df=4,
                          x_log_sigma=0.7, x_outlier_channels=16, x_outlier_mult=50.0,
                          window=window, seed=seed * 100 + k)
        out[name] = wl
    return out


def _gen(seed: int, salt: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000003 + salt)
    return g


def make_weight(wl: Workload, device="cpu", shape=None):
    """Weight tensor W [out, in] in bf16 on ``device``."""
    import torch
    m, n = shape if shape is not None else (wl.out, wl.inp)
    g = _gen(wl.seed, _SEED_W, device)
    if wl.w_dist == "normal":
        w = torch.randn((m, n), generator=g, device=device, dtype=torch.float32)
        w.mul_(wl.w_std)
    elif wl.w_dist == "student_t":
        df = int(wl.w_df)
        z = torch.randn((m, n), generator=g, device=device, dtype=torch.float32)
        chi2 = torch.zeros((m, n), device=device, dtype=torch.float32)
        for _ in range(df):
            e = torch.randn((m, n), generator=g, device=device, dtype=torch.float32)
            chi2.addcmul_(e, e)
            del e
        w = z.div_(chi2.div_(df).sqrt_())
        del chi2
        w.mul_(wl.w_std / float(np.sqrt(df / (df - 2.0))))
    else:
        raise ValueError(wl.w_dist)
    if wl.w_outlier_frac > 0:
        k = int(round(wl.w_outlier_frac * m * n))
        go = _gen(wl.seed, _SEED_W_OUT, device)
        idx = torch.randperm(m * n, generator=go, device=device)[:k]
        w.view(-1)[idx] *= wl.w_outlier_mult
    return w.to(torch.bfloat16)


def channel_sigma(wl: Workload, device="cpu", n=None):
    """Per-channel std of the activations (fp32 [in])."""
    import torch
    n = wl.inp if n is None else n
    g = _gen(wl.seed, _SEED_X_SIGMA, device)
    sigma = torch.randn((n,), generator=g, device=device, dtype=torch.float32)
    sigma = torch.exp(sigma * wl.x_log_sigma)
    if wl.x_outlier_channels > 0:
        go = _gen(wl.seed, _SEED_X_OUT, device)
        idx = torch.randperm(n, generator=go, device=device)[: wl.x_outlier_channels]
        sigma[idx] *= wl.x_outlier_mult
    return sigma


def make_activations(wl: Workload, device="cpu", tokens=None, n=None,
                     chunk_elems: int = 1 << 28):
    """Calibration activations X [tokens, in] in bf16 on ``device``."""
    import torch
    T = wl.tokens if tokens is None else tokens
    n = wl.inp if n is None else n
    sigma = channel_sigma(wl, device, n)
    X = torch.empty((T, n), device=device, dtype=torch.bfloat16)
    g = _gen(wl.seed, _SEED_X, device)
    rows = max(1, chunk_elems // max(n, 1))
    for t0 in range(0, T, rows):
        t1 = min(T, t0 + rows)
        z = torch.randn((t1 - t0, n), generator=g, device=device, dtype=torch.float32)
        z.mul_(sigma)
        X[t0:t1].copy_(z)
        del z
    return X


def harness_global_scale(W) -> float:
    """s_g = fp32(fp32(max|W|) / 2688) as a Python float (exactly an fp32)."""
    import torch
    amax = W.detach().abs().max().float().cpu().item()
    return float(np.float32(amax) / np.float32(2688.0))


def bf16_bits_to_float(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 patterns -> float32 values (exact)."""
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


def tensor_bits(t) -> np.ndarray:
    """A bf16 torch tensor's bit patterns as a host uint16 array."""
    import torch
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)
