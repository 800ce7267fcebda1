"""Seeded synthetic inputs for the OSCAR decode path.

This module only *generates inputs*: queries, new key/value rows, rotation
matrices, sequence lengths, block tables and slot mappings.  It holds none of the
method's arithmetic (no rotation of data, clipping, quantization or attention);
both the GPU library's tests/benchmark and the CPU oracle consume what it makes.

The shapes follow the Qwen3-family attention layers the paper serves (32/8,
64/8 and 96/8 query/KV heads, head dim 128) at the context lengths it
evaluates (up to 32k generated tokens, 128K long-context).  Real activations are
not available; the stand-ins mimic their two salient properties:
  * channel outliers in K/V (a few channels one to two orders of magnitude
    larger than the rest, as in the paper's printed layer-10 token), and
  * a strongly anisotropic query covariance spectrum (the paper's layer-10
    spectrum: top eigenvalue 162.5, geometric-like tail down to 0.009), used to
    build the rotation matrices as eigenvector bases of synthetic covariances.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import torch

HEAD_DIM = 128
PAGE_SIZE = 64
GROUP_SIZE = 32
BASE_SEED = 20260517

# Streams of the per-config seed (seed = BASE_SEED + 1000*config + stream).
S_Q, S_K, S_V, S_RK, S_RV, S_OUTLIER, S_LENS, S_TABLE, S_NEW = 1, 2, 3, 4, 5, 6, 7, 8, 9


@dataclasses.dataclass
class Config:
    """One synthetic workload: a single layer's decode attention."""
    name: str
    index: int
    B: int
    Hq: int
    Hkv: int
    lens: np.ndarray                 # int32 [B], tokens in cache per sequence
    d: int = HEAD_DIM
    P: int = PAGE_SIZE
    G: int = GROUP_SIZE
    clip_k: float = 0.9
    clip_v: float = 0.9
    k_dist: str = "normal"           # "normal" or "student_t3"
    k_outliers: tuple = ()           # channel indices scaled by outlier_scale
    v_outliers: tuple = ()
    outlier_scale: float = 15.0
    spare_tokens: int = PAGE_SIZE    # block-table capacity beyond lens (append room)
    min_splits: int = 0

    @property
    def seed(self) -> int:
        return BASE_SEED + 1000 * self.index

    @property
    def group(self) -> int:
        return self.Hq // self.Hkv

    @property
    def max_pages(self) -> int:
        return int(math.ceil((int(self.lens.max()) + self.spare_tokens) / self.P))

    @property
    def sm_scale(self) -> float:
        return 1.0 / math.sqrt(self.d)


def _rng(seed: int) -> np.random.Generator:
    return np.random.default_rng(seed)


def _outlier_channels(seed: int, n: int, d: int) -> tuple:
    ch = _rng(seed).choice(d, size=n, replace=False)
    return tuple(int(c) for c in sorted(ch))


def config(index: int, batch: int | None = None) -> Config:
    """The workloads (0-4: the five of the hot-path table; 5: one GPU's share of
    workload 3 under 8-way KV-head sharding).  ``batch`` selects batch 1 or 64 for
    config 2."""
    base = BASE_SEED + 1000 * index
    if index == 0:
        # Tiny single layer: 4/1 heads, 256 tokens, K channels 3 and 77 x20.
        return Config("tiny_b1_h4x1_ctx256", 0, 1, 4, 1, np.array([256], np.int32),
                      k_outliers=(3, 77), outlier_scale=20.0)
    if index == 1:
        # Qwen3-4B-shaped layer: 32/8 heads, batch 1, 8192 tokens.
        return Config("qwen3_4b_b1_ctx8192", 1, 1, 32, 8, np.array([8192], np.int32),
                      k_outliers=_outlier_channels(base + S_OUTLIER, 4, HEAD_DIM),
                      v_outliers=_outlier_channels(base + S_OUTLIER + 500, 4, HEAD_DIM))
    if index == 2:
        # Qwen3-8B-shaped layer: 32/8 heads, lengths uniform in [16k, 32k].
        B = 64 if batch is None else int(batch)
        lens = _rng(base + S_LENS).integers(16384, 32768 + 1, size=64).astype(np.int32)[:B]
        if B > 64:
            lens = _rng(base + S_LENS).integers(16384, 32768 + 1, size=B).astype(np.int32)
        return Config("qwen3_8b_b%d_ctx32k" % B, 2, B, 32, 8, lens,
                      k_outliers=_outlier_channels(base + S_OUTLIER, 4, HEAD_DIM),
                      v_outliers=_outlier_channels(base + S_OUTLIER + 500, 4, HEAD_DIM))
    if index == 3:
        # Qwen3-32B-shaped layer: 64/8 heads (GQA 8), batch 128, 32768 tokens.
        B = 128 if batch is None else int(batch)
        return Config("qwen3_32b_b%d_ctx32k" % B, 3, B, 64, 8, np.full(B, 32768, np.int32),
                      k_outliers=_outlier_channels(base + S_OUTLIER, 4, HEAD_DIM),
                      v_outliers=_outlier_channels(base + S_OUTLIER + 500, 4, HEAD_DIM))
    if index == 4:
        # Long context, large GQA: 96/8 heads, batch 16, 131072 tokens,
        # Student-t(3) keys, >= 64 splits per sequence.
        B = 16 if batch is None else int(batch)
        return Config("longctx_b%d_h96x8_ctx128k" % B, 4, B, 96, 8,
                      np.full(B, 131072, np.int32), k_dist="student_t3", min_splits=64)
    if index == 5:
        # One GPU's share of the Qwen3-32B-shaped layer under 8-way KV-head sharding:
        # one KV head and its 8 query heads, batch 128, 32768 tokens.
        B = 128 if batch is None else int(batch)
        return Config("qwen3_32b_tp8_share_b%d_ctx32k" % B, 5, B, 8, 1, np.full(B, 32768, np.int32),
                      k_outliers=_outlier_channels(base + S_OUTLIER, 4, HEAD_DIM),
                      v_outliers=_outlier_channels(base + S_OUTLIER + 500, 4, HEAD_DIM))
    raise ValueError("config index must be 0..5")


def custom(name: str, B: int, Hq: int, Hkv: int, lens, seed_index: int = 90, **kw) -> Config:
    """A free-form workload (fuzz cases, edge cases) with its own seed index."""
    return Config(name, seed_index, B, Hq, Hkv, np.asarray(lens, np.int32).reshape(B), **kw)


# ---------------------------------------------------------------------------
# bf16 packing of generated float32 data (input preparation)
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------------
# Rotation matrices: eigenvector bases of synthetic anisotropic covariances
# ---------------------------------------------------------------------------

def paper_like_spectrum(d: int = HEAD_DIM) -> np.ndarray:
    """Descending spectrum shaped like the paper's layer-10 query covariance:
    geometric from 162.5 down to 0.009 over d eigenvalues."""
    return np.geomspace(162.5, 0.009, d)


def sylvester_hadamard(d: int) -> np.ndarray:
    """Normalized Walsh-Hadamard matrix in natural (Sylvester) order."""
    H = np.ones((1, 1))
    while H.shape[0] < d:
        H = np.block([[H, H], [H, -H]]) / math.sqrt(2.0)
    return H


def bit_reversal_matrix(d: int) -> np.ndarray:
    """Permutation P_br with (P_br)[:, bitrev(k)] = e_k: the k-th channel moves to
    position bitrev(k)."""
    nb = int(math.log2(d))
    P = np.zeros((d, d))
    for k in range(d):
        r = int(format(k, "0%db" % nb)[::-1], 2)
        P[k, r] = 1.0
    return P


def rotation(seed: int, d: int = HEAD_DIM, n_samples: int = 1024, compose: bool = False
             ) -> np.ndarray:
    """fp32 orthogonal matrix: eigenvectors (descending eigenvalue, sign fixed so
    that each column's largest-magnitude entry is positive) of C = X^T X / n,
    X Gaussian with a paper-like spectrum in a random basis.  ``compose`` right-
    multiplies by the Sylvester Hadamard and the bit-reversal permutation."""
    rng = _rng(seed)
    lam = paper_like_spectrum(d)
    basis, _ = np.linalg.qr(rng.standard_normal((d, d)))
    X = rng.standard_normal((n_samples, d)) * np.sqrt(lam)[None, :]
    X = X @ basis.T
    C = X.T @ X / n_samples
    w, U = np.linalg.eigh(C)
    order = np.argsort(w)[::-1]
    U = U[:, order]
    idx = np.argmax(np.abs(U), axis=0)
    U = U * np.sign(U[idx, np.arange(d)])[None, :]
    if compose:
        U = U @ sylvester_hadamard(d) @ bit_reversal_matrix(d)
    return np.ascontiguousarray(U, np.float32)


def rotations(cfg: Config, compose: bool = False):
    return (rotation(cfg.seed + S_RK, cfg.d, compose=compose),
            rotation(cfg.seed + S_RV, cfg.d, compose=compose))


# ---------------------------------------------------------------------------
# Activations (torch, on any device; deterministic per device type)
# ---------------------------------------------------------------------------

def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) & 0x7FFFFFFFFFFFFFFF)
    return g


def _seq_seed(cfg: Config, stream: int, b: int) -> int:
    return (cfg.seed * 1_000_003 + stream * 10_007 + b) & 0x7FFFFFFFFFFF


def queries(cfg: Config, device="cpu") -> torch.Tensor:
    """bf16 [B, Hq, d], N(0, 1)."""
    g = _gen(_seq_seed(cfg, S_Q, 0), device)
    q = torch.randn(cfg.B, cfg.Hq, cfg.d, generator=g, device=device, dtype=torch.float32)
    return q.to(torch.bfloat16)


def _rows(cfg: Config, stream: int, b: int, n: int, device, dist: str, outliers) -> torch.Tensor:
    g = _gen(_seq_seed(cfg, stream, b), device)
    shape = (n, cfg.Hkv, cfg.d)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if dist == "student_t3":
        chi2 = torch.zeros(shape, device=device, dtype=torch.float32)
        for _ in range(3):
            chi2 += torch.randn(shape, generator=g, device=device, dtype=torch.float32) ** 2
        x = x / torch.sqrt(chi2 / 3.0)
    if outliers:
        idx = torch.tensor(list(outliers), device=device)
        x[..., idx] *= cfg.outlier_scale
    return x.to(torch.bfloat16)


def cache_kv(cfg: Config, b: int, device="cpu"):
    """The cached K and V rows of sequence b: bf16 [lens[b], Hkv, d] each."""
    n = int(cfg.lens[b])
    return (_rows(cfg, S_K, b, n, device, cfg.k_dist, cfg.k_outliers),
            _rows(cfg, S_V, b, n, device, "normal", cfg.v_outliers))


def new_kv(cfg: Config, n_per_seq: int, device="cpu"):
    """Fresh rows to append (n_per_seq per sequence): bf16 [B*n_per_seq, Hkv, d]."""
    ks, vs = [], []
    for b in range(cfg.B):
        ks.append(_rows(cfg, S_NEW, b, n_per_seq, device, cfg.k_dist, cfg.k_outliers))
        vs.append(_rows(cfg, S_NEW + 50, b, n_per_seq, device, "normal", cfg.v_outliers))
    return torch.cat(ks), torch.cat(vs)


# ---------------------------------------------------------------------------
# Paging
# ---------------------------------------------------------------------------

def block_table(cfg: Config):
    """Shuffled, non-contiguous page assignment.  Returns (table int32
    [B, max_pages], num_pages).  Every sequence owns max_pages distinct pages of
    a pool of B*max_pages, dealt out from a seeded permutation."""
    mp = cfg.max_pages
    num_pages = cfg.B * mp
    perm = _rng(cfg.seed + S_TABLE).permutation(num_pages).astype(np.int32)
    return perm.reshape(cfg.B, mp), num_pages


def slots_for(table: np.ndarray, b: int, positions, P: int = PAGE_SIZE) -> np.ndarray:
    """slot = page * P + offset for token positions of sequence b."""
    pos = np.asarray(positions, np.int64)
    return table[b, pos // P].astype(np.int64) * P + pos % P


# ---------------------------------------------------------------------------
# Calibration activations (one layer's Q, K, V dump)
# ---------------------------------------------------------------------------

CALIB_TOKENS = 8878  # the paper's calibration pass length per layer


def calib_activations(T: int, Hq: int, Hkv: int, seed: int, d: int = HEAD_DIM,
                      device="cpu"):
    """Synthetic calibration activations, bf16 [T, Hq, d] and [T, Hkv, d] x 2.
    Queries: Gaussian with covariance B diag(lambda) B^T, lambda the paper-like
    descending spectrum (162.5 .. 0.009) and B a seeded random orthogonal basis
    shared by all heads.  Keys: Gaussian with four outlier channels scaled by 15
    and a common offset of 0.5 on eight channels (keys carry a mean).  Values:
    standard Gaussian with two channels scaled by 4."""
    rng = _rng(seed)
    basis, _ = np.linalg.qr(rng.standard_normal((d, d)))
    lam = paper_like_spectrum(d)
    mix = torch.from_numpy((np.sqrt(lam)[:, None] * basis.T).astype(np.float32)).to(device)
    k_out = torch.tensor(sorted(rng.choice(d, 4, replace=False).tolist()), device=device)
    k_mean = torch.tensor(sorted(rng.choice(d, 8, replace=False).tolist()), device=device)
    v_out = torch.tensor(sorted(rng.choice(d, 2, replace=False).tolist()), device=device)
    g = _gen(seed * 7 + 1, device)
    z = torch.randn(T * Hq, d, generator=g, device=device, dtype=torch.float32)
    q = (z @ mix).reshape(T, Hq, d)
    k = torch.randn(T, Hkv, d, generator=g, device=device, dtype=torch.float32)
    k[..., k_out] *= 15.0
    k[..., k_mean] += 0.5
    v = torch.randn(T, Hkv, d, generator=g, device=device, dtype=torch.float32)
    v[..., v_out] *= 4.0
    return q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)
