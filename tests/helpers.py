"""Shared plumbing for the GPU parity tests: build a workload on both sides
(liboscar on the GPU, the CPU oracle on the host) from the same seeded inputs,
and compare the results under the parity rules:

  * append: page bytes bit-exact.  A differing byte is tolerated only when its
    row is within 1e-6 of a rounding boundary in the oracle's own arithmetic
    (the fp64 value of (b-a)/3 or -a/s within 1e-6 relative of a binary16
    rounding midpoint, or a code's y/s + z within 1e-6 of k + 0.5); tolerated
    rows are counted and reported.
  * decode: max |o_gpu - o_oracle| <= 2e-3 on the fp32 output (fp32
    accumulation against the fp64 oracle); the bf16 output equals the
    round-to-nearest-even of the same kernel's fp32 output.
"""
from __future__ import annotations

import dataclasses
import math
import sys

import numpy as np
import torch

import oracle
import paper_2605_17757_amd as ok
import workloads as W

DECODE_TOL = 2e-3


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bits(t: torch.Tensor) -> np.ndarray:
    """uint16 numpy view of a bf16 tensor (any device)."""
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


@dataclasses.dataclass
class Case:
    cfg: W.Config
    Rk: np.ndarray
    Rv: np.ndarray
    table: np.ndarray
    num_pages: int
    q: torch.Tensor          # bf16 [B, Hq, d], CPU
    k: torch.Tensor          # bf16 [n_tok, Hkv, d], CPU (all sequences, concatenated)
    v: torch.Tensor
    slots: np.ndarray        # int64 [n_tok]

    @property
    def layout(self):
        return ok.Layout(num_kv_heads=self.cfg.Hkv, num_pages=self.num_pages)


def make_case(cfg: W.Config, compose: bool = False) -> Case:
    Rk, Rv = W.rotations(cfg, compose=compose)
    table, num_pages = W.block_table(cfg)
    ks, vs, sl = [], [], []
    for b in range(cfg.B):
        k, v = W.cache_kv(cfg, b)
        ks.append(k)
        vs.append(v)
        sl.append(W.slots_for(table, b, np.arange(int(cfg.lens[b]))))
    return Case(cfg, Rk, Rv, table, num_pages, W.queries(cfg), torch.cat(ks), torch.cat(vs),
                np.concatenate(sl))


def gpu_append(case: Case, pool: torch.Tensor | None = None, chunk: int = 1 << 20):
    lay = case.layout
    if pool is None:
        pool = ok.alloc_pool(lay)
    Rk = torch.from_numpy(case.Rk).cuda()
    Rv = torch.from_numpy(case.Rv).cuda()
    slots = torch.from_numpy(case.slots).cuda()
    for i in range(0, len(case.slots), chunk):
        ok.kv_append(lay, pool, case.k[i:i + chunk].cuda(), case.v[i:i + chunk].cuda(),
                     slots[i:i + chunk], Rk, Rv, case.cfg.clip_k, case.cfg.clip_v)
    torch.cuda.synchronize()
    return pool


def oracle_append(case: Case) -> np.ndarray:
    pool = np.zeros(ok.pool_bytes(case.layout), np.uint8)
    oracle.kv_append(pool, d=128, Hkv=case.cfg.Hkv, P=64, G=32, k=bits(case.k), v=bits(case.v),
                     slot_mapping=case.slots, Rk=case.Rk, Rv=case.Rv, clip_k=case.cfg.clip_k,
                     clip_v=case.cfg.clip_v)
    return pool


# ---------------------------------------------------------------------------
# append comparison with the near-boundary rule
# ---------------------------------------------------------------------------

def _f16_midpoint_close(x: float, rel: float = 1e-6) -> bool:
    if not math.isfinite(x) or x == 0.0:
        return False
    h = np.float16(x)
    hv = float(h)
    nb = float(np.nextafter(h, np.float16(np.inf if x > hv else -np.inf)))
    mid = 0.5 * (hv + nb)
    return abs(x - mid) <= rel * abs(x)


def _bf16_round(x: float) -> float:
    return float(torch.tensor([x], dtype=torch.float32).to(torch.bfloat16).float()[0])


def _bf16_midpoint_close(x: float, rel: float = 1e-6) -> bool:
    if not math.isfinite(x) or x == 0.0:
        return False
    # the bf16 grid step at |x| is 2^(floor(log2|x|) - 7); a midpoint is an odd
    # multiple of half a step
    e = math.floor(math.log2(abs(x)))
    half = 2.0 ** (e - 8)
    k = abs(x) / half
    return abs(k - (2 * math.floor(k / 2) + 1)) * half <= rel * abs(x)


def row_near_boundary(xt: np.ndarray, rho: float, G: int = 32, meta: int = 0,
                      clip: int = 0) -> bool:
    """True if quantizing this rotated row involves a decision within 1e-6 of a
    rounding boundary (evaluated from the oracle's fp32 row in fp64).  meta, clip:
    the metadata format (0 binary16, 1 bfloat16) and clip rule (0 group absmax,
    1 token quantile)."""
    close = _bf16_midpoint_close if meta else _f16_midpoint_close
    rnd = _bf16_round if meta else (lambda v: float(np.float16(v)))
    tau_tok = np.float32(oracle.token_quantile(xt, rho)) if clip else None
    for g in range(len(xt) // G):
        x = xt[g * G:(g + 1) * G].astype(np.float32)
        if clip:
            tau = tau_tok
        else:
            m = np.float32(np.abs(x).max())
            tau = np.float32(np.float32(rho) * m)
        y = np.minimum(np.maximum(x, -tau), tau)
        a, b = float(y.min()), float(y.max())
        s_exact = (b - a) / 3.0
        if close(s_exact):
            return True
        s16 = rnd(float(np.float32(np.float32(b - a) / np.float32(3.0))))
        if s16 == 0.0:
            continue
        z_exact = -a / s16
        if close(z_exact):
            return True
        z16 = rnd(float(np.float32(-a) / np.float32(s16)))
        u = y.astype(np.float64) / s16 + z16
        if np.any(np.abs(u - (np.floor(u) + 0.5)) <= 1e-6):
            return True
    return False


def compare_pools(gpu_pool: np.ndarray, ora_pool: np.ndarray, case: Case, meta: int = 0,
                  clip: int = 0, G: int = 32):
    """Returns (n_diff_bytes, n_tolerated_rows); raises AssertionError on any
    difference that the near-boundary rule does not cover."""
    diff = np.nonzero(gpu_pool != ora_pool)[0]
    if diff.size == 0:
        return 0, 0
    hkv = case.cfg.Hkv
    szb = (128 // G) * 64 * 4                      # one (s, z) region
    bph = 4096 + 2 * szb
    slot_to_tok = {int(s): i for i, s in enumerate(case.slots)}
    bad_rows = set()
    for off in diff:
        blk, inner = divmod(int(off), bph)
        page, h = divmod(blk, hkv)
        if inner < 2048:
            t, is_v = inner // 32, 0
        elif inner < 4096:
            t, is_v = (inner - 2048) % 64, 1
        elif inner < 4096 + szb:
            t, is_v = ((inner - 4096) // 4) % 64, 0
        else:
            t, is_v = ((inner - 4096 - szb) // 4) % 64, 1
        bad_rows.add((page * 64 + t, h, is_v))
    untolerated = []
    for slot, h, is_v in sorted(bad_rows):
        i = slot_to_tok.get(slot)
        if i is None:
            untolerated.append((slot, h, is_v, "slot not written"))
            continue
        src = case.v if is_v else case.k
        x = W.bf16_bits_to_f32(bits(src[i, h]))
        R = case.Rv if is_v else case.Rk
        if R is not None and np.ndim(R) == 3:  # one rotation per KV head
            R = R[h]
        xt = oracle.rotate_row(x, R)
        if not row_near_boundary(xt, case.cfg.clip_v if is_v else case.cfg.clip_k, G=G,
                                 meta=meta, clip=clip):
            untolerated.append((slot, h, is_v, "not near a rounding boundary"))
    assert not untolerated, "append mismatches: %s (first of %d rows)" % (untolerated[:5],
                                                                           len(untolerated))
    return int(diff.size), len(bad_rows)


# ---------------------------------------------------------------------------
# decode
# ---------------------------------------------------------------------------

def gpu_decode(case: Case, pool: torch.Tensor, num_splits: int, out_dtype=torch.float32,
               table: np.ndarray | None = None, lens: np.ndarray | None = None):
    lay = case.layout
    cfg = case.cfg
    table = case.table if table is None else table
    lens = cfg.lens if lens is None else lens
    if num_splits == 0:
        num_splits = ok.default_num_splits(lay, cfg.B, cfg.Hq, table.shape[1] * 64)
    ws = ok.alloc_workspace(lay, cfg.B, cfg.Hq, num_splits)
    out = torch.empty(cfg.B, cfg.Hq, 128, dtype=out_dtype, device="cuda")
    ok.decode_attn(lay, pool, case.q.cuda(), torch.from_numpy(table).cuda(),
                   torch.from_numpy(np.asarray(lens, np.int32)).cuda(),
                   torch.from_numpy(case.Rk).cuda(), torch.from_numpy(case.Rv).cuda(),
                   cfg.sm_scale, num_splits, ws, out)
    torch.cuda.synchronize()
    return out


def oracle_decode(case: Case, ora_pool: np.ndarray, table=None, lens=None, pairs=None):
    cfg = case.cfg
    return oracle.decode(ora_pool, d=128, Hkv=cfg.Hkv, P=64, G=32, q=bits(case.q),
                         block_table=case.table if table is None else table,
                         seq_lens=cfg.lens if lens is None else np.asarray(lens, np.int32),
                         Rk=case.Rk, Rv=case.Rv, sm_scale=cfg.sm_scale, pairs=pairs)


def max_abs(a, b) -> float:
    a = a.detach().float().cpu().numpy() if isinstance(a, torch.Tensor) else a
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))
