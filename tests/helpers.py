"""Shared plumbing for the GPU parity tests: build a workload on both sides
(liboscar on the GPU, the CPU oracle on the host) from the same seeded inputs,
and compare the results under the parity rules:

  * append: page bytes bit-exact.  Every differing element (code, scale, zero
    point) is tolerated only when its own decision lies within 1e-6 of a
    rounding boundary in the oracle's own arithmetic (the fp64 value of (b-a)/3
    or -a/s within 1e-6 relative of a rounding midpoint of the metadata format,
    or a code's y/s + z within 1e-6 of k + 0.5; the codes of a tolerated (s, z)
    follow it); tolerated elements are counted and reported.
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


def _meta_value(bits16: int, meta: int) -> float:
    """The stored scale or zero point from its 16 bits (binary16 or bfloat16)."""
    if meta:
        return float(np.array([bits16 << 16], np.uint32).view(np.float32)[0])
    return float(np.array([bits16], np.uint16).view(np.float16)[0])


def _row_fields(pool: np.ndarray, base: int, t: int, is_v: int, G: int):
    """Codes [128] and (s, z) bit patterns [d/G, 2] of token slot t of the
    page-head block at byte `base` (the page layout of include/oscar.h)."""
    ng = 128 // G
    if is_v:
        cb = pool[base + 2048 + np.arange(32) * 64 + t]
    else:
        cb = pool[base + t * 32: base + t * 32 + 32]
    codes = ((cb[:, None].astype(np.int32) >> (2 * np.arange(4))) & 3).reshape(128)
    off = base + 4096 + (ng * 64 * 4 if is_v else 0) + (np.arange(ng) * 64 + t) * 4
    e = pool[off[:, None] + np.arange(4)].astype(np.int64)
    sz = np.stack([e[:, 0] | (e[:, 1] << 8), e[:, 2] | (e[:, 3] << 8)], axis=1)
    return codes, sz


def row_tolerated_elements(xt: np.ndarray, rho: float, gpu_codes, gpu_sz, ora_codes, ora_sz,
                           G: int = 32, meta: int = 0, clip: int = 0):
    """Differing elements (codes, scales, zero points) of one quantized row and
    whether each is a near-boundary case in the oracle's own arithmetic (from its
    fp32 rotated row xt, evaluated in fp64): a scale that differs is tolerated
    only if (b - a)/3 lies within 1e-6 relative of a rounding midpoint of the
    metadata format, a zero point (same scale) only if -a/s does; the codes of
    such a group follow from the other (s, z) and are tolerated with it; a code of
    a group whose (s, z) agree only if its y/s + z lies within 1e-6 of k + 0.5.
    Returns (n_differing_elements, n_untolerated)."""
    close = _bf16_midpoint_close if meta else _f16_midpoint_close
    tau_tok = np.float32(oracle.token_quantile(xt, rho)) if clip else None
    n_diff = n_bad = 0
    for g in range(128 // G):
        sl = slice(g * G, (g + 1) * G)
        dc = np.nonzero(gpu_codes[sl] != ora_codes[sl])[0]
        ds, dz = gpu_sz[g, 0] != ora_sz[g, 0], gpu_sz[g, 1] != ora_sz[g, 1]
        n_here = len(dc) + int(ds) + int(dz)
        if n_here == 0:
            continue
        n_diff += n_here
        x = xt[sl].astype(np.float32)
        if clip:
            tau = tau_tok
        else:
            tau = np.float32(np.float32(rho) * np.float32(np.abs(x).max()))
        y = np.minimum(np.maximum(x, -tau), tau)
        a, b = float(y.min()), float(y.max())
        s16 = _meta_value(int(ora_sz[g, 0]), meta)
        if ds or dz:
            ok_group = close((b - a) / 3.0) if ds else (s16 != 0.0 and close(-a / s16))
            if not ok_group:
                n_bad += n_here
            continue
        z16 = _meta_value(int(ora_sz[g, 1]), meta)
        u = y.astype(np.float64) / s16 + z16
        for c in dc:
            if abs(u[c] - (np.floor(u[c]) + 0.5)) > 1e-6:
                n_bad += 1
    return n_diff, n_bad


def compare_pools(gpu_pool: np.ndarray, ora_pool: np.ndarray, case: Case, meta: int = 0,
                  clip: int = 0, G: int = 32):
    """Returns (n_diff_bytes, n_tolerated_elements): every differing code, scale
    or zero point must be a near-boundary case (row_tolerated_elements); raises
    AssertionError on any other difference."""
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
    untolerated, n_tol = [], 0
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
        page, t = divmod(slot, 64)
        base = (page * hkv + h) * bph
        gc, gsz = _row_fields(gpu_pool, base, t, is_v, G)
        oc, osz = _row_fields(ora_pool, base, t, is_v, G)
        n_diff, n_bad = row_tolerated_elements(
            xt, case.cfg.clip_v if is_v else case.cfg.clip_k, gc, gsz, oc, osz, G=G, meta=meta,
            clip=clip)
        if n_bad:
            untolerated.append((slot, h, is_v, "%d of %d differing elements not near a rounding "
                                "boundary" % (n_bad, n_diff)))
        n_tol += n_diff - n_bad
    assert not untolerated, "append mismatches: %s (first of %d rows)" % (untolerated[:5],
                                                                           len(untolerated))
    return int(diff.size), n_tol


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
