"""oscar_decode_attn_noalloc (the decode entry point that allocates nothing and
uses the library's per-GPU scratch array) against oscar_decode_attn with a
caller workspace: the same output bit for bit, and within the decode tolerance
of the oracle, on two calls in a row, the second with a smaller input (fewer
sequences, heads and pages, so that it reads scratch entries the first call
left behind only if it failed to write them)."""
import numpy as np
import pytest
import torch

import paper_2605_17757_amd as ok
import workloads as W
from helpers import (DECODE_TOL, gpu_append, gpu_decode, log, make_case, max_abs,
                     oracle_append, oracle_decode)

pytestmark = pytest.mark.gpu


def _noalloc(case, pool, num_splits, out_dtype=torch.float32):
    cfg = case.cfg
    out = torch.full((cfg.B, cfg.Hq, 128), float("nan"), dtype=out_dtype, device="cuda")
    ok.decode_attn_noalloc(case.layout, pool, case.q.cuda(), torch.from_numpy(case.table).cuda(),
                           torch.from_numpy(cfg.lens).cuda(), torch.from_numpy(case.Rk).cuda(),
                           torch.from_numpy(case.Rv).cuda(), cfg.sm_scale, num_splits, out)
    torch.cuda.synchronize()
    return out


def _check(case, num_splits):
    log("no-alloc case", case.cfg.name, "B", case.cfg.B, "Hq", case.cfg.Hq, "Hkv", case.cfg.Hkv,
        "lens", list(case.cfg.lens), "splits", num_splits)
    pool = gpu_append(case)
    ref = gpu_decode(case, pool, num_splits)
    got = _noalloc(case, pool, num_splits)
    assert torch.equal(got, ref), "no-alloc output differs from oscar_decode_attn"
    err = max_abs(got, oracle_decode(case, oracle_append(case)))
    log("  max|err| vs oracle = %.3g" % err)
    assert err <= DECODE_TOL
    gotb = _noalloc(case, pool, num_splits, out_dtype=torch.bfloat16)
    assert torch.equal(gotb.cpu(), ref.cpu().to(torch.bfloat16))


def test_noalloc_matches_workspace_entry_point_two_calls():
    big = W.custom("noalloc_big", 3, 32, 8, [8192, 700, 65], seed_index=71,
                   k_outliers=(5, 77), v_outliers=(9,))
    _check(make_case(big), 0)
    small = W.custom("noalloc_small", 2, 8, 2, [129, 1], seed_index=72)
    _check(make_case(small), 3)


def test_noalloc_wide_instances():
    """8, 12 and 16 query heads per KV head (the wide split instances), after each other."""
    for g, seed in ((8, 73), (12, 74), (16, 97)):
        case = make_case(W.custom("noalloc_g%d" % g, 3, 2 * g, 2, [1500, 64, 333], seed_index=seed,
                                  k_outliers=(3, 40)))
        _check(case, 4)


def test_noalloc_rejects_oversized_workspace():
    lay = ok.Layout(num_kv_heads=8, num_pages=1)
    B, Hq, S = 512, 64, 64
    assert ok.decode_workspace_bytes(lay, B, Hq, S) > ok.NOALLOC_SCRATCH_BYTES
    q = torch.zeros(B, Hq, 128, dtype=torch.bfloat16, device="cuda")
    bt = torch.zeros(B, 1, dtype=torch.int32, device="cuda")
    sl = torch.ones(B, dtype=torch.int32, device="cuda")
    out = torch.empty(B, Hq, 128, dtype=torch.float32, device="cuda")
    pool = ok.alloc_pool(lay)
    with pytest.raises(ok.OscarError) as e:
        ok.decode_attn_noalloc(lay, pool, q, bt, sl, None, None, 0.088, S, out)
    assert e.value.status == ok.ERR_WORKSPACE_TOO_SMALL
