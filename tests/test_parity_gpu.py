"""GPU parity of liboscar against the CPU oracle (same seeded inputs, every
output element compared).  Sizes are chosen so the oracle finishes in seconds
while spanning many 64-token pages, several splits and ragged tails."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2605_17757_amd as ok
import workloads as W
from helpers import (DECODE_TOL, Case, bits, compare_pools, gpu_append, gpu_decode, log,
                     make_case, max_abs, oracle_append, oracle_decode)

pytestmark = pytest.mark.gpu


def _run_full(case: Case, num_splits: int = 0, check_bf16: bool = True):
    log("case", case.cfg.name, "B", case.cfg.B, "Hq", case.cfg.Hq, "Hkv", case.cfg.Hkv,
        "lens", list(case.cfg.lens[:4]), "splits", num_splits)
    pool = gpu_append(case)
    ora = oracle_append(case)
    nd, nt = compare_pools(pool.cpu().numpy(), ora, case)
    log("  append: differing bytes", nd, "tolerated near-boundary elements", nt)
    ref = oracle_decode(case, ora)
    out = gpu_decode(case, pool, num_splits)
    err = max_abs(out, ref)
    log("  decode max|err| = %.3g" % err)
    assert err <= DECODE_TOL
    if check_bf16:
        outb = gpu_decode(case, pool, num_splits, out_dtype=torch.bfloat16)
        assert torch.equal(outb.cpu(), out.cpu().to(torch.bfloat16))
    return pool, ora, out


def test_config0_tiny():
    _run_full(make_case(W.config(0)))


def test_config1_qwen3_4b_shape():
    _run_full(make_case(W.config(1)))


def test_config2_qwen3_8b_batch1():
    _run_full(make_case(W.config(2, batch=1)))


def test_config3_shape_reduced_batch_and_length():
    # Qwen3-32B heads (64/8, GQA 8) at batch 3 and 2k-4k tokens
    cfg = W.config(3, batch=3)
    cfg.lens = np.array([4096, 2049, 3007], np.int32)
    _run_full(make_case(cfg))


def test_config5_tp8_share_single_kv_head():
    # one GPU's share of the Qwen3-32B heads under 8-way KV-head sharding: one KV
    # head and its 8 query heads, at batch 5 and ragged 1k-4k tokens
    cfg = W.config(5, batch=5)
    cfg.lens = np.array([4096, 1, 2049, 1000, 3007], np.int32)
    _run_full(make_case(cfg))
    _run_full(make_case(cfg), num_splits=7)


def test_config4_shape_student_t_many_splits():
    # 96/8 heads (GQA 12), Student-t keys, distinct rotations, >= 64 splits
    cfg = W.config(4, batch=2)
    cfg.lens = np.array([8192, 5000], np.int32)
    _run_full(make_case(cfg), num_splits=64)


def test_composed_rotation_hadamard_bitreversal():
    cfg = W.config(1)
    cfg.lens = np.array([3000], np.int32)
    _run_full(make_case(cfg, compose=True))


@pytest.mark.parametrize("g", list(range(1, 17)))
def test_gqa_ratios_and_ragged_lengths(g):
    """Every ratio of query to KV heads up to 16: the int8 instance (1-4), and the
    wide ones at 5-8, 9-12 and 13-16 query heads, whose padding heads (every ratio
    that is not a multiple of 4) take part in the MFMA tiles and are never stored."""
    Hkv = 2
    lens = [1, 63, 64, 65, 129, 700]
    cfg = W.custom("gqa%d" % g, len(lens), g * Hkv, Hkv, lens, seed_index=70 + g,
                   k_outliers=(5, 90), v_outliers=(17,))
    _run_full(make_case(cfg), num_splits=3)


@pytest.mark.parametrize("g", [4, 8, 12])
@pytest.mark.parametrize("num_splits", [1, 3])
def test_zero_length_sequences(g, num_splits):
    """Sequences of length 0 between live ones (a length-0 sequence decodes to a zero
    row): their rows are exactly zero and every other row matches the oracle, in the
    int8 instance (4 query heads per KV head) and the wide ones (8, 12)."""
    Hkv = 2
    lens = np.array([0, 130, 0, 700, 64, 0], np.int32)
    cfg = W.custom("zero_len_g%d" % g, len(lens), g * Hkv, Hkv, lens, seed_index=230 + g)
    case = make_case(cfg)
    log("case", cfg.name, "lens", list(lens), "splits", num_splits)
    pool = gpu_append(case)
    ora = oracle_append(case)
    compare_pools(pool.cpu().numpy(), ora, case)
    live = np.nonzero(lens > 0)[0]
    pairs = np.array([(b, h) for b in live for h in range(cfg.Hq)], np.int32)
    ref = oracle_decode(case, ora, pairs=pairs)
    out = gpu_decode(case, pool, num_splits).cpu().numpy()
    err = max_abs(out[live].reshape(-1, 128), ref)
    log("  decode max|err| = %.3g" % err)
    assert err <= DECODE_TOL
    assert np.all(out[lens == 0] == 0.0)


def test_lengths_outside_the_table_are_clamped(monkeypatch):
    """Without the debug checks a length is clamped to [0, the block-table row's
    capacity]: past the capacity the output equals the one at the capacity, bit for
    bit, and a negative length decodes to a zero row."""
    monkeypatch.delenv("OSCAR_DEBUG", raising=False)
    cfg = W.custom("clamp", 3, 8, 2, [256, 300, 128], seed_index=240)
    case = make_case(cfg)
    pool = gpu_append(case)
    cap = case.table.shape[1] * 64
    for S in (1, 3):
        at_cap = gpu_decode(case, pool, S, lens=np.array([cap, cap, 0], np.int32))
        past = gpu_decode(case, pool, S, lens=np.array([cap + 50, cap + 100000, -5], np.int32))
        assert torch.equal(at_cap, past)
        assert bool((past[2] == 0.0).all())


def test_split_count_invariance():
    cfg = W.config(1)
    cfg.lens = np.array([5000], np.int32)
    case = make_case(cfg)
    pool = gpu_append(case)
    ref = oracle_decode(case, oracle_append(case))
    outs = []
    for S in (1, 2, 3, 7, 20, 64, 79, 256):
        out = gpu_decode(case, pool, S)
        err = max_abs(out, ref)
        log("splits", S, "max|err| %.3g" % err)
        assert err <= DECODE_TOL
        outs.append(out.cpu())
    # the per-page 15-bit scaling of p*s_v depends on the running max, which
    # depends on the split boundaries: different split counts agree to ~1e-4
    for o in outs[1:]:
        assert max_abs(o, outs[0].numpy()) <= 5e-4


def test_page_shuffle_invariance():
    cfg = W.custom("shuffle", 2, 8, 2, [900, 333], seed_index=81)
    case = make_case(cfg)
    pool = gpu_append(case)
    out = gpu_decode(case, pool, 4)
    # move every page to a new position and remap the block table
    bph = ok.page_bytes(case.layout)
    perm = np.random.default_rng(5).permutation(case.num_pages)
    moved = torch.empty_like(pool)
    pv = pool.view(case.num_pages, bph)
    mv = moved.view(case.num_pages, bph)
    mv[torch.from_numpy(perm).cuda()] = pv
    out2 = gpu_decode(case, moved, 4, table=perm[case.table].astype(np.int32))
    assert torch.equal(out.cpu(), out2.cpu())


def test_decode_stages_equal_single_call():
    cfg = W.custom("stages", 3, 16, 4, [300, 64, 1000], seed_index=82)
    case = make_case(cfg)
    pool = gpu_append(case)
    lay = case.layout
    S = 5
    ws = ok.alloc_workspace(lay, cfg.B, cfg.Hq, S)
    out_a = gpu_decode(case, pool, S)
    out_b = torch.empty_like(out_a)
    q = case.q.cuda()
    bt = torch.from_numpy(case.table).cuda()
    sl = torch.from_numpy(cfg.lens).cuda()
    Rk = torch.from_numpy(case.Rk).cuda()
    Rv = torch.from_numpy(case.Rv).cuda()
    ok.decode_prepare(lay, q, Rk, cfg.sm_scale, S, ws)
    ok.decode_split(lay, pool, cfg.B, cfg.Hq, bt, sl, S, ws)
    ok.decode_reduce(lay, cfg.B, cfg.Hq, Rv, S, ws, out_b)
    torch.cuda.synchronize()
    assert torch.equal(out_a.cpu(), out_b.cpu())


def test_decode_step_equals_append_then_attn():
    """oscar_decode_step (cache update and query rotation in one launch, then
    split and reduce) writes the same page bytes and returns the same output,
    bit for bit, as oscar_kv_append followed by oscar_decode_attn; with no new
    token it equals oscar_decode_attn."""
    cfg = W.custom("step", 3, 16, 4, [300, 64, 1000], seed_index=83)
    case = make_case(cfg)
    lay = case.layout
    last = np.cumsum(cfg.lens) - 1                    # each sequence's newest token
    prev = np.setdiff1d(np.arange(len(case.slots)), last)
    Rk = torch.from_numpy(case.Rk).cuda()
    Rv = torch.from_numpy(case.Rv).cuda()
    pool = ok.alloc_pool(lay)
    ok.kv_append(lay, pool, case.k[prev].cuda(), case.v[prev].cuda(),
                 torch.from_numpy(case.slots[prev]).cuda(), Rk, Rv, cfg.clip_k, cfg.clip_v)
    new_k, new_v = case.k[last].cuda(), case.v[last].cuda()
    new_s = torch.from_numpy(case.slots[last]).cuda()
    q = case.q.cuda()
    bt = torch.from_numpy(case.table).cuda()
    sl = torch.from_numpy(cfg.lens).cuda()
    S = 6
    pool_a, pool_b = pool.clone(), pool.clone()
    out_a = torch.empty(cfg.B, cfg.Hq, 128, dtype=torch.float32, device="cuda")
    out_b = torch.empty_like(out_a)
    ws_a = ok.alloc_workspace(lay, cfg.B, cfg.Hq, S)
    ws_b = ok.alloc_workspace(lay, cfg.B, cfg.Hq, S)
    ok.kv_append(lay, pool_a, new_k, new_v, new_s, Rk, Rv, cfg.clip_k, cfg.clip_v)
    ok.decode_attn(lay, pool_a, q, bt, sl, Rk, Rv, cfg.sm_scale, S, ws_a, out_a)
    ok.decode_step(lay, pool_b, new_k, new_v, new_s, cfg.clip_k, cfg.clip_v, q, bt, sl, Rk, Rv,
                   cfg.sm_scale, S, ws_b, out_b)
    torch.cuda.synchronize()
    assert torch.equal(pool_a, pool_b)
    assert torch.equal(out_a, out_b)
    ref = oracle_decode(case, oracle_append(case))
    assert max_abs(out_b, ref) <= DECODE_TOL
    # no new token: the step is the decode alone
    out_c = torch.empty_like(out_a)
    empty = torch.empty(0, dtype=torch.int64, device="cuda")
    ok.decode_step(lay, pool_b, None, None, empty, cfg.clip_k, cfg.clip_v, q, bt, sl, Rk, Rv,
                   cfg.sm_scale, S, ws_b, out_c)
    torch.cuda.synchronize()
    assert torch.equal(out_a, out_c)


def test_append_fuzz_edge_rows():
    rng = np.random.default_rng(11)
    Hkv, num_pages = 3, 40
    cfg = W.custom("fuzz", 1, 3, Hkv, [1], seed_index=83, clip_k=0.5, clip_v=1.0)
    n_tok = 777
    slots = rng.permutation(num_pages * 64)[:n_tok].astype(np.int64)
    x = rng.standard_normal((2, n_tok, Hkv, 128)).astype(np.float32)
    x[:, :50] = 0.0                                      # all-zero rows (degenerate groups)
    x[:, 50:100] = 3.25                                  # constant rows
    x[:, 100:150] *= 1e4                                 # large magnitudes
    x[:, 150:200] *= 1e-6                                # tiny magnitudes
    df = 3.0
    x[:, 200:400] = rng.standard_t(df, size=(2, 200, Hkv, 128))
    x[:, 400:420, :, :40] = 0.0                          # partly zero rows
    k = torch.from_numpy(W.f32_to_bf16_bits(x[0]).view(np.int16)).view(torch.bfloat16)
    v = torch.from_numpy(W.f32_to_bf16_bits(x[1]).view(np.int16)).view(torch.bfloat16)
    for compose in (False, True):
        Rk = W.rotation(901, compose=compose)
        Rv = W.rotation(902, compose=compose)
        case = Case(cfg, Rk, Rv, np.zeros((1, 1), np.int32), num_pages, None, k, v, slots)
        pool = gpu_append(case)
        ora = oracle_append(case)
        nd, nt = compare_pools(pool.cpu().numpy(), ora, case)
        log("fuzz compose=%s differing bytes %d tolerated elements %d" % (compose, nd, nt))


def test_append_only_touches_addressed_slots():
    cfg = W.custom("touch", 1, 4, 2, [1], seed_index=84)
    Rk, Rv = W.rotation(5), W.rotation(6)
    slots = np.array([3, 64 + 17, 5 * 64 + 63], np.int64)
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 3, 2, 128)).astype(np.float32)
    k = torch.from_numpy(W.f32_to_bf16_bits(x[0]).view(np.int16)).view(torch.bfloat16)
    v = torch.from_numpy(W.f32_to_bf16_bits(x[1]).view(np.int16)).view(torch.bfloat16)
    case = Case(cfg, Rk, Rv, np.zeros((1, 1), np.int32), 8, None, k, v, slots)
    pool = torch.full((ok.pool_bytes(case.layout),), 0xA5, dtype=torch.uint8, device="cuda")
    gpu_append(case, pool)
    ora = np.full(ok.pool_bytes(case.layout), 0xA5, np.uint8)
    oracle.kv_append(ora, d=128, Hkv=2, P=64, G=32, k=bits(k), v=bits(v), slot_mapping=slots,
                     Rk=Rk, Rv=Rv, clip_k=cfg.clip_k, clip_v=cfg.clip_v)
    assert np.array_equal(pool.cpu().numpy(), ora)


def test_bf16_baseline_parity():
    cfg = W.custom("bf16base", 3, 24, 2, [1, 1000, 2500], seed_index=85, k_outliers=(3,))
    case = make_case(cfg)
    lay = case.layout
    pool = torch.zeros(ok.bf16_pool_bytes(lay) // 2, dtype=torch.bfloat16, device="cuda")
    ok.bf16_kv_append(lay, pool, case.k.cuda(), case.v.cuda(),
                      torch.from_numpy(case.slots).cuda())
    ora = np.zeros(ok.bf16_pool_bytes(lay) // 2, np.uint16)
    oracle.bf16_append(ora, d=128, Hkv=2, P=64, k=bits(case.k), v=bits(case.v),
                       slot_mapping=case.slots)
    assert np.array_equal(bits(pool), ora)
    ref = oracle.bf16_decode(ora, d=128, Hkv=2, P=64, q=bits(case.q), block_table=case.table,
                             seq_lens=cfg.lens, sm_scale=cfg.sm_scale)
    for S in (1, 6):
        ws = ok.alloc_workspace(lay, cfg.B, cfg.Hq, S)
        out = torch.empty(cfg.B, cfg.Hq, 128, dtype=torch.float32, device="cuda")
        ok.bf16_decode_attn(lay, pool, case.q.cuda(), torch.from_numpy(case.table).cuda(),
                            torch.from_numpy(cfg.lens).cuda(), cfg.sm_scale, S, ws, out)
        torch.cuda.synchronize()
        err = max_abs(out, ref)
        log("bf16 baseline splits", S, "max|err| %.3g" % err)
        assert err <= DECODE_TOL


def test_append_zero_point_sign_and_hand_rows():
    # R = I and rows whose group minimum is exactly 0 (z = -0/s must be stored
    # as +0), all-zero groups (degenerate), and exactly representable groups.
    cfg = W.custom("zeros", 1, 2, 2, [1], seed_index=86, clip_k=1.0, clip_v=1.0)
    eye = np.eye(128, dtype=np.float32)
    rows = np.zeros((2, 4, 2, 128), np.float32)
    rows[:, 0, :, :32] = np.tile([0, 1, 2, 3], 8)          # min exactly 0
    rows[:, 1, :, 32:64] = np.tile([-1.5, -0.5, 0.5, 1.5], 8)
    rows[:, 2, :, 64:96] = -np.tile([0, 1, 2, 3], 8)        # max exactly 0
    rows[:, 3] = np.linspace(-2, 2, 128)
    k = torch.from_numpy(W.f32_to_bf16_bits(rows[0]).view(np.int16)).view(torch.bfloat16)
    v = torch.from_numpy(W.f32_to_bf16_bits(rows[1]).view(np.int16)).view(torch.bfloat16)
    slots = np.array([0, 65, 130, 7], np.int64)
    case = Case(cfg, eye, eye, np.zeros((1, 1), np.int32), 3, None, k, v, slots)
    pool = gpu_append(case)
    ora = oracle_append(case)
    assert np.array_equal(pool.cpu().numpy(), ora)
