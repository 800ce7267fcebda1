"""The page-byte comparison rule of the parity tests (helpers.compare_pools),
checked on the CPU with differences planted in a copy of an oracle-written pool:
a code whose y/s + z lies on a rounding boundary may differ (counted as one
tolerated element); a code, scale or zero point away from any boundary may not.

The row is built so that the arithmetic is exact: R = I, clip ratio 1, group 0
holds 0, 3, 1.5 and integers (a = 0, b = 3, s = 1, z = 0, so y/s + z = y): only
channel 2 (y = 1.5) sits on a boundary, where round-half-even gives code 2."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from helpers import Case, compare_pools, row_tolerated_elements, _row_fields

EYE = np.eye(128, dtype=np.float32)


def _case():
    cfg = W.custom("rule", 1, 1, 1, [1], seed_index=93, clip_k=1.0, clip_v=1.0)
    row = np.zeros(128, np.float32)
    row[:8] = [0.0, 3.0, 1.5, 1.0, 2.0, 3.0, 0.0, 2.0]
    row[32:64] = np.linspace(-1.0, 1.0, 32)
    x = np.stack([row, row])[:, None, :]                       # [2 tokens, 1 head, 128]
    k = torch.from_numpy(W.f32_to_bf16_bits(x).view(np.int16)).view(torch.bfloat16)
    slots = np.array([0, 1], np.int64)
    case = Case(cfg, EYE, EYE, np.zeros((1, 1), np.int32), 1, None, k, k.clone(), slots)
    pool = np.zeros(oracle.page_head_bytes(128, 64, 32), np.uint8)
    oracle.kv_append(pool, d=128, Hkv=1, P=64, G=32, k=W.f32_to_bf16_bits(x), v=W.f32_to_bf16_bits(x),
                     slot_mapping=slots, Rk=EYE, Rv=EYE, clip_k=1.0, clip_v=1.0)
    return case, pool


def _set_code(pool, t, c, code):  # K codes of token t, channel c
    b = t * 32 + c // 4
    sh = 2 * (c % 4)
    pool[b] = (int(pool[b]) & (0xFF ^ (3 << sh))) | (code << sh)


def test_oracle_row_is_as_constructed():
    case, pool = _case()
    codes, sz = _row_fields(pool, 0, 0, 0, 32)
    assert list(codes[:8]) == [0, 3, 2, 1, 2, 3, 0, 2]         # 1.5 -> 2 (half to even)
    assert sz[0, 0] == 0x3C00 and sz[0, 1] == 0                 # s = 1, z = +0


def test_identical_pools_compare_equal():
    case, pool = _case()
    assert compare_pools(pool.copy(), pool, case) == (0, 0)


def test_code_on_a_rounding_boundary_is_one_tolerated_element():
    case, pool = _case()
    gpu = pool.copy()
    _set_code(gpu, 0, 2, 1)                                     # 1.5 rounded the other way
    assert compare_pools(gpu, pool, case) == (1, 1)


@pytest.mark.parametrize("c,code", [(1, 2), (3, 2), (40, 0)])
def test_code_away_from_a_boundary_fails(c, code):
    case, pool = _case()
    gpu = pool.copy()
    _set_code(gpu, 1, c, code)
    with pytest.raises(AssertionError):
        compare_pools(gpu, pool, case)


def test_scale_or_zero_away_from_a_midpoint_fails():
    case, pool = _case()
    for byte in (4096 + 1, 4096 + 2):                           # token 0, group 0: s high byte, z low byte
        gpu = pool.copy()
        gpu[byte] ^= 0x01
        with pytest.raises(AssertionError):
            compare_pools(gpu, pool, case)


def test_element_count_not_row_count():
    # one tolerated and one untolerated code in the same row: the row
    # is not excused as a whole
    case, pool = _case()
    gpu = pool.copy()
    _set_code(gpu, 0, 2, 1)
    _set_code(gpu, 0, 4, 1)                                     # y = 2: far from a boundary
    with pytest.raises(AssertionError):
        compare_pools(gpu, pool, case)
    codes_g, sz_g = _row_fields(gpu, 0, 0, 0, 32)
    codes_o, sz_o = _row_fields(pool, 0, 0, 0, 32)
    xt = oracle.rotate_row(W.bf16_bits_to_f32(W.f32_to_bf16_bits(
        np.r_[[0.0, 3.0, 1.5, 1.0, 2.0, 3.0, 0.0, 2.0], np.zeros(24), np.linspace(-1, 1, 32),
              np.zeros(64)].astype(np.float32))), EYE)
    assert row_tolerated_elements(xt, 1.0, codes_g, sz_g, codes_o, sz_o) == (2, 1)
