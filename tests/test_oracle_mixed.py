"""Pins of the oracle's mixed-precision cache (Sec. 4 "KV Cache Layout"; Alg. 1
DecodeStep): a bf16 sink of S0 tokens and a bf16 window of the W most recent
tokens around the INT2 history, the per-step demotion of the oldest window token,
and decode attention over the three segments.

The caches are built one token per step through ``oracle.mixed_update``, as a
decode loop would.  Pins:
  * keys/values that the INT2 path stores exactly: decode equals plain softmax
    attention over the original rows for any (S0, W), so a token read from the
    wrong segment, slot or position changes the result;
  * general rows: decode equals a brute-force evaluation written here from the
    algorithm's concatenation (dequantize and rotate back the history, take the
    sink and window rows from the segment store at their documented offsets);
  * demotion writes exactly the bytes of a direct cache update of the history
    tokens, and nothing at sink or window positions;
  * S0 = W = 0 is the INT2-only path, byte for byte and output for output.
"""
import math

import numpy as np
import pytest

import oracle
import workloads as W
from test_oracle_pins import _exact_rows, _signed_cyclic

D, P, G = 128, 64, 32


def _orthogonal(seed, d=D):
    q, r = np.linalg.qr(np.random.default_rng(seed).standard_normal((d, d)))
    return (q * np.sign(np.diag(r))).astype(np.float32)


def _build(B, Hq, Hkv, lens, S0, W_, rows_k, rows_v, Rk, Rv, clip, seed):
    """Run the decode loop's cache side from empty caches up to lens[b] tokens."""
    mp = int(math.ceil(max(lens) / P)) + 1
    num_pages = B * mp
    table = np.random.default_rng(seed).permutation(num_pages).astype(np.int32).reshape(B, mp)
    pages = np.zeros(num_pages * Hkv * oracle.page_head_bytes(D, P, G), np.uint8)
    seg = np.zeros(oracle.seg_elems(d=D, Hkv=Hkv, B=B, S0=S0, W=W_), np.uint16)
    chunk = Hkv * 2 * (S0 + W_) * D                  # one sequence's part of the store
    for b in range(B):
        seg_b = seg[b * chunk:(b + 1) * chunk]        # a view: updated in place
        for n in range(1, lens[b] + 1):
            oracle.mixed_update(pages, seg_b, d=D, Hkv=Hkv, P=P, G=G, S0=S0, W=W_,
                                k_new=rows_k[b:b + 1, n - 1], v_new=rows_v[b:b + 1, n - 1],
                                block_table=table[b:b + 1], seq_lens=np.array([n], np.int32),
                                Rk=Rk, Rv=Rv, clip_k=clip, clip_v=clip)
    return pages, seg, table


@pytest.mark.parametrize("S0,W_", [(0, 0), (64, 256), (16, 32), (32, 128), (0, 64), (48, 0)])
def test_exact_rows_mixed_decode_equals_plain_attention(S0, W_):
    """Rows the INT2 path stores exactly: the segments must reproduce every token."""
    B, Hq, Hkv = 3, 8, 2
    lens = [5, 150, 333]
    Rk = _signed_cyclic(D, 5, 1)
    Rv = _signed_cyclic(D, 11, 2)
    nmax = max(lens)
    kt = _exact_rows(B * nmax * Hkv, 30).reshape(B, nmax, Hkv, D)
    vt = _exact_rows(B * nmax * Hkv, 31).reshape(B, nmax, Hkv, D)
    k = (kt @ Rk.T).astype(np.float32)                # k = k~ Rk^T exactly
    v = (vt @ Rv.T).astype(np.float32)
    kb, vb = W.f32_to_bf16_bits(k), W.f32_to_bf16_bits(v)
    assert np.array_equal(W.bf16_bits_to_f32(kb), k)  # the rows are bf16 numbers
    pages, seg, table = _build(B, Hq, Hkv, lens, S0, W_, kb, vb, Rk, Rv, 1.0, 7)
    q = W.f32_to_bf16_bits(np.random.default_rng(8).standard_normal((B, Hq, D)).astype(np.float32))
    sm = 1.0 / math.sqrt(D)
    got = oracle.decode_mixed(pages, seg, d=D, Hkv=Hkv, P=P, G=G, S0=S0, W=W_, q=q,
                              block_table=table, seq_lens=np.array(lens, np.int32), Rk=Rk, Rv=Rv,
                              sm_scale=sm)
    qf = W.bf16_bits_to_f32(q).astype(np.float64)
    for b in range(B):
        for h in range(Hq):
            kvh = h // (Hq // Hkv)
            s = sm * (k[b, :lens[b], kvh].astype(np.float64) @ qf[b, h])
            p = np.exp(s - s.max())
            ref = p @ v[b, :lens[b], kvh].astype(np.float64) / p.sum()
            assert np.max(np.abs(got[b, h] - ref)) < 1e-12, (S0, W_, b, h)


def _brute(pages, seg, table, q, lens, S0, W_, Hkv, Rk, Rv, sm):
    """Alg. 1 DecodeStep written out: concatenate sink, dequantized history
    rotated back, and window; plain softmax attention (numpy, fp64)."""
    B, Hq = q.shape[0], q.shape[1]
    out = np.zeros((B, Hq, D))
    qf = W.bf16_bits_to_f32(q).astype(np.float64)
    segf = W.bf16_bits_to_f32(seg).astype(np.float64)

    def seg_rowv(b, h, is_v, slot):                   # the documented store layout
        base = (((b * Hkv + h) * 2 + is_v) * (S0 + W_) + slot) * D
        return segf[base:base + D]

    for b in range(B):
        n = lens[b]
        lo = min(S0, n)
        hi = max(lo, n - W_)
        for kvh in range(Hkv):
            Kall = np.zeros((n, D))
            Vall = np.zeros((n, D))
            for t in range(n):
                if t < lo or t >= hi:
                    slot = t if t < S0 else S0 + (t - S0) % W_
                    Kall[t] = seg_rowv(b, kvh, 0, slot)
                    Vall[t] = seg_rowv(b, kvh, 1, slot)
                else:
                    page = int(table[b, t // P])
                    for is_v, dst, R in ((0, Kall, Rk), (1, Vall, Rv)):
                        codes, s16, z16 = oracle.read_token(pages, d=D, Hkv=Hkv, P=P, G=G,
                                                            page=page, h=kvh, t=t % P,
                                                            is_v=bool(is_v))
                        s = np.repeat(s16.view(np.float16).astype(np.float64), G)
                        z = np.repeat(z16.view(np.float16).astype(np.float64), G)
                        dst[t] = (s * (codes.astype(np.float64) - z)) @ R.astype(np.float64).T
            for h in range(kvh * (Hq // Hkv), (kvh + 1) * (Hq // Hkv)):
                sc = sm * (Kall @ qf[b, h])
                p = np.exp(sc - sc.max())
                out[b, h] = p @ Vall / p.sum()
    return out


@pytest.mark.parametrize("S0,W_", [(16, 32), (64, 64), (32, 0)])
def test_general_rows_mixed_decode_equals_brute_force(S0, W_):
    B, Hq, Hkv = 2, 4, 1
    lens = [40, 201]
    Rk, Rv = _orthogonal(3), _orthogonal(4)
    nmax = max(lens)
    rng = np.random.default_rng(5)
    kb = W.f32_to_bf16_bits(rng.standard_normal((B, nmax, Hkv, D)).astype(np.float32))
    vb = W.f32_to_bf16_bits(rng.standard_normal((B, nmax, Hkv, D)).astype(np.float32))
    pages, seg, table = _build(B, Hq, Hkv, lens, S0, W_, kb, vb, Rk, Rv, 0.9, 9)
    q = W.f32_to_bf16_bits(rng.standard_normal((B, Hq, D)).astype(np.float32))
    sm = 1.0 / math.sqrt(D)
    got = oracle.decode_mixed(pages, seg, d=D, Hkv=Hkv, P=P, G=G, S0=S0, W=W_, q=q,
                              block_table=table, seq_lens=np.array(lens, np.int32), Rk=Rk, Rv=Rv,
                              sm_scale=sm)
    ref = _brute(pages, seg, table, q, lens, S0, W_, Hkv, Rk, Rv, sm)
    assert np.max(np.abs(got - ref)) < 1e-10


@pytest.mark.parametrize("S0,W_", [(16, 32), (64, 256), (0, 0), (40, 0)])
def test_demotion_writes_the_bytes_of_a_direct_update(S0, W_):
    """After the loop, the history positions [S0, n - W) hold exactly the bytes a
    direct cache update of those tokens writes; sink and window positions hold
    nothing in the INT2 pool."""
    B, Hkv = 2, 2
    lens = [90, 400]
    Rk, Rv = _orthogonal(10), _orthogonal(11)
    nmax = max(lens)
    rng = np.random.default_rng(12)
    kb = W.f32_to_bf16_bits(rng.standard_normal((B, nmax, Hkv, D)).astype(np.float32))
    vb = W.f32_to_bf16_bits(rng.standard_normal((B, nmax, Hkv, D)).astype(np.float32))
    pages, seg, table = _build(B, 4, Hkv, lens, S0, W_, kb, vb, Rk, Rv, 0.9, 13)
    direct = np.zeros_like(pages)
    bph = oracle.page_head_bytes(D, P, G)
    for b in range(B):
        n = lens[b]
        lo = min(S0, n)
        hi = max(lo, n - W_)
        pos = np.arange(lo, hi)
        if len(pos):
            oracle.kv_append(direct, d=D, Hkv=Hkv, P=P, G=G, k=kb[b, pos], v=vb[b, pos],
                             slot_mapping=W.slots_for(table, b, pos), Rk=Rk, Rv=Rv, clip_k=0.9,
                             clip_v=0.9)
    assert np.array_equal(pages, direct)
    assert bph > 0


def test_without_segments_is_the_int2_path():
    B, Hq, Hkv = 2, 8, 2
    lens = [64, 129]
    Rk, Rv = _orthogonal(20), _orthogonal(21)
    nmax = max(lens)
    rng = np.random.default_rng(22)
    kb = W.f32_to_bf16_bits(rng.standard_normal((B, nmax, Hkv, D)).astype(np.float32))
    vb = W.f32_to_bf16_bits(rng.standard_normal((B, nmax, Hkv, D)).astype(np.float32))
    pages, seg, table = _build(B, Hq, Hkv, lens, 0, 0, kb, vb, Rk, Rv, 0.9, 23)
    assert seg.size == 0
    q = W.f32_to_bf16_bits(rng.standard_normal((B, Hq, D)).astype(np.float32))
    sl = np.array(lens, np.int32)
    a = oracle.decode_mixed(pages, seg, d=D, Hkv=Hkv, P=P, G=G, S0=0, W=0, q=q, block_table=table,
                            seq_lens=sl, Rk=Rk, Rv=Rv, sm_scale=0.1)
    b = oracle.decode(pages, d=D, Hkv=Hkv, P=P, G=G, q=q, block_table=table, seq_lens=sl, Rk=Rk,
                      Rv=Rv, sm_scale=0.1)
    assert np.max(np.abs(a - b)) < 1e-12


def test_segment_store_offsets_by_hand():
    """Sequence 1, head 1 of Hkv = 2, S0 = 2, W = 3, d = 128: position 0 -> slot 0,
    position 6 -> slot 2 + (6 - 2) % 3 = 3; K row of slot 3 at element
    (((1*2 + 1)*2 + 0)*5 + 3)*128 = 33*128 = 4224, V row at (((1*2 + 1)*2 + 1)*5 + 3)*128
    = 38*128 = 4864, K row of slot 0 at 30*128 = 3840."""
    Hkv, S0, W_, B = 2, 2, 3, 2
    seg = np.zeros(oracle.seg_elems(d=D, Hkv=Hkv, B=B, S0=S0, W=W_), np.uint16)
    assert seg.size == 2 * 2 * 2 * 5 * 128
    k = np.zeros((2, Hkv, D), np.uint16)
    v = np.zeros((2, Hkv, D), np.uint16)
    k[:, 1, :] = 0x1111
    v[:, 1, :] = 0x2222
    k[1, 1, 5] = 0x3f80
    oracle.seg_write(seg, d=D, Hkv=Hkv, B=B, S0=S0, W=W_, k=k, v=v,
                     seq_idx=np.array([1, 1]), pos=np.array([0, 6]))
    assert np.all(seg[4224:4224 + 128][[i for i in range(128) if i != 5]] == 0x1111)
    assert seg[4224 + 5] == 0x3f80
    assert np.all(seg[4864:4864 + 128] == 0x2222)
    assert np.all(seg[3840:3840 + 128] == 0x1111)  # position 0
    assert np.count_nonzero(seg) == 4 * 128
    with pytest.raises(ValueError):                 # no bf16 slot beyond the sink when W = 0
        oracle.seg_write(np.zeros(oracle.seg_elems(d=D, Hkv=Hkv, B=B, S0=S0, W=0), np.uint16),
                         d=D, Hkv=Hkv, B=B, S0=S0, W=0, k=k[:1], v=v[:1], seq_idx=np.array([0]),
                         pos=np.array([2]))
