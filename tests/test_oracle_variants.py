"""Pins of the oracle's quantizer variants (App. "Scale Determination and Per-token
Clipping Details"; Sec. 4 "KV Cache Update"):

  * bfloat16 conversion of the stored scale and zero: identity on the bf16 grid,
    ties to even, against torch's float32 -> bfloat16 rounding on a large sample
    and on edge values (an independent implementation);
  * the per-token quantile clip threshold: numpy's linear-interpolation quantile
    (fp64) within fp32 rounding, exact order statistics where the position is an
    integer or a half, rho = 1 is the row maximum;
  * the token-wide threshold: one tau for every group of the row, so a group of
    small values is untouched while another group is clipped at tau;
  * quantile clip with rho = 1 is the absmax rule with rho = 1 (no clipping);
  * bf16 metadata: stored s is the bf16 rounding of (b - a)/3, dequantize then
    quantize returns every code, and the reconstruction error bound;
  * group sizes 64 and 128: rows that the quantizer represents exactly decode to
    plain attention;
  * a NULL rotation is the identity: the stored codes are those of the bf16 rows
    themselves, and decode equals plain attention over the rows dequantized and
    evaluated here in numpy.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W

D, P = 128, 64


def _bf16_torch(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


# ---------------------------------------------------------------------------
# bfloat16 conversion
# ---------------------------------------------------------------------------

def test_bf16_conversion_identity_on_grid_and_torch():
    # every finite bf16 value converts to itself
    bits = np.arange(1 << 16, dtype=np.uint32)
    finite = ((bits >> 7) & 0xff) != 0xff
    for h in bits[finite][::97]:
        x = float(W.bf16_bits_to_f32(np.array([h], np.uint16))[0])
        assert oracle.f32_to_bf16_bits(x) == h
    # random fp32 over many binades, and the midpoints between neighbours (ties)
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(20000) * np.exp2(rng.integers(-140, 120, 20000))).astype(np.float32)
    mids = []
    for h in rng.integers(0x0001, 0x7f7f, 2000).astype(np.uint32):
        lo = np.uint32(h) << 16
        mids.append(np.uint32(lo | 0x8000))          # exactly halfway to the next bf16
        mids.append(np.uint32(lo | 0x8001))          # just above halfway
        mids.append(np.uint32(lo | 0x7fff))          # just below halfway
    x = np.concatenate([x, np.array(mids, np.uint32).view(np.float32)])
    ref = _bf16_torch(x)
    got = np.array([oracle.f32_to_bf16_bits(float(v)) for v in x], np.uint16)
    assert np.array_equal(got, ref)
    # overflow to infinity and the largest finite value
    big = np.array([0x7f7f0000, 0x7f7f7fff, 0x7f7f8000, 0x7f7fffff], np.uint32).view(np.float32)
    assert [oracle.f32_to_bf16_bits(float(v)) for v in big] == [0x7f7f, 0x7f7f, 0x7f80, 0x7f80]


# ---------------------------------------------------------------------------
# per-token quantile clip
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("rho", [0.5, 0.9, 0.92, 0.96, 0.999, 0.1, 1.0])
def test_token_quantile_matches_linear_quantile(rho):
    rng = np.random.default_rng(int(rho * 1000))
    for _ in range(50):
        x = (rng.standard_normal(D) * rng.choice([1.0, 10.0], D)).astype(np.float32)
        ax = np.abs(x).astype(np.float64)
        got = oracle.token_quantile(x, rho)
        # numpy's linear quantile at the exact position rho (d - 1): the oracle's
        # position is rounded to fp32 (|dpos| <= 127 * 2^-24)
        ref = float(np.quantile(ax, np.float64(np.float32(rho)), method="linear"))
        gap = float(np.max(np.diff(np.sort(ax))))
        assert abs(got - ref) <= 127 * 2.0 ** -24 * gap + 4 * np.spacing(np.float32(ref))
        # the same interpolation written here in fp64 at the fp32 position
        pos = float(np.float32(np.float32(rho) * np.float32(D - 1)))
        k = min(int(math.floor(pos)), D - 1)
        a = np.sort(ax)
        ref32 = a[k] if k == D - 1 else a[k] + (pos - k) * (a[k + 1] - a[k])
        assert abs(got - ref32) <= 4 * np.spacing(np.float32(ref32)), (rho, got, ref32)


def test_token_quantile_exact_order_statistics():
    # |x| = a permutation of 1..128: position rho*127 picks / averages known values
    rng = np.random.default_rng(3)
    x = (np.arange(1, D + 1) * rng.choice([-1, 1], D))[rng.permutation(D)].astype(np.float32)
    assert oracle.token_quantile(x, 1.0) == 128.0          # the maximum
    assert oracle.token_quantile(x, 0.5) == 64.5           # pos 63.5: (64 + 65) / 2
    assert oracle.token_quantile(x, 0.0) == 1.0            # the minimum


def test_quantile_clip_is_token_wide():
    # group 0 small, group 3 with outliers: one tau for the whole row
    x = np.zeros(D, np.float32)
    x[:32] = np.linspace(-1.0, 1.0, 32)
    x[32:96] = np.linspace(-2.0, 2.0, 64)
    x[96:] = np.linspace(-50.0, 50.0, 32)
    rho = 0.9
    tau = oracle.token_quantile(x, rho)
    assert 2.0 < tau < 50.0
    codes, s16, z16, _ = oracle.quantize_row(x, 32, rho, clip=1)
    # group 0 is below tau: identical to quantizing it without any clipping
    c_free, s_free, z_free, _ = oracle.quantize_row(x, 32, 1.0, clip=0)
    assert np.array_equal(codes[:32], c_free[:32]) and s16[0] == s_free[0] and z16[0] == z_free[0]
    # group 3 is clipped at +-tau: range 2 tau
    assert s16[3] == oracle.f32_to_f16_bits(np.float32(np.float32(2 * np.float32(tau)) / np.float32(3)))
    # the absmax rule would have used 0.9 * 50 for group 3
    _, s_abs, _, _ = oracle.quantize_row(x, 32, rho, clip=0)
    assert s_abs[3] != s16[3]


def test_quantile_clip_rho_one_is_no_clipping():
    rng = np.random.default_rng(5)
    for _ in range(20):
        x = (rng.standard_normal(D) * 3).astype(np.float32)
        for G in (32, 64, 128):
            for meta in (0, 1):
                a = oracle.quantize_row(x, G, 1.0, meta=meta, clip=1)
                b = oracle.quantize_row(x, G, 1.0, meta=meta, clip=0)
                for u, v in zip(a[:3], b[:3]):
                    assert np.array_equal(u, v)


# ---------------------------------------------------------------------------
# bf16 metadata
# ---------------------------------------------------------------------------

def test_bf16_meta_scale_rounding_roundtrip_and_error_bound():
    rng = np.random.default_rng(7)
    for trial in range(200):
        G = (32, 64, 128)[trial % 3]
        x = (rng.standard_normal(D) * np.exp2(rng.integers(-6, 8))).astype(np.float32)
        codes, s16, z16, sat = oracle.quantize_row(x, G, 1.0, meta=1)
        assert sat == 0
        for g in range(D // G):
            y = x[g * G:(g + 1) * G]
            a, b = np.float32(y.min()), np.float32(y.max())
            s_exact = np.float32(np.float32(b - a) / np.float32(3.0))
            assert s16[g] == _bf16_torch(np.array([s_exact]))[0]
            s = float(W.bf16_bits_to_f32(np.array([s16[g]], np.uint16))[0])
            z = float(W.bf16_bits_to_f32(np.array([z16[g]], np.uint16))[0])
            k = codes[g * G:(g + 1) * G].astype(np.float64)
            rec = s * (k - z)
            # half a step, plus the zero point's bf16 rounding (2^-8 relative)
            bound = s * (0.5 + abs(z) * 2.0 ** -8) + 1e-30
            assert np.all(np.abs(rec - y) <= bound * (1 + 1e-6))
            # dequantize, then quantize again with the stored s, z: the same codes
            u = (rec.astype(np.float32) / np.float32(s)).astype(np.float32) + np.float32(z)
            assert np.array_equal(np.clip(np.rint(u), 0, 3).astype(np.uint8), codes[g * G:(g + 1) * G])


# ---------------------------------------------------------------------------
# group sizes 64 / 128 and bf16 metadata: exact rows decode to plain attention
# ---------------------------------------------------------------------------

def _exact_rows_g(n, seed, G):
    """Rows whose every G-group is a + k s (k in 0..3, 0 and 3 present), s and a
    dyadic: the quantizer (rho = 1, either metadata format) stores them exactly."""
    rng = np.random.default_rng(seed)
    out = np.zeros((n, D), np.float32)
    for i in range(n):
        for g in range(D // G):
            s = 2.0 ** int(rng.integers(-2, 2))
            a = s * float(rng.integers(-3, 1))
            ks = rng.integers(0, 4, size=G)
            ks[rng.permutation(G)[:2]] = [0, 3]
            out[i, g * G:(g + 1) * G] = a + s * ks
    return out


@pytest.mark.parametrize("G,meta,clip", [(64, 0, 0), (128, 0, 0), (32, 1, 0), (128, 1, 1),
                                         (64, 1, 1)])
def test_variant_exact_rows_decode_equals_plain_attention(G, meta, clip):
    B, Hq, Hkv = 2, 8, 2
    lens = [70, 193]
    mp = 4
    table = np.random.default_rng(11).permutation(B * mp).astype(np.int32).reshape(B, mp)
    bph = oracle.page_head_bytes(D, P, G)
    pages = np.zeros(B * mp * Hkv * bph, np.uint8)
    K, V = [], []
    for b in range(B):
        k = _exact_rows_g(lens[b] * Hkv, 100 + b, G).reshape(lens[b], Hkv, D)
        v = _exact_rows_g(lens[b] * Hkv, 200 + b, G).reshape(lens[b], Hkv, D)
        K.append(k)
        V.append(v)
        oracle.kv_append(pages, d=D, Hkv=Hkv, P=P, G=G, k=W.f32_to_bf16_bits(k),
                         v=W.f32_to_bf16_bits(v), slot_mapping=W.slots_for(table, b, np.arange(lens[b])),
                         Rk=None, Rv=None, clip_k=1.0, clip_v=1.0, meta=meta, clip=clip)
    q = W.f32_to_bf16_bits(np.random.default_rng(12).standard_normal((B, Hq, D)).astype(np.float32))
    sm = 1.0 / math.sqrt(D)
    got = oracle.decode(pages, d=D, Hkv=Hkv, P=P, G=G, q=q, block_table=table,
                        seq_lens=np.array(lens, np.int32), Rk=None, Rv=None, sm_scale=sm, meta=meta)
    qf = W.bf16_bits_to_f32(q).astype(np.float64)
    for b in range(B):
        for h in range(Hq):
            kvh = h // (Hq // Hkv)
            s = sm * (K[b][:, kvh].astype(np.float64) @ qf[b, h])
            p = np.exp(s - s.max())
            ref = p @ V[b][:, kvh].astype(np.float64) / p.sum()
            assert np.max(np.abs(got[b, h] - ref)) < 1e-12


# ---------------------------------------------------------------------------
# identity rotation
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("meta,clip", [(0, 0), (1, 1)])
def test_null_rotation_is_identity(meta, clip):
    B, Hq, Hkv, G = 2, 4, 2, 32
    lens = [65, 130]
    mp = 4
    table = np.random.default_rng(21).permutation(B * mp).astype(np.int32).reshape(B, mp)
    bph = oracle.page_head_bytes(D, P, G)
    pages = np.zeros(B * mp * Hkv * bph, np.uint8)
    rng = np.random.default_rng(22)
    rows = {}
    for b in range(B):
        kb = W.f32_to_bf16_bits((rng.standard_normal((lens[b], Hkv, D)) * 2).astype(np.float32))
        vb = W.f32_to_bf16_bits(rng.standard_normal((lens[b], Hkv, D)).astype(np.float32))
        rows[b] = (kb, vb)
        oracle.kv_append(pages, d=D, Hkv=Hkv, P=P, G=G, k=kb, v=vb,
                         slot_mapping=W.slots_for(table, b, np.arange(lens[b])), Rk=None, Rv=None,
                         clip_k=0.9, clip_v=0.95, meta=meta, clip=clip)
    # the stored codes are those of the rows themselves
    b, t, h = 1, 77, 1
    for is_v, rho in ((0, 0.9), (1, 0.95)):
        x = W.bf16_bits_to_f32(rows[b][is_v][t, h])
        c_ref, s_ref, z_ref, _ = oracle.quantize_row(x, G, rho, meta=meta, clip=clip)
        c, s16, z16 = oracle.read_token(pages, d=D, Hkv=Hkv, P=P, G=G, page=int(table[b, t // P]),
                                        h=h, t=t % P, is_v=bool(is_v))
        assert np.array_equal(c, c_ref) and np.array_equal(s16, s_ref) and np.array_equal(z16, z_ref)
    # decode = plain attention over the dequantized rows (dequantized here in numpy)
    to_f = W.bf16_bits_to_f32 if meta else (lambda hbits: np.array([oracle.f16_bits_to_f32(int(u)) for u in np.ravel(hbits)], np.float32).reshape(np.shape(hbits)))
    q = W.f32_to_bf16_bits(rng.standard_normal((B, Hq, D)).astype(np.float32))
    sm = 1.0 / math.sqrt(D)
    got = oracle.decode(pages, d=D, Hkv=Hkv, P=P, G=G, q=q, block_table=table,
                        seq_lens=np.array(lens, np.int32), Rk=None, Rv=None, sm_scale=sm, meta=meta)
    qf = W.bf16_bits_to_f32(q).astype(np.float64)
    for b in range(B):
        for hq in range(Hq):
            kvh = hq // (Hq // Hkv)
            deq = {}
            for is_v in (0, 1):
                rr = np.zeros((lens[b], D))
                for t in range(lens[b]):
                    c, s16, z16 = oracle.read_token(pages, d=D, Hkv=Hkv, P=P, G=G,
                                                    page=int(table[b, t // P]), h=kvh, t=t % P,
                                                    is_v=bool(is_v))
                    s = np.repeat(to_f(s16).astype(np.float64), G)
                    z = np.repeat(to_f(z16).astype(np.float64), G)
                    rr[t] = s * (c.astype(np.float64) - z)
                deq[is_v] = rr
            sc = sm * (deq[0] @ qf[b, hq])
            p = np.exp(sc - sc.max())
            ref = p @ deq[1] / p.sum()
            assert np.max(np.abs(got[b, hq] - ref)) < 1e-10


# ---------------------------------------------------------------------------
# one rotation per KV head
# ---------------------------------------------------------------------------

def _signed_perm(rng, d=D):
    """R with x R = a signed permutation of x: R[perm[j], j] = sign[j]."""
    perm = rng.permutation(d)
    sign = rng.choice([-1.0, 1.0], d)
    R = np.zeros((d, d), np.float32)
    R[perm, np.arange(d)] = sign
    return R, perm, sign


def _cache(Rk, Rv, kb, vb, table, lens, Hkv, G=32, meta=0, clip=0):
    pages = np.zeros(table.size * Hkv * oracle.page_head_bytes(D, P, G), np.uint8)
    for b in range(len(lens)):
        oracle.kv_append(pages, d=D, Hkv=Hkv, P=P, G=G, k=kb[b], v=vb[b],
                         slot_mapping=W.slots_for(table, b, np.arange(lens[b])), Rk=Rk, Rv=Rv,
                         clip_k=0.9, clip_v=0.95, meta=meta, clip=clip)
    return pages


def test_per_head_rotation_maps_each_head_to_its_matrix():
    """With R_h a signed permutation per KV head, the cache of head h holds the
    codes of the rows permuted by R_h (bit-exact against the identity-rotation
    cache of those permuted rows), and decode equals the identity-rotation decode
    of the permuted query, rotated back by R_h^T."""
    B, Hq, Hkv, mp = 2, 6, 3, 3
    lens = [70, 129]
    rng = np.random.default_rng(41)
    table = rng.permutation(B * mp).astype(np.int32).reshape(B, mp)
    kb = [W.f32_to_bf16_bits((rng.standard_normal((n, Hkv, D)) * 2).astype(np.float32)) for n in lens]
    vb = [W.f32_to_bf16_bits(rng.standard_normal((n, Hkv, D)).astype(np.float32)) for n in lens]
    Rs = [_signed_perm(rng) for _ in range(2 * Hkv)]
    Rk = np.stack([r[0] for r in Rs[:Hkv]])
    Rv = np.stack([r[0] for r in Rs[Hkv:]])
    pages = _cache(Rk, Rv, kb, vb, table, lens, Hkv)

    def permuted(x, which):  # x~ = x R_h per head (exact: signed permutation of bf16)
        out = np.empty_like(x)
        for h in range(Hkv):
            _, perm, sign = Rs[which * Hkv + h]
            f = W.bf16_bits_to_f32(x[:, h])[:, perm] * sign
            out[:, h] = W.f32_to_bf16_bits(f.astype(np.float32))
        return out

    ref = _cache(None, None, [permuted(k, 0) for k in kb], [permuted(v, 1) for v in vb], table,
                 lens, Hkv)
    assert np.array_equal(pages, ref)
    q = W.f32_to_bf16_bits(rng.standard_normal((B, Hq, D)).astype(np.float32))
    sm = 1.0 / math.sqrt(D)
    got = oracle.decode(pages, d=D, Hkv=Hkv, P=P, G=32, q=q, block_table=table,
                        seq_lens=np.array(lens, np.int32), Rk=Rk, Rv=Rv, sm_scale=sm)
    g = Hq // Hkv
    qp = np.empty_like(q)
    for hq in range(Hq):
        _, perm, sign = Rs[hq // g]
        qp[:, hq] = W.f32_to_bf16_bits((W.bf16_bits_to_f32(q[:, hq])[:, perm] * sign).astype(np.float32))
    base = oracle.decode(pages, d=D, Hkv=Hkv, P=P, G=32, q=qp, block_table=table,
                         seq_lens=np.array(lens, np.int32), Rk=None, Rv=None, sm_scale=sm)
    for hq in range(Hq):
        Rvh = Rv[hq // g].astype(np.float64)
        assert np.max(np.abs(got[:, hq] - base[:, hq] @ Rvh.T)) <= 1e-12
    # the rotated-basis evaluation equals the original-basis brute force
    brute = oracle.decode_brute(pages, d=D, Hkv=Hkv, P=P, G=32, q=q, block_table=table,
                                seq_lens=np.array(lens, np.int32), Rk=Rk, Rv=Rv, sm_scale=sm)
    assert np.max(np.abs(got - brute)) <= 1e-12
    # equal matrices per head = the shared matrix
    R1 = W.rotation(43)
    same = _cache(np.stack([R1] * Hkv), np.stack([R1] * Hkv), kb, vb, table, lens, Hkv)
    assert np.array_equal(same, _cache(R1, R1, kb, vb, table, lens, Hkv))
    with pytest.raises(ValueError):
        _cache(Rk, R1, kb, vb, table, lens, Hkv)   # mixed shared / per-head


def test_per_head_calibration_averages_to_the_shared_one():
    """The per-head C_Q, C_S are the GQA groups' averages, so their mean over the
    heads is the shared (GQA-averaged) covariance; each head's rotation passes
    Lemma 1 against its own covariance."""
    rng = np.random.default_rng(47)
    T, Hq, Hkv = 150, 6, 3
    q = W.f32_to_bf16_bits((rng.standard_normal((T, Hq, D)) * np.linspace(0.2, 3, D)).astype(np.float32))
    k = W.f32_to_bf16_bits(rng.standard_normal((T, Hkv, D)).astype(np.float32))
    v = W.f32_to_bf16_bits(rng.standard_normal((T, Hkv, D)).astype(np.float32))
    ph = oracle.calibrate(q, k, v, per_head=True)
    sh = oracle.calibrate(q, k, v)
    for key in ("C_Q", "C_S"):
        assert ph[key].shape == (Hkv, D, D)
        assert np.max(np.abs(ph[key].mean(axis=0) - sh[key])) <= 1e-13 * np.max(np.abs(sh[key]))
    for h in range(Hkv):
        R, C = ph["R_K"][h], ph["C_Q"][h]
        dg = np.diag(R.T @ C @ R)
        assert np.max(np.abs(dg - np.trace(C) / D)) <= 1e-12 * np.trace(C)
    assert ph["R_K32"].shape == (Hkv, D, D) and ph["c_K"] in oracle.default_clip_candidates()
