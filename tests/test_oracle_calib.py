"""Pins of the calibration oracle (Sec. 3 "Algorithm Design: Offline Calibration
and Justification"; App. "Hadamard transform", "P_K" and the worked example;
Alg. 1 Calibrate) against what the paper and the mathematics fix:

* the Walsh-Hadamard and bit-reversal factors against the worked example's
  printed rows (Step 1 -> Step 2 -> Step 3), the printed top-8 placement and the
  closed form H[i][j] = (-1)^popcount(i & j) / sqrt(d);
* Lemma 1 (Hadamard conjugation equalizes the diagonal) on the whole chain
  C -> eigenvectors -> R = U H P_br, which fails for a transposed or non-eigen U,
  a wrong normalization or a wrong Hadamard;
* C_Q against the trace identity and a matrix product, and an exactly diagonal
  C_Q whose composed rotation has a closed form;
* attention rows and C_S against torch's scaled-dot-product attention (fp64,
  causal and not, GQA head map), against uniform attention (prefix means) and
  T = 1;
* clip errors against hand-computed binary16 quantization of small rows and an
  exactly representable grid (zero error).
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example_layer10_token5.txt")
PRINT_TOL = 0.02  # two-decimal printing: see test_oracle_pins


def _golden():
    rows = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        name, *vals = line.split()
        rows[name] = np.array([float(v) for v in vals], np.float64)
    return rows


def _bf16(x):
    return W.f32_to_bf16_bits(np.asarray(x, np.float32))


def _f(bits):
    return W.bf16_bits_to_f32(bits).astype(np.float64)


# ---------------------------------------------------------------------------
# H_Had, P_br, R = U H P_br
# ---------------------------------------------------------------------------

def test_hadamard_closed_form_and_orthogonality():
    for d in (1, 2, 8, 128):
        H = oracle.hadamard(d)
        i, j = np.meshgrid(np.arange(d), np.arange(d), indexing="ij")
        pc = np.vectorize(lambda a: bin(a).count("1"))(i & j)
        assert np.max(np.abs(H - (-1.0) ** pc / math.sqrt(d))) <= 1e-15
        assert np.max(np.abs(H @ H.T - np.eye(d))) <= 1e-14
    with pytest.raises(ValueError):
        oracle.hadamard(96)


def test_worked_example_steps_through_oracle_factors():
    g = _golden()
    H, P = oracle.hadamard(128), oracle.bit_reversal(128)
    assert np.max(np.abs(g["step1_k_uq"] @ H - g["step2_k_uq_h"])) <= PRINT_TOL
    assert np.max(np.abs(g["raw_k"] @ H - g["pure_hadamard_k_h"])) <= PRINT_TOL
    # P_br only moves printed values: exact
    assert np.array_equal(g["step2_k_uq_h"] @ P, g["step3_k_uq_h_pbr"])
    # R = U H P_br with U = I is H P_br: Step 1 -> Step 3 in one product
    assert np.max(np.abs(g["step1_k_uq"] @ oracle.compose(np.eye(128)) - g["step3_k_uq_h_pbr"])) \
        <= PRINT_TOL
    # printed placement: top-1..8 -> 0, 64, 32, 96, 16, 80, 48, 112
    assert [int(np.argmax(P[k])) for k in range(8)] == [0, 64, 32, 96, 16, 80, 48, 112]


def test_lemma1_on_the_composed_rotation():
    rng = np.random.default_rng(7)
    A = rng.standard_normal((128, 300)) * np.geomspace(10.0, 0.01, 128)[:, None]
    C = A @ A.T / 300
    lam, U = oracle.eigh_desc(C)
    R = oracle.compose(U)
    assert np.max(np.abs(R.T @ R - np.eye(128))) <= 1e-13
    dg = np.diag(R.T @ C @ R)
    assert np.max(np.abs(dg - np.trace(C) / 128)) <= 1e-12 * np.trace(C)
    # a transposed eigenbasis breaks it
    dg_bad = np.diag(oracle.compose(U.T).T @ C @ oracle.compose(U.T))
    assert np.max(np.abs(dg_bad - np.trace(C) / 128)) > 1e-3 * np.trace(C)


def test_eigh_desc_order_residual_and_sign_rule():
    rng = np.random.default_rng(3)
    A = rng.standard_normal((128, 128))
    C = A @ A.T
    lam, U = oracle.eigh_desc(C)
    assert np.all(np.diff(lam) <= 0)
    assert np.max(np.abs(C @ U - U * lam[None, :])) <= 1e-11 * lam[0]
    assert np.max(np.abs(U.T @ U - np.eye(128))) <= 1e-13
    idx = np.argmax(np.abs(U), axis=0)
    assert np.all(U[idx, np.arange(128)] > 0)
    # diagonal input: unit vectors in descending order
    d = np.array([3.0, 7.0, 1.0, 5.0])
    lam, U = oracle.eigh_desc(np.diag(d))
    assert np.array_equal(lam, [7.0, 5.0, 3.0, 1.0])
    assert np.array_equal(U, np.eye(4)[:, [1, 3, 0, 2]])


def test_diagonal_query_covariance_gives_closed_form_rotation():
    """Queries with one nonzero channel each: C_Q is exactly diagonal, so U_Q is
    the permutation sorting the channels by descending C_Q entry and
    R_K[pi(k)][bitrev(k')] = H[k][k'] = (-1)^popcount(k & k') / sqrt(d)."""
    d, T, Hq, Hkv = 128, 128, 4, 2
    rng = np.random.default_rng(11)
    amp = rng.permutation(np.arange(1, d + 1)).astype(np.float32) / 8.0  # distinct, bf16-exact
    q = np.zeros((T, Hq, d), np.float32)
    for t in range(T):
        for i in range(Hq):
            q[t, i, t] = amp[t]          # token t carries channel t in every head
    CQ = oracle.query_cov(_bf16(q), Hkv)
    assert np.array_equal(CQ, np.diag(amp.astype(np.float64) ** 2 / T))
    lam, U = oracle.eigh_desc(CQ)
    pi = np.argsort(-amp, kind="stable")
    assert np.array_equal(U, np.eye(d)[:, pi])
    R = oracle.compose(U)
    br = [int(format(k, "07b")[::-1], 2) for k in range(d)]
    pc = np.vectorize(lambda a: bin(a).count("1"))
    for k in range(d):
        expect = (-1.0) ** pc(k & np.arange(d)) / math.sqrt(d)
        assert np.max(np.abs(R[pi[k], br] - expect)) <= 1e-15


# ---------------------------------------------------------------------------
# C_Q
# ---------------------------------------------------------------------------

def test_query_cov_trace_product_symmetry_scaling():
    rng = np.random.default_rng(5)
    T, Hq, Hkv, d = 37, 6, 2, 128
    q = _bf16(rng.standard_normal((T, Hq, d)) * np.linspace(0.1, 3.0, d))
    C = oracle.query_cov(q, Hkv)
    x = _f(q).reshape(-1, d)
    assert abs(np.trace(C) - np.mean(np.sum(x * x, axis=1))) <= 1e-12 * np.trace(C)
    assert np.max(np.abs(C - x.T @ x / x.shape[0])) <= 1e-12 * np.max(np.abs(C))
    assert np.array_equal(C, C.T)
    assert np.min(np.linalg.eigvalsh(C)) >= -1e-12
    C2 = oracle.query_cov(_bf16(_f(q) * 2.0), Hkv)   # doubling is exact in bf16
    assert np.array_equal(C2, 4.0 * C)
    with pytest.raises(ValueError):
        oracle.query_cov(q, 4)                          # 6 heads do not split into 4 groups


# ---------------------------------------------------------------------------
# Attention rows and C_S
# ---------------------------------------------------------------------------

def _sdpa(q, k, v, causal):
    """torch's scaled-dot-product attention in fp64 on the CPU, GQA by repeating
    each KV head over its g query heads: [T, Hq, d]."""
    Hq, Hkv = q.shape[1], k.shape[1]
    qt = torch.from_numpy(_f(q)).permute(1, 0, 2)[None]
    kt = torch.from_numpy(_f(k)).permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0)[None]
    vt = torch.from_numpy(_f(v)).permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=causal)
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("Hq,Hkv", [(1, 1), (4, 2), (6, 2)])
def test_attn_rows_match_torch_sdpa(causal, Hq, Hkv):
    rng = np.random.default_rng(17 + Hq)
    T, d = 45, 128
    q = _bf16(rng.standard_normal((T, Hq, d)) * 2.0)
    k = _bf16(rng.standard_normal((T, Hkv, d)))
    v = _bf16(rng.standard_normal((T, Hkv, d)) + 0.5)
    o = oracle.attn_rows(q, k, v, causal=causal)
    assert np.max(np.abs(o - _sdpa(q, k, v, causal))) <= 1e-12
    pairs = np.array([[0, 0], [T - 1, Hq - 1], [T // 2, Hq // 2]], np.int32)
    assert np.array_equal(oracle.attn_rows(q, k, v, causal=causal, pairs=pairs),
                          o[pairs[:, 0], pairs[:, 1]])


def test_attn_rows_uniform_attention_and_single_token():
    rng = np.random.default_rng(23)
    T, d = 20, 128
    q = _bf16(np.zeros((T, 2, d)))
    k = _bf16(rng.standard_normal((T, 1, d)))
    v = _bf16(rng.standard_normal((T, 1, d)))
    vf = _f(v)[:, 0]
    prefix = np.cumsum(vf, axis=0) / np.arange(1, T + 1)[:, None]
    o = oracle.attn_rows(q, k, v, causal=True)
    assert np.max(np.abs(o[:, 0] - prefix)) <= 1e-14
    assert np.max(np.abs(o[:, 1] - prefix)) <= 1e-14
    o = oracle.attn_rows(q, k, v, causal=False)
    assert np.max(np.abs(o - vf.mean(axis=0)[None, None])) <= 1e-14
    o1 = oracle.attn_rows(q[:1], k[:1], v[:1], causal=True)
    assert np.array_equal(o1[0, 0], vf[0])


def test_score_cov_is_the_second_moment_of_sdpa_outputs():
    rng = np.random.default_rng(29)
    T, Hq, Hkv, d = 33, 4, 2, 128
    q = _bf16(rng.standard_normal((T, Hq, d)) * 1.5)
    k = _bf16(rng.standard_normal((T, Hkv, d)))
    v = _bf16(rng.standard_normal((T, Hkv, d)))
    for causal in (True, False):
        C = oracle.score_cov(q, k, v, causal=causal)
        o = _sdpa(q, k, v, causal).reshape(-1, d)
        assert np.max(np.abs(C - o.T @ o / o.shape[0])) <= 1e-12 * np.max(np.abs(C))
        assert np.array_equal(C, C.T)


# ---------------------------------------------------------------------------
# Clip errors
# ---------------------------------------------------------------------------

def _f16_rne(x: Fraction) -> Fraction:
    return Fraction(float(np.float16(float(x))))


def test_clip_errors_hand_computed_single_spike():
    """Row: channel 0 = 1, others 0 (G = 32, binary16 metadata, identity rotation).
    rho = 1: s = f16(1/3), z = 0, code 3, so x^ = 3 s.  rho = 1/2: tau = 1/2,
    s = f16(1/6), code 3, x^ = 3 s.  Other groups are constant zero (exact)."""
    x = np.zeros((1, 128), np.float32)
    x[0, 0] = 1.0
    err = oracle.clip_errors(_bf16(x), None, G=32, cands=[1.0, 0.5])
    for n, rho in enumerate([Fraction(1), Fraction(1, 2)]):
        s = _f16_rne(rho / 3)
        expect = (1 - 3 * s) ** 2 / 128
        assert err[n] == float(expect)


def test_clip_errors_zero_on_an_exact_grid_and_positive_when_clipped():
    # every group holds the four levels -1.5, -0.5, 0.5, 1.5: s = 1, z = 1.5 exact
    x = np.tile(np.array([-1.5, -0.5, 0.5, 1.5], np.float32), 32)[None, :]
    for G in (32, 64, 128):
        for meta in (0, 1):
            err = oracle.clip_errors(_bf16(x), None, G=G, cands=[1.0, 0.9], meta=meta)
            assert err[0] == 0.0 and err[1] > 0.0
    # the token-quantile clip at rho = 1 is the row's absmax: also exact
    err = oracle.clip_errors(_bf16(x), None, G=32, cands=[1.0], clip=1)
    assert err[0] == 0.0


def test_clip_errors_rotation_is_applied():
    """With a signed permutation as R the rotated row is the permuted row, so the
    error equals the identity-rotation error of the permuted input."""
    rng = np.random.default_rng(31)
    x = _bf16(rng.standard_normal((50, 128)) * 3.0)
    perm = rng.permutation(128)
    R = np.zeros((128, 128), np.float32)
    R[perm, np.arange(128)] = 1.0   # x~_j = x_{perm[j]}
    cands = oracle.default_clip_candidates()
    a = oracle.clip_errors(x, R, G=32, cands=cands)
    b = oracle.clip_errors(x[:, perm], None, G=32, cands=cands)
    assert np.array_equal(a, b)


def test_calibrate_recovers_a_planted_query_basis():
    """Queries with a planted covariance B diag(lambda) B^T (distinct, well
    separated top eigenvalues): the top eigenvectors of C_Q align with B's
    columns, lambda_Q estimates lambda, and R_K passes Lemma 1 against C_Q."""
    rng = np.random.default_rng(37)
    T, Hq, Hkv, d = 512, 8, 2, 128
    lam = np.concatenate([[100.0, 40.0, 15.0], np.geomspace(5.0, 0.05, d - 3)])
    B, _ = np.linalg.qr(rng.standard_normal((d, d)))
    z = rng.standard_normal((T * Hq, d)) * np.sqrt(lam)[None, :]
    q = _bf16((z @ B.T).reshape(T, Hq, d))
    k = _bf16(rng.standard_normal((T, Hkv, d)))
    v = _bf16(rng.standard_normal((T, Hkv, d)))
    cal = oracle.calibrate(q, k, v, causal=True)
    for j in range(3):
        assert abs(abs(cal["U_Q"][:, j] @ B[:, j]) - 1.0) <= 0.02
    assert abs(cal["lam_Q"][0] / lam[0] - 1.0) <= 0.1
    RK = cal["R_K"]
    dg = np.diag(RK.T @ cal["C_Q"] @ RK)
    assert np.max(np.abs(dg - np.trace(cal["C_Q"]) / d)) <= 1e-10 * np.trace(cal["C_Q"])
    assert cal["c_K"] in oracle.default_clip_candidates()
    assert np.array_equal(cal["R_K32"], RK.astype(np.float32))
