"""GPU parity of the offline calibration (Sec. 3 "Algorithm Design: Offline
Calibration and Justification"; Alg. 1 Calibrate) against the oracle, through
the C ABI.

Tolerances (derived in the design notes, observed values logged):
  * C_Q: exact bf16 products summed in fp32 within a block's rows (<= 1024) and
    in fp64 across blocks: |dC_ij| <= 1024 * 2^-24 * sqrt(C_ii C_jj).
  * attention rows: fp32 score and probability sums, probabilities carried with
    16 significant bits into the value product: |dO| <= 5e-5 max|v| (2e-4 at
    the 8878-token size).
  * C_S: |dC_ij| <= 4e-4 sqrt(C_ii C_jj).
  * eigen-decomposition on identical inputs: |dlam| <= 1e-12 lam_max;
    eigenvector k within 1e-12 lam_max / gap_k (+1e-13); R = U H_Had P_br of the
    GPU's U bit-exact with the oracle's composition; R32 its rounding.
  * clip errors on identical inputs: relative 1e-12; the chosen ratio equal
    unless the oracle's two smallest errors are within 1e-9.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2605_17757_amd as ok
import workloads as W
from helpers import bits, log

pytestmark = pytest.mark.gpu

D = 128
U24 = 2.0 ** -24


def _acts(T, Hq, Hkv, seed):
    return W.calib_activations(T, Hq, Hkv, seed)


def _cov_tol(C, factor):
    dg = np.sqrt(np.abs(np.diag(C)))
    return factor * np.outer(dg, dg) + 1e-300


# ---------------------------------------------------------------------------
# C_Q
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T,Hq,Hkv", [(1, 4, 1), (77, 32, 8), (1000, 12, 4), (513, 6, 6)])
def test_query_cov(T, Hq, Hkv):
    q, _, _ = _acts(T, Hq, Hkv, 100 + T)
    C = ok.calib_query_cov(q.cuda(), Hkv).cpu().numpy()
    ref = oracle.query_cov(bits(q), Hkv)
    err = np.abs(C - ref)
    log("C_Q T=%d %d/%d: max|dC| %.3g (max|C| %.3g)" % (T, Hq, Hkv, err.max(), np.abs(ref).max()))
    assert np.all(err <= _cov_tol(ref, 1024 * U24))
    assert np.array_equal(C, C.T)


# ---------------------------------------------------------------------------
# attention rows and C_S
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("T,Hq,Hkv", [(1, 4, 1), (63, 8, 2), (64, 4, 4), (65, 32, 8),
                                      (300, 12, 4), (257, 3, 1)])
def test_attn_rows(causal, T, Hq, Hkv):
    q, k, v = _acts(T, Hq, Hkv, 200 + T + Hq)
    o = ok.calib_attn(q.cuda(), k.cuda(), v.cuda(), causal=causal).cpu().numpy()
    ref = oracle.attn_rows(bits(q), bits(k), bits(v), causal=causal)
    vmax = float(v.float().abs().max())
    err = float(np.abs(o - ref).max())
    log("attn T=%d %d/%d causal=%d: max|dO| %.3g (max|v| %.3g)" % (T, Hq, Hkv, causal, err, vmax))
    assert err <= 5e-5 * vmax


@pytest.mark.parametrize("causal", [True, False])
def test_score_cov(causal):
    T, Hq, Hkv = 333, 8, 2
    q, k, v = _acts(T, Hq, Hkv, 300)
    C = ok.calib_score_cov(q.cuda(), k.cuda(), v.cuda(), causal=causal).cpu().numpy()
    ref = oracle.score_cov(bits(q), bits(k), bits(v), causal=causal)
    err = np.abs(C - ref)
    log("C_S causal=%d: max|dC| %.3g (max|C| %.3g)" % (causal, err.max(), np.abs(ref).max()))
    assert np.all(err <= _cov_tol(ref, 4e-4))
    assert np.array_equal(C, C.T)


# ---------------------------------------------------------------------------
# eigen-decomposition and composition (identical fp64 inputs)
# ---------------------------------------------------------------------------

def _check_rotation(C, got, idx=0):
    lam = got["lam"][idx].cpu().numpy()
    U = got["U"][idx].cpu().numpy()
    R64 = got["R64"][idx].cpu().numpy()
    R32 = got["R32"][idx].cpu().numpy()
    info = int(got["info"][idx])
    assert info >= 1
    lam_o, U_o = oracle.eigh_desc(C)
    lmax = max(abs(lam_o[0]), abs(lam_o[-1]), 1e-300)
    assert np.max(np.abs(lam - lam_o)) <= 1e-12 * lmax
    assert np.all(np.diff(lam) <= 0)
    # validity: eigen-equation, orthonormality, sign rule
    assert np.max(np.abs(C @ U - U * lam[None, :])) <= 1e-12 * lmax
    assert np.max(np.abs(U.T @ U - np.eye(D))) <= 1e-12
    amax = np.argmax(np.abs(U), axis=0)
    assert np.all(U[amax, np.arange(D)] > 0)
    # each eigenvector within its perturbation bound
    worst = 0.0
    for j in range(D):
        gap = np.min(np.abs(np.delete(lam_o, j) - lam_o[j]))
        if gap <= 1e-9 * lmax:
            continue  # part of a cluster: checked through the projector below
        e = np.max(np.abs(U[:, j] - U_o[:, j]))
        worst = max(worst, e / (1e-12 * lmax / gap + 1e-13))
        assert e <= 1e-12 * lmax / gap + 1e-13, (j, e, gap)
    # the composition of the GPU's eigenvectors is the oracle's, bit for bit
    assert np.array_equal(R64, oracle.compose(U))
    assert np.array_equal(R32, R64.astype(np.float32))
    return info, worst


def test_rotation_of_a_query_covariance():
    q, _, _ = _acts(2000, 8, 2, 400)
    C = oracle.query_cov(bits(q), 2)
    got = ok.calib_rotation(torch.from_numpy(C).cuda())
    torch.cuda.synchronize()
    info, worst = _check_rotation(C, got)
    log("rotation: sweeps %d, worst eigenvector error / bound %.3g" % (info, worst))


def test_rotation_batch_special_matrices():
    rng = np.random.default_rng(5)
    diag = np.diag(rng.permutation(np.arange(1.0, D + 1.0)))     # distinct diagonal
    A = rng.standard_normal((D, D))
    sym = (A + A.T) / 2                                          # indefinite
    B, _ = np.linalg.qr(rng.standard_normal((D, D)))
    lam = np.concatenate([[9.0, 9.0, 9.0], np.linspace(5.0, 0.5, D - 3)])
    clus = (B * lam[None, :]) @ B.T                               # a 3-fold eigenvalue
    Cs = np.stack([diag, sym, clus, np.eye(D), np.zeros((D, D))])
    got = ok.calib_rotation(torch.from_numpy(Cs).cuda())
    torch.cuda.synchronize()
    _check_rotation(diag, got, 0)
    assert np.array_equal(got["U"][0].cpu().numpy(), np.eye(D)[:, np.argsort(-np.diag(diag), kind="stable")])
    _check_rotation(sym, got, 1)
    _check_rotation(clus, got, 2)
    # the cluster's invariant subspace: projector onto the first three vectors
    U = got["U"][2].cpu().numpy()
    Pj = U[:, :3] @ U[:, :3].T
    assert np.max(np.abs(Pj - B[:, :3] @ B[:, :3].T)) <= 1e-12
    # identity and zero: no rotation, U = I
    for i in (3, 4):
        assert np.array_equal(got["U"][i].cpu().numpy(), np.eye(D))
        assert int(got["info"][i]) == 1
    assert np.array_equal(got["lam"][3].cpu().numpy(), np.ones(D))
    assert np.array_equal(got["lam"][4].cpu().numpy(), np.zeros(D))


# ---------------------------------------------------------------------------
# clip calibration (identical rows and rotation)
# ---------------------------------------------------------------------------

# name -> (meta, clip mode, G)
FORMATS = {"default": (0, 0, 32), "paper_format": (1, 1, 128), "g64_bf16": (1, 0, 64)}


@pytest.mark.parametrize("fmt", list(FORMATS))
@pytest.mark.parametrize("rotate", [True, False])
def test_clip_errors(fmt, rotate):
    meta, clip, G = FORMATS[fmt]
    T, Hkv = 97, 3
    _, k, _ = _acts(T, 3, Hkv, 500)
    R = W.rotation(501, compose=True) if rotate else None
    cands = oracle.default_clip_candidates()
    lay = ok.Layout(num_kv_heads=Hkv, num_pages=1, group_size=G, clip_mode=clip, meta_dtype=meta)
    err, best = ok.calib_clip(lay, k.cuda(), None if R is None else torch.from_numpy(R).cuda(),
                              torch.from_numpy(cands).cuda())
    err = err.cpu().numpy()
    ref = oracle.clip_errors(bits(k), R, G=G, cands=cands, meta=meta, clip=clip)
    rel = float(np.max(np.abs(err - ref) / ref))
    log("clip %s rotate=%d: max rel %.3g, best %.2f (oracle %.2f)" % (
        fmt, rotate, rel, float(best), cands[np.argmin(ref)]))
    assert rel <= 1e-12
    srt = np.sort(ref)
    if srt[1] - srt[0] > 1e-9 * srt[0]:
        assert float(best) == float(cands[np.argmin(ref)])


# ---------------------------------------------------------------------------
# the whole layer
# ---------------------------------------------------------------------------

def _layer_checks(cal, q, k, v, T, Hq, Hkv, lay_args, causal, full):
    """Compare oscar_calibrate_layer with the oracle: C_Q-derived quantities
    through their bounds, R's orthogonality and Lemma 1, the spectra, and the
    clip choice on the GPU's own rotations."""
    meta, clip, G = lay_args
    Rk = cal["R_K"].cpu().numpy().astype(np.float64)
    Rv = cal["R_V"].cpu().numpy().astype(np.float64)
    lam = cal["lam"].cpu().numpy()
    info = cal["info"].cpu().numpy()
    assert np.all(info >= 1)
    for R in (Rk, Rv):
        assert np.max(np.abs(R.T @ R - np.eye(D))) <= 2e-6
    CQ = oracle.query_cov(bits(q), Hkv)
    lq, _ = oracle.eigh_desc(CQ)
    assert np.max(np.abs(lam[0] - lq)) <= 1024 * U24 * D * lq[0]
    dg = np.diag(Rk.T @ CQ @ Rk)                       # Lemma 1 on the result
    assert np.max(np.abs(dg - np.trace(CQ) / D)) <= 1e-5 * np.trace(CQ)
    if not full:
        CS = oracle.score_cov(bits(q), bits(k), bits(v), causal=causal)
        ls, _ = oracle.eigh_desc(CS)
        assert np.max(np.abs(lam[1] - ls)) <= 4e-4 * D * ls[0]
    cands = oracle.default_clip_candidates()
    for x, R, c in ((k, cal["R_K"], cal["clip"][0]), (v, cal["R_V"], cal["clip"][1])):
        ref = oracle.clip_errors(bits(x), R.cpu().numpy(), G=G, cands=cands, meta=meta, clip=clip)
        srt = np.sort(ref)
        log("  clip %.2f (oracle on the GPU's R: %.2f)" % (float(c), cands[np.argmin(ref)]))
        if srt[1] - srt[0] > 1e-9 * srt[0]:
            assert float(c) == float(cands[np.argmin(ref)])


def test_calibrate_layer_small():
    T, Hq, Hkv = 300, 8, 2
    q, k, v = _acts(T, Hq, Hkv, 600)
    lay = ok.Layout(num_kv_heads=Hkv, num_pages=1)
    cal = ok.calibrate_layer(lay, q.cuda(), k.cuda(), v.cuda(),
                             torch.from_numpy(oracle.default_clip_candidates()).cuda())
    torch.cuda.synchronize()
    _layer_checks(cal, q, k, v, T, Hq, Hkv, (0, 0, 32), True, False)
    # against the oracle's own calibration: the top eigenvectors through R_K
    ora = oracle.calibrate(bits(q), bits(k), bits(v), causal=True)
    HP = oracle.compose(np.eye(D))                      # R = U (H P_br)
    Ug = cal["R_K"].cpu().numpy().astype(np.float64) @ HP.T
    lq = ora["lam_Q"]
    for j in range(4):
        gap = min(lq[j - 1] - lq[j] if j else np.inf, lq[j] - lq[j + 1])
        e = np.max(np.abs(Ug[:, j] - ora["U_Q"][:, j]))
        assert e <= 1024 * U24 * D * lq[0] / gap + 1e-6, (j, e)


def test_calibrate_layer_paper_format_and_full_size_sampled():
    """The bench workload: 8878 calibration tokens of a Qwen3-8B-shaped layer
    (32/8 heads), the paper's quantizer format (G = 128, bf16 scale/zero,
    per-token quantile clip).  Attention rows sampled against the oracle; C_S
    against the fp64 second moment of the GPU's own rows; the rotations and the
    clip choice against the oracle on the GPU's covariances and rotations."""
    T, Hq, Hkv = W.CALIB_TOKENS, 32, 8
    meta, clip, G = FORMATS["paper_format"]
    q, k, v = _acts(T, Hq, Hkv, 700)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    lay = ok.Layout(num_kv_heads=Hkv, num_pages=1, group_size=G, clip_mode=clip, meta_dtype=meta)
    cands_np = oracle.default_clip_candidates()
    cal = ok.calibrate_layer(lay, qd, kd, vd, torch.from_numpy(cands_np).cuda())
    torch.cuda.synchronize()
    log("full size: calibrated, sweeps", cal["info"].tolist(), "clip", cal["clip"].tolist())
    # attention rows at sampled (t, head)
    o = ok.calib_attn(qd, kd, vd, causal=True)
    torch.cuda.synchronize()
    ts = [0, 1, 63, 64, 127, 128, 4095, 4096, T // 2, T - 65, T - 2, T - 1]
    pairs = np.array([(t, h) for t in ts for h in (0, 5, 31)], np.int32)
    ref = oracle.attn_rows(bits(q), bits(k), bits(v), causal=True, pairs=pairs)
    got = o[torch.from_numpy(pairs[:, 0]).long().cuda(), torch.from_numpy(pairs[:, 1]).long().cuda()]
    vmax = float(v.float().abs().max())
    err = float(np.abs(got.cpu().numpy() - ref).max())
    log("  attn rows: max|dO| %.3g over %d rows (max|v| %.3g)" % (err, len(pairs), vmax))
    assert err <= 2e-4 * vmax
    # C_S = the fp64 second moment of the GPU rows
    CS = ok.calib_score_cov(qd, kd, vd, causal=True).cpu().numpy()
    O = o.double().reshape(-1, D)
    CS_ref = (O.T @ O / O.shape[0]).cpu().numpy()
    assert np.all(np.abs(CS - CS_ref) <= _cov_tol(CS_ref, 1024 * U24))
    del O, o
    # rotations from the GPU's own C_Q and C_S
    CQ = ok.calib_query_cov(qd, Hkv)
    rot = ok.calib_rotation(torch.stack([CQ, torch.from_numpy(CS).cuda()]))
    torch.cuda.synchronize()
    for i, C in enumerate((CQ.cpu().numpy(), CS)):
        _check_rotation(C, rot, i)
    assert torch.equal(rot["R32"][0], cal["R_K"]) and torch.equal(rot["R32"][1], cal["R_V"])
    _layer_checks(cal, q, k, v, T, Hq, Hkv, (meta, clip, G), True, True)


def test_calibrate_layer_one_rotation_per_kv_head():
    """L->rot_per_head: each KV head's C_Q and C_S over its own query heads, its own
    R_K and R_V, one clip ratio per tensor over all heads' rows."""
    T, Hq, Hkv = 300, 8, 2
    q, k, v = _acts(T, Hq, Hkv, 650)
    lay = ok.Layout(num_kv_heads=Hkv, num_pages=1, rot_per_head=1)
    cands_np = oracle.default_clip_candidates()
    cal = ok.calibrate_layer(lay, q.cuda(), k.cuda(), v.cuda(), torch.from_numpy(cands_np).cuda())
    torch.cuda.synchronize()
    ora = oracle.calibrate(bits(q), bits(k), bits(v), per_head=True)
    Rk = cal["R_K"].cpu().numpy().astype(np.float64)
    Rv = cal["R_V"].cpu().numpy().astype(np.float64)
    lam = cal["lam"].cpu().numpy()
    assert Rk.shape == (Hkv, D, D) and lam.shape == (2, Hkv, D)
    assert np.all(cal["info"].cpu().numpy() >= 1)
    for h in range(Hkv):
        for R in (Rk[h], Rv[h]):
            assert np.max(np.abs(R.T @ R - np.eye(D))) <= 2e-6
        lq = ora["lam_Q"][h]
        assert np.max(np.abs(lam[0, h] - lq)) <= 1024 * U24 * D * lq[0]
        ls = ora["lam_S"][h]
        assert np.max(np.abs(lam[1, h] - ls)) <= 4e-4 * D * ls[0]
        C = ora["C_Q"][h]
        dg = np.diag(Rk[h].T @ C @ Rk[h])                  # Lemma 1, head by head
        assert np.max(np.abs(dg - np.trace(C) / D)) <= 1e-5 * np.trace(C)
    for x, R, c in ((k, cal["R_K"], cal["clip"][0]), (v, cal["R_V"], cal["clip"][1])):
        ref = oracle.clip_errors(bits(x), R.cpu().numpy(), G=32, cands=cands_np)
        srt = np.sort(ref)
        log("  per-head clip %.2f (oracle on the GPU's R: %.2f)" % (float(c), cands_np[np.argmin(ref)]))
        if srt[1] - srt[0] > 1e-9 * srt[0]:
            assert float(c) == float(cands_np[np.argmin(ref)])
