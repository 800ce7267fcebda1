"""OSCAR CPU oracle -- test infrastructure only.

Loads ``liboscar_oracle.so`` (plain C, fp64; see ``oscar_oracle.c``) through
ctypes and exposes numpy-in / numpy-out wrappers.  Only the test suite, the
package smoke check and the benchmark's CPU-baseline leg use this module; the
GPU library never imports or links it.

What it computes (arXiv 2605.17757):
  * ``kv_append``     -- rotate, clip, asymmetric-INT2 quantize and pack new K/V
                         rows (Sec. 4 "KV Cache Update"; App. "Scale
                         Determination and Per-token Clipping Details").
  * ``decode``        -- attention over the packed cache, fp64, rotated basis
                         (Alg. 1 DecodeStep; Sec. 2 attention).
  * ``decode_brute``  -- the same in the original basis (dequantize, rotate back,
                         plain softmax attention); tiny inputs only.
  * ``bf16_decode``   -- plain fp64 attention over a bf16 paged cache.
  * ``seg_write``, ``mixed_update``, ``decode_mixed`` -- the mixed-precision
                         cache of Sec. 4 "KV Cache Layout": bf16 sink and recent
                         window around the INT2 history, the per-step demotion of
                         the oldest window token (Alg. 1 DecodeStep) and decode
                         attention over all three segments.
  * ``query_cov``, ``attn_rows``, ``score_cov``, ``hadamard``, ``bit_reversal``,
    ``compose``, ``eigh_desc``, ``clip_errors``, ``calibrate`` -- the offline
                         calibration of Sec. 3 and Alg. 1 Calibrate: the
                         GQA-averaged query covariance C_Q, the score-aware value
                         covariance C_S = V^T S^T S V / N, their eigenvectors
                         (descending, sign fixed), R = U H_Had P_br, and the clip
                         ratio with the smallest quantization error of the
                         rotated rows.

Quantizer variants (keyword arguments, defaults = the hot path's format):
``meta`` 0/1 stores scale and zero as binary16 / bfloat16; ``clip`` 0/1 takes the
clip threshold as ratio x group absmax / the token's ratio-quantile of |x~| (App.
"Scale Determination and Per-token Clipping Details"); ``G`` any divisor of d; a
rotation of ``None`` is the identity.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oscar_oracle.c")
_LIB = os.path.join(_HERE, "liboscar_oracle.so")

CFLAGS = ["-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
          "-fPIC", "-shared", "-Wall", "-Wno-unused-function"]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (IEEE arithmetic, no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f32, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_float, ctypes.c_double
        L.oracle_page_head_bytes.restype = ctypes.c_size_t
        L.oracle_page_head_bytes.argtypes = [i32, i32, i32]
        L.oracle_rotate_row.argtypes = [P, P, i32, P]
        L.oracle_quantize_row.restype = i32
        L.oracle_quantize_row.argtypes = [P, i32, i32, f32, i32, i32, P, P, P]
        L.oracle_token_quantile.restype = f32
        L.oracle_token_quantile.argtypes = [P, i32, f32]
        L.oracle_kv_append.restype = i64
        L.oracle_kv_append.argtypes = [i32, i32, i32, i32, i32, i32, i64, P, P, P, P, i32, P, P,
                                       f32, f32, i32]
        L.oracle_read_token.argtypes = [i32, i32, i32, i32, P, i64, i32, i32, i32, P, P, P]
        L.oracle_decode.restype = i32
        L.oracle_decode.argtypes = [i32, i32, i32, i32, i32, i64, P, P, i32, i32, P, i32, P, P,
                                    P, f64, P, i32, P, i32]
        L.oracle_decode_brute.restype = i32
        L.oracle_decode_brute.argtypes = [i32, i32, i32, i32, i32, i64, P, P, i32, i32, P, i32,
                                          P, P, P, f64, P, i32]
        L.oracle_bf16_decode.restype = i32
        L.oracle_bf16_decode.argtypes = [i32, i32, i32, i64, P, P, i32, i32, P, i32, P, f64,
                                         P, i32, P]
        L.oracle_bf16_append.restype = i32
        L.oracle_bf16_append.argtypes = [i32, i32, i32, i64, P, P, P, P, i32]
        L.oracle_f32_to_f16_rne.restype = ctypes.c_uint16
        L.oracle_f32_to_f16_rne.argtypes = [f32]
        L.oracle_f16_to_f32.restype = f32
        L.oracle_f16_to_f32.argtypes = [ctypes.c_uint16]
        L.oracle_bf16_to_f32.restype = f32
        L.oracle_bf16_to_f32.argtypes = [ctypes.c_uint16]
        L.oracle_f32_to_bf16_rne.restype = ctypes.c_uint16
        L.oracle_f32_to_bf16_rne.argtypes = [f32]
        L.oracle_seg_write.restype = i32
        L.oracle_seg_write.argtypes = [i32, i32, i32, i32, i32, P, P, P, P, P, i32]
        L.oracle_mixed_update.restype = i64
        L.oracle_mixed_update.argtypes = [i32, i32, i32, i32, i32, i32, i64, P, P, i32, i32, i32,
                                          P, P, P, i32, P, P, P, f32, f32, i32]
        L.oracle_decode_mixed.restype = i32
        L.oracle_decode_mixed.argtypes = [i32, i32, i32, i32, i32, i64, P, P, i32, i32, P, i32,
                                          i32, P, i32, P, P, P, f64, P, i32, P, i32]
        L.oracle_query_cov.restype = i32
        L.oracle_query_cov.argtypes = [P, i64, i32, i32, i32, P]
        L.oracle_attn_rows.restype = i32
        L.oracle_attn_rows.argtypes = [P, P, P, i64, i32, i32, i32, i32, P, i64, P]
        L.oracle_score_cov.restype = i32
        L.oracle_score_cov.argtypes = [P, P, P, i64, i32, i32, i32, i32, P]
        L.oracle_hadamard.restype = i32
        L.oracle_hadamard.argtypes = [i32, P]
        L.oracle_bit_reversal.restype = i32
        L.oracle_bit_reversal.argtypes = [i32, P]
        L.oracle_compose.restype = i32
        L.oracle_compose.argtypes = [P, i32, P]
        L.oracle_clip_errors.restype = i32
        L.oracle_clip_errors.argtypes = [P, i64, i32, P, i32, i32, i32, P, i32, P, i32, i32]
        L.oracle_num_threads.restype = i32
        L.oracle_set_num_threads.restype = None
        L.oracle_set_num_threads.argtypes = [i32]
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _rot(R):
    """fp32 rotation matrix pointer, or NULL (identity) for None."""
    if R is None:
        return None, None
    a = _c(R, np.float32)
    return a, _ptr(a)


def _rph(*Rs) -> int:
    """1 when the rotations are per KV head ([Hkv, d, d]), 0 when shared ([d, d]);
    None entries (identity) take either form."""
    kinds = {np.ndim(R) for R in Rs if R is not None}
    if len(kinds) > 1:
        raise ValueError("R_k and R_v must both be shared [d, d] or both per head [Hkv, d, d]")
    return int(kinds == {3})


def num_threads() -> int:
    return int(lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Thread count of the oracle's parallel loops from here on (timing only)."""
    lib().oracle_set_num_threads(int(n))


def page_head_bytes(d: int, P: int, G: int) -> int:
    return int(lib().oracle_page_head_bytes(d, P, G))


def f32_to_f16_bits(x: float) -> int:
    return int(lib().oracle_f32_to_f16_rne(float(x)))


def f16_bits_to_f32(h: int) -> float:
    return float(lib().oracle_f16_to_f32(int(h)))


def f32_to_bf16_bits(x: float) -> int:
    return int(lib().oracle_f32_to_bf16_rne(float(x)))


def bf16_bits_to_f32(h: int) -> float:
    return float(lib().oracle_bf16_to_f32(int(h)))


def token_quantile(xt: np.ndarray, rho: float) -> float:
    """The per-token clip threshold: rho-quantile of |x~| over the row (linear
    interpolation of order statistics, fp32 steps)."""
    xt = _c(xt, np.float32)
    return float(lib().oracle_token_quantile(_ptr(xt), xt.shape[0], float(rho)))


def rotate_row(x: np.ndarray, R) -> np.ndarray:
    """x~ = x R (fp64 accumulation, one rounding to fp32); R None = identity."""
    x = _c(x, np.float32)
    Ra, Rp = _rot(R)
    d = x.shape[0]
    out = np.empty(d, np.float32)
    lib().oracle_rotate_row(_ptr(x), Rp, d, _ptr(out))
    return out


def quantize_row(xt: np.ndarray, G: int, rho: float, *, meta: int = 0, clip: int = 0):
    """Clip + asymmetric INT2 of one rotated row -> (codes[d], s16[d/G], z16[d/G], n_sat)."""
    xt = _c(xt, np.float32)
    d = xt.shape[0]
    codes = np.zeros(d, np.uint8)
    s16 = np.zeros(d // G, np.uint16)
    z16 = np.zeros(d // G, np.uint16)
    sat = lib().oracle_quantize_row(_ptr(xt), d, G, float(rho), int(meta), int(clip),
                                    _ptr(codes), _ptr(s16), _ptr(z16))
    return codes, s16, z16, int(sat)


def kv_append(pages: np.ndarray, *, d: int, Hkv: int, P: int, G: int, k: np.ndarray,
              v: np.ndarray, slot_mapping: np.ndarray, Rk, Rv, clip_k: float, clip_v: float,
              meta: int = 0, clip: int = 0) -> int:
    """Quantize rows into ``pages`` (uint8, modified in place).  Returns the
    number of saturated metadata stores."""
    assert pages.dtype == np.uint8 and pages.flags["C_CONTIGUOUS"]
    k = _c(k, np.uint16)
    v = _c(v, np.uint16)
    slots = _c(slot_mapping, np.int64)
    n_tok = slots.shape[0]
    assert k.size == n_tok * Hkv * d and v.size == n_tok * Hkv * d
    num_pages = pages.size // (Hkv * page_head_bytes(d, P, G))
    Rka, Rkp = _rot(Rk)
    Rva, Rvp = _rot(Rv)
    rc = lib().oracle_kv_append(d, Hkv, P, G, int(meta), int(clip), num_pages, _ptr(pages),
                                _ptr(k), _ptr(v), _ptr(slots), n_tok, Rkp, Rvp, float(clip_k),
                                float(clip_v), _rph(Rk, Rv))
    if rc < 0:
        raise ValueError("oracle kv_append: slot outside the page pool")
    return int(rc)


def read_token(pages: np.ndarray, *, d: int, Hkv: int, P: int, G: int, page: int, h: int,
               t: int, is_v: bool):
    codes = np.zeros(d, np.uint8)
    s16 = np.zeros(d // G, np.uint16)
    z16 = np.zeros(d // G, np.uint16)
    lib().oracle_read_token(d, Hkv, P, G, _ptr(pages), page, h, t, int(is_v), _ptr(codes),
                            _ptr(s16), _ptr(z16))
    return codes, s16, z16


def decode(pages: np.ndarray, *, d: int, Hkv: int, P: int, G: int, q: np.ndarray,
           block_table: np.ndarray, seq_lens: np.ndarray, Rk, Rv, sm_scale: float, pairs=None,
           meta: int = 0) -> np.ndarray:
    """fp64 decode attention.  q: bf16 bits [B, Hq, d].  Returns [B, Hq, d], or
    [n_pairs, d] when ``pairs`` (an [n, 2] array of (b, h)) is given."""
    q = _c(q, np.uint16)
    B, Hq = q.shape[0], q.shape[1]
    bt = _c(block_table, np.int32)
    sl = _c(seq_lens, np.int32)
    num_pages = pages.size // (Hkv * page_head_bytes(d, P, G))
    if pairs is None:
        out = np.zeros((B, Hq, d), np.float64)
        pp, n = None, 0
    else:
        pr = _c(pairs, np.int32).reshape(-1, 2)
        out = np.zeros((pr.shape[0], d), np.float64)
        pp, n = _ptr(pr), pr.shape[0]
    Rka, Rkp = _rot(Rk)
    Rva, Rvp = _rot(Rv)
    rc = lib().oracle_decode(d, Hkv, P, G, int(meta), num_pages, _ptr(pages), _ptr(q), B, Hq,
                             _ptr(bt), bt.shape[1], _ptr(sl), Rkp, Rvp, float(sm_scale), pp, n,
                             _ptr(out), _rph(Rk, Rv))
    if rc:
        raise ValueError("oracle decode: bad page id, length or head")
    return out


def decode_brute(pages: np.ndarray, *, d: int, Hkv: int, P: int, G: int, q: np.ndarray,
                 block_table: np.ndarray, seq_lens: np.ndarray, Rk, Rv, sm_scale: float,
                 meta: int = 0) -> np.ndarray:
    q = _c(q, np.uint16)
    B, Hq = q.shape[0], q.shape[1]
    bt = _c(block_table, np.int32)
    sl = _c(seq_lens, np.int32)
    num_pages = pages.size // (Hkv * page_head_bytes(d, P, G))
    out = np.zeros((B, Hq, d), np.float64)
    Rka, Rkp = _rot(Rk)
    Rva, Rvp = _rot(Rv)
    rc = lib().oracle_decode_brute(d, Hkv, P, G, int(meta), num_pages, _ptr(pages), _ptr(q), B,
                                   Hq, _ptr(bt), bt.shape[1], _ptr(sl), Rkp, Rvp, float(sm_scale),
                                   _ptr(out), _rph(Rk, Rv))
    if rc:
        raise ValueError("oracle decode_brute: bad page id or length")
    return out


def bf16_append(pages: np.ndarray, *, d: int, Hkv: int, P: int, k: np.ndarray, v: np.ndarray,
                slot_mapping: np.ndarray) -> None:
    assert pages.dtype == np.uint16 and pages.flags["C_CONTIGUOUS"]
    slots = _c(slot_mapping, np.int64)
    num_pages = pages.size // (Hkv * 2 * P * d)
    rc = lib().oracle_bf16_append(d, Hkv, P, num_pages, _ptr(pages), _ptr(_c(k, np.uint16)),
                                  _ptr(_c(v, np.uint16)), _ptr(slots), slots.shape[0])
    if rc:
        raise ValueError("oracle bf16_append: slot outside the page pool")


def bf16_decode(pages: np.ndarray, *, d: int, Hkv: int, P: int, q: np.ndarray,
                block_table: np.ndarray, seq_lens: np.ndarray, sm_scale: float,
                pairs=None) -> np.ndarray:
    q = _c(q, np.uint16)
    B, Hq = q.shape[0], q.shape[1]
    bt = _c(block_table, np.int32)
    sl = _c(seq_lens, np.int32)
    num_pages = pages.size // (Hkv * 2 * P * d)
    if pairs is None:
        out = np.zeros((B, Hq, d), np.float64)
        pp, n = None, 0
    else:
        pr = _c(pairs, np.int32).reshape(-1, 2)
        out = np.zeros((pr.shape[0], d), np.float64)
        pp, n = _ptr(pr), pr.shape[0]
    rc = lib().oracle_bf16_decode(d, Hkv, P, num_pages, _ptr(pages), _ptr(q), B, Hq, _ptr(bt),
                                  bt.shape[1], _ptr(sl), float(sm_scale), pp, n, _ptr(out))
    if rc:
        raise ValueError("oracle bf16_decode: bad page id, length or head")
    return out


def seg_elems(*, d: int, Hkv: int, B: int, S0: int, W: int) -> int:
    """bf16 elements of the segment store: [B][Hkv][K, V][S0 + W][d]."""
    return B * Hkv * 2 * (S0 + W) * d


def seg_write(seg: np.ndarray, *, d: int, Hkv: int, B: int, S0: int, W: int, k: np.ndarray,
              v: np.ndarray, seq_idx: np.ndarray, pos: np.ndarray) -> None:
    """Copy bf16 rows (k, v: [n, Hkv, d] bits) of sequence seq_idx[i] at position
    pos[i] into their sink / window slot of ``seg`` (uint16, modified in place)."""
    assert seg.dtype == np.uint16 and seg.flags["C_CONTIGUOUS"]
    si = _c(seq_idx, np.int32)
    ps = _c(pos, np.int64)
    rc = lib().oracle_seg_write(d, Hkv, S0, W, B, _ptr(seg), _ptr(_c(k, np.uint16)),
                                _ptr(_c(v, np.uint16)), _ptr(si), _ptr(ps), si.shape[0])
    if rc:
        raise ValueError("oracle seg_write: bad sequence or a position without a bf16 slot")


def mixed_update(pages: np.ndarray, seg: np.ndarray, *, d: int, Hkv: int, P: int, G: int,
                 S0: int, W: int, k_new: np.ndarray, v_new: np.ndarray, block_table: np.ndarray,
                 seq_lens: np.ndarray, Rk, Rv, clip_k: float, clip_v: float, meta: int = 0,
                 clip: int = 0) -> int:
    """One new token per sequence at position seq_lens[b] - 1 (k_new, v_new:
    [B, Hkv, d] bf16 bits): sink, window with demotion of the oldest window token
    into INT2, or INT2 directly when W = 0.  ``pages`` and ``seg`` change in place."""
    bt = _c(block_table, np.int32)
    sl = _c(seq_lens, np.int32)
    B = sl.shape[0]
    num_pages = pages.size // (Hkv * page_head_bytes(d, P, G))
    Rka, Rkp = _rot(Rk)
    Rva, Rvp = _rot(Rv)
    rc = lib().oracle_mixed_update(d, Hkv, P, G, int(meta), int(clip), num_pages, _ptr(pages),
                                   _ptr(seg), S0, W, B, _ptr(_c(k_new, np.uint16)),
                                   _ptr(_c(v_new, np.uint16)), _ptr(bt), bt.shape[1], _ptr(sl),
                                   Rkp, Rvp, float(clip_k), float(clip_v), _rph(Rk, Rv))
    if rc < 0:
        raise ValueError("oracle mixed_update: bad length or page")
    return int(rc)


def decode_mixed(pages: np.ndarray, seg: np.ndarray, *, d: int, Hkv: int, P: int, G: int,
                 S0: int, W: int, q: np.ndarray, block_table: np.ndarray, seq_lens: np.ndarray,
                 Rk, Rv, sm_scale: float, pairs=None, meta: int = 0) -> np.ndarray:
    """fp64 decode attention over bf16 sink + INT2 history + bf16 window."""
    q = _c(q, np.uint16)
    B, Hq = q.shape[0], q.shape[1]
    bt = _c(block_table, np.int32)
    sl = _c(seq_lens, np.int32)
    num_pages = pages.size // (Hkv * page_head_bytes(d, P, G))
    if pairs is None:
        out = np.zeros((B, Hq, d), np.float64)
        pp, n = None, 0
    else:
        pr = _c(pairs, np.int32).reshape(-1, 2)
        out = np.zeros((pr.shape[0], d), np.float64)
        pp, n = _ptr(pr), pr.shape[0]
    Rka, Rkp = _rot(Rk)
    Rva, Rvp = _rot(Rv)
    rc = lib().oracle_decode_mixed(d, Hkv, P, G, int(meta), num_pages, _ptr(pages),
                                   _ptr(_c(seg, np.uint16)), S0, W, _ptr(q), B, Hq, _ptr(bt),
                                   bt.shape[1], _ptr(sl), Rkp, Rvp, float(sm_scale), pp, n,
                                   _ptr(out), _rph(Rk, Rv))
    if rc:
        raise ValueError("oracle decode_mixed: bad page id, length or head")
    return out


# ---------------------------------------------------------------------------
# Offline calibration (Sec. 3 "Algorithm Design: Offline Calibration and
# Justification"; App. worked example; Alg. 1 Calibrate)
# ---------------------------------------------------------------------------

def query_cov(q: np.ndarray, Hkv: int) -> np.ndarray:
    """GQA-averaged C_Q of bf16 queries q [T, Hq, d] (uint16 bits): [d, d] fp64."""
    q = _c(q, np.uint16)
    T, Hq, d = q.shape
    C = np.zeros((d, d), np.float64)
    if lib().oracle_query_cov(_ptr(q), T, Hq, Hkv, d, _ptr(C)):
        raise ValueError("oracle query_cov: bad shape")
    return C


def attn_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray, *, causal: bool,
              pairs=None) -> np.ndarray:
    """Attention outputs o_{t,i} (fp64) of bf16 q [T, Hq, d], k, v [T, Hkv, d];
    ``pairs`` (t, i) or None for all rows ([T, Hq, d])."""
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    if pairs is None:
        out = np.zeros((T, Hq, d), np.float64)
        pp, n = None, 0
    else:
        pr = _c(pairs, np.int32).reshape(-1, 2)
        out = np.zeros((pr.shape[0], d), np.float64)
        pp, n = _ptr(pr), pr.shape[0]
    if lib().oracle_attn_rows(_ptr(q), _ptr(k), _ptr(v), T, Hq, Hkv, d, int(bool(causal)), pp, n,
                              _ptr(out)):
        raise ValueError("oracle attn_rows: bad shape or pair")
    return out


def score_cov(q: np.ndarray, k: np.ndarray, v: np.ndarray, *, causal: bool) -> np.ndarray:
    """GQA-averaged C_S = (1/N) V^T S^T S V: [d, d] fp64."""
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    T, Hq, d = q.shape
    C = np.zeros((d, d), np.float64)
    if lib().oracle_score_cov(_ptr(q), _ptr(k), _ptr(v), T, Hq, k.shape[1], d, int(bool(causal)),
                              _ptr(C)):
        raise ValueError("oracle score_cov: bad shape")
    return C


def hadamard(d: int) -> np.ndarray:
    H = np.zeros((d, d), np.float64)
    if lib().oracle_hadamard(d, _ptr(H)):
        raise ValueError("oracle hadamard: d must be a power of two")
    return H


def bit_reversal(d: int) -> np.ndarray:
    P = np.zeros((d, d), np.float64)
    if lib().oracle_bit_reversal(d, _ptr(P)):
        raise ValueError("oracle bit_reversal: d must be a power of two")
    return P


def compose(U: np.ndarray) -> np.ndarray:
    """R = U H_Had P_br (fp64)."""
    U = _c(U, np.float64)
    d = U.shape[0]
    R = np.zeros((d, d), np.float64)
    if lib().oracle_compose(_ptr(U), d, _ptr(R)):
        raise ValueError("oracle compose: d must be a power of two")
    return R


def eigh_desc(C: np.ndarray):
    """Eigen-decomposition C = U diag(lam) U^T of a symmetric fp64 matrix (LAPACK
    through numpy), eigenvalues in descending order; each eigenvector's sign is
    fixed so that its entry of largest magnitude (the first such) is positive."""
    w, U = np.linalg.eigh(_c(C, np.float64))
    order = np.argsort(-w, kind="stable")
    w, U = w[order], U[:, order]
    idx = np.argmax(np.abs(U), axis=0)
    sign = np.where(U[idx, np.arange(U.shape[1])] < 0, -1.0, 1.0)
    return w.copy(), np.ascontiguousarray(U * sign[None, :])


def clip_errors(x: np.ndarray, R, *, G: int, cands, meta: int = 0, clip: int = 0) -> np.ndarray:
    """Mean squared quantization error of the rotated rows x [n, d] or [n, Hkv, d]
    (bf16 bits) for each candidate clip ratio (fp32): [n_cands] fp64.  R: [d, d],
    [Hkv, d, d] (row (t, h) rotated by R[h]) or None."""
    x = _c(x, np.uint16)
    d = x.shape[-1]
    Hkv = x.shape[1] if x.ndim == 3 else 1
    rph = _rph(R)
    if rph and (x.ndim != 3 or np.shape(R)[0] != Hkv):
        raise ValueError("per-head R needs rows [n, Hkv, d] with Hkv = R.shape[0]")
    x = x.reshape(-1, d)
    cd = _c(cands, np.float32)
    err = np.zeros(cd.size, np.float64)
    Ra, Rp = _rot(R)
    if lib().oracle_clip_errors(_ptr(x), x.shape[0], d, Rp, G, int(meta), int(clip), _ptr(cd),
                                cd.size, _ptr(err), Hkv, rph):
        raise ValueError("oracle clip_errors: bad shape")
    return err


def default_clip_candidates() -> np.ndarray:
    """0.80, 0.81, ..., 1.00 as fp32."""
    return np.array([round(0.80 + 0.01 * n, 2) for n in range(21)], np.float32)


def calibrate(q: np.ndarray, k: np.ndarray, v: np.ndarray, *, causal: bool = True, G: int = 32,
              meta: int = 0, clip: int = 0, cands=None, per_head: bool = False) -> dict:
    """Alg. 1 Calibrate for one layer from bf16 activations q [T, Hq, d], k, v
    [T, Hkv, d]: C_Q, C_S, their descending eigen-decompositions, R_K and R_V
    (fp64 and rounded to fp32), and the clip ratios c_K, c_V chosen among
    ``cands`` (the first minimum of clip_errors) for rows rotated by the fp32
    matrices the cache update uses.  ``per_head``: one C_Q, C_S and rotation per
    KV head (the average over its g query heads), stacked [Hkv, d, d]; one clip
    ratio per tensor over all heads."""
    cands = default_clip_candidates() if cands is None else _c(cands, np.float32)
    Hkv = k.shape[1]
    if per_head:
        g = q.shape[1] // Hkv
        CQ = np.stack([query_cov(q[:, h * g:(h + 1) * g], 1) for h in range(Hkv)])
        CS = np.stack([score_cov(q[:, h * g:(h + 1) * g], k[:, h:h + 1], v[:, h:h + 1],
                                 causal=causal) for h in range(Hkv)])
        eq = [eigh_desc(C) for C in CQ]
        es = [eigh_desc(C) for C in CS]
        lam_q, UQ = np.stack([e[0] for e in eq]), np.stack([e[1] for e in eq])
        lam_s, US = np.stack([e[0] for e in es]), np.stack([e[1] for e in es])
        RK, RV = np.stack([compose(U) for U in UQ]), np.stack([compose(U) for U in US])
    else:
        CQ = query_cov(q, Hkv)
        CS = score_cov(q, k, v, causal=causal)
        lam_q, UQ = eigh_desc(CQ)
        lam_s, US = eigh_desc(CS)
        RK, RV = compose(UQ), compose(US)
    RK32, RV32 = RK.astype(np.float32), RV.astype(np.float32)
    err_k = clip_errors(k, RK32, G=G, cands=cands, meta=meta, clip=clip)
    err_v = clip_errors(v, RV32, G=G, cands=cands, meta=meta, clip=clip)
    return {"C_Q": CQ, "C_S": CS, "lam_Q": lam_q, "lam_S": lam_s, "U_Q": UQ, "U_S": US,
            "R_K": RK, "R_V": RV, "R_K32": RK32, "R_V32": RV32, "err_K": err_k, "err_V": err_v,
            "c_K": float(cands[int(np.argmin(err_k))]), "c_V": float(cands[int(np.argmin(err_v))])}
