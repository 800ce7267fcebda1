"""Python binding of liboscar (INT2 KV-cache append + paged decode attention for
OSCAR, arXiv 2605.17757, on MI355X / gfx950).

Argument marshalling only: every function checks tensor dtypes, devices and
shapes, then calls the C ABI of ``liboscar.so`` (declared in include/oscar.h)
with raw device pointers and the current HIP stream.  All computation happens
in the library's HIP kernels; there is no fallback of any kind.  If the shared
library is missing, importing works but the first call raises OscarError.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboscar.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE_TOO_SMALL, ERR_HIP = range(5)
OUT_BF16, OUT_F32 = 0, 1

HEAD_DIM, PAGE_SIZE, GROUP_SIZE = 128, 64, 32

# Every symbol include/oscar.h declares.
EXPORTS = (
    "oscar_status_string", "oscar_page_bytes", "oscar_pool_bytes", "oscar_layout_check",
    "oscar_kv_append", "oscar_decode_workspace_bytes", "oscar_default_num_splits",
    "oscar_decode_attn", "oscar_decode_attn_noalloc", "oscar_decode_step", "oscar_decode_prepare", "oscar_decode_split",
    "oscar_decode_reduce",
    "oscar_seg_bytes", "oscar_mixed_workspace_bytes", "oscar_mixed_append",
    "oscar_decode_attn_mixed", "oscar_decode_step_mixed",
    "oscar_bf16_page_bytes", "oscar_bf16_kv_append", "oscar_bf16_decode_workspace_bytes",
    "oscar_bf16_decode_attn",
    "oscar_calib_workspace_bytes", "oscar_calib_query_cov", "oscar_calib_attn",
    "oscar_calib_score_cov", "oscar_calib_rotation_workspace_bytes", "oscar_calib_rotation",
    "oscar_calib_clip_workspace_bytes", "oscar_calib_clip",
    "oscar_calibrate_layer_workspace_bytes", "oscar_calibrate_layer",
    "oscar_hbm_read_probe", "oscar_hbm_read_probe_ex",
)

CALIB_MAX_CANDS = 32


class OscarError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s" % (where, status_string(status) if _lib else status))


CLIP_GROUP_ABSMAX, CLIP_TOKEN_QUANTILE = 0, 1
META_F16, META_BF16 = 0, 1


class Layout(ctypes.Structure):
    """Mirror of ``oscar_layout``."""
    _fields_ = [("head_dim", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("num_pages", ctypes.c_int64), ("clip_mode", ctypes.c_int32),
                ("meta_dtype", ctypes.c_int32), ("rot_per_head", ctypes.c_int32)]

    def __init__(self, num_kv_heads: int, num_pages: int, head_dim: int = HEAD_DIM,
                 page_size: int = PAGE_SIZE, group_size: int = GROUP_SIZE,
                 clip_mode: int = CLIP_GROUP_ABSMAX, meta_dtype: int = META_F16,
                 rot_per_head: int = 0):
        super().__init__(head_dim, num_kv_heads, page_size, group_size, num_pages, clip_mode,
                         meta_dtype, rot_per_head)


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded liboscar.so (raises OscarError(-1) if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise OscarError(-1, "loading %s (not built: run python paper_2605_17757_amd/build.py)"
                             % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, f32, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                ctypes.c_size_t)
        LP = ctypes.POINTER(Layout)
        sigs = {
            "oscar_status_string": (ctypes.c_char_p, [ctypes.c_int]),
            "oscar_page_bytes": (sz, [LP]),
            "oscar_pool_bytes": (sz, [LP]),
            "oscar_layout_check": (ctypes.c_int, [LP]),
            "oscar_kv_append": (ctypes.c_int, [LP, P, P, P, P, i32, P, P, f32, f32, P]),
            "oscar_decode_workspace_bytes": (sz, [LP, i32, i32, i32]),
            "oscar_default_num_splits": (i32, [LP, i32, i32, i32]),
            "oscar_decode_attn": (ctypes.c_int, [LP, P, P, i32, i32, P, i32, P, P, P, f32, i32, P,
                                                 sz, P, ctypes.c_int, P]),
            "oscar_decode_attn_noalloc": (ctypes.c_int, [LP, P, P, i32, i32, P, i32, P, P, P,
                                                         f32, i32, P, ctypes.c_int, P]),
            "oscar_decode_step": (ctypes.c_int, [LP, P, P, P, P, i32, f32, f32, P, i32, i32, P,
                                                 i32, P, P, P, f32, i32, P, sz, P, ctypes.c_int,
                                                 P]),
            "oscar_decode_prepare": (ctypes.c_int, [LP, P, i32, i32, P, f32, i32, P, sz, P]),
            "oscar_decode_split": (ctypes.c_int, [LP, P, i32, i32, P, i32, P, i32, P, sz, P]),
            "oscar_decode_reduce": (ctypes.c_int, [LP, i32, i32, P, i32, P, sz, P, ctypes.c_int,
                                                   P]),
            "oscar_seg_bytes": (sz, [LP, i32, i32, i32]),
            "oscar_mixed_workspace_bytes": (sz, [LP, i32, i32, i32]),
            "oscar_mixed_append": (ctypes.c_int, [LP, P, P, i32, i32, i32, P, P, P, P, i32, P,
                                                  i32, P, P, P, f32, f32, P]),
            "oscar_decode_attn_mixed": (ctypes.c_int, [LP, P, P, i32, i32, P, i32, i32, P, i32,
                                                       P, P, P, f32, i32, P, sz, P, ctypes.c_int,
                                                       P]),
            "oscar_decode_step_mixed": (ctypes.c_int, [LP, P, P, i32, i32, P, P, f32, f32, P,
                                                       i32, i32, P, i32, P, P, P, f32, i32, P, sz,
                                                       P, ctypes.c_int, P]),
            "oscar_bf16_page_bytes": (sz, [LP]),
            "oscar_bf16_kv_append": (ctypes.c_int, [LP, P, P, P, P, i32, P]),
            "oscar_bf16_decode_workspace_bytes": (sz, [LP, i32, i32, i32]),
            "oscar_bf16_decode_attn": (ctypes.c_int, [LP, P, P, i32, i32, P, i32, P, f32, i32, P,
                                                      sz, P, ctypes.c_int, P]),
            "oscar_calib_workspace_bytes": (sz, [i64, i32, i32]),
            "oscar_calib_query_cov": (ctypes.c_int, [P, i64, i32, i32, P, P, sz, P]),
            "oscar_calib_attn": (ctypes.c_int, [P, P, P, i64, i32, i32, i32, P, P]),
            "oscar_calib_score_cov": (ctypes.c_int, [P, P, P, i64, i32, i32, i32, P, P, sz, P]),
            "oscar_calib_rotation_workspace_bytes": (sz, [i32]),
            "oscar_calib_rotation": (ctypes.c_int, [P, i32, P, P, P, P, P, P, sz, P]),
            "oscar_calib_clip_workspace_bytes": (sz, [i64, i32, i32]),
            "oscar_calib_clip": (ctypes.c_int, [LP, P, i64, P, P, i32, P, P, P, sz, P]),
            "oscar_calibrate_layer_workspace_bytes": (sz, [LP, i64, i32, i32]),
            "oscar_calibrate_layer": (ctypes.c_int, [LP, P, P, P, i64, i32, i32, P, i32, P, P, P,
                                                     P, P, P, sz, P]),
            "oscar_hbm_read_probe": (ctypes.c_int, [P, sz, P, i32, P]),
            "oscar_hbm_read_probe_ex": (ctypes.c_int, [P, sz, P, i32, i32, i32, P]),
        }
        for name, (res, args) in sigs.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().oscar_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != OK:
        raise OscarError(status, where)


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _ptr(t: torch.Tensor, dtype, name: str, numel: int | None = None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if numel is not None and t.numel() != numel:
        raise ValueError("%s has %d elements, expected %d" % (name, t.numel(), numel))
    return ctypes.c_void_p(t.data_ptr())


def _rptr(R, name: str, d: int = HEAD_DIM, layout=None):
    """A rotation matrix (fp32 [d, d] on the GPU; [Hkv, d, d] when the layout has
    one per KV head), or None for the identity."""
    if R is None:
        return None
    n = d * d * (layout.num_kv_heads if layout is not None and layout.rot_per_head else 1)
    return _ptr(R, torch.float32, name, n)


# ---------------------------------------------------------------------------
# sizes and helpers
# ---------------------------------------------------------------------------

def page_bytes(layout: Layout) -> int:
    return int(lib().oscar_page_bytes(ctypes.byref(layout)))


def pool_bytes(layout: Layout) -> int:
    return int(lib().oscar_pool_bytes(ctypes.byref(layout)))


def layout_check(layout: Layout) -> int:
    return int(lib().oscar_layout_check(ctypes.byref(layout)))


def decode_workspace_bytes(layout: Layout, B: int, Hq: int, num_splits: int) -> int:
    return int(lib().oscar_decode_workspace_bytes(ctypes.byref(layout), B, Hq, num_splits))


def default_num_splits(layout: Layout, B: int, Hq: int, max_seq_len: int) -> int:
    return int(lib().oscar_default_num_splits(ctypes.byref(layout), B, Hq, max_seq_len))


def alloc_pool(layout: Layout, device="cuda") -> torch.Tensor:
    return torch.zeros(pool_bytes(layout), dtype=torch.uint8, device=device)


def alloc_workspace(layout: Layout, B: int, Hq: int, num_splits: int, device="cuda"):
    n = decode_workspace_bytes(layout, B, Hq, num_splits)
    if n == 0:
        raise OscarError(ERR_INVALID_ARG, "decode_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


# ---------------------------------------------------------------------------
# the hot path
# ---------------------------------------------------------------------------

def kv_append(layout: Layout, pages, k_new, v_new, slot_mapping, R_k, R_v, clip_k: float,
              clip_v: float, stream=None) -> None:
    """Rotate, clip, INT2-quantize and pack n_tok new K/V rows into ``pages``
    (R_k / R_v None: identity)."""
    n_tok = int(slot_mapping.numel())
    d, hkv = layout.head_dim, layout.num_kv_heads
    st = lib().oscar_kv_append(
        ctypes.byref(layout), _ptr(pages, torch.uint8, "pages", pool_bytes(layout)),
        _ptr(k_new, torch.bfloat16, "k_new", n_tok * hkv * d),
        _ptr(v_new, torch.bfloat16, "v_new", n_tok * hkv * d),
        _ptr(slot_mapping, torch.int64, "slot_mapping"), n_tok,
        _rptr(R_k, "R_k", d, layout), _rptr(R_v, "R_v", d, layout),
        float(clip_k), float(clip_v), _stream(stream))
    _check(st, "oscar_kv_append")


def _decode_args(layout, q, block_table, seq_lens):
    if q.dim() != 3:
        raise ValueError("q must be [B, Hq, d]")
    B, Hq = int(q.shape[0]), int(q.shape[1])
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError("block_table must be [B, max_pages_per_seq]")
    return B, Hq, int(block_table.shape[1])


def decode_attn(layout: Layout, pages, q, block_table, seq_lens, R_k, R_v, sm_scale: float,
                num_splits: int, workspace, out, stream=None) -> None:
    """One decode step of attention over the INT2 cache into ``out`` ([B, Hq, d],
    bf16 or fp32)."""
    B, Hq, mp = _decode_args(layout, q, block_table, seq_lens)
    d = layout.head_dim
    out_dtype = OUT_F32 if out.dtype == torch.float32 else OUT_BF16
    st = lib().oscar_decode_attn(
        ctypes.byref(layout), _ptr(pages, torch.uint8, "pages", pool_bytes(layout)),
        _ptr(q, torch.bfloat16, "q", B * Hq * d), B, Hq,
        _ptr(block_table, torch.int32, "block_table", B * mp), mp,
        _ptr(seq_lens, torch.int32, "seq_lens", B), _rptr(R_k, "R_k", d, layout),
        _rptr(R_v, "R_v", d, layout), float(sm_scale), int(num_splits),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _ptr(out, out.dtype, "out", B * Hq * d), out_dtype, _stream(stream))
    _check(st, "oscar_decode_attn")


NOALLOC_SCRATCH_BYTES = 64 << 20


def decode_attn_noalloc(layout: Layout, pages, q, block_table, seq_lens, R_k, R_v,
                        sm_scale: float, num_splits: int, out, stream=None) -> None:
    """decode_attn with the library's per-GPU scratch array as its workspace
    (oscar_decode_attn_noalloc: nothing is allocated; calls that overlap on one
    GPU race)."""
    B, Hq, mp = _decode_args(layout, q, block_table, seq_lens)
    d = layout.head_dim
    out_dtype = OUT_F32 if out.dtype == torch.float32 else OUT_BF16
    st = lib().oscar_decode_attn_noalloc(
        ctypes.byref(layout), _ptr(pages, torch.uint8, "pages", pool_bytes(layout)),
        _ptr(q, torch.bfloat16, "q", B * Hq * d), B, Hq,
        _ptr(block_table, torch.int32, "block_table", B * mp), mp,
        _ptr(seq_lens, torch.int32, "seq_lens", B), _rptr(R_k, "R_k", d, layout),
        _rptr(R_v, "R_v", d, layout), float(sm_scale), int(num_splits),
        _ptr(out, out.dtype, "out", B * Hq * d), out_dtype, _stream(stream))
    _check(st, "oscar_decode_attn_noalloc")


def decode_step(layout: Layout, pages, k_new, v_new, slot_mapping, clip_k: float,
                clip_v: float, q, block_table, seq_lens, R_k, R_v, sm_scale: float,
                num_splits: int, workspace, out, stream=None) -> None:
    """One serving decode step: append the new tokens' K/V (``slot_mapping`` may be
    empty), then attention over the cache into ``out``."""
    B, Hq, mp = _decode_args(layout, q, block_table, seq_lens)
    d, hkv = layout.head_dim, layout.num_kv_heads
    n_new = int(slot_mapping.numel())
    out_dtype = OUT_F32 if out.dtype == torch.float32 else OUT_BF16
    kp = _ptr(k_new, torch.bfloat16, "k_new", n_new * hkv * d) if n_new else None
    vp = _ptr(v_new, torch.bfloat16, "v_new", n_new * hkv * d) if n_new else None
    sp = _ptr(slot_mapping, torch.int64, "slot_mapping") if n_new else None
    st = lib().oscar_decode_step(
        ctypes.byref(layout), _ptr(pages, torch.uint8, "pages", pool_bytes(layout)), kp, vp, sp,
        n_new, float(clip_k), float(clip_v), _ptr(q, torch.bfloat16, "q", B * Hq * d), B, Hq,
        _ptr(block_table, torch.int32, "block_table", B * mp), mp,
        _ptr(seq_lens, torch.int32, "seq_lens", B), _rptr(R_k, "R_k", d, layout),
        _rptr(R_v, "R_v", d, layout), float(sm_scale), int(num_splits),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _ptr(out, out.dtype, "out", B * Hq * d), out_dtype, _stream(stream))
    _check(st, "oscar_decode_step")


def decode_prepare(layout: Layout, q, R_k, sm_scale: float, num_splits: int, workspace,
                   stream=None) -> None:
    B, Hq, d = int(q.shape[0]), int(q.shape[1]), layout.head_dim
    st = lib().oscar_decode_prepare(
        ctypes.byref(layout), _ptr(q, torch.bfloat16, "q", B * Hq * d), B, Hq,
        _rptr(R_k, "R_k", d, layout), float(sm_scale), int(num_splits),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    _check(st, "oscar_decode_prepare")


def decode_split(layout: Layout, pages, B: int, Hq: int, block_table, seq_lens,
                 num_splits: int, workspace, stream=None) -> None:
    mp = int(block_table.shape[1])
    st = lib().oscar_decode_split(
        ctypes.byref(layout), _ptr(pages, torch.uint8, "pages", pool_bytes(layout)), B, Hq,
        _ptr(block_table, torch.int32, "block_table", B * mp), mp,
        _ptr(seq_lens, torch.int32, "seq_lens", B), int(num_splits),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    _check(st, "oscar_decode_split")


def decode_reduce(layout: Layout, B: int, Hq: int, R_v, num_splits: int, workspace, out,
                  stream=None) -> None:
    d = layout.head_dim
    out_dtype = OUT_F32 if out.dtype == torch.float32 else OUT_BF16
    st = lib().oscar_decode_reduce(
        ctypes.byref(layout), B, Hq, _rptr(R_v, "R_v", d, layout), int(num_splits),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _ptr(out, out.dtype, "out", B * Hq * d), out_dtype, _stream(stream))
    _check(st, "oscar_decode_reduce")


# ---------------------------------------------------------------------------
# mixed-precision cache (bf16 sink and recent window around the INT2 history)
# ---------------------------------------------------------------------------

def seg_bytes(layout: Layout, B: int, S0: int, W: int) -> int:
    return int(lib().oscar_seg_bytes(ctypes.byref(layout), B, S0, W))


def mixed_workspace_bytes(layout: Layout, B: int, Hq: int, num_splits: int) -> int:
    return int(lib().oscar_mixed_workspace_bytes(ctypes.byref(layout), B, Hq, num_splits))


def alloc_seg(layout: Layout, B: int, S0: int, W: int, device="cuda") -> torch.Tensor:
    """Zeroed segment store, bf16 [B, Hkv, 2, S0 + W, d]."""
    return torch.zeros(B, layout.num_kv_heads, 2, S0 + W, layout.head_dim, dtype=torch.bfloat16,
                       device=device)


def alloc_mixed_workspace(layout: Layout, B: int, Hq: int, num_splits: int, device="cuda"):
    n = mixed_workspace_bytes(layout, B, Hq, num_splits)
    if n == 0:
        raise OscarError(ERR_INVALID_ARG, "mixed_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


def _seg_ptr(layout, seg, B, S0, W):
    if S0 + W == 0 and seg is None:
        return None
    return _ptr(seg, torch.bfloat16, "seg", seg_bytes(layout, B, S0, W) // 2)


def mixed_append(layout: Layout, pages, seg, S0: int, W: int, k, v, seq_idx, pos, block_table,
                 seq_lens, R_k, R_v, clip_k: float, clip_v: float, stream=None) -> None:
    """Write prompt tokens (k, v: [n, Hkv, d]) of sequences ``seq_idx`` at positions
    ``pos`` where a mixed cache of length ``seq_lens`` keeps them."""
    n_tok = int(pos.numel())
    d, hkv = layout.head_dim, layout.num_kv_heads
    B, mp = int(block_table.shape[0]), int(block_table.shape[1])
    st = lib().oscar_mixed_append(
        ctypes.byref(layout), _ptr(pages, torch.uint8, "pages", pool_bytes(layout)),
        _seg_ptr(layout, seg, B, S0, W), B, int(S0), int(W),
        _ptr(k, torch.bfloat16, "k", n_tok * hkv * d), _ptr(v, torch.bfloat16, "v", n_tok * hkv * d),
        _ptr(seq_idx, torch.int32, "seq_idx", n_tok), _ptr(pos, torch.int64, "pos", n_tok), n_tok,
        _ptr(block_table, torch.int32, "block_table", B * mp), mp,
        _ptr(seq_lens, torch.int32, "seq_lens", B), _rptr(R_k, "R_k", d, layout),
        _rptr(R_v, "R_v", d, layout), float(clip_k), float(clip_v), _stream(stream))
    _check(st, "oscar_mixed_append")


def decode_attn_mixed(layout: Layout, pages, seg, S0: int, W: int, q, block_table, seq_lens, R_k,
                      R_v, sm_scale: float, num_splits: int, workspace, out, stream=None) -> None:
    """Decode attention over the mixed cache into ``out`` ([B, Hq, d], bf16 or fp32)."""
    B, Hq, mp = _decode_args(layout, q, block_table, seq_lens)
    d = layout.head_dim
    out_dtype = OUT_F32 if out.dtype == torch.float32 else OUT_BF16
    st = lib().oscar_decode_attn_mixed(
        ctypes.byref(layout), _ptr(pages, torch.uint8, "pages", pool_bytes(layout)),
        _seg_ptr(layout, seg, B, S0, W), int(S0), int(W),
        _ptr(q, torch.bfloat16, "q", B * Hq * d), B, Hq,
        _ptr(block_table, torch.int32, "block_table", B * mp), mp,
        _ptr(seq_lens, torch.int32, "seq_lens", B), _rptr(R_k, "R_k", d, layout),
        _rptr(R_v, "R_v", d, layout), float(sm_scale), int(num_splits),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _ptr(out, out.dtype, "out", B * Hq * d), out_dtype, _stream(stream))
    _check(st, "oscar_decode_attn_mixed")


def decode_step_mixed(layout: Layout, pages, seg, S0: int, W: int, k_new, v_new, clip_k: float,
                      clip_v: float, q, block_table, seq_lens, R_k, R_v, sm_scale: float,
                      num_splits: int, workspace, out, stream=None) -> None:
    """One decode step over the mixed cache: one new token per sequence (k_new,
    v_new: [B, Hkv, d]) at position seq_lens[b] - 1, then attention into ``out``."""
    B, Hq, mp = _decode_args(layout, q, block_table, seq_lens)
    d, hkv = layout.head_dim, layout.num_kv_heads
    out_dtype = OUT_F32 if out.dtype == torch.float32 else OUT_BF16
    st = lib().oscar_decode_step_mixed(
        ctypes.byref(layout), _ptr(pages, torch.uint8, "pages", pool_bytes(layout)),
        _seg_ptr(layout, seg, B, S0, W), int(S0), int(W),
        _ptr(k_new, torch.bfloat16, "k_new", B * hkv * d),
        _ptr(v_new, torch.bfloat16, "v_new", B * hkv * d), float(clip_k), float(clip_v),
        _ptr(q, torch.bfloat16, "q", B * Hq * d), B, Hq,
        _ptr(block_table, torch.int32, "block_table", B * mp), mp,
        _ptr(seq_lens, torch.int32, "seq_lens", B), _rptr(R_k, "R_k", d, layout),
        _rptr(R_v, "R_v", d, layout), float(sm_scale), int(num_splits),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _ptr(out, out.dtype, "out", B * Hq * d), out_dtype, _stream(stream))
    _check(st, "oscar_decode_step_mixed")


# ---------------------------------------------------------------------------
# bf16 baseline
# ---------------------------------------------------------------------------

def bf16_pool_bytes(layout: Layout) -> int:
    return int(lib().oscar_bf16_page_bytes(ctypes.byref(layout))) * int(layout.num_pages)


def bf16_kv_append(layout: Layout, pages, k_new, v_new, slot_mapping, stream=None) -> None:
    n_tok = int(slot_mapping.numel())
    d, hkv = layout.head_dim, layout.num_kv_heads
    st = lib().oscar_bf16_kv_append(
        ctypes.byref(layout), _ptr(pages, torch.bfloat16, "pages", bf16_pool_bytes(layout) // 2),
        _ptr(k_new, torch.bfloat16, "k_new", n_tok * hkv * d),
        _ptr(v_new, torch.bfloat16, "v_new", n_tok * hkv * d),
        _ptr(slot_mapping, torch.int64, "slot_mapping"), n_tok, _stream(stream))
    _check(st, "oscar_bf16_kv_append")


def bf16_decode_attn(layout: Layout, pages, q, block_table, seq_lens, sm_scale: float,
                     num_splits: int, workspace, out, stream=None) -> None:
    B, Hq, mp = _decode_args(layout, q, block_table, seq_lens)
    d = layout.head_dim
    out_dtype = OUT_F32 if out.dtype == torch.float32 else OUT_BF16
    st = lib().oscar_bf16_decode_attn(
        ctypes.byref(layout), _ptr(pages, torch.bfloat16, "pages", bf16_pool_bytes(layout) // 2),
        _ptr(q, torch.bfloat16, "q", B * Hq * d), B, Hq,
        _ptr(block_table, torch.int32, "block_table", B * mp), mp,
        _ptr(seq_lens, torch.int32, "seq_lens", B), float(sm_scale), int(num_splits),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _ptr(out, out.dtype, "out", B * Hq * d), out_dtype, _stream(stream))
    _check(st, "oscar_bf16_decode_attn")


# ---------------------------------------------------------------------------
# offline calibration (Sec. 3; Alg. 1 Calibrate)
# ---------------------------------------------------------------------------

def _ws(n: int, where: str, device="cuda") -> torch.Tensor:
    if n == 0:
        raise OscarError(ERR_INVALID_ARG, where)
    return torch.empty(n, dtype=torch.uint8, device=device)


def _qkv_shapes(q, k=None, v=None):
    if q.dim() != 3 or q.shape[2] != HEAD_DIM:
        raise ValueError("q must be [T, Hq, %d]" % HEAD_DIM)
    T, Hq = int(q.shape[0]), int(q.shape[1])
    Hkv = None
    if k is not None:
        if k.dim() != 3 or k.shape[0] != T or k.shape[2] != HEAD_DIM or v is None or \
                tuple(v.shape) != tuple(k.shape):
            raise ValueError("k, v must be [T, Hkv, %d] with the same T as q" % HEAD_DIM)
        Hkv = int(k.shape[1])
    return T, Hq, Hkv


def calib_workspace_bytes(T: int, Hq: int, Hkv: int) -> int:
    return int(lib().oscar_calib_workspace_bytes(T, Hq, Hkv))


def calib_query_cov(q, Hkv: int, workspace=None, stream=None) -> torch.Tensor:
    """GQA-averaged C_Q (fp64 [d, d]) of bf16 queries q [T, Hq, d]."""
    T, Hq, _ = _qkv_shapes(q)
    ws = workspace if workspace is not None else _ws(calib_workspace_bytes(T, Hq, Hkv),
                                                     "calib_workspace_bytes")
    C = torch.empty(HEAD_DIM, HEAD_DIM, dtype=torch.float64, device=q.device)
    _check(lib().oscar_calib_query_cov(_ptr(q, torch.bfloat16, "q"), T, Hq, Hkv,
                                       _ptr(C, torch.float64, "C"), _ptr(ws, torch.uint8, "ws"),
                                       ws.numel(), _stream(stream)), "oscar_calib_query_cov")
    return C


def calib_attn(q, k, v, causal: bool = True, out=None, stream=None) -> torch.Tensor:
    """Attention rows of the calibration pass: fp32 [T, Hq, d]."""
    T, Hq, Hkv = _qkv_shapes(q, k, v)
    if out is None:
        out = torch.empty(T, Hq, HEAD_DIM, dtype=torch.float32, device=q.device)
    _check(lib().oscar_calib_attn(_ptr(q, torch.bfloat16, "q"), _ptr(k, torch.bfloat16, "k"),
                                  _ptr(v, torch.bfloat16, "v"), T, Hq, Hkv, int(bool(causal)),
                                  _ptr(out, torch.float32, "out", T * Hq * HEAD_DIM),
                                  _stream(stream)), "oscar_calib_attn")
    return out


def calib_score_cov(q, k, v, causal: bool = True, workspace=None, stream=None) -> torch.Tensor:
    """GQA-averaged C_S = V^T S^T S V / N (fp64 [d, d])."""
    T, Hq, Hkv = _qkv_shapes(q, k, v)
    ws = workspace if workspace is not None else _ws(calib_workspace_bytes(T, Hq, Hkv),
                                                     "calib_workspace_bytes")
    C = torch.empty(HEAD_DIM, HEAD_DIM, dtype=torch.float64, device=q.device)
    _check(lib().oscar_calib_score_cov(_ptr(q, torch.bfloat16, "q"), _ptr(k, torch.bfloat16, "k"),
                                       _ptr(v, torch.bfloat16, "v"), T, Hq, Hkv,
                                       int(bool(causal)), _ptr(C, torch.float64, "C"),
                                       _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream)),
           "oscar_calib_score_cov")
    return C


def calib_rotation(C, workspace=None, stream=None) -> dict:
    """Eigen-decomposition (descending, sign-fixed) and R = U H_Had P_br of
    symmetric fp64 matrices C [n, d, d] (or [d, d])."""
    Cb = C if C.dim() == 3 else C.unsqueeze(0)
    n = int(Cb.shape[0])
    if tuple(Cb.shape[1:]) != (HEAD_DIM, HEAD_DIM):
        raise ValueError("C must be [n, %d, %d]" % (HEAD_DIM, HEAD_DIM))
    Cb = Cb.contiguous()
    dev = Cb.device
    lam = torch.empty(n, HEAD_DIM, dtype=torch.float64, device=dev)
    U = torch.empty(n, HEAD_DIM, HEAD_DIM, dtype=torch.float64, device=dev)
    R64 = torch.empty_like(U)
    R32 = torch.empty(n, HEAD_DIM, HEAD_DIM, dtype=torch.float32, device=dev)
    info = torch.empty(n, dtype=torch.int32, device=dev)
    ws = workspace if workspace is not None else _ws(
        int(lib().oscar_calib_rotation_workspace_bytes(n)), "calib_rotation_workspace_bytes")
    _check(lib().oscar_calib_rotation(_ptr(Cb, torch.float64, "C"), n, _ptr(lam, torch.float64, "lam"),
                                      _ptr(U, torch.float64, "U"), _ptr(R64, torch.float64, "R64"),
                                      _ptr(R32, torch.float32, "R32"), _ptr(info, torch.int32, "info"),
                                      _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream)),
           "oscar_calib_rotation")
    return {"lam": lam, "U": U, "R64": R64, "R32": R32, "info": info}


def calib_clip(layout: Layout, x, R, cands, workspace=None, stream=None):
    """(err [n_cands] fp64, best [1] fp32) for rows x [n_tok, Hkv, d] (bf16)."""
    if x.dim() != 3 or x.shape[1] != layout.num_kv_heads or x.shape[2] != HEAD_DIM:
        raise ValueError("x must be [n_tok, Hkv, %d]" % HEAD_DIM)
    n_tok = int(x.shape[0])
    nc = int(cands.numel())
    err = torch.empty(nc, dtype=torch.float64, device=x.device)
    best = torch.empty(1, dtype=torch.float32, device=x.device)
    ws = workspace if workspace is not None else _ws(
        int(lib().oscar_calib_clip_workspace_bytes(n_tok, layout.num_kv_heads, nc)),
        "calib_clip_workspace_bytes")
    _check(lib().oscar_calib_clip(ctypes.byref(layout), _ptr(x, torch.bfloat16, "x"), n_tok,
                                  _rptr(R, "R", HEAD_DIM, layout), _ptr(cands, torch.float32, "cands"), nc,
                                  _ptr(err, torch.float64, "err"), _ptr(best, torch.float32, "best"),
                                  _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream)),
           "oscar_calib_clip")
    return err, best


def calibrate_layer_workspace_bytes(layout: Layout, T: int, Hq: int, n_cands: int) -> int:
    return int(lib().oscar_calibrate_layer_workspace_bytes(ctypes.byref(layout), T, Hq, n_cands))


def calibrate_layer(layout: Layout, q, k, v, cands, causal: bool = True, workspace=None,
                    stream=None) -> dict:
    """Alg. 1 Calibrate for one layer: R_K, R_V (fp32 [d, d], or [Hkv, d, d] when
    the layout has one rotation per KV head), clip (c_K, c_V), lam (spectra of
    C_Q and C_S) and info."""
    T, Hq, Hkv = _qkv_shapes(q, k, v)
    if Hkv != layout.num_kv_heads:
        raise ValueError("k has %d heads, layout %d" % (Hkv, layout.num_kv_heads))
    nc = int(cands.numel())
    dev = q.device
    hm = (Hkv,) if layout.rot_per_head else ()
    Rk = torch.empty(*hm, HEAD_DIM, HEAD_DIM, dtype=torch.float32, device=dev)
    Rv = torch.empty_like(Rk)
    clip = torch.empty(2, dtype=torch.float32, device=dev)
    lam = torch.empty(2, *hm, HEAD_DIM, dtype=torch.float64, device=dev)
    info = torch.empty(2, *hm, dtype=torch.int32, device=dev)
    ws = workspace if workspace is not None else _ws(
        calibrate_layer_workspace_bytes(layout, T, Hq, nc), "calibrate_layer_workspace_bytes")
    _check(lib().oscar_calibrate_layer(ctypes.byref(layout), _ptr(q, torch.bfloat16, "q"),
                                       _ptr(k, torch.bfloat16, "k"), _ptr(v, torch.bfloat16, "v"),
                                       T, Hq, int(bool(causal)), _ptr(cands, torch.float32, "cands"),
                                       nc, _ptr(Rk, torch.float32, "R_k"),
                                       _ptr(Rv, torch.float32, "R_v"),
                                       _ptr(clip, torch.float32, "clip"),
                                       _ptr(lam, torch.float64, "lam"),
                                       _ptr(info, torch.int32, "info"),
                                       _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream)),
           "oscar_calibrate_layer")
    return {"R_K": Rk, "R_V": Rv, "clip": clip, "lam": lam, "info": info}


# ---------------------------------------------------------------------------
# measurement helper
# ---------------------------------------------------------------------------

PROBE_NONTEMPORAL, PROBE_WAVE_CHUNKS = 1, 2


def hbm_read_probe(src, blocks: int, sink=None, stream=None, loads: int | None = None,
                   flags: int = 0) -> torch.Tensor:
    """Plain streaming read of the bytes of ``src`` (a contiguous GPU tensor, size a
    multiple of 16 bytes) by ``blocks`` blocks of 256 threads; returns the uint32
    sink [blocks * 256] whose xor is the xor of the source words.  ``loads`` (4, 8
    or 16 loads in flight per thread) and ``flags`` (PROBE_NONTEMPORAL,
    PROBE_WAVE_CHUNKS) select oscar_hbm_read_probe_ex; both None/0 call
    oscar_hbm_read_probe."""
    if not isinstance(src, torch.Tensor) or not src.is_cuda or not src.is_contiguous():
        raise ValueError("src must be a contiguous GPU tensor")
    nbytes = src.numel() * src.element_size()
    if sink is None:
        sink = torch.empty(int(blocks) * 256, dtype=torch.int32, device=src.device)
    sp = _ptr(sink, torch.int32, "sink", int(blocks) * 256)
    if loads is None and not flags:
        _check(lib().oscar_hbm_read_probe(ctypes.c_void_p(src.data_ptr()), nbytes, sp,
                                          int(blocks), _stream(stream)), "oscar_hbm_read_probe")
    else:
        _check(lib().oscar_hbm_read_probe_ex(ctypes.c_void_p(src.data_ptr()), nbytes, sp,
                                             int(blocks), int(loads or 4), int(flags),
                                             _stream(stream)), "oscar_hbm_read_probe_ex")
    return sink
