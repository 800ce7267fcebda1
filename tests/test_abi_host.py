"""Host-only checks of the C ABI: the library loads, exports every symbol that
include/oscar.h declares, sizes its buffers as the layout definition says, and
rejects every invalid argument with the documented status before launching
anything (these calls never reach the GPU, so they run without one)."""
import ctypes
import os
import re

import pytest

import oracle
import paper_2605_17757_amd as ok

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "oscar.h")

FAKE = ctypes.c_void_p(0x10000)     # never dereferenced: validation fails first


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(oscar_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(ok.LIB_PATH):
        pytest.fail("liboscar.so is not built (run python paper_2605_17757_amd/build.py)")
    return ok.lib()


def test_exports_every_declared_symbol(L):
    declared = _declared_functions()
    assert set(declared) == set(ok.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def test_status_strings(L):
    assert ok.status_string(0) == "OSCAR_OK"
    assert ok.status_string(3) == "OSCAR_ERR_WORKSPACE_TOO_SMALL"
    assert ok.status_string(99) == "OSCAR_ERR_UNKNOWN"


def test_sizes_follow_layout_definition(L):
    for hkv in (1, 8):
        lay = ok.Layout(num_kv_heads=hkv, num_pages=10)
        # the oracle implements the same byte layout independently
        assert ok.page_bytes(lay) == hkv * oracle.page_head_bytes(128, 64, 32) == hkv * 6144
        assert ok.pool_bytes(lay) == 10 * hkv * 6144
        assert ok.bf16_pool_bytes(lay) == 10 * hkv * 2 * 64 * 128 * 2
    lay = ok.Layout(num_kv_heads=8, num_pages=10)
    ws = ok.decode_workspace_bytes(lay, 64, 32, 8)
    need = 64 * 32 * 128 * 4 + 64 * 32 * 8 * 128 * 4 + 64 * 32 * 8 * 2 * 4
    assert need <= ws <= need + 3 * 256 and ws % 256 == 0


def test_layout_validation(L):
    assert ok.layout_check(ok.Layout(8, 10)) == ok.OK
    assert ok.layout_check(ok.Layout(0, 10)) == ok.ERR_INVALID_ARG
    assert ok.layout_check(ok.Layout(8, 0)) == ok.ERR_INVALID_ARG
    assert ok.layout_check(ok.Layout(8, 10, head_dim=64)) == ok.ERR_UNSUPPORTED
    assert ok.layout_check(ok.Layout(8, 10, page_size=16)) == ok.ERR_UNSUPPORTED
    assert ok.layout_check(ok.Layout(8, 10, group_size=64)) == ok.OK
    assert ok.layout_check(ok.Layout(8, 10, group_size=128)) == ok.OK
    assert ok.layout_check(ok.Layout(8, 10, group_size=16)) == ok.ERR_UNSUPPORTED
    # block sizes follow the layout definition for every group size
    for G in (32, 64, 128):
        lay = ok.Layout(8, 10, group_size=G)
        assert ok.page_bytes(lay) == 8 * oracle.page_head_bytes(128, 64, G) == 8 * (4096 + 2 * (128 // G) * 256)
    assert ok.layout_check(ok.Layout(8, 10, group_size=48)) == ok.ERR_INVALID_ARG   # G does not divide d
    assert L.oscar_layout_check(None) == ok.ERR_INVALID_ARG
    assert ok.page_bytes(ok.Layout(0, 10)) == 0


def _append(L, lay, n_tok=4, clip_k=0.9, clip_v=0.9, pages=FAKE, k=FAKE, slots=FAKE):
    return L.oscar_kv_append(ctypes.byref(lay), pages, k, FAKE, slots, n_tok, FAKE, FAKE,
                             clip_k, clip_v, None)


def test_append_rejects_invalid_arguments(L):
    lay = ok.Layout(8, 10)
    assert _append(L, lay, clip_k=0.0) == ok.ERR_INVALID_ARG
    assert _append(L, lay, clip_v=1.5) == ok.ERR_INVALID_ARG
    assert _append(L, lay, clip_k=float("nan")) == ok.ERR_INVALID_ARG
    assert _append(L, lay, n_tok=-1) == ok.ERR_INVALID_ARG
    assert _append(L, lay, pages=None) == ok.ERR_INVALID_ARG
    assert _append(L, lay, slots=None) == ok.ERR_INVALID_ARG
    assert _append(L, lay, k=ctypes.c_void_p(0x10001)) == ok.ERR_INVALID_ARG     # misaligned
    assert _append(L, ok.Layout(8, 10, head_dim=256)) == ok.ERR_UNSUPPORTED
    # zero tokens: nothing to do, nothing launched
    assert _append(L, lay, n_tok=0, pages=None) == ok.OK


def _decode(L, lay, B=2, Hq=32, mp=4, S=2, ws_bytes=1 << 30, out_dtype=0, sm=0.088,
            ws=FAKE, q=FAKE):
    return L.oscar_decode_attn(ctypes.byref(lay), FAKE, q, B, Hq, FAKE, mp, FAKE, FAKE, FAKE,
                               sm, S, ws, ws_bytes, FAKE, out_dtype, None)


def test_decode_rejects_invalid_arguments(L):
    lay = ok.Layout(8, 10)
    assert _decode(L, lay, Hq=30) == ok.ERR_INVALID_ARG          # Hq % Hkv
    assert _decode(L, lay, Hq=8 * 17) == ok.ERR_UNSUPPORTED      # > 16 heads per kv-head
    assert _decode(L, lay, B=0) == ok.ERR_INVALID_ARG
    assert _decode(L, lay, S=-1) == ok.ERR_INVALID_ARG
    assert _decode(L, lay, mp=0) == ok.ERR_INVALID_ARG
    assert _decode(L, lay, out_dtype=7) == ok.ERR_INVALID_ARG
    assert _decode(L, lay, sm=float("inf")) == ok.ERR_INVALID_ARG
    assert _decode(L, lay, q=None) == ok.ERR_INVALID_ARG
    assert _decode(L, lay, ws=ctypes.c_void_p(0x10010)) == ok.ERR_INVALID_ARG   # not 256-aligned
    need = ok.decode_workspace_bytes(lay, 2, 32, 2)
    assert _decode(L, lay, ws_bytes=need - 1) == ok.ERR_WORKSPACE_TOO_SMALL
    assert _decode(L, ok.Layout(8, 10, page_size=32)) == ok.ERR_UNSUPPORTED
    # default split count on an invalid layout reports the layout error
    assert _decode(L, ok.Layout(0, 10), S=0) == ok.ERR_INVALID_ARG
    assert L.oscar_bf16_decode_attn(ctypes.byref(lay), FAKE, FAKE, 2, 30, FAKE, 4, FAKE, 0.088,
                                    2, FAKE, 1 << 30, FAKE, 0, None) == ok.ERR_INVALID_ARG


def _step(L, lay, n_new=4, clip_k=0.9, B=2, Hq=32, S=2, ws_bytes=1 << 30, k=FAKE, slots=FAKE):
    return L.oscar_decode_step(ctypes.byref(lay), FAKE, k, FAKE, slots, n_new, clip_k, 0.9, FAKE,
                               B, Hq, FAKE, 4, FAKE, FAKE, FAKE, 0.088, S, FAKE, ws_bytes, FAKE,
                               0, None)


def test_decode_step_validates_both_halves(L):
    lay = ok.Layout(8, 10)
    assert _step(L, lay, clip_k=2.0) == ok.ERR_INVALID_ARG          # append half
    assert _step(L, lay, n_new=-1) == ok.ERR_INVALID_ARG
    assert _step(L, lay, k=None) == ok.ERR_INVALID_ARG
    assert _step(L, lay, slots=ctypes.c_void_p(0x10004)) == ok.ERR_INVALID_ARG  # misaligned
    assert _step(L, lay, Hq=30) == ok.ERR_INVALID_ARG               # decode half
    assert _step(L, lay, S=-1) == ok.ERR_INVALID_ARG
    need = ok.decode_workspace_bytes(lay, 2, 32, 2)
    assert _step(L, lay, ws_bytes=need - 1) == ok.ERR_WORKSPACE_TOO_SMALL
    assert _step(L, ok.Layout(8, 10, head_dim=64)) == ok.ERR_UNSUPPORTED


def test_stage_entry_points_validate(L):
    lay = ok.Layout(8, 10)
    need = ok.decode_workspace_bytes(lay, 2, 32, 2)
    assert L.oscar_decode_prepare(ctypes.byref(lay), FAKE, 2, 32, FAKE, 0.088, 2, FAKE,
                                  need - 1, None) == ok.ERR_WORKSPACE_TOO_SMALL
    assert L.oscar_decode_split(ctypes.byref(lay), None, 2, 32, FAKE, 4, FAKE, 2, FAKE, need,
                                None) == ok.ERR_INVALID_ARG
    assert L.oscar_decode_reduce(ctypes.byref(lay), 2, 32, FAKE, 2, FAKE, need, FAKE, 5,
                                 None) == ok.ERR_INVALID_ARG


def test_default_num_splits_bounds(L):
    lay = ok.Layout(8, 10)
    assert ok.default_num_splits(lay, 64, 32, 32768) >= 1
    # never fewer than two pages per split
    assert ok.default_num_splits(lay, 1, 32, 128) == 1
    assert ok.default_num_splits(lay, 1, 32, 8192) <= 8192 // 64 // 2


def test_mixed_sizes(L):
    lay = ok.Layout(8, 10)
    for B, S0, W_ in ((64, 64, 256), (3, 20, 100), (1, 0, 0), (2, 0, 64)):
        # the oracle sizes the same segment store independently
        assert ok.seg_bytes(lay, B, S0, W_) == 2 * oracle.seg_elems(d=128, Hkv=8, B=B, S0=S0, W=W_)
    assert ok.seg_bytes(lay, 64, 64, 256) == 64 * 8 * 2 * 320 * 128 * 2
    assert ok.seg_bytes(lay, 1, -1, 4) == 0
    assert ok.seg_bytes(lay, 1, 4, -1) == 0
    assert ok.seg_bytes(lay, 1, 60000, 6000) == 0      # S0 + W > 65536
    assert ok.seg_bytes(lay, 0, 4, 4) == 0
    # rows of num_splits + 1 partial states
    assert ok.mixed_workspace_bytes(lay, 64, 32, 8) == ok.decode_workspace_bytes(lay, 64, 32, 9)
    assert ok.mixed_workspace_bytes(lay, 64, 30, 8) == 0


def _mixed_append(L, lay, n_tok=4, S0=64, W_=256, seg=FAKE, B=2, clip=0.9, pos=FAKE, mp=4):
    return L.oscar_mixed_append(ctypes.byref(lay), FAKE, seg, B, S0, W_, FAKE, FAKE, FAKE, pos,
                                n_tok, FAKE, mp, FAKE, FAKE, FAKE, clip, 0.9, None)


def test_mixed_append_rejects_invalid_arguments(L):
    lay = ok.Layout(8, 10)
    assert _mixed_append(L, lay, S0=-1) == ok.ERR_INVALID_ARG
    assert _mixed_append(L, lay, W_=-5) == ok.ERR_INVALID_ARG
    assert _mixed_append(L, lay, S0=65536, W_=1) == ok.ERR_INVALID_ARG
    assert _mixed_append(L, lay, seg=None) == ok.ERR_INVALID_ARG         # segments need a store
    assert _mixed_append(L, lay, seg=ctypes.c_void_p(0x10008)) == ok.ERR_INVALID_ARG
    assert _mixed_append(L, lay, pos=ctypes.c_void_p(0x10004)) == ok.ERR_INVALID_ARG
    assert _mixed_append(L, lay, B=0) == ok.ERR_INVALID_ARG
    assert _mixed_append(L, lay, clip=0.0) == ok.ERR_INVALID_ARG
    assert _mixed_append(L, lay, mp=0) == ok.ERR_INVALID_ARG
    assert _mixed_append(L, lay, n_tok=-1) == ok.ERR_INVALID_ARG
    assert _mixed_append(L, ok.Layout(8, 10, head_dim=64)) == ok.ERR_UNSUPPORTED
    assert _mixed_append(L, lay, n_tok=0) == ok.OK                         # nothing launched


def _mixed_decode(L, lay, step=False, S0=64, W_=256, seg=FAKE, B=2, Hq=32, S=2,
                  ws_bytes=1 << 30, k=FAKE, clip=0.9):
    if step:
        return L.oscar_decode_step_mixed(ctypes.byref(lay), FAKE, seg, S0, W_, k, FAKE, clip, 0.9,
                                         FAKE, B, Hq, FAKE, 4, FAKE, FAKE, FAKE, 0.088, S, FAKE,
                                         ws_bytes, FAKE, 0, None)
    return L.oscar_decode_attn_mixed(ctypes.byref(lay), FAKE, seg, S0, W_, FAKE, B, Hq, FAKE, 4,
                                     FAKE, FAKE, FAKE, 0.088, S, FAKE, ws_bytes, FAKE, 0, None)


@pytest.mark.parametrize("step", [False, True])
def test_mixed_decode_rejects_invalid_arguments(L, step):
    lay = ok.Layout(8, 10)
    assert _mixed_decode(L, lay, step, S0=-1) == ok.ERR_INVALID_ARG
    assert _mixed_decode(L, lay, step, seg=None) == ok.ERR_INVALID_ARG
    assert _mixed_decode(L, lay, step, Hq=30) == ok.ERR_INVALID_ARG
    assert _mixed_decode(L, lay, step, Hq=8 * 17) == ok.ERR_UNSUPPORTED
    assert _mixed_decode(L, lay, step, S=-1) == ok.ERR_INVALID_ARG
    # the plain workspace (num_splits slots a row) is one slot short
    plain = ok.decode_workspace_bytes(lay, 2, 32, 2)
    assert _mixed_decode(L, lay, step, ws_bytes=plain) == ok.ERR_WORKSPACE_TOO_SMALL
    need = ok.mixed_workspace_bytes(lay, 2, 32, 2)
    assert _mixed_decode(L, lay, step, ws_bytes=need - 1) == ok.ERR_WORKSPACE_TOO_SMALL
    if step:
        assert _mixed_decode(L, lay, step, k=None) == ok.ERR_INVALID_ARG
        assert _mixed_decode(L, lay, step, clip=1.5) == ok.ERR_INVALID_ARG


def test_quantizer_format_fields(L):
    # the layout's quantizer fields: known values pass, others are invalid arguments
    for clip_mode in (ok.CLIP_GROUP_ABSMAX, ok.CLIP_TOKEN_QUANTILE):
        for meta in (ok.META_F16, ok.META_BF16):
            lay = ok.Layout(8, 10, clip_mode=clip_mode, meta_dtype=meta)
            assert ok.layout_check(lay) == ok.OK
            assert ok.page_bytes(lay) == 8 * 6144           # same bytes for both formats
    assert ok.layout_check(ok.Layout(8, 10, clip_mode=2)) == ok.ERR_INVALID_ARG
    assert ok.layout_check(ok.Layout(8, 10, meta_dtype=-1)) == ok.ERR_INVALID_ARG
    assert _append(L, ok.Layout(8, 10, meta_dtype=7)) == ok.ERR_INVALID_ARG
    # one rotation per KV head: 0 or 1
    assert ok.layout_check(ok.Layout(8, 10, rot_per_head=1)) == ok.OK
    assert ok.layout_check(ok.Layout(8, 10, rot_per_head=2)) == ok.ERR_INVALID_ARG
    assert ctypes.sizeof(ok.Layout) == 40      # 8 x int32 + 1 x int64, 8-byte aligned


def test_null_rotations_pass_validation(L):
    # R_k / R_v NULL are the identity: validation accepts them (nothing launched
    # for an empty append)
    lay = ok.Layout(8, 10)
    assert L.oscar_kv_append(ctypes.byref(lay), FAKE, FAKE, FAKE, FAKE, 0, None, None, 0.9, 0.9,
                             None) == ok.OK
    # a bad argument elsewhere is still reported with NULL rotations
    assert L.oscar_kv_append(ctypes.byref(lay), None, FAKE, FAKE, FAKE, 4, None, None, 0.9, 0.9,
                             None) == ok.ERR_INVALID_ARG
    assert L.oscar_decode_attn(ctypes.byref(lay), FAKE, FAKE, 2, 32, FAKE, 4, FAKE, None, None,
                               0.088, 2, FAKE, 16, FAKE, 0, None) == ok.ERR_WORKSPACE_TOO_SMALL


def test_calibration_sizes(L):
    T, Hq, Hkv = 8878, 32, 8
    ws = L.oscar_calib_workspace_bytes(T, Hq, Hkv)
    o_bytes = T * Hq * 128 * 4
    assert ws % 256 == 0 and ws >= o_bytes + 10 * 1024 * 4    # rows + >= one block's partials
    assert L.oscar_calib_workspace_bytes(0, Hq, Hkv) == 0
    assert L.oscar_calib_workspace_bytes(T, 12, 8) == 0          # 12 heads do not split into 8
    assert L.oscar_calib_workspace_bytes(T, 4, 8) == 0           # fewer query than KV heads
    rot1, rot2 = L.oscar_calib_rotation_workspace_bytes(1), L.oscar_calib_rotation_workspace_bytes(2)
    # per matrix: 32 sweeps x 127 rounds x 64 (c, s) pairs, the vectors and the diagonal
    per = 32 * 127 * 64 * 16 + 128 * 128 * 8 + 128 * 8
    assert per <= rot1 <= per + 5 * 256 and 2 * per <= rot2 <= 2 * per + 5 * 256
    assert L.oscar_calib_rotation_workspace_bytes(0) == 0
    assert L.oscar_calib_clip_workspace_bytes(T, Hkv, 21) > 0
    assert L.oscar_calib_clip_workspace_bytes(T, Hkv, 0) == 0
    assert L.oscar_calib_clip_workspace_bytes(T, Hkv, 33) == 0
    lay = ok.Layout(num_kv_heads=Hkv, num_pages=1)
    lw = L.oscar_calibrate_layer_workspace_bytes(ctypes.byref(lay), T, Hq, 21)
    assert lw >= ws + rot2 + 2 * 128 * 128 * 8 * 2
    assert L.oscar_calibrate_layer_workspace_bytes(ctypes.byref(lay), T, Hq, 40) == 0
    # one rotation per KV head: 2 Hkv matrices
    lph = ok.Layout(num_kv_heads=Hkv, num_pages=1, rot_per_head=1)
    lw_ph = L.oscar_calibrate_layer_workspace_bytes(ctypes.byref(lph), T, Hq, 21)
    assert lw_ph >= ws + L.oscar_calib_rotation_workspace_bytes(2 * Hkv)


def test_calibration_rejects_invalid_arguments(L):
    E, U, W = ok.ERR_INVALID_ARG, ok.ERR_UNSUPPORTED, ok.ERR_WORKSPACE_TOO_SMALL
    ws_n = L.oscar_calib_workspace_bytes(100, 8, 2)
    q = FAKE
    assert L.oscar_calib_query_cov(None, 100, 8, 2, FAKE, FAKE, ws_n, None) == E
    assert L.oscar_calib_query_cov(q, 0, 8, 2, FAKE, FAKE, ws_n, None) == E
    assert L.oscar_calib_query_cov(q, 100, 8, 3, FAKE, FAKE, ws_n, None) == E
    assert L.oscar_calib_query_cov(q, 100, 8, 2, FAKE, FAKE, ws_n - 1, None) == W
    assert L.oscar_calib_query_cov(ctypes.c_void_p(0x10008), 100, 8, 2, FAKE, FAKE, ws_n, None) == E
    assert L.oscar_calib_attn(q, q, None, 100, 8, 2, 1, FAKE, None) == E
    assert L.oscar_calib_attn(q, q, q, 100, 8, 16, 1, FAKE, None) == E
    assert L.oscar_calib_attn(q, q, q, 70000 * 64, 4, 1, 1, FAKE, None) == U   # > 65535 query tiles
    assert L.oscar_calib_score_cov(q, q, q, 100, 8, 2, 1, FAKE, FAKE, ws_n - 256, None) == W
    rw = L.oscar_calib_rotation_workspace_bytes(2)
    assert L.oscar_calib_rotation(FAKE, 0, FAKE, FAKE, None, None, None, FAKE, rw, None) == E
    assert L.oscar_calib_rotation(FAKE, 2, None, FAKE, None, None, None, FAKE, rw, None) == E
    assert L.oscar_calib_rotation(FAKE, 2, FAKE, FAKE, None, None, None, FAKE, rw - 1, None) == W
    lay = ok.Layout(num_kv_heads=2, num_pages=1)
    cw = L.oscar_calib_clip_workspace_bytes(100, 2, 21)
    assert L.oscar_calib_clip(ctypes.byref(lay), q, 100, None, FAKE, 0, FAKE, None, FAKE, cw, None) == E
    assert L.oscar_calib_clip(ctypes.byref(lay), q, 100, None, FAKE, 33, FAKE, None, FAKE, cw, None) == U
    assert L.oscar_calib_clip(ctypes.byref(lay), q, 100, None, None, 21, FAKE, None, FAKE, cw, None) == E
    assert L.oscar_calib_clip(ctypes.byref(lay), q, 100, None, FAKE, 21, FAKE, None, FAKE, cw - 1, None) == W
    bad = ok.Layout(num_kv_heads=2, num_pages=1, group_size=16)
    assert L.oscar_calib_clip(ctypes.byref(bad), q, 100, None, FAKE, 21, FAKE, None, FAKE, cw, None) == U
    lw = L.oscar_calibrate_layer_workspace_bytes(ctypes.byref(lay), 100, 8, 21)
    args = [q, q, q, 100, 8, 1, FAKE, 21, FAKE, FAKE, FAKE, None, None, FAKE]
    assert L.oscar_calibrate_layer(ctypes.byref(lay), *args, lw - 1, None) == W
    assert L.oscar_calibrate_layer(ctypes.byref(ok.Layout(num_kv_heads=3, num_pages=1)), *args, lw,
                                   None) == E
    args2 = list(args)
    args2[9] = None  # R_v
    assert L.oscar_calibrate_layer(ctypes.byref(lay), *args2, lw, None) == E


def test_read_probe_rejects_invalid_arguments(L):
    # every case returns before any HIP call (no device needed)
    buf = ctypes.c_void_p(1 << 20)  # 16-byte aligned, never dereferenced
    sink = ctypes.c_void_p(1 << 21)
    assert L.oscar_hbm_read_probe(None, 16, sink, 1, None) == ok.ERR_INVALID_ARG
    assert L.oscar_hbm_read_probe(buf, 16, None, 1, None) == ok.ERR_INVALID_ARG
    assert L.oscar_hbm_read_probe(buf, 16, sink, 0, None) == ok.ERR_INVALID_ARG
    assert L.oscar_hbm_read_probe(buf, 0, sink, 1, None) == ok.ERR_INVALID_ARG
    assert L.oscar_hbm_read_probe(buf, 24, sink, 1, None) == ok.ERR_INVALID_ARG      # not x16
    assert L.oscar_hbm_read_probe(ctypes.c_void_p((1 << 20) + 8), 16, sink, 1, None) == ok.ERR_INVALID_ARG
    X = L.oscar_hbm_read_probe_ex
    assert X(None, 16, sink, 1, 8, 0, None) == ok.ERR_INVALID_ARG
    assert X(buf, 16, sink, 1, 5, 0, None) == ok.ERR_INVALID_ARG          # 4, 8 or 16 loads
    assert X(buf, 16, sink, 1, 32, 0, None) == ok.ERR_INVALID_ARG
    assert X(buf, 16, sink, 1, 8, 4, None) == ok.ERR_INVALID_ARG          # unknown flag bit
    assert X(buf, 24, sink, 1, 8, 3, None) == ok.ERR_INVALID_ARG


def test_decode_noalloc_validates_before_touching_the_device(L):
    # invalid arguments and an oversized workspace return before the scratch
    # array's address is looked up (no device needed)
    lay = ok.Layout(8, 10)

    def call(B=2, Hq=32, S=2, q=FAKE, out_dtype=0, lay=lay):
        return L.oscar_decode_attn_noalloc(ctypes.byref(lay), FAKE, q, B, Hq, FAKE, 4, FAKE,
                                           FAKE, FAKE, 0.088, S, FAKE, out_dtype, None)

    assert call(Hq=30) == ok.ERR_INVALID_ARG
    assert call(B=0) == ok.ERR_INVALID_ARG
    assert call(S=-1) == ok.ERR_INVALID_ARG
    assert call(q=None) == ok.ERR_INVALID_ARG
    assert call(out_dtype=9) == ok.ERR_INVALID_ARG
    assert call(lay=ok.Layout(8, 10, page_size=32)) == ok.ERR_UNSUPPORTED
    assert ok.decode_workspace_bytes(lay, 4096, 64, 64) > ok.NOALLOC_SCRATCH_BYTES
    assert call(B=4096, Hq=64, S=64) == ok.ERR_WORKSPACE_TOO_SMALL
