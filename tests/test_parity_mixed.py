"""GPU parity of the mixed-precision cache (bf16 sink of S0 tokens and bf16
window of the W most recent tokens around the INT2 history; Sec. 4 "KV Cache
Layout"; Alg. 1 DecodeStep) against the oracle.

The GPU builds the cache the way a server does: oscar_mixed_append with a
sequence's prompt (tokens 0 .. n-2), then oscar_decode_step_mixed with token
n-1 (demoting the window's oldest token when the window is full).  The oracle
runs its decode loop from an empty cache, one token per step
(oracle.mixed_update).  Compared: every byte of the INT2 pool (bit-exact, with
the near-boundary rule of helpers.compare_pools), every element of the segment
store (bit-exact: bf16 copies), and every output element (2e-3 on fp32; the
bf16 output is the round-to-nearest-even of the fp32 one)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2605_17757_amd as ok
import workloads as W
from helpers import DECODE_TOL, Case, bits, compare_pools, log, max_abs

pytestmark = pytest.mark.gpu

D, P, G = 128, 64, 32


def _seg_np(seg: torch.Tensor) -> np.ndarray:
    return seg.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16).reshape(-1)


def _history(n, S0, W_):
    lo = min(S0, n)
    return lo, max(lo, n - W_)


class Mixed:
    """A workload and both sides' caches."""

    def __init__(self, cfg: W.Config, S0: int, W_: int):
        self.cfg, self.S0, self.W = cfg, S0, W_
        self.Rk, self.Rv = W.rotations(cfg)
        self.table, self.num_pages = W.block_table(cfg)
        self.kv = [W.cache_kv(cfg, b) for b in range(cfg.B)]
        self.q = W.queries(cfg)
        self.lay = ok.Layout(num_kv_heads=cfg.Hkv, num_pages=self.num_pages)
        self.Rk_d = torch.from_numpy(self.Rk).cuda()
        self.Rv_d = torch.from_numpy(self.Rv).cuda()
        self.table_d = torch.from_numpy(self.table).cuda()

    # ---- oracle: the decode loop from an empty cache ----
    def oracle_build(self, upto):
        cfg = self.cfg
        pages = np.zeros(ok.pool_bytes(self.lay), np.uint8)
        seg = np.zeros(oracle.seg_elems(d=D, Hkv=cfg.Hkv, B=cfg.B, S0=self.S0, W=self.W), np.uint16)
        chunk = cfg.Hkv * 2 * (self.S0 + self.W) * D
        for b in range(cfg.B):
            kb, vb = bits(self.kv[b][0]), bits(self.kv[b][1])
            seg_b = seg[b * chunk:(b + 1) * chunk]
            for n in range(1, int(upto[b]) + 1):
                oracle.mixed_update(pages, seg_b, d=D, Hkv=cfg.Hkv, P=P, G=G, S0=self.S0,
                                    W=self.W, k_new=kb[n - 1:n], v_new=vb[n - 1:n],
                                    block_table=self.table[b:b + 1],
                                    seq_lens=np.array([n], np.int32), Rk=self.Rk, Rv=self.Rv,
                                    clip_k=cfg.clip_k, clip_v=cfg.clip_v)
        return pages, seg

    def oracle_decode(self, pages, seg, lens):
        return oracle.decode_mixed(pages, seg, d=D, Hkv=self.cfg.Hkv, P=P, G=G, S0=self.S0,
                                   W=self.W, q=bits(self.q), block_table=self.table,
                                   seq_lens=np.asarray(lens, np.int32), Rk=self.Rk, Rv=self.Rv,
                                   sm_scale=self.cfg.sm_scale)

    # ---- GPU ----
    def gpu_prefill(self, lens_pre):
        """oscar_mixed_append of tokens [0, lens_pre[b]) of every sequence, one call."""
        cfg = self.cfg
        pool = ok.alloc_pool(self.lay)
        seg = ok.alloc_seg(self.lay, cfg.B, self.S0, self.W)
        ks, vs, si, ps = [], [], [], []
        for b in range(cfg.B):
            n = int(lens_pre[b])
            ks.append(self.kv[b][0][:n])
            vs.append(self.kv[b][1][:n])
            si.append(np.full(n, b, np.int32))
            ps.append(np.arange(n, dtype=np.int64))
        k = torch.cat(ks).cuda()
        if k.shape[0]:
            ok.mixed_append(self.lay, pool, seg, self.S0, self.W, k, torch.cat(vs).cuda(),
                            torch.from_numpy(np.concatenate(si)).cuda(),
                            torch.from_numpy(np.concatenate(ps)).cuda(), self.table_d,
                            torch.from_numpy(np.asarray(lens_pre, np.int32)).cuda(), self.Rk_d,
                            self.Rv_d, cfg.clip_k, cfg.clip_v)
        return pool, seg

    def gpu_step(self, pool, seg, lens, num_splits=0, out_dtype=torch.float32):
        """oscar_decode_step_mixed with token lens[b] - 1 of every sequence."""
        cfg = self.cfg
        kn = torch.stack([self.kv[b][0][int(lens[b]) - 1] for b in range(cfg.B)]).cuda()
        vn = torch.stack([self.kv[b][1][int(lens[b]) - 1] for b in range(cfg.B)]).cuda()
        S = num_splits or ok.default_num_splits(self.lay, cfg.B, cfg.Hq, self.table.shape[1] * P)
        ws = ok.alloc_mixed_workspace(self.lay, cfg.B, cfg.Hq, S)
        out = torch.empty(cfg.B, cfg.Hq, D, dtype=out_dtype, device="cuda")
        ok.decode_step_mixed(self.lay, pool, seg, self.S0, self.W, kn, vn, cfg.clip_k, cfg.clip_v,
                             self.q.cuda(), self.table_d,
                             torch.from_numpy(np.asarray(lens, np.int32)).cuda(), self.Rk_d,
                             self.Rv_d, cfg.sm_scale, S, ws, out)
        torch.cuda.synchronize()
        return out

    def gpu_decode(self, pool, seg, lens, num_splits=0, out_dtype=torch.float32):
        cfg = self.cfg
        S = num_splits or ok.default_num_splits(self.lay, cfg.B, cfg.Hq, self.table.shape[1] * P)
        ws = ok.alloc_mixed_workspace(self.lay, cfg.B, cfg.Hq, S)
        out = torch.empty(cfg.B, cfg.Hq, D, dtype=out_dtype, device="cuda")
        ok.decode_attn_mixed(self.lay, pool, seg, self.S0, self.W, self.q.cuda(), self.table_d,
                             torch.from_numpy(np.asarray(lens, np.int32)).cuda(), self.Rk_d,
                             self.Rv_d, cfg.sm_scale, S, ws, out)
        torch.cuda.synchronize()
        return out

    def history_case(self, lens):
        """Case of the INT2 history rows (for compare_pools)."""
        ks, vs, sl = [], [], []
        for b in range(self.cfg.B):
            lo, hi = _history(int(lens[b]), self.S0, self.W)
            ks.append(self.kv[b][0][lo:hi])
            vs.append(self.kv[b][1][lo:hi])
            sl.append(W.slots_for(self.table, b, np.arange(lo, hi)))
        return Case(self.cfg, self.Rk, self.Rv, self.table, self.num_pages, self.q, torch.cat(ks),
                    torch.cat(vs), np.concatenate(sl))

    def compare_state(self, pool, seg, ora_pages, ora_seg, lens):
        nd, nt = compare_pools(pool.cpu().numpy(), ora_pages, self.history_case(lens))
        log("  pool: differing bytes", nd, "tolerated near-boundary elements", nt)
        gs = _seg_np(seg)
        assert gs.shape == ora_seg.shape
        bad = np.nonzero(gs != ora_seg)[0]
        assert bad.size == 0, "segment store differs at %d elements, first %s" % (bad.size, bad[:5])


def _mixed_cfg(name, lens, Hq=8, Hkv=2, seed_index=200):
    return W.custom(name, len(lens), Hq, Hkv, lens, seed_index=seed_index, k_outliers=(5, 90),
                    v_outliers=(17,))


# (S0, W, lengths): lengths around every boundary of the segments: n < S0,
# n = S0, S0 < n < S0 + W, n = S0 + W (no demotion yet), n = S0 + W + 1 (the
# first demotion happens in the step), and long histories with a partial first
# page (S0 % 64 != 0) and partial last pages.
CASES = [
    (64, 256, [1, 30, 64, 65, 200, 320, 321, 385, 1000, 1537]),
    (20, 100, [1, 7, 20, 21, 119, 120, 121, 150, 333, 700]),
    (0, 64, [1, 63, 64, 65, 129, 500]),
    (48, 0, [1, 47, 48, 49, 300]),
    (5, 3, [1, 4, 5, 6, 8, 9, 70, 200]),
]


@pytest.mark.parametrize("S0,W_,lens", CASES)
def test_mixed_prefill_then_step(S0, W_, lens):
    cfg = _mixed_cfg("mixed_s%d_w%d" % (S0, W_), lens)
    m = Mixed(cfg, S0, W_)
    lens = np.asarray(lens, np.int32)
    log("case S0", S0, "W", W_, "lens", list(lens))
    pool, seg = m.gpu_prefill(lens - 1)
    out = m.gpu_step(pool, seg, lens)
    ora_pages, ora_seg = m.oracle_build(lens)
    m.compare_state(pool, seg, ora_pages, ora_seg, lens)
    ref = m.oracle_decode(ora_pages, ora_seg, lens)
    err = max_abs(out, ref)
    log("  step decode max|err| = %.3g" % err)
    assert err <= DECODE_TOL
    # attention alone over the same cache, several split counts, bf16 output
    for S in (1, 3, 0):
        o2 = m.gpu_decode(pool, seg, lens, num_splits=S)
        e2 = max_abs(o2, ref)
        log("  decode_attn_mixed splits %d max|err| = %.3g" % (S, e2))
        assert e2 <= DECODE_TOL
    ob = m.gpu_decode(pool, seg, lens, num_splits=3, out_dtype=torch.bfloat16)
    o3 = m.gpu_decode(pool, seg, lens, num_splits=3)
    assert torch.equal(ob.cpu(), o3.cpu().to(torch.bfloat16))


@pytest.mark.parametrize("g", [1, 3, 6, 8, 10, 12, 14, 16])
def test_mixed_gqa_ratios(g):
    """Every query-head grouping the kernels specialize for (4, 8, 12 and 16 heads
    per block, the wide ones also with padding heads), with ragged lengths and a
    window that spans several 64-slot chunks."""
    S0, W_ = 20, 300
    lens = [1, 19, 21, 320, 321, 333, 900]
    cfg = W.custom("mixed_gqa%d" % g, len(lens), 2 * g, 2, lens, seed_index=210 + g,
                   k_outliers=(5, 90), v_outliers=(17,))
    m = Mixed(cfg, S0, W_)
    lens = np.asarray(lens, np.int32)
    pool, seg = m.gpu_prefill(lens - 1)
    out = m.gpu_step(pool, seg, lens, num_splits=3)
    ora_pages, ora_seg = m.oracle_build(lens)
    m.compare_state(pool, seg, ora_pages, ora_seg, lens)
    err = max_abs(out, m.oracle_decode(ora_pages, ora_seg, lens))
    log("  g %d max|err| = %.3g" % (g, err))
    assert err <= DECODE_TOL


def test_mixed_reduce_16_row_blocks():
    """4096 (sequence, head) rows, so that the merge runs 16 rows per block, with the
    bf16 segments' slot (sink 4, window 8) added after the back-rotation."""
    S0, W_ = 4, 8
    lens = np.random.default_rng(220).integers(1, 81, size=128).astype(np.int32)
    cfg = W.custom("mixed_rows4096", 128, 32, 8, lens, seed_index=220, k_outliers=(5, 90),
                   v_outliers=(17,))
    m = Mixed(cfg, S0, W_)
    pool, seg = m.gpu_prefill(lens - 1)
    out = m.gpu_step(pool, seg, lens, num_splits=3)
    ora_pages, ora_seg = m.oracle_build(lens)
    m.compare_state(pool, seg, ora_pages, ora_seg, lens)
    ref = m.oracle_decode(ora_pages, ora_seg, lens)
    err = max_abs(out, ref)
    log("  rows 4096 max|err| = %.3g" % err)
    assert err <= DECODE_TOL
    ob = m.gpu_decode(pool, seg, lens, num_splits=3, out_dtype=torch.bfloat16)
    o3 = m.gpu_decode(pool, seg, lens, num_splits=3)
    assert max_abs(o3, ref) <= DECODE_TOL
    assert torch.equal(ob.cpu(), o3.cpu().to(torch.bfloat16))


def test_mixed_many_steps_demote_in_order():
    """A decode loop on the GPU: prefill, then 150 steps, each compared with the
    oracle's loop (the window wraps, pages fill, tokens are demoted one by one)."""
    S0, W_ = 20, 50
    lens_end = np.array([60, 75, 140, 230], np.int32)
    cfg = _mixed_cfg("mixed_steps", lens_end, seed_index=201)
    m = Mixed(cfg, S0, W_)
    steps = 150
    lens0 = np.maximum(lens_end - steps, 0)
    pool, seg = m.gpu_prefill(lens0)
    ora_pages, ora_seg = m.oracle_build(lens0)
    chunk = cfg.Hkv * 2 * (S0 + W_) * D
    worst = 0.0
    for i in range(1, steps + 1):
        lens = np.maximum(lens_end - steps + i, 0).astype(np.int32)
        # sequences that have not started keep length 0: no update, zero output
        active = [b for b in range(cfg.B) if lens[b] > lens0[b]]
        out = m.gpu_step(pool, seg, lens, num_splits=3)
        for b in active:
            n = int(lens[b])
            oracle.mixed_update(ora_pages, ora_seg[b * chunk:(b + 1) * chunk], d=D, Hkv=cfg.Hkv,
                                P=P, G=G, S0=S0, W=W_, k_new=bits(m.kv[b][0][n - 1:n]),
                                v_new=bits(m.kv[b][1][n - 1:n]), block_table=m.table[b:b + 1],
                                seq_lens=np.array([n], np.int32), Rk=m.Rk, Rv=m.Rv,
                                clip_k=cfg.clip_k, clip_v=cfg.clip_v)
        lens0 = lens
        live = lens > 0
        ref = m.oracle_decode(ora_pages, ora_seg, np.maximum(lens, 1))
        got = out.cpu().numpy()
        err = float(np.max(np.abs(got[live] - ref[live])))
        assert np.all(got[~live] == 0.0)
        worst = max(worst, err)
        assert err <= DECODE_TOL, (i, err)
        if i % 50 == 0 or i == steps:
            m.compare_state(pool, seg, ora_pages, ora_seg, lens)
    log("  150 steps: worst max|err| = %.3g" % worst)


def test_mixed_no_history_window_covers_everything():
    """W larger than every sequence: no INT2 page is read (all splits empty), and the
    result is the bf16 baseline's."""
    S0, W_ = 64, 1024
    lens = np.array([1, 64, 65, 700, 1088], np.int32)
    cfg = _mixed_cfg("mixed_nohist", lens, seed_index=202)
    m = Mixed(cfg, S0, W_)
    pool, seg = m.gpu_prefill(lens - 1)
    out = m.gpu_step(pool, seg, lens, num_splits=4)
    ora_pages, ora_seg = m.oracle_build(lens)
    m.compare_state(pool, seg, ora_pages, ora_seg, lens)
    assert not pool.any().item()  # nothing quantized
    err = max_abs(out, m.oracle_decode(ora_pages, ora_seg, lens))
    log("  max|err| = %.3g" % err)
    assert err <= DECODE_TOL
    # every token bf16: the same attention as the bf16 paged-decode baseline over the
    # same rows (two fp32 evaluations in different orders)
    bf_pool = torch.zeros(ok.bf16_pool_bytes(m.lay) // 2, dtype=torch.bfloat16, device="cuda")
    for b in range(cfg.B):
        n = int(lens[b])
        ok.bf16_kv_append(m.lay, bf_pool, m.kv[b][0][:n].cuda(), m.kv[b][1][:n].cuda(),
                          torch.from_numpy(W.slots_for(m.table, b, np.arange(n))).cuda())
    ws = ok.alloc_workspace(m.lay, cfg.B, cfg.Hq, 4)
    bout = torch.empty_like(out)
    ok.bf16_decode_attn(m.lay, bf_pool, m.q.cuda(), m.table_d, torch.from_numpy(lens).cuda(),
                        cfg.sm_scale, 4, ws, bout)
    torch.cuda.synchronize()
    d = float((out - bout).abs().max())
    log("  vs bf16 baseline max|diff| = %.3g" % d)
    assert d <= 1e-4


def test_mixed_zero_segments_equal_int2_path_bitwise():
    """S0 = W = 0: the mixed entry points compute exactly what the INT2 path does."""
    cfg = W.custom("mixed_zero", 4, 32, 8, [1, 100, 2049, 3000], seed_index=203,
                   k_outliers=(7,), v_outliers=(99,))
    m = Mixed(cfg, 0, 0)
    lens = cfg.lens
    pool_m, _ = m.gpu_prefill(lens - 1)
    # the same prompt through oscar_kv_append
    pool_p = ok.alloc_pool(m.lay)
    for b in range(cfg.B):
        n = int(lens[b]) - 1
        if n:
            ok.kv_append(m.lay, pool_p, m.kv[b][0][:n].cuda(), m.kv[b][1][:n].cuda(),
                         torch.from_numpy(W.slots_for(m.table, b, np.arange(n))).cuda(), m.Rk_d,
                         m.Rv_d, cfg.clip_k, cfg.clip_v)
    torch.cuda.synchronize()
    assert torch.equal(pool_m, pool_p)
    S = 5
    out_m = m.gpu_step(pool_m, None, lens, num_splits=S)
    kn = torch.stack([m.kv[b][0][int(lens[b]) - 1] for b in range(cfg.B)]).cuda()
    vn = torch.stack([m.kv[b][1][int(lens[b]) - 1] for b in range(cfg.B)]).cuda()
    slots = np.array([W.slots_for(m.table, b, [int(lens[b]) - 1])[0] for b in range(cfg.B)])
    ws = ok.alloc_workspace(m.lay, cfg.B, cfg.Hq, S)
    out_p = torch.empty_like(out_m)
    ok.decode_step(m.lay, pool_p, kn, vn, torch.from_numpy(slots).cuda(), cfg.clip_k, cfg.clip_v,
                   m.q.cuda(), m.table_d, torch.from_numpy(lens).cuda(), m.Rk_d, m.Rv_d,
                   cfg.sm_scale, S, ws, out_p)
    torch.cuda.synchronize()
    assert torch.equal(pool_m, pool_p)
    assert torch.equal(out_m, out_p)


def test_mixed_full_size_bench_workload_sampled():
    """64 sequences of 16k-32k tokens, 32/8 heads, S0 = 64, W = 256, in the launch
    configuration the benchmark times: prompt through oscar_mixed_append, one
    oscar_decode_step_mixed.  The oracle builds the sampled sequences' cache
    directly (segment rows by oracle.seg_write, history by oracle.kv_append: the
    oracle's pins show this equals its one-token-per-step loop) and decodes them."""
    S0, W_ = 64, 256
    cfg = W.config(2, batch=64)
    B, Hq, Hkv = cfg.B, cfg.Hq, cfg.Hkv
    lens = cfg.lens.astype(np.int32)
    table, num_pages = W.block_table(cfg)
    lay = ok.Layout(num_kv_heads=Hkv, num_pages=num_pages)
    Rk_np, Rv_np = W.rotations(cfg)
    Rk, Rv = torch.from_numpy(Rk_np).cuda(), torch.from_numpy(Rv_np).cuda()
    sample = sorted({0, int(np.argmax(lens)), int(np.argmin(lens))})
    log("full size mixed: B", B, "pages", num_pages, "sampled", sample)
    host_kv = {b: W.cache_kv(cfg, b) for b in sample}
    pool = ok.alloc_pool(lay)
    seg = ok.alloc_seg(lay, B, S0, W_)
    table_d = torch.from_numpy(table).cuda()
    pre = torch.from_numpy(lens - 1).cuda()
    kn = torch.empty(B, Hkv, D, dtype=torch.bfloat16, device="cuda")
    vn = torch.empty_like(kn)
    for b in range(B):
        if b in host_kv:
            k, v = host_kv[b][0].cuda(), host_kv[b][1].cuda()
        else:
            k, v = W.cache_kv(cfg, b, device="cuda")
        n = int(lens[b])
        ok.mixed_append(lay, pool, seg, S0, W_, k[:n - 1], v[:n - 1],
                        torch.full((n - 1,), b, dtype=torch.int32, device="cuda"),
                        torch.arange(n - 1, dtype=torch.int64, device="cuda"), table_d, pre, Rk, Rv,
                        cfg.clip_k, cfg.clip_v)
        kn[b], vn[b] = k[n - 1], v[n - 1]
        del k, v
    S = ok.default_num_splits(lay, B, Hq, int(table.shape[1]) * P)
    ws = ok.alloc_mixed_workspace(lay, B, Hq, S)
    q = W.queries(cfg)
    out = torch.empty(B, Hq, D, dtype=torch.float32, device="cuda")
    ok.decode_step_mixed(lay, pool, seg, S0, W_, kn, vn, cfg.clip_k, cfg.clip_v, q.cuda(), table_d,
                         torch.from_numpy(lens).cuda(), Rk, Rv, cfg.sm_scale, S, ws, out)
    torch.cuda.synchronize()
    log("  gpu done, splits", S)

    ora = np.zeros(ok.pool_bytes(lay), np.uint8)
    oseg = np.zeros(oracle.seg_elems(d=D, Hkv=Hkv, B=B, S0=S0, W=W_), np.uint16)
    ks, vs, ss = [], [], []
    for b in sample:
        k, v = host_kv[b]
        n = int(lens[b])
        lo, hi = _history(n, S0, W_)
        keep = np.r_[0:lo, hi:n]
        kt = torch.from_numpy(keep)
        oracle.seg_write(oseg, d=D, Hkv=Hkv, B=B, S0=S0, W=W_, k=bits(k[kt]), v=bits(v[kt]),
                         seq_idx=np.full(keep.size, b, np.int32), pos=keep.astype(np.int64))
        sl = W.slots_for(table, b, np.arange(lo, hi))
        oracle.kv_append(ora, d=D, Hkv=Hkv, P=P, G=G, k=bits(k[lo:hi]), v=bits(v[lo:hi]),
                         slot_mapping=sl, Rk=Rk_np, Rv=Rv_np, clip_k=cfg.clip_k,
                         clip_v=cfg.clip_v)
        ks.append(k[lo:hi])
        vs.append(v[lo:hi])
        ss.append(sl)
    pairs = np.array([(b, h) for b in sample for h in range(Hq)], np.int32)
    ref = oracle.decode_mixed(ora, oseg, d=D, Hkv=Hkv, P=P, G=G, S0=S0, W=W_, q=bits(q),
                              block_table=table, seq_lens=lens, Rk=Rk_np, Rv=Rv_np,
                              sm_scale=cfg.sm_scale, pairs=pairs)
    got = out[torch.as_tensor(np.asarray(sample))].reshape(-1, D)
    err = max_abs(got, ref)
    log("  decode max|err| over %d rows = %.3g" % (len(pairs), err))
    assert err <= DECODE_TOL
    # segment rows and pages of the sampled sequences
    gseg = _seg_np(seg).reshape(B, -1)
    assert np.array_equal(gseg[sample], oseg.reshape(B, -1)[sample])
    bph = ok.page_bytes(lay)
    gpu_sel = np.zeros_like(ora)
    pool_pages = pool.view(num_pages, bph)
    for b in sample:
        ids = table[b, :(int(lens[b]) + 63) // 64]
        gpu_sel.reshape(num_pages, bph)[ids] = pool_pages[torch.from_numpy(ids).cuda()].cpu().numpy()
    case = Case(cfg, Rk_np, Rv_np, table, num_pages, q, torch.cat(ks), torch.cat(vs),
                np.concatenate(ss))
    nd, nt = compare_pools(gpu_sel, ora, case)
    log("  pool: differing bytes", nd, "tolerated near-boundary elements", nt)
