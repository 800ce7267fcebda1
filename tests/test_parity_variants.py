"""GPU parity of the quantizer variants (App. "Scale Determination and Per-token
Clipping Details"; Sec. 4 "KV Cache Update") against the oracle, through the C
ABI: bfloat16 scale/zero metadata, the per-token quantile clip threshold, groups
of 64 and 128 channels, all three together (the format the paper states: G = 128,
bf16 scale/zero, quantile clip), and identity rotations (R_V absorbed into the
projection weights; no rotation at all).  Page bytes bit-exact (with
the near-boundary rule of helpers.compare_pools, applied in the variant's own
arithmetic); decode within 2e-3 on the fp32 output."""
import numpy as np
import pytest
import torch

import oracle
import paper_2605_17757_amd as ok
import workloads as W
from helpers import DECODE_TOL, Case, bits, compare_pools, log, max_abs

pytestmark = pytest.mark.gpu

D, P = 128, 64

# name -> (meta_dtype, clip_mode, rotate K, rotate V, group size, one rotation per
# KV head).  The paper's stated format: groups of 128 channels, bf16 scale/zero,
# per-token quantile clip.
VARIANTS = {
    "bf16_meta": (1, 0, True, True, 32, 0),
    "token_quantile": (0, 1, True, True, 32, 0),
    "g64": (0, 0, True, True, 64, 0),
    "g128": (0, 0, True, True, 128, 0),
    "paper_format": (1, 1, True, True, 128, 0),
    "paper_format_g64": (1, 1, True, True, 64, 0),
    "identity_v": (0, 0, True, False, 32, 0),
    "identity_kv_paper_format": (1, 1, False, False, 128, 0),
    "per_head_r": (0, 0, True, True, 32, 1),
    "per_head_paper_format": (1, 1, True, True, 128, 1),
    "per_head_k_identity_v": (0, 0, True, False, 32, 1),
}


def per_head_rotations(cfg: W.Config):
    """One seeded rotation per KV head for K and for V: [Hkv, d, d] each."""
    return (np.stack([W.rotation(cfg.seed + W.S_RK + 7919 * h, cfg.d) for h in range(cfg.Hkv)]),
            np.stack([W.rotation(cfg.seed + W.S_RV + 7919 * h, cfg.d) for h in range(cfg.Hkv)]))


class VCase:
    def __init__(self, cfg: W.Config, variant: str):
        self.cfg = cfg
        self.meta, self.clip, rk, rv, self.G, self.rph = VARIANTS[variant]
        Rk, Rv = per_head_rotations(cfg) if self.rph else W.rotations(cfg)
        self.Rk = Rk if rk else None
        self.Rv = Rv if rv else None
        self.table, self.num_pages = W.block_table(cfg)
        self.lay = ok.Layout(num_kv_heads=cfg.Hkv, num_pages=self.num_pages, group_size=self.G,
                             clip_mode=self.clip, meta_dtype=self.meta, rot_per_head=self.rph)
        self.kv = [W.cache_kv(cfg, b) for b in range(cfg.B)]
        self.q = W.queries(cfg)
        self.Rk_d = None if self.Rk is None else torch.from_numpy(self.Rk).cuda()
        self.Rv_d = None if self.Rv is None else torch.from_numpy(self.Rv).cuda()

    def slots(self, b, n):
        return W.slots_for(self.table, b, np.arange(n))

    def case(self, upto):
        ks = torch.cat([self.kv[b][0][:int(upto[b])] for b in range(self.cfg.B)])
        vs = torch.cat([self.kv[b][1][:int(upto[b])] for b in range(self.cfg.B)])
        sl = np.concatenate([self.slots(b, int(upto[b])) for b in range(self.cfg.B)])
        return Case(self.cfg, self.Rk, self.Rv, self.table, self.num_pages, self.q, ks, vs, sl)

    def gpu_append(self, upto, pool=None):
        pool = ok.alloc_pool(self.lay) if pool is None else pool
        for b in range(self.cfg.B):
            n = int(upto[b])
            if n:
                ok.kv_append(self.lay, pool, self.kv[b][0][:n].cuda(), self.kv[b][1][:n].cuda(),
                             torch.from_numpy(self.slots(b, n)).cuda(), self.Rk_d, self.Rv_d,
                             self.cfg.clip_k, self.cfg.clip_v)
        torch.cuda.synchronize()
        return pool

    def oracle_append(self, upto):
        c = self.case(upto)
        pool = np.zeros(ok.pool_bytes(self.lay), np.uint8)
        oracle.kv_append(pool, d=D, Hkv=self.cfg.Hkv, P=P, G=self.G, k=bits(c.k), v=bits(c.v),
                         slot_mapping=c.slots, Rk=self.Rk, Rv=self.Rv, clip_k=self.cfg.clip_k,
                         clip_v=self.cfg.clip_v, meta=self.meta, clip=self.clip)
        return pool

    def oracle_decode(self, pool, lens):
        return oracle.decode(pool, d=D, Hkv=self.cfg.Hkv, P=P, G=self.G, q=bits(self.q),
                             block_table=self.table, seq_lens=np.asarray(lens, np.int32),
                             Rk=self.Rk, Rv=self.Rv, sm_scale=self.cfg.sm_scale, meta=self.meta)

    def gpu_decode(self, pool, lens, S, out_dtype=torch.float32):
        cfg = self.cfg
        ws = ok.alloc_workspace(self.lay, cfg.B, cfg.Hq, S)
        out = torch.empty(cfg.B, cfg.Hq, D, dtype=out_dtype, device="cuda")
        ok.decode_attn(self.lay, pool, self.q.cuda(), torch.from_numpy(self.table).cuda(),
                       torch.from_numpy(np.asarray(lens, np.int32)).cuda(), self.Rk_d, self.Rv_d,
                       cfg.sm_scale, S, ws, out)
        torch.cuda.synchronize()
        return out

    def compare(self, gpu_pool, ora_pool, upto):
        nd, nt = compare_pools(gpu_pool.cpu().numpy(), ora_pool, self.case(upto), meta=self.meta,
                               clip=self.clip, G=self.G)
        log("  pool: differing bytes", nd, "tolerated near-boundary elements", nt)


def _small_cfg(name, seed):
    return W.custom(name, 6, 8, 2, [1, 63, 64, 65, 129, 700], seed_index=seed,
                    k_outliers=(5, 90), v_outliers=(17,))


@pytest.mark.parametrize("variant", list(VARIANTS))
def test_variant_append_and_decode_small(variant):
    """Ragged lengths, one row per wave (the small-append kernel), 1/3/default splits."""
    vc = VCase(_small_cfg("var_" + variant, 230 + list(VARIANTS).index(variant)), variant)
    lens = vc.cfg.lens
    log("variant", variant, "lens", list(lens))
    pool = vc.gpu_append(lens)
    ora = vc.oracle_append(lens)
    vc.compare(pool, ora, lens)
    ref = vc.oracle_decode(ora, lens)
    for S in (1, 3, ok.default_num_splits(vc.lay, vc.cfg.B, vc.cfg.Hq, vc.table.shape[1] * P)):
        out = vc.gpu_decode(pool, lens, S)
        err = max_abs(out, ref)
        log("  splits %d max|err| = %.3g" % (S, err))
        assert err <= DECODE_TOL
    outb = vc.gpu_decode(pool, lens, 3, torch.bfloat16)
    assert torch.equal(outb.cpu(), vc.gpu_decode(pool, lens, 3).cpu().to(torch.bfloat16))


@pytest.mark.parametrize("variant", ["g64", "paper_format_g64", "paper_format", "bf16_meta",
                                     "token_quantile", "per_head_r"])
@pytest.mark.parametrize("g", [6, 12, 15])
def test_variant_gqa_wide(variant, g):
    """Query heads per KV head that are not a multiple of 4 (padding heads) and the
    wide score path (5-8, 9-12 and 13-16 heads per KV head) in every group size and
    metadata format, ragged lengths, 1 and 3 splits."""
    cfg = W.custom("var_g%d_%s" % (g, variant), 4, 2 * g, 2, [1, 65, 200, 777],
                   seed_index=260 + g + list(VARIANTS).index(variant), k_outliers=(5, 90),
                   v_outliers=(17,))
    vc = VCase(cfg, variant)
    lens = cfg.lens
    pool = vc.gpu_append(lens)
    ora = vc.oracle_append(lens)
    vc.compare(pool, ora, lens)
    ref = vc.oracle_decode(ora, lens)
    for S in (1, 3):
        err = max_abs(vc.gpu_decode(pool, lens, S), ref)
        log("variant", variant, "g", g, "splits %d max|err| = %.3g" % (S, err))
        assert err <= DECODE_TOL


@pytest.mark.parametrize("variant", ["bf16_meta", "g64", "g128", "identity_v", "per_head_r"])
def test_bf16_output_is_rne_of_fp32_every_instance(variant):
    """For every split-kernel instance (1 to 16 query heads per KV head: one chunk,
    the two-row and the one-row-per-head score tiles; each group size and metadata
    format) and both reduce instances (8 and 16 rows per block), with 1 and 3
    splits, the bf16 output is the round-to-nearest-even of the fp32 output of the
    same call: the two differ only in the final store."""
    for g in (1, 4, 6, 8, 12, 16):
        cfg = W.custom("rne_g%d_%s" % (g, variant), 3, 2 * g, 2, [5, 130, 300],
                       seed_index=300 + g + list(VARIANTS).index(variant))
        vc = VCase(cfg, variant)
        pool = vc.gpu_append(cfg.lens)
        for S in (1, 3):
            o32 = vc.gpu_decode(pool, cfg.lens, S)
            o16 = vc.gpu_decode(pool, cfg.lens, S, out_dtype=torch.bfloat16)
            log("rne", variant, "g", g, "splits", S)
            assert torch.equal(o16.cpu(), o32.cpu().to(torch.bfloat16)), (g, S)
    # 4096 rows: the reduce's 16-row blocks
    cfg = W.custom("rne_rows_%s" % variant, 128, 32, 8, np.full(128, 100), seed_index=330)
    vc = VCase(cfg, variant)
    pool = vc.gpu_append(cfg.lens)
    o32 = vc.gpu_decode(pool, cfg.lens, 2)
    o16 = vc.gpu_decode(pool, cfg.lens, 2, out_dtype=torch.bfloat16)
    assert torch.equal(o16.cpu(), o32.cpu().to(torch.bfloat16))


@pytest.mark.parametrize("variant", ["token_quantile", "g64", "paper_format",
                                     "identity_kv_paper_format", "per_head_r",
                                     "per_head_paper_format"])
def test_variant_bulk_append_qwen3_4b_shape(variant):
    """8192 tokens x 8 KV heads: the bulk cache update (two rows per wave, the
    quantile searched per wave half)."""
    cfg = W.config(1)
    vc = VCase(cfg, variant)
    lens = cfg.lens
    pool = vc.gpu_append(lens)
    ora = vc.oracle_append(lens)
    vc.compare(pool, ora, lens)
    err = max_abs(vc.gpu_decode(pool, lens, 8), vc.oracle_decode(ora, lens))
    log("  %s max|err| = %.3g" % (variant, err))
    assert err <= DECODE_TOL


@pytest.mark.parametrize("variant", ["paper_format", "g64", "identity_v", "per_head_r",
                                     "per_head_k_identity_v"])
def test_variant_decode_step(variant):
    """oscar_decode_step (cache update of the newest token + decode) in the variant
    format equals the oracle's append of every token + decode."""
    vc = VCase(_small_cfg("var_step_" + variant, 240), variant)
    cfg = vc.cfg
    lens = cfg.lens
    pool = vc.gpu_append(lens - 1)
    kn = torch.stack([vc.kv[b][0][int(lens[b]) - 1] for b in range(cfg.B)]).cuda()
    vn = torch.stack([vc.kv[b][1][int(lens[b]) - 1] for b in range(cfg.B)]).cuda()
    sl = np.array([vc.slots(b, int(lens[b]))[-1] for b in range(cfg.B)], np.int64)
    S = 3
    ws = ok.alloc_workspace(vc.lay, cfg.B, cfg.Hq, S)
    out = torch.empty(cfg.B, cfg.Hq, D, dtype=torch.float32, device="cuda")
    ok.decode_step(vc.lay, pool, kn, vn, torch.from_numpy(sl).cuda(), cfg.clip_k, cfg.clip_v,
                   vc.q.cuda(), torch.from_numpy(vc.table).cuda(), torch.from_numpy(lens).cuda(),
                   vc.Rk_d, vc.Rv_d, cfg.sm_scale, S, ws, out)
    torch.cuda.synchronize()
    ora = vc.oracle_append(lens)
    vc.compare(pool, ora, lens)
    err = max_abs(out, vc.oracle_decode(ora, lens))
    log("  step max|err| = %.3g" % err)
    assert err <= DECODE_TOL


@pytest.mark.parametrize("variant", ["paper_format", "paper_format_g64", "g64", "per_head_paper_format"])
def test_variant_mixed_cache_paper_format(variant):
    """The mixed-precision cache in the paper's format: bf16 sink 64 and window 256
    around an INT2 history with 128-channel groups, bf16 metadata and the
    per-token quantile clip (and with one rotation per KV head);
    prompt by oscar_mixed_append, newest token by oscar_decode_step_mixed (with
    demotion), against the oracle's one-token-per-step loop."""
    S0, W_ = 64, 256
    vc = VCase(W.custom("var_mixed", 4, 8, 2, [30, 320, 321, 900], seed_index=245,
                        k_outliers=(5, 90), v_outliers=(17,)), variant)
    cfg = vc.cfg
    lens = cfg.lens
    pool = ok.alloc_pool(vc.lay)
    seg = ok.alloc_seg(vc.lay, cfg.B, S0, W_)
    table_d = torch.from_numpy(vc.table).cuda()
    pre = torch.from_numpy(lens - 1).cuda()
    for b in range(cfg.B):
        n = int(lens[b]) - 1
        ok.mixed_append(vc.lay, pool, seg, S0, W_, vc.kv[b][0][:n].cuda(), vc.kv[b][1][:n].cuda(),
                        torch.full((n,), b, dtype=torch.int32, device="cuda"),
                        torch.arange(n, dtype=torch.int64, device="cuda"), table_d, pre, vc.Rk_d,
                        vc.Rv_d, cfg.clip_k, cfg.clip_v)
    kn = torch.stack([vc.kv[b][0][int(lens[b]) - 1] for b in range(cfg.B)]).cuda()
    vn = torch.stack([vc.kv[b][1][int(lens[b]) - 1] for b in range(cfg.B)]).cuda()
    S = 3
    ws = ok.alloc_mixed_workspace(vc.lay, cfg.B, cfg.Hq, S)
    out = torch.empty(cfg.B, cfg.Hq, D, dtype=torch.float32, device="cuda")
    ok.decode_step_mixed(vc.lay, pool, seg, S0, W_, kn, vn, cfg.clip_k, cfg.clip_v, vc.q.cuda(),
                         table_d, torch.from_numpy(lens).cuda(), vc.Rk_d, vc.Rv_d, cfg.sm_scale, S,
                         ws, out)
    torch.cuda.synchronize()
    ora = np.zeros(ok.pool_bytes(vc.lay), np.uint8)
    oseg = np.zeros(oracle.seg_elems(d=D, Hkv=cfg.Hkv, B=cfg.B, S0=S0, W=W_), np.uint16)
    chunk = cfg.Hkv * 2 * (S0 + W_) * D
    for b in range(cfg.B):
        kb, vb = bits(vc.kv[b][0]), bits(vc.kv[b][1])
        for n in range(1, int(lens[b]) + 1):
            oracle.mixed_update(ora, oseg[b * chunk:(b + 1) * chunk], d=D, Hkv=cfg.Hkv, P=P, G=vc.G,
                                S0=S0, W=W_, k_new=kb[n - 1:n], v_new=vb[n - 1:n],
                                block_table=vc.table[b:b + 1], seq_lens=np.array([n], np.int32),
                                Rk=vc.Rk, Rv=vc.Rv, clip_k=cfg.clip_k, clip_v=cfg.clip_v,
                                meta=vc.meta, clip=vc.clip)
    hist = [(min(S0, int(n)), max(min(S0, int(n)), int(n) - W_)) for n in lens]
    ks = torch.cat([vc.kv[b][0][lo:hi] for b, (lo, hi) in enumerate(hist)])
    vs = torch.cat([vc.kv[b][1][lo:hi] for b, (lo, hi) in enumerate(hist)])
    sl = np.concatenate([W.slots_for(vc.table, b, np.arange(lo, hi)) for b, (lo, hi) in enumerate(hist)])
    nd, nt = compare_pools(pool.cpu().numpy(), ora,
                           Case(cfg, vc.Rk, vc.Rv, vc.table, vc.num_pages, vc.q, ks, vs, sl),
                           meta=vc.meta, clip=vc.clip, G=vc.G)
    log("  pool: differing bytes", nd, "tolerated", nt)
    gseg = seg.cpu().contiguous().view(torch.int16).numpy().view(np.uint16).reshape(-1)
    assert np.array_equal(gseg, oseg)
    ref = oracle.decode_mixed(ora, oseg, d=D, Hkv=cfg.Hkv, P=P, G=vc.G, S0=S0, W=W_, q=bits(vc.q),
                              block_table=vc.table, seq_lens=lens, Rk=vc.Rk, Rv=vc.Rv,
                              sm_scale=cfg.sm_scale, meta=vc.meta)
    err = max_abs(out, ref)
    log("  mixed paper format max|err| = %.3g" % err)
    assert err <= DECODE_TOL


def test_variant_full_size_bench_workload_paper_format():
    """The bench workload (64 sequences of 16k-32k tokens, 32/8 heads) in the paper's
    format, as bench.py runs it (cache of tokens 0..n-2, one oscar_decode_step),
    sampled sequences against the oracle."""
    cfg = W.config(2, batch=64)
    meta, clip, G = 1, 1, 128
    B, Hq, Hkv = cfg.B, cfg.Hq, cfg.Hkv
    lens = cfg.lens.astype(np.int64)
    table, num_pages = W.block_table(cfg)
    lay = ok.Layout(num_kv_heads=Hkv, num_pages=num_pages, group_size=G, clip_mode=clip,
                    meta_dtype=meta)
    Rk_np, Rv_np = W.rotations(cfg)
    Rk, Rv = torch.from_numpy(Rk_np).cuda(), torch.from_numpy(Rv_np).cuda()
    sample = sorted({0, int(np.argmax(lens)), int(np.argmin(lens))})
    host_kv = {b: W.cache_kv(cfg, b) for b in sample}
    pool = ok.alloc_pool(lay)
    kn = torch.empty(B, Hkv, D, dtype=torch.bfloat16, device="cuda")
    vn = torch.empty_like(kn)
    new_slots = np.zeros(B, np.int64)
    for b in range(B):
        if b in host_kv:
            k, v = host_kv[b][0].cuda(), host_kv[b][1].cuda()
        else:
            k, v = W.cache_kv(cfg, b, device="cuda")
        n = int(lens[b])
        sl = W.slots_for(table, b, np.arange(n))
        ok.kv_append(lay, pool, k[:n - 1], v[:n - 1], torch.from_numpy(sl[:n - 1]).cuda(), Rk, Rv,
                     cfg.clip_k, cfg.clip_v)
        kn[b], vn[b], new_slots[b] = k[n - 1], v[n - 1], sl[n - 1]
        del k, v
    S = ok.default_num_splits(lay, B, Hq, int(table.shape[1]) * P)
    ws = ok.alloc_workspace(lay, B, Hq, S)
    q = W.queries(cfg)
    out = torch.empty(B, Hq, D, dtype=torch.float32, device="cuda")
    ok.decode_step(lay, pool, kn, vn, torch.from_numpy(new_slots).cuda(), cfg.clip_k, cfg.clip_v,
                   q.cuda(), torch.from_numpy(table).cuda(), torch.from_numpy(cfg.lens).cuda(), Rk,
                   Rv, cfg.sm_scale, S, ws, out)
    torch.cuda.synchronize()
    ora = np.zeros(ok.pool_bytes(lay), np.uint8)
    ks, vs, ss = [], [], []
    for b in sample:
        k, v = host_kv[b]
        sl = W.slots_for(table, b, np.arange(int(lens[b])))
        oracle.kv_append(ora, d=D, Hkv=Hkv, P=P, G=G, k=bits(k), v=bits(v), slot_mapping=sl,
                         Rk=Rk_np, Rv=Rv_np, clip_k=cfg.clip_k, clip_v=cfg.clip_v, meta=meta,
                         clip=clip)
        ks.append(k)
        vs.append(v)
        ss.append(sl)
    pairs = np.array([(b, h) for b in sample for h in range(Hq)], np.int32)
    ref = oracle.decode(ora, d=D, Hkv=Hkv, P=P, G=G, q=bits(q), block_table=table,
                        seq_lens=cfg.lens, Rk=Rk_np, Rv=Rv_np, sm_scale=cfg.sm_scale, pairs=pairs,
                        meta=meta)
    got = out[torch.as_tensor(np.asarray(sample))].reshape(-1, D)
    err = max_abs(got, ref)
    log("  paper format full size: max|err| over %d rows = %.3g" % (len(pairs), err))
    assert err <= DECODE_TOL
    bph = ok.page_bytes(lay)
    gpu_sel = np.zeros_like(ora)
    pool_pages = pool.view(num_pages, bph)
    for b in sample:
        ids = table[b, :(int(lens[b]) + 63) // 64]
        gpu_sel.reshape(num_pages, bph)[ids] = pool_pages[torch.from_numpy(ids).cuda()].cpu().numpy()
    nd, nt = compare_pools(gpu_sel, ora, Case(cfg, Rk_np, Rv_np, table, num_pages, q,
                                              torch.cat(ks), torch.cat(vs), np.concatenate(ss)),
                           meta=meta, clip=clip, G=G)
    log("  pool: differing bytes", nd, "tolerated", nt)
