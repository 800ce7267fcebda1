"""OSCAR_DEBUG=1: the entry points copy their device-resident indices (slots, block
table, sequence lengths) to the host and reject out-of-range values before
launching anything.  Every invalid index used here still lies inside the
tensors' allocations (the pool carries one page beyond the layout's num_pages),
so no kernel could reach memory outside them even if a check let one through.
With valid indices the debug mode gives the same bytes and outputs as without."""
import pytest
import torch

import paper_2605_17757_amd as ok
from helpers import log

pytestmark = pytest.mark.gpu

D, P = 128, 64
HKV, HQ, B, NPG, MP = 2, 8, 2, 8, 4


def _case():
    lay = ok.Layout(num_kv_heads=HKV, num_pages=NPG)
    # the layout's pool as a view of an allocation with one slack page after it
    pool = ok.alloc_pool(ok.Layout(num_kv_heads=HKV, num_pages=NPG + 1))[:ok.pool_bytes(lay)]
    g = torch.Generator().manual_seed(11)
    R = torch.linalg.qr(torch.randn(D, D, generator=g, dtype=torch.float64))[0].float().contiguous().cuda()
    lens = torch.tensor([100, 200], dtype=torch.int32)
    table = torch.tensor([[0, 1, 2, 3], [4, 5, 6, 7]], dtype=torch.int32)
    slots = torch.cat([table[b, torch.arange(int(lens[b])) // P].long() * P + torch.arange(int(lens[b])) % P
                       for b in range(B)])
    n = int(slots.numel())
    k = torch.randn(n, HKV, D, generator=g).bfloat16().cuda()
    v = torch.randn(n, HKV, D, generator=g).bfloat16().cuda()
    q = torch.randn(B, HQ, D, generator=g).bfloat16().cuda()
    return lay, pool, R, lens.cuda(), table.cuda(), slots.cuda(), k, v, q


def _attn(lay, pool, q, table, lens, R):
    S = ok.default_num_splits(lay, B, HQ, MP * P)
    ws = ok.alloc_workspace(lay, B, HQ, S)
    out = torch.full((B, HQ, D), 7.0, dtype=torch.float32, device="cuda")
    ok.decode_attn(lay, pool, q, table, lens, R, R, D ** -0.5, S, ws, out)
    torch.cuda.synchronize()
    return out


def test_valid_indices_same_results(monkeypatch):
    lay, pool, R, lens, table, slots, k, v, q = _case()
    monkeypatch.setenv("OSCAR_DEBUG", "0")
    ok.kv_append(lay, pool, k, v, slots, R, R, 0.9, 0.9)
    ref_pool = pool.clone()
    ref = _attn(lay, pool, q, table, lens, R)
    monkeypatch.setenv("OSCAR_DEBUG", "1")
    pool.zero_()
    ok.kv_append(lay, pool, k, v, slots, R, R, 0.9, 0.9)
    torch.cuda.synchronize()
    assert torch.equal(pool, ref_pool)
    assert torch.equal(_attn(lay, pool, q, table, lens, R), ref)


def test_slot_past_the_pool_rejected_before_launch(monkeypatch):
    lay, pool, R, lens, table, slots, k, v, q = _case()
    monkeypatch.setenv("OSCAR_DEBUG", "1")
    bad = slots.clone()
    bad[5] = NPG * P  # first slot of the slack page
    before = pool.clone()
    with pytest.raises(ok.OscarError) as e:
        ok.kv_append(lay, pool, k, v, bad, R, R, 0.9, 0.9)
    assert e.value.status == ok.ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.equal(pool, before)  # nothing written
    log("slot past the pool:", e.value)


def test_page_id_past_the_pool_rejected_before_launch(monkeypatch):
    lay, pool, R, lens, table, slots, k, v, q = _case()
    ok.kv_append(lay, pool, k, v, slots, R, R, 0.9, 0.9)
    monkeypatch.setenv("OSCAR_DEBUG", "1")
    bad = table.clone()
    bad[1, 3] = NPG  # the slack page, in a page sequence 1 uses (200 tokens: pages 0..3)
    S = ok.default_num_splits(lay, B, HQ, MP * P)
    ws = ok.alloc_workspace(lay, B, HQ, S)
    out = torch.full((B, HQ, D), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(ok.OscarError) as e:
        ok.decode_attn(lay, pool, q, bad, lens, R, R, D ** -0.5, S, ws, out)
    assert e.value.status == ok.ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())  # nothing launched
    # an entry past a sequence's used pages is not read, so it is not checked
    unused = table.clone()
    unused[0, 3] = NPG  # sequence 0 has 100 tokens: pages 0..1
    out2 = _attn(lay, pool, q, unused, lens, R)
    monkeypatch.setenv("OSCAR_DEBUG", "0")
    assert torch.equal(out2, _attn(lay, pool, q, table, lens, R))


def test_length_past_the_block_table_rejected(monkeypatch):
    lay, pool, R, lens, table, slots, k, v, q = _case()
    ok.kv_append(lay, pool, k, v, slots, R, R, 0.9, 0.9)
    monkeypatch.setenv("OSCAR_DEBUG", "1")
    bad = lens.clone()
    bad[0] = MP * P + 1  # one token more than the table row holds (kernels clamp it)
    S = ok.default_num_splits(lay, B, HQ, MP * P)
    ws = ok.alloc_workspace(lay, B, HQ, S)
    out = torch.full((B, HQ, D), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(ok.OscarError) as e:
        ok.decode_attn(lay, pool, q, table, bad, R, R, D ** -0.5, S, ws, out)
    assert e.value.status == ok.ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())


def test_decode_step_checks_its_slots(monkeypatch):
    lay, pool, R, lens, table, slots, k, v, q = _case()
    ok.kv_append(lay, pool, k, v, slots, R, R, 0.9, 0.9)
    monkeypatch.setenv("OSCAR_DEBUG", "1")
    # one new token per sequence at position lens[b], one of them past the pool
    new_slots = torch.tensor([1 * P + 100 % P, NPG * P], dtype=torch.int64, device="cuda")
    kn = torch.zeros(B, HKV, D, dtype=torch.bfloat16, device="cuda")
    S = ok.default_num_splits(lay, B, HQ, MP * P)
    ws = ok.alloc_workspace(lay, B, HQ, S)
    out = torch.full((B, HQ, D), 7.0, dtype=torch.float32, device="cuda")
    before = pool.clone()
    with pytest.raises(ok.OscarError) as e:
        ok.decode_step(lay, pool, kn, kn, new_slots, 0.9, 0.9, q, table, lens + 1, R, R,
                       D ** -0.5, S, ws, out)
    assert e.value.status == ok.ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.equal(pool, before) and bool((out == 7.0).all())
