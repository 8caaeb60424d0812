"""tkv_verify_noalloc -- attention on the library's static workspace -- against tkv_verify on a
caller-uploaded one.

Two calls in a row, the second with a smaller batch, each compared bitwise with tkv_verify on the
same inputs and with the oracle (max |o - o_ref| <= 1e-2, mean <= 1e-3, lse within 2e-3).  The
first batch has 128-row tile items with partials and merges as well as wave-grid items; the
second is a smaller decode-and-verify tree.  A plan larger than the static array is refused.
"""
import numpy as np
import pytest
import torch

import workloads as W
from _harness import oracle_check, realize_native

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS, LSE_ABS = 1e-2, 1e-3, 2e-3


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _both(wl, options=None):
    import paper_2609_39334_amd as tkv
    b = realize_native(wl)[0]
    s = wl.shape
    k, v = wl.kv_values()
    k, v = k.copy(), v.copy()
    W.poison_padding(k, v, b.block_len)
    q = wl.q_values(0, b.n_qtok)
    qi, ki, kb = b.arrays()
    shape = (s.hq, s.hkv, s.d, s.block_size, wl.num_blocks)
    ref = tkv.Plan(shape, qi, ki, kb, b.block_len, b.mult, options=options)              # uploaded workspace
    mine = tkv.Plan(shape, qi, ki, kb, b.block_len, b.mult, options=options, upload=False)  # never uploaded
    need = tkv.tkv_plan_workspace_bytes(mine.h)
    st = mine.stats
    print(f"  {wl.name}: rows {len(b.q_lens)} qtok {b.n_qtok} workspace {need} B items {st['n_items']} "
          f"(wave {st['n_items_wave']}) merges {st['n_merge']}", flush=True)
    assert 0 < need <= tkv.TKV_NOALLOC_MAX_BYTES
    qd, kd, vd = _dev(q), _dev(k), _dev(v)
    outs = []
    for fn, plan in ((tkv.tkv_verify, ref), (tkv.tkv_verify_noalloc, mine)):
        o = torch.full((b.n_qtok, s.hq, s.d), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((b.n_qtok, s.hq), float("nan"), dtype=torch.float32, device="cuda")
        fn(plan.h, qd, kd, vd, o, lse)
        torch.cuda.synchronize()
        outs.append((o, lse))
    (o1, l1), (o2, l2) = outs
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l2.view(torch.int32))
    r = oracle_check(q, W.bf16_bits_to_f32(k), W.bf16_bits_to_f32(v), b.tables, b.block_len, b.q_lens,
                     o2.float().cpu().numpy(), l2.cpu().numpy())
    print(f"    max {r['max']:.2e} mean {r['mean']:.2e} lse {r['lse_max']:.2e} over {r['tokens']} tokens", flush=True)
    assert r["finite"] and r["max"] <= MAX_ABS and r["mean"] <= MEAN_ABS and r["lse_max"] <= LSE_ABS
    return st, need


def test_noalloc_matches_uploaded_workspace_two_calls():
    import paper_2609_39334_amd as tkv
    # first call: shared chunks on 128-row tiles (partials + merge) and on the wave grid
    big = W.random_tree(60, W.Shape(12, 2, 128), n_roots=3, depth=3, max_branch=4, max_step=70)
    st1, need1 = _both(big, options={"wave_max_rows": 8, "tile_min_items": 0})
    assert st1["n_items"] > st1["n_items_wave"] > 0 and st1["n_merge"] > 0
    # second call, smaller: the array keeps the first call's contents, which must not leak in
    small = W.random_tree(61, W.Shape(8, 2, 64), n_roots=2, depth=2, max_branch=3, max_step=40)
    st2, need2 = _both(small)
    assert need2 < need1 and st2["n_qtok"] < st1["n_qtok"]
    assert tkv.TKV_NOALLOC_MAX_BYTES == 64 << 20


def test_noalloc_refuses_a_plan_larger_than_its_array():
    import paper_2609_39334_amd as tkv
    wl = W.mixed_serving(0)
    b = realize_native(wl)[1]
    s = wl.shape
    qi, ki, kb = b.arrays()
    # (chunks of up to 96 rows on the wave kernel: more partial slots, a workspace of about 71 MB)
    plan = tkv.Plan((s.hq, s.hkv, s.d, s.block_size, wl.num_blocks), qi, ki, kb, b.block_len, b.mult, upload=False,
                    options={"wave_max_rows": 96})
    assert tkv.tkv_plan_workspace_bytes(plan.h) > tkv.TKV_NOALLOC_MAX_BYTES
    t = torch.zeros((4, s.hq, s.d), dtype=torch.bfloat16, device="cuda")
    o = torch.full((4, s.hq, s.d), 3.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(tkv.TkvError) as e:
        tkv.tkv_verify_noalloc(plan.h, t, t, t, o)
    assert e.value.code == tkv.TKV_EINVAL and "static" in str(e.value)
    torch.cuda.synchronize()
    assert (o.float() == 3.0).all()      # nothing was enqueued
