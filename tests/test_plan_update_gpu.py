"""GPU: a plan carried through decode steps by tkv_plan_update gives, bit for bit, what a plan made
from scratch gives, and matches the oracle; after each in-place update the upload sends only the
changed descriptor words, and the device copy of the descriptors equals the host image.

Each step grows every decode candidate by one token (new blocks included, some candidates opening
new chunks); the updated plan and a fresh one run the same attention call on the same pool.  The
pool holds finite values everywhere (so a key read past its block's length would change the
result and show against the oracle)."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from _harness import oracle_check
from test_plan_update import BS, DecodeTree

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS, LSE_ABS = 1e-2, 1e-3, 2e-3


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


@pytest.mark.parametrize("shape,verify", [(W.Shape(12, 2, 128), True), (W.Shape(8, 2, 64), False),
                                          (W.Shape(32, 8, 128), True)])
def test_updated_plan_matches_fresh_plan_bitwise(shape, verify):
    import paper_2609_39334_amd as tkv
    tails = [1, 15, 16, 17, 250, 251, 255, 256, 240, 31, 32, 33, 100, 180]
    tree = DecodeTree(21, shape, tails, verify=verify, num_blocks=2048)
    rng = np.random.default_rng(3)
    pool = (tree.num_blocks, shape.hkv, BS, shape.d)
    kbits = W.f32_to_bf16_bits(rng.standard_normal(pool).astype(np.float32))
    vbits = W.f32_to_bf16_bits(rng.standard_normal(pool).astype(np.float32))
    kd, vd = _dev(kbits), _dev(vbits)
    kf, vf = W.bf16_bits_to_f32(kbits), W.bf16_bits_to_f32(vbits)
    n_qtok = int(sum(tree.q_lens))
    plan = None
    n_in_place = n_patched = 0
    for step in range(12):
        tree.step()
        t, ki, kb, bl = tree.tables()
        if plan is None:
            plan = tkv.Plan(tree.dims(), tree.q_indptr(), ki, kb, bl)
        else:
            # update, then upload: in place, only the changed descriptor words go to the device
            in_place = tkv.tkv_plan_update(plan.h, ki, kb, bl)
            n_in_place += in_place
            _, complete = tkv.tkv_plan_dirty(plan.h)
            n_patched += in_place and complete
            nbytes = tkv.tkv_plan_workspace_bytes(plan.h)
            if nbytes > plan.workspace.numel():
                plan.workspace = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
            tkv.tkv_plan_upload(plan.h, plan.workspace)
            img, _ = plan.image()
            torch.cuda.synchronize()
            assert plan.workspace[:len(img)].cpu().numpy().tobytes() == img
        fresh = tkv.Plan(tree.dims(), tree.q_indptr(), ki, kb, bl)
        qbits = W.f32_to_bf16_bits(rng.standard_normal((n_qtok, shape.hq, shape.d)).astype(np.float32))
        qd = _dev(qbits)
        outs = []
        for p in (plan, fresh):
            o = torch.full((n_qtok, shape.hq, shape.d), float("nan"), dtype=torch.bfloat16, device="cuda")
            lse = torch.full((n_qtok, shape.hq), float("nan"), dtype=torch.float32, device="cuda")
            (p.verify if verify else p.decode)(qd, kd, vd, o, lse)
            outs.append((o, lse))
        torch.cuda.synchronize()
        same = torch.equal(outs[0][0].view(torch.int16), outs[1][0].view(torch.int16)) and \
            torch.equal(outs[0][1].view(torch.int32), outs[1][1].view(torch.int32))
        r = oracle_check(qbits, kf, vf, [list(x) for x in t], bl, tree.q_lens,
                         outs[0][0].float().cpu().numpy(), outs[0][1].cpu().numpy())
        _log(f"  step {step}: items {plan.stats['n_items']} idle waves {plan.stats['n_idle_waves']} "
             f"bitwise {same}; max {r['max']:.2e} mean {r['mean']:.2e} lse {r['lse_max']:.2e}")
        assert same
        assert r["finite"] and r["max"] <= MAX_ABS and r["mean"] <= MEAN_ABS and r["lse_max"] <= LSE_ABS
        del fresh
    assert n_in_place >= 8 and n_patched >= 8


def test_plan_destroyed_right_after_upload():
    # the library waits for the copy before a destroyed plan's host image is recycled: the workspace
    # holds the first plan's descriptors even though the next plan reuses its image at once
    import paper_2609_39334_amd as tkv
    tree = DecodeTree(23, W.Shape(12, 2, 128), [3, 70, 255, 256, 31], num_blocks=2048)
    _, ki, kb, bl = tree.tables()
    dims, qi = tree.dims(), tree.q_indptr()
    h = tkv.tkv_plan_create(dims, qi, ki, kb, bl)
    img, _ = tkv.tkv_plan_image(h)
    ws = torch.empty(tkv.tkv_plan_workspace_bytes(h), dtype=torch.uint8, device="cuda")
    busy = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    for _ in range(8):             # queue work ahead of the copy
        busy.add_(1)
    tkv.tkv_plan_upload(h, ws)
    tkv.tkv_plan_destroy(h)
    tree.step()
    _, ki2, kb2, bl2 = tree.tables()
    h2 = tkv.tkv_plan_create(dims, qi, ki2, kb2, bl2)   # takes the recycled image and rewrites it
    img2, _ = tkv.tkv_plan_image(h2)
    torch.cuda.synchronize()
    assert img2 != img
    assert ws[:len(img)].cpu().numpy().tobytes() == img
    tkv.tkv_plan_destroy(h2)
