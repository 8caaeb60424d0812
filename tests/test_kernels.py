"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Tolerance (bf16 inputs, fp32 accumulation, bf16 output): max |o - o_ref| <= 1e-2 and
mean |o - o_ref| <= 1e-3; lse within 2e-3.  Block tables and coalescing are compared exactly.
Padding slots of partial blocks and every free block hold bf16 NaN, so any read of padding shows.
Every workload, the full-size ones included, is compared on every row, in the launch configuration
the benchmark times, and run twice with bitwise-equal results (no atomics in any reduction).
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from _harness import oracle_check, realize_native, realize_oracle

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS, LSE_ABS = 1e-2, 1e-3, 2e-3


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _f64(bits):
    return W.bf16_bits_to_f32(bits).astype(np.float64)


def run_gpu(wl, launch, poison=True, kv=None, repeat=1, options=None):
    """Realise the workload on the C block manager and run one launch on the GPU `repeat` times.
    Returns (batch, o float32 [n_qtok, hq, d], lse [n_qtok, hq], k bits, v bits, q bits, plan stats,
    whether every repeat gave bitwise the first call's o and lse)."""
    import paper_2609_39334_amd as tkv
    b = realize_native(wl)[launch]
    s = wl.shape
    k, v = kv if kv is not None else wl.kv_values()
    if poison:
        k, v = k.copy(), v.copy()
        W.poison_padding(k, v, b.block_len)
    q = wl.q_values(launch, b.n_qtok)
    qi, ki, kb = b.arrays()
    _log(f"  gpu: {wl.name} launch {launch}: rows {len(b.q_lens)} qtok {b.n_qtok} (hq {s.hq} hkv {s.hkv} d {s.d})"
         f" options {options}")
    plan = tkv.Plan((s.hq, s.hkv, s.d, s.block_size, wl.num_blocks), qi, ki, kb, b.block_len, b.mult,
                    options=options)
    qd, kd, vd = _dev(q), _dev(k), _dev(v)
    first, same = None, True
    for _ in range(repeat):
        o = torch.full((b.n_qtok, s.hq, s.d), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((b.n_qtok, s.hq), float("nan"), dtype=torch.float32, device="cuda")
        if b.decode:
            plan.decode(qd, kd, vd, o, lse)
        else:
            plan.verify(qd, kd, vd, o, lse)
        torch.cuda.synchronize()
        if first is None:
            first = (o, lse)
        else:
            same = same and torch.equal(o.view(torch.int16), first[0].view(torch.int16)) and \
                torch.equal(lse.view(torch.int32), first[1].view(torch.int32))
    st = plan.stats
    del plan, qd, kd, vd
    o_np, l_np = first[0].float().cpu().numpy(), first[1].cpu().numpy()
    return b, o_np, l_np, k, v, q, st, same


def compare(wl, launch, rows=None, poison=True, repeat=2, kv=None, options=None):
    """Run one launch on the GPU and compare it with the oracle on `rows` (all rows by default)."""
    b, o, l, k, v, q, st, same = run_gpu(wl, launch, poison=poison, kv=kv, repeat=repeat, options=options)
    ob = realize_oracle(wl)[launch]
    assert ob.tables == b.tables and ob.q_lens == b.q_lens and ob.mult == b.mult
    assert np.array_equal(ob.block_len, b.block_len)
    r = oracle_check(q, W.bf16_bits_to_f32(k), W.bf16_bits_to_f32(v), ob.tables, ob.block_len, ob.q_lens, o, l,
                     rows=rows)
    _log(f"    max {r['max']:.2e} mean {r['mean']:.2e} lse max {r['lse_max']:.2e} over {r['tokens']} tokens"
         f" (of {b.n_qtok}); repeats identical: {same}")
    assert r["finite"]
    assert r["max"] <= MAX_ABS and r["mean"] <= MEAN_ABS
    assert r["lse_max"] <= LSE_ABS
    assert same                  # run-to-run determinism
    return b, st


def test_tiny_decode_full():
    compare(W.tiny_decode(0), 0)


@pytest.mark.parametrize("seed,hq,hkv,d", [(0, 8, 2, 64), (1, 12, 2, 128), (2, 28, 4, 128), (3, 32, 8, 128),
                                           (4, 4, 4, 64), (5, 14, 2, 64), (6, 64, 1, 128), (7, 16, 1, 64),
                                           (8, 15, 5, 128), (9, 10, 2, 64), (14, 40, 8, 128)])
def test_random_trees_full(seed, hq, hkv, d):
    wl = W.random_tree(seed, W.Shape(hq, hkv, d), n_roots=3, depth=3, max_branch=3, max_step=70)
    compare(wl, 0)


def test_verify_long_steps_and_single_token_rows():
    # long verify steps (row items), q_len == kv_len rows (a root verified whole), kv_len 1 rows
    wl = W.Workload("edge", W.Shape(12, 2, 128), 11)
    rt = np.random.default_rng(5)
    root = wl.extend(-1, rt.integers(0, 100, 300), True)
    a = wl.extend(root, rt.integers(0, 100, 256), True)
    b = wl.extend(root, rt.integers(0, 100, 17), True)
    one = wl.extend(-1, [7], True)
    lone = wl.extend(-1, rt.integers(0, 100, 40), True)
    c = wl.extend(one, [], True)            # fork with no new tokens
    wl.launch("mixed", [(a, 256), (b, 17), (one, 1), (lone, 40), (c, 1), (root, 300)])
    wl.finalize()
    compare(wl, 0)


@pytest.mark.parametrize("options", [None, {"wave_max_rows": 8, "tile_min_items": 0}])
def test_long_context(options):
    # a 40,000-token shared context (2,500 blocks: 157 wave chunks, or 40 wide chunks on the tiles, so
    # every decode token merges that many partials), under it decode candidates with private steps and
    # verify candidates whose steps of 54-76 tokens walk the whole context as row items
    wl = W.Workload("long", W.Shape(16, 2, 128), 13)
    rt = np.random.default_rng(9)
    root = wl.extend(-1, rt.integers(0, 1000, 40000), True)
    cands = []
    for i in range(6):
        h = wl.extend(root, rt.integers(0, 1000, int(rt.integers(1, 200))), i % 2 == 1)
        cands.append((h, int(rt.integers(100, 301)) if i % 2 == 1 else 1))
    # the verify candidates' q_len is their own step's length
    cands = [(h, q if q == 1 else len(wl.events[h].tokens)) for h, q in cands]
    wl.launch("long", cands)
    wl.finalize()
    b, st = compare(wl, 0, options=options)
    assert st["n_merge"] > 0 and st["n_items_row"] > 0


@pytest.mark.parametrize("name", ["beam_decode", "step_verify", "spec_prompts"])
def test_full_size_every_row(name):
    compare(W.CONFIGS[name](0), 0)


@pytest.mark.timeout(600)
def test_spec_explosion_every_row():
    b, st = compare(W.spec_explosion(0), 0)
    assert st["n_rows"] < 2048          # identical leaves coalesced
    assert st["n_items"] - st["n_items_wave"] > 0   # the interleaved tile/wave dispatch ran


@pytest.fixture(scope="module")
def mixed_kv():
    return W.mixed_serving(0).kv_values()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("launch", [0, 1])
def test_mixed_serving_every_row(launch, mixed_kv):
    # launch 0: every candidate; launch 1 (the benchmark's): after 30% of them were pruned and refilled
    b, st = compare(W.mixed_serving(0), launch, kv=mixed_kv)
    assert st["n_items_row"] > 0 and st["n_items_wave"] > 0


@pytest.mark.parametrize("seed,hq,hkv,d", [(10, 8, 2, 64), (11, 12, 2, 128), (12, 16, 1, 128), (13, 6, 6, 64)])
def test_shared_chunks_on_tile_kernel(seed, hq, hkv, d):
    # every shared chunk read by more than 8 query rows goes to the 128-row tile kernel (partials,
    # merges and per-token causal limits included), the narrow rest to the wave kernel
    wl = W.random_tree(seed, W.Shape(hq, hkv, d), n_roots=3, depth=3, max_branch=4, max_step=60)
    b, st = compare(wl, 0, options={"wave_max_rows": 8, "tile_min_items": 0})
    assert st["n_items_shared"] - st["n_items_wave"] > 0     # shared chunks did run on the tile kernel


@pytest.mark.parametrize("seed,hq,hkv,d", [(40, 4, 2, 64), (42, 12, 2, 128)])
def test_folded_segments_on_tile_kernel(seed, hq, hkv, d):
    # every shared chunk on the 128-row tiles and every short segment folded into its children's key
    # runs (a child's tiles read the parent's blocks, then its own)
    wl = W.random_tree(seed, W.Shape(hq, hkv, d), n_roots=2, depth=4, max_branch=3, max_step=40, p_verify=0.3)
    b, st = compare(wl, 0, options={"wave_max_rows": 2, "tile_min_items": 0, "fold_blocks": 1000})
    b0, st0 = compare(wl, 0, options={"wave_max_rows": 2, "tile_min_items": 0, "fold_blocks": 0})
    assert st["n_slots"] < st0["n_slots"]


@pytest.mark.parametrize("seed,hq,hkv,d", [(17, 12, 2, 128), (20, 8, 1, 64)])
def test_wide_chunks_on_wave_kernel(seed, hq, hkv, d):
    # chunks read by more than 32 query rows stay on the wave kernel, split into many 32-row tiles
    # over the same blocks (by default they go to 128-row tile items)
    wl = W.random_tree(seed, W.Shape(hq, hkv, d), n_roots=2, depth=3, max_branch=5, max_step=40)
    b, st = compare(wl, 0, options={"tile_min_items": 1000000})
    assert st["n_items_shared"] == st["n_items_wave"]        # no shared chunk on the tile kernel


@pytest.mark.parametrize("waves", [8, 64])
def test_small_wave_grids(waves):
    # a wave grid much smaller than the item count: long per-wave lists, items crossing into the
    # next item's first blocks many times per wave
    # (chunks of up to 96 rows on the wave kernel, so that there are many wave items)
    wl = W.random_tree(20, W.Shape(12, 2, 128), n_roots=4, depth=3, max_branch=3, max_step=70)
    b, st = compare(wl, 0, options={"waves": waves, "wave_max_rows": 96})
    assert 0 < st["n_waves"] < st["n_items_wave"]            # waves walk lists of several items


@pytest.mark.parametrize("options", [None, {"wave_max_rows": 8, "tile_min_items": 0}])
def test_blocks_past_4gib_of_pool(options):
    # block ids whose K/V start more than 4 GiB into each pool (64-bit offsets in every path): a
    # random tree's blocks moved to the top of pools of 4.6 GiB each, the blocks below NaN
    import paper_2609_39334_amd as tkv
    wl = W.random_tree(70, W.Shape(12, 2, 128), n_roots=2, depth=3, max_branch=3, max_step=60)
    b = realize_native(wl)[0]
    ob = realize_oracle(wl)[0]
    s = wl.shape
    k, v = wl.kv_values()
    blk_bytes = s.hkv * s.block_size * s.d * 2
    base = (4 << 30) // blk_bytes + 4096                        # first moved block: past 4 GiB
    nb_big = base + wl.num_blocks
    assert nb_big * blk_bytes > (4 << 30) + wl.num_blocks * blk_bytes
    kd = torch.full((nb_big, s.hkv, s.block_size, s.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    vd = torch.full_like(kd, float("nan"))
    kd[base:] = _dev(k)
    vd[base:] = _dev(v)
    bl = np.zeros(nb_big, dtype=np.int32)
    bl[base:] = b.block_len
    qi, ki, kb = b.arrays()
    q = wl.q_values(0, b.n_qtok)
    plan = tkv.Plan((s.hq, s.hkv, s.d, s.block_size, nb_big), qi, ki, np.asarray(kb, dtype=np.int32) + base, bl,
                    b.mult, options=options)
    o = torch.full((b.n_qtok, s.hq, s.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((b.n_qtok, s.hq), float("nan"), dtype=torch.float32, device="cuda")
    (plan.decode if b.decode else plan.verify)(_dev(q), kd, vd, o, lse)
    torch.cuda.synchronize()
    st = plan.stats
    del plan, kd, vd
    r = oracle_check(q, W.bf16_bits_to_f32(k), W.bf16_bits_to_f32(v), ob.tables, ob.block_len, ob.q_lens,
                     o.float().cpu().numpy(), lse.cpu().numpy())
    _log(f"    pool of {nb_big} blocks; max {r['max']:.2e} mean {r['mean']:.2e} lse {r['lse_max']:.2e}; items {st['n_items']}")
    assert r["finite"] and r["max"] <= MAX_ABS and r["mean"] <= MEAN_ABS and r["lse_max"] <= LSE_ABS
    if options:
        assert st["n_items_shared"] - st["n_items_wave"] > 0    # shared chunks on the tile kernel too


def test_empty_plan_on_gpu():
    import paper_2609_39334_amd as tkv
    plan = tkv.Plan((8, 2, 64, 16, 4), [0], [0], [], [16, 3, 0, 0])
    q = torch.zeros((1, 8, 64), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((4, 2, 16, 64), dtype=torch.bfloat16, device="cuda")
    o = torch.full((1, 8, 64), 7.0, dtype=torch.bfloat16, device="cuda")
    plan.decode(q, kv, kv, o, None)
    plan.verify(q, kv, kv, o, None)
    torch.cuda.synchronize()
    assert (o.float() == 7.0).all()          # no row, nothing written


@pytest.mark.parametrize("seed,hq,hkv,d,tile_rows", [(30, 12, 2, 128, None), (31, 8, 2, 64, None), (32, 12, 2, 128, 8)])
def test_consecutive_calls_new_queries(seed, hq, hkv, d, tile_rows):
    # a plan's partial slots are reused by every call on it: the second and third calls, with new
    # queries, must not see an earlier call's partials (tile_rows "8": shared chunks on the 128-row
    # tiles)
    import paper_2609_39334_amd as tkv
    options = {"wave_max_rows": tile_rows, "tile_min_items": 0} if tile_rows else None
    wl = W.random_tree(seed, W.Shape(hq, hkv, d), n_roots=3, depth=3, max_branch=4, max_step=60)
    b = realize_native(wl)[0]
    ob = realize_oracle(wl)[0]
    s = wl.shape
    k, v = wl.kv_values()
    qi, ki, kb = b.arrays()
    plan = tkv.Plan((s.hq, s.hkv, s.d, s.block_size, wl.num_blocks), qi, ki, kb, b.block_len, b.mult,
                    options=options)
    assert plan.stats["n_merge"] > 0
    kd, vd = _dev(k), _dev(v)
    for call in range(3):
        q = wl.q_values(10 + call, b.n_qtok)                 # new queries each call
        o = torch.full((b.n_qtok, s.hq, s.d), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((b.n_qtok, s.hq), float("nan"), dtype=torch.float32, device="cuda")
        (plan.decode if b.decode else plan.verify)(_dev(q), kd, vd, o, lse)
        torch.cuda.synchronize()
        o_ref, l_ref = oracle.attention(_f64(q), W.bf16_bits_to_f32(k), W.bf16_bits_to_f32(v), ob.tables,
                                        ob.block_len, ob.q_lens)
        err = np.abs(o.float().cpu().numpy() - o_ref)
        lerr = np.abs(lse.cpu().numpy() - l_ref)
        _log(f"    call {call}: max {err.max():.2e} mean {err.mean():.2e} lse max {lerr.max():.2e}")
        assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS and lerr.max() <= LSE_ABS


def _small_verify(seed, shape, n_ctx=2, n_cands=5):
    """Verify-only batch: contexts U{40..600} (sealed), candidate steps long enough that every row's
    query tile reaches 64 rows (q_len * G >= 64), so the plan holds tile items only."""
    rs = np.random.default_rng([seed, 1])
    rt = np.random.default_rng([seed, 2])
    g = shape.hq // shape.hkv
    wl = W.Workload(f"small_verify_{seed}", shape, seed, note="verify-only batch")
    cands, ctxs = [], []
    for _ in range(n_ctx):
        c = wl.extend(-1, rt.integers(0, 32000, int(rs.integers(40, 601))), True)
        ctxs.append(c)
        for _ in range(n_cands):
            n = int(rs.integers(-(-64 // g), 201))
            cands.append((wl.extend(c, rt.integers(0, 32000, n), True), n))
    for c in ctxs:
        wl.prune(c)
    wl.launch("verify", cands)
    return wl.finalize()


@pytest.mark.parametrize("seed,hq,hkv,d", [(40, 28, 4, 128), (41, 8, 2, 64), (42, 16, 2, 128), (43, 4, 4, 64),
                                           (44, 64, 1, 128), (45, 6, 2, 64)])
@pytest.mark.parametrize("tile8_max", [0, 100000])
def test_small_verify_batches_on_both_tile_kernels(seed, hq, hkv, d, tile8_max):
    # a verify-only batch makes tile items alone; a few of them run as 8-wave workgroups (one 16-row
    # column tile per wave), more of them on the 4-wave kernel -- the option forces either
    wl = _small_verify(seed, W.Shape(hq, hkv, d))
    b, st = compare(wl, 0, options={"tile8_max_items": tile8_max})
    assert st["n_items_wave"] == 0 and st["n_items_row"] > 0 and st["n_items"] == st["n_items_row"]

