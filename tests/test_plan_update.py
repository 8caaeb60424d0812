"""tkv_plan_update on CPU: a plan brought forward through decode steps does the work of a plan made
from scratch on the same tables.

The block manager grows each live candidate by one token per step (a new block when its last one
is full); the plan takes the new tables with tkv_plan_update.  After every step the updated plan's
descriptor image is decoded and compared with a fresh plan's: the same tile items and wave items
(blocks, lengths, positions, tokens, causal limits), partial slots in the same path order, the same
merges.  Where only lengths changed the two images are equal byte for byte.  The float64
interpreter of the descriptor format runs the updated plan against the oracle."""
import numpy as np
import pytest

import oracle
import paper_2609_39334_amd as tkv
import workloads as W
from test_plan import execute_plan

BS = 16


def _f64(bits):
    return W.bf16_bits_to_f32(bits).astype(np.float64)


class DecodeTree:
    """Roots with two sealed steps each, open candidates under them, and optionally two verify rows
    whose tables stay fixed (one long enough for 128-row tiles, one short)."""

    def __init__(self, seed, shape, tails, verify=True, num_blocks=4096, n_roots=2):
        self.rng = np.random.default_rng(seed)
        self.shape = shape
        self.num_blocks = num_blocks
        self.bm = tkv.BlockManager(num_blocks, BS, 512)
        toks = lambda n: self.rng.integers(0, 30000, n).astype(np.int32)
        mids = []
        for r in range(n_roots):
            root, _, _ = self.bm.extend(-1, toks(90 + 41 * r), True)
            mids += [self.bm.extend(root, toks(30 + 11 * k + r), True)[0] for k in range(2)]
        self.decode = [self.bm.extend(mids[i % len(mids)], toks(n), False)[0] for i, n in enumerate(tails)]
        self.rows = list(self.decode)
        self.q_lens = [1] * len(self.decode)
        if verify:
            g = shape.hq // shape.hkv
            for m, ql in ((mids[0], -(-64 // g) + 5), (mids[-1], 2)):
                self.rows.append(self.bm.extend(m, toks(ql + 7), False)[0])
                self.q_lens.append(ql)

    def step(self, rows=None):
        """One decode step: one token more for each decode row (or the given ones)."""
        for s in (self.decode if rows is None else rows):
            self.bm.append(s, self.rng.integers(0, 30000, 1).astype(np.int32))

    def tables(self):
        t = [self.bm.table(s) for s in self.rows]
        ki = np.concatenate([[0], np.cumsum([len(x) for x in t])]).astype(np.int32)
        kb = np.concatenate(t).astype(np.int32)
        return t, ki, kb, self.bm.block_len()

    def dims(self):
        s = self.shape
        return (s.hq, s.hkv, s.d, BS, self.num_blocks)

    def q_indptr(self):
        return np.concatenate([[0], np.cumsum(self.q_lens)]).astype(np.int32)

    def plan(self):
        _, ki, kb, bl = self.tables()
        return tkv.Plan(self.dims(), self.q_indptr(), ki, kb, bl, upload=False)


def decode_image(plan):
    """The plan's device image as canonical work: tile items and wave items with their tokens,
    blocks and partial slots named (query token, index in its merge range); merges by token."""
    img, lay = plan.image()
    st = plan.stats
    w = np.frombuffer(img, dtype=np.int32)
    sec = lambda a, b: w[lay[a] // 4:lay[b] // 4]
    merges = sec("merges", "merge_slots").reshape(-1, 4)[:st["n_merge"]]
    mslots = sec("merge_slots", "wave_records")
    canon = {-1: -1}
    for qtok, off, n, _ in merges:
        for k in range(n):
            canon[int(mslots[off + k])] = (int(qtok), k)
    tok = lambda t: (int(t[0]), int(t[1]), canon[int(t[2])])
    n_tile = st["n_items"] - st["n_items_wave"]
    items = sec("items", "toks")[:n_tile * 8].reshape(-1, 8)
    toks = sec("toks", "blks").reshape(-1, 4)
    blks = sec("blks", "merges").reshape(-1, 2)
    tile = sorted((int(kind), int(kvh), int(pos0), tuple(tok(t) for t in toks[to:to + nt]),
                   tuple(map(tuple, blks[bo:bo + nb].tolist())))
                  for kvh, to, nt, bo, nb, pos0, kind, _ in items)
    recs = sec("wave_records", "wave_off")
    recs = recs[:len(recs) // 128 * 128].reshape(-1, 32, 4)
    n_w = st["n_waves"]
    woff = sec("wave_off", "wave_tiles")[:n_w + 1]
    wtiles = sec("wave_tiles", "end")[:n_w]
    wave, idle = [], 0
    for wv in range(n_w):
        T = int(wtiles[wv])
        if T == 0:
            assert not recs[wv].any() and woff[wv] == woff[wv + 1]
            idle += 1
            continue
        for r in [wv] + list(range(woff[wv], woff[wv + 1])):
            e = recs[r]
            kvh, n_tok, nb_run = int(e[0, 3]), int(e[1, 3]), int(e[2, 3])
            n_blk = int((e[:16, 1] > 0).sum())
            assert (e[:n_blk, 1] > 0).all() and nb_run == ((n_blk + 1) & ~1 if T <= 2 else n_blk)
            assert (e[n_blk:16, 0] == e[0, 0]).all() and not e[n_blk:16, 1:3].any()   # padding format
            assert (e[16 + n_tok:, :3] == e[16, :3]).all() and not e[16:, 3].any()
            wave.append((kvh, T, tuple(map(tuple, e[:n_blk, :3].tolist())), tuple(tok(t) for t in e[16:16 + n_tok])))
    assert idle == st["n_idle_waves"]
    return {"tile": tile, "wave": sorted(wave), "merges": sorted((int(q), int(n)) for q, _, n, _ in merges)}


STRUCT_STATS = ("n_rows", "n_qtok", "n_items", "n_items_shared", "n_items_row", "n_merge", "n_segments",
                "n_shared_segments", "n_items_wave", "logical_qtok", "uniq_kv_tokens", "path_kv_tokens", "flops")


def check_against_fresh(tree, plan, lengths_only):
    fresh = tree.plan()
    for k in STRUCT_STATS:
        assert plan.stats[k] == fresh.stats[k], k
    if lengths_only:
        assert plan.image() == fresh.image()
        assert plan.stats == fresh.stats
    assert decode_image(plan) == decode_image(fresh)


@pytest.mark.parametrize("G,d", [(6, 128), (4, 64), (1, 64)])
def test_update_through_decode_steps(G, d):
    # tails around the 16-block (256-token) boundary, so that steps open new chunks
    tails = [1, 15, 16, 17, 250, 251, 255, 256, 240, 31, 32, 33]
    shape = W.Shape(2 * G, 2, d)
    tree = DecodeTree(7 + G, shape, tails)
    plan = tree.plan()
    n_in_place = n_opened = 0
    for step in range(20):
        items_before = plan.stats["n_items"]
        tree.step()
        _, ki, kb, bl = tree.tables()
        in_place = plan.update(ki, kb, bl)
        n_in_place += in_place
        n_opened += in_place and plan.stats["n_items"] > items_before
        check_against_fresh(tree, plan, lengths_only=False)
    assert n_in_place >= 15 and n_opened >= 2


def test_dirty_words_carry_every_change():
    # the words an in-place update lists are all that differ from the image of the last upload (here:
    # the image at creation, since nothing is uploaded on the CPU): a patch upload is exact
    tree = DecodeTree(13, W.Shape(12, 2, 128), [1, 15, 16, 255, 256, 40, 90])
    plan = tree.plan()
    img0 = np.frombuffer(plan.image()[0], dtype=np.int32).copy()
    for _ in range(18):
        tree.step()
        _, ki, kb, bl = tree.tables()
        assert plan.update(ki, kb, bl)
        idx, complete = tkv.tkv_plan_dirty(plan.h)
        assert complete and len(idx) > 0
        now = np.frombuffer(plan.image()[0], dtype=np.int32)
        patched = img0.copy()
        patched[idx] = now[idx]
        assert np.array_equal(patched, now)
        assert set(np.flatnonzero(img0 != now)) <= set(idx.tolist())


def test_update_lengths_only_is_byte_identical():
    tree = DecodeTree(3, W.Shape(12, 2, 128), [3, 40, 77, 130, 200, 9])
    plan = tree.plan()
    for _ in range(5):
        # only rows whose last block has room: no table changes
        t, _, _, bl = tree.tables()
        tree.step([s for s, tb in zip(tree.decode, t) if bl[tb[-1]] < BS])
        _, ki, kb, bl = tree.tables()
        assert plan.update(ki, kb, bl)
        check_against_fresh(tree, plan, lengths_only=True)


def test_updated_plan_executes_to_oracle():
    shape = W.Shape(8, 2, 64)
    tree = DecodeTree(11, shape, [14, 16, 255, 256, 60])
    plan = tree.plan()
    for _ in range(3):
        tree.step()
        _, ki, kb, bl = tree.tables()
        assert plan.update(ki, kb, bl)
    rng = np.random.default_rng(5)
    kp = rng.standard_normal((tree.num_blocks, shape.hkv, BS, shape.d))
    vp = rng.standard_normal((tree.num_blocks, shape.hkv, BS, shape.d))
    n_qtok = int(sum(tree.q_lens))
    q = rng.standard_normal((n_qtok, shape.hq, shape.d))
    t, _, _, bl = tree.tables()
    o_ref, l_ref = oracle.attention(q, kp, vp, [list(x) for x in t], bl, tree.q_lens)
    o, l = execute_plan(plan.view(), (shape.hq, shape.hkv, shape.d), q, kp, vp, n_qtok)
    np.testing.assert_allclose(o, o_ref, atol=1e-11)
    np.testing.assert_allclose(l, l_ref, atol=1e-11)


def test_update_plans_again_when_tables_change_otherwise():
    tree = DecodeTree(5, W.Shape(8, 2, 64), [20, 40, 300])
    plan = tree.plan()
    # a candidate's open step sealed (no duplicate found, so its blocks stay) and a new open step
    # grown from it: the row's table only grew, past a partly filled block -- in place
    tkv.tkv_bm_seal(tree.bm.h, tree.decode[0])
    child, _, _ = tree.bm.extend(tree.decode[0], np.arange(5, dtype=np.int32), False)
    tree.rows[0] = tree.decode[0] = child
    _, ki, kb, bl = tree.tables()
    assert plan.update(ki, kb, bl)
    check_against_fresh(tree, plan, lengths_only=False)
    # a row's last block replaced by a copy (a new id): not growth -- planned again
    bl2 = bl.copy()
    kb2 = kb.copy()
    free = int(np.flatnonzero(bl == 0)[0])
    bl2[free] = bl[kb[ki[1] - 1]]
    kb2[ki[1] - 1] = free
    assert not plan.update(ki, kb2, bl2)
    fresh = tkv.Plan(tree.dims(), tree.q_indptr(), ki, kb2, bl2, upload=False)
    assert plan.image() == fresh.image() and plan.stats == fresh.stats
    # free slots run out: the same row opening a second new chunk plans again
    tree2 = DecodeTree(6, W.Shape(8, 2, 64), [256, 100], verify=False)
    plan2 = tree2.plan()
    flags = []
    for _ in range(2):
        tree2.step([tree2.decode[0]] * 256)     # 256 tokens: one new chunk per update
        _, ki, kb, bl = tree2.tables()
        flags.append(plan2.update(ki, kb, bl))
        check_against_fresh(tree2, plan2, lengths_only=False)
    assert flags == [True, False]


def test_update_errors_leave_the_plan_unchanged():
    tree = DecodeTree(9, W.Shape(8, 2, 64), [5, 17])
    plan = tree.plan()
    before = plan.image()
    tree.step()
    _, ki, kb, bl = tree.tables()
    bad = kb.copy()
    bad[-1] = tree.num_blocks + 3               # an appended block id out of range
    with pytest.raises(tkv.TkvError) as e:
        plan.update(ki, bad, bl)
    assert e.value.code == tkv.TKV_EINVAL and plan.image() == before
    L = tkv.lib()
    assert L.tkv_plan_update(plan.h, None, None, None, None) == tkv.TKV_EINVAL
    assert plan.update(ki, kb, bl)               # the good tables still go in place
    check_against_fresh(tree, plan, lengths_only=False)


def test_update_of_plans_without_wave_tails_plans_again():
    # G = 32 > 16: every chunk runs as 128-row tiles, no row has a tail the update could grow in place
    tree = DecodeTree(17, W.Shape(64, 2, 64), [20, 40, 300], verify=False)
    plan = tree.plan()
    assert plan.stats["n_items_wave"] == 0 and plan.stats["n_idle_waves"] == 0
    for _ in range(3):
        tree.step()
        _, ki, kb, bl = tree.tables()
        assert not plan.update(ki, kb, bl)
        assert plan.image() == tree.plan().image()


def test_update_with_folded_segments():
    # G = 1 and wave_max_rows 2: each root (6 rows) and its sealed steps (3 rows each) go to the tiles,
    # the root folded into its steps' key runs; the one-row tails stay on the wave grid and grow in place
    tails = [1, 15, 16, 17, 250, 251, 255, 256, 240, 31, 32, 33]
    tree = DecodeTree(31, W.Shape(2, 2, 64), tails, verify=False)
    opts = {"wave_max_rows": 2, "tile_min_items": 0, "fold_blocks": 16}
    _, ki, kb, bl = tree.tables()
    plan = tkv.Plan(tree.dims(), tree.q_indptr(), ki, kb, bl, upload=False, options=opts)
    unfolded = tkv.Plan(tree.dims(), tree.q_indptr(), ki, kb, bl, upload=False, options=dict(opts, fold_blocks=0))
    assert plan.stats["n_shared_segments"] < unfolded.stats["n_shared_segments"]
    n_in_place = 0
    for step in range(12):
        tree.step()
        _, ki, kb, bl = tree.tables()
        n_in_place += plan.update(ki, kb, bl)
        fresh = tkv.Plan(tree.dims(), tree.q_indptr(), ki, kb, bl, upload=False, options=opts)
        assert decode_image(plan) == decode_image(fresh)
    assert n_in_place >= 8


def test_update_keeps_the_plan_options():
    tree = DecodeTree(19, W.Shape(8, 2, 64), [5, 70, 250])
    _, ki, kb, bl = tree.tables()
    opts = {"wave_max_rows": 8, "tile_min_items": 0}
    plan = tkv.Plan(tree.dims(), tree.q_indptr(), ki, kb, bl, upload=False, options=opts)
    tkv.tkv_bm_seal(tree.bm.h, tree.decode[1])          # a table change beyond growth: planned again
    child, _, _ = tree.bm.extend(tree.decode[1], np.arange(3, dtype=np.int32), True)
    tree.rows[1] = tree.decode[1] = child
    tree.step([tree.decode[0]])
    t, ki, kb, bl = tree.tables()
    plan.update(ki, kb, bl)
    fresh = tkv.Plan(tree.dims(), tree.q_indptr(), ki, kb, bl, upload=False, options=opts)
    assert decode_image(plan) == decode_image(fresh) and plan.stats["n_items"] == fresh.stats["n_items"]


def test_update_of_an_empty_plan():
    plan = tkv.Plan((8, 2, 64, 16, 4), [0], [0], [], [16, 3, 0, 0], upload=False)
    assert plan.update([0], [], [16, 4, 0, 0])
    assert plan.stats["n_items"] == 0
