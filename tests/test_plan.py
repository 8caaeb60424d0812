"""Planner checks on CPU: the device work list, executed item by item in float64 by a plain NumPy
interpreter of the descriptor format, must reproduce the oracle; structural invariants of the
plan (coverage, positions, causal limits, slots) hold on the full-size workloads."""
import math

import numpy as np
import pytest

import oracle
import paper_2609_39334_amd as tkv
import workloads as W
from _harness import realize_native, realize_oracle


NO_LIMIT = 1 << 30   # causal limit written for q_len-1 tokens


def _f32(bits):
    return W.bf16_bits_to_f32(bits).astype(np.float64)


def execute_plan(view, shape, q, kp, vp, n_qtok):
    """Interpret the plan: each item contracts its tile against its key list with a plain softmax
    (float64), writing final results or partials; merge entries combine partials by log-sum-exp."""
    hq, hkv, d = shape
    G = hq // hkv
    o = np.full((n_qtok, hq, d), np.nan)
    lse = np.full((n_qtok, hq), np.nan)
    n_slots = view["n_slots"]
    po = np.full((n_slots, hq, d), np.nan)
    pl = np.full((n_slots, hq), np.nan)
    for kvh, tok_off, n_tok, blk_off, n_blk, pos0, kind, _ in view["items"]:
        blks = view["blks"][blk_off:blk_off + n_blk]
        K = np.concatenate([kp[b, kvh, :ln] for b, ln in blks])
        V = np.concatenate([vp[b, kvh, :ln] for b, ln in blks])
        pos = pos0 + np.arange(K.shape[0])
        for qtok, limit, slot, _ in view["toks"][tok_off:tok_off + n_tok]:
            for g in range(G):
                h = kvh * G + g
                s = (K @ q[qtok, h]) / math.sqrt(d)
                s = np.where(pos <= limit, s, -np.inf)
                m = s.max()
                if m == -np.inf:
                    oo, ll = np.zeros(d), -np.inf
                else:
                    p = np.exp(s - m)
                    oo, ll = p @ V / p.sum(), m + math.log(p.sum())
                if slot < 0:
                    o[qtok, h], lse[qtok, h] = oo, ll
                else:
                    po[slot, h], pl[slot, h] = oo, ll
    for qtok, off, n, _ in view["merges"]:
        sl = view["merge_slots"][off:off + n]
        M = pl[sl].max(axis=0)
        w = np.exp(pl[sl] - M)
        o[qtok] = (w[..., None] * po[sl]).sum(axis=0) / w.sum(axis=0)[:, None]
        lse[qtok] = M + np.log(w.sum(axis=0))
    return o, lse


def _run(wl, launch=0):
    b = realize_native(wl)[launch]
    s = wl.shape
    qi, ki, kb = b.arrays()
    plan = tkv.Plan((s.hq, s.hkv, s.d, s.block_size, wl.num_blocks), qi, ki, kb, b.block_len, b.mult, upload=False)
    return b, plan


@pytest.mark.parametrize("seed,G,d", [(0, 1, 64), (1, 4, 64), (2, 6, 128), (3, 7, 128), (4, 16, 64),
                                      (5, 4, 128), (6, 2, 64), (7, 64, 64)])
def test_plan_executes_to_oracle(seed, G, d):
    shape = W.Shape(G * 2, 2, d)
    wl = W.random_tree(seed, shape, n_roots=3, depth=3, max_branch=3, max_step=45)
    b, plan = _run(wl)
    ob = realize_oracle(wl)[0]
    assert ob.tables == b.tables and ob.q_lens == b.q_lens and ob.mult == b.mult
    k, v = wl.kv_values()
    q = wl.q_values(0, b.n_qtok)
    kf, vf, qf = _f32(k), _f32(v), _f32(q)
    o_ref, l_ref = oracle.attention(qf, kf, vf, ob.tables, ob.block_len, ob.q_lens)
    o, l = execute_plan(plan.view(), (shape.hq, shape.hkv, shape.d), qf, kf, vf, b.n_qtok)
    np.testing.assert_allclose(o, o_ref, atol=1e-11)
    np.testing.assert_allclose(l, l_ref, atol=1e-11)


@pytest.mark.parametrize("seed,G,d", [(40, 2, 64), (41, 4, 128), (42, 6, 128), (43, 1, 64)])
def test_folded_segments_execute_to_oracle(seed, G, d):
    # every shared chunk on the 128-row tiles (wave_max_rows 2) and short segments folded into their
    # children's key runs: fewer partial slots, the same attention
    shape = W.Shape(G * 2, 2, d)
    wl = W.random_tree(seed, shape, n_roots=2, depth=4, max_branch=3, max_step=40, p_verify=0.3)
    b = realize_native(wl)[0]
    s = wl.shape
    qi, ki, kb = b.arrays()
    dims = (s.hq, s.hkv, s.d, s.block_size, wl.num_blocks)
    base = dict(wave_max_rows=2, tile_min_items=0)
    plain = tkv.Plan(dims, qi, ki, kb, b.block_len, b.mult, upload=False, options=dict(base, fold_blocks=0))
    fold = tkv.Plan(dims, qi, ki, kb, b.block_len, b.mult, upload=False, options=dict(base, fold_blocks=1000))
    assert fold.stats["n_slots"] < plain.stats["n_slots"]
    assert fold.stats["n_shared_segments"] < plain.stats["n_shared_segments"]
    ob = realize_oracle(wl)[0]
    k, v = wl.kv_values()
    q = wl.q_values(0, b.n_qtok)
    kf, vf, qf = _f32(k), _f32(v), _f32(q)
    o_ref, l_ref = oracle.attention(qf, kf, vf, ob.tables, ob.block_len, ob.q_lens)
    o, l = execute_plan(fold.view(), (shape.hq, shape.hkv, shape.d), qf, kf, vf, b.n_qtok)
    np.testing.assert_allclose(o, o_ref, atol=1e-11)
    np.testing.assert_allclose(l, l_ref, atol=1e-11)


def test_plan_tiny_decode_structure():
    b, plan = _run(W.tiny_decode(0))
    st = plan.stats
    assert st["n_rows"] == 4 and st["n_qtok"] == 4
    assert st["uniq_kv_tokens"] == 512 and st["path_kv_tokens"] == 4 * 320
    assert st["n_shared_segments"] == 1 and st["n_segments"] == 5
    v = plan.view()
    # the shared prompt is one chunk contracted against all 4 tokens x 4 heads in one tile per KV head
    shared = [it for it in v["items"] if it[4] == 16]
    assert len(shared) == 2 and all(it[2] == 4 for it in shared)
    # two partials per token (prompt chunk, private tail), and one slot kept free per token for
    # the chunk its tail opens next
    assert st["n_merge"] == 4 and st["n_slots"] == 12
    assert all(m[2] == 2 for m in v["merges"]) and sorted(m[1] for m in v["merges"]) == [0, 3, 6, 9]
    assert st["n_idle_waves"] > 0


@pytest.mark.parametrize("name", ["beam_decode", "step_verify", "spec_explosion", "mixed_serving"])
def test_plan_covers_each_path_exactly_once(name):
    wl = W.CONFIGS[name](0)
    b, plan = _run(wl, launch=len(wl.launches) - 1)
    v = plan.view()
    s = wl.shape
    qi, ki, kb = b.arrays()
    # expected: every (query token, kv head) sees the blocks of its row's path up to its limit
    row_of_tok = np.repeat(np.arange(len(b.q_lens)), b.q_lens)
    rng = np.random.default_rng(0)
    sample = np.arange(b.n_qtok) if b.n_qtok <= 4000 else np.unique(np.concatenate(
        [rng.choice(b.n_qtok, 3000, replace=False), [0, b.n_qtok - 1]]))
    want = np.zeros(b.n_qtok, dtype=bool)
    want[sample] = True
    seen = {}
    for kvh, tok_off, n_tok, blk_off, n_blk, pos0, kind, _ in v["items"]:
        tk = v["toks"][tok_off:tok_off + n_tok]
        tk = tk[want[tk[:, 0]]]
        if not len(tk):
            continue
        blks = [int(x) for x in v["blks"][blk_off:blk_off + n_blk, 0]]
        for qtok, limit, slot, _ in tk:
            seen.setdefault((int(qtok), int(kvh)), []).append((int(pos0), blks, int(slot), int(limit)))
    bl = b.block_len
    for qtok in sample:
        r = row_of_tok[qtok]
        i = qtok - qi[r]
        table = b.tables[r]
        N = int(sum(bl[x] for x in table))
        lim = N - b.q_lens[r] + i
        lim_desc = NO_LIMIT if b.q_lens[r] == 1 else lim   # a decode token sees its whole path
        starts = np.concatenate([[0], np.cumsum([bl[x] for x in table])])
        need = [table[j] for j in range(len(table)) if starts[j] <= lim]
        for kvh in range(s.hkv):
            parts = seen[(qtok, kvh)]
            assert all(p[3] == lim_desc for p in parts)
            got = []
            for pos0, blks, slot, _ in sorted(parts):
                assert pos0 == starts[len(got)]      # contiguous, in path order
                got += blks
            assert got[:len(need)] == need and all(starts[table.index(x)] > lim for x in got[len(need):])
            assert (len(parts) == 1) == (parts[0][2] < 0)
    st = plan.stats
    assert st["n_items"] == len(v["items"])
    if name == "step_verify":
        assert st["n_items_row"] == st["n_items"] and st["n_merge"] == 0
    if name == "beam_decode":
        assert st["n_items_shared"] == st["n_items"] and st["n_shared_segments"] > 0
        # the 16 prompts, each read by 32 live beams x 6 query heads, go to 128-row tile items; the
        # wave grid keeps clear of the workgroup slots (2 per CU, 4 waves each) those take
        n_tile = st["n_items"] - st["n_items_wave"]
        assert 0 < n_tile < 512 and 4 * n_tile + st["n_waves"] - st["n_idle_waves"] <= 2048


@pytest.mark.parametrize("options,max_wave_rows", [(None, 32), ({"wave_max_rows": 96}, 96)])
def test_chunks_route_by_their_query_rows(options, max_wave_rows):
    # a chunk read by at most wave_max_rows query rows (32 by default) goes to the wave grid; a wider
    # one to 128-row tile items, which together hold every one of its tokens
    wl = W.spec_explosion(0)
    b = realize_native(wl)[0]
    s = wl.shape
    G = s.hq // s.hkv
    qi, ki, kb = b.arrays()
    plan = tkv.Plan((s.hq, s.hkv, s.d, s.block_size, wl.num_blocks), qi, ki, kb, b.block_len, b.mult, upload=False,
                    options=options)
    v = plan.view()
    chunk_toks, n_wave = {}, 0
    for kvh, tok_off, n_tok, blk_off, n_blk, pos0, kind, _ in v["items"]:
        if kind == 2:                                  # wave item: one tile of one chunk
            assert n_tok * G <= max_wave_rows
            n_wave += 1
        else:
            assert kind == 0 and n_tok * G <= 128
            chunk_toks[(kvh, blk_off, n_blk)] = chunk_toks.get((kvh, blk_off, n_blk), 0) + n_tok
    assert n_wave > 0 and chunk_toks
    assert all(t * G > max_wave_rows for t in chunk_toks.values())
    # spec_explosion's 16-candidate subtrees (96 query rows) change sides between the two thresholds
    assert any(t * G == 96 for t in chunk_toks.values()) == (max_wave_rows < 96)


def test_plan_rejects_bad_input():
    ok = dict(shape=(8, 2, 64, 16, 4), q_indptr=[0, 1], kv_indptr=[0, 2], kv_blocks=[0, 1], block_len=[16, 3, 0, 0])
    tkv.tkv_plan_destroy(tkv.tkv_plan_create(**ok))
    bad = [
        dict(ok, shape=(8, 3, 64, 16, 4)),             # hq % hkv
        dict(ok, shape=(8, 2, 96, 16, 4)),             # head dim
        dict(ok, shape=(8, 2, 64, 32, 4)),             # block size
        dict(ok, kv_blocks=[0, 2]),                    # free block
        dict(ok, kv_blocks=[0, 7]),                    # out of range
        dict(ok, q_indptr=[0, 20]),                    # q_len > kv_len
        dict(ok, q_indptr=[0, 0]),                     # q_len 0
        dict(ok, shape=(130, 2, 64, 16, 4)),           # group too large
    ]
    for kw in bad:
        with pytest.raises(tkv.TkvError) as e:
            tkv.tkv_plan_create(**kw)
        assert e.value.code == tkv.TKV_EINVAL, kw
    with pytest.raises(tkv.TkvError):
        tkv.tkv_plan_create(**ok, multiplicity=[0])


def test_decode_rejects_verify_rows_without_gpu_work():
    plan = tkv.tkv_plan_create((8, 2, 64, 16, 4), [0, 2], [0, 2], [0, 1], [16, 3, 0, 0])
    L = tkv.lib()
    rc = L.tkv_decode(plan, 1, 1, 1, 1, None, None)     # rejected before any device access
    assert rc == tkv.TKV_EINVAL and "q_len" in tkv.tkv_last_error()
    rc = L.tkv_verify(plan, 1, 1, 1, 1, None, None)      # not uploaded: rejected before any launch
    assert rc == tkv.TKV_EINVAL and "uploaded" in tkv.tkv_last_error()
    tkv.tkv_plan_destroy(plan)


def test_empty_plan():
    plan = tkv.tkv_plan_create((8, 2, 64, 16, 4), [0], [0], [], [16, 3, 0, 0])
    st = tkv.tkv_plan_get_stats(plan)
    assert st["n_items"] == 0 and st["n_rows"] == 0
    assert tkv.tkv_plan_workspace_bytes(plan) >= 256
    tkv.tkv_plan_destroy(plan)


def test_plans_do_not_depend_on_earlier_plans():
    # destroyed plans are recycled with their arrays' storage: a plan must come out the same whatever
    # plans were made and destroyed before it
    cases = {"tiny": W.tiny_decode(0), "rt": W.random_tree(3, W.Shape(12, 2, 128), n_roots=3, depth=3),
             "verify": W.step_verify(0, n_queries=2, n_cands=4)}
    seen = {}
    for order in (["tiny", "rt", "verify"], ["verify", "tiny", "rt"], ["rt", "verify", "tiny"]):
        for name in order:
            b, plan = _run(cases[name])
            got = (plan.image(), plan.stats)
            assert seen.setdefault(name, got) == got, name
            del plan
