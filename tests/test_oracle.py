"""Pins for the oracle: checks that do not come from the oracle itself.

Attention: hand-worked fixture, brute force in pure Python (math module only) on tiny inputs,
closed forms and invariants (single key, equal scores, per-path duplication of shared blocks,
split + log-sum-exp merge, key permutation for decode, GQA == MHA with repeated KV heads,
causal verify == decode over truncated prefixes, padding never read).
Block manager: hand-worked fixtures, the paper's computation-deduplication example, and a
brute-force characterisation of deduplication checked after every operation of random scripts.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle.block_manager import BMError
from workloads import Shape, random_tree, tiny_decode, drive

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# ============================================================================ attention

def _pool(nb, hkv, bs, d, rng):
    return rng.standard_normal((nb, hkv, bs, d))


def test_worked_example_decode_and_verify():
    g = _load("softmax_worked.json")
    d = g["d"]
    k = np.zeros((1, 1, 16, d))
    v = np.zeros((1, 1, 16, d))
    k[0, 0, :3, 0] = [math.log(1), math.log(2), math.log(3)]
    v[0, 0, :3, :] = np.array(g["v"])
    bl = [3]
    q = np.array(g["q"]).reshape(1, 1, d)
    o, lse = oracle.attention(q, k, v, [[0]], bl, [1])
    np.testing.assert_allclose(o[0, 0], g["decode_o"], atol=1e-12)
    assert abs(lse[0, 0] - math.log(6)) < 1e-12
    q2 = np.repeat(q, 2, axis=0)
    o, lse = oracle.attention(q2, k, v, [[0]], bl, [2])
    np.testing.assert_allclose(o[:, 0], g["verify_o"], atol=1e-12)
    np.testing.assert_allclose(lse[:, 0], [math.log(3), math.log(6)], atol=1e-12)


def _brute(q, kp, vp, table, bl, L):
    """Pure-Python scaled dot-product attention for one row (no numpy arithmetic)."""
    nqt, hq, d = q.shape
    hkv = kp.shape[1]
    G = hq // hkv
    keys = [(b, s) for b in table for s in range(bl[b])]
    N = len(keys)
    out_o, out_l = [], []
    for i in range(L):
        oi, li = [], []
        for h in range(hq):
            kv = h // G
            qv = [float(x) for x in q[i, h]]
            sc = []
            for j in range(N - L + i + 1):
                b, s = keys[j]
                sc.append(math.fsum(qv[t] * float(kp[b, kv, s, t]) for t in range(d)) / math.sqrt(d))
            m = max(sc)
            w = [math.exp(x - m) for x in sc]
            tot = math.fsum(w)
            o = []
            for t in range(d):
                o.append(math.fsum(w[j] * float(vp[keys[j][0], kv, keys[j][1], t]) for j in range(len(w))) / tot)
            oi.append(o)
            li.append(m + math.log(tot))
        out_o.append(oi)
        out_l.append(li)
    return np.array(out_o), np.array(out_l)


@pytest.mark.parametrize("G", [1, 4, 6, 7])
def test_brute_force_tiny(G):
    rng = np.random.default_rng(100 + G)
    hkv, d, bs = 2, 8, 4
    hq = G * hkv
    for trial in range(6):
        nb = 14
        kp, vp = _pool(nb, hkv, bs, d, rng), _pool(nb, hkv, bs, d, rng)
        bl = rng.integers(1, bs + 1, size=nb).tolist()
        tables, qls = [], []
        for r in range(3):
            t = rng.permutation(nb)[: rng.integers(1, 8)].tolist()
            N = sum(bl[b] for b in t)
            tables.append(t)
            qls.append(int(rng.integers(1, min(5, N) + 1)))
        q = rng.standard_normal((sum(qls), hq, d))
        o, lse = oracle.attention(q, kp, vp, tables, bl, qls)
        off = 0
        for t, L in zip(tables, qls):
            bo, bl_ = _brute(q[off:off + L], kp, vp, t, bl, L)
            np.testing.assert_allclose(o[off:off + L], bo, rtol=1e-11, atol=1e-12)
            np.testing.assert_allclose(lse[off:off + L], bl_, rtol=1e-11, atol=1e-12)
            off += L


def test_brute_force_long_key_range():
    # kv_len up to 40 single-head keys with several q_len values (the exhaustive corner of the pin).
    rng = np.random.default_rng(7)
    d, bs = 4, 16
    kp, vp = _pool(3, 1, bs, d, rng), _pool(3, 1, bs, d, rng)
    for N in range(1, 41):
        bl = [min(16, N), min(16, max(0, N - 16)), max(0, N - 32)]
        table = [b for b in range(3) if bl[b] > 0]
        for L in range(1, min(5, N) + 1):
            q = rng.standard_normal((L, 1, d))
            o, lse = oracle.attention(q, kp, vp, [table], bl, [L])
            bo, bl_ = _brute(q, kp, vp, table, bl, L)
            np.testing.assert_allclose(o, bo, rtol=1e-11, atol=1e-12)
            np.testing.assert_allclose(lse, bl_, rtol=1e-11, atol=1e-12)


def test_single_key_returns_v():
    rng = np.random.default_rng(1)
    kp, vp = _pool(2, 2, 16, 64, rng), _pool(2, 2, 16, 64, rng)
    q = rng.standard_normal((1, 8, 64))
    o, lse = oracle.attention(q, kp, vp, [[1]], [0, 1], [1])
    for h in range(8):
        np.testing.assert_array_equal(o[0, h], vp[1, h // 4, 0])
        assert lse[0, h] == pytest.approx(float(q[0, h] @ kp[1, h // 4, 0]) / 8.0, abs=1e-12)


def test_equal_scores_give_mean_of_attended_v():
    rng = np.random.default_rng(2)
    kp, vp = _pool(4, 1, 16, 32, rng), _pool(4, 1, 16, 32, rng)
    bl = [16, 5, 16, 9]
    table = [2, 1, 3]
    N = 30
    L = 4
    q = np.zeros((L, 2, 32))
    o, lse = oracle.attention(q, kp, vp, [table], bl, [L])
    allv = np.concatenate([vp[b, 0, :bl[b]] for b in table])
    for i in range(L):
        n = N - L + i + 1
        np.testing.assert_allclose(o[i, 0], allv[:n].mean(axis=0), atol=1e-13)
        assert lse[i, 1] == pytest.approx(math.log(n), abs=1e-13)
    # identical keys with a nonzero query: also equal scores
    kp2 = kp.copy()
    kp2[:, 0] = kp2[0, 0, 0]
    q = rng.standard_normal((1, 2, 32))
    o, _ = oracle.attention(q, kp2, vp, [table], bl, [1])
    np.testing.assert_allclose(o[0, 1], allv.mean(axis=0), atol=1e-12)


def test_duplicating_shared_blocks_changes_nothing():
    shape = Shape(8, 2, 16, 16)
    wl = random_tree(5, shape, n_roots=2, depth=3)
    bm = oracle.BlockManager(wl.num_blocks, 16, wl.max_seqs)
    got = {}
    drive(wl, bm, on_launch=lambda i, l, c: got.setdefault("c", c))
    seqs = got["c"]
    tables = [bm.table(s) for s, _ in seqs]
    qls = [q for _, q in seqs]
    rng = np.random.default_rng(3)
    kp, vp = _pool(wl.num_blocks, 2, 16, 16, rng), _pool(wl.num_blocks, 2, 16, 16, rng)
    bl = list(bm.block_len)
    q = rng.standard_normal((sum(qls), 8, 16))
    o1, l1 = oracle.attention(q, kp, vp, tables, bl, qls)
    # give every row a private copy of every block it references
    n_ref = sum(len(t) for t in tables)
    kp2 = np.zeros((n_ref,) + kp.shape[1:])
    vp2 = np.zeros_like(kp2)
    bl2, tables2, nxt = [], [], 0
    for t in tables:
        nt = []
        for b in t:
            kp2[nxt], vp2[nxt] = kp[b], vp[b]
            bl2.append(bl[b])
            nt.append(nxt)
            nxt += 1
        tables2.append(nt)
    assert n_ref > len(set(b for t in tables for b in t))     # there was sharing to undo
    o2, l2 = oracle.attention(q, kp2, vp2, tables2, bl2, qls)
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(l1, l2)


def test_split_and_lse_merge_equals_whole():
    rng = np.random.default_rng(4)
    kp, vp = _pool(10, 2, 16, 32, rng), _pool(10, 2, 16, 32, rng)
    bl = rng.integers(1, 17, size=10).tolist()
    table = [3, 7, 1, 9, 0, 5]
    q = rng.standard_normal((1, 6, 32))
    o, lse = oracle.attention(q, kp, vp, [table], bl, [1])
    parts = [oracle.attention(q, kp, vp, [table[a:b]], bl, [1]) for a, b in ((0, 2), (2, 3), (3, 6))]
    ls = np.stack([p[1] for p in parts])                  # [3, 1, Hq]
    M = ls.max(axis=0)
    w = np.exp(ls - M)
    merged_lse = M + np.log(w.sum(axis=0))
    merged_o = sum(w[i][..., None] * parts[i][0] for i in range(3)) / w.sum(axis=0)[..., None]
    np.testing.assert_allclose(merged_o, o, atol=1e-12)
    np.testing.assert_allclose(merged_lse, lse, atol=1e-12)


def test_decode_key_permutation_invariance():
    rng = np.random.default_rng(5)
    kp, vp = _pool(8, 2, 16, 32, rng), _pool(8, 2, 16, 32, rng)
    bl = rng.integers(1, 17, size=8).tolist()
    table = [0, 1, 2, 3, 4, 5, 6, 7]
    q = rng.standard_normal((1, 4, 32))
    o1, l1 = oracle.attention(q, kp, vp, [table], bl, [1])
    o2, l2 = oracle.attention(q, kp, vp, [table[::-1]], bl, [1])
    np.testing.assert_allclose(o1, o2, atol=1e-12)
    np.testing.assert_allclose(l1, l2, atol=1e-12)


def test_gqa_equals_mha_with_repeated_kv():
    rng = np.random.default_rng(6)
    G = 6
    kp, vp = _pool(5, 2, 16, 16, rng), _pool(5, 2, 16, 16, rng)
    bl = [16, 16, 7, 16, 3]
    tables = [[0, 1, 2], [0, 3, 4]]
    q = rng.standard_normal((1 + 3, 12, 16))
    o1, l1 = oracle.attention(q, kp, vp, tables, bl, [1, 3])
    kr = np.repeat(kp, G, axis=1)
    vr = np.repeat(vp, G, axis=1)
    o2, l2 = oracle.attention(q, kr, vr, tables, bl, [1, 3])
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-13)     # GEMM shapes differ: rounding order only
    np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-13)


def test_causal_verify_equals_decode_on_truncated_prefixes():
    # one token per block, so a prefix of any length is a whole-block table
    rng = np.random.default_rng(8)
    N, L = 23, 6
    kp, vp = _pool(N, 2, 16, 32, rng), _pool(N, 2, 16, 32, rng)
    bl = [1] * N
    table = list(rng.permutation(N))
    q = rng.standard_normal((L, 4, 32))
    o, lse = oracle.attention(q, kp, vp, [table], bl, [L])
    for i in range(L):
        oi, li = oracle.attention(q[i:i + 1], kp, vp, [table[:N - L + i + 1]], bl, [1])
        np.testing.assert_allclose(o[i], oi[0], atol=1e-12)
        np.testing.assert_allclose(lse[i], li[0], atol=1e-12)


def test_padding_is_never_read():
    rng = np.random.default_rng(9)
    kp, vp = _pool(4, 2, 16, 16, rng), _pool(4, 2, 16, 16, rng)
    bl = [5, 16, 1, 12]
    kn, vn = kp.copy(), vp.copy()
    for b in range(4):
        kn[b, :, bl[b]:] = np.nan
        vn[b, :, bl[b]:] = np.nan
    q = rng.standard_normal((3, 4, 16))
    o1, l1 = oracle.attention(q, kp, vp, [[0, 1, 2, 3]], bl, [3])
    o2, l2 = oracle.attention(q, kn, vn, [[0, 1, 2, 3]], bl, [3])
    assert np.isfinite(o2).all() and np.isfinite(l2).all()
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(l1, l2)


def test_rejects_q_len_beyond_kv_len():
    rng = np.random.default_rng(10)
    kp, vp = _pool(1, 1, 16, 8, rng), _pool(1, 1, 16, 8, rng)
    with pytest.raises(ValueError):
        oracle.attention(np.zeros((4, 1, 8)), kp, vp, [[0]], [3], [4])


# ============================================================================ block manager

def _tokens(spec):
    if isinstance(spec, dict):
        a, b = spec["range"]
        return list(range(a, b))
    return list(spec)


def _expand(spec, n):
    out = np.zeros(n, dtype=np.int64)
    for k, v in spec.items():
        if "-" in k:
            a, b = map(int, k.split("-"))
            out[a:b + 1] = v
        else:
            out[int(k)] = v
    return out


@pytest.mark.parametrize("case", _load("bm_cases.json")["cases"], ids=lambda c: c["name"])
def test_bm_golden_cases(case):
    bm = oracle.BlockManager(case["num_blocks"], case["block_size"], case["max_seqs"])
    for op in case["ops"]:
        exp = op["expect"]
        before = bm.snapshot()
        try:
            if op["op"] == "extend":
                seq, blocks, hits = bm.extend(op["parent"], _tokens(op["tokens"]), bool(op["seal"]))
                got = {"seq": seq, "blocks": blocks, "hits": hits}
            elif op["op"] == "append":
                got = {"dst": bm.append(op["seq"], _tokens(op["tokens"]))}
            elif op["op"] == "seal":
                got = {"replaced": [list(r) for r in bm.seal(op["seq"])]}
            else:
                got = {"freed": bm.prune(op["seq"])}
        except BMError as e:
            got = {"error": e.code}
            after = bm.snapshot()
            for k in ("refcount", "block_len", "indexed"):
                np.testing.assert_array_equal(before[k], after[k])
            assert before["seqs"] == after["seqs"]
        assert got == exp, (op, got)
    fin = case["final"]
    nb = case["num_blocks"]
    snap = bm.snapshot()
    np.testing.assert_array_equal(snap["refcount"], _expand(fin["refcount"], nb))
    np.testing.assert_array_equal(snap["block_len"], _expand(fin["block_len"], nb))
    if "indexed" in fin:
        np.testing.assert_array_equal(snap["indexed"], _expand(fin["indexed"], nb))
    assert {str(s): list(t) for s, (t, _, _) in snap["seqs"].items()} == fin["tables"]
    for s, n in fin["kv_len"].items():
        assert bm.kv_len(int(s)) == n


def test_cd_paris_example():
    g = _load("cd_paris.json")
    bm = oracle.BlockManager(8, g["block_size"], 8)
    p, _, _ = bm.extend(-1, g["prefix"], True)
    blocks, hits, tables = [], [], []
    for t in g["samples"]:
        s, b, h = bm.extend(p, [t], True)
        blocks += b
        hits += h
        tables.append(bm.table(s))
    assert blocks == g["expect"]["sample_blocks"] and hits == g["expect"]["sample_hits"]
    row_of, first, mult = oracle.coalesce(tables, [1] * 4)
    assert row_of == g["expect"]["row_of_candidate"]
    assert mult == g["expect"]["multiplicity"]
    assert first == g["expect"]["first_candidate"]


def test_tiny_decode_workload_structure():
    wl = tiny_decode(0)
    bm = oracle.BlockManager(wl.num_blocks, 16, wl.max_seqs)
    got = {}
    drive(wl, bm, on_launch=lambda i, l, c: got.setdefault("c", c))
    for c, (s, q) in enumerate(got["c"]):
        assert q == 1
        assert bm.table(s) == list(range(16)) + list(range(16 + 4 * c, 20 + 4 * c))
    assert bm.refcount[:16] == [4] * 16 and bm.refcount[16:32] == [1] * 16


class _BruteTracker:
    """Independent model of deduplication: two live table entries hold the same block iff they are
    chunks of sealed steps with the same full chunk history from the root, or are the very same
    chunk of one unsealed step (inherited by nobody, since unsealed sequences cannot be extended)."""

    def __init__(self, bs):
        self.bs = bs
        self.ident = {}        # seq -> list of chunk identities
        self.sealed = {}

    def extend(self, parent, toks, seal, op_id):
        base = [] if parent == -1 else list(self.ident[parent])
        chunks = [tuple(toks[i:i + self.bs]) for i in range(0, len(toks), self.bs)]
        for ci, c in enumerate(chunks):
            if seal:
                prev = base[-1] if base else ("root",)
                base.append(("S", prev, c))
            else:
                base.append(("U", op_id, ci))
        return base


def _check_bm_against_brute(bm, tracker, used_before, new_ids):
    snap = bm.snapshot()
    live = snap["seqs"]
    ref = np.zeros(bm.num_blocks, dtype=np.int64)
    owner = {}
    for s, (table, _, _) in live.items():
        ids = tracker.ident[s]
        assert len(ids) == len(table)
        for b, idn in zip(table, ids):
            ref[b] += 1
            if idn in owner:
                assert owner[idn] == b, "equal chunk histories must share a block"
            owner[idn] = b
    assert len(set(owner.values())) == len(owner), "different chunk histories must not share a block"
    np.testing.assert_array_equal(snap["refcount"], ref)
    assert ((snap["block_len"] > 0) == (ref > 0)).all()
    # fresh blocks are the lowest ids that were free before the operation
    if new_ids:
        free_before = sorted(set(range(bm.num_blocks)) - used_before)
        assert sorted(new_ids) == free_before[:len(new_ids)]


@pytest.mark.parametrize("seed", range(8))
def test_bm_random_scripts_match_brute_force(seed):
    rng = np.random.default_rng(seed)
    bs = 4
    bm = oracle.BlockManager(64, bs, 24)
    tr = _BruteTracker(bs)
    live = []
    sealed = set()
    for op_id in range(150):
        used = set(int(b) for b in np.nonzero(np.array(bm.refcount))[0])
        if live and rng.random() < 0.3:
            s = live.pop(int(rng.integers(0, len(live))))
            bm.prune(s)
            del tr.ident[s]
            sealed.discard(s)
            _check_bm_against_brute(bm, tr, used, [])
            continue
        cands = [s for s in live if s in sealed]
        parent = -1 if not cands or rng.random() < 0.2 else cands[int(rng.integers(0, len(cands)))]
        vocab = 3 if rng.random() < 0.5 else 50          # tiny vocab -> frequent identical steps
        toks = rng.integers(0, vocab, size=int(rng.integers(1 if parent == -1 else 0, 11))).tolist()
        seal = bool(rng.random() < 0.7)
        try:
            s, new_blocks, hits = bm.extend(parent, toks, seal)
        except BMError as e:
            assert e.code == -2           # pool or sequence slots exhausted
            continue
        tr.ident[s] = tr.extend(parent, toks, seal, op_id)
        live.append(s)
        if seal:
            sealed.add(s)
        fresh = [b for b, h in zip(new_blocks, hits) if not h]
        assert all(h == 0 for h in hits[len(new_blocks) - len(fresh):])   # misses never precede hits
        _check_bm_against_brute(bm, tr, used, fresh)


class _StepTracker(_BruteTracker):
    """The brute-force model of deduplication extended to steps grown token by token: a chunk of an
    open step is private (identity: the step and the chunk's place in it), and sealing gives each of
    its chunks the identity a sealed extension would -- its tokens and its predecessor's identity."""

    def __init__(self, bs):
        super().__init__(bs)
        self.open = {}         # seq -> (step id, tokens of the open step)

    def extend_seq(self, s, parent, toks, seal, op_id):
        self.ident[s] = self.extend(parent, toks, seal, op_id)
        if not seal:
            self.open[s] = (op_id, list(toks))

    def append(self, s, toks, op_id):
        if s not in self.open:                          # a sealed sequence starts a new step
            self.open[s] = (op_id, [])
        sid, ot = self.open[s]
        before = -(-len(ot) // self.bs)
        ot.extend(toks)
        self.ident[s] += [("U", sid, ci) for ci in range(before, -(-len(ot) // self.bs))]

    def seal(self, s):
        _, ot = self.open.pop(s)
        chunks = [tuple(ot[i:i + self.bs]) for i in range(0, len(ot), self.bs)]
        base = self.ident[s][:len(self.ident[s]) - len(chunks)]
        for c in chunks:
            base.append(("S", base[-1] if base else ("root",), c))
        self.ident[s] = base

    def drop(self, s):
        del self.ident[s]
        self.open.pop(s, None)


@pytest.mark.parametrize("seed", range(8))
def test_bm_decode_steps_match_brute_force(seed):
    # extensions, token-by-token appends, seals and prunes in random order: after every operation
    # equal chunk histories share a block, different ones do not, refcounts count holders, and fresh
    # blocks are the lowest free ids
    rng = np.random.default_rng(100 + seed)
    bs = 4
    bm = oracle.BlockManager(96, bs, 24)
    tr = _StepTracker(bs)
    live = []
    for op_id in range(250):
        used = set(int(b) for b in np.nonzero(np.array(bm.refcount))[0])
        r = rng.random()
        vocab = 2 if rng.random() < 0.6 else 50            # tiny vocab -> frequent identical steps
        if live and r < 0.15:
            s = live.pop(int(rng.integers(0, len(live))))
            bm.prune(s)
            tr.drop(s)
            _check_bm_against_brute(bm, tr, used, [])
        elif live and r < 0.55:
            s = live[int(rng.integers(0, len(live)))]
            toks = rng.integers(0, vocab, size=int(rng.integers(0, 7))).tolist()
            table_before = bm.table(s)
            try:
                dst = bm.append(s, toks)
            except BMError as e:
                assert e.code == -2
                continue
            tr.append(s, toks, op_id)
            table = bm.table(s)
            fresh = table[len(table_before):]
            # the tokens fill the path's last blocks in order: consecutive slots, block after block
            runs = [d // bs for i, d in enumerate(dst) if i == 0 or d // bs != dst[i - 1] // bs]
            assert runs == table[len(table) - len(runs):]
            assert all(dst[i] + 1 == dst[i + 1] for i in range(len(dst) - 1) if dst[i] // bs == dst[i + 1] // bs)
            assert all(d % bs == 0 for i, d in enumerate(dst) if i > 0 and d // bs != dst[i - 1] // bs)
            _check_bm_against_brute(bm, tr, used, fresh)
        elif live and r < 0.7:
            uns = [s for s in live if s in tr.open]
            if not uns:
                continue
            s = uns[int(rng.integers(0, len(uns)))]
            bm.seal(s)
            tr.seal(s)
            _check_bm_against_brute(bm, tr, used, [])
        else:
            cands = [s for s in live if s not in tr.open]
            parent = -1 if not cands or rng.random() < 0.2 else cands[int(rng.integers(0, len(cands)))]
            toks = rng.integers(0, vocab, size=int(rng.integers(1 if parent == -1 else 0, 9))).tolist()
            seal = bool(rng.random() < 0.5)
            try:
                s, new_blocks, hits = bm.extend(parent, toks, seal)
            except BMError as e:
                assert e.code == -2
                continue
            tr.extend_seq(s, parent, toks, seal, op_id)
            live.append(s)
            _check_bm_against_brute(bm, tr, used, [b for b, h in zip(new_blocks, hits) if not h])


def test_append_then_seal_equals_sealed_extension():
    # a step decoded token by token and sealed ends on the same blocks as the same step extended
    # sealed in one go (here the sealed copy exists first, so every block is a hit)
    bm = oracle.BlockManager(40, 4, 8)
    root, _, _ = bm.extend(-1, [5, 6, 7, 8, 9], True)
    toks = [1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11]
    twin, _, _ = bm.extend(root, toks, True)
    cand, _, _ = bm.extend(root, [], False)
    for t in toks:
        bm.append(cand, [t])
    repl = bm.seal(cand)
    assert bm.table(cand) == bm.table(twin) and len(repl) == 3
    assert all(bm.refcount[b] == 2 for b in bm.table(twin)[2:])
    assert bm.kv_len(cand) == 5 + len(toks)


@pytest.mark.parametrize("seed", range(6))
def test_kv_append_rows_follow_paths(seed):
    # A decode loop writes each new token's K row with oracle.kv_append at the slot the block manager
    # gave it (append: its own slots; a sealed extension: its blocks' slots, none for a hit block).
    # Independently, every path's rows are modelled position by position: a token appended or
    # extended brings its own row, except in a chunk that deduplicated, which shows the rows of the
    # chunk's first writer.  Gathering every live path from the pool must give the modelled rows.
    rng = np.random.default_rng(300 + seed)
    bs, hkv, d = 4, 2, 3
    bm = oracle.BlockManager(80, bs, 16)
    tr = _StepTracker(bs)
    pool = np.full((80, hkv, bs, d), np.nan)
    vpool = np.full((80, hkv, bs, d), np.nan)
    first_rows = {}                  # sealed chunk identity -> rows of its first writer
    open_rows = {}                   # seq -> rows of its open step
    rows = {}                        # seq -> modelled rows, one [hkv, d] array per path position
    live = []

    def fresh(n):
        return rng.standard_normal((n, hkv, d))

    def settle(s):
        # positions of sealed chunks show their first writer's rows
        out, pos = [], 0
        for ci, idn in enumerate(tr.ident[s]):
            n_in = bm.block_len[bm.table(s)[ci]]
            if idn[0] == "S":
                out += list(first_rows[idn])
            else:
                out += list(rows[s][pos:pos + n_in])
            pos += n_in
        rows[s] = out

    for op_id in range(160):
        r = rng.random()
        vocab = 2 if rng.random() < 0.6 else 40
        if live and r < 0.15:
            s = live.pop(int(rng.integers(0, len(live))))
            bm.prune(s)
            tr.drop(s)
            del rows[s]
            continue
        if live and r < 0.55:
            s = live[int(rng.integers(0, len(live)))]
            toks = rng.integers(0, vocab, size=int(rng.integers(0, 6))).tolist()
            try:
                dst = bm.append(s, toks)
            except BMError:
                continue
            tr.append(s, toks, op_id)
            new = fresh(len(toks))
            oracle.kv_append(pool, vpool, dst, new, new)
            rows[s] = rows[s] + list(new)
        elif live and r < 0.7:
            s = live[int(rng.integers(0, len(live)))]
            if s not in tr.open:
                continue
            n_open = -(-len(tr.open[s][1]) // bs)
            base = len(tr.ident[s]) - n_open
            blens = [bm.block_len[b] for b in bm.table(s)]
            start = sum(blens[:base])
            bm.seal(s)
            tr.seal(s)
            pos = start
            for ci in range(base, len(tr.ident[s])):
                n_in = bm.block_len[bm.table(s)[ci]]
                first_rows.setdefault(tr.ident[s][ci], rows[s][pos:pos + n_in])
                pos += n_in
            settle(s)
        else:
            cands = [s for s in live if s not in tr.open]
            parent = -1 if not cands or rng.random() < 0.2 else cands[int(rng.integers(0, len(cands)))]
            toks = rng.integers(0, vocab, size=int(rng.integers(1 if parent == -1 else 0, 9))).tolist()
            seal = bool(rng.random() < 0.5)
            try:
                s, blk, hit = bm.extend(parent, toks, seal)
            except BMError:
                continue
            tr.extend_seq(s, parent, toks, seal, op_id)
            live.append(s)
            dst = [-1 if hit[t // bs] else blk[t // bs] * bs + t % bs for t in range(len(toks))]
            new = fresh(len(toks))
            oracle.kv_append(pool, vpool, dst, new, new)
            rows[s] = (list(rows[parent]) if parent >= 0 else []) + list(new)
            if seal:
                base = len(tr.ident[s]) - len(blk)
                for j in range(len(blk)):
                    a = j * bs
                    first_rows.setdefault(tr.ident[s][base + j], list(new[a:a + bs]))
            settle(s)
        for s in live:
            got = oracle.gather_kv(pool, bm.table(s), bm.block_len)       # [hkv, N, d]
            want = np.stack(rows[s], axis=1) if rows[s] else np.zeros((hkv, 0, d))
            np.testing.assert_array_equal(got, want)


def _softmax_py(logits, temperature):
    # plain Python (math module), independent of the oracle's NumPy
    m = max(logits)
    e = [math.exp((x - m) / temperature) if x != -math.inf else 0.0 for x in logits]
    z = sum(e)
    return [x / z for x in e]


def test_cd_sample_paper_example():
    g = _load("cd_sample_of_that.json")
    p = _softmax_py(g["logits"], g["temperature"])
    cdf = list(itertools.accumulate(p))
    for tok, (a, b) in g["expect"]["cdf_intervals"].items():      # the hand-worked intervals
        t = int(tok)
        assert abs(cdf[t - 1] - a) < 1e-5 and abs(cdf[t] - b) < 1e-5
    draws = oracle.cd_sample.draw(np.array(g["logits"]), g["temperature"], g["uniforms"])
    assert draws == g["expect"]["draws"]
    toks, counts = oracle.cd_sample.group(draws)
    assert toks == g["expect"]["tokens"] and counts == g["expect"]["counts"]
    assert [g["vocab_words"][t] for t in toks] == ["of", "that"]
    # the branch: the parent's open step is sealed, one open child per distinct token
    bm = oracle.BlockManager(16, g["block_size"], 8)
    root, _, _ = bm.extend(-1, g["prefix"], True)
    parent, _, _ = bm.extend(root, g["open_step"], False)
    kids = bm.fork(parent, toks)
    assert kids == g["expect_fork"]["children"]
    assert [bm.table(k) for k in kids] == g["expect_fork"]["child_tables"]
    assert bm.snapshot()["seqs"][parent][1] == g["expect_fork"]["parent_sealed"]


def test_cd_sample_matches_the_distribution():
    # 40,000 independent draws from a 60-token distribution against its probabilities (chi-square)
    from scipy.stats import chi2
    rng = np.random.default_rng(7)
    logits = (rng.standard_normal(60) * 1.5).tolist()
    logits[5] = -math.inf                                          # a masked token is never drawn
    p = np.array(_softmax_py(logits, 0.8))
    u = rng.random(40000)
    draws = oracle.cd_sample.draw(np.array(logits), 0.8, u)
    counts = np.bincount(draws, minlength=60)
    assert counts[5] == 0
    keep = p * len(u) >= 5
    stat = float((((counts - p * len(u)) ** 2) / np.where(keep, p * len(u), 1))[keep].sum())
    assert chi2.sf(stat, int(keep.sum()) - 1) > 1e-4
    toks, cnt = oracle.cd_sample.group(draws)
    assert sum(cnt) == len(u) and toks == sorted(set(draws))


def test_cd_sample_closed_forms():
    V = 37
    u = (np.arange(200) + 0.5) / 200                               # no uniform on a boundary j / V
    assert oracle.cd_sample.draw(np.zeros(V), 1.3, u) == [int(x * V) for x in u]   # equal logits: floor(u V)
    logits = np.random.default_rng(3).standard_normal(50)
    top = int(np.argmax(logits))
    assert set(oracle.cd_sample.draw(logits, 1e-3, u)) == {top}    # temperature -> 0: the argmax
    # scaling logits and temperature together changes nothing
    assert oracle.cd_sample.draw(logits, 0.7, u) == oracle.cd_sample.draw(2 * logits, 1.4, u)
    # rows take consecutive slices of the uniforms
    rows = oracle.cd_sample.cd_sample(np.stack([np.zeros(V), logits[:V]]), 1.0, [3, 2], u[:5])
    assert rows[0][2] == [int(x * V) for x in u[:3]] and len(rows[1][2]) == 2
