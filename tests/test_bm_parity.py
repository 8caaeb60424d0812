"""C++ block manager and row coalescing vs the oracle, bit-exact, on CPU.

Every operation's outputs (sequence id, block ids, hit flags, freed ids) must match, the block
arrays (refcount, block_len, indexed) after every operation, the touched sequence's table after
every operation, and every live table plus the coalesced rows at each launch.
"""
import json
import os

import numpy as np
import pytest

import oracle
import paper_2609_39334_amd as tkv
import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _arrays_equal(a, b):
    for k in ("refcount", "block_len", "indexed"):
        np.testing.assert_array_equal(np.asarray(a[k]), np.asarray(b[k]), err_msg=k)


class _Pair:
    """Runs every operation on both block managers and compares."""

    def __init__(self, num_blocks, block_size, max_seqs):
        self.o = oracle.BlockManager(num_blocks, block_size, max_seqs)
        self.c = tkv.BlockManager(num_blocks, block_size, max_seqs)
        self.ops = 0

    def _cmp_arrays(self, touched):
        """Block arrays at the blocks the operation touched; all blocks every 64 operations."""
        sc = self.c.snapshot(seqs=False)
        idx = list(touched) if self.ops % 64 else range(self.o.num_blocks)
        for b in idx:
            assert (self.o.refcount[b], self.o.block_len[b], int(self.o.key[b] is not None)) == \
                (sc["refcount"][b], sc["block_len"][b], sc["indexed"][b]), b

    def extend(self, parent, tokens, seal):
        err_o = err_c = None
        try:
            ro = self.o.extend(parent, tokens, seal)
        except oracle.BMError as e:
            err_o = e.code
        try:
            rc = self.c.extend(parent, tokens, seal)
        except tkv.TkvError as e:
            err_c = e.code
        assert err_o == err_c
        if err_o is not None:
            raise oracle.BMError(err_o, "both failed")
        assert ro[0] == rc[0]
        assert list(ro[1]) == [int(x) for x in rc[1]]
        assert list(ro[2]) == [int(x) for x in rc[2]]
        table = self.o.table(ro[0])
        assert tuple(table) == tuple(int(x) for x in self.c.table(rc[0]))
        self._cmp_arrays(table)
        self.ops += 1
        return ro

    def prune(self, seq):
        table = self.o.table(seq)
        fo = self.o.prune(seq)
        fc = self.c.prune(seq)
        assert list(fo) == [int(x) for x in fc]
        self._cmp_arrays(table)
        self.ops += 1
        return fo

    def append(self, seq, tokens):
        err_o = err_c = None
        try:
            do = self.o.append(seq, tokens)
        except oracle.BMError as e:
            err_o = e.code
        try:
            dc = self.c.append(seq, tokens)
        except tkv.TkvError as e:
            err_c = e.code
        assert err_o == err_c
        if err_o is not None:
            raise oracle.BMError(err_o, "both failed")
        assert list(do) == [int(x) for x in dc]
        table = self.o.table(seq)
        assert tuple(table) == tuple(int(x) for x in self.c.table(seq))
        self._cmp_arrays(table)
        self.ops += 1
        return do

    def seal(self, seq):
        err_o = err_c = None
        try:
            ro = self.o.seal(seq)
        except oracle.BMError as e:
            err_o = e.code
        try:
            rc = self.c.seal(seq)
        except tkv.TkvError as e:
            err_c = e.code
        assert err_o == err_c
        if err_o is not None:
            raise oracle.BMError(err_o, "both failed")
        assert ro == rc
        table = self.o.table(seq)
        assert tuple(table) == tuple(int(x) for x in self.c.table(seq))
        self._cmp_arrays(list(table) + [own for own, _ in ro])
        self.ops += 1
        return ro

    def fork(self, seq, tokens):
        err_o = err_c = None
        try:
            ko = self.o.fork(seq, tokens)
        except oracle.BMError as e:
            err_o = e.code
        try:
            kc = self.c.fork(seq, tokens)
        except tkv.TkvError as e:
            err_c = e.code
        assert err_o == err_c
        if err_o is not None:
            raise oracle.BMError(err_o, "both failed")
        assert ko == kc
        touched = list(self.o.table(seq))
        for k in ko:
            assert tuple(self.o.table(k)) == tuple(int(x) for x in self.c.table(k))
            touched += self.o.table(k)
        self._cmp_arrays(touched)
        self.ops += 1
        return ko

    def full_compare(self):
        so, sc = self.o.snapshot(), self.c.snapshot()
        _arrays_equal(so, sc)
        assert so["seqs"] == sc["seqs"]


def _tokens(spec):
    if isinstance(spec, dict):
        a, b = spec["range"]
        return list(range(a, b))
    return list(spec)


@pytest.mark.parametrize("case", json.load(open(os.path.join(GOLD, "bm_cases.json")))["cases"],
                         ids=lambda c: c["name"])
def test_golden_cases_lockstep(case):
    p = _Pair(case["num_blocks"], case["block_size"], case["max_seqs"])
    for op in case["ops"]:
        try:
            if op["op"] == "extend":
                p.extend(op["parent"], _tokens(op["tokens"]), bool(op["seal"]))
            elif op["op"] == "append":
                p.append(op["seq"], _tokens(op["tokens"]))
            elif op["op"] == "seal":
                p.seal(op["seq"])
            else:
                try:
                    p.prune(op["seq"])
                except oracle.BMError:
                    with pytest.raises(tkv.TkvError):
                        p.c.prune(op["seq"])
                    continue
        except oracle.BMError:
            pass
        p.full_compare()


@pytest.mark.parametrize("seed", range(10))
def test_random_scripts_lockstep(seed):
    rng = np.random.default_rng(1000 + seed)
    p = _Pair(48, 4, 20)
    live, sealed = [], set()
    for _ in range(200):
        if live and rng.random() < 0.3:
            s = live.pop(int(rng.integers(0, len(live))))
            p.prune(s)
            sealed.discard(s)
            continue
        cands = [s for s in live if s in sealed]
        if cands and rng.random() < 0.05:     # extending an unsealed sequence fails on both sides
            uns = [s for s in live if s not in sealed]
            if uns:
                with pytest.raises(oracle.BMError):
                    p.extend(uns[0], [1, 2, 3], True)
                continue
        parent = -1 if not cands or rng.random() < 0.2 else cands[int(rng.integers(0, len(cands)))]
        vocab = 3 if rng.random() < 0.5 else 40
        toks = rng.integers(0, vocab, size=int(rng.integers(1 if parent == -1 else 0, 14))).tolist()
        seal = bool(rng.random() < 0.7)
        try:
            s, _, _ = p.extend(parent, toks, seal)
        except oracle.BMError:
            continue
        live.append(s)
        if seal:
            sealed.add(s)
        if p.ops % 25 == 0:
            p.full_compare()
    p.full_compare()


@pytest.mark.parametrize("seed", range(10))
def test_decode_loop_scripts_lockstep(seed):
    # extensions, token-by-token appends (decode steps), seals and prunes in random order, with small
    # vocabularies so that sealed steps often find identical blocks
    rng = np.random.default_rng(2000 + seed)
    p = _Pair(64, 4, 16)
    live, open_ = [], set()
    for _ in range(300):
        r = rng.random()
        vocab = 2 if rng.random() < 0.6 else 40
        try:
            if live and r < 0.15:
                s = live.pop(int(rng.integers(0, len(live))))
                p.prune(s)
                open_.discard(s)
            elif live and r < 0.55:
                s = live[int(rng.integers(0, len(live)))]
                p.append(s, rng.integers(0, vocab, size=int(rng.integers(0, 7))).tolist())
                open_.add(s)
            elif live and r < 0.7:
                s = live[int(rng.integers(0, len(live)))]
                if s in open_:
                    p.seal(s)
                    open_.discard(s)
                else:
                    with pytest.raises(oracle.BMError):          # sealing a sealed sequence fails on both
                        p.seal(s)
            elif live and r < 0.78:                              # on-demand branching into 2-4 children
                s = live[int(rng.integers(0, len(live)))]
                kids = p.fork(s, rng.integers(0, vocab, size=int(rng.integers(2, 5))).tolist())
                open_.discard(s)
                live += kids
                open_.update(kids)
            else:
                cands = [s for s in live if s not in open_]
                parent = -1 if not cands or rng.random() < 0.2 else cands[int(rng.integers(0, len(cands)))]
                toks = rng.integers(0, vocab, size=int(rng.integers(1 if parent == -1 else 0, 9))).tolist()
                seal = bool(rng.random() < 0.5)
                s, _, _ = p.extend(parent, toks, seal)
                live.append(s)
                if not seal:
                    open_.add(s)
        except oracle.BMError:
            continue
        if p.ops % 25 == 0:
            p.full_compare()
    p.full_compare()


def test_extend_slots_skip_hit_blocks():
    # the pool slots of a sealed step's tokens: consecutive within each block, none for a hit block
    p = _Pair(20, 4, 8)
    root, _, _ = p.extend(-1, [1, 2, 3, 4, 5], True)
    a, blk, hit = p.extend(root, [7, 8, 9, 10, 11, 12], True)
    b, blk2, hit2 = p.extend(root, [7, 8, 9, 10, 13], True)      # first block a hit, second a miss
    assert list(hit2) == [1, 0]
    dst = tkv.tkv_extend_slots(blk2, hit2, 5, 4)
    assert dst.tolist() == [-1, -1, -1, -1, blk2[1] * 4]
    assert tkv.tkv_extend_slots(blk, hit, 6, 4).tolist() == [blk[0] * 4 + i for i in range(4)] + [blk[1] * 4, blk[1] * 4 + 1]
    with pytest.raises(tkv.TkvError):
        tkv.tkv_extend_slots(blk, hit, 9, 4)                       # 9 tokens need 3 blocks


@pytest.mark.parametrize("name", list(W.CONFIGS))
def test_workload_scripts_lockstep(name):
    wl = W.CONFIGS[name](0)
    p = _Pair(wl.num_blocks, wl.shape.block_size, wl.max_seqs)
    seq_of = []
    launches = 0
    for e in wl.events:
        if isinstance(e, W.Extend):
            parent = -1 if e.parent < 0 else seq_of[e.parent]
            seq_of.append(p.extend(parent, e.tokens, e.seal)[0])
        elif isinstance(e, W.Prune):
            p.prune(seq_of[e.handle])
        else:
            p.full_compare()
            seqs = [seq_of[h] for h, _ in e.cands]
            qls = [q for _, q in e.cands]
            ro, fo, mo = oracle.coalesce([p.o.table(s) for s in seqs], qls)
            rc, fc, mc = p.c.coalesce(seqs, qls)
            assert ro == rc.tolist() and fo == fc.tolist() and mo == mc.tolist()
            launches += 1
    assert launches == len(wl.launches)
    p.full_compare()


def test_spec_explosion_dedups_identical_siblings():
    # identical sibling steps must share blocks; the leaf level's copies coalesce into one row
    wl = W.spec_explosion(0)
    bm = tkv.BlockManager(wl.num_blocks, 16, wl.max_seqs)
    got = {}
    W.drive(wl, bm, on_launch=lambda i, l, c: got.setdefault("c", c))
    seqs = [s for s, _ in got["c"]]
    row_of, first, mult = bm.coalesce(seqs, [1] * len(seqs))
    assert len(seqs) == 2048 and len(first) < len(seqs)
    assert int(mult.sum()) == 2048 and mult.max() >= 2
    tables = [tuple(bm.table(s)) for s in seqs]
    for c, r in enumerate(row_of):
        assert tables[c] == tables[first[r]]
