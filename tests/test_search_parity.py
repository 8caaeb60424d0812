"""The library's search controller (tkv_search_*) in lockstep with the oracle -- CPU only.

Every operation of random scripts -- valid and invalid -- runs on both; return values, error kinds and
the whole state (snapshot) must be equal after each.  The library also reproduces the paper's
early-pruning walk-through and the plain beam search's selections on its own.
"""
import json
import os

import numpy as np
import pytest

import paper_2609_39334_amd as tkv
from oracle import search as S
from _search_driver import beam_search, drive
from test_search_oracle import run_golden

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
KIND = {tkv.TKV_EINVAL: "EINVAL", tkv.TKV_ENOMEM: "ENOMEM", tkv.TKV_ENOSEQ: "ENOSEQ", tkv.TKV_ECAP: "ECAP"}


class _Pair:
    def __init__(self, k, max_nodes, thr, max_def):
        self.c = tkv.Search(k, max_nodes, thr, max_def)
        self.o = S.Search(k, max_nodes, thr, max_def)

    def call(self, name, *args):
        try:
            rc = ("ok", getattr(self.c, name)(*args))
        except tkv.TkvError as e:
            rc = ("err", KIND[e.code])
        try:
            ro = ("ok", getattr(self.o, name)(*args))
        except S.SearchError as e:
            ro = ("err", e.kind)
        if name == "node" and rc[0] == "ok" and rc[1][3] is not None:
            rc = ("ok", rc[1][:3] + (float(np.float32(rc[1][3])),))
        if name == "round" and rc[0] == "ok":
            rc = ("ok", tuple(rc[1]))
            ro = ("ok", tuple(ro[1]))
        assert rc == ro, (name, args, rc, ro)
        assert self.c.snapshot() == self.o.snapshot(), (name, args)
        return ro[1] if ro[0] == "ok" else None


def test_ep_paper_figure_on_the_library():
    with open(os.path.join(GOLDEN, "ep_figure.json")) as f:
        g = json.load(f)
    ctl = tkv.Search(g["k"], 64, g["token_threshold"], g["max_deferrals"])
    run_golden(ctl, g)


@pytest.mark.parametrize("seed", range(16))
def test_random_scripts_lockstep(seed):
    rng = np.random.default_rng(seed)
    k = int(rng.integers(1, 4))
    P = _Pair(k, int(rng.integers(20, 400)), int(rng.choice([0, 300, 2048])), int(rng.integers(0, 5)))
    P.call("expand", -1, int(rng.integers(1, 9)))
    for _ in range(400):
        n = len(P.o.cands)
        r = rng.random()
        if r < 0.25:
            gen = [c for c in range(n) if P.o.cands[c].state == S.GENERATING]
            node = int(rng.choice(gen)) if gen and rng.random() < 0.9 else int(rng.integers(-1, n + 1))
            P.call("complete", node, int(rng.integers(0, 500)) if rng.random() < 0.1 else int(rng.integers(1, 500)))
        elif r < 0.4:
            P.call("tick")
        elif r < 0.5:
            P.call("flush")
        elif r < 0.75:
            waiting = [c for c in range(n) if P.o.cands[c].flushed and not P.o.cands[c].scored]
            if not waiting:
                continue
            take = [int(c) for c in rng.permutation(waiting)[:int(rng.integers(1, len(waiting) + 1))]]
            scores = [1.0 if rng.random() < 0.15 else float(np.float32(rng.random())) for _ in take]
            if rng.random() < 0.05:
                scores[0] = 1.25                       # invalid: the whole call is refused
            if rng.random() < 0.05:
                take.append(take[0])                   # invalid: repeated
                scores.append(0.5)
            P.call("score", take, scores)
            P.call("pruned")
        elif r < 0.9:
            scored = [c for c in range(n) if P.o.cands[c].state in (S.VERIFIED, S.SELECTED)]
            node = int(rng.choice(scored)) if scored and rng.random() < 0.85 else int(rng.integers(-1, n + 1))
            P.call("expand", node, int(rng.integers(0, 5)))
            P.call("pruned")
        else:
            P.call("node", int(rng.integers(0, n))) if n else None
            P.call("round", int(rng.integers(0, 6)))


@pytest.mark.parametrize("n,m,depth,seed,p", [(4, 4, 4, 1, 0.0), (8, 4, 4, 2, 0.0), (8, 2, 3, 3, 0.0),
                                              (16, 4, 3, 5, 0.0), (8, 2, 4, 13, 0.5), (9, 3, 4, 15, 0.4)])
def test_library_search_matches_the_oracle_run(n, m, depth, seed, p):
    ctl = tkv.Search(n // m, 10 ** 5, 2048, 6)
    ref = S.Search(n // m, 10 ** 5, 2048, 6)
    path_c = drive(ctl, n, m, depth, seed, p_perfect=p)
    path_o = drive(ref, n, m, depth, seed, p_perfect=p)
    assert path_c == path_o and ctl.snapshot() == ref.snapshot()
    if p == 0.0:
        assert [sorted(path_c[c] for c in ctl.round(d)[1]) for d in range(depth)] == beam_search(n, m, depth, seed)


def test_search_abi_edges():
    import ctypes
    L = tkv.lib()
    I32 = ctypes.c_int32
    assert L.tkv_search_create(1, 8, 0, 6, None) == tkv.TKV_EINVAL
    h = ctypes.c_void_p()
    for bad in ((0, 8, 0, 6), (1, 0, 0, 6), (1, 8, -1, 6), (1, 8, 0, -1)):
        assert L.tkv_search_create(*bad, ctypes.byref(h)) == tkv.TKV_EINVAL and h.value is None
    s = tkv.Search(1, 8, 10 ** 6, 6)
    first = I32()
    assert L.tkv_search_expand(s.h, -1, 3, None) == tkv.TKV_EINVAL
    assert L.tkv_search_expand(s.h, -1, -1, ctypes.byref(first)) == tkv.TKV_EINVAL
    assert L.tkv_search_expand(s.h, -1, 9, ctypes.byref(first)) == tkv.TKV_ENOMEM   # more than max_nodes
    assert s.expand(-1, 3) == 0
    s.complete(0, 5)
    s.complete(1, 7)
    n = I32()
    out = (I32 * 1)()
    assert L.tkv_search_flush(s.h, out, 1, ctypes.byref(n)) == tkv.TKV_ECAP and n.value == 2
    assert s.snapshot()["queue"] == [0, 1]                                          # nothing taken
    assert s.flush() == [0, 1]
    s.score([0, 1], [0.5, 0.25])
    assert L.tkv_search_pruned(s.h, out, 0, ctypes.byref(n)) == tkv.TKV_ECAP and n.value == 1
    assert s.pruned() == [1] and s.pruned() == []
    dec = I32()
    assert L.tkv_search_round(s.h, -1, out, 1, ctypes.byref(n), ctypes.byref(dec)) == tkv.TKV_EINVAL
    assert s.round(7) == (False, [])
    used = ctypes.c_size_t()
    assert L.tkv_search_snapshot(s.h, None, 0, ctypes.byref(used)) == tkv.TKV_ECAP and used.value > 0
    st, pa, de, sc = I32(), I32(), I32(), ctypes.c_float()
    assert L.tkv_search_node(s.h, 3, ctypes.byref(st), ctypes.byref(pa), ctypes.byref(de), ctypes.byref(sc)) \
        == tkv.TKV_EINVAL
    assert s.node(0) == (tkv.CAND_VERIFIED, -1, 0, 0.5) and s.node(2)[0] == tkv.CAND_GENERATING
