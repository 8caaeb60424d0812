"""Pins of the oracle search controller (early pruning, lazy verification) -- CPU only.

* The paper's early-pruning walk-through (tests/golden/ep_figure.json, worked by hand).
* Rule 1 never changes the selection: under any completion and arrival order, a speculative search
  with rank pruning selects at every step exactly what a plain beam search selects (the paper's claim
  for this rule), the plain beam search being written out independently in tests/_search_driver.py.
* Rule 2: with perfect scores about, each round's selection is the first k perfect members in score
  arrival order when there are k of them, else the plain top k -- computed per round from the final
  record of scores, not incrementally.
* Lazy verification: each policy alone, at its boundary (tokens exceeding the threshold, the last
  sibling completing, the deferral limit), and the degenerate settings (threshold 0, limit 0).
* Invariants after every event of random searches.
* Rule 1 is safe against every future: on tiny searches, each candidate it prunes stays out of its
  step's plain-beam-search selection for every assignment of the scores not yet known.
"""
import json
import os

import numpy as np
import pytest

from oracle import search as S
from _search_driver import beam_search, drive, path_score

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def run_golden(ctl, g):
    for ev in g["events"]:
        op = ev["op"]
        if op == "expand":
            assert ctl.expand(ev["parent"], ev["n"]) == ev["expect_first"]
        elif op == "complete":
            assert ctl.complete(ev["node"], ev["tokens"]) == ev["expect_flush"]
        elif op == "flush":
            assert ctl.flush() == ev["expect"]
        elif op == "score":
            ctl.score(ev["nodes"], ev["scores"])
            assert ctl.pruned() == ev["expect_pruned"], ev
        elif op == "round":
            dec, sel = ctl.round(ev["depth"])
            assert [dec, sel] == ev["expect"]


def test_ep_paper_figure():
    with open(os.path.join(GOLDEN, "ep_figure.json")) as f:
        g = json.load(f)
    ctl = S.Search(g["k"], 64, g["token_threshold"], g["max_deferrals"])
    run_golden(ctl, g)
    names = g["names"]
    assert [names[c] for c in ctl.round(0)[1]] == ["C"]
    assert ctl.node(3)[0] == S.PRUNED and ctl.node(2)[0] == S.SELECTED


def test_lv_token_threshold():
    ctl = S.Search(k=2, max_nodes=64, token_threshold=2048, max_deferrals=100)
    ctl.expand(-1, 4)
    assert not ctl.complete(0, 800)
    assert not ctl.complete(1, 1248)              # 2,048 queued: reaches, does not exceed
    assert ctl.complete(2, 1)                     # 2,049 exceeds
    assert ctl.flush() == [0, 1, 2] and ctl.queue == []


def test_lv_sibling_group():
    ctl = S.Search(k=1, max_nodes=64, token_threshold=10 ** 6, max_deferrals=100)
    ctl.expand(-1, 3)
    assert not ctl.complete(0, 10)
    assert not ctl.complete(1, 10)
    assert ctl.complete(2, 10)                    # the last sibling completes: the group is due
    assert ctl.flush() == [0, 1, 2]
    ctl.score([0, 1, 2], [0.9, 0.5, 0.2])         # k = 1: round 0 settles with candidate 0
    assert ctl.pruned() == [1, 2] and ctl.round(0) == (True, [0])
    f = ctl.expand(0, 3)
    assert not ctl.complete(f, 5) and not ctl.tick()
    assert not ctl.complete(f + 1, 5)
    assert ctl.complete(f + 2, 5)                 # every sibling complete
    assert ctl.flush() == [f, f + 1, f + 2]
    # a group with a pruned member: the pruned one does not hold it back
    ctl.score([f, f + 1, f + 2], [0.3, 0.6, 0.1])
    assert ctl.pruned() == [f, f + 2]             # rule 1 (k = 1) then the round settles on f + 1


def test_lv_deferral_limit():
    ctl = S.Search(k=1, max_nodes=64, token_threshold=10 ** 6, max_deferrals=6)
    ctl.expand(-1, 2)
    assert not ctl.tick()                         # empty queue: nothing to flush, nothing deferred
    assert not ctl.complete(0, 10)
    for i in range(6):
        assert not ctl.tick()                     # deferred 1..6 times
        assert ctl.cands[0].deferrals == i + 1
    assert ctl.tick()                             # a 7th deferral would exceed the limit
    assert ctl.cands[0].deferrals == 6


def test_lv_degenerate_settings():
    ctl = S.Search(k=1, max_nodes=64, token_threshold=0, max_deferrals=100)
    ctl.expand(-1, 3)
    assert ctl.complete(0, 1)                     # threshold 0: every completion is due
    ctl2 = S.Search(k=1, max_nodes=64, token_threshold=10 ** 6, max_deferrals=0)
    ctl2.expand(-1, 3)
    assert ctl2.complete(0, 1)                    # limit 0: never deferred, due at once
    assert ctl2.tick() and ctl2.cands[0].deferrals == 0


@pytest.mark.parametrize("n,m,depth,seed", [(4, 4, 4, 1), (8, 4, 4, 2), (8, 2, 3, 3), (6, 3, 4, 4), (16, 4, 3, 5),
                                            (4, 1, 4, 6), (12, 4, 4, 7), (8, 8, 5, 8)])
def test_rule1_keeps_the_beam_search_selection(n, m, depth, seed):
    ctl = S.Search(n // m, 10 ** 5, 2048, 6)
    path = drive(ctl, n, m, depth, seed)
    got = [sorted(path[c] for c in ctl.round(d)[1]) for d in range(depth)]
    assert got == beam_search(n, m, depth, seed)
    assert any(c.state == S.PRUNED and c.arrival is not None and c.depth < depth - 1 for c in ctl.cands) \
        or n // m == n                             # some candidate pruned once it had a score


def _replay_round(ctl, members):
    """The round's selection from the final record: first k perfect by arrival, else the top k."""
    scored = sorted((c for c in members if ctl.cands[c].arrival is not None), key=lambda c: ctl.cands[c].arrival)
    perfect = [c for c in scored if ctl.cands[c].score == 1.0]
    if len(perfect) >= ctl.k:
        return sorted(perfect[:ctl.k])
    return sorted(sorted(scored, key=lambda c: (-ctl.cands[c].score, ctl.cands[c].arrival))[:ctl.k])


@pytest.mark.parametrize("n,m,depth,seed,p", [(4, 4, 4, 11, 0.3), (8, 4, 4, 12, 0.3), (8, 2, 4, 13, 0.5),
                                              (16, 4, 3, 14, 0.2), (9, 3, 4, 15, 0.4)])
def test_rule2_first_k_perfect(n, m, depth, seed, p):
    ctl = S.Search(n // m, 10 ** 5, 2048, 6)
    drive(ctl, n, m, depth, seed, p_perfect=p)
    n_perfect_rounds = 0
    for d in range(depth):
        members = ctl.roots if d == 0 else [c for par in ctl.round(d - 1)[1] for c in ctl.cands[par].children]
        want = _replay_round(ctl, members)
        assert ctl.round(d) == (True, want), d
        n_perfect_rounds += all(ctl.cands[c].score == 1.0 for c in want)
    assert n_perfect_rounds > 0


def check_invariants(ctl):
    for c, cand in enumerate(ctl.cands):
        assert (cand.state == S.QUEUED) == (c in ctl.queue)
        if cand.state == S.PRUNED:
            assert all(ctl.cands[x].state == S.PRUNED for x in cand.children or [])
        if cand.state == S.SELECTED:
            assert c in ctl.selection[cand.depth]
            assert cand.depth == 0 or ctl.cands[cand.parent].state == S.SELECTED
    for d, sel in ctl.selection.items():
        assert len(sel) <= ctl.k
        members = ctl.roots if d == 0 else [x for p in ctl.selection[d - 1] for x in ctl.cands[p].children or []]
        assert set(sel) <= set(members)
    # rule 1 is at its fixed point in every open round whose members are known
    for d in {cand.depth for cand in ctl.cands} - set(ctl.selection):
        known = ctl._members(d)
        if known is None:
            continue
        live = [c for c in known[0] if ctl.cands[c].state in (S.VERIFIED, S.SELECTED)]
        for c in live:
            assert sum(ctl.cands[o].score > ctl.cands[c].score for o in live) < ctl.k


@pytest.mark.parametrize("seed,p", [(21, 0.0), (22, 0.25), (23, 0.0), (24, 0.5)])
def test_invariants_hold_after_every_event(seed, p):
    n, m = (8, 2) if seed % 2 else (6, 3)
    ctl = S.Search(n // m, 10 ** 5, 600, 3)
    drive(ctl, n, m, 4, seed, p_perfect=p, on_event=check_invariants)
    check_invariants(ctl)


def test_errors():
    ctl = S.Search(k=1, max_nodes=6, token_threshold=0, max_deferrals=6)
    with pytest.raises(S.SearchError) as e:
        ctl.expand(0, 2)
    assert e.value.kind == "EINVAL"                # no candidate 0 yet
    ctl.expand(-1, 3)
    for bad, kind in (((-1, 1), "EINVAL"), ((0, 1), "EINVAL")):   # roots exist; no score yet
        with pytest.raises(S.SearchError) as e:
            ctl.expand(*bad)
        assert e.value.kind == kind
    with pytest.raises(S.SearchError) as e:
        ctl.complete(0, 0)
    assert e.value.kind == "EINVAL"
    ctl.complete(0, 5)
    with pytest.raises(S.SearchError) as e:
        ctl.complete(0, 5)                          # already completed
    assert e.value.kind == "EINVAL"
    with pytest.raises(S.SearchError) as e:
        ctl.score([0], [0.5])                       # queued, not flushed
    assert e.value.kind == "EINVAL"
    assert ctl.flush() == [0]
    for nodes, scores in (([0, 0], [0.1, 0.2]), ([0], [1.5]), ([0], [float("nan")])):
        with pytest.raises(S.SearchError):
            ctl.score(nodes, scores)
    ctl.score([0], [0.5])
    with pytest.raises(S.SearchError) as e:
        ctl.expand(0, 4)                            # 3 + 4 > 6 candidates
    assert e.value.kind == "ENOMEM"
    ctl.expand(0, 3)
    with pytest.raises(S.SearchError) as e:
        ctl.expand(0, 1)                            # already expanded
    assert e.value.kind == "EINVAL"
    ctl.complete(1, 5)
    ctl.score(ctl.flush(), [0.9])                   # 0 now ranks below 1: pruned with its children
    assert ctl.pruned() == [0, 3, 4, 5]
    with pytest.raises(S.SearchError) as e:
        ctl.complete(3, 5)
    assert e.value.kind == "ENOSEQ"


def test_score_of_a_candidate_pruned_in_flight_is_ignored():
    ctl = S.Search(k=1, max_nodes=64, token_threshold=10 ** 6, max_deferrals=100)
    ctl.expand(-1, 3)
    ctl.complete(0, 5)
    ctl.complete(1, 5)
    batch = ctl.flush()
    ctl.complete(2, 5)
    ctl.score(ctl.flush(), [1.0])                   # candidate 2 is perfect: round 0 settles on it
    assert ctl.pruned() == [0, 1]
    ctl.score(batch, [0.4, 1.0])                    # their scores come back afterwards: ignored
    assert ctl.cands[1].arrival is None and ctl.round(0) == (True, [2])
    assert path_score(1, (0,)) == path_score(1, (0,))


def _plain_selection(n, m, scores_by_path, depth):
    """Plain beam search over a full assignment of path scores (distinct values): selected paths per step."""
    k = n // m
    frontier = [(i,) for i in range(n)]
    out = []
    for _ in range(depth):
        keep = sorted(frontier, key=lambda p: -scores_by_path[p])[:k]
        out.append(set(keep))
        frontier = [p + (j,) for p in keep for j in range(m)]
    return out


@pytest.mark.parametrize("seed", range(12))
def test_rule1_prunes_only_candidates_no_future_can_select(seed):
    # tiny speculative searches (beam size 4, width 2, two steps): whenever rule 1 prunes a scored
    # candidate, every assignment of the scores not yet known (five distinct levels each) leaves it out of
    # its step's plain-beam-search selection
    import itertools
    rng = np.random.default_rng(seed)
    n, m, depth = 4, 2, 2
    paths = [(i,) for i in range(n)] + [(i, j) for i in range(n) for j in range(m)]
    known = {p: float(np.float32(rng.random() * 0.9 + 0.05)) for p in paths}
    levels = [0.011, 0.013, 0.017, 0.019, 0.023]          # fresh values: no ties with the known scores
    ctl = S.Search(n // m, 64, 0, 6)
    path_of = {}
    first = ctl.expand(-1, n)
    for i in range(n):
        path_of[first + i] = (i,)
    generating = list(range(first, first + n))
    checked = 0
    while generating:
        c = generating.pop(int(rng.integers(0, len(generating))))
        if ctl.cands[c].state != S.GENERATING:
            continue
        assert ctl.complete(c, 10)                          # threshold 0: verified at once
        ctl.score(ctl.flush(), [known[path_of[c]]])
        newly = ctl.pruned()
        for x in newly:
            cand = ctl.cands[x]
            if cand.arrival is None:
                continue                                    # pruned with its subtree, not by its own rank
            scored = {path_of[y]: ctl.cands[y].score for y in path_of if ctl.cands[y].arrival is not None}
            unknown = [p for p in paths if p not in scored]
            if len(unknown) > 6:
                continue
            for vals in itertools.product(*(levels for _ in unknown)):
                full = dict(scored)
                full.update({p: v + 1e-4 * i for i, (p, v) in enumerate(zip(unknown, vals))})
                assert path_of[x] not in _plain_selection(n, m, full, depth)[cand.depth]
            checked += 1
        if ctl.cands[c].state in (S.VERIFIED, S.SELECTED) and ctl.cands[c].depth < depth - 1:
            f = ctl.expand(c, m)
            for j in range(m):
                path_of[f + j] = path_of[c] + (j,)
                generating.append(f + j)
        generating = [g for g in generating if ctl.cands[g].state == S.GENERATING]
    assert checked > 0
