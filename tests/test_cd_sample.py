"""GPU: the CD branching sampler against the oracle.

A draw is an integer decided by floating point: the oracle takes it on the exact (float64) CDF, the
kernel on its fp32 sums.  Where a uniform lies farther than delta from every boundary of the exact
CDF the two must agree; within delta of a boundary any token in reach is a valid draw.  delta bounds
the kernel's rounding relative to the total: a cumulative weight passes through at most 16 additions
within a thread, 6 in the wave scan, 3 over the wave totals, a scaling and an addition per tile (n_tiles
= vocab / 4096 tiles, each scaled once), so at most (31 + 2 n_tiles) roundings of 2^-24 of the total;
each weight also carries the error of exp2 and of its rounded argument (below 1e-6 of the total for
these logits).  delta = 2 (31 + 2 n_tiles) 2^-24 + 1e-6 doubles the rounding part.  With 151,936 tokens
of a flat distribution many tokens' probability intervals are narrower than delta; there the check is
that every group is explained by draws in reach.  Group counts must sum to the potential.
"""
import math

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

def _delta(vocab):
    return 2 * (31 + 2 * math.ceil(vocab / 4096)) * 2.0 ** -24 + 1e-6


def _acceptable(logits, temperature, uniforms):
    """Per draw: the oracle's token and the set of tokens whose exact CDF interval lies within delta."""
    p = oracle.cd_sample.probabilities(logits, temperature)
    u = np.asarray(uniforms, dtype=np.float64)
    dl = _delta(len(logits))
    exact = oracle.cd_sample.draw(logits, temperature, u)
    lo = oracle.cd_sample.draw(logits, temperature, np.maximum(0.0, u - dl))
    hi = oracle.cd_sample.draw(logits, temperature, np.minimum(1.0 - 1e-12, u + dl))
    sets = [{j for j in range(a, b + 1) if p[j] > 0} for a, b in zip(lo, hi)]
    return exact, sets


def _run(logits, temperature, potential, seed):
    import paper_2609_39334_amd as tkv
    rng = np.random.default_rng(seed)
    off = np.concatenate([[0], np.cumsum(potential)]).astype(np.int32)
    u = rng.random(int(off[-1]), dtype=np.float32)
    tok, cnt, ng = tkv.tkv_cd_sample(torch.from_numpy(np.ascontiguousarray(logits, dtype=np.float32)).cuda(),
                                     temperature, torch.from_numpy(off).cuda(),
                                     torch.from_numpy(u).cuda(), int(max(potential) if len(potential) else 0))
    torch.cuda.synchronize()
    return off, u, tok.cpu().numpy(), cnt.cpu().numpy(), ng.cpu().numpy()


def _check_rows(logits, temperature, potential, off, u, tok, cnt, ng):
    n_amb = 0
    for r, n in enumerate(potential):
        lg = logits[r].astype(np.float64)
        if n == 0:
            assert ng[r] == 0
            continue
        k = int(ng[r])
        got = dict(zip(tok[off[r]:off[r] + k].tolist(), cnt[off[r]:off[r] + k].tolist()))
        assert list(got) == sorted(got) and sum(got.values()) == n and all(c > 0 for c in got.values())
        # draws computed in fp32 on the GPU come from the float32 logits
        exact, sets = _acceptable(lg, temperature, u[off[r]:off[r] + n].astype(np.float64))
        amb = [i for i, s in enumerate(sets) if len(s) > 1]
        n_amb += len(amb)
        want = {}
        for i, t in enumerate(exact):
            if i not in amb:
                want[t] = want.get(t, 0) + 1
        for t, c in got.items():                      # every group is explained by the draws
            extra = c - want.get(t, 0)
            assert extra >= 0, (r, t, c, want.get(t))
            assert extra <= sum(1 for i in amb if t in sets[i]), (r, t)
        assert sum(c - want.get(t, 0) for t, c in got.items()) == len(amb)
        for t, c in want.items():
            assert got.get(t, 0) >= c
    return n_amb


@pytest.mark.parametrize("vocab,temperature,scale", [(32000, 0.8, 2.0), (151936, 0.8, 3.0), (151936, 0.8, 9.0),
                                                     (1000, 1.0, 5.0), (37, 0.3, 1.0), (4099, 1.7, 0.5)])
def test_cd_sample_matches_oracle(vocab, temperature, scale):
    rng = np.random.default_rng(vocab)
    n_rows = 24
    logits = (rng.standard_normal((n_rows, vocab)) * scale).astype(np.float32)
    logits[rng.random((n_rows, vocab)) < 0.05] = -np.inf               # masked tokens are never drawn
    potential = rng.integers(0, 65, size=n_rows)
    potential[0], potential[1], potential[2] = 1, 1024, 0
    off, u, tok, cnt, ng = _run(logits, temperature, potential, vocab + 1)
    n_amb = _check_rows(logits, temperature, potential, off, u, tok, cnt, ng)
    print(f"    vocab {vocab}: {int(off[-1])} draws, {n_amb} within {_delta(vocab):.1e} of a boundary", flush=True)
    for r in range(n_rows):
        toks = tok[off[r]:off[r] + max(0, ng[r])]
        assert all(np.isfinite(logits[r, t]) for t in toks)


def test_cd_sample_distribution():
    # 100 rows of the same 50-token distribution, 1024 draws each: chi-square against the probabilities
    from scipy.stats import chi2
    rng = np.random.default_rng(5)
    base = (rng.standard_normal(50) * 1.5).astype(np.float32)
    logits = np.tile(base, (100, 1))
    potential = np.full(100, 1024)
    off, u, tok, cnt, ng = _run(logits, 0.8, potential, 6)
    counts = np.zeros(50)
    for r in range(100):
        np.add.at(counts, tok[off[r]:off[r] + ng[r]], cnt[off[r]:off[r] + ng[r]])
    p = oracle.cd_sample.probabilities(base.astype(np.float64), 0.8)
    n = counts.sum()
    keep = p * n >= 5
    stat = float((((counts - p * n) ** 2) / np.where(keep, p * n, 1))[keep].sum())
    assert n == 102400 and chi2.sf(stat, int(keep.sum()) - 1) > 1e-4


def test_cd_sample_edge_rows():
    logits = np.full((4, 300), -np.inf, dtype=np.float32)
    logits[1, 123] = 0.0                                                # one finite token
    logits[2, :] = 0.0                                                  # uniform: floor(u * 300)
    logits[3, 299] = 5.0
    potential = np.array([3, 5, 200, 2])
    off, u, tok, cnt, ng = _run(logits, 1.0, potential, 9)
    assert ng[0] == -1                                                  # no finite logit
    assert ng[1] == 1 and tok[off[1]] == 123 and cnt[off[1]] == 5
    assert ng[3] == 1 and tok[off[3]] == 299 and cnt[off[3]] == 2
    uu = u[off[2]:off[3]].astype(np.float64)
    want = np.bincount(np.minimum((uu * 300).astype(int), 299), minlength=300)
    got = np.zeros(300, dtype=int)
    got[tok[off[2]:off[2] + ng[2]]] = cnt[off[2]:off[2] + ng[2]]
    near = np.abs(uu * 300 - np.round(uu * 300)) < _delta(300) * 300
    assert np.abs(got - want).sum() <= 2 * near.sum()


def test_cd_branch_step_end_to_end():
    # one CD step for a coalesced batch: the sampler's groups fork the rows' sequences on the library's
    # block manager and on the oracle's; children's tables agree and their potentials sum to the row's
    import paper_2609_39334_amd as tkv
    rng = np.random.default_rng(11)
    bm_c, bm_o = tkv.BlockManager(400, 16, 128), oracle.BlockManager(400, 16, 128)
    rows = []
    for bm in (bm_c, bm_o):
        r0, _, _ = bm.extend(-1, list(range(40)), True)
        rows.append([bm.extend(r0, [100 + i, 7, 7], False)[0] for i in range(6)])
    assert rows[0] == rows[1]
    potential = np.array([4, 1, 8, 3, 16, 2])
    logits = (rng.standard_normal((6, 64)) * 1.2).astype(np.float32)
    off, u, tok, cnt, ng = _run(logits, 0.8, potential, 12)
    for r, s in enumerate(rows[0]):
        toks = tok[off[r]:off[r] + ng[r]].tolist()
        pots = cnt[off[r]:off[r] + ng[r]].tolist()
        assert sum(pots) == potential[r]
        if len(toks) == 1:
            bm_c.append(s, toks)
            bm_o.append(s, toks)
            continue
        kc, ko = bm_c.fork(s, toks), bm_o.fork(s, toks)
        assert kc == ko
        for k, t in zip(kc, toks):
            assert list(bm_c.table(k)) == bm_o.table(k) and bm_o.table(k)[:-1] == bm_o.table(s)
    assert bm_c.snapshot()["seqs"] == bm_o.snapshot()["seqs"]


@pytest.mark.parametrize("vocab", [4096 * 512, 4096 * 512 - 1])
def test_cd_sample_largest_vocabulary(vocab):
    # 512 tiles of 4,096 logits, the most a row may have; the odd size takes the unaligned path
    rng = np.random.default_rng(vocab % 1000)
    logits = (rng.standard_normal((3, vocab)) * 2.0).astype(np.float32)
    logits[1, rng.random(vocab) < 0.5] = -np.inf
    potential = np.array([1, 1024, 8])
    off, u, tok, cnt, ng = _run(logits, 0.8, potential, vocab)
    n_amb = _check_rows(logits, 0.8, potential, off, u, tok, cnt, ng)
    print(f"    vocab {vocab}: {int(off[-1])} draws, {n_amb} within {_delta(vocab):.1e} of a boundary", flush=True)


def test_cd_sample_rejects_bad_arguments():
    import paper_2609_39334_amd as tkv
    off = torch.tensor([0, 1], dtype=torch.int32, device="cuda")
    u = torch.full((1,), 0.5, dtype=torch.float32, device="cuda")
    too_wide = torch.zeros((1, 4096 * 512 + 1), dtype=torch.float32, device="cuda")
    with pytest.raises(tkv.TkvError) as e:
        tkv.tkv_cd_sample(too_wide, 0.8, off, u, 1)
    assert e.value.code == tkv.TKV_EINVAL
    ok = torch.zeros((1, 10), dtype=torch.float32, device="cuda")
    for temp, mp in ((0.0, 1), (float("inf"), 1), (float("nan"), 1), (0.8, 1025), (0.8, -1)):
        with pytest.raises(tkv.TkvError):
            tkv.tkv_cd_sample(ok, temp, off, u, mp)
    empty = torch.zeros((0, 10), dtype=torch.float32, device="cuda")
    tok, cnt, ng = tkv.tkv_cd_sample(empty, 0.8, torch.zeros(1, dtype=torch.int32, device="cuda"), u, 0)
    assert ng.numel() == 0


def test_cd_sample_refuses_rows_outside_the_arrays():
    # draw offsets are device data: a row whose range leaves the 6-entry arrays (row 1) or runs
    # backwards (row 2) is refused (-1) and touches nothing; rows 0 and 3 are sampled as usual
    import paper_2609_39334_amd as tkv
    logits = torch.zeros((4, 100), dtype=torch.float32, device="cuda")
    off = torch.tensor([0, 2, 9, 4, 6], dtype=torch.int32, device="cuda")
    u = torch.tensor([0.015, 0.5, 0.25, 0.75, 0.125, 0.995], dtype=torch.float32, device="cuda")
    tok, cnt, ng = tkv.tkv_cd_sample(logits, 1.0, off, u, 8)
    torch.cuda.synchronize()
    ng = ng.cpu().tolist()
    assert ng[1] == -1 and ng[2] == -1
    assert ng[0] == 2 and tok[0:2].cpu().tolist() == [1, 50] and cnt[0:2].cpu().tolist() == [1, 1]
    assert ng[3] == 2 and tok[4:6].cpu().tolist() == [12, 99] and cnt[4:6].cpu().tolist() == [1, 1]
