"""GPU: a speculative beam search end to end.  The library's controller (tkv_search_*) decides the
verification batches and the pruning; each batch runs as one tkv_verify call over the block
manager's tables (every candidate's step verified causally against its whole path, the prefill-only
pass of the verifier), and pruned candidates are released with tkv_prune.

The same block-manager operations run on the oracle's manager in lockstep (tables and final state
equal); sampled rows of every batch are compared with the oracle's attention to the attention
tolerance.  Scores are a fixed function of a candidate's path (there is no reward model here).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from _search_driver import beam_search, drive

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS, LSE_ABS = 1e-2, 1e-3, 2e-3
PRUNED = 5


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


@pytest.mark.parametrize("n,m,seed,p", [(8, 4, 31, 0.0), (8, 2, 32, 0.3), (12, 4, 33, 0.0)])
def test_speculative_search_drives_verify_and_prune(n, m, seed, p):
    import paper_2609_39334_amd as tkv
    hq, hkv, d, bs, nb, depth = 8, 2, 128, 16, 6000, 4
    rng = np.random.default_rng([seed, 1])
    kv = W.f32_to_bf16_bits(rng.standard_normal((2, nb, hkv, bs, d)).astype(np.float32))
    k_dev, v_dev = _dev(kv[0]), _dev(kv[1])
    k_ref, v_ref = W.bf16_bits_to_f32(kv[0]).astype(np.float64), W.bf16_bits_to_f32(kv[1]).astype(np.float64)
    bm_c, bm_o = tkv.BlockManager(nb, bs, 4096), oracle.BlockManager(nb, bs, 4096)
    prompt = rng.integers(0, 50, size=300).tolist()
    root = bm_c.extend(-1, prompt, True)[0]
    assert bm_o.extend(-1, prompt, True)[0] == root
    ctl = tkv.Search(n // m, 10 ** 5, 2048, 6)
    seq, steps = {}, {}
    counts = {"batches": 0, "rows": 0, "released": 0}

    def on_complete(c, n_tok):
        parent = ctl.node(c)[1]
        base = root if parent < 0 else seq[parent]
        toks = rng.integers(0, 50, size=n_tok).tolist()
        s = bm_c.extend(base, toks, True)[0]
        assert bm_o.extend(base, toks, True)[0] == s
        seq[c], steps[c] = s, n_tok

    def on_verify(batch):
        live = [c for c in batch if ctl.node(c)[0] != PRUNED]
        if not live:
            return
        seqs, qls = [seq[c] for c in live], [steps[c] for c in live]
        _, first, mult = bm_c.coalesce(seqs, qls)
        tables = [bm_c.table(seqs[f]) for f in first]
        assert [list(t) for t in tables] == [bm_o.table(seqs[f]) for f in first]
        ql = [qls[f] for f in first]
        qi = np.concatenate([[0], np.cumsum(ql)]).astype(np.int32)
        ki = np.concatenate([[0], np.cumsum([len(t) for t in tables])]).astype(np.int32)
        bl = bm_c.block_len()
        plan = tkv.Plan((hq, hkv, d, bs, nb), qi, ki, np.concatenate(tables).astype(np.int32), bl, mult)
        q = W.f32_to_bf16_bits(rng.standard_normal((int(qi[-1]), hq, d)).astype(np.float32))
        o = torch.full((int(qi[-1]), hq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((int(qi[-1]), hq), float("nan"), dtype=torch.float32, device="cuda")
        plan.verify(_dev(q), k_dev, v_dev, o, lse)
        torch.cuda.synchronize()
        rows = sorted(set(np.random.default_rng([seed, counts["batches"]]).integers(0, len(tables), 3).tolist()))
        o_ref, l_ref = oracle.attention(W.bf16_bits_to_f32(q).astype(np.float64), k_ref, v_ref,
                                        [list(t) for t in tables], bm_o.block_len, ql, rows=rows)
        sel = np.concatenate([np.arange(qi[r], qi[r + 1]) for r in rows])
        err = np.abs(o.float().cpu().numpy()[sel] - o_ref[sel])
        lerr = np.abs(lse.cpu().numpy()[sel] - l_ref[sel])
        assert np.isfinite(err).all() and err.max() <= MAX_ABS and err.mean() <= MEAN_ABS and lerr.max() <= LSE_ABS
        counts["batches"] += 1
        counts["rows"] += len(tables)

    def on_pruned(gone):
        for c in gone:
            if c in seq:                             # pruned before its step completed: nothing to free
                s = seq.pop(c)                       # both managers number sequences identically
                assert bm_c.prune(s).tolist() == bm_o.prune(s)
                counts["released"] += 1

    path = drive(ctl, n, m, depth, seed, p_perfect=p, on_complete=on_complete, on_verify=on_verify,
                 on_pruned=on_pruned)

    assert counts["batches"] > 3 and counts["released"] > 0
    assert bm_c.snapshot()["seqs"] == bm_o.snapshot()["seqs"]
    if p == 0.0:
        assert [sorted(path[c] for c in ctl.round(r)[1]) for r in range(depth)] == beam_search(n, m, depth, seed)
    print(f"    search n {n} m {m}: {counts['batches']} verify batches, {counts['rows']} rows, "
          f"{counts['released']} sequences released", flush=True)
