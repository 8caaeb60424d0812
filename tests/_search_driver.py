"""Test helper: drives a speculative beam search on a controller -- the oracle's or the library's,
which share method names (expand, complete, tick, flush, score, pruned, node, round) -- and the
textbook beam search it is compared with.  Holds no controller logic of its own."""
import numpy as np

VERIFIED, SELECTED = 3, 4


def path_score(seed, path, p_perfect=0.0):
    """Verifier score of a candidate, a fixed function of its path (root index, then child indices),
    exactly representable in float32."""
    r = np.random.default_rng([seed, 7, *path])
    if p_perfect and r.random() < p_perfect:
        return 1.0
    return float(np.float32(r.random() * 0.999))


def beam_search(n, m, depth, seed):
    """Plain beam search (beam size n, width m, k = n / m survivors per step): every candidate of a
    step is scored, the k best are kept, each expands into m candidates.  Selected paths per step."""
    k = n // m
    frontier = [(i,) for i in range(n)]
    out = []
    for _ in range(depth):
        scores = [path_score(seed, p) for p in frontier]
        assert len(set(scores)) == len(scores), "tied scores: pick another seed"
        keep = [p for _, p in sorted(zip(scores, frontier), key=lambda t: -t[0])[:k]]
        out.append(sorted(keep))
        frontier = [p + (j,) for p in keep for j in range(m)]
    return out


def drive(S, n, m, depth, seed, p_perfect=0.0, p_done=0.3, p_arrive=0.7, on_event=None, max_iters=20000,
          on_complete=None, on_verify=None, on_pruned=None):
    """Runs the speculative search until round depth-1 is settled.  Each iteration every generating
    candidate completes its step with probability p_done (a flush is taken whenever one is advised),
    then a tick; the oldest verification batch in flight returns its scores with probability p_arrive,
    and every candidate scored and not pruned expands at once into m candidates (speculation) unless
    it is on the last step.  Hooks: on_complete(candidate, n_tokens) when a step completes,
    on_verify(batch) just before a batch's scores are reported, on_pruned(candidates) after each drain.
    Returns {candidate: path}."""
    rng = np.random.default_rng([seed, 99])
    path, generating, in_flight = {}, [], []
    first = S.expand(-1, n)
    for i in range(n):
        path[first + i] = (i,)
        generating.append(first + i)

    def drain():
        gone = S.pruned()
        for c in gone:
            if c in generating:
                generating.remove(c)
        if on_pruned and gone:
            on_pruned(gone)

    for _ in range(max_iters):
        if S.round(depth - 1)[0]:
            return path
        for c in list(generating):
            if rng.random() < p_done:
                generating.remove(c)
                n_tok = int(rng.integers(20, 400))
                if on_complete:
                    on_complete(c, n_tok)
                if S.complete(c, n_tok):
                    in_flight.append(S.flush())
        if S.tick():
            in_flight.append(S.flush())
        if in_flight and rng.random() < p_arrive:
            batch = in_flight.pop(0)
            if on_verify:
                on_verify(batch)
            S.score(batch, [path_score(seed, path[c], p_perfect) for c in batch])
            drain()
            for c in batch:
                state, _, d, _ = S.node(c)
                if state in (VERIFIED, SELECTED) and d < depth - 1:
                    f = S.expand(c, m)
                    for j in range(m):
                        path[f + j] = path[c] + (j,)
                        generating.append(f + j)
                    drain()
        if on_event:
            on_event(S)
    raise AssertionError("the search did not settle its last round")
