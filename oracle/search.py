"""Oracle controller of a speculative beam search: early pruning and lazy verification.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The search (beam search with a process reward model, Sec. 2.2) keeps the k best-scored candidates
of every step -- a round -- and expands each of them into the next step's candidates.  Under
speculation (Sec. 3) a candidate expands as soon as its own score is known, before its round is
settled, so several depths are in flight at once.

Early pruning (Sec. 4.1):
* Rule 1.  A scored candidate is pruned as soon as k scored candidates that are sure to share its
  round outscore it: no later score can lift it into that round's selection.
* Rule 2.  Scores lie in [0, 1] and 1.0 is perfect.  Once k candidates have the perfect score they
  are the selection and every other candidate of the round is pruned.  (The paper notes that this
  rule may change the selection when later candidates would tie at 1.0; the first k to arrive win.)

Readings (the paper does not spell these out):
* Round d's members are the children of round d-1's selection (the prompt's candidates for d = 0).
  While round d-1 is open, a depth-d candidate is speculative: it belongs to round d only if its
  parent is selected, and then so do its siblings.  The rules only use candidates that are sure to
  share the judged candidate's round: its siblings while speculative, all members otherwise.
* Below the top k: at least k of those candidates have a strictly higher score (ties are kept
  until the round is settled).  The first k perfect scores: in the order in which scores arrived.
* A round is settled by rule 2, or once every selected parent has expanded and every unpruned member
  has a score: the k best by (score descending, arrival ascending) are selected.  The other
  candidates of the round are pruned, and pruning a candidate prunes everything expanded from it.

Lazy verification (Sec. 4.3): a completed step is queued rather than verified; the queue is flushed
as one batch when (1) the queued tokens exceed a threshold (2,048 in the paper), (2) the whole sibling
group of a queued candidate has completed its step -- pruned siblings do not hold it back -- or (3) a
queued candidate's deferral count would exceed its limit (6 in the paper), a deferral being a tick
(one iteration of the generator) passed without a flush.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

GENERATING, QUEUED, VERIFYING, VERIFIED, SELECTED, PRUNED = range(6)


class SearchError(Exception):
    def __init__(self, kind: str, msg: str):
        super().__init__(msg)
        self.kind = kind  # "EINVAL" | "ENOSEQ" | "ENOMEM" | "ECAP"


@dataclass
class Candidate:
    parent: int
    depth: int
    children: Optional[List[int]] = None   # None until expanded
    state: int = GENERATING
    tokens: int = 0
    deferrals: int = 0
    arrival: Optional[int] = None          # index of its score in arrival order
    score: Optional[float] = None
    flushed: bool = False
    scored: bool = False


@dataclass
class Search:
    k: int
    max_nodes: int
    token_threshold: int = 2048
    max_deferrals: int = 6
    cands: List[Candidate] = field(default_factory=list)
    roots: Optional[List[int]] = None
    queue: List[int] = field(default_factory=list)
    selection: Dict[int, List[int]] = field(default_factory=dict)   # settled rounds
    newly_pruned: set = field(default_factory=set)
    arrivals: int = 0

    # ---------------------------------------------------------------- helpers
    def _alive(self, c: int) -> bool:
        return self.cands[c].state != PRUNED

    def _scored(self, c: int) -> bool:
        return self.cands[c].state in (VERIFIED, SELECTED)

    def _siblings(self, parent: int) -> List[int]:
        if parent < 0:
            return list(self.roots or [])
        return list(self.cands[parent].children or [])

    def _prune(self, c: int) -> None:
        todo = [c]
        while todo:
            x = todo.pop()
            if self.cands[x].state == PRUNED:
                continue
            if x in self.queue:
                self.queue.remove(x)
            self.cands[x].state = PRUNED
            self.newly_pruned.add(x)
            todo.extend(self.cands[x].children or [])

    def _judge(self, sure: List[int], settles: bool) -> bool:
        """Rules 1 and 2 over a set of candidates sure to share a round.  With settles=True the set is
        the round's membership, and rule 2 settles the round."""
        live = [c for c in sure if self._alive(c)]
        perfect = sorted((c for c in live if self._scored(c) and self.cands[c].score == 1.0),
                         key=lambda c: self.cands[c].arrival)
        if len(perfect) >= self.k:
            winners = perfect[:self.k]
            if settles:
                self._settle_round(self.cands[winners[0]].depth, winners)
                return True
            losers = [c for c in live if c not in winners]
            for c in losers:
                self._prune(c)
            if losers:
                return True
        scored = [c for c in live if self._scored(c)]
        doomed = [c for c in scored
                  if sum(1 for o in scored if self.cands[o].score > self.cands[c].score) >= self.k]
        for c in doomed:
            self._prune(c)
        return bool(doomed)

    def _settle_round(self, depth: int, chosen: List[int]) -> None:
        self.selection[depth] = sorted(chosen)
        for c in chosen:
            self.cands[c].state = SELECTED
        for c, cand in enumerate(self.cands):
            if cand.depth == depth and c not in chosen:
                self._prune(c)

    def _members(self, depth: int):
        """(members, every selected parent expanded) of a round whose parents are settled, else None."""
        if depth == 0:
            return (list(self.roots), True) if self.roots is not None else None
        if depth - 1 not in self.selection:
            return None
        members, expanded = [], True
        for p in self.selection[depth - 1]:
            if self.cands[p].children is None:
                expanded = False
            members += self._siblings(p)
        return members, expanded

    def _update(self) -> None:
        changed = True
        while changed:
            changed = False
            depths = sorted({c.depth for c in self.cands})
            for d in depths:
                if d in self.selection:
                    continue
                known = self._members(d)
                if known is None:
                    for p, cand in enumerate(self.cands):      # speculative sibling groups
                        if cand.depth == d - 1 and self._alive(p) and cand.children:
                            changed |= self._judge(cand.children, settles=False)
                    continue
                members, expanded = known
                if self._judge(members, settles=True):
                    changed = True
                    continue
                live = [c for c in members if self._alive(c)]
                if expanded and all(self._scored(c) for c in live):
                    best = sorted(live, key=lambda c: (-self.cands[c].score, self.cands[c].arrival))
                    self._settle_round(d, best[:self.k])
                    changed = True

    def _flush_due(self) -> bool:
        if not self.queue:
            return False
        if sum(self.cands[c].tokens for c in self.queue) > self.token_threshold:
            return True
        if any(self.cands[c].deferrals >= self.max_deferrals for c in self.queue):
            return True
        return any(all(self.cands[s].state != GENERATING for s in self._siblings(self.cands[c].parent))
                   for c in self.queue)

    def _get(self, c: int, what: str) -> Candidate:
        if not 0 <= c < len(self.cands):
            raise SearchError("EINVAL", f"{what}: no candidate {c}")
        return self.cands[c]

    # ---------------------------------------------------------------- events
    def expand(self, parent: int, n: int) -> int:
        if n < 0:
            raise SearchError("EINVAL", "n < 0")
        if parent == -1:
            if self.roots is not None:
                raise SearchError("EINVAL", "roots exist")
            depth = 0
        else:
            p = self._get(parent, "expand")
            if p.state == PRUNED:
                raise SearchError("ENOSEQ", "parent pruned")
            if p.state not in (VERIFIED, SELECTED):
                raise SearchError("EINVAL", "parent has no score")
            if p.children is not None:
                raise SearchError("EINVAL", "already expanded")
            depth = p.depth + 1
        if len(self.cands) + n > self.max_nodes:
            raise SearchError("ENOMEM", "too many candidates")
        first = len(self.cands)
        ids = list(range(first, first + n))
        self.cands += [Candidate(parent=parent, depth=depth) for _ in ids]
        if parent == -1:
            self.roots = ids
        else:
            self.cands[parent].children = ids
        self._update()
        return first

    def complete(self, c: int, n_tokens: int) -> bool:
        cand = self._get(c, "complete")
        if cand.state == PRUNED:
            raise SearchError("ENOSEQ", "pruned")
        if cand.state != GENERATING:
            raise SearchError("EINVAL", "not generating")
        if n_tokens < 1:
            raise SearchError("EINVAL", "n_tokens < 1")
        cand.state, cand.tokens, cand.deferrals = QUEUED, n_tokens, 0
        self.queue.append(c)
        return self._flush_due()

    def tick(self) -> bool:
        due = self._flush_due()
        if not due:
            for c in self.queue:
                self.cands[c].deferrals += 1
        return due

    def flush(self) -> List[int]:
        batch, self.queue = self.queue, []
        for c in batch:
            self.cands[c].state = VERIFYING
            self.cands[c].flushed = True
        return batch

    def score(self, nodes: List[int], scores: List[float]) -> None:
        if len(nodes) != len(set(nodes)):
            raise SearchError("EINVAL", "repeated candidate")
        for c, s in zip(nodes, scores):
            cand = self._get(c, "score")
            if not cand.flushed or cand.scored:
                raise SearchError("EINVAL", "not awaiting a score")
            if not 0.0 <= s <= 1.0:
                raise SearchError("EINVAL", "score outside [0, 1]")
        for c, s in zip(nodes, scores):
            cand = self.cands[c]
            cand.scored = True
            if cand.state == PRUNED:
                continue
            cand.state, cand.score, cand.arrival = VERIFIED, s, self.arrivals
            self.arrivals += 1
            self._update()

    def pruned(self) -> List[int]:
        out = sorted(self.newly_pruned)
        self.newly_pruned = set()
        return out

    def node(self, c: int):
        """(state, parent, depth, score or None)."""
        cand = self._get(c, "node")
        return cand.state, cand.parent, cand.depth, cand.score if cand.arrival is not None else None

    def round(self, depth: int):
        if depth in self.selection:
            return True, list(self.selection[depth])
        return False, []

    def snapshot(self) -> dict:
        """Same layout as the library's parsed snapshot; scores as float32 bit patterns."""
        import numpy as np
        nodes = []
        for c in self.cands:
            bits = int(np.float32(c.score).view(np.int32)) if c.arrival is not None else 0
            nodes.append((c.parent, c.depth, c.state, -1 if c.children is None else len(c.children), c.tokens,
                          c.deferrals, -1 if c.arrival is None else c.arrival, bits))
        n_rounds = max(self.selection) + 1 if self.selection else 0
        rounds = [(1, tuple(self.selection[d])) if d in self.selection else (0, ()) for d in range(n_rounds)]
        return {"k": self.k, "token_threshold": self.token_threshold, "max_deferrals": self.max_deferrals,
                "n_roots": -1 if self.roots is None else len(self.roots),
                "queued_tokens": sum(self.cands[c].tokens for c in self.queue),
                "nodes": nodes, "queue": list(self.queue), "rounds": rounds}
