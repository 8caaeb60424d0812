"""Seeded synthetic workloads: trees of candidate reasoning paths over one paged KV cache.

This module is shared input plumbing.  It draws token ids, tree shapes and bf16 values from
seeded NumPy streams and describes a workload as a script of block-manager operations
(extend / prune) plus attention launches.  It holds none of the method's arithmetic: no
block deduplication, no attention, no coalescing.  Each side (the oracle and the HIP
library) runs the script through its own block manager.

Structure follows the paper's beam-search workloads (Sec. 2.2 beam search with a PRM,
Sec. 3.2.1 candidate-path explosion under speculation, Sec. 4.2 common-token ratio,
Sec. 4.3 verification batch scale), with the datasets and models replaced by seeded
random tokens and N(0,1) values.

Streams (NumPy PCG64 seeded with a list):
  [seed, 1]             tree structure (step lengths, branching choices, prune choices)
  [seed, 2]             token ids, uniform over a 32,000-entry vocabulary
  [seed, 3, 0, c]       K pool values, [seed, 3, 1, c] V pool values
  [seed, 3, 2 + j, c]   query values of launch j
where c numbers the 2^24-value chunks of the flattened tensor (each chunk has its own stream, so
the chunks are drawn in parallel threads and the values do not depend on the thread count).
Values are drawn as float32 N(0,1) and rounded once to bf16 (round to nearest even).
"""
from __future__ import annotations

import math
import os
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

VOCAB = 32000
BF16_NAN = np.uint16(0x7FC0)


# ----------------------------------------------------------------------------- bf16 bits

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns the uint16 bit patterns.

    Inputs are finite here (normal draws); NaN/inf are not special-cased.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


CHUNK = 1 << 24


def _normal_bf16(key: Sequence[int], shape: Tuple[int, ...]) -> np.ndarray:
    """N(0,1) float32 draws rounded to bf16 bits; chunk c of the flattened tensor comes from the
    stream [*key, c]."""
    from concurrent.futures import ThreadPoolExecutor
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)

    def fill(c):
        s, e = c * CHUNK, min(n, (c + 1) * CHUNK)
        rng = np.random.default_rng([*key, c])
        out[s:e] = f32_to_bf16_bits(rng.standard_normal(e - s, dtype=np.float32))

    n_chunks = -(-n // CHUNK)
    if n_chunks <= 1:
        for c in range(n_chunks):
            fill(c)
    else:
        workers = min(n_chunks, 16, len(os.sched_getaffinity(0)))
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, range(n_chunks)))
    return out.reshape(shape)


# ----------------------------------------------------------------------------- script

@dataclass(frozen=True)
class Shape:
    hq: int
    hkv: int
    d: int
    block_size: int = 16

    @property
    def group(self) -> int:
        return self.hq // self.hkv


@dataclass
class Extend:
    """Create a new sequence = parent's path + `tokens` (parent -1: a new root).

    The new sequence's handle is the number of Extend events before this one.
    """
    parent: int
    tokens: np.ndarray
    seal: bool


@dataclass
class Prune:
    handle: int


@dataclass
class Launch:
    """Submit candidates (handle, q_len) to one attention call.  decode: every q_len == 1."""
    name: str
    cands: List[Tuple[int, int]]
    decode: bool


@dataclass
class Workload:
    name: str
    shape: Shape
    seed: int
    events: list = field(default_factory=list)
    num_blocks: int = 0
    max_seqs: int = 0
    note: str = ""

    # ------------------------------------------------------------------ building helpers
    def _n_extends(self) -> int:
        return sum(1 for e in self.events if isinstance(e, Extend))

    def extend(self, parent: int, tokens: np.ndarray, seal: bool) -> int:
        h = self._n_extends()
        self.events.append(Extend(int(parent), np.asarray(tokens, dtype=np.int32), bool(seal)))
        return h

    def prune(self, handle: int) -> None:
        self.events.append(Prune(int(handle)))

    def launch(self, name: str, cands: Sequence[Tuple[int, int]]) -> None:
        cands = [(int(h), int(q)) for h, q in cands]
        self.events.append(Launch(name, cands, all(q == 1 for _, q in cands)))

    def finalize(self, num_blocks: Optional[int] = None, max_seqs: Optional[int] = None) -> "Workload":
        bs = self.shape.block_size
        upper = sum(-(-len(e.tokens) // bs) for e in self.events if isinstance(e, Extend))
        self.num_blocks = int(num_blocks if num_blocks is not None else max(upper, 1))
        self.max_seqs = int(max_seqs if max_seqs is not None else max(self._n_extends(), 1))
        return self

    @property
    def launches(self) -> List[Launch]:
        return [e for e in self.events if isinstance(e, Launch)]

    # ------------------------------------------------------------------ values
    def kv_values(self) -> Tuple[np.ndarray, np.ndarray]:
        """K and V pools as bf16 bits, [num_blocks, hkv, block_size, d] each."""
        s = self.shape
        shp = (self.num_blocks, s.hkv, s.block_size, s.d)
        k = _normal_bf16([self.seed, 3, 0], shp)
        v = _normal_bf16([self.seed, 3, 1], shp)
        return k, v

    def q_values(self, launch_index: int, n_qtok: int) -> np.ndarray:
        """Queries of launch `launch_index` as bf16 bits, [n_qtok, hq, d]."""
        s = self.shape
        return _normal_bf16([self.seed, 3, 2 + launch_index], (n_qtok, s.hq, s.d))


def poison_padding(k: np.ndarray, v: np.ndarray, block_len: np.ndarray) -> None:
    """Test aid: fill every slot that holds no token (beyond block_len, or a free block) with bf16 NaN,
    so that any read of padding shows up in the result."""
    bs = k.shape[2]
    slot = np.arange(bs)[None, :]
    dead = slot >= np.asarray(block_len)[:, None]          # [num_blocks, bs]
    k[np.nonzero(dead)[0], :, np.nonzero(dead)[1], :] = BF16_NAN
    v[np.nonzero(dead)[0], :, np.nonzero(dead)[1], :] = BF16_NAN


# ----------------------------------------------------------------------------- driver

def drive(wl: Workload, bm, on_launch=None, on_op=None):
    """Run the workload's script against a block manager adapter.

    `bm.extend(parent_seq, tokens, seal) -> (seq, blocks, hits)` and `bm.prune(seq) -> freed`.
    Handles are mapped to the sequence ids the adapter returns.  `on_op(kind, result)` is called
    after every operation, `on_launch(index, launch, [(seq, q_len), ...])` at every launch.
    Returns the handle -> sequence id map.
    """
    seq_of = []
    li = 0
    for e in wl.events:
        if isinstance(e, Extend):
            parent = -1 if e.parent < 0 else seq_of[e.parent]
            res = bm.extend(parent, e.tokens, e.seal)
            seq_of.append(res[0])
            if on_op is not None:
                on_op("extend", res)
        elif isinstance(e, Prune):
            res = bm.prune(seq_of[e.handle])
            if on_op is not None:
                on_op("prune", res)
        else:
            if on_launch is not None:
                on_launch(li, e, [(seq_of[h], q) for h, q in e.cands])
            li += 1
    return seq_of


# ----------------------------------------------------------------------------- configurations

def _rngs(seed: int):
    return np.random.default_rng([seed, 1]), np.random.default_rng([seed, 2])


def _toks(rt: np.random.Generator, n: int) -> np.ndarray:
    return rt.integers(0, VOCAB, size=int(n), dtype=np.int32)


def tiny_decode(seed: int = 0) -> Workload:
    """1 query, 256-token shared prompt, 4 candidates each with a private 64-token suffix;
    8 query heads, 2 KV heads, head_dim 64, block 16; decode (q_len 1)."""
    rs, rt = _rngs(seed)
    wl = Workload("tiny_decode", Shape(8, 2, 64), seed,
                  note="1 query; prompt 256 sealed; 4 x extend(prompt, 64, unsealed); prompt released")
    p = wl.extend(-1, _toks(rt, 256), True)
    cands = [wl.extend(p, _toks(rt, 64), False) for _ in range(4)]
    wl.prune(p)
    wl.launch("decode", [(c, 1) for c in cands])
    return wl.finalize()


def beam_decode(seed: int = 0, n_queries: int = 16) -> Workload:
    """Beam-search decode, small-model shape: 12 query heads, 2 KV heads, head_dim 128.
    Per query: 512-token prompt; completed steps U{64..256} (sealed) with branching 4, 2, 2;
    two live candidates per level-3 node with an in-progress suffix U{1..256} (unsealed);
    interior sequences released.  32 candidates per query, q_len 1."""
    rs, rt = _rngs(seed)
    wl = Workload("beam_decode", Shape(12, 2, 128), seed,
                  note="16 queries x (prompt 512; steps U{64..256} branching 4,2,2; 32 live suffixes U{1..256})")
    interior, leaves = [], []
    for _ in range(n_queries):
        p = wl.extend(-1, _toks(rt, 512), True)
        interior.append(p)
        level = [p]
        for br in (4, 2, 2):
            nxt = []
            for node in level:
                for _ in range(br):
                    nxt.append(wl.extend(node, _toks(rt, rs.integers(64, 257)), True))
            interior.extend(nxt)
            level = nxt
        for node in level:
            for _ in range(2):
                leaves.append(wl.extend(node, _toks(rt, rs.integers(1, 257)), False))
    for h in interior:
        wl.prune(h)
    wl.launch("decode", [(c, 1) for c in leaves])
    return wl.finalize()


def step_verify(seed: int = 0, n_queries: int = 8, n_cands: int = 16) -> Workload:
    """Step verification, 7B reward-model shape: 28 query heads, 4 KV heads, head_dim 128.
    Per query: shared context U{1024..4096} (sealed); 16 candidates each add one sealed step
    U{32..256}; the context sequence is released; q_len = step length, causal within the step."""
    rs, rt = _rngs(seed)
    wl = Workload("step_verify", Shape(28, 4, 128), seed,
                  note="8 queries x (context U{1024..4096}; 16 candidate steps U{32..256}, verified causally)")
    ctxs, cands = [], []
    for _ in range(n_queries):
        c = wl.extend(-1, _toks(rt, rs.integers(1024, 4097)), True)
        ctxs.append(c)
        for _ in range(n_cands):
            n = int(rs.integers(32, 257))
            cands.append((wl.extend(c, _toks(rt, n), True), n))
    for c in ctxs:
        wl.prune(c)
    wl.launch("verify", cands)
    return wl.finalize()


def spec_explosion(seed: int = 0, n_queries: int = 8) -> Workload:
    """Speculative explosion: 12 query heads, 2 KV heads, head_dim 128.
    Per query: prompt U{512..6144}; 4 levels of branching 4 (256 leaves); step length
    clip(round(exp(N(ln 128, 0.6))), 16, 512); in each sibling group, sibling j >= 1 repeats the
    tokens of a uniformly chosen earlier sibling with probability 0.2*4/3 (so about 20% of step
    extensions are token-identical and deduplicate); all steps sealed; interior released; decode."""
    rs, rt = _rngs(seed)
    wl = Workload("spec_explosion", Shape(12, 2, 128), seed,
                  note="8 queries x (prompt U{512..6144}; 4 levels x branching 4; lognormal steps; 20% identical siblings)")
    p_copy = 0.2 * 4.0 / 3.0
    interior, leaves = [], []
    for _ in range(n_queries):
        p = wl.extend(-1, _toks(rt, rs.integers(512, 6145)), True)
        interior.append(p)
        level = [p]
        for lvl in range(4):
            nxt = []
            for node in level:
                sib_tokens = []
                for j in range(4):
                    if j >= 1 and rs.random() < p_copy:
                        toks = sib_tokens[int(rs.integers(0, j))]
                    else:
                        n = int(np.clip(round(math.exp(rs.normal(math.log(128.0), 0.6))), 16, 512))
                        toks = _toks(rt, n)
                    sib_tokens.append(toks)
                    nxt.append(wl.extend(node, toks, True))
            if lvl < 3:
                interior.extend(nxt)
            level = nxt
        leaves.extend(level)
    for h in interior:
        wl.prune(h)
    wl.launch("decode", [(c, 1) for c in leaves])
    return wl.finalize()


def spec_prompts(seed: int = 0, n_queries: int = 8, n_cands: int = 204) -> Workload:
    """The shared-prefix pass of the speculative explosion on its own: 12 query heads, 2 KV heads,
    head_dim 128.  Per query a prompt U{512..6144} (sealed), as in spec_explosion, shared by
    n_cands candidates (about spec_explosion's distinct rows per query), each decoding one token of
    its own (an unsealed 1-token step); prompts released; decode.  Every prompt block is read by
    n_cands x 6 query rows per KV head, so the call's work is almost all the shared pass."""
    rs, rt = _rngs(seed)
    wl = Workload("spec_prompts", Shape(12, 2, 128), seed,
                  note=f"{n_queries} queries x (prompt U{{512..6144}} shared by {n_cands} 1-token candidates)")
    prompts, cands = [], []
    for _ in range(n_queries):
        p = wl.extend(-1, _toks(rt, rs.integers(512, 6145)), True)
        prompts.append(p)
        for _ in range(n_cands):
            cands.append(wl.extend(p, _toks(rt, 1), False))
    for h in prompts:
        wl.prune(h)
    wl.launch("decode", [(c, 1) for c in cands])
    return wl.finalize()


def mixed_serving(seed: int = 0, n_queries: int = 64) -> Workload:
    """Mixed serving batch: 32 query heads, 8 KV heads, head_dim 128.
    Per query: prompt U{256..2048}; U{4..64} candidates in sibling groups of 4, each group under a
    sealed parent step U{64..256}; each candidate is decode (p 0.5: unsealed suffix U{1..256},
    q_len 1) or verify (sealed step U{32..256}, q_len = step length, causal).  Interior sequences
    stay live.  Launch A covers every candidate; then 30% of candidates (seeded choice, ascending
    order) are pruned and as many new candidates extend uniformly chosen group parents; launch B
    covers the survivors followed by the new candidates."""
    rs, rt = _rngs(seed)
    wl = Workload("mixed_serving", Shape(32, 8, 128), seed,
                  note="64 queries; prompts U{256..2048}; 4..64 candidates; half decode / half verify; 30% pruned + refilled")

    def new_cand(parent):
        if rs.random() < 0.5:
            return wl.extend(parent, _toks(rt, rs.integers(1, 257)), False), 1
        n = int(rs.integers(32, 257))
        return wl.extend(parent, _toks(rt, n), True), n

    parents, cands = [], []
    for _ in range(n_queries):
        p = wl.extend(-1, _toks(rt, rs.integers(256, 2049)), True)
        n_c = int(rs.integers(4, 65))
        gp = None
        for c in range(n_c):
            if c % 4 == 0:
                gp = wl.extend(p, _toks(rt, rs.integers(64, 257)), True)
                parents.append(gp)
            cands.append(new_cand(gp))
    wl.launch("A", cands)
    n_prune = int(round(0.3 * len(cands)))
    gone = np.sort(rs.choice(len(cands), size=n_prune, replace=False))
    for i in gone:
        wl.prune(cands[int(i)][0])
    keep = [c for i, c in enumerate(cands) if i not in set(int(g) for g in gone)]
    refill = [new_cand(parents[int(rs.integers(0, len(parents)))]) for _ in range(n_prune)]
    wl.launch("B", keep + refill)
    return wl.finalize()


CONFIGS = {
    "tiny_decode": tiny_decode,
    "beam_decode": beam_decode,
    "step_verify": step_verify,
    "spec_explosion": spec_explosion,
    "mixed_serving": mixed_serving,
    "spec_prompts": spec_prompts,
}


def random_tree(seed: int, shape: Shape, n_roots: int = 2, depth: int = 3, max_branch: int = 3,
                max_step: int = 40, p_dup: float = 0.3, p_verify: float = 0.5, release: bool = True,
                min_root: int = 1) -> Workload:
    """Small random tree for edge-case tests: ragged steps (partial blocks in the middle of paths),
    duplicated sibling steps, unsealed decode leaves and sealed verify leaves in one launch."""
    rs, rt = _rngs(seed)
    wl = Workload(f"random_tree_{seed}", shape, seed, note="random small tree")
    interior, leaves = [], []
    for _ in range(n_roots):
        r = wl.extend(-1, _toks(rt, rs.integers(min_root, max_step + 1)), True)
        interior.append(r)
        level = [r]
        for lvl in range(depth):
            nxt = []
            for node in level:
                prev = []
                for j in range(int(rs.integers(1, max_branch + 1))):
                    last = lvl == depth - 1
                    if prev and rs.random() < p_dup:
                        toks, seal = prev[int(rs.integers(0, len(prev)))], True
                    else:
                        toks = _toks(rt, rs.integers(1, max_step + 1))
                        seal = (not last) or rs.random() < p_verify
                    if seal:
                        prev.append(toks)
                    h = wl.extend(node, toks, seal)
                    if last:
                        leaves.append((h, len(toks) if seal else 1))
                    else:
                        nxt.append(h)
            interior.extend(nxt)
            level = nxt
    if release:
        for h in interior:
            wl.prune(h)
    wl.launch("mixed", leaves)
    return wl.finalize()
