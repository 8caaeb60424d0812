"""Python binding of libtreekv.so: tree-shared paged attention for speculative search on MI355X.

Argument marshalling only -- every step of the path (block manager, coalescing, planning and the
attention kernels) runs in the C/HIP library; PyTorch provides device memory and streams.  The
functions carry the names of the C entry points in include/treekv.h; failures raise TkvError
with the library's message.  The library must be built first (``python -m
paper_2609_39334_amd.build``); any entry point raises if it is missing -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch  # imported before the library so that both share torch's HIP runtime

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtreekv.so")

TKV_OK, TKV_EINVAL, TKV_ENOMEM, TKV_ENOSEQ, TKV_ECAP, TKV_EHIP = 0, -1, -2, -3, -4, -5
TKV_NOALLOC_MAX_BYTES = 64 << 20   # the static workspace of tkv_verify_noalloc (treekv.h)


class TkvError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class tkv_shape(ctypes.Structure):
    _fields_ = [("hq", ctypes.c_int32), ("hkv", ctypes.c_int32), ("d", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("num_blocks", ctypes.c_int32)]


class tkv_plan_options(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("wave_max_rows", "tile_min_items", "waves", "tile8_max_items",
                                              "wide_chunk_blocks", "fold_blocks")]


class tkv_plan_stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_rows", "n_qtok", "n_items", "n_items_shared", "n_items_row",
                                              "n_slots", "n_merge", "n_segments", "n_shared_segments",
                                              "n_items_wave", "n_waves", "n_idle_waves")] + \
               [(n, ctypes.c_int64) for n in ("logical_qtok", "uniq_kv_tokens", "path_kv_tokens", "flops")]


class tkv_plan_layout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in ("items", "toks", "blks", "merges", "merge_slots", "wave_records",
                                               "wave_off", "wave_tiles", "end")]


class tkv_plan_view(ctypes.Structure):
    _fields_ = [(n, ctypes.POINTER(ctypes.c_int32)) for n in ("items", "toks", "blks", "merges", "merge_slots")] + \
               [(n, ctypes.c_int32) for n in ("n_items", "n_toks", "n_blks", "n_merge", "n_merge_slots", "n_slots")]


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_PI32 = ctypes.POINTER(ctypes.c_int32)
_PU8 = ctypes.POINTER(ctypes.c_uint8)
_SIG = {
    "tkv_last_error": (ctypes.c_char_p, []),
    "tkv_bm_create": (ctypes.c_int, [_I32, _I32, _I32, ctypes.POINTER(_P)]),
    "tkv_bm_destroy": (None, [_P]),
    "tkv_bm_extend": (ctypes.c_int, [_P, _I32, _PI32, _I32, _I32, _PI32, _PI32, _PU8, _I32, _PI32]),
    "tkv_prune": (ctypes.c_int, [_P, _I32, _PI32, _I32, _PI32]),
    "tkv_bm_append": (ctypes.c_int, [_P, _I32, _PI32, _I32, _PI32, _I32]),
    "tkv_bm_seal": (ctypes.c_int, [_P, _I32, _PI32, _I32, _PI32]),
    "tkv_bm_fork": (ctypes.c_int, [_P, _I32, _PI32, _I32, _PI32, _I32]),
    "tkv_extend_slots": (ctypes.c_int, [_PI32, _PU8, _I32, _I32, _I32, _PI32]),
    "tkv_bm_table": (ctypes.c_int, [_P, _I32, _PI32, _I32, _PI32, _PI32]),
    "tkv_bm_refcount": (ctypes.c_int, [_P, _I32, _PI32]),
    "tkv_bm_block_len": (ctypes.c_int, [_P, _PI32]),
    "tkv_bm_snapshot": (ctypes.c_int, [_P, _P, ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t)]),
    "tkv_bm_coalesce": (ctypes.c_int, [_P, _I32, _PI32, _PI32, _PI32, _PI32, _PI32, _PI32]),
    "tkv_plan_create": (ctypes.c_int, [ctypes.POINTER(tkv_shape), _I32, _PI32, _PI32, _PI32, _PI32, _PI32,
                                       ctypes.POINTER(_P)]),
    "tkv_plan_create_ex": (ctypes.c_int, [ctypes.POINTER(tkv_shape), _I32, _PI32, _PI32, _PI32, _PI32, _PI32,
                                          ctypes.POINTER(tkv_plan_options), ctypes.POINTER(_P)]),
    "tkv_plan_workspace_bytes": (ctypes.c_size_t, [_P]),
    "tkv_plan_upload": (ctypes.c_int, [_P, _P, ctypes.c_size_t, _P]),
    "tkv_plan_update": (ctypes.c_int, [_P, _P, _P, _P, ctypes.POINTER(ctypes.c_int32)]),
    "tkv_plan_image": (ctypes.c_int, [_P, ctypes.POINTER(_P), ctypes.POINTER(tkv_plan_layout)]),
    "tkv_plan_dirty": (ctypes.c_int, [_P, ctypes.POINTER(_PI32), ctypes.POINTER(ctypes.c_int32),
                                      ctypes.POINTER(ctypes.c_int32)]),
    "tkv_plan_destroy": (None, [_P]),
    "tkv_plan_get_stats": (ctypes.c_int, [_P, ctypes.POINTER(tkv_plan_stats)]),
    "tkv_plan_get_view": (ctypes.c_int, [_P, ctypes.POINTER(tkv_plan_view)]),
    "tkv_decode": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P]),
    "tkv_verify": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P]),
    "tkv_verify_noalloc": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P]),
    "tkv_kv_append": (ctypes.c_int, [ctypes.POINTER(tkv_shape), _P, _I32, _P, _P, _P, _P, _P]),
    "tkv_cd_sample": (ctypes.c_int, [_I32, _I32, ctypes.c_float, _I32, _P, _P, _P, _I32, _P, _P, _P, _P]),
    "tkv_search_create": (ctypes.c_int, [_I32, _I32, _I32, _I32, ctypes.POINTER(_P)]),
    "tkv_search_destroy": (None, [_P]),
    "tkv_search_expand": (ctypes.c_int, [_P, _I32, _I32, _PI32]),
    "tkv_search_complete": (ctypes.c_int, [_P, _I32, _I32, _PI32]),
    "tkv_search_tick": (ctypes.c_int, [_P, _PI32]),
    "tkv_search_flush": (ctypes.c_int, [_P, _PI32, _I32, _PI32]),
    "tkv_search_score": (ctypes.c_int, [_P, _I32, _PI32, ctypes.POINTER(ctypes.c_float)]),
    "tkv_search_pruned": (ctypes.c_int, [_P, _PI32, _I32, _PI32]),
    "tkv_search_node": (ctypes.c_int, [_P, _I32, _PI32, _PI32, _PI32, ctypes.POINTER(ctypes.c_float)]),
    "tkv_search_round": (ctypes.c_int, [_P, _I32, _PI32, _I32, _PI32, _PI32]),
    "tkv_search_snapshot": (ctypes.c_int, [_P, _P, ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t)]),
    "tkv_plan_profile": (ctypes.c_int, [_P, _I32]),
    "tkv_plan_profile_read": (ctypes.c_int, [_P, _PI32, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_float)]),
}
EXPORTED = tuple(_SIG)

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libtreekv.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2609_39334_amd.build` "
                               "(or __graft_entry__.build()) first")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIG.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(rc: int) -> None:
    if rc != TKV_OK:
        raise TkvError(rc, lib().tkv_last_error().decode())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32).reshape(-1))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(_PI32)


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


# ------------------------------------------------------------------------- C entry points

def tkv_last_error() -> str:
    return lib().tkv_last_error().decode()


def tkv_bm_create(num_blocks: int, block_size: int, max_seqs: int) -> int:
    h = _P()
    _check(lib().tkv_bm_create(num_blocks, block_size, max_seqs, ctypes.byref(h)))
    return h.value


def tkv_bm_destroy(bm: int) -> None:
    lib().tkv_bm_destroy(bm)


def tkv_bm_extend(bm: int, parent: int, tokens, seal: bool, block_size: int = 16):
    """Returns (seq, block ids, hit flags) of the new sequence's step."""
    t = _i32(tokens)
    cap = max(1, -(-len(t) // block_size))
    blk = np.zeros(cap, dtype=np.int32)
    hit = np.zeros(cap, dtype=np.uint8)
    child, n = _I32(), _I32()
    _check(lib().tkv_bm_extend(bm, parent, _ptr(t), len(t), int(bool(seal)), ctypes.byref(child), _ptr(blk),
                               hit.ctypes.data_as(_PU8), cap, ctypes.byref(n)))
    return child.value, blk[:n.value].copy(), hit[:n.value].copy()


def tkv_prune(bm: int, seq: int, cap: int = None) -> np.ndarray:
    """Releases a sequence; returns the freed block ids in table order."""
    if cap is None:
        n, _ = _table_len(bm, seq)
        cap = max(1, n)
    out = np.zeros(cap, dtype=np.int32)
    n = _I32()
    _check(lib().tkv_prune(bm, seq, _ptr(out), cap, ctypes.byref(n)))
    return out[:n.value].copy()


def tkv_bm_append(bm: int, seq: int, tokens) -> np.ndarray:
    """Grows a sequence in place; returns each token's pool slot (block * block_size + slot)."""
    t = _i32(tokens)
    dst = np.zeros(max(1, len(t)), dtype=np.int32)
    _check(lib().tkv_bm_append(bm, seq, _ptr(t), len(t), _ptr(dst), len(t)))
    return dst[:len(t)].copy()


def tkv_bm_seal(bm: int, seq: int):
    """Completes the open step of a sequence; returns the (own block, sealed block) replacements."""
    n = _I32()
    rc = lib().tkv_bm_seal(bm, seq, None, 0, ctypes.byref(n))
    if rc == TKV_OK:
        return []
    if rc != TKV_ECAP:
        _check(rc)
    out = np.zeros(2 * n.value, dtype=np.int32)
    _check(lib().tkv_bm_seal(bm, seq, _ptr(out), n.value, ctypes.byref(n)))
    return [(int(out[2 * i]), int(out[2 * i + 1])) for i in range(n.value)]


def tkv_bm_fork(bm: int, seq: int, tokens) -> list:
    """Branches a sequence: seals its open step, then one open child per token; returns the children."""
    t = _i32(tokens)
    out = np.zeros(max(1, len(t)), dtype=np.int32)
    _check(lib().tkv_bm_fork(bm, seq, _ptr(t), len(t), _ptr(out), len(t)))
    return [int(x) for x in out[:len(t)]]


def tkv_extend_slots(blk, hit, n_tok: int, block_size: int = 16) -> np.ndarray:
    """Pool slots of a new step's tokens (-1 where the block was a deduplication hit)."""
    b = _i32(blk)
    h = np.ascontiguousarray(np.asarray(hit, dtype=np.uint8).reshape(-1))
    dst = np.zeros(max(1, n_tok), dtype=np.int32)
    _check(lib().tkv_extend_slots(_ptr(b), h.ctypes.data_as(_PU8), len(b), n_tok, block_size, _ptr(dst)))
    return dst[:n_tok].copy()


def _table_len(bm: int, seq: int):
    n, kv = _I32(), _I32()
    rc = lib().tkv_bm_table(bm, seq, None, 0, ctypes.byref(n), ctypes.byref(kv))
    if rc not in (TKV_OK, TKV_ECAP):
        _check(rc)
    return n.value, kv.value


def tkv_bm_table(bm: int, seq: int):
    """Returns (block table, kv_len)."""
    n, _ = _table_len(bm, seq)
    out = np.zeros(max(1, n), dtype=np.int32)
    nn, kv = _I32(), _I32()
    _check(lib().tkv_bm_table(bm, seq, _ptr(out), len(out), ctypes.byref(nn), ctypes.byref(kv)))
    return out[:nn.value].copy(), kv.value


def tkv_bm_refcount(bm: int, blk: int) -> int:
    rc = _I32()
    _check(lib().tkv_bm_refcount(bm, blk, ctypes.byref(rc)))
    return rc.value


def tkv_bm_block_len(bm: int, num_blocks: int) -> np.ndarray:
    out = np.zeros(num_blocks, dtype=np.int32)
    _check(lib().tkv_bm_block_len(bm, _ptr(out)))
    return out


def tkv_bm_snapshot(bm: int, seqs: bool = True) -> dict:
    """Parsed state; seqs=False skips decoding the per-sequence tables."""
    used = ctypes.c_size_t()
    lib().tkv_bm_snapshot(bm, None, 0, ctypes.byref(used))
    buf = np.zeros(used.value // 4, dtype=np.int32)
    _check(lib().tkv_bm_snapshot(bm, buf.ctypes.data_as(_P), used.value, ctypes.byref(used)))
    nb, bs, ms, nlive = (int(x) for x in buf[:4])
    w = 4
    snap = {"refcount": buf[w:w + nb].copy(), "block_len": buf[w + nb:w + 2 * nb].copy(),
            "indexed": buf[w + 2 * nb:w + 3 * nb].copy(), "seqs": {}}
    w += 3 * nb
    for _ in range(nlive if seqs else 0):
        s, sealed, n_open, n = (int(x) for x in buf[w:w + 4])
        snap["seqs"][s] = (tuple(int(b) for b in buf[w + 4:w + 4 + n]), sealed, n_open)
        w += 4 + n
    return snap


def tkv_bm_coalesce(bm: int, seqs: Sequence[int], q_lens: Sequence[int]):
    """Returns (row of each candidate, first candidate of each row, multiplicity of each row)."""
    s, q = _i32(seqs), _i32(q_lens)
    n = len(s)
    row_of = np.zeros(max(1, n), dtype=np.int32)
    first = np.zeros(max(1, n), dtype=np.int32)
    mult = np.zeros(max(1, n), dtype=np.int32)
    nr = _I32()
    _check(lib().tkv_bm_coalesce(bm, n, _ptr(s), _ptr(q), _ptr(row_of), _ptr(first), _ptr(mult), ctypes.byref(nr)))
    return row_of[:n].copy(), first[:nr.value].copy(), mult[:nr.value].copy()


def tkv_plan_create(shape, q_indptr, kv_indptr, kv_blocks, block_len, multiplicity=None) -> int:
    """shape = (hq, hkv, d, block_size, num_blocks)."""
    sh = tkv_shape(*[int(x) for x in shape])
    qi, ki, kb, bl = _i32(q_indptr), _i32(kv_indptr), _i32(kv_blocks), _i32(block_len)
    mu = None if multiplicity is None else _i32(multiplicity)
    h = _P()
    _check(lib().tkv_plan_create(ctypes.byref(sh), len(qi) - 1, _ptr(qi), _ptr(ki), _ptr(kb) if len(kb) else None,
                                 _ptr(bl), None if mu is None else _ptr(mu), ctypes.byref(h)))
    return h.value


def tkv_plan_create_ex(shape, q_indptr, kv_indptr, kv_blocks, block_len, multiplicity=None, options=None) -> int:
    """tkv_plan_create with placement options: a dict over the tkv_plan_options fields (missing
    fields, or None, keep the defaults)."""
    sh = tkv_shape(*[int(x) for x in shape])
    qi, ki, kb, bl = _i32(q_indptr), _i32(kv_indptr), _i32(kv_blocks), _i32(block_len)
    mu = None if multiplicity is None else _i32(multiplicity)
    opts = None
    if options is not None:
        unknown = set(options) - {f for f, _ in tkv_plan_options._fields_}
        if unknown:
            raise ValueError(f"unknown plan options {sorted(unknown)}")
        opts = tkv_plan_options(*[int(options.get(f, -1)) for f, _ in tkv_plan_options._fields_])
    h = _P()
    _check(lib().tkv_plan_create_ex(ctypes.byref(sh), len(qi) - 1, _ptr(qi), _ptr(ki), _ptr(kb) if len(kb) else None,
                                    _ptr(bl), None if mu is None else _ptr(mu),
                                    None if opts is None else ctypes.byref(opts), ctypes.byref(h)))
    return h.value


def tkv_plan_workspace_bytes(plan: int) -> int:
    return int(lib().tkv_plan_workspace_bytes(plan))


def tkv_plan_upload(plan: int, workspace: torch.Tensor, stream=None) -> None:
    _check(lib().tkv_plan_upload(plan, workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                 _stream(stream)))


def tkv_plan_destroy(plan: int) -> None:
    lib().tkv_plan_destroy(plan)


def tkv_plan_update(plan: int, kv_indptr, kv_blocks, block_len) -> bool:
    """Bring the plan to new tables for the same rows; True if it was patched in place, False if
    it was planned again.  It must be uploaded again either way."""
    ki, kb, bl = _i32(kv_indptr), _i32(kv_blocks), _i32(block_len)
    flag = ctypes.c_int32(0)
    _check(lib().tkv_plan_update(plan, _ptr(ki), _ptr(kb) if len(kb) else None, _ptr(bl), ctypes.byref(flag)))
    return bool(flag.value)


def tkv_plan_dirty(plan: int):
    """(word indices the plan's in-place updates changed since its last upload, complete?)."""
    words, n, complete = _PI32(), ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().tkv_plan_dirty(plan, ctypes.byref(words), ctypes.byref(n), ctypes.byref(complete)))
    idx = np.ctypeslib.as_array(words, shape=(n.value,)).copy() if n.value else np.zeros(0, dtype=np.int32)
    return idx, bool(complete.value)


def tkv_plan_image(plan: int):
    """A copy of the plan's host descriptor image (what tkv_plan_upload copies) and the byte
    offsets of its sections: (bytes, dict)."""
    data, lay = _P(), tkv_plan_layout()
    _check(lib().tkv_plan_image(plan, ctypes.byref(data), ctypes.byref(lay)))
    layout = {f: int(getattr(lay, f)) for f, _ in tkv_plan_layout._fields_}
    return (ctypes.string_at(data.value, layout["end"]) if layout["end"] else b""), layout


def tkv_plan_get_stats(plan: int) -> dict:
    st = tkv_plan_stats()
    _check(lib().tkv_plan_get_stats(plan, ctypes.byref(st)))
    return {n: int(getattr(st, n)) for n, _ in tkv_plan_stats._fields_}


def tkv_plan_get_view(plan: int) -> dict:
    v = tkv_plan_view()
    _check(lib().tkv_plan_get_view(plan, ctypes.byref(v)))

    def arr(p, n, w):
        if n == 0:
            return np.zeros((0, w), dtype=np.int32)
        return np.ctypeslib.as_array(p, shape=(n * w,)).reshape(n, w).copy()
    return {"items": arr(v.items, v.n_items, 8), "toks": arr(v.toks, v.n_toks, 4), "blks": arr(v.blks, v.n_blks, 2),
            "merges": arr(v.merges, v.n_merge, 4),
            "merge_slots": arr(v.merge_slots, v.n_merge_slots, 1).reshape(-1), "n_slots": int(v.n_slots)}


def _attn(fn, plan, q, k, v, o, lse, stream):
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o)):
        if not (t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous()):
            raise TkvError(TKV_EINVAL, f"{name} must be a contiguous bfloat16 device tensor")
    if lse is not None and not (lse.is_cuda and lse.dtype == torch.float32 and lse.is_contiguous()):
        raise TkvError(TKV_EINVAL, "lse must be a contiguous float32 device tensor")
    _check(fn(plan, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
              None if lse is None else lse.data_ptr(), _stream(stream)))


def tkv_decode(plan: int, q, k, v, o, lse=None, stream=None) -> None:
    _attn(lib().tkv_decode, plan, q, k, v, o, lse, stream)


def tkv_verify(plan: int, q, k, v, o, lse=None, stream=None) -> None:
    _attn(lib().tkv_verify, plan, q, k, v, o, lse, stream)


def tkv_verify_noalloc(plan: int, q, k, v, o, lse=None, stream=None) -> None:
    """tkv_verify on the library's static workspace (the plan need not be uploaded)."""
    _attn(lib().tkv_verify_noalloc, plan, q, k, v, o, lse, stream)


def tkv_kv_append(dst: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                  stream=None) -> None:
    """Writes new tokens' K/V rows into the paged pool at their slots (dst int32, -1 = skip).
    k_new, v_new: [n_tok, hkv, d] bf16; k, v: [num_blocks, hkv, block_size, d] bf16 (all on the GPU)."""
    nb, hkv, bs, d = k.shape
    n = int(dst.numel())
    for t, shp in ((k_new, (n, hkv, d)), (v_new, (n, hkv, d)), (v, tuple(k.shape))):
        if tuple(t.shape) != shp or t.dtype != torch.bfloat16 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError(f"tkv_kv_append: expected a contiguous bf16 GPU tensor of shape {shp}, got {tuple(t.shape)}")
    if k.dtype != torch.bfloat16 or not k.is_contiguous() or not k.is_cuda:
        raise ValueError("tkv_kv_append: the pool must be a contiguous bf16 GPU tensor")
    if dst.dtype != torch.int32 or not dst.is_cuda or not dst.is_contiguous():
        raise ValueError("tkv_kv_append: dst must be a contiguous int32 GPU tensor")
    shape = tkv_shape(0, hkv, d, bs, nb)
    _check(lib().tkv_kv_append(ctypes.byref(shape), dst.data_ptr(), n, k_new.data_ptr(), v_new.data_ptr(),
                               k.data_ptr(), v.data_ptr(), _stream(stream)))


def tkv_cd_sample(logits: torch.Tensor, temperature: float, draw_off: torch.Tensor, uniform: torch.Tensor,
                  max_potential: int, stream=None):
    """Draws each row's potential-many tokens and groups them; returns device tensors
    (tokens, counts, n_groups): row r's groups at [draw_off[r], draw_off[r] + n_groups[r]).  A row
    whose draws fall outside `uniform` gets n_groups -1."""
    if logits.dim() != 2 or logits.dtype != torch.float32 or not logits.is_cuda or not logits.is_contiguous():
        raise ValueError("tkv_cd_sample: logits must be a contiguous float32 GPU tensor [n_rows, vocab]")
    n_rows, vocab = logits.shape
    if draw_off.dtype != torch.int32 or draw_off.numel() != n_rows + 1 or not draw_off.is_cuda:
        raise ValueError("tkv_cd_sample: draw_off must be an int32 GPU tensor of n_rows + 1 entries")
    if uniform.dtype != torch.float32 or not uniform.is_cuda or not uniform.is_contiguous():
        raise ValueError("tkv_cd_sample: uniform must be a contiguous float32 GPU tensor")
    n = max(1, int(uniform.numel()))
    tok = torch.empty(n, dtype=torch.int32, device=logits.device)
    cnt = torch.empty(n, dtype=torch.int32, device=logits.device)
    ng = torch.empty(max(1, n_rows), dtype=torch.int32, device=logits.device)
    _check(lib().tkv_cd_sample(n_rows, vocab, float(temperature), int(max_potential), logits.data_ptr(),
                               uniform.data_ptr(), draw_off.data_ptr(), int(uniform.numel()), tok.data_ptr(),
                               cnt.data_ptr(), ng.data_ptr(), _stream(stream)))
    return tok, cnt, ng[:n_rows]


def tkv_plan_profile(plan: int, max_calls: int) -> None:
    _check(lib().tkv_plan_profile(plan, max_calls))


def tkv_plan_profile_read(plan: int):
    """Returns (recorded calls, summed main-kernel ms, summed merge-kernel ms)."""
    n, a, b = _I32(), ctypes.c_float(), ctypes.c_float()
    _check(lib().tkv_plan_profile_read(plan, ctypes.byref(n), ctypes.byref(a), ctypes.byref(b)))
    return n.value, a.value, b.value


CAND_GENERATING, CAND_QUEUED, CAND_VERIFYING, CAND_VERIFIED, CAND_SELECTED, CAND_PRUNED = range(6)


def tkv_search_create(k: int, max_nodes: int, token_threshold: int, max_deferrals: int) -> int:
    h = _P()
    _check(lib().tkv_search_create(k, max_nodes, token_threshold, max_deferrals, ctypes.byref(h)))
    return h.value


def tkv_search_destroy(s: int) -> None:
    lib().tkv_search_destroy(s)


def tkv_search_expand(s: int, parent: int, n: int) -> int:
    first = _I32()
    _check(lib().tkv_search_expand(s, parent, n, ctypes.byref(first)))
    return first.value


def tkv_search_complete(s: int, node: int, n_tokens: int) -> bool:
    f = _I32()
    _check(lib().tkv_search_complete(s, node, n_tokens, ctypes.byref(f)))
    return bool(f.value)


def tkv_search_tick(s: int) -> bool:
    f = _I32()
    _check(lib().tkv_search_tick(s, ctypes.byref(f)))
    return bool(f.value)


def _take(fn, s: int) -> list:
    n = _I32()
    rc = fn(s, None, 0, ctypes.byref(n))
    if rc not in (TKV_OK, TKV_ECAP):
        _check(rc)
    out = np.zeros(max(1, n.value), dtype=np.int32)
    _check(fn(s, _ptr(out), len(out), ctypes.byref(n)))
    return [int(x) for x in out[:n.value]]


def tkv_search_flush(s: int) -> list:
    return _take(lib().tkv_search_flush, s)


def tkv_search_score(s: int, nodes, scores) -> None:
    nd = _i32(nodes)
    sc = np.ascontiguousarray(np.asarray(scores, dtype=np.float32).reshape(-1))
    if len(sc) != len(nd):
        raise ValueError("one score per node")
    _check(lib().tkv_search_score(s, len(nd), _ptr(nd), sc.ctypes.data_as(ctypes.POINTER(ctypes.c_float))))


def tkv_search_pruned(s: int) -> list:
    return _take(lib().tkv_search_pruned, s)


def tkv_search_node(s: int, node: int):
    """Returns (state, parent, depth, score or None)."""
    st, pa, de, sc = _I32(), _I32(), _I32(), ctypes.c_float()
    _check(lib().tkv_search_node(s, node, ctypes.byref(st), ctypes.byref(pa), ctypes.byref(de), ctypes.byref(sc)))
    return st.value, pa.value, de.value, (None if sc.value < 0 else sc.value)


def tkv_search_round(s: int, depth: int):
    """Returns (decided, selected ids ascending)."""
    n, dec = _I32(), _I32()
    rc = lib().tkv_search_round(s, depth, None, 0, ctypes.byref(n), ctypes.byref(dec))
    if rc not in (TKV_OK, TKV_ECAP):
        _check(rc)
    out = np.zeros(max(1, n.value), dtype=np.int32)
    _check(lib().tkv_search_round(s, depth, _ptr(out), len(out), ctypes.byref(n), ctypes.byref(dec)))
    return bool(dec.value), [int(x) for x in out[:n.value]]


def tkv_search_snapshot(s: int) -> dict:
    """Parsed state: nodes as (parent, depth, state, n_children, tokens, deferrals, arrival, score bits)."""
    used = ctypes.c_size_t()
    lib().tkv_search_snapshot(s, None, 0, ctypes.byref(used))
    buf = np.zeros(used.value // 4, dtype=np.int32)
    _check(lib().tkv_search_snapshot(s, buf.ctypes.data_as(_P), used.value, ctypes.byref(used)))
    w = [int(x) for x in buf]
    k, thr, md, n_roots, qtok, n = w[:6]
    i = 6
    nodes = [tuple(w[i + 8 * j:i + 8 * j + 8]) for j in range(n)]
    i += 8 * n
    nq = w[i]
    queue = w[i + 1:i + 1 + nq]
    i += 1 + nq
    rounds = []
    for _ in range(w[i]):
        i += 1
        dec, ns = w[i], w[i + 1]
        rounds.append((dec, tuple(w[i + 2:i + 2 + ns])))
        i += 1 + ns
    return {"k": k, "token_threshold": thr, "max_deferrals": md, "n_roots": n_roots, "queued_tokens": qtok,
            "nodes": nodes, "queue": queue, "rounds": rounds}


# ------------------------------------------------------------------------- owning wrappers

class BlockManager:
    """Owns a tkv_bm handle; methods forward to the C entry points."""

    def __init__(self, num_blocks: int, block_size: int = 16, max_seqs: int = 1024):
        self.num_blocks, self.block_size = num_blocks, block_size
        self.h = tkv_bm_create(num_blocks, block_size, max_seqs)

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            tkv_bm_destroy(self.h)
            self.h = None

    def extend(self, parent, tokens, seal):
        return tkv_bm_extend(self.h, parent, tokens, seal, self.block_size)

    def prune(self, seq):
        return tkv_prune(self.h, seq)

    def append(self, seq, tokens):
        return tkv_bm_append(self.h, seq, tokens)

    def seal(self, seq):
        return tkv_bm_seal(self.h, seq)

    def fork(self, seq, tokens):
        return tkv_bm_fork(self.h, seq, tokens)

    def table(self, seq):
        return tkv_bm_table(self.h, seq)[0]

    def block_len(self):
        return tkv_bm_block_len(self.h, self.num_blocks)

    def snapshot(self, seqs=True):
        return tkv_bm_snapshot(self.h, seqs)

    def coalesce(self, seqs, q_lens):
        return tkv_bm_coalesce(self.h, seqs, q_lens)


class Plan:
    """Owns a tkv_plan handle and the device workspace it was uploaded to."""

    def __init__(self, shape, q_indptr, kv_indptr, kv_blocks, block_len, multiplicity=None,
                 device="cuda", stream=None, upload=True, options=None):
        self.h = tkv_plan_create_ex(shape, q_indptr, kv_indptr, kv_blocks, block_len, multiplicity, options)
        self.workspace = None
        if upload:
            nbytes = tkv_plan_workspace_bytes(self.h)
            self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
            tkv_plan_upload(self.h, self.workspace, stream)

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            tkv_plan_destroy(self.h)
            self.h = None

    @property
    def stats(self):
        return tkv_plan_get_stats(self.h)

    def update(self, kv_indptr, kv_blocks, block_len, stream=None) -> bool:
        """tkv_plan_update, then (for an uploaded plan) the upload again, into a larger workspace
        if the plan now needs one.  Returns whether the plan was patched in place."""
        in_place = tkv_plan_update(self.h, kv_indptr, kv_blocks, block_len)
        if self.workspace is not None:
            nbytes = tkv_plan_workspace_bytes(self.h)
            if nbytes > self.workspace.numel():
                self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.workspace.device)
            tkv_plan_upload(self.h, self.workspace, stream)
        return in_place

    def image(self) -> bytes:
        return tkv_plan_image(self.h)

    def view(self):
        return tkv_plan_get_view(self.h)

    def decode(self, q, k, v, o, lse=None, stream=None):
        tkv_decode(self.h, q, k, v, o, lse, stream)

    def verify(self, q, k, v, o, lse=None, stream=None):
        tkv_verify(self.h, q, k, v, o, lse, stream)


class Search:
    """Owns a tkv_search handle (speculative beam-search controller); methods forward to the C
    entry points."""

    def __init__(self, k: int, max_nodes: int = 4096, token_threshold: int = 2048, max_deferrals: int = 6):
        self.h = tkv_search_create(k, max_nodes, token_threshold, max_deferrals)

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            tkv_search_destroy(self.h)
            self.h = None

    def expand(self, parent, n):
        return tkv_search_expand(self.h, parent, n)

    def complete(self, node, n_tokens):
        return tkv_search_complete(self.h, node, n_tokens)

    def tick(self):
        return tkv_search_tick(self.h)

    def flush(self):
        return tkv_search_flush(self.h)

    def score(self, nodes, scores):
        tkv_search_score(self.h, nodes, scores)

    def pruned(self):
        return tkv_search_pruned(self.h)

    def node(self, node):
        return tkv_search_node(self.h, node)

    def round(self, depth):
        return tkv_search_round(self.h, depth)

    def snapshot(self):
        return tkv_search_snapshot(self.h)
