"""GPU: a multi-layer decode step (paper_2609_39334_amd.model) against a float64 CPU reference.

The reference runs the same synthetic model on the host: float64 arithmetic, the oracle's attention
over the same pools, and bf16 rounding at the points where the device path rounds (GEMM outputs,
RoPE outputs, attention output, norm outputs).  What remains is fp32 (in the BLAS's own summation
order) against float64 accumulation: a GEMM output near a bf16 rounding boundary lands on the
neighbouring bf16 value, one ulp (2^-8 relative) away, and such flips propagate.  The final logits
are themselves rounded to bf16, so about half of them sit one ulp off.  Bars: the largest difference
within 2% of the largest logit magnitude, the mean within 1% of the mean magnitude (~2.5 ulp).
Every new token's pool slot starts as NaN and every padding slot is NaN, so a missing K/V write, a
wrong slot or table, or a read past a block's length shows as NaN; a wrong RoPE position or layer
pool shows as an O(1) difference.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


def _bf(x):
    return W.bf16_bits_to_f32(W.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))).astype(np.float64)


def _np(t):
    return t.float().cpu().numpy().astype(np.float64)


def _reference(model, tokens, positions, dst, tables, block_len, kpools, vpools):
    s = model.shape
    half = s.d // 2
    nq, nk = s.hq * s.d, s.hkv * s.d
    rows = len(tokens)
    inv = s.rope_theta ** (-np.arange(half, dtype=np.float64) * 2.0 / s.d)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]
    cos, sin = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]

    def rms(x, w):
        return _bf(x / np.sqrt((x * x).mean(-1, keepdims=True) + s.eps) * _np(w))

    def rope(t):
        x1, x2 = t[..., :half], t[..., half:]
        return _bf(np.concatenate((x1 * cos - x2 * sin, x2 * cos + x1 * sin), axis=-1))

    x = _np(model.embed)[np.asarray(tokens)]
    for li, w in enumerate(model.layers):
        qkv = _bf(rms(x, w["ln1"]) @ _np(w["wqkv"]))
        q = rope(qkv[:, :nq].reshape(rows, s.hq, s.d))
        k = rope(qkv[:, nq:nq + nk].reshape(rows, s.hkv, s.d))
        v = qkv[:, nq + nk:].reshape(rows, s.hkv, s.d)
        for r, slot in enumerate(dst):
            kpools[li][slot // 16, :, slot % 16, :] = k[r]
            vpools[li][slot // 16, :, slot % 16, :] = v[r]
        o, _ = oracle.attention(q, kpools[li], vpools[li], tables, block_len, [1] * rows)
        x = x + _bf(_bf(o).reshape(rows, nq) @ _np(w["wo"]))
        gu = _bf(rms(x, w["ln2"]) @ _np(w["wgu"]))
        a = _bf(gu[:, :s.inter] / (1.0 + np.exp(-gu[:, :s.inter])) * gu[:, s.inter:])
        x = x + _bf(a @ _np(w["wd"]))
    return _bf(rms(x, model.lnf) @ _np(model.lm))


@pytest.mark.parametrize("seed,layers,hq,hkv,d", [(0, 2, 4, 2, 64), (1, 3, 8, 2, 128)])
def test_decoder_step_matches_reference(seed, layers, hq, hkv, d):
    import paper_2609_39334_amd as tkv
    from paper_2609_39334_amd.model import DecoderShape, SyntheticDecoder
    shape = DecoderShape(layers=layers, hidden=256, hq=hq, hkv=hkv, d=d, inter=512, vocab=1000)
    rng = np.random.default_rng(seed)
    nb, bs = 256, 16
    bm = tkv.BlockManager(nb, bs, 64)
    root = bm.extend(-1, rng.integers(0, 1000, 37).tolist(), True)[0]
    kids = [bm.extend(root, rng.integers(0, 1000, 20).tolist(), True)[0] for _ in range(3)]
    cands = [bm.extend(kd, rng.integers(0, 1000, int(rng.integers(5, 31))).tolist(), False)[0]
             for kd in kids for _ in range(2)]
    tokens = rng.integers(0, shape.vocab, len(cands))
    dst = np.array([int(bm.append(c, [int(t)])[0]) for c, t in zip(cands, tokens)], dtype=np.int32)
    tables = [[int(b) for b in bm.table(c)] for c in cands]
    block_len = bm.block_len()
    positions = np.array([sum(block_len[b] for b in t) - 1 for t in tables], dtype=np.int64)
    rows = len(cands)
    qi = np.arange(rows + 1, dtype=np.int32)
    ki = np.concatenate([[0], np.cumsum([len(t) for t in tables])]).astype(np.int32)
    plan = tkv.Plan((hq, hkv, d, bs, nb), qi, ki, np.concatenate(tables).astype(np.int32), block_len, None)

    kbits, vbits = [], []
    for _ in range(layers):
        kv = W.f32_to_bf16_bits(rng.standard_normal((2, nb, hkv, bs, d)).astype(np.float32))
        k, v = kv[0].copy(), kv[1].copy()
        W.poison_padding(k, v, block_len)
        for slot in dst:                                  # the new tokens' K/V: written by the step
            k[slot // bs, :, slot % bs, :] = W.BF16_NAN
            v[slot // bs, :, slot % bs, :] = W.BF16_NAN
        kbits.append(k)
        vbits.append(v)

    def dev(b):
        return torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).view(torch.bfloat16).cuda()

    model = SyntheticDecoder(shape, "cuda", seed)
    k_pools, v_pools = [dev(b) for b in kbits], [dev(b) for b in vbits]
    logits = model.step(torch.from_numpy(tokens).cuda(), torch.from_numpy(positions).cuda(),
                        torch.from_numpy(dst).cuda(), plan, k_pools, v_pools)
    torch.cuda.synchronize()
    got = logits.cpu().numpy().astype(np.float64)
    want = _reference(model, tokens, positions, dst, tables, block_len,
                      [W.bf16_bits_to_f32(b).astype(np.float64) for b in kbits],
                      [W.bf16_bits_to_f32(b).astype(np.float64) for b in vbits])
    err = np.abs(got - want)
    print(f"    decoder {layers} layers, {rows} rows: max {err.max():.3e} (|ref| max {np.abs(want).max():.2f}), "
          f"mean {err.mean():.3e}", flush=True)
    assert np.isfinite(got).all()
    assert err.max() <= 2e-2 * np.abs(want).max() and err.mean() <= 1e-2 * np.abs(want).mean()
    # the step wrote every new token's K/V into every layer's pool
    for li in range(layers):
        kl = k_pools[li].view(torch.int16).cpu().numpy()
        assert not (kl[dst // bs, :, dst % bs, :].view(np.uint16) == W.BF16_NAN).any()
