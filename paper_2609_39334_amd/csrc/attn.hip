// Tree-shared paged attention kernels for gfx950 (MI355X).
//
// Every work item contracts a tile of query rows -- query tokens x the G query heads of one KV
// head -- against an ordered list of 16-token K/V blocks on bf16 MFMA with fp32 accumulation,
// computing the transposed products so that each lane keeps one query row throughout:
//   S^T = K Q^T     v_mfma_f32_16x16x32_bf16 (A = 16 keys x 32 dims, B = Q^T held in registers),
//   O^T += V^T P^T  v_mfma_f32_16x16x32_bf16 over two blocks at a time (A = V^T of both blocks read
//                   transposed from LDS with ds_read_b64_tr_b16, B = P^T exactly as the two S^T
//                   results sit in the lanes),
// with an online softmax in between (exp2 with the scale folded into one FMA; the exponent base of
// a row moves only when its maximum grows by more than 2^8, so O is rarely rescaled).  Keys past a
// block's length are never loaded (row reads are clamped to the block's last token and masked) and
// keys past a token's causal limit get -inf.
//
// attn_fwd runs two kinds of work items in one launch:
// wave grid:  decode-shaped work (G <= 16, chunks of at most kWaveMaxRows rows): every wave is an
//             independent worker walking its own list of items, each a tile of up to 32 rows over a
//             chunk of <= 16 blocks, with the next two blocks always in flight; no LDS sharing
//             between waves, no barriers.
// tile items: wide tiles (multi-token verify rows, wide shared chunks, G > 16): one workgroup of
//             four waves per item, 128 rows (32 per wave) against 64-key stages of K/V
//             double-buffered through LDS.
// merge_partials: log-sum-exp merge of the partial results of a query token's chunks:
//             lse = log sum_j exp(lse_j),  o = sum_j exp(lse_j - lse) o_j.

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <mutex>
#include "internal.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8_t, u); }

__device__ __forceinline__ f32x4_t mfma_16x16x32(bf16x8_t a, bf16x8_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> packed fp16 pair, round to nearest even (the partial results' storage type).
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, f16x2_t));
}

__device__ __forceinline__ float4 unpack_f16x4(uint2 u) {
    const f32x2_t a = __builtin_convertvector(__builtin_bit_cast(f16x2_t, u.x), f32x2_t);
    const f32x2_t b = __builtin_convertvector(__builtin_bit_cast(f16x2_t, u.y), f32x2_t);
    return make_float4(a[0], a[1], b[0], b[1]);
}

// acc + lo + hi of a packed bf16 pair, in fp32 (v_dot2_f32_bf16 against the pair (1, 1)).
__device__ __forceinline__ float sum_bf16x2(uint32_t p, float acc) {
    const bf16x2_t one{static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, p), one, acc, false);
}

constexpr int kThreads = 256;

// ============================================================================ wave-private kernel
// For tiles of at most 16 query rows (decode rows: the G heads of a few tokens) every wave is an
// independent worker with its own item: no LDS sharing, no barriers; latency is covered by the
// dozen independent waves resident per CU.  Per 16-key block:
//   S^T = K Q^T   on v_mfma_f32_16x16x32_bf16: K comes from HBM straight into the A operand
//                 (lane = key, 16 contiguous bytes of its row per k-step), Q^T held in registers;
//   online softmax on the four scores per lane (row max over the 4 lanes of a row by
//                 v_permlane16/32_swap);
//   O^T += V^T P^T on v_mfma_f32_16x16x16_bf16: P^T is the S^T result as it sits in the lanes;
//                 V is written row-major to the wave's LDS and read back transposed with
//                 ds_read_b64_tr_b16 (lane j of a 16-lane group addresses row 4kg + j/4, column
//                 16ct + 4(j%4); lane i receives V[4kg + e][16ct + i], e = 0..3).
// The next two blocks' K/V loads are in flight while a block is contracted.
typedef short s16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float rowmax4(float x) {  // max over lanes l, l^16, l^32, l^48
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(x, fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1])));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(x, fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1])));
}

template <int D>
struct BlockRegs {
    u32x4_t k[D / 32];  // K[key = lane%16][32ks + 8kg .. +7]
    u32x4_t v[D / 32];  // V chunks c = lane + 64i: key c / (D/8), dims 8(c % (D/8)) .. +7
};

// len = 0 (a block past the item's end) reads row 0 of the block: the fetch is harmless.
template <int D>
__device__ __forceinline__ void load_k(BlockRegs<D>& r, const uint16_t* __restrict__ kpool, size_t boff, int len,
                                       int lane) {
    const int kse = min(lane & 15, max(len - 1, 0));
    const uint16_t* krow = kpool + boff + kse * D + (lane >> 4) * 8;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) r.k[ks] = *reinterpret_cast<const u32x4_t*>(krow + ks * 32);
}
template <int D>
__device__ __forceinline__ void load_v(BlockRegs<D>& r, const uint16_t* __restrict__ vpool, size_t boff, int len,
                                       int lane) {
    const int last = max(len - 1, 0);
#pragma unroll
    for (int i = 0; i < D / 32; ++i) {
        const int c = lane + 64 * i;
        r.v[i] = *reinterpret_cast<const u32x4_t*>(vpool + boff + min(c / (D / 8), last) * D + (c % (D / 8)) * 8);
    }
}

// Running softmax state and output accumulators of a wave's T column tiles of 16 query rows
// (O^T: lane holds columns 16ct + 4kg + r of row lane%16 of each tile).
template <int D, int T>
struct WaveAcc {
    f32x4_t acc[T][D / 16];
    float m[T], l[T];
    __device__ __forceinline__ void reset() {
#pragma unroll
        for (int tt = 0; tt < T; ++tt) {
#pragma unroll
            for (int c = 0; c < D / 16; ++c) acc[tt][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            m[tt] = -INFINITY;
            l[tt] = 0.f;
        }
    }
};

// Online-softmax update of T column tiles with one 16-key block of scores (lane holds keys
// 4kg + x of its row): mask keys past the block's length or the row's causal limit, fold the block
// into the running max / sum, rescale O when a row's max moved, and pack P^T as bf16 for the PV MFMA.
template <int D, int T>
__device__ __forceinline__ void softmax_step(WaveAcc<D, T>& A, f32x4_t (&s)[T], int len, int pos,
                                             const int (&limit)[T], int kg, float sl2, s16x4_t (&pb)[T]) {
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        // mask only partial blocks and rows with a causal limit inside the block
        if (__builtin_amdgcn_ballot_w64(!(len == 16 && limit[tt] >= pos + 15)) != 0) {
            const int vlen = min(len, limit[tt] - pos + 1);
#pragma unroll
            for (int x = 0; x < 4; ++x)
                if (4 * kg + x >= vlen) s[tt][x] = -INFINITY;
        }
        const float mx = rowmax4(fmaxf(fmaxf(s[tt][0], s[tt][1]), fmaxf(s[tt][2], s[tt][3])));
        const float m_new = fmaxf(A.m[tt], mx);
        const float msc = m_new == -INFINITY ? 0.f : m_new * sl2;
        float psum = 0.f;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            s[tt][x] = __builtin_amdgcn_exp2f(fmaf(s[tt][x], sl2, -msc));
            psum += s[tt][x];
        }
        const float alpha = m_new == A.m[tt] ? 1.f : __builtin_amdgcn_exp2f(A.m[tt] * sl2 - msc);
        A.l[tt] = fmaf(A.l[tt], alpha, psum);
        A.m[tt] = m_new;
        if (__builtin_amdgcn_ballot_w64(alpha != 1.f) != 0) {
#pragma unroll
            for (int c = 0; c < D / 16; ++c) A.acc[tt][c] *= alpha;
        }
        pb[tt] = __builtin_bit_cast(s16x4_t, uint2{pack_bf16x2(s[tt][0], s[tt][1]), pack_bf16x2(s[tt][2], s[tt][3])});
    }
}

// The same update for a pair of 16-key blocks (A then B) folded in as one 32-key step; P^T comes
// out as the B operand of v_mfma_f32_16x16x32_bf16 with k = 8kg + e holding key 4kg + e of block A
// (e < 4) and key 4kg + e - 4 of block B (e >= 4) -- the order of the V^T operand built from the
// two blocks' transposed LDS reads.
template <int D, int T>
__device__ __forceinline__ void softmax_pair(WaveAcc<D, T>& A, f32x4_t (&sa)[T], f32x4_t (&sb)[T], int len_a,
                                             int pos_a, int len_b, int pos_b, const int (&limit)[T], int kg,
                                             float sl2, bf16x8_t (&pb)[T]) {
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        if (__builtin_amdgcn_ballot_w64(!(len_a == 16 && limit[tt] >= pos_a + 15)) != 0) {
            const int vlen = min(len_a, limit[tt] - pos_a + 1);
#pragma unroll
            for (int x = 0; x < 4; ++x)
                if (4 * kg + x >= vlen) sa[tt][x] = -INFINITY;
        }
        if (__builtin_amdgcn_ballot_w64(!(len_b == 16 && limit[tt] >= pos_b + 15)) != 0) {
            const int vlen = min(len_b, limit[tt] - pos_b + 1);
#pragma unroll
            for (int x = 0; x < 4; ++x)
                if (4 * kg + x >= vlen) sb[tt][x] = -INFINITY;
        }
        const float mx = rowmax4(fmaxf(fmaxf(fmaxf(sa[tt][0], sa[tt][1]), fmaxf(sa[tt][2], sa[tt][3])),
                                       fmaxf(fmaxf(sb[tt][0], sb[tt][1]), fmaxf(sb[tt][2], sb[tt][3]))));
        const float m_new = fmaxf(A.m[tt], mx);
        const float msc = m_new == -INFINITY ? 0.f : m_new * sl2;
        float psum = 0.f;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            sa[tt][x] = __builtin_amdgcn_exp2f(fmaf(sa[tt][x], sl2, -msc));
            sb[tt][x] = __builtin_amdgcn_exp2f(fmaf(sb[tt][x], sl2, -msc));
            psum += sa[tt][x] + sb[tt][x];
        }
        const float alpha = m_new == A.m[tt] ? 1.f : __builtin_amdgcn_exp2f(A.m[tt] * sl2 - msc);
        A.l[tt] = fmaf(A.l[tt], alpha, psum);
        A.m[tt] = m_new;
        if (__builtin_amdgcn_ballot_w64(alpha != 1.f) != 0) {
#pragma unroll
            for (int c = 0; c < D / 16; ++c) A.acc[tt][c] *= alpha;
        }
        pb[tt] = __builtin_bit_cast(bf16x8_t, uint4{pack_bf16x2(sa[tt][0], sa[tt][1]), pack_bf16x2(sa[tt][2], sa[tt][3]),
                                                    pack_bf16x2(sb[tt][0], sb[tt][1]), pack_bf16x2(sb[tt][2], sb[tt][3])});
    }
}

// Mask the scores of one 16-key block for T column tiles (lane holds keys 4kg + x of its row):
// keys past the block's length or past the row's causal limit get -inf; full, visible blocks skip it.
template <int T>
__device__ __forceinline__ void mask_block(f32x4_t (&s)[T], int len, int pos, const int (&limit)[T], int kg) {
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        if (__builtin_amdgcn_ballot_w64(!(len == 16 && limit[tt] >= pos + 15)) != 0) {
            const int vlen = min(len, limit[tt] - pos + 1);
#pragma unroll
            for (int x = 0; x < 4; ++x)
                if (4 * kg + x >= vlen) s[tt][x] = -INFINITY;
        }
    }
}

// Online softmax over a pair of already-masked 16-key blocks with a lazily moved exponent base: the
// base m (per row) only moves when a row's new maximum exceeds it by more than 2^8 in probability
// scale, so O and l are rescaled rarely; P = exp2((s - m) * scale) then stays below 2^8, well
// inside fp32 / bf16 range, and the result is exact up to rounding for any base (the lse adds m
// back).  P^T is packed as in softmax_pair.
template <int D, int T>
__device__ __forceinline__ void softmax_pair_lazy(WaveAcc<D, T>& A, f32x4_t (&sa)[T], f32x4_t (&sb)[T], float sl2,
                                                  bf16x8_t (&pb)[T]) {
    constexpr float kSlack = 8.f;  // log2 of the largest P allowed before the base moves
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        const float mx = rowmax4(fmaxf(fmaxf(fmaxf(sa[tt][0], sa[tt][1]), fmaxf(sa[tt][2], sa[tt][3])),
                                       fmaxf(fmaxf(sb[tt][0], sb[tt][1]), fmaxf(sb[tt][2], sb[tt][3]))));
        if (__builtin_amdgcn_ballot_w64(mx > A.m[tt] + kSlack / sl2) != 0) {  // false for mx = -inf; true for m = -inf < mx
            const float m_new = fmaxf(A.m[tt], mx);
            const float alpha = A.m[tt] == m_new ? 1.f : __builtin_amdgcn_exp2f((A.m[tt] - m_new) * sl2);
            A.l[tt] *= alpha;
#pragma unroll
            for (int c = 0; c < D / 16; ++c) A.acc[tt][c] *= alpha;
            A.m[tt] = m_new;
        }
        const float msc = A.m[tt] == -INFINITY ? 0.f : A.m[tt] * sl2;
        float psum = 0.f;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            sa[tt][x] = __builtin_amdgcn_exp2f(fmaf(sa[tt][x], sl2, -msc));
            sb[tt][x] = __builtin_amdgcn_exp2f(fmaf(sb[tt][x], sl2, -msc));
            psum += sa[tt][x] + sb[tt][x];
        }
        A.l[tt] += psum;
        pb[tt] = __builtin_bit_cast(bf16x8_t, uint4{pack_bf16x2(sa[tt][0], sa[tt][1]), pack_bf16x2(sa[tt][2], sa[tt][3]),
                                                    pack_bf16x2(sb[tt][0], sb[tt][1]), pack_bf16x2(sb[tt][2], sb[tt][3])});
    }
}

// The lazily moved exponent base for a whole 64-key stage (four blocks of already-masked scores):
// a row's base moves only when the stage's maximum exceeds it by more than 2^8 in probability
// scale (then O and l are rescaled), as in softmax_pair_lazy.
template <int D, int T>
__device__ __forceinline__ void stage_base(WaveAcc<D, T>& A, const f32x4_t (&sc)[4][T], float sl2) {
    constexpr float kSlack = 8.f;
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        // each lane tests its own 16 scores against the base; the row maximum over the four lanes
        // of a row is taken only when some lane needs the base moved (the four lanes of a row hold
        // the same base, so a row needs a move exactly when one of its lanes does)
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < 4; ++j) mx = fmaxf(mx, fmaxf(fmaxf(sc[j][tt][0], sc[j][tt][1]), fmaxf(sc[j][tt][2], sc[j][tt][3])));
        if (__builtin_amdgcn_ballot_w64(mx > A.m[tt] + kSlack / sl2) != 0) {  // false for mx = -inf; true for m = -inf < mx
            mx = rowmax4(mx);
            const float m_new = fmaxf(A.m[tt], mx);
            const float alpha = A.m[tt] == m_new ? 1.f : __builtin_amdgcn_exp2f((A.m[tt] - m_new) * sl2);
            A.l[tt] *= alpha;
#pragma unroll
            for (int c = 0; c < D / 16; ++c) A.acc[tt][c] *= alpha;
            A.m[tt] = m_new;
        }
    }
}

// Normalise one column tile's rows and write them: the final bf16 output and lse (slot < 0) or an
// fp16 partial and its fp32 lse.  Lane holds columns 16ct + 4kg + r of its row; l is summed over the
// four lanes of the row.
template <int D>
__device__ __forceinline__ void write_rows(const f32x4_t (&acc)[D / 16], float m, float l, bool ok, int qtok, int h,
                                           int slot, int kg, uint16_t* __restrict__ o, float* __restrict__ lse,
                                           uint16_t* __restrict__ po, float* __restrict__ plse, int hq, float sl2) {
    float l_tot = l + __shfl_xor(l, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (!ok) return;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse_v = l_tot > 0.f ? (m * sl2 + log2f(l_tot)) * 0.6931471805599453f : -INFINITY;
    if (slot < 0) {
        uint16_t* orow = o + (static_cast<size_t>(qtok) * hq + h) * D;
#pragma unroll
        for (int ct = 0; ct < D / 16; ++ct) {
            uint2 wv;
            wv.x = pack_bf16x2(acc[ct][0] * inv, acc[ct][1] * inv);
            wv.y = pack_bf16x2(acc[ct][2] * inv, acc[ct][3] * inv);
            *reinterpret_cast<uint2*>(orow + ct * 16 + kg * 4) = wv;
        }
        if (lse && kg == 0) lse[static_cast<size_t>(qtok) * hq + h] = lse_v;
    } else {
        uint16_t* prow = po + (static_cast<size_t>(slot) * hq + h) * D;
#pragma unroll
        for (int ct = 0; ct < D / 16; ++ct) {
            uint2 wv;
            wv.x = pack_f16x2(acc[ct][0] * inv, acc[ct][1] * inv);
            wv.y = pack_f16x2(acc[ct][2] * inv, acc[ct][3] * inv);
            *reinterpret_cast<uint2*>(prow + ct * 16 + kg * 4) = wv;
        }
        if (kg == 0) plse[static_cast<size_t>(slot) * hq + h] = lse_v;
    }
}

// 16-byte words of a wave item's record (see tkv::WaveDesc): lane l loads word l % kRecWords, so
// lanes 0-31 hold the record (the upper lanes repeat it and are never read).
constexpr int kRecWords = static_cast<int>(sizeof(tkv::WaveDesc) / 16);
static_assert(kRecWords == 32 && kRecWords == tkv::kWaveBlocks + tkv::kWaveToks, "record layout");

// The item fields a wave needs, decoded from its descriptor (see tkv::WaveDesc): uniform values
// by v_readlane, this lane's token of each tile by ds_bpermute from the token lanes.
template <int T>
struct WaveItem {
    int kvh, n_tok, nb;
    int qtok[T], limit[T], slot[T], h[T];
    bool ok[T];
};

template <int T>
__device__ __forceinline__ WaveItem<T> wave_item(int4 d, const int (&tok)[T], const int (&grp)[T], int G) {
    WaveItem<T> w;
    w.kvh = __builtin_amdgcn_readlane(d.w, 0);
    w.n_tok = __builtin_amdgcn_readlane(d.w, 1);
    w.nb = __builtin_amdgcn_readlane(d.w, 2);
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        const int src = (16 + tok[tt]) * 4;
        w.qtok[tt] = __builtin_amdgcn_ds_bpermute(src, d.x);
        w.limit[tt] = __builtin_amdgcn_ds_bpermute(src, d.y);
        w.slot[tt] = __builtin_amdgcn_ds_bpermute(src, d.z);
        w.ok[tt] = tok[tt] < w.n_tok;
        w.h[tt] = w.kvh * G + grp[tt];
    }
    return w;
}

// This lane's row of each column tile: token index within the tile and query head within the group.
template <int T>
__device__ __forceinline__ void tile_rows(int col, int G, int (&tok)[T], int (&grp)[T]) {
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        const int row = 16 * tt + col;
        tok[tt] = min(row / G, tkv::kWaveToks - 1);
        grp[tt] = row - (row / G) * G;
    }
}

// Only the causal limits stay live across an item's block loop; the output fields are decoded
// again from the descriptor when the item is written.
template <int T>
__device__ __forceinline__ void tile_limits(int4 d, int col, int G, int (&limit)[T]) {
    int tok[T], grp[T];
    tile_rows<T>(col, G, tok, grp);
    const int n_tok = __builtin_amdgcn_readlane(d.w, 1);
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        const int lim = __builtin_amdgcn_ds_bpermute((16 + tok[tt]) * 4, d.y);
        limit[tt] = (16 * tt + col) / G < n_tok ? lim : -1;
    }
}

template <int D, int T>
__device__ __forceinline__ void load_q(bf16x8_t (&qf)[T][D / 32], const uint16_t* __restrict__ q,
                                       const WaveItem<T>& w, int hq, int kg) {
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        const uint16_t* qrow = q + (static_cast<size_t>(w.qtok[tt]) * hq + w.h[tt]) * D + kg * 8;
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) qf[tt][ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qrow + ks * 32));
    }
}

// A wave's list of items: record `first` (= the wave's index), then records rest, rest + 1, ...,
// n items in all.
struct WaveList {
    int first, rest, n;
    __device__ __forceinline__ int at(int k) const { return k == 0 ? first : rest + min(k, n - 1) - 1; }
};

// The same walk for T <= 2, two blocks at a time: two register sets hold a pair of K/V blocks, and
// the next pair's loads (across item boundaries too; every item has an even block count) are in
// flight while the current pair is contracted; the pair goes through one 32-key online-softmax
// step with a lazily moved base and through PV on v_mfma_f32_16x16x32_bf16.
template <int D, int T>
__device__ __forceinline__ void wave_run_pair(const int4* __restrict__ wdesc, const WaveList& L,
                                              const uint16_t* __restrict__ q, const uint16_t* __restrict__ kpool,
                                              const uint16_t* __restrict__ vpool, uint16_t* __restrict__ o,
                                              float* __restrict__ lse, uint16_t* __restrict__ po,
                                              float* __restrict__ plse, int hq, int hkv, int G, float sl2,
                                              uint8_t* vs, int lane) {
    constexpr int VROW = 2 * D + 32;
    const int col = lane & 15, kg = lane >> 4;
    const size_t blk_stride = static_cast<size_t>(hkv) * (16 * D);
    const uint8_t* vra = vs + (4 * kg + (col >> 2)) * VROW + (4 * (col & 3)) * 2;
    const uint8_t* vrb = vra + 16 * VROW;

    int4 dc = wdesc[static_cast<size_t>(L.at(0)) * kRecWords + (lane & (kRecWords - 1))];
    int4 dn = wdesc[static_cast<size_t>(L.at(1)) * kRecWords + (lane & (kRecWords - 1))];
    bf16x8_t qf[T][D / 32];
    int kvh_c, nb_c, limit[T];
    {
        int tok[T], grp[T];
        tile_rows<T>(col, G, tok, grp);
        const WaveItem<T> ic = wave_item<T>(dc, tok, grp, G);
        load_q<D, T>(qf, q, ic, hq, kg);
        kvh_c = ic.kvh;
        nb_c = ic.nb;
    }
    tile_limits<T>(dc, col, G, limit);
    BlockRegs<D> ra, rb;
    {
        const size_t kvh_off = static_cast<size_t>(kvh_c) * (16 * D);
        const int len0 = __builtin_amdgcn_readlane(dc.y, 0), len1 = __builtin_amdgcn_readlane(dc.y, 1);
        const size_t b0 = static_cast<size_t>(__builtin_amdgcn_readlane(dc.x, 0)) * blk_stride + kvh_off;
        const size_t b1 = static_cast<size_t>(__builtin_amdgcn_readlane(dc.x, 1)) * blk_stride + kvh_off;
        load_k<D>(ra, kpool, b0, len0, lane);
        load_v<D>(ra, vpool, b0, len0, lane);
        load_k<D>(rb, kpool, b1, len1, lane);
        load_v<D>(rb, vpool, b1, len1, lane);
    }
    WaveAcc<D, T> A;
    for (int e = 0;; ++e) {
        const bool more = e + 1 < L.n;
        const size_t kvh_off = static_cast<size_t>(kvh_c) * (16 * D);
        const size_t kvh_off_n = static_cast<size_t>(__builtin_amdgcn_readlane(dn.w, 0)) * (16 * D);
        A.reset();
        const int nb = nb_c;  // even
        for (int b = 0; b < nb; b += 2) {
            // the next pair: blocks b + 2, b + 3 of this item, or blocks 0, 1 of the next item
            const bool cross = b + 2 >= nb;
            const int bn = cross ? 0 : b + 2;
            const int src_x = cross ? dn.x : dc.x;
            const int src_y = cross ? (more ? dn.y : 0) : dc.y;
            const size_t off_n = cross ? kvh_off_n : kvh_off;
            const size_t boff_na = static_cast<size_t>(__builtin_amdgcn_readlane(src_x, bn)) * blk_stride + off_n;
            const size_t boff_nb = static_cast<size_t>(__builtin_amdgcn_readlane(src_x, bn + 1)) * blk_stride + off_n;
            const int len_na = __builtin_amdgcn_readlane(src_y, bn), len_nb = __builtin_amdgcn_readlane(src_y, bn + 1);
            const int len_a = __builtin_amdgcn_readlane(dc.y, b), len_b = __builtin_amdgcn_readlane(dc.y, b + 1);
            const int pos_a = __builtin_amdgcn_readlane(dc.z, b), pos_b = __builtin_amdgcn_readlane(dc.z, b + 1);
            // S^T for both blocks, then the K registers take the next pair
            f32x4_t sa[T], sb[T];
#pragma unroll
            for (int tt = 0; tt < T; ++tt) {
                sa[tt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
                sb[tt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int ks = 0; ks < D / 32; ++ks)
#pragma unroll
                for (int tt = 0; tt < T; ++tt) {
                    sa[tt] = mfma_16x16x32(__builtin_bit_cast(bf16x8_t, ra.k[ks]), qf[tt][ks], sa[tt]);
                    sb[tt] = mfma_16x16x32(__builtin_bit_cast(bf16x8_t, rb.k[ks]), qf[tt][ks], sb[tt]);
                }
            load_k<D>(ra, kpool, boff_na, len_na, lane);
            load_k<D>(rb, kpool, boff_nb, len_nb, lane);
            mask_block<T>(sa, len_a, pos_a, limit, kg);
            mask_block<T>(sb, len_b, pos_b, limit, kg);
            bf16x8_t pb[T];
            softmax_pair_lazy<D, T>(A, sa, sb, sl2, pb);
            // both blocks' V rows into this wave's LDS region, then the V registers take the next pair
#pragma unroll
            for (int i = 0; i < D / 32; ++i) {
                const int c = lane + 64 * i;
                *reinterpret_cast<u32x4_t*>(vs + (c / (D / 8)) * VROW + (c % (D / 8)) * 16) = ra.v[i];
                *reinterpret_cast<u32x4_t*>(vs + (16 + c / (D / 8)) * VROW + (c % (D / 8)) * 16) = rb.v[i];
            }
            load_v<D>(ra, vpool, boff_na, len_na, lane);
            load_v<D>(rb, vpool, boff_nb, len_nb, lane);
            // O^T += V^T P^T over the 32 keys: V^T from the two blocks' transposed LDS reads
#pragma unroll
            for (int ct = 0; ct < D / 16; ++ct) {
                const s16x4_t va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4_t*)(const_cast<uint8_t*>(vra + ct * 32)));
                const s16x4_t vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4_t*)(const_cast<uint8_t*>(vrb + ct * 32)));
                const bf16x8_t vab = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(va, vb, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
                for (int tt = 0; tt < T; ++tt) A.acc[tt][ct] = mfma_16x16x32(vab, pb[tt], A.acc[tt][ct]);
            }
        }
        {
            int tok[T], grp[T];
            tile_rows<T>(col, G, tok, grp);
            const WaveItem<T> ic = wave_item<T>(dc, tok, grp, G);
#pragma unroll
            for (int tt = 0; tt < T; ++tt)
                write_rows<D>(A.acc[tt], A.m[tt], A.l[tt], ic.ok[tt], ic.qtok[tt], ic.h[tt], ic.slot[tt], kg, o, lse,
                              po, plse, hq, sl2);
        }
        if (!more) break;
        dc = dn;
        dn = wdesc[static_cast<size_t>(L.at(e + 2)) * kRecWords + (lane & (kRecWords - 1))];
        {
            int tok[T], grp[T];
            tile_rows<T>(col, G, tok, grp);
            const WaveItem<T> ic = wave_item<T>(dc, tok, grp, G);
            load_q<D, T>(qf, q, ic, hq, kg);
            kvh_c = ic.kvh;
            nb_c = ic.nb;
        }
        tile_limits<T>(dc, col, G, limit);
    }
}

// Wave-kernel worker: wave w of the wave grid walks its own list of items with no barrier; its tile
// width T (1 or 2 column tiles of 16 query rows) is fixed per wave by the planner.
template <int D>
__device__ __forceinline__ void wave_worker(int w, int lane, const int4* __restrict__ wdesc,
                                            const int32_t* __restrict__ woff, const int32_t* __restrict__ wtiles,
                                            const uint16_t* __restrict__ q, const uint16_t* __restrict__ kpool,
                                            const uint16_t* __restrict__ vpool, uint16_t* __restrict__ o,
                                            float* __restrict__ lse, uint16_t* __restrict__ po, float* __restrict__ plse,
                                            int hq, int hkv, int G, float sl2, uint8_t* vs) {
    const int T = wtiles[w];
    if (T == 0) return;
    const WaveList L{w, woff[w], woff[w + 1] - woff[w] + 1};
    if (T == 1)
        wave_run_pair<D, 1>(wdesc, L, q, kpool, vpool, o, lse, po, plse, hq, hkv, G, sl2, vs, lane);
    else
        wave_run_pair<D, 2>(wdesc, L, q, kpool, vpool, o, lse, po, plse, hq, hkv, G, sl2, vs, lane);
}

// ============================================================================ tile kernel

// Stage buffers of a tile item: K and V of one 64-key stage (4 blocks), 64 rows of D bf16 each,
// unpadded.  The 16-byte chunks of row r are XOR-swizzled -- chunk c sits at chunk position
// c ^ swz(r) -- so that the reads hit distinct LDS banks: the MFMA-operand reads of K
// (ds_read_b128, 16 rows of one chunk each) and the transposed 8-byte reads of V
// (ds_read_b64_tr_b16, 8 rows of 32 contiguous bytes each per 32 lanes).  K and V take different
// swizzles: the ones below measured zero bank-conflict cycles (SQ_LDS_BANK_CONFLICT) for their own
// read pattern, whereas one swizzle for both cost 4 cycles per K read (or 2 per V read).  Both depend
// on r mod 16 only, so a block's rows carry the same pattern wherever the block sits in the stage.
template <int D>
__device__ __forceinline__ int tile_swz_k(int r) {
    return D == 128 ? r & 15 : r & 7;
}
template <int D>
__device__ __forceinline__ int tile_swz_v(int r) {
    return D == 128 ? (2 * (r & 7)) ^ ((r >> 3) & 1) : r & 7;
}
template <int D>
constexpr int tile_buf_bytes() {
    return 64 * D * 2;
}

typedef __attribute__((address_space(3))) void* lds_void_ptr;

// Fetch one block of a stage straight from global memory into LDS (buffer_load_dwordx4 ... lds:
// lane l of an instruction writes the l-th 16 bytes of a contiguous 1-KB run at the wave-uniform
// destination), each lane fetching the global chunk that the swizzle puts at its slot.  The buffer
// descriptor spans the one block, so the offsets stay small for pools of any size.  (The buffer
// form rather than global_load_lds: the latter also counts as an LDS access of unknown order,
// which forces every later LDS read to wait for all earlier ones.)  Rows past the block's length
// read its last row (masked later); a block past the item's end has len 0 and reads row 0 of a
// valid block.  kdst / vdst: the block's rows in the stage buffers (uniform).
template <int D>
__device__ __forceinline__ void stage_fetch(const uint16_t* __restrict__ kpool, const uint16_t* __restrict__ vpool,
                                            size_t boff, int len, int lane, uint8_t* kdst, uint8_t* vdst) {
    constexpr int CPR = D / 8;     // 16-byte chunks per row
    constexpr int RPI = 64 / CPR;  // rows per 1-KB instruction
    constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit data format
    const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(kpool + boff), 0, 32 * D, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(vpool + boff), 0, 32 * D, kRsrcWord3);
    const int last = max(len - 1, 0);
#pragma unroll
    for (int i = 0; i < 16 / RPI; ++i) {
        const int r = i * RPI + lane / CPR;
        const int row_off = min(r, last) * D * 2;
        const int koff = row_off + (((lane % CPR) ^ tile_swz_k<D>(r)) * 16);
        const int voff = row_off + (((lane % CPR) ^ tile_swz_v<D>(r)) * 16);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_void_ptr)(kdst + i * 1024), 16, koff, 0, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_void_ptr)(vdst + i * 1024), 16, voff, 0, 0, 0);
    }
}

// Wait for this wave's stage fetches, then for every wave's (and for every wave to be done reading
// the buffer that the next fetch overwrites).
__device__ __forceinline__ void stage_barrier() {
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// One workgroup per tile item: a tile of up to 64T query rows (wave w owns rows 16Tw .. 16Tw+16T-1
// as T column tiles) against the item's key blocks, four blocks per stage.  Stage s+1 is fetched into
// the other pair of LDS buffers while stage s is contracted; one barrier per stage (a buffer is
// rewritten only after every wave has passed the barrier that follows its last use).  The stage
// loop is unrolled by two so that each stage names its buffers statically: the compiler then knows
// that the reads of one buffer do not depend on the fetch into the other.
template <int D, int T>
__device__ __forceinline__ void tile_item(const tkv::ItemDesc& it, const tkv::TokDesc* __restrict__ toks,
                                          const tkv::BlkDesc* __restrict__ blks, const uint16_t* __restrict__ q,
                                          const uint16_t* __restrict__ kpool, const uint16_t* __restrict__ vpool,
                                          uint16_t* __restrict__ o, float* __restrict__ lse, uint16_t* __restrict__ po,
                                          float* __restrict__ plse, int hq, int hkv, int G, float sl2, uint8_t* k0,
                                          uint8_t* v0, uint8_t* k1, uint8_t* v1) {
    constexpr int RB = 2 * D;  // bytes per K/V row in the stage buffers
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int col = lane & 15, kg = lane >> 4;
    const size_t blk_stride = static_cast<size_t>(hkv) * (16 * D);
    const size_t kvh_off = static_cast<size_t>(it.kvh) * (16 * D);
    const int2* bd = reinterpret_cast<const int2*>(blks + it.blk_off);
    const int nb = it.n_blk;
    const int n_stages = (nb + 3) / 4;

    // this lane's query row of each column tile (only Q and the causal limits stay live across the
    // stages; the output fields are read again from the token descriptors at the end)
    bf16x8_t qf[T][D / 32];
    int limit[T];
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        const int row = 16 * T * wave + 16 * tt + col;
        const int t = row / G;
        const tkv::TokDesc td = toks[it.tok_off + min(t, it.n_tok - 1)];
        limit[tt] = t < it.n_tok ? td.limit : -1;
        const uint16_t* qrow = q + (static_cast<size_t>(td.qtok) * hq + it.kvh * G + (row - t * G)) * D + kg * 8;
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) qf[tt][ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qrow + ks * 32));
    }
    bool any_row = false;
#pragma unroll
    for (int tt = 0; tt < T; ++tt) any_row = any_row || limit[tt] >= 0;
    const bool wave_active = __builtin_amdgcn_ballot_w64(any_row) != 0;

    // Swizzled read offsets within a block (bytes).  K, S^T A operand: lane (col, kg) reads row col,
    // chunk 4kk + kg, i.e. koff ^ 64kk.  V, transposed reads: lane (col, kg) reads row
    // 4kg + col/4, bytes 8(col & 3) .. +7 of the 32-byte column run of output tile ct, i.e.
    // voff ^ 32ct.  (The XORs touch only the chunk-index bits of the offsets.)
    const int koff = col * RB + 16 * (kg ^ tile_swz_k<D>(col));
    const int vrow = 4 * kg + (col >> 2);
    const int voff = vrow * RB + 16 * (((col & 3) >> 1) ^ tile_swz_v<D>(vrow)) + 8 * (col & 1);

    // block descriptors of a stage: lane l holds block 4s + (l & 3) (the item's last block past its end)
    auto stage_desc = [&](int st) { return bd[min(4 * st + (lane & 3), nb - 1)]; };
    int2 dcur = stage_desc(0), dnxt = stage_desc(1);
    const int wblk = wave * 16 * RB;  // this wave's block within a stage buffer (waves 0-3 fetch)
    if (wave < 4) {
        const int len = wave < nb ? __builtin_amdgcn_readlane(dcur.y, wave) : 0;
        stage_fetch<D>(kpool, vpool, static_cast<size_t>(__builtin_amdgcn_readlane(dcur.x, wave)) * blk_stride + kvh_off,
                       len, lane, k0 + wblk, v0 + wblk);
    }
    WaveAcc<D, T> A;
    A.reset();
    int pos = it.pos0;
    auto stage = [&](int st, const uint8_t* ks, const uint8_t* vs, uint8_t* kn, uint8_t* vn) {
        stage_barrier();
        // fetch the next stage while this one is contracted
        if (st + 1 < n_stages && wave < 4) {
            const int bn = 4 * (st + 1) + wave;
            const int len = bn < nb ? __builtin_amdgcn_readlane(dnxt.y, wave) : 0;
            stage_fetch<D>(kpool, vpool,
                           static_cast<size_t>(__builtin_amdgcn_readlane(dnxt.x, wave)) * blk_stride + kvh_off, len,
                           lane, kn + wblk, vn + wblk);
        }
        const int2 dthis = dcur;
        dcur = dnxt;
        dnxt = stage_desc(st + 2);
        if (!wave_active) return;
        int len[4], bpos[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int lj = __builtin_amdgcn_readlane(dthis.y, j);
            len[j] = 4 * st + j < nb ? lj : 0;
            bpos[j] = pos;
            pos += len[j];
        }
        // S^T for all four blocks first (32 independent MFMAs), so that each pair's softmax below
        // overlaps MFMAs still in flight
        f32x4_t sc[4][T];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int tt = 0; tt < T; ++tt) sc[j][tt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        bf16x8_t kf[D / 32][4];
#pragma unroll
        for (int kk = 0; kk < D / 32; ++kk)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                kf[kk][j] = *reinterpret_cast<const bf16x8_t*>(ks + 16 * j * RB + (koff ^ (64 * kk)));
#pragma unroll
        for (int kk = 0; kk < D / 32; ++kk)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int tt = 0; tt < T; ++tt) sc[j][tt] = mfma_16x16x32(kf[kk][j], qf[tt][kk], sc[j][tt]);
        // K reads two k-steps ahead of the MFMAs that use them
        __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
        for (int kk = 0; kk < D / 32 - 2; ++kk) {
            __builtin_amdgcn_sched_group_barrier(0x008, 4 * T, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 8 * T, 0);
        // one uniform decision per stage: mask only if a block is partial or absent, or some row's
        // causal limit falls inside the stage
        const int stage_end = pos;  // one past the last key position of the stage
        bool cut = false;
#pragma unroll
        for (int tt = 0; tt < T; ++tt) cut = cut || (limit[tt] >= 0 && limit[tt] < stage_end - 1);
        if (len[3] != 16 || len[0] + len[1] + len[2] != 48 || __builtin_amdgcn_ballot_w64(cut) != 0) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int tt = 0; tt < T; ++tt) {
                    const int vlen = min(len[j], limit[tt] - bpos[j] + 1);
#pragma unroll
                    for (int x = 0; x < 4; ++x)
                        if (4 * kg + x >= vlen) sc[j][tt][x] = -INFINITY;
                }
        }
        // the exponent base: one row-max and lazy-move decision per stage and tile, so that the
        // exponentials and PV MFMAs of both pairs below form one branch-free block the scheduler can
        // interleave (a stage past every causal limit of the wave is all -inf and adds nothing)
        stage_base<D, T>(A, sc, sl2);
        float msc[T];
#pragma unroll
        for (int tt = 0; tt < T; ++tt) msc[tt] = A.m[tt] == -INFINITY ? 0.f : A.m[tt] * sl2;
#pragma unroll
        for (int jp = 0; jp < 2; ++jp) {
            const int ja = 2 * jp, jb = 2 * jp + 1;
            bf16x8_t pb[T];
#pragma unroll
            for (int tt = 0; tt < T; ++tt) {
#pragma unroll
                for (int x = 0; x < 4; ++x) {
                    sc[ja][tt][x] = __builtin_amdgcn_exp2f(fmaf(sc[ja][tt][x], sl2, -msc[tt]));
                    sc[jb][tt][x] = __builtin_amdgcn_exp2f(fmaf(sc[jb][tt][x], sl2, -msc[tt]));
                }
                const uint4 pk{pack_bf16x2(sc[ja][tt][0], sc[ja][tt][1]), pack_bf16x2(sc[ja][tt][2], sc[ja][tt][3]),
                               pack_bf16x2(sc[jb][tt][0], sc[jb][tt][1]), pack_bf16x2(sc[jb][tt][2], sc[jb][tt][3])};
                // the row sum over the bf16-rounded P that the PV product uses, two keys per v_dot2
                A.l[tt] = sum_bf16x2(pk.x, sum_bf16x2(pk.y, sum_bf16x2(pk.z, sum_bf16x2(pk.w, A.l[tt]))));
                pb[tt] = __builtin_bit_cast(bf16x8_t, pk);
            }
            const uint8_t* vra = vs + 16 * ja * RB;
            const uint8_t* vrb = vra + 16 * RB;
#pragma unroll
            for (int ct = 0; ct < D / 16; ++ct) {
                const int off = voff ^ (32 * ct);
                const s16x4_t va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4_t*)(const_cast<uint8_t*>(vra + off)));
                const s16x4_t vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4_t*)(const_cast<uint8_t*>(vrb + off)));
                const bf16x8_t vab = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(va, vb, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
                for (int tt = 0; tt < T; ++tt) A.acc[tt][ct] = mfma_16x16x32(vab, pb[tt], A.acc[tt][ct]);
            }
        }
    };
    for (int st = 0; st < n_stages; st += 2) {
        stage(st, k0, v0, k1, v1);
        if (st + 1 < n_stages) stage(st + 1, k1, v1, k0, v0);
    }
    if (!wave_active) return;
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        const int row = 16 * T * wave + 16 * tt + col;
        const int t = row / G;
        const tkv::TokDesc td = toks[it.tok_off + min(t, it.n_tok - 1)];
        write_rows<D>(A.acc[tt], A.m[tt], A.l[tt], t < it.n_tok, td.qtok, it.kvh * G + (row - t * G), td.slot, kg, o,
                      lse, po, plse, hq, sl2);
    }
}


// The attention kernel runs tile items (one workgroup each, longest first, in the planner's XCD
// order) and the wave grid (kWaveWG waves per workgroup) in one launch, so neither waits for the
// other's tail.  Workgroups are dispatched in index order, workgroup b on XCD b % 8, and within an
// XCD the k-th workgroup (k = b / 8) on shader engine k % 4 in a fixed rotation (then on a CU of
// that engine with room).  The first `runs` pairs of runs of kInterleaveRun = 32 alternate -- 32
// tile items, 32 wave-grid workgroups, ... -- so that MFMA-bound tiles and HBM-bound waves share
// the chip from the start when the grid does not fit on it at once: a run of 32 gives each XCD four
// workgroups of one kind, one per engine, so every engine gets both kinds.  (Runs of 8 alternate
// the kinds with period 2 per XCD, which locks each kind onto two of the four engines.)  Then come
// the remaining tile items, then the remaining wave-grid workgroups.  Either way tile item i and
// wave workgroup j run on XCDs i % 8 and j % 8, as the planner assumed.
template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fwd(
    const tkv::ItemDesc* __restrict__ items, int n_tile, int n_wave_wg, int runs, const tkv::TokDesc* __restrict__ toks,
    const tkv::BlkDesc* __restrict__ blks, const int4* __restrict__ wdesc, const int32_t* __restrict__ woff,
    const int32_t* __restrict__ wtiles, const uint16_t* __restrict__ q, const uint16_t* __restrict__ kpool,
    const uint16_t* __restrict__ vpool, uint16_t* __restrict__ o, float* __restrict__ lse, uint16_t* __restrict__ po,
    float* __restrict__ plse, int hq, int hkv, int G, float sl2) {
    // the tile path's two stage buffers of K and V; the wave grid gives one of the four to each wave
    __shared__ __attribute__((aligned(1024))) uint8_t lds_k0[tile_buf_bytes<D>()];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_v0[tile_buf_bytes<D>()];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_k1[tile_buf_bytes<D>()];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_v1[tile_buf_bytes<D>()];
    static_assert(32 * (2 * D + 32) <= tile_buf_bytes<D>(), "a wave-grid wave stages two V blocks in one buffer");
    constexpr int R = tkv::kInterleaveRun;
    const int b = blockIdx.x;
    int tile = -1, wg = -1;
    if (b < 2 * R * runs) {
        const int pair = b / (2 * R), within = b % (2 * R);
        (within >= R ? wg : tile) = R * pair + within % R;
    } else {
        const int r = b - 2 * R * runs;
        const int tiles_left = runs > 0 ? (n_tile + R - 1) / R * R - R * runs : (n_tile + 7) / 8 * 8;
        if (r < tiles_left)
            tile = R * runs + r;
        else
            wg = R * runs + (r - max(tiles_left, 0));
    }
    if (tile >= 0) {
        if (tile >= n_tile) return;
        const tkv::ItemDesc it = items[tile];
        tile_item<D, 2>(it, toks, blks, q, kpool, vpool, o, lse, po, plse, hq, hkv, G, sl2, lds_k0, lds_v0, lds_k1,
                        lds_v1);
        return;
    }
    if (wg >= n_wave_wg) return;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    uint8_t* vs = wave == 0 ? lds_k0 : wave == 1 ? lds_v0 : wave == 2 ? lds_k1 : lds_v1;
    wave_worker<D>(wg * tkv::kWaveWG + wave, lane, wdesc, woff, wtiles, q, kpool, vpool, o, lse, po,
                   plse, hq, hkv, G, sl2, vs);
}

// Few tile items and no wave-grid work (a small verification batch): the chip has a CU for every
// tile, and a tile's walk over its keys sets the call's time.  Eight waves of one 16-row column tile
// each share a 128-row tile (instead of four waves of two), so each wave does half the MFMA and
// softmax work per stage and the walk is shorter.  Waves 0-3 fetch the stages.
template <int D>
__global__ __launch_bounds__(2 * kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_tile8(
    const tkv::ItemDesc* __restrict__ items, int n_tile, const tkv::TokDesc* __restrict__ toks,
    const tkv::BlkDesc* __restrict__ blks, const uint16_t* __restrict__ q, const uint16_t* __restrict__ kpool,
    const uint16_t* __restrict__ vpool, uint16_t* __restrict__ o, float* __restrict__ lse, uint16_t* __restrict__ po,
    float* __restrict__ plse, int hq, int hkv, int G, float sl2) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds_k0[tile_buf_bytes<D>()];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_v0[tile_buf_bytes<D>()];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_k1[tile_buf_bytes<D>()];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_v1[tile_buf_bytes<D>()];
    const int b = blockIdx.x;
    if (b >= n_tile) return;
    const tkv::ItemDesc it = items[b];
    tile_item<D, 1>(it, toks, blks, q, kpool, vpool, o, lse, po, plse, hq, hkv, G, sl2, lds_k0, lds_v0, lds_k1, lds_v1);
}

// Log-sum-exp merge of one query token's partials (one workgroup per token, whose partial slots
// are contiguous, sized to one thread per four columns of the token's heads): every thread folds
// the partials of its column in with an online softmax, eight partials' outputs and lse values in
// flight at a time -- one round of memory latency per eight partials, no barriers.
template <int D>
__global__ __launch_bounds__(1024) void merge_partials(const tkv::MergeDesc* __restrict__ md,
                                                           const uint16_t* __restrict__ po,
                                                           const float* __restrict__ plse,
                                                           uint16_t* __restrict__ o, float* __restrict__ lse, int hq) {
    constexpr int C4 = D / 4;
    const tkv::MergeDesc m = md[blockIdx.x];
    const size_t s0 = static_cast<size_t>(m.slot_off);
    const int n = m.n_slots;
    const uint2* po4 = reinterpret_cast<const uint2*>(po);  // four fp16 columns
    for (int idx = threadIdx.x; idx < hq * C4; idx += blockDim.x) {
        const int h = idx / C4;
        float mx = -INFINITY, sum = 0.f;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int j0 = 0; j0 < n; j0 += 8) {
            float4 x[8];
            float lj[8];
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                const size_t sl = s0 + min(j0 + v, n - 1);
                x[v] = unpack_f16x4(po4[(sl * hq) * C4 + idx]);
                lj[v] = j0 + v < n ? plse[sl * hq + h] : -INFINITY;
            }
            float cm = lj[0];
#pragma unroll
            for (int v = 1; v < 8; ++v) cm = fmaxf(cm, lj[v]);
            const float m_new = fmaxf(mx, cm);
            if (m_new == -INFINITY) continue;  // no key seen yet
            const float a = __expf(mx - m_new);
            sum *= a;
            acc.x *= a;
            acc.y *= a;
            acc.z *= a;
            acc.w *= a;
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                const float wv = __expf(lj[v] - m_new);  // 0 for padding entries (lj = -inf)
                sum += wv;
                acc.x = fmaf(wv, x[v].x, acc.x);
                acc.y = fmaf(wv, x[v].y, acc.y);
                acc.z = fmaf(wv, x[v].z, acc.z);
                acc.w = fmaf(wv, x[v].w, acc.w);
            }
            mx = m_new;
        }
        const float inv = sum > 0.f ? 1.f / sum : 0.f;
        uint2 wv;
        wv.x = pack_bf16x2(acc.x * inv, acc.y * inv);
        wv.y = pack_bf16x2(acc.z * inv, acc.w * inv);
        *reinterpret_cast<uint2*>(o + (static_cast<size_t>(m.qtok) * hq) * D + idx * 4) = wv;
        if (lse && idx % C4 == 0)
            lse[static_cast<size_t>(m.qtok) * hq + h] = sum > 0.f ? mx + __logf(sum) : -INFINITY;
    }
}

// Writes image words into an uploaded workspace: pairs[i] = {word index, value}.  The host builds
// every index from the plan's own image, below its size.
__global__ __launch_bounds__(256) void patch_apply(const int2* __restrict__ pairs, int n, int32_t* __restrict__ ws) {
    const int i = static_cast<int>(blockIdx.x) * 256 + static_cast<int>(threadIdx.x);
    if (i < n) {
        const int2 w = pairs[i];
        ws[w.x] = w.y;
    }
}

}  // namespace

namespace tkv {

void wait_copies(const tkv_plan* p) {
    if (p->copy_pending) {
        (void)hipEventSynchronize(static_cast<hipEvent_t>(p->copy_event));
        p->copy_pending = false;
    }
}

// Records the completion of the copies just enqueued from the plan's host memory.
static int record_copy(const tkv_plan* p, hipStream_t st, const char* fn) {
    if (!p->copy_event) {
        hipEvent_t e;
        const hipError_t rc = hipEventCreateWithFlags(&e, hipEventDisableTiming);
        if (rc != hipSuccess) return set_error(TKV_EHIP, "%s: hipEventCreateWithFlags: %s", fn, hipGetErrorString(rc));
        p->copy_event = e;
    }
    const hipError_t rc = hipEventRecord(static_cast<hipEvent_t>(p->copy_event), st);
    if (rc != hipSuccess) return set_error(TKV_EHIP, "%s: hipEventRecord: %s", fn, hipGetErrorString(rc));
    p->copy_pending = true;
    return TKV_OK;
}

int upload(tkv_plan* p, void* d_ws, size_t bytes, void* stream) {
    (void)bytes;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    wait_copies(p);  // the pair staging below may still be read by the last upload
    // Into the workspace that holds the image of the last upload, only the words in-place updates
    // changed since: (index, value) pairs copied to the patch region, then written in by patch_apply.
    const size_t n_words = p->desc_bytes / sizeof(int32_t);
    bool patch = d_ws == p->ws_image && !p->dirty_over && p->dirty.size() <= static_cast<size_t>(p->patch_cap);
    if (patch && !p->dirty.empty()) {
        const int32_t* img = reinterpret_cast<const int32_t*>(p->image.get());
        std::vector<int32_t>& pairs = p->patch_pairs;
        pairs.resize(2 * p->dirty.size());
        for (size_t i = 0; i < p->dirty.size(); ++i) {
            const int32_t w = p->dirty[i];
            if (w < 0 || static_cast<size_t>(w) >= n_words) {  // cannot happen; never send an index out of the image
                patch = false;
                break;
            }
            pairs[2 * i] = w;
            pairs[2 * i + 1] = img[w];
        }
        if (patch) {
            uint8_t* ws = static_cast<uint8_t*>(d_ws);
            const int n = static_cast<int>(p->dirty.size());
            hipError_t e = hipMemcpyAsync(ws + p->off_patch, pairs.data(), pairs.size() * sizeof(int32_t),
                                          hipMemcpyHostToDevice, st);
            if (e != hipSuccess) return set_error(TKV_EHIP, "tkv_plan_upload: hipMemcpyAsync: %s", hipGetErrorString(e));
            hipLaunchKernelGGL(patch_apply, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, st,
                               reinterpret_cast<const int2*>(ws + p->off_patch), n, reinterpret_cast<int32_t*>(ws));
            e = hipGetLastError();
            if (e != hipSuccess) return set_error(TKV_EHIP, "tkv_plan_upload: patch_apply launch: %s", hipGetErrorString(e));
        }
    }
    if (!patch && p->desc_bytes) {
        const hipError_t e = hipMemcpyAsync(d_ws, p->image.get(), p->desc_bytes, hipMemcpyHostToDevice, st);
        if (e != hipSuccess) return set_error(TKV_EHIP, "tkv_plan_upload: hipMemcpyAsync: %s", hipGetErrorString(e));
    }
    const int rc = record_copy(p, st, "tkv_plan_upload");
    if (rc != TKV_OK) return rc;
    p->d_ws = d_ws;
    p->ws_image = d_ws;
    p->dirty.clear();
    p->dirty_over = false;
    return TKV_OK;
}

template <int D>
static int launch_d(const tkv_plan* p, uint8_t* ws, const void* q, const void* k, const void* v, void* o, float* lse,
                    hipStream_t st) {
    const auto* merges = reinterpret_cast<const MergeDesc*>(ws + p->off_merges);
    const auto* items = reinterpret_cast<const ItemDesc*>(ws + p->off_items);
    const auto* wdesc = reinterpret_cast<const int4*>(ws + p->off_wdesc);
    const auto* woff = reinterpret_cast<const int32_t*>(ws + p->off_woff);
    const auto* wtiles = reinterpret_cast<const int32_t*>(ws + p->off_wtiles);
    const auto* toks = reinterpret_cast<const TokDesc*>(ws + p->off_toks);
    const auto* blks = reinterpret_cast<const BlkDesc*>(ws + p->off_blks);
    uint16_t* po = reinterpret_cast<uint16_t*>(ws + p->off_po);
    float* plse = reinterpret_cast<float*>(ws + p->off_plse);
    const float sl2 = 1.4426950408889634f / std::sqrt(static_cast<float>(D));
    const int hq = p->shape.hq, hkv = p->shape.hkv;
    // Instrumented calls time the kernels by the dispatch packets' own start/end timestamps
    // (hipExtLaunchKernelGGL events): the main phase from the start of its first kernel to the
    // end of its last, and the merge kernel.
    hipEvent_t* ev = nullptr;
    if (p->prof_n < p->prof_max) ev = reinterpret_cast<hipEvent_t*>(p->prof_events.data()) + 4 * p->prof_n++;
    const int n_tile = static_cast<int>(p->items.size());
    const int n_wave_wg = std::max(0, static_cast<int>(p->wave_off.size()) - 1) / kWaveWG;  // waves: a multiple of kWaveWG
    // runs of kInterleaveRun of each kind (the last run of each padded with workgroups that return at
    // once), interleaved when the grid exceeds the workgroup slots of the chip (two per CU)
    constexpr int R = kInterleaveRun;
    const int runs = n_tile + n_wave_wg > kWaveWorkers / kWaveWG ? std::min((n_tile + R - 1) / R, (n_wave_wg + R - 1) / R) : 0;
    const int grid = runs > 0 ? 2 * R * runs + std::max(0, (n_tile + R - 1) / R * R - R * runs) +
                                    std::max(0, (n_wave_wg + 7) / 8 * 8 - R * runs)
                              : (n_tile + 7) / 8 * 8 + (n_wave_wg + 7) / 8 * 8;
    if (p->tile8 && n_wave_wg == 0 && n_tile > 0)
        hipExtLaunchKernelGGL(attn_tile8<D>, dim3(static_cast<unsigned>(n_tile)), dim3(2 * kThreads), 0, st,
                              ev ? ev[0] : nullptr, ev ? ev[1] : nullptr, 0, items, n_tile, toks, blks,
                              static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                              static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), lse, po, plse, hq, hkv,
                              p->group, sl2);
    else if (grid > 0)
        hipExtLaunchKernelGGL(attn_fwd<D>, dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0, st,
                              ev ? ev[0] : nullptr, ev ? ev[1] : nullptr, 0, items, n_tile, n_wave_wg, runs, toks, blks,
                              wdesc, woff, wtiles, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                              static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), lse, po, plse, hq, hkv,
                              p->group, sl2);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(TKV_EHIP, "attention launch: %s", hipGetErrorString(e));
    if (!p->merges.empty()) {
        // one thread per float4 column of the token's heads (up to 1024 threads)
        const int merge_threads = std::min(1024, (hq * (D / 4) + 63) / 64 * 64);
        hipExtLaunchKernelGGL(merge_partials<D>, dim3(static_cast<unsigned>(p->merges.size())), dim3(merge_threads), 0, st,
                              ev ? ev[2] : nullptr, ev ? ev[3] : nullptr, 0, merges,
                              static_cast<const uint16_t*>(po), static_cast<const float*>(plse),
                              static_cast<uint16_t*>(o), lse, hq);
        e = hipGetLastError();
        if (e != hipSuccess) return set_error(TKV_EHIP, "merge launch: %s", hipGetErrorString(e));
    } else if (ev) {
        (void)hipEventRecord(ev[2], st);
        (void)hipEventRecord(ev[3], st);
    }
    return TKV_OK;
}

static int launch_ws(const tkv_plan* p, uint8_t* ws, const void* q, const void* k, const void* v, void* o, float* lse,
                     hipStream_t st) {
    return p->shape.d == 128 ? launch_d<128>(p, ws, q, k, v, o, lse, st) : launch_d<64>(p, ws, q, k, v, o, lse, st);
}

int launch_attention(const tkv_plan* p, const void* q, const void* k, const void* v, void* o, float* lse,
                     void* stream) {
    return launch_ws(p, static_cast<uint8_t*>(p->d_ws), q, k, v, o, lse, static_cast<hipStream_t>(stream));
}

}  // namespace tkv

// ---------------------------------------------------------------------------- no-allocation variant
// A workspace of the library's own, for callers that cannot allocate device memory: a file-scope
// device array that each GPU holds for the life of the process.  Host code never uses its name as
// an address: its per-device address comes from hipGetSymbolAddress, taken once per device with
// that device current.  No part of it needs to start at zero: a call overwrites the descriptor
// region first, and every partial slot is written by its item before the merge reads it.
static constexpr size_t kScratchBytes = size_t{64} << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];
static_assert(TKV_NOALLOC_MAX_BYTES == kScratchBytes, "header limit and device array agree");

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_for_current_device(uint8_t** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return tkv::set_error(TKV_EHIP, "tkv_verify_noalloc: hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return tkv::set_error(TKV_EINVAL, "tkv_verify_noalloc: device %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return tkv::set_error(TKV_EHIP, "tkv_verify_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
        g_scratch_ptr[dev] = ptr;
    }
    *out = static_cast<uint8_t*>(g_scratch_ptr[dev]);
    return TKV_OK;
}
}  // namespace

TKV_EXPORT int tkv_verify_noalloc(const tkv_plan* p, const void* q, const void* k, const void* v, void* o, float* lse,
                                  void* stream) {
    tkv::clear_error();
    if (!p) return tkv::set_error(TKV_EINVAL, "tkv_verify_noalloc: plan is NULL");
    if (p->total_bytes > kScratchBytes)
        return tkv::set_error(TKV_EINVAL, "tkv_verify_noalloc: the plan needs a %zu-byte workspace, more than the %zu bytes "
                              "of the library's static one (use tkv_plan_upload and tkv_verify)", p->total_bytes,
                              kScratchBytes);
    if (p->items.empty() && p->wave_items.empty()) return TKV_OK;
    if (!q || !k || !v || !o) return tkv::set_error(TKV_EINVAL, "tkv_verify_noalloc: NULL tensor pointer");
    uint8_t* ws = nullptr;
    int rc = scratch_for_current_device(&ws);
    if (rc != TKV_OK) return rc;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    if (p->desc_bytes) {
        const hipError_t e = hipMemcpyAsync(ws, p->image.get(), p->desc_bytes, hipMemcpyHostToDevice, st);
        if (e != hipSuccess) return tkv::set_error(TKV_EHIP, "tkv_verify_noalloc: hipMemcpyAsync: %s", hipGetErrorString(e));
        // the copy's completion is recorded with the plan's event if an upload made one (creating
        // one here would allocate)
        if (p->copy_event) {
            rc = tkv::record_copy(p, st, "tkv_verify_noalloc");
            if (rc != TKV_OK) return rc;
        }
    }
    return tkv::launch_ws(p, ws, q, k, v, o, lse, st);
}

static void free_events(const tkv_plan* p) {
    for (void* e : p->prof_events) (void)hipEventDestroy(static_cast<hipEvent_t>(e));
    p->prof_events.clear();
    p->prof_max = p->prof_n = 0;
}

tkv_plan::~tkv_plan() {
    free_events(this);
    tkv::wait_copies(this);
    if (copy_event) (void)hipEventDestroy(static_cast<hipEvent_t>(copy_event));
    tkv::give_image(std::move(image), image_cap);
}

TKV_EXPORT int tkv_plan_profile(tkv_plan* p, int32_t max_calls) {
    tkv::clear_error();
    if (!p || max_calls < 0) return tkv::set_error(TKV_EINVAL, "tkv_plan_profile: bad argument");
    free_events(p);
    for (int32_t i = 0; i < 4 * max_calls; ++i) {
        hipEvent_t e;
        const hipError_t rc = hipEventCreate(&e);
        if (rc != hipSuccess) {
            free_events(p);
            return tkv::set_error(TKV_EHIP, "tkv_plan_profile: hipEventCreate: %s", hipGetErrorString(rc));
        }
        p->prof_events.push_back(e);
    }
    p->prof_max = max_calls;
    return TKV_OK;
}

TKV_EXPORT int tkv_plan_profile_read(tkv_plan* p, int32_t* n_calls, float* ms_main, float* ms_merge) {
    tkv::clear_error();
    if (!p || !n_calls || !ms_main || !ms_merge) return tkv::set_error(TKV_EINVAL, "tkv_plan_profile_read: NULL argument");
    float a = 0.f, b = 0.f;
    for (int32_t i = 0; i < p->prof_n; ++i) {
        hipEvent_t* ev = reinterpret_cast<hipEvent_t*>(p->prof_events.data()) + 4 * i;
        hipError_t rc = hipEventSynchronize(ev[3]);
        float t0 = 0.f, t1 = 0.f;
        if (rc == hipSuccess) rc = hipEventElapsedTime(&t0, ev[0], ev[1]);
        if (rc == hipSuccess) rc = hipEventElapsedTime(&t1, ev[2], ev[3]);
        if (rc != hipSuccess) return tkv::set_error(TKV_EHIP, "tkv_plan_profile_read: %s", hipGetErrorString(rc));
        a += t0;
        b += t1;
    }
    *n_calls = p->prof_n;
    *ms_main = a;
    *ms_merge = b;
    p->prof_n = 0;
    return TKV_OK;
}
