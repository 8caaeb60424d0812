// Tree-shared paged attention kernels for gfx950 (MI355X).
//
// attn_persist: persistent workgroups, each walking its list of work items (see plan.cpp).  An item is a tile of up to 64 query
// rows -- query tokens x the G query heads of one KV head -- and an ordered list of KV blocks.
// K/V blocks are staged through LDS four at a time (64 keys) and every wave contracts them
// against its 16 query rows on bf16 MFMA (v_mfma_f32_16x16x32_bf16, fp32 accumulation):
//   S^T = K Q^T   (A = 16 keys x 32 d from LDS, B = Q^T held in registers),
//   O^T += V^T P^T (A = V^T from a transposed LDS copy, B = P^T straight from the S^T registers),
// with an online softmax in between (exp2, scale folded into one FMA).  Computing the transposed
// products keeps each lane's query row fixed across both contractions, so the running max, sum
// and the O rescale never leave the lane.  Masking is per key: slots beyond a block's length are
// never loaded (zero-filled in LDS) and keys past a token's causal limit get -inf.
//
// merge_partials: log-sum-exp merge of the per-segment partials of one query token (all heads):
//   lse = log sum_j exp(lse_j),  o = sum_j exp(lse_j - lse) o_j.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

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

constexpr int kThreads = 256;
constexpr int kKeysPerStage = 64;  // four 16-token blocks

// One stage as the kernel sees it after decoding its descriptor (scalar registers).
struct StageInfo {
    int len[4], pos[4];
    int kvh, n_tok, flags;
};

// Lane l loads 16-byte word min(l & 7, 4) of the stage descriptor's header: lanes 0..3 hold
// blocks[0..3] = {blk, len, pos, -} and lane 4 holds {kvh, n_tok, flags, -}, so a block's fields
// come out with v_readlane at a (uniform) lane index -- no select chains, no branches.
__device__ __forceinline__ int4 load_hdr(const tkv::StageDesc* __restrict__ stages, int gs, int lane) {
    return reinterpret_cast<const int4*>(stages + gs)[min(lane & 7, 4)];
}
__device__ __forceinline__ int4 load_tok(const tkv::StageDesc* __restrict__ stages, int gs, int t) {
    return reinterpret_cast<const int4*>(stages[gs].toks)[t];
}

__device__ __forceinline__ StageInfo decode_hdr(const int4& h) {
    StageInfo si;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        si.len[j] = __builtin_amdgcn_readlane(h.y, j);
        si.pos[j] = __builtin_amdgcn_readlane(h.z, j);
    }
    si.kvh = __builtin_amdgcn_readlane(h.x, 4);
    si.n_tok = __builtin_amdgcn_readlane(h.y, 4);
    si.flags = __builtin_amdgcn_readlane(h.z, 4);
    return si;
}

// Registers of one stage owned by this thread: K in row layout, V as KPV consecutive keys x 8
// dims (transposed into key-contiguous words on the way to LDS).
template <int D>
struct StageRegs {
    static constexpr int DCH = D / 8;                          // 16-byte chunks per row
    static constexpr int KPT = kKeysPerStage * DCH / kThreads;  // K chunks per thread
    static constexpr int KPV = D == 128 ? 4 : 2;                // V keys per thread
    u32x4_t k[KPT];
    u32x4_t v[KPV];
};

// All loads are straight-line (so the compiler's wait counts stay exact and nothing drains the
// prefetch early).  A thread's block is uniform across its wave, read from the header with
// v_readlane; a slot past the block's length reads the block's last row (masked in the softmax,
// so it contributes exactly 0); an absent block reads the stage's first block.  valid = false
// turns every length to 0 (the fetch past the end of the stream reads one row per block).
template <int D>
__device__ __forceinline__ void stage_load(StageRegs<D>& r, const int4& h, bool valid, int kvh,
                                           const uint16_t* __restrict__ kpool, const uint16_t* __restrict__ vpool,
                                           int hkv, int tid, int wave_u) {
    constexpr int DCH = StageRegs<D>::DCH;
#pragma unroll
    for (int i = 0; i < StageRegs<D>::KPT; ++i) {
        const int c = tid + kThreads * i;
        const int dc = c % DCH, sl = (c / DCH) & 15;
        const int j = D == 128 ? i : 2 * i + (wave_u >> 1);   // c / (16 * DCH), uniform per wave
        const int id = __builtin_amdgcn_readlane(h.x, j);
        const int len = valid ? __builtin_amdgcn_readlane(h.y, j) : 0;
        const int se = min(sl, max(len - 1, 0));
        const uint16_t* base = kpool + (static_cast<size_t>(id) * hkv + kvh) * (16 * D);
        r.k[i] = *reinterpret_cast<const u32x4_t*>(base + se * D + dc * 8);
    }
    constexpr int KPV = StageRegs<D>::KPV;
    const int id = __builtin_amdgcn_readlane(h.x, wave_u);   // this wave's V keys lie in block `wave`
    const int len = valid ? __builtin_amdgcn_readlane(h.y, wave_u) : 0;
    const uint16_t* base = vpool + (static_cast<size_t>(id) * hkv + kvh) * (16 * D);
    const int kq = tid / DCH, dc = tid % DCH;   // keys KPV*kq .. +KPV-1 of the stage, dims 8dc..8dc+7
#pragma unroll
    for (int i = 0; i < KPV; ++i) {
        const int sl = (KPV * kq + i) & 15;
        const int se = min(sl, max(len - 1, 0));
        r.v[i] = *reinterpret_cast<const u32x4_t*>(base + se * D + dc * 8);
    }
}

template <int D, int KSTR, int VSTR>
__device__ __forceinline__ void stage_store(const StageRegs<D>& r, uint16_t* Ks, uint16_t* Vt, int tid) {
    constexpr int DCH = StageRegs<D>::DCH;
#pragma unroll
    for (int i = 0; i < StageRegs<D>::KPT; ++i) {
        const int c = tid + kThreads * i;
        const int dc = c % DCH, key = c / DCH;
        *reinterpret_cast<u32x4_t*>(&Ks[key * KSTR + dc * 8]) = r.k[i];
    }
    const int kq = tid / DCH, dc = tid % DCH;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        // dim 8dc+e of consecutive keys -> bf16 pairs (key 2m in the low half)
        const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
        if constexpr (D == 128) {
            uint2 out;
            out.x = __builtin_amdgcn_perm(r.v[1][e >> 1], r.v[0][e >> 1], sel);
            out.y = __builtin_amdgcn_perm(r.v[3][e >> 1], r.v[2][e >> 1], sel);
            *reinterpret_cast<uint2*>(&Vt[(dc * 8 + e) * VSTR + 4 * kq]) = out;
        } else {
            *reinterpret_cast<uint32_t*>(&Vt[(dc * 8 + e) * VSTR + 2 * kq]) =
                __builtin_amdgcn_perm(r.v[1][e >> 1], r.v[0][e >> 1], sel);
        }
    }
}

// Per-lane view of the current item's query row: lane (wave w, column c) owns tile row 16w + c,
// i.e. query token t = row / G of the tile and head g = row % G of the item's KV head.
template <int D>
struct RowState {
    int qtok, limit, slot, h;
    bool row_ok, wave_active;
    bf16x8_t qf[D / 32];  // this row's query, k-step ks holding dims 32ks + 8kg .. +7
};

// Rows of a stage's item from its decoded header and this lane's token entry (loaded a step
// earlier, so the query loads below depend on nothing in flight).  A row past the tile reads
// token 0's entry of the descriptor (zero-filled) and is never written.
template <int D>
__device__ __forceinline__ void make_rows(RowState<D>& rs, const StageInfo& si, const int4& tk,
                                          const uint16_t* __restrict__ q, int hq, int G, int wave, int t, int g,
                                          int kg) {
    rs.row_ok = t < si.n_tok;
    rs.wave_active = wave * 16 < si.n_tok * G;
    rs.qtok = tk.x;
    rs.limit = tk.y;
    rs.slot = tk.z;
    rs.h = si.kvh * G + g;
    const uint16_t* qrow = q + (static_cast<size_t>(rs.qtok) * hq + rs.h) * D + kg * 8;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) rs.qf[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qrow + ks * 32));
}

// Workgroup barrier that orders LDS only.  __syncthreads() also waits for every outstanding global
// load (its release fence), which would drain the K/V prefetch at each stage.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Compute-side state of the current item.
template <int D>
struct Acc {
    f32x4_t acc[D / 16];
    float m_run, l_run;
    __device__ __forceinline__ void reset() {
#pragma unroll
        for (int c = 0; c < D / 16; ++c) acc[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        m_run = -INFINITY;
        l_run = 0.f;
    }
};

template <int D, int KSTR, int VSTR>
__device__ __forceinline__ void contract_stage(Acc<D>& A, const RowState<D>& rs, const StageInfo& sb,
                                               const uint16_t* Ks, const uint16_t* Vt, int col, int kg, float sl2) {
    constexpr int NKS = D / 32, NCT = D / 16;
    f32x4_t s[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
        s[st] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            const uint4 a = *reinterpret_cast<const uint4*>(&Ks[(st * 16 + col) * KSTR + ks * 32 + kg * 8]);
            s[st] = mfma_16x16x32(as_bf16x8(a), rs.qf[ks], s[st]);
        }
    }
    // lane holds keys st*16 + 4*kg + r (r = 0..3) of its query row.  Masking is needed only when a
    // block is partial or some row of the wave has a causal limit inside the stage (wave-uniform).
    const bool row_full = sb.len[0] + sb.len[1] + sb.len[2] + sb.len[3] == 64 && rs.limit >= sb.pos[0] + 63;
    if (__builtin_amdgcn_ballot_w64(!row_full) != 0) {
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            const int vlen = min(sb.len[st], rs.limit - sb.pos[st] + 1);  // visible slots of this block
#pragma unroll
            for (int r = 0; r < 4; ++r)
                if (4 * kg + r >= vlen) s[st][r] = -INFINITY;
        }
    }
    float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                     fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
    mx = fmaxf(mx, fmaxf(fmaxf(fmaxf(s[2][0], s[2][1]), fmaxf(s[2][2], s[2][3])),
                         fmaxf(fmaxf(s[3][0], s[3][1]), fmaxf(s[3][2], s[3][3]))));
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(A.m_run, mx);
    // exp2(-inf) = 0, so masked keys need no select; a row with no visible key yet keeps msc = 0
    const float msc = m_new == -INFINITY ? 0.f : m_new * sl2;
    float psum = 0.f;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            s[st][r] = __builtin_amdgcn_exp2f(fmaf(s[st][r], sl2, -msc));
            psum += s[st][r];
        }
    const float alpha = m_new == A.m_run ? 1.f : __builtin_amdgcn_exp2f(A.m_run * sl2 - msc);
    A.l_run = fmaf(A.l_run, alpha, psum);
    A.m_run = m_new;
    if (__builtin_amdgcn_ballot_w64(alpha != 1.f) != 0) {  // rescale only when some row's max grew
#pragma unroll
        for (int c = 0; c < NCT; ++c) A.acc[c] *= alpha;
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
        // k index e of this lane: keys 32kk + 4kg + e (e < 4) and 32kk + 16 + 4kg + (e - 4)
        uint4 pu;
        pu.x = pack_bf16x2(s[2 * kk][0], s[2 * kk][1]);
        pu.y = pack_bf16x2(s[2 * kk][2], s[2 * kk][3]);
        pu.z = pack_bf16x2(s[2 * kk + 1][0], s[2 * kk + 1][1]);
        pu.w = pack_bf16x2(s[2 * kk + 1][2], s[2 * kk + 1][3]);
        const bf16x8_t pf = as_bf16x8(pu);
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            const uint16_t* vrow = &Vt[(ct * 16 + col) * VSTR + kk * 32 + kg * 4];
            const uint2 lo = *reinterpret_cast<const uint2*>(vrow);
            const uint2 hi = *reinterpret_cast<const uint2*>(vrow + 16);
            A.acc[ct] = mfma_16x16x32(as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y)), pf, A.acc[ct]);
        }
    }
}

template <int D>
__device__ __forceinline__ void write_item(const Acc<D>& A, const RowState<D>& rs, int kg, uint16_t* __restrict__ o,
                                           float* __restrict__ lse, float* __restrict__ po, float* __restrict__ plse,
                                           int hq, float sl2) {
    constexpr int NCT = D / 16;
    float l_tot = A.l_run + __shfl_xor(A.l_run, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (!rs.row_ok) return;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse_v = l_tot > 0.f ? (A.m_run * sl2 + log2f(l_tot)) * 0.6931471805599453f : -INFINITY;
    // lane holds output columns ct*16 + 4*kg + r of its row
    if (rs.slot < 0) {
        uint16_t* orow = o + (static_cast<size_t>(rs.qtok) * hq + rs.h) * D;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            uint2 w;
            w.x = pack_bf16x2(A.acc[ct][0] * inv, A.acc[ct][1] * inv);
            w.y = pack_bf16x2(A.acc[ct][2] * inv, A.acc[ct][3] * inv);
            *reinterpret_cast<uint2*>(orow + ct * 16 + kg * 4) = w;
        }
        if (lse && kg == 0) lse[static_cast<size_t>(rs.qtok) * hq + rs.h] = lse_v;
    } else {
        float* prow = po + (static_cast<size_t>(rs.slot) * hq + rs.h) * D;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            *reinterpret_cast<float4*>(prow + ct * 16 + kg * 4) =
                make_float4(A.acc[ct][0] * inv, A.acc[ct][1] * inv, A.acc[ct][2] * inv, A.acc[ct][3] * inv);
        if (kg == 0) plse[static_cast<size_t>(rs.slot) * hq + rs.h] = lse_v;
    }
}

// One workgroup per resident slot (persistent): it walks the planner's stream of 64-key stages
// for this slot (items split into stages, items back to back).  While stage k is contracted from
// LDS, stage k+1's K/V and its item's query rows are in flight into registers, and stage k+2's
// descriptor is in flight too -- every load of the loop body is straight-line and depends on
// nothing issued in the same step.  At an item boundary the rows are swapped in by selects.
template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3, 3))) void attn_persist(
    const tkv::StageDesc* __restrict__ stages, const int32_t* __restrict__ wg_off, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ kpool, const uint16_t* __restrict__ vpool, uint16_t* __restrict__ o,
    float* __restrict__ lse, float* __restrict__ po, float* __restrict__ plse, int hq, int hkv, int G, float sl2) {
    constexpr int KSTR = D + 8;                // K row stride in LDS (elements): 16-B reads spread over banks
    constexpr int VSTR = kKeysPerStage + 4;    // V^T row stride (elements): 8-B reads of 16 rows spread over banks
    __shared__ __attribute__((aligned(16))) uint16_t Ks[kKeysPerStage * KSTR];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VSTR];

    const int s0 = wg_off[blockIdx.x], s1 = wg_off[blockIdx.x + 1];
    if (s0 >= s1) return;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const int col = lane & 15, kg = lane >> 4;
    const int mrow = wave * 16 + col;  // this lane's row of the tile (token-major, head-minor)
    const int t = mrow / G, g = mrow - t * G;
    const int trow = min(t, tkv::kTileRows - 1);

    int4 h = load_hdr(stages, s0, lane);
    int4 tk = load_tok(stages, s0, trow);
    StageInfo si = decode_hdr(h);
    StageRegs<D> r;
    stage_load<D>(r, h, true, si.kvh, kpool, vpool, hkv, tid, wave_u);
    RowState<D> rs, rs_n;
    make_rows<D>(rs, si, tk, q, hq, G, wave, t, g, kg);
    int gnext = s0 + 1;  // next stage to fetch
    h = load_hdr(stages, min(gnext, s1 - 1), lane);
    tk = load_tok(stages, min(gnext, s1 - 1), trow);
    Acc<D> A;
    A.reset();

    for (;;) {
        const StageInfo cur = si;
        lds_barrier();  // the previous stage's LDS reads are done
        stage_store<D, KSTR, VSTR>(r, Ks, Vt, tid);
        lds_barrier();
        const bool has_next = gnext < s1;
        si = decode_hdr(h);
        make_rows<D>(rs_n, si, tk, q, hq, G, wave, t, g, kg);
        stage_load<D>(r, h, has_next, si.kvh, kpool, vpool, hkv, tid, wave_u);
        ++gnext;
        h = load_hdr(stages, min(gnext, s1 - 1), lane);
        tk = load_tok(stages, min(gnext, s1 - 1), trow);
        if (__builtin_amdgcn_readfirstlane(rs.wave_active))
            contract_stage<D, KSTR, VSTR>(A, rs, cur, Ks, Vt, col, kg, sl2);
        const bool last = cur.flags & tkv::kStageLast;
        if (last) {
            write_item<D>(A, rs, kg, o, lse, po, plse, hq, sl2);
            if (!has_next) break;
            A.reset();
        }
        rs.qtok = last ? rs_n.qtok : rs.qtok;
        rs.limit = last ? rs_n.limit : rs.limit;
        rs.slot = last ? rs_n.slot : rs.slot;
        rs.h = last ? rs_n.h : rs.h;
        rs.row_ok = last ? rs_n.row_ok : rs.row_ok;
        rs.wave_active = last ? rs_n.wave_active : rs.wave_active;
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) rs.qf[ks] = last ? rs_n.qf[ks] : rs.qf[ks];
    }
}

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

// One 16-key block against the wave's T tiles; the block's registers are refilled with the next
// block of the wave's stream as soon as each half (K, then V) has been consumed.
template <int D, int T, int VROW>
__device__ __forceinline__ void wave_block(WaveAcc<D, T>& A, BlockRegs<D>& r, const bf16x8_t (&qf)[T][D / 32],
                                           int len, int pos, const int (&limit)[T],
                                           const uint16_t* __restrict__ kpool, const uint16_t* __restrict__ vpool,
                                           size_t boff_n, int len_n, uint8_t* vs, const uint8_t* vrd, int lane,
                                           int kg, float sl2) {
    // S^T = K Q^T for every tile (independent MFMA chains), then the K registers take the next loads
    f32x4_t s[T];
#pragma unroll
    for (int tt = 0; tt < T; ++tt) s[tt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
#pragma unroll
        for (int tt = 0; tt < T; ++tt) s[tt] = mfma_16x16x32(__builtin_bit_cast(bf16x8_t, r.k[ks]), qf[tt][ks], s[tt]);
    load_k<D>(r, kpool, boff_n, len_n, lane);
    s16x4_t pb[T];
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        // lane holds keys 4kg + e of its row; mask only partial blocks and rows with a causal limit inside
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
    // V rows into this wave's LDS region, then the V registers take the next loads
#pragma unroll
    for (int i = 0; i < D / 32; ++i) {
        const int c = lane + 64 * i;
        *reinterpret_cast<u32x4_t*>(vs + (c / (D / 8)) * VROW + (c % (D / 8)) * 16) = r.v[i];
    }
    load_v<D>(r, vpool, boff_n, len_n, lane);
    // O^T += V^T P^T: P^T as the S^T result sits in the lanes, V^T by transposing LDS reads
#pragma unroll
    for (int ct = 0; ct < D / 16; ++ct) {
        const s16x4_t va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4_t*)(const_cast<uint8_t*>(vrd + ct * 32)));
#pragma unroll
        for (int tt = 0; tt < T; ++tt)
            A.acc[tt][ct] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, pb[tt], A.acc[tt][ct], 0, 0, 0);
    }
}

// One wave's list of items [e0, e1), all of T column tiles.  The next key block is always in
// flight, across item boundaries too (the last block of an item prefetches the first of the next);
// the next item's descriptor is fetched at the start of an item.
template <int D, int T>
__device__ __forceinline__ void wave_run(const int4* __restrict__ wdesc, int e0, int e1,
                                         const uint16_t* __restrict__ q, const uint16_t* __restrict__ kpool,
                                         const uint16_t* __restrict__ vpool, uint16_t* __restrict__ o,
                                         float* __restrict__ lse, float* __restrict__ po, float* __restrict__ plse,
                                         int hq, int hkv, int G, float sl2, uint8_t* vs, int lane) {
    constexpr int VROW = 2 * D + 32;  // LDS bytes per V row: the padding spreads 4 rows over 32 banks
    const int col = lane & 15, kg = lane >> 4;
    int tok[T], grp[T];
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        const int row = 16 * tt + col;
        tok[tt] = min(row / G, tkv::kWaveToks - 1);
        grp[tt] = row - (row / G) * G;
    }
    const size_t blk_stride = static_cast<size_t>(hkv) * (16 * D);
    const uint8_t* vrd = vs + (4 * kg + (col >> 2)) * VROW + (4 * (col & 3)) * 2;

    int4 dc = wdesc[static_cast<size_t>(e0) * 64 + lane];
    int4 dn = wdesc[static_cast<size_t>(min(e0 + 1, e1 - 1)) * 64 + lane];
    WaveItem<T> ic = wave_item<T>(dc, tok, grp, G);
    bf16x8_t qf[T][D / 32];
    load_q<D, T>(qf, q, ic, hq, kg);
    BlockRegs<D> r;
    {
        const int len0 = __builtin_amdgcn_readlane(dc.y, 0);
        const size_t b0 = static_cast<size_t>(__builtin_amdgcn_readlane(dc.x, 0)) * blk_stride +
                          static_cast<size_t>(ic.kvh) * (16 * D);
        load_k<D>(r, kpool, b0, len0, lane);
        load_v<D>(r, vpool, b0, len0, lane);
    }
    WaveAcc<D, T> A;
    for (int e = e0;; ++e) {
        const bool more = e + 1 < e1;
        const size_t kvh_off = static_cast<size_t>(ic.kvh) * (16 * D);
        const size_t kvh_off_n = static_cast<size_t>(__builtin_amdgcn_readlane(dn.w, 0)) * (16 * D);
        A.reset();
        const int nb = ic.nb;
        for (int b = 0; b < nb; ++b) {
            // the block after this one: the next of this item, or the first of the next item
            // (a lane-wise select of the descriptor, then v_readlane: no branches)
            const bool last = b + 1 == nb;
            const int bn = last ? 0 : b + 1;
            const int src_x = last ? dn.x : dc.x;
            const int src_y = last ? (more ? dn.y : 0) : dc.y;
            const size_t boff_n = static_cast<size_t>(__builtin_amdgcn_readlane(src_x, bn)) * blk_stride +
                                  (last ? kvh_off_n : kvh_off);
            wave_block<D, T, VROW>(A, r, qf, __builtin_amdgcn_readlane(dc.y, b), __builtin_amdgcn_readlane(dc.z, b),
                                   ic.limit, kpool, vpool, boff_n, __builtin_amdgcn_readlane(src_y, bn), vs, vrd,
                                   lane, kg, sl2);
        }
        // normalise and write each tile's final output or partial
#pragma unroll
        for (int tt = 0; tt < T; ++tt) {
            float l_tot = A.l[tt] + __shfl_xor(A.l[tt], 16);
            l_tot += __shfl_xor(l_tot, 32);
            if (!ic.ok[tt]) continue;
            const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
            const float lse_v = l_tot > 0.f ? (A.m[tt] * sl2 + log2f(l_tot)) * 0.6931471805599453f : -INFINITY;
            if (ic.slot[tt] < 0) {
                uint16_t* orow = o + (static_cast<size_t>(ic.qtok[tt]) * hq + ic.h[tt]) * D;
#pragma unroll
                for (int ct = 0; ct < D / 16; ++ct) {
                    uint2 wv;
                    wv.x = pack_bf16x2(A.acc[tt][ct][0] * inv, A.acc[tt][ct][1] * inv);
                    wv.y = pack_bf16x2(A.acc[tt][ct][2] * inv, A.acc[tt][ct][3] * inv);
                    *reinterpret_cast<uint2*>(orow + ct * 16 + kg * 4) = wv;
                }
                if (lse && kg == 0) lse[static_cast<size_t>(ic.qtok[tt]) * hq + ic.h[tt]] = lse_v;
            } else {
                float* prow = po + (static_cast<size_t>(ic.slot[tt]) * hq + ic.h[tt]) * D;
#pragma unroll
                for (int ct = 0; ct < D / 16; ++ct)
                    *reinterpret_cast<float4*>(prow + ct * 16 + kg * 4) =
                        make_float4(A.acc[tt][ct][0] * inv, A.acc[tt][ct][1] * inv, A.acc[tt][ct][2] * inv,
                                    A.acc[tt][ct][3] * inv);
                if (kg == 0) plse[static_cast<size_t>(ic.slot[tt]) * hq + ic.h[tt]] = lse_v;
            }
        }
        if (!more) break;
        dc = dn;
        dn = wdesc[static_cast<size_t>(min(e + 2, e1 - 1)) * 64 + lane];
        ic = wave_item<T>(dc, tok, grp, G);
        load_q<D, T>(qf, q, ic, hq, kg);
    }
}

// Each wave walks its own list of items (a contiguous range of the descriptor stream) with no
// barrier; its tile width T (1..3 tiles of 16 query rows) is fixed per wave by the planner.
template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_wave(
    const int4* __restrict__ wdesc, const int32_t* __restrict__ woff, const int32_t* __restrict__ wtiles,
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kpool, const uint16_t* __restrict__ vpool,
    uint16_t* __restrict__ o, float* __restrict__ lse, float* __restrict__ po, float* __restrict__ plse, int hq,
    int hkv, int G, float sl2) {
    constexpr int VROW = 2 * D + 32;
    __shared__ __attribute__((aligned(16))) uint8_t Vs[4][16 * VROW];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int w = blockIdx.x * 4 + wave;
    const int e0 = woff[w], e1 = woff[w + 1], T = wtiles[w];
    if (e0 >= e1) return;  // waves are independent: no barrier follows
    if (T == 1)
        wave_run<D, 1>(wdesc, e0, e1, q, kpool, vpool, o, lse, po, plse, hq, hkv, G, sl2, Vs[wave], lane);
    else if (T == 2)
        wave_run<D, 2>(wdesc, e0, e1, q, kpool, vpool, o, lse, po, plse, hq, hkv, G, sl2, Vs[wave], lane);
    else
        wave_run<D, 3>(wdesc, e0, e1, q, kpool, vpool, o, lse, po, plse, hq, hkv, G, sl2, Vs[wave], lane);
}

// Log-sum-exp merge of one query token's partials (one workgroup per token, whose partial slots
// are contiguous): every thread owns float4 columns of one head and folds the partials in with an
// online softmax, eight partials' outputs and lse values in flight at a time -- one round of
// memory latency per eight partials, no barriers.
template <int D>
__global__ __launch_bounds__(kThreads) void merge_partials(const tkv::MergeDesc* __restrict__ md,
                                                           const float* __restrict__ po,
                                                           const float* __restrict__ plse,
                                                           uint16_t* __restrict__ o, float* __restrict__ lse, int hq) {
    constexpr int C4 = D / 4;
    const tkv::MergeDesc m = md[blockIdx.x];
    const size_t s0 = static_cast<size_t>(m.slot_off);
    const int n = m.n_slots;
    const float4* po4 = reinterpret_cast<const float4*>(po);
    for (int idx = threadIdx.x; idx < hq * C4; idx += kThreads) {
        const int h = idx / C4;
        float mx = -INFINITY, sum = 0.f;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int j0 = 0; j0 < n; j0 += 8) {
            float4 x[8];
            float lj[8];
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                const size_t sl = s0 + min(j0 + v, n - 1);
                x[v] = po4[(sl * hq) * C4 + idx];
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

}  // namespace

namespace tkv {

int upload(tkv_plan* p, void* d_ws, size_t bytes, void* stream) {
    (void)bytes;
    if (p->desc_bytes) {
        const hipError_t e = hipMemcpyAsync(d_ws, p->image.data(), p->desc_bytes, hipMemcpyHostToDevice,
                                            static_cast<hipStream_t>(stream));
        if (e != hipSuccess) return set_error(TKV_EHIP, "tkv_plan_upload: hipMemcpyAsync: %s", hipGetErrorString(e));
    }
    p->d_ws = d_ws;
    return TKV_OK;
}

template <int D>
static int launch_d(const tkv_plan* p, const void* q, const void* k, const void* v, void* o, float* lse,
                    hipStream_t st) {
    uint8_t* ws = static_cast<uint8_t*>(p->d_ws);
    const auto* merges = reinterpret_cast<const MergeDesc*>(ws + p->off_merges);
    const auto* wg_off = reinterpret_cast<const int32_t*>(ws + p->off_wg);
    const auto* stages = reinterpret_cast<const StageDesc*>(ws + p->off_stages);
    const auto* wdesc = reinterpret_cast<const int4*>(ws + p->off_wdesc);
    const auto* woff = reinterpret_cast<const int32_t*>(ws + p->off_woff);
    const auto* wtiles = reinterpret_cast<const int32_t*>(ws + p->off_wtiles);
    const auto* toks = reinterpret_cast<const TokDesc*>(ws + p->off_toks);
    const auto* blks = reinterpret_cast<const BlkDesc*>(ws + p->off_blks);
    float* po = reinterpret_cast<float*>(ws + p->off_po);
    float* plse = reinterpret_cast<float*>(ws + p->off_plse);
    const float sl2 = 1.4426950408889634f / std::sqrt(static_cast<float>(D));
    const int hq = p->shape.hq, hkv = p->shape.hkv;
    // Instrumented calls time the kernels by the dispatch packets' own start/end timestamps
    // (hipExtLaunchKernelGGL events): the main phase from the start of its first kernel to the
    // end of its last, and the merge kernel.
    hipEvent_t* ev = nullptr;
    if (p->prof_n < p->prof_max) ev = reinterpret_cast<hipEvent_t*>(p->prof_events.data()) + 4 * p->prof_n++;
    const int n_wg = static_cast<int>(p->wg_off.size()) - 1;
    const int n_wave = static_cast<int>(p->wave_off.size()) - 1;  // a multiple of 4
    hipEvent_t main_start = ev ? ev[0] : nullptr, main_stop = ev ? ev[1] : nullptr;
    if (n_wg > 0)
        hipExtLaunchKernelGGL(attn_persist<D>, dim3(static_cast<unsigned>(n_wg)), dim3(kThreads), 0, st, main_start,
                              n_wave > 0 ? nullptr : main_stop, 0, stages, wg_off, static_cast<const uint16_t*>(q),
                              static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v),
                              static_cast<uint16_t*>(o), lse, po, plse, hq, hkv, p->group, sl2);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(TKV_EHIP, "attention launch: %s", hipGetErrorString(e));
    if (n_wave > 0)
        hipExtLaunchKernelGGL(attn_wave<D>, dim3(static_cast<unsigned>(n_wave / 4)), dim3(kThreads), 0, st,
                              n_wg > 0 ? nullptr : main_start, main_stop, 0, wdesc, woff, wtiles,
                              static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                              static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), lse, po, plse, hq, hkv,
                              p->group, sl2);
    e = hipGetLastError();
    if (e != hipSuccess) return set_error(TKV_EHIP, "attention launch: %s", hipGetErrorString(e));
    if (!p->merges.empty()) {
        hipExtLaunchKernelGGL(merge_partials<D>, dim3(static_cast<unsigned>(p->merges.size())), dim3(kThreads), 0, st,
                              ev ? ev[2] : nullptr, ev ? ev[3] : nullptr, 0, merges,
                              static_cast<const float*>(po), static_cast<const float*>(plse),
                              static_cast<uint16_t*>(o), lse, hq);
        e = hipGetLastError();
        if (e != hipSuccess) return set_error(TKV_EHIP, "merge launch: %s", hipGetErrorString(e));
    } else if (ev) {
        (void)hipEventRecord(ev[2], st);
        (void)hipEventRecord(ev[3], st);
    }
    return TKV_OK;
}

int launch_attention(const tkv_plan* p, const void* q, const void* k, const void* v, void* o, float* lse,
                     void* stream) {
    if (!p->d_ws) return set_error(TKV_EINVAL, "attention: plan has not been uploaded");
    if (p->items.empty() && p->wave_items.empty()) return TKV_OK;
    if (!q || !k || !v || !o) return set_error(TKV_EINVAL, "attention: NULL tensor pointer");
    const hipStream_t st = static_cast<hipStream_t>(stream);
    return p->shape.d == 128 ? launch_d<128>(p, q, k, v, o, lse, st) : launch_d<64>(p, q, k, v, o, lse, st);
}

}  // namespace tkv

static void free_events(const tkv_plan* p) {
    for (void* e : p->prof_events) (void)hipEventDestroy(static_cast<hipEvent_t>(e));
    p->prof_events.clear();
    p->prof_max = p->prof_n = 0;
}

tkv_plan::~tkv_plan() { free_events(this); }

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
