// Tree-shared paged attention kernels for gfx950 (MI355X).
//
// attn_items: one workgroup per work item (see plan.cpp).  An item is a tile of up to 64 query
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
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "internal.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8_t, u); }

__device__ __forceinline__ f32x4_t mfma_16x16x32(bf16x8_t a, bf16x8_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint32_t bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) { return bf16_rne(lo) | (bf16_rne(hi) << 16); }

constexpr int kThreads = 256;
constexpr int kKeysPerStage = 64;  // four 16-token blocks

template <int D>
__global__ __launch_bounds__(kThreads) void attn_items(
    const tkv::ItemDesc* __restrict__ items, const tkv::TokDesc* __restrict__ toks,
    const tkv::BlkDesc* __restrict__ blks, const uint16_t* __restrict__ q, const uint16_t* __restrict__ kpool,
    const uint16_t* __restrict__ vpool, uint16_t* __restrict__ o, float* __restrict__ lse,
    float* __restrict__ po, float* __restrict__ plse, int hq, int hkv, int G, float sl2) {
    constexpr int KSTR = D + 8;                // K row stride in LDS (elements): 16-B reads spread over banks
    constexpr int VSTR = kKeysPerStage + 4;    // V^T row stride (elements)
    constexpr int NKS = D / 32;                // k-steps of the QK^T contraction
    constexpr int NCT = D / 16;                // 16-column tiles of the output
    constexpr int DCH = D / 8;                 // 16-byte chunks per K/V row
    __shared__ __attribute__((aligned(16))) uint16_t Ks[kKeysPerStage * KSTR];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VSTR];

    const tkv::ItemDesc it = items[blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, kg = lane >> 4;
    const int mrow = wave * 16 + col;  // this lane's query row in the tile (token-major, head-minor)
    const int t = mrow / G, g = mrow - t * G;
    const bool row_ok = t < it.n_tok;
    const bool wave_active = wave * 16 < it.n_tok * G;
    int qtok = 0, limit = -1, slot = -1;
    if (row_ok) {
        const tkv::TokDesc td = toks[it.tok_off + t];
        qtok = td.qtok;
        limit = td.limit;
        slot = td.slot;
    }
    const int h = it.kvh * G + g;

    bf16x8_t qf[NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
        uint4 u = make_uint4(0, 0, 0, 0);
        if (row_ok) u = *reinterpret_cast<const uint4*>(q + (static_cast<size_t>(qtok) * hq + h) * D + ks * 32 + kg * 8);
        qf[ks] = as_bf16x8(u);
    }
    f32x4_t acc[NCT];
#pragma unroll
    for (int c = 0; c < NCT; ++c) acc[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;
    int pos = it.pos0;

    for (int b0 = 0; b0 < it.n_blk; b0 += 4) {
        const int nb = min(4, it.n_blk - b0);
        int blen[4], bpos[4], bid[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int len = 0, id = 0;
            if (j < nb) {
                const tkv::BlkDesc bd = blks[it.blk_off + b0 + j];
                len = bd.len;
                id = bd.blk;
            }
            blen[j] = len;
            bid[j] = id;
            bpos[j] = pos;
            pos += len;
        }
        __syncthreads();  // the previous stage's LDS reads are done
        for (int c = tid; c < 4 * 16 * DCH; c += kThreads) {
            const int dc = c % DCH, sl = (c / DCH) & 15, j = c / (16 * DCH);
            // select rather than index, so the small arrays stay in registers
            const int len_j = j == 0 ? blen[0] : j == 1 ? blen[1] : j == 2 ? blen[2] : blen[3];
            const int id_j = j == 0 ? bid[0] : j == 1 ? bid[1] : j == 2 ? bid[2] : bid[3];
            uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
            if (sl < len_j) {
                const size_t base = ((static_cast<size_t>(id_j) * hkv + it.kvh) * 16 + sl) * D + dc * 8;
                kv = *reinterpret_cast<const uint4*>(kpool + base);
                vv = *reinterpret_cast<const uint4*>(vpool + base);
            }
            *reinterpret_cast<uint4*>(&Ks[(j * 16 + sl) * KSTR + dc * 8]) = kv;
            const uint32_t vw[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
            for (int e = 0; e < 8; ++e)
                Vt[(dc * 8 + e) * VSTR + j * 16 + sl] = static_cast<uint16_t>(vw[e >> 1] >> (16 * (e & 1)));
        }
        __syncthreads();
        if (!wave_active) continue;

        f32x4_t s[4];
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            s[st] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                const uint4 a = *reinterpret_cast<const uint4*>(&Ks[(st * 16 + col) * KSTR + ks * 32 + kg * 8]);
                s[st] = mfma_16x16x32(as_bf16x8(a), qf[ks], s[st]);
            }
        }
        // lane holds keys st*16 + 4*kg + r (r = 0..3) of its query row
        float mx = -INFINITY;
#pragma unroll
        for (int st = 0; st < 4; ++st)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int sl = 4 * kg + r;
                const bool ok = sl < blen[st] && bpos[st] + sl <= limit;
                const float v = ok ? s[st][r] : -INFINITY;
                s[st][r] = v;
                mx = fmaxf(mx, v);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx);
        float alpha = 1.f, msc = 0.f;
        if (m_new != -INFINITY) {
            alpha = exp2f((m_run - m_new) * sl2);
            msc = m_new * sl2;
        }
        float psum = 0.f;
#pragma unroll
        for (int st = 0; st < 4; ++st)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float v = s[st][r];
                const float p = v == -INFINITY ? 0.f : exp2f(fmaf(v, sl2, -msc));
                s[st][r] = p;
                psum += p;
            }
        l_run = l_run * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int c = 0; c < NCT; ++c) acc[c] *= alpha;
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
                acc[ct] = mfma_16x16x32(as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y)), pf, acc[ct]);
            }
        }
    }

    float l_tot = l_run + __shfl_xor(l_run, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (!row_ok) return;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse_v = l_tot > 0.f ? (m_run * sl2 + log2f(l_tot)) * 0.6931471805599453f : -INFINITY;
    // lane holds output columns ct*16 + 4*kg + r of its row
    if (slot < 0) {
        uint16_t* orow = o + (static_cast<size_t>(qtok) * hq + h) * D;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            uint2 w;
            w.x = pack_bf16x2(acc[ct][0] * inv, acc[ct][1] * inv);
            w.y = pack_bf16x2(acc[ct][2] * inv, acc[ct][3] * inv);
            *reinterpret_cast<uint2*>(orow + ct * 16 + kg * 4) = w;
        }
        if (lse && kg == 0) lse[static_cast<size_t>(qtok) * hq + h] = lse_v;
    } else {
        float* prow = po + (static_cast<size_t>(slot) * hq + h) * D;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            *reinterpret_cast<float4*>(prow + ct * 16 + kg * 4) =
                make_float4(acc[ct][0] * inv, acc[ct][1] * inv, acc[ct][2] * inv, acc[ct][3] * inv);
        if (kg == 0) plse[static_cast<size_t>(slot) * hq + h] = lse_v;
    }
}

template <int D>
__global__ __launch_bounds__(kThreads) void merge_partials(const tkv::MergeDesc* __restrict__ md,
                                                           const int32_t* __restrict__ mslots,
                                                           const float* __restrict__ po,
                                                           const float* __restrict__ plse,
                                                           uint16_t* __restrict__ o, float* __restrict__ lse, int hq) {
    const tkv::MergeDesc m = md[blockIdx.x];
    for (int idx = threadIdx.x; idx < hq * D; idx += kThreads) {
        const int h = idx / D, c = idx - h * D;
        float mx = -INFINITY;
        for (int j = 0; j < m.n_slots; ++j) mx = fmaxf(mx, plse[static_cast<size_t>(mslots[m.slot_off + j]) * hq + h]);
        float ws = 0.f, acc = 0.f;
        if (mx != -INFINITY) {
            for (int j = 0; j < m.n_slots; ++j) {
                const size_t sl = static_cast<size_t>(mslots[m.slot_off + j]);
                const float w = expf(plse[sl * hq + h] - mx);
                ws += w;
                acc += w * po[(sl * hq + h) * D + c];
            }
        }
        o[(static_cast<size_t>(m.qtok) * hq + h) * D + c] = static_cast<uint16_t>(bf16_rne(ws > 0.f ? acc / ws : 0.f));
        if (lse && c == 0) lse[static_cast<size_t>(m.qtok) * hq + h] = ws > 0.f ? mx + logf(ws) : -INFINITY;
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
    const auto* items = reinterpret_cast<const ItemDesc*>(ws + p->off_items);
    const auto* toks = reinterpret_cast<const TokDesc*>(ws + p->off_toks);
    const auto* blks = reinterpret_cast<const BlkDesc*>(ws + p->off_blks);
    const auto* merges = reinterpret_cast<const MergeDesc*>(ws + p->off_merges);
    const auto* mslots = reinterpret_cast<const int32_t*>(ws + p->off_mslots);
    float* po = reinterpret_cast<float*>(ws + p->off_po);
    float* plse = reinterpret_cast<float*>(ws + p->off_plse);
    const float sl2 = 1.4426950408889634f / std::sqrt(static_cast<float>(D));
    const int hq = p->shape.hq, hkv = p->shape.hkv;
    hipEvent_t* ev = nullptr;
    if (p->prof_n < p->prof_max) {
        ev = reinterpret_cast<hipEvent_t*>(p->prof_events.data()) + 3 * p->prof_n++;
        hipEventRecord(ev[0], st);
    }
    hipLaunchKernelGGL(attn_items<D>, dim3(static_cast<unsigned>(p->items.size())), dim3(kThreads), 0, st, items,
                       toks, blks, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                       static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), lse, po, plse, hq, hkv,
                       p->group, sl2);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(TKV_EHIP, "attention launch: %s", hipGetErrorString(e));
    if (ev) hipEventRecord(ev[1], st);
    if (!p->merges.empty()) {
        hipLaunchKernelGGL(merge_partials<D>, dim3(static_cast<unsigned>(p->merges.size())), dim3(kThreads), 0, st,
                           merges, mslots, po, plse, static_cast<uint16_t*>(o), lse, hq);
        e = hipGetLastError();
        if (e != hipSuccess) return set_error(TKV_EHIP, "merge launch: %s", hipGetErrorString(e));
    }
    if (ev) hipEventRecord(ev[2], st);
    return TKV_OK;
}

int launch_attention(const tkv_plan* p, const void* q, const void* k, const void* v, void* o, float* lse,
                     void* stream) {
    if (!p->d_ws) return set_error(TKV_EINVAL, "attention: plan has not been uploaded");
    if (p->items.empty()) return TKV_OK;
    if (!q || !k || !v || !o) return set_error(TKV_EINVAL, "attention: NULL tensor pointer");
    const hipStream_t st = static_cast<hipStream_t>(stream);
    return p->shape.d == 128 ? launch_d<128>(p, q, k, v, o, lse, st) : launch_d<64>(p, q, k, v, o, lse, st);
}

}  // namespace tkv

static void free_events(const tkv_plan* p) {
    for (void* e : p->prof_events) hipEventDestroy(static_cast<hipEvent_t>(e));
    p->prof_events.clear();
    p->prof_max = p->prof_n = 0;
}

tkv_plan::~tkv_plan() { free_events(this); }

TKV_EXPORT int tkv_plan_profile(tkv_plan* p, int32_t max_calls) {
    tkv::clear_error();
    if (!p || max_calls < 0) return tkv::set_error(TKV_EINVAL, "tkv_plan_profile: bad argument");
    free_events(p);
    for (int32_t i = 0; i < 3 * max_calls; ++i) {
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
        hipEvent_t* ev = reinterpret_cast<hipEvent_t*>(p->prof_events.data()) + 3 * i;
        hipError_t rc = hipEventSynchronize(ev[2]);
        float t0 = 0.f, t1 = 0.f;
        if (rc == hipSuccess) rc = hipEventElapsedTime(&t0, ev[0], ev[1]);
        if (rc == hipSuccess) rc = hipEventElapsedTime(&t1, ev[1], ev[2]);
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
