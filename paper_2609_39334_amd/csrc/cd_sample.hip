// Branching sampler of computation deduplication (Sec. 4.2).  A sequence with potential size n
// stands for n identical candidates; one decode step over it yields one row of logits, from which
// n tokens are drawn as independent trials and grouped: one child per distinct token, whose
// potential is the group's size.  The distribution is the temperature softmax of the row (Sec. 2.1).
//
// One workgroup per row, so rows of every potential size run in one launch.  A draw is the inverse
// CDF at the caller's uniform u: the first token (in token order) whose cumulative weight exceeds
// u * Z.  The row is read once, in tiles of 4,096 logits; thread t owns the 16 contiguous logits
// [16t, 16t + 16) of a tile (four 16-byte loads).  The kernel's CDF is defined by its own fp32 sums:
//   tile i: base b_i = the tile's maximum, w_j = exp2((l_j - b_i) * log2(e) / T);
//   s_t = w over thread t's 16 logits, added in token order; within a wave, an inclusive scan of
//   s_t over the lanes by a fixed shuffle pattern; the four wave totals added in order give the
//   tile total T_i and each wave's start;
//   with M the row maximum and f_i = exp2((b_i - M) * log2(e) / T), the tile prefixes
//   P_0 = 0, P_{i+1} = P_i + f_i T_i, one tile at a time, and Z = P_{n_tiles}.
//   Thread t of tile i starts at F_t = P_i + f_i (wave start + lanes before it), and its token j is
//   at F_t + f_i (w of its logits up to j, in token order).
// A draw finds the tile with P_i <= u Z < P_{i+1}, reloads it and repeats the same arithmetic; the
// thread with the largest start F_t <= u Z scans its 16 logits, and a target its rounding leaves
// past its last token goes to its last token with a weight.  Zero weights (logit -inf) are never
// drawn.  Grouping: each draw that is the first of its token counts the token's draws and writes it at
// its rank among the distinct tokens, so groups come out in ascending token order.
#include <hip/hip_runtime.h>
#include <cmath>
#include <cstdint>

#include "internal.h"

namespace {

constexpr int kSampleThreads = 256;
constexpr int kPerThread = 16;                            // contiguous logits per thread and tile
constexpr int kTile = kSampleThreads * kPerThread;        // 4,096 logits per tile
constexpr int kMaxTiles = 512;                            // vocabulary up to 2,097,152
constexpr int kMaxPotential = 1024;                       // draws of one row (grouped in LDS)

// This thread's 16 logits of tile i (positions past the vocabulary read as -inf).
template <bool VEC>
__device__ __forceinline__ void load16(const float* __restrict__ row, int vocab, int i, int t, float (&x)[kPerThread]) {
    const int a = i * kTile + t * kPerThread;
    if (VEC && a + kPerThread <= vocab) {
        const float4* r4 = reinterpret_cast<const float4*>(row + a);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float4 v = r4[k];
            x[4 * k] = v.x;
            x[4 * k + 1] = v.y;
            x[4 * k + 2] = v.z;
            x[4 * k + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < kPerThread; ++k) x[k] = a + k < vocab ? row[a + k] : -INFINITY;
    }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}

// Inclusive scan of v over the 64 lanes (fixed pattern: lane l adds lane l - 2^k when it exists).
__device__ __forceinline__ float wave_scan(float v, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const float u = __shfl_up(v, o);
        if (lane >= o) v += u;
    }
    return v;
}

// Sum of this thread's weights in token order, each w = exp2((x - b) * c).
__device__ __forceinline__ float thread_sum(const float (&x)[kPerThread], float b, float c) {
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) s += __builtin_amdgcn_exp2f((x[k] - b) * c);
    return s;
}

template <bool VEC>
__global__ __launch_bounds__(kSampleThreads) void cd_sample(const float* __restrict__ logits, int vocab, float c,
                                                            const float* __restrict__ uniform,
                                                            const int32_t* __restrict__ draw_off, int32_t n_draws,
                                                            int32_t* __restrict__ out_tok, int32_t* __restrict__ out_cnt,
                                                            int32_t* __restrict__ n_groups) {
    __shared__ float base[kMaxTiles];       // b_i
    __shared__ float tsum[kMaxTiles];       // T_i, then f_i T_i
    __shared__ float P[kMaxTiles + 1];      // tile prefixes
    __shared__ float wred[4];               // per-wave maxima, then wave totals
    __shared__ float target[kMaxPotential];
    __shared__ int32_t tok[kMaxPotential];
    __shared__ int32_t first[kMaxPotential];
    __shared__ int32_t tile_of[kMaxPotential];
    const int r = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
    const float* row = logits + static_cast<size_t>(r) * vocab;
    const int off = draw_off[r], n = draw_off[r + 1] - off;
    const int n_tiles = (vocab + kTile - 1) / kTile;
    // a row whose draws fall outside the caller's arrays (offsets are device data the host cannot
    // check), or too many of them, is refused before anything of it is read or written
    if (n < 0 || off < 0 || static_cast<int64_t>(off) + n > n_draws || n > kMaxPotential || n_tiles > kMaxTiles) {
        if (t == 0) n_groups[r] = -1;
        return;
    }

    // one pass over the row: per tile its maximum and its total over that base (the next tile's
    // loads in flight while one is reduced)
    float x[kPerThread], xn[kPerThread];
    float mx = -INFINITY;
    load16<VEC>(row, vocab, 0, t, xn);
    for (int i = 0; i < n_tiles; ++i) {
#pragma unroll
        for (int k = 0; k < kPerThread; ++k) x[k] = xn[k];
        if (i + 1 < n_tiles) load16<VEC>(row, vocab, i + 1, t, xn);
        float m = x[0];
#pragma unroll
        for (int k = 1; k < kPerThread; ++k) m = fmaxf(m, x[k]);
        m = wave_max(m);
        if (lane == 0) wred[w] = m;
        __syncthreads();
        const float b = fmaxf(fmaxf(wred[0], wred[1]), fmaxf(wred[2], wred[3]));
        __syncthreads();
        mx = fmaxf(mx, b);
        const float s = b == -INFINITY ? 0.f : thread_sum(x, b, c);
        const float incl = wave_scan(s, lane);
        if (lane == 63) wred[w] = incl;
        __syncthreads();
        if (t == 0) {
            base[i] = b;
            tsum[i] = ((wred[0] + wred[1]) + wred[2]) + wred[3];
        }
        __syncthreads();
    }
    if (mx == -INFINITY) {  // no finite logit: no distribution
        if (t == 0) n_groups[r] = -1;
        return;
    }
    if (t == 0) {
        P[0] = 0.f;
        for (int i = 0; i < n_tiles; ++i) {
            const float f = base[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((base[i] - mx) * c);
            tsum[i] = f * tsum[i];
            P[i + 1] = P[i] + tsum[i];
        }
    }
    __syncthreads();
    const float Z = P[n_tiles];

    // each draw's target and tile (first tile with P[i + 1] > target; n_tiles if u Z rounded up to Z)
    for (int k = t; k < n; k += kSampleThreads) {
        const float tg = uniform[off + k] * Z;
        int lo = 0, hi = n_tiles;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (P[mid + 1] > tg) hi = mid; else lo = mid + 1;
        }
        target[k] = tg;
        tile_of[k] = lo;
        tok[k] = -1;
    }
    __syncthreads();

    // resolve the draws tile by tile: reload a tile that holds a draw and repeat its arithmetic
    for (int i = 0; i < n_tiles; ++i) {
        int any = 0;
        for (int k = t; k < n; k += kSampleThreads) any |= tile_of[k] == i;
        if (__syncthreads_or(any) == 0) continue;
        load16<VEC>(row, vocab, i, t, x);
        const float b = base[i];
        const float f = __builtin_amdgcn_exp2f((b - mx) * c);
        const float s = thread_sum(x, b, c);
        const float incl = wave_scan(s, lane);
        float excl = __shfl_up(incl, 1);
        if (lane == 0) excl = 0.f;
        if (lane == 63) wred[w] = incl;
        __syncthreads();
        const float wstart = w == 0 ? 0.f : w == 1 ? wred[0] : w == 2 ? wred[0] + wred[1] : (wred[0] + wred[1]) + wred[2];
        const float start = P[i] + f * (wstart + excl);
        // the next thread's start bounds this thread's targets (the tile's last thread: P[i + 1])
        float nxt = __shfl_down(start, 1);
        const float next_wave_first = w < 3 ? P[i] + f * (w == 0 ? wred[0] : w == 1 ? wred[0] + wred[1]
                                                                                   : (wred[0] + wred[1]) + wred[2])
                                            : P[i + 1];
        if (lane == 63) nxt = next_wave_first;
        for (int k = 0; k < n; ++k) {
            if (tile_of[k] != i) continue;
            const float tg = target[k];
            if (!(start <= tg && tg < nxt)) continue;
            const int a = i * kTile + t * kPerThread;
            int pick = -1, last = -1;
            float acc = 0.f;
#pragma unroll
            for (int q = 0; q < kPerThread; ++q) {
                const float wq = __builtin_amdgcn_exp2f((x[q] - b) * c);
                acc += wq;
                if (wq > 0.f) last = a + q;
                if (pick < 0 && wq > 0.f && start + f * acc > tg) pick = a + q;
            }
            tok[k] = pick >= 0 ? pick : last;
        }
        __syncthreads();
    }
    // targets that no thread claimed (u Z rounded up to Z, or the gap before a zero-weight run):
    // the last token with a weight at or before the target's tile end
    for (int k = t; k < n; k += kSampleThreads) {
        if (tok[k] >= 0) continue;
        int j = min(vocab, (min(tile_of[k], n_tiles - 1) + 1) * kTile) - 1;
        while (j > 0 && row[j] == -INFINITY) --j;
        tok[k] = j;
    }
    __syncthreads();

    // group: first occurrences count their token's draws and go to their rank among distinct tokens
    for (int k = t; k < n; k += kSampleThreads) {
        bool is_first = true;
        for (int j = 0; j < k && is_first; ++j) is_first = tok[j] != tok[k];
        first[k] = is_first ? 1 : 0;
    }
    __syncthreads();
    int mine = 0;
    for (int k = t; k < n; k += kSampleThreads) {
        if (!first[k]) continue;
        int cnt = 0, rank = 0;
        for (int j = 0; j < n; ++j) {
            cnt += tok[j] == tok[k];
            rank += first[j] && tok[j] < tok[k];
        }
        out_tok[off + rank] = tok[k];
        out_cnt[off + rank] = cnt;
        ++mine;
    }
    for (int o = 32; o > 0; o >>= 1) mine += __shfl_xor(mine, o);
    __syncthreads();
    if (lane == 0) wred[w] = __int_as_float(mine);
    __syncthreads();
    if (t == 0)
        n_groups[r] = __float_as_int(wred[0]) + __float_as_int(wred[1]) + __float_as_int(wred[2]) + __float_as_int(wred[3]);
}

}  // namespace

TKV_EXPORT int tkv_cd_sample(int32_t n_rows, int32_t vocab, float temperature, int32_t max_potential,
                             const float* d_logits, const float* d_uniform, const int32_t* d_draw_off,
                             int32_t n_draws, int32_t* d_token, int32_t* d_count, int32_t* d_n_groups, void* stream) {
    tkv::clear_error();
    if (n_rows < 0 || vocab < 1) return tkv::set_error(TKV_EINVAL, "tkv_cd_sample: n_rows %d, vocab %d", n_rows, vocab);
    if (vocab > kMaxTiles * kTile)
        return tkv::set_error(TKV_EINVAL, "tkv_cd_sample: vocabulary %d exceeds %d", vocab, kMaxTiles * kTile);
    if (!(temperature > 0.f) || !std::isfinite(temperature))
        return tkv::set_error(TKV_EINVAL, "tkv_cd_sample: temperature must be positive and finite");
    if (max_potential < 0 || max_potential > kMaxPotential)
        return tkv::set_error(TKV_EINVAL, "tkv_cd_sample: potential up to %d per row (got %d)", kMaxPotential, max_potential);
    if (n_draws < 0) return tkv::set_error(TKV_EINVAL, "tkv_cd_sample: n_draws = %d < 0", n_draws);
    if (n_rows == 0) return TKV_OK;
    if (!d_logits || !d_draw_off || !d_n_groups || (n_draws > 0 && (!d_uniform || !d_token || !d_count)))
        return tkv::set_error(TKV_EINVAL, "tkv_cd_sample: NULL pointer");
    // 16-byte loads when every row starts 16-byte aligned
    const bool vec = vocab % 4 == 0 && reinterpret_cast<uintptr_t>(d_logits) % 16 == 0;
    const float c = 1.4426950408889634f / temperature;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    if (vec)
        hipLaunchKernelGGL(cd_sample<true>, dim3(static_cast<unsigned>(n_rows)), dim3(kSampleThreads), 0, st, d_logits,
                           vocab, c, d_uniform, d_draw_off, n_draws, d_token, d_count, d_n_groups);
    else
        hipLaunchKernelGGL(cd_sample<false>, dim3(static_cast<unsigned>(n_rows)), dim3(kSampleThreads), 0, st, d_logits,
                           vocab, c, d_uniform, d_draw_off, n_draws, d_token, d_count, d_n_groups);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return tkv::set_error(TKV_EHIP, "tkv_cd_sample launch: %s", hipGetErrorString(e));
    return TKV_OK;
}
