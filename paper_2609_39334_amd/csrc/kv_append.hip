// K/V append: the step before attention in a decode loop.  The K and V rows of new tokens (the
// model's projections of them) go to the pool slots the block manager gave them -- tkv_bm_append for
// tokens decoded one at a time, tkv_extend_slots for a completed step -- and a token whose block was
// a deduplication hit (slot -1) is not written at all: the block already holds the same tokens' K/V
// (computation deduplication, Sec. 4.2).
//
// HBM-bound scatter: every thread moves one 16-byte chunk of one (token, KV head) row of K and of V.
// Reads of the new rows are contiguous; each row lands as one contiguous run of d bf16 in its block.
#include <hip/hip_runtime.h>
#include <cstdint>

#include "internal.h"

namespace {

constexpr int kAppendThreads = 256;

template <int D>
__global__ __launch_bounds__(kAppendThreads) void kv_append(const int32_t* __restrict__ dst, int64_t n_chunks,
                                                            int hkv, int32_t n_slots, const uint4* __restrict__ k_new,
                                                            const uint4* __restrict__ v_new, uint4* __restrict__ kpool,
                                                            uint4* __restrict__ vpool) {
    constexpr int CPR = D / 8;  // 16-byte chunks per row
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kAppendThreads + threadIdx.x;
    if (i >= n_chunks) return;
    const int64_t row = i / CPR;  // (token, KV head) row of the new K/V
    const int c = static_cast<int>(i - row * CPR);
    const int64_t t = row / hkv;
    const int h = static_cast<int>(row - t * hkv);
    const int32_t slot = dst[t];
    if (slot < 0 || slot >= n_slots) return;  // a deduplicated block (or no slot): nothing to write
    const int64_t blk = slot / tkv::kBlock, pos = slot - blk * tkv::kBlock;
    const int64_t out = ((blk * hkv + h) * tkv::kBlock + pos) * CPR + c;
    kpool[out] = k_new[i];
    vpool[out] = v_new[i];
}

}  // namespace

TKV_EXPORT int tkv_kv_append(const tkv_shape* shape, const int32_t* d_dst, int32_t n_tok, const void* k_new,
                             const void* v_new, void* k, void* v, void* stream) {
    tkv::clear_error();
    if (!shape) return tkv::set_error(TKV_EINVAL, "tkv_kv_append: shape is NULL");
    const tkv_shape s = *shape;
    if (s.block_size != tkv::kBlock) return tkv::set_error(TKV_EINVAL, "tkv_kv_append: block_size must be 16 (got %d)", s.block_size);
    if (s.d != 64 && s.d != 128) return tkv::set_error(TKV_EINVAL, "tkv_kv_append: head_dim must be 64 or 128 (got %d)", s.d);
    if (s.hkv < 1 || s.num_blocks < 1) return tkv::set_error(TKV_EINVAL, "tkv_kv_append: hkv and num_blocks must be >= 1");
    if (static_cast<int64_t>(s.num_blocks) * s.block_size > INT32_MAX)
        return tkv::set_error(TKV_EINVAL, "tkv_kv_append: %d blocks exceed the int32 slot range", s.num_blocks);
    if (n_tok < 0) return tkv::set_error(TKV_EINVAL, "tkv_kv_append: n_tok = %d < 0", n_tok);
    if (n_tok == 0) return TKV_OK;
    if (!d_dst || !k_new || !v_new || !k || !v) return tkv::set_error(TKV_EINVAL, "tkv_kv_append: NULL pointer");
    const int64_t n_chunks = static_cast<int64_t>(n_tok) * s.hkv * (s.d / 8);
    const int64_t grid = (n_chunks + kAppendThreads - 1) / kAppendThreads;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    const int32_t n_slots = s.num_blocks * s.block_size;
    auto kn = static_cast<const uint4*>(k_new);
    auto vn = static_cast<const uint4*>(v_new);
    auto kp = static_cast<uint4*>(k);
    auto vp = static_cast<uint4*>(v);
    if (s.d == 128)
        hipLaunchKernelGGL(kv_append<128>, dim3(static_cast<unsigned>(grid)), dim3(kAppendThreads), 0, st, d_dst,
                           n_chunks, s.hkv, n_slots, kn, vn, kp, vp);
    else
        hipLaunchKernelGGL(kv_append<64>, dim3(static_cast<unsigned>(grid)), dim3(kAppendThreads), 0, st, d_dst,
                           n_chunks, s.hkv, n_slots, kn, vn, kp, vp);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return tkv::set_error(TKV_EHIP, "tkv_kv_append launch: %s", hipGetErrorString(e));
    return TKV_OK;
}
