// Prefix-tree KV block manager (host, integer) and row coalescing.
//
// Paged KV with prefix sharing is the substrate the paper builds on (Sec. 5.1); candidate paths
// of one request share the blocks of their common prefix, identical candidates collapse into one
// sequence (computation deduplication, Sec. 4.2), and pruning releases a path's blocks (Sec. 4.1).
// Block-level rules (the paper states none): step-aligned blocks; a sealed chunk reuses the live
// sealed block with the same (predecessor block, exact tokens) key; misses take the lowest free id;
// refcount = live sequences holding the block; freed and unindexed at zero; lowest free sequence id.
// A 64-bit FNV-1a hash only selects a bucket -- keys are compared exactly.
// A decode loop grows a path in place (append: the open, unsealed step is private to its sequence,
// so its last block fills up before the lowest free id is taken) and completes a step (seal: each
// open block is looked up with the same key; a hit swaps in the live sealed block and frees the
// sequence's own, a miss indexes the block).
#include <algorithm>
#include <cstring>
#include <functional>
#include <queue>
#include <unordered_map>
#include <vector>

#include "internal.h"

namespace {

struct ChunkKey {
    int32_t pred;
    std::vector<int32_t> toks;
    bool operator==(const ChunkKey& o) const { return pred == o.pred && toks == o.toks; }
};

struct ChunkKeyHash {
    size_t operator()(const ChunkKey& k) const {
        uint64_t h = 1469598103934665603ull;
        auto mix = [&h](uint32_t w) {
            for (int i = 0; i < 4; ++i) {
                h ^= (w >> (8 * i)) & 0xffu;
                h *= 1099511628211ull;
            }
        };
        mix(static_cast<uint32_t>(k.pred));
        for (int32_t t : k.toks) mix(static_cast<uint32_t>(t));
        return static_cast<size_t>(h);
    }
};

using MinHeap = std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>>;

struct Seq {
    bool live = false;
    bool sealed = false;
    std::vector<int32_t> table;
    std::vector<int32_t> open;  // tokens of the open step: the last ceil(size / block_size) blocks
};

}  // namespace

struct tkv_bm {
    int32_t num_blocks = 0, block_size = 0, max_seqs = 0;
    std::vector<int32_t> refcount, block_len;
    std::vector<uint8_t> indexed;
    std::vector<ChunkKey> key;  // valid where indexed
    std::unordered_map<ChunkKey, int32_t, ChunkKeyHash> index;
    MinHeap free_blocks, free_seqs;
    std::vector<Seq> seqs;
    int32_t n_live = 0;
};

using tkv::set_error;

TKV_EXPORT int tkv_bm_create(int32_t num_blocks, int32_t block_size, int32_t max_seqs, tkv_bm** out) {
    tkv::clear_error();
    if (!out) return set_error(TKV_EINVAL, "tkv_bm_create: out is NULL");
    *out = nullptr;
    if (num_blocks < 1 || block_size < 1 || max_seqs < 1)
        return set_error(TKV_EINVAL, "tkv_bm_create: sizes must be >= 1 (got %d, %d, %d)", num_blocks,
                         block_size, max_seqs);
    tkv_bm* bm = new (std::nothrow) tkv_bm();
    if (!bm) return set_error(TKV_ENOMEM, "tkv_bm_create: host allocation failed");
    try {
        bm->num_blocks = num_blocks;
        bm->block_size = block_size;
        bm->max_seqs = max_seqs;
        bm->refcount.assign(num_blocks, 0);
        bm->block_len.assign(num_blocks, 0);
        bm->indexed.assign(num_blocks, 0);
        bm->key.resize(num_blocks);
        bm->seqs.resize(max_seqs);
        std::vector<int32_t> ids(num_blocks);
        for (int32_t i = 0; i < num_blocks; ++i) ids[i] = i;
        bm->free_blocks = MinHeap(std::greater<int32_t>(), std::move(ids));
        std::vector<int32_t> sids(max_seqs);
        for (int32_t i = 0; i < max_seqs; ++i) sids[i] = i;
        bm->free_seqs = MinHeap(std::greater<int32_t>(), std::move(sids));
    } catch (...) {
        delete bm;
        return set_error(TKV_ENOMEM, "tkv_bm_create: host allocation failed");
    }
    *out = bm;
    return TKV_OK;
}

TKV_EXPORT void tkv_bm_destroy(tkv_bm* bm) { delete bm; }

static bool seq_live(const tkv_bm* bm, int32_t s) { return s >= 0 && s < bm->max_seqs && bm->seqs[s].live; }

TKV_EXPORT int tkv_bm_extend(tkv_bm* bm, int32_t parent, const int32_t* tokens, int32_t n, int32_t seal,
                             int32_t* child_out, int32_t* blk_out, uint8_t* hit_out, int32_t cap,
                             int32_t* n_blk_out) {
    tkv::clear_error();
    if (!bm || !child_out || !n_blk_out || (n > 0 && !tokens))
        return set_error(TKV_EINVAL, "tkv_bm_extend: NULL argument");
    if (n < 0) return set_error(TKV_EINVAL, "tkv_bm_extend: n = %d < 0", n);
    if (seal != 0 && seal != 1) return set_error(TKV_EINVAL, "tkv_bm_extend: seal must be 0 or 1");
    const int32_t bs = bm->block_size;
    const int32_t n_chunks = (n + bs - 1) / bs;
    if (parent == -1) {
        if (n < 1) return set_error(TKV_EINVAL, "tkv_bm_extend: a root needs at least one token");
    } else {
        if (!seq_live(bm, parent)) return set_error(TKV_ENOSEQ, "tkv_bm_extend: parent %d is not live", parent);
        if (!bm->seqs[parent].sealed)
            return set_error(TKV_EINVAL, "tkv_bm_extend: parent %d is unsealed (in-progress step)", parent);
    }
    if (cap < n_chunks || (n_chunks > 0 && (!blk_out || !hit_out))) {
        *n_blk_out = n_chunks;
        return set_error(TKV_ECAP, "tkv_bm_extend: output capacity %d < %d blocks", cap, n_chunks);
    }
    if (bm->free_seqs.empty()) return set_error(TKV_ENOMEM, "tkv_bm_extend: no free sequence slot");

    // Resolve the hit prefix before changing anything: once a chunk misses, every later chunk of
    // this extension misses too (a fresh block is nobody's predecessor yet).
    std::vector<int32_t> hits;
    int32_t pred = parent == -1 ? -1
                                : (bm->seqs[parent].table.empty() ? -1 : bm->seqs[parent].table.back());
    ChunkKey probe;
    if (seal) {
        for (int32_t c = 0; c < n_chunks; ++c) {
            const int32_t a = c * bs, e = std::min(n, a + bs);
            probe.pred = pred;
            probe.toks.assign(tokens + a, tokens + e);
            auto it = bm->index.find(probe);
            if (it == bm->index.end()) break;
            hits.push_back(it->second);
            pred = it->second;
        }
    }
    const int32_t n_miss = n_chunks - static_cast<int32_t>(hits.size());
    if (static_cast<size_t>(n_miss) > bm->free_blocks.size())
        return set_error(TKV_ENOMEM, "tkv_bm_extend: pool exhausted (need %d blocks, %zu free)", n_miss,
                         bm->free_blocks.size());

    // Commit.
    const int32_t s = bm->free_seqs.top();
    bm->free_seqs.pop();
    Seq& sq = bm->seqs[s];
    sq.table.clear();
    if (parent != -1) sq.table = bm->seqs[parent].table;
    for (int32_t b : sq.table) bm->refcount[b] += 1;
    pred = sq.table.empty() ? -1 : sq.table.back();
    for (int32_t c = 0; c < n_chunks; ++c) {
        const int32_t a = c * bs, e = std::min(n, a + bs);
        int32_t b;
        uint8_t h;
        if (c < static_cast<int32_t>(hits.size())) {
            b = hits[c];
            h = 1;
        } else {
            b = bm->free_blocks.top();
            bm->free_blocks.pop();
            bm->block_len[b] = e - a;
            if (seal) {
                ChunkKey k{pred, std::vector<int32_t>(tokens + a, tokens + e)};
                bm->index.emplace(k, b);
                bm->key[b] = std::move(k);
                bm->indexed[b] = 1;
            }
            h = 0;
        }
        bm->refcount[b] += 1;
        sq.table.push_back(b);
        blk_out[c] = b;
        hit_out[c] = h;
        pred = b;
    }
    sq.live = true;
    sq.sealed = seal != 0;
    if (seal)
        sq.open.clear();
    else
        sq.open.assign(tokens, tokens + n);
    bm->n_live += 1;
    *child_out = s;
    *n_blk_out = n_chunks;
    return TKV_OK;
}

TKV_EXPORT int tkv_bm_append(tkv_bm* bm, int32_t seq, const int32_t* tokens, int32_t n, int32_t* dst_out,
                             int32_t cap) {
    tkv::clear_error();
    if (!bm || (n > 0 && (!tokens || !dst_out))) return set_error(TKV_EINVAL, "tkv_bm_append: NULL argument");
    if (n < 0) return set_error(TKV_EINVAL, "tkv_bm_append: n = %d < 0", n);
    if (!seq_live(bm, seq)) return set_error(TKV_ENOSEQ, "tkv_bm_append: sequence %d is not live", seq);
    if (cap < n) return set_error(TKV_ECAP, "tkv_bm_append: output capacity %d < %d tokens", cap, n);
    Seq& sq = bm->seqs[seq];
    const int32_t bs = bm->block_size;
    const int64_t open = sq.sealed ? 0 : static_cast<int64_t>(sq.open.size());
    const int64_t room = (bs - open % bs) % bs;  // free slots in the open step's last block
    const int64_t need = (std::max<int64_t>(0, n - room) + bs - 1) / bs;
    if (static_cast<size_t>(need) > bm->free_blocks.size())
        return set_error(TKV_ENOMEM, "tkv_bm_append: pool exhausted (need %lld blocks, %zu free)",
                         static_cast<long long>(need), bm->free_blocks.size());
    if (sq.sealed) {  // a new step, in a fresh block
        sq.sealed = false;
        sq.open.clear();
    }
    for (int32_t i = 0; i < n; ++i) {
        if (sq.open.size() % bs == 0) {
            const int32_t b = bm->free_blocks.top();
            bm->free_blocks.pop();
            bm->refcount[b] = 1;
            sq.table.push_back(b);
        }
        const int32_t b = sq.table.back();
        dst_out[i] = b * bs + bm->block_len[b];
        bm->block_len[b] += 1;
        sq.open.push_back(tokens[i]);
    }
    return TKV_OK;
}

TKV_EXPORT int tkv_bm_seal(tkv_bm* bm, int32_t seq, int32_t* replaced_out, int32_t cap, int32_t* n_replaced_out) {
    tkv::clear_error();
    if (!bm || !n_replaced_out) return set_error(TKV_EINVAL, "tkv_bm_seal: NULL argument");
    if (!seq_live(bm, seq)) return set_error(TKV_ENOSEQ, "tkv_bm_seal: sequence %d is not live", seq);
    Seq& sq = bm->seqs[seq];
    if (sq.sealed) return set_error(TKV_EINVAL, "tkv_bm_seal: sequence %d is already sealed", seq);
    const int32_t bs = bm->block_size;
    const int32_t n_open = static_cast<int32_t>((sq.open.size() + bs - 1) / bs);
    if (cap < n_open || (n_open > 0 && !replaced_out)) {
        *n_replaced_out = n_open;
        return set_error(TKV_ECAP, "tkv_bm_seal: capacity %d < %d open blocks", cap, n_open);
    }
    const int32_t first = static_cast<int32_t>(sq.table.size()) - n_open;
    int32_t nr = 0;
    for (int32_t j = 0; j < n_open; ++j) {
        const int32_t i = first + j;
        const size_t a = static_cast<size_t>(j) * bs, e = std::min(sq.open.size(), a + bs);
        ChunkKey k{i > 0 ? sq.table[i - 1] : -1, std::vector<int32_t>(sq.open.begin() + a, sq.open.begin() + e)};
        const int32_t own = sq.table[i];
        auto it = bm->index.find(k);
        if (it != bm->index.end()) {
            const int32_t hit = it->second;
            sq.table[i] = hit;
            bm->refcount[hit] += 1;
            bm->refcount[own] = 0;
            bm->block_len[own] = 0;
            bm->free_blocks.push(own);
            replaced_out[2 * nr] = own;
            replaced_out[2 * nr + 1] = hit;
            ++nr;
        } else {
            bm->index.emplace(k, own);
            bm->key[own] = std::move(k);
            bm->indexed[own] = 1;
        }
    }
    sq.sealed = true;
    sq.open.clear();
    *n_replaced_out = nr;
    return TKV_OK;
}

TKV_EXPORT int tkv_bm_fork(tkv_bm* bm, int32_t seq, const int32_t* tokens, int32_t n, int32_t* child_out,
                           int32_t cap) {
    tkv::clear_error();
    if (!bm || (n > 0 && (!tokens || !child_out))) return set_error(TKV_EINVAL, "tkv_bm_fork: NULL argument");
    if (n < 0) return set_error(TKV_EINVAL, "tkv_bm_fork: n = %d < 0", n);
    if (!seq_live(bm, seq)) return set_error(TKV_ENOSEQ, "tkv_bm_fork: sequence %d is not live", seq);
    if (cap < n) return set_error(TKV_ECAP, "tkv_bm_fork: output capacity %d < %d children", cap, n);
    if (static_cast<size_t>(n) > bm->free_blocks.size() || static_cast<size_t>(n) > bm->free_seqs.size())
        return set_error(TKV_ENOMEM, "tkv_bm_fork: %d children need as many blocks and sequence slots (%zu, %zu free)", n,
                         bm->free_blocks.size(), bm->free_seqs.size());
    // the point of divergence becomes a step boundary: seal the open step, then one open child per token
    if (!bm->seqs[seq].sealed) {
        const size_t n_open = (bm->seqs[seq].open.size() + bm->block_size - 1) / bm->block_size;
        std::vector<int32_t> replaced(2 * std::max<size_t>(1, n_open));
        int32_t nr = 0;
        const int rc = tkv_bm_seal(bm, seq, replaced.data(), static_cast<int32_t>(n_open), &nr);
        if (rc != TKV_OK) return rc;
    }
    for (int32_t i = 0; i < n; ++i) {
        int32_t blk = 0, nb = 0;
        uint8_t hit = 0;
        const int rc = tkv_bm_extend(bm, seq, tokens + i, 1, 0, child_out + i, &blk, &hit, 1, &nb);
        if (rc != TKV_OK) return rc;  // cannot happen: blocks and slots were checked above
    }
    return TKV_OK;
}

TKV_EXPORT int tkv_extend_slots(const int32_t* blk, const uint8_t* hit, int32_t n_blk, int32_t n_tok,
                                int32_t block_size, int32_t* dst_out) {
    tkv::clear_error();
    if (n_blk < 0 || n_tok < 0 || block_size < 1 || (n_blk > 0 && (!blk || !hit)) || (n_tok > 0 && !dst_out))
        return set_error(TKV_EINVAL, "tkv_extend_slots: bad argument");
    if (n_blk != (static_cast<int64_t>(n_tok) + block_size - 1) / block_size)
        return set_error(TKV_EINVAL, "tkv_extend_slots: %d tokens take %lld blocks of %d, not %d", n_tok,
                         static_cast<long long>((static_cast<int64_t>(n_tok) + block_size - 1) / block_size), block_size, n_blk);
    for (int32_t t = 0; t < n_tok; ++t) {
        const int32_t c = t / block_size;
        dst_out[t] = hit[c] ? -1 : blk[c] * block_size + (t - c * block_size);
    }
    return TKV_OK;
}

TKV_EXPORT int tkv_prune(tkv_bm* bm, int32_t seq, int32_t* freed_out, int32_t cap, int32_t* n_freed_out) {
    tkv::clear_error();
    if (!bm || !n_freed_out) return set_error(TKV_EINVAL, "tkv_prune: NULL argument");
    if (!seq_live(bm, seq)) return set_error(TKV_ENOSEQ, "tkv_prune: sequence %d is not live", seq);
    Seq& sq = bm->seqs[seq];
    const int32_t len = static_cast<int32_t>(sq.table.size());
    if (cap < len || (len > 0 && !freed_out)) {
        *n_freed_out = len;
        return set_error(TKV_ECAP, "tkv_prune: capacity %d < table length %d", cap, len);
    }
    int32_t nf = 0;
    for (int32_t b : sq.table) {
        if (--bm->refcount[b] == 0) {
            if (bm->indexed[b]) {
                bm->index.erase(bm->key[b]);
                bm->key[b] = ChunkKey{};
                bm->indexed[b] = 0;
            }
            bm->block_len[b] = 0;
            bm->free_blocks.push(b);
            freed_out[nf++] = b;
        }
    }
    sq.table.clear();
    sq.open.clear();
    sq.live = false;
    sq.sealed = false;
    bm->free_seqs.push(seq);
    bm->n_live -= 1;
    *n_freed_out = nf;
    return TKV_OK;
}

TKV_EXPORT int tkv_bm_table(const tkv_bm* bm, int32_t seq, int32_t* blk_out, int32_t cap, int32_t* n_out,
                            int32_t* kv_len_out) {
    tkv::clear_error();
    if (!bm || !n_out) return set_error(TKV_EINVAL, "tkv_bm_table: NULL argument");
    if (!seq_live(bm, seq)) return set_error(TKV_ENOSEQ, "tkv_bm_table: sequence %d is not live", seq);
    const auto& t = bm->seqs[seq].table;
    const int32_t len = static_cast<int32_t>(t.size());
    *n_out = len;
    if (cap < len || (len > 0 && !blk_out))
        return set_error(TKV_ECAP, "tkv_bm_table: capacity %d < table length %d", cap, len);
    int32_t kv = 0;
    for (int32_t i = 0; i < len; ++i) {
        blk_out[i] = t[i];
        kv += bm->block_len[t[i]];
    }
    if (kv_len_out) *kv_len_out = kv;
    return TKV_OK;
}

TKV_EXPORT int tkv_bm_refcount(const tkv_bm* bm, int32_t blk, int32_t* rc_out) {
    tkv::clear_error();
    if (!bm || !rc_out) return set_error(TKV_EINVAL, "tkv_bm_refcount: NULL argument");
    if (blk < 0 || blk >= bm->num_blocks) return set_error(TKV_EINVAL, "tkv_bm_refcount: block %d out of range", blk);
    *rc_out = bm->refcount[blk];
    return TKV_OK;
}

TKV_EXPORT int tkv_bm_block_len(const tkv_bm* bm, int32_t* len_out) {
    tkv::clear_error();
    if (!bm || !len_out) return set_error(TKV_EINVAL, "tkv_bm_block_len: NULL argument");
    std::memcpy(len_out, bm->block_len.data(), sizeof(int32_t) * bm->num_blocks);
    return TKV_OK;
}

TKV_EXPORT int tkv_bm_snapshot(const tkv_bm* bm, void* buf, size_t cap, size_t* used) {
    tkv::clear_error();
    if (!bm || !used) return set_error(TKV_EINVAL, "tkv_bm_snapshot: NULL argument");
    size_t words = 4 + 3 * static_cast<size_t>(bm->num_blocks);
    for (const Seq& s : bm->seqs)
        if (s.live) words += 4 + s.table.size();
    *used = words * sizeof(int32_t);
    if (!buf || cap < *used) return set_error(TKV_ECAP, "tkv_bm_snapshot: capacity %zu < %zu bytes", cap, *used);
    int32_t* w = static_cast<int32_t*>(buf);
    *w++ = bm->num_blocks;
    *w++ = bm->block_size;
    *w++ = bm->max_seqs;
    *w++ = bm->n_live;
    for (int32_t b = 0; b < bm->num_blocks; ++b) *w++ = bm->refcount[b];
    for (int32_t b = 0; b < bm->num_blocks; ++b) *w++ = bm->block_len[b];
    for (int32_t b = 0; b < bm->num_blocks; ++b) *w++ = bm->indexed[b];
    for (int32_t s = 0; s < bm->max_seqs; ++s) {
        const Seq& q = bm->seqs[s];
        if (!q.live) continue;
        *w++ = s;
        *w++ = q.sealed ? 1 : 0;
        *w++ = static_cast<int32_t>((q.open.size() + bm->block_size - 1) / bm->block_size);
        *w++ = static_cast<int32_t>(q.table.size());
        for (int32_t b : q.table) *w++ = b;
    }
    return TKV_OK;
}

namespace {
struct RowKeyHash {
    size_t operator()(const std::vector<int32_t>& v) const {
        uint64_t h = 1469598103934665603ull;
        for (int32_t x : v) {
            h ^= static_cast<uint32_t>(x);
            h *= 1099511628211ull;
        }
        return static_cast<size_t>(h);
    }
};
}  // namespace

TKV_EXPORT int tkv_bm_coalesce(const tkv_bm* bm, int32_t n_cand, const int32_t* seqs, const int32_t* q_len,
                               int32_t* row_of_cand_out, int32_t* first_cand_out, int32_t* mult_out,
                               int32_t* n_rows_out) {
    tkv::clear_error();
    if (!bm || !n_rows_out || n_cand < 0 ||
        (n_cand > 0 && (!seqs || !q_len || !row_of_cand_out || !first_cand_out || !mult_out)))
        return set_error(TKV_EINVAL, "tkv_bm_coalesce: bad argument");
    for (int32_t c = 0; c < n_cand; ++c) {
        if (!seq_live(bm, seqs[c])) return set_error(TKV_ENOSEQ, "tkv_bm_coalesce: sequence %d is not live", seqs[c]);
        if (q_len[c] < 1) return set_error(TKV_EINVAL, "tkv_bm_coalesce: q_len[%d] = %d < 1", c, q_len[c]);
    }
    std::unordered_map<std::vector<int32_t>, int32_t, RowKeyHash> first;
    int32_t n_rows = 0;
    std::vector<int32_t> key;
    for (int32_t c = 0; c < n_cand; ++c) {
        const auto& t = bm->seqs[seqs[c]].table;
        key.assign(1, q_len[c]);
        key.insert(key.end(), t.begin(), t.end());
        auto it = first.find(key);
        int32_t r;
        if (it == first.end()) {
            r = n_rows++;
            first.emplace(key, r);
            first_cand_out[r] = c;
            mult_out[r] = 0;
        } else {
            r = it->second;
        }
        mult_out[r] += 1;
        row_of_cand_out[c] = r;
    }
    *n_rows_out = n_rows;
    return TKV_OK;
}
