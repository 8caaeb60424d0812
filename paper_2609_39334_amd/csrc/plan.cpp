// Planner: per-row block tables -> shared segments -> device work lists.
//
// The paper's lever (computation deduplication, Sec. 4.2, over prefix-shared paged KV, Sec. 5.1)
// is that many candidates reference the same prompt and step blocks.  The planner finds those
// blocks with a trie over the rows' tables and emits two kinds of work items:
//
//  * shared items, for rows whose query tile is small (q_len * G < kTileRows: decode rows and
//    short verify rows).  A segment is a maximal run of trie nodes passed by the same set of rows;
//    each segment (split into chunks of <= kChunkBlocks blocks) becomes items whose tile holds the
//    query tokens of *every* row that references it, so each shared K/V block is read once per
//    tile and contracted against all of them.  Each (token, chunk) result is a partial (o, lse)
//    that a log-sum-exp merge combines -- unless the chunk is the token's only one, in which case
//    the item writes the final output.  With G <= 16 these items go to the wave kernel (tiles of
//    up to 32 rows, per-wave work lists built here); segments read by many rows (and G > 16)
//    go to the workgroup kernel's 128-row tiles.
//  * row items, for rows whose own query tokens fill a tile (verify rows with q_len * G >=
//    kTileRows).  A workgroup-kernel tile of one row's tokens (128 rows) walks the row's whole
//    path, truncated at the tile's largest causal limit, and writes the final output; the shared
//    context blocks are re-read from L2 by the tiles of the other rows, which the launch order
//    keeps on the same XCD.
//
// Positions: key j of a row is the j-th token along its path; token i of a row with q_len L and
// kv_len N sees positions <= N - L + i (bottom-right causal, the single-pass verification of
// Sec. 3.2; decode is L = 1).  A shared segment sits at the same positions in every row through
// it, so one per-token limit suffices.
#include <algorithm>
#include <cstring>
#include <map>
#include <mutex>
#include <numeric>
#include <queue>
#include <unordered_map>
#include <vector>

#include "internal.h"

using tkv::BlkDesc;
using tkv::ItemDesc;
using tkv::MergeDesc;
using tkv::set_error;
using tkv::TokDesc;

namespace {

constexpr int kChunkBlocks = 16;      // longest key run of a narrow shared item (256 tokens)
constexpr int kChunkBlocksWide = 64;  // longest key run of a wide (128-row tile) shared item
constexpr int kFoldBlocks = 16;       // longest shared segment folded into its children's key runs
static_assert(kChunkBlocks <= tkv::kWaveBlocks, "a wave item holds its key blocks in one record");

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// The block slots of a wave item's record (see tkv::WaveDesc): {id, length, path position} of each
// key block, {block 0's id, 0, 0} past the item's blocks (a length-0 block hides all its keys,
// wherever it sits); the fourth words of slots 0-2 carry the KV head, the token count and the
// walked block count.
void write_record_blocks(const tkv_plan* p, const ItemDesc& it, int32_t* e) {
    // widths 1 and 2 walk blocks in pairs: an odd key list gets an empty block
    const int32_t nb_run = it.pad <= 2 ? (it.n_blk + 1) & ~1 : it.n_blk;
    int32_t pos = it.pos0;
    for (int32_t j = 0; j < tkv::kWaveBlocks; ++j) {
        const bool in = j < it.n_blk;
        const BlkDesc& bd = p->wblks[it.blk_off + (in ? j : 0)];
        e[4 * j] = bd.blk;
        e[4 * j + 1] = in ? bd.len : 0;
        e[4 * j + 2] = in ? pos : 0;
        e[4 * j + 3] = 0;
        if (in) pos += bd.len;
    }
    e[3] = it.kvh;
    e[7] = it.n_tok;
    e[11] = nb_run;
}

// A wave item's whole record, written in place (zero for item < 0): its block slots, then
// kWaveToks token slots {query token, causal limit, partial slot, 0}, token 0's past the tile.
void write_record(const tkv_plan* p, int32_t item, uint8_t* dst) {
    if (item < 0) {
        std::memset(dst, 0, sizeof(tkv::WaveDesc));
        return;
    }
    static_assert(sizeof(TokDesc) == 16, "a token slot holds one TokDesc (its fourth word is 0)");
    const ItemDesc& it = p->wave_items[item];
    int32_t* e = reinterpret_cast<int32_t*>(dst);
    write_record_blocks(p, it, e);
    TokDesc* slots = reinterpret_cast<TokDesc*>(e + 4 * tkv::kWaveBlocks);
    const TokDesc* src = p->wtoks.data() + it.tok_off;
    std::memcpy(slots, src, static_cast<size_t>(it.n_tok) * sizeof(TokDesc));
    for (int32_t t = it.n_tok; t < tkv::kWaveToks; ++t) slots[t] = src[0];
}

struct Node {
    int32_t parent, blk, len, pos0, count, seg;
};

struct Segment {
    std::vector<int32_t> nodes;
    std::vector<int32_t> rows;
};

struct Chunk {
    int32_t blk_off, n_blk, pos0;  // blk_off: into the segments' block runs
    bool wave;                     // run by the wave kernel
    std::vector<TokDesc> toks;     // slot filled in later
};

// Idle waves a plan keeps for the chunks its decode tails open later (tkv_plan_update): one per
// eight (row, KV head) tails, a multiple of kWaveWG, at most kMaxSpareWaves.
constexpr int32_t kMaxSpareWaves = 512;

// Room a stored row table gets for more blocks when an update moves it (tkv::PlanInputs).
constexpr int32_t kRowSlack = 16;

// Key blocks per wave below which a wave grid beside a chip-filling set of tile items is made smaller.
constexpr int64_t kWaveBlocksPerWave = 8;

// Dense ids for 64-bit keys in first-insertion order (open addressing, linear probing, grown at half
// load).  Keys never equal ~0.
class IdMap {
  public:
    explicit IdMap(size_t expected = 0) { reset(expected); }
    // Empty, sized for `expected` keys (the storage is kept).
    void reset(size_t expected) {
        const size_t want = std::max<size_t>(16, expected * 2);
        size_t cap = 16;
        while (cap < want) cap <<= 1;
        keys_.assign(cap, kEmpty);
        vals_.resize(cap);
        mask_ = cap - 1;
        n_ = 0;
    }
    // The key's id; a new key takes `next_id` (and *fresh is set).
    int32_t get(uint64_t key, int32_t next_id, bool* fresh) {
        if (2 * (n_ + 1) > keys_.size()) rehash(keys_.size() * 2);
        size_t h = mix(key) & mask_;
        while (keys_[h] != kEmpty) {
            if (keys_[h] == key) {
                *fresh = false;
                return vals_[h];
            }
            h = (h + 1) & mask_;
        }
        keys_[h] = key;
        vals_[h] = next_id;
        ++n_;
        *fresh = true;
        return next_id;
    }

  private:
    static constexpr uint64_t kEmpty = ~uint64_t{0};
    static uint64_t mix(uint64_t k) {
        k ^= k >> 33;
        k *= 0xff51afd7ed558ccdull;
        k ^= k >> 33;
        return k;
    }
    void rehash(size_t want) {
        size_t cap = 16;
        while (cap < want) cap <<= 1;
        std::vector<uint64_t> ok;
        std::vector<int32_t> ov;
        ok.swap(keys_);
        ov.swap(vals_);
        keys_.assign(cap, kEmpty);
        vals_.resize(cap);
        mask_ = cap - 1;
        for (size_t i = 0; i < ok.size(); ++i) {
            if (ok[i] == kEmpty) continue;
            size_t h = mix(ok[i]) & mask_;
            while (keys_[h] != kEmpty) h = (h + 1) & mask_;
            keys_[h] = ok[i];
            vals_[h] = ov[i];
        }
    }
    std::vector<uint64_t> keys_;
    std::vector<int32_t> vals_;
    size_t mask_ = 0, n_ = 0;
};

// Stable sort of v by key(x) in [0, kmax], largest first (a counting sort).
template <class T, class K>
void sort_by_small_key_desc(std::vector<T>& v, int32_t kmax, K key) {
    std::vector<size_t> start(kmax + 2, 0);
    for (const T& x : v) ++start[kmax - key(x) + 1];
    for (int32_t k = 1; k <= kmax + 1; ++k) start[k] += start[k - 1];
    std::vector<T> out(v.size());
    for (const T& x : v) out[start[kmax - key(x)]++] = x;
    v.swap(out);
}

// Split n things into near-equal tiles of at most `cap`.
template <class F>
void tile_evenly(int32_t n, int32_t cap, F f) {
    if (n <= 0) return;
    const int32_t tiles = (n + cap - 1) / cap;
    const int32_t per = (n + tiles - 1) / tiles;
    for (int32_t a = 0; a < n; a += per) f(a, std::min(n, a + per));
}

// Split n query tokens into full tiles of `cap` and one last partial tile.  A workgroup-kernel
// tile costs MFMA time per active wave of 32 rows whatever the wave's fill, so full tiles leave
// at most one partly filled wave per row (near-equal tiles leave one per tile).
template <class F>
void tile_full(int32_t n, int32_t cap, F f) {
    for (int32_t a = 0; a < n; a += cap) f(a, std::min(n, a + cap));
}

// The planner's working arrays, kept per thread from one plan to the next (a loop that plans every
// step then fills memory it already holds).
struct Scratch {
    std::vector<int32_t> L, N, path, cover, tail_chunk, slot_next, chunk_run, end_pos, root_last, grp;
    std::vector<uint8_t> seen, folded, absorbed;
    std::vector<int32_t> kid_off, kids, kid_fill;
    std::vector<Node> nodes;
    std::vector<BlkDesc> seg_blks;
    std::vector<ItemDesc> ordered;
    IdMap child, root_id, gid;
};

// Plans destroyed without instrumentation are kept, emptied but with their arrays' capacity, for
// the next tkv_plan_create (at most kPooledPlans; never destroyed: plans may be freed at exit).
struct PlanPool {
    std::mutex m;
    std::vector<tkv_plan*> free;
};
PlanPool& plan_pool() {
    static PlanPool* pool = new PlanPool();
    return *pool;
}
constexpr size_t kPooledPlans = 2;

// Every field back to a new plan's value; vectors keep their storage.  (The field list is
// tkv_plan's; swap_contents below names the same fields.)
void clear_plan(tkv_plan* p) {
    tkv::wait_copies(p);  // its image and pair staging go back for reuse
    p->shape = tkv_shape{};
    p->group = 1;
    p->all_decode = true;
    p->items.clear();
    p->wave_items.clear();
    p->view_items.clear();
    p->view_toks.clear();
    p->view_blks.clear();
    p->toks.clear();
    p->blks.clear();
    p->wtoks.clear();
    p->wblks.clear();
    p->merges.clear();
    p->merge_slots.clear();
    p->wave_rec.clear();
    p->wave_off.clear();
    p->wave_tiles.clear();
    p->n_slots = 0;
    p->tile8 = false;
    p->off_items = p->off_toks = p->off_blks = p->off_merges = p->off_mslots = p->off_wdesc = p->off_woff = p->off_wtiles = 0;
    p->off_po = p->off_plse = p->desc_bytes = p->total_bytes = 0;
    tkv::give_image(std::move(p->image), p->image_cap);
    p->image.reset();
    p->image_cap = 0;
    p->d_ws = nullptr;
    p->ws_image = nullptr;
    p->dirty.clear();
    p->dirty_over = false;
    p->patch_pairs.clear();
    p->off_patch = 0;
    p->patch_cap = 0;
    p->stats = tkv_plan_stats{};
    if (p->in) {
        tkv::PlanInputs& in = *p->in;
        for (auto* v : {&in.q_indptr, &in.kv_blocks, &in.row_len, &in.row_cap, &in.block_len, &in.mult, &in.kv_len,
                        &in.tail_run, &in.spare, &in.merge_of, &in.owner, &in.run_items, &in.rec_of, &in.free_waves})
            v->clear();
        in.row_start.clear();
        in.opts = tkv_plan_options{};
        in.has_opts = false;
        in.indexed = false;
    }
}

tkv_plan* take_plan() {
    PlanPool& pool = plan_pool();
    {
        std::lock_guard<std::mutex> lock(pool.m);
        if (!pool.free.empty()) {
            tkv_plan* p = pool.free.back();
            pool.free.pop_back();
            return p;
        }
    }
    return new (std::nothrow) tkv_plan();
}

void give_plan(tkv_plan* p) {
    if (!p) return;
    if (!p->prof_events.empty() || p->prof_max != 0) {  // instrumented: its events go with it
        delete p;
        return;
    }
    clear_plan(p);
    PlanPool& pool = plan_pool();
    {
        std::lock_guard<std::mutex> lock(pool.m);
        if (pool.free.size() < kPooledPlans) {
            pool.free.push_back(p);
            return;
        }
    }
    delete p;
}

}  // namespace

TKV_EXPORT int tkv_plan_create(const tkv_shape* shape, int32_t n_rows, const int32_t* q_indptr,
                               const int32_t* kv_indptr, const int32_t* kv_blocks, const int32_t* block_len,
                               const int32_t* multiplicity, tkv_plan** out) {
    return tkv_plan_create_ex(shape, n_rows, q_indptr, kv_indptr, kv_blocks, block_len, multiplicity, nullptr, out);
}

TKV_EXPORT int tkv_plan_create_ex(const tkv_shape* shape, int32_t n_rows, const int32_t* q_indptr,
                                  const int32_t* kv_indptr, const int32_t* kv_blocks, const int32_t* block_len,
                                  const int32_t* multiplicity, const tkv_plan_options* opts, tkv_plan** out) {
    tkv::clear_error();
    if (!out) return set_error(TKV_EINVAL, "tkv_plan_create: out is NULL");
    // placement options: a negative field (or no options) keeps the default
    auto opt = [&](int32_t tkv_plan_options::*f, int64_t dflt) -> int64_t {
        return opts && opts->*f >= 0 ? static_cast<int64_t>(opts->*f) : dflt;
    };
    *out = nullptr;
    if (!shape) return set_error(TKV_EINVAL, "tkv_plan_create: shape is NULL");
    const tkv_shape s = *shape;
    if (s.block_size != tkv::kBlock) return set_error(TKV_EINVAL, "tkv_plan_create: block_size must be 16 (got %d)", s.block_size);
    if (s.d != 64 && s.d != 128) return set_error(TKV_EINVAL, "tkv_plan_create: head_dim must be 64 or 128 (got %d)", s.d);
    if (s.hq < 1 || s.hkv < 1 || s.hq % s.hkv)
        return set_error(TKV_EINVAL, "tkv_plan_create: hq (%d) must be a positive multiple of hkv (%d)", s.hq, s.hkv);
    const int32_t G = s.hq / s.hkv;
    if (G > tkv::kTileRows) return set_error(TKV_EINVAL, "tkv_plan_create: hq/hkv = %d exceeds %d", G, tkv::kTileRows);
    if (s.hq > 256) return set_error(TKV_EINVAL, "tkv_plan_create: hq = %d exceeds 256", s.hq);
    if (s.num_blocks < 1) return set_error(TKV_EINVAL, "tkv_plan_create: num_blocks must be >= 1");
    if (n_rows < 0) return set_error(TKV_EINVAL, "tkv_plan_create: n_rows < 0");
    if (n_rows > 0 && (!q_indptr || !kv_indptr || !block_len))
        return set_error(TKV_EINVAL, "tkv_plan_create: NULL array");
    if (n_rows > 0 && (q_indptr[0] != 0 || kv_indptr[0] != 0))
        return set_error(TKV_EINVAL, "tkv_plan_create: q_indptr[0] and kv_indptr[0] must be 0");
    if (n_rows > 0 && kv_indptr[n_rows] > 0 && !kv_blocks) return set_error(TKV_EINVAL, "tkv_plan_create: kv_blocks is NULL");

    // ---------------------------------------------------------------- validate rows
    thread_local Scratch sc;
    std::vector<int32_t>& L = sc.L;
    std::vector<int32_t>& N = sc.N;
    L.assign(n_rows, 0);
    N.assign(n_rows, 0);
    for (int32_t r = 0; r < n_rows; ++r) {
        L[r] = q_indptr[r + 1] - q_indptr[r];
        const int32_t nb = kv_indptr[r + 1] - kv_indptr[r];
        if (L[r] < 1) return set_error(TKV_EINVAL, "tkv_plan_create: row %d has q_len %d < 1", r, L[r]);
        if (nb < 0) return set_error(TKV_EINVAL, "tkv_plan_create: kv_indptr decreases at row %d", r);
        int64_t n = 0;
        for (int32_t j = kv_indptr[r]; j < kv_indptr[r + 1]; ++j) {
            const int32_t b = kv_blocks[j];
            if (b < 0 || b >= s.num_blocks) return set_error(TKV_EINVAL, "tkv_plan_create: row %d block id %d out of range", r, b);
            if (block_len[b] < 1 || block_len[b] > s.block_size)
                return set_error(TKV_EINVAL, "tkv_plan_create: block %d has length %d (free or invalid)", b, block_len[b]);
            n += block_len[b];
        }
        if (n > (1 << 30)) return set_error(TKV_EINVAL, "tkv_plan_create: row %d kv_len too large", r);
        N[r] = static_cast<int32_t>(n);
        if (L[r] > N[r]) return set_error(TKV_EINVAL, "tkv_plan_create: row %d q_len %d > kv_len %d", r, L[r], N[r]);
        if (multiplicity && multiplicity[r] < 1) return set_error(TKV_EINVAL, "tkv_plan_create: multiplicity[%d] < 1", r);
    }

    tkv_plan* p = take_plan();
    if (!p) return set_error(TKV_ENOMEM, "tkv_plan_create: host allocation failed");
    try {
        p->shape = s;
        p->group = G;
        if (!p->in) p->in.reset(new tkv::PlanInputs());
        tkv::PlanInputs& in = *p->in;
        if (n_rows > 0) {
            in.q_indptr.assign(q_indptr, q_indptr + n_rows + 1);
            in.kv_blocks.assign(kv_blocks, kv_blocks + kv_indptr[n_rows]);
            in.row_start.resize(n_rows);
            in.row_len.resize(n_rows);
            for (int32_t r = 0; r < n_rows; ++r) {
                in.row_start[r] = kv_indptr[r];
                in.row_len[r] = kv_indptr[r + 1] - kv_indptr[r];
            }
            in.row_cap = in.row_len;
            in.block_len.assign(block_len, block_len + s.num_blocks);
            if (multiplicity) in.mult.assign(multiplicity, multiplicity + n_rows);
        } else {
            in.q_indptr.assign(1, 0);
            in.block_len.assign(s.num_blocks, 0);
            if (block_len) in.block_len.assign(block_len, block_len + s.num_blocks);
        }
        if (opts) {
            in.opts = *opts;
            in.has_opts = true;
        }
        in.kv_len = N;
        in.tail_run.assign(n_rows, -1);
        in.spare.assign(n_rows, 0);
        in.merge_of.assign(n_rows, -1);
        tkv_plan_stats& st = p->stats;
        st.n_rows = n_rows;
        st.n_qtok = n_rows ? q_indptr[n_rows] : 0;
        const int32_t tpt = tkv::kTileRowsWG / G;  // query tokens per workgroup-kernel tile

        // ------------------------------------------------------------ accounting
        {
            std::vector<uint8_t>& seen = sc.seen;
            seen.assign(s.num_blocks, 0);
            for (int32_t r = 0; r < n_rows; ++r) {
                p->all_decode = p->all_decode && L[r] == 1;
                st.logical_qtok += static_cast<int64_t>(multiplicity ? multiplicity[r] : 1) * L[r];
                st.path_kv_tokens += N[r];
                for (int32_t i = 0; i < L[r]; ++i) st.flops += 4ll * s.d * s.hq * (N[r] - L[r] + i + 1);
                for (int32_t j = kv_indptr[r]; j < kv_indptr[r + 1]; ++j) {
                    const int32_t b = kv_blocks[j];
                    if (!seen[b]) {
                        seen[b] = 1;
                        st.uniq_kv_tokens += block_len[b];
                    }
                }
            }
        }

        // ------------------------------------------------------------ shared items (small rows)
        std::vector<Node>& nodes = sc.nodes;
        nodes.clear();
        IdMap& child = sc.child;  // (parent node + 1, block) -> node
        child.reset(static_cast<size_t>(s.num_blocks));
        std::vector<int32_t>& path = sc.path;  // trie node of each table entry
        path.assign(n_rows ? kv_indptr[n_rows] : 0, -1);
        // the last row walked from each root block: the blocks a row shares with it lead to the
        // same nodes, found without lookups
        IdMap& root_id = sc.root_id;
        root_id.reset(64);
        std::vector<int32_t>& root_last = sc.root_last;
        root_last.clear();
        for (int32_t r = 0; r < n_rows; ++r) {
            if (static_cast<int64_t>(L[r]) * G >= tkv::kTileRows) continue;
            int32_t cur = -1;
            int32_t j = kv_indptr[r];
            bool fresh_root = false;
            const int32_t rid = root_id.get(static_cast<uint32_t>(kv_blocks[j]), static_cast<int32_t>(root_last.size()), &fresh_root);
            if (fresh_root) root_last.push_back(-1);
            const int32_t prev = root_last[rid];
            root_last[rid] = r;
            if (prev >= 0) {
                const int32_t len = std::min(kv_indptr[r + 1] - kv_indptr[r], kv_indptr[prev + 1] - kv_indptr[prev]);
                for (int32_t k = 0; k < len && kv_blocks[j] == kv_blocks[kv_indptr[prev] + k]; ++k, ++j) {
                    cur = path[kv_indptr[prev] + k];
                    nodes[cur].count += 1;
                    path[j] = cur;
                }
            }
            for (; j < kv_indptr[r + 1]; ++j) {
                const int32_t b = kv_blocks[j];
                const uint64_t key = (static_cast<uint64_t>(static_cast<uint32_t>(cur + 1)) << 32) | static_cast<uint32_t>(b);
                bool fresh = false;
                const int32_t nd = child.get(key, static_cast<int32_t>(nodes.size()), &fresh);
                if (fresh) {
                    const int32_t pos0 = cur < 0 ? 0 : nodes[cur].pos0 + nodes[cur].len;
                    nodes.push_back(Node{cur, b, block_len[b], pos0, 0, -1});
                }
                nodes[nd].count += 1;
                path[j] = nd;
                cur = nd;
            }
        }
        std::vector<Segment> segs;
        for (int32_t nd = 0; nd < static_cast<int32_t>(nodes.size()); ++nd) {
            Node& n = nodes[nd];
            if (n.parent >= 0 && nodes[n.parent].count == n.count) {
                n.seg = nodes[n.parent].seg;
            } else {
                n.seg = static_cast<int32_t>(segs.size());
                segs.emplace_back();
            }
            segs[n.seg].nodes.push_back(nd);
        }
        for (int32_t r = 0; r < n_rows; ++r) {
            int32_t last = -1;
            for (int32_t j = kv_indptr[r]; j < kv_indptr[r + 1] && path[j] >= 0; ++j) {
                const int32_t nd = path[j];
                if (nodes[nd].seg != last) {
                    last = nodes[nd].seg;
                    segs[last].rows.push_back(r);
                }
            }
        }
        st.n_segments = static_cast<int32_t>(segs.size());

        // Segments read by more than kWaveMaxRows query rows go to 128-row tile items, which read
        // each K/V block once for all of those rows -- if they make at least kTileMinItems items
        // (none by default: tile items and the wave grid share one launch, and the wave grid
        // gives up the workgroup slots the tile items take); otherwise everything with G <= 16
        // stays on the wave grid.
        int64_t wave_max_rows = opt(&tkv_plan_options::wave_max_rows, tkv::kWaveMaxRows);
        const int32_t chunk_wide = static_cast<int32_t>(std::max<int64_t>(1, opt(&tkv_plan_options::wide_chunk_blocks, kChunkBlocksWide)));
        if (G <= tkv::kWaveRows) {
            int64_t wide_items = 0;
            for (const Segment& sg : segs) {
                int64_t seg_tok = 0;
                for (int32_t r : sg.rows) seg_tok += L[r];
                if (seg_tok * G <= wave_max_rows) continue;
                const int64_t nb = static_cast<int64_t>(sg.nodes.size());
                wide_items += (nb + chunk_wide - 1) / chunk_wide * ((seg_tok + tpt - 1) / tpt) * s.hkv;
            }
            const int64_t min_items = opt(&tkv_plan_options::tile_min_items, tkv::kTileMinItems);
            if (wide_items < min_items) wave_max_rows = int64_t{1} << 40;
        }
        // A short shared segment on the 128-row tiles whose children all go there too, and which
        // holds no row beyond theirs, is read by each child as the head of the child's own key run:
        // its blocks cost one more tile item's worth of reads per child, but its own tile items (short,
        // so mostly start-up) and every token's partial from it go away.  One level only: a segment
        // that takes its parent's blocks is not folded into its own children.
        const int64_t fold_blocks = opt(&tkv_plan_options::fold_blocks, kFoldBlocks);
        std::vector<uint8_t>& folded = sc.folded;
        folded.assign(segs.size(), 0);
        if (fold_blocks > 0 && G <= tkv::kWaveRows && !segs.empty()) {
            auto rows_of = [&](const Segment& sg) {
                int64_t n = 0;
                for (int32_t r : sg.rows) n += static_cast<int64_t>(L[r]) * G;
                return n;
            };
            // children of each segment (segments are numbered parents first)
            std::vector<int32_t>& kid_off = sc.kid_off;
            std::vector<int32_t>& kids = sc.kids;
            kid_off.assign(segs.size() + 1, 0);
            for (const Segment& sg : segs) {
                const int32_t par = nodes[sg.nodes[0]].parent;
                if (par >= 0) kid_off[nodes[par].seg + 1] += 1;
            }
            for (size_t i = 0; i < segs.size(); ++i) kid_off[i + 1] += kid_off[i];
            kids.assign(kid_off[segs.size()], 0);
            std::vector<int32_t>& fill = sc.kid_fill;
            fill.assign(kid_off.begin(), kid_off.end() - 1);
            for (int32_t c = 0; c < static_cast<int32_t>(segs.size()); ++c) {
                const int32_t par = nodes[segs[c].nodes[0]].parent;
                if (par >= 0) kids[fill[nodes[par].seg]++] = c;
            }
            std::vector<uint8_t>& absorbed = sc.absorbed;
            absorbed.assign(segs.size(), 0);
            for (int32_t p = 0; p < static_cast<int32_t>(segs.size()); ++p) {
                Segment& sp = segs[p];
                if (absorbed[p] || sp.rows.size() < 2 || static_cast<int64_t>(sp.nodes.size()) > fold_blocks ||
                    kid_off[p] == kid_off[p + 1] || rows_of(sp) <= wave_max_rows)
                    continue;
                size_t kid_rows = 0;
                bool wide_kids = true;
                for (int32_t k = kid_off[p]; k < kid_off[p + 1]; ++k) {
                    kid_rows += segs[kids[k]].rows.size();
                    wide_kids = wide_kids && rows_of(segs[kids[k]]) > wave_max_rows;
                }
                if (!wide_kids || kid_rows != sp.rows.size()) continue;
                for (int32_t k = kid_off[p]; k < kid_off[p + 1]; ++k) {
                    std::vector<int32_t>& cn = segs[kids[k]].nodes;
                    cn.insert(cn.begin(), sp.nodes.begin(), sp.nodes.end());
                    absorbed[kids[k]] = 1;
                }
                folded[p] = 1;
            }
        }
        std::vector<Chunk> chunks;
        std::vector<BlkDesc>& seg_blks = sc.seg_blks;  // each segment's key blocks, in path order
        seg_blks.clear();
        std::vector<int32_t>& cover = sc.cover;
        cover.assign(st.n_qtok, 0);
        std::vector<int32_t>& tail_chunk = sc.tail_chunk;  // a decode row's tail chunk (see tkv::PlanInputs)
        tail_chunk.assign(n_rows, -1);
        for (size_t si = 0; si < segs.size(); ++si) {
            const Segment& sg = segs[si];
            if (folded[si]) continue;
            if (sg.rows.size() > 1) st.n_shared_segments += 1;
            const int32_t nb = static_cast<int32_t>(sg.nodes.size());
            const int32_t seg_blk_off = static_cast<int32_t>(seg_blks.size());
            for (int32_t nd : sg.nodes) seg_blks.push_back(BlkDesc{nodes[nd].blk, nodes[nd].len});
            // segments read by many query rows go to the 128-row tile kernel in long chunks; the
            // rest to the wave kernel in chunks that fit its records
            int64_t seg_rows = 0;
            for (int32_t r : sg.rows) seg_rows += static_cast<int64_t>(L[r]) * G;
            const bool wide = G > tkv::kWaveRows || seg_rows > wave_max_rows;
            auto cut = [&](int32_t a, int32_t e) {
                Chunk c;
                c.blk_off = seg_blk_off + a;
                c.n_blk = e - a;
                c.pos0 = nodes[sg.nodes[a]].pos0;
                for (int32_t r : sg.rows) {
                    for (int32_t i = 0; i < L[r]; ++i) {
                        const int32_t lim = N[r] - L[r] + i;
                        if (lim < c.pos0) continue;  // the whole chunk is in this token's future
                        c.toks.push_back(TokDesc{q_indptr[r] + i, L[r] == 1 ? tkv::kNoLimit : lim, -1, 0});
                        cover[q_indptr[r] + i] += 1;
                    }
                }
                if (c.toks.empty()) return;
                // Chunks of groups with G <= 16 and at most kWaveMaxRows query rows go to the wave
                // kernel: a wave contracts each K/V block against T column tiles of 16 rows (T = 1, 2
                // as the chunk's rows need).  Wider chunks (and groups with G > 16) use the workgroup
                // kernel's 128-row tiles, which stage each K/V block once for 128 rows.
                const int64_t rows = static_cast<int64_t>(c.toks.size()) * G;
                c.wave = G <= tkv::kWaveRows && rows <= wave_max_rows && c.n_blk <= kChunkBlocks;
                if (sg.rows.size() == 1 && L[sg.rows[0]] == 1 && e == nb && c.wave)
                    tail_chunk[sg.rows[0]] = static_cast<int32_t>(chunks.size());
                chunks.push_back(std::move(c));
            };
            // A segment of one row is cut at fixed multiples of the chunk length from its start: as
            // a decode row's path grows, its last chunk takes the new blocks or a new chunk follows
            // it, and the chunks before stay as they are.  Shared segments are cut evenly.
            if (sg.rows.size() == 1)
                tile_full(nb, wide ? chunk_wide : kChunkBlocks, cut);
            else
                tile_evenly(nb, wide ? chunk_wide : kChunkBlocks, cut);
        }
        // partial slots for tokens covered by more than one chunk: each token's slots are
        // contiguous (in chunk order), so the merge reads a token's partials as one range.  A
        // decode token with a tail chunk has one slot more, unused, for the chunk that its tail
        // opens next (tkv_plan_update).
        std::vector<int32_t>& slot_next = sc.slot_next;
        slot_next.assign(st.n_qtok, -1);
        for (int32_t r = 0; r < n_rows; ++r)
            if (tail_chunk[r] >= 0 && cover[q_indptr[r]] >= 2) in.spare[r] = 1;
        for (int32_t r = 0, q = 0; q < st.n_qtok; ++q) {
            while (q_indptr[r + 1] <= q) ++r;
            if (cover[q] < 2) continue;
            if (L[r] == 1) in.merge_of[r] = static_cast<int32_t>(p->merges.size());
            p->merges.push_back(MergeDesc{q, p->n_slots, cover[q], 0});
            slot_next[q] = p->n_slots;
            p->n_slots += cover[q] + (L[r] == 1 ? in.spare[r] : 0);
        }
        for (Chunk& c : chunks)
            for (TokDesc& t : c.toks)
                if (cover[t.qtok] > 1) t.slot = slot_next[t.qtok]++;
        p->merge_slots.resize(p->n_slots);
        std::iota(p->merge_slots.begin(), p->merge_slots.end(), 0);
        // Items.  A wave chunk's blocks take a run of kWaveBlocks slots in wblks (room for a tail
        // to grow into); its items' tokens go to wtoks.  Both stay on the host: the wave records
        // carry them.  Tile items' blocks and tokens go to blks and toks, which the device reads.
        std::vector<int32_t>& chunk_run = sc.chunk_run;
        chunk_run.assign(chunks.size(), -1);
        for (size_t ci = 0; ci < chunks.size(); ++ci) {
            const Chunk& c = chunks[ci];
            const int64_t rows = static_cast<int64_t>(c.toks.size()) * G;
            const bool wave = c.wave;
            // a wave tile holds 16 T / G tokens, at most the record's kWaveToks
            const int32_t T = static_cast<int32_t>(std::min<int64_t>(
                {tkv::kWaveMaxTiles, (rows + 15) / 16, static_cast<int64_t>(tkv::kWaveToks) * G / tkv::kWaveRows}));
            const int32_t per_tile = wave ? tkv::kWaveRows * T / G : tpt;
            std::vector<BlkDesc>& bv = wave ? p->wblks : p->blks;
            std::vector<TokDesc>& tv = wave ? p->wtoks : p->toks;
            const int32_t blk_off = static_cast<int32_t>(bv.size());
            bv.insert(bv.end(), seg_blks.begin() + c.blk_off, seg_blks.begin() + c.blk_off + c.n_blk);
            if (wave) {
                bv.resize(blk_off + tkv::kWaveBlocks, BlkDesc{0, 0});
                chunk_run[ci] = blk_off / tkv::kWaveBlocks;
            }
            auto emit = [&](int32_t a, int32_t e) {
                const int32_t tok_off = static_cast<int32_t>(tv.size());
                tv.insert(tv.end(), c.toks.begin() + a, c.toks.begin() + e);
                for (int32_t h = 0; h < s.hkv; ++h) {
                    const ItemDesc d{h, tok_off, e - a, blk_off, c.n_blk, c.pos0,
                                     wave ? tkv::kItemWave : tkv::kItemShared, wave ? T : 0};
                    (wave ? p->wave_items : p->items).push_back(d);
                }
            };
            // wave tiles balance the per-wave lists; 128-row tiles are filled (their cost is per wave)
            if (wave)
                tile_evenly(static_cast<int32_t>(c.toks.size()), per_tile, emit);
            else
                tile_full(static_cast<int32_t>(c.toks.size()), per_tile, emit);
        }
        st.n_items_shared = static_cast<int32_t>(p->items.size() + p->wave_items.size());
        int32_t n_tails = 0;
        for (int32_t r = 0; r < n_rows; ++r)
            if (tail_chunk[r] >= 0) {
                in.tail_run[r] = chunk_run[tail_chunk[r]];
                ++n_tails;
            }

        // ------------------------------------------------------------ row items (large rows)
        {
            size_t n_blk = 0, n_tok = 0, n_it = 0;
            for (int32_t r = 0; r < n_rows; ++r) {
                if (static_cast<int64_t>(L[r]) * G < tkv::kTileRows) continue;
                n_blk += kv_indptr[r + 1] - kv_indptr[r];
                n_tok += L[r];
                n_it += static_cast<size_t>((L[r] + tpt - 1) / tpt) * s.hkv;
            }
            p->blks.reserve(p->blks.size() + n_blk);
            p->toks.reserve(p->toks.size() + n_tok);
            p->items.reserve(p->items.size() + n_it);
        }
        std::vector<int32_t>& end_pos = sc.end_pos;  // end position of each block along a row's path
        for (int32_t r = 0; r < n_rows; ++r) {
            if (static_cast<int64_t>(L[r]) * G < tkv::kTileRows) continue;
            const int32_t row_blk_off = static_cast<int32_t>(p->blks.size());
            end_pos.clear();
            int32_t pos = 0;
            for (int32_t j = kv_indptr[r]; j < kv_indptr[r + 1]; ++j) {
                p->blks.push_back(BlkDesc{kv_blocks[j], block_len[kv_blocks[j]]});
                pos += block_len[kv_blocks[j]];
                end_pos.push_back(pos);
            }
            tile_full(L[r], tpt, [&](int32_t a, int32_t e) {
                const int32_t max_lim = N[r] - L[r] + e - 1;
                // blocks whose first position is <= max_lim
                const int32_t nb = static_cast<int32_t>(std::upper_bound(end_pos.begin(), end_pos.end(), max_lim) - end_pos.begin()) + 1;
                const int32_t nbk = std::min<int32_t>(nb, static_cast<int32_t>(end_pos.size()));
                const int32_t tok_off = static_cast<int32_t>(p->toks.size());
                for (int32_t i = a; i < e; ++i)
                    p->toks.push_back(TokDesc{q_indptr[r] + i, L[r] == 1 ? tkv::kNoLimit : N[r] - L[r] + i, -1, 0});
                for (int32_t h = 0; h < s.hkv; ++h)
                    p->items.push_back(ItemDesc{h, tok_off, e - a, row_blk_off, nbk, 0, tkv::kItemRow, 0});
            });
        }
        st.n_items = static_cast<int32_t>(p->items.size() + p->wave_items.size());
        st.n_items_row = st.n_items - st.n_items_shared;
        sort_by_small_key_desc(p->wave_items, tkv::kWaveBlocks, [](const ItemDesc& a) { return a.n_blk; });
        // Wave streams.  Every wave runs items of one tile width T (its code path is fixed); waves
        // are split over the widths in proportion to their work.  Workgroups of kWaveWG waves are
        // dispatched round-robin over the 8 XCDs (each with its own L2), so wave w runs on XCD
        // (w / kWaveWG) % 8: all tiles of one (chunk, KV head), which read the same K/V blocks, go
        // to one XCD.  Groups are assigned to XCDs, and items to the XCD's waves, longest
        // processing time first.
        {
            constexpr int32_t kXcds = 8;
            const int32_t n_items = static_cast<int32_t>(p->wave_items.size());
            // The tile items share the launch with the wave grid and hold a workgroup slot each
            // (two per CU); when they are fewer than the slots, the wave grid takes the slots they
            // leave (at least half), so that no wave workgroup waits for a tile item to finish.
            const int32_t wg_slots = tkv::kWaveWorkers / tkv::kWaveWG;
            const int32_t n_tile = static_cast<int32_t>(p->items.size());
            int32_t target = tkv::kWaveWorkers;
            if (n_tile < wg_slots) target = std::max(wg_slots / 2, wg_slots - n_tile) / kXcds * kXcds * tkv::kWaveWG;
            // A light wave grid (under kWaveBlocksPerWave key blocks per wave) beside many tile items
            // shrinks, down to a quarter of the grid, so that its workgroups hold fewer of the slots
            // the tile items need (the shared-prefix pass of a few long prompts with one-block tails).
            int64_t wave_blocks = 0;
            for (const ItemDesc& it : p->wave_items) wave_blocks += it.n_blk;
            if (n_tile >= wg_slots) {
                const int64_t light = (wave_blocks / kWaveBlocksPerWave + kXcds * tkv::kWaveWG - 1) / (kXcds * tkv::kWaveWG) *
                                      (kXcds * tkv::kWaveWG);
                target = static_cast<int32_t>(std::max<int64_t>(tkv::kWaveWorkers / 4, std::min<int64_t>(target, light)));
            }
            if (opts && opts->waves > 0) target = std::max(kXcds, opts->waves);
            auto cost = [](const ItemDesc& it) { return static_cast<int64_t>(it.n_blk) * (3 + it.pad) + 4; };
            std::vector<std::vector<int32_t>> by_t(tkv::kWaveMaxTiles + 1);
            std::vector<int64_t> cost_t(tkv::kWaveMaxTiles + 1, 0);
            int64_t cost_all = 0;
            for (int32_t i = 0; i < n_items; ++i) {
                by_t[p->wave_items[i].pad].push_back(i);
                cost_t[p->wave_items[i].pad] += cost(p->wave_items[i]);
                cost_all += cost(p->wave_items[i]);
            }
            struct Wave {
                int32_t T;
                const int32_t* items;  // its items, in the XCD's flat list
                int32_t n;
            };
            // waves per XCD of each width: shares of the target in proportion to the work (at
            // least one, at most one per item on the XCD), the remainder going to the widths
            // with the largest fractional share, so that a large batch fills the target exactly
            std::vector<int32_t> per_xt(tkv::kWaveMaxTiles + 1, 0);
            {
                const int32_t target_x = std::max(1, target / kXcds);
                std::vector<double> frac(tkv::kWaveMaxTiles + 1, 0.0);
                int32_t used = 0;
                for (int32_t T = 1; T <= tkv::kWaveMaxTiles; ++T) {
                    if (by_t[T].empty()) continue;
                    const double want = static_cast<double>(target_x) * cost_t[T] / cost_all;
                    const int32_t cap = static_cast<int32_t>((by_t[T].size() + kXcds - 1) / kXcds);
                    per_xt[T] = std::min(cap, std::max(1, static_cast<int32_t>(want)));
                    frac[T] = per_xt[T] < cap ? want - per_xt[T] : -1.0;
                    used += per_xt[T];
                }
                while (used < target_x) {
                    int32_t best = -1;
                    for (int32_t T = 1; T <= tkv::kWaveMaxTiles; ++T)
                        if (frac[T] >= 0.0 && (best < 0 || frac[T] > frac[best])) best = T;
                    if (best < 0) break;
                    ++per_xt[best];
                    ++used;
                    const int32_t cap = static_cast<int32_t>((by_t[best].size() + kXcds - 1) / kXcds);
                    frac[best] = per_xt[best] < cap ? frac[best] - 1.0 + 1e-9 * cost_t[best] : -1.0;
                    if (frac[best] < 0.0 && per_xt[best] < cap) frac[best] = 0.0;
                }
            }
            // Each XCD's wave positions are shared out evenly among the widths (interleaved in
            // launch order); items go to the waves of their width longest processing time first.
            struct Slot {
                int32_t T;
                double key;
            };
            std::vector<std::vector<Wave>> xcd_waves(kXcds);
            std::vector<std::vector<int32_t>> xcd_flat(kXcds);
            std::vector<std::vector<std::vector<int32_t>>> xcd_items_t(kXcds, std::vector<std::vector<int32_t>>(tkv::kWaveMaxTiles + 1));
            for (int32_t T = 1; T <= tkv::kWaveMaxTiles; ++T) {
                const std::vector<int32_t>& its = by_t[T];
                if (its.empty()) continue;
                // groups (a chunk's tiles of one KV head) as lists in first-appearance order, built as
                // offsets into one array; the previous item of a KV head usually shares its group
                IdMap& gid = sc.gid;  // (first key block, KV head) -> group
                gid.reset(its.size());
                std::vector<int32_t>& grp = sc.grp;
                grp.resize(its.size());
                std::vector<int64_t> gcost;
                std::vector<uint64_t> last_key(s.hkv, ~uint64_t{0});
                std::vector<int32_t> last_group(s.hkv, -1);
                for (size_t k2 = 0; k2 < its.size(); ++k2) {
                    const ItemDesc& it = p->wave_items[its[k2]];
                    const uint64_t key = (static_cast<uint64_t>(it.blk_off) << 8) | static_cast<uint32_t>(it.kvh);
                    int32_t g2 = last_key[it.kvh] == key ? last_group[it.kvh] : -1;
                    if (g2 < 0) {
                        bool fresh = false;
                        g2 = gid.get(key, static_cast<int32_t>(gcost.size()), &fresh);
                        if (fresh) gcost.push_back(0);
                        last_key[it.kvh] = key;
                        last_group[it.kvh] = g2;
                    }
                    grp[k2] = g2;
                    gcost[g2] += cost(it);
                }
                std::vector<int32_t> goff(gcost.size() + 1, 0), gitems(its.size());
                for (size_t k2 = 0; k2 < its.size(); ++k2) ++goff[grp[k2] + 1];
                for (size_t g2 = 0; g2 < gcost.size(); ++g2) goff[g2 + 1] += goff[g2];
                {
                    std::vector<int32_t> fill(goff.begin(), goff.end() - 1);
                    for (size_t k2 = 0; k2 < its.size(); ++k2) gitems[fill[grp[k2]]++] = its[k2];
                }
                std::vector<int32_t> gorder(gcost.size());
                std::iota(gorder.begin(), gorder.end(), 0);
                std::stable_sort(gorder.begin(), gorder.end(), [&](int32_t a2, int32_t b2) { return gcost[a2] > gcost[b2]; });
                using Load = std::pair<int64_t, int32_t>;
                std::priority_queue<Load, std::vector<Load>, std::greater<Load>> xheap;
                for (int32_t x = 0; x < kXcds; ++x) xheap.push({0, x});
                for (int32_t g2 : gorder) {
                    Load l = xheap.top();
                    xheap.pop();
                    auto& dst = xcd_items_t[l.second][T];
                    dst.insert(dst.end(), gitems.begin() + goff[g2], gitems.begin() + goff[g2 + 1]);
                    l.first += gcost[g2];
                    xheap.push(l);
                }
            }
            for (int32_t x = 0; x < kXcds; ++x) {
                // this XCD's waves of each width, their positions interleaved in launch order
                std::vector<Slot> slots_x;
                for (int32_t T = 1; T <= tkv::kWaveMaxTiles; ++T) {
                    const int32_t nw = std::min<int32_t>(per_xt[T], static_cast<int32_t>(xcd_items_t[x][T].size()));
                    for (int32_t k = 0; k < nw; ++k) slots_x.push_back(Slot{T, (k + 0.5) / nw});
                }
                std::stable_sort(slots_x.begin(), slots_x.end(), [](const Slot& a2, const Slot& b2) { return a2.key < b2.key; });
                // items to waves longest processing time first, as (wave, item) in the order assigned;
                // then each wave's items gathered into one flat list per XCD, in that order
                std::vector<std::pair<int32_t, int32_t>> asg;
                for (int32_t T = 1; T <= tkv::kWaveMaxTiles; ++T) {
                    auto& items_t = xcd_items_t[x][T];
                    if (items_t.empty()) continue;
                    sort_by_small_key_desc(items_t, tkv::kWaveBlocks, [&](int32_t i) { return p->wave_items[i].n_blk; });
                    using Load = std::pair<int64_t, int32_t>;
                    std::priority_queue<Load, std::vector<Load>, std::greater<Load>> heap;
                    for (size_t j = 0; j < slots_x.size(); ++j)
                        if (slots_x[j].T == T) heap.push({0, static_cast<int32_t>(j)});
                    for (int32_t i : items_t) {
                        Load l = heap.top();
                        heap.pop();
                        asg.emplace_back(l.second, i);
                        l.first += cost(p->wave_items[i]);
                        heap.push(l);
                    }
                }
                std::vector<int32_t> off(slots_x.size() + 1, 0);
                for (const auto& a2 : asg) ++off[a2.first + 1];
                for (size_t j = 0; j < slots_x.size(); ++j) off[j + 1] += off[j];
                std::vector<int32_t>& flat = xcd_flat[x];
                flat.resize(asg.size());
                {
                    std::vector<int32_t> fill(off.begin(), off.end() - 1);
                    for (const auto& a2 : asg) flat[fill[a2.first]++] = a2.second;
                }
                std::vector<Wave> ws(slots_x.size());
                for (size_t j = 0; j < slots_x.size(); ++j) ws[j] = Wave{slots_x[j].T, flat.data() + off[j], off[j + 1] - off[j]};
                xcd_waves[x] = std::move(ws);
            }
            // launch order: workgroup k holds kWaveWG waves of XCD k % 8, in position order; an XCD
            // whose list has run out lends its slots to the longest remaining list
            size_t n_total = 0;
            for (auto& v : xcd_waves) n_total += v.size();
            // idle waves follow the busy ones (kMaxSpareWaves)
            const int64_t n_spare = std::min<int64_t>(kMaxSpareWaves,
                ((static_cast<int64_t>(n_tails) * s.hkv + 7) / 8 + tkv::kWaveWG - 1) / tkv::kWaveWG * tkv::kWaveWG);
            const size_t n_slots_w = (n_total + n_spare + tkv::kWaveWG - 1) / tkv::kWaveWG * tkv::kWaveWG;
            std::vector<size_t> next(kXcds, 0);
            std::vector<const Wave*> slots(n_slots_w, nullptr);
            for (size_t slot = 0; slot < n_slots_w; ++slot) {
                const int32_t x = static_cast<int32_t>((slot / tkv::kWaveWG) % kXcds);
                int32_t src = x;
                if (next[src] >= xcd_waves[src].size()) {
                    size_t best = 0;
                    src = -1;
                    for (int32_t y = 0; y < kXcds; ++y)
                        if (xcd_waves[y].size() - next[y] > best) {
                            best = xcd_waves[y].size() - next[y];
                            src = y;
                        }
                }
                if (src >= 0) slots[slot] = &xcd_waves[src][next[src]++];
            }
            // Wave w's first item is record w (so the wave's first load depends on nothing); its
            // other items follow all first records, as the range [wave_off[w], wave_off[w + 1]).
            p->wave_rec.assign(n_slots_w, -1);
            for (size_t w = 0; w < n_slots_w; ++w)
                if (slots[w] && slots[w]->n > 0) p->wave_rec[w] = slots[w]->items[0];
            p->wave_off.assign(1, static_cast<int32_t>(n_slots_w));
            for (size_t w = 0; w < n_slots_w; ++w) {
                const bool busy = slots[w] && slots[w]->n > 0;
                if (busy)
                    for (int32_t k = 1; k < slots[w]->n; ++k) p->wave_rec.push_back(slots[w]->items[k]);
                p->wave_off.push_back(static_cast<int32_t>(p->wave_rec.size()));
                p->wave_tiles.push_back(busy ? slots[w]->T : 0);
            }
        }
        st.n_items_wave = static_cast<int32_t>(p->wave_items.size());
        st.n_waves = static_cast<int32_t>(p->wave_tiles.size());
        st.n_idle_waves = static_cast<int32_t>(std::count(p->wave_tiles.begin(), p->wave_tiles.end(), 0));
        // a plan of a few tile items and nothing else gives each tile a CU to itself: its 128 rows then
        // run as eight 16-row waves, which shortens the tile's walk
        const int64_t tile8_max = opt(&tkv_plan_options::tile8_max_items, tkv::kTile8MaxItems);
        p->tile8 = p->wave_items.empty() && !p->items.empty() && static_cast<int64_t>(p->items.size()) <= tile8_max;
        st.n_slots = p->n_slots;
        st.n_merge = static_cast<int32_t>(p->merges.size());

        // Tile items run one workgroup each, dispatched in launch order with workgroup i on XCD
        // i % 8.  Items that read the same keys -- the same first block and KV head (a row's path
        // root, or a shared chunk) -- go to one XCD so that their repeated reads hit its L2.  Groups
        // are assigned to XCDs longest processing time first (cost = key blocks x active waves);
        // each XCD's list runs group by group and the lists are interleaved into the launch order.
        {
            constexpr int32_t kXcds = 8;
            auto cost = [&](const ItemDesc& it) {
                return static_cast<int64_t>(it.n_blk) * ((static_cast<int64_t>(it.n_tok) * G + 31) / 32) + 1;
            };
            IdMap& gid = sc.gid;  // (first key block, KV head) -> group
            gid.reset(p->items.size());
            std::vector<std::vector<int32_t>> groups;
            std::vector<int64_t> gcost;
            // items come in runs of one tile per KV head: the previous item of the same KV head is
            // usually in the same group, found without a lookup
            std::vector<uint64_t> last_key(s.hkv, ~uint64_t{0});
            std::vector<int32_t> last_group(s.hkv, -1);
            for (int32_t i = 0; i < static_cast<int32_t>(p->items.size()); ++i) {
                const ItemDesc& it = p->items[i];
                const uint64_t key = (static_cast<uint64_t>(p->blks[it.blk_off].blk) << 8) | static_cast<uint32_t>(it.kvh);
                int32_t g2 = last_key[it.kvh] == key ? last_group[it.kvh] : -1;
                if (g2 < 0) {
                    bool fresh = false;
                    g2 = gid.get(key, static_cast<int32_t>(groups.size()), &fresh);
                    if (fresh) {
                        groups.emplace_back();
                        gcost.push_back(0);
                    }
                    last_key[it.kvh] = key;
                    last_group[it.kvh] = g2;
                }
                groups[g2].push_back(i);
                gcost[g2] += cost(it);
            }
            std::vector<int32_t> gorder(groups.size());
            std::iota(gorder.begin(), gorder.end(), 0);
            std::stable_sort(gorder.begin(), gorder.end(), [&](int32_t a2, int32_t b2) { return gcost[a2] > gcost[b2]; });
            using Load = std::pair<int64_t, int32_t>;
            std::priority_queue<Load, std::vector<Load>, std::greater<Load>> xheap;
            for (int32_t x = 0; x < kXcds; ++x) xheap.push({0, x});
            // group-major: a group's items run together (so that the XCD's L2 holds the keys they
            // share), groups in the order assigned, each group's items longest first
            std::vector<std::vector<int32_t>> xl(kXcds);
            std::vector<std::pair<int64_t, int32_t>> by_cost;  // (-cost, place in the group): longest first, stable
            for (int32_t g2 : gorder) {
                Load l = xheap.top();
                xheap.pop();
                const std::vector<int32_t>& gi = groups[g2];
                by_cost.clear();
                for (size_t k2 = 0; k2 < gi.size(); ++k2)
                    by_cost.emplace_back(-cost(p->items[gi[k2]]), static_cast<int32_t>(k2));
                std::sort(by_cost.begin(), by_cost.end());
                for (const auto& bc : by_cost) xl[l.second].push_back(gi[bc.second]);
                l.first += gcost[g2];
                xheap.push(l);
            }
            std::vector<ItemDesc>& ordered = sc.ordered;
            ordered.clear();
            ordered.reserve(p->items.size());
            std::vector<size_t> next(kXcds, 0);
            while (ordered.size() < p->items.size()) {
                for (int32_t x = 0; x < kXcds && ordered.size() < p->items.size(); ++x) {
                    int32_t src = x;
                    if (next[src] >= xl[src].size()) {  // this XCD's list is done: lend it the longest remaining one
                        size_t best = 0;
                        for (int32_t y = 0; y < kXcds; ++y)
                            if (xl[y].size() - next[y] > best) {
                                best = xl[y].size() - next[y];
                                src = y;
                            }
                    }
                    ordered.push_back(p->items[xl[src][next[src]++]]);
                }
            }
            p->items.swap(ordered);
        }

        // ------------------------------------------------------------ workspace layout
        auto bytes = [](size_t n, size_t e) { return n * e; };
        size_t off = 0;
        p->off_items = off;
        off = align256(off + bytes(p->items.size(), sizeof(ItemDesc)));
        p->off_toks = off;
        off = align256(off + bytes(p->toks.size(), sizeof(TokDesc)));
        p->off_blks = off;
        off = align256(off + bytes(p->blks.size(), sizeof(BlkDesc)));
        p->off_merges = off;
        off = align256(off + bytes(p->merges.size(), sizeof(MergeDesc)));
        p->off_mslots = off;
        off = align256(off + bytes(p->merge_slots.size(), sizeof(int32_t)));
        p->off_wdesc = off;
        off = align256(off + bytes(p->wave_rec.size(), sizeof(tkv::WaveDesc)));
        p->off_woff = off;
        off = align256(off + bytes(p->wave_off.size(), sizeof(int32_t)));
        p->off_wtiles = off;
        off = align256(off + bytes(p->wave_tiles.size(), sizeof(int32_t)));
        p->desc_bytes = off;
        p->off_po = off;
        off = align256(off + bytes(static_cast<size_t>(p->n_slots) * s.hq * s.d, sizeof(uint16_t)));  // fp16 partial o
        p->off_plse = off;
        off = align256(off + bytes(static_cast<size_t>(p->n_slots) * s.hq, sizeof(float)));
        // room for the (word, value) pairs of a patch upload after an in-place update: a lengthened
        // tail changes one word per record; appended blocks and new chunks a few more
        p->patch_cap = n_tails == 0 ? 0 : static_cast<int32_t>(std::min<int64_t>(int64_t{1} << 24, static_cast<int64_t>(n_tails) * s.hkv * 4 + 8192));
        p->off_patch = off;
        off = align256(off + bytes(static_cast<size_t>(p->patch_cap), 2 * sizeof(int32_t)));
        p->total_bytes = std::max<size_t>(off, 256);
        // the image is written once: each section, its records in place, the padding zeroed
        p->image = tkv::take_image(p->desc_bytes, &p->image_cap);
        uint8_t* img = p->image.get();
        size_t filled = 0;
        auto put = [&](size_t o, const void* src, size_t n) {
            if (o > filled) std::memset(img + filled, 0, o - filled);
            if (n) std::memcpy(img + o, src, n);
            filled = o + n;
        };
        put(p->off_items, p->items.data(), bytes(p->items.size(), sizeof(ItemDesc)));
        put(p->off_toks, p->toks.data(), bytes(p->toks.size(), sizeof(TokDesc)));
        put(p->off_blks, p->blks.data(), bytes(p->blks.size(), sizeof(BlkDesc)));
        put(p->off_merges, p->merges.data(), bytes(p->merges.size(), sizeof(MergeDesc)));
        put(p->off_mslots, p->merge_slots.data(), bytes(p->merge_slots.size(), sizeof(int32_t)));
        put(p->off_wdesc, nullptr, 0);
        for (size_t r = 0; r < p->wave_rec.size(); ++r)
            write_record(p, p->wave_rec[r], img + p->off_wdesc + r * sizeof(tkv::WaveDesc));
        filled = p->off_wdesc + p->wave_rec.size() * sizeof(tkv::WaveDesc);
        put(p->off_woff, p->wave_off.data(), bytes(p->wave_off.size(), sizeof(int32_t)));
        put(p->off_wtiles, p->wave_tiles.data(), bytes(p->wave_tiles.size(), sizeof(int32_t)));
        if (p->desc_bytes > filled) std::memset(img + filled, 0, p->desc_bytes - filled);
    } catch (...) {
        give_plan(p);
        return set_error(TKV_ENOMEM, "tkv_plan_create: host allocation failed");
    }
    *out = p;
    return TKV_OK;
}

namespace tkv {
namespace {
struct ImagePool {
    std::mutex m;
    std::vector<std::pair<size_t, std::unique_ptr<uint8_t[]>>> free;  // (capacity, buffer)
};
// never destroyed: plans may be freed while the process exits
ImagePool& image_pool() {
    static ImagePool* pool = new ImagePool();
    return *pool;
}
constexpr size_t kPooledImages = 2;
}  // namespace

std::unique_ptr<uint8_t[]> take_image(size_t bytes, size_t* cap) {
    ImagePool& pool = image_pool();
    {
        std::lock_guard<std::mutex> lock(pool.m);
        size_t best = pool.free.size();
        for (size_t i = 0; i < pool.free.size(); ++i)
            if (pool.free[i].first >= bytes && (best == pool.free.size() || pool.free[i].first < pool.free[best].first))
                best = i;
        if (best < pool.free.size()) {
            *cap = pool.free[best].first;
            std::unique_ptr<uint8_t[]> img = std::move(pool.free[best].second);
            pool.free.erase(pool.free.begin() + static_cast<std::ptrdiff_t>(best));
            return img;
        }
    }
    *cap = std::max<size_t>(bytes + bytes / 8, 256);  // headroom for the next, slightly larger plan
    return std::unique_ptr<uint8_t[]>(new uint8_t[*cap]);
}

void give_image(std::unique_ptr<uint8_t[]> image, size_t cap) {
    if (!image) return;
    ImagePool& pool = image_pool();
    std::lock_guard<std::mutex> lock(pool.m);
    pool.free.emplace_back(cap, std::move(image));
    if (pool.free.size() > kPooledImages) {  // keep the largest
        auto smallest = std::min_element(pool.free.begin(), pool.free.end(),
                                         [](const auto& a, const auto& b) { return a.first < b.first; });
        pool.free.erase(smallest);
    }
}
}  // namespace tkv

TKV_EXPORT size_t tkv_plan_workspace_bytes(const tkv_plan* p) { return p ? p->total_bytes : 0; }

TKV_EXPORT void tkv_plan_destroy(tkv_plan* p) { give_plan(p); }

TKV_EXPORT int tkv_plan_get_stats(const tkv_plan* p, tkv_plan_stats* out) {
    tkv::clear_error();
    if (!p || !out) return set_error(TKV_EINVAL, "tkv_plan_get_stats: NULL argument");
    *out = p->stats;
    return TKV_OK;
}

TKV_EXPORT int tkv_plan_get_view(const tkv_plan* cp, tkv_plan_view* out) {
    tkv_plan* p = const_cast<tkv_plan*>(cp);
    tkv::clear_error();
    if (!p || !out) return set_error(TKV_EINVAL, "tkv_plan_get_view: NULL argument");
    // tile items, then wave items with their tokens and blocks placed after the tile items' ones
    try {
        p->view_items.assign(p->items.begin(), p->items.end());
        const int32_t nt = static_cast<int32_t>(p->toks.size()), nbk = static_cast<int32_t>(p->blks.size());
        for (ItemDesc it : p->wave_items) {
            it.tok_off += nt;
            it.blk_off += nbk;
            p->view_items.push_back(it);
        }
        p->view_toks.assign(p->toks.begin(), p->toks.end());
        p->view_toks.insert(p->view_toks.end(), p->wtoks.begin(), p->wtoks.end());
        p->view_blks.assign(p->blks.begin(), p->blks.end());
        p->view_blks.insert(p->view_blks.end(), p->wblks.begin(), p->wblks.end());
    } catch (...) {
        return set_error(TKV_ENOMEM, "tkv_plan_get_view: host allocation failed");
    }
    out->items = reinterpret_cast<const int32_t*>(p->view_items.data());
    out->toks = reinterpret_cast<const int32_t*>(p->view_toks.data());
    out->blks = reinterpret_cast<const int32_t*>(p->view_blks.data());
    out->merges = reinterpret_cast<const int32_t*>(p->merges.data());
    out->merge_slots = p->merge_slots.data();
    out->n_items = static_cast<int32_t>(p->view_items.size());
    out->n_toks = static_cast<int32_t>(p->view_toks.size());
    out->n_blks = static_cast<int32_t>(p->view_blks.size());
    out->n_merge = static_cast<int32_t>(p->merges.size());
    out->n_merge_slots = static_cast<int32_t>(p->merge_slots.size());
    out->n_slots = p->n_slots;
    return TKV_OK;
}

// ---------------------------------------------------------------------------- plan update
namespace {

// Every field of a plan's contents, exchanged (the instrumentation state stays with each object).
void swap_contents(tkv_plan* a, tkv_plan* b) {
    using std::swap;
    swap(a->shape, b->shape);
    swap(a->group, b->group);
    swap(a->all_decode, b->all_decode);
    swap(a->items, b->items);
    swap(a->wave_items, b->wave_items);
    swap(a->view_items, b->view_items);
    swap(a->view_toks, b->view_toks);
    swap(a->view_blks, b->view_blks);
    swap(a->toks, b->toks);
    swap(a->blks, b->blks);
    swap(a->wtoks, b->wtoks);
    swap(a->wblks, b->wblks);
    swap(a->merges, b->merges);
    swap(a->merge_slots, b->merge_slots);
    swap(a->wave_rec, b->wave_rec);
    swap(a->wave_off, b->wave_off);
    swap(a->wave_tiles, b->wave_tiles);
    swap(a->n_slots, b->n_slots);
    swap(a->tile8, b->tile8);
    swap(a->off_items, b->off_items);
    swap(a->off_toks, b->off_toks);
    swap(a->off_blks, b->off_blks);
    swap(a->off_merges, b->off_merges);
    swap(a->off_mslots, b->off_mslots);
    swap(a->off_wdesc, b->off_wdesc);
    swap(a->off_woff, b->off_woff);
    swap(a->off_wtiles, b->off_wtiles);
    swap(a->off_po, b->off_po);
    swap(a->off_plse, b->off_plse);
    swap(a->desc_bytes, b->desc_bytes);
    swap(a->total_bytes, b->total_bytes);
    swap(a->image, b->image);
    swap(a->image_cap, b->image_cap);
    swap(a->d_ws, b->d_ws);
    swap(a->ws_image, b->ws_image);
    swap(a->dirty, b->dirty);
    swap(a->dirty_over, b->dirty_over);
    swap(a->patch_pairs, b->patch_pairs);
    swap(a->off_patch, b->off_patch);
    swap(a->patch_cap, b->patch_cap);
    swap(a->stats, b->stats);
    swap(a->in, b->in);
}

// Room for `more` elements after the last, grown geometrically (an update appends a few each time).
template <class V>
void reserve_more(V& v, size_t more) {
    if (v.size() + more > v.capacity()) v.reserve(std::max(v.size() + more, 2 * v.capacity()));
}

// The lookups an in-place update needs, built once per plan.
void index_plan(tkv_plan* p) {
    tkv::PlanInputs& in = *p->in;
    const int32_t n_rows = p->stats.n_rows, hkv = p->shape.hkv;
    in.owner.assign(p->shape.num_blocks, -1);
    for (int32_t r = 0; r < n_rows; ++r)
        for (int64_t j = in.row_start[r]; j < in.row_start[r] + in.row_len[r]; ++j) {
            int32_t& o = in.owner[in.kv_blocks[j]];
            o = o == -1 || o == r ? r : -2;
        }
    in.rec_of.assign(p->wave_items.size(), -1);
    for (size_t w = 0; w < p->wave_rec.size(); ++w)
        if (p->wave_rec[w] >= 0) in.rec_of[p->wave_rec[w]] = static_cast<int32_t>(w);
    in.run_items.assign(p->wblks.size() / tkv::kWaveBlocks * hkv, -1);
    std::vector<uint8_t> is_tail(p->wblks.size() / tkv::kWaveBlocks, 0);
    for (int32_t r = 0; r < n_rows; ++r)
        if (in.tail_run[r] >= 0) is_tail[in.tail_run[r]] = 1;
    for (size_t i = 0; i < p->wave_items.size(); ++i) {
        const ItemDesc& it = p->wave_items[i];
        const int32_t run = it.blk_off / tkv::kWaveBlocks;
        if (is_tail[run]) in.run_items[static_cast<size_t>(run) * hkv + it.kvh] = static_cast<int32_t>(i);
    }
    in.free_waves.clear();
    const int32_t n_first = p->wave_off.empty() ? 0 : p->wave_off[0];
    for (int32_t w = n_first - 1; w >= 0; --w)
        if (p->wave_rec[w] < 0 && p->wave_tiles[w] == 0) in.free_waves.push_back(w);
    in.indexed = true;
}

}  // namespace

TKV_EXPORT int tkv_plan_update(tkv_plan* p, const int32_t* kv_indptr, const int32_t* kv_blocks,
                               const int32_t* block_len, int32_t* in_place) {
    tkv::clear_error();
    if (in_place) *in_place = 0;
    if (!p || !kv_indptr || !block_len) return set_error(TKV_EINVAL, "tkv_plan_update: NULL argument");
    tkv::PlanInputs& in = *p->in;
    const tkv_shape s = p->shape;
    const int32_t n_rows = p->stats.n_rows, hkv = s.hkv;
    if (kv_indptr[0] != 0) return set_error(TKV_EINVAL, "tkv_plan_update: kv_indptr[0] must be 0");
    if (n_rows > 0 && kv_indptr[n_rows] > 0 && !kv_blocks) return set_error(TKV_EINVAL, "tkv_plan_update: kv_blocks is NULL");
    auto is_decode = [&](int32_t r) { return in.q_indptr[r + 1] - in.q_indptr[r] == 1; };
    auto tail_item = [&](int32_t run, int32_t h) { return in.run_items[static_cast<size_t>(run) * hkv + h]; };
    tkv::wait_copies(p);  // the image is about to change (or move, when planned again)

    // ------------------------------------------------ can the plan take the new tables in place?
    // Every row keeps its blocks and may append new ones; a block changes length only as the last
    // block of a decode row's path or as one of its new blocks.  Such a row must have a tail chunk;
    // the new blocks fill it up to kWaveBlocks and may open one new chunk (its items on idle waves,
    // its partial in the token's free slot).  Checked first, then applied: nothing changes unless
    // all of it fits.  New blocks are marked in `owner` as taken by their row while checking.
    std::vector<int32_t> grown, lengthened;  // rows with new blocks; rows whose last block grew
    auto unmark = [&]() {
        for (int32_t r : grown)
            for (int32_t j = kv_indptr[r] + in.row_len[r]; j < kv_indptr[r + 1]; ++j)
                if (kv_blocks[j] >= 0 && kv_blocks[j] < s.num_blocks && in.owner[kv_blocks[j]] == -3 - r)
                    in.owner[kv_blocks[j]] = -1;
    };
    bool fits = true;
    size_t n_open = 0;      // new chunks
    size_t n_moved = 0;     // table entries of rows that outgrow their room
    std::vector<uint8_t> touched;  // rows the patch changes
    try {
        if (!in.indexed) index_plan(p);
        for (int32_t r = 0; r < n_rows && fits; ++r) {
            const int64_t o0 = in.row_start[r];
            const int32_t n_old = in.row_len[r];
            const int32_t n0 = kv_indptr[r], n_new = kv_indptr[r + 1] - n0;
            if (n_new < n_old || (n_old > 0 && std::memcmp(in.kv_blocks.data() + o0, kv_blocks + n0, n_old * sizeof(int32_t)))) {
                fits = false;
                break;
            }
            if (n_new == n_old) continue;
            if (!is_decode(r) || in.tail_run[r] < 0) {
                fits = false;
                break;
            }
            grown.push_back(r);
            for (int32_t j = n0 + n_old; j < n0 + n_new && fits; ++j) {
                const int32_t b = kv_blocks[j];
                if (b < 0 || b >= s.num_blocks || block_len[b] < 1 || block_len[b] > s.block_size || in.owner[b] != -1)
                    fits = false;
                else
                    in.owner[b] = -3 - r;
            }
            const int32_t room = tkv::kWaveBlocks - p->wave_items[tail_item(in.tail_run[r], 0)].n_blk;
            const int32_t extra = n_new - n_old;
            if (n_new > in.row_cap[r]) n_moved += static_cast<size_t>(n_new) + kRowSlack;
            if (extra > room) {  // one new chunk at most, and only into the token's free slot
                if (extra - room > tkv::kWaveBlocks || !in.spare[r] || in.merge_of[r] < 0) fits = false;
                n_open += 1;
            }
        }
        if (n_open * hkv > in.free_waves.size()) fits = false;
        for (int32_t b = 0; b < s.num_blocks && fits; ++b) {
            if (block_len[b] == in.block_len[b]) continue;
            const int32_t o = in.owner[b];
            if (o == -1 || o <= -3) continue;  // in no table, or one of this update's new blocks
            if (o == -2 || !is_decode(o) || in.tail_run[o] < 0 || in.kv_blocks[in.row_start[o] + in.row_len[o] - 1] != b ||
                block_len[b] < in.block_len[b] || block_len[b] > s.block_size)
                fits = false;
            else
                lengthened.push_back(o);
        }
        if (fits) {  // everything the patch appends to, so that it cannot fail half way
            touched.assign(n_rows, 0);
            reserve_more(p->wtoks, n_open);
            reserve_more(p->wblks, n_open * tkv::kWaveBlocks);
            reserve_more(p->wave_items, n_open * hkv);
            reserve_more(in.rec_of, n_open * hkv);
            reserve_more(in.run_items, n_open * hkv);
            reserve_more(in.kv_blocks, n_moved);
            if (p->dirty.capacity() < static_cast<size_t>(p->patch_cap)) p->dirty.reserve(p->patch_cap);
        }
    } catch (...) {
        unmark();
        return set_error(TKV_ENOMEM, "tkv_plan_update: host allocation failed");
    }
    if (!fits) {
        unmark();
        // plan the new tables from scratch, with the plan's own query layout and options
        tkv_plan* q = nullptr;
        const int rc = tkv_plan_create_ex(&s, n_rows, in.q_indptr.data(), kv_indptr, kv_blocks, block_len,
                                          in.mult.empty() ? nullptr : in.mult.data(), in.has_opts ? &in.opts : nullptr, &q);
        if (rc != TKV_OK) return rc;  // create's error message; the plan is unchanged
        swap_contents(p, q);
        tkv_plan_destroy(q);
        p->d_ws = nullptr;
        return TKV_OK;
    }

    // ------------------------------------------------ in place
    uint8_t* img = p->image.get();
    auto record = [&](int32_t item) {
        return reinterpret_cast<int32_t*>(img + p->off_wdesc + static_cast<size_t>(in.rec_of[item]) * sizeof(tkv::WaveDesc));
    };
    // the image words changed, for the next upload (within the reserved capacity; past it the
    // next upload copies the whole image)
    auto note = [&](const int32_t* e, int32_t n_words) {
        if (p->dirty_over || p->dirty.size() + n_words > static_cast<size_t>(p->patch_cap)) {
            p->dirty_over = true;
            return;
        }
        const int32_t base = static_cast<int32_t>(e - reinterpret_cast<const int32_t*>(img));
        for (int32_t k = 0; k < n_words; ++k) p->dirty.push_back(base + k);
    };
    constexpr int32_t kBlockWords = 4 * tkv::kWaveBlocks;
    auto rewrite_blocks = [&](int32_t item) {  // a record's block slots, noting the words that change
        int32_t* e = record(item);
        int32_t before[kBlockWords];
        std::memcpy(before, e, sizeof(before));
        write_record_blocks(p, p->wave_items[item], e);
        for (int32_t k = 0; k < kBlockWords; ++k)
            if (e[k] != before[k]) note(e + k, 1);
    };
    tkv_plan_stats& st = p->stats;
    const int64_t flops_per_key = 4ll * s.d * s.hq;
    for (int32_t r : lengthened) touched[r] = 1;
    for (int32_t r : grown) touched[r] = 1;
    for (int32_t r = 0; r < n_rows; ++r) {
        if (!touched[r]) continue;
        const int64_t o0 = in.row_start[r];
        const int32_t n_old = in.row_len[r];
        const int32_t n0 = kv_indptr[r], n_new = kv_indptr[r + 1] - n0;
        int32_t run = in.tail_run[r];
        BlkDesc* wb = &p->wblks[static_cast<size_t>(run) * tkv::kWaveBlocks];
        int32_t n = p->wave_items[tail_item(run, 0)].n_blk;
        int64_t added = 0;
        // the path's last block (the tail chunk's last) took new tokens
        const int32_t last = in.kv_blocks[o0 + n_old - 1];
        const int32_t grew = block_len[last] - in.block_len[last];
        if (grew) {
            added += grew;
            wb[n - 1].len = block_len[last];
            in.block_len[last] = block_len[last];
        }
        if (n_new == n_old) {  // no new block: only the records' last block length changes
            for (int32_t h = 0; h < hkv; ++h) {
                int32_t* e = record(tail_item(run, h)) + 4 * (n - 1) + 1;
                *e += grew;
                note(e, 1);
            }
            in.kv_len[r] += grew;
            st.path_kv_tokens += grew;
            st.uniq_kv_tokens += grew;
            st.flops += flops_per_key * grew;
            continue;
        }
        int32_t end = p->wave_items[tail_item(run, 0)].pos0;
        for (int32_t j = 0; j < n; ++j) end += wb[j].len;
        bool opened = false;
        for (int32_t j = n0 + n_old; j < n0 + n_new; ++j) {
            const int32_t b = kv_blocks[j];
            if (n == tkv::kWaveBlocks) {
                // The tail chunk is full, its items final.  A new chunk of the row's token takes the
                // following blocks; its partial goes to the token's free slot, after the others.
                for (int32_t h = 0; h < hkv; ++h) {
                    const int32_t i = tail_item(run, h);
                    p->wave_items[i].n_blk = n;
                    rewrite_blocks(i);
                }
                const int32_t T = p->wave_items[tail_item(run, 0)].pad;
                MergeDesc& md = p->merges[in.merge_of[r]];
                const int32_t slot = md.slot_off + md.n_slots;
                md.n_slots += 1;
                std::memcpy(img + p->off_merges + static_cast<size_t>(in.merge_of[r]) * sizeof(MergeDesc), &md, sizeof(MergeDesc));
                note(reinterpret_cast<const int32_t*>(img + p->off_merges) + static_cast<size_t>(in.merge_of[r]) * 4, 4);
                in.spare[r] = 0;
                const int32_t tok_off = static_cast<int32_t>(p->wtoks.size());
                p->wtoks.push_back(TokDesc{in.q_indptr[r], tkv::kNoLimit, slot, 0});
                run = static_cast<int32_t>(p->wblks.size() / tkv::kWaveBlocks);
                p->wblks.resize(p->wblks.size() + tkv::kWaveBlocks, BlkDesc{0, 0});
                wb = &p->wblks[static_cast<size_t>(run) * tkv::kWaveBlocks];
                n = 0;
                in.run_items.resize(in.run_items.size() + hkv, -1);
                for (int32_t h = 0; h < hkv; ++h) {
                    const int32_t i = static_cast<int32_t>(p->wave_items.size());
                    p->wave_items.push_back(ItemDesc{h, tok_off, 1, run * tkv::kWaveBlocks, 0, end, tkv::kItemWave, T});
                    const int32_t w = in.free_waves.back();
                    in.free_waves.pop_back();
                    p->wave_rec[w] = i;
                    p->wave_tiles[w] = T;
                    std::memcpy(img + p->off_wtiles + static_cast<size_t>(w) * sizeof(int32_t), &T, sizeof(int32_t));
                    note(reinterpret_cast<const int32_t*>(img + p->off_wtiles) + w, 1);
                    in.rec_of.push_back(w);
                    in.run_items[static_cast<size_t>(run) * hkv + h] = i;
                }
                in.tail_run[r] = run;
                st.n_items += hkv;
                st.n_items_shared += hkv;
                st.n_items_wave += hkv;
                st.n_idle_waves -= hkv;
                opened = true;
            }
            wb[n++] = BlkDesc{b, block_len[b]};
            end += block_len[b];
            added += block_len[b];
            in.owner[b] = r;
            in.block_len[b] = block_len[b];
        }
        for (int32_t h = 0; h < hkv; ++h) {
            const int32_t i = tail_item(run, h);
            p->wave_items[i].n_blk = n;
            if (opened) {
                write_record(p, i, reinterpret_cast<uint8_t*>(record(i)));
                note(record(i), static_cast<int32_t>(sizeof(tkv::WaveDesc) / sizeof(int32_t)));
            } else {
                rewrite_blocks(i);
            }
        }
        // the row's stored table takes the new blocks (moving to the end if it has no room)
        if (n_new > in.row_cap[r]) {
            const int64_t start = static_cast<int64_t>(in.kv_blocks.size());
            in.kv_blocks.resize(in.kv_blocks.size() + n_new + kRowSlack);  // within the reserved capacity
            std::memcpy(in.kv_blocks.data() + start, in.kv_blocks.data() + o0, n_old * sizeof(int32_t));
            in.row_start[r] = start;
            in.row_cap[r] = n_new + kRowSlack;
        }
        std::memcpy(in.kv_blocks.data() + in.row_start[r] + n_old, kv_blocks + n0 + n_old, (n_new - n_old) * sizeof(int32_t));
        in.row_len[r] = n_new;
        in.kv_len[r] += static_cast<int32_t>(added);
        st.path_kv_tokens += added;
        st.uniq_kv_tokens += added;  // a tail's blocks are its row's alone
        st.flops += flops_per_key * added;
    }
    // (in.block_len is kept for the blocks in the tables, above; a block in no table is skipped by
    // the check whatever its length there)
    p->d_ws = nullptr;
    if (in_place) *in_place = 1;
    return TKV_OK;
}

TKV_EXPORT int tkv_plan_dirty(const tkv_plan* p, const int32_t** words, int32_t* n, int32_t* complete) {
    tkv::clear_error();
    if (!p || !words || !n || !complete) return set_error(TKV_EINVAL, "tkv_plan_dirty: NULL argument");
    *words = p->dirty.data();
    *n = static_cast<int32_t>(p->dirty.size());
    *complete = p->dirty_over ? 0 : 1;
    return TKV_OK;
}

TKV_EXPORT int tkv_plan_image(const tkv_plan* p, const void** data, tkv_plan_layout* layout) {
    tkv::clear_error();
    if (!p || !data || !layout) return set_error(TKV_EINVAL, "tkv_plan_image: NULL argument");
    *data = p->image.get();
    *layout = tkv_plan_layout{p->off_items, p->off_toks, p->off_blks, p->off_merges, p->off_mslots,
                              p->off_wdesc, p->off_woff, p->off_wtiles, p->desc_bytes};
    return TKV_OK;
}

TKV_EXPORT int tkv_plan_upload(tkv_plan* p, void* d_ws, size_t bytes, void* stream) {
    tkv::clear_error();
    if (!p || !d_ws) return set_error(TKV_EINVAL, "tkv_plan_upload: NULL argument");
    if (bytes < p->total_bytes)
        return set_error(TKV_EINVAL, "tkv_plan_upload: workspace of %zu bytes < %zu needed", bytes, p->total_bytes);
    if (reinterpret_cast<uintptr_t>(d_ws) & 255) return set_error(TKV_EINVAL, "tkv_plan_upload: workspace not 256-byte aligned");
    return tkv::upload(p, d_ws, bytes, stream);
}

// The checks of an attention call before anything is enqueued; then the launch (attn.hip).
static int attention_call(const char* fn, const tkv_plan* p, const void* q, const void* k, const void* v, void* o,
                          float* lse, void* stream) {
    if (!p->d_ws) return set_error(TKV_EINVAL, "%s: plan has not been uploaded", fn);
    if (p->items.empty() && p->wave_items.empty()) return TKV_OK;
    if (!q || !k || !v || !o) return set_error(TKV_EINVAL, "%s: NULL tensor pointer", fn);
    return tkv::launch_attention(p, q, k, v, o, lse, stream);
}

TKV_EXPORT int tkv_decode(const tkv_plan* p, const void* q, const void* k, const void* v, void* o, float* lse,
                          void* stream) {
    tkv::clear_error();
    if (!p) return set_error(TKV_EINVAL, "tkv_decode: plan is NULL");
    if (!p->all_decode) return set_error(TKV_EINVAL, "tkv_decode: every row must have q_len 1 (use tkv_verify)");
    return attention_call("tkv_decode", p, q, k, v, o, lse, stream);
}

TKV_EXPORT int tkv_verify(const tkv_plan* p, const void* q, const void* k, const void* v, void* o, float* lse,
                          void* stream) {
    tkv::clear_error();
    if (!p) return set_error(TKV_EINVAL, "tkv_verify: plan is NULL");
    return attention_call("tkv_verify", p, q, k, v, o, lse, stream);
}
