// Internal declarations shared by the host library (block manager, planner, C entry points) and
// the HIP kernels.  Not part of the public ABI (include/treekv.h is).
#pragma once

#include <cstddef>
#include <cstdint>
#include <memory>
#include <string>
#include <vector>

#include "treekv.h"

#define TKV_EXPORT extern "C" __attribute__((visibility("default")))

namespace tkv {

// Records the message for tkv_last_error() and returns `code`.
int set_error(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// ------------------------------------------------------------------ device descriptors
constexpr int kBlock = 16;     // tokens per KV block
constexpr int kTileRows = 64;     // rows (q_len x G) from which a row is verified whole, not through segments
constexpr int kTileRowsWG = 128;  // query rows of a workgroup-kernel tile (4 waves x 2 column tiles x 16)
constexpr int kItemShared = 0;  // tile of several rows' tokens over one segment chunk (workgroup kernel)
constexpr int kItemRow = 1;     // tile of one row's tokens over its whole path (workgroup kernel)
constexpr int kItemWave = 2;    // tile of <= 16 T rows over one segment chunk (wave kernel)
constexpr int kWaveRows = 16;   // query rows of one MFMA column tile of the wave kernel
constexpr int kWaveMaxTiles = 2;  // column tiles a wave contracts against each K/V block
constexpr int kWaveMaxRows = 32;  // widest chunk (query rows) the wave kernel takes; wider ones use 128-row tiles
constexpr int kTileMinItems = 0;  // wide chunks go to the tile kernel only if they make this many items
constexpr int kWaveBlocks = 16; // key blocks of a wave-kernel item
constexpr int kWaveToks = 16;   // token slots of a wave-kernel record (a wave tile holds 16 T / G tokens,
                                // so G = 1 takes T = 1)
constexpr int kWaveWorkers = 2048;  // waves of the wave kernel: 2 workgroups of kWaveWG on each of 256 CUs
constexpr int kWaveWG = 4;      // waves per workgroup of the wave kernel (independent; no barriers)
constexpr int kTile8MaxItems = 256;  // tile items (and no wave grid) up to which 8-wave workgroups run them: one per CU
constexpr int kInterleaveRun = 32;   // workgroups per run when tile items and wave-grid workgroups alternate:
                                     // 8 XCDs x 4 shader engines, one workgroup of a kind per engine
constexpr int32_t kNoLimit = 1 << 30;  // causal limit of a q_len-1 token: it sees its whole path (kv_len <= 2^30)

// One work item: a tile of query tokens (each with all G query heads of one KV
// head) contracted against an ordered list of KV blocks.  Every query token of the tile sees the
// keys at positions <= its `limit`; keys are numbered along the path starting at `pos0`.
struct ItemDesc {
    int32_t kvh;      // KV head
    int32_t tok_off;  // first TokDesc of the tile
    int32_t n_tok;    // query tokens in the tile (n_tok * G <= kTileRowsWG, or <= 16 tiles for the wave kernel)
    int32_t blk_off;  // first BlkDesc of the key list
    int32_t n_blk;    // blocks in the key list
    int32_t pos0;     // path position of the first key
    int32_t kind;     // kItemShared (partials of shared/private segments) or kItemRow (whole path)
    int32_t pad;
};

struct TokDesc {
    int32_t qtok;   // query token index (row of q / o)
    int32_t limit;  // largest visible key position
    int32_t slot;   // partial slot (>= 0) or -1: this item covers the token's whole path -> o, lse
    int32_t pad;
};

struct BlkDesc {
    int32_t blk;  // pool block id
    int32_t len;  // tokens in the block (1..16)
};

// A wave-kernel item as one 512-byte record that a wave loads with one 16-byte load per lane (lane l
// gets word l % 32); block fields come out with v_readlane, token fields with ds_bpermute.
//   word j      (j < 16): {pool block id, length, path position, header word j} of key block j
//                         ({block 0's id, 0, 0} past the item's blocks); header words:
//                         0 KV head, 1 tile tokens, 2 key blocks (rounded up to even for tile widths
//                         1 and 2, whose waves walk blocks in pairs)
//   word 16 + t (t < 16): {query token, causal limit, partial slot (-1: final output), 0} of tile
//                         token t (token 0's past the tile)
struct WaveDesc {
    int32_t e[4 * (kWaveBlocks + kWaveToks)];
};

struct MergeDesc {
    int32_t qtok;
    int32_t slot_off;  // first partial slot of the token (its slots are contiguous)
    int32_t n_slots;
    int32_t pad;
};

// What tkv_plan_update needs beyond the plan itself: the inputs the plan was made from (to check
// that tables only grew, and to plan again when they did not grow in place) and, per row, its tail
// chunk -- the last chunk of a decode row's private segment when the wave kernel runs it.
struct PlanInputs {
    std::vector<int32_t> q_indptr, block_len, mult;
    // each row's table: kv_blocks[row_start[r] .. + row_len[r]), with room up to row_cap[r] (a row
    // that outgrows its room moves to the end of kv_blocks, with room for kRowSlack more)
    std::vector<int32_t> kv_blocks, row_len, row_cap;
    std::vector<int64_t> row_start;
    tkv_plan_options opts{};
    bool has_opts = false;
    std::vector<int32_t> kv_len;     // [n_rows]
    std::vector<int32_t> tail_run;   // [n_rows] wblks run (index / kWaveBlocks) of the tail chunk, or -1
    std::vector<int32_t> spare;      // [n_rows] 1: the token's partial range ends in an unused slot
    std::vector<int32_t> merge_of;   // [n_rows] the token's MergeDesc, or -1
    // built on the first in-place update
    bool indexed = false;
    std::vector<int32_t> owner;      // [num_blocks] the one row whose table holds the block, -1 none, -2 several
    std::vector<int32_t> run_items;  // [n_runs * hkv] wave items of each tail run, by KV head (-1: none)
    std::vector<int32_t> rec_of;     // [n wave items] record index
    std::vector<int32_t> free_waves; // idle waves (first records unused), taken from the back
};

}  // namespace tkv

// ------------------------------------------------------------------ plan (host)
// Every field below is also named by clear_plan and swap_contents in plan.cpp.
struct tkv_plan {
    tkv_shape shape{};
    int32_t group = 1;
    bool all_decode = true;
    std::vector<tkv::ItemDesc> items;       // workgroup-kernel items
    std::vector<tkv::ItemDesc> wave_items;  // wave-kernel items, longest first
    std::vector<tkv::ItemDesc> view_items;  // items then wave_items (tkv_plan_get_view)
    std::vector<tkv::TokDesc> view_toks;    // toks then wtoks
    std::vector<tkv::BlkDesc> view_blks;    // blks then wblks
    std::vector<tkv::TokDesc> toks;         // tile items' tokens (device image)
    std::vector<tkv::BlkDesc> blks;         // tile items' key blocks (device image)
    std::vector<tkv::TokDesc> wtoks;        // wave items' tokens (host: the records carry them)
    std::vector<tkv::BlkDesc> wblks;        // wave chunks' key blocks, kWaveBlocks slots per chunk (host)
    std::vector<tkv::MergeDesc> merges;
    std::vector<int32_t> merge_slots;
    std::vector<int32_t> wave_rec;            // wave-kernel records, as the wave item each holds (-1: none):
                                              // record w is wave w's first item, then each wave's further
                                              // items contiguously (written into the image by the layout)
    std::vector<int32_t> wave_off;            // [n_waves + 1] wave w's further items: [off[w], off[w+1])
    std::vector<int32_t> wave_tiles;          // [n_waves] column tiles of the wave's items (0: no work)
    int32_t n_slots = 0;
    bool tile8 = false;  // tile items only, few enough to run as 8-wave workgroups (kTile8MaxItems)
    // workspace layout (byte offsets)
    size_t off_items = 0, off_toks = 0, off_blks = 0, off_merges = 0, off_mslots = 0, off_wdesc = 0, off_woff = 0, off_wtiles = 0;
    size_t off_po = 0, off_plse = 0, desc_bytes = 0, total_bytes = 0;
    std::unique_ptr<uint8_t[]> image;  // host copy of the descriptor region (desc_bytes)
    size_t image_cap = 0;              // bytes allocated for it (returned to the image pool on destroy)
    void* d_ws = nullptr;        // uploaded workspace (caller-owned)
    // Patch uploads: ws_image is the workspace that holds the image as of the last upload; `dirty`
    // lists the image words in-place updates changed since (word indices, repeats allowed), complete
    // unless dirty_over.  The next upload into ws_image sends only those words, as (index, value)
    // pairs into the workspace's patch region (patch_cap pairs at off_patch; 0 for plans that cannot
    // be updated in place), and a small kernel writes them in.
    void* ws_image = nullptr;
    std::vector<int32_t> dirty;
    bool dirty_over = false;
    std::vector<int32_t> patch_pairs;  // host staging of the pairs
    size_t off_patch = 0;
    int32_t patch_cap = 0;
    tkv_plan_stats stats{};
    std::unique_ptr<tkv::PlanInputs> in;  // for tkv_plan_update
    // The last copy from this plan's host memory (upload, no-allocation call): an event recorded on
    // the stream after it, waited for before that memory is changed, reused or recycled.
    mutable void* copy_event = nullptr;
    mutable bool copy_pending = false;
    // instrumentation: 3 HIP events per recorded call (see tkv_plan_profile)
    mutable int32_t prof_max = 0;
    mutable int32_t prof_n = 0;
    mutable std::vector<void*> prof_events;
    ~tkv_plan();
};

namespace tkv {
// Plan images of destroyed plans, kept for the next plans (plan.cpp): a decode loop that plans every
// step then writes into memory that is already mapped.  take_image returns at least `bytes`.
std::unique_ptr<uint8_t[]> take_image(size_t bytes, size_t* cap);
void give_image(std::unique_ptr<uint8_t[]> image, size_t cap);
// Launchers (attn.hip).  launch_attention: an uploaded plan with work and non-NULL tensors (the
// entry points check these first).
int launch_attention(const tkv_plan* p, const void* q, const void* k, const void* v, void* o,
                     float* lse, void* stream);
int upload(tkv_plan* p, void* d_ws, size_t bytes, void* stream);
// Waits until the last copy from the plan's host memory has completed (attn.hip).
void wait_copies(const tkv_plan* p);
}  // namespace tkv
