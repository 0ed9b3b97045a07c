// Plan tables shared by the host builder (plan.cpp) and the HIP kernels.
//
// The plan is everything about a probe that depends only on the token layout,
// the sparse rule and the head counts: the region-relative block partition,
// the CSR of active (query block, key block) pairs, the attention work list in
// launch order, and the bookkeeping the evidence kernels need. It is built
// once on the host and uploaded as one device allocation.
#pragma once
#include <cstdint>
#include <string>
#include <vector>

namespace evisel {

enum Region : int32_t { kSys = 0, kVis = 1, kTxt = 2 };

// One region block: a query tile and a key tile at the same time.
struct BlockDesc {
  int32_t start;   // first token (global, packed)
  int32_t len;     // 1..B tokens
  int32_t region;  // Region
  int32_t aux;     // visual: global frame id of its first token;
                   // query: global query-row id of its first token; else -1
};

// Per video.
struct SeqDesc {
  int32_t tok0, vis0, txt0, end;        // token offsets
  int32_t frame0, n_frames;             // global frame range
  int32_t textrow0, n_text;             // global query-row range
  int64_t segbase;                      // offset of the [n_text][n_frames]
                                        // partial-LSE block (per head)
  int32_t tile0, n_tiles;               // query-token tiles (TextTile index)
};

// Query heads per work item. The heads of one item share a kv head, so each
// key/value tile staged in LDS serves all of them.
constexpr int kHeadsPerItem = 2;

// One attention work item: a query block, up to kHeadsPerItem consecutive
// query heads of one kv head, and a contiguous run of the block's CSR row.
// Items of split query-token rows carry the first head's partial slot; head
// head+i uses slot + i*nch.
// A paired item (qblock2 >= 0) holds a single head for two query blocks of
// one video and region, qblock for the first half of the work-group and
// qblock2 for the second, so that the odd head of a kv group does not leave
// half a work-group idle. Its key tiles are the two blocks' CSR runs merged
// by key block: entries [kb_begin, kb_end) of the paired-tile list.
struct WorkItem {
  int32_t qblock;    // -1: padding, exits immediately
  int32_t head;      // first query head
  int32_t nheads;    // 1..kHeadsPerItem (1 for a paired item)
  int32_t kb_begin;  // CSR positions [kb_begin, kb_end) (paired: tiles)
  int32_t kb_end;
  int32_t slot;      // -1 for visual/system rows; else first head's slot
  int32_t seq;       // video of the query block
  int32_t nch;       // chunks of this query-token row (0 for other rows)
  int32_t qblock2;   // -1, or the second query block of a paired item
  int32_t slot2;     // paired query-token item: qblock2's slot, else -1
  // Copies of the descriptors the kernel needs before its first loads, so
  // that the query rows and the first key/value tiles are fetched right
  // after the item itself: the two halves' query blocks (start token,
  // length) and the item's first two key tiles (static rule; k1len = 0
  // when the item has one tile).
  int32_t q0start, q0len, q1start, q1len;
  int32_t k0start, k0len;
  int32_t k1start, k1len;
};

// Key tile of a paired item: the key block and its CSR position in the row
// of each of the two query blocks (-1: not active for that query block).
struct PairedTile {
  int32_t block;
  int32_t pos[2];
};

// A query-token block and its chunk slots: slot(h, c) = slot0 + h*n_chunks + c.
struct TextTile {
  int32_t qblock;
  int32_t seq;
  int32_t n_chunks;
  int32_t slot0;
};

// A (query frame, earlier key frame) pair of one video that the sparse
// pattern can connect (cross-frame cue): the key frame lies in the key tile
// at CSR position `pos` of the query frame's block.
struct FramePair {
  int32_t pos;      // CSR position (query block row, key tile)
  int32_t a, b;     // global query and key frame, b < a
  int32_t qblock;   // block holding frame a's rows
  int32_t roff;     // first row of frame a within qblock
  int32_t koff;     // frame index of b within the key tile
};

struct Layout {
  std::vector<int32_t> n_sys, n_frames, n_text;
  int32_t Nv = 0;
};

// Sparse rule. tau > 0 selects the paper's adaptive top-p retention: the
// candidate key blocks of a row are then its whole causal history (the CSR
// is the all-causal one) and the retained subset is decided per (head, row)
// on the device; sink and window are ignored.
struct Rule {
  int32_t block = 64, sink = 1, window = -1;
  float tau = 0.f;
};

// Top-p mode: most candidate key blocks one attention work item may hold
// (its compacted list lives in LDS).
constexpr int kMaxItemCandidates = 2048;

struct Plan {
  // inputs
  Layout layout;
  Rule rule;
  int32_t hq = 0, hkv = 0;
  // sizes
  int64_t S = 0, T = 0, n_text_rows = 0, segtot = 0, n_slots = 0;
  int32_t chunk_blocks = 0;   // max key blocks per split item
  // tables
  std::vector<BlockDesc> blocks;
  std::vector<int32_t> row_ptr, col;
  std::vector<BlockDesc> col_desc;  // [nnz] descriptor of col[p]'s block
  std::vector<WorkItem> items;      // launch order
  std::vector<PairedTile> ptile;    // key tiles of paired items
  std::vector<BlockDesc> ptile_desc;  // descriptor of ptile[i].block
  std::vector<SeqDesc> seqs;
  std::vector<TextTile> tiles;
  std::vector<int32_t> frame_seq;   // [T] video of each global frame
  // top-p retention: per block its index among its video's selectable
  // (non-system) blocks in token order (-1 for system blocks); a block's
  // history H is local blocks [0, local). hist_words 32-bit words hold one
  // row's retained-history bits.
  std::vector<int32_t> blk_local;
  int32_t hist_words = 0;
  int32_t max_item_candidates = 0;
  // cross-frame cue: every connectable frame pair, and per frame the pairs
  // where it is the query frame (out) and the key frame (in), in pair order
  std::vector<FramePair> pairs;
  std::vector<int32_t> ff_out_ptr, ff_out_idx, ff_in_ptr, ff_in_idx;
};

// Builds the plan; returns "" on success or an error message.
std::string build_plan(const Layout& layout, const Rule& rule, int32_t hq,
                       int32_t hkv, Plan* out);

// Number of hardware queues the launch order interleaves (one per XCD).
constexpr int kXcds = 8;
// Concurrent work items the split heuristic aims to fill (256 CUs x 1).
constexpr int kTargetSlots = 512;

}  // namespace evisel
