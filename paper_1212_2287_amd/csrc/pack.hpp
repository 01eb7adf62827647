// pack.hpp -- host-side model packer for the gfx950 tree-ensemble scorer.
//
// Turns the caller's flat creation-order arrays into the device layout the kernels walk:
// one 8-byte record per node, trees re-laid out breadth-first with the two children of a node
// in adjacent slots (the contiguous Struct+ layout of Section 3, which keeps explicit child
// links so unbalanced trees pack without empty slots), trees ordered by their expected lockstep
// length, and a plan of LDS tiles (runs of whole trees that fit the per-workgroup LDS budget).
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace treeens {

// One node record, 8 bytes: {thr, w}.
//   internal node: thr = threshold (nudged to the next float up under the strict rule)
//   leaf:          thr = leaf value
// w packs the feature column and the child link in one of two formats:
//   narrow: w = (left child link << 16) | column byte offset             (column < 64 KiB)
//   wide:   w = (left child link << kWideChildShift) | column byte offset (column < 128 KiB)
// In `nodes` the link is tree-relative (the node's index in its tree). In the tile images the
// kernels walk, it is the child's absolute LDS record index (LDS byte address / 8), so a step
// needs no per-tree base. The right child follows the left one. A leaf links to itself and has
// column offset 0.
// The column byte offset of feature f is (f + 1) * docs_per_block * elem_bytes: the offset of
// f's column in the staged document tile, so a lane's feature address is
// (w & column mask) | (lane * elem_bytes).
// Column 0 of the tile holds NaN (or code 0) for every document, so a leaf compares it with its
// value, gets "left" and its link is itself: leaves absorb any further steps, and a lane is at a
// leaf exactly when its record's column offset is 0.
struct NodeRec {
    uint32_t thr_bits;
    uint32_t w;
};
static_assert(sizeof(NodeRec) == 8, "node record must be 8 bytes");
constexpr int kWideChildShift = 17;
constexpr uint32_t kNarrowColMask = 0xffffu;
constexpr uint32_t kWideColMask = (1u << kWideChildShift) - 1; // column offsets < 128 KiB
constexpr int kNarrowMaxTreeNodes = 1 << 16;                    // 16-bit child index
// Largest tree accepted (nodes): 32,768 leaves.
constexpr int kMaxTreeNodes = 65535;

// Big trees: a tree whose records do not fit one LDS tile slot (with the tile's header and K
// root copies) is not tiled. It is packed after all tiled trees, in its own record format, and
// the scoring kernel walks it from device memory (the records stay in L2), reading the
// documents' features from the staged LDS tile as for every other tree:
//   w = (tree-relative left child << kBigLinkShift) | column index (f + 1; 0 for a leaf)
// with thr as in NodeRec. The right child follows the left one, a leaf links to itself, and
// column 0 is the NaN (or code 0) column, so leaves absorb further steps here too.
constexpr int kBigLinkShift = 16;
constexpr uint32_t kBigColMask = 0xffffu;

// A run of whole trees [tree_begin, tree_end) (packed order) staged into LDS together.
struct Tile {
    int32_t tree_begin;
    int32_t tree_end;
    int32_t max_depth;      // deepest tree in the run
    int32_t node_begin;     // packed node offset of tree_begin
    int32_t complete_depth; // d if every tree of the run is complete of depth d, else -1
};
constexpr int kMaxTileTrees = 1024;

// Tile image: what one tile's LDS slot holds, laid out in device memory exactly as it is
// copied (records of 8 bytes):
//   word 0     number of trees n in the tile
//   word 1     complete depth d if every tree is complete of depth d, else -1 (as int32)
//   word 2     packed index of the tile's first tree
//   word 3     records to copy for the next tile of the same tiling (0 after the last one)
//   records 2.. a copy of each tree's root record, padded up to a multiple of the interleave K
//              with the all-zero self-linked leaf (value 0), so a walker reads its K roots with
//              one or two broadcast reads
//   then the node records of the n trees, child links as absolute LDS record indices.
// Images of one tiling sit at a fixed stride (the largest image of that tiling), so the
// kernel locates tile t without a table.
constexpr int kHeaderFixedWords = 4;

// Walker packets. In plans of 64- or 32-document blocks each of the 16 waves streams packets
// through a sub-slot of its own, so walkers never wait for one another between tiles. Walker h
// of wave v (one walker per wave for 64-document blocks, two half-waves for 32; walker index
// v * P + h of HW = 16 * P) owns groups of K trees g = v * P + h + r * HW, r = 0, 1, ... (rounds).
// Two-workgroup plans cut the tile slot into the 16 sub-slots; one-workgroup plans cut all of
// the LDS past the document tile but a zero record of their own (their feature trace, whose
// bitmasks sit past the shared tiles, keeps walking the shared tiles). A packet is a run of
// consecutive rounds of one wave that fits the sub-slot, in P equal parts, one per walker,
// each laid out as
//   record 0   number of groups n in the packet (the same in every part); the complete depth d
//              common to every tree of the packet, else -1
//   record 1   index of the walker's first group in the packet (later ones follow at stride HW)
//   records 2.. the K root copies of each group (the zero record for slots past the last tree)
//   then       the LDS record index of each tree's first record, 16 bits each (for leaf ids),
//              padded to a whole record
//   then       the trees' records, child links as absolute LDS record indices of the part.
// A wave loads its next packet into registers while it walks the current one. Plans in which
// one group outgrows a part keep the shared tiles.
constexpr int kPacketHeaderRecs = 2;
constexpr int kPacketWalkers = 16;

// Compact packets: coded plans of 64-document blocks with one workgroup per CU, whose trees have
// at most 511 nodes. A node is one 32-bit record
//   bits 21..31  threshold code k + 1 (2047 for a NaN threshold, which never sends right; a
//                leaf: 2047 if it is the left child of its pair, 0 if the right one)
//   bits 11..20  column index f + 1 (0 for a leaf)
//   bits  3..10  byte offset of the node's children pair in its window (a leaf: its own pair)
//   bit   2      a leaf's side in its pair (0 for an internal node)
// and a tree is its root record plus its children pairs (breadth-first, as in `nodes`), the
// pairs 8-byte aligned. A step reads the document's staged value and the whole children pair
// together (one dependent LDS round trip per step, not two) and keeps the side the comparison
// picks. Documents are staged as code << kCompactCodeShift | 31, so that the unsigned compare of
// that 16-bit value with the record's upper half is code >= threshold (the column bits below
// the threshold are absorbed by the 31). Leaf values stay in device memory: each packet has a
// payload array of the same shape holding, at a leaf's position, its value's bits (the
// leaf-vector row + 1 for vector-valued leaves) and, in a second array, its input node id.
// Each wave's LDS holds K = 2 windows of 2 KiB (window i takes slot i of
// every group of the packet; its last 8 bytes are a pair of zero records, {2047 << 21 | own
// offset}, for idle slots, payload 0) past the document tile. A packet is, in device memory,
// its windows then a header of kCompactHeaderBytes, which the kernel keeps in registers:
//   word 0 groups n, word 1 complete depth d (or -1), word 2 the wave's first group in the packet
//   (later ones follow at stride 16), word 3 zero, words 4.. the K root records of each group.
constexpr int kCompactTrees = 2;          // K: trees per lane, one window each
constexpr int kCompactWindowBytes = 4096; // all windows of one wave
constexpr int kCompactHeaderBytes = 512;
constexpr int kCompactPacketBytes = kCompactWindowBytes + kCompactHeaderBytes;
constexpr int kCompactHeaderWords = 4;
constexpr int kCompactThrShift = 21;
constexpr int kCompactColShift = 11;
constexpr uint32_t kCompactNeverRight = 2047u;
constexpr int kCompactMaxColumns = 1023;  // column index field
constexpr int kCompactMaxTreeNodes = 511; // root + 255 pairs: 2,040 bytes, one 2 KiB window
constexpr int kCompactCodeShift = 5;
// LDS byte address of the first window (windows are aligned to their size, at most 2 KiB)
inline int32_t compact_window_base(int32_t xs_bytes) { return (xs_bytes + 2047) & ~2047; }

// Launch plan fixed at create time from the model's feature range.
struct LdsPlan {
    int32_t docs_per_block; // documents a workgroup stages (power of two, 8..64)
    int32_t xs_bytes;       // staged document tile: (n_cols + 1) columns x docs_per_block floats
    int32_t tile_bytes;     // LDS bytes of a tile slot (header + node records)
    int32_t zero_rec;       // LDS byte address of the all-zero self-linked leaf (after the slot)
    int32_t wg_threads;     // workgroup size
    int32_t lds_bytes;      // total dynamic LDS per workgroup
    int32_t interleave;     // trees each lane walks at once (K)
    int32_t narrow;         // 1: narrow record format (see NodeRec), 0: wide
    int32_t coded;          // 1: documents are staged as 16-bit threshold codes (see below)
    int32_t elem_bytes;     // bytes per staged feature value: 4 (float) or 2 (code)
    // feature-access trace: LDS byte address of the per-document feature bitmasks
    // (ceil(n_cols / 32) words per document, [word][docs_per_block]); with two-workgroup plans
    // it lies past their half of the LDS, so the trace runs one workgroup per CU
    int32_t usage_off;
};

// Coded features (exact). For each feature f let T_f be the model's distinct thresholds of f,
// sorted (after the strict-rule nudge; -0.0 folded into +0.0; NaN thresholds left out), and
// code_f(x) = |{t in T_f : x >= t}| (0 for a NaN x). Then x >= T_f[k] <=> code_f(x) >= k + 1,
// so a node on threshold T_f[k] stores k + 1 and compares codes as unsigned integers; a node
// whose threshold is NaN (never "right") stores 0xFFFF, above every code. A leaf keeps its
// value's bits in the threshold slot, with +0.0 stored as -0.0 so the bits are never 0: the
// leaves' code column holds 0, and 0 >= bits is false, so leaves still go "left" to themselves.
// Coding halves the staged bytes per document; it is used when float features would not fit
// 64 documents in the LDS document tile.
// The coding kernel takes the features in chunks. A chunk of s search steps gives each of its
// features 2^s - 1 table entries, slots 1 .. 2^s - 1 of a complete search tree in breadth-first
// order (slot i has children 2i and 2i + 1; slot i is entry i - 1): the feature's sorted list
// padded with NaN. Descending i = 2i + (x >= slot i) for s steps from i = 1 ends at
// 2^s + code_f(x): NaN entries never compare true (and sort after every threshold), so they
// count nothing, and a NaN x never goes right. The odd stride puts the same slot of successive
// features in different LDS banks.
struct CodeChunk {
    int32_t f_begin, f_end;         // features [f_begin, f_end)
    int32_t table_begin, table_end; // their (f_end - f_begin) * (2^s - 1) entries in code_search
    int32_t search_steps;           // s: bits of the longest threshold list of the chunk
};
constexpr int kCodeTableFloats = 16384;  // LDS table slots per coding workgroup (64 KiB)
constexpr int kCodeChunkFeatures = 256;  // features per coding workgroup at most
constexpr uint32_t kMaxCode = 0xFFFEu;    // codes are 16-bit; 0xFFFF = "never right"

constexpr int kLdsPerCu = 160 * 1024;  // gfx950 LDS per compute unit
// The kernels prefetch tiles into registers (1,024 threads x kPrefetch records): at most 6
// records per thread (one tile) when two workgroups share a CU (64 VGPRs each); 16 when one
// owns it, as two tiles of up to 8 records per thread each (64 KiB) in flight at once.
constexpr int kPrefetchHalf = 6;
constexpr int kPrefetchFull = 16;
constexpr int kXsMaxBytes = 96 * 1024; // cap on the staged document tile
constexpr int kTwoWgXsBytes = 40 * 1024; // tiles up to this size leave room for 2 workgroups/CU
constexpr int kTileLevels = 5;         // tilings at budget, budget/2, ..., budget/16
// bitmask bytes of a two-workgroup plan's 64-document tile at most (n_cols + 1 <= 160 columns)
constexpr int kUsageHalfBytes = ((kTwoWgXsBytes / (64 * 4) - 1 + 31) / 32) * 64 * 4;

struct Packed {
    int32_t n_trees = 0;
    int32_t n_small = 0;   // trees [0, n_small) are tiled; [n_small, n_trees) are big trees
    int32_t n_cols = 0;    // 1 + largest feature id read (0 if none)
    int32_t max_depth = 0; // over all trees
    LdsPlan plan{};
    std::vector<NodeRec> nodes;          // all trees, packed order
    std::vector<uint32_t> tree_node_off; // [n_trees + 1] packed node offset of each tree
    std::vector<uint32_t> tree_depth;    // [n_trees]
    std::vector<int32_t> tree_orig;      // [n_trees] input index of packed tree t
    std::vector<int32_t> orig_id;        // [n_nodes] input tree-local id of packed node
    std::vector<Tile> tiles;             // all tiling levels, concatenated
    int32_t level_begin[kTileLevels + 1] = {};
    // tile images (see above), all tilings concatenated
    std::vector<NodeRec> images;
    int64_t level_image_off[kTileLevels] = {}; // first record of each tiling's images
    int32_t level_slot_recs[kTileLevels] = {}; // image stride of each tiling, in records
    std::vector<uint32_t> tile_recs;           // [tiles] records to copy for each tile
    // walker rounds (groups of walkers x interleave trees) of the fullest tile of each tiling,
    // and of all tiles of tiling 0: the launch planner's unit of time
    int32_t level_max_rounds[kTileLevels] = {};
    int64_t total_rounds = 0;
    // feature trace of a two-workgroup plan: LDS byte address of the bitmasks in the tile slot
    // past the largest tiling-0 image (past the walkers' sub-slots with packets), or -1 when
    // they do not fit before the zero record
    int32_t usage_slot_off = -1;
    // Walker packets (see kPacketHeaderRecs): wave
    // v's packet q is packets[(v * pk_per_walker + q) * pk_recs, ...), linked for its sub-slot
    // at LDS record xs_bytes / 8 + v * pk_recs. pk_recs == 0: the plan walks shared tiles.
    int32_t pk_recs = 0;
    int32_t pk_zero_rec = 0; // LDS byte address of the zero record the packets' padding links to
    int32_t pk_per_walker = 0;
    int32_t pk_max_groups = 0;   // groups in the fullest packet
    int64_t pk_total_rounds = 0; // sum over packet indices of the most groups any walker has there
    std::vector<NodeRec> packets;
    // Compact packets (see kCompactWindowBytes), used in place of the packets above when
    // cp_k > 0: trees per lane, packets per wave, groups in the fullest packet, the planner's
    // rounds, wave v's packet q at cp_packets[(v * cp_per_walker + q) * kCompactPacketBytes / 4],
    // and the leaf payloads and input node ids at the same positions.
    int32_t cp_k = 0;
    int32_t cp_per_walker = 0;
    int32_t cp_max_groups = 0;
    int64_t cp_total_rounds = 0;
    std::vector<uint32_t> cp_packets;
    std::vector<uint32_t> cp_leaf;
    std::vector<int32_t> cp_leaf_id;
    // vector-valued leaves (n_outputs > 1): a leaf's threshold slot holds 2 + its packed node
    // index instead of a value, and row (thr - 1) of leaf_vec holds its n_outputs values,
    // padded to vec_stride (a multiple of 4) floats; row 0 is zero (the all-zero record's row)
    int32_t n_outputs = 1;
    int32_t vec_stride = 0;
    std::vector<float> leaf_vec;
    // coded models only
    std::vector<float> code_table;         // T_0, T_1, ... concatenated
    std::vector<uint32_t> code_table_off;  // [n_cols + 1] start of T_f in code_table
    std::vector<CodeChunk> code_chunks;    // features grouped for the coding kernel
    std::vector<float> code_search;        // the chunks' search tables (see CodeChunk)
};

// Outputs per leaf at most (vector-valued leaves).
constexpr int kMaxOutputs = 256;

// Threshold slot of the all-zero self-linked record (idle walker slots, root-copy padding):
// value 0.0 for float leaves, -0.0 for coded ones (never zero bits), and row 0 of the
// leaf-vector table (all zeros) for vector-valued leaves.
inline uint32_t zero_record_value(const LdsPlan &plan, bool vec) {
    return vec ? 1u : plan.coded ? 0x80000000u : 0u;
}

// Kernels specialised for one model (create flag TREE_ENS_CODEGEN): limits of the generated
// program and its block size.
constexpr uint32_t kCodegenFlag = 2u;
constexpr int kCodegenMaxNodes = 1 << 16;
constexpr int kCodegenMaxDepth = 64;
constexpr int kCodegenThreads = 256;
constexpr int kCodegenTreesPerFunction = 32;

// Status codes match the public header.
constexpr int kOk = 0, kErrArg = -1, kErrModel = -2;

// Validate and pack. Returns kOk or an error code with a message in `err`. Pure host code:
// no HIP call is made, so every model error is reported without a device.
// value holds n_outputs floats per node ([n_nodes][n_outputs], read at leaves only).
int pack_model(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
               const float *threshold, const int32_t *left, const int32_t *right,
               const float *value, int32_t n_outputs, uint32_t flags, Packed &out,
               std::string &err);

// HIP source of a scoring kernel specialised for the model (nested if/else with constant
// feature ids, thresholds and leaf values; entry point `tree_ens_cg`). Validates the model as
// pack_model does; kErrModel beyond kCodegenMaxNodes nodes or depth kCodegenMaxDepth.
int codegen_source(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                   const float *threshold, const int32_t *left, const int32_t *right,
                   const float *value, uint32_t flags, std::string &src, std::string &err);

} // namespace treeens
