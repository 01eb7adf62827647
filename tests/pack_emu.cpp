// pack_emu.cpp -- host emulation of the scoring kernel's addressing, for CPU tests.
//
// Test infrastructure: packs a model with the library's own packer (pack.cpp) and walks every
// tile image of one tiling the way the kernel does -- LDS byte layout, feature addresses built
// by OR-ing the column offset with the lane offset, child links as absolute LDS record
// indices, the all-zero self-linked record for padding slots -- checking that every LDS
// access stays inside the region it must read. The tests compare the leaf ids it reports with
// the oracle's, so a packing or addressing mistake shows up on the CPU before any GPU run.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <functional>
#include <string>
#include <vector>

#include "pack.hpp"

namespace {

std::string g_msg;

int bad(const std::string &m) {
    g_msg = m;
    return 1;
}

float as_float(uint32_t u) {
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// code_f(x) = number of distinct thresholds t of f with x >= t (0 for NaN)
uint16_t code_of(const treeens::Packed &p, int f, float x) {
    const float *b = p.code_table.data() + p.code_table_off[size_t(f)];
    const float *e = p.code_table.data() + p.code_table_off[size_t(f) + 1];
    uint16_t c = 0;
    for (const float *t = b; t < e; ++t)
        if (x >= *t)
            ++c;
    return c;
}

// code_f(x) by the coding kernel's descent over its chunk's search table: s steps of
// i = 2i + (x >= slot i) from i = 1, code = i - 2^s. Returns -1 when the chunk layout cannot
// hold feature f's search (sizes, slot count, the LDS table).
int32_t code_by_descent(const treeens::Packed &p, int f, float x) {
    for (const treeens::CodeChunk &ch : p.code_chunks) {
        if (f < ch.f_begin || f >= ch.f_end)
            continue;
        const uint32_t len = p.code_table_off[size_t(f) + 1] - p.code_table_off[size_t(f)];
        const int s = ch.search_steps;
        if (s < 0 || s > 14 || (uint64_t(1) << s) - 1 < len || ch.f_end - ch.f_begin > treeens::kCodeChunkFeatures ||
            int64_t(ch.table_end - ch.table_begin) != int64_t(ch.f_end - ch.f_begin) * ((int64_t(1) << s) - 1) ||
            ch.table_end - ch.table_begin > treeens::kCodeTableFloats || ch.table_begin < 0 ||
            size_t(ch.table_end) > p.code_search.size())
            return -1;
        // entry i - 1 of feature f's 2^s - 1 entries holds slot i
        const size_t t0 = size_t(ch.table_begin) + size_t(f - ch.f_begin) * ((size_t(1) << s) - 1);
        uint32_t i = 1;
        for (int k = 0; k < s; ++k)
            i = 2u * i + (x >= p.code_search[t0 + i - 1] ? 1u : 0u);
        return int32_t(i - (1u << s));
    }
    return -1;
}

} // namespace

extern "C" {

const char *emu_message(void) { return g_msg.c_str(); }

// Walk all documents through tiling `level`. Outputs leaf ids [n_docs][n_trees] (input node ids)
// and fp64 scores [n_docs][n_outputs] (vector-valued leaves read through the leaf-vector table).
// plan_out (10 ints): docs per block, trees per lane, record format, coded, tiles at tiling 0,
// LDS bytes, tile slot bytes, records of the largest tiling-0 image, walker sub-slot records
// (0: shared tiles), tiled trees (the rest are big trees walked from device memory). Returns 0, or 1 with a message naming the first violated
// invariant, or a negative packer status.
int emu_walk(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
             const float *threshold, const int32_t *left, const int32_t *right, const float *value,
             int32_t n_outputs, uint32_t flags, const float *X, int64_t n_docs, int32_t n_features,
             int32_t level, int32_t *leaf_ids, double *scores, int32_t *plan_out) {
    treeens::Packed p;
    std::string err;
    const int rc = treeens::pack_model(n_trees, tree_offsets, feature, threshold, left, right, value,
                                       n_outputs, flags, p, err);
    if (rc != treeens::kOk) {
        g_msg = err;
        return rc;
    }
    const treeens::LdsPlan &pl = p.plan;
    if (plan_out) {
        plan_out[0] = pl.docs_per_block;
        plan_out[1] = pl.interleave;
        plan_out[2] = pl.narrow;
        plan_out[3] = pl.coded;
        plan_out[4] = p.level_begin[1] - p.level_begin[0];
        plan_out[5] = pl.lds_bytes;
        plan_out[6] = pl.tile_bytes;
        plan_out[7] = p.level_slot_recs[0];
        plan_out[8] = p.pk_recs;
        plan_out[9] = p.n_small;
    }
    const int DL = pl.docs_per_block, K = pl.interleave, E = pl.elem_bytes;
    const int shift = pl.narrow ? 16 : treeens::kWideChildShift;
    const uint32_t mask = pl.narrow ? treeens::kNarrowColMask : treeens::kWideColMask;
    const uint32_t xs = uint32_t(pl.xs_bytes), zero = uint32_t(pl.zero_rec);
    const uint32_t leaf_col = uint32_t(DL * E);
    if (xs % 16 || zero % 8 || zero + 8 > uint32_t(pl.lds_bytes) || xs + uint32_t(pl.tile_bytes) > zero)
        return bad("LDS plan regions overlap or exceed the workgroup's LDS");
    if (int64_t(p.n_cols + 1) * DL * E != pl.xs_bytes)
        return bad("document tile size does not match the column count");
    {
        // the feature-access trace's bitmasks: after the zero record, within the LDS the usage
        // launch declares (two-workgroup plans: past their half, plus kUsageHalfBytes)
        const int64_t usage_end = int64_t(pl.usage_off) + int64_t(p.n_cols + 31) / 32 * DL * 4;
        const int64_t lds_end = pl.lds_bytes == treeens::kLdsPerCu
                                    ? treeens::kLdsPerCu
                                    : treeens::kLdsPerCu / 2 + treeens::kUsageHalfBytes;
        if (pl.usage_off % 16 || pl.usage_off < int64_t(zero) + 8 || usage_end > lds_end)
            return bad("feature bitmask region overlaps the tile or exceeds the LDS");
        // the in-slot placement of two-workgroup plans: past every tiling-0 image, before the
        // zero record
        if (p.usage_slot_off >= 0) {
            const int64_t mask_bytes = int64_t(p.n_cols + 31) / 32 * DL * 4;
            // with walker packets the bitmasks follow the sub-slots, else the tiling-0 images
            const int64_t used = p.pk_recs > 0 ? int64_t(treeens::kPacketWalkers) * p.pk_recs
                                               : int64_t(p.level_slot_recs[0]);
            if (pl.lds_bytes != treeens::kLdsPerCu / 2 || p.usage_slot_off % 16 ||
                p.usage_slot_off < int64_t(xs) + used * 8 || p.usage_slot_off + mask_bytes > int64_t(zero))
                return bad("in-slot feature bitmasks overlap a tile image or the zero record");
            if (p.pk_recs == 0)
                for (int32_t t = p.level_begin[0]; t < p.level_begin[1]; t++)
                    if (int64_t(xs) + int64_t(p.tile_recs[size_t(t)]) * 8 > p.usage_slot_off)
                        return bad("a tiling-0 image reaches the in-slot feature bitmasks");
        }
    }
    std::vector<uint8_t> lds(size_t(pl.lds_bytes), 0);
    auto rec_at = [&](uint32_t a) {
        treeens::NodeRec r;
        std::memcpy(&r, lds.data() + a, 8);
        return r;
    };
    const int32_t t0 = p.level_begin[level], t1 = p.level_begin[level + 1];
    const int64_t slot = p.level_slot_recs[level];
    if (slot * 8 > pl.tile_bytes)
        return bad("image stride exceeds the LDS slot");
    // prefetch capacity: one tile in 6 records per thread with two workgroups per CU; windows
    // of whole 1,024-record chunks, at most 8 per tile, with one
    if (pl.lds_bytes == treeens::kLdsPerCu) {
        const int64_t chunks = (slot + 1023) / 1024;
        // the kernel writes whole chunks: they must fit the prefetch registers and the slot
        if (chunks > treeens::kPrefetchFull / 2 || chunks * 1024 * 8 > pl.tile_bytes)
            return bad("tile window exceeds the registers or the LDS slot");
        const int64_t last = p.level_image_off[level] + int64_t(t1 - t0 - 1) * slot;
        if (t1 > t0 && last + chunks * 1024 > int64_t(p.images.size()))
            return bad("the last tile's window reads past the images");
    } else if (slot > int64_t(treeens::kPrefetchHalf) * 1024) {
        return bad("tile image exceeds the prefetch registers");
    }
    if (p.pk_recs > 0) {
        // walker packets: whole 64-lane loads that fit the prefetch registers, one packet stream
        // per walker; two-workgroup plans: sub-slots inside the tile slot, before the plan's zero
        // record; one-workgroup plans: sub-slots up to the packets' own zero record
        const bool half = pl.lds_bytes == treeens::kLdsPerCu / 2;
        const int64_t sub_end = int64_t(xs) + int64_t(treeens::kPacketWalkers) * p.pk_recs * 8;
        if ((DL != 64 && DL != 32) || p.pk_recs % 64 ||
            p.pk_recs / 64 > (half ? treeens::kPrefetchHalf : treeens::kPrefetchFull) ||
            (half ? (p.pk_zero_rec != int32_t(zero) || sub_end > int64_t(xs) + pl.tile_bytes)
                  : (p.pk_zero_rec % 8 || sub_end > p.pk_zero_rec ||
                     int64_t(p.pk_zero_rec) + 8 > pl.lds_bytes)))
            return bad("walker sub-slots do not fit the plan");
        if (p.packets.size() != size_t(treeens::kPacketWalkers) * size_t(p.pk_per_walker) * size_t(p.pk_recs))
            return bad("packet buffer has the wrong size");
    }
    std::vector<int32_t> seen(size_t(n_trees), 0);
    for (int64_t i = 0; i < n_docs * n_trees; i++)
        leaf_ids[i] = -1;
    const bool vec = n_outputs > 1;
    if (vec && (p.vec_stride < n_outputs || p.vec_stride % 4 ||
                p.leaf_vec.size() != size_t(p.nodes.size() + 1) * size_t(p.vec_stride)))
        return bad("leaf-vector table has the wrong shape");
    for (int64_t d = 0; d < n_docs * n_outputs; d++)
        scores[d] = 0.0;

    for (int64_t doc0 = 0; doc0 < n_docs; doc0 += DL) {
        // document tile: column 0 NaN (or code 0), column f + 1 = feature f, lane = document
        for (int c = 0; c <= p.n_cols; c++) {
            for (int dl = 0; dl < DL; dl++) {
                const int64_t doc = doc0 + dl;
                uint8_t *dst = lds.data() + (size_t(c) * DL + dl) * E;
                if (E == 4) {
                    float v = c == 0 ? NAN : (doc < n_docs ? X[doc * n_features + c - 1] : 0.0f);
                    std::memcpy(dst, &v, 4);
                } else {
                    uint16_t v = c == 0 || doc >= n_docs ? 0 : code_of(p, c - 1, X[doc * n_features + c - 1]);
                    if (c > 0 && doc < n_docs &&
                        code_by_descent(p, c - 1, X[doc * n_features + c - 1]) != int32_t(v))
                        return bad("the coding kernel's descent disagrees with the threshold count");
                    std::memcpy(dst, &v, 2);
                }
            }
        }
        const treeens::NodeRec z{treeens::zero_record_value(pl, vec), (zero / 8u) << shift};
        std::memcpy(lds.data() + zero, &z, 8);

        // Walk every document of the block through packed tree gt whose root copy is at
        // root_copy (LDS byte address) and whose first record is LDS record root_idx.
        auto walk_tree = [&](int gt, uint32_t root_copy, uint32_t root_idx, int complete,
                             const std::function<bool(uint32_t)> &valid) -> int {
            const int64_t tree_n = int64_t(p.tree_node_off[size_t(gt) + 1] - p.tree_node_off[size_t(gt)]);
            for (int dl = 0; dl < DL && doc0 + dl < n_docs; dl++) {
                const int64_t doc = doc0 + dl;
                treeens::NodeRec r = rec_at(root_copy);
                int steps = 0;
                uint32_t last = root_idx * 8u; // LDS byte address of the record r came from
                for (;;) {
                    // complete trees: a fixed number of steps (their leaf records hold a double)
                    if (complete >= 0 && steps == complete)
                        break;
                    const uint32_t fa = (r.w & mask) | uint32_t(dl * E);
                    if (fa != (r.w & mask) + uint32_t(dl * E))
                        return bad("column offset and lane offset overlap");
                    if (fa + uint32_t(E) > xs)
                        return bad("feature address outside the document tile");
                    if (complete < 0 && fa < leaf_col)
                        break;
                    bool right_side;
                    if (E == 4) {
                        float x;
                        std::memcpy(&x, lds.data() + fa, 4);
                        right_side = x >= as_float(r.thr_bits);
                    } else {
                        uint16_t x;
                        std::memcpy(&x, lds.data() + fa, 2);
                        right_side = uint32_t(x) >= r.thr_bits;
                    }
                    const uint32_t a = ((r.w >> shift) + (right_side ? 1u : 0u)) * 8u;
                    if (!valid(a))
                        return bad("child address outside the tile's records");
                    r = rec_at(a);
                    last = a;
                    if (++steps > p.max_depth + 1)
                        return bad("walk longer than the deepest tree");
                }
                if (complete >= 0) {
                    // the record reached must be a leaf of the tree, stored as its value in double
                    const int64_t self = int64_t(last / 8u) - int64_t(root_idx);
                    if (self < 0 || self >= tree_n)
                        return bad("complete walk ended outside its tree");
                    const treeens::NodeRec orig = p.nodes[p.tree_node_off[size_t(gt)] + size_t(self)];
                    const bool vec_model = n_outputs > 1;
                    if ((orig.w & mask) != 0)
                        return bad("complete walk ended on an internal node");
                    if (!vec_model) {
                        const double want = double(as_float(orig.thr_bits));
                        double got;
                        std::memcpy(&got, &r, 8);
                        if (std::memcmp(&got, &want, 8) != 0)
                            return bad("complete tree's leaf record does not hold its value as a double");
                        leaf_ids[doc * n_trees + p.tree_orig[size_t(gt)]] =
                            p.orig_id[p.tree_node_off[size_t(gt)] + size_t(self)];
                        scores[doc] += got;
                        continue;
                    }
                }
                if ((r.w & mask) != 0)
                    return bad("walk ended on an internal node");
                {
                    // one more step from a leaf must come back to the same record
                    bool right_side;
                    if (E == 4) {
                        float x;
                        std::memcpy(&x, lds.data() + (r.w & mask) + dl * E, 4);
                        right_side = x >= as_float(r.thr_bits);
                    } else {
                        uint16_t x;
                        std::memcpy(&x, lds.data() + (r.w & mask) + dl * E, 2);
                        right_side = uint32_t(x) >= r.thr_bits;
                    }
                    const uint32_t a = ((r.w >> shift) + (right_side ? 1u : 0u)) * 8u;
                    if (!valid(a) || std::memcmp(lds.data() + a, &r, 8) != 0)
                        return bad("a leaf does not absorb a further step");
                }
                const int64_t self = int64_t(r.w >> shift) - int64_t(root_idx);
                if (self < 0 || self >= tree_n)
                    return bad("leaf outside its tree");
                const int32_t orig_tree = p.tree_orig[size_t(gt)];
                leaf_ids[doc * n_trees + orig_tree] = p.orig_id[p.tree_node_off[size_t(gt)] + size_t(self)];
                if (vec) {
                    const int64_t row = int64_t(r.thr_bits) - 1;
                    if (row < 1 || row > int64_t(p.nodes.size()))
                        return bad("leaf names a row outside the leaf-vector table");
                    for (int c = 0; c < n_outputs; c++)
                        scores[doc * n_outputs + c] +=
                            double(p.leaf_vec[size_t(row) * size_t(p.vec_stride) + size_t(c)]);
                } else {
                    scores[doc] += double(as_float(r.thr_bits));
                }
            }
            seen[size_t(p.tree_orig[size_t(gt)])]++;
            return 0;
        };

        // big trees: records read from the packed array in the big-tree format (tree-relative
        // links, column indices), features from the LDS document tile
        for (int32_t gt = p.n_small; gt < n_trees; gt++) {
            const uint32_t first = p.tree_node_off[size_t(gt)];
            const int64_t tree_n = int64_t(p.tree_node_off[size_t(gt) + 1]) - int64_t(first);
            for (int dl = 0; dl < DL && doc0 + dl < n_docs; dl++) {
                const int64_t doc = doc0 + dl;
                int64_t cur = 0;
                int steps = 0;
                auto step = [&](int64_t at, bool *internal) -> int64_t {
                    const treeens::NodeRec r = p.nodes[size_t(first) + size_t(at)];
                    const uint32_t col = r.w & treeens::kBigColMask;
                    if (col > uint32_t(p.n_cols))
                        return -2;
                    const uint32_t fa = col * uint32_t(DL * E) + uint32_t(dl * E);
                    *internal = fa >= leaf_col;
                    bool right_side;
                    if (E == 4) {
                        float x;
                        std::memcpy(&x, lds.data() + fa, 4);
                        right_side = x >= as_float(r.thr_bits);
                    } else {
                        uint16_t x;
                        std::memcpy(&x, lds.data() + fa, 2);
                        right_side = uint32_t(x) >= r.thr_bits;
                    }
                    return int64_t(r.w >> treeens::kBigLinkShift) + (right_side ? 1 : 0);
                };
                for (;;) {
                    bool internal = false;
                    const int64_t nxt = step(cur, &internal);
                    if (nxt == -2)
                        return bad("big tree: column index beyond the document tile");
                    if (!internal) {
                        if (nxt != cur)
                            return bad("big tree: a leaf does not absorb a further step");
                        break;
                    }
                    if (nxt < 0 || nxt >= tree_n)
                        return bad("big tree: child outside the tree's records");
                    cur = nxt;
                    if (++steps > p.max_depth + 1)
                        return bad("big tree: walk longer than the deepest tree");
                }
                const treeens::NodeRec r = p.nodes[size_t(first) + size_t(cur)];
                leaf_ids[doc * n_trees + p.tree_orig[size_t(gt)]] = p.orig_id[size_t(first) + size_t(cur)];
                if (vec) {
                    const int64_t row = int64_t(r.thr_bits) - 1;
                    if (row < 1 || row > int64_t(p.nodes.size()))
                        return bad("big tree: leaf names a row outside the leaf-vector table");
                    for (int c = 0; c < n_outputs; c++)
                        scores[doc * n_outputs + c] +=
                            double(p.leaf_vec[size_t(row) * size_t(p.vec_stride) + size_t(c)]);
                } else {
                    scores[doc] += double(as_float(r.thr_bits));
                }
            }
            seen[size_t(p.tree_orig[size_t(gt)])]++;
        }

        if (p.pk_recs > 0) {
            // each walker copies its packets, in order, into its own sub-slot and walks them;
            // padding links to the packets' zero record (the plan's own in two-workgroup plans)
            constexpr int32_t W = treeens::kPacketWalkers;
            const int32_t sub = p.pk_recs, per = p.pk_per_walker;
            const uint32_t pzero = uint32_t(p.pk_zero_rec);
            const treeens::NodeRec zp{treeens::zero_record_value(pl, vec), (pzero / 8u) << shift};
            std::memcpy(lds.data() + pzero, &zp, 8);
            // P walkers per wave (two half-waves for 32-document blocks), each with its own part
            const int32_t P = 64 / DL, HW = W * P, part = sub / P;
            if (sub % P || part % 2)
                return bad("packet parts are not whole, 16-byte aligned halves");
            for (int32_t w = 0; w < W; w++) {
                for (int32_t q = 0; q < per; q++) {
                    const treeens::NodeRec *img = p.packets.data() + (size_t(w) * size_t(per) + size_t(q)) * size_t(sub);
                    std::memcpy(lds.data() + xs + uint32_t(w * sub) * 8u, img, size_t(sub) * 8);
                    const treeens::NodeRec c0 = rec_at(xs + uint32_t(w * sub) * 8u);
                    for (int32_t h = 0; h < P; h++) {
                        const uint32_t lo_b = xs + uint32_t(w * sub + h * part) * 8u, hi_b = lo_b + uint32_t(part) * 8u;
                        const treeens::NodeRec h0 = rec_at(lo_b), h1 = rec_at(lo_b + 8);
                        const int ng = int(h0.thr_bits), complete = int32_t(h0.w), g0 = int(h1.thr_bits);
                        // the kernel takes the group count and complete depth from any lane
                        if (h0.thr_bits != c0.thr_bits || h0.w != c0.w)
                            return bad("packet parts disagree on the group count or complete depth");
                        if (ng == 0)
                            continue;
                        const int table = treeens::kPacketHeaderRecs + ng * K;
                        const int rec_begin = table + (ng * K + 3) / 4;
                        if (ng < 0 || rec_begin > part)
                            return bad("packet header out of range");
                        const uint32_t rec_lo = lo_b + uint32_t(rec_begin) * 8u;
                        auto valid = [&](uint32_t a) { return a % 8 == 0 && ((a >= rec_lo && a + 8 <= hi_b) || a == pzero); };
                        for (int j = 0; j < ng; j++) {
                            const int g = g0 + j * HW;
                            if (g % HW != w * P + h)
                                return bad("a packet holds a group of another walker");
                            for (int i = 0; i < K; i++) {
                                const int gt = g * K + i;
                                const uint32_t root_copy = lo_b + 8u * uint32_t(treeens::kPacketHeaderRecs + j * K + i);
                                // the kernel reads two roots per 16-byte read when K is even
                                if (K % 2 == 0 && i % 2 == 0 && root_copy % 16 != 0)
                                    return bad("packet: a pair of root copies is not 16-byte aligned");
                                if (gt >= p.n_small) {
                                    if (complete >= 0)
                                        return bad("packet: a complete packet has an idle slot");
                                    if (std::memcmp(lds.data() + root_copy, lds.data() + pzero, 8) != 0)
                                        return bad("packet: padding root is not the zero record");
                                    continue;
                                }
                                uint16_t first_rec;
                                std::memcpy(&first_rec, lds.data() + lo_b + uint32_t(table) * 8u + 2u * uint32_t(j * K + i), 2);
                                const uint32_t root_idx = first_rec;
                                if (!valid(root_idx * 8u) ||
                                    std::memcmp(lds.data() + root_idx * 8u, lds.data() + root_copy, 8) != 0)
                                    return bad("packet: root copy does not match the tree's root record");
                                if (const int e = walk_tree(gt, root_copy, root_idx, complete, valid))
                                    return e;
                            }
                        }
                    }
                }
            }
            continue;
        }
        for (int32_t t = t0; t < t1; t++) {
            const uint32_t recs = p.tile_recs[size_t(t)];
            if (recs > uint32_t(slot))
                return bad("tile image longer than its stride");
            const treeens::NodeRec *img = p.images.data() + p.level_image_off[level] + (t - t0) * slot;
            std::memcpy(lds.data() + xs, img, size_t(recs) * 8);
            uint32_t h[4];
            std::memcpy(h, lds.data() + xs, 16);
            const int ntr = int(h[0]), complete = int32_t(h[1]), tb = int(h[2]);
            const uint32_t next = h[3];
            if (next != (t + 1 < t1 ? p.tile_recs[size_t(t) + 1] : 0u))
                return bad("header: next tile size is wrong");
            if (ntr < 1 || tb < 0 || tb + ntr > n_trees)
                return bad("header: tree range out of bounds");
            const int padded = (ntr + K - 1) / K * K;
            const uint32_t hdr_bytes = uint32_t(treeens::kHeaderFixedWords / 2 + padded) * 8u;
            const uint32_t lo = xs + hdr_bytes, hi = xs + recs * 8u;
            auto valid = [&](uint32_t a) { return a % 8 == 0 && ((a >= lo && a + 8 <= hi) || a == zero); };
            // root copies: records 2.. of the header; padding slots hold the zero record
            const uint32_t root0 = xs + 8u * uint32_t(treeens::kHeaderFixedWords / 2);
            // the kernel reads two roots per 16-byte read when K is even
            if (K % 2 == 0 && root0 % 16 != 0)
                return bad("header: the root copies are not 16-byte aligned");
            for (int s = ntr; s < padded; s++)
                if (std::memcmp(lds.data() + root0 + 8u * s, lds.data() + zero, 8) != 0)
                    return bad("header: padding root is not the zero record");
            if (complete >= 0 && padded != ntr)
                return bad("header: a complete tile has an idle slot");
            const uint32_t rec0 = xs / 8u + hdr_bytes / 8u; // LDS index of the first tree record
            for (int s = 0; s < ntr; s++) {
                const int gt = tb + s;
                const uint32_t root_idx = rec0 + p.tree_node_off[size_t(gt)] - p.tree_node_off[size_t(tb)];
                if (!valid(root_idx * 8u) || std::memcmp(lds.data() + root_idx * 8u, lds.data() + root0 + 8u * s, 8) != 0)
                    return bad("root copy does not match the tree's root record");
                if (const int e = walk_tree(gt, root0 + 8u * s, root_idx, complete, valid))
                    return e;
            }
        }
    }
    const int64_t blocks = (n_docs + DL - 1) / DL;
    for (int32_t t = 0; t < n_trees; t++)
        if (seen[size_t(t)] != blocks)
            return bad("tree " + std::to_string(t) + " is not walked exactly once per block");
    return 0;
}

// Walk all documents through the compact packets (4-byte records, pair reads, leaf payloads in
// their own arrays) the way the kernel addresses them: documents staged as code << 5 | 31,
// per wave K windows of 4096 / K bytes after the document tile (aligned to their size), each
// packet's header read from its image (the kernel keeps it in registers: header words 2l and
// 2l + 1 in lane l, so every word it reads must lie in the 64 lanes' 512 bytes). Every feature read must stay in the document tile and every pair
// read in the window of its slot. Outputs as emu_walk; returns 2 when the model has no compact
// packets, else 0 or 1 with a message, or a negative packer status. k_out[0]: trees per lane,
// k_out[1]: groups in the fullest packet.
int emu_walk_compact(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                     const float *threshold, const int32_t *left, const int32_t *right,
                     const float *value, int32_t n_outputs, uint32_t flags, const float *X,
                     int64_t n_docs, int32_t n_features, int32_t *leaf_ids, double *scores,
                     int32_t *k_out) {
    treeens::Packed p;
    std::string err;
    const int rc = treeens::pack_model(n_trees, tree_offsets, feature, threshold, left, right, value,
                                       n_outputs, flags, p, err);
    if (rc != treeens::kOk) {
        g_msg = err;
        return rc;
    }
    if (k_out) {
        k_out[0] = p.cp_k;
        k_out[1] = p.cp_max_groups;
    }
    if (p.cp_k == 0) {
        g_msg = "no compact packets";
        return 2;
    }
    const treeens::LdsPlan &pl = p.plan;
    constexpr int32_t W = treeens::kPacketWalkers;
    constexpr int32_t kWords = treeens::kCompactPacketBytes / 4;
    const int DL = pl.docs_per_block, K = p.cp_k;
    if (DL != 64 || !pl.coded || pl.elem_bytes != 2 || (K != 2 && K != 4) || p.n_small != n_trees)
        return bad("compact packets on a plan they do not support");
    const uint32_t xs = uint32_t(pl.xs_bytes);
    const uint32_t cw = uint32_t(treeens::compact_window_base(pl.xs_bytes));
    const uint32_t win = uint32_t(treeens::kCompactWindowBytes / K);
    if (cw % win || cw + uint32_t(W) * treeens::kCompactWindowBytes > uint32_t(treeens::kLdsPerCu))
        return bad("compact windows do not fit the LDS");
    if (treeens::kCompactHeaderBytes != 64 * 8)
        return bad("compact header is not one 8-byte row of 64 lanes");
    const size_t total = size_t(W) * size_t(p.cp_per_walker) * size_t(kWords);
    if (p.cp_packets.size() != total || p.cp_leaf.size() != total || p.cp_leaf_id.size() != total)
        return bad("compact packet arrays have the wrong size");
    std::vector<uint8_t> lds(size_t(treeens::kLdsPerCu), 0);
    auto u32_at = [&](uint32_t a) {
        uint32_t v;
        std::memcpy(&v, lds.data() + a, 4);
        return v;
    };
    const bool vec = n_outputs > 1;
    std::vector<int32_t> seen(size_t(n_trees), 0);
    for (int64_t i = 0; i < n_docs * n_trees; i++)
        leaf_ids[i] = -1;
    for (int64_t d = 0; d < n_docs * n_outputs; d++)
        scores[d] = 0.0;
    for (int64_t doc0 = 0; doc0 < n_docs; doc0 += DL) {
        for (int c = 0; c <= p.n_cols; c++) {
            for (int dl = 0; dl < DL; dl++) {
                const int64_t doc = doc0 + dl;
                const uint32_t code = c == 0 || doc >= n_docs ? 0u : code_of(p, c - 1, X[doc * n_features + c - 1]);
                if (code >= treeens::kCompactNeverRight)
                    return bad("a code reaches the never-right threshold");
                const uint16_t v = uint16_t((code << treeens::kCompactCodeShift) | 31u);
                std::memcpy(lds.data() + (size_t(c) * DL + dl) * 2, &v, 2);
            }
        }
        for (int32_t v = 0; v < W; v++) {
            for (int32_t q = 0; q < p.cp_per_walker; q++) {
                const size_t at = (size_t(v) * size_t(p.cp_per_walker) + size_t(q)) * size_t(kWords);
                const uint32_t my_win = cw + uint32_t(v) * treeens::kCompactWindowBytes;
                std::memcpy(lds.data() + my_win, p.cp_packets.data() + at, treeens::kCompactWindowBytes);
                const uint32_t *hdr = p.cp_packets.data() + at + treeens::kCompactWindowBytes / 4;
                const int ng = int(hdr[0]), complete = int32_t(hdr[1]);
                const int g0 = int(hdr[2]);
                if (ng < 0 || treeens::kCompactHeaderWords + ng * K > treeens::kCompactHeaderBytes / 4)
                    return bad("compact header out of range");
                for (int j = 0; j < ng; j++) {
                    const int g = g0 + j * W;
                    if (g % W != v)
                        return bad("a compact packet holds a group of another wave");
                    // group j's K = 2 roots: header words 4 + 2j, 5 + 2j, i.e. lane 2 + j's pair
                    const uint32_t root_word = uint32_t(treeens::kCompactHeaderWords + j * K);
                    if (root_word % 2 != 0 || root_word / 2 != uint32_t(2 + j) || root_word / 2 > 63)
                        return bad("a group's roots are not one lane's word pair of the header row");
                    for (int i = 0; i < K; i++) {
                        const int gt = g * K + i;
                        const uint32_t tb = my_win + uint32_t(i) * win;
                        if (gt >= n_trees && complete >= 0)
                            return bad("compact: a complete packet has an idle slot");
                        for (int dl = 0; dl < DL && doc0 + dl < n_docs; dl++) {
                            const int64_t doc = doc0 + dl;
                            uint32_t r = hdr[root_word + uint32_t(i)];
                            int steps = 0;
                            auto step = [&](uint32_t cur, uint32_t *next) -> int {
                                const uint32_t fa = ((cur >> 4) & 0x1FF80u) | uint32_t(dl * 2);
                                if (fa + 2 > xs)
                                    return bad("compact: feature address outside the document tile");
                                const uint32_t pa = (cur & 0x7F8u) | tb;
                                if (pa != (cur & 0x7F8u) + tb || pa < tb || pa + 8 > tb + win)
                                    return bad("compact: pair read outside the slot's window");
                                uint16_t x;
                                std::memcpy(&x, lds.data() + fa, 2);
                                const bool right_side = uint32_t(x) >= (cur >> 16);
                                *next = u32_at(pa + (right_side ? 4u : 0u));
                                return 0;
                            };
                            for (;;) {
                                if (complete >= 0 ? steps == complete : ((r >> 4) & 0x1FF80u) == 0u)
                                    break;
                                uint32_t nxt;
                                if (const int e = step(r, &nxt))
                                    return e;
                                r = nxt;
                                if (++steps > p.max_depth + 1)
                                    return bad("compact: walk longer than the deepest tree");
                            }
                            if (((r >> 4) & 0x1FF80u) != 0u)
                                return bad("compact: walk ended on an internal node");
                            uint32_t again;
                            if (const int e = step(r, &again))
                                return e;
                            if (again != r)
                                return bad("compact: a leaf does not absorb a further step");
                            const size_t w = at + size_t((r & 0x7FCu) + uint32_t(i) * win) / 4;
                            if (gt >= n_trees) {
                                if (p.cp_leaf[w] != (vec ? 1u : 0u))
                                    return bad("compact: an idle slot's payload is not zero");
                                continue;
                            }
                            const int32_t id = p.cp_leaf_id[w];
                            const int32_t orig_tree = p.tree_orig[size_t(gt)];
                            const int64_t tn = tree_offsets[orig_tree + 1] - tree_offsets[orig_tree];
                            if (id < 0 || id >= tn || feature[tree_offsets[orig_tree] + id] >= 0)
                                return bad("compact: the payload's node id is not a leaf of the tree");
                            leaf_ids[doc * n_trees + orig_tree] = id;
                            if (vec) {
                                const int64_t row = int64_t(p.cp_leaf[w]) - 1;
                                if (row < 1 || row > int64_t(p.nodes.size()))
                                    return bad("compact: leaf names a row outside the leaf-vector table");
                                for (int c = 0; c < n_outputs; c++)
                                    scores[doc * n_outputs + c] +=
                                        double(p.leaf_vec[size_t(row) * size_t(p.vec_stride) + size_t(c)]);
                            } else {
                                scores[doc] += double(as_float(p.cp_leaf[w]));
                            }
                        }
                        if (gt < n_trees)
                            seen[size_t(p.tree_orig[size_t(gt)])]++;
                    }
                }
            }
        }
    }
    const int64_t blocks = (n_docs + DL - 1) / DL;
    for (int32_t t = 0; t < n_trees; t++)
        if (seen[size_t(t)] != blocks)
            return bad("compact: tree " + std::to_string(t) + " is not walked exactly once per block");
    return 0;
}

// Every coded feature's search table against a plain count: at each of its thresholds, just
// below each, at +-inf, +-0 and NaN, the descent must give |{t : x >= t}|. Returns 2 when the
// model is not coded, else 0 or 1 with a message.
int emu_code_check(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                   const float *threshold, const int32_t *left, const int32_t *right,
                   const float *value, uint32_t flags, int64_t *checked) {
    treeens::Packed p;
    std::string err;
    const int rc = treeens::pack_model(n_trees, tree_offsets, feature, threshold, left, right, value, 1,
                                       flags, p, err);
    if (rc != treeens::kOk) {
        g_msg = err;
        return rc;
    }
    if (!p.plan.coded) {
        g_msg = "model is not coded";
        return 2;
    }
    int64_t n = 0;
    for (int f = 0; f < p.n_cols; f++) {
        std::vector<float> xs = {INFINITY, -INFINITY, 0.0f, -0.0f, NAN};
        for (uint32_t k = p.code_table_off[size_t(f)]; k < p.code_table_off[size_t(f) + 1]; k++) {
            xs.push_back(p.code_table[k]);
            xs.push_back(std::nextafter(p.code_table[k], -INFINITY));
        }
        for (float x : xs) {
            const int32_t got = code_by_descent(p, f, x);
            if (got < 0)
                return bad("feature " + std::to_string(f) + ": the coding chunks do not hold its search");
            if (got != int32_t(code_of(p, f, x)))
                return bad("feature " + std::to_string(f) + ": the search gives " + std::to_string(got) +
                           " where the count is " + std::to_string(code_of(p, f, x)));
            n++;
        }
    }
    if (checked)
        *checked = n;
    return 0;
}

// The packer's tree order (order[i] = input index of the i-th packed tree) and, per tile of
// tiling 0, its complete depth (-1: not all trees complete of one depth). Returns the number
// of tiles (at most max_tiles are written), or a negative packer status.
int emu_tree_order(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                   const float *threshold, const int32_t *left, const int32_t *right, const float *value,
                   uint32_t flags, int32_t *order, int32_t *tile_complete, int32_t max_tiles) {
    treeens::Packed p;
    std::string err;
    const int rc = treeens::pack_model(n_trees, tree_offsets, feature, threshold, left, right, value, 1,
                                       flags, p, err);
    if (rc != treeens::kOk) {
        g_msg = err;
        return rc;
    }
    for (int32_t t = 0; t < n_trees; t++)
        order[t] = p.tree_orig[size_t(t)];
    const int32_t n_tiles = p.level_begin[1] - p.level_begin[0];
    for (int32_t i = 0; i < n_tiles && i < max_tiles; i++)
        tile_complete[i] = p.tiles[size_t(p.level_begin[0] + i)].complete_depth;
    return n_tiles;
}

} // extern "C"
