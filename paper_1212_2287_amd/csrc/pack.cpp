// pack.cpp -- validation, breadth-first re-layout and LDS tile planning (host only).
#include "pack.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>

namespace treeens {

namespace {

uint32_t float_bits(float f) {
    uint32_t u;
    std::memcpy(&u, &f, sizeof u);
    return u;
}

// Under the strict rule (right iff x > theta) store the next float above theta: no float lies
// strictly between theta and its successor, so x > theta <=> x >= successor for every non-NaN
// x. +inf has no successor; x > +inf never holds, which a NaN threshold reproduces under >=.
float strict_to_inclusive(float theta) {
    if (std::isinf(theta) && theta > 0)
        return std::nanf("");
    return std::nextafter(theta, INFINITY);
}

// A tree of n nodes whose longest root-to-leaf path has d edges is complete (every leaf at depth
// d) exactly when n = 2^(d+1) - 1. Deep trees (d up to the node count) never are, and the shift
// must not overflow.
bool is_complete(int64_t n, int64_t d) { return d < 62 && n == (int64_t(2) << d) - 1; }

// Leaf records of tiles and packets whose trees are all complete of one depth: the walk there
// takes a fixed number of steps and never tests a leaf, so a leaf record needs neither its
// column nor its link and holds the leaf value as a double (the 8 bytes of the record), which
// the kernel adds to its fp64 sum without a conversion. Internal records are unchanged.
NodeRec complete_leaf(NodeRec r, uint32_t col_mask) {
    if ((r.w & col_mask) != 0)
        return r; // internal node (its column offset is never 0)
    float v;
    std::memcpy(&v, &r.thr_bits, 4);
    const double d = double(v);
    uint64_t b;
    std::memcpy(&b, &d, 8);
    return NodeRec{uint32_t(b), uint32_t(b >> 32)};
}

// avg_tree_bytes: mean packed size of a tree, to pick how many trees a lane walks at once.
// elem_bytes: 4 for float features, 2 for codes.
LdsPlan plan_lds(int32_t n_cols, double avg_tree_bytes, int elem_bytes) {
    LdsPlan p{};
    p.elem_bytes = elem_bytes;
    p.coded = elem_bytes == 2;
    const int64_t cols = int64_t(n_cols) + 1; // + the NaN (or zero-code) column the leaves read
    for (int dl = 64; dl >= 8; dl /= 2) {
        if (cols * dl * elem_bytes <= kXsMaxBytes) {
            p.docs_per_block = dl;
            break;
        }
    }
    if (p.docs_per_block == 0)
        return p;
    p.xs_bytes = int32_t(cols * p.docs_per_block * elem_bytes);
    const int reserve = 64; // the all-zero record, slack
    // 16 waves per workgroup; two workgroups per CU when the document tile is small
    p.wg_threads = 1024;
    p.lds_bytes = (p.xs_bytes <= kTwoWgXsBytes && !p.coded) ? kLdsPerCu / 2 : kLdsPerCu;
    // records per thread a tile may take in the registers that prefetch it: all of the
    // prefetch registers with two workgroups per CU, half of them (two tiles in flight) with one
    const int prefetch = p.lds_bytes == kLdsPerCu / 2 ? kPrefetchHalf : kPrefetchFull / 2;
    // one-workgroup plans keep room for the trace's bitmasks after the zero record
    const int usage_bytes = int((int64_t(n_cols) + 31) / 32 * p.docs_per_block * 4);
    const int usage_room = p.lds_bytes == kLdsPerCu ? (usage_bytes + 15) & ~15 : 0;
    p.tile_bytes = std::min(p.lds_bytes - p.xs_bytes - reserve - usage_room, prefetch * 1024 * 8) & ~15;
    // One-workgroup plans copy a tile window as whole chunks of 1,024 records (one per thread):
    // a slot of whole chunks keeps that copy off the zero record and the trace's bitmasks.
    if (p.lds_bytes == kLdsPerCu)
        p.tile_bytes = p.tile_bytes / (1024 * 8) * (1024 * 8);
    p.zero_rec = p.xs_bytes + p.tile_bytes;
    p.usage_off = p.lds_bytes == kLdsPerCu ? (p.zero_rec + 8 + 15) & ~15 : kLdsPerCu / 2;
    // Interleave K trees per lane (latency hiding) only when a tile holds at least K rounds of
    // walker groups; otherwise most walkers would sit idle.
    const double fit = avg_tree_bytes > 0 ? p.tile_bytes / avg_tree_bytes : 1e9;
    const int walkers = 1024 / p.docs_per_block;
    p.interleave = fit >= 4.0 * walkers ? 4 : fit >= 2.0 * walkers ? 2 : 1;
    return p;
}

} // namespace

int pack_model(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
               const float *threshold, const int32_t *left, const int32_t *right,
               const float *value, int32_t n_outputs, uint32_t flags, Packed &out,
               std::string &err) {
    if (n_trees < 0) {
        err = "n_trees must be >= 0";
        return kErrArg;
    }
    if (n_outputs < 1 || n_outputs > kMaxOutputs) {
        err = "n_outputs must be in [1, " + std::to_string(kMaxOutputs) + "]";
        return kErrArg;
    }
    const bool vec = n_outputs > 1;
    if ((flags & ~(1u | kCodegenFlag)) != 0) {
        err = "unknown flag bits";
        return kErrArg;
    }
    const bool strict = (flags & 1u) != 0;
    if (n_trees > 0 && !tree_offsets) {
        err = "tree_offsets is NULL";
        return kErrArg;
    }
    if (n_trees > 0 && tree_offsets[0] != 0) {
        err = "tree_offsets[0] must be 0";
        return kErrModel;
    }
    int64_t n_nodes = n_trees > 0 ? tree_offsets[n_trees] : 0;
    for (int32_t t = 0; t < n_trees; t++) {
        if (tree_offsets[t + 1] - tree_offsets[t] < 1) {
            err = "tree " + std::to_string(t) + " has no node (tree_offsets must increase)";
            return kErrModel;
        }
    }
    if (n_nodes > 0 && (!feature || !threshold || !left || !right || !value)) {
        err = "a node array is NULL";
        return kErrArg;
    }
    if (n_nodes >= (int64_t(1) << 32) || (vec && n_nodes >= (int64_t(1) << 31))) {
        err = vec ? "more than 2^31 nodes with vector-valued leaves" : "more than 2^32 nodes";
        return kErrModel;
    }

    // ---- pass 1: per-tree validation, depth, largest feature id ------------------------
    int32_t max_fid = -1;
    std::vector<int32_t> depth_of(size_t(n_trees), 0);
    std::vector<int32_t> parents, level, order;
    for (int32_t t = 0; t < n_trees; t++) {
        const int64_t a = tree_offsets[t];
        const int64_t n = tree_offsets[t + 1] - a;
        const std::string where = "tree " + std::to_string(t) + ": ";
        if (n > kMaxTreeNodes) {
            err = where + "more than " + std::to_string(kMaxTreeNodes) + " nodes";
            return kErrModel;
        }
        parents.assign(size_t(n), 0);
        for (int64_t i = 0; i < n; i++) {
            const int32_t f = feature[a + i];
            if (f < -1) {
                err = where + "node " + std::to_string(i) + " has feature id " + std::to_string(f);
                return kErrModel;
            }
            if (f < 0)
                continue;
            if (std::isnan(threshold[a + i])) {
                err = where + "node " + std::to_string(i) + " has a NaN threshold";
                return kErrModel;
            }
            const int32_t l = left[a + i], r = right[a + i];
            if (l <= 0 || l >= n || r <= 0 || r >= n) {
                err = where + "node " + std::to_string(i) +
                      " has a child id out of range or naming the root";
                return kErrModel;
            }
            if (l == r) {
                err = where + "node " + std::to_string(i) + " has the same left and right child";
                return kErrModel;
            }
            parents[size_t(l)]++;
            parents[size_t(r)]++;
            max_fid = std::max(max_fid, f);
        }
        for (int64_t i = 1; i < n; i++) {
            if (parents[size_t(i)] != 1) {
                err = where + "node " + std::to_string(i) +
                      (parents[size_t(i)] == 0 ? " is unreachable (no parent)" : " has two parents");
                return kErrModel;
            }
        }
        // breadth-first from the root: with one parent per non-root node, every node is reached
        // exactly once unless part of the tree hangs in a cycle away from the root
        level.assign(size_t(n), 0);
        order.clear();
        order.push_back(0);
        int32_t dmax = 0;
        for (size_t q = 0; q < order.size(); q++) {
            const int32_t i = order[q];
            if (feature[a + i] >= 0) {
                for (int32_t c : {left[a + i], right[a + i]}) {
                    level[size_t(c)] = level[size_t(i)] + 1;
                    dmax = std::max(dmax, level[size_t(c)]);
                    order.push_back(c);
                }
            }
            if (int64_t(order.size()) > n)
                break;
        }
        if (int64_t(order.size()) != n) {
            err = where + "some nodes are not reachable from the root (a cycle)";
            return kErrModel;
        }
        depth_of[size_t(t)] = dmax;
    }

    const int32_t n_cols = max_fid + 1;
    auto canon = [&](float th) {
        float v = strict ? strict_to_inclusive(th) : th;
        return v == 0.0f ? 0.0f : v; // fold -0.0 into +0.0 (equal under every comparison)
    };

    // ---- coded features: per-feature sorted distinct thresholds -----------------------------
    // Possible when every feature's thresholds fit one coding workgroup and 16-bit codes; used
    // when float documents leave too few per block for the model's trees (below).
    std::vector<std::vector<float>> thr_of;
    int code_ok = -1; // -1: not computed yet
    auto can_code = [&]() {
        if (code_ok < 0) {
            code_ok = 1;
            thr_of.assign(size_t(n_cols), {});
            for (int64_t i = 0; i < n_nodes; i++) {
                if (feature[i] < 0)
                    continue;
                const float v = canon(threshold[i]);
                if (!std::isnan(v))
                    thr_of[size_t(feature[i])].push_back(v);
            }
            for (auto &tv : thr_of) {
                std::sort(tv.begin(), tv.end());
                tv.erase(std::unique(tv.begin(), tv.end()), tv.end());
                if (tv.size() > kMaxCode || tv.size() >= size_t(kCodeTableFloats))
                    code_ok = 0;
            }
        }
        return code_ok == 1;
    };

    // ---- LDS plan and the trees too large for one tile ---------------------------------------
    // A tree whose records (plus a tile's header and K root copies) exceed the plan's tile slot
    // is a "big" tree: it stays out of the tiles and is walked from device memory. The plan
    // depends on the mean size of the tiled trees, and the slot size on the plan, so the two are
    // settled together (a few rounds at most; the last plan's slot decides).
    std::vector<uint8_t> is_big(size_t(n_trees), 0);
    LdsPlan plan{};
    bool coded = false;
    int64_t max_nodes_per_tree = 0;
    for (int round = 0; round < 4; round++) {
        int64_t small_nodes = 0, n_small_trees = 0;
        for (int32_t t = 0; t < n_trees; t++)
            if (!is_big[size_t(t)]) {
                small_nodes += tree_offsets[t + 1] - tree_offsets[t];
                n_small_trees++;
            }
        const double avg_tree_bytes = n_small_trees > 0 ? 8.0 * double(small_nodes) / double(n_small_trees) : 0.0;
        plan = plan_lds(n_cols, avg_tree_bytes, 4);
        // Coding pays when float documents leave too few per block for the model's trees: when
        // a float tile cannot hold one tree for each walker, most walkers would idle.
        coded = plan.docs_per_block > 0 && plan.docs_per_block < 64 &&
                avg_tree_bytes * (1024 / plan.docs_per_block) > plan.tile_bytes && can_code();
        if (coded)
            plan = plan_lds(n_cols, avg_tree_bytes, 2);
        if (plan.docs_per_block == 0)
            break;
        // a one-tree tile holds the fixed header words and the root copies (padded to K records)
        max_nodes_per_tree = plan.tile_bytes / int64_t(sizeof(NodeRec)) - (kHeaderFixedWords / 2 + plan.interleave);
        bool changed = false;
        for (int32_t t = 0; t < n_trees; t++) {
            const uint8_t big = tree_offsets[t + 1] - tree_offsets[t] > max_nodes_per_tree;
            changed |= big != is_big[size_t(t)];
            is_big[size_t(t)] = big;
        }
        if (!changed)
            break;
    }
    if (plan.docs_per_block == 0) {
        err = "feature id " + std::to_string(max_fid) + " is beyond the LDS document-tile limit (" +
              std::to_string(kXsMaxBytes / (8 * 4) - 2) + ")";
        return kErrModel;
    }
    // the final plan's slot decides which trees are tiled
    int64_t largest_tree = 0;
    int32_t n_small = 0;
    for (int32_t t = 0; t < n_trees; t++) {
        const int64_t n = tree_offsets[t + 1] - tree_offsets[t];
        is_big[size_t(t)] = n > max_nodes_per_tree;
        if (!is_big[size_t(t)]) {
            largest_tree = std::max(largest_tree, n);
            n_small++;
        }
    }
    // the narrow format needs column offsets below 64 KiB and links below 2^16 (absolute LDS
    // record indices are below 160 KiB / 8 = 20480; tree-relative ones below the tree's size)
    plan.narrow = (plan.xs_bytes <= 65536 && largest_tree <= kNarrowMaxTreeNodes) ? 1 : 0;

    // ---- tree order: expected lockstep length ----------------------------------------------
    // A wave steps through a tree until the longest of its 64 documents' paths ends, so the trees
    // walked side by side (a group of K, the walkers of one round) should end together. With no
    // documents at hand, a split's chance of sending a document right is estimated from the
    // model's own thresholds on that feature (the share of them below this one: thresholds are
    // cut where the training data lies, so their spread follows the feature's); a tree's
    // leaf-depth distribution follows, and its key is the expected longest of 64 independent
    // paths. Complete trees (every path equally long) get exactly their depth, and come before
    // any other tree of an equal key, so that they still form complete-depth tiles. The order
    // changes only the rounding of the sums.
    std::vector<double> lock_key(size_t(n_trees), 0.0);
    std::vector<uint8_t> complete_tree(size_t(n_trees), 0);
    {
        std::vector<std::vector<float>> thr_sorted(static_cast<size_t>(n_cols));
        for (int64_t i = 0; i < n_nodes; i++) {
            const float v = feature[i] >= 0 ? canon(threshold[i]) : 0.0f;
            if (feature[i] >= 0 && !std::isnan(v)) // NaN: a strict +inf split, never right
                thr_sorted[size_t(feature[i])].push_back(v);
        }
        for (auto &v : thr_sorted)
            std::sort(v.begin(), v.end());
        std::vector<double> reach, at_depth;
        for (int32_t t = 0; t < n_trees; t++) {
            const int64_t a = tree_offsets[t];
            const int64_t n = tree_offsets[t + 1] - a;
            complete_tree[size_t(t)] = is_complete(n, depth_of[size_t(t)]);
            reach.assign(size_t(n), 0.0);
            level.assign(size_t(n), 0);
            at_depth.assign(size_t(depth_of[size_t(t)]) + 1, 0.0);
            reach[0] = 1.0;
            order.clear();
            order.push_back(0);
            for (size_t q = 0; q < order.size(); q++) {
                const int32_t i = order[q];
                if (feature[a + i] < 0) {
                    at_depth[size_t(level[size_t(i)])] += reach[size_t(i)];
                    continue;
                }
                const auto &ts = thr_sorted[size_t(feature[a + i])];
                const float v = canon(threshold[a + i]);
                const size_t below = size_t(std::lower_bound(ts.begin(), ts.end(), v) - ts.begin());
                const double p_right = std::isnan(v) ? 0.0 : 1.0 - double(below) / double(ts.size());
                const int32_t l = left[a + i], r = right[a + i];
                reach[size_t(r)] = reach[size_t(i)] * p_right;
                reach[size_t(l)] = reach[size_t(i)] * (1.0 - p_right);
                level[size_t(l)] = level[size_t(r)] = level[size_t(i)] + 1;
                order.push_back(l);
                order.push_back(r);
            }
            // E[max of 64 paths] = sum over d of P(some path is longer than d)
            double cdf = 0.0, key = 0.0;
            for (int32_t d = 0; d < depth_of[size_t(t)]; d++) {
                cdf = std::min(cdf + at_depth[size_t(d)], 1.0);
                double c = cdf;
                for (int k = 0; k < 6; k++)
                    c *= c; // cdf^64
                key += 1.0 - c;
            }
            lock_key[size_t(t)] = complete_tree[size_t(t)] ? double(depth_of[size_t(t)]) : key;
        }
    }

    // ---- pass 2: order trees by expected lockstep length (longest first), re-lay each out
    // breadth-first ------------------------------------------------------------------------------
    Packed p;
    p.n_trees = n_trees;
    p.n_cols = n_cols;
    p.plan = plan;
    p.n_outputs = n_outputs;
    if (vec) {
        p.vec_stride = (n_outputs + 3) / 4 * 4;
        p.leaf_vec.assign(size_t(n_nodes + 1) * size_t(p.vec_stride), 0.0f);
    }
    p.tree_orig.resize(size_t(n_trees));
    std::iota(p.tree_orig.begin(), p.tree_orig.end(), 0);
    std::stable_sort(p.tree_orig.begin(), p.tree_orig.end(), [&](int32_t x, int32_t y) {
        if (is_big[size_t(x)] != is_big[size_t(y)])
            return is_big[size_t(x)] < is_big[size_t(y)]; // tiled trees first, big ones last
        if (lock_key[size_t(x)] != lock_key[size_t(y)])
            return lock_key[size_t(x)] > lock_key[size_t(y)];
        if (complete_tree[size_t(x)] != complete_tree[size_t(y)])
            return complete_tree[size_t(x)] > complete_tree[size_t(y)];
        return depth_of[size_t(x)] > depth_of[size_t(y)];
    });
    p.n_small = n_small;
    p.nodes.reserve(size_t(n_nodes));
    p.orig_id.reserve(size_t(n_nodes));
    p.tree_node_off.resize(size_t(n_trees) + 1, 0);
    p.tree_depth.resize(size_t(n_trees), 0);
    std::vector<int32_t> new_id;
    for (int32_t pt = 0; pt < n_trees; pt++) {
        const int32_t t = p.tree_orig[size_t(pt)];
        // big trees (packed last) take the big-tree record format (see kBigLinkShift)
        const bool big_tree = pt >= n_small;
        auto link = [&](uint32_t child) {
            return big_tree ? child << kBigLinkShift : plan.narrow ? child << 16 : child << kWideChildShift;
        };
        const int64_t a = tree_offsets[t];
        const int64_t n = tree_offsets[t + 1] - a;
        // breadth-first numbering in which the two children of a node take adjacent slots
        order.clear();
        order.push_back(0);
        new_id.assign(size_t(n), -1);
        new_id[0] = 0;
        int32_t next = 1;
        for (size_t q = 0; q < order.size(); q++) {
            const int32_t i = order[q];
            if (feature[a + i] >= 0) {
                new_id[size_t(left[a + i])] = next;
                new_id[size_t(right[a + i])] = next + 1;
                next += 2;
                order.push_back(left[a + i]);
                order.push_back(right[a + i]);
            }
        }
        const size_t base = p.nodes.size();
        p.tree_node_off[size_t(pt)] = uint32_t(base);
        p.nodes.resize(base + size_t(n));
        p.orig_id.resize(base + size_t(n));
        for (int64_t i = 0; i < n; i++) {
            const int32_t ni = new_id[size_t(i)];
            NodeRec &r = p.nodes[base + size_t(ni)];
            p.orig_id[base + size_t(ni)] = int32_t(i);
            if (feature[a + i] >= 0) {
                const float th = strict ? strict_to_inclusive(threshold[a + i]) : threshold[a + i];
                r.thr_bits = float_bits(th);
                if (plan.coded) {
                    const float v = canon(threshold[a + i]);
                    const auto &tv = thr_of[size_t(feature[a + i])];
                    r.thr_bits = std::isnan(v) ? 0xFFFFu
                                               : uint32_t(std::lower_bound(tv.begin(), tv.end(), v) -
                                                          tv.begin()) + 1u;
                }
                const uint32_t col = big_tree ? uint32_t(feature[a + i] + 1)
                                              : uint32_t(feature[a + i] + 1) * uint32_t(plan.docs_per_block) *
                                                    uint32_t(plan.elem_bytes);
                r.w = link(uint32_t(new_id[size_t(left[a + i])])) | col;
            } else if (vec) {
                // never 0: a coded leaf (code 0 >= thr is false) stays put as well
                const size_t packed = base + size_t(ni);
                r.thr_bits = uint32_t(packed) + 2u;
                for (int32_t c = 0; c < n_outputs; c++)
                    p.leaf_vec[(packed + 1) * size_t(p.vec_stride) + size_t(c)] =
                        value[(a + i) * n_outputs + c];
                r.w = link(uint32_t(ni));
            } else {
                r.thr_bits = float_bits(value[a + i]);
                if (plan.coded && r.thr_bits == 0u)
                    r.thr_bits = 0x80000000u; // +0.0 as -0.0: never 0, so the leaf stays put
                r.w = link(uint32_t(ni));
            }
        }
        p.tree_depth[size_t(pt)] = uint32_t(depth_of[size_t(t)]);
        p.max_depth = std::max(p.max_depth, depth_of[size_t(t)]);
    }
    p.tree_node_off[size_t(n_trees)] = uint32_t(p.nodes.size());

    // ---- pass 3: tilings at budget / 2^k -------------------------------------------------
    // A tile is a run of whole trees whose image (header + records) fits the byte budget. When
    // more than one round of walker groups fits, the run is cut to a whole number of rounds
    // (walkers x interleave trees), so that statically assigned groups finish together.
    const int32_t K = plan.interleave;
    const int32_t round = (1024 / plan.docs_per_block) * K;
    // header records of a tile of n trees: fixed words + root copies padded to K
    auto header_recs = [&](int32_t n) { return kHeaderFixedWords / 2 + (n + K - 1) / K * K; };
    for (int k = 0; k < kTileLevels; k++) {
        p.level_begin[k] = int32_t(p.tiles.size());
        const int64_t budget = std::max<int64_t>(plan.tile_bytes >> k, 16);
        int32_t tb = 0;
        while (tb < n_small) {
            int32_t fit = 0;
            for (int64_t recs = 0; tb + fit < n_small && fit < kMaxTileTrees; fit++) {
                const int64_t nn = int64_t(p.tree_node_off[size_t(tb + fit) + 1] -
                                           p.tree_node_off[size_t(tb + fit)]);
                if (fit > 0 && (header_recs(fit + 1) + recs + nn) * 8 > budget)
                    break;
                recs += nn;
            }
            const int32_t limit = (fit > round && tb + fit < n_small) ? fit / round * round : fit;
            int32_t te = tb;
            int32_t dmax = 0;
            int32_t complete = -2; // -2: no tree yet
            while (te < tb + limit) {
                const int64_t nn = int64_t(p.tree_node_off[size_t(te) + 1] - p.tree_node_off[size_t(te)]);
                const int32_t d = int32_t(p.tree_depth[size_t(te)]);
                dmax = std::max(dmax, d);
                const bool full = is_complete(nn, d);
                complete = (complete == -2 || complete == d) && full ? d : -1;
                te++;
            }
            // a tile whose last group has idle slots (the zero record) is walked as a general
            // one: complete walks add every slot's leaf record as a double
            if ((te - tb) % K != 0)
                complete = -1;
            p.tiles.push_back(Tile{tb, te, dmax, int32_t(p.tree_node_off[size_t(tb)]), complete});
            tb = te;
        }
    }
    p.level_begin[kTileLevels] = int32_t(p.tiles.size());

    // ---- pass 4: tile images --------------------------------------------------------------
    // Records keep their column offsets; links become absolute LDS record indices: the slot
    // starts right after the document tile, the records right after the header.
    const int shift = plan.narrow ? 16 : kWideChildShift;
    const uint32_t col_mask = plan.narrow ? kNarrowColMask : kWideColMask;
    const uint32_t zero_addr = uint32_t(plan.zero_rec);
    for (int k = 0; k < kTileLevels; k++) {
        for (int32_t i = p.level_begin[k]; i < p.level_begin[k + 1]; i++) {
            const Tile &tl = p.tiles[size_t(i)];
            const int32_t r = (tl.tree_end - tl.tree_begin + round - 1) / round;
            p.level_max_rounds[k] = std::max(p.level_max_rounds[k], r);
            if (k == 0)
                p.total_rounds += r;
        }
    }
    p.tile_recs.resize(p.tiles.size());
    for (size_t i = 0; i < p.tiles.size(); i++) {
        const Tile &tl = p.tiles[i];
        p.tile_recs[i] = uint32_t(header_recs(tl.tree_end - tl.tree_begin)) +
                         (p.tree_node_off[size_t(tl.tree_end)] - uint32_t(tl.node_begin));
    }
    for (int k = 0; k < kTileLevels; k++) {
        uint32_t slot = 2;
        for (int32_t i = p.level_begin[k]; i < p.level_begin[k + 1]; i++)
            slot = std::max(slot, p.tile_recs[size_t(i)]);
        p.level_slot_recs[k] = int32_t(slot);
        p.level_image_off[k] = int64_t(p.images.size());
        const int32_t n_level = p.level_begin[k + 1] - p.level_begin[k];
        p.images.resize(p.images.size() + size_t(n_level) * slot, NodeRec{0u, 0u});
        for (int32_t i = 0; i < n_level; i++) {
            const Tile &tl = p.tiles[size_t(p.level_begin[k] + i)];
            NodeRec *img = p.images.data() + p.level_image_off[k] + int64_t(i) * slot;
            const int32_t ntr = tl.tree_end - tl.tree_begin;
            const int32_t hrecs = header_recs(ntr);
            const uint32_t rec0 = uint32_t(plan.xs_bytes / 8 + hrecs); // LDS index of record 0
            img[0] = NodeRec{uint32_t(ntr), uint32_t(tl.complete_depth)};
            img[1] = NodeRec{uint32_t(tl.tree_begin),
                             i + 1 < n_level ? p.tile_recs[size_t(p.level_begin[k] + i + 1)] : 0u};
            const NodeRec zero_leaf{zero_record_value(plan, vec), (zero_addr / 8u) << shift};
            const bool f64_leaves = tl.complete_depth >= 0 && !vec;
            for (int32_t t = 0; t < hrecs - kHeaderFixedWords / 2; t++) {
                NodeRec r = zero_leaf;
                if (t < ntr) {
                    const uint32_t first = p.tree_node_off[size_t(tl.tree_begin + t)];
                    const uint32_t tree_rec = rec0 + first - uint32_t(tl.node_begin);
                    r = p.nodes[first];
                    r.w = ((tree_rec + (r.w >> shift)) << shift) | (r.w & col_mask);
                    if (f64_leaves)
                        r = complete_leaf(r, col_mask);
                }
                img[kHeaderFixedWords / 2 + t] = r;
            }
            for (int32_t t = tl.tree_begin; t < tl.tree_end; t++) {
                const uint32_t first = p.tree_node_off[size_t(t)];
                const uint32_t tree_rec = rec0 + first - uint32_t(tl.node_begin);
                for (uint32_t n = first; n < p.tree_node_off[size_t(t) + 1]; n++) {
                    NodeRec r = p.nodes[n];
                    r.w = ((tree_rec + (r.w >> shift)) << shift) | (r.w & col_mask);
                    if (f64_leaves)
                        r = complete_leaf(r, col_mask);
                    img[hrecs + int64_t(n - uint32_t(tl.node_begin))] = r;
                }
            }
        }
    }

    // ---- walker packets (plans of 64- or 32-document blocks; see pack.hpp) -----------------------
    if ((plan.docs_per_block == 64 || plan.docs_per_block == 32) && n_small > 0) {
        constexpr int32_t W = kPacketWalkers;       // waves, one packet stream each
        const int32_t P = 64 / plan.docs_per_block; // walkers per wave
        const int32_t HW = W * P;                   // walkers
        const bool half = plan.lds_bytes == kLdsPerCu / 2;
        // two workgroups per CU: the sub-slots share the tile slot (the zero record after it);
        // one: they take the LDS past the document tile, then their own zero record
        const int64_t region = half ? int64_t(plan.tile_bytes) : int64_t(plan.lds_bytes) - plan.xs_bytes - 16;
        const int32_t sub = int32_t(std::max<int64_t>(region, 0) / 8 / W / 64 * 64); // records per sub-slot
        const int32_t part = sub / P; // records of one walker's part of a packet
        const int32_t pk_zero = half ? plan.zero_rec : plan.xs_bytes + W * sub * 8;
        const int32_t n_groups = (n_small + K - 1) / K;
        // walker h of wave v (walker index v * P + h) takes groups v * P + h + r * HW, r = 0, 1, ...
        auto group_of = [&](int32_t v, int32_t h, int32_t r) { return v * P + h + r * HW; };
        auto group_recs = [&](int32_t g) {
            if (g >= n_groups)
                return int64_t(0); // past the last group: zero roots, no records
            const int32_t t0 = g * K, t1 = std::min(n_small, t0 + K);
            return int64_t(p.tree_node_off[size_t(t1)]) - int64_t(p.tree_node_off[size_t(t0)]);
        };
        auto packet_recs = [&](int32_t ng, int64_t tree_recs) {
            return int64_t(kPacketHeaderRecs) + int64_t(ng) * K + (int64_t(ng) * K + 3) / 4 + tree_recs;
        };
        // per wave: runs (first round, rounds) of consecutive rounds whose groups fit every
        // walker's part of the sub-slot; all walkers of a wave step through the same rounds
        std::vector<std::vector<std::pair<int32_t, int32_t>>> runs(static_cast<size_t>(W));
        bool fits = sub > 0 && part % 2 == 0 && sub / 64 <= (half ? kPrefetchHalf : kPrefetchFull);
        for (int32_t v = 0; v < W && fits; v++) {
            int32_t rounds = 0;
            while (group_of(v, 0, rounds) < n_groups)
                rounds++;
            int32_t first = -1, count = 0;
            std::vector<int64_t> recs(static_cast<size_t>(P), 0);
            for (int32_t r = 0; r < rounds; r++) {
                bool more = first >= 0;
                for (int32_t h = 0; h < P && more; h++)
                    more = packet_recs(count + 1, recs[size_t(h)] + group_recs(group_of(v, h, r))) <= part;
                if (more) {
                    count++;
                    for (int32_t h = 0; h < P; h++)
                        recs[size_t(h)] += group_recs(group_of(v, h, r));
                    continue;
                }
                if (first >= 0)
                    runs[size_t(v)].push_back({first, count});
                for (int32_t h = 0; h < P; h++)
                    if (packet_recs(1, group_recs(group_of(v, h, r))) > part)
                        fits = false;
                if (!fits)
                    break;
                first = r;
                count = 1;
                for (int32_t h = 0; h < P; h++)
                    recs[size_t(h)] = group_recs(group_of(v, h, r));
            }
            if (fits && first >= 0)
                runs[size_t(v)].push_back({first, count});
        }
        int32_t per = 0;
        for (const auto &r : runs)
            per = std::max(per, int32_t(r.size()));
        // the kernel addresses packets with 32-bit byte offsets
        if (int64_t(W) * per * sub * int64_t(sizeof(NodeRec)) >= (int64_t(1) << 31))
            fits = false;
        if (fits) {
            p.pk_recs = sub;
            p.pk_zero_rec = pk_zero;
            p.pk_per_walker = per;
            p.packets.assign(size_t(W) * size_t(per) * size_t(sub), NodeRec{0u, 0u});
            std::vector<int32_t> most(static_cast<size_t>(per), 0);
            const NodeRec zero_leaf{zero_record_value(plan, vec), (uint32_t(pk_zero) / 8u) << shift};
            for (int32_t v = 0; v < W; v++) {
                for (size_t q = 0; q < runs[size_t(v)].size(); q++) {
                    const int32_t r0 = runs[size_t(v)][q].first, ng = runs[size_t(v)][q].second;
                    p.pk_max_groups = std::max(p.pk_max_groups, ng);
                    most[q] = std::max(most[q], ng);
                    // the common complete depth of every tree of the packet, else -1
                    int32_t complete = -2; // -2: no tree yet
                    bool idle = false;
                    for (int32_t h = 0; h < P; h++) {
                        for (int32_t j = 0; j < ng; j++) {
                            for (int32_t i = 0; i < K; i++) {
                                const int32_t t = group_of(v, h, r0 + j) * K + i;
                                if (t >= n_small) {
                                    idle = true; // an idle slot: the packet is walked as general
                                    continue;
                                }
                                const int32_t d = int32_t(p.tree_depth[size_t(t)]);
                                const int64_t nn = int64_t(p.tree_node_off[size_t(t) + 1] - p.tree_node_off[size_t(t)]);
                                const bool full = is_complete(nn, d);
                                complete = (complete == -2 || complete == d) && full ? d : -1;
                            }
                        }
                    }
                    if (idle)
                        complete = -1;
                    for (int32_t h = 0; h < P; h++) {
                        const uint32_t base = uint32_t(plan.xs_bytes / 8) + uint32_t(v * sub + h * part); // in LDS
                        NodeRec *img = p.packets.data() + (size_t(v) * size_t(per) + q) * size_t(sub) + size_t(h * part);
                        img[0] = NodeRec{uint32_t(ng), uint32_t(complete)};
                        img[1] = NodeRec{uint32_t(group_of(v, h, r0)), 0u};
                        const int32_t table = kPacketHeaderRecs + ng * K;
                        uint16_t *first_rec = reinterpret_cast<uint16_t *>(img + table);
                        int32_t pos = table + (ng * K + 3) / 4;
                        for (int32_t j = 0; j < ng; j++) {
                            for (int32_t i = 0; i < K; i++) {
                                const int32_t t = group_of(v, h, r0 + j) * K + i;
                                NodeRec root = zero_leaf;
                                if (t < n_small) {
                                    const uint32_t first = p.tree_node_off[size_t(t)];
                                    const uint32_t nn = p.tree_node_off[size_t(t) + 1] - first;
                                    const uint32_t tree_rec = base + uint32_t(pos);
                                    first_rec[j * K + i] = uint16_t(tree_rec);
                                    for (uint32_t n = 0; n < nn; n++) {
                                        NodeRec r = p.nodes[first + n];
                                        r.w = ((tree_rec + (r.w >> shift)) << shift) | (r.w & col_mask);
                                        if (complete >= 0 && !vec)
                                            r = complete_leaf(r, col_mask);
                                        img[pos + int32_t(n)] = r;
                                    }
                                    root = img[pos];
                                    pos += int32_t(nn);
                                }
                                img[kPacketHeaderRecs + j * K + i] = root;
                            }
                        }
                    }
                }
            }
            for (int32_t m : most)
                p.pk_total_rounds += m;
        }
    }

    // ---- compact packets (coded plans of 64-document blocks; see kCompactWindowBytes) ------------
    {
        constexpr int32_t W = kPacketWalkers;
        constexpr int32_t kWords = kCompactPacketBytes / 4;
        int64_t max_nodes = 0;
        for (int32_t t = 0; t < n_small; t++)
            max_nodes = std::max<int64_t>(max_nodes, p.tree_node_off[size_t(t) + 1] - p.tree_node_off[size_t(t)]);
        size_t max_thr = 0;
        if (plan.coded)
            for (const auto &tv : thr_of)
                max_thr = std::max(max_thr, tv.size());
        const int64_t cw = compact_window_base(plan.xs_bytes);
        // bytes of tree t's children pairs (a lone leaf: one pair of itself)
        auto body = [&](int32_t t) {
            const int64_t n = int64_t(p.tree_node_off[size_t(t) + 1]) - int64_t(p.tree_node_off[size_t(t)]);
            return int32_t(4 * std::max<int64_t>(2, n - 1));
        };
        constexpr int32_t K = kCompactTrees;
        const int32_t win = kCompactWindowBytes / K, cap = win - 8;
        const int32_t n_groups = (n_trees + K - 1) / K;
        const int32_t max_ng = (kCompactHeaderBytes / 4 - kCompactHeaderWords) / K;
        bool ok = plan.coded && plan.docs_per_block == 64 && plan.lds_bytes == kLdsPerCu && n_trees > 0 &&
                  n_small == n_trees && n_cols + 1 <= kCompactMaxColumns && max_thr < kCompactNeverRight &&
                  max_nodes <= kCompactMaxTreeNodes && cw + int64_t(W) * kCompactWindowBytes <= kLdsPerCu;
        // per wave: runs (first round, groups) of consecutive rounds whose trees fit every window
        std::vector<std::vector<std::pair<int32_t, int32_t>>> runs(static_cast<size_t>(W));
        for (int32_t v = 0; v < W && ok; v++) {
            int32_t first = -1, count = 0;
            std::vector<int32_t> used(static_cast<size_t>(K), 0);
            for (int32_t r = 0; v + r * W < n_groups; r++) {
                const int32_t g = v + r * W;
                bool more = first >= 0 && count < max_ng;
                for (int32_t i = 0; i < K && more; i++) {
                    const int32_t t = g * K + i;
                    more = t >= n_trees || used[size_t(i)] + body(t) <= cap;
                }
                if (!more) {
                    if (first >= 0)
                        runs[size_t(v)].push_back({first, count});
                    first = r;
                    count = 0;
                    std::fill(used.begin(), used.end(), 0);
                }
                count++;
                for (int32_t i = 0; i < K; i++)
                    if (g * K + i < n_trees)
                        used[size_t(i)] += body(g * K + i);
            }
            if (first >= 0)
                runs[size_t(v)].push_back({first, count});
        }
        int32_t per = 0;
        for (const auto &r : runs)
            per = std::max(per, int32_t(r.size()));
        // the kernel addresses packets (and their payloads) with 32-bit byte offsets
        if (int64_t(W) * per * kCompactPacketBytes >= (int64_t(1) << 31))
            ok = false;
        if (ok) {
            const int shift_c = plan.narrow ? 16 : kWideChildShift;
            const uint32_t cmask = plan.narrow ? kNarrowColMask : kWideColMask;
            const uint32_t col_bytes = uint32_t(plan.docs_per_block * plan.elem_bytes);
            p.cp_k = K;
            p.cp_per_walker = per;
            const size_t total = size_t(W) * size_t(per) * size_t(kWords);
            p.cp_packets.assign(total, 0u);
            p.cp_leaf.assign(total, 0u);
            p.cp_leaf_id.assign(total, -1);
            std::vector<int32_t> most(static_cast<size_t>(per), 0);
            for (int32_t v = 0; v < W; v++) {
                for (size_t q = 0; q < runs[size_t(v)].size(); q++) {
                    const int32_t r0 = runs[size_t(v)][q].first, ng = runs[size_t(v)][q].second;
                    const size_t at = (size_t(v) * size_t(per) + q) * size_t(kWords);
                    uint32_t *img = p.cp_packets.data() + at;
                    uint32_t *pay = p.cp_leaf.data() + at;
                    int32_t *ids = p.cp_leaf_id.data() + at;
                    uint32_t *hdr = img + kCompactWindowBytes / 4;
                    p.cp_max_groups = std::max(p.cp_max_groups, ng);
                    most[q] = std::max(most[q], ng);
                    // the zero pair at the end of each window: a left-side leaf of payload 0
                    const uint32_t zero = (kCompactNeverRight << kCompactThrShift) | uint32_t(cap);
                    for (int32_t i = 0; i < K; i++) {
                        const size_t zw = size_t(i * win + cap) / 4;
                        img[zw] = img[zw + 1] = zero;
                        pay[zw] = pay[zw + 1] = vec ? 1u : 0u;
                    }
                    // the common complete depth of every tree of the packet, else -1
                    int32_t complete = -2;
                    for (int32_t j = 0; j < ng; j++)
                        for (int32_t i = 0; i < K; i++) {
                            const int32_t t = (v + (r0 + j) * W) * K + i;
                            if (t >= n_trees) {
                                complete = -1; // an idle slot
                                continue;
                            }
                            const int32_t d = int32_t(p.tree_depth[size_t(t)]);
                            const int64_t nn = int64_t(p.tree_node_off[size_t(t) + 1] - p.tree_node_off[size_t(t)]);
                            complete = (complete == -2 || complete == d) && is_complete(nn, d) ? d : -1;
                        }
                    hdr[0] = uint32_t(ng);
                    hdr[1] = uint32_t(complete);
                    hdr[2] = uint32_t(v + r0 * W);
                    hdr[3] = 0u;
                    std::vector<uint32_t> off(static_cast<size_t>(K), 0u);
                    for (int32_t j = 0; j < ng; j++) {
                        for (int32_t i = 0; i < K; i++) {
                            const int32_t t = (v + (r0 + j) * W) * K + i;
                            uint32_t &root = hdr[kCompactHeaderWords + j * K + i];
                            if (t >= n_trees) {
                                root = zero;
                                continue;
                            }
                            const uint32_t first = p.tree_node_off[size_t(t)];
                            const uint32_t nn = p.tree_node_off[size_t(t) + 1] - first;
                            const uint32_t o = off[size_t(i)];
                            // window byte offset of node k (k >= 1: its slot among the pairs; a
                            // lone root leaf: the first slot of its own pair)
                            auto pos_of = [&](uint32_t k) { return k == 0 ? o : o + (k - 1) * 4u; };
                            auto enc = [&](uint32_t k) {
                                const NodeRec &r = p.nodes[first + k];
                                const uint32_t colb = r.w & cmask;
                                if (colb != 0) {
                                    const uint32_t lc = r.w >> shift_c; // left child (tree-relative)
                                    const uint32_t thr = r.thr_bits > kMaxCode ? kCompactNeverRight : r.thr_bits;
                                    return (thr << kCompactThrShift) | ((colb / col_bytes) << kCompactColShift) |
                                           (o + (lc - 1) * 4u);
                                }
                                const uint32_t pos = pos_of(k);
                                return (((pos >> 2) & 1u) ? 0u : kCompactNeverRight << kCompactThrShift) | pos;
                            };
                            auto put = [&](uint32_t k) {
                                const size_t w = size_t(uint32_t(i * win) + pos_of(k)) / 4;
                                img[w] = enc(k);
                                if ((p.nodes[first + k].w & cmask) == 0) {
                                    pay[w] = p.nodes[first + k].thr_bits;
                                    ids[w] = p.orig_id[first + k];
                                }
                            };
                            root = enc(0);
                            if (nn == 1) {
                                put(0);
                                img[size_t(uint32_t(i * win) + o) / 4 + 1] = root;
                            } else {
                                for (uint32_t k = 1; k < nn; k++)
                                    put(k);
                            }
                            off[size_t(i)] += uint32_t(body(t));
                        }
                    }
                }
            }
            for (int32_t m : most)
                p.cp_total_rounds += m;
        }
    }

    if (plan.lds_bytes == kLdsPerCu / 2) {
        const int64_t used = p.pk_recs > 0 ? int64_t(kPacketWalkers) * p.pk_recs : int64_t(p.level_slot_recs[0]);
        const int64_t off = (int64_t(plan.xs_bytes) + used * 8 + 15) & ~int64_t(15);
        const int64_t mask_bytes = (int64_t(n_cols) + 31) / 32 * plan.docs_per_block * 4;
        if (off + mask_bytes <= plan.zero_rec)
            p.usage_slot_off = int32_t(off);
    }

    // The one-workgroup-per-CU kernels copy whole windows of 1,024-record chunks: pad the images
    // so that the window of the last tile stays inside the buffer.
    p.images.resize(p.images.size() + size_t(kPrefetchFull / 2) * 1024, NodeRec{0u, 0u});

    // ---- coded models: threshold table and coding chunks ------------------------------------
    if (plan.coded) {
        p.code_table_off.assign(size_t(n_cols) + 1, 0);
        for (int32_t f = 0; f < n_cols; f++) {
            p.code_table_off[size_t(f)] = uint32_t(p.code_table.size());
            p.code_table.insert(p.code_table.end(), thr_of[size_t(f)].begin(), thr_of[size_t(f)].end());
        }
        p.code_table_off[size_t(n_cols)] = uint32_t(p.code_table.size());
        // bits of a feature's search: the least s with 2^s - 1 >= |T_f|
        auto bits = [&](int32_t f) {
            int32_t s = 0;
            while ((uint32_t(1) << s) - 1u < p.code_table_off[size_t(f) + 1] - p.code_table_off[size_t(f)])
                s++;
            return s;
        };
        std::vector<float> sorted;
        int32_t fb = 0;
        while (fb < n_cols) {
            int32_t fe = fb + 1, steps = bits(fb);
            while (fe < n_cols && fe - fb < kCodeChunkFeatures) {
                const int32_t s = std::max(steps, bits(fe));
                if (int64_t(fe + 1 - fb) * ((int64_t(1) << s) - 1) > kCodeTableFloats)
                    break;
                steps = s;
                fe++;
            }
            const int32_t slots = 1 << steps;
            const int32_t begin = int32_t(p.code_search.size());
            p.code_search.resize(p.code_search.size() + size_t(fe - fb) * size_t(slots - 1), std::nanf(""));
            for (int32_t f = fb; f < fe; f++) {
                // in-order walk of the complete tree of slots 1 .. slots - 1 takes the sorted list
                sorted.assign(p.code_table.begin() + p.code_table_off[size_t(f)],
                              p.code_table.begin() + p.code_table_off[size_t(f) + 1]);
                sorted.resize(size_t(slots - 1), std::nanf(""));
                float *dst = p.code_search.data() + begin + size_t(f - fb) * size_t(slots - 1) - 1; // slot i
                size_t next = 0;
                std::vector<std::pair<int32_t, bool>> stack; // (slot, children done)
                stack.push_back({1, false});
                while (!stack.empty()) {
                    auto [i, done] = stack.back();
                    stack.pop_back();
                    if (i >= slots)
                        continue;
                    if (done) {
                        dst[i] = sorted[next++];
                        stack.push_back({2 * i + 1, false});
                    } else {
                        stack.push_back({i, true});
                        stack.push_back({2 * i, false});
                    }
                }
            }
            p.code_chunks.push_back(CodeChunk{fb, fe, begin, int32_t(p.code_search.size()), steps});
            fb = fe;
        }
    }
    out = std::move(p);
    return kOk;
}

} // namespace treeens
