// tree_ens.hip -- gfx950 kernels and the C ABI of the tree-ensemble scorer.
//
// Work decomposition (one scoring launch per predict call):
//   * a workgroup owns a block of DL consecutive documents and stages their features into LDS
//     once, feature-major ([column][DL] values, column 0 = NaN, column f+1 = feature f), so a
//     lane's read of any feature of its own document is a conflict-free LDS access whatever
//     feature the lane's current node names;
//   * the trees are streamed through an LDS slot in tiles: self-describing images (header,
//     root copies, node records with absolute child links) copied global -> registers -> LDS,
//     the next one loading while the current one is walked;
//   * lanes are documents; each group of DL lanes (a "walker", a whole wave when DL = 64) walks
//     K trees of the tile at a time so that their LDS latencies overlap (the vectorisation
//     idea of Section 3, VPred, applied to trees instead of instances);
//   * each step is the branch-free predicated update of Section 3 (Pred) over explicit,
//     sibling-adjacent children: idx = left(idx) + (x[fid(idx)] >= theta(idx)); a wave stops
//     as soon as all its lanes sit on leaves (trees are unbalanced; most paths are short);
//   * leaf values are summed per lane in double precision, then reduced across walkers through
//     LDS in a fixed order and rounded once to float.
// Blocks of a last, partial round of workgroups (and every block of a small batch) are split
// over the tiles; the per-split partial sums are reduced by a second, tiny kernel in a fixed
// order, so results are deterministic.
// The same kernel has three more modes: leaf ids (the reached leaf of every (document, tree)),
// the feature-access trace (the set of distinct features each document's walks compare, the
// measure of Section 6 / Table 4: per-document bitmasks in LDS, set with an LDS atomic OR at
// every internal step), and vector-valued leaves (a leaf names a row of a leaf-vector table in
// global memory; a launch sums four of its components).
#include <hip/hip_runtime.h>
#include <hip/hiprtc.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <type_traits>
#include <vector>

#include "pack.hpp"
#include "status.hpp"
#include "tree_ens.h"

using treeens::NodeRec;
using treeens::Packed;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string &msg) {
    g_err = msg;
    return code;
}

int hip_fail(hipError_t e, const char *what) {
    return fail(TREE_ENS_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

constexpr int kNumCus = 256;
constexpr int kXcds = 8; // accelerator complex dies, each with its own L2
// s_waitcnt immediate for gfx9: vmcnt(0), expcnt and lgkmcnt left at their maxima (no wait)
constexpr int kWaitVmcnt0 = 0x0F70;
// the same with lgkmcnt(0) (LDS and scalar memory) and vmcnt, expcnt at their maxima
constexpr int kWaitLgkmcnt0 = 0xC07F;
constexpr int kPrefetchDepth = 2; // tiles in flight with one workgroup per CU
constexpr int kThreads = 1024; // workgroup size of the scoring kernel (16 waves)
// what a launch of the scoring kernel produces
constexpr int kModeScore = 0;  // scores
constexpr int kModeLeaves = 1; // leaf ids
constexpr int kModeUsage = 2;  // per-document feature bitmasks and their popcounts
constexpr int kModeUsageSlot = 4; // the same with the bitmasks in the unused end of the tile slot
constexpr int kModeVector = 3; // four components of vector-valued scores
constexpr int kVecPerLaunch = 4;

// ------------------------------------------------------------------------------------------
// kernels
// ------------------------------------------------------------------------------------------

// (w & mask) | b in one VALU op. The feature column offset is a multiple of DL * 4 and the lane
// offset is below DL * 4, so the OR is the sum the address needs.
__device__ __forceinline__ uint32_t and_or(uint32_t w, uint32_t mask, uint32_t b) {
    uint32_t r;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(w), "s"(mask), "v"(b));
    return r;
}
// One 8-byte node record from LDS, as one ds_read_b64, kept as one 64-bit value (threshold or
// leaf value in the low half, w in the high half) so that the pair stays in one register pair. A
// relaxed atomic load cannot be split: plain loads of the record get split by the compiler into
// two 4-byte reads (the threshold half sunk past the wave-wide leaf test), doubling the LDS
// reads per step.
__device__ __forceinline__ uint64_t read_record(const unsigned char *p) {
    return __hip_atomic_load(reinterpret_cast<const uint64_t *>(p), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ uint32_t rec_thr(uint64_t r) { return uint32_t(r); }
__device__ __forceinline__ uint32_t rec_w(uint64_t r) { return uint32_t(r >> 32); }

// Child index of a narrow record plus the comparison bit, in two VALU ops: the compare writes
// VCC and an SDWA add-with-carry adds it to the high half-word of w. The s_nop covers the
// VALU-writes-VCC / VALU-reads-carry hazard (two wait states, as the compiler itself emits).
__device__ __forceinline__ uint32_t narrow_child(uint32_t w, float x, float thr) {
    uint32_t r;
    asm("v_cmp_ge_f32 vcc, %1, %2\n\t"
        "s_nop 1\n\t"
        "v_addc_co_u32_sdwa %0, vcc, %3, 0, vcc dst_sel:DWORD dst_unused:UNUSED_PAD "
        "src0_sel:WORD_1 src1_sel:DWORD"
        : "=v"(r)
        : "v"(x), "v"(thr), "v"(w)
        : "vcc");
    return r;
}

// The same for coded documents: unsigned compare of 16-bit codes.
__device__ __forceinline__ uint32_t narrow_child_coded(uint32_t w, uint32_t code, uint32_t q) {
    uint32_t r;
    asm("v_cmp_ge_u32 vcc, %1, %2\n\t"
        "s_nop 1\n\t"
        "v_addc_co_u32_sdwa %0, vcc, %3, 0, vcc dst_sel:DWORD dst_unused:UNUSED_PAD "
        "src0_sel:WORD_1 src1_sel:DWORD"
        : "=v"(r)
        : "v"(code), "v"(q), "v"(w)
        : "vcc");
    return r;
}

// Compact records: the side of the children pair {lo, hi} that a 4-byte record r sends a
// document to, whose staged value is x = code << 5 | 31: x >= the record's upper half is
// code >= threshold. Plain code: the compiler reads the upper half in place with an SDWA
// compare and places the compare-to-select wait states itself (filling them with the other
// trees' work).
__device__ __forceinline__ uint32_t compact_child(uint32_t x, uint32_t r, uint32_t lo, uint32_t hi) {
    return x >= (r >> 16) ? hi : lo;
}

template <int DL, int K, bool HALF, bool NARROW, bool CODED, int MODE, bool COMPACT>
// min waves per SIMD: 2 or 1 workgroups per CU (a feature trace holds a CU alone)
__global__ void __launch_bounds__(kThreads, HALF && MODE != kModeUsage ? 8 : 4)
score_kernel(const void *__restrict__ Xv, int64_t n_docs, int32_t n_features, int32_t n_cols,
             const uint2 *__restrict__ images, int32_t slot_recs,
             const uint32_t *__restrict__ tile_recs, int32_t n_tiles, int32_t head_blocks,
             int32_t tail_splits,
             int32_t xs_bytes, int32_t zero_rec, double *__restrict__ partials,
             float *__restrict__ scores, int32_t *__restrict__ leaf_ids,
             const int32_t *__restrict__ orig_id, const uint32_t *__restrict__ tree_node_off,
             const int32_t *__restrict__ tree_orig, int32_t n_trees,
             uint32_t *__restrict__ masks, int32_t mask_words, int32_t usage_off,
             const float4 *__restrict__ leaf_vec, int32_t vec_stride4, int32_t n_out,
             int32_t chunk, double out_scale, int32_t pk_recs, const uint2 *__restrict__ big,
             int32_t n_small, uint32_t big_off0, const uint32_t *__restrict__ cleaf,
             const int32_t *__restrict__ cleaf_id) {
    // Static allocation: the LDS base is address 0, so feature and node addresses need no add.
    // HALF = half a CU's LDS, so that two workgroups share a CU. CODED = documents arrive as
    // 16-bit threshold codes (rows of n_features codes) instead of floats. Layout:
    //   [0, xs_bytes)            document tile, [(n_cols + 1) x DL] values
    //   [xs_bytes, zero_rec)     tile slot: the current tile image (header, then node records);
    //                            after the last tile, the cross-walker reduction (1,024 doubles,
    //                            4 x 1,024 with vector-valued leaves)
    //   zero_rec (8 bytes)       all-zero self-linked leaf of value 0, for idle walker slots
    //                            (walker packets of one-workgroup plans fill the LDS from
    //                            xs_bytes up to a zero record of their own, passed here)
    //   usage_off                usage modes: word j of document lane dl's feature bitmask at
    //                            [j * DL + dl] (32 feature ids a word); in the slot past the
    //                            largest tile image when it fits there (kModeUsageSlot, two
    //                            workgroups per CU as for scoring), else past the 80 KB half of
    //                            two-workgroup plans (kModeUsage: the launch holds a CU alone)
    constexpr bool LEAVES = MODE == kModeLeaves;
    constexpr bool USAGE = MODE == kModeUsage || MODE == kModeUsageSlot;
    constexpr bool VEC = MODE == kModeVector;
    constexpr int kLds = HALF ? treeens::kLdsPerCu / 2 + (MODE == kModeUsage ? treeens::kUsageHalfBytes : 0)
                              : treeens::kLdsPerCu;
    __shared__ __align__(16) unsigned char lds[kLds];
    constexpr int kPre = HALF ? treeens::kPrefetchHalf : treeens::kPrefetchFull; // records per thread
    constexpr int kShift = NARROW ? 16 : treeens::kWideChildShift;
    uint2 *slot = reinterpret_cast<uint2 *>(lds + xs_bytes);
    const uint32_t *hdr = reinterpret_cast<const uint32_t *>(lds + xs_bytes);
    using Elem = std::conditional_t<CODED, uint16_t, float>;
    const Elem *X = reinterpret_cast<const Elem *>(Xv);
    Elem *xs = reinterpret_cast<Elem *>(lds);

    const int tid = threadIdx.x;
    const int nthr = kThreads;
    const int dl = tid & (DL - 1);
    // with 64-document blocks a walker is a whole wave: make that visible to the compiler so
    // the group loop is scalar
    const int walker = DL == 64 ? __builtin_amdgcn_readfirstlane(tid / DL) : tid / DL;
    const int n_walkers = nthr / DL;
    const uint32_t lane_off = uint32_t(dl) * uint32_t(sizeof(Elem));
    // a feature address is column * DL * sizeof(Elem) + lane offset (below DL * sizeof(Elem))
    constexpr int kColShift = __builtin_ctz(unsigned(DL * sizeof(Elem)));
    uint32_t *umask = reinterpret_cast<uint32_t *>(lds + usage_off);
    const int model_words = (n_cols + 31) / 32;

    const uint32_t col_mask =
        __builtin_amdgcn_readfirstlane(NARROW ? treeens::kNarrowColMask : treeens::kWideColMask);
    // column offsets below this are column 0 (NaN, or code 0), which only leaves name
    constexpr uint32_t kLeafCol = uint32_t(DL) * uint32_t(sizeof(Elem));
    // Workgroups [0, head_blocks) each walk all tiles for one document block; after them, each
    // remaining block is split over tail_splits workgroups that walk a contiguous share of the
    // tiles each and leave fp64 partial sums (the tail fills what would be a last, mostly idle
    // round of workgroups; small batches have no head at all).
    // After a head of whole rounds (a multiple of the XCD count), the splits of one tail block
    // are given workgroup indices of one residue mod kXcds: workgroups are dealt to the XCDs in
    // index order, so all splits of a block share one XCD's L2 and its document rows come from
    // HBM once. Indices past the last block (padding to whole XCD columns) exit at once.
    int64_t block = blockIdx.x;
    int split = 0, n_splits = 1;
    if (block >= head_blocks) {
        const int64_t t = block - head_blocks;
        if (head_blocks > 0) {
            const int64_t x = t % kXcds, r = t / kXcds;
            block = head_blocks + (r / tail_splits) * kXcds + x;
            split = int(r % tail_splits);
            if (block * DL >= n_docs)
                return;
        } else {
            block = head_blocks + t / tail_splits;
            split = int(t % tail_splits);
        }
        n_splits = tail_splits;
    }
    const int64_t doc0 = block * DL;
    const int t_lo = int((int64_t(n_tiles) * split) / n_splits);
    const int t_hi = int((int64_t(n_tiles) * (split + 1)) / n_splits);

    // Tile images are loaded into registers while the previous tile is walked, so the
    // global-memory latency of a tile load is hidden; the tile loop issues no scalar memory load
    // (those share a wait counter with LDS reads and would stall the walk).
    //  * HALF (two workgroups per CU, walk-bound): one tile in flight, its exact record count
    //    taken from the current tile's header.
    //  * full CU: two tiles in flight (one per register half), each a fixed window of
    //    kWin x kThreads records (the packer caps these tiles at that size and pads the images),
    //    loaded unconditionally so that the compiler counts the outstanding loads exactly.
    constexpr int kWin = treeens::kPrefetchFull / 2;
    constexpr int kDepth = HALF ? 1 : kPrefetchDepth; // tiles in flight
    constexpr int kPreA = kPre; // shared tiles of two-workgroup plans, or walker packets
    uint2 pa[kPreA], win[kDepth][HALF ? 1 : kWin];
    int cur_recs = 0;
    const int chunks = (slot_recs + kThreads - 1) / kThreads;
    auto fetch = [&](int ti, int n_rec) {
        const uint2 *src = images + int64_t(ti) * slot_recs;
#pragma unroll
        for (int j = 0; j < kPre; ++j) {
            const int i = tid + j * kThreads;
            if (i < n_rec)
                pa[j] = src[i];
        }
    };
    auto fetch_window = [&](uint2 (&dst)[kWin], int ti) {
        // unconditional: past the last tile it reloads that tile (exact wait counts)
        const uint2 *src = images + int64_t(min(ti, t_hi - 1)) * slot_recs + tid;
#pragma unroll
        for (int j = 0; j < kWin; ++j)
            dst[j] = src[(j < chunks ? j : 0) * kThreads];
    };
    // Walker packets (pk_recs > 0, plans of 64- or 32-document blocks): wave v's packet q is
    // images[(v * n_tiles + q) * pk_recs, ...), one part of pk_recs * DL / 64 records for each
    // of its walkers; each lane loads pk_recs / 64 records of it.
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int pk_lane = pk_recs / 64;
    // The loads are raw buffer loads: the packet's offset in a scalar register, each lane's
    // record offset in a vector register and the record's position in the instruction's
    // immediate, so no address arithmetic runs per packet (the packer keeps the packets below
    // 2 GiB).
    const __amdgpu_buffer_rsrc_t pk_rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint2 *>(images), 0, 0x7fffffff, 0x00020000);
    const int pk_lane_off = lane * 8;
    auto fetch_packet = [&](int q) {
        const int soff = (wave * n_tiles + q) * pk_recs * 8;
#pragma unroll
        for (int j = 0; j < kPre; ++j) {
            if (j < pk_lane) {
                const auto v = __builtin_amdgcn_raw_buffer_load_b64(pk_rsrc, pk_lane_off + j * 512, soff, 0);
                pa[j] = make_uint2(v[0], v[1]);
            }
        }
    };
    // Compact packets: kCompactPacketBytes per packet, one 8-byte row of 64 lanes per 512 bytes,
    // read with raw buffer loads as above.
    constexpr int kCpRows = treeens::kCompactPacketBytes / 512;
    auto fetch_compact = [&](int q) {
        const int soff = (wave * n_tiles + q) * treeens::kCompactPacketBytes;
#pragma unroll
        for (int j = 0; j < kCpRows; ++j) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(pk_rsrc, pk_lane_off + j * 512, soff, 0);
            pa[j] = make_uint2(v[0], v[1]);
        }
    };
    if constexpr (COMPACT) {
        if (t_lo < t_hi)
            fetch_compact(t_lo);
    } else if constexpr (HALF) {
        if (pk_recs > 0) {
            if (t_lo < t_hi)
                fetch_packet(t_lo);
        } else {
            cur_recs = t_lo < t_hi ? int(tile_recs[t_lo]) : 0;
            if (t_lo < t_hi)
                fetch(t_lo, cur_recs);
        }
    } else {
        if (pk_recs > 0) {
            if (t_lo < t_hi)
                fetch_packet(t_lo);
        } else if (t_lo < t_hi) {
#pragma unroll
            for (int d = 0; d < kDepth; ++d)
                fetch_window(win[d], t_lo + d);
        }
    }

    if constexpr (USAGE) {
        for (int i = tid; i < model_words * DL; i += kThreads)
            umask[i] = 0u;
    }
    // Stage the document tile: lane = document, so each LDS write is conflict-free (bank =
    // lane). The workgroup size is a multiple of DL, so a thread's document (and row) is fixed
    // and it takes every (kThreads / DL)-th group of columns. When rows are 16-byte aligned a
    // lane reads 16 bytes of its row at a time (4 floats or 8 codes: a quarter or an eighth of
    // the strided row reads), else one value. Loads are unconditional (clamped to the row) so
    // that a pass's loads are in flight together before any is written.
    {
        constexpr int kColStep = kThreads / DL;
        constexpr int kUnroll = 8;
        constexpr int kVec = 16 / int(sizeof(Elem)); // values per 16-byte load
        const int64_t doc = doc0 + dl;
        const bool live = doc < n_docs;
        const Elem *row = X + (live ? doc : n_docs - 1) * int64_t(n_features);
        // (compact packets: code 0 staged as 0 << 5 | 31)
        const Elem leaf_col = COMPACT ? Elem(31) : CODED ? Elem(0) : Elem(__builtin_nanf(""));
        if (tid < DL)
            xs[dl] = leaf_col;
        const bool vec = (n_features % kVec) == 0 && (reinterpret_cast<uintptr_t>(X) & 15u) == 0;
        if (vec) {
            const uint4 *row4 = reinterpret_cast<const uint4 *>(row);
            const int n_groups = (n_cols + kVec - 1) / kVec; // within the row: n_features % kVec == 0
            const int last = n_groups > 0 ? n_groups - 1 : 0;
            constexpr int kVecUnroll = 4;
            for (int q0 = tid / DL; q0 < n_groups; q0 += kColStep * kVecUnroll) {
                uint4 v[kVecUnroll];
#pragma unroll
                for (int u = 0; u < kVecUnroll; ++u)
                    v[u] = row4[min(q0 + u * kColStep, last)];
#pragma unroll
                for (int u = 0; u < kVecUnroll; ++u) {
                    const int q = q0 + u * kColStep;
                    if (q < n_groups) {
                        const Elem *e = reinterpret_cast<const Elem *>(&v[u]);
#pragma unroll
                        for (int k = 0; k < kVec; ++k) {
                            const int c = q * kVec + k + 1; // tile column of feature q * kVec + k
                            if (c <= n_cols)
                                xs[c * DL + dl] = live ? e[k] : Elem(0);
                        }
                    }
                }
            }
        } else {
            const int last = n_cols > 0 ? n_cols - 1 : 0;
            for (int c0 = tid / DL + 1; c0 <= n_cols; c0 += kColStep * kUnroll) {
                Elem v[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
                    v[u] = row[min(c0 + u * kColStep - 1, last)];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const int c = c0 + u * kColStep;
                    if (c <= n_cols)
                        xs[c * DL + dl] = live ? v[u] : Elem(0);
                }
            }
        }
    }
    if (!COMPACT && tid == 0) {
        // value 0 (as -0.0 for codes, whose leaves never hold zero bits; the all-zero row 0 of
        // the leaf-vector table for vector-valued leaves), column 0, self link
        const uint32_t thr = VEC ? 1u : CODED ? 0x80000000u : 0u;
        *reinterpret_cast<uint2 *>(lds + zero_rec) = make_uint2(thr, (uint32_t(zero_rec) / 8u) << kShift);
    }

    double acc = 0.0;
    double accv[kVecPerLaunch] = {0.0, 0.0, 0.0, 0.0};
    // Walk one group of K trees whose K root copies are the records at rc. tree_of(i) gives the
    // packed index of the tree in slot i (-1: an idle slot) and, for leaf ids, the LDS record
    // index of that tree's first record.
    auto walk_group = [&](const unsigned char *rc, auto complete_tag, int complete_depth, auto &&tree_of) {
        constexpr bool kComplete = decltype(complete_tag)::value;
        // the K root records (broadcast reads)
        uint64_t nd[K];
        if constexpr (K % 2 == 0) {
            // two roots per 16-byte read (a group's roots start 16-byte aligned when K is even)
#pragma unroll
            for (int i = 0; i < K; i += 2) {
                const uint4 r2 = *reinterpret_cast<const uint4 *>(rc + 8 * i);
                nd[i] = uint64_t(r2.x) | uint64_t(r2.y) << 32;
                nd[i + 1] = uint64_t(r2.z) | uint64_t(r2.w) << 32;
            }
        } else {
#pragma unroll
            for (int i = 0; i < K; ++i)
                nd[i] = read_record(rc + 8 * i);
        }
        // One predicated step: feature addresses fa from the records, read the features
        // xv, compare, child link + bit (the right child follows the left one), read
        // that record.
        uint32_t fa[K];
        std::conditional_t<CODED, uint32_t, float> xv[K];
        auto read_features = [&]() {
#pragma unroll
            for (int i = 0; i < K; ++i) {
                fa[i] = and_or(rec_w(nd[i]), col_mask, lane_off);
                if constexpr (CODED)
                    xv[i] = *reinterpret_cast<const uint16_t *>(lds + fa[i]);
                else
                    xv[i] = *reinterpret_cast<const float *>(lds + fa[i]);
                if constexpr (USAGE) {
                    // column c > 0 holds feature c - 1; column 0 is a leaf's (no
                    // comparison, nothing recorded)
                    const uint32_t col = fa[i] >> kColShift;
                    if (col > 0u)
                        atomicOr(&umask[((col - 1u) >> 5) * DL + dl], 1u << ((col - 1u) & 31u));
                }
            }
        };
        uint32_t addr[K]; // byte addresses of the records read by the last step
        auto descend = [&]() {
#pragma unroll
            for (int i = 0; i < K; ++i) {
                uint32_t child;
                const uint32_t w = rec_w(nd[i]), thr = rec_thr(nd[i]);
                if constexpr (CODED) {
                    if constexpr (NARROW)
                        child = narrow_child_coded(w, xv[i], thr);
                    else
                        child = (w >> kShift) + (xv[i] >= thr ? 1u : 0u);
                } else {
                    if constexpr (NARROW)
                        child = narrow_child(w, xv[i], __uint_as_float(thr));
                    else
                        child = (w >> kShift) + (xv[i] >= __uint_as_float(thr) ? 1u : 0u);
                }
                addr[i] = child * 8u;
            }
#pragma unroll
            for (int i = 0; i < K; ++i)
                nd[i] = read_record(lds + addr[i]);
        };
        if constexpr (kComplete) {
            // every path has the same length: no leaf test needed
            for (int s = 0; s < complete_depth; ++s) {
                read_features();
                descend();
            }
        } else {
            // Every lane steps until all lanes of the wave sit on leaves (a leaf's
            // feature address is the NaN column, below kLeafCol); the record that shows
            // a lane is at a leaf holds the leaf's value. Every path of a validated tree
            // reaches a leaf and leaves link to themselves, so the exit is always taken.
            // The next feature reads are issued before the test, so the test overlaps
            // their latency (after the last step they read the NaN column: harmless).
            auto any_internal = [&]() {
                bool internal = false;
#pragma unroll
                for (int i = 0; i < K; ++i)
                    internal |= fa[i] >= kLeafCol;
                return __builtin_amdgcn_ballot_w64(internal) != 0;
            };
            // Trees sit in the packed order longest expected lockstep walk first, so the
            // group's first tree usually ends last: step while its lanes are not all on
            // leaves (one compare per step), then while any of the K trees is not (the full
            // test, rarely true by then). The first step is taken untested: a group whose K
            // roots are all leaves (single-leaf trees, idle slots) is rare, and a leaf absorbs
            // the extra step.
            auto lead_internal = [&]() {
                return __builtin_amdgcn_ballot_w64(fa[0] >= kLeafCol) != 0;
            };
            read_features();
            for (;;) {
                descend();
                read_features();
                if (!lead_internal() && (K == 1 || !any_internal()))
                    break;
            }
            // The exit path "uses" the last feature reads, so the compiler cannot sink
            // them below the test (where they would serialise with it again).
#pragma unroll
            for (int i = 0; i < K; ++i)
                asm volatile("" ::"v"(xv[i]));
        }
        if constexpr (LEAVES) {
            const int64_t doc = doc0 + dl;
#pragma unroll
            for (int i = 0; i < K; ++i) {
                // a leaf's link is its own LDS record index; minus that of its tree's
                // first record, it is the leaf's position in the tree
                const int2 tr = tree_of(i);
                if (tr.x >= 0 && doc < n_docs) {
                    const int gt = tr.x;
                    // complete trees: the leaf's record index is the address the last step
                    // read (their leaf records carry no link); else the leaf's own link
                    const uint32_t rec = kComplete ? (complete_depth > 0 ? addr[i] / 8u : uint32_t(tr.y))
                                                   : rec_w(nd[i]) >> kShift;
                    const uint32_t self = rec - uint32_t(tr.y);
                    leaf_ids[doc * n_trees + tree_orig[gt]] = orig_id[tree_node_off[gt] + self];
                }
            }
        } else if constexpr (VEC) {
            // a leaf's threshold slot holds its table row + 1 (idle slots: row 0, zeros);
            // each component added to its double accumulator in tree order
#pragma unroll
            for (int i = 0; i < K; ++i) {
                const float4 v = leaf_vec[int64_t(rec_thr(nd[i]) - 1u) * vec_stride4 + chunk];
                accv[0] += double(v.x);
                accv[1] += double(v.y);
                accv[2] += double(v.z);
                accv[3] += double(v.w);
            }
        } else if constexpr (!USAGE) {
            // the K leaf values, each added to the double accumulator in tree order (a
            // float sum of the group first can miss the tolerance when a score cancels
            // near zero); idle slots hold the zero record. Complete trees' leaf records hold
            // the value as a double (tiles and packets with an idle slot are never complete).
#pragma unroll
            for (int i = 0; i < K; ++i) {
                if constexpr (kComplete)
                    acc += __longlong_as_double(static_cast<long long>(nd[i]));
                else
                    acc += double(__uint_as_float(rec_thr(nd[i])));
            }
        }
    };
    // Walk the tile image in the LDS slot: walker w takes groups w, w + n_walkers, ... of K
    // consecutive trees (the packer sizes tiles to a multiple of n_walkers * K trees where it
    // can, and pads the header's root copies to a multiple of K with the zero record).
    auto walk_tile = [&]() {
        const uint4 h = *reinterpret_cast<const uint4 *>(hdr);
        const int ntr = __builtin_amdgcn_readfirstlane(int(h.x));
        const int complete_depth = __builtin_amdgcn_readfirstlane(int(h.y));
        const int tree_begin = __builtin_amdgcn_readfirstlane(int(h.z));
        const int n_groups = (ntr + K - 1) / K;
        // records of the tile's trees start after the fixed header words and the root copies
        const uint32_t rec0 = uint32_t(xs_bytes) / 8u + uint32_t(treeens::kHeaderFixedWords / 2 + n_groups * K);
        auto walk_groups = [&](auto complete_tag) {
            for (int g = walker; g < n_groups; g += n_walkers) {
                const unsigned char *rc = lds + xs_bytes + 8 * (treeens::kHeaderFixedWords / 2 + g * K);
                auto tree_of = [&](int i) {
                    const int t = g * K + i;
                    return t < ntr ? make_int2(tree_begin + t,
                                               int(rec0 + tree_node_off[tree_begin + t] - tree_node_off[tree_begin]))
                                   : make_int2(-1, 0);
                };
                walk_group(rc, complete_tag, complete_depth, tree_of);
            }
        };
        // the branch on the tile's complete depth outside the group loop, so that each loop
        // keeps its records in the registers it reads them into
        if (complete_depth >= 0)
            walk_groups(std::true_type{});
        else
            walk_groups(std::false_type{});
    };
    // Walk one of this walker's packets in its sub-slot, which starts at LDS record base: its
    // groups are first_group, first_group + n_walkers, ...
    auto walk_packet = [&](uint32_t base) {
        const uint2 h0 = *reinterpret_cast<const uint2 *>(lds + 8 * base);
        const uint2 h1 = *reinterpret_cast<const uint2 *>(lds + 8 * (base + 1));
        const int ng = __builtin_amdgcn_readfirstlane(int(h0.x));
        const int complete_depth = __builtin_amdgcn_readfirstlane(int(h0.y));
        // group count and complete depth are common to the walkers of a wave; first groups not
        const int first_group = DL == 64 ? __builtin_amdgcn_readfirstlane(int(h1.x)) : int(h1.x);
        const uint16_t *first_rec =
            reinterpret_cast<const uint16_t *>(lds + 8 * (base + treeens::kPacketHeaderRecs + ng * K));
        auto walk_groups = [&](auto complete_tag) {
            for (int j = 0; j < ng; ++j) {
                const unsigned char *rc = lds + 8 * (base + treeens::kPacketHeaderRecs + j * K);
                auto tree_of = [&](int i) {
                    const int gt = (first_group + j * n_walkers) * K + i;
                    return gt < n_small ? make_int2(gt, int(first_rec[j * K + i])) : make_int2(-1, 0);
                };
                walk_group(rc, complete_tag, complete_depth, tree_of);
            }
        };
        // as in walk_tile, the branch on the complete depth outside the group loop
        if (complete_depth >= 0)
            walk_groups(std::true_type{});
        else
            walk_groups(std::false_type{});
    };
    // Each walker streams its own packets through its own sub-slot: no barrier between packets,
    // so a walker never waits for the slowest one of a tile.
    auto walk_packets = [&]() {
        const uint32_t my_base = uint32_t(xs_bytes) / 8u + uint32_t(wave * pk_recs);
        uint2 *my = reinterpret_cast<uint2 *>(lds) + my_base;
        // this walker's part of the wave's sub-slot
        const uint32_t part_base = my_base + uint32_t(DL == 64 ? 0 : (lane / DL) * (pk_recs * DL / 64));
        __syncthreads(); // the document tile and the zero record are written
        for (int q = t_lo; q < t_hi; ++q) {
            // this packet's records (and, before the first, the document rows) have landed
            __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
#pragma unroll
            for (int j = 0; j < kPre; ++j)
                if (j < pk_lane)
                    my[lane + j * 64] = pa[j];
            // the wave's own writes complete before it reads the packet back
            __builtin_amdgcn_s_waitcnt(kWaitLgkmcnt0);
            if (q + 1 < t_hi)
                fetch_packet(q + 1);
            walk_packet(part_base);
        }
    };
    // Compact packets (4-byte records): wave v owns K windows of kCompactWindowBytes / K bytes past
    // the document tile; the packet's header row stays in registers. A step reads the lane's staged value and
    // the current record's whole children pair together (one dependent LDS round trip) and keeps
    // the side the comparison picks. Leaves hold no value: the leaf's position in its window
    // locates its payload (value bits, leaf-vector row + 1 or input node id) in arrays shaped
    // like the packets in device memory. Scores add each group's payloads after the next group
    // is walked, so their loads have a whole walk to land (the sum keeps tree order).
    auto walk_compact = [&]() {
        if constexpr (COMPACT) {
            constexpr uint32_t kCpWin = treeens::kCompactWindowBytes / K;
            static_assert(K == treeens::kCompactTrees && kCpWin == 2048, "compact windows of 2 KiB");
            const uint32_t cw = (uint32_t(xs_bytes) + 2047u) & ~2047u;
            const uint32_t my_win = cw + uint32_t(wave) * treeens::kCompactWindowBytes;
            const __amdgpu_buffer_rsrc_t leaf_rsrc =
                __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t *>(cleaf), 0, 0x7fffffff, 0x00020000);
            const __amdgpu_buffer_rsrc_t id_rsrc =
                __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t *>(cleaf_id), 0, 0x7fffffff, 0x00020000);
            // the column field moved to a feature address (column * DL * 2 bytes), the pair offset
            const uint32_t col_sel = __builtin_amdgcn_readfirstlane(0x1FF80u);
            const uint32_t pair_sel = __builtin_amdgcn_readfirstlane(0x7F8u);
            // window bases (aligned to the window size: OR adds the pair offset), held in vector
            // registers for the whole walk (opaque to the compiler, which would otherwise copy
            // one from a scalar register at every step)
            uint32_t tb[K];
#pragma unroll
            for (int i = 0; i < K; ++i)
                asm volatile("v_mov_b32 %0, %1" : "=v"(tb[i]) : "s"(my_win + uint32_t(i) * kCpWin));
            uint32_t pend[K]; // leaf payloads of the last group walked (scores)
#pragma unroll
            for (int i = 0; i < K; ++i)
                pend[i] = 0u;
            if constexpr (MODE == kModeScore) {
                // Loads of the zero pairs' payloads (0.0) before the first packet, so that every
                // packet's copy finds K payload loads issued after its rows, as on later packets.
                if (t_lo < t_hi) {
                    const int soff = (wave * n_tiles + t_lo) * treeens::kCompactPacketBytes;
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        pend[i] = __builtin_amdgcn_raw_buffer_load_b32(leaf_rsrc, i * kCpWin + kCpWin - 8, soff, 0);
                }
            }
            __syncthreads(); // the document tile is written
            for (int q = t_lo; q < t_hi; ++q) {
                const int soff = (wave * n_tiles + q) * treeens::kCompactPacketBytes;
                // this packet's rows have landed (the last group's payload loads may not have)
                __builtin_amdgcn_s_waitcnt(MODE == kModeScore ? kWaitVmcnt0 | K : kWaitVmcnt0);
#pragma unroll
                for (int j = 0; j < kCpRows - 1; ++j)
                    *reinterpret_cast<uint2 *>(lds + my_win + uint32_t(j) * 512u + uint32_t(pk_lane_off)) = pa[j];
                // The header row stays in registers (lane l holds header words 2l and 2l + 1):
                // its fields and the groups' roots are read from there with v_readlane.
                const uint2 hrow = pa[kCpRows - 1];
                // the wave's own writes complete before it reads the packet back
                __builtin_amdgcn_s_waitcnt(kWaitLgkmcnt0);
                // the next packet (the last one again after the last: the loads stay
                // unconditional, so the compiler counts them exactly when it waits for payloads)
                fetch_compact(min(q + 1, t_hi - 1));
                const int ng = __builtin_amdgcn_readlane(int(hrow.x), 0);
                const int complete_depth = __builtin_amdgcn_readlane(int(hrow.y), 0);
                const int first_group = __builtin_amdgcn_readlane(int(hrow.x), 1);
                auto walk_groups = [&](auto complete_tag) {
                    constexpr bool kComplete = decltype(complete_tag)::value;
                    for (int j = 0; j < ng; ++j) {
                        // group j's roots: header words 4 + 2j and 5 + 2j, lane 2 + j
                        static_assert(treeens::kCompactHeaderWords == 4 && K == 2, "root lane");
                        uint32_t r[K];
                        r[0] = uint32_t(__builtin_amdgcn_readlane(int(hrow.x), 2 + j));
                        r[1] = uint32_t(__builtin_amdgcn_readlane(int(hrow.y), 2 + j));
                        uint32_t fa[K], xv[K], lo[K], hi[K];
                        auto issue = [&]() {
#pragma unroll
                            for (int i = 0; i < K; ++i) {
                                fa[i] = and_or(r[i] >> 4, col_sel, lane_off);
                                const uint32_t pa_i = and_or(r[i], pair_sel, tb[i]);
                                xv[i] = *reinterpret_cast<const uint16_t *>(lds + fa[i]);
                                const uint64_t pr = read_record(lds + pa_i);
                                lo[i] = uint32_t(pr);
                                hi[i] = uint32_t(pr >> 32);
                            }
                        };
                        auto select = [&]() {
#pragma unroll
                            for (int i = 0; i < K; ++i)
                                r[i] = compact_child(xv[i], r[i], lo[i], hi[i]);
                        };
                        if constexpr (kComplete) {
                            for (int s = 0; s < complete_depth; ++s) {
                                issue();
                                select();
                            }
                        } else {
                            // as in walk_group: the first step untested, then step until the lead
                            // tree's lanes, then all K trees' lanes, sit on leaves (column 0); the
                            // next reads are issued before the test
                            issue();
                            for (;;) {
                                select();
                                issue();
                                if (__builtin_amdgcn_ballot_w64(fa[0] >= kLeafCol) == 0) {
                                    bool internal = false;
#pragma unroll
                                    for (int i = 1; i < K; ++i)
                                        internal |= fa[i] >= kLeafCol;
                                    if (__builtin_amdgcn_ballot_w64(internal) == 0)
                                        break;
                                }
                            }
#pragma unroll
                            for (int i = 0; i < K; ++i)
                                asm volatile("" ::"v"(xv[i]), "v"(lo[i]), "v"(hi[i]));
                        }
                        // byte offset of each leaf's payload in the packet
                        uint32_t voff[K];
#pragma unroll
                        for (int i = 0; i < K; ++i)
                            voff[i] = (r[i] & 0x7FCu) + uint32_t(i) * kCpWin;
                        if constexpr (MODE == kModeScore) {
#pragma unroll
                            for (int i = 0; i < K; ++i)
                                acc += double(__uint_as_float(pend[i]));
#pragma unroll
                            for (int i = 0; i < K; ++i)
                                pend[i] = __builtin_amdgcn_raw_buffer_load_b32(leaf_rsrc, voff[i], soff, 0);
                        } else if constexpr (LEAVES) {
                            const int64_t doc = doc0 + dl;
#pragma unroll
                            for (int i = 0; i < K; ++i) {
                                const int gt = (first_group + j * treeens::kPacketWalkers) * K + i;
                                if (gt < n_trees && doc < n_docs)
                                    leaf_ids[doc * n_trees + tree_orig[gt]] =
                                        __builtin_amdgcn_raw_buffer_load_b32(id_rsrc, voff[i], soff, 0);
                            }
                        } else if constexpr (VEC) {
#pragma unroll
                            for (int i = 0; i < K; ++i) {
                                const uint32_t row = __builtin_amdgcn_raw_buffer_load_b32(leaf_rsrc, voff[i], soff, 0);
                                const float4 v = leaf_vec[int64_t(row - 1u) * vec_stride4 + chunk];
                                accv[0] += double(v.x);
                                accv[1] += double(v.y);
                                accv[2] += double(v.z);
                                accv[3] += double(v.w);
                            }
                        }
                    }
                };
                if (complete_depth >= 0)
                    walk_groups(std::true_type{});
                else
                    walk_groups(std::false_type{});
            }
            if constexpr (MODE == kModeScore) {
#pragma unroll
                for (int i = 0; i < K; ++i)
                    acc += double(__uint_as_float(pend[i]));
            }
        }
    };
    if constexpr (COMPACT) {
        walk_compact();
    } else if constexpr (HALF) {
        if (pk_recs > 0)
            walk_packets();
        else
        for (int ti = t_lo; ti < t_hi; ++ti) {
            __syncthreads(); // the previous tile is fully walked (and the document tile written)
            // All outstanding global loads (this tile's records, and the document rows before
            // the first tile) land here, unconditionally: otherwise the compiler cannot prove
            // them complete on every path and waits for them again inside the walk.
            __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
#pragma unroll
            for (int j = 0; j < kPre; ++j) {
                const int i = tid + j * kThreads;
                if (i < cur_recs)
                    slot[i] = pa[j];
            }
            __syncthreads();
            cur_recs = __builtin_amdgcn_readfirstlane(int(hdr[3])); // the next tile's size
            if (ti + 1 < t_hi)
                fetch(ti + 1, cur_recs);
            walk_tile();
        }
    } else if (pk_recs > 0) {
        walk_packets();
    } else {
        // the document rows (loaded after the first two tiles) land before the first barrier
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        // windows are written as whole 1,024-record chunks: the packer sizes the slot of these
        // plans to whole chunks, so the zero record and the trace's bitmasks after it are safe
        auto write_window = [&](const uint2 (&src)[kWin]) {
#pragma unroll
            for (int j = 0; j < kWin; ++j)
                if (j < chunks)
                    slot[tid + j * kThreads] = src[j];
        };
        for (int ti = t_lo; ti < t_hi; ti += kDepth) {
#pragma unroll
            for (int d = 0; d < kDepth; ++d) {
                __syncthreads(); // the previous tile is fully walked (and the document tile written)
                write_window(win[d]);
                __syncthreads();
                fetch_window(win[d], ti + d + kDepth);
                if (d == 0 || ti + d < t_hi)
                    walk_tile();
            }
        }
    }
    // Big trees (too large for a tile; packed after the tiled ones): walked from device memory,
    // one tree per walker at a time, the records staying in L2. A record is {thr, w} with
    // w = (tree-relative left child << 16) | column index; the features come from the LDS
    // document tile as for every other tree, and leaves absorb further steps (column 0). Big
    // tree b goes to split b % n_splits and, within it, to walker (b / n_splits) % n_walkers.
    if (!COMPACT && n_small < n_trees) {
        __syncthreads(); // the document tile is written (no tile may have been walked)
        const int n_big = n_trees - n_small;
        for (int b = split + n_splits * walker; b < n_big; b += n_splits * n_walkers) {
            const int gt = n_small + b;
            const uint2 *tr = big + (tree_node_off[gt] - big_off0);
            uint2 r = tr[0];
            for (;;) {
                const uint32_t fa = ((r.y & treeens::kBigColMask) << kColShift) | lane_off;
                const Elem x = *reinterpret_cast<const Elem *>(lds + fa);
                if constexpr (USAGE) {
                    const uint32_t col = r.y & treeens::kBigColMask;
                    if (col > 0u)
                        atomicOr(&umask[((col - 1u) >> 5) * DL + dl], 1u << ((col - 1u) & 31u));
                }
                if (__builtin_amdgcn_ballot_w64(fa >= kLeafCol) == 0)
                    break;
                bool right;
                if constexpr (CODED)
                    right = uint32_t(x) >= r.x;
                else
                    right = x >= __uint_as_float(r.x);
                r = tr[(r.y >> treeens::kBigLinkShift) + (right ? 1u : 0u)];
            }
            if constexpr (LEAVES) {
                const int64_t doc = doc0 + dl;
                if (doc < n_docs)
                    leaf_ids[doc * n_trees + tree_orig[gt]] =
                        orig_id[tree_node_off[gt] + (r.y >> treeens::kBigLinkShift)];
            } else if constexpr (VEC) {
                const float4 v = leaf_vec[int64_t(r.x - 1u) * vec_stride4 + chunk];
                accv[0] += double(v.x);
                accv[1] += double(v.y);
                accv[2] += double(v.z);
                accv[3] += double(v.w);
            } else if constexpr (!USAGE) {
                acc += double(__uint_as_float(r.x));
            }
        }
    }
    if constexpr (USAGE) {
        __syncthreads();
        // rows of mask_words words (>= model_words; the words past the model's are zero)
        const int64_t n_here = min<int64_t>(DL, n_docs - doc0);
        if (masks) {
            for (int e = tid; e < n_here * mask_words; e += kThreads) {
                const int d = e / mask_words, j = e - d * mask_words;
                masks[(doc0 + d) * mask_words + j] = j < model_words ? umask[j * DL + d] : 0u;
            }
        }
        if (walker == 0 && dl < n_here) {
            int count = 0;
            for (int j = 0; j < model_words; ++j)
                count += __popc(umask[j * DL + dl]);
            leaf_ids[doc0 + dl] = count;
        }
    }
    if constexpr (VEC) {
        __syncthreads();
        double *red = reinterpret_cast<double *>(lds + xs_bytes); // 4 x 1,024 doubles (32 KiB)
#pragma unroll
        for (int c = 0; c < kVecPerLaunch; ++c)
            red[(c * n_walkers + walker) * DL + dl] = accv[c];
        __syncthreads();
        if (walker == 0) {
            const int64_t doc = doc0 + dl;
            for (int c = 0; c < kVecPerLaunch; ++c) {
                double sum = 0.0;
                for (int w = 0; w < n_walkers; ++w)
                    sum += red[(c * n_walkers + w) * DL + dl];
                const int oc = kVecPerLaunch * chunk + c;
                if (doc < n_docs) {
                    if (n_splits == 1) {
                        if (oc < n_out)
                            scores[doc * n_out + oc] = float(sum * out_scale);
                    } else {
                        const int64_t tail0 = int64_t(head_blocks) * DL;
                        partials[(int64_t(split) * (n_docs - tail0) + (doc - tail0)) * kVecPerLaunch + c] = sum;
                    }
                }
            }
        }
    }
    if constexpr (MODE == kModeScore) {
        __syncthreads();
        double *red = reinterpret_cast<double *>(lds + xs_bytes);
        red[walker * DL + dl] = acc;
        __syncthreads();
        if (walker == 0) {
            const int64_t doc = doc0 + dl;
            double sum = 0.0;
            for (int w = 0; w < n_walkers; ++w)
                sum += red[w * DL + dl];
            if (doc < n_docs) {
                if (n_splits == 1) {
                    scores[doc] = float(sum * out_scale);
                } else {
                    const int64_t tail0 = int64_t(head_blocks) * DL;
                    partials[int64_t(split) * (n_docs - tail0) + (doc - tail0)] = sum;
                }
            }
        }
    }
}

// Sum of the split partials of each entry in a fixed order (so the rounding never changes).
// Entry j is component j % comps of document j / comps; it goes to output column
// c_base + j % comps of a row of n_out scores (if that column exists), scaled by out_scale.
// Few splits: one thread per entry, in split order. Many splits (small batches): one wave per
// entry, lanes interleave the splits, then a fixed butterfly.
struct ReduceOut {
    float *scores;
    int32_t comps, n_out, c_base;
    double scale;
    __device__ void store(int64_t j, double s) const {
        const int64_t doc = j / comps;
        const int c = c_base + int(j - doc * comps);
        if (c < n_out)
            scores[doc * n_out + c] = float(s * scale);
    }
};

__global__ void reduce_partials_thread_kernel(const double *__restrict__ partials, int32_t n_splits,
                                              int64_t n_docs, ReduceOut out) {
    const int64_t d = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (d < n_docs) {
        // eight independent loads in flight, then summed in split order
        double s = 0.0;
        int k = 0;
        for (; k + 8 <= n_splits; k += 8) {
            double v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                v[u] = partials[int64_t(k + u) * n_docs + d];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                s += v[u];
        }
        for (; k < n_splits; ++k)
            s += partials[int64_t(k) * n_docs + d];
        out.store(d, s);
    }
}

__global__ void __launch_bounds__(64)
reduce_partials_wave_kernel(const double *__restrict__ partials, int32_t n_splits, int64_t n_docs,
                            ReduceOut out) {
    const int64_t d = blockIdx.x;
    double s = 0.0;
    for (int k = threadIdx.x; k < n_splits; k += 64)
        s += partials[int64_t(k) * n_docs + d];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        s += __shfl_xor(s, off);
    if (threadIdx.x == 0)
        out.store(d, s);
}

__global__ void fill_zero_kernel(float *__restrict__ scores, int64_t n) {
    const int64_t d = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (d < n)
        scores[d] = 0.0f;
}

// Threshold codes of a block of documents for a chunk of features: code_f(x) is the number of
// f's sorted distinct thresholds t with x >= t (a NaN x compares false everywhere and gets 0).
// The chunk's search tables are staged in LDS: feature j's 2^s - 1 entries hold its list as a
// complete search tree in breadth-first order (slot i at entry i - 1), padded with NaN (which
// never compares true), so the count is s steps of i = 2i + (x >= slot i) from i = 1, the same
// for every lane, and code = i - 2^s. Thread e takes elements e, e + 1,024, ... of the block's [doc][feature] order,
// stepping its (document, feature) pair without a division. Output rows hold n_cols 16-bit
// codes, each stored as code << code_shift with the shifted-out bits set (code_shift 5 for the
// compact records' comparison, else 0).
constexpr int kCodeThreads = 1024;
// One step of the search: 2i + (x >= t) as a compare into VCC and an add-with-carry of i to
// itself (two VALU ops; the s_nop as in narrow_child).
__device__ __forceinline__ uint32_t search_step(uint32_t i, float x, float t) {
    uint32_t r;
    asm("v_cmp_ge_f32 vcc, %1, %2\n\t"
        "s_nop 1\n\t"
        "v_addc_co_u32 %0, vcc, %3, %3, vcc"
        : "=v"(r)
        : "v"(x), "v"(t), "v"(i)
        : "vcc");
    return r;
}
__global__ void __launch_bounds__(kCodeThreads)
code_kernel(const float *__restrict__ X, int64_t n_docs, int32_t n_features, int32_t n_cols,
            int32_t docs_per_wg, const float *__restrict__ table,
            const treeens::CodeChunk *__restrict__ chunks, int32_t n_chunks, int32_t code_shift,
            uint16_t *__restrict__ codes) {
    __shared__ float tab[treeens::kCodeTableFloats];
    // Workgroups are dealt to the XCDs in index order: index L runs chunk (L % (8C)) / 8 of
    // document block (L / (8C)) * 8 + L % 8, so all C chunks of a block share one XCD and run
    // one after another there, and the cache lines of a row that two neighbouring chunks
    // share come from HBM once.
    const int64_t L = blockIdx.x;
    const int64_t per = int64_t(kXcds) * n_chunks;
    const int chunk = int((L % per) / kXcds);
    const int64_t block = (L / per) * kXcds + L % kXcds;
    if (block * docs_per_wg >= n_docs)
        return;
    const treeens::CodeChunk ch = chunks[chunk];
    const int nf = ch.f_end - ch.f_begin;
    const int steps = ch.search_steps;
    for (int i = threadIdx.x; i < ch.table_end - ch.table_begin; i += kCodeThreads)
        tab[i] = table[ch.table_begin + i];
    __syncthreads();
    const int64_t d0 = block * docs_per_wg;
    const int n = int(min<int64_t>(docs_per_wg, n_docs - d0)) * nf;
    // nf <= 256: every step moves at least 4 documents on
    const int step_d = kCodeThreads / nf, step_j = kCodeThreads - step_d * nf;
    int d = int(threadIdx.x) / nf, j = int(threadIdx.x) - d * nf;
    const uint32_t leaf0 = 1u << steps;
    // kCodeBatch elements per thread at a time: their feature values load together, then their
    // searches interleave (independent LDS round trips in flight)
    constexpr int kCodeBatch = 4;
    for (int e0 = threadIdx.x; e0 < n; e0 += kCodeBatch * kCodeThreads) {
        float x[kCodeBatch];
        int64_t at[kCodeBatch];
        int t0[kCodeBatch];
        uint32_t i[kCodeBatch];
#pragma unroll
        for (int u = 0; u < kCodeBatch; ++u) {
            const bool live = e0 + u * kCodeThreads < n;
            const int64_t doc = d0 + d;
            at[u] = live ? doc * n_cols + ch.f_begin + j : -1;
            x[u] = live ? X[doc * n_features + ch.f_begin + j] : 0.0f;
            t0[u] = j * int(leaf0 - 1u) - 1; // slot i of feature j is tab[t0 + i]
            i[u] = 1u;
            d += step_d;
            j += step_j;
            if (j >= nf) {
                j -= nf;
                ++d;
            }
        }
        for (int s = 0; s < steps; ++s) {
#pragma unroll
            for (int u = 0; u < kCodeBatch; ++u)
                i[u] = search_step(i[u], x[u], tab[t0[u] + int(i[u])]);
        }
#pragma unroll
        for (int u = 0; u < kCodeBatch; ++u) {
            const uint32_t code = i[u] - leaf0;
            if (at[u] >= 0)
                codes[at[u]] = uint16_t((code << code_shift) | ((1u << code_shift) - 1u));
        }
    }
}

using ScoreFn = void (*)(const void *, int64_t, int32_t, int32_t, const uint2 *, int32_t,
                         const uint32_t *, int32_t, int32_t, int32_t, int32_t, int32_t, double *,
                         float *, int32_t *, const int32_t *, const uint32_t *, const int32_t *,
                         int32_t, uint32_t *, int32_t, int32_t, const float4 *, int32_t,
                         int32_t, int32_t, double, int32_t, const uint2 *, int32_t, uint32_t,
                         const uint32_t *, const int32_t *);

template <int DL, bool HALF, bool NARROW, bool CODED, int MODE>
ScoreFn pick_k(int k) {
    switch (k) {
    case 1: return score_kernel<DL, 1, HALF, NARROW, CODED, MODE, false>;
    case 2: return score_kernel<DL, 2, HALF, NARROW, CODED, MODE, false>;
    case 4: return score_kernel<DL, 4, HALF, NARROW, CODED, MODE, false>;
    default: return nullptr;
    }
}

template <bool NARROW, bool CODED, int MODE>
ScoreFn pick_dl(const treeens::LdsPlan &p) {
    if (p.lds_bytes == treeens::kLdsPerCu / 2) {
        // two workgroups per CU: only small float tiles of 64-document blocks
        if constexpr (CODED)
            return nullptr;
        else
            return p.docs_per_block == 64 ? pick_k<64, true, NARROW, false, MODE>(p.interleave) : nullptr;
    }
    if constexpr (MODE == kModeUsageSlot)
        return nullptr; // one-workgroup plans keep room for the bitmasks after the zero record
    else
    switch (p.docs_per_block) {
    case 64: return pick_k<64, false, NARROW, CODED, MODE>(p.interleave);
    case 32: return pick_k<32, false, NARROW, CODED, MODE>(p.interleave);
    case 16: return pick_k<16, false, NARROW, CODED, MODE>(p.interleave);
    case 8: return pick_k<8, false, NARROW, CODED, MODE>(p.interleave);
    default: return nullptr;
    }
}

template <int MODE>
ScoreFn pick_kernel(const treeens::LdsPlan &p, bool compact) {
    if (compact) {
        // compact packets: coded 64-document blocks, one workgroup per CU (not the trace)
        if constexpr (MODE == kModeScore || MODE == kModeLeaves || MODE == kModeVector)
            return p.coded && p.docs_per_block == 64 && p.lds_bytes == treeens::kLdsPerCu
                       ? score_kernel<64, treeens::kCompactTrees, false, false, true, MODE, true>
                       : nullptr;
        else
            return nullptr;
    }
    if (p.lds_bytes != treeens::kLdsPerCu / 2 && p.lds_bytes != treeens::kLdsPerCu)
        return nullptr;
    if (p.coded)
        return p.narrow ? pick_dl<true, true, MODE>(p) : pick_dl<false, true, MODE>(p);
    return p.narrow ? pick_dl<true, false, MODE>(p) : pick_dl<false, false, MODE>(p);
}

} // namespace

namespace treeens {
int set_error(int code, const std::string &message) {
    g_err = message;
    return code;
}
void clear_error() { g_err.clear(); }
} // namespace treeens

// ------------------------------------------------------------------------------------------
// handle
// ------------------------------------------------------------------------------------------
struct tree_ens {
    int device = 0;
    int32_t n_trees = 0;
    int32_t n_cols = 0;
    int32_t max_depth = 0;
    int64_t n_nodes = 0;
    treeens::LdsPlan plan{};
    int32_t level_begin[treeens::kTileLevels + 1] = {};
    int32_t level_max_rounds[treeens::kTileLevels] = {}; // walker rounds of the fullest tile
    int64_t total_rounds = 0;                            // walker rounds of all tiles, tiling 0
    int32_t usage_slot_off = -1; // feature-trace bitmasks in the tile slot (two-workgroup plans)
    int64_t level_image_off[treeens::kTileLevels] = {};
    int32_t level_slot_recs[treeens::kTileLevels] = {};
    uint2 *d_images = nullptr;      // tile images of every tiling
    uint32_t *d_tile_recs = nullptr; // records of each tile image
    // walker packets (plans of 64- and 32-document blocks): records per sub-slot (0: the plan
    // walks shared tiles), the packets' zero record, packets per wave, the planner's rounds,
    // and the images
    int32_t pk_recs = 0;
    int32_t pk_zero_rec = 0;
    int32_t pk_per_walker = 0;
    int32_t pk_max_groups = 0;
    int64_t pk_total_rounds = 0;
    uint2 *d_packets = nullptr;
    // compact packets (coded 64-document plans; in place of the packets above for scores, leaf
    // ids and vector-valued leaves): trees per lane (0: none), packets per wave, the planner's
    // figures, the packets, and the leaf payloads and input node ids at the leaves' positions
    int32_t cp_k = 0;
    int32_t cp_per_walker = 0;
    int32_t cp_max_groups = 0;
    int64_t cp_total_rounds = 0;
    uint32_t *d_cpackets = nullptr;
    uint32_t *d_cleaf = nullptr;
    int32_t *d_cleaf_id = nullptr;
    // big trees (packed indices [n_small, n_trees)): their records in the big-tree format, the
    // first at packed node offset big_off0
    int32_t n_small = 0;
    uint32_t big_off0 = 0;
    uint2 *d_big = nullptr;
    // leaf-id output: packed tree -> input tree, packed node -> input node id
    uint32_t *d_tree_node_off = nullptr;
    int32_t *d_tree_orig = nullptr;
    int32_t *d_orig_id = nullptr;
    // vector-valued leaves and bagging: outputs per document, the table of leaf rows, and the
    // factor 1 / n_bags applied to every sum
    int32_t n_outputs = 1;
    int32_t n_bags = 1;
    int32_t vec_stride = 0;
    float *d_leaf_vec = nullptr;
    // coded models
    float *d_code_search = nullptr; // the coding chunks' search tables
    treeens::CodeChunk *d_code_chunks = nullptr;
    int32_t n_code_chunks = 0;
    // kernel specialised for the model (TREE_ENS_CODEGEN), used by tree_ens_predict
    hipModule_t cg_module = nullptr;
    hipFunction_t cg_fn = nullptr;
    // Small batches: partial sums of the tile splits, reused by every eager call (no
    // allocation per call). Eager calls from different streams are ordered with an event, so
    // they never share the scratch at the same time.
    double *d_scratch = nullptr;
    hipEvent_t scratch_done = nullptr;
    mutable std::mutex scratch_mu;
    mutable hipStream_t scratch_stream = nullptr;
    mutable bool scratch_used = false;
    // Calls captured into a HIP graph take none of the above (a replay is ordered with nothing
    // the handle records): each captured call gets a buffer of its own for its partial sums and
    // threshold codes, allocated when it is captured and kept until destroy.
    mutable std::mutex capture_mu;
    mutable std::vector<void *> capture_bufs;
    // Kernel timing (tree_ens_kernel_timing): while `timing` is set, eager predicts record
    // t_start[i] / t_stop[i] around the i-th scoring launch, i < t_used <= kMaxTimedLaunches.
    mutable std::mutex timing_mu;
    mutable bool timing = false;
    mutable std::vector<hipEvent_t> t_start, t_stop;
    mutable int32_t t_used = 0;
    // launch shape of the last batch size seen (callers usually repeat one batch size)
    mutable std::mutex shape_mu;
    mutable int64_t shape_blocks = -1;
    mutable int shape_level = 0;
    mutable int64_t shape_head = 0;
    mutable int shape_splits = 1;
};

namespace {
constexpr size_t kScratchDoubles = size_t(1) << 17; // 1 MiB of split partials
constexpr int kMaxTimedLaunches = 1024;             // event pairs of tree_ens_kernel_timing

// Scratch of the allocation-free entry point (tree_ens_predict_noalloc): split partial sums and
// threshold codes in one static array, which every device the library runs on holds until the
// process ends. In host code `scratch` is only a stand-in for the symbol: its device address
// comes from hipGetSymbolAddress, once per device, and only that address reaches a kernel or a
// copy.
constexpr size_t kStaticScratchBytes = size_t(16) << 20; // 16 MiB
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_static_mu;
unsigned char *g_static_ptr[kMaxDevices] = {};

// Device address of `scratch` on `device` (the current device), looked up on the first use.
int static_scratch(int device, unsigned char **out) {
    if (device < 0 || device >= kMaxDevices)
        return fail(TREE_ENS_E_DEVICE, "device index beyond the allocation-free scratch table");
    std::lock_guard<std::mutex> lock(g_static_mu);
    if (!g_static_ptr[device]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress(scratch)");
        g_static_ptr[device] = static_cast<unsigned char *>(p);
    }
    *out = g_static_ptr[device];
    return TREE_ENS_OK;
}
} // namespace

namespace {

void free_device(tree_ens *h) {
    (void)hipFree(h->d_images);
    (void)hipFree(h->d_packets);
    (void)hipFree(h->d_cpackets);
    (void)hipFree(h->d_cleaf);
    (void)hipFree(h->d_cleaf_id);
    (void)hipFree(h->d_big);
    (void)hipFree(h->d_tile_recs);
    (void)hipFree(h->d_tree_node_off);
    (void)hipFree(h->d_tree_orig);
    (void)hipFree(h->d_orig_id);
    (void)hipFree(h->d_leaf_vec);
    (void)hipFree(h->d_code_search);
    (void)hipFree(h->d_code_chunks);
    (void)hipFree(h->d_scratch);
    if (h->scratch_done)
        (void)hipEventDestroy(h->scratch_done);
    for (void *b : h->capture_bufs)
        (void)hipFree(b);
    for (hipEvent_t ev : h->t_start)
        (void)hipEventDestroy(ev);
    for (hipEvent_t ev : h->t_stop)
        (void)hipEventDestroy(ev);
    if (h->cg_module)
        (void)hipModuleUnload(h->cg_module);
}

// Compile generated HIP source for gfx950 with hiprtc (host only: no device is needed).
int compile_codegen(const std::string &src, std::vector<char> &code, std::string &err) {
    hiprtcProgram prog;
    hiprtcResult r = hiprtcCreateProgram(&prog, src.c_str(), "tree_ens_cg.hip", 0, nullptr, nullptr);
    if (r != HIPRTC_SUCCESS) {
        err = std::string("hiprtcCreateProgram: ") + hiprtcGetErrorString(r);
        return TREE_ENS_E_DEVICE;
    }
    // the same code-generation settings as the library's own kernels
    const char *opts[] = {"--offload-arch=gfx950", "-O3", "-fno-gpu-flush-denormals-to-zero",
                          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"};
    r = hiprtcCompileProgram(prog, int(sizeof opts / sizeof opts[0]), opts);
    if (r != HIPRTC_SUCCESS) {
        size_t n = 0;
        std::string log;
        if (hiprtcGetProgramLogSize(prog, &n) == HIPRTC_SUCCESS && n > 1) {
            log.resize(n);
            if (hiprtcGetProgramLog(prog, &log[0]) != HIPRTC_SUCCESS)
                log.clear();
        }
        err = std::string("code generation: hiprtc failed (") + hiprtcGetErrorString(r) + ")" +
              (log.empty() ? "" : ": " + log.substr(0, 2000));
        (void)hiprtcDestroyProgram(&prog);
        return TREE_ENS_E_DEVICE;
    }
    size_t size = 0;
    r = hiprtcGetCodeSize(prog, &size);
    if (r == HIPRTC_SUCCESS) {
        code.resize(size);
        r = hiprtcGetCode(prog, code.data());
    }
    (void)hiprtcDestroyProgram(&prog);
    if (r != HIPRTC_SUCCESS) {
        err = std::string("code generation: ") + hiprtcGetErrorString(r);
        return TREE_ENS_E_DEVICE;
    }
    return TREE_ENS_OK;
}

template <typename T>
hipError_t upload(T **dst, const std::vector<T> &src) {
    const size_t bytes = std::max<size_t>(src.size() * sizeof(T), sizeof(T));
    hipError_t e = hipMalloc(reinterpret_cast<void **>(dst), bytes);
    if (e != hipSuccess)
        return e;
    if (!src.empty())
        e = hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice);
    return e;
}

// Launch shape for a batch of n_blocks document blocks: a tiling level, a number of head
// blocks walked whole by one workgroup each, and the split count of the remaining (tail)
// blocks, each split over that many workgroups that walk a contiguous share of the tiles. Time
// is counted in walker rounds (every walker walking one group of K trees: a tile takes as long
// as its fullest round, so tiles smaller than one round save nothing). With W resident
// workgroups, the estimated makespan in units of one block walking all trees is
//     head / W * (1 + c_wg)
//     + ceil(tail blocks * splits / W) * (share + c_wg)
//     + (splits > 1 ? c_reduce : 0) + tiny * workgroups,
// where share = ceil(tiles / splits) * (rounds of the fullest tile + c_tile) / (rounds of all
// tiles + tiles * c_tile) at tiling 0, c_tile is the cost of switching tiles (two barriers, the
// copy into LDS, the part of the next tile's load the walk does not hide: about half a round on
// 20,000 depth-3 trees, measured), c_wg is the per-workgroup cost (staging, prologue, epilogue)
// and the last term prefers fewer
// workgroups (fewer partial sums) among equal estimates. Candidates: everything split
// uniformly (no head; small batches spread over the GPU), and whole rounds of workgroups as
// head with the remainder split to fill the last round (a batch of 1,563 blocks on 512 resident
// workgroups would otherwise run a fourth round at 5% occupancy).
struct LaunchShape {
    int level = 0;
    int64_t head = 0;
    int splits = 1;
};

LaunchShape choose_launch(const tree_ens *h, int64_t n_blocks) {
    constexpr double kItemCost = 0.2;    // staging, prologue and restaging of one workgroup (measured)
    constexpr double kReduceCost = 0.05; // the second kernel
    constexpr double kPerWorkgroup = 1e-6;
    constexpr double kTileRounds = 0.5;    // switching tiles, in walker rounds
    constexpr double kPacketRounds = 0.1;  // switching packets (no barrier), in walker rounds
    const int wg_per_cu = h->plan.lds_bytes <= treeens::kLdsPerCu / 2 ? 2 : 1;
    const int64_t slots = int64_t(kNumCus) * wg_per_cu;
    // walker packets (8-byte or compact records): one level, each walker's packets in place of
    // the tiles
    const bool cp = h->cp_k > 0;
    const bool pk = cp || h->pk_recs > 0;
    const int n_levels = pk ? 1 : treeens::kTileLevels;
    auto tiles_at = [&](int level) {
        return cp ? h->cp_per_walker : pk ? h->pk_per_walker : h->level_begin[level + 1] - h->level_begin[level];
    };
    auto rounds_at = [&](int level) {
        return cp ? h->cp_max_groups : pk ? h->pk_max_groups : h->level_max_rounds[level];
    };
    const double switch_rounds = pk ? kPacketRounds : kTileRounds;
    const double total =
        double(std::max<int64_t>(cp ? h->cp_total_rounds : pk ? h->pk_total_rounds : h->total_rounds, 1)) +
        switch_rounds * double(tiles_at(0));
    double best = 1e300;
    LaunchShape pick;
    auto consider = [&](int level, int64_t head, int sp) {
        const int nt = tiles_at(level);
        const int64_t tail = n_blocks - head;
        const double share = double((nt + sp - 1) / sp) * (rounds_at(level) + switch_rounds) / total;
        const double cost = double(head / slots) * (1.0 + kItemCost) +
                            double((tail * sp + slots - 1) / slots) * (share + kItemCost) +
                            (sp > 1 ? kReduceCost : 0.0) + kPerWorkgroup * double(head + tail * sp);
        if (cost < best - 1e-9) {
            best = cost;
            pick = LaunchShape{level, head, sp};
        }
    };
    for (int k = 0; k < n_levels; ++k) {
        const int nt = tiles_at(k);
        for (int sp = 1; sp <= std::min(nt, 1024); ++sp)
            consider(k, 0, sp);
    }
    const int64_t rem = n_blocks % slots;
    if (n_blocks > slots && rem > 0) {
        const int nt = tiles_at(0);
        for (int sp = 2; sp <= std::min<int64_t>(nt, slots / rem); ++sp)
            consider(0, n_blocks - rem, sp);
    }
    return pick;
}

struct DeviceGuard {
    int prev = -1;
    hipError_t err = hipSuccess;
    explicit DeviceGuard(int dev) {
        err = hipGetDevice(&prev);
        if (err == hipSuccess && prev != dev)
            err = hipSetDevice(dev);
        else
            prev = -1;
    }
    ~DeviceGuard() {
        if (prev >= 0)
            (void)hipSetDevice(prev);
    }
};

int check_predict_args(const tree_ens *h, const float *X, int64_t n_docs, int32_t n_features,
                       const void *out) {
    if (!h)
        return fail(TREE_ENS_E_ARG, "handle is NULL");
    if (n_docs < 0)
        return fail(TREE_ENS_E_ARG, "n_docs must be >= 0");
    if (n_docs == 0)
        return TREE_ENS_OK;
    if (!X || !out)
        return fail(TREE_ENS_E_ARG, "X or the output pointer is NULL");
    if ((reinterpret_cast<uintptr_t>(X) & 3u) != 0 || (reinterpret_cast<uintptr_t>(out) & 3u) != 0)
        return fail(TREE_ENS_E_ARG, "X and the output must be 4-byte aligned");
    if (n_features < h->n_cols)
        return fail(TREE_ENS_E_SHAPE, "documents carry " + std::to_string(n_features) +
                                          " features; the model reads feature " +
                                          std::to_string(h->n_cols - 1));
    if (n_features < 1)
        return fail(TREE_ENS_E_SHAPE, "n_features must be >= 1");
    return TREE_ENS_OK;
}

// MODE kModeScore writes scores; kModeVector writes scores [n_docs][n_outputs] (one launch per
// four outputs); kModeLeaves writes leaf_ids [n_docs][n_trees]; kModeUsage writes per-document
// feature counts into leaf_ids and, if masks is not NULL, the bitmasks (rows of mask_words
// words).
// Where a call's scratch (split partial sums, threshold codes) comes from.
enum class ScratchSource {
    kHandle, // the handle's shared buffer or stream-ordered allocations (eager calls), a buffer
             // of the call's own kept by the handle (calls captured into a graph)
    kStatic, // the library's static device array only (tree_ens_predict_noalloc)
};

template <int MODE>
int launch_predict(const tree_ens *h, hipStream_t stream, const float *X, int64_t n_docs,
                   int32_t n_features, float *scores, int32_t *leaf_ids, uint32_t *masks = nullptr,
                   int32_t mask_words = 0, ScratchSource source = ScratchSource::kHandle) {
    constexpr bool kScores = MODE == kModeScore || MODE == kModeVector; // split partial sums
    // entries per document in the partial sums, and launches (four outputs each)
    const int comps = MODE == kModeVector ? kVecPerLaunch : 1;
    const int n_chunks = MODE == kModeVector ? (h->n_outputs + kVecPerLaunch - 1) / kVecPerLaunch : 1;
    if (MODE == kModeVector && h->plan.tile_bytes < kThreads * kVecPerLaunch * int(sizeof(double)))
        return fail(TREE_ENS_E_ARG, "the tile slot cannot hold the vector reduction");
    const int dl = h->plan.docs_per_block;
    const int64_t n_blocks = (n_docs + dl - 1) / dl;
    if (n_blocks > 0x7fffffff)
        return fail(TREE_ENS_E_ARG, "too many documents for one launch");
    LaunchShape shape;
    int32_t usage_off = h->plan.usage_off;
    if (MODE == kModeUsage || MODE == kModeUsageSlot) {
        // one workgroup walks every tile of its block: its bitmasks are complete in LDS
        shape = LaunchShape{0, n_blocks, 1};
        const int64_t mask_bytes = int64_t((h->n_cols + 31) / 32) * dl * 4;
        if (MODE == kModeUsageSlot) {
            usage_off = h->usage_slot_off;
            if (usage_off < 0 || usage_off + mask_bytes > h->plan.zero_rec)
                return fail(TREE_ENS_E_ARG, "feature bitmasks do not fit the tile slot");
        } else {
            const int64_t lds_end = h->plan.lds_bytes == treeens::kLdsPerCu
                                        ? treeens::kLdsPerCu
                                        : treeens::kLdsPerCu / 2 + treeens::kUsageHalfBytes;
            if (usage_off + mask_bytes > lds_end)
                return fail(TREE_ENS_E_ARG, "feature bitmasks do not fit the LDS plan");
        }
    } else {
        std::lock_guard<std::mutex> lock(h->shape_mu);
        if (h->shape_blocks == n_blocks) {
            shape = LaunchShape{h->shape_level, h->shape_head, h->shape_splits};
        } else {
            shape = choose_launch(h, n_blocks);
            h->shape_blocks = n_blocks;
            h->shape_level = shape.level;
            h->shape_head = shape.head;
            h->shape_splits = shape.splits;
        }
    }
    {
        // grid of the chosen shape (the no-split shape the allocation-free path may fall back
        // to is never larger): every tail block split into the shape's splits, plus the padding
        // to whole XCD columns
        const int64_t tail_blocks = n_blocks - shape.head;
        const int64_t tail_slots = shape.head > 0 ? (tail_blocks + kXcds - 1) / kXcds * kXcds : tail_blocks;
        if (shape.head + tail_slots * shape.splits > 0x7fffffff)
            return fail(TREE_ENS_E_ARG, "too many documents for one launch");
    }
    // compact packets, where the model has them, for every mode but the feature trace
    const bool cp = h->cp_k > 0 && (MODE == kModeScore || MODE == kModeLeaves || MODE == kModeVector);
    ScoreFn fn = pick_kernel<MODE>(h->plan, cp);
    if (!fn)
        return fail(TREE_ENS_E_ARG, "unsupported document block size");
    hipError_t e = hipSuccess;
    // scratch of this call: split partial sums (score modes with splits) and threshold codes
    // (coded models), each 256-byte aligned
    auto align256 = [](size_t b) { return (b + 255) & ~size_t(255); };
    const size_t codes_bytes = h->plan.coded ? align256(size_t(n_docs) * size_t(h->n_cols) * sizeof(uint16_t)) : 0;
    auto partial_bytes = [&](const LaunchShape &sh) {
        return kScores && sh.splits > 1
                   ? align256(size_t(sh.splits) * size_t(n_docs - sh.head * dl) * size_t(comps) * sizeof(double))
                   : size_t(0);
    };
    double *partials = nullptr;
    uint16_t *codes = nullptr;
    bool shared_scratch = false; // partials in the handle's event-ordered buffer
    bool async_alloc = false;    // partials and codes from hipMallocAsync, freed on the stream
    void *async_buf = nullptr;
    std::unique_lock<std::mutex> scratch_lock;
    if (source == ScratchSource::kStatic) {
        // the static array only: a shape whose partials do not fit takes no splits (every
        // workgroup walks all tiles of its block); codes that do not fit are an error
        if (codes_bytes > kStaticScratchBytes)
            return fail(TREE_ENS_E_ARG,
                        "the batch's threshold codes (" + std::to_string(codes_bytes) +
                            " bytes) exceed the allocation-free scratch of " +
                            std::to_string(kStaticScratchBytes) + " bytes");
        if (codes_bytes + partial_bytes(shape) > kStaticScratchBytes)
            shape = LaunchShape{0, n_blocks, 1};
        unsigned char *base = nullptr;
        const int rc = static_scratch(h->device, &base);
        if (rc != TREE_ENS_OK)
            return rc;
        codes = h->plan.coded ? reinterpret_cast<uint16_t *>(base) : nullptr;
        partials = partial_bytes(shape) ? reinterpret_cast<double *>(base + codes_bytes) : nullptr;
    } else {
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(stream, &cap) != hipSuccess)
            cap = hipStreamCaptureStatusNone;
        (void)hipGetLastError();
        const size_t need = codes_bytes + partial_bytes(shape);
        if (cap == hipStreamCaptureStatusActive) {
            // a buffer of this call's own, kept by the handle: replays of the graph never share
            // it with eager calls or other graphs (allocated outside the stream's order, so the
            // capture mode is relaxed for the allocation)
            if (need > 0) {
                void *buf = nullptr;
                hipStreamCaptureMode mode = hipStreamCaptureModeRelaxed;
                (void)hipThreadExchangeStreamCaptureMode(&mode);
                e = hipMalloc(&buf, need);
                (void)hipThreadExchangeStreamCaptureMode(&mode);
                if (e != hipSuccess)
                    return hip_fail(e, "hipMalloc(scratch of a captured call)");
                std::lock_guard<std::mutex> lock(h->capture_mu);
                h->capture_bufs.push_back(buf);
                codes = h->plan.coded ? static_cast<uint16_t *>(buf) : nullptr;
                partials = partial_bytes(shape)
                               ? reinterpret_cast<double *>(static_cast<unsigned char *>(buf) + codes_bytes)
                               : nullptr;
            }
        } else {
            const size_t pb = partial_bytes(shape);
            if (pb > 0 && pb <= kScratchDoubles * sizeof(double) && codes_bytes == 0) {
                scratch_lock = std::unique_lock<std::mutex>(h->scratch_mu);
                if (h->scratch_used && h->scratch_stream != stream) {
                    e = hipStreamWaitEvent(stream, h->scratch_done, 0);
                    if (e != hipSuccess)
                        return hip_fail(e, "hipStreamWaitEvent");
                }
                partials = h->d_scratch;
                shared_scratch = true;
            } else if (need > 0) {
                e = hipMallocAsync(&async_buf, need, stream);
                if (e != hipSuccess)
                    return hip_fail(e, "hipMallocAsync(scratch)");
                async_alloc = true;
                codes = h->plan.coded ? static_cast<uint16_t *>(async_buf) : nullptr;
                partials = pb ? reinterpret_cast<double *>(static_cast<unsigned char *>(async_buf) + codes_bytes)
                              : nullptr;
            }
        }
    }
    const int level = shape.level, splits = shape.splits;
    const int64_t tail_docs = n_docs - shape.head * dl;
    // tail blocks after a head are laid out in whole XCD columns (see the kernel)
    const int64_t tail_blocks = n_blocks - shape.head;
    const int64_t tail_slots = shape.head > 0 ? (tail_blocks + kXcds - 1) / kXcds * kXcds : tail_blocks;
    const int64_t n_wgs = shape.head + tail_slots * splits;
    // walker packets (pk_recs > 0) stand in for the tiles: n_tiles is then packets per walker.
    // The feature trace of one-workgroup plans keeps the shared tiles: its bitmasks sit past
    // their zero record, where the packets' sub-slots reach.
    const bool pk = h->pk_recs > 0 && !(MODE == kModeUsage && h->plan.lds_bytes == treeens::kLdsPerCu);
    const uint2 *images = cp   ? reinterpret_cast<const uint2 *>(h->d_cpackets)
                          : pk ? h->d_packets
                               : h->d_images + h->level_image_off[level];
    const uint32_t *tile_recs = h->d_tile_recs + (pk || cp ? 0 : h->level_begin[level]);
    const int n_tiles = cp   ? h->cp_per_walker
                        : pk ? h->pk_per_walker
                             : h->level_begin[level + 1] - h->level_begin[level];
    const int32_t slot_recs = cp ? treeens::kCompactPacketBytes / 8 : pk ? h->pk_recs : h->level_slot_recs[level];
    (void)hipGetLastError();
    // coded models: one pass turns the float features into 16-bit threshold codes
    const void *docs = X;
    int32_t row_stride = n_features;
    if (h->plan.coded) {
        // documents per coding workgroup: enough workgroups to fill the GPU twice over, but
        // each one long enough to pay for loading its chunk's thresholds into LDS
        int64_t per_wg = 256;
        while (per_wg < 4096 && ((n_docs + per_wg - 1) / per_wg) * h->n_code_chunks > 4 * kNumCus)
            per_wg *= 2;
        const int64_t code_blocks = (n_docs + per_wg - 1) / per_wg;
        hipLaunchKernelGGL(code_kernel,
                           dim3(unsigned((code_blocks + kXcds - 1) / kXcds * kXcds * h->n_code_chunks)),
                           dim3(kCodeThreads), 0, stream, X, n_docs, n_features, h->n_cols,
                           int32_t(per_wg), h->d_code_search, h->d_code_chunks, h->n_code_chunks,
                           cp ? treeens::kCompactCodeShift : 0, codes);
        docs = codes;
        row_stride = h->n_cols;
    }
    const double scale = 1.0 / double(h->n_bags);
    const int n_out = MODE == kModeVector ? h->n_outputs : 1;
    for (int chunk = 0; chunk < n_chunks && e == hipSuccess; ++chunk) {
        // kernel timing: an event pair around this launch (eager calls only)
        hipEvent_t t0 = nullptr, t1 = nullptr;
        {
            std::lock_guard<std::mutex> lock(h->timing_mu);
            if (h->timing && h->t_used < int32_t(h->t_start.size())) {
                hipStreamCaptureStatus tc = hipStreamCaptureStatusNone;
                if (hipStreamIsCapturing(stream, &tc) != hipSuccess)
                    tc = hipStreamCaptureStatusActive;
                (void)hipGetLastError();
                if (tc == hipStreamCaptureStatusNone) {
                    t0 = h->t_start[size_t(h->t_used)];
                    t1 = h->t_stop[size_t(h->t_used)];
                    h->t_used++;
                }
            }
        }
        if (t0 && (e = hipEventRecord(t0, stream)) != hipSuccess)
            break;
        hipLaunchKernelGGL(fn, dim3(unsigned(n_wgs)), dim3(kThreads), 0, stream, docs, n_docs,
                           row_stride, h->n_cols, images, slot_recs, tile_recs,
                           n_tiles, int32_t(shape.head), splits, h->plan.xs_bytes,
                           pk ? h->pk_zero_rec : h->plan.zero_rec,
                           partials, scores, leaf_ids, h->d_orig_id, h->d_tree_node_off,
                           h->d_tree_orig, h->n_trees, masks, mask_words, usage_off,
                           reinterpret_cast<const float4 *>(h->d_leaf_vec), h->vec_stride / 4, n_out,
                           chunk, scale, cp ? treeens::kCompactPacketBytes / 8 : pk ? h->pk_recs : 0,
                           h->d_big, h->n_small, h->big_off0, h->d_cleaf, h->d_cleaf_id);
        e = hipGetLastError();
        if (e == hipSuccess && t1)
            e = hipEventRecord(t1, stream);
        if (e == hipSuccess && partials) {
            // the tail blocks' entries, in [doc][component] order
            const int64_t n_entries = tail_docs * comps;
            const ReduceOut out{scores + shape.head * dl * n_out, comps, n_out, chunk * comps, scale};
            if (splits <= 64)
                hipLaunchKernelGGL(reduce_partials_thread_kernel,
                                   dim3(unsigned((n_entries + 255) / 256)), dim3(256), 0, stream,
                                   partials, splits, n_entries, out);
            else
                hipLaunchKernelGGL(reduce_partials_wave_kernel, dim3(unsigned(n_entries)), dim3(64),
                                   0, stream, partials, splits, n_entries, out);
            e = hipGetLastError();
        }
    }
    if (shared_scratch) {
        // the next eager call from another stream waits for this one's reduction
        if (e == hipSuccess)
            e = hipEventRecord(h->scratch_done, stream);
        h->scratch_stream = stream;
        h->scratch_used = true;
    } else if (async_alloc) {
        hipError_t e2 = hipFreeAsync(async_buf, stream);
        if (e == hipSuccess)
            e = e2;
    }
    if (e != hipSuccess)
        return hip_fail(e, "kernel launch");
    return TREE_ENS_OK;
}

} // namespace

extern "C" {

int tree_ens_create(tree_ens_t **out, int32_t n_trees, const int64_t *tree_offsets,
                    const int32_t *feature, const float *threshold, const int32_t *left,
                    const int32_t *right, const float *value, uint32_t flags) {
    return tree_ens_create_multi(out, n_trees, tree_offsets, feature, threshold, left, right, value,
                                 1, 1, flags);
}

int tree_ens_create_multi(tree_ens_t **out, int32_t n_trees, const int64_t *tree_offsets,
                          const int32_t *feature, const float *threshold, const int32_t *left,
                          const int32_t *right, const float *value, int32_t n_outputs,
                          int32_t n_bags, uint32_t flags) {
    g_err.clear();
    if (!out)
        return fail(TREE_ENS_E_ARG, "out is NULL");
    *out = nullptr;
    if (n_bags < 1)
        return fail(TREE_ENS_E_ARG, "n_bags must be >= 1");
    const bool codegen = (flags & TREE_ENS_CODEGEN) != 0;
    if (codegen && n_outputs != 1)
        return fail(TREE_ENS_E_ARG, "code generation supports one value per leaf");
    Packed p;
    std::string err;
    int rc;
    try {
        rc = treeens::pack_model(n_trees, tree_offsets, feature, threshold, left, right, value, n_outputs, flags,
                                 p, err);
    } catch (const std::bad_alloc &) {
        return fail(TREE_ENS_E_NOMEM, "host allocation failed while packing");
    }
    if (rc != treeens::kOk)
        return fail(rc, err);
    std::vector<char> cg_code;
    if (codegen && n_trees > 0) {
        std::string src;
        try {
            rc = treeens::codegen_source(n_trees, tree_offsets, feature, threshold, left, right, value,
                                         flags, src, err);
        } catch (const std::bad_alloc &) {
            return fail(TREE_ENS_E_NOMEM, "host allocation failed while generating code");
        }
        if (rc != treeens::kOk)
            return fail(rc, err);
        rc = compile_codegen(src, cg_code, err);
        if (rc != TREE_ENS_OK)
            return fail(rc, err);
    }

    tree_ens *h = new (std::nothrow) tree_ens();
    if (!h)
        return fail(TREE_ENS_E_NOMEM, "host allocation failed");
    h->n_trees = p.n_trees;
    h->n_cols = p.n_cols;
    h->max_depth = p.max_depth;
    h->n_nodes = int64_t(p.nodes.size());
    h->plan = p.plan;
    h->n_outputs = p.n_outputs;
    h->n_bags = n_bags;
    h->vec_stride = p.vec_stride;
    std::memcpy(h->level_begin, p.level_begin, sizeof h->level_begin);
    hipError_t e = hipGetDevice(&h->device);
    std::memcpy(h->level_image_off, p.level_image_off, sizeof h->level_image_off);
    std::memcpy(h->level_max_rounds, p.level_max_rounds, sizeof h->level_max_rounds);
    h->total_rounds = p.total_rounds;
    h->usage_slot_off = p.usage_slot_off;
    h->pk_recs = p.pk_recs;
    h->pk_zero_rec = p.pk_zero_rec;
    h->pk_per_walker = p.pk_per_walker;
    h->pk_max_groups = p.pk_max_groups;
    h->pk_total_rounds = p.pk_total_rounds;
    std::memcpy(h->level_slot_recs, p.level_slot_recs, sizeof h->level_slot_recs);
    std::vector<uint2> images(p.images.size());
    if (!p.images.empty())
        std::memcpy(images.data(), p.images.data(), p.images.size() * sizeof(NodeRec));
    if (e == hipSuccess)
        e = upload(&h->d_images, images);
    if (e == hipSuccess)
        e = upload(&h->d_tile_recs, p.tile_recs);
    h->cp_k = p.cp_k;
    h->cp_per_walker = p.cp_per_walker;
    h->cp_max_groups = p.cp_max_groups;
    h->cp_total_rounds = p.cp_total_rounds;
    if (e == hipSuccess && p.cp_k > 0) {
        // the compact packets replace the 8-byte ones (the feature trace walks the shared tiles)
        h->pk_recs = 0;
        e = upload(&h->d_cpackets, p.cp_packets);
        if (e == hipSuccess)
            e = upload(&h->d_cleaf, p.cp_leaf);
        if (e == hipSuccess)
            e = upload(&h->d_cleaf_id, p.cp_leaf_id);
    } else if (e == hipSuccess && p.pk_recs > 0) {
        std::vector<uint2> packets(p.packets.size());
        std::memcpy(packets.data(), p.packets.data(), p.packets.size() * sizeof(NodeRec));
        e = upload(&h->d_packets, packets);
    }
    h->n_small = p.n_small;
    h->big_off0 = p.tree_node_off[size_t(p.n_small)];
    if (e == hipSuccess && p.n_small < p.n_trees) {
        std::vector<uint2> big(p.nodes.size() - h->big_off0);
        std::memcpy(big.data(), p.nodes.data() + h->big_off0, big.size() * sizeof(NodeRec));
        e = upload(&h->d_big, big);
    }
    if (e == hipSuccess)
        e = upload(&h->d_tree_node_off, p.tree_node_off);
    if (e == hipSuccess)
        e = upload(&h->d_tree_orig, p.tree_orig);
    if (e == hipSuccess)
        e = upload(&h->d_orig_id, p.orig_id);
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&h->d_scratch), kScratchDoubles * sizeof(double));
    if (e == hipSuccess)
        e = hipEventCreateWithFlags(&h->scratch_done, hipEventDisableTiming);
    if (e == hipSuccess && p.n_outputs > 1)
        e = upload(&h->d_leaf_vec, p.leaf_vec);
    if (e == hipSuccess && !cg_code.empty()) {
        e = hipModuleLoadData(&h->cg_module, cg_code.data());
        if (e == hipSuccess)
            e = hipModuleGetFunction(&h->cg_fn, h->cg_module, "tree_ens_cg");
    }
    if (e == hipSuccess && p.plan.coded) {
        e = upload(&h->d_code_search, p.code_search);
        if (e == hipSuccess)
            e = upload(&h->d_code_chunks, p.code_chunks);
        h->n_code_chunks = int32_t(p.code_chunks.size());
    }
    if (e != hipSuccess) {
        free_device(h);
        delete h;
        return fail(e == hipErrorOutOfMemory ? TREE_ENS_E_NOMEM : TREE_ENS_E_DEVICE,
                    std::string("device upload failed: ") + hipGetErrorString(e));
    }
    *out = h;
    return TREE_ENS_OK;
}

int tree_ens_predict(const tree_ens_t *h, void *stream, const float *X, int64_t n_docs,
                     int32_t n_features, float *scores) {
    g_err.clear();
    int rc = check_predict_args(h, X, n_docs, n_features, scores);
    if (rc != TREE_ENS_OK || n_docs == 0)
        return rc;
    DeviceGuard g(h->device);
    if (g.err != hipSuccess)
        return hip_fail(g.err, "hipSetDevice");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (h->n_trees == 0) {
        const int bs = 256;
        const int64_t n = n_docs * h->n_outputs;
        hipLaunchKernelGGL(fill_zero_kernel, dim3(unsigned((n + bs - 1) / bs)), dim3(bs), 0, s,
                           scores, n);
        hipError_t e = hipGetLastError();
        return e == hipSuccess ? TREE_ENS_OK : hip_fail(e, "kernel launch");
    }
    if (h->n_outputs > 1)
        return launch_predict<kModeVector>(h, s, X, n_docs, n_features, scores, nullptr);
    if (h->cg_fn) {
        // the model's own kernel: one document per thread
        const float *x = X;
        long long n = n_docs;
        int nf = n_features;
        float *out = scores;
        double scale = 1.0 / double(h->n_bags);
        void *args[] = {&x, &n, &nf, &out, &scale};
        const int64_t blocks = (n_docs + treeens::kCodegenThreads - 1) / treeens::kCodegenThreads;
        if (blocks > 0x7fffffff)
            return fail(TREE_ENS_E_ARG, "too many documents for one launch");
        (void)hipGetLastError();
        hipError_t e = hipModuleLaunchKernel(h->cg_fn, unsigned(blocks), 1, 1, treeens::kCodegenThreads,
                                             1, 1, 0, s, args, nullptr);
        return e == hipSuccess ? TREE_ENS_OK : hip_fail(e, "specialised kernel launch");
    }
    return launch_predict<kModeScore>(h, s, X, n_docs, n_features, scores, nullptr);
}

int tree_ens_predict_noalloc(const tree_ens_t *h, void *stream, const float *X, int64_t n_docs,
                             int32_t n_features, float *scores) {
    g_err.clear();
    int rc = check_predict_args(h, X, n_docs, n_features, scores);
    if (rc != TREE_ENS_OK || n_docs == 0)
        return rc;
    DeviceGuard g(h->device);
    if (g.err != hipSuccess)
        return hip_fail(g.err, "hipSetDevice");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (h->n_trees == 0 || h->cg_fn)
        return tree_ens_predict(h, stream, X, n_docs, n_features, scores); // no scratch used
    if (h->n_outputs > 1)
        return launch_predict<kModeVector>(h, s, X, n_docs, n_features, scores, nullptr, nullptr, 0,
                                           ScratchSource::kStatic);
    return launch_predict<kModeScore>(h, s, X, n_docs, n_features, scores, nullptr, nullptr, 0,
                                      ScratchSource::kStatic);
}

int tree_ens_predict_leaves(const tree_ens_t *h, void *stream, const float *X, int64_t n_docs,
                            int32_t n_features, int32_t *leaf_ids) {
    g_err.clear();
    int rc = check_predict_args(h, X, n_docs, n_features, leaf_ids);
    if (rc != TREE_ENS_OK || n_docs == 0 || h->n_trees == 0)
        return rc;
    DeviceGuard g(h->device);
    if (g.err != hipSuccess)
        return hip_fail(g.err, "hipSetDevice");
    return launch_predict<kModeLeaves>(h, reinterpret_cast<hipStream_t>(stream), X, n_docs,
                                       n_features, nullptr, leaf_ids);
}

int tree_ens_predict_topk(const tree_ens_t *h, void *stream, const float *X, int64_t n_docs,
                          int32_t n_features, const int64_t *group_offsets, int64_t n_groups,
                          int32_t k, float *scores, int32_t *top_idx, float *top_scores) {
    if (h && h->n_outputs != 1)
        return fail(TREE_ENS_E_ARG, "reranking needs one score per document (n_outputs = 1)");
    int rc = tree_ens_predict(h, stream, X, n_docs, n_features, scores);
    if (rc != TREE_ENS_OK)
        return rc;
    return tree_ens_topk(stream, scores, n_docs, group_offsets, n_groups, k, top_idx, top_scores);
}

int tree_ens_feature_usage(const tree_ens_t *h, void *stream, const float *X, int64_t n_docs,
                           int32_t n_features, int32_t *counts, uint32_t *masks) {
    g_err.clear();
    int rc = check_predict_args(h, X, n_docs, n_features, counts);
    if (rc != TREE_ENS_OK || n_docs == 0)
        return rc;
    if (masks && (reinterpret_cast<uintptr_t>(masks) & 3u) != 0)
        return fail(TREE_ENS_E_ARG, "masks must be 4-byte aligned");
    DeviceGuard g(h->device);
    if (g.err != hipSuccess)
        return hip_fail(g.err, "hipSetDevice");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int32_t words = (n_features + 31) / 32;
    if (h->n_trees == 0) {
        const int bs = 256;
        hipLaunchKernelGGL(fill_zero_kernel, dim3(unsigned((n_docs + bs - 1) / bs)), dim3(bs), 0, s,
                           reinterpret_cast<float *>(counts), n_docs);
        if (masks)
            hipLaunchKernelGGL(fill_zero_kernel, dim3(unsigned((n_docs * words + bs - 1) / bs)),
                               dim3(bs), 0, s, reinterpret_cast<float *>(masks), n_docs * words);
        hipError_t e = hipGetLastError();
        return e == hipSuccess ? TREE_ENS_OK : hip_fail(e, "kernel launch");
    }
    // two-workgroup plans whose level-0 tiles leave room in the slot keep two workgroups per CU
    if (h->usage_slot_off >= 0)
        return launch_predict<kModeUsageSlot>(h, s, X, n_docs, n_features, nullptr, counts, masks,
                                              words);
    return launch_predict<kModeUsage>(h, s, X, n_docs, n_features, nullptr, counts, masks, words);
}

int tree_ens_info(const tree_ens_t *h, int32_t *n_trees, int32_t *min_features, int32_t *max_depth,
                  int64_t *packed_bytes, int32_t *n_tiles, int32_t *docs_per_block) {
    g_err.clear();
    if (!h)
        return fail(TREE_ENS_E_ARG, "handle is NULL");
    if (n_trees)
        *n_trees = h->n_trees;
    if (min_features)
        *min_features = h->n_cols;
    if (max_depth)
        *max_depth = h->max_depth;
    if (packed_bytes)
        *packed_bytes = h->n_nodes * int64_t(sizeof(NodeRec));
    if (n_tiles)
        *n_tiles = h->level_begin[1] - h->level_begin[0];
    if (docs_per_block)
        *docs_per_block = h->plan.docs_per_block;
    return TREE_ENS_OK;
}

int tree_ens_codegen_source(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                            const float *threshold, const int32_t *left, const int32_t *right,
                            const float *value, uint32_t flags, char *buf, int64_t buf_size,
                            int64_t *src_len) {
    g_err.clear();
    if (buf_size < 0 || (buf_size > 0 && !buf))
        return fail(TREE_ENS_E_ARG, "buf is NULL with a positive buf_size");
    std::string src, err;
    int rc;
    try {
        rc = treeens::codegen_source(n_trees, tree_offsets, feature, threshold, left, right, value,
                                     flags | TREE_ENS_CODEGEN, src, err);
    } catch (const std::bad_alloc &) {
        return fail(TREE_ENS_E_NOMEM, "host allocation failed while generating code");
    }
    if (rc != treeens::kOk)
        return fail(rc, err);
    if (src_len)
        *src_len = int64_t(src.size());
    if (buf_size > 0) {
        const size_t n = std::min(src.size(), size_t(buf_size - 1));
        std::memcpy(buf, src.data(), n);
        buf[n] = '\0';
    }
    return TREE_ENS_OK;
}

int tree_ens_kernel_timing(const tree_ens_t *h, int32_t enable) {
    g_err.clear();
    if (!h)
        return fail(TREE_ENS_E_ARG, "handle is NULL");
    std::lock_guard<std::mutex> lock(h->timing_mu);
    if (!enable) {
        h->timing = false;
        return TREE_ENS_OK;
    }
    if (h->t_start.empty()) {
        DeviceGuard g(h->device);
        if (g.err != hipSuccess)
            return hip_fail(g.err, "hipSetDevice");
        for (int i = 0; i < kMaxTimedLaunches; ++i) {
            hipEvent_t a = nullptr, b = nullptr;
            hipError_t e = hipEventCreate(&a);
            if (e == hipSuccess)
                e = hipEventCreate(&b);
            if (e != hipSuccess) {
                if (a)
                    (void)hipEventDestroy(a);
                for (hipEvent_t ev : h->t_start)
                    (void)hipEventDestroy(ev);
                for (hipEvent_t ev : h->t_stop)
                    (void)hipEventDestroy(ev);
                h->t_start.clear();
                h->t_stop.clear();
                return hip_fail(e, "hipEventCreate");
            }
            h->t_start.push_back(a);
            h->t_stop.push_back(b);
        }
    }
    h->t_used = 0;
    h->timing = true;
    return TREE_ENS_OK;
}

int tree_ens_kernel_time(const tree_ens_t *h, double *total_ms, int32_t *launches) {
    g_err.clear();
    if (!h)
        return fail(TREE_ENS_E_ARG, "handle is NULL");
    std::lock_guard<std::mutex> lock(h->timing_mu);
    double sum = 0.0;
    for (int32_t i = 0; i < h->t_used; ++i) {
        hipError_t e = hipEventSynchronize(h->t_stop[size_t(i)]);
        float ms = 0.0f;
        if (e == hipSuccess)
            e = hipEventElapsedTime(&ms, h->t_start[size_t(i)], h->t_stop[size_t(i)]);
        if (e != hipSuccess)
            return hip_fail(e, "timing events");
        sum += double(ms);
    }
    if (total_ms)
        *total_ms = sum;
    if (launches)
        *launches = h->t_used;
    return TREE_ENS_OK;
}

int tree_ens_outputs(const tree_ens_t *h, int32_t *n_outputs, int32_t *n_bags) {
    g_err.clear();
    if (!h)
        return fail(TREE_ENS_E_ARG, "handle is NULL");
    if (n_outputs)
        *n_outputs = h->n_outputs;
    if (n_bags)
        *n_bags = h->n_bags;
    return TREE_ENS_OK;
}

void tree_ens_destroy(tree_ens_t *h) {
    if (!h)
        return;
    DeviceGuard g(h->device);
    free_device(h);
    delete h;
}

const char *tree_ens_last_error(void) { return g_err.c_str(); }

} // extern "C"
