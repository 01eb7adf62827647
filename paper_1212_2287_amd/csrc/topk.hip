// topk.hip -- per-query top-k reranking of scores on gfx950 (Section 6 of the paper: the
// scorer reranks a query's candidate documents, e.g. 200, into the final list of the best 20).
//
// One wave per query group. The order is total: higher score first; equal scores (-0.0 equals
// +0.0) by increasing document index; NaN after every number. Each score maps to a 32-bit key
// that increases along that order's reverse (NaN -> 0), so "the k first documents" are those
// with the k largest (key, -index) pairs:
//   1. radix select, most significant byte first: four histogram passes over the group's keys
//      find the key t of the k-th document and how many documents with key t it takes;
//   2. selection in index order: every document with key > t, and the first `need` ones with
//      key == t (per-lane contiguous chunks and a wave prefix sum keep index order);
//   3. the at most k survivors are ranked by counting the survivors ahead of each.
// Work per group is O(n + k^2) for n documents; no group size limit.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "status.hpp"
#include "tree_ens.h"

namespace {

constexpr int kWave = 64;
constexpr int kMaxK = 1024;      // survivors staged in LDS
constexpr int kKeyCache = 2048;  // groups up to this size keep their keys in LDS

// Key of a score: larger keys come first. -0.0 folds into +0.0; NaN is 0, below every number
// (the smallest number, -inf, maps to 0x007FFFFF).
__device__ __forceinline__ uint32_t order_key(float s) {
    if (s != s)
        return 0u;
    const uint32_t u = __float_as_uint(s == 0.0f ? 0.0f : s);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inclusive prefix sum over the wave (lane order).
__device__ __forceinline__ uint32_t wave_inclusive_sum(uint32_t v, int lane) {
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const uint32_t o = __shfl_up(v, off);
        if (lane >= off)
            v += o;
    }
    return v;
}

__global__ void __launch_bounds__(kWave)
topk_kernel(const float *__restrict__ scores, int64_t n_docs, const int64_t *__restrict__ offsets,
            int32_t k, int32_t *__restrict__ top_idx, float *__restrict__ top_scores) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t keys[kKeyCache];
    __shared__ uint32_t cand_key[kMaxK];
    __shared__ int32_t cand_doc[kMaxK];
    const int lane = threadIdx.x;
    const int64_t g = blockIdx.x;
    // ill-formed offsets are clamped into [0, n_docs], never read past the scores
    const int64_t a = min(max(offsets[g], int64_t(0)), n_docs);
    const int64_t b = min(max(offsets[g + 1], a), n_docs);
    const int64_t n = b - a;
    int32_t *out_idx = top_idx + g * k;
    float *out_val = top_scores ? top_scores + g * k : nullptr;
    // every pass below reads the group's keys: from LDS when they fit, else from the scores
    const bool cached = n <= kKeyCache;
    if (cached) {
        for (int64_t i = lane; i < n; i += kWave)
            keys[i] = order_key(scores[a + i]);
        __syncthreads();
    }
    auto key_at = [&](int64_t i) { return cached ? keys[i] : order_key(scores[a + i]); };

    // 1. radix select: after the passes, t is the key of the k-th document and `need` the
    //    number of documents with key t among the k first (all documents when n <= k)
    uint32_t t = 0, need = uint32_t(min<int64_t>(n, k));
    if (n > k) {
        uint32_t prefix = 0;
        need = uint32_t(k);
        for (int byte = 3; byte >= 0; --byte) {
            for (int i = lane; i < 256; i += kWave)
                hist[i] = 0;
            __syncthreads();
            const int hi = 8 * (byte + 1);
            for (int64_t i = lane; i < n; i += kWave) {
                const uint32_t key = key_at(i);
                const bool match = hi == 32 || (key >> hi) == (prefix >> hi);
                if (match)
                    atomicAdd(&hist[(key >> (8 * byte)) & 255u], 1u);
            }
            __syncthreads();
            // lane l owns buckets 255-4l .. 252-4l (descending); find the bucket where the
            // running count from the top reaches `need`
            uint32_t c[4], own = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                c[j] = hist[255 - 4 * lane - j];
                own += c[j];
            }
            const uint32_t incl = wave_inclusive_sum(own, lane);
            const uint32_t excl = incl - own;
            const uint64_t hit = __ballot(incl >= need && excl < need);
            const int owner = __ffsll(static_cast<long long>(hit)) - 1;
            uint32_t digit = 0, above = 0;
            if (lane == owner) {
                uint32_t run = excl;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (run + c[j] >= need) {
                        digit = uint32_t(255 - 4 * lane - j);
                        above = run;
                        break;
                    }
                    run += c[j];
                }
            }
            digit = __shfl(digit, owner);
            above = __shfl(above, owner);
            prefix |= digit << (8 * byte);
            need -= above;
            __syncthreads(); // hist is reused by the next pass
        }
        t = prefix;
    }

    // 2. survivors in index order: lane l scans the contiguous chunk [l*chunk, (l+1)*chunk)
    const int64_t chunk = (n + kWave - 1) / kWave;
    const int64_t lo = min<int64_t>(n, lane * chunk), hi_ = min<int64_t>(n, lo + chunk);
    uint32_t n_gt = 0, n_eq = 0;
    if (n > k) {
        for (int64_t i = lo; i < hi_; ++i) {
            const uint32_t key = key_at(i);
            n_gt += key > t;
            n_eq += key == t;
        }
    }
    const uint32_t gt_excl = wave_inclusive_sum(n_gt, lane) - n_gt;
    const uint32_t eq_excl = wave_inclusive_sum(n_eq, lane) - n_eq;
    const uint32_t total_gt = __shfl(gt_excl + n_gt, kWave - 1);
    uint32_t pos_gt = gt_excl, pos_eq = eq_excl;
    for (int64_t i = lo; i < hi_; ++i) {
        const uint32_t key = key_at(i);
        int32_t slot = -1;
        if (n <= k) {
            slot = int32_t(i);
        } else if (key > t) {
            slot = int32_t(pos_gt++);
        } else if (key == t) {
            if (pos_eq < need)
                slot = int32_t(total_gt + pos_eq);
            ++pos_eq;
        }
        if (slot >= 0) {
            cand_key[slot] = key;
            cand_doc[slot] = int32_t(i);
        }
    }
    __syncthreads();

    // 3. rank the m survivors: those ahead of c have a larger key, or an equal key and a
    //    lower document index
    const int m = int(min<int64_t>(n, k));
    for (int c = lane; c < m; c += kWave) {
        const uint32_t key = cand_key[c];
        const int32_t doc = cand_doc[c];
        int rank = 0;
        for (int j = 0; j < m; ++j) {
            const uint32_t kj = cand_key[j];
            rank += kj > key || (kj == key && cand_doc[j] < doc);
        }
        out_idx[rank] = int32_t(a + doc);
        if (out_val)
            out_val[rank] = scores[a + doc];
    }
    for (int r = m + lane; r < k; r += kWave) {
        out_idx[r] = -1;
        if (out_val)
            out_val[r] = __builtin_nanf("");
    }
}

} // namespace

extern "C" {

int tree_ens_topk(void *stream, const float *scores, int64_t n_docs, const int64_t *group_offsets,
                  int64_t n_groups, int32_t k, int32_t *top_idx, float *top_scores) {
    using treeens::set_error;
    treeens::clear_error();
    if (n_groups < 0 || n_docs < 0)
        return set_error(TREE_ENS_E_ARG, "n_groups and n_docs must be >= 0");
    if (k < 1 || k > kMaxK)
        return set_error(TREE_ENS_E_ARG, "k must be in [1, " + std::to_string(kMaxK) + "]");
    if (n_docs > INT32_MAX || n_groups > INT32_MAX)
        return set_error(TREE_ENS_E_ARG, "document indices and group counts must fit int32");
    if (n_groups == 0)
        return TREE_ENS_OK;
    if (!group_offsets || !top_idx || (n_docs > 0 && !scores))
        return set_error(TREE_ENS_E_ARG, "scores, group_offsets or top_idx is NULL");
    (void)hipGetLastError();
    hipLaunchKernelGGL(topk_kernel, dim3(unsigned(n_groups)), dim3(kWave), 0,
                       reinterpret_cast<hipStream_t>(stream), scores, n_docs, group_offsets, k,
                       top_idx, top_scores);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return set_error(TREE_ENS_E_DEVICE, std::string("top-k launch: ") + hipGetErrorString(e));
    return TREE_ENS_OK;
}

} // extern "C"
