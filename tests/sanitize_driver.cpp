// sanitize_driver.cpp -- host code under AddressSanitizer and UndefinedBehaviorSanitizer.
//
// Built by tests/test_sanitize.py with g++ -fsanitize=address,undefined (host code only: the
// packer, the code generator, the tile-image emulator of tests/pack_emu.cpp and the oracle).
// Each input file holds one model and a batch of documents written by the test from the seeded
// generators; for both tie rules the driver packs the model, walks every tiling level in the
// emulator (which checks every LDS access of the images), runs the oracle's walks, the feature
// trace and, for vector-valued leaves, the multi-output sum, generates the specialised kernel
// source, and requires the emulator's leaf ids to equal the oracle's. Malformed models must be
// rejected by the packer (and run through the oracle without a memory error). Any sanitizer
// report aborts the process; exit status 0 means every file passed.
//
// File layout (little-endian): int32 n_trees, int32 n_features, int64 n_nodes, int64 n_docs,
// int32 n_outputs, int32 valid, then int64 tree_offsets[n_trees + 1], int32 feature[n_nodes],
// float threshold[n_nodes], int32 left[n_nodes], int32 right[n_nodes],
// float value[n_nodes * n_outputs], float X[n_docs * n_features].
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "pack.hpp"

extern "C" {
int emu_walk(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
             const float *threshold, const int32_t *left, const int32_t *right, const float *value,
             int32_t n_outputs, uint32_t flags, const float *X, int64_t n_docs, int32_t n_features,
             int32_t level, int32_t *leaf_ids, double *scores, int32_t *plan_out);
const char *emu_message(void);
int oracle_score(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                 const float *threshold, const int32_t *left, const int32_t *right,
                 const float *value, const float *X, int64_t n_docs, int32_t n_features,
                 int32_t rule, int32_t walk, int32_t n_threads, double *scores,
                 int32_t *leaf_ids, int64_t *visits);
int oracle_score_multi(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                       const float *threshold, const int32_t *left, const int32_t *right,
                       const float *value, int32_t n_outputs, int32_t n_bags, const float *X,
                       int64_t n_docs, int32_t n_features, int32_t rule, int32_t n_threads,
                       double *scores);
int oracle_feature_usage(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                         const float *threshold, const int32_t *left, const int32_t *right,
                         const float *X, int64_t n_docs, int32_t n_features, int32_t rule,
                         int32_t n_threads, int32_t *counts, uint32_t *masks);
}

namespace {

template <typename T> bool read_vec(FILE *f, std::vector<T> &v, int64_t n) {
    v.resize(size_t(n));
    return n == 0 || std::fread(v.data(), sizeof(T), size_t(n), f) == size_t(n);
}

int check_file(const char *path) {
    FILE *f = std::fopen(path, "rb");
    if (!f) {
        std::fprintf(stderr, "%s: cannot open\n", path);
        return 1;
    }
    int32_t n_trees = 0, n_features = 0, n_outputs = 0, valid = 0;
    int64_t n_nodes = 0, n_docs = 0;
    bool ok = std::fread(&n_trees, 4, 1, f) == 1 && std::fread(&n_features, 4, 1, f) == 1 &&
              std::fread(&n_nodes, 8, 1, f) == 1 && std::fread(&n_docs, 8, 1, f) == 1 &&
              std::fread(&n_outputs, 4, 1, f) == 1 && std::fread(&valid, 4, 1, f) == 1;
    std::vector<int64_t> off;
    std::vector<int32_t> feature, left, right;
    std::vector<float> threshold, value, X;
    ok = ok && read_vec(f, off, int64_t(n_trees) + 1) && read_vec(f, feature, n_nodes) &&
         read_vec(f, threshold, n_nodes) && read_vec(f, left, n_nodes) && read_vec(f, right, n_nodes) &&
         read_vec(f, value, n_nodes * n_outputs) && read_vec(f, X, n_docs * n_features);
    std::fclose(f);
    if (!ok) {
        std::fprintf(stderr, "%s: short file\n", path);
        return 1;
    }
    const size_t cells = size_t(n_docs) * size_t(n_trees);
    for (int rule = 0; rule < 2; rule++) {
        std::vector<double> o_scores(static_cast<size_t>(n_docs));
        std::vector<double> e_scores(static_cast<size_t>(n_docs) * size_t(n_outputs));
        std::vector<int32_t> o_leaves(cells), e_leaves(cells);
        int64_t visits = 0;
        const int orc = oracle_score(n_trees, off.data(), feature.data(), threshold.data(), left.data(),
                                     right.data(), value.data(), X.data(), n_docs, n_features, rule, 0, 1,
                                     o_scores.data(), o_leaves.data(), &visits);
        std::vector<int32_t> counts(static_cast<size_t>(n_docs));
        std::vector<uint32_t> masks(size_t(n_docs) * size_t((n_features + 31) / 32));
        if (n_features > 0)
            oracle_feature_usage(n_trees, off.data(), feature.data(), threshold.data(), left.data(),
                                 right.data(), X.data(), n_docs, n_features, rule, 1, counts.data(),
                                 masks.data());
        std::string src, err;
        const int cg = treeens::codegen_source(n_trees, off.data(), feature.data(), threshold.data(),
                                               left.data(), right.data(), value.data(), uint32_t(rule), src, err);
        for (int level = 0; level < treeens::kTileLevels; level++) {
            int32_t plan[10] = {};
            const int erc = emu_walk(n_trees, off.data(), feature.data(), threshold.data(), left.data(),
                                     right.data(), value.data(), n_outputs, uint32_t(rule), X.data(), n_docs,
                                     n_features, level, e_leaves.data(), e_scores.data(), plan);
            if (!valid) {
                if (erc != treeens::kErrModel) {
                    std::fprintf(stderr, "%s: malformed model not rejected (rc %d)\n", path, erc);
                    return 1;
                }
                break;
            }
            if (erc != 0) {
                std::fprintf(stderr, "%s rule %d level %d: emulator: %s\n", path, rule, level, emu_message());
                return 1;
            }
            if (orc != 0 || e_leaves != o_leaves) {
                std::fprintf(stderr, "%s rule %d level %d: leaf ids differ from the oracle (oracle rc %d)\n",
                             path, rule, level, orc);
                return 1;
            }
        }
        if (valid && cg != treeens::kOk && n_nodes <= treeens::kCodegenMaxNodes) {
            std::fprintf(stderr, "%s: code generation failed: %s\n", path, err.c_str());
            return 1;
        }
        if (valid && n_outputs > 1) {
            std::vector<double> m(size_t(n_docs) * size_t(n_outputs));
            if (oracle_score_multi(n_trees, off.data(), feature.data(), threshold.data(), left.data(),
                                   right.data(), value.data(), n_outputs, 3, X.data(), n_docs, n_features,
                                   rule, 1, m.data()) != 0) {
                std::fprintf(stderr, "%s: oracle_score_multi failed\n", path);
                return 1;
            }
            for (size_t i = 0; i < m.size(); i++)
                if (std::fabs(m[i] * 3.0 - e_scores[i]) > 1e-9 * (1.0 + std::fabs(e_scores[i]))) {
                    std::fprintf(stderr, "%s: vector scores differ at %zu\n", path, i);
                    return 1;
                }
        }
    }
    std::printf("ok %s\n", path);
    return 0;
}

} // namespace

int main(int argc, char **argv) {
    for (int i = 1; i < argc; i++)
        if (check_file(argv[i]) != 0)
            return 1;
    return 0;
}
