// codegen.cpp -- source of a scoring kernel specialised for one model (the CodeGen form of
// Section 3: the trees become nested if/else blocks whose feature ids, thresholds and leaf
// values are constants of the program), compiled at create time with hiprtc.
//
// The generated kernel takes one document per thread, reads its features straight from the
// row (constant offsets), walks every tree by branches on `x[f] >= theta` (or `>` under the
// strict rule) and adds each reached leaf's value to a double accumulator in tree order; the
// sum times the bag scale is rounded once to float. The trees are emitted in non-inlined
// functions of kCodegenTreesPerFunction trees each (one function holding thousands of nested
// branches takes the compiler minutes; these compile in linear time), each returning its
// trees' double sum. Host code only: no HIP call here.
#include <cmath>
#include <cstdio>
#include <string>
#include <vector>

#include "pack.hpp"

namespace treeens {

namespace {

// A float as an exact C literal (hexadecimal for finite values).
std::string float_literal(float v) {
    if (std::isnan(v))
        return "__builtin_nanf(\"\")";
    if (std::isinf(v))
        return v > 0 ? "__builtin_inff()" : "(-__builtin_inff())";
    char buf[64];
    std::snprintf(buf, sizeof buf, "%af", double(v));
    return buf;
}

} // namespace

int codegen_source(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                   const float *threshold, const int32_t *left, const int32_t *right,
                   const float *value, uint32_t flags, std::string &src, std::string &err) {
    // validate exactly as for packing
    Packed p;
    int rc = pack_model(n_trees, tree_offsets, feature, threshold, left, right, value, 1,
                        flags & ~kCodegenFlag, p, err);
    if (rc != kOk)
        return rc;
    if (p.nodes.size() > size_t(kCodegenMaxNodes) || p.max_depth > kCodegenMaxDepth) {
        err = "code generation takes at most " + std::to_string(kCodegenMaxNodes) + " nodes and depth " +
              std::to_string(kCodegenMaxDepth) + " (model: " + std::to_string(p.nodes.size()) +
              " nodes, depth " + std::to_string(p.max_depth) + ")";
        return kErrModel;
    }
    const bool strict = (flags & 1u) != 0;
    const char *cmp = strict ? " > " : " >= ";
    std::string s;
    s.reserve(size_t(64) * p.nodes.size() + 1024);
    s += "// generated: " + std::to_string(n_trees) + " trees, " + std::to_string(p.nodes.size()) +
         " nodes, right iff x" + cmp + "theta\n";
    const int32_t n_funcs = (n_trees + kCodegenTreesPerFunction - 1) / kCodegenTreesPerFunction;
    // explicit stack: (node, depth, phase) with phase 0 = open the node, 1 = between branches,
    // 2 = close
    struct Item {
        int32_t node, depth, phase;
    };
    std::vector<Item> stack;
    for (int32_t t = 0; t < n_trees; t++) {
        const int64_t a = tree_offsets[t];
        if (t % kCodegenTreesPerFunction == 0)
            s += "__device__ __attribute__((noinline)) double trees_" +
                 std::to_string(t / kCodegenTreesPerFunction) +
                 "(const float *__restrict__ x) {\n    double acc = 0.0;\n    float v;\n";
        s += "    // tree " + std::to_string(t) + "\n";
        stack.assign(1, Item{0, 1, 0});
        while (!stack.empty()) {
            Item it = stack.back();
            stack.pop_back();
            const std::string ind(size_t(4 * it.depth), ' ');
            const int64_t n = a + it.node;
            if (feature[n] < 0) {
                s += ind + "v = " + float_literal(value[n]) + ";\n";
                continue;
            }
            if (it.phase == 0) {
                s += ind + "if (x[" + std::to_string(feature[n]) + "]" + cmp + float_literal(threshold[n]) +
                     ") {\n";
                stack.push_back(Item{it.node, it.depth, 1});
                stack.push_back(Item{right[n], it.depth + 1, 0});
            } else if (it.phase == 1) {
                s += ind + "} else {\n";
                stack.push_back(Item{it.node, it.depth, 2});
                stack.push_back(Item{left[n], it.depth + 1, 0});
            } else {
                s += ind + "}\n";
            }
        }
        s += "    acc += (double)v;\n";
        if (t % kCodegenTreesPerFunction == kCodegenTreesPerFunction - 1 || t == n_trees - 1)
            s += "    return acc;\n}\n";
    }
    s += "extern \"C\" __global__ void __launch_bounds__(" + std::to_string(kCodegenThreads) + ")\n";
    s += "tree_ens_cg(const float *__restrict__ X, long long n_docs, int n_features,\n"
         "            float *__restrict__ scores, double scale) {\n";
    s += "    const long long d = (long long)blockIdx.x * " + std::to_string(kCodegenThreads) +
         " + threadIdx.x;\n";
    s += "    if (d >= n_docs)\n        return;\n";
    s += "    const float *__restrict__ x = X + d * (long long)n_features;\n";
    s += "    double acc = 0.0;\n";
    for (int32_t k = 0; k < n_funcs; k++)
        s += "    acc += trees_" + std::to_string(k) + "(x);\n";
    s += "    scores[d] = (float)(acc * scale);\n}\n";
    src = std::move(s);
    return kOk;
}

} // namespace treeens
