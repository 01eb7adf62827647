/* Lets the HIP source that TREE_ENS_CODEGEN generates compile as plain C++ on the CPU (tests
 * only): the launch attributes vanish and the block and thread indices are globals that the
 * driver sets before calling the entry point once per document. */
#define __global__
#define __device__
#define __launch_bounds__(x)
struct CgIndex {
    unsigned x;
};
static CgIndex blockIdx, threadIdx;
