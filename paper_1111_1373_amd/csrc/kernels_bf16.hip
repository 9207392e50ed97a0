// Single-tree kernels for bfloat16 records (kernel templates in kernels_impl.hpp).
#include "kernels_impl.hpp"

namespace dtree {

const void *kernel_for_bf16(int algo, int row_stride, int load_mode, bool tables_in_lds, int depth) {
    return single_tree_kernel<kXBF16>(algo, row_stride, load_mode, tables_in_lds, depth);
}

}  // namespace dtree
