// Single-tree kernels for uint8 (ordered discrete) records (kernel templates in kernels_impl.hpp).
#include "kernels_impl.hpp"

namespace dtree {

const void *kernel_for_u8(int algo, int row_stride, int load_mode, bool tables_in_lds, int depth) {
    return single_tree_kernel<kXU8>(algo, row_stride, load_mode, tables_in_lds, depth);
}

}  // namespace dtree
