// Single-tree kernels for IEEE binary16 records (kernel templates in kernels_impl.hpp).
#include "kernels_impl.hpp"

namespace dtree {

const void *kernel_for_f16(int algo, int row_stride, int load_mode, bool tables_in_lds, int depth) {
    return single_tree_kernel<kXF16>(algo, row_stride, load_mode, tables_in_lds, depth);
}

}  // namespace dtree
