// Forest kernel instances for int16 exit codes (kernel template in forest_impl.hpp).
#include "forest_impl.hpp"

namespace dtree {

const void *forest_kernel_for_ex16(int algo, int row_stride, int load_mode, bool tables_in_lds,
                                   int vote_words, int depth) {
    return forest_kernel_for_ex<int16_t>(algo, row_stride, load_mode, tables_in_lds,
                                         vote_words, depth);
}

}  // namespace dtree
