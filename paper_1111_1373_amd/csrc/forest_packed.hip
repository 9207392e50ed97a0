// Forest kernel instances with exit codes packed into the windows' bottom slots (kernel
// template in forest_impl.hpp; data walk only).
#include "forest_impl.hpp"

namespace dtree {

const void *forest_kernel_for_packed(int algo, int row_stride, int load_mode,
                                     bool tables_in_lds, int vote_words, int depth) {
    if (algo != kAlgoData) return nullptr;
    return forest_kernel_for_ex<dev::PackedExits>(algo, row_stride, load_mode, tables_in_lds,
                                                  vote_words, depth);
}

}  // namespace dtree
