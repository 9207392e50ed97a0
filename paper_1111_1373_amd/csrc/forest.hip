// gfx950 forest kernel: majority vote of many trees over every record (kernel template in
// forest_impl.hpp).  This unit holds the instances for int32 exit codes and the launch.
#include "forest_impl.hpp"

namespace dtree {

const void *forest_kernel_for(int algo, int row_stride, int load_mode, bool tables_in_lds,
                              int vote_words, int depth, int exit_mode) {
    if (exit_mode == 2)
        return forest_kernel_for_packed(algo, row_stride, load_mode, tables_in_lds, vote_words,
                                        depth);
    if (exit_mode == 1)
        return forest_kernel_for_ex16(algo, row_stride, load_mode, tables_in_lds, vote_words,
                                      depth);
    return forest_kernel_for_ex<int32_t>(algo, row_stride, load_mode, tables_in_lds,
                                         vote_words, depth);
}

hipError_t launch_forest(const void *fn, const FArgs &args, int blocks, int lds_bytes,
                         hipStream_t stream) {
    FArgs a = args;
    void *params[] = {&a};
    return hipLaunchKernel(fn, dim3(unsigned(blocks)), dim3(unsigned(args.waves * 64)), params,
                           size_t(lds_bytes), stream);
}

}  // namespace dtree
