// Single-tree kernels for fp32 records, and the dispatch over element types, load modes and
// algorithms (kernel templates in kernels_impl.hpp).
#include "kernels_impl.hpp"

namespace dtree {

const void *kernel_for_f32(int algo, int row_stride, int load_mode, bool tables_in_lds, int depth) {
    return single_tree_kernel<kXF32>(algo, row_stride, load_mode, tables_in_lds, depth);
}

const void *kernel_for(int algo, int elem_type, int row_stride, int load_mode, bool tables_in_lds,
                       int depth) {
    if (algo == kAlgoPath)
        return elem_type == kXF32 ? path_kernel_for(row_stride, load_mode, tables_in_lds, depth)
                                  : nullptr;
    switch (elem_type) {
        case kXF32: return kernel_for_f32(algo, row_stride, load_mode, tables_in_lds, depth);
        case kXF16: return kernel_for_f16(algo, row_stride, load_mode, tables_in_lds, depth);
        case kXBF16: return kernel_for_bf16(algo, row_stride, load_mode, tables_in_lds, depth);
        case kXU8: return kernel_for_u8(algo, row_stride, load_mode, tables_in_lds, depth);
        default: return nullptr;
    }
}

hipError_t prepare_kernel(const void *fn, int max_lds_bytes) {
    return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, max_lds_bytes);
}

hipError_t launch_kernel(const void *fn, const KArgs &args, int blocks, int lds_bytes,
                         hipStream_t stream) {
    KArgs a = args;
    void *params[] = {&a};
    return hipLaunchKernel(fn, dim3(unsigned(blocks)), dim3(unsigned(args.waves * 64)), params,
                           size_t(lds_bytes), stream);
}

}  // namespace dtree
