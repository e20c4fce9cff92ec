// Decode kernel instantiations: bf16, head_dim 128, prefix on MFMA tiles of 16/32/64/128 padded rows, 1 or 2 query heads per KV head.
#include "layers.h"

namespace infs {
namespace {

#define INFS_ENTRY(bf, d, hpk, mf, pr) {{bf, d, hpk, mf, pr, 0}, {decode_kernel<Shape<bf, d, hpk, mf, pr>, false>, decode_kernel<Shape<bf, d, hpk, mf, pr>, true>}, {layers_kernel<Shape<bf, d, hpk, mf, pr>, false>, layers_kernel<Shape<bf, d, hpk, mf, pr>, true>}},

const KernelEntry kEntries[] = {
    INFS_ENTRY(true, 128, 1, true, 16)
    INFS_ENTRY(true, 128, 1, true, 32)
    INFS_ENTRY(true, 128, 1, true, 64)
    INFS_ENTRY(true, 128, 2, true, 16)
    INFS_ENTRY(true, 128, 2, true, 32)
    INFS_ENTRY(true, 128, 2, true, 64)
    INFS_ENTRY(true, 128, 2, true, 128)
};

}  // namespace

KernelTable kernels_mfma_d128a() { return {kEntries, (int)(sizeof(kEntries) / sizeof(kEntries[0]))}; }

}  // namespace infs
