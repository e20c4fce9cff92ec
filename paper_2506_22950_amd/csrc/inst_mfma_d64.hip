// Decode kernel instantiations: bf16, head_dim 64, prefix on MFMA tiles of 16/32/64/128 padded rows, 1/2/4/8 query heads per KV head.
#include "layers.h"

namespace infs {
namespace {

#define INFS_ENTRY(bf, d, hpk, mf, pr) {{bf, d, hpk, mf, pr, 0}, {decode_kernel<Shape<bf, d, hpk, mf, pr>, false>, decode_kernel<Shape<bf, d, hpk, mf, pr>, true>}, {layers_kernel<Shape<bf, d, hpk, mf, pr>, false>, layers_kernel<Shape<bf, d, hpk, mf, pr>, true>}},

const KernelEntry kEntries[] = {
    INFS_ENTRY(true, 64, 1, true, 16)
    INFS_ENTRY(true, 64, 1, true, 32)
    INFS_ENTRY(true, 64, 1, true, 64)
    INFS_ENTRY(true, 64, 2, true, 16)
    INFS_ENTRY(true, 64, 2, true, 32)
    INFS_ENTRY(true, 64, 2, true, 64)
    INFS_ENTRY(true, 64, 2, true, 128)
    INFS_ENTRY(true, 64, 4, true, 16)
    INFS_ENTRY(true, 64, 4, true, 32)
    INFS_ENTRY(true, 64, 4, true, 64)
    INFS_ENTRY(true, 64, 4, true, 128)
    INFS_ENTRY(true, 64, 8, true, 16)
    INFS_ENTRY(true, 64, 8, true, 32)
    INFS_ENTRY(true, 64, 8, true, 64)
    INFS_ENTRY(true, 64, 8, true, 128)
};

}  // namespace

KernelTable kernels_mfma_d64() { return {kEntries, (int)(sizeof(kEntries) / sizeof(kEntries[0]))}; }

}  // namespace infs
