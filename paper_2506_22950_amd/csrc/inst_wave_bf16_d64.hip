// Decode kernel instantiations: bf16 with fewer than 16 prefix rows, head_dim 64, wavefront reductions; 1/2/4/8 query heads per KV head, 8 or 16 padded rows.
#include "layers.h"

namespace infs {
namespace {

#define INFS_ENTRY(bf, d, hpk, mf, pr) {{bf, d, hpk, mf, pr, 0}, {decode_kernel<Shape<bf, d, hpk, mf, pr>, false>, decode_kernel<Shape<bf, d, hpk, mf, pr>, true>}, {layers_kernel<Shape<bf, d, hpk, mf, pr>, false>, layers_kernel<Shape<bf, d, hpk, mf, pr>, true>}},

const KernelEntry kEntries[] = {
    INFS_ENTRY(true, 64, 1, false, 8)
    INFS_ENTRY(true, 64, 1, false, 16)
    INFS_ENTRY(true, 64, 2, false, 8)
    INFS_ENTRY(true, 64, 2, false, 16)
    INFS_ENTRY(true, 64, 4, false, 8)
    INFS_ENTRY(true, 64, 4, false, 16)
    INFS_ENTRY(true, 64, 8, false, 8)
    INFS_ENTRY(true, 64, 8, false, 16)
};

}  // namespace

KernelTable kernels_wave_bf16_d64() { return {kEntries, (int)(sizeof(kEntries) / sizeof(kEntries[0]))}; }

}  // namespace infs
