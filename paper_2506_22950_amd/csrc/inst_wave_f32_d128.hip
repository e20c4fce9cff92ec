// Decode kernel instantiations: fp32 Q/K/V, head_dim 128, wavefront reductions; 1/2/4/8 query heads per KV head, 8 or 16 padded rows.
#include "layers.h"

namespace infs {
namespace {

#define INFS_ENTRY(bf, d, hpk, mf, pr) {{bf, d, hpk, mf, pr, 0}, {decode_kernel<Shape<bf, d, hpk, mf, pr>, false>, decode_kernel<Shape<bf, d, hpk, mf, pr>, true>}, {layers_kernel<Shape<bf, d, hpk, mf, pr>, false>, layers_kernel<Shape<bf, d, hpk, mf, pr>, true>}},

const KernelEntry kEntries[] = {
    INFS_ENTRY(false, 128, 1, false, 8)
    INFS_ENTRY(false, 128, 1, false, 16)
    INFS_ENTRY(false, 128, 2, false, 8)
    INFS_ENTRY(false, 128, 2, false, 16)
    INFS_ENTRY(false, 128, 4, false, 8)
    INFS_ENTRY(false, 128, 4, false, 16)
    INFS_ENTRY(false, 128, 8, false, 8)
    INFS_ENTRY(false, 128, 8, false, 16)
};

}  // namespace

KernelTable kernels_wave_f32_d128() { return {kEntries, (int)(sizeof(kEntries) / sizeof(kEntries[0]))}; }

}  // namespace infs
