// Decode kernel instantiations: E4M3 K/V cache, bf16 compute, head_dim 128, MFMA prefix tiles, 4 or 8 query heads per KV head.
#include "layers.h"

namespace infs {
namespace {

#define INFS_ENTRY(d, hpk, pr) {{1, d, hpk, 1, pr, 1}, {decode_kernel<Shape<true, d, hpk, true, pr, true>, false>, decode_kernel<Shape<true, d, hpk, true, pr, true>, true>}, {layers_kernel<Shape<true, d, hpk, true, pr, true>, false>, layers_kernel<Shape<true, d, hpk, true, pr, true>, true>}},

const KernelEntry kEntries[] = {
    INFS_ENTRY(128, 4, 16)
    INFS_ENTRY(128, 4, 32)
    INFS_ENTRY(128, 4, 64)
    INFS_ENTRY(128, 4, 128)
    INFS_ENTRY(128, 8, 16)
    INFS_ENTRY(128, 8, 32)
    INFS_ENTRY(128, 8, 64)
    INFS_ENTRY(128, 8, 128)
};

}  // namespace

KernelTable kernels_kv8b() { return {kEntries, (int)(sizeof(kEntries) / sizeof(kEntries[0]))}; }

}  // namespace infs
