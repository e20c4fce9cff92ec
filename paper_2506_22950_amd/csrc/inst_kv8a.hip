// Decode kernel instantiations: E4M3 K/V cache, bf16 compute, head_dim 128, MFMA prefix tiles, 1 or 2 query heads per KV head.
#include "layers.h"

namespace infs {
namespace {

#define INFS_ENTRY(d, hpk, pr) {{1, d, hpk, 1, pr, 1}, {decode_kernel<Shape<true, d, hpk, true, pr, true>, false>, decode_kernel<Shape<true, d, hpk, true, pr, true>, true>}, {layers_kernel<Shape<true, d, hpk, true, pr, true>, false>, layers_kernel<Shape<true, d, hpk, true, pr, true>, true>}},

const KernelEntry kEntries[] = {
    INFS_ENTRY(128, 1, 16)
    INFS_ENTRY(128, 1, 32)
    INFS_ENTRY(128, 1, 64)
    INFS_ENTRY(128, 2, 16)
    INFS_ENTRY(128, 2, 32)
    INFS_ENTRY(128, 2, 64)
    INFS_ENTRY(128, 2, 128)
};

}  // namespace

KernelTable kernels_kv8a() { return {kEntries, (int)(sizeof(kEntries) / sizeof(kEntries[0]))}; }

}  // namespace infs
