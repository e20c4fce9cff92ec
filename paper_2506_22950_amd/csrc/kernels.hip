// Host side of the decode kernels: the instantiation registry, kernel
// selection, the launches, and the prefill kernels.  The device code (and what
// the kernels compute) is in decode.h; the decode kernel instantiations are in
// inst_*.hip.
#include "layers.h"

namespace infs {
namespace {

const KernelEntry* find_entry(const KernelKey& k) {
  static const KernelTable tables[] = {kernels_wave_f32_d64(),  kernels_wave_f32_d128(), kernels_wave_bf16_d64(),
                                       kernels_wave_bf16_d128(), kernels_mfma_d64(),      kernels_mfma_d128a(),
                                       kernels_mfma_d128b(), kernels_kv8a(),     kernels_kv8b()};
  for (const KernelTable& t : tables)
    for (int i = 0; i < t.count; ++i) {
      const KernelEntry& e = t.entries[i];
      if (e.key.bf16 == k.bf16 && e.key.head_dim == k.head_dim && e.key.hpk == k.hpk && e.key.mfma == k.mfma &&
          e.key.prefix_rows == k.prefix_rows && e.key.kv8 == k.kv8)
        return &e;
    }
  return nullptr;
}

}  // namespace

bool select_kernel(int bf16, int head_dim, int hpk, int rows, int kv8, KernelKey* key) {
  return select_kernel_path(bf16, head_dim, hpk, rows, bf16 && rows >= 16, kv8, key);
}

bool select_kernel_path(int bf16, int head_dim, int hpk, int rows, int mfma, int kv8, KernelKey* key) {
  KernelKey k{bf16, head_dim, hpk, mfma && bf16 ? 1 : 0, 0, kv8 ? 1 : 0};
  if (k.mfma)
    k.prefix_rows = rows <= 16 ? 16 : rows <= 32 ? 32 : rows <= 64 ? 64 : rows <= 128 ? 128 : 0;
  else
    k.prefix_rows = rows <= 8 ? 8 : rows <= 16 ? 16 : 0;
  if (k.prefix_rows == 0 || !find_entry(k)) return false;
  *key = k;
  return true;
}

int64_t workspace_records(const KernelKey& key, int num_prompts, int hkv, int prefix_chunks_max, int num_slots,
                          int suffix_chunks_max) {
  return (int64_t)num_prompts * prefix_chunks_max * hkv * key.prefix_rows +
         (int64_t)num_slots * suffix_chunks_max * hkv * key.hpk;
}

int64_t prefix_elems_per_head(const KernelKey& key, int pmax_padded) {
  // elements, whatever their size (E4M3 bytes with key.kv8)
  return (int64_t)2 * pmax_padded * key.head_dim;
}

hipError_t launch_decode(const KernelKey& key, const StepArgs& args, int grid, hipStream_t stream) {
  const KernelEntry* e = find_entry(key);
  if (!e) return hipErrorInvalidValue;
  hipLaunchKernelGGL(e->decode[args.l2_xcds > 0 ? 1 : 0], dim3(grid), dim3(kBlockThreads), 0, stream, args);
  return hipGetLastError();
}

hipError_t launch_layers(const KernelKey& key, const StepArgs& args, int grid, hipStream_t stream) {
  const KernelEntry* e = find_entry(key);
  if (!e) return hipErrorInvalidValue;
  hipLaunchKernelGGL(e->layers[args.l2_xcds > 0 ? 1 : 0], dim3(grid), dim3(kBlockThreads), 0, stream, args);
  return hipGetLastError();
}

hipError_t layers_resident(const KernelKey& key, int* resident) {
  const KernelEntry* e = find_entry(key);
  if (!e) return hipErrorInvalidValue;
  int per_cu = 0, dev = 0, cus = 0;
  hipError_t err = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, e->layers[0], kBlockThreads, 0);
  if (err == hipSuccess) err = hipGetDevice(&dev);
  if (err == hipSuccess) err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (err != hipSuccess) return err;
  *resident = per_cu * cus;
  return hipSuccess;
}

#define INFS_PREFILL_CASE(bf, d, mf, k8)                                                               \
  if (key.bf16 == bf && key.head_dim == d && key.mfma == mf && key.kv8 == (k8 ? 1 : 0)) {              \
    using SH = Shape<bf, d, 1, mf, mf ? 16 : 8, k8>;                                                   \
    if constexpr (mf)                                                                                  \
      hipLaunchKernelGGL(prefill_mfma_kernel<SH>, dim3(grid), dim3(256), 0, stream, (char*)store,      \
                         (const uint16_t*)k, (const uint16_t*)v, prompt, plen, hkv, pmax);             \
    else                                                                                               \
      hipLaunchKernelGGL(prefill_plain_kernel<SH>, dim3(grid), dim3(256), 0, stream, (char*)store,     \
                         (const char*)k, (const char*)v, prompt, plen, hkv, pmax);                     \
    return hipGetLastError();                                                                          \
  }

namespace {
__global__ __launch_bounds__(64) void xcd_probe_kernel(int32_t* out) {
  if (threadIdx.x == 0) out[blockIdx.x] = __builtin_amdgcn_s_getreg(kXccIdReg) & 15;
}
}  // namespace

hipError_t launch_xcd_probe(int32_t* out, int blocks, hipStream_t stream) {
  hipLaunchKernelGGL(xcd_probe_kernel, dim3(blocks), dim3(64), 0, stream, out);
  return hipGetLastError();
}

hipError_t launch_prefill(const KernelKey& key, void* store, const void* k, const void* v, int prompt, int plen,
                          int hkv, int pmax, hipStream_t stream) {
  if (plen == 0) return hipSuccess;
  const int64_t units = (int64_t)hkv * 2 * ((plen + 31) / 32) * 32 * key.head_dim;
  const int grid = (int)((units / 8 + 255) / 256 < 4096 ? (units / 8 + 255) / 256 : 4096);
  INFS_PREFILL_CASE(false, 64, 0, false)
  INFS_PREFILL_CASE(false, 128, 0, false)
  INFS_PREFILL_CASE(true, 64, 0, false)
  INFS_PREFILL_CASE(true, 128, 0, false)
  INFS_PREFILL_CASE(true, 64, 1, false)
  INFS_PREFILL_CASE(true, 128, 1, false)
  INFS_PREFILL_CASE(true, 128, 1, true)
  return hipErrorInvalidValue;
}

}  // namespace infs
