// Launch entry points of the HIP kernels (host side).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.h"

namespace infs {

// Which instantiation of the decode kernel serves a context.
struct KernelKey {
  int bf16;        // 0: fp32 Q/K/V, 1: bf16
  int head_dim;    // 64 or 128
  int hpk;         // query heads per KV head
  int mfma;        // 1: prefix rows go through MFMA tiles, 0: wavefront reductions
  int prefix_rows; // rows of one prompt's prefix work item, padded (wave: 8/16; MFMA: 16/32/64/128)
  int kv8;         // 1: K/V stored as E4M3 (bf16 MFMA shapes of head_dim 128)
};

// Resolve the padded prefix row count and path for a shape; false if no
// instantiation exists.
bool select_kernel(int bf16, int head_dim, int hpk, int prefix_rows_real, int kv8, KernelKey* key);

// The same with the prefix path fixed (mfma 1: MFMA tiles, 0: wavefront
// reductions): a second kernel of a context must read the prefix store in the
// layout its first kernel chose.
bool select_kernel_path(int bf16, int head_dim, int hpk, int prefix_rows_real, int mfma, int kv8, KernelKey* key);

// Record layout of the split-K workspace for a key.
int64_t workspace_records(const KernelKey& key, int num_prompts, int hkv, int prefix_chunks_max,
                          int num_slots, int suffix_chunks_max);

// Prefix store elements per (prompt, kv head) for a key and capacity.
int64_t prefix_elems_per_head(const KernelKey& key, int max_prompt_len_padded);

hipError_t launch_decode(const KernelKey& key, const StepArgs& args, int grid, hipStream_t stream);

// The step launch through every layer (args.num_layers layers).
hipError_t launch_layers(const KernelKey& key, const StepArgs& args, int grid, hipStream_t stream);

// Work-groups of the step-launch kernel of `key` that the current device keeps
// resident at once (occupancy per compute unit times compute units).
hipError_t layers_resident(const KernelKey& key, int* resident);

// The decode kernel instantiations, spread over several translation units
// (inst_*.hip) so that they compile in parallel.
struct KernelEntry {
  KernelKey key;
  void (*decode[2])(const StepArgs);  // [0]: partials through the coherence point, [1]: through the XCD's L2
  void (*layers[2])(const StepArgs);  // step launch through every layer: [0] partials through the coherence
                                      // point, [1] through the XCD's L2
};
struct KernelTable {
  const KernelEntry* entries;
  int count;
};
KernelTable kernels_wave_f32_d64();    // fp32, head_dim 64 (wavefront reductions)
KernelTable kernels_wave_f32_d128();   // fp32, head_dim 128
KernelTable kernels_wave_bf16_d64();   // bf16 below 16 prefix rows, head_dim 64
KernelTable kernels_wave_bf16_d128();  // bf16 below 16 prefix rows, head_dim 128
KernelTable kernels_mfma_d64();    // bf16, head_dim 64, MFMA prefix tiles
KernelTable kernels_mfma_d128a();  // bf16, head_dim 128, hpk 1 and 2
KernelTable kernels_mfma_d128b();  // bf16, head_dim 128, hpk 4 and 8
KernelTable kernels_kv8a();        // E4M3 K/V, head_dim 128, hpk 1 and 2
KernelTable kernels_kv8b();        // E4M3 K/V, head_dim 128, hpk 4 and 8

// Record the XCD each of `blocks` work-groups runs on: out[b] = XCC id of work-group b.
hipError_t launch_xcd_probe(int32_t* out, int blocks, hipStream_t stream);

// Device address of this GPU's static scratch array (kStaticScratchBytes,
// 256-byte aligned), looked up with hipGetSymbolAddress on the first call for
// the current device and kept per device.
hipError_t static_scratch_ptr(void** out);

// Zero n 32-bit words at p on `stream` (a small fill kernel).
hipError_t launch_zero_words(uint32_t* p, int64_t n, hipStream_t stream);

// Copy one prompt's K/V [plen, Hkv, D] into the shared-prefix store (layout chosen by key).
hipError_t launch_prefill(const KernelKey& key, void* prefix_layer, const void* k, const void* v,
                          int prompt, int plen, int hkv, int max_prompt_len_padded, hipStream_t stream);

}  // namespace infs
