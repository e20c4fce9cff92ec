// Step launch through every layer: one persistent launch decodes all layers of
// a running step (every decode step passes through all layers, Section 2.1).
//
// The grid holds as many work-groups as the GPU keeps resident at once, so
// every work-group runs from the start and none waits for a slot.  Per KV
// head g, n_pre_wg work-groups take the step's prefix chunks and n_suf_wg its
// response pieces (each live response cut into near-equal page ranges, see
// step_plan.h), round robin, for every layer in turn (the same items every
// layer).  Of the n_merge_wg merge work-groups of the head, wavefront k
// handles slots k, k + 4 * n_merge_wg, ... of every layer, one (slot, KV
// head) merge per wavefront at a time (an idle slot only gets its O rows
// zeroed).
//
// Layer order.  In a real model the queries and the new K/V rows of layer l
// come from layer l-1's outputs, so a producer of layer l > 0 reads them only
// after every merge of layer l-1 of its prompt has completed (a per-prompt
// "merged" counter); the cached prefix and response K/V of layer l do not
// depend on layer l-1, so a producer issues those loads first and waits only
// before it needs the queries.  Merges count on the merged counter after
// their O stores have completed, and the merge that completes a layer raises
// a per-KV-head flag that the producers of that head poll.
//
// Split-K partials go through the device coherence point (write-through
// stores, loads that miss the caches) or, in the XCD-local exchange (every
// work-group of a KV head on one XCD, as in the per-layer launch), through
// that XCD's L2 (stores stop there).  With several layers per launch the same
// record addresses are rewritten and reread, so a merge's loads miss the CU's
// L1 in both modes (device-scope loads): an L1 line kept from an earlier
// layer's read is never returned.  The workspace is safe to rewrite because a producer of
// layer l writes only after every merge of layer l-1 of its prompt has read
// its partials.
//
// Every wait is bounded by merge_polls (and gives up at once once any wait of
// the launch has given up, or when merge_polls < 0); a wait that gives up sets
// the status word and the launch runs to its end with invalid outputs.
//
// Memory-queue sharing.  The GPU keeps two of these work-groups on every CU,
// and the vector memory instructions of a CU pass through one queue to the
// memory system, which a CU drains at a bounded rate.  A work-group that
// issues its next layer's K/V loads while the other work-group of its CU
// still has this layer's partial stores or merges to do puts those behind
// the whole stream.  So a response work-group issues its next layer's loads
// only once its CU mate is past its part of the layer (or after a short
// bound), a prefix work-group -- whose chunk is small and whose partial is
// needed early -- loads its next layer's chunk only when that layer may
// start, and the host places the merge work-groups on the CUs of prefix
// work-groups, whose queues are then empty while the merges run.  Which
// work-groups share a CU is read from the hardware (see mate_gate); none of
// this affects results.
#pragma once
#include <type_traits>

#include "decode.h"
#include "step_plan.h"

namespace infs {
namespace {

// Layer-l views of the launch's buffers.
struct LayerView {
  const char* q;       // [S, Hq, d]
  const char* knew;    // [S, Hkv, d]
  const char* vnew;
  float* o;            // [S, Hq, d]
  const char* prefix;  // shared-prefix store of the layer
  char* pool;          // response page pool of the layer
  int layer;
};

__device__ __forceinline__ LayerView layer_view(const StepArgs& a, int l) {
  LayerView v;
  v.q = (const char*)a.q + l * a.q_layer_stride;
  v.knew = (const char*)a.knew + l * a.kv_layer_stride;
  v.vnew = (const char*)a.vnew + l * a.kv_layer_stride;
  v.o = (float*)((char*)a.o + l * a.o_layer_stride);
  v.prefix = (const char*)a.prefix + l * a.prefix_layer_bytes;
  v.pool = (char*)a.pool + l * a.pool_layer_bytes;
  v.layer = l;
  return v;
}

// One lane: wait until *ctr has reached target, polling at most merge_polls
// times.  Gives up at once when merge_polls < 0 or when the status word
// shows that another wait of the launch has given up.
__device__ bool bounded_wait(const StepArgs& a, const int32_t* ctr, int32_t target) {
  if (a.merge_polls < 0) return false;
  if (reached(ctr, target)) return true;
  if (__hip_atomic_load(a.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) return false;
  for (int spins = 0; spins < a.merge_polls; ++spins) {
    __builtin_amdgcn_s_sleep(2);
    if (reached(ctr, target)) return true;
  }
  return false;
}

// The "layer done" flag of prompt p for KV head g: the merge that completes a
// layer of the prompt (the last one to count on its merged counter) writes the
// counter's final value into one flag line per KV head, and producers poll the
// line of their own head -- one counter line polled by every producer of the
// GPU would hold up the merges' own atomics on it.
__device__ __forceinline__ int32_t* layer_flag(const StepArgs& a, int p, int g) {
  return a.merged + ((int64_t)a.num_prompts + (int64_t)p * a.Hkv + g) * kCounterStride;
}

// All threads of a producer work-group of KV head g: wait until every merge of
// layer l-1 of prompt p has completed.
__device__ void wait_layer(const StepArgs& a, int p, int l) {
  if (threadIdx.x == 0) {
    const int32_t target = (int32_t)((uint32_t)a.merged_base[p] + (uint32_t)l * (uint32_t)a.merged_per_layer[p]);
    if (!bounded_wait(a, layer_flag(a, p, blockIdx.x % a.Hkv), target))
      __hip_atomic_store(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
}

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding: vmcnt
// bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).  Vector memory operations of
// one wavefront complete in issue order, so when only the n most recent ones
// may still be outstanding, every earlier one has completed.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// A producer work-group has stored its partial and then issued the loads of its
// next item (NEXT load instructions per wavefront, 0 without a next item): once
// every wavefront's stores have completed -- all but its NEXT most recent
// memory operations -- count one arrival on each live slot among first ..
// first + n - 1, as arrive() does.  The next item's loads stay in flight.
template <int NEXT>
__device__ __forceinline__ void arrive_behind(const StepArgs& a, int first, int n, int g) {
  asm volatile("" ::: "memory");
  wait_vmcnt<NEXT>();
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  // liveness from the plan's bitmask: reading a.slot[first + lane] would be a
  // per-lane read of the argument block, a vector load whose wait would also
  // wait for the next item's loads
  if ((int)threadIdx.x < n && ((a.live_mask >> (first + threadIdx.x)) & 1))
    __hip_atomic_fetch_add(a.counters + (int64_t)((first + threadIdx.x) * a.Hkv + g) * kCounterStride, 1,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wavefront path registers: one load round of K and V (U 16-byte chunks each).
template <class SH, int NR>
struct WaveRegs {
  static constexpr int U = WaveCfg<SH, NR>::U;
  u32x4 kk[U], vv[U];
};

// Issue the loads of one round (tokens base .. base + U * TPI - 1 of the
// wavefront range [t0, t1)) into R; 2 * U load instructions.  Rows past t1 are
// loaded in bounds and masked later.
template <class SH, int NR, class Addr>
__device__ __forceinline__ void wave_load_round(const Addr& ad, int t0, int t1, int base, WaveRegs<SH, NR>& R) {
  constexpr int TPI = SH::TPI, U = WaveRegs<SH, NR>::U;
  constexpr int SB = U >= 8 ? 4 : U;
  constexpr int NSB = U / SB;
  constexpr int PGI = (U * TPI + 15) / 16;
  int pg[PGI];
#pragma unroll
  for (int i = 0; i < PGI; ++i) pg[i] = ad.page(((base - t0) >> 4) + i);
#pragma unroll
  for (int b = 0; b < NSB; ++b) {
#pragma unroll
    for (int kind = 0; kind < 2; ++kind)
#pragma unroll
      for (int u = b * SB; u < b * SB + SB; ++u) {
        u32x4& dst = kind ? R.vv[u] : R.kk[u];
        dst = ld_kv<SH, Addr::kNonTemporal>(ad.row(kind, base + u * TPI, base - t0 + u * TPI, pg[(u * TPI) >> 4], t1));
      }
  }
}

// wave_partial over [t0, t1) with the first round already in R (loaded by
// wave_load_round(ad, t0, t1, t0, R)); later rounds are loaded here.
template <class SH, int NR, class Addr>
__device__ __forceinline__ void wave_compute(const Addr& ad, int t0, int t1, const u32x4 (&q)[NR], float sl2,
                                             WaveRegs<SH, NR>& R, float (&m)[NR], float (&l)[NR],
                                             float (&o)[NR][SH::EPL]) {
  constexpr int LPT = SH::LPT, TPI = SH::TPI, EPL = SH::EPL, U = WaveRegs<SH, NR>::U;
  constexpr int SB = U >= 8 ? 4 : U;
  constexpr int NSB = U / SB;
  static_assert(U % SB == 0 && SB % 2 == 0, "sub-blocks of token pairs");
  const int lane = threadIdx.x & 63, ts = lane / LPT;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    m[r] = NEG_INF;
    l[r] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[r][e] = 0.f;
  }
  for (int base = t0; base < t1; base += U * TPI) {
    if (base != t0) wave_load_round<SH, NR>(ad, t0, t1, base, R);
#pragma unroll
    for (int b = 0; b < NSB; ++b) {
      float s[SB][NR];
#pragma unroll
      for (int x = 0; x < SB; ++x) {
        const int u = b * SB + x;
        const bool ok = base + u * TPI + ts < t1;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          const float y = group_sum<LPT>(dot16B<SH::BF>(R.kk[u], q[r])) * sl2;
          s[x][r] = ok ? y : NEG_INF;
        }
      }
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        float mb = s[0][r];
#pragma unroll
        for (int x = 1; x < SB; ++x) mb = fmaxf(mb, s[x][r]);
        const float mn = fmaxf(m[r], mb);
        const float mu = (mn == NEG_INF) ? 0.f : mn;
        const float corr = exp2_fast(m[r] - mu);
        m[r] = mn;
        l[r] *= corr;
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[r][e] *= corr;
        if constexpr (SH::BF) {
#pragma unroll
          for (int x = 0; x < SB; x += 2) {
            const int u = b * SB + x;
            const __bf16 h0 = (__bf16)exp2_fast(s[x][r] - mu), h1 = (__bf16)exp2_fast(s[x + 1][r] - mu);
            l[r] += (float)h0 + (float)h1;
            const bf16x2 pb = {h0, h1};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const uint32_t lo = __builtin_amdgcn_perm(R.vv[u + 1][k], R.vv[u][k], 0x05040100u);
              const uint32_t hi = __builtin_amdgcn_perm(R.vv[u + 1][k], R.vv[u][k], 0x07060302u);
              o[r][2 * k] = __builtin_amdgcn_fdot2_f32_bf16(pb, __builtin_bit_cast(bf16x2, lo), o[r][2 * k], false);
              o[r][2 * k + 1] = __builtin_amdgcn_fdot2_f32_bf16(pb, __builtin_bit_cast(bf16x2, hi), o[r][2 * k + 1], false);
            }
          }
        } else {
#pragma unroll
          for (int x = 0; x < SB; ++x) {
            const float p = exp2_fast(s[x][r] - mu);
            l[r] += p;
            axpy16B<false>(o[r], p, R.vv[b * SB + x]);
          }
        }
      }
    }
  }
}

// Query rows of the prefix work item of prompt p, KV head g (rows
// slot_in_prompt * hpk + j; rows of idle slots and padding rows are zero).
template <class SH, int PR>
__device__ __forceinline__ void load_prefix_q(const StepArgs& a, const LayerView& V, int p, int g, u32x4 (&q)[PR]) {
  constexpr int HPK = SH::HPK;
  const int ch = (threadIdx.x & 63) % SH::LPT;
#pragma unroll
  for (int r = 0; r < PR; ++r) {
    const int si = r / HPK, j = r - si * HPK, s = p * a.m + min(si, a.m - 1);
    if (r < a.prefix_rows && a.slot[s].len > 0)
      q[r] = *((const u32x4*)(V.q + ((int64_t)s * a.Hq + g * HPK + j) * SH::ROWB) + ch);
    else
      q[r] = u32x4{0, 0, 0, 0};
  }
}

// Prefix item k of the step (prompt p, chunk c) and this wavefront's range.
struct PrefixItem {
  int p, c, t0, t1;
  int nbc;  // 32-token blocks of a whole chunk (the MFMA tiles split them over their token groups)
};
__device__ __forceinline__ PrefixItem prefix_item(const StepArgs& a, int k) {
  int p = 0;
  while (p < a.num_prompts - 1 && !(a.prompt[p].nchunks > 0 && k < a.prompt[p].item_begin + a.prompt[p].nchunks)) ++p;
  PrefixItem it;
  it.p = p;
  it.c = k - a.prompt[p].item_begin;
  it.t0 = it.c * a.prefix_split;
  it.t1 = min(it.t0 + a.prefix_split, a.prompt[p].plen);
  it.nbc = a.prefix_split / kMfmaBlock;
  return it;
}

// ---- Prefix chunk on the wavefront path (see prefix_wave) -------------------
template <class SH, bool L2>
struct PrefixWave {
  using Regs = WaveRegs<SH, SH::PR>;
  static constexpr int kLoads = 2 * Regs::U;  // load instructions of issue()
  __device__ __forceinline__ static void range(const StepArgs& a, const PrefixItem& it, int& wt0, int& wt1) {
    const int w = threadIdx.x >> 6, sub = a.prefix_split / 4;
    wt0 = min(it.t0 + w * sub, it.t1);
    wt1 = min(wt0 + sub, it.t1);
  }
  __device__ __forceinline__ static PrefixAddr<SH> addr(const StepArgs& a, const LayerView& V, int p, int g) {
    const int64_t head = ((int64_t)p * a.Hkv + g) * 2;
    return PrefixAddr<SH>{{V.prefix + head * a.max_prompt_len * SH::KROWB,
                           V.prefix + (head + 1) * a.max_prompt_len * SH::KROWB}};
  }
  // Loads of the first round (also for an empty range: in bounds, masked).
  __device__ __forceinline__ static void issue(const StepArgs& a, const LayerView& V, const PrefixItem& it, int g, Regs& R) {
    int wt0, wt1;
    range(a, it, wt0, wt1);
    wave_load_round<SH, SH::PR>(addr(a, V, it.p, g), wt0, wt1, wt0, R);
  }
  template <class Before, class After>
  __device__ __forceinline__ static void finish(const StepArgs& a, const LayerView& V, const PrefixItem& it, int g, float* smem,
                                Regs& R, Before&& before, After&& after_stores) {
    constexpr int PR = SH::PR;
    int wt0, wt1;
    range(a, it, wt0, wt1);
    before();
    u32x4 q[PR];
    load_prefix_q<SH, PR>(a, V, it.p, g, q);
    float m[PR], l[PR], o[PR][SH::EPL];
    wave_compute<SH, PR>(addr(a, V, it.p, g), wt0, wt1, q, a.scale_log2, R, m, l, o);
    wave_combine_groups<SH, PR>(m, l, o);
    const int64_t rec0 = (((int64_t)it.p * a.Hkv + g) * a.prefix_chunks_max + it.c) * PR;
    block_store_partial<SH, PR, L2>(smem, m, l, o, Exchange<L2>(a), rec0);
    after_stores();
  }
};

// ---- Prefix chunk on MFMA tiles (see prefix_mfma) ---------------------------
template <class SH, bool L2>
struct PrefixMfma {
  static constexpr int D = SH::D, KB = SH::KB, DB = SH::DB;
  static constexpr bool PREFETCH_V = SH::NBW == 1;
  // issue() loads a second block only where a wavefront can have two
  static constexpr bool ISSUE_TWO = PREFETCH_V && SH::BPW > 1;
  struct Regs {
    bf16x8 ka[2][KB], va[DB], kn[2][KB], vn[DB];
  };
  static constexpr int kBlockLoads = 2 * KB + DB;  // load instructions of one block
  // This wavefront's blocks [b0, b1) of the chunk: its token group's share of
  // the chunk's blocks (a step launch's chunks hold twice the per-layer
  // launch's, see kStepPrefixSplit).
  __device__ __forceinline__ static void blocks(const PrefixItem& it, int& nblk, int& b0, int& b1) {
    const int tg = (threadIdx.x >> 6) / SH::RG, bpw = it.nbc / SH::TG;
    nblk = (it.t1 - it.t0 + kMfmaBlock - 1) / kMfmaBlock;
    b0 = tg * bpw;
    b1 = min(b0 + bpw, nblk);
  }
  __device__ __forceinline__ static const char* head(const StepArgs& a, const LayerView& V, const PrefixItem& it, int g) {
    return V.prefix + ((int64_t)(it.p * a.Hkv + g) * (a.max_prompt_len / kMfmaBlock)) * (2 * kMfmaBlock * D * SH::KES);
  }
  __device__ __forceinline__ static void fetch_k(const char* hd, const PrefixItem& it, int b, bf16x8 (&ka)[2][KB]) {
    const int lane = threadIdx.x & 63;
    const char* kblk = hd + (int64_t)((it.t0 + b * kMfmaBlock) / kMfmaBlock) * (2 * kMfmaBlock * D * SH::KES);
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        ka[mb][kb] = __builtin_bit_cast(bf16x8, ld_kv<SH, false>(kblk + ((mb * KB + kb) * 64 + lane) * 8 * SH::KES));
  }
  __device__ __forceinline__ static void fetch_v(const char* hd, const PrefixItem& it, int b, bf16x8 (&va)[DB]) {
    const int lane = threadIdx.x & 63;
    const char* vblk = hd + (int64_t)((it.t0 + b * kMfmaBlock) / kMfmaBlock) * (2 * kMfmaBlock * D * SH::KES) +
                       kMfmaBlock * D * SH::KES;
#pragma unroll
    for (int db = 0; db < DB; ++db) va[db] = __builtin_bit_cast(bf16x8, ld_kv<SH, false>(vblk + (db * 64 + lane) * 8 * SH::KES));
  }
  // Whether issue() also loads the wavefront's second block.
  __device__ __forceinline__ static bool pre_next(const PrefixItem& it) {
    int nblk, b0, b1;
    blocks(it, nblk, b0, b1);
    return ISSUE_TWO && b0 + 1 < b1;
  }
  // The wavefront's first block (a wavefront without blocks loads the chunk's
  // last block -- in bounds, never used) and, with one tile per wavefront, its
  // second: kBlockLoads or 2 * kBlockLoads load instructions.
  __device__ __forceinline__ static void issue(const StepArgs& a, const LayerView& V, const PrefixItem& it, int g, Regs& R) {
    int nblk, b0, b1;
    blocks(it, nblk, b0, b1);
    const char* hd = head(a, V, it, g);
    const int bf = b0 < b1 ? b0 : nblk - 1;
    fetch_k(hd, it, bf, R.ka);
    fetch_v(hd, it, bf, R.va);
    if (ISSUE_TWO && b0 + 1 < b1) {
      fetch_k(hd, it, b0 + 1, R.kn);
      fetch_v(hd, it, b0 + 1, R.vn);
    }
  }
  template <class Before, class After>
  __device__ __forceinline__ static void finish(const StepArgs& a, const LayerView& V, const PrefixItem& it, int g, float* smem,
                                Regs& R, Before&& before, After&& after_stores) {
    constexpr int HPK = SH::HPK, NBW = SH::NBW, RG = SH::RG, TG = SH::TG;
    using WS = Shape<true, D, HPK, true, NBW * 16>;
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, q4 = lane >> 4, r16 = lane & 15;
    const int rg = w % RG, tg = w / RG;
    int nblk, b0, b1;
    blocks(it, nblk, b0, b1);
    const bool pre = ISSUE_TWO && b0 + 1 < b1;
    const char* hd = head(a, V, it, g);
    before();
    bf16x8 bq[NBW][KB];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      const int row = (rg * NBW + nb) * 16 + r16, si = row / HPK, j = row - si * HPK, s = it.p * a.m + min(si, a.m - 1);
      const bool ok = row < a.prefix_rows && a.slot[s].len > 0;
      const uint16_t* qr = (const uint16_t*)V.q + ((int64_t)s * a.Hq + g * HPK + j) * D;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) bq[nb][kb] = ok ? *(const bf16x8*)(qr + kb * 32 + q4 * 8) : bf16x8{};
    }
    f32x4 acc[NBW][DB];
    float mrow[NBW], lrow[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      mrow[nb] = NEG_INF;
      lrow[nb] = 0.f;
#pragma unroll
      for (int db = 0; db < DB; ++db) acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    // The next block's loads are in flight while a block is multiplied (with two
    // tiles per wavefront, only its K).  Where issue() loads a second block it
    // lands in R.kn / R.vn; elsewhere the next block goes to local registers.
    if constexpr (ISSUE_TWO) {
      for (int b = b0; b < b1; ++b) {
        const bool more = b + 1 < b1;
        if (more && !(b == b0 && pre)) {
          fetch_k(hd, it, b + 1, R.kn);
          fetch_v(hd, it, b + 1, R.vn);
        }
        mfma_block<WS>(R.ka, R.va, bq, it.t0 + b * kMfmaBlock, it.t1, a.scale_log2, acc, mrow, lrow);
        if (more) {
#pragma unroll
          for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) R.ka[mb][kb] = R.kn[mb][kb];
#pragma unroll
          for (int db = 0; db < DB; ++db) R.va[db] = R.vn[db];
        }
      }
    } else {
      bf16x8 kn[2][KB], vn[DB];
      for (int b = b0; b < b1; ++b) {
        const bool more = b + 1 < b1;
        if (more) {
          fetch_k(hd, it, b + 1, kn);
          if constexpr (PREFETCH_V) fetch_v(hd, it, b + 1, vn);
        }
        mfma_block<WS>(R.ka, R.va, bq, it.t0 + b * kMfmaBlock, it.t1, a.scale_log2, acc, mrow, lrow);
        if (more) {
#pragma unroll
          for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) R.ka[mb][kb] = kn[mb][kb];
          if constexpr (PREFETCH_V) {
#pragma unroll
            for (int db = 0; db < DB; ++db) R.va[db] = vn[db];
          } else {
            fetch_v(hd, it, b + 1, R.va);
          }
        }
      }
    }
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      lrow[nb] += __shfl_xor(lrow[nb], 16);
      lrow[nb] += __shfl_xor(lrow[nb], 32);
    }
    const int64_t rec0 = (((int64_t)it.p * a.Hkv + g) * a.prefix_chunks_max + it.c) * SH::PR;
    const Exchange<L2> ex(a);
    if constexpr (TG == 1) {
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) {
        const int64_t rec = rec0 + (rg * NBW + nb) * 16 + r16;
#pragma unroll
        for (int db = 0; db < DB; ++db) ex.store4((uint32_t)((rec * D + db * 16 + q4 * 4) * 4), acc[nb][db]);
        if (q4 == 0) ex.store_ml(rec, mrow[nb], lrow[nb]);
      }
    } else {
      constexpr int OFL = NBW * DB * 64 * 4;
      {
        float* sl = smem + w * SH::MFMA_SLOT;
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) {
#pragma unroll
          for (int db = 0; db < DB; ++db) *(f32x4*)(sl + ((nb * DB + db) * 64 + lane) * 4) = acc[nb][db];
          sl[OFL + nb * 64 + lane] = mrow[nb];
          sl[OFL + NBW * 64 + nb * 64 + lane] = lrow[nb];
        }
      }
      __syncthreads();
      constexpr int DBW = DB / TG;
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) {
        float M = NEG_INF;
#pragma unroll
        for (int t = 0; t < TG; ++t) M = fmaxf(M, smem[(t * RG + rg) * SH::MFMA_SLOT + OFL + nb * 64 + lane]);
        const float Mu = (M == NEG_INF) ? 0.f : M;
        float wv[TG], L = 0.f;
#pragma unroll
        for (int t = 0; t < TG; ++t) {
          const float* sl = smem + (t * RG + rg) * SH::MFMA_SLOT;
          wv[t] = exp2_fast(sl[OFL + nb * 64 + lane] - Mu);
          L += wv[t] * sl[OFL + NBW * 64 + nb * 64 + lane];
        }
        const int64_t rec = rec0 + (rg * NBW + nb) * 16 + r16;
#pragma unroll
        for (int x = 0; x < DBW; ++x) {
          const int db = tg * DBW + x;
          f32x4 acc4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int t = 0; t < TG; ++t)
            acc4 += *(const f32x4*)(smem + (t * RG + rg) * SH::MFMA_SLOT + ((nb * DB + db) * 64 + lane) * 4) * wv[t];
          ex.store4((uint32_t)((rec * D + db * 16 + q4 * 4) * 4), acc4);
        }
        if (tg == 0 && q4 == 0) ex.store_ml(rec, M, L);
      }
    }
    after_stores();
  }
};

// ---- Response chunk, fp32 pages on wavefront dot products (see suffix_chunk) -
struct RespItem {
  int s, c, len, wt0, wt1, last;
  bool has_new;  // this wavefront's range holds the newest token
  bool tail;     // the item is the slot's last piece
};
__device__ __forceinline__ RespItem resp_item(const StepArgs& a, int it) {
  // The slot of response item `it`: slots' first items never decrease and an
  // idle slot adds none, so it is the last slot whose first item is <= it.  A
  // binary search with uniform indices reads the plan with scalar loads only.
  int lo = 0, hi = a.S - 1;
  while (lo < hi) {
    const int mid = __builtin_amdgcn_readfirstlane((lo + hi + 1) >> 1);
    if (a.slot[mid].item_begin <= it)
      lo = mid;
    else
      hi = mid - 1;
  }
  const int s = __builtin_amdgcn_readfirstlane(lo);
  RespItem r;
  r.s = s;
  r.c = it - a.slot[s].item_begin;
  r.len = a.slot[s].len;
  const int n = a.slot[s].pieces, w = threadIdx.x >> 6;
  if (a.resp_cut) {
    // piece c of n near-equal page ranges; wavefront w takes the w-th run of
    // ppw pages of it
    const int pages = (r.len + kPageTokens - 1) / kPageTokens;
    const int pg0 = piece_first_page(r.c, pages, n), pg1 = piece_first_page(r.c + 1, pages, n);
    const int ppw = piece_wave_pages(pg1 - pg0);
    const int t1 = min(pg1 * kPageTokens, r.len);
    r.wt0 = min((pg0 + w * ppw) * kPageTokens, t1);
    r.wt1 = min(r.wt0 + ppw * kPageTokens, t1);
  } else {
    // chunk c of `split` tokens, a quarter per wavefront
    const int sub = a.split / kWaves, t0 = r.c * a.split, t1 = min(t0 + a.split, r.len);
    r.wt0 = min(t0 + w * sub, t1);
    r.wt1 = min(r.wt0 + sub, t1);
  }
  r.tail = r.c == n - 1;
  r.last = r.len - 1;
  r.has_new = r.last >= r.wt0 && r.last < r.wt1;
  return r;
}
// Page numbers of this wavefront's range (lane i: its i-th 16-token page).
__device__ __forceinline__ int resp_pages(const StepArgs& a, const RespItem& r) {
  const int lane = threadIdx.x & 63;
  const int npg = (r.wt1 - r.wt0 + kPageTokens - 1) / kPageTokens;
  const int32_t* ptab = a.page_table + (int64_t)a.slot[r.s].seq * a.pages_per_slot + (r.wt0 >> 4);
  return lane < npg ? ptab[lane] : 0;
}

template <class SH, bool L2>
struct Resp {
  static constexpr int HPK = SH::HPK;
  using Regs = WaveRegs<SH, HPK>;
  static constexpr int kLoads = 2 * Regs::U;
  __device__ __forceinline__ static void issue(const StepArgs& a, const LayerView& V, const RespItem& r, int pages, int g, Regs& R) {
    SuffixAddr<SH> ad{(const char*)V.pool, pages, a.Hkv, g};
    wave_load_round<SH, HPK>(ad, r.wt0, r.has_new ? r.last : r.wt1, r.wt0, R);
  }
  template <class Before, class After>
  __device__ __forceinline__ static void finish(const StepArgs& a, const LayerView& V, const RespItem& r, int pages, int g,
                                float* smem, Regs& R, Before&& before, After&& after_stores) {
    const int lane = threadIdx.x & 63, ch = lane % SH::LPT;
    const SlotPlan& sp = a.slot[r.s];
    const int64_t newrow = ((int64_t)r.s * a.Hkv + g) * SH::ROWB;
    before();
    u32x4 q[HPK];
#pragma unroll
    for (int i = 0; i < HPK; ++i) q[i] = *((const u32x4*)(V.q + ((int64_t)r.s * a.Hq + g * HPK + i) * SH::ROWB) + ch);
    u32x4 knew = u32x4{0, 0, 0, 0}, vnew = u32x4{0, 0, 0, 0};
    if (r.has_new) {
      knew = *((const u32x4*)(V.knew + newrow) + ch);
      vnew = *((const u32x4*)(V.vnew + newrow) + ch);
      if constexpr (SH::KV8) {
        knew = widen_e4m3(narrow_e4m3(knew));
        vnew = widen_e4m3(narrow_e4m3(vnew));
      }
    }
    SuffixAddr<SH> ad{(const char*)V.pool, pages, a.Hkv, g};
    float m[HPK], l[HPK], o[HPK][SH::EPL];
    wave_compute<SH, HPK>(ad, r.wt0, r.has_new ? r.last : r.wt1, q, a.scale_log2, R, m, l, o);
    if (r.has_new) {
      fold_token<SH, HPK>(knew, vnew, q, a.scale_log2, m, l, o);
      if (lane < SH::LPT) {
        char* row = V.pool + (int64_t)(sp.cur_page * a.Hkv + g) * 2 * SH::PAGEB + (r.last & 15) * SH::KROWB + ch * SH::LANEB;
        st_kv<SH>(row, knew);
        st_kv<SH>(row + SH::PAGEB, vnew);
      }
    }
    wave_combine_groups<SH, HPK>(m, l, o);
    if (V.layer == 0 && r.tail && g == 0 && threadIdx.x == 0) {
      // bookkeeping of this step's token, once per step (its K/V are stored above)
      a.page_table[(int64_t)sp.seq * a.pages_per_slot + (r.last >> 4)] = sp.cur_page;
      __hip_atomic_fetch_add(&a.tokens[(r.s / a.m) * a.G + sp.sample], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const int64_t rec0 = prefix_records(a, SH::PR) + (((int64_t)r.s * a.Hkv + g) * a.suffix_chunks_max + r.c) * HPK;
    block_store_partial<SH, HPK, L2>(smem, m, l, o, Exchange<L2>(a), rec0);
    after_stores();
  }
};

// The same response item on MFMA tiles (bf16 and E4M3 pages; see RespMfma):
// issue() loads the wavefront's first round, finish() runs the rest once the
// item's queries may be read.
template <class SH, bool L2>
struct RespTiles {
  using RM = RespMfma<SH>;
  using Regs = typename RM::Regs;
  static constexpr int HPK = SH::HPK;
  static constexpr int kLoads = RM::kLoads;
  __device__ __forceinline__ static void issue(const StepArgs& a, const LayerView& V, const RespItem& r, int pages, int g, Regs& R) {
    RM::load_round(V.pool, pages, a.Hkv, g, 0, R);
  }
  template <class Before, class After>
  __device__ __forceinline__ static void finish(const StepArgs& a, const LayerView& V, const RespItem& r, int pages, int g,
                                float* smem, Regs& R, Before&& before, After&& after_stores) {
    const SlotPlan& sp = a.slot[r.s];
    const int te = r.has_new ? r.last : r.wt1;
    before();
    // queries and the newest token's rows in one batch of loads, issued as soon
    // as the layer may read them; that token is folded in first
    bf16x8 bq[SH::KB];
    RM::load_q(V.q, (int64_t)r.s * a.Hq + g * HPK, bq);
    typename RM::NewRows N;
    if (r.has_new) {
      const int64_t newrow = ((int64_t)r.s * a.Hkv + g) * SH::ROWB;
      RM::load_new(V.knew + newrow, V.vnew + newrow, N);
    }
    typename RM::Acc A;
    if (r.has_new) {
      RM::round_new(N);
      RM::start_new(N, bq, a.scale_log2, A);
      RM::store_new((char*)RM::page(V.pool, sp.cur_page, a.Hkv, g), r.last & 15, N);
    } else {
      RM::init(A);
    }
    for (int base = r.wt0; base < te; base += RM::TOK) {
      if (base != r.wt0) RM::load_round(V.pool, pages, a.Hkv, g, (base - r.wt0) >> 4, R);
      RM::round(R, bq, base, te, a.scale_log2, A);
    }
    if (V.layer == 0 && r.tail && g == 0 && threadIdx.x == 0) {
      // bookkeeping of this step's token, once per step (its K/V are stored above)
      a.page_table[(int64_t)sp.seq * a.pages_per_slot + (r.last >> 4)] = sp.cur_page;
      __hip_atomic_fetch_add(&a.tokens[(r.s / a.m) * a.G + sp.sample], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    RM::publish(smem, A);
    const int64_t rec0 = prefix_records(a, SH::PR) + (((int64_t)r.s * a.Hkv + g) * a.suffix_chunks_max + r.c) * HPK;
    combine_store_partial<SH, HPK, L2>(smem, Exchange<L2>(a), rec0);
    after_stores();
  }
};

// One wavefront merges every partial of (slot s, KV head g) of one layer and
// writes O rows g*hpk .. +hpk-1 (the log-sum-exp combination of the split-K
// partial softmaxes, in partial order).  Lane x of vector v holds outputs
// 4 * (v * 64 + x) .. +3; partials are loaded MCW at a time.
template <class SH>
struct MergeWaveShape {
  static constexpr int OPP = SH::HPK * SH::D;
  static constexpr int MV = (OPP / 4 + 63) / 64;
  static constexpr int MCW = MV == 1 ? 24 : MV == 2 ? 8 : 4;
};

template <class SH, bool L2>
__device__ void merge_wave(const StepArgs& a, const LayerView& V, int s, int g, int32_t target) {
  using MW = MergeWaveShape<SH>;
  constexpr int D = SH::D, HPK = SH::HPK, MV = MW::MV, MCW = MW::MCW;
  const int lane = threadIdx.x & 63;
  const int p = s / a.m, si = s - p * a.m;
  float* orow = V.o + ((int64_t)s * a.Hq + g * HPK) * D;
  int ok = 0;
  if (lane == 0) {
    ok = bounded_wait(a, slot_counter(a, s, g), target);
    if (!ok) __hip_atomic_store(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  ok = __builtin_amdgcn_readfirstlane(ok);
  if (!ok) {
#pragma unroll
    for (int v = 0; v < MV; ++v) {
      const int x = (v * 64 + lane) * 4;
      if (x < MW::OPP) *(f32x4*)(orow + x) = f32x4{1.f, 1.f, 1.f, 1.f} * __builtin_nanf("");
    }
    return;
  }
  const int nP = a.prompt[p].nchunks;
  const int n = nP + a.slot[s].pieces;
  const int64_t pbase = ((int64_t)p * a.Hkv + g) * a.prefix_chunks_max * SH::PR + si * HPK;
  const int64_t sbase = prefix_records(a, SH::PR) + ((int64_t)s * a.Hkv + g) * a.suffix_chunks_max * HPK;
  auto rec = [&](int c, int j) -> int64_t { return (c < nP ? pbase + (int64_t)c * SH::PR : sbase + (int64_t)(c - nP) * HPK) + j; };
  const Exchange<L2, true> ex(a);
  float M[MV], L[MV];
  f32x4 O[MV];
#pragma unroll
  for (int v = 0; v < MV; ++v) {
    M[v] = NEG_INF;
    L[v] = 0.f;
    O[v] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int c0 = 0; c0 < n; c0 += MCW) {
    u32x2 ml[MCW][MV];
    f32x4 ov[MCW][MV];
#pragma unroll
    for (int u = 0; u < MCW; ++u) {
      const int c = c0 + u;
#pragma unroll
      for (int v = 0; v < MV; ++v) {
        const int x = (v * 64 + lane) * 4, j = x / D, d = x - j * D;
        if (c < n && x < MW::OPP) {
          const int64_t r = rec(c, j);
          ml[u][v] = ex.load_ml(r);
          ov[u][v] = ex.load4((uint32_t)((r * D + d) * 4));
        } else {
          ml[u][v] = u32x2{__float_as_uint(NEG_INF), 0u};
          ov[u][v] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
    }
#pragma unroll
    for (int u = 0; u < MCW; ++u)
#pragma unroll
      for (int v = 0; v < MV; ++v) {
        const float mc = __uint_as_float(ml[u][v].x), lc = __uint_as_float(ml[u][v].y);
        const float nm = fmaxf(M[v], mc);
        const float base = nm == NEG_INF ? 0.f : nm;
        const float al = exp2_fast(M[v] - base), be = mc == NEG_INF ? 0.f : exp2_fast(mc - base);
        L[v] = L[v] * al + lc * be;
        O[v] = O[v] * al + ov[u][v] * be;
        M[v] = nm;
      }
  }
#pragma unroll
  for (int v = 0; v < MV; ++v) {
    const int x = (v * 64 + lane) * 4;
    if (x < MW::OPP) *(f32x4*)(orow + x) = O[v] * (1.f / L[v]);
  }
}

// Role of work-group index j of a KV head (see StepArgs::merge_j0): 0 prefix,
// 1 response, 2 merge, with its index among the work-groups of that role.
__device__ __forceinline__ int wg_role(const StepArgs& a, int j, int& idx) {
  if (j < a.n_pre_wg) {
    idx = j;
    return 0;
  }
  if (j >= a.merge_j0 && j < a.merge_j0 + a.n_merge_wg) {
    idx = j - a.merge_j0;
    return 2;
  }
  idx = j - a.n_pre_wg - (j >= a.merge_j0 + a.n_merge_wg ? a.n_merge_wg : 0);
  return 1;
}

// Hardware id of the CU running this work-group (XCD, shader engine, array, CU).
__device__ __forceinline__ int32_t cu_id() {
  const int32_t hw = __builtin_amdgcn_s_getreg(4 | (31 << 11));  // HW_REG_HW_ID: CU id in bits 8..15
  return ((hw >> 8) & 0xff) | ((__builtin_amdgcn_s_getreg(kXccIdReg) & 15) << 8);
}
__device__ __forceinline__ int32_t* peer_line(const StepArgs& a, int b) { return a.peer + (int64_t)b * kCounterStride; }
// Wavefront w of this work-group (a producer: the work-group, w = 0) is done with layer l.
__device__ __forceinline__ void peer_mark(const StepArgs& a, int l, int w) {
  __hip_atomic_store(peer_line(a, blockIdx.x) + w, (int32_t)((uint32_t)a.peer_base + (uint32_t)l + 1u),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// All threads of a producer work-group that is done with layer l: wait until
// the other work-group of its CU is too, at most kMateWaitTicks.  The grid
// holds two work-groups per CU and the dispatcher gives every CU one before
// any gets a second, so work-group b shares its CU with b +- gridDim.x / 2,
// which for KV head g is index j +- nj / 2; the pair waits only when the CU
// ids they recorded at their start agree.
__device__ void mate_gate(const StepArgs& a, int l) {
  const int nj = gridDim.x / a.Hkv;
  if (threadIdx.x < kWaves && (nj & 1) == 0 && a.merge_polls >= 0) {
    const int g = blockIdx.x % a.Hkv, j = blockIdx.x / a.Hkv;
    const int jm = j < nj / 2 ? j + nj / 2 : j - nj / 2;
    const int w = threadIdx.x;
    // a merge mate is not waited for: its part of the layer comes last (the host places merges
    // opposite prefix work-groups, which load their next layer only when it may start)
    int im;
    const int rm = wg_role(a, jm, im);
    const bool need = w == 0 && (rm == 0 ? im < a.n_prefix_items : rm == 1 ? im < a.n_suffix_items : false);
    const int32_t* line = peer_line(a, jm * a.Hkv + g);
    if (need && __hip_atomic_load(line + 4, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == cu_id() + 1) {
      const int32_t target = (int32_t)((uint32_t)a.peer_base + (uint32_t)l + 1u);
      const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
      while (__hip_atomic_load(line + w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) - target < 0 &&
             __builtin_amdgcn_s_memrealtime() - t0 < (uint64_t)kMateWaitTicks)
        __builtin_amdgcn_s_sleep(2);
    }
  }
  __syncthreads();
}

// Layer l > 0 of prompt p may start once the prompt's layer l-1 is merged;
// `ready` remembers the prompts a work-group has already seen done in l.
__device__ __forceinline__ void layer_gate(const StepArgs& a, int p, int l, uint32_t& ready) {
  if (l > 0 && !((ready >> p) & 1u)) {
    wait_layer(a, p, l);
    ready |= 1u << p;
  }
}

// Prefix-chunk work-group jp of KV head g: prefix items jp, jp + n_pre_wg, ...
// of every layer.  The layer's first item is loaded once the layer may start;
// a later item of the same layer is loaded right behind the previous item's
// stores.
template <class SH, bool L2>
__device__ __forceinline__ void prefix_loop(const StepArgs& a, int g, int jp, float* smem) {
  if (jp >= a.n_prefix_items) return;
  const int nk = (a.n_prefix_items - jp + a.n_pre_wg - 1) / a.n_pre_wg;
  using P = std::conditional_t<SH::MFMA, PrefixMfma<SH, L2>, PrefixWave<SH, L2>>;
  typename P::Regs R;
  for (int l = 0; l < a.num_layers; ++l) {
    const LayerView V = layer_view(a, l);
    uint32_t ready = 0;
    for (int k = 0; k < nk; ++k) {
      const PrefixItem it = prefix_item(a, jp + k * a.n_pre_wg);
      if (k == 0) {
        layer_gate(a, it.p, l, ready);
        P::issue(a, V, it, g, R);
      }
      P::finish(a, V, it, g, smem, R, [&]() { layer_gate(a, it.p, l, ready); },
                [&]() {
                  arrive_behind<0>(a, it.p * a.m, a.m, g);
                  if (k + 1 < nk)
                    P::issue(a, V, prefix_item(a, jp + (k + 1) * a.n_pre_wg), g, R);
                  else if (threadIdx.x == 0)
                    peer_mark(a, l, 0);
                });
    }
  }
}

// Response-chunk work-group jr of KV head g: response items jr, jr + n_suf_wg,
// ... of every layer, each with the next item's loads issued behind its stores
// (behind the CU mate's part of the layer when the next item is in the next
// layer).
template <class SH, bool L2>
__device__ __forceinline__ void suffix_loop(const StepArgs& a, int g, int jr, float* smem) {
  if (jr >= a.n_suffix_items) return;
  const int nk = (a.n_suffix_items - jr + a.n_suf_wg - 1) / a.n_suf_wg;
  using P = std::conditional_t<SH::BF, RespTiles<SH, L2>, Resp<SH, L2>>;
  typename P::Regs R;
  RespItem it = resp_item(a, jr);
  int pages = resp_pages(a, it);
  P::issue(a, layer_view(a, 0), it, pages, g, R);
  for (int l = 0; l < a.num_layers; ++l) {
    const LayerView V = layer_view(a, l);
    uint32_t ready = 0;
    for (int k = 0; k < nk; ++k) {
      it = resp_item(a, jr + k * a.n_suf_wg);
      const bool has_next = k + 1 < nk || l + 1 < a.num_layers;
      const int ln = k + 1 < nk ? l : l + 1;
      P::finish(a, V, it, pages, g, smem, R, [&]() { layer_gate(a, it.s / a.m, l, ready); },
                [&]() {
                  if (!has_next) {
                    arrive_behind<0>(a, it.s, 1, g);
                    if (threadIdx.x == 0) peer_mark(a, l, 0);
                    return;
                  }
                  // With one item per layer the next item is this one in the next layer, on the same
                  // pages; otherwise its page numbers are read here, and the wait for them also
                  // waits for this item's stores.
                  const RespItem nx = resp_item(a, jr + (k + 1 < nk ? k + 1 : 0) * a.n_suf_wg);
                  if (nk != 1) pages = resp_pages(a, nx);
                  arrive_behind<0>(a, it.s, 1, g);
                  if (ln != l) {  // the next item is in the next layer: let the CU mate finish this one first
                    if (threadIdx.x == 0) peer_mark(a, l, 0);
                    mate_gate(a, l);
                  }
                  P::issue(a, layer_view(a, ln), nx, pages, g, R);
                });
    }
  }
}

template <class SH, bool L2>
__device__ void merge_loop(const StepArgs& a, int g, int mj) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int nent = a.n_merge_items + a.n_zero_items;
  for (int l = 0; l < a.num_layers; ++l) {
    const LayerView V = layer_view(a, l);
    for (int e = mj * kWaves + w; e < nent; e += a.n_merge_wg * kWaves) {
      if (e < a.n_merge_items) {
        const int s = a.live_slot[e];
        const int p = s / a.m;
        const uint32_t per = (uint32_t)(a.slot[s].pieces + a.prompt[p].nchunks);
        const int32_t target = (int32_t)((uint32_t)a.slot[s].target + (uint32_t)(l + 1) * per);
        merge_wave<SH, L2>(a, V, s, g, target);
        // Counted once this wavefront's partial loads and O stores have completed;
        // the merge that completes the prompt's layer raises every head's flag.
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_s_waitcnt(0);
        int32_t before_count = 0;
        if (lane == 0)
          before_count = __hip_atomic_fetch_add(a.merged + (int64_t)p * kCounterStride, 1, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
        before_count = __builtin_amdgcn_readfirstlane(before_count);
        const int32_t done =
            (int32_t)((uint32_t)a.merged_base[p] + (uint32_t)(l + 1) * (uint32_t)a.merged_per_layer[p]);
        if (before_count + 1 == done && lane < a.Hkv)
          __hip_atomic_store(layer_flag(a, p, lane), done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      } else {
        const int s = a.zero_slot[e - a.n_merge_items];
        float* orow = V.o + ((int64_t)s * a.Hq + g * SH::HPK) * SH::D;
        for (int x = lane * 4; x < SH::HPK * SH::D; x += 256) *(f32x4*)(orow + x) = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    if (lane == 0) peer_mark(a, l, w);
  }
}

// The step launch.  Timing mode as in decode_kernel (one start / end pair for
// the whole launch).
template <class SH, bool L2>
__global__ __launch_bounds__(kBlockThreads, SH::MIN_WAVES) void layers_kernel(const StepArgs a) {
  __shared__ __attribute__((aligned(16))) float smem[SH::SMEM > 4 ? SH::SMEM : 4];
  const int cs = (blockIdx.x % kClockSlots) * kClockStride;
  if (a.clock_start && threadIdx.x == 0)
    __hip_atomic_fetch_min(a.clock_start + cs, (unsigned long long)__builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
  if (threadIdx.x == 0) __hip_atomic_store(peer_line(a, blockIdx.x) + 4, cu_id() + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (L2 && threadIdx.x == 0 &&
      (__builtin_amdgcn_s_getreg(kXccIdReg) & 15) != (int)((blockIdx.x + a.l2_check_shift) % a.l2_xcds))
    __hip_atomic_store(a.status, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int g = blockIdx.x % a.Hkv, j = blockIdx.x / a.Hkv;
  int idx;
  const int role = wg_role(a, j, idx);
  if (role == 0)
    prefix_loop<SH, L2>(a, g, idx, smem);
  else if (role == 1)
    suffix_loop<SH, L2>(a, g, idx, smem);
  else
    merge_loop<SH, L2>(a, g, idx);
  if (a.clock_start) {
    __syncthreads();
    if (threadIdx.x == 0)
      __hip_atomic_fetch_max(a.clock_end + cs, (unsigned long long)__builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
  }
}

}  // namespace
}  // namespace infs
