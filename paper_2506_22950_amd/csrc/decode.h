// HIP kernels for gfx950 (CDNA4): shared-prefix continuous-sampling decode.
//
// One launch per layer-step does all the device work of that layer:
//   * append: each live slot's new K/V row goes into its response pages;
//   * split-K attention over the shared prefix: one work-group per
//     (prompt, KV head, prefix chunk: 128 tokens on MFMA tiles, `split`
//     tokens otherwise).  Every K/V byte of the chunk is read from HBM once
//     and used by all m * hpk query rows of that
//     KV head -- the rows of every live slot of the prompt.  With >= 16 rows
//     the two contractions run on MFMA tiles (v_mfma_f32_16x16x32_bf16);
//     below that, on wavefront dot products;
//   * split-K attention over each live slot's private response (hpk rows per
//     KV byte, wavefront dot products);
//   * log-sum-exp merge: one work-group per live (slot, KV head), placed at
//     the end of the grid, waits (bounded) until every chunk of that slot has
//     published its partial, combines the partial softmaxes and writes O.
// Idle slots get O = 0.
//
// A partial over a key set J is (M, L, O) with scores in log2 units
// (s_j = scale * log2(e) * q.k_j): M = max_j s_j, L = sum_j 2^(s_j - M),
// O = sum_j 2^(s_j - M) v_j.  Two partials combine exactly as
// M = max(M1, M2), L = 2^(M1-M) L1 + 2^(M2-M) L2, O likewise, and the result
// is O / L.
//
// This header holds the device code; every kernel translation unit includes it
// and instantiates the shapes it serves (its copies have internal linkage).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "kernels.h"

namespace infs {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

#define NEG_INF (-__builtin_huge_valf())

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Lane permutations inside 16-lane DPP rows (row_mask = bank_mask = all).
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over each aligned group of N consecutive lanes; every lane gets its group's sum.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(N == 2 || N == 4 || N == 8 || N == 16 || N == 32 || N == 64, "group size");
  x += dpp<0xB1>(x);                       // quad_perm [1,0,3,2]: lane ^ 1
  if constexpr (N >= 4) x += dpp<0x4E>(x); // quad_perm [2,3,0,1]: lane ^ 2
  if constexpr (N == 8) x += dpp<0x141>(x);  // row_half_mirror: quad 0 <-> quad 1
  if constexpr (N >= 16) {
    x += dpp<0x124>(x);                    // row_ror:4
    x += dpp<0x128>(x);                    // row_ror:8
  }
  if constexpr (N >= 32) x += __shfl_xor(x, 16);
  if constexpr (N >= 64) x += __shfl_xor(x, 32);
  return x;
}

// Combine partial (m2, l2) into (m, l); returns the weights of the old and new parts.
__device__ __forceinline__ void lse_combine(float& m, float& l, float m2, float l2, float& a, float& b) {
  const float mn = fmaxf(m, m2);
  const float mu = (mn == NEG_INF) ? 0.f : mn;
  a = exp2_fast(m - mu);
  b = exp2_fast(m2 - mu);
  l = l * a + l2 * b;
  m = mn;
}

// 16-byte chunk helpers: 8 bf16 or 4 fp32 elements.
template <bool BF>
__device__ __forceinline__ float dot16B(const u32x4& k, const u32x4& q) {
  if constexpr (BF) {
    // Pairs are taken with shufflevector from a whole-vector cast: casting the
    // individual 32-bit lanes to bf16x2 is mis-lowered by this compiler (all
    // four dots read the same dword).
    const bf16x8 kv = __builtin_bit_cast(bf16x8, k), qv = __builtin_bit_cast(bf16x8, q);
    float s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(kv, kv, 0, 1), __builtin_shufflevector(qv, qv, 0, 1), 0.f, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(kv, kv, 2, 3), __builtin_shufflevector(qv, qv, 2, 3), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(kv, kv, 4, 5), __builtin_shufflevector(qv, qv, 4, 5), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(kv, kv, 6, 7), __builtin_shufflevector(qv, qv, 6, 7), s, false);
    return s;
  } else {
    float s = __uint_as_float(k.x) * __uint_as_float(q.x);
    s = fmaf(__uint_as_float(k.y), __uint_as_float(q.y), s);
    s = fmaf(__uint_as_float(k.z), __uint_as_float(q.z), s);
    s = fmaf(__uint_as_float(k.w), __uint_as_float(q.w), s);
    return s;
  }
}

template <bool BF>
__device__ __forceinline__ void axpy16B(float* o, float p, const u32x4& v) {
  if constexpr (BF) {
    o[0] = fmaf(p, bf_lo(v.x), o[0]); o[1] = fmaf(p, bf_hi(v.x), o[1]);
    o[2] = fmaf(p, bf_lo(v.y), o[2]); o[3] = fmaf(p, bf_hi(v.y), o[3]);
    o[4] = fmaf(p, bf_lo(v.z), o[4]); o[5] = fmaf(p, bf_hi(v.z), o[5]);
    o[6] = fmaf(p, bf_lo(v.w), o[6]); o[7] = fmaf(p, bf_hi(v.w), o[7]);
  } else {
    o[0] = fmaf(p, __uint_as_float(v.x), o[0]); o[1] = fmaf(p, __uint_as_float(v.y), o[1]);
    o[2] = fmaf(p, __uint_as_float(v.z), o[2]); o[3] = fmaf(p, __uint_as_float(v.w), o[3]);
  }
}

// Compile-time shape of one kernel instantiation.
template <bool BF_, int D_, int HPK_, bool MFMA_, int PR_, bool KV8_ = false>
struct Shape {
  static constexpr bool BF = BF_;
  // KV8: the prefix store and the pages hold K/V as E4M3 bytes; the kernels
  // widen them to bf16 in registers (exact) and compute as for bf16.
  static constexpr bool KV8 = KV8_;
  static constexpr int D = D_;
  static constexpr int HPK = HPK_;
  static constexpr bool MFMA = MFMA_;
  static constexpr int PR = PR_;                  // prefix rows per record group (padded)
  static constexpr int ES = BF ? 2 : 4;            // element bytes
  static constexpr int EPL = 16 / ES;              // elements per lane chunk
  static constexpr int ROWB = D * ES;              // bytes of one K or V row of one head
  static constexpr int LPT = ROWB / 16;            // lanes per token (wavefront path)
  static constexpr int TPI = 64 / LPT;             // tokens per load instruction
  static constexpr int KES = KV8 ? 1 : ES;        // bytes per stored K/V element
  static constexpr int KROWB = D * KES;            // bytes of one stored K or V row of one head
  static constexpr int LANEB = EPL * KES;          // stored bytes behind one lane's EPL elements
  static constexpr int PAGEB = kPageTokens * KROWB; // bytes of one page of one head, K or V
  static constexpr int NB = PR / 16;               // MFMA row blocks
  static constexpr int KB = D / 32;                // MFMA k-blocks over head_dim
  static constexpr int DB = D / 16;                // MFMA 16-wide head_dim blocks
  // MFMA prefix work split over the four wavefronts: RG row groups of NBW
  // 16-row tiles times TG token groups of BPW 32-token blocks of the chunk
  // (16 rows: 1 x 4, 32 rows: 2 x 2, 64 rows: 4 x 1, 128 rows: 4 x 1 with two
  // tiles per wavefront).  Token groups of one row group combine through LDS.
  static constexpr int NBW = NB >= 8 ? 2 : 1;
  static constexpr int RG = MFMA ? NB / NBW : 1;
  static constexpr int TG = kWaves / RG;
  static constexpr int BPW = (kMfmaPrefixSplit / kMfmaBlock) / TG;
  static constexpr int WAVE_NR = (!MFMA && PR > HPK) ? PR : HPK;
  static constexpr int WAVE_SMEM = 4 * WAVE_NR * (D + 2);
  static constexpr int MFMA_SLOT = (MFMA && TG > 1) ? (NBW * DB * 64 * 4 + 2 * NBW * 64) : 0;
  static constexpr int MFMA_SMEM = kWaves * MFMA_SLOT;
  static constexpr int SMEM = WAVE_SMEM > MFMA_SMEM ? WAVE_SMEM : MFMA_SMEM;
  // 16 wavefront rows keep as many accumulators live as fill a SIMD's
  // registers at two wavefronts: that shape runs one per SIMD rather than
  // spill; every other shape runs (at least) two per SIMD.
  static constexpr int MIN_WAVES = (!MFMA && PR >= 16) ? 1 : 2;
  static_assert(LPT >= 2 && LPT <= 64, "row size");
  static_assert(!MFMA || BF, "MFMA path is bf16");
  static_assert(!KV8 || (BF && MFMA), "FP8 KV on the bf16 MFMA shapes");
  static_assert(!MFMA || (PR % 16 == 0), "MFMA rows");
  static_assert(!MFMA || (NB % NBW == 0 && kWaves % RG == 0 && DB % TG == 0 && BPW >= 1), "MFMA work split");
};

// ----------------------------------------------------------------------------
// Partial exchange between work-groups.  Producers store their partials, wait
// until the stores have completed and count an arrival; a merge reads them
// once its counters show every arrival.  Two cache policies:
//  * coherent: stores write through to the device coherence point and loads
//    bypass the XCD's L2 (the policy of agent-scope atomic stores and loads),
//    for producers and merges on any XCDs;
//  * XCD-local (StepArgs::l2_xcds > 0): stores stop in the XCD's L2 and loads
//    are served by the XCD's L2 or by the CU's L1.  The L1 is clean when a
//    launch starts, and a merge first reads a record line only after every
//    producer of that line has arrived, so the L1 never returns an older
//    copy within one launch that writes each record once.  Valid when every
//    work-group of a KV head runs on one XCD: work-group b on XCD
//    b % l2_xcds with Hkv a multiple of l2_xcds, which the host verified
//    when it created the context and which every work-group checks again (a
//    mismatch sets the status word).
// Neither needs an agent-scope fence (on this chip one writes back the whole
// L2).  Raw buffer resources over the workspace let a lane's 16 bytes leave
// as one write; offsets are in bytes and below ws_o_bytes / ws_ml_bytes.  The
// policy is a template parameter: the kernel picks one instantiation of its
// work-group body per launch, so no load or store waits behind a branch.
// ----------------------------------------------------------------------------
constexpr int kRawBufferWord3 = 0x00020000;
constexpr int kStoreThrough = 16;  // sc1
constexpr int kLoadCoherent = 16;  // sc1
constexpr int kStoreL2 = 0;
constexpr int kLoadL2 = 1;         // sc0: coherent at work-group scope: may hit the CU's L1 (clean at a launch's start), else the XCD's L2
constexpr int kXccIdReg = 20 | (3 << 11);  // s_getreg operand: HW_REG_XCC_ID bits 3:0

// MISS_L1: loads miss the CU's L1 also in the XCD-local exchange (sc0 loads
// are coherent only at work-group scope and may hit a line the L1 kept from
// an earlier read; a launch that rewrites and rereads the same records, as
// the step launch through every layer does, needs this).  Stores are the same
// either way.
template <bool L2, bool MISS_L1 = false>
struct Exchange {
  static constexpr int kStore = L2 ? kStoreL2 : kStoreThrough;
  static constexpr int kLoad = (L2 && !MISS_L1) ? kLoadL2 : kLoadCoherent;
  __amdgpu_buffer_rsrc_t o, ml;
  __device__ explicit Exchange(const StepArgs& a)
      : o(__builtin_amdgcn_make_buffer_rsrc(a.ws_o, 0, (int)a.ws_o_bytes, kRawBufferWord3)),
        ml(__builtin_amdgcn_make_buffer_rsrc(a.ws_ml, 0, (int)a.ws_ml_bytes, kRawBufferWord3)) {}
  __device__ void store(uint32_t off, float v) const {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), o, off, 0, kStore);
  }
  __device__ void store4(uint32_t off, f32x4 v) const {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), o, off, 0, kStore);
  }
  // (M, L) of record rec.
  __device__ void store_ml(int64_t rec, float m, float l) const {
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(m), __float_as_uint(l)}, ml, (uint32_t)(rec * 8), 0,
                                          kStore);
  }
  __device__ f32x4 load4(uint32_t off) const {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(o, off, 0, kLoad));
  }
  __device__ u32x2 load_ml(int64_t rec) const {
    return __builtin_amdgcn_raw_buffer_load_b64(ml, (uint32_t)(rec * 8), 0, kLoad);
  }
};

// E4M3 (OCP) <-> bf16.  Widening is exact: every E4M3 value is a bf16 value.
// Narrowing rounds to nearest even; magnitudes beyond 448 are clamped first,
// so the conversion saturates instead of producing NaN.
__device__ __forceinline__ u32x4 widen_e4m3(uint2 w) {
  u32x4 r;
  r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w.x, 1.0f, false));
  r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w.x, 1.0f, true));
  r.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w.y, 1.0f, false));
  r.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w.y, 1.0f, true));
  return r;
}
__device__ __forceinline__ float sat_e4m3(float x) { return fminf(fmaxf(x, -448.f), 448.f); }
__device__ __forceinline__ uint32_t narrow4_e4m3(uint32_t lo, uint32_t hi) {  // 4 bf16 -> 4 E4M3 bytes
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(sat_e4m3(__uint_as_float(lo << 16)), sat_e4m3(__uint_as_float(lo & 0xffff0000u)),
                                          0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(sat_e4m3(__uint_as_float(hi << 16)), sat_e4m3(__uint_as_float(hi & 0xffff0000u)),
                                      w, true);
  return (uint32_t)w;
}
__device__ __forceinline__ uint2 narrow_e4m3(const u32x4& v) {  // 8 bf16 -> 8 E4M3 bytes
  return uint2{narrow4_e4m3(v.x, v.y), narrow4_e4m3(v.z, v.w)};
}
// One lane's EPL stored elements as a 16-byte register of the compute type.
// Load one lane's EPL stored elements, widened to the compute type.  Every
// K/V byte is read once per launch.  Response K/V (NT) is loaded
// non-temporal, so its stream through the XCD's L2 does not push out the
// split-K partials that the merges read back from there; the shared prefix,
// a fifth of the bytes and read again by every step, keeps the default policy
// (measured slightly faster than non-temporal).
template <class SH, bool NT>
__device__ __forceinline__ u32x4 ld_kv(const char* p) {
  if constexpr (SH::KV8) {
    u32x2 w;
    if constexpr (NT)
      w = __builtin_nontemporal_load((const u32x2*)p);
    else
      w = *(const u32x2*)p;
    return widen_e4m3(uint2{w.x, w.y});
  } else if constexpr (NT) {
    return __builtin_nontemporal_load((const u32x4*)p);
  } else {
    return *(const u32x4*)p;
  }
}
// Store one lane's EPL elements (given in the compute type) into a stored row.
template <class SH>
__device__ __forceinline__ void st_kv(char* p, const u32x4& v) {
  if constexpr (SH::KV8)
    *(uint2*)p = narrow_e4m3(v);
  else
    *(u32x4*)p = v;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) x = fmaxf(x, __shfl_xor(x, s));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) x += __shfl_xor(x, s);
  return x;
}

// ----------------------------------------------------------------------------
// Wavefront path: NR query rows over the token range [t0, t1) of one KV head.
// LPT consecutive lanes hold one token's row (16 B each), so a load
// instruction covers TPI tokens; U loads per lane for K and for V are issued
// together before any arithmetic.  Each token group keeps its own running
// (m, l, o); the groups are combined at the end.  t0 must be a multiple of 16
// (page-aligned) so that every load instruction stays inside one page.
// ----------------------------------------------------------------------------
template <class SH, int NR>
struct WaveCfg {
  // Loads per lane per iteration, sized so that K/V buffers, scores and
  // accumulators of NR rows stay within the two-wavefronts-per-SIMD budget.
  static constexpr int UMAX = NR <= 2 ? 16 : NR <= 4 ? 8 : 4;
  static constexpr int U = (64 / SH::TPI) < UMAX ? (64 / SH::TPI) : UMAX;
  static_assert(16 % SH::TPI == 0, "a load instruction must not straddle a page");
};

template <class SH, int NR, class Addr>
__device__ __forceinline__ void wave_partial(const Addr& ad, int t0, int t1, const u32x4 (&q)[NR], float sl2,
                                             float (&m)[NR], float (&l)[NR], float (&o)[NR][SH::EPL]) {
  constexpr int LPT = SH::LPT, TPI = SH::TPI, EPL = SH::EPL, U = WaveCfg<SH, NR>::U;
  // Loads are issued in sub-blocks of SB per lane (K, then V) and the online
  // softmax runs per sub-block, so the arithmetic on early sub-blocks overlaps
  // the arrival of later ones.  Every load is unconditional: tokens past t1
  // read a valid row (Addr keeps addresses in bounds) and are masked to -inf.
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
  constexpr int PGI = (U * TPI + 15) / 16;  // 16-token pages touched per iteration
  for (int base = t0; base < t1; base += U * TPI) {
    // Page numbers first, in straight-line code: the compiler then waits for
    // the page-table load once instead of before every K/V load.
    int pg[PGI];
#pragma unroll
    for (int i = 0; i < PGI; ++i) pg[i] = ad.page(((base - t0) >> 4) + i);
    u32x4 kk[U], vv[U];
#pragma unroll
    for (int b = 0; b < NSB; ++b) {
#pragma unroll
      for (int kind = 0; kind < 2; ++kind)
#pragma unroll
        for (int u = b * SB; u < b * SB + SB; ++u) {
          u32x4& dst = kind ? vv[u] : kk[u];
          dst = ld_kv<SH, Addr::kNonTemporal>(ad.row(kind, base + u * TPI, base - t0 + u * TPI, pg[(u * TPI) >> 4], t1));
        }
    }
#pragma unroll
    for (int b = 0; b < NSB; ++b) {
      float s[SB][NR];
#pragma unroll
      for (int x = 0; x < SB; ++x) {
        const int u = b * SB + x;
        const bool ok = base + u * TPI + ts < t1;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          const float y = group_sum<LPT>(dot16B<SH::BF>(kk[u], q[r])) * sl2;
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
          // P.V two tokens at a time with bf16 dot products: the probabilities
          // are rounded to bf16 and the normaliser sums the same rounded values.
#pragma unroll
          for (int x = 0; x < SB; x += 2) {
            const int u = b * SB + x;
            const __bf16 h0 = (__bf16)exp2_fast(s[x][r] - mu), h1 = (__bf16)exp2_fast(s[x + 1][r] - mu);
            l[r] += (float)h0 + (float)h1;
            const bf16x2 pb = {h0, h1};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const uint32_t lo = __builtin_amdgcn_perm(vv[u + 1][k], vv[u][k], 0x05040100u);  // elems 2k
              const uint32_t hi = __builtin_amdgcn_perm(vv[u + 1][k], vv[u][k], 0x07060302u);  // elems 2k+1
              o[r][2 * k] = __builtin_amdgcn_fdot2_f32_bf16(pb, __builtin_bit_cast(bf16x2, lo), o[r][2 * k], false);
              o[r][2 * k + 1] = __builtin_amdgcn_fdot2_f32_bf16(pb, __builtin_bit_cast(bf16x2, hi), o[r][2 * k + 1], false);
            }
          }
        } else {
#pragma unroll
          for (int x = 0; x < SB; ++x) {
            const float p = exp2_fast(s[x][r] - mu);
            l[r] += p;
            axpy16B<false>(o[r], p, vv[b * SB + x]);
          }
        }
      }
    }
  }
}

// Fold one token (K row chunk k, V row chunk v held by every token group) into
// token group 0's running partial.  All lanes take part in the reduction.
template <class SH, int NR>
__device__ __forceinline__ void fold_token(const u32x4& k, const u32x4& v, const u32x4 (&q)[NR], float sl2,
                                           float (&m)[NR], float (&l)[NR], float (&o)[NR][SH::EPL]) {
  const bool mine = (threadIdx.x & 63) < SH::LPT;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const float x = group_sum<SH::LPT>(dot16B<SH::BF>(k, q[r])) * sl2;
    if (mine) {
      const float mn = fmaxf(m[r], x);
      const float corr = exp2_fast(m[r] - mn);
      const float p = exp2_fast(x - mn);
      m[r] = mn;
      l[r] = l[r] * corr + p;
#pragma unroll
      for (int e = 0; e < SH::EPL; ++e) o[r][e] *= corr;
      axpy16B<SH::BF>(o[r], p, v);
    }
  }
}

// Combine the TPI token groups of a wavefront (lanes ch, ch+LPT, ...).
template <class SH, int NR>
__device__ __forceinline__ void wave_combine_groups(float (&m)[NR], float (&l)[NR], float (&o)[NR][SH::EPL]) {
#pragma unroll
  for (int mask = SH::LPT; mask < 64; mask <<= 1) {
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const float m2 = __shfl_xor(m[r], mask);
      const float l2 = __shfl_xor(l[r], mask);
      float a, b;
      lse_combine(m[r], l[r], m2, l2, a, b);
#pragma unroll
      for (int e = 0; e < SH::EPL; ++e) o[r][e] = o[r][e] * a + __shfl_xor(o[r][e], mask) * b;
    }
  }
}

template <class SH, int NR, bool L2>
__device__ __forceinline__ void combine_store_partial(float* smem, const Exchange<L2>& ex, int64_t rec0);

// Combine the four wavefronts' partials through LDS and store the block's
// partial rows [0, NR) at records rec0 + r.
template <class SH, int NR, bool L2>
__device__ __forceinline__ void block_store_partial(float* smem, const float (&m)[NR], const float (&l)[NR],
                                                    const float (&o)[NR][SH::EPL], const Exchange<L2>& ex,
                                                    int64_t rec0) {
  constexpr int D = SH::D, EPL = SH::EPL;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float* so = smem;                   // [4][NR][D]
  float* sml = smem + 4 * NR * D;     // [4][NR][2]
  if (lane < SH::LPT) {
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
      for (int e = 0; e < EPL; ++e) so[(w * NR + r) * D + lane * EPL + e] = o[r][e];
  }
  if (lane == 0) {
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      sml[(w * NR + r) * 2 + 0] = m[r];
      sml[(w * NR + r) * 2 + 1] = l[r];
    }
  }
  combine_store_partial<SH, NR, L2>(smem, ex, rec0);
}

// Second half of block_store_partial: after every wavefront has published its
// partial rows to LDS (so = [4][NR][D] unnormalised outputs, then
// sml = [4][NR][2] (m, l)), combine them and store rows [0, NR) at records
// rec0 + r.
template <class SH, int NR, bool L2>
__device__ __forceinline__ void combine_store_partial(float* smem, const Exchange<L2>& ex, int64_t rec0) {
  constexpr int D = SH::D;
  const float* so = smem;
  const float* sml = smem + 4 * NR * D;
  __syncthreads();
  for (int idx = threadIdx.x; idx < NR * D; idx += kBlockThreads) {
    const int r = idx / D, d = idx - r * D;
    float M = NEG_INF;
#pragma unroll
    for (int v = 0; v < 4; ++v) M = fmaxf(M, sml[(v * NR + r) * 2]);
    const float Mu = (M == NEG_INF) ? 0.f : M;
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float wgt = exp2_fast(sml[(v * NR + r) * 2] - Mu);
      L += wgt * sml[(v * NR + r) * 2 + 1];
      O += wgt * so[(v * NR + r) * D + d];
    }
    ex.store((uint32_t)(((rec0 + r) * D + d) * 4), O);
    if (d == 0) ex.store_ml(rec0 + r, M, L);
  }
}

// Addressing of the plain prefix store: [prompt][kv][K|V][max_prompt_len][D].
// Row of token tokbase + (lane / LPT), clamped below `end` so that masked
// tokens still read inside this head's region.
template <class SH>
struct PrefixAddr {
  static constexpr bool kNonTemporal = false;
  const char* base[2];
  __device__ int page(int) const { return 0; }
  __device__ const char* row(int kind, int tokbase, int, int, int end) const {
    const int lane = threadIdx.x & 63;
    const int tok = min(tokbase + lane / SH::LPT, end - 1);
    return base[kind] + (int64_t)tok * SH::KROWB + (lane % SH::LPT) * SH::LANEB;
  }
};

// Addressing of a slot's stored response tokens: pages [page][kv][K|V][16][D].
// Lane i of `pages` holds the page of the wave's i-th 16-token group.  A load
// instruction covers TPI consecutive tokens of one page, so its address is
// (page base) + (token in page) * KROWB + lane * LANEB -- uniform plus lane offset.
template <class SH>
struct SuffixAddr {
  static constexpr bool kNonTemporal = true;
  const char* pool;
  int pages;
  int hkv, g;
  __device__ int page(int pslot) const { return __builtin_amdgcn_readlane(pages, pslot); }
  __device__ const char* row(int kind, int tokbase, int, int pg, int) const {
    const int lane = threadIdx.x & 63;
    return pool + ((int64_t)(pg * hkv + g) * 2 + kind) * SH::PAGEB + (tokbase & 15) * SH::KROWB + lane * SH::LANEB;
  }
};

// ----------------------------------------------------------------------------
// Response chunk on MFMA tiles (bf16 and E4M3 pages).  A page holds 16 tokens
// of one KV head, K then V, each in MFMA operand order:
//   K unit (kb, lane), 8 elements: token lane%16, dims 32kb + 8(lane/16) + e;
//   V unit (db, lane), 4 elements: dim 16db + lane%16, tokens 4(lane/16) + e;
// so a wavefront reads one operand tile with one coalesced load per lane
// (16 / 8 bytes for bf16).  Per page, S^T[tok][col] = K[tok] . Q[col] is one
// 16x16 tile (A = K units, B = Q^T, col = query row of the KV head: HPK of
// the 16 columns carry rows, the rest are zero).  Two consecutive pages form
// one 32-token k-block of O^T[d][col] += V^T[d][tok] P^T[tok][col]: the P^T
// operand is the eight probabilities a lane holds after the pages' two S^T
// tiles (the first page's four, then the second's) and the V^T operand is the
// two pages' V units side by side, so the contraction index is the same
// token permutation on both operands.  The running (m, l) and O^T are indexed
// by col = lane % 16 as on the prefix tiles; l is a per-lane sum until
// publish() adds the four lane groups.
// ----------------------------------------------------------------------------
template <class SH>
struct RespMfma {
  static constexpr int D = SH::D, KB = SH::KB, DB = SH::DB, HPK = SH::HPK, KES = SH::KES;
  static constexpr int NPG = D >= 128 ? 4 : 8;        // pages per load round
  static constexpr int TOK = 16 * NPG;                // tokens per load round
  static constexpr int KUB = 8 * KES, VUB = 4 * KES;  // bytes of one K / V unit
  using KUnit = std::conditional_t<SH::KV8, u32x2, u32x4>;
  using VUnit = std::conditional_t<SH::KV8, uint32_t, u32x2>;
  using VPair = std::conditional_t<SH::KV8, u32x2, u32x4>;  // two pages' V units, side by side
  struct Regs {
    KUnit k[NPG][KB];
    VPair v[NPG / 2][DB];
  };
  static constexpr int kLoads = NPG * (KB + DB);  // load instructions of one round
  // Running partial: O^T tiles, m per column and, in lt, the column's sum of
  // probabilities (every element; an all-ones V^T tile through the same MFMA).
  struct Acc {
    f32x4 o[DB];
    f32x4 lt;
    float m;
  };
  // The newest token's rows, loaded with the queries: kq[kb] = K dims
  // 32kb + 8(lane/16) .. +7 and vq[db] = V dims 16db + 4(lane/16) .. +3.
  struct NewRows {
    u32x4 kq[KB];
    u32x2 vq[DB];
  };
  static_assert(HPK <= 16 && KB * 32 == D && DB * 16 == D, "response tile shape");

  __device__ __forceinline__ static int k_unit(int kb, int lane) { return (kb * 64 + lane) * KUB; }
  __device__ __forceinline__ static int v_unit(int db, int lane) { return (db * 64 + lane) * VUB; }
  // Page pg of KV head g: K at the returned address, V PAGEB bytes later.
  __device__ __forceinline__ static const char* page(const char* pool, int pg, int hkv, int g) {
    return pool + (int64_t)(pg * hkv + g) * 2 * SH::PAGEB;
  }

  // Loads of the round whose first page is entry ps of the wavefront's page
  // list (lane i of `pages`: its i-th page; entries past the range name page
  // 0, so every load stays inside the pool).  K of every page, then V, each
  // pair's V units straight into one MFMA operand register.
  __device__ __forceinline__ static void load_round(const char* pool, int pages, int hkv, int g, int ps, Regs& R) {
    const int lane = threadIdx.x & 63;
    const char* pp[NPG];
#pragma unroll
    for (int pr = 0; pr < NPG; ++pr) pp[pr] = page(pool, __builtin_amdgcn_readlane(pages, min(ps + pr, 63)), hkv, g);
#pragma unroll
    for (int pr = 0; pr < NPG; ++pr)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) R.k[pr][kb] = __builtin_nontemporal_load((const KUnit*)(pp[pr] + k_unit(kb, lane)));
#pragma unroll
    for (int j = 0; j < NPG / 2; ++j)
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const VUnit a0 = __builtin_nontemporal_load((const VUnit*)(pp[2 * j] + SH::PAGEB + v_unit(db, lane)));
        const VUnit a1 = __builtin_nontemporal_load((const VUnit*)(pp[2 * j + 1] + SH::PAGEB + v_unit(db, lane)));
        if constexpr (SH::KV8)
          R.v[j][db] = u32x2{a0, a1};
        else
          R.v[j][db] = __builtin_shufflevector(a0, a1, 0, 1, 2, 3);
      }
  }

  __device__ __forceinline__ static bf16x8 k_op(const KUnit& u) {
    if constexpr (SH::KV8)
      return __builtin_bit_cast(bf16x8, widen_e4m3(uint2{u.x, u.y}));
    else
      return __builtin_bit_cast(bf16x8, u);
  }
  __device__ __forceinline__ static u32x4 v_op(const VPair& u) {  // eight elements as bf16
    if constexpr (SH::KV8)
      return widen_e4m3(uint2{u.x, u.y});
    else
      return u;
  }
  // Bits of elements 2k and 2k + 1 of a four-element V unit that belong to
  // the first n tokens.
  __device__ __forceinline__ static uint32_t keep(int n, int k) {
    return (n > 2 * k ? 0x0000ffffu : 0u) | (n > 2 * k + 1 ? 0xffff0000u : 0u);
  }

  // Q^T operand: lane l holds query row row0 + l%16 (zero from HPK on), dims
  // 32kb + 8(l/16) .. +7.
  __device__ __forceinline__ static void load_q(const void* q, int64_t row0, bf16x8 (&bq)[KB]) {
    const int lane = threadIdx.x & 63, col = lane & 15, h = lane >> 4;
    const uint16_t* qr = (const uint16_t*)q + (row0 + col) * D + h * 8;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) bq[kb] = col < HPK ? *(const bf16x8*)(qr + kb * 32) : bf16x8{};
  }
  // The newest token's K / V rows (bf16, the caller's row layout), rounded to
  // E4M3 and back for E4M3 pages: the token is attended as its page stores it.
  __device__ __forceinline__ static void load_new(const char* krow, const char* vrow, NewRows& N) {
    const int h = (threadIdx.x & 63) >> 4;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) N.kq[kb] = *(const u32x4*)(krow + (kb * 32 + h * 8) * 2);
#pragma unroll
    for (int db = 0; db < DB; ++db) N.vq[db] = *(const u32x2*)(vrow + (db * 16 + h * 4) * 2);
  }
  __device__ __forceinline__ static void round_new(NewRows& N) {
    if constexpr (SH::KV8) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) N.kq[kb] = widen_e4m3(narrow_e4m3(N.kq[kb]));
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int b = (int)narrow4_e4m3(N.vq[db].x, N.vq[db].y);
        N.vq[db] = u32x2{__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(b, 1.0f, false)),
                         __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(b, 1.0f, true))};
      }
    }
  }

  // A partial that holds only the newest token (A's first contribution).
  __device__ __forceinline__ static void start_new(const NewRows& N, const bf16x8 (&bq)[KB], float sl2, Acc& A) {
    float s = 0.f;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) s += dot16B<true>(N.kq[kb], __builtin_bit_cast(u32x4, bq[kb]));
    s += __shfl_xor(s, 16);
    s += __shfl_xor(s, 32);
    // the token's own weight is 2^(x - m) = 1 with m = x
    A.m = s * sl2;
    A.lt = f32x4{1.f, 1.f, 1.f, 1.f};
#pragma unroll
    for (int db = 0; db < DB; ++db) A.o[db] = f32x4{bf_lo(N.vq[db].x), bf_hi(N.vq[db].x), bf_lo(N.vq[db].y), bf_hi(N.vq[db].y)};
  }

  __device__ __forceinline__ static void init(Acc& A) {
    A.m = NEG_INF;
    A.lt = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int db = 0; db < DB; ++db) A.o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Tokens base .. base + TOK - 1 (the round held in R), of which those below
  // t1 count: one online-softmax step per page pair (32 tokens).
  __device__ __forceinline__ static void round(const Regs& R, const bf16x8 (&bq)[KB], int base, int t1, float sl2,
                                               Acc& A) {
    const int lane = threadIdx.x & 63, h = lane >> 4;
    const bf16x8 ones = __builtin_bit_cast(bf16x8, u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});
#pragma unroll
    for (int j = 0; j < NPG / 2; ++j) {
      const int pb0 = base + 32 * j;
      if (pb0 >= t1) break;
      // a pair that reaches past t1 masks its tail (scores and V elements)
      const bool edge = pb0 + 32 > t1;
      f32x4 st[2];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
          t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k_op(R.k[2 * j + mb][kb]), bq[kb], t, 0, 0, 0);
        t *= sl2;
        if (edge) {
#pragma unroll
          for (int e = 0; e < 4; ++e) t[e] = (pb0 + 16 * mb + 4 * h + e < t1) ? t[e] : NEG_INF;
        }
        st[mb] = t;
      }
      float mx = fmaxf(fmaxf(fmaxf(st[0][0], st[0][1]), fmaxf(st[0][2], st[0][3])),
                       fmaxf(fmaxf(st[1][0], st[1][1]), fmaxf(st[1][2], st[1][3])));
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mn = fmaxf(A.m, mx);
      const float mu = (mn == NEG_INF) ? 0.f : mn;
      const float corr = exp2_fast(A.m - mu);
      A.m = mn;
      A.lt *= corr;
#pragma unroll
      for (int db = 0; db < DB; ++db) A.o[db] *= corr;
      bf16x8 pb;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pb[e] = (__bf16)exp2_fast(st[0][e] - mu);
        pb[4 + e] = (__bf16)exp2_fast(st[1][e] - mu);
      }
      A.lt = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb, A.lt, 0, 0, 0);
      // V elements of tokens at or past t1 (a page's unused tail holds whatever
      // was there) are cleared so that their zero weights give exact zeros.
      const int n0 = min(max(t1 - (pb0 + 4 * h), 0), 4), n1 = min(max(t1 - (pb0 + 16 + 4 * h), 0), 4);
      const u32x4 vm = {keep(n0, 0), keep(n0, 1), keep(n1, 0), keep(n1, 1)};
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        u32x4 va = v_op(R.v[j][db]);
        if (edge) va &= vm;
        A.o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, va), pb, A.o[db], 0, 0, 0);
      }
    }
  }

  // Store the newest token (position t, 0..15, of the page at pgk) in operand
  // order from the rows in N: K unit (kb, 16h + t) from the lanes with
  // lane % 16 == 0 (lane group h), V element (dim 16db + 4h + i, token t) from
  // lane 16h + i, i < 4.
  __device__ __forceinline__ static void store_new(char* pgk, int t, const NewRows& N) {
    const int lane = threadIdx.x & 63, h = lane >> 4, i = lane & 15;
    if (i == 0) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) st_kv<SH>(pgk + k_unit(kb, h * 16 + t), N.kq[kb]);
    }
    if (i < 4) {
      char* vb = pgk + SH::PAGEB + (t & 3) * KES;
      const int l0 = 16 * (t >> 2) + 4 * h + i;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const uint32_t w = (i & 2) ? N.vq[db].y : N.vq[db].x;
        const uint32_t bits = (i & 1) ? (w >> 16) : (w & 0xffffu);
        if constexpr (SH::KV8) {
          // N.vq holds E4M3 values widened to bf16: narrowing again is exact
          const uint32_t b = narrow4_e4m3(bits, 0u) & 0xffu;
          *(uint8_t*)(vb + v_unit(db, l0)) = (uint8_t)b;
        } else {
          *(uint16_t*)(vb + v_unit(db, l0)) = (uint16_t)bits;
        }
      }
    }
  }

  // Publish the wavefront's partial rows to LDS in block_store_partial's
  // layout (finish with combine_store_partial<SH, HPK, L2>).
  __device__ __forceinline__ static void publish(float* smem, const Acc& A) {
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, col = lane & 15, h = lane >> 4;
    float* so = smem;
    float* sml = smem + 4 * HPK * D;
    if (col < HPK) {
#pragma unroll
      for (int db = 0; db < DB; ++db) *(f32x4*)(so + (w * HPK + col) * D + db * 16 + h * 4) = A.o[db];
      if (h == 0) {
        sml[(w * HPK + col) * 2 + 0] = A.m;
        sml[(w * HPK + col) * 2 + 1] = A.lt[0];
      }
    }
  }
};

__device__ __forceinline__ int64_t prefix_records(const StepArgs& a, int pr) {
  return (int64_t)a.num_prompts * a.prefix_chunks_max * a.Hkv * pr;
}

// ----------------------------------------------------------------------------
// Prefix chunk, wavefront path (fewer than 16 rows): rows r = slot_in_prompt * hpk + j.
// ----------------------------------------------------------------------------
template <class SH, bool L2>
__device__ void prefix_wave(const StepArgs& a, int p, int c, int g, float* smem) {
  constexpr int PR = SH::PR, HPK = SH::HPK;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, ch = lane % SH::LPT;
  const int plen = a.prompt[p].plen;
  const int t0 = c * a.prefix_split, t1 = min(t0 + a.prefix_split, plen);
  const int sub = a.prefix_split / 4;
  const int wt0 = min(t0 + w * sub, t1), wt1 = min(wt0 + sub, t1);
  u32x4 q[PR];
#pragma unroll
  for (int r = 0; r < PR; ++r) {
    const int si = r / HPK, j = r - si * HPK, s = p * a.m + min(si, a.m - 1);
    if (r < a.prefix_rows && a.slot[s].len > 0)
      q[r] = *((const u32x4*)((const char*)a.q + ((int64_t)s * a.Hq + g * HPK + j) * SH::ROWB) + ch);
    else
      q[r] = u32x4{0, 0, 0, 0};
  }
  const int64_t head = ((int64_t)p * a.Hkv + g) * 2;
  PrefixAddr<SH> ad{{(const char*)a.prefix + head * a.max_prompt_len * SH::KROWB,
                     (const char*)a.prefix + (head + 1) * a.max_prompt_len * SH::KROWB}};
  float m[PR], l[PR], o[PR][SH::EPL];
  wave_partial<SH, PR>(ad, wt0, wt1, q, a.scale_log2, m, l, o);
  wave_combine_groups<SH, PR>(m, l, o);
  const int64_t rec0 = (((int64_t)p * a.Hkv + g) * a.prefix_chunks_max + c) * PR;
  block_store_partial<SH, PR, L2>(smem, m, l, o, Exchange<L2>(a), rec0);
}

// ----------------------------------------------------------------------------
// Prefix chunk, MFMA path (R = NB*16 rows).  Per 32-token block:
//   S^T[tok][row] = K[tok][:] . Q[row][:]     (A = K block, B = Q^T; 2 x NB tiles of 16x16)
//   O^T[d][row]  += V^T[d][tok] P^T[tok][row] (A = V^T, B = P^T; NB x DB tiles)
// With S^T, O^T and the running (m, l) all indexed by row = lane % 16, the
// online-softmax rescale needs no cross-lane transpose.  The P^T operand takes
// the 8 probabilities a lane already holds; the contraction index (token) is
// the same permutation on both operands, and the prefix store keeps V in that
// order (see prefill_mfma_kernel).  Each wavefront keeps one block in flight
// (the accumulators of 32+ rows leave no registers for a second).
// ----------------------------------------------------------------------------
template <class SH>
__device__ __forceinline__ void mfma_block(const bf16x8 (&ka)[2][SH::KB], const bf16x8 (&va)[SH::DB],
                                           const bf16x8 (&bq)[SH::NB][SH::KB], int tb, int t1, float sl2,
                                           f32x4 (&acc)[SH::NB][SH::DB], float (&mrow)[SH::NB],
                                           float (&lrow)[SH::NB]) {
  constexpr int NB = SH::NB, KB = SH::KB, DB = SH::DB;
  const int lane = threadIdx.x & 63, q4 = lane >> 4;
  f32x4 st[2][NB];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[mb][kb], bq[nb][kb], t, 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int tok = tb + mb * 16 + q4 * 4 + e;
        t[e] = (tok < t1) ? t[e] * sl2 : NEG_INF;
      }
      st[mb][nb] = t;
    }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float mb_ = fmaxf(fmaxf(fmaxf(st[0][nb][0], st[0][nb][1]), fmaxf(st[0][nb][2], st[0][nb][3])),
                      fmaxf(fmaxf(st[1][nb][0], st[1][nb][1]), fmaxf(st[1][nb][2], st[1][nb][3])));
    mb_ = fmaxf(mb_, __shfl_xor(mb_, 16));
    mb_ = fmaxf(mb_, __shfl_xor(mb_, 32));
    const float mn = fmaxf(mrow[nb], mb_);
    const float mu = (mn == NEG_INF) ? 0.f : mn;
    const float corr = exp2_fast(mrow[nb] - mu);
    mrow[nb] = mn;
    lrow[nb] *= corr;
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[nb][db] *= corr;
    bf16x8 pb;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const __bf16 h = (__bf16)exp2_fast(st[mb][nb][e] - mu);
        pb[mb * 4 + e] = h;
        lrow[nb] += (float)h;
      }
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[nb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[db], pb, acc[nb][db], 0, 0, 0);
  }
}

// ----------------------------------------------------------------------------
// Prefix chunk on MFMA tiles.  Wavefront w takes row group rg = w % RG (its
// NBW 16-row tiles) and token group tg = w / RG (BPW consecutive 32-token
// blocks of the chunk), walking its blocks with the next block's loads in
// flight while the current one is multiplied (with two tiles per wavefront,
// only the next K).  With one token group the
// wavefront stores its rows' partial directly; otherwise the token groups of
// a row group publish their partials to LDS and, after one barrier, each
// combines DB / TG of the head-dimension blocks of its row group and stores
// them.
// ----------------------------------------------------------------------------
template <class SH, bool L2>
__device__ void prefix_mfma(const StepArgs& a, int p, int c, int g, float* smem) {
  constexpr int D = SH::D, KB = SH::KB, DB = SH::DB, HPK = SH::HPK;
  constexpr int NBW = SH::NBW, RG = SH::RG, TG = SH::TG, BPW = SH::BPW;
  using WS = Shape<true, D, HPK, true, NBW * 16>;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, q4 = lane >> 4, r16 = lane & 15;
  const int rg = w % RG, tg = w / RG;
  const int plen = a.prompt[p].plen;
  const int t0 = c * a.prefix_split, t1 = min(t0 + a.prefix_split, plen);
  const int nblk = (t1 - t0 + kMfmaBlock - 1) / kMfmaBlock;
  const int b0 = tg * BPW, b1 = min(b0 + BPW, nblk);
  const float sl2 = a.scale_log2;

  bf16x8 bq[NBW][KB];
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb) {
    const int row = (rg * NBW + nb) * 16 + r16, si = row / HPK, j = row - si * HPK, s = p * a.m + min(si, a.m - 1);
    const bool ok = row < a.prefix_rows && a.slot[s].len > 0;
    const uint16_t* qr = (const uint16_t*)a.q + ((int64_t)s * a.Hq + g * HPK + j) * D;
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
  const char* head = (const char*)a.prefix +
                     ((int64_t)(p * a.Hkv + g) * (a.max_prompt_len / kMfmaBlock)) * (2 * kMfmaBlock * D * SH::KES);
  auto fetch_k = [&](int b, bf16x8 (&ka)[2][KB]) {
    const char* kblk = head + (int64_t)((t0 + b * kMfmaBlock) / kMfmaBlock) * (2 * kMfmaBlock * D * SH::KES);
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        ka[mb][kb] = __builtin_bit_cast(bf16x8, ld_kv<SH, false>(kblk + ((mb * KB + kb) * 64 + lane) * 8 * SH::KES));
  };
  auto fetch_v = [&](int b, bf16x8 (&va)[DB]) {
    const char* vblk = head + (int64_t)((t0 + b * kMfmaBlock) / kMfmaBlock) * (2 * kMfmaBlock * D * SH::KES) +
                       kMfmaBlock * D * SH::KES;
#pragma unroll
    for (int db = 0; db < DB; ++db) va[db] = __builtin_bit_cast(bf16x8, ld_kv<SH, false>(vblk + (db * 64 + lane) * 8 * SH::KES));
  };
  // With two tiles per wavefront the accumulators leave room to prefetch only
  // the next block's K; its V is fetched once the current block is done.
  constexpr bool PREFETCH_V = NBW == 1;
  if (b0 < b1) {
    bf16x8 ka[2][KB], va[DB];
    fetch_k(b0, ka);
    fetch_v(b0, va);
    for (int b = b0; b < b1; ++b) {
      const bool more = b + 1 < b1;
      bf16x8 kn[2][KB], vn[DB];
      if (more) {
        fetch_k(b + 1, kn);
        if constexpr (PREFETCH_V) fetch_v(b + 1, vn);
      }
      mfma_block<WS>(ka, va, bq, t0 + b * kMfmaBlock, t1, sl2, acc, mrow, lrow);
      if (more) {
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) ka[mb][kb] = kn[mb][kb];
        if constexpr (PREFETCH_V) {
#pragma unroll
          for (int db = 0; db < DB; ++db) va[db] = vn[db];
        } else {
          fetch_v(b + 1, va);
        }
      }
    }
  }
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb) {
    lrow[nb] += __shfl_xor(lrow[nb], 16);
    lrow[nb] += __shfl_xor(lrow[nb], 32);
  }
  const int64_t rec0 = (((int64_t)p * a.Hkv + g) * a.prefix_chunks_max + c) * SH::PR;
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
    constexpr int DBW = DB / TG;  // head-dim blocks this wavefront combines and stores
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
}

// ----------------------------------------------------------------------------
// Response chunk of one live slot (hpk rows), plus the append of this step's
// K/V when the chunk holds the newest position.
// ----------------------------------------------------------------------------
template <class SH, bool L2>
__device__ void suffix_chunk_mfma(const StepArgs& a, int s, int c, int g, float* smem);

template <class SH, bool L2>
__device__ void suffix_chunk(const StepArgs& a, int s, int c, int g, float* smem) {
  if constexpr (SH::BF) {
    suffix_chunk_mfma<SH, L2>(a, s, c, g, smem);
    return;
  }
  constexpr int HPK = SH::HPK;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, ch = lane % SH::LPT;
  const SlotPlan& sp = a.slot[s];
  const int len = sp.len;
  const int t0 = c * a.split, t1 = min(t0 + a.split, len);
  const int sub = a.split / 4;
  const int wt0 = min(t0 + w * sub, t1), wt1 = min(wt0 + sub, t1);
  // Page indices of this wavefront's range (lane i: the i-th 16-token group) and
  // the query rows, loaded together.
  const int npg = (wt1 - wt0 + kPageTokens - 1) / kPageTokens;
  const int32_t* ptab = a.page_table + (int64_t)sp.seq * a.pages_per_slot + (wt0 >> 4);
  const int pages = lane < npg ? ptab[lane] : 0;
  u32x4 q[HPK];
#pragma unroll
  for (int r = 0; r < HPK; ++r)
    q[r] = *((const u32x4*)((const char*)a.q + ((int64_t)s * a.Hq + g * HPK + r) * SH::ROWB) + ch);
  // The newest token (position len-1) comes from the caller's rows: the wave
  // whose range holds it loads it up front, folds it in after the stored
  // tokens, and stores it into its page.
  const int last = len - 1;
  const bool has_new = last >= wt0 && last < wt1;
  const int64_t newrow = ((int64_t)s * a.Hkv + g) * SH::ROWB;
  u32x4 knew = u32x4{0, 0, 0, 0}, vnew = u32x4{0, 0, 0, 0};
  if (has_new) {
    knew = *((const u32x4*)((const char*)a.knew + newrow) + ch);
    vnew = *((const u32x4*)((const char*)a.vnew + newrow) + ch);
    if constexpr (SH::KV8) {  // attend to the token as the cache stores it
      knew = widen_e4m3(narrow_e4m3(knew));
      vnew = widen_e4m3(narrow_e4m3(vnew));
    }
  }
  SuffixAddr<SH> ad{(const char*)a.pool, pages, a.Hkv, g};
  float m[HPK], l[HPK], o[HPK][SH::EPL];
  wave_partial<SH, HPK>(ad, wt0, has_new ? last : wt1, q, a.scale_log2, m, l, o);
  if (has_new) {
    fold_token<SH, HPK>(knew, vnew, q, a.scale_log2, m, l, o);
    if (lane < SH::LPT) {
      char* row = (char*)a.pool + (int64_t)(sp.cur_page * a.Hkv + g) * 2 * SH::PAGEB + (last & 15) * SH::KROWB +
                  ch * SH::LANEB;
      st_kv<SH>(row, knew);
      st_kv<SH>(row + SH::PAGEB, vnew);
    }
  }
  wave_combine_groups<SH, HPK>(m, l, o);
  const int64_t rec0 = prefix_records(a, SH::PR) + (((int64_t)s * a.Hkv + g) * a.suffix_chunks_max + c) * HPK;
  block_store_partial<SH, HPK, L2>(smem, m, l, o, Exchange<L2>(a), rec0);

  if (t1 == len && g == 0 && threadIdx.x == 0) {  // bookkeeping of this step's token (K/V stored above)
    const int pos = len - 1;
    a.page_table[(int64_t)sp.seq * a.pages_per_slot + (pos >> 4)] = sp.cur_page;
    if (a.count_tokens)
      __hip_atomic_fetch_add(&a.tokens[(s / a.m) * a.G + sp.sample], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Response chunk of one live slot on MFMA tiles (bf16 and E4M3 pages; see
// RespMfma): wavefront w takes tokens [wt0, wt1) of the chunk in rounds of
// RespMfma::TOK; the wavefront whose range holds the newest position starts
// from that token (read from the caller's rows together with the queries) and
// stores it into its page; the four wavefronts' partials combine through LDS.
template <class SH, bool L2>
__device__ void suffix_chunk_mfma(const StepArgs& a, int s, int c, int g, float* smem) {
  using RM = RespMfma<SH>;
  constexpr int HPK = SH::HPK;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const SlotPlan& sp = a.slot[s];
  const int len = sp.len;
  const int t0 = c * a.split, t1 = min(t0 + a.split, len);
  const int sub = a.split / 4;
  const int wt0 = min(t0 + w * sub, t1), wt1 = min(wt0 + sub, t1);
  const int npg = (wt1 - wt0 + kPageTokens - 1) / kPageTokens;
  const int32_t* ptab = a.page_table + (int64_t)sp.seq * a.pages_per_slot + (wt0 >> 4);
  const int pages = lane < npg ? ptab[lane] : 0;
  const int last = len - 1;
  const bool has_new = last >= wt0 && last < wt1;
  const int te = has_new ? last : wt1;  // stored tokens of this wavefront: [wt0, te)
  typename RM::Regs R;
  RM::load_round((const char*)a.pool, pages, a.Hkv, g, 0, R);
  // queries and the newest token's rows in one batch of loads; that token is
  // folded in first and stored into its page
  bf16x8 bq[SH::KB];
  RM::load_q(a.q, (int64_t)s * a.Hq + g * HPK, bq);
  typename RM::NewRows N;
  if (has_new) {
    const int64_t newrow = ((int64_t)s * a.Hkv + g) * SH::ROWB;
    RM::load_new((const char*)a.knew + newrow, (const char*)a.vnew + newrow, N);
  }
  typename RM::Acc A;
  if (has_new) {
    RM::round_new(N);
    RM::start_new(N, bq, a.scale_log2, A);
    RM::store_new((char*)RM::page((const char*)a.pool, sp.cur_page, a.Hkv, g), last & 15, N);
  } else {
    RM::init(A);
  }
  for (int base = wt0; base < te; base += RM::TOK) {
    if (base != wt0) RM::load_round((const char*)a.pool, pages, a.Hkv, g, (base - wt0) >> 4, R);
    RM::round(R, bq, base, te, a.scale_log2, A);
  }
  RM::publish(smem, A);
  const int64_t rec0 = prefix_records(a, SH::PR) + (((int64_t)s * a.Hkv + g) * a.suffix_chunks_max + c) * HPK;
  combine_store_partial<SH, HPK, L2>(smem, Exchange<L2>(a), rec0);

  if (t1 == len && g == 0 && threadIdx.x == 0) {  // bookkeeping of this step's token (K/V stored above)
    const int pos = len - 1;
    a.page_table[(int64_t)sp.seq * a.pages_per_slot + (pos >> 4)] = sp.cur_page;
    if (a.count_tokens)
      __hip_atomic_fetch_add(&a.tokens[(s / a.m) * a.G + sp.sample], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ----------------------------------------------------------------------------
// Merge all partials of (slot s, KV head g) and write O rows g*hpk .. +hpk-1
// (the log-sum-exp combination of split-K partial softmaxes).  Partial c < nP
// is prefix chunk c, then the response chunks.  The hpk*d outputs are cut into
// 4-float vectors, one per lane (MV vectors per lane when they exceed 64); the
// partials are dealt round-robin to the four wavefronts, each of which loads a
// round of MCU partials at once (16-byte loads, no load waits on another) and
// folds them into a running (max, sum, output); the four wavefronts' results
// are then combined through LDS.
// ----------------------------------------------------------------------------
template <class SH>
struct MergeShape {
  static constexpr int OPP = SH::HPK * SH::D;          // outputs per partial
  static constexpr int NVEC = OPP / 4;                 // 4-float vectors per partial
  static constexpr int MV = (NVEC + 63) / 64;          // vectors per lane
  static constexpr int MCU = MV == 1 ? 8 : 4;          // partials per load round and wavefront
  static constexpr int SMEM = 4 * 64 * MV * 8;         // per wave and lane vector: max, sum, 2 pad, 4 outputs
  static_assert(SH::D % 4 == 0, "vectors");
};

template <class SH, bool L2>
__device__ void merge_outputs(const StepArgs& a, int s, int g, float* smem) {
  using MS = MergeShape<SH>;
  constexpr int D = SH::D, HPK = SH::HPK, MV = MS::MV, MCU = MS::MCU;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int p = s / a.m, si = s - p * a.m;
  const int nP = a.prompt[p].nchunks;
  const int n = nP + (a.slot[s].len + a.split - 1) / a.split;
  const int64_t pbase = ((int64_t)p * a.Hkv + g) * a.prefix_chunks_max * SH::PR + si * HPK;
  const int64_t pstride = SH::PR;
  const int64_t sbase = prefix_records(a, SH::PR) + ((int64_t)s * a.Hkv + g) * a.suffix_chunks_max * HPK;
  const int64_t sstride = HPK;
  auto rec = [&](int c, int j) -> int64_t { return (c < nP ? pbase + c * pstride : sbase + (c - nP) * sstride) + j; };
  const Exchange<L2> ex(a);

  float M[MV], L[MV];
  f32x4 O[MV];
#pragma unroll
  for (int v = 0; v < MV; ++v) {
    M[v] = NEG_INF;
    L[v] = 0.f;
    O[v] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int c0 = w; c0 < n; c0 += 4 * MCU) {
    u32x2 ml[MCU][MV];
    f32x4 ov[MCU][MV];
#pragma unroll
    for (int u = 0; u < MCU; ++u) {
      const int c = c0 + 4 * u;
#pragma unroll
      for (int v = 0; v < MV; ++v) {
        const int x = (v * 64 + lane) * 4, j = x / D, d = x - j * D;
        if (c < n && x < MS::OPP) {
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
    for (int u = 0; u < MCU; ++u)
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
    float* e = smem + ((w * MV + v) * 64 + lane) * 8;
    e[0] = M[v];
    e[1] = L[v];
    *(f32x4*)(e + 4) = O[v];
  }
  __syncthreads();
  for (int t = threadIdx.x; t < MS::NVEC; t += kBlockThreads) {
    const int v = t >> 6, ln = t & 63;
    float mw[4], mx = NEG_INF;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      mw[q] = smem[((q * MV + v) * 64 + ln) * 8];
      mx = fmaxf(mx, mw[q]);
    }
    const float base = mx == NEG_INF ? 0.f : mx;
    float Lt = 0.f;
    f32x4 Ot = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float* e = smem + ((q * MV + v) * 64 + ln) * 8;
      const float wq = mw[q] == NEG_INF ? 0.f : exp2_fast(mw[q] - base);
      Lt += wq * e[1];
      Ot += *(const f32x4*)(e + 4) * wq;
    }
    const int x = t * 4, j = x / D, d = x - j * D;
    *(f32x4*)(a.o + ((int64_t)s * a.Hq + g * HPK + j) * D + d) = Ot * (1.f / Lt);
  }
}

// A producer block has stored its partial: once every thread's stores have
// completed, count one arrival on the counter of each live slot among slots
// first .. first + n - 1 (lane i adds for slot first + i; n <= 64).  A
// response chunk counts on its own slot, a prefix chunk on every live slot of
// its prompt, so a merge waits on a single counter that no other merge polls.
__device__ __forceinline__ void arrive(const StepArgs& a, int first, int n, int g) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_waitcnt(0);  // this thread's partial stores have completed
  __syncthreads();                // ... and so have every thread's
  if ((int)threadIdx.x < n && a.slot[first + threadIdx.x].len > 0)
    __hip_atomic_fetch_add(a.counters + (int64_t)((first + threadIdx.x) * a.Hkv + g) * kCounterStride, 1,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t* slot_counter(const StepArgs& a, int s, int g) {
  return a.counters + (int64_t)(s * a.Hkv + g) * kCounterStride;
}
// Counters wrap: `reached` compares by the sign of the difference.
__device__ __forceinline__ bool reached(const int32_t* ctr, int32_t target) {
  const int32_t v = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return (int32_t)((uint32_t)v - (uint32_t)target) >= 0;
}

// Merge block of (slot s, KV head g): wait until the prefix chunks of its
// prompt and its own response chunks have all arrived on its counter
// (bounded), then merge.
template <class SH, bool L2>
__device__ void merge_block(const StepArgs& a, int s, int g, unsigned long long* flag, float* smem) {
  if (threadIdx.x == 0) {
    const int32_t* sc = slot_counter(a, s, g);
    const int32_t target = a.slot[s].target;
    bool ok = false;
    if (a.merge_polls >= 0) {
      ok = reached(sc, target);
      for (int spins = 0; !ok && spins < a.merge_polls; ++spins) {
        __builtin_amdgcn_s_sleep(2);
        ok = reached(sc, target);
      }
    }
    *flag = ok;
  }
  __syncthreads();
  if (!*flag) {
    if (threadIdx.x == 0) __hip_atomic_store(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    float* o = a.o + ((int64_t)s * a.Hq + g * SH::HPK) * SH::D;
    for (int idx = threadIdx.x; idx < SH::HPK * SH::D; idx += kBlockThreads) o[idx] = __builtin_nanf("");
    return;
  }
  merge_outputs<SH, L2>(a, s, g, smem);
}

template <class SH, bool L2>
__device__ __forceinline__ void decode_block(const StepArgs& a, float* smem, unsigned long long* flagp) {
  const int item = blockIdx.x / a.Hkv;
  const int g = blockIdx.x - item * a.Hkv;
  if (L2 && threadIdx.x == 0 &&
      (__builtin_amdgcn_s_getreg(kXccIdReg) & 15) != (int)((blockIdx.x + a.l2_check_shift) % a.l2_xcds))
    __hip_atomic_store(a.status, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (item < a.n_prefix_items) {
    int p = 0;
    while (p < a.num_prompts - 1 && !(a.prompt[p].nchunks > 0 && item < a.prompt[p].item_begin + a.prompt[p].nchunks))
      ++p;
    const int c = item - a.prompt[p].item_begin;
    if constexpr (SH::MFMA)
      prefix_mfma<SH, L2>(a, p, c, g, smem);
    else
      prefix_wave<SH, L2>(a, p, c, g, smem);
    arrive(a, p * a.m, a.m, g);
    return;
  }
  int it = item - a.n_prefix_items;
  if (it < a.n_suffix_items) {
    const int lane = threadIdx.x & 63;
    bool hit = false;
    if (lane < a.S) {
      const int len = a.slot[lane].len, b = a.slot[lane].item_begin;
      hit = len > 0 && it >= b && it < b + (len + a.split - 1) / a.split;
    }
    const int s = __ffsll((long long)__ballot(hit)) - 1;
    if (s < 0) return;  // unreachable with a consistent plan
    const int c = it - a.slot[s].item_begin;
    suffix_chunk<SH, L2>(a, s, c, g, smem);
    arrive(a, s, 1, g);
    return;
  }
  it -= a.n_suffix_items;
  if (it < a.n_zero_items) {
    const int s = a.zero_slot[it];
    float* o = a.o + ((int64_t)s * a.Hq + g * SH::HPK) * SH::D;
    for (int idx = threadIdx.x; idx < SH::HPK * SH::D; idx += kBlockThreads) o[idx] = 0.f;
    return;
  }
  it -= a.n_zero_items;
  merge_block<SH, L2>(a, a.live_slot[it], g, flagp, smem);
}

// One kernel per shape and exchange policy (L2: partials through the XCD's
// L2; the host launches the one that matches StepArgs::l2_xcds).  Timing mode
// (a.clock_start != null): every block folds its start and end time (device
// wall clock) into one of this launch's start / end slots.
template <class SH, bool L2>
__global__ __launch_bounds__(kBlockThreads, SH::MIN_WAVES) void decode_kernel(const StepArgs a) {
  constexpr int SMEM = SH::SMEM > MergeShape<SH>::SMEM ? SH::SMEM : MergeShape<SH>::SMEM;
  __shared__ __attribute__((aligned(16))) float smem[SMEM];
  __shared__ unsigned long long flag;
  const int cs = (blockIdx.x % kClockSlots) * kClockStride;
  if (a.clock_start && threadIdx.x == 0)
    __hip_atomic_fetch_min(a.clock_start + cs, (unsigned long long)__builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
  decode_block<SH, L2>(a, smem, &flag);
  if (a.clock_start) {
    __syncthreads();
    if (threadIdx.x == 0)
      __hip_atomic_fetch_max(a.clock_end + cs, (unsigned long long)__builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ----------------------------------------------------------------------------
// Prefill: [plen, Hkv, D] -> prefix store.  One thread per 16-byte unit.
// ----------------------------------------------------------------------------
template <class SH>
__global__ __launch_bounds__(256) void prefill_plain_kernel(char* store, const char* k, const char* v, int prompt,
                                                           int plen, int hkv, int pmax) {
  const int64_t units = (int64_t)hkv * 2 * plen * SH::LPT;
  for (int64_t u = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; u < units; u += (int64_t)gridDim.x * blockDim.x) {
    const int ch = u % SH::LPT;
    const int64_t r = u / SH::LPT;
    const int j = r % plen;
    const int kind = (r / plen) % 2;
    const int g = r / (2 * plen);
    const u32x4* src = (const u32x4*)((kind ? v : k) + ((int64_t)j * hkv + g) * SH::ROWB) + ch;
    char* dst = store + (((int64_t)prompt * hkv + g) * 2 + kind) * pmax * SH::ROWB + (int64_t)j * SH::ROWB;
    *((u32x4*)dst + ch) = *src;
  }
}

// MFMA layout per (prompt, kv head), per 32-token block: a K block of
// [2 token halves][KB][64 lanes][8] and a V block of [DB][64 lanes][8].
// K unit (mb, kb, lane): tokens mb*16 + lane%16, dims kb*32 + 8*(lane/16) + e.
// V unit (db, lane): dim db*16 + lane%16, tokens tau(8*(lane/16) + e) where
// tau(8q+e) = 4q+e for e < 4 and 16+4q+(e-4) otherwise -- the order in which
// a lane holds probabilities after the S^T tiles.  Padding tokens are zero.
template <class SH>
__global__ __launch_bounds__(256) void prefill_mfma_kernel(char* store, const uint16_t* k, const uint16_t* v,
                                                          int prompt, int plen, int hkv, int pmax) {
  constexpr int D = SH::D, KB = SH::KB, DB = SH::DB, KES = SH::KES;
  constexpr int KU = 2 * KB * 64, VU = DB * 64, BU = KU + VU;
  const int nblk = (plen + kMfmaBlock - 1) / kMfmaBlock;
  const int64_t units = (int64_t)hkv * nblk * BU;
  for (int64_t u = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; u < units; u += (int64_t)gridDim.x * blockDim.x) {
    const int g = u / ((int64_t)nblk * BU);
    const int rem = u - (int64_t)g * nblk * BU;
    const int b = rem / BU;
    int x = rem - b * BU;
    char* blk = store + (((int64_t)prompt * hkv + g) * (pmax / kMfmaBlock) + b) * (2 * kMfmaBlock * D * KES);
    uint16_t vals[8];
    char* dst;
    if (x < KU) {
      const int lane = x & 63, sub = x >> 6, mb = sub / KB, kb = sub - mb * KB;
      const int tok = b * kMfmaBlock + mb * 16 + (lane & 15);
      const int d0 = kb * 32 + (lane >> 4) * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) vals[e] = tok < plen ? k[((int64_t)tok * hkv + g) * D + d0 + e] : 0;
      dst = blk + (int64_t)x * 8 * KES;
    } else {
      x -= KU;
      const int lane = x & 63, db = x >> 6, qq = lane >> 4;
      const int d = db * 16 + (lane & 15);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int tok = b * kMfmaBlock + (e < 4 ? 4 * qq + e : 16 + 4 * qq + (e - 4));
        vals[e] = tok < plen ? v[((int64_t)tok * hkv + g) * D + d] : 0;
      }
      dst = blk + (int64_t)kMfmaBlock * D * KES + (int64_t)x * 8 * KES;
    }
    u32x4 w;
    w.x = vals[0] | ((uint32_t)vals[1] << 16);
    w.y = vals[2] | ((uint32_t)vals[3] << 16);
    w.z = vals[4] | ((uint32_t)vals[5] << 16);
    w.w = vals[6] | ((uint32_t)vals[7] << 16);
    st_kv<SH>(dst, w);
  }
}

}  // namespace
}  // namespace infs
