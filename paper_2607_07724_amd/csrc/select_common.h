// Helpers shared by the scoring/selection kernels and the diagnostics
// kernels: the Quest split of a query row into its negative and positive
// parts, order-preserving score keys, the radix k-th largest, top-R
// compaction and a wave-local LDS bitonic sort.
#pragma once
#include "ugbs_internal.h"

namespace ugbs {
namespace {

// bf16 lanes of v with the sign bit set (negative part) / clear (positive
// part), the other lanes zeroed: q- = min(q, 0) and q+ = max(q, 0) exactly.
__device__ __forceinline__ uint4 neg_part(uint4 v) {
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t m = ((w[e] >> 15) & 0x00010001u) * 0xffffu;
    w[e] &= m;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ uint4 pos_part(uint4 v) {
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t m = ((w[e] >> 15) & 0x00010001u) * 0xffffu;
    w[e] &= ~m;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

typedef __attribute__((__vector_size__(16 * sizeof(__bf16)))) __bf16 bf16x16;
struct U4Pair {
  uint4 lo, hi;
};
__device__ __forceinline__ bf16x16 as_bf16x16(uint4 lo, uint4 hi) {
  return __builtin_bit_cast(bf16x16, (U4Pair{lo, hi}));
}

// The Quest bound of Eq. (quest-score) as a 2:4-sparse contraction.  For
// each channel c, max(q_c kmax_c, q_c kmin_c) = q_c * (q_c > 0 ? kmax_c :
// kmin_c).  With the uncompressed operand ordered k = 2 c + {0: kmin, 1:
// kmax}, every group of four k (channels 2i, 2i + 1) holds exactly two
// selected entries, so v_smfmac_f32_16x16x64_bf16 computes the bound of 32
// channels per k-step with the raw query values as its compressed A operand
// (lane group g of a k-step holds channels 8 g .. 8 g + 7, element e being
// channel 8 g + e, the second of its group when e is odd) and these indices:
// element e sits at position 2 (e mod 2) + [q > 0] of its group, two bits
// per element, element 0 lowest.  q = +0 or -0 selects kmin (a zero
// product either way).
__device__ __forceinline__ uint32_t quest_index(uint4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t idx = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = w[i] & 0xffffu, hi = w[i] >> 16;
    const uint32_t plo = (lo != 0u && !(lo & 0x8000u)) ? 1u : 0u;
    const uint32_t phi = 2u + ((hi != 0u && !(hi & 0x8000u)) ? 1u : 0u);
    idx |= (plo << (4 * i)) | (phi << (4 * i + 2));
  }
  return idx;
}

// Set bits of the wave mask m held by lanes below this one (v_mbcnt: two
// VALU operations, no mask-and-popcount per lane).
__device__ __forceinline__ int lanes_below(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Integer minimum (a mixed-type min() call can resolve to the floating-point
// overload and go through double precision).
__device__ __forceinline__ int imin(int a, int b) { return a < b ? a : b; }

// fp32 score -> 32-bit key with the same order (-0 folded into +0, so equal
// scores give equal keys); key_value inverts it.
__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f == 0.0f ? 0.0f : f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Largest thr with at least R of the keys held in key[0..nslots) at or above
// it (0 = empty slot): a most-significant-bit-first radix descent that
// counts with wave ballots.  *exact: exactly R keys are >= thr.
template <int S>
__device__ __forceinline__ uint32_t kth_largest(const uint32_t (&key)[S], int nslots, int R, bool* exact) {
  uint32_t thr = 0;
  *exact = false;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = thr | (1u << bit);
    int cnt = 0;
#pragma unroll
    for (int sl = 0; sl < S; ++sl)
      if (sl < nslots) cnt += __popcll(__ballot(key[sl] >= cand));
    if (cnt >= R) {
      thr = cand;
      if (cnt == R) {
        *exact = true;
        break;
      }
    }
  }
  return thr;
}

// R largest of the keys held in key[0..nslots) (0 = empty; entries in
// position order slot by slot, lane by lane), written to s_sel[0..R) as
// (key << 32) | ~position, unsorted: the R-th largest key thr comes from
// kth_largest, then keys above thr and the lowest-position keys equal to
// thr are compacted.
template <int S>
__device__ __forceinline__ void select_top(const uint32_t (&key)[S], const uint32_t (&pos)[S],
                                           int nslots, int R, uint64_t* s_sel, int lane) {
  bool exact;
  const uint32_t thr = kth_largest<S>(key, nslots, R, &exact);
  int base = 0;
#pragma unroll
  for (int sl = 0; sl < S; ++sl) {
    if (sl < nslots) {
      const bool take = exact ? (key[sl] >= thr) : (key[sl] > thr);
      const uint64_t mk = __ballot(take);
      if (take) s_sel[base + lanes_below(mk)] = ((uint64_t)key[sl] << 32) | (0xffffffffu - pos[sl]);
      base += __popcll(mk);
    }
  }
  if (!exact) {
    int need = R - base;
#pragma unroll
    for (int sl = 0; sl < S; ++sl) {
      if (sl < nslots && need > 0) {
        const bool eq = key[sl] == thr;
        const uint64_t mk = __ballot(eq);
        const int r = lanes_below(mk);
        if (eq && r < need) s_sel[base + r] = ((uint64_t)thr << 32) | (0xffffffffu - pos[sl]);
        const int took = imin(__popcll(mk), need);
        base += took;
        need -= took;
      }
    }
  }
}

// The same R largest keys as select_top, reported through
// take(slot) on the lane that holds each of them (no order, no storage).
// Returns nothing; every lane of the wave must call it.
template <int S, typename Take>
__device__ __forceinline__ void select_top_each(const uint32_t (&key)[S], int nslots, int R, int lane,
                                                Take&& take) {
  bool exact;
  const uint32_t thr = kth_largest<S>(key, nslots, R, &exact);
  int above = 0;
#pragma unroll
  for (int sl = 0; sl < S; ++sl) {
    if (sl < nslots) {
      const bool tk = exact ? (key[sl] >= thr) : (key[sl] > thr);
      if (tk) take(sl);
      above += __popcll(__ballot(tk));
    }
  }
  if (!exact) {
    int need = R - above;
#pragma unroll
    for (int sl = 0; sl < S; ++sl) {
      if (sl < nslots && need > 0) {
        const bool eq = key[sl] == thr;
        const uint64_t mk = __ballot(eq);
        if (eq && lanes_below(mk) < need) take(sl);
        need -= imin(__popcll(mk), need);
      }
    }
  }
}

// LDS hand-off between lanes of one wave: LDS operations of a wave complete
// in order, so waiting for this wave's outstanding ones is enough.
__device__ __forceinline__ void wave_lds_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_wave_barrier();
}

// Descending bitonic sort of s[0..n2) (n2 a power of two) by one wave.
__device__ __forceinline__ void lds_bitonic_desc(uint64_t* s, int n2, int lane) {
  for (int size = 2; size <= n2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = lane; i < (n2 >> 1); i += 64) {
        const int lo = 2 * stride * (i / stride) + (i % stride);
        const int hi = lo + stride;
        const uint64_t x = s[lo], y = s[hi];
        const bool desc = (lo & size) == 0;
        if (desc ? (x < y) : (x > y)) {
          s[lo] = y;
          s[hi] = x;
        }
      }
      wave_lds_sync();
    }
  }
}

}  // namespace
}  // namespace ugbs
