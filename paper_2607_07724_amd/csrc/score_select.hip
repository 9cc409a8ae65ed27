// Stages 2+3: tile scores, forcing, sorted top-2k and the cutoff margin
// (A.2-A.6; Eqs. (tile-score), (sigma-def)).
//
// One wave per (batch, query head, Q-tile) unit.
//
// Scoring is a dense contraction on bf16 MFMA (v_mfma_f32_16x16x32_bf16):
//   S[64 rows x 16 blocks] = Qx[64 x KD] * Mx[KD x 16 blocks]
// with, for K-mean, Qx = Q and Mx = kbar (KD = d), and for Quest the exact
// split form of Eq. (quest-score): for kmax >= kmin,
//   max(q kmax, q kmin) = min(q,0) kmin + max(q,0) kmax,
// so Qx = [q- | q+] and Mx = [kmin | kmax] (KD = 2d, the metadata row as
// stored).  Every product is an exact bf16 x bf16 product; sums are fp32.
// The 64-row Qx tile stays in registers as the A operand; metadata rows are
// the B operand, loaded straight from global memory (they are shared by all
// tiles of a kv head and stay L2-resident).  The max over the tile's rows
// (A.3) is the max over a lane's 16 accumulators and then across the four
// 16-lane groups.
//
// Selection: tile scores become order-preserving 32-bit keys in LDS
// (-0 folded into +0).  The R-th largest key (R = min(2k - |F|, |C|)) is found
// by a most-significant-bit-first radix descent that counts with wave ballots,
// the survivors are compacted (equal keys at the threshold by lower block
// index), and a bitonic sort of (key, ~index) pairs orders them.  sigma uses
// IEEE fp32 subtract and divide.
#include "ugbs_internal.h"

namespace ugbs {
namespace {

struct SelParams {
  Shape s;
  const uint16_t* Q;
  const uint16_t* meta;
  const float* scores_in;
  float* scores_out;
  int32_t* idx_sorted;
  float* sigma;
  int n_units;
  int sel_cap;  // power of two >= max survivors
};

__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f == 0.0f ? 0.0f : f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

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

__device__ __forceinline__ float wave_max16(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}

// Scores of candidate blocks 1..t-1 of one unit -> keys in s_key[blk - 1].
template <int D, bool QUEST>
__device__ __forceinline__ void score_unit(const SelParams& P, const Unit& u, int nc,
                                           uint32_t* s_key) {
  constexpr int KD = QUEST ? 2 * D : D;
  constexpr int KS = KD / 32;
  const Shape& s = P.s;
  const int lane = threadIdx.x;
  const int g = lane >> 4, c16 = lane & 15;
  const int kvh = u.h / s.G;

  // A operand: 4 row tiles x KS k-steps, 8 bf16 per lane each.
  bf16x8 a[4][KS];
  const uint16_t* qtile = P.Q + (((size_t)u.b * s.H + u.h) * s.N + (size_t)u.t * kBlock) * D;
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    const uint16_t* qrow = qtile + (size_t)(16 * rt + c16) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if constexpr (QUEST) {
        const int kk = (ks % (D / 32)) * 32 + 8 * g;
        const uint4 v = *reinterpret_cast<const uint4*>(qrow + kk);
        a[rt][ks] = as_bf16x8(ks < D / 32 ? neg_part(v) : pos_part(v));
      } else {
        a[rt][ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qrow + 32 * ks + 8 * g));
      }
    }
  }

  const uint16_t* mhead = P.meta + ((size_t)u.b * s.Hkv + kvh) * s.NB * KD;
  const int nchunks = (nc + 15) / 16;
  auto load_b = [&](int c, bf16x8* b) {
    int blk = 1 + 16 * c + c16;
    if (blk > nc) blk = 1;  // lanes past the last candidate read a valid row
    const uint16_t* mrow = mhead + (size_t)blk * KD + 8 * g;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) b[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(mrow + 32 * ks));
  };

  bf16x8 bcur[KS], bnext[KS];
  load_b(0, bcur);
  for (int c = 0; c < nchunks; ++c) {
    if (c + 1 < nchunks) load_b(c + 1, bnext);
    f32x4 acc[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
        acc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rt][ks], bcur[ks], acc[rt], 0, 0, 0);
    float m = acc[0][0];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int i = 0; i < 4; ++i) m = fmaxf(m, acc[rt][i]);
    m = wave_max16(m);
    const int pos = 16 * c + c16;
    if (g == 0 && pos < nc) s_key[pos] = order_key(m);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) bcur[ks] = bnext[ks];
  }
}

template <int D, bool QUEST>
__global__ void __launch_bounds__(64) score_select_kernel(SelParams P) {
  extern __shared__ __align__(16) unsigned char smem[];
  const Shape& s = P.s;
  uint32_t* s_key = reinterpret_cast<uint32_t*>(smem);                       // [NB]
  uint64_t* s_sel = reinterpret_cast<uint64_t*>(smem + ((s.NB * 4 + 15) & ~15));  // [sel_cap]
  const int lane = threadIdx.x;

  const int uid = xcd_remap(blockIdx.x, P.n_units);
  if (uid >= P.n_units) return;
  const Unit u = unit_of(uid, s);
  const size_t row = ((size_t)u.b * s.H + u.h) * s.T + u.t;
  const int nf = (u.t == 0) ? 1 : 2;
  const int nc = (u.t >= 1) ? u.t - 1 : 0;
  const int m = s.k - nf;
  const int W = s.W;
  const int R = min(W - nf, nc);

  if (nc > 0) {
    if (P.scores_in) {
      const float* src = P.scores_in + row * s.NB + 1;
      for (int p = lane; p < nc; p += 64) s_key[p] = order_key(src[p]);
    } else {
      score_unit<D, QUEST>(P, u, nc, s_key);
    }
  }
  __syncthreads();

  if (P.scores_out) {
    float* dst = P.scores_out + row * s.NB;
    for (int p = lane; p < s.NB; p += 64)
      dst[p] = (p >= 1 && p <= nc) ? key_value(s_key[p - 1]) : -__builtin_huge_valf();
  }

  int32_t* out = P.idx_sorted + row * W;
  if (nc == 0) {
    for (int p = lane; p < W; p += 64) out[p] = (p < nf) ? (p == 0 ? 0 : u.t) : s.NB;
    if (lane == 0) P.sigma[row] = -1.0f;
    return;
  }

  // ---- R-th largest key by radix descent over the 32 key bits -------------
  constexpr int kMaxSlots = UGBS_MAX_BLOCKS / 64;
  const int nslots = (nc + 63) / 64;
  uint32_t keys[kMaxSlots];
#pragma unroll
  for (int sl = 0; sl < kMaxSlots; ++sl) {
    const int p = 64 * sl + lane;
    keys[sl] = (sl < nslots && p < nc) ? s_key[p] : 0u;  // valid keys are >= 0x007fffff
  }
  uint32_t thr = 0;
  bool exact = false;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = thr | (1u << bit);
    int cnt = 0;
#pragma unroll
    for (int sl = 0; sl < kMaxSlots; ++sl)
      if (sl < nslots) cnt += __popcll(__ballot(keys[sl] >= cand));
    if (cnt >= R) {
      thr = cand;
      if (cnt == R) {
        exact = true;
        break;
      }
    }
  }

  // ---- compact the survivors as (key, ~position) pairs --------------------
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int base = 0;
#pragma unroll
  for (int sl = 0; sl < kMaxSlots; ++sl) {
    if (sl < nslots) {
      const bool take = exact ? (keys[sl] >= thr) : (keys[sl] > thr);
      const uint64_t mk = __ballot(take);
      if (take) {
        const uint32_t pos = 64 * sl + lane;
        s_sel[base + __popcll(mk & lt_mask)] = ((uint64_t)keys[sl] << 32) | (0xffffffffu - pos);
      }
      base += __popcll(mk);
    }
  }
  if (!exact) {
    int need = R - base;
#pragma unroll
    for (int sl = 0; sl < kMaxSlots; ++sl) {
      if (sl < nslots && need > 0) {
        const bool eq = keys[sl] == thr;
        const uint64_t mk = __ballot(eq);
        const int r = __popcll(mk & lt_mask);
        if (eq && r < need) {
          const uint32_t pos = 64 * sl + lane;
          s_sel[base + r] = ((uint64_t)thr << 32) | (0xffffffffu - pos);
        }
        const int took = min(__popcll(mk), need);
        base += took;
        need -= took;
      }
    }
  }
  int n2 = 2;
  while (n2 < R) n2 <<= 1;
  for (int p = R + lane; p < n2; p += 64) s_sel[p] = 0ull;
  __syncthreads();

  // ---- bitonic sort, descending -------------------------------------------
  for (int size = 2; size <= n2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = lane; i < (n2 >> 1); i += 64) {
        const int lo = 2 * stride * (i / stride) + (i % stride);
        const int hi = lo + stride;
        const uint64_t x = s_sel[lo], y = s_sel[hi];
        const bool desc = (lo & size) == 0;
        if (desc ? (x < y) : (x > y)) {
          s_sel[lo] = y;
          s_sel[hi] = x;
        }
      }
      __syncthreads();
    }
  }

  // ---- outputs --------------------------------------------------------------
  for (int p = lane; p < W; p += 64) {
    int v;
    if (p < nf)
      v = (p == 0) ? 0 : u.t;
    else if (p - nf < R)
      v = 1 + (int)(0xffffffffu - (uint32_t)(s_sel[p - nf] & 0xffffffffu));
    else
      v = s.NB;
    out[p] = v;
  }
  if (lane == 0) {
    float sg = -1.0f;
    if (nc > m) {
#pragma clang fp contract(off)
      const float c0 = key_value((uint32_t)(s_sel[0] >> 32));
      const float cm1 = key_value((uint32_t)(s_sel[m - 1] >> 32));
      const float cm = key_value((uint32_t)(s_sel[m] >> 32));
      const float num = cm1 - cm;
      const float den = c0 - cm;
      sg = (den == 0.0f) ? 0.0f : __fdiv_rn(num, den);
    }
    P.sigma[row] = sg;
  }
}

template <int D, bool QUEST>
hipError_t launch_t(const SelParams& P, hipStream_t stream) {
  const size_t smem = ((P.s.NB * 4 + 15) & ~15) + sizeof(uint64_t) * (size_t)P.sel_cap;
  const int grid = ((P.n_units + 7) / 8) * 8;
  score_select_kernel<D, QUEST><<<grid, 64, smem, stream>>>(P);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score_select(const Shape& s, const uint16_t* Q, const uint16_t* meta,
                               const float* scores_in, float* scores_out,
                               int32_t* idx_sorted, float* sigma, hipStream_t stream) {
  SelParams P;
  P.s = s;
  P.Q = Q;
  P.meta = meta;
  P.scores_in = scores_in;
  P.scores_out = scores_out;
  P.idx_sorted = idx_sorted;
  P.sigma = sigma;
  P.n_units = s.B * s.H * s.T;
  int cap = 2;
  const int rmax = s.W < s.NB ? s.W : s.NB;
  while (cap < rmax) cap <<= 1;
  P.sel_cap = cap;
  if (s.d == 128)
    return s.backbone == UGBS_QUEST ? launch_t<128, true>(P, stream) : launch_t<128, false>(P, stream);
  return s.backbone == UGBS_QUEST ? launch_t<64, true>(P, stream) : launch_t<64, false>(P, stream);
}

}  // namespace ugbs
