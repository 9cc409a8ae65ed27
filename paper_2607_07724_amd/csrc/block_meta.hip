// Stage 1: per-key-block metadata (A.1; Quest pair of Eq. (quest-score)).
//
// One wave per (batch, kv head, block): lane l owns 8 consecutive channels
// (column group l mod d/8) of the block's keys in part l / (d/8), a range of
// 64 / (64 / (d/8)) consecutive keys, read with 16-byte loads; d/8
// consecutive lanes cover a key row, so each row is one contiguous segment.
// The parts are combined across lanes (XOR shuffles).  K is streamed exactly
// once: the kernel is HBM-bound (algorithmic bytes per block: 64*d*2 read +
// c*d*2 written, c = 1 K-mean, 2 Quest).  Quest rows hold, per channel, the
// pair (minimum, maximum) adjacently.
//
// K-mean: the 64 values of a channel are summed in fp64 (every partial sum
// is exact when the nonzero values' binary exponents lie within 39 of each
// other: 8 significant bits each plus 6 bits of carry fit in 53, so the
// grouping of the sum does not matter there), divided by 64 (exact), and rounded to bf16 once: fp64 -> fp32 with round-to-odd, then fp32 -> bf16 nearest-even,
// which equals direct nearest-even rounding because fp32 keeps >= 2 extra
// bits.  Quest: element-wise fp32 min / max (exact).  Zeros are written +0.
#include "ugbs_internal.h"

namespace ugbs {
namespace {

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 holding a bf16 value (or +-0) -> its bf16 pattern, with -0 -> +0.
__device__ __forceinline__ uint32_t exact_bf16_bits(float x) {
  return x == 0.0f ? 0u : (__float_as_uint(x) >> 16);
}

__device__ __forceinline__ uint32_t bf16_from_f64(double x) {
  if (x == 0.0) return 0u;
  float f = __double2float_rz(x);
  uint32_t u = __float_as_uint(f);
  if ((double)f != x) u |= 1u;                       // round to odd (sticky bit)
  u += 0x7fffu + ((u >> 16) & 1u);                   // nearest-even to 16 bits
  return u >> 16;
}

// 16-byte streaming load (K is read once here)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_nt(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// Cross-lane combine of the per-part partial results (lanes l and l ^ m).
__device__ __forceinline__ double xor_add(double x, int m) {
  const int lo = __shfl_xor(__double2loint(x), m), hi = __shfl_xor(__double2hiint(x), m);
  return x + __hiloint2double(hi, lo);
}

template <int D, bool QUEST>
__global__ void __launch_bounds__(256) block_meta_kernel(const uint16_t* __restrict__ K,
                                                         uint16_t* __restrict__ meta,
                                                         long n_blocks, int N) {
  constexpr int CG = D / 8;            // 16-byte column groups per key row
  constexpr int PARTS = 64 / CG;       // key ranges per block, one wave per block
  constexpr int KPP = kBlock / PARTS;  // keys per part
  const long bh_blk = (long)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
  if (bh_blk >= n_blocks) return;      // whole waves leave together
  const int lane = threadIdx.x & 63;
  const int cg = lane % CG, part = lane / CG;
  const int NB = N / kBlock;
  const long bh = bh_blk / NB;
  const int blk = (int)(bh_blk % NB);
  // one load instruction of the wave reads PARTS rows of d*2 contiguous bytes
  const uint4* src = reinterpret_cast<const uint4*>(
      K + ((size_t)bh * N + (size_t)blk * kBlock + (size_t)part * KPP) * D + cg * 8);
  constexpr int kRowStride = D / 8;                  // in uint4

  if constexpr (!QUEST) {
    // partial sums of KPP keys each; all partial and total sums are exact in
    // fp64, so the grouping does not change the result
    double acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0;
#pragma unroll
    for (int j = 0; j < KPP; ++j) {
      const uint4 v = load_nt(src + (size_t)j * kRowStride);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] += (double)bf16_lo(w[e]);
        acc[2 * e + 1] += (double)bf16_hi(w[e]);
      }
    }
#pragma unroll
    for (int m = CG; m < 64; m *= 2)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = xor_add(acc[e], m);
    if (part == 0) {
      uint32_t o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = bf16_from_f64(acc[2 * e] * (1.0 / kBlock)) |
               (bf16_from_f64(acc[2 * e + 1] * (1.0 / kBlock)) << 16);
      uint4* dst = reinterpret_cast<uint4*>(meta + (size_t)bh_blk * D + cg * 8);
      *dst = make_uint4(o[0], o[1], o[2], o[3]);
    }
  } else {
    float lo[8], hi[8];
    {
      const uint4 v = load_nt(src);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[2 * e] = hi[2 * e] = bf16_lo(w[e]);
        lo[2 * e + 1] = hi[2 * e + 1] = bf16_hi(w[e]);
      }
    }
#pragma unroll
    for (int j = 1; j < KPP; ++j) {
      const uint4 v = load_nt(src + (size_t)j * kRowStride);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = bf16_lo(w[e]), b = bf16_hi(w[e]);
        lo[2 * e] = a < lo[2 * e] ? a : lo[2 * e];
        hi[2 * e] = a > hi[2 * e] ? a : hi[2 * e];
        lo[2 * e + 1] = b < lo[2 * e + 1] ? b : lo[2 * e + 1];
        hi[2 * e + 1] = b > hi[2 * e + 1] ? b : hi[2 * e + 1];
      }
    }
#pragma unroll
    for (int m = CG; m < 64; m *= 2)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float a = __shfl_xor(lo[e], m), b = __shfl_xor(hi[e], m);
        lo[e] = a < lo[e] ? a : lo[e];
        hi[e] = b > hi[e] ? b : hi[e];
      }
    if (part == 0) {
      // channel pairs (min, max) adjacent: the lane's 8 channels are 32
      // contiguous bytes of the block's 2 d-long row
      uint32_t pr[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) pr[e] = exact_bf16_bits(lo[e]) | (exact_bf16_bits(hi[e]) << 16);
      uint16_t* row = meta + (size_t)bh_blk * 2 * D + 2 * cg * 8;
      *reinterpret_cast<uint4*>(row) = make_uint4(pr[0], pr[1], pr[2], pr[3]);
      *reinterpret_cast<uint4*>(row + 8) = make_uint4(pr[4], pr[5], pr[6], pr[7]);
    }
  }
}

}  // namespace

hipError_t launch_block_meta(const Shape& s, const uint16_t* K, uint16_t* meta,
                             hipStream_t stream) {
  const long n_items = (long)s.B * s.Hkv * s.NB;   // key blocks, one wave each
  const int threads = 256;
  const unsigned grid = (unsigned)((n_items + threads / 64 - 1) / (threads / 64));
  if (s.d == 256) {
    if (s.backbone == UGBS_QUEST)
      block_meta_kernel<256, true><<<grid, threads, 0, stream>>>(K, meta, n_items, s.N);
    else
      block_meta_kernel<256, false><<<grid, threads, 0, stream>>>(K, meta, n_items, s.N);
  } else if (s.d == 128) {
    if (s.backbone == UGBS_QUEST)
      block_meta_kernel<128, true><<<grid, threads, 0, stream>>>(K, meta, n_items, s.N);
    else
      block_meta_kernel<128, false><<<grid, threads, 0, stream>>>(K, meta, n_items, s.N);
  } else {
    if (s.backbone == UGBS_QUEST)
      block_meta_kernel<64, true><<<grid, threads, 0, stream>>>(K, meta, n_items, s.N);
    else
      block_meta_kernel<64, false><<<grid, threads, 0, stream>>>(K, meta, n_items, s.N);
  }
  return hipGetLastError();
}

}  // namespace ugbs
