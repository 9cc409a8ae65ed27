// Stage 1: per-key-block metadata (A.1; Quest pair of Eq. (quest-score)).
//
// One thread owns 8 consecutive channels of one (batch, kv head, block) and
// walks the block's 64 keys with 16-byte loads; d/8 consecutive threads cover
// a key row, so each row is read as one contiguous segment.  K is streamed
// exactly once: the kernel is HBM-bound (algorithmic bytes per block:
// 64*d*2 read + c*d*2 written, c = 1 K-mean, 2 Quest).
//
// K-mean: the 64 values of a channel are summed in fp64 in key order (exact
// for bf16 inputs of ordinary range), divided by 64 (exact), and rounded to
// bf16 once: fp64 -> fp32 with round-to-odd, then fp32 -> bf16 nearest-even,
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

template <int D, bool QUEST>
__global__ void __launch_bounds__(256) block_meta_kernel(const uint16_t* __restrict__ K,
                                                         uint16_t* __restrict__ meta,
                                                         long n_items, int N) {
  constexpr int CG = D / 8;  // 16-byte column groups per key row
  const long item = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (item >= n_items) return;
  const int cg = (int)(item % CG);
  const long bh_blk = item / CG;                     // (b*Hkv + kvh) * NB + blk
  const int NB = N / kBlock;
  const long bh = bh_blk / NB;
  const int blk = (int)(bh_blk % NB);
  const uint4* src = reinterpret_cast<const uint4*>(
      K + ((size_t)bh * N + (size_t)blk * kBlock) * D + cg * 8);
  constexpr int kRowStride = D / 8;                  // in uint4

  if constexpr (!QUEST) {
    double acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0;
#pragma unroll 8
    for (int j = 0; j < kBlock; ++j) {
      const uint4 v = *(src + (size_t)j * kRowStride);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] += (double)bf16_lo(w[e]);
        acc[2 * e + 1] += (double)bf16_hi(w[e]);
      }
    }
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      o[e] = bf16_from_f64(acc[2 * e] * (1.0 / kBlock)) |
             (bf16_from_f64(acc[2 * e + 1] * (1.0 / kBlock)) << 16);
    uint4* dst = reinterpret_cast<uint4*>(meta + (size_t)bh_blk * D + cg * 8);
    *dst = make_uint4(o[0], o[1], o[2], o[3]);
  } else {
    float lo[8], hi[8];
    {
      const uint4 v = *(src);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[2 * e] = hi[2 * e] = bf16_lo(w[e]);
        lo[2 * e + 1] = hi[2 * e + 1] = bf16_hi(w[e]);
      }
    }
#pragma unroll 8
    for (int j = 1; j < kBlock; ++j) {
      const uint4 v = *(src + (size_t)j * kRowStride);
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
    uint32_t omin[4], omax[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      omin[e] = exact_bf16_bits(lo[2 * e]) | (exact_bf16_bits(lo[2 * e + 1]) << 16);
      omax[e] = exact_bf16_bits(hi[2 * e]) | (exact_bf16_bits(hi[2 * e + 1]) << 16);
    }
    uint16_t* row = meta + (size_t)bh_blk * 2 * D + cg * 8;
    *reinterpret_cast<uint4*>(row) = make_uint4(omin[0], omin[1], omin[2], omin[3]);
    *reinterpret_cast<uint4*>(row + D) = make_uint4(omax[0], omax[1], omax[2], omax[3]);
  }
}

}  // namespace

hipError_t launch_block_meta(const Shape& s, const uint16_t* K, uint16_t* meta,
                             hipStream_t stream) {
  const long n_items = (long)s.B * s.Hkv * s.NB * (s.d / 8);
  const int threads = 256;
  const unsigned grid = (unsigned)((n_items + threads - 1) / threads);
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
