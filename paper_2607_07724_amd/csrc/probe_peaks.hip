// Matrix-core and LDS-fill ceilings of the device this runs on, for the
// benchmark's roofline context (libugbs_probe.so; not part of the method's
// path).
//
// Each wave issues back-to-back matrix instructions on eight independent
// accumulator chains (enough to keep the pipeline full at two or more waves
// per SIMD) for `iters` iterations; the A/B operands alternate between two
// register sets of pseudo-random bf16 values every iteration, so the
// multipliers toggle as they do on real data (constant operands would draw
// less power and let the chip hold a higher clock).  The accumulators are
// summed and stored, so nothing is dead code.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ugbs_probe.h"

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(__bf16)))) __bf16 bf16x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kChains = 8;
constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t mix(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

// bf16 lanes with exponents near 1.0 (sign, exponent 126-127, random mantissa)
__device__ __forceinline__ uint32_t rnd_pair(uint32_t s) {
  const uint32_t r = mix(s);
  return (r & 0x807f807fu) | 0x3f003f80u;
}

template <int N>
__device__ __forceinline__ void fill(uint32_t (&w)[N], uint32_t seed) {
#pragma unroll
  for (int i = 0; i < N; ++i) w[i] = rnd_pair(seed * 131u + i);
}

template <bool SPARSE>
__global__ void __launch_bounds__(kThreads) mfma_loop(float* out, int iters) {
  const uint32_t tid = blockIdx.x * kThreads + threadIdx.x;
  f32x4 acc[kChains];
#pragma unroll
  for (int j = 0; j < kChains; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  if constexpr (!SPARSE) {
    uint32_t a0[4], a1[4], b0[4], b1[4];
    fill(a0, tid * 4 + 0);
    fill(a1, tid * 4 + 1);
    fill(b0, tid * 4 + 2);
    fill(b1, tid * 4 + 3);
    const bf16x8 A0 = __builtin_bit_cast(bf16x8, a0), A1 = __builtin_bit_cast(bf16x8, a1);
    const bf16x8 B0 = __builtin_bit_cast(bf16x8, b0), B1 = __builtin_bit_cast(bf16x8, b1);
    for (int i = 0; i < iters; ++i) {
#pragma unroll
      for (int j = 0; j < kChains; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16((j & 1) ? A1 : A0, (j & 2) ? B1 : B0, acc[j], 0, 0, 0);
#pragma unroll
      for (int j = 0; j < kChains; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16((j & 1) ? A0 : A1, (j & 2) ? B0 : B1, acc[j], 0, 0, 0);
    }
  } else {
    uint32_t a0[4], a1[4], b0[8], b1[8];
    fill(a0, tid * 4 + 0);
    fill(a1, tid * 4 + 1);
    fill(b0, tid * 4 + 2);
    fill(b1, tid * 4 + 3);
    const bf16x8 A0 = __builtin_bit_cast(bf16x8, a0), A1 = __builtin_bit_cast(bf16x8, a1);
    const bf16x16 B0 = __builtin_bit_cast(bf16x16, b0), B1 = __builtin_bit_cast(bf16x16, b1);
    // sparsity indices, two bits per compressed element, element 0 lowest:
    // in each group of four k positions the first element picks 0 or 1 and
    // the second 2 or 3 (the pattern of the Quest scoring), varying by lane
    const int idx0 = (int)((mix(tid) & 0x5555u) | 0x8888u), idx1 = (int)((mix(tid + 7u) & 0x5555u) | 0x8888u);
    for (int i = 0; i < iters; ++i) {
#pragma unroll
      for (int j = 0; j < kChains; ++j)
        acc[j] = __builtin_amdgcn_smfmac_f32_16x16x64_bf16((j & 1) ? A1 : A0, (j & 2) ? B1 : B0, acc[j],
                                                           (j & 1) ? idx1 : idx0, 0, 0);
#pragma unroll
      for (int j = 0; j < kChains; ++j)
        acc[j] = __builtin_amdgcn_smfmac_f32_16x16x64_bf16((j & 1) ? A0 : A1, (j & 2) ? B0 : B1, acc[j],
                                                           (j & 1) ? idx0 : idx1, 0, 0);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kChains; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
  out[tid] = s;
}

// Fill rate of 16 KiB tiles from a source region into LDS by direct loads
// (global_load_lds_dwordx4), the attention kernel's staging path: each
// workgroup of 128 threads (two waves, as the attention units) streams
// tiles chosen by a per-workgroup random sequence over the region, each
// wave issuing eight 1 KiB loads per tile, with up to two tiles in flight
// (two 16 KiB LDS slots, so four workgroups fit a CU as the attention's
// units do).  One lane of workgroup 0 records the shader-clock and
// constant-clock counters over its run, from which the host derives the
// clock.  Every load stays inside tile (h mod n_tiles) of the region.
__device__ __forceinline__ void fill_dma16(const uint16_t* base, uint32_t voff, uint32_t lds_byte_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds_byte_addr)
               : "memory");
}

template <int DEPTH>
__global__ void __launch_bounds__(128) fill_loop(const uint16_t* src, uint32_t n_tiles, int iters,
                                                 unsigned long long* clk, float* out) {
  __shared__ __align__(16) uint16_t s_buf[2 * 8192];   // two 16 KiB tiles
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t lds0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)s_buf;
  unsigned long long t0 = 0, r0 = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    t0 = __builtin_amdgcn_s_memtime();
    r0 = __builtin_amdgcn_s_memrealtime();
  }
  uint32_t h = blockIdx.x * 2654435761u;
  for (int i = 0; i < iters; ++i) {
    h = h * 1664525u + 1013904223u;
    const uint16_t* base = src + (size_t)(h % n_tiles) * 8192 + (size_t)w * 4096;   // this wave's 8 KiB
    const uint32_t slot = lds0 + (uint32_t)((i % 2) * 16384 + w * 8192);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      fill_dma16(base + j * 512, (uint32_t)(lane * 16), __builtin_amdgcn_readfirstlane(slot + j * 1024));
    // at most DEPTH - 1 tiles of this wave still in flight (loads complete in issue order)
    __builtin_amdgcn_s_waitcnt(DEPTH == 1 ? 0x0f70 : 0x0f78);
  }
  __builtin_amdgcn_s_waitcnt(0x0f70);
  __syncthreads();
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    clk[0] = __builtin_amdgcn_s_memtime() - t0;
    clk[1] = __builtin_amdgcn_s_memrealtime() - r0;
  }
  out[blockIdx.x * 128 + threadIdx.x] = (float)s_buf[threadIdx.x];
}

}  // namespace

extern "C" {

int ugbs_probe_fill(int depth, const void* src, unsigned n_tiles, int n_workgroups, int iters,
                    unsigned long long* clk, float* out, void* stream) {
  if ((depth != 1 && depth != 2) || !src || !clk || !out || n_tiles < 1 || n_workgroups < 1 || iters < 1)
    return 1;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const uint16_t* p = static_cast<const uint16_t*>(src);
  if (depth == 1)
    fill_loop<1><<<n_workgroups, 128, 0, s>>>(p, n_tiles, iters, clk, out);
  else
    fill_loop<2><<<n_workgroups, 128, 0, s>>>(p, n_tiles, iters, clk, out);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

int ugbs_probe_mfma(int kind, int n_workgroups, int iters, float* out, void* stream) {
  if (n_workgroups < 1 || iters < 1 || !out || (kind != UGBS_PROBE_MFMA_BF16 && kind != UGBS_PROBE_SMFMAC_BF16))
    return 1;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (kind == UGBS_PROBE_MFMA_BF16)
    mfma_loop<false><<<n_workgroups, kThreads, 0, s>>>(out, iters);
  else
    mfma_loop<true><<<n_workgroups, kThreads, 0, s>>>(out, iters);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

double ugbs_probe_flop(int kind, int n_workgroups, int iters) {
  // dense-equivalent FLOP per instruction: 16 x 16 x K x 2 (K = 32 dense, 64 for the 2:4-sparse form)
  const double per = (kind == UGBS_PROBE_SMFMAC_BF16 ? 64.0 : 32.0) * 16.0 * 16.0 * 2.0;
  return per * 2.0 * kChains * (double)iters * (double)n_workgroups * (kThreads / 64);
}

int ugbs_probe_out_floats(int n_workgroups) { return n_workgroups * kThreads; }

}  // extern "C"
