// Helpers shared by the attention kernels: direct-to-LDS staging of K/V
// tiles in a bank-conflict-free swizzled layout, explicit wait counts,
// LDS-only barriers, the cross-row max and bf16 packing.
#pragma once
#include "select_common.h"

namespace ugbs {
namespace {

typedef short v4i16 __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))
#define GLB_AS __attribute__((address_space(1)))

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// two fp32 -> packed bf16 pair (round to nearest even), one v_cvt_pk_bf16_f32
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, bf16x2));
}

// s_waitcnt immediates (gfx9 encoding): vmcnt in bits 3:0 and 15:14,
// expcnt 6:4, lgkmcnt 11:8.  Other counters are left at "no wait".
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | 0x70 | 0xf00);
}
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xc07f); }

// Workgroup barrier for LDS hand-offs only: no memory fence, so in-flight
// direct-to-LDS prefetches are not drained.  Callers wait on the counters
// they need first.  The empty asm keeps the compiler from moving memory
// operations across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
}

// max over the four 16-lane rows holding one query row (lanes l, l^16,
// l^32, l^48) with the gfx950 row-swap permutes (VALU, no LDS round trip):
// permlane32_swap pairs row r with row r^2, permlane16_swap row r with r^1.
__device__ __forceinline__ float rows_max(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

template <int D>
struct TileGeom {
  static constexpr int CPR = D / 8;                 // 16-byte chunks per key row
  static constexpr int kElems = kBlock * D;         // one K or V block
  static constexpr int kLoads = kBlock * CPR / 64;  // direct loads per block (64 chunks each)
  static constexpr int kRowsPerLoad = 64 / CPR;
  // Element offset of 16-byte column c of row r.  K: column c ^ (r mod CPR),
  // so the 16 rows read by one K-operand load hit 16 different columns.
  // V: column c ^ (2r mod CPR), so the 4-row x 2-column patches read by the
  // transposing loads of one 16-lane group hit 8 different columns.
  __device__ static __forceinline__ int swz(int r, bool v) { return (v ? 2 * r : r) & (CPR - 1); }
  __device__ static __forceinline__ int off(int r, int c, bool v) { return (r * CPR + (c ^ swz(r, v))) * 8; }
};

// One direct-to-LDS 16-byte load per lane from base + voff (base is
// wave-uniform, in SGPRs); M0 holds the wave-uniform LDS destination and
// lane l's 16 bytes land at M0 + 16 l.  Issued from inline asm so the
// compiler's wait-count insertion does not drain it before unrelated LDS
// reads; the kernel waits on vmcnt explicitly (no other vector memory
// operation is in flight while these are).
__device__ __forceinline__ void dma16(const uint16_t* base, uint32_t voff, uint32_t lds_byte_addr) {
  // M0 is written here and read by nothing else in these kernels (no
  // indirect register moves, no GWS, no LDS parameter loads).
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds_byte_addr)
               : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const LDS_AS void*)p;
}

// Direct-load plan of one K or V tile.  Load `inst` (0..kLoads-1) moves key
// rows inst*R .. inst*R+R-1 (R = kRowsPerLoad) into LDS bytes inst*1024 ..
// +1023, lane l writing LDS chunk inst*64+l, which holds global chunk
// (l mod CPR) ^ swizzle(row).  The swizzle depends on the load index only
// through inst mod M, so each lane keeps the byte offsets (row within the
// load and column) of its wave's first min(M, loads per wave) loads, and
// the rows of the load are added to the wave-uniform base.
template <int D, bool V, int NWV>
struct FetchPlanT {
  using L = TileGeom<D>;
  static constexpr int kLoadsPerWave = L::kLoads / NWV;   // the tile's loads split over NWV waves
  static constexpr int M = V ? (L::CPR > 2 * L::kRowsPerLoad ? L::CPR / (2 * L::kRowsPerLoad) : 1)
                             : (L::CPR > L::kRowsPerLoad ? L::CPR / L::kRowsPerLoad : 1);
  static constexpr int MW = M < kLoadsPerWave ? M : kLoadsPerWave;
  // either the wave's loads wrap around the M offsets whole, or there are
  // at most M of them
  static_assert(kLoadsPerWave % M == 0 || kLoadsPerWave <= M, "load plan");
  uint32_t voff[MW];
  __device__ __forceinline__ void init(int lane, int w) {
#pragma unroll
    for (int m = 0; m < MW; ++m) {
      const int inst = w * kLoadsPerWave + m;
      const int r = inst * L::kRowsPerLoad + lane / L::CPR;
      const int c = (lane % L::CPR) ^ L::swz(r, V);
      voff[m] = (uint32_t)(((lane / L::CPR) * D + c * 8) * 2);
    }
  }
  __device__ __forceinline__ void fetch(const uint16_t* src_blk, uint32_t tile_lds, int w) const {
#pragma unroll
    for (int i = 0; i < kLoadsPerWave; ++i) {
      const int inst = w * kLoadsPerWave + i;
      dma16(src_blk + (size_t)inst * L::kRowsPerLoad * D, voff[i % MW], tile_lds + (uint32_t)(inst * 64 * 16));
    }
  }
};

}  // namespace
}  // namespace ugbs
