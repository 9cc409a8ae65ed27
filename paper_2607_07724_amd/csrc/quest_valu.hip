// The Quest tile scores of Eq. (quest-score) on the vector ALU: the literal
// per-channel form, built for comparison with the 2:4-sparse MFMA form of
// the score kernel (same output contract as ugbs_score_select's
// scores_out: [B, H, T, N_B] fp32, -inf outside C(t)).
//
// For channel c the bound term max(q_c kmax_c, q_c kmin_c) equals
// q+_c kmax_c + q-_c kmin_c with q+ = max(q, 0), q- = min(q, 0) (one of the
// two is zero).  The metadata holds (kmin_c, kmax_c) as one 32-bit bf16
// pair, so with the query staged as the pair (q-_c, q+_c) the term is one
// v_dot2c_f32_bf16 (fp32 accumulation; both products are exact in fp32 and
// one of them is zero).  One instruction per (row, block, channel): 64 d
// per (tile, block) pair against 64 d / 32 sparse-MFMA lane-steps.
//
// One workgroup (4 waves) per (b, h, t) unit, heaviest tile first: the
// tile's 64 query rows go to LDS as (q-, q+) pairs; each wave takes groups
// of 64 candidate blocks (one per lane), reads a block's metadata pairs in
// chunks of 16 channels into registers and accumulates all 64 rows
// (broadcast LDS reads of the query pairs), then the maximum over the rows.
#include "ugbs_internal.h"

namespace ugbs {
namespace {

constexpr int kValuWaves = 4;
constexpr int kValuChan = 16;   // metadata channels held in registers at a time

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

template <int D>
__global__ void __launch_bounds__(64 * kValuWaves) __attribute__((amdgpu_waves_per_eu(4))) quest_valu_kernel(Shape s, const uint16_t* Q,
                                                                     const uint32_t* meta, float* out) {
  // (q-, q+) of row r, channel c at r * D + c: low half q- (the bf16 of q
  // when its sign bit is set), high half q+ (otherwise)
  __shared__ __align__(16) uint32_t s_q[kBlock * D];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int uid = blockIdx.x;
  if (uid >= s.B * s.H * s.T) return;
  const Unit u = unit_of(uid, s);
  const int t = u.t;
  const int nc = (t >= 1) ? t - 1 : 0;
  float* row = out + (((size_t)u.b * s.H + u.h) * s.T + t) * s.NB;
  // -inf outside C(t) = {1 .. t - 1}
  for (int j = threadIdx.x; j < s.NB; j += 64 * kValuWaves)
    if (j == 0 || j >= t) row[j] = -__builtin_inff();
  if (nc == 0) return;

  const uint16_t* qtile = Q + (((size_t)u.b * s.H + u.h) * s.N + (size_t)t * kBlock) * D;
  for (int i = threadIdx.x; i < kBlock * D; i += 64 * kValuWaves) {
    const uint32_t q = qtile[i];
    s_q[i] = (q & 0x8000u) ? q : (q << 16);
  }
  __syncthreads();

  const uint32_t* mhead = meta + ((size_t)u.b * s.Hkv + u.h / s.G) * s.NB * D;
  for (int j0 = 64 * w; j0 < nc; j0 += 64 * kValuWaves) {
    const int p = j0 + lane;                       // candidate block 1 + p
    const uint32_t* mrow = mhead + (size_t)(1 + (p < nc ? p : 0)) * D;
    float acc[kBlock];
#pragma unroll
    for (int r = 0; r < kBlock; ++r) acc[r] = 0.f;
#pragma unroll 1
    for (int c0 = 0; c0 < D; c0 += kValuChan) {
      uint32_t kv[kValuChan];
#pragma unroll
      for (int v = 0; v < kValuChan / 4; ++v) {
        const uint4 x = *reinterpret_cast<const uint4*>(mrow + c0 + 4 * v);
        kv[4 * v] = x.x;
        kv[4 * v + 1] = x.y;
        kv[4 * v + 2] = x.z;
        kv[4 * v + 3] = x.w;
      }
#pragma unroll
      for (int r = 0; r < kBlock; ++r) {
#pragma unroll
        for (int v = 0; v < kValuChan / 4; ++v) {
          const uint4 a = *reinterpret_cast<const uint4*>(s_q + r * D + c0 + 4 * v);  // same address: broadcast
          acc[r] = dot2(a.x, kv[4 * v], acc[r]);
          acc[r] = dot2(a.y, kv[4 * v + 1], acc[r]);
          acc[r] = dot2(a.z, kv[4 * v + 2], acc[r]);
          acc[r] = dot2(a.w, kv[4 * v + 3], acc[r]);
        }
      }
    }
    float mx = acc[0];
#pragma unroll
    for (int r = 1; r < kBlock; ++r) mx = fmaxf(mx, acc[r]);
    if (p < nc) row[1 + p] = mx;
  }
}

template <int D>
hipError_t launch_quest_valu_d(const Shape& s, const uint16_t* Q, const uint16_t* meta, float* out,
                               hipStream_t stream) {
  const int n_units = s.B * s.H * s.T;
  quest_valu_kernel<D><<<n_units, 64 * kValuWaves, 0, stream>>>(s, Q, reinterpret_cast<const uint32_t*>(meta), out);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quest_valu(const Shape& s, const uint16_t* Q, const uint16_t* meta, float* scores_out,
                             hipStream_t stream) {
  if (s.d == 256) return launch_quest_valu_d<256>(s, Q, meta, scores_out, stream);
  if (s.d == 128) return launch_quest_valu_d<128>(s, Q, meta, scores_out, stream);
  return launch_quest_valu_d<64>(s, Q, meta, scores_out, stream);
}

}  // namespace ugbs
