// Per-row selection scattered into a per-tile block bitmap: the variant the
// Limitations of Section 4 name for the per-tile granularity of Section
// 3.2.  Every query row of a tile ranks the candidate blocks C(t) = {1..t-1}
// by its own score (A.2 before the max over rows), keeps the forced blocks
// [0] or [0, t] and its R best candidates, R = (trigger ? rho k : k) - |F|
// (all of C(t) when fewer), and the tile attends to the union over its 64
// rows, handed to the attention kernel as a bitmap of N_B bits.
//
// One workgroup (16 waves) per (b, h, t) unit, kv head by kv head, heaviest
// tile first.  The 64 rows go in four quarters of 16:
//   scores     wave w computes the 16 x 16 score blocks of chunks w, w + 16,
//              ... on bf16 MFMA (the 16 query rows in registers as the A
//              operand, the chunk's metadata rows straight from L2 as the B
//              operand; Quest as the 2:4-sparse contraction of quest_index
//              on v_smfmac) into an LDS array [16 rows x N_B];
//   selection  wave w takes row w: keys, the top-3 pre-filter and the radix
//              threshold of the selection kernel (the survivors staged in
//              the row's own LDS space once its keys are in registers), and
//              an atomic OR of each kept block into the LDS bitmap.
// The bitmap words of blocks 0..t are then stored (the rest zero).
#include "select_common.h"

namespace ugbs {
namespace {

constexpr int kRowWaves = 16;  // four per SIMD, one row each: the selection is latency-bound
constexpr int kQuarter = 16;                 // query rows per pass
constexpr int kRowSlots = UGBS_MAX_BLOCKS_ROWS / 64;
constexpr int kSurvivors = 256;               // pre-filter survivors per row
constexpr int kMinPitch = 2 * kSurvivors;     // floats: a row's LDS region holds its survivors

struct RowParams {
  Shape s;
  const uint16_t* Q;
  const uint16_t* meta;
  const float* row_scores;  // nullptr, or [B, H, N, N_B] fp32 replacing the computed ones
  const uint8_t* trigger;   // [B, T] trigger flags
  uint32_t* bitmap;         // [B, H, T, nw]
  int nw;
  int pitch;                // floats per LDS score row (>= kMinPitch)
};

// The R best keys of one row (positions 0..nc-1 = blocks 1..nc) set in bits.
__device__ __forceinline__ void row_top(const float* row, int nc, int R, int lane_in, uint32_t* bits,
                                        uint64_t* s_surv) {
  // the lane index passes through an opaque move, so the per-slot values
  // derived from it are recomputed per row instead of being hoisted out of
  // the row loop (and spilled: 16 waves leave 128 registers per lane)
  int lane;
  asm volatile("v_mov_b32 %0, %1" : "=v"(lane) : "v"(lane_in));
  const int nslots = (nc + 63) / 64;
  uint32_t keys[kRowSlots];
#pragma unroll
  for (int sl = 0; sl < kRowSlots; ++sl) {
    const int p = 64 * sl + lane;
    keys[sl] = (sl < nslots && p < nc) ? order_key(row[p]) : 0u;
  }
  bool done = false;
  if (R <= 192) {
    uint32_t top3[3] = {0u, 0u, 0u};
#pragma unroll
    for (int sl = 0; sl < kRowSlots; ++sl) {
      if (sl < nslots) {
        const uint32_t x = keys[sl];
        top3[2] = max(top3[2], min(top3[1], x));
        top3[1] = max(top3[1], min(top3[0], x));
        top3[0] = max(top3[0], x);
      }
    }
    bool exact0;
    const uint32_t t0 = kth_largest<3>(top3, 3, R, &exact0);
    constexpr int kSurv = kSurvivors;
    wave_lds_sync();  // the row's keys are in registers: s_surv may reuse its space
    int ns = 0;
#pragma unroll
    for (int sl = 0; sl < kRowSlots; ++sl) {
      if (sl < nslots) {
        const bool tk = t0 > 0u && keys[sl] >= t0;
        const uint64_t mk = __ballot(tk);
        const int at = ns + lanes_below(mk);
        if (tk && at < kSurv) s_surv[at] = ((uint64_t)keys[sl] << 32) | (uint32_t)(64 * sl + lane);
        ns += __popcll(mk);
      }
    }
    if (t0 > 0u && ns <= kSurv) {
      wave_lds_sync();
      uint32_t k2[kSurv / 64], p2[kSurv / 64];
#pragma unroll
      for (int sl = 0; sl < kSurv / 64; ++sl) {
        const int i = 64 * sl + lane;
        const uint64_t v = (i < ns) ? s_surv[i] : 0ull;
        k2[sl] = (uint32_t)(v >> 32);
        p2[sl] = (uint32_t)v;
      }
      wave_lds_sync();  // the survivors are read before the next row reuses s_surv
      select_top_each<kSurv / 64>(k2, (ns + 63) / 64, R, lane, [&](int sl) {
        const int blk = 1 + (int)p2[sl];
        atomicOr(&bits[blk >> 5], 1u << (blk & 31));
      });
      done = true;
    }
  }
  if (!done)
    select_top_each<kRowSlots>(keys, nslots, R, lane, [&](int sl) {
      const int blk = 1 + 64 * sl + lane;
      atomicOr(&bits[blk >> 5], 1u << (blk & 31));
    });
}

template <int D, bool QUEST>
__global__ void __launch_bounds__(64 * kRowWaves) rowsel_kernel(RowParams P) {
  constexpr int KD = QUEST ? 2 * D : D;        // metadata row length
  constexpr int KS = D / 32;                   // k-steps of 32 channels (raw query rows)
  // [16][pitch]: the quarter's scores; row r's region then holds the
  // survivors of row r (also when the scores come from memory)
  extern __shared__ __align__(16) float s_rows[];
  __shared__ uint32_t s_bits[UGBS_MAX_BLOCKS_ROWS / 32];
  const Shape& s = P.s;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const int n_units = s.B * s.H * s.T;
  const int uid = blockIdx.x;
  if (uid >= n_units) return;
  const Unit u = unit_of(uid, s);
  const int t = u.t;
  const size_t rowid = ((size_t)u.b * s.H + u.h) * s.T + t;
  const int nf = (t == 0) ? 1 : 2;
  const int nc = (t >= 1) ? t - 1 : 0;
  // read for every tile, into a scalar register (no branch around the load)
  const int flag = __builtin_amdgcn_readfirstlane((int)P.trigger[(size_t)u.b * s.T + t]);
  const int R = min((flag != 0 ? s.W : s.k) - nf, nc);
  const int nwords = (t >> 5) + 1;

  for (int i = threadIdx.x; i < P.nw; i += 64 * kRowWaves) s_bits[i] = 0u;
  __syncthreads();
  if (threadIdx.x == 0) {
    atomicOr(&s_bits[0], 1u);
    if (t > 0) atomicOr(&s_bits[t >> 5], 1u << (t & 31));
  }
  if (R >= nc) {  // every candidate is kept by every row
    for (int blk = 1 + threadIdx.x; blk <= nc; blk += 64 * kRowWaves) atomicOr(&s_bits[blk >> 5], 1u << (blk & 31));
  } else {
    const int kvh = u.h / s.G;
    const uint16_t* mhead = P.meta + ((size_t)u.b * s.Hkv + kvh) * s.NB * KD;
    const uint16_t* qtile = P.Q + (((size_t)u.b * s.H + u.h) * s.N + (size_t)t * kBlock) * D;
    const int nchunks = (nc + 15) / 16;
    for (int qr = 0; qr < kBlock / kQuarter; ++qr) {
      const float* rows;     // 16 rows of scores of this quarter, row stride `stride`
      size_t stride;
      if (P.row_scores) {
        rows = P.row_scores + (((size_t)u.b * s.H + u.h) * s.N + (size_t)t * kBlock + kQuarter * qr) * s.NB + 1;
        stride = s.NB;
      } else {
        // ---- scores of rows 16 qr .. 16 qr + 15, chunk by chunk ----------
        bf16x8 a[KS];
        uint32_t qidx[QUEST ? KS : 1];
        const uint16_t* qrow = qtile + (size_t)(kQuarter * qr + c16) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const uint4 v = *reinterpret_cast<const uint4*>(qrow + 32 * ks + 8 * g);
          a[ks] = as_bf16x8(v);
          if constexpr (QUEST) qidx[ks] = quest_index(v);
        }
        // the chunk's metadata rows straight from L2 as the B operand; Quest:
        // per k-step the (kmin, kmax) pairs of channels 32 ks + 4 g .. + 3 and
        // 32 ks + 16 + 4 g .. + 3 (see quest_index)
        constexpr int KB = QUEST ? 2 * KS : KS;
        auto load_b = [&](int c, uint4 (&bv)[KB]) {
          const int p = 16 * c + c16;  // block 1 + p; past the last candidate block 1 is read
          const uint16_t* mrow = mhead + (size_t)(1 + (p < nc ? p : 0)) * KD;
#pragma unroll
          for (int j = 0; j < KB; ++j) {
            const int off = QUEST ? 64 * (j / 2) + 32 * (j % 2) + 8 * g : 32 * j + 8 * g;
            bv[j] = *reinterpret_cast<const uint4*>(mrow + off);
          }
        };
        for (int c = w; c < nchunks; c += kRowWaves) {
          uint4 cur[KB];
          load_b(c, cur);
          const int p = 16 * c + c16;
          f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
          if constexpr (QUEST) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a[ks], as_bf16x16(cur[2 * ks], cur[2 * ks + 1]), acc,
                                                              (int)qidx[ks], 0, 0);
          } else {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks], as_bf16x8(cur[ks]), acc, 0, 0, 0);
          }
          // lane holds rows 4g + i of the quarter, block column c16
          if (p < nc) {
#pragma unroll
            for (int i = 0; i < 4; ++i) s_rows[(4 * g + i) * P.pitch + p] = acc[i];
          }
        }
        __syncthreads();
        rows = s_rows;
        stride = (size_t)P.pitch;
      }
      // ---- selection: wave w takes row w ------------------------------------
      for (int r = w; r < kQuarter; r += kRowWaves)
        row_top(rows + (size_t)r * stride, nc, R, lane, s_bits,
                reinterpret_cast<uint64_t*>(s_rows + (size_t)r * P.pitch));
      __syncthreads();  // s_rows is rewritten by the next quarter
    }
  }
  __syncthreads();
  uint32_t* out = P.bitmap + rowid * P.nw;
  for (int i = threadIdx.x; i < P.nw; i += 64 * kRowWaves) out[i] = (i < nwords) ? s_bits[i] : 0u;
}

template <int D, bool QUEST>
hipError_t launch_rows(RowParams P, hipStream_t stream) {
  const size_t smem = sizeof(float) * (size_t)kQuarter * P.pitch;
  if (smem + sizeof(uint32_t) * (UGBS_MAX_BLOCKS_ROWS / 32) > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)rowsel_kernel<D, QUEST>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
  }
  const int n_units = P.s.B * P.s.H * P.s.T;
  const int grid = ((n_units + 7) / 8) * 8;
  rowsel_kernel<D, QUEST><<<grid, 64 * kRowWaves, smem, stream>>>(P);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_select_rows(const Shape& s, const uint16_t* Q, const uint16_t* meta,
                              const float* row_scores, const uint8_t* trigger, uint32_t* bitmap,
                              hipStream_t stream) {
  RowParams P{};
  P.s = s;
  P.Q = Q;
  P.meta = meta;
  P.row_scores = row_scores;
  P.trigger = trigger;
  P.bitmap = bitmap;
  P.nw = (s.NB + 31) / 32;
  // padded against bank conflicts of the column writes; with scores from
  // memory the rows only hold survivors
  P.pitch = row_scores ? kMinPitch : std::max(((s.NB + 3) & ~3) + 4, kMinPitch);
  const bool quest = s.backbone == UGBS_QUEST;
  if (s.d == 256) return quest ? launch_rows<256, true>(P, stream) : launch_rows<256, false>(P, stream);
  if (s.d == 128) return quest ? launch_rows<128, true>(P, stream) : launch_rows<128, false>(P, stream);
  return quest ? launch_rows<64, true>(P, stream) : launch_rows<64, false>(P, stream);
}

}  // namespace ugbs
