// Per-row selection scattered into a per-tile block bitmap: the variant the
// Limitations of Section 4 name for the per-tile granularity of Section
// 3.2.  Every query row of a tile ranks the candidate blocks C(t) = {1..t-1}
// by its own score (A.2 before the max over rows), keeps the forced blocks
// [0] or [0, t] and its R best candidates, R = (trigger ? rho k : k) - |F|
// (all of C(t) when fewer), and the tile attends to the union over its 64
// rows, handed to the attention kernel as a bitmap of N_B bits.
//
// One workgroup (16 waves) per (b, h, t) unit, kv head by kv head, heaviest
// tile first.  Two forms:
//
// Two passes over the scores (R <= kTwoPassMaxR).  The candidates stream
// through an LDS ring in super-chunks of 64 consecutive blocks (1 KiB
// direct-to-LDS loads shared by the workgroup); wave w computes row tile
// w mod 4 (its 16 query rows in registers as the A operand) against column
// tile w / 4 of every super-chunk on bf16 MFMA (Quest as the 2:4-sparse
// contraction of quest_index on v_smfmac), so a lane sees, for 4 rows, the
// candidates p = 64 m + j of one stream j (64 streams per row).
//   pass 1   every lane keeps the 4 largest scores of each of its (row,
//            stream) pairs.  Any R of these 256 values per row are R
//            distinct scores of the row, so their R-th largest is a lower
//            bound L on the row's R-th largest score.
//   pass 2   the same contraction again (same instructions, same values);
//            the scores >= L go to the row's list in LDS with their
//            positions (1.00 R - 1.02 R of them on the synthetic workloads).
//   pass 3   wave w takes rows 4 w .. 4 w + 3 together: a list of exactly R
//            is kept whole; otherwise the exact R-th largest key by a radix
//            descent from the list's common key prefix, ties at it by a
//            radix over positions (lowest first).  Kept blocks are ORed
//            into the LDS bitmap.
//   Nothing of size N_B per row is stored; the metadata is read twice.  A
//   list longer than kCap (many equal scores) sends its row to the quarter
//   form below.
//
// Quarters (R > kTwoPassMaxR, and rows whose lists overflowed): the 64 rows
// in four passes of 16; the waves compute the 16 x 16 score blocks of
// interleaved chunks into an LDS array [16 rows x N_B], then wave w selects
// row w with the keys, top-3 pre-filter and radix threshold of the
// selection kernel.
//
// The bitmap words of blocks 0..t are then stored (the rest zero).
#include "attend_common.h"

namespace ugbs {
namespace {

constexpr int kRowWaves = 16;  // four per SIMD: the selection steps are latency-bound
constexpr int kQuarter = 16;                 // query rows per pass of the quarter form
constexpr int kRowSlots = UGBS_MAX_BLOCKS_ROWS / 64;
constexpr int kSurvivors = 256;               // pre-filter survivors per row (quarter form)
constexpr int kMinPitch = 2 * kSurvivors;     // floats: a row's LDS region holds its survivors
constexpr int kStreams = 64;                  // two-pass form: column streams per row
constexpr int kTop = 4;                       // largest scores kept per (row, stream)
constexpr int kBoundVals = kStreams * kTop;   // values per row the lower bound is taken over
constexpr int kCap = 176;                     // two-pass form: list entries per row
constexpr int kTwoPassMaxR = 128;             // largest R of the two-pass form
constexpr int kRegionA = 65536;               // metadata ring, then the per-row stream values

static_assert(kTwoPassMaxR < kBoundVals, "more bound values than kept candidates");
static_assert(sizeof(uint32_t) * kBlock * kBoundVals <= kRegionA, "stream values fit the ring's space");
static_assert(kRowWaves == 16 && kStreams == 64, "16 waves: four row tiles x four 16-column tiles");

// Two-pass metadata super-chunk: 64 consecutive candidate blocks, fetched
// into LDS by the workgroup with 1 KiB direct loads, rows as 16-byte columns
// XOR-swizzled by row (conflict-free B reads); two ring slots where they fit
// in kRegionA (one at d = 256 Quest, 64 KiB per super-chunk).
template <int D, bool QUEST>
struct RowChunk {
  static constexpr int kBlocks = 64;
  static constexpr int KD = QUEST ? 2 * D : D;
  static constexpr int CPR = KD / 8;
  static constexpr int SWZ = (CPR < 16 ? CPR : 16) - 1;
  static constexpr int kBytes = kBlocks * KD * 2;
  static constexpr int kLoads = kBytes / 1024;
  static constexpr int kRing = 2 * kBytes <= kRegionA ? 2 : 1;
  static constexpr int kPerWave = (kLoads + kRowWaves - 1) / kRowWaves;
  static_assert(kRing * kBytes <= kRegionA, "ring fits its region");
  __device__ static __forceinline__ int off(int r, int c) { return (r * CPR + (c ^ (r & SWZ))) * 16; }
};
constexpr size_t kTwoPassBytes = kRegionA + sizeof(uint64_t) * kBlock * kCap;

struct RowParams {
  Shape s;
  const uint16_t* Q;
  const uint16_t* meta;
  const float* row_scores;  // nullptr, or [B, H, N, N_B] fp32 replacing the computed ones
  const uint8_t* trigger;   // [B, T] trigger flags
  uint32_t* bitmap;         // [B, H, T, nw]
  int nw;
  int pitch;                // floats per LDS score row of the quarter form (>= kMinPitch)
};

// Wave-wide maximum / minimum of 32-bit keys (xor butterfly through the LDS
// crossbar), uniform across the wave.
__device__ __forceinline__ uint32_t wave_max_key(uint32_t x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = max(x, (uint32_t)__shfl_xor((int)x, m));
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)x);
}

__device__ __forceinline__ uint32_t wave_min_key(uint32_t x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = min(x, (uint32_t)__shfl_xor((int)x, m));
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)x);
}

// Common prefix of the keys in [lo, hi]: the bits above the highest bit in
// which lo and hi differ, and that bit (-1 when lo == hi).
__device__ __forceinline__ uint32_t key_prefix(uint32_t lo, uint32_t hi, int* top) {
  if (lo == hi) {
    *top = -1;
    return hi;
  }
  const int sb = 31 - __builtin_clz(lo ^ hi);
  *top = sb;
  return sb == 31 ? 0u : hi & ~((2u << sb) - 1u);
}

// Radix descent of M rows at once (independent chains, interleaved): for
// every row j in the mask open, the largest thr[j] with at least R of
// key[j][..] >= thr[j], resolved from bit top down.  thr[j] enters holding
// the row's common key prefix; a bit inside a row's prefix leaves its thr
// unchanged (every key has it, or none), so all rows descend from the
// highest top.  A row leaves the descent once exactly R keys are >= its
// candidate: that candidate is then the answer (fewer steps than bits on
// distinct scores).  Empty entries hold key 0 and never count (every
// candidate is >= 1).
template <int M, int S>
__device__ __forceinline__ void descend(const uint32_t (&key)[M][S], uint32_t (&thr)[M], int R, int top,
                                        uint32_t open) {
  for (int bit = top; bit >= 0 && open != 0u; --bit) {
#pragma unroll
    for (int j = 0; j < M; ++j) {
      if ((open >> j) & 1u) {
        const uint32_t cand = thr[j] | (1u << bit);
        int cnt = 0;
#pragma unroll
        for (int sl = 0; sl < S; ++sl) cnt += (int)__popcll(__ballot(key[j][sl] >= cand));
        if (cnt >= R) {
          thr[j] = cand;
          if (cnt == R) open &= ~(1u << j);
        }
      }
    }
  }
}

// The score at or above which a score's key is >= the bound key L (keys of
// finite scores are >= 0x00800000; a smaller L admits every score).
__device__ __forceinline__ float bound_value(uint32_t L) {
  return L < 0x00800000u ? -__builtin_inff() : key_value(L);
}

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

// Quarter form for the rows set in rowmask (bit r = row r of the tile).
template <int D, bool QUEST, bool GIVEN>
__device__ void quarter_rows(const RowParams& P, float* s_rows, uint32_t* s_bits, const uint16_t* mhead,
                             const uint16_t* qtile, size_t rowbase, int nc, int R, uint64_t rowmask, int w,
                             int lane) {
  constexpr int KD = QUEST ? 2 * D : D;  // metadata row length
  constexpr int KS = D / 32;             // k-steps of 32 channels (raw query rows)
  const int g = lane >> 4, c16 = lane & 15;
  const int nchunks = (nc + 15) / 16;
  for (int qr = 0; qr < kBlock / kQuarter; ++qr) {
    const uint32_t qmask = (uint32_t)(rowmask >> (kQuarter * qr)) & 0xffffu;
    if (qmask == 0u) continue;
    const float* rows;  // 16 rows of scores of this quarter, row stride `stride`
    size_t stride;
    if constexpr (GIVEN) {
      rows = P.row_scores + (rowbase + (size_t)kQuarter * qr) * P.s.NB + 1;
      stride = P.s.NB;
    } else {
      // ---- scores of rows 16 qr .. 16 qr + 15, chunk by chunk --------------
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
      for (int c = w; c < nchunks; c += kRowWaves) {
        const int p = 16 * c + c16;  // block 1 + p; past the last candidate block 1 is read
        const uint16_t* mrow = mhead + (size_t)(1 + (p < nc ? p : 0)) * KD;
        uint4 cur[KB];
#pragma unroll
        for (int j = 0; j < KB; ++j)
          cur[j] = *reinterpret_cast<const uint4*>(mrow + (QUEST ? 64 * (j / 2) + 32 * (j % 2) + 8 * g
                                                                 : 32 * j + 8 * g));
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
    // ---- selection: wave w takes row w --------------------------------------
    for (int r = w; r < kQuarter; r += kRowWaves)
      if ((qmask >> r) & 1u)
        row_top(rows + (size_t)r * stride, nc, R, lane, s_bits,
                reinterpret_cast<uint64_t*>(s_rows + (size_t)r * P.pitch));
    __syncthreads();  // s_rows is rewritten by the next quarter
  }
}

// Two-pass form for all 64 rows of the tile; the rows whose lists overflowed
// are left set in the 64-bit mask s_small[128..129] for the quarter form.
template <int D, bool QUEST, bool GIVEN>
__device__ void two_pass_rows(const RowParams& P, unsigned char* s_dyn, uint32_t* s_bits, uint32_t* s_small,
                              const uint16_t* mhead, const uint16_t* qtile, size_t rowbase, int nc, int R,
                              int w, int lane) {
  using C = RowChunk<D, QUEST>;
  constexpr int KS = D / 32;   // k-steps of 32 channels (raw query rows)
  uint32_t* s_max = reinterpret_cast<uint32_t*>(s_dyn);                   // [64][kBoundVals] after pass 1
  uint64_t* s_list = reinterpret_cast<uint64_t*>(s_dyn + kRegionA);       // [64][kCap]
  uint32_t* s_cnt = s_small;            // [64] list lengths
  uint32_t* s_bound = s_small + 64;     // [64] bound keys L
  uint32_t* s_over = s_small + 128;     // [2]  overflowed rows (bit mask)
  float* s_fbound = reinterpret_cast<float*>(s_small + 132);  // [64] bounds as scores
  const int g = lane >> 4, c16 = lane & 15;
  const int rt = w & 3, qd = w >> 2;   // this wave: row tile rt, column tile qd of every super-chunk
  const int nsc = (nc + C::kBlocks - 1) / C::kBlocks;
  const int NB = P.s.NB;

  if (threadIdx.x < kBlock) s_cnt[threadIdx.x] = 0u;

  // ---- A operand: rows 16 rt + c16, raw; Quest adds the 2:4 indices --------
  bf16x8 a[GIVEN ? 1 : KS];
  uint32_t qidx[(QUEST && !GIVEN) ? KS : 1];
  if constexpr (!GIVEN) {
    const uint16_t* qrow = qtile + (size_t)(16 * rt + c16) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint4 v = *reinterpret_cast<const uint4*>(qrow + 32 * ks + 8 * g);
      a[ks] = as_bf16x8(v);
      if constexpr (QUEST) qidx[ks] = quest_index(v);
    }
    wait_vmcnt<0>();  // Q in registers: the loop's vmcnt waits count ring loads only
  }
  const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(lds_addr(s_dyn));
  // this wave's 1 KiB loads of super-chunk sc: i = w, w + 16, ... < kLoads;
  // rows past the last candidate re-read the super-chunk's first row (block
  // 1 + 64 sc <= nc for every super-chunk issued)
  auto issue = [&](int sc) {
    const uint32_t slot = ring_lds + (uint32_t)((sc % C::kRing) * C::kBytes);
    const uint16_t* base = mhead + (size_t)__builtin_amdgcn_readfirstlane(1 + C::kBlocks * sc) * C::KD;
#pragma unroll
    for (int j = 0; j < C::kPerWave; ++j) {
      const int i = w + kRowWaves * j;
      if (i < C::kLoads) {
        const int p16 = i * 64 + lane;  // 16-byte unit of the slot
        const int r = p16 / C::CPR;
        const int col = (p16 % C::CPR) ^ (r & C::SWZ);
        const int rr = (C::kBlocks * sc + r < nc) ? r : 0;
        dma16(base, (uint32_t)((rr * C::KD + col * 8) * 2), __builtin_amdgcn_readfirstlane(slot + i * 1024));
      }
    }
  };
  // scores of super-chunk sc for this wave: rows 16 rt + 4 g + i, column
  // 16 qd + c16 (candidate p = 64 sc + 16 qd + c16, block 1 + p)
  auto scores = [&](int sc, f32x4& acc) {
    const int p = C::kBlocks * sc + 16 * qd + c16;
    if constexpr (GIVEN) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        acc[i] = p < nc ? P.row_scores[(rowbase + 16 * rt + 4 * g + i) * NB + 1 + p] : 0.f;
    } else {
      const unsigned char* slot = s_dyn + (sc % C::kRing) * C::kBytes;
      const int br = 16 * qd + c16;
      // every B operand of the step read before the first MFMA: one LDS
      // round trip per step, not one per k-step (the steps are short and
      // barrier-separated, so their latency is not hidden by other waves)
      // (in groups of at most 8 operands, 32 registers)
      constexpr int NBV = QUEST ? 2 * KS : KS;
      constexpr int GRP = NBV < 8 ? NBV : 8;
      constexpr int KG = QUEST ? GRP / 2 : GRP;   // k-steps per group
      acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k0 = 0; k0 < KS; k0 += KG) {
        uint4 bv[GRP];
#pragma unroll
        for (int j = 0; j < GRP; ++j) {
          const int c = QUEST ? 8 * (k0 + j / 2) + 4 * (j % 2) + g : 4 * (k0 + j) + g;
          bv[j] = *reinterpret_cast<const uint4*>(slot + C::off(br, c));
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < KG; ++kk) {
          const int ks = k0 + kk;
          if constexpr (QUEST)
            acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a[ks], as_bf16x16(bv[2 * kk], bv[2 * kk + 1]), acc,
                                                            (int)qidx[ks], 0, 0);
          else
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks], as_bf16x8(bv[kk]), acc, 0, 0, 0);
        }
      }
    }
  };
  // one pass over the super-chunks: body(sc, acc, in)
  auto sweep = [&](auto&& body) {
    if constexpr (GIVEN) {
      for (int sc = 0; sc < nsc; ++sc) {
        f32x4 acc;
        scores(sc, acc);
        body(acc, C::kBlocks * sc + 16 * qd + c16 < nc, C::kBlocks * sc + 16 * qd + c16);
      }
    } else if constexpr (C::kRing == 2) {
      issue(0);
      for (int sc = 0; sc < nsc; ++sc) {
        wait_vmcnt<0>();  // this wave's loads of sc landed
        lds_barrier();    // everyone's did; everyone is done reading sc - 1's slot
        if (sc + 1 < nsc) issue(sc + 1);
        f32x4 acc;
        scores(sc, acc);
        body(acc, C::kBlocks * sc + 16 * qd + c16 < nc, C::kBlocks * sc + 16 * qd + c16);
      }
    } else {
      for (int sc = 0; sc < nsc; ++sc) {
        issue(sc);
        wait_vmcnt<0>();
        lds_barrier();
        f32x4 acc;
        scores(sc, acc);
        body(acc, C::kBlocks * sc + 16 * qd + c16 < nc, C::kBlocks * sc + 16 * qd + c16);
        wait_lgkm0();
        lds_barrier();    // the slot is free for the next issue
      }
    }
    wait_lgkm0();
    __syncthreads();      // the ring's last reads are done: its space is reused
  };

  // ---- pass 1: the four largest scores of every (row, stream) --------------
  {
    float top[4][kTop];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < kTop; ++j) top[i][j] = -__builtin_inff();
    sweep([&](const f32x4& acc, bool in, int) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // insertion into the sorted four (top[0] >= .. >= top[3]), each new
        // entry from the old ones: new top[j] = med3(top[j - 1], top[j], x)
        const float x = in ? acc[i] : -__builtin_inff();
        float nt[kTop];
        nt[0] = __builtin_amdgcn_fmed3f(top[i][0], x, __builtin_inff());
#pragma unroll
        for (int j = 1; j < kTop; ++j) nt[j] = __builtin_amdgcn_fmed3f(top[i][j - 1], top[i][j], x);
#pragma unroll
        for (int j = 0; j < kTop; ++j) top[i][j] = nt[j];
      }
    });
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < kTop; ++j)
        s_max[(16 * rt + 4 * g + i) * kBoundVals + (16 * qd + c16) * kTop + j] =
            top[i][j] == -__builtin_inff() ? 0u : order_key(top[i][j]);
  }
  __syncthreads();

  // ---- bounds: wave w, rows 4 w + j ----------------------------------------
  {
    constexpr int SL = kBoundVals / 64;
    uint32_t key[4][SL], thr[4];
    int top = -1;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t hi = 0u, lo = 0xffffffffu;
#pragma unroll
      for (int sl = 0; sl < SL; ++sl) {
        key[j][sl] = s_max[(4 * w + j) * kBoundVals + 64 * sl + lane];
        hi = max(hi, key[j][sl]);
        lo = min(lo, key[j][sl] == 0u ? 0xffffffffu : key[j][sl]);
      }
      int tj;
      thr[j] = key_prefix(wave_min_key(lo), wave_max_key(hi), &tj);
      top = tj > top ? tj : top;
    }
    descend<4, SL>(key, thr, R, top, 0xfu);
    if (lane == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        s_bound[4 * w + j] = thr[j];
        s_fbound[4 * w + j] = bound_value(thr[j]);
      }
    }
  }
  __syncthreads();  // the stream values are read: the ring takes their space again

  // ---- pass 2: lists of the scores >= L ------------------------------------
  {
    const float4 fb = *reinterpret_cast<const float4*>(s_fbound + 16 * rt + 4 * g);
    const float fl[4] = {fb.x, fb.y, fb.z, fb.w};
    sweep([&](const f32x4& acc, bool in, int p) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (in && acc[i] >= fl[i]) {
          const int r = 16 * rt + 4 * g + i;
          const uint32_t at = atomicAdd(&s_cnt[r], 1u);
          if (at < (uint32_t)kCap) s_list[r * kCap + at] = ((uint64_t)order_key(acc[i]) << 32) | (uint32_t)p;
        }
      }
    });
  }

  // ---- pass 3: exact top R of each list ------------------------------------
  {
    constexpr int SL = (kCap + 63) / 64;
    uint32_t key[4][SL], pos[4][SL], thr[4];
    int n[4];
    int top = -1;
    uint32_t open = 0u;   // rows whose lists need the descent
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = 4 * w + j;
      n[j] = __builtin_amdgcn_readfirstlane((int)s_cnt[r]);
      // a list shorter than R cannot happen (pass 2 recomputes pass 1's
      // scores exactly); it is sent to the quarter form like an overflow
      const bool ok = n[j] >= R && n[j] <= kCap;
      uint32_t hi = 0u, lo = 0xffffffffu;
#pragma unroll
      for (int sl = 0; sl < SL; ++sl) {
        const int e = 64 * sl + lane;
        const uint64_t v = (ok && e < n[j]) ? s_list[r * kCap + e] : 0ull;
        key[j][sl] = (uint32_t)(v >> 32);
        pos[j][sl] = (uint32_t)v;
        hi = max(hi, key[j][sl]);
        lo = min(lo, key[j][sl] == 0u ? 0xffffffffu : key[j][sl]);
      }
      int tj = -1;
      thr[j] = 0u;
      if (ok && n[j] > R) {  // a list of exactly R is kept whole
        thr[j] = key_prefix(wave_min_key(lo), wave_max_key(hi), &tj);
        open |= 1u << j;
      } else if (!ok && lane == 0) {
        atomicOr(&s_over[r >> 5], 1u << (r & 31));
      }
      n[j] = ok ? n[j] : 0;
      top = tj > top ? tj : top;
    }
    descend<4, SL>(key, thr, R, top, open);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (n[j] == 0) continue;
      uint32_t last = 0xffffffffu;  // keys == thr kept up to this position
      uint32_t t = thr[j];
      if (n[j] == R) {
        t = 0u;  // every entry (keys are >= 1)
      } else {
        int above = 0, eq = 0;
#pragma unroll
        for (int sl = 0; sl < SL; ++sl) {
          above += (int)__popcll(__ballot(key[j][sl] > t));
          eq += (int)__popcll(__ballot(key[j][sl] == t));
        }
        // the keys equal to thr are taken lowest position first: the need-th
        // smallest of their positions (positions < 2048) by a radix descent
        if (above + eq > R) {
          const int need = R - above;
          uint32_t lo = 0u;
          for (int bit = 10; bit >= 0; --bit) {
            int c = 0;
#pragma unroll
            for (int sl = 0; sl < SL; ++sl)
              c += (int)__popcll(__ballot(key[j][sl] == t && pos[j][sl] < lo + (1u << bit)));
            if (c < need) lo += 1u << bit;
          }
          last = lo;
        }
      }
#pragma unroll
      for (int sl = 0; sl < SL; ++sl) {
        const bool take = n[j] == R ? key[j][sl] != 0u
                                    : (key[j][sl] > t || (key[j][sl] == t && pos[j][sl] <= last));
        if (take) {
          const int blk = 1 + (int)pos[j][sl];
          atomicOr(&s_bits[blk >> 5], 1u << (blk & 31));
        }
      }
    }
  }
  __syncthreads();
}

// GIVEN: the scores come from P.row_scores (D and QUEST then unused)
template <int D, bool QUEST, bool GIVEN>
__global__ void __launch_bounds__(64 * kRowWaves) rowsel_kernel(RowParams P) {
  constexpr int KD = QUEST ? 2 * D : D;  // metadata row length
  // quarter form: [16][pitch] scores of a quarter, row r's region then
  // holding the survivors of row r; two-pass form: staged queries and lists
  extern __shared__ __align__(16) unsigned char s_dyn[];
  __shared__ uint32_t s_bits[UGBS_MAX_BLOCKS_ROWS / 32];
  __shared__ __align__(16) uint32_t s_small[196];
  const Shape& s = P.s;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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
  if (threadIdx.x < 2) s_small[128 + threadIdx.x] = 0u;
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
    const size_t rowbase = ((size_t)u.b * s.H + u.h) * s.N + (size_t)t * kBlock;
    uint64_t rest = ~0ull;  // rows for the quarter form
    if (R <= kTwoPassMaxR) {
      two_pass_rows<D, QUEST, GIVEN>(P, s_dyn, s_bits, s_small, mhead, qtile, rowbase, nc, R, w, lane);
      rest = ((uint64_t)s_small[129] << 32) | s_small[128];  // read after the last barrier of the pass
    }
    if (rest != 0ull)
      quarter_rows<D, QUEST, GIVEN>(P, reinterpret_cast<float*>(s_dyn), s_bits, mhead, qtile, rowbase, nc, R, rest, w,
                             lane);
  }
  __syncthreads();
  uint32_t* out = P.bitmap + rowid * P.nw;
  for (int i = threadIdx.x; i < P.nw; i += 64 * kRowWaves) out[i] = (i < nwords) ? s_bits[i] : 0u;
}

template <int D, bool QUEST, bool GIVEN>
hipError_t launch_rows(RowParams P, hipStream_t stream) {
  const size_t smem = std::max(sizeof(float) * (size_t)kQuarter * P.pitch, kTwoPassBytes);
  const size_t fixed = sizeof(uint32_t) * (UGBS_MAX_BLOCKS_ROWS / 32 + 196);
  if (smem + fixed > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)rowsel_kernel<D, QUEST, GIVEN>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
  }
  const int n_units = P.s.B * P.s.H * P.s.T;
  const int grid = ((n_units + 7) / 8) * 8;
  rowsel_kernel<D, QUEST, GIVEN><<<grid, 64 * kRowWaves, smem, stream>>>(P);
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
  if (row_scores) return launch_rows<64, false, true>(P, stream);
  const bool quest = s.backbone == UGBS_QUEST;
  if (s.d == 256) return quest ? launch_rows<256, true, false>(P, stream) : launch_rows<256, false, false>(P, stream);
  if (s.d == 128) return quest ? launch_rows<128, true, false>(P, stream) : launch_rows<128, false, false>(P, stream);
  return quest ? launch_rows<64, true, false>(P, stream) : launch_rows<64, false, false>(P, stream);
}

}  // namespace ugbs
