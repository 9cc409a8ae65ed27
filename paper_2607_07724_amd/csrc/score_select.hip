// Stages 2+3: tile scores, forcing, sorted top-2k and the cutoff margin
// (A.2-A.6; Eqs. (tile-score), (sigma-def)).  Two kernels on one stream.
//
// score_kernel: one workgroup per 4 consecutive (Q-tile, query head) units
// of one (batch, kv head), sibling heads of one tile or of two adjacent
// tiles (see Group); each wave owns one unit (64 rows of its tile).
// Scoring is a contraction on the matrix cores:
//   S[64 rows x 16 blocks] = Q[64 x d] * M[d x 16 blocks]
// K-mean: M = kbar, dense bf16 MFMA (v_mfma_f32_16x16x32_bf16).  Quest: the
// bound of Eq. (quest-score), sum_c q_c (q_c > 0 ? kmax_c : kmin_c), as a
// 2:4-sparse contraction (v_smfmac_f32_16x16x64_bf16, twice the dense rate):
// the uncompressed operand interleaves (kmin_c, kmax_c), which is how the
// metadata rows are stored, the raw query values are the compressed operand
// and their signs the sparsity indices (quest_index).  Every product is an
// exact bf16 x bf16 product; sums are fp32.  The wave's 64 raw query rows
// stay in registers as the A operand (with the indices for Quest).  Metadata
// rows (the B operand) come in chunks of 16 or 32 blocks that the workgroup's
// waves fetch together with direct-to-LDS loads into a ring of 3 or 4 slots
// (two or three chunks in flight), so each chunk crosses L2 once per
// workgroup; in LDS the 16-byte column c of row r sits at c ^ (r mod 16),
// which makes the operand reads bank-conflict free.  Occupancy decides the
// speed: Quest d 128 and K-mean d 128 launch the same body through entries
// held to fewer registers (three and five waves per SIMD, see
// score_kernel_q128 / score_kernel_k128).  Where registers allow (Quest d <=
// 128, K-mean d 256) a column tile's B operands are all read before its
// first matrix instruction, so each column tile waits on the LDS once, and
// the next column tile's reads go out before this tile's max and store.  The max over the tile's rows (A.3) is
// the max over a lane's 16 accumulators and then across the four 16-lane
// groups; each chunk's 16 tile scores go straight to memory, into the
// caller's [.., N_B] score tensor or into packed rows of the workspace (row
// (b, h, t) holds the t-1 candidates 1..t-1).
//
// select_kernel: one wave per unit, heaviest tile first.  Tile scores
// become order-preserving 32-bit keys (-0 folded into +0).  A per-lane
// top-3 pre-filter bounds the R-th largest key from below (R = min(max(W -
// |F|, m + 1), |C|): the listed candidates, and at least the m + 1 that
// sigma needs), the R-th largest key is found among the survivors by a
// most-significant-bit-first radix descent that counts with wave ballots,
// the top R are compacted (equal keys at the threshold by lower block
// index) and ordered by (key, ~index) with a bitonic sort: in registers
// across lanes for R <= 128, in LDS above.  sigma uses IEEE fp32 subtract and
// divide.  The kernel is bound by instruction issue, not by its reads: on
// the 128K layer about 1,620 VALU instructions per unit keep the SIMDs'
// VALU issue ~84% busy.  Splitting the stages keeps each kernel at its own
// occupancy (the scoring kernel is bound by registers, the selection
// kernel by instruction issue).
#include "select_common.h"

namespace ugbs {
namespace {

constexpr int kMaxGroup = 4;    // sibling query heads per workgroup
constexpr int kSelWaves = 4;    // units (waves) per selection workgroup

#define LDS_AS __attribute__((address_space(3)))

struct SelParams {
  Shape s;
  const uint16_t* Q;
  const uint16_t* meta;
  const float* scores_in;
  float* scores_out;
  int32_t* idx_sorted;
  float* sigma;
  float* scratch; // packed candidate scores (workspace), when neither scores_in nor scores_out
  double* rough;  // per-unit row roughness (diagnostics mode of the score kernel)
  int GW;         // waves (query heads) per workgroup of the score kernel
  int n_groups;   // score workgroups per (b, kv head) = ceil(T G / GW)
  int n_wg;       // score-kernel workgroups
  int wave_lds;   // bytes of per-wave LDS of the selection kernel (survivors)
  int ring_lds;   // bytes of the metadata ring
};

// max over the four 16-lane rows (lanes l, l^16, l^32, l^48) with the gfx950
// row-swap permutes: permlane32_swap pairs row r with r^2, permlane16_swap
// row r with r^1 (VALU only, no LDS round trip).
__device__ __forceinline__ float wave_max16(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

constexpr int kSurvivors = 256;   // pre-filter survivors handled in registers

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = min(x, (uint32_t)__shfl_xor((int)x, o));
  return x;
}

// Workgroup barrier without a memory fence (the metadata ring's direct-to-LDS
// fetches stay in flight); callers wait on vmcnt first.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt vmcnt(n) for a wave-uniform runtime n (gfx9 encoding: vmcnt in
// bits 3:0 and 15:14; expcnt and lgkmcnt left at "no wait").  n >= 32 (never
// reached: at most 8 loads x 2 chunks) falls back to a full wait.
template <int N>
__device__ __forceinline__ void wait_vm() {
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | 0x70 | 0xf00);
}
__device__ __forceinline__ void wait_vmcnt_dyn(int n) {
  switch (n) {
#define W_(N) case N: wait_vm<N>(); break;
    W_(0) W_(1) W_(2) W_(3) W_(4) W_(5) W_(6) W_(7) W_(8) W_(9) W_(10) W_(11) W_(12) W_(13)
    W_(14) W_(15) W_(16) W_(17) W_(18) W_(19) W_(20) W_(21) W_(22) W_(23) W_(24) W_(25)
    W_(26) W_(27) W_(28) W_(29) W_(30) W_(31)
#undef W_
    default: wait_vm<0>(); break;
  }
}

// Direct-to-LDS 16-byte load per lane (see attend.hip): M0 = LDS
// destination of lane 0, lane l lands at M0 + 16 l.  Hidden from the
// compiler's wait-count insertion; waited on explicitly.
__device__ __forceinline__ void dma16(const uint16_t* base, uint32_t voff, uint32_t lds_byte_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds_byte_addr)
               : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const LDS_AS void*)p;
}

// Blocks per metadata chunk: 32 (two 16-block MFMA column tiles per
// barrier) for Quest d 128 and K-mean d 256, 16 elsewhere, where the second
// accumulator set would cost a wave (measured: 4-7% faster, 3-4% slower
// respectively).  Ring slots (slots - 1 chunks in flight): 3 for Quest d 128
// (48 KiB, three workgroups per CU, see score_kernel_q128), 4 elsewhere.
template <int D, bool QUEST>
struct MetaChunk {
  static constexpr int kBlocks = ((QUEST && D == 128) || (!QUEST && D == 256)) ? 32 : 16;
  static constexpr int kRingSlots = (QUEST && D == 128) ? 3 : 4;
  static constexpr int KD = QUEST ? 2 * D : D;
  static constexpr int CPR = KD / 8;                   // 16-byte columns per metadata row
  static constexpr int SWZ = (CPR < 16 ? CPR : 16) - 1;
  static constexpr int kBytes = kBlocks * KD * 2;
  static constexpr int kLoads = kBytes / 1024;         // 1 KiB direct loads per chunk
  __device__ static __forceinline__ int off(int r, int c) { return (r * CPR + (c ^ (r & SWZ))) * 16; }
};

// Workgroup ordering (ids dealt round-robin to the XCDs, see Unit): (b, kv
// head) outermost; within it the units (tile, query head) in the order
// heaviest tile first, sibling heads adjacent, taken GW at a time.  With G
// a multiple of GW a workgroup holds sibling heads of one tile; otherwise
// (G = 7: 4 + 3) a workgroup may hold the last heads of tile t and the
// first of tile t - 1, whose candidate ranges differ by one block, so the
// metadata chunks are still shared and no wave idles.
struct Group {
  int b, kvh, u0;   // u0: the first unit (tile rank * G + head) of the workgroup
};

__device__ __forceinline__ Group group_of(int id, const SelParams& P) {
  Group r;
  r.u0 = (id % P.n_groups) * P.GW;
  const int rest = id / P.n_groups;
  r.kvh = rest % P.s.Hkv;
  r.b = rest / P.s.Hkv;
  return r;
}

// What the score kernel produces per unit: the tile-score row (full
// [.., N_B] layout or a packed workspace row), or, for the noise-scale
// diagnostic of Appendix D, the sum over candidates and adjacent row pairs
// of the squared row-to-row score difference.
enum Out { kOutFull = 0, kOutPacked = 1, kOutRough = 2 };

// Sum over this lane's column of the squared differences between adjacent
// rows of the 64 x 16 score block.  Lane l holds column l % 16 and rows
// 16 rt + 4 (l / 16) + i in acc[rt][i]; the successor of a lane's last row
// in a row tile sits in the next 16-lane group (or, for the last group, in
// the first group's next row tile).
__device__ __forceinline__ float row_diff_sq(const f32x4 (&acc)[4], int lane) {
  const int g = lane >> 4;
  float nx[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) nx[rt] = __shfl(acc[rt][0], (lane + 16) & 63);
  float sq = 0.f;
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      const float dd = acc[rt][i + 1] - acc[rt][i];
      sq += dd * dd;
    }
    const bool has_next = g < 3 || rt < 3;
    const float nxt = (g < 3) ? nx[rt] : nx[rt < 3 ? rt + 1 : 3];
    const float dd = nxt - acc[rt][3];
    sq += has_next ? dd * dd : 0.f;
  }
  return sq;
}

template <int D, bool QUEST, int OUT>
__device__ __forceinline__ void score_body(const SelParams& P) {
  constexpr bool PACKED = OUT == kOutPacked;
  constexpr bool ROUGH = OUT == kOutRough;
  using MC = MetaChunk<D, QUEST>;
  constexpr int KD = MC::KD;
  constexpr int KS = KD / 32;
  extern __shared__ __align__(16) unsigned char smem[];
  const Shape& s = P.s;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4, c16 = lane & 15;

  const int id = blockIdx.x;
  if (id >= P.n_wg) return;
  const Group gr = group_of(id, P);
  const int x = gr.u0 + w;                            // this wave's unit within the (b, kv head)
  const bool active = x < s.T * s.G;                  // the last workgroup may be partial
  const int xs = active ? x : gr.u0;
  const int h = gr.kvh * s.G + xs % s.G;
  const int t = s.T - 1 - xs / s.G;
  const size_t row = ((size_t)gr.b * s.H + h) * s.T + t;
  const int nc = (t >= 1) ? t - 1 : 0;
  // the workgroup's heaviest tile (wave 0's) sets the candidate range the
  // metadata chunks cover; waves of the next tile use one block less
  const int t_top = s.T - 1 - gr.u0 / s.G;
  const int nc_top = (t_top >= 1) ? t_top - 1 : 0;

  unsigned char* ring = smem;

  // this unit's candidate scores 1..nc: packed rows, or the full [.., N_B] row
  float* dst = PACKED ? P.scratch + packed_row(gr.b * s.H + h, t, s.T)
                      : (ROUGH ? nullptr : P.scores_out + row * s.NB + 1);
  double rough = 0.0;
  if (nc_top > 0) {
    // ---- A operand: this wave's 64 query rows, raw, for both backbones;
    // Quest adds the 2:4 sparsity indices that select kmax or kmin per
    // channel by the sign of q (see quest_index)
    constexpr int KA = D / 32;
    bf16x8 a[4][KA];
    uint32_t qidx[4][QUEST ? KA : 1];
    const uint16_t* qtile = P.Q + (((size_t)gr.b * s.H + h) * s.N + (size_t)t * kBlock) * D;
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      const uint16_t* qrow = qtile + (size_t)(16 * rt + c16) * D;
#pragma unroll
      for (int ks = 0; ks < KA; ++ks) {
        const uint4 v = *reinterpret_cast<const uint4*>(qrow + 32 * ks + 8 * g);
        a[rt][ks] = as_bf16x8(v);
        if constexpr (QUEST) qidx[rt][ks] = quest_index(v);
      }
    }
    __builtin_amdgcn_s_waitcnt(0x70 | 0xf00);  // vmcnt(0): Q is in registers

    // ---- metadata ring: chunk c holds candidate blocks 1 + 16c .. 16c + 16
    const uint16_t* mhead = P.meta + ((size_t)gr.b * s.Hkv + gr.kvh) * s.NB * KD;
    const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(lds_addr(ring));
    const int nchunks = (nc_top + MC::kBlocks - 1) / MC::kBlocks;
    // this wave issues the chunk's 1 KiB loads i = w, w + GW, ...
    const int n_mine = (MC::kLoads - w + P.GW - 1) / P.GW;
    // this wave's share of a chunk: loads i = w, w + GW, ... (at most
    // kMine); the lane offsets within a chunk are the same for every chunk
    // but the last, computed once
    constexpr int kMaxMine = MC::kLoads;
    constexpr int kMine = MC::kLoads >= 4 ? MC::kLoads / 4 : 1;   // loads per wave of four
    auto lane_off = [&](int i, int c, bool last) {
      const int p = i * 64 + lane;                  // 16-byte LDS chunk of the slot
      const int r = p / MC::CPR;                    // block row within the chunk
      const int col = (p % MC::CPR) ^ (r & MC::SWZ);
      // rows past the last candidate re-read the chunk's first row, which
      // is a candidate (1 + kBlocks c <= nc_top for every issued chunk)
      const int rr = (last && 1 + MC::kBlocks * c + r > nc_top) ? 0 : r;
      return (uint32_t)((rr * KD + col * 8) * 2);
    };
    uint32_t off0[kMine];
    const bool fast = P.GW == 4 && (MC::kLoads % 4) == 0;   // loads i = w + 4 j, j < kLoads / 4
#pragma unroll
    for (int j = 0; j < kMine; ++j) off0[j] = lane_off(w + 4 * j, 0, false);
    auto issue = [&](int c) {
      const uint32_t slot = ring_lds + (uint32_t)((c % MC::kRingSlots) * MC::kBytes);
      const uint16_t* base = mhead + (size_t)__builtin_amdgcn_readfirstlane(1 + MC::kBlocks * c) * KD;
      const bool last = MC::kBlocks * (c + 1) >= nc_top;   // workgroup-uniform
      if (fast && !last) {
#pragma unroll
        for (int j = 0; j < kMine; ++j) {
          const int i = w + 4 * j;
          dma16(base, off0[j], __builtin_amdgcn_readfirstlane(slot + i * 1024));
        }
        return;
      }
#pragma unroll 1
      for (int j = 0; j < kMaxMine; ++j) {
        const int i = w + j * P.GW;
        if (i < MC::kLoads) dma16(base, lane_off(i, c, last), __builtin_amdgcn_readfirstlane(slot + i * 1024));
      }
    };
    for (int c = 0; c < MC::kRingSlots - 1 && c < nchunks; ++c) issue(c);

    for (int c = 0; c < nchunks; ++c) {
      const int after = min(MC::kRingSlots - 2, nchunks - 1 - c);  // chunks issued after c
      if (fast) {
        // each wave issues kMine loads per chunk: one uniform branch
        if (after <= 0) wait_vm<0>();
        else if (after == 1) wait_vm<kMine>();
        else wait_vmcnt_dyn(kMine * after);
      } else {
        wait_vmcnt_dyn(n_mine * after);
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave's reads of chunk c-1 are done
      lds_barrier();                                    // chunk c landed; chunk c-1 is free
      if (c + MC::kRingSlots - 1 < nchunks) issue(c + MC::kRingSlots - 1);
      if (active) {
        const unsigned char* slot = ring + (c % MC::kRingSlots) * MC::kBytes;
        constexpr int NCT = MC::kBlocks / 16;            // 16-block column tiles per chunk
        // Read-ahead form (Quest d <= 128, K-mean d 256; elsewhere the
        // registers are not there): all B operands of a column tile are read
        // before its first matrix instruction, so the tile waits on the LDS
        // once, and the next column tile's reads are issued right after this
        // tile's matrix instructions, ahead of its max and store.  Quest: B
        // holds the (kmin, kmax) pairs of channels 4 g .. 4 g + 3 and 16 + 4 g
        // .. 16 + 4 g + 3 of each 32-channel k-step (two 16-byte columns).
        constexpr bool AHEAD = QUEST ? (KA <= 4) : (D == 256);
        constexpr int NRD = QUEST ? 2 * KA : KS;          // 16-byte operand reads per column tile
        uint4 bb[AHEAD ? NRD : 1];
        auto read_b = [&](int ct) {
          const int br = 16 * ct + c16;
#pragma unroll
          for (int j = 0; j < NRD; ++j) {
            const int col = QUEST ? 8 * (j >> 1) + 4 * (j & 1) + g : 4 * j + g;
            bb[j] = *reinterpret_cast<const uint4*>(slot + MC::off(br, col));
          }
        };
        // the roughness mode keeps its registers for the row differences and
        // reads each column tile's operands at the tile's start
        constexpr bool EARLY = AHEAD && !ROUGH;
        if constexpr (AHEAD) {
          read_b(0);
          __builtin_amdgcn_sched_barrier(0);   // keep the reads ahead of the matrix instructions
        }
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
          const int br = 16 * ct + c16;                  // block row of this lane's column
          if constexpr (AHEAD && !EARLY) {
            if (ct > 0) read_b(ct);
            __builtin_amdgcn_sched_barrier(0);
          }
          f32x4 acc[4];
#pragma unroll
          for (int rt = 0; rt < 4; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
          if constexpr (AHEAD) {
#pragma unroll
            for (int ks = 0; ks < KS / (QUEST ? 2 : 1); ++ks) {
              if constexpr (QUEST) {
                const bf16x16 b = as_bf16x16(bb[2 * ks], bb[2 * ks + 1]);
#pragma unroll
                for (int rt = 0; rt < 4; ++rt)
                  acc[rt] = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a[rt][ks], b, acc[rt], (int)qidx[rt][ks], 0, 0);
              } else {
                const bf16x8 b = as_bf16x8(bb[ks]);
#pragma unroll
                for (int rt = 0; rt < 4; ++rt)
                  acc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rt][ks], b, acc[rt], 0, 0, 0);
              }
            }
            if constexpr (EARLY) {
              __builtin_amdgcn_sched_barrier(0);
              if (ct + 1 < NCT) read_b(ct + 1);
              __builtin_amdgcn_sched_barrier(0);
            }
          } else if constexpr (QUEST) {
            // sum over the k-step's 32 channels of q * (q > 0 ? kmax : kmin)
#pragma unroll
            for (int ks = 0; ks < KA; ++ks) {
              const uint4 b0 = *reinterpret_cast<const uint4*>(slot + MC::off(br, 8 * ks + g));
              const uint4 b1 = *reinterpret_cast<const uint4*>(slot + MC::off(br, 8 * ks + 4 + g));
              const bf16x16 b = as_bf16x16(b0, b1);
#pragma unroll
              for (int rt = 0; rt < 4; ++rt)
                acc[rt] = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a[rt][ks], b, acc[rt], (int)qidx[rt][ks], 0, 0);
            }
          } else {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
              const bf16x8 b = as_bf16x8(*reinterpret_cast<const uint4*>(slot + MC::off(br, 4 * ks + g)));
#pragma unroll
              for (int rt = 0; rt < 4; ++rt)
                acc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rt][ks], b, acc[rt], 0, 0, 0);
            }
          }
          const int pos = MC::kBlocks * c + br;
          if constexpr (ROUGH) {
            const float sq = row_diff_sq(acc, lane);
            rough += (pos < nc) ? (double)sq : 0.0;
          } else {
            float mx = acc[0][0];
#pragma unroll
            for (int rt = 0; rt < 4; ++rt)
#pragma unroll
              for (int i = 0; i < 4; ++i) mx = fmaxf(mx, acc[rt][i]);
            mx = wave_max16(mx);
            // straight to memory: a 64-byte store per column tile.  The loop's vmcnt
            // waits still count ring loads correctly: loads complete in issue
            // order, so while a chunk is pending every later ring load is too,
            // and an earlier store in flight can only lengthen a wait
            if (g == 0 && pos < nc) dst[pos] = mx;
          }
        }
      }
    }
  }
  if constexpr (ROUGH) {
    if (active) {
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) rough += __shfl_xor(rough, o);
      if (lane == 0) P.rough[row] = rough;
    }
    return;
  }
  if (!active || PACKED) return;
  // full layout: -inf outside C(t) = {1..t-1}
  float* full = P.scores_out + row * s.NB;
  for (int p = lane; p < s.NB; p += 64)
    if (p == 0 || p > nc) full[p] = -__builtin_huge_valf();
}

template <int D, bool QUEST, int OUT>
__global__ void __launch_bounds__(64 * kMaxGroup) score_kernel(SelParams P) {
  score_body<D, QUEST, OUT>(P);
}

// Quest d 128 tile scores (full or packed rows): the same body held to 168
// registers, so three waves share each SIMD (three workgroups per CU with
// the 3-slot ring) instead of two; the query tile, its sparsity indices and
// one column tile's operands fit without spilling.  Measured at 128K:
// score + select 1.50 -> 1.36 ms (P7 1.28 -> 1.18, C3 0.45 -> 0.41),
// outputs bit-identical.
template <int OUT>
__global__ void __launch_bounds__(64 * kMaxGroup) __attribute__((amdgpu_waves_per_eu(3, 3)))
score_kernel_q128(SelParams P) {
  score_body<128, true, OUT>(P);
}

// K-mean d 128 tile scores: the body held to 96 registers, five waves per
// SIMD instead of four (the 16 KiB ring allows it; a few values spill to
// scratch): score + select 1.09 -> 0.99 ms on the 28/4-head d 128 layer at
// 128K, outputs bit-identical.  (K-mean d 256 held to three waves spills
// 65 registers and runs 1.5x slower; it keeps two.)
template <int OUT>
__global__ void __launch_bounds__(64 * kMaxGroup) __attribute__((amdgpu_waves_per_eu(5, 5)))
score_kernel_k128(SelParams P) {
  score_body<128, false, OUT>(P);
}

// One wave per (b, h, t) unit, heaviest tile first; reads the unit's
// candidate scores (packed rows of the score kernel, or a full [.., N_B] row)
// SLOTS: candidates per lane held in registers (N_B / 64 rounded up to 32 or
// 64: rows of up to 2048 or 4096 blocks).
template <bool PACKED, int SLOTS>
__global__ void __launch_bounds__(64 * kSelWaves) select_kernel(SelParams P) {
  extern __shared__ __align__(16) unsigned char smem[];
  const Shape& s = P.s;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n_units = s.B * s.H * s.T;
  const int n_wg = (n_units + kSelWaves - 1) / kSelWaves;
  const int wg = blockIdx.x;
  if (wg >= n_wg) return;
  const int u = wg * kSelWaves + w;
  if (u >= n_units) return;
  const int h = u % s.H;
  const int rest = u / s.H;
  const int t = s.T - 1 - rest % s.T;
  const int b = rest / s.T;
  const size_t row = ((size_t)b * s.H + h) * s.T + t;
  const int nf = (t == 0) ? 1 : 2;
  const int nc = (t >= 1) ? t - 1 : 0;
  const int m = s.k - nf;
  const int W = s.W;
  // the row lists R_out = min(W - |F|, |C|) candidates; sigma needs the m + 1
  // largest, more than the row holds when rho = 1; without idx_sorted only
  // sigma is wanted
  const int R_out = min(W - nf, nc);
  const int R = P.idx_sorted ? min(max(W - nf, m + 1), nc) : min(m + 1, nc);
  uint64_t* s_sel = reinterpret_cast<uint64_t*>(smem + w * P.wave_lds);
  const float* src = PACKED ? P.scratch + packed_row(b * s.H + h, t, s.T) : P.scores_in + row * s.NB + 1;

  int32_t* out = P.idx_sorted ? P.idx_sorted + row * W : nullptr;
  if (nc == 0) {
    if (out)
      for (int p = lane; p < W; p += 64) out[p] = (p < nf) ? (p == 0 ? 0 : t) : s.NB;
    if (lane == 0) P.sigma[row] = -1.0f;
    return;
  }

  // ---- the R largest keys, compacted into s_sel as (key, ~position) -------
  // Pre-filter: each lane's three largest keys form a subset of the keys, so
  // the R-th largest of those 192 values, T0, is at most the R-th largest
  // key (R <= 192): the R largest are among {key >= T0}, typically R plus a
  // few dozen of up to 2046.  Those survivors, in position order, go
  // through the exact selection; otherwise every candidate does.
  constexpr int kMaxSlots = SLOTS;
  const int nslots = (nc + 63) / 64;
  uint32_t keys[kMaxSlots];
  {
    // every load first (clamped in-row addresses), then the conversions, so
    // the loads are in flight together
    float raw[kMaxSlots];
#pragma unroll
    for (int sl = 0; sl < kMaxSlots; ++sl) {
      const int p = 64 * sl + lane;
      raw[sl] = (sl < nslots) ? src[p < nc ? p : nc - 1] : 0.f;
    }
#pragma unroll
    for (int sl = 0; sl < kMaxSlots; ++sl) {
      const int p = 64 * sl + lane;
      keys[sl] = (sl < nslots && p < nc) ? order_key(raw[sl]) : 0u;  // valid keys are >= 0x007fffff
    }
  }
  bool filtered = false, sort_all = false;
  if (R <= 192 && nc > R) {
    // (slots past the row hold key 0, the smallest: no guard needed here or
    // in the compaction below, where only keys >= t0 > 0 are taken)
    uint32_t top3[3] = {0u, 0u, 0u};
#pragma unroll
    for (int sl = 0; sl < kMaxSlots; ++sl) {
      const uint32_t x = keys[sl];
      top3[2] = max(top3[2], min(top3[1], x));
      top3[1] = max(top3[1], min(top3[0], x));
      top3[0] = max(top3[0], x);
    }
    bool exact0;
    const uint32_t t0 = kth_largest<3>(top3, 3, R, &exact0);
    if (t0 > 0u) {
      int ns = 0;
#pragma unroll
      for (int sl = 0; sl < kMaxSlots; ++sl) {
        const bool take = keys[sl] >= t0;
        const uint64_t mk = __ballot(take);
        const int at = ns + lanes_below(mk);
        if (take && at < kSurvivors)
          s_sel[at] = ((uint64_t)keys[sl] << 32) | (uint32_t)(64 * sl + lane);
        ns += __popcll(mk);
      }
      if (ns <= 128 && R <= 128) {
        // few survivors: the register sort below orders all of them, and
        // the R largest lead (the order (key, ~position) is strict and every
        // key that can be among the R largest survived), so no exact
        // threshold search is needed.  Each lane rewrites its own entries
        // as (key, ~position); unused entries up to 128 become 0.
        wave_lds_sync();
#pragma unroll
        for (int sl = 0; sl < 2; ++sl) {
          const int i = 64 * sl + lane;
          const uint64_t v = (i < ns) ? s_sel[i] : 0ull;
          s_sel[i] = (i < ns) ? ((v & 0xffffffff00000000ull) | (0xffffffffu - (uint32_t)v)) : 0ull;
        }
        sort_all = true;
        filtered = true;
      } else if (ns <= kSurvivors) {
        wave_lds_sync();
        uint32_t k2[kSurvivors / 64], p2[kSurvivors / 64];
#pragma unroll
        for (int sl = 0; sl < kSurvivors / 64; ++sl) {
          const int i = 64 * sl + lane;
          const uint64_t v = (i < ns) ? s_sel[i] : 0ull;
          k2[sl] = (uint32_t)(v >> 32);
          p2[sl] = (uint32_t)v;
        }
        wave_lds_sync();
        select_top<kSurvivors / 64>(k2, p2, (ns + 63) / 64, R, s_sel, lane);
        filtered = true;
      }
    }
  }
  if (!filtered) {
    uint32_t pos[kMaxSlots];
#pragma unroll
    for (int sl = 0; sl < kMaxSlots; ++sl) pos[sl] = (uint32_t)(64 * sl + lane);
    select_top<kMaxSlots>(keys, pos, nslots, R, s_sel, lane);
  }
  if (R <= 128) {
    // ---- bitonic sort of the R winners (2 per lane, slot-major index
    // i = 64 slot + lane; empty entries are 0 and sort last), descending;
    // partners within a slot are exchanged across lanes, across slots in
    // registers
    wave_lds_sync();
    const int n_in = sort_all ? 128 : R;   // entries to order (unused ones are 0)
    uint64_t e[2];
    e[0] = (lane < n_in) ? s_sel[lane] : 0ull;
    e[1] = (64 + lane < n_in) ? s_sel[64 + lane] : 0ull;
#pragma unroll
    for (int size = 2; size <= 128; size <<= 1) {
#pragma unroll
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        if (stride == 64) {
          // i = lane, j = 64 + lane, (i & 128) == 0: descending
          const uint64_t hi = e[0] > e[1] ? e[0] : e[1];
          const uint64_t lo = e[0] > e[1] ? e[1] : e[0];
          e[0] = hi;
          e[1] = lo;
        } else {
          const bool lower = (lane & stride) == 0;
#pragma unroll
          for (int sl = 0; sl < 2; ++sl) {
            const int i = 64 * sl + lane;
            const bool desc = (i & size) == 0;
            const uint32_t plo = (uint32_t)__shfl_xor((int)(uint32_t)e[sl], stride);
            const uint32_t phi = (uint32_t)__shfl_xor((int)(uint32_t)(e[sl] >> 32), stride);
            const uint64_t pv = ((uint64_t)phi << 32) | plo;
            const bool keep_max = (lower == desc);
            const bool take = keep_max ? (pv > e[sl]) : (pv < e[sl]);
            e[sl] = take ? pv : e[sl];
          }
        }
      }
    }
    wave_lds_sync();
    s_sel[lane] = e[0];
    s_sel[64 + lane] = e[1];
    wave_lds_sync();
  } else {
    int n2 = 2;
    while (n2 < R) n2 <<= 1;
    for (int p = R + lane; p < n2; p += 64) s_sel[p] = 0ull;
    wave_lds_sync();
    // ---- bitonic sort, descending -----------------------------------------
    lds_bitonic_desc(s_sel, n2, lane);
  }

  // ---- outputs --------------------------------------------------------------
  for (int p = lane; out && p < W; p += 64) {
    int v;
    if (p < nf)
      v = (p == 0) ? 0 : t;
    else if (p - nf < R_out)
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

template <int D, bool QUEST, int OUT>
hipError_t launch_score(SelParams P, hipStream_t stream) {
  using MC = MetaChunk<D, QUEST>;
  P.ring_lds = MC::kRingSlots * MC::kBytes;
  const size_t smem = (size_t)P.ring_lds;
  if (smem > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)score_kernel<D, QUEST, OUT>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
  }
  const int grid = ((P.n_wg + 7) / 8) * 8;
  if constexpr (D == 128 && QUEST && OUT != kOutRough) {
    static_assert(MetaChunk<D, QUEST>::kRingSlots * MetaChunk<D, QUEST>::kBytes <= 65536, "static LDS limit");
    score_kernel_q128<OUT><<<grid, 64 * P.GW, smem, stream>>>(P);
  } else if constexpr (D == 128 && !QUEST && OUT != kOutRough) {
    score_kernel_k128<OUT><<<grid, 64 * P.GW, smem, stream>>>(P);
  } else {
    score_kernel<D, QUEST, OUT><<<grid, 64 * P.GW, smem, stream>>>(P);
  }
  return hipGetLastError();
}

template <bool PACKED, int SLOTS>
hipError_t launch_select_s(const SelParams& P, hipStream_t stream) {
  const size_t smem = (size_t)kSelWaves * P.wave_lds;
  if (smem > 65536) {  // large budgets (k near N_B): raise the dynamic-LDS limit
    const hipError_t e = hipFuncSetAttribute((const void*)select_kernel<PACKED, SLOTS>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
  }
  const int n_units = P.s.B * P.s.H * P.s.T;
  const int n_wg = (n_units + kSelWaves - 1) / kSelWaves;
  const int grid = ((n_wg + 7) / 8) * 8;
  select_kernel<PACKED, SLOTS><<<grid, 64 * kSelWaves, smem, stream>>>(P);
  return hipGetLastError();
}

template <bool PACKED>
hipError_t launch_select(const SelParams& P, hipStream_t stream) {
  static_assert(UGBS_MAX_BLOCKS <= 64 * 64, "at most 64 slots per lane");
  return P.s.NB <= 32 * 64 ? launch_select_s<PACKED, 32>(P, stream) : launch_select_s<PACKED, 64>(P, stream);
}

template <int OUT>
hipError_t launch_score_d(const SelParams& P, hipStream_t stream) {
  const Shape& s = P.s;
  if (s.d == 256)
    return s.backbone == UGBS_QUEST ? launch_score<256, true, OUT>(P, stream)
                                    : launch_score<256, false, OUT>(P, stream);
  if (s.d == 128)
    return s.backbone == UGBS_QUEST ? launch_score<128, true, OUT>(P, stream)
                                    : launch_score<128, false, OUT>(P, stream);
  return s.backbone == UGBS_QUEST ? launch_score<64, true, OUT>(P, stream)
                                  : launch_score<64, false, OUT>(P, stream);
}

SelParams score_params(const Shape& s, const uint16_t* Q, const uint16_t* meta) {
  SelParams P{};
  P.s = s;
  P.Q = Q;
  P.meta = meta;
  P.GW = s.G < kMaxGroup ? s.G : kMaxGroup;
  P.n_groups = (s.T * s.G + P.GW - 1) / P.GW;   // workgroups per (b, kv head)
  P.n_wg = s.B * s.Hkv * P.n_groups;
  return P;
}

}  // namespace

size_t score_scratch_bytes(const Shape& s) {
  const size_t tri = (s.T >= 2) ? (size_t)(s.T - 1) * (s.T - 2) / 2 : 0;
  return sizeof(float) * (size_t)s.B * s.H * tri;
}

hipError_t launch_score_select(const Shape& s, const uint16_t* Q, const uint16_t* meta,
                               const float* scores_in, float* scores_out,
                               int32_t* idx_sorted, float* sigma, void* workspace,
                               hipStream_t stream) {
  SelParams P = score_params(s, Q, meta);
  P.scores_in = scores_in;
  P.scores_out = scores_out;
  P.idx_sorted = idx_sorted;
  P.sigma = sigma;
  P.scratch = workspace ? reinterpret_cast<float*>(static_cast<unsigned char*>(workspace) + ws_scores_off(s))
                        : nullptr;
  int cap = 2;
  const int rmax = s.W < s.NB ? s.W : s.NB;
  while (cap < rmax) cap <<= 1;
  int sel_bytes = 8 * cap;
  if (sel_bytes < 8 * kSurvivors) sel_bytes = 8 * kSurvivors;
  P.wave_lds = sel_bytes;
  P.ring_lds = 0;
  if (scores_in) return launch_select<false>(P, stream);
  if (scores_out) {
    const hipError_t e = launch_score_d<kOutFull>(P, stream);
    if (e != hipSuccess) return e;
    P.scores_in = scores_out;
    return launch_select<false>(P, stream);
  }
  const hipError_t e = launch_score_d<kOutPacked>(P, stream);
  if (e != hipSuccess) return e;
  return launch_select<true>(P, stream);
}

hipError_t launch_row_roughness(const Shape& s, const uint16_t* Q, const uint16_t* meta,
                                double* rough, hipStream_t stream) {
  SelParams P = score_params(s, Q, meta);
  P.rough = rough;
  return launch_score_d<kOutRough>(P, stream);
}

}  // namespace ugbs
