// Stage 5: block-sparse causal attention over kv_idx (A.10; Eq. (Attn)).
//
// One workgroup per (batch, query head, Q-tile) unit: two waves of 32 query
// rows (d <= 128) or four waves of 16 rows (d = 256); wave w owns rows
// RPW w .. RPW w + RPW - 1 of the tile.  The tile's kv_idx row is first
// turned into an ascending list of distinct blocks in 0..t (so the diagonal
// block comes last), then the listed key blocks are visited one by one.
//
// Staging.  K and V blocks (64 keys x d, bf16) go global -> LDS with
// direct-to-LDS loads (global_load_lds_dwordx4: no registers, no VALU).
// Both live unpadded in natural [key][d] layout with the 16-byte columns of
// each row permuted by an XOR swizzle (column c of row r of K at c ^ (r mod
// d/8), of V at c ^ (2r mod d/8)), chosen so that the K-operand reads and the
// transposing V reads below are free of LDS bank conflicts.  K and V have one
// buffer each and are refilled in a split ping-pong: K(i+1) is fetched as
// soon as all waves have finished S(i), V(i+1) as soon as all have
// finished PV(i), so the fetches overlap the softmax and the other matrix
// product.
//
// Compute, per block and wave (v_mfma_f32_16x16x32_bf16):
//   S^T = K Q^T   K rows from LDS (ds_read_b128) are the A operand; the
//                 wave's query rows (32, or 16 at d = 256) stay in
//                 registers as the B operand;
//                 each lane ends up holding 16 keys of one query row.  S of
//                 the next block is issued together with the softmax of the
//                 current one, so the matrix cores and the VALU overlap.
//   softmax       fp32 online softmax in base 2 (log2 e folded into the
//                 scale); only the diagonal block t is masked (key > row);
//                 the reference max is raised only when a row max exceeds
//                 it by more than 2^8, so O is rarely rescaled.
//   O^T += V^T P^T  the lane's probabilities, packed to bf16, already are
//                 the B operand; V^T comes straight from the natural-layout
//                 LDS tile through the transposing read ds_read_b64_tr_b16
//                 (16 lanes fetch a 4-key x 16-channel patch and each lane
//                 receives the 4 keys of one channel).
// Per listed block and unit: 4*64*64*d FLOP on 2*64*d*2 bytes of K/V.
#include <atomic>
#include <type_traits>

#include "attend_common.h"

namespace ugbs {
namespace {

struct AttnParams {
  Shape s;
  const uint16_t* Q;
  const uint16_t* K;
  const uint16_t* V;
  const int32_t* kv_idx;
  uint16_t* O;
  int kv_width;
  int n_units;
  int conc;          // units resident at once on one XCD (rotation period)
  float scale_log2;
  // in-kernel selection (ugbs_attend_select)
  const float* sel_scores;    // [B, H, T, N_B] tile scores, or nullptr: packed rows
  const float* sel_packed;    // packed candidate rows (workspace)
  const uint8_t* sel_trigger; // [B, T] trigger flags
  // block bitmaps (ugbs_attend_bitmap)
  const uint32_t* bitmap;     // [B, H, T, nw]
  int nw;
};

// Where a tile's blocks come from.  kSelectWide: kSelect for rows of more
// than 2048 candidate blocks (64 instead of 32 candidates per lane).
enum Mode { kLists = 0, kSelect = 1, kBitmap = 2, kSelectWide = 3 };

// Waves per unit and 16-row tiles per wave: d <= 128 runs two waves of 32
// query rows; d = 256 four waves of 16 rows (half the accumulators per wave,
// so two waves still fit on a SIMD).
template <int D>
struct Geo {
  static constexpr int RT = D > 128 ? 1 : 2;   // 16-row tiles per wave
  static constexpr int NWV = 4 / RT;           // waves per unit (64 rows)
  static constexpr int kThreads = 64 * NWV;
};

template <int D>
struct Tile : TileGeom<D> {
  static constexpr int kLoadsPerWave = TileGeom<D>::kLoads / Geo<D>::NWV;
};
template <int D, bool V>
using FetchPlan = FetchPlanT<D, V, Geo<D>::NWV>;


// Two waves per SIMD at every d (at d = 256 through the four-wave geometry).
template <int D, int MODE>
__global__ void __launch_bounds__(Geo<D>::kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
attend_kernel(AttnParams P) {
  using L = Tile<D>;
  constexpr int KS = D / 32;      // k-steps of QK^T
  constexpr int DT = D / 16;      // 16-channel tiles of O^T
  constexpr int NW = L::kLoadsPerWave;
  constexpr int RT = Geo<D>::RT;
  constexpr int RPW = 16 * RT;    // query rows per wave
  __shared__ __align__(16) uint16_t s_k[L::kElems];
  __shared__ __align__(16) uint16_t s_v[L::kElems];
  extern __shared__ int32_t s_list[];          // [kv_width]: at most kv_width distinct blocks
  __shared__ uint32_t s_bits[UGBS_MAX_BLOCKS / 32];
  __shared__ int s_n, s_below;

  const Shape& s = P.s;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, uniform per wave
  const int g = lane >> 4, c16 = lane & 15;
  // Work order: two kv heads at a time across the whole device (XCDs 0-3 on
  // one, 4-7 on the other, so the memory-side cache holds the working set),
  // one kv head at a time when the (batch, kv head) count is odd; within a
  // kv head the XCDs of its group take its tiles round-robin (heaviest
  // first, every tile size on every XCD), the sibling query heads of a tile
  // one after another on the same XCD.  Workgroup j runs on XCD j mod 8.
  Unit u;
  {
    const int nbh = s.B * s.Hkv;
    const int hpp = (nbh % 2 == 0 && s.T % 4 == 0) ? 2 : 1;   // kv heads in flight
    const int stride = 8 / hpp;                                // XCDs per kv head
    const int n_x = blockIdx.x >> 3, x = blockIdx.x & 7;
    if (s.T % stride != 0) {                                   // fall back: units dealt round-robin to the XCDs
      const int uid = blockIdx.x;
      if (uid >= P.n_units) return;
      u = unit_of(uid, s);
    } else {
      const int tiles_x = s.T / stride;                        // tiles per XCD and kv head
      const int phase = n_x / (tiles_x * s.G);
      const int within = n_x - phase * tiles_x * s.G;
      const int hh = hpp * phase + x / stride;                 // (batch, kv head) index
      if (hh >= nbh) return;
      const int tr = stride * (within / s.G) + x % stride;
      u.b = hh / s.Hkv;
      u.h = (hh % s.Hkv) * s.G + within % s.G;
      u.t = s.T - 1 - tr;
    }
  }
  const int kvh = u.h / s.G;
  const size_t rowid = ((size_t)u.b * s.H + u.h) * s.T + u.t;

  // ---- the tile's kept blocks, ascending (wave 0): kv_idx entries outside
  // 0..t are dropped and repeated entries count once (set semantics, as in
  // Eq. (Attn)), so the diagonal block t, the only one needing the causal
  // mask, is the last entry when present.
  //
  // Visiting order.  The j-th workgroup an XCD receives starts its walk at
  // the first listed block >= (j mod 2 conc) / (2 conc) of its key range and
  // wraps around (the diagonal block stays last).  Workgroups follow each
  // other on an XCD in the order of j, conc of them at a time, so the ones
  // resident together sweep the key range in step and blocks they share
  // stay in that XCD's L2.  Measured at 128K: with kv_idx lists (about 70
  // blocks per tile, or every visible block) a period of 2 conc is best (1
  // and 4 conc slower); with the per-row bitmaps (hundreds of blocks per
  // tile) 1 conc is 9% faster than 2 conc.  The order changes only the
  // summation order of the softmax.
  const int j_xcd = blockIdx.x >> 3;
  const int period = (MODE == kBitmap ? 1 : 2) * P.conc;
  const int start_blk = (int)(((long long)(j_xcd % period) * u.t) / period);
  // Selection modes, shared part: the unit's waves split the candidate
  // loads, the keys, each lane's top-3 pre-filter and the survivor
  // compaction (wave v takes the v-th contiguous slice of the slots, so the
  // survivors land in position order, as one wave would write them); the
  // exact threshold among the survivors stays with wave 0 below.  A lane's
  // top 3 over the waves' slices is its top 3 over every slot, so the bound
  // t0, the survivors and the kept set are those of the one-wave form.
  int staged = -1;                                     // survivors staged in s_k, or -1
  if constexpr (MODE == kSelect || MODE == kSelectWide) {
    const int t = u.t;
    const int nf = (t == 0) ? 1 : 2;
    const int nc = (t >= 1) ? t - 1 : 0;
    const int flag = __builtin_amdgcn_readfirstlane((int)P.sel_trigger[(size_t)u.b * s.T + t]);
    const int R = min((flag != 0 ? s.W : s.k) - nf, nc);
    if (R < nc && R <= 192) {
      constexpr int NWV = Geo<D>::NWV;
      constexpr int kSlots = MODE == kSelectWide ? UGBS_MAX_BLOCKS / 64 : 32;
      static_assert(kSlots % NWV == 0, "slots split evenly over the waves");
      constexpr int kPer = kSlots / NWV;
      const int nslots = (nc + 63) / 64;
      const float* src = P.sel_scores ? P.sel_scores + rowid * s.NB + 1
                                      : P.sel_packed + packed_row(u.b * s.H + u.h, t, s.T);
      uint32_t keys[kPer];
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        const int sl = w * kPer + j;
        const int p = 64 * sl + lane;
        keys[j] = (sl < nslots && p < nc) ? order_key(src[p]) : 0u;
      }
      uint32_t top3[3] = {0u, 0u, 0u};
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        const uint32_t x = keys[j];
        top3[2] = max(top3[2], min(top3[1], x));
        top3[1] = max(top3[1], min(top3[0], x));
        top3[0] = max(top3[0], x);
      }
      uint32_t* s_t3 = reinterpret_cast<uint32_t*>(s_v);            // [NWV][3][64]
      int* s_cnt = reinterpret_cast<int*>(s_t3 + NWV * 3 * 64);      // [NWV]
#pragma unroll
      for (int i = 0; i < 3; ++i) s_t3[(w * 3 + i) * 64 + lane] = top3[i];
      __syncthreads();
      uint32_t m3[3] = {0u, 0u, 0u};
#pragma unroll
      for (int v = 0; v < NWV * 3; ++v) {
        const uint32_t x = s_t3[v * 64 + lane];
        m3[2] = max(m3[2], min(m3[1], x));
        m3[1] = max(m3[1], min(m3[0], x));
        m3[0] = max(m3[0], x);
      }
      bool exact0;
      const uint32_t t0 = kth_largest<3>(m3, 3, R, &exact0);
      int mine = 0;
#pragma unroll
      for (int j = 0; j < kPer; ++j) mine += __popcll(__ballot(t0 > 0u && keys[j] >= t0));
      if (lane == 0) s_cnt[w] = mine;
      __syncthreads();
      int off = 0, ns = 0;
#pragma unroll
      for (int v = 0; v < NWV; ++v) {
        const int c = s_cnt[v];
        off += (v < w) ? c : 0;
        ns += c;
      }
      constexpr int kSurv = 256;
      if (t0 > 0u && ns <= kSurv) {
        uint64_t* s_surv = reinterpret_cast<uint64_t*>(s_k);
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
          const bool tk = keys[j] >= t0;
          const uint64_t mk = __ballot(tk);
          if (tk) s_surv[off + lanes_below(mk)] = ((uint64_t)keys[j] << 32) | (uint32_t)(64 * (w * kPer + j) + lane);
          off += __popcll(mk);
        }
        staged = ns;
      }
      __syncthreads();
    }
  }
  if (w == 0) {
    const int nwords = (u.t >> 5) + 1;                 // bitmap words covering blocks 0..t
    for (int i = lane; i < nwords; i += 64) s_bits[i] = 0u;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
    if constexpr (MODE == kBitmap) {
      // the caller's bitmap row; bits of blocks after t are dropped
      const uint32_t* br = P.bitmap + rowid * P.nw;
      for (int i = lane; i < nwords; i += 64) {
        uint32_t v = br[i];
        if (i == (u.t >> 5)) v &= (u.t & 31) == 31 ? 0xffffffffu : ((2u << (u.t & 31)) - 1u);
        s_bits[i] = v;
      }
    } else if constexpr (MODE == kLists) {
      const int32_t* kr = P.kv_idx + rowid * P.kv_width;
      for (int base = 0; base < P.kv_width; base += 64) {
        const int sl = base + lane;
        const int blk = (sl < P.kv_width) ? kr[sl] : -1;
        if (blk >= 0 && blk <= u.t) atomicOr(&s_bits[blk >> 5], 1u << (blk & 31));
      }
    } else {
      // selection (A.4-A.5, A.9) from the tile scores: the forced sink and
      // self blocks, then the R best candidates of C(t) = {1..t-1} by (score
      // descending, block ascending), R = (trigger ? rho k : k) - |F|, all
      // of them when fewer: the same set as the kept prefix of kv_idx
      const int t = u.t;
      const int nf = (t == 0) ? 1 : 2;
      const int nc = (t >= 1) ? t - 1 : 0;
      // The flag is loaded unconditionally (every (b, t) has one) and moved
      // to a scalar register: written as a load guarded by nc > 0, the
      // branch around the load and the k / rho k phi after it came out of
      // this compiler with the phi's rho k copy executed unconditionally.
      // With nc == 0, R is 0 whatever the flag.
      const int flag = __builtin_amdgcn_readfirstlane((int)P.sel_trigger[(size_t)u.b * s.T + t]);
      const int R = min((flag != 0 ? s.W : s.k) - nf, nc);
      if (lane == 0) {
        atomicOr(&s_bits[0], 1u);
        if (t > 0) atomicOr(&s_bits[t >> 5], 1u << (t & 31));
      }
      if (R >= nc) {
        for (int blk = 1 + lane; blk <= nc; blk += 64) atomicOr(&s_bits[blk >> 5], 1u << (blk & 31));
      } else if (staged >= 0) {
        // the survivors the waves staged: the exact R largest among them
        constexpr int kSurv = 256;
        const uint64_t* s_surv = reinterpret_cast<const uint64_t*>(s_k);
        uint32_t k2[kSurv / 64], p2[kSurv / 64];
#pragma unroll
        for (int sl = 0; sl < kSurv / 64; ++sl) {
          const int i = 64 * sl + lane;
          const uint64_t v = (i < staged) ? s_surv[i] : 0ull;
          k2[sl] = (uint32_t)(v >> 32);
          p2[sl] = (uint32_t)v;
        }
        select_top_each<kSurv / 64>(k2, (staged + 63) / 64, R, lane, [&](int sl) {
          const int blk = 1 + (int)p2[sl];
          atomicOr(&s_bits[blk >> 5], 1u << (blk & 31));
        });
      } else {
        const float* src = P.sel_scores ? P.sel_scores + rowid * s.NB + 1
                                        : P.sel_packed + packed_row(u.b * s.H + u.h, t, s.T);
        constexpr int kSlots = MODE == kSelectWide ? UGBS_MAX_BLOCKS / 64 : 32;
        static_assert(UGBS_MAX_BLOCKS <= 64 * 64, "at most 64 slots per lane");
        const int nslots = (nc + 63) / 64;
        uint32_t keys[kSlots];
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
          const int p = 64 * sl + lane;
          keys[sl] = (sl < nslots && p < nc) ? order_key(src[p]) : 0u;
        }
        // Pre-filter as in the selection kernel: the R-th largest of the
        // lanes' three largest keys bounds the R-th largest key from below;
        // the survivors (keys at or above it, in position order) go through
        // the exact threshold on 4 slots per lane instead of 32.  The K
        // tile's LDS holds them (no K block is in flight yet).
        bool done = false;
        if (R <= 192) {
          uint32_t top3[3] = {0u, 0u, 0u};
#pragma unroll
          for (int sl = 0; sl < kSlots; ++sl) {
            if (sl < nslots) {
              const uint32_t x = keys[sl];
              top3[2] = max(top3[2], min(top3[1], x));
              top3[1] = max(top3[1], min(top3[0], x));
              top3[0] = max(top3[0], x);
            }
          }
          bool exact0;
          const uint32_t t0 = kth_largest<3>(top3, 3, R, &exact0);
          constexpr int kSurv = 256;
          uint64_t* s_surv = reinterpret_cast<uint64_t*>(s_k);
          int ns = 0;
#pragma unroll
          for (int sl = 0; sl < kSlots; ++sl) {
            if (sl < nslots) {
              const bool tk = t0 > 0u && keys[sl] >= t0;
              const uint64_t mk = __ballot(tk);
              const int at = ns + lanes_below(mk);
              if (tk && at < kSurv) s_surv[at] = ((uint64_t)keys[sl] << 32) | (uint32_t)(64 * sl + lane);
              ns += __popcll(mk);
            }
          }
          if (t0 > 0u && ns <= kSurv) {
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            __builtin_amdgcn_wave_barrier();
            uint32_t k2[kSurv / 64], p2[kSurv / 64];
#pragma unroll
            for (int sl = 0; sl < kSurv / 64; ++sl) {
              const int i = 64 * sl + lane;
              const uint64_t v = (i < ns) ? s_surv[i] : 0ull;
              k2[sl] = (uint32_t)(v >> 32);
              p2[sl] = (uint32_t)v;
            }
            select_top_each<kSurv / 64>(k2, (ns + 63) / 64, R, lane, [&](int sl) {
              const int blk = 1 + (int)p2[sl];
              atomicOr(&s_bits[blk >> 5], 1u << (blk & 31));
            });
            done = true;
          }
        }
        if (!done)
          select_top_each<kSlots>(keys, nslots, R, lane, [&](int sl) {
            const int blk = 1 + 64 * sl + lane;
            atomicOr(&s_bits[blk >> 5], 1u << (blk & 31));
          });
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
    int n = 0, below = 0;
    for (int base = 0; base <= u.t; base += 64) {
      const int blk = base + lane;
      const bool on = blk <= u.t && ((s_bits[blk >> 5] >> (blk & 31)) & 1u);
      const uint64_t m = __ballot(on);
      if (on) s_list[n + lanes_below(m)] = blk;
      n += __popcll(m);
      below += __popcll(__ballot(on && blk < start_blk));
    }
    if (lane == 0) {
      s_n = n;
      s_below = below;
    }
  }
  __syncthreads();
  const int n = __builtin_amdgcn_readfirstlane(s_n);
  const bool diag_last = n > 0 && s_list[n - 1] == u.t;
  // entries 0..n_rot-1 are visited from position rot0 on, cyclically
  const int n_rot = __builtin_amdgcn_readfirstlane(diag_last ? n - 1 : n);
  const int rot0 = __builtin_amdgcn_readfirstlane(s_below < n_rot ? s_below : 0);
  // listed_raw: the i-th block to visit as a per-lane LDS value (every lane
  // the same); listed: the same, moved to a scalar register
  auto listed_raw = [&](int i) {
    int p = i;
    if (i < n_rot) {
      p = i + rot0;
      if (p >= n_rot) p -= n_rot;
    }
    return s_list[p];
  };
  auto listed = [&](int i) { return __builtin_amdgcn_readfirstlane(listed_raw(i)); };

  const size_t qo_base = ((size_t)u.b * s.H + u.h) * s.N + (size_t)u.t * kBlock;
  if (n == 0) {  // no attended key: O = 0
    for (int i = tid; i < kBlock * D / 8; i += Geo<D>::kThreads)
      reinterpret_cast<uint4*>(P.O + qo_base * D)[i] = make_uint4(0, 0, 0, 0);
    return;
  }

  // ---- query rows as the B operand --------------------------------------
  bf16x8 bq[RT][KS];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const uint16_t* qr = P.Q + (qo_base + RPW * w + 16 * rt + c16) * D + 8 * g;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) bq[rt][ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qr + 32 * ks));
  }
  wait_vmcnt<0>();

  const uint16_t* Kh = P.K + ((size_t)u.b * s.Hkv + kvh) * s.N * D;
  const uint16_t* Vh = P.V + ((size_t)u.b * s.Hkv + kvh) * s.N * D;
  // Who issues a tile's sixteen 1 KiB loads.  At d <= 128 the first wave
  // issues all of a K tile and the last wave all of a V tile, so while one
  // wave waits for the texture unit to accept its loads the other keeps
  // computing (1-2% faster at 32K-128K than each wave issuing half of
  // every tile, same output bits).  At d = 256 each wave issues its share:
  // one issuer would need more offset registers than that kernel has.
  const uint32_t k_lds = __builtin_amdgcn_readfirstlane(lds_addr(s_k));
  const uint32_t v_lds = __builtin_amdgcn_readfirstlane(lds_addr(s_v));
  constexpr bool kSplitIssue = D <= 128;
  constexpr int kIssuers = kSplitIssue ? 1 : Geo<D>::NWV;
  FetchPlanT<D, false, kIssuers> kplan;
  FetchPlanT<D, true, kIssuers> vplan;
  const int iw = kSplitIssue ? 0 : w;             // index within the issuing waves
  kplan.init(lane, iw);
  vplan.init(lane, iw);
  auto fetch_k = [&](int b) {
    if (!kSplitIssue || w == 0) kplan.fetch(Kh + (size_t)b * Tile<D>::kElems, k_lds, iw);
  };
  auto fetch_v = [&](int b) {
    if (!kSplitIssue || w == Geo<D>::NWV - 1) vplan.fetch(Vh + (size_t)b * Tile<D>::kElems, v_lds, iw);
  };

  f32x4 acc_o[DT][RT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc_o[dt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[RT], l_run[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    m_run[rt] = -__builtin_huge_valf();
    l_run[rt] = 0.f;
  }

  // S^T = K Q^T : [64 keys x 32 rows] per wave, K from LDS
  auto compute_s = [&](f32x4 (&sc)[4][RT]) {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) sc[kt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const int r = 16 * kt + c16;
        const bf16x8 ak = as_bf16x8(*reinterpret_cast<const uint4*>(s_k + L::off(r, 4 * ks + g, false)));
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          sc[kt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ak, bq[rt][ks], sc[kt][rt], 0, 0, 0);
      }
    }
  };

  // Pipeline per listed block i (K and V have one LDS buffer each):
  //   S(i+1) on the matrix cores overlaps the softmax of S(i) on the VALU,
  //   then O += P(i) V(i).  K(i+2) is fetched once S(i+1) is done, V(i+1)
  //   once PV(i) is done.  Fetch order per wave: K0 V0 K1 | K2 V1 | K3 V2 ...
  //   Two barriers per block: each one both frees a buffer (all waves done
  //   reading it) and publishes the one load then in flight (V(i) before
  //   PV(i), K(i+2) before the next S), so every wait is for all loads.
  int blk = listed(0);
  fetch_k(blk);
  fetch_v(blk);
  f32x4 sc[4][RT];
  // K0 landed (V0 may still be in flight)
  if constexpr (kSplitIssue) {
    if (w == 0) wait_vmcnt<0>();
  } else {
    wait_vmcnt<NW>();
  }
  lds_barrier();
  compute_s(sc);
  wait_lgkm0();
  lds_barrier();                         // all waves are done reading s_k
  // The indices of the next two blocks travel one step ahead: the LDS read
  // of block it + 3 goes out at the end of step it, and its scalar copy is
  // taken where step it + 1 needs it, so no list read waits on the LDS
  // right after a barrier.
  int nb1 = (n > 1) ? listed(1) : 0;     // block it + 1
  int raw2 = (n > 2) ? listed_raw(2) : 0;  // block it + 2, per-lane copy
  if (n > 1) {
    fetch_k(nb1);
    wait_vmcnt<0>();                     // K1 (and V0) landed
    lds_barrier();
  }

  // One pipeline step for listed block `it`; MASK: it is the diagonal block
  // (always the last one), whose keys after the query row are masked.
  auto step = [&](int it, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const bool has_next = it + 1 < n;
    const bool has_next2 = it + 2 < n;
    const int nblk = has_next ? nb1 : 0;

    // S(it+1): on the last block this re-reads s_k (no fetch is pending) and is discarded
    f32x4 sn[4][RT];
    __builtin_amdgcn_s_setprio(1);       // matrix-core phases issue ahead of other waves' fetch phases
    compute_s(sn);

    // online softmax of S(it) (base 2); lane holds row (32w + 16rt + c16),
    // keys 16kt + 4g + i.  The reference max m_run only moves when a row max
    // exceeds it by more than 2^8, so p <= 256 and O is rescaled rarely.
    if constexpr (MASK) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int r = RPW * w + 16 * rt + c16;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if ((16 * kt + 4 * g + i) > r) sc[kt][rt][i] = -__builtin_huge_valf();
      }
    }
    float alpha[RT];
    uint32_t pb[RT][2][4];
    bool moved = false;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      float mx = fmaxf(fmaxf(sc[0][rt][0], sc[0][rt][1]), fmaxf(sc[0][rt][2], sc[0][rt][3]));
#pragma unroll
      for (int kt = 1; kt < 4; ++kt)
        mx = fmaxf(mx, fmaxf(fmaxf(sc[kt][rt][0], sc[kt][rt][1]), fmaxf(sc[kt][rt][2], sc[kt][rt][3])));
      mx = rows_max(mx) * P.scale_log2;
      const bool up = mx > m_run[rt] + 8.0f;
      const float m_new = up ? mx : m_run[rt];
      alpha[rt] = up ? __builtin_amdgcn_exp2f(m_run[rt] - m_new) : 1.0f;
      moved |= up;
      m_run[rt] = m_new;
      float ls = 0.f;
      float p[4][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          p[kt][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[kt][rt][i], P.scale_log2, -m_new));
          ls += p[kt][i];
        }
      l_run[rt] = l_run[rt] * alpha[rt] + ls;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        pb[rt][j][0] = pack_bf16(p[2 * j][0], p[2 * j][1]);
        pb[rt][j][1] = pack_bf16(p[2 * j][2], p[2 * j][3]);
        pb[rt][j][2] = pack_bf16(p[2 * j + 1][0], p[2 * j + 1][1]);
        pb[rt][j][3] = pack_bf16(p[2 * j + 1][2], p[2 * j + 1][3]);
      }
    }
    // interleave, in two halves: the K-operand reads, then one MFMA of
    // S(it+1) per few softmax VALU instructions (8 reads, 16 x (1 + 5) at
    // d = 128)
    constexpr int kHalfReads = 2 * KS, kHalfMfma = 2 * KS * RT, kVpm = RT == 2 ? 5 : 2;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      __builtin_amdgcn_sched_group_barrier(0x100, kHalfReads, 0);
#pragma unroll
      for (int i = 0; i < kHalfMfma; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, kVpm, 0);
      }
    }

    // the whole softmax stays above the barrier, where it overlaps the
    // landing of V(it)
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(0);
    // one barrier: every wave is done reading s_k, and V(it), the only load
    // in flight, has landed
    wait_lgkm0();
    wait_vmcnt<0>();
    lds_barrier();
    if (has_next2) fetch_k(__builtin_amdgcn_readfirstlane(raw2));

    __builtin_amdgcn_s_setprio(1);
    if (__ballot(moved)) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc_o[dt][rt][i] *= alpha[rt];
    }

    // O^T += V^T P^T ; lane (channel 16dt + c16, group g) takes keys
    // 32j + 4g + 0..3 and 32j + 16 + 4g + 0..3 through two transposing reads
    const int tr_row = 4 * g + (c16 >> 2);
    const int tr_col = (c16 & 3) >> 1, tr_half = (c16 & 1) * 4;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int r0 = 32 * j + tr_row, r1 = r0 + 16;
        const int c = 2 * dt + tr_col;
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (LDS_AS v4i16*)(s_v + L::off(r0, c, true) + tr_half));
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (LDS_AS v4i16*)(s_v + L::off(r1, c, true) + tr_half));
        const bf16x8 av = __builtin_bit_cast(
            bf16x8, (short __attribute__((ext_vector_type(8)))){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const bf16x8 bp = as_bf16x8(make_uint4(pb[rt][j][0], pb[rt][j][1], pb[rt][j][2], pb[rt][j][3]));
          acc_o[dt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bp, acc_o[dt][rt], 0, 0, 0);
        }
      }
    }
    __builtin_amdgcn_s_setprio(0);
    if (has_next) {
      // one barrier: every wave is done reading s_v, and K(it+2), the only
      // load in flight (if any), has landed for the next step's S
      wait_lgkm0();
      wait_vmcnt<0>();
      lds_barrier();
      fetch_v(nblk);
    }
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) sc[kt][rt] = sn[kt][rt];
    nb1 = __builtin_amdgcn_readfirstlane(raw2);
    raw2 = (it + 3 < n) ? listed_raw(it + 3) : 0;
  };

  for (int it = 0; it + 1 < n; ++it) step(it, std::false_type{});
  if (diag_last) step(n - 1, std::true_type{});
  else step(n - 1, std::false_type{});

  // ---- normalise and store: lane holds O^T[16dt + 4g + i][row] ------------
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float l = l_run[rt];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const float inv = (l > 0.f) ? 1.0f / l : 0.f;
    const int r = RPW * w + 16 * rt + c16;
    uint16_t* orow = P.O + (qo_base + r) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const f32x4 a = acc_o[dt][rt];
      *reinterpret_cast<uint2*>(orow + 16 * dt + 4 * g) =
          make_uint2(pack_bf16(a[0] * inv, a[1] * inv), pack_bf16(a[2] * inv, a[3] * inv));
    }
  }
}

// Workgroups of attend_kernel<D, MODE> resident at once on one XCD, for the given
// dynamic LDS size (occupancy per CU x CUs per XCD).  Cached per device as
// one packed word (smem << 32 | value); a stale or missing entry only costs
// a recomputation.  The value steers the visiting order, never the result.
constexpr int kMaxDevices = 64;
template <int D, int MODE>
int xcd_concurrency(size_t smem) {
  static std::atomic<uint64_t> cache[kMaxDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev >= kMaxDevices) dev = -1;
  if (dev >= 0) {
    const uint64_t e = cache[dev].load(std::memory_order_relaxed);
    if (e != 0 && (e >> 32) == (uint64_t)smem) return (int)(uint32_t)e;
  }
  int per_cu = 0, n_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attend_kernel<D, MODE>, Geo<D>::kThreads, smem) !=
      hipSuccess)
    per_cu = 1;
  if (dev < 0 || hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) n_cu = 8;
  const int conc = per_cu * n_cu / 8 > 0 ? per_cu * n_cu / 8 : 1;
  if (dev >= 0) cache[dev].store(((uint64_t)smem << 32) | (uint32_t)conc, std::memory_order_relaxed);
  return conc;
}

template <int D, int MODE>
hipError_t launch_t(AttnParams P, hipStream_t stream) {
  const size_t smem = sizeof(int32_t) * (size_t)P.kv_width;
  const int grid = ((P.n_units + 7) / 8) * 8;
  if (D > 128) {  // the K and V tiles alone take 64 KB of static LDS
    const hipError_t e = hipFuncSetAttribute((const void*)attend_kernel<D, MODE>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
  }
  P.conc = xcd_concurrency<D, MODE>(smem);
  attend_kernel<D, MODE><<<grid, Geo<D>::kThreads, smem, stream>>>(P);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attend(const Shape& s, const uint16_t* Q, const uint16_t* K,
                         const uint16_t* V, const int32_t* kv_idx, int kv_width,
                         uint16_t* O, hipStream_t stream) {
  AttnParams P{};
  P.s = s;
  P.Q = Q;
  P.K = K;
  P.V = V;
  P.kv_idx = kv_idx;
  P.O = O;
  P.kv_width = kv_width;
  P.n_units = s.B * s.H * s.T;
  P.scale_log2 = s.scale * 1.4426950408889634f;
  if (s.d == 256) return launch_t<256, kLists>(P, stream);
  return s.d == 128 ? launch_t<128, kLists>(P, stream) : launch_t<64, kLists>(P, stream);
}

hipError_t launch_attend_select(const Shape& s, const uint16_t* Q, const uint16_t* K,
                                const uint16_t* V, const float* scores, const uint8_t* trigger,
                                const void* workspace, uint16_t* O, hipStream_t stream) {
  AttnParams P{};
  P.s = s;
  P.Q = Q;
  P.K = K;
  P.V = V;
  P.O = O;
  // at most |F| + (rho k - |F|) distinct blocks per tile, and never more than t + 1
  P.kv_width = s.W < s.NB ? s.W : s.NB;
  P.n_units = s.B * s.H * s.T;
  P.scale_log2 = s.scale * 1.4426950408889634f;
  const unsigned char* ws = static_cast<const unsigned char*>(workspace);
  P.sel_scores = scores;
  P.sel_packed = ws ? reinterpret_cast<const float*>(ws + ws_scores_off(s)) : nullptr;
  P.sel_trigger = trigger ? trigger : ws + ws_trigger_off(s);
  if (s.NB > 32 * 64) {
    if (s.d == 256) return launch_t<256, kSelectWide>(P, stream);
    return s.d == 128 ? launch_t<128, kSelectWide>(P, stream) : launch_t<64, kSelectWide>(P, stream);
  }
  if (s.d == 256) return launch_t<256, kSelect>(P, stream);
  return s.d == 128 ? launch_t<128, kSelect>(P, stream) : launch_t<64, kSelect>(P, stream);
}

hipError_t launch_attend_bitmap(const Shape& s, const uint16_t* Q, const uint16_t* K,
                                const uint16_t* V, const uint32_t* bitmap, uint16_t* O,
                                hipStream_t stream) {
  AttnParams P{};
  P.s = s;
  P.Q = Q;
  P.K = K;
  P.V = V;
  P.O = O;
  P.kv_width = s.NB;  // a row may list every visible block
  P.n_units = s.B * s.H * s.T;
  P.scale_log2 = s.scale * 1.4426950408889634f;
  P.bitmap = bitmap;
  P.nw = (s.NB + 31) / 32;
  if (s.d == 256) return launch_t<256, kBitmap>(P, stream);
  return s.d == 128 ? launch_t<128, kBitmap>(P, stream) : launch_t<64, kBitmap>(P, stream);
}

}  // namespace ugbs
