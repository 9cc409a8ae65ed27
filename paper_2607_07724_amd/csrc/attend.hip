// Stage 5: block-sparse causal attention over kv_idx (A.10; Eq. (Attn)).
//
// One workgroup of two waves per (batch, query head, Q-tile) unit; wave w
// owns query rows 32w..32w+31 of the tile.  The tile's kv_idx row is first
// compacted into LDS (entries outside 0..t are dropped, order kept), then
// the listed key blocks are visited one by one:
//   - the next block's K and V are fetched into registers while the current
//     block is computed, then written to LDS: K as [key][d], V transposed as
//     [d][key] (both rows padded by 16 bytes against bank conflicts);
//   - S^T = K Q^T on v_mfma_f32_16x16x32_bf16 (K from LDS is the A operand,
//     the wave's 32 query rows stay in registers as the B operand), so each
//     lane holds the scores of one query row for 16 keys;
//   - fp32 online softmax in base 2 (the log2(e) factor is folded into the
//     scale); only the diagonal block t is masked (key > row);
//   - O^T += V^T P^T on the same MFMA: the lane's probabilities, packed to
//     bf16, are already the B operand, and V^T rows from LDS are the A
//     operand.
// Per listed block and unit: 4*64*64*d FLOP on 2*64*d*2 bytes of K/V.
#include "ugbs_internal.h"

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
  float scale_log2;
};

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  const __bf16 x = (__bf16)a, y = (__bf16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

template <int D>
struct Smem {
  static constexpr int kStride = D + 8;      // K row stride (bf16)
  static constexpr int vStride = kBlock + 8; // V^T row stride (bf16)
  static constexpr int kBytes = kBlock * kStride * 2;
  static constexpr int vBytes = D * vStride * 2;
  static constexpr int listOff = kBytes + vBytes;
};

template <int D>
__global__ void __launch_bounds__(128) attend_kernel(AttnParams P) {
  using L = Smem<D>;
  constexpr int KS = D / 32;      // k-steps of QK^T
  constexpr int DT = D / 16;      // 16-wide d tiles of O^T
  constexpr int KCH = kBlock * D / 8 / 128;  // 16-byte K chunks per thread
  constexpr int VP = D / 64;      // V passes (8 d-groups of 8 channels each)
  extern __shared__ __align__(16) unsigned char smem[];
  uint16_t* s_k = reinterpret_cast<uint16_t*>(smem);
  uint16_t* s_vt = reinterpret_cast<uint16_t*>(smem + L::kBytes);
  int32_t* s_list = reinterpret_cast<int32_t*>(smem + L::listOff);
  __shared__ int s_n;

  const Shape& s = P.s;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const int uid = xcd_remap(blockIdx.x, P.n_units);
  if (uid >= P.n_units) return;
  const Unit u = unit_of(uid, s);
  const int kvh = u.h / s.G;
  const size_t rowid = ((size_t)u.b * s.H + u.h) * s.T + u.t;

  // ---- compact the kv_idx row (wave 0), preserving slot order -------------
  if (w == 0) {
    const int32_t* kr = P.kv_idx + rowid * P.kv_width;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int n = 0;
    for (int base = 0; base < P.kv_width; base += 64) {
      const int sl = base + lane;
      const int blk = (sl < P.kv_width) ? kr[sl] : -1;
      const bool ok = blk >= 0 && blk <= u.t;
      const uint64_t m = __ballot(ok);
      if (ok) s_list[n + __popcll(m & lt)] = blk;
      n += __popcll(m);
    }
    if (lane == 0) s_n = n;
  }
  __syncthreads();
  const int n = s_n;

  const size_t qo_base = ((size_t)u.b * s.H + u.h) * s.N + (size_t)u.t * kBlock;
  if (n == 0) {  // no attended key: O = 0
    for (int i = tid; i < kBlock * D / 8; i += 128)
      reinterpret_cast<uint4*>(P.O + qo_base * D)[i] = make_uint4(0, 0, 0, 0);
    return;
  }

  // ---- query rows as the B operand --------------------------------------
  bf16x8 bq[2][KS];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const uint16_t* qr = P.Q + (qo_base + 32 * w + 16 * rt + c16) * D + 8 * g;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) bq[rt][ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qr + 32 * ks));
  }

  const uint16_t* Kh = P.K + ((size_t)u.b * s.Hkv + kvh) * s.N * D;
  const uint16_t* Vh = P.V + ((size_t)u.b * s.Hkv + kvh) * s.N * D;

  uint4 rk[KCH];
  uint4 rv[VP][4];
  const int vkg = tid & 15, vdg = tid >> 4;  // V: keys 4*vkg..+3, channels 8*vdg..+7 (+64 per pass)
  auto fetch = [&](int blk) {
    const uint16_t* kb = Kh + (size_t)blk * kBlock * D;
#pragma unroll
    for (int j = 0; j < KCH; ++j) {
      const int c = tid + 128 * j;
      rk[j] = *reinterpret_cast<const uint4*>(kb + (size_t)(c / (D / 8)) * D + (c % (D / 8)) * 8);
    }
    const uint16_t* vb = Vh + (size_t)blk * kBlock * D;
#pragma unroll
    for (int pv = 0; pv < VP; ++pv)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        rv[pv][r] = *reinterpret_cast<const uint4*>(vb + (size_t)(4 * vkg + r) * D + 64 * pv + 8 * vdg);
  };
  auto stash = [&]() {
#pragma unroll
    for (int j = 0; j < KCH; ++j) {
      const int c = tid + 128 * j;
      *reinterpret_cast<uint4*>(s_k + (c / (D / 8)) * L::kStride + (c % (D / 8)) * 8) = rk[j];
    }
#pragma unroll
    for (int pv = 0; pv < VP; ++pv) {
      const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&rv[pv][0]);
      const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&rv[pv][1]);
      const uint32_t* r2 = reinterpret_cast<const uint32_t*>(&rv[pv][2]);
      const uint32_t* r3 = reinterpret_cast<const uint32_t*>(&rv[pv][3]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int wd = e >> 1, sh = (e & 1) * 16;
        const uint32_t x0 = (r0[wd] >> sh) & 0xffffu, x1 = (r1[wd] >> sh) & 0xffffu;
        const uint32_t x2 = (r2[wd] >> sh) & 0xffffu, x3 = (r3[wd] >> sh) & 0xffffu;
        uint2 pk = make_uint2(x0 | (x1 << 16), x2 | (x3 << 16));
        *reinterpret_cast<uint2*>(s_vt + (64 * pv + 8 * vdg + e) * L::vStride + 4 * vkg) = pk;
      }
    }
  };

  f32x4 acc_o[DT][2];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) acc_o[dt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {-__builtin_huge_valf(), -__builtin_huge_valf()};
  float l_run[2] = {0.f, 0.f};

  fetch(s_list[0]);
  stash();
  __syncthreads();

  for (int it = 0; it < n; ++it) {
    const int blk = s_list[it];
    if (it + 1 < n) fetch(s_list[it + 1]);

    // S^T = K Q^T : [64 keys x 32 rows] per wave
    f32x4 sc[4][2];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) sc[kt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const bf16x8 ak = as_bf16x8(*reinterpret_cast<const uint4*>(
            s_k + (16 * kt + c16) * L::kStride + 32 * ks + 8 * g));
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
          sc[kt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ak, bq[rt][ks], sc[kt][rt], 0, 0, 0);
      }
    }

    // online softmax (base 2); lane holds row (32w + 16rt + c16), keys 16kt + 4g + i
    const bool diag = (blk == u.t);
    float alpha[2];
    uint32_t pb[2][2][4];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const int r = 32 * w + 16 * rt + c16;
      float mx = -__builtin_huge_valf();
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = sc[kt][rt][i] * P.scale_log2;
          if (diag && (16 * kt + 4 * g + i) > r) v = -__builtin_huge_valf();
          sc[kt][rt][i] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[rt], mx);
      alpha[rt] = exp2f(m_run[rt] - m_new);
      m_run[rt] = m_new;
      float ls = 0.f;
      float p[4][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          p[kt][i] = exp2f(sc[kt][rt][i] - m_new);
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
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc_o[dt][rt][i] *= alpha[rt];

    // O^T += V^T P^T
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const uint16_t* vr = s_vt + (16 * dt + c16) * L::vStride + 32 * j + 4 * g;
        const uint2 lo = *reinterpret_cast<const uint2*>(vr);
        const uint2 hi = *reinterpret_cast<const uint2*>(vr + 16);
        const bf16x8 av = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          const bf16x8 bp = as_bf16x8(make_uint4(pb[rt][j][0], pb[rt][j][1], pb[rt][j][2], pb[rt][j][3]));
          acc_o[dt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bp, acc_o[dt][rt], 0, 0, 0);
        }
      }
    }

    __syncthreads();
    if (it + 1 < n) {
      stash();
      __syncthreads();
    }
  }

  // ---- normalise and store: lane holds O^T[16dt + 4g + i][row] ------------
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    float l = l_run[rt];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const float inv = (l > 0.f) ? 1.0f / l : 0.f;
    const int r = 32 * w + 16 * rt + c16;
    uint16_t* orow = P.O + (qo_base + r) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const f32x4 a = acc_o[dt][rt];
      *reinterpret_cast<uint2*>(orow + 16 * dt + 4 * g) =
          make_uint2(pack_bf16(a[0] * inv, a[1] * inv), pack_bf16(a[2] * inv, a[3] * inv));
    }
  }
}

template <int D>
hipError_t launch_t(const AttnParams& P, hipStream_t stream) {
  using L = Smem<D>;
  const size_t smem = L::listOff + sizeof(int32_t) * (size_t)P.kv_width;
  const int grid = ((P.n_units + 7) / 8) * 8;
  attend_kernel<D><<<grid, 128, smem, stream>>>(P);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attend(const Shape& s, const uint16_t* Q, const uint16_t* K,
                         const uint16_t* V, const int32_t* kv_idx, int kv_width,
                         uint16_t* O, hipStream_t stream) {
  AttnParams P;
  P.s = s;
  P.Q = Q;
  P.K = K;
  P.V = V;
  P.kv_idx = kv_idx;
  P.O = O;
  P.kv_width = kv_width;
  P.n_units = s.B * s.H * s.T;
  P.scale_log2 = s.scale * 1.4426950408889634f;
  return s.d == 128 ? launch_t<128>(P, stream) : launch_t<64>(P, stream);
}

}  // namespace ugbs
