// Appendix D diagnostics: sigma read as a best-arm identification index.
//
// noise_kernel     tau[b, h] from the per-unit row roughness the score kernel
//                  produces in its roughness mode (recipe step 3: adjacent
//                  rows of a tile differ by two independent noise draws, so
//                  the mean squared difference is 2 tau^2).
// bai_tile_kernel  one wave per (b, h, t): the sorted top rho k - |F| + 1
//                  candidate scores (same key order as the selection kernel:
//                  score descending, lower block first), the gaps g, G, r and
//                  sigma of Eq. (gaps), the smallest secondary spacing among
//                  ranks 0..R' (assumption (A1)), and a Monte Carlo count of
//                  identification failures of the empirical top-m and top-R'
//                  sets under mu ~ N(s, tau^2 I) with caller-supplied normals.
// bai_head_kernel  one workgroup per (b, h): the aggregates over the tiles
//                  with at least rho k + 1 visible blocks: mean and CV of r,
//                  the empirical quantile sigma_(q) and gamma_q, the band mass
//                  m_q(beta), spacing quantiles, the closed forms chi, eps_bar,
//                  C_q of the Lemma and the Proposition, the bound, and the
//                  Monte Carlo error rates and regret R_q.
//
// Floating-point order: the gaps use fp32 subtract and an IEEE divide; mu is
// fp32(s + fp32(tau z)) without contraction; the head sums of r run in tile
// order in fp64, one thread, so they equal a left-to-right sum.
#include <math.h>

#include "select_common.h"

namespace ugbs {
namespace {

constexpr int kRho = 2;
constexpr int kBaiWaves = 4;
constexpr int kBaiSlots = UGBS_MAX_BLOCKS / 64;
constexpr int kHeadThreads = 256;

struct TileParams {
  Shape s;
  const float* scores;  // [B, H, T, N_B]
  const float* tau;     // [B, H]
  const float* z;       // [n_s, N_B]
  int n_s;
  ugbs_bai_tile* tiles; // [B, H, T]
};

__device__ __forceinline__ float wave_min_f(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fminf(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ float wave_max_f(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

__global__ void __launch_bounds__(64 * kBaiWaves) bai_tile_kernel(TileParams P) {
#pragma clang fp contract(off)
  extern __shared__ __align__(16) unsigned char smem[];
  const Shape& s = P.s;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n_units = s.B * s.H * s.T;
  const int n_wg = (n_units + kBaiWaves - 1) / kBaiWaves;
  const int wg = xcd_remap(blockIdx.x, n_wg);
  if (wg >= n_wg) return;
  const int u = wg * kBaiWaves + w;
  if (u >= n_units) return;
  const int h = u % s.H;
  const int rest = u / s.H;
  const int t = s.T - 1 - rest % s.T;
  const int b = rest / s.T;
  const size_t row = ((size_t)b * s.H + h) * s.T + t;
  const int nf = (t == 0) ? 1 : 2;
  const int nc = (t >= 1) ? t - 1 : 0;
  const int m = s.k - nf;              // kept non-forced slots
  const int Rp = kRho * s.k - nf;      // non-forced slots after expansion
  ugbs_bai_tile* out = P.tiles + row;
  if (nc < Rp + 1 || nc <= m) {
    if (lane == 0) {
      const float nan = __builtin_nanf("");
      *out = ugbs_bai_tile{nan, nan, nan, nan, nan, 0, 0, 0};
    }
    return;
  }
  uint64_t* s_sel = reinterpret_cast<uint64_t*>(smem) + (size_t)w * UGBS_MAX_BLOCKS;
  const float* src = P.scores + row * s.NB + 1;
  const int nslots = (nc + 63) / 64;

  uint32_t keys[kBaiSlots], pos[kBaiSlots];
#pragma unroll
  for (int sl = 0; sl < kBaiSlots; ++sl) {
    const int p = 64 * sl + lane;
    keys[sl] = (sl < nslots && p < nc) ? order_key(src[p]) : 0u;
    pos[sl] = (uint32_t)p;
  }
  // sorted top R' + 1 as (key << 32) | ~position, descending
  const int R1 = Rp + 1;
  select_top<kBaiSlots>(keys, pos, nslots, R1, s_sel, lane);
  int n2 = 2;
  while (n2 < R1) n2 <<= 1;
  for (int p = R1 + lane; p < n2; p += 64) s_sel[p] = 0ull;
  wave_lds_sync();
  lds_bitonic_desc(s_sel, n2, lane);

  auto cs = [&](int j) { return key_value((uint32_t)(s_sel[j] >> 32)); };
  // smallest secondary spacing: ranks j, j + 1 for j = 0..R'-1 except the cut
  float d2 = __builtin_huge_valf();
  for (int j = lane; j < Rp; j += 64)
    if (j != m - 1) d2 = fminf(d2, cs(j) - cs(j + 1));
  d2 = wave_min_f(d2);

  // ---- Monte Carlo identification failures -------------------------------
  const uint64_t thr_k = s_sel[m - 1], thr_r = s_sel[Rp - 1];
  uint32_t in_k = 0u, in_r = 0u, cand = 0u;
  float sc[kBaiSlots];
#pragma unroll
  for (int sl = 0; sl < kBaiSlots; ++sl) {
    const int p = 64 * sl + lane;
    const uint64_t k64 = ((uint64_t)keys[sl] << 32) | (0xffffffffu - (uint32_t)p);
    const bool c = sl < nslots && p < nc;
    cand |= (uint32_t)c << sl;
    in_k |= (uint32_t)(c && k64 >= thr_k) << sl;
    in_r |= (uint32_t)(c && k64 >= thr_r) << sl;
    sc[sl] = key_value(keys[sl]);   // the candidate score with -0 read as +0
  }
  const float tau = P.n_s > 0 ? P.tau[(size_t)b * s.H + h] : 0.f;
  int fail_k = 0, fail_rk = 0;
  for (int smp = 0; smp < P.n_s; ++smp) {
    const float* zr = P.z + (size_t)smp * s.NB + 1;
    float mu[kBaiSlots];
    float mn_k = __builtin_huge_valf(), mx_nk = -__builtin_huge_valf(), mx_nr = -__builtin_huge_valf();
#pragma unroll
    for (int sl = 0; sl < kBaiSlots; ++sl) {
      if (sl < nslots) {
        const int p = 64 * sl + lane;
        const float zv = zr[p < nc ? p : nc - 1];
        mu[sl] = __fadd_rn(sc[sl], __fmul_rn(tau, zv));
        if ((cand >> sl) & 1u) {
          if ((in_k >> sl) & 1u) mn_k = fminf(mn_k, mu[sl]);
          else mx_nk = fmaxf(mx_nk, mu[sl]);
          if (!((in_r >> sl) & 1u)) mx_nr = fmaxf(mx_nr, mu[sl]);
        }
      }
    }
    mn_k = wave_min_f(mn_k);
    mx_nk = wave_max_f(mx_nk);
    mx_nr = wave_max_f(mx_nr);
    int above = 0;
#pragma unroll
    for (int sl = 0; sl < kBaiSlots; ++sl)
      if (sl < nslots) above += __popcll(__ballot(((in_r >> sl) & 1u) && mu[sl] > mx_nr));
    fail_k += !(mn_k > mx_nk);
    fail_rk += above < m;
  }

  if (lane == 0) {
    const float c0 = cs(0), cm1 = cs(m - 1), cm = cs(m), cR = cs(Rp);
    const float g = cm1 - cm, G = cm1 - cR, r = c0 - cm;
    const float sg = (r == 0.0f) ? 0.0f : __fdiv_rn(g, r);
    *out = ugbs_bai_tile{g, G, r, sg, d2, fail_k, fail_rk, 1};
  }
}

// ---- noise scale ------------------------------------------------------------

__global__ void __launch_bounds__(64) noise_kernel(Shape s, const double* rough, float* tau) {
  const int bh = blockIdx.x;
  const int lane = threadIdx.x;
  double acc = 0.0;
  for (int t = lane; t < s.T; t += 64) acc += rough[(size_t)bh * s.T + t];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
  // 63 adjacent row pairs per candidate block, candidates 1..t-1 of tile t
  const double terms = 63.0 * ((s.T >= 2) ? (double)(s.T - 1) * (double)(s.T - 2) / 2.0 : 0.0);
  if (lane == 0) tau[bh] = terms > 0.0 ? (float)sqrt(acc / (2.0 * terms)) : __builtin_nanf("");
}

// ---- per-head aggregates ----------------------------------------------------

struct HeadParams {
  Shape s;
  const ugbs_bai_tile* tiles;
  const float* tau;
  int n_s;
  ugbs_bai_head* heads;
};

__device__ double std_normal_cdf(double x) { return 0.5 * erfc(-x / sqrt(2.0)); }

__device__ double std_normal_pdf(double x) { return exp(-0.5 * x * x) / sqrt(2.0 * M_PI); }

__device__ __forceinline__ double block_sum(double x, double* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  __syncthreads();
  if (lane == 0) red[w] = x;
  __syncthreads();
  double r = 0.0;
  for (int i = 0; i < kHeadThreads / 64; ++i) r += red[i];
  return r;
}

__device__ __forceinline__ long long block_sum_i(long long x, long long* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  __syncthreads();
  if (lane == 0) red[w] = x;
  __syncthreads();
  long long r = 0;
  for (int i = 0; i < kHeadThreads / 64; ++i) r += red[i];
  return r;
}

__global__ void __launch_bounds__(kHeadThreads) bai_head_kernel(HeadParams P) {
#pragma clang fp contract(off)
  __shared__ float s_sig[UGBS_MAX_BLOCKS], s_g[UGBS_MAX_BLOCKS], s_r[UGBS_MAX_BLOCKS],
      s_d2[UGBS_MAX_BLOCKS];
  __shared__ int s_dk[UGBS_MAX_BLOCKS];
  __shared__ int s_n;
  __shared__ double s_red[kHeadThreads / 64];
  __shared__ long long s_redi[kHeadThreads / 64];
  __shared__ float s_pick[3];  // delta2 quantiles 5% / 50%, sigma_(q)
  __shared__ double s_rmean, s_rcv;
  const Shape& s = P.s;
  const int bh = blockIdx.x;
  const int tid = threadIdx.x;
  const double nan = __builtin_nan("");
  ugbs_bai_head* out = P.heads + bh;
  const ugbs_bai_tile* tl = P.tiles + (size_t)bh * s.T;
  const double q = s.q;

  // ---- compact the valid tiles in tile order (wave 0) ---------------------
  if (tid < 64) {
    const uint64_t lt_mask = (tid == 0) ? 0ull : (~0ull >> (64 - tid));
    int base = 0;
    for (int t0 = 0; t0 < s.T; t0 += 64) {
      const int t = t0 + tid;
      ugbs_bai_tile x;
      const bool v = t < s.T && (x = tl[t], x.valid != 0);
      const uint64_t mk = __ballot(v);
      if (v) {
        const int i = base + __popcll(mk & lt_mask);
        s_sig[i] = x.sigma;
        s_g[i] = x.g;
        s_r[i] = x.r;
        s_d2[i] = x.delta2;
        s_dk[i] = x.fail_k - x.fail_rk;
      }
      base += __popcll(mk);
    }
    if (tid == 0) s_n = base;
  }
  __syncthreads();
  const int n = s_n;
  if (n == 0) {
    if (tid == 0) {
      ugbs_bai_head hd;
      hd.n_tiles = 0;
      hd.n_q = 0;
      hd.pad[0] = hd.pad[1] = 0;
      double* f = &hd.r_mean;
      for (int i = 0; i < 18; ++i) f[i] = nan;
      *out = hd;
    }
    return;
  }
  const int nq = (int)ceil(q * (double)n);
  const int i05 = (int)floor(0.05 * (double)(n - 1));
  const int i50 = (int)floor(0.5 * (double)(n - 1));

  // ---- mean and CV of r: left-to-right fp64 sums in tile order ------------
  if (tid == 0) {
    double sum = 0.0;
    for (int i = 0; i < n; ++i) sum += (double)s_r[i];
    const double mean = sum / n;
    double var = 0.0;
    for (int i = 0; i < n; ++i) {
      const double dx = (double)s_r[i] - mean;
      var += dx * dx;
    }
    var = var / n;
    s_rmean = mean;
    s_rcv = (mean != 0.0) ? __dsqrt_rn(var) / mean : nan;
  }

  // ---- order statistics by rank counting ----------------------------------
  // rank of tile i among the spacings (value, then tile order) and among the
  // sigmas (value, then tile order: the router takes the nq smallest, lower
  // tile first on ties); failure differences d = fail_k - fail_rk ranked
  // descending for the oracle-best set
  long long top_d = 0, rsig_d = 0;
  for (int i = tid; i < n; i += kHeadThreads) {
    const float di = s_d2[i], si = s_sig[i];
    const int ki = s_dk[i];
    int rd = 0, rs = 0, rk = 0;
    for (int j = 0; j < n; ++j) {
      const float dj = s_d2[j], sj = s_sig[j];
      const int kj = s_dk[j];
      rd += (dj < di) || (dj == di && j < i);
      rs += (sj < si) || (sj == si && j < i);
      rk += (kj > ki) || (kj == ki && j < i);
    }
    if (rd == i05) s_pick[0] = di;
    if (rd == i50) s_pick[1] = di;
    if (nq > 0 && rs == nq - 1) s_pick[2] = si;
    if (rk < nq) top_d += ki;
    if (rs < nq) rsig_d += ki;
  }
  const long long top = block_sum_i(top_d, s_redi);
  const long long rsig = block_sum_i(rsig_d, s_redi);
  // (block_sum_i synchronises, so s_pick, s_rmean and s_rcv are visible)
  const float p05 = s_pick[0];
  const double r_mean = s_rmean, r_cv = s_rcv;
  const double sq = nq > 0 ? (double)s_pick[2] : nan;
  const double gamma = sq * r_mean, beta = r_cv;
  const double lo = gamma * (1.0 - beta), hi = gamma * (1.0 + beta);

  long long below = 0, band = 0, fk = 0, fr = 0;
  for (int i = tid; i < n; i += kHeadThreads) {
    below += s_d2[i] < p05;
    const double gi = (double)s_g[i];
    band += (lo <= gi && gi <= hi);
  }
  // failure totals straight from the tile records (integers: order-free)
  for (int t = tid; t < s.T; t += kHeadThreads) {
    const ugbs_bai_tile x = tl[t];
    if (x.valid) {
      fk += x.fail_k;
      fr += x.fail_rk;
    }
  }
  const long long n_below = block_sum_i(below, s_redi);
  const long long n_band = nq > 0 ? block_sum_i(band, s_redi) : 0;
  const long long sum_fk = block_sum_i(fk, s_redi);
  const long long sum_fr = block_sum_i(fr, s_redi);

  // ---- chi = sum_{j>=1} (j+1) exp(-j^2 a), a = Delta_2^2 / (4 tau^2) ------
  const double tb = (double)P.tau[bh];
  const bool have_tau = nq > 0 && tb > 0.0;
  double chi = nan;
  if (have_tau) {
    const double d2 = (double)p05;
    bool inf = !(d2 > 0.0);
    double a = 0.0, M = 0.0;
    if (!inf) {
      a = d2 * d2 / (4.0 * tb * tb);
      M = floor(__dsqrt_rn(745.0 / a));  // last term before exp underflows
      inf = M > 1.0e6;
    }
    if (inf) {
      chi = __builtin_huge_val();
    } else {
      double part = 0.0;
      const int Mi = (int)M;
      for (int j = 1 + tid; j <= Mi; j += kHeadThreads) part += (double)(j + 1) * exp(-((double)j * (double)j) * a);
      chi = block_sum(part, s_red);
    }
  }

  if (tid != 0) return;
  ugbs_bai_head hd;
  hd.n_tiles = n;
  hd.n_q = nq;
  hd.pad[0] = hd.pad[1] = 0;
  hd.r_mean = r_mean;
  hd.r_cv = r_cv;
  hd.delta2_p05 = (double)p05;
  hd.delta2_p50 = (double)s_pick[1];
  hd.pi2 = (double)n_below / n;
  hd.tau = tb;
  const int ns = P.n_s;
  hd.mc_err_k = ns > 0 ? (double)sum_fk / ((double)n * ns) : nan;
  hd.mc_err_rk = ns > 0 ? (double)sum_fr / ((double)n * ns) : nan;
  hd.sigma_q = sq;
  hd.gamma_q = nq > 0 ? gamma : nan;
  hd.band_mass = nq > 0 ? (double)n_band / n : nan;
  hd.chi = hd.eps_bar = hd.C_q = hd.vbar_gamma = hd.bound = hd.bound_band = nan;
  if (have_tau) {
    double eb = __builtin_huge_val();
    if (!__builtin_isinf(chi)) {
      const double x = (double)(kRho - 1) * s.k * (double)p05;
      eb = chi + (1.0 + chi) * exp(-(x * x) / (4.0 * tb * tb));
    }
    const double bandt = sqrt(2.0) * beta * gamma / tb * std_normal_pdf(gamma * (1.0 - beta) / (sqrt(2.0) * tb));
    const double cq = fmin(fmin(1.0, (1.0 + eb) / 2.0), bandt + eb);
    hd.chi = chi;
    hd.eps_bar = eb;
    hd.C_q = cq;
    hd.vbar_gamma = std_normal_cdf(-gamma / (sqrt(2.0) * tb));
    hd.bound = fmin(q, 1.0 - q) * cq + hd.pi2;
    hd.bound_band = 0.5 * hd.band_mass * cq + hd.pi2;
  }
  // regret: mean per-tile V over the oracle-best nq tiles minus the router's
  hd.mc_regret = (ns > 0 && nq > 0) ? ((double)top / ns - (double)rsig / ns) / n : nan;
  *out = hd;
}

}  // namespace

hipError_t launch_noise_scale(const Shape& s, const double* rough, float* tau, hipStream_t stream) {
  noise_kernel<<<s.B * s.H, 64, 0, stream>>>(s, rough, tau);
  return hipGetLastError();
}

hipError_t launch_bai_tiles(const Shape& s, const float* scores, const float* tau,
                            const float* z, int n_s, ugbs_bai_tile* tiles, hipStream_t stream) {
  TileParams P{s, scores, tau, z, n_s, tiles};
  const size_t smem = (size_t)kBaiWaves * UGBS_MAX_BLOCKS * sizeof(uint64_t);
  if (smem > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)bai_tile_kernel,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
  }
  const int n_units = s.B * s.H * s.T;
  const int n_wg = (n_units + kBaiWaves - 1) / kBaiWaves;
  const int grid = ((n_wg + 7) / 8) * 8;
  bai_tile_kernel<<<grid, 64 * kBaiWaves, smem, stream>>>(P);
  return hipGetLastError();
}

hipError_t launch_bai_heads(const Shape& s, const ugbs_bai_tile* tiles, const float* tau, int n_s,
                            ugbs_bai_head* heads, hipStream_t stream) {
  HeadParams P{s, tiles, tau, n_s, heads};
  bai_head_kernel<<<s.B * s.H, kHeadThreads, 0, stream>>>(P);
  return hipGetLastError();
}

}  // namespace ugbs
