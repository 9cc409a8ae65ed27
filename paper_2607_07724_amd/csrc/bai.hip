// Appendix D diagnostics: sigma read as a best-arm identification index.
//
// noise_kernel     tau[b, h] from the per-unit row roughness the score kernel
//                  produces in its roughness mode (recipe step 3: adjacent
//                  rows of a tile differ by two independent noise draws, so
//                  the mean squared difference is 2 tau^2).
// bai_tile_kernel  per (b, h, t): the sorted top rho k - |F| + 1 candidate
//                  scores (same key order as the selection kernel: score
//                  descending, lower block first), the gaps g, G, r and
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
// fp32(s + fp32(tau z)), a multiply and an add each rounded (the kernels
// switch floating-point contraction off, so no fused multiply-add); the head
// sums of r run in tile order in fp64, one thread, so they equal a
// left-to-right sum.
#include <math.h>

#include "select_common.h"

namespace ugbs {
namespace {

constexpr int kBaiUnits = 4;   // query heads of one tile per workgroup (one wave each)
constexpr int kBaiSlots = UGBS_MAX_BLOCKS_ROWS / 64;
constexpr int kHeadThreads = 256;

struct TileParams {
  Shape s;
  const float* scores;  // [B, H, T, N_B]
  const float* tau;     // [B, H]
  const float* zT;      // [N_B, n_s]: sample s of block b at zT[b * n_s + s]
  int n_s;
  ugbs_bai_tile* tiles; // [B, H, T]
  int n_hg;             // head groups per tile, ceil(H / kBaiUnits)
  int n_wg;             // B * T * n_hg
  int sel_bytes;        // per-unit LDS: sort buffer, then the masked score row
  int top_bytes;        // per-unit LDS: the top R' (value, position)
};

__device__ __forceinline__ float wave_min_f(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fminf(x, __shfl_xor(x, o));
  return x;
}

// One workgroup per (b, t, group of up to 4 query heads): all units share
// the candidate set C(t) and so every draw z[b', s].
//
// Phase 1, wave u = unit u: the sorted top R' + 1 (keys as in the
// selection kernel), the gaps and the smallest secondary spacing; then, in
// LDS, the top R' as (value, position) and the unit's score row with the top
// R' masked to -inf (the candidates outside the expanded set).
//
// Phase 2, Monte Carlo with one sample per lane (wave w takes samples w*64 +
// lane + 256 i): for every unit, mu = fp32(s + fp32(tau z)) is maxed over
// the masked row (max over the candidates outside the top R'), then the top
// R' are visited in rank order: the min over ranks < m, the max over ranks
// m..R'-1, and the count of ranks < R' whose mu beats the outside max.  The
// draws of a block are read once per workgroup-sample and used by every
// unit; no cross-lane reduction is needed until the failure counts.
__global__ void __launch_bounds__(64 * kBaiUnits) bai_tile_kernel(TileParams P) {
#pragma clang fp contract(off)
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int s_fail[kBaiUnits][kBaiUnits][2];
  const Shape& s = P.s;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int id = blockIdx.x;
  if (id >= P.n_wg) return;
  const int hg = id % P.n_hg;
  const int rest = id / P.n_hg;
  const int t = s.T - 1 - rest % s.T;
  const int b = rest / s.T;
  const int h0 = hg * kBaiUnits;
  const int n_act = min(kBaiUnits, s.H - h0);
  const int nf = (t == 0) ? 1 : 2;
  const int nc = (t >= 1) ? t - 1 : 0;
  const int m = s.k - nf;              // kept non-forced slots
  const int Rp = s.W - nf;             // non-forced slots after expansion (rho k - |F|)
  if (nc < Rp + 1 || nc <= m) {        // outside the diagnostic mask (uniform: depends on t)
    if (w < n_act && lane == 0) {
      const float nan = __builtin_nanf("");
      P.tiles[((size_t)b * s.H + h0 + w) * s.T + t] = ugbs_bai_tile{nan, nan, nan, nan, nan, 0, 0, 0};
    }
    return;
  }
  auto sel_of = [&](int u) { return smem + (size_t)u * P.sel_bytes; };
  auto top_of = [&](int u) { return smem + (size_t)kBaiUnits * P.sel_bytes + (size_t)u * P.top_bytes; };

  // ---- phase 1: order statistics of unit w ---------------------------------
  float g = 0.f, G = 0.f, r = 0.f, sg = 0.f, d2 = 0.f;
  if (w < n_act) {
    const int h = h0 + w;
    uint64_t* s_sel = reinterpret_cast<uint64_t*>(sel_of(w));
    const float* src = P.scores + (((size_t)b * s.H + h) * s.T + t) * s.NB + 1;
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
    float dm = __builtin_huge_valf();
    for (int j = lane; j < Rp; j += 64)
      if (j != m - 1) dm = fminf(dm, cs(j) - cs(j + 1));
    d2 = wave_min_f(dm);
    if (Rp < 2) d2 = __builtin_nanf("");  // no spacing besides the cut (rho = 1, m = 1)
    {
      const float c0 = cs(0), cm1 = cs(m - 1), cm = cs(m), cR = cs(Rp);
      g = cm1 - cm;
      G = cm1 - cR;
      r = c0 - cm;
      sg = (r == 0.0f) ? 0.0f : __fdiv_rn(g, r);
    }
    // the top R' in rank order, and the row with them masked out
    float* tv = reinterpret_cast<float*>(top_of(w));
    int32_t* tp = reinterpret_cast<int32_t*>(tv + Rp);
    for (int j = lane; j < Rp; j += 64) {
      const uint64_t e = s_sel[j];
      tv[j] = key_value((uint32_t)(e >> 32));
      tp[j] = (int32_t)(0xffffffffu - (uint32_t)e);
    }
    const uint64_t thr_r = s_sel[Rp - 1];
    wave_lds_sync();  // every read of the sort buffer is done before the row overwrites it
    float* row = reinterpret_cast<float*>(s_sel);
#pragma unroll
    for (int sl = 0; sl < kBaiSlots; ++sl) {
      const int p = 64 * sl + lane;
      if (sl < nslots && p < nc) {
        const uint64_t k64 = ((uint64_t)keys[sl] << 32) | (0xffffffffu - (uint32_t)p);
        row[p] = (k64 >= thr_r) ? -__builtin_huge_valf() : key_value(keys[sl]);
      }
    }
    const int nc8 = (nc + 7) & ~7;
    if (lane < nc8 - nc) row[nc + lane] = -__builtin_huge_valf();
  }
  __syncthreads();

  // ---- phase 2: Monte Carlo, one sample per lane ---------------------------
  float tau_u[kBaiUnits];
#pragma unroll
  for (int u = 0; u < kBaiUnits; ++u)
    tau_u[u] = (u < n_act && P.n_s > 0) ? P.tau[(size_t)b * s.H + h0 + u] : 0.f;  // tau may be NULL without samples
  int fk_acc[kBaiUnits] = {0, 0, 0, 0}, fr_acc[kBaiUnits] = {0, 0, 0, 0};
  const int nc8 = (nc + 7) & ~7;
  const size_t ns = (size_t)P.n_s;
  for (int s0 = 64 * w; s0 < P.n_s; s0 += 64 * kBaiUnits) {
    const int smp = s0 + lane;
    const bool live = smp < P.n_s;
    // draw of block b' for this lane's sample: (zT + b' n_s)[smp_c], with the
    // block offset uniform (scalar base) and the sample offset per lane
    const int smp_c = live ? smp : P.n_s - 1;
    auto zdraw = [&](int blk) { return (P.zT + (size_t)blk * ns)[smp_c]; };
    float mx_out[kBaiUnits];
#pragma unroll
    for (int u = 0; u < kBaiUnits; ++u) mx_out[u] = -__builtin_huge_valf();
    // candidates outside the top R' (the masked row: the top R' and the
    // padding read -inf, which no draw changes); the next 8 draws are in
    // flight while the current 8 are used
    float zn[8];
    auto load8 = [&](int p0, float (&zz)[8]) {
#pragma unroll
      for (int i = 0; i < 8; ++i) zz[i] = zdraw(min(1 + p0 + i, s.NB - 1));
    };
    load8(0, zn);
    for (int p = 0; p < nc8; p += 8) {
      float zz[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) zz[i] = zn[i];
      if (p + 8 < nc8) load8(p + 8, zn);
#pragma unroll
      for (int u = 0; u < kBaiUnits; ++u) {
        if (u < n_act) {
          const float* rw = reinterpret_cast<const float*>(sel_of(u)) + p;
          const float4 ra = *reinterpret_cast<const float4*>(rw);
          const float4 rb = *reinterpret_cast<const float4*>(rw + 4);
          const float rv[8] = {ra.x, ra.y, ra.z, ra.w, rb.x, rb.y, rb.z, rb.w};
          float mx = mx_out[u];
#pragma unroll
          for (int i = 0; i < 8; ++i) mx = fmaxf(mx, rv[i] + tau_u[u] * zz[i]);
          mx_out[u] = mx;
        }
      }
    }
    // the top R' in rank order, 8 draws at a time: ranks < m (min, and the
    // count above the outside max), then ranks m..R'-1 (max, and the count)
#pragma unroll
    for (int u = 0; u < kBaiUnits; ++u) {
      if (u < n_act) {
        const float* tv = reinterpret_cast<const float*>(top_of(u));
        const int32_t* tp = reinterpret_cast<const int32_t*>(tv + Rp);
        const float tu = tau_u[u], mo = mx_out[u];
        float mn_in = __builtin_huge_valf(), mx_mid = -__builtin_huge_valf();
        int above = 0;
        for (int j0 = 0; j0 < Rp; j0 += 8) {
          float zz[8];
#pragma unroll
          for (int i = 0; i < 8; ++i)
            zz[i] = zdraw(1 + __builtin_amdgcn_readfirstlane(tp[min(j0 + i, Rp - 1)]));
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const int j = j0 + i;
            if (j < Rp) {
              const float x = tv[j] + tu * zz[i];
              if (j < m) mn_in = fminf(mn_in, x);
              else mx_mid = fmaxf(mx_mid, x);
              above += x > mo;
            }
          }
        }
        const bool fail_k = !(mn_in > fmaxf(mx_mid, mo));
        const bool fail_rk = above < m;
        fk_acc[u] += __popcll(__ballot(live && fail_k));
        fr_acc[u] += __popcll(__ballot(live && fail_rk));
      }
    }
  }
  if (lane == 0) {
#pragma unroll
    for (int u = 0; u < kBaiUnits; ++u) {
      s_fail[w][u][0] = fk_acc[u];
      s_fail[w][u][1] = fr_acc[u];
    }
  }
  __syncthreads();
  if (w < n_act && lane == 0) {
    int fk = 0, fr = 0;
    for (int v = 0; v < kBaiUnits; ++v) {
      fk += s_fail[v][w][0];
      fr += s_fail[v][w][1];
    }
    P.tiles[((size_t)b * s.H + h0 + w) * s.T + t] = ugbs_bai_tile{g, G, r, sg, d2, fk, fr, 1};
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
  __shared__ float s_sig[UGBS_MAX_BLOCKS_ROWS], s_g[UGBS_MAX_BLOCKS_ROWS], s_r[UGBS_MAX_BLOCKS_ROWS],
      s_d2[UGBS_MAX_BLOCKS_ROWS];
  __shared__ int s_dk[UGBS_MAX_BLOCKS_ROWS];
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
    int base = 0;
    for (int t0 = 0; t0 < s.T; t0 += 64) {
      const int t = t0 + tid;
      ugbs_bai_tile x;
      const bool v = t < s.T && (x = tl[t], x.valid != 0);
      const uint64_t mk = __ballot(v);
      if (v) {
        const int i = base + lanes_below(mk);
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
      const double x = (double)(s.rho - 1) * s.k * (double)p05;
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
                            const float* zT, int n_s, ugbs_bai_tile* tiles, hipStream_t stream) {
  TileParams P{};
  P.s = s;
  P.scores = scores;
  P.tau = tau;
  P.zT = zT;
  P.n_s = n_s;
  P.tiles = tiles;
  P.n_hg = (s.H + kBaiUnits - 1) / kBaiUnits;
  P.n_wg = s.B * s.T * P.n_hg;
  // sort buffer for the top R' + 1 (a power of two of 8-byte entries; only
  // tiles with R' + 1 <= |C(t)| <= N_B - 2 are sorted), reused for the
  // masked score row (N_B floats, padded to a multiple of 8)
  const int r1 = s.W - 1;
  int n2 = 2;
  while (n2 < r1 && n2 < s.NB) n2 <<= 1;
  const int sel = 8 * n2 > 4 * (s.NB + 8) ? 8 * n2 : 4 * (s.NB + 8);
  P.sel_bytes = (sel + 15) & ~15;
  P.top_bytes = (8 * s.W + 15) & ~15;
  const size_t smem = (size_t)kBaiUnits * (P.sel_bytes + P.top_bytes);
  if (smem > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)bai_tile_kernel,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
  }
  const int grid = ((P.n_wg + 7) / 8) * 8;
  bai_tile_kernel<<<grid, 64 * kBaiUnits, smem, stream>>>(P);
  return hipGetLastError();
}

hipError_t launch_bai_heads(const Shape& s, const ugbs_bai_tile* tiles, const float* tau, int n_s,
                            ugbs_bai_head* heads, hipStream_t stream) {
  HeadParams P{s, tiles, tau, n_s, heads};
  bai_head_kernel<<<s.B * s.H, kHeadThreads, 0, stream>>>(P);
  return hipGetLastError();
}

}  // namespace ugbs
