// Stage 4: head mean of sigma, per-layer quantile trigger and padded
// expansion (A.7-A.9; Eq. (trigger)).
//
// The quantile couples every tile of a sequence, so this is the pipeline's
// one device-wide step.  It runs as two launches:
//   route_stats : one 1024-thread workgroup per sequence.  sigma_bar[t] is
//                 the fp32 sum over heads in head order, divided by H.  The
//                 n_trig-th smallest sigma_bar of the population is found by
//                 a most-significant-bit-first radix descent (sigma_bar >= 0,
//                 so its bit pattern is order preserving); trigger[t] is
//                 (t in P) and sigma_bar[t] <= tau.
//   route_patch : one thread per kv_idx slot; slots k..2k-1 of tiles that
//                 do not trigger become the sentinel N_B.
// n_pop and n_trig = ceil(q n_pop) depend only on N, k and q and are
// computed on the host, so no device-to-host synchronisation is needed.
#include "ugbs_internal.h"

namespace ugbs {
namespace {

constexpr int kStatsThreads = 1024;

__device__ __forceinline__ bool in_population(int t, int k) {
  const int nf = (t == 0) ? 1 : 2;
  const int nc = (t >= 1) ? t - 1 : 0;
  return nc > k - nf;
}

struct RouteParams {
  Shape s;
  int n_trig;
  const float* sigma;
  const int32_t* idx_sorted;
  int32_t* kv_idx;
  float* sigma_bar;   // optional user copy
  float* tau;         // optional user copy
  uint8_t* trigger;   // optional user copy
  float* ws_sigma_bar;
  float* ws_tau;
  uint8_t* ws_trigger;
};

__global__ void __launch_bounds__(kStatsThreads) route_stats_kernel(RouteParams P) {
  __shared__ uint32_t s_key[UGBS_MAX_BLOCKS];
  __shared__ int s_cnt[2][kStatsThreads / 64];
  __shared__ float s_tau;
  const Shape& s = P.s;
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;

  for (int t = tid; t < s.T; t += kStatsThreads) {
    float sb = -1.0f;
    uint32_t key = 0xffffffffu;
    if (in_population(t, s.k)) {
#pragma clang fp contract(off)
      float acc = 0.0f;
      for (int h = 0; h < s.H; ++h) acc += P.sigma[((size_t)b * s.H + h) * s.T + t];
      sb = __fdiv_rn(acc, (float)s.H);
      if (sb == 0.0f) sb = 0.0f;
      key = __float_as_uint(sb);
    }
    s_key[t] = key;
    P.ws_sigma_bar[(size_t)b * s.T + t] = sb;
    if (P.sigma_bar) P.sigma_bar[(size_t)b * s.T + t] = sb;
  }
  __syncthreads();

  float tau = -1.0f;
  if (P.n_trig > 0) {
    // smallest v with #{key <= v} >= n_trig
    uint32_t ans = 0;
    for (int bit = 31; bit >= 0; --bit) {
      const uint32_t c = ans | ((1u << bit) - 1u);
      int local = 0;
      for (int t = tid; t < s.T; t += kStatsThreads) local += (s_key[t] <= c) ? 1 : 0;
      // local is 0..2 for T <= 2048; wave-reduce with two ballots
      const int wsum = __popcll(__ballot(local & 1)) + 2 * __popcll(__ballot(local & 2));
      const int buf = bit & 1;
      if (lane == 0) s_cnt[buf][wv] = wsum;
      __syncthreads();
      int cnt = 0;
#pragma unroll
      for (int w = 0; w < kStatsThreads / 64; ++w) cnt += s_cnt[buf][w];
      if (cnt < P.n_trig) ans |= (1u << bit);
    }
    tau = __uint_as_float(ans);
  }
  if (tid == 0) s_tau = tau;
  __syncthreads();
  tau = s_tau;
  if (tid == 0) {
    P.ws_tau[b] = tau;
    if (P.tau) P.tau[b] = tau;
  }
  for (int t = tid; t < s.T; t += kStatsThreads) {
    const uint8_t trig = (P.n_trig > 0 && s_key[t] != 0xffffffffu &&
                          __uint_as_float(s_key[t]) <= tau) ? 1 : 0;
    P.ws_trigger[(size_t)b * s.T + t] = trig;
    if (P.trigger) P.trigger[(size_t)b * s.T + t] = trig;
  }
}

__global__ void __launch_bounds__(256) route_patch_kernel(RouteParams P, long n_slots,
                                                          int in_place) {
  const Shape& s = P.s;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n_slots;
       i += (long)gridDim.x * blockDim.x) {
    const int slot = (int)(i % s.W);
    const long row = i / s.W;                 // (b*H + h)*T + t
    const int t = (int)(row % s.T);
    const int b = (int)(row / ((long)s.T * s.H));
    const bool keep = slot < s.k || P.ws_trigger[(size_t)b * s.T + t];
    if (in_place) {
      if (!keep) P.kv_idx[i] = s.NB;
    } else {
      P.kv_idx[i] = keep ? P.idx_sorted[i] : s.NB;
    }
  }
}

}  // namespace

hipError_t launch_route(const Shape& s, int n_pop, int n_trig, const float* sigma,
                        const int32_t* idx_sorted, int32_t* kv_idx, float* sigma_bar,
                        float* tau, uint8_t* trigger, void* workspace, hipStream_t stream) {
  (void)n_pop;
  RouteParams P;
  P.s = s;
  P.n_trig = n_trig;
  P.sigma = sigma;
  P.idx_sorted = idx_sorted;
  P.kv_idx = kv_idx;
  P.sigma_bar = sigma_bar;
  P.tau = tau;
  P.trigger = trigger;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  P.ws_sigma_bar = reinterpret_cast<float*>(ws + ws_sigma_bar_off(s));
  P.ws_tau = reinterpret_cast<float*>(ws + ws_tau_off(s));
  P.ws_trigger = ws + ws_trigger_off(s);
  route_stats_kernel<<<s.B, kStatsThreads, 0, stream>>>(P);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !kv_idx) return e;  // no lists to patch: flags only
  const long n_slots = (long)s.B * s.H * s.T * s.W;
  long blocks = (n_slots + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  route_patch_kernel<<<(unsigned)blocks, 256, 0, stream>>>(P, n_slots,
                                                           idx_sorted == kv_idx ? 1 : 0);
  return hipGetLastError();
}

}  // namespace ugbs
