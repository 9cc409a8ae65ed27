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
//   route_patch : one wave per kv_idx row; slots k..W-1 of tiles that do
//                 not trigger become the sentinel N_B.
// n_pop and n_trig = ceil(q n_pop) depend only on N, k and q and are
// computed on the host, so no device-to-host synchronisation is needed.
#include <mutex>

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
      // fp32 sum in head order; the loads of 8 heads are issued together
      // before their adds (the order of the adds is unchanged)
      const float* col = P.sigma + (size_t)b * s.H * s.T + t;
      float acc = 0.0f;
      for (int h0 = 0; h0 < s.H; h0 += 8) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (h0 + j < s.H) ? col[(size_t)(h0 + j) * s.T] : 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (h0 + j < s.H) acc += v[j];
      }
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
      // local is 0..4 for T <= 4096 (1024 threads); wave-reduce bit by bit
      static_assert(UGBS_MAX_BLOCKS <= 7 * kStatsThreads, "per-thread count must fit in 3 bits");
      const int wsum = __popcll(__ballot(local & 1)) + 2 * __popcll(__ballot(local & 2)) +
                       4 * __popcll(__ballot(local & 4));
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

// One wave per kv_idx row (b, h, t), rows grid-strided.  In place only the
// slots k..W-1 of rows whose tile does not trigger are written.
__global__ void __launch_bounds__(256) route_patch_kernel(RouteParams P, long n_rows,
                                                          int in_place) {
  const Shape& s = P.s;
  const int lane = threadIdx.x & 63;
  const long wave0 = (long)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
  const long n_waves = (long)gridDim.x * (blockDim.x / 64);
  for (long row = wave0; row < n_rows; row += n_waves) {
    const int t = (int)(row % s.T);
    const int b = (int)(row / ((long)s.T * s.H));
    const bool trig = P.ws_trigger[(size_t)b * s.T + t] != 0;
    int32_t* dst = P.kv_idx + row * s.W;
    if (in_place) {
      if (trig) continue;
      for (int slot = s.k + lane; slot < s.W; slot += 64) dst[slot] = s.NB;
    } else {
      const int32_t* src = P.idx_sorted + row * s.W;
      for (int slot = lane; slot < s.W; slot += 64) dst[slot] = (slot < s.k || trig) ? src[slot] : s.NB;
    }
  }
}

// Route sections (sigma_bar | tau | trigger) of ugbs_route_noalloc, in device
// memory the library owns: one copy of this array per GPU, held until the
// process ends.  Host code must not pass `scratch` itself to a kernel (on the
// host it names a stand-in, not a device address); the per-device address
// comes from hipGetSymbolAddress below.
static __device__ __align__(256) unsigned char scratch[kRouteScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch`, per device

}  // namespace

// Device address of the current device's `scratch`, looked up once per
// device with that device current.
hipError_t route_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

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
  const long n_rows = (long)s.B * s.H * s.T;
  long blocks = (n_rows + 3) / 4;
  if (blocks > 65536) blocks = 65536;
  route_patch_kernel<<<(unsigned)blocks, 256, 0, stream>>>(P, n_rows,
                                                           idx_sorted == kv_idx ? 1 : 0);
  return hipGetLastError();
}

}  // namespace ugbs
