// Internal declarations shared by the HIP translation units of libugbs.
// Device helpers here are the GPU path's own; nothing is shared with the
// reference oracle.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ugbs.h"

namespace ugbs {

constexpr int kBlock = UGBS_BLOCK;

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

// Validated problem with derived sizes; passed by value to launchers.
struct Shape {
  int B, H, Hkv, G, N, d, NB, T, k, W, backbone, rho;  // W = rho k
  double q;
  float scale;
};

// Launchers (each enqueues on `stream` and returns hipGetLastError()).
hipError_t launch_block_meta(const Shape& s, const uint16_t* K, uint16_t* meta,
                             hipStream_t stream);
hipError_t launch_score_select(const Shape& s, const uint16_t* Q, const uint16_t* meta,
                               const float* scores_in, float* scores_out,
                               int32_t* idx_sorted, float* sigma, void* workspace,
                               hipStream_t stream);
// Quest tile scores on the vector ALU (the literal per-channel form), into a
// [B, H, T, N_B] fp32 tensor.
hipError_t launch_quest_valu(const Shape& s, const uint16_t* Q, const uint16_t* meta, float* scores_out,
                             hipStream_t stream);
// Bytes of packed candidate scores the score kernel writes into the workspace
// when the caller supplies neither scores_in nor scores_out.
size_t score_scratch_bytes(const Shape& s);
hipError_t launch_route(const Shape& s, int n_pop, int n_trig, const float* sigma,
                        const int32_t* idx_sorted, int32_t* kv_idx, float* sigma_bar,
                        float* tau, uint8_t* trigger, void* workspace, hipStream_t stream);
// The route without a caller's workspace: its sections live in a static
// device array of kRouteScratchBytes per GPU (route.hip); route_scratch gives
// the current device's address of it.
constexpr size_t kRouteScratchBytes = UGBS_ROUTE_SCRATCH_BYTES;
hipError_t route_scratch(void** ptr);
// Per-row selection into tile bitmaps, and attention over bitmaps.
hipError_t launch_select_rows(const Shape& s, const uint16_t* Q, const uint16_t* meta,
                              const float* row_scores, const uint8_t* trigger, uint32_t* bitmap,
                              hipStream_t stream);
hipError_t launch_attend_bitmap(const Shape& s, const uint16_t* Q, const uint16_t* K,
                                const uint16_t* V, const uint32_t* bitmap, uint16_t* O,
                                hipStream_t stream);
// Appendix D diagnostics.
hipError_t launch_row_roughness(const Shape& s, const uint16_t* Q, const uint16_t* meta,
                                double* rough, hipStream_t stream);
hipError_t launch_noise_scale(const Shape& s, const double* rough, float* tau, hipStream_t stream);
hipError_t launch_bai_tiles(const Shape& s, const float* scores, const float* tau,
                            const float* z, int n_s, ugbs_bai_tile* tiles, hipStream_t stream);
hipError_t launch_bai_heads(const Shape& s, const ugbs_bai_tile* tiles, const float* tau, int n_s,
                            ugbs_bai_head* heads, hipStream_t stream);
hipError_t launch_attend(const Shape& s, const uint16_t* Q, const uint16_t* K,
                         const uint16_t* V, const int32_t* kv_idx, int kv_width,
                         uint16_t* O, hipStream_t stream);
// Attention with the selection done in the kernel: scores (full layout) or
// the packed rows in `workspace`; trigger flags or the ones ugbs_route left
// in `workspace`.
hipError_t launch_attend_select(const Shape& s, const uint16_t* Q, const uint16_t* K,
                                const uint16_t* V, const float* scores, const uint8_t* trigger,
                                const void* workspace, uint16_t* O, hipStream_t stream);

// Route workspace layout: sigma_bar [B*T] f32 | tau [B] f32 | trigger [B*T] u8.
inline size_t ws_align(size_t x) { return (x + 255) & ~size_t(255); }
inline size_t ws_sigma_bar_off(const Shape&) { return 0; }
inline size_t ws_tau_off(const Shape& s) { return ws_align(sizeof(float) * size_t(s.B) * s.T); }
inline size_t ws_trigger_off(const Shape& s) {
  return ws_tau_off(s) + ws_align(sizeof(float) * size_t(s.B));
}
inline size_t ws_route_total(const Shape& s) { return ws_trigger_off(s) + ws_align(size_t(s.B) * s.T); }
// One workspace serves the whole layer: the route sections first, then the
// packed candidate scores of the score kernel (which ugbs_attend_select may
// read after ugbs_route has written the trigger flags).
inline size_t ws_scores_off(const Shape& s) { return ws_route_total(s); }
inline size_t ws_total(const Shape& s) { return ws_scores_off(s) + ws_align(score_scratch_bytes(s)); }

// Offset (floats) of the packed candidate row of unit (bh, t) in the packed
// score section: rows of one (b, h) follow each other, row t holding the
// t - 1 scores of blocks 1..t-1.
__host__ __device__ inline size_t packed_row(int bh, int t, int T) {
  const size_t tri = (T >= 2) ? (size_t)(T - 1) * (T - 2) / 2 : 0;
  const size_t off = (t >= 2) ? (size_t)(t - 1) * (t - 2) / 2 : 0;
  return (size_t)bh * tri + off;
}

// Work-unit ordering used by the per-(tile, head) kernels: kv head by kv
// head, heaviest tile first (work grows with t), sibling query heads
// adjacent.  The hardware deals consecutive workgroup ids round-robin to the
// 8 XCDs, so taking the id as the unit index gives every XCD the same mix of
// heavy and light tiles, with all XCDs on the same kv head (its metadata is
// read by each XCD's L2).  Remapping ids to contiguous per-XCD ranges keeps
// a kv head on one XCD, but is balanced only when a range holds whole kv
// heads: with 7 or 8 query heads per kv head, or 2 kv heads, it left one XCD
// the heaviest tiles (scoring 1.4x, per-row selection 1.3-1.5x slower
// measured).
struct Unit {
  int b, h, t;
};

__device__ __forceinline__ Unit unit_of(int u, const Shape& s) {
  Unit r;
  const int g = u % s.G;
  int rest = u / s.G;
  const int tr = rest % s.T;
  rest /= s.T;
  const int kvh = rest % s.Hkv;
  r.b = rest / s.Hkv;
  r.t = s.T - 1 - tr;
  r.h = kvh * s.G + g;
  return r;
}

}  // namespace ugbs
