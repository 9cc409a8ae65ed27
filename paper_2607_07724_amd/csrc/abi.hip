// extern "C" boundary of libugbs: argument validation, derived sizes and
// dispatch to the kernel launchers.  Every check runs before anything is
// enqueued; nothing here allocates, frees or synchronises.
#include <cmath>
#include <cstdint>

#include "ugbs_internal.h"

namespace {

using ugbs::Shape;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int make_shape(const ugbs_problem* p, Shape* s) {
  if (!p) return UGBS_ERR_NULL;
  if (p->batch < 1 || p->n_heads < 1 || p->n_kv_heads < 1 || p->n_heads % p->n_kv_heads)
    return UGBS_ERR_SHAPE;
  if (p->head_dim != 64 && p->head_dim != 128 && p->head_dim != 256) return UGBS_ERR_SHAPE;
  if (p->block != UGBS_BLOCK) return UGBS_ERR_SHAPE;
  if (p->seq_len < UGBS_BLOCK || p->seq_len % UGBS_BLOCK) return UGBS_ERR_SHAPE;
  const int NB = p->seq_len / UGBS_BLOCK;
  if (NB > UGBS_MAX_BLOCKS) return UGBS_ERR_SHAPE;
  // unit counts index grids with int; element counts use size_t
  if ((int64_t)p->batch * p->n_heads * NB > (int64_t)INT32_MAX / 2) return UGBS_ERR_SHAPE;
  if (p->backbone != UGBS_KMEAN && p->backbone != UGBS_QUEST) return UGBS_ERR_BACKBONE;
  const int rho = p->rho == 0 ? 2 : p->rho;
  if (rho < 1 || rho > UGBS_MAX_RHO) return UGBS_ERR_BUDGET;
  if (p->k_budget < 3 || (int64_t)rho * p->k_budget > UGBS_MAX_KV_WIDTH) return UGBS_ERR_BUDGET;
  if (!(p->q >= 0.0 && p->q <= 1.0)) return UGBS_ERR_Q;
  if (!std::isfinite(p->softmax_scale) || p->softmax_scale < 0.0f) return UGBS_ERR_SCALE;
  s->B = p->batch;
  s->H = p->n_heads;
  s->Hkv = p->n_kv_heads;
  s->G = p->n_heads / p->n_kv_heads;
  s->N = p->seq_len;
  s->d = p->head_dim;
  s->NB = NB;
  s->T = NB;
  s->k = p->k_budget;
  s->W = rho * p->k_budget;
  s->rho = rho;
  s->backbone = p->backbone;
  s->q = p->q;
  s->scale = p->softmax_scale > 0.0f ? p->softmax_scale : 1.0f / std::sqrt((float)p->head_dim);
  return UGBS_OK;
}

// Tiles with more non-forced candidates (t - 1) than kept slots (k - |F|).
int population_size(const Shape& s) {
  int n = 0;
  for (int t = 0; t < s.T; ++t) {
    const int nf = (t == 0) ? 1 : 2;
    const int nc = (t >= 1) ? t - 1 : 0;
    if (nc > s.k - nf) ++n;
  }
  return n;
}

int hip_status(hipError_t e) { return e == hipSuccess ? UGBS_OK : UGBS_ERR_HIP; }

}  // namespace

extern "C" {

int ugbs_abi_version(void) { return UGBS_ABI_VERSION; }

const char* ugbs_status_string(int status) {
  switch (status) {
    case UGBS_OK: return "ok";
    case UGBS_ERR_NULL: return "a required pointer is NULL";
    case UGBS_ERR_SHAPE: return "invalid shape (batch, heads, seq_len, head_dim, block or kv_width)";
    case UGBS_ERR_BUDGET: return "k_budget < 3, rho outside [1, UGBS_MAX_RHO] or rho * k_budget > UGBS_MAX_KV_WIDTH";
    case UGBS_ERR_Q: return "q outside [0, 1]";
    case UGBS_ERR_BACKBONE: return "unknown backbone";
    case UGBS_ERR_ALIGN: return "pointer misaligned";
    case UGBS_ERR_WORKSPACE: return "workspace missing or too small";
    case UGBS_ERR_HIP: return "HIP launch failed";
    case UGBS_ERR_SCALE: return "softmax_scale negative or not finite";
    case UGBS_ERR_SCRATCH: return "problem exceeds the static scratch of ugbs_route_noalloc";
    default: return "unknown status";
  }
}

size_t ugbs_workspace_bytes(const ugbs_problem* p) {
  Shape s;
  if (make_shape(p, &s) != UGBS_OK) return 0;
  return ugbs::ws_total(s);
}

int ugbs_block_meta(const ugbs_problem* p, const void* K, void* meta, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (!K || !meta) return UGBS_ERR_NULL;
  if (!aligned(K, 16) || !aligned(meta, 16)) return UGBS_ERR_ALIGN;
  return hip_status(ugbs::launch_block_meta(s, static_cast<const uint16_t*>(K),
                                            static_cast<uint16_t*>(meta),
                                            static_cast<hipStream_t>(stream)));
}

int ugbs_score_select(const ugbs_problem* p, const void* Q, const void* meta,
                      const float* scores_in, float* scores_out, int32_t* idx_sorted,
                      float* sigma, void* workspace, size_t workspace_bytes, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (!Q || !meta || !sigma) return UGBS_ERR_NULL;
  const bool needs_ws = !scores_in && !scores_out;
  if (needs_ws && (!workspace || workspace_bytes < ugbs::ws_total(s))) return UGBS_ERR_WORKSPACE;
  if (!aligned(Q, 16) || !aligned(meta, 16) || !aligned(idx_sorted, 4) || !aligned(sigma, 4) ||
      !aligned(scores_in, 4) || !aligned(scores_out, 4) || (needs_ws && !aligned(workspace, 256)))
    return UGBS_ERR_ALIGN;
  return hip_status(ugbs::launch_score_select(
      s, static_cast<const uint16_t*>(Q), static_cast<const uint16_t*>(meta), scores_in,
      scores_out, idx_sorted, sigma, needs_ws ? workspace : nullptr,
      static_cast<hipStream_t>(stream)));
}

int ugbs_quest_scores_valu(const ugbs_problem* p, const void* Q, const void* meta, float* scores_out,
                           void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (s.backbone != UGBS_QUEST) return UGBS_ERR_BACKBONE;
  if (!Q || !meta || !scores_out) return UGBS_ERR_NULL;
  if (!aligned(Q, 16) || !aligned(meta, 16) || !aligned(scores_out, 4)) return UGBS_ERR_ALIGN;
  return hip_status(ugbs::launch_quest_valu(s, static_cast<const uint16_t*>(Q), static_cast<const uint16_t*>(meta),
                                            scores_out, static_cast<hipStream_t>(stream)));
}

int ugbs_route(const ugbs_problem* p, const float* sigma, const int32_t* idx_sorted,
               int32_t* kv_idx, float* sigma_bar, float* tau, uint8_t* trigger,
               void* workspace, size_t workspace_bytes, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (!sigma || (!idx_sorted != !kv_idx)) return UGBS_ERR_NULL;
  if (!workspace || workspace_bytes < ugbs::ws_total(s)) return UGBS_ERR_WORKSPACE;
  if (!aligned(sigma, 4) || !aligned(idx_sorted, 4) || !aligned(kv_idx, 4) ||
      !aligned(sigma_bar, 4) || !aligned(tau, 4) || !aligned(workspace, 256))
    return UGBS_ERR_ALIGN;
  const int n_pop = population_size(s);
  const int n_trig = (int)std::ceil(s.q * (double)n_pop);
  return hip_status(ugbs::launch_route(s, n_pop, n_trig, sigma, idx_sorted, kv_idx, sigma_bar,
                                       tau, trigger, workspace,
                                       static_cast<hipStream_t>(stream)));
}

int ugbs_route_noalloc(const ugbs_problem* p, const float* sigma, const int32_t* idx_sorted,
                       int32_t* kv_idx, float* sigma_bar, float* tau, uint8_t* trigger, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (!sigma || (!idx_sorted != !kv_idx)) return UGBS_ERR_NULL;
  if (!aligned(sigma, 4) || !aligned(idx_sorted, 4) || !aligned(kv_idx, 4) ||
      !aligned(sigma_bar, 4) || !aligned(tau, 4))
    return UGBS_ERR_ALIGN;
  if (ugbs::ws_route_total(s) > ugbs::kRouteScratchBytes) return UGBS_ERR_SCRATCH;
  void* scratch_ptr = nullptr;
  if (ugbs::route_scratch(&scratch_ptr) != hipSuccess) return UGBS_ERR_HIP;
  const int n_pop = population_size(s);
  const int n_trig = (int)std::ceil(s.q * (double)n_pop);
  return hip_status(ugbs::launch_route(s, n_pop, n_trig, sigma, idx_sorted, kv_idx, sigma_bar,
                                       tau, trigger, scratch_ptr,
                                       static_cast<hipStream_t>(stream)));
}

int ugbs_attend_select(const ugbs_problem* p, const void* Q, const void* K, const void* V,
                       const float* scores, const uint8_t* trigger, const void* workspace,
                       size_t workspace_bytes, void* O, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (!Q || !K || !V || !O) return UGBS_ERR_NULL;
  const bool needs_ws = !scores || !trigger;
  if (needs_ws && (!workspace || workspace_bytes < ugbs::ws_total(s))) return UGBS_ERR_WORKSPACE;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) ||
      !aligned(scores, 4) || (needs_ws && !aligned(workspace, 256)))
    return UGBS_ERR_ALIGN;
  return hip_status(ugbs::launch_attend_select(
      s, static_cast<const uint16_t*>(Q), static_cast<const uint16_t*>(K),
      static_cast<const uint16_t*>(V), scores, trigger, needs_ws ? workspace : nullptr,
      static_cast<uint16_t*>(O), static_cast<hipStream_t>(stream)));
}

int ugbs_select_rows(const ugbs_problem* p, const void* Q, const void* meta, const float* row_scores,
                     const uint8_t* trigger, uint32_t* bitmap, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (s.NB > UGBS_MAX_BLOCKS_ROWS) return UGBS_ERR_SHAPE;
  if (!trigger || !bitmap || (!row_scores && (!Q || !meta))) return UGBS_ERR_NULL;
  if (!aligned(Q, 16) || !aligned(meta, 16) || !aligned(row_scores, 4) || !aligned(bitmap, 4))
    return UGBS_ERR_ALIGN;
  return hip_status(ugbs::launch_select_rows(s, static_cast<const uint16_t*>(Q),
                                             static_cast<const uint16_t*>(meta), row_scores, trigger,
                                             bitmap, static_cast<hipStream_t>(stream)));
}

int ugbs_attend_bitmap(const ugbs_problem* p, const void* Q, const void* K, const void* V,
                       const uint32_t* bitmap, void* O, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (!Q || !K || !V || !bitmap || !O) return UGBS_ERR_NULL;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) || !aligned(bitmap, 4))
    return UGBS_ERR_ALIGN;
  return hip_status(ugbs::launch_attend_bitmap(s, static_cast<const uint16_t*>(Q),
                                               static_cast<const uint16_t*>(K),
                                               static_cast<const uint16_t*>(V), bitmap,
                                               static_cast<uint16_t*>(O),
                                               static_cast<hipStream_t>(stream)));
}

int ugbs_noise_scale(const ugbs_problem* p, const void* Q, const void* meta, double* rough,
                     float* tau, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (!Q || !meta || !rough || !tau) return UGBS_ERR_NULL;
  if (!aligned(Q, 16) || !aligned(meta, 16) || !aligned(rough, 8) || !aligned(tau, 4))
    return UGBS_ERR_ALIGN;
  const hipStream_t hs = static_cast<hipStream_t>(stream);
  const hipError_t e = ugbs::launch_row_roughness(s, static_cast<const uint16_t*>(Q),
                                                  static_cast<const uint16_t*>(meta), rough, hs);
  if (e != hipSuccess) return UGBS_ERR_HIP;
  return hip_status(ugbs::launch_noise_scale(s, rough, tau, hs));
}

int ugbs_bai_tiles(const ugbs_problem* p, const float* scores, const float* tau, const float* z,
                   int32_t n_samples, ugbs_bai_tile* tiles, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (s.NB > UGBS_MAX_BLOCKS_ROWS) return UGBS_ERR_SHAPE;
  if (n_samples < 0 || n_samples > (1 << 20)) return UGBS_ERR_SHAPE;
  if (!scores || !tiles || (n_samples > 0 && (!tau || !z))) return UGBS_ERR_NULL;
  if (!aligned(scores, 4) || !aligned(tau, 4) || !aligned(z, 4) || !aligned(tiles, 8))
    return UGBS_ERR_ALIGN;
  return hip_status(ugbs::launch_bai_tiles(s, scores, tau, z, n_samples, tiles,
                                           static_cast<hipStream_t>(stream)));
}

int ugbs_bai_heads(const ugbs_problem* p, const ugbs_bai_tile* tiles, const float* tau,
                   int32_t n_samples, ugbs_bai_head* heads, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (s.NB > UGBS_MAX_BLOCKS_ROWS) return UGBS_ERR_SHAPE;
  if (n_samples < 0 || n_samples > (1 << 20)) return UGBS_ERR_SHAPE;
  if (!tiles || !tau || !heads) return UGBS_ERR_NULL;
  if (!aligned(tiles, 8) || !aligned(tau, 4) || !aligned(heads, 8)) return UGBS_ERR_ALIGN;
  return hip_status(ugbs::launch_bai_heads(s, tiles, tau, n_samples, heads,
                                           static_cast<hipStream_t>(stream)));
}

int ugbs_attend(const ugbs_problem* p, const void* Q, const void* K, const void* V,
                const int32_t* kv_idx, int32_t kv_width, void* O, void* stream) {
  Shape s;
  int st = make_shape(p, &s);
  if (st) return st;
  if (!Q || !K || !V || !kv_idx || !O) return UGBS_ERR_NULL;
  if (kv_width < 1 || kv_width > UGBS_MAX_KV_WIDTH) return UGBS_ERR_SHAPE;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) ||
      !aligned(kv_idx, 4))
    return UGBS_ERR_ALIGN;
  return hip_status(ugbs::launch_attend(s, static_cast<const uint16_t*>(Q),
                                        static_cast<const uint16_t*>(K),
                                        static_cast<const uint16_t*>(V), kv_idx, kv_width,
                                        static_cast<uint16_t*>(O),
                                        static_cast<hipStream_t>(stream)));
}

}  // extern "C"
