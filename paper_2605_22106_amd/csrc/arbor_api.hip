// C ABI entry points of libarbor: host-side argument validation and dispatch.
// The kernels live in one translation unit per step of the path.
#include <math.h>

#include "arbor_internal.h"

namespace arbor {
int launch_score(const arbor_geom_t *, const arbor_tree_t *, const arbor_pool_t *, const int32_t *,
                 int32_t, const void *, int32_t, const int32_t *, int32_t, const float *,
                 const float *, float *, int64_t *, float *, float *, const arbor_params_t *,
                 int32_t *, void *, size_t, hipStream_t);
int launch_allocate(const arbor_tree_t *, const int32_t *, int32_t, int64_t, const float *,
                    const arbor_params_t *, int32_t *, int32_t *, uint8_t *, int32_t *, void *,
                    size_t, hipStream_t, int gate);
int launch_select(const arbor_geom_t *, const arbor_tree_t *, const arbor_pool_t *, const float *,
                  const int32_t *, const arbor_params_t *, int32_t *, int32_t *, hipStream_t);
int launch_compact(const arbor_geom_t *, arbor_tree_t *, arbor_pool_t *, const int32_t *,
                   const int32_t *, int32_t *, void *, size_t, hipStream_t);
int launch_select_compact(const arbor_geom_t *, arbor_tree_t *, arbor_pool_t *, const float *,
                          const int32_t *, const arbor_params_t *, int32_t *, int32_t *, void *,
                          size_t, hipStream_t);
int launch_rehydrate(const arbor_geom_t *, arbor_tree_t *, arbor_pool_t *, const uint8_t *,
                     const void *, const void *, int32_t *, void *, size_t, hipStream_t);
int launch_decode(const arbor_geom_t *, const arbor_tree_t *, const arbor_pool_t *,
                  const int32_t *, int32_t, int32_t, int32_t, const void *, void *, int32_t,
                  float *, float, const arbor_decode_credit_t *, int32_t *, void *, size_t,
                  hipStream_t);
int launch_uncertainty(const void *, int32_t, int32_t, int64_t, int32_t, const int32_t *, float *,
                       int32_t, int32_t *, void *, size_t, hipStream_t);
size_t uncertainty_workspace(int32_t, int64_t, int32_t);
size_t score_workspace(const arbor_geom_t *, const arbor_sizes_t *);
size_t allocate_workspace(const arbor_sizes_t *);
size_t compact_workspace(const arbor_sizes_t *);
size_t rehydrate_workspace(const arbor_sizes_t *);
size_t decode_workspace(const arbor_geom_t *, const arbor_sizes_t *);
}  // namespace arbor

using namespace arbor;

static int check_geom(const arbor_geom_t *g) {
  if (!g) return ARBOR_EINVAL;
  if (g->num_layers <= 0 || g->num_kv_heads <= 0 || g->q_per_kv <= 0 || g->num_pages < 0)
    return ARBOR_EINVAL;
  if (g->dtype != ARBOR_BF16 && g->dtype != ARBOR_F32) return ARBOR_EUNSUPPORTED;
  if (g->head_dim != 64 && g->head_dim != 128) return ARBOR_EUNSUPPORTED;
  if (g->page_size <= 0 || g->page_size % 16 != 0 || g->page_size > 256) return ARBOR_EUNSUPPORTED;
  if (g->num_pages > INT32_MAX) return ARBOR_EUNSUPPORTED;
  if (g->timing) {
    const arbor_timing_t *tm = g->timing;
    if (tm->kernel < 0 || tm->kernel >= ARBOR_KERNEL_COUNT || !tm->start || !tm->stop)
      return ARBOR_EINVAL;
  }
  return ARBOR_OK;
}

static int check_tree(const arbor_tree_t *t) {
  if (!t || t->num_nodes < 0 || t->num_tokens < 0) return ARBOR_EINVAL;
  if (t->num_nodes > 0 && (!t->parent || !t->n_full || !t->tok_off || !t->page_off ||
                           !t->n_kept || !t->page_table))
    return ARBOR_EINVAL;
  if (t->num_tokens > INT32_MAX) return ARBOR_EUNSUPPORTED;
  return ARBOR_OK;
}

static int check_pool(const arbor_pool_t *p) {
  if (!p || !p->k || !p->v || !p->slot_pos || !p->free_stack || !p->free_top) return ARBOR_EINVAL;
  return ARBOR_OK;
}

#define ARBOR_TRY(x)           \
  do {                         \
    const int rc_ = (x);       \
    if (rc_ != ARBOR_OK) return rc_; \
  } while (0)

extern "C" {

size_t arbor_workspace_size(const arbor_geom_t *geom, const arbor_sizes_t *sz) {
  if (!geom || !sz) return 0;
  size_t b = 0;
  const size_t parts[5] = {score_workspace(geom, sz), allocate_workspace(sz),
                           compact_workspace(sz), rehydrate_workspace(sz),
                           decode_workspace(geom, sz)};
  for (size_t e = 0; e < 5; ++e) b = parts[e] > b ? parts[e] : b;
  return b + 65536;
}

const char *arbor_strerror(int code) {
  switch (code) {
    case ARBOR_OK: return "ok";
    case ARBOR_OVER_BUDGET: return "over budget: minimum counts exceed the budget";
    case ARBOR_EINVAL: return "invalid argument";
    case ARBOR_ENOPAGES: return "not enough free pages";
    case ARBOR_EHIP: return "HIP launch failure";
    case ARBOR_EUNSUPPORTED: return "unsupported shape";
    case ARBOR_ENONFINITE: return "non-finite score";
    case ARBOR_EWORKSPACE: return "workspace too small";
    case ARBOR_ECORRUPT: return "inconsistent pool bookkeeping";
    default: return "unknown status";
  }
}

int arbor_score(const arbor_geom_t *geom, const arbor_tree_t *tree, const arbor_pool_t *pool,
                const int32_t *observers, int32_t n_obs, const void *q_win, int32_t window,
                const int32_t *slice_layers, int32_t n_slice, const float *v_in,
                const float *u_in, float *A, int64_t *rows_seen, float *a_out, float *s_out,
                const arbor_params_t *params, int32_t *status, void *workspace,
                size_t workspace_bytes, hipStream_t stream) {
  ARBOR_TRY(check_geom(geom));
  ARBOR_TRY(check_tree(tree));
  ARBOR_TRY(check_pool(pool));
  if (!params || !status || !v_in || !u_in || !A || !rows_seen || !a_out || !s_out)
    return ARBOR_EINVAL;
  if (n_obs < 0 || (n_obs > 0 && (!observers || !q_win))) return ARBOR_EINVAL;
  if (n_obs > 65535) return ARBOR_EUNSUPPORTED;
  if (window <= 0 || n_slice <= 0 || n_slice > 8 || !slice_layers) return ARBOR_EINVAL;
  for (int e = 0; e < n_slice; ++e)
    if (slice_layers[e] < 0 || slice_layers[e] >= geom->num_layers) return ARBOR_EINVAL;
  if (params->score_self_window != 0 && params->score_self_window != 1) return ARBOR_EINVAL;
  return launch_score(geom, tree, pool, observers, n_obs, q_win, window, slice_layers, n_slice,
                      v_in, u_in, A, rows_seen, a_out, s_out, params, status, workspace,
                      workspace_bytes, stream);
}

int arbor_allocate(const arbor_tree_t *tree, const int32_t *active, int32_t n_active,
                   int64_t budget_tokens, const float *s, const arbor_params_t *params,
                   int32_t *k_out, int32_t *delta_out, uint8_t *on_path_out, int32_t *status,
                   void *workspace, size_t workspace_bytes, hipStream_t stream) {
  ARBOR_TRY(check_tree(tree));
  if (!params || !status || !s || !k_out || !delta_out || !on_path_out) return ARBOR_EINVAL;
  if (n_active < 1 || !active) return ARBOR_EINVAL;
  if (!(params->eta > 0.0 && params->eta <= 1.0) || params->k_min < 0 || params->l_tail < 0 ||
      !(params->r_min >= 0.0 && params->r_min <= 1.0) || isnan(params->gamma) ||
      isnan(params->lambda_d) || isnan(params->lambda_delta) || isnan(params->alpha_max) ||
      !(params->alpha_max > 0.0) || params->k_protect < 0 ||
      (params->lazy_rehydration != 0 && params->lazy_rehydration != 1))
    return ARBOR_EINVAL;
  return launch_allocate(tree, active, n_active, budget_tokens, s, params, k_out, delta_out,
                         on_path_out, status, workspace, workspace_bytes, stream, 0);
}

int arbor_select(const arbor_geom_t *geom, const arbor_tree_t *tree, const arbor_pool_t *pool,
                 const float *A, const int32_t *k, const arbor_params_t *params,
                 int32_t *sel_pos, int32_t *status, hipStream_t stream) {
  ARBOR_TRY(check_geom(geom));
  ARBOR_TRY(check_tree(tree));
  ARBOR_TRY(check_pool(pool));
  if (!params || !status || !A || !k || !sel_pos) return ARBOR_EINVAL;
  if (params->l_tail < 0 || params->n_sinks < 0) return ARBOR_EINVAL;
  if (params->select_mode != ARBOR_SELECT_TAIL_HEAVY &&
      params->select_mode != ARBOR_SELECT_TAIL_ONLY &&
      params->select_mode != ARBOR_SELECT_SINKS_TAIL)
    return ARBOR_EINVAL;
  return launch_select(geom, tree, pool, A, k, params, sel_pos, status, stream);
}

int arbor_compact(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                  const int32_t *k, const int32_t *sel_pos, int32_t *status, void *workspace,
                  size_t workspace_bytes, hipStream_t stream) {
  ARBOR_TRY(check_geom(geom));
  ARBOR_TRY(check_tree(tree));
  ARBOR_TRY(check_pool(pool));
  if (!status || !k || !sel_pos) return ARBOR_EINVAL;
  return launch_compact(geom, tree, pool, k, sel_pos, status, workspace, workspace_bytes, stream);
}

int arbor_select_compact(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                         const float *A, const int32_t *k, const arbor_params_t *params,
                         int32_t *sel_pos, int32_t *status, void *workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  ARBOR_TRY(check_geom(geom));
  ARBOR_TRY(check_tree(tree));
  ARBOR_TRY(check_pool(pool));
  if (!params || !status || !A || !k || !sel_pos) return ARBOR_EINVAL;
  if (params->l_tail < 0 || params->n_sinks < 0) return ARBOR_EINVAL;
  if (params->select_mode != ARBOR_SELECT_TAIL_HEAVY &&
      params->select_mode != ARBOR_SELECT_TAIL_ONLY &&
      params->select_mode != ARBOR_SELECT_SINKS_TAIL)
    return ARBOR_EINVAL;
  return launch_select_compact(geom, tree, pool, A, k, params, sel_pos, status, workspace,
                               workspace_bytes, stream);
}

int arbor_rehydrate(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                    const uint8_t *on_path, const void *host_k, const void *host_v,
                    int32_t *status, void *workspace, size_t workspace_bytes,
                    hipStream_t stream) {
  ARBOR_TRY(check_geom(geom));
  ARBOR_TRY(check_tree(tree));
  ARBOR_TRY(check_pool(pool));
  if (!status || !on_path || !host_k || !host_v) return ARBOR_EINVAL;
  return launch_rehydrate(geom, tree, pool, on_path, host_k, host_v, status, workspace,
                          workspace_bytes, stream);
}

int arbor_tree_decode_attn(const arbor_geom_t *geom, const arbor_tree_t *tree,
                           const arbor_pool_t *pool, const int32_t *leaves, int32_t n_leaves,
                           int32_t layer_begin, int32_t layer_end, const void *q, void *out,
                           int32_t out_dtype, float *lse_out, float softmax_scale,
                           int32_t *status, void *workspace, size_t workspace_bytes,
                           hipStream_t stream) {
  ARBOR_TRY(check_geom(geom));
  ARBOR_TRY(check_tree(tree));
  ARBOR_TRY(check_pool(pool));
  if (!status || n_leaves < 0 || (n_leaves > 0 && (!leaves || !q || !out))) return ARBOR_EINVAL;
  if (layer_begin < 0 || layer_end > geom->num_layers || layer_end < layer_begin)
    return ARBOR_EINVAL;
  if (out_dtype != ARBOR_BF16 && out_dtype != ARBOR_F32) return ARBOR_EINVAL;
  return launch_decode(geom, tree, pool, leaves, n_leaves, layer_begin, layer_end, q, out,
                       out_dtype, lse_out, softmax_scale, nullptr, status, workspace,
                       workspace_bytes, stream);
}

int arbor_tree_decode_attn_scored(const arbor_geom_t *geom, const arbor_tree_t *tree,
                                  const arbor_pool_t *pool, const int32_t *leaves,
                                  int32_t n_leaves, int32_t layer_begin, int32_t layer_end,
                                  const void *q, void *out, int32_t out_dtype, float *lse_out,
                                  float softmax_scale, const arbor_decode_credit_t *credit,
                                  int32_t *status, void *workspace, size_t workspace_bytes,
                                  hipStream_t stream) {
  ARBOR_TRY(check_geom(geom));
  ARBOR_TRY(check_tree(tree));
  ARBOR_TRY(check_pool(pool));
  if (!status || !credit || n_leaves < 0 || (n_leaves > 0 && (!leaves || !q || !out)))
    return ARBOR_EINVAL;
  if (layer_begin < 0 || layer_end > geom->num_layers || layer_end < layer_begin)
    return ARBOR_EINVAL;
  if (out_dtype != ARBOR_BF16 && out_dtype != ARBOR_F32) return ARBOR_EINVAL;
  if (credit->n_slice < 1 || credit->n_slice > 8 || !credit->slice_layers) return ARBOR_EINVAL;
  for (int e = 0; e < credit->n_slice; ++e)
    if (credit->slice_layers[e] < layer_begin || credit->slice_layers[e] >= layer_end)
      return ARBOR_EINVAL;
  if (credit->self_window != 0 && credit->self_window != 1) return ARBOR_EINVAL;
  if (n_leaves > 0 && (!credit->A || !credit->rows_seen)) return ARBOR_EINVAL;
  return launch_decode(geom, tree, pool, leaves, n_leaves, layer_begin, layer_end, q, out,
                       out_dtype, lse_out, softmax_scale, credit, status, workspace,
                       workspace_bytes, stream);
}

size_t arbor_uncertainty_workspace_size(int32_t n_rows, int64_t vocab, int32_t dtype) {
  if (n_rows < 0 || vocab < 2) return 0;
  return uncertainty_workspace(n_rows, vocab, dtype);
}

int arbor_uncertainty(const void *logits, int32_t dtype, int32_t n_rows, int64_t vocab,
                      int32_t top_k, const int32_t *dst, float *u_out, int32_t n_out,
                      int32_t *status, void *workspace, size_t workspace_bytes,
                      hipStream_t stream) {
  if (!status || !u_out || n_rows < 0 || (n_rows > 0 && !logits)) return ARBOR_EINVAL;
  if (vocab < 2 || top_k < 0 || n_out < 0 || (!dst && n_rows > n_out)) return ARBOR_EINVAL;
  if (dtype != ARBOR_BF16 && dtype != ARBOR_F32) return ARBOR_EUNSUPPORTED;
  // rows are read as 16-byte vectors
  const int64_t per16 = dtype == ARBOR_BF16 ? 8 : 4;
  if (vocab % per16 != 0 || reinterpret_cast<uintptr_t>(logits) % 16 != 0 ||
      vocab > ((int64_t)1 << 31))
    return ARBOR_EUNSUPPORTED;
  return launch_uncertainty(logits, dtype, n_rows, vocab, top_k, dst, u_out, n_out, status,
                            workspace, workspace_bytes, stream);
}

}  // extern "C"
