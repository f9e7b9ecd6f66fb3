// arbor_walk: the event-driven controller of Alg. 2 (Transition events with
// lazy rehydration, the scoring of the new active leaf, eviction, and the
// Pressure event raised when the resident tokens reach the budget minus a
// margin) for a whole sequence of active-leaf switches, enqueued at once.
// Every step reads its active leaf from the device, so the host issues all
// launches of all steps without waiting on the device; a failed step leaves a
// negative sticky status that every later kernel checks.
#include "arbor_internal.h"

namespace arbor {
int launch_allocate(const arbor_tree_t *, const int32_t *, int32_t, int64_t, const float *,
                    const arbor_params_t *, int32_t *, int32_t *, uint8_t *, int32_t *, void *,
                    size_t, hipStream_t, int gate);
int launch_walk_stats(const arbor_tree_t *, const int32_t *, const uint8_t *, int64_t, int, int,
                      int64_t *, int32_t *, hipStream_t);
}  // namespace arbor

using namespace arbor;

#define WALK_TRY(x)                    \
  do {                                 \
    const int rc_ = (x);               \
    if (rc_ != ARBOR_OK) return rc_;   \
  } while (0)

extern "C" int arbor_walk(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                          const arbor_walk_t *w, const arbor_params_t *params, int32_t *status,
                          void *workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!geom || !tree || !pool || !w || !params || !status) return ARBOR_EINVAL;
  if (w->n_steps < 0 || (w->n_steps > 0 && !w->targets)) return ARBOR_EINVAL;
  if (!w->A || !w->s || !w->k || !w->delta || !w->on_path || !w->sel_pos) return ARBOR_EINVAL;
  if (params->lazy_rehydration && (!w->host_k || !w->host_v)) return ARBOR_EINVAL;
  if (w->pressure_margin < 0) return ARBOR_EINVAL;
  const bool scored = w->q_win != nullptr;
  if (scored && (!w->v_in || !w->u_in || !w->rows_seen || !w->a_out || !w->slice_layers ||
                 w->n_slice < 1 || w->n_slice > 8 || w->window <= 0))
    return ARBOR_EINVAL;
  const int64_t q_stride = scored ? (int64_t)w->n_slice * geom->num_kv_heads * geom->q_per_kv *
                                        w->window * geom->head_dim *
                                        (geom->dtype == ARBOR_BF16 ? 2 : 4)
                                  : 0;
  const int64_t b_p = w->budget_tokens - w->pressure_margin;
  for (int e = 0; e < w->n_steps; ++e) {
    const int32_t *leaf = w->targets + e;
    int64_t *row = w->stats ? w->stats + 4 * (int64_t)e : nullptr;
    // Transition: reallocate for the new Path*
    WALK_TRY(arbor_allocate(tree, leaf, 1, w->budget_tokens, w->s, params, w->k, w->delta,
                            w->on_path, status, workspace, workspace_bytes, stream));
    if (row)
      WALK_TRY(launch_walk_stats(tree, w->k, w->on_path, w->budget_tokens, 1,
                                 params->lazy_rehydration, row, status, stream));
    // lazy rehydration of the new chain before it is attended
    if (params->lazy_rehydration)
      WALK_TRY(arbor_rehydrate(geom, tree, pool, w->on_path, w->host_k, w->host_v, status,
                               workspace, workspace_bytes, stream));
    // the new leaf's window queries credit its ancestors
    if (scored)
      WALK_TRY(arbor_score(geom, tree, pool, leaf, 1,
                           static_cast<const char *>(w->q_win) + e * q_stride, w->window,
                           w->slice_layers, w->n_slice, w->v_in, w->u_in, w->A, w->rows_seen,
                           w->a_out, w->s, params, status, workspace, workspace_bytes, stream));
    WALK_TRY(arbor_select_compact(geom, tree, pool, w->A, w->k, params, w->sel_pos, status,
                                  workspace, workspace_bytes, stream));
    if (w->pressure_margin > 0) {
      // RaisePressureEvent: fires on the device when M >= B - delta
      WALK_TRY(launch_allocate(tree, leaf, 1, b_p, w->s, params, w->k, w->delta, w->on_path,
                               status, workspace, workspace_bytes, stream, 1));
      if (row)
        WALK_TRY(launch_walk_stats(tree, w->k, w->on_path, b_p, 0, params->lazy_rehydration,
                                   row, status, stream));
      WALK_TRY(arbor_select_compact(geom, tree, pool, w->A, w->k, params, w->sel_pos, status,
                                    workspace, workspace_bytes, stream));
    }
  }
  return ARBOR_OK;
}
