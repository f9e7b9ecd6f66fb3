// arbor_select: per-block retained set: global sinks of the root prompt, block
// tail and heavy hitters (Sec. 4 Execution, Alg. 1 Evict, Table 7's rules),
// one wave per block (the selection itself is in select_impl.h).
#include "select_impl.h"

namespace arbor {

namespace {

// writes the kept positions of a block in slot order
struct PosEmit {
  int32_t *out;
  __device__ __forceinline__ void operator()(int dst, int, int pos) const { out[dst] = pos; }
};

__global__ __launch_bounds__(256) void select_kernel(Tree t, Pool pl, const float *__restrict__ A,
                                                     const int32_t *__restrict__ k, int l_tail,
                                                     int n_sinks, int mode,
                                                     int32_t *__restrict__ sel_pos,
                                                     int32_t *status) {
  __shared__ SelectLds<4> lds;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= t.V) return;
  const PosEmit emit{sel_pos + t.tok_off[i]};
  select_node(t, pl, A, k, l_tail, n_sinks, mode, i, lds, emit, status);
}

}  // namespace

int launch_select(const arbor_geom_t *geom, const arbor_tree_t *tree, const arbor_pool_t *pool,
                  const float *A, const int32_t *k, const arbor_params_t *params,
                  int32_t *sel_pos, int32_t *status, hipStream_t stream) {
  Tree t = make_tree(tree);
  Pool pl = make_pool(geom, pool);
  if (t.V <= 0) return ARBOR_OK;
  dim3 grid((t.V + 3) / 4);
  timing_begin(geom, ARBOR_KERNEL_SELECT, stream);
  hipLaunchKernelGGL(select_kernel, grid, dim3(256), 0, stream, t, pl, A, k, params->l_tail,
                     params->n_sinks, params->select_mode, sel_pos, status);
  timing_end(geom, ARBOR_KERNEL_SELECT, stream);
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
