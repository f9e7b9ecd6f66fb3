// arbor_rehydrate: lazy rehydration of evicted blocks that re-enter Path*
// (Sec. 4 "Lazy rehydration"; Alg. 2 Transition branch).  The token span of a
// block is never discarded; its K/V record lives in a token-major host store
// [N][L][Hkv][D] that the kernels read directly over the host link.
//
// Launches on one stream:
//   plan     one workgroup: pages needed per node, (node, page)-ordered pop
//            offsets, ENOPAGES check before any change, new free-stack top;
//   assign   one wave per rehydrated node: new page-table entries and a
//            resident-position mask of the node;
//   move     one wave per (node, layer, kv head) plane: resident rows move to
//            slot = position (higher slots only, so chunks are staged in
//            registers and walked from the top), then the evicted rows are
//            copied from the host store;
//   finalize slot_pos = identity, c_i = n_i.
#include "arbor_internal.h"

namespace arbor {

namespace {

__global__ __launch_bounds__(1024) void rehyd_plan(Tree t, Pool pl, const uint8_t *__restrict__ on_path,
                                                   int32_t *__restrict__ pop_base,
                                                   int32_t *__restrict__ todo,
                                                   int32_t *__restrict__ meta, int32_t *status) {
  __shared__ int64_t sm[2 * 16];
  if (status_failed(status)) {
    if (threadIdx.x == 0) meta[0] = 0;
    return;
  }
  const int P = pl.P;
  // each thread takes a run of consecutive blocks (their path flags loaded
  // eight at a time; only Path* blocks load their sizes), and one scan
  // places the runs, so the blocks are listed in ascending id
  constexpr int kGrp = 8;
  const int nt = blockDim.x;
  const int per = (t.V + nt - 1) / nt;
  const int r0 = min(t.V, (int)threadIdx.x * per), r1 = min(t.V, r0 + per);
  auto need_of = [&](int i) -> int64_t {
    const int n = t.n_full[i], c = t.n_kept[i];
    return c < n ? (int64_t)((n + P - 1) / P - (c + P - 1) / P) : -1;   // -1: nothing to restore
  };
  int64_t my_pages = 0, my_nodes = 0;
  for (int ib = r0; ib < r1; ib += kGrp) {
    uint8_t f[kGrp];
#pragma unroll
    for (int u = 0; u < kGrp; ++u) f[u] = ib + u < r1 ? on_path[ib + u] : 0;
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      if (f[u]) {
        const int64_t nd = need_of(ib + u);
        if (nd >= 0) {
          my_pages += nd;
          ++my_nodes;
        }
      }
    }
  }
  const int64_t v[2] = {my_pages, my_nodes};
  int64_t ex[2], tot[2];
  block_exclusive_scan_n<2>(v, ex, tot, sm);
  const int64_t run_pages = tot[0], run_nodes = tot[1];
  int64_t op = ex[0], on = ex[1];
  for (int ib = r0; ib < r1 && my_nodes > 0; ib += kGrp) {
    uint8_t f[kGrp];
#pragma unroll
    for (int u = 0; u < kGrp; ++u) f[u] = ib + u < r1 ? on_path[ib + u] : 0;
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      if (f[u]) {
        const int64_t nd = need_of(ib + u);
        if (nd >= 0) {
          pop_base[ib + u] = (int32_t)op;
          todo[on] = ib + u;
          op += nd;
          ++on;
        }
      }
    }
  }
  if (threadIdx.x == 0) {
    const int top = *pl.free_top;
    if (run_pages > top) {
      status_error(status, ARBOR_ENOPAGES);
      meta[0] = 0;
      return;
    }
    meta[0] = (int32_t)run_nodes;
    meta[1] = top;
    *pl.free_top = top - (int32_t)run_pages;
  }
}

__global__ __launch_bounds__(256) void rehyd_assign(Tree t, Pool pl, const int32_t *__restrict__ pop_base,
                                                    const int32_t *__restrict__ todo,
                                                    const int32_t *__restrict__ meta,
                                                    uint8_t *__restrict__ kept_mask,
                                                    int32_t *status) {
  if (status_failed(status)) return;
  const int lane = lane_id();
  const int P = pl.P;
  const int top = meta[1];
  for (int w = blockIdx.x * 4 + (threadIdx.x >> 6); w < meta[0]; w += gridDim.x * 4) {
    const int i = todo[w];
    const int n = t.n_full[i], c = t.n_kept[i];
    const int64_t po = t.page_off[i];
    const int64_t tb = t.tok_off[i];
    const int old_pages = (c + P - 1) / P;
    const int new_pages = (n + P - 1) / P;
    for (int p = lane; p < n; p += kWave) kept_mask[tb + p] = 0;
    // the clearing stores complete before the marking stores issue
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
    for (int s = lane; s < c; s += kWave) {
      const int page = t.page_table[po + s / P];
      kept_mask[tb + pl.slot_pos[(int64_t)page * P + s % P]] = 1;
    }
    for (int q = old_pages + lane; q < new_pages; q += kWave)
      t.page_table[po + q] = pl.free_stack[top - 1 - (pop_base[i] + (q - old_pages))];
  }
}

template <int LPR>
__device__ void rehyd_plane(const Tree &t, const Pool &pl, int i, int l, int g,
                            const char *__restrict__ hk, const char *__restrict__ hv,
                            const uint8_t *__restrict__ kept_mask, int lane) {
  constexpr int RPP = kWave / LPR;
  constexpr int PASSES = 8;
  constexpr int CH = RPP * PASSES;
  const int P = pl.P;
  const int n = t.n_full[i], c = t.n_kept[i];
  const int64_t po = t.page_off[i];
  const int64_t tb = t.tok_off[i];
  char *kb = static_cast<char *>(pl.k);
  char *vb = static_cast<char *>(pl.v);
  const int sub = lane % LPR;
  const int rsel = lane / LPR;
  const int64_t row_bytes = (int64_t)pl.D * pl.esize;
  // resident rows: slot s -> slot pos(s) >= s; from the top chunk downwards
  for (int ctop = c; ctop > 0; ctop -= CH) {
    uint4 kr[PASSES], vr[PASSES];
    int64_t dst[PASSES];
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
      const int s = ctop - CH + ps * RPP + rsel;
      dst[ps] = -1;
      if (s >= 0 && s < ctop) {
        const int spage = t.page_table[po + s / P];
        const int p = pl.slot_pos[(int64_t)spage * P + s % P];
        if (p != s) {
          const int64_t so = row_byte_offset(pl, l, spage, g, s % P) + sub * 16;
          kr[ps] = *reinterpret_cast<const uint4 *>(kb + so);
          vr[ps] = *reinterpret_cast<const uint4 *>(vb + so);
          dst[ps] = row_byte_offset(pl, l, t.page_table[po + p / P], g, p % P) + sub * 16;
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
      if (dst[ps] >= 0) {
        *reinterpret_cast<uint4 *>(kb + dst[ps]) = kr[ps];
        *reinterpret_cast<uint4 *>(vb + dst[ps]) = vr[ps];
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  // evicted rows from the token-span record
  const int64_t hstride = (int64_t)pl.L * pl.Hkv * row_bytes;
  const int64_t hoff = ((int64_t)l * pl.Hkv + g) * row_bytes + sub * 16;
  for (int pb = 0; pb < n; pb += RPP * PASSES) {
    uint4 kr[PASSES], vr[PASSES];
    int64_t dst[PASSES];
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
      const int p = pb + ps * RPP + rsel;
      dst[ps] = -1;
      if (p < n && !kept_mask[tb + p]) {
        const int64_t so = (tb + p) * hstride + hoff;
        kr[ps] = *reinterpret_cast<const uint4 *>(hk + so);
        vr[ps] = *reinterpret_cast<const uint4 *>(hv + so);
        dst[ps] = row_byte_offset(pl, l, t.page_table[po + p / P], g, p % P) + sub * 16;
      }
    }
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
      if (dst[ps] >= 0) {
        *reinterpret_cast<uint4 *>(kb + dst[ps]) = kr[ps];
        *reinterpret_cast<uint4 *>(vb + dst[ps]) = vr[ps];
      }
    }
  }
}

__global__ __launch_bounds__(256) void rehyd_move(Tree t, Pool pl, const char *__restrict__ hk,
                                                  const char *__restrict__ hv,
                                                  const int32_t *__restrict__ todo,
                                                  const int32_t *__restrict__ meta,
                                                  const uint8_t *__restrict__ kept_mask,
                                                  int32_t *status) {
  if (status_failed(status)) return;
  const int lane = lane_id();
  const int planes = pl.L * pl.Hkv;
  const int64_t total = (int64_t)meta[0] * planes;
  const int row_bytes = pl.D * pl.esize;
  for (int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); w < total;
       w += (int64_t)gridDim.x * 4) {
    const int i = todo[w / planes];
    const int rem = (int)(w % planes);
    const int l = rem / pl.Hkv;
    const int g = rem % pl.Hkv;
    if (row_bytes == 128) rehyd_plane<8>(t, pl, i, l, g, hk, hv, kept_mask, lane);
    else if (row_bytes == 256) rehyd_plane<16>(t, pl, i, l, g, hk, hv, kept_mask, lane);
    else rehyd_plane<32>(t, pl, i, l, g, hk, hv, kept_mask, lane);
  }
}

__global__ __launch_bounds__(256) void rehyd_finalize(Tree t, Pool pl, const int32_t *__restrict__ todo,
                                                      const int32_t *__restrict__ meta,
                                                      int32_t *status) {
  if (status_failed(status)) return;
  const int lane = lane_id();
  const int P = pl.P;
  for (int w = blockIdx.x * 4 + (threadIdx.x >> 6); w < meta[0]; w += gridDim.x * 4) {
    const int i = todo[w];
    const int n = t.n_full[i];
    const int64_t po = t.page_off[i];
    const int np_ = (n + P - 1) / P;
    for (int s = lane; s < np_ * P; s += kWave) {
      const int page = t.page_table[po + s / P];
      pl.slot_pos[(int64_t)page * P + s % P] = s < n ? s : -1;
    }
    if (lane == 0) t.n_kept[i] = n;
  }
}

}  // namespace

size_t rehydrate_workspace(const arbor_sizes_t *sz) {
  return (size_t)sz->num_tokens + (size_t)sz->num_nodes * 8 + 4096;
}

int launch_rehydrate(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                     const uint8_t *on_path, const void *host_k, const void *host_v,
                     int32_t *status, void *workspace, size_t workspace_bytes,
                     hipStream_t stream) {
  Tree t = make_tree(tree);
  Pool pl = make_pool(geom, pool);
  if (t.V <= 0) return ARBOR_OK;
  Carve cv(workspace, workspace_bytes);
  int32_t *pop_base = cv.take<int32_t>(t.V);
  int32_t *todo = cv.take<int32_t>(t.V);
  int32_t *meta = cv.take<int32_t>(4);
  uint8_t *kept_mask = cv.take<uint8_t>((size_t)t.N);
  if (!cv.ok) return ARBOR_EWORKSPACE;
  const dim3 node_grid((t.V + 3) / 4 < 4096 ? (t.V + 3) / 4 : 4096);
  hipLaunchKernelGGL(rehyd_plan, dim3(1), dim3(1024), 0, stream, t, pl, on_path, pop_base, todo,
                     meta, status);
  hipLaunchKernelGGL(rehyd_assign, node_grid, dim3(256), 0, stream, t, pl, pop_base, todo, meta,
                     kept_mask, status);
  const int64_t planes = (int64_t)t.V * pl.L * pl.Hkv;
  const int move_blocks = (int)((planes + 3) / 4 < 8192 ? (planes + 3) / 4 : 8192);
  hipLaunchKernelGGL(rehyd_move, dim3(move_blocks), dim3(256), 0, stream, t, pl,
                     static_cast<const char *>(host_k), static_cast<const char *>(host_v), todo,
                     meta, kept_mask, status);
  hipLaunchKernelGGL(rehyd_finalize, node_grid, dim3(256), 0, stream, t, pl, todo, meta, status);
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
