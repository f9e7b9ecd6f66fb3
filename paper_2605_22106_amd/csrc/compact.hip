// arbor_compact: token-extractive, order-preserving compaction of the retained
// K/V rows inside the paged tree KV pool (Sec. 4 Execution: retained entries
// stay, the other entries are freed).
//
// Two launches on one stream:
//   plan     one wave per node: validate the selection, locate each kept
//            position's source slot; one more workgroup of the same launch
//            scans the nodes for the (node, page)-ordered free-stack offsets
//            and the list of changed nodes (a node releases ceil(c / P) -
//            ceil(k / P) pages, so the scan needs nothing from the plan);
//   move     one wave per (changed node, layer, kv head) plane: rows move to
//            lower slots only, so a wave stages a chunk of rows in registers
//            (all loads of the chunk retire before its stores issue) and walks
//            the chunks in ascending slot order -- in-place safe; extra
//            workgroups of the same launch finalize the changed nodes
//            (slot_pos, page table, free stack and its top, c_i).
// The plan and the scan only write the workspace (and the status word), so
// an error either of them finds leaves the state unchanged.
#include <climits>

#include "arbor_internal.h"
#include "select_impl.h"

namespace arbor {

namespace {

constexpr int kPlanPos = 1024;   // per-wave LDS positions in the compaction plan

__device__ __forceinline__ int pos_at(const Tree &t, const Pool &pl, int64_t po, int s) {
  const int page = t.page_table[po + s / pl.P];
  return pl.slot_pos[(int64_t)page * pl.P + (s % pl.P)];
}

// Row of slot s of a node within every (layer, kv head) plane: page * Hkv * P
// + s % P (the plane adds layer * num_pages * Hkv * P + g * P).
__device__ __forceinline__ int plane_row(const Tree &t, const Pool &pl, int64_t po, int s) {
  return t.page_table[po + s / pl.P] * pl.Hkv * pl.P + s % pl.P;
}

__device__ void plan_node(const Tree &t, const Pool &pl, const int32_t *__restrict__ k,
                          const int32_t *__restrict__ sel_pos, int32_t *__restrict__ src_slot,
                          int32_t *__restrict__ mv_src, int32_t *__restrict__ mv_dst,
                          int32_t *__restrict__ first_moved, int32_t *status) {
  // each wave's node positions, slot order, when the node holds at most
  // kPlanPos resident tokens: the binary searches then run in LDS
  __shared__ int s_pos[4][kPlanPos];
  const int lane = lane_id();
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= t.V) return;
  // the node's scalars are loaded together with the status word
  const int c = t.n_kept[i];
  const int ki = k[i];
  const int n = t.n_full[i];
  const int64_t tb = t.tok_off[i];
  const int64_t po = t.page_off[i];
  if (status_failed(status)) return;
  if (ki >= c) return;
  bool bad = ki < 0;
  int *lp = s_pos[threadIdx.x >> 6];
  const bool in_lds = c <= kPlanPos;
  if (in_lds) {
    for (int s = lane; s < c; s += kWave) lp[s] = pos_at(t, pl, po, s);
    // LDS operations of one wave complete in order: the reads below see these
    // writes once the compiler keeps them in program order
    __builtin_amdgcn_wave_barrier();
  }
  for (int s = lane; s < ki; s += kWave) {
    const int p = sel_pos[tb + s];
    bad |= p < 0 || p >= n || (s > 0 && sel_pos[tb + s - 1] >= p);
    // source slot: the resident positions ascend, and the kept ones are a
    // subsequence, so the source of destination s lies in [s, c)
    int lo = s, hi = c - 1, found = -1;
    while (!bad && lo <= hi) {
      const int mid = (lo + hi) >> 1;
      const int pm = in_lds ? lp[mid] : pos_at(t, pl, po, mid);
      if (pm == p) {
        found = mid;
        break;
      }
      if (pm < p) lo = mid + 1;
      else hi = mid - 1;
    }
    bad |= found < 0;
    src_slot[tb + s] = found;
    if (!bad) {
      mv_src[tb + s] = plane_row(t, pl, po, found);
      mv_dst[tb + s] = plane_row(t, pl, po, s);
    }
  }
  if (ballot(bad)) {
    if (lane == 0) status_error(status, ARBOR_EINVAL);
    return;
  }
  // slots already holding their row form a prefix (sources ascend and src >= s)
  int s0 = ki;
  for (int base = 0; base < ki; base += kWave) {
    const int s = base + lane;
    const uint64_t mv = ballot(s < ki && src_slot[tb + s] != s);
    if (mv) {
      s0 = base + __builtin_ctzll(mv);
      break;
    }
  }
  if (lane == 0) first_moved[i] = s0;
}

// meta[0] = number of changed nodes, meta[1] = free-stack top before pushes,
// meta[2] = pages pushed.  One workgroup.
__device__ void scan_nodes(const Tree &t, const Pool &pl, const int32_t *__restrict__ k,
                           int32_t *__restrict__ push_base, int32_t *__restrict__ changed,
                           int32_t *__restrict__ meta, int32_t *status) {
  __shared__ int64_t sm[2 * 16];
  const int V = t.V;
  const int nt = blockDim.x, tid = threadIdx.x;
  const int P = pl.P;
  // each thread takes a run of consecutive nodes, so its loads are issued
  // together and one exchange gives every offset
  const int per = (V + nt - 1) / nt;
  const int i0 = min(V, tid * per), i1 = min(V, i0 + per);
  const int top = tid == 0 ? *pl.free_top : 0;
  auto freed = [&](int c, int ki) { return ki < c ? (c + P - 1) / P - (ki + P - 1) / P : 0; };
  int64_t pages = 0, nodes = 0;
#pragma unroll 4
  for (int i = i0; i < i1; ++i) {
    const int c = t.n_kept[i], ki = k[i];
    pages += freed(c, ki);
    nodes += ki < c ? 1 : 0;
  }
  if (status_failed(status)) {
    if (threadIdx.x == 0) meta[0] = 0;
    return;
  }
  const int64_t v2[2] = {pages, nodes};
  int64_t ex[2], tot[2];
  block_exclusive_scan_n<2>(v2, ex, tot, sm);
  int64_t run_pages = ex[0], run_nodes = ex[1];
  for (int i = i0; i < i1; ++i) {
    const int c = t.n_kept[i], ki = k[i];
    if (ki < c) {
      push_base[i] = (int32_t)run_pages;
      changed[run_nodes] = i;
      run_pages += freed(c, ki);
      ++run_nodes;
    }
  }
  if (threadIdx.x == 0) {
    if (top < 0 || (int64_t)top + tot[0] > pl.num_pages) {
      status_error(status, ARBOR_ECORRUPT);
      meta[0] = 0;
      return;
    }
    meta[0] = (int32_t)tot[1];
    meta[1] = top;
    meta[2] = (int32_t)tot[0];
  }
}

// The plan: workgroups below node_blocks plan four nodes each, the last one
// scans.
__global__ __launch_bounds__(256) void compact_plan(Tree t, Pool pl, const int32_t *__restrict__ k,
                                                    const int32_t *__restrict__ sel_pos,
                                                    int32_t *__restrict__ src_slot,
                                                    int32_t *__restrict__ mv_src,
                                                    int32_t *__restrict__ mv_dst,
                                                    int32_t *__restrict__ first_moved,
                                                    int32_t *__restrict__ push_base,
                                                    int32_t *__restrict__ changed,
                                                    int32_t *__restrict__ meta, int node_blocks,
                                                    int32_t *status) {
  if ((int)blockIdx.x == node_blocks) {
    scan_nodes(t, pl, k, push_base, changed, meta, status);
    return;
  }
  plan_node(t, pl, k, sel_pos, src_slot, mv_src, mv_dst, first_moved, status);
}

// The fused select-and-compact entry point: the wave that selects a block's
// retained set also writes the block's plan, since it knows the source slot
// of every kept position; the moving rows form a suffix of the destinations
// (sources ascend and are at or after their destinations).
struct PlanEmit {
  int32_t *sel;                  // kept positions of the block
  int32_t *mv_src, *mv_dst;      // plane rows of the moving slots
  const int32_t *pt;             // the block's page table
  int P, Hkv;
  int &first;                    // this lane's first moving destination
  __device__ __forceinline__ int row(int s) const { return pt[s / P] * Hkv * P + s % P; }
  __device__ __forceinline__ void operator()(int dst, int src, int pos) const {
    sel[dst] = pos;
    if (src != dst) {
      mv_src[dst] = row(src);
      mv_dst[dst] = row(dst);
      first = min(first, dst);
    }
  }
};

// workgroups below node_blocks select and plan kSelWaves nodes each (one per
// wave; their other waves exit at once, so the selections spread over as many
// CUs as with small workgroups), the last one scans with all kScanWaves waves
constexpr int kSelWaves = 4;
constexpr int kScanWaves = 16;
__global__ __launch_bounds__(kScanWaves * kWave) void select_plan(Tree t, Pool pl, const float *__restrict__ A,
                                                   const int32_t *__restrict__ k, int l_tail,
                                                   int n_sinks, int mode,
                                                   int32_t *__restrict__ sel_pos,
                                                   int32_t *__restrict__ mv_src,
                                                   int32_t *__restrict__ mv_dst,
                                                   int32_t *__restrict__ first_moved,
                                                   int32_t *__restrict__ push_base,
                                                   int32_t *__restrict__ changed,
                                                   int32_t *__restrict__ meta, int node_blocks,
                                                   int32_t *status) {
  __shared__ SelectLds<kSelWaves> lds;
  if ((int)blockIdx.x == node_blocks) {
    scan_nodes(t, pl, k, push_base, changed, meta, status);
    return;
  }
  if ((int)(threadIdx.x >> 6) >= kSelWaves) return;
  const int i = blockIdx.x * kSelWaves + (threadIdx.x >> 6);
  if (i >= t.V) return;
  const int64_t tb = t.tok_off[i];
  int first = INT_MAX;
  const PlanEmit emit{sel_pos + tb, mv_src + tb, mv_dst + tb, t.page_table + t.page_off[i],
                      pl.P, pl.Hkv, first};
  if (select_node(t, pl, A, k, l_tail, n_sinks, mode, i, lds, emit, status)) {
    first = wave_allreduce(first, [](int x, int y) { return min(x, y); });
    if (lane_id() == 0) first_moved[i] = first == INT_MAX ? k[i] : first;
  }
}

// Node bookkeeping of the changed nodes: slot_pos, page table, free stack, c_i.
// It touches no K/V bytes and the moves read none of it (they use the plan's
// tables), so it runs in the same launch as the moves.
__device__ void finalize_nodes(const Tree &t, const Pool &pl, const int32_t *__restrict__ k,
                               const int32_t *__restrict__ sel_pos,
                               const int32_t *__restrict__ push_base,
                               const int32_t *__restrict__ changed,
                               const int32_t *__restrict__ meta, int wave0, int nwaves) {
  const int lane = lane_id();
  const int nch = meta[0];
  const int top = meta[1];
  const int P = pl.P;
  if (wave0 == 0 && lane == 0 && nch > 0) *pl.free_top = top + meta[2];
  for (int w = wave0; w < nch; w += nwaves) {
    const int i = changed[w];
    const int ki = k[i];
    const int c = t.n_kept[i];
    const int64_t tb = t.tok_off[i];
    const int64_t po = t.page_off[i];
    const int keep_pages = (ki + P - 1) / P;
    const int old_pages = (c + P - 1) / P;
    for (int s = lane; s < keep_pages * P; s += kWave) {
      const int page = t.page_table[po + s / P];
      pl.slot_pos[(int64_t)page * P + s % P] = s < ki ? sel_pos[tb + s] : -1;
    }
    const int nfree = old_pages - keep_pages;
    for (int e = lane; e < nfree * P; e += kWave) {
      const int q = keep_pages + e / P;
      const int page = t.page_table[po + q];
      pl.slot_pos[(int64_t)page * P + e % P] = -1;
    }
    __builtin_amdgcn_wave_barrier();
    for (int e = lane; e < nfree; e += kWave) {
      const int q = keep_pages + e;
      pl.free_stack[top + push_base[i] + e] = t.page_table[po + q];
      t.page_table[po + q] = -1;
    }
    if (lane == 0) t.n_kept[i] = ki;
  }
}

// Rows of one (layer, kv head) plane: LPR lanes per row, 16 bytes per lane.
template <int LPR>
__device__ void move_plane(const Pool &pl, int64_t tb, int s0, int ki, int l, int g,
                           const int32_t *__restrict__ mv_src, const int32_t *__restrict__ mv_dst,
                           int lane) {
  constexpr int RPP = kWave / LPR;   // rows per wave pass
  constexpr int PASSES = 8;          // passes per chunk
  constexpr int CH = RPP * PASSES;   // rows staged per chunk
  const int64_t plane = ((int64_t)l * pl.num_pages * pl.Hkv + g) * pl.P;
  const int64_t row_bytes = (int64_t)pl.D * pl.esize;
  char *kb = static_cast<char *>(pl.k) + plane * row_bytes;
  char *vb = static_cast<char *>(pl.v) + plane * row_bytes;
  const int sub = lane % LPR;
  const int rsel = lane / LPR;
  for (int cbase = s0; cbase < ki; cbase += CH) {
    uint4 kr[PASSES], vr[PASSES];
    int64_t dst[PASSES];
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
      const int s = cbase + ps * RPP + rsel;
      dst[ps] = -1;
      if (s < ki) {
        const int64_t so = (int64_t)mv_src[tb + s] * row_bytes + sub * 16;
        kr[ps] = *reinterpret_cast<const uint4 *>(kb + so);
        vr[ps] = *reinterpret_cast<const uint4 *>(vb + so);
        dst[ps] = (int64_t)mv_dst[tb + s] * row_bytes + sub * 16;
      }
    }
    // every lane's loads of this chunk have returned before any store below
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
      if (dst[ps] >= 0) {
        store16_nt(kb + dst[ps], kr[ps]);
        store16_nt(vb + dst[ps], vr[ps]);
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

__global__ __launch_bounds__(256) void compact_move(Tree t, Pool pl, const int32_t *__restrict__ k,
                                                    const int32_t *__restrict__ mv_src,
                                                    const int32_t *__restrict__ mv_dst,
                                                    const int32_t *__restrict__ first_moved,
                                                    const int32_t *__restrict__ sel_pos,
                                                    const int32_t *__restrict__ push_base,
                                                    const int32_t *__restrict__ changed,
                                                    const int32_t *__restrict__ meta,
                                                    int move_blocks, int32_t *status) {
  if (status_failed(status)) return;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if ((int)blockIdx.x >= move_blocks) {
    const int fb = (int)blockIdx.x - move_blocks;
    finalize_nodes(t, pl, k, sel_pos, push_base, changed, meta, fb * 4 + wave,
                   ((int)gridDim.x - move_blocks) * 4);
    return;
  }
  const int planes = pl.L * pl.Hkv;
  const int64_t total = (int64_t)meta[0] * planes;
  const int row_bytes = pl.D * pl.esize;
  for (int64_t w = (int64_t)blockIdx.x * 4 + wave; w < total; w += (int64_t)move_blocks * 4) {
    const int i = changed[w / planes];
    const int rem = (int)(w % planes);
    const int l = rem / pl.Hkv;
    const int g = rem % pl.Hkv;
    const int ki = k[i];
    const int s0 = first_moved[i];
    const int64_t tb = t.tok_off[i];
    if (row_bytes == 128) move_plane<8>(pl, tb, s0, ki, l, g, mv_src, mv_dst, lane);
    else if (row_bytes == 256) move_plane<16>(pl, tb, s0, ki, l, g, mv_src, mv_dst, lane);
    else move_plane<32>(pl, tb, s0, ki, l, g, mv_src, mv_dst, lane);
  }
}

}  // namespace

size_t compact_workspace(const arbor_sizes_t *sz) {
  return (size_t)sz->num_tokens * 12 + (size_t)sz->num_nodes * 16 + 4096;
}

int launch_compact(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                   const int32_t *k, const int32_t *sel_pos, int32_t *status, void *workspace,
                   size_t workspace_bytes, hipStream_t stream) {
  Tree t = make_tree(tree);
  Pool pl = make_pool(geom, pool);
  if (t.V <= 0) return ARBOR_OK;
  Carve cv(workspace, workspace_bytes);
  if ((int64_t)pl.num_pages * pl.Hkv * pl.P >= ((int64_t)1 << 31)) return ARBOR_EUNSUPPORTED;
  int32_t *src_slot = cv.take<int32_t>((size_t)t.N);
  int32_t *mv_src = cv.take<int32_t>((size_t)t.N);
  int32_t *mv_dst = cv.take<int32_t>((size_t)t.N);
  int32_t *first_moved = cv.take<int32_t>(t.V);
  int32_t *push_base = cv.take<int32_t>(t.V);
  int32_t *changed = cv.take<int32_t>(t.V);
  int32_t *meta = cv.take<int32_t>(4);
  if (!cv.ok) return ARBOR_EWORKSPACE;
  const int node_blocks = (t.V + 3) / 4;
  hipLaunchKernelGGL(compact_plan, dim3(node_blocks + 1), dim3(256), 0, stream, t, pl, k, sel_pos,
                     src_slot, mv_src, mv_dst, first_moved, push_base, changed, meta, node_blocks,
                     status);
  const int64_t planes = (int64_t)t.V * pl.L * pl.Hkv;
  const int move_blocks = (int)((planes + 3) / 4 < 8192 ? (planes + 3) / 4 : 8192);
  const int fin_blocks = (t.V + 3) / 4;
  timing_begin(geom, ARBOR_KERNEL_COMPACT_MOVE, stream);
  hipLaunchKernelGGL(compact_move, dim3(move_blocks + fin_blocks), dim3(256), 0, stream, t, pl, k,
                     mv_src, mv_dst, first_moved, sel_pos, push_base, changed, meta, move_blocks,
                     status);
  timing_end(geom, ARBOR_KERNEL_COMPACT_MOVE, stream);
  return hip_ok(hipGetLastError());
}

int launch_select_compact(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                          const float *A, const int32_t *k, const arbor_params_t *params,
                          int32_t *sel_pos, int32_t *status, void *workspace,
                          size_t workspace_bytes, hipStream_t stream) {
  Tree t = make_tree(tree);
  Pool pl = make_pool(geom, pool);
  if (t.V <= 0) return ARBOR_OK;
  Carve cv(workspace, workspace_bytes);
  if ((int64_t)pl.num_pages * pl.Hkv * pl.P >= ((int64_t)1 << 31)) return ARBOR_EUNSUPPORTED;
  int32_t *mv_src = cv.take<int32_t>((size_t)t.N);
  int32_t *mv_dst = cv.take<int32_t>((size_t)t.N);
  int32_t *first_moved = cv.take<int32_t>(t.V);
  int32_t *push_base = cv.take<int32_t>(t.V);
  int32_t *changed = cv.take<int32_t>(t.V);
  int32_t *meta = cv.take<int32_t>(4);
  if (!cv.ok) return ARBOR_EWORKSPACE;
  const int node_blocks = (t.V + kSelWaves - 1) / kSelWaves;
  timing_begin(geom, ARBOR_KERNEL_SELECT, stream);
  hipLaunchKernelGGL(select_plan, dim3(node_blocks + 1), dim3(kScanWaves * kWave), 0, stream, t,
                     pl, A, k,
                     params->l_tail, params->n_sinks, params->select_mode, sel_pos, mv_src, mv_dst,
                     first_moved, push_base, changed, meta, node_blocks, status);
  timing_end(geom, ARBOR_KERNEL_SELECT, stream);
  const int64_t planes = (int64_t)t.V * pl.L * pl.Hkv;
  const int move_blocks = (int)((planes + 3) / 4 < 8192 ? (planes + 3) / 4 : 8192);
  const int fin_blocks = (t.V + 3) / 4;
  timing_begin(geom, ARBOR_KERNEL_COMPACT_MOVE, stream);
  hipLaunchKernelGGL(compact_move, dim3(move_blocks + fin_blocks), dim3(256), 0, stream, t, pl, k,
                     mv_src, mv_dst, first_moved, sel_pos, push_base, changed, meta, move_blocks,
                     status);
  timing_end(geom, ARBOR_KERNEL_COMPACT_MOVE, stream);
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
