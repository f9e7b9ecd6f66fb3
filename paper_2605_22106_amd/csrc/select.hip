// arbor_select: per-block retained set, tail + heavy hitters (Sec. 4 Execution,
// Alg. 1 Evict).  One wavefront per node; the m-th largest accumulated
// attention key is found by an MSB-first radix select over 4-bit digits whose
// bins are counted with wavefront ballots and popcounts, then the kept
// positions are emitted in slot (= position) order with a ballot prefix sum.
#include "arbor_internal.h"

namespace arbor {

namespace {

struct NodeView {
  const int32_t *page_table;
  const int32_t *slot_pos;
  int64_t po;
  int P;
  __device__ __forceinline__ int pos(int s) const {
    int page = page_table[po + s / P];
    return slot_pos[(int64_t)page * P + (s % P)];
  }
};

__global__ __launch_bounds__(256) void select_kernel(Tree t, Pool pl, const float *__restrict__ A,
                                                     const int32_t *__restrict__ k, int l_tail,
                                                     int mode, int32_t *__restrict__ sel_pos,
                                                     int32_t *status) {
  if (status_failed(status)) return;
  const int lane = lane_id();
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= t.V) return;
  const int c = t.n_kept[i];
  const int ki = k[i];
  if (ki >= c) return;
  if (ki < 0) {
    if (lane == 0) status_error(status, ARBOR_EINVAL);
    return;
  }
  const int n = t.n_full[i];
  const int64_t tb = t.tok_off[i];
  const NodeView nv{t.page_table, pl.slot_pos, t.page_off[i], pl.P};
  const int thr = n - l_tail;

  // Resident positions are ascending in slot order, so the tail is a suffix.
  int n_head = 0;
  bool nan = false;
  for (int base = 0; base < c; base += kWave) {
    const int s = base + lane;
    const bool v = s < c;
    const int p = v ? nv.pos(s) : 0;
    const float a = v ? A[tb + p] : 0.f;
    nan |= v && (a != a);
    n_head += popc(ballot(v && p < thr));
  }
  if (ballot(nan)) {
    if (lane == 0) status_error(status, ARBOR_ENONFINITE);
    return;
  }
  const int n_tail = c - n_head;
  int32_t *out = sel_pos + tb;
  if (mode == ARBOR_SELECT_TAIL_ONLY || ki <= n_tail) {
    for (int s = lane; s < ki; s += kWave) out[s] = nv.pos(c - ki + s);
    return;
  }

  // m-th largest key among the head slots [0, n_head).
  const int m = ki - n_tail;
  uint32_t prefix = 0, pmask = 0;
  int remaining = m;
  for (int shift = 28; shift >= 0; shift -= 4) {
    int cnt[16];
#pragma unroll
    for (int b = 0; b < 16; ++b) cnt[b] = 0;
    for (int base = 0; base < n_head; base += kWave) {
      const int s = base + lane;
      const bool v = s < n_head;
      const uint32_t key = v ? ordered_key(A[tb + nv.pos(s)]) : 0u;
      const bool match = v && ((key & pmask) == prefix);
      const uint32_t dig = (key >> shift) & 15u;
      const uint64_t bm = ballot(match);
      const uint64_t b0 = ballot(match && (dig & 1u));
      const uint64_t b1 = ballot(match && (dig & 2u));
      const uint64_t b2 = ballot(match && (dig & 4u));
      const uint64_t b3 = ballot(match && (dig & 8u));
#pragma unroll
      for (int b = 0; b < 16; ++b) {
        const uint64_t mm = bm & ((b & 1) ? b0 : ~b0) & ((b & 2) ? b1 : ~b1) &
                            ((b & 4) ? b2 : ~b2) & ((b & 8) ? b3 : ~b3);
        cnt[b] += popc(mm);
      }
    }
    int chosen = 0;
    for (int b = 15; b >= 0; --b) {
      if (cnt[b] >= remaining) {
        chosen = b;
        break;
      }
      remaining -= cnt[b];
    }
    prefix |= (uint32_t)chosen << shift;
    pmask |= 15u << shift;
  }

  // Keys above the threshold, then `remaining` of the tied keys in slot order.
  int written = 0, ties = 0;
  for (int base = 0; base < n_head; base += kWave) {
    const int s = base + lane;
    const bool v = s < n_head;
    const int p = v ? nv.pos(s) : 0;
    const uint32_t key = v ? ordered_key(A[tb + p]) : 0u;
    const bool gt = v && key > prefix;
    const bool eq = v && key == prefix;
    const uint64_t beq = ballot(eq);
    const bool take = gt || (eq && ties + rank_below(beq, lane) < remaining);
    const uint64_t bt = ballot(take);
    const int dst = written + rank_below(bt, lane);
    if (take && dst < m) out[dst] = p;
    written += popc(bt);
    ties += popc(beq);
  }
  if (written != m && lane == 0) status_error(status, ARBOR_ECORRUPT);
  for (int s = lane; s < n_tail; s += kWave) out[m + s] = nv.pos(n_head + s);
}

}  // namespace

int launch_select(const arbor_geom_t *geom, const arbor_tree_t *tree, const arbor_pool_t *pool,
                  const float *A, const int32_t *k, const arbor_params_t *params,
                  int32_t *sel_pos, int32_t *status, hipStream_t stream) {
  Tree t = make_tree(tree);
  Pool pl = make_pool(geom, pool);
  if (t.V <= 0) return ARBOR_OK;
  dim3 grid((t.V + 3) / 4);
  hipLaunchKernelGGL(select_kernel, grid, dim3(256), 0, stream, t, pl, A, k, params->l_tail,
                     params->select_mode, sel_pos, status);
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
