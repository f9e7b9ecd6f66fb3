// Retained set of one block (Sec. 4 Execution, Alg. 1 Evict, Table 7's
// rules), shared by arbor_select and the fused select-and-compact entry
// point.  One wavefront per node; the m-th largest accumulated attention key
// is found by an MSB-first radix select over 8-bit digits whose bins are
// counted in a per-wave LDS histogram, then the kept positions are emitted in
// slot (= position) order with a ballot prefix sum: the emitter receives
// (destination index, source slot, position) for every kept slot.
#pragma once

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

constexpr int kCached = 8;   // resident slots per lane held in registers

// One wave's 256-bin histogram of the current 8-bit digit, in LDS.  LDS
// operations of one wave execute in order, so no barrier is needed between
// clearing, counting and reading it.
struct Hist {
  unsigned *h;
  __device__ __forceinline__ void clear(int lane) const {
#pragma unroll
    for (int b = 0; b < 256 / kWave; ++b) h[b * kWave + lane] = 0u;
  }
  __device__ __forceinline__ void add(bool match, uint32_t key, int shift) const {
    if (match) atomicAdd(&h[(key >> shift) & 255u], 1u);
  }
  // Digit holding the `remaining`-th largest counted key; updates remaining
  // to its rank within that digit.  Lane l holds bins 255 - 4l - 3 .. 255 - 4l,
  // so a lane-order prefix sum runs from the largest digit down.
  __device__ __forceinline__ int pick(int &remaining, int lane) const {
    const int top = 255 - 4 * lane;
    const int c0 = (int)h[top], c1 = (int)h[top - 1], c2 = (int)h[top - 2], c3 = (int)h[top - 3];
    const int mine = c0 + c1 + c2 + c3;
    const int inc = wave_inclusive_scan(mine);
    const uint64_t hit = ballot(inc >= remaining);
    const int l = (int)__builtin_ctzll(hit);            // the key is counted, so hit != 0
    int before = lane_value(inc - mine, l);
    const int b0 = lane_value(c0, l), b1 = lane_value(c1, l), b2 = lane_value(c2, l);
    int d = 255 - 4 * l;
    if (before + b0 >= remaining) {
    } else if (before + b0 + b1 >= remaining) {
      before += b0;
      d -= 1;
    } else if (before + b0 + b1 + b2 >= remaining) {
      before += b0 + b1;
      d -= 2;
    } else {
      before += b0 + b1 + b2;
      d -= 3;
    }
    remaining -= before;
    return d;
  }
};

// Slot ranges of one node.  Resident positions ascend with the slot, so the
// sinks (positions < sk), the heavy-hitter candidates and the tail (positions
// >= max(n - L_tail, sk)) are consecutive slot ranges: sinks [0, lo),
// candidates [lo, hi), tail [hi, c).  The kept set is
//   - the first a = min(k, lo) slots and the last k - a slots, when k <= lo,
//     in the recency modes, or when the sinks and the tail hold k already;
//   - otherwise the sinks, the tail and the k - lo - (c - hi) candidates with
//     the largest keys (ties to the lower slot).
struct Ranges {
  int lo, hi;
};

__device__ __forceinline__ bool recency_only(int mode, int ki, int c, const Ranges &rg) {
  return ki <= rg.lo || mode != ARBOR_SELECT_TAIL_HEAVY || ki - rg.lo <= c - rg.hi;
}

// Nodes with at most 64 * kCached resident slots: keys and positions stay in
// registers for every radix pass.  When the block's n <= kStageA positions fit,
// its whole row of A is first copied to LDS with loads issued together with
// the page-table loads, so the keys are read from LDS once the positions are
// known (one global round trip fewer).
constexpr int kStageA = 512;
template <class Emit>
__device__ void select_cached(const NodeView &nv, const float *__restrict__ A, int c, int ki,
                              int thr, int sk, int mode, const Emit &out, int32_t *status,
                              int lane, const Hist &hist, int n, float *__restrict__ a_lds) {
  uint32_t key[kCached];
  int pos[kCached];
  bool nan = false;
  Ranges rg{0, 0};
  const int hthr = thr > sk ? thr : sk;
  const bool staged = n <= kStageA;
  int page[kCached];
#pragma unroll
  for (int r = 0; r < kCached; ++r) {
    const int s = r * kWave + lane;
    page[r] = s < c ? nv.page_table[nv.po + s / nv.P] : 0;
  }
  if (staged) {
#pragma unroll
    for (int r = 0; r < kStageA / kWave; ++r) {
      const int p = r * kWave + lane;
      if (p < n) a_lds[p] = A[p];
    }
    // LDS operations of one wave complete in order; this keeps the compiler
    // from moving the reads below above these writes
    __builtin_amdgcn_wave_barrier();
  }
#pragma unroll
  for (int r = 0; r < kCached; ++r) {
    const int s = r * kWave + lane;
    const bool v = s < c;
    const int p = v ? nv.slot_pos[(int64_t)page[r] * nv.P + (s % nv.P)] : 0;
    const float a = v ? (staged ? a_lds[p] : A[p]) : 0.f;
    nan |= v && (a != a);
    key[r] = ordered_key(a);
    pos[r] = p;
    if (r * kWave < c) {
      rg.lo += popc(ballot(v && p < sk));
      rg.hi += popc(ballot(v && p < hthr));
    }
  }
  if (ballot(nan)) {
    if (lane == 0) status_error(status, ARBOR_ENONFINITE);
    return;
  }
  if (recency_only(mode, ki, c, rg)) {
    const int a = ki < rg.lo ? ki : rg.lo;
    const int b0 = c - (ki - a);   // first of the last ki - a slots
#pragma unroll
    for (int r = 0; r < kCached; ++r) {
      const int s = r * kWave + lane;
      if (s < a) out(s, s, pos[r]);
      else if (s >= b0 && s < c) out(a + s - b0, s, pos[r]);
    }
    return;
  }
  const int m = ki - rg.lo - (c - rg.hi);   // heavy hitters among the candidates
  uint32_t prefix = 0, pmask = 0;
  int remaining = m;
  for (int shift = 24; shift >= 0; shift -= 8) {
    hist.clear(lane);
#pragma unroll
    for (int r = 0; r < kCached; ++r) {
      if (r * kWave >= rg.hi) break;
      const int s = r * kWave + lane;
      hist.add(s >= rg.lo && s < rg.hi && ((key[r] & pmask) == prefix), key[r], shift);
    }
    prefix |= (uint32_t)hist.pick(remaining, lane) << shift;
    pmask |= 255u << shift;
  }
  int written = 0, ties = 0;
#pragma unroll
  for (int r = 0; r < kCached; ++r) {
    if (r * kWave >= c) break;
    const int s = r * kWave + lane;
    const bool cand = s >= rg.lo && s < rg.hi;
    const bool gt = cand && key[r] > prefix;
    const bool eq = cand && key[r] == prefix;
    const uint64_t beq = ballot(eq);
    const bool take = gt || (eq && ties + rank_below(beq, lane) < remaining);
    const uint64_t bt = ballot(take);
    const int dst = written + rank_below(bt, lane);
    if (take && dst < m) out(rg.lo + dst, s, pos[r]);
    written += popc(bt);
    ties += popc(beq);
    if (s < rg.lo) out(s, s, pos[r]);                                   // the sinks
    if (s >= rg.hi && s < c) out(rg.lo + m + s - rg.hi, s, pos[r]);     // the tail, in order
  }
  if (written != m && lane == 0) status_error(status, ARBOR_ECORRUPT);
}

// Larger nodes: every pass streams the keys again (L2-resident).
template <class Emit>
__device__ void select_streamed(const NodeView &nv, const float *__restrict__ A, int c, int ki,
                                int thr, int sk, int mode, const Emit &out, int32_t *status,
                                int lane, const Hist &hist) {
  Ranges rg{0, 0};
  const int hthr = thr > sk ? thr : sk;
  bool nan = false;
  for (int base = 0; base < c; base += kWave) {
    const int s = base + lane;
    const bool v = s < c;
    const int p = v ? nv.pos(s) : 0;
    const float a = v ? A[p] : 0.f;
    nan |= v && (a != a);
    rg.lo += popc(ballot(v && p < sk));
    rg.hi += popc(ballot(v && p < hthr));
  }
  if (ballot(nan)) {
    if (lane == 0) status_error(status, ARBOR_ENONFINITE);
    return;
  }
  if (recency_only(mode, ki, c, rg)) {
    const int a = ki < rg.lo ? ki : rg.lo;
    for (int s = lane; s < ki; s += kWave) {
      const int src = s < a ? s : c - ki + s;
      out(s, src, nv.pos(src));
    }
    return;
  }
  const int m = ki - rg.lo - (c - rg.hi);
  uint32_t prefix = 0, pmask = 0;
  int remaining = m;
  for (int shift = 24; shift >= 0; shift -= 8) {
    hist.clear(lane);
    for (int base = rg.lo; base < rg.hi; base += kWave) {
      const int s = base + lane;
      const bool v = s < rg.hi;
      const uint32_t key = v ? ordered_key(A[nv.pos(s)]) : 0u;
      hist.add(v && ((key & pmask) == prefix), key, shift);
    }
    prefix |= (uint32_t)hist.pick(remaining, lane) << shift;
    pmask |= 255u << shift;
  }
  int written = 0, ties = 0;
  for (int base = rg.lo; base < rg.hi; base += kWave) {
    const int s = base + lane;
    const bool v = s < rg.hi;
    const int p = v ? nv.pos(s) : 0;
    const uint32_t key = v ? ordered_key(A[p]) : 0u;
    const bool gt = v && key > prefix;
    const bool eq = v && key == prefix;
    const uint64_t beq = ballot(eq);
    const bool take = gt || (eq && ties + rank_below(beq, lane) < remaining);
    const uint64_t bt = ballot(take);
    const int dst = written + rank_below(bt, lane);
    if (take && dst < m) out(rg.lo + dst, s, p);
    written += popc(bt);
    ties += popc(beq);
  }
  if (written != m && lane == 0) status_error(status, ARBOR_ECORRUPT);
  for (int s = lane; s < rg.lo; s += kWave) out(s, s, nv.pos(s));
  for (int s = lane; s < c - rg.hi; s += kWave) out(rg.lo + m + s, rg.hi + s, nv.pos(rg.hi + s));
}

// Per-wave LDS of the selection for workgroups of W waves: a histogram and a
// staged row of A.
template <int W>
struct SelectLds {
  unsigned hist[W][256];
  float a[W][kStageA];
};

// The retained set of node i (one wave); returns false when the node keeps
// every resident slot (or on an error), having emitted nothing.
template <int W, class Emit>
__device__ bool select_node(const Tree &t, const Pool &pl, const float *__restrict__ A,
                            const int32_t *__restrict__ k, int l_tail, int n_sinks, int mode, int i,
                            SelectLds<W> &lds, const Emit &emit, int32_t *status) {
  const int lane = lane_id();
  const int w = threadIdx.x >> 6;
  const Hist hist{lds.hist[w]};
  // the node's scalars are loaded together with the status word
  const int c = t.n_kept[i];
  const int ki = k[i];
  const int n = t.n_full[i];
  const int64_t tb = t.tok_off[i];
  const int64_t po = t.page_off[i];
  if (status_failed(status)) return false;
  if (ki >= c) return false;
  if (ki < 0) {
    if (lane == 0) status_error(status, ARBOR_EINVAL);
    return false;
  }
  const NodeView nv{t.page_table, pl.slot_pos, po, pl.P};
  // the global sinks are the first positions of the root block (the prompt)
  const int sk = (i == 0 && mode != ARBOR_SELECT_TAIL_ONLY) ? n_sinks : 0;
  if (c <= kWave * kCached)
    select_cached(nv, A + tb, c, ki, n - l_tail, sk, mode, emit, status, lane, hist, n, lds.a[w]);
  else
    select_streamed(nv, A + tb, c, ki, n - l_tail, sk, mode, emit, status, lane, hist);
  return true;
}

}  // namespace

}  // namespace arbor
