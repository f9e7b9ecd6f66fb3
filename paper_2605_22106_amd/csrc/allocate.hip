// arbor_allocate: tree-aware keep-counts under a global token budget.
//
// Eq. 2 gives the off-path retention ratio r_i = clip(alpha w_i, r_min, 1) with
// w_i = eta s_i^gamma e^{-lambda_d d_i} e^{-lambda_Delta Delta_i}; Eq. 3 turns it
// into k_i = min(n_i, max(K_min, |T_i|, floor(r_i n_i))).  The KKT view of
// Sec. 4 sets the one global scale alpha so that the total meets the budget.
// Token j of block i is kept exactly when alpha >= j / (w_i n_i) ("price"), so
// the largest feasible alpha keeps every price below the (E+1)-th smallest one,
// E being the budget left after the floors.  Path* nodes (Alg. 2 Transition)
// are pinned at n_i; when the floors alone overflow (Alg. 2 Pressure) the
// lowest-priority blocks are drained towards K_min, found by a weighted radix
// select over the bit patterns of w_i.
//
// Finding the (E+1)-th smallest price without listing every token: the prices
// of block i are j / W_i for consecutive j, so the number of prices up to x is
// floor(x W_i) - F_i (clamped), exact up to rounding at the two ends.  A
// search over x with that count brackets the order statistic between two
// values whose exact counts lie on either side of E; only the few prices in
// the bracket are listed, and an MSB-first radix select over their fp64 bit
// patterns (positive doubles order like their bits) picks the exact one.
//
// Everything runs in one 1024-thread workgroup: the work is O(V) per search
// step and latency bound.  Per-node state sits in LDS when the tree is small
// enough, else in the workspace.  fp64, no contraction, so the prices are the
// same IEEE quotients any fp64 implementation computes.
#include "arbor_internal.h"

#pragma clang fp contract(off)

namespace arbor {

namespace {

constexpr int AT = 1024;
constexpr int kLdsNodes = 512;    // per-node state in LDS up to this many nodes
constexpr int kGeoNodes = 10240;  // parent, depth and down links in LDS up to this many
constexpr int kCandLds = 1536;    // listed prices selected in LDS up to this many
constexpr int kNodeBytes = 2 * 8 + 8 * 4 + 1;
constexpr int kSearchWaves = AT / kWave / 2;   // waves per bracket end
constexpr int kPtsPerWave = 4;                  // test points of each wave
constexpr int kSearchPts = kSearchWaves * kPtsPerWave;   // test points per end
constexpr int kDecay = 128;                    // tabulated depths and distances

// The decay factors exp(-lambda_d d) and exp(-lambda_Delta Delta) for small
// integer d and Delta are tabulated per call by the host with the C library's
// exp, the same doubles an fp64 reference on the host obtains, so that ties
// between prices of different nodes break the same way (a device exp may
// round the last bit differently).
struct AllocParams {
  double alpha_max, gamma, lambda_d, lambda_delta, eta, r_min;
  int k_min, l_tail;
  int rehydrate;   // Path* blocks count n_i (restored) or their resident c_i
  int k_protect;   // 0: Path* blocks pinned; > 0: they take part with this floor
  double dexp[kDecay], texp[kDecay];
};

// s^gamma, correctly rounded for the integer exponents 1..4: s is an fp32
// value, so s * s is exact in fp64 and one more product rounds once
__device__ __forceinline__ double pow_gamma(double s, double gamma) {
  if (gamma == 1.0) return s;
  if (gamma == 2.0) return s * s;
  if (gamma == 3.0) return (s * s) * s;
  if (gamma == 4.0) return (s * s) * (s * s);
  return pow(s, gamma);
}

// Per-node working state.  parent / n_full / n_kept are the tree's arrays or
// LDS copies of them; `path` is the on-path output or its LDS copy.
struct Nodes {
  int32_t *parent, *n_full, *n_kept;
  int32_t *depth, *down, *F, *cnt, *cap;
  double *W, *w;
  uint8_t *path;
};

struct AllocWs {
  int32_t *depth, *down, *F, *cnt, *cap;
  double *W, *w;
  uint64_t *buf0, *buf1;
  int64_t buf_cap;
  int32_t *eF, *eC;     // the blocks with eligible prices: F, count
  double *eW;            // and W, side by side (trees beyond LDS mode)
};

__device__ __forceinline__ double price(int j, double W) {
  return W > 0.0 ? (double)j / W : __builtin_inf();
}

// Number of j in (F, c] whose price satisfies pred (prices ascend with j).
template <class Pred>
__device__ int count_prefix(int F, int c, double W, Pred pred) {
  int lo = F + 1, hi = c, ans = F;
  while (lo <= hi) {
    const int mid = lo + ((hi - lo) >> 1);
    if (pred(price(mid, W))) {
      ans = mid;
      lo = mid + 1;
    } else {
      hi = mid - 1;
    }
  }
  return ans - F;
}

// Largest m in [F, F + cnt] with price(m) <= x (m = F: none), starting from
// the rounded estimate floor(x W) and correcting it by exact comparisons.
// The product y = x W carries a relative error of at most 2^-53, and so does
// each quotient j / W: an integer j with j > y (1 + 2^-50) has a price above
// x, one with j < y (1 - 2^-50) a price below it.  Only an estimate that close
// to the boundary needs the divisions.
__device__ int last_le(double x, int F, int cnt, double W) {
  const double yr = x * W;
  double y = __builtin_floor(yr);
  // (a NaN estimate, 0 * inf, starts from F)
  y = !(y >= (double)F) ? (double)F : (y > (double)(F + cnt) ? (double)(F + cnt) : y);
  int m = (int)y;
  const bool up_ok = m == F + cnt || (double)(m + 1) > yr * (1.0 + 0x1p-50);
  const bool down_ok = m == F || (double)m < yr * (1.0 - 0x1p-50);
  if (up_ok && down_ok && yr < __builtin_inf()) return m;
  while (m < F + cnt && price(m + 1, W) <= x) ++m;
  while (m > F && price(m, W) > x) --m;
  return m;
}

// Largest m in [F, F + cnt] with price(m) < x (m = F: none), as last_le.
__device__ int last_lt(double x, int F, int cnt, double W) {
  const double yr = x * W;
  double y = __builtin_floor(yr);
  y = !(y >= (double)F) ? (double)F : (y > (double)(F + cnt) ? (double)(F + cnt) : y);
  int m = (int)y;
  const bool up_ok = m == F + cnt || (double)(m + 1) > yr * (1.0 + 0x1p-50);
  const bool down_ok = m == F || (double)m < yr * (1.0 - 0x1p-50);
  if (up_ok && down_ok && yr < __builtin_inf()) return m;
  while (m < F + cnt && price(m + 1, W) < x) ++m;
  while (m > F && !(price(m, W) < x)) --m;
  return m;
}

// Eligible prices of a block: those in (F, cap] that are finite and at most
// amax.  Prices ascend with j, so when the last one qualifies they all do.
__device__ int eligible(int F, int cap, double W, double amax) {
  if (cap <= F || !(W > 0.0)) return 0;
  const double last = price(cap, W);
  if (last <= amax && last < __builtin_inf()) return cap - F;
  if (last < __builtin_inf()) return last_le(amax, F, cap - F, W) - F;
  return count_prefix(F, cap, W, [amax](double x) { return x <= amax && x < __builtin_inf(); });
}

// Rounded count of prices <= x of one node (exact up to one price at each end).
__device__ __forceinline__ double approx_le(double x, int F, int cnt, double W) {
  double y = __builtin_floor(x * W) - (double)F;
  return y < 0.0 ? 0.0 : (y > (double)cnt ? (double)cnt : y);
}

// three block-wide sums in one exchange; sm holds 48 values
__device__ void block_sum3(int64_t (&v)[3], int64_t *sm) {
  const int lane = lane_id(), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
  for (int q = 0; q < 3; ++q) v[q] = wave_sum(v[q]);
  if (lane == 0)
#pragma unroll
    for (int q = 0; q < 3; ++q) sm[16 * q + w] = v[q];
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 3; ++q) v[q] = wave_sum(lane < nw ? sm[16 * q + lane] : (int64_t)0);
  __syncthreads();
}

__device__ __forceinline__ int64_t wave_min_i64(int64_t v) {
  return wave_allreduce(v, [](int64_t a, int64_t b) { return a < b ? a : b; });
}

// block-wide sums of v[0..NS) and minima of v[NS..N) in one exchange; sm
// holds 16 N values
// Threads from `live` on hold the identities, so their waves skip the
// wave-level reductions; the wave totals are combined by wave 0 alone, which
// hands the results back through sm.
template <int NS, int N>
__device__ void block_reduce_n(int64_t (&v)[N], int64_t *sm, int live) {
  const int lane = lane_id(), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  if (w * kWave < live) {
#pragma unroll
    for (int q = 0; q < N; ++q) v[q] = q < NS ? wave_sum(v[q]) : wave_min_i64(v[q]);
  }
  if (lane == 0)
#pragma unroll
    for (int q = 0; q < N; ++q) sm[16 * q + w] = v[q];
  __syncthreads();
  if (w == 0) {
    const bool in = lane < nw;
#pragma unroll
    for (int q = 0; q < N; ++q) {
      const int64_t r = q < NS ? wave_sum(in ? sm[16 * q + lane] : (int64_t)0)
                               : wave_min_i64(in ? sm[16 * q + lane] : INT64_MAX);
      if (lane == 0) sm[16 * q] = r;
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < N; ++q) v[q] = sm[16 * q];
  __syncthreads();
}

// block-wide sum of v[0] and minima of v[1], v[2] in one exchange
__device__ void block_min_sum3(int64_t (&v)[3], int64_t *sm) {
  const int lane = lane_id(), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v[0] = wave_sum(v[0]);
  v[1] = wave_min_i64(v[1]);
  v[2] = wave_min_i64(v[2]);
  if (lane == 0)
#pragma unroll
    for (int q = 0; q < 3; ++q) sm[16 * q + w] = v[q];
  __syncthreads();
  const bool in = lane < nw;
  v[0] = wave_sum(in ? sm[lane] : (int64_t)0);
  v[1] = wave_min_i64(in ? sm[16 + lane] : INT64_MAX);
  v[2] = wave_min_i64(in ? sm[32 + lane] : INT64_MAX);
  __syncthreads();
}

// The rank-th smallest (0-based) of the keys src[0, n), 0 <= rank < n.  Keys
// are taken relative to the smallest one, and each pass splits the remaining
// range [lo, lo + span] into 256 equal power-of-two buckets: the listed prices
// are spread fairly evenly over their small range, so one pass usually leaves
// at most 64 candidates, which one wave then ranks directly.  src and dst
// (room for n keys) may be LDS or global memory; both are overwritten.
// Called by the whole block; contains __syncthreads.
__device__ uint64_t select_rank(uint64_t *src, uint64_t *dst, int64_t n, int64_t rank,
                                int64_t *sm, bool known = false, uint64_t kmin = 0,
                                uint64_t kmax = 0) {
  __shared__ unsigned hist4[4 * 256];
  __shared__ int64_t s_wtot[4];
  __shared__ int s_chosen;
  __shared__ int64_t s_below;
  __shared__ unsigned s_ncand;
  __shared__ uint64_t s_key;
  const int tid = threadIdx.x, lane = lane_id();
  uint64_t cmin = kmin, cmax = kmax;
  if (!known) {
    cmin = ~0ull;
    cmax = 0ull;
    for (int64_t e = tid; e < n; e += blockDim.x) {
      const uint64_t key = src[e];
      cmin = key < cmin ? key : cmin;
      cmax = key > cmax ? key : cmax;
    }
    // both extremes in one exchange (keys of finite positive doubles < 2^63)
    int64_t v3[3] = {0, cmin == ~0ull ? INT64_MAX : (int64_t)cmin, INT64_MAX - (int64_t)cmax};
    block_min_sum3(v3, sm);
    cmin = (uint64_t)v3[1];
    cmax = (uint64_t)(INT64_MAX - v3[2]);
  }
  if (cmin == cmax) return cmin;
  int64_t ncand = n;
  uint64_t lo = cmin, span = cmax - cmin;
  while (ncand > kWave) {
    if (span == 0) return lo;   // every candidate left is lo
    // buckets of 2^shift keys: span >> shift < 256
    const int bits = 64 - __builtin_clzll(span);
    const int shift = bits > 8 ? bits - 8 : 0;
    for (int bn = tid; bn < 4 * 256; bn += blockDim.x) hist4[bn] = 0;
    __syncthreads();
    unsigned *myh = hist4 + 256 * ((tid >> 6) & 3);
    for (int64_t e = tid; e < ncand; e += blockDim.x)
      atomicAdd(&myh[(src[e] - lo) >> shift], 1u);
    __syncthreads();
    // bucket holding the element of rank `rank` (first 256 threads, 4 waves)
    const unsigned h =
        tid < 256 ? hist4[tid] + hist4[256 + tid] + hist4[512 + tid] + hist4[768 + tid] : 0u;
    const int64_t inc = wave_inclusive_scan<int64_t>((int64_t)h);
    if (tid < 256 && lane == kWave - 1) s_wtot[tid >> 6] = inc;
    __syncthreads();
    if (tid < 256) {
      int64_t base = 0;
      for (int w = 0; w < (tid >> 6); ++w) base += s_wtot[w];
      const int64_t ex = base + inc - (int64_t)h;
      if (ex <= rank && rank < ex + (int64_t)h) {
        s_chosen = tid;
        s_below = ex;
      }
    }
    __syncthreads();
    const uint64_t chosen = (uint64_t)s_chosen;
    rank -= s_below;
    const uint64_t blo = chosen << shift;
    if (shift == 0) return lo + blo;
    if (tid == 0) s_ncand = 0;
    __syncthreads();
    for (int64_t e0 = 0; e0 < ncand; e0 += blockDim.x) {
      const int64_t e = e0 + tid;
      const bool keep = e < ncand && ((src[e] - lo) >> shift) == chosen;
      const uint64_t bk = ballot(keep);
      unsigned base = 0;
      if (lane == 0 && bk) base = atomicAdd(&s_ncand, (unsigned)popc(bk));
      base = lane_value(base, 0);
      if (keep) dst[base + rank_below(bk, lane)] = src[e];
    }
    __syncthreads();
    ncand = s_ncand;
    const uint64_t rest = span - blo;
    lo += blo;
    span = rest < (1ull << shift) - 1ull ? rest : (1ull << shift) - 1ull;
    uint64_t *tmp = src;
    src = dst;
    dst = tmp;
    __syncthreads();
  }
  // at most 64 left: lane l holds candidate l and counts the smaller ones
  if (tid < kWave) {
    const uint64_t k = lane < ncand ? src[lane] : ~0ull;
    int less = 0, leq = 0;
    for (int j = 0; j < (int)ncand; ++j) {
      const uint64_t kj = lane_value(k, j);
      less += kj < k ? 1 : 0;
      leq += kj <= k ? 1 : 0;
    }
    if (lane < ncand && less <= rank && rank < leq) s_key = k;
  }
  __syncthreads();
  return s_key;
}

__device__ __forceinline__ double key_value(uint64_t k) {
  return __longlong_as_double((long long)k);
}

// test point q (0-based) of N splitting (lo, lo + span) into N + 1 parts
template <int N>
__device__ __forceinline__ uint64_t split_point(uint64_t lo, uint64_t span, int q) {
  const uint64_t m = (uint64_t)(q + 1);
  return lo + (span / (N + 1)) * m + ((span % (N + 1)) * m) / (N + 1);
}

// MODE 1: all per-node state in LDS; 2: the geometry (parent, depth, down)
// in LDS, the rest in the workspace; 0: everything in the workspace.  The
// mode is a template argument so that every access compiles to an LDS or a
// global instruction rather than a flat one.
template <int MODE>
__global__ __launch_bounds__(AT) void allocate_kernel(Tree t, const int32_t *__restrict__ active,
                                                      int n_active, int64_t budget,
                                                      const float *__restrict__ s_in, AllocParams p,
                                                      int32_t *__restrict__ k_out,
                                                      int32_t *__restrict__ delta_out,
                                                      uint8_t *__restrict__ on_path,
                                                      int32_t *status, AllocWs ws, int gate) {
  constexpr int in_lds = MODE;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn[];
  __shared__ int64_t sm[7 * 16];
  __shared__ int s_err;
  __shared__ unsigned long long hist64[256];
  __shared__ double s_cnt[2][2 * kSearchPts];
  __shared__ uint64_t s_x[2][2 * kSearchPts];
  __shared__ double s_dexp[kDecay], s_texp[kDecay];
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = lane_id();
  const int V = t.V;
  // each thread's first node, its score and the decay tables: loads issued
  // together, ahead of the status check, so they cost one round trip
  int par0 = 0, nf0 = 0, nk0 = 0;
  float s0 = 0.f;
  if (tid < V) {
    par0 = t.parent[tid];
    nf0 = t.n_full[tid];
    nk0 = t.n_kept[tid];
    s0 = s_in[tid];
  }
  double dx = 0.0, tx = 0.0;
  if (tid < kDecay) {
    dx = p.dexp[tid];
    tx = p.texp[tid];
  }
  if (status_failed(status)) return;
  if (tid < kDecay) {
    s_dexp[tid] = dx;
    s_texp[tid] = tx;
  }
  if (tid == 0) s_err = 0;
  if (gate) {
    // a Pressure event (Alg. 2): it fires only when the resident tokens
    // reach the budget it is given; otherwise every count stays as it is
    int64_t m = 0;
    for (int i = tid; i < V; i += AT) m += i == tid ? nk0 : t.n_kept[i];
    m = block_sum<int64_t>(m, sm);
    if (m < budget) {
      for (int i = tid; i < V; i += AT) k_out[i] = i == tid ? nk0 : t.n_kept[i];
      return;
    }
  }

  // listed prices: LDS after the node state when few enough, else workspace
  const size_t node_lds = in_lds == 1 ? ((size_t)V * kNodeBytes + 15) / 16 * 16
                                      : (in_lds == 2 ? ((size_t)V * 12 + 15) / 16 * 16 : 0);
  uint64_t *const cand_lds = reinterpret_cast<uint64_t *>(dyn + node_lds);
  // per-wave counts of the search (in LDS mode only)
  double *const s_part = reinterpret_cast<double *>(cand_lds + 2 * kCandLds);
  Nodes nd;
  if (in_lds == 1) {
    double *dp = reinterpret_cast<double *>(dyn);
    nd.W = dp;
    nd.w = dp + V;
    int32_t *ip = reinterpret_cast<int32_t *>(dp + 2 * V);
    nd.parent = ip;
    nd.n_full = ip + V;
    nd.n_kept = ip + 2 * V;
    nd.depth = ip + 3 * V;
    nd.down = ip + 4 * V;
    nd.F = ip + 5 * V;
    nd.cnt = ip + 6 * V;
    nd.cap = ip + 7 * V;
    nd.path = reinterpret_cast<uint8_t *>(ip + 8 * V);

    for (int i = tid; i < V; i += AT) {
      nd.parent[i] = i == tid ? par0 : t.parent[i];
      nd.n_full[i] = i == tid ? nf0 : t.n_full[i];
      nd.n_kept[i] = i == tid ? nk0 : t.n_kept[i];
    }
  } else {
    nd.parent = const_cast<int32_t *>(t.parent);
    nd.n_full = const_cast<int32_t *>(t.n_full);
    nd.n_kept = t.n_kept;
    nd.depth = ws.depth;
    nd.down = ws.down;
    if (in_lds == 2) {
      // the chain walks of the geometry (and the listing that later reuses
      // depth / down) run on LDS copies
      int32_t *ip = reinterpret_cast<int32_t *>(dyn);
      nd.parent = ip;
      nd.depth = ip + V;
      nd.down = ip + 2 * V;
      for (int i = tid; i < V; i += AT) nd.parent[i] = i == tid ? par0 : t.parent[i];
    }
    nd.F = ws.F;
    nd.cnt = ws.cnt;
    nd.cap = ws.cap;
    nd.W = ws.W;
    nd.w = ws.w;
    nd.path = on_path;
  }
  __syncthreads();

  // ---- geometry: validation, depth d_i, Path*, Delta_i (Sec. 3) ----------
  for (int i = tid; i < V; i += AT) {
    const int par = i == tid ? par0 : nd.parent[i];
    const int n = i == tid ? nf0 : nd.n_full[i];
    const int c = i == tid ? nk0 : nd.n_kept[i];
    bool ok = (i == 0) ? (par == -1) : (par >= 0 && par < i);
    ok = ok && n >= 0 && c >= 0 && c <= n;
    int d = 0;
    for (int a = i; ok && a > 0;) {
      const int pa = nd.parent[a];
      if (pa < 0 || pa >= a) {
        ok = false;
        break;
      }
      a = pa;
      ++d;
    }
    if (!ok) atomicOr(&s_err, 1);
    nd.depth[i] = d;
    nd.down[i] = 0x7fffffff;
    nd.path[i] = 0;
  }
  __syncthreads();
  if (n_active < 1) s_err = 1;
  __syncthreads();
  for (int j = tid; j < n_active && !s_err; j += AT) {
    const int l = active[j];
    if (l < 0 || l >= V) {
      atomicOr(&s_err, 1);
      continue;
    }
    const int dl = nd.depth[l];
    for (int a = l; a >= 0; a = nd.parent[a]) {
      nd.path[a] = 1;
      atomicMin(&nd.down[a], dl - nd.depth[a]);
    }
  }
  __syncthreads();
  if (s_err) {
    if (tid == 0) status_error(status, ARBOR_EINVAL);
    return;
  }
  // Delta_i = min over ancestors a (incl. i) of (d_i - d_a) + (distance from a
  // down to its nearest active leaf)
  // The eligible prices of each block (finite, at most alpha_max) and their
  // key range are counted here too, so one exchange gives every total.
  const double amax = p.alpha_max;
  int64_t path_tok = 0, sum_F = 0, sum_red = 0, total = 0, n_elig = 0;
  uint64_t kmin = ~0ull, kmax = 0ull;
  for (int i = tid; i < V; i += AT) {
    int best = 0x7fffffff;
    const int di = nd.depth[i];
    for (int a = i; a >= 0; a = nd.parent[a]) {
      const int dn = nd.down[a];
      if (dn != 0x7fffffff) best = min(best, di - nd.depth[a] + dn);
    }
    delta_out[i] = best;
    const int n = i == tid ? nf0 : nd.n_full[i];
    const int c = i == tid ? nk0 : nd.n_kept[i];
    const bool on = nd.path[i] != 0;
    if (in_lds == 1) on_path[i] = nd.path[i];
    // the most a block can keep: a Path* block is restored to n_i by
    // rehydration (or keeps c_i when evicted tokens stay lost), any other
    // block only ever loses tokens
    const int cap = on && p.rehydrate ? n : c;
    nd.cap[i] = cap;
    if (on && p.k_protect == 0) {
      // pinned (invariant (i), full protection)
      k_out[i] = cap;
      path_tok += cap;
      nd.F[i] = 0;
      nd.W[i] = 0.0;
      nd.w[i] = 0.0;
      nd.cnt[i] = 0;
      continue;
    }
    // s_i = clip(sigmoid(.), 0, 1) lies in [0, 1]
    const float sf = i == tid ? s0 : s_in[i];
    if (!(sf == sf)) atomicOr(&s_err, 2);
    else if (!(sf >= 0.f && sf <= 1.f)) atomicOr(&s_err, 4);
    const double s = (double)sf;
    // Eq. 3 at the ratio floor r_min, capped; a Path* block under floor
    // protection keeps at least k_protect
    int f = max(p.k_min, min(p.l_tail, n));
    f = max(f, (int)floor(p.r_min * (double)n));
    f = min(cap, min(n, f));
    if (on) f = max(f, min(cap, p.k_protect));
    nd.F[i] = f;
    // the Eq. 2 weight without alpha, in the same operation order as
    // ((eta^[off path] * s^gamma) * e^{-lambda_d d}) * e^{-lambda_Delta Delta}
    double w = (on ? 1.0 : p.eta) * pow_gamma(s, p.gamma);
    w = w * (di < kDecay ? s_dexp[di] : exp(-p.lambda_d * (double)di));
    w = w * (best < kDecay ? s_texp[best] : exp(-p.lambda_delta * (double)best));
    // -0 (s = -0 with an odd gamma) as +0: the Pressure order compares bit
    // patterns, in which -0 would rank above every positive weight
    w = w == 0.0 ? 0.0 : w;
    nd.w[i] = w;
    const double W = w * (double)n;
    nd.W[i] = W;
    sum_F += f;
    // Pressure lowers only off-path blocks
    if (!on) sum_red += f - min(p.k_min, c);
    const int cnt = eligible(f, cap, W, amax);
    nd.cnt[i] = cnt;
    total += cnt;
    if (cnt > 0) {
      const uint64_t lo = (uint64_t)__double_as_longlong(price(f + 1, W));
      const uint64_t hi = (uint64_t)__double_as_longlong(price(f + cnt, W));
      kmin = lo < kmin ? lo : kmin;
      kmax = hi > kmax ? hi : kmax;
      ++n_elig;
    }
  }
  {
    // five sums and two minima in one exchange (finite positive keys are
    // below 2^63: the maximum is taken as the minimum of INT64_MAX - key)
    int64_t v[7] = {path_tok, sum_F, sum_red, total, n_elig,
                    kmin == ~0ull ? INT64_MAX : (int64_t)kmin, INT64_MAX - (int64_t)kmax};
    block_reduce_n<5>(v, sm, V);
    path_tok = v[0];
    sum_F = v[1];
    sum_red = v[2];
    total = v[3];
    n_elig = v[4];
    kmin = (uint64_t)v[5];
    kmax = (uint64_t)(INT64_MAX - v[6]);
  }
  if (s_err) {
    if (tid == 0) status_error(status, (s_err & 2) ? ARBOR_ENONFINITE : ARBOR_EINVAL);
    return;
  }
  const int64_t b_off = budget - path_tok;

  if (sum_F <= b_off) {
    // ---- budget mode: alpha from the price order statistic ---------------
    const int64_t E = b_off - sum_F;
    if (total <= E) {
      for (int i = tid; i < V; i += AT)
        if (!(nd.path[i] && p.k_protect == 0)) k_out[i] = nd.F[i] + nd.cnt[i];
      return;
    }

    // Beyond LDS mode the blocks with eligible prices are listed once (F,
    // cnt, W side by side in the workspace), so that the search rounds, the
    // listing and the fill below visit only them.
    const int32_t *eF = nd.F;
    int32_t *eC = nd.cnt;
    const double *eW = nd.W;
    int ne = V;
    if constexpr (MODE != 1) {
      const int per = (V + AT - 1) / AT;
      const int i0 = min(V, tid * per), i1 = min(V, i0 + per);
      int64_t mine = 0;
#pragma unroll 4
      for (int i = i0; i < i1; ++i) mine += nd.cnt[i] > 0 ? 1 : 0;
      int64_t tot;
      int64_t off = block_exclusive_scan<int64_t>(mine, sm, &tot);
      for (int i = i0; i < i1; ++i) {
        const int cnt = nd.cnt[i];
        if (cnt > 0) {
          ws.eF[off] = nd.F[i];
          ws.eC[off] = cnt;
          ws.eW[off] = nd.W[i];
          ++off;
        }
      }
      __syncthreads();
      eF = ws.eF;
      eC = ws.eC;
      eW = ws.eW;
      ne = (int)tot;
    }

    // -- bracket: keys a (few prices <= a) and b (enough prices <= b) --------
    // The rounded count is off by at most two prices per node, so
    //   approx(a) <= E - 2 n_elig - 1  ->  exact(a) <= E - 1, and
    //   approx(b) >= E + 2 n_elig + 1  ->  exact(b) >= E + 1:
    // the order statistic lies in (a, b].  Each end has its own bracket
    // [lo, hi] around the crossing of its threshold; waves 0..7 test 32
    // points (four each) inside the bracket of a, waves 8..15 inside that of b.
    const double t_lo = (double)(E - 2 * n_elig - 1);
    const double t_hi = (double)(E + 2 * n_elig + 1);
    // a: approx(a_lo) <= t_lo < approx(a_hi); b: approx(b_lo) < t_hi, and
    // b_hi == kmax (exact count = total > E) or approx(b_hi) >= t_hi
    // (a zero price -- W_i infinite -- leaves no key below the smallest one:
    // then a stays "below everything" and every price up to b is listed)
    const bool a_none = kmin == 0;
    uint64_t a_lo = a_none ? 0 : kmin - 1, a_hi = kmax, b_lo = a_lo, b_hi = kmax;
    double ca = 0.0, cb = (double)total;
    bool a_done = a_none || t_lo < 0.0, b_done = a_none || t_hi > (double)total;
    // stop once the bracket holds few prices: listing them costs less than
    // another round
    const double enough = 256.0 + 4.0 * (double)n_elig;
    static_assert(2 * kSearchPts == kWave, "one lane per test point in the narrowing");
    // (trees held in LDS skip this search: their exact counts below cost
    // about as much as the rounded ones)
    for (int round = 0; MODE != 1 && !(a_done && b_done) && cb - ca > enough; ++round) {
      const bool end_b = wave >= kSearchWaves;
      const int q0 = (wave % kSearchWaves) * kPtsPerWave;
      const uint64_t lo = end_b ? b_lo : a_lo;
      const uint64_t span = (end_b ? b_hi : a_hi) - lo;
      uint64_t x[kPtsPerWave];
      double xv[kPtsPerWave], c[kPtsPerWave];
#pragma unroll
      for (int p = 0; p < kPtsPerWave; ++p) {
        x[p] = split_point<kSearchPts>(lo, span, q0 + p);
        xv[p] = key_value(x[p]);
        c[p] = 0.0;
      }
      if (!(end_b ? b_done : a_done)) {
        // (selects rather than a branch, so that the loads of several nodes
        // are in flight together; blocks without prices add 0)
#pragma unroll 4
        for (int e = lane; e < ne; e += kWave) {
          const int cnt = eC[e];
          const int F = eF[e];
          const double W = eW[e];
#pragma unroll
          for (int p = 0; p < kPtsPerWave; ++p) {
            const double y = approx_le(xv[p], F, cnt, W);
            c[p] += cnt > 0 ? y : 0.0;
          }
        }
#pragma unroll
        for (int p = 0; p < kPtsPerWave; ++p) c[p] = wave_sum(c[p]);
      }
      if (lane < kPtsPerWave) {
        const int slot = (end_b ? kSearchPts : 0) + q0 + lane;
        double cl = c[0];
        uint64_t xl = x[0];
#pragma unroll
        for (int p = 1; p < kPtsPerWave; ++p) {
          cl = lane == p ? c[p] : cl;
          xl = lane == p ? x[p] : xl;
        }
        s_cnt[round & 1][slot] = cl;
        s_x[round & 1][slot] = xl;
      }
      __syncthreads();
      // every wave narrows both brackets from the same counts: lane l holds
      // point l of end a (l < 32) or point l - 32 of end b.  The points ascend
      // and the counts with them, so the points at or below a threshold form
      // a prefix: one ballot finds its last point and the first point after it.
      const uint64_t xq = s_x[round & 1][lane];
      const double cq = s_cnt[round & 1][lane];
      const uint64_t m_a = ballot(lane < kSearchPts && cq <= t_lo);
      const uint64_t m_b = ballot(lane >= kSearchPts && cq < t_hi) >> kSearchPts;
      constexpr uint64_t kAll = (1ull << kSearchPts) - 1;
      if (!a_done) {
        if (m_a) {
          const int ql = 63 - __builtin_clzll(m_a);
          a_lo = lane_value(xq, ql);
          ca = lane_value(cq, ql);
        }
        const uint64_t above = ~m_a & kAll;
        if (above) {
          const uint64_t xh = lane_value(xq, __builtin_ctzll(above));
          a_hi = xh < a_hi ? xh : a_hi;
        }
        if (a_hi - a_lo <= 1) a_done = true;
      }
      if (!b_done) {
        if (m_b) {
          const uint64_t xl = lane_value(xq, kSearchPts + 63 - __builtin_clzll(m_b));
          b_lo = xl > b_lo ? xl : b_lo;
        }
        const uint64_t reach = ~m_b & kAll;
        if (reach) {
          const int qh = kSearchPts + __builtin_ctzll(reach);
          b_hi = lane_value(xq, qh);
          cb = lane_value(cq, qh);
        }
        if (b_hi - b_lo <= 1) b_done = true;
      }
    }
    const uint64_t a = a_lo, b = b_hi;

    if constexpr (MODE == 1) {
      // -- few nodes: narrow on exact counts --------------------------------
      // Keys ka < kb with count(<= ka) <= E < count(<= kb), from ka = the
      // smallest price's key - 1 (-1 when that price is 0: below every
      // price) and kb = the largest one's.  Each round tests ka, kb and 62
      // keys between them, one key per lane; the waves split the blocks,
      // whose exact counts (last_le) are added in wave order.  It stops when
      // kb - ka = 1 (the answer is kb) or when at most 64 prices lie in
      // (ka, kb], which are then listed and ranked by one wave.
      int64_t ka = a_none ? -1 : (int64_t)a, kb = (int64_t)b;
      int64_t cA = 0, cB = 0;
      bool counted = false;
      uint64_t answer = 0;
      bool found = false;
      for (int round = 0;; ++round) {
        if (kb - ka <= 1) {
          answer = (uint64_t)kb;
          found = true;
          break;
        }
        if (counted && cB - cA <= kWave) break;
        const uint64_t span = (uint64_t)(kb - ka);
        const uint64_t m = (uint64_t)lane;
        const int64_t x = lane == kWave - 1
                              ? kb
                              : ka + (int64_t)((span / (kWave - 1)) * m +
                                               ((span % (kWave - 1)) * m) / (kWave - 1));
        double c = 0.0;
        if (x >= 0) {
          const double xv = key_value((uint64_t)x);
#pragma unroll 4
          for (int i = wave; i < V; i += AT / kWave) {
            const int cnt = nd.cnt[i];
            const int F = nd.F[i];
            const int mm = cnt > 0 ? last_le(xv, F, cnt, nd.W[i]) : F;
            c += (double)(mm - F);
          }
        }
        s_part[tid] = c;
        __syncthreads();
        if (tid < kWave) {
          double sum = 0.0;
          for (int w = 0; w < AT / kWave; ++w) sum += s_part[w * kWave + tid];
          s_cnt[round & 1][tid] = sum;
          s_x[round & 1][tid] = (uint64_t)x;
        }
        __syncthreads();
        // the keys ascend and their counts with them: the last one with
        // count <= E is the new ka (lane 0 at least), the first one above E
        // the new kb (lane 63 at least)
        const double cq = s_cnt[round & 1][lane];
        const int64_t xq = (int64_t)s_x[round & 1][lane];
        const uint64_t le = ballot(cq <= (double)E);
        const int qa = 63 - __builtin_clzll(le);
        const int qb = __builtin_ctzll(~le);
        ka = lane_value(xq, qa);
        kb = lane_value(xq, qb);
        cA = (int64_t)lane_value(cq, qa);
        cB = (int64_t)lane_value(cq, qb);
        counted = true;
      }
      if (!found) {
        // the cB - cA <= 64 prices in (ka, kb], placed by a block scan and
        // ranked by one wave
        uint64_t *const lst = cand_lds;
        const double av1 = ka >= 0 ? key_value((uint64_t)ka) : 0.0, bv1 = key_value((uint64_t)kb);
        int m_lo = 0, m_hi = 0;
        double Wt = 0.0;
        if (tid < V && nd.cnt[tid] > 0) {
          const int F = nd.F[tid], cnt = nd.cnt[tid];
          Wt = nd.W[tid];
          m_lo = ka >= 0 ? last_le(av1, F, cnt, Wt) : F;
          m_hi = last_le(bv1, F, cnt, Wt);
        }
        int64_t tot;
        const int64_t off = block_exclusive_scan<int64_t>((int64_t)(m_hi - m_lo), sm, &tot);
        for (int j = m_lo; j < m_hi; ++j)
          lst[off + (j - m_lo)] = (uint64_t)__double_as_longlong(price(j + 1, Wt));
        __syncthreads();
        if (wave == 0) {
          const int n = (int)tot;
          const int64_t r = E - cA;
          const uint64_t key = lane < n ? lst[lane] : ~0ull;
          int less = 0, leq = 0;
          for (int q = 0; q < n; ++q) {
            const uint64_t kq = lane_value(key, q);
            less += kq < key ? 1 : 0;
            leq += kq <= key ? 1 : 0;
          }
          if (lane < n && less <= r && r < leq) s_x[0][0] = key;
        }
        __syncthreads();
        answer = s_x[0][0];
      }
      const double cut = key_value(answer);
      for (int i = tid; i < V; i += AT) {
        if (nd.path[i] && p.k_protect == 0) continue;
        const int F = nd.F[i];
        const double W = nd.W[i];
        k_out[i] = W > 0.0 ? last_lt(cut, F, nd.cap[i] - F, W) : F;
      }
      return;
    }

    // -- list the prices in (a, b] and count those <= a exactly -------------
    // per listed block e: first listed j - 1 in depth[e], how many in
    // down[e], offset in eC[e] (the geometry fields are no longer needed)
    const double av = key_value(a), bv = key_value(b);
    int64_t below = 0, run = 0;
    for (int base = 0; base < ne; base += AT) {
      const int e = base + tid;
      int m_lo = 0, m_hi = 0, F = 0;
      if (e < ne) {
        const int cnt = eC[e];
        if (cnt > 0) {
          F = eF[e];
          const double W = eW[e];
          m_lo = a_none ? F : last_le(av, F, cnt, W);
          m_hi = last_le(bv, F, cnt, W);
        }
      }
      // offsets of the listed prices, and the count of prices <= a
      const int64_t v2[2] = {(int64_t)(m_hi - m_lo), (int64_t)(m_lo - F)};
      int64_t ex[2], tot[2];
      block_exclusive_scan_n<2>(v2, ex, tot, sm, ne - base);
      if (e < ne) {
        nd.depth[e] = m_lo;
        nd.down[e] = m_hi - m_lo;
        eC[e] = (int)(run + ex[0]);
      }
      run += tot[0];
      below += tot[1];
    }
    const int64_t total_c = run;
    if (total_c > ws.buf_cap || total_c > 0x7fffffff) {
      if (tid == 0) status_error(status, ARBOR_EWORKSPACE);
      return;
    }
    // the listed prices and their order statistic (every listed key lies in
    // (a, b]); LDS and workspace buffers take separate code paths, so that
    // each compiles to its own kind of memory instruction
    auto order_stat = [&](uint64_t *cand, uint64_t *cand2) __attribute__((always_inline)) {
      // one thread per node over its listed prices (a few per node: the
      // bracket holds a few hundred in all)
      for (int e = tid; e < ne; e += AT) {
        const int nl = nd.down[e];
        const int m_lo = nd.depth[e], o = eC[e];
        const double W = eW[e];
        for (int j = 0; j < nl; ++j)
          cand[o + j] = (uint64_t)__double_as_longlong(price(m_lo + 1 + j, W));
      }
      __syncthreads();
      return select_rank(cand, cand2, total_c, E - below, sm, true, a_none ? 0 : a + 1, b);
    };
    const uint64_t prefix = total_c <= kCandLds ? order_stat(cand_lds, cand_lds + kCandLds)
                                                : order_stat(ws.buf0, ws.buf1);
    const double cut = key_value(prefix);
    for (int i = tid; i < V; i += AT) {
      if (nd.path[i] && p.k_protect == 0) continue;
      const int F = nd.F[i];
      const double W = nd.W[i];
      // the prices below the cut (none when W_i = 0: all infinite)
      k_out[i] = W > 0.0 ? last_lt(cut, F, nd.cap[i] - F, W) : F;
    }
    return;
  }

  // ---- pressure: drain the lowest-priority blocks (Alg. 2) ---------------
  int64_t excess = sum_F - b_off;
  if (sum_red < excess) {
    for (int i = tid; i < V; i += AT) {
      if (!nd.path[i]) k_out[i] = min(p.k_min, nd.n_kept[i]);
      else if (p.k_protect > 0) k_out[i] = nd.F[i];   // Path* keeps its floor
    }
    if (tid == 0) status_warn(status, ARBOR_OVER_BUDGET);
    return;
  }
  // smallest priority value W* whose cumulative reducible count reaches excess
  uint64_t prefix = 0, pmask = 0;
  int64_t need = excess;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int b = tid; b < 256; b += AT) hist64[b] = 0;
    __syncthreads();
    for (int i = tid; i < V; i += AT) {
      if (nd.path[i]) continue;
      const uint64_t key = (uint64_t)__double_as_longlong(nd.w[i]);
      if ((key & pmask) != prefix) continue;
      const int red = nd.F[i] - min(p.k_min, nd.n_kept[i]);
      if (red > 0) atomicAdd(&hist64[(key >> shift) & 255ull], (unsigned long long)red);
    }
    __syncthreads();
    int chosen = 255;
    int64_t acc = 0;
    for (int b = 0; b < 256; ++b) {
      const int64_t h = (int64_t)hist64[b];
      if (acc + h >= need) {
        chosen = b;
        break;
      }
      acc += h;
    }
    need -= acc;
    prefix |= (uint64_t)chosen << shift;
    pmask |= 255ull << shift;
    __syncthreads();
  }
  // nodes below W* drain fully; nodes at W* drain in id order until `need`
  int64_t run = 0;
  for (int base = 0; base < V; base += AT) {
    const int i = base + tid;
    int64_t red = 0;
    uint64_t key = 0;
    const bool off = i < V && !nd.path[i];
    if (off) {
      red = nd.F[i] - min(p.k_min, nd.n_kept[i]);
      key = (uint64_t)__double_as_longlong(nd.w[i]);
    }
    const bool tie = off && key == prefix;
    int64_t tot;
    const int64_t ex = block_exclusive_scan<int64_t>(tie ? red : 0, sm, &tot);
    if (off) {
      int kk = nd.F[i];
      if (key < prefix) {
        kk -= (int)red;
      } else if (tie) {
        const int64_t before = run + ex;
        if (before < need) kk -= (int)min<int64_t>(red, need - before);
      }
      k_out[i] = kk;
    } else if (i < V && p.k_protect > 0) {
      k_out[i] = nd.F[i];                                // Path* keeps its floor
    }
    run += tot;
  }
}

}  // namespace

size_t allocate_workspace(const arbor_sizes_t *sz) {
  return (size_t)sz->num_nodes * (5 * 4 + 8 * 2 + 2 * 4 + 8 + 64) +
         (size_t)sz->num_tokens * 16 + 8192;
}

// Per-event statistics of the device-side controller (arbor_walk): one
// workgroup after each allocation of a step.  transition = 1: row[0] = sum of
// the keep-counts, row[1] = tokens the rehydration of this step restores from
// the token store (Path* blocks with c_i < n_i), row[2] = tokens evicted
// (sum of c_i - k_i where k_i < c_i), row[3] = 0.  transition = 0 (the gated
// Pressure event, budget `budget`): if it fired (resident tokens >= budget),
// row[0] = the new sum, row[2] += its evictions, row[3] = 1.
__global__ __launch_bounds__(AT) void walk_stats(Tree t, const int32_t *__restrict__ k,
                                                 const uint8_t *__restrict__ on_path,
                                                 int64_t budget, int transition, int rehydrate,
                                                 int64_t *__restrict__ row, int32_t *status) {
  __shared__ int64_t sm[3 * 16];
  if (status_failed(status)) return;
  int64_t v[3] = {0, 0, 0};   // sum k, evicted, restored or resident
#pragma unroll 4
  for (int i = threadIdx.x; i < t.V; i += AT) {
    const int c = t.n_kept[i], ki = k[i], n = t.n_full[i];
    v[0] += ki;
    v[1] += ki < c ? c - ki : 0;
    v[2] += transition ? (on_path[i] && rehydrate && c < n ? n - c : 0) : c;
  }
  block_sum3(v, sm);
  if (threadIdx.x == 0) {
    if (transition) {
      row[0] = v[0];
      row[1] = v[2];
      row[2] = v[1];
      row[3] = 0;
    } else if (v[2] >= budget) {
      row[0] = v[0];
      row[2] += v[1];
      row[3] = 1;
    }
  }
}

int launch_walk_stats(const arbor_tree_t *tree, const int32_t *k, const uint8_t *on_path,
                      int64_t budget, int transition, int rehydrate, int64_t *row,
                      int32_t *status, hipStream_t stream) {
  Tree t = make_tree(tree);
  if (t.V <= 0) return ARBOR_OK;
  hipLaunchKernelGGL(walk_stats, dim3(1), dim3(AT), 0, stream, t, k, on_path, budget, transition,
                     rehydrate, row, status);
  return hip_ok(hipGetLastError());
}

int launch_allocate(const arbor_tree_t *tree, const int32_t *active, int32_t n_active,
                    int64_t budget_tokens, const float *s, const arbor_params_t *params,
                    int32_t *k_out, int32_t *delta_out, uint8_t *on_path_out, int32_t *status,
                    void *workspace, size_t workspace_bytes, hipStream_t stream, int gate) {
  Tree t = make_tree(tree);
  if (t.V <= 0) return ARBOR_OK;
  Carve cv(workspace, workspace_bytes);
  AllocWs ws;
  ws.depth = cv.take<int32_t>(t.V);
  ws.down = cv.take<int32_t>(t.V);
  ws.F = cv.take<int32_t>(t.V);
  ws.cnt = cv.take<int32_t>(t.V);
  ws.cap = cv.take<int32_t>(t.V);
  ws.W = cv.take<double>(t.V);
  ws.w = cv.take<double>(t.V);
  ws.eF = cv.take<int32_t>(t.V);
  ws.eC = cv.take<int32_t>(t.V);
  ws.eW = cv.take<double>(t.V);
  ws.buf0 = cv.take<uint64_t>((size_t)t.N);
  ws.buf1 = cv.take<uint64_t>((size_t)t.N);
  ws.buf_cap = t.N;
  if (!cv.ok) return ARBOR_EWORKSPACE;
  AllocParams p{params->alpha_max, params->gamma, params->lambda_d, params->lambda_delta,
                params->eta, params->r_min, params->k_min, params->l_tail,
                params->lazy_rehydration, params->k_protect, {}, {}};
  for (int i = 0; i < kDecay; ++i) {
    p.dexp[i] = exp(-params->lambda_d * (double)i);
    p.texp[i] = exp(-params->lambda_delta * (double)i);
  }
  const int in_lds = t.V <= kLdsNodes ? 1 : (t.V <= kGeoNodes ? 2 : 0);
  const void *fn = in_lds == 1 ? reinterpret_cast<const void *>(&allocate_kernel<1>)
                               : (in_lds == 2 ? reinterpret_cast<const void *>(&allocate_kernel<2>)
                                              : reinterpret_cast<const void *>(&allocate_kernel<0>));
  const size_t lds = (in_lds == 1 ? ((size_t)t.V * kNodeBytes + 15) / 16 * 16 + AT * 8
                                  : (in_lds == 2 ? ((size_t)t.V * 12 + 15) / 16 * 16 : 0)) +
                     2 * (size_t)kCandLds * sizeof(uint64_t);
  // more than 64 KiB of dynamic LDS has to be allowed explicitly
  static_assert(kGeoNodes * 12 + 2 * kCandLds * 8 <= 150 * 1024, "within the LDS of a CU");
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return ARBOR_EHIP;
#define ARBOR_ALLOC_LAUNCH(M)                                                                   \
  hipLaunchKernelGGL(allocate_kernel<M>, dim3(1), dim3(AT), lds, stream, t, active, n_active,    \
                     (int64_t)budget_tokens, s, p, k_out, delta_out, on_path_out, status, ws, gate)
  if (in_lds == 1) ARBOR_ALLOC_LAUNCH(1);
  else if (in_lds == 2) ARBOR_ALLOC_LAUNCH(2);
  else ARBOR_ALLOC_LAUNCH(0);
#undef ARBOR_ALLOC_LAUNCH
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
