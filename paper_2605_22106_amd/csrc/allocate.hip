// arbor_allocate: tree-aware keep-counts under a global token budget.
//
// Eq. 2 gives the off-path retention ratio r_i = clip(alpha w_i, r_min, 1) with
// w_i = eta s_i^gamma e^{-lambda_d d_i} e^{-lambda_Delta Delta_i}; Eq. 3 turns it
// into k_i = min(n_i, max(K_min, |T_i|, floor(r_i n_i))).  The KKT view of
// Sec. 4 sets the one global scale alpha so that the total meets the budget.
// Token j of block i is kept exactly when alpha >= j / (w_i n_i) ("price"), so
// the largest feasible alpha keeps every price below the (E+1)-th smallest one,
// E being the budget left after the floors.  That order statistic is found by
// an MSB-first radix select over the fp64 bit patterns of the prices (positive
// doubles order like their bits).  Path* nodes (Alg. 2 Transition) are pinned
// at n_i; when the floors alone overflow (Alg. 2 Pressure) the lowest-priority
// blocks are drained towards K_min, found by a weighted radix select over the
// bit patterns of w_i.
//
// Everything runs in one 1024-thread workgroup: the work is O(V + sum of
// candidate tokens) and latency bound.  fp64, no contraction, so the prices
// are the same IEEE quotients any fp64 implementation computes.
#include "arbor_internal.h"

#pragma clang fp contract(off)

namespace arbor {

namespace {

constexpr int AT = 1024;

struct AllocParams {
  double alpha_max, gamma, lambda_d, lambda_delta, eta, r_min;
  int k_min, l_tail;
};

struct AllocWs {
  int32_t *depth;
  int32_t *down;
  int32_t *F;
  int32_t *cnt;        // eligible prices per node
  int64_t *cnt_off;    // exclusive prefix of cnt
  double *W;           // w_i * n_i
  double *w;
  uint64_t *buf0;
  uint64_t *buf1;
  int64_t buf_cap;
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

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
  for (int d = kWave / 2; d > 0; d >>= 1) {
    const uint64_t o = __shfl_xor(v, d, kWave);
    v = o < v ? o : v;
  }
  return v;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int d = kWave / 2; d > 0; d >>= 1) {
    const uint64_t o = __shfl_xor(v, d, kWave);
    v = o > v ? o : v;
  }
  return v;
}
__device__ uint64_t block_min_u64(uint64_t v, uint64_t *sm) {
  v = wave_min_u64(v);
  if (lane_id() == 0) sm[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t r = sm[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) r = sm[w] < r ? sm[w] : r;
  __syncthreads();
  return r;
}
__device__ uint64_t block_max_u64(uint64_t v, uint64_t *sm) {
  v = wave_max_u64(v);
  if (lane_id() == 0) sm[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t r = sm[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) r = sm[w] > r ? sm[w] : r;
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(AT) void allocate_kernel(Tree t, const int32_t *__restrict__ active,
                                                      int n_active, int64_t budget,
                                                      const float *__restrict__ s_in, AllocParams p,
                                                      int32_t *__restrict__ k_out,
                                                      int32_t *__restrict__ delta_out,
                                                      uint8_t *__restrict__ on_path,
                                                      int32_t *status, AllocWs ws) {
  __shared__ int64_t sm[17];
  __shared__ int s_err;
  __shared__ unsigned hist4[4 * 256];
  __shared__ unsigned long long hist64[256];
  __shared__ unsigned s_ncand;
  __shared__ uint64_t s_u64[17];
  __shared__ int64_t s_wtot[4];
  __shared__ int s_chosen;
  __shared__ int64_t s_below;
  if (status_failed(status)) return;
  const int tid = threadIdx.x;
  const int V = t.V;
  if (tid == 0) s_err = 0;
  __syncthreads();

  // ---- geometry: validation, depth d_i, Path*, Delta_i (Sec. 3) ----------
  for (int i = tid; i < V; i += AT) {
    const int par = t.parent[i];
    const int n = t.n_full[i];
    const int c = t.n_kept[i];
    bool ok = (i == 0) ? (par == -1) : (par >= 0 && par < i);
    ok = ok && n >= 0 && c >= 0 && c <= n;
    int d = 0;
    for (int a = i; ok && a > 0;) {
      const int pa = t.parent[a];
      if (pa < 0 || pa >= a) {
        ok = false;
        break;
      }
      a = pa;
      ++d;
    }
    if (!ok) atomicOr(&s_err, 1);
    ws.depth[i] = d;
    ws.down[i] = 0x7fffffff;
    on_path[i] = 0;
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
    const int dl = ws.depth[l];
    for (int a = l; a >= 0; a = t.parent[a]) {
      on_path[a] = 1;
      atomicMin(&ws.down[a], dl - ws.depth[a]);
    }
  }
  __syncthreads();
  if (s_err) {
    if (tid == 0) status_error(status, ARBOR_EINVAL);
    return;
  }
  // Delta_i = min over ancestors a (incl. i) of (d_i - d_a) + (distance from a
  // down to its nearest active leaf)
  int64_t path_tok = 0, sum_F = 0, sum_red = 0;
  for (int i = tid; i < V; i += AT) {
    int best = 0x7fffffff;
    const int di = ws.depth[i];
    for (int a = i; a >= 0; a = t.parent[a]) {
      const int dn = ws.down[a];
      if (dn != 0x7fffffff) best = min(best, di - ws.depth[a] + dn);
    }
    delta_out[i] = best;
    const int n = t.n_full[i];
    const int c = t.n_kept[i];
    if (on_path[i]) {
      k_out[i] = n;
      path_tok += n;
      ws.F[i] = 0;
      ws.W[i] = 0.0;
      ws.w[i] = 0.0;
      continue;
    }
    const float sf = s_in[i];
    if (!(sf == sf)) atomicOr(&s_err, 2);
    const double s = (double)sf;
    // Eq. 3 at the ratio floor r_min, capped at the resident count
    int f = max(p.k_min, min(p.l_tail, n));
    f = max(f, (int)floor(p.r_min * (double)n));
    f = min(c, min(n, f));
    ws.F[i] = f;
    // the off-path Eq. 2 weight without alpha, in the same operation order as
    // ((eta * s^gamma) * e^{-lambda_d d}) * e^{-lambda_Delta Delta}
    double w = p.eta * pow(s, p.gamma);
    w = w * exp(-p.lambda_d * (double)di);
    w = w * exp(-p.lambda_delta * (double)best);
    ws.w[i] = w;
    ws.W[i] = w * (double)n;
    sum_F += f;
    sum_red += f - min(p.k_min, c);
  }
  path_tok = block_sum<int64_t>(path_tok, sm);
  sum_F = block_sum<int64_t>(sum_F, sm);
  sum_red = block_sum<int64_t>(sum_red, sm);
  if (s_err) {
    if (tid == 0) status_error(status, ARBOR_ENONFINITE);
    return;
  }
  const int64_t b_off = budget - path_tok;

  if (sum_F <= b_off) {
    // ---- budget mode: alpha from the price order statistic ---------------
    const int64_t E = b_off - sum_F;
    const double amax = p.alpha_max;
    int64_t total = 0;
    for (int i = tid; i < V; i += AT) {
      int cnt = 0;
      if (!on_path[i]) {
        const double W = ws.W[i];
        cnt = count_prefix(ws.F[i], t.n_kept[i], W,
                           [amax](double x) { return x <= amax && x < __builtin_inf(); });
      }
      ws.cnt[i] = cnt;
      total += cnt;
    }
    total = block_sum<int64_t>(total, sm);
    if (total <= E) {
      for (int i = tid; i < V; i += AT)
        if (!on_path[i]) k_out[i] = ws.F[i] + ws.cnt[i];
      return;
    }
    if (total > ws.buf_cap) {
      if (tid == 0) status_error(status, ARBOR_EWORKSPACE);
      return;
    }
    // node offsets of the eligible prices
    int64_t run = 0;
    for (int base = 0; base < V; base += AT) {
      const int i = base + tid;
      const int64_t c = i < V ? ws.cnt[i] : 0;
      int64_t tot;
      const int64_t ex = block_exclusive_scan<int64_t>(c, sm, &tot);
      if (i < V) ws.cnt_off[i] = run + ex;
      run += tot;
    }
    __syncthreads();
    // materialise the price bit patterns, one wave per node
    {
      const int wave = tid >> 6, lane = lane_id();
      for (int i = wave; i < V; i += AT / kWave) {
        const int c = ws.cnt[i];
        if (c == 0) continue;
        const int64_t o = ws.cnt_off[i];
        const double W = ws.W[i];
        const int F = ws.F[i];
        for (int j = lane; j < c; j += kWave)
          ws.buf0[o + j] = (uint64_t)__double_as_longlong(price(F + 1 + j, W));
      }
    }
    __syncthreads();
    // the common high bits of all candidates need no pass
    uint64_t kmin = ~0ull, kmax = 0ull;
    for (int64_t e = tid; e < total; e += AT) {
      const uint64_t key = ws.buf0[e];
      kmin = key < kmin ? key : kmin;
      kmax = key > kmax ? key : kmax;
    }
    kmin = block_min_u64(kmin, s_u64);
    kmax = block_max_u64(kmax, s_u64);
    uint64_t prefix = kmin;
    int64_t rank = E;
    int64_t ncand = total;
    uint64_t *src = ws.buf0, *dst = ws.buf1;
    if (kmin != kmax) {
      const int top = 63 - __builtin_clzll(kmin ^ kmax);
      int shift = (top / 8) * 8;
      prefix = kmin & ~((shift + 8 >= 64) ? ~0ull : ((1ull << (shift + 8)) - 1ull));
      for (; shift >= 0; shift -= 8) {
        for (int b = tid; b < 4 * 256; b += AT) hist4[b] = 0;
        __syncthreads();
        unsigned *myh = hist4 + 256 * ((tid >> 6) & 3);
        for (int64_t e = tid; e < ncand; e += AT)
          atomicAdd(&myh[(src[e] >> shift) & 255ull], 1u);
        __syncthreads();
        // bin holding the element of rank `rank` (first 256 threads, 4 waves)
        const unsigned h = tid < 256
                               ? hist4[tid] + hist4[256 + tid] + hist4[512 + tid] + hist4[768 + tid]
                               : 0u;
        const int64_t inc = wave_inclusive_scan<int64_t>((int64_t)h);
        if (tid < 256 && lane_id() == kWave - 1) s_wtot[tid >> 6] = inc;
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
        const int chosen = s_chosen;
        rank -= s_below;
        prefix |= (uint64_t)chosen << shift;
        if (shift == 0) break;
        if (tid == 0) s_ncand = 0;
        __syncthreads();
        for (int64_t e0 = 0; e0 < ncand; e0 += AT) {
          const int64_t e = e0 + tid;
          const bool keep = e < ncand && (int)((src[e] >> shift) & 255ull) == chosen;
          const uint64_t bk = ballot(keep);
          unsigned base = 0;
          if (lane_id() == 0 && bk) base = atomicAdd(&s_ncand, (unsigned)popc(bk));
          base = __shfl(base, 0, kWave);
          if (keep) dst[base + rank_below(bk, lane_id())] = src[e];
        }
        __syncthreads();
        ncand = s_ncand;
        uint64_t *tmp = src;
        src = dst;
        dst = tmp;
        __syncthreads();
      }
    }
    const double cut = __longlong_as_double((long long)prefix);
    for (int i = tid; i < V; i += AT) {
      if (on_path[i]) continue;
      const int kept = count_prefix(ws.F[i], t.n_kept[i], ws.W[i],
                                    [cut](double x) { return x < cut; });
      k_out[i] = ws.F[i] + kept;
    }
    return;
  }

  // ---- pressure: drain the lowest-priority blocks (Alg. 2) ---------------
  int64_t excess = sum_F - b_off;
  if (sum_red < excess) {
    for (int i = tid; i < V; i += AT)
      if (!on_path[i]) k_out[i] = min(p.k_min, t.n_kept[i]);
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
      if (on_path[i]) continue;
      const uint64_t key = (uint64_t)__double_as_longlong(ws.w[i]);
      if ((key & pmask) != prefix) continue;
      const int red = ws.F[i] - min(p.k_min, t.n_kept[i]);
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
    if (i < V && !on_path[i]) {
      red = ws.F[i] - min(p.k_min, t.n_kept[i]);
      key = (uint64_t)__double_as_longlong(ws.w[i]);
    }
    const bool tie = i < V && !on_path[i] && key == prefix;
    int64_t tot;
    const int64_t ex = block_exclusive_scan<int64_t>(tie ? red : 0, sm, &tot);
    if (i < V && !on_path[i]) {
      int kk = ws.F[i];
      if (key < prefix) {
        kk -= (int)red;
      } else if (tie) {
        const int64_t before = run + ex;
        if (before < need) kk -= (int)min<int64_t>(red, need - before);
      }
      k_out[i] = kk;
    }
    run += tot;
  }
}

}  // namespace

size_t allocate_workspace(const arbor_sizes_t *sz) {
  return (size_t)sz->num_nodes * (4 * 4 + 8 * 3 + 64) + (size_t)sz->num_tokens * 16 + 8192;
}

int launch_allocate(const arbor_tree_t *tree, const int32_t *active, int32_t n_active,
                    int64_t budget_tokens, const float *s, const arbor_params_t *params,
                    int32_t *k_out, int32_t *delta_out, uint8_t *on_path_out, int32_t *status,
                    void *workspace, size_t workspace_bytes, hipStream_t stream) {
  Tree t = make_tree(tree);
  if (t.V <= 0) return ARBOR_OK;
  Carve cv(workspace, workspace_bytes);
  AllocWs ws;
  ws.depth = cv.take<int32_t>(t.V);
  ws.down = cv.take<int32_t>(t.V);
  ws.F = cv.take<int32_t>(t.V);
  ws.cnt = cv.take<int32_t>(t.V);
  ws.cnt_off = cv.take<int64_t>(t.V);
  ws.W = cv.take<double>(t.V);
  ws.w = cv.take<double>(t.V);
  ws.buf0 = cv.take<uint64_t>((size_t)t.N);
  ws.buf1 = cv.take<uint64_t>((size_t)t.N);
  ws.buf_cap = t.N;
  if (!cv.ok) return ARBOR_EWORKSPACE;
  AllocParams p{params->alpha_max, params->gamma, params->lambda_d, params->lambda_delta,
                params->eta, params->r_min, params->k_min, params->l_tail};
  hipLaunchKernelGGL(allocate_kernel, dim3(1), dim3(AT), 0, stream, t, active, n_active,
                     (int64_t)budget_tokens, s, p, k_out, delta_out, on_path_out, status, ws);
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
