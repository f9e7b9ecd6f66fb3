// arbor_score: MSVE scoring (Sec. 4 "Multi-Signal Value Estimation").
//
// The accumulated attention A_i(t) sums, over later query positions, over a
// thin slice of layers and over query heads, the softmax probability that each
// query puts on token t.  Here the later queries are the last-W window rows of
// every observer block j; a row's softmax runs over j's whole resident causal
// context (proper ancestors + own tokens up to the row), and the probability is
// credited to tokens of proper ancestors (u > b_i).
//
// A row's normaliser spans its whole chain, so there are two passes over the
// same (row, key) pairs, both as MFMA tiles of 16 keys (one 16-slot sub-page of
// the paged pool) by 16 query rows:
//   lse     C = K Q^T  (keys along M): each lane owns one query row and four
//           keys, so the running max / sum stay in-lane; rows are merged over
//           lane groups and waves at the end -> log2-sum-exp per row;
//   colsum  C = Q K^T  (rows along M): each lane owns one key and four rows, so
//           p = exp2(z - lse) sums over rows in-lane; one partial per
//           (observer, slice layer, kv head, row group, context key), no atomics;
//   reduce  per block i and 64-slot chunk: sum the partials of every observer
//           below i in observer order (fp64) into A, rows_seen;
//   final   a_i = sum_p A_i(p) / rows_seen_i, s_i = clip(sigmoid(theta.phi)).
// The Q operand of a wave stays in registers for the whole chain; keys are
// split over the 4 waves of a workgroup by sub-page.  The reduction dimension
// (head_dim) is permuted identically in both operands so that every lane reads
// one contiguous quarter of a K or Q row (64 B for bf16 d=128).
#include "arbor_internal.h"
#include "mfma_ops.h"

namespace arbor {

namespace {

constexpr int MAXD = ARBOR_MAX_DEPTH + 1;
constexpr float kLog2e = 1.4426950408889634f;

struct ScoreArgs {
  Tree t;
  Pool pl;
  const int32_t *obs;
  int n_obs;
  const void *q_win;
  int W;
  int S;
  int slice[8];
  int n_rg;
  float sl2;        // softmax scale * log2(e)
  int self_window;
  float *lse;       // [n_obs][S][Hkv][n_rg][16*NB]
  float *part;      // partial column sums
  const int64_t *pbase;   // [n_obs]
  const int32_t *ctxlen;  // [n_obs]
  const int32_t *odepth;  // [n_obs]
  const int32_t *anc;     // [n_obs][MAXD]
  int32_t *status;
};

// Chain of observer j in LDS, root first.
struct ChainLds {
  int node[MAXD];
  int c[MAXD];
  int64_t po[MAXD];
  int ctx[MAXD];      // context offset of the node's first slot
  int sp_off[MAXD + 1];
  int depth;
};

__device__ void build_chain(const Tree &t, int j, ChainLds &ch) {
  int d = 0;
  for (int x = t.parent[j]; x >= 0 && d < MAXD - 1; x = t.parent[x]) ++d;
  ch.depth = d;
  int e = d;
  for (int x = j; x >= 0 && e >= 0; x = t.parent[x]) ch.node[e--] = x;
  int ctx = 0, sp = 0;
  for (e = 0; e <= d; ++e) {
    const int x = ch.node[e];
    const int c = t.n_kept[x];
    ch.c[e] = c;
    ch.po[e] = t.page_off[x];
    ch.ctx[e] = ctx;
    ch.sp_off[e] = sp;
    ctx += c;
    sp += (c + 15) / 16;
  }
  ch.sp_off[d + 1] = sp;
}

template <int PASS, class T, int D, int NB>
__global__ __launch_bounds__(256) void score_pass(ScoreArgs a) {
  using O = Op<T>;
  constexpr int KS = D / 4 / O::kPerStep;  // MFMA k-steps over head_dim
  constexpr int QTR = D / 4;               // elements of a row per lane group
  __shared__ ChainLds ch;
  __shared__ float sm_m[4][16 * NB];
  __shared__ float sm_l[4][16 * NB];
  if (status_failed(a.status)) return;
  const Tree &t = a.t;
  const Pool &pl = a.pl;
  const int o = blockIdx.x;
  const int slg = blockIdx.y;
  const int rg = blockIdx.z;
  const int si = slg / pl.Hkv;
  const int g = slg % pl.Hkv;
  const int layer = a.slice[si];
  const int j = a.obs[o];
  if (threadIdx.x == 0) build_chain(t, j, ch);
  __syncthreads();
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int rr = lane & 15;
  const int g4 = lane >> 4;
  const int G = pl.G;
  const int nj = t.n_full[j];
  const int wj = min(a.W, nj);
  const int rows_total = G * a.W;
  const int own_d = ch.depth;

  // Q operand rows (query row of this lane in block nb: rg*16NB + nb*16 + rr)
  typename O::reg q[NB][KS];
  const T *qbase = static_cast<const T *>(a.q_win) +
                   ((((int64_t)o * a.S + si) * (pl.Hkv * G) + (int64_t)g * G) * a.W) * D;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int r = rg * 16 * NB + nb * 16 + rr;
    const bool rv = r < rows_total;
    const T *rp = qbase + (int64_t)(rv ? r : 0) * D + g4 * QTR;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) q[nb][ks] = rv ? O::load(rp + ks * O::kPerStep) : O::zero();
  }
  // window position u of a row, or -1 for an unused row
  auto row_u = [&](int r) -> int {
    if (r >= rows_total) return -1;
    const int tt = r % a.W;
    return tt < wj ? nj - wj + tt : -1;
  };

  const int64_t lse_base = ((((int64_t)o * a.S + si) * pl.Hkv + g) * a.n_rg + rg) * (16 * NB);
  const char *kbase = static_cast<const char *>(pl.k);
  const int esz = sizeof(T);

  if (PASS == 0) {
    int urow[NB];
    float m[NB], l[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      urow[nb] = row_u(rg * 16 * NB + nb * 16 + rr);
      m[nb] = -__builtin_inff();
      l[nb] = 0.f;
    }
    const int n_sp = ch.sp_off[own_d + 1];
    int d = 0;
    for (int sp = wave; sp < n_sp; sp += 4) {
      while (sp >= ch.sp_off[d + 1]) ++d;
      const int q0 = (sp - ch.sp_off[d]) * 16;      // first slot of the sub-page
      const int page = t.page_table[ch.po[d] + q0 / pl.P];
      const int r0 = q0 % pl.P;
      const int nvalid = min(16, ch.c[d] - q0);
      const bool own = d == own_d;
      // K operand: key rr of the sub-page
      typename O::reg kr[KS];
      const T *kp = reinterpret_cast<const T *>(kbase + row_byte_offset(pl, layer, page, g, r0 + rr)) +
                    g4 * QTR;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kr[ks] = O::load(kp + ks * O::kPerStep);
      int kpos[4] = {0, 0, 0, 0};
      if (own) {
        const int4 pv = *reinterpret_cast<const int4 *>(pl.slot_pos + (int64_t)page * pl.P + r0 + 4 * g4);
        kpos[0] = pv.x;
        kpos[1] = pv.y;
        kpos[2] = pv.z;
        kpos[3] = pv.w;
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) acc = O::mma(kr[ks], q[nb][ks], acc);
        float z[4];
        float mx = -__builtin_inff();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = 4 * g4 + e;
          const bool ok = key < nvalid && (!own || kpos[e] <= urow[nb]);
          z[e] = ok ? acc[e] * a.sl2 : -__builtin_inff();
          mx = fmaxf(mx, z[e]);
        }
        if (mx > m[nb]) {
          if (m[nb] > -__builtin_inff()) l[nb] *= __builtin_amdgcn_exp2f(m[nb] - mx);
          m[nb] = mx;
        }
        if (m[nb] > -__builtin_inff()) {
#pragma unroll
          for (int e = 0; e < 4; ++e) l[nb] += __builtin_amdgcn_exp2f(z[e] - m[nb]);
        }
      }
    }
    // merge the four lane groups that share a query row, then the waves
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int off = 16; off <= 32; off <<= 1) {
        const float mo = __shfl_xor(m[nb], off, kWave);
        const float lo = __shfl_xor(l[nb], off, kWave);
        const float mn = fmaxf(m[nb], mo);
        float ln = 0.f;
        if (mn > -__builtin_inff()) {
          ln = (m[nb] > -__builtin_inff() ? l[nb] * __builtin_amdgcn_exp2f(m[nb] - mn) : 0.f) +
               (mo > -__builtin_inff() ? lo * __builtin_amdgcn_exp2f(mo - mn) : 0.f);
        }
        m[nb] = mn;
        l[nb] = ln;
      }
      if (g4 == 0) {
        sm_m[wave][nb * 16 + rr] = m[nb];
        sm_l[wave][nb * 16 + rr] = l[nb];
      }
    }
    __syncthreads();
    for (int r = threadIdx.x; r < 16 * NB; r += blockDim.x) {
      float M = -__builtin_inff();
      for (int w = 0; w < 4; ++w) M = fmaxf(M, sm_m[w][r]);
      float L = 0.f;
      if (M > -__builtin_inff())
        for (int w = 0; w < 4; ++w)
          if (sm_m[w][r] > -__builtin_inff()) L += sm_l[w][r] * __builtin_amdgcn_exp2f(sm_m[w][r] - M);
      const bool valid = row_u(rg * 16 * NB + r) >= 0 && L > 0.f;
      a.lse[lse_base + r] = valid ? M + __log2f(L) : __builtin_inff();
    }
    return;
  }

  // ---- PASS 1: column sums of p = exp2(z - lse) over this row group -------
  float lse[NB][4];
  int urow[NB][4];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = nb * 16 + 4 * g4 + e;
      lse[nb][e] = a.lse[lse_base + r];
      urow[nb][e] = row_u(rg * 16 * NB + r);
    }
  const int n_sp = a.self_window ? ch.sp_off[own_d + 1] : ch.sp_off[own_d];
  float *pout = a.part + a.pbase[o] + (int64_t)(slg * a.n_rg + rg) * a.ctxlen[o];
  int d = 0;
  for (int sp = wave; sp < n_sp; sp += 4) {
    while (sp >= ch.sp_off[d + 1]) ++d;
    const int q0 = (sp - ch.sp_off[d]) * 16;
    const int page = t.page_table[ch.po[d] + q0 / pl.P];
    const int r0 = q0 % pl.P;
    const int nvalid = min(16, ch.c[d] - q0);
    const bool own = d == own_d;
    typename O::reg kr[KS];
    const T *kp = reinterpret_cast<const T *>(kbase + row_byte_offset(pl, layer, page, g, r0 + rr)) +
                  g4 * QTR;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kr[ks] = O::load(kp + ks * O::kPerStep);
    const int kpos = own ? pl.slot_pos[(int64_t)page * pl.P + r0 + rr] : 0;
    const bool kvalid = rr < nvalid;
    float colsum = 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) acc = O::mma(q[nb][ks], kr[ks], acc);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool ok = kvalid && (!own || kpos < urow[nb][e]);
        const float pz = __builtin_amdgcn_exp2f(acc[e] * a.sl2 - lse[nb][e]);
        colsum += ok ? pz : 0.f;
      }
    }
    colsum += __shfl_xor(colsum, 16, kWave);
    colsum += __shfl_xor(colsum, 32, kWave);
    if (g4 == 0 && kvalid) pout[ch.ctx[d] + q0 + rr] = colsum;
  }
}

// Observer chains, partial offsets and validation (one workgroup).
__global__ __launch_bounds__(1024) void score_plan(Tree t, const int32_t *__restrict__ obs, int n_obs,
                                                   int S, int Hkv, int n_rg, int64_t part_cap,
                                                   int64_t *__restrict__ pbase,
                                                   int32_t *__restrict__ ctxlen,
                                                   int32_t *__restrict__ odepth,
                                                   int32_t *__restrict__ anc, int32_t *status) {
  __shared__ int64_t sm[17];
  __shared__ int s_err;
  if (status_failed(status)) return;
  if (threadIdx.x == 0) s_err = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < t.V; i += blockDim.x) {
    const int par = t.parent[i];
    const bool ok = (i == 0) ? par == -1 : (par >= 0 && par < i);
    const int c = t.n_kept[i];
    if (!ok || c < 0 || c > t.n_full[i]) atomicOr(&s_err, 1);
  }
  __syncthreads();
  int64_t run = 0;
  for (int base = 0; base < n_obs; base += blockDim.x) {
    const int o = base + threadIdx.x;
    int64_t len = 0;
    if (o < n_obs) {
      const int j = obs[o];
      if (j < 0 || j >= t.V) {
        atomicOr(&s_err, 1);
      } else {
        int chainv[MAXD];
        int d = 0;
        bool ok = true;
        for (int x = j; x >= 0; x = t.parent[x]) {
          if (d >= MAXD || (x > 0 && (t.parent[x] < 0 || t.parent[x] >= x)) ||
              (x == 0 && t.parent[x] != -1)) {
            ok = false;
            break;
          }
          chainv[d++] = x;
          len += t.n_kept[x];
        }
        if (!ok) {
          atomicOr(&s_err, 2);
          d = 1;
        }
        odepth[o] = d - 1;
        for (int e = 0; e < d; ++e) anc[(int64_t)o * MAXD + e] = chainv[d - 1 - e];
      }
      ctxlen[o] = (int32_t)len;
    }
    int64_t tot;
    const int64_t ex = block_exclusive_scan<int64_t>(len * S * Hkv * n_rg, sm, &tot);
    if (o < n_obs) pbase[o] = run + ex;
    run += tot;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    if (s_err & 1) status_error(status, ARBOR_EINVAL);
    else if (s_err & 2) status_error(status, ARBOR_EUNSUPPORTED);
    else if (run > part_cap) status_error(status, ARBOR_EWORKSPACE);
  }
}

// A += partials of every observer below block i; rows_seen_i grows.
__global__ __launch_bounds__(256) void score_reduce(ScoreArgs a, float *__restrict__ A,
                                                    int64_t *__restrict__ rows_seen) {
  __shared__ int hits[256];
  __shared__ int s_nh;
  __shared__ int s_wcnt[4];
  __shared__ double s_acc[4][64];
  if (status_failed(a.status)) return;
  const Tree &t = a.t;
  const Pool &pl = a.pl;
  const int i = blockIdx.x;
  const int c = t.n_kept[i];
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  // depth and context offset of block i
  int di = 0, ctxoff = 0;
  for (int x = t.parent[i]; x >= 0 && di < MAXD; x = t.parent[x]) {
    ++di;
    ctxoff += t.n_kept[x];
  }
  const int nslab = a.S * pl.Hkv * a.n_rg;
  const int64_t tb = t.tok_off[i];
  const int64_t po = t.page_off[i];
  int64_t rows_add = 0;
  for (int ob = 0; ob < a.n_obs; ob += 256) {
    // observers that credit block i, in observer order
    const int o = ob + threadIdx.x;
    bool hit = false;
    if (o < a.n_obs) {
      const int od = a.odepth[o];
      hit = (od > di && a.anc[(int64_t)o * MAXD + di] == i) || (a.self_window && a.obs[o] == i);
    }
    const uint64_t bm = ballot(hit);
    if (lane == 0) s_wcnt[wave] = popc(bm);
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wave; ++w) before += s_wcnt[w];
    if (hit) hits[before + rank_below(bm, lane)] = o;
    if (threadIdx.x == 0) s_nh = s_wcnt[0] + s_wcnt[1] + s_wcnt[2] + s_wcnt[3];
    __syncthreads();
    const int nh = s_nh;
    if (blockIdx.y == 0 && threadIdx.x == 0) {
      for (int h = 0; h < nh; ++h) {
        const int jj = a.obs[hits[h]];
        rows_add += (int64_t)a.S * pl.Hkv * pl.G * min(a.W, t.n_full[jj]);
      }
    }
    // chunks of 64 slots; the 4 waves split the (hit, slab) pairs
    for (int chk = blockIdx.y; chk * 64 < c; chk += gridDim.y) {
      const int s = chk * 64 + lane;
      double acc = 0.0;
      if (s < c) {
        for (int e = wave; e < nh * nslab; e += 4) {
          const int h = e / nslab;
          const int sl = e % nslab;
          const int oo = hits[h];
          acc += (double)a.part[a.pbase[oo] + (int64_t)sl * a.ctxlen[oo] + ctxoff + s];
        }
      }
      s_acc[wave][lane] = acc;
      __syncthreads();
      if (wave == 0 && s < c) {
        const double tot = ((s_acc[0][lane] + s_acc[1][lane]) + s_acc[2][lane]) + s_acc[3][lane];
        const int page = t.page_table[po + s / pl.P];
        const int pos = pl.slot_pos[(int64_t)page * pl.P + s % pl.P];
        A[tb + pos] = (float)((double)A[tb + pos] + tot);
      }
      __syncthreads();
    }
  }
  if (blockIdx.y == 0 && threadIdx.x == 0) rows_seen[i] += rows_add;
}

// a_i and s_i from the updated A (one wave per block).
__global__ __launch_bounds__(256) void score_final(Tree t, const float *__restrict__ A,
                                                   const int64_t *__restrict__ rows_seen,
                                                   const float *__restrict__ v_in,
                                                   const float *__restrict__ u_in, float th0,
                                                   float th1, float th2, float *__restrict__ a_out,
                                                   float *__restrict__ s_out, int32_t *status) {
  if (status_failed(status)) return;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= t.V) return;
  const int lane = lane_id();
  const int64_t tb = t.tok_off[i];
  const int n = t.n_full[i];
  double sum = 0.0;
  for (int p = lane; p < n; p += kWave) sum += (double)A[tb + p];
  sum = wave_sum<double>(sum);
  if (lane == 0) {
    const int64_t rs = rows_seen[i];
    const double av = rs > 0 ? sum / (double)rs : 0.0;
    const double x = (double)th0 * (double)v_in[i] + (double)th1 * (double)u_in[i] + (double)th2 * av;
    double sv = 1.0 / (1.0 + exp(-x));
    sv = fmin(1.0, fmax(0.0, sv));
    a_out[i] = (float)av;
    s_out[i] = (float)sv;
  }
}

template <int PASS, class T, int D>
void launch_pass_nb(int NB, dim3 grid, hipStream_t stream, const ScoreArgs &a) {
  switch (NB) {
    case 1: hipLaunchKernelGGL((score_pass<PASS, T, D, 1>), grid, dim3(256), 0, stream, a); break;
    case 2: hipLaunchKernelGGL((score_pass<PASS, T, D, 2>), grid, dim3(256), 0, stream, a); break;
    case 4: hipLaunchKernelGGL((score_pass<PASS, T, D, 4>), grid, dim3(256), 0, stream, a); break;
    default: hipLaunchKernelGGL((score_pass<PASS, T, D, 8>), grid, dim3(256), 0, stream, a); break;
  }
}

template <int PASS>
void launch_pass(int dtype, int D, int NB, dim3 grid, hipStream_t stream, const ScoreArgs &a) {
  if (dtype == ARBOR_BF16) {
    if (D == 128) launch_pass_nb<PASS, __bf16, 128>(NB, grid, stream, a);
    else launch_pass_nb<PASS, __bf16, 64>(NB, grid, stream, a);
  } else {
    if (D == 128) launch_pass_nb<PASS, float, 128>(NB, grid, stream, a);
    else launch_pass_nb<PASS, float, 64>(NB, grid, stream, a);
  }
}

int rows_per_group(int rows_total) {
  int nb = (rows_total + 15) / 16;
  if (nb <= 1) return 1;
  if (nb <= 2) return 2;
  if (nb <= 4) return 4;
  return 8;
}

}  // namespace

size_t score_workspace(const arbor_geom_t *g, const arbor_sizes_t *sz) {
  const int rows_total = g->q_per_kv * sz->window;
  const int NB = rows_per_group(rows_total);
  const int n_rg = (rows_total + 16 * NB - 1) / (16 * NB);
  const size_t nobs = (size_t)(sz->max_observers > 0 ? sz->max_observers : 0);
  const size_t slabs = (size_t)sz->n_slice * g->num_kv_heads * n_rg;
  size_t b = 0;
  b += nobs * 8 + nobs * 4 * 2 + nobs * MAXD * 4 + 4 * 256;
  b += nobs * slabs * 16 * NB * 4 + 256;
  b += nobs * slabs * (size_t)sz->max_context * 4 + 256;
  return b;
}

int launch_score(const arbor_geom_t *geom, const arbor_tree_t *tree, const arbor_pool_t *pool,
                 const int32_t *observers, int32_t n_obs, const void *q_win, int32_t window,
                 const int32_t *slice_layers, int32_t n_slice, const float *v_in,
                 const float *u_in, float *A, int64_t *rows_seen, float *a_out, float *s_out,
                 const arbor_params_t *params, int32_t *status, void *workspace,
                 size_t workspace_bytes, hipStream_t stream) {
  Tree t = make_tree(tree);
  Pool pl = make_pool(geom, pool);
  if (t.V <= 0) return ARBOR_OK;
  ScoreArgs a;
  a.t = t;
  a.pl = pl;
  a.obs = observers;
  a.n_obs = n_obs;
  a.q_win = q_win;
  a.W = window;
  a.S = n_slice;
  for (int e = 0; e < 8; ++e) a.slice[e] = e < n_slice ? slice_layers[e] : 0;
  const int rows_total = pl.G * window;
  const int NB = rows_per_group(rows_total);
  a.n_rg = (rows_total + 16 * NB - 1) / (16 * NB);
  const float scale = params->softmax_scale > 0.f ? params->softmax_scale
                                                  : 1.0f / sqrtf((float)geom->head_dim);
  a.sl2 = scale * kLog2e;
  a.self_window = params->score_self_window;
  a.status = status;
  Carve cv(workspace, workspace_bytes);
  const size_t nobs = n_obs > 0 ? (size_t)n_obs : 1;
  int64_t *pbase = cv.take<int64_t>(nobs);
  int32_t *ctxlen = cv.take<int32_t>(nobs);
  int32_t *odepth = cv.take<int32_t>(nobs);
  int32_t *anc = cv.take<int32_t>(nobs * MAXD);
  const size_t slabs = (size_t)n_slice * pl.Hkv * a.n_rg;
  float *lse = cv.take<float>(nobs * slabs * 16 * NB);
  if (!cv.ok) return ARBOR_EWORKSPACE;
  float *part = reinterpret_cast<float *>(cv.rest());
  const int64_t part_cap = (int64_t)(cv.remaining() / 4);
  a.lse = lse;
  a.part = part;
  a.pbase = pbase;
  a.ctxlen = ctxlen;
  a.odepth = odepth;
  a.anc = anc;
  if (n_obs > 0) {
    hipLaunchKernelGGL(score_plan, dim3(1), dim3(1024), 0, stream, t, observers, n_obs, n_slice,
                       pl.Hkv, a.n_rg, part_cap, pbase, ctxlen, odepth, anc, status);
    const dim3 grid(n_obs, n_slice * pl.Hkv, a.n_rg);
    launch_pass<0>(geom->dtype, geom->head_dim, NB, grid, stream, a);
    launch_pass<1>(geom->dtype, geom->head_dim, NB, grid, stream, a);
    hipLaunchKernelGGL(score_reduce, dim3(t.V, 8), dim3(256), 0, stream, a, A, rows_seen);
  }
  hipLaunchKernelGGL(score_final, dim3((t.V + 3) / 4), dim3(256), 0, stream, t, A, rows_seen,
                     v_in, u_in, params->theta[0], params->theta[1], params->theta[2], a_out,
                     s_out, status);
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
