// arbor_tree_decode_attn: decode attention of every active leaf over the
// resident tokens of its root-to-leaf chain (Sec. 1, Sec. 3: the next decoding
// step depends only on the ancestor chain).
//
// Tree-aware split-K: a work unit is (chain node a, chunk of a's slots, layer,
// kv head).  Its rows are the G query heads of every active leaf below a, so a
// shared ancestor is streamed from HBM once for all leaves that need it.  A
// wave computes S = K Q^T with bf16 MFMA (keys along M, so each lane owns one
// query row), an online softmax at 64-key granularity, and O += P V with fp32
// MFMA (16x16x4) so P is never rounded to bf16; the key order inside each MFMA
// step is permuted so P needs no cross-lane movement.  Each unit writes an
// unnormalised partial (max, sum, o); the merge kernel combines the partials of
// a leaf in root-to-leaf order, so results are bitwise reproducible.
#include "arbor_internal.h"
#include "mfma_ops.h"

namespace arbor {

namespace {

constexpr int MAXD = ARBOR_MAX_DEPTH + 1;
constexpr int CHUNK = 512;        // slots per work unit
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct DecArgs {
  Tree t;
  Pool pl;
  const int32_t *leaves;
  int n_leaves;
  int l0, Lr;
  const void *q;
  float sl2;
  // plan outputs
  const int32_t *meta;        // [0..2] items per class, [3] total rows
  const int32_t *cls_items;   // [3][max_items]
  int max_items;
  const int32_t *item_node;   // [items]
  const int32_t *item_chunk;
  const int32_t *item_rowbase;
  const int32_t *node_nl;     // leaves below a node (0 off the path)
  const int32_t *node_leaf_off;
  const int32_t *leaf_list;   // leaves below each node, in leaf order
  const int32_t *node_item0;  // first item of each path node
  const int32_t *node_rowbase;
  const int32_t *lanc;        // [n_leaves][MAXD]
  const int32_t *ldepth;
  const int32_t *lrank;       // [n_leaves][MAXD]
  float *part;
  int64_t part_cap;
  int32_t *status;
};

__global__ __launch_bounds__(1024) void decode_plan(DecArgs a, int32_t *meta, int32_t *cls_items,
                                                    int32_t *item_node, int32_t *item_chunk,
                                                    int32_t *item_rowbase, int32_t *node_nl,
                                                    int32_t *node_leaf_off, int32_t *leaf_list,
                                                    int32_t *node_item0, int32_t *node_rowbase,
                                                    int32_t *lanc, int32_t *ldepth,
                                                    int32_t *lrank) {
  __shared__ int64_t sm[17];
  __shared__ int s_err;
  if (status_failed(a.status)) {
    if (threadIdx.x == 0) meta[0] = meta[1] = meta[2] = 0;
    return;
  }
  const Tree &t = a.t;
  const int V = t.V;
  const int G = a.pl.G;
  if (threadIdx.x == 0) s_err = 0;
  for (int i = threadIdx.x; i < V; i += blockDim.x) node_nl[i] = 0;
  __syncthreads();
  for (int b = threadIdx.x; b < a.n_leaves; b += blockDim.x) {
    const int l = a.leaves[b];
    if (l < 0 || l >= V) {
      atomicOr(&s_err, 1);
      ldepth[b] = -1;
      continue;
    }
    int tmp[MAXD];
    int d = 0;
    bool ok = true;
    for (int x = l; x >= 0; x = t.parent[x]) {
      if (d >= MAXD || (x > 0 && (t.parent[x] < 0 || t.parent[x] >= x)) ||
          (x == 0 && t.parent[x] != -1)) {
        ok = false;
        break;
      }
      tmp[d++] = x;
    }
    if (!ok) {
      atomicOr(&s_err, 2);
      ldepth[b] = -1;
      continue;
    }
    ldepth[b] = d - 1;
    for (int e = 0; e < d; ++e) {
      const int x = tmp[d - 1 - e];
      lanc[(int64_t)b * MAXD + e] = x;
      atomicAdd(&node_nl[x], 1);
    }
  }
  __syncthreads();
  if (s_err) {
    if (threadIdx.x == 0) {
      status_error(a.status, (s_err & 1) ? ARBOR_EINVAL : ARBOR_EUNSUPPORTED);
      meta[0] = meta[1] = meta[2] = 0;
    }
    return;
  }
  // rank of each leaf among the leaves below each of its chain nodes
  for (int e = threadIdx.x; e < a.n_leaves * MAXD; e += blockDim.x) {
    const int b = e / MAXD, d = e % MAXD;
    if (d > ldepth[b]) continue;
    const int x = lanc[(int64_t)b * MAXD + d];
    int r = 0;
    for (int b2 = 0; b2 < b; ++b2)
      if (ldepth[b2] >= d && lanc[(int64_t)b2 * MAXD + d] == x) ++r;
    lrank[(int64_t)b * MAXD + d] = r;
  }
  // per-node offsets: leaf lists, items, partial rows; and class lists
  int64_t run_leaf = 0, run_item = 0, run_rows = 0, run_cls[3] = {0, 0, 0};
  for (int base = 0; base < V; base += blockDim.x) {
    const int i = base + threadIdx.x;
    const int nl = i < V ? node_nl[i] : 0;
    const int c = (i < V && nl > 0) ? t.n_kept[i] : 0;
    const int chunks = (c + CHUNK - 1) / CHUNK;
    const int rows = nl * G;
    const int nbr = (rows + 15) / 16;
    const int cls = nbr <= 1 ? 0 : (nbr <= 2 ? 1 : 2);
    int64_t tl, ti, tr, tc0, tc1, tc2;
    const int64_t el = block_exclusive_scan<int64_t>(nl, sm, &tl);
    const int64_t ei = block_exclusive_scan<int64_t>(chunks, sm, &ti);
    const int64_t er = block_exclusive_scan<int64_t>((int64_t)chunks * rows, sm, &tr);
    const int64_t e0 = block_exclusive_scan<int64_t>(cls == 0 ? chunks : 0, sm, &tc0);
    const int64_t e1 = block_exclusive_scan<int64_t>(cls == 1 ? chunks : 0, sm, &tc1);
    const int64_t e2 = block_exclusive_scan<int64_t>(cls == 2 ? chunks : 0, sm, &tc2);
    if (i < V) {
      node_leaf_off[i] = (int32_t)(run_leaf + el);
      node_item0[i] = (int32_t)(run_item + ei);
      node_rowbase[i] = (int32_t)(run_rows + er);
      const int64_t ce = cls == 0 ? run_cls[0] + e0 : (cls == 1 ? run_cls[1] + e1 : run_cls[2] + e2);
      for (int s = 0; s < chunks; ++s) {
        const int64_t it = run_item + ei + s;
        item_node[it] = i;
        item_chunk[it] = s;
        item_rowbase[it] = (int32_t)(run_rows + er + (int64_t)s * rows);
        cls_items[(int64_t)cls * a.max_items + ce + s] = (int32_t)it;
      }
    }
    run_leaf += tl;
    run_item += ti;
    run_rows += tr;
    run_cls[0] += tc0;
    run_cls[1] += tc1;
    run_cls[2] += tc2;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < a.n_leaves * MAXD; e += blockDim.x) {
    const int b = e / MAXD, d = e % MAXD;
    if (d > ldepth[b]) continue;
    const int x = lanc[(int64_t)b * MAXD + d];
    leaf_list[node_leaf_off[x] + lrank[(int64_t)b * MAXD + d]] = b;
  }
  if (threadIdx.x == 0) {
    const int64_t need = run_rows * a.Lr * a.pl.Hkv * (int64_t)(a.pl.D + 2);
    if (run_item > a.max_items || need > a.part_cap) {
      status_error(a.status, ARBOR_EWORKSPACE);
      meta[0] = meta[1] = meta[2] = 0;
      return;
    }
    meta[0] = (int32_t)run_cls[0];
    meta[1] = (int32_t)run_cls[1];
    meta[2] = (int32_t)run_cls[2];
    meta[3] = (int32_t)run_rows;
  }
}

// One wave: one work unit, rows [rbase, rbase + 16 NB).
template <class T, int D, int NB>
__device__ void decode_unit(const DecArgs &a, int item, int lr, int g, int rbase) {
  using O = Op<T>;
  constexpr int KS = D / 4 / O::kPerStep;  // MFMA k-steps over head_dim (S = K Q^T)
  constexpr int QTR = D / 4;
  constexpr int NC = D / 16;               // output column chunks; lane owns NC columns
  const Tree &t = a.t;
  const Pool &pl = a.pl;
  const int lane = lane_id();
  const int rr = lane & 15;
  const int g4 = lane >> 4;
  const int G = pl.G;
  const int node = a.item_node[item];
  const int chunk = a.item_chunk[item];
  const int nl = a.node_nl[node];
  const int R = nl * G;
  const int c = t.n_kept[node];
  const int s_begin = chunk * CHUNK;
  const int s_end = min(c, s_begin + CHUNK);
  const int layer = a.l0 + lr;
  const int Hq = pl.Hkv * G;
  const int64_t po = t.page_off[node];
  const int loff = a.node_leaf_off[node];

  // Q operand (S layout: lane owns row rbase + nb*16 + rr)
  typename O::reg q[NB][KS];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int r = rbase + nb * 16 + rr;
    if (r < R) {
      const int b = a.leaf_list[loff + r / G];
      const int h = g * G + r % G;
      const T *qp = static_cast<const T *>(a.q) + (((int64_t)b * a.Lr + lr) * Hq + h) * D + g4 * QTR;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) q[nb][ks] = O::load(qp + ks * O::kPerStep);
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) q[nb][ks] = O::zero();
    }
  }
  float m_run[NB], l_run[NB];
  f32x4 o[NB][NC];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m_run[nb] = -__builtin_inff();
    l_run[nb] = 0.f;
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) o[nb][cc] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const char *kb = static_cast<const char *>(pl.k);
  const char *vb = static_cast<const char *>(pl.v);
  for (int gs = s_begin; gs < s_end; gs += 64) {
    // phase A: logits of up to 4 sub-pages (64 keys)
    float sv[4][NB][4];
    float gmax[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) gmax[nb] = -__builtin_inff();
#pragma unroll
    for (int sp = 0; sp < 4; ++sp) {
      const int q0 = gs + sp * 16;
      if (q0 >= s_end) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int e = 0; e < 4; ++e) sv[sp][nb][e] = -__builtin_inff();
        continue;
      }
      const int page = t.page_table[po + q0 / pl.P];
      const int r0 = q0 % pl.P;
      const int nvalid = min(16, s_end - q0);
      const T *kp = reinterpret_cast<const T *>(kb + row_byte_offset(pl, layer, page, g, r0 + rr)) + g4 * QTR;
      typename O::reg kr[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kr[ks] = O::load(kp + ks * O::kPerStep);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) acc = O::mma(kr[ks], q[nb][ks], acc);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float z = (4 * g4 + e < nvalid) ? acc[e] * a.sl2 : -__builtin_inff();
          sv[sp][nb][e] = z;
          gmax[nb] = fmaxf(gmax[nb], z);
        }
      }
    }
    // row max over the group; rescale the running state
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      gmax[nb] = fmaxf(gmax[nb], __shfl_xor(gmax[nb], 16, kWave));
      gmax[nb] = fmaxf(gmax[nb], __shfl_xor(gmax[nb], 32, kWave));
      const float mn = fmaxf(m_run[nb], gmax[nb]);
      const float alpha = (m_run[nb] > -__builtin_inff()) ? __builtin_amdgcn_exp2f(m_run[nb] - mn) : 0.f;
      m_run[nb] = mn;
      l_run[nb] *= alpha;
      // O rows 4*g4+e take the factor of S-layout row 4*g4+e
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float fe = __shfl(alpha, 4 * g4 + e, kWave);
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) o[nb][cc][e] *= fe;
      }
    }
    // phase B: probabilities and O += P V (key 4*g4 + ks of the sub-page in
    // k-step ks, so P stays in the lane that computed it)
#pragma unroll
    for (int sp = 0; sp < 4; ++sp) {
      const int q0 = gs + sp * 16;
      if (q0 >= s_end) continue;
      const int page = t.page_table[po + q0 / pl.P];
      const int r0 = q0 % pl.P;
      float vr[4][NC];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const T *vp = reinterpret_cast<const T *>(vb + row_byte_offset(pl, layer, page, g, r0 + 4 * g4 + ks)) + NC * rr;
        load_row_f32<T, NC>(vp, vr[ks]);
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        float p[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          p[e] = (m_run[nb] > -__builtin_inff()) ? __builtin_amdgcn_exp2f(sv[sp][nb][e] - m_run[nb]) : 0.f;
          l_run[nb] += p[e];
        }
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
          for (int cc = 0; cc < NC; ++cc) o[nb][cc] = mma_f32(p[ks], vr[ks][cc], o[nb][cc]);
      }
    }
  }
  // write the unit's partial rows: [m, l, o(0..D-1)], o column NC*rr + cc
  const int64_t stride = D + 2;
  const int64_t slab = ((int64_t)lr * pl.Hkv + g) * a.meta[3];
  float *base = a.part + (slab + a.item_rowbase[item]) * stride;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float l = l_run[nb];
    l += __shfl_xor(l, 16, kWave);
    l += __shfl_xor(l, 32, kWave);
    const int rs = rbase + nb * 16 + rr;
    if (g4 == 0 && rs < R) {
      base[rs * stride + 0] = m_run[nb];
      base[rs * stride + 1] = l;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int ro = rbase + nb * 16 + 4 * g4 + e;
      if (ro < R) {
        float *op = base + ro * stride + 2 + NC * rr;
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) op[cc] = o[nb][cc][e];
      }
    }
  }
}

template <class T, int D, int NB>
__global__ __launch_bounds__(256) void decode_attn(DecArgs a, int cls) {
  if (status_failed(a.status)) return;
  const int n_items = a.meta[cls];
  const int planes = a.Lr * a.pl.Hkv;
  const int64_t total = (int64_t)n_items * planes;
  for (int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); w < total;
       w += (int64_t)gridDim.x * 4) {
    const int item = a.cls_items[(int64_t)cls * a.max_items + w / planes];
    const int rem = (int)(w % planes);
    const int lr = rem / a.pl.Hkv;
    const int g = rem % a.pl.Hkv;
    const int R = a.node_nl[a.item_node[item]] * a.pl.G;
    for (int rbase = 0; rbase < R; rbase += 16 * NB) decode_unit<T, D, NB>(a, item, lr, g, rbase);
  }
}

// One wave per (leaf, layer, kv head): merge the chain's partials root first.
template <int D>
__global__ __launch_bounds__(256) void decode_merge(DecArgs a, void *out, int out_dtype,
                                                    float *lse_out) {
  constexpr int EPL = D / 64;  // output columns per lane
  if (status_failed(a.status)) return;
  const Tree &t = a.t;
  const Pool &pl = a.pl;
  const int lane = lane_id();
  const int G = pl.G;
  const int Hq = pl.Hkv * G;
  const int64_t total = (int64_t)a.n_leaves * a.Lr * pl.Hkv;
  const int64_t stride = D + 2;
  for (int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); w < total;
       w += (int64_t)gridDim.x * 4) {
    const int b = (int)(w / (a.Lr * pl.Hkv));
    const int rem = (int)(w % (a.Lr * pl.Hkv));
    const int lr = rem / pl.Hkv;
    const int g = rem % pl.Hkv;
    const int64_t slab = ((int64_t)lr * pl.Hkv + g) * a.meta[3];
    const int dep = a.ldepth[b];
    for (int hl = 0; hl < G; ++hl) {
      float M = -__builtin_inff(), L = 0.f, ov[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) ov[e] = 0.f;
      for (int d = 0; d <= dep; ++d) {
        const int x = a.lanc[(int64_t)b * MAXD + d];
        const int row = a.lrank[(int64_t)b * MAXD + d] * G + hl;
        const int nch = (t.n_kept[x] + CHUNK - 1) / CHUNK;
        const int it0 = a.node_item0[x];
        for (int s = 0; s < nch; ++s) {
          const float *pp = a.part + (slab + a.item_rowbase[it0 + s] + row) * stride;
          const float m = pp[0];
          if (!(m > -__builtin_inff())) continue;
          const float l = pp[1];
          const float mn = fmaxf(M, m);
          const float fa = (M > -__builtin_inff()) ? __builtin_amdgcn_exp2f(M - mn) : 0.f;
          const float fb = __builtin_amdgcn_exp2f(m - mn);
          L = L * fa + l * fb;
#pragma unroll
          for (int e = 0; e < EPL; ++e) ov[e] = ov[e] * fa + pp[2 + 64 * e + lane] * fb;
          M = mn;
        }
      }
      const int h = g * G + hl;
      const int64_t oi = (((int64_t)b * a.Lr + lr) * Hq + h) * D;
      const float inv = L > 0.f ? 1.0f / L : 0.f;
      if (out_dtype == ARBOR_BF16) {
        __bf16 *op = static_cast<__bf16 *>(out) + oi;
#pragma unroll
        for (int e = 0; e < EPL; ++e) op[64 * e + lane] = (__bf16)(ov[e] * inv);
      } else {
        float *op = static_cast<float *>(out) + oi;
#pragma unroll
        for (int e = 0; e < EPL; ++e) op[64 * e + lane] = ov[e] * inv;
      }
      if (lse_out && lane == 0)
        lse_out[((int64_t)b * a.Lr + lr) * Hq + h] =
            L > 0.f ? (M + __log2f(L)) * kLn2 : -__builtin_inff();
    }
  }
}

template <class T, int D>
void launch_decode_kernels(const DecArgs &a, void *out, int out_dtype, float *lse_out,
                           hipStream_t stream) {
  const int grid = 2048;
  hipLaunchKernelGGL((decode_attn<T, D, 1>), dim3(grid), dim3(256), 0, stream, a, 0);
  hipLaunchKernelGGL((decode_attn<T, D, 2>), dim3(grid / 2), dim3(256), 0, stream, a, 1);
  hipLaunchKernelGGL((decode_attn<T, D, 4>), dim3(grid / 4), dim3(256), 0, stream, a, 2);
  const int64_t mw = (int64_t)a.n_leaves * a.Lr * a.pl.Hkv;
  const int mgrid = (int)((mw + 3) / 4 < 8192 ? (mw + 3) / 4 : 8192);
  hipLaunchKernelGGL((decode_merge<D>), dim3(mgrid), dim3(256), 0, stream, a, out, out_dtype,
                     lse_out);
}

}  // namespace

static size_t decode_max_items(const arbor_sizes_t *sz) {
  return (size_t)sz->num_nodes + (size_t)(sz->num_tokens / CHUNK) + 1;
}

size_t decode_workspace(const arbor_geom_t *g, const arbor_sizes_t *sz) {
  const size_t V = (size_t)sz->num_nodes;
  const size_t nl = (size_t)(sz->max_leaves > 0 ? sz->max_leaves : 1);
  const size_t items = decode_max_items(sz);
  const size_t per_leaf = (size_t)(sz->max_context / CHUNK) + MAXD + 1;
  const size_t rows = nl * per_leaf * g->q_per_kv;
  size_t b = 16 * 256;
  b += 3 * items * 4 + 3 * items * 4 + V * 4 * 4 + nl * MAXD * 4 * 3 + nl * 4 + nl * MAXD * 4;
  b += rows * (size_t)sz->max_layers * g->num_kv_heads * (g->head_dim + 2) * 4;
  return b;
}

int launch_decode(const arbor_geom_t *geom, const arbor_tree_t *tree, const arbor_pool_t *pool,
                  const int32_t *leaves, int32_t n_leaves, int32_t layer_begin, int32_t layer_end,
                  const void *q, void *out, int32_t out_dtype, float *lse_out, float softmax_scale,
                  int32_t *status, void *workspace, size_t workspace_bytes, hipStream_t stream) {
  Tree t = make_tree(tree);
  Pool pl = make_pool(geom, pool);
  if (t.V <= 0 || n_leaves <= 0 || layer_end <= layer_begin) return ARBOR_OK;
  arbor_sizes_t sz{};
  sz.num_nodes = t.V;
  sz.num_tokens = t.N;
  sz.max_context = t.N;
  sz.max_leaves = n_leaves;
  const int max_items = (int)decode_max_items(&sz);
  DecArgs a;
  a.t = t;
  a.pl = pl;
  a.leaves = leaves;
  a.n_leaves = n_leaves;
  a.l0 = layer_begin;
  a.Lr = layer_end - layer_begin;
  a.q = q;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf((float)geom->head_dim);
  a.sl2 = scale * kLog2e;
  a.max_items = max_items;
  a.status = status;
  Carve cv(workspace, workspace_bytes);
  int32_t *meta = cv.take<int32_t>(8);
  int32_t *cls_items = cv.take<int32_t>((size_t)3 * max_items);
  int32_t *item_node = cv.take<int32_t>(max_items);
  int32_t *item_chunk = cv.take<int32_t>(max_items);
  int32_t *item_rowbase = cv.take<int32_t>(max_items);
  int32_t *node_nl = cv.take<int32_t>(t.V);
  int32_t *node_leaf_off = cv.take<int32_t>(t.V);
  int32_t *node_item0 = cv.take<int32_t>(t.V);
  int32_t *node_rowbase = cv.take<int32_t>(t.V);
  int32_t *leaf_list = cv.take<int32_t>((size_t)n_leaves * MAXD);
  int32_t *lanc = cv.take<int32_t>((size_t)n_leaves * MAXD);
  int32_t *ldepth = cv.take<int32_t>(n_leaves);
  int32_t *lrank = cv.take<int32_t>((size_t)n_leaves * MAXD);
  if (!cv.ok) return ARBOR_EWORKSPACE;
  a.meta = meta;
  a.cls_items = cls_items;
  a.item_node = item_node;
  a.item_chunk = item_chunk;
  a.item_rowbase = item_rowbase;
  a.node_nl = node_nl;
  a.node_leaf_off = node_leaf_off;
  a.leaf_list = leaf_list;
  a.node_item0 = node_item0;
  a.node_rowbase = node_rowbase;
  a.lanc = lanc;
  a.ldepth = ldepth;
  a.lrank = lrank;
  a.part = reinterpret_cast<float *>(cv.rest());
  a.part_cap = (int64_t)(cv.remaining() / 4);
  hipLaunchKernelGGL(decode_plan, dim3(1), dim3(1024), 0, stream, a, meta, cls_items, item_node,
                     item_chunk, item_rowbase, node_nl, node_leaf_off, leaf_list, node_item0,
                     node_rowbase, lanc, ldepth, lrank);
  if (geom->dtype == ARBOR_BF16) {
    if (geom->head_dim == 128) launch_decode_kernels<__bf16, 128>(a, out, out_dtype, lse_out, stream);
    else launch_decode_kernels<__bf16, 64>(a, out, out_dtype, lse_out, stream);
  } else {
    if (geom->head_dim == 128) launch_decode_kernels<float, 128>(a, out, out_dtype, lse_out, stream);
    else launch_decode_kernels<float, 64>(a, out, out_dtype, lse_out, stream);
  }
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
