// arbor_tree_decode_attn: decode attention of every active leaf over the
// resident tokens of its root-to-leaf chain (Sec. 1, Sec. 3: the next decoding
// step depends only on the ancestor chain).
//
// Tree-aware split-K: a work unit is (chain node a, chunk of a's slots, layer,
// kv head).  Its rows are the G query heads of every active leaf below a, so a
// shared ancestor is streamed from HBM once for all leaves that need it.  A
// wave computes S = K Q^T with bf16 MFMA (keys along M, so each lane owns one
// query row), an online softmax per fragment of keys, and O += P V.  For
// bf16 pools P is split into a bf16 high part and a bf16 remainder, both
// multiplied with the exact bf16 V by bf16 MFMAs (fp32-level accuracy of P);
// fp32 pools use the fp32 MFMA (16x16x4).  The key order inside each MFMA
// step is permuted so P needs no cross-lane movement.  Each unit writes an
// unnormalised partial (max, sum, o); the merge kernel combines the partials of
// a leaf in root-to-leaf order, so results are bitwise reproducible.
#include <type_traits>

#include "arbor_internal.h"
#include "mfma_ops.h"

namespace arbor {

namespace {

constexpr int MAXD = ARBOR_MAX_DEPTH + 1;
static_assert(MAXD == kWave, "one wave covers a chain");
constexpr int CHUNK = 256;        // slots per work unit
constexpr int kPlanLds = 4096;    // trees up to this many nodes are planned from LDS
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
  const int32_t *leaf_np;     // partials of each leaf's chain
  const int32_t *leaf_part;   // [n_leaves][max_parts]: first partial row of the leaf's heads
  int max_parts;
  float *part;
  int64_t part_cap;
  int zS;                     // credit calls: distinct slice layers whose logits the units keep
  int zlr[8];                 //   (relative to l0); zS = 0 otherwise
  int32_t *status;
};

// The decode-time credit of accumulated attention: slice layers relative to
// the call's first layer, the crediting mode and the caller's A / rows_seen.
struct CreditArgs {
  int S;          // slice entries (a layer may be listed more than once)
  int U;          // distinct slice layers: the units keep logits for these
  int slice[8];   // distinct slice layers
  int mult[8];    //   and how often each is listed
  int self_window;
  float *A;
  int64_t *rows_seen;
};

// Plan of one call, in one workgroup: each active leaf's chain (root first),
// the leaves below every node (in leaf order), the work units (chunks of the
// chain nodes' slots, per class of row count), each unit's partial rows and
// each leaf's list of partials, root first.  The per-node and per-leaf state
// sits in LDS for trees of up to kPlanLds nodes and up to kPlanLeaves leaves,
// so the chain walks, ranks and scans wait on global memory only for the
// tree's arrays.  SMALL / FEW are template arguments, so that every access
// compiles to an LDS or a global instruction rather than a flat one.
constexpr int kPlanLeaves = 64;
template <bool SMALL, bool FEW>
__global__ __launch_bounds__(1024) void decode_plan(DecArgs a, int32_t *meta, int32_t *cls_items,
                                                    int32_t *item_node, int32_t *item_chunk,
                                                    int32_t *item_rowbase, int32_t *node_nl,
                                                    int32_t *node_leaf_off, int32_t *leaf_list,
                                                    int32_t *node_item0, int32_t *node_rowbase,
                                                    int32_t *lanc, int32_t *ldepth,
                                                    int32_t *lrank, int32_t *leaf_np,
                                                    int32_t *leaf_part) {
  __shared__ int64_t sm[6 * 16];
  __shared__ int s_err;
  __shared__ int32_t s_par[kPlanLds], s_nl[kPlanLds], s_kept[kPlanLds], s_loff[kPlanLds],
      s_rbase[kPlanLds], s_item0[kPlanLds];
  __shared__ int32_t s_lanc[kPlanLeaves * MAXD], s_lrank[kPlanLeaves * MAXD], s_ldep[kPlanLeaves];
  const Tree &t = a.t;
  const int V = t.V;
  const int G = a.pl.G;
  const int nt = blockDim.x;
  const int tid = threadIdx.x;
  // each thread's first node and leaf are loaded together with the status word
  const int par0 = tid < V ? t.parent[tid] : 0, kept0 = tid < V ? t.n_kept[tid] : 0;
  const int leaf0 = tid < a.n_leaves ? a.leaves[tid] : 0;
  if (status_failed(a.status)) {
    if (threadIdx.x == 0) meta[0] = meta[1] = meta[2] = 0;
    return;
  }
  constexpr bool small = SMALL;
  constexpr bool few = FEW;
  const int32_t *par = small ? s_par : t.parent;
  const int32_t *kept = small ? s_kept : t.n_kept;
  int32_t *nlp = small ? s_nl : node_nl;
  int32_t *loffp = small ? s_loff : node_leaf_off;
  int32_t *rbasep = small ? s_rbase : node_rowbase;
  int32_t *item0p = small ? s_item0 : node_item0;
  int32_t *lancp = few ? s_lanc : lanc;
  int32_t *lrankp = few ? s_lrank : lrank;
  int32_t *ldepp = few ? s_ldep : ldepth;
  if (tid == 0) s_err = 0;
  for (int i = tid; i < V; i += nt) {
    nlp[i] = 0;
    if (small) {
      s_par[i] = i == tid ? par0 : t.parent[i];
      s_kept[i] = i == tid ? kept0 : t.n_kept[i];
    }
  }
  __syncthreads();
  for (int b = tid; b < a.n_leaves; b += nt) {
    const int l = b == tid ? leaf0 : a.leaves[b];
    if (l < 0 || l >= V) {
      atomicOr(&s_err, 1);
      ldepp[b] = -1;
      continue;
    }
    // validate and measure the chain, then write it root first (two walks up
    // the parent links keep the chain out of per-lane scratch memory)
    int d = 0, bad = 0;
    for (int x = l; x >= 0; x = par[x]) {
      if ((x > 0 && (par[x] < 0 || par[x] >= x)) || (x == 0 && par[x] != -1)) {
        bad = 1;
        break;
      }
      if (++d > MAXD) {
        bad = 2;
        break;
      }
    }
    if (bad) {
      atomicOr(&s_err, bad);
      ldepp[b] = -1;
      continue;
    }
    ldepp[b] = d - 1;
    int e = d - 1;
    for (int x = l; x >= 0; x = par[x], --e) {
      lancp[(int64_t)b * MAXD + e] = x;
      atomicAdd(&nlp[x], 1);
    }
  }
  __syncthreads();
  if (s_err) {
    if (tid == 0) {
      status_error(a.status, (s_err & 1) ? ARBOR_EINVAL : ARBOR_EUNSUPPORTED);
      meta[0] = meta[1] = meta[2] = 0;
    }
    return;
  }
  // rank of each leaf among the leaves below each of its chain nodes
  for (int e = tid; e < a.n_leaves * MAXD; e += nt) {
    const int b = e / MAXD, d = e % MAXD;
    if (d > ldepp[b]) continue;
    const int x = lancp[(int64_t)b * MAXD + d];
    int r = 0;
    for (int b2 = 0; b2 < b; ++b2)
      if (ldepp[b2] >= d && lancp[(int64_t)b2 * MAXD + d] == x) ++r;
    lrankp[(int64_t)b * MAXD + d] = r;
  }
  // per-node offsets: leaf lists, items, partial rows; and class lists
  int64_t run_leaf = 0, run_item = 0, run_rows = 0, run_cls[3] = {0, 0, 0};
  for (int base = 0; base < V; base += nt) {
    const int i = base + tid;
    const int nl = i < V ? nlp[i] : 0;
    if (small && i < V) node_nl[i] = nl;
    const int c = (i < V && nl > 0) ? kept[i] : 0;
    const int chunks = (c + CHUNK - 1) / CHUNK;
    const int rows = nl * G;
    const int nbr = (rows + 15) / 16;
    const int cls = nbr <= 1 ? 0 : (nbr <= 2 ? 1 : 2);
    const int64_t sv[6] = {nl, chunks, (int64_t)chunks * rows, cls == 0 ? chunks : 0,
                           cls == 1 ? chunks : 0, cls == 2 ? chunks : 0};
    int64_t sx[6], stot[6];
    block_exclusive_scan_n<6>(sv, sx, stot, sm);
    if (i < V) {
      const int lo = (int32_t)(run_leaf + sx[0]);
      const int it0 = (int32_t)(run_item + sx[1]);
      const int rb = (int32_t)(run_rows + sx[2]);
      loffp[i] = lo;
      item0p[i] = it0;
      rbasep[i] = rb;
      if (small) {
        node_leaf_off[i] = lo;
        node_item0[i] = it0;
        node_rowbase[i] = rb;
      }
      const int64_t ce = cls == 0 ? run_cls[0] + sx[3]
                                  : (cls == 1 ? run_cls[1] + sx[4] : run_cls[2] + sx[5]);
      for (int q = 0; q < chunks; ++q) {
        const int64_t it = it0 + q;
        item_node[it] = i;
        item_chunk[it] = q;
        item_rowbase[it] = (int32_t)(rb + (int64_t)q * rows);
        cls_items[(int64_t)cls * a.max_items + ce + q] = (int32_t)it;
      }
    }
    run_leaf += stot[0];
    run_item += stot[1];
    run_rows += stot[2];
    run_cls[0] += stot[3];
    run_cls[1] += stot[4];
    run_cls[2] += stot[5];
  }
  __syncthreads();
  for (int e = tid; e < a.n_leaves * MAXD; e += nt) {
    const int b = e / MAXD, d = e % MAXD;
    if (d > ldepp[b]) continue;
    const int x = lancp[(int64_t)b * MAXD + d];
    leaf_list[loffp[x] + lrankp[(int64_t)b * MAXD + d]] = b;
    if (few) lanc[(int64_t)b * MAXD + d] = x;
  }
  if (few)
    for (int b = tid; b < a.n_leaves; b += nt) ldepth[b] = s_ldep[b];
  // each leaf's partials, root first, so the merge needs no chain walk: one
  // thread per (leaf, chain depth); the offsets come from a per-leaf scan of
  // the chunk counts along the chain (at most MAXD entries)
  for (int b0 = 0; b0 < a.n_leaves; b0 += nt / MAXD) {
    const int b = b0 + tid / MAXD;
    const int d = tid % MAXD;
    const bool live = b < a.n_leaves && d <= ldepp[b];
    int x = 0, nch = 0;
    if (live) {
      x = lancp[(int64_t)b * MAXD + d];
      nch = (kept[x] + CHUNK - 1) / CHUNK;
    }
    // inclusive scan over the MAXD threads of this leaf (MAXD = kWave)
    const int incl = wave_inclusive_scan<int>(nch);
    const int np = incl - nch;
    if (live) {
      const int r = lrankp[(int64_t)b * MAXD + d] * G;
      const int rows = nlp[x] * G;
      if (incl > a.max_parts) {
        atomicOr(&s_err, 4);  // more resident tokens than the workspace was sized for
      } else {
        for (int q = 0; q < nch; ++q)
          leaf_part[(int64_t)b * a.max_parts + np + q] = rbasep[x] + q * rows + r;
      }
      if (d == ldepp[b]) leaf_np[b] = min(incl, a.max_parts);
    }
  }
  __syncthreads();
  if (tid == 0) {
    // the partials, then (credit calls) the slice-layer logits of every unit
    // row and slot: [slice][kv head][row][CHUNK]
    const int64_t need_p = (run_rows * a.Lr * a.pl.Hkv * (int64_t)(a.pl.D + 2) + 3) & ~(int64_t)3;
    const int64_t need = need_p + (int64_t)a.zS * a.pl.Hkv * run_rows * CHUNK;
    if (run_item > a.max_items || need > a.part_cap || need_p > INT32_MAX || s_err) {
      status_error(a.status, ARBOR_EWORKSPACE);
      meta[0] = meta[1] = meta[2] = 0;
      return;
    }
    meta[0] = (int32_t)run_cls[0];
    meta[1] = (int32_t)run_cls[1];
    meta[2] = (int32_t)run_cls[2];
    meta[3] = (int32_t)run_rows;
    meta[4] = (int32_t)need_p;
  }
}

// K and V of GSP consecutive 16-slot sub-pages of one unit, in MFMA operand
// layout: lane (rr, g4) holds key row rr of each sub-page (S = K Q^T), and
// value rows 4 g4 + e, columns NC rr .. NC rr + NC - 1 (O += P V).
template <class T, int D, int GSP>
struct KVFrag {
  typedef typename std::conditional<sizeof(T) == 2, __bf16, float>::type VT;
  static constexpr int KS = D / 4 / Op<T>::kPerStep;
  static constexpr int NC = D / 16;
  typename Op<T>::reg k[GSP][KS];
  VT v[GSP][4][NC];
  int nval[GSP];  // valid slots of each sub-page (0: padding, never counted); wave-uniform
};

// Where a unit's rows live: the (layer, kv head) plane of K and V at page 0,
// the bytes between pages, and this lane's offsets within a 16-row sub-page.
struct UnitAddr {
  const char *k, *v;
  int64_t page_bytes;
  int row_bytes;
  uint32_t koff, voff;
};

template <class T, int D, int GSP>
__device__ __forceinline__ KVFrag<T, D, GSP> fetch_kv(const UnitAddr &ua, int pg, int s_begin,
                                                      int s_end, int n_sub, int sub0, int P) {
  typedef KVFrag<T, D, GSP> F;
  F f;
#pragma unroll
  for (int sp = 0; sp < GSP; ++sp) {
    // clamped to a valid sub-page so that every load is unconditional
    const int sub = min(sub0 + sp, n_sub - 1);
    const int q0 = s_begin + sub * 16;
    f.nval[sp] = sub0 + sp < n_sub ? min(16, s_end - q0) : 0;
    // lane j holds sub-page j's page; the page base is wave-uniform
    const int page = __builtin_amdgcn_readlane(pg, sub);
    const int64_t base = (int64_t)page * ua.page_bytes + (int64_t)(q0 % P) * ua.row_bytes;
    const char *kp = ua.k + base + ua.koff;
    const char *vp = ua.v + base + ua.voff;
#pragma unroll
    for (int ks = 0; ks < F::KS; ++ks)
      f.k[sp][ks] = Op<T>::load(reinterpret_cast<const T *>(kp + frag_col<T>(ks, 0) * (int)sizeof(T)));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const typename F::VT *vr = reinterpret_cast<const typename F::VT *>(vp + e * ua.row_bytes);
#pragma unroll
      for (int cc = 0; cc < F::NC; ++cc) f.v[sp][e][cc] = vr[cc];
    }
  }
  return f;
}

// Online-softmax update of one wave's rows with one fragment.  Slots past a
// sub-page's resident count may hold anything: only a ragged sub-page (the
// last of a node) masks its logits and zeroes its value rows.  The output is
// rescaled only when some row's running max moved.
// zs (when keep_z) receives the fragment's masked logits in log2 units, the
// weights the decode-time credit normalises later; the caller stores them.
template <class T, int D, int NB, int GSP>
__device__ __forceinline__ void attend(KVFrag<T, D, GSP> &f,
                                       const typename Op<T>::reg (&q)[NB][KVFrag<T, D, GSP>::KS],
                                       float sl2, int g4, float (&m_run)[NB], float (&l_run)[NB],
                                       f32x4 (&o)[NB][D / 16], bool keep_z,
                                       float (&zs)[GSP][NB][4]) {
  typedef KVFrag<T, D, GSP> F;
  constexpr int NC = F::NC;
  float sv[GSP][NB][4];
  float gmax[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) gmax[nb] = -__builtin_inff();
#pragma unroll
  for (int sp = 0; sp < GSP; ++sp) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < F::KS; ++ks) acc = Op<T>::mma(f.k[sp][ks], q[nb][ks], acc);
#pragma unroll
      for (int e = 0; e < 4; ++e) sv[sp][nb][e] = acc[e] * sl2;
    }
    if (f.nval[sp] < 16) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sv[sp][nb][e] = 4 * g4 + e < f.nval[sp] ? sv[sp][nb][e] : -__builtin_inff();
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int cc = 0; cc < NC; ++cc)
          f.v[sp][e][cc] = 4 * g4 + e < f.nval[sp] ? f.v[sp][e][cc] : (typename F::VT)0.f;
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      gmax[nb] = fmaxf(gmax[nb], fmaxf(fmaxf(sv[sp][nb][0], sv[sp][nb][1]),
                                       fmaxf(sv[sp][nb][2], sv[sp][nb][3])));
    if (keep_z) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int e = 0; e < 4; ++e) zs[sp][nb][e] = sv[sp][nb][e];
    }
  }
  bool moved = false;
  float alpha[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    gmax[nb] = across_rows(gmax[nb], [](float x, float y) { return fmaxf(x, y); });
    const float mn = fmaxf(m_run[nb], gmax[nb]);
    moved |= mn != m_run[nb];
    alpha[nb] = (m_run[nb] > -__builtin_inff()) ? __builtin_amdgcn_exp2f(m_run[nb] - mn) : 0.f;
    m_run[nb] = mn;
  }
  if (__builtin_amdgcn_ballot_w64(moved) != 0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      l_run[nb] *= alpha[nb];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float fe = __shfl(alpha[nb], 4 * g4 + e, kWave);
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) o[nb][cc][e] *= fe;
      }
    }
  }
  if constexpr (sizeof(T) == 2) {
    // bf16 values: O += P V as bf16 MFMAs (16x16x32), one per 16 output
    // columns and pair of sub-pages sp0, sp0 + 1 of the fragment, element t =
    // 4 (sp - sp0) + e of a lane's k-slice being key 4 g4 + e of sub-page sp
    // (zero past GSP sub-pages).  P is split into a bf16 high part and a bf16
    // remainder, p = hi + lo to about 2^-17 relative, and both are multiplied
    // by the exact bf16 V, so the product keeps fp32-level accuracy at a
    // quarter of the fp32 MFMA's issue time.
#pragma unroll
    for (int sp0 = 0; sp0 < GSP; sp0 += 2) {
      bf16x8 ph[NB], pl[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const float nm = m_run[nb] > -__builtin_inff() ? -m_run[nb] : 0.f;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int sp = sp0 + t / 4, e = t % 4;
          if (sp < GSP) {
            const float p = __builtin_amdgcn_exp2f(sv[sp][nb][e] + nm);
            l_run[nb] += p;
            const __bf16 hi = (__bf16)p;
            ph[nb][t] = hi;
            pl[nb][t] = (__bf16)(p - (float)hi);
          } else {
            ph[nb][t] = (__bf16)0.f;
            pl[nb][t] = (__bf16)0.f;
          }
        }
      }
#pragma unroll
      for (int cc = 0; cc < NC; ++cc) {
        bf16x8 vv;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int sp = sp0 + t / 4;
          vv[t] = sp < GSP ? (__bf16)f.v[sp < GSP ? sp : 0][t % 4][cc] : (__bf16)0.f;
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          o[nb][cc] = Op<__bf16>::mma(ph[nb], vv, o[nb][cc]);
          o[nb][cc] = Op<__bf16>::mma(pl[nb], vv, o[nb][cc]);
        }
      }
    }
  } else {
#pragma unroll
    for (int sp = 0; sp < GSP; ++sp) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        float p[4];
        const float nm = m_run[nb] > -__builtin_inff() ? -m_run[nb] : 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          p[e] = __builtin_amdgcn_exp2f(sv[sp][nb][e] + nm);
          l_run[nb] += p[e];
        }
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
          for (int cc = 0; cc < NC; ++cc)
            o[nb][cc] = mma_f32(p[ks], (float)f.v[sp][ks][cc], o[nb][cc]);
      }
    }
  }
}

// Sub-pages a wave loads at once: 16 KB of K and V in flight per wave, one
// fragment at a time.  Measured on the llama8b and dpts trees: with a single
// buffer the 16-row waves fit three to a SIMD, whose loads overlap one
// another's work; double-buffered fragments, or larger ones, leave one or
// two waves per SIMD and stream HBM more slowly.
template <class T, int D, int NB>
constexpr int sub_pages_per_fetch() {
  constexpr int per = 32 * D * (int)sizeof(T);   // K and V of one 16-slot sub-page
  return (16 << 10) / per < 1 ? 1 : (16 << 10) / per;
}

// One wave: one work unit (a CHUNK of a chain node's slots, one layer, one kv
// head), rows [rbase, rbase + 16 NB).  The unit's sub-pages are taken GSP at
// a time (the last fragment of a unit re-reads its last sub-page in the
// unused places, which the cache serves); other waves of the SIMD attend
// while one waits for its fragment.
// KZ: the call credits (some slice layers keep their logits); a plain call
// compiles without that path and its registers.
template <class T, int D, int NB, bool KZ>
__device__ void decode_unit(const DecArgs &a, int item, int lr, int g, int rbase) {
  using O = Op<T>;
  constexpr int GSP = sub_pages_per_fetch<T, D, NB>();
  typedef KVFrag<T, D, GSP> F;
  constexpr int KS = F::KS;
  constexpr int NC = F::NC;
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
  const int n_sub = (s_end - s_begin + 15) / 16;
  const int n_grp = (n_sub + GSP - 1) / GSP;
  // page ids of all sub-pages up front: a dependent load inside the pipeline
  // would make every wait cover the fragment still in flight
  static_assert(CHUNK / 16 <= kWave, "one lane per sub-page");
  const int pg = lane < n_sub ? t.page_table[po + (s_begin + 16 * lane) / pl.P] : 0;

  int qleaf[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int r = rbase + nb * 16 + rr;
    qleaf[nb] = r < R ? a.leaf_list[loff + r / G] : -1;
  }
  typename O::reg q[NB][KS];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int r = rbase + nb * 16 + rr;
    if (qleaf[nb] >= 0) {
      const int h = g * G + r % G;
      const T *qp = static_cast<const T *>(a.q) + (((int64_t)qleaf[nb] * a.Lr + lr) * Hq + h) * D;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) q[nb][ks] = O::load(qp + frag_col<T>(ks, g4));
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) q[nb][ks] = O::zero();
    }
  }
  UnitAddr ua;
  {
    const int esz = (int)sizeof(T);
    ua.row_bytes = D * esz;
    ua.page_bytes = (int64_t)pl.Hkv * pl.P * D * esz;
    const int64_t plane = ((int64_t)layer * pl.num_pages * pl.Hkv + g) * pl.P * D * esz;
    ua.k = static_cast<const char *>(pl.k) + plane;
    ua.v = static_cast<const char *>(pl.v) + plane;
    ua.koff = (uint32_t)(rr * D * esz + frag_col<T>(0, g4) * esz);
    ua.voff = (uint32_t)(4 * g4 * D * esz + F::NC * rr * esz);
  }
  // a credited slice layer keeps its logits: [slice][kv head][unit row][slot]
  float *zrow = nullptr;
  for (int z = 0; KZ && z < a.zS; ++z)
    if (a.zlr[z] == lr) {
      zrow = a.part + a.meta[4] +
             (((int64_t)z * pl.Hkv + g) * a.meta[3] + a.item_rowbase[item]) * CHUNK;
      break;
    }
  F cur = fetch_kv<T, D, GSP>(ua, pg, s_begin, s_end, n_sub, 0, pl.P);
  float m_run[NB], l_run[NB];
  f32x4 o[NB][NC];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m_run[nb] = -__builtin_inff();
    l_run[nb] = 0.f;
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) o[nb][cc] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // the logits of fragment gi are stored after fragment gi + 1's loads are
  // issued: a wave's loads and stores share one counter, so a wait for loads
  // issued after the stores would wait for the stores as well
  float zs[GSP][NB][4];
  auto store_z = [&](int gz) __attribute__((always_inline)) {
    // lane (rr, g4) holds keys 4 g4 .. 4 g4 + 3 of each sub-page for row rr:
    // zrow + r * CHUNK + 16 sub + key for query row r < R of the unit
#pragma unroll
    for (int sp = 0; sp < GSP; ++sp) {
      if (gz * GSP + sp >= n_sub) continue;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int r = rbase + nb * 16 + rr;
        if (r < R)
          *reinterpret_cast<float4 *>(zrow + (int64_t)r * CHUNK + 16 * (gz * GSP + sp) + 4 * g4) =
              make_float4(zs[sp][nb][0], zs[sp][nb][1], zs[sp][nb][2], zs[sp][nb][3]);
      }
    }
  };
  for (int gi = 0; gi < n_grp; ++gi) {
    if (gi > 0) {
      cur = fetch_kv<T, D, GSP>(ua, pg, s_begin, s_end, n_sub, gi * GSP, pl.P);
      if (KZ && zrow) store_z(gi - 1);
    }
    attend<T, D, NB, GSP>(cur, q, a.sl2, g4, m_run, l_run, o, KZ && zrow != nullptr, zs);
  }
  if (KZ && zrow && n_grp > 0) store_z(n_grp - 1);
  // partial rows [m, l, o(0..D-1)] of this unit
  const int64_t stride = D + 2;
  const int64_t slab = ((int64_t)lr * pl.Hkv + g) * a.meta[3];
  float *outp = a.part + (slab + a.item_rowbase[item]) * stride;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const float l = across_rows(l_run[nb], [](float x, float y) { return x + y; });
    const int row = rbase + nb * 16 + rr;
    if (g4 == 0 && row < R) {
      outp[row * stride] = m_run[nb];
      outp[row * stride + 1] = l;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int orow = rbase + nb * 16 + 4 * g4 + e;
      if (orow < R) {
        float *op = outp + orow * stride + 2 + NC * rr;
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) op[cc] = o[nb][cc][e];
      }
    }
  }
}

template <class T, int D, int NB, bool KZ>
__global__ __launch_bounds__(256) void decode_attn(DecArgs a, int cls) {
  if (status_failed(a.status)) return;
  const int n_items = a.meta[cls];
  const int planes = a.Lr * a.pl.Hkv;
  const int64_t total = (int64_t)n_items * planes;
  // the wave index is wave-uniform: keep the unit's bookkeeping scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int64_t w = (int64_t)blockIdx.x * 4 + wave; w < total; w += (int64_t)gridDim.x * 4) {
    const int item = a.cls_items[(int64_t)cls * a.max_items + w / planes];
    const int rem = (int)(w % planes);
    const int lr = rem / a.pl.Hkv;
    const int g = rem % a.pl.Hkv;
    const int R = a.node_nl[a.item_node[item]] * a.pl.G;
    for (int rbase = 0; rbase < R; rbase += 16 * NB) decode_unit<T, D, NB, KZ>(a, item, lr, g, rbase);
  }
}

// One wave per (leaf, layer, query head): merge the partials of the leaf's
// chain.  Lane k holds partial k's (max, sum); the running max and the weights
// come from fixed-order wave reductions, and o is accumulated in partial order,
// so the result does not depend on scheduling.  Workgroups blk of nblk take
// the rows in turn.
template <int D>
__device__ __forceinline__ void merge_rows(const DecArgs &a, void *out, int out_dtype,
                                           float *lse_out, int blk, int nblk) {
  constexpr int EPL = D / 64;  // output columns per lane
  constexpr int U = 4;         // partial rows loaded together
  constexpr int kPreO = 8;     // partial rows read ahead of the max
  const Pool &pl = a.pl;
  const int lane = lane_id();
  const int G = pl.G;
  const int Hq = pl.Hkv * G;
  const int64_t total = (int64_t)a.n_leaves * a.Lr * Hq;
  const int64_t stride = D + 2;
  const int wpb = blockDim.x / kWave;
  for (int64_t w = (int64_t)blk * wpb + threadIdx.x / kWave; w < total;
       w += (int64_t)nblk * wpb) {
    const int b = (int)(w / (a.Lr * Hq));
    const int rem = (int)(w % (a.Lr * Hq));
    const int lr = rem / Hq;
    const int h = rem % Hq;
    const int g = h / G;
    const int hl = h % G;
    const float *base = a.part + (((int64_t)lr * pl.Hkv + g) * a.meta[3] + hl) * stride;
    const int32_t *lp = a.leaf_part + (int64_t)b * a.max_parts;
    const int np = a.leaf_np[b];
    // global max over the chain's partials; the first kWave partials'
    // offsets, maxima and sums stay in registers for the second pass (longer
    // chains reload the rest there)
    int64_t off0 = 0;
    float m0 = -__builtin_inff(), l0 = 0.f;
    if (lane < np) {
      off0 = (int64_t)lp[lane] * stride;
      m0 = base[off0];
      l0 = base[off0 + 1];
    }
    // the output rows of the first kPreO partials are read together with
    // their (max, sum), before the max is known
    float xv0[kPreO][EPL];
#pragma unroll
    for (int u = 0; u < kPreO; ++u) {
      const int64_t oj = lane_value(off0, u < np ? u : 0);
#pragma unroll
      for (int e = 0; e < EPL; ++e) xv0[u][e] = u < np ? base[oj + 2 + 64 * e + lane] : 0.f;
    }
    float M = m0;
    for (int k0 = kWave; k0 < np; k0 += kWave) {
      const int k = k0 + lane;
      const float m = k < np ? base[(int64_t)lp[k] * stride] : -__builtin_inff();
      M = fmaxf(M, m);
    }
    M = wave_allreduce(M, [](float x, float y) { return fmaxf(x, y); });
    float L = 0.f, ov[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) ov[e] = 0.f;
    if (M > -__builtin_inff()) {
      for (int k0 = 0; k0 < np; k0 += kWave) {
        const int k = k0 + lane;
        int64_t off = 0;
        float f = 0.f, lk = 0.f;
        if (k < np) {
          float m = m0;
          off = off0;
          lk = l0;
          if (k0 > 0) {
            off = (int64_t)lp[k] * stride;
            m = base[off];
            lk = base[off + 1];
          }
          f = m > -__builtin_inff() ? __builtin_amdgcn_exp2f(m - M) : 0.f;
        }
        L += wave_sum(lk * f);
        const int nk = min(kWave, np - k0);
        int jstart = 0;
        if (k0 == 0) {
#pragma unroll
          for (int u = 0; u < kPreO; ++u) {
            const float fu = u < nk ? lane_value(f, u) : 0.f;
#pragma unroll
            for (int e = 0; e < EPL; ++e) ov[e] += (fu > 0.f ? xv0[u][e] * fu : 0.f);
          }
          jstart = kPreO;
        }
        for (int j0 = jstart; j0 < nk; j0 += U) {
          float xv[U][EPL], fj[U];
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const int j = min(j0 + u, nk - 1);
            const int64_t oj = lane_value(off, j);
            fj[u] = j0 + u < nk ? lane_value(f, j) : 0.f;
#pragma unroll
            for (int e = 0; e < EPL; ++e) xv[u][e] = base[oj + 2 + 64 * e + lane];
          }
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < EPL; ++e) ov[e] += (fj[u] > 0.f ? xv[u][e] * fj[u] : 0.f);
        }
      }
    }
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
    if (lane == 0) {
      const float l2 = L > 0.f ? M + __log2f(L) : -__builtin_inff();
      const int64_t li = ((int64_t)b * a.Lr + lr) * Hq + h;
      if (lse_out) lse_out[li] = L > 0.f ? l2 * kLn2 : -__builtin_inff();
    }
  }
}

// Decode-time credit (Sec. 4 Execution (iii)): the softmax weight exp2(z -
// lse2) of every decode query row on every key of a unit, from the logits z
// the attention units kept for the credited slice layers, summed over the
// rows whose leaf lies strictly below the unit's node (and, in the
// self-window mode, the leaf's own rows on keys before its newest position)
// and over the slice layers (a layer listed m times counts m times) and kv
// heads, and added to A at the key's token.  A row's log2 LSE, lse2 = M +
// log2(sum_k l_k exp2(m_k - M)) over the (max m_k, sum l_k) of the partials of
// its leaf's chain, is formed here from those partials, so the credit does not
// wait for the merge and runs beside it in the same launch.
// One workgroup of kCreditWaves waves per quarter (64 slots) of a unit, one
// lane per slot.  The unit's (row, distinct slice layer, kv head) triples, in
// the order (r * U + z) * Hkv + g, are staged in LDS up to kCreditTile at a
// time (one thread per triple): each triple's lse2 and its weight, the layer's
// multiplicity, negated when the row is the node's own leaf's.  Wave v takes
// the triples v, v + kCreditWaves, ... in order, kCreditBatch logit loads at a
// time, the next batch in flight while one is summed; the first batch is
// issued before the tables are built (a triple's logit row, (z * Hkv + g) *
// rows + r, is known without them), and for up to kCreditWaves * kCreditBatch
// triples it is the only one.  The rows of other leaves and the node's own
// rows are kept in two sums; the waves' sums are added in wave order, so each
// token's sum has one owner and a fixed order.  Workgroup 0 also adds the row
// counts to rows_seen (integer atomics: order-free).
constexpr int kCreditWaves = 16;
constexpr int kCreditThreads = kCreditWaves * kWave;
constexpr int kCreditTile = 1024;
constexpr int kCreditBatch = 16;
constexpr int kQuarters = CHUNK / kWave;
constexpr int kLsePar = 8;            // partials of a chain loaded together
static_assert(CHUNK % kWave == 0, "a unit is a whole number of 64-slot quarters");
static_assert(kCreditTile % (kCreditWaves * kCreditBatch) == 0, "batches do not straddle tiles");

// a triple as (row r, zg = z * Hkv + g), stepped without divisions
struct Triple {
  int r, zg;
  __device__ __forceinline__ void step(int k, int per) {
    zg += k;
    while (zg >= per) {
      zg -= per;
      ++r;
    }
  }
};

// logits of the batch of triples it, it + kCreditWaves, ... (it is left at
// the next batch's first triple): zb points at the unit's first logit row and
// the lane's slot; triples past the unit's R rows are not read
__device__ __forceinline__ void credit_load(float (&zv)[kCreditBatch], const float *zb, Triple &it,
                                            int R, int per, int64_t rows_total) {
#pragma unroll
  for (int u = 0; u < kCreditBatch; ++u) {
    zv[u] = it.r < R ? zb[((int64_t)it.zg * rows_total + it.r) * CHUNK] : 0.f;
    it.step(kCreditWaves, per);
  }
}

// log2 LSE of query row (leaf b, layer lr, head g * G + hl) over the partials
// of b's chain, with the maximum taken kLsePar partials at a time
template <int D>
__device__ __forceinline__ float chain_lse2(const DecArgs &a, int b, int lr, int g, int hl) {
  const int64_t stride = D + 2;
  const float *base = a.part + (((int64_t)lr * a.pl.Hkv + g) * a.meta[3] + hl) * stride;
  const int32_t *lp = a.leaf_part + (int64_t)b * a.max_parts;
  const int np = a.leaf_np[b];
  float M = -__builtin_inff(), L = 0.f;
  for (int k0 = 0; k0 < np; k0 += kLsePar) {
    float m[kLsePar], l[kLsePar];
#pragma unroll
    for (int u = 0; u < kLsePar; ++u) {
      const int64_t off = k0 + u < np ? (int64_t)lp[k0 + u] * stride : 0;
      m[u] = k0 + u < np ? base[off] : -__builtin_inff();
      l[u] = k0 + u < np ? base[off + 1] : 0.f;
    }
    float Mn = M;
#pragma unroll
    for (int u = 0; u < kLsePar; ++u) Mn = fmaxf(Mn, m[u]);
    if (Mn == -__builtin_inff()) continue;
    L = M > -__builtin_inff() ? L * __builtin_amdgcn_exp2f(M - Mn) : 0.f;
#pragma unroll
    for (int u = 0; u < kLsePar; ++u)
      L += m[u] > -__builtin_inff() ? l[u] * __builtin_amdgcn_exp2f(m[u] - Mn) : 0.f;
    M = Mn;
  }
  return L > 0.f ? M + __log2f(L) : -__builtin_inff();
}

// the credit of the quarters blk, blk + nblk, ... of the plan's units
template <int D>
__device__ __forceinline__ void credit_quarters(const DecArgs &a, const CreditArgs &cr, int blk,
                                                int nblk) {
  __shared__ float s_oth[kCreditWaves][kWave], s_own[kCreditWaves][kWave];
  __shared__ float s_l2[kCreditTile], s_w[kCreditTile];
  const Tree &t = a.t;
  const Pool &pl = a.pl;
  const int G = pl.G, Hkv = pl.Hkv;
  const int Hq = Hkv * G;
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  // the launch covers at most max_items units, so the first unit's fields can
  // be read before the plan's unit count is known
  const int n_items = a.meta[0] + a.meta[1] + a.meta[2];
  const int64_t rows_total = a.meta[3];
  const int item0 = blk / kQuarters;
  const int node0 = a.item_node[item0];
  const int chunk0 = a.item_chunk[item0];
  const int rb0 = a.item_rowbase[item0];
  if (status_failed(a.status)) return;
  if (blk == 0) {
    const unsigned long long per = (unsigned long long)cr.S * Hq;
    for (int e = threadIdx.x; e < a.n_leaves * MAXD; e += blockDim.x) {
      const int b = e / MAXD, d = e % MAXD;
      const int dl = a.ldepth[b];
      if (d < dl || (d == dl && cr.self_window))
        atomicAdd(reinterpret_cast<unsigned long long *>(cr.rows_seen) +
                      a.lanc[(int64_t)b * MAXD + d],
                  per);
    }
  }
  const float *z0 = a.part + a.meta[4];
  const int per = cr.U * Hkv;
  constexpr int kLast = kCreditWaves - 1;
  for (int w = blk; w < n_items * kQuarters; w += nblk) {
    const int item = w / kQuarters;
    const bool first = w == blk;
    const int node = first ? node0 : a.item_node[item];
    const int k0 = (first ? chunk0 : a.item_chunk[item]) * CHUNK;
    const int rb = first ? rb0 : a.item_rowbase[item];
    const int c = t.n_kept[node];
    const int s0 = k0 + (w % kQuarters) * kWave;
    if (s0 >= c) continue;                    // uniform over the workgroup
    const int slot = s0 + lane;
    const bool key_ok = slot < c;
    const int R = a.node_nl[node] * G;
    const int loff = a.node_leaf_off[node];
    const int n = R * per;
    // the leaf of this thread's first table entry, read before the logits so
    // that waiting for it does not wait for them
    const int b_first = (int)threadIdx.x < min(n, kCreditTile)
                            ? a.leaf_list[loff + (int)threadIdx.x / per / G] : 0;
    // logit rows hold CHUNK slots each, so the lane's slot is in bounds for
    // every lane; lanes past the node's count are masked after the load
    const float *zb = z0 + (int64_t)rb * CHUNK + (slot - k0);
    float cur[kCreditBatch];
    Triple it{0, 0};
    it.step(wv, per);
    credit_load(cur, zb, it, R, per, rows_total);
    // the last wave fetches the lane's token and its A entry meanwhile; each
    // token has one owner, so A is read before the sums
    int64_t tok = 0;
    float a_old = 0.f;
    bool own_ok = false;
    if (wv == kLast && key_ok) {
      const int page = t.page_table[t.page_off[node] + slot / pl.P];
      const int pos = pl.slot_pos[(int64_t)page * pl.P + slot % pl.P];
      tok = t.tok_off[node] + pos;
      a_old = cr.A[tok];
      // own rows (the node is the row's leaf) are credited only on earlier
      // keys in the self-window mode
      own_ok = cr.self_window && pos < t.n_full[node] - 1;
    }
    float oth = 0.f, own = 0.f;
    int e0 = wv;
    for (int t0 = 0; t0 < n; t0 += kCreditTile) {
      const int nt = min(kCreditTile, n - t0);
      for (int i = threadIdx.x; i < nt; i += blockDim.x) {
        const int e = t0 + i;
        const int r = e / per, zg = e % per;
        const int z = zg / Hkv, g = zg % Hkv;
        const int b = t0 == 0 && i == (int)threadIdx.x ? b_first : a.leaf_list[loff + r / G];
        s_l2[i] = chain_lse2<D>(a, b, cr.slice[z], g, r % G);
        const float m = (float)cr.mult[z];
        s_w[i] = a.leaves[b] == node ? -m : m;
      }
      __syncthreads();
      for (; e0 < t0 + nt; e0 += kCreditWaves * kCreditBatch) {
        float nxt[kCreditBatch];
        const bool more = e0 + kCreditWaves * kCreditBatch < n;
        if (more) credit_load(nxt, zb, it, R, per, rows_total);
#pragma unroll
        for (int u = 0; u < kCreditBatch; ++u) {
          const int i = e0 + kCreditWaves * u - t0;
          if (i < nt) {
            const float p = key_ok ? __builtin_amdgcn_exp2f(cur[u] - s_l2[i]) : 0.f;
            const float wt = s_w[i];
            if (wt < 0.f) own += -wt * p;
            else oth += wt * p;
          }
        }
        if (more) {
#pragma unroll
          for (int u = 0; u < kCreditBatch; ++u) cur[u] = nxt[u];
        }
      }
      __syncthreads();                        // the tables are reused by the next tile
    }
    s_oth[wv][lane] = oth;
    s_own[wv][lane] = own;
    __syncthreads();
    if (wv == kLast && key_ok) {
      float tot = 0.f;
#pragma unroll
      for (int v = 0; v < kCreditWaves; ++v) tot += s_oth[v][lane];
      if (own_ok) {
#pragma unroll
        for (int v = 0; v < kCreditWaves; ++v) tot += s_own[v][lane];
      }
      cr.A[tok] = a_old + tot;
    }
    __syncthreads();                          // the sums are reused by the next quarter
  }
}

template <int D>
__global__ __launch_bounds__(256) void decode_merge(DecArgs a, void *out, int out_dtype,
                                                    float *lse_out) {
  if (status_failed(a.status)) return;
  merge_rows<D>(a, out, out_dtype, lse_out, blockIdx.x, gridDim.x);
}

// scored calls: the first credit_blocks workgroups credit (their chain of
// loads is the longer one, so they are dispatched first), the rest merge
template <int D>
__global__ __launch_bounds__(kCreditThreads) void decode_merge_credit(DecArgs a, CreditArgs cr,
                                                                      void *out, int out_dtype,
                                                                      float *lse_out,
                                                                      int credit_blocks) {
  if ((int)blockIdx.x < credit_blocks) {
    credit_quarters<D>(a, cr, blockIdx.x, credit_blocks);
    return;
  }
  if (status_failed(a.status)) return;
  merge_rows<D>(a, out, out_dtype, lse_out, blockIdx.x - credit_blocks,
                gridDim.x - credit_blocks);
}

template <class T, int D>
void launch_decode_kernels(const arbor_geom_t *geom, const DecArgs &a, void *out, int out_dtype,
                           float *lse_out, const CreditArgs *cr, hipStream_t stream) {
  const int grid = 2048;
  // rows of a work unit are at most n_leaves * G: only the row classes that
  // can occur are launched
  const int max_rows = a.n_leaves * a.pl.G;
  timing_begin(geom, ARBOR_KERNEL_DECODE_ATTN, stream);
  if (cr) {
    hipLaunchKernelGGL((decode_attn<T, D, 1, true>), dim3(grid), dim3(256), 0, stream, a, 0);
    if (max_rows > 16)
      hipLaunchKernelGGL((decode_attn<T, D, 2, true>), dim3(grid / 2), dim3(256), 0, stream, a, 1);
    if (max_rows > 32)
      hipLaunchKernelGGL((decode_attn<T, D, 4, true>), dim3(grid / 4), dim3(256), 0, stream, a, 2);
  } else {
    hipLaunchKernelGGL((decode_attn<T, D, 1, false>), dim3(grid), dim3(256), 0, stream, a, 0);
    if (max_rows > 16)
      hipLaunchKernelGGL((decode_attn<T, D, 2, false>), dim3(grid / 2), dim3(256), 0, stream, a, 1);
    if (max_rows > 32)
      hipLaunchKernelGGL((decode_attn<T, D, 4, false>), dim3(grid / 4), dim3(256), 0, stream, a, 2);
  }
  timing_end(geom, ARBOR_KERNEL_DECODE_ATTN, stream);
  const int64_t mw = (int64_t)a.n_leaves * a.Lr * a.pl.Hkv * a.pl.G;
  if (!cr) {
    const int mgrid = (int)((mw + 3) / 4 < 8192 ? (mw + 3) / 4 : 8192);
    hipLaunchKernelGGL((decode_merge<D>), dim3(mgrid), dim3(256), 0, stream, a, out, out_dtype,
                       lse_out);
    return;
  }
  // credit workgroups stride over the quarters of the plan's units (at most
  // half the chip's wave slots, so that the merge workgroups start beside
  // them); merge workgroups hold kCreditWaves rows each
  const int cgrid = std::min(a.max_items * kQuarters, 256);
  const int64_t mb = (mw + kCreditWaves - 1) / kCreditWaves;
  const int mgrid = (int)(mb < 2048 ? mb : 2048);
  timing_begin(geom, ARBOR_KERNEL_DECODE_CREDIT, stream);
  hipLaunchKernelGGL((decode_merge_credit<D>), dim3(cgrid + mgrid), dim3(kCreditThreads), 0,
                     stream, a, *cr, out, out_dtype, lse_out, cgrid);
  timing_end(geom, ARBOR_KERNEL_DECODE_CREDIT, stream);
}

}  // namespace

static size_t decode_max_items(const arbor_sizes_t *sz) {
  return (size_t)sz->num_nodes + (size_t)(sz->num_tokens / CHUNK) + 1;
}

// partials along one chain: at most one ragged chunk per chain node
static size_t decode_max_parts(const arbor_sizes_t *sz) {
  return (size_t)(sz->num_tokens / CHUNK) + MAXD + 1;
}

size_t decode_workspace(const arbor_geom_t *g, const arbor_sizes_t *sz) {
  const size_t V = (size_t)sz->num_nodes;
  const size_t nl = (size_t)(sz->max_leaves > 0 ? sz->max_leaves : 1);
  const size_t items = decode_max_items(sz);
  const size_t per_leaf = (size_t)(sz->max_context / CHUNK) + MAXD + 1;
  const size_t rows = nl * per_leaf * g->q_per_kv;
  size_t b = 19 * 256;
  b += 3 * items * 4 + 3 * items * 4 + V * 4 * 4 + nl * MAXD * 4 * 3 + nl * 4 + nl * MAXD * 4;
  b += nl * 4 + nl * decode_max_parts(sz) * 4;
  b += rows * (size_t)sz->max_layers * g->num_kv_heads * (g->head_dim + 2) * 4;
  // logits of the credited slice layers (scored decode)
  b += rows * (size_t)(sz->n_slice > 0 ? sz->n_slice : 0) * g->num_kv_heads * CHUNK * 4 + 16;
  return b;
}

int launch_decode(const arbor_geom_t *geom, const arbor_tree_t *tree, const arbor_pool_t *pool,
                  const int32_t *leaves, int32_t n_leaves, int32_t layer_begin, int32_t layer_end,
                  const void *q, void *out, int32_t out_dtype, float *lse_out, float softmax_scale,
                  const arbor_decode_credit_t *credit, int32_t *status, void *workspace,
                  size_t workspace_bytes, hipStream_t stream) {
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
  const int max_parts = (int)decode_max_parts(&sz);
  int32_t *leaf_np = cv.take<int32_t>(n_leaves);
  int32_t *leaf_part = cv.take<int32_t>((size_t)n_leaves * max_parts);
  if (!cv.ok) return ARBOR_EWORKSPACE;
  CreditArgs cr{};
  if (credit) {
    cr.S = credit->n_slice;
    for (int e = 0; e < credit->n_slice; ++e) {
      const int lr = credit->slice_layers[e] - layer_begin;
      int u = 0;
      while (u < cr.U && cr.slice[u] != lr) ++u;
      if (u == cr.U) cr.slice[cr.U++] = lr;
      ++cr.mult[u];
    }
    cr.self_window = credit->self_window;
    cr.A = credit->A;
    cr.rows_seen = credit->rows_seen;
  }
  a.zS = credit ? cr.U : 0;
  for (int e = 0; e < 8; ++e) a.zlr[e] = credit && e < cr.U ? cr.slice[e] : -1;
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
  a.leaf_np = leaf_np;
  a.leaf_part = leaf_part;
  a.max_parts = max_parts;
  a.part = reinterpret_cast<float *>(cv.rest());
  a.part_cap = (int64_t)(cv.remaining() / 4);
  // one thread per node, and one wave per leaf for the per-leaf scans: a
  // small tree takes a smaller workgroup, whose barriers are cheaper
  const int64_t plan_need = std::max<int64_t>(t.V, (int64_t)n_leaves * MAXD);
  const int plan_threads = (int)std::min<int64_t>(1024, (plan_need + kWave - 1) / kWave * kWave);
#define ARBOR_PLAN_LAUNCH(S, F)                                                                \
  hipLaunchKernelGGL((decode_plan<S, F>), dim3(1), dim3(plan_threads), 0, stream, a, meta,       \
                     cls_items, item_node, item_chunk, item_rowbase, node_nl, node_leaf_off,      \
                     leaf_list, node_item0, node_rowbase, lanc, ldepth, lrank, leaf_np, leaf_part)
  const bool small = t.V <= kPlanLds, few = n_leaves <= kPlanLeaves;
  if (small && few) ARBOR_PLAN_LAUNCH(true, true);
  else if (small) ARBOR_PLAN_LAUNCH(true, false);
  else if (few) ARBOR_PLAN_LAUNCH(false, true);
  else ARBOR_PLAN_LAUNCH(false, false);
#undef ARBOR_PLAN_LAUNCH
  const CreditArgs *crp = credit ? &cr : nullptr;
  if (geom->dtype == ARBOR_BF16) {
    if (geom->head_dim == 128)
      launch_decode_kernels<__bf16, 128>(geom, a, out, out_dtype, lse_out, crp, stream);
    else
      launch_decode_kernels<__bf16, 64>(geom, a, out, out_dtype, lse_out, crp, stream);
  } else {
    if (geom->head_dim == 128)
      launch_decode_kernels<float, 128>(geom, a, out, out_dtype, lse_out, crp, stream);
    else
      launch_decode_kernels<float, 64>(geom, a, out, out_dtype, lse_out, crp, stream);
  }
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
