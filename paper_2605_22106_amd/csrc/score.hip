// arbor_score: MSVE scoring (Sec. 4 "Multi-Signal Value Estimation").
//
// The accumulated attention A_i(t) sums, over later query positions, over a
// thin slice of layers and over query heads, the softmax probability that each
// query puts on token t.  Here the later queries are the last-W window rows of
// every observer block j; a row's softmax runs over j's whole resident causal
// context (proper ancestors + own tokens up to the row), and the probability is
// credited to tokens of proper ancestors (u > b_i).
//
// Launches on one stream:
//   setup   one workgroup per observer: every workgroup walks all observer
//           chains for the partial / table offsets (a prefix over observers),
//           writes its own observer's chain data and 16-slot sub-page table;
//           workgroup 0 also validates the tree;
//   attn    per (observer, slice layer, kv head, row group), two passes over
//           the same (row, key) pairs as MFMA tiles of 16 keys x 16 rows:
//           C = K Q^T for the row log-sum-exp, then C = Q K^T for per-key
//           sums of exp2(z - lse) -> one partial per credited context key;
//   fold    per observer: sum its (slice layer, kv head, row group) partials;
//   reduce  per block i and 64-slot chunk: sum the folded partials of every
//           observer below i in observer order (fp64) into A, rows_seen;
//   final   a_i = sum_p A_i(p) / rows_seen_i, s_i = clip(sigmoid(theta.phi)).
// No atomics anywhere, so A is bitwise reproducible.  The reduction dimension
// (head_dim) is permuted identically in both MFMA operands so that every lane
// reads one contiguous quarter of a K or Q row (64 B for bf16 d = 128).
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
  float *part;      // partial column sums
  const int64_t *pbase;   // [n_obs]
  const int64_t *tbase;   // [n_obs]: float offset (in part) of the observer's sub-page table
  const int32_t *nsp;     // [n_obs][2]: sub-pages of the chain, and of the credited part
  const int32_t *ctxlen;  // [n_obs]
  const int32_t *odepth;  // [n_obs]
  const int32_t *anc;     // [n_obs][MAXD]
  int32_t *status;
};

// Chain of observer j in LDS, root first, with a table of its 16-slot
// sub-pages so the key loop needs no dependent page-table load.
constexpr int SPCAP = 512;
struct ChainLds {
  int node[MAXD];
  int c[MAXD];
  int64_t po[MAXD];
  int ctx[MAXD];       // context offset of the node's first slot
  int sp_off[MAXD + 1];
  int depth;
  int sp_row[SPCAP];   // page * Hkv * P + r0: row of the sub-page within a (layer, kv head) plane
  int sp_slot[SPCAP];  // page * P + r0: index into slot_pos
  int sp_ctx[SPCAP];   // context position of the sub-page's first slot
  int sp_meta[SPCAP];  // chain depth | valid slots << 8
};

__device__ __forceinline__ void build_chain(const Tree &t, const Pool &pl, int j, ChainLds &ch) {
  if (threadIdx.x == 0) {
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
  __syncthreads();
  const int n_sp = min(ch.sp_off[ch.depth + 1], SPCAP);
  for (int sp = threadIdx.x; sp < n_sp; sp += blockDim.x) {
    int d = 0;
    while (sp >= ch.sp_off[d + 1]) ++d;
    const int q0 = (sp - ch.sp_off[d]) * 16;
    const int page = t.page_table[ch.po[d] + q0 / pl.P];
    const int r0 = q0 % pl.P;
    ch.sp_row[sp] = page * pl.Hkv * pl.P + r0;
    ch.sp_slot[sp] = page * pl.P + r0;
    ch.sp_ctx[sp] = ch.ctx[d] + q0;
    ch.sp_meta[sp] = d | (min(16, ch.c[d] - q0) << 8);
  }
  __syncthreads();
}

struct SubPage {
  int row, slot, ctx, d, nvalid;
};

__device__ __forceinline__ SubPage sub_page(const Tree &t, const Pool &pl, const ChainLds &ch,
                                            int sp) {
  SubPage r;
  if (sp < SPCAP) {
    r.row = ch.sp_row[sp];
    r.slot = ch.sp_slot[sp];
    r.ctx = ch.sp_ctx[sp];
    r.d = ch.sp_meta[sp] & 255;
    r.nvalid = ch.sp_meta[sp] >> 8;
  } else {
    int d = 0;
    while (sp >= ch.sp_off[d + 1]) ++d;
    const int q0 = (sp - ch.sp_off[d]) * 16;
    const int page = t.page_table[ch.po[d] + q0 / pl.P];
    const int r0 = q0 % pl.P;
    r.row = page * pl.Hkv * pl.P + r0;
    r.slot = page * pl.P + r0;
    r.ctx = ch.ctx[d] + q0;
    r.d = d;
    r.nvalid = min(16, ch.c[d] - q0);
  }
  return r;
}

// Layout of one 16-key sub-page of K in LDS: unit u = blk * 64 + lane is 16
// bytes: key (lane % 16), quarter (lane / 16), bytes [16 blk, 16 blk + 16) of
// that quarter row, so the MFMA operand of a k-step is one conflict-free
// 16-byte read per lane.
template <class T, int D>
struct Stage {
  static constexpr int QB = D / 4 * (int)sizeof(T);  // bytes of a quarter row
  static constexpr int NBLK = QB / 16;                // 16-byte units per lane
  static constexpr int UNITS = NBLK * kWave;          // units per sub-page
  static constexpr int BYTES = UNITS * 16;
};

// ---------------------------------------------------------------------------
// Fused two-pass kernel.  Keys stream through a ring of RING stages of GS
// sub-pages in LDS, filled by direct global->LDS loads; each wave owns 16 NBW
// query rows and keeps their Q in registers for both passes:
//   pass 0  C = K Q^T: running max / sum of each row over the chain -> lse;
//   pass 1  C = Q K^T: per key, sum over the wave's rows of exp2(z - lse);
//           the four waves' sums are added in wave order and stored as the
//           row group's partial for that key.
// One barrier per stage: a wave waits for its own loads of the stage, then the
// barrier makes every wave's loads visible and frees the slot the next load
// refills.  Ring slots are distinct LDS arrays (the loop is unrolled by RING),
// so the compiler can tell a slot being filled from the one being read.
constexpr int kGS = 4;         // sub-pages per stage
constexpr int kRing = 3;       // stages in the ring
constexpr int kXcds = 8;       // accelerator dies of the device; workgroups go round-robin
template <int N>
using Ic = std::integral_constant<int, N>;

// v_max3 without the quieting the IEEE maxnum lowering adds to each operand:
// the operands are MFMA results or -inf, never signalling NaNs.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Direct global -> LDS loads: lane L's `size` bytes land at lds + size * L.
__device__ __forceinline__ void load_to_lds16(const void *g, void *lds) {
  __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
}
__device__ __forceinline__ void load_to_lds4(const void *g, void *lds) {
  __builtin_amdgcn_global_load_lds(g, lds, 4, 0, 0);
}

// sum over the four 16-lane groups of the wave (lanes l, l ^ 16, l ^ 32,
// l ^ 48), in every lane
__device__ __forceinline__ float group_sum(float x) {
  return across_rows(x, [](float a, float b) { return a + b; });
}

template <int N>
__device__ __forceinline__ float tree_sum(const float (&v)[N]) {
  static_assert((N & (N - 1)) == 0, "power of two");
  float w[N];
#pragma unroll
  for (int i = 0; i < N; ++i) w[i] = v[i];
#pragma unroll
  for (int h = N / 2; h >= 1; h /= 2)
#pragma unroll
    for (int i = 0; i < h; ++i) w[i] = w[i] + w[i + h];
  return w[0];
}

// max of v[] and m, three operands per instruction
template <int N>
__device__ __forceinline__ float tree_max(const float (&v)[N], float m) {
  static_assert(N == 16, "one stage of a row block");
  const float x0 = max3f(v[0], v[1], v[2]), x1 = max3f(v[3], v[4], v[5]);
  const float x2 = max3f(v[6], v[7], v[8]), x3 = max3f(v[9], v[10], v[11]);
  const float x4 = max3f(v[12], v[13], v[14]);
  return max3f(max3f(x0, x1, x2), max3f(x3, x4, v[15]), m);
}

template <class T, int D>
struct Ring {
  typedef Stage<T, D> SG;
  __attribute__((aligned(16))) char k[kGS][SG::BYTES];
  __attribute__((aligned(16))) int pos[kGS][16];
};
// per-stage column sums of the four waves (not a load target, so reading it
// never has to wait for loads in flight)
struct Red {
  float v[kGS][4][16];
};

template <class T, int D, int NBW>
__global__ __launch_bounds__(256) void score_attn(ScoreArgs a) {
  using O = Op<T>;
  using SG = Stage<T, D>;
  constexpr int KS = D / 4 / O::kPerStep;   // MFMA k-steps over head_dim
  constexpr int RW = 64 * NBW;              // rows of the workgroup
  constexpr int DPW = kGS * SG::NBLK / 4;   // K loads per wave per stage
  constexpr int VM = DPW + 1;               // vector-memory ops per wave per stage
  static_assert(kGS == 4, "one position load per wave per stage");
  static_assert((kRing - 2) * VM <= 15, "vmcnt immediate");
  constexpr float kFloor = -1e30f;
  __shared__ Ring<T, D> r0, r1, r2;
  __shared__ Red d0, d1, d2;
  __shared__ int s_bad;
  // XCD-aware order: workgroup n runs on XCD n % 8, so XCD x takes the
  // (slice layer, kv head, row group) planes p = x, x + 8, ... and, within a
  // plane, the observers in id order -- siblings, which share their whole
  // ancestor chain, run together and read those keys from the XCD's L2
  const int n_planes = a.S * a.pl.Hkv * a.n_rg;
  const int xcd = (int)blockIdx.x % kXcds;
  const int idx = (int)blockIdx.x / kXcds;
  const int o = idx % a.n_obs;
  const int plane = (idx / a.n_obs) * kXcds + xcd;
  if (plane >= n_planes) return;
  if (threadIdx.x == 0) s_bad = status_failed(a.status);
  __syncthreads();
  if (s_bad) return;
  const Tree &t = a.t;
  const Pool &pl = a.pl;
  const int slg = plane / a.n_rg;
  const int rg = plane % a.n_rg;
  const int si = slg / pl.Hkv;
  const int g = slg % pl.Hkv;
  const int layer = a.slice[si];
  const int j = a.obs[o];
  // the chain's sub-page table, read with scalar loads (constant address space)
  // entry sp: [4 sp] plane row, [4 sp + 1] slot, [4 sp + 2] context offset,
  // [4 sp + 3] valid slots | own << 8
  typedef const __attribute__((address_space(4))) int *TabPtr;
  const TabPtr tab = (TabPtr)(a.part + a.tbase[o]);
  const int tid = threadIdx.x;
  const int lane = lane_id();
  // (& 3: four waves; lets the compiler resolve each load's sub-page statically)
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & 3;
  const int rr = lane & 15;
  const int g4 = lane >> 4;
  const int G = pl.G;
  const int nj = t.n_full[j];
  const int wj = min(a.W, nj);
  const int rows_total = G * a.W;
  const int row0 = rg * RW + wave * 16 * NBW;   // first row of this wave
  const float sl2 = a.sl2;
  auto row_u = [&](int r) __attribute__((always_inline)) -> int {
    if (r >= rows_total) return -1;
    const int tt = r % a.W;
    return tt < wj ? nj - wj + tt : -1;
  };

  typename O::reg q[NBW][KS];
  const T *qbase = static_cast<const T *>(a.q_win) +
                   ((((int64_t)o * a.S + si) * (pl.Hkv * G) + (int64_t)g * G) * a.W) * D;
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb) {
    const int r = row0 + nb * 16 + rr;
    const bool rv = r < rows_total;
    const T *rp = qbase + (int64_t)(rv ? r : 0) * D + g4 * (D / 4);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) q[nb][ks] = rv ? O::load(rp + ks * O::kPerStep) : O::zero();
  }
  const int64_t plane_row0 = (int64_t)layer * pl.num_pages * pl.Hkv * pl.P + (int64_t)g * pl.P;
  const char *kplane = static_cast<const char *>(pl.k) + plane_row0 * D * (int64_t)sizeof(T);
  // this lane's 16-byte unit of a key tile: key rr, quarter g4
  const int64_t lane_off = (int64_t)rr * (D * (int)sizeof(T)) + g4 * SG::QB;

  // direct loads of stage st (sub-pages st*GS .. st*GS+GS-1, clamped) into R;
  // all addresses are formed before the first load is issued
  auto issue = [&](Ring<T, D> &R, int st, int n_sp) __attribute__((always_inline)) {
    int rows[kGS], slots[kGS];
#pragma unroll
    for (int k = 0; k < kGS; ++k) {
      const int sp = min(st * kGS + k, n_sp - 1);
      rows[k] = tab[4 * sp];
      slots[k] = tab[4 * sp + 1];
    }
    // lane L: position (L & 15) of sub-page L >> 4
    int lane_slot = slots[0];
#pragma unroll
    for (int k = 1; k < kGS; ++k) lane_slot = g4 == k ? slots[k] : lane_slot;
#pragma unroll
    for (int i = 0; i < DPW; ++i) {
      const int u = wave + 4 * i;          // unit (sub-page k, 16-byte block blk)
      const int k = u / SG::NBLK, blk = u % SG::NBLK;
      int row = rows[0];
#pragma unroll
      for (int kk = 1; kk < kGS; ++kk) row = k == kk ? rows[kk] : row;
      const char *src = kplane + (int64_t)row * (D * (int)sizeof(T)) + lane_off + blk * 16;
      load_to_lds16(src, &R.k[k][blk * kWave * 16]);
    }
    // the key positions of all four sub-pages, loaded by every wave (the
    // waves write the same values).  An unmasked load: a load under a lane
    // mask gives the compiler paths with different numbers of loads in
    // flight, and it then waits for all of them before each read of the ring.
    load_to_lds4(pl.slot_pos + lane_slot + rr, &R.pos[0][0]);
  };
  // my loads of the stage about to be computed are done; everyone's are visible
  // (s_waitcnt immediate: vmcnt in bits 3:0, expcnt 6:4, lgkmcnt 11:8.)  The
  // LDS writes of this wave are complete too (lgkmcnt 0), so no release fence
  // is needed -- one would also wait for the loads still filling later slots.
  // (`later`: how many stages' loads may stay in flight, a compile-time count)
  auto stage_sync = [&](auto later) __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0x070 | (decltype(later)::value * VM));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  };
  auto operand = [&](const Ring<T, D> &R, int k, typename O::reg (&kr)[KS]) __attribute__((always_inline)) {
    const char *base = &R.k[k][0] + lane * 16;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int byte = ks * O::kPerStep * (int)sizeof(T);   // within the quarter row
      kr[ks] = O::load(reinterpret_cast<const T *>(base + (byte / 16) * (kWave * 16) + byte % 16));
    }
  };

  // ---- pass 0: row log2-sum-exp ----
  float m[NBW], l[NBW];
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb) {
    m[nb] = kFloor;
    l[nb] = 0.f;
  }
  auto lse_stage = [&](const Ring<T, D> &R, int st, int n_sp, auto &&between)
                       __attribute__((always_inline)) {
    f32x4 acc[kGS][NBW];
    int meta[kGS];
    typename O::reg kr[kGS][KS];   // all operands of the stage first: one LDS wait
#pragma unroll
    for (int k = 0; k < kGS; ++k) operand(R, k, kr[k]);
    between();
#pragma unroll
    for (int k = 0; k < kGS; ++k) {
      const int sp = st * kGS + k;
      meta[k] = sp < n_sp ? tab[4 * sp + 3] : 0;
    }
#pragma unroll
    for (int k = 0; k < kGS; ++k)
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) {
        acc[k][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) acc[k][nb] = O::mma(kr[k][ks], q[nb][ks], acc[k][nb]);
      }
    // meta == 16: a full sub-page of ancestor keys, nothing to mask
    const bool any_mask = ((meta[0] ^ 16) | (meta[1] ^ 16) | (meta[2] ^ 16) | (meta[3] ^ 16)) != 0;
#pragma unroll
    for (int k = 0; k < kGS; ++k) {
      const int nvalid = meta[k] & 255;
      const bool own = (meta[k] >> 8) != 0;
      if (any_mask && (own || nvalid < 16)) {
        int kpos[4] = {0, 0, 0, 0};
        if (own) {
          const int4 pv = *reinterpret_cast<const int4 *>(&R.pos[k][4 * g4]);
          kpos[0] = pv.x;
          kpos[1] = pv.y;
          kpos[2] = pv.z;
          kpos[3] = pv.w;
        }
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) {
          const int ur = row_u(row0 + nb * 16 + rr);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool ok = 4 * g4 + e < nvalid && (!own || kpos[e] <= ur);
            acc[k][nb][e] = ok ? acc[k][nb][e] : -__builtin_inff();
          }
        }
      }
    }
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      // reductions as trees: short dependency chains keep the VALU busy
      float v[4 * kGS];
#pragma unroll
      for (int k = 0; k < kGS; ++k)
#pragma unroll
        for (int e = 0; e < 4; ++e) v[4 * k + e] = acc[k][nb][e];
      const float mx = tree_max(v, m[nb]);
      const float nm = -mx * sl2;
#pragma unroll
      for (int i = 0; i < 4 * kGS; ++i) v[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(v[i], sl2, nm));
      // (m - mx) is exactly 0 while the max is unchanged
      l[nb] = __builtin_fmaf(l[nb], __builtin_amdgcn_exp2f((m[nb] - mx) * sl2), tree_sum(v));
      m[nb] = mx;
    }
  };

  // ---- pass 1: credited column sums ----
  float nlse[NBW][4];
  float *pout = a.part + a.pbase[o] + (int64_t)(slg * a.n_rg + rg) * a.ctxlen[o];
  auto col_stage = [&](Ring<T, D> &R, Red &RD, int st, int n_sp, auto &&between)
                       __attribute__((always_inline)) {
    typename O::reg kr[kGS][KS];   // all operands of the stage first: one LDS wait
#pragma unroll
    for (int k = 0; k < kGS; ++k) operand(R, k, kr[k]);
    between();
    int meta[kGS];
#pragma unroll
    for (int k = 0; k < kGS; ++k) {
      const int sp = st * kGS + k;
      meta[k] = sp < n_sp ? tab[4 * sp + 3] : 0;
    }
    const bool any_own = ((meta[0] | meta[1] | meta[2] | meta[3]) >> 8) != 0;
#pragma unroll
    for (int k = 0; k < kGS; ++k) {
      const bool own = any_own && (meta[k] >> 8) != 0;
      f32x4 acc[NBW];
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) {
        acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) acc[nb] = O::mma(q[nb][ks], kr[k][ks], acc[nb]);
      }
      float pz[4 * NBW];
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          pz[4 * nb + e] = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[nb][e], sl2, nlse[nb][e]));
      if (own) {
        // own tokens are credited only by later rows of the window
        const int kp = R.pos[k][rr];
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            pz[4 * nb + e] = kp < row_u(row0 + nb * 16 + 4 * g4 + e) ? pz[4 * nb + e] : 0.f;
      }
      const float colsum = group_sum(tree_sum(pz));
      if (lane < 16) RD.v[k][wave][lane] = colsum;
    }
  };
  // the previous stage's sums of all four waves, in wave order
  auto finish = [&](const Red &RD, int st, int n_sp) __attribute__((always_inline)) {
    if (wave == 0) {
      // table entries by scalar loads (a per-lane load would wait behind the
      // direct loads in flight)
#pragma unroll
      for (int k = 0; k < kGS; ++k) {
        const int sp = st * kGS + k;
        if (sp >= 0 && sp < n_sp) {
          const int ctx = tab[4 * sp + 2], nvalid = tab[4 * sp + 3] & 255;
          if ((lane >> 4) == k && rr < nvalid)
            pout[ctx + rr] = ((RD.v[k][0][rr] + RD.v[k][1][rr]) + RD.v[k][2][rr]) + RD.v[k][3][rr];
        }
      }
    }
  };

  // one pass over the chain's sub-pages with the ring; `work` computes a
  // stage from a slot, `after` runs (for the previous stage) right after the
  // stage barrier
  auto run = [&](int n_sp, auto &&work, auto &&after) __attribute__((always_inline)) {
    if (n_sp <= 0) return;
    const int n_st = (n_sp + kGS - 1) / kGS;
    issue(r0, 0, n_sp);
    issue(r1, 1, n_sp);
    // A stage reads its operands from the slot first and only then issues the
    // loads that refill the previous slot.  `after` of the previous stage runs
    // once the current stage is computed: its data became visible at this
    // stage's barrier.  Whole rounds of three stages run in a loop with one
    // exit, so every path into a stage has the same loads in flight and the
    // compiler keeps the partial waits.
    int st = 0;
    for (; st + 3 <= n_st; st += 3) {
      stage_sync(Ic<kRing - 2>{});
      work(r0, d0, st, n_sp, [&]() __attribute__((always_inline)) { issue(r2, st + 2, n_sp); });
      after(d2, st - 1, n_sp);   // nothing to finish before the first stage (st - 1 < 0)
      stage_sync(Ic<kRing - 2>{});
      work(r1, d1, st + 1, n_sp, [&]() __attribute__((always_inline)) { issue(r0, st + 3, n_sp); });
      after(d0, st, n_sp);
      stage_sync(Ic<kRing - 2>{});
      work(r2, d2, st + 2, n_sp, [&]() __attribute__((always_inline)) { issue(r1, st + 4, n_sp); });
      after(d1, st + 1, n_sp);
    }
    // the last one or two stages: their loads are already in flight
    auto none = []() __attribute__((always_inline)) {};
    if (st < n_st) {
      stage_sync(Ic<1>{});
      work(r0, d0, st, n_sp, none);
      after(d2, st - 1, n_sp);
      if (st + 1 < n_st) {
        stage_sync(Ic<0>{});
        work(r1, d1, st + 1, n_sp, none);
        after(d0, st, n_sp);
      }
    }
    // drain: every load has landed and the last stage's results are visible
    __builtin_amdgcn_s_waitcnt(0x070);
    __syncthreads();
    const int last = n_st - 1;
    after(last % 3 == 0 ? d0 : (last % 3 == 1 ? d1 : d2), last, n_sp);
    __syncthreads();
  };
  auto nothing = [](const Red &, int, int) __attribute__((always_inline)) {};

  const int n_sp0 = a.nsp[2 * o];
  run(n_sp0,
      [&](Ring<T, D> &R, Red &, int st, int n, auto &&between) __attribute__((always_inline)) {
        lse_stage(R, st, n, between);
      },
      nothing);
  // rows: lane groups merged (log2 units), then each lane takes the lse of
  // the rows it holds in the pass-1 layout (rows 4 g4 + e of each block)
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb) {
    float mm = m[nb] > kFloor ? m[nb] * sl2 : -__builtin_inff();
    float ll = l[nb];
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float mo = __shfl_xor(mm, off, kWave);
      const float lo = __shfl_xor(ll, off, kWave);
      const float mn = fmaxf(mm, mo);
      float ln = 0.f;
      if (mn > -__builtin_inff())
        ln = (mm > -__builtin_inff() ? ll * __builtin_amdgcn_exp2f(mm - mn) : 0.f) +
             (mo > -__builtin_inff() ? lo * __builtin_amdgcn_exp2f(mo - mn) : 0.f);
      mm = mn;
      ll = ln;
    }
    const bool valid = row_u(row0 + nb * 16 + rr) >= 0 && ll > 0.f;
    const float lse = valid ? mm + __log2f(ll) : __builtin_inff();
#pragma unroll
    for (int e = 0; e < 4; ++e) nlse[nb][e] = -__shfl(lse, 4 * g4 + e, kWave);
  }
  const int n_sp1 = a.nsp[2 * o + 1];
  run(n_sp1,
      [&](Ring<T, D> &R, Red &RD, int st, int n, auto &&between) __attribute__((always_inline)) {
        col_stage(R, RD, st, n, between);
      },
      [&](const Red &RD, int st, int n) __attribute__((always_inline)) { finish(RD, st, n); });
}

// Chain length and sub-page count of observer j, with the same checks as the
// validation (a malformed chain gives ok = false and no sub-pages).
struct ObsChain {
  int64_t len, subs;
  int depth;
  bool ok;
};
__device__ ObsChain walk_chain(const Tree &t, int j, int32_t *anc_out) {
  ObsChain r{0, 0, 0, true};
  int chainv[MAXD];
  int d = 0;
  for (int x = j; x >= 0; x = t.parent[x]) {
    if (d >= MAXD || (x > 0 && (t.parent[x] < 0 || t.parent[x] >= x)) ||
        (x == 0 && t.parent[x] != -1)) {
      r.ok = false;
      break;
    }
    const int c = t.n_kept[x];
    if (c < 0 || c > t.n_full[x]) {
      r.ok = false;
      break;
    }
    chainv[d++] = x;
    r.len += c;
    r.subs += (c + 15) / 16;
  }
  if (!r.ok) {
    r.subs = 0;
    d = 1;
    chainv[0] = j;
  }
  r.depth = d - 1;
  if (anc_out)
    for (int e = 0; e < d; ++e) anc_out[e] = chainv[d - 1 - e];
  return r;
}

// One workgroup per observer.  Offsets of the partials and sub-page tables are
// prefixes over observers, so every workgroup walks every observer chain (in
// parallel, one per thread) and keeps its own observer's offsets; it then
// writes that observer's chain data and sub-page table, root first, as
// 16-byte entries (plane row, slot, context offset, valid slots | own << 8)
// that the streaming kernel reads with scalar loads.  Workgroup 0 validates
// the whole tree.
__global__ __launch_bounds__(256) void score_setup(ScoreArgs a, int64_t part_cap,
                                                   int64_t *__restrict__ pbase,
                                                   int64_t *__restrict__ fbase,
                                                   int64_t *__restrict__ tbase,
                                                   int32_t *__restrict__ nsp,
                                                   int32_t *__restrict__ ctxlen,
                                                   int32_t *__restrict__ odepth,
                                                   int32_t *__restrict__ anc) {
  __shared__ int64_t sm[17];
  __shared__ int s_err;
  __shared__ int64_t s_mine[4];
  __shared__ ChainLds ch;
  if (status_failed(a.status)) return;
  const Tree &t = a.t;
  const int me = blockIdx.x;
  const int tid = threadIdx.x;
  if (tid == 0) s_err = 0;
  __syncthreads();
  if (me == 0) {
    for (int i = tid; i < t.V; i += blockDim.x) {
      const int par = t.parent[i];
      const bool ok = (i == 0) ? par == -1 : (par >= 0 && par < i);
      const int c = t.n_kept[i];
      if (!ok || c < 0 || c > t.n_full[i]) atomicOr(&s_err, 1);
    }
  }
  const int slabs = a.S * a.pl.Hkv * a.n_rg;
  int64_t run = 0, frun = 0, trun = 0;
  for (int base = 0; base < a.n_obs; base += blockDim.x) {
    const int o = base + tid;
    int64_t len = 0, subs = 0;
    if (o < a.n_obs) {
      const int j = a.obs[o];
      if (j < 0 || j >= t.V) {
        atomicOr(&s_err, 1);
      } else {
        const ObsChain r = walk_chain(t, j, o == me ? anc + (int64_t)o * MAXD : nullptr);
        if (!r.ok) atomicOr(&s_err, 2);
        len = r.len;
        subs = r.subs;
        if (o == me) {
          odepth[o] = r.depth;
          const int own = r.ok ? (t.n_kept[j] + 15) / 16 : 0;
          nsp[2 * o] = (int32_t)subs;
          nsp[2 * o + 1] = r.ok ? (int32_t)(a.self_window ? subs : subs - own) : 0;
          ctxlen[o] = (int32_t)len;
          s_mine[2] = subs;
        }
      }
    }
    int64_t tot, ftot, ttot;
    const int64_t ex = block_exclusive_scan<int64_t>(len * slabs, sm, &tot);
    const int64_t fx = block_exclusive_scan<int64_t>(len, sm, &ftot);
    const int64_t tx = block_exclusive_scan<int64_t>(subs, sm, &ttot);
    if (o == me) {
      s_mine[0] = run + ex;
      s_mine[1] = trun + tx;
      s_mine[3] = frun + fx;
    }
    run += tot;
    frun += ftot;
    trun += ttot;
  }
  __syncthreads();
  // the folded sums follow the partials, then the sub-page tables (16-byte
  // entries, 16-byte aligned)
  const int64_t tab0 = (run + frun + 3) & ~(int64_t)3;
  const bool fits = tab0 + 4 * trun <= part_cap;
  if (tid == 0) {
    pbase[me] = s_mine[0];
    fbase[me] = run + s_mine[3];
    tbase[me] = tab0 + 4 * s_mine[1];
    if (me == 0) {
      if (s_err & 1) status_error(a.status, ARBOR_EINVAL);
      else if (s_err & 2) status_error(a.status, ARBOR_EUNSUPPORTED);
      else if (!fits) status_error(a.status, ARBOR_EWORKSPACE);
    }
  }
  const int j = a.obs[me];
  if (s_err || !fits || j < 0 || j >= t.V) return;   // uniform: s_err settled at the sync
  build_chain(t, a.pl, j, ch);
  const int n = (int)s_mine[2];
  int4 *tab = reinterpret_cast<int4 *>(a.part + tab0 + 4 * s_mine[1]);
  for (int sp = tid; sp < n; sp += blockDim.x) {
    const SubPage e = sub_page(t, a.pl, ch, sp);
    tab[sp] = make_int4(e.row, e.slot, e.ctx, e.nvalid | ((e.d == ch.depth ? 1 : 0) << 8));
  }
}

// Fold the (slice layer, kv head, row group) slabs of every observer: one
// column sum per (observer, credited context key), summed in slab order.
__global__ __launch_bounds__(256) void score_fold(ScoreArgs a, const int64_t *__restrict__ fbase) {
  if (status_failed(a.status)) return;
  const int o = blockIdx.x;
  const int len = a.ctxlen[o];
  const int own_c = a.t.n_kept[a.obs[o]];
  const int credited = a.self_window ? len : len - own_c;
  const int nslab = a.S * a.pl.Hkv * a.n_rg;
  const float *src = a.part + a.pbase[o];
  float *dst = a.part + fbase[o];
  for (int x = blockIdx.y * blockDim.x + threadIdx.x; x < credited; x += gridDim.y * blockDim.x) {
    float acc = 0.f;
    for (int sl = 0; sl < nslab; ++sl) acc += src[(int64_t)sl * len + x];
    dst[x] = acc;
  }
}

// a_i and s_i of block i from its A (one wave).
__device__ void block_final(const Tree &t, int i, const float *__restrict__ A,
                            const int64_t *__restrict__ rows_seen, const float *__restrict__ v_in,
                            const float *__restrict__ u_in, float th0, float th1, float th2,
                            float *__restrict__ a_out, float *__restrict__ s_out) {
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

struct FinalArgs {
  const float *v_in, *u_in;
  float th0, th1, th2;
  float *a_out, *s_out;
};

// A += folded sums of every observer below block i (observer order, fp64);
// rows_seen_i grows.  The four waves of a workgroup split the observers of a
// 64-slot chunk and are combined in wave order.
__global__ __launch_bounds__(256) void score_reduce(ScoreArgs a, const int64_t *__restrict__ fbase,
                                                    float *__restrict__ A,
                                                    int64_t *__restrict__ rows_seen) {
  __shared__ int64_t hbase[256];
  __shared__ int s_wcnt[4];
  __shared__ double s_acc[4][64];
  if (status_failed(a.status)) return;
  const Tree &t = a.t;
  const Pool &pl = a.pl;
  const int i = blockIdx.x;
  const int c = t.n_kept[i];
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const float *fold = a.part;
  int di = 0, ctxoff = 0;
  for (int x = t.parent[i]; x >= 0 && di < MAXD; x = t.parent[x]) {
    ++di;
    ctxoff += t.n_kept[x];
  }
  const int64_t tb = t.tok_off[i];
  const int64_t po = t.page_off[i];
  int64_t rows_add = 0;
  const int nchunk = (c + 63) / 64;
  for (int ob = 0; ob < a.n_obs; ob += 256) {
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
    const int nh = s_wcnt[0] + s_wcnt[1] + s_wcnt[2] + s_wcnt[3];
    if (hit) {
      hbase[before + rank_below(bm, lane)] = fbase[o] + ctxoff;
      if (blockIdx.y == 0) rows_add += (int64_t)a.S * pl.Hkv * pl.G * min(a.W, t.n_full[a.obs[o]]);
    }
    __syncthreads();
    if (nh > 0) {
      for (int chk = blockIdx.y; chk < nchunk; chk += gridDim.y) {
        const int s = chk * 64 + lane;
        double acc = 0.0;
        if (s < c) {
          int h = wave;
          for (; h + 12 < nh; h += 16) {
            const float f0 = fold[hbase[h] + s];
            const float f1 = fold[hbase[h + 4] + s];
            const float f2 = fold[hbase[h + 8] + s];
            const float f3 = fold[hbase[h + 12] + s];
            acc += (double)f0;
            acc += (double)f1;
            acc += (double)f2;
            acc += (double)f3;
          }
          for (; h < nh; h += 4) acc += (double)fold[hbase[h] + s];
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
  }
  if (blockIdx.y == 0) {
    rows_add = block_sum<int64_t>(rows_add, reinterpret_cast<int64_t *>(&s_acc[0][0]));
    if (threadIdx.x == 0) rows_seen[i] += rows_add;
  }
}

// a_i and s_i from the updated A (one wave per block).
__global__ __launch_bounds__(256) void score_final(Tree t, const float *__restrict__ A,
                                                   const int64_t *__restrict__ rows_seen,
                                                   FinalArgs fa, int32_t *status) {
  if (status_failed(status)) return;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= t.V) return;
  block_final(t, i, A, rows_seen, fa.v_in, fa.u_in, fa.th0, fa.th1, fa.th2, fa.a_out, fa.s_out);
}

template <class T, int D>
void launch_attn_nb(int NBW, dim3 grid, hipStream_t stream, const ScoreArgs &a) {
  switch (NBW) {
    case 1: hipLaunchKernelGGL((score_attn<T, D, 1>), grid, dim3(256), 0, stream, a); break;
    case 2: hipLaunchKernelGGL((score_attn<T, D, 2>), grid, dim3(256), 0, stream, a); break;
    default: hipLaunchKernelGGL((score_attn<T, D, 4>), grid, dim3(256), 0, stream, a); break;
  }
}

void launch_attn(int dtype, int D, int NBW, dim3 grid, hipStream_t stream, const ScoreArgs &a) {
  if (dtype == ARBOR_BF16) {
    if (D == 128) launch_attn_nb<__bf16, 128>(NBW, grid, stream, a);
    else launch_attn_nb<__bf16, 64>(NBW, grid, stream, a);
  } else {
    if (D == 128) launch_attn_nb<float, 128>(NBW, grid, stream, a);
    else launch_attn_nb<float, 64>(NBW, grid, stream, a);
  }
}

// Row blocks per wave: the workgroup (4 waves) covers 64 * NBW query rows.
int blocks_per_wave(int rows_total) {
  if (rows_total <= 64) return 1;
  if (rows_total <= 128) return 2;
  return 4;
}

}  // namespace

size_t score_workspace(const arbor_geom_t *g, const arbor_sizes_t *sz) {
  const int rows_total = g->q_per_kv * sz->window;
  const int NB = 4 * blocks_per_wave(rows_total);
  const int n_rg = (rows_total + 16 * NB - 1) / (16 * NB);
  const size_t nobs = (size_t)(sz->max_observers > 0 ? sz->max_observers : 0);
  const size_t slabs = (size_t)sz->n_slice * g->num_kv_heads * n_rg;
  size_t b = 0;
  // offsets, counts, chains (each carve rounds up to 256 B)
  b += nobs * (8 * 3 + 4 * 4) + nobs * MAXD * 4 + 8 * 256;
  // partials and their folded sums
  b += nobs * (slabs + 1) * (size_t)sz->max_context * 4 + 256;
  // sub-page tables: at most one ragged sub-page per chain node
  b += nobs * ((size_t)sz->max_context / 16 + MAXD + 1) * 16 + 256;
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
  if ((int64_t)pl.num_pages * pl.Hkv * pl.P >= ((int64_t)1 << 31)) return ARBOR_EUNSUPPORTED;
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
  const int NBW = blocks_per_wave(rows_total);
  const int NB = 4 * NBW;
  a.n_rg = (rows_total + 16 * NB - 1) / (16 * NB);
  const float scale = params->softmax_scale > 0.f ? params->softmax_scale
                                                  : 1.0f / sqrtf((float)geom->head_dim);
  a.sl2 = scale * kLog2e;
  a.self_window = params->score_self_window;
  a.status = status;
  Carve cv(workspace, workspace_bytes);
  const size_t nobs = n_obs > 0 ? (size_t)n_obs : 1;
  int64_t *pbase = cv.take<int64_t>(nobs);
  int64_t *fbase = cv.take<int64_t>(nobs);
  int64_t *tbase = cv.take<int64_t>(nobs);
  int32_t *nsp = cv.take<int32_t>(2 * nobs);
  int32_t *ctxlen = cv.take<int32_t>(nobs);
  int32_t *odepth = cv.take<int32_t>(nobs);
  int32_t *anc = cv.take<int32_t>(nobs * MAXD);
  if (!cv.ok) return ARBOR_EWORKSPACE;
  float *part = reinterpret_cast<float *>(cv.rest());
  const int64_t part_cap = (int64_t)(cv.remaining() / 4);
  a.part = part;
  a.pbase = pbase;
  a.tbase = tbase;
  a.nsp = nsp;
  a.ctxlen = ctxlen;
  a.odepth = odepth;
  a.anc = anc;
  const FinalArgs fa{v_in, u_in, params->theta[0], params->theta[1], params->theta[2], a_out, s_out};
  if (n_obs > 0) {
    hipLaunchKernelGGL(score_setup, dim3(n_obs), dim3(256), 0, stream, a, part_cap, pbase, fbase,
                       tbase, nsp, ctxlen, odepth, anc);
    const int n_planes = n_slice * pl.Hkv * a.n_rg;
    const dim3 grid((unsigned)(((n_planes + kXcds - 1) / kXcds) * n_obs * kXcds));
    timing_begin(ARBOR_KERNEL_SCORE_ATTN, stream);
    launch_attn(geom->dtype, geom->head_dim, NBW, grid, stream, a);
    timing_end(ARBOR_KERNEL_SCORE_ATTN, stream);
    hipLaunchKernelGGL(score_fold, dim3(n_obs, 8), dim3(256), 0, stream, a, fbase);
    hipLaunchKernelGGL(score_reduce, dim3(t.V, 16), dim3(256), 0, stream, a, fbase, A, rows_seen);
  }
  hipLaunchKernelGGL(score_final, dim3((t.V + 3) / 4), dim3(256), 0, stream, t, A, rows_seen, fa,
                     status);
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
