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
//   setup   one workgroup: validates the tree, walks every observer chain
//           (one thread per observer) for the partial / table offsets (prefix
//           sums over observers) and lists the blocks that receive credit;
//   tables  one workgroup per observer: its 16-slot sub-page table (up to
//           512 observers, in the setup's launch: each table workgroup walks
//           the observer chains itself for its offset);
//   attn    per (observer, slice layer, kv head, 1, 2 or 4 groups of up to
//           64 rows), two passes over the same (row, key) pairs as MFMA tiles
//           of 16 keys x 16 rows, one wave per (row group, key split), the
//           waves of a row group taking alternate 16-key sub-pages:
//           C = K Q^T for the row log-sum-exp, then C = Q K^T for per-key
//           sums of exp2(z - lse) -> one partial per credited context key
//           and workgroup (its row groups added in order);
//   fold    per observer: sum its (slice layer, kv head, workgroup) partials;
//   reduce  per credited block i and 64-slot chunk: sum the folded partials of
//           every observer below i in observer order (fp64) into A, rows_seen;
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
  int n_slab;       // partial slabs per (slice layer, kv head): one per workgroup's row groups
  float sl2;        // softmax scale * log2(e)
  int self_window;
  float *part;      // partial column sums
  const int64_t *pbase;   // [n_obs]
  const int64_t *tbase;   // [n_obs]: float offset (in part) of the observer's sub-page table
  const int32_t *nsp;     // [n_obs][2]: sub-pages of the chain, and of the credited part
  const int32_t *ctxlen;  // [n_obs]
  const int32_t *odepth;  // [n_obs]
  const int32_t *anc;     // [n_obs][MAXD]
  const int32_t *nctx;    // [V]: context offset of each chain node's first token (setup)
  const int32_t *ndep;    // [V]: its depth
  int32_t *status;
};

// Chain of observer j in LDS, root first, with a table of its 16-slot
// sub-pages so the key loop needs no dependent page-table load.
constexpr int SPCAP = 512;
constexpr int kSetupLds = 2048;   // trees up to this many nodes are walked from LDS
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

// The chain's in-LDS sub-page table (the first SPCAP sub-pages; longer chains
// compute the rest on demand).
__device__ __forceinline__ void fill_table(const Tree &t, const Pool &pl, ChainLds &ch, int n) {
  const int n_sp = min(n, SPCAP);
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

// ---------------------------------------------------------------------------
template <class T, int D>
struct KTile {
  static constexpr int R = D * (int)sizeof(T) / 16;   // 16-byte pieces of a key row
  static constexpr int RQ = R / 4;                     // pieces of one lane group
  static constexpr int XM = (R < 16 ? R : 16) - 1;     // piece swizzle mask
  static constexpr int BYTES = 16 * R * 16;            // one 16-key sub-page
  static constexpr int NDMA = BYTES / 1024;            // 1 KB direct loads per sub-page
  static constexpr int ND = NDMA;
  static constexpr int KS = D / 4 / Op<T>::kPerStep;   // MFMA k-steps over head_dim
  static constexpr int SPP = KS / RQ;                   // k-steps per 16-byte piece
};

typedef __attribute__((address_space(3))) void *LdsPtr;
// This wave's part of the direct loads (global -> LDS) of one BYTES-long tile
// at src: its loads m < n are the tile's loads c = c0 + step m, and lane L's
// 16 bytes of load c land at lds + 1024 c + 16 L.  A buffer resource over the
// tile (scalar registers) leaves each lane a 32-bit offset, and bounds every
// access to the tile.
// (host-device so the kernel's host-device lambdas can call it; the host
// pass of the compiler never runs it)
template <int NW, int BYTES>
__host__ __device__ __forceinline__ void dma_part(const char *src, char *lds, int c0, int step,
                                                  int n, const int (&off)[NW]) {
#if defined(__HIP_DEVICE_COMPILE__)
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(src), 0, BYTES, 0x00020000);
#pragma unroll
  for (int m = 0; m < NW; ++m)
    if (m < n)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (LdsPtr)(lds + 1024 * (c0 + step * m)), 16,
                                               off[m], 0, 0, 0);
#endif
}
template <class T, int D>
struct KBuf {
  __attribute__((aligned(16))) char k[KTile<T, D>::BYTES];
};
constexpr int kXcds = 8;     // accelerator dies of the device; workgroups go round-robin
constexpr int kMask0 = 1 << 9;    // table flag: pass 0 must mask keys of this sub-page
constexpr int kMask1 = 1 << 10;   // table flag: pass 1 must mask keys of this sub-page

// v_max3 without the quieting the IEEE maxnum lowering adds to each operand:
// the operands are MFMA results or -inf, never signalling NaNs.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Wait until at most n vector-memory operations of this wave are in flight
// (gfx9 encoding: vmcnt bits 3:0 and 15:14; expcnt and lgkmcnt not waited).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
  asm volatile("" ::: "memory");
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

// MFMA operand of k-step c within a 16-byte piece
template <class T>
__device__ __forceinline__ typename Op<T>::reg piece_op(const uint4 &p, int c);
template <>
__device__ __forceinline__ bf16x8 piece_op<__bf16>(const uint4 &p, int) {
  return __builtin_bit_cast(bf16x8, p);
}
template <>
__device__ __forceinline__ float piece_op<float>(const uint4 &p, int c) {
  return __uint_as_float(c == 0 ? p.x : (c == 1 ? p.y : (c == 2 ? p.z : p.w)));
}

// Streaming kernel.  One workgroup of four waves per (observer, slice layer,
// kv head, RGW groups of up to 16 NRB query rows), RGW = 1, 2 or 4.  Wave w
// is (row group w % RGW, key split w / RGW): the 4 / RGW key splits take the
// chain's 16-key sub-pages round-robin (split x takes sub-pages x, x + 4 /
// RGW, ...), and every wave holds the Q of its row group in registers.  The
// RGW waves of a key split work on the same sub-page at each step: each loads
// a part of it into their shared ring of LDS slots and they meet at a barrier
// before reading it, so a key tile moves from L2 to LDS once for RGW row
// groups.  A key's sum over a row group never leaves its wave; the RGW sums
// of a key meet in LDS and are stored as one partial.
//   pass 0  C = K Q^T: each lane keeps a running max / sum of one row over its
//           keys; lanes, then the key splits, are merged into the row's
//           log2-sum-exp;
//   pass 1  C = Q K^T: per key, the sum over the group's rows of
//           exp2(z - lse); the workgroup's partial for that key is the sum
//           of its row groups' values, in row-group order.
// Keys reach the ring by direct global->LDS loads in which each 16-lane group
// reads one whole 256-byte key row (coalesced).  The 16-byte pieces of key r
// are stored XOR-permuted by r, so the sixteen lanes of an MFMA operand read
// (keys 0..15, one piece each) hit distinct banks.  A wave waits only for its
// own loads; the barrier (RGW > 1 only) does not wait for memory.
template <class T, int D, int NRB, int RGW>
__global__ __launch_bounds__(256, 3) void score_attn(ScoreArgs a) {
  using O = Op<T>;
  using KT = KTile<T, D>;
  using Buf = KBuf<T, D>;
  constexpr int R = KT::R, RQ = KT::RQ, KS = KT::KS, SPP = KT::SPP, ND = KT::ND;
  constexpr int ROWS = 16 * NRB;            // rows of one wave (a row group)
  constexpr int KSW = 4 / RGW;              // key splits of the workgroup
  constexpr int NDW = (ND + RGW - 1) / RGW; // direct loads of a wave per tile (at most)
  static_assert(RGW == 1 || RGW == 2 || RGW == 4, "row groups per workgroup");
  constexpr float kFloor = -1e30f;
  // one ring slot per object, so the compiler can tell a buffer being filled
  // from the one being read; slot [x] belongs to key split x
  __shared__ Buf b0[KSW], b1[KSW], b2[KSW];
  __shared__ float2 s_ml[KSW][RGW * ROWS];
  __shared__ __attribute__((aligned(16))) float s_lse[RGW * ROWS];
  // pass 1: the key sums of the last four steps, per key split, key and row
  // group (used when RGW > 1)
  __shared__ __attribute__((aligned(16))) float s_cs[KSW][4][16 * RGW];
  __shared__ int s_bad;
  // XCD-aware order: workgroup n runs on XCD n % 8, so XCD x takes the
  // (slice layer, kv head, RGW row groups) planes p = x, x + 8, ...; it runs the
  // observers in reverse list order, each over all its planes in turn.  For
  // observers listed in id order of a tree numbered level by level (children
  // after their parents) that is deepest first: the longest work starts
  // first, so the grid ends on the shortest, and siblings, which share their
  // whole ancestor chain, run together and read those keys from the XCD's L2
  // (any other order is as correct, only slower)
  const int n_rgp = (a.n_rg + RGW - 1) / RGW;
  const int n_planes = a.S * a.pl.Hkv * n_rgp;
  const int xcd = (int)blockIdx.x % kXcds;
  const int idx = (int)blockIdx.x / kXcds;
  const int ppx = (n_planes + kXcds - 1) / kXcds;   // planes per XCD
  const int o = a.n_obs - 1 - idx / ppx;
  const int plane = (idx % ppx) * kXcds + xcd;
  if (plane >= n_planes) return;
  if (threadIdx.x == 0) s_bad = status_failed(a.status);
  __syncthreads();
  if (s_bad) return;
  const Tree &t = a.t;
  const Pool &pl = a.pl;
  const int slg = plane / n_rgp;
  const int si = slg / pl.Hkv;
  const int g = slg % pl.Hkv;
  const int layer = a.slice[si];
  const int j = a.obs[o];
  // the chain's sub-page table: entry sp = (plane row, slot, context offset,
  // valid slots | own << 8 | mask flags)
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // wave = (key split ksw, row group rgw of the workgroup): the RGW waves of
  // a key split share its key tiles, each loading a part of every tile
  const int rgw = wave % RGW;
  const int ksw = wave / RGW;
  const int rg = (plane % n_rgp) * RGW + rgw;   // may be >= n_rg: rows all invalid
  const int r = lane & 15;
  const int q = lane >> 4;
  const int G = pl.G;
  const int nj = t.n_full[j];
  const int wj = min(a.W, nj);
  const int rows_total = G * a.W;
  const int row0 = rg * ROWS;
  const float sl2 = a.sl2;
  // position of window row `row` of the group, -1 if none
  auto urow = [&](int row) __attribute__((always_inline)) -> int {
    row += row0;
    if (row >= rows_total) return -1;
    const int tt = row % a.W;
    return tt < wj ? nj - wj + tt : -1;
  };

  // Q of every row of the group: lane (r, q) holds the q-th quarter of row
  // 16 rb + r, as RQ 16-byte pieces
  uint4 qp[NRB][RQ];
  const T *qbase = static_cast<const T *>(a.q_win) +
                   ((((int64_t)o * a.S + si) * (pl.Hkv * G) + (int64_t)g * G) * a.W) * D;
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    const int row = row0 + rb * 16 + r;
    const bool rv = row < rows_total;
    const uint4 *rp = reinterpret_cast<const uint4 *>(qbase + (int64_t)(rv ? row : 0) * D) + q * RQ;
#pragma unroll
    for (int jp = 0; jp < RQ; ++jp) qp[rb][jp] = rv ? rp[jp] : make_uint4(0, 0, 0, 0);
  }
  const int64_t plane_row0 = (int64_t)layer * pl.num_pages * pl.Hkv * pl.P + (int64_t)g * pl.P;
  const char *kplane = static_cast<const char *>(pl.k) + plane_row0 * D * (int64_t)sizeof(T);
  // byte offset, within a sub-page, of the piece lane L fetches for this
  // wave's direct load m (load c = rgw + RGW m of the tile, if c < ND)
  int src_off[NDW];
#pragma unroll
  for (int m = 0; m < NDW; ++m) {
    const int c = rgw + RGW * m;
    const int sig = 64 * c + lane;           // LDS slot: key sig / R, stored piece sig % R
    const int kr = sig / R;
    src_off[m] = 16 * (R * kr + ((sig % R) ^ (kr & KT::XM)));
  }
  const int n_dma = ND >= RGW ? NDW : (rgw < ND ? 1 : 0);   // this wave's loads per tile
  // LDS byte offset of piece jp of this lane's quarter of key r
  const int lbase = 16 * (R * r + ((q * RQ) ^ (r & KT::XM)));

  // the chain's sub-page table as 16-byte vectors (read into registers)
  const int4 *tabv = reinterpret_cast<const int4 *>(a.part + a.tbase[o]);
  // one sub-page: a buffer resource over its BYTES (set up in scalar
  // registers), so each lane supplies only a 32-bit offset
  auto issue = [&](Buf &B, int row) __attribute__((always_inline)) {
    dma_part<NDW, KT::BYTES>(kplane + (int64_t)row * (D * (int)sizeof(T)), B.k, rgw, RGW, n_dma,
                             src_off);
  };
  // offsets of this lane's pieces from the start of a ring (slot `ksw`
  // included), so a read addresses the ring's fixed LDS base plus a register
  int roff[RQ];
#pragma unroll
  for (int jp = 0; jp < RQ; ++jp) roff[jp] = ksw * (int)sizeof(Buf) + (lbase ^ (16 * jp));
  auto read_k = [&](const Buf (&ring)[KSW], uint4 (&kp)[RQ]) __attribute__((always_inline)) {
#pragma unroll
    for (int jp = 0; jp < RQ; ++jp)
      kp[jp] = *reinterpret_cast<const uint4 *>(reinterpret_cast<const char *>(ring) + roff[jp]);
  };

  // One pass over this key split's sub-pages sp = ksw + KSW i of the first
  // n_sp of the chain, software-pipelined over a ring of three LDS slots.
  // Step i waits for this wave's part of sub-page i (the next one may stay in
  // flight) and, when RGW waves share the tiles, meets them at a barrier, so
  // every part has landed and every wave is done with sub-page i - 1; it
  // refills the slot of sub-page i - 1 with sub-page i + 2, reads its
  // operands, then runs
  //   fix(prev)  rare, branchy corrections of sub-page i - 1 (key masks);
  //   mm(kp)     the MFMAs of sub-page i, interleaved in one straight-line
  //   hot(prev)  block with the VALU work of sub-page i - 1, so the matrix
  //              core and the VALU work side by side within the wave;
  //   post(prev) rare corrections after the fact, and stores;
  // flush() runs once a window's last barrier has passed (empty unless
  // results are combined across the waves of a key split).
  // The table entries of a window of up to 64 steps sit in registers (lane L
  // holds step L) and are read with readlane, so the loop has no scalar loads.
  // Every wave of the workgroup runs the same steps (those of key split 0):
  // a split with one sub-page fewer runs its last step on a copy of its
  // previous entry with no valid slots (masked in pass 0, not stored in
  // pass 1), so the barriers pair up.
  struct StepState {
    f32x4 acc[NRB];
    int meta, ctx, slot;
  };
  // the barrier of the waves sharing a tile (the whole workgroup), without
  // the wait for all memory operations that a fenced barrier would add
  auto tile_sync = [&]() __attribute__((always_inline)) {
    if constexpr (RGW > 1) asm volatile("s_barrier" ::: "memory");
  };
  auto run = [&](int n_sp, auto &&mm, auto &&fix, auto &&hot, auto &&post,
                 auto &&flush)
                 __attribute__((always_inline)) {
    const int cnt = (n_sp + KSW - 1) / KSW;
    for (int base = 0; base < cnt; base += 64) {
      const int wc = min(64, cnt - base);
      int4 e = make_int4(0, 0, 0, 0);
      if (lane < wc) {
        const int sp = ksw + KSW * (base + lane);
        if (sp < n_sp) {
          e = tabv[sp];
        } else {
          e = tabv[n_sp - 1];
          e.w = kMask0;
        }
      }
      // a field of window step i (clamped to the last step)
      auto ent = [&](int i, int v) __attribute__((always_inline)) -> int {
        return __builtin_amdgcn_readlane(v, min(i, wc - 1));
      };
      auto issue_i = [&](Buf &B, int i) __attribute__((always_inline)) {
        issue(B, ent(i, e.x));
      };
      issue_i(b0[ksw], 0);
      issue_i(b1[ksw], 1);
      StepState prev;
      {
        wait_vm<NDW>();
        tile_sync();
        uint4 kp[RQ];
        read_k(b0, kp);
        issue_i(b2[ksw], 2);
        prev = mm(kp, ent(0, e.y), ent(0, e.w), ent(0, e.z));
      }
      auto body = [&](const Buf (&ring)[KSW], int i) __attribute__((always_inline)) {
        uint4 kp[RQ];
        read_k(ring, kp);
        fix(prev);
        const StepState cur = mm(kp, ent(i, e.y), ent(i, e.w), ent(i, e.z));
        hot(prev);
#pragma unroll
        for (int k = 0; k < KS * NRB; ++k) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
        }
        post(prev, false);
        prev = cur;
      };
      int i = 1;
      for (; i + 3 <= wc; i += 3) {
        wait_vm<NDW>();
        tile_sync();
        issue_i(b0[ksw], i + 2);
        body(b1, i);
        wait_vm<NDW>();
        tile_sync();
        issue_i(b1[ksw], i + 3);
        body(b2, i + 1);
        wait_vm<NDW>();
        tile_sync();
        issue_i(b2[ksw], i + 4);
        body(b0, i + 2);
      }
      // the last one or two sub-pages (i in slot 1, i + 1 in slot 2)
      if (i < wc) {
        wait_vm<NDW>();
        tile_sync();
        body(b1, i);
        if (i + 1 < wc) {
          wait_vm<0>();
          tile_sync();
          body(b2, i + 1);
        }
      }
      fix(prev);
      hot(prev);
      post(prev, true);
      // drain (the clamped reloads past the end), and let every wave finish
      // reading, before the ring is reused; the LDS writes of the last steps
      // complete before the barrier, so flush() sees them
      wait_vm<0>();
      if constexpr (RGW > 1) asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      tile_sync();
      flush();
    }
  };

  // ---- pass 0: row log2-sum-exp ----
  // The running sum l of a row is kept relative to a reference max m, held as
  // nm = -m sl2 (log2 units; nm0 while the row has no reference).  m moves
  // only when the terms of a sub-page grow large: the terms are computed
  // against the current reference first, and if the four terms of any lane of
  // any row add up to more than 2^64 (or overflow), the wave moves every row's
  // reference to its max, rescales the sum and recomputes that sub-page's
  // terms.  In practice only a wave's first sub-page sets the reference: a
  // term stays below 2^64 unless a key's logit exceeds the reference by 64
  // bits, and a row's sum of at most 2^20 such terms stays far below the fp32
  // range, while terms that fall far below the reference were negligible
  // against the sum (at least 1) anyway.  The common step needs no max.
  constexpr float kGrow = 0x1p64f;
  const float nm0 = -kFloor * sl2;
  float nm[NRB], l[NRB], lt[NRB];
  bool grow = false;
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    nm[rb] = nm0;
    l[rb] = 0.f;
  }
  run(a.nsp[2 * o],
      [&](const uint4 (&kp)[RQ], int slot, int meta, int ctx) __attribute__((always_inline)) {
        StepState st;
        st.meta = meta;
        st.ctx = ctx;
        st.slot = slot;
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) st.acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int rb = 0; rb < NRB; ++rb)
            st.acc[rb] = O::mma(piece_op<T>(kp[ks / SPP], ks % SPP),
                                piece_op<T>(qp[rb][ks / SPP], ks % SPP), st.acc[rb]);
        return st;
      },
      [&](StepState &st) __attribute__((always_inline)) {
        if (st.meta & kMask0) {
          // a ragged sub-page, or own keys some rows may not see (position > row)
          const int nvalid = st.meta & 255;
          const bool own = ((st.meta >> 8) & 1) != 0;
          int kpos[4] = {0, 0, 0, 0};
          if (own) {
            const int4 pv = *reinterpret_cast<const int4 *>(pl.slot_pos + st.slot + 4 * q);
            kpos[0] = pv.x;
            kpos[1] = pv.y;
            kpos[2] = pv.z;
            kpos[3] = pv.w;
          }
#pragma unroll
          for (int rb = 0; rb < NRB; ++rb) {
            const int ur = urow(rb * 16 + r);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const bool ok = 4 * q + e < nvalid && (!own || kpos[e] <= ur);
              st.acc[rb][e] = ok ? st.acc[rb][e] : -__builtin_inff();
            }
          }
        }
      },
      [&](const StepState &st) __attribute__((always_inline)) {
        grow = false;
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
          float e4[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            e4[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(st.acc[rb][e], sl2, nm[rb]));
          lt[rb] = tree_sum(e4);
          // computed here, inside the block shared with the MFMAs (the
          // compiler would otherwise sink it into the branch that uses it)
          asm volatile("" : "+v"(lt[rb]));
          grow |= !(lt[rb] <= kGrow);          // also true for +inf
        }
      },
      [&](const StepState &st, bool) __attribute__((always_inline)) {
        if (__builtin_amdgcn_ballot_w64(grow) != 0) {
#pragma unroll
          for (int rb = 0; rb < NRB; ++rb) {
            // the new reference in log2 units, and the factor that moves the
            // sum onto it (exactly 1 for a row whose max is unchanged)
            const float mxs = fmaxf(
                max3f(max3f(st.acc[rb][0], st.acc[rb][1], st.acc[rb][2]), st.acc[rb][3],
                      st.acc[rb][3]) * sl2,
                -nm[rb]);
            const float sc = __builtin_amdgcn_exp2f(-mxs - nm[rb]);
            nm[rb] = -mxs;
            float e4[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
              e4[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(st.acc[rb][e], sl2, nm[rb]));
            l[rb] = __builtin_fmaf(l[rb], sc, tree_sum(e4));
          }
        } else {
#pragma unroll
          for (int rb = 0; rb < NRB; ++rb) l[rb] += lt[rb];
        }
      },
      []() {});
  // merge the four lane groups (log2 units), then the four waves, in order
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    float mm = nm[rb] < nm0 ? -nm[rb] : -__builtin_inff();
    float ll = l[rb];
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
    if (lane < 16) s_ml[ksw][rgw * ROWS + rb * 16 + lane] = make_float2(mm, ll);
  }
  __syncthreads();
  for (int x = tid; x < RGW * ROWS; x += blockDim.x) {
    float mm = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < KSW; ++w) mm = fmaxf(mm, s_ml[w][x].x);
    float ll = 0.f;
    if (mm > -__builtin_inff()) {
#pragma unroll
      for (int w = 0; w < KSW; ++w) {
        const float2 v = s_ml[w][x];
        ll += v.x > -__builtin_inff() ? v.y * __builtin_amdgcn_exp2f(v.x - mm) : 0.f;
      }
    }
    // (urow counts rows from this wave's group: re-base to group x / ROWS)
    const bool valid = urow(x - rgw * ROWS) >= 0 && ll > 0.f;
    s_lse[x] = valid ? mm + __log2f(ll) : __builtin_inff();
  }
  __syncthreads();
  // pass-1 layout: this lane holds rows 16 rb + 4 q + e of its key
  float nlse[NRB][4];
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    const float4 v = *reinterpret_cast<const float4 *>(&s_lse[rgw * ROWS + rb * 16 + 4 * q]);
    nlse[rb][0] = -v.x;
    nlse[rb][1] = -v.y;
    nlse[rb][2] = -v.z;
    nlse[rb][3] = -v.w;
  }

  // ---- pass 1: credited column sums ----
  // With RGW row groups per workgroup, the waves of a key split add their sums
  // of a key into one slab: each wave writes its sums of step m into a ring of
  // four LDS slots, and two steps later (after two barriers, by which every
  // wave's write has completed) the wave rgw = m mod RGW adds the RGW values
  // in row-group order and stores them; a window's last three steps are
  // stored after its final barrier.
  float *pout = a.part + a.pbase[o] + (int64_t)(slg * a.n_slab + rg / RGW) * a.ctxlen[o];
  float colsum = 0.f;
  int m = 0;                            // step of the window (stores pending)
  int ctx1 = 0, ctx2 = 0, ctx3 = 0;     // context offsets of steps m-1, m-2, m-3
  int nv1 = 0, nv2 = 0, nv3 = 0;        // and their valid slots
  auto load_sums = [&](int step, float (&v)[RGW]) __attribute__((always_inline)) {
    const float *src = &s_cs[ksw][step & 3][(lane & 15) * RGW];
    if constexpr (RGW == 4) {
      const float4 x = *reinterpret_cast<const float4 *>(src);
      v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
    } else if constexpr (RGW == 2) {
      const float2 x = *reinterpret_cast<const float2 *>(src);
      v[0] = x.x; v[1] = x.y;
    } else {
      v[0] = src[0];
    }
  };
  auto store_sums = [&](const float (&v)[RGW], int ctx, int nv) __attribute__((always_inline)) {
    float x = v[0];
#pragma unroll
    for (int u = 1; u < RGW; ++u) x += v[u];
    if (lane < nv) pout[ctx + lane] = x;
  };
  run(a.nsp[2 * o + 1],
      [&](const uint4 (&kp)[RQ], int slot, int meta, int ctx) __attribute__((always_inline)) {
        StepState st;
        st.meta = meta;
        st.ctx = ctx;
        st.slot = slot;
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) st.acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int rb = 0; rb < NRB; ++rb)
            st.acc[rb] = O::mma(piece_op<T>(qp[rb][ks / SPP], ks % SPP),
                                piece_op<T>(kp[ks / SPP], ks % SPP), st.acc[rb]);
        return st;
      },
      [&](StepState &st) __attribute__((always_inline)) {
        if (st.meta & kMask1) {
          // own tokens are credited only by later rows of the window (this
          // lane's key is slot r of the sub-page; a rare step, so the
          // position comes by a plain load)
          const int kpos = pl.slot_pos[st.slot + r];
#pragma unroll
          for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
            for (int e = 0; e < 4; ++e)
              st.acc[rb][e] = kpos < urow(rb * 16 + 4 * q + e) ? st.acc[rb][e] : -__builtin_inff();
        }
      },
      [&](const StepState &st) __attribute__((always_inline)) {
        float pz[4 * NRB];
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            pz[4 * rb + e] = __builtin_amdgcn_exp2f(__builtin_fmaf(st.acc[rb][e], sl2, nlse[rb][e]));
        colsum = group_sum(tree_sum(pz));
        asm volatile("" : "+v"(colsum));
      },
      [&](const StepState &st, bool tail) __attribute__((always_inline)) {
        if constexpr (RGW == 1) {
          // wave-uniform base (scalar registers) plus the lane's offset
          float *const dst = pout + st.ctx;
          if (rg < a.n_rg && lane < (st.meta & 255)) dst[lane] = colsum;
        } else {
          if (lane < 16) s_cs[ksw][m & 3][lane * RGW + rgw] = colsum;
          if (!tail && m >= 2 && (m - 2) % RGW == rgw) {
            // (written before the barrier this step passed)
            float v[RGW];
            load_sums(m - 2, v);
            store_sums(v, ctx2, nv2);
          }
          ctx3 = ctx2;
          ctx2 = ctx1;
          ctx1 = st.ctx;
          nv3 = nv2;
          nv2 = nv1;
          nv1 = st.meta & 255;
          ++m;
        }
      },
      [&]() __attribute__((always_inline)) {
        if constexpr (RGW > 1) {
          float v[RGW];
          if (m >= 3 && (m - 3) % RGW == rgw) {
            load_sums(m - 3, v);
            store_sums(v, ctx3, nv3);
          }
          if (m >= 2 && (m - 2) % RGW == rgw) {
            load_sums(m - 2, v);
            store_sums(v, ctx2, nv2);
          }
          if (m >= 1 && (m - 1) % RGW == rgw) {
            load_sums(m - 1, v);
            store_sums(v, ctx1, nv1);
          }
          m = 0;
        }
      });
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
    ++d;
    r.len += c;
    r.subs += (c + 15) / 16;
  }
  if (!r.ok) {
    r.subs = 0;
    r.depth = 0;
    if (anc_out) anc_out[0] = j;
    return r;
  }
  r.depth = d - 1;
  // the chain root first, by a second walk up the parent links (no per-lane
  // copy of the chain)
  if (anc_out) {
    int e = d - 1;
    for (int x = j; x >= 0; x = t.parent[x], --e) anc_out[e] = x;
  }
  return r;
}

// One workgroup for the whole call, O(V + n_obs depth): validates the tree,
// walks every observer chain (one thread per observer, root first into anc),
// forms the offsets of the partials, folded sums and sub-page tables as
// prefixes over observers, and lists the blocks that receive credit (proper
// ancestors of some observer; the observers themselves in the self-window
// mode) in ascending id, so that the reduction visits only those.
// fbase / tbase hold the prefixes of the chain lengths and sub-page counts
// until the totals are known.
// IN_LDS (trees of up to kSetupLds nodes) is a template argument, so that the
// tree's arrays are read with LDS or global instructions rather than flat ones.
template <bool IN_LDS>
__device__ __forceinline__ void setup_body(const ScoreArgs &a, int64_t part_cap,
                                                    int64_t *__restrict__ pbase,
                                                    int64_t *__restrict__ fbase,
                                                    int64_t *__restrict__ tbase,
                                                    int32_t *__restrict__ nsp,
                                                    int32_t *__restrict__ ctxlen,
                                                    int32_t *__restrict__ odepth,
                                                    int32_t *__restrict__ anc,
                                                    int32_t *__restrict__ flag,
                                                    int32_t *__restrict__ nctx,
                                                    int32_t *__restrict__ ndep,
                                                    int32_t *__restrict__ cred) {
  __shared__ int64_t sm[17];
  __shared__ int s_err;
  // parent links and block sizes in LDS for trees of up to kSetupLds nodes, so
  // the chain walks do not wait on global memory at every step
  __shared__ int32_t s_par[kSetupLds], s_full[kSetupLds], s_kept[kSetupLds];
  Tree t = a.t;
  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  // each thread's first node and observer, loaded together with the status
  const bool n0 = tid < t.V;
  const int par0 = n0 ? t.parent[tid] : 0, nf0 = n0 ? t.n_full[tid] : 0,
            c0 = n0 ? t.n_kept[tid] : 0;
  const int obs0 = tid < a.n_obs ? a.obs[tid] : 0;
  if (status_failed(a.status)) {
    if (threadIdx.x == 0) cred[0] = 0;
    return;
  }
  if (tid == 0) s_err = 0;
  constexpr bool in_lds = IN_LDS;
  // trees beyond LDS take eight of the thread's nodes at a time: their loads
  // in flight together (the flag stores of one node would otherwise hold up
  // the next node's loads, which share the counter of outstanding memory
  // operations); a tree in LDS takes at most two nodes per thread
  constexpr int kGrp = IN_LDS ? 1 : 8;
  for (int ib = tid; ib < t.V; ib += kGrp * nt) {
    int par[kGrp], nf[kGrp], c[kGrp];
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      const int i = ib + u * nt;
      par[u] = nf[u] = c[u] = 0;
      if (i < t.V) {
        par[u] = i == tid ? par0 : t.parent[i];
        nf[u] = i == tid ? nf0 : t.n_full[i];
        c[u] = i == tid ? c0 : t.n_kept[i];
      }
    }
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      const int i = ib + u * nt;
      if (i < t.V) {
        const bool ok = (i == 0) ? par[u] == -1 : (par[u] >= 0 && par[u] < i);
        if (!ok || c[u] < 0 || c[u] > nf[u]) atomicOr(&s_err, 1);
        if (in_lds) {
          s_par[i] = par[u];
          s_full[i] = nf[u];
          s_kept[i] = c[u];
        }
        flag[i] = 0;
      }
    }
  }
  if (in_lds) {
    t.parent = s_par;
    t.n_full = s_full;
    t.n_kept = s_kept;
  }
  __syncthreads();
  const int slabs = a.S * a.pl.Hkv * a.n_slab;
  int64_t run = 0, frun = 0, trun = 0;
  for (int base = 0; base < a.n_obs; base += nt) {
    const int o = base + tid;
    int64_t len = 0, subs = 0;
    if (o < a.n_obs) {
      const int j = base == 0 ? obs0 : a.obs[o];
      if (j < 0 || j >= t.V) {
        atomicOr(&s_err, 1);
        odepth[o] = -1;
        nsp[2 * o] = nsp[2 * o + 1] = 0;
        ctxlen[o] = 0;
      } else {
        int32_t *ao = anc + (int64_t)o * MAXD;
        const ObsChain r = walk_chain(t, j, ao);
        if (!r.ok) atomicOr(&s_err, 2);
        len = r.len;
        subs = r.subs;
        odepth[o] = r.ok ? r.depth : -1;
        const int own = r.ok ? (t.n_kept[j] + 15) / 16 : 0;
        nsp[2 * o] = (int32_t)subs;
        nsp[2 * o + 1] = r.ok ? (int32_t)(a.self_window ? subs : subs - own) : 0;
        ctxlen[o] = (int32_t)len;
        if (r.ok) {
          // blocks this observer credits, and the depth and context offset
          // of each block of its chain (benign races: every writer of an
          // entry stores the same value)
          int ctx = 0;
          for (int e = 0; e <= r.depth; ++e) {
            const int x = ao[e];
            if (e < r.depth) flag[x] = 1;
            nctx[x] = ctx;
            ndep[x] = e;
            ctx += t.n_kept[x];
          }
          if (a.self_window) flag[j] = 1;
        }
      }
    }
    int64_t tot, ftot, ttot;
    const int64_t ex = block_exclusive_scan<int64_t>(len * slabs, sm, &tot);
    const int64_t fx = block_exclusive_scan<int64_t>(len, sm, &ftot);
    const int64_t tx = block_exclusive_scan<int64_t>(subs, sm, &ttot);
    if (o < a.n_obs) {
      pbase[o] = run + ex;
      fbase[o] = frun + fx;
      tbase[o] = trun + tx;
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
  for (int o = tid; o < a.n_obs; o += nt) {
    fbase[o] += run;
    tbase[o] = tab0 + 4 * tbase[o];
  }
  if (tid == 0) {
    if (s_err & 1) status_error(a.status, ARBOR_EINVAL);
    else if (s_err & 2) status_error(a.status, ARBOR_EUNSUPPORTED);
    else if (!fits) status_error(a.status, ARBOR_EWORKSPACE);
  }
  // the credited blocks in ascending id
  int64_t crun = 0;
  if constexpr (IN_LDS) {
    for (int base = 0; base < t.V; base += nt) {
      const int i = base + tid;
      const int f = i < t.V ? flag[i] : 0;
      int64_t ctot;
      const int64_t cx = block_exclusive_scan<int64_t>(f, sm, &ctot);
      if (f) cred[1 + crun + cx] = i;
      crun += ctot;
    }
  } else {
    // each thread takes a run of consecutive blocks (their flags loaded eight
    // at a time), and one scan places the runs
    const int per = (t.V + nt - 1) / nt;
    const int r0 = min(t.V, tid * per), r1 = min(t.V, r0 + per);
    int64_t mine = 0;
    for (int ib = r0; ib < r1; ib += kGrp) {
      int f[kGrp];
#pragma unroll
      for (int u = 0; u < kGrp; ++u) f[u] = ib + u < r1 ? flag[ib + u] : 0;
#pragma unroll
      for (int u = 0; u < kGrp; ++u) mine += f[u];
    }
    int64_t off = block_exclusive_scan<int64_t>(mine, sm, &crun);
    for (int ib = r0; ib < r1 && mine > 0; ib += kGrp) {
      int f[kGrp];
#pragma unroll
      for (int u = 0; u < kGrp; ++u) f[u] = ib + u < r1 ? flag[ib + u] : 0;
#pragma unroll
      for (int u = 0; u < kGrp; ++u)
        if (f[u]) cred[1 + off++] = ib + u;
    }
  }
  if (tid == 0) cred[0] = (s_err || !fits) ? 0 : (int32_t)crun;
}

template <bool IN_LDS>
__global__ __launch_bounds__(1024) void score_setup(ScoreArgs a, int64_t part_cap,
                                                    int64_t *__restrict__ pbase,
                                                    int64_t *__restrict__ fbase,
                                                    int64_t *__restrict__ tbase,
                                                    int32_t *__restrict__ nsp,
                                                    int32_t *__restrict__ ctxlen,
                                                    int32_t *__restrict__ odepth,
                                                    int32_t *__restrict__ anc,
                                                    int32_t *__restrict__ flag,
                                                    int32_t *__restrict__ nctx,
                                                    int32_t *__restrict__ ndep,
                                                    int32_t *__restrict__ cred) {
  setup_body<IN_LDS>(a, part_cap, pbase, fbase, tbase, nsp, ctxlen, odepth, anc, flag, nctx,
                     ndep, cred);
}

// The sub-page table of observer o at tab, as 16-byte entries (plane row,
// slot, context offset, valid slots | own << 8 | mask flags) that the
// streaming kernel reads into registers; ch holds o's chain (node, depth).
__device__ __forceinline__ void table_body(const ScoreArgs &a, ChainLds &ch, int j, int4 *tab) {
  const Tree &t = a.t;
  const int tid = threadIdx.x;
  const int depth = ch.depth;
  if (tid <= depth) {
    const int x = ch.node[tid];
    ch.c[tid] = t.n_kept[x];
    ch.po[tid] = t.page_off[x];
  }
  __syncthreads();
  if (tid == 0) {
    int ctx = 0, sp = 0;
    for (int e = 0; e <= depth; ++e) {
      const int c = ch.c[e];
      ch.ctx[e] = ctx;
      ch.sp_off[e] = sp;
      ctx += c;
      sp += (c + 15) / 16;
    }
    ch.sp_off[depth + 1] = sp;
  }
  __syncthreads();
  const int n = ch.sp_off[depth + 1];
  fill_table(t, a.pl, ch, n);
  // the window rows see own positions up to u >= u_min: an own sub-page whose
  // last position is above u_min needs per-key masking in pass 0; in the
  // self-window mode, one whose last position reaches u_min needs it in pass 1
  const int u_min = t.n_full[j] - min(a.W, t.n_full[j]);
  for (int sp = tid; sp < n; sp += blockDim.x) {
    const SubPage e = sub_page(t, a.pl, ch, sp);
    const bool own = e.d == depth;
    const int last = own ? a.pl.slot_pos[e.slot + e.nvalid - 1] : 0;
    const bool m0 = e.nvalid < 16 || (own && last > u_min);
    const bool m1 = a.self_window && own && last >= u_min;
    tab[sp] = make_int4(e.row, e.slot, e.ctx,
                        e.nvalid | (own ? 1 << 8 : 0) | (m0 ? kMask0 : 0) | (m1 ? kMask1 : 0));
  }
}

// One workgroup per observer: its chain (root first, from the setup's walk)
// and its sub-page table.
__global__ __launch_bounds__(256) void score_tables(ScoreArgs a) {
  __shared__ ChainLds ch;
  const int o = blockIdx.x;
  const int tid = threadIdx.x;
  // (loaded together with the status word)
  const int j = a.obs[o];
  const int depth = a.odepth[o];
  if (status_failed(a.status)) return;   // also set by the setup on any error
  if (tid == 0) ch.depth = depth;
  if (tid <= depth) ch.node[tid] = a.anc[(int64_t)o * MAXD + tid];
  __syncthreads();
  table_body(a, ch, j, reinterpret_cast<int4 *>(a.part + a.tbase[o]));
}

// Setup and tables in one launch (up to kPrepObs observers): workgroup 0 runs
// the setup; workgroup 1 + o builds observer o's table without waiting for
// it.  It walks every observer's chain itself (one thread per observer, the
// setup's checks) for the sums that place the tables after the partials and
// folded sums, and the prefix of the sub-page counts that places o's table:
// the same integers the setup computes, so the offsets agree.  A malformed
// chain or a workspace too small leaves o's table unwritten (the setup
// reports the error, and no later kernel runs).
constexpr int kPrepObs = 512;
template <bool IN_LDS>
__global__ __launch_bounds__(1024) void score_prep(ScoreArgs a, int64_t part_cap,
                                                   int64_t *__restrict__ pbase,
                                                   int64_t *__restrict__ fbase,
                                                   int64_t *__restrict__ tbase,
                                                   int32_t *__restrict__ nsp,
                                                   int32_t *__restrict__ ctxlen,
                                                   int32_t *__restrict__ odepth,
                                                   int32_t *__restrict__ anc,
                                                   int32_t *__restrict__ flag,
                                                   int32_t *__restrict__ nctx,
                                                   int32_t *__restrict__ ndep,
                                                   int32_t *__restrict__ cred) {
  if (blockIdx.x == 0) {
    setup_body<IN_LDS>(a, part_cap, pbase, fbase, tbase, nsp, ctxlen, odepth, anc, flag, nctx,
                       ndep, cred);
    return;
  }
  __shared__ ChainLds ch;
  __shared__ int64_t sm[17];
  __shared__ int64_t s_pre;
  __shared__ int s_bad;
  const Tree &t = a.t;
  const int o = (int)blockIdx.x - 1;
  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  const int j = a.obs[o];
  if (status_failed(a.status)) return;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  const int slabs = a.S * a.pl.Hkv * a.n_slab;
  int64_t run = 0, frun = 0, trun = 0;
  for (int base = 0; base < a.n_obs; base += nt) {
    const int oo = base + tid;
    int64_t len = 0, subs = 0;
    if (oo < a.n_obs) {
      const int jj = a.obs[oo];
      if (jj < 0 || jj >= t.V) {
        s_bad = 1;
      } else {
        const ObsChain r = walk_chain(t, jj, oo == o ? ch.node : nullptr);
        if (!r.ok) s_bad = 1;
        len = r.len;
        subs = r.subs;
        if (oo == o) ch.depth = r.depth;
      }
    }
    int64_t tot, ftot, ttot;
    block_exclusive_scan<int64_t>(len * slabs, sm, &tot);
    block_exclusive_scan<int64_t>(len, sm, &ftot);
    const int64_t tx = block_exclusive_scan<int64_t>(subs, sm, &ttot);
    if (oo == o) s_pre = trun + tx;
    run += tot;
    frun += ftot;
    trun += ttot;
  }
  __syncthreads();
  const int64_t tab0 = (run + frun + 3) & ~(int64_t)3;
  if (s_bad || tab0 + 4 * trun > part_cap) return;
  table_body(a, ch, j, reinterpret_cast<int4 *>(a.part + tab0 + 4 * s_pre));
}

// Fold the (slice layer, kv head, workgroup) slabs of every observer: one
// column sum per (observer, credited context key), summed in slab order.
__global__ __launch_bounds__(256) void score_fold(ScoreArgs a, const int64_t *__restrict__ fbase) {
  const int o = blockIdx.x;
  // (loaded together with the status word)
  const int len = a.ctxlen[o];
  const int jo = a.obs[o];
  const int64_t pb = a.pbase[o], fb = fbase[o];
  if (status_failed(a.status)) return;
  const int own_c = a.t.n_kept[jo];
  const int credited = a.self_window ? len : len - own_c;
  const int nslab = a.S * a.pl.Hkv * a.n_slab;
  const float *src = a.part + pb;
  float *dst = a.part + fb;
  for (int x = blockIdx.y * blockDim.x + threadIdx.x; x < credited; x += gridDim.y * blockDim.x) {
    // eight loads in flight, added in slab order
    float acc = 0.f;
    int sl = 0;
    for (; sl + 8 <= nslab; sl += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = src[(int64_t)(sl + u) * len + x];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += v[u];
    }
    for (; sl < nslab; ++sl) acc += src[(int64_t)sl * len + x];
    dst[x] = acc;
  }
}

// a_i and s_i of block i from its A (one wave).
__device__ void block_final(const Tree &t, int i, const float *__restrict__ A,
                            const int64_t *__restrict__ rows_seen, const float *__restrict__ v_in,
                            const float *__restrict__ u_in, float th0, float th1, float th2,
                            float *__restrict__ a_out, float *__restrict__ s_out) {
  const int lane = lane_id();
  // the block's fields and signals in one round trip, then its A eight loads
  // at a time (added in the same order as one at a time)
  const int64_t tb = t.tok_off[i];
  const int n = t.n_full[i];
  const int64_t rs = rows_seen[i];
  const float vi = v_in[i], ui = u_in[i];
  double sum = 0.0;
  int p = lane;
  for (; p + 7 * kWave < n; p += 8 * kWave) {
    float x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = A[tb + p + u * kWave];
#pragma unroll
    for (int u = 0; u < 8; ++u) sum += (double)x[u];
  }
  for (; p < n; p += kWave) sum += (double)A[tb + p];
  sum = wave_sum<double>(sum);
  if (lane == 0) {
    const double av = rs > 0 ? sum / (double)rs : 0.0;
    const double x = (double)th0 * (double)vi + (double)th1 * (double)ui + (double)th2 * av;
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
// rows_seen_i grows.  Workgroup x takes the x-th credited block of the setup's
// list.  The four waves of a workgroup split the observers of a 64-slot chunk
// and are combined in wave order.
__global__ __launch_bounds__(256) void score_reduce(ScoreArgs a, const int64_t *__restrict__ fbase,
                                                    const int32_t *__restrict__ cred,
                                                    float *__restrict__ A,
                                                    int64_t *__restrict__ rows_seen) {
  __shared__ int64_t hbase[256];
  __shared__ int s_wcnt[4];
  __shared__ double s_acc[4][64];
  // (loaded together with the status word; the list entry past its end is
  // allocated, and unused then; so are the first 256 observers' depths and
  // window sizes, which do not depend on the block)
  const int ncred = cred[0];
  const int i = cred[1 + blockIdx.x];
  const bool o0 = (int)threadIdx.x < a.n_obs;
  const int od0 = o0 ? a.odepth[threadIdx.x] : -1;
  const int64_t fb0 = o0 ? fbase[threadIdx.x] : 0;
  const int wn0 = o0 ? min(a.W, a.t.n_full[a.obs[threadIdx.x]]) : 0;
  if (status_failed(a.status)) return;
  if ((int)blockIdx.x >= ncred) return;
  const Tree &t = a.t;
  const Pool &pl = a.pl;
  const int c = t.n_kept[i];
  // chunk splits past the block's last chunk have nothing to add (split 0
  // still counts the rows)
  if (blockIdx.y > 0 && (int)blockIdx.y * 64 >= c) return;
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const float *fold = a.part;
  // (every credited block lies on an observer's chain, whose depth and
  // context offset the setup recorded)
  const int di = a.ndep[i], ctxoff = a.nctx[i];
  const int64_t tb = t.tok_off[i];
  const int64_t po = t.page_off[i];
  int64_t rows_add = 0;
  const int nchunk = (c + 63) / 64;
  for (int ob = 0; ob < a.n_obs; ob += 256) {
    const int o = ob + threadIdx.x;
    bool hit = false;
    if (o < a.n_obs) {
      const int od = ob == 0 ? od0 : a.odepth[o];
      hit = (od > di && a.anc[(int64_t)o * MAXD + di] == i) || (a.self_window && a.obs[o] == i);
    }
    const uint64_t bm = ballot(hit);
    if (lane == 0) s_wcnt[wave] = popc(bm);
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wave; ++w) before += s_wcnt[w];
    const int nh = s_wcnt[0] + s_wcnt[1] + s_wcnt[2] + s_wcnt[3];
    if (hit) {
      hbase[before + rank_below(bm, lane)] = (ob == 0 ? fb0 : fbase[o]) + ctxoff;
      if (blockIdx.y == 0)
        rows_add += (int64_t)a.S * pl.Hkv * pl.G *
                    (ob == 0 ? wn0 : min(a.W, t.n_full[a.obs[o]]));
    }
    __syncthreads();
    if (nh > 0) {
      for (int chk = blockIdx.y; chk < nchunk; chk += gridDim.y) {
        const int s = chk * 64 + lane;
        double acc = 0.0;
        if (s < c) {
          // (sixteen, then four loads in flight, added one by one in order)
          int h = wave;
          for (; h + 60 < nh; h += 64) {
            float f[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) f[u] = fold[hbase[h + 4 * u] + s];
#pragma unroll
            for (int u = 0; u < 16; ++u) acc += (double)f[u];
          }
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

template <class T, int D, int NRB>
void launch_attn_rg(int RGW, dim3 grid, hipStream_t stream, const ScoreArgs &a) {
  switch (RGW) {
    case 1: hipLaunchKernelGGL((score_attn<T, D, NRB, 1>), grid, dim3(256), 0, stream, a); break;
    case 2: hipLaunchKernelGGL((score_attn<T, D, NRB, 2>), grid, dim3(256), 0, stream, a); break;
    default: hipLaunchKernelGGL((score_attn<T, D, NRB, 4>), grid, dim3(256), 0, stream, a); break;
  }
}

// Fewer than the full 16 NRB rows fit in one row group: one group, no sharing.
template <class T, int D>
void launch_attn_nb(int NRB, int RGW, dim3 grid, hipStream_t stream, const ScoreArgs &a) {
  constexpr int cap = sizeof(T) == 2 ? 4 : 2;
  if (NRB < cap) {
    if (NRB == 1) hipLaunchKernelGGL((score_attn<T, D, 1, 1>), grid, dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((score_attn<T, D, 2, 1>), grid, dim3(256), 0, stream, a);
    return;
  }
  launch_attn_rg<T, D, cap>(RGW, grid, stream, a);
}

void launch_attn(int dtype, int D, int NRB, int RGW, dim3 grid, hipStream_t stream,
                 const ScoreArgs &a) {
  if (dtype == ARBOR_BF16) {
    if (D == 128) launch_attn_nb<__bf16, 128>(NRB, RGW, grid, stream, a);
    else launch_attn_nb<__bf16, 64>(NRB, RGW, grid, stream, a);
  } else {
    if (D == 128) launch_attn_nb<float, 128>(NRB, RGW, grid, stream, a);
    else launch_attn_nb<float, 64>(NRB, RGW, grid, stream, a);
  }
}

// 16-row blocks of a row group: enough for all the rows up to 64 (32 for fp32,
// whose operands take four times the registers), a power of two.  A wave
// holds the Q of its group's rows; 64 rows (bf16) keep three waves per SIMD.
// Row groups per workgroup: they share its key tiles and one partial slab (a
// power of two, as in the kernel's template).
int rg_per_wg(int n_rg) { return n_rg >= 4 ? 4 : (n_rg >= 2 ? 2 : 1); }

int row_blocks(int rows_total, int dtype) {
  const int cap = dtype == ARBOR_BF16 ? 4 : 2;
  int nrb = 1;
  while (nrb < cap && 16 * nrb < rows_total) nrb *= 2;
  return nrb;
}

}  // namespace

size_t score_workspace(const arbor_geom_t *g, const arbor_sizes_t *sz) {
  const int rows_total = g->q_per_kv * sz->window;
  const int NRB = row_blocks(rows_total, g->dtype);
  const int n_rg = (rows_total + 16 * NRB - 1) / (16 * NRB);
  const int RGW = rg_per_wg(n_rg);
  const size_t nobs = (size_t)(sz->max_observers > 0 ? sz->max_observers : 0);
  const size_t slabs = (size_t)sz->n_slice * g->num_kv_heads * ((n_rg + RGW - 1) / RGW);
  size_t b = 0;
  // offsets, counts, chains, credited-block flags and list (each carve
  // rounds up to 256 B)
  b += nobs * (8 * 3 + 4 * 4) + nobs * MAXD * 4 + (size_t)sz->num_nodes * 16 + 14 * 256;
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
  const int NRB = row_blocks(rows_total, geom->dtype);
  a.n_rg = (rows_total + 16 * NRB - 1) / (16 * NRB);
  const int RGW = rg_per_wg(a.n_rg);
  a.n_slab = (a.n_rg + RGW - 1) / RGW;
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
  int32_t *flag = cv.take<int32_t>((size_t)t.V);
  int32_t *nctx = cv.take<int32_t>((size_t)t.V);
  int32_t *ndep = cv.take<int32_t>((size_t)t.V);
  int32_t *cred = cv.take<int32_t>((size_t)t.V + 1);
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
  a.nctx = nctx;
  a.ndep = ndep;
  const FinalArgs fa{v_in, u_in, params->theta[0], params->theta[1], params->theta[2], a_out, s_out};
  if (n_obs > 0) {
    // one thread per node and per observer, in one workgroup (a small tree
    // takes a smaller one, whose barriers are cheaper); with few observers
    // the tables are built in the same launch
    const int64_t need = std::max<int64_t>(t.V, n_obs);
    const int st = (int)std::min<int64_t>(1024, (need + kWave - 1) / kWave * kWave);
    if (n_obs <= kPrepObs) {
      const dim3 grid((unsigned)n_obs + 1), blk((unsigned)std::max(st, 256));
      if (t.V <= kSetupLds)
        hipLaunchKernelGGL(score_prep<true>, grid, blk, 0, stream, a, part_cap, pbase, fbase,
                           tbase, nsp, ctxlen, odepth, anc, flag, nctx, ndep, cred);
      else
        hipLaunchKernelGGL(score_prep<false>, grid, blk, 0, stream, a, part_cap, pbase, fbase,
                           tbase, nsp, ctxlen, odepth, anc, flag, nctx, ndep, cred);
    } else {
      if (t.V <= kSetupLds)
        hipLaunchKernelGGL(score_setup<true>, dim3(1), dim3(st), 0, stream, a, part_cap, pbase,
                           fbase, tbase, nsp, ctxlen, odepth, anc, flag, nctx, ndep, cred);
      else
        hipLaunchKernelGGL(score_setup<false>, dim3(1), dim3(st), 0, stream, a, part_cap, pbase,
                           fbase, tbase, nsp, ctxlen, odepth, anc, flag, nctx, ndep, cred);
      hipLaunchKernelGGL(score_tables, dim3(n_obs), dim3(256), 0, stream, a);
    }
    const int n_planes = n_slice * pl.Hkv * a.n_slab;
    const dim3 grid((unsigned)(((n_planes + kXcds - 1) / kXcds) * n_obs * kXcds));
    timing_begin(geom, ARBOR_KERNEL_SCORE_ATTN, stream);
    launch_attn(geom->dtype, geom->head_dim, NRB, RGW, grid, stream, a);
    timing_end(geom, ARBOR_KERNEL_SCORE_ATTN, stream);
    hipLaunchKernelGGL(score_fold, dim3(n_obs, 8), dim3(256), 0, stream, a, fbase);
    // at most V credited blocks, and at most MAXD per observer
    const int64_t max_cred = std::min<int64_t>(t.V, (int64_t)n_obs * MAXD);
    // 64-slot chunk splits per block: 64 (one chunk each up to 4,096 kept
    // slots) while the grid stays small, else 16
    const unsigned ysplit = max_cred <= 512 ? 64u : 16u;
    hipLaunchKernelGGL(score_reduce, dim3((unsigned)max_cred, ysplit), dim3(256), 0, stream, a,
                       fbase, cred, A, rows_seen);
  }
  hipLaunchKernelGGL(score_final, dim3((t.V + 3) / 4), dim3(256), 0, stream, t, A, rows_seen, fa,
                     status);
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
