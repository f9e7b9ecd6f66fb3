// Internal definitions shared by the HIP translation units of libarbor.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/arbor.h"

namespace arbor {

constexpr int kWave = 64;

// Kernel-side copy of the tree description.
struct Tree {
  int32_t V;
  int64_t N;
  const int32_t *parent;
  const int32_t *n_full;
  const int64_t *tok_off;
  const int64_t *page_off;
  int32_t *n_kept;
  int32_t *page_table;
};

// Kernel-side copy of the pool description.
struct Pool {
  void *k;
  void *v;
  int32_t *slot_pos;
  int32_t *free_stack;
  int32_t *free_top;
  int64_t num_pages;
  int32_t L, Hkv, G, D, P;
  int32_t esize;  // bytes per element of K/V (2 = bf16, 4 = f32)
};

inline Tree make_tree(const arbor_tree_t *t) {
  return Tree{t->num_nodes, t->num_tokens, t->parent, t->n_full, t->tok_off,
              t->page_off, t->n_kept, t->page_table};
}

inline Pool make_pool(const arbor_geom_t *g, const arbor_pool_t *p) {
  return Pool{p->k, p->v, p->slot_pos, p->free_stack, p->free_top, g->num_pages,
              g->num_layers, g->num_kv_heads, g->q_per_kv, g->head_dim, g->page_size,
              g->dtype == ARBOR_BF16 ? 2 : 4};
}

// Byte offset of row `r` of page `page` in plane (layer l, kv head g).
__device__ __forceinline__ int64_t row_byte_offset(const Pool &pl, int l, int64_t page, int g,
                                                   int r) {
  return ((((int64_t)l * pl.num_pages + page) * pl.Hkv + g) * pl.P + r) * (int64_t)pl.D *
         pl.esize;
}

// ---- sticky device status ------------------------------------------------
// 16-byte store with the non-temporal hint: rows a kernel moves are not read
// again soon, and keeping them out of the caches spares the next kernel the
// write-back of their dirty lines.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void store16_nt(void *dst, uint4 v) {
  const u32x4 w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, static_cast<u32x4 *>(dst));
}

__device__ __forceinline__ bool status_failed(const int32_t *st) {
  // (the status word is device-accessible global memory: a global load, not
  // a flat one)
  return *(const __attribute__((address_space(1))) volatile int32_t *)st < 0;
}
__device__ __forceinline__ void status_error(int32_t *st, int32_t code) { atomicMin(st, code); }
__device__ __forceinline__ void status_warn(int32_t *st, int32_t code) { atomicCAS(st, 0, code); }

// ---- wavefront helpers (wave64) -------------------------------------------
__device__ __forceinline__ int lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0));
}
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }
__device__ __forceinline__ int rank_below(uint64_t m, int lane) {
  return __popcll(m & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
}

// fp32 value -> unsigned key whose order is the numeric order; -0 == +0.
__device__ __forceinline__ uint32_t ordered_key(float x) {
  uint32_t b = __float_as_uint(x);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// ---- cross-lane steps on the VALU ----------------------------------------
// DPP moves within 16-lane rows and lane swaps across rows: no round trip
// through the LDS permute unit.  Values of 4 or 8 bytes; 8-byte values move
// as two 32-bit halves.
namespace dpp {
constexpr int kQuadXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141;  // lane i <- 7 - i within each 8
constexpr int kRowMirror = 0x140;      // lane i <- 15 - i within each row
constexpr int kRowShr = 0x110;         // + n: lane i <- i - n within the row
constexpr int kRowBcast15 = 0x142;     // lane 15 of each row -> the next row
constexpr int kRowBcast31 = 0x143;     // lane 31 -> rows 2 and 3
}  // namespace dpp

template <class T>
__device__ __forceinline__ uint64_t bits64(T v) {
  if constexpr (sizeof(T) == 4)
    return (uint64_t)__builtin_bit_cast(uint32_t, v);
  else
    return __builtin_bit_cast(uint64_t, v);
}
template <class T>
__device__ __forceinline__ T from_bits64(uint64_t b) {
  if constexpr (sizeof(T) == 4)
    return __builtin_bit_cast(T, (uint32_t)b);
  else
    return __builtin_bit_cast(T, b);
}

// v moved by a DPP control; lanes without a source (or outside row_mask) get 0
template <int CTRL, int ROW_MASK = 0xF, class T>
__device__ __forceinline__ T dpp_move(T v) {
  static_assert(sizeof(T) == 4 || sizeof(T) == 8, "4- or 8-byte lanes");
  const uint64_t b = bits64(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, ROW_MASK,
                                                            0xF, true);
  if constexpr (sizeof(T) == 4) {
    return from_bits64<T>(lo);
  } else {
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), CTRL,
                                                              ROW_MASK, 0xF, true);
    return from_bits64<T>((uint64_t)lo | ((uint64_t)hi << 32));
  }
}

// the pair (own value, value of lane ^ 16) or (.., lane ^ 32), in either order
template <bool X32, class T>
__device__ __forceinline__ void row_swap(T v, T &a, T &b) {
  const uint64_t u = bits64(v);
  const uint32_t lo = (uint32_t)u;
  auto rl = X32 ? __builtin_amdgcn_permlane32_swap(lo, lo, false, false)
                : __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
  if constexpr (sizeof(T) == 4) {
    a = from_bits64<T>(rl[0]);
    b = from_bits64<T>(rl[1]);
  } else {
    const uint32_t hi = (uint32_t)(u >> 32);
    auto rh = X32 ? __builtin_amdgcn_permlane32_swap(hi, hi, false, false)
                  : __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    a = from_bits64<T>((uint64_t)rl[0] | ((uint64_t)rh[0] << 32));
    b = from_bits64<T>((uint64_t)rl[1] | ((uint64_t)rh[1] << 32));
  }
}

// op over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the same position in each
// 16-lane row), result in every lane
template <class T, class Op>
__device__ __forceinline__ T across_rows(T v, Op op) {
  T a, b;
  row_swap<false>(v, a, b);
  v = op(a, b);
  row_swap<true>(v, a, b);
  return op(a, b);
}

// op over all 64 lanes (op commutative and associative), result in every lane
template <class T, class Op>
__device__ __forceinline__ T wave_allreduce(T v, Op op) {
  v = op(v, dpp_move<dpp::kQuadXor1>(v));
  v = op(v, dpp_move<dpp::kQuadXor2>(v));
  v = op(v, dpp_move<dpp::kRowHalfMirror>(v));
  v = op(v, dpp_move<dpp::kRowMirror>(v));
  T a, b;
  row_swap<false>(v, a, b);
  v = op(a, b);
  row_swap<true>(v, a, b);
  return op(a, b);
}

template <class T>
__device__ __forceinline__ T wave_sum(T v) {
  return wave_allreduce(v, [](T x, T y) { return x + y; });
}

// value of lane `l` (wave-uniform l) in every lane
template <class T>
__device__ __forceinline__ T lane_value(T v, int l) {
  const uint64_t u = bits64(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
  if constexpr (sizeof(T) == 4) {
    return from_bits64<T>(lo);
  } else {
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
    return from_bits64<T>((uint64_t)lo | ((uint64_t)hi << 32));
  }
}

// ---- block-wide scans (blockDim.x a multiple of 64, at most 1024) ----------
// Inclusive prefix sum over the wave in lane order: shifts by 1, 2, 4, 8
// within each row, then the row totals carried by two row broadcasts.
template <class T>
__device__ __forceinline__ T wave_inclusive_scan(T v) {
  v = v + dpp_move<dpp::kRowShr + 1>(v);
  v = v + dpp_move<dpp::kRowShr + 2>(v);
  v = v + dpp_move<dpp::kRowShr + 4>(v);
  v = v + dpp_move<dpp::kRowShr + 8>(v);
  v = v + dpp_move<dpp::kRowBcast15, 0xA>(v);
  v = v + dpp_move<dpp::kRowBcast31, 0xC>(v);
  return v;
}

// Exclusive prefix of v over the block in thread order; *total gets the sum.
// `smem` holds at least 17 elements.  Contains __syncthreads.  Every wave
// scans the (at most 16) wave totals itself, so no thread walks them serially.
template <class T>
__device__ T block_exclusive_scan(T v, T *smem, T *total) {
  const int lane = lane_id();
  const int w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const T inc = wave_inclusive_scan(v);
  if (lane == kWave - 1) smem[w] = inc;
  __syncthreads();
  const T t = lane < nw ? smem[lane] : T(0);
  const T tinc = wave_inclusive_scan(t);
  const T base = lane_value(tinc, w) - lane_value(t, w);
  *total = lane_value(tinc, nw - 1);
  __syncthreads();
  return base + inc - v;
}

// N exclusive scans over the block in one exchange (two barriers in all);
// smem holds N * 16 values.  Threads from `live` on contribute zeros, so
// their waves skip the wave-level scans.
template <int N>
__device__ void block_exclusive_scan_n(const int64_t (&v)[N], int64_t (&ex)[N],
                                       int64_t (&total)[N], int64_t *smem,
                                       int live = 1 << 30) {
  const int lane = lane_id();
  const int w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const bool scan = w * kWave < live;
  int64_t inc[N];
#pragma unroll
  for (int k = 0; k < N; ++k) {
    inc[k] = scan ? wave_inclusive_scan(v[k]) : (int64_t)0;
    if (lane == kWave - 1) smem[k * 16 + w] = inc[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < N; ++k) {
    const int64_t t = lane < nw ? smem[k * 16 + lane] : 0;
    const int64_t tinc = wave_inclusive_scan(t);
    ex[k] = lane_value(tinc, w) - lane_value(t, w) + inc[k] - v[k];
    total[k] = lane_value(tinc, nw - 1);
  }
  __syncthreads();
}

template <class T>
__device__ T block_sum(T v, T *smem) {
  T tot;
  block_exclusive_scan(v, smem, &tot);
  return tot;
}

// ---- host-side workspace carving -------------------------------------------
struct Carve {
  char *base;
  size_t cap;
  size_t off = 0;
  bool ok = true;
  Carve(void *b, size_t c) : base(static_cast<char *>(b)), cap(c) {}
  template <class T>
  T *take(size_t n) {
    size_t o = (off + 255) & ~size_t(255);
    size_t bytes = n * sizeof(T);
    if (base == nullptr || o + bytes > cap) {
      ok = false;
      off = o + bytes;
      return nullptr;
    }
    off = o + bytes;
    return reinterpret_cast<T *>(base + o);
  }
  size_t remaining() const { return off >= cap ? 0 : cap - ((off + 255) & ~size_t(255)); }
  char *rest() { return base + ((off + 255) & ~size_t(255)); }
};

static inline int hip_ok(hipError_t e) { return e == hipSuccess ? ARBOR_OK : ARBOR_EHIP; }

// The call's own timing request (arbor_geom_t.timing): events recorded on the
// launch stream around the launches of one named kernel.
inline void timing_begin(const arbor_geom_t *g, int kernel, hipStream_t s) {
  const arbor_timing_t *tm = g->timing;
  if (tm && tm->kernel == kernel && tm->start) (void)hipEventRecord(tm->start, s);
}
inline void timing_end(const arbor_geom_t *g, int kernel, hipStream_t s) {
  const arbor_timing_t *tm = g->timing;
  if (tm && tm->kernel == kernel && tm->stop) (void)hipEventRecord(tm->stop, s);
}

}  // namespace arbor
