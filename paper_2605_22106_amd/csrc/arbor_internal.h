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
  return *reinterpret_cast<const volatile int32_t *>(st) < 0;
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

// ---- block-wide scans (blockDim.x a multiple of 64, at most 1024) ----------
template <class T>
__device__ __forceinline__ T wave_inclusive_scan(T v) {
  const int lane = lane_id();
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    T o = __shfl_up(v, d, kWave);
    if (lane >= d) v += o;
  }
  return v;
}

template <class T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int d = kWave / 2; d > 0; d >>= 1) v += __shfl_xor(v, d, kWave);
  return v;
}

// Exclusive prefix of v over the block in thread order; *total gets the sum.
// `smem` holds at least 17 elements.  Contains __syncthreads.
template <class T>
__device__ T block_exclusive_scan(T v, T *smem, T *total) {
  const int lane = lane_id();
  const int w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  T inc = wave_inclusive_scan(v);
  if (lane == kWave - 1) smem[w] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    T run = 0;
    for (int j = 0; j < nw; ++j) {
      T x = smem[j];
      smem[j] = run;
      run += x;
    }
    smem[16] = run;
  }
  __syncthreads();
  T ex = smem[w] + inc - v;
  *total = smem[16];
  __syncthreads();
  return ex;
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

}  // namespace arbor
