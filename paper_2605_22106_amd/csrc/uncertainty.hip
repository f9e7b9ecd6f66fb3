// arbor_uncertainty: normalised next-token entropy at block boundaries
// (Sec. 4 MSVE, Eq. 1): u = 1 - H / ln|V| of the softmax of one logit row,
// H over the whole vocabulary, or over its K largest probabilities plus one
// "other" outcome carrying the rest of the mass.
//
// Everything is kept in log2 units: with x = z log2(e), m = max x and
//   S = sum 2^(x - m),   T = sum (x - m) 2^(x - m),
// the entropy is H = ln 2 (log2 S - T / S).  A thread keeps (m, S, T) of its
// elements, rescaled when its max grows; threads are merged by a fixed
// butterfly and the waves in order.
//   full vocabulary: each row is split into chunks of whole 16-byte vectors,
//     one 256-thread workgroup per (row, chunk) streams its chunk into a
//     partial (m, S, T); a second kernel merges a row's partials in chunk
//     order (enough workgroups to cover the chip even for few rows);
//   top-K, K <= KMAX: the same chunks also keep their own K largest values
//     (the values above a bound taken from the threads' maxima, then a radix
//     select over their order-preserving 32-bit keys, 8 bits per LDS
//     histogram pass); the row's top K lie among those candidates, so a merge
//     workgroup per row selects the K-th largest among them and sums the top
//     K against the merged (m, S);
//   top-K, larger K: one workgroup per row finds the K-th largest logit by a
//     radix select over the whole row (11 + 11 + 10 bits), then sums the top
//     and the rest in one more pass.
// Fixed reduction orders throughout: bitwise reproducible.
#include "arbor_internal.h"

namespace arbor {

namespace {

constexpr int UT = 1024;                     // threads per row
constexpr int UW = UT / kWave;               // waves per row
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct Ent {
  float m, s, t;   // max (log2 units), sum of 2^(x-m), sum of (x-m) 2^(x-m)
};

__device__ __forceinline__ Ent ent_merge(Ent a, Ent b) {
  const float m = fmaxf(a.m, b.m);
  if (m == -__builtin_inff()) return Ent{m, 0.f, 0.f};
  Ent r{m, 0.f, 0.f};
  if (a.m > -__builtin_inff()) {
    const float d = a.m - m, f = __builtin_amdgcn_exp2f(d);
    r.s += a.s * f;
    r.t += (a.t + d * a.s) * f;
  }
  if (b.m > -__builtin_inff()) {
    const float d = b.m - m, f = __builtin_amdgcn_exp2f(d);
    r.s += b.s * f;
    r.t += (b.t + d * b.s) * f;
  }
  return r;
}

// elements of one 16-byte load, widened to float
template <class T>
struct Vec;
template <>
struct Vec<__bf16> {
  static constexpr int N = 8;
  static __device__ __forceinline__ void get(const uint4 &u, float (&x)[8]) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};
template <>
struct Vec<float> {
  static constexpr int N = 4;
  static __device__ __forceinline__ void get(const uint4 &u, float (&x)[4]) {
    x[0] = __uint_as_float(u.x);
    x[1] = __uint_as_float(u.y);
    x[2] = __uint_as_float(u.z);
    x[3] = __uint_as_float(u.w);
  }
};

// inverse of ordered_key
__device__ __forceinline__ float key_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// fixed-order block sum of a float (every thread gets the result)
__device__ float block_sum_f(float v, float *sm) {
  v = wave_sum(v);
  if (lane_id() == 0) sm[threadIdx.x >> 6] = v;
  __syncthreads();
  float r = 0.f;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) r += sm[w];
  __syncthreads();
  return r;
}

// f(vector) for every vector in [v0, v1) of a row, this thread's share
// (v0 + tid, v0 + tid + UT, ...).  Eight loads are issued before any is used;
// past the end they re-read the last vector (clamped, so every load is
// unconditional) and are not used.
template <int NT, class F>
__device__ __forceinline__ void for_vecs(const uint4 *row, int64_t v0, int64_t v1, F &&f) {
  constexpr int U = 8;
  if (v1 <= v0) return;
  for (int64_t i = v0 + threadIdx.x; i < v1; i += U * NT) {
    uint4 u[U];
#pragma unroll
    for (int j = 0; j < U; ++j) u[j] = row[min(i + (int64_t)j * NT, v1 - 1)];
#pragma unroll
    for (int j = 0; j < U; ++j)
      if (i + (int64_t)j * NT < v1) f(u[j]);
  }
}

// (m, S, T) of vectors [v0, v1) of a row over the whole workgroup (every
// thread gets the result); *bad_flag is set (LDS) if any value is NaN or
// infinite.
template <class T, int NT, class Each>
__device__ Ent block_stats(const uint4 *row, int64_t v0, int64_t v1, bool &bad, Ent *s_ent,
                           int *bad_flag, Each &&each) {
  constexpr int N = Vec<T>::N;
  const int tid = threadIdx.x;
  Ent e{-__builtin_inff(), 0.f, 0.f};
  auto add = [&](const uint4 &u) __attribute__((always_inline)) {
    float x[N];
    Vec<T>::get(u, x);
    float vm = -__builtin_inff();
#pragma unroll
    for (int k = 0; k < N; ++k) {
      bad |= !(__builtin_fabsf(x[k]) <= 3.4e38f);   // NaN or infinite
      each(x[k]);
      x[k] *= kLog2e;
      vm = fmaxf(vm, x[k]);
    }
    if (vm > e.m) {
      if (e.m > -__builtin_inff()) {
        const float d = e.m - vm, f = __builtin_amdgcn_exp2f(d);
        e.t = (e.t + d * e.s) * f;
        e.s *= f;
      }
      e.m = vm;
    }
#pragma unroll
    for (int k = 0; k < N; ++k) {
      const float d = x[k] - e.m;
      const float p = __builtin_amdgcn_exp2f(d);
      e.s += p;
      e.t = __builtin_fmaf(d, p, e.t);
    }
  };
  for_vecs<NT>(row, v0, v1, add);
  if (bad) atomicOr(bad_flag, 1);
  // butterfly within the wave, then the waves in order
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    Ent o{__shfl_xor(e.m, off, kWave), __shfl_xor(e.s, off, kWave), __shfl_xor(e.t, off, kWave)};
    e = ent_merge(e, o);
  }
  if (lane_id() == 0) s_ent[tid >> 6] = e;
  __syncthreads();
  Ent all = s_ent[0];
#pragma unroll
  for (int w = 1; w < NT / kWave; ++w) all = ent_merge(all, s_ent[w]);
  return all;
}

// Top-K variant: one workgroup per row.
template <class T>
__global__ __launch_bounds__(UT) void uncert_topk(const T *__restrict__ logits, int64_t vocab,
                                                    int top_k, const int32_t *__restrict__ dst,
                                                    float *__restrict__ u_out, int n_out,
                                                    int32_t *status) {
  typedef Vec<T> VV;
  constexpr int N = VV::N;
  __shared__ Ent s_ent[UW];
  __shared__ float s_f[UW];
  __shared__ unsigned hist[2048];
  __shared__ int s_bin, s_above, s_bad;
  __shared__ int64_t s_scan[17];
  if (status_failed(status)) return;
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const uint4 *row = reinterpret_cast<const uint4 *>(logits + (int64_t)r * vocab);
  const int64_t nvec = vocab / N;
  if (tid == 0) s_bad = 0;
  __syncthreads();

  // ---- pass 1: (m, S, T) of the whole row -------------------------------
  bool bad = false;
  const Ent all = block_stats<T, UT>(row, 0, nvec, bad, s_ent, &s_bad, [](float) {});
  if (s_bad) {
    if (tid == 0) status_error(status, ARBOR_ENONFINITE);
    return;
  }
  float H;
  {
    // ---- K-th largest key: radix select from the top ----------------------
    uint32_t prefix = 0, pmask = 0;
    int need = top_k;
    unsigned eq_count = 0;
    for (int pass = 0; pass < 3; ++pass) {
      const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
      const int nb = pass == 2 ? 1024 : 2048;
      for (int b = tid; b < 2048; b += UT) hist[b] = 0;
      __syncthreads();
      for_vecs<UT>(row, 0, nvec, [&](const uint4 &u) __attribute__((always_inline)) {
        float x[N];
        VV::get(u, x);
#pragma unroll
        for (int k = 0; k < N; ++k) {
          const uint32_t key = ordered_key(x[k]);
          if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & (nb - 1)], 1u);
        }
      });
      __syncthreads();
      // thread t owns bins nb-1-2t and nb-2-2t (from the top); counts above
      // them by a prefix over threads
      const int hi = nb - 1 - 2 * tid, lo = hi - 1;
      const unsigned ch = hi >= 0 ? hist[hi] : 0u, cl = lo >= 0 ? hist[lo] : 0u;
      int64_t tot;
      const int64_t above = block_exclusive_scan<int64_t>((int64_t)ch + cl, s_scan, &tot);
      if (hi >= 0) {
        if (above < need && need <= above + (int64_t)ch) {
          s_bin = hi;
          s_above = (int)above;
        } else if (lo >= 0 && above + (int64_t)ch < need && need <= above + (int64_t)ch + cl) {
          s_bin = lo;
          s_above = (int)(above + ch);
        }
      }
      __syncthreads();
      const int b = s_bin;
      need -= s_above;
      eq_count = hist[b];
      prefix |= (uint32_t)b << shift;
      pmask |= (uint32_t)(nb - 1) << shift;
      __syncthreads();
    }
    // prefix is the K-th largest key; `need` of its eq_count copies are in the top
    // ---- sums over the top and over the rest -------------------------------
    float st = 0.f, tt = 0.f, sr = 0.f;
    for_vecs<UT>(row, 0, nvec, [&](const uint4 &u) __attribute__((always_inline)) {
      float x[N];
      VV::get(u, x);
#pragma unroll
      for (int k = 0; k < N; ++k) {
        const uint32_t key = ordered_key(x[k]);
        const float d = x[k] * kLog2e - all.m;
        const float p = __builtin_amdgcn_exp2f(d);
        if (key > prefix) {
          st += p;
          tt = __builtin_fmaf(d, p, tt);
        } else if (key < prefix) {
          sr += p;
        }
      }
    });
    st = block_sum_f(st, s_f);
    tt = block_sum_f(tt, s_f);
    sr = block_sum_f(sr, s_f);
    const float dk = key_float(prefix) * kLog2e - all.m;
    const float pk = __builtin_amdgcn_exp2f(dk);
    st += (float)need * pk;
    tt += (float)need * dk * pk;
    sr += (float)(eq_count - (unsigned)need) * pk;
    const float stot = st + sr;
    // - sum_top p ln p = -ln2 (T_top / S - (S_top / S) log2 S); "other" = S_rest / S
    H = -kLn2 * (tt / stot - (st / stot) * __log2f(stot));
    const float po = sr / stot;
    if (po > 0.f) H -= po * __logf(po);
  }
  if (tid == 0) {
    const int o = dst ? dst[r] : r;
    if (o < 0 || o >= n_out)
      status_error(status, ARBOR_EINVAL);
    else
      u_out[o] = 1.0f - H / __logf((float)vocab);
  }
}

// Full vocabulary, part 1: workgroup (chunk c, row r) -> partial (m, S, T).
constexpr int PT = 256;   // threads per chunk
template <class T>
__global__ __launch_bounds__(PT) void uncert_part(const T *__restrict__ logits, int64_t vocab,
                                                  int n_chunk, float4 *__restrict__ part,
                                                  int32_t *status) {
  __shared__ Ent s_ent[PT / kWave];
  __shared__ int s_bad;
  if (status_failed(status)) return;
  const int c = blockIdx.x, r = blockIdx.y;
  const uint4 *row = reinterpret_cast<const uint4 *>(logits + (int64_t)r * vocab);
  const int64_t nvec = vocab / Vec<T>::N;
  const int64_t per = (nvec + n_chunk - 1) / n_chunk;
  const int64_t v0 = min(nvec, (int64_t)c * per), v1 = min(nvec, v0 + per);
  if (threadIdx.x == 0) s_bad = 0;
  __syncthreads();
  bool bad = false;
  const Ent e = block_stats<T, PT>(row, v0, v1, bad, s_ent, &s_bad, [](float) {});
  if (threadIdx.x == 0) part[(int64_t)r * n_chunk + c] = make_float4(e.m, e.s, e.t, s_bad ? 1.f : 0.f);
}

// Full vocabulary, part 2: one wave per row merges its partials in chunk order.
__global__ __launch_bounds__(256) void uncert_merge(const float4 *__restrict__ part, int n_rows,
                                                    int n_chunk, int64_t vocab,
                                                    const int32_t *__restrict__ dst,
                                                    float *__restrict__ u_out, int n_out,
                                                    int32_t *status) {
  if (status_failed(status)) return;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= n_rows || lane_id() != 0) return;
  Ent all{-__builtin_inff(), 0.f, 0.f};
  bool bad = false;
  for (int c = 0; c < n_chunk; ++c) {
    const float4 p = part[(int64_t)r * n_chunk + c];
    bad |= p.w != 0.f;
    all = ent_merge(all, Ent{p.x, p.y, p.z});
  }
  if (bad) {
    status_error(status, ARBOR_ENONFINITE);
    return;
  }
  const float H = kLn2 * (__log2f(all.s) - all.t / all.s);
  const int o = dst ? dst[r] : r;
  if (o < 0 || o >= n_out)
    status_error(status, ARBOR_EINVAL);
  else
    u_out[o] = 1.0f - H / __logf((float)vocab);
}

// ---- top-K over chunks ------------------------------------------------------
constexpr int KMAX = 256;   // largest K of the chunked top-K path

// Radix select over the workgroup: the key of rank `need` (1 = largest) among
// the keys f(visit) hands out, counted 8 bits at a time from the top in the
// LDS histogram `hist` (256 bins).  Returns the key; `need` becomes its rank
// among the keys equal to it.  Every thread gets the same result.
template <class Visit>
__device__ uint32_t block_select(Visit &&visit, int &need, unsigned *hist, int *s_pick,
                                 int64_t *s_scan) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0, pmask = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = tid; b < 256; b += blockDim.x) hist[b] = 0;
    __syncthreads();
    visit([&](uint32_t key) __attribute__((always_inline)) {
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    });
    __syncthreads();
    // thread t owns bin 255 - t: the counts above it by a prefix over threads
    const int b = 255 - tid;
    const unsigned cnt = (tid < 256) ? hist[b] : 0u;
    int64_t tot;
    const int64_t above = block_exclusive_scan<int64_t>((int64_t)cnt, s_scan, &tot);
    if (tid < 256 && above < need && need <= above + (int64_t)cnt) {
      s_pick[0] = b;
      s_pick[1] = (int)above;
    }
    __syncthreads();
    prefix |= (uint32_t)s_pick[0] << shift;
    pmask |= 255u << shift;
    need -= s_pick[1];
    __syncthreads();
  }
  return prefix;
}

constexpr int CMAX = 2048;  // candidates selected in LDS by the chunk workgroups
constexpr int MMAX = 1024;  // candidates selected in LDS by the merge workgroups

// Top-K, part 1: workgroup (chunk c, row r) -> partial (m, S, T) and the
// chunk's K largest values (all of them if the chunk holds fewer), with their
// count.  A bound from the threads' maxima (below) lies at or under the
// chunk's K-th largest value, so only the values at or above it can be among
// the chunk's top K.  Those few are copied to LDS in a fixed order, a radix
// select finds the K-th largest among them, and the values above it (in
// order) and then the needed copies of it are written: the K-th largest is
// always the last of a full list.  If too many values tie at the bound, the
// radix select runs over the chunk itself.
template <class T>
__global__ __launch_bounds__(PT) void uncert_topk_part(const T *__restrict__ logits, int64_t vocab,
                                                       int n_chunk, int top_k,
                                                       float4 *__restrict__ part,
                                                       float *__restrict__ cand,
                                                       int32_t *__restrict__ cand_n,
                                                       int32_t *status) {
  typedef Vec<T> VV;
  constexpr int N = VV::N;
  __shared__ Ent s_ent[PT / kWave];
  __shared__ int s_bad;
  __shared__ __attribute__((aligned(16))) uint32_t s_key[CMAX];
  __shared__ unsigned hist[256];
  __shared__ int s_pick[2];
  __shared__ int64_t s_scan[17];
  if (status_failed(status)) return;
  const int c = blockIdx.x, r = blockIdx.y;
  const int tid = threadIdx.x;
  const uint4 *row = reinterpret_cast<const uint4 *>(logits + (int64_t)r * vocab);
  const int64_t nvec = vocab / N;
  const int64_t per = (nvec + n_chunk - 1) / n_chunk;
  const int64_t v0 = min(nvec, (int64_t)c * per), v1 = min(nvec, v0 + per);
  if (tid == 0) s_bad = 0;
  __syncthreads();
  bool bad = false;
  uint32_t kmax = 0u;             // 0: this thread holds no value
  const Ent e = block_stats<T, PT>(row, v0, v1, bad, s_ent, &s_bad, [&](float x) {
    const uint32_t k = ordered_key(x);
    kmax = k > kmax ? k : kmax;
  });
  const int64_t slot = (int64_t)r * n_chunk + c;
  if (tid == 0) part[slot] = make_float4(e.m, e.s, e.t, s_bad ? 1.f : 0.f);
  if (s_bad) return;                                  // uniform: settled at the stats' sync
  float *out = cand + slot * KMAX;
  // this thread's values in a fixed order (vectors v0 + tid, v0 + tid + PT, ...)
  auto visit = [&](auto &&f) __attribute__((always_inline)) {
    for_vecs<PT>(row, v0, v1, [&](const uint4 &u) __attribute__((always_inline)) {
      float x[N];
      VV::get(u, x);
#pragma unroll
      for (int k = 0; k < N; ++k) f(ordered_key(x[k]));
    });
  };
  // the bound: with K' = ceil(K / 4), a wave's K'-th largest thread maximum
  // has K' of the wave's maxima at or above it, so the smallest of the four
  // waves' has at least 4 K' >= K values of the chunk at or above it (0, which
  // keeps everything, if a wave holds fewer than K' values)
  {
    const int lane = lane_id();
    const int kq = (top_k + 3) / 4;
    int rk = 0;
    for (int j = 0; j < kWave; ++j) {
      const uint32_t kj = (uint32_t)__builtin_amdgcn_readlane((int)kmax, j);
      rk += (kj > kmax || (kj == kmax && j < lane)) ? 1 : 0;
    }
    if (rk == kq - 1) s_key[tid >> 6] = kmax;       // one lane per wave
  }
  __syncthreads();
  uint32_t theta = s_key[0];
#pragma unroll
  for (int w = 1; w < PT / kWave; ++w) theta = min(theta, s_key[w]);
  __syncthreads();                                  // s_key is reused below
  int mine = 0;
  visit([&](uint32_t key) __attribute__((always_inline)) { mine += key >= theta ? 1 : 0; });
  int64_t n_c;
  int o = (int)block_exclusive_scan<int64_t>(mine, s_scan, &n_c);
  int n_keep;
  if (n_c <= CMAX) {
    visit([&](uint32_t key) __attribute__((always_inline)) {
      if (key >= theta) s_key[o++] = key;
    });
    __syncthreads();
    const int n = (int)n_c;
    auto visit_lds = [&](auto &&f) __attribute__((always_inline)) {
      for (int i = tid; i < n; i += PT) f(s_key[i]);
    };
    if (n < top_k) {
      // fewer than K values in the chunk: all copied, in index order
      for (int i = tid; i < n; i += PT) out[i] = key_float(s_key[i]);
      n_keep = n;
    } else {
      int need = top_k;
      const uint32_t tau = block_select(visit_lds, need, hist, s_pick, s_scan);
      // keys above tau in index order, then `need` copies of tau (the K-th
      // largest lands last)
      int gt = 0;
      visit_lds([&](uint32_t key) __attribute__((always_inline)) { gt += key > tau ? 1 : 0; });
      int64_t tot_gt;
      int o_gt = (int)block_exclusive_scan<int64_t>(gt, s_scan, &tot_gt);
      visit_lds([&](uint32_t key) __attribute__((always_inline)) {
        if (key > tau) out[o_gt++] = key_float(key);
      });
      if (tid < need) out[tot_gt + tid] = key_float(tau);
      n_keep = top_k;
    }
  } else {
    int need = top_k;
    const uint32_t tau = block_select(visit, need, hist, s_pick, s_scan);
    // copy: keys > tau at their rank among them, then `need` copies of tau
    int gt = 0, eq = 0;
    visit([&](uint32_t key) __attribute__((always_inline)) {
      gt += key > tau ? 1 : 0;
      eq += key == tau ? 1 : 0;
    });
    int64_t tot_gt, tot_eq;
    int o_gt = (int)block_exclusive_scan<int64_t>(gt, s_scan, &tot_gt);
    int o_eq = (int)block_exclusive_scan<int64_t>(eq, s_scan, &tot_eq);
    visit([&](uint32_t key) __attribute__((always_inline)) {
      if (key > tau) {
        out[o_gt++] = key_float(key);
      } else if (key == tau) {
        if (o_eq < need) out[tot_gt + o_eq] = key_float(key);
        ++o_eq;
      }
    });
    n_keep = top_k;
  }
  if (tid == 0) cand_n[slot] = n_keep;
}

// Top-K, part 2: one workgroup per row.  Merges the chunks' (m, S) in chunk
// order; the row's top K are all among the chunks' candidates (a value among
// the row's top K has fewer than K larger values in its chunk), so the top K
// of the candidates are the row's: ranked in LDS when few, else found by a
// radix select.  The rest of the mass is the "other" outcome.
__global__ __launch_bounds__(PT) void uncert_topk_merge(const float4 *__restrict__ part,
                                                        const float *__restrict__ cand,
                                                        const int32_t *__restrict__ cand_n,
                                                        int n_chunk, int top_k, int64_t vocab,
                                                        const int32_t *__restrict__ dst,
                                                        float *__restrict__ u_out, int n_out,
                                                        int32_t *status) {
  __shared__ __attribute__((aligned(16))) uint32_t s_key[MMAX];
  __shared__ unsigned hist[256];
  __shared__ int s_pick[2];
  __shared__ int64_t s_scan[17];
  __shared__ float s_f[PT / kWave];
  __shared__ Ent s_all;
  __shared__ int s_bad;
  if (status_failed(status)) return;
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  if (tid == 0) {
    Ent all{-__builtin_inff(), 0.f, 0.f};
    int bad = 0;
    for (int c = 0; c < n_chunk; ++c) {
      const float4 p = part[(int64_t)r * n_chunk + c];
      bad |= p.w != 0.f;
      all = ent_merge(all, Ent{p.x, p.y, p.z});
    }
    s_all = all;
    s_bad = bad;
  }
  __syncthreads();
  if (s_bad) {
    if (tid == 0) status_error(status, ARBOR_ENONFINITE);
    return;
  }
  const Ent all = s_all;
  const float *cr = cand + (int64_t)r * n_chunk * KMAX;
  const int32_t *cn = cand_n + (int64_t)r * n_chunk;
  // candidate j of chunk c sits at cr[c * KMAX + j], j < cn[c]
  // candidate counts in LDS when the chunks are few enough
  __shared__ int s_cn[PT];
  if (n_chunk <= PT) s_cn[tid] = tid < n_chunk ? cn[tid] : 0;
  __syncthreads();
  float st = 0.f, tt = 0.f;
  auto add = [&](float x) __attribute__((always_inline)) {
    const float d = x * kLog2e - all.m;
    const float p = __builtin_amdgcn_exp2f(d);
    st += p;
    tt = __builtin_fmaf(d, p, tt);
  };
  int need = 0;
  uint32_t tau = 0u;
  // a lower bound on the row's K-th largest: a chunk that kept K candidates
  // holds K values at or above its own K-th largest, which it wrote last
  __shared__ uint32_t s_lb;
  if (tid == 0) s_lb = 0u;
  __syncthreads();
  for (int c = tid; c < n_chunk; c += PT)
    if (cn[c] == top_k) atomicMax(&s_lb, ordered_key(cr[(int64_t)c * KMAX + top_k - 1]));
  __syncthreads();
  const uint32_t lb = s_lb;
  static_assert(KMAX == PT, "one candidate slot per thread");
  // thread t looks at candidate t of every chunk (loads of eight chunks in
  // flight; unconditional, since slot t always lies in the buffer)
  auto each_cand = [&](auto &&f) __attribute__((always_inline)) {
    for (int c0 = 0; c0 < n_chunk; c0 += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = cr[(int64_t)min(c0 + u, n_chunk - 1) * KMAX + tid];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t key = ordered_key(v[u]);
        if (c0 + u < n_chunk && tid < s_cn[c0 + u] && key >= lb) f(key);
      }
    }
  };
  int n_f = 0;
  if (n_chunk <= PT) {
    int mine = 0;
    each_cand([&](uint32_t) __attribute__((always_inline)) { ++mine; });
    int64_t t;
    int o = (int)block_exclusive_scan<int64_t>(mine, s_scan, &t);
    n_f = (int)t;
    if (n_f <= MMAX) {
      each_cand([&](uint32_t key) __attribute__((always_inline)) { s_key[o++] = key; });
      __syncthreads();
    }
  }
  if (n_chunk <= PT && n_f <= MMAX) {
    // the top K of the row among the candidates at or above lb: the K-th
    // largest, the values above it, and `need` copies of it
    auto visit_lds = [&](auto &&f) __attribute__((always_inline)) {
      for (int i = tid; i < n_f; i += PT) f(s_key[i]);
    };
    need = top_k;
    tau = block_select(visit_lds, need, hist, s_pick, s_scan);
    visit_lds([&](uint32_t key) __attribute__((always_inline)) {
      if (key > tau) add(key_float(key));
    });
  } else {
    auto visit_v = [&](auto &&f) __attribute__((always_inline)) {
      for (int q = tid; q < n_chunk * KMAX; q += PT) {
        const int c = q / KMAX, j = q % KMAX;
        if (j < cn[c]) f(cr[q]);
      }
    };
    auto visit = [&](auto &&f) __attribute__((always_inline)) {
      visit_v([&](float x) __attribute__((always_inline)) { f(ordered_key(x)); });
    };
    need = top_k;
    tau = block_select(visit, need, hist, s_pick, s_scan);
    visit_v([&](float x) __attribute__((always_inline)) {
      if (ordered_key(x) > tau) add(x);
    });
  }
  st = block_sum_f(st, s_f);
  tt = block_sum_f(tt, s_f);
  if (tid == 0) {
    if (need > 0) {          // `need` copies of tau complete the top K
      const float dk = key_float(tau) * kLog2e - all.m;
      const float pk = __builtin_amdgcn_exp2f(dk);
      st += (float)need * pk;
      tt += (float)need * dk * pk;
    }
    const float stot = all.s;
    const float sr = stot - st > 0.f ? stot - st : 0.f;
    // - sum_top p ln p = -ln2 (T_top / S - (S_top / S) log2 S); "other" = S_rest / S
    float H = -kLn2 * (tt / stot - (st / stot) * __log2f(stot));
    const float po = sr / stot;
    if (po > 0.f) H -= po * __logf(po);
    const int o = dst ? dst[r] : r;
    if (o < 0 || o >= n_out)
      status_error(status, ARBOR_EINVAL);
    else
      u_out[o] = 1.0f - H / __logf((float)vocab);
  }
}

// chunks per row for the full-vocabulary path: about 2048 workgroups in all
// (eight per CU), each with at least four vectors per thread
int uncert_chunks(int32_t n_rows, int64_t vocab, int per16) {
  const int64_t nvec = vocab / per16;
  int64_t ch = (2048 + (int64_t)n_rows - 1) / (n_rows > 0 ? n_rows : 1);
  ch = ch < 1 ? 1 : ch;
  const int64_t cap = nvec / (4 * PT) > 0 ? nvec / (4 * PT) : 1;
  return (int)(ch < cap ? ch : cap);
}

}  // namespace

// workspace: chunk partials, then the top-K candidates and their counts
size_t uncertainty_workspace(int32_t n_rows, int64_t vocab, int32_t dtype) {
  if (n_rows <= 0) return 256;
  const size_t slots = (size_t)n_rows * uncert_chunks(n_rows, vocab, dtype == ARBOR_BF16 ? 8 : 4);
  return slots * (sizeof(float4) + KMAX * sizeof(float) + sizeof(int32_t)) + 3 * 256;
}

int launch_uncertainty(const void *logits, int32_t dtype, int32_t n_rows, int64_t vocab,
                       int32_t top_k, const int32_t *dst, float *u_out, int32_t n_out,
                       int32_t *status, void *workspace, size_t workspace_bytes,
                       hipStream_t stream) {
  if (n_rows == 0) return ARBOR_OK;
  const bool bf = dtype == ARBOR_BF16;
  const int ch = uncert_chunks(n_rows, vocab, bf ? 8 : 4);
  const bool topk = top_k > 0 && (int64_t)top_k < vocab;
  if (topk && top_k <= KMAX) {
    if (workspace_bytes < uncertainty_workspace(n_rows, vocab, dtype) || !workspace)
      return ARBOR_EWORKSPACE;
    Carve cv(workspace, workspace_bytes);
    const size_t slots = (size_t)n_rows * ch;
    float4 *part = cv.take<float4>(slots);
    float *cand = cv.take<float>(slots * KMAX);
    int32_t *cand_n = cv.take<int32_t>(slots);
    if (!cv.ok) return ARBOR_EWORKSPACE;
    if (bf)
      hipLaunchKernelGGL(uncert_topk_part<__bf16>, dim3(ch, n_rows), dim3(PT), 0, stream,
                         static_cast<const __bf16 *>(logits), vocab, ch, top_k, part, cand,
                         cand_n, status);
    else
      hipLaunchKernelGGL(uncert_topk_part<float>, dim3(ch, n_rows), dim3(PT), 0, stream,
                         static_cast<const float *>(logits), vocab, ch, top_k, part, cand,
                         cand_n, status);
    hipLaunchKernelGGL(uncert_topk_merge, dim3(n_rows), dim3(PT), 0, stream, part, cand, cand_n,
                       ch, top_k, vocab, dst, u_out, n_out, status);
    return hip_ok(hipGetLastError());
  }
  if (topk) {
    if (bf)
      hipLaunchKernelGGL(uncert_topk<__bf16>, dim3(n_rows), dim3(UT), 0, stream,
                         static_cast<const __bf16 *>(logits), vocab, top_k, dst, u_out, n_out,
                         status);
    else
      hipLaunchKernelGGL(uncert_topk<float>, dim3(n_rows), dim3(UT), 0, stream,
                         static_cast<const float *>(logits), vocab, top_k, dst, u_out, n_out,
                         status);
    return hip_ok(hipGetLastError());
  }
  if (workspace_bytes < uncertainty_workspace(n_rows, vocab, dtype) || !workspace)
    return ARBOR_EWORKSPACE;
  float4 *part = static_cast<float4 *>(workspace);
  if (bf)
    hipLaunchKernelGGL(uncert_part<__bf16>, dim3(ch, n_rows), dim3(PT), 0, stream,
                       static_cast<const __bf16 *>(logits), vocab, ch, part, status);
  else
    hipLaunchKernelGGL(uncert_part<float>, dim3(ch, n_rows), dim3(PT), 0, stream,
                       static_cast<const float *>(logits), vocab, ch, part, status);
  hipLaunchKernelGGL(uncert_merge, dim3((n_rows + 3) / 4), dim3(256), 0, stream, part, n_rows, ch,
                     vocab, dst, u_out, n_out, status);
  return hip_ok(hipGetLastError());
}

}  // namespace arbor
