// arbor_compact_noalloc: arbor_compact with its scratch in a fixed device
// array of this library instead of a caller workspace, for callers that
// cannot allocate (code under stream capture, tight serving loops).
//
// The scratch holds what the compaction kernels pass between their launches:
// a source slot and the two plane rows of every kept token (12 bytes per
// token) and four per-node arrays plus a few counters.  Every kernel writes
// each entry it later reads within the same call, so nothing in it has to
// start at zero.  Each GPU that runs the library holds one copy of the array
// until the process ends; its device address is looked up once per device
// (with that device current) and kept here.  Calls on one GPU share the
// array, so calls that overlap on one GPU (different streams, no ordering)
// race on it.
#include <atomic>

#include "arbor_internal.h"

namespace arbor {
int launch_compact(const arbor_geom_t *, arbor_tree_t *, arbor_pool_t *, const int32_t *,
                   const int32_t *, int32_t *, void *, size_t, hipStream_t);
size_t compact_workspace(const arbor_sizes_t *);
}  // namespace arbor

using namespace arbor;

namespace {

constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[ARBOR_NOALLOC_SCRATCH_BYTES];

// per-device address of `scratch`, set once per device by the first call
std::atomic<void *> g_scratch_addr[kMaxDevices];

int scratch_address(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return ARBOR_EHIP;
  if (dev >= kMaxDevices) return ARBOR_EUNSUPPORTED;
  void *p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    // the host-side name of the array is not a device address: ask the
    // runtime for this device's copy (threads that race here store the same
    // value)
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return ARBOR_EHIP;
    g_scratch_addr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return ARBOR_OK;
}

}  // namespace

extern "C" int arbor_compact_noalloc(const arbor_geom_t *geom, arbor_tree_t *tree,
                                     arbor_pool_t *pool, const int32_t *k,
                                     const int32_t *sel_pos, int32_t *status,
                                     hipStream_t stream) {
  if (!geom || !tree || !pool || !status || !k || !sel_pos) return ARBOR_EINVAL;
  if (tree->num_nodes < 0 || tree->num_tokens < 0) return ARBOR_EINVAL;
  arbor_sizes_t sz{};
  sz.num_nodes = tree->num_nodes;
  sz.num_tokens = tree->num_tokens;
  // the same carve as the workspace path, plus its 256-byte alignment slack
  if (compact_workspace(&sz) + 16 * 256 > (size_t)ARBOR_NOALLOC_SCRATCH_BYTES)
    return ARBOR_EWORKSPACE;
  void *ws = nullptr;
  const int rc = scratch_address(&ws);
  if (rc != ARBOR_OK) return rc;
  return arbor_compact(geom, tree, pool, k, sel_pos, status, ws,
                       (size_t)ARBOR_NOALLOC_SCRATCH_BYTES, stream);
}
