// The block forward with its arena in a static device array of the library,
// for callers that cannot allocate device memory (xema_static.h).
#include <mutex>

#include "kernels.h"
#include "xema_internal.h"
#include "xema_static.h"

namespace {

// The arena of xema_dit_block_fwd_static.  Each GPU holds its own copy at its
// own address; in host code this name is only a stand-in for the symbol, so
// it is never passed to a kernel or a copy: the address comes from
// hipGetSymbolAddress, once per device, below.
static __device__ __align__(256) uint8_t scratch[XEMA_STATIC_ARENA_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_arena[kMaxDevices] = {};

}  // namespace

namespace xema {

int static_arena(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return XEMA_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (g_arena[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return XEMA_ERR_HIP;
    g_arena[dev] = p;
  }
  *ptr = g_arena[dev];
  return XEMA_OK;
}

}  // namespace xema

extern "C" int xema_dit_block_fwd_static(const xema_block_cfg* cfg, const xema_request* req,
                                         const void* tokens, const xema_block_weights* weights,
                                         const void* cond, int32_t chunk_tokens, void* out,
                                         void* stream) {
  int st = xema::validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  xema_plan plan;
  st = xema::layout_for_chunk(*cfg, *req, xema::effective_chunk(xema::seq_len(*req), chunk_tokens), &plan);
  if (st != XEMA_OK) return st;
  if (plan.workspace_bytes > XEMA_STATIC_ARENA_BYTES) return XEMA_ERR_WORKSPACE_TOO_SMALL;
  void* arena = nullptr;
  st = xema::static_arena(&arena);
  if (st != XEMA_OK) return st;
  // one stream: the two-stream schedule would create events
  return xema::block_fwd(cfg, req, tokens, weights, cond, req->batch, chunk_tokens, arena,
                         XEMA_STATIC_ARENA_BYTES, out, stream, nullptr);
}
