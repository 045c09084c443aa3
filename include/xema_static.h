/*
 * xema_static.h -- the DiT block forward without a caller workspace.
 *
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * block's arena is a static device array inside libxema, one copy per GPU
 * the library runs on, each held until the process ends.  Nothing is
 * allocated or freed by the call; the caller still passes the inputs and
 * the output.  Include xema.h first.
 */
#ifndef XEMA_STATIC_H_
#define XEMA_STATIC_H_

#include <stdint.h>

#include "xema.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Size of the static arena on each device: 64 MiB, enough for the tiny
 * workload unchunked (about 3 MB) and for any request whose layout
 * (xema_workspace_bytes) fits in it. */
#define XEMA_STATIC_ARENA_BYTES ((int64_t)64 << 20)

/* xema_dit_block_fwd with its arena in the library's static device array of
 * the current device (the device of `stream`, which must be current).
 * Arguments, semantics and output are those of xema_dit_block_fwd, and the
 * output is bit-identical to it; there is no workspace argument.
 *   - Calls no hipMalloc, hipFree or any other allocating routine.
 *   - The first call on a device looks up that device's copy of the array
 *     (hipGetSymbolAddress) and keeps its address.
 *   - Every call on a GPU shares that GPU's array and leaves its
 *     intermediates there; the call rewrites everything it reads (the
 *     padding of Q/K/V and the range flags included), so no state carries
 *     over between calls.  Calls that overlap on one GPU (concurrent
 *     streams, threads) race on the array: order them on one stream.
 *   - xema_block_status(&plan, NULL, stream, &flags), with the layout of
 *     the request at chunk_tokens, reads the range flags of the last call.
 * Errors: as xema_dit_block_fwd, raised before any launch;
 * XEMA_ERR_WORKSPACE_TOO_SMALL when the layout at chunk_tokens needs more
 * than XEMA_STATIC_ARENA_BYTES (chunk the request or use
 * xema_dit_block_fwd); XEMA_ERR_HIP when the array's address cannot be
 * obtained or a launch fails.                                             */
XEMA_API int xema_dit_block_fwd_static(const xema_block_cfg* cfg, const xema_request* req,
                                       const void* tokens, const xema_block_weights* weights,
                                       const void* cond, int32_t chunk_tokens, void* out,
                                       void* stream);

#ifdef __cplusplus
}
#endif

#endif /* XEMA_STATIC_H_ */
