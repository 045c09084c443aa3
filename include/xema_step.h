/*
 * xema_step.h -- C ABI of an N-block denoising step with selective weight
 * offloading, on top of the block forward of xema.h.
 *
 * A denoiser is a stack of N DiT blocks with distinct weights (Sec. 2.1).
 * When the weights of all N blocks do not fit the device's weight budget,
 * the paper offloads only as many blocks as needed (Sec. 5.1, "Applying Only
 * as Much Mitigation as Needed", objective pi*): the smallest K that fits,
 * with the K offloaded blocks spread uniformly so that about N/K blocks of
 * computation separate two transfers and can hide them ("Selective
 * offloading and HSDP").  Offloaded weights stay in pinned host memory and
 * are copied into device staging slots ahead of their block on a second
 * stream; the copy stream and the compute stream synchronise by events.
 *
 * Numerics: x_0 = tokens (bf16); x_{i+1} = block_i(x_i), the residual stream
 * kept in fp32 between blocks; out = x_N.  Offloading changes where weights
 * live, never what is computed: the output is bit-identical for every K,
 * every staging depth and every chunk size.
 *
 * Conventions of xema.h apply (status codes, validation before any launch,
 * no device allocation, 16-byte device pointers, 256-byte workspace).
 */
#ifndef XEMA_STEP_H_
#define XEMA_STEP_H_

#include <stdint.h>

#include "xema.h"

#ifdef __cplusplus
extern "C" {
#endif

#define XEMA_MAX_BLOCKS 256

/* Result of offload planning for n_blocks blocks of one configuration.
 *   n_offloaded          K, blocks whose weights stay in pinned host memory
 *   n_staging            device staging slots (min(requested, K); 0 if K = 0)
 *   offloaded[i]         1 if block i is offloaded (i < n_blocks)
 *   block_weight_bytes   one block's weight tensors packed into a staging
 *                        slot, each tensor at a 256-byte boundary
 *   resident_weight_bytes  (N - K) blocks' tensors, unpacked sum
 *   device_weight_bytes  resident + staging: what counts against the budget */
typedef struct {
  int32_t n_blocks;
  int32_t n_offloaded;
  int32_t n_staging;
  int32_t offloaded[XEMA_MAX_BLOCKS];
  int64_t block_weight_bytes;
  int64_t resident_weight_bytes;
  int64_t staging_bytes;
  int64_t device_weight_bytes;
} xema_offload_plan;

/* Offload plan with a given K (0 <= K <= n_blocks): block i is offloaded iff
 * i = floor((j + 1) N / K) - 1 for some j in [0, K), i.e. the K blocks are
 * spread uniformly and the last block is always among them (Sec. 5.1,
 * selective offloading).  n_staging >= 1.
 * Errors: INVALID_ARG for NULL, n_blocks outside [1, XEMA_MAX_BLOCKS], K
 * outside [0, n_blocks] or n_staging < 1; shape errors of validate as in
 * xema_workspace_plan (the request's shape is not needed here).            */
XEMA_API int xema_offload_plan_k(const xema_block_cfg* cfg, int32_t n_blocks, int32_t n_offloaded,
                                 int32_t n_staging, xema_offload_plan* out);

/* The smallest K whose device_weight_bytes fits weight_budget_bytes (the
 * pi* objective with offloading as the only mitigation: every extra
 * offloaded block adds transfer latency and saves nothing once the budget
 * holds).  BUDGET_TOO_SMALL when even K = n_blocks does not fit (the staging
 * slots alone exceed the budget); out->device_weight_bytes then holds the
 * requirement at K = n_blocks.                                            */
XEMA_API int xema_offload_plan_budget(const xema_block_cfg* cfg, int32_t n_blocks,
                                      int64_t weight_budget_bytes, int32_t n_staging,
                                      xema_offload_plan* out);

/* Workspace of xema_dit_step_fwd at chunk_tokens (0 = unchunked): the
 * block's activation arena (xema_workspace_bytes), then an fp32 [B, L, D]
 * buffer for the residual stream, then the plan's staging slots, each at a
 * 256-byte boundary.                                                       */
XEMA_API int xema_step_workspace_bytes(const xema_block_cfg* cfg, const xema_request* req,
                                       int32_t chunk_tokens, const xema_offload_plan* plan,
                                       int64_t* bytes);

/* Runs the plan's n_blocks blocks on `tokens`.
 *   tokens      device, bf16 [B, L, D]
 *   weights     array of n_blocks weight sets (xema.h layout): device
 *               pointers for resident blocks; for offloaded blocks pointers
 *               to pinned host memory (hipHostMalloc), read by DMA
 *   cond        device, bf16 [B, D_c], shared by all blocks (each block has
 *               its own AdaLN map)
 *   workspace   device, xema_step_workspace_bytes bytes
 *   out         device, fp32 [B, L, D]; must not overlap any input
 *   stream      hipStream_t running the blocks (NULL: default stream)
 *   copy_stream hipStream_t for the host-to-device weight copies; it must
 *               differ from `stream` to overlap copies with compute (NULL or
 *               equal to `stream`: copies run in order on `stream`)
 * Asynchronous on `stream`: when work queued on `stream` after this call
 * starts, every copy has landed.  The call creates and releases its HIP
 * events.  Calls that share a workspace must be ordered on one stream.    */
XEMA_API int xema_dit_step_fwd(const xema_block_cfg* cfg, const xema_request* req,
                               const void* tokens, const xema_block_weights* weights,
                               const xema_offload_plan* plan, const void* cond,
                               int32_t chunk_tokens, void* workspace, int64_t workspace_bytes,
                               void* out, void* stream, void* copy_stream);

#ifdef __cplusplus
}
#endif

#endif /* XEMA_STEP_H_ */
