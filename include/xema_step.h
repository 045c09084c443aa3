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

/* Workspace of xema_dit_step_fwd at chunk_tokens (0 = unchunked), without
 * serialization: the step's static layout (xema_step_plan below) with
 * batch_group = batch.                                                     */
XEMA_API int xema_step_workspace_bytes(const xema_block_cfg* cfg, const xema_request* req,
                                       int32_t chunk_tokens, const xema_offload_plan* plan,
                                       int64_t* bytes);

/* The rates of the step planner's latency model, measured on the device:
 *   h2d_gbytes_per_s  pinned host-to-device copy rate of block weights (one
 *                     MI355X over PCIe measured 56)
 *   block_tflops      the block's throughput on launches that fill the GPU
 *                     (one MI355X measured 1000-1150)                      */
typedef struct {
  double h2d_gbytes_per_s;
  double block_tflops;
} xema_step_costs;

/* A whole-step plan: which blocks are offloaded (Sec. 5.1), the group size of
 * temporary serialization (Sec. 5.2), the chunk size, and the step's static
 * layout (Sec. 6.1).
 *   offload          K, the staging slots and the offloaded blocks
 *   batch_group      g: sequences per group, a divisor of the batch; every
 *                    block runs its batch in groups of g, and the residual
 *                    stream between blocks holds the whole batch
 *                    (serialization is local to the blocks, the batch
 *                    rejoins between them); g = batch: no serialization
 *   chunk_tokens     c: tokens per chunk, c = L: unchunked
 *   workspace_bytes  Algorithm 1's peak over the step's lifetime trace: the
 *                    slots of every block's arena at steps 10 i + s (s the
 *                    block's own step, see xema.h), the fp32 residual stream
 *                    buffers between blocks that live in the workspace (the
 *                    caller's `out` holds every other one: block i writes
 *                    `out` when N - 1 - i is even), live from the first
 *                    step of the loop that writes them (block i's step 9
 *                    repeats per chunk and the block per group, so: step 5
 *                    when chunked, step 0 with several groups, else step 9)
 *                    to the end of the next block, and the staging slots,
 *                    live throughout
 *   device_bytes     resident weight bytes + workspace_bytes: what a device
 *                    budget bounds (the caller's tokens, conditioning and
 *                    output are not counted, as for xema_workspace_plan)
 *   est_ms           the step time the latency model predicts (below)    */
typedef struct {
  xema_offload_plan offload;
  int32_t batch_group;
  int32_t chunk_tokens;
  int64_t workspace_bytes;
  int64_t device_bytes;
  double est_ms;
} xema_step_plan;

/* The plan for given (K, staging, g, c) (chunk_tokens <= 0 or >= L: c = L).
 * Latency model: a block's time is the sum over its launches of the rounds
 * of workgroups over the 256 CUs, each round costing one workgroup's
 * FLOPs at block_tflops / 256 per CU (the GEMMs in 256 x 256 tiles, the
 * attention in query blocks of 512 at head_dim 64 and 256 at 128, all L keys
 * each); the copy of one block's weights takes block_weight_bytes at
 * h2d_gbytes_per_s; the copies run in order on a copy stream, the copy of
 * offloaded block k starting once copy k-1 is done and the block that used
 * its staging slot (offloaded block k - staging) has finished; an offloaded
 * block starts when the previous block and its copy are done.  est_ms is the
 * end of the last block.
 * Errors: INVALID_ARG (NULL, n_blocks outside [1, XEMA_MAX_BLOCKS], K outside
 * [0, n_blocks], staging < 1, batch_group not dividing the batch, costs not
 * positive), shape errors as xema_workspace_plan.                          */
XEMA_API int xema_step_plan_fixed(const xema_block_cfg* cfg, const xema_request* req,
                                  int32_t n_blocks, int32_t n_offloaded, int32_t n_staging,
                                  int32_t batch_group, int32_t chunk_tokens,
                                  const xema_step_costs* costs, xema_step_plan* out);

/* "Only as much mitigation as needed" for the whole step (Sec. 5.1, pi*):
 * among every (K, g, c) - K in [0, n_blocks], g a divisor of the batch, c = L
 * or a multiple of XEMA_CHUNK_GRANULE below L - whose device_bytes fit
 * device_budget_bytes, the one with the least est_ms (ties: fewer offloaded
 * blocks, then the larger group, then the larger chunk).  One budget bounds
 * the resident weights and the activations together.
 * Errors: as xema_step_plan_fixed; BUDGET_TOO_SMALL when nothing fits
 * (out->device_bytes then holds the least device_bytes of any candidate).  */
XEMA_API int xema_step_plan_budget(const xema_block_cfg* cfg, const xema_request* req,
                                   int32_t n_blocks, int32_t n_staging, int64_t device_budget_bytes,
                                   const xema_step_costs* costs, xema_step_plan* out);

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

/* xema_dit_step_fwd with a whole-step plan (xema_step_plan_fixed or
 * xema_step_plan_budget for this cfg and request): offloading by
 * plan->offload, every block run in groups of plan->batch_group sequences
 * and chunks of plan->chunk_tokens tokens, the intermediates of every block
 * and the residual stream at the offsets of the step's static layout.  The
 * output is bit-identical for every plan.  workspace_bytes must be at least
 * plan->workspace_bytes.  Other arguments and errors as xema_dit_step_fwd;
 * INVALID_ARG for a plan the library did not make for this configuration. */
XEMA_API int xema_dit_step_fwd_planned(const xema_block_cfg* cfg, const xema_request* req,
                                       const void* tokens, const xema_block_weights* weights,
                                       const xema_step_plan* plan, const void* cond, void* workspace,
                                       int64_t workspace_bytes, void* out, void* stream,
                                       void* copy_stream);

#ifdef __cplusplus
}
#endif

#endif /* XEMA_STEP_H_ */
