/*
 * xema.h -- C ABI of the DiT block forward for AMD Instinct MI355X (gfx950).
 *
 * One call runs one Diffusion-Transformer denoising-step block: the stage the
 * paper identifies as dominating diffusion inference (Sec. 2.1: the denoiser
 * is a stack of repeated transformer blocks), whose activations grow with the
 * latent sequence length H x W x T (Sec. 2.2), token-chunked under a per-call
 * activation budget.  Chunking is the paper's "only as much mitigation as
 * needed" (Sec. 5.1, objective pi*) applied to the operators it names for
 * chunking, DiT attention and its neighbours (Sec. 5.2, "Localized chunking
 * and fusion"; Sec. 8, memory mitigation primitives).  All intermediates live
 * in one caller-owned arena at offsets fixed offline by the paper's static
 * layout, Algorithm 1 (Sec. 6.1), so runtime allocation is a table lookup
 * (Sec. 8, "Static memory runtime").
 *
 * Conventions for every function here:
 *   - Return value: XEMA_OK (0) or a negative xema_status.  Nothing throws.
 *   - Every argument is validated on the host before any device work; on an
 *     error no kernel has been launched and no output byte was written.
 *   - The library never allocates or frees device memory and keeps no global
 *     device state.  All functions are thread-safe.
 *   - Device pointers must be 16-byte aligned; the workspace 256-byte aligned.
 *   - Token/weight/conditioning inputs are bfloat16 (bit patterns, uint16).
 *
 * Precision contract (where this library departs from a bf16-everywhere
 * block, and why).  The block output `out` and the residual stream x1 are
 * fp32: one bf16 rounding of the output alone costs a mean absolute error of
 * about 2e-3 on unit-variance activations, the whole accuracy bar of the
 * path, so the output is handed over unrounded and a caller that stores bf16
 * rounds once itself.  The contractions of attention, the output projection
 * and the MLP run fp16 MFMA (fp32 accumulation): V, the attention
 * probabilities P, the attention output O, the LN2 output h2, the MLP hidden
 * activations g and the fp16 copies of W_o, W_up and W_down are fp16, which
 * has three more mantissa bits than bf16 and the same MFMA rate on gfx950,
 * but a range of +-65504.  The QKV projection is bf16 MFMA on the bf16 LN1
 * output and the caller's bf16 W_qkv; Q and K are stored fp16 after
 * QK-RMSNorm, RoPE and the softmax factor.  Range limits:
 *   - V, h2 and g must stay below 65504 in magnitude (they round to inf
 *     at 65520 and above); O is a convex combination of V rows and cannot
 *     leave the range when V does not;
 *   - Q and K are bounded by sqrt(d) |gamma| after the RMS normalisation;
 *   - weights converted to fp16 must be below 65504 in magnitude, and lose
 *     relative precision below 2^-14 (fp16 subnormals) and vanish below
 *     2^-25.
 * Every fp16 store of V, Q, K, h2 and g and every converted weight is
 * checked: a value at or beyond the fp16 range (or NaN) sets a flag in the
 * arena's status slot, which xema_block_status reads after the call.  A
 * call whose status is not clean has produced non-finite or saturated
 * intermediates and its output must not be used.
 */
#ifndef XEMA_H_
#define XEMA_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define XEMA_API __attribute__((visibility("default")))

typedef enum {
  XEMA_OK = 0,
  XEMA_ERR_INVALID_ARG = -1,          /* NULL pointer, non-positive size, aliasing */
  XEMA_ERR_UNSUPPORTED = -2,          /* shape outside what the kernels handle */
  XEMA_ERR_BUDGET_TOO_SMALL = -3,     /* even the smallest chunk exceeds the budget */
  XEMA_ERR_WORKSPACE_TOO_SMALL = -4,  /* workspace_bytes below the plan's arena size */
  XEMA_ERR_MISALIGNED = -5,           /* pointer alignment violated */
  XEMA_ERR_HIP = -6,                  /* a HIP launch or runtime call failed */
  XEMA_ERR_RANGE = -7                 /* an fp16 intermediate left its range (xema_block_status) */
} xema_status;

/* Bits of the range status (xema_block_status): which fp16 intermediate
 * held a value at or beyond +-65520 (rounds to inf) or a NaN.             */
enum {
  XEMA_RANGE_QKV = 1,       /* Q, K or V written by the QKV projection's epilogue */
  XEMA_RANGE_LN2 = 2,       /* h2, the LN2 + modulation output */
  XEMA_RANGE_MLP = 4,       /* g, the MLP hidden activations after GELU */
  XEMA_RANGE_WEIGHTS = 8    /* a phase-B weight converted to fp16 in the call */
};
#define XEMA_STATUS_WORDS 4

#define XEMA_MAX_SLOTS 16
#define XEMA_CHUNK_GRANULE 256        /* planned chunks are multiples of this, or all */
#define XEMA_SEQ_PAD 128              /* per-head Q/K/V storage pads L to this */

/* Block hyper-parameters: the "model" part of a request template
 * r = (model, H, W, T) (Sec. 2.1).
 *   hidden      D = heads * head_dim, a multiple of 256, at most 8192
 *   heads       H
 *   head_dim    d, 64 or 128
 *   mlp_hidden  F, a multiple of 256
 *   cond_dim    D_c, width of the conditioning vector, a multiple of 8
 *   rope_dims   (d_t, d_h, d_w): even widths of the contiguous [t | y | w]
 *               RoPE segments of each head vector, sum <= head_dim
 *   rope_theta  RoPE base (10000 in every shipped config)
 *   ln_eps      LayerNorm epsilon; qk_eps  QK-RMSNorm epsilon
 *   modulation_streams  1 (or 0): one AdaLN map modulates every token;
 *               2: dual-stream block, whose text tokens take their shift,
 *               scale and gate from a second AdaLN map of their own
 *               (xema_block_weights.ada_txt_w / ada_txt_b), the visual
 *               tokens from ada_w / ada_b; every other weight is shared
 *   weights_f16 0: o_w, up_w and down_w are bf16 like every other weight and
 *               each call converts them into fp16 arena slots;
 *               1: the caller passes o_w, up_w and down_w already in fp16
 *               (converted once per model, e.g. with xema_op_convert_f16),
 *               which the block reads directly (no conversion, no arena
 *               slots for the copies; bit-identical output)              */
typedef struct {
  int32_t hidden, heads, head_dim, mlp_hidden, cond_dim;
  int32_t rope_dims[3];
  float rope_theta, ln_eps, qk_eps;
  int32_t modulation_streams;
  int32_t weights_f16;
} xema_block_cfg;

/* One batched call: `batch` requests of one template (the paper batches only
 * within a template, Sec. 2.3 "Concurrency"), each a sequence of text_len text
 * tokens followed by grid_t * grid_h * grid_w visual tokens in t-major, then
 * row, then column order.  L = text_len + grid_t * grid_h * grid_w.        */
typedef struct {
  int32_t batch, text_len, grid_t, grid_h, grid_w;
} xema_request;

/* Device pointers to the block weights, bfloat16, nn.Linear layout [out, in]:
 *   ada_w [6D, D_c]  ada_b [6D]     AdaLN map, rows ordered (shift1, scale1,
 *                                   gate1, shift2, scale2, gate2)
 *   qkv_w [3D, D]    qkv_b [3D]     rows ordered (q | k | v), head j owns rows
 *                                   [j d, (j+1) d) of each part
 *   q_gamma [d]      k_gamma [d]    QK-RMSNorm gains shared by all heads
 *   o_w [D, D]       o_b [D]        attention output projection
 *   up_w [F, D]      up_b [F]       MLP up projection (GELU-tanh follows)
 *   down_w [D, F]    down_b [D]     MLP down projection
 *                                   (o_w, up_w, down_w are fp16 instead
 *                                   when xema_block_cfg.weights_f16 = 1)
 *   ada_txt_w [6D, D_c]  ada_txt_b [6D]  the text tokens' AdaLN map of a
 *                                   dual-stream block (modulation_streams = 2),
 *                                   rows ordered as ada_w; ignored otherwise */
typedef struct {
  const void *ada_w, *ada_b, *qkv_w, *qkv_b, *q_gamma, *k_gamma;
  const void *o_w, *o_b, *up_w, *up_b, *down_w, *down_b;
  const void *ada_txt_w, *ada_txt_b;
} xema_block_weights;

/* A static arena layout: the tensor-id -> offset table of Sec. 8 ("Static
 * memory runtime") produced by Algorithm 1 (Sec. 6.1) over the block's slot
 * lifetimes.  slot_begin/slot_end are half-open step lifetimes.           */
typedef struct {
  int32_t chunk_tokens;               /* tokens per sequence per chunk; == L means unchunked */
  int32_t n_slots;
  int64_t workspace_bytes;            /* arena size at chunk_tokens (Algorithm 1 peak) */
  int64_t min_workspace_bytes;        /* the smallest arena over the candidate chunks */
  int64_t slot_offset[XEMA_MAX_SLOTS];
  int64_t slot_bytes[XEMA_MAX_SLOTS];
  int32_t slot_begin[XEMA_MAX_SLOTS];
  int32_t slot_end[XEMA_MAX_SLOTS];
} xema_plan;

/* Slot ids of xema_plan.  Steps: 0 AdaLN map + RoPE table; phase A (per token
 * chunk) 1 LN1, 2 QKV projection, 3 QK-norm/RoPE scatter; 4 fp16 copies of the
 * phase-B weights; phase B (per query chunk) 5 attention, 6 out-projection +
 * gated residual, 7 LN2, 8 MLP up + GELU, 9 MLP down + gated residual.
 * The qkv slot is empty: head_dim is 64 or 128, where the QKV GEMM's
 * epilogue writes Q, K and V^T itself; the three weight-copy slots are
 * empty when cfg.weights_f16 = 1.                                          */
enum {
  XEMA_SLOT_MOD = 0,   /* fp32 [S, B, 6D], S modulation streams (visual first) life [0, 10) */
  XEMA_SLOT_ROPE,      /* fp32 cos/sin per axis position     life [0, 4)  */
  XEMA_SLOT_Q,         /* fp16 [B, H, Lp, d]                 life [1, 10) */
  XEMA_SLOT_K,         /* fp16 [B, H, Lp, d]                 life [1, 10) */
  XEMA_SLOT_VT,        /* fp16 [B, H, d, Lp] (transposed)    life [1, 10) */
  XEMA_SLOT_LN1,       /* bf16 [B*c, D]                      life [1, 3)  */
  XEMA_SLOT_QKV,       /* fp16 [B*c, 3D]  life [2, 4); empty at head_dim 64 and 128,
                          where the QKV GEMM writes Q, K and V^T itself */
  XEMA_SLOT_WO16,      /* fp16 [D, D]                        life [4, 10) */
  XEMA_SLOT_WUP16,     /* fp16 [F, D]                        life [4, 10) */
  XEMA_SLOT_WDOWN16,   /* fp16 [D, F]                        life [4, 10) */
  XEMA_SLOT_ATTN,      /* fp16 [B*c, D]      life [5, 7); [5, 10) when chunked (the
                          next chunk's attention may overlap this chunk's MLP) */
  XEMA_SLOT_X1,        /* fp32 [B*c, D]                      life [6, 10) */
  XEMA_SLOT_LN2,       /* fp16 [B*c, D]                      life [7, 9)  */
  XEMA_SLOT_HID,       /* fp16 [B*c, F]                      life [8, 10) */
  XEMA_SLOT_STATUS,    /* uint32 [XEMA_STATUS_WORDS] range flags, cleared at
                          step 0                             life [0, 10) */
  XEMA_NUM_SLOTS
};

/* Fill `out` from a request template r = (model, H, W, T) (Sec. 2.1): the
 * latent grid is grid_h = ceil(H / 16), grid_w = ceil(W / 16) (8x spatial VAE
 * downsampling and 2x2 patches) and grid_t = (T - 1) / 4 + 1 (4x temporal VAE
 * downsampling; T = 1 is an image).  Host only.
 * Errors: XEMA_ERR_INVALID_ARG for NULL pointers or non-positive sizes.     */
XEMA_API int xema_request_from_template(const xema_block_cfg* cfg, int32_t height, int32_t width,
                               int32_t frames, int32_t batch, int32_t text_len,
                               xema_request* out);

/* Arena layout for a given chunk size (chunk_tokens <= 0 or >= L means
 * unchunked): slot sizes and lifetimes of the block, packed by Algorithm 1
 * (Sec. 6.1).  Host only.
 * Errors: XEMA_ERR_INVALID_ARG, XEMA_ERR_UNSUPPORTED (shape checks).       */
XEMA_API int xema_workspace_layout(const xema_block_cfg* cfg, const xema_request* req,
                          int32_t chunk_tokens, xema_plan* out);

/* Arena bytes needed at chunk_tokens (the layout's workspace_bytes).  Host only. */
XEMA_API int xema_workspace_bytes(const xema_block_cfg* cfg, const xema_request* req,
                         int32_t chunk_tokens, int64_t* bytes);

/* "Only as much mitigation as needed" (Sec. 5.1, pi*): the largest candidate
 * chunk (L itself, or a multiple of XEMA_CHUNK_GRANULE below L) whose arena
 * fits budget_bytes, with its layout.  The budget counts arena bytes only;
 * caller-owned tokens, weights, conditioning and output are not in it.
 * Host only.
 * Errors: XEMA_ERR_BUDGET_TOO_SMALL when no candidate fits (out->chunk_tokens
 * is then 0 and out->min_workspace_bytes holds the smallest arena over the
 * candidates);
 * XEMA_ERR_INVALID_ARG, XEMA_ERR_UNSUPPORTED.                              */
XEMA_API int xema_workspace_plan(const xema_block_cfg* cfg, const xema_request* req,
                        int64_t budget_bytes, xema_plan* out);

/* One DiT block forward, asynchronous on `stream` (a hipStream_t; NULL means
 * the default stream).
 *   tokens   device, bf16 [B, L, D] row-major, read only
 *   weights  device pointers, see xema_block_weights
 *   cond     device, bf16 [B, D_c], the conditioning vector of each request
 *   chunk_tokens  tokens per sequence per chunk for both phases; <= 0 or >= L
 *            means unchunked; any positive value is accepted (the last chunk
 *            may be shorter).  The result is bit-identical for every value.
 *   workspace, workspace_bytes  device arena of at least
 *            xema_workspace_bytes(cfg, req, chunk_tokens) bytes, 256-byte
 *            aligned, owned by the caller.  Its contents on entry are ignored;
 *            on return it holds the intermediates at the layout's offsets.
 *   out      device, fp32 [B, L, D] (fp32, not bf16: see the precision
 *            contract above), written once per element; must not overlap
 *            tokens, weights, cond or the workspace.
 * Computes, per batch element (the block definition: AdaLN-modulated
 * LayerNorm, QKV projection, QK-RMSNorm, 3D RoPE, joint full self-attention,
 * gated output projection, LayerNorm, GELU-tanh MLP, gated residual):
 *   m = W_ada c + b_ada = (shift1, scale1, gate1, shift2, scale2, gate2)
 *   (a dual-stream block uses m_txt = W_ada_txt c + b_ada_txt on its text
 *   tokens, positions below text_len, and m on the visual tokens)
 *   h = LN(x)(1 + scale1) + shift1;  [q|k|v] = h W_qkv^T + b_qkv
 *   q, k <- RoPE(RMSNorm(.) * gamma) per head;  o = softmax(q k^T / sqrt(d)) v
 *   x1 = x + gate1 (o W_o^T + b_o);  h2 = LN(x1)(1 + scale2) + shift2
 *   out = x1 + gate2 (GELU_tanh(h2 W_up^T + b_up) W_down^T + b_down)
 * Errors (all raised before any launch): XEMA_ERR_INVALID_ARG,
 * XEMA_ERR_UNSUPPORTED, XEMA_ERR_MISALIGNED, XEMA_ERR_WORKSPACE_TOO_SMALL;
 * XEMA_ERR_HIP if a launch fails.                                          */
XEMA_API int xema_dit_block_fwd(const xema_block_cfg* cfg, const xema_request* req,
                       const void* tokens, const xema_block_weights* weights,
                       const void* cond, int32_t chunk_tokens,
                       void* workspace, int64_t workspace_bytes,
                       void* out, void* stream);

/* Temporary serialization (Sec. 5.2, "Temporary serialization") together
 * with chunking: a batch whose arena exceeds the budget can run its
 * sequences through the block in equal groups of g < batch (g divides the
 * batch), one group after another, each group seeing the arena of a
 * g-sequence request; elsewhere the batch keeps its size.  For each g the
 * plan takes the largest chunk whose arena fits budget_bytes, and among
 * those (g, chunk) pairs the least modelled block time, then the larger g:
 * the least latency overhead of pi* (Sec. 5.1) under the latency model of
 * xema_step_plan_budget (xema_step.h), the rounds of workgroups of every
 * launch over the 256 CUs.  Groups and chunks never remove a round, so with
 * an ample budget it is (batch, L): no mitigation.
 * *batch_group receives g and `out` the layout for a g-sequence request.
 * Host only.
 * Errors: as xema_workspace_plan; BUDGET_TOO_SMALL when even one sequence at
 * the smallest chunk does not fit (out->min_workspace_bytes then holds that
 * arena, *batch_group is 0).                                              */
XEMA_API int xema_workspace_plan_serial(const xema_block_cfg* cfg, const xema_request* req,
                               int64_t budget_bytes, int32_t* batch_group, xema_plan* out);

/* xema_dit_block_fwd with the batch run in groups of batch_group sequences
 * (1 <= batch_group; >= batch means one group).  The workspace needs the
 * arena of a batch_group-sequence request and of the shorter last group
 * (xema_workspace_plan_serial reports the larger).  The output is
 * bit-identical for every batch_group and chunk_tokens.  Errors as
 * xema_dit_block_fwd.                                                     */
XEMA_API int xema_dit_block_fwd_serial(const xema_block_cfg* cfg, const xema_request* req,
                              const void* tokens, const xema_block_weights* weights,
                              const void* cond, int32_t batch_group, int32_t chunk_tokens,
                              void* workspace, int64_t workspace_bytes,
                              void* out, void* stream);

/* xema_dit_block_fwd_serial with the attention of each query chunk on a
 * second stream: with two chunks or more, the attention of chunk k runs on
 * aux_stream as soon as the out-projection of chunk k-1 has read the
 * attention buffer, alongside the LN2 and MLP of chunk k-1 on `stream`, so
 * the last, partly filled round of workgroups of one kernel overlaps the
 * other's (chunking should cost only what the budget needs, Sec. 5.1; this
 * trims what a chunk too small to fill the GPU costs).  The chunked layout
 * keeps the attention buffer apart from the MLP's buffers for this.  HIP
 * events created and released by the call order the streams; the output is
 * bit-identical to xema_dit_block_fwd.  aux_stream NULL or equal to
 * `stream`, or an unchunked call, runs everything on `stream`.
 * Asynchronous on `stream`: when work queued on `stream` after this call
 * starts, the aux_stream work of this call has finished.  Calls that share a
 * workspace must be ordered on `stream`; aux_stream must have the default
 * priority.  Errors as xema_dit_block_fwd.                                 */
XEMA_API int xema_dit_block_fwd_pipelined(const xema_block_cfg* cfg, const xema_request* req,
                                 const void* tokens, const xema_block_weights* weights,
                                 const void* cond, int32_t batch_group, int32_t chunk_tokens,
                                 void* workspace, int64_t workspace_bytes,
                                 void* out, void* stream, void* aux_stream);

/* Range status of the last block call that used this workspace with this
 * layout (any xema_dit_block_fwd* entry point; workspace NULL: the static
 * arena of xema_dit_block_fwd_static on the current device): waits for
 * `stream`, copies the status slot to the host and sets *flags to the
 * XEMA_RANGE_* bits of the fp16 intermediates that left their range (0:
 * none).  Returns XEMA_OK when *flags is 0 and XEMA_ERR_RANGE otherwise;
 * XEMA_ERR_INVALID_ARG for NULL plan or flags or a layout without a status
 * slot; XEMA_ERR_HIP if the copy fails.  Synchronous; allocates nothing.  */
XEMA_API int xema_block_status(const xema_plan* plan, const void* workspace, void* stream,
                               uint32_t* flags);

/* Static string naming a status code. */
XEMA_API const char* xema_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* XEMA_H_ */
