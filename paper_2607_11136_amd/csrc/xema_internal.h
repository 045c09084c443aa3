// Internal declarations shared by the host-side sources of libxema.
#pragma once

#include <cstddef>
#include <cstdint>

#include "xema.h"
#include "xema_ops.h"

namespace xema {

constexpr int64_t kAlign = 256;

inline int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

inline int64_t seq_len(const xema_request& r) {
  return (int64_t)r.text_len + (int64_t)r.grid_t * r.grid_h * r.grid_w;
}
inline int64_t padded_len(int64_t L) { return round_up(L, XEMA_SEQ_PAD); }

// Shape checks shared by planning and the forward call.
int validate_shapes(const xema_block_cfg* cfg, const xema_request* req);

// Chunk size actually used for a requested chunk_tokens.
inline int64_t effective_chunk(int64_t L, int64_t chunk) {
  return (chunk <= 0 || chunk >= L) ? L : chunk;
}

// Fill `out` with the slot table at chunk `c` and its Algorithm 1 offsets.
int layout_for_chunk(const xema_block_cfg& cfg, const xema_request& req, int64_t c,
                     xema_plan* out);

// A block's weight tensors in the order of xema_block_weights: the twelve
// shared ones, then the text tokens' AdaLN map of a dual-stream block (size 0
// for a single-stream block).
constexpr int kWeightTensors = 14;
inline bool dual_stream(const xema_block_cfg& c) { return c.modulation_streams == 2; }
void block_weight_sizes(const xema_block_cfg& cfg, int64_t bytes[kWeightTensors]);
inline const void* const* weight_ptrs(const xema_block_weights& w) { return &w.ada_w; }
inline const void** weight_ptrs(xema_block_weights& w) { return &w.ada_w; }
static_assert(sizeof(xema_block_weights) == kWeightTensors * sizeof(void*), "weight struct layout");

// The block forward behind every xema_dit_block_fwd* entry point: validates
// the call (the workspace must hold the layout of a batch_group-sequence
// request at chunk_tokens), then runs the groups; aux_stream as in
// xema_dit_block_fwd_pipelined.
int block_fwd(const xema_block_cfg* cfg, const xema_request* req, const void* tokens,
              const xema_block_weights* w, const void* cond, int32_t batch_group, int32_t chunk_tokens,
              void* workspace, int64_t workspace_bytes, void* out, void* stream, void* aux_stream);

// Address of the current device's static arena (xema_static.h), looked up
// once per device.  XEMA_ERR_HIP if it cannot be obtained.
int static_arena(void** ptr);

}  // namespace xema

#ifdef __HIPCC__
#include <hip/hip_runtime.h>
namespace xema {
// One block forward on stream s (arguments validated by the caller): x is
// [B, L, D] in x_dtype (XEMA_BF16 or XEMA_F32), the arena follows `plan`,
// out is [B, L, D] fp32.  With a second stream `aux` (not null, not s) and
// two chunks or more, each chunk's attention runs on aux, overlapping the
// previous chunk's projections; the output is the same.
int run_block(const xema_block_cfg& c, const xema_request& r, const void* tokens, int x_dtype,
              const xema_block_weights& w, const void* cond, int64_t ch, uint8_t* ws,
              const xema_plan& plan, float* out, hipStream_t s, hipStream_t aux = nullptr);
}  // namespace xema
#endif

namespace xema {

}  // namespace xema
