// Internal declarations shared by the host-side sources of libxema.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include "xema.h"
#include "xema_ops.h"
#include "xema_step.h"

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

// A tensor of a static layout: `size` bytes (already rounded to kAlign),
// alive over the half-open step range [begin, end).
struct LayoutRect {
  int id;
  int64_t size;
  int begin, end;
};

// Algorithm 1 (Sec. 6.1) over `rects`: offsets in input order; returns the
// peak address.
int64_t static_layout(const std::vector<LayoutRect>& rects, std::vector<int64_t>* offsets);

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

// -- the N-block step (step_plan.cpp) --

// Offsets of a block's tensors packed in a staging slot (a tensor the block
// does not use takes no space); returns the slot size.
int64_t packed_offsets(const xema_block_cfg& c, int64_t off[kWeightTensors]);
// The block hyper-parameters alone (a one-token request stands in).
int validate_cfg(const xema_block_cfg* cfg);
// The offload plan with K = k of n blocks (blocks floor((j+1) n / k) - 1).
void fill_offload_plan(const xema_block_cfg& c, int n, int k, int staging, xema_offload_plan* out);
// XEMA_OK when `plan` is the plan fill_offload_plan makes for this cfg.
int check_offload_plan(const xema_block_cfg& c, const xema_offload_plan* plan);

// The step's static layout (Algorithm 1 over its lifetime trace): the
// block's slot table for a group-sequence request at the chunk, the offset
// of every block's every slot, of each residual buffer the workspace holds
// (block i's output; -1 where the caller's out holds it) and of each staging
// slot, and the peak.
struct StepLayout {
  xema_plan block;
  std::vector<int64_t> slot_off;     // [n_blocks * XEMA_NUM_SLOTS]
  std::vector<int64_t> resid_off;    // [n_blocks]
  std::vector<int64_t> staging_off;  // [n_staging]
  int64_t peak = 0;
};
int step_layout(const xema_block_cfg& c, const xema_request& r, int n_blocks, int group, int64_t chunk,
                int n_staging, int64_t slot_bytes, StepLayout* out);
// Modelled time of one block, milliseconds, with the batch in groups of g
// sequences and chunks of ch tokens: the rounds of workgroups of each launch
// over the 256 CUs, a round costing one workgroup's FLOPs at tflops / 256 per
// CU (the latency model of the step plan; xema_workspace_plan_serial ranks
// by it too).
double block_ms(const xema_block_cfg& c, const xema_request& r, int64_t g, int64_t ch, double tflops);

// xema_step_plan_fixed without the argument checks.
int make_step_plan(const xema_block_cfg& c, const xema_request& r, int n_blocks, int n_offloaded, int n_staging,
                   int group, int64_t chunk, const xema_step_costs& costs, xema_step_plan* out);

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
// previous chunk's projections; the output is the same.  clear_status:
// whether this run starts the range flags from zero (the first run of a
// call; later groups and blocks of the call add to them).
int run_block(const xema_block_cfg& c, const xema_request& r, const void* tokens, int x_dtype,
              const xema_block_weights& w, const void* cond, int64_t ch, uint8_t* ws,
              const xema_plan& plan, float* out, hipStream_t s, hipStream_t aux = nullptr,
              bool clear_status = true);
}  // namespace xema
#endif

namespace xema {

}  // namespace xema
