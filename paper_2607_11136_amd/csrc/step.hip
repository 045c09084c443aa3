// Host driver of the N-block denoising step (xema_step.h): the blocks in
// order, each run in groups of g sequences (temporary serialization, Sec.
// 5.2) and chunks of c tokens, their intermediates and the residual stream at
// the offsets of the step's static layout (Algorithm 1, Sec. 6.1), and the
// offloaded blocks' weights prefetched from pinned host memory into device
// staging slots on a copy stream while earlier blocks compute (selective
// offloading, Sec. 5.1).  The plans come from step_plan.cpp.
#include <algorithm>
#include <cstring>
#include <vector>

#include "kernels.h"
#include "xema_internal.h"
#include "xema_step.h"

using namespace xema;

namespace {

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

bool overlaps(const void* a, int64_t an, const void* b, int64_t bn) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + (uintptr_t)bn && b0 < a0 + (uintptr_t)an;
}

const void* tensor(const xema_block_weights& w, int i) { return weight_ptrs(w)[i]; }

xema_block_weights packed_weights(uint8_t* slot, const int64_t off[kWeightTensors]) {
  xema_block_weights w;
  const void** p = weight_ptrs(w);
  for (int i = 0; i < kWeightTensors; ++i) p[i] = slot + off[i];
  return w;
}

// The step with offload plan `op`, groups of g sequences and chunks of ch
// tokens; arguments other than the plan are validated here.
int run_step(const xema_block_cfg& c, const xema_request& r, const void* tokens,
             const xema_block_weights* weights, const xema_offload_plan& op, int g, int64_t ch,
             const void* cond, void* workspace, int64_t workspace_bytes, void* out, void* stream,
             void* copy_stream) {
  if (!tokens || !weights || !cond || !workspace || !out || workspace_bytes <= 0)
    return XEMA_ERR_INVALID_ARG;
  const int N = op.n_blocks, K = op.n_offloaded, S = op.n_staging;
  StepLayout lay;
  int st = step_layout(c, r, N, g, ch, S, op.block_weight_bytes, &lay);
  if (st != XEMA_OK) return st;
  if (workspace_bytes < lay.peak) return XEMA_ERR_WORKSPACE_TOO_SMALL;

  int64_t wb[kWeightTensors];
  block_weight_sizes(c, wb);
  for (int i = 0; i < N; ++i)
    for (int t = 0; t < kWeightTensors; ++t) {
      if (!wb[t]) continue;  // a tensor the block does not use
      const void* p = tensor(weights[i], t);
      if (!p) return XEMA_ERR_INVALID_ARG;
      if (!aligned(p, 16)) return XEMA_ERR_MISALIGNED;
    }
  if (!aligned(tokens, 16) || !aligned(cond, 16) || !aligned(out, 16)) return XEMA_ERR_MISALIGNED;
  if (!aligned(workspace, 256)) return XEMA_ERR_MISALIGNED;

  const int64_t B = r.batch, L = seq_len(r), D = c.hidden, Dc = c.cond_dim;
  const int64_t out_bytes = B * L * D * 4;
  if (overlaps(out, out_bytes, tokens, B * L * D * 2) || overlaps(out, out_bytes, cond, B * Dc * 2) ||
      overlaps(out, out_bytes, workspace, workspace_bytes) ||
      overlaps(workspace, workspace_bytes, tokens, B * L * D * 2) ||
      overlaps(workspace, workspace_bytes, cond, B * Dc * 2))
    return XEMA_ERR_INVALID_ARG;
  for (int i = 0; i < N; ++i) {
    if (op.offloaded[i]) continue;  // host memory cannot alias device buffers
    for (int t = 0; t < kWeightTensors; ++t) {
      const void* p = tensor(weights[i], t);
      if (wb[t] && (overlaps(out, out_bytes, p, wb[t]) || overlaps(workspace, workspace_bytes, p, wb[t])))
        return XEMA_ERR_INVALID_ARG;
    }
  }

  uint8_t* ws = (uint8_t*)workspace;
  int64_t off[kWeightTensors];
  packed_offsets(c, off);
  const hipStream_t s = (hipStream_t)stream;
  const hipStream_t cs = (hipStream_t)copy_stream;
  const bool overlap = K > 0 && cs != nullptr && cs != s;
  xema_request rg = r;
  rg.batch = g;

  std::vector<int> offloaded;  // the offloaded blocks, by ordinal
  for (int i = 0; i < N; ++i)
    if (op.offloaded[i]) offloaded.push_back(i);
  auto staging = [&](int k) { return ws + lay.staging_off[(size_t)(k % S)]; };

  std::vector<hipEvent_t> events;
  auto new_event = [&](hipEvent_t* e) {
    if (hipEventCreateWithFlags(e, hipEventDisableTiming) != hipSuccess) return false;
    events.push_back(*e);
    return true;
  };
  auto release = [&](int status) {
    for (hipEvent_t e : events) (void)hipEventDestroy(e);  // released once complete
    return status;
  };
  // copy offloaded block #k (ordinal) into its staging slot on stream q
  auto copy_in = [&](int k, hipStream_t q) {
    uint8_t* slot = staging(k);
    const xema_block_weights& w = weights[offloaded[(size_t)k]];
    for (int t = 0; t < kWeightTensors; ++t)
      if (wb[t] &&
          hipMemcpyAsync(slot + off[t], tensor(w, t), wb[t], hipMemcpyHostToDevice, q) != hipSuccess)
        return false;
    return true;
  };

  std::vector<hipEvent_t> ready((size_t)K), freed((size_t)K);
  if (overlap) {
    // the slots may still be read by work queued earlier on `stream`
    hipEvent_t start;
    if (!new_event(&start) || hipEventRecord(start, s) != hipSuccess ||
        hipStreamWaitEvent(cs, start, 0) != hipSuccess)
      return release(XEMA_ERR_HIP);
    for (int k = 0; k < K; ++k)
      if (!new_event(&ready[(size_t)k]) || !new_event(&freed[(size_t)k])) return release(XEMA_ERR_HIP);
    for (int k = 0; k < std::min(S, K); ++k)
      if (!copy_in(k, cs) || hipEventRecord(ready[(size_t)k], cs) != hipSuccess)
        return release(XEMA_ERR_HIP);
  }

  // x_{i+1}, the output of block i: the caller's out when N - 1 - i is even
  // (the last block ends in out), else the workspace's buffer
  auto out_of = [&](int i) {
    return (N - 1 - i) % 2 == 0 ? (float*)out : (float*)(ws + lay.resid_off[(size_t)i]);
  };
  int k = 0;
  for (int i = 0; i < N; ++i) {
    xema_block_weights w = weights[i];
    if (op.offloaded[i]) {
      if (overlap) {
        if (hipStreamWaitEvent(s, ready[(size_t)k], 0) != hipSuccess) return release(XEMA_ERR_HIP);
      } else if (!copy_in(k, s)) {
        return release(XEMA_ERR_HIP);
      }
      w = packed_weights(staging(k), off);
    }
    // block i's slots at its own offsets of the step layout
    xema_plan bp = lay.block;
    for (int sl = 0; sl < XEMA_NUM_SLOTS; ++sl)
      bp.slot_offset[sl] = lay.slot_off[(size_t)i * XEMA_NUM_SLOTS + sl];
    float* dst = out_of(i);
    for (int64_t b0 = 0; b0 < B; b0 += g) {  // the batch in groups of g sequences
      const void* x = i == 0 ? (const void*)((const uint16_t*)tokens + b0 * L * D)
                             : (const void*)(out_of(i - 1) + b0 * L * D);
      st = run_block(c, rg, x, i == 0 ? XEMA_BF16 : XEMA_F32, w, (const uint16_t*)cond + b0 * Dc, ch, ws, bp,
                     dst + b0 * L * D, s, nullptr, b0 == 0);  // each block its own status slot
      if (st != XEMA_OK) return release(st);
    }
    if (op.offloaded[i]) {
      if (overlap && k + S < K) {
        // the slot is refilled with offloaded block #k+S once block i is done
        if (hipEventRecord(freed[(size_t)k], s) != hipSuccess ||
            hipStreamWaitEvent(cs, freed[(size_t)k], 0) != hipSuccess || !copy_in(k + S, cs) ||
            hipEventRecord(ready[(size_t)(k + S)], cs) != hipSuccess)
          return release(XEMA_ERR_HIP);
      }
      ++k;
    }
  }
  return release(XEMA_OK);
}

}  // namespace

extern "C" int xema_dit_step_fwd(const xema_block_cfg* cfg, const xema_request* req,
                                 const void* tokens, const xema_block_weights* weights,
                                 const xema_offload_plan* plan, const void* cond,
                                 int32_t chunk_tokens, void* workspace, int64_t workspace_bytes,
                                 void* out, void* stream, void* copy_stream) {
  int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  st = check_offload_plan(*cfg, plan);
  if (st != XEMA_OK) return st;
  return run_step(*cfg, *req, tokens, weights, *plan, req->batch, effective_chunk(seq_len(*req), chunk_tokens),
                  cond, workspace, workspace_bytes, out, stream, copy_stream);
}

extern "C" int xema_dit_step_fwd_planned(const xema_block_cfg* cfg, const xema_request* req,
                                         const void* tokens, const xema_block_weights* weights,
                                         const xema_step_plan* plan, const void* cond, void* workspace,
                                         int64_t workspace_bytes, void* out, void* stream, void* copy_stream) {
  int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  if (!plan) return XEMA_ERR_INVALID_ARG;
  st = check_offload_plan(*cfg, &plan->offload);
  if (st != XEMA_OK) return st;
  const int g = plan->batch_group;
  if (g < 1 || g > req->batch || req->batch % g) return XEMA_ERR_INVALID_ARG;
  // the plan must be the one the library makes for these choices
  const xema_step_costs unit{1.0, 1.0};  // the rates change only est_ms
  xema_step_plan ref;
  st = make_step_plan(*cfg, *req, plan->offload.n_blocks, plan->offload.n_offloaded,
                      std::max(plan->offload.n_staging, 1), g, plan->chunk_tokens, unit, &ref);
  if (st != XEMA_OK) return st;
  if (ref.chunk_tokens != plan->chunk_tokens || ref.workspace_bytes != plan->workspace_bytes ||
      ref.device_bytes != plan->device_bytes)
    return XEMA_ERR_INVALID_ARG;
  return run_step(*cfg, *req, tokens, weights, plan->offload, g, plan->chunk_tokens, cond, workspace,
                  workspace_bytes, out, stream, copy_stream);
}
