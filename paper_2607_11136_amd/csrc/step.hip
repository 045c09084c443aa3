// Host driver of the N-block denoising step with selective weight
// offloading (xema_step.h): offload planning (Sec. 5.1, pi* with offloading
// as the mitigation, K offloaded blocks spread uniformly) and the step itself,
// which prefetches each offloaded block's weights from pinned host memory into
// a device staging slot on a copy stream while earlier blocks compute.
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

// Offsets of the block's tensors packed in a staging slot (a tensor the block
// does not use takes no space); returns the slot size.
int64_t packed_offsets(const xema_block_cfg& c, int64_t off[kWeightTensors]) {
  int64_t b[kWeightTensors];
  block_weight_sizes(c, b);
  int64_t pos = 0;
  for (int i = 0; i < kWeightTensors; ++i) {
    off[i] = pos;
    pos += round_up(b[i], kAlign);
  }
  return pos;
}

// The block hyper-parameters alone (a one-token request stands in for the
// request, which offload planning does not need).
int validate_cfg(const xema_block_cfg* cfg) {
  xema_request one{1, 1, 0, 0, 0};
  return validate_shapes(cfg, &one);
}

void fill_plan(const xema_block_cfg& c, int n, int k, int staging, xema_offload_plan* out) {
  std::memset(out, 0, sizeof(*out));
  int64_t off[kWeightTensors], b[kWeightTensors];
  const int64_t slot = packed_offsets(c, off);
  block_weight_sizes(c, b);
  int64_t sum = 0;
  for (int i = 0; i < kWeightTensors; ++i) sum += b[i];
  out->n_blocks = n;
  out->n_offloaded = k;
  out->n_staging = k > 0 ? std::min(staging, k) : 0;
  // the j-th offloaded block ends the j-th of K equal spans of the stack
  for (int j = 0; j < k; ++j) out->offloaded[(int)((int64_t)(j + 1) * n / k) - 1] = 1;
  out->block_weight_bytes = slot;
  out->resident_weight_bytes = (int64_t)(n - k) * sum;
  out->staging_bytes = (int64_t)out->n_staging * slot;
  out->device_weight_bytes = out->resident_weight_bytes + out->staging_bytes;
}

const void* tensor(const xema_block_weights& w, int i) { return weight_ptrs(w)[i]; }

xema_block_weights packed_weights(uint8_t* slot, const int64_t off[kWeightTensors]) {
  xema_block_weights w;
  const void** p = weight_ptrs(w);
  for (int i = 0; i < kWeightTensors; ++i) p[i] = slot + off[i];
  return w;
}

}  // namespace

extern "C" int xema_offload_plan_k(const xema_block_cfg* cfg, int32_t n_blocks, int32_t n_offloaded,
                                   int32_t n_staging, xema_offload_plan* out) {
  if (!cfg || !out || n_blocks < 1 || n_blocks > XEMA_MAX_BLOCKS || n_offloaded < 0 ||
      n_offloaded > n_blocks || n_staging < 1)
    return XEMA_ERR_INVALID_ARG;
  const int st = validate_cfg(cfg);
  if (st != XEMA_OK) return st;
  fill_plan(*cfg, n_blocks, n_offloaded, n_staging, out);
  return XEMA_OK;
}

extern "C" int xema_offload_plan_budget(const xema_block_cfg* cfg, int32_t n_blocks,
                                        int64_t weight_budget_bytes, int32_t n_staging,
                                        xema_offload_plan* out) {
  if (!cfg || !out || n_blocks < 1 || n_blocks > XEMA_MAX_BLOCKS || n_staging < 1 ||
      weight_budget_bytes < 0)
    return XEMA_ERR_INVALID_ARG;
  const int st = validate_cfg(cfg);
  if (st != XEMA_OK) return st;
  for (int k = 0; k <= n_blocks; ++k) {
    fill_plan(*cfg, n_blocks, k, n_staging, out);
    if (out->device_weight_bytes <= weight_budget_bytes) return XEMA_OK;
  }
  fill_plan(*cfg, n_blocks, n_blocks, n_staging, out);
  return XEMA_ERR_BUDGET_TOO_SMALL;
}

namespace {

int check_plan(const xema_block_cfg& c, const xema_offload_plan* plan) {
  if (!plan || plan->n_blocks < 1 || plan->n_blocks > XEMA_MAX_BLOCKS) return XEMA_ERR_INVALID_ARG;
  xema_offload_plan ref;
  fill_plan(c, plan->n_blocks, plan->n_offloaded, std::max(plan->n_staging, 1), &ref);
  if (plan->n_offloaded < 0 || plan->n_offloaded > plan->n_blocks ||
      (plan->n_offloaded > 0 && plan->n_staging < 1) ||
      std::memcmp(&ref, plan, sizeof(ref)) != 0)
    return XEMA_ERR_INVALID_ARG;  // not a plan the library made for this configuration
  return XEMA_OK;
}

int step_layout(const xema_block_cfg& c, const xema_request& r, int32_t chunk_tokens,
                const xema_offload_plan& plan, xema_plan* arena, int64_t* resid_off,
                int64_t* staging_off, int64_t* total) {
  const int64_t L = seq_len(r);
  const int st = layout_for_chunk(c, r, effective_chunk(L, chunk_tokens), arena);
  if (st != XEMA_OK) return st;
  *resid_off = round_up(arena->workspace_bytes, kAlign);
  *staging_off = *resid_off + round_up((int64_t)r.batch * L * c.hidden * 4, kAlign);
  *total = *staging_off + plan.staging_bytes;
  return XEMA_OK;
}

}  // namespace

extern "C" int xema_step_workspace_bytes(const xema_block_cfg* cfg, const xema_request* req,
                                         int32_t chunk_tokens, const xema_offload_plan* plan,
                                         int64_t* bytes) {
  int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  if (!bytes) return XEMA_ERR_INVALID_ARG;
  st = check_plan(*cfg, plan);
  if (st != XEMA_OK) return st;
  xema_plan arena;
  int64_t ro, so;
  return step_layout(*cfg, *req, chunk_tokens, *plan, &arena, &ro, &so, bytes);
}

extern "C" int xema_dit_step_fwd(const xema_block_cfg* cfg, const xema_request* req,
                                 const void* tokens, const xema_block_weights* weights,
                                 const xema_offload_plan* plan, const void* cond,
                                 int32_t chunk_tokens, void* workspace, int64_t workspace_bytes,
                                 void* out, void* stream, void* copy_stream) {
  int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  if (!tokens || !weights || !cond || !workspace || !out || workspace_bytes <= 0)
    return XEMA_ERR_INVALID_ARG;
  const xema_block_cfg& c = *cfg;
  const xema_request& r = *req;
  st = check_plan(c, plan);
  if (st != XEMA_OK) return st;
  const int N = plan->n_blocks, K = plan->n_offloaded, S = plan->n_staging;
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

  xema_plan arena;
  int64_t resid_off, staging_off, total;
  st = step_layout(c, r, chunk_tokens, *plan, &arena, &resid_off, &staging_off, &total);
  if (st != XEMA_OK) return st;
  if (workspace_bytes < total) return XEMA_ERR_WORKSPACE_TOO_SMALL;

  const int64_t B = r.batch, L = seq_len(r), D = c.hidden, Dc = c.cond_dim;
  const int64_t out_bytes = B * L * D * 4;
  if (overlaps(out, out_bytes, tokens, B * L * D * 2) || overlaps(out, out_bytes, cond, B * Dc * 2) ||
      overlaps(out, out_bytes, workspace, workspace_bytes) ||
      overlaps(workspace, workspace_bytes, tokens, B * L * D * 2) ||
      overlaps(workspace, workspace_bytes, cond, B * Dc * 2))
    return XEMA_ERR_INVALID_ARG;
  for (int i = 0; i < N; ++i) {
    if (plan->offloaded[i]) continue;  // host memory cannot alias device buffers
    for (int t = 0; t < kWeightTensors; ++t) {
      const void* p = tensor(weights[i], t);
      if (wb[t] && (overlaps(out, out_bytes, p, wb[t]) || overlaps(workspace, workspace_bytes, p, wb[t])))
        return XEMA_ERR_INVALID_ARG;
    }
  }

  uint8_t* ws = (uint8_t*)workspace;
  float* resid = (float*)(ws + resid_off);
  uint8_t* staging = ws + staging_off;
  int64_t off[kWeightTensors];
  const int64_t slot_bytes = packed_offsets(c, off);
  const hipStream_t s = (hipStream_t)stream;
  const hipStream_t cs = (hipStream_t)copy_stream;
  const bool overlap = K > 0 && cs != nullptr && cs != s;
  const int64_t ch = effective_chunk(L, chunk_tokens);

  // ordinal of each offloaded block among the offloaded ones
  std::vector<int> offloaded;
  for (int i = 0; i < N; ++i)
    if (plan->offloaded[i]) offloaded.push_back(i);

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
    uint8_t* slot = staging + (int64_t)(k % S) * slot_bytes;
    const xema_block_weights& w = weights[offloaded[k]];
    for (int t = 0; t < kWeightTensors; ++t)
      if (wb[t] &&
          hipMemcpyAsync(slot + off[t], tensor(w, t), wb[t], hipMemcpyHostToDevice, q) != hipSuccess)
        return false;
    return true;
  };

  std::vector<hipEvent_t> ready(K), freed(K);
  if (overlap) {
    // the slots may still be read by work queued earlier on `stream`
    hipEvent_t start;
    if (!new_event(&start) || hipEventRecord(start, s) != hipSuccess ||
        hipStreamWaitEvent(cs, start, 0) != hipSuccess)
      return release(XEMA_ERR_HIP);
    for (int k = 0; k < K; ++k)
      if (!new_event(&ready[k]) || !new_event(&freed[k])) return release(XEMA_ERR_HIP);
    for (int k = 0; k < std::min(S, K); ++k)
      if (!copy_in(k, cs) || hipEventRecord(ready[k], cs) != hipSuccess)
        return release(XEMA_ERR_HIP);
  }

  // residual stream: block i writes buf[(N-1-i) % 2], so the last block ends in out
  float* buf[2] = {(float*)out, resid};
  int k = 0;
  for (int i = 0; i < N; ++i) {
    xema_block_weights w = weights[i];
    if (plan->offloaded[i]) {
      if (overlap) {
        if (hipStreamWaitEvent(s, ready[k], 0) != hipSuccess) return release(XEMA_ERR_HIP);
      } else if (!copy_in(k, s)) {
        return release(XEMA_ERR_HIP);
      }
      w = packed_weights(staging + (int64_t)(k % S) * slot_bytes, off);
    }
    const void* x = i == 0 ? tokens : (const void*)buf[(N - i) % 2];
    st = run_block(c, r, x, i == 0 ? XEMA_BF16 : XEMA_F32, w, cond, ch, ws, arena,
                   buf[(N - 1 - i) % 2], s);
    if (st != XEMA_OK) return release(st);
    if (plan->offloaded[i]) {
      if (overlap && k + S < K) {
        // the slot is refilled with offloaded block #k+S once block i is done
        if (hipEventRecord(freed[k], s) != hipSuccess || hipStreamWaitEvent(cs, freed[k], 0) != hipSuccess ||
            !copy_in(k + S, cs) || hipEventRecord(ready[k + S], cs) != hipSuccess)
          return release(XEMA_ERR_HIP);
      }
      ++k;
    }
  }
  return release(XEMA_OK);
}
