// Host-side planning of the N-block denoising step (xema_step.h), pure C++:
//   - selective offloading: the K offloaded blocks spread uniformly over the
//     stack (Sec. 5.1, "Selective offloading and HSDP");
//   - the step's static layout: Algorithm 1 (Sec. 6.1) over the lifetime
//     trace of the whole step, written out from the block's slot table
//     instead of recorded from a shape-only run (Sec. 7.2, memory analyzer);
//   - the choice of offloading, temporary serialization and chunking under
//     one device budget by the least modelled latency (Sec. 5.1, pi*).
#include <algorithm>
#include <cstring>
#include <map>
#include <tuple>
#include <vector>

#include "xema_internal.h"
#include "xema_step.h"

namespace xema {

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

int validate_cfg(const xema_block_cfg* cfg) {
  xema_request one{1, 1, 0, 0, 0};
  return validate_shapes(cfg, &one);
}

void fill_offload_plan(const xema_block_cfg& c, int n, int k, int staging, xema_offload_plan* out) {
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

int check_offload_plan(const xema_block_cfg& c, const xema_offload_plan* plan) {
  if (!plan || plan->n_blocks < 1 || plan->n_blocks > XEMA_MAX_BLOCKS) return XEMA_ERR_INVALID_ARG;
  if (plan->n_offloaded < 0 || plan->n_offloaded > plan->n_blocks ||
      (plan->n_offloaded > 0 && plan->n_staging < 1))
    return XEMA_ERR_INVALID_ARG;
  xema_offload_plan ref;
  fill_offload_plan(c, plan->n_blocks, plan->n_offloaded, std::max(plan->n_staging, 1), &ref);
  if (std::memcmp(&ref, plan, sizeof(ref)) != 0)
    return XEMA_ERR_INVALID_ARG;  // not a plan the library made for this configuration
  return XEMA_OK;
}

int step_layout(const xema_block_cfg& c, const xema_request& r, int n_blocks, int group, int64_t chunk,
                int n_staging, int64_t slot_bytes, StepLayout* out) {
  xema_request rg = r;
  rg.batch = group;
  const int64_t L = seq_len(r);
  const int st = layout_for_chunk(c, rg, effective_chunk(L, chunk), &out->block);
  if (st != XEMA_OK) return st;
  const int N = n_blocks, NS = XEMA_NUM_SLOTS;
  std::vector<LayoutRect> rects;
  std::vector<std::pair<int, int>> what;  // (kind 0 slot / 1 residual / 2 staging, index)
  // block i's slots at steps 10 i + (the block's own steps)
  for (int i = 0; i < N; ++i)
    for (int s = 0; s < NS; ++s)
      if (out->block.slot_bytes[s] > 0) {
        rects.push_back({i * NS + s, out->block.slot_bytes[s], 10 * i + out->block.slot_begin[s],
                         10 * i + out->block.slot_end[s]});
        what.emplace_back(0, i * NS + s);
      }
  // x_{i+1}, written by block i at its step 9 and read by block i+1 through
  // its last step; the workspace holds it when N - 1 - i is odd, the
  // caller's out otherwise.  Step 9 repeats for every chunk (phase B, steps
  // 5-9) and the whole block for every group, so the first write comes
  // before later chunks or groups use the block's other slots: the buffer
  // is live from the first step of the loop that writes it (5 when chunked,
  // 0 with several groups, 9 for one unchunked pass).
  const int64_t resid = round_up((int64_t)r.batch * L * c.hidden * 4, kAlign);
  const int first = group < r.batch ? 0 : effective_chunk(L, chunk) < L ? 5 : 9;
  for (int i = 0; i + 1 < N; ++i)
    if ((N - 1 - i) % 2 == 1) {
      rects.push_back({N * NS + i, resid, 10 * i + first, 10 * i + 20});
      what.emplace_back(1, i);
    }
  // the staging slots of offloaded weights, live throughout the step
  for (int j = 0; j < n_staging; ++j) {
    rects.push_back({N * NS + N + j, round_up(slot_bytes, kAlign), 0, 10 * N});
    what.emplace_back(2, j);
  }
  std::vector<int64_t> offsets;
  out->peak = static_layout(rects, &offsets);
  out->slot_off.assign((size_t)N * NS, 0);
  out->resid_off.assign((size_t)N, -1);
  out->staging_off.assign((size_t)n_staging, -1);
  for (size_t k = 0; k < rects.size(); ++k) {
    if (what[k].first == 0) out->slot_off[(size_t)what[k].second] = offsets[k];
    else if (what[k].first == 1) out->resid_off[(size_t)what[k].second] = offsets[k];
    else out->staging_off[(size_t)what[k].second] = offsets[k];
  }
  return XEMA_OK;
}

// Modelled time of one block (all its groups and chunks), milliseconds: the
// rounds of workgroups of each launch over the 256 CUs, a round costing one
// workgroup's FLOPs at block_tflops / 256 per CU.
double block_ms(const xema_block_cfg& c, const xema_request& r, int64_t g, int64_t ch, double tflops) {
  const int64_t B = r.batch, L = seq_len(r), D = c.hidden, F = c.mlp_hidden, H = c.heads, d = c.head_dim;
  const int64_t qwg = d == 64 ? 512 : 256;  // queries per attention workgroup
  auto rounds = [](int64_t wgs) { return (double)((wgs + 255) / 256); };
  auto gemm = [&](int64_t M, int64_t N, int64_t K) {
    return rounds((M + 255) / 256 * (N / 256)) * 2.0 * 256.0 * 256.0 * (double)K;
  };
  double flops = 0.0;  // FLOPs of the rounds, per CU
  for (int64_t t0 = 0; t0 < L; t0 += ch) {
    const int64_t ck = std::min(ch, L - t0), M = g * ck;
    flops += gemm(M, 3 * D, D) + gemm(M, D, D) + gemm(M, F, D) + gemm(M, D, F);
    flops += rounds((ck + qwg - 1) / qwg * H * g) * 4.0 * (double)qwg * (double)L * (double)d;
  }
  return flops * (double)(B / g) / (tflops * 1e12 / 256.0) * 1e3;
}

namespace {

bool costs_ok(const xema_step_costs* k) {
  return k && k->h2d_gbytes_per_s > 0.0 && k->block_tflops > 0.0;
}

// End of the last block: the copy stream runs the copies of the offloaded
// blocks in order, copy k starting when copy k-1 is done and the block that
// used its staging slot (offloaded block k - S) has finished; a block
// starts when its predecessor has finished and, if offloaded, its copy.
double step_ms(const xema_offload_plan& op, double t_blk, double t_x) {
  const int N = op.n_blocks, S = std::max(op.n_staging, 1);
  std::vector<int> blk;
  for (int i = 0; i < N; ++i)
    if (op.offloaded[i]) blk.push_back(i);
  std::vector<double> block_end((size_t)N, 0.0), copy_end(blk.size(), 0.0);
  double t = 0.0, copy_free = 0.0;
  size_t k = 0, next_copy = 0;
  for (int i = 0; i < N; ++i) {
    double start = t;
    if (op.offloaded[i]) {
      for (; next_copy <= k; ++next_copy) {
        double ready = copy_free;
        if (next_copy >= (size_t)S) ready = std::max(ready, block_end[(size_t)blk[next_copy - S]]);
        copy_free = ready + t_x;
        copy_end[next_copy] = copy_free;
      }
      start = std::max(start, copy_end[k]);
      ++k;
    }
    block_end[(size_t)i] = start + t_blk;
    t = block_end[(size_t)i];
  }
  return t;
}

int check_step_args(const xema_block_cfg* cfg, const xema_request* req, int32_t n_blocks, int32_t n_staging,
                    const xema_step_costs* costs, const xema_step_plan* out) {
  if (!out || !costs_ok(costs) || n_blocks < 1 || n_blocks > XEMA_MAX_BLOCKS || n_staging < 1)
    return XEMA_ERR_INVALID_ARG;
  return validate_shapes(cfg, req);
}

}  // namespace

int make_step_plan(const xema_block_cfg& c, const xema_request& r, int n_blocks, int n_offloaded, int n_staging,
                   int group, int64_t chunk, const xema_step_costs& costs, xema_step_plan* out) {
  std::memset(out, 0, sizeof(*out));
  fill_offload_plan(c, n_blocks, n_offloaded, n_staging, &out->offload);
  const int64_t L = seq_len(r), ch = effective_chunk(L, chunk);
  StepLayout lay;
  const int st = step_layout(c, r, n_blocks, group, ch, out->offload.n_staging, out->offload.block_weight_bytes,
                             &lay);
  if (st != XEMA_OK) return st;
  out->batch_group = group;
  out->chunk_tokens = (int32_t)ch;
  out->workspace_bytes = lay.peak;
  out->device_bytes = out->offload.resident_weight_bytes + lay.peak;
  const double t_x = (double)out->offload.block_weight_bytes / (costs.h2d_gbytes_per_s * 1e9) * 1e3;
  out->est_ms = step_ms(out->offload, block_ms(c, r, group, ch, costs.block_tflops), t_x);
  return XEMA_OK;
}

}  // namespace xema

using namespace xema;

extern "C" int xema_offload_plan_k(const xema_block_cfg* cfg, int32_t n_blocks, int32_t n_offloaded,
                                   int32_t n_staging, xema_offload_plan* out) {
  if (!cfg || !out || n_blocks < 1 || n_blocks > XEMA_MAX_BLOCKS || n_offloaded < 0 ||
      n_offloaded > n_blocks || n_staging < 1)
    return XEMA_ERR_INVALID_ARG;
  const int st = validate_cfg(cfg);
  if (st != XEMA_OK) return st;
  fill_offload_plan(*cfg, n_blocks, n_offloaded, n_staging, out);
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
    fill_offload_plan(*cfg, n_blocks, k, n_staging, out);
    if (out->device_weight_bytes <= weight_budget_bytes) return XEMA_OK;
  }
  fill_offload_plan(*cfg, n_blocks, n_blocks, n_staging, out);
  return XEMA_ERR_BUDGET_TOO_SMALL;
}

extern "C" int xema_step_workspace_bytes(const xema_block_cfg* cfg, const xema_request* req,
                                         int32_t chunk_tokens, const xema_offload_plan* plan,
                                         int64_t* bytes) {
  int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  if (!bytes) return XEMA_ERR_INVALID_ARG;
  st = check_offload_plan(*cfg, plan);
  if (st != XEMA_OK) return st;
  StepLayout lay;
  st = step_layout(*cfg, *req, plan->n_blocks, req->batch, effective_chunk(seq_len(*req), chunk_tokens),
                   plan->n_staging, plan->block_weight_bytes, &lay);
  if (st == XEMA_OK) *bytes = lay.peak;
  return st;
}

extern "C" int xema_step_plan_fixed(const xema_block_cfg* cfg, const xema_request* req, int32_t n_blocks,
                                    int32_t n_offloaded, int32_t n_staging, int32_t batch_group,
                                    int32_t chunk_tokens, const xema_step_costs* costs, xema_step_plan* out) {
  int st = check_step_args(cfg, req, n_blocks, n_staging, costs, out);
  if (st != XEMA_OK) return st;
  if (n_offloaded < 0 || n_offloaded > n_blocks || batch_group < 1 || batch_group > req->batch ||
      req->batch % batch_group)
    return XEMA_ERR_INVALID_ARG;
  return make_step_plan(*cfg, *req, n_blocks, n_offloaded, n_staging, batch_group, chunk_tokens, *costs, out);
}

extern "C" int xema_step_plan_budget(const xema_block_cfg* cfg, const xema_request* req, int32_t n_blocks,
                                     int32_t n_staging, int64_t device_budget_bytes,
                                     const xema_step_costs* costs, xema_step_plan* out) {
  int st = check_step_args(cfg, req, n_blocks, n_staging, costs, out);
  if (st != XEMA_OK) return st;
  if (device_budget_bytes < 0) return XEMA_ERR_INVALID_ARG;
  const xema_block_cfg& c = *cfg;
  const xema_request& r = *req;
  const int64_t B = r.batch, L = seq_len(r);
  std::vector<int64_t> cands{L};
  for (int64_t ch = (L - 1) / XEMA_CHUNK_GRANULE * XEMA_CHUNK_GRANULE; ch > 0; ch -= XEMA_CHUNK_GRANULE)
    cands.push_back(ch);
  std::vector<int> groups;
  for (int g = (int)B; g >= 1; --g)
    if (B % g == 0) groups.push_back(g);
  // the step's workspace for (group, chunk, staging slots), laid out on demand
  std::map<std::tuple<int, int64_t, int>, int64_t> ws_cache;
  std::map<std::pair<int, int64_t>, double> blk_cache;
  xema_offload_plan any;
  fill_offload_plan(c, n_blocks, 0, n_staging, &any);
  const int64_t slot = any.block_weight_bytes;
  auto workspace = [&](int g, int64_t ch, int s, int64_t* bytes) -> int {
    const auto key = std::make_tuple(g, ch, s);
    auto it = ws_cache.find(key);
    if (it == ws_cache.end()) {
      StepLayout lay;
      const int e = step_layout(c, r, n_blocks, g, ch, s, slot, &lay);
      if (e != XEMA_OK) return e;
      it = ws_cache.emplace(key, lay.peak).first;
    }
    *bytes = it->second;
    return XEMA_OK;
  };
  const double t_x = (double)slot / (costs->h2d_gbytes_per_s * 1e9) * 1e3;
  bool found = false;
  int64_t least = -1;
  std::tuple<double, int, int, int64_t> best{0.0, 0, 0, 0};  // (est, K, -g, -c)
  xema_step_plan pick;
  std::memset(&pick, 0, sizeof(pick));
  for (int k = 0; k <= n_blocks; ++k) {
    xema_offload_plan op;
    fill_offload_plan(c, n_blocks, k, n_staging, &op);
    for (int g : groups)
      for (int64_t ch : cands) {
        int64_t ws = 0;
        st = workspace(g, ch, op.n_staging, &ws);
        if (st != XEMA_OK) return st;
        const int64_t dev = op.resident_weight_bytes + ws;
        if (least < 0 || dev < least) least = dev;
        if (dev > device_budget_bytes) continue;
        auto bit = blk_cache.find({g, ch});
        if (bit == blk_cache.end())
          bit = blk_cache.emplace(std::make_pair(g, ch), block_ms(c, r, g, ch, costs->block_tflops)).first;
        const double est = step_ms(op, bit->second, t_x);
        const auto key = std::make_tuple(est, k, -g, -ch);
        if (!found || key < best) {
          found = true;
          best = key;
          pick.offload = op;
          pick.batch_group = g;
          pick.chunk_tokens = (int32_t)ch;
          pick.workspace_bytes = ws;
          pick.device_bytes = dev;
          pick.est_ms = est;
        }
      }
  }
  if (!found) {
    std::memset(out, 0, sizeof(*out));
    out->device_bytes = least;
    return XEMA_ERR_BUDGET_TOO_SMALL;
  }
  *out = pick;
  return XEMA_OK;
}
