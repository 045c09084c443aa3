// Host-side planning: the block's slot table, the offline static layout of
// Algorithm 1 (Sec. 6.1) and the "only as much mitigation as needed" chunk
// choice (Sec. 5.1, objective pi*).  Pure C++; no device calls.
#include <algorithm>
#include <cstring>
#include <vector>

#include "xema_internal.h"

namespace xema {

// Algorithm 1: largest tensor first (ties: earlier lifetime start, then id);
// each tensor goes to the bottom of the smallest gap, among the holes left by
// already-placed tensors with overlapping lifetimes, that can hold it (ties:
// lower address); with no such gap it goes right above those tensors.  The
// placed tensors alive at each step are kept in per-step lists, so the
// tensors whose lifetimes overlap the next one are found without scanning
// every placed tensor (the set, and so the placement, is the same).
int64_t static_layout(const std::vector<LayoutRect>& rects, std::vector<int64_t>* offsets) {
  const size_t n = rects.size();
  std::vector<size_t> order(n);
  int horizon = 0;
  for (size_t i = 0; i < n; ++i) {
    order[i] = i;
    horizon = std::max(horizon, rects[i].end);
  }
  std::sort(order.begin(), order.end(), [&](size_t x, size_t y) {
    if (rects[x].size != rects[y].size) return rects[x].size > rects[y].size;
    if (rects[x].begin != rects[y].begin) return rects[x].begin < rects[y].begin;
    return rects[x].id < rects[y].id;
  });
  offsets->assign(n, -1);
  std::vector<std::vector<size_t>> alive((size_t)std::max(horizon, 0));
  std::vector<size_t> seen(n, (size_t)-1);
  std::vector<std::pair<int64_t, int64_t>> busy;
  for (size_t i : order) {
    busy.clear();
    for (int t = std::max(rects[i].begin, 0); t < rects[i].end; ++t)
      for (size_t j : alive[(size_t)t])
        if (seen[j] != i) {
          seen[j] = i;
          busy.emplace_back((*offsets)[j], (*offsets)[j] + rects[j].size);
        }
    std::sort(busy.begin(), busy.end());
    int64_t cursor = 0, top = 0;
    int64_t best_addr = -1, best_len = 0;
    for (const auto& iv : busy) {
      if (iv.first > cursor) {
        const int64_t len = iv.first - cursor;
        if (len >= rects[i].size && (best_addr < 0 || len < best_len)) {
          best_addr = cursor;
          best_len = len;
        }
      }
      cursor = std::max(cursor, iv.second);
      top = std::max(top, iv.second);
    }
    (*offsets)[i] = best_addr >= 0 ? best_addr : top;
    for (int t = std::max(rects[i].begin, 0); t < rects[i].end; ++t) alive[(size_t)t].push_back(i);
  }
  int64_t peak = 0;
  for (size_t i = 0; i < n; ++i) peak = std::max(peak, (*offsets)[i] + rects[i].size);
  return peak;
}

namespace {

int64_t rope_table_bytes(const xema_block_cfg& cfg, const xema_request& req) {
  const int64_t g[3] = {req.grid_t, req.grid_h, req.grid_w};
  int64_t n = 0;
  for (int a = 0; a < 3; ++a) n += g[a] * (cfg.rope_dims[a] / 2);
  return 8 * n;
}

}  // namespace

int validate_shapes(const xema_block_cfg* cfg, const xema_request* req) {
  if (!cfg || !req) return XEMA_ERR_INVALID_ARG;
  const xema_block_cfg& c = *cfg;
  const xema_request& r = *req;
  if (c.hidden <= 0 || c.heads <= 0 || c.head_dim <= 0 || c.mlp_hidden <= 0 || c.cond_dim <= 0)
    return XEMA_ERR_INVALID_ARG;
  if (r.batch <= 0 || r.text_len < 0 || r.grid_t < 0 || r.grid_h < 0 || r.grid_w < 0)
    return XEMA_ERR_INVALID_ARG;
  if ((int64_t)c.heads * c.head_dim != c.hidden) return XEMA_ERR_INVALID_ARG;
  int64_t rope_sum = 0;
  for (int a = 0; a < 3; ++a) {
    if (c.rope_dims[a] < 0 || (c.rope_dims[a] & 1)) return XEMA_ERR_INVALID_ARG;
    rope_sum += c.rope_dims[a];
  }
  if (rope_sum > c.head_dim) return XEMA_ERR_INVALID_ARG;
  if (!(c.rope_theta > 0.f) || !(c.ln_eps > 0.f) || !(c.qk_eps > 0.f)) return XEMA_ERR_INVALID_ARG;
  if (c.modulation_streams < 0 || c.modulation_streams > 2) return XEMA_ERR_INVALID_ARG;
  if (c.weights_f16 != 0 && c.weights_f16 != 1) return XEMA_ERR_INVALID_ARG;
  const int64_t L = seq_len(r);
  if (L <= 0) return XEMA_ERR_INVALID_ARG;
  // what the kernels handle
  if (c.head_dim != 64 && c.head_dim != 128) return XEMA_ERR_UNSUPPORTED;
  if (c.hidden % 256 != 0 || c.hidden > 8192) return XEMA_ERR_UNSUPPORTED;
  if (c.mlp_hidden % 256 != 0) return XEMA_ERR_UNSUPPORTED;
  if (c.cond_dim % 8 != 0) return XEMA_ERR_UNSUPPORTED;
  if (L > (int64_t)1 << 30 || (int64_t)r.batch * L > (int64_t)1 << 31) return XEMA_ERR_UNSUPPORTED;
  return XEMA_OK;
}

void block_weight_sizes(const xema_block_cfg& c, int64_t bytes[kWeightTensors]) {
  const int64_t D = c.hidden, F = c.mlp_hidden, Dc = c.cond_dim, d = c.head_dim;
  const int64_t t = dual_stream(c) ? 1 : 0;
  const int64_t b[kWeightTensors] = {6 * D * Dc * 2, 6 * D * 2, 3 * D * D * 2, 3 * D * 2,
                                     d * 2,          d * 2,     D * D * 2,     D * 2,
                                     F * D * 2,      F * 2,     D * F * 2,     D * 2,
                                     t * 6 * D * Dc * 2, t * 6 * D * 2};
  for (int i = 0; i < kWeightTensors; ++i) bytes[i] = b[i];
}

int layout_for_chunk(const xema_block_cfg& cfg, const xema_request& req, int64_t c,
                     xema_plan* out) {
  const int64_t B = req.batch, D = cfg.hidden, F = cfg.mlp_hidden;
  const int64_t L = seq_len(req);
  const int64_t lp = padded_len(L);
  const bool chunked = c < L;
  const int64_t copies = cfg.weights_f16 ? 0 : 1;  // fp16 weight copies made by the call
  struct Spec { int64_t bytes; int begin, end; };
  const Spec spec[XEMA_NUM_SLOTS] = {
      {24 * B * D * (dual_stream(cfg) ? 2 : 1), 0, 10},  // XEMA_SLOT_MOD
      {rope_table_bytes(cfg, req), 0, 4},          // XEMA_SLOT_ROPE
      {2 * B * D * lp, 1, 10},                     // XEMA_SLOT_Q
      {2 * B * D * lp, 1, 10},                     // XEMA_SLOT_K
      {2 * B * D * lp, 1, 10},                     // XEMA_SLOT_VT
      {2 * B * c * D, 1, 3},                       // XEMA_SLOT_LN1
      {0, 2, 4},                                   // XEMA_SLOT_QKV: the QKV GEMM writes the heads itself
      {copies * 2 * D * D, 4, 10},                 // XEMA_SLOT_WO16
      {copies * 2 * F * D, 4, 10},                 // XEMA_SLOT_WUP16
      {copies * 2 * D * F, 4, 10},                 // XEMA_SLOT_WDOWN16
      {2 * B * c * D, 5, chunked ? 10 : 7},        // XEMA_SLOT_ATTN
      {4 * B * c * D, 6, 10},                      // XEMA_SLOT_X1
      {2 * B * c * D, 7, 9},                       // XEMA_SLOT_LN2
      {2 * B * c * F, 8, 10},                      // XEMA_SLOT_HID
      {4 * XEMA_STATUS_WORDS, 0, 10},              // XEMA_SLOT_STATUS
  };
  std::vector<LayoutRect> rects;
  for (int i = 0; i < XEMA_NUM_SLOTS; ++i)
    rects.push_back({i, round_up(spec[i].bytes, kAlign), spec[i].begin, spec[i].end});
  std::vector<int64_t> offsets;
  const int64_t peak = static_layout(rects, &offsets);
  std::memset(out, 0, sizeof(*out));
  out->chunk_tokens = (int32_t)c;
  out->n_slots = XEMA_NUM_SLOTS;
  out->workspace_bytes = peak;
  for (int i = 0; i < XEMA_NUM_SLOTS; ++i) {
    out->slot_offset[i] = offsets[i];
    out->slot_bytes[i] = rects[i].size;
    out->slot_begin[i] = rects[i].begin;
    out->slot_end[i] = rects[i].end;
  }
  return XEMA_OK;
}

}  // namespace xema

using namespace xema;

extern "C" int xema_request_from_template(const xema_block_cfg* cfg, int32_t height,
                                          int32_t width, int32_t frames, int32_t batch,
                                          int32_t text_len, xema_request* out) {
  if (!cfg || !out || height <= 0 || width <= 0 || frames <= 0 || batch <= 0 || text_len < 0)
    return XEMA_ERR_INVALID_ARG;
  out->batch = batch;
  out->text_len = text_len;
  out->grid_h = (height + 15) / 16;
  out->grid_w = (width + 15) / 16;
  out->grid_t = (frames - 1) / 4 + 1;
  return XEMA_OK;
}

extern "C" int xema_workspace_layout(const xema_block_cfg* cfg, const xema_request* req,
                                     int32_t chunk_tokens, xema_plan* out) {
  if (!out) return XEMA_ERR_INVALID_ARG;
  const int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  const int64_t L = seq_len(*req);
  int rc = layout_for_chunk(*cfg, *req, effective_chunk(L, chunk_tokens), out);
  if (rc != XEMA_OK) return rc;
  xema_plan smallest;
  rc = layout_for_chunk(*cfg, *req, std::min<int64_t>(L, XEMA_CHUNK_GRANULE), &smallest);
  out->min_workspace_bytes = smallest.workspace_bytes;
  return rc;
}

extern "C" int xema_workspace_bytes(const xema_block_cfg* cfg, const xema_request* req,
                                    int32_t chunk_tokens, int64_t* bytes) {
  if (!bytes) return XEMA_ERR_INVALID_ARG;
  xema_plan p;
  const int rc = xema_workspace_layout(cfg, req, chunk_tokens, &p);
  if (rc == XEMA_OK) *bytes = p.workspace_bytes;
  return rc;
}

namespace {

// The smallest arena over the candidate chunks.  Usually the smallest chunk's,
// but on short sequences a chunked layout (whose attention buffer stays live
// through the MLP) can exceed the unchunked one.
int64_t min_arena(const xema_block_cfg& cfg, const xema_request& req, const std::vector<int64_t>& cands) {
  int64_t best = -1;
  for (int64_t c : cands) {
    xema_plan p;
    layout_for_chunk(cfg, req, c, &p);
    if (best < 0 || p.workspace_bytes < best) best = p.workspace_bytes;
  }
  return best;
}

}  // namespace

extern "C" int xema_workspace_plan(const xema_block_cfg* cfg, const xema_request* req,
                                   int64_t budget_bytes, xema_plan* out) {
  if (!out) return XEMA_ERR_INVALID_ARG;
  const int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  const int64_t L = seq_len(*req);
  // candidates, largest first: L itself, then every granule multiple below L
  std::vector<int64_t> cands{L};
  for (int64_t c = (L - 1) / XEMA_CHUNK_GRANULE * XEMA_CHUNK_GRANULE; c > 0; c -= XEMA_CHUNK_GRANULE)
    cands.push_back(c);
  const int64_t smallest = min_arena(*cfg, *req, cands);
  for (int64_t c : cands) {
    xema_plan p;
    layout_for_chunk(*cfg, *req, c, &p);
    if (p.workspace_bytes <= budget_bytes) {
      *out = p;
      out->min_workspace_bytes = smallest;
      return XEMA_OK;
    }
  }
  std::memset(out, 0, sizeof(*out));
  out->min_workspace_bytes = smallest;
  return XEMA_ERR_BUDGET_TOO_SMALL;
}

// The rate the ranking of xema_workspace_plan_serial assumes; any positive
// value gives the same ranking, since the model's time is proportional to it.
constexpr double kPlanTflops = 1000.0;

extern "C" int xema_workspace_plan_serial(const xema_block_cfg* cfg, const xema_request* req,
                                          int64_t budget_bytes, int32_t* batch_group,
                                          xema_plan* out) {
  if (!out || !batch_group) return XEMA_ERR_INVALID_ARG;
  const int st = validate_shapes(cfg, req);
  if (st != XEMA_OK) return st;
  *batch_group = 0;
  const int64_t L = seq_len(*req);
  std::vector<int64_t> cands{L};
  for (int64_t c = (L - 1) / XEMA_CHUNK_GRANULE * XEMA_CHUNK_GRANULE; c > 0; c -= XEMA_CHUNK_GRANULE)
    cands.push_back(c);
  // For each group size g the largest chunk whose arena fits (a smaller
  // chunk never shortens the modelled time); among those the least modelled
  // time of the block (block_ms), then the larger g.  Neither groups nor
  // chunks ever remove a round of the model, so with an ample budget this
  // is (batch, L): no mitigation at all.
  double best_ms = 0.0;
  for (int32_t g = req->batch; g >= 1; --g) {
    if (req->batch % g) continue;  // equal groups only
    xema_request rg = *req;
    rg.batch = g;
    for (int64_t c : cands) {
      xema_plan pg;
      layout_for_chunk(*cfg, rg, c, &pg);
      if (pg.workspace_bytes <= budget_bytes) {
        const double ms = block_ms(*cfg, *req, g, c, kPlanTflops);
        if (*batch_group == 0 || ms < best_ms * (1.0 - 1e-12)) {
          *out = pg;
          *batch_group = g;
          best_ms = ms;
        }
        break;  // the largest fitting chunk for this g
      }
    }
  }
  xema_request r1 = *req;
  r1.batch = 1;
  const int64_t smallest = min_arena(*cfg, r1, cands);
  if (*batch_group == 0) {
    std::memset(out, 0, sizeof(*out));
    out->min_workspace_bytes = smallest;
    return XEMA_ERR_BUDGET_TOO_SMALL;
  }
  out->min_workspace_bytes = smallest;
  return XEMA_OK;
}

extern "C" const char* xema_status_str(int status) {
  switch (status) {
    case XEMA_OK: return "ok";
    case XEMA_ERR_INVALID_ARG: return "invalid argument";
    case XEMA_ERR_UNSUPPORTED: return "unsupported shape";
    case XEMA_ERR_BUDGET_TOO_SMALL: return "activation budget too small";
    case XEMA_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case XEMA_ERR_MISALIGNED: return "misaligned pointer";
    case XEMA_ERR_HIP: return "HIP error";
    case XEMA_ERR_RANGE: return "an fp16 intermediate left its range";
    default: return "unknown status";
  }
}
