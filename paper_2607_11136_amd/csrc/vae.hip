// Host entry points of the VAE decoder's fused upsampling stage
// (include/xema_vae.h): argument validation, then the launches of k_upconv.hip.
#include "kernels.h"
#include "xema_internal.h"
#include "xema_vae.h"

using namespace xema;

namespace {

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

bool overlaps(const void* a, int64_t an, const void* b, int64_t bn) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + (uintptr_t)bn && b0 < a0 + (uintptr_t)an;
}

int check_channels(int32_t ci, int32_t co) {
  if (ci <= 0 || co <= 0) return XEMA_ERR_INVALID_ARG;
  if (ci % 64 || co % 256) return XEMA_ERR_UNSUPPORTED;
  if ((int64_t)64 * ci * co >= ((int64_t)1 << 31)) return XEMA_ERR_UNSUPPORTED;
  return XEMA_OK;
}

}  // namespace

extern "C" int xema_vae_upconv_weight_bytes(int32_t ci, int32_t co, int64_t* bytes) {
  if (!bytes) return XEMA_ERR_INVALID_ARG;
  const int st = check_channels(ci, co);
  if (st != XEMA_OK) return st;
  *bytes = (int64_t)64 * ci * co;
  return XEMA_OK;
}

extern "C" int xema_vae_upconv_prepare(const void* w, int32_t ci, int32_t co, void* wp, void* stream) {
  if (!w || !wp) return XEMA_ERR_INVALID_ARG;
  const int st = check_channels(ci, co);
  if (st != XEMA_OK) return st;
  if (!aligned(w, 16) || !aligned(wp, 16)) return XEMA_ERR_MISALIGNED;
  if (overlaps(w, (int64_t)18 * ci * co, wp, (int64_t)64 * ci * co)) return XEMA_ERR_INVALID_ARG;
  return launch_upconv_prep((const uint16_t*)w, ci, co, (uint16_t*)wp, (hipStream_t)stream) ==
                 hipSuccess
             ? XEMA_OK
             : XEMA_ERR_HIP;
}

extern "C" int xema_vae_upconv(const void* x, int32_t n, int32_t h, int32_t w, int32_t ci,
                               const void* wp, const void* bias, int32_t co, int32_t row_begin,
                               int32_t row_count, void* y, void* stream) {
  if (!x || !wp || !bias || !y || n <= 0 || h <= 0 || w <= 0) return XEMA_ERR_INVALID_ARG;
  int st = check_channels(ci, co);
  if (st != XEMA_OK) return st;
  if (row_begin < 0 || row_count <= 0 || (int64_t)row_begin + row_count > h) return XEMA_ERR_INVALID_ARG;
  const int64_t x_bytes = (int64_t)n * h * w * ci * 2;
  const int64_t y_bytes = (int64_t)n * 4 * h * w * co * 2;
  if (x_bytes >= ((int64_t)1 << 31)) return XEMA_ERR_UNSUPPORTED;
  if ((int64_t)n * h * w > ((int64_t)1 << 30)) return XEMA_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(wp, 16) || !aligned(bias, 16) || !aligned(y, 16))
    return XEMA_ERR_MISALIGNED;
  if (overlaps(y, y_bytes, x, x_bytes) || overlaps(y, y_bytes, wp, (int64_t)64 * ci * co) ||
      overlaps(y, y_bytes, bias, (int64_t)co * 2))
    return XEMA_ERR_INVALID_ARG;
  UpconvParams p;
  p.x = (const uint16_t*)x; p.wp = (const uint16_t*)wp; p.bias = (const uint16_t*)bias;
  p.y = (uint16_t*)y;
  p.n = n; p.h = h; p.w = w; p.ci = ci; p.co = co;
  p.row_begin = row_begin; p.row_count = row_count;
  return launch_upconv(p, (hipStream_t)stream) == hipSuccess ? XEMA_OK : XEMA_ERR_HIP;
}
