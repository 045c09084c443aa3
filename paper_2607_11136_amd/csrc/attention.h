// Launch interface of the joint-attention kernels (step a4), kept apart from
// the other kernels' declarations so that the attention kernel is built from
// k_attention.hip, this header and device_common.h alone.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xema {

// Q, K: [batch, heads, padded_len, head_dim] fp16 (queries pre-multiplied by
// log2(e)/sqrt(head_dim)); V^T: [batch, heads, head_dim, padded_len] fp16;
// tokens [seq_len, padded_len) hold zeros.  O: [batch, q_count, heads *
// head_dim] fp16, the outputs of queries [q_begin, q_begin + q_count).
struct AttnParams {
  const _Float16* q;
  const _Float16* k;
  const _Float16* vt;
  _Float16* o;
  int batch, heads, seq_len, padded_len, q_begin, q_count;
};

hipError_t launch_attention(const AttnParams& p, int head_dim, hipStream_t s);

}  // namespace xema
