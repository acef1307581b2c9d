// Launch configuration of the attention kernels (tppsd_attention.hip): the
// KV cache slab stride, key splits and their partials, and the launcher.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tppsd {

// Positions per (sequence, head) slab of a KV cache: the event capacity
// rounded up to a multiple of 8 (bf16 values are stored in 8-position blocks).
inline int kv_stride(int cap) { return (cap + 7) / 8 * 8; }

// Key splits of the attention for B sequences x H heads over at most max_keys
// keys (one workgroup serves all query tiles of a pair): up to 512
// workgroups, each split keeping at least 512 keys (shorter splits do not pay
// for the merge launch). Measured at 32 sequences x 4096 events: aiming at
// 1024 workgroups (8 draft splits, 4 verify splits) was slower than 512 (4
// and 2): verify attention 42.1 -> 38.8 us.
inline int attn_splits(int B, int H, int max_keys) {
  const long items = (long)B * H;
  int s = 1;
  while (s < 8 && items * s < 512 && max_keys / (2 * s) >= 512) s *= 2;
  return s;
}
// floats of split partials for up to qtiles_max query tiles of 16
inline size_t attn_part_floats(int B, int H, int dh, int qtiles_max, int max_keys) {
  const int s = attn_splits(B, H, max_keys);
  return s > 1 ? (size_t)B * H * qtiles_max * 16 * s * (dh + 2) : 0;
}
// sink: AttNHP normalisation 1 + sum f (an extra key of score 0, value 0)
void launch_attention(const void *q, const void *kc, const void *vc, void *o, int bf16,
                      const int32_t *start, int start_off, const int32_t *done, int B, int P, int H,
                      int dh, int cap, float *part, int sink, int verify, hipEvent_t ev0, hipEvent_t ev1,
                      hipStream_t st);
}  // namespace tppsd
