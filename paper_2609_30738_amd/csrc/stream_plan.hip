// Host-side planning of the streaming window kernels: which shapes they take, how a batch is cut
// into segments, and the workspace those segments need.
#include "stream_common.h"

namespace kv {

bool stream_shape_ok(const Shape& s, float scale) {
  const int G = s.group();
  // pass 1 takes a tile's maximum logit as the scaled maximum of the raw dot products
  return s.dtype == kDtBf16 && s.w == 32 && (s.d == 64 || s.d == 128) &&
         (G == 1 || G == 2 || G == 4) && scale > 0.f;
}

StreamPlan stream_plan(const Shape& s, int64_t total_keys) {
  // about one segment per compute unit (256 on MI355X), whole 256-key steps of the eight waves
  constexpr int64_t kTarget = 256, kStep = stream::kWaves * stream::kTileKeys, kMinSeg = 1024;
  int64_t seg = (total_keys + kTarget - 1) / kTarget;
  seg = std::max<int64_t>(kMinSeg, (seg + kStep - 1) / kStep * kStep);
  seg = std::min<int64_t>(seg, ((int64_t)s.max_len + kStep - 1) / kStep * kStep);
  StreamPlan plan;
  plan.seg_keys = (int)seg;
  plan.max_segs = (int)(((int64_t)s.max_len + seg - 1) / seg);
  return plan;
}

size_t stream_counter_offset(const Shape& s, const StreamPlan& plan) {
  const size_t part = (size_t)s.n_prob * s.h_kv * plan.max_segs * s.group() * 32 * sizeof(float2);
  return (part + 255) & ~(size_t)255;
}

size_t stream_ws_bytes(const Shape& s, const StreamPlan& plan) {
  // segment partials, then one arrival counter per unit (both passes in one launch)
  return stream_counter_offset(s, plan) + (size_t)s.n_prob * s.h_kv * sizeof(uint32_t);
}

}  // namespace kv
