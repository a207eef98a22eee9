// Base scores from mu / sigma rows (section 3.2, Eq. (5)), for batches whose window statistics
// come from the chunked window path or the two-launch streaming path (the other paths form them
// inside their second pass).
#include <algorithm>

#include "common.h"

namespace kv {
namespace {

constexpr int kScoreThreads = 256;

// s = fma(lambda1[p], sigma, w_mu mu) for every key of the batch (the same rounding as the
// selection kernel's own base score); blockIdx.x is the (problem, kv head) unit, the blocks along
// y share its keys.
__global__ __launch_bounds__(kScoreThreads) void base_score_kernel(
    const float* __restrict__ mu, const float* __restrict__ sigma, const int32_t* __restrict__ lens,
    const int64_t* __restrict__ tok_off, const float* __restrict__ lambda1, float w_mu, int h_kv,
    float* __restrict__ score) {
  const int unit = blockIdx.x, p = unit / h_kv, g = unit % h_kv;
  const int L = lens[p];
  const size_t base = (size_t)tok_off[p] * h_kv + (size_t)g * L;
  const float lam1 = lambda1[p];
  for (int i = blockIdx.y * kScoreThreads + (int)threadIdx.x; i < L; i += gridDim.y * kScoreThreads)
    score[base + i] = fmaf(lam1, sigma[base + i], w_mu * mu[base + i]);
}

}  // namespace

hipError_t launch_base_scores(const Shape& s, const float* mu, const float* sigma,
                              const float* lambda1, float w_mu, float* score, hipStream_t stream) {
  const unsigned units = (unsigned)(s.n_prob * s.h_kv);
  if (units == 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min(64, (s.max_len + kScoreThreads - 1) / kScoreThreads);
  base_score_kernel<<<dim3(units, blocks), kScoreThreads, 0, stream>>>(
      mu, sigma, s.lens, s.tok_off, lambda1, w_mu, s.h_kv, score);
  return hipGetLastError();
}

}  // namespace kv
