// Routing and grouping kernels (Sec. 3.1 Eq. 1, Fig. 1 "tokens are grouped by
// selected expert", Sec. 3.4).  The arithmetic lives in device_route.h.
//
//   router_logits_kernel: z[t][e] = fp32(sum_i h[t][i] * W_r[e][i]), fp64 sum.
//   topk_kernel:          k largest logits per token (ties -> lower expert id)
//                         and their softmax mixture weights in fp64.
//   group_kernel:         per-expert counts, exclusive offsets, a stable
//                         counting sort of pair ids, the ascending active list
//                         and (optionally) the MFMA row-tile prefix sum.
#include "device_route.h"

namespace emoe {
namespace {

// A wavefront computes a kTokW x kExpW block of logits.
constexpr int kTokW = 4;
constexpr int kExpW = 4;

__global__ __launch_bounds__(256) void router_logits_kernel(int tokens, int n_experts, int d,
                                                            const uint16_t* __restrict__ h,
                                                            const uint16_t* __restrict__ wr,
                                                            float* __restrict__ logits) {
  const int wave = threadIdx.x >> 6;
  const int t0 = blockIdx.x * kTokW;
  const int e0 = (blockIdx.y * 4 + wave) * kExpW;
  if (e0 >= n_experts) return;
  wave_router_logits<kTokW, kExpW, false>(tokens, n_experts, d, t0, e0, h, wr, logits);
}

__global__ __launch_bounds__(256) void topk_kernel(int tokens, int n_experts, int top_k,
                                                   int renormalize, const float* __restrict__ logits,
                                                   int32_t* __restrict__ topk_ids,
                                                   float* __restrict__ topk_w) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= tokens) return;
  wave_topk<false>(logits + (int64_t)t * n_experts, n_experts, top_k, renormalize,
            topk_ids + (int64_t)t * top_k, topk_w + (int64_t)t * top_k);
}

constexpr int kGroupThreads = 1024;

__global__ __launch_bounds__(kGroupThreads) void group_kernel(
    int pairs, int n_experts, const int32_t* __restrict__ ids, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ sorted_pairs, int32_t* __restrict__ active,
    int32_t* __restrict__ n_active, int32_t* __restrict__ tile_offsets) {
  __shared__ GroupShared<kGroupThreads> sh;
  block_group<kGroupThreads, false>(sh, pairs, n_experts, ids, counts, offsets, sorted_pairs,
                                    active, n_active, tile_offsets, nullptr);
}

}  // namespace

hipError_t launch_router_logits(int tokens, int n_experts, int d, const uint16_t* h,
                                const uint16_t* w_router, float* logits, hipStream_t stream) {
  if (tokens == 0) return hipSuccess;
  dim3 grid((tokens + kTokW - 1) / kTokW, (n_experts + 4 * kExpW - 1) / (4 * kExpW));
  launch(router_logits_kernel, grid, dim3(256), stream, tokens, n_experts, d, h, w_router, logits);
  return hipGetLastError();
}

hipError_t launch_topk(int tokens, int n_experts, int top_k, int renormalize, const float* logits,
                       int32_t* topk_ids, float* topk_w, hipStream_t stream) {
  if (tokens == 0) return hipSuccess;
  launch(topk_kernel, dim3((tokens + 3) / 4), dim3(256), stream, tokens, n_experts, top_k,
         renormalize, logits, topk_ids, topk_w);
  return hipGetLastError();
}

hipError_t launch_group(int pairs, int n_experts, const int32_t* topk_ids, int32_t* counts,
                        int32_t* offsets, int32_t* sorted_pairs, int32_t* active,
                        int32_t* n_active, int32_t* tile_offsets, hipStream_t stream) {
  launch(group_kernel, dim3(1), dim3(kGroupThreads), stream, pairs, n_experts, topk_ids, counts,
         offsets, sorted_pairs, active, n_active, tile_offsets);
  return hipGetLastError();
}

}  // namespace emoe
