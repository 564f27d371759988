// Routing and grouping (Sec. 3.1 Eq. 1, Fig. 1 "tokens are grouped by
// selected expert", Sec. 3.4).
//
//   router_logits_kernel: z[t][e] = fp32(sum_i h[t][i] * W_r[e][i]), fp64 sum.
//   topk_kernel:          k largest logits per token (ties -> lower expert id)
//                         and their softmax mixture weights in fp64.
//   group_kernel:         per-expert counts, exclusive offsets, a stable
//                         counting sort of pair ids, the ascending active list
//                         and (optionally) the MFMA row-tile prefix sum.
#include "common.h"

namespace emoe {
namespace {

// ----------------------------------------------------------------- router
// A wavefront computes a kTokW x kExpW block of logits; lanes split the
// hidden dimension in 8-element chunks, so every load is a coalesced 16-byte
// read of h or W_r.  Products of two bf16 values are exact in fp64 and the
// fp64 sum is rounded once to fp32.
constexpr int kTokW = 4;
constexpr int kExpW = 4;

__device__ __forceinline__ void bf16x8_to_f64(const uint4 v, double* out) {
  const uint32_t dw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    out[2 * p] = (double)bf16_to_f32(dw[p] & 0xffffu);
    out[2 * p + 1] = (double)bf16_to_f32(dw[p] >> 16);
  }
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

__global__ __launch_bounds__(256) void router_logits_kernel(int tokens, int n_experts, int d,
                                                            const uint16_t* __restrict__ h,
                                                            const uint16_t* __restrict__ wr,
                                                            float* __restrict__ logits) {
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int t0 = blockIdx.x * kTokW;
  const int e0 = (blockIdx.y * 4 + wave) * kExpW;
  if (e0 >= n_experts) return;

  double acc[kTokW][kExpW];
#pragma unroll
  for (int a = 0; a < kTokW; ++a)
#pragma unroll
    for (int b = 0; b < kExpW; ++b) acc[a][b] = 0.0;

  for (int k0 = 8 * lane; k0 < d; k0 += 512) {
    double wv[kExpW][8];
#pragma unroll
    for (int b = 0; b < kExpW; ++b) {
      const int e = e0 + b;
      if (e < n_experts) {
        bf16x8_to_f64(*reinterpret_cast<const uint4*>(wr + (int64_t)e * d + k0), wv[b]);
      } else {
#pragma unroll
        for (int r = 0; r < 8; ++r) wv[b][r] = 0.0;
      }
    }
#pragma unroll
    for (int a = 0; a < kTokW; ++a) {
      const int t = t0 + a;
      if (t >= tokens) break;
      double hv[8];
      bf16x8_to_f64(*reinterpret_cast<const uint4*>(h + (int64_t)t * d + k0), hv);
#pragma unroll
      for (int b = 0; b < kExpW; ++b)
#pragma unroll
        for (int r = 0; r < 8; ++r) acc[a][b] = fma(hv[r], wv[b][r], acc[a][b]);
    }
  }
#pragma unroll
  for (int a = 0; a < kTokW; ++a) {
#pragma unroll
    for (int b = 0; b < kExpW; ++b) {
      const double s = wave_sum_f64(acc[a][b]);
      const int t = t0 + a, e = e0 + b;
      if (lane == 0 && t < tokens && e < n_experts) logits[(int64_t)t * n_experts + e] = (float)s;
    }
  }
}

// ----------------------------------------------------------------- top-k
// One wavefront per token; lane l holds the logits of experts l, l+64, ...
// The 64-bit key orders by logit (a monotone integer image of the fp32 value,
// -0 folded onto +0) and then by lower expert id.
__device__ __forceinline__ uint64_t topk_key(float z, int e) {
  uint32_t u = __float_as_uint(z + 0.0f);  // -0 -> +0
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint32_t)(0xffffffffu - (uint32_t)e);
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t o = __shfl_xor(v, off);
    v = o > v ? o : v;
  }
  return v;
}

constexpr int kPerLane = EMOE_MAX_EXPERTS / 64;

__global__ __launch_bounds__(256) void topk_kernel(int tokens, int n_experts, int top_k,
                                                   int renormalize, const float* __restrict__ logits,
                                                   int32_t* __restrict__ topk_ids,
                                                   float* __restrict__ topk_w) {
  const int lane = lane_id();
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= tokens) return;
  const float* z = logits + (int64_t)t * n_experts;

  float v[kPerLane];
  bool taken[kPerLane];
#pragma unroll
  for (int c = 0; c < kPerLane; ++c) {
    const int e = lane + 64 * c;
    v[c] = e < n_experts ? z[e] : 0.f;
    taken[c] = e >= n_experts;
  }
  // Selected ids and logits of rank j live in lane j % 64, register j / 64.
  int sel_id[kPerLane];
  float sel_z[kPerLane];
  float zmax = 0.f;
  for (int j = 0; j < top_k; ++j) {
    uint64_t best = 0;
#pragma unroll
    for (int c = 0; c < kPerLane; ++c) {
      if (!taken[c]) {
        const uint64_t key = topk_key(v[c], lane + 64 * c);
        best = key > best ? key : best;
      }
    }
    best = wave_max_u64(best);
    const int e = (int)(0xffffffffu - (uint32_t)(best & 0xffffffffu));
    // The owner lane marks the winner and broadcasts its logit.
    float zw = 0.f;
#pragma unroll
    for (int c = 0; c < kPerLane; ++c) {
      if (lane + 64 * c == e) {
        taken[c] = true;
        zw = v[c];
      }
    }
    zw = __shfl(zw, e & 63);
    if (j == 0) zmax = zw;
#pragma unroll
    for (int c = 0; c < kPerLane; ++c) {
      if (j == lane + 64 * c) {
        sel_id[c] = e;
        sel_z[c] = zw;
      }
    }
  }

  // Mixture weights in fp64: p_j = exp(z_j - zmax) / denominator.
  double part = 0.0;
  if (renormalize) {
#pragma unroll
    for (int c = 0; c < kPerLane; ++c)
      if (lane + 64 * c < top_k) part += exp((double)sel_z[c] - (double)zmax);
  } else {
#pragma unroll
    for (int c = 0; c < kPerLane; ++c)
      if (lane + 64 * c < n_experts) part += exp((double)v[c] - (double)zmax);
  }
  const double denom = wave_sum_f64(part);
#pragma unroll
  for (int c = 0; c < kPerLane; ++c) {
    const int j = lane + 64 * c;
    if (j < top_k) {
      topk_ids[(int64_t)t * top_k + j] = sel_id[c];
      topk_w[(int64_t)t * top_k + j] = (float)(exp((double)sel_z[c] - (double)zmax) / denom);
    }
  }
}

// ----------------------------------------------------------------- grouping
constexpr int kGroupThreads = 1024;
constexpr int kGroupWaves = kGroupThreads / 64;

__device__ __forceinline__ int wave_exclusive_scan(int v, int& total) {
  const int lane = lane_id();
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  total = __shfl(x, 63);
  return x - v;
}

__global__ __launch_bounds__(kGroupThreads) void group_kernel(
    int pairs, int n_experts, const int32_t* __restrict__ ids, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ sorted_pairs, int32_t* __restrict__ active,
    int32_t* __restrict__ n_active, int32_t* __restrict__ tile_offsets) {
  __shared__ int cnt[EMOE_MAX_EXPERTS];
  __shared__ int off[EMOE_MAX_EXPERTS];
  __shared__ int placed[EMOE_MAX_EXPERTS];
  __shared__ int wcnt[kGroupWaves][EMOE_MAX_EXPERTS];

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  for (int e = tid; e < EMOE_MAX_EXPERTS; e += kGroupThreads) {
    cnt[e] = 0;
    placed[e] = 0;
  }
  __syncthreads();
  for (int i = tid; i < pairs; i += kGroupThreads) atomicAdd(&cnt[ids[i]], 1);
  __syncthreads();

  // Scans over experts by wavefront 0: lane l owns experts 4l .. 4l+3.
  if (wave == 0) {
    int c[kPerLane], local = 0, nz = 0, tl = 0;
#pragma unroll
    for (int q = 0; q < kPerLane; ++q) {
      const int e = kPerLane * lane + q;
      c[q] = e < n_experts ? cnt[e] : 0;
      local += c[q];
      nz += c[q] > 0;
      tl += (c[q] + kMfmaRows - 1) / kMfmaRows;
    }
    int total, nz_total, tl_total;
    int base = wave_exclusive_scan(local, total);
    int nz_base = wave_exclusive_scan(nz, nz_total);
    int tl_base = wave_exclusive_scan(tl, tl_total);
#pragma unroll
    for (int q = 0; q < kPerLane; ++q) {
      const int e = kPerLane * lane + q;
      if (e < n_experts) {
        off[e] = base;
        counts[e] = c[q];
        offsets[e] = base;
        if (tile_offsets) tile_offsets[e] = tl_base;
        if (c[q] > 0) active[nz_base++] = e;
      }
      base += c[q];
      tl_base += (c[q] + kMfmaRows - 1) / kMfmaRows;
    }
    if (lane == 0) {
      offsets[n_experts] = total;
      if (tile_offsets) tile_offsets[n_experts] = tl_total;
      *n_active = nz_total;
    }
  }
  __syncthreads();

  // Stable scatter, 1024 pairs per round.  Within a wavefront, lanes with the
  // same expert are found by ballots over the expert id bits; the rank of a
  // pair is its position among those lanes, after earlier wavefronts and
  // earlier rounds.
  int bits = 0;
  while ((1 << bits) < n_experts) ++bits;
  for (int base = 0; base < pairs; base += kGroupThreads) {
    for (int e = lane; e < EMOE_MAX_EXPERTS; e += 64) wcnt[wave][e] = 0;
    __syncthreads();
    const int i = base + tid;
    const bool valid = i < pairs;
    const int e = valid ? ids[i] : 0;
    uint64_t match = __ballot(valid);
    for (int b = 0; b < bits; ++b) {
      const uint64_t m = __ballot(valid && ((e >> b) & 1));
      match &= ((e >> b) & 1) ? m : ~m;
    }
    const uint64_t lt = (1ull << lane) - 1ull;
    const int rank = __popcll(match & lt);
    if (valid && rank == 0) wcnt[wave][e] = __popcll(match);
    __syncthreads();
    if (valid) {
      int pos = placed[e] + rank;
      for (int w = 0; w < wave; ++w) pos += wcnt[w][e];
      sorted_pairs[off[e] + pos] = i;
    }
    __syncthreads();
    for (int x = tid; x < n_experts; x += kGroupThreads) {
      int s = 0;
      for (int w = 0; w < kGroupWaves; ++w) s += wcnt[w][x];
      placed[x] += s;
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_router_logits(int tokens, int n_experts, int d, const uint16_t* h,
                                const uint16_t* w_router, float* logits, hipStream_t stream) {
  if (tokens == 0) return hipSuccess;
  dim3 grid((tokens + kTokW - 1) / kTokW, (n_experts + 4 * kExpW - 1) / (4 * kExpW));
  launch(router_logits_kernel, grid, dim3(256), stream, tokens, n_experts, d, h,
                     w_router, logits);
  return hipGetLastError();
}

hipError_t launch_topk(int tokens, int n_experts, int top_k, int renormalize, const float* logits,
                       int32_t* topk_ids, float* topk_w, hipStream_t stream) {
  if (tokens == 0) return hipSuccess;
  launch(topk_kernel, dim3((tokens + 3) / 4), dim3(256), stream, tokens, n_experts,
                     top_k, renormalize, logits, topk_ids, topk_w);
  return hipGetLastError();
}

hipError_t launch_group(int pairs, int n_experts, const int32_t* topk_ids, int32_t* counts,
                        int32_t* offsets, int32_t* sorted_pairs, int32_t* active,
                        int32_t* n_active, int32_t* tile_offsets, hipStream_t stream) {
  launch(group_kernel, dim3(1), dim3(kGroupThreads), stream, pairs, n_experts,
                     topk_ids, counts, offsets, sorted_pairs, active, n_active, tile_offsets);
  return hipGetLastError();
}

}  // namespace emoe
