// Routing and grouping kernels (Sec. 3.1 Eq. 1; Fig. 1 and Sec. 3.4, where the
// token-expert pairs are gathered by the expert they select).  The arithmetic
// lives in device_route.h.
//
//   router_logits_kernel: z[t][e] = fp32(sum_i h[t][i] * W_r[e][i]), fp64 sum
//                         on fp64 MFMA.
//   topk_kernel:          k largest logits per token (ties -> lower expert id)
//                         and their softmax mixture weights in fp64.
//   topk_count_kernel:    the same for the 64 / k tokens of one 64-pair chunk
//                         per workgroup, plus that chunk's per-expert counts.
//   group_kernel:         per-expert counts, exclusive offsets, a stable
//                         counting sort of pair ids, the ascending active list
//                         and (optionally) the MFMA row-tile prefix sum.
#include "device_route.h"

namespace emoe {
namespace {

typedef double f64x4_t __attribute__((ext_vector_type(4)));

// Router logits on fp64 MFMA (v_mfma_f64_16x16x4f64): a workgroup computes a
// 16-token x 16-expert tile and its four wavefronts split d into quarters.
// Per 32 inputs, lane l loads 8 consecutive bf16 of token row l%16 and of
// expert row l%16 (inputs 8*(l/16) .. +7) and feeds them to 8 MFMAs; A and B
// take the same input for the same lane, so every product h_k * w_k is
// formed once and exactly, and summed in fp64.  The four partial sums are
// added in wavefront order and rounded once to fp32.
__global__ __launch_bounds__(256) void router_logits_kernel(int tokens, int n_experts, int d,
                                                            const uint16_t* __restrict__ h,
                                                            const uint16_t* __restrict__ wr,
                                                            float* __restrict__ logits,
                                                            float* __restrict__ tok_bias) {
  __shared__ double part[4][4][64];
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int t0 = blockIdx.x * 16, e0 = blockIdx.y * 16;
  const int row = lane & 15, q = lane >> 4;
  // Rows past the end repeat the last row; their results are not stored.
  const int t = min(t0 + row, tokens - 1);
  const int e = min(e0 + row, n_experts - 1);
  const int kq = d / 4;
  const uint16_t* hp = h + (int64_t)t * d + wave * kq + 8 * q;
  const uint16_t* wp = wr + (int64_t)e * d + wave * kq + 8 * q;
  f64x4_t acc = {0.0, 0.0, 0.0, 0.0};
  // Loads run kAhead steps of 32 inputs ahead of the MFMAs.
  constexpr int kAhead = 4;
  const int n = kq / 32;
  // With tok_bias (d a multiple of 512, so every iteration of the loop below
  // is one 128-input group), the first expert tile's workgroups also sum each
  // group of their token rows.
  const bool sums = tok_bias != nullptr && blockIdx.y == 0;
  uint4 hb[kAhead], wb[kAhead];
#pragma unroll
  for (int j = 0; j < kAhead; ++j) {
    if (j < n) {
      hb[j] = *reinterpret_cast<const uint4*>(hp + 32 * j);
      wb[j] = *reinterpret_cast<const uint4*>(wp + 32 * j);
    }
  }
  for (int i = 0; i < n; i += kAhead) {
    float gsum = 0.f;
#pragma unroll
    for (int j = 0; j < kAhead; ++j) {
      if (i + j < n) {
        double hv[8], wv[8];
        bf16x8_to_f64(hb[j], hv);
        bf16x8_to_f64(wb[j], wv);
        if (i + j + kAhead < n) {
          hb[j] = *reinterpret_cast<const uint4*>(hp + 32 * (i + j + kAhead));
          wb[j] = *reinterpret_cast<const uint4*>(wp + 32 * (i + j + kAhead));
        }
#pragma unroll
        for (int s = 0; s < 8; ++s) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(hv[s], wv[s], acc, 0, 0, 0);
        if (sums) {
#pragma unroll
          for (int s = 0; s < 8; ++s) gsum += (float)hv[s];
        }
      }
    }
    if (sums) {
      // The lane's 32 inputs of the group, then the four lanes of the row.
      gsum += __shfl_xor(gsum, 16);
      gsum += __shfl_xor(gsum, 32);
      const int g = (wave * kq + 32 * i) / kGroup;
      if (q == 0 && t0 + row < tokens) tok_bias[(int64_t)(t0 + row) * (d / kGroup) + g] = -136.f * gsum;
    }
  }
  // Lane l holds rows (tokens) l/16 + 4*r of column (expert) l%16 (the fp64
  // MFMA interleaves its output rows by register).
#pragma unroll
  for (int r = 0; r < 4; ++r) part[wave][r][lane] = acc[r];
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const double z = ((part[0][r][lane] + part[1][r][lane]) + part[2][r][lane]) + part[3][r][lane];
      const int tt = t0 + q + 4 * r, ee = e0 + row;
      if (tt < tokens && ee < n_experts) logits[(int64_t)tt * n_experts + ee] = (float)z;
    }
  }
}

__global__ __launch_bounds__(256) void topk_kernel(int tokens, int n_experts, int top_k,
                                                   int renormalize, const float* __restrict__ logits,
                                                   int32_t* __restrict__ topk_ids,
                                                   float* __restrict__ topk_w) {
  __shared__ uint64_t s_rank[4][64];  // per-wavefront top-k scratch
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= tokens) return;
  wave_topk<false>(logits + (int64_t)t * n_experts, n_experts, top_k, renormalize,
                   topk_ids + (int64_t)t * top_k, topk_w + (int64_t)t * top_k,
                   s_rank[threadIdx.x >> 6]);
}

// Top-k of 64 / top_k tokens per workgroup, one wavefront each, when top_k
// divides 64: the workgroup's pairs are then exactly one 64-pair chunk of the
// wide grouping (chunk c = blockIdx.x), and after its selections it also
// writes that chunk's per-expert counts (chunk_count_kernel's row), which
// saves that launch.  Ids and weights as topk_kernel writes them.
__global__ __launch_bounds__(1024) void topk_count_kernel(int tokens, int n_experts, int top_k,
                                                          int renormalize,
                                                          const float* __restrict__ logits,
                                                          int32_t* __restrict__ topk_ids,
                                                          float* __restrict__ topk_w,
                                                          int32_t* __restrict__ chunk_counts) {
  __shared__ uint64_t s_rank[16][64];  // per-wavefront top-k scratch
  __shared__ int s_pair[64];           // the chunk's expert ids, pair order
  __shared__ int row[EMOE_MAX_EXPERTS];
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int c = blockIdx.x;
  const int t = c * (64 / top_k) + wave;
  for (int e = threadIdx.x; e < n_experts; e += blockDim.x) row[e] = 0;
  if (t < tokens) {
    TopkState st;
    wave_topk_select<false>(logits + (int64_t)t * n_experts, n_experts, top_k, st, s_rank[wave]);
    wave_topk_store_ids<false>(st, top_k, topk_ids + (int64_t)t * top_k);
#pragma unroll
    for (int r = 0; r < kPerLane; ++r)
      if (lane + 64 * r < top_k) s_pair[wave * top_k + lane + 64 * r] = st.sel_id[r];
    wave_topk_weights<false>(st, n_experts, top_k, renormalize, topk_w + (int64_t)t * top_k);
  }
  __syncthreads();
  if (wave == 0) {
    int bits = 0;
    while ((1 << bits) < n_experts) ++bits;
    const bool valid = 64 * c + lane < tokens * top_k;
    const int e = valid ? s_pair[lane] : 0;
    const uint64_t m = match_expert(valid, e, bits);
    const int rank = __popcll(m & ((1ull << lane) - 1ull));
    if (valid && rank == 0) row[e] = __popcll(m);  // one wavefront: LDS accesses stay in order
    for (int x = lane; x < n_experts; x += 64) chunk_counts[(int64_t)c * n_experts + x] = row[x];
  }
}

constexpr int kGroupThreads = 1024;

__global__ __launch_bounds__(kGroupThreads) void group_kernel(
    int pairs, int n_experts, const int32_t* __restrict__ ids, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ sorted_pairs, int32_t* __restrict__ active,
    int32_t* __restrict__ n_active, int32_t* __restrict__ tile_offsets,
    int32_t* __restrict__ pair_pos, int mfma_rows) {
  __shared__ GroupShared<kGroupThreads> sh;
  block_group<kGroupThreads, false>(sh, pairs, n_experts, ids, counts, offsets, sorted_pairs,
                                    active, n_active, tile_offsets, pair_pos, mfma_rows);
}

// Grouping spread over many workgroups (large calls): 64-pair chunks, one per
// wavefront, kChunkWaves chunks per workgroup.
constexpr int kChunkWaves = 16;

// chunk_counts[c][e]: pairs of chunk c (pairs 64c .. 64c+63) routed to e.
__global__ __launch_bounds__(64 * kChunkWaves) void chunk_count_kernel(
    int pairs, int n_experts, const int32_t* __restrict__ ids, int32_t* __restrict__ chunk_counts) {
  __shared__ int row[kChunkWaves][EMOE_MAX_EXPERTS];
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int c = blockIdx.x * kChunkWaves + wave;
  if (c >= (pairs + 63) / 64) return;  // whole wavefront; no barrier below
  int bits = 0;
  while ((1 << bits) < n_experts) ++bits;
  int* r = row[wave];
  for (int e = lane; e < n_experts; e += 64) r[e] = 0;
  const int i = 64 * c + lane;
  const bool valid = i < pairs;
  const int e = valid ? ids[i] : 0;
  const uint64_t m = match_expert(valid, e, bits);
  const int rank = __popcll(m & ((1ull << lane) - 1ull));
  if (valid && rank == 0) r[e] = __popcll(m);  // one wavefront: LDS accesses stay in order
  for (int x = lane; x < n_experts; x += 64) chunk_counts[(int64_t)c * n_experts + x] = r[x];
}

// Each workgroup sums the chunk table (all chunks, and those before its own),
// derives the exclusive offsets and its chunks' first positions per expert,
// and places its chunks' pairs in order (stable).  Workgroup 0 also writes
// counts, offsets, the active list, n_active and the row-tile prefix sum.
__global__ __launch_bounds__(64 * kChunkWaves) void chunk_place_kernel(
    int pairs, int n_experts, const int32_t* __restrict__ ids,
    const int32_t* __restrict__ chunk_counts, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ sorted_pairs,
    int32_t* __restrict__ active, int32_t* __restrict__ n_active,
    int32_t* __restrict__ tile_offsets, int32_t* __restrict__ pair_pos, int mfma_rows) {
  __shared__ int part_all[kChunkWaves][EMOE_MAX_EXPERTS];
  __shared__ int part_pre[kChunkWaves][EMOE_MAX_EXPERTS];
  __shared__ int base[kChunkWaves][EMOE_MAX_EXPERTS];
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int n_chunks = (pairs + 63) / 64;
  const int c0 = blockIdx.x * kChunkWaves;
  // Wavefront w sums chunks w, w + 16, ...: all of them, and those before c0.
#pragma unroll
  for (int q = 0; q < kPerLane; ++q) {
    const int e = 64 * q + lane;
    if (e >= n_experts) break;
    int all = 0, pre = 0;
    // Loads in batches of 8, so one memory latency covers 8 chunks.
    for (int cb = wave; cb < n_chunks; cb += 8 * kChunkWaves) {
      int v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int c = cb + j * kChunkWaves;
        v[j] = c < n_chunks ? chunk_counts[(int64_t)c * n_experts + e] : 0;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        all += v[j];
        if (cb + j * kChunkWaves < c0) pre += v[j];
      }
    }
    part_all[wave][e] = all;
    part_pre[wave][e] = pre;
  }
  __syncthreads();
  if (wave == 0) {
    int cnt[kPerLane], pre[kPerLane], local = 0, nz = 0, tl = 0;
#pragma unroll
    for (int q = 0; q < kPerLane; ++q) {
      const int e = kPerLane * lane + q;
      cnt[q] = 0;
      pre[q] = 0;
      if (e < n_experts)
        for (int w = 0; w < kChunkWaves; ++w) {
          cnt[q] += part_all[w][e];
          pre[q] += part_pre[w][e];
        }
      local += cnt[q];
      nz += cnt[q] > 0;
      tl += mfma_row_tiles(cnt[q], mfma_rows);
    }
    int total, nz_total, tl_total;
    int off = wave_exclusive_scan(local, total);
    int nz_base = wave_exclusive_scan(nz, nz_total);
    int tl_base = wave_exclusive_scan(tl, tl_total);
    const bool writer = blockIdx.x == 0;
#pragma unroll
    for (int q = 0; q < kPerLane; ++q) {
      const int e = kPerLane * lane + q;
      if (e < n_experts) {
        if (writer) {
          counts[e] = cnt[q];
          offsets[e] = off;
          tile_offsets[e] = tl_base;
          if (cnt[q] > 0) active[nz_base++] = e;
        }
        int own[kChunkWaves];
#pragma unroll
        for (int w = 0; w < kChunkWaves; ++w)
          own[w] = c0 + w < n_chunks ? chunk_counts[(int64_t)(c0 + w) * n_experts + e] : 0;
        int run = off + pre[q];
#pragma unroll
        for (int w = 0; w < kChunkWaves; ++w) {
          base[w][e] = run;
          run += own[w];
        }
      }
      off += cnt[q];
      tl_base += mfma_row_tiles(cnt[q], mfma_rows);
    }
    if (writer && lane == 0) {
      offsets[n_experts] = total;
      tile_offsets[n_experts] = tl_total;
      *n_active = nz_total;
    }
  }
  __syncthreads();
  const int c = c0 + wave;
  if (c >= n_chunks) return;
  int bits = 0;
  while ((1 << bits) < n_experts) ++bits;
  const int i = 64 * c + lane;
  const bool valid = i < pairs;
  const int e = valid ? ids[i] : 0;
  const uint64_t m = match_expert(valid, e, bits);
  const int rank = __popcll(m & ((1ull << lane) - 1ull));
  if (valid) {
    const int pos = base[wave][e] + rank;
    sorted_pairs[pos] = i;
    pair_pos[i] = pos;
  }
}

}  // namespace

hipError_t launch_group_count(int pairs, int n_experts, const int32_t* topk_ids,
                              int32_t* chunk_counts, hipStream_t stream) {
  const int n_wg = ((pairs + 63) / 64 + kChunkWaves - 1) / kChunkWaves;
  if (n_wg == 0) return hipSuccess;
  launch(chunk_count_kernel, dim3(n_wg), dim3(64 * kChunkWaves), stream, pairs, n_experts, topk_ids,
         chunk_counts);
  return hipGetLastError();
}

hipError_t launch_group_place(int pairs, int n_experts, const int32_t* topk_ids,
                              const int32_t* chunk_counts, int32_t* counts, int32_t* offsets,
                              int32_t* sorted_pairs, int32_t* active, int32_t* n_active,
                              int32_t* tile_offsets, int32_t* pair_pos, int mfma_rows,
                              hipStream_t stream) {
  const int n_wg = ((pairs + 63) / 64 + kChunkWaves - 1) / kChunkWaves;
  if (n_wg == 0) return hipSuccess;
  launch(chunk_place_kernel, dim3(n_wg), dim3(64 * kChunkWaves), stream, pairs, n_experts, topk_ids,
         chunk_counts, counts, offsets, sorted_pairs, active, n_active, tile_offsets, pair_pos,
         mfma_rows);
  return hipGetLastError();
}

hipError_t launch_router_logits(int tokens, int n_experts, int d, const uint16_t* h,
                                const uint16_t* w_router, float* logits, hipStream_t stream,
                                float* tok_bias) {
  if (tokens == 0) return hipSuccess;
  if (d % 512 != 0) tok_bias = nullptr;
  dim3 grid((tokens + 15) / 16, (n_experts + 15) / 16);
  launch(router_logits_kernel, grid, dim3(256), stream, tokens, n_experts, d, h, w_router, logits,
         tok_bias);
  return hipGetLastError();
}

hipError_t launch_topk(int tokens, int n_experts, int top_k, int renormalize, const float* logits,
                       int32_t* topk_ids, float* topk_w, hipStream_t stream) {
  if (tokens == 0) return hipSuccess;
  launch(topk_kernel, dim3((tokens + 3) / 4), dim3(256), stream, tokens, n_experts, top_k,
         renormalize, logits, topk_ids, topk_w);
  return hipGetLastError();
}

hipError_t launch_topk_count(int tokens, int n_experts, int top_k, int renormalize,
                             const float* logits, int32_t* topk_ids, float* topk_w,
                             int32_t* chunk_counts, hipStream_t stream) {
  if (tokens == 0) return hipSuccess;
  if (top_k < 1 || 64 % top_k != 0 || 64 / top_k > 16) return hipErrorInvalidValue;
  const int per = 64 / top_k;  // tokens (wavefronts) per chunk
  launch(topk_count_kernel, dim3((tokens + per - 1) / per), dim3(64 * per), stream, tokens,
         n_experts, top_k, renormalize, logits, topk_ids, topk_w, chunk_counts);
  return hipGetLastError();
}

hipError_t launch_group(int pairs, int n_experts, const int32_t* topk_ids, int32_t* counts,
                        int32_t* offsets, int32_t* sorted_pairs, int32_t* active,
                        int32_t* n_active, int32_t* tile_offsets, int32_t* pair_pos,
                        int mfma_rows, hipStream_t stream) {
  launch(group_kernel, dim3(1), dim3(kGroupThreads), stream, pairs, n_experts, topk_ids, counts,
         offsets, sorted_pairs, active, n_active, tile_offsets, pair_pos, mfma_rows);
  return hipGetLastError();
}

}  // namespace emoe
