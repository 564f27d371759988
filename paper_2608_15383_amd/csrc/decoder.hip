// Synthetic decoder around the routed-expert layer (exactmoe_decoder.h):
// embedding gather, residual add + RMSNorm, rotary positions with the KV
// cache append, causal attention and the greedy argmax as gfx950 kernels; the
// dense bf16 projections (QKV, output, LM head) as weight-streaming GEMV
// kernels for up to four tokens (decode steps) and through rocBLAS for more
// (prompts); the routed experts through emoe_moe_forward.
#include <rocblas/rocblas.h>

#include <cmath>
#include <new>
#include <vector>

#include "common.h"
#include "exactmoe_decoder.h"

using namespace emoe;

namespace {

constexpr int kThreads = 256;
constexpr int kMaxHeadDim = 256;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- kernels
// Y[t][n] = sum_k X[t][k] W[n][k] (+ C[t][n]) for kT <= 4 tokens: a
// weight-streaming GEMV.  Each wavefront owns kR rows of W; lane l reads the
// 16-byte chunks k = 8l + 512u of every row (and of the token rows), all
// loads of a 2048-input row block issued before any product, and the fp32
// dot products (bf16 pairs) are summed over the lanes by butterfly.  Output
// bf16 (rounded to nearest even after adding C) or fp32.
constexpr int kDenseMaxTokens = 4;
constexpr int kDenseUnroll = 4;  // 512-input chunks per lane in flight

__device__ __forceinline__ float dot8_bf16(uint4 a, uint4 b, float c) {
  c = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.x),
                                      __builtin_bit_cast(bf16x2_t, b.x), c, false);
  c = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.y),
                                      __builtin_bit_cast(bf16x2_t, b.y), c, false);
  c = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.z),
                                      __builtin_bit_cast(bf16x2_t, b.z), c, false);
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.w),
                                         __builtin_bit_cast(bf16x2_t, b.w), c, false);
}

template <int kR, int kT>
__global__ __launch_bounds__(kThreads) void dense_gemv_kernel(int N, int K, const uint16_t* X,
                                                              const uint16_t* W, const uint16_t* C,
                                                              void* Y, int out_f32) {
  const int lane = threadIdx.x & 63;
  const int n0 = (blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)) * kR;
  if (n0 >= N) return;
  float acc[kR][kT];
#pragma unroll
  for (int r = 0; r < kR; ++r)
#pragma unroll
    for (int t = 0; t < kT; ++t) acc[r][t] = 0.f;
  for (int k0 = 8 * lane; k0 < K; k0 += 512 * kDenseUnroll) {
    uint4 w[kDenseUnroll][kR], x[kDenseUnroll][kT];
#pragma unroll
    for (int u = 0; u < kDenseUnroll; ++u) {
      const int k = k0 + 512 * u;
      if (k < K) {
#pragma unroll
        for (int r = 0; r < kR; ++r) {
          const int n = min(n0 + r, N - 1);  // rows past N repeat the last (not stored)
          w[u][r] = *reinterpret_cast<const uint4*>(W + (int64_t)n * K + k);
        }
#pragma unroll
        for (int t = 0; t < kT; ++t) x[u][t] = *reinterpret_cast<const uint4*>(X + (int64_t)t * K + k);
      }
    }
#pragma unroll
    for (int u = 0; u < kDenseUnroll; ++u) {
      if (k0 + 512 * u < K) {
#pragma unroll
        for (int r = 0; r < kR; ++r)
#pragma unroll
          for (int t = 0; t < kT; ++t) acc[r][t] = dot8_bf16(w[u][r], x[u][t], acc[r][t]);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < kR; ++r)
#pragma unroll
    for (int t = 0; t < kT; ++t) {
      float v = acc[r][t];
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
      const int n = n0 + r;
      if (lane == 0 && n < N) {
        const int64_t at = (int64_t)t * N + n;
        if (out_f32) {
          static_cast<float*>(Y)[at] = v;
        } else {
          if (C) v += __uint_as_float((uint32_t)C[at] << 16);
          static_cast<uint16_t*>(Y)[at] = (uint16_t)f32_to_bf16_rne(v);
        }
      }
    }
}

// x[t] = embed[clamp(tokens[t])], one workgroup per token, 16-byte copies.
__global__ __launch_bounds__(kThreads) void embed_kernel(int V, int d, const int32_t* tokens,
                                                         const uint16_t* embed, uint16_t* x) {
  const int t = blockIdx.x;
  int tok = tokens[t];
  tok = tok < 0 ? 0 : (tok >= V ? V - 1 : tok);
  const uint4* src = reinterpret_cast<const uint4*>(embed + (int64_t)tok * d);
  uint4* dst = reinterpret_cast<uint4*>(x + (int64_t)t * d);
  for (int i = threadIdx.x; i < d / 8; i += kThreads) dst[i] = src[i];
}

// Sum over the workgroup in a fixed order (wavefront butterflies, then the
// four wavefront sums in order); every thread gets the total.
__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

__device__ __forceinline__ float block_max(float v, float* red) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// Per token row: if delta, x = bf16(x + delta) (written back); then
// out = bf16(x / sqrt(mean(x^2) + eps) * g), in fp32.  d is a multiple of 8
// and at most 8 * 256 * 4 (four 8-element chunks per thread).
__global__ __launch_bounds__(kThreads) void add_rmsnorm_kernel(int d, uint16_t* x,
                                                               const uint16_t* delta,
                                                               const uint16_t* g, float eps,
                                                               uint16_t* out) {
  __shared__ float red[4];
  const int t = blockIdx.x;
  uint4* xr = reinterpret_cast<uint4*>(x + (int64_t)t * d);
  const uint4* dr = delta ? reinterpret_cast<const uint4*>(delta + (int64_t)t * d) : nullptr;
  const int n8 = d / 8;
  float v[4][8];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int i = threadIdx.x + c * kThreads;
    if (i >= n8) break;
    uint4 a = xr[i];
    uint32_t w[4] = {a.x, a.y, a.z, a.w};
    if (dr) {
      const uint4 b = dr[i];
      const uint32_t u[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const float lo = bf16_to_f32(w[p] & 0xffffu) + bf16_to_f32(u[p] & 0xffffu);
        const float hi = bf16_to_f32(w[p] >> 16) + bf16_to_f32(u[p] >> 16);
        w[p] = f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
      }
      xr[i] = make_uint4(w[0], w[1], w[2], w[3]);
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      v[c][2 * p] = bf16_to_f32(w[p] & 0xffffu);
      v[c][2 * p + 1] = bf16_to_f32(w[p] >> 16);
      ss = fmaf(v[c][2 * p], v[c][2 * p], ss);
      ss = fmaf(v[c][2 * p + 1], v[c][2 * p + 1], ss);
    }
  }
  const float inv = 1.0f / sqrtf(block_sum(ss, red) / (float)d + eps);
  const uint4* gr = reinterpret_cast<const uint4*>(g);
  uint4* orow = reinterpret_cast<uint4*>(out + (int64_t)t * d);
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int i = threadIdx.x + c * kThreads;
    if (i >= n8) break;
    const uint4 gv = gr[i];
    const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w};
    uint32_t o[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const float lo = v[c][2 * p] * inv * bf16_to_f32(gw[p] & 0xffffu);
      const float hi = v[c][2 * p + 1] * inv * bf16_to_f32(gw[p] >> 16);
      o[p] = f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
    }
    orow[i] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// Rotary positions on q (in place in qkv) and k, and the cache append of k
// and v, for token t at position pos0 + t.  Element i < Dh/2 of a head pairs
// with i + Dh/2; the angle p * base^(-2i/Dh) and its sine and cosine are
// taken in fp64, the rotation in fp32.  qkv row: [q (H*Dh) | k | v].
__global__ __launch_bounds__(kThreads) void rope_kv_kernel(int H, int Dh, int pos0, float base,
                                                           uint16_t* qkv, uint16_t* k_cache,
                                                           uint16_t* v_cache) {
  __shared__ float cs[kMaxHeadDim / 2][2];
  const int t = blockIdx.x;
  const int d = H * Dh, half = Dh / 2;
  const int p = pos0 + t;
  for (int i = threadIdx.x; i < half; i += kThreads) {
    const double ang = (double)p * pow((double)base, -2.0 * (double)i / (double)Dh);
    cs[i][0] = (float)cos(ang);
    cs[i][1] = (float)sin(ang);
  }
  __syncthreads();
  uint16_t* q = qkv + (int64_t)t * 3 * d;
  const uint16_t* k = q + d;
  const uint16_t* v = q + 2 * d;
  uint16_t* kc = k_cache + (int64_t)p * d;
  uint16_t* vc = v_cache + (int64_t)p * d;
  for (int j = threadIdx.x; j < H * half; j += kThreads) {
    const int h = j / half, i = j % half;
    const float c = cs[i][0], s = cs[i][1];
    const int a = h * Dh + i, b = a + half;
    const float qa = bf16_to_f32(q[a]), qb = bf16_to_f32(q[b]);
    q[a] = (uint16_t)f32_to_bf16_rne(qa * c - qb * s);
    q[b] = (uint16_t)f32_to_bf16_rne(qb * c + qa * s);
    const float ka = bf16_to_f32(k[a]), kb = bf16_to_f32(k[b]);
    kc[a] = (uint16_t)f32_to_bf16_rne(ka * c - kb * s);
    kc[b] = (uint16_t)f32_to_bf16_rne(kb * c + ka * s);
  }
  const uint4* vs = reinterpret_cast<const uint4*>(v);
  uint4* vd = reinterpret_cast<uint4*>(vc);
  for (int i = threadIdx.x; i < d / 8; i += kThreads) vd[i] = vs[i];
}

// Causal attention of token t (position pos0 + t), head h, over cache
// positions 0 .. pos0 + t: scores q.k / sqrt(Dh) (bf16 products summed in
// fp32), softmax in fp32, output bf16.  One workgroup per (head, token).
// Scores: a thread per key, the key row's 16-byte chunks all loaded before
// use.  Output: a thread per (8-dimension chunk, key stripe), 16-byte value
// loads eight keys at a time, the stripes' partial sums added in stripe order.
template <int kDh>
__global__ __launch_bounds__(kThreads) void attention_kernel(int H, int pos0, const uint16_t* qkv,
                                                             const uint16_t* k_cache,
                                                             const uint16_t* v_cache,
                                                             uint16_t* out) {
  constexpr int kChunks = kDh / 8;
  constexpr int kStripes = kThreads / kChunks;
  __shared__ float score[EMOE_DECODER_MAX_POSITIONS];
  __shared__ uint32_t qs[kDh / 2];
  __shared__ float part[kStripes][kDh];
  __shared__ float red[4];
  const int h = blockIdx.x, t = blockIdx.y;
  const int d = H * kDh;
  const int n = pos0 + t + 1;
  const uint16_t* q = qkv + (int64_t)t * 3 * d + h * kDh;
  for (int i = threadIdx.x; i < kDh / 2; i += kThreads)
    qs[i] = reinterpret_cast<const uint32_t*>(q)[i];
  __syncthreads();
  const float scale = 1.0f / sqrtf((float)kDh);
  float mx = -INFINITY;
  for (int j = threadIdx.x; j < n; j += kThreads) {
    const uint4* kr = reinterpret_cast<const uint4*>(k_cache + (int64_t)j * d + h * kDh);
    uint4 kv[kChunks];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) kv[c] = kr[c];
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const uint32_t kw[4] = {kv[c].x, kv[c].y, kv[c].z, kv[c].w};
#pragma unroll
      for (int p = 0; p < 4; ++p)
        acc[p] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, kw[p]),
                                                 __builtin_bit_cast(bf16x2_t, qs[4 * c + p]),
                                                 acc[p], false);
    }
    const float s = ((acc[0] + acc[1]) + (acc[2] + acc[3])) * scale;
    score[j] = s;
    mx = fmaxf(mx, s);
  }
  mx = block_max(mx, red);
  float sum = 0.f;
  for (int j = threadIdx.x; j < n; j += kThreads) {
    const float e = expf(score[j] - mx);
    score[j] = e;
    sum += e;
  }
  sum = block_sum(sum, red);  // its barriers also publish score[]
  const int chunk = threadIdx.x % kChunks, stripe = threadIdx.x / kChunks;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const uint16_t* vcol = v_cache + h * kDh + chunk * 8;
  // Eight keys' value loads in flight per stripe (a decode step's few
  // hundred keys take two rounds), then the rest one at a time.
  auto add_key = [&](const uint4 a, float pa) {
    const uint32_t aw[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      acc[2 * p] = fmaf(pa, bf16_to_f32(aw[p] & 0xffffu), acc[2 * p]);
      acc[2 * p + 1] = fmaf(pa, bf16_to_f32(aw[p] >> 16), acc[2 * p + 1]);
    }
  };
  constexpr int kVKeys = 8;
  int j = stripe;
  for (; j + (kVKeys - 1) * kStripes < n; j += kVKeys * kStripes) {
    uint4 a[kVKeys];
#pragma unroll
    for (int u = 0; u < kVKeys; ++u)
      a[u] = *reinterpret_cast<const uint4*>(vcol + (int64_t)(j + u * kStripes) * d);
#pragma unroll
    for (int u = 0; u < kVKeys; ++u) add_key(a[u], score[j + u * kStripes]);
  }
  for (; j < n; j += kStripes)
    add_key(*reinterpret_cast<const uint4*>(vcol + (int64_t)j * d), score[j]);
#pragma unroll
  for (int e = 0; e < 8; ++e) part[stripe][chunk * 8 + e] = acc[e];
  __syncthreads();
  for (int i = threadIdx.x; i < kDh; i += kThreads) {
    float o = 0.f;
    for (int st = 0; st < kStripes; ++st) o += part[st][i];
    out[(int64_t)t * d + h * kDh + i] = (uint16_t)f32_to_bf16_rne(o / sum);
  }
}

// Greedy next token: index of the largest logit, ties to the lower index.
__global__ __launch_bounds__(1024) void argmax_kernel(int V, const float* logits, int32_t* out) {
  __shared__ float bv[16];
  __shared__ int bi[16];
  float best = -INFINITY;
  int idx = 0x7fffffff;
  for (int i = threadIdx.x; i < V; i += 1024) {
    const float v = logits[i];
    if (v > best) {
      best = v;
      idx = i;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(best, off);
    const int oi = __shfl_xor(idx, off);
    if (ov > best || (ov == best && oi < idx)) {
      best = ov;
      idx = oi;
    }
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    bv[w] = best;
    bi[w] = idx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < 16; ++k)
      if (bv[k] > best || (bv[k] == best && bi[k] < idx)) {
        best = bv[k];
        idx = bi[k];
      }
    *out = idx < V ? idx : 0;
  }
}

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

int32_t check_decoder_dims(const emoe_decoder_dims* dd) {
  if (!dd) return report_error(EMOE_EINVAL, "dims is NULL");
  const int32_t st = emoe_check_dims(&dd->moe);
  if (st) return st;
  const int d = dd->moe.d_model;
  const int dh = dd->head_dim;
  if (dd->n_layers < 1 || dd->n_heads < 1 || (dh != 64 && dh != 128 && dh != 256) ||
      dd->n_heads * dh != d)
    return report_error(EMOE_ESHAPE,
                        "need n_layers >= 1 and n_heads * head_dim == d_model with head_dim "
                        "64, 128 or 256 (got %d x %d for d_model %d)", dd->n_heads, dh, d);
  if (d > 8 * kThreads * 4) return report_error(EMOE_ESHAPE, "d_model %d above %d", d, 8 * kThreads * 4);
  if (dd->vocab < 1) return report_error(EMOE_ESHAPE, "vocab %d < 1", dd->vocab);
  if (dd->max_positions < 1 || dd->max_positions > EMOE_DECODER_MAX_POSITIONS)
    return report_error(EMOE_ESHAPE, "max_positions %d outside [1, %d]", dd->max_positions,
                        EMOE_DECODER_MAX_POSITIONS);
  if (!(dd->rope_base > 1.0f) || !(dd->rms_eps >= 0.0f))
    return report_error(EMOE_EINVAL, "rope_base must exceed 1 and rms_eps be >= 0");
  return EMOE_OK;
}

struct WsLayout {
  size_t x0, x1, n, qkv, attn, moe_y, moe_ws, moe_ws_bytes, total;
};

WsLayout decoder_ws_layout(const emoe_decoder_dims& dd, int T) {
  WsLayout L{};
  const size_t d = dd.moe.d_model;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align_up(bytes);
    return at;
  };
  L.x0 = take((size_t)T * d * 2);
  L.x1 = take((size_t)T * d * 2);
  L.n = take((size_t)T * d * 2);
  L.qkv = take((size_t)T * 3 * d * 2);
  L.attn = take((size_t)T * d * 2);
  L.moe_y = take((size_t)T * d * 2);
  L.moe_ws_bytes = emoe_workspace_bytes(&dd.moe, T);
  L.moe_ws = take(L.moe_ws_bytes);
  L.total = off;
  return L;
}

const char* rocblas_name(rocblas_status s) { return rocblas_status_to_string(s); }

}  // namespace

struct emoe_decoder {
  emoe_decoder_dims dims;
  const uint16_t* embed = nullptr;
  const uint16_t* lm_head = nullptr;
  const uint16_t* final_norm = nullptr;
  std::vector<const uint16_t*> attn_norm, wqkv, wo, moe_norm, w_router;
  std::vector<emoe_cache*> caches;
  uint16_t* kv = nullptr;
  rocblas_handle blas = nullptr;
};

namespace {

// Y[T][N] (+ C) = X[T][K] W[N][K]^T with bf16 inputs, fp32 accumulation.
// out_f32 selects an fp32 output (C unused); otherwise bf16 out with
// Y = X W^T + C when C is given.
int32_t dense(emoe_decoder* dec, int T, int N, int K, const uint16_t* X, const uint16_t* W,
              const uint16_t* C, void* Y, bool out_f32, hipStream_t stream) {
  if (T <= kDenseMaxTokens && K % 8 == 0) {
    // Decode steps: the weight-streaming GEMV, two rows per wavefront when
    // that still gives every CU a workgroup or two, else one.
    const int per_wg_2 = 2 * (kThreads / 64);
    const bool two = (N + per_wg_2 - 1) / per_wg_2 >= 256;
    const int per_wg = two ? per_wg_2 : kThreads / 64;
    const dim3 grid((N + per_wg - 1) / per_wg);
    const uint16_t* c = out_f32 ? nullptr : C;
    const int f32 = out_f32 ? 1 : 0;
#define DENSE_CASE(R, TT)                                                                        \
  hipLaunchKernelGGL((dense_gemv_kernel<R, TT>), grid, dim3(kThreads), 0, stream, N, K, X, W, c, Y, \
                     f32)
    switch ((two ? 8 : 0) + T) {
      case 1: DENSE_CASE(1, 1); break;
      case 2: DENSE_CASE(1, 2); break;
      case 3: DENSE_CASE(1, 3); break;
      case 4: DENSE_CASE(1, 4); break;
      case 9: DENSE_CASE(2, 1); break;
      case 10: DENSE_CASE(2, 2); break;
      case 11: DENSE_CASE(2, 3); break;
      default: DENSE_CASE(2, 4); break;
    }
#undef DENSE_CASE
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return report_error(EMOE_EHIP, "dense_gemv_kernel launch: %s", hipGetErrorString(e));
    return EMOE_OK;
  }
  const float alpha = 1.0f, beta = (C && !out_f32) ? 1.0f : 0.0f;
  const rocblas_datatype io = out_f32 ? rocblas_datatype_f32_r : rocblas_datatype_bf16_r;
  const void* c = (C && !out_f32) ? static_cast<const void*>(C) : static_cast<const void*>(Y);
  const rocblas_status st = rocblas_gemm_ex(
      dec->blas, rocblas_operation_transpose, rocblas_operation_none, N, T, K, &alpha, W,
      rocblas_datatype_bf16_r, K, X, rocblas_datatype_bf16_r, K, &beta, c, io, N, Y, io, N,
      rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  if (st != rocblas_status_success)
    return report_error(EMOE_EHIP, "rocblas_gemm_ex (%d x %d x %d): %s", N, T, K, rocblas_name(st));
  return EMOE_OK;
}

#define DEC_LAUNCH(...)                                                                 \
  do {                                                                                  \
    hipLaunchKernelGGL(__VA_ARGS__);                                                    \
    const hipError_t e_ = hipGetLastError();                                            \
    if (e_ != hipSuccess) return report_error(EMOE_EHIP, "decoder kernel launch: %s",   \
                                              hipGetErrorString(e_));                   \
  } while (0)

}  // namespace

extern "C" {

size_t emoe_decoder_kv_bytes(const emoe_decoder_dims* dims) {
  if (check_decoder_dims(dims) != EMOE_OK) return 0;
  return (size_t)dims->n_layers * 2 * dims->max_positions * dims->moe.d_model * 2;
}

size_t emoe_decoder_workspace_bytes(const emoe_decoder_dims* dims, int32_t max_tokens) {
  if (check_decoder_dims(dims) != EMOE_OK || max_tokens < 1) return 0;
  return decoder_ws_layout(*dims, max_tokens).total;
}

int32_t emoe_decoder_create(const emoe_decoder_dims* dims, const emoe_decoder_weights* w,
                            emoe_cache* const* caches, void* kv_cache, emoe_decoder** out) {
  int32_t st = check_decoder_dims(dims);
  if (st) return st;
  if (!w || !caches || !kv_cache || !out) return report_error(EMOE_EINVAL, "NULL argument");
  *out = nullptr;
  const int L = dims->n_layers;
  if (!w->embed || !w->lm_head || !w->final_norm || !w->attn_norm || !w->wqkv || !w->wo ||
      !w->moe_norm || !w->w_router)
    return report_error(EMOE_EINVAL, "NULL weight pointer");
  for (int l = 0; l < L; ++l) {
    if (!w->attn_norm[l] || !w->wqkv[l] || !w->wo[l] || !w->moe_norm[l] || !w->w_router[l] ||
        !caches[l])
      return report_error(EMOE_EINVAL, "NULL weight or cache of layer %d", l);
  }
  emoe_decoder* dec = new (std::nothrow) emoe_decoder();
  if (!dec) return report_error(EMOE_EINVAL, "out of host memory");
  dec->dims = *dims;
  dec->embed = w->embed;
  dec->lm_head = w->lm_head;
  dec->final_norm = w->final_norm;
  dec->attn_norm.assign(w->attn_norm, w->attn_norm + L);
  dec->wqkv.assign(w->wqkv, w->wqkv + L);
  dec->wo.assign(w->wo, w->wo + L);
  dec->moe_norm.assign(w->moe_norm, w->moe_norm + L);
  dec->w_router.assign(w->w_router, w->w_router + L);
  dec->caches.assign(caches, caches + L);
  dec->kv = static_cast<uint16_t*>(kv_cache);
  const rocblas_status rs = rocblas_create_handle(&dec->blas);
  if (rs != rocblas_status_success) {
    delete dec;
    return report_error(EMOE_EHIP, "rocblas_create_handle: %s", rocblas_name(rs));
  }
  *out = dec;
  return EMOE_OK;
}

int32_t emoe_decoder_destroy(emoe_decoder* dec) {
  if (!dec) return EMOE_OK;
  if (dec->blas) (void)rocblas_destroy_handle(dec->blas);
  delete dec;
  return EMOE_OK;
}

int32_t emoe_decoder_forward(emoe_decoder* dec, const int32_t* tokens, int32_t T, int32_t pos0,
                             float* logits, int32_t* next_token, void* workspace, size_t ws_bytes,
                             hipStream_t stream, emoe_stats* stats) {
  if (!dec) return report_error(EMOE_EINVAL, "decoder is NULL");
  const emoe_decoder_dims& D = dec->dims;
  if (T < 1 || pos0 < 0 || (int64_t)pos0 + T > D.max_positions)
    return report_error(EMOE_EINVAL, "tokens %d at position %d exceed the cache of %d positions",
                        T, pos0, D.max_positions);
  if (!tokens || !logits || !next_token || !workspace)
    return report_error(EMOE_EINVAL, "NULL tokens, logits, next_token or workspace");
  const WsLayout L = decoder_ws_layout(D, T);
  if (ws_bytes < L.total)
    return report_error(EMOE_EINVAL, "workspace of %zu bytes < %zu needed", ws_bytes, L.total);
  const int d = D.moe.d_model, H = D.n_heads, Dh = D.head_dim;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  uint16_t* xa = reinterpret_cast<uint16_t*>(ws + L.x0);
  uint16_t* xb = reinterpret_cast<uint16_t*>(ws + L.x1);
  uint16_t* n = reinterpret_cast<uint16_t*>(ws + L.n);
  uint16_t* qkv = reinterpret_cast<uint16_t*>(ws + L.qkv);
  uint16_t* attn = reinterpret_cast<uint16_t*>(ws + L.attn);
  uint16_t* moe_y = reinterpret_cast<uint16_t*>(ws + L.moe_y);
  void* moe_ws = ws + L.moe_ws;
  const rocblas_status rs = rocblas_set_stream(dec->blas, stream);
  if (rs != rocblas_status_success)
    return report_error(EMOE_EHIP, "rocblas_set_stream: %s", rocblas_name(rs));

  DEC_LAUNCH(embed_kernel, dim3(T), dim3(kThreads), 0, stream, D.vocab, d, tokens, dec->embed, xa);
  const uint16_t* delta = nullptr;
  const size_t kv_layer = (size_t)2 * D.max_positions * d;
  int32_t st;
  for (int l = 0; l < D.n_layers; ++l) {
    uint16_t* kc = dec->kv + (size_t)l * kv_layer;
    uint16_t* vc = kc + (size_t)D.max_positions * d;
    DEC_LAUNCH(add_rmsnorm_kernel, dim3(T), dim3(kThreads), 0, stream, d, xa, delta,
               dec->attn_norm[l], D.rms_eps, n);
    if ((st = dense(dec, T, 3 * d, d, n, dec->wqkv[l], nullptr, qkv, false, stream))) return st;
    DEC_LAUNCH(rope_kv_kernel, dim3(T), dim3(kThreads), 0, stream, H, Dh, pos0, D.rope_base, qkv,
               kc, vc);
    if (Dh == 64)
      DEC_LAUNCH(attention_kernel<64>, dim3(H, T), dim3(kThreads), 0, stream, H, pos0, qkv, kc, vc,
                 attn);
    else if (Dh == 128)
      DEC_LAUNCH(attention_kernel<128>, dim3(H, T), dim3(kThreads), 0, stream, H, pos0, qkv, kc,
                 vc, attn);
    else
      DEC_LAUNCH(attention_kernel<256>, dim3(H, T), dim3(kThreads), 0, stream, H, pos0, qkv, kc,
                 vc, attn);
    if ((st = dense(dec, T, d, d, attn, dec->wo[l], xa, xb, false, stream))) return st;  // x += attn Wo^T
    std::swap(xa, xb);
    DEC_LAUNCH(add_rmsnorm_kernel, dim3(T), dim3(kThreads), 0, stream, d, xa, nullptr,
               dec->moe_norm[l], D.rms_eps, n);
    if ((st = emoe_moe_forward(dec->caches[l], T, n, dec->w_router[l], nullptr, D.renormalize,
                               EMOE_PATH_AUTO, moe_y, moe_ws, L.moe_ws_bytes, stream, stats)))
      return st;
    delta = moe_y;
  }
  DEC_LAUNCH(add_rmsnorm_kernel, dim3(T), dim3(kThreads), 0, stream, d, xa, delta, dec->final_norm,
             D.rms_eps, n);
  if ((st = dense(dec, 1, D.vocab, d, n + (size_t)(T - 1) * d, dec->lm_head, nullptr, logits, true,
                  stream)))
    return st;
  DEC_LAUNCH(argmax_kernel, dim3(1), dim3(1024), 0, stream, D.vocab, logits, next_token);
  return EMOE_OK;
}

}  // extern "C"
