// Weight-streaming grouped projections for the few-tokens-per-expert regime
// (decode and small batches), plus the top-k weighted combine.
//
// At one token per expert every packed weight is used once, so the layer is
// bound by HBM bandwidth: these kernels stream the packed int4 tiles with
// 16-byte coalesced loads, issue all loads of a wavefront before using them,
// dequantize in registers and accumulate with v_dot2c_f32_bf16.
//
// In-register dequantization: for a code dword, ((dw >> 4p) & 0x000f000f) |
// 0x43004300 is the bf16 pair (128 + u_2p, 128 + u_2p+1), exact because bf16
// represents the integers 128..143.  With u = q + 8 the dot product over a
// lane's 32 inputs is sum (u - 8) h = sum (128 + u) h - 136 sum h, so each
// group needs one correction with the activations' sum before the per-group
// FP16 scale is applied in fp32 (Sec. 3.2: W_hat = s q, never rounded).
#include "common.h"

namespace emoe {
namespace {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;       // wavefronts per workgroup
constexpr int kTokChunk = 4;    // token rows processed per pass over the weights
constexpr int kBatch = 4;       // tiles per matrix loaded together by one wavefront
constexpr int kDownBatch = 8;   // tiles loaded together by one wavefront (down)
constexpr uint32_t kOnes = 0x3f803f80u;  // bf16 pair (1, 1)

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                        __builtin_bit_cast(bf16x2_t, b), c, false);
}

__device__ __forceinline__ void dequant_dword(uint32_t dw, uint32_t* out) {
#pragma unroll
  for (int p = 0; p < 4; ++p) out[p] = ((dw >> (4 * p)) & 0x000f000fu) | 0x43004300u;
}

// Dot product of one lane's 32 codes of a group (its row, its inputs) with the
// 32 matching activations x (4 x uint4): returns sum (128 + u) x and, when
// want_xs, adds sum x to xs.
__device__ __forceinline__ float lane_group_dot(const uint4 codes, const uint4* x, float& xs,
                                                bool want_xs) {
  const uint32_t c[4] = {codes.x, codes.y, codes.z, codes.w};
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t wp[4];
    dequant_dword(c[i], wp);
    const uint32_t xv[4] = {x[i].x, x[i].y, x[i].z, x[i].w};
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      acc = dot2(wp[p], xv[p], acc);
      if (want_xs) xs = dot2(kOnes, xv[p], xs);
    }
  }
  return acc;
}

__device__ __forceinline__ void load_x32(const uint16_t* row, uint4* x) {
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = *reinterpret_cast<const uint4*>(row + 32 * i);
}

__device__ __forceinline__ float silu_mul(float g, float u) {
  return g / (1.0f + expf(-g)) * u;
}

// ----------------------------------------------------------------- gate/up
// Workgroup = (gate/up row-block pair b, wave expert w); its four wavefronts
// split the input groups round-robin and meet in LDS.  Output: the SwiGLU
// activation phi(g) * u as bf16 at the pair's grouped position.
__global__ __launch_bounds__(256) void gateup_gemv_kernel(int d, int f, int top_k,
                                                          const uint16_t* __restrict__ h,
                                                          GroupView gv, WaveArg wave,
                                                          const uint8_t* __restrict__ slot_bank,
                                                          int64_t record_bytes,
                                                          uint16_t* __restrict__ act) {
  __shared__ float red[kWaves][kTokChunk][2][16];
  const int lane = lane_id();
  const int wi = threadIdx.x >> 6;
  int expert, slot;
  if (!resolve_wave_expert(wave, gv, blockIdx.y, expert, slot)) return;
  const int begin = gv.offsets[expert];
  const int end = gv.offsets[expert + 1];

  const int G = d / kGroup;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* rec = slot_bank + (int64_t)slot * record_bytes;
  const int b = blockIdx.x;
  const uint8_t* gate_codes = rec + L.w13_codes + (int64_t)(2 * b) * G * kTileBytes + 16 * lane;
  const uint8_t* up_codes = gate_codes + (int64_t)G * kTileBytes;
  const int n_local = lane & 15;
  const int quarter = lane >> 4;
  const uint16_t* scales = reinterpret_cast<const uint16_t*>(rec + L.w13_scales);
  const uint16_t* gate_sc = scales + (int64_t)(32 * b + n_local) * G;
  const uint16_t* up_sc = scales + (int64_t)(32 * b + 16 + n_local) * G;

  for (int m0 = begin; m0 < end; m0 += kTokChunk) {
    const int mc = min(kTokChunk, end - m0);
    const uint16_t* xrow[kTokChunk];
#pragma unroll
    for (int m = 0; m < kTokChunk; ++m) {
      const int t = m < mc ? gv.sorted_pairs[m0 + m] / top_k : 0;
      xrow[m] = h + (int64_t)t * d + 8 * quarter;
    }
    float accg[kTokChunk], accu[kTokChunk];
#pragma unroll
    for (int m = 0; m < kTokChunk; ++m) accg[m] = accu[m] = 0.f;

    for (int g0 = wi; g0 < G; g0 += kWaves * kBatch) {
      uint4 cg[kBatch], cu[kBatch];
      float sg[kBatch], su[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int g = g0 + kWaves * j;
        if (g < G) {
          cg[j] = *reinterpret_cast<const uint4*>(gate_codes + (int64_t)g * kTileBytes);
          cu[j] = *reinterpret_cast<const uint4*>(up_codes + (int64_t)g * kTileBytes);
          sg[j] = half_bits_to_f32(gate_sc[g]);
          su[j] = half_bits_to_f32(up_sc[g]);
        }
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int g = g0 + kWaves * j;
        if (g >= G) break;
#pragma unroll
        for (int m = 0; m < kTokChunk; ++m) {
          if (m >= mc) break;
          uint4 x[4];
          load_x32(xrow[m] + g * kGroup, x);
          float xs = 0.f;
          const float pg = lane_group_dot(cg[j], x, xs, true);
          const float pu = lane_group_dot(cu[j], x, xs, false);
          accg[m] = fmaf(sg[j], fmaf(-136.f, xs, pg), accg[m]);
          accu[m] = fmaf(su[j], fmaf(-136.f, xs, pu), accu[m]);
        }
      }
    }
#pragma unroll
    for (int m = 0; m < kTokChunk; ++m) {
      accg[m] += __shfl_xor(accg[m], 16);
      accg[m] += __shfl_xor(accg[m], 32);
      accu[m] += __shfl_xor(accu[m], 16);
      accu[m] += __shfl_xor(accu[m], 32);
      if (quarter == 0) {
        red[wi][m][0][n_local] = accg[m];
        red[wi][m][1][n_local] = accu[m];
      }
    }
    __syncthreads();
    if (wi == 0) {
      const int m = lane >> 4;
      if (m < mc) {
        float g = 0.f, u = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
          g += red[w][m][0][n_local];
          u += red[w][m][1][n_local];
        }
        act[(int64_t)(m0 + m) * f + 16 * b + n_local] = (uint16_t)f32_to_bf16_rne(silu_mul(g, u));
      }
    }
    __syncthreads();
  }
}

// ----------------------------------------------------------------- down
// Workgroup = (four 16-row blocks of the output, wave expert w); each
// wavefront owns one row block over the whole input (d_ff).  Output: fp32
// expert output per pair id.
__global__ __launch_bounds__(256) void down_gemv_kernel(int d, int f, int top_k,
                                                        const uint16_t* __restrict__ act,
                                                        GroupView gv, WaveArg wave,
                                                        const uint8_t* __restrict__ slot_bank,
                                                        int64_t record_bytes,
                                                        float* __restrict__ pair_out) {
  const int lane = lane_id();
  const int wi = threadIdx.x >> 6;
  int expert, slot;
  if (!resolve_wave_expert(wave, gv, blockIdx.y, expert, slot)) return;
  const int begin = gv.offsets[expert];
  const int end = gv.offsets[expert + 1];

  const int G = f / kGroup;
  const int rb = blockIdx.x * kWaves + wi;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* rec = slot_bank + (int64_t)slot * record_bytes;
  const uint8_t* codes = rec + L.w2_codes + (int64_t)rb * G * kTileBytes + 16 * lane;
  const int n_local = lane & 15;
  const int quarter = lane >> 4;
  const uint16_t* sc = reinterpret_cast<const uint16_t*>(rec + L.w2_scales) +
                       (int64_t)(16 * rb + n_local) * G;

  for (int m0 = begin; m0 < end; m0 += kTokChunk) {
    const int mc = min(kTokChunk, end - m0);
    float acc[kTokChunk];
#pragma unroll
    for (int m = 0; m < kTokChunk; ++m) acc[m] = 0.f;
    for (int g0 = 0; g0 < G; g0 += kDownBatch) {
      uint4 c[kDownBatch];
      float s[kDownBatch];
#pragma unroll
      for (int j = 0; j < kDownBatch; ++j) {
        if (g0 + j < G) {
          c[j] = *reinterpret_cast<const uint4*>(codes + (int64_t)(g0 + j) * kTileBytes);
          s[j] = half_bits_to_f32(sc[g0 + j]);
        }
      }
#pragma unroll
      for (int j = 0; j < kDownBatch; ++j) {
        const int g = g0 + j;
        if (g >= G) break;
#pragma unroll
        for (int m = 0; m < kTokChunk; ++m) {
          if (m >= mc) break;
          uint4 x[4];
          load_x32(act + (int64_t)(m0 + m) * f + g * kGroup + 8 * quarter, x);
          float xs = 0.f;
          const float p = lane_group_dot(c[j], x, xs, true);
          acc[m] = fmaf(s[j], fmaf(-136.f, xs, p), acc[m]);
        }
      }
    }
#pragma unroll
    for (int m = 0; m < kTokChunk; ++m) {
      acc[m] += __shfl_xor(acc[m], 16);
      acc[m] += __shfl_xor(acc[m], 32);
      if (quarter == 0 && m < mc) {
        const int pi = gv.sorted_pairs[m0 + m];
        pair_out[(int64_t)pi * d + 16 * rb + n_local] = acc[m];
      }
    }
  }
}

// ----------------------------------------------------------------- combine
// y[t] = sum_j p[t][j] * o[t*k + j], j in rank order, fp32, rounded to bf16.
__global__ __launch_bounds__(256) void combine_kernel(int tokens, int d, int top_k,
                                                      const float* __restrict__ topk_w,
                                                      const float* __restrict__ pair_out,
                                                      uint16_t* __restrict__ y) {
  const int quads = d / 4;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)tokens * quads) return;
  const int t = (int)(idx / quads);
  const int c = (int)(idx % quads);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < top_k; ++j) {
    const int64_t pi = (int64_t)t * top_k + j;
    const float w = topk_w[pi];
    const float4 o = *reinterpret_cast<const float4*>(pair_out + pi * d + 4 * c);
    acc.x = fmaf(w, o.x, acc.x);
    acc.y = fmaf(w, o.y, acc.y);
    acc.z = fmaf(w, o.z, acc.z);
    acc.w = fmaf(w, o.w, acc.w);
  }
  const uint32_t lo = f32_to_bf16_rne(acc.x) | (f32_to_bf16_rne(acc.y) << 16);
  const uint32_t hi = f32_to_bf16_rne(acc.z) | (f32_to_bf16_rne(acc.w) << 16);
  *reinterpret_cast<uint2*>(y + (int64_t)t * d + 4 * c) = make_uint2(lo, hi);
}

}  // namespace

hipError_t launch_gateup_gemv(int d, int f, int top_k, int pairs, int n_experts,
                              const uint16_t* h, const GroupView& gv, const WaveArg& wave,
                              const uint8_t* slot_bank, int64_t record_bytes, uint16_t* act,
                              hipStream_t stream) {
  const int ge = grid_experts(wave, n_experts, pairs);
  if (ge == 0) return hipSuccess;
  dim3 grid(f / kTileRows, ge);
  launch(gateup_gemv_kernel, grid, dim3(64 * kWaves), stream, d, f, top_k, h, gv,
                     wave, slot_bank, record_bytes, act);
  return hipGetLastError();
}

hipError_t launch_down_gemv(int d, int f, int top_k, int pairs, int n_experts,
                            const uint16_t* act, const GroupView& gv, const WaveArg& wave,
                            const uint8_t* slot_bank, int64_t record_bytes, float* pair_out,
                            hipStream_t stream) {
  const int ge = grid_experts(wave, n_experts, pairs);
  if (ge == 0) return hipSuccess;
  dim3 grid(d / (kTileRows * kWaves), ge);
  launch(down_gemv_kernel, grid, dim3(64 * kWaves), stream, d, f, top_k, act, gv,
                     wave, slot_bank, record_bytes, pair_out);
  return hipGetLastError();
}

hipError_t launch_combine(int tokens, int d, int top_k, const float* topk_w,
                          const float* pair_out, uint16_t* y, hipStream_t stream) {
  const int64_t n = (int64_t)tokens * (d / 4);
  if (n == 0) return hipSuccess;
  launch(combine_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), stream, tokens, d, top_k,
         topk_w, pair_out, y);
  return hipGetLastError();
}

}  // namespace emoe
