// Weight-streaming grouped projections for the few-tokens-per-expert regime
// (decode and small batches), plus the top-k weighted combine.
//
// At one token per expert every packed weight is used once, so the layer is
// bound by HBM bandwidth: these kernels stream the packed int4 tiles with
// 16-byte coalesced loads, issue a wavefront's loads before using them,
// dequantize in registers and accumulate with v_dot2c_f32_bf16
// (device_gemv.h).
#include "device_gemv.h"

namespace emoe {
namespace {

// Workgroup = (gate/up row-block pair b, row chunk y: up to kGemvRows rows of
// one wave expert, so an expert with many rows spreads over many
// workgroups).  Output: the SwiGLU activation phi(g) * u as bf16 at each
// pair's grouped position.
__global__ __launch_bounds__(256) void gateup_gemv_kernel(int d, int f, int top_k,
                                                          const uint16_t* __restrict__ h,
                                                          GroupView gv, WaveArg wave,
                                                          const uint8_t* __restrict__ slot_bank,
                                                          int64_t record_bytes,
                                                          uint16_t* __restrict__ act) {
  __shared__ GateUpShared sh;
  int expert, slot, begin, end;
  if (!resolve_wave_chunk(wave, gv, blockIdx.y, expert, slot, begin, end)) return;
  gateup_block<false>(sh, d, f, top_k, h, gv.sorted_pairs, begin, end,
                      slot_bank + (int64_t)slot * record_bytes, blockIdx.x, act);
}

// Workgroup = (four 16-row blocks of the output, row chunk y as above); each
// wavefront owns one row block over the whole input (d_ff).  Output: fp32
// expert output per pair id.
__global__ __launch_bounds__(256) void down_gemv_kernel(int d, int f, int top_k,
                                                        const uint16_t* __restrict__ act,
                                                        GroupView gv, WaveArg wave,
                                                        const uint8_t* __restrict__ slot_bank,
                                                        int64_t record_bytes,
                                                        float* __restrict__ pair_out) {
  (void)top_k;
  const int lane = lane_id();
  int expert, slot, begin, end;
  if (!resolve_wave_chunk(wave, gv, blockIdx.y, expert, slot, begin, end)) return;
  const int G = f / kGroup;
  const int rb = blockIdx.x * kGemvWaves + (threadIdx.x >> 6);
  const uint8_t* rec = slot_bank + (int64_t)slot * record_bytes;

  for (int m0 = begin; m0 < end; m0 += kTokChunk) {
    const int mc = min(kTokChunk, end - m0);
    auto xload = [&](int m, int k) {
      return *reinterpret_cast<const uint4*>(act + (int64_t)(m0 + m) * f + k);
    };
    float acc[kTokChunk][4];
#pragma unroll
    for (int m = 0; m < kTokChunk; ++m)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[m][c] = 0.f;
    for (int g0 = 0; g0 < G; g0 += kDownBatch) {
      DownBatch bt;
      down_load_batch(rec, d, f, rb, g0, bt);
      down_apply_batch(bt, f, g0, xload, mc, acc);
    }
#pragma unroll
    for (int m = 0; m < kTokChunk; ++m) {
      const float o = down_class_total(acc[m]);
      if (lane < 16 && m < mc) {
        const int pi = gv.sorted_pairs[m0 + m];
        pair_out[(int64_t)pi * d + 16 * rb + lane] = o;
      }
    }
  }
}

// y[t] = sum_j p[t][j] * o[t*k + j], j in rank order, fp32, rounded to bf16.
// The pair outputs o are fp32 (kBf16 = false) or bf16.
template <bool kBf16>
__global__ __launch_bounds__(256) void combine_kernel(int tokens, int d, int top_k,
                                                      const float* __restrict__ topk_w,
                                                      const void* __restrict__ pair_out,
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
    float4 o;
    if (kBf16) {
      const uint2 v = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(pair_out) + pi * d + 4 * c);
      o = make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                      __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
    } else {
      o = *reinterpret_cast<const float4*>(static_cast<const float*>(pair_out) + pi * d + 4 * c);
    }
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
  const int gc = grid_chunks(wave, n_experts, pairs);
  if (gc == 0) return hipSuccess;
  launch(gateup_gemv_kernel, dim3(f / kTileRows, gc), dim3(64 * kGemvWaves), stream, d, f, top_k,
         h, gv, wave, slot_bank, record_bytes, act);
  return hipGetLastError();
}

hipError_t launch_down_gemv(int d, int f, int top_k, int pairs, int n_experts,
                            const uint16_t* act, const GroupView& gv, const WaveArg& wave,
                            const uint8_t* slot_bank, int64_t record_bytes, float* pair_out,
                            hipStream_t stream) {
  const int gc = grid_chunks(wave, n_experts, pairs);
  if (gc == 0) return hipSuccess;
  launch(down_gemv_kernel, dim3(d / (kTileRows * kGemvWaves), gc), dim3(64 * kGemvWaves), stream,
         d, f, top_k, act, gv, wave, slot_bank, record_bytes, pair_out);
  return hipGetLastError();
}

hipError_t launch_combine(int tokens, int d, int top_k, const float* topk_w, const void* pair_out,
                          bool pair_out_bf16, uint16_t* y, hipStream_t stream) {
  const int64_t n = (int64_t)tokens * (d / 4);
  if (n == 0) return hipSuccess;
  const dim3 grid((unsigned)((n + 255) / 256));
  if (pair_out_bf16)
    launch(combine_kernel<true>, grid, dim3(256), stream, tokens, d, top_k, topk_w, pair_out, y);
  else
    launch(combine_kernel<false>, grid, dim3(256), stream, tokens, d, top_k, topk_w, pair_out, y);
  return hipGetLastError();
}

}  // namespace emoe
