// Offline conversion (Sec. 3.2, Eq. 3): symmetric group-128 INT4 quantization
// of gate, up and down, packed into the record layout of common.h.
//
// One wavefront per 16 x 128 tile.  Lane l reads exactly the 32 weights it
// will write as codes (row 16*rb + l%16, inputs 128*g + 32*i + 8*(l/16) + r),
// so the row absmax is a reduction over the four lanes that share a row.
#include "common.h"

namespace emoe {
namespace {

constexpr int kWavesPerBlock = 4;

__global__ __launch_bounds__(256) void quantize_kernel(int d, int f, int tiles_w13,
                                                       int tiles_total, const uint16_t* __restrict__ w_gate,
                                                       const uint16_t* __restrict__ w_up,
                                                       const uint16_t* __restrict__ w_down,
                                                       uint8_t* __restrict__ records,
                                                       int64_t record_bytes,
                                                       int32_t* __restrict__ range_flag) {
  const int lane = lane_id();
  const int tile = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  const int expert = blockIdx.y;
  if (tile >= tiles_total) return;

  const RecordLayout L = record_layout(d, f);
  uint8_t* rec = records + (int64_t)expert * record_bytes;

  // Which matrix, source rows and group this tile covers.
  const uint16_t* src;
  int src_row0, K, rb, g, G;
  int64_t codes_off, scales_off;
  if (tile < tiles_w13) {
    G = d / kGroup;
    K = d;
    rb = tile / G;
    g = tile % G;
    const int b = rb >> 1;
    src = ((rb & 1) ? w_up : w_gate) + (int64_t)expert * f * d;
    src_row0 = b * kTileRows;
    codes_off = L.w13_codes;
    scales_off = L.w13_scales;
  } else {
    const int t = tile - tiles_w13;
    G = f / kGroup;
    K = f;
    rb = t / G;
    g = t % G;
    src = w_down + (int64_t)expert * d * f;
    src_row0 = rb * kTileRows;
    codes_off = L.w2_codes;
    scales_off = L.w2_scales;
  }

  const int n_local = lane & 15;
  const int quarter = lane >> 4;
  const uint16_t* row = src + (int64_t)(src_row0 + n_local) * K + g * kGroup + 8 * quarter;

  float w[32];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint4 v = *reinterpret_cast<const uint4*>(row + 32 * i);
    const uint32_t dw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      w[8 * i + 2 * p] = bf16_to_f32(dw[p] & 0xffffu);
      w[8 * i + 2 * p + 1] = bf16_to_f32(dw[p] >> 16);
    }
  }
  float amax = 0.f;
#pragma unroll
  for (int j = 0; j < 32; ++j) amax = fmaxf(amax, fabsf(w[j]));
  amax = fmaxf(amax, __shfl_xor(amax, 16));
  amax = fmaxf(amax, __shfl_xor(amax, 32));

  const float s32 = amax / 7.0f;  // IEEE fp32 division
  const __half s16h = __float2half_rn(s32);
  const float s16 = __half2float(s16h);
  if (__builtin_isinf(s16) && quarter == 0) atomicOr(range_flag, 1);  // one lane per row
  const bool zero = (amax == 0.f) || (s16 == 0.f);

  uint32_t out[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t dw = 0;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      float q = zero ? 0.f : rintf(w[8 * i + r] / s32);
      q = fminf(fmaxf(q, -8.f), 7.f);
      const uint32_t u = (uint32_t)((int)q + 8);
      dw |= u << (4 * (r >> 1) + 16 * (r & 1));
    }
    out[i] = dw;
  }
  uint8_t* tile_ptr = rec + codes_off + ((int64_t)rb * G + g) * kTileBytes + 16 * lane;
  *reinterpret_cast<uint4*>(tile_ptr) = make_uint4(out[0], out[1], out[2], out[3]);
  if (quarter == 0) {
    const int n = rb * kTileRows + n_local;  // row in this matrix (W13 row order for W13)
    uint16_t* sc = reinterpret_cast<uint16_t*>(rec + scales_off);
    sc[scale_index(n, g, G)] = zero ? (uint16_t)0 : __half_as_ushort(s16h);
  }
}

}  // namespace

hipError_t launch_quantize(int d, int f, int n_experts, const uint16_t* w_gate,
                           const uint16_t* w_up, const uint16_t* w_down, uint8_t* records,
                           int32_t* range_flag, hipStream_t stream) {
  const int tiles_w13 = (2 * f / kTileRows) * (d / kGroup);
  const int tiles_w2 = (d / kTileRows) * (f / kGroup);
  const int tiles = tiles_w13 + tiles_w2;
  const int64_t rec = record_layout(d, f).bytes;
  dim3 grid((tiles + kWavesPerBlock - 1) / kWavesPerBlock, n_experts);
  launch(quantize_kernel, grid, dim3(64 * kWavesPerBlock), stream, d, f, tiles_w13,
                     tiles, w_gate, w_up, w_down, records, rec, range_flag);
  return hipGetLastError();
}

}  // namespace emoe
