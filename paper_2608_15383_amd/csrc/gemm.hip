// Grouped projections on bf16 MFMA for the many-tokens-per-expert regime
// (prefill / large batches), where each expert's projection is a dense
// contraction over its token rows.
//
// A workgroup owns one row-tile (up to 64 token rows of one expert, grouped
// order) and one column tile of the expert's weights.  Token rows are staged
// group by group (128 inputs) in LDS, double buffered, together with their
// per-group sums.  Each wavefront loads its weight tiles straight from the
// packed record: one coalesced 16-byte load per lane per tile, whose four
// dwords expand in registers to the four B operands of
// v_mfma_f32_16x16x32_bf16 (layout in common.h).  The codes enter the MFMA as
// bf16 (128 + u); per group and output the fp32 result is corrected by
// -136 * (row sum) and scaled by the FP16 group scale in fp32, so the
// dequantized weight s * q is never rounded (Sec. 3.2).
#include "common.h"

namespace emoe {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kRows = kMfmaRows;         // 64 token rows per tile
constexpr int kLdsStride = kGroup + 8;   // staged row length in bf16 (16-byte pad)

__device__ __forceinline__ bf16x8_t dequant_b(uint32_t dw) {
  uint32_t p[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) p[j] = ((dw >> (4 * j)) & 0x000f000fu) | 0x43004300u;
  return __builtin_bit_cast(bf16x8_t, make_uint4(p[0], p[1], p[2], p[3]));
}

__device__ __forceinline__ float bf16x8_sum(const uint4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) s += bf16_to_f32(w[j] & 0xffffu) + bf16_to_f32(w[j] >> 16);
  return s;
}

template <bool kGateUp>
__global__ __launch_bounds__(256) void grouped_mfma_kernel(
    int d, int f, int top_k, int n_experts, const uint16_t* __restrict__ x, GroupView gv,
    WaveArg wave, const uint8_t* __restrict__ slot_bank, int64_t record_bytes,
    uint16_t* __restrict__ act_out, float* __restrict__ pair_out) {
  // 16-row weight blocks per wavefront: gate/up takes two (gate, up) pairs.
  constexpr int NPW = kGateUp ? 4 : 2;
  __shared__ __attribute__((aligned(16))) uint16_t As[2][kRows][kLdsStride];
  __shared__ __attribute__((aligned(16))) float hs[2][kRows];

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wi = tid >> 6;

  // Row tile -> expert (largest e with tile_offsets[e] <= tile).
  const int tile = blockIdx.y;
  if (tile >= gv.tile_offsets[n_experts]) return;
  int lo = 0, hi = n_experts;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (gv.tile_offsets[mid] <= tile) lo = mid; else hi = mid;
  }
  const int expert = lo;
  const int slot = wave.n < 0 ? expert : (int)wave.slot_of[expert];
  if (slot < 0) return;  // expert not in this wave
  const int row0 = gv.offsets[expert] + kRows * (tile - gv.tile_offsets[expert]);
  const int rows = min(kRows, gv.offsets[expert + 1] - row0);

  const int K = kGateUp ? d : f;
  const int G = K / kGroup;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* rec = slot_bank + (int64_t)slot * record_bytes;
  const uint8_t* codes = rec + (kGateUp ? L.w13_codes : L.w2_codes);
  const uint16_t* scales = reinterpret_cast<const uint16_t*>(rec + (kGateUp ? L.w13_scales : L.w2_scales));
  const int rb0 = NPW * (blockIdx.x * kWaves + wi);
  const int n_local = lane & 15;
  const int quarter = lane >> 4;

  // Staging assignment: thread -> (row m, 32-input quarter c) of the group.
  const int sm = tid >> 2;
  const int sc = tid & 3;
  const uint16_t* src = nullptr;
  if (sm < rows) {
    if (kGateUp) {
      const int t = gv.sorted_pairs[row0 + sm] / top_k;
      src = x + (int64_t)t * d;
    } else {
      src = x + (int64_t)(row0 + sm) * f;
    }
    src += 32 * sc;
  }
  uint4 stage[4];
  auto fetch = [&](int g) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      stage[i] = src ? *reinterpret_cast<const uint4*>(src + g * kGroup + 8 * i)
                     : make_uint4(0u, 0u, 0u, 0u);
  };
  auto commit = [&](int buf) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<uint4*>(&As[buf][sm][32 * sc + 8 * i]) = stage[i];
      s += bf16x8_sum(stage[i]);
    }
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    if (sc == 0) hs[buf][sm] = s;
  };

  f32x4_t acc[NPW][4];
#pragma unroll
  for (int r = 0; r < NPW; ++r)
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) acc[r][mi] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  fetch(0);
  commit(0);
  __syncthreads();

  for (int g = 0; g < G; ++g) {
    const int buf = g & 1;
    if (g + 1 < G) fetch(g + 1);
    uint4 wc[NPW];
    float ws[NPW];
#pragma unroll
    for (int r = 0; r < NPW; ++r) {
      wc[r] = *reinterpret_cast<const uint4*>(codes + ((int64_t)(rb0 + r) * G + g) * kTileBytes +
                                              16 * lane);
      ws[r] = half_bits_to_f32(scales[(int64_t)(16 * (rb0 + r) + n_local) * G + g]);
    }
    f32x4_t tmp[NPW][4];
#pragma unroll
    for (int r = 0; r < NPW; ++r)
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) tmp[r][mi] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bf16x8_t a[4];
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
        a[mi] = *reinterpret_cast<const bf16x8_t*>(&As[buf][16 * mi + n_local][32 * i + 8 * quarter]);
#pragma unroll
      for (int r = 0; r < NPW; ++r) {
        const uint32_t dw = i == 0 ? wc[r].x : i == 1 ? wc[r].y : i == 2 ? wc[r].z : wc[r].w;
        const bf16x8_t b = dequant_b(dw);
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
          tmp[r][mi] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mi], b, tmp[r][mi], 0, 0, 0);
      }
    }
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
      const float4 hv = *reinterpret_cast<const float4*>(&hs[buf][16 * mi + 4 * quarter]);
      const float hj[4] = {hv.x, hv.y, hv.z, hv.w};
#pragma unroll
      for (int r = 0; r < NPW; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[r][mi][j] = fmaf(ws[r], fmaf(-136.f, hj[j], tmp[r][mi][j]), acc[r][mi][j]);
    }
    if (g + 1 < G) commit(buf ^ 1);
    __syncthreads();
  }

  // Epilogue.  Lane holds rows m = 16*mi + 4*quarter + j of output column n_local.
#pragma unroll
  for (int mi = 0; mi < 4; ++mi) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = 16 * mi + 4 * quarter + j;
      if (m >= rows) continue;
      if (kGateUp) {
#pragma unroll
        for (int p = 0; p < NPW / 2; ++p) {
          const float gv_ = acc[2 * p][mi][j];
          const float uv = acc[2 * p + 1][mi][j];
          const float a = gv_ / (1.0f + expf(-gv_)) * uv;
          const int col = 16 * ((rb0 >> 1) + p) + n_local;
          act_out[(int64_t)(row0 + m) * f + col] = (uint16_t)f32_to_bf16_rne(a);
        }
      } else {
        const int pi = gv.sorted_pairs[row0 + m];
#pragma unroll
        for (int r = 0; r < NPW; ++r)
          pair_out[(int64_t)pi * d + 16 * (rb0 + r) + n_local] = acc[r][mi][j];
      }
    }
  }
}

inline int max_row_tiles(int pairs, int n_experts) {
  const int e = pairs < n_experts ? pairs : n_experts;
  return (pairs + kRows - 1) / kRows + e;
}

}  // namespace

hipError_t launch_gateup_mfma(int d, int f, int top_k, int pairs, int n_experts,
                              const uint16_t* h, const GroupView& gv, const WaveArg& wave,
                              const uint8_t* slot_bank, int64_t record_bytes, uint16_t* act,
                              hipStream_t stream) {
  if (pairs == 0) return hipSuccess;
  // Column tile: 4 wavefronts x 2 (gate, up) pairs x 16 outputs = 128 act columns.
  dim3 grid(f / 128, max_row_tiles(pairs, n_experts));
  launch(grouped_mfma_kernel<true>, grid, dim3(64 * kWaves), stream, d, f, top_k,
                     n_experts, h, gv, wave, slot_bank, record_bytes, act, (float*)nullptr);
  return hipGetLastError();
}

hipError_t launch_down_mfma(int d, int f, int top_k, int pairs, int n_experts,
                            const uint16_t* act, const GroupView& gv, const WaveArg& wave,
                            const uint8_t* slot_bank, int64_t record_bytes, float* pair_out,
                            hipStream_t stream) {
  if (pairs == 0) return hipSuccess;
  // Column tile: 4 wavefronts x 2 row blocks x 16 outputs = 128 output columns.
  dim3 grid(d / 128, max_row_tiles(pairs, n_experts));
  launch(grouped_mfma_kernel<false>, grid, dim3(64 * kWaves), stream, d, f, top_k,
                     n_experts, act, gv, wave, slot_bank, record_bytes, (uint16_t*)nullptr,
                     pair_out);
  return hipGetLastError();
}

}  // namespace emoe
