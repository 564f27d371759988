// Device routines of the weight-streaming (few tokens per expert) projections,
// shared by the grouped GEMV kernels (gemv.hip) and the fused decode kernel
// (decode.hip), so both produce bit-identical results.  kCo selects
// device-coherent accesses for data exchanged between workgroups.
//
// In-register dequantization: for a code dword, ((dw >> 4p) & 0x000f000f) |
// 0x43004300 is the bf16 pair (128 + u_2p, 128 + u_2p+1), exact because bf16
// represents the integers 128..143.  With u = q + 8 the dot product over a
// lane's 32 inputs is sum (u - 8) x = sum (128 + u) x - 136 sum x, so each
// group needs one correction with the activations' sum before the FP16 group
// scale is applied in fp32 (Sec. 3.2: W_hat = s q is never rounded).
#pragma once

#include "common.h"

namespace emoe {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

constexpr int kGemvWaves = 4;      // wavefronts per workgroup
constexpr int kTokChunk = 4;       // token rows per pass over the weights
constexpr int kGateBatch = 4;      // tiles per matrix one wavefront loads together (gate/up)
constexpr int kDownBatch = 8;      // tiles one wavefront loads together (down)
constexpr uint32_t kOnesBf16x2 = 0x3f803f80u;  // bf16 pair (1, 1)

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                        __builtin_bit_cast(bf16x2_t, b), c, false);
}

// A loaded value made opaque here: the compiler cannot consume it (and so
// wait for its load) any earlier, which keeps a prefetched batch's loads in
// flight until the batch is used.
__device__ __forceinline__ uint32_t at_use(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}

// Mask and magic are hidden from constant folding (the empty asm statements
// emit nothing; identical ones are merged), mask in an SGPR and magic in a
// VGPR, so each pair is one v_and_or_b32 (gfx9 VOP3 takes no literal).
__device__ __forceinline__ void dequant_dword(uint32_t dw, uint32_t* out) {
  uint32_t mask = 0x000f000fu, magic = 0x43004300u;
  asm("" : "+s"(mask));
  asm("" : "+v"(magic));
#pragma unroll
  for (int p = 0; p < 4; ++p) out[p] = ((dw >> (4 * p)) & mask) | magic;
}

// Dot product of one lane's 32 codes of a group (its row, its inputs) with the
// 32 matching activations x (4 x uint4): returns sum (128 + u) x and, when
// want_xs, adds sum x to xs.  Four independent accumulators (one per code
// dword) and two for sum x keep the dependent chains short; the partial sums
// are added in a fixed order, so every caller gets the same bits.
__device__ __forceinline__ float lane_group_dot(const uint4 codes, const uint4* x, float& xs,
                                                bool want_xs) {
  const uint32_t c[4] = {codes.x, codes.y, codes.z, codes.w};
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  float xsum[2] = {0.f, 0.f};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t wp[4];
    dequant_dword(c[i], wp);
    const uint32_t xv[4] = {x[i].x, x[i].y, x[i].z, x[i].w};
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      acc[i] = dot2(wp[p], xv[p], acc[i]);
      if (want_xs) xsum[i & 1] = dot2(kOnesBf16x2, xv[p], xsum[i & 1]);
    }
  }
  if (want_xs) xs += xsum[0] + xsum[1];
  return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

__device__ __forceinline__ void load_x32(const uint16_t* row, uint4* x) {
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = *reinterpret_cast<const uint4*>(row + 32 * i);
}

__device__ __forceinline__ float silu_mul(float g, float u) {
  return g / (1.0f + expf(-g)) * u;
}

struct GateUpShared {
  float red[kGemvWaves][kTokChunk][2][16];
};

// One workgroup of kGemvWaves wavefronts computes the SwiGLU activation
// phi(W_g h) * (W_u h) of gate/up row-block pair b (outputs 16b .. 16b+15) for
// the rows s in [begin, end) of one expert whose packed record is `rec`;
// x_row(s) points at the d activations of row s (global memory or LDS), and
// store(s, n, v) receives outputs n, n+1 of row s (n even) as a bf16 pair in
// v (low half: output n).  The wavefronts split the input groups round-robin
// and meet in LDS in wavefront order.  Each row's result depends only on that
// row, not on which rows share the pass.
template <typename XRow, typename Store>
__device__ __forceinline__ void gateup_rows(GateUpShared& sh, int d, int f, XRow x_row, int begin,
                                            int end, const uint8_t* __restrict__ rec, int b,
                                            Store store);

// Tiles of one wavefront for gate/up row-block pair b: the gate and up tiles
// of its input groups g = wi + 4j (j < kGateBatch) and their scale words.
struct GateUpBatch {
  uint4 cg[kGateBatch], cu[kGateBatch];
  uint32_t sgu[kGateBatch];
};

// Every load is issued (slots past the last group read the last group again,
// unused), so a caller's wait counts do not depend on the shape.
__device__ __forceinline__ void gateup_load_batch(const uint8_t* __restrict__ rec, int d, int f,
                                                  int b, GateUpBatch& bt) {
  const int lane = lane_id();
  const int wi = threadIdx.x >> 6;
  const int G = d / kGroup;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* gate_codes = rec + L.w13_codes + (int64_t)(2 * b) * G * kTileBytes + 16 * lane;
  const uint8_t* up_codes = gate_codes + (int64_t)G * kTileBytes;
  const uint32_t* scales = reinterpret_cast<const uint32_t*>(rec + L.w13_scales);
  const int gate_n = 32 * b + (lane & 15);
#pragma unroll
  for (int j = 0; j < kGateBatch; ++j) {
    const int g = min(wi + kGemvWaves * j, G - 1);
    bt.cg[j] = *reinterpret_cast<const uint4*>(gate_codes + (int64_t)g * kTileBytes);
    bt.cu[j] = *reinterpret_cast<const uint4*>(up_codes + (int64_t)g * kTileBytes);
    bt.sgu[j] = scales[scale_index(gate_n, g, G) >> 1];
  }
}

// Gate/up row-block pair b for one activation row x (row `row`) from its
// loaded tiles (d <= kGemvWaves * kGateBatch * 128): the same arithmetic, in
// the same order, as gateup_rows, so the same bits.  Touches no global memory
// before the store.  kFull: d is exactly kGemvWaves * kGateBatch * 128, so
// every slot of the batch is a group and the code has no branch on the
// group count (a branch would let the compiler sink a tile's load into it,
// behind any loads the caller issued after the batch's, and wait for those).
// kXs: 0 forms each group's activation sum inline, 1 also keeps it in xsv[j],
// 2 takes it from xsv[j] (the same value: the row and the groups are the same
// for every pair of an item).
template <bool kFull = false, int kXs = 0, typename Store>
__device__ __forceinline__ void gateup_pair_compute(GateUpShared& sh, int d, const uint16_t* x,
                                                    int row, const GateUpBatch& cur, int b,
                                                    Store store, float* xsv = nullptr) {
  const int lane = lane_id();
  const int wi = threadIdx.x >> 6;
  const int G = kFull ? kGemvWaves * kGateBatch : d / kGroup;
  const int n_local = lane & 15;
  const int quarter = lane >> 4;
  const uint16_t* xrow = x + 8 * quarter;
  float accg = 0.f, accu = 0.f;
  uint4 xc[4];
  load_x32(xrow + wi * kGroup, xc);
#pragma unroll
  for (int j = 0; j < kGateBatch; ++j) {
    const int g = wi + kGemvWaves * j;
    if (!kFull && g >= G) break;
    const bool more = j + 1 < kGateBatch && (kFull || g + kGemvWaves < G);
    uint4 xn[4];
    if (more) load_x32(xrow + (g + kGemvWaves) * kGroup, xn);
    float xs = kXs == 2 ? xsv[j] : 0.f;
    const float pg = lane_group_dot(cur.cg[j], xc, xs, kXs != 2);
    const float pu = lane_group_dot(cur.cu[j], xc, xs, false);
    if (kXs == 1) xsv[j] = xs;
    accg = fmaf(half_bits_to_f32(cur.sgu[j] & 0xffffu), fmaf(-136.f, xs, pg), accg);
    accu = fmaf(half_bits_to_f32(cur.sgu[j] >> 16), fmaf(-136.f, xs, pu), accu);
    if (more) {
#pragma unroll
      for (int i = 0; i < 4; ++i) xc[i] = xn[i];
    }
  }
  accg += __shfl_xor(accg, 16);
  accg += __shfl_xor(accg, 32);
  accu += __shfl_xor(accu, 16);
  accu += __shfl_xor(accu, 32);
  if (quarter == 0) {
    sh.red[wi][0][0][n_local] = accg;
    sh.red[wi][0][1][n_local] = accu;
  }
  __syncthreads();
  if (wi == 0) {
    float gs = 0.f, us = 0.f;
#pragma unroll
    for (int w = 0; w < kGemvWaves; ++w) {
      gs += sh.red[w][0][0][n_local];
      us += sh.red[w][0][1][n_local];
    }
    const uint32_t a16 = f32_to_bf16_rne(silu_mul(gs, us));
    const uint32_t next = __shfl_down(a16, 1);
    if (lane < 16 && (n_local & 1) == 0) store(row, 16 * b + n_local, a16 | (next << 16));
  }
  __syncthreads();
}

// gateup_pair_compute over the row-block pairs b0 .. b1-1 (b1 - b0 >= 2),
// with the next pair's tiles loaded while the current pair is computed; in
// place of a next pair, the last pair runs after `last_loads()`, the caller's
// loads for what follows (all of them issued unconditionally, so the wait
// for the last pair's tiles stays exact).
template <typename Store, typename LastLoads>
__device__ __forceinline__ void gateup_row_blocks(GateUpShared& sh, int d, int f,
                                                  const uint16_t* x, int row,
                                                  const uint8_t* __restrict__ rec, int b0, int b1,
                                                  Store store, LastLoads last_loads) {
  GateUpBatch cur;
  gateup_load_batch(rec, d, f, b0, cur);
  // The first pair forms the groups' activation sums, the others reuse them.
  float xsv[kGateBatch];
  {
    GateUpBatch nxt;
    gateup_load_batch(rec, d, f, b0 + 1, nxt);
    gateup_pair_compute<false, 1>(sh, d, x, row, cur, b0, store, xsv);
    cur = nxt;
  }
  for (int b = b0 + 1; b < b1 - 1; ++b) {
    GateUpBatch nxt;
    gateup_load_batch(rec, d, f, b + 1, nxt);
    gateup_pair_compute<false, 2>(sh, d, x, row, cur, b, store, xsv);
    cur = nxt;
  }
  last_loads();
  gateup_pair_compute<false, 2>(sh, d, x, row, cur, b1 - 1, store, xsv);
}

// The grouped rows [begin, end) of one expert; the token of grouped row s is
// sorted_pairs[s] / top_k.
template <bool kCo>
__device__ __forceinline__ void gateup_block(GateUpShared& sh, int d, int f, int top_k,
                                             const uint16_t* __restrict__ h,
                                             const int32_t* __restrict__ sorted_pairs, int begin,
                                             int end, const uint8_t* __restrict__ rec, int b,
                                             uint16_t* __restrict__ act) {
  gateup_rows(
      sh, d, f, [&](int s) { return h + (int64_t)(ld_i32<kCo>(sorted_pairs + s) / top_k) * d; },
      begin, end, rec, b,
      [&](int s, int n, uint32_t v) { st_u32<kCo>(act + (int64_t)s * f + n, v); });
}

template <typename XRow, typename Store>
__device__ __forceinline__ void gateup_rows(GateUpShared& sh, int d, int f, XRow x_row, int begin,
                                            int end, const uint8_t* __restrict__ rec, int b,
                                            Store store) {
  const int lane = lane_id();
  const int wi = threadIdx.x >> 6;
  const int G = d / kGroup;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* gate_codes = rec + L.w13_codes + (int64_t)(2 * b) * G * kTileBytes + 16 * lane;
  const uint8_t* up_codes = gate_codes + (int64_t)G * kTileBytes;
  const int n_local = lane & 15;
  const int quarter = lane >> 4;
  // The gate and up rows of a lane (blocks 2b and 2b+1) have adjacent scales:
  // one 32-bit word per group, gate in the low half.
  const uint32_t* scales = reinterpret_cast<const uint32_t*>(rec + L.w13_scales);
  const int gate_n = 32 * b + n_local;

  for (int m0 = begin; m0 < end; m0 += kTokChunk) {
    const int mc = min(kTokChunk, end - m0);
    const uint16_t* xrow[kTokChunk];
#pragma unroll
    for (int m = 0; m < kTokChunk; ++m) xrow[m] = x_row(m < mc ? m0 + m : m0) + 8 * quarter;
    float accg[kTokChunk], accu[kTokChunk];
#pragma unroll
    for (int m = 0; m < kTokChunk; ++m) accg[m] = accu[m] = 0.f;

    for (int g0 = wi; g0 < G; g0 += kGemvWaves * kGateBatch) {
      // The whole batch is loaded before any of it is used: scales stay raw
      // fp16 bits until the arithmetic, so no load waits for another.
      uint4 cg[kGateBatch], cu[kGateBatch];
      uint32_t sgu[kGateBatch];
#pragma unroll
      for (int j = 0; j < kGateBatch; ++j) {
        const int g = g0 + kGemvWaves * j;
        if (g < G) {
          cg[j] = *reinterpret_cast<const uint4*>(gate_codes + (int64_t)g * kTileBytes);
          cu[j] = *reinterpret_cast<const uint4*>(up_codes + (int64_t)g * kTileBytes);
          sgu[j] = scales[scale_index(gate_n, g, G) >> 1];
        }
      }
      // Row by row over the batch's groups (each row's sum still runs in
      // group order), the next group's activations read while this one's
      // are used, so their load latency is not paid group after group.
#pragma unroll
      for (int m = 0; m < kTokChunk; ++m) {
        if (m >= mc) break;
        uint4 xc[4];
        load_x32(xrow[m] + g0 * kGroup, xc);
#pragma unroll
        for (int j = 0; j < kGateBatch; ++j) {
          const int g = g0 + kGemvWaves * j;
          if (g >= G) break;
          const bool more = j + 1 < kGateBatch && g + kGemvWaves < G;
          uint4 xn[4];
          if (more) load_x32(xrow[m] + (g + kGemvWaves) * kGroup, xn);
          float xs = 0.f;
          const float pg = lane_group_dot(cg[j], xc, xs, true);
          const float pu = lane_group_dot(cu[j], xc, xs, false);
          accg[m] = fmaf(half_bits_to_f32(sgu[j] & 0xffffu), fmaf(-136.f, xs, pg), accg[m]);
          accu[m] = fmaf(half_bits_to_f32(sgu[j] >> 16), fmaf(-136.f, xs, pu), accu[m]);
          if (more) {
#pragma unroll
            for (int i = 0; i < 4; ++i) xc[i] = xn[i];
          }
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
        sh.red[wi][m][0][n_local] = accg[m];
        sh.red[wi][m][1][n_local] = accu[m];
      }
    }
    __syncthreads();
    if (wi == 0) {
      const int m = lane >> 4;  // lane = 16 m + n
      float g = 0.f, u = 0.f;
#pragma unroll
      for (int w = 0; w < kGemvWaves; ++w) {
        g += sh.red[w][m][0][n_local];
        u += sh.red[w][m][1][n_local];
      }
      const uint32_t a16 = f32_to_bf16_rne(silu_mul(g, u));
      const uint32_t next = __shfl_down(a16, 1);
      if (m < mc && (n_local & 1) == 0) store(m0 + m, 16 * b + n_local, a16 | (next << 16));
    }
    __syncthreads();
  }
}

// Down projection tiles of one wavefront: row-block rb, input groups
// g0 .. g0+kDownBatch-1 (those < G).
struct DownBatch {
  uint4 c[kDownBatch];
  uint16_t s[kDownBatch];  // raw fp16 scales: converted at use, so loads never wait on each other
};

__device__ __forceinline__ void down_load_batch(const uint8_t* __restrict__ rec, int d, int f,
                                                int rb, int g0, DownBatch& bt) {
  const int lane = lane_id();
  const int G = f / kGroup;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* codes = rec + L.w2_codes + (int64_t)rb * G * kTileBytes + 16 * lane;
  const uint16_t* sc = reinterpret_cast<const uint16_t*>(rec + L.w2_scales);
  const int n = 16 * rb + (lane & 15);
#pragma unroll
  for (int j = 0; j < kDownBatch; ++j) {
    if (g0 + j < G) {
      bt.c[j] = *reinterpret_cast<const uint4*>(codes + (int64_t)(g0 + j) * kTileBytes);
      bt.s[j] = sc[scale_index(n, g0 + j, G)];
    }
  }
}

// This lane's 32 activations of group g of row m (4 x uint4) through xload.
template <typename XLoad>
__device__ __forceinline__ void load_x_group(XLoad xload, int m, int g, uint4* x) {
  const int quarter = lane_id() >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = xload(m, g * kGroup + 8 * quarter + 32 * i);
}

// Sum a lane's partials over the four lanes of its row: afterwards lanes
// 0..15 hold the outputs of rows 16*rb + lane.
__device__ __forceinline__ float reduce_quarters(float v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}

// The down projection accumulates each output in four classes of input
// groups, class c holding the groups g with g % 4 == c in ascending order
// (so four wavefronts can split the groups of a row between them, as the
// fused decode launch does, with the same result).  The output is the sum of
// the classes in a fixed order, each first summed over the lanes of its row.
__device__ __forceinline__ float down_class_total(const float* acc) {
  return (reduce_quarters(acc[0]) + reduce_quarters(acc[1])) +
         (reduce_quarters(acc[2]) + reduce_quarters(acc[3]));
}

// acc[m][g % 4] += contribution of group g of the loaded batch to activation
// row m < mc; xload(m, k) returns the 8 bf16 activations k .. k+7 of row m.
// Row by row, groups in order; the next group's activations are read while
// this one's are used.
template <typename XLoad>
__device__ __forceinline__ void down_apply_batch(const DownBatch& bt, int f, int g0, XLoad xload,
                                                 int mc, float (*acc)[4]) {
  static_assert(kDownBatch % 4 == 0, "batches start at a group of class 0");
  const int G = f / kGroup;
  if (g0 >= G) return;
#pragma unroll
  for (int m = 0; m < kTokChunk; ++m) {
    if (m >= mc) break;
    uint4 xc[4];
    load_x_group(xload, m, g0, xc);
#pragma unroll
    for (int j = 0; j < kDownBatch; ++j) {
      const int g = g0 + j;
      if (g >= G) break;
      const bool more = j + 1 < kDownBatch && g + 1 < G;
      uint4 xn[4];
      if (more) load_x_group(xload, m, g + 1, xn);
      float xs = 0.f;
      const float p = lane_group_dot(bt.c[j], xc, xs, true);
      acc[m][j & 3] = fmaf(half_bits_to_f32(at_use(bt.s[j])), fmaf(-136.f, xs, p), acc[m][j & 3]);
      if (more) {
#pragma unroll
        for (int i = 0; i < 4; ++i) xc[i] = xn[i];
      }
    }
  }
}

// Sum of the 32 activations x (4 x uint4) of one lane's inputs of a group, in
// the order lane_group_dot accumulates it.
__device__ __forceinline__ float lane_group_xsum(const uint4* x) {
  float xsum[2] = {0.f, 0.f};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t xv[4] = {x[i].x, x[i].y, x[i].z, x[i].w};
#pragma unroll
    for (int p = 0; p < 4; ++p) xsum[i & 1] = dot2(kOnesBf16x2, xv[p], xsum[i & 1]);
  }
  return 0.f + (xsum[0] + xsum[1]);
}

}  // namespace emoe
