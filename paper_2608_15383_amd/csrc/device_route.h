// Device routines of routing and grouping (Sec. 3.1 Eq. 1, Fig. 1, Sec. 3.4),
// shared by the stand-alone kernels (route.hip) and the fused decode kernel
// (decode.hip) so both compute bit-identical results.  kCo selects
// device-coherent global accesses (fused launch) or ordinary ones.
#pragma once

#include "common.h"

namespace emoe {

constexpr int kPerLane = EMOE_MAX_EXPERTS / 64;  // experts held per lane in top-k / scans

__device__ __forceinline__ void bf16x8_to_f64(const uint4 v, double* out) {
  const uint32_t dw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    out[2 * p] = (double)bf16_to_f32(dw[p] & 0xffffu);
    out[2 * p + 1] = (double)bf16_to_f32(dw[p] >> 16);
  }
}

// Sum of a double over the wavefront (butterfly of lane exchanges), returned in
// every lane.
__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// Sum of a double over the wavefront with DPP lane moves (quad swaps, the
// half-row and row mirrors, then the two row broadcasts), no LDS round trip;
// the total is read from lane 63 and returned in every lane.  Lanes that a
// move does not reach add 0.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ double dpp_add_f64(double v) {
  const int lo = __double2loint(v), hi = __double2hiint(v);
  const int lo2 = __builtin_amdgcn_update_dpp(0, lo, kCtrl, kRowMask, 0xF, false);
  const int hi2 = __builtin_amdgcn_update_dpp(0, hi, kCtrl, kRowMask, 0xF, false);
  return v + __hiloint2double(hi2, lo2);
}

__device__ __forceinline__ double wave_sum_f64_dpp(double v) {
  v = dpp_add_f64<0xB1, 0xF>(v);   // quad_perm [1, 0, 3, 2]
  v = dpp_add_f64<0x4E, 0xF>(v);   // quad_perm [2, 3, 0, 1]
  v = dpp_add_f64<0x141, 0xF>(v);  // row_half_mirror
  v = dpp_add_f64<0x140, 0xF>(v);  // row_mirror
  v = dpp_add_f64<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
  v = dpp_add_f64<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
  const int lo = __builtin_amdgcn_readlane(__double2loint(v), 63);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(v), 63);
  return __hiloint2double(hi, lo);
}

// Logit sums of expert e for kT consecutive tokens by one wavefront over the
// inputs [k0, k0 + kn) (kn a multiple of 8), with every load of a pass issued
// before any is used: lanes take 8-input chunks k = 8*lane + 512*i, kC chunks
// per pass and token, so the kT tokens with kn <= 512 kC cost one memory
// round trip together.  Chunks past kn are read at a clamped in-bounds address
// and contribute 0.  Products of bf16 values are exact in fp64 and so, at
// these magnitudes, is the sum, whatever its order.  store(t, sum) receives
// each token's sum (the same in every lane).
template <int kT, int kC = 4, typename Store>
__device__ __forceinline__ void wave_router_dot_tokens(int t0, int d, int k0, int kn,
                                                       const uint16_t* __restrict__ wrow,
                                                       const uint16_t* __restrict__ h, Store store) {
  const int lane = lane_id();
  double acc[kT];
#pragma unroll
  for (int t = 0; t < kT; ++t) acc[t] = 0.0;
  for (int base = 0; base < kn; base += 512 * kC) {
    uint4 w[kC], x[kT][kC];
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      const int k = base + 512 * i + 8 * lane;
      const int kc = k0 + (k < kn ? k : kn - 8);
      w[i] = *reinterpret_cast<const uint4*>(wrow + kc);
#pragma unroll
      for (int t = 0; t < kT; ++t)
        x[t][i] = *reinterpret_cast<const uint4*>(h + (int64_t)(t0 + t) * d + kc);
    }
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      const bool ok = base + 512 * i + 8 * lane < kn;
      double wv[8];
      bf16x8_to_f64(w[i], wv);
#pragma unroll
      for (int r = 0; r < 8; ++r) wv[r] = ok ? wv[r] : 0.0;
#pragma unroll
      for (int t = 0; t < kT; ++t) {
        double hv[8];
        bf16x8_to_f64(x[t][i], hv);
#pragma unroll
        for (int r = 0; r < 8; ++r) acc[t] = fma(hv[r], wv[r], acc[t]);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < kT; ++t) store(t0 + t, wave_sum_f64_dpp(acc[t]));
}

// Logit sums of expert e for tokens [t0, t1) over all d inputs: two tokens
// per pass (four would hold more loaded registers than the fused decode
// kernel has to spare).
template <typename Store>
__device__ __forceinline__ void wave_router_dot(int t0, int t1, int d, int e,
                                                const uint16_t* __restrict__ h,
                                                const uint16_t* __restrict__ wr, Store store) {
  const uint16_t* wrow = wr + (int64_t)e * d;
  for (; t0 + 2 <= t1; t0 += 2) wave_router_dot_tokens<2>(t0, d, 0, d, wrow, h, store);
  if (t0 < t1) wave_router_dot_tokens<1>(t0, d, 0, d, wrow, h, store);
}

// The same over the inputs [k0, k0 + kn) only, one 512-input chunk per lane
// and pass (a quarter of d <= 2048 in one pass).
template <typename Store>
__device__ __forceinline__ void wave_router_dot_part(int t0, int t1, int d, int k0, int kn, int e,
                                                     const uint16_t* __restrict__ h,
                                                     const uint16_t* __restrict__ wr, Store store) {
  const uint16_t* wrow = wr + (int64_t)e * d;
  for (; t0 + 2 <= t1; t0 += 2) wave_router_dot_tokens<2, 1>(t0, d, k0, kn, wrow, h, store);
  if (t0 < t1) wave_router_dot_tokens<1, 1>(t0, d, k0, kn, wrow, h, store);
}

// Wavefront-wide max / min of a 32-bit unsigned value with DPP lane moves
// (xor 1, xor 2, half-row mirror, row mirror, then the row broadcasts), the
// result read from lane 63 so every lane gets it.
template <bool kMax>
__device__ __forceinline__ uint32_t dpp_combine(uint32_t a, uint32_t b) {
  return kMax ? (a > b ? a : b) : (a < b ? a : b);
}

template <bool kMax>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v) {
  const int x = (int)v;
  v = dpp_combine<kMax>(v, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));
  int y = (int)v;
  v = dpp_combine<kMax>(v, (uint32_t)__builtin_amdgcn_update_dpp(y, y, 0x4E, 0xF, 0xF, false));
  y = (int)v;
  v = dpp_combine<kMax>(v, (uint32_t)__builtin_amdgcn_update_dpp(y, y, 0x141, 0xF, 0xF, false));
  y = (int)v;
  v = dpp_combine<kMax>(v, (uint32_t)__builtin_amdgcn_update_dpp(y, y, 0x140, 0xF, 0xF, false));
  y = (int)v;
  v = dpp_combine<kMax>(v, (uint32_t)__builtin_amdgcn_update_dpp(y, y, 0x142, 0xA, 0xF, false));
  y = (int)v;
  v = dpp_combine<kMax>(v, (uint32_t)__builtin_amdgcn_update_dpp(y, y, 0x143, 0xC, 0xF, false));
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Top-k of one token's logits z[E] by one wavefront, and its mixture weights
// (softmax over the selected logits when renormalize, else over all E), fp64.
// Order: larger logit first (order key: a monotone integer image of the fp32
// value, -0 folded onto +0) and, among equal logits, the lower expert id.  Up
// to 64 experts use a ballot radix select; more experts take k rounds of a
// wavefront max.  kCo: device-coherent loads of z; kCoStore: device-coherent
// result stores.
// wave_topk_select leaves the selection in registers (TopkState);
// wave_topk_store_ids and wave_topk_weights write it out.
struct TopkState {
  float v[kPerLane];       // this lane's logits
  int sel_id[kPerLane];    // rank j lives in lane j % 64, register j / 64
  float sel_z[kPerLane];
  float zmax;
};

// At most 64 experts, one per lane: the lane's 64-bit rank key, the order key
// of its logit above 63 - lane, so the key is unique and a larger logit, then
// the lower expert id, compares greater.  Lanes past n_experts get order key
// 0, below every expert.
__device__ __forceinline__ uint64_t topk_lane_key(const TopkState& st, int n_experts) {
  const int lane = lane_id();
  const uint32_t u = __float_as_uint(st.v[0] + 0.0f);  // -0 -> +0
  const uint32_t key = lane < n_experts ? ((u & 0x80000000u) ? ~u : (u | 0x80000000u)) : 0u;
  return ((uint64_t)key << 32) | (uint32_t)(63 - lane);
}

// Number of keys[0 .. kN) (kN even) greater than mine: broadcast reads of the
// published keys.
template <int kN>
__device__ __forceinline__ int topk_count_greater(const uint64_t* keys, uint64_t mine) {
  int rank = 0;
#pragma unroll
  for (int j = 0; j < kN; j += 2) {
    const uint64_t k0 = keys[j], k1 = keys[j + 1];
    rank += (k0 > mine) + (k1 > mine);
  }
  return rank;
}

// At most 64 experts, one per lane, each lane knowing its rank among the keys
// (0 = largest): the selected lanes (rank < k) drop (logit, expert) into slot
// rank of the wavefront's 64 words of LDS scratch, which lane j reads.
__device__ __forceinline__ void topk_select_ranked(int rank, int top_k, TopkState& st,
                                                   uint64_t* scratch) {
  const int lane = lane_id();
  __builtin_amdgcn_wave_barrier();
  if (rank < top_k) scratch[rank] = ((uint64_t)__float_as_uint(st.v[0]) << 32) | (uint32_t)lane;
  __builtin_amdgcn_wave_barrier();
  if (lane < top_k) {
    const uint64_t w = scratch[lane];
    st.sel_id[0] = (int)(uint32_t)w;
    st.sel_z[0] = __uint_as_float((uint32_t)(w >> 32));
  }
  st.zmax = __uint_as_float((uint32_t)(scratch[0] >> 32));
  __builtin_amdgcn_wave_barrier();
}

// Selection from the logits already in st.v (lane l holds expert l + 64c in
// register c).  scratch: 64 words of LDS private to the wavefront, or null.
__device__ __forceinline__ void wave_topk_select_loaded(int n_experts, int top_k, TopkState& st,
                                                        uint64_t* scratch = nullptr) {
  const int lane = lane_id();
  const int nc = (n_experts + 63) / 64;  // logits per lane in use
  float* v = st.v;
  int* sel_id = st.sel_id;
  float* sel_z = st.sel_z;
  if (nc == 1 && scratch) {
    // At most 64 experts with LDS: every lane publishes its unique key, reads
    // all 64 back and counts the larger ones, which is its rank.
    const uint64_t mine = topk_lane_key(st, n_experts);
    scratch[lane] = mine;
    __builtin_amdgcn_wave_barrier();
    const int rank = topk_count_greater<64>(scratch, mine);
    topk_select_ranked(rank, top_k, st, scratch);
    return;
  }
  uint32_t key[kPerLane];  // 0 = not a candidate (keys of non-NaN floats are > 0)
#pragma unroll
  for (int c = 0; c < kPerLane; ++c) {
    const int e = lane + 64 * c;
    const uint32_t u = __float_as_uint(v[c] + 0.0f);  // -0 -> +0
    key[c] = e < n_experts ? ((u & 0x80000000u) ? ~u : (u | 0x80000000u)) : 0u;
  }
  float zmax = 0.f;
  if (nc == 1) {
    // At most 64 experts, one per lane.  Radix select of the k-th largest key
    // from the top bit down with ballots (lanes still tied on the bits seen
    // so far in `cand`, lanes certainly selected in `sel`), the lowest lanes
    // (expert ids) first among equal keys; then each selected lane's rank is
    // the number of selected lanes ahead of it.
    uint64_t cand = __ballot(lane < n_experts);
    uint64_t sel = 0;
    int need = top_k;
    // The 32 bit-plane ballots do not depend on each other; unrolled, they
    // issue back to back and only the scalar mask updates form a chain.
    uint64_t plane[32];
#pragma unroll
    for (int b = 0; b < 32; ++b) plane[b] = __ballot((key[0] >> b) & 1u);
#pragma unroll
    for (int b = 31; b >= 0; --b) {
      const uint64_t ones = plane[b] & cand;
      const int n1 = __popcll(ones);
      if (n1 >= need) {
        cand = ones;
      } else {
        sel |= ones;
        need -= n1;
        cand &= ~ones;
      }
    }
    for (; need > 0; --need) {
      sel |= cand & (~cand + 1ull);  // lowest remaining tied lane
      cand &= cand - 1ull;
    }
    for (uint64_t m = sel; m != 0; m &= m - 1ull) {
      const int s = (int)__builtin_ctzll(m);
      const uint32_t ks = (uint32_t)__builtin_amdgcn_readlane((int)key[0], s);
      const float zs = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(v[0]), s));
      const uint64_t ahead = (__ballot(key[0] > ks) & sel) | (__ballot(key[0] == ks) & sel & ((1ull << s) - 1ull));
      const int r = __popcll(ahead);
      if (lane == r) {
        sel_id[0] = s;
        sel_z[0] = zs;
      }
      if (r == 0) zmax = zs;
    }
    st.zmax = zmax;
    return;
  }
  for (int j = 0; j < top_k; ++j) {
    uint32_t best = 0;
#pragma unroll
    for (int c = 0; c < kPerLane; ++c)
      if (c < nc) best = key[c] > best ? key[c] : best;
    const uint32_t m = wave_reduce_u32<true>(best);
    uint32_t idx = 0xffffffffu;
#pragma unroll
    for (int c = kPerLane - 1; c >= 0; --c)
      if (c < nc && key[c] == m) idx = (uint32_t)(lane + 64 * c);
    const int e = (int)wave_reduce_u32<false>(idx);
    const int ce = e >> 6;
    float vw = v[0];
#pragma unroll
    for (int c = 1; c < kPerLane; ++c)
      if (ce == c) vw = v[c];
    const float zw = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(vw), e & 63));
#pragma unroll
    for (int c = 0; c < kPerLane; ++c)
      if (lane + 64 * c == e) key[c] = 0u;
    if (j == 0) zmax = zw;
#pragma unroll
    for (int c = 0; c < kPerLane; ++c) {
      if (j == lane + 64 * c) {
        sel_id[c] = e;
        sel_z[c] = zw;
      }
    }
  }
  st.zmax = zmax;
}

template <bool kCo>
__device__ __forceinline__ void wave_topk_select(const float* __restrict__ z, int n_experts,
                                                 int top_k, TopkState& st,
                                                 uint64_t* scratch = nullptr) {
  const int lane = lane_id();
#pragma unroll
  for (int c = 0; c < kPerLane; ++c) {
    const int e = lane + 64 * c;
    st.v[c] = e < n_experts ? ld_f32<kCo>(z + e) : 0.f;
  }
  wave_topk_select_loaded(n_experts, top_k, st, scratch);
}

template <bool kCoStore>
__device__ __forceinline__ void wave_topk_store_ids(const TopkState& st, int top_k,
                                                    int32_t* __restrict__ ids_out) {
  const int lane = lane_id();
#pragma unroll
  for (int c = 0; c < kPerLane; ++c)
    if (lane + 64 * c < top_k) st_u32<kCoStore>(ids_out + lane + 64 * c, (uint32_t)st.sel_id[c]);
}

template <bool kCoStore>
__device__ __forceinline__ void wave_topk_weights(const TopkState& st, int n_experts, int top_k,
                                                  int renormalize, float* __restrict__ w_out) {
  const int lane = lane_id();
  const float* v = st.v;
  const float* sel_z = st.sel_z;
  const float zmax = st.zmax;
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
    if (j < top_k)
      st_u32<kCoStore>(w_out + j,
                       __float_as_uint((float)(exp((double)sel_z[c] - (double)zmax) / denom)));
  }
}

template <bool kCo, bool kCoStore = kCo>
__device__ __forceinline__ void wave_topk(const float* __restrict__ z, int n_experts, int top_k,
                                          int renormalize, int32_t* __restrict__ ids_out,
                                          float* __restrict__ w_out, uint64_t* scratch = nullptr) {
  TopkState st;
  wave_topk_select<kCo>(z, n_experts, top_k, st, scratch);
  wave_topk_store_ids<kCoStore>(st, top_k, ids_out);
  wave_topk_weights<kCoStore>(st, n_experts, top_k, renormalize, w_out);
}

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

// LDS of the block-wide grouping: per wavefront and expert, first the
// wavefront's count, then its first grouped position.
template <int kThreads>
struct GroupShared {
  int wbase[kThreads / 64][EMOE_MAX_EXPERTS];
};

// Lanes of the wavefront whose expert equals this lane's (valid lanes only),
// found with one ballot per bit of the expert id.
__device__ __forceinline__ uint64_t match_expert(bool valid, int e, int bits) {
  uint64_t m = __ballot(valid);
  for (int b = 0; b < bits; ++b) {
    const bool set = (e >> b) & 1;
    const uint64_t x = __ballot(valid && set);
    m &= set ? x : ~x;
  }
  return m;
}

// Grouping of the P pairs by expert, by one workgroup of kThreads threads:
// counts, exclusive offsets, a stable counting sort of the pair ids (pairs of
// one expert keep ascending id), the ascending active list, n_active and,
// when the pointers are non-null, the MFMA row-tile prefix sum and the
// inverse permutation pair_pos[pi] = grouped position.
// Each wavefront owns a contiguous range of 64-pair chunks: pass 1 counts its
// pairs per expert, a scan turns the counts into each wavefront's first
// position per expert, and pass 2 places its pairs in order.
template <int kThreads, bool kCo>
__device__ __forceinline__ void block_group(
    GroupShared<kThreads>& sh, int pairs, int n_experts, const int32_t* __restrict__ ids,
    int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ sorted_pairs, int32_t* __restrict__ active,
    int32_t* __restrict__ n_active, int32_t* __restrict__ tile_offsets,
    int32_t* __restrict__ pair_pos, int mfma_rows) {
  constexpr int kWaves = kThreads / 64;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  int bits = 0;
  while ((1 << bits) < n_experts) ++bits;
  const int n_chunks = (pairs + 63) / 64;
  const int per_wave = (n_chunks + kWaves - 1) / kWaves;
  const int c0 = min(n_chunks, wave * per_wave);
  const int c1 = min(n_chunks, c0 + per_wave);
  int* wb = sh.wbase[wave];
  for (int e = lane; e < n_experts; e += 64) wb[e] = 0;

  // The expert ids of kBatch chunks are loaded together, so one memory
  // latency covers kBatch chunks.
  constexpr int kBatch = 8;
  auto load_batch = [&](int cb, int (&eb)[kBatch]) {
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = 64 * (cb + j) + lane;
      eb[j] = (cb + j < c1 && i < pairs) ? ld_i32<kCo>(ids + i) : 0;
    }
  };

  // Pass 1: this wavefront's count per expert.
  for (int cb = c0; cb < c1; cb += kBatch) {
    int eb[kBatch];
    load_batch(cb, eb);
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (cb + j >= c1) break;
      const int i = 64 * (cb + j) + lane;
      const bool valid = i < pairs;
      const int e = eb[j];
      const uint64_t m = match_expert(valid, e, bits);
      const int rank = __popcll(m & ((1ull << lane) - 1ull));
      if (valid && rank == 0) wb[e] += __popcll(m);
    }
  }
  __syncthreads();

  // Totals, offsets, active list, row tiles; then each wavefront's base.
  if (wave == 0) {
    int c[kPerLane], local = 0, nz = 0, tl = 0;
#pragma unroll
    for (int q = 0; q < kPerLane; ++q) {
      const int e = kPerLane * lane + q;
      c[q] = 0;
      if (e < n_experts)
        for (int w = 0; w < kWaves; ++w) c[q] += sh.wbase[w][e];
      local += c[q];
      nz += c[q] > 0;
      tl += mfma_row_tiles(c[q], mfma_rows);
    }
    int total, nz_total, tl_total;
    int base = wave_exclusive_scan(local, total);
    int nz_base = wave_exclusive_scan(nz, nz_total);
    int tl_base = wave_exclusive_scan(tl, tl_total);
#pragma unroll
    for (int q = 0; q < kPerLane; ++q) {
      const int e = kPerLane * lane + q;
      if (e < n_experts) {
        st_u32<kCo>(counts + e, (uint32_t)c[q]);
        st_u32<kCo>(offsets + e, (uint32_t)base);
        if (tile_offsets) st_u32<kCo>(tile_offsets + e, (uint32_t)tl_base);
        if (c[q] > 0) st_u32<kCo>(active + nz_base++, (uint32_t)e);
        int run = base;
        for (int w = 0; w < kWaves; ++w) {
          const int n = sh.wbase[w][e];
          sh.wbase[w][e] = run;
          run += n;
        }
      }
      base += c[q];
      tl_base += mfma_row_tiles(c[q], mfma_rows);
    }
    if (lane == 0) {
      st_u32<kCo>(offsets + n_experts, (uint32_t)total);
      if (tile_offsets) st_u32<kCo>(tile_offsets + n_experts, (uint32_t)tl_total);
      st_u32<kCo>(n_active, (uint32_t)nz_total);
    }
  }
  __syncthreads();

  // Pass 2: stable placement.  Every lane reads its expert's base before the
  // group leader advances it (one wavefront's LDS accesses run in order).
  for (int cb = c0; cb < c1; cb += kBatch) {
    int eb[kBatch];
    load_batch(cb, eb);
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (cb + j >= c1) break;
      const int i = 64 * (cb + j) + lane;
      const bool valid = i < pairs;
      const int e = eb[j];
      const uint64_t m = match_expert(valid, e, bits);
      const int rank = __popcll(m & ((1ull << lane) - 1ull));
      if (valid) {
        const int pos = wb[e] + rank;
        st_u32<kCo>(sorted_pairs + pos, (uint32_t)i);
        if (pair_pos) st_u32<kCo>(pair_pos + i, (uint32_t)pos);
      }
      if (valid && rank == 0) wb[e] += __popcll(m);
    }
  }
}

}  // namespace emoe
