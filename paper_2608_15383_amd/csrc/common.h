// Internal definitions shared by the gfx950 kernels and the host runtime of
// libexactmoe.so: the packed record layout, the wave descriptor passed to the
// grouped kernels, small device helpers and the kernel launchers.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "exactmoe.h"

namespace emoe {

constexpr int kGroup = EMOE_GROUP;  // quantization group along K (Sec. 3.2)
constexpr int kTileRows = 16;       // output rows per packed tile
constexpr int kTileBytes = 1024;    // codes of one 16 x 128 tile (4 bits each)
constexpr int kMaxWave = EMOE_MAX_EXPERTS;
constexpr int kGemvRows = 8;  // activation rows of one expert per GEMV workgroup
constexpr int kMfmaRows = 64;       // token rows per MFMA row-tile
constexpr int kMfmaMaxGroups = 64;  // K / 128 of an MFMA projection (d, d_ff <= 8192)

// ---------------------------------------------------------------------------
// Packed expert record (our CDNA4 layout; the paper packs its own GPU's format
// offline once, Sec. 3.2, and keeps the identical bytes in host and GPU
// memory, Sec. 3.3).
//
//   [W13 codes][W13 scales][W2 codes][W2 scales]
//
// W13 holds gate and up (each d_ff x d_model) as 2*d_ff rows interleaved per
// 16-row block: row-block 2b is gate rows 16b..16b+15, row-block 2b+1 is up
// rows 16b..16b+15, so one workgroup sees matching gate and up outputs.
// W2 is down (d_model x d_ff).
//
// Codes of a matrix with N rows and K inputs: (N/16) x (K/128) tiles of
// 1024 B, tile (rb, g) at byte (rb*(K/128) + g)*1024.  Inside a tile, lane l
// of a wavefront owns the 16 bytes at 16*l: output row n = 16*rb + l%16 and
// the four dwords i = 0..3 hold inputs k = 128*g + 32*i + 8*(l/16) + r,
// r = 0..7, with r even in bits 4*(r/2)..+3 and r odd in bits 16+4*(r/2)..+3.
// A 4-bit code is u = q + 8 (offset binary).  One wavefront load of a tile is
// therefore fully coalesced, each dword expands to four bf16 pairs (k, k+1)
// that line up with bf16 activations in memory, and the four dwords are the
// B operands of four v_mfma_f32_16x16x32_bf16 steps.
// Scales: fp16, after the codes, N*(K/128) of them in 128-byte lines: the 64
// scales of rows 64c .. 64c+63 and group g fill line c*(K/128) + g, ordered by
// (n%16, (n/16)%4), so the four row blocks a wavefront owns give each lane
// its four scales as one 8-byte load (scale_index).  N is a multiple of 64
// (d_model and d_ff are multiples of 128).
// ---------------------------------------------------------------------------
struct RecordLayout {
  int64_t w13_codes, w13_scales, w2_codes, w2_scales, bytes;
};

// Position (in fp16 units) of the scale of stored row n and group g of a
// matrix with G groups per row.
__host__ __device__ inline int64_t scale_index(int n, int g, int G) {
  return ((int64_t)(n >> 6) * G + g) * 64 + (n & 15) * 4 + ((n >> 4) & 3);
}

__host__ __device__ inline RecordLayout record_layout(int d, int f) {
  RecordLayout r;
  const int64_t fd = (int64_t)f * d;
  r.w13_codes = 0;
  r.w13_scales = fd;                   // 2f*d codes at 4 bits
  r.w2_codes = fd + fd / 32;           // + 2f * (d/128) fp16 scales
  r.w2_scales = r.w2_codes + fd / 2;   // + d*f codes at 4 bits
  r.bytes = r.w2_scales + fd / 64;     // + d * (f/128) fp16 scales
  return r;
}

// Experts of one wave (Sec. 3.4 step 2).  n < 0: every active expert of the
// call, resident in the slot of the same index (full residency, Sec. 3.3);
// the kernels then read the device-side active list.  n >= 0: the wave's
// experts expert[0..n) and the global-to-slot map slot_of[E], -1 being the
// inactive sentinel for every expert outside the wave.
struct WaveArg {
  int32_t n;
  int16_t expert[kMaxWave];
  int16_t slot_of[kMaxWave];
  // GEMV row chunks (kGemvRows rows of one expert each): chunk0[i] = chunks
  // of wave positions before i, chunk0[n] = all (n >= 0 only).
  int32_t chunk0[kMaxWave + 1];
};

// Device-side views used by the grouped projection kernels.
struct GroupView {
  const int32_t* sorted_pairs;  // [P] pair ids grouped by expert
  const int32_t* offsets;       // [E+1]
  const int32_t* active;        // [E]
  const int32_t* n_active;      // [1]
  const int32_t* tile_offsets;  // [E+1] MFMA row-tile prefix sum (MFMA path)
  // Experts with at least this many rows in the call run on the MFMA kernels
  // (their row tiles are in tile_offsets), the others on the GEMV kernels.
  int32_t mfma_rows;
};

// MFMA row tiles of an expert with cnt rows when experts with at least
// mfma_rows rows take the MFMA kernels.
__host__ __device__ inline int mfma_row_tiles(int cnt, int mfma_rows) {
  return cnt >= mfma_rows ? (cnt + kMfmaRows - 1) / kMfmaRows : 0;
}

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float x) {
  return __builtin_bit_cast(uint16_t, (__bf16)x);  // v_cvt_pk_bf16_f32, nearest even
}

__device__ __forceinline__ float half_bits_to_f32(uint16_t b) {
  return __half2float(__ushort_as_half(b));
}

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

// ---------------------------------------------------------------------------
// Device-coherent access.  Inside the fused decode launch, workgroups on
// different XCDs exchange data; the per-XCD L2 caches are not coherent with
// each other, and cache-wide writeback / invalidate fences cost microseconds
// per workgroup.  Data crossing workgroups is therefore written and read with
// device-coherent accesses (sc1) instead, and ordered with an explicit wait
// for outstanding memory operations.  kCo = false gives ordinary accesses.
// ---------------------------------------------------------------------------
template <bool kCo>
__device__ __forceinline__ void st_u32(void* p, uint32_t v) {
  if (kCo) __hip_atomic_store(static_cast<uint32_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else *static_cast<uint32_t*>(p) = v;
}

template <bool kCo>
__device__ __forceinline__ uint32_t ld_u32(const void* p) {
  if (kCo) return __hip_atomic_load(static_cast<const uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return *static_cast<const uint32_t*>(p);
}

template <bool kCo>
__device__ __forceinline__ int32_t ld_i32(const int32_t* p) { return (int32_t)ld_u32<kCo>(p); }

template <bool kCo>
__device__ __forceinline__ float ld_f32(const float* p) { return __uint_as_float(ld_u32<kCo>(p)); }

// 16-byte loads from one buffer (base pointer uniform across the wavefront).
// The coherent form is a raw buffer load with the sc1 cache policy.
template <bool kCo>
struct Buf128 {
  const uint8_t* base;
  __amdgpu_buffer_rsrc_t rsrc;
  __device__ __forceinline__ Buf128(const void* b, uint32_t bytes)
      : base(static_cast<const uint8_t*>(b)) {
    if (kCo) rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(b), (short)0, (int)bytes,
                                                      0x00020000);
  }
  __device__ __forceinline__ uint4 load(uint32_t byte_offset) const {
    if (kCo) {
      typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
      const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)byte_offset, 0, /*sc1*/ 16);
      return make_uint4(v.x, v.y, v.z, v.w);
    }
    return *reinterpret_cast<const uint4*>(base + byte_offset);
  }
};

// Wait until this wavefront's memory operations have completed (made
// device-visible for coherent stores), without moving memory operations
// across it.
__device__ __forceinline__ void wait_memory() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Resolve the wave-local expert index w to (expert, slot); false if unused.
// Workgroup y's chunk of an expert's grouped rows for the GEMV kernels: the
// wave's experts in order (wave.expert, or the active list when n < 0), each
// split into ceil(rows / kGemvRows) chunks of consecutive rows [begin, end).
// False past the last chunk.  Every lane returns the same.
__device__ __forceinline__ bool resolve_wave_chunk(const WaveArg& wave, const GroupView& gv, int y,
                                                   int& expert, int& slot, int& begin, int& end) {
  int c;
  if (wave.n >= 0) {
    if (y >= wave.chunk0[wave.n]) return false;
    int lo = 0, hi = wave.n;  // chunk0[lo] <= y < chunk0[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (wave.chunk0[mid] <= y) lo = mid; else hi = mid;
    }
    expert = wave.expert[lo];
    slot = wave.slot_of[expert];
    c = y - wave.chunk0[lo];
  } else {
    // Every active expert; lane l takes list positions 4l .. 4l+3.
    const int n = *gv.n_active;
    const int lane = lane_id();
    int cnt[4], local = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int w = 4 * lane + i;
      cnt[i] = 0;
      if (w < n) {
        const int e = gv.active[w];
        const int rows = gv.offsets[e + 1] - gv.offsets[e];
        cnt[i] = rows < gv.mfma_rows ? (rows + kGemvRows - 1) / kGemvRows : 0;
      }
      local += cnt[i];
    }
    int incl = local;
#pragma unroll
    for (int dl = 1; dl < 64; dl <<= 1) {
      const int t = __shfl_up(incl, dl);
      if (lane >= dl) incl += t;
    }
    const int start = incl - local;
    const uint64_t hit = __ballot(y >= start && y < incl);
    if (hit == 0) return false;
    const int src = (int)__builtin_ctzll(hit);
    // Position within the source lane's four.
    int i = 0, at = start;
#pragma unroll
    for (int k = 0; k < 3; ++k)
      if (i == k && y >= at + cnt[k]) {
        at += cnt[k];
        i = k + 1;
      }
    i = __builtin_amdgcn_readlane(i, src);
    at = __builtin_amdgcn_readlane(at, src);
    expert = gv.active[4 * src + i];
    slot = expert;
    c = y - at;
  }
  begin = gv.offsets[expert] + c * kGemvRows;
  end = min(begin + kGemvRows, gv.offsets[expert + 1]);
  return true;
}

// ---------------------------------------------------------------------------
// Kernel launch.  While the C ABI's profiler is on, the next launch records a
// start/stop event pair at dispatch (hipExtLaunchKernelGGL), which times the
// kernel itself rather than the stream around it.
// ---------------------------------------------------------------------------
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
  bool used = false;
};
LaunchEvents& launch_events();  // per host thread

template <typename Kernel, typename... Args>
inline void launch(Kernel kernel, dim3 grid, dim3 block, hipStream_t stream, Args... args) {
  LaunchEvents& ev = launch_events();
  hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, ev.start, ev.stop, 0, args...);
  ev.used = true;
}

// Record the calling thread's emoe_last_error() message and return status
// (used by C ABI entry points outside capi.hip).
int32_t report_error(int32_t status, const char* fmt, ...);

// ---------------------------------------------------------------------------
// Launchers (return the launch status; arguments are validated by the caller)
// ---------------------------------------------------------------------------
hipError_t launch_quantize(int d, int f, int n_experts, const uint16_t* w_gate,
                           const uint16_t* w_up, const uint16_t* w_down, uint8_t* records,
                           int32_t* range_flag, hipStream_t stream);

// tok_bias (optional, d a multiple of 512): also -136 * the sum of each
// 128-input group of every token row, fp32 [tokens][d/128].
hipError_t launch_router_logits(int tokens, int n_experts, int d, const uint16_t* h,
                                const uint16_t* w_router, float* logits, hipStream_t stream,
                                float* tok_bias = nullptr);

hipError_t launch_topk(int tokens, int n_experts, int top_k, int renormalize, const float* logits,
                       int32_t* topk_ids, float* topk_w, hipStream_t stream);

// Grouping by expert (Sec. 3.4 step 1) in one workgroup; pair_pos receives
// the inverse permutation (grouped position of each pair id), tile_offsets
// the MFMA row tiles of the experts with at least mfma_rows rows.
hipError_t launch_group(int pairs, int n_experts, const int32_t* topk_ids, int32_t* counts,
                        int32_t* offsets, int32_t* sorted_pairs, int32_t* active,
                        int32_t* n_active, int32_t* tile_offsets, int32_t* pair_pos,
                        int mfma_rows, hipStream_t stream);

// The same grouping over many workgroups, for large calls (pairs > 0): per
// 64-pair chunk expert counts into chunk_counts [ceil(pairs/64)][E], then the
// offsets and a stable placement (identical results to launch_group).
hipError_t launch_group_count(int pairs, int n_experts, const int32_t* topk_ids,
                              int32_t* chunk_counts, hipStream_t stream);
// Top-k (as launch_topk) together with launch_group_count's chunk_counts, in
// one launch; only for top_k dividing 64 with 64 / top_k <= 16.
constexpr bool topk_count_fits(int top_k) { return top_k >= 4 && 64 % top_k == 0; }
hipError_t launch_topk_count(int tokens, int n_experts, int top_k, int renormalize,
                             const float* logits, int32_t* topk_ids, float* topk_w,
                             int32_t* chunk_counts, hipStream_t stream);
hipError_t launch_group_place(int pairs, int n_experts, const int32_t* topk_ids,
                              const int32_t* chunk_counts, int32_t* counts, int32_t* offsets,
                              int32_t* sorted_pairs, int32_t* active, int32_t* n_active,
                              int32_t* tile_offsets, int32_t* pair_pos, int mfma_rows,
                              hipStream_t stream);
constexpr int kGroupWideMinPairs = 1024;  // smaller calls group in one workgroup

// Number of wave-local expert indices a grouped launch must cover.
// GEMV row chunks to launch: exact for a wave, else a bound (each active
// expert adds at most one partial chunk).
inline int grid_chunks(const WaveArg& wave, int n_experts, int pairs) {
  if (wave.n >= 0) return wave.chunk0[wave.n];
  return (pairs + kGemvRows - 1) / kGemvRows + (pairs < n_experts ? pairs : n_experts);
}

hipError_t launch_gateup_gemv(int d, int f, int top_k, int pairs, int n_experts,
                              const uint16_t* h, const GroupView& gv, const WaveArg& wave,
                              const uint8_t* slot_bank, int64_t record_bytes, uint16_t* act,
                              hipStream_t stream);

hipError_t launch_down_gemv(int d, int f, int top_k, int pairs, int n_experts,
                            const uint16_t* act, const GroupView& gv, const WaveArg& wave,
                            const uint8_t* slot_bank, int64_t record_bytes, float* pair_out,
                            hipStream_t stream);

// Grouped MFMA projections.  h_bias / act_bias: -136 * the sum of each
// 128-input group of the projection's input rows: h_bias per token, fp32
// [tokens][d/128] (from the router, or launch_row_bias); act_bias by grouped
// position, fp32 [f/128][pairs], written by the gate/up launch for the down
// launch.  Each workgroup gathers its row tile's values once.
hipError_t launch_row_bias(int tokens, int K, const uint16_t* x, float* bias, hipStream_t stream);

hipError_t launch_gateup_mfma(int tokens, int d, int f, int top_k, int n_experts, const uint16_t* h,
                              const float* h_bias, const GroupView& gv, const WaveArg& wave,
                              const uint8_t* slot_bank, int64_t record_bytes, uint16_t* act,
                              float* act_bias, hipStream_t stream);

// The MFMA down projection writes its pair outputs in bf16 (pair_out_f32
// null) or in fp32 (into pair_out_f32; the per-expert path choice, where the
// GEMV kernels write the other pairs' outputs in fp32).
hipError_t launch_down_mfma(int tokens, int d, int f, int top_k, int n_experts, const uint16_t* act,
                            const float* act_bias, const GroupView& gv, const WaveArg& wave,
                            const uint8_t* slot_bank, int64_t record_bytes, uint16_t* pair_out,
                            float* pair_out_f32, hipStream_t stream);

// pair_out: fp32 (GEMV paths) or bf16 (pair_out_bf16, MFMA path).
hipError_t launch_combine(int tokens, int d, int top_k, const float* topk_w, const void* pair_out,
                          bool pair_out_bf16, uint16_t* y, hipStream_t stream);

}  // namespace emoe
