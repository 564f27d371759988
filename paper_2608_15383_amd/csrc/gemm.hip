// Grouped projections on bf16 MFMA for the many-tokens-per-expert regime
// (prefill / large batches), where each expert's projection is a dense
// contraction over its token rows.
//
// A workgroup of 4 wavefronts owns one row tile (up to 64 token rows of one
// expert, grouped order) and one column tile of 256 weight rows; each
// wavefront owns 4 weight row-blocks (64 outputs) for all 64 rows.  Two
// workgroups share a CU (34 KB of LDS each, 256 VGPRs per lane), and their
// wavefronts, not barrier-aligned with each other, fill each other's load
// and barrier gaps on the matrix cores.
//  - Per 128-input group, the token rows (16 KB, shared by the workgroup) are
//    copied from memory straight into LDS by buffer loads with the LDS
//    destination, and each wavefront's four packed weight tiles (its 16 bytes
//    of each) go straight into registers; both one group ahead of their use,
//    in a ring of two stages.  The 16-byte chunks of a token row are
//    XOR-swizzled by the row index, which makes the MFMA A-fragment reads free
//    of bank conflicts.  The per-row bias of the group is one contiguous
//    256-byte run and the wavefront's 64 scales one 8-byte load per lane, so a
//    group costs each wavefront 10 vector memory instructions, issued in four
//    parts spread over the previous group's k-steps.
//  - Each dword of codes expands in registers to one B operand of
//    v_mfma_f32_16x16x32_bf16 (record layout in common.h): the codes enter as
//    bf16 (128 + u), and the chain of four MFMAs of a group starts from the
//    accumulator value -136 * (row sum of the group), precomputed per row, so
//    the fp32 chain result is sum_k x_k * q_k with q = u - 8.  It is scaled by
//    the FP16 group scale in fp32; the dequantized weight s * q is never
//    rounded (Sec. 3.2).
//  - The stages are handed over with one barrier per group; waits count only
//    this wavefront's outstanding loads.
// Work items (row tile, column tile) are dealt to the XCDs in contiguous
// eighths, so the column tiles of a row tile and the row tiles of an expert
// share one L2.  The gate/up launch is persistent (each workgroup takes
// several items of its XCD's eighth in turn); the down launch takes one item
// per workgroup.
#include <mutex>
#include <type_traits>

#include "common.h"


namespace emoe {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kNPW = 4;                                   // 16-row weight blocks per wavefront
constexpr int kRows = kMfmaRows;                          // 64 token rows per tile
constexpr int kChunks = kGroup / 8;                       // 16-byte chunks per row and group
constexpr float kCodeBias = 136.f;                        // 128 (magic number) + 8 (offset binary)
constexpr int kXcds = 8;                                  // accelerator complex dies per device
constexpr bool kIssueFirst = true;  // a group's load part goes out before its k-step's MFMAs

// Shape of a grouped-projection launch: kWaves wavefronts per workgroup, each
// owning 4 weight row blocks (64 outputs) of a 64-token row tile, and a ring
// of two stages (LDS for the token rows, registers for the weights).
template <int kWaves_>
struct Shape {
  static constexpr int kWaves = kWaves_;
  static constexpr int kStages = 2;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kCols = kWaves * kNPW * kTileRows;   // weight rows per workgroup
  static constexpr int kDma = kRows * kChunks / kThreads;   // token-row chunk copies per thread
  // Workgroups per CU: two wavefronts share each SIMD either way.
  static constexpr int kBlocksPerCu = 8 / kWaves;
};

// One stage of the LDS ring.  The stages are separate LDS variables, so the
// compiler can tell the loads landing in one stage from the reads of another.
template <int kWaves>
struct Stage {
  uint16_t a[kRows * kGroup];            // token rows of the group (swizzled chunks)
  float spare[kWaves][kRows];            // room for the epilogue's padded output tile
};

constexpr int kMaxBiasGroups = kMfmaMaxGroups;

// Stage S of the ring of a kWaves-wide workgroup (one LDS variable each).
template <int kWaves, int S>
__device__ __forceinline__ Stage<kWaves>& stage_mem() {
  __shared__ __attribute__((aligned(16))) Stage<kWaves> st;
  return st;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Buffer loads of 16 (4) bytes per lane into LDS at lds + 16 (4) * lane.
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t rsrc, void* lds, uint32_t voffset,
                                           uint32_t soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)lds, 16,
                                           (int)voffset, (int)soffset, 0, 0);
}
__device__ __forceinline__ void load_lds4(__amdgpu_buffer_rsrc_t rsrc, void* lds, uint32_t voffset,
                                          uint32_t soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)lds, 4,
                                           (int)voffset, (int)soffset, 0, 0);
}

// Wait until at most n of this wavefront's vector memory loads are in flight.
template <int n>
__device__ __forceinline__ void wait_loads() {
  static_assert(n >= 0 && n < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier that orders LDS accesses but does not wait for loads.
__device__ __forceinline__ void barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Four bf16 pairs (128 + u) from one dword of codes: ((dw >> 4p) & mask) |
// magic.  The caller passes mask and magic as opaque register values, so the
// compiler emits one v_and_or_b32 per pair (gfx9 VOP3 takes no literal) and
// still sees every instruction for its MFMA operand hazard checks.
__device__ __forceinline__ bf16x8_t dequant_b(uint32_t dw, uint32_t mask, uint32_t magic) {
  const uint32_t p0 = (dw & mask) | magic;
  const uint32_t p1 = ((dw >> 4) & mask) | magic;
  const uint32_t p2 = ((dw >> 8) & mask) | magic;
  const uint32_t p3 = ((dw >> 12) & mask) | magic;
  return __builtin_bit_cast(bf16x8_t, make_uint4(p0, p1, p2, p3));
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// silu(x) = x / (1 + e^-x) with the hardware exp2 and reciprocal (about 1 ulp
// each in fp32; the result is rounded to bf16 next).  Large negative x gives
// e^-x = inf and a zero reciprocal, so silu -> -0 as in exact arithmetic.
__device__ __forceinline__ float silu_fast(float x) {
  const float e = __builtin_amdgcn_exp2f(-x * 1.44269504088896340736f);
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}

// kGateUp: x = h [tokens][d] gathered through the grouped pair ids, bias the
// per-token table [tokens][d/128], weights W13, output act (bf16, grouped
// order) plus the bias table of act for the down projection.  Otherwise:
// x = act [pairs][f] in grouped order, bias act's table [f/128][pairs] by
// grouped position, weights W2, output pair_out (bf16, pair-id order), or
// pair_out_f32 (fp32) when that is given.
// bias holds -136 * the sum of each 128-input group of each input row.
template <bool kGateUp, typename Sh>
__global__ __launch_bounds__(Sh::kThreads, Sh::kBlocksPerCu) void grouped_mfma_kernel(
    int d, int f, int top_k, int n_experts, const uint16_t* __restrict__ x, uint32_t x_bytes,
    const float* __restrict__ bias, int pairs, GroupView gv, WaveArg wave,
    const uint8_t* __restrict__ slot_bank, int64_t record_bytes, int n_ctiles,
    uint16_t* __restrict__ act_out, float* __restrict__ act_bias_out, uint16_t* __restrict__ pair_out,
    float* __restrict__ pair_out_f32) {
  constexpr int kWaves = Sh::kWaves;
  constexpr int kStages = Sh::kStages;
  constexpr int kCols = Sh::kCols;
  constexpr int kDma = Sh::kDma;
  using StageT = Stage<kWaves>;
  static_assert(kStages * sizeof(StageT) * Sh::kBlocksPerCu <= 160 * 1024, "LDS");
  static_assert(kRows * (kCols / 2 + 8) * 2 <= sizeof(StageT), "gate/up epilogue tile");
  static_assert(kRows / 2 * (kCols + 8) * 2 <= sizeof(StageT), "down epilogue half tile");
  auto stage_of = [&](auto stage) __attribute__((always_inline)) -> StageT& {
    return stage_mem<kWaves, decltype(stage)::value>();
  };
  StageT& st0 = stage_mem<kWaves, 0>();
  StageT& st1 = stage_mem<kWaves, 1>();
  // The tile's bias, [group][row], gathered once in the prologue.
  __shared__ __attribute__((aligned(16))) float bias_lds[kMaxBiasGroups][kRows];
  // Down: the pair id of each tile row, read in the prologue for the epilogue.
  __shared__ int pair_lds[kRows];

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wi = __builtin_amdgcn_readfirstlane(tid >> 6);

  // Work item -> (row tile, column tile).  Workgroup i runs on XCD i % 8;
  // each XCD takes one contiguous eighth of the items in (row tile, column
  // tile) order, so the column tiles of a row tile and the row tiles of an
  // expert meet in one L2 and its token rows and weights cross the fabric
  // about once.
  // Gate/up: the grid holds at most the co-resident workgroups, and
  // workgroup i takes the items i / 8, i / 8 + gridDim / 8, ... of its XCD's
  // eighth in turn (no workgroup launch per item); down: one item per
  // workgroup.
  const int n_items = gv.tile_offsets[n_experts] * n_ctiles;
  const int per_xcd = (n_items + kXcds - 1) / kXcds;
  auto run_item = [&](const int item) __attribute__((always_inline)) {
  const int tile = item / n_ctiles;
  const int ctile = item - tile * n_ctiles;
  // Row tile -> expert (largest e with tile_offsets[e] <= tile).
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
  const int n_blocks = (kGateUp ? 2 * f : d) / kTileRows;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* rec = slot_bank + (int64_t)slot * record_bytes;
  // A wavefront's 4 row blocks are all valid or all past the end (the number
  // of row blocks is a multiple of 8); a wavefront past the end loads row
  // block 0 so every wavefront issues the same loads, and computes nothing.
  const int rb_raw = kNPW * (ctile * kWaves + wi);
  const bool wvalid = rb_raw < n_blocks;
  const int rb0 = wvalid ? rb_raw : 0;
  const int n_local = lane & 15;
  const int quarter = lane >> 4;

  const __amdgpu_buffer_rsrc_t x_rsrc = make_rsrc(x, x_bytes);
  const __amdgpu_buffer_rsrc_t w_rsrc = make_rsrc(rec, (uint32_t)record_bytes);

  // Source row of a tile row (rows past the tile's end repeat its last row;
  // their results are discarded).
  auto src_row = [&](int m) __attribute__((always_inline)) -> int {
    const int mc = min(m, rows - 1);
    return kGateUp ? gv.sorted_pairs[row0 + mc] / top_k : row0 + mc;
  };
  // Token-row chunks this thread copies: stage chunk (kDma*wi + j)*64 + lane
  // is row m = 4*(kDma*wi + j) + lane/16, slot p = lane%16, holding chunk
  // p ^ (m%16).
  uint32_t a_off[kDma];
#pragma unroll
  for (int j = 0; j < kDma; ++j) {
    const int m = 4 * (kDma * wi + j) + (lane >> 4);
    const int c = (lane & 15) ^ (m & 15);
    a_off[j] = (uint32_t)src_row(m) * (uint32_t)(K * 2) + 16u * c;
  }
  // Bias gather: thread t fills row t % 64 of every kWaves-th group from
  // t / 64 on; its source row (a token for gate/up, a grouped position for
  // down) is known now, so the gather overlaps the first group's loads.
  const int b_row = tid & (kRows - 1);
  const int b_src = src_row(b_row);
  const uint32_t w_off = (uint32_t)((kGateUp ? L.w13_codes : L.w2_codes) +
                                    (int64_t)rb0 * G * kTileBytes) + 16u * lane;
  // Scales of the wavefront's four row blocks for one group: 128 bytes, the
  // lane's four (blocks 0..3 of row n_local) in 8 consecutive bytes.
  const uint32_t s_off = (uint32_t)((kGateUp ? L.w13_scales : L.w2_scales) +
                                    scale_index(16 * rb0, 0, G) * 2) + 8u * n_local;

  // Registers of the groups in flight: fp16 scales (block r in half r) and
  // the codes of the four weight tiles (lane's 16 bytes of each).
  uint2 sc[kStages];
  uint4 wreg[kStages][kNPW];

  // The loads of group g into stage S (same count in every thread), in four
  // parts: 0 and 1 copy half of the token-row chunks each into LDS, 2 and 3
  // load two weight tiles each into registers (3 also the scales).  The parts
  // go out one per k-step of the group being computed, so the wavefronts of
  // a workgroup do not all queue their loads on the CU's address path at the
  // same moment.
  auto issue_part = [&](int g, auto stage, auto part) __attribute__((always_inline)) {
    constexpr int S = decltype(stage)::value;
    constexpr int P = decltype(part)::value;
    StageT& sm = stage_of(stage);
    if constexpr (P < 2) {
#pragma unroll
      for (int j = P * (kDma / 2); j < (P + 1) * (kDma / 2); ++j)
        load_lds16(x_rsrc, &sm.a[(kDma * wi + j) * 64 * 8], a_off[j], (uint32_t)g * kGroup * 2);
    } else {
#pragma unroll
      for (int r = 2 * (P - 2); r < 2 * (P - 1); ++r)
        wreg[S][r] = __builtin_bit_cast(
            uint4, __builtin_amdgcn_raw_buffer_load_b128(
                       w_rsrc, (int)(w_off + (uint32_t)(r * G * kTileBytes)), g * kTileBytes, 0));
      if constexpr (P == 3)
        sc[S] = __builtin_bit_cast(
            uint2, __builtin_amdgcn_raw_buffer_load_b64(w_rsrc, (int)s_off, g * 128, 0));
    }
  };
  static_assert(kDma % 2 == 0 && kNPW == 4, "four load parts");
  auto issue = [&](int g, auto stage) __attribute__((always_inline)) {
    issue_part(g, stage, std::integral_constant<int, 0>());
    issue_part(g, stage, std::integral_constant<int, 1>());
    issue_part(g, stage, std::integral_constant<int, 2>());
    issue_part(g, stage, std::integral_constant<int, 3>());
  };

  // Dequantization constants, hidden from constant folding (the empty asm
  // statements emit nothing): mask in an SGPR, magic in a VGPR.
  uint32_t kMask = 0x000f000fu, kMagic = 0x43004300u;
  asm("" : "+s"(kMask));
  asm("" : "+v"(kMagic));

  f32x4_t acc[kNPW][4];
#pragma unroll
  for (int r = 0; r < kNPW; ++r)
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) acc[r][mi] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // kMB: row blocks holding tile rows (the last tile of an expert may fill
  // fewer than 4; the blocks past its rows are skipped).
  // With `more`, k-step i also issues load part i of group g + 1 into the
  // other stage (before the k-step's MFMAs when kIssueFirst).
  auto compute = [&](int g, auto stage, auto mb, auto more) __attribute__((always_inline)) {
    constexpr int S = decltype(stage)::value;
    constexpr int kMB = decltype(mb)::value;
    constexpr bool kMore = decltype(more)::value;
    using Next = std::integral_constant<int, S ^ 1>;
    const StageT& sm = stage_of(stage);
    f32x4_t c0[4];
#pragma unroll
    for (int mi = 0; mi < kMB; ++mi)
      c0[mi] = *reinterpret_cast<const f32x4_t*>(&bias_lds[g][16 * mi + 4 * quarter]);
    uint4 wc[kNPW];
#pragma unroll
    for (int r = 0; r < kNPW; ++r) wc[r] = wreg[S][r];
    f32x4_t tmp[kNPW][4];
    auto kstep = [&](auto ic) __attribute__((always_inline)) {
      constexpr int i = decltype(ic)::value;
      if constexpr (kMore && kIssueFirst) {
        __builtin_amdgcn_sched_barrier(0);
        issue_part(g + 1, Next(), ic);
        __builtin_amdgcn_sched_barrier(0);
      }
      bf16x8_t a[4];
#pragma unroll
      for (int mi = 0; mi < kMB; ++mi) {
        const int m = 16 * mi + n_local;
        a[mi] = *reinterpret_cast<const bf16x8_t*>(&sm.a[m * kGroup + 8 * ((4 * i + quarter) ^ n_local)]);
      }
#pragma unroll
      for (int r = 0; r < kNPW; ++r) {
        const uint32_t dw = i == 0 ? wc[r].x : i == 1 ? wc[r].y : i == 2 ? wc[r].z : wc[r].w;
        const bf16x8_t b = dequant_b(dw, kMask, kMagic);
#pragma unroll
        for (int mi = 0; mi < kMB; ++mi)
          tmp[r][mi] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mi], b, i == 0 ? c0[mi] : tmp[r][mi], 0, 0, 0);
      }
      if constexpr (kMore && !kIssueFirst) {
        __builtin_amdgcn_sched_barrier(0);
        issue_part(g + 1, Next(), ic);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    kstep(std::integral_constant<int, 0>());
    kstep(std::integral_constant<int, 1>());
    kstep(std::integral_constant<int, 2>());
    kstep(std::integral_constant<int, 3>());
#pragma unroll
    for (int r = 0; r < kNPW; ++r) {
      const uint32_t sw = r < 2 ? sc[S].x : sc[S].y;
      const float s = half_bits_to_f32((r & 1) ? sw >> 16 : sw & 0xffffu);
#pragma unroll
      for (int mi = 0; mi < kMB; ++mi)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[r][mi][j] = fmaf(s, tmp[r][mi][j], acc[r][mi][j]);
    }
  };

  // One group: load the next group into the other stage, compute this one,
  // then wait for the loads and hand the stages over.  Issuing is decided at
  // compile time so the wait counts stay exact.
  auto step = [&](int g, auto stage, auto more, auto mb) __attribute__((always_inline)) {
    constexpr int S = decltype(stage)::value;
    if (wvalid) {
      compute(g, stage, mb, more);
    } else if constexpr (decltype(more)::value) {
      issue(g + 1, std::integral_constant<int, S ^ 1>());
    }
    wait_loads<0>();
    barrier();
  };
  using Yes = std::true_type;
  using No = std::false_type;
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;

  issue(0, S0());
  // Gather the tile's bias while the first group loads.
  for (int gg = wi; gg < G; gg += kWaves)
    bias_lds[gg][b_row] = kGateUp ? bias[(int64_t)b_src * G + gg] : bias[(int64_t)gg * pairs + b_src];
  if (!kGateUp && tid < kRows) pair_lds[tid] = gv.sorted_pairs[b_src];
  wait_loads<0>();
  barrier();
  // Groups 0 .. G-2 issue the next group; pairs of steps run in the loop.
  auto main_loop = [&](auto mb) __attribute__((always_inline)) {
    int g = 0;
    for (; g + 2 <= G - 1; g += 2) {
      step(g, S0(), Yes(), mb);
      step(g + 1, S1(), Yes(), mb);
    }
    if (G - 1 - g == 1) {
      step(g, S0(), Yes(), mb);
      step(g + 1, S1(), No(), mb);
    } else {
      step(g, S0(), No(), mb);
    }
  };
  const int n_mb = (rows + 15) >> 4;
  if (n_mb >= 4)
    main_loop(std::integral_constant<int, 4>());
  else if (n_mb == 3)
    main_loop(std::integral_constant<int, 3>());
  else if (n_mb == 2)
    main_loop(std::integral_constant<int, 2>());
  else
    main_loop(std::integral_constant<int, 1>());

  // Epilogue.  Lane holds rows m = 16*mi + 4*quarter + j of output column
  // n_local of its row blocks.  Outputs are rounded to bf16, staged in LDS
  // (the stages are free now) and written as 16-byte chunks.
  if (kGateUp) {
    // act = silu(gate) * up (row block 2p is gate, 2p+1 up); the workgroup's
    // kCols/2 act columns start at kCols/2 * ctile.
    constexpr int kActCols = kCols / 2;   // act columns of this workgroup
    constexpr int kStride = kActCols + 8;  // row pitch in bf16 (padded against bank conflicts)
    uint16_t* tile_act = reinterpret_cast<uint16_t*>(&st0);
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int p = 0; p < kNPW / 2; ++p) {
          const float gv_ = acc[2 * p][mi][j];
          const float uv = acc[2 * p + 1][mi][j];
          tile_act[(16 * mi + 4 * quarter + j) * kStride + 16 * (2 * wi + p) + n_local] =
              (uint16_t)f32_to_bf16_rne(silu_fast(gv_) * uv);
        }
    barrier();
    // Thread t copies chunks (row t/R + (kThreads/R)q, column chunk t%R, with
    // R = kActCols/8 chunks per row) and sums each chunk; the 16 threads of
    // one 128-column group then add their sums (butterfly), giving the bias
    // of that row and group for the down kernel.
    constexpr int R = kActCols / 8;
    const int cc = tid % R;
    const int col = kActCols * ctile + 8 * cc;
    const int Gf = f / kGroup;
    const int g = col / kGroup;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int m = tid / R + (Sh::kThreads / R) * q;
      const uint4 v = *reinterpret_cast<const uint4*>(&tile_act[m * kStride + 8 * cc]);
      const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
      float sum = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sum += bf16_bits_to_f32(w4[e] & 0xffffu);
        sum += bf16_bits_to_f32(w4[e] >> 16);
      }
      sum += __shfl_xor(sum, 1);
      sum += __shfl_xor(sum, 2);
      sum += __shfl_xor(sum, 4);
      sum += __shfl_xor(sum, 8);
      if (m < rows && col < f) {
        *reinterpret_cast<uint4*>(act_out + (int64_t)(row0 + m) * f + col) = v;
        if ((tid & 15) == 0) act_bias_out[(int64_t)g * pairs + row0 + m] = -kCodeBias * sum;
      }
    }
  } else if (pair_out_f32) {
    // fp32 outputs straight from the accumulators: 16 consecutive columns
    // (64 bytes) of one row per 16 lanes.
    if (wvalid) {
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int m = 16 * mi + 4 * quarter + j;
          if (m < rows) {
            float* out = pair_out_f32 + (int64_t)pair_lds[m] * d + 16 * rb0 + n_local;
#pragma unroll
            for (int r = 0; r < kNPW; ++r) out[16 * r] = acc[r][mi][j];
          }
        }
    }
  } else {
    // Rows 0..31 are staged in stage 0, rows 32..63 in stage 1.
    constexpr int kStride = kCols + 8;
    uint16_t* half0 = reinterpret_cast<uint16_t*>(&st0);
    uint16_t* half1 = reinterpret_cast<uint16_t*>(&st1);
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
      uint16_t* t = mi < 2 ? half0 : half1;
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < kNPW; ++r)
          t[(16 * (mi & 1) + 4 * quarter + j) * kStride + 16 * (kNPW * wi + r) + n_local] =
              (uint16_t)f32_to_bf16_rne(acc[r][mi][j]);
    }
    barrier();
    constexpr int R = kCols / 8;   // chunks per output row
    const int cc = tid % R;
    const int col = kCols * ctile + 8 * cc;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int m = tid / R + (Sh::kThreads / R) * q;
      const uint16_t* t = m < 32 ? half0 : half1;
      if (m < rows && col < d) {
        const uint4 v = *reinterpret_cast<const uint4*>(&t[(m & 31) * kStride + 8 * cc]);
        const int pi = pair_lds[m];
        *reinterpret_cast<uint4*>(pair_out + (int64_t)pi * d + col) = v;
      }
    }
  }
  };
  if constexpr (kGateUp) {
    const int xstride = (int)gridDim.x / kXcds;
    for (int xj = blockIdx.x / kXcds; xj < per_xcd; xj += xstride) {
      const int item = (blockIdx.x % kXcds) * per_xcd + xj;
      if (item >= n_items) break;
      run_item(item);
      barrier();  // the next item's prologue writes the LDS this epilogue reads
    }
  } else {
    const int xj = blockIdx.x / kXcds;
    if (xj >= per_xcd) return;
    const int item = (blockIdx.x % kXcds) * per_xcd + xj;
    if (item >= n_items) return;
    run_item(item);
  }
}

// bias[t][g] = -136 * sum of x[t][128g .. 128g+127] (fp32, fixed order): the
// accumulator start of the gate/up MFMA chains of every pair of token t.
__global__ __launch_bounds__(256) void row_bias_kernel(int tokens, int K, const uint16_t* __restrict__ x,
                                                       float* __restrict__ bias) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= tokens) return;
  const int lane = lane_id();
  const uint16_t* xr = x + (int64_t)t * K;
  for (int c0 = 0; c0 < K / 8; c0 += 64) {
    const int c = c0 + lane;
    float s = 0.f;
    if (c < K / 8) {
      const uint4 v = *reinterpret_cast<const uint4*>(xr + 8 * c);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        s += bf16_bits_to_f32(w[q] & 0xffffu);
        s += bf16_bits_to_f32(w[q] >> 16);
      }
    }
    // Sum over the 16 lanes holding one group.
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 4);
    s += __shfl_xor(s, 8);
    if ((lane & 15) == 0 && c < K / 8) bias[(int64_t)t * (K / kGroup) + c / kChunks] = -kCodeBias * s;
  }
}

inline int max_row_tiles(int pairs, int n_experts) {
  const int e = pairs < n_experts ? pairs : n_experts;
  return (pairs + kRows - 1) / kRows + e;
}

// Launch shape of both projections.
using MfmaShape = Shape<4>;

// Co-resident workgroups of the gate/up projection on the current device,
// rounded down to a multiple of the XCD count (0 if unknown).
int gateup_resident() {
  static std::mutex mu;
  static int cap[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  std::lock_guard<std::mutex> lk(mu);
  if (cap[dev] == 0) {
    int n = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, reinterpret_cast<const void*>(grouped_mfma_kernel<true, MfmaShape>),
            MfmaShape::kThreads, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    cap[dev] = n * cus / kXcds * kXcds;
  }
  return cap[dev];
}

// Workgroups for n_ctiles column tiles and up to max_row_tiles row tiles: a
// multiple of the XCD count, so every XCD gets its eighth of the items; at
// most `limit` (then each takes several items in turn) when limit >= 8.
inline int mfma_grid(int n_ctiles, int pairs, int n_experts, int limit) {
  const int n = n_ctiles * max_row_tiles(pairs, n_experts);
  const int all = (n + kXcds - 1) / kXcds * kXcds;
  return limit >= kXcds && limit < all ? limit : all;
}

}  // namespace

hipError_t launch_row_bias(int tokens, int K, const uint16_t* x, float* bias, hipStream_t stream) {
  if (tokens == 0) return hipSuccess;
  launch(row_bias_kernel, dim3((tokens + 3) / 4), dim3(256), stream, tokens, K, x, bias);
  return hipGetLastError();
}

hipError_t launch_gateup_mfma(int tokens, int d, int f, int top_k, int n_experts, const uint16_t* h,
                              const float* h_bias, const GroupView& gv, const WaveArg& wave,
                              const uint8_t* slot_bank, int64_t record_bytes, uint16_t* act,
                              float* act_bias, hipStream_t stream) {
  const int pairs = tokens * top_k;
  if (pairs == 0) return hipSuccess;
  constexpr int kCols = MfmaShape::kCols;
  const int n_ctiles = (2 * f + kCols - 1) / kCols;
  launch(grouped_mfma_kernel<true, MfmaShape>,
         dim3(mfma_grid(n_ctiles, pairs, n_experts, gateup_resident())),
         dim3(MfmaShape::kThreads), stream, d, f, top_k, n_experts, h,
         (uint32_t)((int64_t)tokens * d * 2), h_bias, pairs,
         gv, wave, slot_bank, record_bytes, n_ctiles, act, act_bias, (uint16_t*)nullptr,
         (float*)nullptr);
  return hipGetLastError();
}

hipError_t launch_down_mfma(int tokens, int d, int f, int top_k, int n_experts, const uint16_t* act,
                            const float* act_bias, const GroupView& gv, const WaveArg& wave,
                            const uint8_t* slot_bank, int64_t record_bytes, uint16_t* pair_out,
                            float* pair_out_f32, hipStream_t stream) {
  const int pairs = tokens * top_k;
  if (pairs == 0) return hipSuccess;
  constexpr int kCols = MfmaShape::kCols;
  const int n_ctiles = (d + kCols - 1) / kCols;
  launch(grouped_mfma_kernel<false, MfmaShape>, dim3(mfma_grid(n_ctiles, pairs, n_experts, 0)),
         dim3(MfmaShape::kThreads), stream, d, f, top_k, n_experts, act,
         (uint32_t)((int64_t)pairs * f * 2), act_bias, pairs,
         gv, wave, slot_bank, record_bytes, n_ctiles, (uint16_t*)nullptr, (float*)nullptr, pair_out,
         pair_out_f32);
  return hipGetLastError();
}

}  // namespace emoe
