// Fused single-launch decode layer for a few tokens with every expert
// resident (C = E, Sec. 3.3): route, top-k, gate/up + SwiGLU, down and the
// weighted combine in one kernel.
//
// On MI355X a kernel boundary costs about 2.4 us and a dependent round trip to
// memory about 1 us under load, against roughly 5 us to stream the decode
// layer's 26 MB of packed weights.  The six-kernel sequence is therefore
// replaced by one grid whose workgroups play these roles by index:
//   [0, nR)        router items: logits of one expert (its inputs split
//                  over the four wavefronts) or of four experts, for one or
//                  two tokens (with more than two tokens the items split
//                  them);
//   [nR, nR+nG)    gate/up workers: worker j runs gate/up item j (pair
//                  p = j / chunks, some of its row-block pairs; pairs in
//                  token-major order), then down_r output row blocks of pair
//                  p - down_lag;
//   [nR+nG, ...)   tail workers: tail_r output row blocks of one of the
//                  last tail_pairs pairs (the gate/up workers of the last
//                  tail_pairs - down_lag pairs have no down work).
// Every worker waits for the router items, reads the logits and runs the
// top-k itself (cheap, and it saves the round trips of publishing the
// selection); gate/up workers stage the token rows in LDS while they wait.
// Each worker loads the first down tiles of its pair while the gate/up items
// stream theirs, picks up that pair's activation row once it is complete and
// splits each row block's input groups over its four wavefronts.  Items
// finish roughly in dispatch order, so with a lag of two pairs a gate/up
// worker that finishes its item finds its down pair's row already complete,
// and the rows that complete last go to the tail workers, idle since their
// top-k.  Every pair's down projection is spread over as many workgroups as
// gate/up items, and a pair's activations come from workers of lower index
// than the ones that read them.  The
// workers holding the last pair of a token then read the token's other k - 1
// expert outputs (also from workers of lower index) and add the k outputs in
// rank order.  The first tail worker finally writes the routing and grouping
// arrays to the workspace, as the unfused path does.
//
// Data crossing workgroups (logits, activation rows, expert outputs) travels
// as 64-bit words tagged with the launch's epoch, written and read
// device-coherently: the reader polls the data itself, so one store is both the payload and the
// signal, and nothing needs resetting between launches.  The host numbers
// launches itself; a launch captured into a graph instead takes its epoch
// from device memory and advances it there, so that every replay has a new
// one (the two kinds use disjoint halves of the tag space).  A workgroup only
// waits for workgroups of lower index, which the hardware dispatches first,
// and the grid is sized to be co-resident on an idle GPU.  Every wait is
// still bounded and counts a timeout instead of spinning forever.
//
// The arithmetic is that of the stand-alone kernels (device_route.h,
// device_gemv.h), so the result is bit-identical to the unfused path.
#include <mutex>

#include "decode.h"
#include "device_gemv.h"
#include "device_route.h"

namespace emoe {
namespace {

// Phase timestamps for measurement builds (compiled with -DEMOE_PHASE_TRACE by
// phase_trace.py; absent otherwise): word 16 b + i holds the wall clock
// (100 MHz) at which workgroup b passed phase i.  Thread 0 keeps them in LDS
// while the workgroup runs and copies them out as it exits, so the trace adds
// no stores to the vector-memory counter that the kernel's own waits count.
#ifdef EMOE_PHASE_TRACE
__device__ uint64_t g_phase_trace[kFusedMaxBlocks * 16];
#define EMOE_TRACE_LDS __shared__ uint64_t s_trace[16]
#define EMOE_TRACE_INIT()                                                               \
  do {                                                                                  \
    if (threadIdx.x == 0)                                                               \
      for (int k_ = 0; k_ < 16; ++k_) s_trace[k_] = 0;                                  \
  } while (0)
#define EMOE_PHASE(i)                                                                   \
  do {                                                                                  \
    if (threadIdx.x == 0) s_trace[i] = wall_clock64();                                  \
  } while (0)
#define EMOE_PHASE_WAVE(i)                                                              \
  do {                                                                                  \
    if (threadIdx.x == 0) s_trace[i] = wall_clock64();                                  \
  } while (0)
#define EMOE_TRACE_SET(i, v)                                                            \
  do {                                                                                  \
    if (threadIdx.x == 0) s_trace[i] = (v);                                             \
  } while (0)
#define EMOE_TRACE_FLUSH()                                                              \
  do {                                                                                  \
    if (threadIdx.x == 0)                                                               \
      for (int k_ = 0; k_ < 16; ++k_) g_phase_trace[blockIdx.x * 16 + k_] = s_trace[k_]; \
  } while (0)
#else
#define EMOE_TRACE_LDS static_assert(true, "")
#define EMOE_TRACE_INIT() do {} while (0)
#define EMOE_PHASE(i) do {} while (0)
#define EMOE_PHASE_WAVE(i) do {} while (0)
#define EMOE_TRACE_SET(i, v) do {} while (0)
#define EMOE_TRACE_FLUSH() do {} while (0)
#endif

// Polls before the epoch advance of captured launches gives up; the
// hand-over waits take theirs from DecodeArgs::spin_limit (the same 2^20
// unless a test lowers it).
constexpr uint32_t kSpinLimit = 1u << 20;
constexpr int kPollSleep = 1;  // s_sleep units (64 clocks) between polls
// Between polls of the logits with several tokens: then every wavefront of a
// worker that has a token polls, while the router items still stream their
// weights (one token: wavefront 0 alone, kPollSleep).
constexpr int kLogitPollSleep = 4;

// Token t's logits into st.v: from logits_override, or from the router
// items' tagged words (replica `replica`), read until every word carries this
// launch's epoch (bounded).
__device__ __forceinline__ bool load_logits(DecodeSync* sy, const DecodeArgs& a, uint32_t epoch,
                                            int replica, int t, TopkState& st) {
  const int lane = lane_id();
  const int E = a.n_experts;
  if (a.logits_override) {
#pragma unroll
    for (int c = 0; c < kPerLane; ++c) {
      const int e = lane + 64 * c;
      st.v[c] = e < E ? a.logits_override[(int64_t)t * E + e] : 0.f;
    }
    return false;
  }
  const uint64_t* zt = sy->logits[replica] + t * E;
  uint32_t it = 0;
  while (true) {
    bool ok = true;
#pragma unroll
    for (int c = 0; c < kPerLane; ++c) {
      const int e = lane + 64 * c;
      if (e < E) {
        const uint64_t x = __hip_atomic_load(zt + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = ok && (uint32_t)(x >> 32) == (epoch ^ a.tag_xor);
        st.v[c] = __uint_as_float((uint32_t)x);
      } else {
        st.v[c] = 0.f;
      }
    }
    if (__all(ok)) return false;
    if (++it > a.spin_limit) {
      if (lane == 0) atomicAdd(&sy->timeouts, 1u);
      return true;
    }
    if (a.tokens > 1)
      __builtin_amdgcn_s_sleep(kLogitPollSleep);
    else
      __builtin_amdgcn_s_sleep(kPollSleep);
  }
}

// The epoch of a captured launch, as the last one left it.  The same in every
// lane; used as loaded, so the first wait for the load is at the first use.
__device__ __forceinline__ uint32_t launch_epoch(DecodeSync* sy) {
  return __hip_atomic_load(&sy->epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Record that workgroup blk has read this launch's epoch (one thread).  The
// word is a plain store to the workgroup's own location, so nothing contends;
// the empty asm takes the epoch as an operand, so the store is issued only
// once the load of the old epoch has returned.
__device__ __forceinline__ void arrive(DecodeSync* sy, uint32_t epoch, int blk) {
  uint32_t e = epoch;
  asm volatile("" : "+v"(e));
  __hip_atomic_store(&sy->arrived[blk], e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Router workgroup 0, one wavefront: once every workgroup of the launch has
// recorded this epoch (bounded wait), store the next one (skipping 0, the tag
// of zeroed memory).  No
// workgroup waits on this one after its logits are out, so the wait ends
// whether or not the grid is co-resident.
__device__ __forceinline__ void advance_epoch(DecodeSync* sy, uint32_t epoch, int n_blocks) {
  constexpr int kPer = kFusedMaxBlocks / 64;
  const int lane = lane_id();
  uint32_t it = 0;
  while (true) {
    bool ok = true;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int b = lane + 64 * k;
      if (b < n_blocks)
        ok = ok && __hip_atomic_load(&sy->arrived[b], __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT) == epoch;
    }
    if (__all(ok)) break;
    if (++it > kSpinLimit) {
      if (lane == 0) atomicAdd(&sy->timeouts, 1u);
      break;
    }
    __builtin_amdgcn_s_sleep(kPollSleep);
  }
  const uint32_t next = epoch + 1u == 0u ? kDeviceEpoch0 : epoch + 1u;
  if (lane == 0) __hip_atomic_store(&sy->epoch, next, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Copy `bytes` (a multiple of 256) from coherent global memory to LDS with
// buffer loads that target LDS (one wavefront, 4 bytes per lane per load,
// device-coherent: sc1).  Completion is this wavefront's vmcnt.
__device__ __forceinline__ void wave_copy_to_lds(const void* src, uint32_t bytes, void* lds) {
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(src), (short)0, (int)bytes, 0x00020000);
  const uint32_t voff = 4u * (uint32_t)lane_id();
  for (uint32_t off = 0; off < bytes; off += 256)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc, (__attribute__((address_space(3))) void*)(static_cast<uint8_t*>(lds) + off), 4,
        (int)voff, (int)off, 0, /*sc1*/ 16);
}

// Down tiles of one wavefront for up to kUnits row blocks: input groups
// g = wi + 4j (j < kGW) of each, codes (this lane's 16 bytes of the tile) and
// raw fp16 scales (converted at use, so no load waits for another).
template <int kGW, int kU = 16 / kGW>
struct DownTiles {
  static constexpr int kUnits = kU;  // row blocks per batch (at most 64 code registers)
  uint4 c[kUnits][kGW];
  uint16_t s[kUnits][kGW];
};

// Load this wavefront's tiles of row blocks rb .. rb+nb-1 (nb <= kUnits).
template <int kGW, int kU>
__device__ __forceinline__ void load_down_tiles(const uint8_t* __restrict__ rec, int d, int f,
                                                int rb, int nb, DownTiles<kGW, kU>& t) {
  const int lane = lane_id();
  const int wi = threadIdx.x >> 6;
  const int G = f / kGroup;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* codes = rec + L.w2_codes + 16 * lane;
  const uint16_t* sc = reinterpret_cast<const uint16_t*>(rec + L.w2_scales);
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    if (u < nb) {
      const int n = 16 * (rb + u) + (lane & 15);
#pragma unroll
      for (int j = 0; j < kGW; ++j) {
        const int g = wi + 4 * j;
        if (g < G) {
          t.c[u][j] = *reinterpret_cast<const uint4*>(codes + ((int64_t)(rb + u) * G + g) * kTileBytes);
          t.s[u][j] = sc[scale_index(n, g, G)];
        }
      }
    }
  }
}

// Units kFrom .. nb-1 of a batch (row blocks rb + kFrom ..).
template <int kGW, int kFrom, int kU>
__device__ __forceinline__ void load_down_tiles_from(const uint8_t* __restrict__ rec, int d, int f,
                                                     int rb, int nb, DownTiles<kGW, kU>& t) {
  const int lane = lane_id();
  const int wi = threadIdx.x >> 6;
  const int G = f / kGroup;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* codes = rec + L.w2_codes + 16 * lane;
  const uint16_t* sc = reinterpret_cast<const uint16_t*>(rec + L.w2_scales);
#pragma unroll
  for (int u = kFrom; u < kU; ++u) {
    if (u < nb) {
      const int n = 16 * (rb + u) + (lane & 15);
#pragma unroll
      for (int j = 0; j < kGW; ++j) {
        const int g = wi + 4 * j;
        if (g < G) {
          t.c[u][j] = *reinterpret_cast<const uint4*>(codes + ((int64_t)(rb + u) * G + g) * kTileBytes);
          t.s[u][j] = sc[scale_index(n, g, G)];
        }
      }
    }
  }
}

// Row blocks rb .. rb+kN-1 into units 0 .. kN-1, every load issued so that
// the waits for loads issued before these stay exact: a unit past nb reads
// unit nb-1 again, a row block past the last reads the last one and a slot
// past the last group reads the last group (all unused).
template <int kGW, int kN, int kU>
__device__ __forceinline__ void load_down_tiles_all(const uint8_t* __restrict__ rec, int d, int f,
                                                    int rb, int nb, DownTiles<kGW, kU>& t) {
  static_assert(kN <= kU, "units of one batch");
  const int lane = lane_id();
  const int wi = threadIdx.x >> 6;
  const int G = f / kGroup;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* codes = rec + L.w2_codes + 16 * lane;
  const uint16_t* sc = reinterpret_cast<const uint16_t*>(rec + L.w2_scales);
#pragma unroll
  for (int u = 0; u < kN; ++u) {
    const int r = min(rb + min(u, nb - 1), d / kTileRows - 1);
    const int n = 16 * r + (lane & 15);
#pragma unroll
    for (int j = 0; j < kGW; ++j) {
      const int g = min(wi + 4 * j, G - 1);
      t.c[u][j] = *reinterpret_cast<const uint4*>(codes + ((int64_t)r * G + g) * kTileBytes);
      t.s[u][j] = sc[scale_index(n, g, G)];
    }
  }
}

// Down row blocks a gate/up worker loads with its gate/up tiles: with those
// of a one-pair item, and with the last pair's of a several-pair item (the
// rest of its first batch follows in the down part).
constexpr int kDownEarly = 2;
template <int kGW>
constexpr int kDownEarlyMany = 8 / kGW;  // eight tiles per wavefront

}  // namespace

// The down row blocks [rb0, rb0 + nu) of pair q that worker wk of a planned
// launch computes (nu = 0: none): gate/up worker wk (wk < n_gate, pair
// p = wk / chunks) takes pair p - down_lag unless that is one of the last
// tail_pairs pairs, which the tail workers take, per_pair workers of tail_r
// row blocks per pair.  Host and device share it (the kernel and the plan
// checks).
__host__ __device__ FusedDownWork fused_down_work(const DecodeArgs& a, int wk) {
  const int P = a.tokens * a.top_k;
  const int n_rb = a.d / kTileRows;
  const int chunks = (a.f / kTileRows + a.pairs_per_item - 1) / a.pairs_per_item;
  FusedDownWork w;
  const bool is_gate = wk < a.n_gate;
  if (is_gate) {
    w.q = wk / chunks - a.down_lag;
    if (w.q >= P - a.tail_pairs) w.q = -1;  // the tail workers' pairs
    w.rb0 = (wk % chunks) * a.down_r;
  } else {
    // Tail worker j: pair P - tail_pairs + j / per_pair, row-block set j % per_pair.
    const int per_pair = (n_rb + a.tail_r - 1) / a.tail_r;
    int j = wk - a.n_gate;
    w.q = P - a.tail_pairs;
    while (j >= per_pair) {
      j -= per_pair;
      ++w.q;
    }
    w.rb0 = j * a.tail_r;
  }
  const int r = is_gate ? a.down_r : a.tail_r;
  w.nu = w.q < 0 ? 0 : (n_rb - w.rb0 < r ? n_rb - w.rb0 : r);
  if (w.nu < 0) w.nu = 0;
  return w;
}

namespace {

// kDevEpoch: the launch is being captured into a graph and reads its epoch
// from DecodeSync (a.epoch is 0); otherwise a.epoch is the host's number.
// kGW: input groups of the down projection per wavefront (d_ff <= 512 kGW).
// kMany: gate/up items may hold several row-block pairs (pairs_per_item > 1);
// without it the launch has one-pair items only and compiles without the
// several-pair code, which leaves that code's registers to the rest.
template <bool kDevEpoch, int kGW, bool kMany>
__global__ __launch_bounds__(256, 3) void decode_fused_kernel(DecodeArgs a) {
  __shared__ GroupShared<256> gsh;
  __shared__ GateUpShared gush;
  __shared__ int32_t s_ids[kFusedMaxPairs];
  __shared__ float s_w[kFusedMaxPairs];
  __shared__ uint4 s_act[kFusedActLdsBytes / 16];
  __shared__ uint32_t s_xw[kGemvWaves][kGW * kGroup / 2];        // staged activations
  __shared__ float s_part[kGemvWaves][kFusedMaxDownUnits][16];    // per-class down outputs
  __shared__ uint64_t s_topk[kFusedMaxTokens][64];                // top-k scratch per token
  __shared__ double s_rsum[kGemvWaves][2];                         // router: quarter sums
  __shared__ int s_rank[kGemvWaves][64];                          // partial ranks (one token)
  __shared__ int s_late[2][kGemvWaves];  // per wavefront: a bounded wait gave up (route, down)

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wi = tid >> 6;
  const int blk = blockIdx.x;
  DecodeSync* sy = a.sync;
  const int P = a.tokens * a.top_k;
  const uint32_t epoch = kDevEpoch ? launch_epoch(sy) : a.epoch;
  EMOE_TRACE_LDS;
  EMOE_TRACE_INIT();
  EMOE_PHASE(0);  // start
  if (blk == 0) {  // the layout, for reading the trace
    EMOE_TRACE_SET(14, (uint64_t)a.n_router | (uint64_t)a.n_gate << 16 | (uint64_t)a.n_work << 32);
    EMOE_TRACE_SET(15, (uint64_t)a.pairs_per_item | (uint64_t)a.down_r << 16 |
                           (uint64_t)a.tail_r << 32 | (uint64_t)a.down_lag << 48 |
                           (uint64_t)a.tail_pairs << 56);
  }

  if (blk < a.n_router) {
    // ---------------------------------------------------------------- router
    // Each logit goes to the workspace and, tagged with the epoch, to
    // kSyncLanes replicas, so the hundreds of readers below spread over as
    // many memory locations.
    if (!a.logits_override) {
      // With router_shift 1, items 2i and 2i + 1 take expert group i for
      // tokens 0, 1 and 2, 3; with 0, item i takes group i for every token.
      // A group is one expert whose inputs the four wavefronts split in
      // quarters (router_experts 1), or four experts, one per wavefront.
      static_assert(kFusedMaxTokens <= 4, "two router items per expert group at most");
      const int t0 = 2 * (blk & a.router_shift);
      const int t1 = min(a.tokens, t0 + 2);
      auto publish = [&](int t, int e, double sum) {
        const uint32_t v = __float_as_uint((float)sum);
        const int at = t * a.n_experts + e;
        if (lane < kSyncLanes)
          __hip_atomic_store(&sy->logits[lane][at], ((uint64_t)epoch << 32) | v,
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (lane == kSyncLanes) st_u32<false>(a.logits + at, v);
      };
      if (a.router_experts == 1) {
        const int e = blk >> a.router_shift;
        const int kq = a.d / kGemvWaves;
        wave_router_dot_part(t0, t1, a.d, wi * kq, kq, e, a.h, a.w_router,
                             [&](int t, double sum) { s_rsum[wi][t - t0] = sum; });
        __syncthreads();
        // The quarters in wavefront order (the sum is exact, so any order
        // gives these bits).
        if (wi == 0)
          for (int t = t0; t < t1; ++t)
            publish(t, e, ((s_rsum[0][t - t0] + s_rsum[1][t - t0]) + s_rsum[2][t - t0]) +
                              s_rsum[3][t - t0]);
      } else {
        const int e0 = 4 * (blk >> a.router_shift) + wi;
        if (e0 < a.n_experts)
          wave_router_dot(t0, t1, a.d, e0, a.h, a.w_router,
                          [&](int t, double sum) { publish(t, e0, sum); });
      }
    }
    EMOE_PHASE(1);  // router: logits stored
    if (kDevEpoch) {
      if (tid == 0) arrive(sy, epoch, blk);
      if (blk == 0 && wi == 0) advance_epoch(sy, epoch, (int)gridDim.x);
    }
    EMOE_TRACE_FLUSH();
    return;
  }

  // Worker wk runs gate/up item wk (pair p = wk / chunks, chunk wk % chunks)
  // and then the down row blocks [rb0, rb0 + nu) of pair q = p - down_lag,
  // whose activation row is complete by the time this later-dispatched item
  // is; the tail workers (wk >= n_gate), idle since their top-k, take the
  // down row blocks of the last tail_pairs pairs (>= down_lag), whose rows
  // complete last, so the items of the last tail_pairs - down_lag pairs,
  // which finish last, have no down work.  Every wait is for lower-indexed
  // workgroups.  The workers that hold the last pair of a token combine that
  // token's outputs.
  const int wk = blk - a.n_router;
  const bool is_gate = wk < a.n_gate;
  const int chunks = (a.f / kTileRows + a.pairs_per_item - 1) / a.pairs_per_item;
  const FusedDownWork dw = fused_down_work(a, wk);
  const int q = dw.q, rb0 = dw.rb0, nu = dw.nu;
  const bool is_comb = nu > 0 && q % a.top_k == a.top_k - 1;  // combines token q / k
  const bool writes_routing = wk == a.n_gate;                  // the first tail worker

  // Gate/up workers stage the token rows of h in LDS (s_act) while the router
  // runs: 256-byte chunks round-robin over the wavefronts.
  const uint16_t* h_lds = reinterpret_cast<const uint16_t*>(s_act);
  if (is_gate) {
    const uint32_t bytes = (uint32_t)a.tokens * (uint32_t)a.d * 2u;
    for (uint32_t off = 256u * wi; off < bytes; off += 256u * kGemvWaves)
      wave_copy_to_lds(reinterpret_cast<const uint8_t*>(a.h) + off, 256u,
                       reinterpret_cast<uint8_t*>(s_act) + off);
  }

  // Every worker: token t's logits (this launch's epoch in every tag) and its
  // selection.  One token: wavefront 0 loads the logits and publishes the
  // rank keys, each wavefront counts, for every expert, the larger keys in
  // its quarter of them, and wavefront 0 adds the counts.  Several tokens:
  // wavefront t < T ranks token t alone.
  const int replica = blk % kSyncLanes;
  TopkState st;
  bool late = false;  // a bounded wait of this wavefront gave up
  if (a.tokens == 1 && a.n_experts <= 64) {
    static_assert(kGemvWaves * 16 == 64, "a quarter of 64 keys per wavefront");
    uint64_t* keys = s_topk[1];
    if (wi == 0) {
      late = load_logits(sy, a, epoch, replica, 0, st);
      EMOE_PHASE_WAVE(1);  // worker: logits seen
      keys[lane] = topk_lane_key(st, a.n_experts);
    }
    __syncthreads();
    s_rank[wi][lane] = topk_count_greater<16>(keys + 16 * wi, keys[lane]);
    __syncthreads();
    if (wi == 0) {
      int rank = 0;
#pragma unroll
      for (int w = 0; w < kGemvWaves; ++w) rank += s_rank[w][lane];
      topk_select_ranked(rank, a.top_k, st, s_topk[0]);
      wave_topk_store_ids<false>(st, a.top_k, s_ids);
    }
  } else if (wi < a.tokens) {
    late = load_logits(sy, a, epoch, replica, wi, st);
    wave_topk_select_loaded(a.n_experts, a.top_k, st, s_topk[wi]);
    wave_topk_store_ids<false>(st, a.top_k, s_ids + wi * a.top_k);
  }
  // The mixture weights, for the combining workers (their token's) and the
  // one that writes the routing arrays (every token's).
  if (wi < a.tokens && (writes_routing || (is_comb && wi == q / a.top_k)))
    wave_topk_weights<false>(st, a.n_experts, a.top_k, a.renormalize, s_w + wi * a.top_k);
  if (is_gate) wait_memory();  // the staged rows
  if (lane == 0) s_late[0][wi] = late;
  __syncthreads();
  // Logits that never arrived leave this workgroup's selection invalid: its
  // outputs become NaN rather than passing as valid results.
  const bool route_late = s_late[0][0] | s_late[0][1] | s_late[0][2] | s_late[0][3];
  EMOE_PHASE(2);  // top-k done
  // A read epoch has been waited for by now (the logits' tags): from here on
  // a scalar.  Tail workers record it before their first tile loads, so that
  // no later wait covers the store; gate/up workers after their item.
  const uint32_t ep = kDevEpoch ? __builtin_amdgcn_readfirstlane(epoch) : a.epoch;
  if (kDevEpoch && !is_gate && tid == 0) arrive(sy, ep, blk);
  const uint64_t tag = (uint64_t)ep << 32;


  // The first batch of this worker's down tiles (pair q's record).
  // One-pair launches take their down work in batches of kDownEarly row
  // blocks (all of it at OLMoE shape), which keeps the unrolled arithmetic,
  // run by every workgroup at the same moment, short.
  using Tiles = DownTiles<kGW, kMany ? 16 / kGW : kDownEarly>;
  Tiles dn;
  const uint8_t* drec = a.slot_bank + (int64_t)s_ids[max(q, 0)] * a.record_bytes;
  // Gate/up item: pair pi, row-block pairs b0 .. b1-1.
  const int pi = wk / chunks;
  const int b0 = (wk % chunks) * a.pairs_per_item;
  const int b1 = min(b0 + a.pairs_per_item, a.f / kTileRows);
  // Items whose tiles all load in one batch per pair issue this worker's
  // first batch of down tiles with their last gate/up tiles: a one-pair item
  // (down_r <= kDownEarly) with the pair's tiles, a several-pair item in
  // place of the next pair's.
  const bool one_batch = a.d <= kGemvWaves * kGateBatch * kGroup;
  const bool early_one = is_gate && b1 - b0 == 1 && a.down_r <= kDownEarly &&
                         a.d == kGemvWaves * kGateBatch * kGroup;
  const bool early_many = kMany && is_gate && b1 - b0 > 1 && one_batch;
  const bool early = early_one || early_many;

  if (is_gate) {
    // ---------------------------------------------------------------- gate/up
    // Item = (pair pi, row-block pairs b0 ..): one token row of one expert.
    // The activation goes to act row pi (pair order).
    const int e = s_ids[pi];
    const int top_k = a.top_k;
    // The activation goes out as tagged words (DecodeSync::act), which the
    // down workers poll directly: the store is the signal.
    const int d = a.d, f = a.f;
    const uint32_t nan_mask = route_late ? 0x7fc07fc0u : 0u;  // bf16 NaN pair
    uint64_t* act_tag = sy->act;
    auto store_act = [=](int s, int n, uint32_t v) {
      __hip_atomic_store(act_tag + ((s * f + n) >> 1), tag | v | nan_mask, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    };
    const uint8_t* rec = a.slot_bank + (int64_t)e * a.record_bytes;
    // (A worker of pair 0, which has no down work, reads pair 0's tiles,
    // unused.)
    if (early_one) {
      // The pair's tiles, then this worker's down tiles, are issued before
      // the pair is computed, so the down tiles stream with the gate/up
      // weights.
      GateUpBatch gb;
      gateup_load_batch(rec, d, f, b0, gb);
      load_down_tiles_all<kGW, kDownEarly>(drec, d, f, rb0, max(nu, 1), dn);
      gateup_pair_compute<true>(gush, d, h_lds + (pi / top_k) * d, pi, gb, b0, store_act);
    } else if (early_many) {
      // The next row-block pair's tiles load while this one is computed, and
      // the down tiles while the last one is.
      if constexpr (kMany)
        gateup_row_blocks(gush, d, f, h_lds + (pi / top_k) * d, pi, rec, b0, b1, store_act, [&] {
          load_down_tiles_all<kGW, kDownEarlyMany<kGW>>(
              drec, d, f, rb0, max(min(nu, kDownEarlyMany<kGW>), 1), dn);
        });
    } else {
      for (int b = b0; b < b1; ++b)
        gateup_rows(gush, d, f, [=](int s) { return h_lds + (s / top_k) * d; }, pi, pi + 1, rec,
                    b, store_act);
    }
    EMOE_PHASE(4);  // gate/up item done
    if (kDevEpoch && tid == 0) arrive(sy, ep, blk);
  }

  // ------------------------------------------------------------------ down
  // The down tiles of pair q: wavefront wi takes the input groups g = wi + 4j
  // (j < kGW) of every row block.  A tail worker reaches this point right
  // after its top-k, so its first batch streams in while the gate/up items
  // stream theirs; a gate/up worker after its item (loads issued before the
  // item's would be waited for with them).
  const int G = a.f / kGroup;
  EMOE_PHASE(3);  // down part reached
  bool act_late = false;
  if (nu > 0) {
    if (!early)
      load_down_tiles<kGW>(drec, a.d, a.f, rb0, min(nu, Tiles::kUnits), dn);
    else if (kMany && early_many)
      load_down_tiles_from<kGW, kDownEarlyMany<kGW>>(drec, a.d, a.f, rb0, min(nu, Tiles::kUnits),
                                                     dn);
    // This wavefront's groups of activation row q, from the tagged words
    // (one per lane and group, all read before any is checked; bounded wait)
    // into its LDS slot.
    uint32_t* xw = s_xw[wi];
    const uint64_t* src = sy->act + (int64_t)q * (a.f / 2);
    uint32_t it = 0;
    while (wi < G) {  // a wavefront without groups (d_ff < 512) has nothing to read
      uint64_t x[kGW];
#pragma unroll
      for (int j = 0; j < kGW; ++j)  // slots past G read group wi's words again
        x[j] = __hip_atomic_load(src + (wi + 4 * j < G ? wi + 4 * j : wi) * (kGroup / 2) + lane,
                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      bool ok = true;
#pragma unroll
      for (int j = 0; j < kGW; ++j) {
        ok &= (uint32_t)(x[j] >> 32) == (ep ^ a.tag_xor);
        xw[j * (kGroup / 2) + lane] = (uint32_t)x[j];
      }
      if (__all(ok)) break;
      if (++it > a.spin_limit) {
        if (lane == 0) atomicAdd(&sy->timeouts, 1u);
        act_late = true;
        break;
      }
      __builtin_amdgcn_s_sleep(kPollSleep);
    }
    __builtin_amdgcn_wave_barrier();
    EMOE_PHASE(5);  // activation row staged (wavefront 0)
    const uint16_t* xh = reinterpret_cast<const uint16_t*>(xw);
    const int quarter = lane >> 4;
    // The lane's 32 activations of group slot j (4 x uint4).
    auto xload = [&](int j, uint4* x) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        x[i] = *reinterpret_cast<const uint4*>(xh + j * kGroup + 8 * quarter + 32 * i);
    };
    float xs[kGW];
#pragma unroll
    for (int j = 0; j < kGW; ++j) {
      uint4 x[4];
      xload(j, x);
      xs[j] = lane_group_xsum(x);
    }
    // Batches of Tiles::kUnits row blocks (one batch unless d_ff is large).
    // Per row block the wavefront's groups are added in order into one
    // accumulator: its class (groups g with g % 4 == wi) of the output
    // (device_gemv.h, down_class_total).
    for (int u0 = 0; u0 < nu; u0 += Tiles::kUnits) {
      const int nb = min(Tiles::kUnits, nu - u0);
      if (u0 > 0) load_down_tiles<kGW>(drec, a.d, a.f, rb0 + u0, nb, dn);
      float acc[Tiles::kUnits];
#pragma unroll
      for (int u = 0; u < Tiles::kUnits; ++u) acc[u] = 0.f;
#pragma unroll
      for (int j = 0; j < kGW; ++j) {
        if (wi + 4 * j >= G) break;
        uint4 x[4];
        xload(j, x);
#pragma unroll
        for (int u = 0; u < Tiles::kUnits; ++u) {
          if (u < nb) {
            float unused = 0.f;
            const float pr = lane_group_dot(dn.c[u][j], x, unused, false);
            acc[u] = fmaf(half_bits_to_f32(at_use(dn.s[u][j])), fmaf(-136.f, xs[j], pr), acc[u]);
          }
        }
      }
#pragma unroll
      for (int u = 0; u < Tiles::kUnits; ++u) {
        if (u < nb) {
          const float v = reduce_quarters(acc[u]);
          if (lane < 16) s_part[wi][u0 + u][lane] = v;
        }
      }
    }
  }
  EMOE_PHASE(6);  // down tiles computed (wavefront 0)
  if (lane == 0) s_late[1][wi] = act_late;
  __syncthreads();
  if (nu > 0 && tid < 16 * nu) {
    // Output of pair q, rows 16 (rb0 + u) + n: the four classes in the fixed
    // order, handed on as a tagged word (NaN when a wait of this workgroup
    // gave up).
    const int u = tid >> 4, n = tid & 15;
    const int row = 16 * (rb0 + u) + n;
    const bool bad = route_late | s_late[1][0] | s_late[1][1] | s_late[1][2] | s_late[1][3];
    const float o = bad ? __uint_as_float(0x7fc00000u)
                        : (s_part[0][u][n] + s_part[1][u][n]) + (s_part[2][u][n] + s_part[3][u][n]);
    a.pair_out[(int64_t)q * a.d + row] = o;
    if (!is_comb) {
      __hip_atomic_store(sy->out + (int64_t)q * a.d + row, tag | __float_as_uint(o),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      // The token's other k - 1 outputs of this row (bounded wait), then the
      // weighted sum in rank order.
      const int t = q / a.top_k;
      const int p0 = t * a.top_k;
      // Eight words at a time, all read before any is checked (bounded
      // wait); a word with this launch's tag holds its final value.
      const uint64_t* ow = sy->out + (int64_t)p0 * a.d + row;
      const int nk = a.top_k - 1;
      bool comb_late = false;
      float acc = 0.f;
      for (int j0 = 0; j0 < nk; j0 += 8) {
        uint64_t x[8];
        for (uint32_t it = 0;; ++it) {
#pragma unroll
          for (int i = 0; i < 8; ++i)  // past the k - 1 words: read the last again
            x[i] = __hip_atomic_load(ow + (int64_t)min(j0 + i, nk - 1) * a.d, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
          bool ok = true;
#pragma unroll
          for (int i = 0; i < 8; ++i) ok &= (uint32_t)(x[i] >> 32) == (ep ^ a.tag_xor);
          if (ok) break;
          if (it > a.spin_limit) {
            atomicAdd(&sy->timeouts, 1u);
            comb_late = true;
            break;
          }
          __builtin_amdgcn_s_sleep(kPollSleep);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (j0 + i < nk) acc = fmaf(s_w[p0 + j0 + i], __uint_as_float((uint32_t)x[i]), acc);
      }
      EMOE_PHASE(7);  // combining worker: the token's other outputs seen
      acc = fmaf(s_w[p0 + nk], o, acc);
      a.y[(int64_t)t * a.d + row] = (bad | comb_late) ? 0x7fc0 : (uint16_t)f32_to_bf16_rne(acc);
    }
  }

  EMOE_PHASE(9);  // end (before the routing arrays)
  if (writes_routing) {
    // The workspace's routing and grouping arrays, as the unfused path writes them.
    for (int j = tid; j < P; j += 256) {
      a.topk_ids[j] = s_ids[j];
      a.topk_w[j] = s_w[j];
    }
    block_group<256, false>(gsh, P, a.n_experts, s_ids, a.counts, a.offsets, a.sorted_pairs,
                            a.active, a.n_active, nullptr, a.pair_pos, 1);
  }
  EMOE_TRACE_FLUSH();
}

// Co-resident workgroups of the fused kernel (either form) on the current
// device.
int fused_capacity() {
  static std::mutex mu;
  static int cap[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  std::lock_guard<std::mutex> lk(mu);
  if (cap[dev] == 0) {
    // Every instantiation (epoch source, down groups per wavefront, items
    // of several pairs or not) must fit the same number per CU.
    const void* kernels[8] = {
        reinterpret_cast<const void*>(decode_fused_kernel<false, 2, false>),
        reinterpret_cast<const void*>(decode_fused_kernel<true, 2, false>),
        reinterpret_cast<const void*>(decode_fused_kernel<false, 4, false>),
        reinterpret_cast<const void*>(decode_fused_kernel<true, 4, false>),
        reinterpret_cast<const void*>(decode_fused_kernel<false, 2, true>),
        reinterpret_cast<const void*>(decode_fused_kernel<true, 2, true>),
        reinterpret_cast<const void*>(decode_fused_kernel<false, 4, true>),
        reinterpret_cast<const void*>(decode_fused_kernel<true, 4, true>)};
    int per_cu = 1 << 30, cus = 0;
    for (const void* k : kernels) {
      int n = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, 256, 0) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
      }
      per_cu = min(per_cu, n);
    }
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    cap[dev] = per_cu * cus;
  }
  return cap[dev];
}

}  // namespace

bool decode_fused_plan(DecodeArgs& a) {
  return decode_fused_plan_for(a, min(fused_capacity(), kFusedMaxBlocks));
}

bool decode_fused_plan_for(DecodeArgs& a, int cap) {
  if (a.tokens < 1 || a.tokens > kFusedMaxTokens || a.tokens * a.top_k > kFusedMaxPairs)
    return false;
  if (a.d > kFusedMaxD || a.f > 4 * 4 * kGroup) return false;  // sync words; kGW <= 4
  if ((int64_t)a.tokens * a.top_k * (a.f / 2) > kFusedActWords) return false;
  if ((int64_t)a.tokens * a.d * 2 > kFusedActLdsBytes) return false;  // staged token rows
  const int P = a.tokens * a.top_k;
  const int pairs_of_f = a.f / kTileRows;
  const int n_rb = a.d / kTileRows;
  a.gw = a.f <= 8 * kGroup ? 2 : 4;
  // Router items: by (at most) two tokens, one pass each, one expert (its
  // inputs split over the four wavefronts) for at most two tokens and 64
  // experts, else four experts, one per wavefront (with more tokens the
  // one-expert items would fill the grid's last slots for little gain).
  a.router_shift = a.tokens > 2 ? 1 : 0;
  a.router_experts = a.n_experts <= 64 && a.tokens <= 2 ? 1 : 4;
  a.n_router = a.logits_override
                   ? 1
                   : ((a.n_experts + a.router_experts - 1) / a.router_experts) << a.router_shift;
  cap = min(cap, kFusedMaxBlocks);
  // The most gate/up items (fewest row-block pairs each) that fit, with the
  // down row blocks of each pair spread over the items of pair p + lag and
  // the last tail pairs' over as many tail workers as the remaining room
  // allows.
  for (int ppi = 1; ppi <= pairs_of_f; ppi *= 2) {
    // Items of one row-block pair finish with little slack, so there the
    // last pair's items get no down work (one more tail pair than the lag).
    const int tail = min(P, ppi == 1 ? kFusedTailPairs : kFusedDownLag);
    const int lag = min(tail, kFusedDownLag);
    const int chunks = (pairs_of_f + ppi - 1) / ppi;
    const int down_r = (n_rb + chunks - 1) / chunks;
    if (down_r > kFusedMaxDownUnits) break;  // fewer items only raise it
    const int n_gate = P * chunks;
    const int room = min(cap - a.n_router - n_gate, tail * n_rb);
    if (room < tail) continue;
    // Row blocks per tail worker: the fewest for which the tail pairs' worth
    // of workers fit the room.
    int tail_r = (tail * n_rb + room - 1) / room;
    while (tail_r <= kFusedMaxDownUnits && tail * ((n_rb + tail_r - 1) / tail_r) > room) ++tail_r;
    if (tail_r > kFusedMaxDownUnits) continue;
    a.pairs_per_item = ppi;
    a.n_gate = n_gate;
    a.down_r = down_r;
    a.tail_r = tail_r;
    a.down_lag = lag;
    a.tail_pairs = tail;
    a.n_work = n_gate + tail * ((n_rb + tail_r - 1) / tail_r);
    return true;
  }
  return false;
}

hipError_t launch_decode_fused(DecodeArgs& a, DecodeProgress& prog, hipStream_t stream) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(stream, &cs);
  if (e != hipSuccess) return e;
  if (cs == hipStreamCaptureStatusNone) {
    a.epoch = prog.epoch + 1u >= kDeviceEpoch0 ? 1u : prog.epoch + 1u;
  } else {
    a.epoch = 0u;  // replays number themselves in device memory
  }
  const dim3 grid(a.n_router + a.n_work);
  const bool dev_epoch = a.epoch == 0u;
  const bool many = a.pairs_per_item > 1;
  const int form = (dev_epoch ? 1 : 0) | (a.gw == 2 ? 0 : 2) | (many ? 4 : 0);
  switch (form) {
    case 0: launch(decode_fused_kernel<false, 2, false>, grid, dim3(256), stream, a); break;
    case 1: launch(decode_fused_kernel<true, 2, false>, grid, dim3(256), stream, a); break;
    case 2: launch(decode_fused_kernel<false, 4, false>, grid, dim3(256), stream, a); break;
    case 3: launch(decode_fused_kernel<true, 4, false>, grid, dim3(256), stream, a); break;
    case 4: launch(decode_fused_kernel<false, 2, true>, grid, dim3(256), stream, a); break;
    case 5: launch(decode_fused_kernel<true, 2, true>, grid, dim3(256), stream, a); break;
    case 6: launch(decode_fused_kernel<false, 4, true>, grid, dim3(256), stream, a); break;
    default: launch(decode_fused_kernel<true, 4, true>, grid, dim3(256), stream, a); break;
  }
  e = hipGetLastError();
  if (e == hipSuccess && !dev_epoch) prog.epoch = a.epoch;
  return e;
}

}  // namespace emoe

// Host only: the fused launch's plan for `capacity` co-resident workgroups
// and every worker's down work (see exactmoe.h).
extern "C" int32_t emoe_debug_fused_plan(const emoe_dims* dims, int32_t tokens, int32_t capacity,
                                         int32_t* plan, int32_t* work, int32_t max_workers) {
  if (!dims || !plan || (max_workers > 0 && !work) || max_workers < 0 || capacity < 1)
    return EMOE_EINVAL;
  if (emoe_check_dims(dims) != EMOE_OK) return EMOE_ESHAPE;
  emoe::DecodeArgs a{};
  a.tokens = tokens;
  a.d = dims->d_model;
  a.f = dims->d_ff;
  a.n_experts = dims->n_experts;
  a.top_k = dims->top_k;
  if (!emoe::decode_fused_plan_for(a, capacity)) return EMOE_ESHAPE;
  const int32_t v[9] = {a.n_router, a.n_gate,   a.n_work,    a.pairs_per_item, a.down_r,
                        a.tail_r,   a.down_lag, a.tail_pairs, a.gw};
  for (int i = 0; i < 9; ++i) plan[i] = v[i];
  for (int wk = 0; wk < a.n_work && wk < max_workers; ++wk) {
    const emoe::FusedDownWork w = emoe::fused_down_work(a, wk);
    work[3 * wk] = w.q;
    work[3 * wk + 1] = w.rb0;
    work[3 * wk + 2] = w.nu;
  }
  return EMOE_OK;
}

#ifdef EMOE_PHASE_TRACE
// Measurement builds only: copy the phase timestamps of the first n_blocks
// workgroups of the latest fused launch to host memory (16 words each).
extern "C" int32_t emoe_debug_phase_trace(uint64_t* host_out, int32_t n_blocks) {
  if (!host_out || n_blocks < 0 || n_blocks > emoe::kFusedMaxBlocks) return EMOE_EINVAL;
  return hipMemcpyFromSymbol(host_out, HIP_SYMBOL(emoe::g_phase_trace), (size_t)n_blocks * 16 * 8,
                             0, hipMemcpyDeviceToHost) == hipSuccess
             ? EMOE_OK
             : EMOE_EHIP;
}
#endif
