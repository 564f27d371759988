// Fused single-launch decode layer for a few tokens with every expert
// resident (C = E, Sec. 3.3): route, top-k, gate/up + SwiGLU, down and the
// weighted combine in one kernel.
//
// On MI355X a kernel boundary costs about 2.4 us and a dependent round trip to
// memory about 1 us under load, against roughly 5 us to stream the decode
// layer's 26 MB of packed weights.  The six-kernel sequence is therefore
// replaced by one grid whose workgroups play three roles by index:
//   [0, nR)        router items: logits of 4 experts for every token;
//   [nR, nR+nW)    workers: worker j runs gate/up item j (one token-expert
//                  pair, some row-block pairs; items in token-major order),
//                  if j < nG, and then down unit j - D0 (output row block rb
//                  of one token t), if that is in [0, T * d/16).
// D0 places every down unit of token t after the last gate/up item of t, so
// a workgroup only ever waits for workgroups of lower index.  With one token
// the two ranges are disjoint (D0 = nG); with more tokens the later gate/up
// workers take a down unit of an earlier token afterwards, which spreads the
// down work over many more workgroups than the d/16 row blocks.
// Every worker waits for the router items, reads the logits and runs the
// top-k itself (cheap, and it saves the round trips of publishing the
// selection); gate/up items stage the token rows in LDS while they wait.
// Down-only workers prefetch their down tiles while the gate/up items stream
// theirs; every down unit picks up each activation row of its token as it is
// produced and adds the token's k expert outputs in rank order.  Down unit 0
// finally writes the routing and grouping arrays to the workspace, as the
// unfused path does.
//
// Data crossing workgroups (logits, activation rows) travels as 64-bit words
// tagged with the launch's epoch, written and read device-coherently: the
// reader polls the data itself, so one store is both the payload and the
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

constexpr uint32_t kSpinLimit = 1u << 20;
constexpr int kPollSleep = 8;  // s_sleep units (64 clocks) between polls

// Stage the activation row of pair pi from the tagged words (DecodeSync::act)
// in LDS at dst (f bf16), reading it until every word carries this launch's
// epoch (bounded); one wavefront.
__device__ __forceinline__ bool wave_stage_act_row(DecodeSync* sy, const DecodeArgs& a,
                                                   uint32_t epoch, int pi, uint32_t* dst) {
  constexpr int kWords = 8;  // words per lane per read
  const int lane = lane_id();
  const int nw = a.f / 2;  // words per row, a multiple of 64
  const uint64_t* src = sy->act + (int64_t)pi * nw;
  bool timed_out = false;
  for (int w0 = 0; w0 < nw; w0 += 64 * kWords) {
    uint32_t it = 0;
    while (true) {
      uint64_t x[kWords];
#pragma unroll
      for (int k = 0; k < kWords; ++k) {
        const int w = w0 + 64 * k + lane;
        x[k] = w < nw ? __hip_atomic_load(src + w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                      : ((uint64_t)epoch << 32);
      }
      bool ok = true;
#pragma unroll
      for (int k = 0; k < kWords; ++k) {
        const int w = w0 + 64 * k + lane;
        ok = ok && (uint32_t)(x[k] >> 32) == epoch;
        if (w < nw) dst[w] = (uint32_t)x[k];
      }
      if (__all(ok)) break;
      if (++it > kSpinLimit) {
        if (lane == 0) atomicAdd(&sy->timeouts, 1u);
        timed_out = true;
        break;
      }
      __builtin_amdgcn_s_sleep(kPollSleep);
    }
  }
  return timed_out;
}

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
        ok = ok && (uint32_t)(x >> 32) == epoch;
        st.v[c] = __uint_as_float((uint32_t)x);
      } else {
        st.v[c] = 0.f;
      }
    }
    if (__all(ok)) return false;
    if (++it > kSpinLimit) {
      if (lane == 0) atomicAdd(&sy->timeouts, 1u);
      return true;
    }
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

// kDevEpoch: the launch is being captured into a graph and reads its epoch
// from DecodeSync (a.epoch is 0); otherwise a.epoch is the host's number.
template <bool kDevEpoch>
__global__ __launch_bounds__(256, 3) void decode_fused_kernel(DecodeArgs a) {
  __shared__ GroupShared<256> gsh;
  __shared__ GateUpShared gush;
  __shared__ float o_lds[kFusedMaxPairs][16];
  __shared__ int32_t s_ids[kFusedMaxPairs];
  __shared__ float s_w[kFusedMaxPairs];
  __shared__ uint4 s_act[kFusedActLdsBytes / 16];
  __shared__ float s_xs[kGemvWaves][kFusedActLdsBytes / (2 * kGroup * kGemvWaves) * 4];  // [wave][group][quarter]
  __shared__ uint64_t s_topk[kFusedMaxTokens][64];                // top-k scratch per token
  __shared__ int s_rank[kGemvWaves][64];                          // partial ranks (one token)
  __shared__ int s_late[2][kGemvWaves];  // per wavefront: a bounded wait gave up (route, down)

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wi = tid >> 6;
  const int blk = blockIdx.x;
  DecodeSync* sy = a.sync;
  const int P = a.tokens * a.top_k;
  const uint32_t epoch = kDevEpoch ? launch_epoch(sy) : a.epoch;

  if (blk < a.n_router) {
    // ---------------------------------------------------------------- router
    // Each logit goes to the workspace and, tagged with the epoch, to
    // kSyncLanes replicas, so the hundreds of readers below spread over as
    // many memory locations.
    if (!a.logits_override) {
      const int e0 = 4 * blk + wi;
      if (e0 < a.n_experts) {
        wave_router_dot(a.tokens, a.d, e0, a.h, a.w_router, [&](int t, double sum) {
          const uint32_t v = __float_as_uint((float)sum);
          const int at = t * a.n_experts + e0;
          if (lane < kSyncLanes)
            __hip_atomic_store(&sy->logits[lane][at], ((uint64_t)epoch << 32) | v,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if (lane == kSyncLanes) st_u32<false>(a.logits + at, v);
        });
      }
    }
    if (kDevEpoch) {
      if (tid == 0) arrive(sy, epoch, blk);
      if (blk == 0 && wi == 0) advance_epoch(sy, epoch, (int)gridDim.x);
    }
    return;
  }

  // Gate/up workgroups stage the token rows of h in LDS (s_act, which only
  // down workgroups use otherwise) while the router runs: 256-byte chunks
  // round-robin over the wavefronts.
  const int wk = blk - a.n_router;  // worker index
  const bool is_gate = wk < a.n_gate;
  const int unit = wk - a.down0;    // down unit (valid when is_down)
  const bool is_down = unit >= 0 && unit < a.n_down;
  const uint16_t* h_lds = reinterpret_cast<const uint16_t*>(s_act);
  if (is_gate) {
    const uint32_t bytes = (uint32_t)a.tokens * (uint32_t)a.d * 2u;
    for (uint32_t off = 256u * wi; off < bytes; off += 256u * kGemvWaves)
      wave_copy_to_lds(reinterpret_cast<const uint8_t*>(a.h) + off, 256u,
                       reinterpret_cast<uint8_t*>(s_act) + off);
  }

  // Every other workgroup: token t's logits (this launch's epoch in every tag)
  // and its selection.  One token: wavefront 0 loads the logits and publishes
  // the rank keys, each wavefront counts, for every expert, the larger keys in
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
  if (is_gate) wait_memory();  // the staged rows
  if (lane == 0) s_late[0][wi] = late;
  __syncthreads();
  // Logits that never arrived leave this workgroup's selection invalid: its
  // outputs become NaN rather than passing as valid results.
  const bool route_late = s_late[0][0] | s_late[0][1] | s_late[0][2] | s_late[0][3];
  // A read epoch has been waited for by now (the logits' tags): from here on
  // a scalar.  Down workgroups record it before their first tile loads, so
  // that no later wait covers the store; gate/up workgroups at their end.
  const uint32_t ep = kDevEpoch ? __builtin_amdgcn_readfirstlane(epoch) : a.epoch;
  if (kDevEpoch && !is_gate && tid == 0) arrive(sy, ep, blk);

  // The mixture weights are needed only by the combine.  A worker that also
  // runs a gate/up item computes them first (so the selection need not stay
  // in registers through it); a down-only worker while its tiles stream in.
  if (is_gate && is_down && wi < a.tokens)
    wave_topk_weights<false>(st, a.n_experts, a.top_k, a.renormalize, s_w + wi * a.top_k);

  if (is_gate) {
    // ---------------------------------------------------------------- gate/up
    // Item = (pair pi, row-block pairs b0 ..): one token row of one expert.
    // The activation goes to act row pi (pair order).
    const int item = wk;
    const int pairs_of_f = a.f / kTileRows;
    const int chunks = (pairs_of_f + a.pairs_per_item - 1) / a.pairs_per_item;
    const int pi = item / chunks;
    const int b0 = (item % chunks) * a.pairs_per_item;
    const int b1 = min(b0 + a.pairs_per_item, pairs_of_f);
    const int e = s_ids[pi];
    const int top_k = a.top_k;
    // The activation goes out as tagged words (DecodeSync::act), which the
    // down workgroups poll directly: the store is the signal.
    const int d = a.d, f = a.f;
    const uint64_t tag = (uint64_t)ep << 32;
    const uint32_t nan_mask = route_late ? 0x7fc07fc0u : 0u;  // bf16 NaN pair
    uint64_t* act_tag = sy->act;
    for (int b = b0; b < b1; ++b)
      gateup_rows(gush, a.d, a.f, [=](int s) { return h_lds + (s / top_k) * d; }, pi, pi + 1,
                  a.slot_bank + (int64_t)e * a.record_bytes, b, [=](int s, int n, uint32_t v) {
                    __hip_atomic_store(act_tag + ((s * f + n) >> 1), tag | v | nan_mask,
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                  });
    if (kDevEpoch && tid == 0) arrive(sy, ep, blk);
    if (!is_down) return;
    __syncthreads();  // the staged token rows are no longer read: s_act is free
  }

  // ------------------------------------------------------------------ down + combine
  // Unit = (token tu, output row block rb): the token's k pairs p0 .. p1-1.
  const int n_rb = a.d / kTileRows;
  const int tu = unit / n_rb;
  const int rb = unit - tu * n_rb;
  const int p0 = tu * a.top_k, p1 = p0 + a.top_k;
  const int G = a.f / kGroup;
  // Wavefront wi owns pairs p0+wi, p0+wi+4, ...; the first two are prefetched
  // (by a down-only worker while the gate/up items stream).
  DownBatch pre0, pre1;
  if (p0 + wi < p1)
    down_load_batch(a.slot_bank + (int64_t)s_ids[p0 + wi] * a.record_bytes, a.d, a.f, rb, 0, pre0);
  if (p0 + wi + kGemvWaves < p1)
    down_load_batch(a.slot_bank + (int64_t)s_ids[p0 + wi + kGemvWaves] * a.record_bytes, a.d, a.f,
                    rb, 0, pre1);
  if (!is_gate && wi < a.tokens)
    wave_topk_weights<false>(st, a.n_experts, a.top_k, a.renormalize, s_w + wi * a.top_k);

  // Each wavefront stages the activation row of the pair it is computing in
  // its own slot of s_act (f bf16), one pair after another.
  const int slot = __builtin_amdgcn_readfirstlane(wi);  // uniform: scalar slot addresses
  const uint16_t* act_lds = reinterpret_cast<const uint16_t*>(s_act) + slot * a.f;
  uint32_t* act_lds32 = reinterpret_cast<uint32_t*>(s_act) + slot * (a.f / 2);
  float* xs_w = s_xs[slot];
  // Per-(group, quarter) activation sums of pair pi, groups [g0, g1).
  auto xs_sums = [&](int pi, int g0, int g1) {
    for (int i = 4 * g0 + lane; i < 4 * g1; i += 64) {
      const int g = i >> 2, q = i & 3;
      uint4 x[4];
#pragma unroll
      for (int k = 0; k < 4; ++k)
        x[k] = *reinterpret_cast<const uint4*>(act_lds + g * kGroup + 8 * q + 32 * k);
      xs_w[i] = lane_group_xsum(x);
    }
  };
  // Expert output of pair pi for this row block from its staged activation
  // row; `first` is its first batch of tiles (prefetched when has_first).
  auto pair_output = [&](int pi, DownBatch first, bool has_first) {
    const uint8_t* rec = a.slot_bank + (int64_t)s_ids[pi] * a.record_bytes;
    auto xload = [&](int, int k) {
      return *reinterpret_cast<const uint4*>(act_lds + k);
    };
    auto xsload = [&](int, int g) { return xs_w[g * 4 + (lane >> 4)]; };
    float acc[kTokChunk] = {0.f, 0.f, 0.f, 0.f};
    if (!has_first) down_load_batch(rec, a.d, a.f, rb, 0, first);
    down_apply_batch_xs(first, a.f, 0, xload, xsload, 1, acc);
    for (int g0 = kDownBatch; g0 < G; g0 += kDownBatch) {
      DownBatch bt;
      down_load_batch(rec, a.d, a.f, rb, g0, bt);
      down_apply_batch_xs(bt, a.f, g0, xload, xsload, 1, acc);
    }
    const float o = reduce_quarters(acc[0]);
    if (lane < 16) {
      o_lds[pi][lane] = o;
      a.pair_out[(int64_t)pi * a.d + 16 * rb + lane] = o;
    }
  };
  // Pair by pair as each activation row arrives (its first two pairs'
  // tiles are prefetched), so computing one pair overlaps the wait for the
  // next.
  bool act_late = false;
  auto stage = [&](int pi) {
    act_late |= wave_stage_act_row(sy, a, ep, pi, act_lds32);
    xs_sums(pi, 0, G);
  };
  if (p0 + wi < p1) {
    stage(p0 + wi);
    pair_output(p0 + wi, pre0, true);
  }
  if (p0 + wi + kGemvWaves < p1) {
    stage(p0 + wi + kGemvWaves);
    pair_output(p0 + wi + kGemvWaves, pre1, true);
  }
  for (int pi = p0 + wi + 2 * kGemvWaves; pi < p1; pi += kGemvWaves) {
    stage(pi);
    pair_output(pi, pre0, false);
  }
  if (lane == 0) s_late[1][wi] = act_late;
  __syncthreads();
  if (tid < 16) {
    const int n = tid;
    float acc = 0.f;
    for (int j = 0; j < a.top_k; ++j) acc = fmaf(s_w[p0 + j], o_lds[p0 + j][n], acc);
    const bool late_any =
        route_late | s_late[1][0] | s_late[1][1] | s_late[1][2] | s_late[1][3];
    a.y[(int64_t)tu * a.d + 16 * rb + n] = late_any ? 0x7fc0 : (uint16_t)f32_to_bf16_rne(acc);
  }

  if (unit == 0) {
    // The workspace's routing and grouping arrays, as the unfused path writes them.
    for (int j = tid; j < P; j += 256) {
      a.topk_ids[j] = s_ids[j];
      a.topk_w[j] = s_w[j];
    }
    block_group<256, false>(gsh, P, a.n_experts, s_ids, a.counts, a.offsets, a.sorted_pairs,
                            a.active, a.n_active, nullptr, a.pair_pos);
  }
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
    int per_cu = 0, per_cu_dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_fused_kernel<false>, 256,
                                                     0) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu_dev, decode_fused_kernel<true>, 256,
                                                     0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    cap[dev] = min(per_cu, per_cu_dev) * cus;
  }
  return cap[dev];
}

}  // namespace

bool decode_fused_plan(DecodeArgs& a) {
  if (a.tokens < 1 || a.tokens > kFusedMaxTokens || a.tokens * a.top_k > kFusedMaxPairs)
    return false;
  if ((int64_t)kGemvWaves * a.f * 2 > kFusedActLdsBytes) return false;  // a row per wavefront
  if ((int64_t)a.tokens * a.top_k * (a.f / 2) > kFusedActWords) return false;
  if ((int64_t)a.tokens * a.d * 2 > kFusedActLdsBytes) return false;  // staged token rows
  const int T = a.tokens;
  const int pairs_of_f = a.f / kTileRows;
  const int n_rb = a.d / kTileRows;
  a.n_router = a.logits_override ? 1 : (a.n_experts + 3) / 4;
  a.n_down = T * n_rb;
  const int cap = min(fused_capacity(), kFusedMaxBlocks);
  // The most gate/up items (fewest row-block pairs each) that fit.  Token t's
  // items are workers [t*It, (t+1)*It); its down units start at worker
  // D0 + t*n_rb, which must not come before (t+1)*It.
  for (int ppi = 1; ppi <= pairs_of_f; ppi *= 2) {
    const int chunks = (pairs_of_f + ppi - 1) / ppi;
    const int It = a.top_k * chunks;
    int down0 = It;
    for (int t = 1; t < T; ++t) down0 = max(down0, (t + 1) * It - t * n_rb);
    const int n_work = max(T * It, down0 + a.n_down);
    if (a.n_router + n_work <= cap) {
      a.pairs_per_item = ppi;
      a.n_gate = T * It;
      a.down0 = down0;
      a.n_work = n_work;
      return true;
    }
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
  if (a.epoch != 0u)
    launch(decode_fused_kernel<false>, grid, dim3(256), stream, a);
  else
    launch(decode_fused_kernel<true>, grid, dim3(256), stream, a);
  e = hipGetLastError();
  if (e == hipSuccess && a.epoch != 0u) prog.epoch = a.epoch;
  return e;
}

}  // namespace emoe
