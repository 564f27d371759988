// Fused decode launch (decode.hip): arguments, the per-cache synchronization
// block, the host-side progress that sets each launch's counter targets, and
// the planning rule.
#pragma once

#include "common.h"

namespace emoe {

constexpr int kFusedMaxTokens = 4;   // tokens per fused call (one top-k wavefront each)
constexpr int kFusedMaxPairs = 32;   // token-expert pairs per fused call
constexpr int kSyncLanes = 16;       // spread counters, 64 B apart
constexpr int kFusedActLdsBytes = 32768;  // LDS staging of all pairs' activation rows

// Counters of the fused launches of one cache, in device memory owned by the
// cache (zeroed at creation).  They only grow (modulo 2^32); each launch waits
// for targets that the host derives from its running totals, so no reset is
// needed between launches.  `timeouts` counts bounded waits that gave up.
struct DecodeSync {
  uint32_t route_done[kSyncLanes][16]; // router workgroups finished (replicated)
  uint32_t gate_done[kSyncLanes][16];  // gate/up workgroups finished, spread by index
  uint32_t timeouts;
  uint32_t pad1[15];
  // Replicated copies of the logits, [replica][token][expert].
  float logits[kSyncLanes][kFusedMaxTokens * EMOE_MAX_EXPERTS];
};

// Host-side totals of the launches made so far on one cache.
struct DecodeProgress {
  uint32_t route_total = 0;
  uint32_t gate_total[kSyncLanes] = {};
};

struct DecodeArgs {
  int tokens, d, f, n_experts, top_k, renormalize;
  const uint16_t* h;
  const uint16_t* w_router;
  const float* logits_override;
  const uint8_t* slot_bank;  // expert e in slot e
  int64_t record_bytes;
  float* logits;
  int32_t* topk_ids;
  float* topk_w;
  int32_t* counts;
  int32_t* offsets;
  int32_t* sorted_pairs;
  int32_t* active;
  int32_t* n_active;
  int32_t* pair_pos;
  uint16_t* act;
  float* pair_out;
  uint16_t* y;
  DecodeSync* sync;
  // Filled by decode_fused_plan / launch_decode_fused.
  int n_router, n_gate, n_down;
  int pairs_per_item;             // gate/up row-block pairs per gate item
  uint32_t route_target;          // route_done value once this launch's router items finished
  uint32_t gate_target[kSyncLanes];
};

// Size the grid; false if the layer does not fit one co-resident fused launch.
bool decode_fused_plan(DecodeArgs& a);
// Set the targets from `prog`, launch, advance `prog` on success.
hipError_t launch_decode_fused(DecodeArgs& a, DecodeProgress& prog, hipStream_t stream);

}  // namespace emoe
