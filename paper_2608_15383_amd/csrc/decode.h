// Fused decode launch (decode.hip): arguments, the per-cache synchronization
// block, the host-side progress that sets each launch's counter targets, and
// the planning rule.
#pragma once

#include "common.h"

namespace emoe {

constexpr int kFusedMaxTokens = 4;   // tokens per fused call (one top-k wavefront each)
constexpr int kFusedMaxPairs = 32;   // token-expert pairs per fused call
constexpr int kSyncLanes = 16;       // spread counters, 64 B apart
constexpr int kGateCounters = 32;    // gate/up completion counters, a fixed subset per pair
static_assert(kFusedMaxPairs <= kGateCounters, "every pair owns at least one counter");
constexpr int kFusedActLdsBytes = 32768;  // LDS staging of all pairs' activation rows

// Counters of the fused launches of one cache, in device memory owned by the
// cache (zeroed at creation).  They only grow (modulo 2^32); each launch waits
// for targets that the host derives from its running totals, so no reset is
// needed between launches.  `timeouts` counts bounded waits that gave up.
struct DecodeSync {
  uint32_t gate_done[kGateCounters][16];  // gate/up workgroups finished; pair pi owns
                                          // counters pi*cpp .. pi*cpp+cpp-1
  uint32_t timeouts;
  uint32_t pad1[15];
  // Replicated copies of the logits, [replica][token][expert], each tagged
  // with the launch's epoch in the high word: a reader polls the values
  // themselves (one 64-bit store is seen whole or not at all).
  uint64_t logits[kSyncLanes][kFusedMaxTokens * EMOE_MAX_EXPERTS];
};

// Host-side totals of the launches made so far on one cache.
struct DecodeProgress {
  uint32_t epoch = 0;  // of the last launch; the memory starts zeroed (epoch 0 never used)
  uint32_t gate_total[kGateCounters] = {};
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
  int items_per_pair;             // gate items of one pair
  int counters_per_pair;          // cpp: gate/up counters owned by each pair
  uint32_t epoch;                 // this launch's logit tag
  uint32_t gate_target[kGateCounters];
};

// Size the grid; false if the layer does not fit one co-resident fused launch.
bool decode_fused_plan(DecodeArgs& a);
// Set the targets from `prog`, launch, advance `prog` on success.
hipError_t launch_decode_fused(DecodeArgs& a, DecodeProgress& prog, hipStream_t stream);

}  // namespace emoe
