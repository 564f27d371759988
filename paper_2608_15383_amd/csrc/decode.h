// Fused decode launch (decode.hip): arguments, the per-cache synchronization
// block and the planning rule.
#pragma once

#include "common.h"

namespace emoe {

constexpr int kFusedMaxTokens = 4;   // tokens per fused call (one top-k wavefront each)
constexpr int kFusedMaxPairs = 32;   // token-expert pairs per fused call
constexpr int kSyncLanes = 16;       // logit replicas
constexpr int kFusedActLdsBytes = 32768;  // LDS: the token rows (gate/up)
constexpr int kFusedActWords = kFusedMaxPairs * 2048;  // activation words handed over (d_ff <= 4096)
constexpr int kFusedMaxBlocks = 1024;  // workgroups per fused launch
constexpr int kFusedMaxD = 4096;       // d_model of a fused launch (DecodeSync::out)
constexpr int kFusedMaxDownUnits = 8;  // down row blocks per worker
constexpr int kFusedDownLag = 2;       // pairs between a gate/up item's pair and its down pair
constexpr int kFusedTailPairs = 3;     // ... and last pairs whose down the tail workers take (one-pair items)
constexpr uint32_t kDeviceEpoch0 = 0x80000000u;  // first epoch of captured launches

// Data the workgroups of one fused launch hand to each other, in device
// memory owned by the cache (zeroed at creation).  Every word carries the
// launch's epoch in its high half and the payload in the low half: a reader
// polls the data itself (one 64-bit store is seen whole or not at all), so no
// per-word reset is needed between launches.  A launch made directly takes its
// epoch from the host (1 .. kDeviceEpoch0 - 1, cycling; 0 is the zeroed
// memory's tag and is never used).  A launch captured into a graph would
// replay one argument forever, so it takes its epoch from `epoch` here
// (kDeviceEpoch0 .. 2^32 - 1, cycling): every workgroup reads it at its start,
// stores it in its own `arrived` word once it has used it, and router
// workgroup 0, when every word of the grid holds it, stores the next one.
// `timeouts` counts bounded waits that gave up.
struct DecodeSync {
  uint32_t timeouts;
  uint32_t pad0[15];
  // Replicated copies of the logits, [replica][token][expert].
  uint64_t logits[kSyncLanes][kFusedMaxTokens * EMOE_MAX_EXPERTS];
  // Activation rows in pair order: word w of pair pi holds act[pi][2w .. 2w+1]
  // (bf16, low column in the low 16 bits) at pi * d_ff / 2 + w.
  uint64_t act[kFusedActWords];
  // Expert outputs in pair order: word pi * d_model + n holds the fp32 bits of
  // output n of pair pi (written for every pair but the last of each token).
  uint64_t out[kFusedMaxPairs * kFusedMaxD];
  uint32_t epoch;  // tag of the next captured launch (kDeviceEpoch0 after creation)
  uint32_t pad1[15];
  // Word b: the epoch that workgroup b of the latest launch used.
  uint32_t arrived[kFusedMaxBlocks];
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
  // Filled by decode_fused_plan / launch_decode_fused.  Workgroup
  // n_router + j (worker j) runs gate/up item j (j < n_gate: pair j / chunks,
  // with chunks items per pair) and then down_r output row blocks of pair
  // j / chunks - down_lag (none past pair P - tail_pairs - 1); the tail
  // workers (n_gate <= j < n_work) take the last tail_pairs pairs, tail_r row
  // blocks each, pair by pair.
  int n_router, n_gate, n_work;
  int router_shift;               // log2 of the router items per expert group (0 or 1)
  int router_experts;             // experts per router item (1 or 4)
  int pairs_per_item;             // gate/up row-block pairs per gate item
  int down_r, tail_r;             // down row blocks per gate/up and per tail worker
  int down_lag;                   // pairs between a gate/up item's pair and its down pair
  int tail_pairs;                 // last pairs whose down row blocks the tail workers take
  int gw;                         // down input groups per wavefront (template argument)
  uint32_t epoch;                 // this launch's tag; 0: read it from DecodeSync
  // Bounded waits (tests force them to give up): polls before a wait gives
  // up, and a mask xor-ed into the tag the readers wait for (0: the launch's
  // own; anything else: a tag no writer uses, so every wait gives up).
  uint32_t spin_limit = 1u << 20;
  uint32_t tag_xor = 0;
};

// Host side: the epoch of the last direct launch on one cache.
struct DecodeProgress {
  uint32_t epoch = 0;
};

// Size the grid; false if the layer does not fit one co-resident fused launch.
bool decode_fused_plan(DecodeArgs& a);
// The same for `cap` co-resident workgroups (no device query).
bool decode_fused_plan_for(DecodeArgs& a, int cap);

// The output row blocks [rb0, rb0 + nu) of pair q that worker wk (workgroup
// n_router + wk) of a planned launch computes; nu = 0: none.
struct FusedDownWork {
  int q = -1, rb0 = 0, nu = 0;
};
__host__ __device__ FusedDownWork fused_down_work(const DecodeArgs& a, int wk);
// Launch a planned call on `stream` (no host synchronization): a direct
// launch takes the next epoch from `prog`, a launch being captured into a
// graph takes its epochs from device memory.
hipError_t launch_decode_fused(DecodeArgs& a, DecodeProgress& prog, hipStream_t stream);

}  // namespace emoe
