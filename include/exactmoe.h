/*
 * exactmoe.h -- C ABI of the MI355X (gfx950) fused W4A16 routed-expert layer.
 *
 * The layer follows "Every Expert Counts: ExactMoE for Memory-Efficient W4A16
 * Inference":
 *   Sec. 3.1, Eq. 1  router logits z = W_r h and top-k selection S_t;
 *   Sec. 3.1, Eq. 2  y_t = sum_{e in S_t} p_{t,e} W_d,e [phi(W_g,e h) * W_u,e h];
 *   Sec. 3.2, Eq. 3  symmetric group-128 INT4 weights with FP16 scales;
 *   Sec. 3.3         per-layer slot cache (global-to-slot map, LRU, events);
 *   Sec. 3.4         grouped execution in waves of at most C experts.
 *
 * Conventions for every call:
 *   - Return value is an emoe_status (0 = success, < 0 = error).  Nothing is
 *     enqueued when an argument check fails; emoe_last_error() then holds a
 *     message for the calling thread.  HIP failures map to EMOE_EHIP.
 *   - "device" pointers are HIP device memory, "host" pointers are ordinary
 *     host memory, "pinned" pointers are page-locked host memory
 *     (hipHostMalloc).  The caller owns every buffer passed in; the library
 *     owns only the opaque emoe_cache object and what it creates.
 *   - bf16 values travel as uint16_t bit patterns.  Matrices are row-major in
 *     nn.Linear order: a projection W[N][K] maps K inputs to N outputs.
 *   - All device work is enqueued on the stream argument (0 = the null
 *     stream) and is asynchronous unless the call says otherwise.
 */
#ifndef EXACTMOE_H
#define EXACTMOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum emoe_status {
  EMOE_OK = 0,
  EMOE_EINVAL = -1,     /* null pointer, bad flag, short buffer, non-pinned host bank */
  EMOE_ESHAPE = -2,     /* d_model or d_ff not a multiple of 128, bad top_k / expert count */
  EMOE_ERANGE = -3,     /* a group scale max|W|/7 overflows FP16 */
  EMOE_ECAPACITY = -4,  /* capacity C outside [top_k, n_experts] */
  EMOE_EHIP = -5,       /* a HIP runtime call failed */
  EMOE_ESTATE = -6      /* call not valid for this cache (e.g. no slot bank attached) */
};

/* Quantization group along the input dimension (Sec. 3.2). */
#define EMOE_GROUP 128
/* Largest supported expert count per layer. */
#define EMOE_MAX_EXPERTS 256

/* Execution path of the expert projections (every path computes Eq. 2-3 on
 * the same packed records; they differ in summation order and in the
 * precision of the stored pair outputs):
 *   GEMV:  VALU weight-streaming kernels for every expert (with full
 *          residency and few tokens, the fused decode launch);
 *   MFMA:  grouped bf16 MFMA GEMM for every expert, pair outputs rounded to bf16;
 *   MIXED: per expert, by its own row count in the call: experts with at
 *          least EMOE_MIXED_MFMA_ROWS token rows on the MFMA kernels, the
 *          others on the GEMV kernels, pair outputs fp32.
 * AUTO takes GEMV for at most EMOE_GEMV_MAX_TOKENS tokens and MFMA above (on
 * MI355X the MFMA kernels are faster from 5 tokens on, also with one or two
 * rows per expert).  What decides the arithmetic of a pair depends only on
 * the call's (tokens, top_k, n_experts) and on its own expert's row count,
 * never on the cache or the wave partition, so every wave of a call uses the
 * same arithmetic.  The MFMA kernels need tokens*d_model*2 and
 * tokens*top_k*d_ff*2 below 2^31 bytes and d_model, d_ff <= 8192 (AUTO takes
 * the GEMV otherwise; an explicit MFMA or MIXED request fails with
 * EMOE_ESHAPE). */
enum emoe_path { EMOE_PATH_AUTO = 0, EMOE_PATH_GEMV = 1, EMOE_PATH_MFMA = 2, EMOE_PATH_MIXED = 3 };
#define EMOE_GEMV_MAX_TOKENS 4
#define EMOE_MIXED_MFMA_ROWS 16

typedef struct emoe_dims {
  int32_t d_model;    /* hidden size d; multiple of 128 */
  int32_t d_ff;       /* expert intermediate size f; multiple of 128 */
  int32_t n_experts;  /* E, 1..EMOE_MAX_EXPERTS */
  int32_t top_k;      /* k, 1..E */
} emoe_dims;

/* Counters of Sec. 4.2 / Sec. 5.3 (cache events, transferred bytes, grouped
 * GEMM calls, sequential expert calls).  Calls that take an emoe_stats*
 * ADD to it; pass NULL to skip. */
typedef struct emoe_stats {
  int64_t layer_calls;         /* moe_forward / moe_forward_sequential calls */
  int64_t waves;               /* waves executed */
  int64_t hits;                /* wave experts found resident (C < E only) */
  int64_t misses;              /* wave experts copied from the host bank */
  int64_t h2d_bytes;           /* bytes copied host bank -> slot bank */
  int64_t grouped_gemm_calls;  /* grouped projection launches (2 per wave) */
  int64_t seq_expert_calls;    /* per-expert launches of the sequential path */
  int64_t kernel_launches;     /* every kernel launch made by the call */
} emoe_stats;

/* Byte offsets of the per-call arrays inside a forward workspace. */
typedef struct emoe_ws_layout {
  size_t logits;        /* f32   [T][E]   router logits z (Eq. 1) */
  size_t topk_ids;      /* i32   [T][k]   selected experts, rank order */
  size_t topk_w;        /* f32   [T][k]   mixture weights p */
  size_t counts;        /* i32   [E]      pairs per expert */
  size_t offsets;       /* i32   [E+1]    exclusive prefix sum of counts */
  size_t sorted_pairs;  /* i32   [T*k]    pair ids pi = t*k+j grouped by expert */
  size_t active;        /* i32   [E]      active experts, ascending */
  size_t n_active;      /* i32   [1]      number of active experts */
  size_t tile_offsets;  /* i32   [E+1]    MFMA row-tile prefix sum (experts on the MFMA kernels) */
  size_t pair_pos;      /* i32   [T*k]    grouped position of each pair id */
  size_t act;           /* bf16  [T*k][d_ff]    phi(g)*u per pair, grouped order */
  size_t pair_out;      /* expert output per pair id, [T*k][d_model]: f32 on the GEMV and
                           mixed paths, bf16 (in the first half of the field) on the MFMA path */
  size_t act_bias;      /* f32   [d_ff/128][T*k]    -136 * group sums of act, by grouped
                                                      position (MFMA kernels) */
  size_t chunk_counts;  /* i32   [ceil(T*k/64)][E]  pairs per expert in each 64-pair chunk
                                                      (grouping of large calls) */
  size_t tok_bias;      /* f32   [T][d_model/128]   -136 * group sums of each token row of h
                                                      (MFMA kernels) */
  size_t total;         /* bytes needed */
} emoe_ws_layout;

typedef struct emoe_cache emoe_cache; /* opaque; owned by the library */

/* ---------------------------------------------------------------- basics */
const char* emoe_status_string(int32_t status);
/* Message of the last failing call on this thread ("" if none). */
const char* emoe_last_error(void);
/* EMOE_OK if the shape is supported, else EMOE_ESHAPE / EMOE_EINVAL. */
int32_t emoe_check_dims(const emoe_dims* dims);

/* Bytes of one packed expert record: 3*f*d/2 code bytes + 3*f*d/64 scale
 * bytes, i.e. Eq. 4's 4/8 + 16/(128*8) bytes per weight with no padding
 * (3,244,032 B at d = 2048, f = 1024).  0 for unsupported dims. */
size_t emoe_expert_record_bytes(const emoe_dims* dims);

/* Workspace of emoe_moe_forward for up to max_tokens tokens. */
int32_t emoe_workspace_layout(const emoe_dims* dims, int32_t max_tokens, emoe_ws_layout* out);
size_t emoe_workspace_bytes(const emoe_dims* dims, int32_t max_tokens);

/* ---------------------------------------------------------------- offline conversion */
/* Sec. 3.2, Eq. 3: quantize n experts and pack them into records.
 *   w_gate, w_up: device bf16 [n][d_ff][d_model];  w_down: device bf16 [n][d_model][d_ff].
 *   records: device, n * emoe_expert_record_bytes bytes, written in expert order.
 * Per (row, 128-wide input group): s = fp32(max|W|)/7 (IEEE divide),
 * q = clip(round_half_even(W/s), -8, 7) from the fp32 s, stored scale =
 * fp16(s) (round to nearest even); an all-zero group, or one whose FP16
 * scale underflows to zero, stores s = 0 and q = 0.
 * Synchronizes `stream` to report EMOE_ERANGE when a scale overflows FP16
 * (the records are then incomplete). */
int32_t emoe_quantize_experts(const emoe_dims* dims, int32_t n,
                              const uint16_t* w_gate, const uint16_t* w_up,
                              const uint16_t* w_down, void* records, hipStream_t stream);

/* Host-side decode of one packed record (host memory) into plain arrays:
 *   q_gate, q_up int8 [d_ff][d_model], s_gate, s_up fp16 bits [d_ff][d_model/128];
 *   q_down int8 [d_model][d_ff], s_down fp16 bits [d_model][d_ff/128].
 * Any output pointer may be NULL to skip it. */
int32_t emoe_unpack_expert(const emoe_dims* dims, const void* record,
                           int8_t* q_gate, uint16_t* s_gate, int8_t* q_up, uint16_t* s_up,
                           int8_t* q_down, uint16_t* s_down);
/* Inverse of emoe_unpack_expert (host memory).  Codes must lie in [-8, 7]. */
int32_t emoe_pack_expert(const emoe_dims* dims, const int8_t* q_gate, const uint16_t* s_gate,
                         const int8_t* q_up, const uint16_t* s_up, const int8_t* q_down,
                         const uint16_t* s_down, void* record);

/* ---------------------------------------------------------------- routing and grouping */
/* Sec. 3.1, Eq. 1 and the grouping of Fig. 1, on the device:
 *   z[t][e] = fp32( sum_i h[t][i] * w_router[e][i] ) with an fp64 sum
 *     (or z = logits_override, device f32 [T][E], when non-NULL);
 *   topk_ids[t][j]: the k largest logits, rank j ordered by logit descending,
 *     ties to the lower expert id;
 *   topk_w[t][j]: softmax weights of the selected experts; renormalize != 0
 *     divides by the sum over the selected experts, 0 by the sum over all E;
 *   counts[e], offsets[E+1] (exclusive scan), sorted_pairs[T*k] (pair ids
 *     pi = t*k+j stably sorted by expert), active[<=E] (ascending experts with
 *     counts > 0) and n_active[1].
 * h: device bf16 [T][d_model]; w_router: device bf16 [E][d_model] (may be
 * NULL when logits_override is given); logits: device f32 [T][E] output (may
 * be NULL with an override).  Logits must not be NaN.  T may be 0. */
int32_t emoe_route(const emoe_dims* dims, int32_t tokens, const uint16_t* h,
                   const uint16_t* w_router, const float* logits_override, int32_t renormalize,
                   float* logits, int32_t* topk_ids, float* topk_w, int32_t* counts,
                   int32_t* offsets, int32_t* sorted_pairs, int32_t* active, int32_t* n_active,
                   hipStream_t stream);

/* ---------------------------------------------------------------- slot cache (Sec. 3.3) */
/* Create the per-layer cache with C = capacity slots, top_k <= C <= E.
 *   slot_bank: device, C * record_bytes (caller-owned), or NULL;
 *   host_bank: pinned, E * record_bytes holding this layer's records in
 *              expert order (caller-owned), or NULL.
 * With both NULL the cache only plans (emoe_plan_waves / emoe_build_slot_map).
 * With a slot bank and C = E, emoe_cache_preload_all makes every expert
 * resident (its record already in slot e, or copied from the host bank).
 * With a slot bank and C < E a host bank is required; the cache creates two
 * copy streams (default priority) and one completion event per slot. */
int32_t emoe_cache_create(const emoe_dims* dims, int32_t capacity, void* slot_bank,
                          const void* host_bank, emoe_cache** out);
/* Waits for the cache's copy streams and frees what the cache allocated
 * (events, streams, the hand-over block of the fused decode launch).  Device
 * work that uses the cache, including replays of graphs captured from its
 * layer calls, must have finished and must not be enqueued again. */
int32_t emoe_cache_destroy(emoe_cache* cache);
/* C = E only: identity map, no replacement and no hit accounting afterwards.
 * Copies the host bank into the slot bank on `stream` when a host bank is
 * attached; otherwise the slot bank must already hold expert e in slot e. */
int32_t emoe_cache_preload_all(emoe_cache* cache, hipStream_t stream);
/* Snapshot: slot_of_expert[E] (-1 absent), expert_of_slot[C] (-1 empty),
 * stamp_of_slot[C] (-1 never used).  Any pointer may be NULL. */
int32_t emoe_cache_state(const emoe_cache* cache, int32_t* slot_of_expert,
                         int32_t* expert_of_slot, int64_t* stamp_of_slot);

/* Number of bounded device-side waits of the fused decode launch that gave
 * up (0 in correct operation; a nonzero value means results of some call
 * are invalid).  Blocking: reads device memory after the device is idle. */
int32_t emoe_cache_sync_timeouts(const emoe_cache* cache, int64_t* timeouts);

/* Copy/compute overlap across waves (Sec. 3.3 lets a slot be refilled once
 * its preceding computation has finished).  enable = 1: when a call's active
 * set does not fit in the C slots, its waves hold at most max(1, C/2)
 * experts.  Under the LRU rule the previous wave's slots carry the newest
 * stamps, so every miss of a wave then takes a slot the previous wave does
 * not use, and its copy (ordered only by that slot's completion event)
 * proceeds while the previous wave computes.  Sets that fit stay one wave.
 * Default 0: waves of up to C.  Results are bit-identical either way. */
int32_t emoe_cache_set_wave_overlap(emoe_cache* cache, int32_t enable);

/* Sec. 3.4: split the active set into waves of at most C experts.
 * counts: host [E].  Order: experts resident now (ascending id), then the
 * others (ascending id), cut into chunks of C (of max(1, C/2) under
 * emoe_cache_set_wave_overlap when they do not fit at once).  Outputs (host):
 * wave_experts[<=E], wave_offsets[<=E+1] (wave w = wave_experts[off[w]..off[w+1])),
 * n_waves.  Does not change the cache. */
int32_t emoe_plan_waves(const emoe_cache* cache, const int32_t* counts,
                        int32_t* wave_experts, int32_t* wave_offsets, int32_t* n_waves);

/* Sec. 3.3 / Sec. 3.4 steps 1-2: resolve one wave (n distinct experts, n <= C).
 * Resident experts are hits and are protected; each missing expert, in
 * ascending id order, takes the unprotected slot with the smallest
 * (stamp, slot index) -- empty slots first -- evicting its occupant.  Every
 * slot the wave uses is stamped with a clock that ticks once per wave.
 * Outputs (host): slot_map[E] (-1 = inactive sentinel), fill_expert[n],
 * fill_slot[n], n_fill.  Updates the cache and adds hits/misses/h2d_bytes. */
int32_t emoe_build_slot_map(emoe_cache* cache, const int32_t* wave_experts, int32_t n,
                            int32_t* slot_map, int32_t* fill_expert, int32_t* fill_slot,
                            int32_t* n_fill, emoe_stats* stats);

/* Host-bank slot fill (Sec. 3.3): copy each listed record from the pinned host
 * bank to its slot with hipMemcpyAsync, alternating between the cache's two
 * copy streams, each copy first waiting for the slot's completion event (the
 * end of the last wave that computed on the slot), so a slot is never
 * overwritten before its preceding computation finishes; `stream` is then
 * made to wait for the copies.  No host synchronization on success.
 * On a HIP failure (EMOE_EHIP) the call waits for the copies it did enqueue
 * and marks every listed slot empty (no expert maps to it, stamp -1), since
 * its record can no longer be trusted; nothing has been made to wait on
 * `stream`. */
int32_t emoe_fill_slots(emoe_cache* cache, const int32_t* fill_expert, const int32_t* fill_slot,
                        int32_t n_fill, hipStream_t stream);

/* ---------------------------------------------------------------- the layer */
/* Sec. 3.1 Eq. 1-2 executed as in Sec. 3.4: route and group, then for each
 * wave resolve/fill its slots, run one grouped gate/up+SwiGLU launch and one
 * grouped down launch over the whole token matrix, and record slot completion
 * events; finally add the k weighted expert outputs of every token in rank
 * order (weights are never renormalized per wave).
 *   h: device bf16 [T][d_model];  y: device bf16 [T][d_model];
 *   w_router: device bf16 [E][d_model] (NULL allowed with logits_override);
 *   workspace: device, >= emoe_workspace_bytes(dims, T) bytes;
 *   path: an emoe_path value.
 * With a fully resident cache (C = E after preload) the call never blocks the
 * host.  Otherwise it copies counts[E] to the host once (one batched expert-id
 * transfer) and synchronizes `stream` to plan the waves.  If a wave's fill
 * fails the call returns EMOE_EHIP without writing y: the slots of that
 * wave's fill list are left empty (see emoe_fill_slots) and every other slot
 * keeps the expert, stamp and clock it had before the wave, so the next call
 * refills what it needs and computes on correct records.  Waves enqueued
 * before the failing one still complete on `stream`.
 * With full residency, the GEMV path, at most 4 tokens (and 32 pairs),
 * d_ff <= 2048, d_model <= 4096 and tokens*d_model <= 16384 the whole layer
 * runs as one fused kernel launch with the same arithmetic (and
 * bit-identical results).  Calls
 * on one cache must not overlap in time (use one stream, or order the
 * streams): the cache holds the words that launch's workgroups hand over.
 * With full residency the call may be captured into a HIP graph: a captured
 * fused launch numbers its hand-over words from device memory, so every
 * replay is distinct, and replays and direct calls on one cache may be mixed
 * in any order.  Without full residency the call synchronizes `stream` and
 * cannot be captured. */
int32_t emoe_moe_forward(emoe_cache* cache, int32_t tokens, const uint16_t* h,
                         const uint16_t* w_router, const float* logits_override,
                         int32_t renormalize, int32_t path, uint16_t* y, void* workspace,
                         size_t workspace_bytes, hipStream_t stream, emoe_stats* stats);

/* Sequential W4 reference path (Sec. 3.4, Sec. 5.3): same routing, cache
 * handling and arithmetic, but one gate/up and one down launch per active
 * expert instead of per wave.  Output is bit-identical to emoe_moe_forward
 * with the same path. */
int32_t emoe_moe_forward_sequential(emoe_cache* cache, int32_t tokens, const uint16_t* h,
                                    const uint16_t* w_router, const float* logits_override,
                                    int32_t renormalize, int32_t path, uint16_t* y,
                                    void* workspace, size_t workspace_bytes,
                                    hipStream_t stream, emoe_stats* stats);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * layer call as emoe_moe_forward, with the workspace taken from a fixed
 * device array inside the library instead of a caller buffer.  The call
 * allocates nothing (no hipMalloc, hipFree or other allocating routine, no
 * host heap).  The array holds EMOE_NOALLOC_SCRATCH_BYTES on every GPU the
 * library runs on, until the process ends; a call whose
 * emoe_workspace_bytes(dims, tokens) exceeds it fails with EMOE_EINVAL before
 * anything is enqueued (about 400 tokens at d_model 2048, d_ff 1024, 64
 * experts, top-8).  Nothing in the array needs to start at zero: every call
 * writes each part it reads.  All calls on one GPU share that GPU's array and
 * it keeps the last call's contents, so calls that overlap in time on one GPU
 * (any cache, any stream) race; order them.  The cache must have a slot bank
 * (its creation looks up the array's device address).  Results equal
 * emoe_moe_forward's bit for bit. */
#define EMOE_NOALLOC_SCRATCH_BYTES (32u << 20)
int32_t emoe_moe_forward_noalloc(emoe_cache* cache, int32_t tokens, const uint16_t* h,
                                 const uint16_t* w_router, const float* logits_override,
                                 int32_t renormalize, int32_t path, uint16_t* y,
                                 hipStream_t stream, emoe_stats* stats);

/* ---------------------------------------------------------------- test hooks */
/* Failure injection for tests of the fill error path (Sec. 3.3 slot reuse):
 * after `copies` more slot copies have been enqueued by emoe_fill_slots (in
 * any cache, process-wide), the next one fails on the host with
 * hipErrorInvalidValue before it is enqueued; -1 disarms.  Nothing faults on
 * the device. */
int32_t emoe_test_fail_copy_after(int64_t copies);
/* Race-window widening for tests of event-ordered slot reuse (Sec. 3.3):
 * before each wave's projections, the layer calls on this cache enqueue a
 * kernel on `stream` that spins for `microseconds` (0..1000; 0 = off) and
 * exits, so a fill that did not wait for the slot's completion event would
 * overwrite records still being read.  Off by default. */
int32_t emoe_test_set_wave_delay(emoe_cache* cache, int32_t microseconds);
/* Failure forcing for tests of the fused decode launch's bounded waits (the
 * hand-over of logits, activation rows and expert outputs between its
 * workgroups): a wait gives up after `spin_limit` polls (1 .. 2^20; 2^20 is
 * the default), and with `unmatched` = 1 the readers wait for a tag that no
 * writer uses, so every wait gives up.  A workgroup whose wait gave up writes
 * NaN outputs and counts the timeout (emoe_cache_sync_timeouts); every
 * workgroup still exits.  (2^20, 0) restores the normal launch. */
int32_t emoe_test_set_decode_waits(emoe_cache* cache, int32_t spin_limit, int32_t unmatched);
/* Host-only inspection of the fused decode launch (no GPU call), for tests of
 * its work assignment: the plan of a `tokens`-token call with `capacity`
 * co-resident workgroups into plan[9] = {router workgroups, gate/up workers,
 * workers, row-block pairs per gate/up item, down row blocks per gate/up
 * worker, per tail worker, down lag (pairs), tail pairs, down input groups
 * per wavefront}, and for workers 0 .. min(workers, max_workers) - 1 (worker
 * w is workgroup routers + w) the down work work[3w .. 3w+2] = {pair, first
 * row block, row blocks} (pair -1 / 0 row blocks: none).  Gate/up worker w
 * computes the gate/up item w of pair w / c, with c = ceil(d_ff / 16 / row-block
 * pairs per item) items per pair; every wait of a worker is for workgroups of
 * lower index.  EMOE_ESHAPE when
 * the call does not fit one fused launch, EMOE_EINVAL for NULL pointers or a
 * capacity below 1. */
int32_t emoe_debug_fused_plan(const emoe_dims* dims, int32_t tokens, int32_t capacity,
                              int32_t* plan, int32_t* work, int32_t max_workers);

/* ---------------------------------------------------------------- kernel timing */
/* Kernels launched by the layer calls, as reported by emoe_profile_end. */
enum emoe_kernel {
  EMOE_K_ROUTER = 0, EMOE_K_TOPK = 1, EMOE_K_GROUP = 2, EMOE_K_GATEUP_GEMV = 3,
  EMOE_K_DOWN_GEMV = 4, EMOE_K_GATEUP_MFMA = 5, EMOE_K_DOWN_MFMA = 6, EMOE_K_COMBINE = 7,
  EMOE_K_DECODE_FUSED = 8, EMOE_K_ROW_BIAS = 9, EMOE_K_GROUP_COUNT = 10
};
/* Start recording a HIP event pair around each kernel that emoe_route,
 * emoe_moe_forward and emoe_moe_forward_sequential launch from this thread,
 * on the stream the kernel is launched on, for up to max_kernels launches.
 * Creates the events (host call, not for use under graph capture). */
int32_t emoe_profile_begin(int32_t max_kernels);
/* Stop recording, wait for the recorded events and return, in launch order,
 * each kernel's kind (emoe_kernel) and duration in milliseconds; n_out =
 * number of kernels recorded (at most max_out are written).  Frees the events. */
int32_t emoe_profile_end(int32_t* kinds, float* ms, int32_t max_out, int32_t* n_out);

#ifdef __cplusplus
}
#endif
#endif /* EXACTMOE_H */
