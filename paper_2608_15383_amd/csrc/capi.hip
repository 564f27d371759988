// Host runtime and C ABI of libexactmoe.so: argument checks, the workspace
// layout, the per-layer slot cache with LRU replacement and event-ordered
// slot reuse (Sec. 3.3), wave planning and the per-wave execution loop of
// Sec. 3.4, and the sequential per-expert comparison path.
#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "common.h"
#include "decode.h"

using namespace emoe;

namespace {
thread_local char g_last_error[512] = "";
}  // namespace

namespace emoe {
namespace {
thread_local LaunchEvents t_launch_events;
}
LaunchEvents& launch_events() { return t_launch_events; }

int32_t report_error(int32_t status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return status;
}
}  // namespace emoe

// ------------------------------------------------------------------ errors
namespace {

int32_t fail(int32_t status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return status;
}

int32_t hip_fail(hipError_t e, const char* what) {
  return fail(EMOE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define EMOE_HIP(call)                                  \
  do {                                                  \
    hipError_t e_ = (call);                             \
    if (e_ != hipSuccess) return hip_fail(e_, #call);   \
  } while (0)

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

// Optional per-thread kernel timing (emoe_profile_begin / emoe_profile_end).
struct Profiler {
  bool on = false;
  int max = 0;
  std::vector<hipEvent_t> start, stop;
  std::vector<int32_t> kind;
  int used = 0;
};
thread_local Profiler g_prof;

// Run one launcher; while profiling, its kernel records the next event pair at
// dispatch.  Launchers that launch nothing (empty inputs) record nothing.
hipError_t timed_launch(int32_t kind, hipStream_t stream, hipError_t (*fn)(void*), void* ctx) {
  (void)stream;
  Profiler& p = g_prof;
  LaunchEvents& le = launch_events();
  const bool rec = p.on && p.used < p.max;
  le = LaunchEvents();
  if (rec) {
    le.start = p.start[p.used];
    le.stop = p.stop[p.used];
  }
  hipError_t e = fn(ctx);
  const bool launched = le.used;
  le = LaunchEvents();
  if (e == hipSuccess && rec && launched) p.kind[p.used++] = kind;
  return e;
}

// EMOE_LAUNCH(kind, stream, expr): run the launcher expression `expr`, with a
// timing event pair around it while profiling is on; return on failure.
#define EMOE_LAUNCH(kind, stream, expr)                                              \
  do {                                                                               \
    auto fn_ = [&]() -> hipError_t { return (expr); };                               \
    hipError_t e_ = timed_launch((kind), (stream),                                   \
                                 [](void* c) { return (*static_cast<decltype(fn_)*>(c))(); }, \
                                 &fn_);                                              \
    if (e_ != hipSuccess) return hip_fail(e_, #expr);                                \
  } while (0)

}  // namespace

// ------------------------------------------------------------------ cache object
struct emoe_cache {
  emoe_dims dims;
  int32_t capacity = 0;
  int64_t record_bytes = 0;
  uint8_t* slot_bank = nullptr;
  const uint8_t* host_bank = nullptr;
  bool resident_all = false;
  std::vector<int32_t> slot_of;     // [E]
  std::vector<int32_t> expert_of;   // [C]
  std::vector<int64_t> stamp;       // [C]
  int64_t clock = 0;
  int device = -1;
  // Fills alternate between two copy streams: one stream leaves a gap between
  // consecutive record copies that the other fills (pinned H2D of 46 records
  // of 3.24 MB: about 45 GB/s on one stream, 56 GB/s on two).
  static constexpr int kCopyStreams = 2;
  hipStream_t copy_stream[kCopyStreams] = {};
  std::vector<hipEvent_t> release;           // [C] completion of the last wave using the slot
  hipEvent_t ready[kCopyStreams] = {};       // completion of each stream's last fills
  int32_t* counts_host = nullptr;   // pinned [E]: the batched expert-id transfer
  DecodeSync* sync = nullptr;       // device: hand-over data of the fused decode launches
  DecodeProgress prog;              // host: epoch of the last direct fused launch
  int32_t wave_delay_us = 0;        // test hook: spin before each wave's projections
  uint32_t decode_spin_limit = 1u << 20;  // test hook: polls before a fused-launch wait gives up
  uint32_t decode_tag_xor = 0;            // test hook: nonzero, the fused launch's waits never match
  bool overlap = false;             // waves of C/2 so fills overlap the previous wave
  void* scratch = nullptr;          // device address of this device's no-alloc workspace
};

// Workspace of emoe_moe_forward_noalloc: one fixed array per device, held
// until the process ends.  Host code never passes `scratch` itself (on the
// host it is only a stand-in for the symbol); it uses the device address that
// hipGetSymbolAddress returns for the current device, looked up once per
// device at set-up (emoe_cache_create) and kept in g_scratch_addr.
static __device__ __align__(256) uint8_t scratch[EMOE_NOALLOC_SCRATCH_BYTES];

namespace {

std::mutex g_scratch_mu;
void* g_scratch_addr[64] = {};

// Device address of this device's scratch array (dev must be current).
hipError_t scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return hipSuccess;
}

// Mark slot s empty: its record is no longer trusted, so no expert maps to it
// and it is the first victim of the next miss.
void vacate_slot(emoe_cache* c, int s) {
  const int old = c->expert_of[s];
  if (old >= 0 && c->slot_of[old] == s) c->slot_of[old] = -1;
  c->expert_of[s] = -1;
  c->stamp[s] = -1;
}

int32_t check_dims(const emoe_dims* d) {
  if (!d) return fail(EMOE_EINVAL, "dims is NULL");
  if (d->d_model <= 0 || d->d_ff <= 0 || d->d_model % EMOE_GROUP || d->d_ff % EMOE_GROUP)
    return fail(EMOE_ESHAPE, "d_model=%d and d_ff=%d must be positive multiples of %d",
                d->d_model, d->d_ff, EMOE_GROUP);
  if (d->n_experts < 1 || d->n_experts > EMOE_MAX_EXPERTS)
    return fail(EMOE_ESHAPE, "n_experts=%d outside [1, %d]", d->n_experts, EMOE_MAX_EXPERTS);
  if (d->top_k < 1 || d->top_k > d->n_experts)
    return fail(EMOE_ESHAPE, "top_k=%d outside [1, n_experts=%d]", d->top_k, d->n_experts);
  return EMOE_OK;
}

emoe_ws_layout make_layout(const emoe_dims& d, int32_t T) {
  emoe_ws_layout L{};
  const size_t E = d.n_experts, k = d.top_k, P = (size_t)T * k;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align_up(bytes);
    return at;
  };
  L.logits = take((size_t)T * E * 4);
  L.topk_ids = take(P * 4);
  L.topk_w = take(P * 4);
  L.counts = take(E * 4);
  L.offsets = take((E + 1) * 4);
  L.sorted_pairs = take(P * 4);
  L.active = take(E * 4);
  L.n_active = take(4);
  L.tile_offsets = take((E + 1) * 4);
  L.pair_pos = take(P * 4);
  L.act = take(P * (size_t)d.d_ff * 2);
  L.pair_out = take(P * (size_t)d.d_model * 4);
  L.act_bias = take(P * (size_t)(d.d_ff / EMOE_GROUP) * 4);
  L.chunk_counts = take((P + 63) / 64 * E * 4);
  L.tok_bias = take((size_t)T * (d.d_model / EMOE_GROUP) * 4);
  L.total = off;
  return L;
}

// Per-device scratch flag of the quantizer (allocated once per device).
std::mutex g_flag_mu;
int32_t* g_range_flag[64] = {};

int32_t range_flag_for_current_device(int32_t** out) {
  int dev = 0;
  EMOE_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return fail(EMOE_EINVAL, "device index %d unsupported", dev);
  std::lock_guard<std::mutex> lk(g_flag_mu);
  if (!g_range_flag[dev]) EMOE_HIP(hipMalloc(&g_range_flag[dev], 256));
  *out = g_range_flag[dev];
  return EMOE_OK;
}

// Test hook emoe_test_fail_copy_after: number of slot copies that still
// succeed before one fails (-1: none fails).  Process-wide.
std::atomic<int64_t> g_copies_before_failure{-1};

// True when the copy about to be enqueued must fail instead (consumes the hook).
bool take_injected_copy_failure() {
  int64_t left = g_copies_before_failure.load();
  while (left >= 0) {
    if (g_copies_before_failure.compare_exchange_weak(left, left - 1)) return left == 0;
  }
  return false;
}

void add_stats(emoe_stats* s, const emoe_stats& d) {
  if (!s) return;
  s->layer_calls += d.layer_calls;
  s->waves += d.waves;
  s->hits += d.hits;
  s->misses += d.misses;
  s->h2d_bytes += d.h2d_bytes;
  s->grouped_gemm_calls += d.grouped_gemm_calls;
  s->seq_expert_calls += d.seq_expert_calls;
  s->kernel_launches += d.kernel_launches;
}

// Test hook: one wavefront that spins for `ticks` of the constant-rate wall
// clock and exits.  Bounded twice: by the clock, and by a poll count that
// covers the delay even if the clock stood still (each poll sleeps 512
// shader clocks, at least 0.2 us).
__global__ void delay_kernel(uint64_t ticks, uint64_t max_polls) {
  const uint64_t t0 = wall_clock64();
  for (uint64_t it = 0; it < max_polls; ++it) {
    if (wall_clock64() - t0 >= ticks) break;
    __builtin_amdgcn_s_sleep(8);
  }
}

hipError_t launch_delay(int32_t us, hipStream_t stream) {
  int dev = 0, khz = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
  if (e != hipSuccess) return e;
  const uint64_t ticks = (uint64_t)us * (uint64_t)(khz > 0 ? khz : 100000) / 1000u;
  hipLaunchKernelGGL(delay_kernel, dim3(1), dim3(64), 0, stream, ticks, (uint64_t)us * 5u + 64u);
  return hipGetLastError();
}

}  // namespace

extern "C" {

const char* emoe_status_string(int32_t st) {
  switch (st) {
    case EMOE_OK: return "ok";
    case EMOE_EINVAL: return "invalid argument";
    case EMOE_ESHAPE: return "unsupported shape";
    case EMOE_ERANGE: return "scale out of FP16 range";
    case EMOE_ECAPACITY: return "capacity outside [top_k, n_experts]";
    case EMOE_EHIP: return "HIP runtime error";
    case EMOE_ESTATE: return "call not valid for this cache";
    default: return "unknown status";
  }
}

const char* emoe_last_error(void) { return g_last_error; }

int32_t emoe_check_dims(const emoe_dims* dims) { return check_dims(dims); }

size_t emoe_expert_record_bytes(const emoe_dims* dims) {
  if (check_dims(dims) != EMOE_OK) return 0;
  return (size_t)record_layout(dims->d_model, dims->d_ff).bytes;
}

int32_t emoe_workspace_layout(const emoe_dims* dims, int32_t max_tokens, emoe_ws_layout* out) {
  int32_t st = check_dims(dims);
  if (st) return st;
  if (max_tokens < 0 || !out) return fail(EMOE_EINVAL, "bad max_tokens or NULL output");
  *out = make_layout(*dims, max_tokens);
  return EMOE_OK;
}

size_t emoe_workspace_bytes(const emoe_dims* dims, int32_t max_tokens) {
  if (check_dims(dims) != EMOE_OK || max_tokens < 0) return 0;
  return make_layout(*dims, max_tokens).total;
}

// ------------------------------------------------------------------ quantization
int32_t emoe_quantize_experts(const emoe_dims* dims, int32_t n, const uint16_t* w_gate,
                              const uint16_t* w_up, const uint16_t* w_down, void* records,
                              hipStream_t stream) {
  int32_t st = check_dims(dims);
  if (st) return st;
  if (n < 0 || n > 65535) return fail(EMOE_EINVAL, "n=%d experts out of range", n);
  if (n == 0) return EMOE_OK;
  if (!w_gate || !w_up || !w_down || !records) return fail(EMOE_EINVAL, "NULL buffer");
  int32_t* flag = nullptr;
  if ((st = range_flag_for_current_device(&flag))) return st;
  EMOE_HIP(hipMemsetAsync(flag, 0, sizeof(int32_t), stream));
  EMOE_HIP(launch_quantize(dims->d_model, dims->d_ff, n, w_gate, w_up, w_down,
                           static_cast<uint8_t*>(records), flag, stream));
  int32_t host_flag = 0;
  EMOE_HIP(hipMemcpyAsync(&host_flag, flag, sizeof host_flag, hipMemcpyDeviceToHost, stream));
  EMOE_HIP(hipStreamSynchronize(stream));
  if (host_flag) return fail(EMOE_ERANGE, "a group scale max|W|/7 overflows FP16");
  return EMOE_OK;
}

int32_t emoe_unpack_expert(const emoe_dims* dims, const void* record, int8_t* q_gate,
                           uint16_t* s_gate, int8_t* q_up, uint16_t* s_up, int8_t* q_down,
                           uint16_t* s_down) {
  int32_t st = check_dims(dims);
  if (st) return st;
  if (!record) return fail(EMOE_EINVAL, "record is NULL");
  const int d = dims->d_model, f = dims->d_ff;
  const RecordLayout L = record_layout(d, f);
  const uint8_t* rec = static_cast<const uint8_t*>(record);
  // Decode one matrix (N x K codes at `codes`, fp16 scales at `sc`) into
  // row-major outputs; `row_of(n)` maps the stored row to the output row or -1.
  auto decode = [&](int N, int K, int64_t codes_off, int64_t sc_off, auto row_of, int8_t* q,
                    uint16_t* s) {
    const int G = K / kGroup;
    for (int rb = 0; rb < N / kTileRows; ++rb)
      for (int g = 0; g < G; ++g) {
        const uint8_t* tile = rec + codes_off + ((int64_t)rb * G + g) * kTileBytes;
        for (int l = 0; l < 64; ++l) {
          const int out_row = row_of(rb * kTileRows + (l & 15));
          if (out_row < 0 || !q) continue;
          for (int i = 0; i < 4; ++i) {
            uint32_t dw;
            std::memcpy(&dw, tile + 16 * l + 4 * i, 4);
            for (int r = 0; r < 8; ++r) {
              const int kk = g * kGroup + 32 * i + 8 * (l >> 4) + r;
              const uint32_t u = (dw >> (4 * (r >> 1) + 16 * (r & 1))) & 0xfu;
              q[(int64_t)out_row * K + kk] = (int8_t)((int)u - 8);
            }
          }
        }
      }
    if (s) {
      const uint16_t* sp = reinterpret_cast<const uint16_t*>(rec + sc_off);
      for (int n = 0; n < N; ++n) {
        const int out_row = row_of(n);
        if (out_row < 0) continue;
        for (int g = 0; g < G; ++g) s[(int64_t)out_row * G + g] = sp[scale_index(n, g, G)];
      }
    }
  };
  // W13 stored row n -> gate row (block parity 0) or up row (parity 1).
  auto gate_row = [](int n) { return ((n >> 4) & 1) ? -1 : ((n >> 5) << 4) + (n & 15); };
  auto up_row = [](int n) { return ((n >> 4) & 1) ? ((n >> 5) << 4) + (n & 15) : -1; };
  auto same_row = [](int n) { return n; };
  decode(2 * f, d, L.w13_codes, L.w13_scales, gate_row, q_gate, s_gate);
  decode(2 * f, d, L.w13_codes, L.w13_scales, up_row, q_up, s_up);
  decode(d, f, L.w2_codes, L.w2_scales, same_row, q_down, s_down);
  return EMOE_OK;
}

int32_t emoe_pack_expert(const emoe_dims* dims, const int8_t* q_gate, const uint16_t* s_gate,
                         const int8_t* q_up, const uint16_t* s_up, const int8_t* q_down,
                         const uint16_t* s_down, void* record) {
  int32_t st = check_dims(dims);
  if (st) return st;
  if (!q_gate || !s_gate || !q_up || !s_up || !q_down || !s_down || !record)
    return fail(EMOE_EINVAL, "NULL buffer");
  const int d = dims->d_model, f = dims->d_ff;
  const RecordLayout L = record_layout(d, f);
  uint8_t* rec = static_cast<uint8_t*>(record);
  auto encode = [&](int N, int K, int64_t codes_off, int64_t sc_off, auto src_of) -> int32_t {
    const int G = K / kGroup;
    for (int rb = 0; rb < N / kTileRows; ++rb)
      for (int g = 0; g < G; ++g) {
        uint8_t* tile = rec + codes_off + ((int64_t)rb * G + g) * kTileBytes;
        for (int l = 0; l < 64; ++l) {
          const int8_t* qrow;
          const uint16_t* srow;
          src_of(rb * kTileRows + (l & 15), qrow, srow);
          for (int i = 0; i < 4; ++i) {
            uint32_t dw = 0;
            for (int r = 0; r < 8; ++r) {
              const int v = qrow[g * kGroup + 32 * i + 8 * (l >> 4) + r];
              if (v < -8 || v > 7) return fail(EMOE_ERANGE, "code %d outside [-8, 7]", v);
              dw |= (uint32_t)(v + 8) << (4 * (r >> 1) + 16 * (r & 1));
            }
            std::memcpy(tile + 16 * l + 4 * i, &dw, 4);
          }
        }
      }
    uint16_t* sp = reinterpret_cast<uint16_t*>(rec + sc_off);
    for (int n = 0; n < N; ++n) {
      const int8_t* qrow;
      const uint16_t* srow;
      src_of(n, qrow, srow);
      for (int g = 0; g < G; ++g) sp[scale_index(n, g, G)] = srow[g];
    }
    return EMOE_OK;
  };
  const int Gd = d / kGroup, Gf = f / kGroup;
  auto w13_src = [&](int n, const int8_t*& qrow, const uint16_t*& srow) {
    const int row = ((n >> 5) << 4) + (n & 15);
    const bool up = (n >> 4) & 1;
    qrow = (up ? q_up : q_gate) + (int64_t)row * d;
    srow = (up ? s_up : s_gate) + (int64_t)row * Gd;
  };
  auto w2_src = [&](int n, const int8_t*& qrow, const uint16_t*& srow) {
    qrow = q_down + (int64_t)n * f;
    srow = s_down + (int64_t)n * Gf;
  };
  if ((st = encode(2 * f, d, L.w13_codes, L.w13_scales, w13_src))) return st;
  return encode(d, f, L.w2_codes, L.w2_scales, w2_src);
}

// ------------------------------------------------------------------ routing
int32_t emoe_route(const emoe_dims* dims, int32_t T, const uint16_t* h, const uint16_t* w_router,
                   const float* logits_override, int32_t renormalize, float* logits,
                   int32_t* topk_ids, float* topk_w, int32_t* counts, int32_t* offsets,
                   int32_t* sorted_pairs, int32_t* active, int32_t* n_active, hipStream_t stream) {
  int32_t st = check_dims(dims);
  if (st) return st;
  if (T < 0) return fail(EMOE_EINVAL, "tokens=%d < 0", T);
  if (!counts || !offsets || !active || !n_active) return fail(EMOE_EINVAL, "NULL output");
  if (T > 0) {
    if (!topk_ids || !topk_w || !sorted_pairs) return fail(EMOE_EINVAL, "NULL output");
    if (!logits_override && (!h || !w_router || !logits))
      return fail(EMOE_EINVAL, "h, w_router and logits are required without logits_override");
  }
  const int E = dims->n_experts, k = dims->top_k;
  const float* z = logits_override ? logits_override : logits;
  if (T > 0 && !logits_override)
    EMOE_LAUNCH(EMOE_K_ROUTER, stream,
                launch_router_logits(T, E, dims->d_model, h, w_router, logits, stream));
  if (T > 0)
    EMOE_LAUNCH(EMOE_K_TOPK, stream, launch_topk(T, E, k, renormalize, z, topk_ids, topk_w, stream));
  EMOE_LAUNCH(EMOE_K_GROUP, stream,
              launch_group(T * k, E, topk_ids, counts, offsets, sorted_pairs, active, n_active,
                           nullptr, nullptr, 1, stream));
  return EMOE_OK;
}

// ------------------------------------------------------------------ cache
int32_t emoe_cache_create(const emoe_dims* dims, int32_t capacity, void* slot_bank,
                          const void* host_bank, emoe_cache** out) {
  int32_t st = check_dims(dims);
  if (st) return st;
  if (!out) return fail(EMOE_EINVAL, "out is NULL");
  *out = nullptr;
  if (capacity < dims->top_k || capacity > dims->n_experts)
    return fail(EMOE_ECAPACITY, "capacity %d outside [top_k=%d, n_experts=%d]", capacity,
                dims->top_k, dims->n_experts);
  if (!slot_bank && host_bank) return fail(EMOE_EINVAL, "a host bank needs a slot bank");
  if (slot_bank && !host_bank && capacity != dims->n_experts)
    return fail(EMOE_EINVAL, "C < E needs a pinned host bank to fill slots from");
  if (host_bank) {
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, host_bank) != hipSuccess || attr.type != hipMemoryTypeHost) {
      (void)hipGetLastError();
      return fail(EMOE_EINVAL, "host_bank is not pinned host memory (use hipHostMalloc)");
    }
  }
  emoe_cache* c = new (std::nothrow) emoe_cache();
  if (!c) return fail(EMOE_EINVAL, "out of host memory");
  c->dims = *dims;
  c->capacity = capacity;
  c->record_bytes = record_layout(dims->d_model, dims->d_ff).bytes;
  c->slot_bank = static_cast<uint8_t*>(slot_bank);
  c->host_bank = static_cast<const uint8_t*>(host_bank);
  c->slot_of.assign(dims->n_experts, -1);
  c->expert_of.assign(capacity, -1);
  c->stamp.assign(capacity, -1);
  if (slot_bank) {
    hipError_t e = hipGetDevice(&c->device);
    if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void**>(&c->counts_host),
                                           sizeof(int32_t) * dims->n_experts, hipHostMallocDefault);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&c->sync), sizeof(DecodeSync));
    if (e == hipSuccess) e = hipMemset(c->sync, 0, sizeof(DecodeSync));
    const uint32_t first_epoch = kDeviceEpoch0;  // returns once the zeroing is done, too
    if (e == hipSuccess)
      e = hipMemcpy(&c->sync->epoch, &first_epoch, sizeof first_epoch, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = scratch_address(c->device, &c->scratch);
    if (e == hipSuccess && host_bank) {
      for (int j = 0; j < emoe_cache::kCopyStreams && e == hipSuccess; ++j) {
        e = hipStreamCreateWithFlags(&c->copy_stream[j], hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ready[j], hipEventDisableTiming);
      }
      c->release.assign(capacity, nullptr);
      for (int s = 0; s < capacity && e == hipSuccess; ++s)
        e = hipEventCreateWithFlags(&c->release[s], hipEventDisableTiming);
    }
    if (e != hipSuccess) {
      emoe_cache_destroy(c);
      return hip_fail(e, "cache resources");
    }
  }
  *out = c;
  return EMOE_OK;
}

int32_t emoe_cache_destroy(emoe_cache* c) {
  if (!c) return EMOE_OK;
  for (hipStream_t cs : c->copy_stream)
    if (cs) (void)hipStreamSynchronize(cs);
  for (hipEvent_t ev : c->release)
    if (ev) (void)hipEventDestroy(ev);
  for (int j = 0; j < emoe_cache::kCopyStreams; ++j) {
    if (c->ready[j]) (void)hipEventDestroy(c->ready[j]);
    if (c->copy_stream[j]) (void)hipStreamDestroy(c->copy_stream[j]);
  }
  if (c->counts_host) (void)hipHostFree(c->counts_host);
  if (c->sync) (void)hipFree(c->sync);
  delete c;
  return EMOE_OK;
}

int32_t emoe_cache_sync_timeouts(const emoe_cache* c, int64_t* timeouts) {
  if (!c || !timeouts) return fail(EMOE_EINVAL, "NULL argument");
  *timeouts = 0;
  if (!c->sync) return EMOE_OK;
  EMOE_HIP(hipDeviceSynchronize());
  uint32_t t = 0;
  EMOE_HIP(hipMemcpy(&t, &c->sync->timeouts, sizeof t, hipMemcpyDeviceToHost));
  *timeouts = t;
  return EMOE_OK;
}

int32_t emoe_cache_preload_all(emoe_cache* c, hipStream_t stream) {
  if (!c) return fail(EMOE_EINVAL, "cache is NULL");
  if (c->capacity != c->dims.n_experts)
    return fail(EMOE_ESTATE, "full residency needs capacity == n_experts");
  if (!c->slot_bank) return fail(EMOE_ESTATE, "no slot bank attached");
  if (c->host_bank)
    EMOE_HIP(hipMemcpyAsync(c->slot_bank, c->host_bank,
                            (size_t)c->record_bytes * c->capacity, hipMemcpyHostToDevice, stream));
  for (int e = 0; e < c->dims.n_experts; ++e) {
    c->slot_of[e] = e;
    c->expert_of[e] = e;
  }
  c->resident_all = true;
  return EMOE_OK;
}

int32_t emoe_cache_set_wave_overlap(emoe_cache* c, int32_t enable) {
  if (!c) return fail(EMOE_EINVAL, "cache is NULL");
  if (enable != 0 && enable != 1) return fail(EMOE_EINVAL, "enable=%d is not 0 or 1", enable);
  c->overlap = enable != 0;
  return EMOE_OK;
}

int32_t emoe_cache_state(const emoe_cache* c, int32_t* slot_of_expert, int32_t* expert_of_slot,
                         int64_t* stamp_of_slot) {
  if (!c) return fail(EMOE_EINVAL, "cache is NULL");
  if (slot_of_expert) std::copy(c->slot_of.begin(), c->slot_of.end(), slot_of_expert);
  if (expert_of_slot) std::copy(c->expert_of.begin(), c->expert_of.end(), expert_of_slot);
  if (stamp_of_slot) std::copy(c->stamp.begin(), c->stamp.end(), stamp_of_slot);
  return EMOE_OK;
}

int32_t emoe_plan_waves(const emoe_cache* c, const int32_t* counts, int32_t* wave_experts,
                        int32_t* wave_offsets, int32_t* n_waves) {
  if (!c || !counts || !wave_experts || !wave_offsets || !n_waves)
    return fail(EMOE_EINVAL, "NULL argument");
  const int E = c->dims.n_experts;
  int n = 0;
  for (int pass = 0; pass < 2; ++pass)  // resident first, then the rest
    for (int e = 0; e < E; ++e) {
      if (counts[e] < 0) return fail(EMOE_EINVAL, "counts[%d] < 0", e);
      if (counts[e] > 0 && ((c->slot_of[e] >= 0) == (pass == 0))) wave_experts[n++] = e;
    }
  // Overlap plan: a set that does not fit is cut into waves of C/2, whose
  // misses (under the LRU rule) never take the previous wave's slots.
  const int size = (c->overlap && n > c->capacity) ? std::max(1, c->capacity / 2) : c->capacity;
  int w = 0;
  for (int at = 0; at < n; at += size) wave_offsets[w++] = at;
  wave_offsets[w] = n;
  *n_waves = w;
  return EMOE_OK;
}

int32_t emoe_build_slot_map(emoe_cache* c, const int32_t* wave, int32_t n, int32_t* slot_map,
                            int32_t* fill_expert, int32_t* fill_slot, int32_t* n_fill,
                            emoe_stats* stats) {
  if (!c || (n > 0 && !wave) || !slot_map || !n_fill) return fail(EMOE_EINVAL, "NULL argument");
  const int E = c->dims.n_experts, C = c->capacity;
  if (n < 0 || n > C) return fail(EMOE_ECAPACITY, "wave of %d experts exceeds capacity %d", n, C);
  // Fixed-size scratch on the stack: the layer calls allocate nothing.
  char seen[EMOE_MAX_EXPERTS] = {};
  for (int i = 0; i < n; ++i) {
    if (wave[i] < 0 || wave[i] >= E) return fail(EMOE_EINVAL, "expert %d out of range", wave[i]);
    if (seen[wave[i]]++) return fail(EMOE_EINVAL, "expert %d repeated in a wave", wave[i]);
  }
  std::fill(slot_map, slot_map + E, -1);
  *n_fill = 0;
  if (c->resident_all) {
    for (int i = 0; i < n; ++i) slot_map[wave[i]] = wave[i];
    return EMOE_OK;
  }
  if (n > 0 && (!fill_expert || !fill_slot)) return fail(EMOE_EINVAL, "NULL fill list");
  emoe_stats d{};
  c->clock += 1;
  char prot[EMOE_MAX_EXPERTS] = {};
  for (int i = 0; i < n; ++i) {
    const int s = c->slot_of[wave[i]];
    if (s >= 0) {
      d.hits += 1;
      prot[s] = 1;
      c->stamp[s] = c->clock;
    }
  }
  // Misses in ascending expert id: `seen` marks the wave's experts.
  for (int e = 0; e < E; ++e) {
    if (!seen[e] || c->slot_of[e] >= 0) continue;
    int victim = -1;
    for (int s = 0; s < C; ++s) {
      if (prot[s]) continue;
      if (victim < 0 || c->stamp[s] < c->stamp[victim]) victim = s;
    }
    const int old = c->expert_of[victim];
    if (old >= 0) c->slot_of[old] = -1;
    c->expert_of[victim] = e;
    c->slot_of[e] = victim;
    c->stamp[victim] = c->clock;
    prot[victim] = 1;
    fill_expert[*n_fill] = e;
    fill_slot[*n_fill] = victim;
    *n_fill += 1;
    d.misses += 1;
    d.h2d_bytes += c->record_bytes;
  }
  for (int i = 0; i < n; ++i) slot_map[wave[i]] = c->slot_of[wave[i]];
  add_stats(stats, d);
  return EMOE_OK;
}

int32_t emoe_fill_slots(emoe_cache* c, const int32_t* fill_expert, const int32_t* fill_slot,
                        int32_t n_fill, hipStream_t stream) {
  if (!c) return fail(EMOE_EINVAL, "cache is NULL");
  if (n_fill == 0) return EMOE_OK;
  if (n_fill < 0 || !fill_expert || !fill_slot) return fail(EMOE_EINVAL, "bad fill list");
  if (!c->slot_bank || !c->host_bank || !c->copy_stream[0])
    return fail(EMOE_ESTATE, "cache has no slot bank / host bank");
  for (int i = 0; i < n_fill; ++i) {
    const int e = fill_expert[i], s = fill_slot[i];
    if (e < 0 || e >= c->dims.n_experts || s < 0 || s >= c->capacity)
      return fail(EMOE_EINVAL, "fill (%d -> %d) out of range", e, s);
  }
  hipError_t e_hip = hipSuccess;
  const char* what = "";
  for (int i = 0; i < n_fill && e_hip == hipSuccess; ++i) {
    const int e = fill_expert[i], s = fill_slot[i];
    hipStream_t cs = c->copy_stream[i % emoe_cache::kCopyStreams];
    e_hip = hipStreamWaitEvent(cs, c->release[s], 0);
    what = "hipStreamWaitEvent(copy stream, slot release)";
    if (e_hip == hipSuccess && take_injected_copy_failure()) {
      e_hip = hipErrorInvalidValue;
      what = "hipMemcpyAsync (failure injected by emoe_test_fail_copy_after)";
    }
    if (e_hip == hipSuccess) {
      e_hip = hipMemcpyAsync(c->slot_bank + (int64_t)s * c->record_bytes,
                             c->host_bank + (int64_t)e * c->record_bytes, c->record_bytes,
                             hipMemcpyHostToDevice, cs);
      what = "hipMemcpyAsync(slot <- host bank)";
    }
  }
  for (int j = 0; j < emoe_cache::kCopyStreams && j < n_fill && e_hip == hipSuccess; ++j) {
    e_hip = hipEventRecord(c->ready[j], c->copy_stream[j]);
    if (e_hip == hipSuccess) e_hip = hipStreamWaitEvent(stream, c->ready[j], 0);
    what = "hipEventRecord / hipStreamWaitEvent(fills ready)";
  }
  if (e_hip == hipSuccess) return EMOE_OK;
  // Some copies may have been enqueued and may (partly) have overwritten their
  // slots, and `stream` does not wait for them.  Let them finish, then mark
  // every listed slot empty, so that no later call takes a partly written
  // slot for a resident expert and no later fill races an earlier one.
  for (hipStream_t cs : c->copy_stream) (void)hipStreamSynchronize(cs);
  for (int i = 0; i < n_fill; ++i) vacate_slot(c, fill_slot[i]);
  return hip_fail(e_hip, what);
}

}  // extern "C"

// ------------------------------------------------------------------ forward
namespace {

// GEMV row chunks of a wave from the experts' row counts.
// GEMV row chunks of the wave's experts (those with fewer than mfma_rows rows).
void set_wave_chunks(WaveArg& wa, const int32_t* counts, int mfma_rows) {
  int32_t acc = 0;
  for (int i = 0; i < wa.n; ++i) {
    wa.chunk0[i] = acc;
    const int rows = counts[wa.expert[i]];
    acc += rows < mfma_rows ? (rows + kGemvRows - 1) / kGemvRows : 0;
  }
  wa.chunk0[wa.n] = acc;
}

// Slot contents and recency before a wave, kept to undo the wave's map
// update when its fills fail (fixed size: the layer calls allocate nothing).
struct CacheSnapshot {
  int32_t expert_of[EMOE_MAX_EXPERTS];
  int64_t stamp[EMOE_MAX_EXPERTS];
  int64_t clock;
  void take(const emoe_cache* c) {
    std::copy(c->expert_of.begin(), c->expert_of.end(), expert_of);
    std::copy(c->stamp.begin(), c->stamp.end(), stamp);
    clock = c->clock;
  }
  // A failed wave: slots in its fill list were vacated by emoe_fill_slots
  // (their records may be partly overwritten); every other slot gets back its
  // expert and stamp, and the clock its value, as if the wave never ran.
  void restore_except_filled(emoe_cache* c, const int32_t* fill_slot, int n_fill) const {
    char filled[EMOE_MAX_EXPERTS] = {};
    for (int i = 0; i < n_fill; ++i) filled[fill_slot[i]] = 1;
    std::fill(c->slot_of.begin(), c->slot_of.end(), -1);
    for (int s = 0; s < c->capacity; ++s) {
      if (filled[s]) {
        c->expert_of[s] = -1;
        c->stamp[s] = -1;
      } else {
        c->expert_of[s] = expert_of[s];
        c->stamp[s] = stamp[s];
      }
      if (c->expert_of[s] >= 0) c->slot_of[c->expert_of[s]] = s;
    }
    c->clock = clock;
  }
};

int32_t forward_impl(emoe_cache* c, int32_t T, const uint16_t* h, const uint16_t* w_router,
                     const float* logits_override, int32_t renormalize, int32_t path, uint16_t* y,
                     void* workspace, size_t ws_bytes, hipStream_t stream, emoe_stats* stats,
                     bool sequential) {
  if (!c) return fail(EMOE_EINVAL, "cache is NULL");
  if (!c->slot_bank) return fail(EMOE_ESTATE, "no slot bank attached");
  if (!c->resident_all && !c->host_bank)
    return fail(EMOE_ESTATE, "cache is neither fully resident nor backed by a host bank");
  const emoe_dims& D = c->dims;
  if (T < 0) return fail(EMOE_EINVAL, "tokens=%d < 0", T);
  if (path < EMOE_PATH_AUTO || path > EMOE_PATH_MIXED) return fail(EMOE_EINVAL, "bad path %d", path);
  emoe_stats ds{};
  ds.layer_calls = 1;
  if (T == 0) {
    add_stats(stats, ds);
    return EMOE_OK;
  }
  if (!h || !y || !workspace) return fail(EMOE_EINVAL, "NULL h, y or workspace");
  if (!w_router && !logits_override) return fail(EMOE_EINVAL, "need w_router or logits_override");
  const emoe_ws_layout L = make_layout(D, T);
  if (ws_bytes < L.total)
    return fail(EMOE_EINVAL, "workspace of %zu bytes < %zu needed", ws_bytes, L.total);
  const int E = D.n_experts, k = D.top_k, d = D.d_model, f = D.d_ff;
  const int P = T * k;
  // The MFMA kernels address activations with 32-bit buffer offsets.
  const bool mfma_fits = (int64_t)P * f * 2 <= INT32_MAX && (int64_t)T * d * 2 <= INT32_MAX &&
                         d / EMOE_GROUP <= kMfmaMaxGroups && f / EMOE_GROUP <= kMfmaMaxGroups &&
                         c->record_bytes <= INT32_MAX;
  if (path == EMOE_PATH_AUTO)
    path = (T > EMOE_GEMV_MAX_TOKENS && mfma_fits) ? EMOE_PATH_MFMA : EMOE_PATH_GEMV;
  if (path != EMOE_PATH_GEMV && !mfma_fits)
    return fail(EMOE_ESHAPE, "MFMA kernels: %d tokens exceed their 2 GiB activation addressing, "
                             "or d_model / d_ff exceed %d groups", T, kMfmaMaxGroups);
  // Experts with at least mfma_rows rows run on the MFMA kernels.
  const int mfma_rows = path == EMOE_PATH_MFMA    ? 1
                        : path == EMOE_PATH_MIXED ? EMOE_MIXED_MFMA_ROWS
                                                  : INT32_MAX;

  uint8_t* ws = static_cast<uint8_t*>(workspace);
  float* logits = reinterpret_cast<float*>(ws + L.logits);
  int32_t* ids = reinterpret_cast<int32_t*>(ws + L.topk_ids);
  float* wts = reinterpret_cast<float*>(ws + L.topk_w);
  int32_t* counts = reinterpret_cast<int32_t*>(ws + L.counts);
  int32_t* offsets = reinterpret_cast<int32_t*>(ws + L.offsets);
  int32_t* sorted = reinterpret_cast<int32_t*>(ws + L.sorted_pairs);
  int32_t* active = reinterpret_cast<int32_t*>(ws + L.active);
  int32_t* n_active = reinterpret_cast<int32_t*>(ws + L.n_active);
  int32_t* tiles = reinterpret_cast<int32_t*>(ws + L.tile_offsets);
  uint16_t* act = reinterpret_cast<uint16_t*>(ws + L.act);
  float* pair_out = reinterpret_cast<float*>(ws + L.pair_out);
  float* act_bias = reinterpret_cast<float*>(ws + L.act_bias);

  int32_t* pair_pos = reinterpret_cast<int32_t*>(ws + L.pair_pos);
  DecodeArgs a{};
  if (c->resident_all && !sequential && path == EMOE_PATH_GEMV && c->sync) {
    a.tokens = T;
    a.d = d;
    a.f = f;
    a.n_experts = E;
    a.top_k = k;
    a.renormalize = renormalize ? 1 : 0;
    a.h = h;
    a.w_router = w_router;
    a.logits_override = logits_override;
    a.slot_bank = c->slot_bank;
    a.record_bytes = c->record_bytes;
    a.logits = logits;
    a.topk_ids = ids;
    a.topk_w = wts;
    a.counts = counts;
    a.offsets = offsets;
    a.sorted_pairs = sorted;
    a.active = active;
    a.n_active = n_active;
    a.pair_pos = pair_pos;
    a.act = act;
    a.pair_out = pair_out;
    a.y = y;
    a.sync = c->sync;
    a.spin_limit = c->decode_spin_limit;
    a.tag_xor = c->decode_tag_xor;
  }
  if (a.sync && decode_fused_plan(a)) {
    // Few tokens, every expert resident: the whole layer in one launch.
    EMOE_LAUNCH(EMOE_K_DECODE_FUSED, stream, launch_decode_fused(a, c->prog, stream));
    ds.kernel_launches = 1;
    ds.waves = 1;
    ds.grouped_gemm_calls = 2;
    add_stats(stats, ds);
    return EMOE_OK;
  }

  // Route (Eq. 1) and group by expert.  On the MFMA path the router also sums
  // each token row's input groups (the accumulator starts of the gate/up MFMA
  // chains) when d is a multiple of 512; otherwise a separate pass forms them
  // below.
  const float* z = logits_override ? logits_override : logits;
  float* tok_bias = reinterpret_cast<float*>(ws + L.tok_bias);
  const bool uses_mfma = path != EMOE_PATH_GEMV;
  const bool fused_bias = uses_mfma && !logits_override && d % 512 == 0;
  if (!logits_override) {
    EMOE_LAUNCH(EMOE_K_ROUTER, stream,
                launch_router_logits(T, E, d, h, w_router, logits, stream,
                                     fused_bias ? tok_bias : nullptr));
    ds.kernel_launches += 1;
  }
  if (P > kGroupWideMinPairs) {
    // Wide grouping: per-chunk counts (with the top-k when top_k divides 64),
    // then the placement.
    int32_t* chunk_counts = reinterpret_cast<int32_t*>(ws + L.chunk_counts);
    if (topk_count_fits(k)) {
      EMOE_LAUNCH(EMOE_K_TOPK, stream,
                  launch_topk_count(T, E, k, renormalize, z, ids, wts, chunk_counts, stream));
      ds.kernel_launches += 1;
    } else {
      EMOE_LAUNCH(EMOE_K_TOPK, stream, launch_topk(T, E, k, renormalize, z, ids, wts, stream));
      EMOE_LAUNCH(EMOE_K_GROUP_COUNT, stream, launch_group_count(P, E, ids, chunk_counts, stream));
      ds.kernel_launches += 2;
    }
    EMOE_LAUNCH(EMOE_K_GROUP, stream,
                launch_group_place(P, E, ids, chunk_counts, counts, offsets, sorted, active,
                                   n_active, tiles, pair_pos, mfma_rows, stream));
    ds.kernel_launches += 1;
  } else {
    EMOE_LAUNCH(EMOE_K_TOPK, stream, launch_topk(T, E, k, renormalize, z, ids, wts, stream));
    EMOE_LAUNCH(EMOE_K_GROUP, stream,
                launch_group(P, E, ids, counts, offsets, sorted, active, n_active, tiles, pair_pos,
                             mfma_rows, stream));
    ds.kernel_launches += 2;
  }
  const GroupView gv{sorted, offsets, active, n_active, tiles, mfma_rows};
  if (uses_mfma && !fused_bias) {
    // Accumulator start of the gate/up MFMA chains, once per call.
    EMOE_LAUNCH(EMOE_K_ROW_BIAS, stream, launch_row_bias(T, d, h, tok_bias, stream));
    ds.kernel_launches += 1;
  }

  // One wave's projections: the GEMV kernels for the experts below mfma_rows
  // rows, the MFMA kernels for the others (on the mixed path both, gate/up
  // before down; fp32 pair outputs unless every expert is on MFMA).
  auto run_wave = [&](const WaveArg& wa) -> int32_t {
    const bool gemv = path != EMOE_PATH_MFMA;
    if (gemv) {
      EMOE_LAUNCH(EMOE_K_GATEUP_GEMV, stream,
                  launch_gateup_gemv(d, f, k, P, E, h, gv, wa, c->slot_bank, c->record_bytes, act, stream));
      ds.kernel_launches += 1;
    }
    if (uses_mfma) {
      EMOE_LAUNCH(EMOE_K_GATEUP_MFMA, stream,
                  launch_gateup_mfma(T, d, f, k, E, h, tok_bias, gv, wa, c->slot_bank, c->record_bytes,
                                     act, act_bias, stream));
      ds.kernel_launches += 1;
    }
    if (gemv) {
      EMOE_LAUNCH(EMOE_K_DOWN_GEMV, stream,
                  launch_down_gemv(d, f, k, P, E, act, gv, wa, c->slot_bank, c->record_bytes, pair_out, stream));
      ds.kernel_launches += 1;
    }
    if (uses_mfma) {
      EMOE_LAUNCH(EMOE_K_DOWN_MFMA, stream,
                  launch_down_mfma(T, d, f, k, E, act, act_bias, gv, wa, c->slot_bank, c->record_bytes,
                                   reinterpret_cast<uint16_t*>(pair_out), gemv ? pair_out : nullptr,
                                   stream));
      ds.kernel_launches += 1;
    }
    return EMOE_OK;
  };

  int32_t st;
  if (c->resident_all && !sequential) {
    // Full residency (Sec. 3.3): identity map, no expert-id transfer.
    WaveArg wa;
    wa.n = -1;
    if ((st = run_wave(wa))) return st;
    ds.waves = 1;
    ds.grouped_gemm_calls = 2;
  } else {
    // One batched expert-id transfer per layer (Sec. 1), then the waves of Sec. 3.4.
    EMOE_HIP(hipMemcpyAsync(c->counts_host, counts, sizeof(int32_t) * E, hipMemcpyDeviceToHost, stream));
    EMOE_HIP(hipStreamSynchronize(stream));
    int32_t wexp[EMOE_MAX_EXPERTS], woff[EMOE_MAX_EXPERTS + 1], smap[EMOE_MAX_EXPERTS];
    int32_t fexp[EMOE_MAX_EXPERTS], fslot[EMOE_MAX_EXPERTS];
    int32_t n_waves = 0;
    if ((st = emoe_plan_waves(c, c->counts_host, wexp, woff, &n_waves))) return st;
    CacheSnapshot snap;
    for (int w = 0; w < n_waves; ++w) {
      const int n = woff[w + 1] - woff[w];
      const int32_t* we = wexp + woff[w];
      snap.take(c);
      emoe_stats wstats{};
      int32_t n_fill = 0;
      if ((st = emoe_build_slot_map(c, we, n, smap, fexp, fslot, &n_fill, &wstats))) return st;
      if (!c->resident_all) {
        st = emoe_fill_slots(c, fexp, fslot, n_fill, stream);
        if (st) {
          snap.restore_except_filled(c, fslot, n_fill);
          return st;
        }
      }
      if (c->wave_delay_us > 0) {
        // Test hook: hold the wave's projections back (bounded spin on `stream`).
        EMOE_HIP(launch_delay(c->wave_delay_us, stream));
        ds.kernel_launches += 1;
      }
      ds.hits += wstats.hits;
      ds.misses += wstats.misses;
      ds.h2d_bytes += wstats.h2d_bytes;
      WaveArg wa;
      wa.n = n;
      for (int e = 0; e < E; ++e) wa.slot_of[e] = (int16_t)smap[e];
      for (int i = 0; i < n; ++i) wa.expert[i] = (int16_t)we[i];
      set_wave_chunks(wa, c->counts_host, mfma_rows);
      if (sequential) {
        for (int i = 0; i < n; ++i) {
          WaveArg one;
          one.n = 1;
          one.expert[0] = (int16_t)we[i];
          for (int e = 0; e < E; ++e) one.slot_of[e] = -1;
          one.slot_of[we[i]] = (int16_t)smap[we[i]];
          set_wave_chunks(one, c->counts_host, mfma_rows);
          if ((st = run_wave(one))) return st;
          ds.seq_expert_calls += 1;
        }
      } else {
        if ((st = run_wave(wa))) return st;
        ds.grouped_gemm_calls += 2;
      }
      ds.waves += 1;
      if (!c->resident_all)
        for (int i = 0; i < n; ++i) EMOE_HIP(hipEventRecord(c->release[smap[we[i]]], stream));
    }
  }
  EMOE_LAUNCH(EMOE_K_COMBINE, stream,
              launch_combine(T, d, k, wts, pair_out, path == EMOE_PATH_MFMA, y, stream));
  ds.kernel_launches += 1;
  add_stats(stats, ds);
  return EMOE_OK;
}

}  // namespace

extern "C" {

int32_t emoe_moe_forward(emoe_cache* cache, int32_t tokens, const uint16_t* h,
                         const uint16_t* w_router, const float* logits_override,
                         int32_t renormalize, int32_t path, uint16_t* y, void* workspace,
                         size_t workspace_bytes, hipStream_t stream, emoe_stats* stats) {
  return forward_impl(cache, tokens, h, w_router, logits_override, renormalize, path, y, workspace,
                      workspace_bytes, stream, stats, false);
}

int32_t emoe_moe_forward_sequential(emoe_cache* cache, int32_t tokens, const uint16_t* h,
                                    const uint16_t* w_router, const float* logits_override,
                                    int32_t renormalize, int32_t path, uint16_t* y,
                                    void* workspace, size_t workspace_bytes,
                                    hipStream_t stream, emoe_stats* stats) {
  return forward_impl(cache, tokens, h, w_router, logits_override, renormalize, path, y, workspace,
                      workspace_bytes, stream, stats, true);
}

int32_t emoe_moe_forward_noalloc(emoe_cache* cache, int32_t tokens, const uint16_t* h,
                                 const uint16_t* w_router, const float* logits_override,
                                 int32_t renormalize, int32_t path, uint16_t* y,
                                 hipStream_t stream, emoe_stats* stats) {
  if (!cache) return fail(EMOE_EINVAL, "cache is NULL");
  if (!cache->slot_bank || !cache->scratch) return fail(EMOE_ESTATE, "no slot bank attached");
  if (tokens < 0) return fail(EMOE_EINVAL, "tokens=%d < 0", tokens);
  const size_t need = make_layout(cache->dims, tokens).total;
  if (need > (size_t)EMOE_NOALLOC_SCRATCH_BYTES)
    return fail(EMOE_EINVAL,
                "%d tokens need %zu workspace bytes; the no-allocation call's scratch holds %zu "
                "(use emoe_moe_forward with a caller workspace)",
                tokens, need, (size_t)EMOE_NOALLOC_SCRATCH_BYTES);
  return forward_impl(cache, tokens, h, w_router, logits_override, renormalize, path, y,
                      cache->scratch, (size_t)EMOE_NOALLOC_SCRATCH_BYTES, stream, stats, false);
}

int32_t emoe_test_fail_copy_after(int64_t copies) {
  if (copies < -1) return fail(EMOE_EINVAL, "copies=%lld < -1", (long long)copies);
  g_copies_before_failure.store(copies);
  return EMOE_OK;
}

int32_t emoe_test_set_wave_delay(emoe_cache* c, int32_t microseconds) {
  if (!c) return fail(EMOE_EINVAL, "cache is NULL");
  if (microseconds < 0 || microseconds > 1000)
    return fail(EMOE_EINVAL, "wave delay %d us outside [0, 1000]", microseconds);
  c->wave_delay_us = microseconds;
  return EMOE_OK;
}

int32_t emoe_test_set_decode_waits(emoe_cache* c, int32_t spin_limit, int32_t unmatched) {
  if (!c) return fail(EMOE_EINVAL, "cache is NULL");
  if (spin_limit < 1 || spin_limit > (1 << 20))
    return fail(EMOE_EINVAL, "spin limit %d outside [1, 2^20]", spin_limit);
  if (unmatched != 0 && unmatched != 1) return fail(EMOE_EINVAL, "unmatched must be 0 or 1");
  c->decode_spin_limit = (uint32_t)spin_limit;
  c->decode_tag_xor = unmatched ? 0x40000000u : 0u;
  return EMOE_OK;
}

int32_t emoe_profile_begin(int32_t max_kernels) {
  if (max_kernels <= 0 || max_kernels > (1 << 20)) return fail(EMOE_EINVAL, "bad max_kernels");
  Profiler& p = g_prof;
  if (p.on) return fail(EMOE_ESTATE, "profiling already active on this thread");
  p.start.assign(max_kernels, nullptr);
  p.stop.assign(max_kernels, nullptr);
  p.kind.assign(max_kernels, -1);
  p.max = max_kernels;
  p.used = 0;
  for (int i = 0; i < max_kernels; ++i) {
    hipError_t e = hipEventCreate(&p.start[i]);
    if (e == hipSuccess) e = hipEventCreate(&p.stop[i]);
    if (e != hipSuccess) {
      for (hipEvent_t ev : p.start) if (ev) (void)hipEventDestroy(ev);
      for (hipEvent_t ev : p.stop) if (ev) (void)hipEventDestroy(ev);
      p = Profiler();
      return hip_fail(e, "hipEventCreate");
    }
  }
  p.on = true;
  return EMOE_OK;
}

int32_t emoe_profile_end(int32_t* kinds, float* ms, int32_t max_out, int32_t* n_out) {
  Profiler& p = g_prof;
  if (!p.on) return fail(EMOE_ESTATE, "profiling not active on this thread");
  int32_t st = EMOE_OK;
  const int n = p.used;
  for (int i = 0; i < n && st == EMOE_OK; ++i) {
    hipError_t e = hipEventSynchronize(p.stop[i]);
    float t = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, p.start[i], p.stop[i]);
    if (e != hipSuccess) {
      st = hip_fail(e, "kernel timing events");
      break;
    }
    if (i < max_out) {
      if (kinds) kinds[i] = p.kind[i];
      if (ms) ms[i] = t;
    }
  }
  if (n_out) *n_out = n;
  for (hipEvent_t ev : p.start) (void)hipEventDestroy(ev);
  for (hipEvent_t ev : p.stop) (void)hipEventDestroy(ev);
  p = Profiler();
  return st;
}

}  // extern "C"
