// Internal declarations shared by the HIP sources of libcavs.so (gfx950).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "cavs.h"

// One timed launch: events recorded on the context stream around it.
struct cavs_timed_launch {
  const char* name;
  int row0, rows;
  hipEvent_t start, stop;
};

struct cavs_ctx {
  int device = 0;
  hipStream_t stream = nullptr;
  int32_t* host_stage = nullptr;  // pinned, kHostStageInts entries (coherent, mapped)
  int32_t* host_stage_dev = nullptr;  // the same memory as the device sees it
  std::string err;
  bool timing = false;
  std::vector<cavs_timed_launch> timed;   // pending records
  std::vector<hipEvent_t> event_pool;     // reusable events
  hipEvent_t stage_ready = nullptr;       // the schedule's host stage has arrived
  int32_t* dev_err = nullptr;             // pinned, coherent, mapped: set by kernels whose
  int32_t* dev_err_dev = nullptr;         // bounded waits gave up (device view of dev_err)
  void* sched_scratch = nullptr;          // this device's static scheduling scratch
  hipStream_t side = nullptr;             // the two-stream ablation's second stream and its
  hipEvent_t fork_ev = nullptr;           // fork / join events (created on first use)
  hipEvent_t join_ev = nullptr;
  // The XCD loop's owner array that the last forward left in its workspace:
  // valid for the matching backward (same workspace, schedule and suffix).
  struct {
    const void* ws = nullptr;
    const int* parent_pos = nullptr;
    int base = -1, V = -1;
  } xcd_owner;
};

namespace cavs {

constexpr int kHostStageInts = 4096 + 32;
constexpr int kWave = 64;

typedef float v4f __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// error plumbing
// ---------------------------------------------------------------------------
cavs_status fail(cavs_ctx* ctx, cavs_status st, const char* fmt, ...);
// After the context's stream has been synchronised: CAVS_OK, or the error a
// kernel recorded in ctx->dev_err since the last check (then cleared).
cavs_status device_errors(cavs_ctx* ctx);
// Clears `bytes` (a multiple of 4) at p with a kernel on stream s.
hipError_t zero_async(void* p, size_t bytes, hipStream_t s);

#define CAVS_HIP_CHECK(ctx, call)                                              \
  do {                                                                         \
    hipError_t e_ = (call);                                                    \
    if (e_ != hipSuccess)                                                      \
      return ::cavs::fail((ctx), CAVS_ERR_HIP, "%s failed: %s (%s:%d)", #call, \
                          hipGetErrorString(e_), __FILE__, __LINE__);          \
  } while (0)

#define CAVS_LAUNCH_CHECK(ctx) CAVS_HIP_CHECK(ctx, hipGetLastError())

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int cdiv(long a, long b) { return (int)((a + b - 1) / b); }

// ---------------------------------------------------------------------------
// device math.  The gate nonlinearities use the hardware base-2 exponential
// and reciprocal (v_exp_f32, v_rcp_f32, each within about one ulp):
//   sigmoid(a) = 1 / (1 + 2^(-a log2 e)), which saturates to 0 or 1 through
//   the exponential's overflow / underflow;
//   tanh(x) = sign(x) (1 - 2 / (1 + 2^(2|x| log2 e))) for |x| >= 0.4 (the
//   subtraction from 1 loses at most a couple of ulp there), and the odd
//   Taylor series x - x^3/3 + 2x^5/15 - 17x^7/315 + 62x^9/2835
//   - 1382x^11/155925 + 21844x^13/6081075 below (truncation under 1e-8
//   relative at 0.4).
// ---------------------------------------------------------------------------
constexpr float kLog2e = 1.44269504088896340736f;

__device__ __forceinline__ float sigmoidf_(float a) {
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-kLog2e * a));
}

__device__ __forceinline__ float tanh_(float x) {
  const float ax = fabsf(x);
  const float e = __builtin_amdgcn_exp2f(2.f * kLog2e * ax);
  const float big = 1.f - 2.f * __builtin_amdgcn_rcpf(1.f + e);
  const float x2 = x * x;
  float q = 21844.f / 6081075.f;
  q = fmaf(q, x2, -1382.f / 155925.f);
  q = fmaf(q, x2, 62.f / 2835.f);
  q = fmaf(q, x2, -17.f / 315.f);
  q = fmaf(q, x2, 2.f / 15.f);
  q = fmaf(q, x2, -1.f / 3.f);
  const float small = fmaf(q * x2, x, x);
  return ax < 0.4f ? small : copysignf(big, x);
}

__device__ __forceinline__ v4f mfma_f32_16x16x4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// deterministic wave-wide sum (butterfly over all 64 lanes)
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// ---------------------------------------------------------------------------
// optional per-launch timing (cavs_timing_enable): the API entry points make
// their context current; launchers wrap each kernel in a TimedScope.
// ---------------------------------------------------------------------------
extern thread_local cavs_ctx* t_active_ctx;

struct ActiveCtx {
  explicit ActiveCtx(cavs_ctx* c) { t_active_ctx = c; }
  ~ActiveCtx() { t_active_ctx = nullptr; }
};

hipEvent_t timing_event(cavs_ctx* c);

// A timed launch hands its two events to the dispatch itself
// (hipExtLaunchKernelGGL), so they carry the kernel's own start and end and
// leave out the queue gap before it.  Cooperative launches have no such form:
// those record the events on the stream around the launch (bracket = true).
struct TimedScope {
  cavs_ctx* c;
  cavs_timed_launch rec;
  bool bracket;
  TimedScope(const char* name, hipStream_t s, int row0 = 0, int rows = 0, bool bracket_ = false)
      : c(t_active_ctx), bracket(bracket_) {
    if (!c || !c->timing) {
      c = nullptr;
      return;
    }
    rec.name = name;
    rec.row0 = row0;
    rec.rows = rows;
    rec.start = timing_event(c);
    rec.stop = timing_event(c);
    stream = s;
    if (bracket) (void)hipEventRecord(rec.start, s);
  }
  hipEvent_t start_ev() const { return c && !bracket ? rec.start : nullptr; }
  hipEvent_t stop_ev() const { return c && !bracket ? rec.stop : nullptr; }
  ~TimedScope() {
    if (!c) return;
    if (bracket) (void)hipEventRecord(rec.stop, stream);
    c->timed.push_back(rec);
  }
  hipStream_t stream = nullptr;
};

}  // namespace cavs

// Launch on `stream`; with timing enabled the dispatch records its own
// start and end events.
#define CAVS_LAUNCH(name, kernel, grid, block, shmem, stream, ...)            \
  do {                                                                      \
    ::cavs::TimedScope ts_(name, stream);                                   \
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ts_.start_ev(), \
                          ts_.stop_ev(), 0, __VA_ARGS__);                   \
  } while (0)

// Same, recording the level-major rows [row0, row0 + rows) the launch covers.
#define CAVS_LAUNCH_ROWS(name, row0, rows, kernel, grid, block, shmem, stream, ...) \
  do {                                                                            \
    ::cavs::TimedScope ts_(name, stream, row0, rows);                             \
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ts_.start_ev(),     \
                          ts_.stop_ev(), 0, __VA_ARGS__);                         \
  } while (0)

// ---------------------------------------------------------------------------
// host entry points implemented in the individual sources
// ---------------------------------------------------------------------------
namespace cavs {

struct SchedWs;

// schedule.hip
size_t schedule_ws_bytes(int32_t V, int32_t N, int32_t n_x);
cavs_status schedule_run(cavs_ctx* ctx, const cavs_graphs* g, cavs_sched* s, void* ws,
                         size_t ws_bytes);
// Address of the static scheduling scratch (CAVS_SCHEDULE_STATIC_BYTES) on
// `device`, which must be current; taken once per device.  *out = NULL for
// device ids past the supported range.
cavs_status static_sched_scratch(cavs_ctx* ctx, int device, void** out);

}  // namespace cavs
