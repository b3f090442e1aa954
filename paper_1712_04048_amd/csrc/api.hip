// C ABI of libcavs.so: context management, workspace layout and the
// forward / backward drivers (Algorithm 1: tasks in order for F, popped in
// reverse for dF; Algorithm 2: level-major dynamic tensors).
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>

#include "kernels.h"

namespace cavs {

thread_local cavs_ctx* t_active_ctx = nullptr;

hipEvent_t timing_event(cavs_ctx* c) {
  if (!c->event_pool.empty()) {
    hipEvent_t e = c->event_pool.back();
    c->event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  (void)hipEventCreate(&e);
  return e;
}

cavs_status fail(cavs_ctx* ctx, cavs_status st, const char* fmt, ...) {
  if (ctx) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    ctx->err = buf;
  }
  return st;
}

// Zero fill by a kernel rather than hipMemsetAsync, so that a caller may
// capture the calls into a HIP graph (memset nodes in captured graphs have
// given wrong results on replay on this platform).
__global__ void k_zero_words(uint32_t* p, long long n) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0u;
}

hipError_t zero_async(void* p, size_t bytes, hipStream_t s) {
  const long long n = (long long)(bytes / 4);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_zero_words, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                     (uint32_t*)p, n);
  return hipGetLastError();
}

cavs_status device_errors(cavs_ctx* ctx) {
  if (!ctx->dev_err || !ctx->dev_err[0]) return CAVS_OK;
  ctx->dev_err[0] = 0;
  return fail(ctx, CAVS_ERR_HIP,
              "a persistent or XCD-local level loop's grid barrier gave up waiting in an "
              "earlier call on "
              "this context: that call's states and gradients are invalid");
}

namespace {

// Workspace of forward + backward, all level-major (row = position).  In
// inference only the states, the pull projection, the transposed weights and
// the loss terms are kept: the saved gates and every gradient buffer take no
// space.
struct WsLayout {
  size_t P, UT, WxT, zrow, Hs, Cs, Gs, dZ, lossv, dHL, dHp, dCp, dA, dAb, part, bpart, bar, total;
  size_t part_floats;
  size_t gHt, gDt, gEh, gEc, gdAx, gpart;   // generic engine
  size_t WsT, dHLx;
  size_t gpart_floats;
  size_t pack, pack_elems;                  // bf16 lazy products: packed operands
  size_t Ub, UTb;                           // bf16 copies of U and U^T
  size_t xcd;                               // the XCD-local level loop's words and owners
};

bool lm_head(const cavs_params* p) { return p->loss == CAVS_LOSS_CE && p->C > kSmallHeadC; }

// bf16 values of the largest packed lazy product of the fused Tree-LSTM
// path (rows: the A columns padded to the product tile, then the B columns;
// each row the contraction length padded to the pack segment)
size_t bf_pack_elems(const cavs_params* p, const cavs_sched* s) {
  if (p->prec != CAVS_BF16 || p->cell != CAVS_TREE_LSTM || s->V <= 0) return 0;
  const size_t H = (size_t)p->H, D = (size_t)p->D;
  const size_t MI = s->T > 1 ? (size_t)(s->V - s->level_offsets_host[1]) : 0;
  auto qp = [](size_t q) { return (q + kPackSeg - 1) / kPackSeg * kPackSeg; };
  auto mp = [](size_t m) { return (m + kPackTile - 1) / kPackTile * kPackTile; };
  size_t e = (mp(H) + 4 * H) * qp(MI);                              // dU_iou
  if (p->N == 2) e = std::max(e, (mp(H) + H) * qp(2 * MI));         // dU_f
  if (D > 0) e = std::max(e, (mp(D) + 4 * H) * qp((size_t)s->n_pull));  // dW_x
  return e;
}

bool env_on(const char* name) {
  const char* e = getenv(name);
  return e && e[0] && e[0] != '0';
}

// Graph inputs and vertices with more than two child slots run the generic
// engine (generic.hip); CAVS_GENERIC=1 sends trees there too.
bool generic_mode(const cavs_params* p, const cavs_sched* s) {
  return s->dag || p->N > 2 || env_on("CAVS_GENERIC");
}

WsLayout ws_layout(const cavs_params* p, const cavs_sched* s, bool train) {
  WsLayout L{};
  const bool gen = p->cell == CAVS_TREE_LSTM && generic_mode(p, s);
  const size_t tr = train ? 1 : 0;
  const size_t V = (size_t)(s->V > 0 ? s->V : 1), H = (size_t)p->H;
  const bool lstm = p->cell == CAVS_TREE_LSTM;
  const size_t GW = lstm ? (size_t)(3 + p->N) * H : H;
  const size_t C = p->loss == CAVS_LOSS_CE ? (size_t)(p->C + 3) / 4 * 4 : 0;
  const bool lm = lm_head(p);
  size_t o = 0;
  auto take = [&](size_t floats) {
    size_t r = o;
    o = align_up(o + floats * sizeof(float), 256);
    return r;
  };
  L.P = take(lstm ? V * 4 * H : 0);
  L.UT = take(lstm ? 4 * H * H : (size_t)p->N * H * H);
  L.WxT = take(lstm ? 4 * H * (size_t)p->D : 0);
  L.zrow = take(H);
  L.Hs = take(V * H);
  L.Cs = take(lstm ? V * H : 0);
  L.Gs = take((tr || gen) ? (lstm ? V * GW : 0) : 0);   // the generic forward stages in it
  L.dZ = take((tr || lm) ? V * (C > 0 ? C : 1) : 0);   // the LM head's logits in inference
  L.lossv = take(V);
  L.dHL = take(tr * V * H);
  L.dHp = take(tr * (lstm ? V * H : 0));
  L.dCp = take(tr * (lstm ? V * H : 0));
  L.dA = take(tr * V * GW);
  L.part_floats = tr * lazy_part_floats(s->V, p->D, p->H, p->N, p->C);
  L.part = take(3 * L.part_floats);   // dU_iou, dU_f and dW_x split-K sums side by side
  L.bpart = take(tr * bias_part_floats(p->H, (p->loss == CAVS_LOSS_CE && !lm) ? p->C : 0));
  L.bar = take(256);
  L.WsT = take(lm ? C * H : 0);
  L.dHLx = take(tr * V * H);
  L.pack_elems = (tr && !gen) ? bf_pack_elems(p, s) : 0;
  L.pack = take((L.pack_elems + 1) / 2);
  L.xcd = take(lstm && !gen ? xcd_ws_bytes(s->V) / 4 + 1 : 0);
  const bool ubf = lstm && !gen && p->prec == CAVS_BF16;
  L.Ub = take(ubf ? 2 * H * H : 0);    // 4 H^2 bf16 values each
  L.UTb = take(ubf ? 2 * H * H : 0);
  L.dAb = take(ubf && tr ? V * GW / 2 : 0);   // V GW bf16 values
  if (lm && !gen) {
    L.gpart_floats = tr * gen_part_floats(p->D, p->H, (int)C);
    L.gpart = take(L.gpart_floats);
  }
  if (gen) {
    const size_t N = (size_t)p->N;
    L.gHt = take(V * H);
    L.gDt = take(tr * V * H);
    L.gEh = take(tr * V * N * H);
    L.gEc = take(tr * V * N * H);
    L.gdAx = take(tr * V * 4 * H);
    L.gpart_floats = tr * gen_part_floats(p->D, p->H, (int)C);
    L.gpart = take(L.gpart_floats);
  }
  L.total = o;
  return L;
}

cavs_status check_args(cavs_ctx* ctx, const cavs_params* p, const cavs_sched* s,
                       const cavs_inputs* in) {
  if (!ctx) return CAVS_ERR_ARG;
  if (!p || !s || !in) return fail(ctx, CAVS_ERR_ARG, "null params / sched / inputs");
  if (p->cell != CAVS_TREE_LSTM && p->cell != CAVS_TREE_FC)
    return fail(ctx, CAVS_ERR_ARG, "unknown cell %d", p->cell);
  if (p->loss != CAVS_LOSS_CE && p->loss != CAVS_LOSS_L2 && p->loss != CAVS_LOSS_NONE)
    return fail(ctx, CAVS_ERR_ARG, "unknown loss %d", p->loss);
  if (p->prec != CAVS_FP32 && p->prec != CAVS_BF16)
    return fail(ctx, CAVS_ERR_ARG, "unknown precision %d", p->prec);
  if (p->H <= 0 || p->D < 0 || p->N <= 0) return fail(ctx, CAVS_ERR_ARG, "bad D/H/N");
  if (p->N != s->N) return fail(ctx, CAVS_ERR_ARG, "params N=%d != schedule N=%d", p->N, s->N);
  if (p->N > kMaxSlots)
    return fail(ctx, CAVS_ERR_UNSUPPORTED, "N=%d child slots (max %d)", p->N, kMaxSlots);
  if (generic_mode(p, s)) {
    if (p->cell != CAVS_TREE_LSTM)
      return fail(ctx, CAVS_ERR_UNSUPPORTED,
                  "graph inputs and more than two child slots are built for the Tree-LSTM only");
    if (p->prec != CAVS_FP32)
      return fail(ctx, CAVS_ERR_UNSUPPORTED,
                  "graph inputs and more than two child slots run in fp32 only");
    if (s->dag && s->V > 0 && (!s->in_offsets || !s->in_edges))
      return fail(ctx, CAVS_ERR_ARG, "graph inputs need the schedule's in_offsets / in_edges");
  }
  if (p->H % 64 != 0) return fail(ctx, CAVS_ERR_UNSUPPORTED, "H=%d not a multiple of 64", p->H);
  if (p->prec == CAVS_BF16 && p->cell != CAVS_TREE_LSTM)
    return fail(ctx, CAVS_ERR_UNSUPPORTED, "bf16 products are built for the Tree-LSTM only");
  if (s->V < 0 || s->T < 0 || (s->V > 0 && s->T <= 0))
    return fail(ctx, CAVS_ERR_ARG, "schedule not built");
  if (s->V > 0 && (!s->child_pos || !s->parent_pos || !s->pull_pos || !s->push_pos ||
                   !s->order || !s->pull_list || !s->level_offsets_host))
    return fail(ctx, CAVS_ERR_ARG, "schedule arrays missing");
  if (!p->U || !p->b) return fail(ctx, CAVS_ERR_ARG, "U and b are required");
  if (p->loss == CAVS_LOSS_CE) {
    if (p->C <= 0) return fail(ctx, CAVS_ERR_ARG, "C=%d classes", p->C);
    if (p->C > kSmallHeadC && p->C % 4 != 0)
      return fail(ctx, CAVS_ERR_UNSUPPORTED, "C=%d: more than %d classes must be a multiple of 4",
                  p->C, kSmallHeadC);
    if (s->n_push != p->C) return fail(ctx, CAVS_ERR_ARG, "schedule n_push != C");
    if (!p->Ws || !p->bs) return fail(ctx, CAVS_ERR_ARG, "Ws and bs are required for CE");
  } else if (p->loss == CAVS_LOSS_L2) {
    if (s->n_push != in->n_y) return fail(ctx, CAVS_ERR_ARG, "schedule n_push != n_y");
    if (s->n_labelled > 0 && !in->Y) return fail(ctx, CAVS_ERR_ARG, "Y is required for L2");
  }
  if (s->n_pull > 0 && !in->X) return fail(ctx, CAVS_ERR_ARG, "X is required");
  if (p->cell == CAVS_TREE_LSTM) {
    if (p->D % 4 != 0) return fail(ctx, CAVS_ERR_UNSUPPORTED, "D=%d not a multiple of 4", p->D);
    if (s->n_pull > 0 && !p->Wx) return fail(ctx, CAVS_ERR_ARG, "Wx is required");
  } else {
    if (p->D != p->H) return fail(ctx, CAVS_ERR_ARG, "Tree-FC needs D == H");
    if (s->n_leaf_noinput != 0 || s->n_inner_input != 0)
      return fail(ctx, CAVS_ERR_ARG, "Tree-FC: a vertex must pull an input iff it is a leaf");
  }
  return CAVS_OK;
}

// Ablation of lazy batching (CAVS_EAGER_DW=1; Tree-LSTM only): the recurrent
// weight gradients dU are formed level by level, as each task's dA is known,
// and summed into dU in reverse task order, instead of as one product over
// every internal vertex after the level loop (Section 3.5).  dW_x, the bias
// and the loss head stay lazy.  Measured with bench.py; off by default.
bool eager_dw_enabled() { return env_on("CAVS_EAGER_DW"); }

// Ablation of kernel fusion in the backward pass (CAVS_UNFUSED_BWD_GATES=1):
// no child's dA is formed in its parent's product epilogue; every level gets
// its own elementwise gates kernel, as the levels above 256 positions always
// do.  Measured with bench.py; off by default.
bool unfused_bwd_gates() { return env_on("CAVS_UNFUSED_BWD_GATES"); }

// Ablation of kernel fusion in the forward pass (CAVS_UNFUSED_FWD_GATES=1):
// each level's product kernel stores its pre-activation parts and an
// elementwise kernel applies the gates, cell update and scatter; the leaves
// too get their cells from that kernel instead of the pull product's
// epilogue.  Measured with bench.py; off by default.
bool unfused_fwd_gates() { return env_on("CAVS_UNFUSED_FWD_GATES"); }

// Ablation of the single-stream lazy phase (CAVS_TWO_STREAM=1; fused
// Tree-LSTM path with inputs): the input-side products (dW_x, dX) run on a
// second stream beside the recurrent ones (dU), joined before the split-K
// reductions.  The second stream keeps the default priority.
bool two_stream_lazy() { return env_on("CAVS_TWO_STREAM"); }

hipError_t side_stream(cavs_ctx* ctx) {
  if (ctx->side) return hipSuccess;
  hipError_t e = hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&ctx->fork_ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&ctx->join_ev, hipEventDisableTiming);
  return e;
}

// dU contributions of the internal positions [off, off + M): queued split-K
// products whose reductions add into dU (acc) or overwrite it (first level).
bool lstm_dU_level(const Net& n, int off, int M, float* dU, float* part, size_t pf, bool acc,
                   hipStream_t str) {
  SplitJobs jobs;
  lstm_dU_iou(n, off, dU, part, pf, str, &jobs, M);
  lstm_dU_f(n, off, dU, part + pf, pf, str, &jobs, M);
  if (jobs.n != (n.N == 2 ? 2 : 1)) return false;   // a reduction ran unqueued (overwrote dU)
  for (int k = 0; k < jobs.n; ++k) jobs.j[k].acc = acc;
  reduce_split_jobs(jobs, str);
  return true;
}

Net make_net(const cavs_params* p, const cavs_sched* s, const cavs_inputs* in, void* ws,
             const WsLayout& L, bool train) {
  Net n{};
  char* base = (char*)ws;
  n.V = s->V;
  n.N = p->N;
  n.D = p->D;
  n.H = p->H;
  n.C = p->C;
  n.CP = p->loss == CAVS_LOSS_CE ? (p->C + 3) / 4 * 4 : 0;
  n.loss = p->loss;
  n.bf = p->prec == CAVS_BF16;
  n.GW = p->cell == CAVS_TREE_LSTM ? (3 + p->N) * p->H : p->H;
  n.inv_denom = 1.f / (float)(s->n_labelled > 0 ? s->n_labelled : 1);
  n.child_pos = s->child_pos;
  n.parent_pos = s->parent_pos;
  n.pull_pos = s->pull_pos;
  n.push_pos = s->push_pos;
  n.order = s->order;
  n.pull_list = s->pull_list;
  n.Wx = p->Wx;
  n.U = p->U;
  n.b = p->b;
  n.Ws = p->Ws;
  n.bs = p->bs;
  n.WsT = (float*)((char*)ws + L.WsT);
  n.X = in->X;
  n.Y = in->Y;
  n.P = (float*)(base + L.P);
  n.UT = (float*)(base + L.UT);
  n.zrow = (float*)(base + L.zrow);
  n.WxT = (float*)(base + L.WxT);
  n.fuse_from = s->V;
  n.f_unread_below = 0;
  n.Hs = (float*)(base + L.Hs);
  n.Cs = (float*)(base + L.Cs);
  n.Gs = (float*)(base + L.Gs);
  n.dZ = (float*)(base + L.dZ);
  n.lossv = (float*)(base + L.lossv);
  n.dHL = (float*)(base + L.dHL);
  n.dHp = (float*)(base + L.dHp);
  n.dCp = (float*)(base + L.dCp);
  n.dA = (float*)(base + L.dA);
  n.pack = L.pack_elems > 0 ? (unsigned short*)(base + L.pack) : nullptr;
  const bool ubf = p->cell == CAVS_TREE_LSTM && p->prec == CAVS_BF16 && !generic_mode(p, s);
  n.Ub = ubf ? (unsigned short*)(base + L.Ub) : nullptr;
  n.UTb = ubf ? (unsigned short*)(base + L.UTb) : nullptr;
  n.dAb = ubf && train ? (unsigned short*)(base + L.dAb) : nullptr;
  n.pack_elems = L.pack_elems;
  if (!train) {   // the kernels test these for null and skip what only backward reads
    if (!(p->cell == CAVS_TREE_LSTM && generic_mode(p, s))) n.Gs = nullptr;
    if (!lm_head(p)) n.dZ = nullptr;
    n.dHL = nullptr;
    n.dHp = nullptr;
    n.dCp = nullptr;
    n.dA = nullptr;
  }
  return n;
}

GenBufDev gen_bufs(const cavs_sched* s, void* ws, const WsLayout& L) {
  char* base = (char*)ws;
  GenBufDev b{};
  b.Ht = (float*)(base + L.gHt);
  b.Dt = (float*)(base + L.gDt);
  b.Eh = (float*)(base + L.gEh);
  b.Ec = (float*)(base + L.gEc);
  b.dAx = (float*)(base + L.gdAx);
  b.part = (float*)(base + L.gpart);
  b.part_cap = L.gpart_floats;
  b.in_off = s->dag ? s->in_offsets : nullptr;
  b.in_edge = s->dag ? s->in_edges : nullptr;
  return b;
}

}  // namespace
}  // namespace cavs

using namespace cavs;

extern "C" {

cavs_status cavs_create(cavs_ctx** out, int32_t device, void* hip_stream) {
  if (!out) return CAVS_ERR_ARG;
  *out = nullptr;
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev)
    return CAVS_ERR_ARG;
  cavs_ctx* ctx = new cavs_ctx();
  ctx->device = device;
  ctx->stream = (hipStream_t)hip_stream;
  // The host stage is coherent mapped memory: the scheduler's first kernel
  // writes it directly (no device->host copy on the stream), and the host
  // reads it once the event recorded after that kernel has completed.
  if (hipSetDevice(device) != hipSuccess ||
      hipHostMalloc((void**)&ctx->host_stage, sizeof(int32_t) * kHostStageInts,
                    hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess ||
      hipHostGetDevicePointer((void**)&ctx->host_stage_dev, ctx->host_stage, 0) != hipSuccess ||
      hipEventCreateWithFlags(&ctx->stage_ready, hipEventDisableTiming) != hipSuccess ||
      hipHostMalloc((void**)&ctx->dev_err, 64, hipHostMallocMapped | hipHostMallocCoherent) !=
          hipSuccess ||
      hipHostGetDevicePointer((void**)&ctx->dev_err_dev, ctx->dev_err, 0) != hipSuccess) {
    if (ctx->host_stage) (void)hipHostFree(ctx->host_stage);
    if (ctx->dev_err) (void)hipHostFree(ctx->dev_err);
    if (ctx->stage_ready) (void)hipEventDestroy(ctx->stage_ready);
    delete ctx;
    return CAVS_ERR_HIP;
  }
  ctx->dev_err[0] = 0;
  if (static_sched_scratch(ctx, device, &ctx->sched_scratch) != CAVS_OK) {
    (void)hipHostFree(ctx->host_stage);
    (void)hipHostFree(ctx->dev_err);
    (void)hipEventDestroy(ctx->stage_ready);
    delete ctx;
    return CAVS_ERR_HIP;
  }
  *out = ctx;
  return CAVS_OK;
}

cavs_status cavs_set_stream(cavs_ctx* ctx, void* hip_stream) {
  if (!ctx) return CAVS_ERR_ARG;
  ctx->stream = (hipStream_t)hip_stream;
  return CAVS_OK;
}

void cavs_destroy(cavs_ctx* ctx) {
  if (!ctx) return;
  if (ctx->host_stage) (void)hipHostFree(ctx->host_stage);
  if (ctx->dev_err) (void)hipHostFree(ctx->dev_err);
  if (ctx->stage_ready) (void)hipEventDestroy(ctx->stage_ready);
  for (auto& r : ctx->timed) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  for (auto e : ctx->event_pool) (void)hipEventDestroy(e);
  if (ctx->side) (void)hipStreamDestroy(ctx->side);
  if (ctx->fork_ev) (void)hipEventDestroy(ctx->fork_ev);
  if (ctx->join_ev) (void)hipEventDestroy(ctx->join_ev);
  delete ctx;
}

cavs_status cavs_timing_enable(cavs_ctx* ctx, int32_t on) {
  if (!ctx) return CAVS_ERR_ARG;
  for (auto& r : ctx->timed) {
    ctx->event_pool.push_back(r.start);
    ctx->event_pool.push_back(r.stop);
  }
  ctx->timed.clear();
  ctx->timing = on != 0;
  return CAVS_OK;
}

int32_t cavs_timing_read(cavs_ctx* ctx, cavs_launch_time* out, int32_t max) {
  if (!ctx || (max > 0 && !out)) return CAVS_ERR_ARG;
  if (hipStreamSynchronize(ctx->stream) != hipSuccess)
    return fail(ctx, CAVS_ERR_HIP, "hipStreamSynchronize failed");
  const cavs_status derr = device_errors(ctx);
  int32_t n = 0;
  for (auto& r : ctx->timed) {
    float ms = 0.f;
    (void)hipEventElapsedTime(&ms, r.start, r.stop);
    if (n < max) {
      memset(out[n].name, 0, sizeof out[n].name);
      strncpy(out[n].name, r.name, sizeof out[n].name - 1);
      out[n].row0 = r.row0;
      out[n].rows = r.rows;
      out[n].ms = ms;
    }
    ++n;
    ctx->event_pool.push_back(r.start);
    ctx->event_pool.push_back(r.stop);
  }
  ctx->timed.clear();
  return derr != CAVS_OK ? derr : n;
}

cavs_status cavs_sync(cavs_ctx* ctx) {
  if (!ctx) return CAVS_ERR_ARG;
  ctx->err.clear();
  CAVS_HIP_CHECK(ctx, hipSetDevice(ctx->device));
  CAVS_HIP_CHECK(ctx, hipStreamSynchronize(ctx->stream));
  return device_errors(ctx);
}

const char* cavs_last_error(const cavs_ctx* ctx) {
  if (!ctx) return "null context";
  return ctx->err.c_str();
}

size_t cavs_schedule_workspace_bytes(int32_t V, int32_t N, int32_t n_x) {
  return schedule_ws_bytes(V, N, n_x);
}

static cavs_status schedule_checks(cavs_ctx* ctx, const cavs_graphs* g, cavs_sched* s) {
  if (!g || !s) return fail(ctx, CAVS_ERR_ARG, "null graphs / sched");
  if (g->V < 0 || g->n_x < 0 || g->n_push < 0) return fail(ctx, CAVS_ERR_ARG, "negative size");
  if (g->N < 1 || g->N > kMaxSlots)
    return fail(ctx, CAVS_ERR_UNSUPPORTED, "N=%d child slots", g->N);
  if (g->V > 0 && !g->child) return fail(ctx, CAVS_ERR_ARG, "the child array is required");
  if (g->V > 0 && !g->parent && (!s->in_offsets || !s->in_edges))
    return fail(ctx, CAVS_ERR_ARG, "graph inputs need in_offsets / in_edges in the schedule");
  if (g->V > 0 && (!s->level || !s->order || !s->pos || !s->child_pos || !s->parent_pos ||
                   !s->pull_pos || !s->push_pos || !s->pull_list || !s->level_offsets))
    return fail(ctx, CAVS_ERR_ARG, "schedule output arrays are required");
  if (!s->level_offsets_host) return fail(ctx, CAVS_ERR_ARG, "level_offsets_host is required");
  return CAVS_OK;
}

cavs_status cavs_schedule(cavs_ctx* ctx, const cavs_graphs* g, cavs_sched* s, void* ws,
                          size_t ws_bytes) {
  if (!ctx) return CAVS_ERR_ARG;
  ctx->err.clear();
  cavs_status st = schedule_checks(ctx, g, s);
  if (st != CAVS_OK) return st;
  if (g->V > 0 && !ws) return fail(ctx, CAVS_ERR_ARG, "workspace is required");
  if (hipSetDevice(ctx->device) != hipSuccess) return fail(ctx, CAVS_ERR_HIP, "hipSetDevice");
  ActiveCtx active(ctx);
  return schedule_run(ctx, g, s, ws, ws_bytes);
}

cavs_status cavs_schedule_static(cavs_ctx* ctx, const cavs_graphs* g, cavs_sched* s) {
  if (!ctx) return CAVS_ERR_ARG;
  ctx->err.clear();
  cavs_status st = schedule_checks(ctx, g, s);
  if (st != CAVS_OK) return st;
  if (!ctx->sched_scratch)
    return fail(ctx, CAVS_ERR_UNSUPPORTED, "no static scheduling scratch for device %d",
                ctx->device);
  const size_t need = schedule_ws_bytes(g->V, g->N, g->n_x);
  if (need > (size_t)CAVS_SCHEDULE_STATIC_BYTES)
    return fail(ctx, CAVS_ERR_WORKSPACE,
                "cavs_schedule_static: V=%d, n_x=%d need %zu bytes of scratch, the static "
                "array holds %zu; use cavs_schedule with a workspace",
                g->V, g->n_x, need, (size_t)CAVS_SCHEDULE_STATIC_BYTES);
  if (hipSetDevice(ctx->device) != hipSuccess) return fail(ctx, CAVS_ERR_HIP, "hipSetDevice");
  ActiveCtx active(ctx);
  return schedule_run(ctx, g, s, ctx->sched_scratch, (size_t)CAVS_SCHEDULE_STATIC_BYTES);
}

size_t cavs_workspace_bytes(const cavs_params* p, const cavs_sched* s) {
  if (!p || !s || p->H <= 0 || p->N <= 0 || s->V < 0) return 0;
  return ws_layout(p, s, true).total;
}

size_t cavs_infer_workspace_bytes(const cavs_params* p, const cavs_sched* s) {
  if (!p || !s || p->H <= 0 || p->N <= 0 || s->V < 0) return 0;
  return ws_layout(p, s, false).total;
}

// Forward of Algorithm 1 over every task, then the loss head.  train:
// also keep what the backward reads (saved gates, the head's gradients).
static cavs_status run_forward(cavs_ctx* ctx, const cavs_params* p, const cavs_sched* s,
                        const cavs_inputs* in, float* h_out, float* c_out, float* loss_out,
                        void* ws, size_t ws_bytes, bool train) {
  if (!ctx) return CAVS_ERR_ARG;
  ctx->err.clear();
  cavs_status st = check_args(ctx, p, s, in);
  if (st != CAVS_OK) return st;
  if (!loss_out || (s->V > 0 && !h_out)) return fail(ctx, CAVS_ERR_ARG, "null output");
  WsLayout L = ws_layout(p, s, train);
  if (!ws || ws_bytes < L.total)
    return fail(ctx, CAVS_ERR_WORKSPACE, "workspace too small: %zu < %zu", ws_bytes, L.total);
  CAVS_HIP_CHECK(ctx, hipSetDevice(ctx->device));
  ActiveCtx active(ctx);
  hipStream_t str = ctx->stream;
  if (s->V == 0) {
    CAVS_HIP_CHECK(ctx, zero_async(loss_out, sizeof(float), str));
    return CAVS_OK;
  }
  Net n = make_net(p, s, in, ws, L, train);
  n.h_out = h_out;
  n.c_out = p->cell == CAVS_TREE_LSTM ? c_out : nullptr;
  const int* lo = s->level_offsets_host;
  ctx->xcd_owner = {};
  if (n.Ub && s->T > 1) lstm_round_u(n, str);   // bf16 weight operands of the level products
  if (p->cell == CAVS_TREE_LSTM && generic_mode(p, s)) {
    lstm_transpose_u(n, str);
    pull_gemm(n, s->n_pull, s->n_inner_input > 0, 0, str);   // P for every pulling row
    lstm_fwd_gates(n, lo[0], lo[1] - lo[0], false, str);
    gen_forward_levels(n, gen_bufs(s, ws, L), lo, s->T, str);
  } else if (p->cell == CAVS_TREE_LSTM && train && unfused_fwd_gates()) {
    n.fwd_unfused = 1;
    if ((s->T > 1 && lstm_tile_applies(n, lo[2] - lo[1])) || pull_tile_applies(n, s->n_pull))
      lstm_transpose_u(n, str);
    pull_gemm(n, s->n_pull, s->n_inner_input > 0, 0, str);
    lstm_fwd_gates(n, lo[0], lo[1] - lo[0], false, str);
    for (int t = 1; t < s->T; ++t) {
      lstm_fwd_level(n, lo[t], lo[t + 1] - lo[t], str);
      lstm_fwd_gates(n, lo[t], lo[t + 1] - lo[t], true, str);
    }
  } else if (p->cell == CAVS_TREE_LSTM) {
    const int tx = xcd_first_level(n, lo, s->T);
    void* xws = (char*)ws + L.xcd;
    if ((s->T > 1 && lstm_tile_applies(n, lo[2] - lo[1])) || pull_tile_applies(n, s->n_pull))
      lstm_transpose_u(n, str);
    pull_gemm(n, s->n_pull, s->n_inner_input > 0, lo[1], str);
    // fp32: pulled leaves were finished by the pull product
    if (n.bf || s->n_leaf_noinput > 0) lstm_fwd_leaf(n, lo[0], lo[1] - lo[0], !n.bf, str);
    const int ts = tx < s->T ? tx : persist_first_level(n, lo, s->T);
    for (int t = 1; t < ts; ++t) lstm_fwd_level(n, lo[t], lo[t + 1] - lo[t], str);
    int* bar = (int*)((char*)ws + L.bar);
    if (tx < s->T) {
      // the loop's owner array depends on the schedule alone: the matching
      // backward reuses it
      xcd_owner(n, lo, tx, xws, str);
      ctx->xcd_owner = {ws, n.parent_pos, lo[tx], s->V};
      if (!lstm_fwd_xcd(n, s->level_offsets, lo, tx, s->T, xws, true, str))
        for (int t = tx; t < s->T; ++t) lstm_fwd_level(n, lo[t], lo[t + 1] - lo[t], str);
    } else if (!lstm_fwd_persist(n, s->level_offsets, lo, ts, s->T, bar, str)) {
      for (int t = ts; t < s->T; ++t) lstm_fwd_level(n, lo[t], lo[t + 1] - lo[t], str);
    }
  } else {
    if (s->T > 1) fc_transpose(n, str);
    fc_fwd_leaf(n, lo[0], lo[1] - lo[0], str);
    for (int t = 1; t < s->T; ++t) fc_fwd_level(n, lo[t], lo[t + 1] - lo[t], str);
  }
  loss_fwd(n, loss_out, str);
  CAVS_LAUNCH_CHECK(ctx);
  return CAVS_OK;
}

cavs_status cavs_forward(cavs_ctx* ctx, const cavs_params* p, const cavs_sched* s,
                         const cavs_inputs* in, float* h_out, float* c_out, float* loss_out,
                         void* ws, size_t ws_bytes) {
  return run_forward(ctx, p, s, in, h_out, c_out, loss_out, ws, ws_bytes, true);
}

cavs_status cavs_infer(cavs_ctx* ctx, const cavs_params* p, const cavs_sched* s,
                       const cavs_inputs* in, float* h_out, float* c_out, float* loss_out,
                       void* ws, size_t ws_bytes) {
  return run_forward(ctx, p, s, in, h_out, c_out, loss_out, ws, ws_bytes, false);
}

cavs_status cavs_backward(cavs_ctx* ctx, const cavs_params* p, const cavs_sched* s,
                          const cavs_inputs* in, void* ws, size_t ws_bytes,
                          const cavs_grads* g) {
  if (!ctx) return CAVS_ERR_ARG;
  ctx->err.clear();
  cavs_status st = check_args(ctx, p, s, in);
  if (st != CAVS_OK) return st;
  if (!g || !g->dU || !g->db) return fail(ctx, CAVS_ERR_ARG, "null gradient output");
  if (p->cell == CAVS_TREE_LSTM && p->D > 0 && !g->dWx)
    return fail(ctx, CAVS_ERR_ARG, "dWx is required");
  if (p->loss == CAVS_LOSS_CE && (!g->dWs || !g->dbs))
    return fail(ctx, CAVS_ERR_ARG, "dWs / dbs are required for CE");
  if (s->n_x > 0 && !g->dX) return fail(ctx, CAVS_ERR_ARG, "dX is required");
  WsLayout L = ws_layout(p, s, true);
  if (!ws || ws_bytes < L.total)
    return fail(ctx, CAVS_ERR_WORKSPACE, "workspace too small: %zu < %zu", ws_bytes, L.total);
  CAVS_HIP_CHECK(ctx, hipSetDevice(ctx->device));
  ActiveCtx active(ctx);
  hipStream_t str = ctx->stream;
  const int H = p->H, D = p->D;
  const bool lstm = p->cell == CAVS_TREE_LSTM;
  if (s->V == 0) {
    const size_t nU = lstm ? (size_t)H * 4 * H : (size_t)p->N * H * H;
    CAVS_HIP_CHECK(ctx, zero_async(g->dU, nU * sizeof(float), str));
    CAVS_HIP_CHECK(ctx, zero_async(g->db, (lstm ? 4 * H : H) * sizeof(float), str));
    if (lstm && D > 0)
      CAVS_HIP_CHECK(ctx, zero_async(g->dWx, (size_t)D * 4 * H * sizeof(float), str));
    if (p->loss == CAVS_LOSS_CE) {
      CAVS_HIP_CHECK(ctx, zero_async(g->dWs, (size_t)H * p->C * sizeof(float), str));
      CAVS_HIP_CHECK(ctx, zero_async(g->dbs, (size_t)p->C * sizeof(float), str));
    }
    if (s->n_x > 0)
      CAVS_HIP_CHECK(ctx, zero_async(g->dX, (size_t)s->n_x * D * sizeof(float), str));
    return CAVS_OK;
  }
  Net n = make_net(p, s, in, ws, L, true);
  if (in->dH_ext) {   // the push connector's gradient joins the loss head's term
    float* dhlx = (float*)((char*)ws + L.dHLx);
    add_external_grad(n, in->dH_ext, dhlx, str);
    n.dHL = dhlx;
  }
  float* part = (float*)((char*)ws + L.part);
  float* bpart = (float*)((char*)ws + L.bpart);
  const int* lo = s->level_offsets_host;
  const int T = s->T;
  const int off1 = T > 1 ? lo[1] : s->V;
  if (s->n_x > 0 && s->n_pull < s->n_x)
    CAVS_HIP_CHECK(ctx, zero_async(g->dX, (size_t)s->n_x * D * sizeof(float), str));
  if (lstm && generic_mode(p, s)) {
    gen_backward(n, gen_bufs(s, ws, L), lo, T, s->n_pull, g->dU, g->db, g->dWx, g->dX, g->dWs,
                 g->dbs, str);
  } else if (lstm) {
    // Levels tf.. get dA in their parent's level epilogue (roots: one
    // kernel); levels below tf by an elementwise kernel just before their
    // own product, once every parent has stored dL/dh and dL/dc.
    const int tf = unfused_bwd_gates() ? T : lstm_fuse_level(lo, T);
    n.fuse_from = lo[tf];
    n.f_unread_below = s->n_inner_input > 0 ? 0 : lo[1];
    const bool eager = T > 1 && eager_dw_enabled();
    const size_t pf = L.part_floats;
    lstm_bwd_roots(n, str);
    // the XCD-local loop takes fused levels only (every child of its levels
    // is finished in the parent's epilogue or left dL/dh below fuse_from)
    const int tx = eager ? T : xcd_first_level(n, lo, T);
    int ts = T;
    if (tx < T && tf <= tx) {
      const auto& o = ctx->xcd_owner;
      const bool owned = o.ws == ws && o.parent_pos == n.parent_pos && o.base == lo[tx] &&
                         o.V == s->V;
      if (lstm_bwd_xcd(n, s->level_offsets, lo, tx, T, (char*)ws + L.xcd, owned, str)) ts = tx;
    } else {
      ts = eager ? T : persist_first_level(n, lo, T);
      if (ts < tf) ts = tf;
      int* bar = (int*)((char*)ws + L.bar);
      if (!lstm_bwd_persist(n, s->level_offsets, lo, ts, T, bar, str)) ts = T;
    }
    for (int t = ts - 1; t >= 0; --t) {
      const int M = lo[t + 1] - lo[t];
      if (t < tf) lstm_bwd_gates(n, lo[t], M, str);
      if (t >= 1) lstm_bwd_level(n, lo[t], M, str);
      // level t's dA is complete once its own product has been enqueued
      if (eager && t >= 1 && !lstm_dU_level(n, lo[t], M, g->dU, part, pf, t < T - 1, str))
        return fail(ctx, CAVS_ERR_UNSUPPORTED, "per-level dU reduction could not be queued");
    }
    // the lazy products keep their split-K sums in separate scratch and share
    // one reduction launch
    const bool with_f = s->n_inner_input > 0;
    SplitJobs jobs;
    const bool two = !eager && D > 0 && two_stream_lazy();
    if (two) {
      CAVS_HIP_CHECK(ctx, side_stream(ctx));
      CAVS_HIP_CHECK(ctx, hipEventRecord(ctx->fork_ev, str));
      CAVS_HIP_CHECK(ctx, hipStreamWaitEvent(ctx->side, ctx->fork_ev, 0));
      lstm_dWx(n, s->n_pull, with_f, g->dWx, part + 2 * pf, pf, ctx->side, &jobs);
      dx_gemm(n, s->n_pull, with_f, g->dX, ctx->side);
      CAVS_HIP_CHECK(ctx, hipEventRecord(ctx->join_ev, ctx->side));
      lstm_dU_iou(n, off1, g->dU, part, pf, str, &jobs);
      lstm_dU_f(n, off1, g->dU, part + pf, pf, str, &jobs);
    } else if (eager) {
      if (D > 0) lstm_dWx(n, s->n_pull, with_f, g->dWx, part + 2 * pf, pf, str, &jobs);
    } else if (!lstm_lazy_grouped(n, off1, s->n_pull, with_f, g->dU, g->dWx, part, pf, str,
                                  &jobs)) {
      lstm_dU_iou(n, off1, g->dU, part, pf, str, &jobs);
      lstm_dU_f(n, off1, g->dU, part + pf, pf, str, &jobs);
      if (D > 0) lstm_dWx(n, s->n_pull, with_f, g->dWx, part + 2 * pf, pf, str, &jobs);
    }
    bias_head_grads(n, 0, s->V, off1, g->db, g->dWs, g->dbs, bpart, str, &jobs);
    if (two) CAVS_HIP_CHECK(ctx, hipStreamWaitEvent(str, ctx->join_ev, 0));
    reduce_split_jobs(jobs, str);
    if (lm_head(p))
      lm_head_grads(n, g->dWs, g->dbs, (float*)((char*)ws + L.gpart), L.gpart_floats, str);
    if (!two) dx_gemm(n, s->n_pull, with_f, g->dX, str);
  } else {
    // roots first; every other vertex's delta (or a leaf's input gradient)
    // comes from its parent's level product
    n.dX = g->dX;
    n.leaf_end = off1;
    fc_bwd_roots(n, str);
    for (int t = T - 1; t >= 1; --t) fc_bwd_level(n, lo[t], lo[t + 1] - lo[t], str);
    SplitJobs jobs;
    fc_dW(n, off1, g->dU, part, L.part_floats, str, &jobs);
    bias_head_grads(n, off1, s->V, off1, g->db, g->dWs, g->dbs, bpart, str, &jobs);
    reduce_split_jobs(jobs, str);
    if (lm_head(p))
      lm_head_grads(n, g->dWs, g->dbs, (float*)((char*)ws + L.gpart), L.gpart_floats, str);
  }
  CAVS_LAUNCH_CHECK(ctx);
  return CAVS_OK;
}

}  // extern "C"
