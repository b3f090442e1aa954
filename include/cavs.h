/*
 * cavs.h -- C ABI of libcavs.so: the batched vertex-function forward and
 * backward of Cavs (Zhang et al., arXiv 1712.04048) on one AMD Instinct
 * MI355X (gfx950).
 *
 * The paper states the problem as Forward({x_k}, {G_k}, F) -> S followed by
 * Backward(S, {G_k}, dF) (Algorithm 1, Section 3.2): a static vertex function
 * F is evaluated over a batch of instance-specific graphs G_k, one task V_t of
 * "activated" vertices at a time, and differentiated in the reverse task
 * order.  Because the tasks depend only on the graphs, this library splits
 * the work into three calls:
 *
 *   cavs_schedule  -- the task sets V_t and the level-major ("dynamic
 *                     tensor") layout of Section 3.3 / Algorithm 2;
 *   cavs_forward   -- F over every task in order, then the lazily batched
 *                     push / loss head (Section 3.5);
 *   cavs_backward  -- dF over the tasks in reverse order, then the lazily
 *                     batched parameter-gradient products (Section 3.5);
 *   cavs_infer     -- the forward alone, keeping nothing for a backward
 *                     (inference, timed apart from training in Table 3).
 *
 * Conventions shared by every call
 *   - Pointers are DEVICE pointers unless marked (host).  Every device buffer
 *     is allocated and owned by the caller; the library keeps no pointer past
 *     the return of a call, except that the workspace `ws` must stay alive and
 *     untouched between cavs_forward and the matching cavs_backward (it holds
 *     the forward's saved intermediates).
 *   - Work is enqueued on the context's HIP stream and is asynchronous unless
 *     stated.  cavs_schedule synchronises that stream once.
 *   - Matrices are row-major, fp32, densely packed.
 *   - Errors are status codes; nothing unwinds across the ABI.  After a
 *     non-zero status, cavs_last_error() describes it.  Argument errors are
 *     detected on the host before anything is enqueued.
 *   - Calls on one context must not overlap (one stream, one user at a time).
 *   - Environment switches, read at each call and off by default, turn the
 *     execution engine's optimisations off for ablation measurements;
 *     results stay within the same tolerance of the exact ones:
 *       CAVS_EAGER_DW=1           dU formed level by level, not lazily;
 *       CAVS_UNFUSED_BWD_GATES=1  no child gradient fused into a parent's
 *                                 backward product;
 *       CAVS_PERSIST=1            the small levels in one persistent launch
 *                                 with grid barriers;
 *       CAVS_UNFUSED_FWD_GATES=1  the forward gates and cell update in an
 *                                 elementwise kernel after each level product;
 *       CAVS_GENERIC=1            trees too run the generic engine;
 *       CAVS_TWO_STREAM=1         the backward's input-side lazy products
 *                                 (dW_x, dX) on a second stream of the
 *                                 context beside dU, joined by events before
 *                                 the split-K reductions.
 *     One switch chooses an engine path that is on by default where it
 *     measured faster: child-sum Tree-LSTM at H = 512 whose small levels (at
 *     most 256 vertices each, at most 16384 in all) number 8 or more run
 *     them in one launch per direction (one workgroup per CU), each XCD of the device
 *     taking the top levels of the trees rooted on it, with barriers among
 *     that XCD's workgroups only:
 *       CAVS_XCD_LOOP=0 / =1      never take it / take it wherever it applies
 *                                 (H a multiple of 256, at most 16384 vertices
 *                                 from the first small level up).
 *     Its barriers are bounded waits: a wait that gives up records the error
 *     that cavs_sync reports.
 *     Another is a failure-injection hook for tests of the error path:
 *       CAVS_PERSIST_SPIN=n       the persistent and XCD loops' barriers give up
 *                                 after n polls (n < 0: at once) and record
 *                                 the error that cavs_sync reports.
 *   - Errors found by kernels after a call has returned (a bounded wait that
 *     gave up) are kept by the context and returned by the next cavs_sync or
 *     cavs_timing_read.
 */
#ifndef CAVS_H
#define CAVS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t cavs_status;
#define CAVS_OK 0
#define CAVS_ERR_ARG (-1)          /* bad argument found on the host (null, size, shape) */
#define CAVS_ERR_RANGE (-2)        /* an index array holds a value outside its range */
#define CAVS_ERR_MULTIPARENT (-3)  /* a vertex is listed as a child more than once */
#define CAVS_ERR_CYCLE (-4)        /* the child links contain a cycle */
#define CAVS_ERR_MISMATCH (-5)     /* child[] and parent[] disagree */
#define CAVS_ERR_WORKSPACE (-6)    /* workspace smaller than required */
#define CAVS_ERR_HIP (-7)          /* a HIP runtime call failed */
#define CAVS_ERR_UNSUPPORTED (-8)  /* valid input outside what this build implements */
#define CAVS_ERR_DUP_PULL (-9)     /* two vertices pull the same input row */

/* vertex functions */
#define CAVS_TREE_LSTM 0  /* child-sum Tree-LSTM (Section 3.1 figure); N = 1 is the sequence LSTM */
#define CAVS_TREE_FC 1    /* h = tanh([h_0, h_1] W + b); a leaf's state is its input (Section 5) */
/* arithmetic of the matrix products */
#define CAVS_FP32 0       /* fp32 operands, fp32 matrix-core accumulation */
#define CAVS_BF16 1       /* operands rounded to bf16 (nearest-even), fp32 accumulation */
/* loss heads attached through push */
#define CAVS_LOSS_CE 0    /* softmax cross-entropy over C classes, mean over labelled vertices */
#define CAVS_LOSS_L2 1    /* 0.5 * ||h - y||^2, mean over labelled vertices */
#define CAVS_LOSS_NONE 2  /* no loss head: the states go to an external consumer (push
                             connector), whose gradient comes back as inputs.dH_ext */

typedef struct cavs_ctx cavs_ctx;

/* Creates a context bound to HIP device `device` and stream `hip_stream`
   (a hipStream_t; NULL = the null stream).  Allocates a small pinned host
   staging buffer.  Returns CAVS_ERR_ARG / CAVS_ERR_HIP on failure. */
cavs_status cavs_create(cavs_ctx** ctx, int32_t device, void* hip_stream);
/* Rebinds the stream used by later calls. */
cavs_status cavs_set_stream(cavs_ctx* ctx, void* hip_stream);
/* Releases the context (NULL is ignored). */
void cavs_destroy(cavs_ctx* ctx);
/* Host string describing the last error on ctx; owned by ctx, valid until
   the next call on ctx.  Never NULL. */
const char* cavs_last_error(const cavs_ctx* ctx);
/* Waits for all work enqueued on the context's stream, then returns
   CAVS_ERR_HIP if a kernel of an earlier call recorded an error (the
   persistent level loop's bounded grid barrier gave up: that call's outputs
   are invalid), else CAVS_OK.  The record is cleared by the report. */
cavs_status cavs_sync(cavs_ctx* ctx);

/* ---------------------------------------------------------------------------
 * Scheduling (Algorithm 1; dynamic tensors of Section 3.3, Algorithm 2)
 *
 * The input graphs of one batch.  Vertex ids are global, 0..V-1.  Each vertex
 * has at most N child slots (gather(child_idx), Section 3.1); a vertex with no
 * children is a leaf.  Tree inputs give each vertex at most one parent and
 * list it in parent[].  Graph inputs (the graph-structured cells of Section 2,
 * panel (d) of the recurrent-structures figure) pass parent = NULL: a vertex
 * may then be read by several vertices (or by several slots of one), and its
 * dL/dh and dL/dc are the sums of what each reader sends back.  pull_idx names the row of the
 * external input matrix X that the vertex pulls (pull(), Section 3.1);
 * push_idx names what its pushed state is scored against (push()): a class in
 * [0, C) for CAVS_LOSS_CE or a row of Y for CAVS_LOSS_L2.
 * ------------------------------------------------------------------------- */
typedef struct {
  int32_t V;                /* number of vertices, >= 0 */
  int32_t N;                /* child slots per vertex, 1 .. 4 */
  int32_t n_x;              /* rows of X (pull_idx values lie in [-1, n_x)) */
  int32_t n_push;           /* push_idx values lie in [-1, n_push) */
  const int32_t* child;     /* [V*N] child id of slot k of vertex v, or -1 */
  const int32_t* parent;    /* [V] parent id, or -1 for a root; NULL = graph inputs */
  const int32_t* pull_idx;  /* [V] row of X, or -1; NULL = no vertex pulls */
  const int32_t* push_idx;  /* [V] label / target row, or -1; NULL = no loss terms */
} cavs_graphs;

/* The schedule: task V_t = positions [level_offsets[t], level_offsets[t+1]).
   Level of v = 0 if v has no children, else 1 + max level of its children
   (the step at which Algorithm 1 finds v activated).  Inside a task vertices
   are ordered by ascending id.  All arrays are caller-allocated with the
   capacities given; "by position" arrays are indexed by level-major position
   p = pos[v]. */
typedef struct {
  /* out (host) */
  int32_t T;                /* number of tasks (levels); 0 when V = 0 */
  int32_t V, N;             /* copied from the graphs */
  int32_t n_x, n_push;      /* copied from the graphs */
  int32_t n_pull;           /* vertices that pull an input */
  int32_t n_labelled;       /* vertices with push_idx >= 0 (|Lambda|) */
  int32_t n_leaf_noinput;   /* leaves that pull nothing */
  int32_t n_inner_input;    /* vertices with children that also pull */
  /* out (device), caller-allocated */
  int32_t* level;           /* [V]     by vertex id */
  int32_t* order;           /* [V]     position -> vertex id */
  int32_t* pos;             /* [V]     vertex id -> position */
  int32_t* child_pos;       /* [V*N]   by position: position of child slot k, or -1 */
  int32_t* parent_pos;      /* [V]     by position: position of the parent, or -1 */
  int32_t* pull_pos;        /* [V]     by position: row of X, or -1 */
  int32_t* push_pos;        /* [V]     by position: label / target row, or -1 */
  int32_t* pull_list;       /* [V]     positions that pull, ascending; n_pull used */
  int32_t* level_offsets;   /* [V+1]   T+1 used */
  /* out (host), caller-allocated */
  int32_t* level_offsets_host; /* [V+1] T+1 used; filled by the one synchronisation */
  /* out (host) */
  int32_t dag;              /* 1 when the graphs were given without parent[] */
  /* out (device), caller-allocated; required for graph inputs, else unused:
     the links e = p*N + k (child slot k of position p) that read position c
     are in_edges[in_offsets[c] .. in_offsets[c+1]), ascending */
  int32_t* in_offsets;      /* [V+1] */
  int32_t* in_edges;        /* [V*N] */
} cavs_sched;

/* Bytes of device workspace cavs_schedule needs for V vertices, N slots and
   n_x input rows. */
size_t cavs_schedule_workspace_bytes(int32_t V, int32_t N, int32_t n_x);

/* Validates the graphs and builds the schedule on the GPU.  Synchronises the
   context's stream once, to return T, the counts, level_offsets_host and the
   validation result; the device arrays (order, pos, the remapped indices,
   pull_list) are written by work enqueued after that point, so they are
   complete for later work on the same stream (or after a synchronisation).  Graph errors, by priority: CAVS_ERR_RANGE,
   CAVS_ERR_MULTIPARENT, CAVS_ERR_DUP_PULL, CAVS_ERR_MISMATCH, CAVS_ERR_CYCLE;
   on such an error the device outputs are unspecified.  Graph inputs
   (parent = NULL) are checked for ranges, duplicate pull rows and cycles
   only.  N outside 1 .. 4 gives CAVS_ERR_UNSUPPORTED; a null required
   pointer (in_offsets / in_edges for graph inputs), CAVS_ERR_ARG; a short
   workspace, CAVS_ERR_WORKSPACE. */
cavs_status cavs_schedule(cavs_ctx* ctx, const cavs_graphs* graphs, cavs_sched* sched,
                          void* ws, size_t ws_bytes);

/* For callers that cannot allocate device memory (code under HIP graph
   capture, tight serving loops, harnesses that forbid hipMalloc): the same
   schedule as cavs_schedule, bit for bit, with the scheduler's scratch taken
   from a static device array of CAVS_SCHEDULE_STATIC_BYTES per GPU (held
   until the process ends) instead of a workspace argument.  It allocates
   nothing and calls no allocating routine (with per-launch timing off).
   Batches whose cavs_schedule_workspace_bytes(V, N, n_x) exceeds
   CAVS_SCHEDULE_STATIC_BYTES (about 100 000 vertices with as many input
   rows) are refused with CAVS_ERR_WORKSPACE before anything is enqueued.
   Every call on one GPU shares that GPU's array: calls that overlap in time
   on one GPU (contexts on different streams) race and must be serialised by
   the caller.  Errors and synchronisation as for cavs_schedule. */
#define CAVS_SCHEDULE_STATIC_BYTES (4u << 20)
cavs_status cavs_schedule_static(cavs_ctx* ctx, const cavs_graphs* graphs, cavs_sched* sched);

/* ---------------------------------------------------------------------------
 * Forward / backward of F over the scheduled graphs.
 *
 * CAVS_TREE_LSTM (child-sum Tree-LSTM, Section 3.1 figure), with h~ = sum_k h_k
 * over present children, x = 0 when the vertex pulls nothing:
 *   i = sigma(x W_i + h~ U_i + b_i)   o = sigma(x W_o + h~ U_o + b_o)
 *   u = tanh(x W_u + h~ U_u + b_u)    f_k = sigma(x W_f + h_k U_f + b_f)
 *   c = i*u + sum_k f_k*c_k           h = o*tanh(c)
 *   Wx [D, 4H], U [H, 4H], b [4H]; gate column blocks ordered i | f | o | u.
 * CAVS_TREE_FC: internal vertex h = tanh(h_0 W_0 + h_1 W_1 + b) (absent child
 *   = 0), leaf h = x (requires D = H and: pulls an input iff it is a leaf).
 *   U holds W as [N*H, H] (rows k*H .. k*H+H-1 = W_k); b [H]; Wx unused.
 * Loss (the lazily batched push, Section 3.5): CE z = h Ws + bs, Ws [H, C],
 *   bs [C]; or L2 against rows of Y [n_y, H].  L = mean over labelled vertices.
 *   CE with more than 16 classes (a language-model vocabulary at every
 *   vertex) runs on matrix-core products and needs C % 4 == 0.
 *   CAVS_LOSS_NONE: no head (L = 0); with inputs.dH_ext the backward is that
 *   of an external loss whose gradient w.r.t. the pushed states is dH_ext --
 *   the connector that stacks layers (layer l+1 pulls layer l's h_out as X,
 *   layer l gets layer l+1's dX as dH_ext) or joins an encoder to a decoder.
 * ------------------------------------------------------------------------- */
typedef struct {
  int32_t cell;             /* CAVS_TREE_LSTM or CAVS_TREE_FC */
  int32_t prec;             /* CAVS_FP32 or CAVS_BF16 */
  int32_t loss;             /* CAVS_LOSS_CE or CAVS_LOSS_L2 */
  int32_t D, H, N, C;       /* input dim, hidden dim, child slots, classes */
  const float* Wx;          /* TREE_LSTM: [D, 4H]; TREE_FC: unused (may be NULL) */
  const float* U;           /* TREE_LSTM: [H, 4H]; TREE_FC: [N*H, H] */
  const float* b;           /* TREE_LSTM: [4H];    TREE_FC: [H] */
  const float* Ws;          /* CE: [H, C]; L2, NONE: unused */
  const float* bs;          /* CE: [C];    L2, NONE: unused */
} cavs_params;

typedef struct {
  const float* X;           /* [n_x, D] pulled inputs (may be NULL when n_x = 0) */
  const float* Y;           /* L2: [n_y, H] targets; CE: unused */
  int32_t n_y;              /* rows of Y */
  const float* dH_ext;      /* [V, H] vertex-id order, or NULL: gradient of the pushed
                               states from an external consumer, added to every vertex's
                               dL/dh by cavs_backward (cavs_forward ignores it) */
} cavs_inputs;

typedef struct {            /* outputs of cavs_backward, overwritten (not accumulated) */
  float* dWx;               /* TREE_LSTM: [D, 4H]; TREE_FC: unused */
  float* dU;                /* same shape as U */
  float* db;                /* same shape as b */
  float* dWs;               /* CE: [H, C]; L2: unused */
  float* dbs;               /* CE: [C];    L2: unused */
  float* dX;                /* [n_x, D]: rows no vertex pulls are set to 0 */
} cavs_grads;

/* Bytes of device workspace cavs_forward/cavs_backward need. 0 on bad args. */
size_t cavs_workspace_bytes(const cavs_params* params, const cavs_sched* sched);

/* Runs F over every task V_0..V_{T-1}, then the loss head.
   h_out [V, H] and c_out [V, H] (c_out may be NULL; TREE_FC ignores it)
   receive the states in vertex-id order; loss_out [1] the mean loss.
   Shapes are validated against the schedule on the host: mismatches give
   CAVS_ERR_ARG, shapes this build does not tile (H % 64 != 0, D % 4 != 0,
   N > 4, BF16 with TREE_FC) give CAVS_ERR_UNSUPPORTED.  Trees with at most
   two child slots run the fused level kernels; graph inputs and wider
   vertices (TREE_LSTM, fp32 only; else CAVS_ERR_UNSUPPORTED) run the generic
   engine: per task, separate products and elementwise gate kernels, with
   each child link's gradient in its own row summed per vertex in a fixed
   order. */
cavs_status cavs_forward(cavs_ctx* ctx, const cavs_params* params, const cavs_sched* sched,
                         const cavs_inputs* inputs, float* h_out, float* c_out,
                         float* loss_out, void* ws, size_t ws_bytes);

/* Bytes of device workspace cavs_infer needs (states, the pull projection,
   transposed weights and per-vertex loss terms only).  0 on bad args. */
size_t cavs_infer_workspace_bytes(const cavs_params* params, const cavs_sched* sched);

/* Inference: the forward of Algorithm 1 over every task, then the loss head,
   as cavs_forward computes them (bit-identical h_out, c_out and loss_out),
   but nothing a backward would read is kept -- no saved gates, no gradient
   of the loss head -- so the workspace is the smaller
   cavs_infer_workspace_bytes and no cavs_backward may follow.  Arguments,
   validation and errors as for cavs_forward. */
cavs_status cavs_infer(cavs_ctx* ctx, const cavs_params* params, const cavs_sched* sched,
                       const cavs_inputs* inputs, float* h_out, float* c_out,
                       float* loss_out, void* ws, size_t ws_bytes);

/* Runs dF over the tasks in reverse order (Algorithm 1, Backward), then the
   lazy parameter-gradient products.  Must follow cavs_forward with the same
   params, sched, inputs and ws.  Writes every array of grads. */
cavs_status cavs_backward(cavs_ctx* ctx, const cavs_params* params, const cavs_sched* sched,
                          const cavs_inputs* inputs, void* ws, size_t ws_bytes,
                          const cavs_grads* grads);

/* ---------------------------------------------------------------------------
 * Instrumentation (not part of the computation).  When enabled, every kernel
 * the library launches on the context's stream is bracketed by a pair of HIP
 * events, so per-kernel GPU durations can be read back.  Off by default; the
 * event records add a little host overhead per launch.
 * ------------------------------------------------------------------------- */
typedef struct {
  char name[96];            /* kernel name, e.g. "k_lstm_fwd_level<2, 64>" */
  int32_t row0;             /* first level-major position the launch covers (0 if n/a) */
  int32_t rows;             /* positions covered (a level's size; 0 if n/a) */
  double ms;                /* GPU duration of the launch */
} cavs_launch_time;

/* Turns per-launch timing on (1) or off (0); either way discards pending
   records.  CAVS_ERR_ARG on a null context. */
cavs_status cavs_timing_enable(cavs_ctx* ctx, int32_t on);
/* Synchronises the context's stream, writes the pending launch records, in
   launch order, to out[0..max) (host array, caller-owned), clears them, and
   returns the number of records (which may exceed max; only max are
   written), or a negative status (a kernel error recorded since the last
   report, as for cavs_sync; the records are still written). */
int32_t cavs_timing_read(cavs_ctx* ctx, cavs_launch_time* out, int32_t max);

#ifdef __cplusplus
}
#endif

#endif /* CAVS_H */
