/*
 * oracle.c -- plain, slow, obviously-correct CPU reference for the batched
 * vertex-function forward and backward of Cavs (Zhang et al., "Cavs: A
 * Vertex-centric Programming Interface for Dynamic Neural Networks",
 * arXiv 1712.04048).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark load this file's library.  The product
 * path (the HIP library) never links, calls or executes it, and the two share
 * no source, header, table or helper.
 *
 * Precision: the arithmetic type `real` is fixed at compile time.  The parity
 * build (liboracle.so) uses IEEE fp64; the same source compiled with
 * -DORC_FLOAT (liboracle_f32.so) evaluates the identical definitions in IEEE
 * fp32, which measures how far a plain fp32 evaluation strays from fp64 and
 * is the timed CPU baseline.  Optionally, operands of the matrix products are
 * rounded to bfloat16 (round-to-nearest-even) at the points where a bf16
 * matrix-core path rounds them; see bf().
 *
 * Every function evaluates the plain definition:
 *   - the schedule is the level of each vertex (Section 3.2: a vertex becomes
 *     activated once every vertex it depends on has been evaluated, and all
 *     activated vertices form one task V_t), computed both by the recursive
 *     height and by peeling ready vertices off the graph;
 *   - the forward pass is F evaluated vertex by vertex, children first
 *     (child-sum Tree-LSTM figure of Section 3.1, for any number of child
 *     slots N; Tree-FC cell of Section 5);
 *   - the backward pass is the hand-derived gradient of F applied vertex by
 *     vertex in reverse evaluation order, with gradients accumulated
 *     (Section 3.3, the backward memory rule; Section 3.4, gather/scatter are
 *     each other's gradient).
 *
 * Graphs.  Tree inputs give each vertex at most one parent and list it in
 * parent[].  Graph inputs (the graph-structured RNNs of Section 2, panel (d)
 * of the recurrent-structures figure) pass parent = NULL: a vertex may then
 * be the child of several vertices (or of several slots of one vertex), its
 * state is read by each of them, and its dL/dh and dL/dc are the sums of what
 * each of them sends back.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

#ifdef ORC_FLOAT
typedef float real;
#define R_EXP expf
#define R_LOG logf
#define R_TANH tanhf
#else
typedef double real;
#define R_EXP exp
#define R_LOG log
#define R_TANH tanh
#endif
#define R(x) ((real)(x))

/* status codes (numerically equal to the library's, defined independently) */
#define ORC_OK 0
#define ORC_ERR_ARG (-1)
#define ORC_ERR_RANGE (-2)
#define ORC_ERR_MULTIPARENT (-3)
#define ORC_ERR_CYCLE (-4)
#define ORC_ERR_MISMATCH (-5)
#define ORC_ERR_DUP_PULL (-9)

#define LOSS_CE 0
#define LOSS_L2 1
#define LOSS_NONE 2   /* no loss head: the state is pushed to an external consumer */

/* ------------------------------------------------------------------------ */
/* bf16 emulation: round x to 8 significant bits, ties to even.              */
/* ------------------------------------------------------------------------ */
static int g_bf16 = 0;

static double bf_d(double x) {
  if (x == 0.0 || !isfinite(x)) return x;
  int e;
  double m = frexp(x, &e);           /* x = m * 2^e, 0.5 <= |m| < 1 */
  double r = nearbyint(m * 256.0);   /* 8 significant bits, ties to even */
  return ldexp(r / 256.0, e);
}

/* a bf16 value is exact in float and in double */
static real bf(real x) { return g_bf16 ? (real)bf_d((double)x) : x; }

/* ------------------------------------------------------------------------ */
/* levels by peeling (Section 3.2's activation rule)                         */
/* ------------------------------------------------------------------------ */

/*
 * Every vertex starts with a count of its present child links.  The vertices
 * whose count is zero are ready; they form the first task.  Evaluating a task
 * removes each of its vertices from the counts of the vertices that read it
 * (each child link counts once, so a vertex listed twice by one parent is
 * removed twice); the vertices whose count drops to zero form the next task.
 * The parents of each vertex are found by inverting the child links.
 * level[v] receives v's task index; returns the number of tasks, or -1 when
 * some vertex never becomes ready (the links contain a cycle).
 */
static int peel_levels(int V, int N, const int* child, int* level) {
  int* remaining = (int*)calloc((size_t)V + 1, sizeof(int));
  int* first_in = (int*)malloc(sizeof(int) * ((size_t)V + 2));
  int* readers = (int*)malloc(sizeof(int) * ((size_t)V * N + 1));
  int* fill = (int*)calloc((size_t)V + 1, sizeof(int));
  int* ready = (int*)malloc(sizeof(int) * ((size_t)V + 1));
  /* readers of vertex c (one entry per child link pointing at c) */
  for (int v = 0; v < V; ++v)
    for (int k = 0; k < N; ++k) {
      int c = child[v * N + k];
      if (c >= 0) { ++remaining[v]; ++fill[c]; }
    }
  first_in[0] = 0;
  for (int c = 0; c < V; ++c) first_in[c + 1] = first_in[c] + fill[c];
  for (int c = 0; c < V; ++c) fill[c] = first_in[c];
  for (int v = 0; v < V; ++v)
    for (int k = 0; k < N; ++k) {
      int c = child[v * N + k];
      if (c >= 0) readers[fill[c]++] = v;
    }
  int n_ready = 0, done = 0, t = 0;
  for (int v = 0; v < V; ++v) {
    level[v] = -1;
    if (remaining[v] == 0) ready[n_ready++] = v;
  }
  /* ready[head .. n_ready) holds the current task; vertices freed by it are
     appended behind it and become the next task */
  int head = 0;
  while (head < n_ready) {
    int end = n_ready;
    for (int i = head; i < end; ++i) {
      int v = ready[i];
      level[v] = t;
      ++done;
      for (int e = first_in[v]; e < first_in[v + 1]; ++e)
        if (--remaining[readers[e]] == 0) ready[n_ready++] = readers[e];
    }
    head = end;
    ++t;
  }
  free(remaining); free(first_in); free(readers); free(fill); free(ready);
  return done == V ? t : -1;
}

/* ------------------------------------------------------------------------ */
/* validation                                                                */
/* ------------------------------------------------------------------------ */

/*
 * Checks the input graphs.  When several problems are present the first in
 * this order is reported: RANGE, MULTIPARENT, DUP_PULL, MISMATCH, CYCLE.
 * pull_idx / push_idx may be NULL (no inputs / no loss terms).  parent = NULL
 * declares graph (DAG) inputs: MULTIPARENT and MISMATCH do not apply.
 */
int orc_validate(int V, int N, const int* child, const int* parent,
                 const int* pull_idx, int n_x, const int* push_idx, int n_push) {
  if (V < 0 || N < 1 || n_x < 0 || n_push < 0) return ORC_ERR_ARG;
  for (int v = 0; v < V; ++v) {
    for (int k = 0; k < N; ++k) {
      int c = child[v * N + k];
      if (c < -1 || c >= V) return ORC_ERR_RANGE;
    }
    if (parent && (parent[v] < -1 || parent[v] >= V)) return ORC_ERR_RANGE;
    if (pull_idx && (pull_idx[v] < -1 || pull_idx[v] >= n_x)) return ORC_ERR_RANGE;
    if (push_idx && (push_idx[v] < -1 || push_idx[v] >= n_push)) return ORC_ERR_RANGE;
  }
  int* cnt = (int*)calloc((size_t)(V > n_x ? V : n_x) + 1, sizeof(int));
  int status = ORC_OK;
  if (parent)
    for (int v = 0; v < V && status == ORC_OK; ++v)
      for (int k = 0; k < N; ++k) {
        int c = child[v * N + k];
        if (c >= 0 && ++cnt[c] > 1) { status = ORC_ERR_MULTIPARENT; break; }
      }
  if (status == ORC_OK && pull_idx) {
    memset(cnt, 0, sizeof(int) * ((size_t)(V > n_x ? V : n_x) + 1));
    for (int v = 0; v < V; ++v)
      if (pull_idx[v] >= 0 && ++cnt[pull_idx[v]] > 1) { status = ORC_ERR_DUP_PULL; break; }
  }
  free(cnt);
  if (status != ORC_OK) return status;
  if (parent) {
    /* every child link c -> v must be mirrored by parent[c] == v, and every
       parent pointer must be such a link */
    long links = 0, with_parent = 0;
    for (int v = 0; v < V; ++v) {
      if (parent[v] >= 0) ++with_parent;
      for (int k = 0; k < N; ++k) {
        int c = child[v * N + k];
        if (c < 0) continue;
        ++links;
        if (parent[c] != v) return ORC_ERR_MISMATCH;
      }
    }
    if (links != with_parent) return ORC_ERR_MISMATCH;
  }
  int* level = (int*)malloc(sizeof(int) * ((size_t)V + 1));
  if (peel_levels(V, N, child, level) < 0) status = ORC_ERR_CYCLE;
  free(level);
  return status;
}

/* ------------------------------------------------------------------------ */
/* levels, two independent ways                                              */
/* ------------------------------------------------------------------------ */

static int height_rec(int v, int N, const int* child, int* level) {
  if (level[v] >= 0) return level[v];
  int h = 0, any = 0;
  for (int k = 0; k < N; ++k) {
    int c = child[v * N + k];
    if (c < 0) continue;
    int hc = height_rec(c, N, child, level);
    if (!any || hc + 1 > h) h = hc + 1;
    any = 1;
  }
  level[v] = h;
  return h;
}

/* level[v] = 0 for a vertex without children, else 1 + max over children.
   Returns T = 1 + max level (0 for V = 0).  Input must be valid. */
int orc_levels_recursive(int V, int N, const int* child, int* level) {
  for (int v = 0; v < V; ++v) level[v] = -1;
  int T = 0;
  for (int v = 0; v < V; ++v) {
    int h = height_rec(v, N, child, level);
    if (h + 1 > T) T = h + 1;
  }
  return T;
}

/* The task index at which each vertex becomes activated (Section 3.2,
   Algorithm 1), found by peeling ready vertices (peel_levels).  Returns T,
   or -1 on a cycle. */
int orc_levels_frontier(int V, int N, const int* child, int* level) {
  return peel_levels(V, N, child, level);
}

/*
 * The level-major layout of the dynamic tensors (Section 3.3, Algorithm 2):
 * task V_t occupies positions [level_offsets[t], level_offsets[t+1]); inside a
 * task vertices appear in ascending id.  Also remaps the index arrays to
 * positions and lists the positions that pull an input, ascending.
 * parent = NULL (graph inputs): parent_pos is set to -1 everywhere.
 * mode 0 takes levels from the recursive height, mode 1 from peeling.
 * Returns T, or a negative status.
 */
int orc_schedule(int V, int N, const int* child, const int* parent,
                 const int* pull_idx, const int* push_idx, int mode,
                 int* level, int* order, int* pos, int* child_pos, int* parent_pos,
                 int* pull_pos, int* push_pos, int* level_offsets, int* pull_list,
                 int* n_pull_out) {
  int T = mode == 0 ? orc_levels_recursive(V, N, child, level)
                    : orc_levels_frontier(V, N, child, level);
  if (T < 0) return ORC_ERR_CYCLE;
  int p = 0;
  for (int t = 0; t < T; ++t) {
    level_offsets[t] = p;
    for (int v = 0; v < V; ++v)
      if (level[v] == t) order[p++] = v;
  }
  level_offsets[T] = p;
  for (int q = 0; q < V; ++q) pos[order[q]] = q;
  int np = 0;
  for (int q = 0; q < V; ++q) {
    int v = order[q];
    for (int k = 0; k < N; ++k) {
      int c = child[v * N + k];
      child_pos[q * N + k] = c >= 0 ? pos[c] : -1;
    }
    parent_pos[q] = parent && parent[v] >= 0 ? pos[parent[v]] : -1;
    pull_pos[q] = pull_idx ? pull_idx[v] : -1;
    push_pos[q] = push_idx ? push_idx[v] : -1;
    if (pull_pos[q] >= 0) pull_list[np++] = q;
  }
  *n_pull_out = np;
  return T;
}

/* ------------------------------------------------------------------------ */
/* shared model state                                                        */
/* ------------------------------------------------------------------------ */

typedef struct {
  int V, N, D, H, C, loss_kind, cell;   /* cell 0 = Tree-LSTM, 1 = Tree-FC */
  const int *child, *parent, *pull_idx, *push_idx;
  const real *X, *Y, *Wx, *U, *b, *Ws, *bs;
  real denom;
  /* forward results */
  real *h, *c, *gates, *lossv;
  /* backward */
  const real* dh_ext;   /* [V, H] or NULL: gradient of the pushed states from an
                           external consumer (push connector), added to dL/dh */
  real *dh, *dc;
  real *dWx, *dU, *db, *dWs, *dbs, *dX;
  int do_bwd;
} model_t;

static real sigmoid(real a) {
  if (a >= R(0)) return R(1) / (R(1) + R_EXP(-a));
  real e = R_EXP(a);
  return e / (R(1) + e);
}

/* ---- loss head (the lazily batched push; Section 3.5) ------------------- */
/* Writes this vertex's loss term and adds dL/dh_v into dh[v] (when the
   backward pass is requested). */
static void loss_vertex(model_t* m, int v) {
  int H = m->H, C = m->C;
  int y = m->push_idx ? m->push_idx[v] : -1;
  m->lossv[v] = R(0);
  if (y < 0 || m->loss_kind == LOSS_NONE) return;
  const real* hv = m->h + (size_t)v * H;
  if (m->loss_kind == LOSS_CE) {
    real* z = (real*)malloc(sizeof(real) * C);
    real zmax = -INFINITY;
    for (int c = 0; c < C; ++c) {
      real s = m->bs[c];
      for (int j = 0; j < H; ++j) s += hv[j] * m->Ws[j * C + c];
      z[c] = s;
      if (s > zmax) zmax = s;
    }
    real se = R(0);
    for (int c = 0; c < C; ++c) se += R_EXP(z[c] - zmax);
    real lse = zmax + R_LOG(se);
    m->lossv[v] = lse - z[y];
    if (m->do_bwd) {
      for (int c = 0; c < C; ++c) {
        real dz = (R_EXP(z[c] - lse) - (c == y ? R(1) : R(0))) / m->denom;
        m->dbs[c] += dz;
        for (int j = 0; j < H; ++j) {
          m->dWs[j * C + c] += hv[j] * dz;
          m->dh[(size_t)v * H + j] += dz * m->Ws[j * C + c];
        }
      }
    }
    free(z);
  } else {
    const real* yv = m->Y + (size_t)y * H;
    real s = R(0);
    for (int j = 0; j < H; ++j) {
      real r = hv[j] - yv[j];
      s += r * r;
      if (m->do_bwd) m->dh[(size_t)v * H + j] += r / m->denom;
    }
    m->lossv[v] = R(0.5) * s;
  }
}

/* ---- child-sum Tree-LSTM (figure in Section 3.1) ------------------------ */
/* Parameter columns are ordered [i | f | o | u], each H wide.  The oracle's
   saved gates per vertex are [i | o | u | f_0 .. f_{N-1}]. */
#define GI 0
#define GF 1
#define GO 2
#define GU 3

static void lstm_fwd_vertex(model_t* m, int v) {
  int N = m->N, D = m->D, H = m->H, H4 = 4 * H;
  int row = m->pull_idx ? m->pull_idx[v] : -1;
  const real* x = row >= 0 ? m->X + (size_t)row * D : NULL;
  real* hs = (real*)calloc((size_t)H, sizeof(real));     /* h~ = sum_k h_k */
  real* xw = (real*)calloc((size_t)H4, sizeof(real));    /* x W + b */
  real* a = (real*)calloc((size_t)H4, sizeof(real));     /* i,o,u pre-activations */
  real* af = (real*)calloc((size_t)N * H, sizeof(real)); /* f_k pre-activations */
  for (int col = 0; col < H4; ++col) xw[col] = m->b[col];
  if (x)
    for (int d = 0; d < D; ++d) {
      real xd = bf(x[d]);
      for (int col = 0; col < H4; ++col) xw[col] += xd * bf(m->Wx[(size_t)d * H4 + col]);
    }
  for (int k = 0; k < N; ++k) {
    int ch = m->child[v * N + k];
    if (ch < 0) continue;
    for (int r = 0; r < H; ++r) hs[r] += m->h[(size_t)ch * H + r];
  }
  for (int col = 0; col < H4; ++col) a[col] = xw[col];
  for (int r = 0; r < H; ++r) {
    real hr = bf(hs[r]);
    const real* Ur = m->U + (size_t)r * H4;
    for (int j = 0; j < H; ++j) {
      a[GI * H + j] += hr * bf(Ur[GI * H + j]);
      a[GO * H + j] += hr * bf(Ur[GO * H + j]);
      a[GU * H + j] += hr * bf(Ur[GU * H + j]);
    }
  }
  for (int k = 0; k < N; ++k) {
    int ch = m->child[v * N + k];
    if (ch < 0) continue;
    for (int j = 0; j < H; ++j) af[k * H + j] = xw[GF * H + j];
    for (int r = 0; r < H; ++r) {
      real hr = bf(m->h[(size_t)ch * H + r]);
      const real* Ur = m->U + (size_t)r * H4;
      for (int j = 0; j < H; ++j) af[k * H + j] += hr * bf(Ur[GF * H + j]);
    }
  }
  real* g = m->gates + (size_t)v * (3 + N) * H;
  real* cv = m->c + (size_t)v * H;
  real* hv = m->h + (size_t)v * H;
  for (int j = 0; j < H; ++j) {
    real ig = sigmoid(a[GI * H + j]), og = sigmoid(a[GO * H + j]), ug = R_TANH(a[GU * H + j]);
    real cj = ig * ug;
    for (int k = 0; k < N; ++k) {
      int ch = m->child[v * N + k];
      real fk = R(0);
      if (ch >= 0) {
        fk = sigmoid(af[k * H + j]);
        cj += fk * m->c[(size_t)ch * H + j];
      }
      g[(3 + k) * H + j] = fk;
    }
    g[0 * H + j] = ig;
    g[1 * H + j] = og;
    g[2 * H + j] = ug;
    cv[j] = cj;
    hv[j] = og * R_TANH(cj);
  }
  free(hs);
  free(xw);
  free(a);
  free(af);
}

static void lstm_bwd_vertex(model_t* m, int v) {
  int N = m->N, D = m->D, H = m->H, H4 = 4 * H;
  int row = m->pull_idx ? m->pull_idx[v] : -1;
  const real* x = row >= 0 ? m->X + (size_t)row * D : NULL;
  const real* g = m->gates + (size_t)v * (3 + N) * H;
  const real* cv = m->c + (size_t)v * H;
  const real* gh = m->dh + (size_t)v * H;
  const real* gcin = m->dc + (size_t)v * H;
  real* di = (real*)calloc((size_t)H, sizeof(real));
  real* dO = (real*)calloc((size_t)H, sizeof(real));
  real* du = (real*)calloc((size_t)H, sizeof(real));
  real* gc = (real*)calloc((size_t)H, sizeof(real));
  real* df = (real*)calloc((size_t)N * H, sizeof(real));   /* delta_f_k */
  real* dfs = (real*)calloc((size_t)H, sizeof(real));      /* sum_k delta_f_k */
  real* hs = (real*)calloc((size_t)H, sizeof(real));
  for (int j = 0; j < H; ++j) {
    real ig = g[j], og = g[H + j], ug = g[2 * H + j];
    real tau = R_TANH(cv[j]);
    dO[j] = gh[j] * tau * og * (R(1) - og);
    gc[j] = gcin[j] + gh[j] * og * (R(1) - tau * tau);
    di[j] = gc[j] * ug * ig * (R(1) - ig);
    du[j] = gc[j] * ig * (R(1) - ug * ug);
    for (int k = 0; k < N; ++k) {
      int ch = m->child[v * N + k];
      if (ch < 0) continue;
      real fk = g[(3 + k) * H + j];
      df[k * H + j] = gc[j] * m->c[(size_t)ch * H + j] * fk * (R(1) - fk);
      dfs[j] += df[k * H + j];
    }
  }
  for (int k = 0; k < N; ++k) {
    int ch = m->child[v * N + k];
    if (ch < 0) continue;
    for (int r = 0; r < H; ++r) hs[r] += m->h[(size_t)ch * H + r];
  }
  /* gradient into the children (scatter is the gradient of gather); a child
     read by several vertices sums what each sends back */
  for (int k = 0; k < N; ++k) {
    int ch = m->child[v * N + k];
    if (ch < 0) continue;
    for (int r = 0; r < H; ++r) {
      real s = R(0);
      for (int j = 0; j < H; ++j) {
        s += bf(di[j]) * bf(m->U[(size_t)r * H4 + GI * H + j]);
        s += bf(dO[j]) * bf(m->U[(size_t)r * H4 + GO * H + j]);
        s += bf(du[j]) * bf(m->U[(size_t)r * H4 + GU * H + j]);
      }
      real sf = R(0);
      for (int j = 0; j < H; ++j)
        sf += bf(df[k * H + j]) * bf(m->U[(size_t)r * H4 + GF * H + j]);
      m->dh[(size_t)ch * H + r] += s + sf;
    }
    for (int j = 0; j < H; ++j)
      m->dc[(size_t)ch * H + j] += gc[j] * g[(3 + k) * H + j];
  }
  /* parameter gradients (lazy operators; order does not matter) */
  for (int j = 0; j < H; ++j) {
    m->db[GI * H + j] += di[j];
    m->db[GF * H + j] += dfs[j];
    m->db[GO * H + j] += dO[j];
    m->db[GU * H + j] += du[j];
  }
  for (int r = 0; r < H; ++r) {
    real hr = bf(hs[r]);
    for (int j = 0; j < H; ++j) {
      m->dU[(size_t)r * H4 + GI * H + j] += hr * bf(di[j]);
      m->dU[(size_t)r * H4 + GO * H + j] += hr * bf(dO[j]);
      m->dU[(size_t)r * H4 + GU * H + j] += hr * bf(du[j]);
    }
  }
  for (int k = 0; k < N; ++k) {
    int ch = m->child[v * N + k];
    if (ch < 0) continue;
    for (int r = 0; r < H; ++r) {
      real hr = bf(m->h[(size_t)ch * H + r]);
      for (int j = 0; j < H; ++j)
        m->dU[(size_t)r * H4 + GF * H + j] += hr * bf(df[k * H + j]);
    }
  }
  if (x) {
    real* dxr = m->dX + (size_t)row * D;
    for (int d = 0; d < D; ++d) {
      real xd = bf(x[d]), s = R(0);
      for (int j = 0; j < H; ++j) {
        m->dWx[(size_t)d * H4 + GI * H + j] += xd * bf(di[j]);
        m->dWx[(size_t)d * H4 + GF * H + j] += xd * bf(dfs[j]);
        m->dWx[(size_t)d * H4 + GO * H + j] += xd * bf(dO[j]);
        m->dWx[(size_t)d * H4 + GU * H + j] += xd * bf(du[j]);
        s += bf(di[j]) * bf(m->Wx[(size_t)d * H4 + GI * H + j]);
        s += bf(dfs[j]) * bf(m->Wx[(size_t)d * H4 + GF * H + j]);
        s += bf(dO[j]) * bf(m->Wx[(size_t)d * H4 + GO * H + j]);
        s += bf(du[j]) * bf(m->Wx[(size_t)d * H4 + GU * H + j]);
      }
      dxr[d] = s;
    }
  }
  free(di); free(dO); free(du); free(gc); free(df); free(dfs); free(hs);
}

/* ---- Tree-FC: h = tanh([h_0, .., h_{N-1}] W + b); a leaf's state is its
        input (Section 5, Tree-FC) ----------------------------------------- */
static void fc_fwd_vertex(model_t* m, int v) {
  int N = m->N, H = m->H;
  real* hv = m->h + (size_t)v * H;
  int leaf = 1;
  for (int k = 0; k < N; ++k) if (m->child[v * N + k] >= 0) leaf = 0;
  if (leaf) {
    const real* x = m->X + (size_t)m->pull_idx[v] * H;
    for (int j = 0; j < H; ++j) hv[j] = x[j];
    return;
  }
  real* z = (real*)malloc(sizeof(real) * H);
  for (int j = 0; j < H; ++j) z[j] = m->b[j];
  for (int k = 0; k < N; ++k) {
    int ch = m->child[v * N + k];
    if (ch < 0) continue;
    for (int r = 0; r < H; ++r) {
      real hr = bf(m->h[(size_t)ch * H + r]);
      const real* Wr = m->U + ((size_t)k * H + r) * H;
      for (int j = 0; j < H; ++j) z[j] += hr * bf(Wr[j]);
    }
  }
  for (int j = 0; j < H; ++j) hv[j] = R_TANH(z[j]);
  free(z);
}

static void fc_bwd_vertex(model_t* m, int v) {
  int N = m->N, H = m->H;
  const real* hv = m->h + (size_t)v * H;
  const real* gh = m->dh + (size_t)v * H;
  int leaf = 1;
  for (int k = 0; k < N; ++k) if (m->child[v * N + k] >= 0) leaf = 0;
  if (leaf) {
    real* dx = m->dX + (size_t)m->pull_idx[v] * H;
    for (int j = 0; j < H; ++j) dx[j] = gh[j];
    return;
  }
  real* dl = (real*)malloc(sizeof(real) * H);
  for (int j = 0; j < H; ++j) {
    dl[j] = gh[j] * (R(1) - hv[j] * hv[j]);
    m->db[j] += dl[j];
  }
  for (int k = 0; k < N; ++k) {
    int ch = m->child[v * N + k];
    if (ch < 0) continue;
    for (int r = 0; r < H; ++r) {
      real s = R(0);
      real hr = bf(m->h[(size_t)ch * H + r]);
      for (int j = 0; j < H; ++j) {
        real w = bf(m->U[((size_t)k * H + r) * H + j]);
        s += bf(dl[j]) * w;
        m->dU[((size_t)k * H + r) * H + j] += hr * bf(dl[j]);
      }
      m->dh[(size_t)ch * H + r] += s;
    }
  }
  free(dl);
}

/* ---- drivers ------------------------------------------------------------ */
static void fwd_vertex(model_t* m, int v) {
  if (m->cell == 0) lstm_fwd_vertex(m, v); else fc_fwd_vertex(m, v);
}
static void bwd_vertex(model_t* m, int v) {
  if (m->cell == 0) lstm_bwd_vertex(m, v); else fc_bwd_vertex(m, v);
}

/* Recursive evaluation: children first, each vertex once (a vertex shared by
   several readers is evaluated the first time it is reached); the vertex is
   appended to `post`, the evaluation order. */
static void fwd_rec(model_t* m, int v, char* seen, int* post, int* n_post) {
  if (seen[v]) return;
  seen[v] = 1;
  for (int k = 0; k < m->N; ++k) {
    int ch = m->child[v * m->N + k];
    if (ch >= 0) fwd_rec(m, ch, seen, post, n_post);
  }
  fwd_vertex(m, v);
  post[(*n_post)++] = v;
}

/*
 * Runs forward (+ loss) and, if do_bwd, backward over all graphs.
 *   order_mode 0: recursive per-vertex evaluation from the vertices nobody
 *                 reads (the roots, ascending id), children first; the
 *                 backward visits the vertices in the reverse of that
 *                 evaluation order, so each vertex's dL/dh and dL/dc are
 *                 complete when it is reached;
 *   order_mode 1: Algorithm 1 order -- tasks V_0..V_{T-1} forward, then the
 *                 task stack popped in reverse for backward.
 * denom > 0 overrides the loss normaliser |Lambda| (number of labelled
 * vertices).  Outputs are indexed by vertex id.  Gradient arrays are
 * overwritten.  Returns ORC_OK or a status from orc_validate.
 */
static int run_model(model_t* m, int order_mode, real* loss_out) {
  int V = m->V, N = m->N, H = m->H;
  int n_x = 0;
  if (m->pull_idx)
    for (int v = 0; v < V; ++v) if (m->pull_idx[v] + 1 > n_x) n_x = m->pull_idx[v] + 1;
  int st = orc_validate(V, N, m->child, m->parent, m->pull_idx, n_x, NULL, 0);
  if (st != ORC_OK) return st;
  if (m->cell == 1) {
    for (int v = 0; v < V; ++v) {
      int leaf = 1;
      for (int k = 0; k < N; ++k) if (m->child[v * N + k] >= 0) leaf = 0;
      int has_x = m->pull_idx && m->pull_idx[v] >= 0;
      if (leaf != has_x) return ORC_ERR_ARG;
    }
  }
  if (!(m->denom > R(0))) {
    long nl = 0;
    if (m->push_idx) for (int v = 0; v < V; ++v) nl += m->push_idx[v] >= 0;
    m->denom = nl > 0 ? (real)nl : R(1);
  }
  if (m->do_bwd) {
    memset(m->dh, 0, sizeof(real) * (size_t)V * H);
    memset(m->dc, 0, sizeof(real) * (size_t)V * H);
  }
  int* level = NULL;
  int* post = NULL;
  int T = 0, n_post = 0;
  if (order_mode == 1) {
    level = (int*)malloc(sizeof(int) * ((size_t)V + 1));
    T = orc_levels_frontier(V, N, m->child, level);
    for (int t = 0; t < T; ++t)
      for (int v = 0; v < V; ++v)
        if (level[v] == t) fwd_vertex(m, v);
  } else {
    /* roots: vertices no child link points at */
    char* read = (char*)calloc((size_t)V + 1, 1);
    char* seen = (char*)calloc((size_t)V + 1, 1);
    post = (int*)malloc(sizeof(int) * ((size_t)V + 1));
    for (int v = 0; v < V; ++v)
      for (int k = 0; k < N; ++k)
        if (m->child[v * N + k] >= 0) read[m->child[v * N + k]] = 1;
    for (int v = 0; v < V; ++v)
      if (!read[v]) fwd_rec(m, v, seen, post, &n_post);
    free(read);
    free(seen);
  }
  real L = R(0);
  for (int v = 0; v < V; ++v) {
    loss_vertex(m, v);
    L += m->lossv[v];
  }
  *loss_out = L / m->denom;
  if (m->do_bwd && m->dh_ext)
    for (size_t i = 0; i < (size_t)V * H; ++i) m->dh[i] += m->dh_ext[i];
  if (m->do_bwd) {
    if (order_mode == 1) {
      for (int t = T - 1; t >= 0; --t)
        for (int v = 0; v < V; ++v)
          if (level[v] == t) bwd_vertex(m, v);
    } else {
      for (int i = n_post - 1; i >= 0; --i) bwd_vertex(m, post[i]);
    }
  }
  free(level);
  free(post);
  return ORC_OK;
}

int orc_treelstm(int V, int N, int D, int H, int C, int loss_kind, int bf16, int order_mode,
                 const int* child, const int* parent, const int* pull_idx, const int* push_idx,
                 const real* X, const real* Y, const real* Wx, const real* U,
                 const real* b, const real* Ws, const real* bs, real denom,
                 real* h, real* c, real* gates, real* lossv, real* loss,
                 int do_bwd, real* dh, real* dc, real* dWx, real* dU, real* db,
                 real* dWs, real* dbs, real* dX, const real* dh_ext) {
  model_t m;
  memset(&m, 0, sizeof m);
  m.dh_ext = dh_ext;
  m.V = V; m.N = N; m.D = D; m.H = H; m.C = C; m.loss_kind = loss_kind; m.cell = 0;
  m.child = child; m.parent = parent; m.pull_idx = pull_idx; m.push_idx = push_idx;
  m.X = X; m.Y = Y; m.Wx = Wx; m.U = U; m.b = b; m.Ws = Ws; m.bs = bs; m.denom = denom;
  m.h = h; m.c = c; m.gates = gates; m.lossv = lossv;
  m.do_bwd = do_bwd; m.dh = dh; m.dc = dc;
  m.dWx = dWx; m.dU = dU; m.db = db; m.dWs = dWs; m.dbs = dbs; m.dX = dX;
  if (do_bwd) {
    memset(dWx, 0, sizeof(real) * (size_t)D * 4 * H);
    memset(dU, 0, sizeof(real) * (size_t)H * 4 * H);
    memset(db, 0, sizeof(real) * (size_t)4 * H);
    if (loss_kind == LOSS_CE) {
      memset(dWs, 0, sizeof(real) * (size_t)H * C);
      memset(dbs, 0, sizeof(real) * (size_t)C);
    }
    int n_x = 0;
    if (pull_idx) for (int v = 0; v < V; ++v) if (pull_idx[v] + 1 > n_x) n_x = pull_idx[v] + 1;
    memset(dX, 0, sizeof(real) * (size_t)n_x * D);
  }
  g_bf16 = bf16;
  int st = run_model(&m, order_mode, loss);
  g_bf16 = 0;
  return st;
}

int orc_treefc(int V, int N, int H, int C, int loss_kind, int bf16, int order_mode,
               const int* child, const int* parent, const int* pull_idx, const int* push_idx,
               const real* X, const real* Y, const real* W, const real* b,
               const real* Ws, const real* bs, real denom,
               real* h, real* lossv, real* loss,
               int do_bwd, real* dh, real* dc_scratch, real* dW, real* db,
               real* dWs, real* dbs, real* dX, const real* dh_ext) {
  model_t m;
  memset(&m, 0, sizeof m);
  m.dh_ext = dh_ext;
  m.V = V; m.N = N; m.D = H; m.H = H; m.C = C; m.loss_kind = loss_kind; m.cell = 1;
  m.child = child; m.parent = parent; m.pull_idx = pull_idx; m.push_idx = push_idx;
  m.X = X; m.Y = Y; m.U = W; m.b = b; m.Ws = Ws; m.bs = bs; m.denom = denom;
  m.h = h; m.lossv = lossv;
  m.do_bwd = do_bwd; m.dh = dh; m.dc = dc_scratch;
  m.dU = dW; m.db = db; m.dWs = dWs; m.dbs = dbs; m.dX = dX;
  if (do_bwd) {
    memset(dW, 0, sizeof(real) * (size_t)N * H * H);
    memset(db, 0, sizeof(real) * (size_t)H);
    if (loss_kind == LOSS_CE) {
      memset(dWs, 0, sizeof(real) * (size_t)H * C);
      memset(dbs, 0, sizeof(real) * (size_t)C);
    }
    int n_x = 0;
    if (pull_idx) for (int v = 0; v < V; ++v) if (pull_idx[v] + 1 > n_x) n_x = pull_idx[v] + 1;
    memset(dX, 0, sizeof(real) * (size_t)n_x * H);
  }
  g_bf16 = bf16;
  int st = run_model(&m, order_mode, loss);
  g_bf16 = 0;
  return st;
}

/* exposed for tests of the rounding helper */
double orc_bf16_round(double x) { return bf_d(x); }

/* sizeof(real): lets the loader check which instantiation it opened */
int orc_real_bytes(void) { return (int)sizeof(real); }
