// Generic engine: the child-sum Tree-LSTM (Section 3.1 figure) for any
// number of child slots up to kMaxSlots, over tree inputs or graph inputs
// whose vertices may be read by several vertices (Section 2, the
// graph-structured panel of the recurrent-structures figure).
//
// The fused engine (lstm*.hip) is specialised for at most two slots and one
// reader per vertex.  Here each task V_t is instead evaluated in separate,
// simpler steps, all on MFMA for the products:
//   forward:  h~ rows gathered (sum over present children), the i|o|u
//             products h~ U, one f product per child link (h_k U_f), all
//             written as pre-activations into the saved-gate rows, then an
//             elementwise gates kernel (cell update, scatter of h and c);
//   backward: an elementwise gates kernel forms dA from the vertex's total
//             dL/dh and dL/dc -- the loss head's term plus, for every link
//             that reads the vertex, what that reader sent back, summed in
//             a fixed order (the reader's position, then its slot) -- and
//             the dc it sends to each child; then dh~ = dA_iou U_iou^T and,
//             per child link, dh~ + dA_fk U_f^T into that link's row.
// Every store has one writer (per-link rows instead of a scatter into the
// child), so no atomics are needed and the results are deterministic.  The
// lazy weight-gradient products (Section 3.5) are split-K products over all
// positions or all links with a fixed-order reduction.
//
// The same forward gates kernel finishes the fused engine's levels when its
// gates are unfused for the fusion ablation (CAVS_UNFUSED_FWD_GATES).
#include "lstm_dev.h"

namespace cavs {

namespace {

// --------------------------------------------------------------- addressing
// Where row r of a product operand or result starts (element offset from the
// base), or -1 for an absent row (read as zeros, never stored).
enum RowMode : int {
  RM_DIRECT = 0,       // row0 + r
  RM_CHILD = 1,        // link e = row0 + r: the row of its child (child_pos[e])
  RM_EDGE_FSLOT = 2,   // link e = (p, k): p's row at the f_k block of a gate row
  RM_EDGE_PARENT = 3,  // link e = (p, k): p's row
  RM_PULL_ROW = 4,     // r-th pulling position p: its input row pull_pos[p]
  RM_PULL_POS = 5,     // r-th pulling position p: row p
};

struct RowSel {
  const float* base;
  int ld, mode, row0;
};

struct GenIdx {
  const int* child_pos;
  const int* pull_list;
  const int* pull_pos;
  int N, H;
};

__device__ __forceinline__ int fslot(int k, int H) { return k == 0 ? H : (3 + k) * H; }

__device__ __forceinline__ long long row_off(const RowSel& s, const GenIdx& g, int r) {
  const int i = s.row0 + r;
  switch (s.mode) {
    case RM_DIRECT:
      return (long long)i * s.ld;
    case RM_CHILD: {
      const int c = g.child_pos[i];
      return c < 0 ? -1 : (long long)c * s.ld;
    }
    case RM_EDGE_FSLOT: {
      if (g.child_pos[i] < 0) return -1;
      const int p = i / g.N, k = i - p * g.N;
      return (long long)p * s.ld + fslot(k, g.H);
    }
    case RM_EDGE_PARENT:
      if (g.child_pos[i] < 0) return -1;
      return (long long)(i / g.N) * s.ld;
    case RM_PULL_ROW:
      return (long long)g.pull_pos[g.pull_list[i]] * s.ld;
    case RM_PULL_POS:
      return (long long)g.pull_list[i] * s.ld;
  }
  return -1;
}

constexpr int kGT = 64;            // output tile edge
constexpr int kGK = 32;            // contraction chunk
constexpr int kGLD = kGK + 4;      // LDS row stride of k-contiguous tiles
constexpr int kTLD = kGT + 4;      // LDS row stride of row-major (k-major) tiles
constexpr int kMaxSplits = 16;

// C[rc(r)][c] = (beta ? C0[r0(r)][c] : 0) + sum_k A[ra(r)][k] * BT[c][k]
// for r < R, c < Nc, k < K (K a multiple of 4).  64 x 64 tiles, four
// wavefronts of 32 x 32, K in chunks of 32 staged k-contiguous in LDS.
__global__ void __launch_bounds__(256) k_gen_nt(int R, int Nc, int K, RowSel ra,
                                                const float* __restrict__ BT, int ldb, RowSel rc,
                                                RowSel r0, int beta, GenIdx g) {
  __shared__ __attribute__((aligned(16))) float As[kGT * kGLD];
  __shared__ __attribute__((aligned(16))) float Bs[kGT * kGLD];
  __shared__ long long aoff[kGT];
  const int tid = threadIdx.x;
  const int row_base = blockIdx.x * kGT, col_base = blockIdx.y * kGT;
  if (tid < kGT) {
    const int r = row_base + tid;
    aoff[tid] = r < R ? row_off(ra, g, r) : -1;
  }
  __syncthreads();
  const int w = tid >> 6, wr = (w >> 1) * 32, wc = (w & 1) * 32;
  const int lr = tid >> 3, lk = (tid & 7) * 4;
  v4f acc[2][2];
  zero_acc(acc);
  for (int k0 = 0; k0 < K; k0 += kGK) {
    float4 av[2], bv[2];
    const int kk = k0 + lk;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int row = lr + 32 * h;
      const long long o = aoff[row];
      av[h] = (o >= 0 && kk < K) ? ldg4(ra.base + o + kk) : f4zero();
      const int col = col_base + row;
      bv[h] = (col < Nc && kk < K) ? ldg4(BT + (size_t)col * ldb + kk) : f4zero();
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      st4(&As[(lr + 32 * h) * kGLD + lk], av[h]);
      st4(&Bs[(lr + 32 * h) * kGLD + lk], bv[h]);
    }
    __syncthreads();
    mfma_chunk<2, 2, true, true, kGLD, kGLD>(As, Bs, wr, wc, acc);
  }
  const int lane = tid & 63, gq = lane >> 4, rl = lane & 15;
#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = row_base + wr + 16 * tm + 4 * gq + i;
      if (row >= R) continue;
      const long long co = row_off(rc, g, row);
      if (co < 0) continue;
      long long o0 = 0;
      if (beta) {
        o0 = row_off(r0, g, row);
        if (o0 < 0) continue;
      }
      float* crow = const_cast<float*>(rc.base) + co;
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) {
        const int col = col_base + wc + 16 * tn + rl;
        if (col >= Nc) continue;
        float v = acc[tm][tn][i];
        if (beta) v += r0.base[o0 + col];
        crow[col] = v;
      }
    }
}

// part[s][a][b] = sum over the rows r of split s of A[ra(r)][a] * B[rb(r)][b]
// (a < Ka, b < Nb, both multiples of 4): the split-K half of a lazy product;
// the rows are the contraction index.  Tiles 64 x 64 over (a, b); the rows
// in chunks of 32 staged row-major in LDS.
__global__ void __launch_bounds__(256) k_gen_tn(int R, int Ka, int Nb, RowSel ra, RowSel rb,
                                                GenIdx g, int rows_per_split,
                                                float* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) float As[kGK * kTLD];
  __shared__ __attribute__((aligned(16))) float Bs[kGK * kTLD];
  const int tid = threadIdx.x;
  const int a_base = blockIdx.x * kGT, b_base = blockIdx.y * kGT, split = blockIdx.z;
  const int rbeg = split * rows_per_split, rend = min(R, rbeg + rows_per_split);
  const int w = tid >> 6, wr = (w >> 1) * 32, wc = (w & 1) * 32;
  const int lr = tid >> 4, lc = (tid & 15) * 4;
  v4f acc[2][2];
  zero_acc(acc);
  for (int r0 = rbeg; r0 < rend; r0 += kGK) {
    float4 av[2], bv[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = r0 + lr + 16 * h;
      long long oa = -1, ob = -1;
      if (r < rend) {
        oa = row_off(ra, g, r);
        ob = row_off(rb, g, r);
      }
      const int a = a_base + lc, b = b_base + lc;
      av[h] = (oa >= 0 && ob >= 0 && a < Ka) ? ldg4(ra.base + oa + a) : f4zero();
      bv[h] = (oa >= 0 && ob >= 0 && b < Nb) ? ldg4(rb.base + ob + b) : f4zero();
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      st4(&As[(lr + 16 * h) * kTLD + lc], av[h]);
      st4(&Bs[(lr + 16 * h) * kTLD + lc], bv[h]);
    }
    __syncthreads();
    mfma_chunk<2, 2, false, false, kTLD, kTLD>(As, Bs, wr, wc, acc);
  }
  const int lane = tid & 63, gq = lane >> 4, rl = lane & 15;
  float* out = part + (size_t)split * Ka * Nb;
#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int a = a_base + wr + 16 * tm + 4 * gq + i;
      if (a >= Ka) continue;
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) {
        const int b = b_base + wc + 16 * tn + rl;
        if (b < Nb) out[(size_t)a * Nb + b] = acc[tm][tn][i];
      }
    }
}

// part[s][b] = sum over the rows of split s of B[rb(r)][b], b < Nb.
__global__ void __launch_bounds__(256) k_gen_colsum(int R, int Nb, RowSel rb, GenIdx g,
                                                    int rows_per_split, float* __restrict__ part) {
  const int b = blockIdx.x * 256 + threadIdx.x, split = blockIdx.y;
  if (b >= Nb) return;
  const int rbeg = split * rows_per_split, rend = min(R, rbeg + rows_per_split);
  float s = 0.f;
  for (int r = rbeg; r < rend; ++r) {
    const long long o = row_off(rb, g, r);
    if (o >= 0) s += rb.base[o + b];
  }
  part[(size_t)split * Nb + b] = s;
}

// C[a][b] (= or +=) sum over s = 0 .. S-1 in order of part[s][a][b], for
// b < Nb_out (the partial rows are Nb wide).
__global__ void __launch_bounds__(256) k_gen_reduce(int S, int Ka, int Nb, int Nb_out,
                                                    const float* __restrict__ part, float* C,
                                                    int ldc, int accumulate) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long long)Ka * Nb_out) return;
  const int a = (int)(i / Nb_out), b = (int)(i - (long long)a * Nb_out);
  float s = 0.f;
  for (int k = 0; k < S; ++k) s += part[((size_t)k * Ka + a) * Nb + b];
  float* dst = C + (size_t)a * ldc + b;
  *dst = accumulate ? *dst + s : s;
}

// h~ rows of positions [off, off + M): the sum over present children.
template <int NCH>
__global__ void __launch_bounds__(256) k_gen_hsum(Net n, float* __restrict__ Ht, int off, int M) {
  const int H = n.H, q = H / 4;
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long long)M * q) return;
  const int p = off + (int)(i / q), j0 = 4 * (int)(i % q);
  float4 s = f4zero();
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int c = n.child_pos[(size_t)p * NCH + k];
    if (c >= 0) s = add4(s, ldg4(n.Hs + (size_t)c * H + j0));
  }
  st4(Ht + (size_t)p * H + j0, s);
}

// Forward gates of positions [off, off + M), four units per thread: the
// saved-gate row holds the matrix-product parts of the pre-activations (i,
// f_0, o, u, f_1 .. f_{N-1}; zero when has_product is 0, i.e. leaves); bias
// and pulled term are added with the fused epilogues' association, and the
// row is overwritten with the gate values.
template <int NCH>
__global__ void __launch_bounds__(256) k_gen_fwd_gates(Net n, int off, int M, int has_product) {
  const int H = n.H, q = H / 4;
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long long)M * q) return;
  const int p = off + (int)(idx / q), j0 = 4 * (int)(idx % q);
  float* g = n.Gs + (size_t)p * n.GW + j0;
  const int pr = n.pull_pos[p];
  const float4 zero = f4zero();
  float4 zi = zero, zo = zero, zu = zero;
  if (has_product) {
    zi = ldg4(g);
    zo = ldg4(g + 2 * H);
    zu = ldg4(g + 3 * H);
  }
  const float4 bi = ldg4(n.b + G_I * H + j0), bf = ldg4(n.b + G_F * H + j0);
  const float4 bo = ldg4(n.b + G_O * H + j0), bu = ldg4(n.b + G_U * H + j0);
  float4 pi = zero, pf = zero, po = zero, pu = zero;
  if (pr >= 0) {
    const float* Pp = n.P + (size_t)p * 4 * H + j0;
    pi = ldg4(Pp + G_I * H);
    pf = ldg4(Pp + G_F * H);
    po = ldg4(Pp + G_O * H);
    pu = ldg4(Pp + G_U * H);
  }
  int cp[NCH];
  float4 zf[NCH], cc[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    cp[k] = n.child_pos[(size_t)p * NCH + k];
    zf[k] = (cp[k] >= 0 && has_product) ? ldg4(g + (k == 0 ? H : (3 + k) * H)) : zero;
    cc[k] = cp[k] >= 0 ? ldg4(n.Cs + (size_t)cp[k] * H + j0) : zero;
  }
  auto el = [](const float4& v, int e) { return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w; };
  float ig[4], og[4], ug[4], c[4], h[4], fk[NCH][4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float ai = el(zi, e) + el(bi, e), ao = el(zo, e) + el(bo, e), au = el(zu, e) + el(bu, e);
    if (pr >= 0) {
      ai += el(pi, e);
      ao += el(po, e);
      au += el(pu, e);
    }
    const float fb = pr >= 0 ? el(bf, e) + el(pf, e) : el(bf, e);
    ig[e] = sigmoidf_(ai);
    og[e] = sigmoidf_(ao);
    ug[e] = tanh_(au);
    c[e] = ig[e] * ug[e];
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      fk[k][e] = 0.f;
      if (cp[k] >= 0) {
        fk[k][e] = sigmoidf_(el(zf[k], e) + fb);
        c[e] += fk[k][e] * el(cc[k], e);
      }
    }
    h[e] = og[e] * tanh_(c[e]);
  }
  auto f4 = [](const float (&x)[4]) { return make_float4(x[0], x[1], x[2], x[3]); };
  st4(n.Hs + (size_t)p * H + j0, f4(h));
  st4(n.Cs + (size_t)p * H + j0, f4(c));
  st4(g, f4(ig));
  st4(g + 2 * H, f4(og));
  st4(g + 3 * H, f4(ug));
#pragma unroll
  for (int k = 0; k < NCH; ++k) st4(g + (k == 0 ? H : (3 + k) * H), f4(fk[k]));
  const int v = n.order[p];
  st4(n.h_out + (size_t)v * H + j0, f4(h));
  if (n.c_out) st4(n.c_out + (size_t)v * H + j0, f4(c));
}

// Backward gates of positions [off, off + M), four units per thread.  The
// vertex's dL/dh is the loss head's term plus the rows Eh of the links that
// read it, its dL/dc the sum of their rows Ec: with graph inputs the links
// listed in in_edge[in_off[p] ..] (ascending link id: the reader's
// position, then its slot), for trees the one link of parent_pos[p].
// Writes dA (i, f_0, o, u, f_1 ..), dAx = (d_i, sum_k d_fk, d_o, d_u) for
// the input and bias gradients, and Ec of its own child links.
template <int NCH>
__global__ void __launch_bounds__(256) k_gen_bwd_gates(Net n, GenBufDev b, int off, int M) {
  const int H = n.H, q = H / 4;
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long long)M * q) return;
  const int p = off + (int)(idx / q), j0 = 4 * (int)(idx % q);
  float4 gh = ldg4(n.dHL + (size_t)p * H + j0), gcin = f4zero();
  if (b.in_off) {
    const int e0 = b.in_off[p], e1 = b.in_off[p + 1];
    for (int t = e0; t < e1; ++t) {
      const int e = b.in_edge[t];
      gh = add4(gh, ldg4(b.Eh + (size_t)e * H + j0));
      gcin = add4(gcin, ldg4(b.Ec + (size_t)e * H + j0));
    }
  } else {
    const int par = n.parent_pos[p];
    if (par >= 0) {
      int e = par * NCH;
#pragma unroll
      for (int k = 0; k < NCH; ++k)
        if (n.child_pos[(size_t)par * NCH + k] == p) e = par * NCH + k;
      gh = add4(gh, ldg4(b.Eh + (size_t)e * H + j0));
      gcin = ldg4(b.Ec + (size_t)e * H + j0);
    }
  }
  const float* g = n.Gs + (size_t)p * n.GW + j0;
  const float4 ig4 = ldg4(g), og4 = ldg4(g + 2 * H), ug4 = ldg4(g + 3 * H);
  const float4 c4 = ldg4(n.Cs + (size_t)p * H + j0);
  int cp[NCH];
  float4 fk4[NCH], ck4[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    cp[k] = n.child_pos[(size_t)p * NCH + k];
    fk4[k] = cp[k] >= 0 ? ldg4(g + (k == 0 ? H : (3 + k) * H)) : f4zero();
    ck4[k] = cp[k] >= 0 ? ldg4(n.Cs + (size_t)cp[k] * H + j0) : f4zero();
  }
  auto el = [](const float4& v, int e) { return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w; };
  float di[4], dO[4], du[4], dfs[4], gc[4], df[NCH][4], dck[NCH][4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float ig = el(ig4, e), og = el(og4, e), ug = el(ug4, e), ghe = el(gh, e);
    const float tau = tanh_(el(c4, e));
    dO[e] = ghe * tau * og * (1.f - og);
    gc[e] = el(gcin, e) + ghe * og * (1.f - tau * tau);
    di[e] = gc[e] * ug * ig * (1.f - ig);
    du[e] = gc[e] * ig * (1.f - ug * ug);
    dfs[e] = 0.f;
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const float fk = el(fk4[k], e);
      df[k][e] = cp[k] >= 0 ? gc[e] * el(ck4[k], e) * fk * (1.f - fk) : 0.f;
      dck[k][e] = gc[e] * fk;
      dfs[e] += df[k][e];
    }
  }
  auto f4 = [](const float (&x)[4]) { return make_float4(x[0], x[1], x[2], x[3]); };
  float* da = n.dA + (size_t)p * n.GW + j0;
  st4(da, f4(di));
  st4(da + 2 * H, f4(dO));
  st4(da + 3 * H, f4(du));
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    st4(da + (k == 0 ? H : (3 + k) * H), f4(df[k]));
    if (cp[k] >= 0) st4(b.Ec + ((size_t)p * NCH + k) * H + j0, f4(dck[k]));
  }
  float* dx = b.dAx + (size_t)p * 4 * H + j0;
  st4(dx + G_I * H, f4(di));
  st4(dx + G_F * H, f4(dfs));
  st4(dx + G_O * H, f4(dO));
  st4(dx + G_U * H, f4(du));
}

// ---------------------------------------------------------- the LM head
// A softmax loss over a large vocabulary at every labelled vertex (the LM
// models of Section 5): logits Z = h W_s + b_s by an NT product into the dZ
// rows, then one workgroup per position forms the log-sum-exp and dZ in
// fp64, and dL/dh = dZ W_s^T by a second NT product.

// dst[c][r] = src[r][c] for an R x Cc row-major src.
__global__ void __launch_bounds__(256) k_gen_transpose(const float* __restrict__ src, int R,
                                                       int Cc, float* __restrict__ dst) {
  __shared__ float t[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int y = ty; y < 32; y += 8)
    if (r0 + y < R && c0 + tx < Cc) t[y][tx] = src[(size_t)(r0 + y) * Cc + c0 + tx];
  __syncthreads();
  for (int y = ty; y < 32; y += 8)
    if (c0 + y < Cc && r0 + tx < R) dst[(size_t)(c0 + y) * R + r0 + tx] = t[tx][y];
}

__device__ __forceinline__ double block_reduce(double v, bool is_max, double* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const double x = __shfl_xor(v, o, kWave);
    v = is_max ? fmax(v, x) : v + x;
  }
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  double r = red[0];
  for (int i = 1; i < (int)(blockDim.x >> 6); ++i) r = is_max ? fmax(r, red[i]) : r + red[i];
  return r;
}

// Position p = blockIdx.x: its logits row (dZ[p], C wide) plus b_s; labelled:
// lossv = lse - z_y and (with write_dz) dZ = (softmax - e_y) / |Lambda|;
// unlabelled: lossv = 0, dZ = 0.
__global__ void __launch_bounds__(256) k_lm_softmax(Net n, int write_dz) {
  __shared__ double red[4];
  const int p = blockIdx.x, C = n.C, tid = threadIdx.x;
  float* row = n.dZ + (size_t)p * C;
  const int y = n.push_pos[p];
  const double zy = y >= 0 ? (double)row[y] + (double)n.bs[y] : 0.0;
  double m = -INFINITY;
  for (int c = tid; c < C; c += 256) m = fmax(m, (double)row[c] + (double)n.bs[c]);
  m = block_reduce(m, true, red);
  double se = 0.0;
  for (int c = tid; c < C; c += 256) se += exp((double)row[c] + (double)n.bs[c] - m);
  se = block_reduce(se, false, red);
  const double lse = m + log(se);
  if (tid == 0) n.lossv[p] = y >= 0 ? (float)(lse - zy) : 0.f;
  if (!write_dz) return;
  const double inv = (double)n.inv_denom;
  for (int c = tid; c < C; c += 256) {
    const double z = (double)row[c] + (double)n.bs[c];
    row[c] = y >= 0 ? (float)((exp(z - lse) - (c == y ? 1.0 : 0.0)) * inv) : 0.f;
  }
}

// ----------------------------------------------------------------- launchers
GenIdx gen_idx(const Net& n) { return GenIdx{n.child_pos, n.pull_list, n.pull_pos, n.N, n.H}; }
RowSel sel(const float* base, int ld, int mode = RM_DIRECT, int row0 = 0) {
  return RowSel{base, ld, mode, row0};
}

void gen_nt(const char* name, const Net& n, int R, int Nc, int K, RowSel ra, const float* BT,
            int ldb, RowSel rc, RowSel r0, bool beta, hipStream_t s, int row0_rec = 0) {
  if (R <= 0 || Nc <= 0) return;
  CAVS_LAUNCH_ROWS(name, row0_rec, R, k_gen_nt, dim3(cdiv(R, kGT), cdiv(Nc, kGT)), dim3(256), 0,
                   s, R, Nc, K, ra, BT, ldb, rc, r0, (int)beta, gen_idx(n));
}

// the split count: about 512 workgroups, at least 64 rows per split
int gen_splits(int R, int tiles) {
  int S = cdiv(512, tiles > 0 ? tiles : 1);
  S = S < 1 ? 1 : (S > kMaxSplits ? kMaxSplits : S);
  const int maxS = cdiv(R, 64);
  return S > maxS ? (maxS > 0 ? maxS : 1) : S;
}

// C (ldc; columns < Nb_out) (= or +=) sum_r A_r^T B_r
void gen_tn(const char* name, const Net& n, int R, int Ka, int Nb, int Nb_out, RowSel ra,
            RowSel rb, float* C, int ldc, bool accumulate, float* part, hipStream_t s,
            size_t part_cap = 0) {
  const int tiles = cdiv(Ka, kGT) * cdiv(Nb, kGT);
  int S = gen_splits(R, tiles);
  if (part_cap) {   // at least one split always fits (the scratch is sized for it)
    const size_t fit = part_cap / ((size_t)Ka * Nb);
    if ((size_t)S > fit) S = fit > 0 ? (int)fit : 1;
  }
  const int per = (R > 0 ? cdiv(cdiv(R, S), kGK) : 1) * kGK;
  CAVS_LAUNCH(name, k_gen_tn, dim3(cdiv(Ka, kGT), cdiv(Nb, kGT), S), dim3(256), 0, s, R, Ka, Nb,
              ra, rb, gen_idx(n), per, part);
  CAVS_LAUNCH("k_gen_reduce", k_gen_reduce, dim3(cdiv((long)Ka * Nb_out, 256)), dim3(256), 0, s,
              S, Ka, Nb, Nb_out, (const float*)part, C, ldc, (int)accumulate);
}

void gen_colsum(const Net& n, int R, int Nb, int Nb_out, RowSel rb, float* C, float* part,
                hipStream_t s) {
  const int S = R >= 4096 ? kMaxSplits : (R >= 1024 ? 4 : 1);
  const int per = R > 0 ? cdiv(R, S) : 1;
  CAVS_LAUNCH("k_gen_colsum", k_gen_colsum, dim3(cdiv(Nb, 256), S), dim3(256), 0, s, R, Nb, rb,
              gen_idx(n), per, part);
  CAVS_LAUNCH("k_gen_reduce", k_gen_reduce, dim3(cdiv(Nb_out, 256)), dim3(256), 0, s, S, 1, Nb,
              Nb_out, (const float*)part, C, Nb_out, 0);
}

template <int NCH>
void gen_gates_fwd_t(const Net& n, int off, int M, bool has_product, hipStream_t s) {
  const long long th = (long long)M * (n.H / 4);
  CAVS_LAUNCH_ROWS("k_gen_fwd_gates", off, M, k_gen_fwd_gates<NCH>, dim3(cdiv(th, 256)),
                   dim3(256), 0, s, n, off, M, (int)has_product);
}

template <int NCH>
void gen_gates_bwd_t(const Net& n, const GenBufDev& b, int off, int M, hipStream_t s) {
  const long long th = (long long)M * (n.H / 4);
  CAVS_LAUNCH_ROWS("k_gen_bwd_gates", off, M, k_gen_bwd_gates<NCH>, dim3(cdiv(th, 256)),
                   dim3(256), 0, s, n, b, off, M);
}

template <int NCH>
void gen_hsum_t(const Net& n, float* Ht, int off, int M, hipStream_t s) {
  const long long th = (long long)M * (n.H / 4);
  CAVS_LAUNCH_ROWS("k_gen_hsum", off, M, k_gen_hsum<NCH>, dim3(cdiv(th, 256)), dim3(256), 0, s,
                   n, Ht, off, M);
}

#define CAVS_GEN_DISPATCH(FN, ...)          \
  do {                                      \
    switch (n.N) {                          \
      case 1: FN<1>(__VA_ARGS__); break;    \
      case 2: FN<2>(__VA_ARGS__); break;    \
      case 3: FN<3>(__VA_ARGS__); break;    \
      default: FN<4>(__VA_ARGS__); break;   \
    }                                       \
  } while (0)

}  // namespace

void lstm_fwd_gates(const Net& n, int off, int M, bool has_product, hipStream_t s) {
  if (M <= 0) return;
  CAVS_GEN_DISPATCH(gen_gates_fwd_t, n, off, M, has_product, s);
}

// Forward over tasks 1 .. T-1 (the leaves are finished by lstm_fwd_gates
// after the pull product): h~ gather, the i | o | u and f products into the
// saved-gate rows, then the gates.
void gen_forward_levels(const Net& n, const GenBufDev& b, const int* lo, int T, hipStream_t s) {
  const int H = n.H, N = n.N, GW = n.GW;
  const RowSel none = sel(nullptr, 0);
  for (int t = 1; t < T; ++t) {
    const int off = lo[t], M = lo[t + 1] - lo[t];
    CAVS_GEN_DISPATCH(gen_hsum_t, n, b.Ht, off, M, s);
    gen_nt("k_gen_nt<fwd_i>", n, M, H, H, sel(b.Ht, H, RM_DIRECT, off), n.UT, H,
           sel(n.Gs, GW, RM_DIRECT, off), none, false, s, off);
    gen_nt("k_gen_nt<fwd_ou>", n, M, 2 * H, H, sel(b.Ht, H, RM_DIRECT, off),
           n.UT + (size_t)2 * H * H, H, sel(n.Gs + 2 * H, GW, RM_DIRECT, off), none, false, s,
           off);
    gen_nt("k_gen_nt<fwd_f>", n, M * N, H, H, sel(n.Hs, H, RM_CHILD, off * N),
           n.UT + (size_t)H * H, H, sel(n.Gs, GW, RM_EDGE_FSLOT, off * N), none, false, s, off);
    lstm_fwd_gates(n, off, M, true, s);
  }
}

// Backward: tasks T-1 .. 0 (gates; then, above the leaves, the products
// that send dL/dh to each child link), then the lazy products.
void gen_backward(const Net& n, const GenBufDev& b, const int* lo, int T, int n_pull,
                  float* dU, float* db, float* dWx, float* dX, float* dWs, float* dbs,
                  hipStream_t s) {
  const int H = n.H, N = n.N, GW = n.GW, V = n.V, D = n.D;
  const RowSel none = sel(nullptr, 0);
  for (int t = T - 1; t >= 0; --t) {
    const int off = lo[t], M = lo[t + 1] - lo[t];
    CAVS_GEN_DISPATCH(gen_gates_bwd_t, n, b, off, M, s);
    if (t == 0) continue;
    // dh~ = dA_i U_i^T + dA_ou U_ou^T
    gen_nt("k_gen_nt<bwd_hi>", n, M, H, H, sel(n.dA, GW, RM_DIRECT, off), n.U, 4 * H,
           sel(b.Dt, H, RM_DIRECT, off), none, false, s, off);
    gen_nt("k_gen_nt<bwd_hou>", n, M, H, 2 * H, sel(n.dA + 2 * H, GW, RM_DIRECT, off),
           n.U + 2 * H, 4 * H, sel(b.Dt, H, RM_DIRECT, off), sel(b.Dt, H, RM_DIRECT, off), true,
           s, off);
    // per child link (p, k): dh~_p + dA_fk U_f^T
    gen_nt("k_gen_nt<bwd_f>", n, M * N, H, H, sel(n.dA, GW, RM_EDGE_FSLOT, off * N), n.U + H,
           4 * H, sel(b.Eh, H, RM_DIRECT, off * N), sel(b.Dt, H, RM_EDGE_PARENT, off * N), true,
           s, off);
  }
  const int off1 = T > 1 ? lo[1] : V;
  const int inner = V - off1;
  float* part = b.part;
  // dU: the i, o | u blocks over internal positions (h~ rows), f over child links
  gen_tn("k_gen_tn<dU_i>", n, inner, H, H, H, sel(b.Ht, H, RM_DIRECT, off1),
         sel(n.dA, GW, RM_DIRECT, off1), dU, 4 * H, false, part, s);
  gen_tn("k_gen_tn<dU_ou>", n, inner, H, 2 * H, 2 * H, sel(b.Ht, H, RM_DIRECT, off1),
         sel(n.dA + 2 * H, GW, RM_DIRECT, off1), dU + 2 * H, 4 * H, false, part, s);
  gen_tn("k_gen_tn<dU_f>", n, inner * N, H, H, H, sel(n.Hs, H, RM_CHILD, off1 * N),
         sel(n.dA, GW, RM_EDGE_FSLOT, off1 * N), dU + H, 4 * H, false, part, s);
  if (D > 0 && n_pull > 0) {
    gen_tn("k_gen_tn<dWx>", n, n_pull, D, 4 * H, 4 * H, sel(n.X, D, RM_PULL_ROW),
           sel(b.dAx, 4 * H, RM_PULL_POS), dWx, 4 * H, false, part, s);
    gen_nt("k_gen_nt<dX>", n, n_pull, D, 4 * H, sel(b.dAx, 4 * H, RM_PULL_POS), n.Wx, 4 * H,
           sel(dX, D, RM_PULL_ROW), none, false, s);
  } else if (D > 0) {
    CAVS_LAUNCH("k_gen_reduce", k_gen_reduce, dim3(cdiv((long)D * 4 * H, 256)), dim3(256), 0, s,
                0, D, 4 * H, 4 * H, (const float*)part, dWx, 4 * H, 0);
  }
  gen_colsum(n, V, 4 * H, 4 * H, sel(b.dAx, 4 * H), db, part, s);
  if (n.loss == CAVS_LOSS_CE) {
    gen_tn("k_gen_tn<dWs>", n, V, H, n.CP, n.C, sel(n.Hs, H), sel(n.dZ, n.CP), dWs, n.C, false,
           part, s, b.part_cap);
    gen_colsum(n, V, n.CP, n.C, sel(n.dZ, n.CP), dbs, part, s);
  }
}

size_t gen_part_floats(int D, int H, int CP) {
  size_t m = (size_t)2 * H * H;
  if ((size_t)D * 4 * H > m) m = (size_t)D * 4 * H;
  const int cs = CP < 4 ? 4 : (CP > 16 ? 16 : CP);
  if ((size_t)H * cs > m) m = (size_t)H * cs;
  if ((size_t)4 * H > m) m = (size_t)4 * H;
  size_t total = m * kMaxSplits;
  if (CP > 16) {   // LM head: dW_s in one split, db_s in up to kMaxSplits
    const size_t lm = (size_t)H * CP + (size_t)kMaxSplits * CP;
    if (lm > total) total = lm;
  }
  return total;
}

void lm_head_fwd(const Net& n, hipStream_t s) {
  const int H = n.H, C = n.C, V = n.V;
  const RowSel none = sel(nullptr, 0);
  CAVS_LAUNCH("k_gen_transpose", k_gen_transpose, dim3(cdiv(C, 32), cdiv(H, 32)), dim3(256), 0,
              s, n.Ws, H, C, n.WsT);
  gen_nt("k_gen_nt<lm_logits>", n, V, C, H, sel(n.Hs, H), n.WsT, H, sel(n.dZ, C), none, false,
         s);
  CAVS_LAUNCH("k_lm_softmax", k_lm_softmax, dim3(V), dim3(256), 0, s, n, (int)(n.dHL != nullptr));
  if (n.dHL)
    gen_nt("k_gen_nt<lm_dh>", n, V, H, C, sel(n.dZ, C), n.Ws, C, sel(n.dHL, H), none, false, s);
}

void lm_head_grads(const Net& n, float* dWs, float* dbs, float* part, size_t part_cap,
                   hipStream_t s) {
  const int H = n.H, C = n.C, V = n.V;
  gen_tn("k_gen_tn<lm_dWs>", n, V, H, C, C, sel(n.Hs, H), sel(n.dZ, C), dWs, C, false, part, s,
         part_cap);
  gen_colsum(n, V, C, C, sel(n.dZ, C), dbs, part, s);
}

}  // namespace cavs
