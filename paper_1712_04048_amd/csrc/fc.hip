// Tree-FC vertex function (Section 5, Tree-FC: a single fully-connected layer
// as the cell): internal vertex h = tanh(h_0 W_0 + h_1 W_1 + b); a leaf's
// state is its pulled input.  One batching task (level) per launch.
//
// Level products.  Levels of at least kTileMinRows positions run LDS-ring
// tiles (the staging scheme of the Tree-LSTM tiles, lds_ring.h): per 32-deep
// chunk of the hidden index, a stage holds the tile's child rows of every
// slot and the matching rows of each slot's weight block, so the K = N H
// contraction runs as H / 32 chunks with one MFMA block per slot.  Smaller
// levels run split-K kernels (16 x 16 outputs per workgroup, the contraction
// split over its wavefronts).  In both the weight fragment is the MFMA's A
// operand, so lane (r, gq) ends up holding four consecutive columns of one
// position (float4 epilogue accesses).
//
// Backward: a vertex has one parent, so the parent's level product is its
// whole dL/dh from above; the product's epilogue adds the child's loss term
// and stores the child's delta (or a leaf's input gradient) directly.  Roots
// get theirs from one elementwise kernel before the first level.
#include "lds_ring.h"
#include "lstm_dev.h"

namespace cavs {
namespace {

__global__ void __launch_bounds__(256) k_fc_leaf(Net n, int off, int M) {
  const int H4 = n.H / 4;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)M * H4) return;
  const int p = off + (int)(idx / H4), j = 4 * (int)(idx % H4);
  const float4 h = ldg4(n.X + (size_t)n.pull_pos[p] * n.H + j);
  st4(n.Hs + (size_t)p * n.H + j, h);
  st4(n.h_out + (size_t)n.order[p] * n.H + j, h);
}

// dL/dh of position p from above is g; with p's own loss term it gives
// delta = dL/dh (1 - h^2), or, for a leaf (h = x), the gradient of its
// input row.
__device__ __forceinline__ void fc_finish_grad(const Net& n, int p, int col0, float4 g) {
  const size_t e = (size_t)p * n.H + col0;
  const float4 l = ldg4(n.dHL + e);
  g.x += l.x; g.y += l.y; g.z += l.z; g.w += l.w;
  if (p < n.leaf_end) {
    st4(n.dX + (size_t)n.pull_pos[p] * n.H + col0, g);
    return;
  }
  const float4 h = ldg4(n.Hs + e);
  st4(n.dA + e, make_float4(g.x * (1.f - h.x * h.x), g.y * (1.f - h.y * h.y),
                            g.z * (1.f - h.z * h.z), g.w * (1.f - h.w * h.w)));
}

// Roots (no parent, at any level): the gradient from the loss term alone,
// four units per thread.
__global__ void __launch_bounds__(256) k_fc_bwd_roots(Net n) {
  const int H4 = n.H / 4;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)n.V * H4) return;
  const int p = (int)(idx / H4);
  if (n.parent_pos[p] >= 0) return;
  fc_finish_grad(n, p, 4 * (int)(idx % H4), make_float4(0.f, 0.f, 0.f, 0.f));
}

// WT[k][n][j] = U[k H + j][n]: each slot's [H, H] block of the Tree-FC
// weight transposed, so that the forward's weight rows are contiguous in the
// contraction index.  Block (0, 0) also clears the zero row read for absent
// children and for rows past a level.
__global__ void __launch_bounds__(256) k_fc_transpose(const float* __restrict__ U,
                                                      float* __restrict__ WT,
                                                      float* __restrict__ zrow, int H) {
  __shared__ float t[32][33];
  const int n0 = blockIdx.x * 32, r0 = blockIdx.y * 32;   // r0: row of U in [0, N H)
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  if (blockIdx.x == 0 && blockIdx.y == 0)
    for (int j = threadIdx.x; j < H; j += 256) zrow[j] = 0.f;
  for (int y = ty; y < 32; y += 8) t[y][tx] = U[(size_t)(r0 + y) * H + n0 + tx];
  __syncthreads();
  const int k = r0 / H, j0 = r0 % H;   // 32 | H: a block stays inside one slot
  for (int y = ty; y < 32; y += 8) WT[((size_t)k * H + n0 + y) * H + j0 + tx] = t[tx][y];
}

// Forward tile: BM positions x BN units; per chunk the stage holds, for each
// slot k, the BM child rows h_k (a zero row where a child is absent or past
// the level) and the BN rows of W_k^T; z = sum_k h_k W_k, then tanh(z + b).
template <int NCH, int BM, int BN, int S>
__global__ void __launch_bounds__(256) k_fc_fwd_tile(Net n, int off, int M) {
  constexpr int TM = BM / 32, TN = BN / 32;    // 16 x 16 blocks per wavefront
  // copies interleaved with the MFMAs: measured faster for 64 x 64 tiles,
  // slower for 32 x 32
  constexpr bool ILV = BM >= 64 && S == 2;
  constexpr int AROWS = NCH * BM, ROWS = AROWS + NCH * BN;
  constexpr int IPW = ROWS / 32;               // copies per wavefront per chunk
  static_assert(IPW * 32 == ROWS && S >= 2 && S <= 4, "tile shape");
  __shared__ __attribute__((aligned(1024))) float L0[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L1[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L2[S > 2 ? ROWS * 32 : 4];
  __shared__ __attribute__((aligned(1024))) float L3[S > 3 ? ROWS * 32 : 4];
  const Ring<ROWS, S> ring{L0, L1, L2, L3};

  const int H = n.H;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w & 1, wn = w >> 1;
  int rt, ut;
  xcd_tile(H / BN, rt, ut);
  const int row0 = off + rt * BM, rowend = off + M, n0 = ut * BN;

  // epilogue operands, fetched before the product
  int vout[TM];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int p = row0 + wr * (BM / 2) + tm * 16 + r;
    vout[tm] = p < rowend ? n.order[p] : -1;
  }
  float4 bias[TN];
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) bias[tn] = ldg4(n.b + n0 + wn * (BN / 2) + tn * 16 + 4 * gq);

  // LDS rows [0, AROWS): child rows, slot k of position row0 + rr at k BM + rr;
  // then NCH blocks of BN rows of W_k^T
  const float* src[IPW];
#pragma unroll
  for (int t = 0; t < IPW; ++t) {
    const int row = (w * IPW + t) * 8 + (lane >> 3), qg = (lane & 7) ^ (row & 7);
    const float* ptr;
    if (row < AROWS) {
      const int k = row / BM, p = row0 + row % BM;
      ptr = n.zrow;
      if (p < rowend) {
        const int cp = n.child_pos[(size_t)p * NCH + k];
        if (cp >= 0) ptr = n.Hs + (size_t)cp * H;
      }
    } else {
      const int b = row - AROWS, k = b / BN, u = n0 + b % BN;
      ptr = n.UT + ((size_t)k * H + u) * H;
    }
    src[t] = ptr + 4 * qg;
  }
  const int wofs = __builtin_amdgcn_readfirstlane(w * IPW * 256);

  v4f acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = v4f{0.f, 0.f, 0.f, 0.f};

  auto issue = [&](auto sc, int c) {
    ring_issue<IPW, ILV>(ring.at(sc), wofs, [&](int t) { return src[t] + c * kBK; });
  };
  struct Frag {
    float a[NCH][TM][8], b[NCH][TN][8];
  };
  auto read = [&](const float* Ls, Frag& f) {
#pragma unroll
    for (int k = 0; k < NCH; ++k)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        frag_sw(Ls, AROWS + k * BN + wn * (BN / 2) + tn * 16 + r, gq, f.b[k][tn]);
#pragma unroll
    for (int k = 0; k < NCH; ++k)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) frag_sw(Ls, k * BM + wr * (BM / 2) + tm * 16 + r, gq, f.a[k][tm]);
  };
  // A = weight fragment (units), B = child fragment (positions)
  auto mma = [&](const Frag& f) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int k = 0; k < NCH; ++k) acc[tm][tn] = mfma_chunk8<false>(f.b[k][tn], f.a[k][tm], acc[tm][tn]);
  };
  auto body = [&](const float* Lnext, Frag& cur, Frag& nxt, int) {
    read(Lnext, nxt);
    mma(cur);
    ring_schedule<ILV, IPW, 2 * NCH * (TN + TM), TM * TN * NCH * 8>();
  };
  ring_loop_db<S, IPW, Frag, ILV>(H / kBK, ring, issue, read, body);

#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int p = row0 + wr * (BM / 2) + tm * 16 + r;
    if (p >= rowend) continue;
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int col0 = n0 + wn * (BN / 2) + tn * 16 + 4 * gq;
      const float4 h = make_float4(tanh_(acc[tm][tn][0] + bias[tn].x), tanh_(acc[tm][tn][1] + bias[tn].y),
                                   tanh_(acc[tm][tn][2] + bias[tn].z), tanh_(acc[tm][tn][3] + bias[tn].w));
      st4(n.Hs + (size_t)p * H + col0, h);
      st4(n.h_out + (size_t)vout[tm] * H + col0, h);
    }
  }
}

// Backward tile: dL/dh_k = delta W_k^T over BM positions x BN columns j of
// every slot; per chunk of the unit index the stage holds the BM delta rows
// (rows past the level repeat its last row; their products are never
// stored) and, for each slot k, rows k H + j of U (contiguous in the unit
// index).  Each slot's result finishes its child's gradient (trees: one
// writer per row).
template <int NCH, int BM, int BN, int S>
__global__ void __launch_bounds__(256) k_fc_bwd_tile(Net n, int off, int M) {
  constexpr int TM = BM / 32, TN = BN / 32;
  constexpr bool ILV = BM >= 64 && S == 2;   // as in the forward tile
  constexpr int ROWS = BM + NCH * BN;
  constexpr int IPW = ROWS / 32;
  static_assert(IPW * 32 == ROWS && S >= 2 && S <= 4, "tile shape");
  __shared__ __attribute__((aligned(1024))) float L0[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L1[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L2[S > 2 ? ROWS * 32 : 4];
  __shared__ __attribute__((aligned(1024))) float L3[S > 3 ? ROWS * 32 : 4];
  const Ring<ROWS, S> ring{L0, L1, L2, L3};

  const int H = n.H;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w & 1, wn = w >> 1;
  int rt, ut;
  xcd_tile(H / BN, rt, ut);
  const int row0 = off + rt * BM, rowend = off + M, n0 = ut * BN;

  int cpos[TM][NCH];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int p = row0 + wr * (BM / 2) + tm * 16 + r;
#pragma unroll
    for (int k = 0; k < NCH; ++k) cpos[tm][k] = p < rowend ? n.child_pos[(size_t)p * NCH + k] : -1;
  }

  const float* src[IPW];
#pragma unroll
  for (int t = 0; t < IPW; ++t) {
    const int row = (w * IPW + t) * 8 + (lane >> 3), qg = (lane & 7) ^ (row & 7);
    const float* ptr;
    if (row < BM) {
      ptr = n.dA + (size_t)min(row0 + row, rowend - 1) * H;
    } else {
      const int b = row - BM, k = b / BN, j = n0 + b % BN;
      ptr = n.U + ((size_t)k * H + j) * H;
    }
    src[t] = ptr + 4 * qg;
  }
  const int wofs = __builtin_amdgcn_readfirstlane(w * IPW * 256);

  v4f acc[TM][TN][NCH];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int k = 0; k < NCH; ++k) acc[tm][tn][k] = v4f{0.f, 0.f, 0.f, 0.f};

  auto issue = [&](auto sc, int c) {
    ring_issue<IPW, ILV>(ring.at(sc), wofs, [&](int t) { return src[t] + c * kBK; });
  };
  struct Frag {
    float a[TM][8], b[NCH][TN][8];
  };
  auto read = [&](const float* Ls, Frag& f) {
#pragma unroll
    for (int k = 0; k < NCH; ++k)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        frag_sw(Ls, BM + k * BN + wn * (BN / 2) + tn * 16 + r, gq, f.b[k][tn]);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) frag_sw(Ls, wr * (BM / 2) + tm * 16 + r, gq, f.a[tm]);
  };
  auto mma = [&](const Frag& f) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int k = 0; k < NCH; ++k)
          acc[tm][tn][k] = mfma_chunk8<false>(f.b[k][tn], f.a[tm], acc[tm][tn][k]);
  };
  auto body = [&](const float* Lnext, Frag& cur, Frag& nxt, int) {
    read(Lnext, nxt);
    mma(cur);
    ring_schedule<ILV, IPW, 2 * (NCH * TN + TM), TM * TN * NCH * 8>();
  };
  ring_loop_db<S, IPW, Frag, ILV>(H / kBK, ring, issue, read, body);

#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int col0 = n0 + wn * (BN / 2) + tn * 16 + 4 * gq;
#pragma unroll
      for (int k = 0; k < NCH; ++k) {
        const int cp = cpos[tm][k];
        if (cp >= 0)
          fc_finish_grad(n, cp, col0,
                         make_float4(acc[tm][tn][k][0], acc[tm][tn][k][1], acc[tm][tn][k][2], acc[tm][tn][k][3]));
      }
    }
}

// Split-K kernels for levels below the tile threshold: a workgroup owns 16
// positions x 16 units (forward) or 16 positions x 16 columns of every slot
// (backward); wavefront w multiplies the w-th share of the 32-deep chunks of
// the contraction with fragments loaded straight from global memory (the
// weight rows k-contiguous: W^T for the forward, U for the backward), and
// wavefront 0 sums the KW partial blocks in a fixed order (deterministic)
// and finishes.
template <int NCH, int KW>
__global__ void __launch_bounds__(64 * KW) k_fc_fwd_sk(Net n, int off, int M) {
  __shared__ float4 red[KW][64];
  const int H = n.H;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  int rt, ut;
  xcd_tile(H / 16, rt, ut);
  const int row0 = off + rt * 16, rowend = off + M, u0 = ut * 16;
  const int p = row0 + r;
  const float* ap[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int cp = p < rowend ? n.child_pos[(size_t)p * NCH + k] : -1;
    ap[k] = cp >= 0 ? n.Hs + (size_t)cp * H : n.zrow;
  }
  const float* bp = n.UT + (size_t)(u0 + r) * H;
  const int nch = NCH * H / kBK, c0 = w * nch / KW, c1 = (w + 1) * nch / KW;
  struct Frag {
    float a[8], b[8];
  };
  auto load = [&](int c, Frag& f) {
    const int k = c * kBK, slot = k / H, kk = k - slot * H + 8 * gq;
    ld8((slot == 0 ? ap[0] : ap[NCH - 1]) + kk, f.a);
    ld8(bp + (size_t)slot * H * H + kk, f.b);
  };
  v4f acc{0.f, 0.f, 0.f, 0.f};
  Frag fa, fb;
  if (c0 < c1) load(c0, fa);
  for (int c = c0; c < c1; c += 2) {
    if (c + 1 < c1) load(c + 1, fb);
    __builtin_amdgcn_sched_barrier(0);
    acc = mfma_chunk8<false>(fa.b, fa.a, acc);
    if (c + 1 >= c1) break;
    if (c + 2 < c1) load(c + 2, fa);
    acc = mfma_chunk8<false>(fb.b, fb.a, acc);
  }
  red[w][lane] = make_float4(acc[0], acc[1], acc[2], acc[3]);
  __syncthreads();
  if (w != 0 || p >= rowend) return;
  float4 z = red[0][lane];
#pragma unroll
  for (int q = 1; q < KW; ++q) {
    const float4 t = red[q][lane];
    z.x += t.x; z.y += t.y; z.z += t.z; z.w += t.w;
  }
  const int col0 = u0 + 4 * gq;
  const float4 bias = ldg4(n.b + col0);
  const float4 h = make_float4(tanh_(z.x + bias.x), tanh_(z.y + bias.y), tanh_(z.z + bias.z),
                               tanh_(z.w + bias.w));
  st4(n.Hs + (size_t)p * H + col0, h);
  st4(n.h_out + (size_t)n.order[p] * H + col0, h);
}

template <int NCH, int KW>
__global__ void __launch_bounds__(64 * KW) k_fc_bwd_sk(Net n, int off, int M) {
  __shared__ float4 red[KW][NCH][64];
  const int H = n.H;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  int rt, ut;
  xcd_tile(H / 16, rt, ut);
  const int row0 = off + rt * 16, rowend = off + M, j0 = ut * 16;
  const int p = row0 + r;
  // rows past the level read its last delta row (never stored)
  const float* ap = n.dA + (size_t)min(p, rowend - 1) * H;
  const float* bp[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) bp[k] = n.U + ((size_t)k * H + j0 + r) * H;
  const int nch = H / kBK, c0 = w * nch / KW, c1 = (w + 1) * nch / KW;
  struct Frag {
    float a[8], b[NCH][8];
  };
  auto load = [&](int c, Frag& f) {
    const int kk = c * kBK + 8 * gq;
    ld8(ap + kk, f.a);
#pragma unroll
    for (int k = 0; k < NCH; ++k) ld8(bp[k] + kk, f.b[k]);
  };
  v4f acc[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) acc[k] = v4f{0.f, 0.f, 0.f, 0.f};
  auto mma = [&](const Frag& f) {
#pragma unroll
    for (int k = 0; k < NCH; ++k) acc[k] = mfma_chunk8<false>(f.b[k], f.a, acc[k]);
  };
  Frag fa, fb;
  if (c0 < c1) load(c0, fa);
  for (int c = c0; c < c1; c += 2) {
    if (c + 1 < c1) load(c + 1, fb);
    __builtin_amdgcn_sched_barrier(0);
    mma(fa);
    if (c + 1 >= c1) break;
    if (c + 2 < c1) load(c + 2, fa);
    mma(fb);
  }
#pragma unroll
  for (int k = 0; k < NCH; ++k) red[w][k][lane] = make_float4(acc[k][0], acc[k][1], acc[k][2], acc[k][3]);
  __syncthreads();
  if (w != 0 || p >= rowend) return;
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int cp = n.child_pos[(size_t)p * NCH + k];
    if (cp < 0) continue;
    float4 z = red[0][k][lane];
#pragma unroll
    for (int q = 1; q < KW; ++q) {
      const float4 t = red[q][k][lane];
      z.x += t.x; z.y += t.y; z.z += t.z; z.w += t.w;
    }
    fc_finish_grad(n, cp, j0 + 4 * gq, z);
  }
}

}  // namespace

void fc_fwd_leaf(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  CAVS_LAUNCH_ROWS("k_fc_leaf", off, M, k_fc_leaf, dim3(cdiv((long)M * (n.H / 4), 256)), dim3(256), 0, s,
                   n, off, M);
}

void fc_transpose(const Net& n, hipStream_t s) {
  CAVS_LAUNCH("k_fc_transpose", k_fc_transpose, dim3(n.H / 32, n.N * n.H / 32), dim3(256), 0, s, n.U,
              n.UT, n.zrow, n.H);
}

#define CAVS_FC_TILE(KIND, NCH, BM, BN, S)                                                  \
  CAVS_LAUNCH_ROWS("k_fc_" #KIND "_tile<" #NCH ", " #BM ", " #BN ", " #S ">", off, M,        \
                   (k_fc_##KIND##_tile<NCH, BM, BN, S>), dim3(cdiv(M, BM) * (n.H / BN)),     \
                   dim3(256), 0, s, n, off, M)

#define CAVS_FC_SK(KIND, NCH, KW)                                                           \
  CAVS_LAUNCH_ROWS("k_fc_" #KIND "_sk<" #NCH ", " #KW ">", off, M, (k_fc_##KIND##_sk<NCH, KW>), \
                   dim3(cdiv(M, 16) * (n.H / 16)), dim3(64 * KW), 0, s, n, off, M)

// Variant by level size, measured on MI355X (H = 512): split-K below
// kTileMinRows positions, 32 x 32 tiles up to 4096, 64 x 64 tiles above.
// 0: split-K, 1: 32 x 32 tile, 2: 64 x 64 tile
static int fc_variant(int M) {
  return M > 4096 ? 2 : M >= kTileMinRows ? 1 : 0;
}

#define CAVS_FC_LEVEL(KIND)                                                                 \
  do {                                                                                      \
    const int var = fc_variant(M);                                                          \
    if (n.N == 2) {                                                                         \
      if (var == 2) CAVS_FC_TILE(KIND, 2, 64, 64, 2);                                       \
      else if (var == 1) CAVS_FC_TILE(KIND, 2, 32, 32, 2);                                  \
      else CAVS_FC_SK(KIND, 2, 8);                                                          \
    } else {                                                                                \
      if (var == 2) CAVS_FC_TILE(KIND, 1, 64, 64, 2);                                       \
      else if (var == 1) CAVS_FC_TILE(KIND, 1, 32, 32, 2);                                  \
      else CAVS_FC_SK(KIND, 1, 8);                                                          \
    }                                                                                       \
  } while (0)

void fc_fwd_level(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  CAVS_FC_LEVEL(fwd);
}

void fc_bwd_roots(const Net& n, hipStream_t s) {
  if (n.V <= 0) return;
  CAVS_LAUNCH("k_fc_bwd_roots", k_fc_bwd_roots, dim3(cdiv((long)n.V * (n.H / 4), 256)), dim3(256), 0,
              s, n);
}

void fc_bwd_level(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  CAVS_FC_LEVEL(bwd);
}

}  // namespace cavs
