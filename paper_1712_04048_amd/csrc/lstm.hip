// Child-sum Tree-LSTM vertex function F and its gradient dF, one batching
// task (level) per launch (Algorithm 1; F as in the Tree-LSTM figure of
// Section 3.1).
//
// Forward, level t >= 1 (every vertex has a child): one kernel gathers the
// children's h rows straight from the level-major state buffer into LDS (the
// gather of Algorithm 2 fused into the operand load), forms h~ = h_0 + h_1 in
// registers, runs the five products h~ U_i, h~ U_o, h~ U_u, h_0 U_f, h_1 U_f
// on the matrix cores, and applies the gates, the cell update and the scatter
// of (c, h) in the epilogue (the elementwise fusion of Section 3.5).  The
// pulled-input term x W_x was produced beforehand by one GEMM over all
// vertices (pull is eager).  Level 0 (leaves) is elementwise.
//
// Backward, reverse level order: one GEMM kernel per level computes
// dL/dh_k = dA_iou U_iou^T + dA_fk U_f^T for every child k.  A vertex has one
// parent, so that product is the child's whole dL/dh: the epilogue turns it
// (with the dL/dc scattered earlier and the child's own loss term) into the
// child's pre-activation gradients dA, kept level-major for the lazy weight
// gradients, and scatters dL/dc_k' = g_c * f_k' to the grandchildren.  Roots
// are handled by one kernel before the level loop.  Every child row is
// written by exactly one thread: plain stores, no atomics.
#include <stdlib.h>

#include <map>

#include "lstm_dev.h"

namespace cavs {
namespace {

// ------------------------------------------------------------------ forward
__global__ void __launch_bounds__(256) k_lstm_leaf(Net n, int off, int M, int skip_pulled) {
  const int H = n.H;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)M * H) return;
  const int p = off + (int)(idx / H), j = (int)(idx % H);
  const int pr = n.pull_pos[p];
  if (skip_pulled && pr >= 0) return;   // finished by the pull product
  float ai = n.b[G_I * H + j], ao = n.b[G_O * H + j], au = n.b[G_U * H + j];
  if (pr >= 0) {
    const float* Pp = n.P + (size_t)p * 4 * H;
    ai += Pp[G_I * H + j];
    ao += Pp[G_O * H + j];
    au += Pp[G_U * H + j];
  }
  const float i = sigmoidf_(ai), o = sigmoidf_(ao), u = tanh_(au);
  const float c = i * u, h = o * tanh_(c);
  n.Hs[(size_t)p * H + j] = h;
  n.Cs[(size_t)p * H + j] = c;
  // a leaf has no forget gates: their saved columns are never read
  if (n.Gs) {   // null in inference
    float* g = n.Gs + (size_t)p * n.GW;
    g[j] = i;
    g[2 * H + j] = o;
    g[3 * H + j] = u;
  }
  const int v = n.order[p];
  n.h_out[(size_t)v * H + j] = h;
  if (n.c_out) n.c_out[(size_t)v * H + j] = c;
}

// dA of every position of a level below n.fuse_from (dL/dh, dL/dc stored by
// the parent; zero at a root), four consecutive units per thread with
// 16-byte accesses; with wb also its bf16 copy dAb (the operand rows of the
// bf16 backward product, rounded as that product rounds them).  LEAF:
// the level is the leaves (no children).  Loads are unconditional (a root's
// parent terms and an absent child's state read stale rows, masked by
// selects), and each element's arithmetic is that of lstm_gates_fin.
template <int NCH, bool LEAF>
__global__ void __launch_bounds__(256) k_lstm_bwd_gates4(Net n, int off, int M, int wb) {
  const int H = n.H, Hq = H / 4;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)M * Hq) return;
  const int p = off + (int)(idx / Hq), j0 = 4 * (int)(idx % Hq);
  const size_t row = (size_t)p * H + j0;
  const bool root = n.parent_pos[p] < 0;
  const float* g = n.Gs + (size_t)p * n.GW + j0;
  const float4 ig4 = ldg4(g), og4 = ldg4(g + 2 * H), ug4 = ldg4(g + 3 * H);
  const float4 c4 = ldg4(n.Cs + row), lg4 = ldg4(n.dHL + row);
  const float4 gh4 = ldg4(n.dHp + row), gi4 = ldg4(n.dCp + row);
  int cp[NCH];
  float4 fk4[NCH], ck4[NCH];
  if constexpr (!LEAF) {
#pragma unroll
    for (int k = 0; k < NCH; ++k) cp[k] = n.child_pos[(size_t)p * NCH + k];
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      fk4[k] = ldg4(g + (k == 0 ? H : 4 * H));
      ck4[k] = ldg4(n.Cs + (size_t)max(cp[k], 0) * H + j0);
    }
  }
  const float ig[4] = {ig4.x, ig4.y, ig4.z, ig4.w}, og[4] = {og4.x, og4.y, og4.z, og4.w};
  const float ug[4] = {ug4.x, ug4.y, ug4.z, ug4.w}, cc[4] = {c4.x, c4.y, c4.z, c4.w};
  const float lg[4] = {lg4.x, lg4.y, lg4.z, lg4.w};
  const float ghp[4] = {gh4.x, gh4.y, gh4.z, gh4.w}, gci[4] = {gi4.x, gi4.y, gi4.z, gi4.w};
  float di[4], dO[4], du[4], df[NCH][4], dc[NCH][4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float gh = (root ? 0.f : ghp[e]) + lg[e];
    const float tau = tanh_(cc[e]);
    dO[e] = gh * tau * og[e] * (1.f - og[e]);
    const float gc = (root ? 0.f : gci[e]) + gh * og[e] * (1.f - tau * tau);
    di[e] = gc * ug[e] * ig[e] * (1.f - ig[e]);
    du[e] = gc * ig[e] * (1.f - ug[e] * ug[e]);
    if constexpr (!LEAF) {
#pragma unroll
      for (int k = 0; k < NCH; ++k) {
        const float fk[4] = {fk4[k].x, fk4[k].y, fk4[k].z, fk4[k].w};
        const float ck[4] = {ck4[k].x, ck4[k].y, ck4[k].z, ck4[k].w};
        df[k][e] = cp[k] >= 0 ? gc * ck[e] * fk[e] * (1.f - fk[e]) : 0.f;
        dc[k][e] = gc * fk[e];
      }
    }
  }
  auto f4 = [](const float (&x)[4]) { return make_float4(x[0], x[1], x[2], x[3]); };
  float* da = n.dA + (size_t)p * n.GW + j0;
  unsigned short* db = wb ? n.dAb + (size_t)p * n.GW + j0 : nullptr;
  auto st = [&](int col, const float (&x)[4]) {
    st4(da + col, f4(x));
    if (db) {
      const unsigned lo = f2bf(x[0]) | ((unsigned)f2bf(x[1]) << 16);
      const unsigned hi = f2bf(x[2]) | ((unsigned)f2bf(x[3]) << 16);
      *reinterpret_cast<uint2*>(db + col) = make_uint2(lo, hi);
    }
  };
  st(0, di);
  st(2 * H, dO);
  st(3 * H, du);
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const bool has = !LEAF && cp[k] >= 0;
    if (has || p >= n.f_unread_below) {
      float z[4] = {0.f, 0.f, 0.f, 0.f};
      if constexpr (!LEAF) {
#pragma unroll
        for (int e = 0; e < 4; ++e) z[e] = df[k][e];
      }
      st(k == 0 ? H : 4 * H, z);
    }
    if constexpr (!LEAF)
      if (has) st4(n.dCp + (size_t)cp[k] * H + j0, f4(dc[k]));
  }
}

// Roots at positions >= n.fuse_from: one workgroup per position (the others
// exit at once); every other position there gets its dA in the epilogue of
// its parent's level product.
__global__ void __launch_bounds__(256) k_lstm_bwd_roots(Net n) {
  const int p = n.fuse_from + blockIdx.x;
  if (n.parent_pos[p] >= 0) return;
  for (int j = threadIdx.x; j < n.H; j += 256) {
    if (n.N == 2) lstm_gates_elem<2>(n, p, j, 0.f, 0.f);
    else lstm_gates_elem<1>(n, p, j, 0.f, 0.f);
  }
}

// Tile: BM positions x BHU hidden units; 4 wavefronts arranged WR x WU, each
// owning TR = BM / (16 WR) row tiles of 16 positions x 16 units and all
// (3 + NCH) gate accumulators for them (B fragments are reused across the
// TR row tiles).  With XCD set, the 1D grid is mapped so that each XCD
// touches 1/8 of the unit tiles (see xcd_tile).
template <int NCH, int BM, int WR, bool XCD>
__global__ void __launch_bounds__(256) k_lstm_fwd_level(Net n, int off, int M) {
  constexpr int WU = 4 / WR, BHU = 16 * WU, TR = BM / (16 * WR);
  constexpr int LDA = kBK + 4;
  constexpr int LDB = BHU + 2;
  constexpr int A_N = BM * NCH * (kBK / 4);          // float4 per chunk
  constexpr int A_PER = (A_N + 255) / 256;
  constexpr int B_ROW4 = BHU / 4;                    // float4 per (gate, k) row
  constexpr int B_N = 4 * kBK * B_ROW4;
  constexpr int B_PER = B_N / 256;
  constexpr int NACC = 3 + NCH;
  static_assert(B_N % 256 == 0, "B tile must split evenly");
  __shared__ __attribute__((aligned(16))) float As[NCH][BM * LDA];
  __shared__ float Bs[4][kBK * LDB];

  const int H = n.H, H4 = 4 * H;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w % WR, wu = w / WR;
  int rt, utile;
  if constexpr (XCD) {
    const int nut = H / BHU, bid = blockIdx.x, xcd = bid & 7, local = bid >> 3, per = nut >> 3;
    utile = xcd + 8 * (local % per);
    rt = local / per;
  } else {
    rt = blockIdx.x;
    utile = blockIdx.y;
  }
  const int row0 = off + rt * BM;
  const int rowend = off + M;
  const int u0 = utile * BHU;

  const float* asrc[A_PER];
  int adst[A_PER];
#pragma unroll
  for (int a = 0; a < A_PER; ++a) {
    const int idx = tid + 256 * a;
    asrc[a] = nullptr;
    adst[a] = -1;
    if (idx < A_N) {
      const int row = idx / (NCH * 8), ch = (idx / 8) % NCH, q = idx % 8;
      adst[a] = ch * (BM * LDA) + row * LDA + 4 * q;
      const int p = row0 + row;
      if (p < rowend) {
        const int cp = n.child_pos[(size_t)p * NCH + ch];
        if (cp >= 0) asrc[a] = n.Hs + (size_t)cp * H + 4 * q;
      }
    }
  }
  const float* bsrc[B_PER];
  int bdst[B_PER];
#pragma unroll
  for (int bq = 0; bq < B_PER; ++bq) {
    const int idx = tid + 256 * bq;
    const int g = idx / (kBK * B_ROW4), rem = idx % (kBK * B_ROW4);
    const int k = rem / B_ROW4, q = rem % B_ROW4;
    bsrc[bq] = n.U + (size_t)k * H4 + g * H + u0 + 4 * q;
    bdst[bq] = g * (kBK * LDB) + k * LDB + 4 * q;
  }
  float4 ra[A_PER], rb[B_PER];
  auto gload = [&](int k0) {
#pragma unroll
    for (int a = 0; a < A_PER; ++a) ra[a] = asrc[a] ? ldg4(asrc[a] + k0) : f4zero();
#pragma unroll
    for (int bq = 0; bq < B_PER; ++bq) rb[bq] = ldg4(bsrc[bq] + (size_t)k0 * H4);
  };
  float* As_flat = &As[0][0];
  float* Bs_flat = &Bs[0][0];
  auto sstore = [&]() {
#pragma unroll
    for (int a = 0; a < A_PER; ++a)
      if (adst[a] >= 0) st4(As_flat + adst[a], ra[a]);
#pragma unroll
    for (int bq = 0; bq < B_PER; ++bq) st4_scalar(Bs_flat + bdst[bq], rb[bq]);
  };

  v4f acc[TR][NACC];
#pragma unroll
  for (int tr = 0; tr < TR; ++tr)
#pragma unroll
    for (int g = 0; g < NACC; ++g) acc[tr][g] = v4f{0.f, 0.f, 0.f, 0.f};
  gload(0);
  for (int k0 = 0; k0 < H; k0 += kBK) {
    __syncthreads();
    sstore();
    __syncthreads();
    if (k0 + kBK < H) gload(k0 + kBK);
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      float bi[4], bf[4], bo[4], bu[4];
      load_frag4<false, LDB>(Bs[G_I], wu * 16 + r, gq, half, bi);
      load_frag4<false, LDB>(Bs[G_F], wu * 16 + r, gq, half, bf);
      load_frag4<false, LDB>(Bs[G_O], wu * 16 + r, gq, half, bo);
      load_frag4<false, LDB>(Bs[G_U], wu * 16 + r, gq, half, bu);
#pragma unroll
      for (int tr = 0; tr < TR; ++tr) {
        const int row = (wr * TR + tr) * 16 + r;
        float a0[4], a1[4];
        load_frag4<true, LDA>(As[0], row, gq, half, a0);
        if constexpr (NCH == 2) load_frag4<true, LDA>(As[NCH - 1], row, gq, half, a1);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          float ah = a0[s];
          if constexpr (NCH == 2) ah = a0[s] + a1[s];
          acc[tr][0] = mfma_f32_16x16x4(ah, bi[s], acc[tr][0]);
          acc[tr][1] = mfma_f32_16x16x4(ah, bo[s], acc[tr][1]);
          acc[tr][2] = mfma_f32_16x16x4(ah, bu[s], acc[tr][2]);
          acc[tr][3] = mfma_f32_16x16x4(a0[s], bf[s], acc[tr][3]);
          if constexpr (NCH == 2) acc[tr][4] = mfma_f32_16x16x4(a1[s], bf[s], acc[tr][4]);
        }
      }
    }
  }

  // epilogue: gates, cell update, scatter of (c, h)
  const int j = u0 + wu * 16 + r;
#pragma unroll
  for (int tr = 0; tr < TR; ++tr)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = row0 + (wr * TR + tr) * 16 + 4 * gq + i;
      if (p < rowend)
        lstm_fwd_epilogue<NCH>(n, p, j, acc[tr][0][i], acc[tr][1][i], acc[tr][2][i],
                               acc[tr][3][i], NCH == 2 ? acc[tr][NACC - 1][i] : 0.f);
    }
}

// dL/dh_k for every vertex of the level: tile BM positions x 64 hidden units.
// NCH == 2: acc_h = dA[:, i|o|u] U[:, i|o|u]^T (K = 3H), then acc_fk =
// dA[:, f_k] U[:, f]^T (K = H) with one shared B tile; child k receives
// acc_h + acc_fk.  NCH == 1: one K = 4H product over all gate columns.
template <int NCH, int BM>
__global__ void __launch_bounds__(256) k_lstm_bwd_level(Net n, int off, int M) {
  constexpr int BN = 64;
  constexpr int WRW = BM == 64 ? 2 : 1, WCW = 4 / WRW;
  constexpr int TM = BM / 16 / WRW, TN = BN / 16 / WCW;
  constexpr int LDA = kBK + 4, LDB = kBK + 4;
  constexpr int A_N = BM * 8;
  constexpr int A_PER = (A_N + 255) / 256;
  constexpr int B_PER = BN * 8 / 256;
  __shared__ __attribute__((aligned(16))) float As[NCH][BM * LDA];
  __shared__ __attribute__((aligned(16))) float Bs[BN * LDB];

  const int H = n.H, H4 = 4 * H, GW = n.GW;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wrow = (w / WCW) * TM * 16, wcol = (w % WCW) * TN * 16;
  const int row0 = off + blockIdx.x * BM, rowend = off + M;
  const int n0 = blockIdx.y * BN;

  // per-thread A rows (positions) and B rows (hidden units)
  int arow[A_PER], aq[A_PER];
  bool aval[A_PER];
#pragma unroll
  for (int a = 0; a < A_PER; ++a) {
    const int idx = tid + 256 * a;
    arow[a] = idx / 8;
    aq[a] = idx % 8;
    aval[a] = idx < A_N && row0 + arow[a] < rowend;
  }
  int brow[B_PER], bq4[B_PER];
#pragma unroll
  for (int b = 0; b < B_PER; ++b) {
    const int idx = tid + 256 * b;
    brow[b] = idx / 8;
    bq4[b] = idx % 8;
  }
  float4 ra[NCH][A_PER], rb[B_PER];
  // phase 1 chunk kc covers dA / U columns col0 .. col0+31
  auto col_phase1 = [&](int kc) {
    const int c = kc * kBK;
    if constexpr (NCH == 1) return c;
    return c < H ? c : c + H;   // skip the f block
  };
  auto gload = [&](int colA0, int colA1, int colB) {
#pragma unroll
    for (int a = 0; a < A_PER; ++a) {
      const float* src = n.dA + (size_t)(row0 + arow[a]) * GW + 4 * aq[a];
      ra[0][a] = aval[a] ? ldg4(src + colA0) : f4zero();
      if constexpr (NCH == 2) ra[1][a] = (aval[a] && colA1 >= 0) ? ldg4(src + colA1) : f4zero();
    }
#pragma unroll
    for (int b = 0; b < B_PER; ++b)
      rb[b] = ldg4(n.U + (size_t)(n0 + brow[b]) * H4 + colB + 4 * bq4[b]);
  };
  auto sstore = [&](int nA) {
#pragma unroll
    for (int a = 0; a < A_PER; ++a)
      if (tid + 256 * a < A_N) {
        st4(&As[0][arow[a] * LDA + 4 * aq[a]], ra[0][a]);
        if constexpr (NCH == 2)
          if (nA == 2) st4(&As[1][arow[a] * LDA + 4 * aq[a]], ra[1][a]);
      }
#pragma unroll
    for (int b = 0; b < B_PER; ++b) st4(&Bs[brow[b] * LDB + 4 * bq4[b]], rb[b]);
  };

  v4f acc_h[TM][TN], acc_f0[TM][TN], acc_f1[TM][TN];
  zero_acc(acc_h);
  zero_acc(acc_f0);
  zero_acc(acc_f1);

  // phase 1
  const int nk1 = (NCH == 1 ? H4 : 3 * H) / kBK;
  gload(col_phase1(0), -1, col_phase1(0));
  for (int kc = 0; kc < nk1; ++kc) {
    __syncthreads();
    sstore(1);
    __syncthreads();
    if (kc + 1 < nk1) {
      const int c = col_phase1(kc + 1);
      gload(c, -1, c);
    } else if constexpr (NCH == 2) {
      gload(H, 4 * H, H);   // first chunk of phase 2
    }
    mfma_chunk<TM, TN, true, true, LDA, LDB>(As[0], Bs, wrow, wcol, acc_h);
  }
  // phase 2 (two children): the f columns
  if constexpr (NCH == 2) {
    const int nk2 = H / kBK;
    for (int kc = 0; kc < nk2; ++kc) {
      __syncthreads();
      sstore(2);
      __syncthreads();
      if (kc + 1 < nk2) {
        const int c = (kc + 1) * kBK;
        gload(H + c, 4 * H + c, H + c);
      }
      mfma_chunk<TM, TN, true, true, LDA, LDB>(As[0], Bs, wrow, wcol, acc_f0);
      mfma_chunk<TM, TN, true, true, LDA, LDB>(As[1], Bs, wrow, wcol, acc_f1);
    }
  }

  // epilogue: scatter dL/dh_k to the children (one writer per child row)
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = row0 + wrow + tm * 16 + 4 * gq + i;
      if (p >= rowend) continue;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        lstm_bwd_scatter<NCH>(n, p, n0 + wcol + tn * 16 + r, acc_h[tm][tn][i], acc_f0[tm][tn][i],
                              acc_f1[tm][tn][i]);
    }
}

// ------------------------------------------------------------ bf16 variants
// Same tiling and epilogues as above; operands are rounded to bf16 while they
// are staged into LDS (h~ = h_0 + h_1 is formed in fp32 first), one
// v_mfma_f32_16x16x32_bf16 per 32-deep chunk and output tile.
template <int NCH, int BM>
__global__ void __launch_bounds__(256) k_lstm_fwd_level_bf(Net n, int off, int M) {
  constexpr int WR = BM / 16, WU = 4 / WR, BHU = 16 * WU;
  constexpr int NA = NCH == 2 ? 3 : 1;               // tiles: h_0 (, h_1, h~)
  constexpr int A_N = BM * (kBK / 4);                // (row, k-quad) pairs per chunk
  constexpr int A_PER = (A_N + 255) / 256;
  constexpr int B_ROW4 = BHU / 4;
  constexpr int B_N = 4 * kBK * B_ROW4;
  constexpr int B_PER = B_N / 256;
  static_assert(B_N % 256 == 0, "B tile must split evenly");
  __shared__ __attribute__((aligned(16))) u16 As[NA][BM * kLDH];
  __shared__ __attribute__((aligned(16))) u16 Bs[4][BHU * kLDH];

  const int H = n.H, H4 = 4 * H;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w % WR, wu = w / WR;
  const int row0 = off + blockIdx.x * BM, rowend = off + M;
  const int u0 = blockIdx.y * BHU;

  const float* asrc[A_PER][NCH];
  int adst[A_PER];
#pragma unroll
  for (int a = 0; a < A_PER; ++a) {
    const int idx = tid + 256 * a;
    adst[a] = -1;
#pragma unroll
    for (int c = 0; c < NCH; ++c) asrc[a][c] = nullptr;
    if (idx < A_N) {
      const int row = idx / 8, q = idx % 8;
      adst[a] = row * kLDH + 4 * q;
      const int p = row0 + row;
      if (p < rowend) {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          const int cp = n.child_pos[(size_t)p * NCH + c];
          if (cp >= 0) asrc[a][c] = n.Hs + (size_t)cp * H + 4 * q;
        }
      }
    }
  }
  const float* bsrc[B_PER];
  int bdst[B_PER];
#pragma unroll
  for (int bq = 0; bq < B_PER; ++bq) {
    const int idx = tid + 256 * bq;
    const int g = idx / (kBK * B_ROW4), rem = idx % (kBK * B_ROW4);
    const int k = rem / B_ROW4, q = rem % B_ROW4;
    bsrc[bq] = n.U + (size_t)k * H4 + g * H + u0 + 4 * q;
    bdst[bq] = g * (BHU * kLDH) + (4 * q) * kLDH + k;     // transposed: [gate][unit][k]
  }
  float4 ra[A_PER][NCH], rb[B_PER];
  auto gload = [&](int k0) {
#pragma unroll
    for (int a = 0; a < A_PER; ++a)
#pragma unroll
      for (int c = 0; c < NCH; ++c) ra[a][c] = asrc[a][c] ? ldg4(asrc[a][c] + k0) : f4zero();
#pragma unroll
    for (int bq = 0; bq < B_PER; ++bq) rb[bq] = ldg4(bsrc[bq] + (size_t)k0 * H4);
  };
  u16* As_flat = &As[0][0];
  u16* Bs_flat = &Bs[0][0];
  auto sstore = [&]() {
#pragma unroll
    for (int a = 0; a < A_PER; ++a)
      if (adst[a] >= 0) {
        st_bf4(As_flat + adst[a], ra[a][0]);
        if constexpr (NCH == 2) {
          st_bf4(As_flat + BM * kLDH + adst[a], ra[a][1]);
          st_bf4(As_flat + 2 * BM * kLDH + adst[a], add4(ra[a][0], ra[a][1]));
        }
      }
#pragma unroll
    for (int bq = 0; bq < B_PER; ++bq) st_bf4_t(Bs_flat + bdst[bq], kLDH, rb[bq]);
  };

  v4f acc_i = {0.f, 0.f, 0.f, 0.f}, acc_o = acc_i, acc_u = acc_i, acc_f0 = acc_i, acc_f1 = acc_i;
  gload(0);
  for (int k0 = 0; k0 < H; k0 += kBK) {
    __syncthreads();
    sstore();
    __syncthreads();
    if (k0 + kBK < H) gload(k0 + kBK);
    const bf16x8 a0 = frag_bf(As[0], wr * 16 + r, gq);
    const bf16x8 ah = frag_bf(As[NA - 1], wr * 16 + r, gq);
    const bf16x8 bi = frag_bf(Bs[G_I], wu * 16 + r, gq);
    const bf16x8 bfg = frag_bf(Bs[G_F], wu * 16 + r, gq);
    const bf16x8 bo = frag_bf(Bs[G_O], wu * 16 + r, gq);
    const bf16x8 bu = frag_bf(Bs[G_U], wu * 16 + r, gq);
    acc_i = mfma_bf16_16x16x32(ah, bi, acc_i);
    acc_o = mfma_bf16_16x16x32(ah, bo, acc_o);
    acc_u = mfma_bf16_16x16x32(ah, bu, acc_u);
    acc_f0 = mfma_bf16_16x16x32(a0, bfg, acc_f0);
    if constexpr (NCH == 2) {
      const bf16x8 a1 = frag_bf(As[1], wr * 16 + r, gq);
      acc_f1 = mfma_bf16_16x16x32(a1, bfg, acc_f1);
    }
  }
  const int j = u0 + wu * 16 + r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int p = row0 + wr * 16 + 4 * gq + i;
    if (p < rowend) lstm_fwd_epilogue<NCH>(n, p, j, acc_i[i], acc_o[i], acc_u[i], acc_f0[i], acc_f1[i]);
  }
}

template <int NCH, int BM>
__global__ void __launch_bounds__(256) k_lstm_bwd_level_bf(Net n, int off, int M) {
  constexpr int BN = 64;
  constexpr int WRW = BM == 64 ? 2 : 1, WCW = 4 / WRW;
  constexpr int TM = BM / 16 / WRW, TN = BN / 16 / WCW;
  constexpr int A_N = BM * 8;
  constexpr int A_PER = (A_N + 255) / 256;
  constexpr int B_PER = BN * 8 / 256;
  __shared__ __attribute__((aligned(16))) u16 As[NCH][BM * kLDH];
  __shared__ __attribute__((aligned(16))) u16 Bs[BN * kLDH];

  const int H = n.H, H4 = 4 * H, GW = n.GW;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wrow = (w / WCW) * TM * 16, wcol = (w % WCW) * TN * 16;
  const int row0 = off + blockIdx.x * BM, rowend = off + M;
  const int n0 = blockIdx.y * BN;
  int arow[A_PER], aq[A_PER];
  bool aval[A_PER];
#pragma unroll
  for (int a = 0; a < A_PER; ++a) {
    const int idx = tid + 256 * a;
    arow[a] = idx / 8;
    aq[a] = idx % 8;
    aval[a] = idx < A_N && row0 + arow[a] < rowend;
  }
  float4 ra[NCH][A_PER], rb[B_PER];
  auto col_phase1 = [&](int kc) {
    const int c = kc * kBK;
    if constexpr (NCH == 1) return c;
    return c < H ? c : c + H;
  };
  auto gload = [&](int colA0, int colA1, int colB) {
#pragma unroll
    for (int a = 0; a < A_PER; ++a) {
      const float* src = n.dA + (size_t)(row0 + arow[a]) * GW + 4 * aq[a];
      ra[0][a] = aval[a] ? ldg4(src + colA0) : f4zero();
      if constexpr (NCH == 2) ra[1][a] = (aval[a] && colA1 >= 0) ? ldg4(src + colA1) : f4zero();
    }
#pragma unroll
    for (int b = 0; b < B_PER; ++b) {
      const int idx = tid + 256 * b;
      rb[b] = ldg4(n.U + (size_t)(n0 + idx / 8) * H4 + colB + 4 * (idx % 8));
    }
  };
  auto sstore = [&](int nA) {
#pragma unroll
    for (int a = 0; a < A_PER; ++a)
      if (tid + 256 * a < A_N) {
        st_bf4(&As[0][arow[a] * kLDH + 4 * aq[a]], ra[0][a]);
        if constexpr (NCH == 2)
          if (nA == 2) st_bf4(&As[1][arow[a] * kLDH + 4 * aq[a]], ra[1][a]);
      }
#pragma unroll
    for (int b = 0; b < B_PER; ++b) {
      const int idx = tid + 256 * b;
      st_bf4(&Bs[(idx / 8) * kLDH + 4 * (idx % 8)], rb[b]);
    }
  };
  v4f acc_h[TM][TN], acc_f0[TM][TN], acc_f1[TM][TN];
  zero_acc(acc_h);
  zero_acc(acc_f0);
  zero_acc(acc_f1);
  const int nk1 = (NCH == 1 ? H4 : 3 * H) / kBK;
  gload(col_phase1(0), -1, col_phase1(0));
  for (int kc = 0; kc < nk1; ++kc) {
    __syncthreads();
    sstore(1);
    __syncthreads();
    if (kc + 1 < nk1) {
      const int c = col_phase1(kc + 1);
      gload(c, -1, c);
    } else if constexpr (NCH == 2) {
      gload(H, 4 * H, H);
    }
    mfma_chunk_bf<TM, TN>(As[0], Bs, wrow, wcol, acc_h);
  }
  if constexpr (NCH == 2) {
    const int nk2 = H / kBK;
    for (int kc = 0; kc < nk2; ++kc) {
      __syncthreads();
      sstore(2);
      __syncthreads();
      if (kc + 1 < nk2) {
        const int c = (kc + 1) * kBK;
        gload(H + c, 4 * H + c, H + c);
      }
      mfma_chunk_bf<TM, TN>(As[0], Bs, wrow, wcol, acc_f0);
      mfma_chunk_bf<TM, TN>(As[1], Bs, wrow, wcol, acc_f1);
    }
  }
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = row0 + wrow + tm * 16 + 4 * gq + i;
      if (p >= rowend) continue;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        lstm_bwd_scatter<NCH>(n, p, n0 + wcol + tn * 16 + r, acc_h[tm][tn][i], acc_f0[tm][tn][i],
                              acc_f1[tm][tn][i]);
    }
}

// --------------------------------------------------- split-K level kernels
// For levels too small to fill the chip with the tiles above: a workgroup
// owns 16 positions x 16 units (forward) or 16 positions x 16 columns
// (backward); wavefront w accumulates the w-th quarter of the contraction.
// MFMA fragments are loaded straight from global memory into registers: in
// the permuted-K order lane group g needs k = 8g .. 8g+7 of its A row (two
// float4) and of its B column.  The four partial sums are reduced in LDS in
// a fixed order (deterministic) and the epilogue is shared with the tiled
// kernels.  BF selects bf16 operands (one 16x16x32 MFMA per 32-deep chunk)
// instead of fp32 (eight 16x16x4 steps).
template <int NCH, int TR, int KW = 4>
struct FwdRed {
  float v[KW][TR][3 + NCH][4][64];
};

// One 16*TR-position x 16-unit forward tile (row tile rt, unit tile ut).
// Wavefronts 0 .. KW-1 split the contraction.  With EPI, four more
// wavefronts (KW .. KW+3) own the epilogue: they read everything it needs
// besides the product (bias, pulled term, children's c) while the others
// multiply, then finish element i = w - KW of every row tile.  Without EPI
// (persistent loop, 64*KW threads) the contraction wavefronts finish it.
// Rows: the positions of the tile's 16*TR rows (RangeRows or ListRows).
// COH: the children's rows may have been written earlier in the same launch
// (the XCD-local level loop), so they are read with coherent loads.
// WL: the weight columns of this unit tile are resident in LDS (wl: column
// c = 16 g + r of the tile, k-contiguous, row stride WLD elements; fp32, or
// bf16 pre-rounded); otherwise they are read from global memory.
// FOLD (with EPI): the partial sums of contraction wavefronts KW/2 .. KW-1
// are first added to those of wavefronts 0 .. KW/2-1 (own + partner, in that
// order), so the reduction buffer holds KW/2 slots.
template <int NCH, bool BF, int TR, int KW, bool EPI, class Rows = RangeRows, bool COH = false,
          int WLD = 0, bool FOLD = false>
__device__ __forceinline__ void lstm_fwd_sk_tile(const Net& n, const Rows& rows, int ut,
                                                 FwdRed<NCH, TR, FOLD ? KW / 2 : KW>& R,
                                                 const void* wl = nullptr) {
  constexpr int NACC = 3 + NCH, RKW = FOLD ? KW / 2 : KW;
  static_assert(!FOLD || (EPI && KW % 2 == 0), "fold");
  auto& red = R.v;
  const int H = n.H, H4 = 4 * H;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int u0 = ut * 16;
  v4f acc[TR][NACC];
  if (w < KW) {
    // A rows of this lane: the children of the position of tile row 16 tr + r.
    // An absent child (or a row past the level) reads row 0 with weight 0,
    // so the loads are unconditional.
    const float* ap[TR][NCH];
    size_t aoff[TR][NCH];
    float am[TR][NCH];
#pragma unroll
    for (int tr = 0; tr < TR; ++tr) {
      const int pa = rows.pos(16 * tr + r);
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const int cp = pa >= 0 ? n.child_pos[(size_t)pa * NCH + c] : -1;
        aoff[tr][c] = (size_t)(cp >= 0 ? cp : 0) * H;
        ap[tr][c] = n.Hs + aoff[tr][c];
        am[tr][c] = cp >= 0 ? 1.f : 0.f;
      }
    }
    const CohBuf hb = COH ? coh_buf(n.Hs, (size_t)n.V * H) : CohBuf{};
    const float* ub = n.U + u0 + r;          // column u0 + r of each gate block
    const int kq = H / KW, kbeg = w * kq, kend = kbeg + kq;
#pragma unroll
    for (int tr = 0; tr < TR; ++tr)
#pragma unroll
      for (int g = 0; g < NACC; ++g) acc[tr][g] = v4f{0.f, 0.f, 0.f, 0.f};

    // bf16: the weight fragment comes pre-rounded from n.UTb (U^T, one
    // 16-byte load per gate); fp32: eight loads down a column of U
    struct Frag {
      float a[TR][NCH][8];
      float b[BF ? 1 : 4][8];
      bf16x8 bq[BF ? 4 : 1];
    };
    const u16* utb = BF ? n.UTb + (size_t)(u0 + r) * H : nullptr;
    auto load_a = [&](int k0, Frag& f) {
      const int kk = k0 + 8 * gq;
#pragma unroll
      for (int tr = 0; tr < TR; ++tr)
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          if constexpr (COH) {
            const float4 x = coh_ld4(hb, aoff[tr][c] + kk), y = coh_ld4(hb, aoff[tr][c] + kk + 4);
            float* d = f.a[tr][c];
            d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
            d[4] = y.x; d[5] = y.y; d[6] = y.z; d[7] = y.w;
          } else {
            ld8(ap[tr][c] + kk, f.a[tr][c]);
          }
        }
    };
    auto load_b = [&](int k0, Frag& f) {
      const int kk = k0 + 8 * gq;
      if constexpr (WLD > 0 && BF) {
#pragma unroll
        for (int g = 0; g < 4; ++g)
          f.bq[g] = *reinterpret_cast<const bf16x8*>(static_cast<const u16*>(wl) +
                                                     (16 * g + r) * WLD + kk);
      } else if constexpr (WLD > 0) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float* bp = static_cast<const float*>(wl) + (16 * g + r) * WLD + kk;
          const float4 x = *reinterpret_cast<const float4*>(bp);
          const float4 y = *reinterpret_cast<const float4*>(bp + 4);
          f.b[g][0] = x.x; f.b[g][1] = x.y; f.b[g][2] = x.z; f.b[g][3] = x.w;
          f.b[g][4] = y.x; f.b[g][5] = y.y; f.b[g][6] = y.z; f.b[g][7] = y.w;
        }
      } else if constexpr (BF) {
#pragma unroll
        for (int g = 0; g < 4; ++g)
          f.bq[g] = *reinterpret_cast<const bf16x8*>(utb + (size_t)g * H * H + kk);
      } else {
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
          for (int s = 0; s < 8; ++s) f.b[g][s] = ub[(size_t)(kk + s) * H4 + g * H];
      }
    };
    auto load = [&](int k0, Frag& f) {
      load_a(k0, f);
      load_b(k0, f);
    };
    auto compute = [&](const Frag& f) {
#pragma unroll
      for (int tr = 0; tr < TR; ++tr) {
        float a0[8], a1[8], ah[8];
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          a0[s] = f.a[tr][0][s] * am[tr][0];
          a1[s] = NCH == 2 ? f.a[tr][NCH - 1][s] * am[tr][NCH - 1] : 0.f;
          ah[s] = NCH == 2 ? a0[s] + a1[s] : a0[s];
        }
        if constexpr (BF) {
          const bf16x8 hb = to_bf8(ah), b0 = to_bf8(a0);
          acc[tr][0] = mfma_bf16_16x16x32(hb, f.bq[G_I], acc[tr][0]);
          acc[tr][1] = mfma_bf16_16x16x32(hb, f.bq[G_O], acc[tr][1]);
          acc[tr][2] = mfma_bf16_16x16x32(hb, f.bq[G_U], acc[tr][2]);
          acc[tr][3] = mfma_bf16_16x16x32(b0, f.bq[G_F], acc[tr][3]);
          if constexpr (NCH == 2) acc[tr][4] = mfma_bf16_16x16x32(to_bf8(a1), f.bq[G_F], acc[tr][4]);
        } else {
          acc[tr][0] = mfma_chunk8<BF>(ah, f.b[G_I], acc[tr][0]);
          acc[tr][1] = mfma_chunk8<BF>(ah, f.b[G_O], acc[tr][1]);
          acc[tr][2] = mfma_chunk8<BF>(ah, f.b[G_U], acc[tr][2]);
          acc[tr][3] = mfma_chunk8<BF>(a0, f.b[G_F], acc[tr][3]);
          if constexpr (NCH == 2) acc[tr][4] = mfma_chunk8<BF>(a1, f.b[G_F], acc[tr][4]);
        }
      }
    };
    if constexpr (WLD > 0) {
      // weights in LDS: every chunk's child rows are requested at once (one
      // memory latency); the weight fragments are read chunk by chunk
      constexpr int NCK = kXcdWsH / KW / kBK;
      Frag f[NCK];
#pragma unroll
      for (int c = 0; c < NCK; ++c) load_a(kbeg + c * kBK, f[c]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int c = 0; c < NCK; ++c) {
        load_b(kbeg + c * kBK, f[c]);
        compute(f[c]);
      }
    } else {
      // two register buffers: loads of the next chunk overlap the current MFMAs
      Frag fa, fb;
      load(kbeg, fa);
      for (int k0 = kbeg; k0 < kend; k0 += 2 * kBK) {
        load(k0 + kBK, fb);
        __builtin_amdgcn_sched_barrier(0);   // the next chunk's loads go out before these MFMAs
        compute(fa);
        if (k0 + 2 * kBK < kend) load(k0 + 2 * kBK, fa);
        compute(fb);
      }
    }
#pragma unroll
    for (int tr = 0; tr < TR; ++tr)
#pragma unroll
      for (int g = 0; g < NACC; ++g)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (!FOLD || w >= RKW) red[w % RKW][tr][g][i][lane] = acc[tr][g][i];
  }
  auto zsum = [&](int tr, int i, float (&z)[NACC]) {
#pragma unroll
    for (int g = 0; g < NACC; ++g) {
      float t = red[0][tr][g][i][lane];
#pragma unroll
      for (int q = 1; q < RKW; ++q) t += red[q][tr][g][i][lane];
      z[g] = t;
    }
  };
  if constexpr (EPI) {
    const int i = w - KW;
    FwdPre<NCH> pre[TR];
    if (w >= KW) {
#pragma unroll
      for (int tr = 0; tr < TR; ++tr) {
        // rows past the level read its last row (unused), so the loads
        // are unconditional
        lstm_fwd_pre<NCH, COH>(n, rows.clamp(16 * tr + 4 * gq + i), u0 + r, pre[tr]);
      }
    }
    __syncthreads();
    if constexpr (FOLD) {
      if (w < RKW) {
#pragma unroll
        for (int tr = 0; tr < TR; ++tr)
#pragma unroll
          for (int g = 0; g < NACC; ++g)
#pragma unroll
            for (int i = 0; i < 4; ++i) red[w][tr][g][i][lane] = acc[tr][g][i] + red[w][tr][g][i][lane];
      }
      __syncthreads();
    }
    if (w < KW) return;
#pragma unroll
    for (int tr = 0; tr < TR; ++tr) {
      const int p = rows.pos(16 * tr + 4 * gq + i);
      if (p < 0) continue;
      float z[NACC];
      zsum(tr, i, z);
      lstm_fwd_fin<NCH>(n, p, u0 + r, pre[tr], z[0], z[1], z[2], z[3],
                        NCH == 2 ? z[NACC - 1] : 0.f);
    }
  } else {
    __syncthreads();
    // wave w finishes element i = w % 4 of row tiles tr = w / 4, w / 4 + KW / 4, ...
    const int i = w & 3;
#pragma unroll
    for (int tr = w >> 2; tr < TR; tr += KW / 4) {
      const int p = rows.pos(16 * tr + 4 * gq + i);
      if (p < 0) continue;
      float z[NACC];
      zsum(tr, i, z);
      lstm_fwd_epilogue<NCH, COH>(n, p, u0 + r, z[0], z[1], z[2], z[3],
                                  NCH == 2 ? z[NACC - 1] : 0.f);
    }
  }
}

template <int NCH, bool BF, int TR, int KW>
__global__ void __launch_bounds__(64 * (KW + 4)) k_lstm_fwd_level_sk(Net n, int off, int M) {
  __shared__ FwdRed<NCH, TR, KW> red;
  int rt, ut;
  xcd_tile(n.H / 16, rt, ut);
  lstm_fwd_sk_tile<NCH, BF, TR, KW, true>(n, RangeRows{off + rt * 16 * TR, off + M}, ut, red);
}

template <int NCH, int TR, int KW = 4>
struct BwdRed {
  float v[KW][TR][NCH == 2 ? 3 : 1][4][64];
};

// One 16*TR-position x 16-column backward tile (row tile rt, column tile ut);
// wavefront roles as in the forward tile (EPI: four epilogue wavefronts
// that prefetch the children's saved state while the others multiply).
// Rows, COH and WL (rows n0 .. n0+15 of U resident in LDS, row stride WLD)
// as in the forward tile; COH also covers the dA rows of the level (written
// by the parents' epilogues in the same launch).
template <int NCH, bool BF, int TR, int KW, bool EPI, class Rows = RangeRows, bool COH = false,
          int WLD = 0>
__device__ __forceinline__ void lstm_bwd_sk_tile(const Net& n, const Rows& rows, int ut,
                                                 BwdRed<NCH, TR, KW>& R,
                                                 const void* wl = nullptr) {
  constexpr int NACC = 1 + (NCH == 2 ? 2 : 0);
  auto& red = R.v;
  const int H = n.H, H4 = 4 * H, GW = n.GW;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int n0 = ut * 16;
  if (w < KW) {
    // rows past the level read its last row: their sums are never used
    const float* da[TR];
    size_t daoff[TR];
#pragma unroll
    for (int tr = 0; tr < TR; ++tr) {
      daoff[tr] = (size_t)rows.clamp(16 * tr + r) * GW;
      da[tr] = n.dA + daoff[tr];
    }
    // bf16: dA's bf16 copy (written with dA, rounded as the product rounds
    // it): eight values in one 16-byte load, no conversion
    const CohBuf ab = !COH ? CohBuf{}
                      : BF ? coh_buf(reinterpret_cast<const float*>(n.dAb), (size_t)n.V * GW / 2)
                           : coh_buf(n.dA, (size_t)n.V * GW);
    auto lda = [&](int tr, int col, float (&v)[BF ? 1 : 8], bf16x8& q) {
      if constexpr (BF && COH) {
        q = __builtin_bit_cast(bf16x8, coh_ld4(ab, (daoff[tr] + col) / 2));
      } else if constexpr (BF) {
        q = *reinterpret_cast<const bf16x8*>(n.dAb + daoff[tr] + col);
      } else if constexpr (COH) {
        const float4 x = coh_ld4(ab, daoff[tr] + col), y = coh_ld4(ab, daoff[tr] + col + 4);
        v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
        v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
      } else {
        ld8(da[tr] + col, v);
      }
    };
    // the U fragment: row n0 + r of U at columns col .. col+7
    auto ldu = [&](int col, float (&v)[8], bf16x8& q) {
      if constexpr (WLD > 0 && BF) {
        q = *reinterpret_cast<const bf16x8*>(static_cast<const u16*>(wl) + r * WLD + col);
      } else if constexpr (WLD > 0) {
        const float* bp = static_cast<const float*>(wl) + r * WLD + col;
        const float4 x = *reinterpret_cast<const float4*>(bp);
        const float4 y = *reinterpret_cast<const float4*>(bp + 4);
        v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
        v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
      } else if constexpr (BF) {
        q = *reinterpret_cast<const bf16x8*>(n.Ub + (size_t)(n0 + r) * H4 + col);
      } else {
        ld8(n.U + (size_t)(n0 + r) * H4 + col, v);
      }
    };
    v4f acc[TR][NACC];
#pragma unroll
    for (int tr = 0; tr < TR; ++tr)
#pragma unroll
      for (int g = 0; g < NACC; ++g) acc[tr][g] = v4f{0.f, 0.f, 0.f, 0.f};
    // phase 1: i|o|u columns (all four blocks with one child slot)
    struct F1 {
      float a[TR][BF ? 1 : 8], b[BF ? 1 : 8];
      bf16x8 aq[TR], bq;
    };
    const int K1 = NCH == 1 ? H4 : 3 * H, q1 = K1 / KW;
    auto load1 = [&](int c0, F1& f) {
      const int col = (NCH == 2 && c0 >= H ? c0 + H : c0) + 8 * gq;
#pragma unroll
      for (int tr = 0; tr < TR; ++tr) lda(tr, col, f.a[tr], f.aq[tr]);
      float dummy[8];
      if constexpr (BF) ldu(col, dummy, f.bq);
      else ldu(col, f.b, f.bq);
    };
    auto comp1 = [&](const F1& f) {
#pragma unroll
      for (int tr = 0; tr < TR; ++tr) {
        if constexpr (BF) acc[tr][0] = mfma_bf16_16x16x32(f.aq[tr], f.bq, acc[tr][0]);
        else acc[tr][0] = mfma_chunk8<BF>(f.a[tr], f.b, acc[tr][0]);
      }
    };
    // groups of G chunks: all loads of a group are in flight together, so a
    // small level pays about one memory latency per group, not per chunk.
    // A wavefront's share is a whole number of groups (K1 / (32 KW) is a
    // multiple of 6 with two children and of 8 with one, for the H this
    // kernel is launched with: H % 512 == 0 at KW = 8, H % 256 == 0 at
    // KW = 4), so the loads are unconditional.
    constexpr int G1 = NCH == 2 ? 6 : 8;
    const int end1 = (w + 1) * q1;
    if constexpr (NCH == 2) {
      // the two phases' loads go out together: one memory latency per level
      struct F2 {
        float a0[TR][BF ? 1 : 8], a1[TR][BF ? 1 : 8], b[BF ? 1 : 8];
        bf16x8 aq0[TR], aq1[TR], bq;
      };
      const int q2 = H / KW;
      auto load2 = [&](int c0, F2& f) {
        const int col = c0 + 8 * gq;
#pragma unroll
        for (int tr = 0; tr < TR; ++tr) {
          lda(tr, H + col, f.a0[tr], f.aq0[tr]);
          lda(tr, 4 * H + col, f.a1[tr], f.aq1[tr]);
        }
        float dummy[8];
        if constexpr (BF) ldu(H + col, dummy, f.bq);
        else ldu(H + col, f.b, f.bq);
      };
      auto comp2 = [&](const F2& f) {
#pragma unroll
        for (int tr = 0; tr < TR; ++tr) {
          if constexpr (BF) {
            acc[tr][1] = mfma_bf16_16x16x32(f.aq0[tr], f.bq, acc[tr][1]);
            acc[tr][2] = mfma_bf16_16x16x32(f.aq1[tr], f.bq, acc[tr][2]);
          } else {
            acc[tr][1] = mfma_chunk8<BF>(f.a0[tr], f.b, acc[tr][1]);
            acc[tr][2] = mfma_chunk8<BF>(f.a1[tr], f.b, acc[tr][2]);
          }
        }
      };
      constexpr int G2 = 2;   // H / (32 KW) is even
      const int end2 = (w + 1) * q2;
      // per group: the phase-2 chunks and the first half of the phase-1
      // chunks load together; the second half loads into the registers the
      // phase-2 fragments free, while the first half is multiplied
      constexpr int GH = G1 / 2;
      int c1 = w * q1;
      for (int c0 = w * q2; c0 < end2; c0 += G2 * kBK, c1 += G1 * kBK) {
        F2 f2[G2];
        F1 fa[GH], fb[GH];
#pragma unroll
        for (int g = 0; g < G2; ++g) load2(c0 + g * kBK, f2[g]);
#pragma unroll
        for (int g = 0; g < GH; ++g) load1(c1 + g * kBK, fa[g]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int g = 0; g < G2; ++g) comp2(f2[g]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int g = 0; g < GH; ++g) load1(c1 + (GH + g) * kBK, fb[g]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int g = 0; g < GH; ++g) comp1(fa[g]);
#pragma unroll
        for (int g = 0; g < GH; ++g) comp1(fb[g]);
      }
    } else {
      for (int c0 = w * q1; c0 < end1; c0 += G1 * kBK) {
        F1 f[G1];
#pragma unroll
        for (int g = 0; g < G1; ++g) load1(c0 + g * kBK, f[g]);
        __builtin_amdgcn_sched_barrier(0);   // keep every load of the group ahead of the MFMAs
#pragma unroll
        for (int g = 0; g < G1; ++g) comp1(f[g]);
      }
    }
#pragma unroll
    for (int tr = 0; tr < TR; ++tr)
#pragma unroll
      for (int g = 0; g < NACC; ++g)
#pragma unroll
        for (int i = 0; i < 4; ++i) red[w][tr][g][i][lane] = acc[tr][g][i];
  }
  auto zsum = [&](int tr, int i, float (&z)[NACC]) {
#pragma unroll
    for (int g = 0; g < NACC; ++g) {
      float t = red[0][tr][g][i][lane];
#pragma unroll
      for (int q = 1; q < KW; ++q) t += red[q][tr][g][i][lane];
      z[g] = t;
    }
  };
  if constexpr (EPI) {
    const int i = w - KW;
    BwdPre<NCH> pre[TR];
    if (w >= KW) {
#pragma unroll
      for (int tr = 0; tr < TR; ++tr) {
        // rows past the level read its last row (unused), so the loads
        // are unconditional
        lstm_bwd_pre<NCH, COH>(n, rows.clamp(16 * tr + 4 * gq + i), n0 + r, pre[tr]);
      }
    }
    __syncthreads();
    if (w < KW) return;
#pragma unroll
    for (int tr = 0; tr < TR; ++tr) {
      const int p = rows.pos(16 * tr + 4 * gq + i);
      if (p < 0) continue;
      float z[NACC];
      zsum(tr, i, z);
      lstm_bwd_fin<NCH>(n, n0 + r, pre[tr], z[0], NCH == 2 ? z[1] : 0.f,
                        NCH == 2 ? z[NACC - 1] : 0.f);
    }
  } else {
    __syncthreads();
    const int i = w & 3;
#pragma unroll
    for (int tr = w >> 2; tr < TR; tr += KW / 4) {
      const int p = rows.pos(16 * tr + 4 * gq + i);
      if (p < 0) continue;
      float z[NACC];
      zsum(tr, i, z);
      lstm_bwd_scatter<NCH, COH>(n, p, n0 + r, z[0], NCH == 2 ? z[1] : 0.f,
                                 NCH == 2 ? z[NACC - 1] : 0.f);
    }
  }
}

template <int NCH, bool BF, int TR, int KW>
__global__ void __launch_bounds__(64 * (KW + 4)) k_lstm_bwd_level_sk(Net n, int off, int M) {
  __shared__ BwdRed<NCH, TR, KW> red;
  int rt, ut;
  xcd_tile(n.H / 16, rt, ut);
  lstm_bwd_sk_tile<NCH, BF, TR, KW, true>(n, RangeRows{off + rt * 16 * TR, off + M}, ut, red);
}

// ----------------------------------------------- persistent small-level loop
// Levels shrink towards the roots (each vertex of level t+1 has its own child
// on level t), so the small levels form a suffix of the schedule.  One
// cooperative launch runs that whole suffix: tiles of a level are spread over
// the grid, and a grid barrier separates dependent levels, instead of one or
// two kernel launches per level.  Level offsets are read on the device.
//
// Grid barrier: counters only grow (zeroed before the launch).  Barrier e
// completes when the root counter reaches (e+1) * groups; the last arrival
// publishes gen = e+1.  Waiting is bounded: after `spin` polls (kBarrierSpin
// unless the CAVS_PERSIST_SPIN test hook sets another; a negative value gives
// up at once) the barrier records an error flag -- in the workspace and in
// the context's mapped host word, which cavs_sync reports -- and returns
// rather than hang.  The launch's results are then invalid.
constexpr int kBarrierSpin = 1 << 24;

struct GridBar {
  int* cnt;   // [1 + groups]: root, then one counter per group of 16 workgroups
  int* gen;
  int* err;
  int* host_err;   // mapped pinned word of the context (may be null)
  int spin;
};

__device__ __forceinline__ void grid_bar_gave_up(const GridBar& b) {
  atomicOr(b.err, 1);
  if (b.host_err) __hip_atomic_store(b.host_err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ __forceinline__ void grid_sync(const GridBar& b, int& epoch) {
  __syncthreads();
  if (threadIdx.x == 0) {
    const int G = gridDim.x, grp = blockIdx.x >> 4;
    const int gsize = min(16, G - (grp << 4)), ngroups = (G + 15) >> 4;
    __threadfence();   // release this workgroup's writes
    const int old = atomicAdd(&b.cnt[1 + grp], 1);
    bool release = false;
    if (old == epoch * gsize + gsize - 1) {
      const int o2 = atomicAdd(&b.cnt[0], 1);
      release = o2 == epoch * ngroups + ngroups - 1;
    }
    if (release) {
      __threadfence();
      atomicAdd(b.gen, 1);
    } else if (b.spin < 0) {
      grid_bar_gave_up(b);
    } else {
      int it = 0;
      while (__hip_atomic_load(b.gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <= epoch) {
        if (++it > b.spin) {
          grid_bar_gave_up(b);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    __threadfence();   // acquire
  }
  ++epoch;
  __syncthreads();
}

template <int NCH, bool BF>
__global__ void __launch_bounds__(256) k_lstm_fwd_persist(Net n, const int* lo, int t0, int t1,
                                                          GridBar bar) {
  __shared__ FwdRed<NCH, 1> red;
  const int ut = n.H / 16;
  int epoch = 0;
  for (int t = t0; t < t1; ++t) {
    const int off = lo[t], M = lo[t + 1] - off;
    const int tiles = cdiv_dev(M, 16) * ut;
    for (int tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
      lstm_fwd_sk_tile<NCH, BF, 1, 4, false>(n, RangeRows{off + tile / ut * 16, off + M}, tile % ut,
                                             red);
      __syncthreads();
    }
    if (t + 1 < t1) grid_sync(bar, epoch);
  }
}

// Levels t1-1 down to t0 (all with children): the dh_k products, whose
// epilogue forms the children's dA, then a barrier.
template <int NCH, bool BF>
__global__ void __launch_bounds__(256) k_lstm_bwd_persist(Net n, const int* lo, int t0, int t1,
                                                          GridBar bar) {
  __shared__ BwdRed<NCH, 1> red;
  const int ut = n.H / 16;
  int epoch = 0;
  for (int t = t1 - 1; t >= t0; --t) {
    const int off = lo[t], M = lo[t + 1] - off;
    const int tiles = cdiv_dev(M, 16) * ut;
    for (int tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
      lstm_bwd_sk_tile<NCH, BF, 1, 4, false>(n, RangeRows{off + tile / ut * 16, off + M}, tile % ut,
                                             red);
      __syncthreads();
    }
    if (t > t0) grid_sync(bar, epoch);
  }
}
}  // namespace

void lstm_fwd_leaf(const Net& n, int off, int M, bool skip_pulled, hipStream_t s) {
  if (M <= 0) return;
  CAVS_LAUNCH_ROWS("k_lstm_leaf", off, M, k_lstm_leaf, dim3(cdiv((long)M * n.H, 256)), dim3(256), 0,
                   s, n, off, M, (int)skip_pulled);
}

// bf16 levels from this many positions (below the tile threshold) run the
// split-K products with two 16-position row tiles per workgroup and four
// contraction wavefronts: each weight fragment loaded serves 32 positions,
// where the levels of 64-256 positions are bound by the operand stream.
// Measured on the H = 1024 batch: 7.60 -> 7.18 ms per step; from 32 or 96
// positions it gains less, and the smallest levels need the eight-wavefront
// split's parallelism.
constexpr int kSkTwoRowsFrom = 64;

void lstm_fwd_level(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  if (lstm_tile_applies(n, M)) {
    lstm_fwd_tile(n, off, M, s);
    return;
  }
  if (n.H % 256 == 0) {
    const bool kw8 = (n.H / 8) % 64 == 0;
    dim3 g(cdiv(M, 16) * (n.H / 16));
    if (n.bf && M >= kSkTwoRowsFrom) {
      dim3 g2(cdiv(M, 32) * (n.H / 16));
      if (n.N == 2)
        CAVS_LAUNCH_ROWS("k_lstm_fwd_level_sk<2, true, 2, 4>", off, M,
                         (k_lstm_fwd_level_sk<2, true, 2, 4>), g2, dim3(512), 0, s, n, off, M);
      else
        CAVS_LAUNCH_ROWS("k_lstm_fwd_level_sk<1, true, 2, 4>", off, M,
                         (k_lstm_fwd_level_sk<1, true, 2, 4>), g2, dim3(512), 0, s, n, off, M);
      return;
    }
#define CAVS_FWD_SK(NCH, BF)                                                                   \
  do {                                                                                         \
    if (kw8) CAVS_LAUNCH_ROWS("k_lstm_fwd_level_sk<" #NCH ", " #BF ", 1, 8>", off, M,            \
                              (k_lstm_fwd_level_sk<NCH, BF, 1, 8>), g, dim3(768), 0, s, n, off, M); \
    else CAVS_LAUNCH_ROWS("k_lstm_fwd_level_sk<" #NCH ", " #BF ", 1, 4>", off, M,                \
                          (k_lstm_fwd_level_sk<NCH, BF, 1, 4>), g, dim3(512), 0, s, n, off, M);  \
  } while (0)
    if (n.N == 2) {
      if (n.bf) CAVS_FWD_SK(2, true);
      else CAVS_FWD_SK(2, false);
    } else {
      if (n.bf) CAVS_FWD_SK(1, true);
      else CAVS_FWD_SK(1, false);
    }
#undef CAVS_FWD_SK
    return;
  }
  const bool small = M <= 32;
  dim3 grid = small ? dim3(cdiv(M, 16), n.H / 64) : dim3(cdiv(M, 64), n.H / 16);
#define CAVS_FWD(NCH, BM)                                                                      \
  do {                                                                                         \
    if (n.bf) CAVS_LAUNCH_ROWS("k_lstm_fwd_level_bf<" #NCH ", " #BM ">", off, M, (k_lstm_fwd_level_bf<NCH, BM>), \
                          grid, dim3(256), 0, s, n, off, M);                                   \
    else if (BM == 64 && xcd)                                                                  \
      CAVS_LAUNCH_ROWS("k_lstm_fwd_level<" #NCH ", 64, 2, xcd>", off, M,                        \
                       (k_lstm_fwd_level<NCH, 64, 2, true>), dim3(cdiv(M, 64) * (n.H / 32)),     \
                       dim3(256), 0, s, n, off, M);                                            \
    else CAVS_LAUNCH_ROWS("k_lstm_fwd_level<" #NCH ", " #BM ">", off, M, (k_lstm_fwd_level<NCH, BM, BM / 16, false>), grid,    \
                     dim3(256), 0, s, n, off, M);                                              \
  } while (0)
  const bool xcd = (n.H / 32) % 8 == 0;
  if (small) {
    if (n.N == 2) CAVS_FWD(2, 16);
    else CAVS_FWD(1, 16);
  } else {
    if (n.N == 2) CAVS_FWD(2, 64);
    else CAVS_FWD(1, 64);
  }
#undef CAVS_FWD
}

void lstm_bwd_gates(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  // level 0 (off == 0) holds the leaves, which have no children; an internal
  // bf16 level also gets the bf16 copy of its dA (its product's operand)
  const dim3 g4(cdiv((long)M * (n.H / 4), 256));
  const int wb = n.dAb && off > 0;
#define CAVS_G4(NCH, LEAF)                                                                   \
  CAVS_LAUNCH_ROWS("k_lstm_bwd_gates4<" #NCH ", " #LEAF ">", off, M,                          \
                   (k_lstm_bwd_gates4<NCH, LEAF>), g4, dim3(256), 0, s, n, off, M, wb)
  if (n.N == 2) {
    if (off == 0) CAVS_G4(2, true);
    else CAVS_G4(2, false);
  } else {
    if (off == 0) CAVS_G4(1, true);
    else CAVS_G4(1, false);
  }
#undef CAVS_G4
}

void lstm_bwd_roots(const Net& n, hipStream_t s) {
  if (n.fuse_from >= n.V) return;
  CAVS_LAUNCH("k_lstm_bwd_roots", k_lstm_bwd_roots, dim3(n.V - n.fuse_from), dim3(256), 0, s, n);
}

int lstm_fuse_level(const int* lo_host, int T) {
  for (int t = 0; t < T; ++t)
    if (lo_host[t + 1] - lo_host[t] <= kFuseRows) return t;
  return T;
}

void lstm_bwd_level(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  if (lstm_tile_applies(n, M)) {
    lstm_bwd_tile(n, off, M, s);
    return;
  }
  if (n.H % 256 == 0) {
    // eight K wavefronts at most 128 positions (one round); four above, where
    // two workgroups per CU keep the whole level co-resident
    const bool kw8 = (n.H / 8) % 64 == 0 && (3 * n.H / 8) % 64 == 0 && M <= 128;
    dim3 g(cdiv(M, 16) * (n.H / 16));
    if (n.bf && M >= kSkTwoRowsFrom) {
      dim3 g2(cdiv(M, 32) * (n.H / 16));
      if (n.N == 2)
        CAVS_LAUNCH_ROWS("k_lstm_bwd_level_sk<2, true, 2, 4>", off, M,
                         (k_lstm_bwd_level_sk<2, true, 2, 4>), g2, dim3(512), 0, s, n, off, M);
      else
        CAVS_LAUNCH_ROWS("k_lstm_bwd_level_sk<1, true, 2, 4>", off, M,
                         (k_lstm_bwd_level_sk<1, true, 2, 4>), g2, dim3(512), 0, s, n, off, M);
      return;
    }
#define CAVS_BWD_SK(NCH, BF)                                                                   \
  do {                                                                                         \
    if (kw8) CAVS_LAUNCH_ROWS("k_lstm_bwd_level_sk<" #NCH ", " #BF ", 1, 8>", off, M,            \
                              (k_lstm_bwd_level_sk<NCH, BF, 1, 8>), g, dim3(768), 0, s, n, off, M); \
    else CAVS_LAUNCH_ROWS("k_lstm_bwd_level_sk<" #NCH ", " #BF ", 1, 4>", off, M,                \
                          (k_lstm_bwd_level_sk<NCH, BF, 1, 4>), g, dim3(512), 0, s, n, off, M);  \
  } while (0)
    if (n.N == 2) {
      if (n.bf) CAVS_BWD_SK(2, true);
      else CAVS_BWD_SK(2, false);
    } else {
      if (n.bf) CAVS_BWD_SK(1, true);
      else CAVS_BWD_SK(1, false);
    }
#undef CAVS_BWD_SK
    return;
  }
  const bool small = M <= 32;
  dim3 grid(cdiv(M, small ? 16 : 64), n.H / 64);
#define CAVS_BWD(NCH, BM)                                                                      \
  do {                                                                                         \
    if (n.bf) CAVS_LAUNCH_ROWS("k_lstm_bwd_level_bf<" #NCH ", " #BM ">", off, M, (k_lstm_bwd_level_bf<NCH, BM>), \
                          grid, dim3(256), 0, s, n, off, M);                                   \
    else CAVS_LAUNCH_ROWS("k_lstm_bwd_level<" #NCH ", " #BM ">", off, M, (k_lstm_bwd_level<NCH, BM>), grid,    \
                     dim3(256), 0, s, n, off, M);                                              \
  } while (0)
  if (small) {
    if (n.N == 2) CAVS_BWD(2, 16);
    else CAVS_BWD(1, 16);
  } else {
    if (n.N == 2) CAVS_BWD(2, 64);
    else CAVS_BWD(1, 64);
  }
#undef CAVS_BWD
}

namespace {

// Levels of at most this many positions run in the persistent loop.
constexpr int kPersistRows = 256;

// The persistent loop is an opt-in ablation (CAVS_PERSIST=1): measured on
// MI355X, one grid barrier with the agent-scope fences it needs costs
// 2.7-17 us (32-512 workgroups) against 2.4 us for a back-to-back kernel
// launch, so per-level launches are the default.
bool persist_enabled() {
  const char* e = getenv("CAVS_PERSIST");
  return e && e[0] && e[0] != '0';
}

int coresident_blocks(const void* fn) {
  static std::map<const void*, int> cache;
  auto it = cache.find(fn);
  if (it != cache.end()) return it->second;
  int dev = 0, ncu = 0, per = 0, coop = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, fn, 256, 0) != hipSuccess || !coop)
    per = 0;
  const int v = per * ncu;
  cache[fn] = v;
  return v;
}

bool launch_persist(const char* name, const void* fn, const Net& n, const int* lo,
                    const int* lo_host, int t0, int t1, int* bar, int max_rows, hipStream_t s) {
  const int tiles = cdiv(max_rows, 16) * (n.H / 16);
  int G = coresident_blocks(fn);
  if (G > 512) G = 512;
  if (G > tiles) G = tiles;
  if (G <= 0) return false;
  int spin = kBarrierSpin;
  if (const char* e = getenv("CAVS_PERSIST_SPIN")) spin = atoi(e);
  GridBar gb{bar, bar + 64, bar + 65, t_active_ctx ? t_active_ctx->dev_err_dev : nullptr, spin};
  void* args[] = {(void*)&n, (void*)&lo, (void*)&t0, (void*)&t1, (void*)&gb};
  if (zero_async(bar, 256 * sizeof(int), s) != hipSuccess) return false;
  TimedScope ts(name, s, lo_host[t0], lo_host[t1] - lo_host[t0], /*bracket=*/true);
  return hipLaunchCooperativeKernel(fn, dim3(G), dim3(256), args, 0, s) == hipSuccess;
}

}  // namespace

// ------------------------------------------ XCD-local small-level loop
// The small levels near the roots in one launch per direction, without
// grid-wide barriers.  The graphs of a batch are independent, so the top of
// every tree (its positions in the suffix of small levels) is given to one
// of the eight XCDs, and the workgroups running on an XCD (its hardware id
// read from XCC_ID) process only their XCD's positions, level by level,
// separated by a barrier among themselves.  Everything one level writes and
// the next reads then stays inside one XCD: its CUs share one L2, stores
// reach it through the write-through L1, and the readers' device-scope
// loads (sc1) miss their own L1 and read it.  No level needs the L2
// write-back and invalidation that make a grid-wide barrier cost as much as
// a kernel launch.
constexpr int kXcdRows = 256;          // levels of at most this many positions
constexpr int kXcdMaxSuffix = 16384;   // suffix positions the owner kernel holds
constexpr int kXcdWords = 1024;        // barrier words
constexpr int kXcdSpin = 1 << 21;      // bounded waits (polls) before giving up
// contraction wavefronts of the weight-stationary tiles: the forward's
// partial sums are folded in pairs (its reduction buffer is that of four);
// the backward's buffer of eight fits beside its 16 rows of U.  Against
// four: 3.5 us less per SST-shaped forward loop, 15 us less per backward
// loop (104 us on 99 chain levels)
constexpr int kXcdFwdKW = 8;
constexpr int kXcdBwdKW = 8;

// Barrier words: [0] grid arrivals, [1] grid generation, [32 + x] the
// ticket (rank counter) of XCD x, [64 + 32 x] arrivals at XCD x's barrier,
// [64 + 32 x + 16] its generation.  Counters return to zero by themselves
// (the last arriver resets them); the owner kernel zeroes them first.
struct XcdLoop {
  int* w;
  const unsigned char* own;   // owner XCD of suffix position p (indexed p - base)
  int base;
  int spin;
  int* host_err;              // mapped pinned error word of the context (may be null)
};

__device__ __forceinline__ int xcc_id() {
  int v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return v & 7;
}

__device__ __forceinline__ int ld_sc1(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void xcd_gave_up(const XcdLoop& xl) {
  atomicOr(&xl.w[2], 1);
  if (xl.host_err) __hip_atomic_store(xl.host_err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Owner of every suffix position: the rank of its tree's root among the
// suffix roots (in position order), modulo 8.  Roots by pointer doubling in
// LDS (a parent always lies in the suffix: it is on a higher level).  One
// workgroup; also clears the barrier words.
__global__ void __launch_bounds__(1024) k_xcd_owner(const int* __restrict__ parent_pos, int base,
                                                    int S, unsigned char* __restrict__ own,
                                                    int* __restrict__ words) {
  __shared__ short ra[kXcdMaxSuffix], rb[kXcdMaxSuffix];
  __shared__ int wcnt[16], changed[2];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  for (int i = tid; i < kXcdWords; i += 1024) words[i] = 0;
  for (int q = tid; q < S; q += 1024) {
    const int pp = parent_pos[base + q];
    ra[q] = (short)(pp >= base && pp < base + S ? pp - base : q);
  }
  if (tid < 2) changed[tid] = 0;
  __syncthreads();
  short* a = ra;
  short* b = rb;
  for (int it = 0; it < 16; ++it) {   // 2^15 > kXcdMaxSuffix: enough rounds
    int ch = 0;
    for (int q = tid; q < S; q += 1024) {
      const short v = a[a[q]];
      b[q] = v;
      ch |= v != a[q];
    }
    if (ch) changed[it & 1] = 1;
    __syncthreads();
    const bool more = changed[it & 1] != 0;
    if (tid == 0) changed[(it + 1) & 1] = 0;
    short* t = a;
    a = b;
    b = t;
    __syncthreads();
    if (!more) break;
  }
  // ranks of the roots (a[q] == q) in position order: each thread a
  // contiguous chunk, a block-wide exclusive scan of the chunk counts
  const int per = (S + 1023) / 1024, q0 = min(S, tid * per), q1 = min(S, q0 + per);
  int c = 0;
  for (int q = q0; q < q1; ++q) c += a[q] == q;
  int incl = c;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wcnt[wv] = incl;
  __syncthreads();
  int rank = incl - c;
  for (int k = 0; k < wv; ++k) rank += wcnt[k];
  for (int q = q0; q < q1; ++q)
    if (a[q] == q) b[q] = (short)(rank++);
  __syncthreads();
  for (int q = tid; q < S; q += 1024) own[q] = (unsigned char)(b[a[q]] & 7);
}

// Group formation: rank of this workgroup among those on its XCD (s[1],
// known at once), then, after a one-time grid-wide arrival, their number
// (s[2]: every ticket is final).  Work that needs only the rank can run
// between the two halves.
__device__ __forceinline__ void xcd_arrive(const XcdLoop& xl, int* s) {
  if (threadIdx.x == 0) {
    const int x = xcc_id();
    const int rank = atomicAdd(&xl.w[32 + x], 1);
    const int g0 = ld_sc1(&xl.w[1]);
    __builtin_amdgcn_s_waitcnt(0);
    const int old = atomicAdd(&xl.w[0], 1);
    if (old == (int)gridDim.x - 1) {
      atomicExch(&xl.w[0], 0);
      __builtin_amdgcn_s_waitcnt(0);
      atomicAdd(&xl.w[1], 1);
      s[5] = -1;   // released the grid: nothing to wait for
    } else {
      s[5] = g0;
    }
    s[0] = x;
    s[1] = rank;
  }
  __syncthreads();
}

__device__ __forceinline__ void xcd_wait(const XcdLoop& xl, int* s) {
  if (threadIdx.x == 0) {
    const int x = s[0], g0 = s[5];
    if (g0 != -1) {
      int it = 0;
      while (ld_sc1(&xl.w[1]) == g0) {
        if (++it > xl.spin || ld_sc1(&xl.w[2])) {
          xcd_gave_up(xl);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    s[2] = ld_sc1(&xl.w[32 + x]);
    s[3] = ld_sc1(&xl.w[64 + 32 * x + 16]);
    s[4] = ld_sc1(&xl.w[2]);
  }
  __syncthreads();
}

__device__ __forceinline__ void xcd_begin(const XcdLoop& xl, int* s) {
  xcd_arrive(xl, s);
  xcd_wait(xl, s);
}

// Barrier among the gs workgroups of XCD x; s[3] is the generation this
// workgroup waits to see change, s[4] set when a wait gave up.  touch()
// runs between arriving and leaving: loads of the next level's static
// operands (schedule rows, saved state), issued while the barrier is
// pending so that the next tile finds them in cache.
template <class Touch>
__device__ __forceinline__ void xcd_sync(const XcdLoop& xl, int x, int gs, int* s, Touch&& touch) {
  __builtin_amdgcn_s_waitcnt(0);   // this wavefront's stores have reached the L2
  __syncthreads();
  int* cnt = &xl.w[64 + 32 * x];
  int* gen = cnt + 16;
  bool last = false;
  if (threadIdx.x == 0) {
    last = atomicAdd(cnt, 1) == gs - 1;
    if (last) {
      atomicExch(cnt, 0);
      __builtin_amdgcn_s_waitcnt(0);
      atomicAdd(gen, 1);
    }
  }
  const float keep = touch();
  if (threadIdx.x == 0) {
    const int g0 = s[3];
    if (!last) {
      int it = 0;
      while (ld_sc1(gen) == g0) {
        if (++it > xl.spin || ld_sc1(&xl.w[2])) {
          xcd_gave_up(xl);
          s[4] = 1;
          break;
        }
      }
    }
    s[3] = g0 + 1;
  }
  if (keep == 1.5e-44f) s[6] = 1;   // never true; keeps the touch loads
  __syncthreads();
}

__device__ __forceinline__ void xcd_sync(const XcdLoop& xl, int x, int gs, int* s) {
  xcd_sync(xl, x, gs, s, [] { return 0.f; });
}

// The static operands of the first row tile of a level (positions
// base + lst[0 .. m)) for unit / column tile u0, as the split-K tiles with
// KW contraction wavefronts read them: their child positions, and the
// epilogue wavefronts' prefetch (forward: lstm_fwd_pre; backward:
// lstm_bwd_pre, whose dL/dc word may be stale here and is read again
// coherently by the tile).
template <int NCH, bool FWD, int KW = 4>
__device__ __forceinline__ float xcd_touch(const Net& n, const short* lst, int m, int base, int u0) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, gq = lane >> 4, r = lane & 15;
  if (m <= 0) return 0.f;
  float acc = 0.f;
  if (w < KW) {
    const int p = base + lst[min(r, m - 1)];
#pragma unroll
    for (int c = 0; c < NCH; ++c) acc += (float)n.child_pos[(size_t)p * NCH + c];
  } else if (w < KW + 4) {
    const int p = base + lst[min(4 * gq + (w - KW), m - 1)];
    if constexpr (FWD) {
      FwdPre<NCH> q;
      lstm_fwd_pre<NCH, false>(n, p, u0 + r, q);
      acc += q.bi + q.pi + q.fb + q.cc[0];
    } else {
      BwdPre<NCH> e;
      lstm_bwd_pre<NCH, false>(n, p, u0 + r, e);
      acc += e.q[0].ig + e.q[0].c + e.q[0].ck[0] + e.q[0].lg;
    }
  }
  return acc;
}

// This XCD's positions of the level [l0, l1) (offsets from l0, in order)
// into lst and their number into *m; wavefront 0.
__device__ __forceinline__ void xcd_level_list(const XcdLoop& xl, int x, int l0, int l1,
                                               short* lst, int* m) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    int cnt = 0;
    for (int i0 = l0; i0 < l1; i0 += 64) {
      const int p = i0 + lane;
      const bool mine = p < l1 && xl.own[p - xl.base] == x;
      const unsigned long long bal = __ballot(mine);
      if (mine) lst[cnt + __popcll(bal & ((1ull << lane) - 1ull))] = (short)(p - l0);
      cnt += __popcll(bal);
    }
    if (lane == 0) *m = cnt;
  }
}

template <int NCH, bool BF>
__global__ void __launch_bounds__(768) k_lstm_fwd_xcd(Net n, const int* lo, int t0, int t1,
                                                      XcdLoop xl) {
  __shared__ FwdRed<NCH, 1, 8> red;
  __shared__ short lst[2][kXcdRows];
  __shared__ int s[8];
  __shared__ int sm[2];
  xcd_begin(xl, s);
  const int x = s[0], rank = s[1], gs = s[2];
  const int nut = n.H / 16;
  xcd_level_list(xl, x, lo[t0], lo[t0 + 1], lst[0], &sm[0]);
  __syncthreads();
  for (int t = t0; t < t1 && !s[4]; ++t) {
    const int cur = (t - t0) & 1, m = sm[cur], base = lo[t];
    const int jobs = cdiv_dev(m, 16) * nut;
    for (int j = rank; j < jobs; j += gs) {
      const int rt = j / nut;
      lstm_fwd_sk_tile<NCH, BF, 1, 8, true, ListRows, true>(
          n, ListRows{lst[cur] + 16 * rt, m - 16 * rt, base}, j % nut, red);
      __syncthreads();
    }
    if (t + 1 < t1) xcd_level_list(xl, x, lo[t + 1], lo[t + 2], lst[cur ^ 1], &sm[cur ^ 1]);
    // the last barrier also tells every workgroup of the XCD that the
    // ticket (read at the start) can be cleared
    xcd_sync(xl, x, gs, s);
  }
  if (threadIdx.x == 0 && rank == 0 && !s[4]) atomicExch(&xl.w[32 + x], 0);
}

// Weight-stationary variant: with H = 16 x (workgroups per XCD), workgroup
// `rank` of an XCD owns unit tile `rank` for the whole loop and keeps that
// tile's weight columns (H x 64: four gates x 16 units) in LDS, so a level
// reads only the children's rows; every workgroup of an XCD runs every row
// tile of its XCD's positions at its unit tile.
template <bool BF>
struct WsLds {
  static constexpr int LD = kXcdWsH + (BF ? 8 : 4);   // padded row: conflict-free 16-byte reads
  static constexpr int BYTES = 64 * LD * (BF ? 2 : 4);
};

template <int NCH, bool BF, int KW>
__global__ void __launch_bounds__(64 * (KW + 4)) k_lstm_fwd_xcd_ws(Net n, const int* lo, int t0,
                                                                  int t1, XcdLoop xl) {
  constexpr int NT = 64 * (KW + 4), FOLD = KW > 4;
  using WS = WsLds<BF>;
  __shared__ __attribute__((aligned(16))) unsigned char wl[WS::BYTES];
  __shared__ FwdRed<NCH, 1, FOLD ? KW / 2 : KW> red;
  __shared__ short lst[2][kXcdRows];
  __shared__ int s[8];
  __shared__ int sm[2];
  xcd_arrive(xl, s);
  const int H = n.H, ut = min(s[1], H / 16 - 1);
  // this unit tile's weight columns (while the grid-wide arrival completes):
  // column c = 16 g + r is column g H + 16 ut + r of U
  for (int i = threadIdx.x; i < 64 * (H / 4); i += NT) {
    const int c = i / (H / 4), k4 = 4 * (i % (H / 4));
    const int col = (c >> 4) * H + 16 * ut + (c & 15);
    if constexpr (BF) {
      const u16* src = n.UTb + (size_t)col * H + k4;
      u16* d = reinterpret_cast<u16*>(wl) + c * WS::LD + k4;
      d[0] = src[0]; d[1] = src[1]; d[2] = src[2]; d[3] = src[3];
    } else {   // n.UT: U transposed, k-contiguous (written earlier in the pass)
      *reinterpret_cast<float4*>(reinterpret_cast<float*>(wl) + c * WS::LD + k4) =
          ldg4(n.UT + (size_t)col * H + k4);
    }
  }
  xcd_wait(xl, s);
  const int x = s[0], rank = s[1], gs = s[2];
  if (gs * 16 != H) {   // the host launches this only when it holds; record, do nothing
    if (threadIdx.x == 0) xcd_gave_up(xl);
    return;
  }
  xcd_level_list(xl, x, lo[t0], lo[t0 + 1], lst[0], &sm[0]);
  __syncthreads();
  for (int t = t0; t < t1 && !s[4]; ++t) {
    const int cur = (t - t0) & 1, m = sm[cur], base = lo[t];
    for (int rt = 0; rt < cdiv_dev(m, 16); ++rt) {
      lstm_fwd_sk_tile<NCH, BF, 1, KW, true, ListRows, true, WS::LD, FOLD>(
          n, ListRows{lst[cur] + 16 * rt, m - 16 * rt, base}, ut, red, wl);
      __syncthreads();
    }
    if (t + 1 < t1) xcd_level_list(xl, x, lo[t + 1], lo[t + 2], lst[cur ^ 1], &sm[cur ^ 1]);
    __syncthreads();
    const int nb = t + 1 < t1 ? lo[t + 1] : 0, nm = t + 1 < t1 ? sm[cur ^ 1] : 0;
    xcd_sync(xl, x, gs, s,
             [&] { return xcd_touch<NCH, true, KW>(n, lst[cur ^ 1], nm, nb, 16 * ut); });
  }
  if (threadIdx.x == 0 && rank == 0 && !s[4]) atomicExch(&xl.w[32 + x], 0);
}

template <bool BF>
struct WsLdsB {
  static constexpr int LD = 4 * kXcdWsH + (BF ? 8 : 4);   // rows n0 .. n0+15 of U, padded
  static constexpr int BYTES = 16 * LD * (BF ? 2 : 4);
};

// Backward, top level first: workgroup `rank` of an XCD owns output column
// tile `rank` (rows 16 rank .. 16 rank + 15 of U resident in LDS) and runs
// every row tile of its XCD's positions of a level; each child's dA (or,
// below the loop, its dL/dh) is finished in the epilogue.
template <int NCH, bool BF, int KW>
__global__ void __launch_bounds__(64 * (KW + 4)) k_lstm_bwd_xcd_ws(Net n, const int* lo, int t0,
                                                                  int t1, XcdLoop xl) {
  constexpr int NT = 64 * (KW + 4);
  using WS = WsLdsB<BF>;
  __shared__ __attribute__((aligned(16))) unsigned char wl[WS::BYTES];
  __shared__ BwdRed<NCH, 1, KW> red;
  __shared__ short lst[2][kXcdRows];
  __shared__ int s[8];
  __shared__ int sm[2];
  xcd_arrive(xl, s);
  const int H = n.H, H4 = 4 * H, ut = min(s[1], H / 16 - 1);
  for (int i = threadIdx.x; i < 16 * (H4 / 4); i += NT) {
    const int row = i / (H4 / 4), c4 = 4 * (i % (H4 / 4));
    const size_t src = (size_t)(16 * ut + row) * H4 + c4;
    if constexpr (BF) {
      u16* d = reinterpret_cast<u16*>(wl) + row * WS::LD + c4;
      d[0] = n.Ub[src]; d[1] = n.Ub[src + 1]; d[2] = n.Ub[src + 2]; d[3] = n.Ub[src + 3];
    } else {
      *reinterpret_cast<float4*>(reinterpret_cast<float*>(wl) + row * WS::LD + c4) = ldg4(n.U + src);
    }
  }
  xcd_wait(xl, s);
  const int x = s[0], rank = s[1], gs = s[2];
  if (gs * 16 != H) {
    if (threadIdx.x == 0) xcd_gave_up(xl);
    return;
  }
  xcd_level_list(xl, x, lo[t1 - 1], lo[t1], lst[0], &sm[0]);
  __syncthreads();
  for (int t = t1 - 1; t >= t0 && !s[4]; --t) {
    const int cur = (t1 - 1 - t) & 1, m = sm[cur], base = lo[t];
    for (int rt = 0; rt < cdiv_dev(m, 16); ++rt) {
      lstm_bwd_sk_tile<NCH, BF, 1, KW, true, ListRows, true, WS::LD>(
          n, ListRows{lst[cur] + 16 * rt, m - 16 * rt, base}, ut, red, wl);
      __syncthreads();
    }
    if (t > t0) xcd_level_list(xl, x, lo[t - 1], lo[t], lst[cur ^ 1], &sm[cur ^ 1]);
    __syncthreads();
    const int nb = t > t0 ? lo[t - 1] : 0, nm = t > t0 ? sm[cur ^ 1] : 0;
    xcd_sync(xl, x, gs, s,
             [&] { return xcd_touch<NCH, false, KW>(n, lst[cur ^ 1], nm, nb, 16 * ut); });
  }
  if (threadIdx.x == 0 && rank == 0 && !s[4]) atomicExch(&xl.w[32 + x], 0);
}

int persist_first_level(const Net& n, const int* lo_host, int T) {
  if (!persist_enabled() || n.H % 256 != 0) return T;
  for (int t = 1; t < T; ++t)
    if (lo_host[t + 1] - lo_host[t] <= kPersistRows) return t;
  return T;
}

bool lstm_fwd_persist(const Net& n, const int* lo, const int* lo_host, int t0, int t1, int* bar,
                      hipStream_t s) {
  if (t0 >= t1) return true;
  const int maxM = lo_host[t0 + 1] - lo_host[t0];
#define CAVS_FP(NCH, BF)                                                                   \
  launch_persist("k_lstm_fwd_persist<" #NCH ", " #BF ">",                                  \
                 reinterpret_cast<const void*>(&k_lstm_fwd_persist<NCH, BF>), n, lo, lo_host, \
                 t0, t1, bar, maxM, s)
  if (n.N == 2) return n.bf ? CAVS_FP(2, true) : CAVS_FP(2, false);
  return n.bf ? CAVS_FP(1, true) : CAVS_FP(1, false);
#undef CAVS_FP
}

// On by default where it measured faster than per-level launches: weights
// resident in LDS and a suffix of at least 8 small levels (each level then
// costs a tile and an XCD barrier instead of a launch, against a fixed start
// of about 10 us per direction).  CAVS_XCD_LOOP=1 takes it wherever it
// applies, =0 never.
constexpr int kXcdMinLevels = 8;

int xcd_mode() {
  const char* e = getenv("CAVS_XCD_LOOP");
  return e && e[0] ? (e[0] == '0' ? 0 : 1) : -1;
}

int xcd_first_level(const Net& n, const int* lo_host, int T) {
  const int mode = xcd_mode();
  if (mode == 0 || n.H % 256 != 0 || (n.H / 8) % 64 != 0) return T;
  if ((size_t)n.V * n.GW >= (1u << 29)) return T;   // 32-bit offsets of the coherent loads
  for (int t = 1; t < T; ++t)
    if (lo_host[t + 1] - lo_host[t] <= kXcdRows) {
      if (n.V - lo_host[t] > kXcdMaxSuffix) return T;
      for (int u = t + 1; u < T; ++u)   // every level of the loop fits its position lists
        if (lo_host[u + 1] - lo_host[u] > kXcdRows) return T;
      if (mode < 0 && (T - t < kXcdMinLevels || n.H != kXcdWsH)) return T;
      return t;
    }
  return T;
}

size_t xcd_ws_bytes(int V) { return (size_t)kXcdWords * 4 + (size_t)V; }

namespace {

template <int NCH, bool BF>
const void* xcd_kernel(bool fwd, bool ws) {
  if (fwd) return ws ? reinterpret_cast<const void*>(&k_lstm_fwd_xcd_ws<NCH, BF, kXcdFwdKW>)
                     : reinterpret_cast<const void*>(&k_lstm_fwd_xcd<NCH, BF>);
  return ws ? reinterpret_cast<const void*>(&k_lstm_bwd_xcd_ws<NCH, BF, kXcdBwdKW>) : nullptr;
}

// Owner kernel, then the launch of the forward or backward loop
// over levels [t0, T); false when none could be launched.
bool xcd_launch(bool fwd, const Net& n, const int* lo, const int* lo_host, int t0, int T,
                void* xws, bool owner_ready, hipStream_t s) {
  if (t0 >= T) return true;
  int* words = (int*)xws;
  unsigned char* own = (unsigned char*)xws + (size_t)kXcdWords * 4;
  const int base = lo_host[t0];
  int dev = 0, ncu = 0, per = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return false;
  const int G = ncu / 8 * 8;   // one workgroup per CU, the same number on every XCD
  // weight-stationary: one unit (column) tile per workgroup of an XCD
  const bool ws = n.H == kXcdWsH && G / 8 * 16 == n.H;
  if (!ws && xcd_mode() < 0) return false;   // the default takes only the weight-stationary loop
  const void* fn = n.N == 2 ? (n.bf ? xcd_kernel<2, true>(fwd, ws) : xcd_kernel<2, false>(fwd, ws))
                            : (n.bf ? xcd_kernel<1, true>(fwd, ws) : xcd_kernel<1, false>(fwd, ws));
  const int threads = 768;   // eight contraction and four epilogue wavefronts
  if (!fn || G < 8 ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, fn, threads, 0) != hipSuccess || per < 1)
    return false;
  if (!owner_ready) xcd_owner(n, lo_host, t0, xws, s);
  int spin = kXcdSpin;
  if (const char* e = getenv("CAVS_PERSIST_SPIN")) spin = atoi(e);
  XcdLoop xl{words, own, base, spin, t_active_ctx ? t_active_ctx->dev_err_dev : nullptr};
  int a0 = t0, a1 = T;
  void* args[] = {(void*)&n, (void*)&lo, (void*)&a0, (void*)&a1, (void*)&xl};
  // timing names carry the template arguments, as the kernels' symbols do
  static_assert(kXcdFwdKW == 8 && kXcdBwdKW == 8, "timing names below");
  static const char* const kNames[3][2][2] = {
      {{"k_lstm_fwd_xcd<1, false>", "k_lstm_fwd_xcd<1, true>"},
       {"k_lstm_fwd_xcd<2, false>", "k_lstm_fwd_xcd<2, true>"}},
      {{"k_lstm_fwd_xcd_ws<1, false, 8>", "k_lstm_fwd_xcd_ws<1, true, 8>"},
       {"k_lstm_fwd_xcd_ws<2, false, 8>", "k_lstm_fwd_xcd_ws<2, true, 8>"}},
      {{"k_lstm_bwd_xcd_ws<1, false, 8>", "k_lstm_bwd_xcd_ws<1, true, 8>"},
       {"k_lstm_bwd_xcd_ws<2, false, 8>", "k_lstm_bwd_xcd_ws<2, true, 8>"}}};
  const char* name = kNames[fwd ? (ws ? 1 : 0) : 2][n.N == 2 ? 1 : 0][n.bf ? 1 : 0];
  TimedScope ts(name, s, lo_host[t0], lo_host[T] - lo_host[t0], /*bracket=*/true);
  // A plain launch: one workgroup per CU fits (checked above), and the
  // stream has drained every earlier kernel of the library, so on a device
  // shared with nobody else all G workgroups are resident at once.  The
  // cooperative launch API guarantees no more than that and measured about
  // 15 us slower per launch.  Should another process hold CUs, the
  // workgroups that are resident wait, boundedly, for the rest; a wait that
  // gives up is reported through cavs_sync.
  return hipLaunchKernel(fn, dim3(G), dim3(threads), args, 0, s) == hipSuccess;
}

}  // namespace

void xcd_owner(const Net& n, const int* lo_host, int t0, void* xws, hipStream_t s) {
  const int base = lo_host[t0];
  CAVS_LAUNCH("k_xcd_owner", k_xcd_owner, dim3(1), dim3(1024), 0, s, n.parent_pos, base,
              n.V - base, (unsigned char*)xws + (size_t)kXcdWords * 4, (int*)xws);
}

bool lstm_fwd_xcd(const Net& n, const int* lo, const int* lo_host, int t0, int T, void* xws,
                  bool owner_ready, hipStream_t s) {
  return xcd_launch(true, n, lo, lo_host, t0, T, xws, owner_ready, s);
}

bool lstm_bwd_xcd(const Net& n, const int* lo, const int* lo_host, int t0, int T, void* xws,
                  bool owner_ready, hipStream_t s) {
  return xcd_launch(false, n, lo, lo_host, t0, T, xws, owner_ready, s);
}

bool lstm_bwd_persist(const Net& n, const int* lo, const int* lo_host, int t0, int t1, int* bar,
                      hipStream_t s) {
  if (t0 >= t1) return true;
  const int maxM = lo_host[t0 + 1] - lo_host[t0];
#define CAVS_BP(NCH, BF)                                                                   \
  launch_persist("k_lstm_bwd_persist<" #NCH ", " #BF ">",                                  \
                 reinterpret_cast<const void*>(&k_lstm_bwd_persist<NCH, BF>), n, lo, lo_host, \
                 t0, t1, bar, maxM, s)
  if (n.N == 2) return n.bf ? CAVS_BP(2, true) : CAVS_BP(2, false);
  return n.bf ? CAVS_BP(1, true) : CAVS_BP(1, false);
#undef CAVS_BP
}

}  // namespace cavs
