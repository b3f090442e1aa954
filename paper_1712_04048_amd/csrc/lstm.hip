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
// Backward, reverse level order: an elementwise kernel turns dL/dh, dL/dc of
// the level into the pre-activation gradients dA (kept level-major for the
// lazy weight gradients) and scatters dL/dc_k = g_c * f_k to the children; a
// GEMM kernel computes dL/dh_k = dA_iou U_iou^T + dA_fk U_f^T and scatters it
// to child k.  Every vertex has one parent, so each child row is written by
// exactly one thread: plain stores, no atomics.
#include "kernels.h"

namespace cavs {
namespace {

// ------------------------------------------------------------------ forward
__global__ void __launch_bounds__(256) k_lstm_leaf(Net n, int off, int M) {
  const int H = n.H;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)M * H) return;
  const int p = off + (int)(idx / H), j = (int)(idx % H);
  const int pr = n.pull_pos[p];
  float ai = n.b[G_I * H + j], ao = n.b[G_O * H + j], au = n.b[G_U * H + j];
  if (pr >= 0) {
    const float* Pp = n.P + (size_t)p * 4 * H;
    ai += Pp[G_I * H + j];
    ao += Pp[G_O * H + j];
    au += Pp[G_U * H + j];
  }
  const float i = sigmoidf_(ai), o = sigmoidf_(ao), u = tanhf(au);
  const float c = i * u, h = o * tanhf(c);
  n.Hs[(size_t)p * H + j] = h;
  n.Cs[(size_t)p * H + j] = c;
  float* g = n.Gs + (size_t)p * n.GW;
  g[j] = i;
  g[H + j] = 0.f;
  g[2 * H + j] = o;
  g[3 * H + j] = u;
  if (n.N == 2) g[4 * H + j] = 0.f;
  const int v = n.order[p];
  n.h_out[(size_t)v * H + j] = h;
  if (n.c_out) n.c_out[(size_t)v * H + j] = c;
}

// Gates, cell update and the scatter of (c, h) for position p, unit j, from
// the matrix-product parts of the pre-activations (shared by both precisions).
template <int NCH>
__device__ __forceinline__ void lstm_fwd_epilogue(const Net& n, int p, int j, float zi, float zo,
                                                  float zu, float zf0, float zf1) {
  const int H = n.H, H4 = 4 * H;
  const int pr = n.pull_pos[p];
  float ai = zi + n.b[G_I * H + j], ao = zo + n.b[G_O * H + j], au = zu + n.b[G_U * H + j];
  float fb = n.b[G_F * H + j];
  if (pr >= 0) {
    const float* Pp = n.P + (size_t)p * H4;
    ai += Pp[G_I * H + j];
    ao += Pp[G_O * H + j];
    au += Pp[G_U * H + j];
    fb += Pp[G_F * H + j];
  }
  const float ig = sigmoidf_(ai), og = sigmoidf_(ao), ug = tanhf(au);
  float c = ig * ug;
  float f0 = 0.f, f1 = 0.f;
  const int cp0 = n.child_pos[(size_t)p * NCH];
  if (cp0 >= 0) {
    f0 = sigmoidf_(zf0 + fb);
    c += f0 * n.Cs[(size_t)cp0 * H + j];
  }
  if constexpr (NCH == 2) {
    const int cp1 = n.child_pos[(size_t)p * NCH + 1];
    if (cp1 >= 0) {
      f1 = sigmoidf_(zf1 + fb);
      c += f1 * n.Cs[(size_t)cp1 * H + j];
    }
  }
  const float h = og * tanhf(c);
  n.Hs[(size_t)p * H + j] = h;
  n.Cs[(size_t)p * H + j] = c;
  float* g = n.Gs + (size_t)p * n.GW;
  g[j] = ig;
  g[H + j] = f0;
  g[2 * H + j] = og;
  g[3 * H + j] = ug;
  if constexpr (NCH == 2) g[4 * H + j] = f1;
  const int v = n.order[p];
  n.h_out[(size_t)v * H + j] = h;
  if (n.c_out) n.c_out[(size_t)v * H + j] = c;
}

// Child scatter of the backward level product for position p, column col.
template <int NCH>
__device__ __forceinline__ void lstm_bwd_scatter(const Net& n, int p, int col, float zh, float zf0,
                                                 float zf1) {
  const int cp0 = n.child_pos[(size_t)p * NCH];
  if (cp0 >= 0) n.dHp[(size_t)cp0 * n.H + col] = zh + zf0;
  if constexpr (NCH == 2) {
    const int cp1 = n.child_pos[(size_t)p * NCH + 1];
    if (cp1 >= 0) n.dHp[(size_t)cp1 * n.H + col] = zh + zf1;
  }
}

// Tile: BM positions x BHU hidden units; 4 wavefronts arranged WR x WU, each
// owning 16 positions x 16 units and all (3 + NCH) gate accumulators for them.
template <int NCH, int BM>
__global__ void __launch_bounds__(256) k_lstm_fwd_level(Net n, int off, int M) {
  constexpr int WR = BM / 16, WU = 4 / WR, BHU = 16 * WU;
  constexpr int LDA = kBK + 4;
  constexpr int LDB = BHU + 2;
  constexpr int A_N = BM * NCH * (kBK / 4);          // float4 per chunk
  constexpr int A_PER = (A_N + 255) / 256;
  constexpr int B_ROW4 = BHU / 4;                    // float4 per (gate, k) row
  constexpr int B_N = 4 * kBK * B_ROW4;
  constexpr int B_PER = B_N / 256;
  static_assert(B_N % 256 == 0, "B tile must split evenly");
  __shared__ __attribute__((aligned(16))) float As[NCH][BM * LDA];
  __shared__ float Bs[4][kBK * LDB];

  const int H = n.H, H4 = 4 * H;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w % WR, wu = w / WR;
  const int row0 = off + blockIdx.x * BM;
  const int rowend = off + M;
  const int u0 = blockIdx.y * BHU;

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

  v4f acc_i = {0.f, 0.f, 0.f, 0.f}, acc_o = acc_i, acc_u = acc_i, acc_f0 = acc_i, acc_f1 = acc_i;
  gload(0);
  for (int k0 = 0; k0 < H; k0 += kBK) {
    __syncthreads();
    sstore();
    __syncthreads();
    if (k0 + kBK < H) gload(k0 + kBK);
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      float a0[4], a1[4], bi[4], bf[4], bo[4], bu[4];
      load_frag4<true, LDA>(As[0], wr * 16 + r, gq, half, a0);
      if constexpr (NCH == 2) load_frag4<true, LDA>(As[NCH - 1], wr * 16 + r, gq, half, a1);
      load_frag4<false, LDB>(Bs[G_I], wu * 16 + r, gq, half, bi);
      load_frag4<false, LDB>(Bs[G_F], wu * 16 + r, gq, half, bf);
      load_frag4<false, LDB>(Bs[G_O], wu * 16 + r, gq, half, bo);
      load_frag4<false, LDB>(Bs[G_U], wu * 16 + r, gq, half, bu);
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        float ah = a0[s];
        if constexpr (NCH == 2) ah = a0[s] + a1[s];
        acc_i = mfma_f32_16x16x4(ah, bi[s], acc_i);
        acc_o = mfma_f32_16x16x4(ah, bo[s], acc_o);
        acc_u = mfma_f32_16x16x4(ah, bu[s], acc_u);
        acc_f0 = mfma_f32_16x16x4(a0[s], bf[s], acc_f0);
        if constexpr (NCH == 2) acc_f1 = mfma_f32_16x16x4(a1[s], bf[s], acc_f1);
      }
    }
  }

  // epilogue: gates, cell update, scatter of (c, h)
  const int j = u0 + wu * 16 + r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int p = row0 + wr * 16 + 4 * gq + i;
    if (p < rowend) lstm_fwd_epilogue<NCH>(n, p, j, acc_i[i], acc_o[i], acc_u[i], acc_f0[i], acc_f1[i]);
  }
}

// ----------------------------------------------------------------- backward
__global__ void __launch_bounds__(256) k_lstm_bwd_gates(Net n, int off, int M) {
  const int H = n.H;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)M * H) return;
  const int p = off + (int)(idx / H), j = (int)(idx % H);
  const int par = n.parent_pos[p];
  float gh = par >= 0 ? n.dHp[(size_t)p * H + j] : 0.f;
  float gcin = par >= 0 ? n.dCp[(size_t)p * H + j] : 0.f;
  const int q = n.push_pos[p];
  if (q >= 0) {
    if (n.loss == CAVS_LOSS_CE) {
      const float* dz = n.dZ + (size_t)p * n.C;
      const float* ws = n.Ws + (size_t)j * n.C;
      float s = 0.f;
      for (int c = 0; c < n.C; ++c) s += dz[c] * ws[c];
      gh += s;
    } else {
      gh += (n.Hs[(size_t)p * H + j] - n.Y[(size_t)q * H + j]) * n.inv_denom;
    }
  }
  const float* g = n.Gs + (size_t)p * n.GW;
  const float ig = g[j], og = g[2 * H + j], ug = g[3 * H + j];
  const float c = n.Cs[(size_t)p * H + j];
  const float tau = tanhf(c);
  const float d_o = gh * tau * og * (1.f - og);
  const float gc = gcin + gh * og * (1.f - tau * tau);
  const float d_i = gc * ug * ig * (1.f - ig);
  const float d_u = gc * ig * (1.f - ug * ug);
  float* da = n.dA + (size_t)p * n.GW;
  for (int k = 0; k < n.N; ++k) {
    const int cp = n.child_pos[(size_t)p * n.N + k];
    const int col = k == 0 ? H : 4 * H;
    float d_f = 0.f;
    if (cp >= 0) {
      const float fk = g[col + j];
      d_f = gc * n.Cs[(size_t)cp * H + j] * fk * (1.f - fk);
      n.dCp[(size_t)cp * H + j] = gc * fk;
    }
    da[col + j] = d_f;
  }
  da[j] = d_i;
  da[2 * H + j] = d_o;
  da[3 * H + j] = d_u;
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
}  // namespace

void lstm_fwd_leaf(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  CAVS_LAUNCH("k_lstm_leaf", k_lstm_leaf, dim3(cdiv((long)M * n.H, 256)), dim3(256), 0, s, n, off, M);
}

void lstm_fwd_level(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  const bool small = M <= 32;
  dim3 grid = small ? dim3(cdiv(M, 16), n.H / 64) : dim3(cdiv(M, 64), n.H / 16);
#define CAVS_FWD(NCH, BM)                                                                      \
  do {                                                                                         \
    if (n.bf) CAVS_LAUNCH("k_lstm_fwd_level_bf<" #NCH ", " #BM ">", (k_lstm_fwd_level_bf<NCH, BM>), \
                          grid, dim3(256), 0, s, n, off, M);                                   \
    else CAVS_LAUNCH("k_lstm_fwd_level<" #NCH ", " #BM ">", (k_lstm_fwd_level<NCH, BM>), grid,    \
                     dim3(256), 0, s, n, off, M);                                              \
  } while (0)
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
  CAVS_LAUNCH("k_lstm_bwd_gates", k_lstm_bwd_gates, dim3(cdiv((long)M * n.H, 256)), dim3(256), 0, s, n, off,
                     M);
}

void lstm_bwd_level(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  const bool small = M <= 32;
  dim3 grid(cdiv(M, small ? 16 : 64), n.H / 64);
#define CAVS_BWD(NCH, BM)                                                                      \
  do {                                                                                         \
    if (n.bf) CAVS_LAUNCH("k_lstm_bwd_level_bf<" #NCH ", " #BM ">", (k_lstm_bwd_level_bf<NCH, BM>), \
                          grid, dim3(256), 0, s, n, off, M);                                   \
    else CAVS_LAUNCH("k_lstm_bwd_level<" #NCH ", " #BM ">", (k_lstm_bwd_level<NCH, BM>), grid,    \
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

}  // namespace cavs
