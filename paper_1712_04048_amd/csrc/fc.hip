// Tree-FC vertex function (Section 5, Tree-FC: a single fully-connected layer
// as the cell): internal vertex h = tanh(h_0 W_0 + h_1 W_1 + b); a leaf's
// state is its pulled input.  One batching task (level) per launch.
#include "kernels.h"

namespace cavs {
namespace {

__global__ void __launch_bounds__(256) k_fc_leaf(Net n, int off, int M) {
  const int H = n.H;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)M * H) return;
  const int p = off + (int)(idx / H), j = (int)(idx % H);
  const float h = n.X[(size_t)n.pull_pos[p] * H + j];
  n.Hs[(size_t)p * H + j] = h;
  n.h_out[(size_t)n.order[p] * H + j] = h;
}

// z = [h_0, h_1] W + b over a tile of BM positions x 64 units; K = 2H runs
// through child slot 0's rows then slot 1's (gathered from the state buffer).
template <int BM>
__global__ void __launch_bounds__(256) k_fc_fwd_level(Net n, int off, int M) {
  constexpr int BN = 64;
  constexpr int WRW = BM == 64 ? 2 : 1, WCW = 4 / WRW;
  constexpr int TM = BM / 16 / WRW, TN = BN / 16 / WCW;
  constexpr int LDA = kBK + 4, LDB = BN + 2;
  constexpr int A_N = BM * 8, A_PER = (A_N + 255) / 256;
  constexpr int B_PER = kBK * (BN / 4) / 256;
  __shared__ __attribute__((aligned(16))) float As[BM * LDA];
  __shared__ float Bs[kBK * LDB];
  const int H = n.H, N = n.N;
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
  // child rows of this thread's A row, looked up once (slots 0 and 1)
  const float* crow[A_PER][2];
#pragma unroll
  for (int a = 0; a < A_PER; ++a)
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      crow[a][k] = nullptr;
      if (aval[a] && k < N) {
        const int cp = n.child_pos[(size_t)(row0 + arow[a]) * N + k];
        if (cp >= 0) crow[a][k] = n.Hs + (size_t)cp * H + 4 * aq[a];
      }
    }
  float4 ra[A_PER], rb[B_PER];
  auto gload = [&](int kc) {
    const int k0 = kc * kBK, slot = k0 / H, r0 = k0 % H;
#pragma unroll
    for (int a = 0; a < A_PER; ++a) {
      const float* src = slot == 0 ? crow[a][0] : crow[a][1];
      ra[a] = src ? ldg4(src + r0) : f4zero();
    }
#pragma unroll
    for (int b = 0; b < B_PER; ++b) {
      const int idx = tid + 256 * b, kk = idx / (BN / 4), q = idx % (BN / 4);
      rb[b] = ldg4(n.U + (size_t)(k0 + kk) * H + n0 + 4 * q);
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int a = 0; a < A_PER; ++a)
      if (tid + 256 * a < A_N) st4(&As[arow[a] * LDA + 4 * aq[a]], ra[a]);
#pragma unroll
    for (int b = 0; b < B_PER; ++b) {
      const int idx = tid + 256 * b, kk = idx / (BN / 4), q = idx % (BN / 4);
      st4_scalar(&Bs[kk * LDB + 4 * q], rb[b]);
    }
  };
  v4f acc[TM][TN];
  zero_acc(acc);
  const int nk = N * H / kBK;
  gload(0);
  for (int kc = 0; kc < nk; ++kc) {
    __syncthreads();
    sstore();
    __syncthreads();
    if (kc + 1 < nk) gload(kc + 1);
    mfma_chunk<TM, TN, true, false, LDA, LDB>(As, Bs, wrow, wcol, acc);
  }
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = row0 + wrow + tm * 16 + 4 * gq + i;
      if (p >= rowend) continue;
      const int v = n.order[p];
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int col = n0 + wcol + tn * 16 + r;
        const float h = tanh_(acc[tm][tn][i] + n.b[col]);
        n.Hs[(size_t)p * H + col] = h;
        n.h_out[(size_t)v * H + col] = h;
      }
    }
}

// delta = dL/dh * (1 - h^2) for internal vertices; a leaf passes dL/dh to
// its input row (h = x).
__global__ void __launch_bounds__(256) k_fc_bwd_gates(Net n, int off, int M, int leaf,
                                                      float* dX) {
  const int H = n.H;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)M * H) return;
  const int p = off + (int)(idx / H), j = (int)(idx % H);
  const int par = n.parent_pos[p];
  float gh = par >= 0 ? n.dHp[(size_t)p * H + j] : 0.f;
  const float h = n.Hs[(size_t)p * H + j];
  gh += n.dHL[(size_t)p * H + j];
  if (leaf) dX[(size_t)n.pull_pos[p] * H + j] = gh;
  else n.dA[(size_t)p * H + j] = gh * (1.f - h * h);
}

// dL/dh_k = delta W_k^T for both child slots; tile BM positions x 64 units.
template <int BM>
__global__ void __launch_bounds__(256) k_fc_bwd_level(Net n, int off, int M) {
  constexpr int BN = 64;
  constexpr int WRW = BM == 64 ? 2 : 1, WCW = 4 / WRW;
  constexpr int TM = BM / 16 / WRW, TN = BN / 16 / WCW;
  constexpr int LDA = kBK + 4, LDB = kBK + 4;
  constexpr int A_N = BM * 8, A_PER = (A_N + 255) / 256;
  constexpr int B_PER = BN * 8 / 256;
  __shared__ __attribute__((aligned(16))) float As[BM * LDA];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN * LDB];
  const int H = n.H, N = n.N;
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
  float4 ra[A_PER], rb[2][B_PER];
  auto gload = [&](int k0) {
#pragma unroll
    for (int a = 0; a < A_PER; ++a)
      ra[a] = aval[a] ? ldg4(n.dA + (size_t)(row0 + arow[a]) * H + k0 + 4 * aq[a]) : f4zero();
#pragma unroll
    for (int b = 0; b < B_PER; ++b) {
      const int idx = tid + 256 * b, nr = idx / 8, q = idx % 8;
#pragma unroll
      for (int k = 0; k < 2; ++k)
        rb[k][b] = k < N ? ldg4(n.U + (size_t)(k * H + n0 + nr) * H + k0 + 4 * q) : f4zero();
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int a = 0; a < A_PER; ++a)
      if (tid + 256 * a < A_N) st4(&As[arow[a] * LDA + 4 * aq[a]], ra[a]);
#pragma unroll
    for (int b = 0; b < B_PER; ++b) {
      const int idx = tid + 256 * b, nr = idx / 8, q = idx % 8;
      st4(&Bs[0][nr * LDB + 4 * q], rb[0][b]);
      st4(&Bs[1][nr * LDB + 4 * q], rb[1][b]);
    }
  };
  v4f acc0[TM][TN], acc1[TM][TN];
  zero_acc(acc0);
  zero_acc(acc1);
  const int nk = H / kBK;
  gload(0);
  for (int kc = 0; kc < nk; ++kc) {
    __syncthreads();
    sstore();
    __syncthreads();
    if (kc + 1 < nk) gload((kc + 1) * kBK);
    mfma_chunk<TM, TN, true, true, LDA, LDB>(As, Bs[0], wrow, wcol, acc0);
    mfma_chunk<TM, TN, true, true, LDA, LDB>(As, Bs[1], wrow, wcol, acc1);
  }
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = row0 + wrow + tm * 16 + 4 * gq + i;
      if (p >= rowend) continue;
      const int cp0 = n.child_pos[(size_t)p * N];
      const int cp1 = N == 2 ? n.child_pos[(size_t)p * N + 1] : -1;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int col = n0 + wcol + tn * 16 + r;
        if (cp0 >= 0) n.dHp[(size_t)cp0 * H + col] = acc0[tm][tn][i];
        if (cp1 >= 0) n.dHp[(size_t)cp1 * H + col] = acc1[tm][tn][i];
      }
    }
}

}  // namespace

void fc_fwd_leaf(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  CAVS_LAUNCH_ROWS("k_fc_leaf", off, M, k_fc_leaf, dim3(cdiv((long)M * n.H, 256)), dim3(256), 0, s, n, off, M);
}

void fc_fwd_level(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  if (M <= 32)
    CAVS_LAUNCH_ROWS("k_fc_fwd_level<16>", off, M, (k_fc_fwd_level<16>), dim3(cdiv(M, 16), n.H / 64), dim3(256), 0, s, n, off,
                       M);
  else
    CAVS_LAUNCH_ROWS("k_fc_fwd_level<64>", off, M, (k_fc_fwd_level<64>), dim3(cdiv(M, 64), n.H / 64), dim3(256), 0, s, n, off,
                       M);
}

void fc_bwd_gates(const Net& n, int off, int M, int leaf, float* dX, hipStream_t s) {
  if (M <= 0) return;
  CAVS_LAUNCH_ROWS("k_fc_bwd_gates", off, M, k_fc_bwd_gates, dim3(cdiv((long)M * n.H, 256)), dim3(256), 0, s, n, off, M,
                     leaf, dX);
}

void fc_bwd_level(const Net& n, int off, int M, hipStream_t s) {
  if (M <= 0) return;
  if (M <= 32)
    CAVS_LAUNCH_ROWS("k_fc_bwd_level<16>", off, M, (k_fc_bwd_level<16>), dim3(cdiv(M, 16), n.H / 64), dim3(256), 0, s, n, off,
                       M);
  else
    CAVS_LAUNCH_ROWS("k_fc_bwd_level<64>", off, M, (k_fc_bwd_level<64>), dim3(cdiv(M, 64), n.H / 64), dim3(256), 0, s, n, off,
                       M);
}

}  // namespace cavs
