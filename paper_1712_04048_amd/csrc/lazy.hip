// Operators that are not on a gather->scatter path of F or dF and therefore
// run batched over all vertices at once (lazy batching, Section 3.5), plus
// the eager pull projection:
//   - pull:   P = X W_x for every vertex that pulls an input (one GEMM);
//   - push:   the loss head over every labelled vertex (z = h W_s + b_s);
//   - dF:     dW_x, dU, db, dX, dW_s, db_s as long-K products over all
//             vertices, with deterministic split-K (fixed-order reduction).
#include <algorithm>
#include <vector>

#include "lds_ring.h"
#include "lstm_dev.h"

namespace cavs {
namespace {

constexpr int kMaxSplits = 16;   // sizes the split-K scratch: 16 x (4H x H) floats
constexpr int kSplitCap = 32;    // more splits only where the scratch holds them

// ------------------------------------------------------------- pull GEMM
// P[p, n] = X[pull_pos[p], :] W_x[:, n] for p = pull_list[m]; tile 64 x 64.
// Column tiles cover the gate blocks i,f,o,u (with_f) or i,o,u.
// Pull projection P = x W_x fused with the cell of the pulled leaves: a
// workgroup owns 64 pulled rows x 32 hidden units for all NG gate blocks
// (i|o|u when no vertex with children pulls, else i|f|o|u); wavefront w owns
// rows 16w.. of the tile and every gate block of its units, so each lane
// holds all gates of its (row, unit).  A leaf row (position below lo1)
// finishes its cell here (h, c, saved gates, outputs); any other pulled row
// stores its P row for the level epilogue.  K = D runs in 32-deep chunks
// through two LDS stages (the last chunk zero-filled past D).
template <int NG>
__global__ void __launch_bounds__(256) k_pull_leaf(Net n, int n_pull, int lo1) {
  constexpr int BM = 64, BU = 32, NB = NG * BU / 16;
  constexpr int LDA = kBK + 4, LDB = NG * BU + 2;
  constexpr int B4 = NG * BU / 4;                     // float4 per B k-row
  __shared__ __attribute__((aligned(16))) float As[2][BM * LDA];
  __shared__ float Bs[2][kBK * LDB];
  const int H = n.H, H4 = 4 * H, D = n.D;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int m0 = blockIdx.x * BM, u0 = blockIdx.y * BU;
  auto gcol = [&](int g) { return NG == 4 ? g : (g == 0 ? G_I : g + 1); };
  const float* asrc[2];
  int adst[2], aq[2];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int idx = tid + 256 * a, row = idx / 8;
    aq[a] = idx % 8;
    adst[a] = row * LDA + 4 * aq[a];
    asrc[a] = m0 + row < n_pull ? n.X + (size_t)n.pull_pos[n.pull_list[m0 + row]] * D : nullptr;
  }
  float4 ra[2], rb[NG];
  auto gload = [&](int k0) {
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int k = k0 + 4 * aq[a];
      ra[a] = (asrc[a] && k < D) ? ldg4(asrc[a] + k) : f4zero();
    }
#pragma unroll
    for (int b = 0; b < NG; ++b) {
      const int idx = tid + 256 * b, kk = idx / B4, c = 4 * (idx % B4);
      rb[b] = k0 + kk < D ? ldg4(n.Wx + (size_t)(k0 + kk) * H4 + gcol(c / BU) * H + u0 + c % BU)
                          : f4zero();
    }
  };
  auto sstore = [&](int st) {
#pragma unroll
    for (int a = 0; a < 2; ++a) st4(&As[st][adst[a]], ra[a]);
#pragma unroll
    for (int b = 0; b < NG; ++b) {
      const int idx = tid + 256 * b, kk = idx / B4, c = 4 * (idx % B4);
      st4_scalar(&Bs[st][kk * LDB + c], rb[b]);
    }
  };
  auto barrier = []() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): this wave's LDS writes done
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  v4f acc[1][NB];
  zero_acc(acc);
  const int nk = (D + kBK - 1) / kBK;
  gload(0);
  sstore(0);
  barrier();
  for (int kc = 0; kc < nk; ++kc) {
    const int st = kc & 1;
    if (kc + 1 < nk) gload((kc + 1) * kBK);
    mfma_chunk<1, NB, true, false, LDA, LDB>(As[st], Bs[st], 16 * w, 0, acc);
    if (kc + 1 < nk) sstore(st ^ 1);
    barrier();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + 16 * w + 4 * gq + i;
    if (m >= n_pull) continue;
    const int p = n.pull_list[m];
#pragma unroll
    for (int ub = 0; ub < 2; ++ub) {
      const int j = u0 + 16 * ub + r;
      // block of gate g, unit block ub: columns [32 g + 16 ub, +16)
      if (p < lo1) {
        const float zi = acc[0][0 * 2 + ub][i];
        const float zo = acc[0][(NG == 4 ? 2 : 1) * 2 + ub][i];
        const float zu = acc[0][(NG == 4 ? 3 : 2) * 2 + ub][i];
        float ai = n.b[G_I * H + j], ao = n.b[G_O * H + j], au = n.b[G_U * H + j];
        ai += zi;
        ao += zo;
        au += zu;
        const float ig = sigmoidf_(ai), og = sigmoidf_(ao), ug = tanh_(au);
        const float c = ig * ug, h = og * tanh_(c);
        n.Hs[(size_t)p * H + j] = h;
        n.Cs[(size_t)p * H + j] = c;
        if (n.Gs) {   // a leaf's forget gates are never read; null in inference
          float* g = n.Gs + (size_t)p * n.GW;
          g[j] = ig;
          g[2 * H + j] = og;
          g[3 * H + j] = ug;
        }
        const int v = n.order[p];
        n.h_out[(size_t)v * H + j] = h;
        if (n.c_out) n.c_out[(size_t)v * H + j] = c;
      } else {
#pragma unroll
        for (int g = 0; g < NG; ++g) n.P[(size_t)p * H4 + gcol(g) * H + j] = acc[0][g * 2 + ub][i];
      }
    }
  }
}

// The same product on the direct-to-LDS ring of the level tiles: a
// workgroup owns 64 pulled rows x 32 units x NG gate blocks.  Stage rows:
// the 64 x rows (gathered through pull_list and pull_pos), then the rows of
// W_x^T for each gate block's 32 units; chunks past D read the zero row.
// Four wavefronts as 2 x 2 (32 rows x 16 units each); the weight fragment
// is the MFMA's A operand, so a lane holds four consecutive units of one
// row (float4 epilogue).  Fragments are double-buffered in registers.
template <int NG, int BM, int S>
__global__ void __launch_bounds__(256) k_pull_tile(Net n, int n_pull, int lo1) {
  constexpr int BU = 32, TM = BM / 32;
  constexpr int ROWS = BM + NG * BU, IPW = ROWS / 32;
  static_assert(IPW * 32 == ROWS && S >= 2 && S <= 4, "tile shape");
  __shared__ __attribute__((aligned(1024))) float L0[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L1[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L2[S > 2 ? ROWS * 32 : 4];
  __shared__ __attribute__((aligned(1024))) float L3[S > 3 ? ROWS * 32 : 4];
  const Ring<ROWS, S> ring{L0, L1, L2, L3};
  const int H = n.H, H4 = 4 * H, D = n.D;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w & 1, wu = w >> 1;
  int rt, ut;
  xcd_tile(H / BU, rt, ut);
  const int m0 = rt * BM, u0 = ut * BU;
  auto gcol = [](int g) { return NG == 4 ? g : (g == 0 ? G_I : g + 1); };

  // epilogue operands first: the position and vertex of each row, the bias
  const int j0 = u0 + wu * 16 + 4 * gq;
  int pos[TM], vid[TM];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int m = m0 + wr * (BM / 2) + tm * 16 + r;
    pos[tm] = m < n_pull ? n.pull_list[m] : -1;
    vid[tm] = pos[tm] >= 0 && pos[tm] < lo1 ? n.order[pos[tm]] : 0;
  }
  Bias4 bias;
  lstm_bias4(n, j0, bias);

  const float* src[IPW];
  int kq[IPW];
#pragma unroll
  for (int t = 0; t < IPW; ++t) {
    const int row = (w * IPW + t) * 8 + (lane >> 3), qg = (lane & 7) ^ (row & 7);
    kq[t] = 4 * qg;
    if (row < BM) {
      const int p = n.pull_list[min(m0 + row, n_pull - 1)];
      src[t] = n.X + (size_t)n.pull_pos[p] * D + 4 * qg;
    } else {
      const int b = row - BM, g = b / BU, u = b % BU;
      src[t] = n.WxT + (size_t)(gcol(g) * H + u0 + u) * D + 4 * qg;
    }
  }
  const int wofs = __builtin_amdgcn_readfirstlane(w * IPW * 256);
  v4f acc[TM][NG];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int g = 0; g < NG; ++g) acc[tm][g] = v4f{0.f, 0.f, 0.f, 0.f};

  auto issue = [&](auto sc, int c) {
    const uint32_t base = __builtin_amdgcn_readfirstlane(lds_addr_of(ring.at(sc)) + 4u * wofs);
    const int k0 = c * kBK;
#pragma unroll
    for (int t = 0; t < IPW; ++t)
      copy16_to_lds(k0 + kq[t] < D ? src[t] + k0 : n.zrow, base + 1024u * t);
  };
  struct Frag {
    float a[TM][8], b[NG][8];
  };
  auto read = [&](const float* Ls, Frag& f) {
#pragma unroll
    for (int g = 0; g < NG; ++g) frag_sw(Ls, BM + g * BU + wu * 16 + r, gq, f.b[g]);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) frag_sw(Ls, wr * (BM / 2) + tm * 16 + r, gq, f.a[tm]);
  };
  auto body = [&](const float* Lnext, Frag& cur, Frag& nxt, int) {
    read(Lnext, nxt);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int g = 0; g < NG; ++g) acc[tm][g] = mfma_chunk8<false>(cur.b[g], cur.a[tm], acc[tm][g]);
    interleave_reads<2 * (NG + TM), TM * NG * 8>();
  };
  ring_loop_db<S, IPW, Frag>((D + kBK - 1) / kBK, ring, issue, read, body);

#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int p = pos[tm];
    if (p < 0) continue;
    if (p < lo1) {
      const v4f zi = acc[tm][0], zo = acc[tm][NG == 4 ? 2 : 1], zu = acc[tm][NG == 4 ? 3 : 2];
      const float bi[4] = {bias.i.x, bias.i.y, bias.i.z, bias.i.w};
      const float bo[4] = {bias.o.x, bias.o.y, bias.o.z, bias.o.w};
      const float bu[4] = {bias.u.x, bias.u.y, bias.u.z, bias.u.w};
      float ig[4], og[4], ug[4], c[4], h[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ig[e] = sigmoidf_(zi[e] + bi[e]);
        og[e] = sigmoidf_(zo[e] + bo[e]);
        ug[e] = tanh_(zu[e] + bu[e]);
        c[e] = ig[e] * ug[e];
        h[e] = og[e] * tanh_(c[e]);
      }
      auto f4 = [](const float (&x)[4]) { return make_float4(x[0], x[1], x[2], x[3]); };
      st4(n.Hs + (size_t)p * H + j0, f4(h));
      st4(n.Cs + (size_t)p * H + j0, f4(c));
      if (n.Gs) {   // a leaf's forget gates are never read; null in inference
        float* gs = n.Gs + (size_t)p * n.GW + j0;
        st4(gs, f4(ig));
        st4(gs + 2 * H, f4(og));
        st4(gs + 3 * H, f4(ug));
      }
      st4(n.h_out + (size_t)vid[tm] * H + j0, f4(h));
      if (n.c_out) st4(n.c_out + (size_t)vid[tm] * H + j0, f4(c));
    } else {
#pragma unroll
      for (int g = 0; g < NG; ++g)
        st4(n.P + (size_t)p * H4 + gcol(g) * H + j0,
            make_float4(acc[tm][g][0], acc[tm][g][1], acc[tm][g][2], acc[tm][g][3]));
    }
  }
}

// --------------------------------------------------------------- dX GEMM
// dX[pull_pos[p], d] = sum_k dA_x[p, k] W_x[d, k], k over the gate columns
// (i,f,o,u or i,o,u); the f column of dA_x is delta_f0 + delta_f1.
__global__ void __launch_bounds__(256) k_dx_gemm(Net n, int n_pull, int with_f, float* dX) {
  constexpr int BM = 64, BN = 64, LDA = kBK + 4, LDB = kBK + 4;
  __shared__ __attribute__((aligned(16))) float As[BM * LDA];
  __shared__ __attribute__((aligned(16))) float Bs[BN * LDB];
  const int H = n.H, H4 = 4 * H, D = n.D, GW = n.GW, N = n.N;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wrow = (w >> 1) * 32, wcol = (w & 1) * 32;
  const int m0 = blockIdx.x * BM, d0 = blockIdx.y * BN;
  const float* asrc[2];
  int arow[2], aq[2];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int idx = tid + 256 * a;
    arow[a] = idx / 8;
    aq[a] = idx % 8;
    asrc[a] = m0 + arow[a] < n_pull ? n.dA + (size_t)n.pull_list[m0 + arow[a]] * GW : nullptr;
  }
  float4 ra[2], rb[2];
  auto col_of = [&](int kc) {
    const int c = kc * kBK;
    if (with_f) return c;
    return c < H ? c : c + H;
  };
  auto gload = [&](int kc) {
    const int c0 = col_of(kc);
    const bool fblock = c0 >= H && c0 < 2 * H;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      float4 v = f4zero();
      if (asrc[a]) {
        v = ldg4(asrc[a] + c0 + 4 * aq[a]);
        if (fblock && N == 2) v = add4(v, ldg4(asrc[a] + 3 * H + c0 + 4 * aq[a]));
      }
      ra[a] = v;
    }
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int idx = tid + 256 * b, dr = idx / 8, q = idx % 8;
      rb[b] = d0 + dr < D ? ldg4(n.Wx + (size_t)(d0 + dr) * H4 + c0 + 4 * q) : f4zero();
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int a = 0; a < 2; ++a) st4(&As[arow[a] * LDA + 4 * aq[a]], ra[a]);
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int idx = tid + 256 * b, dr = idx / 8, q = idx % 8;
      st4(&Bs[dr * LDB + 4 * q], rb[b]);
    }
  };
  v4f acc[2][2];
  zero_acc(acc);
  const int nk = (with_f ? H4 : 3 * H) / kBK;
  gload(0);
  for (int kc = 0; kc < nk; ++kc) {
    __syncthreads();
    sstore();
    __syncthreads();
    if (kc + 1 < nk) gload(kc + 1);
    mfma_chunk<2, 2, true, true, LDA, LDB>(As, Bs, wrow, wcol, acc);
  }
#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + wrow + tm * 16 + 4 * gq + i;
      if (m >= n_pull) continue;
      const int row = n.pull_pos[n.pull_list[m]];
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) {
        const int d = d0 + wcol + tn * 16 + r;
        if (d < D) dX[(size_t)row * D + d] = acc[tm][tn][i];
      }
    }
}

// ------------------------------------------------ long-K "A^T B" products
// out[s][m][n] = sum_{q in split s} A(q, m) B(q, n).  The loader supplies
// 4 consecutive m (or n) of row q; rows outside [0, Q) are never requested.
struct LdDUiou {  // dU[:, i|o|u] (or all four blocks when N == 1): A = h~, B = dA
  static constexpr const char* kName = "k_tn_gemm<LdDUiou, 64, 4>";
  static constexpr const char* kName128 = "k_tn_gemm<LdDUiou, 128, 8>";
  static constexpr const char* kNameBf = "k_tn_gemm_bf<LdDUiou>";
  static constexpr const char* kNamePack = "k_pack_bf<LdDUiou>";
  static constexpr const char* kNameNt = "k_nt_bf<LdDUiou>";
  static constexpr const char* kNameDl128 = "k_tn_dl<LdDUiou, 128, 256, 2>";
  static constexpr const char* kNameDl64 = "k_tn_dl<LdDUiou, 64, 256, 3>";
  static constexpr const char* kNameDl128n = "k_tn_dl<LdDUiou, 128, 128, 3>";
  struct Idx {
    int c0, c1;
  };
  Net n;
  int off1;
  __device__ Idx idx(int q) const {
    const int p = off1 + q;
    return {n.child_pos[(size_t)p * n.N], n.N == 2 ? n.child_pos[(size_t)p * n.N + 1] : -1};
  }
  __device__ float4 a4(const Idx& x, int q, int m) const {
    float4 s = x.c0 >= 0 ? ldg4(n.Hs + (size_t)x.c0 * n.H + m) : f4zero();
    if (x.c1 >= 0) s = add4(s, ldg4(n.Hs + (size_t)x.c1 * n.H + m));
    return s;
  }
  __device__ float4 b4(const Idx&, int q, int c) const {
    const int p = off1 + q;
    const int col = (n.N == 2 && c >= n.H) ? c + n.H : c;
    return ldg4(n.dA + (size_t)p * n.GW + col);
  }
  // row offsets for the direct-to-LDS product: A = h_0 + h_1 (two rows),
  // B = the dA row; B column n0 of the product is dA column bcol(n0)
  static constexpr int NA = 2;
  bool direct() const { return true; }
  __device__ void offs(int q, int& a0, int& a1, int& b) const {
    const int p = off1 + q;
    const int c0 = n.child_pos[(size_t)p * n.N], c1 = n.child_pos[(size_t)p * n.N + n.N - 1];
    a0 = c0 >= 0 ? c0 * n.H : -1;
    a1 = (n.N == 2 && c1 >= 0) ? c1 * n.H : -1;
    b = p * n.GW;
  }
  __device__ int bcol(int n0) const { return (n.N == 2 && n0 >= n.H) ? n0 + n.H : n0; }
  __device__ const float* abase() const { return n.Hs; }
  __device__ const float* bbase() const { return n.dA; }
};

struct LdDUf {  // dU[:, f] with two children: q in [0, 2 MI), A = h_k, B = dA_fk
  static constexpr const char* kName = "k_tn_gemm<LdDUf, 64, 4>";
  static constexpr const char* kName128 = "k_tn_gemm<LdDUf, 128, 8>";
  static constexpr const char* kNameBf = "k_tn_gemm_bf<LdDUf>";
  static constexpr const char* kNamePack = "k_pack_bf<LdDUf>";
  static constexpr const char* kNameNt = "k_nt_bf<LdDUf>";
  static constexpr const char* kNameDl128 = "k_tn_dl<LdDUf, 128, 256, 3>";
  static constexpr const char* kNameDl64 = "k_tn_dl<LdDUf, 64, 256, 3>";
  static constexpr const char* kNameDl128n = "k_tn_dl<LdDUf, 128, 128, 4>";
  struct Idx {
    int cp;
  };
  Net n;
  int off1, MI;
  __device__ Idx idx(int q) const {
    const int k = q >= MI, p = off1 + q - k * MI;
    return {n.child_pos[(size_t)p * 2 + k]};
  }
  __device__ float4 a4(const Idx& x, int q, int m) const {
    return x.cp >= 0 ? ldg4(n.Hs + (size_t)x.cp * n.H + m) : f4zero();
  }
  __device__ float4 b4(const Idx&, int q, int c) const {
    const int k = q >= MI, p = off1 + q - k * MI;
    return ldg4(n.dA + (size_t)p * n.GW + (k ? 4 * n.H : n.H) + c);
  }
  static constexpr int NA = 1;
  bool direct() const { return true; }
  __device__ void offs(int q, int& a0, int& a1, int& b) const {
    const int k = q >= MI, p = off1 + q - k * MI;
    const int cp = n.child_pos[(size_t)p * 2 + k];
    a0 = cp >= 0 ? cp * n.H : -1;
    a1 = -1;
    b = p * n.GW + (k ? 4 * n.H : n.H);
  }
  __device__ int bcol(int n0) const { return n0; }
  __device__ const float* abase() const { return n.Hs; }
  __device__ const float* bbase() const { return n.dA; }
};

struct LdDWx {  // dW_x: q over pulling vertices, A = x, B = dA_x (f = f_0 + f_1)
  static constexpr const char* kName = "k_tn_gemm<LdDWx, 64, 4>";
  static constexpr const char* kName128 = "k_tn_gemm<LdDWx, 128, 8>";
  static constexpr const char* kNameBf = "k_tn_gemm_bf<LdDWx>";
  static constexpr const char* kNamePack = "k_pack_bf<LdDWx>";
  static constexpr const char* kNameNt = "k_nt_bf<LdDWx>";
  static constexpr const char* kNameDl128 = "k_tn_dl<LdDWx, 128, 256, 3>";
  static constexpr const char* kNameDl64 = "k_tn_dl<LdDWx, 64, 256, 3>";
  static constexpr const char* kNameDl128n = "k_tn_dl<LdDWx, 128, 128, 4>";
  struct Idx {
    int p, row;
  };
  Net n;
  int with_f;
  __device__ Idx idx(int q) const {
    const int p = n.pull_list[q];
    return {p, n.pull_pos[p]};
  }
  __device__ float4 a4(const Idx& x, int q, int m) const {
    return m < n.D ? ldg4(n.X + (size_t)x.row * n.D + m) : f4zero();
  }
  __device__ float4 b4(const Idx& x, int q, int c) const {
    const int H = n.H;
    const int col = (with_f || c < H) ? c : c + H;
    const float* row = n.dA + (size_t)x.p * n.GW;
    float4 v = ldg4(row + col);
    if (n.N == 2 && col >= H && col < 2 * H) v = add4(v, ldg4(row + 3 * H + col));
    return v;
  }
  // direct-to-LDS only when every B column is a single dA column (the f
  // block with two children sums f_0 and f_1)
  static constexpr int NA = 1;
  bool direct() const { return !(with_f && n.N == 2); }
  __device__ void offs(int q, int& a0, int& a1, int& b) const {
    const int p = n.pull_list[q];
    a0 = n.pull_pos[p] * n.D;
    a1 = -1;
    b = p * n.GW;
  }
  __device__ int bcol(int n0) const { return (with_f || n0 < n.H) ? n0 : n0 + n.H; }
  __device__ const float* abase() const { return n.X; }
  __device__ const float* bbase() const { return n.dA; }
};

struct LdFCdW {  // Tree-FC dW_k: A = h_k, B = delta, q over internal vertices
  static constexpr const char* kName = "k_tn_gemm<LdFCdW, 64, 4>";
  static constexpr const char* kName128 = "k_tn_gemm<LdFCdW, 128, 8>";
  static constexpr const char* kNameBf = "k_tn_gemm_bf<LdFCdW>";
  static constexpr const char* kNamePack = "k_pack_bf<LdFCdW>";
  static constexpr const char* kNameNt = "k_nt_bf<LdFCdW>";
  static constexpr const char* kNameDl128 = "k_tn_dl<LdFCdW, 128, 256, 3>";
  static constexpr const char* kNameDl64 = "k_tn_dl<LdFCdW, 64, 256, 3>";
  static constexpr const char* kNameDl128n = "k_tn_dl<LdFCdW, 128, 128, 4>";
  struct Idx {
    int cp;
  };
  Net n;
  int off1, slot;
  __device__ Idx idx(int q) const {
    return {n.child_pos[(size_t)(off1 + q) * n.N + slot]};
  }
  __device__ float4 a4(const Idx& x, int q, int m) const {
    return x.cp >= 0 ? ldg4(n.Hs + (size_t)x.cp * n.H + m) : f4zero();
  }
  __device__ float4 b4(const Idx&, int q, int c) const {
    return ldg4(n.dA + (size_t)(off1 + q) * n.H + c);
  }
  static constexpr int NA = 1;
  bool direct() const { return true; }
  __device__ void offs(int q, int& a0, int& a1, int& b) const {
    const int cp = n.child_pos[(size_t)(off1 + q) * n.N + slot];
    a0 = cp >= 0 ? cp * n.H : -1;
    a1 = -1;
    b = (off1 + q) * n.H;
  }
  __device__ int bcol(int n0) const { return n0; }
  __device__ const float* abase() const { return n.Hs; }
  __device__ const float* bbase() const { return n.dA; }
};

template <class L, int BT, int NW>
__global__ void __launch_bounds__(64 * NW) k_tn_gemm(L ld, int Q, int qchunk, int Mo, int No,
                                                     float* out) {
  // BT x BT output tile; NW wavefronts as 2 x NW/2 of (BT/2) x (2BT/NW); K
  // (= q) chunks of 32 in two LDS stages.  While chunk c is multiplied, the
  // data of chunk c+1 and the per-row indices (gathers) of chunk c+2 are
  // loaded, so no data load waits on an index load; chunk c+1 is then stored
  // to the other stage and one barrier per chunk separates the stages.  The
  // barrier is a bare s_barrier after the LDS writes have completed: the
  // workgroup fence of __syncthreads would also wait for the loads in flight.
  // LDS rows hold 32 q x BT columns; float4 c4 of row q sits at quad
  // c4 ^ 4((q >> 3) & 3), so the fragment reads of the four lane groups
  // (rows 8g + ...) fall in four different bank ranges.
  constexpr int NT = 64 * NW, TM = BT / 32, TN = BT / (8 * NW), C4 = BT / 4;
  constexpr int PER = kBK * C4 / NT;
  static_assert(PER * NT == kBK * C4 && TN >= 1, "tile split");
  using Idx = typename L::Idx;
  __shared__ __attribute__((aligned(16))) float As[2][kBK * BT];
  __shared__ __attribute__((aligned(16))) float Bs[2][kBK * BT];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wrow = (w / (NW / 2)) * (BT / 2), wcol = (w % (NW / 2)) * (16 * TN);
  const int n0 = blockIdx.x * BT, m0 = blockIdx.y * BT, s = blockIdx.z;
  const int q_lo = s * qchunk, q_hi = min(Q, q_lo + qchunk);
  float4 ra[PER], rb[PER];
  Idx ix_next[PER];
  auto load_idx = [&](int q0, Idx (&ix)[PER]) {
#pragma unroll
    for (int a = 0; a < PER; ++a) {
      const int q = q0 + (tid + NT * a) / C4;
      if (q < q_hi) ix[a] = ld.idx(q);
    }
  };
  auto gload = [&](int q0, const Idx (&ix)[PER]) {
#pragma unroll
    for (int a = 0; a < PER; ++a) {
      const int idx = tid + NT * a, qq = idx / C4, c4 = idx % C4;
      const int q = q0 + qq;
      ra[a] = (q < q_hi && m0 + 4 * c4 < Mo) ? ld.a4(ix[a], q, m0 + 4 * c4) : f4zero();
      rb[a] = (q < q_hi) ? ld.b4(ix[a], q, n0 + 4 * c4) : f4zero();
    }
  };
  auto sstore = [&](int st) {
#pragma unroll
    for (int a = 0; a < PER; ++a) {
      const int idx = tid + NT * a, qq = idx / C4, c4 = idx % C4;
      const int col = 4 * (c4 ^ (4 * ((qq >> 3) & 3)));
      st4(&As[st][qq * BT + col], ra[a]);
      st4(&Bs[st][qq * BT + col], rb[a]);
    }
  };
  // k = 8 gq + 4 h + e of column x (lane group gq reads rows 8 gq ..)
  auto frag = [&](const float* S, int x, int h, float (&f)[4]) {
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = S[(8 * gq + 4 * h + e) * BT + (x ^ (16 * gq))];
  };
  auto barrier = []() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): this wave's LDS writes done
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  v4f acc[TM][TN];
  zero_acc(acc);
  {
    Idx ix0[PER];
    load_idx(q_lo, ix0);
    load_idx(q_lo + kBK, ix_next);
    gload(q_lo, ix0);
  }
  sstore(0);
  barrier();
  int st = 0;
  for (int q0 = q_lo; q0 < q_hi; q0 += kBK) {
    const bool more = q0 + kBK < q_hi;
    if (more) {
      gload(q0 + kBK, ix_next);
      load_idx(q0 + 2 * kBK, ix_next);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float af[TM][4], bf[TN][4];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) frag(As[st], wrow + 16 * tm + r, h, af[tm]);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) frag(Bs[st], wcol + 16 * tn + r, h, bf[tn]);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
            acc[tm][tn] = mfma_f32_16x16x4(af[tm][e], bf[tn][e], acc[tm][tn]);
    }
    if (more) sstore(st ^ 1);
    barrier();
    st ^= 1;
  }
  float* o = out + (size_t)s * Mo * No;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + wrow + tm * 16 + 4 * gq + i;
      if (m >= Mo) continue;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) o[(size_t)m * No + n0 + wcol + tn * 16 + r] = acc[tm][tn][i];
    }
}
// dX through the LDS ring (lds_ring.h), for gate columns that need no
// f_0 + f_1 sum (i|o|u, or all four blocks with one child slot): a
// workgroup owns BM pulled rows x BN input columns; stage rows [0, BM) are
// dA rows (gathered through pull_list), [BM, BM + BN) rows of W_x.  Rows
// past n_pull or D read the last valid row; their products are not stored.
template <int BM, int BN, int S>
__global__ void __launch_bounds__(256) k_dx_tile(Net n, int n_pull, int four, float* dX) {
  constexpr int TM = BM / 32, TN = BN / 32, ROWS = BM + BN, IPW = ROWS / 32;
  static_assert(IPW * 32 == ROWS && S >= 2 && S <= 4, "tile shape");
  __shared__ __attribute__((aligned(1024))) float L0[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L1[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L2[S > 2 ? ROWS * 32 : 4];
  __shared__ __attribute__((aligned(1024))) float L3[S > 3 ? ROWS * 32 : 4];
  const Ring<ROWS, S> ring{L0, L1, L2, L3};
  const int H = n.H, H4 = 4 * H, D = n.D, GW = n.GW;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w & 1, wn = w >> 1;
  const int m0 = blockIdx.x * BM, d0 = blockIdx.y * BN;
  // output rows of this lane (one per row block), fetched before the product
  int orow[TM];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int m = m0 + wr * (BM / 2) + tm * 16 + r;
    orow[tm] = m < n_pull ? n.pull_pos[n.pull_list[m]] : -1;
  }
  const float* src[IPW];
#pragma unroll
  for (int t = 0; t < IPW; ++t) {
    const int row = (w * IPW + t) * 8 + (lane >> 3), qg = (lane & 7) ^ (row & 7);
    const float* ptr;
    if (row < BM) ptr = n.dA + (size_t)n.pull_list[min(m0 + row, n_pull - 1)] * GW;
    else ptr = n.Wx + (size_t)min(d0 + row - BM, D - 1) * H4;
    src[t] = ptr + 4 * qg;
  }
  const int wofs = __builtin_amdgcn_readfirstlane(w * IPW * 256);
  v4f acc[TM][TN];
  zero_acc(acc);
  auto issue = [&](auto sc, int c) {
    const uint32_t base = __builtin_amdgcn_readfirstlane(lds_addr_of(ring.at(sc)) + 4u * wofs);
    const int k0 = c * kBK, col = (four || k0 < H) ? k0 : k0 + H;
#pragma unroll
    for (int t = 0; t < IPW; ++t) copy16_to_lds(src[t] + col, base + 1024u * t);
  };
  struct Frag {
    float a[TM][8], b[TN][8];
  };
  auto read = [&](const float* Ls, Frag& f) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) frag_sw(Ls, BM + wn * (BN / 2) + tn * 16 + r, gq, f.b[tn]);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) frag_sw(Ls, wr * (BM / 2) + tm * 16 + r, gq, f.a[tm]);
  };
  // A = W_x fragment (d), B = dA fragment (rows): a lane holds four
  // consecutive d of one row
  auto body = [&](const float* Lnext, Frag& cur, Frag& nxt, int) {
    read(Lnext, nxt);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = mfma_chunk8<false>(cur.b[tn], cur.a[tm], acc[tm][tn]);
    interleave_reads<2 * (TM + TN), TM * TN * 8>();
  };
  ring_loop_db<S, IPW, Frag>((four ? H4 : 3 * H) / kBK, ring, issue, read, body);
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    if (orow[tm] < 0) continue;
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int d = d0 + wn * (BN / 2) + tn * 16 + 4 * gq;
      if (d < D)   // D % 4 == 0: the four d are all in range or all out
        st4(dX + (size_t)orow[tm] * D + d,
            make_float4(acc[tm][tn][0], acc[tm][tn][1], acc[tm][tn][2], acc[tm][tn][3]));
    }
  }
}

// ------------------------------------------------------------ bf16 variants
// Same tiles as the fp32 kernels above; operands are rounded to bf16 while
// they are staged into LDS (k-contiguous rows), accumulation is fp32.
__global__ void __launch_bounds__(256) k_pull_gemm_bf(Net n, int n_pull, int with_f) {
  constexpr int BM = 64, BN = 64;
  __shared__ __attribute__((aligned(16))) u16 As[BM * kLDH];
  __shared__ __attribute__((aligned(16))) u16 Bs[BN * kLDH];
  const int H = n.H, H4 = 4 * H, D = n.D;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wrow = (w >> 1) * 32, wcol = (w & 1) * 32;
  const int m0 = blockIdx.x * BM;
  const int tpg = H / BN, gsel = blockIdx.y / tpg;
  const int gate = with_f ? gsel : (gsel == 0 ? G_I : gsel + 1);
  const int n0 = gate * H + (blockIdx.y % tpg) * BN;
  const float* asrc[2];
  int arow[2], aq[2];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int idx = tid + 256 * a;
    arow[a] = idx / 8;
    aq[a] = idx % 8;
    asrc[a] = nullptr;
    if (m0 + arow[a] < n_pull) asrc[a] = n.X + (size_t)n.pull_pos[n.pull_list[m0 + arow[a]]] * D;
  }
  float4 ra[2], rb[2];
  auto gload = [&](int k0) {
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int k = k0 + 4 * aq[a];
      ra[a] = (asrc[a] && k < D) ? ldg4(asrc[a] + k) : f4zero();
    }
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int idx = tid + 256 * b, kk = idx / 16, q = idx % 16;
      rb[b] = k0 + kk < D ? ldg4(n.Wx + (size_t)(k0 + kk) * H4 + n0 + 4 * q) : f4zero();
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int a = 0; a < 2; ++a) st_bf4(&As[arow[a] * kLDH + 4 * aq[a]], ra[a]);
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int idx = tid + 256 * b, kk = idx / 16, q = idx % 16;
      st_bf4_t(&Bs[(4 * q) * kLDH + kk], kLDH, rb[b]);
    }
  };
  v4f acc[2][2];
  zero_acc(acc);
  const int nk = (D + kBK - 1) / kBK;
  gload(0);
  for (int kc = 0; kc < nk; ++kc) {
    __syncthreads();
    sstore();
    __syncthreads();
    if (kc + 1 < nk) gload((kc + 1) * kBK);
    mfma_chunk_bf<2, 2>(As, Bs, wrow, wcol, acc);
  }
#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + wrow + tm * 16 + 4 * gq + i;
      if (m >= n_pull) continue;
      const int p = n.pull_list[m];
#pragma unroll
      for (int tn = 0; tn < 2; ++tn)
        n.P[(size_t)p * H4 + n0 + wcol + tn * 16 + r] = acc[tm][tn][i];
    }
}

__global__ void __launch_bounds__(256) k_dx_gemm_bf(Net n, int n_pull, int with_f, float* dX) {
  constexpr int BM = 64, BN = 64;
  __shared__ __attribute__((aligned(16))) u16 As[BM * kLDH];
  __shared__ __attribute__((aligned(16))) u16 Bs[BN * kLDH];
  const int H = n.H, H4 = 4 * H, D = n.D, GW = n.GW, N = n.N;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wrow = (w >> 1) * 32, wcol = (w & 1) * 32;
  const int m0 = blockIdx.x * BM, d0 = blockIdx.y * BN;
  const float* asrc[2];
  int arow[2], aq[2];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int idx = tid + 256 * a;
    arow[a] = idx / 8;
    aq[a] = idx % 8;
    asrc[a] = m0 + arow[a] < n_pull ? n.dA + (size_t)n.pull_list[m0 + arow[a]] * GW : nullptr;
  }
  float4 ra[2], rb[2];
  auto col_of = [&](int kc) {
    const int c = kc * kBK;
    if (with_f) return c;
    return c < H ? c : c + H;
  };
  auto gload = [&](int kc) {
    const int c0 = col_of(kc);
    const bool fblock = c0 >= H && c0 < 2 * H;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      float4 v = f4zero();
      if (asrc[a]) {
        v = ldg4(asrc[a] + c0 + 4 * aq[a]);
        if (fblock && N == 2) v = add4(v, ldg4(asrc[a] + 3 * H + c0 + 4 * aq[a]));
      }
      ra[a] = v;
    }
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int idx = tid + 256 * b, dr = idx / 8, q = idx % 8;
      rb[b] = d0 + dr < D ? ldg4(n.Wx + (size_t)(d0 + dr) * H4 + c0 + 4 * q) : f4zero();
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int a = 0; a < 2; ++a) st_bf4(&As[arow[a] * kLDH + 4 * aq[a]], ra[a]);
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int idx = tid + 256 * b;
      st_bf4(&Bs[(idx / 8) * kLDH + 4 * (idx % 8)], rb[b]);
    }
  };
  v4f acc[2][2];
  zero_acc(acc);
  const int nk = (with_f ? H4 : 3 * H) / kBK;
  gload(0);
  for (int kc = 0; kc < nk; ++kc) {
    __syncthreads();
    sstore();
    __syncthreads();
    if (kc + 1 < nk) gload(kc + 1);
    mfma_chunk_bf<2, 2>(As, Bs, wrow, wcol, acc);
  }
#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + wrow + tm * 16 + 4 * gq + i;
      if (m >= n_pull) continue;
      const int row = n.pull_pos[n.pull_list[m]];
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) {
        const int d = d0 + wcol + tn * 16 + r;
        if (d < D) dX[(size_t)row * D + d] = acc[tm][tn][i];
      }
    }
}

template <class L>
__global__ void __launch_bounds__(256) k_tn_gemm_bf(L ld, int Q, int qchunk, int Mo, int No,
                                                    float* out) {
  constexpr int BM = 64, BN = 64;
  __shared__ __attribute__((aligned(16))) u16 As[BM * kLDH];
  __shared__ __attribute__((aligned(16))) u16 Bs[BN * kLDH];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wrow = (w >> 1) * 32, wcol = (w & 1) * 32;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM, s = blockIdx.z;
  const int q_lo = s * qchunk, q_hi = min(Q, q_lo + qchunk);
  float4 ra[2], rb[2];
  auto gload = [&](int q0) {
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int idx = tid + 256 * a, qq = idx / 16, c4 = idx % 16;
      const int q = q0 + qq;
      if (q < q_hi) {
        const typename L::Idx ix = ld.idx(q);
        ra[a] = m0 + 4 * c4 < Mo ? ld.a4(ix, q, m0 + 4 * c4) : f4zero();
        rb[a] = ld.b4(ix, q, n0 + 4 * c4);
      } else {
        ra[a] = f4zero();
        rb[a] = f4zero();
      }
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int idx = tid + 256 * a, qq = idx / 16, c4 = idx % 16;
      st_bf4_t(&As[(4 * c4) * kLDH + qq], kLDH, ra[a]);
      st_bf4_t(&Bs[(4 * c4) * kLDH + qq], kLDH, rb[a]);
    }
  };
  v4f acc[2][2];
  zero_acc(acc);
  gload(q_lo);
  for (int q0 = q_lo; q0 < q_hi; q0 += kBK) {
    __syncthreads();
    sstore();
    __syncthreads();
    if (q0 + kBK < q_hi) gload(q0 + kBK);
    mfma_chunk_bf<2, 2>(As, Bs, wrow, wcol, acc);
  }
  float* o = out + (size_t)s * Mo * No;
#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + wrow + tm * 16 + 4 * gq + i;
      if (m >= Mo) continue;
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) o[(size_t)m * No + n0 + wcol + tn * 16 + r] = acc[tm][tn][i];
    }
}

// dst[m, col(n)] = sum_s part[s][m][n] in split order; col(n) = col_off + n
// (+ gap for n >= gap_start).
__global__ void k_reduce_splits(const float* __restrict__ part, int S, int Mo, int No,
                                float* __restrict__ dst, int ldd, int col_off, int gap_start,
                                int gap) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)Mo * No) return;
  const int m = (int)(idx / No), nn = (int)(idx % No);
  float s = 0.f;
  for (int k = 0; k < S; ++k) s += part[(size_t)k * Mo * No + idx];
  dst[(size_t)m * ldd + col_off + nn + (nn >= gap_start ? gap : 0)] = s;
}

// Lazy products through direct-to-LDS copies: out[m][n] = sum over q of
// A[q][m] B[q][n] for q in one split [q_lo, q_hi), with A row q = the sum of
// the loader's NA source rows (or zero where a row is absent) and B row q a
// source row starting at the loader's offset plus bcol(n0).  Eight
// wavefronts own a BM x BN output tile (BM = 128: 2 x 4 wavefronts of
// 64 x BN/4; BM = 64: 1 x 8 of 64 x BN/8) as 4 x TN MFMA blocks whose rows
// and columns are interleaved (block b row i is tile row 4i + b, block c
// column j is column TN j + c), so one 16-byte LDS read gives a lane its A
// values of all four row blocks.  Stage rows are k (one vertex each) with
// the tile's columns contiguous, filled by global_load_lds_dwordx4 through
// an S-stage ring; the source offsets of a segment of rows are computed
// into LDS first, so issuing a chunk's copies waits on nothing but LDS.
constexpr int kTnSeg = 1024;

// LDS of one tile shape: S stages of 32 k x ROWS floats, then the segment's
// row offsets (NA A rows and one B row per k).
template <class L, int BM, int BN, int S>
struct TnShape {
  static constexpr int ROWS = L::NA * BM + BN;
  static constexpr int FLOATS = S * ROWS * 32;
  static constexpr int INTS = (L::NA + 1) * kTnSeg;
};

// Output tile (bx, by) of split s; lds holds TnShape::FLOATS floats
// (1 KB-aligned), offs TnShape::INTS ints.
template <class L, int BM, int BN, int S>
__device__ __forceinline__ void tn_dl_tile(const L& ld, int Q, int qchunk, int Mo, int No,
                                           float* out, int bx, int by, int s, float* lds,
                                           int* offs) {
  constexpr int NA = L::NA, WM = BM / 64, WN = 8 / WM, WTN = BN / WN, TN = WTN / 16;
  constexpr int ROWS = NA * BM + BN;                 // a stage is 32 k x ROWS floats
  constexpr int IA = BM * 32 / 256 / 8, IB = BN * 32 / 256 / 8;
  constexpr int IPW = NA * IA + IB;                  // copies per wavefront per chunk
  constexpr int APC = 256 / BM, BPC = 256 / BN;      // operand rows per copy
  static_assert((TN == 2 || TN == 4) && IA >= 1 && IB >= 1 && S >= 2 && S <= 4, "tile shape");
  const Ring<ROWS, S> ring{lds, lds + ROWS * 32, lds + (S > 2 ? 2 : 0) * ROWS * 32,
                           lds + (S > 3 ? 3 : 0) * ROWS * 32};
  int* oa0 = offs;
  int* oa1 = offs + kTnSeg;
  int* ob = offs + NA * kTnSeg;

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, g = lane >> 4, r = lane & 15;
  const int wr = w / WN, wc = w % WN, ws = __builtin_amdgcn_readfirstlane(w);
  const int n0 = bx * BN, m0 = by * BM;
  const int q_lo = s * qchunk, q_hi = min(Q, q_lo + qchunk);
  const float* A = ld.abase();
  const float* B = ld.bbase() + ld.bcol(n0);
  const float* zero = ld.n.zrow;
  const int arow = lane / (BM / 4), acol = 4 * (lane % (BM / 4));
  const int brow = lane / (BN / 4), bcolw = 4 * (lane % (BN / 4));
  const bool acol_ok = m0 + acol < Mo;

  v4f acc[4][TN];
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int c = 0; c < TN; ++c) acc[b][c] = v4f{0.f, 0.f, 0.f, 0.f};

  for (int seg = q_lo; seg < q_hi; seg += kTnSeg) {
    const int nq = min(kTnSeg, q_hi - seg);
    __syncthreads();   // the previous segment's stages and offsets are consumed
    for (int i = tid; i < nq; i += 512) {
      int a0, a1, b;
      ld.offs(seg + i, a0, a1, b);
      oa0[i] = a0;
      if constexpr (NA == 2) oa1[i] = a1;
      ob[i] = b;
    }
    __syncthreads();
    auto issue = [&](auto sc, int c) {
      const uint32_t base = __builtin_amdgcn_readfirstlane(lds_addr_of(ring.at(sc)));
      const int q0 = 32 * c;
      // every offset first, then the copies (a copy's asm statement orders
      // memory, so interleaving would wait on each LDS read); rows past the
      // segment read the zero row (A) or the segment's last row (B)
      int o0[IA], o1[IA], ov[IB];
#pragma unroll
      for (int t = 0; t < IA; ++t) {
        const int qi = q0 + APC * (ws * IA + t) + arow;
        const bool ok = qi < nq && acol_ok;
        const int qc = min(qi, nq - 1);
        o0[t] = ok ? oa0[qc] : -1;
        if constexpr (NA == 2) o1[t] = ok ? oa1[qc] : -1;
      }
#pragma unroll
      for (int t = 0; t < IB; ++t) ov[t] = ob[min(q0 + BPC * (ws * IB + t) + brow, nq - 1)];
#pragma unroll
      for (int t = 0; t < IA; ++t) {
        const uint32_t j = ws * IA + t;
        copy16_to_lds(o0[t] >= 0 ? A + o0[t] + m0 + acol : zero, base + 1024u * j);
        if constexpr (NA == 2)
          copy16_to_lds(o1[t] >= 0 ? A + o1[t] + m0 + acol : zero, base + 128u * BM + 1024u * j);
      }
#pragma unroll
      for (int t = 0; t < IB; ++t)
        copy16_to_lds(B + ov[t] + bcolw, base + 128u * NA * BM + 1024u * (ws * IB + t));
    };
    // the LDS reads of k step t+1 are issued before the MFMAs of step t (two
    // register sets), so each wait finds them landed
    struct KStep {
      float4 a, a1;
      float bv[TN];
    };
    auto compute = [&](const float* Ls, int) {
      const float* A0 = Ls + wr * 64 + 4 * r;
      const float* A1 = A0 + 32 * BM;
      const float* Bp = Ls + NA * 32 * BM + wc * WTN + TN * r;
      auto rd = [&](int t, KStep& f) {
        const int k = 4 * t + g;
        f.a = *reinterpret_cast<const float4*>(A0 + k * BM);
        if constexpr (NA == 2) f.a1 = *reinterpret_cast<const float4*>(A1 + k * BM);
        if constexpr (TN == 4) {
          const float4 b4 = *reinterpret_cast<const float4*>(Bp + k * BN);
          f.bv[0] = b4.x; f.bv[1] = b4.y; f.bv[2] = b4.z; f.bv[3] = b4.w;
        } else {
          const float2 b2 = *reinterpret_cast<const float2*>(Bp + k * BN);
          f.bv[0] = b2.x; f.bv[TN - 1] = b2.y;
        }
      };
      auto mm = [&](const KStep& f) {
        float4 a = f.a;
        if constexpr (NA == 2) {
          a.x += f.a1.x; a.y += f.a1.y; a.z += f.a1.z; a.w += f.a1.w;
        }
        const float av[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
          for (int c = 0; c < TN; ++c) acc[b][c] = mfma_f32_16x16x4(av[b], f.bv[c], acc[b][c]);
      };
      KStep f0, f1;
      rd(0, f0);
#pragma unroll
      for (int t = 0; t < 8; t += 2) {
        rd(t + 1, f1);
        mm(f0);
        if (t + 2 < 8) rd(t + 2, f0);
        mm(f1);
      }
      // keep that order: per step the next step's reads, the h~ adds, the MFMAs
      constexpr int NR = NA + 1, NM = 4 * TN;
      __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        if (t + 1 < 8) __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);
        if constexpr (NA == 2) __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
      }
    };
    ring_loop<S, IPW>((nq + 31) / 32, ring, issue, compute);
  }

  float* o = out + (size_t)s * Mo * No;
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = m0 + wr * 64 + 16 * g + 4 * e + b;
      if (m >= Mo) continue;
      float* dst = o + (size_t)m * No + n0 + wc * WTN + TN * r;
      if constexpr (TN == 4)
        st4(dst, make_float4(acc[b][0][e], acc[b][1][e], acc[b][2][e], acc[b][3][e]));
      else
        *reinterpret_cast<float2*>(dst) = make_float2(acc[b][0][e], acc[b][TN - 1][e]);
    }
}

template <class L, int BM, int BN, int S>
__global__ void __launch_bounds__(512) k_tn_dl(L ld, int Q, int qchunk, int Mo, int No,
                                               float* out) {
  using T = TnShape<L, BM, BN, S>;
  __shared__ __attribute__((aligned(1024))) float lds[T::FLOATS];
  __shared__ int offs[T::INTS];
  tn_dl_tile<L, BM, BN, S>(ld, Q, qchunk, Mo, No, out, blockIdx.x, blockIdx.y, blockIdx.z, lds,
                           offs);
}

// Up to three lazy products in one launch (the lazy batching of Section
// 3.5 taken one step further: the parameter-gradient products of a pass are
// independent, so they share one grid).  Workgroups [0, j[0].wg_end) run
// product A, then B, then C; inside a product, workgroup i is output tile
// (i % tx, i / tx % ty) of split i / (tx ty).  The split counts are chosen
// on the host so that every workgroup carries about the same MFMA work.
struct TnJob {
  int Q, qchunk, Mo, No, tx, ty, wg_end;
  float* out;
};

template <class LA, class LB, class LC>
struct TnGroupArgs {
  LA a;
  LB b;
  LC c;
  TnJob j[3];
};

constexpr int cmax3(int a, int b, int c) { return a > b ? (a > c ? a : c) : (b > c ? b : c); }

template <class LA, int BMA, int BNA, int SA, class LB, int BMB, int BNB, int SB, class LC,
          int BMC, int BNC, int SC>
__global__ void __launch_bounds__(512) k_tn_group(TnGroupArgs<LA, LB, LC> g) {
  using TA = TnShape<LA, BMA, BNA, SA>;
  using TB = TnShape<LB, BMB, BNB, SB>;
  using TC = TnShape<LC, BMC, BNC, SC>;
  __shared__ __attribute__((aligned(1024))) float lds[cmax3(TA::FLOATS, TB::FLOATS, TC::FLOATS)];
  __shared__ int offs[cmax3(TA::INTS, TB::INTS, TC::INTS)];
  const int b = blockIdx.x;
  if (b < g.j[0].wg_end) {
    const TnJob& J = g.j[0];
    tn_dl_tile<LA, BMA, BNA, SA>(g.a, J.Q, J.qchunk, J.Mo, J.No, J.out, b % J.tx, b / J.tx % J.ty,
                                 b / (J.tx * J.ty), lds, offs);
  } else if (b < g.j[1].wg_end) {
    const TnJob& J = g.j[1];
    const int i = b - g.j[0].wg_end;
    tn_dl_tile<LB, BMB, BNB, SB>(g.b, J.Q, J.qchunk, J.Mo, J.No, J.out, i % J.tx, i / J.tx % J.ty,
                                 i / (J.tx * J.ty), lds, offs);
  } else {
    const TnJob& J = g.j[2];
    const int i = b - g.j[1].wg_end;
    tn_dl_tile<LC, BMC, BNC, SC>(g.c, J.Q, J.qchunk, J.Mo, J.No, J.out, i % J.tx, i / J.tx % J.ty,
                                 i / (J.tx * J.ty), lds, offs);
  }
}

// All pending split-K sums in one launch: blockIdx.y picks the job.  Kind 0:
// each thread adds four adjacent outputs with float4 access (every such
// job's No, ldd, col_off, gap_start and gap are multiples of 4, checked on
// the host).  Kind 1 (column sums with many partial rows): see below.
__global__ void __launch_bounds__(1024) k_reduce_jobs(SplitJobs jobs) {
  const SplitJob& J = jobs.j[blockIdx.y];
  if (J.kind == 1) {
    // 64 columns per block; wavefront y adds partial rows y, y + 16, ...,
    // then the 16 sums are added in order
    __shared__ float red[16][64];
    const int x = threadIdx.x & 63, y = threadIdx.x >> 6;
    const int col = blockIdx.x * 64 + x;
    if (blockIdx.x * 64 >= J.No) return;   // the whole block
    float t = 0.f;
    if (col < J.No)
      for (int k = y; k < J.S; k += 16) t += J.part[(size_t)k * J.No + col];
    red[y][x] = t;
    __syncthreads();
    if (y != 0 || col >= J.No) return;
    float u = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) u += red[k][x];
    J.dst[col] = u;
    return;
  }
  const long idx = 4 * ((long)blockIdx.x * 1024 + threadIdx.x);
  const long total = (long)J.Mo * J.No;
  if (idx >= total) return;
  const size_t stride = (size_t)total;
  const int m = (int)(idx / J.No), nn = (int)(idx % J.No);
  float4 s = f4zero();
#pragma unroll 4
  for (int k = 0; k < J.S; ++k) {
    const float4 v = ldg4(J.part + k * stride + idx);
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  float* d = J.dst + (size_t)m * J.ldd + J.col_off + nn + (nn >= J.gap_start ? J.gap : 0);
  if (J.acc) {
    const float4 o = ldg4(d);
    s = make_float4(o.x + s.x, o.y + s.y, o.z + s.z, o.w + s.w);
  }
  st4(d, s);
}

// The reduction of a split-K product: queued on `jobs` when given (the
// caller then launches reduce_split_jobs), else launched at once.
void split_sum(const float* part, int S, int Mo, int No, float* dst, int ldd, int col_off,
               int gap_start, int gap, hipStream_t st, SplitJobs* jobs) {
  const bool by4 = No % 4 == 0 && ldd % 4 == 0 && col_off % 4 == 0 && gap % 4 == 0 &&
                   (gap_start % 4 == 0 || gap_start >= No) && (uintptr_t)dst % 16 == 0;
  if (jobs && jobs->n < SplitJobs::kMax && by4) {
    jobs->j[jobs->n++] = SplitJob{part, dst, S, Mo, No, ldd, col_off, gap_start, gap};
    return;
  }
  CAVS_LAUNCH("k_reduce_splits", k_reduce_splits, dim3(cdiv((long)Mo * No, 256)), dim3(256), 0, st,
              part, S, Mo, No, dst, ldd, col_off, gap_start, gap);
}

// ------------------------------------------- bf16 lazy products, packed
// With bf16 matrix-product operands a lazy product first packs both
// operands, rounded to bf16 (nearest-even) where the fp32 path would feed
// them to the matrix core, into rows that are contiguous in the contraction
// index q: pack row c < Mp is column m = c of A (zero for m >= Mo), row
// Mp + n is column n of B; every row holds Qp values (zero for q >= Q).  The
// product is then an "A B^T" over those rows, staged straight into LDS.
constexpr int kPackQ = kPackSeg;
constexpr int kNtTile = kPackTile;

template <class L>
__global__ void __launch_bounds__(256) k_pack_bf(L ld, int Q, int Qp, int Mo, int Mp,
                                                 u16* __restrict__ pk) {
  __shared__ u16 t[64][kPackQ + 8];   // [column][q]
  const int c0 = blockIdx.x * 64, q0 = blockIdx.y * kPackQ;
  const int tid = threadIdx.x, c4 = tid & 15, qr = tid >> 4;
  const bool aside = c0 < Mp;        // 64 | Mp: a block is all A or all B columns
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ql = qr + 16 * i, q = q0 + ql;
    float4 v = f4zero();
    if (q < Q) {
      const auto x = ld.idx(q);
      if (aside) {
        const int m = c0 + 4 * c4;
        if (m < Mo) v = ld.a4(x, q, m);
      } else {
        v = ld.b4(x, q, c0 - Mp + 4 * c4);
      }
    }
    t[4 * c4 + 0][ql] = f2bf(v.x);
    t[4 * c4 + 1][ql] = f2bf(v.y);
    t[4 * c4 + 2][ql] = f2bf(v.z);
    t[4 * c4 + 3][ql] = f2bf(v.w);
  }
  __syncthreads();
  // 64 columns x 64 q: thread (row, seg) writes 16 q (32 bytes) of one row
  const int row = tid >> 2, seg = tid & 3;
  const uint4* sp = reinterpret_cast<const uint4*>(&t[row][16 * seg]);
  uint4* dp = reinterpret_cast<uint4*>(pk + (size_t)(c0 + row) * Qp + q0 + 16 * seg);
  dp[0] = sp[0];
  dp[1] = sp[1];
}

// out[s][m][n] = sum over q in split s of pack[m][q] pack[Mp + n][q] for
// m < Mo: a 128 x 128 tile, four wavefronts of 64 x 64 (4 x 4 blocks of
// v_mfma_f32_16x16x32_bf16), 64-deep chunks through an S-stage ring of
// 128-byte LDS rows (quads XOR-swizzled by row & 7).  The n fragment is the
// MFMA's A operand, so lane (r, g) holds four consecutive n of one m.
__device__ __forceinline__ bf16x8 quad_sw(const float* L, int row, int q) {
  return *reinterpret_cast<const bf16x8*>(L + row * 32 + 4 * (q ^ (row & 7)));
}

template <int S>
__global__ void __launch_bounds__(256) k_nt_bf(const u16* __restrict__ pk, int Qp, int qchunk,
                                               int Mo, int Mp, int No, float* __restrict__ out) {
  constexpr int BM = kNtTile, BN = kNtTile, ROWS = BM + BN, IPW = ROWS / 32;
  __shared__ __attribute__((aligned(1024))) float L0[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L1[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L2[S > 2 ? ROWS * 32 : 4];
  __shared__ __attribute__((aligned(1024))) float L3[S > 3 ? ROWS * 32 : 4];
  const Ring<ROWS, S> ring{L0, L1, L2, L3};
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, g = lane >> 4, r = lane & 15;
  const int wm = w & 1, wn = w >> 1;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM, s = blockIdx.z;
  const int q_lo = s * qchunk, nch = (min(Qp, q_lo + qchunk) - q_lo) / kPackQ;
  // LDS rows [0, BM): pack rows m0 + row; [BM, ROWS): pack rows Mp + n0 + row - BM
  const char* src[IPW];
#pragma unroll
  for (int t = 0; t < IPW; ++t) {
    const int row = (w * IPW + t) * 8 + (lane >> 3), qg = (lane & 7) ^ (row & 7);
    const int prow = row < BM ? m0 + row : Mp + n0 + row - BM;
    src[t] = reinterpret_cast<const char*>(pk + (size_t)prow * Qp + q_lo) + 16 * qg;
  }
  const int wofs = __builtin_amdgcn_readfirstlane(w * IPW * 256);
  v4f acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = v4f{0.f, 0.f, 0.f, 0.f};
  auto issue = [&](auto sc, int c) {
    const uint32_t base = __builtin_amdgcn_readfirstlane(lds_addr_of(ring.at(sc)) + 4u * wofs);
#pragma unroll
    for (int t = 0; t < IPW; ++t)
      copy16_to_lds(reinterpret_cast<const float*>(src[t] + 128 * c), base + 1024u * t);
  };
  struct Frag {
    bf16x8 m[4][2], n[4][2];
  };
  auto read = [&](const float* Ls, Frag& f) {
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        f.n[b][h] = quad_sw(Ls, BM + wn * 64 + b * 16 + r, 4 * h + g);
        f.m[b][h] = quad_sw(Ls, wm * 64 + b * 16 + r, 4 * h + g);
      }
  };
  auto mma = [&](const Frag& f) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = mfma_bf16_16x16x32(f.n[b][h], f.m[a][h], acc[a][b]);
  };
  auto body = [&](const float* Lnext, Frag& cur, Frag& nxt, int) {
    read(Lnext, nxt);
    mma(cur);
    interleave_reads<16, 32>();
  };
  if (nch > 0) ring_loop_db<S, IPW, Frag>(nch, ring, issue, read, body);
  float* o = out + (size_t)s * Mo * No;
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int m = m0 + wm * 64 + a * 16 + r;
    if (m >= Mo) continue;
#pragma unroll
    for (int b = 0; b < 4; ++b)
      st4(o + (size_t)m * No + n0 + wn * 64 + b * 16 + 4 * g,
          make_float4(acc[a][b][0], acc[a][b][1], acc[a][b][2], acc[a][b][3]));
  }
}

// The direct-to-LDS kernel applies: fp32, 256-column tiles that stay inside
// one gate block, row offsets that fit an int.
bool tn_direct_ok(const Net& n, bool direct, int Mo, int No) {
  const long big = (long)n.V * (n.GW > n.H ? n.GW : n.H) + (long)n.V * n.D;
  return !n.bf && direct && n.H % 256 == 0 && No % 256 == 0 && Mo % 4 == 0 && big < (1L << 31);
}

template <class L>
void tn_product(const L& ld, int Q, int Mo, int No, float* dst, int ldd, int col_off,
                int gap_start, int gap, float* part, size_t part_floats, hipStream_t st,
                SplitJobs* jobs = nullptr) {
  if (Q <= 0) {
    // empty contraction: zero output columns
    split_sum(part, 0, Mo, No, dst, ldd, col_off, gap_start, gap, st, jobs);
    return;
  }
  // the direct-to-LDS kernel, one workgroup per CU
  const Net& n = ld.n;
  if (tn_direct_ok(n, ld.direct(), Mo, No)) {
    const int pad128 = cdiv(Mo, 128) * 128 - Mo, pad64 = cdiv(Mo, 64) * 64 - Mo;
    const int BM = pad64 < pad128 ? 64 : 128;
    // 128-wide column tiles where the 256-wide ones would be few (16 or
    // less): half the K splits, so longer K ranges per workgroup and half the
    // partial sums (measured on dU_f; with more tiles the wider tile's
    // operand reuse wins)
    const int BN = BM == 128 && (No / 256) * cdiv(Mo, BM) <= 16 ? 128 : 256;
    const int tiles = (No / BN) * cdiv(Mo, BM);
    int S = 256 / tiles;
    S = S < 1 ? 1 : S;
    if (S > cdiv(Q, kBK)) S = cdiv(Q, kBK);
    while (S > 1 && (size_t)S * Mo * No > part_floats) --S;
    const int qchunk = cdiv(cdiv(Q, S), kBK) * kBK;
    S = cdiv(Q, qchunk);
    const dim3 grid(No / BN, cdiv(Mo, BM), S);
    // ring depth: the deepest ring whose stages fit in 160 KB of LDS
    constexpr int S128 = L::NA == 2 ? 2 : 3, S128n = L::NA == 2 ? 3 : 4;
    if (BN == 128)
      CAVS_LAUNCH(L::kNameDl128n, (k_tn_dl<L, 128, 128, S128n>), grid, dim3(512), 0, st, ld, Q,
                  qchunk, Mo, No, part);
    else if (BM == 64)
      CAVS_LAUNCH(L::kNameDl64, (k_tn_dl<L, 64, 256, 3>), grid, dim3(512), 0, st, ld, Q, qchunk,
                  Mo, No, part);
    else
      CAVS_LAUNCH(L::kNameDl128, (k_tn_dl<L, 128, 256, S128>), grid, dim3(512), 0, st, ld, Q,
                  qchunk, Mo, No, part);
    split_sum(part, S, Mo, No, dst, ldd, col_off, gap_start, gap, st, jobs);
    return;
  }
  // bf16: pack, then the packed product
  const int Mp = cdiv(Mo, kNtTile) * kNtTile, Qp = cdiv(Q, kPackQ) * kPackQ;
  if (n.bf && n.pack && No % kNtTile == 0 && (size_t)(Mp + No) * Qp <= n.pack_elems) {
    CAVS_LAUNCH(L::kNamePack, k_pack_bf<L>, dim3((Mp + No) / 64, Qp / kPackQ), dim3(256), 0, st, ld,
                Q, Qp, Mo, Mp, n.pack);
    const int tiles = (No / kNtTile) * (Mp / kNtTile);
    int S = 256 / tiles;
    S = S < 1 ? 1 : S;
    if (S > Qp / kPackQ) S = Qp / kPackQ;
    while (S > 1 && (size_t)S * Mo * No > part_floats) --S;
    const int qchunk = cdiv(cdiv(Qp, S), kPackQ) * kPackQ;
    S = cdiv(Qp, qchunk);
    CAVS_LAUNCH(L::kNameNt, k_nt_bf<3>, dim3(No / kNtTile, Mp / kNtTile, S), dim3(256), 0, st,
                n.pack, Qp, qchunk, Mo, Mp, No, part);
    split_sum(part, S, Mo, No, dst, ldd, col_off, gap_start, gap, st, jobs);
    return;
  }
  const int BT = (!ld.n.bf && No % 128 == 0) ? 128 : 64;
  const int tiles = (No / BT) * cdiv(Mo, BT);
  // about two workgroups per CU (256 CUs), never three on some: a CU's
  // co-resident workgroups share its matrix cores, so the busiest CU sets
  // the time
  int S = 512 / tiles;
  S = S < 1 ? 1 : S;
  S = S > kSplitCap ? kSplitCap : S;
  int maxS = cdiv(Q, 256);
  if (S > maxS) S = maxS;
  while (S > 1 && (size_t)S * Mo * No > part_floats) --S;
  int qchunk = cdiv(cdiv(Q, S), kBK) * kBK;
  S = cdiv(Q, qchunk);
  if (ld.n.bf)
    CAVS_LAUNCH(L::kNameBf, k_tn_gemm_bf<L>, dim3(No / 64, cdiv(Mo, 64), S), dim3(256), 0, st, ld,
                Q, qchunk, Mo, No, part);
  else if (BT == 128)
    CAVS_LAUNCH(L::kName128, (k_tn_gemm<L, 128, 8>), dim3(No / 128, cdiv(Mo, 128), S), dim3(512),
                0, st, ld, Q, qchunk, Mo, No, part);
  else
    CAVS_LAUNCH(L::kName, (k_tn_gemm<L, 64, 4>), dim3(No / 64, cdiv(Mo, 64), S), dim3(256), 0, st,
                ld, Q, qchunk, Mo, No, part);
  split_sum(part, S, Mo, No, dst, ldd, col_off, gap_start, gap, st, jobs);
}

// -------------------------------------------------------------- col sums
// The bias and head gradients are column sums over the level-major rows
// (lazy batching, Section 3.4): db sums dA (LSTM: 4H columns with
// f = f_0 + f_1; FC: H columns) over rows [row0, row1); dW_s[j][c] sums
// h_j dZ_c and db_s[c] sums dZ_c over all rows.  One launch writes per-chunk
// partials (each thread: 4 adjacent columns, its chunk's rows in order); the
// split-K reduction launch adds the chunks in order, so the result is
// deterministic.
constexpr int kBiasChunks = 256;

// Partial sums of chunk y: db columns at part[y * wA + c], dW_s at
// part[nchunk * wA + y * H C + j C + c], db_s at
// part[nchunk * (wA + H C) + y C + c]: three arrays whose chunk-major rows
// are each one split-K reduction job.
template <int CP4>
__global__ void __launch_bounds__(256) k_bias_part(Net n, int row0, int row1, int lo1,
                                                   int rows_per, int bxA, int wA, int nchunk,
                                                   float* __restrict__ part) {
  const int H = n.H;
  const int lo = blockIdx.y * rows_per, hi = min(n.V, lo + rows_per);
  if ((int)blockIdx.x < bxA) {
    const int c = 4 * (blockIdx.x * 256 + threadIdx.x);
    if (c >= wA) return;
    int r0 = max(lo, row0);
    const int r1 = min(hi, row1);
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (n.GW == H) {  // Tree-FC
#pragma unroll 4
      for (int p = r0; p < r1; ++p) {
        const float4 v = *reinterpret_cast<const float4*>(n.dA + (size_t)p * H + c);
        s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
      }
    } else {
      const bool fcol = c >= G_F * H && c < (G_F + 1) * H;
      if (fcol) r0 = max(r0, lo1);  // level-0 rows have no children: f is zero
      const bool two = fcol && n.N == 2;
#pragma unroll 4
      for (int p = r0; p < r1; ++p) {
        const float* row = n.dA + (size_t)p * n.GW;
        float4 v = *reinterpret_cast<const float4*>(row + c);
        if (two) {
          const float4 u = *reinterpret_cast<const float4*>(row + 3 * H + c);
          v.x += u.x; v.y += u.y; v.z += u.z; v.w += u.w;
        }
        s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
      }
    }
    *reinterpret_cast<float4*>(part + (size_t)blockIdx.y * wA + c) = s;
    return;
  }
  // head: columns wA + j*C + c (dW_s row-major), then wA + H*C + c (db_s);
  // dZ rows hold CP = 4 CP4 columns, zero past C
  const int j = 4 * ((blockIdx.x - bxA) * 256 + threadIdx.x);
  if (j >= H) return;
  const int C = n.C;
  constexpr int CP = 4 * CP4;
  float acc[4][CP], zs[CP];
#pragma unroll
  for (int c = 0; c < CP; ++c) {
    zs[c] = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e][c] = 0.f;
  }
#pragma unroll 4
  for (int p = lo; p < hi; ++p) {
    const float4 h = *reinterpret_cast<const float4*>(n.Hs + (size_t)p * H + j);
    const float4* dz = reinterpret_cast<const float4*>(n.dZ + (size_t)p * CP);
#pragma unroll
    for (int c4 = 0; c4 < CP4; ++c4) {
      const float4 z4 = dz[c4];
      const float z[4] = {z4.x, z4.y, z4.z, z4.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = 4 * c4 + e;
        acc[0][c] += h.x * z[e];
        acc[1][c] += h.y * z[e];
        acc[2][c] += h.z * z[e];
        acc[3][c] += h.w * z[e];
        zs[c] += z[e];
      }
    }
  }
  const size_t HC = (size_t)H * C;
  float* o = part + (size_t)nchunk * wA + blockIdx.y * HC + (size_t)j * C;
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int c = 0; c < CP; ++c)
      if (c < C) o[e * C + c] = acc[e][c];
  if (j == 0) {
    float* ob = part + (size_t)nchunk * (wA + HC) + (size_t)blockIdx.y * C;
#pragma unroll
    for (int c = 0; c < CP; ++c)
      if (c < C) ob[c] = zs[c];
  }
}

// ---------------------------------------------------------------- loss
// Cross-entropy head over every position (the push of Section 3.4, batched
// lazily).  A workgroup owns 16 positions; its eight wavefronts split both
// products:
//   z = h W_s + b_s       16 positions x 16 class columns on MFMA, wavefront
//                         w taking the K chunks w, w+8, ... (MC at a time,
//                         loads first); the eight partial blocks are added in
//                         order in LDS (columns >= C repeat class C-1 and are
//                         masked);
//   log-sum-exp and softmax across the 16 lanes that hold a row's classes;
//   dZ = (softmax - onehot(label)) / |Lambda| for labelled positions, zero
//   rows otherwise (row stride CP, pad columns zero);
//   dHL = dZ W_s^T, the head's share of dL/dh, on MFMA (K = CP), wavefront w
//   taking the 16-unit blocks w, w+8, ...
// Inference (dZ and dHL null) stops after the per-position loss terms.
constexpr int kLossWaves = 8;

template <int MC>
__global__ void __launch_bounds__(64 * kLossWaves) k_loss_ce(Net n) {
  constexpr int NW = kLossWaves;
  __shared__ float zp[NW][16][17];
  __shared__ float dzl[16][17];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, r = lane & 15;
  const int p0 = blockIdx.x * 16;
  const int H = n.H, C = n.C, CP = n.CP, V = n.V;
  if (blockIdx.x == 0)   // the zero row the lazy products read for absent rows
    for (int j = threadIdx.x; j < H; j += 64 * kLossWaves) n.zrow[j] = 0.f;
  const int cm = min(r, C - 1);
  const bool cval = r < C;
  // loads unconditional (rows past V read row V-1, masked below), so that
  // they issue together
  int q[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) q[i] = n.push_pos[min(p0 + 4 * g + i, V - 1)];
#pragma unroll
  for (int i = 0; i < 4; ++i) q[i] = p0 + 4 * g + i < V ? q[i] : -1;
  const float bsc = n.bs[cm];

  const float* hrow = n.Hs + (size_t)min(p0 + r, V - 1) * H + 8 * g;
  const float* wcol = n.Ws + cm;
  const int nch = H / kBK;
  v4f acc = {0.f, 0.f, 0.f, 0.f};
  for (int c0 = w; c0 < nch; c0 += NW * MC) {
    float a[MC][8], b[MC][8];
#pragma unroll
    for (int t = 0; t < MC; ++t) {
      const int k0 = min(c0 + NW * t, nch - 1) * kBK;
      ld8(hrow + k0, a[t]);
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) b[t][s2] = wcol[(size_t)(k0 + 8 * g + s2) * C];
    }
#pragma unroll
    for (int t = 0; t < MC; ++t)
      if (c0 + NW * t < nch) acc = mfma_chunk8<false>(a[t], b[t], acc);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) zp[w][4 * g + i][r] = acc[i];
  __syncthreads();

  // wavefront i < 4 finishes row i of each lane group (16 lanes per row,
  // one class per lane)
  if (w < 4) {
    const int i = w;
    const int p = p0 + 4 * g + i;
    float z = zp[0][4 * g + i][r];
#pragma unroll
    for (int v = 1; v < NW; ++v) z += zp[v][4 * g + i][r];
    z += bsc;
    // log-sum-exp and softmax of the logits in fp64 (C exponentials per
    // vertex, a negligible cost): with small logits every vertex computes
    // nearly the same lse, so an fp32 rounding of it would repeat in every
    // row of dZ and add up coherently in the sums over vertices (db, db_s)
    const double zd = (double)z;
    double m = cval ? zd : -INFINITY;
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) m = fmax(m, __shfl_xor(m, o, kWave));
    double se = cval ? exp(zd - m) : 0.0;
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) se += __shfl_xor(se, o, kWave);
    const double lse = m + log(se);
    float d = 0.f;
    if (q[i] >= 0 && cval)
      d = (float)((exp(zd - lse) - (r == q[i] ? 1.0 : 0.0)) * (double)n.inv_denom);
    dzl[4 * g + i][r] = d;
    if (p < V) {
      if (r < CP && n.dZ) n.dZ[(size_t)p * CP + r] = d;
      if (q[i] < 0 && r == 0) n.lossv[p] = 0.f;
      if (q[i] >= 0 && r == q[i]) n.lossv[p] = (float)(lse - zd);
    }
  }
  if (!n.dHL) return;   // inference: no gradient of the head
  __syncthreads();
  float a[4];
  const int KT = CP / 4;
#pragma unroll
  for (int t = 0; t < 4; ++t) a[t] = t < KT ? dzl[r][4 * t + g] : 0.f;
  const int nb = H / 16;
  constexpr int MB = 4;
  for (int b0 = w; b0 < nb; b0 += NW * MB) {
    float wb[MB][4];
#pragma unroll
    for (int u = 0; u < MB; ++u) {
      const float* wrow = n.Ws + (size_t)(min(b0 + NW * u, nb - 1) * 16 + r) * C;
#pragma unroll
      for (int t = 0; t < 4; ++t) wb[u][t] = wrow[min(4 * t + g, C - 1)];
    }
    // classes past CP are never multiplied (t < KT below)
#pragma unroll
    for (int u = 0; u < MB; ++u) {
      const int jb = b0 + NW * u;
      if (jb >= nb) break;
      v4f o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (t < KT) o = mfma_f32_16x16x4(a[t], wb[u][t], o);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = p0 + 4 * g + i;
        if (p < V) n.dHL[(size_t)p * H + jb * 16 + r] = o[i];
      }
    }
  }
}

// Squared-error head: one wavefront per position; loss 0.5 |h - y|^2 and
// dHL = (h - y) / |Lambda| (zero rows for unlabelled positions; not written
// in inference, where dHL is null).
__global__ void __launch_bounds__(256) k_loss_l2(Net n) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int p = blockIdx.x * 4 + w;
  if (blockIdx.x == 0)   // the zero row the lazy products read for absent rows
    for (int j = threadIdx.x; j < n.H; j += 256) n.zrow[j] = 0.f;
  if (p >= n.V) return;
  const int q = n.push_pos[p], H = n.H;
  const float* h = n.Hs + (size_t)p * H;
  float* dh = n.dHL ? n.dHL + (size_t)p * H : nullptr;   // null in inference
  if (q < 0) {
    if (lane == 0) n.lossv[p] = 0.f;
    if (dh)
      for (int j = lane; j < H; j += 64) dh[j] = 0.f;
    return;
  }
  const float* y = n.Y + (size_t)q * H;
  float s = 0.f;
  for (int j = lane; j < H; j += 64) {
    const float d = h[j] - y[j];
    s += d * d;
    if (dh) dh[j] = d * n.inv_denom;
  }
  s = wave_sum(s);
  if (lane == 0) n.lossv[p] = 0.5f * s;
}

__global__ void __launch_bounds__(1024) k_loss_sum(const float* __restrict__ lossv, int V,
                                                   float scale, float* out) {
  __shared__ float red[1024];
  float s = 0.f;
  for (int i = threadIdx.x; i < V; i += 1024) s += lossv[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int o = 512; o >= 1; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = red[0] * scale;
}

}  // namespace

size_t lazy_part_floats(int V, int D, int H, int N, int C) {
  (void)V;
  size_t a = (size_t)kMaxSplits * 4 * H * (size_t)H;        // dU / FC dW
  size_t b = (size_t)kMaxSplits * 4 * H * (size_t)(D + 64);  // dW_x (m tail padding)
  size_t c = (size_t)kBiasChunks * (4 * H + (size_t)(H + 1) * (C > 0 ? C : 0));
  (void)N;
  size_t m = a > b ? a : b;
  return m > c ? m : c;
}

void pull_gemm(const Net& n, int n_pull, bool with_f, int lo1, hipStream_t s) {
  if (n_pull <= 0) return;
  if (n.bf) {
    dim3 grid(cdiv(n_pull, 64), (with_f ? 4 : 3) * (n.H / 64));
    CAVS_LAUNCH("k_pull_gemm_bf", k_pull_gemm_bf, grid, dim3(256), 0, s, n, n_pull, (int)with_f);
    return;
  }
  if (pull_tile_applies(n, n_pull)) {
    const dim3 grid(cdiv(n_pull, 64) * (n.H / 32));
    if (with_f)
      CAVS_LAUNCH("k_pull_tile<4, 64, 2>", (k_pull_tile<4, 64, 2>), grid, dim3(256), 0, s, n,
                  n_pull, lo1);
    else
      CAVS_LAUNCH("k_pull_tile<3, 64, 2>", (k_pull_tile<3, 64, 2>), grid, dim3(256), 0, s, n,
                  n_pull, lo1);
    return;
  }
  dim3 grid(cdiv(n_pull, 64), n.H / 32);
  if (with_f)
    CAVS_LAUNCH("k_pull_leaf<4>", k_pull_leaf<4>, grid, dim3(256), 0, s, n, n_pull, lo1);
  else
    CAVS_LAUNCH("k_pull_leaf<3>", k_pull_leaf<3>, grid, dim3(256), 0, s, n, n_pull, lo1);
}

bool pull_tile_applies(const Net& n, int n_pull) {
  return !n.bf && n_pull > 0 && n.H % 256 == 0 && n.D > 0 && n.D % 4 == 0;
}

void dx_gemm(const Net& n, int n_pull, bool with_f, float* dX, hipStream_t s) {
  if (n_pull <= 0) return;
  dim3 grid(cdiv(n_pull, 64), cdiv(n.D, 64));
  if (!n.bf && (!with_f || n.N == 1) && n.D % 4 == 0) {
    // 32-row tiles: about three workgroups per CU at the benchmark shapes
    const dim3 g32(cdiv(n_pull, 32), cdiv(n.D, 64));
    CAVS_LAUNCH("k_dx_tile<32, 64, 3>", (k_dx_tile<32, 64, 3>), g32, dim3(256), 0, s, n, n_pull,
                (int)with_f, dX);
    return;
  }
  if (n.bf)
    CAVS_LAUNCH("k_dx_gemm_bf", k_dx_gemm_bf, grid, dim3(256), 0, s, n, n_pull, (int)with_f, dX);
  else
    CAVS_LAUNCH("k_dx_gemm", k_dx_gemm, grid, dim3(256), 0, s, n, n_pull, (int)with_f, dX);
}

// dhlx[p] = dHL[p] + ext[vertex of p]: the gradient an external consumer of
// the pushed states sends back (vertex-id rows), joined to the loss head's.
__global__ void __launch_bounds__(256) k_add_ext(Net n, const float* __restrict__ ext,
                                                 float* __restrict__ dhlx) {
  const int q = n.H / 4;
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long long)n.V * q) return;
  const int p = (int)(i / q), j0 = 4 * (int)(i % q);
  const int v = n.order[p];
  st4(dhlx + (size_t)p * n.H + j0,
      add4(ldg4(n.dHL + (size_t)p * n.H + j0), ldg4(ext + (size_t)v * n.H + j0)));
}

void add_external_grad(const Net& n, const float* ext, float* dhlx, hipStream_t s) {
  if (n.V <= 0) return;
  CAVS_LAUNCH("k_add_ext", k_add_ext, dim3(cdiv((long)n.V * (n.H / 4), 256)), dim3(256), 0, s, n,
              ext, dhlx);
}

void loss_fwd(const Net& n, float* loss_out, hipStream_t s) {
  if (n.loss == CAVS_LOSS_NONE || (n.loss == CAVS_LOSS_CE && n.C > kSmallHeadC))
    (void)zero_async(n.zrow, (size_t)n.H * sizeof(float), s);   // the small heads' kernels clear it
  if (n.loss == CAVS_LOSS_NONE) {   // states pushed to an external consumer only
    (void)zero_async(n.lossv, (size_t)n.V * sizeof(float), s);
    if (n.dHL) (void)zero_async(n.dHL, (size_t)n.V * n.H * sizeof(float), s);
  } else if (n.loss == CAVS_LOSS_CE && n.C > kSmallHeadC) {
    lm_head_fwd(n, s);
  } else if (n.loss == CAVS_LOSS_CE) {
    const int per = cdiv(n.H / kBK, kLossWaves);  // K chunks per wavefront
    const dim3 grid(cdiv(n.V, 16)), block(64 * kLossWaves);
    if (per <= 1) CAVS_LAUNCH("k_loss_ce<1>", k_loss_ce<1>, grid, block, 0, s, n);
    else if (per <= 2) CAVS_LAUNCH("k_loss_ce<2>", k_loss_ce<2>, grid, block, 0, s, n);
    else CAVS_LAUNCH("k_loss_ce<4>", k_loss_ce<4>, grid, block, 0, s, n);
  } else {
    CAVS_LAUNCH("k_loss_l2", k_loss_l2, dim3(cdiv(n.V, 4)), dim3(256), 0, s, n);
  }
  CAVS_LAUNCH("k_loss_sum", k_loss_sum, dim3(1), dim3(1024), 0, s, (const float*)n.lossv, n.V,
                     n.inv_denom, loss_out);
}

// One product of a grouped launch: out[:, cols] = sum over q < Q of
// A(q)^T B(q) ([Mo, No]), reduced from its split-K partials (part) into dst
// as split_sum does; BM x BN is the tile shape the kernel instantiation
// gives it.
struct TnPlan {
  bool on;
  int Q, Mo, No;
  float* dst;
  int ldd, col_off, gap_start, gap;
  float* part;
  size_t part_floats;
  int BM, BN;
};

// At most this many workgroups per grouped launch: one round, one per CU (a
// product workgroup holds 120-156 KB of LDS).
constexpr int kTnGroupWGs = 256;

// Split counts: the smallest per-workgroup MFMA work u (32-deep chunks x
// tile area, in 128 x 256 units) for which every product, split so that no
// workgroup carries more than u, fits the launch in one round.
template <class K, class LA, class LB, class LC>
void tn_group_launch(K kernel, const char* name, TnGroupArgs<LA, LB, LC>& g, const TnPlan (&P)[3],
                     hipStream_t st, SplitJobs* jobs) {
  int nch[3] = {0, 0, 0}, tiles[3] = {0, 0, 0}, area[3] = {0, 0, 0}, cap[3] = {0, 0, 0};
  std::vector<long> cand;
  for (int k = 0; k < 3; ++k) {
    if (!P[k].on || P[k].Q <= 0) continue;
    nch[k] = cdiv(P[k].Q, kBK);
    tiles[k] = (P[k].No / P[k].BN) * cdiv(P[k].Mo, P[k].BM);
    area[k] = P[k].BM * P[k].BN / (64 * 128);   // 1, 2 or 4
    cap[k] = nch[k];
    while (cap[k] > 1 && (size_t)cap[k] * P[k].Mo * P[k].No > P[k].part_floats) --cap[k];
    for (int c = 1; c <= nch[k]; ++c) cand.push_back((long)c * area[k]);
  }
  auto splits = [&](int k, long u) {   // fewest splits with at most u per workgroup
    const long per = u / area[k];
    int sk = per < 1 ? cap[k] : (int)cdiv(nch[k], (int)(per < nch[k] ? per : nch[k]));
    return sk > cap[k] ? cap[k] : sk;
  };
  auto wgs = [&](long u) {
    long t = 0;
    for (int k = 0; k < 3; ++k)
      if (nch[k] > 0) t += (long)tiles[k] * splits(k, u);
    return t;
  };
  long u = 0;
  if (!cand.empty()) {
    std::sort(cand.begin(), cand.end());
    cand.erase(std::unique(cand.begin(), cand.end()), cand.end());
    size_t lo = 0, hi = cand.size() - 1;   // wgs() does not increase with u
    while (lo < hi) {
      const size_t mid = (lo + hi) / 2;
      if (wgs(cand[mid]) <= kTnGroupWGs) hi = mid;
      else lo = mid + 1;
    }
    u = cand[lo];
  }
  int end = 0, S[3] = {0, 0, 0};
  for (int k = 0; k < 3; ++k) {
    TnJob& J = g.j[k];
    J = TnJob{0, 0, 0, 0, 1, 1, end, nullptr};
    if (nch[k] == 0) continue;
    const int qchunk = cdiv(cdiv(P[k].Q, splits(k, u)), kBK) * kBK;
    S[k] = cdiv(P[k].Q, qchunk);
    end += tiles[k] * S[k];
    J = TnJob{P[k].Q, qchunk, P[k].Mo, P[k].No, P[k].No / P[k].BN, cdiv(P[k].Mo, P[k].BM), end,
              P[k].part};
  }
  if (end > 0) CAVS_LAUNCH(name, kernel, dim3(end), dim3(512), 0, st, g);
  for (int k = 0; k < 3; ++k)
    if (P[k].on)
      split_sum(P[k].part, S[k], P[k].Mo, P[k].No, P[k].dst, P[k].ldd, P[k].col_off,
                P[k].gap_start, P[k].gap, st, jobs);
}

bool lstm_lazy_grouped(const Net& n, int off1, int n_pull, bool with_f, float* dU, float* dWx,
                       float* part, size_t pf, hipStream_t s, SplitJobs* jobs) {
  const int H = n.H, D = n.D, MI = n.V - off1;
  if (n.N != 2 || D <= 0) return false;
  TnGroupArgs<LdDUf, LdDWx, LdDWx> g{LdDUf{n, off1, MI}, LdDWx{n, (int)with_f},
                                     LdDWx{n, (int)with_f}, {}};
  const int NoC = with_f ? 4 * H : 3 * H;
  if (!tn_direct_ok(n, g.a.direct(), H, H) || !tn_direct_ok(n, g.b.direct(), D, NoC)) return false;
  // dU_iou (the largest) alone fills the chip; dU_f and dW_x share a launch
  lstm_dU_iou(n, off1, dU, part, pf, s, jobs);
  // dW_x: 64-row tiles where they waste fewer rows of D
  const bool c64 = cdiv(D, 64) * 64 - D < cdiv(D, 128) * 128 - D;
  const TnPlan P[3] = {
      {true, 2 * MI, H, H, dU, 4 * H, H, 1 << 30, 0, part + pf, pf, 128, 128},
      {true, n_pull, D, NoC, dWx, 4 * H, 0, with_f ? 1 << 30 : H, with_f ? 0 : H, part + 2 * pf,
       pf, c64 ? 64 : 128, 256},
      {false, 0, 0, 0, nullptr, 0, 0, 0, 0, nullptr, 0, 128, 256}};
  if (c64)
    tn_group_launch(k_tn_group<LdDUf, 128, 128, 4, LdDWx, 64, 256, 3, LdDWx, 64, 256, 3>,
                    "k_tn_group<dUf, dWx64>", g, P, s, jobs);
  else
    tn_group_launch(k_tn_group<LdDUf, 128, 128, 4, LdDWx, 128, 256, 3, LdDWx, 128, 256, 3>,
                    "k_tn_group<dUf, dWx128>", g, P, s, jobs);
  // the f block of dW_x is exactly zero when no vertex with children pulls
  if (!with_f) split_sum(part + 2 * pf, 0, D, H, dWx, 4 * H, H, 1 << 30, 0, s, jobs);
  return true;
}

void lstm_dU_iou(const Net& n, int off1, float* dU, float* part, size_t part_floats,
                 hipStream_t s, SplitJobs* jobs, int rows) {
  const int H = n.H, MI = rows >= 0 ? rows : n.V - off1;
  LdDUiou ld{n, off1};
  if (n.N == 1) tn_product(ld, MI, H, 4 * H, dU, 4 * H, 0, 1 << 30, 0, part, part_floats, s, jobs);
  else tn_product(ld, MI, H, 3 * H, dU, 4 * H, 0, H, H, part, part_floats, s, jobs);
}

void lstm_dU_f(const Net& n, int off1, float* dU, float* part, size_t part_floats, hipStream_t s,
               SplitJobs* jobs, int rows) {
  if (n.N != 2) return;
  const int H = n.H, MI = rows >= 0 ? rows : n.V - off1;
  LdDUf lf{n, off1, MI};
  tn_product(lf, 2 * MI, H, H, dU, 4 * H, H, 1 << 30, 0, part, part_floats, s, jobs);
}

void reduce_split_jobs(const SplitJobs& jobs, hipStream_t s) {
  if (jobs.n == 0) return;
  long most = 0;
  for (int k = 0; k < jobs.n; ++k) {
    const SplitJob& J = jobs.j[k];
    // elements per block: 4096 (four per thread), or 64 columns of a kind-1 job
    const long e = J.kind == 1 ? (long)cdiv(J.No, 64) * 4096 : (long)J.Mo * J.No;
    most = e > most ? e : most;
  }
  CAVS_LAUNCH("k_reduce_jobs", k_reduce_jobs, dim3(cdiv(most, 4096), jobs.n), dim3(1024), 0, s,
              jobs);
}

void lstm_dWx(const Net& n, int n_pull, bool with_f, float* dWx, float* part,
              size_t part_floats, hipStream_t s, SplitJobs* jobs) {
  const int H = n.H;
  LdDWx ld{n, (int)with_f};
  if (with_f) {
    tn_product(ld, n_pull, n.D, 4 * H, dWx, 4 * H, 0, 1 << 30, 0, part, part_floats, s, jobs);
  } else {
    tn_product(ld, n_pull, n.D, 3 * H, dWx, 4 * H, 0, H, H, part, part_floats, s, jobs);
    // the f block of dW_x is exactly zero: no vertex with children pulls
    split_sum(part, 0, n.D, H, dWx, 4 * H, H, 1 << 30, 0, s, jobs);
  }
}

void fc_dW(const Net& n, int off1, float* dW, float* part, size_t part_floats, hipStream_t s,
           SplitJobs* jobs) {
  const int H = n.H, MI = n.V - off1;
  TnGroupArgs<LdFCdW, LdFCdW, LdFCdW> g{LdFCdW{n, off1, 0}, LdFCdW{n, off1, 1}, LdFCdW{n, off1, 0},
                                        {}};
  if (n.N <= 2 && tn_direct_ok(n, g.a.direct(), H, H)) {
    // both child slots' products share one launch; their split-K partials
    // sit side by side
    TnPlan P[3];
    for (int k = 0; k < 3; ++k)
      P[k] = TnPlan{k < n.N, MI, H, H, dW + (size_t)k * H * H, H, 0, 1 << 30, 0,
                    part + k * part_floats, part_floats, 128, 128};
    tn_group_launch(k_tn_group<LdFCdW, 128, 128, 4, LdFCdW, 128, 128, 4, LdFCdW, 128, 128, 4>,
                    "k_tn_group<FCdW>", g, P, s, jobs);
    return;
  }
  for (int k = 0; k < n.N; ++k) {
    LdFCdW ld{n, off1, k};
    tn_product(ld, MI, H, H, dW + (size_t)k * H * H, H, 0, 1 << 30, 0, part, part_floats, s);
  }
}

size_t bias_part_floats(int H, int C) {
  return (size_t)kBiasChunks * (4 * (size_t)H + (size_t)H * (C > 0 ? C : 0) + (C > 0 ? C : 0));
}

void bias_head_grads(const Net& n, int row0, int row1, int lo1, float* db, float* dWs, float* dbs,
                     float* part, hipStream_t s, SplitJobs* jobs) {
  const int wA = n.GW == n.H ? n.H : 4 * n.H;
  const bool head = n.loss == CAVS_LOSS_CE && n.C <= kSmallHeadC;   // the LM head has its own
  const int HC = head ? n.H * n.C : 0;
  int nchunk = cdiv(n.V, 16);
  if (nchunk > kBiasChunks) nchunk = kBiasChunks;
  if (nchunk < 1) nchunk = 1;
  const int rows_per = cdiv(n.V > 0 ? n.V : 1, nchunk);
  nchunk = cdiv(n.V > 0 ? n.V : 1, rows_per);
  const int bxA = cdiv(wA / 4, 256), bxB = head ? cdiv(n.H / 4, 256) : 0;
  const dim3 grid(bxA + bxB, nchunk);
  auto part_launch = [&](auto kern, const char* name) {
    CAVS_LAUNCH(name, kern, grid, dim3(256), 0, s, n, row0, row1, lo1, rows_per, bxA, wA, nchunk,
                part);
  };
  switch (head ? n.CP / 4 : 1) {
    case 1: part_launch(k_bias_part<1>, "k_bias_part<1>"); break;
    case 2: part_launch(k_bias_part<2>, "k_bias_part<2>"); break;
    case 3: part_launch(k_bias_part<3>, "k_bias_part<3>"); break;
    default: part_launch(k_bias_part<4>, "k_bias_part<4>"); break;
  }
  auto queue = [&](const float* p, int No, float* dst) {
    jobs->j[jobs->n++] = SplitJob{p, dst, nchunk, 1, No, No, 0, 1 << 30, 0, 1};
  };
  queue(part, wA, db);
  if (head) {
    queue(part + (size_t)nchunk * wA, HC, dWs);
    queue(part + (size_t)nchunk * (wA + HC), n.C, dbs);
  }
}

}  // namespace cavs
