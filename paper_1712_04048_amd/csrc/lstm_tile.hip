// LDS-tiled Tree-LSTM level products for the large batching tasks (levels
// with many vertices, Algorithm 1): the same products and fused epilogues as
// the split-K kernels, with operand tiles staged through LDS so that each
// element fetched from L2 feeds many MFMAs.
//
// A workgroup (4 wavefronts, 2 x 2) owns BM positions x BU hidden units.
// Each 32-deep chunk of both operands is copied global -> registers -> LDS
// with two LDS stages: the loads of chunk c+1 are in flight while chunk c is
// multiplied, and one barrier per chunk separates the stages.  Rows are
// stored k-contiguous (padded to kLDK floats), so every MFMA fragment is two
// 16-byte LDS reads in the permuted-K order of mfma_chunk8.
//
// Forward: A = the gathered child rows h_0, h_1 (h~ = h_0 + h_1 is formed in
// registers), B = U^T (U transposed once per forward pass so that B rows are
// k-contiguous too); five accumulators per 16 x 16 block (i, o, u from h~,
// f_0 from h_0, f_1 from h_1).
// Backward: A = dA rows of the level, B = U (row n of U is column n of U^T);
// phase 1 contracts the i|o|u columns, phase 2 the f_0 and f_1 columns with
// the shared U_f block.
#include "lstm_dev.h"

namespace cavs {
namespace {

constexpr int kLDK = kBK + 4;

// UT[c][k] = U[k][c] for the [H, 4H] recurrent weight.
__global__ void __launch_bounds__(256) k_transpose_u(const float* __restrict__ U,
                                                     float* __restrict__ UT, int H) {
  __shared__ float t[32][33];
  const int H4 = 4 * H;
  const int c0 = blockIdx.x * 32, k0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int y = ty; y < 32; y += 8) t[y][tx] = U[(size_t)(k0 + y) * H4 + c0 + tx];
  __syncthreads();
  for (int y = ty; y < 32; y += 8) UT[(size_t)(c0 + y) * H + k0 + tx] = t[tx][y];
}

__device__ __forceinline__ void lds8(const float* p, float (&v)[8]) {
  const float4 x = *reinterpret_cast<const float4*>(p);
  const float4 y = *reinterpret_cast<const float4*>(p + 4);
  v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
}

template <int NCH, bool BF, int BM, int BU>
__global__ void __launch_bounds__(256) k_lstm_fwd_tile(Net n, int off, int M) {
  constexpr int TM = BM / 32, TU = BU / 32;   // 16 x 16 blocks per wavefront
  constexpr int NACC = 3 + NCH;
  constexpr int A_PER = BM * NCH * 8 / 256;   // float4 per thread per chunk
  constexpr int B_PER = 4 * BU * 8 / 256;
  static_assert(A_PER * 256 == BM * NCH * 8 && B_PER * 256 == 4 * BU * 8, "tile split");
  __shared__ __attribute__((aligned(16))) float As[2][NCH][BM][kLDK];
  __shared__ __attribute__((aligned(16))) float Bs[2][4][BU][kLDK];

  const int H = n.H;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w & 1, wu = w >> 1;
  int rt, ut;
  xcd_tile(H / BU, rt, ut);
  const int row0 = off + rt * BM, rowend = off + M, u0 = ut * BU;

  const float* asrc[A_PER];
  int adst[A_PER];
#pragma unroll
  for (int a = 0; a < A_PER; ++a) {
    const int idx = tid + 256 * a, row = idx / (NCH * 8), ch = (idx / 8) % NCH, q = idx & 7;
    adst[a] = (ch * BM + row) * kLDK + 4 * q;
    asrc[a] = nullptr;
    const int p = row0 + row;
    if (p < rowend) {
      const int cp = n.child_pos[(size_t)p * NCH + ch];
      if (cp >= 0) asrc[a] = n.Hs + (size_t)cp * H + 4 * q;
    }
  }
  const float* bsrc[B_PER];
  int bdst[B_PER];
#pragma unroll
  for (int b = 0; b < B_PER; ++b) {
    const int idx = tid + 256 * b, g = idx / (BU * 8), u = (idx / 8) % BU, q = idx & 7;
    bsrc[b] = n.UT + (size_t)(g * H + u0 + u) * H + 4 * q;
    bdst[b] = (g * BU + u) * kLDK + 4 * q;
  }
  float4 ra[A_PER], rb[B_PER];
  auto gload = [&](int k0) {
#pragma unroll
    for (int a = 0; a < A_PER; ++a) ra[a] = asrc[a] ? ldg4(asrc[a] + k0) : f4zero();
#pragma unroll
    for (int b = 0; b < B_PER; ++b) rb[b] = ldg4(bsrc[b] + k0);
  };
  auto sstore = [&](int st) {
    float* A = &As[st][0][0][0];
    float* B = &Bs[st][0][0][0];
#pragma unroll
    for (int a = 0; a < A_PER; ++a) st4(A + adst[a], ra[a]);
#pragma unroll
    for (int b = 0; b < B_PER; ++b) st4(B + bdst[b], rb[b]);
  };

  v4f acc[TM][TU][NACC];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tu = 0; tu < TU; ++tu)
#pragma unroll
      for (int g = 0; g < NACC; ++g) acc[tm][tu][g] = v4f{0.f, 0.f, 0.f, 0.f};

  const int nch = H / kBK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    const int st = c & 1;
    if (c + 1 < nch) gload((c + 1) * kBK);
    float bfr[4][TU][8];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int tu = 0; tu < TU; ++tu)
        lds8(&Bs[st][g][wu * (BU / 2) + tu * 16 + r][8 * gq], bfr[g][tu]);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int row = wr * (BM / 2) + tm * 16 + r;
      float a0[8], a1[8], ah[8];
      lds8(&As[st][0][row][8 * gq], a0);
      if constexpr (NCH == 2) {
        lds8(&As[st][NCH - 1][row][8 * gq], a1);
#pragma unroll
        for (int s = 0; s < 8; ++s) ah[s] = a0[s] + a1[s];
      } else {
#pragma unroll
        for (int s = 0; s < 8; ++s) ah[s] = a0[s];
      }
#pragma unroll
      for (int tu = 0; tu < TU; ++tu) {
        acc[tm][tu][0] = mfma_chunk8<BF>(ah, bfr[G_I][tu], acc[tm][tu][0]);
        acc[tm][tu][1] = mfma_chunk8<BF>(ah, bfr[G_O][tu], acc[tm][tu][1]);
        acc[tm][tu][2] = mfma_chunk8<BF>(ah, bfr[G_U][tu], acc[tm][tu][2]);
        acc[tm][tu][3] = mfma_chunk8<BF>(a0, bfr[G_F][tu], acc[tm][tu][3]);
        if constexpr (NCH == 2) acc[tm][tu][4] = mfma_chunk8<BF>(a1, bfr[G_F][tu], acc[tm][tu][4]);
      }
    }
    if (c + 1 < nch) sstore(st ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tu = 0; tu < TU; ++tu)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = row0 + wr * (BM / 2) + tm * 16 + 4 * gq + i;
        const int j = u0 + wu * (BU / 2) + tu * 16 + r;
        if (p < rowend)
          lstm_fwd_epilogue<NCH>(n, p, j, acc[tm][tu][0][i], acc[tm][tu][1][i], acc[tm][tu][2][i],
                                 acc[tm][tu][3][i], NCH == 2 ? acc[tm][tu][NACC - 1][i] : 0.f);
      }
}

template <int NCH, bool BF, int BM, int BN>
__global__ void __launch_bounds__(256) k_lstm_bwd_tile(Net n, int off, int M) {
  constexpr int TM = BM / 32, TN = BN / 32;
  constexpr int NA = NCH == 2 ? 2 : 1;        // A operands of phase 2
  constexpr int NACC = NCH == 2 ? 3 : 1;
  constexpr int A_PER = BM * 8 / 256;         // float4 per thread per operand per chunk
  constexpr int B_PER = BN * 8 / 256;
  static_assert(A_PER * 256 == BM * 8 && B_PER * 256 == BN * 8, "tile split");
  __shared__ __attribute__((aligned(16))) float As[2][NA][BM][kLDK];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN][kLDK];

  const int H = n.H, H4 = 4 * H, GW = n.GW;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w & 1, wn = w >> 1;
  int rt, ut;
  xcd_tile(H / BN, rt, ut);
  const int row0 = off + rt * BM, rowend = off + M, n0 = ut * BN;

  const float* asrc[A_PER];
  int adst[A_PER];
#pragma unroll
  for (int a = 0; a < A_PER; ++a) {
    const int idx = tid + 256 * a, row = idx / 8, q = idx & 7;
    const int p = row0 + row;
    asrc[a] = p < rowend ? n.dA + (size_t)p * GW + 4 * q : nullptr;
    adst[a] = row * kLDK + 4 * q;
  }
  const float* bsrc[B_PER];
  int bdst[B_PER];
#pragma unroll
  for (int b = 0; b < B_PER; ++b) {
    const int idx = tid + 256 * b, nn = idx / 8, q = idx & 7;
    bsrc[b] = n.U + (size_t)(n0 + nn) * H4 + 4 * q;
    bdst[b] = nn * kLDK + 4 * q;
  }
  // phase 1: NCH == 2 contracts i|o|u (dA / U columns [0,H) and [2H,4H));
  // NCH == 1 all 4H columns.  Phase 2 (NCH == 2): f_0 at H, f_1 at 4H of dA,
  // both against U columns [H, 2H).
  const int nc1 = (NCH == 2 ? 3 * H : H4) / kBK, nc2 = NCH == 2 ? H / kBK : 0;
  const int nch = nc1 + nc2;
  float4 ra[NA][A_PER], rb[B_PER];
  auto gload = [&](int c) {
    if (c < nc1) {
      const int k0 = c * kBK, col = (NCH == 2 && k0 >= H) ? k0 + H : k0;
#pragma unroll
      for (int a = 0; a < A_PER; ++a) ra[0][a] = asrc[a] ? ldg4(asrc[a] + col) : f4zero();
#pragma unroll
      for (int b = 0; b < B_PER; ++b) rb[b] = ldg4(bsrc[b] + col);
    } else {
      const int k0 = (c - nc1) * kBK;
#pragma unroll
      for (int a = 0; a < A_PER; ++a) {
        ra[0][a] = asrc[a] ? ldg4(asrc[a] + H + k0) : f4zero();
        ra[NA - 1][a] = asrc[a] ? ldg4(asrc[a] + 4 * H + k0) : f4zero();
      }
#pragma unroll
      for (int b = 0; b < B_PER; ++b) rb[b] = ldg4(bsrc[b] + H + k0);
    }
  };
  auto sstore = [&](int st, int c) {
#pragma unroll
    for (int a = 0; a < A_PER; ++a) st4(&As[st][0][0][0] + adst[a], ra[0][a]);
    if (NCH == 2 && c >= nc1)
#pragma unroll
      for (int a = 0; a < A_PER; ++a) st4(&As[st][NA - 1][0][0] + adst[a], ra[NA - 1][a]);
#pragma unroll
    for (int b = 0; b < B_PER; ++b) st4(&Bs[st][0][0] + bdst[b], rb[b]);
  };

  v4f acc[TM][TN][NACC];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int g = 0; g < NACC; ++g) acc[tm][tn][g] = v4f{0.f, 0.f, 0.f, 0.f};

  gload(0);
  sstore(0, 0);
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    const int st = c & 1;
    if (c + 1 < nch) gload(c + 1);
    float bfr[TN][8];
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) lds8(&Bs[st][wn * (BN / 2) + tn * 16 + r][8 * gq], bfr[tn]);
    if (c < nc1) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        float a[8];
        lds8(&As[st][0][wr * (BM / 2) + tm * 16 + r][8 * gq], a);
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) acc[tm][tn][0] = mfma_chunk8<BF>(a, bfr[tn], acc[tm][tn][0]);
      }
    } else if constexpr (NCH == 2) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        float a0[8], a1[8];
        lds8(&As[st][0][wr * (BM / 2) + tm * 16 + r][8 * gq], a0);
        lds8(&As[st][NA - 1][wr * (BM / 2) + tm * 16 + r][8 * gq], a1);
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          acc[tm][tn][1] = mfma_chunk8<BF>(a0, bfr[tn], acc[tm][tn][1]);
          acc[tm][tn][NACC - 1] = mfma_chunk8<BF>(a1, bfr[tn], acc[tm][tn][NACC - 1]);
        }
      }
    }
    if (c + 1 < nch) sstore(st ^ 1, c + 1);
    __syncthreads();
  }

#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = row0 + wr * (BM / 2) + tm * 16 + 4 * gq + i;
        const int col = n0 + wn * (BN / 2) + tn * 16 + r;
        if (p < rowend)
          lstm_bwd_scatter<NCH>(n, p, col, acc[tm][tn][0][i], NCH == 2 ? acc[tm][tn][1][i] : 0.f,
                                NCH == 2 ? acc[tm][tn][NACC - 1][i] : 0.f);
      }
}

}  // namespace

void lstm_transpose_u(const Net& n, hipStream_t s) {
  CAVS_LAUNCH("k_transpose_u", k_transpose_u, dim3(4 * n.H / 32, n.H / 32), dim3(256), 0, s, n.U,
              n.UT, n.H);
}

#define CAVS_TILE_LAUNCH(KIND, NCH, BF, BM, BU)                                                \
  CAVS_LAUNCH_ROWS("k_lstm_" #KIND "_tile<" #NCH ", " #BF ", " #BM ", " #BU ">", off, M,        \
                   (k_lstm_##KIND##_tile<NCH, BF, BM, BU>),                                     \
                   dim3(cdiv(M, BM) * (n.H / BU)), dim3(256), 0, s, n, off, M)

#define CAVS_TILE_DISPATCH(KIND, BM, BU)                                                       \
  do {                                                                                         \
    if (n.N == 2) {                                                                            \
      if (n.bf) CAVS_TILE_LAUNCH(KIND, 2, true, BM, BU);                                       \
      else CAVS_TILE_LAUNCH(KIND, 2, false, BM, BU);                                           \
    } else {                                                                                   \
      if (n.bf) CAVS_TILE_LAUNCH(KIND, 1, true, BM, BU);                                       \
      else CAVS_TILE_LAUNCH(KIND, 1, false, BM, BU);                                           \
    }                                                                                          \
  } while (0)

bool lstm_tile_applies(const Net& n, int M) {
  return n.H % 256 == 0 && M >= kTileMinRows;
}

void lstm_fwd_tile(const Net& n, int off, int M, hipStream_t s) {
  if (M >= 1024) CAVS_TILE_DISPATCH(fwd, 64, 32);
  else CAVS_TILE_DISPATCH(fwd, 32, 32);
}

void lstm_bwd_tile(const Net& n, int off, int M, hipStream_t s) {
  if (M >= 1024) CAVS_TILE_DISPATCH(bwd, 64, 32);
  else CAVS_TILE_DISPATCH(bwd, 32, 32);
}

}  // namespace cavs
