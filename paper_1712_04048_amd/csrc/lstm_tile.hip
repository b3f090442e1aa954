// LDS-tiled Tree-LSTM level products for the large batching tasks (levels
// with many vertices, Algorithm 1): the same products and fused epilogues as
// the split-K kernels, with operand tiles staged through LDS so that each
// element fetched from L2 feeds many MFMAs.
//
// A workgroup (4 wavefronts, 2 x 2) owns BM positions x BU hidden units.
// Operands move in 32-deep chunks straight from global memory into LDS
// (global_load_lds_dwordx4: lane i of a wavefront writes 16 bytes at
// m0 + 16 i, so one copy fills eight 128-byte LDS rows).  S stages form a
// ring: the copies of chunk c+S-1 are in flight while chunk c is multiplied.
// Each LDS row holds the 32 k of one operand row with its eight 16-byte
// quads XOR-swizzled by (row & 7), and each MFMA fragment is two 16-byte
// reads in the permuted-K order of mfma_chunk8.
//
// The copies are issued by inline asm, so the compiler neither counts them
// as LDS writes (it would otherwise wait for every copy in flight before
// each LDS read) nor orders them: the kernel waits for its own copies with
// s_waitcnt vmcnt(n) and separates the stages with a bare s_barrier (the
// workgroup fence of __syncthreads would also wait for every copy).  No
// other vector memory operation is issued inside the chunk loop, so vmcnt
// counts exactly these copies; the stages are distinct LDS variables.
//
// Forward: A = the gathered child rows h_0, h_1 (h~ = h_0 + h_1 is formed in
// registers; an absent child reads a zero row), B = U^T (U transposed once
// per forward pass so that B rows are k-contiguous too); five accumulators
// per 16 x 16 block (i, o, u from h~, f_0 from h_0, f_1 from h_1).
// Backward: A = dA rows of the level, B = U (row n of U is column n of U^T);
// phase 1 contracts the i|o|u columns, phase 2 the f_0 and f_1 columns with
// the shared U_f block.
#include "lds_ring.h"
#include "lstm_dev.h"

namespace cavs {
namespace {

// UT[c][k] = U[k][c] for the [H, 4H] recurrent weight (block rows y < H/32)
// and WxT[c][k] = W_x[k][c] for the [D, 4H] input weight (the rows above);
// block (0, 0) also clears the zero row read for absent operand rows.
__global__ void __launch_bounds__(256) k_transpose_u(const float* __restrict__ U,
                                                     float* __restrict__ UT,
                                                     const float* __restrict__ Wx,
                                                     float* __restrict__ WxT,
                                                     float* __restrict__ zrow, int H, int D) {
  __shared__ float t[32][33];
  const int H4 = 4 * H, yu = H / 32;
  const bool wx = (int)blockIdx.y >= yu;
  const float* src = wx ? Wx : U;
  float* dst = wx ? WxT : UT;
  const int K = wx ? D : H;
  const int c0 = blockIdx.x * 32, k0 = (wx ? blockIdx.y - yu : blockIdx.y) * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  if (blockIdx.x == 0 && blockIdx.y == 0)
    for (int j = threadIdx.x; j < H; j += 256) zrow[j] = 0.f;
  for (int y = ty; y < 32; y += 8)
    if (k0 + y < K) t[y][tx] = src[(size_t)(k0 + y) * H4 + c0 + tx];
  __syncthreads();
  if (k0 + tx < K)
    for (int y = ty; y < 32; y += 8) dst[(size_t)(c0 + y) * K + k0 + tx] = t[tx][y];
}

// Ub[k][c] = bf16(U[k][c]) and UTb[c][k] = bf16(U[k][c]) for the [H, 4H]
// recurrent weight: the bf16 operands of the split-K level products, rounded
// once per pass (nearest-even, as every other bf16 operand).
__global__ void __launch_bounds__(256) k_round_u(const float* __restrict__ U, u16* __restrict__ Ub,
                                                 u16* __restrict__ UTb, int H) {
  __shared__ u16 t[32][34];
  const int H4 = 4 * H, c0 = blockIdx.x * 32, k0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int y = ty; y < 32; y += 8) {
    const u16 v = f2bf(U[(size_t)(k0 + y) * H4 + c0 + tx]);
    Ub[(size_t)(k0 + y) * H4 + c0 + tx] = v;
    t[y][tx] = v;
  }
  __syncthreads();
  for (int y = ty; y < 32; y += 8) UTb[(size_t)(c0 + y) * H + k0 + tx] = t[tx][y];
}

template <int NCH, bool BF, int BM, int BU, int S>
__global__ void __launch_bounds__(256) k_lstm_fwd_tile(Net n, int off, int M) {
  constexpr int TM = BM / 32, TU = BU / 32;   // 16 x 16 blocks per wavefront
  constexpr int NACC = 3 + NCH;
  constexpr int AROWS = NCH * BM, ROWS = AROWS + 4 * BU;
  constexpr bool ILV = S == 2;   // copies interleaved with the MFMAs (measured faster)
  constexpr int IPW = ROWS / 32;               // copies per wavefront per chunk
  static_assert(IPW * 32 == ROWS && S >= 2 && S <= 4, "tile shape");
  __shared__ __attribute__((aligned(1024))) float L0[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L1[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L2[S > 2 ? ROWS * 32 : 4];
  __shared__ __attribute__((aligned(1024))) float L3[S > 3 ? ROWS * 32 : 4];
  const Ring<ROWS, S> ring{L0, L1, L2, L3};

  const int H = n.H;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w & 1, wu = w >> 1;
  int rt, ut;
  xcd_tile(H / BU, rt, ut);
  const int row0 = off + rt * BM, rowend = off + M, u0 = ut * BU;

  // Epilogue operands, prefetched before the product.  The weight fragment
  // is the MFMA's A operand, so in block (tm, tu) lane (r, gq) holds units
  // j0 .. j0+3 of one position p (four consecutive units: float4 access).
  FwdPos pos[TM];
  Bias4 bias[TU];
  FwdCell4<NCH> cell[TM][TU];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int p = row0 + wr * (BM / 2) + tm * 16 + r;
    pos[tm] = FwdPos{-1, -1, 0, -1};
    if (p < rowend) lstm_fwd_pos<NCH>(n, p, pos[tm]);
  }
#pragma unroll
  for (int tu = 0; tu < TU; ++tu) lstm_bias4(n, u0 + wu * (BU / 2) + tu * 16 + 4 * gq, bias[tu]);
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tu = 0; tu < TU; ++tu)
      lstm_fwd_cell4<NCH>(n, pos[tm], u0 + wu * (BU / 2) + tu * 16 + 4 * gq, cell[tm][tu]);

  // source of each of this lane's copies: LDS rows [0, AROWS) are child
  // rows (child slot ch of position row0 + rr), the rest rows of U^T
  const float* src[IPW];
#pragma unroll
  for (int t = 0; t < IPW; ++t) {
    const int row = (w * IPW + t) * 8 + (lane >> 3), qg = (lane & 7) ^ (row & 7);
    if (row < AROWS) {
      const int ch = row / BM, p = row0 + row % BM;
      const float* ptr = n.zrow;
      if (p < rowend) {
        const int cp = n.child_pos[(size_t)p * NCH + ch];
        if (cp >= 0) ptr = n.Hs + (size_t)cp * H;
      }
      src[t] = ptr + 4 * qg;
    } else {
      const int b = row - AROWS, g = b / BU, u = b % BU;
      src[t] = n.UT + (size_t)(g * H + u0 + u) * H + 4 * qg;
    }
  }
  const int wofs = __builtin_amdgcn_readfirstlane(w * IPW * 256);

  v4f acc[TM][TU][NACC];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tu = 0; tu < TU; ++tu)
#pragma unroll
      for (int g = 0; g < NACC; ++g) acc[tm][tu][g] = v4f{0.f, 0.f, 0.f, 0.f};

  auto issue = [&](auto sc, int c) {
    ring_issue<IPW, ILV>(ring.at(sc), wofs, [&](int t) { return src[t] + c * kBK; });
  };
  struct Frag {
    float a0[TM][8], a1[TM][8], b[4][TU][8];
  };
  auto read = [&](const float* Ls, Frag& f) {
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int tu = 0; tu < TU; ++tu)
        frag_sw(Ls, AROWS + g * BU + wu * (BU / 2) + tu * 16 + r, gq, f.b[g][tu]);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int ra = wr * (BM / 2) + tm * 16 + r;
      frag_sw(Ls, ra, gq, f.a0[tm]);
      if constexpr (NCH == 2) frag_sw(Ls, BM + ra, gq, f.a1[tm]);
    }
  };
  // A = weight fragment (units), B = child fragment (positions)
  auto mma = [&](const Frag& f) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      float ah[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) ah[s] = NCH == 2 ? f.a0[tm][s] + f.a1[tm][s] : f.a0[tm][s];
#pragma unroll
      for (int tu = 0; tu < TU; ++tu) {
        acc[tm][tu][0] = mfma_chunk8<BF>(f.b[G_I][tu], ah, acc[tm][tu][0]);
        acc[tm][tu][1] = mfma_chunk8<BF>(f.b[G_O][tu], ah, acc[tm][tu][1]);
        acc[tm][tu][2] = mfma_chunk8<BF>(f.b[G_U][tu], ah, acc[tm][tu][2]);
        acc[tm][tu][3] = mfma_chunk8<BF>(f.b[G_F][tu], f.a0[tm], acc[tm][tu][3]);
        if constexpr (NCH == 2)
          acc[tm][tu][4] = mfma_chunk8<BF>(f.b[G_F][tu], f.a1[tm], acc[tm][tu][4]);
      }
    }
  };
  auto body = [&](const float* Lnext, Frag& cur, Frag& nxt, int) {
    read(Lnext, nxt);
    mma(cur);
    ring_schedule<ILV, IPW, 2 * (4 * TU + NCH * TM), TM * TU * NACC * (BF ? 1 : 8)>();
  };
  ring_loop_db<S, IPW, Frag, ILV>(H / kBK, ring, issue, read, body);

#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int p = row0 + wr * (BM / 2) + tm * 16 + r;
    if (p >= rowend) continue;
#pragma unroll
    for (int tu = 0; tu < TU; ++tu)
      lstm_fwd_fin4<NCH>(n, p, u0 + wu * (BU / 2) + tu * 16 + 4 * gq, pos[tm], bias[tu],
                         cell[tm][tu], acc[tm][tu][0], acc[tm][tu][1], acc[tm][tu][2],
                         acc[tm][tu][3], NCH == 2 ? acc[tm][tu][NACC - 1] : v4f{0.f, 0.f, 0.f, 0.f});
  }
}

// Backward level product, organised like the forward: per 32-deep chunk of
// the unit index k, the stage holds the dA rows of the tile's positions for
// every gate block (i, o, u, f_0[, f_1]) and rows n of U for the tile's
// columns at each gate block, so one chunk feeds 3 + NCH MFMA blocks per
// 16 x 16 output block:
//   dL/dh~ += dA_i U_i^T + dA_o U_o^T + dA_u U_u^T,  dL/dh_k += dA_fk U_f^T
// (one child: the f block joins the single accumulator).  bf16: the operand
// rows are staged already rounded (dAb, written by the gates kernel, and
// Ub), so a 128-byte LDS row holds 64 k and a fragment's two 16-byte quads
// are the operands of two bf16 MFMA steps, with no conversion.
template <int NCH, bool BF, int BM, int BN, int S>
__global__ void __launch_bounds__(256) k_lstm_bwd_tile(Net n, int off, int M) {
  constexpr int TM = BM / 32, TN = BN / 32;
  constexpr int NGA = 3 + NCH;                 // dA blocks per chunk
  constexpr int NACC = NCH == 2 ? 3 : 1;
  constexpr int AROWS = NGA * BM, ROWS = AROWS + 4 * BN;
  // copies interleaved with the MFMAs: measured faster in fp32, slower with
  // bf16's half-length MFMA stream
  constexpr bool ILV = !BF && S == 2;
  constexpr int IPW = ROWS / 32;
  static_assert(IPW * 32 == ROWS && S >= 2 && S <= 4, "tile shape");
  __shared__ __attribute__((aligned(1024))) float L0[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L1[ROWS * 32];
  __shared__ __attribute__((aligned(1024))) float L2[S > 2 ? ROWS * 32 : 4];
  __shared__ __attribute__((aligned(1024))) float L3[S > 3 ? ROWS * 32 : 4];
  const Ring<ROWS, S> ring{L0, L1, L2, L3};

  const int H = n.H, H4 = 4 * H, GW = n.GW;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, gq = lane >> 4, r = lane & 15;
  const int wr = w & 1, wn = w >> 1;
  int rt, ut;
  xcd_tile(H / BN, rt, ut);
  const int row0 = off + rt * BM, rowend = off + M, n0 = ut * BN;

  // The weight fragment is the MFMA's A operand: in block (tm, tn) lane
  // (r, gq) holds columns 4gq .. 4gq+3 of one position.  Its children's
  // positions are fetched before the product.
  int cpos[TM][NCH];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int p = row0 + wr * (BM / 2) + tm * 16 + r;
#pragma unroll
    for (int k = 0; k < NCH; ++k) cpos[tm][k] = p < rowend ? n.child_pos[(size_t)p * NCH + k] : -1;
  }

  // Stage rows: [0, AROWS) dA rows, block a (0..NGA-1) for gate i, o, u,
  // f_0, f_1 (columns 0, 2H, 3H, H, 4H of the dA row; one child: i, o, u,
  // f); then 4 blocks of BN rows n of U at gate columns i, o, u, f.  Rows
  // past the level read its last row (their products are never stored).
  const float* src[IPW];
#pragma unroll
  for (int t = 0; t < IPW; ++t) {
    const int row = (w * IPW + t) * 8 + (lane >> 3), qg = (lane & 7) ^ (row & 7);
    size_t e;   // element offset of the row's k = 0
    if (row < AROWS) {
      const int a = row / BM, p = min(row0 + row % BM, rowend - 1);
      const int col = a == 0 ? 0 : a == 1 ? 2 * H : a == 2 ? 3 * H : a == 3 ? H : 4 * H;
      e = (size_t)p * GW + col;
    } else {
      const int b = row - AROWS, g = b / BN, nn = n0 + b % BN;
      e = (size_t)nn * H4 + (g == 0 ? G_I : g == 1 ? G_O : g == 2 ? G_U : G_F) * H;
    }
    if constexpr (BF) {   // 16-byte quad qg of bf16 values, addressed in floats' units
      const unsigned short* base16 = row < AROWS ? n.dAb : n.Ub;
      src[t] = reinterpret_cast<const float*>(base16 + e + 8 * qg);
    } else {
      src[t] = (row < AROWS ? n.dA : n.U) + e + 4 * qg;
    }
  }
  const int wofs = __builtin_amdgcn_readfirstlane(w * IPW * 256);

  v4f acc[TM][TN][NACC];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int g = 0; g < NACC; ++g) acc[tm][tn][g] = v4f{0.f, 0.f, 0.f, 0.f};

  auto issue = [&](auto sc, int c) {
    ring_issue<IPW, ILV>(ring.at(sc), wofs, [&](int t) { return src[t] + c * kBK; });
  };
  struct Frag {
    float a[NGA][TM][8], b[4][TN][8];
  };
  auto read = [&](const float* Ls, Frag& f) {
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        frag_sw(Ls, AROWS + g * BN + wn * (BN / 2) + tn * 16 + r, gq, f.b[g][tn]);
#pragma unroll
    for (int a = 0; a < NGA; ++a)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) frag_sw(Ls, a * BM + wr * (BM / 2) + tm * 16 + r, gq, f.a[a][tm]);
  };
  // A = weight fragment (columns), B = dA fragment (positions); bf16: the
  // two quads of a fragment are two 32-deep steps
  auto step = [&](const float (&w)[8], const float (&d)[8], v4f c) {
    if constexpr (BF) {
      const float4 w0 = make_float4(w[0], w[1], w[2], w[3]), w1 = make_float4(w[4], w[5], w[6], w[7]);
      const float4 d0 = make_float4(d[0], d[1], d[2], d[3]), d1 = make_float4(d[4], d[5], d[6], d[7]);
      c = mfma_bf16_16x16x32(__builtin_bit_cast(bf16x8, w0), __builtin_bit_cast(bf16x8, d0), c);
      return mfma_bf16_16x16x32(__builtin_bit_cast(bf16x8, w1), __builtin_bit_cast(bf16x8, d1), c);
    } else {
      return mfma_chunk8<false>(w, d, c);
    }
  };
  auto mma = [&](const Frag& f) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        v4f h = acc[tm][tn][0];
        h = step(f.b[0][tn], f.a[0][tm], h);
        h = step(f.b[1][tn], f.a[1][tm], h);
        h = step(f.b[2][tn], f.a[2][tm], h);
        if constexpr (NCH == 2) {
          acc[tm][tn][0] = h;
          acc[tm][tn][1] = step(f.b[3][tn], f.a[3][tm], acc[tm][tn][1]);
          acc[tm][tn][2] = step(f.b[3][tn], f.a[4][tm], acc[tm][tn][2]);
        } else {
          acc[tm][tn][0] = step(f.b[3][tn], f.a[3][tm], h);
        }
      }
  };
  auto body = [&](const float* Lnext, Frag& cur, Frag& nxt, int) {
    read(Lnext, nxt);
    mma(cur);
    ring_schedule<ILV, IPW, 2 * (4 * TN + NGA * TM), TM * TN * (3 + NCH) * (BF ? 2 : 8)>();
  };
  // a chunk is 32 k in fp32, 64 in bf16 (128 bytes per LDS row either way)
  ring_loop_db<S, IPW, Frag, ILV>(H / (BF ? 2 * kBK : kBK), ring, issue, read, body);

#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int p = row0 + wr * (BM / 2) + tm * 16 + r;
    if (p >= rowend) continue;
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int col0 = n0 + wn * (BN / 2) + tn * 16 + 4 * gq;
#pragma unroll
      for (int k = 0; k < NCH; ++k) {
        const int cp = cpos[tm][k];
        if (cp < 0) continue;
        v4f gh = acc[tm][tn][0];
        if constexpr (NCH == 2) gh += acc[tm][tn][1 + k];
        if (cp < n.fuse_from) {
          st4(n.dHp + (size_t)cp * H + col0, make_float4(gh[0], gh[1], gh[2], gh[3]));
        } else {
          // a child in the fused top levels (levels there never reach tile
          // size, so this path only keeps the kernel general)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            lstm_gates_elem<NCH>(n, cp, col0 + e, gh[e], n.dCp[(size_t)cp * H + col0 + e]);
        }
      }
    }
  }
}

}  // namespace

void lstm_transpose_u(const Net& n, hipStream_t s) {
  const int yw = n.Wx && n.D > 0 ? cdiv(n.D, 32) : 0;
  CAVS_LAUNCH("k_transpose_u", k_transpose_u, dim3(4 * n.H / 32, n.H / 32 + yw), dim3(256), 0, s,
              n.U, n.UT, n.Wx, n.WxT, n.zrow, n.H, n.D);
}

void lstm_round_u(const Net& n, hipStream_t s) {
  CAVS_LAUNCH("k_round_u", k_round_u, dim3(4 * n.H / 32, n.H / 32), dim3(256), 0, s, n.U, n.Ub,
              n.UTb, n.H);
}

#define CAVS_TILE_LAUNCH(KIND, NCH, BF, BM, BU, S)                                             \
  CAVS_LAUNCH_ROWS("k_lstm_" #KIND "_tile<" #NCH ", " #BF ", " #BM ", " #BU ", " #S ">", off, M, \
                   (k_lstm_##KIND##_tile<NCH, BF, BM, BU, S>),                                  \
                   dim3(cdiv(M, BM) * (n.H / BU)), dim3(256), 0, s, n, off, M)

#define CAVS_TILE_DISPATCH(KIND, BM, BU, S)                                                    \
  do {                                                                                         \
    if (n.N == 2) {                                                                            \
      if (n.bf) CAVS_TILE_LAUNCH(KIND, 2, true, BM, BU, S);                                    \
      else CAVS_TILE_LAUNCH(KIND, 2, false, BM, BU, S);                                        \
    } else {                                                                                   \
      if (n.bf) CAVS_TILE_LAUNCH(KIND, 1, true, BM, BU, S);                                    \
      else CAVS_TILE_LAUNCH(KIND, 1, false, BM, BU, S);                                        \
    }                                                                                          \
  } while (0)

bool lstm_tile_applies(const Net& n, int M) {
  return n.H % 256 == 0 && M >= kTileMinRows;
}

// Tile shapes and ring depths measured on MI355X (H = 512): the forward
// takes 64-position tiles once a level fills the chip twice over and 32
// below; the backward, with its larger per-tile stage, measured faster with
// 32-position tiles at every level size.
void lstm_fwd_tile(const Net& n, int off, int M, hipStream_t s) {
  if (M >= 1024) CAVS_TILE_DISPATCH(fwd, 64, 32, 2);
  else CAVS_TILE_DISPATCH(fwd, 32, 32, 2);
}

void lstm_bwd_tile(const Net& n, int off, int M, hipStream_t s) {
  CAVS_TILE_DISPATCH(bwd, 32, 32, 2);
}

}  // namespace cavs
