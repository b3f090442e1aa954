// Kernel argument blocks, launchers and the fp32 MFMA tile engine shared by
// the forward / backward sources.
#pragma once

#include "cavs_internal.h"

namespace cavs {

// Per-batch device views.  All "by position" arrays use the level-major
// layout produced by the scheduler: task V_t = positions [off_t, off_{t+1}).
struct Net {
  int V, N, D, H, C, loss;
  int CP;                       // row stride of dZ: C rounded up to a multiple of 4
  int bf;                       // 1: matrix-product operands rounded to bf16
  int GW;                       // saved-gate / dA row width: (3+N)H (LSTM) or H (FC)
  float inv_denom;              // 1 / |Lambda|
  int fuse_from;                // LSTM backward: positions >= this get dA in the parent's epilogue
  int f_unread_below;           // LSTM backward: rows below this (leaves, when no vertex with
                                // children pulls) skip their dA forget columns: nothing reads them
  int fwd_unfused;              // LSTM forward: the level products store their pre-activation
                                // parts in the saved-gate rows and lstm_fwd_gates finishes
                                // (the fusion ablation)
  // schedule
  const int* child_pos;         // [V*N]
  const int* parent_pos;        // [V]
  const int* pull_pos;          // [V]
  const int* push_pos;          // [V]
  const int* order;             // [V]
  const int* pull_list;         // [n_pull]
  // parameters and inputs
  const float* Wx;              // [D, 4H]
  const float* U;               // LSTM [H, 4H]; FC [N*H, H]
  float* UT;                    // LSTM: U transposed, [4H, H]; FC: each slot's block
                                // transposed, [N, H, H] (workspace)
  float* WxT;                   // LSTM: W_x transposed, [4H, D] (workspace)
  unsigned short* Ub;           // LSTM bf16: U rounded to bf16, [H, 4H] (workspace; null in
  unsigned short* UTb;          // fp32) and U^T rounded to bf16, [4H, H]; written per pass
  unsigned short* dAb;          // LSTM bf16 training: dA rounded to bf16, [V, GW], written
                                // with dA for internal positions (the backward products'
                                // operand rows; null otherwise)
  float* zrow;                  // H zeros (workspace): the row an absent operand row reads;
                                // cleared by the transpose kernel and by the loss kernel
  const float* b;
  const float* Ws;              // [H, C]
  float* WsT;                   // [C, H] W_s transposed (workspace; the LM head)
  const float* bs;              // [C]
  const float* X;               // [n_x, D]
  const float* Y;               // [n_y, H]
  // workspace (level-major)
  float* P;                     // [V, 4H] pull projection x W_x (rows that pull)
  float* Hs;                    // [V, H]
  float* Cs;                    // [V, H]
  float* Gs;                    // [V, GW] saved gates  i | f_0 | o | u | f_1
  float* dZ;                    // [V, CP] d loss / d logits (columns >= C are zero)
  float* dHL;                   // [V, H]  the loss head's share of dL/dh (zero if unlabelled)
  float* lossv;                 // [V]     per-vertex loss terms
  float* dHp;                   // [V, H]  dL/dh contributed by the parent (LSTM)
  float* dCp;                   // [V, H]  dL/dc contributed by the parent
  float* dA;                    // [V, GW] pre-activation gradients, same layout as Gs
  unsigned short* pack;         // bf16 lazy products: operands packed q-contiguous (workspace;
  size_t pack_elems;            // null: the unpacked kernels), capacity in bf16 values
  // outputs in vertex-id order
  float* dX;                    // [n_x, D] input gradient (FC backward)
  int leaf_end;                 // FC backward: positions below this are leaves (level 0)
  float* h_out;
  float* c_out;
};

// gate column blocks of Wx / U / b (each H wide)
enum { G_I = 0, G_F = 1, G_O = 2, G_U = 3 };

// Most child slots the generic engine (generic.hip) takes; the fused engine
// takes two.
constexpr int kMaxSlots = 4;

// Workspace buffers of the generic engine (level-major; a link e = p * N + k
// is child slot k of position p).
struct GenBufDev {
  float* Ht;          // [V, H]     h~ = sum of the present children's h
  float* Dt;          // [V, H]     dL/dh~
  float* Eh;          // [V*N, H]   dL/dh sent back along each child link
  float* Ec;          // [V*N, H]   dL/dc sent back along each child link
  float* dAx;         // [V, 4H]    (d_i, sum_k d_fk, d_o, d_u): input and bias gradients
  float* part;        // split-K partial sums (gen_part_floats)
  size_t part_cap;    // floats in part
  const int* in_off;  // graph inputs: [V+1] offsets into in_edge per position; null for trees
  const int* in_edge; // graph inputs: links reading each position, ascending
};

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
// lstm.hip
void lstm_fwd_leaf(const Net& n, int off, int M, bool skip_pulled, hipStream_t s);
void lstm_fwd_level(const Net& n, int off, int M, hipStream_t s);
// Backward dA of the levels below n.fuse_from: elementwise over level rows
// (dL/dh and dL/dc as stored by the parents); roots at or above it.
void lstm_bwd_gates(const Net& n, int off, int M, hipStream_t s);
void lstm_bwd_roots(const Net& n, hipStream_t s);
void lstm_bwd_level(const Net& n, int off, int M, hipStream_t s);
// First level whose rows (and those of every level above) get their dA in
// the parent's epilogue: levels of at most kFuseRows positions.
constexpr int kFuseRows = 256;
// the hidden width the weight-stationary XCD-local level loop is built for
constexpr int kXcdWsH = 512;
int lstm_fuse_level(const int* lo_host, int T);
// lstm_tile.hip: LDS-tiled level products for levels of >= kTileMinRows
// positions (needs n.UT, written by lstm_transpose_u in the same pass).
constexpr int kTileMinRows = 300;
bool lstm_tile_applies(const Net& n, int M);
void lstm_transpose_u(const Net& n, hipStream_t s);
// bf16: n.Ub and n.UTb from n.U (before any level product of the pass)
void lstm_round_u(const Net& n, hipStream_t s);
void lstm_fwd_tile(const Net& n, int off, int M, hipStream_t s);
void lstm_bwd_tile(const Net& n, int off, int M, hipStream_t s);
// Persistent loop over levels [t0, t1) (forward) or t1-1 .. t0 (backward:
// gates and products) in one cooperative launch.  `lo` is the device copy of
// the level offsets, `lo_host` the host copy, `bar` 256 zeroed ints of
// barrier state.  Returns false (nothing launched) when the path does not
// apply or the cooperative launch is refused; the caller then falls back to
// per-level launches.
bool lstm_fwd_persist(const Net& n, const int* lo, const int* lo_host, int t0, int t1, int* bar,
                      hipStream_t s);
bool lstm_bwd_persist(const Net& n, const int* lo, const int* lo_host, int t0, int t1, int* bar,
                      hipStream_t s);
// First level >= 1 small enough for the persistent loop (T if none).
int persist_first_level(const Net& n, const int* lo_host, int T);
// XCD-local small-level loop: the first level it takes (T: none), its
// workspace, the owner computation of the suffix from level t0 (also clears
// the loop's barrier words), and the two loops (false: nothing suitable
// launched, run the levels one by one).  With owner_ready the caller has
// already queued xcd_owner for this suffix and workspace, ordered before the
// loop.
int xcd_first_level(const Net& n, const int* lo_host, int T);
size_t xcd_ws_bytes(int V);
void xcd_owner(const Net& n, const int* lo_host, int t0, void* xws, hipStream_t s);
bool lstm_fwd_xcd(const Net& n, const int* lo, const int* lo_host, int t0, int T, void* xws,
                  bool owner_ready, hipStream_t s);
bool lstm_bwd_xcd(const Net& n, const int* lo, const int* lo_host, int t0, int T, void* xws,
                  bool owner_ready, hipStream_t s);
// generic.hip
// Forward gates of positions [off, off + M) from the pre-activation parts in
// the saved-gate rows (has_product false: none, as for leaves).
void lstm_fwd_gates(const Net& n, int off, int M, bool has_product, hipStream_t s);
void gen_forward_levels(const Net& n, const GenBufDev& b, const int* lo_host, int T,
                        hipStream_t s);
void gen_backward(const Net& n, const GenBufDev& b, const int* lo_host, int T, int n_pull,
                  float* dU, float* db, float* dWx, float* dX, float* dWs, float* dbs,
                  hipStream_t s);
size_t gen_part_floats(int D, int H, int CP);
// Softmax heads with more than kSmallHeadC classes (a language-model
// vocabulary): logits, log-sum-exp, dZ and dL/dh on the generic products.
constexpr int kSmallHeadC = 16;
// per-vertex loss terms into lossv (and dZ, dL/dh when training)
void lm_head_fwd(const Net& n, hipStream_t s);
void lm_head_grads(const Net& n, float* dWs, float* dbs, float* part, size_t part_cap,
                   hipStream_t s);
// fc.hip
void fc_fwd_leaf(const Net& n, int off, int M, hipStream_t s);
void fc_fwd_level(const Net& n, int off, int M, hipStream_t s);
// backward: fc_bwd_roots, then fc_bwd_level for t = T-1 .. 1 (needs n.dX,
// n.leaf_end)
void fc_bwd_roots(const Net& n, hipStream_t s);
void fc_bwd_level(const Net& n, int off, int M, hipStream_t s);
// fc_fwd_level reads n.UT and n.zrow, written by fc_transpose earlier in the
// same pass
void fc_transpose(const Net& n, hipStream_t s);
// lazy.hip
// Pull projection; in fp32 the cell of every pulled leaf (position < lo1) is
// finished in the same kernel, so lstm_fwd_leaf only handles leaves without
// input (skip_pulled); in bf16 it writes P for all pulled rows.
void pull_gemm(const Net& n, int n_pull, bool with_f, int lo1, hipStream_t s);
// The pull product runs on the LDS ring (reading n.WxT, written by
// lstm_transpose_u earlier in the same pass).
bool pull_tile_applies(const Net& n, int n_pull);
void loss_fwd(const Net& n, float* loss_out, hipStream_t s);
// dhlx = the loss head's dL/dh plus an external gradient of the pushed
// states (vertex-id rows).
void add_external_grad(const Net& n, const float* ext, float* dhlx, hipStream_t s);
void dx_gemm(const Net& n, int n_pull, bool with_f, float* dX, hipStream_t s);
// Lazy weight-gradient products; `part` is split-K scratch of part_floats floats.
// Split-K sums waiting for their reduction: the lazy products append one
// job each (their partial sums must then stay in distinct scratch) and one
// launch reduces them all.
struct SplitJob {
  const float* part;
  float* dst;
  int S, Mo, No, ldd, col_off, gap_start, gap;
  int kind;     // 0: float4 sums; 1: Mo = 1, any No, the S partial rows split over 16 wavefronts
  int acc;      // kind 0: add the sum to what dst holds instead of overwriting it
};
struct SplitJobs {
  static constexpr int kMax = 8;
  SplitJob j[kMax];
  int n = 0;
};
void reduce_split_jobs(const SplitJobs& jobs, hipStream_t s);

// the lazy dU products: dU_iou (all four blocks with one child) and, with
// two children, dU_f (a no-op with one child)
// rows = the positions from off1 the products sum over (-1: every position
// from off1 to the end)
void lstm_dU_iou(const Net& n, int off1, float* dU, float* part, size_t part_floats,
                 hipStream_t s, SplitJobs* jobs = nullptr, int rows = -1);
void lstm_dU_f(const Net& n, int off1, float* dU, float* part, size_t part_floats, hipStream_t s,
               SplitJobs* jobs = nullptr, int rows = -1);
void lstm_dWx(const Net& n, int n_pull, bool with_f, float* dWx, float* part,
              size_t part_floats, hipStream_t s, SplitJobs* jobs = nullptr);
// the lazy weight-gradient products of the fused Tree-LSTM path: dU_iou,
// then dU_f and dW_x in one grouped launch, reductions queued on jobs;
// false (and nothing launched or queued) where the grouped kernel does not
// apply (one child slot, no inputs, bf16)
bool lstm_lazy_grouped(const Net& n, int off1, int n_pull, bool with_f, float* dU, float* dWx,
                       float* part, size_t pf, hipStream_t s, SplitJobs* jobs);
// part holds 3 part_floats (the slots' partials side by side); reductions
// are queued on jobs
void fc_dW(const Net& n, int off1, float* dW, float* part, size_t part_floats, hipStream_t s,
           SplitJobs* jobs);
// column sums over positions [row0, row1) of the gate gradients -> db
// db over rows [row0, row1) and, for the CE head, dW_s and db_s over all rows;
// rows below lo1 are level 0 (no children).  The per-chunk partial sums go
// to `part` (bias_part_floats floats); their reduction is queued on `jobs`.
size_t bias_part_floats(int H, int C);
void bias_head_grads(const Net& n, int row0, int row1, int lo1, float* db, float* dWs, float* dbs,
                     float* part, hipStream_t s, SplitJobs* jobs);
size_t lazy_part_floats(int V, int D, int H, int N, int C);

// ---------------------------------------------------------------------------
// fp32 MFMA tile engine (v_mfma_f32_16x16x4_f32, 64-lane wavefronts)
//
// Lane l = 16*g + r of a wavefront supplies A[row r][k_g] and B[k_g][col r]
// for one 4-deep K step and receives C[row 4g+i][col r], i = 0..3.  Inside a
// 32-deep LDS chunk the K index is permuted so that lane group g covers
// k = 8g .. 8g+7: an M-major ("MK", k contiguous) operand tile then serves
// four K steps per 128-bit LDS read.  A and B use the same permutation, so
// the sum over k is unchanged.
// ---------------------------------------------------------------------------
constexpr int kBK = 32;

template <bool MK, int LD>
__device__ __forceinline__ void load_frag4(const float* __restrict__ S, int idx, int gq, int half,
                                           float (&f)[4]) {
  if constexpr (MK) {
    const float4 t = *reinterpret_cast<const float4*>(&S[idx * LD + 8 * gq + 4 * half]);
    f[0] = t.x;
    f[1] = t.y;
    f[2] = t.z;
    f[3] = t.w;
  } else {
#pragma unroll
    for (int s = 0; s < 4; ++s) f[s] = S[(8 * gq + 4 * half + s) * LD + idx];
  }
}

// acc[tm][tn] += A[wrow + 16 tm .., :] * B[:, wcol + 16 tn ..] over one chunk.
template <int TM, int TN, bool A_MK, bool B_MK, int LDA, int LDB>
__device__ __forceinline__ void mfma_chunk(const float* __restrict__ As,
                                           const float* __restrict__ Bs, int wrow, int wcol,
                                           v4f (&acc)[TM][TN]) {
  const int lane = threadIdx.x & 63, gq = lane >> 4, r = lane & 15;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    float a[TM][4], b[TN][4];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) load_frag4<A_MK, LDA>(As, wrow + 16 * tm + r, gq, half, a[tm]);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) load_frag4<B_MK, LDB>(Bs, wcol + 16 * tn + r, gq, half, b[tn]);
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = mfma_f32_16x16x4(a[tm][s], b[tn][s], acc[tm][tn]);
  }
}

template <int TM, int TN>
__device__ __forceinline__ void zero_acc(v4f (&acc)[TM][TN]) {
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = v4f{0.f, 0.f, 0.f, 0.f};
}

__device__ __forceinline__ int cdiv_dev(int a, int b) { return (a + b - 1) / b; }
__device__ __forceinline__ float4 f4zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
__device__ __forceinline__ float4 ldg4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ void st4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
__device__ __forceinline__ void st4_scalar(float* p, float4 v) {
  p[0] = v.x;
  p[1] = v.y;
  p[2] = v.z;
  p[3] = v.w;
}
__device__ __forceinline__ float4 add4(float4 a, float4 b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

// ---------------------------------------------------------------------------
// bf16 MFMA engine (v_mfma_f32_16x16x32_bf16): lane l = 16*g + r supplies
// A[row r][k = 8g .. 8g+7] and B[k = 8g .. 8g+7][col r] as 8 bf16 values and
// receives C[row 4g+i][col r].  Tiles live in LDS as rows of kBK bf16 values
// (k contiguous), padded to kLDH, so each operand fragment is one 16-byte
// read.  Operands are rounded to bf16 (nearest-even) when staged into LDS;
// accumulation is fp32.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
// packed bf16 lazy products: q per 128-byte pack segment (the product's
// chunk) and the output tile of the packed product (both sides)
constexpr int kPackSeg = 64;
constexpr int kPackTile = 128;
typedef unsigned short u16;
constexpr int kLDH = kBK + 8;   // 40 bf16 = 80 bytes per row (16-byte aligned)

__device__ __forceinline__ u16 f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest, ties to even (finite inputs)
  return (u16)(u >> 16);
}

// 4 consecutive k of one row (8-byte store)
__device__ __forceinline__ void st_bf4(u16* dst, float4 v) {
  uint2 w;
  w.x = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
  w.y = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
  *reinterpret_cast<uint2*>(dst) = w;
}

// the same 4 values into 4 consecutive rows at column k (transposed store)
__device__ __forceinline__ void st_bf4_t(u16* dst, int ld, float4 v) {
  dst[0] = f2bf(v.x);
  dst[ld] = f2bf(v.y);
  dst[2 * ld] = f2bf(v.z);
  dst[3 * ld] = f2bf(v.w);
}

__device__ __forceinline__ bf16x8 frag_bf(const u16* S, int row, int gq) {
  return *reinterpret_cast<const bf16x8*>(&S[row * kLDH + 8 * gq]);
}

__device__ __forceinline__ v4f mfma_bf16_16x16x32(bf16x8 a, bf16x8 b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <int TM, int TN>
__device__ __forceinline__ void mfma_chunk_bf(const u16* __restrict__ As,
                                              const u16* __restrict__ Bs, int wrow, int wcol,
                                              v4f (&acc)[TM][TN]) {
  const int lane = threadIdx.x & 63, gq = lane >> 4, r = lane & 15;
  bf16x8 a[TM], b[TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) a[tm] = frag_bf(As, wrow + 16 * tm + r, gq);
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) b[tn] = frag_bf(Bs, wcol + 16 * tn + r, gq);
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = mfma_bf16_16x16x32(a[tm], b[tn], acc[tm][tn]);
}

}  // namespace cavs
