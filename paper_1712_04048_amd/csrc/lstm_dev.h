// Device helpers shared by the Tree-LSTM level kernels (split-K and
// LDS-tiled): the fused epilogues and the register-direct MFMA chunk.
#pragma once

#include "kernels.h"

namespace cavs {

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

// ----------------------------------------------------------------- backward
// dA of position p, unit j, and the dc scatter to its children, given the
// parent's contributions gh = dL/dh and gcin = dL/dc (zero at a root); the
// vertex's own loss term is added here.
__device__ __forceinline__ void lstm_bwd_gates_elem(const Net& n, int p, int j, float gh,
                                                    float gcin) {
  const int H = n.H;
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

// Epilogue of the backward level product for position p, unit col: child k
// receives dL/dh_k = zh + zf_k.  p is the child's only parent, so that is the
// child's whole dL/dh: a child at a position >= n.fuse_from (the small top
// levels) gets its dA and dc scatter here at once (its dL/dc was scattered
// when p's dA was formed); a child below that stores dL/dh for the
// elementwise gates kernel of its level.
template <int NCH>
__device__ __forceinline__ void lstm_bwd_scatter(const Net& n, int p, int col, float zh, float zf0,
                                                 float zf1) {
  const int H = n.H;
  const int cp0 = n.child_pos[(size_t)p * NCH];
  if (cp0 >= 0) {
    if (cp0 >= n.fuse_from) lstm_bwd_gates_elem(n, cp0, col, zh + zf0, n.dCp[(size_t)cp0 * H + col]);
    else n.dHp[(size_t)cp0 * H + col] = zh + zf0;
  }
  if constexpr (NCH == 2) {
    const int cp1 = n.child_pos[(size_t)p * NCH + 1];
    if (cp1 >= 0) {
      if (cp1 >= n.fuse_from) lstm_bwd_gates_elem(n, cp1, col, zh + zf1, n.dCp[(size_t)cp1 * H + col]);
      else n.dHp[(size_t)cp1 * H + col] = zh + zf1;
    }
  }
}

// Register-direct MFMA chunk: a[s], b[s] hold k = 8g + s of a 32-deep chunk
// (lane group g), so eight fp32 16x16x4 steps (or one bf16 16x16x32 step
// with the operands rounded to bf16) cover the chunk.
template <bool BF>
__device__ __forceinline__ v4f mfma_chunk8(const float (&a)[8], const float (&b)[8], v4f acc) {
  if constexpr (BF) {
    bf16x8 av, bv;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const u16 ua = f2bf(a[s]), ub = f2bf(b[s]);
      av[s] = __builtin_bit_cast(__bf16, ua);
      bv[s] = __builtin_bit_cast(__bf16, ub);
    }
    return mfma_bf16_16x16x32(av, bv, acc);
  } else {
#pragma unroll
    for (int s = 0; s < 8; ++s) acc = mfma_f32_16x16x4(a[s], b[s], acc);
    return acc;
  }
}

__device__ __forceinline__ void ld8(const float* p, float (&v)[8]) {
  const float4 x = ldg4(p), y = ldg4(p + 4);
  v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
}

// Workgroup b of a launch runs on XCD b % 8 (round-robin dispatch), and each
// XCD has its own L2.  Tiles are mapped so that XCD x only touches unit tiles
// x, x+8, ...: each L2 then holds 1/8 of the weight columns instead of all.
__device__ __forceinline__ void xcd_tile(int n_unit_tiles, int& row_tile, int& unit_tile) {
  const int bid = blockIdx.x, xcd = bid & 7, local = bid >> 3, per = n_unit_tiles >> 3;
  unit_tile = xcd + 8 * (local % per);
  row_tile = local / per;
}

}  // namespace cavs
