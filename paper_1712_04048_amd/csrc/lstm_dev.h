// Device helpers shared by the Tree-LSTM level kernels (split-K and
// LDS-tiled): the fused epilogues and the register-direct MFMA chunk.
#pragma once

#include "kernels.h"
#include "xcd_map.h"

namespace cavs {

// The epilogues are split into a part that needs only saved state (issued
// early, e.g. by wavefronts that wait for the matrix product) and a part
// that consumes the product.

// ------------------------------------------------------------------ forward
// Everything the forward epilogue of position p, unit j reads besides the
// matrix-product terms: bias (+ pulled input term) and the children's c.
template <int NCH>
struct FwdPre {
  float bi, bo, bu, pi, po, pu, fb;
  float cc[NCH];
  int cp[NCH], v, pulled;
};

// Loads of rows that other workgroups of the same launch wrote (the
// XCD-local level loop): device-scope buffer loads (sc1), which miss the
// CU's L1 and read the XCD's L2, where the writers' stores have landed.
// Offsets are 32-bit: the buffers hold fewer than 2^29 floats (checked on
// the host before such a launch).
constexpr int kRsrcWord3 = 0x00020000;   // raw buffer, 32-bit elements
constexpr int kLoadSc1 = 1 << 4;         // cache policy: device scope
struct CohBuf {
  __amdgpu_buffer_rsrc_t rs;
};
__device__ __forceinline__ CohBuf coh_buf(const float* base, size_t floats) {
  const size_t bytes = floats * 4;
  return CohBuf{__builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), 0,
                                                   (int)(bytes < 0x7fffffffu ? bytes : 0x7fffffffu),
                                                   kRsrcWord3)};
}
__device__ __forceinline__ float4 coh_ld4(const CohBuf& b, size_t idx) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(b.rs, (int)(idx * 4), 0,
                                                                         kLoadSc1));
}
__device__ __forceinline__ float coh_ld1(const CohBuf& b, size_t idx) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(b.rs, (int)(idx * 4), 0,
                                                                       kLoadSc1));
}

// Every load is unconditional (an absent child reads row 0, a position that
// pulls nothing its own unused row of P; both are masked by selects): a
// loaded value merged with a constant on a branch makes the compiler wait
// for that load on its own.  COH: the children's c rows may have been
// written by this launch (coherent loads).
template <int NCH, bool COH = false>
__device__ __forceinline__ void lstm_fwd_pre(const Net& n, int p, int j, FwdPre<NCH>& q) {
  const int H = n.H;
  const int pr = n.pull_pos[p];
  int cp[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) cp[k] = n.child_pos[(size_t)p * NCH + k];
  q.v = n.order[p];
  const float bi = n.b[G_I * H + j], bo = n.b[G_O * H + j], bu = n.b[G_U * H + j];
  const float bf = n.b[G_F * H + j];
  const float* Pp = n.P + (size_t)p * 4 * H;
  const float pi = Pp[G_I * H + j], po = Pp[G_O * H + j], pu = Pp[G_U * H + j];
  const float pf = Pp[G_F * H + j];
  float cc[NCH];
  if constexpr (COH) {
    const CohBuf cb = coh_buf(n.Cs, (size_t)n.V * H);
#pragma unroll
    for (int k = 0; k < NCH; ++k) cc[k] = coh_ld1(cb, (size_t)max(cp[k], 0) * H + j);
  } else {
#pragma unroll
    for (int k = 0; k < NCH; ++k) cc[k] = n.Cs[(size_t)max(cp[k], 0) * H + j];
  }
  q.pulled = pr >= 0;
  q.bi = bi;
  q.bo = bo;
  q.bu = bu;
  q.pi = q.pulled ? pi : 0.f;
  q.po = q.pulled ? po : 0.f;
  q.pu = q.pulled ? pu : 0.f;
  q.fb = q.pulled ? bf + pf : bf;
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    q.cp[k] = cp[k];
    q.cc[k] = cp[k] >= 0 ? cc[k] : 0.f;
  }
}

// Gates, cell update and the scatter of (c, h) for position p, unit j, from
// the matrix-product parts of the pre-activations (shared by both precisions).
template <int NCH>
__device__ __forceinline__ void lstm_fwd_fin(const Net& n, int p, int j, const FwdPre<NCH>& q,
                                             float zi, float zo, float zu, float zf0, float zf1) {
  const int H = n.H;
  if (n.fwd_unfused) {   // fusion ablation: the gates run in their own kernel
    float* g = n.Gs + (size_t)p * n.GW;
    g[j] = zi;
    g[H + j] = zf0;
    g[2 * H + j] = zo;
    g[3 * H + j] = zu;
    if constexpr (NCH == 2) g[4 * H + j] = zf1;
    return;
  }
  float ai = zi + q.bi, ao = zo + q.bo, au = zu + q.bu;
  if (q.pulled) {
    ai += q.pi;
    ao += q.po;
    au += q.pu;
  }
  const float ig = sigmoidf_(ai), og = sigmoidf_(ao), ug = tanh_(au);
  float c = ig * ug;
  float f0 = 0.f, f1 = 0.f;
  if (q.cp[0] >= 0) {
    f0 = sigmoidf_(zf0 + q.fb);
    c += f0 * q.cc[0];
  }
  if constexpr (NCH == 2) {
    if (q.cp[NCH - 1] >= 0) {
      f1 = sigmoidf_(zf1 + q.fb);
      c += f1 * q.cc[NCH - 1];
    }
  }
  const float h = og * tanh_(c);
  n.Hs[(size_t)p * H + j] = h;
  n.Cs[(size_t)p * H + j] = c;
  if (n.Gs) {   // null in inference: nothing reads the gates back
    float* g = n.Gs + (size_t)p * n.GW;
    g[j] = ig;
    g[H + j] = f0;
    g[2 * H + j] = og;
    g[3 * H + j] = ug;
    if constexpr (NCH == 2) g[4 * H + j] = f1;
  }
  n.h_out[(size_t)q.v * H + j] = h;
  if (n.c_out) n.c_out[(size_t)q.v * H + j] = c;
}

template <int NCH, bool COH = false>
__device__ __forceinline__ void lstm_fwd_epilogue(const Net& n, int p, int j, float zi, float zo,
                                                  float zu, float zf0, float zf1) {
  FwdPre<NCH> q;
  lstm_fwd_pre<NCH, COH>(n, p, j, q);
  lstm_fwd_fin<NCH>(n, p, j, q, zi, zo, zu, zf0, zf1);
}

// Forward epilogue over four consecutive units j0 .. j0+3 of one position
// (the layout of an MFMA block whose A operand is the weight fragment: lane
// (r, g) holds units 4g .. 4g+3 of position r).  What depends only on the
// position, only on the units, or on both is prefetched separately, before
// the product, so that its latency overlaps the matrix work.
struct FwdPos {
  int cp0, cp1, v, pr;  // child positions (-1 absent), vertex id, pull row (-1 none)
};
struct Bias4 {
  float4 i, f, o, u;
};
template <int NCH>
struct FwdCell4 {
  float4 cc[NCH];       // the children's c at the four units (zero if absent)
};

template <int NCH>
__device__ __forceinline__ void lstm_fwd_pos(const Net& n, int p, FwdPos& q) {
  q.cp0 = n.child_pos[(size_t)p * NCH];
  q.cp1 = NCH == 2 ? n.child_pos[(size_t)p * NCH + 1] : -1;
  q.v = n.order[p];
  q.pr = n.pull_pos[p];
}

__device__ __forceinline__ void lstm_bias4(const Net& n, int j0, Bias4& b) {
  const int H = n.H;
  b.i = ldg4(n.b + G_I * H + j0);
  b.f = ldg4(n.b + G_F * H + j0);
  b.o = ldg4(n.b + G_O * H + j0);
  b.u = ldg4(n.b + G_U * H + j0);
}

template <int NCH>
__device__ __forceinline__ void lstm_fwd_cell4(const Net& n, const FwdPos& q, int j0,
                                               FwdCell4<NCH>& e) {
  const int H = n.H;
  e.cc[0] = q.cp0 >= 0 ? ldg4(n.Cs + (size_t)q.cp0 * H + j0) : f4zero();
  if constexpr (NCH == 2) e.cc[1] = q.cp1 >= 0 ? ldg4(n.Cs + (size_t)q.cp1 * H + j0) : f4zero();
}

// Gates, cell update and the scatter of (c, h) for units j0 .. j0+3 of
// position p; z* hold the matrix-product parts of the pre-activations.
template <int NCH>
__device__ __forceinline__ void lstm_fwd_fin4(const Net& n, int p, int j0, const FwdPos& q,
                                              const Bias4& b, const FwdCell4<NCH>& e, v4f zi,
                                              v4f zo, v4f zu, v4f zf0, v4f zf1) {
  const int H = n.H;
  if (n.fwd_unfused) {   // fusion ablation: the gates run in their own kernel
    float* g = n.Gs + (size_t)p * n.GW + j0;
    auto v2f = [](v4f v) { return make_float4(v[0], v[1], v[2], v[3]); };
    st4(g, v2f(zi));
    st4(g + H, v2f(zf0));
    st4(g + 2 * H, v2f(zo));
    st4(g + 3 * H, v2f(zu));
    if constexpr (NCH == 2) st4(g + 4 * H, v2f(zf1));
    return;
  }
  float4 pi = f4zero(), pf = f4zero(), po = f4zero(), pu = f4zero();
  if (q.pr >= 0) {
    const float* Pp = n.P + (size_t)p * 4 * H + j0;
    pi = ldg4(Pp + G_I * H);
    pf = ldg4(Pp + G_F * H);
    po = ldg4(Pp + G_O * H);
    pu = ldg4(Pp + G_U * H);
  }
  // same association as the scalar epilogue: (z + b) + pulled term for
  // i, o, u; z + (b + pulled term) for f
  const float bi[4] = {b.i.x, b.i.y, b.i.z, b.i.w}, qi[4] = {pi.x, pi.y, pi.z, pi.w};
  const float bo[4] = {b.o.x, b.o.y, b.o.z, b.o.w}, qo[4] = {po.x, po.y, po.z, po.w};
  const float bu[4] = {b.u.x, b.u.y, b.u.z, b.u.w}, qu[4] = {pu.x, pu.y, pu.z, pu.w};
  const float bf[4] = {b.f.x + pf.x, b.f.y + pf.y, b.f.z + pf.z, b.f.w + pf.w};
  const float c0[4] = {e.cc[0].x, e.cc[0].y, e.cc[0].z, e.cc[0].w};
  float c1[4] = {0.f, 0.f, 0.f, 0.f};
  if constexpr (NCH == 2) {
    c1[0] = e.cc[1].x; c1[1] = e.cc[1].y; c1[2] = e.cc[1].z; c1[3] = e.cc[1].w;
  }
  float ig[4], og[4], ug[4], f0[4], f1[4], c[4], h[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    float ai = zi[k] + bi[k], ao = zo[k] + bo[k], au = zu[k] + bu[k];
    if (q.pr >= 0) {
      ai += qi[k];
      ao += qo[k];
      au += qu[k];
    }
    ig[k] = sigmoidf_(ai);
    og[k] = sigmoidf_(ao);
    ug[k] = tanh_(au);
    c[k] = ig[k] * ug[k];
    f0[k] = 0.f;
    f1[k] = 0.f;
    if (q.cp0 >= 0) {
      f0[k] = sigmoidf_(zf0[k] + bf[k]);
      c[k] += f0[k] * c0[k];
    }
    if constexpr (NCH == 2) {
      if (q.cp1 >= 0) {
        f1[k] = sigmoidf_(zf1[k] + bf[k]);
        c[k] += f1[k] * c1[k];
      }
    }
    h[k] = og[k] * tanh_(c[k]);
  }
  auto f4 = [](const float (&x)[4]) { return make_float4(x[0], x[1], x[2], x[3]); };
  st4(n.Hs + (size_t)p * H + j0, f4(h));
  st4(n.Cs + (size_t)p * H + j0, f4(c));
  if (n.Gs) {   // null in inference: nothing reads the gates back
    float* g = n.Gs + (size_t)p * n.GW + j0;
    st4(g, f4(ig));
    st4(g + H, f4(f0));
    st4(g + 2 * H, f4(og));
    st4(g + 3 * H, f4(ug));
    if constexpr (NCH == 2) st4(g + 4 * H, f4(f1));
  }
  st4(n.h_out + (size_t)q.v * H + j0, f4(h));
  if (n.c_out) st4(n.c_out + (size_t)q.v * H + j0, f4(c));
}

// ----------------------------------------------------------------- backward
// Everything dA of position p, unit j reads besides the parent's dL/dh: the
// loss head's term of dL/dh (written by the loss kernel), dL/dc from the
// parent, the saved gates and c, and the children's f_k and c_k.
template <int NCH>
struct GatePre {
  float lg, gcin, ig, og, ug, c;
  float fk[NCH], ck[NCH];
  int cp[NCH];
};

template <int NCH>
__device__ __forceinline__ void lstm_gates_pre(const Net& n, int p, int j, float gcin,
                                               GatePre<NCH>& q) {
  const int H = n.H;
  q.lg = n.dHL[(size_t)p * H + j];
  q.gcin = gcin;
  const float* g = n.Gs + (size_t)p * n.GW;
  q.ig = g[j];
  q.og = g[2 * H + j];
  q.ug = g[3 * H + j];
  q.c = n.Cs[(size_t)p * H + j];
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int cp = n.child_pos[(size_t)p * NCH + k];
    q.cp[k] = cp;
    q.fk[k] = cp >= 0 ? g[(k == 0 ? H : 4 * H) + j] : 0.f;
    q.ck[k] = cp >= 0 ? n.Cs[(size_t)cp * H + j] : 0.f;
  }
}

// dA of position p, unit j, and the dc scatter to its children, from the
// parent's dL/dh (gh_parent; zero at a root) and the prefetched state.
template <int NCH>
__device__ __forceinline__ void lstm_gates_fin(const Net& n, int p, int j, float gh_parent,
                                               const GatePre<NCH>& q) {
  const int H = n.H;
  const float gh = gh_parent + q.lg;
  const float tau = tanh_(q.c);
  const float d_o = gh * tau * q.og * (1.f - q.og);
  const float gc = q.gcin + gh * q.og * (1.f - tau * tau);
  const float d_i = gc * q.ug * q.ig * (1.f - q.ig);
  const float d_u = gc * q.ig * (1.f - q.ug * q.ug);
  float* da = n.dA + (size_t)p * n.GW;
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    float d_f = 0.f;
    if (q.cp[k] >= 0) {
      d_f = gc * q.ck[k] * q.fk[k] * (1.f - q.fk[k]);
      n.dCp[(size_t)q.cp[k] * H + j] = gc * q.fk[k];
    }
    if (q.cp[k] >= 0 || p >= n.f_unread_below) {
      da[(k == 0 ? H : 4 * H) + j] = d_f;
      if (n.dAb) n.dAb[(size_t)p * n.GW + (k == 0 ? H : 4 * H) + j] = f2bf(d_f);
    }
  }
  da[j] = d_i;
  da[2 * H + j] = d_o;
  da[3 * H + j] = d_u;
  if (n.dAb) {   // bf16: the copy the backward products read, rounded as they round it
    unsigned short* db = n.dAb + (size_t)p * n.GW;
    db[j] = f2bf(d_i);
    db[2 * H + j] = f2bf(d_o);
    db[3 * H + j] = f2bf(d_u);
  }
}

// dA of position p, unit j given the parent's contributions gh = dL/dh and
// gcin = dL/dc (zero at a root).
template <int NCH>
__device__ __forceinline__ void lstm_gates_elem(const Net& n, int p, int j, float gh, float gcin) {
  GatePre<NCH> q;
  lstm_gates_pre<NCH>(n, p, j, gcin, q);
  lstm_gates_fin<NCH>(n, p, j, gh, q);
}

// The same reads with every load unconditional (absent children read row
// 0 and are masked by selects; see lstm_fwd_pre), including dL/dc from the
// parent, for the small levels' fused epilogue.
// COH: dL/dc from the parent may have been written in the same launch.
template <int NCH, bool COH = false>
__device__ __forceinline__ void lstm_gates_pre_all(const Net& n, int p, int j, GatePre<NCH>& q) {
  const int H = n.H;
  const float* g = n.Gs + (size_t)p * n.GW;
  q.lg = n.dHL[(size_t)p * H + j];
  if constexpr (COH) q.gcin = coh_ld1(coh_buf(n.dCp, (size_t)n.V * H), (size_t)p * H + j);
  else q.gcin = n.dCp[(size_t)p * H + j];
  q.ig = g[j];
  q.og = g[2 * H + j];
  q.ug = g[3 * H + j];
  q.c = n.Cs[(size_t)p * H + j];
  int cp[NCH];
  float fk[NCH], ck[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    cp[k] = n.child_pos[(size_t)p * NCH + k];
    fk[k] = g[(k == 0 ? H : 4 * H) + j];
  }
#pragma unroll
  for (int k = 0; k < NCH; ++k) ck[k] = n.Cs[(size_t)max(cp[k], 0) * H + j];
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    q.cp[k] = cp[k];
    q.fk[k] = cp[k] >= 0 ? fk[k] : 0.f;
    q.ck[k] = cp[k] >= 0 ? ck[k] : 0.f;
  }
}

// Backward level epilogue for position p, unit col: child k receives
// dL/dh_k = zh + zf_k.  p is the child's only parent, so that is the child's
// whole dL/dh: a child at a position >= n.fuse_from (the small top levels)
// gets its dA and dc scatter here at once (its dL/dc was scattered when p's
// dA was formed); a child below that stores dL/dh for the elementwise gates
// kernel of its level.  BwdPre holds what can be read before the product.
template <int NCH>
struct BwdPre {
  GatePre<NCH> q[NCH];
  int cp[NCH];
};

template <int NCH, bool COH = false>
__device__ __forceinline__ void lstm_bwd_pre(const Net& n, int p, int col, BwdPre<NCH>& e) {
  int cp[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) cp[k] = n.child_pos[(size_t)p * NCH + k];
  // a child below fuse_from (or absent) reads row 0 here, unused
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    e.cp[k] = cp[k];
    lstm_gates_pre_all<NCH, COH>(n, cp[k] >= n.fuse_from ? cp[k] : 0, col, e.q[k]);
  }
}

template <int NCH>
__device__ __forceinline__ void lstm_bwd_fin(const Net& n, int col, const BwdPre<NCH>& e, float zh,
                                             float zf0, float zf1) {
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int cp = e.cp[k];
    if (cp < 0) continue;
    const float gh = zh + (k == 0 ? zf0 : zf1);
    if (cp >= n.fuse_from) lstm_gates_fin<NCH>(n, cp, col, gh, e.q[k]);
    else n.dHp[(size_t)cp * n.H + col] = gh;
  }
}

template <int NCH, bool COH = false>
__device__ __forceinline__ void lstm_bwd_scatter(const Net& n, int p, int col, float zh, float zf0,
                                                 float zf1) {
  BwdPre<NCH> e;
  lstm_bwd_pre<NCH, COH>(n, p, col, e);
  lstm_bwd_fin<NCH>(n, col, e, zh, zf0, zf1);
}

// Rows of a small-level tile: tile row i is position pos(i), or none (-1);
// clamp(i) is a valid position for the unconditional loads of row i.
// A contiguous range of a level ...
struct RangeRows {
  int row0, rowend;
  __device__ int pos(int i) const { return row0 + i < rowend ? row0 + i : -1; }
  __device__ int clamp(int i) const { return min(row0 + i, rowend - 1); }
};
// ... or m entries of a list of positions (relative to base) in LDS.
struct ListRows {
  const short* list;
  int m, base;
  __device__ int pos(int i) const { return i < m ? base + list[i] : -1; }
  __device__ int clamp(int i) const { return base + list[min(i, m - 1)]; }
};

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

// eight values rounded to bf16 (nearest-even), as one MFMA operand
__device__ __forceinline__ bf16x8 to_bf8(const float (&v)[8]) {
  bf16x8 b;
#pragma unroll
  for (int s = 0; s < 8; ++s) b[s] = __builtin_bit_cast(__bf16, f2bf(v[s]));
  return b;
}

__device__ __forceinline__ void ld8(const float* p, float (&v)[8]) {
  const float4 x = ldg4(p), y = ldg4(p + 4);
  v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
}

// XCD-aware tile order of a launch (xcd_map.h).
__device__ __forceinline__ void xcd_tile(int n_unit_tiles, int& row_tile, int& unit_tile) {
  const TileIdx t = xcd_tile_map(blockIdx.x, n_unit_tiles);
  row_tile = t.row_tile;
  unit_tile = t.unit_tile;
}

}  // namespace cavs
