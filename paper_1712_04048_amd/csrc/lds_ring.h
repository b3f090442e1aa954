// Direct-to-LDS operand staging (gfx950 global_load_lds_dwordx4) with a
// ring of LDS stages, shared by the LDS-tiled products.
//
// A wavefront's copy instruction moves 16 bytes per lane from any global
// address to LDS at m0 + 16 * lane, i.e. eight 128-byte LDS rows.  Rows hold
// 32 floats (one 32-deep K chunk of an operand row) with their 16-byte quads
// XOR-swizzled by (row & 7).  The copies are issued by inline asm: the
// compiler then neither counts them as LDS writes (it would wait for every
// copy in flight before each LDS read) nor orders them, and the ring waits
// for its own copies with s_waitcnt vmcnt(n) and a bare s_barrier (the
// workgroup fence of __syncthreads would also wait for every copy in
// flight).  Inside the chunk loop no other vector memory operation may be
// issued, so that vmcnt counts exactly these copies.
#pragma once

#include <type_traits>

#include "kernels.h"

namespace cavs {

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // gfx9 s_waitcnt: vmcnt in bits [3:0] and [15:14]; expcnt, lgkmcnt at max
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// s_waitcnt vmcnt(N) lgkmcnt(0): this wavefront's older copies beyond the
// newest N have landed and its LDS reads have returned.
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
}

__device__ __forceinline__ void barrier_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// 16 bytes per lane from g into LDS at lds_addr + 16 * lane.
__device__ __forceinline__ void copy16_to_lds(const float* g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(g), "s"(lds_addr) : "memory", "m0");
}

// The same copy through the compiler's builtin, to LDS pointer `lds`
// (wavefront-uniform): the scheduler sees a vector-memory load it may place
// between MFMAs, where the inline-asm form stays where it is written.
__device__ __forceinline__ void copy16_to_lds_s(const float* g, float* lds) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

__device__ __forceinline__ uint32_t lds_addr_of(const float* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) float*)p;
}

// k = 8 gq .. 8 gq + 7 of LDS row `row` (quads swizzled by row & 7)
__device__ __forceinline__ void frag_sw(const float* L, int row, int gq, float (&v)[8]) {
  const float* rp = L + row * 32;
  const int sw = row & 7;
  const float4 x = *reinterpret_cast<const float4*>(rp + 4 * ((2 * gq) ^ sw));
  const float4 y = *reinterpret_cast<const float4*>(rp + 4 * ((2 * gq + 1) ^ sw));
  v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
}

template <int K>
using IC = std::integral_constant<int, K>;

// Stage ring: S distinct LDS arrays of ROWS x 32 floats, selected at compile
// time (the chunk loop is unrolled by S).
template <int ROWS, int S>
struct Ring {
  float* s0;
  float* s1;
  float* s2;
  float* s3;
  template <int K>
  __device__ __forceinline__ float* at(IC<K>) const {
    if constexpr (K == 0) return s0;
    else if constexpr (K == 1) return s1;
    else if constexpr (K == 2) return s2;
    else return s3;
  }
};

// Runs chunks 0 .. nch-1 through an S-stage ring: issue(stage, c) starts the
// IPW copies of chunk c, compute(stage ptr, c) consumes it.
template <int S, int IPW, class Issue, class Compute, class RingT>
__device__ __forceinline__ void ring_loop(int nch, const RingT& ring, Issue&& issue,
                                          Compute&& compute) {
  issue(IC<0>{}, 0);
  if constexpr (S > 2) if (1 < nch) issue(IC<1>{}, 1);
  if constexpr (S > 3) if (2 < nch) issue(IC<2>{}, 2);
  auto step = [&](auto sc, int c) {
    constexpr int k = decltype(sc)::value;
    if (c + S - 2 < nch) wait_vmcnt<(S - 2) * IPW>();
    else wait_vmcnt<0>();
    barrier_nofence();
    if (c + S - 1 < nch) issue(IC<(k + S - 1) % S>{}, c + S - 1);
    compute(ring.at(sc), c);
  };
  for (int c = 0; c < nch; c += S) {
    step(IC<0>{}, c);
    if (c + 1 < nch) step(IC<1>{}, c + 1);
    if constexpr (S > 2) if (c + 2 < nch) step(IC<2>{}, c + 2);
    if constexpr (S > 3) if (c + 3 < nch) step(IC<3>{}, c + 3);
  }
}

// The same ring with the MFMA fragments double-buffered in registers: while
// chunk c is multiplied from one register set, the LDS reads of chunk c+1
// fill the other, interleaved with the MFMAs (sched_group_barrier) so that
// they issue while the matrix core is busy.  One barrier per chunk covers
// both hazards: after it every wavefront holds chunk c's fragments (so the
// copies of chunk c+S may overwrite its stage) and chunk c+1 has landed.
//   issue(stage, c): the IPW copies of chunk c;
//   read0(stage ptr, F&): the LDS reads of chunk 0;
//   body(stage ptr of chunk c+1, F& cur, F& nxt, c): the LDS reads of chunk
//     c+1 into nxt and the MFMAs of chunk c from cur (past the last chunk the
//     reads see a stale stage: in bounds, never used).
//   ALWAYS: every step issues a chunk (past the last one it copies the last
//     chunk again, into a stage nothing reads any more), so the copies sit
//     in the same basic block as the MFMAs and can be interleaved with
//     them; the loop ends with every copy landed.  Two stages only: with
//     three or four the compiler's own wait insertion makes some steps wait
//     for the copy just issued before reading the other stage.
template <int S, int IPW, class F, bool ALWAYS = false, class Issue, class Read0, class Body,
          class RingT>
__device__ __forceinline__ void ring_loop_db(int nch, const RingT& ring, Issue&& issue,
                                             Read0&& read0, Body&& body) {
  static_assert(!ALWAYS || S == 2, "interleaved builtin copies need a two-stage ring");
  issue(IC<0>{}, 0);
  if (1 < nch) issue(IC<1>{}, 1);
  if constexpr (S > 2) if (2 < nch) issue(IC<2>{}, 2);
  if constexpr (S > 3) if (3 < nch) issue(IC<3>{}, 3);
  if (S - 1 < nch) wait_vmcnt<(S - 1) * IPW>();
  else wait_vmcnt<0>();
  barrier_nofence();
  F f0, f1;
  read0(ring.at(IC<0>{}), f0);
  auto step = [&](auto sc, F& cur, F& nxt, int c) {
    constexpr int k = decltype(sc)::value;
    if (c + S - 1 < nch) wait_vmcnt_lgkm0<(S - 2) * IPW>();
    else wait_vmcnt_lgkm0<0>();
    barrier_nofence();
    if constexpr (ALWAYS) issue(IC<k>{}, c + S < nch ? c + S : nch - 1);
    else if (c + S < nch) issue(IC<k>{}, c + S);
    body(ring.at(IC<(k + 1) % S>{}), cur, nxt, c);
  };
  for (int c = 0; c < nch; c += 2 * S) {
    step(IC<0>{}, f0, f1, c);
    if (c + 1 < nch) step(IC<1 % S>{}, f1, f0, c + 1);
    if (c + 2 < nch) step(IC<2 % S>{}, f0, f1, c + 2);
    if (c + 3 < nch) step(IC<3 % S>{}, f1, f0, c + 3);
    if constexpr (S > 2) {
      if (c + 4 < nch) step(IC<4 % S>{}, f0, f1, c + 4);
      if (c + 5 < nch) step(IC<5 % S>{}, f1, f0, c + 5);
    }
    if constexpr (S > 3) {
      if (c + 6 < nch) step(IC<6 % S>{}, f0, f1, c + 6);
      if (c + 7 < nch) step(IC<7 % S>{}, f1, f0, c + 7);
    }
  }
  if constexpr (ALWAYS) wait_vmcnt<0>();
}

// The IPW copies of one chunk into `stage` (this wavefront's rows start
// `wofs` floats in; copy t reads src(t)): through the builtin when they are
// to be interleaved with the MFMAs (ILV, see ring_loop_db's ALWAYS), else the
// inline-asm form, issued together ahead of them.
template <int IPW, bool ILV, class Src>
__device__ __forceinline__ void ring_issue(float* stage, int wofs, Src&& src) {
  if constexpr (ILV) {
    float* const base = stage + wofs;
#pragma unroll
    for (int t = 0; t < IPW; ++t) copy16_to_lds_s(src(t), base + 256 * t);
  } else {
    const uint32_t base = __builtin_amdgcn_readfirstlane(lds_addr_of(stage) + 4u * wofs);
#pragma unroll
    for (int t = 0; t < IPW; ++t) copy16_to_lds(src(t), base + 1024u * t);
  }
}

// sched_group_barrier sequence for one chunk: NR LDS reads spread evenly
// between NM MFMAs.
template <int NR, int NM>
__device__ __forceinline__ void interleave_reads() {
  constexpr int PER = NM / NR > 0 ? NM / NR : 1;
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one DS read
    __builtin_amdgcn_sched_group_barrier(0x008, PER, 0); // PER MFMAs
  }
  __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
}

// The same with the chunk's NV ring copies (vector-memory loads) spread
// over the first part of the MFMAs, ahead of the LDS reads.
template <int NV, int NR, int NM>
__device__ __forceinline__ void interleave_copies_reads() {
  constexpr int NI = NV > NR ? NV : NR;
  constexpr int PER = NM / NI > 0 ? NM / NI : 1;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    if (i < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // one copy
    if (i < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one DS read
    __builtin_amdgcn_sched_group_barrier(0x008, PER, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
}

// The schedule of one chunk's body to match ring_issue<IPW, ILV>.
template <bool ILV, int IPW, int NR, int NM>
__device__ __forceinline__ void ring_schedule() {
  if constexpr (ILV) interleave_copies_reads<IPW, NR, NM>();
  else interleave_reads<NR, NM>();
}

}  // namespace cavs
