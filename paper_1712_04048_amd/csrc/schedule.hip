// GPU scheduler: the batching tasks V_t of Algorithm 1 (Section 3.2) and the
// level-major "dynamic tensor" layout of Section 3.3 / Algorithm 2.
//
// A vertex is activated once all of its children are evaluated, so the task
// that evaluates v is its level: 0 for a leaf, else 1 + the largest level of
// its children.  The schedule is built on the GPU:
//   1. validation counters (range, references per vertex, pull rows, links);
//   2. level assignment: one thread per leaf walks towards the root; at each
//      parent it bumps an arrival counter and only the last child to arrive
//      continues, so every vertex is assigned exactly once, in O(V) total;
//   3. per-level histogram and exclusive scan -> level_offsets;
//   4. one device->host copy of T, the counts, the error flags and the
//      offsets, and the only stream synchronisation: everything the host
//      needs is known at this point, and T fixes the number of sort passes;
//   5. stable LSD radix sort of vertex ids by level (8-bit digits, ranks from
//      wavefront ballots), giving ascending ids inside each task; its last
//      pass also writes pos and the list of positions that pull an input
//      (their ranks counted the same way over the pulling subset);
//   6. index remap to positions.
// Steps 5 and 6 are only enqueued: later calls on the stream see them done.
#include <stdarg.h>
#include <stdio.h>

#include "cavs_internal.h"

namespace cavs {

namespace {

enum Flag {
  F_RANGE = 0,
  F_MULTI = 1,
  F_DUP = 2,
  F_MISMATCH = 3,
  F_CYCLE = 4,
  F_T = 5,
  F_LINKS = 6,
  F_WITHPARENT = 7,
  F_LABELLED = 8,
  F_LEAF_NOIN = 9,
  F_INNER_IN = 10,
  F_NPULL = 11,
  F_COUNT = 32
};

constexpr int kTile = 1024;      // radix tile: 256 threads x 4 rounds
constexpr int kStageHead = 32;   // stage = flags[32] then offsets

__device__ __forceinline__ int ld_acquire_int(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_relaxed_int(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// -------------------------------------------------------------------------
// 1. validation counters
// -------------------------------------------------------------------------
__global__ void k_scan_edges(int V, int N, int n_x, int n_push, const int* __restrict__ child,
                             const int* __restrict__ parent, const int* __restrict__ pull_idx,
                             const int* __restrict__ push_idx, int* ref_cnt, int* pull_cnt,
                             int* nchild, int* flags) {
  int v = blockIdx.x * blockDim.x + threadIdx.x;
  int links = 0, withp = 0, lab = 0, leafnoin = 0, innerin = 0, npull = 0, bad = 0;
  if (v < V) {
    int nc = 0;
    for (int k = 0; k < N; ++k) {
      int c = child[(size_t)v * N + k];
      if (c < -1 || c >= V) {
        bad = 1;
      } else if (c >= 0) {
        atomicAdd(&ref_cnt[c], 1);
        ++nc;
      }
    }
    int p = parent[v];
    if (p < -1 || p >= V) bad = 1;
    else if (p >= 0) withp = 1;
    int r = pull_idx ? pull_idx[v] : -1;
    if (r < -1 || r >= n_x) {
      bad = 1;
      r = -1;
    } else if (r >= 0) {
      atomicAdd(&pull_cnt[r], 1);
      npull = 1;
    }
    int q = push_idx ? push_idx[v] : -1;
    if (q < -1 || q >= n_push) bad = 1;
    else if (q >= 0) lab = 1;
    nchild[v] = nc;
    links = nc;
    leafnoin = (nc == 0 && r < 0);
    innerin = (nc > 0 && r >= 0);
  }
  // counts summed per wavefront, then per workgroup in LDS: one atomic per
  // workgroup and counter (the counters are few, contended addresses)
  __shared__ int part[7][4];
  int cnt[7] = {links, withp, lab, leafnoin, innerin, npull, bad};
  const int w = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < 7; ++i) {
    cnt[i] = wave_sum_int(cnt[i]);
    if (lane_id() == 0) part[i][w] = cnt[i];
  }
  __syncthreads();
  if (threadIdx.x < 7) {
    const int i = threadIdx.x;
    const int t = part[i][0] + part[i][1] + part[i][2] + part[i][3];
    constexpr int dst[7] = {F_LINKS, F_WITHPARENT, F_LABELLED, F_LEAF_NOIN, F_INNER_IN, F_NPULL,
                            F_RANGE};
    if (t) {
      if (i == 6) atomicOr(&flags[F_RANGE], 1);
      else atomicAdd(&flags[dst[i]], t);
    }
  }
}

__device__ __forceinline__ void check_links_of(int v, int V, int N, int n_x,
                                               const int* __restrict__ child,
                                               const int* __restrict__ parent,
                                               const int* __restrict__ ref_cnt,
                                               const int* __restrict__ pull_cnt, int* flags) {
  if (v < V) {
    if (ref_cnt[v] > 1) atomicOr(&flags[F_MULTI], 1);
    for (int k = 0; k < N; ++k) {
      int c = child[(size_t)v * N + k];
      if (c >= 0 && c < V && parent[c] != v) atomicOr(&flags[F_MISMATCH], 1);
    }
  }
  if (v < n_x && pull_cnt[v] > 1) atomicOr(&flags[F_DUP], 1);
}

// -------------------------------------------------------------------------
// 2. levels: leaf-to-root walks with arrival counters
// -------------------------------------------------------------------------
// arrive[p] packs the number of children that have arrived at p (low 32
// bits) with the sum of their levels (high 32 bits).  With at most two child
// slots, the child that arrives second reads the first one's level from the
// value its own atomic returns, so the walk needs no other communication
// (and no memory fences).  The count never wraps, so only the arrival that
// completes p continues: each vertex is passed by at most one walker.
// The same launch runs the link checks of step 1 (like the walk, they only
// read the counters of k_scan_edges).
__global__ void k_links_levels(int V, int N, int n_x, const int* __restrict__ child,
                               const int* __restrict__ parent, const int* __restrict__ ref_cnt,
                               const int* __restrict__ pull_cnt, const int* __restrict__ nchild,
                               unsigned long long* arrive, int* level, int* flags) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  check_links_of(v, V, N, n_x, child, parent, ref_cnt, pull_cnt, flags);
  if (v >= V || nchild[v] != 0) return;
  level[v] = 0;
  int cur = v, lev = 0;
  for (int step = 0; step < V; ++step) {
    const int p = parent[cur];
    if (p < 0 || p >= V) break;
    const unsigned long long old =
        atomicAdd(&arrive[p], 1ull | ((unsigned long long)(unsigned)lev << 32));
    const unsigned cnt = (unsigned)(old & 0xFFFFFFFFull);
    if ((int)cnt + 1 != nchild[p]) break;
    if (cnt == 1) lev = max(lev, (int)(old >> 32));   // the other child's level
    lev += 1;
    level[p] = lev;
    cur = p;
  }
}

// Clears the counters of steps 1-3 and marks every level unassigned (-1),
// in one launch.
__global__ void k_sched_init(int* zero_base, long zero_ints, int* level, int V) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < zero_ints) zero_base[i] = 0;
  if (i < V) level[i] = -1;
}

// -------------------------------------------------------------------------
// 3. per-level histogram, T, cycle detection, and the offsets scan
// -------------------------------------------------------------------------
constexpr int kHistLds = 256;   // levels below this are counted in LDS first

__global__ void __launch_bounds__(256) k_level_hist(int V, const int* __restrict__ level,
                                                    int* hist, int* flags) {
  __shared__ int h[kHistLds];
  h[threadIdx.x] = 0;
  __syncthreads();
  int v = blockIdx.x * blockDim.x + threadIdx.x;
  int tmax = 0, cyc = 0;
  if (v < V) {
    int l = level[v];
    if (l < 0 || l >= V) {
      cyc = 1;
    } else {
      if (l < kHistLds) atomicAdd(&h[l], 1);
      else atomicAdd(&hist[l], 1);
      tmax = l + 1;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) tmax = max(tmax, __shfl_xor(tmax, o, kWave));
  cyc = wave_sum_int(cyc);
  if (lane_id() == 0) {
    if (tmax) atomicMax(&flags[F_T], tmax);
    if (cyc) atomicOr(&flags[F_CYCLE], 1);
  }
  __syncthreads();
  if (h[threadIdx.x]) atomicAdd(&hist[threadIdx.x], h[threadIdx.x]);
}

// Single-block exclusive scan of n ints (src may equal dst).  If n_dev is
// non-null the element count is *n_dev + 1 (scan of hist[0..T]).  With
// stage set, the block then fills the host staging area: the flags and
// the first cap scanned values (the level offsets).
__global__ void __launch_bounds__(1024) k_scan_excl(const int* src, int* dst, int n,
                                                    const int* n_dev, const int* flags, int cap,
                                                    int* stage) {
  __shared__ int wsum[16];
  __shared__ int carry_s;
  if (n_dev) n = *n_dev + 1;
  int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (tid == 0) carry_s = 0;
  __syncthreads();
  for (int base = 0; base < n; base += 1024) {
    int i = base + tid;
    int x = i < n ? src[i] : 0;
    int incl = x;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int t = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += t;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    if (w == 0) {
      int s = lane < 16 ? wsum[lane] : 0;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        int t = __shfl_up(s, o, kWave);
        if (lane >= o) s += t;
      }
      if (lane < 16) wsum[lane] = s;  // inclusive over waves
    }
    __syncthreads();
    int carry = carry_s;
    int wave_off = w > 0 ? wsum[w - 1] : 0;
    if (i < n) dst[i] = carry + wave_off + incl - x;
    __syncthreads();
    if (tid == 0) carry_s = carry + wsum[15];
    __syncthreads();
  }
  if (stage) {
    const int m = min(n, cap);
    for (int i = tid; i < kStageHead; i += 1024) stage[i] = flags[i];
    for (int i = tid; i < m; i += 1024) stage[kStageHead + i] = dst[i];
  }
}

// -------------------------------------------------------------------------
// 5. stable LSD radix sort, 8-bit digits
// -------------------------------------------------------------------------
__device__ __forceinline__ unsigned digit_of(int key, int shift) {
  return ((unsigned)key >> shift) & 255u;
}

// tile_hist is digit-major: entry [d * ntiles + tile].  With pull_idx set
// (last pass) the counts of elements whose vertex pulls an input follow at
// [(256 + d) * ntiles + tile]; vals_in == nullptr means value = index.
__global__ void __launch_bounds__(256) k_radix_hist(const int* __restrict__ keys,
                                                    const int* __restrict__ vals_in, int n,
                                                    int shift, int ntiles,
                                                    const int* __restrict__ pull_idx,
                                                    int* tile_hist) {
  __shared__ int h[2][256];
  int tid = threadIdx.x;
  h[0][tid] = 0;
  h[1][tid] = 0;
  __syncthreads();
  int base = blockIdx.x * kTile;
#pragma unroll
  for (int r = 0; r < kTile / 256; ++r) {
    int e = base + r * 256 + tid;
    if (e < n) {
      const unsigned d = digit_of(keys[e], shift);
      atomicAdd(&h[0][d], 1);
      if (pull_idx) {
        const int v = vals_in ? vals_in[e] : e;
        if (pull_idx[v] >= 0) atomicAdd(&h[1][d], 1);
      }
    }
  }
  __syncthreads();
  tile_hist[tid * ntiles + blockIdx.x] = h[0][tid];
  if (pull_idx) tile_hist[(256 + tid) * ntiles + blockIdx.x] = h[1][tid];
}

// vals_in == nullptr means the identity (value = element index).  In the
// last pass (pos_out set) every value v also gets pos_out[v] = dst, and with
// pull_idx set the values that pull an input are listed in order: their
// rank among the pulling elements of the same digit comes from the same
// ballots restricted to the pulling lanes, and offs[(256 + d) * ntiles +
// tile] - n counts the pulling elements before them (the scan ran over both
// tables, and the first one sums to n).
__global__ void __launch_bounds__(256) k_radix_scatter(const int* __restrict__ keys_in,
                                                       const int* __restrict__ vals_in, int n,
                                                       int shift, int ntiles,
                                                       const int* __restrict__ offs,
                                                       int* __restrict__ keys_out,
                                                       int* __restrict__ vals_out,
                                                       int* __restrict__ pos_out,
                                                       const int* __restrict__ pull_idx,
                                                       int* __restrict__ pull_list) {
  __shared__ int base_cnt[2][256];
  __shared__ int wcnt[2][4][256];
  int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  base_cnt[0][tid] = 0;
  base_cnt[1][tid] = 0;
  const unsigned long long lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int tile = blockIdx.x;
  for (int r = 0; r < kTile / 256; ++r) {
    int e = tile * kTile + r * 256 + tid;
    bool valid = e < n;
    int key = valid ? keys_in[e] : 0;
    int val = valid ? (vals_in ? vals_in[e] : e) : 0;
    const bool pulls = valid && pull_idx && pull_idx[val] >= 0;
    unsigned d = digit_of(key, shift);
    unsigned long long peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      bool bit = (d >> b) & 1u;
      unsigned long long bb = __ballot(valid && bit);
      peers &= bit ? bb : ~bb;
    }
    const unsigned long long ppeers = peers & __ballot(pulls);
    const int rank_in_wave = __popcll(peers & lt_mask);
    const int wave_cnt = __popcll(peers);
    const int prank_in_wave = __popcll(ppeers & lt_mask);
    const int pwave_cnt = __popcll(ppeers);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      wcnt[0][q][tid] = 0;
      wcnt[1][q][tid] = 0;
    }
    __syncthreads();
    if (valid && rank_in_wave == 0) {
      wcnt[0][w][d] = wave_cnt;
      wcnt[1][w][d] = pwave_cnt;
    }
    __syncthreads();
    if (valid) {
      int rank = base_cnt[0][d] + rank_in_wave;
      for (int q = 0; q < w; ++q) rank += wcnt[0][q][d];
      const int dst = offs[d * ntiles + tile] + rank;
      keys_out[dst] = key;
      vals_out[dst] = val;
      if (pos_out) pos_out[val] = dst;
      if (pulls) {
        int prank = base_cnt[1][d] + prank_in_wave;
        for (int q = 0; q < w; ++q) prank += wcnt[1][q][d];
        pull_list[offs[(256 + d) * ntiles + tile] - n + prank] = dst;
      }
    }
    __syncthreads();
    base_cnt[0][tid] += wcnt[0][0][tid] + wcnt[0][1][tid] + wcnt[0][2][tid] + wcnt[0][3][tid];
    base_cnt[1][tid] += wcnt[1][0][tid] + wcnt[1][1][tid] + wcnt[1][2][tid] + wcnt[1][3][tid];
    __syncthreads();
  }
}

// -------------------------------------------------------------------------
// 6. remap to positions
// -------------------------------------------------------------------------
__global__ void k_remap(int V, int N, const int* __restrict__ order, const int* __restrict__ pos,
                        const int* __restrict__ child, const int* __restrict__ parent,
                        const int* __restrict__ pull_idx, const int* __restrict__ push_idx,
                        int* child_pos, int* parent_pos, int* pull_pos, int* push_pos) {
  int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= V) return;
  int v = order[p];
  if (v < 0 || v >= V) v = 0;
  for (int k = 0; k < N; ++k) {
    int c = child[(size_t)v * N + k];
    child_pos[(size_t)p * N + k] = (c >= 0 && c < V) ? pos[c] : -1;
  }
  int q = parent[v];
  parent_pos[p] = (q >= 0 && q < V) ? pos[q] : -1;
  int r = pull_idx ? pull_idx[v] : -1;
  pull_pos[p] = r;
  push_pos[p] = push_idx ? push_idx[v] : -1;
}

// -------------------------------------------------------------------------
// 4. staging for the single device->host copy: done by the offsets scan
// -------------------------------------------------------------------------

struct Layout {
  size_t flags, ref_cnt, arrive, pull_cnt, hist, zero_end;
  size_t nchild, keysA, valsA, keysB, valsB, tile_hist, stage, total;
  int ntiles;
};

Layout layout(int32_t V, int32_t N, int32_t n_x) {
  (void)N;
  Layout L;
  size_t o = 0;
  auto take = [&](size_t ints) {
    size_t r = o;
    o = align_up(o + ints * sizeof(int), 256);
    return r;
  };
  L.ntiles = cdiv(V > 0 ? V : 1, kTile);
  L.flags = take(F_COUNT);
  L.ref_cnt = take((size_t)V + 1);
  L.arrive = take(2 * ((size_t)V + 1));   // 64-bit words
  L.pull_cnt = take((size_t)n_x + 1);
  L.hist = take((size_t)(V + 2 > 256 ? V + 2 : 256));
  L.zero_end = o;
  L.nchild = take((size_t)V + 1);
  L.keysA = take((size_t)V + 1);
  L.valsA = take((size_t)V + 1);
  L.keysB = take((size_t)V + 1);
  L.valsB = take((size_t)V + 1);
  L.tile_hist = take((size_t)512 * L.ntiles);   // digit counts, then pulling counts
  L.stage = take(kHostStageInts);
  L.total = o;
  return L;
}

// Sorts (keys_in, vals_in) by key.  Pass p writes keys to bufK[p % 2] and
// values to bufV[p % 2], except that the last pass writes its values to
// vals_final, pos_final[value] = its position and, for the values whose
// vertex pulls an input, their positions to pull_list in order.  keys_in
// must not alias bufK[0].
cavs_status radix_sort(cavs_ctx* ctx, const int* keys_in, const int* vals_in, int n, int passes,
                       int* const bufK[2], int* const bufV[2], int* vals_final, int* pos_final,
                       const int* pull_idx, int* pull_list, int* tile_hist, int ntiles) {
  const int* ki = keys_in;
  const int* vi = vals_in;
  for (int pass = 0; pass < passes; ++pass) {
    const bool last = pass == passes - 1;
    int* ko = bufK[pass % 2];
    int* vo = last ? vals_final : bufV[pass % 2];
    const int* pl = last ? pull_idx : nullptr;
    const int shift = 8 * pass;
    CAVS_LAUNCH("k_radix_hist", k_radix_hist, dim3(ntiles), dim3(256), 0, ctx->stream, ki, vi, n,
                shift, ntiles, pl, tile_hist);
    CAVS_LAUNCH("k_scan_excl", k_scan_excl, dim3(1), dim3(1024), 0, ctx->stream, tile_hist,
                tile_hist, (pl ? 512 : 256) * ntiles, (const int*)nullptr, (const int*)nullptr, 0,
                (int*)nullptr);
    CAVS_LAUNCH("k_radix_scatter", k_radix_scatter, dim3(ntiles), dim3(256), 0, ctx->stream, ki,
                vi, n, shift, ntiles, (const int*)tile_hist, ko, vo, last ? pos_final : nullptr, pl,
                last ? pull_list : nullptr);
    CAVS_LAUNCH_CHECK(ctx);
    ki = ko;
    vi = vo;
  }
  return CAVS_OK;
}

}  // namespace

size_t schedule_ws_bytes(int32_t V, int32_t N, int32_t n_x) {
  if (V < 0 || N < 1 || n_x < 0) return 0;
  return layout(V, N, n_x).total;
}

cavs_status schedule_run(cavs_ctx* ctx, const cavs_graphs* g, cavs_sched* s, void* ws,
                         size_t ws_bytes) {
  const int V = g->V, N = g->N, n_x = g->n_x;
  Layout L = layout(V, N, n_x);
  if (ws_bytes < L.total)
    return fail(ctx, CAVS_ERR_WORKSPACE, "schedule workspace too small: %zu < %zu", ws_bytes,
                L.total);
  char* base = (char*)ws;
  int* flags = (int*)(base + L.flags);
  int* ref_cnt = (int*)(base + L.ref_cnt);
  unsigned long long* arrive = (unsigned long long*)(base + L.arrive);
  int* pull_cnt = (int*)(base + L.pull_cnt);
  int* hist = (int*)(base + L.hist);
  int* nchild = (int*)(base + L.nchild);
  int* kA = (int*)(base + L.keysA);
  int* vA = (int*)(base + L.valsA);
  int* kB = (int*)(base + L.keysB);
  int* vB = (int*)(base + L.valsB);
  int* tile_hist = (int*)(base + L.tile_hist);
  int* stage = (int*)(base + L.stage);
  hipStream_t st = ctx->stream;
  s->V = V;
  s->N = N;
  s->n_x = n_x;
  s->n_push = g->n_push;
  if (V == 0) {  // nothing to schedule: no launches, no device access
    s->T = 0;
    s->n_pull = s->n_labelled = s->n_leaf_noinput = s->n_inner_input = 0;
    s->level_offsets_host[0] = 0;
    return CAVS_OK;
  }

  const int nb = cdiv(V, 256);
  const long zero_ints = (long)(L.zero_end / sizeof(int));
  CAVS_LAUNCH("k_sched_init", k_sched_init, dim3(cdiv(zero_ints > V ? zero_ints : V, 256)),
              dim3(256), 0, st, (int*)base, zero_ints, s->level, V);
  CAVS_LAUNCH("k_scan_edges", k_scan_edges, dim3(nb), dim3(256), 0, st, V, N, n_x, g->n_push,
              g->child, g->parent, g->pull_idx, g->push_idx, ref_cnt, pull_cnt, nchild, flags);
  CAVS_LAUNCH("k_links_levels", k_links_levels, dim3(cdiv(V > n_x ? V : n_x, 256)), dim3(256), 0,
              st, V, N, n_x, g->child, g->parent, (const int*)ref_cnt, (const int*)pull_cnt,
              (const int*)nchild, arrive, s->level, flags);
  CAVS_LAUNCH("k_level_hist", k_level_hist, dim3(nb), dim3(256), 0, st, V, s->level, hist, flags);
  const int cap = kHostStageInts - kStageHead;
  CAVS_LAUNCH("k_scan_excl", k_scan_excl, dim3(1), dim3(1024), 0, st, hist, s->level_offsets, 0,
              (const int*)(flags + F_T), (const int*)flags, cap, stage);
  CAVS_LAUNCH_CHECK(ctx);
  CAVS_HIP_CHECK(ctx, hipMemcpyAsync(ctx->host_stage, stage, sizeof(int) * kHostStageInts,
                                     hipMemcpyDeviceToHost, st));
  CAVS_HIP_CHECK(ctx, hipEventRecord(ctx->stage_ready, st));
  // While the host waits for the stage, the device already sorts assuming
  // fewer than 256 levels (one radix pass) and remaps; with more levels the
  // sort and remap run again below and overwrite these results.  On a graph
  // that fails validation they write only schedule outputs.
  int* const lvK[2] = {kA, kB};
  int* const lvV[2] = {vA, vB};
  auto sort_and_remap = [&](int passes) {
    cavs_status r = radix_sort(ctx, s->level, nullptr, V, passes, lvK, lvV, s->order, s->pos,
                               g->pull_idx, s->pull_list, tile_hist, L.ntiles);
    if (r != CAVS_OK) return r;
    CAVS_LAUNCH("k_remap", k_remap, dim3(nb), dim3(256), 0, st, V, N, (const int*)s->order,
                (const int*)s->pos, g->child, g->parent, g->pull_idx, g->push_idx, s->child_pos,
                s->parent_pos, s->pull_pos, s->push_pos);
    CAVS_LAUNCH_CHECK(ctx);
    return CAVS_OK;
  };
  cavs_status r = sort_and_remap(1);
  if (r != CAVS_OK) return r;
  CAVS_HIP_CHECK(ctx, hipEventSynchronize(ctx->stage_ready));
  const int* h = ctx->host_stage;
  if (h[F_RANGE]) return fail(ctx, CAVS_ERR_RANGE, "an index array holds an out-of-range value");
  if (h[F_MULTI]) return fail(ctx, CAVS_ERR_MULTIPARENT, "a vertex is a child more than once");
  if (h[F_DUP]) return fail(ctx, CAVS_ERR_DUP_PULL, "two vertices pull the same input row");
  if (h[F_MISMATCH] || h[F_LINKS] != h[F_WITHPARENT])
    return fail(ctx, CAVS_ERR_MISMATCH, "child[] and parent[] disagree");
  if (h[F_CYCLE]) return fail(ctx, CAVS_ERR_CYCLE, "the child links contain a cycle");
  const int T = h[F_T];
  s->T = T;
  s->n_pull = h[F_NPULL];
  s->n_labelled = h[F_LABELLED];
  s->n_leaf_noinput = h[F_LEAF_NOIN];
  s->n_inner_input = h[F_INNER_IN];
  int n = T + 1 < cap ? T + 1 : cap;
  for (int i = 0; i < n; ++i) s->level_offsets_host[i] = h[kStageHead + i];
  if (T + 1 > cap) {
    CAVS_HIP_CHECK(ctx, hipMemcpyAsync(s->level_offsets_host + cap, s->level_offsets + cap,
                                       sizeof(int) * (size_t)(T + 1 - cap),
                                       hipMemcpyDeviceToHost, st));
    CAVS_HIP_CHECK(ctx, hipStreamSynchronize(st));
  }
  // levels lie in [0, T): enough 8-bit digits for T - 1
  int passes = 1;
  while (passes < 4 && ((long)(T > 0 ? T - 1 : 0) >> (8 * passes)) > 0) ++passes;
  return passes > 1 ? sort_and_remap(passes) : CAVS_OK;
}

}  // namespace cavs
