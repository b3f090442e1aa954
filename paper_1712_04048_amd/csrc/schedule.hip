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
// Batches of at most kSmallV vertices run steps 1-4 and steps 5-6 as two
// one-workgroup launches instead (k_sched_small_levels, k_sched_small_sort).
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <type_traits>

#include "cavs_internal.h"

// Scratch of the allocation-free entry point cavs_schedule_static: one copy
// per GPU, alive until the process ends.  Host code never uses this name as
// an address: static_sched_scratch() takes each device's address of it once
// (hipGetSymbolAddress, with that device current) and everything else uses
// that pointer.
static __device__ __align__(256) unsigned char scratch[CAVS_SCHEDULE_STATIC_BYTES];

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
  F_FALLBACK = 12,   // the one-workgroup scheduler could not finish (more than kSmallT levels)
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
    int p = parent ? parent[v] : -1;
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
// 2'. levels of graph inputs (no parent array: a vertex may be read by
// several vertices) and of trees with more than two child slots, by peeling:
// a vertex is ready once every vertex it reads has its level.  The readers
// of each vertex are listed first (rd_off, from the reference counts, and
// rd_list); one workgroup then takes the ready vertices round by round: the
// round-t list gets level t, and each of its vertices counts itself off
// every reader's number of unfinished children (once per link); a reader
// whose count reaches zero goes into the next list.  The list lengths are
// the level histogram.  A vertex never reached lies on a cycle.
// -------------------------------------------------------------------------
__global__ void k_check_links(int V, int N, int n_x, const int* __restrict__ child,
                              const int* __restrict__ parent, const int* __restrict__ ref_cnt,
                              const int* __restrict__ pull_cnt, int* flags) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (parent) check_links_of(v, V, N, n_x, child, parent, ref_cnt, pull_cnt, flags);
  else if (v < n_x && pull_cnt[v] > 1) atomicOr(&flags[F_DUP], 1);
}

__global__ void k_graph_readers(int V, int N, const int* __restrict__ child,
                                const int* __restrict__ rd_off, int* rd_cur, int* rd_list) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= V) return;
  for (int k = 0; k < N; ++k) {
    const int c = child[(size_t)v * N + k];
    if (c >= 0 && c < V) rd_list[rd_off[c] + atomicAdd(&rd_cur[c], 1)] = v;
  }
}

__global__ void __launch_bounds__(1024) k_graph_levels(int V, const int* __restrict__ nchild,
                                                       const int* __restrict__ rd_off,
                                                       const int* __restrict__ rd_list,
                                                       int* nrem, int* listA, int* listB,
                                                       int* level, int* hist, int* flags) {
  __shared__ int cur_n, next_n, done_n;
  const int tid = threadIdx.x;
  if (tid == 0) {
    cur_n = 0;
    next_n = 0;
    done_n = 0;
  }
  __syncthreads();
  for (int v = tid; v < V; v += 1024) {
    const int c = nchild[v];
    nrem[v] = c;
    if (c == 0) listA[atomicAdd(&cur_n, 1)] = v;
  }
  __syncthreads();
  int* cur = listA;
  int* nxt = listB;
  int t = 0;
  while (cur_n > 0 && t < V) {
    const int n = cur_n;
    for (int i = tid; i < n; i += 1024) {
      const int v = cur[i];
      level[v] = t;
      for (int e = rd_off[v]; e < rd_off[v + 1]; ++e) {
        const int r = rd_list[e];
        if (atomicSub(&nrem[r], 1) == 1) nxt[atomicAdd(&next_n, 1)] = r;
      }
    }
    __syncthreads();
    if (tid == 0) {
      hist[t] = n;
      done_n += n;
      cur_n = next_n;
      next_n = 0;
    }
    int* sw = cur;
    cur = nxt;
    nxt = sw;
    ++t;
    __syncthreads();
  }
  if (tid == 0) {
    flags[F_T] = t;
    if (done_n != V) flags[F_CYCLE] = 1;
  }
}

// In-link lists by position (graph inputs): the links e = p * N + k whose
// child is position c, ascending, in in_edge[in_off[c] .. in_off[c+1]).
__global__ void k_in_count(int E, const int* __restrict__ child_pos, int* in_cnt) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e < E && child_pos[e] >= 0) atomicAdd(&in_cnt[child_pos[e]], 1);
}

__global__ void k_in_fill(int E, const int* __restrict__ child_pos,
                          const int* __restrict__ in_off, int* in_cur, int* in_edge) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int c = child_pos[e];
  if (c >= 0) in_edge[in_off[c] + atomicAdd(&in_cur[c], 1)] = e;
}

__global__ void k_in_sort(int V, const int* __restrict__ in_off, int* in_edge) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= V) return;
  const int a = in_off[c], b = in_off[c + 1];
  for (int i = a + 1; i < b; ++i) {   // insertion sort: lists are short
    const int x = in_edge[i];
    int j = i - 1;
    while (j >= a && in_edge[j] > x) {
      in_edge[j + 1] = in_edge[j];
      --j;
    }
    in_edge[j + 1] = x;
  }
}

__global__ void k_zero_ints(int* p, long n) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
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
  int q = parent ? parent[v] : -1;
  parent_pos[p] = (q >= 0 && q < V) ? pos[q] : -1;
  int r = pull_idx ? pull_idx[v] : -1;
  pull_pos[p] = r;
  push_pos[p] = push_idx ? push_idx[v] : -1;
}

// -------------------------------------------------------------------------
// Small batches: the same steps in two one-workgroup launches
// -------------------------------------------------------------------------
// With at most kSmallV vertices the parent links, the arrival counters and
// the level histogram fit in one workgroup's LDS, so steps 1-4 run as one
// launch without global atomics or kernel boundaries between them, and steps
// 5-6 as a second launch that the host does not wait for.  A batch with
// kSmallT levels or more sets F_FALLBACK and is scheduled again by the
// general path.
constexpr int kSmallV = 16384;
constexpr int kSmallNx = 1 << 18;   // input rows tracked by the LDS bitset
constexpr int kSmallT = 256;
constexpr int kSmallThreads = 1024;
constexpr int kSmallPer = kSmallV / kSmallThreads;
constexpr int kSmallWaves = kSmallThreads / kWave;

// Steps 1-4.  The stage (flags, then offsets) goes both to `stage` in device
// memory, for the sort kernel, and to `hstage`, the host's coherent mapped
// copy.  Vertex v belongs to thread v % 1024 for the validation.  The
// levels are then found level-synchronously instead of by walks: round t
// takes the list of level-t vertices, sets their level and counts each one
// off its parent's number of children not yet reached; a parent whose count
// drops to zero has all its children at levels <= t, one of them at t, so it
// is on level t + 1 and goes into the next list (compacted with a ballot and
// one LDS atomic per wavefront).  The list lengths are the level histogram.
// Every round is dense work for the whole workgroup, where leaf-to-root
// walks would leave most lanes of a wavefront idle.
__global__ void __launch_bounds__(kSmallThreads) k_sched_small_levels(
    int V, int N, int n_x, int n_push, const int* __restrict__ child,
    const int* __restrict__ parent, const int* __restrict__ pull_idx,
    const int* __restrict__ push_idx, int* __restrict__ level, int* __restrict__ level_offsets,
    int* __restrict__ stage, int* __restrict__ hstage) {
  __shared__ short par[kSmallV];              // parent, or -1, or -2 when out of range
  __shared__ unsigned nrem[kSmallV / 4];      // one byte per vertex: children not yet reached
  __shared__ int lists[kSmallV];              // two level lists of int16, or reference counts
  __shared__ unsigned pbits[kSmallNx / 32];   // input rows already pulled
  __shared__ int fcnt[kSmallT + 1];           // list lengths = the level histogram
  __shared__ int fl[F_COUNT];
  __shared__ int red[2];                      // rounds and vertices reached
  short* const fr0 = reinterpret_cast<short*>(lists);
  short* const fr1 = fr0 + kSmallV;
  unsigned char* const nrem8 = reinterpret_cast<unsigned char*>(nrem);
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const unsigned long long lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));

  // 1. parents into LDS, counters cleared.  The loads are unconditional
  // (indices clamped to V - 1; the copies past V are never used), so that
  // each array costs one memory latency.
  for (int i = tid; i < (n_x + 31) / 32; i += kSmallThreads) pbits[i] = 0;
  for (int i = tid; i <= kSmallT; i += kSmallThreads) fcnt[i] = 0;
  if (tid < F_COUNT) fl[tid] = 0;
  int bad = 0, withp = 0;
  {
    int pv[kSmallPer];
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) pv[i] = parent[min(tid + i * kSmallThreads, V - 1)];
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
      const int v = tid + i * kSmallThreads;
      if (v < V) {
        const int p = pv[i];
        const bool pb = p < -1 || p >= V;
        bad |= pb;
        withp += !pb && p >= 0;
        par[v] = (short)(pb ? -2 : p);
      }
    }
  }
  __syncthreads();

  // validation counters, the children counts and the leaves (the level-0 list)
  int links = 0, lab = 0, leafnoin = 0, innerin = 0, npull = 0, multi = 0, dup = 0, mism = 0;
  unsigned leafmask = 0;   // bit i: vertex tid + 1024 i is a leaf
  {
    int cs[kSmallPer][2];
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
      const size_t v = (size_t)min(tid + i * kSmallThreads, V - 1);
      cs[i][0] = child[v * N];
      cs[i][1] = N == 2 ? child[v * N + 1] : -1;
    }
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
      const int v = tid + i * kSmallThreads;
      if (i * kSmallThreads < V && v < V) {   // the first test skips whole trips
        int nc = 0;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const int c = cs[i][k];
          if (c < -1 || c >= V) {
            bad = 1;
          } else if (c >= 0) {
            mism |= (int)par[c] != v;
            ++nc;
          }
        }
        // the same child in both slots; a child listed by two different
        // vertices shows as a mismatch first (see below)
        multi |= cs[i][0] >= 0 && cs[i][0] < V && cs[i][0] == cs[i][1];
        nrem8[v] = (unsigned char)nc;
        if (!nc) leafmask |= 1u << i;
        links += nc;
      }
    }
  }
  if (pull_idx) {
    int rr[kSmallPer];
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) rr[i] = pull_idx[min(tid + i * kSmallThreads, V - 1)];
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
      if (i * kSmallThreads < V && tid + i * kSmallThreads < V) {
        int r = rr[i];
        if (r < -1 || r >= n_x) {
          bad = 1;
          r = -1;
        } else if (r >= 0) {
          ++npull;
          const unsigned bit = 1u << (r & 31);
          dup |= (atomicOr(&pbits[r >> 5], bit) & bit) != 0;
        }
        const bool leaf = (leafmask >> i) & 1u;
        leafnoin += leaf && r < 0;
        innerin += !leaf && r >= 0;
      }
    }
  } else {
    leafnoin = __popc(leafmask);
  }
  if (push_idx) {
    int qq[kSmallPer];
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) qq[i] = push_idx[min(tid + i * kSmallThreads, V - 1)];
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
      const int q = qq[i];
      if (i * kSmallThreads < V && tid + i * kSmallThreads < V) {
        if (q < -1 || q >= n_push) bad = 1;
        else if (q >= 0) ++lab;
      }
    }
  }
  {
    // this thread's leaves go to the level-0 list: one LDS atomic per wavefront
    const int nl = __popc(leafmask);
    int incl = nl;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int x = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += x;
    }
    int base = 0;
    if (lane == kWave - 1 && incl) base = atomicAdd(&fcnt[0], incl);
    base = __shfl(base, kWave - 1, kWave) + incl - nl;
    for (unsigned m = leafmask; m; m &= m - 1) fr0[base++] = (short)(tid + __builtin_ctz(m) * kSmallThreads);
  }
  // per-wavefront sums, two 16-bit counts to a word (a thread adds at most
  // 2 * kSmallPer to each), and the error flags as ballots
  auto add2 = [&](int idx_lo, int lo, int idx_hi, int hi) {
    const int x = wave_sum_int(lo | (hi << 16));
    if (lane == 0 && x) {
      atomicAdd(&fl[idx_lo], x & 0xFFFF);
      atomicAdd(&fl[idx_hi], x >> 16);
    }
  };
  auto flag = [&](int idx, int x) {
    if (__ballot(x != 0) && lane == 0) atomicOr(&fl[idx], 1);
  };
  add2(F_LINKS, links, F_WITHPARENT, withp);
  add2(F_LABELLED, lab, F_NPULL, npull);
  add2(F_LEAF_NOIN, leafnoin, F_INNER_IN, innerin);
  flag(F_RANGE, bad);
  flag(F_MULTI, multi);
  flag(F_DUP, dup);
  flag(F_MISMATCH, mism);
  __syncthreads();

  // A vertex listed as a child by two different vertices has a parent that
  // differs from at least one of them, so references are only counted
  // (to tell F_MULTI from F_MISMATCH) when a mismatch was seen.
  if (fl[F_MISMATCH]) {
    int* ref = lists;
    for (int i = tid; i < V; i += kSmallThreads) ref[i] = 0;
    __syncthreads();
    int mu = 0;
    for (int v = tid; v < V; v += kSmallThreads)
      for (int k = 0; k < N; ++k) {
        const int c = child[(size_t)v * N + k];
        if (c >= 0 && c < V) mu |= atomicAdd(&ref[c], 1) != 0;
      }
    flag(F_MULTI, mu);
    __syncthreads();
  }
  const bool err = (fl[F_RANGE] | fl[F_MULTI] | fl[F_DUP] | fl[F_MISMATCH]) != 0 ||
                   fl[F_LINKS] != fl[F_WITHPARENT];

  // 2-3. rounds (skipped on a graph that failed validation: the host reports
  // the error); at most kSmallT of them, more levels fall back
  // One round: the list of level T (size entries) in chunks of `stride`
  // lanes from lane `first`; the completed parents are appended to the next
  // list (LDS executes each wavefront's atomics in order, so a wavefront's
  // append is complete before its next round reads the count).
  auto round = [&](int T, int size, int first, int stride) {
    const short* cur = (T & 1) ? fr1 : fr0;
    short* nxt = (T & 1) ? fr0 : fr1;
    for (int k0 = 0; k0 < size; k0 += stride) {
      const int k = k0 + first;
      bool done = false;
      int p = -1;
      if (k < size && k < kSmallV) {
        const int v = cur[k];
        level[v] = T;
        p = par[v];
        if (p >= 0) {
          const unsigned sh = 8u * (p & 3);
          done = ((atomicSub(&nrem[p >> 2], 1u << sh) >> sh) & 255u) == 1u;
        }
      }
      const unsigned long long m = __ballot(done);
      int base = 0;
      if (lane == 0 && m) base = atomicAdd(&fcnt[T + 1], __popcll(m));
      base = __builtin_amdgcn_readfirstlane(base) + __popcll(m & lt);
      if (done && base < kSmallV) nxt[base] = (short)p;
    }
  };
  int T = 0, total = 0;
  bool deep = false;
  if (!err) {
    // whole-workgroup rounds while a list is longer than one wavefront ...
    for (; T < kSmallT; ++T) {
      const int size = fcnt[T];   // complete: written before the last barrier
      if (size <= kWave) break;
      total += size;
      round(T, size, tid, kSmallThreads);
      __syncthreads();
    }
    // ... then wavefront 0 alone, without barriers
    if (tid < kWave) {
      for (; T < kSmallT; ++T) {
        const int size = fcnt[T];
        if (size == 0) break;
        total += size;
        round(T, size, lane, kWave);
      }
      if (lane == 0) red[0] = T, red[1] = total;
    }
    __syncthreads();
    T = red[0];
    total = red[1];
    deep = T == kSmallT && fcnt[kSmallT] > 0;
  }

  // 4. flags, the offsets scan, and the host stage
  if (tid == 0) {
    fl[F_T] = deep ? kSmallT + 1 : T;
    if (!err && !deep && total < V) fl[F_CYCLE] = 1;   // some vertex was never reached
    if (deep) fl[F_FALLBACK] = 1;
  }
  __syncthreads();
  if (tid < kWave) {
    // exclusive scan of the list lengths into offsets 0..T, five entries per lane
    constexpr int E = (kSmallT + kWave) / kWave;
    int a[E], sum = 0;
#pragma unroll
    for (int j = 0; j < E; ++j) {
      const int idx = E * lane + j;
      a[j] = idx < T ? fcnt[idx] : 0;
      sum += a[j];
    }
    int incl = sum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int x = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += x;
    }
    int run = incl - sum;
#pragma unroll
    for (int j = 0; j < E; ++j) {
      const int idx = E * lane + j;
      if (idx <= T && idx <= V) {
        level_offsets[idx] = run;
        stage[kStageHead + idx] = run;
        hstage[kStageHead + idx] = run;
      }
      run += a[j];
    }
  } else if (tid < kWave + F_COUNT) {
    stage[tid - kWave] = fl[tid - kWave];
    hstage[tid - kWave] = fl[tid - kWave];
  }
}

// Steps 5-6.  Wavefront w ranks vertices [w S, w S + S) in id order, 64 at a
// time (chunk j = vertices w S + 64 j ..): the lanes with the same level find
// each other through a per-level lane mask in LDS, and a per-wavefront
// running count per level gives each its rank; the counts
// scanned over levels and wavefronts give the bases.  Pulling vertices are
// ranked the same way over the pulling lanes.  The ranking is cheap and every
// workgroup of the launch repeats it (so each holds all positions in LDS);
// workgroup g then writes the outputs of chunk g of every wavefront, which
// spreads the scattered stores over as many CUs as there are chunks.  Runs
// only if steps 1-4 found a valid graph with fewer than kSmallT levels (read
// from the stage on the device).
__device__ __forceinline__ int small_sort_span(int V) {
  return ((V + kSmallWaves - 1) / kSmallWaves + kWave - 1) / kWave * kWave;
}

__global__ void __launch_bounds__(kSmallThreads) k_sched_small_sort(
    int V, int N, const int* __restrict__ child, const int* __restrict__ parent,
    const int* __restrict__ pull_idx, const int* __restrict__ push_idx,
    const int* __restrict__ level, const int* __restrict__ stage, int* __restrict__ order,
    int* __restrict__ pos, int* __restrict__ child_pos, int* __restrict__ parent_pos,
    int* __restrict__ pull_pos, int* __restrict__ push_pos, int* __restrict__ pull_list) {
  __shared__ int cnt[2][kSmallWaves][kSmallT];   // all vertices, pulling vertices
  __shared__ int wsum[2][kSmallT / kWave];
  __shared__ int posl[kSmallV];
  __shared__ unsigned long long lanes[kSmallWaves][kSmallT];   // per level: lanes of a chunk
  const int* f = stage;
  const bool ok = !(f[F_RANGE] | f[F_MULTI] | f[F_DUP] | f[F_MISMATCH] | f[F_CYCLE] |
                    f[F_FALLBACK]) &&
                  f[F_LINKS] == f[F_WITHPARENT];
  if (!ok) return;   // the same for every thread
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & (kWave - 1), g = blockIdx.x;
  for (int i = tid; i < 2 * kSmallWaves * kSmallT; i += kSmallThreads) (&cnt[0][0][0])[i] = 0;
  for (int i = tid; i < kSmallWaves * kSmallT; i += kSmallThreads) (&lanes[0][0])[i] = 0;
  const int S = small_sort_span(V);
  const int nch = S / kWave, v0 = w * S;
  const unsigned long long lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  // the inputs of this workgroup's own chunk, loaded while it ranks
  const int vg = v0 + g * kWave + lane, vgc = min(vg, V - 1);
  const int a0 = child[(size_t)vgc * N], a1 = child[(size_t)vgc * N + N - 1];
  const int pa = parent[vgc];
  const int pl = pull_idx ? pull_idx[vgc] : -1, ps = push_idx ? push_idx[vgc] : -1;
  // unconditional loads (indices clamped to V - 1; copies past V are unused)
  int lv[kSmallPer], rk[kSmallPer];   // level; rank | pulling rank << 16
  unsigned pm = 0;                    // bit j: the vertex of chunk j pulls
#pragma unroll
  for (int j = 0; j < kSmallPer; ++j) lv[j] = level[min(v0 + j * kWave + lane, V - 1)];
  if (pull_idx) {
    int pr[kSmallPer];
#pragma unroll
    for (int j = 0; j < kSmallPer; ++j) pr[j] = pull_idx[min(v0 + j * kWave + lane, V - 1)];
#pragma unroll
    for (int j = 0; j < kSmallPer; ++j) pm |= (unsigned)(pr[j] >= 0) << j;
  }
  // the chunk inputs are needed here, so their loads are not moved past the
  // ranking to their conditional uses
  asm volatile("" ::"v"(a0), "v"(a1), "v"(pa), "v"(pl), "v"(ps));
  __syncthreads();
  // The lanes of a chunk with the same level: every lane ORs its bit into its
  // level's mask (this wavefront's row), reads the mask back, and the first
  // lane of each level clears it after the running counts are updated.  The
  // LDS executes one wavefront's instructions in order.
#pragma unroll
  for (int j = 0; j < kSmallPer; ++j) {
    if (j >= nch) continue;   // the same for the whole workgroup
    const bool valid = v0 + j * kWave + lane < V;
    const unsigned d = (unsigned)lv[j] & (kSmallT - 1);   // levels of a valid graph are below kSmallT
    if (valid) atomicOr(&lanes[w][d], 1ull << lane);
    const unsigned long long peers = valid ? lanes[w][d] : 0ull;
    const unsigned long long pp = peers & __ballot((pm >> j) & 1u);
    const int r0 = __popcll(peers & lt), p0 = __popcll(pp & lt);
    int a = 0, b = 0;
    if (valid) {
      a = cnt[0][w][d];
      b = cnt[1][w][d];
    }
    rk[j] = (a + r0) | ((b + p0) << 16);
    if (valid && r0 == 0) {   // one lane per level in this chunk
      cnt[0][w][d] = a + __popcll(peers);
      cnt[1][w][d] = b + __popcll(pp);
      lanes[w][d] = 0ull;
    }
  }
  __syncthreads();
  // bases: thread l < kSmallT owns level l
  int t0 = 0, t1 = 0, i0 = 0, i1 = 0;
  if (tid < kSmallT) {
#pragma unroll
    for (int q = 0; q < kSmallWaves; ++q) {
      t0 += cnt[0][q][tid];
      t1 += cnt[1][q][tid];
    }
    i0 = t0;
    i1 = t1;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int x = __shfl_up(i0, o, kWave), y = __shfl_up(i1, o, kWave);
      if (lane >= o) {
        i0 += x;
        i1 += y;
      }
    }
    if (lane == kWave - 1) {
      wsum[0][w] = i0;
      wsum[1][w] = i1;
    }
  }
  __syncthreads();
  if (tid < kSmallT) {
    int run0 = i0 - t0, run1 = i1 - t1;
    for (int q = 0; q < w; ++q) {
      run0 += wsum[0][q];
      run1 += wsum[1][q];
    }
#pragma unroll
    for (int q = 0; q < kSmallWaves; ++q) {
      const int c0 = cnt[0][q][tid], c1 = cnt[1][q][tid];
      cnt[0][q][tid] = run0;
      cnt[1][q][tid] = run1;
      run0 += c0;
      run1 += c1;
    }
  }
  __syncthreads();
  // every position into LDS; this workgroup's chunk keeps its own
  int myp = -1, mypp = -1;
#pragma unroll
  for (int j = 0; j < kSmallPer; ++j) {
    const int v = v0 + j * kWave + lane;
    if (j < nch && v < V) {
      const int d = lv[j] & (kSmallT - 1);
      const int dst = cnt[0][w][d] + (rk[j] & 0xFFFF);
      posl[v] = dst;
      if (j == g) {
        myp = dst;
        mypp = cnt[1][w][d] + (rk[j] >> 16);
      }
    }
  }
  __syncthreads();
  // 5-6. outputs of chunk g: order, pos, pull_list, and the remap
  if (vg >= V || (unsigned)myp >= (unsigned)V) return;   // the latter only if the graph was not valid
  order[myp] = vg;
  pos[vg] = myp;
  if (pl >= 0 && (unsigned)mypp < (unsigned)V) pull_list[mypp] = myp;
  child_pos[(size_t)myp * N] = a0 >= 0 && a0 < V ? posl[a0] : -1;
  if (N == 2) child_pos[(size_t)myp * N + 1] = a1 >= 0 && a1 < V ? posl[a1] : -1;
  parent_pos[myp] = pa >= 0 && pa < V ? posl[pa] : -1;
  pull_pos[myp] = pl;
  push_pos[myp] = ps;
}

// -------------------------------------------------------------------------
// 4. staging for the single device->host copy: done by the offsets scan
// -------------------------------------------------------------------------

struct Layout {
  size_t flags, ref_cnt, arrive, pull_cnt, hist, rd_cur, zero_end;
  size_t rd_off, rd_list, nrem, listA, listB, in_cnt;
  size_t nchild, keysA, valsA, keysB, valsB, tile_hist, stage, total;
  int ntiles;
};

Layout layout(int32_t V, int32_t N, int32_t n_x) {
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
  L.rd_cur = take((size_t)V + 1);
  L.zero_end = o;
  L.rd_off = take((size_t)V + 1);
  L.rd_list = take((size_t)V * N + 1);
  L.nrem = take((size_t)V + 1);
  L.listA = take((size_t)V + 1);
  L.listB = take((size_t)V + 1);
  L.in_cnt = take(2 * ((size_t)V + 1));   // counts, then fill cursors
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

// Waits for the stage by polling the event: the stage is a few hundred bytes
// that the host needs before it can enqueue the forward pass, and a blocking
// wait adds the scheduler's wake-up latency to every step.
hipError_t wait_stage(cavs_ctx* ctx) {
  hipError_t e;
  while ((e = hipEventQuery(ctx->stage_ready)) == hipErrorNotReady) {
  }
  return e;
}

// The validation result, T, the counts and the level offsets from the host
// stage; offsets past the first cap come from level_offsets on the device.
cavs_status read_stage(cavs_ctx* ctx, cavs_sched* s, int cap, const int* level_offsets,
                       bool dag = false) {
  const int* h = ctx->host_stage;
  if (h[F_RANGE]) return fail(ctx, CAVS_ERR_RANGE, "an index array holds an out-of-range value");
  if (h[F_MULTI]) return fail(ctx, CAVS_ERR_MULTIPARENT, "a vertex is a child more than once");
  if (h[F_DUP]) return fail(ctx, CAVS_ERR_DUP_PULL, "two vertices pull the same input row");
  if (!dag && (h[F_MISMATCH] || h[F_LINKS] != h[F_WITHPARENT]))
    return fail(ctx, CAVS_ERR_MISMATCH, "child[] and parent[] disagree");
  if (h[F_CYCLE]) return fail(ctx, CAVS_ERR_CYCLE, "the child links contain a cycle");
  const int T = h[F_T];
  s->T = T;
  s->n_pull = h[F_NPULL];
  s->n_labelled = h[F_LABELLED];
  s->n_leaf_noinput = h[F_LEAF_NOIN];
  s->n_inner_input = h[F_INNER_IN];
  const int n = T + 1 < cap ? T + 1 : cap;
  for (int i = 0; i < n; ++i) s->level_offsets_host[i] = h[kStageHead + i];
  if (T + 1 > cap) {
    if (!level_offsets) return fail(ctx, CAVS_ERR_HIP, "level offsets past the stage");
    CAVS_HIP_CHECK(ctx, hipMemcpyAsync(s->level_offsets_host + cap, level_offsets + cap,
                                       sizeof(int) * (size_t)(T + 1 - cap),
                                       hipMemcpyDeviceToHost, ctx->stream));
    CAVS_HIP_CHECK(ctx, hipStreamSynchronize(ctx->stream));
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
  const bool dag = g->parent == nullptr && V > 0;
  // graph inputs and more than two slots: levels by peeling (k_graph_levels)
  const bool peel = dag || N > 2;
  s->V = V;
  s->N = N;
  s->n_x = n_x;
  s->n_push = g->n_push;
  s->dag = dag ? 1 : 0;
  if (V == 0) {  // nothing to schedule: no launches, no device access
    s->T = 0;
    s->n_pull = s->n_labelled = s->n_leaf_noinput = s->n_inner_input = 0;
    s->level_offsets_host[0] = 0;
    return CAVS_OK;
  }

  if (!peel && V <= kSmallV && n_x <= kSmallNx) {
    CAVS_LAUNCH("k_sched_small_levels", k_sched_small_levels, dim3(1), dim3(kSmallThreads), 0, st,
                V, N, n_x, g->n_push, g->child, g->parent, g->pull_idx, g->push_idx, s->level,
                s->level_offsets, stage, ctx->host_stage_dev);
    CAVS_LAUNCH_CHECK(ctx);
    CAVS_HIP_CHECK(ctx, hipEventRecord(ctx->stage_ready, st));
    // enqueued before the host has seen the stage: it checks the flags itself
    const int chunks = cdiv(cdiv(V, kSmallWaves), kWave);
    CAVS_LAUNCH("k_sched_small_sort", k_sched_small_sort, dim3(chunks), dim3(kSmallThreads), 0, st, V,
                N, g->child, g->parent, g->pull_idx, g->push_idx, (const int*)s->level,
                (const int*)stage, s->order, s->pos, s->child_pos, s->parent_pos, s->pull_pos,
                s->push_pos, s->pull_list);
    CAVS_LAUNCH_CHECK(ctx);
    CAVS_HIP_CHECK(ctx, wait_stage(ctx));
    if (!ctx->host_stage[F_FALLBACK]) return read_stage(ctx, s, kSmallT + 1, nullptr);
  }

  const int nb = cdiv(V, 256);
  const long zero_ints = (long)(L.zero_end / sizeof(int));
  CAVS_LAUNCH("k_sched_init", k_sched_init, dim3(cdiv(zero_ints > V ? zero_ints : V, 256)),
              dim3(256), 0, st, (int*)base, zero_ints, s->level, V);
  CAVS_LAUNCH("k_scan_edges", k_scan_edges, dim3(nb), dim3(256), 0, st, V, N, n_x, g->n_push,
              g->child, g->parent, g->pull_idx, g->push_idx, ref_cnt, pull_cnt, nchild, flags);
  if (!peel) {
    CAVS_LAUNCH("k_links_levels", k_links_levels, dim3(cdiv(V > n_x ? V : n_x, 256)), dim3(256),
                0, st, V, N, n_x, g->child, g->parent, (const int*)ref_cnt,
                (const int*)pull_cnt, (const int*)nchild, arrive, s->level, flags);
    CAVS_LAUNCH("k_level_hist", k_level_hist, dim3(nb), dim3(256), 0, st, V, s->level, hist,
                flags);
  } else {
    int* rd_off = (int*)(base + L.rd_off);
    int* rd_list = (int*)(base + L.rd_list);
    CAVS_LAUNCH("k_check_links", k_check_links, dim3(cdiv(V > n_x ? V : n_x, 256)), dim3(256),
                0, st, V, N, n_x, g->child, g->parent, (const int*)ref_cnt, (const int*)pull_cnt,
                flags);
    CAVS_LAUNCH("k_scan_excl", k_scan_excl, dim3(1), dim3(1024), 0, st, (const int*)ref_cnt,
                rd_off, V + 1, (const int*)nullptr, (const int*)nullptr, 0, (int*)nullptr);
    CAVS_LAUNCH("k_graph_readers", k_graph_readers, dim3(nb), dim3(256), 0, st, V, N, g->child,
                (const int*)rd_off, (int*)(base + L.rd_cur), rd_list);
    CAVS_LAUNCH("k_graph_levels", k_graph_levels, dim3(1), dim3(1024), 0, st, V,
                (const int*)nchild, (const int*)rd_off, (const int*)rd_list,
                (int*)(base + L.nrem), (int*)(base + L.listA), (int*)(base + L.listB), s->level,
                hist, flags);
  }
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
    if (dag) {   // the links reading each position, for the backward's sums
      int* in_cnt = (int*)(base + L.in_cnt);
      int* in_cur = in_cnt + V + 1;
      const int E = V * N;
      CAVS_LAUNCH("k_zero_ints", k_zero_ints, dim3(cdiv(2L * (V + 1), 256)), dim3(256), 0, st,
                  in_cnt, 2L * (V + 1));
      CAVS_LAUNCH("k_in_count", k_in_count, dim3(cdiv(E, 256)), dim3(256), 0, st, E,
                  (const int*)s->child_pos, in_cnt);
      CAVS_LAUNCH("k_scan_excl", k_scan_excl, dim3(1), dim3(1024), 0, st, (const int*)in_cnt,
                  s->in_offsets, V + 1, (const int*)nullptr, (const int*)nullptr, 0,
                  (int*)nullptr);
      CAVS_LAUNCH("k_in_fill", k_in_fill, dim3(cdiv(E, 256)), dim3(256), 0, st, E,
                  (const int*)s->child_pos, (const int*)s->in_offsets, in_cur, s->in_edges);
      CAVS_LAUNCH("k_in_sort", k_in_sort, dim3(nb), dim3(256), 0, st, V,
                  (const int*)s->in_offsets, s->in_edges);
    }
    CAVS_LAUNCH_CHECK(ctx);
    return CAVS_OK;
  };
  cavs_status r = sort_and_remap(1);
  if (r != CAVS_OK) return r;
  CAVS_HIP_CHECK(ctx, wait_stage(ctx));
  r = read_stage(ctx, s, cap, s->level_offsets, dag);
  if (r != CAVS_OK) return r;
  // levels lie in [0, T): enough 8-bit digits for T - 1
  const int T = s->T;
  int passes = 1;
  while (passes < 4 && ((long)(T > 0 ? T - 1 : 0) >> (8 * passes)) > 0) ++passes;
  return passes > 1 ? sort_and_remap(passes) : CAVS_OK;
}

// Device address of `scratch` on the current device (`device`), taken once
// per device and kept for every later context on it.
cavs_status static_sched_scratch(cavs_ctx* ctx, int device, void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return CAVS_OK;   // the static entry point refuses
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(ctx, CAVS_ERR_HIP, "hipGetSymbolAddress(scratch) failed: %s",
                  hipGetErrorString(e));
    addr[device] = p;
  }
  *out = addr[device];
  return CAVS_OK;
}

}  // namespace cavs
