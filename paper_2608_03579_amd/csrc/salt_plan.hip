// The device segment plan of libsalt (Sec. 3.3: the frontend groups requests by
// their centroid).  Tokens are ordered by the key (centroid id, residual slot,
// token index), ascending, with -1 ids first; the token index makes every key
// unique, so the order, the segments (runs of equal (centroid, slot)) and the
// groups (runs of equal centroid) are unique and bit-exact.
//
//   k_plan_sort:   one block per chunk of kSortChunk tokens sorts its keys
//                  (bitonic network: in-wave steps on registers, the others in
//                  LDS).  A batch of one chunk is finished in the
//                  same block; larger batches write their sorted chunks.
//   k_plan_merge:  (more than one chunk) a key's place is its place in its own
//                  chunk plus, for every other chunk, the number of keys below
//                  it there (binary search).
//   k_plan_finish: (more than one chunk) one block derives the segments and
//                  groups from the sorted keys.
// The tiles the apply kernels read come from the host, which counts the tokens
// of every centroid when it stages the maps; the finish checks them against the
// sorted order and counts any mismatch in the plan's meta words.
// Every index written is a place in [0, T): a rank below T by construction,
// clamped as well.
#include "salt_internal.h"
#include "salt_layout.h"

namespace salt {
namespace {

constexpr int kPlanThreads = 1024;
constexpr uint64_t kPad = ~0ull;
constexpr uint64_t kTokMask = (1ull << 21) - 1;

// (c + 1) << 42 | (u + 1) << 21 | t: c + 1 <= 64, u + 1 <= 2^20, t < 2^16.
__device__ __forceinline__ uint64_t plan_key(int c, int u, int t) {
  return ((uint64_t)(uint32_t)(c + 1) << 42) | ((uint64_t)(uint32_t)(u + 1) << 21) | (uint64_t)(uint32_t)t;
}
__device__ __forceinline__ int key_c(uint64_t k) { return (int)(k >> 42) - 1; }
__device__ __forceinline__ int key_u(uint64_t k) { return (int)((k >> 21) & kTokMask) - 1; }
__device__ __forceinline__ int key_tok(uint64_t k) { return (int)(k & kTokMask); }

// Sorted record at place p: token t of key k with its slot (from the key), rank
// r and gamma bits gb.
__device__ __forceinline__ void write_record(const PlanLaunch& a, int p, uint64_t k, int r, int gb) {
  const int t = iclamp(key_tok(k), 0, a.T - 1);
  const int q = iclamp(p, 0, a.T - 1);
  a.srt[q] = make_int4(t, key_u(k), r, gb);
  a.perm[q] = t;
}
__device__ __forceinline__ void write_place(const PlanLaunch& a, int p, uint64_t k) {
  const int4 m = a.maps[iclamp(key_tok(k), 0, a.T - 1)];
  write_record(a, p, k, m.z, m.w);
}

// Exclusive block-wide prefix of two counts (1024 threads); totals to all.
__device__ __forceinline__ void block_scan2(int c0, int c1, int& e0, int& e1, int& t0, int& t1, int* s_w) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int i0 = c0, i1 = c1;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int a0 = __shfl_up(i0, off), a1 = __shfl_up(i1, off);
    if (lane >= off) {
      i0 += a0;
      i1 += a1;
    }
  }
  if (lane == 63) {
    s_w[wave] = i0;
    s_w[32 + wave] = i1;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int r0 = 0, r1 = 0;
    for (int w = 0; w < kPlanThreads / 64; ++w) {
      const int v0 = s_w[w], v1 = s_w[32 + w];
      s_w[w] = r0;
      s_w[32 + w] = r1;
      r0 += v0;
      r1 += v1;
    }
    s_w[16] = r0;
    s_w[48] = r1;
  }
  __syncthreads();
  e0 = s_w[wave] + i0 - c0;
  e1 = s_w[32 + wave] + i1 - c1;
  t0 = s_w[16];
  t1 = s_w[48];
  __syncthreads();
}

// Segments and groups of the sorted keys keys[0, T) (LDS or global memory),
// the meta words, and the check of the host's tiles.  One block of 1024 threads;
// thread i takes places [i per, (i + 1) per).
__device__ void plan_finish(const PlanLaunch& a, const uint64_t* keys, int* s_w) {
  const int T = a.T, tid = threadIdx.x;
  const int per = cdiv(T, kPlanThreads);
  const int p0 = imin(T, tid * per), p1 = imin(T, p0 + per);
  auto seg_start = [&](int p) { return p == 0 || (keys[p] >> 21) != (keys[p - 1] >> 21); };
  auto grp_start = [&](int p) { return p == 0 || (keys[p] >> 42) != (keys[p - 1] >> 42); };
  int ns = 0, ng = 0;
  for (int p = p0; p < p1; ++p) {
    ns += seg_start(p);
    ng += grp_start(p);
  }
  int es, eg, n_seg, n_grp;
  block_scan2(ns, ng, es, eg, n_seg, n_grp, s_w);
  for (int p = p0; p < p1; ++p) {
    const uint64_t k = keys[p];
    if (grp_start(p)) {
      a.grp_off[iclamp(eg, 0, T)] = es;           // a group starts with a segment
      ++eg;
    }
    if (seg_start(p)) {
      const int si = iclamp(es, 0, T - 1);
      a.seg_off[si] = p;
      a.seg_c[si] = key_c(k);
      a.seg_u[si] = key_u(k);
      ++es;
    }
  }
  // tiles staged by the host: each list covers [0, T) with consecutive tiles,
  // and each tile holds tokens of its own centroid only, which for sorted keys
  // (centroid first) holds exactly when its first and last keys carry it
  int bad = 0;
  for (int tau = tid; tau < a.n_tiles; tau += kPlanThreads) {
    const int4 h = a.tiles[tau];
    const int i0 = iclamp(h.x, 0, T - 1), n = iclamp(h.y, 0, T - i0);
    const bool first = tau == 0 || tau == a.n_list0, last = tau == a.n_tiles - 1 || tau == a.n_list0 - 1;
    int start = 0;
    if (!first) {
      const int4 g = a.tiles[tau - 1];
      start = g.x + g.y;
    }
    if (n != h.y || i0 != h.x || n <= 0 || i0 != start || (last && i0 + n != T) || key_c(keys[i0]) != h.z ||
        key_c(keys[i0 + n - 1]) != h.z)
      ++bad;
  }
  if (bad) atomicAdd(a.meta + kMetaErr, bad);
  if (tid == 0) {
    a.seg_off[iclamp(n_seg, 0, T)] = T;
    a.grp_off[iclamp(n_grp, 0, T)] = n_seg;
    a.meta[kMetaNSeg] = n_seg;
    a.meta[kMetaNGrp] = n_grp;
    a.meta[kMetaT] = T;
    a.meta[kMetaNTiles] = a.n_tiles;
  }
}

// Keys a thread of k_plan_sort holds at most: places tid + kPlanThreads e.
constexpr int kKeysPerThread = kSortChunk / kPlanThreads;
static_assert(kSortChunk % kPlanThreads == 0, "a sort chunk is whole keys per thread");

// One compare-exchange step of the bitonic network (merge size k, distance j <
// 64) on the key x at place p, whose partner p ^ j is lane ^ j of the same
// wave: the pair ends ascending when (p & k) == 0 and descending otherwise, so
// the lower place keeps the smaller key exactly when the two conditions agree.
__device__ __forceinline__ uint64_t exchange_in_wave(uint64_t x, int p, int j, int k) {
  const uint64_t y = __shfl_xor(x, j);
  const bool keep_min = ((p & k) == 0) == ((p & j) == 0);
  return keep_min == (x < y) ? x : y;
}

__global__ void __launch_bounds__(kPlanThreads) k_plan_sort(const PlanLaunch a) {
  __shared__ uint64_t s_keys[kSortChunk];
  __shared__ int s_gb[kSortChunk];                   // gamma bits and rank of the chunk's tokens,
  __shared__ uint8_t s_r[kSortChunk];                // for the records of a one-chunk batch
  __shared__ int s_w[64];
  const int tid = threadIdx.x;
  const int base = blockIdx.x * kSortChunk;
  const int cnt = imin(kSortChunk, a.T - base);
  if (tid == 0 && blockIdx.x == 0) a.meta[kMetaErr] = 0;
  // the network spans the smallest power of two >= cnt (padding keys sort last)
  int n2 = 2;
  while (n2 < cnt) n2 <<= 1;
  // Bitonic sort, ascending.  Thread tid holds the places tid + kPlanThreads e,
  // e < ne; steps whose partners lie within a wave (distance j < 64) run on
  // registers through lane shuffles, in the waves that hold places; steps of a
  // larger distance run in LDS, one pair per thread, with a block barrier after
  // each.  (All loop bounds and the wave test are uniform over a wave.)
  const int ne = imax(1, n2 / kPlanThreads);
  const bool holds = (tid & ~63) < n2;
  uint64_t r[kKeysPerThread];
#pragma unroll
  for (int e = 0; e < kKeysPerThread; ++e) {
    const int p = tid + kPlanThreads * e;
    r[e] = kPad;
    if (e < ne && p < cnt) {
      const int4 m = a.maps[base + p];
      r[e] = plan_key(m.x, m.y, base + p);
      s_gb[p] = m.w;
      s_r[p] = (uint8_t)iclamp(m.z, 0, 255);
    }
  }
  for (int k = 2; k <= n2; k <<= 1) {
    if (k / 2 >= 64) {
#pragma unroll
      for (int e = 0; e < kKeysPerThread; ++e)
        if (e < ne && tid + kPlanThreads * e < n2) s_keys[tid + kPlanThreads * e] = r[e];
      __syncthreads();
      for (int j = k >> 1; j >= 64; j >>= 1) {
        for (int i = tid; i < n2 / 2; i += kPlanThreads) {
          const int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1)), hi = lo + j;
          const uint64_t x = s_keys[lo], y = s_keys[hi];
          if ((x > y) == ((lo & k) == 0)) {
            s_keys[lo] = y;
            s_keys[hi] = x;
          }
        }
        __syncthreads();
      }
#pragma unroll
      for (int e = 0; e < kKeysPerThread; ++e)
        if (e < ne && tid + kPlanThreads * e < n2) r[e] = s_keys[tid + kPlanThreads * e];
    }
    if (holds) {
      for (int j = imin(k >> 1, 32); j > 0; j >>= 1) {
#pragma unroll
        for (int e = 0; e < kKeysPerThread; ++e)
          if (e < ne) r[e] = exchange_in_wave(r[e], tid + kPlanThreads * e, j, k);
      }
    }
  }
  if (gridDim.x == 1) {
    // (a thread writes the places it alone read last)
#pragma unroll
    for (int e = 0; e < kKeysPerThread; ++e)
      if (e < ne && tid + kPlanThreads * e < n2) s_keys[tid + kPlanThreads * e] = r[e];
    __syncthreads();
    for (int i = tid; i < cnt; i += kPlanThreads) {
      const uint64_t k = s_keys[i];
      const int t = iclamp(key_tok(k), 0, cnt - 1);   // (one chunk: base is 0)
      write_record(a, i, k, s_r[t], s_gb[t]);
    }
    plan_finish(a, s_keys, s_w);
  } else {
#pragma unroll
    for (int e = 0; e < kKeysPerThread; ++e)
      if (e < ne && tid + kPlanThreads * e < cnt) a.keys[base + tid + kPlanThreads * e] = r[e];
  }
}

// Entries of the ascending run l[0, n) below k.
__device__ __forceinline__ int count_below(const uint64_t* l, int n, uint64_t k) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (l[mid] < k) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

__global__ void __launch_bounds__(256) k_plan_merge(const PlanLaunch a) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= a.T) return;
  const uint64_t k = a.keys[i];
  const int ch = i / kSortChunk;
  int rank = i - ch * kSortChunk;
  const int nch = cdiv(a.T, kSortChunk);
  for (int c = 0; c < nch; ++c) {
    if (c == ch) continue;
    const int lo = c * kSortChunk;
    rank += count_below(a.keys + lo, imin(kSortChunk, a.T - lo), k);
  }
  rank = iclamp(rank, 0, a.T - 1);
  a.keys_sorted[rank] = k;
  write_place(a, rank, k);
}

__global__ void __launch_bounds__(kPlanThreads) k_plan_finish(const PlanLaunch a) {
  __shared__ int s_w[64];
  plan_finish(a, a.keys_sorted, s_w);
}

}  // namespace

hipError_t launch_plan(const PlanLaunch& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  if (a.T > kMaxTokens) return hipErrorInvalidValue;
  const int nch = cdiv(a.T, kSortChunk);
  hipLaunchKernelGGL(k_plan_sort, dim3(nch), dim3(kPlanThreads), 0, s, a);
  if (nch > 1) {
    hipLaunchKernelGGL(k_plan_merge, dim3(cdiv(a.T, 256)), dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_plan_finish, dim3(1), dim3(kPlanThreads), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace salt
