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

// Exclusive block-wide prefix of two counts (NT threads, at most 16 waves);
// totals to all.
template <int NT>
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
    for (int w = 0; w < NT / 64; ++w) {
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
// the meta words, and the check of the host's tiles.  One block of NT threads;
// thread i takes places [i per, (i + 1) per).
template <int NT>
__device__ void plan_finish(const PlanLaunch& a, const uint64_t* keys, int* s_w) {
  const int T = a.T, tid = threadIdx.x;
  const int per = cdiv(T, NT);
  const int p0 = imin(T, tid * per), p1 = imin(T, p0 + per);
  auto seg_start = [&](int p) { return p == 0 || (keys[p] >> 21) != (keys[p - 1] >> 21); };
  auto grp_start = [&](int p) { return p == 0 || (keys[p] >> 42) != (keys[p - 1] >> 42); };
  int ns = 0, ng = 0;
  for (int p = p0; p < p1; ++p) {
    ns += seg_start(p);
    ng += grp_start(p);
  }
  int es, eg, n_seg, n_grp;
  block_scan2<NT>(ns, ng, es, eg, n_seg, n_grp, s_w);
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
  for (int tau = tid; tau < a.n_tiles; tau += NT) {
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

// One block of NT threads per chunk of at most NC = NT * KPT keys: NT = 1024
// for batches of more than 512 tokens (KPT = 4, a chunk of kSortChunk keys),
// otherwise the smallest of 64, 256 or 512 threads that holds the batch (KPT = 1).
template <int NT>
__global__ void __launch_bounds__(NT) k_plan_sort(const PlanLaunch a) {
  constexpr int KPT = NT == kPlanThreads ? kSortChunk / kPlanThreads : 1;   // keys per thread, at most
  constexpr int NC = NT * KPT;
  __shared__ uint64_t s_keys[NC];
  __shared__ int s_gb[NC];                   // gamma bits and rank of the chunk's tokens,
  __shared__ uint8_t s_r[NC];                // for the records of a one-chunk batch
  __shared__ int s_w[64];
  const int tid = threadIdx.x;
  const int base = blockIdx.x * NC;
  const int cnt = imin(NC, a.T - base);
  if (tid == 0 && blockIdx.x == 0) a.meta[kMetaErr] = 0;
  // the network spans the smallest power of two >= cnt (padding keys sort last)
  int n2 = 2;
  while (n2 < cnt) n2 <<= 1;
  // Bitonic sort, ascending.  Thread tid holds the places tid + NT e,
  // e < ne; steps whose partners lie within a wave (distance j < 64) run on
  // registers through lane shuffles, in the waves that hold places; steps of a
  // larger distance run in LDS, one pair per thread, with a block barrier after
  // each.  (All loop bounds and the wave test are uniform over a wave.)
  const int ne = imax(1, n2 / NT);
  const bool holds = (tid & ~63) < n2;
  uint64_t r[KPT];
#pragma unroll
  for (int e = 0; e < KPT; ++e) {
    const int p = tid + NT * e;
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
      for (int e = 0; e < KPT; ++e)
        if (e < ne && tid + NT * e < n2) s_keys[tid + NT * e] = r[e];
      __syncthreads();
      for (int j = k >> 1; j >= 64; j >>= 1) {
        for (int i = tid; i < n2 / 2; i += NT) {
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
      for (int e = 0; e < KPT; ++e)
        if (e < ne && tid + NT * e < n2) r[e] = s_keys[tid + NT * e];
    }
    if (holds) {
      for (int j = imin(k >> 1, 32); j > 0; j >>= 1) {
#pragma unroll
        for (int e = 0; e < KPT; ++e)
          if (e < ne) r[e] = exchange_in_wave(r[e], tid + NT * e, j, k);
      }
    }
  }
  if (gridDim.x == 1) {
    // (a thread writes the places it alone read last)
#pragma unroll
    for (int e = 0; e < KPT; ++e)
      if (e < ne && tid + NT * e < n2) s_keys[tid + NT * e] = r[e];
    __syncthreads();
    for (int i = tid; i < cnt; i += NT) {
      const uint64_t k = s_keys[i];
      const int t = iclamp(key_tok(k), 0, cnt - 1);   // (one chunk: base is 0)
      write_record(a, i, k, s_r[t], s_gb[t]);
    }
    plan_finish<NT>(a, s_keys, s_w);
  } else {
#pragma unroll
    for (int e = 0; e < KPT; ++e)
      if (e < ne && tid + NT * e < cnt) a.keys[base + tid + NT * e] = r[e];
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
  plan_finish<kPlanThreads>(a, a.keys_sorted, s_w);
}

}  // namespace

hipError_t launch_plan(const PlanLaunch& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  if (a.T > kMaxTokens) return hipErrorInvalidValue;
  const int nch = cdiv(a.T, kSortChunk);
  if (a.T <= 64) hipLaunchKernelGGL(k_plan_sort<64>, dim3(1), dim3(64), 0, s, a);
  else if (a.T <= 256) hipLaunchKernelGGL(k_plan_sort<256>, dim3(1), dim3(256), 0, s, a);
  else if (a.T <= 512) hipLaunchKernelGGL(k_plan_sort<512>, dim3(1), dim3(512), 0, s, a);
  else hipLaunchKernelGGL(k_plan_sort<kPlanThreads>, dim3(nch), dim3(kPlanThreads), 0, s, a);
  if (nch > 1) {
    hipLaunchKernelGGL(k_plan_merge, dim3(cdiv(a.T, 256)), dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_plan_finish, dim3(1), dim3(kPlanThreads), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace salt
