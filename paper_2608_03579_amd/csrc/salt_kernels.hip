// HIP kernels of libsalt for gfx950 (MI355X): the device plan builder and the
// fused centroid + residual apply.
//
// Per token t of a plan (the served weight of Sec. 3.3 minus W_base):
//     v_t = x_t [A_c | A_u]              shrink: one rank-(r_c + r_u) contraction
//     v_t[0:r_c] *= gamma_t              centroid scale (Sec. 3.3)
//     y_t = rne(y_t + v_t [B_c ; B_u])   expand and accumulate, fp32 math
//
// Tokens are cut into tiles of M = 16, 32 or 64 sorted tokens that share one
// centroid.  For a tile, the centroid part of the shrink, [M x in] . [in x r_c],
// and of the expand, [M x r_c] . [r_c x out], are dense skinny GEMMs and run on
// MFMA (v_mfma_f32_16x16x32_bf16); the residual part differs per token, has
// rank <= 2 (<= 16 for plain LoRA baselines) and runs on the vector ALUs, with
// lane shuffles for the reductions.
//
// One launch per apply holds two kinds of blocks.  Shrink blocks (the first
// n_tiles * S block ids) each reduce one tile over one K range into a split-K
// partial of v.  By default they add it into v with fp32 device atomics and
// raise their own ready word of the tile to this apply's epoch; the expand
// waits for all S words (one word per writer: no contended counter).  In the
// deterministic mode they store the partial instead, and the last of a tile's
// S blocks to arrive sums the partials in split order, stores v and raises the
// tile's ready word to this apply's epoch.  Expand blocks (the rest) prefetch
// their y, B_c and B_u slices, wait, read v, scale its centroid part by gamma
// and update y.  Arrival counts and epochs only grow between plan builds; the
// host passes the values this apply reaches.
// Blocks are dispatched in id order, so every shrink block has started before
// any expand block waits on it, and shrink blocks never wait: the wait always
// ends.  It is still bounded; a block that gives up records an error in the
// plan's meta words and leaves its slice of y untouched.
#include <hip/hip_ext.h>

#include <algorithm>

#include "salt_internal.h"

namespace salt {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr uint32_t kSpinMax = 1u << 24;   // ~0.5 s of polling before giving up
constexpr int kYS = kNC + 4;              // LDS row stride of the expand's y tile (floats)

// ---------------------------------------------------------------------------
// element types: bf16 (uint16 storage) and fp32, 8 elements per vector
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16, round to nearest even: gfx950's packed conversion
// (v_cvt_pk_bf16_f32), two values per instruction; `lo` lands in the low half.
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) { return pack_bf16x2(f, 0.f) & 0xffffu; }

template <typename E>
struct Ops;

template <>
struct Ops<uint16_t> {
  using Vec = uint4;
  static __device__ __forceinline__ Vec zero() { return make_uint4(0u, 0u, 0u, 0u); }
  static __device__ __forceinline__ Vec load(const uint16_t* p) {
    return *reinterpret_cast<const uint4*>(p);
  }
  static __device__ __forceinline__ void to_f32(const Vec& v, float* o) {
    o[0] = bf_lo(v.x); o[1] = bf_hi(v.x); o[2] = bf_lo(v.y); o[3] = bf_hi(v.y);
    o[4] = bf_lo(v.z); o[5] = bf_hi(v.z); o[6] = bf_lo(v.w); o[7] = bf_hi(v.w);
  }
  static __device__ __forceinline__ void store(uint16_t* p, const float* f) {
    uint4 w;
    w.x = pack_bf16x2(f[0], f[1]);
    w.y = pack_bf16x2(f[2], f[3]);
    w.z = pack_bf16x2(f[4], f[5]);
    w.w = pack_bf16x2(f[6], f[7]);
    *reinterpret_cast<uint4*>(p) = w;
  }
  // acc + sum_e a[e] * b[e], products exact in fp32
  static __device__ __forceinline__ float dot(const Vec& a, const Vec& b, float acc) {
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.x), __builtin_bit_cast(bf16x2, b.x), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.y), __builtin_bit_cast(bf16x2, b.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.z), __builtin_bit_cast(bf16x2, b.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.w), __builtin_bit_cast(bf16x2, b.w), acc, false);
    return acc;
  }
  // One 16x16x32 step: lane l brings row (l & 15) of the left operand and column
  // (l & 15) of the right one, 8 consecutive k each.
  static __device__ __forceinline__ f32x4 mma(const Vec& a, const Vec& b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
  // Same with an fp32 right operand: v = hi + lo with hi, lo bf16, so the
  // product keeps about 16 significant bits of v (two MFMA steps).
  static __device__ __forceinline__ f32x4 mma_f32rhs(const Vec& a, const float* v, f32x4 c) {
    uint32_t h[8], l[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      h[e] = f32_to_bf16_rne(v[e]);
      l[e] = f32_to_bf16_rne(v[e] - __uint_as_float(h[e] << 16));
    }
    const uint4 hi = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
    const uint4 lo = make_uint4(l[0] | (l[1] << 16), l[2] | (l[3] << 16), l[4] | (l[5] << 16), l[6] | (l[7] << 16));
    c = mma(a, hi, c);
    return mma(a, lo, c);
  }
};

template <>
struct Ops<float> {
  struct Vec {
    float4 lo, hi;
  };
  static __device__ __forceinline__ Vec zero() {
    return Vec{make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
  }
  static __device__ __forceinline__ Vec load(const float* p) {
    return Vec{*reinterpret_cast<const float4*>(p), *reinterpret_cast<const float4*>(p + 4)};
  }
  static __device__ __forceinline__ void to_f32(const Vec& v, float* o) {
    o[0] = v.lo.x; o[1] = v.lo.y; o[2] = v.lo.z; o[3] = v.lo.w;
    o[4] = v.hi.x; o[5] = v.hi.y; o[6] = v.hi.z; o[7] = v.hi.w;
  }
  static __device__ __forceinline__ void store(float* p, const float* f) {
    *reinterpret_cast<float4*>(p) = make_float4(f[0], f[1], f[2], f[3]);
    *reinterpret_cast<float4*>(p + 4) = make_float4(f[4], f[5], f[6], f[7]);
  }
  static __device__ __forceinline__ float dot(const Vec& a, const Vec& b, float acc) {
    float x[8], y[8];
    to_f32(a, x);
    to_f32(b, y);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fmaf(x[e], y[e], acc);
    return acc;
  }
  // Eight 16x16x4 fp32 steps: in step e, lane group g = l >> 4 supplies k = 8g + e,
  // so the eight steps together cover the same 32 k as one bf16 step.
  static __device__ __forceinline__ f32x4 mma(const Vec& a, const Vec& b, f32x4 c) {
    float x[8], y[8];
    to_f32(a, x);
    to_f32(b, y);
#pragma unroll
    for (int e = 0; e < 8; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[e], y[e], c, 0, 0, 0);
    return c;
  }
  static __device__ __forceinline__ f32x4 mma_f32rhs(const Vec& a, const float* v, f32x4 c) {
    float x[8];
    to_f32(a, x);
#pragma unroll
    for (int e = 0; e < 8; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[e], v[e], c, 0, 0, 0);
    return c;
  }
};

// Hand-off of split-K partials between blocks, with no cache-wide fences.
// Partials and v are written and read with device-coherent 16-byte buffer
// accesses (cache policy sc1: stores write through to the device-coherent
// level, loads never return a stale cached copy) or added with device-scope
// atomics, which are performed at that level.  A shrink block waits until its
// stores or atomics have completed (s_waitcnt), meets its other waves, and only
// then bumps the tile's arrival count; a block that consumes the data issues
// its loads only after it has seen the count.  Completed device-coherent writes
// are visible to every later device-coherent load, so the counter orders the
// data without writing back or invalidating the L2.
constexpr int kCoherent = 16;                 // buffer cache policy: sc1 (device scope)
constexpr int kRawBufferWord3 = 0x00020000;   // gfx9 raw buffer resource, dword 3

__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRawBufferWord3);
}
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 load4_coherent(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, kCoherent));
}
__device__ __forceinline__ void store4_coherent(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, float4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, (int)byte_off, 0, kCoherent);
}

// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------
constexpr int kPlanThreads = 256;     // threads of a plan block (the large-batch ranking, an apply's writer)
constexpr int kPlanSmallThreads = 1024;   // threads of the one-block plan: one wave per run of 64 keys
constexpr int kPlanTokPerBlock = 64;  // multi-block ranking: four lanes per token
constexpr int kPlanChunk = 2048;      // keys staged in LDS per pass (multi-block ranking)
constexpr int kMaxGroups = 72;        // centroid groups: C + 1 <= 65

// Total order key (centroid, slot, token), -1 ids first: each field is shifted by
// one so that -1 becomes 0.  Fields are 21 bits wide.
__device__ __forceinline__ uint64_t plan_key(int c, int u, int t) {
  return (uint64_t(uint32_t(c + 1)) << 42) | (uint64_t(uint32_t(u + 1)) << 21) |
         uint64_t(uint32_t(t));
}
constexpr uint64_t kNoKey = ~0ull;    // pads a run; above every real key

// The 64 keys of a wave (one per lane) sorted ascending across the lanes: a
// bitonic network of compare-exchanges between lanes l and l ^ stride.
__device__ __forceinline__ uint64_t wave_sort64(uint64_t k) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      const uint64_t o = __shfl_xor(k, stride);
      // blocks of `size` lanes alternate ascending / descending; the lower lane
      // of an ascending pair keeps the minimum
      const bool keep_min = ((lane & size) == 0) == ((lane & stride) == 0);
      k = keep_min ? (o < k ? o : k) : (o < k ? k : o);
    }
  }
  return k;
}

// Entries of the ascending run l[0:64] below k (branch-free binary search).
__device__ __forceinline__ int count_below64(const uint64_t* l, uint64_t k) {
  int lo = 0;
#pragma unroll
  for (int step = 32; step > 0; step >>= 1) lo += (l[lo + step - 1] < k) ? step : 0;
  return lo + (l[lo] < k ? 1 : 0);
}

// Exclusive counts of two predicates over the threads of the block, and their
// totals: per-wave ballots, then one wave scans the per-wave counts.
__device__ __forceinline__ void block_excl_count2(bool p0, bool p1, int* s_wave, int& r0, int& r1, int& tot0,
                                                  int& tot1) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const uint64_t m0 = __ballot(p0), m1 = __ballot(p1);
  const int in0 = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m0 >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m0, 0u));
  const int in1 = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m1 >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m1, 0u));
  if (lane == 0) {
    s_wave[wave] = __popcll(m0);
    s_wave[16 + wave] = __popcll(m1);
  }
  __syncthreads();
  if (wave == 0) {
    // lanes 0..15: counts of predicate 0, lanes 16..31: predicate 1 (nw <= 16)
    const int w = lane & 15;
    int c = (lane < 32 && w < nw) ? s_wave[(lane >> 4) * 16 + w] : 0;
    int incl = c;
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const int v = __shfl_up(incl, off, 16);
      if (w >= off) incl += v;
    }
    if (lane < 32) {
      s_wave[32 + lane] = incl - c;                       // exclusive prefix per wave
      if (w == 15) s_wave[64 + (lane >> 4)] = incl;       // totals
    }
  }
  __syncthreads();
  r0 = s_wave[32 + wave] + in0;
  r1 = s_wave[48 + wave] + in1;
  tot0 = s_wave[64];
  tot1 = s_wave[65];
  __syncthreads();
}

// Group and tile bookkeeping of one plan, in LDS.
struct PlanShared {
  int s_wave[72];
  int g_start[kMaxGroups + 1];   // first sorted position of each group, then T
  int g_c[kMaxGroups];           // centroid of each group
  int g_tile[kMaxGroups + 1];    // first tile of each group, then the tile count
  int n_seg, n_grp, n_tiles;
};

// A batch sorted in LDS by one block: up to CAP tokens.
template <int CAP>
struct PlanLds {
  static_assert(CAP % 64 == 0, "whole runs of 64 keys");
  uint64_t key[CAP];     // ascending runs of 64 keys
  int4 maps[CAP];        // staged maps (c, u, r, gamma bits) by token
  int4 srt[CAP];         // (token, u, r, gamma bits) by sorted position
  int32_t c[CAP];        // centroid id by sorted position
  PlanShared sh;
};

// Sorts maps[0:T] (T <= CAP) by plan key into L.srt / L.c.  Each wave sorts
// runs of 64 keys across its lanes; a key's rank is its place in its own run
// plus the number of keys below it in every other run (binary searches).
template <int CAP, int NT = kPlanThreads>
__device__ __forceinline__ void plan_sort(const int4* maps, int T, PlanLds<CAP>& L) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nrun = (T + 63) >> 6;
  for (int i = tid; i < T; i += NT) L.maps[i] = maps[i];
  __syncthreads();
  for (int run = wave; run < nrun; run += NT / 64) {
    const int t = run * 64 + lane;
    uint64_t k = kNoKey;
    if (t < T) {
      const int4 m = L.maps[t];
      k = plan_key(m.x, m.y, t);
    }
    L.key[t] = wave_sort64(k);
  }
  __syncthreads();
  for (int run = wave; run < nrun; run += NT / 64) {
    const uint64_t k = L.key[run * 64 + lane];
    if (k != kNoKey) {
      // the searches in different runs are independent: unrolled, they overlap
      int rank = lane;
#pragma unroll
      for (int o = 0; o < CAP / 64; ++o)
        if (o < nrun && o != run) rank += count_below64(L.key + o * 64, k);
      const int t = (int)(k & 0x1fffffu);
      const int4 m = L.maps[t];
      L.srt[rank] = make_int4(t, m.y, m.z, m.w);
      L.c[rank] = m.x;
    }
  }
  __syncthreads();
}

// Segments (equal centroid and slot) and groups (equal centroid) of the sorted
// batch srt / srt_c (LDS or global memory), and the tiles of M tokens that cut
// each group.  Writes the segment and group arrays of `out` when `write` is set.
// (Inlined everywhere: a plan buffer struct whose address escapes would be
// copied to scratch memory.)
__device__ __forceinline__ void plan_groups(bool write, const PlanBuffers& out, const int4* srt,
                                            const int32_t* srt_c, int T, int M, PlanShared& sh) {
  const int tid = threadIdx.x, nt = blockDim.x;
  int seg_base = 0, grp_base = 0;
  for (int base = 0; base < T; base += nt) {
    const int i = base + tid;
    int c = 0, u = 0;
    bool ns = false, ng = false;
    if (i < T) {
      c = srt_c[i];
      u = srt[i].y;
      if (i == 0) {
        ns = ng = true;
      } else {
        const int cp = srt_c[i - 1], up = srt[i - 1].y;
        ng = (c != cp);
        ns = ng || (u != up);
      }
    }
    int seg_tot, grp_tot, sr, gr;
    block_excl_count2(ns, ng, sh.s_wave, sr, gr, seg_tot, grp_tot);
    if (ns && write) {
      const int sg = seg_base + sr;
      out.seg_off[sg] = i;
      out.seg_c[sg] = c;
      out.seg_u[sg] = u;
    }
    if (ng) {
      const int g = grp_base + gr;
      if (write) {
        out.grp_off[g] = seg_base + sr;
        out.grp_tok[g] = i;
        out.grp_c[g] = c;
      }
      if (g < kMaxGroups) {
        sh.g_start[g] = i;
        sh.g_c[g] = c;
      }
    }
    seg_base += seg_tot;
    grp_base += grp_tot;
  }
  if (tid == 0) {
    const int ng = grp_base < kMaxGroups ? grp_base : kMaxGroups;
    sh.g_start[ng] = T;
    int acc = 0;
    for (int g = 0; g < ng; ++g) {
      sh.g_tile[g] = acc;
      acc += (sh.g_start[g + 1] - sh.g_start[g] + M - 1) / M;
    }
    sh.g_tile[ng] = acc;
    sh.n_seg = seg_base;
    sh.n_grp = grp_base;
    sh.n_tiles = grp_base < kMaxGroups ? acc : -1;
    if (write) {
      out.seg_off[seg_base] = T;
      out.grp_off[grp_base] = seg_base;
      out.grp_tok[grp_base] = T;
    }
  }
  __syncthreads();
}

// First sorted position, token count and centroid of tile tau.
__device__ __forceinline__ int4 tile_header(const PlanShared& sh, int tau, int M) {
  int lo = 0, hi = sh.n_grp - 1;    // last group whose first tile <= tau
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (sh.g_tile[mid] <= tau) lo = mid;
    else hi = mid - 1;
  }
  const int i0 = sh.g_start[lo] + (tau - sh.g_tile[lo]) * M;
  return make_int4(i0, min(M, sh.g_start[lo + 1] - i0), sh.g_c[lo], 0);
}

// Record k of tile tau: k = 0 the header, k = 1 .. M its sorted tokens, padded
// with (0, -1, 0, 0) past the tile's count.
__device__ __forceinline__ int4 tile_record(const PlanShared& sh, const int4* srt, int tau, int k, int M) {
  const int4 h = tile_header(sh, tau, M);
  if (k == 0) return h;
  return k - 1 < h.y ? srt[h.x + k - 1] : make_int4(0, -1, 0, 0);
}

// Tile records and meta words of a plan whose groups are in `sh`; checks that
// the tiles fit the plan's buffers (else n_tiles = -1 in the meta words).
__device__ __forceinline__ void plan_write_tiles(const PlanBuffers& b, const int4* srt, int T, int M,
                                                 const PlanShared& sh) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const int n_tiles = sh.n_tiles;
  const bool fits = n_tiles >= 0 && (size_t)n_tiles * (M + 1) <= b.tile_cap && n_tiles <= b.tiles_max;
  if (fits)
    for (int e = tid; e < n_tiles * (M + 1); e += nt) b.tiles[e] = tile_record(sh, srt, e / (M + 1), e % (M + 1), M);
  if (tid == 0) {
    b.meta[kMetaNSeg] = sh.n_seg;
    b.meta[kMetaNGrp] = sh.n_grp;
    b.meta[kMetaT] = T;
    b.meta[kMetaNTiles] = fits ? n_tiles : -1;
  }
}

// Per-tile words a standalone build resets: the arrival counters (the ordered
// sums count arrivals from zero after every build) and, when asked, the ready
// words (epochs restart).
__device__ __forceinline__ void plan_reset_words(const PlanArgs& a, int first, int step) {
  const PlanBuffers& b = a.b;
  for (int t = first; t < b.tiles_max; t += step) b.arrive[(size_t)t * kCounterStride] = 0u;
  if (a.reset_ready)
    for (int e = first; e < b.tiles_max * kMaxSplit; e += step)
      b.ready[(size_t)(e / kMaxSplit) * kReadyPerTile + (size_t)(e % kMaxSplit) * kReadyStride] = 0u;
}

// Batches of up to kPlanSmallT tokens: one block of 16 waves sorts in LDS
// (each wave one run of 64 keys).
__global__ void __launch_bounds__(kPlanSmallThreads) k_plan_small(PlanArgs a) {
  static_assert(kPlanSmallT <= 64 * (kPlanSmallThreads / 64), "one run of 64 keys per wave");
  __shared__ PlanLds<kPlanSmallT> L;
  const int T = a.T, tid = threadIdx.x;
  plan_reset_words(a, tid, kPlanSmallThreads);
  plan_sort<kPlanSmallT, kPlanSmallThreads>(a.b.maps, T, L);
  for (int i = tid; i < T; i += kPlanSmallThreads) {
    a.b.perm[i] = L.srt[i].x;
    a.b.srt[i] = L.srt[i];
    a.b.srt_c[i] = L.c[i];
  }
  plan_groups(true, a.b, L.srt, L.c, T, a.M, L.sh);
  plan_write_tiles(a.b, L.srt, T, a.M, L.sh);
}

// Larger batches: rank by counting smaller keys across blocks; the last block to
// arrive finishes the plan from global memory.
__global__ void __launch_bounds__(kPlanThreads) k_plan_large(PlanArgs a) {
  __shared__ uint64_t skey[kPlanChunk];
  __shared__ PlanShared sh;
  __shared__ int s_last;
  const PlanBuffers& b = a.b;
  const int T = a.T, tid = threadIdx.x;
  plan_reset_words(a, blockIdx.x * kPlanThreads + tid, gridDim.x * kPlanThreads);
  const int t = blockIdx.x * kPlanTokPerBlock + (tid >> 2);
  const int q = tid & 3;
  int4 mine = make_int4(0, 0, 0, 0);
  uint64_t my = kNoKey;
  if (t < T) {
    mine = b.maps[t];
    my = plan_key(mine.x, mine.y, t);
  }
  int cnt = 0;
  for (int base = 0; base < T; base += kPlanChunk) {
    const int n = min(kPlanChunk, T - base);
    __syncthreads();
    for (int i = tid; i < n; i += kPlanThreads) {
      const int4 m = b.maps[base + i];
      skey[i] = plan_key(m.x, m.y, base + i);
    }
    __syncthreads();
    for (int i = q; i < n; i += 4) cnt += (skey[i] < my) ? 1 : 0;
  }
  cnt += __shfl_xor(cnt, 1);
  cnt += __shfl_xor(cnt, 2);
  if (t < T && q == 0) {
    b.perm[cnt] = t;
    b.srt[cnt] = make_int4(t, mine.y, mine.z, mine.w);
    b.srt_c[cnt] = mine.x;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (tid == 0) {
    const uint32_t old = __hip_atomic_fetch_add(b.counter, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (old == gridDim.x - 1) ? 1 : 0;
  }
  __syncthreads();
  if (!s_last) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  plan_groups(true, b, b.srt, b.srt_c, T, a.M, sh);
  plan_write_tiles(b, b.srt, T, a.M, sh);
  if (tid == 0) __hip_atomic_store(b.counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One tile of a batch of T <= kPlanFusedT tokens (one token per thread), cut
// straight from the maps by an apply block that plans for itself.  Groups are the
// centroid ids in order (-1 first), so a per-id token count and its prefix sums
// give every group's first position and first tile.  Inside its group a token's
// place is its rank in batch order (ballots): the apply needs each tile to hold
// tokens of one centroid, not the canonical slot order within the group, which the
// plan written by the launch's last block keeps.
static_assert(kPlanFusedT <= kPlanThreads, "one token per thread of an apply block");
struct TileLds {
  int cnt[80];                 // tokens per centroid id + 1 (0 .. 64)
  int wcnt[kPlanThreads / 64]; // tokens of the block's group in each wave
  int4 hdr;                    // (i0, n, c, c + 1) of the block's tile
  int chunk;                   // the tile is chunk `chunk` of its group
  int n_tiles;
};

// Writes the header and the M token records of tile tau to s_tile; returns
// false (for the whole block) if the batch does not cut into n_tiles tiles.
__device__ __forceinline__ bool tile_from_maps(const int4* maps, int T, int M, int tau, int n_tiles, TileLds& L,
                                               int4* s_tile) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int4 m = make_int4(0, 0, 0, 0);
  if (tid < T) m = maps[tid];
  if (tid < 80) L.cnt[tid] = 0;
  // every record starts as padding, so none is ever left unset
  if (tid < M) s_tile[1 + tid] = make_int4(0, -1, 0, 0);
  __syncthreads();
  if (tid < T) atomicAdd(&L.cnt[m.x + 1], 1);
  __syncthreads();
  if (tid < 64) {
    // lane l: centroid id l; id 64 (c = 63) follows lane 63
    const int cnt_l = L.cnt[lane], tiles_l = (cnt_l + M - 1) / M;
    int inc_c = cnt_l, inc_t = tiles_l;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int ac = __shfl_up(inc_c, off), at = __shfl_up(inc_t, off);
      if (lane >= off) {
        inc_c += ac;
        inc_t += at;
      }
    }
    const int start_l = inc_c - cnt_l, tbase_l = inc_t - tiles_l;
    const int cnt64 = L.cnt[64], start64 = __shfl(inc_c, 63), tbase64 = __shfl(inc_t, 63);
    const int tiles64 = (cnt64 + M - 1) / M;
    if (tau >= tbase_l && tau < tbase_l + tiles_l) {
      const int k = tau - tbase_l;
      L.hdr = make_int4(start_l + k * M, min(M, cnt_l - k * M), lane - 1, lane);
      L.chunk = k;
    }
    if (lane == 0) {
      L.n_tiles = tbase64 + tiles64;
      if (tau >= tbase64 && tau < tbase64 + tiles64) {
        const int k = tau - tbase64;
        L.hdr = make_int4(start64 + k * M, min(M, cnt64 - k * M), 63, 64);
        L.chunk = k;
      }
    }
  }
  __syncthreads();
  if (L.n_tiles != n_tiles) return false;
  const int4 h = L.hdr;
  const bool mine = tid < T && m.x + 1 == h.w;
  const uint64_t bal = __ballot(mine);
  if (lane == 0) L.wcnt[wave] = __popcll(bal);
  __syncthreads();
  if (mine) {
    int r = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
    for (int w = 0; w < wave; ++w) r += L.wcnt[w];
    r -= L.chunk * M;
    if (r >= 0 && r < h.y) s_tile[1 + r] = make_int4(tid, m.y, m.z, m.w);
  }
  if (tid == 0) s_tile[0] = make_int4(h.x, h.y, h.z, 0);
  __syncthreads();
  return true;
}

// ---------------------------------------------------------------------------
// apply
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int tile_bytes(int M) { return ((M + 1) * 16 + 255) / 256 * 256; }

// Keeps a prefetched value in registers here: the compiler may not sink its load
// below this point (e.g. past a wait loop).
template <typename V>
__device__ __forceinline__ void pin_regs(const V& v) {
  static_assert(sizeof(V) % 4 == 0, "pin whole 32-bit words");
  uint32_t w[sizeof(V) / 4];
  __builtin_memcpy(w, &v, sizeof(V));
#pragma unroll
  for (int i = 0; i < (int)(sizeof(V) / 4); ++i) asm volatile("" ::"v"(w[i]));
}


// All waves' coherent stores have completed, then one thread adds 1 to
// `counter`; returns (to every thread) the count after the addition.
__device__ __forceinline__ uint32_t publish_add(uint32_t* counter, uint32_t* s_word) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0)
    *s_word = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u;
  __syncthreads();
  return *s_word;
}

// All waves' coherent stores and atomics have completed, then one thread stores `value`.
__device__ __forceinline__ void publish_store(uint32_t* word, uint32_t value) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_store(word, value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wait until words[k * kReadyStride], k < n, all reach `target` (wrap-safe,
// n <= 64): wave 0 polls them with one coherent load per lane.  Returns false
// (and counts an error) if it gives up.
__device__ __forceinline__ bool await_words(const uint32_t* words, int n, uint32_t target, int32_t* err,
                                            int* s_flag) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    uint32_t spins = 0;
    int ok = 1;
    while (true) {
      const uint32_t w = lane < n ? __hip_atomic_load(const_cast<uint32_t*>(words + lane * kReadyStride), __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT)
                                  : target;
      if (__all((int32_t)(w - target) >= 0)) break;
      __builtin_amdgcn_s_sleep(2);
      if (++spins > kSpinMax) {
        if (lane == 0) atomicAdd(err, 1);
        ok = 0;
        break;
      }
    }
    if (lane == 0) *s_flag = ok;
  }
  __syncthreads();
  return *s_flag != 0;
}

// v entries idx .. idx+3 of a tile (row-major [token][R]): the centroid ranks
// j < r_c are scaled by the token's gamma (Sec. 3.3).
__device__ __forceinline__ float4 scale_centroid(float4 v, int idx, int R, int rc, const int4* s_tile) {
  const int t = idx / R, j = idx - t * R;      // the 4 entries share a row (R % 4 == 0)
  const float g = __int_as_float(s_tile[1 + t].w);
  if (j + 0 < rc) v.x *= g;
  if (j + 1 < rc) v.y *= g;
  if (j + 2 < rc) v.z *= g;
  if (j + 3 < rc) v.w *= g;
  return v;
}

// Staged shrink of a 64-token tile (bf16): wave w computes M-block w (16
// tokens) over 64-wide K units [kblk, kblk + 64 * nunit).  An MFMA operand
// fragment is 64 bytes of each of 16 rows, so register loads in that layout
// fetch half lines; from L2 (the centroid rows, shared by every tile of the
// group) that halves what a compute unit can pull.  Here x rows and A_c rows
// are instead loaded as whole 128-byte lines (8 lanes per row) and written to
// LDS, from where each lane reads its fragment.  A 16-byte chunk ch of row r
// sits in slot ch ^ ((r >> 1) & 7) of the row's 8 slots, so that both the
// line-wise writes and the fragment reads hit every LDS bank once per 16
// lanes.  The per-token A_u rows stay register loads in fragment layout
// (lanes of one segment read the same row).  Units rotate through kStageD
// register sets (loads of unit u + kStageD are issued while unit u computes)
// and two LDS stages (one barrier per unit).
constexpr int kStageD = 4;
template <int NBM>
__host__ __device__ constexpr int stage_bytes() { return 4 * 2048 + NBM * 2048; }

template <int NBM, int RU>
__device__ __forceinline__ void shrink_staged_units(const ApplyArgs& a, char* stg, const int4* s_tile, int wave,
                                                    int lane, int n, int c, bool has_c, int kblk, int nunit,
                                                    const uint16_t* const (&aurow)[RU], f32x4 (&acc)[NBM],
                                                    float (&accu)[RU]) {
  using O = Ops<uint16_t>;
  using Vec = O::Vec;
  constexpr int NA = NBM / 2;                   // line loads of A_c per lane and unit (NBM * 16 rows / 8 / 4 waves)
  constexpr int SB = stage_bytes<NBM>();
  if (nunit <= 0) return;
  const int in = a.in_dim, rc = a.r_c;
  const uint16_t* x = reinterpret_cast<const uint16_t*>(a.x);
  // line-load sources: row r8 = lane >> 3 of each 8-row group, slot lane & 7
  const uint16_t* xsrc[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int r = 8 * q + (lane >> 3);          // row within this wave's M-block
    const int t = wave * 16 + r;
    const int ch = (lane & 7) ^ ((r >> 1) & 7);
    xsrc[q] = x + (size_t)s_tile[1 + (t < n ? t : 0)].x * in + kblk + 8 * ch;
  }
  const uint16_t* asrc[NA];
#pragma unroll
  for (int q = 0; q < NA; ++q) {
    const int J = 8 * (wave * NA + q) + (lane >> 3);   // rank row of the block's A_c stage
    const int ch = (lane & 7) ^ ((J >> 1) & 7);
    // without a centroid term (or past r_c) the loads read x's first row / rank 0
    asrc[q] = has_c ? reinterpret_cast<const uint16_t*>(a.cent_at) + ((size_t)c * rc + (J < rc ? J : 0)) * in + kblk + 8 * ch
                    : x + kblk + 8 * ch;
  }
  const int kfrag = 8 * (lane >> 4);            // element offset of this lane's fragment in a 32-wide half
  struct Set {
    Vec xl[2], al[NA], ul[2][RU];
  } set[kStageD];
  auto load = [&](Set& L, int u) {
    const int off = 64 * (u < nunit ? u : nunit - 1);
#pragma unroll
    for (int q = 0; q < 2; ++q) L.xl[q] = O::load(xsrc[q] + off);
#pragma unroll
    for (int q = 0; q < NA; ++q) L.al[q] = O::load(asrc[q] + off);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int j = 0; j < RU; ++j) L.ul[h][j] = O::load(aurow[j] + kblk + off + 32 * h + kfrag);
  };
  // issued in set order (the waits below count on it)
#pragma unroll
  for (int d = 0; d < kStageD; ++d) {
    load(set[d], d);
    __builtin_amdgcn_sched_barrier(0);
  }
  // fragment read offsets (bytes inside a stage): row r = lane & 15, chunk 4h + g
  const int r = lane & 15, g = lane >> 4, sw = (r >> 1) & 7;
  const int xoff = wave * 2048 + r * 128, aoff = 4 * 2048 + r * 128;
  const int nround = (nunit + kStageD - 1) / kStageD;
  for (int rr = 0; rr < nround; ++rr) {
#pragma unroll
    for (int d = 0; d < kStageD; ++d) {
      const int u = rr * kStageD + d;
      char* st = stg + (u & 1) * SB;
      // this unit's lines into the stage, in lane order
#pragma unroll
      for (int q = 0; q < 2; ++q) *reinterpret_cast<Vec*>(st + wave * 2048 + (64 * q + lane) * 16) = set[d].xl[q];
#pragma unroll
      for (int q = 0; q < NA; ++q) *reinterpret_cast<Vec*>(st + 4 * 2048 + (64 * (wave * NA + q) + lane) * 16) = set[d].al[q];
      Vec ul[2][RU];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int j = 0; j < RU; ++j) ul[h][j] = set[d].ul[h][j];
      __syncthreads();
      load(set[d], u + kStageD);
      if (u < nunit) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int slot = ((4 * h + g) ^ sw) * 16;
          const Vec xf = *reinterpret_cast<const Vec*>(st + xoff + slot);
          if (has_c) {
#pragma unroll
            for (int nb = 0; nb < NBM; ++nb)
              acc[nb] = O::mma(xf, *reinterpret_cast<const Vec*>(st + aoff + nb * 2048 + slot), acc[nb]);
          }
#pragma unroll
          for (int j = 0; j < RU; ++j) accu[j] = O::dot(xf, ul[h][j], accu[j]);
        }
      }
    }
  }
}

// Shrink block: tile `tau`, K range `s` of the apply.  Computes the tile's
// split-K partial sums P[s][token][0 : r_c + r_u_max].  In the single-launch
// apply it adds them into v with atomics (default) or stores them for an
// ordered sum (deterministic mode), and counts its arrival; with one K range it
// stores v directly.  In the two-launch apply it stores them for the expand
// launch, which sums the K ranges in order.
// Wave layout: each wave covers MBW of the tile's MB 16-token M-blocks and
// 1/KW of the K range (KW = 4 * MBW / MB waves along K).  With MBW = MB every
// wave holds all of the tile's tokens, so the centroid rows it loads serve
// 16 * MB tokens.
// STG (bf16, 64-token tiles, one M-block per wave): x and A_c pass through LDS
// (see shrink_staged_units).
template <typename E, int MB, int MBW, int RU, int NBM, bool STG = false>
__device__ __forceinline__ void shrink_block(const ApplyArgs& a, int tau, int s, char* lds) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  static_assert(MB % MBW == 0 && 4 % (MB / MBW) == 0, "waves tile the M-blocks");
  constexpr int M = 16 * MB, MG = MB / MBW, KW = 4 / MG;
  constexpr int U0 = shrink_batch((int)(sizeof(Vec) / 4), MBW, NBM, RU) / 2;
  constexpr int U = U0 < 1 ? 1 : U0;            // steps per register buffer
  constexpr int kStepRegs = (int)(sizeof(Vec) / 4) * (MBW + NBM + MBW * RU);   // VGPRs of one step's operands
  int4* s_tile = reinterpret_cast<int4*>(lds);
  float* s_part = reinterpret_cast<float*>(lds + tile_bytes(M));   // [KW][M][R]
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int i0 = __builtin_amdgcn_readfirstlane(s_tile[0].x), n = __builtin_amdgcn_readfirstlane(s_tile[0].y),
            c = __builtin_amdgcn_readfirstlane(s_tile[0].z);   // tile header: uniform
  const int R = a.R, in = a.in_dim, rc = a.r_c;
  // shrink block s of the tile: K range s % sk and, for residual ranks above
  // kRankChunk, rank chunk s / sk (ranks r0 .. r0 + RU - 1); the centroid
  // term belongs to chunk 0
  int sk = s, r0 = 0;
  if constexpr (RU == kRankChunk) {
    sk = s % a.sk;
    r0 = (s / a.sk) * RU;
  }
  const bool has_c = c >= 0 && rc > 0 && r0 == 0;
  const int mg = wave % MG, kq = wave / MG;
  const int kseg = (lane >> 4) * 8;             // k offset of this lane inside a 32-wide step
  int tl[MBW], ru[MBW];                         // lane's token (within the tile) per M-block
  bool tok_ok[MBW];
  const E* xrow[MBW];
  const E* au[MBW];
#pragma unroll
  for (int m = 0; m < MBW; ++m) {
    tl[m] = (mg * MBW + m) * 16 + (lane & 15);
    const int4 tk = s_tile[1 + tl[m]];
    tok_ok[m] = tl[m] < n;
    ru[m] = (tok_ok[m] && tk.y >= 0) ? tk.z : 0;
    xrow[m] = reinterpret_cast<const E*>(a.x) + (size_t)(tok_ok[m] ? tk.x : 0) * in;
    // rank-0 tokens read x's first row instead (a base the compiler cannot
    // merge with the x load, which would make the x load wait)
    const E* slot_a = reinterpret_cast<const E*>(a.pool + (size_t)(tk.y > 0 ? tk.y : 0) * a.slot_stride) +
                      (int64_t)ru[m] * a.tab_prefix;
    au[m] = ru[m] ? slot_a : reinterpret_cast<const E*>(a.x);
  }
  const E* arow[NBM];                           // A_c^T row of this lane per 16-rank block
  bool aok[NBM];
#pragma unroll
  for (int nb = 0; nb < NBM; ++nb) {
    const int j = nb * 16 + (lane & 15);
    aok[nb] = has_c && j < rc;
    // without a centroid term the (never multiplied) loads read the x row
    arow[nb] = has_c ? reinterpret_cast<const E*>(a.cent_at) + ((size_t)c * rc + (aok[nb] ? j : 0)) * in : xrow[0];
  }

  // The block's K range is [kblk, kend), in 32-wide steps; the KW waves along K
  // take its steps in turn (wave kq: steps kq, kq + KW, ...), so that at any
  // time they read neighbouring pieces of the same x rows.
  const int kblk = sk * a.Kc;
  const int kend = min(in, kblk + a.Kc);
  const int nstep_blk = kend > kblk ? (kend - kblk) / 32 : 0;   // whole steps of the block

  f32x4 acc[MBW][NBM];
#pragma unroll
  for (int m = 0; m < MBW; ++m)
#pragma unroll
    for (int nb = 0; nb < NBM; ++nb) acc[m][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float accu[MBW][RU];
#pragma unroll
  for (int m = 0; m < MBW; ++m)
#pragma unroll
    for (int j = 0; j < RU; ++j) accu[m][j] = 0.f;

  // A_u row of rank j for this lane's token: a rank past the token's own reads
  // its rank-0 row (or its x row) instead, so that every load of a whole step
  // is unconditional; those sums are dropped when the partial is written.  In
  // the same way rows past the tile's tokens read row 0 of x and ranks past
  // r_c read rank 0 of the centroid: they only feed MFMA outputs that are
  // never written.
  const E* aurow[MBW][RU];
#pragma unroll
  for (int m = 0; m < MBW; ++m)
#pragma unroll
    for (int j = 0; j < RU; ++j) aurow[m][j] = au[m] + (size_t)(r0 + j < ru[m] ? r0 + j : 0) * in;

  // two register buffers of up to U steps each: the loads of batch b + 1 are
  // in flight while batch b is multiplied.  Every batch issues the same loads
  // (a step past the wave's last, in a short last batch or a batch past the
  // end, re-reads that last step and is not multiplied), so the wait before
  // each multiply counts the loads exactly and never waits for the batch
  // behind it.
  Vec xv[2][U][MBW], av[2][U][NBM], uv[2][U][MBW][RU];
  auto mul_steps = [&](const Vec (&x_)[U][MBW], const Vec (&a_)[U][NBM], const Vec (&u_)[U][MBW][RU], int ns) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (u < ns) {
        if (has_c) {
#pragma unroll
          for (int m = 0; m < MBW; ++m)
#pragma unroll
            for (int nb = 0; nb < NBM; ++nb) acc[m][nb] = O::mma(x_[u][m], a_[u][nb], acc[m][nb]);
        }
#pragma unroll
        for (int m = 0; m < MBW; ++m)
#pragma unroll
          for (int j = 0; j < RU; ++j) accu[m][j] = O::dot(x_[u][m], u_[u][m][j], accu[m][j]);
      }
    }
  };
  // a residual rank chunk past every rank of this wave's tokens has nothing to
  // add: its loads and products are skipped (its partial stays zero)
  bool idle = false;
  if constexpr (RU == kRankChunk && !STG) {      // (the staged loop has block barriers)
    bool busy = false;
#pragma unroll
    for (int m = 0; m < MBW; ++m) busy |= ru[m] > r0;
    idle = r0 > 0 && __ballot(busy) == 0ull;
  }
  if (!idle) {
    if constexpr (STG) {
      static_assert(sizeof(E) == 2 && MB == 4 && MBW == 1, "staged shrink: bf16, 64-token tiles, one M-block per wave");
      // whole 64-wide units through LDS, then an odd last 32-wide step from
      // registers (the ragged end below takes whatever is left)
      const int nunit = (kend - kblk) / 64;
      shrink_staged_units<NBM, RU>(a, lds + tile_bytes(M) + sizeof(float) * (size_t)M * R, s_tile, wave, lane, n,
                                   c, has_c, kblk, nunit, aurow[0], acc[0], accu[0]);
      if (nstep_blk > 2 * nunit) {
        const int kk = kblk + 64 * nunit + kseg;
        xv[0][0][0] = O::load(xrow[0] + kk);
#pragma unroll
        for (int nb = 0; nb < NBM; ++nb) av[0][0][nb] = O::load(arow[nb] + kk);
#pragma unroll
        for (int j = 0; j < RU; ++j) uv[0][0][0][j] = O::load(aurow[0][j] + kk);
        if (has_c) {
#pragma unroll
          for (int nb = 0; nb < NBM; ++nb) acc[0][nb] = O::mma(xv[0][0][0], av[0][0][nb], acc[0][nb]);
        }
#pragma unroll
        for (int j = 0; j < RU; ++j) accu[0][j] = O::dot(xv[0][0][0], uv[0][0][0][j], accu[0][j]);
      }
    } else {
      const int nfull = nstep_blk > kq ? (nstep_blk - kq + KW - 1) / KW : 0;   // this wave's whole steps
      auto load_steps = [&](Vec (&x_)[U][MBW], Vec (&a_)[U][NBM], Vec (&u_)[U][MBW][RU], int step0) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int kk = kblk + 32 * (kq + KW * (step0 + u < nfull ? step0 + u : nfull - 1)) + kseg;
#pragma unroll
          for (int m = 0; m < MBW; ++m) x_[u][m] = O::load(xrow[m] + kk);
#pragma unroll
          for (int nb = 0; nb < NBM; ++nb) a_[u][nb] = O::load(arow[nb] + kk);
#pragma unroll
          for (int m = 0; m < MBW; ++m)
#pragma unroll
            for (int j = 0; j < RU; ++j) u_[u][m][j] = O::load(aurow[m][j] + kk);
        }
      };
      const int nbat = (nfull + U - 1) / U;
      auto steps_of = [&](int b) { return min(U, nfull - b * U); };
      if (nbat == 1) {
        // one batch (short K ranges of small batches): nothing to overlap
        load_steps(xv[0], av[0], uv[0], 0);
        mul_steps(xv[0], av[0], uv[0], steps_of(0));
      } else if (kStepRegs <= 128 && nbat == 2) {
        // two batches: both in flight at once
        load_steps(xv[0], av[0], uv[0], 0);
        load_steps(xv[1], av[1], uv[1], U);
        mul_steps(xv[0], av[0], uv[0], steps_of(0));
        mul_steps(xv[1], av[1], uv[1], steps_of(1));
      } else if constexpr (kStepRegs <= 128) {
        if (nbat > 1) {
          // (a peeled last pair would need a second set of accumulators)
          load_steps(xv[0], av[0], uv[0], 0);
          for (int b = 0; b < nbat; b += 2) {
            load_steps(xv[1], av[1], uv[1], (b + 1) * U);
            mul_steps(xv[0], av[0], uv[0], steps_of(b));
            load_steps(xv[0], av[0], uv[0], (b + 2) * U);
            if (b + 1 < nbat) mul_steps(xv[1], av[1], uv[1], steps_of(b + 1));
          }
        }
      } else {
        // one step's operands alone fill most of the register file (fp32 with
        // wide centroid and residual ranks): no second buffer
        for (int b = 0; b < nbat; ++b) {
          load_steps(xv[0], av[0], uv[0], b * U);
          mul_steps(xv[0], av[0], uv[0], steps_of(b));
        }
      }
    }
    if (kend > kblk + 32 * nstep_blk && nstep_blk % KW == kq) {
      // ragged end of the K range (in_dim not a multiple of 32), taken by the wave
      // whose turn it is: k >= kend reads zero
      const int kk = kblk + 32 * nstep_blk + kseg;
      const bool kin = kk < kend;
#pragma unroll
      for (int m = 0; m < MBW; ++m) xv[0][0][m] = kin ? O::load(xrow[m] + kk) : O::zero();
      if (has_c) {
#pragma unroll
        for (int nb = 0; nb < NBM; ++nb) av[0][0][nb] = kin ? O::load(arow[nb] + kk) : O::zero();
      }
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int j = 0; j < RU; ++j) uv[0][0][m][j] = kin ? O::load(aurow[m][j] + kk) : O::zero();
      mul_steps(xv[0], av[0], uv[0], 1);
    }
  }
  // residual: lanes l, l^16, l^32, l^48 hold the four k offsets of one token
#pragma unroll
  for (int m = 0; m < MBW; ++m)
#pragma unroll
    for (int j = 0; j < RU; ++j) {
      accu[m][j] += __shfl_xor(accu[m][j], 16);
      accu[m][j] += __shfl_xor(accu[m][j], 32);
    }
  // this wave's partial -> LDS [kq][token][j]
  float* P = s_part + (size_t)kq * M * R;
#pragma unroll
  for (int m = 0; m < MBW; ++m)
#pragma unroll
    for (int nb = 0; nb < NBM; ++nb) {
      const int j = nb * 16 + (lane & 15);
      if (j < rc) {
#pragma unroll
        for (int e = 0; e < 4; ++e) P[((mg * MBW + m) * 16 + 4 * (lane >> 4) + e) * R + j] = acc[m][nb][e];
      }
    }
  if (lane < 16) {
#pragma unroll
    for (int m = 0; m < MBW; ++m) {
#pragma unroll
      for (int j = 0; j < RU; ++j)
        if (r0 + j < a.r_u_max) P[tl[m] * R + rc + r0 + j] = r0 + j < ru[m] ? accu[m][j] : 0.f;
      if (RU == kRankChunk && a.S > a.sk && !a.atomic_sum)   // the other chunks' residual columns
        for (int j = 0; j < a.r_u_max; ++j)
          if (j < r0 || j >= r0 + RU) P[tl[m] * R + rc + j] = 0.f;
      for (int j = rc + a.r_u_max; j < R; ++j) P[tl[m] * R + j] = 0.f;   // row padding
    }
  }
  __syncthreads();
  // R is a multiple of 4: rows are whole float4 vectors
  const int nR4 = n * R / 4;
  if (a.two_pass && !a.atomic_sum) {
    // two-launch apply, ordered sums: this K range's partial for the expand launch
    float4* dst = reinterpret_cast<float4*>(a.partials + ((size_t)s * a.T + i0) * R);
    for (int i4 = tid; i4 < nR4; i4 += 256) {
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int q = 0; q < KW; ++q) {
        const float4 p = *reinterpret_cast<const float4*>(s_part + (size_t)q * M * R + 4 * i4);
        v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
      }
      dst[i4] = v;
    }
    return;
  }
  const __amdgpu_buffer_rsrc_t rv = coherent_rsrc(a.v + (size_t)i0 * R, (uint32_t)(nR4 * 16));
  if (a.atomic_sum) {
    // the next apply of the plan adds into the other v buffer: split 0 clears
    // this tile's rows, and all shrink blocks share the rows past the batch
    // that an earlier, larger batch left behind
    if (s == 0) {
      const __amdgpu_buffer_rsrc_t rz = coherent_rsrc(a.v_clear + (size_t)i0 * R, (uint32_t)(nR4 * 16));
      for (int i4 = tid; i4 < nR4; i4 += 256) store4_coherent(rz, 16u * i4, make_float4(0.f, 0.f, 0.f, 0.f));
    }
    if (a.clear_rows > a.T) {
      const int n4 = (a.clear_rows - a.T) * R / 4;
      const __amdgpu_buffer_rsrc_t rz = coherent_rsrc(a.v_clear + (size_t)a.T * R, (uint32_t)(n4 * 16));
      const int nb = a.n_tiles * a.S;
      for (int i4 = (s * a.n_tiles + tau) * 256 + tid; i4 < n4; i4 += nb * 256)
        store4_coherent(rz, 16u * i4, make_float4(0.f, 0.f, 0.f, 0.f));
    }
  }
  if (a.S == 1) {
    // one K range: this block writes v itself
    for (int i4 = tid; i4 < nR4; i4 += 256) {
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int q = 0; q < KW; ++q) {
        const float4 p = *reinterpret_cast<const float4*>(s_part + (size_t)q * M * R + 4 * i4);
        v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
      }
      store4_coherent(rv, 16u * i4, v);
    }
  } else if (a.atomic_sum) {
    // add this K range's partial into v (cleared by the previous apply or the build)
    float* vt = a.v + (size_t)i0 * R;
    if (RU == kRankChunk && a.S > a.sk && r0 > 0) {
      // a rank chunk past the first adds only its own ranks of the tokens that
      // have them (every other entry of its partial is zero)
      for (int i = tid; i < n * RU; i += 256) {
        const int t = i / RU, j = r0 + i % RU;
        const int4 tk = s_tile[1 + t];
        if (tk.y >= 0 && j < tk.z) {
          float p = 0.f;
#pragma unroll
          for (int q = 0; q < KW; ++q) p += s_part[(size_t)q * M * R + t * R + rc + j];
          __hip_atomic_fetch_add(vt + t * R + rc + j, p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    } else if (RU == kRankChunk && a.S > a.sk) {
      // the first rank chunk: the centroid ranks and residual ranks 0 .. RU - 1
      const int w = rc + RU;
      for (int i = tid; i < n * w; i += 256) {
        const int t = i / w, j = i % w;
        float p = 0.f;
#pragma unroll
        for (int q = 0; q < KW; ++q) p += s_part[(size_t)q * M * R + t * R + j];
        __hip_atomic_fetch_add(vt + t * R + j, p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    } else {
      for (int i = tid; i < n * R; i += 256) {
        float p = 0.f;
#pragma unroll
        for (int q = 0; q < KW; ++q) p += s_part[(size_t)q * M * R + i];
        __hip_atomic_fetch_add(vt + i, p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  } else {
    const __amdgpu_buffer_rsrc_t rp =
        coherent_rsrc(a.partials + ((size_t)s * a.T + i0) * R, (uint32_t)(nR4 * 16));
    for (int i4 = tid; i4 < nR4; i4 += 256) {
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int q = 0; q < KW; ++q) {
        const float4 p = *reinterpret_cast<const float4*>(s_part + (size_t)q * M * R + 4 * i4);
        v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
      }
      store4_coherent(rp, 16u * i4, v);
    }
    __shared__ uint32_t s_count;
    if (publish_add(a.arrive + (size_t)tau * kCounterStride, &s_count) != a.target) return;
    // the last of the tile's S blocks: sum the splits in order
    const size_t split_bytes = (size_t)a.T * R * 4;
    const __amdgpu_buffer_rsrc_t rall = coherent_rsrc(a.partials + (size_t)i0 * R,
                                                      (uint32_t)((a.S - 1) * split_bytes + nR4 * 16));
    constexpr int Q = 2, SG = 8;                 // vectors x splits in flight per thread
    for (int base = 0; base < nR4; base += 256 * Q) {
      float4 v[Q];
#pragma unroll
      for (int q = 0; q < Q; ++q) v[q] = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int s0 = 0; s0 < a.S; s0 += SG) {
        float4 p[Q][SG];
#pragma unroll
        for (int q = 0; q < Q; ++q) {
          const int i4 = base + tid + 256 * q;
#pragma unroll
          for (int e = 0; e < SG; ++e)
            p[q][e] = (i4 < nR4 && s0 + e < a.S)
                          ? load4_coherent(rall, (uint32_t)((s0 + e) * split_bytes + 16u * i4))
                          : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int q = 0; q < Q; ++q)
#pragma unroll
          for (int e = 0; e < SG; ++e) {
            v[q].x += p[q][e].x; v[q].y += p[q][e].y; v[q].z += p[q][e].z; v[q].w += p[q][e].w;
          }
      }
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int i4 = base + tid + 256 * q;
        if (i4 < nR4) store4_coherent(rv, 16u * i4, v[q]);
      }
    }
  }
  // the two-launch apply hands v over at the kernel boundary
  if (a.two_pass) return;
  // atomic sums: this block's own ready word; ordered sums: the tile's one word
  publish_store(a.ready + (size_t)tau * kReadyPerTile + (a.atomic_sum ? s * kReadyStride : 0), a.epoch);
}

// Operands of one expand chunk (kNC columns of y for the tile's tokens) that a
// thread holds in registers: y and B_u slices of its (token, 8-column) items and
// the B_c^T operands of its wave's MFMA column blocks.
template <typename E, int MB, int RU, int NBM>
struct ExpandRegs {
  using Vec = typename Ops<E>::Vec;
  static constexpr int M = 16 * MB;
  static constexpr int CG = kNC / 8;            // 8-column groups per chunk
  static constexpr int ITEMS = M * CG / 256;    // (token, column group) items per thread
  static constexpr int RP = RU < 2 ? RU : 2;    // residual ranks held in registers
  static constexpr int NBW = kNC / 16 / 4;      // 16-column MFMA blocks per wave
  static constexpr int KS = (NBM + 1) / 2;      // 32-rank MFMA steps
  Vec yold[ITEMS];
  Vec bu[ITEMS][RP > 0 ? RP : 1];
  Vec bct[NBW][KS];

  // Unconditional loads: a row past the tile's tokens reads the tile's first
  // token, a column past out_dim reads column 0 and a residual rank past the
  // token's rank reads that token's y; none of those values is ever stored or
  // added.  Centroid ranks past r_c are zeroed: they meet zero v entries in the
  // MFMA, which must not see a non-finite table value.
  __device__ __forceinline__ void load(const ApplyArgs& a, const int4* s_tile, int n, bool has_c, int c, int n0) {
    using O = Ops<E>;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int out = a.out_dim, rc = a.r_c;
    const int tok0 = s_tile[1].x;
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int idx = tid + 256 * it, t = idx / CG, col = n0 + (idx % CG) * 8;
      const int4 tk = s_tile[1 + t];
      const bool ok = t < n;
      const int colc = col < out ? col : 0;
      const int ru = (ok && tk.y >= 0) ? tk.z : 0;
      const E* yp = reinterpret_cast<const E*>(a.y) + (size_t)(ok ? tk.x : tok0) * out + colc;
      yold[it] = O::load(yp);
      // rank-0 tokens read the first token's y row (a base the compiler cannot
      // merge with yp, which would make the y load wait)
      const E* slot_b = reinterpret_cast<const E*>(a.pool + (size_t)(tk.y > 0 ? tk.y : 0) * a.slot_stride) +
                        (int64_t)ru * (a.tab_prefix + a.in_dim) + colc;
      const E* bup = ru ? slot_b : reinterpret_cast<const E*>(a.y) + (size_t)tok0 * out + colc;
#pragma unroll
      for (int j = 0; j < RP; ++j) bu[it][j] = O::load(bup + (size_t)(j < ru ? j : 0) * out);
    }
    // without a centroid term the (zeroed) operands read the first token's y
    const E* bt = has_c ? reinterpret_cast<const E*>(a.cent_bt) + (size_t)c * out * rc : nullptr;
    const E* safe = reinterpret_cast<const E*>(a.y) + (size_t)tok0 * out;
#pragma unroll
    for (int w = 0; w < NBW; ++w) {
      const int col = n0 + (wave + 4 * w) * 16 + (lane & 15);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int j = ks * 32 + (lane >> 4) * 8;
        const Vec b = O::load(has_c ? bt + (size_t)(col < out ? col : 0) * rc + (j < rc ? j : 0) : safe);
        bct[w][ks] = (has_c && j < rc) ? b : O::zero();
      }
    }
  }

  __device__ __forceinline__ void pin() const {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      pin_regs(yold[it]);
#pragma unroll
      for (int j = 0; j < RP; ++j) pin_regs(bu[it][j]);
    }
#pragma unroll
    for (int w = 0; w < NBW; ++w)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) pin_regs(bct[w][ks]);
  }
};

// One chunk of an expand block: kNC columns of y for the tile's tokens, with
// the operands already in `regs`.  Leaves s_y free for the next chunk.
template <typename E, int MB, int RU, int NBM>
__device__ __forceinline__ void expand_chunk(const ApplyArgs& a, const ExpandRegs<E, MB, RU, NBM>& regs,
                                             const int4* s_tile, const float* s_v, float* s_y,
                                             const uint16_t* s_vh, const uint16_t* s_vl, int n, bool has_c,
                                             int n0) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  using Regs = ExpandRegs<E, MB, RU, NBM>;
  constexpr int CG = Regs::CG, ITEMS = Regs::ITEMS, RP = Regs::RP, NBW = Regs::NBW, KS = Regs::KS;
  constexpr int VS = expand_vs(NBM);
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int R = a.R, out = a.out_dim, rc = a.r_c, in = a.in_dim;
  // ---- centroid part on MFMA: y^T block [16 cols x 16 tokens] = B_c^T . v_c^T ----
  if (has_c) {
#pragma unroll
    for (int w = 0; w < NBW; ++w) {
      const int cb = (wave + 4 * w) * 16;       // first column of the block, local
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
        const int t = mb * 16 + (lane & 15);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int j = ks * 32 + (lane >> 4) * 8;
          if constexpr (sizeof(E) == 2) {
            const uint4 hi = *reinterpret_cast<const uint4*>(s_vh + t * VS + j);
            const uint4 lo = *reinterpret_cast<const uint4*>(s_vl + t * VS + j);
            acc = O::mma(regs.bct[w][ks], hi, acc);
            acc = O::mma(regs.bct[w][ks], lo, acc);
          } else {
            float vv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) vv[e] = (j + e < rc) ? s_v[t * R + j + e] : 0.f;
            acc = O::mma_f32rhs(regs.bct[w][ks], vv, acc);
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) s_y[t * kYS + cb + 4 * (lane >> 4) + e] = acc[e];
      }
    }
  }
  __syncthreads();

  // ---- residual part, add, round, store (lanes with nothing to write store
  // to the sink, so that every path issues the same stores) ----
  if constexpr (RU <= RP) {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int idx = tid + 256 * it, t = idx / CG, cl = (idx % CG) * 8, col = n0 + cl;
      const bool ok = t < n && col < out;
      const int4 tk = s_tile[1 + t];
      const int ru = tk.y >= 0 ? tk.z : 0;
      float accv[8], yv[8];
      if (has_c) {
#pragma unroll
        for (int e = 0; e < 8; ++e) accv[e] = s_y[t * kYS + cl + e];
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) accv[e] = 0.f;
      }
      const float* vt = s_v + t * R + rc;
      // the ranks come from the registers loaded ahead
#pragma unroll
      for (int j = 0; j < RP; ++j) {
        if (j < ru) {
          float b8[8];
          O::to_f32(regs.bu[it][j], b8);
          const float vj = vt[j];
#pragma unroll
          for (int e = 0; e < 8; ++e) accv[e] = fmaf(vj, b8[e], accv[e]);
        }
      }
      O::to_f32(regs.yold[it], yv);
#pragma unroll
      for (int e = 0; e < 8; ++e) yv[e] += accv[e];
      E* dst = ok ? reinterpret_cast<E*>(a.y) + (size_t)tk.x * out + col : reinterpret_cast<E*>(a.sink + tid * 32);
      O::store(dst, yv);
    }
  } else {
    float accv[ITEMS][8];
    int ruv[ITEMS];
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int idx = tid + 256 * it, t = idx / CG, cl = (idx % CG) * 8;
      const int4 tk = s_tile[1 + t];
      const int ru = tk.y >= 0 ? tk.z : 0;
      ruv[it] = ru;
      if (has_c) {
#pragma unroll
        for (int e = 0; e < 8; ++e) accv[it][e] = s_y[t * kYS + cl + e];
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) accv[it][e] = 0.f;
      }
      const float* vt = s_v + t * R + rc;
      // the first RP ranks come from the registers loaded ahead
#pragma unroll
      for (int j = 0; j < RP; ++j) {
        if (j < ru) {
          float b8[8];
          O::to_f32(regs.bu[it][j], b8);
          const float vj = vt[j];
#pragma unroll
          for (int e = 0; e < 8; ++e) accv[it][e] = fmaf(vj, b8[e], accv[it][e]);
        }
      }
    }
    // the rest (any rank up to r_u_max) straight from the slots: QN rows of
    // every item of the thread in flight at a time.  A row past a token's rank
    // re-reads its last row and is not added; a token without ranks past RP
    // reads its first row of B (any rank >= 1) or the tile's first y row, and a
    // column past out_dim reads column 0.
    constexpr int QN = ITEMS >= 2 ? 8 : 16;
    const E* bup[ITEMS];
    int rmax = 0;
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int idx = tid + 256 * it, t = idx / CG, col = n0 + (idx % CG) * 8;
      const int4 tk = s_tile[1 + t];
      const int ru = ruv[it], colc = col < out ? col : 0;
      bup[it] = ru ? reinterpret_cast<const E*>(a.pool + (size_t)(tk.y > 0 ? tk.y : 0) * a.slot_stride) +
                         (int64_t)ru * (a.tab_prefix + in) + colc
                   : reinterpret_cast<const E*>(a.y) + (size_t)s_tile[1].x * out + colc;
      rmax = max(rmax, ru);
    }
    for (int j0 = RP; j0 < rmax; j0 += QN) {
      Vec bv[ITEMS][QN];
#pragma unroll
      for (int it = 0; it < ITEMS; ++it) {
        const int last = ruv[it] > 0 ? ruv[it] - 1 : 0;
#pragma unroll
        for (int q = 0; q < QN; ++q) bv[it][q] = O::load(bup[it] + (size_t)(j0 + q < last ? j0 + q : last) * out);
      }
#pragma unroll
      for (int it = 0; it < ITEMS; ++it) {
        const int idx = tid + 256 * it, t = idx / CG;
        const float* vt = s_v + t * R + rc;
#pragma unroll
        for (int q = 0; q < QN; ++q) {
          if (j0 + q < ruv[it]) {
            float b8[8];
            O::to_f32(bv[it][q], b8);
            const float vj = vt[j0 + q];
#pragma unroll
            for (int e = 0; e < 8; ++e) accv[it][e] = fmaf(vj, b8[e], accv[it][e]);
          }
        }
      }
    }

#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int idx = tid + 256 * it, t = idx / CG, col = n0 + (idx % CG) * 8;
      const bool ok = t < n && col < out;
      float yv[8];
      O::to_f32(regs.yold[it], yv);
#pragma unroll
      for (int e = 0; e < 8; ++e) yv[e] += accv[it][e];
      E* dst = ok ? reinterpret_cast<E*>(a.y) + (size_t)s_tile[1 + t].x * out + col
                  : reinterpret_cast<E*>(a.sink + tid * 32);
      O::store(dst, yv);
    }
  }
  __syncthreads();                              // s_y consumed
}

// Expand block: tile `tau`, column chunks [q * cpb, q * cpb + cpb) of kNC
// columns each.  Two register sets alternate between chunks: the first two
// chunks' operands are loaded before the wait for v, and chunk k + 2 loads
// while chunk k + 1 is computed.
template <typename E, int MB, int RU, int NBM>
__device__ __forceinline__ void expand_block(const ApplyArgs& a, int tau, int q, char* lds) {
  using Regs = ExpandRegs<E, MB, RU, NBM>;
  constexpr int M = Regs::M, KS = Regs::KS, VS = expand_vs(NBM);
  int4* s_tile = reinterpret_cast<int4*>(lds);
  float* s_v = reinterpret_cast<float*>(lds + tile_bytes(M));     // [M][R]
  float* s_y = s_v + (size_t)M * a.R;                             // [M][kYS]
  // bf16: hi and lo halves of the centroid part of v, [M][VS] each, built once
  uint16_t* s_vh = reinterpret_cast<uint16_t*>(s_y + (size_t)M * kYS);
  uint16_t* s_vl = s_vh + (size_t)M * VS;
  __shared__ int s_flag;
  const int tid = threadIdx.x;
  const int i0 = __builtin_amdgcn_readfirstlane(s_tile[0].x), n = __builtin_amdgcn_readfirstlane(s_tile[0].y),
            c = __builtin_amdgcn_readfirstlane(s_tile[0].z);   // tile header: uniform
  const int R = a.R, out = a.out_dim, rc = a.r_c;
  const bool has_c = c >= 0 && rc > 0;
  const int chunk0 = q * a.cpb;
  const int nch = min(a.cpb, (out + kNC - 1) / kNC - chunk0);   // chunks of this block, >= 1
  // operands of chunk k; a prefetch past the block's last chunk re-reads it
  auto n0_of = [&](int k) { return (chunk0 + (k < nch ? k : nch - 1)) * kNC; };

  Regs ra, rb;
  const int nR4 = n * R / 4, MR4 = M * R / 4;
  if (a.two_pass) {
    // two-launch apply: v is complete (kernel boundary).  Its loads go out
    // first and the first two chunks' operands right behind them, so that
    // filling s_v waits only for v.
    constexpr int VQ = (M * padded_rank(16 * NBM, 2) / 4 + 255) / 256;   // float4s of v per thread
    float4 vv[VQ];
    if (a.atomic_sum) {
      const float4* pv = reinterpret_cast<const float4*>(a.v + (size_t)i0 * R);
#pragma unroll
      for (int k = 0; k < VQ; ++k) {
        const int i4 = tid + 256 * k;
        vv[k] = i4 < nR4 ? pv[i4] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    } else {
      // ordered sums: the shrink launch's K-range partials, added in K order
      const size_t split = (size_t)a.T * R / 4;   // float4s between K ranges
      const float4* p = reinterpret_cast<const float4*>(a.partials + (size_t)i0 * R);
#pragma unroll
      for (int k = 0; k < VQ; ++k) {
        const int i4 = tid + 256 * k;
        vv[k] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (i4 < nR4)
          for (int q = 0; q < a.S; ++q) {
            const float4 t4 = p[(size_t)q * split + i4];
            vv[k].x += t4.x; vv[k].y += t4.y; vv[k].z += t4.z; vv[k].w += t4.w;
          }
      }
    }
    ra.load(a, s_tile, n, has_c, c, n0_of(0));
    if (nch > 1) rb.load(a, s_tile, n, has_c, c, n0_of(1));
#pragma unroll
    for (int k = 0; k < VQ; ++k) {
      const int i4 = tid + 256 * k;
      if (i4 < MR4) reinterpret_cast<float4*>(s_v)[i4] = scale_centroid(vv[k], 4 * i4, R, rc, s_tile);
    }
  } else {
    ra.load(a, s_tile, n, has_c, c, n0_of(0));
    if (nch > 1) rb.load(a, s_tile, n, has_c, c, n0_of(1));
    ra.pin();
    if (nch > 1) rb.pin();
    // ---- wait for the tile's v: the S ready words (atomic sums) or the one word ----
    const bool ok = await_words(a.ready + (size_t)tau * kReadyPerTile, a.atomic_sum ? a.S : 1, a.epoch,
                                a.meta + kMetaErr, &s_flag);
    if (!ok) return;
    const __amdgpu_buffer_rsrc_t rv = coherent_rsrc(a.v + (size_t)i0 * R, (uint32_t)(nR4 * 16));
    for (int i4 = tid; i4 < MR4; i4 += 256)   // past n rows: zeros
      reinterpret_cast<float4*>(s_v)[i4] = scale_centroid(load4_coherent(rv, 16u * i4), 4 * i4, R, rc, s_tile);
  }
  __syncthreads();
  if constexpr (sizeof(E) == 2) {
    // v_c = hi + lo, both bf16 (hi = rne(v), lo = rne(v - hi)): about 16
    // significant bits of v reach the MFMA; ranks past r_c are zero
    for (int i = tid; i < M * KS * 32; i += 256) {
      const int t = i / (KS * 32), j = i - t * (KS * 32);
      const float v = j < rc ? s_v[t * R + j] : 0.f;
      const uint32_t h = f32_to_bf16_rne(v);
      s_vh[t * VS + j] = (uint16_t)h;
      s_vl[t * VS + j] = (uint16_t)f32_to_bf16_rne(v - __uint_as_float(h << 16));
    }
    __syncthreads();
  }

  // pairs of chunks while the next two exist (no conditional memory operation
  // inside the loop), then the last one to three chunks (ra holds chunk cc,
  // rb chunk cc + 1)
  int cc = 0;
  for (; cc + 3 < nch; cc += 2) {
    expand_chunk(a, ra, s_tile, s_v, s_y, s_vh, s_vl, n, has_c, (chunk0 + cc) * kNC);
    ra.load(a, s_tile, n, has_c, c, n0_of(cc + 2));
    expand_chunk(a, rb, s_tile, s_v, s_y, s_vh, s_vl, n, has_c, (chunk0 + cc + 1) * kNC);
    rb.load(a, s_tile, n, has_c, c, n0_of(cc + 3));
  }
  const int rem = nch - cc;
  expand_chunk(a, ra, s_tile, s_v, s_y, s_vh, s_vl, n, has_c, (chunk0 + cc) * kNC);
  if (rem == 3) ra.load(a, s_tile, n, has_c, c, n0_of(cc + 2));
  if (rem >= 2) expand_chunk(a, rb, s_tile, s_v, s_y, s_vh, s_vl, n, has_c, (chunk0 + cc + 1) * kNC);
  if (rem == 3) expand_chunk(a, ra, s_tile, s_v, s_y, s_vh, s_vl, n, has_c, (chunk0 + cc + 2) * kNC);
}

// The plan a launch builds for itself, written out by its first block.
template <int CAP>
__device__ __forceinline__ void write_plan(const ApplyArgs& a, int M, PlanLds<CAP>& L) {
  plan_sort(a.pb.maps, a.T, L);
  for (int i = threadIdx.x; i < a.T; i += 256) {
    a.pb.perm[i] = L.srt[i].x;
    a.pb.srt[i] = L.srt[i];
    a.pb.srt_c[i] = L.c[i];
  }
  plan_groups(true, a.pb, L.srt, L.c, a.T, M, L.sh);
  plan_write_tiles(a.pb, L.srt, a.T, M, L.sh);
}

template <typename E, int MB, int RU, int NBM>
__global__ void __launch_bounds__(256) k_apply(ApplyArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  constexpr int M = 16 * MB;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int n_shrink = a.n_tiles * a.S;
  const bool shrink = b < n_shrink;
  const int tau = (shrink ? b : b - n_shrink) % a.n_tiles;
  int4* s_tile = reinterpret_cast<int4*>(lds);
  if (a.fused_plan) {
    // This launch also builds the plan (batches of up to kPlanFusedT tokens).
    // One extra block, the last, sorts the whole batch and writes the plan out
    // for later applies and plan queries; every other block cuts its own tile
    // from the maps.
    if (b == a.writer) {
      write_plan(a, M, *reinterpret_cast<PlanLds<kPlanFusedT>*>(lds));
      return;
    }
    auto& L = *reinterpret_cast<TileLds*>(lds + tile_bytes(M));
    if (!tile_from_maps(a.maps, a.T, M, tau, a.n_tiles, L, s_tile)) {
      if (tid == 0) atomicAdd(a.meta + kMetaErr, 1);   // cannot happen: the host counts the same tiles
      return;
    }
  } else {
    const int4* trec = a.tiles + (size_t)tau * (M + 1);
    for (int k = tid; k < M + 1; k += 256) s_tile[k] = trec[k];
    __syncthreads();
  }
  if (shrink) shrink_block<E, MB, 1, RU, NBM>(a, tau, b / a.n_tiles, lds);
  else expand_block<E, MB, RU, NBM>(a, tau, (b - n_shrink) / a.n_tiles, lds);
}

// The two-launch apply of large batches (tiles of kTwoPassM tokens).  The
// shrink launch: one block per (tile, K range); wave w covers M-block w over
// the whole K range, x and A_c staged through LDS.  Block ids run over tiles
// first.
template <typename E, int MB, int RU, int NBM>
__global__ void __launch_bounds__(256) k_shrink(ApplyArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  constexpr int M = 16 * MB;
  const int b = blockIdx.x, tau = b % a.n_tiles;
  int4* s_tile = reinterpret_cast<int4*>(lds);
  const int4* trec = a.tiles + (size_t)tau * (M + 1);
  for (int k = threadIdx.x; k < M + 1; k += 256) s_tile[k] = trec[k];
  __syncthreads();
  shrink_block<E, MB, 1, RU, NBM, true>(a, tau, b / a.n_tiles, lds);
}

// The expand launch: one block per (tile, range of cpb column chunks).
template <typename E, int MB, int RU, int NBM>
__global__ void __launch_bounds__(256) k_expand(ApplyArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  constexpr int M = 16 * MB;
  const int b = blockIdx.x, tau = b % a.n_tiles;
  int4* s_tile = reinterpret_cast<int4*>(lds);
  const int4* trec = a.tiles + (size_t)tau * (M + 1);
  for (int k = threadIdx.x; k < M + 1; k += 256) s_tile[k] = trec[k];
  __syncthreads();
  expand_block<E, MB, RU, NBM>(a, tau, b / a.n_tiles, lds);
}

// LDS of the block roles.  Shrink: tile records + the per-wave partials
// [KW][M][R] (KW * M = 64 in the single launch, 4 * M in the two-launch one).
size_t lds_shrink(int M, int R, int kw_m) {
  return (size_t)tile_bytes(M) + sizeof(float) * (size_t)kw_m * R;
}
// Two-launch shrink: tile records, partials [M][R], two staging buffers.
template <int NBM>
size_t lds_shrink_staged(int R) {
  return lds_shrink(kTwoPassM, R, kTwoPassM) + 2 * (size_t)stage_bytes<NBM>();
}
// Expand: tile records, v [M][R], the MFMA output [M][kYS] and the bf16 hi/lo
// copies of v's centroid part [2][M][VS].
size_t lds_expand(int M, int R, int nbm) {
  return (size_t)tile_bytes(M) + sizeof(float) * ((size_t)M * R + (size_t)M * kYS) +
         2 * sizeof(uint16_t) * (size_t)M * expand_vs(nbm);
}
// Single launch; fused_T: batch size of a launch that builds its plan, else 0.
size_t apply_lds(int M, int R, int nbm, int fused_T) {
  const size_t plan = fused_T > 0 ? std::max(sizeof(PlanLds<kPlanFusedT>), tile_bytes(M) + sizeof(TileLds)) : 0;
  return std::max({lds_shrink(M, R, 64), lds_expand(M, R, nbm), plan});
}

// A launch; with events, they record the kernel's own start and end.
template <typename K, typename Args>
void launch_k(K kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s, const Args& a, hipEvent_t e0,
              hipEvent_t e1) {
  if (e0 || e1) hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, s, e0, e1, 0u, a);
  else hipLaunchKernelGGL(kernel, grid, block, lds, s, a);
}

template <typename E, int RU, int NBM>
hipError_t launch_nbm(const ApplyArgs& a, int M, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.two_pass) {
    // shrink launch, then expand launch; the events bracket both
    if constexpr (sizeof(E) == 2 && RU <= 2) {
      if (M != kTwoPassM) return hipErrorInvalidValue;
      constexpr int MB = kTwoPassM / 16;
      launch_k(k_shrink<E, MB, RU, NBM>, dim3(a.n_tiles * a.S), dim3(256), lds_shrink_staged<NBM>(a.R), s, a, e0,
               nullptr);
      launch_k(k_expand<E, MB, RU, NBM>, dim3(a.n_tiles * a.n_col), dim3(256), lds_expand(M, a.R, NBM), s, a,
               nullptr, e1);
      return hipGetLastError();
    } else {
      return hipErrorInvalidValue;
    }
  }
  // n_col: column blocks of cpb chunks; one more block, the last, writes a plan
  // built in this launch
  const dim3 grid(a.n_tiles * (a.S + a.n_col) + a.fused_plan), block(256);
  const size_t lds = apply_lds(M, a.R, NBM, a.fused_plan ? a.T : 0);
  if (M == 16) {
    launch_k(k_apply<E, 1, RU, NBM>, grid, block, lds, s, a, e0, e1);
  } else if constexpr (sizeof(E) == 2) {
    if (M == 32) launch_k(k_apply<E, 2, RU, NBM>, grid, block, lds, s, a, e0, e1);
    else return hipErrorInvalidValue;
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// NBM: 16-rank blocks of the centroid held per lane (r_c <= 16 * NBM)
template <typename E, int RU>
hipError_t launch_typed(const ApplyArgs& a, int M, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  switch (centroid_blocks(a.r_c)) {
    case 2: return launch_nbm<E, RU, 2>(a, M, s, e0, e1);
    case 4: return launch_nbm<E, RU, 4>(a, M, s, e0, e1);
    default: return launch_nbm<E, RU, 8>(a, M, s, e0, e1);
  }
}

template <int RU, int NBM>
hipError_t two_pass_occ(int R, int* shrink_per_cu, int* expand_per_cu) {
  constexpr int MB = kTwoPassM / 16;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
      shrink_per_cu, reinterpret_cast<const void*>(k_shrink<uint16_t, MB, RU, NBM>), 256,
      lds_shrink_staged<NBM>(R));
  if (e != hipSuccess) return e;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(
      expand_per_cu, reinterpret_cast<const void*>(k_expand<uint16_t, MB, RU, NBM>), 256,
      lds_expand(kTwoPassM, R, NBM));
}


// ---------------------------------------------------------------------------
// centroid fused into a base weight
// ---------------------------------------------------------------------------
// Raw elements of an operand vector (8 per lane).
__device__ __forceinline__ void vec_elems(const uint4& v, uint16_t (&e)[8]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int k = 0; k < 8; ++k) e[k] = (uint16_t)(w[k >> 1] >> (16 * (k & 1)));
}
__device__ __forceinline__ void vec_elems(const Ops<float>::Vec& v, float (&e)[8]) {
  e[0] = v.lo.x; e[1] = v.lo.y; e[2] = v.lo.z; e[3] = v.lo.w;
  e[4] = v.hi.x; e[5] = v.hi.y; e[6] = v.hi.z; e[7] = v.hi.w;
}

constexpr int kFuseTI = 64, kFuseTO = 128, kFuseDS = kFuseTO + 4;
// Row stride (elements) of the transposed A_c tile: 32 * KS ranks + 8 of padding.
__host__ __device__ constexpr int fuse_rp(int ks) { return 32 * ks + 8; }
size_t fuse_lds(int ks, int esize) {
  return std::max((size_t)kFuseTI * fuse_rp(ks) * esize, sizeof(float) * kFuseTI * kFuseDS);
}

// W[i][o] <- rne(W[i][o] + gamma * sum_r A_c[i][r] B_c[r][o]) over a 64 x 128
// tile of W (in rows i, out columns o).  The rank-r_c product is an MFMA
// contraction over the ranks: D[o][i] = sum_r Bt_c[o][r] At_c[r][i], with the
// rows of Bt_c (8 consecutive ranks per lane) read straight from the pinned
// transposed B and At_c's columns taken from an LDS copy of the tile transposed
// to [i][r].  The fp32 delta goes through LDS so that W is read and written in
// whole rows, once, with one rounding.
template <typename E, int KS>
__global__ void __launch_bounds__(256) k_fuse(FuseArgs f) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  constexpr int TI = kFuseTI, TO = kFuseTO, DS = kFuseDS, RP = fuse_rp(KS);
  extern __shared__ __attribute__((aligned(16))) char lds[];
  E* s_a = reinterpret_cast<E*>(lds);            // [TI][RP]: A_c[i][r], ranks past r_c zero
  float* s_d = reinterpret_cast<float*>(lds);    // [TI][DS] delta, after s_a is consumed
  const int i0 = blockIdx.x * TI, o0 = blockIdx.y * TO;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4;
  const int in = f.in_dim, out = f.out_dim, rc = f.r_c;
  const E* at = reinterpret_cast<const E*>(f.at);   // [r_c][in] of the centroid
  const E* bt = reinterpret_cast<const E*>(f.bt);   // [out][r_c]

  for (int k = tid; k < 32 * KS * (TI / 8); k += 256) {
    const int r = k / (TI / 8), i8 = (k % (TI / 8)) * 8;
    E e[8];
    if (r < rc && i0 + i8 < in) {
      vec_elems(O::load(at + (size_t)r * in + i0 + i8), e);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) e[q] = E(0);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) s_a[(i8 + q) * RP + r] = e[q];
  }
  __syncthreads();

  f32x4 acc[2][4];
#pragma unroll
  for (int ob = 0; ob < 2; ++ob)
#pragma unroll
    for (int ib = 0; ib < 4; ++ib) acc[ob][ib] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int r8 = 32 * ks + 8 * g;               // this lane's 8 ranks (r_c is a multiple of 8)
    Vec bfr[2];
#pragma unroll
    for (int ob = 0; ob < 2; ++ob) {
      const int o = o0 + 32 * wave + 16 * ob + (lane & 15);
      bfr[ob] = (o < out && r8 < rc) ? O::load(bt + (size_t)o * rc + r8) : O::zero();
    }
#pragma unroll
    for (int ib = 0; ib < 4; ++ib) {
      const Vec afr = *reinterpret_cast<const Vec*>(s_a + (16 * ib + (lane & 15)) * RP + r8);
#pragma unroll
      for (int ob = 0; ob < 2; ++ob) acc[ob][ib] = O::mma(bfr[ob], afr, acc[ob][ib]);
    }
  }
  __syncthreads();                                // s_a consumed; s_d reuses it
  // D[o][i]: lane holds o = 4g + e (of its 16-row block), i = lane & 15
#pragma unroll
  for (int ob = 0; ob < 2; ++ob)
#pragma unroll
    for (int ib = 0; ib < 4; ++ib)
      *reinterpret_cast<float4*>(s_d + (16 * ib + (lane & 15)) * DS + 32 * wave + 16 * ob + 4 * g) =
          make_float4(acc[ob][ib][0], acc[ob][ib][1], acc[ob][ib][2], acc[ob][ib][3]);
  __syncthreads();

  for (int k = tid; k < TI * (TO / 8); k += 256) {
    const int i = k / (TO / 8), o8 = (k % (TO / 8)) * 8;
    if (i0 + i >= in || o0 + o8 >= out) continue;
    E* w = reinterpret_cast<E*>(f.w) + (size_t)(i0 + i) * f.ldw + o0 + o8;
    float v[8];
    O::to_f32(O::load(w), v);
    const float4 d0 = *reinterpret_cast<const float4*>(s_d + i * DS + o8);
    const float4 d1 = *reinterpret_cast<const float4*>(s_d + i * DS + o8 + 4);
    v[0] += f.gamma * d0.x; v[1] += f.gamma * d0.y; v[2] += f.gamma * d0.z; v[3] += f.gamma * d0.w;
    v[4] += f.gamma * d1.x; v[5] += f.gamma * d1.y; v[6] += f.gamma * d1.z; v[7] += f.gamma * d1.w;
    O::store(w, v);
  }
}

// ---------------------------------------------------------------------------
// adapter Gram products (matrix cosine in factor space)
// ---------------------------------------------------------------------------
// One block per work item: table t = blockIdx.y, factor side (0: the At
// factors, contracted over in; 1: the B factors, contracted over out), K chunk
// q of kGramKC elements (blockIdx.x over both sides; blocks past the table's
// chunks return at once).  The block adds the chunk's part of the three Gram
// matrices X1 X2^T, X1 X1^T and X2 X2^T (X = the side's [r][K] factors, rows
// padded to 16 with zeros) into g with fp32 atomics.  Each 16 x 16 tile is an
// MFMA contraction over K: both operands are 16 rank rows with 8 consecutive k
// per lane.  With both ranks <= 16 * NB (NB = 1, 2) every wave takes a quarter
// of the chunk's 32-wide steps for all tiles, loading each rank block's
// fragment once per step, and the four waves' tiles are summed in LDS before
// the atomics; otherwise (NB = 0) the waves split the tiles.
constexpr int kGramKC = 2048;

template <int NB>
__host__ __device__ constexpr int gram_lds() { return NB > 0 ? 4 * 3 * NB * NB * 256 * 4 : 0; }

template <typename E, int NB>
__global__ void __launch_bounds__(256) k_gram(GramArgs a) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  const int t = blockIdx.y, local = blockIdx.x;
  const GramTable tab = a.tabs[t];
  const int nq_in = (tab.in_dim + kGramKC - 1) / kGramKC, nq_out = (tab.out_dim + kGramKC - 1) / kGramKC;
  if (local >= nq_in + nq_out) return;
  const int side = local < nq_in ? 0 : 1;
  const int q = side == 0 ? local : local - nq_in;
  const int K = side == 0 ? tab.in_dim : tab.out_dim;
  const int k0 = q * kGramKC, kend = min(K, k0 + kGramKC);
  const E* x1 = reinterpret_cast<const E*>(side == 0 ? tab.at1 : tab.b1);
  const E* x2 = reinterpret_cast<const E*>(side == 0 ? tab.at2 : tab.b2);
  const int r1 = a.r1, r2 = a.r2, nb1 = (r1 + 15) / 16, nb2 = (r2 + 15) / 16;
  float* g = a.g + (size_t)t * a.g_table + (size_t)side * a.g_side;
  // tiles: [0, nb1 * nb2) of G12, then nb1 * nb1 of G11, then nb2 * nb2 of G22
  const int n12 = nb1 * nb2, n11 = nb1 * nb1, ntile = n12 + n11 + nb2 * nb2;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g8 = lane >> 4;
  // where tile `tile` goes: its Gram, its rank blocks, the Gram's row length
  auto place = [&](int tile, float*& gt, int& ba, int& bb, int& ldg) {
    if (tile < n12) {
      ba = tile / nb2; bb = tile % nb2; ldg = nb2 * 16; gt = g;
    } else if (tile < n12 + n11) {
      const int u = tile - n12;
      ba = u / nb1; bb = u % nb1; ldg = nb1 * 16; gt = g + a.g_12;
    } else {
      const int u = tile - n12 - n11;
      ba = u / nb2; bb = u % nb2; ldg = nb2 * 16; gt = g + a.g_12 + a.g_11;
    }
  };
  if constexpr (NB > 0) {
    constexpr int NT = 3 * NB * NB;
    extern __shared__ __attribute__((aligned(16))) char lds[];
    float* s_red = reinterpret_cast<float*>(lds);   // [4 waves][NT][256]
    f32x4 acc[NT];
#pragma unroll
    for (int u = 0; u < NT; ++u) acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int k = k0 + 32 * wave; k < kend; k += 128) {
      const int kk = k + 8 * g8;                     // K is a multiple of 8: a lane's 8 are all in or all out
      const bool kin = kk < kend;
      Vec f1[NB], f2[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int i1 = b * 16 + (lane & 15);
        f1[b] = (kin && i1 < r1) ? O::load(x1 + (size_t)i1 * K + kk) : O::zero();
        f2[b] = (kin && i1 < r2) ? O::load(x2 + (size_t)i1 * K + kk) : O::zero();
      }
#pragma unroll
      for (int b1 = 0; b1 < NB; ++b1)
#pragma unroll
        for (int b2 = 0; b2 < NB; ++b2) {
          acc[b1 * NB + b2] = O::mma(f1[b1], f2[b2], acc[b1 * NB + b2]);
          acc[NB * NB + b1 * NB + b2] = O::mma(f1[b1], f1[b2], acc[NB * NB + b1 * NB + b2]);
          acc[2 * NB * NB + b1 * NB + b2] = O::mma(f2[b1], f2[b2], acc[2 * NB * NB + b1 * NB + b2]);
        }
    }
    // lane holds rows 4 g8 + e, column lane & 15 of each tile
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) s_red[((size_t)wave * NT + u) * 256 + (4 * g8 + e) * 16 + (lane & 15)] = acc[u][e];
    __syncthreads();
    for (int i = threadIdx.x; i < NT * 256; i += 256) {
      const int u = i / 256, rc16 = i % 256;
      const int gram = u / (NB * NB), b1 = (u % (NB * NB)) / NB, b2 = u % NB;
      const int na = gram == 2 ? nb2 : nb1, nbb = gram == 0 ? nb2 : (gram == 1 ? nb1 : nb2);
      if (b1 >= na || b2 >= nbb) continue;                 // rank blocks this call does not have
      const int tile = gram == 0 ? b1 * nb2 + b2 : (gram == 1 ? n12 + b1 * nb1 + b2 : n12 + n11 + b1 * nb2 + b2);
      float* gt;
      int ba, bb, ldg;
      place(tile, gt, ba, bb, ldg);
      const float v = s_red[(size_t)u * 256 + rc16] + s_red[((size_t)NT + u) * 256 + rc16] +
                      s_red[((size_t)2 * NT + u) * 256 + rc16] + s_red[((size_t)3 * NT + u) * 256 + rc16];
      atomicAdd(gt + (size_t)(ba * 16 + rc16 / 16) * ldg + bb * 16 + rc16 % 16, v);
    }
  } else {
    for (int tile = wave; tile < ntile; tile += 4) {
      float* gt;
      int ba, bb, ldg;
      place(tile, gt, ba, bb, ldg);
      const E* xa = tile < n12 + n11 ? x1 : x2;
      const E* xb = tile < n12 ? x2 : (tile < n12 + n11 ? x1 : x2);
      const int ra = tile < n12 + n11 ? r1 : r2;
      const int rb = tile < n12 ? r2 : (tile < n12 + n11 ? r1 : r2);
      const int ia = ba * 16 + (lane & 15), ib = bb * 16 + (lane & 15);
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int k = k0; k < kend; k += 32) {
        const int kk = k + 8 * g8;
        const bool kin = kk < kend;
        const Vec va = (kin && ia < ra) ? O::load(xa + (size_t)ia * K + kk) : O::zero();
        const Vec vb = (kin && ib < rb) ? O::load(xb + (size_t)ib * K + kk) : O::zero();
        acc = O::mma(va, vb, acc);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) atomicAdd(gt + (size_t)(ba * 16 + 4 * g8 + e) * ldg + ib, acc[e]);
    }
  }
}

// Per table: sum of the elementwise products of the At-side and B-side Grams,
// in float64: Tr(dW1^T dW2), ||dW1||_F^2, ||dW2||_F^2.
__global__ void __launch_bounds__(256) k_gram_finish(GramArgs a) {
  const int t = blockIdx.x;
  const float* gA = a.g + (size_t)t * a.g_table;
  const float* gB = gA + a.g_side;
  const int sizes[3] = {a.g_12, a.g_11, a.g_22};
  const int offs[3] = {0, a.g_12, a.g_12 + a.g_11};
  __shared__ double s_red[3][4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int m = 0; m < 3; ++m) {
    double acc = 0.0;
    for (int i = threadIdx.x; i < sizes[m]; i += 256) acc += (double)gA[offs[m] + i] * (double)gB[offs[m] + i];
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_down(acc, off);
    if (lane == 0) s_red[m][wave] = acc;
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    const int m = threadIdx.x;
    a.out[3 * t + m] = s_red[m][0] + s_red[m][1] + s_red[m][2] + s_red[m][3];
  }
}

template <typename E>
hipError_t launch_gram_t(const GramArgs& a, int max_items, hipStream_t s) {
  const dim3 grid(max_items, a.n_tables), block(256);
  const int r = a.r1 > a.r2 ? a.r1 : a.r2;
  if (r <= 16) hipLaunchKernelGGL((k_gram<E, 1>), grid, block, gram_lds<1>(), s, a);
  else if (r <= 32) hipLaunchKernelGGL((k_gram<E, 2>), grid, block, gram_lds<2>(), s, a);
  else hipLaunchKernelGGL((k_gram<E, 0>), grid, block, 0, s, a);
  hipLaunchKernelGGL(k_gram_finish, dim3(a.n_tables), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename E>
hipError_t launch_fuse_t(const FuseArgs& f, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid((f.in_dim + kFuseTI - 1) / kFuseTI, (f.out_dim + kFuseTO - 1) / kFuseTO), block(256);
  const int ks = (f.r_c + 31) / 32;
  const size_t lds = fuse_lds(ks, (int)sizeof(E));
  switch (ks) {
    case 1: launch_k(k_fuse<E, 1>, grid, block, lds, s, f, e0, e1); break;
    case 2: launch_k(k_fuse<E, 2>, grid, block, lds, s, f, e0, e1); break;
    case 3: launch_k(k_fuse<E, 3>, grid, block, lds, s, f, e0, e1); break;
    case 4: launch_k(k_fuse<E, 4>, grid, block, lds, s, f, e0, e1); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
}  // namespace

// Blocks of the two-launch apply's kernels that one compute unit holds at once.
hipError_t two_pass_occupancy(int r_c, int r_u_max, int R, int* shrink_per_cu, int* expand_per_cu) {
  const int nbm = centroid_blocks(r_c);
  if (r_u_max <= 1) {
    if (nbm == 2) return two_pass_occ<1, 2>(R, shrink_per_cu, expand_per_cu);
    if (nbm == 4) return two_pass_occ<1, 4>(R, shrink_per_cu, expand_per_cu);
    return two_pass_occ<1, 8>(R, shrink_per_cu, expand_per_cu);
  }
  if (nbm == 2) return two_pass_occ<2, 2>(R, shrink_per_cu, expand_per_cu);
  if (nbm == 4) return two_pass_occ<2, 4>(R, shrink_per_cu, expand_per_cu);
  return two_pass_occ<2, 8>(R, shrink_per_cu, expand_per_cu);
}

// Per-device set-up: checks that the device has the LDS the apply kernels may
// ask for (gfx950: 160 KiB per workgroup; dynamic LDS needs no opt-in on AMD).
hipError_t kernels_init(int device) {
  static bool done[64] = {};
  if (device < 0 || device >= 64) return hipErrorInvalidDevice;
  if (done[device]) return hipSuccess;
  int lds_max = 0;
  hipError_t e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, device);
  if (e != hipSuccess) return e;
  const size_t need = std::max({apply_lds(32, padded_rank(kMaxRc, kMaxRu), 8, kPlanFusedT),
                                lds_shrink_staged<8>(padded_rank(kMaxRc, 2)),
                                lds_expand(kTwoPassM, padded_rank(kMaxRc, 2), 8)});
  if ((size_t)lds_max < need + 1024) return hipErrorInvalidConfiguration;
  done[device] = true;
  return hipSuccess;
}

hipError_t launch_plan(const PlanArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  if (a.T <= kPlanSmallT) {
    hipLaunchKernelGGL(k_plan_small, dim3(1), dim3(kPlanSmallThreads), 0, s, a);
  } else {
    const int blocks = (a.T + kPlanTokPerBlock - 1) / kPlanTokPerBlock;
    hipLaunchKernelGGL(k_plan_large, dim3(blocks), dim3(kPlanThreads), 0, s, a);
  }
  return hipGetLastError();
}

// RU: residual ranks held per lane (1, 2 or kRankChunk; larger ranks in chunks).  fp32 plans use 16-token
// tiles only.
hipError_t launch_apply(const ApplyArgs& a, int bf16, int M, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.T <= 0 || a.n_tiles <= 0) return hipSuccess;
  if (!bf16) {
    if (M != 16) return hipErrorInvalidValue;
    if (a.r_u_max <= 1) return launch_typed<float, 1>(a, M, s, e0, e1);
    if (a.r_u_max <= 2) return launch_typed<float, 2>(a, M, s, e0, e1);
    return launch_typed<float, kRankChunk>(a, M, s, e0, e1);
  }
  if (a.r_u_max <= 1) return launch_typed<uint16_t, 1>(a, M, s, e0, e1);
  if (a.r_u_max <= 2) return launch_typed<uint16_t, 2>(a, M, s, e0, e1);
  return launch_typed<uint16_t, kRankChunk>(a, M, s, e0, e1);
}

hipError_t launch_fuse(const FuseArgs& f, int bf16, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (f.r_c < 8 || f.r_c > kMaxRc || f.r_c % 8 || f.in_dim <= 0 || f.out_dim <= 0) return hipErrorInvalidValue;
  return bf16 ? launch_fuse_t<uint16_t>(f, s, e0, e1) : launch_fuse_t<float>(f, s, e0, e1);
}

hipError_t launch_gram(const GramArgs& a, int max_in, int max_out, int bf16, hipStream_t s) {
  if (a.n_tables < 1 || a.n_tables > 65535 || a.r1 < 1 || a.r2 < 1 || max_in < 8 || max_out < 8)
    return hipErrorInvalidValue;
  const int items = (max_in + kGramKC - 1) / kGramKC + (max_out + kGramKC - 1) / kGramKC;
  return bf16 ? launch_gram_t<uint16_t>(a, items, s) : launch_gram_t<float>(a, items, s);
}

}  // namespace salt
