// HIP kernels of libsalt for gfx950 (MI355X): device plan builder and the
// centroid + residual apply (gathered split-K shrink, expand with fused y update).
//
// The apply computes, per token t of a plan (Sec. 3.3 served weight minus W_base):
//     v_t = x_t [A_c | A_u]                (shrink: one rank-(r_c + r_u) contraction)
//     v_t[0:r_c] *= gamma_t                (centroid scale, Sec. 3.3)
//     y_t = rne(y_t + v_t [B_c ; B_u])     (expand + accumulate, fp32 math)
// Tokens are processed in tiles of up to kTileM tokens that share one centroid,
// so each tile streams its centroid's A/B chunk once for all of its tokens.
#include "salt_internal.h"

namespace salt {
namespace {

// ---------------------------------------------------------------------------
// element access: 8 consecutive elements <-> 8 floats
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16, round to nearest even (NaN stays a quiet NaN).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ void ld8(const uint16_t* p, float* o) {
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  o[0] = bf_lo(v.x); o[1] = bf_hi(v.x); o[2] = bf_lo(v.y); o[3] = bf_hi(v.y);
  o[4] = bf_lo(v.z); o[5] = bf_hi(v.z); o[6] = bf_lo(v.w); o[7] = bf_hi(v.w);
}
__device__ __forceinline__ void ld8(const float* p, float* o) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
  o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}
__device__ __forceinline__ void st8(uint16_t* p, const float* v) {
  uint4 w;
  w.x = f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16);
  w.y = f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16);
  w.z = f32_to_bf16_rne(v[4]) | (f32_to_bf16_rne(v[5]) << 16);
  w.w = f32_to_bf16_rne(v[6]) | (f32_to_bf16_rne(v[7]) << 16);
  *reinterpret_cast<uint4*>(p) = w;
}
__device__ __forceinline__ void st8(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------
constexpr int kPlanThreads = 256;
constexpr int kPlanTokPerBlock = 64;  // four lanes count the rank of one token
constexpr int kPlanChunk = 2048;      // keys staged in LDS per pass

// Total order key (centroid, slot, token), -1 ids first: each field is shifted by
// one so that -1 becomes 0.  Fields are 21 bits wide (T, slots, centroids < 2^21 - 1).
__device__ __forceinline__ uint64_t plan_key(int c, int u, int t) {
  return (uint64_t(uint32_t(c + 1)) << 42) | (uint64_t(uint32_t(u + 1)) << 21) |
         uint64_t(uint32_t(t));
}

// Exclusive count of `pred` over the 256 threads of a block, and the block total.
__device__ __forceinline__ int block_excl_count(bool pred, int* s_wave, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t m = __ballot(pred);
  const int in_wave = (int)__builtin_amdgcn_mbcnt_hi(
      (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
  if (lane == 0) s_wave[wave] = __popcll(m);
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kPlanThreads / 64; ++w) {
    const int c = s_wave[w];
    off += (w < wave) ? c : 0;
    tot += c;
  }
  __syncthreads();
  total = tot;
  return off + in_wave;
}

// Rank of every token in the (c, u, t) order by counting smaller keys, then the
// last block to arrive cuts the sorted order into segments and groups.
__global__ void __launch_bounds__(kPlanThreads) k_plan(PlanBuffers b, int T) {
  __shared__ uint64_t skey[kPlanChunk];
  __shared__ int s_wave[kPlanThreads / 64];
  __shared__ int s_last;
  const int tid = threadIdx.x;
  const int t = blockIdx.x * kPlanTokPerBlock + (tid >> 2);
  const int q = tid & 3;
  int4 mine = make_int4(0, 0, 0, 0);
  uint64_t my = ~0ull;
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

  // the last block to arrive sees every block's scatter
  __threadfence();
  __syncthreads();
  if (tid == 0) s_last = (atomicAdd(b.counter, 1u) == gridDim.x - 1) ? 1 : 0;
  __syncthreads();
  if (!s_last) return;
  __threadfence();

  int seg_base = 0, grp_base = 0;
  for (int base = 0; base < T; base += kPlanThreads) {
    const int i = base + tid;
    int c = 0, u = 0;
    bool ns = false, ng = false;
    if (i < T) {
      c = b.srt_c[i];
      u = b.srt[i].y;
      if (i == 0) {
        ns = ng = true;
      } else {
        const int cp = b.srt_c[i - 1], up = b.srt[i - 1].y;
        ng = (c != cp);
        ns = ng || (u != up);
      }
    }
    int seg_tot, grp_tot;
    const int sr = block_excl_count(ns, s_wave, seg_tot);
    const int gr = block_excl_count(ng, s_wave, grp_tot);
    if (ns) {
      const int s = seg_base + sr;
      b.seg_off[s] = i;
      b.seg_c[s] = c;
      b.seg_u[s] = u;
    }
    if (ng) {
      const int g = grp_base + gr;
      b.grp_off[g] = seg_base + sr;
      b.grp_tok[g] = i;
      b.grp_c[g] = c;
    }
    seg_base += seg_tot;
    grp_base += grp_tot;
  }
  if (tid == 0) {
    b.seg_off[seg_base] = T;
    b.grp_off[grp_base] = seg_base;
    b.grp_tok[grp_base] = T;
    b.meta[0] = seg_base;
    b.meta[1] = grp_base;
    b.meta[2] = T;
    *b.counter = 0u;
  }
}

// ---------------------------------------------------------------------------
// tiles: groups of equal centroid cut into runs of at most M sorted tokens
// ---------------------------------------------------------------------------
struct TileInfo {
  int i0, n, c;
};

// Wave 0 finds tile `tile` (in group order); writes n = 0 if there is none.
__device__ void find_tile(const int32_t* grp_tok, const int32_t* grp_c, const int32_t* meta,
                          int M, int tile, TileInfo* out) {
  const int lane = threadIdx.x & 63;
  if (lane == 0) out->n = 0;
  const int n_grp = meta[1];
  int carry = 0;
  for (int gb = 0; gb < n_grp; gb += 64) {
    const int g = gb + lane;
    int start = 0, len = 0, cnt = 0;
    if (g < n_grp) {
      start = grp_tok[g];
      len = grp_tok[g + 1] - start;
      cnt = (len + M - 1) / M;
    }
    int incl = cnt;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(incl, off);
      if (lane >= off) incl += v;
    }
    const int excl = carry + incl - cnt;
    if (g < n_grp && tile >= excl && tile < excl + cnt) {
      const int k = tile - excl;
      out->i0 = start + k * M;
      out->n = min(M, len - k * M);
      out->c = grp_c[g];
    }
    carry += __shfl(incl, 63);
  }
}

// ---------------------------------------------------------------------------
// shrink: split-K partial sums of v = x [A_c | A_u] for one tile and one K range
// ---------------------------------------------------------------------------
constexpr int kKS = 64;               // K sub-chunk staged in LDS
constexpr int kLds = kKS + 1;         // padded row stride (floats), avoids bank conflicts
constexpr int kMaxR = 128 + 16;       // r_c + r_u_max upper bound
constexpr int kQ = (kTileM * kMaxR + 255) / 256;
constexpr int kLdsBudget = 120 * 1024;   // largest dynamic LDS any apply launch requests

template <typename E>
__global__ void __launch_bounds__(256) k_shrink(ApplyArgs a) {
  extern __shared__ float lds[];
  __shared__ TileInfo s_tile;
  __shared__ int s_row[kTileM], s_r[kTileM];
  __shared__ const E* s_au[kTileM];
  const int tid = threadIdx.x;
  if (tid < 64) find_tile(a.grp_tok, a.grp_c, a.meta, kTileM, blockIdx.x, &s_tile);
  __syncthreads();
  const int n = s_tile.n;
  if (n == 0) return;
  const int i0 = s_tile.i0, c = s_tile.c;
  if (tid < n) {
    const int4 e = a.srt[i0 + tid];
    const int r = (e.y >= 0) ? e.z : 0;
    s_row[tid] = e.x;
    s_r[tid] = r;
    s_au[tid] = r ? reinterpret_cast<const E*>(a.pool + (size_t)e.y * a.slot_stride) +
                        (int64_t)r * a.tab_prefix
                  : nullptr;
  }
  __syncthreads();

  const int R = a.R, rc = (c >= 0) ? a.r_c : 0, rum = a.r_u_max, in = a.in_dim;
  float* X = lds;                        // [kTileM][kLds]
  float* AC = X + kTileM * kLds;         // [r_c][kLds]
  float* AU = AC + a.r_c * kLds;         // [kTileM * r_u_max][kLds]
  const E* at_c = reinterpret_cast<const E*>(a.cent_at) + (size_t)(c >= 0 ? c : 0) * a.r_c * in;
  const int k0 = blockIdx.y * a.Kc, k1 = min(in, k0 + a.Kc);

  float acc[kQ];
#pragma unroll
  for (int q = 0; q < kQ; ++q) acc[q] = 0.f;

  for (int kb = k0; kb < k1; kb += kKS) {
    const int kw = min(kKS, k1 - kb);
    __syncthreads();
    for (int v = tid; v < kTileM * (kKS / 8); v += 256) {
      const int i = v / (kKS / 8), kk = (v % (kKS / 8)) * 8;
      float tmp[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      if (i < n && kk < kw) ld8(reinterpret_cast<const E*>(a.x) + (size_t)s_row[i] * in + kb + kk, tmp);
#pragma unroll
      for (int e = 0; e < 8; ++e) X[i * kLds + kk + e] = tmp[e];
    }
    for (int v = tid; v < rc * (kKS / 8); v += 256) {
      const int j = v / (kKS / 8), kk = (v % (kKS / 8)) * 8;
      float tmp[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      if (kk < kw) ld8(at_c + (size_t)j * in + kb + kk, tmp);
#pragma unroll
      for (int e = 0; e < 8; ++e) AC[j * kLds + kk + e] = tmp[e];
    }
    for (int v = tid; v < kTileM * rum * (kKS / 8); v += 256) {
      const int row = v / (kKS / 8), kk = (v % (kKS / 8)) * 8;
      const int i = row / rum, j = row % rum;
      float tmp[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      if (i < n && j < s_r[i] && kk < kw) ld8(s_au[i] + (size_t)j * in + kb + kk, tmp);
#pragma unroll
      for (int e = 0; e < 8; ++e) AU[row * kLds + kk + e] = tmp[e];
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const int o = tid + 256 * q;
      if (o < n * R) {
        const int i = o / R, j = o % R;
        const float* ar = nullptr;
        if (j < rc) ar = AC + j * kLds;
        else if (j >= a.r_c && j - a.r_c < s_r[i]) ar = AU + (i * rum + (j - a.r_c)) * kLds;
        if (ar) {
          const float* xr = X + i * kLds;
          float s = 0.f;
#pragma unroll 16
          for (int kk = 0; kk < kKS; ++kk) s += xr[kk] * ar[kk];
          acc[q] += s;
        }
      }
    }
  }
  float* P = a.partials + ((size_t)blockIdx.y * a.T + i0) * R;
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    const int o = tid + 256 * q;
    if (o < n * R) P[o] = acc[q];
  }
}

// ---------------------------------------------------------------------------
// expand: y rows of one tile, one column chunk: y += v [g*B_c ; B_u]
// ---------------------------------------------------------------------------
template <typename E>
__global__ void __launch_bounds__(256) k_expand(ApplyArgs a) {
  extern __shared__ float lds[];
  __shared__ TileInfo s_tile;
  __shared__ int s_row[kTileM], s_r[kTileM];
  __shared__ float s_g[kTileM];
  __shared__ const E* s_bu[kTileM];
  const int tid = threadIdx.x;
  if (tid < 64) find_tile(a.grp_tok, a.grp_c, a.meta, kTileM, blockIdx.x, &s_tile);
  __syncthreads();
  const int n = s_tile.n;
  if (n == 0) return;
  const int i0 = s_tile.i0, c = s_tile.c;
  const int R = a.R, rc = (c >= 0) ? a.r_c : 0, out = a.out_dim, NC = a.NC;
  if (tid < n) {
    const int4 e = a.srt[i0 + tid];
    const int r = (e.y >= 0) ? e.z : 0;
    s_row[tid] = e.x;
    s_r[tid] = r;
    s_g[tid] = __int_as_float(e.w);
    s_bu[tid] = r ? reinterpret_cast<const E*>(a.pool + (size_t)e.y * a.slot_stride) +
                        (int64_t)r * (a.tab_prefix + a.in_dim)
                  : nullptr;
  }
  __syncthreads();

  float* V = lds;                  // [kTileM][R]
  float* BC = V + kTileM * R;      // [r_c][NC]
  for (int idx = tid; idx < n * R; idx += 256) {
    const float* P = a.partials + (size_t)i0 * R + idx;
    float s = 0.f;
    for (int sp = 0; sp < a.S; ++sp) s += P[(size_t)sp * a.T * R];
    const int i = idx / R, j = idx % R;
    if (j < a.r_c) s *= s_g[i];
    V[idx] = s;
  }
  const int n0 = blockIdx.y * NC;
  const int ncols = min(NC, out - n0);
  const E* bc = reinterpret_cast<const E*>(a.cent_b) + (size_t)(c >= 0 ? c : 0) * a.r_c * out;
  for (int v = tid; v < rc * (NC / 8); v += 256) {
    const int j = v / (NC / 8), cc = (v % (NC / 8)) * 8;
    float tmp[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (cc < ncols) ld8(bc + (size_t)j * out + n0 + cc, tmp);
#pragma unroll
    for (int e = 0; e < 8; ++e) BC[j * NC + cc + e] = tmp[e];
  }
  __syncthreads();

  const int CG = NC / 8, TL = 256 / CG;
  const int cg = tid % CG, tl = tid / CG;
  if (tl >= TL || cg * 8 >= ncols) return;
  const int col = n0 + cg * 8;
  for (int i = tl; i < n; i += TL) {
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    const float* vi = V + i * R;
    for (int j = 0; j < rc; ++j) {
      const float vj = vi[j];
      const float* b = BC + j * NC + cg * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += vj * b[e];
    }
    for (int j = 0; j < s_r[i]; ++j) {
      float b[8];
      ld8(s_bu[i] + (size_t)j * out + col, b);
      const float vj = vi[a.r_c + j];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += vj * b[e];
    }
    E* yp = reinterpret_cast<E*>(a.y) + (size_t)s_row[i] * out + col;
    float yv[8];
    ld8(yp, yv);
#pragma unroll
    for (int e = 0; e < 8; ++e) yv[e] += acc[e];
    st8(yp, yv);
  }
}

size_t shrink_lds(const ApplyArgs& a) {
  return sizeof(float) * (size_t)(kTileM + a.r_c + kTileM * a.r_u_max) * kLds;
}
size_t expand_lds(const ApplyArgs& a) {
  return sizeof(float) * ((size_t)kTileM * a.R + (size_t)a.r_c * a.NC);
}

}  // namespace

// Per-device set-up: checks that the device has the LDS the apply kernels may
// ask for (gfx950: 160 KiB per workgroup; dynamic LDS needs no opt-in on AMD).
hipError_t kernels_init(int device) {
  static bool done[64] = {};
  if (device < 0 || device >= 64) return hipErrorInvalidDevice;
  if (done[device]) return hipSuccess;
  int lds_max = 0;
  hipError_t e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, device);
  if (e != hipSuccess) return e;
  if (lds_max < kLdsBudget) return hipErrorInvalidConfiguration;
  done[device] = true;
  return hipSuccess;
}

hipError_t launch_plan(const PlanBuffers& b, int32_t T, int32_t, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const int blocks = (T + kPlanTokPerBlock - 1) / kPlanTokPerBlock;
  hipLaunchKernelGGL(k_plan, dim3(blocks), dim3(kPlanThreads), 0, s, b, T);
  return hipGetLastError();
}

hipError_t launch_apply(const ApplyArgs& a, int bf16, int32_t tiles_ub, hipStream_t s) {
  if (a.T <= 0 || tiles_ub <= 0) return hipSuccess;
  const dim3 g1(tiles_ub, a.S), g2(tiles_ub, (a.out_dim + a.NC - 1) / a.NC);
  if (bf16) {
    hipLaunchKernelGGL(k_shrink<uint16_t>, g1, dim3(256), shrink_lds(a), s, a);
    hipLaunchKernelGGL(k_expand<uint16_t>, g2, dim3(256), expand_lds(a), s, a);
  } else {
    hipLaunchKernelGGL(k_shrink<float>, g1, dim3(256), shrink_lds(a), s, a);
    hipLaunchKernelGGL(k_expand<float>, g2, dim3(256), expand_lds(a), s, a);
  }
  return hipGetLastError();
}

}  // namespace salt
