// The batched centroid + residual LoRA apply on gfx950 (MI355X).
//
// For every token t of a plan and every table (job) of the launch, with the
// served weight of Sec. 3.3 minus W_base:
//     v_t = x_t [A_c | A_u]               shrink: one rank-(r_c + r_u) contraction
//     v_t[0:r_c] *= gamma_t               centroid scale of Sec. 3.3
//     y_t = rne(y_t + v_t [B_c ; B_u])    expand with fused accumulation, fp32 math
//
// Two launches on the caller's stream, one after the other; no block ever
// waits for another block, so every launch drains whatever the data holds.
//   k_shrink: one block per (table, tile, K range, residual rank chunk).  The
//     tile's tokens share one centroid, so the centroid part [M x K] . [K x r_c]
//     is a dense GEMM on MFMA (v_mfma_f32_16x16x32_bf16; 16x16x4f32 for fp32).
//     The residual part differs per token and has rank <= 2 (<= 16 per chunk for
//     plain LoRA baselines and long-tail adapters): per-token dot products on the
//     vector ALUs (v_dot2_f32_bf16), reduced across lanes with shuffles.  Each
//     block stores its split-K partial sums; every (K range, position, column)
//     is written by exactly one block.
//   k_expand: one block per (table, tile, column block).  It sums the tile's
//     partials in K-range order (deterministic), scales the centroid part by
//     gamma, and streams its columns: the centroid part on MFMA with v split
//     into two bf16 halves (hi + lo, ~16 significant bits), the residual part
//     as fp32 FMAs, added to y and rounded once.
// Every global address is formed by the clamped offset functions of
// salt_layout.h.
#include <hip/hip_ext.h>

#include <algorithm>

#include "salt_device.h"
#include "salt_internal.h"
#include "salt_layout.h"

namespace salt {
namespace {

// ---------------------------------------------------------------------------
// shrink
// ---------------------------------------------------------------------------
// E: element type; M: tokens per tile (16 TB, TB token blocks of 16); NB: 16-rank
// blocks of the centroid (r_c <= 16 NB; 0 without centroids); RU: residual
// ranks of one chunk.  Wave w takes token block w % TB and every (4 / TB)-th
// kStepK-wide step of the block's K range, starting at w / TB.  A lane holds
// token (lane & 15) of its block and the 16 consecutive k at 16 (lane >> 4) of
// a step, as two 8-element vectors h = 0, 1; MFMA h multiplies vector h of x
// and of A_c, so the two MFMAs of a step together cover its 64 k.
template <int NB, int RU>
constexpr int shrink_wc() { return 16 * NB + RU; }

template <typename E, int M, int NB, int RU>
__global__ void __launch_bounds__(kThreads) k_shrink(const ApplyLaunch a) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  constexpr int TB = M / 16, KW = kWaves / TB, WC = shrink_wc<NB, RU>();
  extern __shared__ __attribute__((aligned(16))) char lds[];
  float* s_red = reinterpret_cast<float*>(lds);   // [KW][M][WC] per-wave sums

  const int b = blockIdx.x;
  const Job& jb = a.jobs[job_of_shrink(a, b)];
  const ShrinkCoord sc = shrink_coord(a, jb, b);
  const TileHdr th = clamp_tile(a, a.tiles[sc.tau]);
  if (th.n <= 0) return;                          // (no tile is empty; the whole block leaves)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int mb = wave % TB, kq = wave / TB, row = lane & 15, g = lane >> 4;
  const int kt = mb * 16 + row;                   // this lane's token within the tile
  const TokRec tr = clamp_tok(a, a.srt[tile_pos(th, kt)], kt < th.n);
  const int r0 = sc.q * kRankChunk;               // first residual rank of this block
  const bool has_c = NB > 0 && th.c >= 0 && sc.q == 0;
  const E* x = reinterpret_cast<const E*>(jb.x);
  const E* atc = reinterpret_cast<const E*>(jb.at_c);

  f32x4 acc[NB > 0 ? NB : 1];
#pragma unroll
  for (int nb = 0; nb < (NB > 0 ? NB : 1); ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float accu[RU];
#pragma unroll
  for (int j = 0; j < RU; ++j) accu[j] = 0.f;

  const int klo = k_lo(jb, sc.s), khi = k_hi(jb, sc.s), nst = k_steps(jb, sc.s);
  for (int st = kq; st < nst; st += KW) {
    const int kb = klo + st * kStepK + 16 * g;
    Vec xv[2];
    bool kv[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      kv[h] = kb + 8 * h + 8 <= khi;              // in, Kc are multiples of 8: a vector is all in or all out
      xv[h] = kv[h] ? O::load(x + x_off(a, jb, tr.t, kb + 8 * h)) : O::zero();
    }
    if constexpr (NB > 0) {
      if (has_c) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          Vec av[2];
#pragma unroll
          for (int h = 0; h < 2; ++h)
            av[h] = kv[h] ? O::load(atc + atc_off(a, jb, th.c, 16 * nb + row, kb + 8 * h)) : O::zero();
#pragma unroll
          for (int h = 0; h < 2; ++h) acc[nb] = O::mma(xv[h], av[h], acc[nb]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < RU; ++j) {
      const int rho = r0 + j;
      if (tr.res && rho < tr.r) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const Vec uv = kv[h] ? O::load(reinterpret_cast<const E*>(a.pool + atu_byte(a, jb, tr.u, tr.r, rho, kb + 8 * h)))
                               : O::zero();
          accu[j] = O::dot(xv[h], uv, accu[j]);
        }
      }
    }
  }
  // residual: lanes l, l ^ 16, l ^ 32, l ^ 48 hold the four k offsets of one token
#pragma unroll
  for (int j = 0; j < RU; ++j) {
    accu[j] += __shfl_xor(accu[j], 16);
    accu[j] += __shfl_xor(accu[j], 32);
  }
  float* P = s_red + (size_t)kq * M * WC;
  if constexpr (NB > 0) {
    if (has_c) {
      // MFMA output: lane holds rank column 16 nb + row of tokens 4 g + e
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int e = 0; e < 4; ++e) P[(mb * 16 + 4 * g + e) * WC + 16 * nb + row] = acc[nb][e];
    }
  }
  if (g == 0) {
#pragma unroll
    for (int j = 0; j < RU; ++j) P[kt * WC + 16 * NB + j] = accu[j];
  }
  __syncthreads();
  // the tile's partial: centroid columns [0, r_c) (chunk 0 only; zero without a
  // centroid term), residual columns r_c + r0 + [0, nres)
  const int ncent = sc.q == 0 ? a.r_c : 0;
  const int nres = imax(0, imin(RU, a.r_u - r0));
  const int ncols = ncent + nres;
  for (int idx = tid; idx < th.n * ncols; idx += kThreads) {
    const int k = idx / ncols, cc = idx - k * ncols;
    float v = 0.f;
    int col;
    if (cc < ncent) {
      col = cc;
      if (has_c) {
#pragma unroll
        for (int w = 0; w < KW; ++w) v += s_red[((size_t)w * M + k) * WC + cc];
      }
    } else {
      const int j = cc - ncent;
      col = a.r_c + r0 + j;
#pragma unroll
      for (int w = 0; w < KW; ++w) v += s_red[((size_t)w * M + k) * WC + 16 * NB + j];
    }
    a.partials[part_off(a, jb, sc.s, th.i0 + k, col)] = v;
  }
}

// ---------------------------------------------------------------------------
// expand
// ---------------------------------------------------------------------------
// Wave w takes token block w % TB and every (4 / TB)-th 64-column chunk of the
// block's columns, starting at w / TB.  Per chunk the centroid part is four
// 16 x 16 MFMA tiles D[col][token] = Bt_c[col][:] . v_c[token][:]; A-operand row
// i of tile b4 is column expand_col(col0, i, b4), so that output lane (token =
// lane & 15, g = lane >> 4) holds the 16 consecutive columns col0 + 16 g + 0..15
// of its token: y is read and written as 32 contiguous bytes (bf16) per lane.
template <typename E, int M, int NB, int RU>
__global__ void __launch_bounds__(kThreads) k_expand(const ApplyLaunch a) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  constexpr bool kBf16 = sizeof(E) == 2;
  constexpr int TB = M / 16, CW = kWaves / TB, KS = (NB + 1) / 2;
  extern __shared__ __attribute__((aligned(16))) char lds[];
  int4* s_rec = reinterpret_cast<int4*>(lds);               // [M] token records
  float* s_v = reinterpret_cast<float*>(lds + M * 16);      // [M][R] v of the tile

  const int b = blockIdx.x;
  const Job& jb = a.jobs[job_of_expand(a, b)];
  const ExpandCoord ec = expand_coord(a, jb, b);
  const TileHdr th = clamp_tile(a, a.tiles[ec.tau]);
  if (th.n <= 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int R = a.R, VW = imin(a.r_c + a.r_u, R);

  if (tid < M) s_rec[tid] = a.srt[tile_pos(th, tid)];
  // v of the tile: the K ranges' partials summed in order
  for (int idx = tid; idx < M * VW; idx += kThreads) {
    const int k = idx / VW, col = idx - k * VW;
    float v = 0.f;
    if (k < th.n) {
      const int p = th.i0 + k;
      int s = 0;
      for (; s + 4 <= jb.S; s += 4) {
        const float p0 = a.partials[part_off(a, jb, s, p, col)];
        const float p1 = a.partials[part_off(a, jb, s + 1, p, col)];
        const float p2 = a.partials[part_off(a, jb, s + 2, p, col)];
        const float p3 = a.partials[part_off(a, jb, s + 3, p, col)];
        v += p0;
        v += p1;
        v += p2;
        v += p3;
      }
      for (; s < jb.S; ++s) v += a.partials[part_off(a, jb, s, p, col)];
    }
    s_v[k * R + col] = v;
  }
  __syncthreads();

  const int mb = wave % TB, cq = wave / TB, row = lane & 15, g = lane >> 4;
  const int kt = mb * 16 + row;                   // this lane's token within the tile
  const TokRec tr = clamp_tok(a, s_rec[kt], kt < th.n);
  const bool has_c = NB > 0 && th.c >= 0;
  const float gam = __uint_as_float(tr.gamma_bits);
  const float* vrow = s_v + kt * R;

  // centroid v as the MFMA's right operand: column = token, k = ranks
  // 32 ks + 8 g .. + 7, scaled by gamma; ranks past r_c are zero
  Vec vhi[KS > 0 ? KS : 1], vlo[KS > 0 ? KS : 1];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    float f[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int j = 32 * ks + 8 * g + e;
      f[e] = (tr.tok && j < a.r_c) ? vrow[j] * gam : 0.f;
    }
    if constexpr (kBf16) {
      uint32_t h[8], l[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        h[e] = f32_to_bf16_rne(f[e]);
        l[e] = f32_to_bf16_rne(f[e] - __uint_as_float(h[e] << 16));
      }
      vhi[ks] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
      vlo[ks] = make_uint4(l[0] | (l[1] << 16), l[2] | (l[3] << 16), l[4] | (l[5] << 16), l[6] | (l[7] << 16));
    } else {
      vhi[ks].lo = make_float4(f[0], f[1], f[2], f[3]);
      vhi[ks].hi = make_float4(f[4], f[5], f[6], f[7]);
      vlo[ks] = O::zero();
    }
  }

  E* y = reinterpret_cast<E*>(jb.y);
  const E* btc = reinterpret_cast<const E*>(jb.bt_c);
  const int clo = c_lo(jb, ec.cb), chi = c_hi(jb, ec.cb), nch = c_chunks(jb, ec.cb);
  for (int ch = cq; ch < nch; ch += CW) {
    const int col0 = clo + ch * kChunkCols;
    const int cl = col0 + 16 * g;                 // this lane's first column
    bool cv[2];
    Vec yv[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      cv[h] = tr.tok && cl + 8 * h + 8 <= chi;    // out, cpb are multiples of 8
      yv[h] = cv[h] ? O::load(y + y_off(a, jb, tr.t, cl + 8 * h)) : O::zero();
    }
    f32x4 d[4];
#pragma unroll
    for (int b4 = 0; b4 < 4; ++b4) d[b4] = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (NB > 0) {
      if (has_c) {
#pragma unroll
        for (int b4 = 0; b4 < 4; ++b4) {
          const int o = expand_col(col0, row, b4);
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const int j = 32 * ks + 8 * g;
            const Vec bf = j < a.r_c ? O::load(btc + btc_off(a, jb, th.c, o, j)) : O::zero();
            d[b4] = O::mma(bf, vhi[ks], d[b4]);
            if constexpr (kBf16) d[b4] = O::mma(bf, vlo[ks], d[b4]);
          }
        }
      }
    }
    float yf[16];
    O::to_f32(yv[0], yf);
    O::to_f32(yv[1], yf + 8);
#pragma unroll
    for (int b4 = 0; b4 < 4; ++b4)
#pragma unroll
      for (int e = 0; e < 4; ++e) yf[4 * b4 + e] += d[b4][e];
    if (tr.res) {
      for (int q = 0; q < a.nq; ++q) {
#pragma unroll
        for (int j = 0; j < RU; ++j) {
          const int rho = q * kRankChunk + j;
          if (rho < tr.r) {
            const float vr = vrow[a.r_c + rho];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              if (cv[h]) {
                float bu[8];
                O::to_f32(O::load(reinterpret_cast<const E*>(a.pool + bu_byte(a, jb, tr.u, tr.r, rho, cl + 8 * h))), bu);
#pragma unroll
                for (int e = 0; e < 8; ++e) yf[8 * h + e] = fmaf(vr, bu[e], yf[8 * h + e]);
              }
            }
          }
        }
      }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
      if (cv[h]) O::store(y + y_off(a, jb, tr.t, cl + 8 * h), yf + 8 * h);
  }
}

// ---------------------------------------------------------------------------
// launch
// ---------------------------------------------------------------------------
template <typename K>
void launch_k(K kernel, int blocks, size_t lds, hipStream_t s, const ApplyLaunch& a, hipEvent_t e0,
              hipEvent_t e1) {
  if (e0 || e1) hipExtLaunchKernelGGL(kernel, dim3(blocks), dim3(kThreads), (uint32_t)lds, s, e0, e1, 0u, a);
  else hipLaunchKernelGGL(kernel, dim3(blocks), dim3(kThreads), lds, s, a);
}

template <typename E, int M, int NB, int RU>
hipError_t launch_mnr(const ApplyLaunch& a, hipStream_t s, hipEvent_t* ev) {
  const size_t lds_s = sizeof(float) * (size_t)(kWaves / (M / 16)) * M * shrink_wc<NB, RU>();
  const size_t lds_e = (size_t)M * 16 + sizeof(float) * (size_t)M * a.R;
  launch_k(k_shrink<E, M, NB, RU>, a.shrink_blocks, lds_s, s, a, ev ? ev[0] : nullptr, ev ? ev[1] : nullptr);
  launch_k(k_expand<E, M, NB, RU>, a.expand_blocks, lds_e, s, a, ev ? ev[2] : nullptr, ev ? ev[3] : nullptr);
  return hipGetLastError();
}

template <typename E, int M, int NB>
hipError_t launch_mn(const ApplyLaunch& a, hipStream_t s, hipEvent_t* ev) {
  if (a.r_u <= 1) return launch_mnr<E, M, NB, 1>(a, s, ev);
  if (a.r_u <= 2) return launch_mnr<E, M, NB, 2>(a, s, ev);
  return launch_mnr<E, M, NB, kRankChunk>(a, s, ev);
}

template <typename E, int M>
hipError_t launch_m(const ApplyLaunch& a, hipStream_t s, hipEvent_t* ev) {
  switch (centroid_blocks(a.r_c)) {
    case 0: return launch_mn<E, M, 0>(a, s, ev);
    case 2: return launch_mn<E, M, 2>(a, s, ev);
    case 4: return launch_mn<E, M, 4>(a, s, ev);
    default: return launch_mn<E, M, 8>(a, s, ev);
  }
}

}  // namespace

hipError_t launch_apply(const ApplyLaunch& a, hipStream_t s, hipEvent_t* ev) {
  if (a.T <= 0 || a.n_tiles <= 0 || a.n_jobs <= 0) return hipSuccess;
  if (a.n_jobs > kMaxJobs || a.shrink_blocks <= 0 || a.expand_blocks <= 0 || a.r_c > kMaxRc || a.r_u > kMaxRu)
    return hipErrorInvalidValue;
  if (a.esize == 4) {
    if (a.M != 16) return hipErrorInvalidValue;
    return launch_m<float, 16>(a, s, ev);
  }
  switch (a.M) {
    case 16: return launch_m<uint16_t, 16>(a, s, ev);
    case 32: return launch_m<uint16_t, 32>(a, s, ev);
    case 64: return launch_m<uint16_t, 64>(a, s, ev);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace salt

namespace salt {

// Per-device set-up: checks that a workgroup may hold the LDS the apply and
// plan kernels ask for (the expand of 64-token tiles at the largest ranks).
hipError_t kernels_init(int device) {
  static bool done[64] = {};
  if (device < 0 || device >= 64) return hipErrorInvalidDevice;
  if (done[device]) return hipSuccess;
  int lds_max = 0;
  hipError_t e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, device);
  if (e != hipSuccess) return e;
  const size_t R = (size_t)padded_rank(kMaxRc, kMaxRu);
  const size_t need_expand = 64 * 16 + sizeof(float) * 64 * R;
  const size_t need_shrink = sizeof(float) * 64 * (16 * centroid_blocks(kMaxRc) + kRankChunk);
  const size_t need_plan = sizeof(uint64_t) * kSortChunk + 256;
  const size_t need = std::max(need_expand, std::max(need_shrink, need_plan));
  if ((size_t)lds_max < need) return hipErrorInvalidConfiguration;
  done[device] = true;
  return hipSuccess;
}

}  // namespace salt
