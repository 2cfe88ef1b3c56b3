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
// shared shapes
// ---------------------------------------------------------------------------
// M tokens per tile = TB token blocks of 16.  A block's 4 waves split as
// (token block, K quarter) in the shrink and (token block, column phase) in the
// expand: KW = CW = 4 / TB.  With TB > 1 (32- and 64-token tiles, bf16) several
// waves need the same centroid operand at the same time (A_c in the shrink, B_c
// in the expand); the block then loads it once, cooperatively, into an LDS
// stage from which each wave reads its MFMA fragments.
template <int M>
constexpr int waves_along() { return kWaves / (M / 16); }
template <typename E, int M, int NB>
constexpr bool staged() { return sizeof(E) == 2 && M > 16 && NB > 0; }
// Register batches: block-steps (shrink) or block-chunks (expand) whose loads
// are issued together; two batches alternate, so one is in flight while the
// other computes.
template <typename E, int M, int NB, int RU>
constexpr int batch_len() { return (M == 64 && NB <= 4 && RU <= 2) ? 2 : 1; }
// Staged rows carry 8 elements of padding: consecutive rows then start 4 LDS
// banks apart, so a fragment read (16 rows x 16 bytes per 8-lane phase) hits
// every bank once.
template <int M>
constexpr int stage_row_a() { return kStepK * waves_along<M>() + 8; }
template <int NB>
constexpr int stage_row_b() { return 16 * NB + 8; }
template <int NB, int RU>
constexpr int shrink_wc() { return 16 * NB + RU; }

__device__ __forceinline__ uint4 sel(bool p, uint4 v) { return p ? v : make_uint4(0u, 0u, 0u, 0u); }
__device__ __forceinline__ Ops<float>::Vec sel(bool p, Ops<float>::Vec v) { return p ? v : Ops<float>::zero(); }

// ---------------------------------------------------------------------------
// shrink
// ---------------------------------------------------------------------------
// Wave w takes token block mb = w % TB and the kStepK-wide steps kq, kq + KW, ...
// (kq = w / TB) of the block's K range: block-step j covers steps j KW .. j KW +
// KW - 1, one per K quarter.  A lane holds token (lane & 15) of its block and the
// 16 consecutive k at 16 (lane >> 4) of a step, as two 8-element vectors h = 0,
// 1; MFMA h multiplies vector h of x and of A_c, so the two MFMAs of a step
// together cover its 64 k.  Every load is issued unconditionally at an address
// inside the block's own data (a step past the wave's last re-reads that last
// step, the ragged end of K re-reads the last full vector, a token without a
// centroid or residual term reads its own x row), and masked by a select, so
// that the compiler's waits on outstanding loads count them exactly and a batch
// stays in flight while the other one computes.
template <typename E, int M, int NB, int RU>
__global__ void __launch_bounds__(kThreads) k_shrink(const ApplyLaunch a) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  constexpr int TB = M / 16, KW = waves_along<M>(), WC = shrink_wc<NB, RU>();
  constexpr bool kStage = staged<E, M, NB>();
  constexpr int U = batch_len<E, M, NB, RU>();
  constexpr int NBL = NB > 0 ? NB : 1;
  constexpr int SR = stage_row_a<M>();                       // elements per staged A_c row
  constexpr int NCV = kStage ? NB * KW / 2 : 1;              // staged A_c vectors per thread and block-step
  constexpr int NAC = kStage ? NCV : 2 * NBL;                // A_c vectors per lane and step
  constexpr int RUP = RU <= 2 ? RU : 1;                      // residual ranks in the pipelined batch (wider: read in place)
  extern __shared__ __attribute__((aligned(16))) char lds[];
  float* s_red = reinterpret_cast<float*>(lds);              // [KW][M][WC], after the K loop
  E* s_a = reinterpret_cast<E*>(lds);                        // [2][U][16 NB][SR], during the K loop

  const int b = blockIdx.x;
  const Job& jb = a.jobs[job_of_shrink(a, b)];
  const ShrinkCoord sc = shrink_coord(a, jb, b);
  const TileHdr th = clamp_tile(a, a.tiles[sc.tau]);
  if (th.n <= 0) return;                                     // (no tile is empty; the whole block leaves)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int mb = wave % TB, kq = wave / TB, row = lane & 15, g = lane >> 4;
  const int kt = mb * 16 + row;                              // this lane's token within the tile
  const TokRec tr = clamp_tok(a, a.srt[tile_pos(th, kt)], kt < th.n);
  // x row of the tile's first token: the address of loads whose value is
  // masked (it is read by the tile anyway, and differs from the lane's own
  // operands, so each such load stays a plain unconditional load)
  const int t0 = clamp_tok(a, a.srt[th.i0], true).t;
  const int r0 = sc.q * kRankChunk;                          // first residual rank of this block
  const bool has_c = NB > 0 && th.c >= 0 && sc.q == 0;
  const E* x = reinterpret_cast<const E*>(jb.x);
  const E* atc = reinterpret_cast<const E*>(jb.at_c);
  const int klo = k_lo(jb, sc.s), khi = k_hi(jb, sc.s), nst = k_steps(jb, sc.s);
  const int nbs = cdiv(nst, KW);                             // block-steps
  const int klast = imax(klo, khi - 8);                      // last whole vector of the K range

  f32x4 acc[NBL];
#pragma unroll
  for (int nb = 0; nb < NBL; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float accu[RU];
#pragma unroll
  for (int j = 0; j < RU; ++j) accu[j] = 0.f;

  struct Batch {
    Vec ac[U][NAC];
    Vec x[U][2];
    Vec u[U][RUP][2];
  };
  // first k of this wave's step in block-step j (past the end: its last step)
  auto step_k = [&](int j) { return klo + imin(j * KW + kq, nst - 1) * kStepK; };
  auto load = [&](Batch& B, int j0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u;
      const int kb = step_k(j) + 16 * g;
      if constexpr (kStage) {
        // the block's A_c slice of block-step j: 16 NB rows x 64 KW k, one 16-byte
        // piece per (thread, q); rows are whole 128 KW-byte runs of global memory
        const int kj = klo + imin(j, nbs - 1) * kStepK * KW;
#pragma unroll
        for (int q = 0; q < NCV; ++q) {
          const int L = q * kThreads + tid, r = L / (8 * KW), c16 = L % (8 * KW);
          const int kk = imin(kj + 8 * c16, klast);
          const E* p = has_c ? atc + atc_off(a, jb, th.c, r, kk) : x + x_off(a, jb, t0, kk);
          B.ac[u][q] = O::load(p);
        }
      } else if constexpr (NB > 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int kk = imin(kb + 8 * h, klast);
            const E* p = has_c ? atc + atc_off(a, jb, th.c, 16 * nb + row, kk) : x + x_off(a, jb, t0, kk);
            B.ac[u][2 * nb + h] = O::load(p);
          }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) B.x[u][h] = O::load(x + x_off(a, jb, tr.t, imin(kb + 8 * h, klast)));
#pragma unroll
      for (int jj = 0; jj < RUP; ++jj)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int kk = imin(kb + 8 * h, klast);
          const E* p = tr.res ? reinterpret_cast<const E*>(a.pool + atu_byte(a, jb, tr.u, tr.r, r0 + jj, kk))
                              : x + x_off(a, jb, t0, kk);
          B.u[u][jj][h] = O::load(p);
        }
    }
  };
  // the staged copy of a batch's A_c slices (rows past r_c and k past the range
  // are zero)
  auto stage = [&](const Batch& B, int half, int j0) {
    if constexpr (kStage) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int kj = klo + imin(j0 + u, nbs - 1) * kStepK * KW;
#pragma unroll
        for (int q = 0; q < NCV; ++q) {
          const int L = q * kThreads + tid, r = L / (8 * KW), c16 = L % (8 * KW);
          const bool ok = r < a.r_c && kj + 8 * c16 + 8 <= khi;
          *reinterpret_cast<Vec*>(s_a + ((size_t)(half * U + u) * 16 * NB + r) * SR + 8 * c16) = sel(ok, B.ac[u][q]);
        }
      }
    }
  };
  auto compute = [&](const Batch& B, int half, int j0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u, st = j * KW + kq;
      const int kb = klo + imin(st, nst - 1) * kStepK + 16 * g;
      Vec xv[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) xv[h] = sel(st < nst && kb + 8 * h + 8 <= khi, B.x[u][h]);
      if constexpr (NB > 0) {
        if (has_c) {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              Vec af;
              if constexpr (kStage)
                af = *reinterpret_cast<const Vec*>(s_a + ((size_t)(half * U + u) * 16 * NB + 16 * nb + row) * SR +
                                                   kq * kStepK + 16 * g + 8 * h);
              else
                af = B.ac[u][2 * nb + h];
              acc[nb] = O::mma(xv[h], af, acc[nb]);
            }
        }
      }
      if constexpr (RU <= 2) {
#pragma unroll
        for (int jj = 0; jj < RU; ++jj) {
          const bool live = tr.res && r0 + jj < tr.r;
#pragma unroll
          for (int h = 0; h < 2; ++h) accu[jj] = O::dot(xv[h], sel(live, B.u[u][jj][h]), accu[jj]);
        }
      } else {
        // wide residual ranks: this step's rows of 8 ranks at a time, loaded together here
#pragma unroll
        for (int j8 = 0; j8 < RU; j8 += 8) {
          Vec uv[8][2];
#pragma unroll
          for (int jj = 0; jj < 8; ++jj)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int kk = imin(kb + 8 * h, klast);
              const E* p = tr.res ? reinterpret_cast<const E*>(a.pool + atu_byte(a, jb, tr.u, tr.r, r0 + j8 + jj, kk))
                                  : x + x_off(a, jb, t0, kk);
              uv[jj][h] = O::load(p);
            }
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) {
            const bool live = tr.res && r0 + j8 + jj < tr.r;
#pragma unroll
            for (int h = 0; h < 2; ++h) accu[j8 + jj] = O::dot(xv[h], sel(live, uv[jj][h]), accu[j8 + jj]);
          }
        }
      }
    }
  };

  Batch A;
  if constexpr (sizeof(E) == 4) {
    // fp32: one register batch, loaded then used (its vectors are twice as wide)
    for (int j0 = 0; j0 < nbs; j0 += U) {
      load(A, j0);
      compute(A, 0, j0);
    }
  } else {
  Batch Bb;
  load(A, 0);
  if constexpr (kStage) {
    stage(A, 0, 0);
    __syncthreads();
  }
  for (int j0 = 0; j0 < nbs; j0 += 2 * U) {
    load(Bb, j0 + U);
    compute(A, 0, j0);
    if constexpr (kStage) {
      stage(Bb, 1, j0 + U);
      __syncthreads();
    }
    if (j0 + U >= nbs) break;                                // (block-uniform)
    load(A, j0 + 2 * U);
    compute(Bb, 1, j0 + U);
    if constexpr (kStage) {
      stage(A, 0, j0 + 2 * U);
      __syncthreads();
    }
  }
  }
  if constexpr (kStage) __syncthreads();                     // s_red reuses the stages

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
// Wave w takes token block mb = w % TB and, in block-chunk j, the 64-column chunk
// j CW + cq (cq = w / TB) of the block's columns.  Per chunk the centroid part is
// four 16 x 16 MFMA tiles D[col][token] = Bt_c[col][:] . v_c[token][:]; A-operand
// row i of tile b4 is column expand_col(col0, i, b4), so that output lane (token
// = lane & 15, g = lane >> 4) holds the 16 consecutive columns col0 + 16 g + 0..15
// of its token: y is read and written as 32 contiguous bytes (bf16) per lane.  A
// staged B_c chunk keeps the columns in that MFMA order (LDS row of column o:
// 64 (o / 64) + 16 b4 + i), so a fragment read takes 16 consecutive rows.  Loads
// are unconditional and masked by selects as in the shrink.
template <typename E, int M, int NB, int RU>
__global__ void __launch_bounds__(kThreads) k_expand(const ApplyLaunch a) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  constexpr bool kBf16 = sizeof(E) == 2;
  constexpr int TB = M / 16, CW = waves_along<M>(), KS = (NB + 1) / 2;
  constexpr bool kStage = staged<E, M, NB>();
  constexpr int U = batch_len<E, M, NB, RU>();
  constexpr int KSL = KS > 0 ? KS : 1;
  constexpr int SRB = stage_row_b<NB>();                     // elements per staged B_c row (one column)
  constexpr int NCV = kStage ? CW * NB / 2 : 1;              // staged B_c vectors per thread and block-chunk
  constexpr int NBC = kStage ? NCV : 4 * KSL;                // B_c vectors per lane and chunk
  constexpr int RUP = RU <= 2 ? RU : 1;                      // residual ranks in the pipelined batch (wider: read in place)
  extern __shared__ __attribute__((aligned(16))) char lds[];
  float* s_v = reinterpret_cast<float*>(lds);                // [M][R] v of the tile
  E* s_b = reinterpret_cast<E*>(lds + sizeof(float) * (size_t)M * a.R);   // [2][U][64 CW][SRB]

  const int b = blockIdx.x;
  const Job& jb = a.jobs[job_of_expand(a, b)];
  const ExpandCoord ec = expand_coord(a, jb, b);
  const TileHdr th = clamp_tile(a, a.tiles[ec.tau]);
  if (th.n <= 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int R = a.R, VW = imin(a.r_c + a.r_u, R);
  const int mb = wave % TB, cq = wave / TB, row = lane & 15, g = lane >> 4;
  const int kt = mb * 16 + row;                              // this lane's token within the tile
  const TokRec tr = clamp_tok(a, a.srt[tile_pos(th, kt)], kt < th.n);
  const int t0 = clamp_tok(a, a.srt[th.i0], true).t;       // masked loads read this token's y row
  const bool has_c = NB > 0 && th.c >= 0;
  E* y = reinterpret_cast<E*>(jb.y);
  const E* btc = reinterpret_cast<const E*>(jb.bt_c);
  const int clo = c_lo(jb, ec.cb), chi = c_hi(jb, ec.cb), nch = c_chunks(jb, ec.cb);
  const int nbj = cdiv(nch, CW);                             // block-chunks
  const int clast = imax(clo, chi - 8);

  struct Batch {
    Vec bc[U][NBC];
    Vec y[U][2];
    Vec u[U][RUP][2];
  };
  auto chunk_col = [&](int j) { return clo + imin(j * CW + cq, nch - 1) * kChunkCols; };
  auto load = [&](Batch& B, int j0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u;
      const int cl = chunk_col(j) + 16 * g;
      if constexpr (kStage) {
        // the block's B_c chunk of block-chunk j: columns [cj, cj + 64 CW), all
        // r_c ranks of each, contiguous in global memory
        const int cj = clo + imin(j, nbj - 1) * kChunkCols * CW;
#pragma unroll
        for (int q = 0; q < NCV; ++q) {
          const int e = 8 * (q * kThreads + tid);            // element of the chunk
          const int o = cj + e / imax(a.r_c, 8), rk = e % imax(a.r_c, 8);
          const E* p = has_c ? btc + btc_off(a, jb, th.c, o, rk) : y + y_off(a, jb, t0, imin(cl, clast));
          B.bc[u][q] = O::load(p);
        }
      } else if constexpr (NB > 0) {
#pragma unroll
        for (int b4 = 0; b4 < 4; ++b4)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
          {
            const E* p = has_c ? btc + btc_off(a, jb, th.c, expand_col(chunk_col(j), row, b4), 32 * ks + 8 * g)
                               : y + y_off(a, jb, t0, imin(cl, clast));
            B.bc[u][b4 * KS + ks] = O::load(p);
          }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) B.y[u][h] = O::load(y + y_off(a, jb, tr.t, imin(cl + 8 * h, clast)));
#pragma unroll
      for (int jj = 0; jj < RUP; ++jj)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int cc = imin(cl + 8 * h, clast);
          const E* p = tr.res ? reinterpret_cast<const E*>(a.pool + bu_byte(a, jb, tr.u, tr.r, jj, cc))
                              : y + y_off(a, jb, t0, cc);
          B.u[u][jj][h] = O::load(p);
        }
    }
  };

  // first loads (they need no v), then v of the tile: the K ranges' partials
  // summed in order
  Batch A;
  load(A, 0);
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
  if constexpr (kStage) {
    // the staged rows' rank padding [r_c, 16 NB) reads as zero
    const int padr = 16 * NB - a.r_c;
    for (int i = tid; i < 2 * U * 64 * CW * padr; i += kThreads) {
      const int r = i / padr, k = a.r_c + i % padr;
      s_b[(size_t)r * SRB + k] = E(0);
    }
  }
  __syncthreads();

  const float gam = __uint_as_float(tr.gamma_bits);
  const float* vrow = s_v + kt * R;
  // centroid v as the MFMA's right operand: column = token, k = ranks
  // 32 ks + 8 g .. + 7, scaled by gamma; ranks past r_c are zero
  Vec vhi[KSL], vlo[KSL];
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
  float vu[RU];
#pragma unroll
  for (int jj = 0; jj < RU; ++jj) vu[jj] = (tr.res && jj < tr.r) ? vrow[a.r_c + jj] : 0.f;

  auto stage = [&](const Batch& B, int half, int j0) {
    if constexpr (kStage) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int cj = clo + imin(j0 + u, nbj - 1) * kChunkCols * CW;
#pragma unroll
        for (int q = 0; q < NCV; ++q) {
          const int e = 8 * (q * kThreads + tid);
          const int rc8 = imax(a.r_c, 8);
          const int oc = e / rc8, rk = e % rc8;              // column of the chunk, first rank
          if (oc < 64 * CW) {
            const int o = oc & 63;
            const int r = (oc >> 6) * 64 + ((o >> 2) & 3) * 16 + (o >> 4) * 4 + (o & 3);
            const bool ok = cj + oc < chi;
            *reinterpret_cast<Vec*>(s_b + ((size_t)(half * U + u) * 64 * CW + r) * SRB + rk) = sel(ok, B.bc[u][q]);
          }
        }
      }
    }
  };
  auto compute = [&](const Batch& B, int half, int j0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u, ch = j * CW + cq;
      const int cl = chunk_col(j) + 16 * g;
      bool cv[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) cv[h] = ch < nch && tr.tok && cl + 8 * h + 8 <= chi;
      f32x4 d[4];
#pragma unroll
      for (int b4 = 0; b4 < 4; ++b4) d[b4] = f32x4{0.f, 0.f, 0.f, 0.f};
      if constexpr (NB > 0) {
        if (has_c) {
#pragma unroll
          for (int b4 = 0; b4 < 4; ++b4)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
              Vec bf;
              if constexpr (kStage)
                bf = *reinterpret_cast<const Vec*>(s_b + ((size_t)(half * U + u) * 64 * CW + cq * 64 + b4 * 16 + row) *
                                                       SRB + 32 * ks + 8 * g);
              else
                bf = B.bc[u][b4 * KS + ks];
              d[b4] = O::mma(bf, vhi[ks], d[b4]);
              if constexpr (kBf16) d[b4] = O::mma(bf, vlo[ks], d[b4]);
            }
        }
      }
      float yf[16];
      O::to_f32(B.y[u][0], yf);
      O::to_f32(B.y[u][1], yf + 8);
#pragma unroll
      for (int b4 = 0; b4 < 4; ++b4)
#pragma unroll
        for (int e = 0; e < 4; ++e) yf[4 * b4 + e] += d[b4][e];
      if constexpr (RU <= 2) {
#pragma unroll
        for (int jj = 0; jj < RU; ++jj) {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            float bu[8];
            O::to_f32(B.u[u][jj][h], bu);
#pragma unroll
            for (int e = 0; e < 8; ++e) yf[8 * h + e] = fmaf(vu[jj], bu[e], yf[8 * h + e]);
          }
        }
      } else {
        // wide residual ranks: this chunk's columns of 8 ranks at a time, loaded together here
#pragma unroll
        for (int j8 = 0; j8 < RU; j8 += 8) {
          Vec bv[8][2];
#pragma unroll
          for (int jj = 0; jj < 8; ++jj)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int cc = imin(cl + 8 * h, clast);
              const E* p = tr.res ? reinterpret_cast<const E*>(a.pool + bu_byte(a, jb, tr.u, tr.r, j8 + jj, cc))
                                  : y + y_off(a, jb, t0, cc);
              bv[jj][h] = O::load(p);
            }
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              float bu[8];
              O::to_f32(bv[jj][h], bu);
#pragma unroll
              for (int e = 0; e < 8; ++e) yf[8 * h + e] = fmaf(vu[j8 + jj], bu[e], yf[8 * h + e]);
            }
          }
        }
      }
      // residual ranks past the first chunk (long-tail adapters): read here
      if (RU == kRankChunk && tr.res && tr.r > RU) {
        for (int rho = RU; rho < tr.r; ++rho) {
          const float vr = vrow[a.r_c + rho];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            float bu[8];
            O::to_f32(O::load(reinterpret_cast<const E*>(a.pool + bu_byte(a, jb, tr.u, tr.r, rho,
                                                                          imin(cl + 8 * h, clast)))), bu);
#pragma unroll
            for (int e = 0; e < 8; ++e) yf[8 * h + e] = fmaf(vr, bu[e], yf[8 * h + e]);
          }
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h)
        if (cv[h]) O::store(y + y_off(a, jb, tr.t, cl + 8 * h), yf + 8 * h);
    }
  };

  if constexpr (sizeof(E) == 4) {
    compute(A, 0, 0);
    for (int j0 = U; j0 < nbj; j0 += U) {
      load(A, j0);
      compute(A, 0, j0);
    }
    return;
  } else {
  Batch Bb;
  if constexpr (kStage) {
    stage(A, 0, 0);
    __syncthreads();
  }
  for (int j0 = 0; j0 < nbj; j0 += 2 * U) {
    load(Bb, j0 + U);
    compute(A, 0, j0);
    if constexpr (kStage) {
      stage(Bb, 1, j0 + U);
      __syncthreads();
    }
    if (j0 + U >= nbj) break;                                // (block-uniform)
    load(A, j0 + 2 * U);
    compute(Bb, 1, j0 + U);
    if constexpr (kStage) {
      stage(A, 0, j0 + 2 * U);
      __syncthreads();
    }
  }
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
size_t shrink_lds() {
  const size_t red = sizeof(float) * (size_t)waves_along<M>() * M * shrink_wc<NB, RU>();
  const size_t stg = staged<E, M, NB>() ? sizeof(E) * 2 * batch_len<E, M, NB, RU>() * 16 * NB * stage_row_a<M>() : 0;
  return red > stg ? red : stg;
}
template <typename E, int M, int NB, int RU>
size_t expand_lds(int R) {
  const size_t stg = staged<E, M, NB>() ? sizeof(E) * 2 * batch_len<E, M, NB, RU>() * 64 * waves_along<M>() *
                                              stage_row_b<NB>()
                                        : 0;
  return sizeof(float) * (size_t)M * R + stg;
}

template <typename E, int M, int NB, int RU>
hipError_t launch_mnr(const ApplyLaunch& a, hipStream_t s, hipEvent_t* ev) {
  launch_k(k_shrink<E, M, NB, RU>, a.shrink_blocks, shrink_lds<E, M, NB, RU>(), s, a, ev ? ev[0] : nullptr,
           ev ? ev[1] : nullptr);
  launch_k(k_expand<E, M, NB, RU>, a.expand_blocks, expand_lds<E, M, NB, RU>(a.R), s, a, ev ? ev[2] : nullptr,
           ev ? ev[3] : nullptr);
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
  const int R = padded_rank(kMaxRc, kMaxRu);
  const size_t need_expand = std::max({expand_lds<uint16_t, 64, 8, kRankChunk>(R), expand_lds<uint16_t, 32, 8, kRankChunk>(R),
                                       expand_lds<uint16_t, 64, 4, 2>(padded_rank(64, 2)),
                                       expand_lds<uint16_t, 32, 4, 2>(padded_rank(64, 2))});
  const size_t need_shrink = std::max({shrink_lds<uint16_t, 64, 8, kRankChunk>(), shrink_lds<uint16_t, 32, 8, kRankChunk>(),
                                       shrink_lds<uint16_t, 64, 4, 2>(), shrink_lds<uint16_t, 32, 4, 2>()});
  const size_t need_plan = sizeof(uint64_t) * kSortChunk + 256;
  const size_t need = std::max(need_expand, std::max(need_shrink, need_plan));
  if ((size_t)lds_max < need) return hipErrorInvalidConfiguration;
  done[device] = true;
  return hipSuccess;
}

}  // namespace salt
