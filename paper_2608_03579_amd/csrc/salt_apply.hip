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
#include <atomic>
#include <mutex>

#include "salt_device.h"
#include "salt_internal.h"
#include "salt_layout.h"

namespace salt {
namespace {

// ---------------------------------------------------------------------------
// shared shapes
// ---------------------------------------------------------------------------
// M tokens per tile = TB token blocks of 16.  A block has waves_of(M) waves:
// four for tiles of up to 32 tokens, eight for 64, one per token block beyond
// (waves_of in salt_layout.h).  They split as
// (token block, K quarter) in the shrink and (token block, column phase) in the
// expand: KW = CW = waves / TB.  With TB > 1 (32-, 64- and 128-token tiles,
// bf16) several waves need the same centroid operand at the same time (A_c in
// the shrink, B_c in the expand); the block then loads it once, cooperatively,
// into an LDS stage from which each wave reads its MFMA fragments, so the
// operand is read from L2 once per M tokens.
template <int M>
constexpr int waves_along() { return waves_of(M) / (M / 16); }
template <int M>
constexpr int threads_of() { return 64 * waves_of(M); }
// Waves per SIMD the kernels for 128-token tiles are compiled for (two blocks
// of 8 waves per compute unit) where their registers fit that without
// spilling: r_c <= 32 with residual ranks up to 2, r_c <= 64 with rank 1.
// Other kernels keep the compiler's choice.
template <typename E, int M, int NB, int RU>
constexpr int min_waves() {
  return (sizeof(E) == 2 && M == 128 && ((NB <= 2 && RU <= 2) || (NB <= 4 && RU <= 1))) ? 4 : 1;
}
template <typename E, int M, int NB>
constexpr bool staged() { return sizeof(E) == 2 && M > 16 && NB > 0; }
// Staged rows carry 8 elements of padding: consecutive rows then start 4 LDS
// banks apart, so a fragment read (16 rows x 16 bytes per 8-lane phase) hits
// every bank once.
template <int M>
constexpr int stage_row_a() { return kStepK * waves_along<M>() + 8; }
template <int NB>
constexpr int stage_row_b() { return 16 * NB + 8; }
template <int NB, int RU>
constexpr int shrink_wc() { return 16 * NB + RU; }
// Block-steps (shrink) or block-chunks (expand) per batch: the loads of one
// batch are in flight while the previous batch computes.  One: a second step
// per batch costs more in occupancy (registers) than it gains in loads in
// flight on every workload measured.
template <typename E, int M, int NB, int RU>
constexpr int depth() { return 1; }


// ---------------------------------------------------------------------------
// shrink
// ---------------------------------------------------------------------------
// Wave w takes token block mb = w % TB and the kStepK-wide steps kq, kq + KW, ...
// (kq = w / TB) of the block's K range: block-step j covers steps j KW .. j KW +
// KW - 1, one per K quarter.  A lane holds token (lane & 15) of its block and,
// of a step, the two 8-element vectors h = 0, 1 at k = 8 (lane >> 4) + kPiece h:
// one load instruction then reads 64 contiguous bytes of each token row.  MFMA
// h multiplies vector h of x and of A_c, so the two MFMAs of a step together
// cover its 64 k.
//
// x and A_c are read through buffer resources (a masked lane reads at kOob and
// gets zeros); the residual rows through per-lane pointers fixed for the whole
// block (a lane without that residual row points at the zero page).  Block-step
// j + 1's per-lane operands are loaded while block-step j computes; with a
// staged A_c, block-step j + 2's A_c slice is loaded while block-step j + 1's is
// written into the other half of the LDS stage, so every wait is for loads that
// were issued a whole block-step earlier.
template <typename E, int M, int NB, int RU>
__global__ void __launch_bounds__(threads_of<M>()) __attribute__((amdgpu_waves_per_eu(min_waves<E, M, NB, RU>(), 8)))
k_shrink(const ApplyLaunch a) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  constexpr int ES = sizeof(E);
  constexpr int TB = M / 16, KW = waves_along<M>(), WC = shrink_wc<NB, RU>();
  constexpr bool kStage = staged<E, M, NB>();
  constexpr int NBL = NB > 0 ? NB : 1;
  constexpr int SR = stage_row_a<M>();                       // elements per staged A_c row
  constexpr int NT = threads_of<M>(), NW = waves_of(M);
  constexpr int PIECES = 16 * NB * 8 * KW;                   // 16-byte pieces of a block-step's A_c slice
  constexpr int NCV = kStage ? (PIECES + NT - 1) / NT : 1;   // staged A_c vectors per thread and block-step
  constexpr int NAC = kStage ? 1 : 2 * NBL;                  // per-lane A_c vectors per step (unstaged)
  constexpr int RUP = RU <= 2 ? RU : 0;                      // residual ranks in the pipelined operands
  constexpr int U = depth<E, M, NB, RU>();
  extern __shared__ __attribute__((aligned(16))) char lds[];
  float* s_red = reinterpret_cast<float*>(lds);              // [KW][M][WC], after the K loop
  E* s_a = reinterpret_cast<E*>(lds);                        // [2][U][16 NB][SR], during the K loop

  const Job& jb = a.jobs[job_of_shrink(a, blockIdx.x)];
  const ShrinkCoord sc = shrink_coord(a, jb, blockIdx.x);
  const TileHdr th = shrink_tile(a, sc.tau);
  if (th.n <= 0) return;                                     // (no tile is empty; the whole block leaves)
  const int in = jb.in;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int mb = wave % TB, kq = wave / TB, row = lane & 15, g = lane >> 4;
  const int kt = mb * 16 + row;                              // this lane's token within the tile
  const TokRec tr = clamp_tok(a, a.srt[tile_pos(th, kt)], kt < th.n);
  const int r0 = sc.q * kRankChunk;                          // first residual rank of this block
  const bool has_c = NB > 0 && th.c >= 0 && sc.q == 0;
  const int klo = k_lo(jb, sc.s), khi = k_hi(jb, sc.s), nst = k_steps(jb, sc.s);
  const int nbs = cdiv(nst, KW);                             // block-steps
  const int klast = imax(0, in - 8);                         // last whole vector of a row

  const Rsrc rx = make_rsrc(jb.x, (uint32_t)((int64_t)a.T * in * ES));
  const Rsrc rac = make_rsrc(has_c ? static_cast<const char*>(jb.at_c) + (int64_t)th.c * a.r_c * in * ES : nullptr,
                             has_c ? (uint32_t)((int64_t)a.r_c * in * ES) : 0u);
  const uint32_t xrow = tr.tok ? (uint32_t)tr.t * (uint32_t)(in * ES) : kOob;
  // residual rows r0 + jj of this lane's slot (the zero page where there is none)
  const char* au[RUP > 0 ? RUP : 1];
#pragma unroll
  for (int jj = 0; jj < RUP; ++jj)
    au[jj] = (tr.res && r0 + jj < tr.r) ? a.pool + atu_byte(a, jb, tr.u, tr.r, r0 + jj, 0) : a.zeros;
  const char* au_wide = tr.res ? a.pool + atu_byte(a, jb, tr.u, tr.r, r0, 0) : a.zeros;

  f32x4 acc[NBL];
#pragma unroll
  for (int nb = 0; nb < NBL; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float accu[RU];
#pragma unroll
  for (int j = 0; j < RU; ++j) accu[j] = 0.f;

  // the per-lane operands of a batch: block-steps j0 .. j0 + U - 1
  struct Ops1 {
    Vec x[U][2];
    Vec u[U][RUP > 0 ? RUP : 1][2];
    Vec ac[U][NAC];
  };
  // first k of this lane's vectors in block-step j (a step past the K range
  // reads nothing: its x offsets are out of range)
  auto lane_k = [&](int j) { return klo + (j * KW + kq) * kStepK + 8 * g; };
  auto load = [&](Ops1& B, int j0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u, kb = lane_k(j);
      const bool step_ok = j * KW + kq < nst;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k = kb + kPiece * h;
        B.x[u][h] = O::bload(rx, oob_unless(step_ok && k + 8 <= khi, xrow + (uint32_t)(k * ES)));
      }
#pragma unroll
      for (int jj = 0; jj < RUP; ++jj)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          B.u[u][jj][h] = O::load(reinterpret_cast<const E*>(au[jj] + imin(kb + kPiece * h, klast) * ES));
      if constexpr (!kStage && NB > 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int k = kb + kPiece * h, r = 16 * nb + row;
            B.ac[u][2 * nb + h] =
                O::bload(rac, oob_unless(step_ok && r < a.r_c && k + 8 <= khi, (uint32_t)((r * in + k) * ES)));
          }
      }
    }
  };
  // the block's A_c slice of block-step j (16 NB ranks x 64 KW k), one 16-byte
  // piece per (thread, q); ranks past r_c and k past the range read as zero
  Vec stg[U][NCV];
  auto load_stage = [&](int j0) {
    if constexpr (kStage) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int kj = klo + (j0 + u) * kStepK * KW;
#pragma unroll
        for (int q = 0; q < NCV; ++q) {
          const int L = q * NT + tid, r = L / (8 * KW), k = kj + 8 * (L % (8 * KW));
          stg[u][q] = O::bload(rac, oob_unless(L < PIECES && r < a.r_c && k + 8 <= khi, (uint32_t)((r * in + k) * ES)));
        }
      }
    }
  };
  auto write_stage = [&](int half) {
    if constexpr (kStage) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int q = 0; q < NCV; ++q) {
          const int L = q * NT + tid, r = L / (8 * KW), c16 = L % (8 * KW);
          if (L < PIECES) *reinterpret_cast<Vec*>(s_a + ((size_t)(half * U + u) * 16 * NB + r) * SR + 8 * c16) = stg[u][q];
        }
    }
  };
  auto compute = [&](const Ops1& B, int half) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if constexpr (NB > 0) {
        if (has_c) {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              Vec af;
              if constexpr (kStage)
                af = *reinterpret_cast<const Vec*>(s_a + ((size_t)(half * U + u) * 16 * NB + 16 * nb + row) * SR +
                                                   kq * kStepK + 8 * g + kPiece * h);
              else
                af = B.ac[u][2 * nb + h];
              acc[nb] = O::mma(B.x[u][h], af, acc[nb]);
            }
        }
      }
      if constexpr (RU <= 2) {
#pragma unroll
        for (int jj = 0; jj < RU; ++jj)
#pragma unroll
          for (int h = 0; h < 2; ++h) accu[jj] = O::dot(B.x[u][h], B.u[u][jj][h], accu[jj]);
      }
    }
  };
  // wide residual ranks: the step's rows of 8 ranks at a time, read in place
  // (U is 1 for wide ranks)
  auto compute_wide = [&](const Ops1& B, int j) {
    if constexpr (RU > 2) {
      static_assert(U == 1, "wide residual ranks run one block-step per batch");
      const int kb = lane_k(j);
      const int64_t rs = (int64_t)in * ES;
#pragma unroll
      for (int j8 = 0; j8 < RU; j8 += 8) {
        Vec uv[8][2];
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const char* base = (tr.res && r0 + j8 + jj < tr.r) ? au_wide + (j8 + jj) * rs : a.zeros;
#pragma unroll
          for (int h = 0; h < 2; ++h)
            uv[jj][h] = O::load(reinterpret_cast<const E*>(base + imin(kb + kPiece * h, klast) * ES));
        }
#pragma unroll
        for (int jj = 0; jj < 8; ++jj)
#pragma unroll
          for (int h = 0; h < 2; ++h) accu[j8 + jj] = O::dot(B.x[0][h], uv[jj][h], accu[j8 + jj]);
      }
    }
  };

  Ops1 A;
  if constexpr (ES == 4) {
    // fp32: one set of operands, loaded then used (its vectors are twice as wide)
    for (int j = 0; j < nbs; ++j) {
      load(A, j);
      compute(A, 0);
      compute_wide(A, j);
    }
  } else {
    Ops1 Bb;
    load_stage(0);
    load(A, 0);
    write_stage(0);
    load_stage(U);
    if constexpr (kStage) __syncthreads();
    for (int j = 0; j < nbs; j += 2 * U) {
      load(Bb, j + U);
      write_stage(1);
      load_stage(j + 2 * U);
      compute(A, 0);
      compute_wide(A, j);
      if constexpr (kStage) __syncthreads();
      if (j + U >= nbs) break;                               // (block-uniform)
      load(A, j + 2 * U);
      write_stage(0);
      load_stage(j + 3 * U);
      compute(Bb, 1);
      compute_wide(Bb, j + U);
      if constexpr (kStage) __syncthreads();
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
  const Rsrc rp = make_rsrc(a.partials + jb.poff, (uint32_t)((int64_t)jb.S * a.T * a.R * 4));
  for (int k = wave; k < th.n; k += NW) {
    for (int cc = lane; cc < ncols; cc += 64) {
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
      buf_store_f32(rp, (uint32_t)(part_off(a, jb, sc.s, th.i0 + k, col) - jb.poff) * 4u, v);
    }
  }
}

// ---------------------------------------------------------------------------
// expand
// ---------------------------------------------------------------------------
// Wave w takes token block mb = w % TB and, in block-chunk j, the 64-column chunk
// j CW + cq (cq = w / TB) of the block's columns.  Per chunk the centroid part is
// four 16 x 16 MFMA tiles D[col][token] = Bt_c[col][:] . v_c[token][:]; A-operand
// row i of tile b4 is column expand_col(col0, i, b4), so that output lane (token
// = lane & 15, g = lane >> 4) holds the columns col0 + 8 g + kPiece h + 0..7, h =
// 0, 1, of its token: each y load or store instruction covers 64 contiguous bytes
// (bf16) of every token row.  A staged B_c chunk keeps the columns in that MFMA
// order (LDS row of column o: 64 (o / 64) + 16 b4 + i), so a fragment read takes
// 16 consecutive rows.
// y and B_c go through buffer resources (masked lanes load zeros at kOob, and
// their stores are dropped), the residual rows through per-lane pointers; the
// loads are pipelined one block-chunk ahead as in the shrink.
template <typename E, int M, int NB, int RU>
__device__ __forceinline__ void expand_segment(const ApplyLaunch& a, const ExpandSeg& sg, char* lds) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  constexpr int ES = sizeof(E);
  constexpr bool kBf16 = ES == 2;
  constexpr int TB = M / 16, CW = waves_along<M>(), KS = (NB + 1) / 2;
  constexpr bool kStage = staged<E, M, NB>();
  constexpr int KSL = KS > 0 ? KS : 1;
  constexpr int SRB = stage_row_b<NB>();                     // elements per staged B_c row (one column)
  constexpr int NT = threads_of<M>();
  constexpr int NCV = kStage ? (128 * CW * NB + NT - 1) / NT : 1;   // staged B_c vectors per thread and block-chunk
  constexpr int NBC = kStage ? 1 : 4 * KSL;                  // per-lane B_c vectors per chunk (unstaged)
  constexpr int RUP = RU <= 2 ? RU : 0;                      // residual ranks in the pipelined operands
  constexpr int U = depth<E, M, NB, RU>();
  float* s_v = reinterpret_cast<float*>(lds);                // [M][R] v of the tile

  const Job& jb = a.jobs[sg.job];
  const TileHdr th = expand_tile(a, sg.tau);
  if (th.n <= 0) return;                                     // (no tile is empty)
  const int out = jb.out;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int R = a.R, VW = imin(a.r_c + a.r_u, R);
  const int mb = wave % TB, cq = wave / TB, row = lane & 15, g = lane >> 4;
  const int kt = mb * 16 + row;                              // this lane's token within the tile
  const TokRec tr = clamp_tok(a, a.srt[tile_pos(th, kt)], kt < th.n);
  const bool has_c = NB > 0 && th.c >= 0;
  // the segment's columns: block-chunks [j0, j1) of the tile
  const int clo = imin(out, sg.j0 * jb.cpb), chi = imin(out, sg.j1 * jb.cpb);
  const int nch = cdiv(chi - clo, kChunkCols);               // 64-column chunks
  const int nbj = cdiv(nch, CW);                             // block-chunks
  const int olast = imax(0, out - 8);
  // residual ranks past the first chunk (long-tail adapters) are read from s_v
  // inside the column loop, so the stage then sits after it; otherwise s_v is
  // dead once v is in registers and the stage takes its place
  const bool long_tail = RU == kRankChunk && a.r_u > RU;
  E* s_b = reinterpret_cast<E*>(lds + (long_tail ? sizeof(float) * (size_t)M * R : 0));   // [2][U][64 CW][SRB]

  const Rsrc ry = make_rsrc(jb.y, (uint32_t)((int64_t)a.T * out * ES));
  const Rsrc rb = make_rsrc(has_c ? static_cast<const char*>(jb.bt_c) + (int64_t)th.c * out * a.r_c * ES : nullptr,
                            has_c ? (uint32_t)((int64_t)out * a.r_c * ES) : 0u);
  const uint32_t yrow = tr.tok ? (uint32_t)tr.t * (uint32_t)(out * ES) : kOob;
  const char* bu[RUP > 0 ? RUP : 1];
#pragma unroll
  for (int jj = 0; jj < RUP; ++jj)
    bu[jj] = (tr.res && jj < tr.r) ? a.pool + bu_byte(a, jb, tr.u, tr.r, jj, 0) : a.zeros;
  const char* bu_wide = tr.res ? a.pool + bu_byte(a, jb, tr.u, tr.r, 0, 0) : a.zeros;

  // the per-lane operands of a batch: block-chunks j0 .. j0 + U - 1
  struct Ops1 {
    Vec y[U][2];
    Vec u[U][RUP > 0 ? RUP : 1][2];
    Vec bc[U][NBC];
  };
  // this lane's first column in block-chunk j
  auto lane_col = [&](int j) { return clo + (j * CW + cq) * kChunkCols + 8 * g; };
  auto y_off = [&](int j, int h) {
    const int col = lane_col(j) + kPiece * h;
    return oob_unless(j * CW + cq < nch && col + 8 <= chi, yrow + (uint32_t)(col * ES));
  };
  auto load = [&](Ops1& B, int j0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u, cl = lane_col(j);
#pragma unroll
      for (int h = 0; h < 2; ++h) B.y[u][h] = O::bload(ry, y_off(j, h));
#pragma unroll
      for (int jj = 0; jj < RUP; ++jj)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          B.u[u][jj][h] = O::load(reinterpret_cast<const E*>(bu[jj] + imin(cl + kPiece * h, olast) * ES));
      if constexpr (!kStage && NB > 0) {
        const bool chunk_ok = j * CW + cq < nch;
        const int col0 = clo + (j * CW + cq) * kChunkCols;
#pragma unroll
        for (int b4 = 0; b4 < 4; ++b4)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const int o = expand_col(col0, row, b4), rk = 32 * ks + 8 * g;
            B.bc[u][b4 * KS + ks] =
                O::bload(rb, oob_unless(chunk_ok && o < chi && rk < a.r_c, (uint32_t)((o * a.r_c + rk) * ES)));
          }
      }
    }
  };
  // the block's B_c chunk of block-chunk j: columns [cj, cj + 64 CW), all r_c
  // ranks of each, contiguous in global memory; thread piece q holds the 8
  // ranks from st_rk[q] of chunk column st_oc[q] (fixed for the block)
  Vec stg[U][NCV];
  int st_oc[NCV], st_rk[NCV];
  if constexpr (kStage) {
    const int rc8 = imax(a.r_c, 8);
#pragma unroll
    for (int q = 0; q < NCV; ++q) {
      const int e = 8 * (q * NT + tid);
      st_oc[q] = e / rc8;
      st_rk[q] = e - st_oc[q] * rc8;
    }
  }
  auto load_stage = [&](int j0) {
    if constexpr (kStage) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int cj = clo + (j0 + u) * kChunkCols * CW;
#pragma unroll
        for (int q = 0; q < NCV; ++q) {
          const bool ok = st_oc[q] < kChunkCols * CW && cj + st_oc[q] < chi;
          stg[u][q] = O::bload(rb, oob_unless(ok, (uint32_t)(((cj + st_oc[q]) * a.r_c + st_rk[q]) * ES)));
        }
      }
    }
  };
  auto write_stage = [&](int half) {
    if constexpr (kStage) {
#pragma unroll
      for (int q = 0; q < NCV; ++q) {
        const int oc = st_oc[q];
        if (oc < kChunkCols * CW) {
          const int o = oc & 63;
          const int r = (oc >> 6) * 64 + (2 * (o >> 5) + ((o >> 2) & 1)) * 16 + 4 * ((o >> 3) & 3) + (o & 3);
#pragma unroll
          for (int u = 0; u < U; ++u)
            *reinterpret_cast<Vec*>(s_b + ((size_t)(half * U + u) * 64 * CW + r) * SRB + st_rk[q]) = stg[u][q];
        }
      }
    }
  };

  // first loads (they need no v), then v of the tile: the K ranges' partials
  // summed in order
  Ops1 A;
  load_stage(0);
  load(A, 0);
  {
    // the tile's rows of one K range are contiguous: (n R / 4) float4 from row
    // i0; per pass, thread t sums float4 q0 + t and q0 + t + NT over the
    // K ranges in order, with four K ranges' loads in flight at a time (rows
    // past n read zero)
    const Rsrc rp = make_rsrc(a.partials + jb.poff, (uint32_t)((int64_t)jb.S * a.T * a.R * 4));
    const uint32_t sstride = (uint32_t)a.T * (uint32_t)R * 4u;
    const uint32_t tile0 = (uint32_t)th.i0 * (uint32_t)R * 4u;
    const int n4 = th.n * R / 4, m4 = M * R / 4;
    constexpr int QMAX = 2;                                  // float4 per thread and pass
    for (int q0 = tid; q0 < m4; q0 += QMAX * NT) {
      float4 v[QMAX];
      uint32_t off[QMAX];
#pragma unroll
      for (int i = 0; i < QMAX; ++i) {
        const int q = q0 + i * NT;
        v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        off[i] = oob_unless(q < n4, tile0 + 16u * (uint32_t)q);
      }
      int sl = 0;
      for (; sl + 4 <= jb.S; sl += 4) {
        float4 p[4][QMAX];
#pragma unroll
        for (int d = 0; d < 4; ++d)
#pragma unroll
          for (int i = 0; i < QMAX; ++i) p[d][i] = buf_load_f32x4(rp, off[i] + (uint32_t)(sl + d) * sstride);
#pragma unroll
        for (int d = 0; d < 4; ++d)
#pragma unroll
          for (int i = 0; i < QMAX; ++i) v[i] = f4_add(v[i], p[d][i]);
      }
      for (; sl < jb.S; ++sl) {
        float4 p[QMAX];
#pragma unroll
        for (int i = 0; i < QMAX; ++i) p[i] = buf_load_f32x4(rp, off[i] + (uint32_t)sl * sstride);
#pragma unroll
        for (int i = 0; i < QMAX; ++i) v[i] = f4_add(v[i], p[i]);
      }
#pragma unroll
      for (int i = 0; i < QMAX; ++i) {
        const int q = q0 + i * NT;
        if (q < m4) reinterpret_cast<float4*>(s_v)[q] = v[i];
      }
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
    // (r_c is a multiple of 8: a group of 8 ranks is wholly inside or past it)
    float4 va = make_float4(0.f, 0.f, 0.f, 0.f), vb = va;
    if (tr.tok && 32 * ks + 8 * g < a.r_c) {
      va = reinterpret_cast<const float4*>(vrow + 32 * ks + 8 * g)[0];
      vb = reinterpret_cast<const float4*>(vrow + 32 * ks + 8 * g)[1];
    }
    float f[8] = {va.x * gam, va.y * gam, va.z * gam, va.w * gam, vb.x * gam, vb.y * gam, vb.z * gam, vb.w * gam};
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
  if constexpr (kStage) {
    __syncthreads();
    // the staged rows' rank padding [r_c, 16 NB) reads as zero
    const int padr = 16 * NB - a.r_c;
    for (int i = tid; i < 2 * U * 64 * CW * padr; i += NT) {
      const int r = i / padr, k = a.r_c + i % padr;
      s_b[(size_t)r * SRB + k] = E(0);
    }
    write_stage(0);
    load_stage(U);
    __syncthreads();
  }

  auto compute1 = [&](const Ops1& B, int half, int u, int j) {
    const int cl = lane_col(j);
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
      for (int jj = 0; jj < RU; ++jj)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          float b[8];
          O::to_f32(B.u[u][jj][h], b);
#pragma unroll
          for (int e = 0; e < 8; ++e) yf[8 * h + e] = fmaf(vu[jj], b[e], yf[8 * h + e]);
        }
    } else {
      // wide residual ranks: this chunk's columns of 8 ranks at a time, read in place
      const int64_t rs = (int64_t)out * ES;
#pragma unroll
      for (int j8 = 0; j8 < RU; j8 += 8) {
        Vec bv[8][2];
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const char* base = (tr.res && j8 + jj < tr.r) ? bu_wide + (j8 + jj) * rs : a.zeros;
#pragma unroll
          for (int h = 0; h < 2; ++h)
            bv[jj][h] = O::load(reinterpret_cast<const E*>(base + imin(cl + kPiece * h, olast) * ES));
        }
#pragma unroll
        for (int jj = 0; jj < 8; ++jj)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            float b[8];
            O::to_f32(bv[jj][h], b);
#pragma unroll
            for (int e = 0; e < 8; ++e) yf[8 * h + e] = fmaf(vu[j8 + jj], b[e], yf[8 * h + e]);
          }
      }
      if (long_tail) {
        // ranks past the first chunk (their v from s_v), eight rows at a time up
        // to the batch's largest rank, so that eight rows' loads are in flight
        // together; a lane past its own rank reads the zero page with a zero v
        for (int r8 = RU; r8 < a.r_u; r8 += 8) {
          Vec bv[8][2];
          float vr[8];
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) {
            const int rho = r8 + jj;
            const bool ok = tr.res && rho < tr.r;
            const char* base = ok ? bu_wide + rho * rs : a.zeros;
            vr[jj] = ok ? vrow[a.r_c + rho] : 0.f;
#pragma unroll
            for (int h = 0; h < 2; ++h)
              bv[jj][h] = O::load(reinterpret_cast<const E*>(base + imin(cl + kPiece * h, olast) * ES));
          }
#pragma unroll
          for (int jj = 0; jj < 8; ++jj)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              float b[8];
              O::to_f32(bv[jj][h], b);
#pragma unroll
              for (int e = 0; e < 8; ++e) yf[8 * h + e] = fmaf(vr[jj], b[e], yf[8 * h + e]);
            }
        }
      }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) O::bstore(ry, y_off(j, h), yf + 8 * h);
  };
  auto compute = [&](const Ops1& B, int half, int j0) {
#pragma unroll
    for (int u = 0; u < U; ++u) compute1(B, half, u, j0 + u);
  };

  if constexpr (ES == 4) {
    compute(A, 0, 0);
    for (int j = U; j < nbj; j += U) {
      load(A, j);
      compute(A, 0, j);
    }
  } else {
    Ops1 Bb;
    for (int j = 0; j < nbj; j += 2 * U) {
      load(Bb, j + U);
      write_stage(1);
      load_stage(j + 2 * U);
      compute(A, 0, j);
      if constexpr (kStage) __syncthreads();
      if (j + U >= nbj) break;                               // (block-uniform)
      load(A, j + 2 * U);
      write_stage(0);
      load_stage(j + 3 * U);
      compute(Bb, 1, j + U);
      if constexpr (kStage) __syncthreads();
    }
  }
}

// One round of blocks; block b walks its contiguous share of the launch's work
// items segment by segment (a segment: the block-chunks of one tile).  Every
// segment starts behind a block barrier, so its LDS writes never meet the
// previous segment's reads.
template <typename E, int M, int NB, int RU>
__global__ void __launch_bounds__(threads_of<M>()) __attribute__((amdgpu_waves_per_eu(min_waves<E, M, NB, RU>(), 8)))
k_expand(const ApplyLaunch a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int end = expand_begin(a, blockIdx.x + 1, gridDim.x);
  for (int pos = expand_begin(a, blockIdx.x, gridDim.x); pos < end;) {
    const ExpandSeg sg = expand_seg(a, pos, end);
    __syncthreads();
    expand_segment<E, M, NB, RU>(a, sg, lds);
    pos += sg.j1 - sg.j0;                                    // (>= 1)
  }
}

// ---------------------------------------------------------------------------
// launch
// ---------------------------------------------------------------------------
template <typename K>
void launch_k(K kernel, int blocks, int threads, size_t lds, hipStream_t s, const ApplyLaunch& a, hipEvent_t e0,
              hipEvent_t e1) {
  if (e0 || e1) hipExtLaunchKernelGGL(kernel, dim3(blocks), dim3(threads), (uint32_t)lds, s, e0, e1, 0u, a);
  else hipLaunchKernelGGL(kernel, dim3(blocks), dim3(threads), lds, s, a);
}

template <typename E, int M, int NB, int RU>
size_t shrink_lds() {
  const size_t red = sizeof(float) * (size_t)waves_along<M>() * M * shrink_wc<NB, RU>();
  const size_t stg = staged<E, M, NB>() ? sizeof(E) * 2 * depth<E, M, NB, RU>() * 16 * NB * stage_row_a<M>() : 0;
  return red > stg ? red : stg;
}
template <typename E, int M, int NB, int RU>
size_t expand_lds(int R, int r_u) {
  const size_t stg =
      staged<E, M, NB>() ? sizeof(E) * 2 * depth<E, M, NB, RU>() * 64 * waves_along<M>() * stage_row_b<NB>() : 0;
  const size_t sv = sizeof(float) * (size_t)M * R;
  // the stage takes the place of v unless long-tail ranks read v in the column loop
  return (RU == kRankChunk && r_u > RU) ? sv + stg : std::max(sv, stg);
}

// Blocks of `kernel` with `lds` bytes of LDS that one compute unit holds at once
// (cached per kernel for the last LDS size asked).
template <typename K>
int resident_blocks(K kernel, int threads, size_t lds) {
  static std::atomic<uint64_t> cache{0};                     // (lds << 32) | blocks
  const uint64_t c = cache.load(std::memory_order_relaxed);
  if (c != 0 && (c >> 32) == (uint64_t)lds) return (int)(c & 0xffffffffu);
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(kernel), threads, lds) !=
          hipSuccess ||
      n < 1) {
    (void)hipGetLastError();
    n = 1;
  }
  cache.store(((uint64_t)lds << 32) | (uint32_t)n, std::memory_order_relaxed);
  return n;
}

template <typename E, int M, int NB, int RU>
hipError_t launch_mnr(const ApplyLaunch& a, hipStream_t s, hipEvent_t* ev) {
  constexpr int NT = threads_of<M>();
  constexpr int MS = M > 64 ? 64 : M;                         // tokens per shrink tile
  if (a.MS != MS) return hipErrorInvalidValue;
  launch_k(k_shrink<E, MS, NB, RU>, a.shrink_blocks, threads_of<MS>(), shrink_lds<E, MS, NB, RU>(), s, a,
           ev ? ev[0] : nullptr, ev ? ev[1] : nullptr);
  const size_t lds = expand_lds<E, M, NB, RU>(a.R, a.r_u);
  const int round = resident_blocks(k_expand<E, M, NB, RU>, NT, lds) * std::max(1, a.n_cu);
  launch_k(k_expand<E, M, NB, RU>, std::min(a.expand_items, round), NT, lds, s, a, ev ? ev[2] : nullptr,
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

template <typename E, int MS>
int shrink_round_m(const ApplyLaunch& a) {
  auto round = [&](auto kernel, size_t lds) { return resident_blocks(kernel, threads_of<MS>(), lds) * std::max(1, a.n_cu); };
  const int nb = centroid_blocks(a.r_c);
  const int ru = a.r_u <= 1 ? 1 : (a.r_u <= 2 ? 2 : kRankChunk);
#define SALT_ROUND(NB_, RU_) \
  if (nb == NB_ && ru == RU_) return round(k_shrink<E, MS, NB_, RU_>, shrink_lds<E, MS, NB_, RU_>());
  SALT_ROUND(0, 1) SALT_ROUND(0, 2) SALT_ROUND(0, kRankChunk)
  SALT_ROUND(2, 1) SALT_ROUND(2, 2) SALT_ROUND(2, kRankChunk)
  SALT_ROUND(4, 1) SALT_ROUND(4, 2) SALT_ROUND(4, kRankChunk)
  SALT_ROUND(8, 1) SALT_ROUND(8, 2) SALT_ROUND(8, kRankChunk)
#undef SALT_ROUND
  return 0;
}

}  // namespace

int shrink_round_blocks(const ApplyLaunch& a) {
  if (a.esize == 4) return shrink_round_m<float, 16>(a);
  switch (a.MS) {
    case 16: return shrink_round_m<uint16_t, 16>(a);
    case 32: return shrink_round_m<uint16_t, 32>(a);
    case 64: return shrink_round_m<uint16_t, 64>(a);
    default: return 0;
  }
}

hipError_t launch_apply(const ApplyLaunch& a, hipStream_t s, hipEvent_t* ev) {
  if (a.T <= 0 || a.n_tiles <= 0 || a.n_jobs <= 0) return hipSuccess;
  if (a.n_jobs > kMaxJobs || a.shrink_blocks <= 0 || a.expand_items <= 0 || a.r_c > kMaxRc || a.r_u > kMaxRu)
    return hipErrorInvalidValue;
  if (a.esize == 4) {
    if (a.M != 16) return hipErrorInvalidValue;
    return launch_m<float, 16>(a, s, ev);
  }
  switch (a.M) {
    case 16: return launch_m<uint16_t, 16>(a, s, ev);
    case 32: return launch_m<uint16_t, 32>(a, s, ev);
    case 64: return launch_m<uint16_t, 64>(a, s, ev);
    case 128: return launch_m<uint16_t, 128>(a, s, ev);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace salt

namespace salt {

// Device scratch of salt_apply_batch_noalloc: the split-K partial sums of its
// launches.  Each device that runs the library holds its own copy until the
// process ends; its device address is resolved once per device, in
// kernels_init, and only that address is ever handed to a kernel.
static __device__ __align__(256) float scratch[kScratchFloats];

namespace {
std::mutex g_init_mu;
bool g_init_done[kMaxDevices] = {};
float* g_scratch[kMaxDevices] = {};
}  // namespace

// Per-device set-up: checks that a workgroup may hold the LDS the apply and
// plan kernels ask for (the expand of 64-token tiles at the largest ranks), and
// resolves this device's copy of the scratch array.  Call with `device` current.
hipError_t kernels_init(int device) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_init_mu);
  if (g_init_done[device]) return hipSuccess;
  int lds_max = 0;
  hipError_t e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, device);
  if (e != hipSuccess) return e;
  const int R = padded_rank(kMaxRc, kMaxRu);
  const size_t need_expand = std::max({expand_lds<uint16_t, 64, 8, kRankChunk>(R, kMaxRu),
                                       expand_lds<uint16_t, 32, 8, kRankChunk>(R, kMaxRu),
                                       expand_lds<uint16_t, 128, 8, kRankChunk>(R, kMaxRu),
                                       expand_lds<uint16_t, 128, 4, 2>(padded_rank(64, 2), 2),
                                       expand_lds<uint16_t, 64, 4, 2>(padded_rank(64, 2), 2),
                                       expand_lds<uint16_t, 32, 4, 2>(padded_rank(64, 2), 2)});
  const size_t need_shrink = std::max({shrink_lds<uint16_t, 128, 8, kRankChunk>(),
                                       shrink_lds<uint16_t, 64, 8, kRankChunk>(), shrink_lds<uint16_t, 32, 8, kRankChunk>(),
                                       shrink_lds<uint16_t, 64, 4, 2>(), shrink_lds<uint16_t, 32, 4, 2>()});
  const size_t need_plan = (sizeof(uint64_t) + sizeof(int) + 1) * kSortChunk + 256;
  const size_t need = std::max(need_expand, std::max(need_shrink, need_plan));
  if ((size_t)lds_max < need) return hipErrorInvalidConfiguration;
  float* p = nullptr;
  e = hipGetSymbolAddress(reinterpret_cast<void**>(&p), HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!p) return hipErrorInvalidSymbol;
  g_scratch[device] = p;
  g_init_done[device] = true;
  return hipSuccess;
}

float* static_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> g(g_init_mu);
  return g_init_done[device] ? g_scratch[device] : nullptr;
}

}  // namespace salt
