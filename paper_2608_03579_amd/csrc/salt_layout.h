// Launch records and index arithmetic of the apply kernels, shared by the HIP
// kernels and by host code (the runtime that fills the records, and a plain
// C++ build of this header that walks every block of a launch and checks each
// address against its buffer).  No HIP types: it compiles with g++ as well.
//
// Every global address an apply kernel forms is `base + offset`, with the
// offset computed here from indices that are first clamped into the range of
// their buffer (token < T, slot < n_slots, rank < rank of the slot, column <
// out, k < in, sorted position < T).  A value read from device memory (a token
// record, a tile header) can therefore never move an access outside the
// allocation it belongs to, whatever it holds.
#pragma once

#include <stdint.h>

// SALT_HOST_ONLY: a plain C++ build (no HIP headers) for host-side checks.
#if defined(SALT_HOST_ONLY)
#define SALT_HD inline
struct int4 {
  int x, y, z, w;
};
#else
#include <hip/hip_runtime.h>
#define SALT_HD __host__ __device__ __forceinline__
#endif

namespace salt {

// ---- fixed shapes -----------------------------------------------------------
constexpr int kWaves = 4;            // waves of an apply block for tiles of up to 32 tokens
constexpr int kStepK = 64;           // k elements one wave takes per shrink step
constexpr int kChunkCols = 64;       // output columns one wave takes per expand chunk
constexpr int kMaxJobs = 16;         // tables one apply launch serves
constexpr int kRankChunk = 16;       // residual ranks one shrink block accumulates
constexpr int kMaxRc = 128;          // largest centroid rank
constexpr int kMaxRu = 72;           // largest residual rank (long-tail concatenated adapters)
constexpr int kMaxC = 64;            // largest centroid library
constexpr int kMaxTokens = 65536;    // largest batch of one plan
constexpr int kSortChunk = 4096;     // keys one plan block sorts in LDS
constexpr int64_t kMaxBufferBytes = (int64_t)1 << 31;   // bound of every buffer an apply kernel addresses with 32-bit offsets

SALT_HD int imin(int a, int b) { return a < b ? a : b; }
SALT_HD int imax(int a, int b) { return a > b ? a : b; }
SALT_HD int iclamp(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }
SALT_HD int cdiv(int a, int b) { return (a + b - 1) / b; }

// Waves of an apply block for tiles of M tokens: four for up to 32 tokens,
// eight for 64 (two per 16-token block: two K halves in the shrink, two column
// phases in the expand), one per 16-token block beyond.
SALT_HD constexpr int waves_of(int M) { return M > 64 ? M / 16 : (M == 64 ? 2 * kWaves : kWaves); }

// Row stride of the split-K partials: r_c + r_u rounded up to whole float4s.
SALT_HD int padded_rank(int r_c, int r_u) {
  const int r = r_c + r_u;
  return r < 4 ? 4 : (r + 3) / 4 * 4;
}

// ---- records ------------------------------------------------------------------
// A tile is a run of at most M sorted tokens of one centroid group: header
// (first sorted position i0, token count n, centroid c or -1, 0).  A token
// record at sorted position p is (token t, slot u or -1, residual rank r,
// gamma bits).

// One table served by an apply launch.
struct Job {
  const void* x;           // [T][in], caller-owned
  void* y;                 // [T][out], caller-owned
  const void* at_c;        // [C][r_c][in]   centroid A, transposed
  const void* bt_c;        // [C][out][r_c]  centroid B, transposed
  int64_t prefix;          // sum of (in + out) over the context's earlier tables
  int64_t poff;            // first float of this job's partials
  int32_t in, out;
  int32_t S;               // K ranges of the shrink
  int32_t Kc;              // length of one K range (a multiple of kStepK)
  int32_t cpb;             // output columns of one expand block-chunk (kChunkCols x the waves along the columns)
  int32_t n_col;           // expand block-chunks per tile: cdiv(out, cpb)
  int32_t shrink_base;     // first shrink block of this job
  int32_t expand_base;     // first expand work item of this job
};

struct ApplyLaunch {
  Job jobs[kMaxJobs];
  const int4* tiles;       // [n_tiles]
  const int4* srt;         // [T] token records in sorted order
  const char* pool;        // residual slot pool
  float* partials;         // split-K partial sums
  const char* zeros;       // zero page: >= max(in, out) * esize bytes of zeros (read in place of missing residual rows)
  int64_t slot_stride;     // bytes between slots
  int64_t partial_cap;     // floats of `partials`
  int32_t n_jobs;
  int32_t T;
  int32_t n_tiles;
  const int4* stiles;      // [n_stiles] the shrink's tiles (the expand's tiles unless those exceed 64 tokens)
  int32_t n_stiles;
  int32_t MS;              // tokens per shrink tile (min(M, 64))
  int32_t M;               // tokens per tile (16, 32 or 64)
  int32_t C, r_c;
  int32_t n_slots;
  int32_t r_u;             // largest residual rank of the batch (<= kMaxRu)
  int32_t nq;              // residual rank chunks: ceil(r_u / kRankChunk), >= 1
  int32_t R;               // partial row stride, padded_rank(r_c, r_u)
  int32_t esize;           // bytes per element (2: bf16, 4: fp32)
  int32_t shrink_blocks;
  int32_t expand_items;    // expand work items: sum over jobs of n_tiles x n_col
  int32_t n_cu;            // compute units of the device (sizes the expand grid)
};

struct TileHdr {
  int i0, n, c;
};
struct TokRec {
  int t, u, r;
  uint32_t gamma_bits;
  bool tok;                // a real token of the tile
  bool res;                // has a residual term (slot >= 0, rank > 0)
};

// A tile header with every field clamped: 0 <= i0 < T, 0 <= n <= min(M, T -
// i0), -1 <= c < C (M: the tile size of the list it comes from).
SALT_HD TileHdr clamp_tile(const ApplyLaunch& a, int4 h, int M) {
  TileHdr r;
  r.i0 = iclamp(h.x, 0, imax(a.T - 1, 0));
  r.n = iclamp(h.y, 0, imin(M, a.T - r.i0));
  r.c = (a.r_c > 0) ? iclamp(h.z, -1, a.C - 1) : -1;
  return r;
}

// Token k of a tile (k >= n reads the tile's first token and is not a real one).
SALT_HD int tile_pos(const TileHdr& h, int k) { return h.i0 + (k < h.n ? k : 0); }

SALT_HD TokRec clamp_tok(const ApplyLaunch& a, int4 rec, bool real) {
  TokRec r;
  r.t = iclamp(rec.x, 0, a.T - 1);
  r.u = iclamp(rec.y, -1, a.n_slots - 1);
  r.r = (r.u >= 0) ? iclamp(rec.z, 0, a.r_u) : 0;
  r.gamma_bits = (uint32_t)rec.w;
  r.tok = real;
  r.res = real && r.u >= 0 && r.r > 0;
  return r;
}

// ---- block decomposition ----------------------------------------------------------
SALT_HD int job_of_shrink(const ApplyLaunch& a, int b) {
  int j = 0;
  while (j + 1 < a.n_jobs && b >= a.jobs[j + 1].shrink_base) ++j;
  return j;
}
SALT_HD int job_of_expand(const ApplyLaunch& a, int b) {
  int j = 0;
  while (j + 1 < a.n_jobs && b >= a.jobs[j + 1].expand_base) ++j;
  return j;
}

// Shrink item i of job j: shrink tile tau, K range s, residual rank chunk q
// (items of a job: (q, s, tau) with tau fastest).
struct ShrinkCoord {
  int tau, s, q;
};
SALT_HD int shrink_tiles(const ApplyLaunch& a) { return a.n_stiles; }
SALT_HD ShrinkCoord shrink_coord(const ApplyLaunch& a, const Job& jb, int item) {
  const int local = item - jb.shrink_base, nt = imax(shrink_tiles(a), 1);
  ShrinkCoord c;
  c.tau = local % nt;
  const int rest = local / nt;
  c.s = rest % jb.S;
  c.q = iclamp(rest / jb.S, 0, a.nq - 1);
  return c;
}
SALT_HD TileHdr shrink_tile(const ApplyLaunch& a, int tau) {
  return clamp_tile(a, a.stiles[iclamp(tau, 0, a.n_stiles - 1)], a.MS);
}
SALT_HD TileHdr expand_tile(const ApplyLaunch& a, int tau) {
  return clamp_tile(a, a.tiles[iclamp(tau, 0, a.n_tiles - 1)], a.M);
}

// Expand work items: (job, tile, block-chunk), job-major, then tile, block-chunk
// fastest; block-chunk bc of a job covers columns [bc cpb, min(out, (bc + 1)
// cpb)).  A launch of G blocks gives block b the contiguous items [b N / G,
// (b + 1) N / G), N = expand_items, so every block carries the same number of
// block-chunks (to within one) and walks them tile by tile, reading a tile's v
// once per visit.
SALT_HD int expand_begin(const ApplyLaunch& a, int b, int G) {
  return (int)((int64_t)iclamp(b, 0, G) * a.expand_items / imax(G, 1));
}
// Block-chunks [j0, j1) of tile tau of job `job`: the run of items that starts at
// item pos and ends at the tile's last block-chunk or at item end, whichever
// comes first (pos < end).
struct ExpandSeg {
  int job, tau, j0, j1;
};
SALT_HD ExpandSeg expand_seg(const ApplyLaunch& a, int pos, int end) {
  ExpandSeg sg;
  sg.job = job_of_expand(a, pos);
  const Job& jb = a.jobs[sg.job];
  const int local = imax(0, pos - jb.expand_base), nc = imax(jb.n_col, 1);
  sg.tau = iclamp(local / nc, 0, a.n_tiles - 1);
  sg.j0 = local - (local / nc) * nc;
  sg.j1 = imin(nc, sg.j0 + imax(1, end - pos));
  return sg;
}

// ---- element offsets (in elements of the context dtype unless stated) --------------
// x[t][k .. k+7]: k clamped to a whole 8-element vector inside the row.
SALT_HD int64_t x_off(const ApplyLaunch& a, const Job& jb, int t, int k) {
  return (int64_t)iclamp(t, 0, a.T - 1) * jb.in + iclamp(k, 0, jb.in - 8);
}
// A_c^T[c][j][k .. k+7]
SALT_HD int64_t atc_off(const ApplyLaunch& a, const Job& jb, int c, int j, int k) {
  return ((int64_t)iclamp(c, 0, a.C - 1) * a.r_c + iclamp(j, 0, a.r_c - 1)) * jb.in + iclamp(k, 0, jb.in - 8);
}
// B_c^T[c][o][j .. j+7] (j a multiple of 8 below r_c)
SALT_HD int64_t btc_off(const ApplyLaunch& a, const Job& jb, int c, int o, int j) {
  return ((int64_t)iclamp(c, 0, a.C - 1) * jb.out + iclamp(o, 0, jb.out - 1)) * a.r_c + iclamp(j, 0, a.r_c - 8);
}
// y[t][o .. o+7]
SALT_HD int64_t y_off(const ApplyLaunch& a, const Job& jb, int t, int o) {
  return (int64_t)iclamp(t, 0, a.T - 1) * jb.out + iclamp(o, 0, jb.out - 8);
}
// Byte offset in the slot pool of A_u^T[rho][k .. k+7] of slot u holding rank r:
// the slot's blob holds, table after table, At_u [r][in] then B_u [r][out].
SALT_HD int64_t atu_byte(const ApplyLaunch& a, const Job& jb, int u, int r, int rho, int k) {
  const int rr = iclamp(r, 1, a.r_u);
  const int64_t e = (int64_t)rr * jb.prefix + (int64_t)iclamp(rho, 0, rr - 1) * jb.in + iclamp(k, 0, jb.in - 8);
  return (int64_t)iclamp(u, 0, a.n_slots - 1) * a.slot_stride + e * a.esize;
}
// Byte offset in the slot pool of B_u[rho][o .. o+7] of slot u holding rank r.
SALT_HD int64_t bu_byte(const ApplyLaunch& a, const Job& jb, int u, int r, int rho, int o) {
  const int rr = iclamp(r, 1, a.r_u);
  const int64_t e = (int64_t)rr * jb.prefix + (int64_t)rr * jb.in + (int64_t)iclamp(rho, 0, rr - 1) * jb.out +
                    iclamp(o, 0, jb.out - 8);
  return (int64_t)iclamp(u, 0, a.n_slots - 1) * a.slot_stride + e * a.esize;
}
// Partial sum of K range s, sorted position p, column col (floats), inside the
// job's own region [poff, poff + S * T * R).
SALT_HD int64_t part_off(const ApplyLaunch& a, const Job& jb, int s, int p, int col) {
  return jb.poff + ((int64_t)iclamp(s, 0, jb.S - 1) * a.T + iclamp(p, 0, a.T - 1)) * a.R + iclamp(col, 0, a.R - 1);
}

// ---- loop ranges ---------------------------------------------------------------
// K range s of a job: [k_lo, k_hi).  Its kStepK-wide steps are shared by the
// kw waves along K, wave kq taking steps kq, kq + kw, ...
SALT_HD int k_lo(const Job& jb, int s) { return imin(jb.in, s * jb.Kc); }
SALT_HD int k_hi(const Job& jb, int s) { return imin(jb.in, (s + 1) * jb.Kc); }
SALT_HD int k_steps(const Job& jb, int s) { return cdiv(k_hi(jb, s) - k_lo(jb, s), kStepK); }

// Elements between the two 8-element vectors a lane holds of a 64-wide shrink
// step or expand chunk: lane group g holds g 8 + 0..7 and kPiece + g 8 + 0..7,
// so that the four groups' vector h covers 32 contiguous elements.
constexpr int kPiece = 32;

// Output column of expand A-operand row i (lane & 15) in column block b4 of a
// 64-column chunk starting at col0: arranged so that MFMA output lane (token,
// g), which receives rows 4 g + e of tile b4, holds columns col0 + 8 g + kPiece h
// + 4 (b4 & 1) + e with h = b4 >> 1, i.e. the vectors col0 + 8 g + kPiece h + 0..7.
SALT_HD int expand_col(int col0, int i, int b4) {
  return col0 + kPiece * (b4 >> 1) + 8 * (i >> 2) + 4 * (b4 & 1) + (i & 3);
}

}  // namespace salt
