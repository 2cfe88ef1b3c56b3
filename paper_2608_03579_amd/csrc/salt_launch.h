// Host-side choices of an apply: tokens per tile, the tiles of a batch, the K
// split of the shrink and the column blocks of the expand.  Header-only and free
// of HIP calls, so that the runtime and the host-side address checks use the
// same code.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <vector>

#include "salt_layout.h"

namespace salt {

// Tokens per tile, from the mean size of the batch's centroid groups: short
// groups (decode batches) take 16-token tiles, groups of up to ~100 tokens 32,
// up to ~400 tokens 64, longer ones (prefill) 128 when there is a centroid
// operand, which each block stages once per tile: the larger the tile, the
// fewer times it is read.  fp32 contexts always use 16.
inline int choose_tile_tokens(int esize, int T, int n_groups, bool centroids) {
  if (esize == 4 || n_groups <= 0) return 16;
  const double mean = (double)T / n_groups;
  if (mean <= 24.0) return 16;
  if (mean <= 96.0) return 32;
  if (mean <= 384.0 || !centroids) return 64;
  return 128;
}

// Tiles of a batch from the token counts of its centroid groups, per_c[c + 1]
// for c = -1 .. C - 1 (the sorted order puts c = -1 first).  A group of n tokens
// becomes k = ceil(n / M) tiles: for tiles of up to 64 tokens of near-equal
// size, the first n mod k of them one token longer; for larger tiles
// k - 1 full tiles and the remainder (the expand of 128-token tiles splits
// its work by column chunks, not by tiles, so their sizes need not match).
// Tiles are contiguous in sorted order and cover [0, T).
inline void cut_tiles(const std::vector<int>& per_c, int M, std::vector<int4>& tiles) {
  tiles.clear();
  int start = 0;
  for (size_t g = 0; g < per_c.size(); ++g) {
    const int n = per_c[g];
    if (n <= 0) continue;
    const int k = cdiv(n, M), base = n / k, extra = n % k;
    int p = start;
    for (int i = 0; i < k; ++i) {
      const int len = M > 64 ? imin(M, n - i * M) : base + (i < extra ? 1 : 0);
      int4 t;
      t.x = p;
      t.y = len;
      t.z = (int)g - 1;
      t.w = 0;
      tiles.push_back(t);
      p += len;
    }
    start += n;
  }
}

// Split-K partial floats a plan of up to T tokens holds (rows of R floats): two
// K ranges per token row for a full launch of kMaxJobs tables, or one if that
// would pass 256 MiB; small batches get up to 16 Mi floats (64 MiB, at most 64
// ranges per table), so that a decode launch can split K finely enough to fill
// the device.
inline size_t plan_partial_cap(size_t T, size_t R) {
  const size_t two = 2 * (size_t)kMaxJobs * T * R;
  const size_t small = std::min((size_t)16 << 20, 64 * (size_t)kMaxJobs * T * R);
  if (two < small) return small;
  return two * 4 <= ((size_t)256 << 20) ? two : (size_t)kMaxJobs * T * R;
}

// Largest number of tiles a batch of T tokens over C centroids can cut into.
inline int max_tiles(int T, int C) { return cdiv(T, 16) + C + 1; }

// K ranges, expand block-chunks and work offsets of launch `a`, whose jobs (in,
// out, prefix, pointers) and batch fields (T, M, n_tiles, MS, n_stiles, C, r_c, r_u, nq, R,
// esize, partial_cap) are set.  n_groups_c: centroids the batch references;
// sum_rank: residual ranks summed over the slots it references (both for the
// byte counts that bound the partial traffic).  Returns false if the partials
// of a one-range shrink do not fit.
// shrink_round: shrink blocks one round of the device holds at once (0: unknown).
inline bool configure_launch(ApplyLaunch& a, int n_cu, int n_groups_c, int64_t sum_rank, int shrink_round = 0) {
  const int KW = waves_of(a.MS) / (a.MS / 16), CW = waves_of(a.M) / (a.M / 16);
  const int target = 8 * std::max(1, n_cu);        // blocks per launch: a few rounds of the whole device
  const double es = (double)a.esize;
  const double adapters = (double)n_groups_c * a.r_c + (double)sum_rank;
  int64_t sum_in = 0;
  for (int j = 0; j < a.n_jobs; ++j) sum_in += a.jobs[j].in;
  // shrink: one K-range length for the whole launch, so that blocks of every
  // table carry about the same work, sized for ~target blocks; each table's
  // split is capped so that its partials (written, then read) stay within a
  // tenth of its bytes
  const int gran = kStepK * KW;
  const double pairs = (double)shrink_tiles(a) * a.nq;
  const int kc_target = std::max(gran, cdiv((int)std::ceil((double)sum_in * pairs / target), gran) * gran);
  const double part_row = 8.0 * a.T * a.R;        // bytes of one K range's partials, written and read
  std::vector<int> S(a.n_jobs), s_cap(a.n_jobs);
  for (int j = 0; j < a.n_jobs; ++j) {
    const Job& jb = a.jobs[j];
    const double bytes = es * ((double)a.T * (jb.in + 2.0 * jb.out) + adapters * (jb.in + jb.out));
    const int s_traffic = std::max(1, (int)(0.1 * bytes / part_row));
    s_cap[j] = std::max(1, std::min(s_traffic, cdiv(jb.in, gran)));
    S[j] = std::max(1, std::min(cdiv(jb.in, kc_target), s_cap[j]));
  }
  // Shrink tiles of 64 tokens (long groups, many tokens).  If one K range as
  // long as the smallest table's K already gives a round of the device's
  // blocks, K is split no finer: tables with more K take ranges of about that
  // length (blocks of equal length), and a finer split would only add partials
  // for the expand to sum.  Otherwise each block is long, so a round of the
  // device that is only partly filled costs real time: the K-range length is
  // then the one that minimises (rounds of blocks) x (the longest range); ties
  // go to the longer length (fewer partials).
  bool fills = false;
  if (a.MS >= 64 && shrink_round > 0) {
    int min_in = a.jobs[0].in;
    for (int j = 1; j < a.n_jobs; ++j) min_in = std::min(min_in, a.jobs[j].in);
    const int kc = cdiv(min_in, gran) * gran;
    int64_t blocks = 0;
    std::vector<int> Sm(a.n_jobs);
    for (int j = 0; j < a.n_jobs; ++j) {
      Sm[j] = std::max(1, std::min(cdiv(a.jobs[j].in, kc), s_cap[j]));
      blocks += (int64_t)shrink_tiles(a) * a.nq * Sm[j];
    }
    if (blocks >= shrink_round) {
      S = Sm;
      fills = true;
    }
  }
  if (a.MS >= 64 && shrink_round > 0 && !fills) {
    int max_in = 0;
    for (int j = 0; j < a.n_jobs; ++j) max_in = std::max(max_in, a.jobs[j].in);
    double best = 0.0;
    for (int kc = gran; kc < max_in + gran; kc += gran) {
      int64_t blocks = 0;
      int longest = 0;
      for (int j = 0; j < a.n_jobs; ++j) {
        const int sj = std::max(1, std::min(cdiv(a.jobs[j].in, kc), s_cap[j]));
        blocks += (int64_t)shrink_tiles(a) * a.nq * sj;
        longest = std::max(longest, cdiv(cdiv(a.jobs[j].in, sj), gran) * gran);
      }
      const double est = (double)((blocks + shrink_round - 1) / shrink_round) * longest;
      if (best == 0.0 || est <= best) {
        best = est;
        for (int j = 0; j < a.n_jobs; ++j) S[j] = std::max(1, std::min(cdiv(a.jobs[j].in, kc), s_cap[j]));
      }
    }
  }
  // partials must fit, and each table's region stays below kMaxBufferBytes:
  // shrink the largest split until they do
  auto total = [&]() {
    int64_t t = 0;
    for (int j = 0; j < a.n_jobs; ++j) t += (int64_t)S[j] * a.T * a.R;
    return t;
  };
  auto too_big = [&]() {
    for (int j = 0; j < a.n_jobs; ++j)
      if ((int64_t)S[j] * a.T * a.R * 4 >= kMaxBufferBytes) return true;
    return false;
  };
  while (total() > a.partial_cap || too_big()) {
    int jm = 0;
    for (int j = 1; j < a.n_jobs; ++j)
      if (S[j] > S[jm]) jm = j;
    if (S[jm] == 1) return false;
    S[jm] = (S[jm] + 1) / 2;
  }
  int64_t poff = 0;
  int sb = 0, eb = 0;
  for (int j = 0; j < a.n_jobs; ++j) {
    Job& jb = a.jobs[j];
    jb.Kc = cdiv(cdiv(jb.in, S[j]), gran) * gran;
    jb.S = cdiv(jb.in, jb.Kc);
    jb.poff = poff;
    poff += (int64_t)jb.S * a.T * a.R;
    // expand: work items of one block-chunk (kChunkCols per wave along the
    // columns); the launch splits them evenly over one round of blocks
    jb.cpb = kChunkCols * CW;
    jb.n_col = cdiv(jb.out, jb.cpb);
    jb.shrink_base = sb;
    jb.expand_base = eb;
    sb += shrink_tiles(a) * jb.S * a.nq;
    eb += a.n_tiles * jb.n_col;
  }
  a.shrink_blocks = sb;
  a.expand_items = eb;
  return true;
}

}  // namespace salt
