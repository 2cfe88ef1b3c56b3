// Host walk of the apply launch decomposition (salt_launch.h / salt_layout.h
// built without HIP).  For seeded random batches and table sets it checks:
//  - cut_tiles covers the sorted order [0, T) with contiguous tiles of at most
//    M tokens, each inside one centroid group;
//  - configure_launch: the shrink items of a launch enumerate every (table,
//    tile, K range, rank chunk) exactly once; the expand's item ranges, split
//    over any number of blocks and walked segment by segment as the kernel
//    does, cover every (table, tile, block-chunk) exactly once; the K ranges of
//    a table partition [0, in) and its block-chunks [0, out); the tables'
//    partial regions are disjoint and inside the buffer.
// Prints the first failure and exits 1, else prints "ok".
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <tuple>
#include <vector>

#include "salt_launch.h"

using namespace salt;

static int fail(const char* what, long a = 0, long b = 0, long c = 0) {
  std::printf("FAIL %s (%ld %ld %ld)\n", what, a, b, c);
  std::exit(1);
}

int main() {
  std::mt19937 rng(2608);
  const int in_choices[] = {64, 136, 264, 520, 1032, 3072, 4096, 8192, 14336};
  for (int trial = 0; trial < 400; ++trial) {
    const int C = std::uniform_int_distribution<int>(0, 16)(rng);
    const int T = std::uniform_int_distribution<int>(1, trial % 4 == 0 ? 8192 : 600)(rng);
    const int esize = trial % 7 == 0 ? 4 : 2;
    // per-centroid counts (c = -1 first) from a random assignment
    std::vector<int> per_c(C + 1, 0);
    for (int t = 0; t < T; ++t) {
      const int g = std::uniform_int_distribution<int>(C ? 0 : 0, C)(rng);
      per_c[(C && (rng() % 8)) ? g : 0]++;
    }
    int n_groups = 0;
    for (int g = 1; g <= C; ++g) n_groups += per_c[g] > 0;
    const int M = choose_tile_tokens(esize, T, std::max(1, n_groups + (per_c[0] > 0)), n_groups > 0);
    std::vector<int4> tiles;
    cut_tiles(per_c, M, tiles);
    if ((int)tiles.size() > max_tiles(T, C)) fail("more tiles than max_tiles", tiles.size(), max_tiles(T, C));
    int pos = 0, start = 0;
    size_t ti = 0;
    for (int g = 0; g <= C; ++g) {
      const int end = start + per_c[g];
      while (ti < tiles.size() && tiles[ti].x < end) {
        const int4& h = tiles[ti];
        if (h.x != pos || h.y < 1 || h.y > M || h.x + h.y > end || h.z != g - 1) fail("bad tile", trial, ti, h.x);
        pos += h.y;
        ++ti;
      }
      start = end;
    }
    if (pos != T || ti != tiles.size()) fail("tiles do not cover the batch", trial, pos, T);

    ApplyLaunch a{};
    a.n_jobs = std::uniform_int_distribution<int>(1, kMaxJobs)(rng);
    a.T = T;
    a.n_tiles = (int)tiles.size();
    a.tiles = tiles.data();
    a.MS = M > 64 ? 64 : M;
    std::vector<int4> stiles;
    if (a.MS != M) cut_tiles(per_c, a.MS, stiles);
    a.stiles = a.MS != M ? stiles.data() : tiles.data();
    a.n_stiles = a.MS != M ? (int)stiles.size() : a.n_tiles;
    a.M = M;
    a.C = C;
    a.r_c = C ? 8 << (rng() % 5) : 0;
    if (a.r_c > kMaxRc) a.r_c = kMaxRc;
    a.r_u = (int)(rng() % 3 == 0 ? rng() % (kMaxRu + 1) : rng() % 3);
    a.nq = std::max(1, cdiv(a.r_u, kRankChunk));
    a.R = padded_rank(a.r_c, a.r_u);
    a.esize = esize;
    a.partial_cap = (int64_t)T * a.R * (1 + (int)(rng() % 64));
    int64_t prefix = 0;
    for (int j = 0; j < a.n_jobs; ++j) {
      a.jobs[j].in = in_choices[rng() % 9];
      a.jobs[j].out = in_choices[rng() % 9];
      a.jobs[j].prefix = prefix;
      prefix += a.jobs[j].in + a.jobs[j].out;
    }
    if (!configure_launch(a, 256, n_groups, (int64_t)a.r_u * 50, (trial % 2) ? 64 + (int)(rng() % 3000) : 0)) {
      if (a.partial_cap >= (int64_t)a.n_jobs * T * a.R) fail("configure_launch refused a launch that fits", trial);
      continue;
    }
    std::set<std::tuple<int, int, int, int>> sh;
    for (int b = 0; b < a.shrink_blocks; ++b) {
      const int item = b;
      const int j = job_of_shrink(a, item);
      const ShrinkCoord sc = shrink_coord(a, a.jobs[j], item);
      if (sc.tau < 0 || sc.tau >= shrink_tiles(a) || sc.s < 0 || sc.s >= a.jobs[j].S) fail("shrink coord", trial, b);
      if (!sh.insert({j, sc.tau, sc.s, sc.q}).second) fail("shrink item twice", trial, b);
    }
    // expand: the item ranges of G blocks, walked segment by segment as the
    // kernel does, visit every (job, tile, block-chunk) exactly once
    std::set<std::tuple<int, int, int>> ex;
    const int G = 1 + (int)(rng() % 3000);
    for (int b = 0; b < G; ++b) {
      const int end = expand_begin(a, b + 1, G);
      for (int pos = expand_begin(a, b, G); pos < end;) {
        const ExpandSeg sg = expand_seg(a, pos, end);
        const Job& jb = a.jobs[sg.job];
        if (sg.j0 < 0 || sg.j1 > jb.n_col || sg.j0 >= sg.j1 || sg.tau < 0 || sg.tau >= a.n_tiles)
          fail("expand segment", trial, b, pos);
        for (int j = sg.j0; j < sg.j1; ++j)
          if (!ex.insert({sg.job, sg.tau, j}).second) fail("expand item twice", trial, b, j);
        pos += sg.j1 - sg.j0;
      }
    }
    int64_t want_sh = 0, want_ex = 0, poff = 0;
    for (int j = 0; j < a.n_jobs; ++j) {
      const Job& jb = a.jobs[j];
      want_sh += (int64_t)shrink_tiles(a) * jb.S * a.nq;
      want_ex += (int64_t)a.n_tiles * jb.n_col;
      if (jb.Kc % kStepK || jb.cpb % kChunkCols || jb.n_col * jb.cpb < jb.out || (jb.n_col - 1) * jb.cpb >= jb.out)
        fail("range granularity", trial, j);
      int k = 0;
      for (int s = 0; s < jb.S; ++s) {
        if (k_lo(jb, s) != k || k_hi(jb, s) <= k) fail("K ranges", trial, j, s);
        k = k_hi(jb, s);
      }
      if (k != jb.in) fail("K ranges do not cover in", trial, j, k);
      if (jb.poff != poff) fail("partial regions", trial, j);
      poff += (int64_t)jb.S * T * a.R;
    }
    if (poff > a.partial_cap) fail("partials overflow", trial, poff, a.partial_cap);
    if ((int64_t)sh.size() != want_sh || (int64_t)ex.size() != want_ex) fail("items missing", trial);
    // the shrink's tiles cover the batch like the expand's: contiguous, inside
    // one centroid group each, at most MS tokens
    {
      int pos2 = 0;
      for (int t = 0; t < a.n_stiles; ++t) {
        const TileHdr h = shrink_tile(a, t);
        if (h.i0 != pos2 || h.n < 1 || h.n > a.MS || h.n != a.stiles[t].y) fail("shrink tile", trial, t, h.i0);
        pos2 += h.n;
      }
      if (pos2 != T) fail("shrink tiles do not cover the batch", trial, pos2, T);
    }
  }
  std::printf("ok\n");
  return 0;
}
