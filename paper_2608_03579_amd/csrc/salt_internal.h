// Internal declarations shared by the libsalt host runtime and its HIP kernels.
// Not part of the public ABI (include/salt.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace salt {

// Slots of the per-plan meta word array.
enum Meta { kMetaNSeg = 0, kMetaNGrp = 1, kMetaT = 2, kMetaNTiles = 3, kMetaErr = 4, kMetaWords = 16 };

// Device buffers of one plan.  "Sorted position" is the position of a token in
// the canonical (centroid, slot, token) order.
struct PlanBuffers {
  int4* maps;         // [max_T] staged maps: (c, u, r, gamma bits) per token
  int32_t* perm;      // [max_T] token index at each sorted position
  int4* srt;          // [max_T] (token, u, r, gamma bits) at each sorted position
  int32_t* srt_c;     // [max_T] centroid id at each sorted position
  int32_t* seg_off;   // [max_T + 1]
  int32_t* seg_c;     // [max_T]
  int32_t* seg_u;     // [max_T]
  int32_t* grp_off;   // [max_T + 1] segment index where each centroid group starts
  int32_t* grp_tok;   // [max_T + 1] sorted position where each centroid group starts
  int32_t* grp_c;     // [max_T] centroid id of each group
  int4* tiles;        // [tile_cap]: per tile (i0, n, c, 0) then M token records
  uint32_t* arrive;   // [max tiles * kCounterStride] shrink blocks done with each tile since the build
  uint32_t* ready;    // [max tiles * kReadyPerTile] epoch of the last apply whose v of the tile is
                      // complete: word 0 (ordered sums), or word s * kReadyStride per K range s
                      // (atomic sums)
  float* v;           // [2][max_T][R] v = x [A_c | A_u] (R padded to 4); two buffers
  size_t v_stride;    // floats between the two v buffers
  int32_t* meta;      // [kMetaWords]
  uint32_t* counter;  // [64] arrival counter of the multi-block plan build
  float* partials;    // [partial_cap] split-K partial sums of the shrink
  size_t partial_cap; // floats
  size_t tile_cap;    // int4 entries
  int32_t tiles_max;  // entries of arrive
};

struct PlanArgs {
  PlanBuffers b;
  int32_t T;
  int32_t M;            // tokens per tile (16, 32 or 64)
  int32_t reset_ready;  // 1: zero every ready word (the plan's epochs restart)
};

// Everything one apply launch needs, passed by value.
struct ApplyArgs {
  const void* x;            // [T][in]
  void* y;                  // [T][out]
  const void* cent_at;      // [C][r_c][in]  centroid A, transposed
  const void* cent_bt;      // [C][out][r_c] centroid B, transposed (internal layout)
  const char* pool;         // residual slot pool
  size_t slot_stride;       // bytes between slots
  int64_t tab_prefix;       // sum of (in + out) over earlier tables (elements per rank)
  const int4* tiles;
  float* partials;          // [S][T][R] (ordered sums only)
  float* v;                 // [T][R] v of this apply, centroid part not yet scaled by gamma
  float* v_clear;           // v buffer of the next apply: rows [0, clear_rows) cleared here (atomic sums only)
  int32_t clear_rows;       // >= T
  uint32_t* arrive;
  uint32_t* ready;
  int32_t* meta;
  uint32_t target;          // arrival count of every tile once this apply's shrink is done
  uint32_t epoch;           // 1, 2, ... per apply of the plan since its build
  int32_t T, in_dim, out_dim, r_c, r_u_max, R;
  int32_t n_tiles, S, Kc;
  int32_t n_col;            // expand blocks per tile
  int32_t cpb;              // kNC-column chunks per expand block
  int32_t atomic_sum;       // 1: split partials are added into v with device atomics
  int32_t fused_plan;       // 1: this launch also builds the plan (T <= kPlanFusedT)
  PlanBuffers pb;           // the plan's buffers (fused_plan only)
};

hipError_t kernels_init(int device);
hipError_t launch_plan(const PlanArgs& a, hipStream_t s);
// e0 / e1: if set, HIP events that record the apply kernel's own start and end.
hipError_t launch_apply(const ApplyArgs& a, int bf16, int M, hipStream_t s, hipEvent_t e0, hipEvent_t e1);

// Columns of y per expand chunk.
constexpr int kNC = 128;
// Batches a single plan block sorts in LDS, and batches an apply launch plans
// for itself.
constexpr int kPlanSmallT = 1024;
constexpr int kPlanFusedT = 256;

// Row stride of the partials and of v: r_c + r_u_max rounded up to whole float4s.
constexpr int padded_rank(int r_c, int r_u_max) {
  const int r = r_c + r_u_max;
  return r < 4 ? 4 : (r + 3) / 4 * 4;
}
// Per-tile arrival counters sit 256 bytes apart (no two share a cache line).
constexpr int kCounterStride = 64;
// Largest K split of one apply.
constexpr int kMaxSplit = 32;
// Ready words: kMaxSplit per tile, 64 bytes apart, so that the S blocks of a
// tile that raise them concurrently never write the same 64-byte sector.
constexpr int kReadyStride = 16;
constexpr int kReadyPerTile = kMaxSplit * kReadyStride;

// 32-wide K steps whose loads a shrink wave issues together: about 96 VGPRs of
// operands (x, nbm A_c rows, ru A_u rows per step, vec_regs registers each).
constexpr int shrink_batch(int vec_regs, int nbm, int ru) {
  const int u = 96 / (vec_regs * (1 + nbm + ru));
  return u < 1 ? 1 : (u > 4 ? 4 : u);
}
// Largest supported ranks.
constexpr int kMaxRc = 128;
constexpr int kMaxRu = 16;

}  // namespace salt
