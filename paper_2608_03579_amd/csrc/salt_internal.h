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
  char* sink;         // [kSinkBytes] target of the y stores of lanes with nothing to write (never read)
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

// Everything one apply launch needs, passed by value.  The first 64 bytes hold
// what every block reads before its first data load (its role, its tile and
// where the tile's tokens come from), so that they arrive in one scalar
// cache line.
struct alignas(64) ApplyArgs {
  int32_t n_tiles, S;       // tiles; shrink blocks per tile (K ranges x residual rank chunks)
  int32_t sk;               // K ranges per tile (S = sk x rank chunks)
  int32_t n_col;            // expand blocks per tile
  int32_t fused_plan;       // 1: this launch also builds the plan (T <= kPlanFusedT)
  int32_t writer;           // block that writes the plan (fused_plan), else -1
  int32_t T;
  const int4* tiles;        // tile records of a built plan
  const int4* maps;         // staged maps (c, u, r, gamma bits) by token (fused_plan)
  int32_t Kc;               // K range length of one shrink block
  int32_t cpb;              // kNC-column chunks per expand block
  int32_t atomic_sum;       // 1: split partials are added into v with device atomics
  int32_t two_pass;         // 1: a shrink launch stores split partials, an expand launch sums them
  int32_t in_dim, out_dim, r_c, r_u_max, R;
  const void* x;            // [T][in]
  void* y;                  // [T][out]
  const void* cent_at;      // [C][r_c][in]  centroid A, transposed
  const void* cent_bt;      // [C][out][r_c] centroid B, transposed (internal layout)
  const char* pool;         // residual slot pool
  size_t slot_stride;       // bytes between slots
  int64_t tab_prefix;       // sum of (in + out) over earlier tables (elements per rank)
  float* partials;          // [S][T][R] (ordered sums only)
  float* v;                 // [T][R] v of this apply, centroid part not yet scaled by gamma
  float* v_clear;           // v buffer of the next apply: rows [0, clear_rows) cleared here (atomic sums only)
  int32_t clear_rows;       // >= T
  uint32_t target;          // arrival count of every tile once this apply's shrink is done
  uint32_t epoch;           // 1, 2, ... per apply of the plan since its build
  uint32_t* arrive;
  uint32_t* ready;
  int32_t* meta;
  char* sink;               // kSinkBytes that absorb the y stores of lanes with nothing to write
  PlanBuffers pb;           // the plan's buffers (fused_plan only)
};
static_assert(offsetof(ApplyArgs, maps) + sizeof(void*) <= 64, "the fields a block reads first share one 64-byte line");

// One centroid fused into a base weight: W <- rne(W + gamma * A_c B_c).
struct FuseArgs {
  const void* at;           // [r_c][in] A_c^T of the centroid
  const void* bt;           // [out][r_c] B_c^T of the centroid (internal layout)
  void* w;                  // [in][ldw] base weight, row-major
  int64_t ldw;              // elements between rows of w (multiple of 8, >= out)
  int32_t in_dim, out_dim, r_c;
  float gamma;
};

// Gram products of two low-rank updates dW_k = A_k B_k per table (factor form):
// g holds, per table and factor side (At: over in, B: over out), the Grams
// X1 X2^T [nb1*16][nb2*16], X1 X1^T [nb1*16][nb1*16], X2 X2^T [nb2*16][nb2*16]
// (ranks padded to 16); out[3 t + 0..2] = Tr(dW1^T dW2), ||dW1||^2, ||dW2||^2.
struct GramTable {
  const void* at1;          // [r1][in]
  const void* b1;           // [r1][out]
  const void* at2;          // [r2][in]
  const void* b2;           // [r2][out]
  int32_t in_dim, out_dim;
};
struct GramArgs {
  const GramTable* tabs;    // [n_tables], device
  int32_t n_tables, r1, r2;
  float* g;                 // zeroed by the caller
  size_t g_table, g_side;   // floats per table, per factor side
  int32_t g_12, g_11, g_22; // floats of each Gram
  double* out;              // [n_tables][3], device
};

hipError_t kernels_init(int device);
hipError_t launch_plan(const PlanArgs& a, hipStream_t s);
// e0 / e1: if set, HIP events that record the apply kernel's own start and end.
hipError_t launch_apply(const ApplyArgs& a, int bf16, int M, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
// e0 / e1 as for launch_apply.
hipError_t launch_fuse(const FuseArgs& f, int bf16, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
// k_gram then k_gram_finish on s; max_in / max_out: largest in / out over the tables.
hipError_t launch_gram(const GramArgs& a, int max_in, int max_out, int bf16, hipStream_t s);
// Blocks of the two-launch apply's shrink and expand kernels one compute unit
// holds at once (bf16, r_u_max <= 2).
hipError_t two_pass_occupancy(int r_c, int r_u_max, int R, int* shrink_per_cu, int* expand_per_cu);

// Columns of y per expand chunk.
constexpr int kNC = 128;
// Sink for the y stores of lanes past the tile or past out_dim: one 32-byte
// slot per thread of a block.  An expand issues the same stores on every path,
// so its waits on outstanding memory operations count them exactly.
constexpr int kSinkBytes = 256 * 32;
// Tokens per tile of the two-launch apply (large batches).
constexpr int kTwoPassM = 64;
// 16-rank blocks of the centroid a lane holds for rank r_c: r_c <= 16 * nbm.
constexpr int centroid_blocks(int r_c) { return r_c <= 32 ? 2 : (r_c <= 64 ? 4 : 8); }
// Row stride (bf16 elements) of the expand's bf16 copies of v's centroid part:
// 32-rank MFMA steps plus 8 elements of padding.
constexpr int expand_vs(int nbm) { return (nbm + 1) / 2 * 32 + 8; }
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
constexpr int kMaxSplit = 64;
// Ready words: kMaxSplit per tile, 64 bytes apart, so that the S blocks of a
// tile that raise them concurrently never write the same 64-byte sector.
constexpr int kReadyStride = 16;
constexpr int kReadyPerTile = kMaxSplit * kReadyStride;

// 32-wide K steps whose loads a shrink wave issues together: about 96 VGPRs of
// operands (per step: x and ru A_u rows for each of its mbw M-blocks, nbm A_c
// rows; vec_regs registers each).
constexpr int shrink_batch(int vec_regs, int mbw, int nbm, int ru) {
  const int u = 96 / (vec_regs * (mbw + nbm + mbw * ru));
  return u < 1 ? 1 : (u > 4 ? 4 : u);
}
// Largest supported ranks.  Residual ranks above 16 (long-tail adapters that
// concatenate a centroid and a residual, e.g. r = 17 / 33 / 65) run in chunks
// of kRankChunk ranks, one shrink block per (K range, chunk).
constexpr int kMaxRc = 128;
constexpr int kMaxRu = 72;
constexpr int kRankChunk = 16;

}  // namespace salt
