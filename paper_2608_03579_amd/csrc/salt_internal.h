// Internal declarations shared by the libsalt host runtime and its HIP kernels.
// Not part of the public ABI (include/salt.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace salt {

// Device buffers of one plan.  Sorted-position arrays are indexed by the
// position of a token in the canonical (centroid, slot, token) order.
struct PlanBuffers {
  int4* maps;        // [max_T] staged maps: (c, u, r, gamma bits) per token
  int32_t* perm;     // [max_T] token index at each sorted position
  int4* srt;         // [max_T] (token, u, r, gamma bits) at each sorted position
  int32_t* srt_c;    // [max_T] centroid id at each sorted position
  int32_t* seg_off;  // [max_T + 1]
  int32_t* seg_c;    // [max_T]
  int32_t* seg_u;    // [max_T]
  int32_t* grp_off;  // [max_T + 1] segment index where each centroid group starts
  int32_t* grp_tok;  // [max_T + 1] sorted position where each centroid group starts
  int32_t* grp_c;    // [max_T] centroid id of each group
  int32_t* meta;     // [16]: [0] n_seg, [1] n_grp, [2] T
  uint32_t* counter; // [64] arrival counters, zero between launches
  float* partials;   // [partial_cap] fp32 split-K partial sums of the shrink
  size_t partial_cap;
};

// Everything one salt_apply launch needs, passed by value.
struct ApplyArgs {
  const void* x;            // [T][in]
  void* y;                  // [T][out]
  const void* cent_at;      // [C][r_c][in] of this table
  const void* cent_b;       // [C][r_c][out] of this table
  const char* pool;         // slot pool base
  size_t slot_stride;       // bytes between slots
  int64_t tab_prefix;       // sum of (in + out) over earlier tables, in elements per rank
  const int4* srt;
  const int32_t* grp_tok;
  const int32_t* grp_c;
  const int32_t* meta;
  float* partials;          // [S][T][R]
  int32_t T, in_dim, out_dim, r_c, r_u_max, R;
  int32_t S, Kc, NC;        // K-splits, K per split, columns per expand block
};

hipError_t launch_plan(const PlanBuffers& b, int32_t T, int32_t n_centroids, hipStream_t s);
hipError_t launch_apply(const ApplyArgs& a, int dtype_bf16, int32_t tiles_ub, hipStream_t s);
hipError_t kernels_init(int device);

// Tile size (tokens of one centroid group) of the VALU apply kernels.
constexpr int kTileM = 16;

}  // namespace salt
