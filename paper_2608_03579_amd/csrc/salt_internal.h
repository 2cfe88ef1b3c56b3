// Internal declarations shared by the libsalt host runtime and its HIP kernels.
// Not part of the public ABI (include/salt.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "salt_layout.h"

namespace salt {

// Slots of the per-plan meta word array.
enum Meta { kMetaNSeg = 0, kMetaNGrp = 1, kMetaT = 2, kMetaNTiles = 3, kMetaErr = 4, kMetaWords = 16 };

// Device buffers of one plan build.  "Place" is the position of a token in the
// canonical (centroid, slot, token) order.
struct PlanLaunch {
  const int4* maps;     // [T] staged maps: (c, u, r, gamma bits) by token
  const int4* tiles;    // [n_tiles] tile headers staged by the host: (i0, n, c, 0)
  uint64_t* keys;       // [T] chunk-sorted keys (batches of more than one chunk)
  uint64_t* keys_sorted;// [T] sorted keys (idem)
  int4* srt;            // [T] (token, slot, rank, gamma bits) at each place
  int32_t* perm;        // [T] token at each place
  int32_t* seg_off;     // [T + 1]
  int32_t* seg_c;       // [T]
  int32_t* seg_u;       // [T]
  int32_t* grp_off;     // [T + 1]
  int32_t* meta;        // [kMetaWords]
  int32_t T;
  int32_t n_tiles;      // tiles [0, n_list0) and [n_list0, n_tiles): two lists, each covering [0, T)
  int32_t n_list0;      // (== n_tiles: one list)
};

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

// Residual blobs one swap launch gathers from mapped page-locked host memory:
// blob i is vecs[i] 16-byte vectors from src[i] (a device-visible host address)
// into dst[i] (its slot in the pool).
constexpr int kSwapMax = 64;
struct SwapArgs {
  const uint4* src[kSwapMax];
  uint4* dst[kSwapMax];
  int64_t vecs[kSwapMax];
  int32_t n;
};

// 16-rank blocks of the centroid a shrink lane holds for rank r_c (r_c <= 16 * result).
constexpr int centroid_blocks(int r_c) { return r_c == 0 ? 0 : (r_c <= 32 ? 2 : (r_c <= 64 ? 4 : 8)); }

hipError_t kernels_init(int device);
// Floats of the static device scratch that salt_apply_batch_noalloc's launches
// keep their split-K partials in (64 MiB per device).
constexpr size_t kScratchFloats = (size_t)16 << 20;
constexpr int kMaxDevices = 64;
// This device's copy of the scratch (resolved by kernels_init), or null.
float* static_scratch(int device);
hipError_t launch_plan(const PlanLaunch& a, hipStream_t s);
// The apply: k_shrink then k_expand on s.  ev (may be null): four HIP events
// that record the start and end of the shrink kernel (ev[0], ev[1]) and of the
// expand kernel (ev[2], ev[3]); null entries are skipped.
hipError_t launch_apply(const ApplyLaunch& a, hipStream_t s, hipEvent_t* ev);
// Shrink blocks of launch `a` (esize, M, MS, r_c, r_u set) that one round of the
// device holds at once: the kernel's occupancy per compute unit x n_cu.
int shrink_round_blocks(const ApplyLaunch& a);
// e0 / e1: if set, HIP events that record the fuse kernel's own start and end.
hipError_t launch_fuse(const FuseArgs& f, int bf16, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
// k_gram then k_gram_finish on s; max_in / max_out: largest in / out over the tables.
// k_swap_gather on s: every blob of a (n <= kSwapMax) in one launch.
hipError_t launch_swap(const SwapArgs& a, hipStream_t s);
hipError_t launch_gram(const GramArgs& a, int max_in, int max_out, int bf16, hipStream_t s);

}  // namespace salt
