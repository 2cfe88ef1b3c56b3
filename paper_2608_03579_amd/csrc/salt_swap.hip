// Residual swaps as one gather kernel (Sec. 3.1: only a user's small residual
// moves into HBM when the user becomes active; Sec. 4.4 contrasts that swap
// with the full adapter's).
//
// A step's swaps are many small blobs (one user's residual of every table, e.g.
// 327,680 B at rank 2 for a Llama-3.1-8B layer).  Copied one DMA transfer per
// blob, each pays the copy engine's fixed set-up cost, which dominates at this
// size.  When the blobs sit in page-locked memory that the device maps
// (salt_host_alloc), one kernel reads all of them over PCIe instead: block
// (c, i) copies chunk c of blob i, 16-byte vectors, kSwapUnroll loads per
// thread in flight before any store, so one launch keeps enough reads
// outstanding to run at the link's rate.
#include "salt_internal.h"

namespace salt {
namespace {

constexpr int kSwapThreads = 256;
constexpr int kSwapUnroll = 4;
constexpr int64_t kSwapChunkVecs = (int64_t)kSwapThreads * kSwapUnroll;   // 16 KiB per block

__global__ void __launch_bounds__(kSwapThreads) k_swap_gather(const SwapArgs a) {
  const int i = blockIdx.y;
  if (i >= a.n) return;
  const int64_t nvec = a.vecs[i];
  const int64_t v0 = (int64_t)blockIdx.x * kSwapChunkVecs + threadIdx.x;
  if (v0 >= nvec) return;
  const uint4* src = a.src[i];
  uint4* dst = a.dst[i];
  uint4 v[kSwapUnroll];
#pragma unroll
  for (int u = 0; u < kSwapUnroll; ++u) {
    const int64_t k = v0 + (int64_t)u * kSwapThreads;
    if (k < nvec) v[u] = src[k];
  }
#pragma unroll
  for (int u = 0; u < kSwapUnroll; ++u) {
    const int64_t k = v0 + (int64_t)u * kSwapThreads;
    if (k < nvec) dst[k] = v[u];
  }
}

}  // namespace

hipError_t launch_swap(const SwapArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  if (a.n > kSwapMax) return hipErrorInvalidValue;
  int64_t most = 0;
  for (int i = 0; i < a.n; ++i) {
    if (a.vecs[i] < 0 || !a.src[i] || !a.dst[i]) return hipErrorInvalidValue;
    most = a.vecs[i] > most ? a.vecs[i] : most;
  }
  if (most == 0) return hipSuccess;
  const int64_t chunks = (most + kSwapChunkVecs - 1) / kSwapChunkVecs;
  if (chunks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_swap_gather, dim3((unsigned)chunks, (unsigned)a.n), dim3(kSwapThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace salt
