// HBM streaming ceiling of the device: read-only, copy and in-place read-modify-write
// kernels over 1 GiB buffers, 16 bytes per lane, several grid sizes.  These bound what
// any kernel of the same access mix can reach, next to the published 8 TB/s peak.
// Every index stays below n16 (the buffer size in 16-byte units).
#include <hip/hip_runtime.h>
#include <cstdio>
#include <vector>
#define CK(x) do { hipError_t e = (x); if (e) { printf("err %s line %d\n", hipGetErrorString(e), __LINE__); return 1; } } while (0)

template <int U>
__global__ void __launch_bounds__(256) k_read(const uint4* __restrict__ a, size_t n16, uint4* __restrict__ out) {
  uint32_t acc = 0;
  const size_t stride = (size_t)gridDim.x * 256 * U;
  for (size_t base = (size_t)blockIdx.x * 256 * U + threadIdx.x; base < n16; base += stride) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) { size_t i = base + (size_t)u * 256; v[u] = i < n16 ? a[i] : make_uint4(0,0,0,0); }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (acc == 0x12345678u) out[0] = make_uint4(acc, 0, 0, 0);
}
template <int U>
__global__ void __launch_bounds__(256) k_copy(const uint4* __restrict__ a, uint4* __restrict__ b, size_t n16) {
  const size_t stride = (size_t)gridDim.x * 256 * U;
  for (size_t base = (size_t)blockIdx.x * 256 * U + threadIdx.x; base < n16; base += stride) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) { size_t i = base + (size_t)u * 256; if (i < n16) v[u] = a[i]; }
#pragma unroll
    for (int u = 0; u < U; ++u) { size_t i = base + (size_t)u * 256; if (i < n16) b[i] = v[u]; }
  }
}
template <int U>
__global__ void __launch_bounds__(256) k_rmw(uint4* __restrict__ a, size_t n16) {
  const size_t stride = (size_t)gridDim.x * 256 * U;
  for (size_t base = (size_t)blockIdx.x * 256 * U + threadIdx.x; base < n16; base += stride) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) { size_t i = base + (size_t)u * 256; if (i < n16) v[u] = a[i]; }
#pragma unroll
    for (int u = 0; u < U; ++u) { size_t i = base + (size_t)u * 256; if (i < n16) { v[u].x += 1; a[i] = v[u]; } }
  }
}

int main() {
  const size_t bytes = (size_t)1 << 30;   // 1 GiB per buffer
  const size_t n16 = bytes / 16;
  uint4 *a, *b, *o;
  CK(hipMalloc(&a, bytes)); CK(hipMalloc(&b, bytes)); CK(hipMalloc(&o, 64));
  CK(hipMemset(a, 1, bytes)); CK(hipMemset(b, 2, bytes));
  hipEvent_t e0, e1; CK(hipEventCreate(&e0)); CK(hipEventCreate(&e1));
  auto timeit = [&](const char* name, auto launch, double moved) -> int {
    for (int i = 0; i < 2; ++i) launch();
    CK(hipDeviceSynchronize());
    CK(hipEventRecord(e0, 0));
    const int reps = 10;
    for (int i = 0; i < reps; ++i) launch();
    CK(hipEventRecord(e1, 0)); CK(hipEventSynchronize(e1));
    float ms; CK(hipEventElapsedTime(&ms, e0, e1));
    printf("%-34s %8.1f us  %7.0f GB/s\n", name, ms * 1e3 / reps, moved / (ms * 1e-3 / reps) / 1e9);
    fflush(stdout);
    return 0;
  };
  for (int grid : {1024, 2048, 4096, 8192}) {
    char nm[64];
    snprintf(nm, 64, "read   U=4 grid=%d", grid);
    timeit(nm, [&] { k_read<4><<<grid, 256>>>(a, n16, o); }, (double)bytes);
    snprintf(nm, 64, "read   U=8 grid=%d", grid);
    timeit(nm, [&] { k_read<8><<<grid, 256>>>(a, n16, o); }, (double)bytes);
    snprintf(nm, 64, "copy   U=4 grid=%d", grid);
    timeit(nm, [&] { k_copy<4><<<grid, 256>>>(a, b, n16); }, 2.0 * bytes);
    snprintf(nm, 64, "rmw    U=4 grid=%d", grid);
    timeit(nm, [&] { k_rmw<4><<<grid, 256>>>(b, n16); }, 2.0 * bytes);
  }
  CK(hipGetLastError());
  printf("done\n");
  return 0;
}
