// A host build of libsalt for tests: this header stands in for the HIP runtime
// and the device builtins, so that the library's own sources (runtime and
// kernels, unchanged) compile for the CPU and run there, one block at a time.
//
// The threads of a block are cooperative fibers on one OS thread.  A block
// barrier (__syncthreads) waits for every live thread of the block; a wave
// operation (lane shuffle, MFMA) waits for the 64 threads of the wave, which
// deposit their operands and then read what they need.  MFMA follows the lane
// layout of gfx950's v_mfma_f32_16x16x32_bf16 and v_mfma_f32_16x16x4_f32: lane l
// brings row (l & 15) of A and column (l & 15) of B with k-slot group l >> 4
// (8 k per lane for bf16, one for fp32) and receives column (l & 15), rows
// 4 (l >> 4) .. + 3 of D.  Device memory is host memory of the exact size
// requested, so AddressSanitizer reports any access outside an allocation, as
// it does for the dynamic LDS of each launch.  A block whose threads wait at
// different barriers is reported as a deadlock.
//
// Test infrastructure only: nothing in the library includes it.
#pragma once

#include <setjmp.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <ucontext.h>

#include <math.h>

#include <functional>
#include <map>
#include <vector>

#if defined(__has_feature)
#if __has_feature(address_sanitizer)
#define SALT_CPU_ASAN 1
#include <sanitizer/common_interface_defs.h>
#endif
#endif

#define __global__
#define __device__
#define __host__
#define __forceinline__ inline
#define __launch_bounds__(...)
#define amdgpu_waves_per_eu(...)   // an occupancy hint for the GPU compiler only
#define __shared__ static
#define __align__(n) __attribute__((aligned(n)))

struct int4 {
  int x, y, z, w;
};
struct uint4 {
  unsigned x, y, z, w;
};
struct float4 {
  float x, y, z, w;
};
inline int4 make_int4(int x, int y, int z, int w) { return int4{x, y, z, w}; }
inline uint4 make_uint4(unsigned x, unsigned y, unsigned z, unsigned w) { return uint4{x, y, z, w}; }
inline float4 make_float4(float x, float y, float z, float w) { return float4{x, y, z, w}; }
struct dim3 {
  unsigned x, y, z;
  dim3(unsigned a = 1, unsigned b = 1, unsigned c = 1) : x(a), y(b), z(c) {}
};

inline float __uint_as_float(uint32_t u) {
  float f;
  memcpy(&f, &u, 4);
  return f;
}
inline float __int_as_float(int32_t u) {
  float f;
  memcpy(&f, &u, 4);
  return f;
}
inline uint32_t __float_as_uint(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return u;
}
inline int min(int a, int b) { return a < b ? a : b; }
inline int max(int a, int b) { return a > b ? a : b; }

// ---- runtime types -----------------------------------------------------------
typedef enum {
  hipSuccess = 0,
  hipErrorInvalidValue = 1,
  hipErrorOutOfMemory = 2,
  hipErrorInvalidConfiguration = 9,
  hipErrorInvalidDevice = 101,
  hipErrorInvalidSymbol = 13,
  hipErrorLaunchFailure = 719
} hipError_t;
typedef struct salt_cpu_stream* hipStream_t;
typedef struct salt_cpu_event* hipEvent_t;
typedef enum {
  hipMemcpyHostToHost = 0,
  hipMemcpyHostToDevice = 1,
  hipMemcpyDeviceToHost = 2,
  hipMemcpyDeviceToDevice = 3,
  hipMemcpyDefault = 4
} hipMemcpyKind;
typedef enum { hipDeviceAttributeMultiprocessorCount, hipDeviceAttributeMaxSharedMemoryPerBlock } hipDeviceAttribute_t;
typedef enum { hipMemoryTypeUnregistered = 0, hipMemoryTypeHost = 1, hipMemoryTypeDevice = 2 } hipMemoryType;
struct hipPointerAttribute_t {
  hipMemoryType type;
  int device;
  void* devicePointer;
  void* hostPointer;
};
#define hipHostMallocDefault 0u
#define hipStreamNonBlocking 1u
#define hipEventDisableTiming 2u

namespace salt_cpu {

// ---- fibers ------------------------------------------------------------------
enum { kRun = 0, kWave = 1, kBlock = 2, kDone = 3 };
struct Fiber {
  jmp_buf jb;
  ucontext_t uc;
  char* stack = nullptr;
  size_t stack_size = 0;
  int state = kRun;
  bool started = false;
  void* fake = nullptr;
};
constexpr size_t kStack = 256 * 1024;
constexpr int kMaxThreads = 1024;

inline std::vector<Fiber>& fibers() {
  static std::vector<Fiber> f(kMaxThreads);
  return f;
}
inline int g_cur = -1, g_nthreads = 0;
inline dim3 g_block_idx, g_block_dim, g_grid_dim;
inline jmp_buf g_sched;
inline void* g_sched_fake = nullptr;
inline const void* g_main_bottom = nullptr;
inline size_t g_main_size = 0;
inline std::function<void()>* g_body = nullptr;
inline char* g_dyn_lds = nullptr;
inline int g_n_cu = 256;
alignas(16) inline unsigned char g_wave_buf[kMaxThreads / 64][64][128];

inline void to_scheduler(bool exiting) {
  Fiber& f = fibers()[g_cur];
#ifdef SALT_CPU_ASAN
  __sanitizer_start_switch_fiber(exiting ? nullptr : &f.fake, g_main_bottom, g_main_size);
#endif
  if (exiting) _longjmp(g_sched, 1);
  if (_setjmp(f.jb) == 0) _longjmp(g_sched, 1);
#ifdef SALT_CPU_ASAN
  __sanitizer_finish_switch_fiber(f.fake, &g_main_bottom, &g_main_size);
#endif
}

inline void fiber_entry() {
#ifdef SALT_CPU_ASAN
  __sanitizer_finish_switch_fiber(nullptr, &g_main_bottom, &g_main_size);
#endif
  (*g_body)();
  fibers()[g_cur].state = kDone;
  to_scheduler(true);
}

inline void wait_at(int state) {
  fibers()[g_cur].state = state;
  to_scheduler(false);
}

// Runs g_body on n threads of the current block until all have returned.
inline void run_block(int n) {
  std::vector<Fiber>& fs = fibers();
  for (int i = 0; i < n; ++i) {
    Fiber& f = fs[i];
    if (!f.stack) {
      f.stack = static_cast<char*>(malloc(kStack));
      f.stack_size = kStack;
    }
    f.state = kRun;
    f.started = false;
    f.fake = nullptr;
  }
  g_nthreads = n;
  for (;;) {
    for (int i = 0; i < n; ++i) {
      Fiber& f = fs[i];
      if (f.state != kRun) continue;
      g_cur = i;
      if (_setjmp(g_sched) == 0) {
#ifdef SALT_CPU_ASAN
        __sanitizer_start_switch_fiber(&g_sched_fake, f.stack, f.stack_size);
#endif
        if (!f.started) {
          f.started = true;
          getcontext(&f.uc);
          f.uc.uc_stack.ss_sp = f.stack;
          f.uc.uc_stack.ss_size = f.stack_size;
          f.uc.uc_link = nullptr;
          makecontext(&f.uc, fiber_entry, 0);
          setcontext(&f.uc);
        } else {
          _longjmp(f.jb, 1);
        }
      }
#ifdef SALT_CPU_ASAN
      __sanitizer_finish_switch_fiber(g_sched_fake, nullptr, nullptr);
#endif
    }
    g_cur = -1;
    // release waves whose live lanes all wait at a wave operation
    bool any = false, all_done = true, all_block = true;
    for (int w = 0; w * 64 < n; ++w) {
      bool live = false, all_wave = true;
      for (int i = w * 64; i < n && i < w * 64 + 64; ++i) {
        if (fs[i].state == kDone) continue;
        live = true;
        all_wave = all_wave && fs[i].state == kWave;
      }
      if (live && all_wave) {
        for (int i = w * 64; i < n && i < w * 64 + 64; ++i)
          if (fs[i].state == kWave) fs[i].state = kRun;
        any = true;
      }
    }
    for (int i = 0; i < n; ++i) {
      if (fs[i].state != kDone) all_done = false;
      if (fs[i].state != kDone && fs[i].state != kBlock) all_block = false;
    }
    if (all_done) break;
    if (!any && all_block) {
      for (int i = 0; i < n; ++i)
        if (fs[i].state == kBlock) fs[i].state = kRun;
      any = true;
    }
    if (!any) {
      fprintf(stderr, "salt_cpu: deadlock in block (%u, %u): threads wait at different barriers\n", g_block_idx.x,
              g_block_idx.y);
      abort();
    }
  }
}

inline dim3 thread_idx() {
  const int t = g_cur;
  return dim3((unsigned)(t % g_block_dim.x), (unsigned)((t / g_block_dim.x) % g_block_dim.y),
              (unsigned)(t / (g_block_dim.x * g_block_dim.y)));
}
inline int lane() { return g_cur & 63; }
inline int wave() { return g_cur >> 6; }

template <typename T>
inline T wave_xchg(T v, int src) {
  static_assert(sizeof(T) <= 128, "operand too large");
  memcpy(g_wave_buf[wave()][lane()], &v, sizeof(T));
  wait_at(kWave);
  T r;
  memcpy(&r, g_wave_buf[wave()][src & 63], sizeof(T));
  wait_at(kWave);
  return r;
}

template <class F>
inline void launch(dim3 grid, dim3 block, size_t lds, F&& body) {
  const int n = (int)(block.x * block.y * block.z);
  if (n <= 0 || n > kMaxThreads) {
    fprintf(stderr, "salt_cpu: block of %d threads\n", n);
    abort();
  }
  g_grid_dim = grid;
  g_block_dim = block;
  std::function<void()> fn = body;
  g_body = &fn;
  for (unsigned z = 0; z < grid.z; ++z)
    for (unsigned y = 0; y < grid.y; ++y)
      for (unsigned x = 0; x < grid.x; ++x) {
        g_block_idx = dim3(x, y, z);
        g_dyn_lds = lds ? static_cast<char*>(malloc(lds)) : nullptr;
        if (g_dyn_lds) memset(g_dyn_lds, 0xA5, lds);   // LDS starts undefined
        run_block(n);
        free(g_dyn_lds);
        g_dyn_lds = nullptr;
      }
  g_body = nullptr;
}

// ---- allocations -------------------------------------------------------------
struct Alloc {
  size_t size;
  bool host;
};
inline std::map<uintptr_t, Alloc>& allocs() {
  static std::map<uintptr_t, Alloc> m;
  return m;
}
inline void* alloc(size_t n, bool host) {
  void* p = malloc(n ? n : 1);
  if (p) allocs()[reinterpret_cast<uintptr_t>(p)] = Alloc{n, host};
  return p;
}
inline bool release(void* p) {
  auto it = allocs().find(reinterpret_cast<uintptr_t>(p));
  if (it == allocs().end()) return false;
  allocs().erase(it);
  free(p);
  return true;
}
inline const Alloc* find(const void* p) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  auto it = allocs().upper_bound(a);
  if (it == allocs().begin()) return nullptr;
  --it;
  return a < it->first + (it->second.size ? it->second.size : 1) ? &it->second : nullptr;
}

}  // namespace salt_cpu

#define threadIdx (salt_cpu::thread_idx())
#define blockIdx (salt_cpu::g_block_idx)
#define blockDim (salt_cpu::g_block_dim)
#define gridDim (salt_cpu::g_grid_dim)

inline void __syncthreads() { salt_cpu::wait_at(salt_cpu::kBlock); }
template <typename T>
inline T __shfl_xor(T v, int m, int = 64) {
  return salt_cpu::wave_xchg(v, salt_cpu::lane() ^ m);
}
template <typename T>
inline T __shfl_up(T v, unsigned d, int = 64) {
  const int l = salt_cpu::lane();
  return salt_cpu::wave_xchg(v, l >= (int)d ? l - (int)d : l);
}
template <typename T>
inline T __shfl_down(T v, unsigned d, int = 64) {
  const int l = salt_cpu::lane();
  return salt_cpu::wave_xchg(v, l + (int)d < 64 ? l + (int)d : l);
}
inline int atomicAdd(int* p, int v) {
  const int o = *p;
  *p = o + v;
  return o;
}
inline float atomicAdd(float* p, float v) {
  const float o = *p;
  *p = o + v;
  return o;
}

// ---- MFMA and dot products (gfx950 lane layouts) ----------------------------------
typedef __bf16 salt_cpu_bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 salt_cpu_bf16x2 __attribute__((ext_vector_type(2)));
typedef float salt_cpu_f32x4 __attribute__((ext_vector_type(4)));

inline salt_cpu_f32x4 salt_cpu_mfma_bf16(salt_cpu_bf16x8 a, salt_cpu_bf16x8 b, salt_cpu_f32x4 c, int, int, int) {
  struct Op {
    float a[8], b[8];
  };
  Op mine;
  for (int e = 0; e < 8; ++e) {
    mine.a[e] = (float)a[e];
    mine.b[e] = (float)b[e];
  }
  const int l = salt_cpu::lane(), w = salt_cpu::wave();
  memcpy(salt_cpu::g_wave_buf[w][l], &mine, sizeof mine);
  salt_cpu::wait_at(salt_cpu::kWave);
  salt_cpu_f32x4 d;
  const int col = l & 15, g = l >> 4;
  for (int e = 0; e < 4; ++e) {
    const int row = 4 * g + e;
    double acc = c[e];
    for (int k = 0; k < 32; ++k) {
      Op A, B;
      memcpy(&A, salt_cpu::g_wave_buf[w][row + 16 * (k / 8)], sizeof A);
      memcpy(&B, salt_cpu::g_wave_buf[w][col + 16 * (k / 8)], sizeof B);
      acc += (double)A.a[k % 8] * (double)B.b[k % 8];
    }
    d[e] = (float)acc;
  }
  salt_cpu::wait_at(salt_cpu::kWave);
  return d;
}

inline salt_cpu_f32x4 salt_cpu_mfma_f32(float a, float b, salt_cpu_f32x4 c, int, int, int) {
  float mine[2] = {a, b};
  const int l = salt_cpu::lane(), w = salt_cpu::wave();
  memcpy(salt_cpu::g_wave_buf[w][l], mine, sizeof mine);
  salt_cpu::wait_at(salt_cpu::kWave);
  salt_cpu_f32x4 d;
  const int col = l & 15, g = l >> 4;
  for (int e = 0; e < 4; ++e) {
    const int row = 4 * g + e;
    double acc = c[e];
    for (int k = 0; k < 4; ++k) {
      float A[2], B[2];
      memcpy(A, salt_cpu::g_wave_buf[w][row + 16 * k], sizeof A);
      memcpy(B, salt_cpu::g_wave_buf[w][col + 16 * k], sizeof B);
      acc += (double)A[0] * (double)B[1];
    }
    d[e] = (float)acc;
  }
  salt_cpu::wait_at(salt_cpu::kWave);
  return d;
}

inline float salt_cpu_fdot2_bf16(salt_cpu_bf16x2 a, salt_cpu_bf16x2 b, float c, bool) {
  return (float)((double)c + (double)(float)a[0] * (double)(float)b[0] + (double)(float)a[1] * (double)(float)b[1]);
}

// ---- raw buffer resources ------------------------------------------------------------
// (base, size in bytes); an access at an offset >= size reads zero and a store
// there is dropped, as the hardware range check does.  An access that starts
// inside the buffer but ends past it is a kernel bug here (the kernels never
// make one) and aborts the run.
struct salt_cpu_rsrc {
  const char* base;
  uint32_t n;
};
typedef unsigned int salt_cpu_u32x4 __attribute__((ext_vector_type(4)));
inline salt_cpu_rsrc salt_cpu_make_rsrc(void* p, short, int n, int) { return salt_cpu_rsrc{(const char*)p, (uint32_t)n}; }
inline bool salt_cpu_buf_in(salt_cpu_rsrc r, int off, int soff, uint32_t size) {
  const uint32_t o = (uint32_t)off + (uint32_t)soff;
  if (o >= r.n) return false;
  if (o + size > r.n || o + size < o) {
    fprintf(stderr, "buffer access [%u, %u) straddles the end of a %u-byte buffer\n", o, o + size, r.n);
    abort();
  }
  return true;
}
inline salt_cpu_u32x4 salt_cpu_buf_load_b128(salt_cpu_rsrc r, int off, int soff, int) {
  salt_cpu_u32x4 v = {0u, 0u, 0u, 0u};
  if (salt_cpu_buf_in(r, off, soff, 16)) memcpy(&v, r.base + (uint32_t)off + (uint32_t)soff, 16);
  return v;
}
inline unsigned salt_cpu_buf_load_b32(salt_cpu_rsrc r, int off, int soff, int) {
  unsigned v = 0u;
  if (salt_cpu_buf_in(r, off, soff, 4)) memcpy(&v, r.base + (uint32_t)off + (uint32_t)soff, 4);
  return v;
}
inline void salt_cpu_buf_store_b128(salt_cpu_u32x4 v, salt_cpu_rsrc r, int off, int soff, int) {
  if (salt_cpu_buf_in(r, off, soff, 16)) memcpy(const_cast<char*>(r.base) + (uint32_t)off + (uint32_t)soff, &v, 16);
}
inline void salt_cpu_buf_store_b32(unsigned v, salt_cpu_rsrc r, int off, int soff, int) {
  if (salt_cpu_buf_in(r, off, soff, 4)) memcpy(const_cast<char*>(r.base) + (uint32_t)off + (uint32_t)soff, &v, 4);
}
#define __amdgpu_buffer_rsrc_t salt_cpu_rsrc
#define __builtin_amdgcn_make_buffer_rsrc salt_cpu_make_rsrc
#define __builtin_amdgcn_raw_buffer_load_b128 salt_cpu_buf_load_b128
#define __builtin_amdgcn_raw_buffer_load_b32 salt_cpu_buf_load_b32
#define __builtin_amdgcn_raw_buffer_store_b128 salt_cpu_buf_store_b128
#define __builtin_amdgcn_raw_buffer_store_b32 salt_cpu_buf_store_b32

#define __builtin_amdgcn_mfma_f32_16x16x32_bf16 salt_cpu_mfma_bf16
#define __builtin_amdgcn_mfma_f32_16x16x4f32 salt_cpu_mfma_f32
#define __builtin_amdgcn_fdot2_f32_bf16 salt_cpu_fdot2_bf16

// ---- runtime API (synchronous) -------------------------------------------------------
// a file-scope __device__ array is a host array here; its "device address" is its address
#define HIP_SYMBOL(x) (&(x))
inline hipError_t hipGetSymbolAddress(void** p, const void* sym) {
  *p = const_cast<void*>(sym);
  return hipSuccess;
}
inline hipError_t hipGetLastError() { return hipSuccess; }
inline const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "cpu runtime error"; }
inline hipError_t hipSetDevice(int d) { return d == 0 ? hipSuccess : hipErrorInvalidDevice; }
inline hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
inline hipError_t hipDeviceSynchronize() { return hipSuccess; }
template <typename F>
inline hipError_t hipOccupancyMaxActiveBlocksPerMultiprocessor(int* n, F, int, size_t) {
  *n = 2;
  return hipSuccess;
}
inline hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t a, int) {
  *v = a == hipDeviceAttributeMultiprocessorCount ? salt_cpu::g_n_cu : 160 * 1024;
  return hipSuccess;
}
inline hipError_t hipMalloc(void** p, size_t n) {
  *p = salt_cpu::alloc(n, false);
  return *p ? hipSuccess : hipErrorOutOfMemory;
}
template <typename T>
inline hipError_t hipMalloc(T** p, size_t n) {
  return hipMalloc(reinterpret_cast<void**>(p), n);
}
inline hipError_t hipFree(void* p) { return (!p || salt_cpu::release(p)) ? hipSuccess : hipErrorInvalidValue; }
inline hipError_t hipHostMalloc(void** p, size_t n, unsigned) {
  *p = salt_cpu::alloc(n, true);
  return *p ? hipSuccess : hipErrorOutOfMemory;
}
template <typename T>
inline hipError_t hipHostMalloc(T** p, size_t n, unsigned f) {
  return hipHostMalloc(reinterpret_cast<void**>(p), n, f);
}
inline hipError_t hipHostFree(void* p) { return hipFree(p); }
inline hipError_t hipHostGetDevicePointer(void** d, void* h, unsigned) {
  const salt_cpu::Alloc* al = salt_cpu::find(h);
  if (!al || !al->host) return hipErrorInvalidValue;
  *d = h;
  return hipSuccess;
}
inline hipError_t hipMemcpy(void* d, const void* s, size_t n, hipMemcpyKind) {
  if (n) memcpy(d, s, n);
  return hipSuccess;
}
inline hipError_t hipMemcpyAsync(void* d, const void* s, size_t n, hipMemcpyKind k, hipStream_t) {
  return hipMemcpy(d, s, n, k);
}
inline hipError_t hipMemset(void* d, int v, size_t n) {
  if (n) memset(d, v, n);
  return hipSuccess;
}
inline hipError_t hipMemsetAsync(void* d, int v, size_t n, hipStream_t) { return hipMemset(d, v, n); }
inline hipError_t hipStreamCreateWithFlags(hipStream_t* s, unsigned) {
  *s = reinterpret_cast<hipStream_t>(new int(0));
  return hipSuccess;
}
inline hipError_t hipStreamDestroy(hipStream_t s) {
  delete reinterpret_cast<int*>(s);
  return hipSuccess;
}
inline hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
inline hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned) { return hipSuccess; }
inline hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) {
  *e = reinterpret_cast<hipEvent_t>(new int(0));
  return hipSuccess;
}
inline hipError_t hipEventCreate(hipEvent_t* e) { return hipEventCreateWithFlags(e, 0); }
inline hipError_t hipEventDestroy(hipEvent_t e) {
  delete reinterpret_cast<int*>(e);
  return hipSuccess;
}
inline hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
inline hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
inline hipError_t hipPointerGetAttributes(hipPointerAttribute_t* a, const void* p) {
  const salt_cpu::Alloc* al = salt_cpu::find(p);
  if (!al) return hipErrorInvalidValue;
  a->type = al->host ? hipMemoryTypeHost : hipMemoryTypeDevice;
  a->device = 0;
  a->devicePointer = const_cast<void*>(p);
  a->hostPointer = al->host ? const_cast<void*>(p) : nullptr;
  return hipSuccess;
}

template <typename... KArgs, typename... Args>
inline void hipLaunchKernelGGL(void (*k)(KArgs...), dim3 grid, dim3 block, size_t lds, hipStream_t,
                               Args&&... args) {
  salt_cpu::launch(grid, block, lds, [&]() { k(args...); });
}
template <typename... KArgs, typename... Args>
inline void hipExtLaunchKernelGGL(void (*k)(KArgs...), dim3 grid, dim3 block, size_t lds, hipStream_t, hipEvent_t,
                                  hipEvent_t, unsigned, Args&&... args) {
  salt_cpu::launch(grid, block, lds, [&]() { k(args...); });
}
