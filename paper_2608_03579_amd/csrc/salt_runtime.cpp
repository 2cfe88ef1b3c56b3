// libsalt host runtime: the C ABI of include/salt.h.
//
// Owns the pinned centroid store, the residual slot pool, the side stream that
// swaps residuals in, plan buffers, and the stream/event bookkeeping that keeps a
// swap from overwriting a slot an in-flight apply still reads (Sec. 3.1 / 3.3:
// pin the centroid once, swap only the rank <= 2 residual).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/salt.h"
#include "salt_internal.h"

using salt::ApplyArgs;
using salt::PlanBuffers;

namespace {

constexpr int kEvRing = 1024;         // reader / loader event rings
constexpr size_t kAlign = 256;

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
size_t esize_of(salt_dtype d) { return d == SALT_F32 ? 4 : 2; }

// A ring of events with monotone sequence numbers.  Before slot k % N is
// re-recorded, the event it held (sequence k - N) is synchronised, so every
// sequence <= `done` is known complete.
struct EventRing {
  std::vector<hipEvent_t> ev;
  int64_t next = 0;   // sequence number of the next record
  int64_t done = -1;  // all sequences <= done have completed
};

}  // namespace

struct salt_plan {
  PlanBuffers dev{};
  int4* staging = nullptr;          // pinned host copy of the maps
  hipEvent_t staged = nullptr;      // recorded after the H2D copy of the maps
  bool staged_pending = false;
  int32_t T = 0;
  bool built = false;
  std::vector<int32_t> slots;       // distinct referenced slots
  std::vector<int32_t> slot_rank;   // rank of each at set_maps time
  int32_t M = 16;                   // tokens per tile
  int32_t n_tiles = 0;
  int32_t n_groups_c = 0;           // groups with a centroid
  int64_t sum_ru = 0;               // residual rank summed over tokens
  uint32_t arrivals = 0;            // per-tile arrival count after the last enqueued apply (ordered sums)
  uint32_t epoch = 0;               // applies enqueued since creation or the last epoch reset
  // A build of a small batch is deferred: the next apply on the same stream
  // plans the batch itself.  Any other use of the plan first launches the
  // deferred build on the stream it was requested on.
  mutable bool build_pending = false;   // running the deferred build changes no visible state
  hipStream_t build_stream = nullptr;
  // atomic sums: rows of each v buffer that may be nonzero (all rows below)
  int32_t v_dirty[2] = {0, 0};
  // Applies of this plan enqueued on reader_stream since its last reader event:
  // the event that covers them (a swap of one of the plan's slots waits for
  // it) is recorded only when something needs it, not after every apply.
  bool readers_open = false;
  hipStream_t reader_stream = nullptr;
};

struct salt_ctx {
  salt_config cfg{};
  std::vector<salt_shape> tables;
  std::vector<int64_t> tab_prefix;       // sum of (in + out) over earlier tables
  int64_t sum_io = 0;
  size_t esize = 2;
  int device = 0;
  int n_cu = 256;                        // compute units of the device
  int occ_shrink = 0, occ_expand = 0;    // blocks per compute unit of the two-launch kernels (0: not asked yet)
  // device memory
  std::vector<char*> cent_at, cent_b;    // per table
  std::vector<uint8_t> cent_pinned;      // per table x centroid
  char* pool = nullptr;
  size_t slot_stride = 0;
  hipStream_t side = nullptr;
  // bookkeeping
  std::vector<int32_t> slot_rank;        // -1 = never loaded
  std::vector<int64_t> slot_reader;      // apply sequence of the last reader
  std::vector<int64_t> slot_loader;      // load sequence of the last swap
  EventRing readers, loaders;
  std::vector<salt_plan*> plans;
  bool poisoned = false;
  std::string err;
};

namespace {

// message of the last salt_create failure on this thread (salt_last_error(NULL))
thread_local std::string g_create_err;

salt_status fail(salt_ctx* c, salt_status s, const char* fmt, ...) {
  if (c) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    c->err = buf;
  }
  return s;
}

salt_status hip_fail(salt_ctx* c, hipError_t e, const char* what) {
  if (c) {
    c->poisoned = true;
    c->err = std::string(what) + ": " + hipGetErrorString(e);
  }
  return SALT_ERR_HIP;
}

#define SALT_HIP(ctx, call)                                   \
  do {                                                        \
    hipError_t e_ = (call);                                   \
    if (e_ != hipSuccess) return hip_fail((ctx), e_, #call);  \
  } while (0)

// dst[i][o][j] = src[i][j][o] for n matrices of rc x out elements.
template <typename W>
void transpose_rank_major(const W* src, W* dst, size_t n, size_t rc, size_t out) {
  for (size_t i = 0; i < n; ++i) {
    const W* s = src + i * rc * out;
    W* d = dst + i * out * rc;
    for (size_t o0 = 0; o0 < out; o0 += 64)
      for (size_t j = 0; j < rc; ++j)
        for (size_t o = o0; o < std::min(out, o0 + 64); ++o) d[o * rc + j] = s[j * out + o];
  }
}

constexpr int kMaxGramRank = 256;   // largest adapter rank of salt_adapter_gram
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Split-K partial sums go through device atomics unless the context asked for
// bit-reproducible results.
bool atomic_sums(const salt_ctx* c) { return (c->cfg.flags & SALT_DETERMINISTIC) == 0; }

// Epochs are compared modulo 2^32 by signed difference; restart them well before
// a ready word could fall 2^31 epochs behind.
constexpr uint32_t kEpochReset = 1u << 30;

// Launches the plan kernel now.  reset_ready restarts the plan's epochs.
hipError_t launch_build(const salt_plan* plan, hipStream_t s, bool reset_ready) {
  salt::PlanArgs pa{};
  pa.b = plan->dev;
  pa.T = plan->T;
  pa.M = plan->M;
  pa.reset_ready = reset_ready ? 1 : 0;
  return salt::launch_plan(pa, s);
}

// Runs a deferred build (see salt_plan) on the stream it was requested on.
hipError_t flush_build(const salt_plan* plan) {
  if (!plan->build_pending) return hipSuccess;
  plan->build_pending = false;
  return launch_build(plan, plan->build_stream, false);
}

hipError_t ring_record(EventRing& r, hipStream_t s, int64_t* seq_out) {
  const int64_t seq = r.next;
  const int k = (int)(seq % (int64_t)r.ev.size());
  if (seq >= (int64_t)r.ev.size() && seq - (int64_t)r.ev.size() > r.done) {
    hipError_t e = hipEventSynchronize(r.ev[k]);
    if (e != hipSuccess) return e;
    r.done = seq - (int64_t)r.ev.size();
  }
  hipError_t e = hipEventRecord(r.ev[k], s);
  if (e != hipSuccess) return e;
  r.next = seq + 1;
  *seq_out = seq;
  return hipSuccess;
}

// Make `s` wait for sequence `seq` of ring `r` unless it is known complete.
hipError_t ring_wait(EventRing& r, hipStream_t s, int64_t seq) {
  if (seq < 0 || seq <= r.done) return hipSuccess;
  return hipStreamWaitEvent(s, r.ev[(int)(seq % (int64_t)r.ev.size())], 0);
}

// Record the reader event that covers the plan's open applies and hand its
// sequence to every slot the plan references.
hipError_t close_readers(salt_ctx* ctx, salt_plan* plan) {
  if (!plan->readers_open) return hipSuccess;
  int64_t seq;
  hipError_t e = ring_record(ctx->readers, plan->reader_stream, &seq);
  if (e != hipSuccess) return e;
  for (int slot : plan->slots) ctx->slot_reader[slot] = std::max(ctx->slot_reader[slot], seq);
  plan->readers_open = false;
  return hipSuccess;
}

// After an apply of `plan` on `s`: its reads of the plan's slots are open.
hipError_t open_readers(salt_ctx* ctx, salt_plan* plan, hipStream_t s) {
  if (plan->readers_open && plan->reader_stream != s) {
    hipError_t e = close_readers(ctx, plan);
    if (e != hipSuccess) return e;
  }
  plan->readers_open = true;
  plan->reader_stream = s;
  return hipSuccess;
}

void free_plan_buffers(salt_plan* p) {
  PlanBuffers& b = p->dev;
  void* ptrs[] = {b.maps, b.perm, b.srt, b.srt_c, b.seg_off, b.seg_c, b.seg_u, b.grp_off,
                  b.grp_tok, b.grp_c, b.tiles, b.arrive, b.ready, b.meta, b.counter, b.partials, b.v,
                  b.sink};
  for (void* q : ptrs)
    if (q) (void)hipFree(q);
  if (p->staging) (void)hipHostFree(p->staging);
  if (p->staged) (void)hipEventDestroy(p->staged);
}

void destroy_ctx_memory(salt_ctx* c) {
  for (char* p : c->cent_at)
    if (p) (void)hipFree(p);
  for (char* p : c->cent_b)
    if (p) (void)hipFree(p);
  if (c->pool) (void)hipFree(c->pool);
  for (hipEvent_t e : c->readers.ev)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : c->loaders.ev)
    if (e) (void)hipEventDestroy(e);
  if (c->side) (void)hipStreamDestroy(c->side);
}

}  // namespace

extern "C" {

const char* salt_status_str(salt_status s) {
  switch (s) {
    case SALT_OK: return "ok";
    case SALT_ERR_INVALID_ARG: return "invalid argument";
    case SALT_ERR_OUT_OF_RANGE: return "out of range";
    case SALT_ERR_OUT_OF_MEMORY: return "out of memory";
    case SALT_ERR_NOT_PINNED: return "residual blob is not page-locked";
    case SALT_ERR_SLOT_EMPTY: return "slot was never loaded";
    case SALT_ERR_HIP: return "HIP runtime error";
    case SALT_ERR_BAD_STATE: return "bad state";
  }
  return "unknown status";
}

const char* salt_last_error(const salt_ctx* ctx) { return ctx ? ctx->err.c_str() : g_create_err.c_str(); }

int32_t salt_version(void) { return SALT_VERSION; }

size_t salt_residual_bytes_for(salt_dtype dtype, int32_t n_tables, const salt_shape* tables,
                               int32_t r_u) {
  if (!tables || n_tables <= 0 || r_u < 0 || (dtype != SALT_F32 && dtype != SALT_BF16)) return 0;
  size_t sum = 0;
  for (int i = 0; i < n_tables; ++i) {
    if (tables[i].in_dim <= 0 || tables[i].out_dim <= 0) return 0;
    sum += (size_t)tables[i].in_dim + (size_t)tables[i].out_dim;
  }
  return (size_t)r_u * sum * esize_of(dtype);
}

size_t salt_residual_bytes(const salt_ctx* ctx, int32_t r_u) {
  if (!ctx || r_u < 0 || r_u > ctx->cfg.r_u_max) return 0;
  return (size_t)r_u * (size_t)ctx->sum_io * ctx->esize;
}

salt_status salt_host_alloc(size_t bytes, void** out) {
  if (!out || bytes == 0) return SALT_ERR_INVALID_ARG;
  *out = nullptr;
  if (hipHostMalloc(out, bytes, hipHostMallocDefault) != hipSuccess) {
    *out = nullptr;
    return SALT_ERR_OUT_OF_MEMORY;
  }
  return SALT_OK;
}

void salt_host_free(void* p) {
  if (p) (void)hipHostFree(p);
}

salt_status salt_create(const salt_config* cfg, salt_ctx** out) {
  if (!cfg || !out) return SALT_ERR_INVALID_ARG;
  *out = nullptr;
  g_create_err = "invalid configuration";
  if (cfg->dtype != SALT_F32 && cfg->dtype != SALT_BF16) return SALT_ERR_INVALID_ARG;
  if (cfg->n_tables < 1 || !cfg->tables) return SALT_ERR_INVALID_ARG;
  if (cfg->n_centroids < 0 || cfg->n_centroids > 64 || cfg->r_c < 0 || cfg->r_c > salt::kMaxRc ||
      cfg->r_c % 8 != 0 || (cfg->n_centroids == 0) != (cfg->r_c == 0))
    return SALT_ERR_OUT_OF_RANGE;
  if (cfg->n_slots < 1 || cfg->n_slots > (1 << 20) || cfg->r_u_max < 0 || cfg->r_u_max > salt::kMaxRu)
    return SALT_ERR_OUT_OF_RANGE;
  if (cfg->max_tokens < 1 || cfg->max_tokens > (1 << 20)) return SALT_ERR_OUT_OF_RANGE;
  if (cfg->flags & ~SALT_DETERMINISTIC) return SALT_ERR_INVALID_ARG;
  for (int i = 0; i < cfg->n_tables; ++i) {
    const salt_shape s = cfg->tables[i];
    if (s.in_dim <= 0 || s.out_dim <= 0 || s.in_dim % 8 || s.out_dim % 8 || s.in_dim > (1 << 20) ||
        s.out_dim > (1 << 20))
      return SALT_ERR_INVALID_ARG;
  }
  salt_ctx* c = new (std::nothrow) salt_ctx();
  if (!c) return SALT_ERR_OUT_OF_MEMORY;
  c->cfg = *cfg;
  c->tables.assign(cfg->tables, cfg->tables + cfg->n_tables);
  c->cfg.tables = c->tables.data();
  c->esize = esize_of(cfg->dtype);
  c->device = cfg->device;
  int64_t acc = 0;
  for (const salt_shape& s : c->tables) {
    c->tab_prefix.push_back(acc);
    acc += (int64_t)s.in_dim + s.out_dim;
  }
  c->sum_io = acc;

  auto bail = [&](salt_status st, hipError_t e, const char* what) {
    if (st == SALT_ERR_HIP) hip_fail(c, e, what);
    else c->err = "device allocation failed";
    g_create_err = c->err;
    destroy_ctx_memory(c);
    delete c;
    return st;
  };
  hipError_t e = hipSetDevice(cfg->device);
  if (e != hipSuccess) return bail(SALT_ERR_HIP, e, "hipSetDevice");
  e = salt::kernels_init(cfg->device);
  if (e != hipSuccess) return bail(SALT_ERR_HIP, e, "kernels_init");
  e = hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, cfg->device);
  if (e != hipSuccess) return bail(SALT_ERR_HIP, e, "hipDeviceGetAttribute");
  const size_t C = (size_t)cfg->n_centroids, rc = (size_t)cfg->r_c;
  c->cent_at.assign(cfg->n_tables, nullptr);
  c->cent_b.assign(cfg->n_tables, nullptr);
  c->cent_pinned.assign((size_t)cfg->n_tables * C, 0);
  if (C > 0) {
    for (int t = 0; t < cfg->n_tables; ++t) {
      const salt_shape s = c->tables[t];
      if (hipMalloc((void**)&c->cent_at[t], C * rc * s.in_dim * c->esize) != hipSuccess ||
          hipMalloc((void**)&c->cent_b[t], C * rc * s.out_dim * c->esize) != hipSuccess) {
        (void)hipGetLastError();
        return bail(SALT_ERR_OUT_OF_MEMORY, hipSuccess, "");
      }
    }
  }
  c->slot_stride = round_up(std::max<size_t>(1, salt_residual_bytes(c, cfg->r_u_max)), kAlign);
  if (hipMalloc((void**)&c->pool, c->slot_stride * (size_t)cfg->n_slots) != hipSuccess) {
    (void)hipGetLastError();
    return bail(SALT_ERR_OUT_OF_MEMORY, hipSuccess, "");
  }
  e = hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking);
  if (e != hipSuccess) return bail(SALT_ERR_HIP, e, "hipStreamCreateWithFlags");
  c->readers.ev.assign(kEvRing, nullptr);
  c->loaders.ev.assign(kEvRing, nullptr);
  for (int i = 0; i < kEvRing; ++i) {
    if ((e = hipEventCreateWithFlags(&c->readers.ev[i], hipEventDisableTiming)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&c->loaders.ev[i], hipEventDisableTiming)) != hipSuccess)
      return bail(SALT_ERR_HIP, e, "hipEventCreateWithFlags");
  }
  c->slot_rank.assign(cfg->n_slots, -1);
  c->slot_reader.assign(cfg->n_slots, -1);
  c->slot_loader.assign(cfg->n_slots, -1);
  g_create_err.clear();
  *out = c;
  return SALT_OK;
}

void salt_destroy(salt_ctx* ctx) {
  if (!ctx) return;
  (void)hipSetDevice(ctx->device);
  (void)hipDeviceSynchronize();
  for (salt_plan* p : ctx->plans) {
    free_plan_buffers(p);
    delete p;
  }
  destroy_ctx_memory(ctx);
  delete ctx;
}

salt_status salt_pin_centroids(salt_ctx* ctx, int32_t table, int32_t c0, int32_t n,
                               const void* At_host, const void* B_host) {
  if (!ctx) return SALT_ERR_INVALID_ARG;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  if (table < 0 || table >= ctx->cfg.n_tables)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "table %d not in [0, %d)", table, ctx->cfg.n_tables);
  if (n < 0 || c0 < 0 || c0 + n > ctx->cfg.n_centroids)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "centroids [%d, %d) not in [0, %d)", c0, c0 + n,
                ctx->cfg.n_centroids);
  if (n == 0) return SALT_OK;
  if (!At_host || !B_host) return fail(ctx, SALT_ERR_INVALID_ARG, "null centroid array");
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  const salt_shape s = ctx->tables[table];
  const size_t rc = ctx->cfg.r_c, es = ctx->esize, out = s.out_dim;
  const size_t a_bytes = (size_t)n * rc * s.in_dim * es;
  SALT_HIP(ctx, hipMemcpy(ctx->cent_at[table] + (size_t)c0 * rc * s.in_dim * es, At_host, a_bytes,
                          hipMemcpyHostToDevice));
  // B is kept transposed on the device, [C][out][r_c], so that the expand reads
  // the 8 consecutive ranks of one output column with one 16-byte load
  std::vector<char> bt((size_t)n * rc * out * es);
  if (es == 2)
    transpose_rank_major(static_cast<const uint16_t*>(B_host), reinterpret_cast<uint16_t*>(bt.data()), n, rc, out);
  else
    transpose_rank_major(static_cast<const uint32_t*>(B_host), reinterpret_cast<uint32_t*>(bt.data()), n, rc, out);
  SALT_HIP(ctx, hipMemcpy(ctx->cent_b[table] + (size_t)c0 * rc * out * es, bt.data(), bt.size(),
                          hipMemcpyHostToDevice));
  for (int i = c0; i < c0 + n; ++i) ctx->cent_pinned[(size_t)table * ctx->cfg.n_centroids + i] = 1;
  return SALT_OK;
}

salt_status salt_load_residual(salt_ctx* ctx, int32_t slot, int32_t r_u, const void* blob,
                               size_t bytes) {
  if (!ctx) return SALT_ERR_INVALID_ARG;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  if (slot < 0 || slot >= ctx->cfg.n_slots)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "slot %d not in [0, %d)", slot, ctx->cfg.n_slots);
  if (r_u < 0 || r_u > ctx->cfg.r_u_max)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "rank %d not in [0, %d]", r_u, ctx->cfg.r_u_max);
  const size_t want = salt_residual_bytes(ctx, r_u);
  if (bytes != want)
    return fail(ctx, SALT_ERR_INVALID_ARG, "blob is %zu bytes, rank %d needs %zu", bytes, r_u, want);
  if (want > 0) {
    if (!blob || !aligned16(blob)) return fail(ctx, SALT_ERR_INVALID_ARG, "null or misaligned blob");
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, blob);
    if (e != hipSuccess || attr.type != hipMemoryTypeHost) {
      (void)hipGetLastError();
      return fail(ctx, SALT_ERR_NOT_PINNED, "blob %p is not page-locked host memory", blob);
    }
  }
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  // the swap may not overwrite what an enqueued apply still reads
  for (salt_plan* p : ctx->plans)
    if (p->readers_open && std::binary_search(p->slots.begin(), p->slots.end(), slot))
      SALT_HIP(ctx, close_readers(ctx, p));
  SALT_HIP(ctx, ring_wait(ctx->readers, ctx->side, ctx->slot_reader[slot]));
  if (want > 0)
    SALT_HIP(ctx, hipMemcpyAsync(ctx->pool + (size_t)slot * ctx->slot_stride, blob, want,
                                 hipMemcpyHostToDevice, ctx->side));
  int64_t seq;
  SALT_HIP(ctx, ring_record(ctx->loaders, ctx->side, &seq));
  ctx->slot_loader[slot] = seq;
  ctx->slot_rank[slot] = r_u;
  return SALT_OK;
}

salt_status salt_wait_loads(salt_ctx* ctx) {
  if (!ctx) return SALT_ERR_INVALID_ARG;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  SALT_HIP(ctx, hipStreamSynchronize(ctx->side));
  ctx->loaders.done = ctx->loaders.next - 1;
  return SALT_OK;
}

salt_status salt_plan_create(salt_ctx* ctx, salt_plan** out) {
  if (!ctx || !out) return SALT_ERR_INVALID_ARG;
  *out = nullptr;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  salt_plan* p = new (std::nothrow) salt_plan();
  if (!p) return SALT_ERR_OUT_OF_MEMORY;
  const size_t T = (size_t)ctx->cfg.max_tokens;
  const size_t R = salt::padded_rank(ctx->cfg.r_c, ctx->cfg.r_u_max);
  PlanBuffers& b = p->dev;
  // split-K partials for up to max(8 T, 64K) (split, token) pairs
  b.partial_cap = std::max<size_t>(8 * T, 65536) * R;
  b.v_stride = T * R;
  // tiles: at most ceil(T / M) + one partial tile per centroid group (<= 65)
  b.tiles_max = (int32_t)((T + 15) / 16 + 66);
  b.tile_cap = 0;
  for (size_t M : {16, 32, 64}) b.tile_cap = std::max(b.tile_cap, ((T + M - 1) / M + 66) * (M + 1));
  bool ok = hipMalloc((void**)&b.maps, T * sizeof(int4)) == hipSuccess &&
            hipMalloc((void**)&b.perm, T * 4) == hipSuccess &&
            hipMalloc((void**)&b.srt, T * sizeof(int4)) == hipSuccess &&
            hipMalloc((void**)&b.srt_c, T * 4) == hipSuccess &&
            hipMalloc((void**)&b.seg_off, (T + 1) * 4) == hipSuccess &&
            hipMalloc((void**)&b.seg_c, T * 4) == hipSuccess &&
            hipMalloc((void**)&b.seg_u, T * 4) == hipSuccess &&
            hipMalloc((void**)&b.grp_off, (T + 1) * 4) == hipSuccess &&
            hipMalloc((void**)&b.grp_tok, (T + 1) * 4) == hipSuccess &&
            hipMalloc((void**)&b.grp_c, T * 4) == hipSuccess &&
            hipMalloc((void**)&b.tiles, b.tile_cap * sizeof(int4)) == hipSuccess &&
            hipMalloc((void**)&b.arrive, (size_t)b.tiles_max * salt::kCounterStride * 4) == hipSuccess &&
            hipMalloc((void**)&b.ready, (size_t)b.tiles_max * salt::kReadyPerTile * 4) == hipSuccess &&
            hipMalloc((void**)&b.v, 2 * T * R * 4) == hipSuccess &&
            hipMalloc((void**)&b.meta, salt::kMetaWords * 4) == hipSuccess &&
            hipMalloc((void**)&b.counter, 64 * 4) == hipSuccess &&
            hipMalloc((void**)&b.partials, b.partial_cap * 4) == hipSuccess &&
            hipMalloc((void**)&b.sink, salt::kSinkBytes) == hipSuccess &&
            hipHostMalloc((void**)&p->staging, T * sizeof(int4), hipHostMallocDefault) == hipSuccess;
  if (!ok) {
    (void)hipGetLastError();
    free_plan_buffers(p);
    delete p;
    return fail(ctx, SALT_ERR_OUT_OF_MEMORY, "plan buffers for %zu tokens do not fit", T);
  }
  hipError_t e = hipEventCreateWithFlags(&p->staged, hipEventDisableTiming);
  if (e == hipSuccess) e = hipMemset(b.counter, 0, 64 * 4);
  if (e == hipSuccess) e = hipMemset(b.meta, 0, salt::kMetaWords * 4);
  if (e == hipSuccess) e = hipMemset(b.arrive, 0, (size_t)b.tiles_max * salt::kCounterStride * 4);
  if (e == hipSuccess) e = hipMemset(b.ready, 0, (size_t)b.tiles_max * salt::kReadyPerTile * 4);
  if (e == hipSuccess) e = hipMemset(b.v, 0, 2 * T * R * 4);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    free_plan_buffers(p);
    delete p;
    return hip_fail(ctx, e, "plan init");
  }
  ctx->plans.push_back(p);
  *out = p;
  return SALT_OK;
}

void salt_plan_destroy(salt_ctx* ctx, salt_plan* plan) {
  if (!ctx || !plan) return;
  auto it = std::find(ctx->plans.begin(), ctx->plans.end(), plan);
  if (it == ctx->plans.end()) return;
  (void)hipSetDevice(ctx->device);
  (void)hipDeviceSynchronize();
  ctx->plans.erase(it);
  free_plan_buffers(plan);
  delete plan;
}

salt_status salt_plan_set_maps(salt_ctx* ctx, salt_plan* plan, int32_t T, const int32_t* tok_c,
                               const int32_t* tok_u, const float* tok_gamma, void* stream) {
  if (!ctx || !plan) return SALT_ERR_INVALID_ARG;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  if (T < 0 || T > ctx->cfg.max_tokens)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "T = %d not in [0, %d]", T, ctx->cfg.max_tokens);
  if (T > 0 && (!tok_c || !tok_u)) return fail(ctx, SALT_ERR_INVALID_ARG, "null map");
  const int C = ctx->cfg.n_centroids, S = ctx->cfg.n_slots;
  for (int t = 0; t < T; ++t) {
    if (tok_c[t] < -1 || tok_c[t] >= C)
      return fail(ctx, SALT_ERR_OUT_OF_RANGE, "tok_c[%d] = %d not in [-1, %d)", t, tok_c[t], C);
    if (tok_u[t] < -1 || tok_u[t] >= S)
      return fail(ctx, SALT_ERR_OUT_OF_RANGE, "tok_u[%d] = %d not in [-1, %d)", t, tok_u[t], S);
    if (tok_u[t] >= 0 && ctx->slot_rank[tok_u[t]] < 0)
      return fail(ctx, SALT_ERR_SLOT_EMPTY, "tok_u[%d] = %d: slot never loaded", t, tok_u[t]);
    if (tok_gamma && !std::isfinite(tok_gamma[t]))
      return fail(ctx, SALT_ERR_INVALID_ARG, "tok_gamma[%d] is not finite", t);
  }
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  hipStream_t s = (hipStream_t)stream;
  SALT_HIP(ctx, flush_build(plan));
  // the staging buffer may still feed the previous copy
  if (plan->staged_pending) {
    SALT_HIP(ctx, hipEventSynchronize(plan->staged));
    plan->staged_pending = false;
  }
  std::vector<int32_t> slots;
  std::vector<int32_t> per_c((size_t)C + 1, 0);   // tokens per centroid id (+1 for c = -1)
  int64_t sum_ru = 0;
  for (int t = 0; t < T; ++t) {
    const int u = tok_u[t];
    const int r = u >= 0 ? ctx->slot_rank[u] : 0;
    const float g = tok_gamma ? tok_gamma[t] : 1.0f;
    int32_t gbits;
    std::memcpy(&gbits, &g, 4);
    plan->staging[t] = make_int4(tok_c[t], u, r, gbits);
    if (u >= 0) slots.push_back(u);
    per_c[(size_t)tok_c[t] + 1]++;
    sum_ru += r;
  }
  std::sort(slots.begin(), slots.end());
  slots.erase(std::unique(slots.begin(), slots.end()), slots.end());
  // the previous batch's applies still read the old slots
  SALT_HIP(ctx, close_readers(ctx, plan));
  plan->slots = slots;
  plan->slot_rank.resize(slots.size());
  for (size_t i = 0; i < slots.size(); ++i) plan->slot_rank[i] = ctx->slot_rank[slots[i]];
  // tile size from the mean group size; the tile count is exact
  int n_groups = 0, n_groups_c = 0;
  for (int g = 0; g <= C; ++g)
    if (per_c[g]) {
      ++n_groups;
      n_groups_c += (g > 0);
    }
  const double mean = n_groups ? (double)T / n_groups : 0.0;
  plan->M = (ctx->cfg.dtype == SALT_F32 || mean <= 24.0) ? 16 : 32;
  // large bf16 batches with long centroid groups and residual rank <= 2: the
  // two-launch apply with 64-token tiles (bandwidth bound; no in-launch hand-off)
  if (ctx->cfg.dtype == SALT_BF16 && T > salt::kPlanFusedT && ctx->cfg.r_u_max <= 2 && mean >= 96.0)
    plan->M = salt::kTwoPassM;
  int n_tiles = 0;
  for (int g = 0; g <= C; ++g) n_tiles += (per_c[g] + plan->M - 1) / plan->M;
  plan->n_tiles = n_tiles;
  plan->n_groups_c = n_groups_c;
  plan->sum_ru = sum_ru;
  plan->T = T;
  plan->built = false;
  if (T > 0) {
    SALT_HIP(ctx, hipMemcpyAsync(plan->dev.maps, plan->staging, (size_t)T * sizeof(int4),
                                 hipMemcpyHostToDevice, s));
    SALT_HIP(ctx, hipEventRecord(plan->staged, s));
    plan->staged_pending = true;
  }
  return SALT_OK;
}

salt_status salt_plan_build(salt_ctx* ctx, salt_plan* plan, void* stream) {
  if (!ctx || !plan) return SALT_ERR_INVALID_ARG;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  SALT_HIP(ctx, flush_build(plan));
  const bool reset = plan->epoch >= kEpochReset;
  if (reset) plan->epoch &= 1u;   // keeps the parity that picks the v buffer
  if (!reset && atomic_sums(ctx) && plan->T > 0 && plan->T <= salt::kPlanFusedT) {
    plan->build_pending = true;
    plan->build_stream = (hipStream_t)stream;
  } else {
    SALT_HIP(ctx, launch_build(plan, (hipStream_t)stream, reset));
  }
  plan->built = true;
  plan->arrivals = 0;
  return SALT_OK;
}

salt_status salt_plan_tiling(salt_ctx* ctx, const salt_plan* plan, int32_t* tile_tokens, int32_t* n_tiles,
                             int32_t* launches) {
  if (!ctx || !plan) return SALT_ERR_INVALID_ARG;
  if (plan->T < 0 || plan->M <= 0) return fail(ctx, SALT_ERR_BAD_STATE, "no maps were set on the plan");
  if (tile_tokens) *tile_tokens = plan->M;
  if (n_tiles) *n_tiles = plan->n_tiles;
  if (launches) *launches = plan->M == salt::kTwoPassM ? 2 : 1;
  return SALT_OK;
}

salt_status salt_plan_errors(salt_ctx* ctx, const salt_plan* plan, void* stream, int32_t* n_errors) {
  if (!ctx || !plan || !n_errors) return SALT_ERR_INVALID_ARG;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  *n_errors = 0;
  if (!plan->built || plan->T == 0) return SALT_OK;
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  SALT_HIP(ctx, flush_build(plan));
  SALT_HIP(ctx, hipStreamSynchronize((hipStream_t)stream));
  if (plan->build_stream && plan->build_stream != (hipStream_t)stream)
    SALT_HIP(ctx, hipStreamSynchronize(plan->build_stream));
  int32_t meta[salt::kMetaWords];
  SALT_HIP(ctx, hipMemcpy(meta, plan->dev.meta, sizeof meta, hipMemcpyDeviceToHost));
  if (meta[salt::kMetaNTiles] != plan->n_tiles) {
    *n_errors = 1;
    return fail(ctx, SALT_ERR_BAD_STATE, "device plan has %d tiles, host expected %d",
                meta[salt::kMetaNTiles], plan->n_tiles);
  }
  *n_errors = meta[salt::kMetaErr];
  if (meta[salt::kMetaErr] != 0) {
    const int32_t zero = 0;
    SALT_HIP(ctx, hipMemcpy(plan->dev.meta + salt::kMetaErr, &zero, 4, hipMemcpyHostToDevice));
  }
  return SALT_OK;
}

salt_status salt_plan_download(salt_ctx* ctx, const salt_plan* plan, void* stream, int32_t* perm,
                               int32_t* seg_off, int32_t* seg_c, int32_t* seg_u, int32_t* grp_off,
                               int32_t* n_seg, int32_t* n_grp) {
  if (!ctx || !plan) return SALT_ERR_INVALID_ARG;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  if (!plan->built) return fail(ctx, SALT_ERR_BAD_STATE, "plan was not built");
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  hipStream_t s = (hipStream_t)stream;
  SALT_HIP(ctx, flush_build(plan));
  SALT_HIP(ctx, hipStreamSynchronize(s));
  if (plan->build_stream && plan->build_stream != s) SALT_HIP(ctx, hipStreamSynchronize(plan->build_stream));
  const int T = plan->T;
  int32_t meta[3] = {0, 0, 0};
  if (T > 0) SALT_HIP(ctx, hipMemcpy(meta, plan->dev.meta, sizeof meta, hipMemcpyDeviceToHost));
  const int ns = meta[0], ng = meta[1];
  if (n_seg) *n_seg = ns;
  if (n_grp) *n_grp = ng;
  if (T == 0) {
    if (seg_off) seg_off[0] = 0;
    if (grp_off) grp_off[0] = 0;
    return SALT_OK;
  }
  if (perm) SALT_HIP(ctx, hipMemcpy(perm, plan->dev.perm, (size_t)T * 4, hipMemcpyDeviceToHost));
  if (seg_off) SALT_HIP(ctx, hipMemcpy(seg_off, plan->dev.seg_off, (size_t)(ns + 1) * 4, hipMemcpyDeviceToHost));
  if (seg_c) SALT_HIP(ctx, hipMemcpy(seg_c, plan->dev.seg_c, (size_t)ns * 4, hipMemcpyDeviceToHost));
  if (seg_u) SALT_HIP(ctx, hipMemcpy(seg_u, plan->dev.seg_u, (size_t)ns * 4, hipMemcpyDeviceToHost));
  if (grp_off) SALT_HIP(ctx, hipMemcpy(grp_off, plan->dev.grp_off, (size_t)(ng + 1) * 4, hipMemcpyDeviceToHost));
  return SALT_OK;
}

namespace {
salt_status apply_impl(salt_ctx* ctx, int32_t table, salt_plan* plan, const void* x, void* y, void* stream,
                       hipEvent_t e0, hipEvent_t e1);
salt_status fuse_impl(salt_ctx* ctx, int32_t table, int32_t c, float gamma, void* w, int64_t ldw, void* stream,
                      hipEvent_t e0, hipEvent_t e1);
}  // namespace

salt_status salt_apply(salt_ctx* ctx, int32_t table, salt_plan* plan, const void* x, void* y,
                       void* stream) {
  return apply_impl(ctx, table, plan, x, y, stream, nullptr, nullptr);
}

salt_status salt_apply_timed(salt_ctx* ctx, int32_t table, salt_plan* plan, const void* x, void* y,
                             void* stream, void* start_event, void* stop_event) {
  if (!start_event || !stop_event) return fail(ctx, SALT_ERR_INVALID_ARG, "null event");
  return apply_impl(ctx, table, plan, x, y, stream, (hipEvent_t)start_event, (hipEvent_t)stop_event);
}

salt_status salt_fuse_centroid(salt_ctx* ctx, int32_t table, int32_t c, float gamma, void* w, int64_t ldw,
                               void* stream) {
  return fuse_impl(ctx, table, c, gamma, w, ldw, stream, nullptr, nullptr);
}

salt_status salt_fuse_centroid_timed(salt_ctx* ctx, int32_t table, int32_t c, float gamma, void* w, int64_t ldw,
                                     void* stream, void* start_event, void* stop_event) {
  if (!start_event || !stop_event) return fail(ctx, SALT_ERR_INVALID_ARG, "null event");
  return fuse_impl(ctx, table, c, gamma, w, ldw, stream, (hipEvent_t)start_event, (hipEvent_t)stop_event);
}

salt_status salt_route(int32_t K, const double* n_k, const double* mu_n, const double* sigma_n,
                       const double* mu_r, const double* sigma_r, double tau_n, double tau_r, double* z_n,
                       double* z_r, salt_route_result* out) {
  if (K < 2 || !n_k || !mu_n || !sigma_n || !mu_r || !sigma_r || !out) return SALT_ERR_INVALID_ARG;
  if (!std::isfinite(tau_n) || !std::isfinite(tau_r)) return SALT_ERR_INVALID_ARG;
  double total = 0.0;
  for (int k = 0; k < K; ++k) {
    if (!std::isfinite(n_k[k]) || n_k[k] < 0.0 || !std::isfinite(mu_n[k]) || !std::isfinite(mu_r[k]) ||
        !(sigma_n[k] > 0.0) || !(sigma_r[k] > 0.0) || !std::isfinite(sigma_n[k]) || !std::isfinite(sigma_r[k]))
      return SALT_ERR_INVALID_ARG;
    total += n_k[k];
  }
  for (int k = 0; k < K; ++k)
    if (!(total - n_k[k] > 0.0)) return SALT_ERR_INVALID_ARG;   // mean of the others must be positive
  salt_route_result r{};
  r.k_star = -1;
  // stage 1: distance of each norm from its centroid's calibrated range
  double zn_min = 0.0;
  for (int k = 0; k < K; ++k) {
    const double z = std::fabs(n_k[k] - mu_n[k]) / sigma_n[k];
    if (z_n) z_n[k] = z;
    if (k == 0 || z < zn_min) zn_min = z;
  }
  r.z_n_min = zn_min;
  if (zn_min > tau_n) {
    r.ood = 1;
    *out = r;
    return SALT_OK;
  }
  // stage 2: dominance ratio against the mean of the other centroids
  int best = 0;
  double zr_min = 0.0;
  for (int k = 0; k < K; ++k) {
    const double others = (total - n_k[k]) / (double)(K - 1);
    const double z = std::fabs(n_k[k] / others - mu_r[k]) / sigma_r[k];
    if (z_r) z_r[k] = z;
    if (k == 0 || z < zr_min) {
      zr_min = z;
      best = k;
    }
  }
  r.z_r_min = zr_min;
  if (zr_min > tau_r) r.blended = 1;
  else r.k_star = best;
  *out = r;
  return SALT_OK;
}

salt_status salt_adapter_gram(salt_ctx* ctx, const void* blob1, int32_t r1, const void* blob2, int32_t r2,
                              double* out, void* stream) {
  if (!ctx || !out) return SALT_ERR_INVALID_ARG;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  if (r1 < 1 || r1 > kMaxGramRank || r2 < 1 || r2 > kMaxGramRank)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "adapter ranks %d, %d not in [1, %d]", r1, r2, kMaxGramRank);
  if (!blob1 || !blob2 || !aligned16(blob1) || !aligned16(blob2))
    return fail(ctx, SALT_ERR_INVALID_ARG, "null or misaligned adapter");
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  hipStream_t s = (hipStream_t)stream;
  const int nt = ctx->cfg.n_tables;
  const size_t es = ctx->esize;
  std::vector<salt::GramTable> tabs(nt);
  size_t prefix = 0;
  int max_in = 0, max_out = 0;
  for (int t = 0; t < nt; ++t) {
    const salt_shape sh = ctx->tables[t];
    salt::GramTable& g = tabs[t];
    g.at1 = static_cast<const char*>(blob1) + (size_t)r1 * prefix * es;
    g.b1 = static_cast<const char*>(g.at1) + (size_t)r1 * sh.in_dim * es;
    g.at2 = static_cast<const char*>(blob2) + (size_t)r2 * prefix * es;
    g.b2 = static_cast<const char*>(g.at2) + (size_t)r2 * sh.in_dim * es;
    g.in_dim = sh.in_dim;
    g.out_dim = sh.out_dim;
    prefix += (size_t)sh.in_dim + sh.out_dim;
    max_in = std::max(max_in, sh.in_dim);
    max_out = std::max(max_out, sh.out_dim);
  }
  const int p1 = (r1 + 15) / 16 * 16, p2 = (r2 + 15) / 16 * 16;
  salt::GramArgs a{};
  a.n_tables = nt;
  a.r1 = r1;
  a.r2 = r2;
  a.g_12 = p1 * p2;
  a.g_11 = p1 * p1;
  a.g_22 = p2 * p2;
  a.g_side = (size_t)a.g_12 + a.g_11 + a.g_22;
  a.g_table = 2 * a.g_side;
  const size_t g_bytes = sizeof(float) * a.g_table * nt;
  void* tabs_d = nullptr;
  void* g_d = nullptr;
  void* out_d = nullptr;
  auto release = [&]() {
    if (tabs_d) (void)hipFree(tabs_d);
    if (g_d) (void)hipFree(g_d);
    if (out_d) (void)hipFree(out_d);
  };
  if (hipMalloc(&tabs_d, sizeof(salt::GramTable) * nt) != hipSuccess || hipMalloc(&g_d, g_bytes) != hipSuccess ||
      hipMalloc(&out_d, sizeof(double) * 3 * nt) != hipSuccess) {
    (void)hipGetLastError();
    release();
    return fail(ctx, SALT_ERR_OUT_OF_MEMORY, "adapter Gram scratch (%zu bytes)", g_bytes);
  }
  a.tabs = static_cast<const salt::GramTable*>(tabs_d);
  a.g = static_cast<float*>(g_d);
  a.out = static_cast<double*>(out_d);
  hipError_t e = hipMemcpyAsync(tabs_d, tabs.data(), sizeof(salt::GramTable) * nt, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipMemsetAsync(g_d, 0, g_bytes, s);
  if (e == hipSuccess) e = salt::launch_gram(a, max_in, max_out, ctx->cfg.dtype == SALT_BF16, s);
  if (e == hipSuccess) e = hipMemcpyAsync(out, out_d, sizeof(double) * 3 * nt, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  release();
  SALT_HIP(ctx, e);
  return SALT_OK;
}

}  // extern "C"

namespace {
salt_status fuse_impl(salt_ctx* ctx, int32_t table, int32_t c, float gamma, void* w, int64_t ldw, void* stream,
                      hipEvent_t e0, hipEvent_t e1) {
  if (!ctx) return SALT_ERR_INVALID_ARG;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  if (table < 0 || table >= ctx->cfg.n_tables)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "table %d not in [0, %d)", table, ctx->cfg.n_tables);
  const int C = ctx->cfg.n_centroids;
  if (c < 0 || c >= C) return fail(ctx, SALT_ERR_OUT_OF_RANGE, "centroid %d not in [0, %d)", c, C);
  if (!ctx->cent_pinned[(size_t)table * C + c])
    return fail(ctx, SALT_ERR_BAD_STATE, "centroid %d of table %d was never pinned", c, table);
  const salt_shape sh = ctx->tables[table];
  if (!w || !aligned16(w)) return fail(ctx, SALT_ERR_INVALID_ARG, "null or misaligned weight");
  if (ldw < sh.out_dim || ldw % 8 != 0)
    return fail(ctx, SALT_ERR_INVALID_ARG, "ldw %lld: need a multiple of 8 and >= out_dim %d", (long long)ldw,
                sh.out_dim);
  if (!std::isfinite(gamma)) return fail(ctx, SALT_ERR_INVALID_ARG, "gamma is not finite");
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  const size_t rc = ctx->cfg.r_c, es = ctx->esize;
  salt::FuseArgs f{};
  f.at = ctx->cent_at[table] + (size_t)c * rc * sh.in_dim * es;
  f.bt = ctx->cent_b[table] + (size_t)c * rc * sh.out_dim * es;
  f.w = w;
  f.ldw = ldw;
  f.in_dim = sh.in_dim;
  f.out_dim = sh.out_dim;
  f.r_c = (int32_t)rc;
  f.gamma = gamma;
  SALT_HIP(ctx, salt::launch_fuse(f, ctx->cfg.dtype == SALT_BF16, (hipStream_t)stream, e0, e1));
  return SALT_OK;
}

salt_status apply_impl(salt_ctx* ctx, int32_t table, salt_plan* plan, const void* x, void* y, void* stream,
                       hipEvent_t e0, hipEvent_t e1) {
  if (!ctx || !plan) return SALT_ERR_INVALID_ARG;
  if (ctx->poisoned) return fail(ctx, SALT_ERR_BAD_STATE, "context is poisoned: %s", ctx->err.c_str());
  if (table < 0 || table >= ctx->cfg.n_tables)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "table %d not in [0, %d)", table, ctx->cfg.n_tables);
  if (!plan->built) return fail(ctx, SALT_ERR_BAD_STATE, "plan was not built");
  const int T = plan->T;
  if (T == 0) return SALT_OK;
  if (!x || !y || !aligned16(x) || !aligned16(y))
    return fail(ctx, SALT_ERR_INVALID_ARG, "null or misaligned x / y");
  const int C = ctx->cfg.n_centroids;
  for (int i = 0; i < C; ++i)
    if (!ctx->cent_pinned[(size_t)table * C + i])
      return fail(ctx, SALT_ERR_BAD_STATE, "centroid %d of table %d was never pinned", i, table);
  int64_t need_load = -1;
  for (size_t i = 0; i < plan->slots.size(); ++i) {
    const int s = plan->slots[i];
    if (ctx->slot_rank[s] != plan->slot_rank[i])
      return fail(ctx, SALT_ERR_BAD_STATE,
                  "slot %d was reloaded with rank %d after the plan's maps were set (rank %d)", s,
                  ctx->slot_rank[s], plan->slot_rank[i]);
    need_load = std::max(need_load, ctx->slot_loader[s]);
  }
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  hipStream_t s = (hipStream_t)stream;
  // a deferred build runs inside this launch when it was requested on this stream
  const bool fused_plan = plan->build_pending && plan->build_stream == s;
  if (!fused_plan) SALT_HIP(ctx, flush_build(plan));
  SALT_HIP(ctx, ring_wait(ctx->loaders, s, need_load));

  const salt_shape sh = ctx->tables[table];
  ApplyArgs a{};
  a.x = x;
  a.y = y;
  a.cent_at = C ? ctx->cent_at[table] : nullptr;
  a.cent_bt = C ? ctx->cent_b[table] : nullptr;
  a.pool = ctx->pool;
  a.slot_stride = ctx->slot_stride;
  a.tab_prefix = ctx->tab_prefix[table];
  a.tiles = plan->dev.tiles;
  a.partials = plan->dev.partials;
  a.arrive = plan->dev.arrive;
  a.ready = plan->dev.ready;
  a.meta = plan->dev.meta;
  a.sink = plan->dev.sink;
  a.T = T;
  a.in_dim = sh.in_dim;
  a.out_dim = sh.out_dim;
  a.r_c = ctx->cfg.r_c;
  a.r_u_max = ctx->cfg.r_u_max;
  a.R = salt::padded_rank(a.r_c, a.r_u_max);
  a.n_tiles = plan->n_tiles;
  if (plan->M == salt::kTwoPassM) {
    // Two launches, each sized to what the device holds at once (one round of
    // blocks).  Shrink: (tile, K range) blocks, K ranges a multiple of 4 waves x
    // 32.  Expand: (tile, column range) blocks, each streaming its chunks two
    // at a time.
    if (!ctx->occ_shrink) {
      SALT_HIP(ctx, salt::two_pass_occupancy(a.r_c, a.r_u_max, a.R, &ctx->occ_shrink, &ctx->occ_expand));
      ctx->occ_shrink = std::max(1, ctx->occ_shrink);
      ctx->occ_expand = std::max(1, ctx->occ_expand);
    }
    const bool atomic = atomic_sums(ctx);
    const int gran = 128;
    int S = (int)std::max<int64_t>(1, (int64_t)ctx->occ_shrink * ctx->n_cu / a.n_tiles);
    S = std::min({S, 8, (sh.in_dim + gran - 1) / gran});
    while (!atomic && S > 1 && (size_t)S * T * a.R > plan->dev.partial_cap) --S;
    a.Kc = ((sh.in_dim + S - 1) / S + gran - 1) / gran * gran;
    a.S = (sh.in_dim + a.Kc - 1) / a.Kc;
    a.sk = a.S;
    const int chunks = (sh.out_dim + salt::kNC - 1) / salt::kNC;
    const int n_col = (int)std::min<int64_t>(
        chunks, std::max<int64_t>(1, (int64_t)ctx->occ_expand * ctx->n_cu / a.n_tiles));
    a.cpb = (chunks + n_col - 1) / n_col;
    a.n_col = (chunks + a.cpb - 1) / a.cpb;
    a.two_pass = 1;
    a.fused_plan = 0;
    a.writer = -1;
    a.maps = plan->dev.maps;
    a.partials = plan->dev.partials;
    a.atomic_sum = atomic ? 1 : 0;
    a.epoch = ++plan->epoch;
    a.clear_rows = T;
    if (atomic) {
      // the same alternating v buffers as the single-launch atomic sums
      const int p = (int)(a.epoch & 1u), q = p ^ 1;
      a.v = plan->dev.v + (size_t)p * plan->dev.v_stride;
      a.v_clear = plan->dev.v + (size_t)q * plan->dev.v_stride;
      a.clear_rows = std::max(T, plan->v_dirty[q]);
      plan->v_dirty[q] = 0;
      plan->v_dirty[p] = T;
    } else {
      a.v = plan->dev.v;
      a.v_clear = nullptr;
    }
    SALT_HIP(ctx, salt::launch_apply(a, 1, salt::kTwoPassM, s, e0, e1));
    SALT_HIP(ctx, open_readers(ctx, plan, s));
    return SALT_OK;
  }
  // K split.  Small (decode) batches are latency bound: spread the shrink input
  // over many blocks (~16 KiB each) so no CU streams much more than its share,
  // and let partial traffic reach half of the input.  Large (prefill) batches
  // are bandwidth bound: ~64 KiB blocks, partial traffic under a fifth.
  const int M = plan->M, KW = 64 / M;
  const double es = (double)ctx->esize;
  const double shrink_bytes = es * sh.in_dim * ((double)T + (double)plan->n_groups_c * a.r_c + (double)plan->sum_ru);
  const bool small = T <= 1024;
  const double block_bytes = small ? 16384.0 : 65536.0;
  const int s_bytes = (int)std::ceil(shrink_bytes / ((double)a.n_tiles * block_bytes));
  const int s_traffic = std::max(1, (int)((small ? 0.5 : 0.2) * shrink_bytes / ((double)T * a.R * 8.0)));
  const int gran = 32 * KW;
  // the last block of a tile sums S x M x R partials: keep that within ~64 KiB
  const bool atomic = atomic_sums(ctx);
  const int s_reduce = atomic ? salt::kMaxSplit : std::max(1, (int)(65536 / ((size_t)M * a.R * 4)));
  int S = std::max(1, std::min({s_bytes, s_traffic, s_reduce, salt::kMaxSplit, (sh.in_dim + gran - 1) / gran}));
  if (small) {
    // at most two register batches of U steps per wave (U as the kernel picks
    // it), so that the shrink loop runs straight through with every load in flight
    const int ru_t = a.r_u_max <= 1 ? 1 : (a.r_u_max <= 2 ? 2 : salt::kRankChunk);
    const int U = std::max(1, salt::shrink_batch(ctx->esize == 2 ? 4 : 8, 1, salt::centroid_blocks(a.r_c), ru_t) / 2);
    const int s_steps = (sh.in_dim + 2 * U * gran - 1) / (2 * U * gran);
    S = std::max(S, std::min({s_steps, salt::kMaxSplit, (sh.in_dim + gran - 1) / gran}));
  }
  // residual ranks above kRankChunk: one shrink block per (K range, chunk)
  const int nq = a.r_u_max > salt::kRankChunk ? (a.r_u_max + salt::kRankChunk - 1) / salt::kRankChunk : 1;
  S = std::max(1, std::min(S, salt::kMaxSplit / nq));
  while (S > 1 && (size_t)S * nq * T * a.R > plan->dev.partial_cap) --S;
  const int Kc = ((sh.in_dim + S - 1) / S + gran - 1) / gran * gran;
  a.Kc = Kc;
  a.sk = (sh.in_dim + Kc - 1) / Kc;   // <= S
  a.S = a.sk * nq;
  // expand: one kNC-column chunk per block while the launch fits the device
  // at about four blocks per compute unit; past that, each block streams several
  // chunks (two in flight), so that the expand blocks left beside the shrink
  // blocks are all resident and load their first chunks before v is ready
  const int chunks = (sh.out_dim + salt::kNC - 1) / salt::kNC;
  const int64_t n_exp = std::max<int64_t>({(int64_t)a.n_tiles, 4 * (int64_t)ctx->n_cu - (int64_t)a.n_tiles * a.S,
                                           2 * (int64_t)ctx->n_cu});
  a.cpb = (int)std::max<int64_t>(1, ((int64_t)a.n_tiles * chunks + n_exp - 1) / n_exp);
  a.n_col = (chunks + a.cpb - 1) / a.cpb;
  if (!atomic && a.S > 1) plan->arrivals += (uint32_t)a.S;
  a.target = plan->arrivals;
  a.epoch = ++plan->epoch;
  a.atomic_sum = atomic ? 1 : 0;
  a.clear_rows = T;
  if (atomic) {
    // v buffers alternate between applies: this apply sums into buffer
    // p = epoch & 1 (all zero: the previous apply cleared it) and clears the
    // other one, including rows an earlier larger batch used
    const int p = (int)(a.epoch & 1u), q = p ^ 1;
    a.v = plan->dev.v + (size_t)p * plan->dev.v_stride;
    a.v_clear = plan->dev.v + (size_t)q * plan->dev.v_stride;
    a.clear_rows = std::max(T, plan->v_dirty[q]);
    plan->v_dirty[q] = 0;
    plan->v_dirty[p] = T;
  } else {
    a.v = plan->dev.v;
    a.v_clear = nullptr;
  }
  a.fused_plan = fused_plan ? 1 : 0;
  a.writer = -1;
  a.maps = plan->dev.maps;
  if (fused_plan) {
    a.pb = plan->dev;
    a.writer = a.n_tiles * (a.S + a.n_col);   // one block past the apply's own
    plan->build_pending = false;
  }
  SALT_HIP(ctx, salt::launch_apply(a, ctx->cfg.dtype == SALT_BF16, M, s, e0, e1));
  SALT_HIP(ctx, open_readers(ctx, plan, s));
  return SALT_OK;
}

}  // namespace
