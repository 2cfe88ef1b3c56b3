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
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/salt.h"
#include "salt_internal.h"
#include "salt_launch.h"

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

// Page-locked ranges handed out by salt_host_alloc, with the address under
// which the device reads each (null if it has none): a blob inside one of them
// needs no pointer query before its swap, and one with a device view can be
// gathered by a kernel.
struct HostRange {
  uintptr_t start;
  size_t size;
  uintptr_t dev;      // device address of start, valid on device `device`
  int device;
};
struct HostRanges {
  std::mutex mu;
  std::vector<HostRange> r;   // sorted by start
  // The range holding [p, p + n), or null (call with mu held).
  const HostRange* find(const void* p, size_t n) const {
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    auto it = std::upper_bound(r.begin(), r.end(), a, [](uintptr_t x, const HostRange& h) { return x < h.start; });
    if (it == r.begin()) return nullptr;
    --it;
    return (a >= it->start && a - it->start <= it->size && n <= it->size - (a - it->start)) ? &*it : nullptr;
  }
  bool contains(const void* p, size_t n) {
    std::lock_guard<std::mutex> g(mu);
    return find(p, n) != nullptr;
  }
  // Address under which `device` reads host bytes [p, p + n), or null.
  const void* device_view(const void* p, size_t n, int device) {
    std::lock_guard<std::mutex> g(mu);
    const HostRange* h = find(p, n);
    if (!h || !h->dev || h->device != device) return nullptr;
    return reinterpret_cast<const void*>(h->dev + (reinterpret_cast<uintptr_t>(p) - h->start));
  }
  void add(void* p, size_t n, void* dev, int device) {
    std::lock_guard<std::mutex> g(mu);
    const HostRange v{reinterpret_cast<uintptr_t>(p), n, reinterpret_cast<uintptr_t>(dev), device};
    r.insert(std::upper_bound(r.begin(), r.end(), v.start,
                              [](uintptr_t x, const HostRange& h) { return x < h.start; }),
             v);
  }
  void remove(void* p) {
    std::lock_guard<std::mutex> g(mu);
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    for (auto it = r.begin(); it != r.end(); ++it)
      if (it->start == a) {
        r.erase(it);
        return;
      }
  }
};
HostRanges g_host_ranges;

}  // namespace

struct salt_plan {
  // device buffers, sized for max_tokens
  int4* staged_dev = nullptr;       // [max_T + 2 tile_cap]: the batch's maps [T], its tiles, its shrink tiles
  uint64_t* keys = nullptr;         // [2][max_T]
  int4* srt = nullptr;              // [max_T]
  int32_t* ints = nullptr;          // perm [max_T], seg_off / grp_off [max_T + 1], seg_c / seg_u [max_T]
  int32_t* meta = nullptr;          // [kMetaWords]
  float* partials = nullptr;
  size_t partial_cap = 0;           // floats
  int4* staging = nullptr;          // pinned host copy of maps + tiles
  hipEvent_t staged = nullptr;      // recorded after the H2D copy of the staging buffer
  bool staged_pending = false;
  hipEvent_t hop = nullptr;         // orders the plan's work across streams
  int32_t max_T = 0, tile_cap = 0;
  // the batch
  int32_t T = -1;                   // -1: no maps set
  bool built = false;
  int32_t M = 16;                   // tokens per tile
  int32_t n_tiles = 0;
  int32_t MS = 16;                  // tokens per shrink tile
  int32_t n_stiles = 0;             // shrink tiles: 0 when they are the tiles themselves
  int32_t n_groups_c = 0;           // centroids referenced
  int32_t ru_max = 0;               // largest residual rank referenced
  int64_t sum_rank = 0;             // ranks summed over the distinct referenced slots
  std::vector<int32_t> slots;       // distinct referenced slots
  std::vector<int32_t> slot_rank;   // rank of each at set_maps time
  // the stream of the last operation that touched the plan's device buffers
  bool used = false;
  hipStream_t last_stream = nullptr;
  // Applies of this plan enqueued on reader_stream since its last reader event:
  // the event that covers them (a swap of one of the plan's slots waits for
  // it) is recorded only when something needs it, not after every apply.
  bool readers_open = false;
  hipStream_t reader_stream = nullptr;

  int32_t* perm() const { return ints; }
  int32_t* seg_off() const { return ints + max_T; }
  int32_t* grp_off() const { return ints + 2 * max_T + 1; }
  int32_t* seg_c() const { return ints + 3 * max_T + 2; }
  int32_t* seg_u() const { return ints + 4 * max_T + 2; }
  static size_t n_ints(size_t T) { return 5 * T + 2; }
};

struct salt_ctx {
  salt_config cfg{};
  std::vector<salt_shape> tables;
  std::vector<int64_t> tab_prefix;       // sum of (in + out) over earlier tables
  int64_t sum_io = 0;
  size_t esize = 2;
  int device = 0;
  int n_cu = 256;                        // compute units of the device
  // device memory
  std::vector<char*> cent_at, cent_b;    // per table
  std::vector<uint8_t> cent_pinned;      // per table x centroid
  std::vector<uint8_t> table_ready;      // per table: every centroid pinned
  char* pool = nullptr;
  size_t slot_stride = 0;
  char* zeros = nullptr;                 // zero page of max(in, out) * esize bytes, never written after set-up
  char* gram = nullptr;                  // salt_adapter_gram's device scratch, grown on demand
  size_t gram_bytes = 0;
  hipStream_t side = nullptr;
  // bookkeeping
  std::vector<int32_t> slot_rank;        // -1 = never loaded
  std::vector<int64_t> slot_reader;      // reader sequence of the last apply that read the slot
  std::vector<int64_t> slot_loader;      // load sequence of the last swap
  EventRing readers, loaders;
  std::vector<salt_plan*> plans;
  salt_plan* map_plan = nullptr;         // the plan salt_apply_map builds and applies
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

#define SALT_LIVE(ctx)                                                                          \
  do {                                                                                          \
    if (!(ctx)) return SALT_ERR_INVALID_ARG;                                                    \
    if ((ctx)->poisoned) return fail((ctx), SALT_ERR_BAD_STATE, "context is poisoned: %s", (ctx)->err.c_str()); \
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

// Work on the plan's device buffers is about to be enqueued on `s`: if the
// plan's last work went to another stream, `s` first waits for it.  Work on a
// single stream needs no event.
hipError_t use_stream(salt_ctx* ctx, salt_plan* plan, hipStream_t s) {
  if (plan->used && plan->last_stream != s) {
    hipError_t e = close_readers(ctx, plan);
    if (e != hipSuccess) return e;
    e = hipEventRecord(plan->hop, plan->last_stream);
    if (e != hipSuccess) return e;
    e = hipStreamWaitEvent(s, plan->hop, 0);
    if (e != hipSuccess) return e;
  }
  plan->used = true;
  plan->last_stream = s;
  return hipSuccess;
}

void free_plan(salt_plan* p) {
  void* dev[] = {p->staged_dev, p->keys, p->srt, p->ints, p->meta, p->partials};
  for (void* q : dev)
    if (q) (void)hipFree(q);
  if (p->staging) (void)hipHostFree(p->staging);
  if (p->staged) (void)hipEventDestroy(p->staged);
  if (p->hop) (void)hipEventDestroy(p->hop);
  delete p;
}

void destroy_ctx_memory(salt_ctx* c) {
  for (char* p : c->cent_at)
    if (p) (void)hipFree(p);
  for (char* p : c->cent_b)
    if (p) (void)hipFree(p);
  if (c->pool) (void)hipFree(c->pool);
  if (c->zeros) (void)hipFree(c->zeros);
  if (c->gram) (void)hipFree(c->gram);
  for (hipEvent_t e : c->readers.ev)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : c->loaders.ev)
    if (e) (void)hipEventDestroy(e);
  if (c->side) (void)hipStreamDestroy(c->side);
}

salt_status plan_create(salt_ctx* ctx, salt_plan** out) {
  salt_plan* p = new (std::nothrow) salt_plan();
  if (!p) return fail(ctx, SALT_ERR_OUT_OF_MEMORY, "plan");
  const size_t T = (size_t)ctx->cfg.max_tokens;
  const size_t R = salt::padded_rank(ctx->cfg.r_c, ctx->cfg.r_u_max);
  p->max_T = (int32_t)T;
  p->tile_cap = salt::max_tiles((int)T, ctx->cfg.n_centroids);
  p->partial_cap = salt::plan_partial_cap(T, R);
  const size_t staged = T + 2 * (size_t)p->tile_cap;
  bool ok = hipMalloc((void**)&p->staged_dev, staged * sizeof(int4)) == hipSuccess &&
            hipMalloc((void**)&p->keys, 2 * T * sizeof(uint64_t)) == hipSuccess &&
            hipMalloc((void**)&p->srt, T * sizeof(int4)) == hipSuccess &&
            hipMalloc((void**)&p->ints, salt_plan::n_ints(T) * 4) == hipSuccess &&
            hipMalloc((void**)&p->meta, salt::kMetaWords * 4) == hipSuccess &&
            hipMalloc((void**)&p->partials, p->partial_cap * 4) == hipSuccess &&
            hipHostMalloc((void**)&p->staging, staged * sizeof(int4), hipHostMallocDefault) == hipSuccess;
  if (!ok) {
    (void)hipGetLastError();
    free_plan(p);
    return fail(ctx, SALT_ERR_OUT_OF_MEMORY, "plan buffers for %zu tokens do not fit", T);
  }
  hipError_t e = hipEventCreateWithFlags(&p->staged, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&p->hop, hipEventDisableTiming);
  if (e == hipSuccess) e = hipMemset(p->meta, 0, salt::kMetaWords * 4);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    free_plan(p);
    return hip_fail(ctx, e, "plan init");
  }
  ctx->plans.push_back(p);
  *out = p;
  return SALT_OK;
}

salt_status set_maps_impl(salt_ctx* ctx, salt_plan* plan, int32_t T, const int32_t* tok_c, const int32_t* tok_u,
                          const float* tok_gamma, hipStream_t s) {
  if (T < 0 || T > plan->max_T)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "T = %d not in [0, %d]", T, plan->max_T);
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
  // the staging buffer may still feed the previous copy
  if (plan->staged_pending) {
    SALT_HIP(ctx, hipEventSynchronize(plan->staged));
    plan->staged_pending = false;
  }
  // the previous batch's applies still read the old slots
  SALT_HIP(ctx, close_readers(ctx, plan));
  std::vector<int32_t> slots;
  std::vector<int> per_c((size_t)C + 1, 0);   // tokens per centroid id (+1 for c = -1)
  int ru_max = 0;
  for (int t = 0; t < T; ++t) {
    const int u = tok_u[t];
    const int r = u >= 0 ? ctx->slot_rank[u] : 0;
    const float g = tok_gamma ? tok_gamma[t] : 1.0f;
    int32_t gbits;
    std::memcpy(&gbits, &g, 4);
    plan->staging[t] = make_int4(tok_c[t], u, r, gbits);
    if (u >= 0) slots.push_back(u);
    per_c[(size_t)tok_c[t] + 1]++;
    ru_max = std::max(ru_max, r);
  }
  std::sort(slots.begin(), slots.end());
  slots.erase(std::unique(slots.begin(), slots.end()), slots.end());
  plan->slots = slots;
  plan->slot_rank.resize(slots.size());
  int64_t sum_rank = 0;
  for (size_t i = 0; i < slots.size(); ++i) {
    plan->slot_rank[i] = ctx->slot_rank[slots[i]];
    sum_rank += plan->slot_rank[i];
  }
  int n_groups = 0, n_groups_c = 0;
  for (int g = 0; g <= C; ++g)
    if (per_c[g]) {
      ++n_groups;
      n_groups_c += (g > 0);
    }
  plan->M = salt::choose_tile_tokens((int)ctx->esize, T, n_groups, n_groups_c > 0);
  // tiles of more than 64 tokens serve the expand only; the shrink then runs
  // its own 64-token tiles of the same sorted order
  std::vector<int4> tiles, stiles;
  salt::cut_tiles(per_c, plan->M, tiles);
  plan->MS = std::min(plan->M, 64);
  if (plan->MS != plan->M) salt::cut_tiles(per_c, plan->MS, stiles);
  if ((int)tiles.size() > plan->tile_cap || (int)stiles.size() > plan->tile_cap)
    return fail(ctx, SALT_ERR_BAD_STATE, "%zu tiles exceed the plan's %d", std::max(tiles.size(), stiles.size()),
                plan->tile_cap);
  std::copy(tiles.begin(), tiles.end(), plan->staging + T);
  std::copy(stiles.begin(), stiles.end(), plan->staging + T + tiles.size());
  plan->n_tiles = (int32_t)tiles.size();
  plan->n_stiles = (int32_t)stiles.size();
  plan->n_groups_c = n_groups_c;
  plan->ru_max = ru_max;
  plan->sum_rank = sum_rank;
  plan->T = T;
  plan->built = false;
  if (T > 0) {
    SALT_HIP(ctx, use_stream(ctx, plan, s));
    SALT_HIP(ctx, hipMemcpyAsync(plan->staged_dev, plan->staging,
                                 ((size_t)T + tiles.size() + stiles.size()) * sizeof(int4), hipMemcpyHostToDevice, s));
    SALT_HIP(ctx, hipEventRecord(plan->staged, s));
    plan->staged_pending = true;
  }
  return SALT_OK;
}

salt_status build_impl(salt_ctx* ctx, salt_plan* plan, hipStream_t s) {
  if (plan->T < 0) return fail(ctx, SALT_ERR_BAD_STATE, "no maps were set on the plan");
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  if (plan->T > 0) {
    SALT_HIP(ctx, use_stream(ctx, plan, s));
    salt::PlanLaunch pl{};
    pl.maps = plan->staged_dev;
    pl.tiles = plan->staged_dev + plan->T;
    pl.keys = plan->keys;
    pl.keys_sorted = plan->keys + plan->max_T;
    pl.srt = plan->srt;
    pl.perm = plan->perm();
    pl.seg_off = plan->seg_off();
    pl.seg_c = plan->seg_c();
    pl.seg_u = plan->seg_u();
    pl.grp_off = plan->grp_off();
    pl.meta = plan->meta;
    pl.T = plan->T;
    pl.n_tiles = plan->n_tiles + plan->n_stiles;              // both lists, checked alike
    pl.n_list0 = plan->n_tiles;
    SALT_HIP(ctx, salt::launch_plan(pl, s));
  }
  plan->built = true;
  return SALT_OK;
}

// The apply of `n` tables (ids `tables`, activations xs, outputs ys) on a
// built plan, in launches of at most kMaxJobs tables.  ev: null, or four events
// per launch (the timed form allows one launch).
// `scratch`: the launches keep their split-K partials in the device's static
// scratch (salt_apply_batch_noalloc) instead of the plan's own buffer.
salt_status apply_impl(salt_ctx* ctx, int32_t n, const int32_t* tables, salt_plan* plan, const void* const* xs,
                       void* const* ys, hipStream_t s, hipEvent_t* ev, bool scratch = false) {
  SALT_LIVE(ctx);
  if (!plan || n < 0 || (n > 0 && (!tables || !xs || !ys))) return fail(ctx, SALT_ERR_INVALID_ARG, "null argument");
  if (!plan->built) return fail(ctx, SALT_ERR_BAD_STATE, "plan was not built");
  if (ev && n > salt::kMaxJobs)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "a timed apply serves at most %d tables", salt::kMaxJobs);
  for (int i = 0; i < n; ++i) {
    const int t = tables[i];
    if (t < 0 || t >= ctx->cfg.n_tables)
      return fail(ctx, SALT_ERR_OUT_OF_RANGE, "table %d not in [0, %d)", t, ctx->cfg.n_tables);
    if (!ctx->table_ready[t])
      return fail(ctx, SALT_ERR_BAD_STATE, "centroids of table %d were not all pinned", t);
    if (plan->T > 0 && (!xs[i] || !ys[i] || !aligned16(xs[i]) || !aligned16(ys[i])))
      return fail(ctx, SALT_ERR_INVALID_ARG, "null or misaligned x / y of table %d", t);
  }
  const int T = plan->T;
  if (T == 0 || n == 0) return SALT_OK;
  int64_t need_load = -1;
  for (size_t i = 0; i < plan->slots.size(); ++i) {
    const int sl = plan->slots[i];
    if (ctx->slot_rank[sl] != plan->slot_rank[i])
      return fail(ctx, SALT_ERR_BAD_STATE,
                  "slot %d was reloaded with rank %d after the plan's maps were set (rank %d)", sl,
                  ctx->slot_rank[sl], plan->slot_rank[i]);
    need_load = std::max(need_load, ctx->slot_loader[sl]);
  }
  float* partials = plan->partials;
  int64_t partial_cap = (int64_t)plan->partial_cap;
  if (scratch) {
    // the plan's own capacity where it is smaller, so that the launch (and its
    // K split) is the one salt_apply_batch makes whenever the plan's fits
    partials = salt::static_scratch(ctx->device);
    partial_cap = std::min(partial_cap, (int64_t)salt::kScratchFloats);
    if (!partials) return fail(ctx, SALT_ERR_BAD_STATE, "the static scratch of device %d is not set up", ctx->device);
  }
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  SALT_HIP(ctx, use_stream(ctx, plan, s));
  SALT_HIP(ctx, ring_wait(ctx->loaders, s, need_load));
  const int C = ctx->cfg.n_centroids;
  for (int first = 0; first < n; first += salt::kMaxJobs) {
    const int nj = std::min(salt::kMaxJobs, n - first);
    salt::ApplyLaunch a{};
    a.tiles = plan->staged_dev + T;
    a.stiles = plan->n_stiles ? plan->staged_dev + T + plan->n_tiles : a.tiles;
    a.n_stiles = plan->n_stiles ? plan->n_stiles : plan->n_tiles;
    a.MS = plan->MS;
    a.srt = plan->srt;
    a.pool = ctx->pool;
    a.partials = partials;
    a.zeros = ctx->zeros;
    a.slot_stride = (int64_t)ctx->slot_stride;
    a.partial_cap = partial_cap;
    a.n_jobs = nj;
    a.T = T;
    a.n_tiles = plan->n_tiles;
    a.M = plan->M;
    a.C = C;
    a.r_c = ctx->cfg.r_c;
    a.n_slots = ctx->cfg.n_slots;
    a.r_u = plan->ru_max;
    a.nq = std::max(1, salt::cdiv(plan->ru_max, salt::kRankChunk));
    a.R = salt::padded_rank(a.r_c, a.r_u);
    a.esize = (int32_t)ctx->esize;
    a.n_cu = ctx->n_cu;
    for (int j = 0; j < nj; ++j) {
      const int t = tables[first + j];
      const salt_shape sh = ctx->tables[t];
      salt::Job& jb = a.jobs[j];
      jb.x = xs[first + j];
      jb.y = ys[first + j];
      jb.at_c = C ? ctx->cent_at[t] : nullptr;
      jb.bt_c = C ? ctx->cent_b[t] : nullptr;
      jb.prefix = ctx->tab_prefix[t];
      jb.in = sh.in_dim;
      jb.out = sh.out_dim;
    }
    if (!salt::configure_launch(a, ctx->n_cu, plan->n_groups_c, plan->sum_rank, salt::shrink_round_blocks(a))) {
      if (scratch)
        return fail(ctx, SALT_ERR_OUT_OF_RANGE,
                    "split-K partials of %d tables x %d tokens x %d ranks exceed the static scratch (%zu floats)", nj,
                    T, a.R, salt::kScratchFloats);
      return fail(ctx, SALT_ERR_BAD_STATE, "split-K partials of %d tables do not fit the plan", nj);
    }
    SALT_HIP(ctx, salt::launch_apply(a, s, ev));
  }
  SALT_HIP(ctx, open_readers(ctx, plan, s));
  return SALT_OK;
}

// Residual swaps of n slots: validated first (an invalid batch changes no
// state), then enqueued on the side stream behind the applies that read the
// slots, with one loader event for the batch.
salt_status load_impl(salt_ctx* ctx, int32_t n, const int32_t* slots, const int32_t* ranks, const void* const* blobs,
                      const size_t* bytes) {
  SALT_LIVE(ctx);
  if (n < 0 || (n > 0 && (!slots || !ranks || !blobs || !bytes)))
    return fail(ctx, SALT_ERR_INVALID_ARG, "null argument");
  for (int i = 0; i < n; ++i) {
    const int slot = slots[i], r_u = ranks[i];
    if (slot < 0 || slot >= ctx->cfg.n_slots)
      return fail(ctx, SALT_ERR_OUT_OF_RANGE, "slot %d not in [0, %d)", slot, ctx->cfg.n_slots);
    if (r_u < 0 || r_u > ctx->cfg.r_u_max)
      return fail(ctx, SALT_ERR_OUT_OF_RANGE, "rank %d not in [0, %d]", r_u, ctx->cfg.r_u_max);
    const size_t want = salt_residual_bytes(ctx, r_u);
    if (bytes[i] != want)
      return fail(ctx, SALT_ERR_INVALID_ARG, "blob %d is %zu bytes, rank %d needs %zu", i, bytes[i], r_u, want);
    if (want == 0) continue;
    const void* blob = blobs[i];
    if (!blob || !aligned16(blob)) return fail(ctx, SALT_ERR_INVALID_ARG, "null or misaligned blob %d", i);
    if (!g_host_ranges.contains(blob, want)) {
      hipPointerAttribute_t attr;
      hipError_t e = hipPointerGetAttributes(&attr, blob);
      if (e != hipSuccess || attr.type != hipMemoryTypeHost) {
        (void)hipGetLastError();
        return fail(ctx, SALT_ERR_NOT_PINNED, "blob %p is not page-locked host memory", blob);
      }
    }
  }
  if (n == 0) return SALT_OK;
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  // the swaps may not overwrite what an enqueued apply still reads
  int64_t wait_reader = -1;
  for (salt_plan* p : ctx->plans) {
    if (!p->readers_open) continue;
    for (int i = 0; i < n; ++i)
      if (std::binary_search(p->slots.begin(), p->slots.end(), slots[i])) {
        SALT_HIP(ctx, close_readers(ctx, p));
        break;
      }
  }
  for (int i = 0; i < n; ++i) wait_reader = std::max(wait_reader, ctx->slot_reader[slots[i]]);
  SALT_HIP(ctx, ring_wait(ctx->readers, ctx->side, wait_reader));
  // One gather kernel per kSwapMax blobs when every blob has a device view and
  // no slot repeats; otherwise one DMA copy per blob, in order (so that a slot
  // listed twice receives its last blob).
  std::vector<const void*> views((size_t)n, nullptr);
  bool gather = true;
  for (int i = 0; i < n && gather; ++i)
    if (bytes[i] > 0)
      gather = (views[(size_t)i] = g_host_ranges.device_view(blobs[i], bytes[i], ctx->device)) != nullptr;
  if (gather) {
    std::vector<int32_t> sorted(slots, slots + n);
    std::sort(sorted.begin(), sorted.end());
    gather = std::adjacent_find(sorted.begin(), sorted.end()) == sorted.end();
  }
  if (gather) {
    salt::SwapArgs g{};
    for (int i = 0; i < n; ++i) {
      if (bytes[i] == 0) continue;
      g.src[g.n] = static_cast<const uint4*>(views[(size_t)i]);
      g.dst[g.n] = reinterpret_cast<uint4*>(ctx->pool + (size_t)slots[i] * ctx->slot_stride);
      g.vecs[g.n] = (int64_t)(bytes[i] / 16);                 // (bytes: rank x sum of multiples of 8 x esize)
      if (++g.n == salt::kSwapMax) {
        SALT_HIP(ctx, salt::launch_swap(g, ctx->side));
        g.n = 0;
      }
    }
    SALT_HIP(ctx, salt::launch_swap(g, ctx->side));
  } else {
    for (int i = 0; i < n; ++i)
      if (bytes[i] > 0)
        SALT_HIP(ctx, hipMemcpyAsync(ctx->pool + (size_t)slots[i] * ctx->slot_stride, blobs[i], bytes[i],
                                     hipMemcpyHostToDevice, ctx->side));
  }
  int64_t seq;
  SALT_HIP(ctx, ring_record(ctx->loaders, ctx->side, &seq));
  for (int i = 0; i < n; ++i) {
    ctx->slot_loader[slots[i]] = seq;
    ctx->slot_rank[slots[i]] = ranks[i];
  }
  return SALT_OK;
}

salt_status fuse_impl(salt_ctx* ctx, int32_t table, int32_t c, float gamma, void* w, int64_t ldw, void* stream,
                      hipEvent_t e0, hipEvent_t e1) {
  SALT_LIVE(ctx);
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

size_t salt_residual_bytes_for(salt_dtype dtype, int32_t n_tables, const salt_shape* tables, int32_t r_u) {
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
  // the address under which the current device reads the buffer (swaps of a
  // context on that device gather from it)
  void* dev = nullptr;
  int device = -1;
  if (hipGetDevice(&device) != hipSuccess || hipHostGetDevicePointer(&dev, *out, 0) != hipSuccess) {
    (void)hipGetLastError();
    dev = nullptr;
  }
  g_host_ranges.add(*out, bytes, dev, device);
  return SALT_OK;
}

void salt_host_free(void* p) {
  if (!p) return;
  g_host_ranges.remove(p);
  (void)hipHostFree(p);
}

salt_status salt_create(const salt_config* cfg, salt_ctx** out) {
  if (!cfg || !out) return SALT_ERR_INVALID_ARG;
  *out = nullptr;
  g_create_err = "invalid configuration";
  if (cfg->dtype != SALT_F32 && cfg->dtype != SALT_BF16) return SALT_ERR_INVALID_ARG;
  if (cfg->n_tables < 1 || !cfg->tables) return SALT_ERR_INVALID_ARG;
  if (cfg->n_centroids < 0 || cfg->n_centroids > salt::kMaxC || cfg->r_c < 0 || cfg->r_c > salt::kMaxRc ||
      cfg->r_c % 8 != 0 || (cfg->n_centroids == 0) != (cfg->r_c == 0))
    return SALT_ERR_OUT_OF_RANGE;
  if (cfg->n_slots < 1 || cfg->n_slots > (1 << 20) || cfg->r_u_max < 0 || cfg->r_u_max > salt::kMaxRu)
    return SALT_ERR_OUT_OF_RANGE;
  if (cfg->max_tokens < 1 || cfg->max_tokens > salt::kMaxTokens) return SALT_ERR_OUT_OF_RANGE;
  if (cfg->flags != 0) return SALT_ERR_INVALID_ARG;
  for (int i = 0; i < cfg->n_tables; ++i) {
    const salt_shape s = cfg->tables[i];
    if (s.in_dim <= 0 || s.out_dim <= 0 || s.in_dim % 8 || s.out_dim % 8 || s.in_dim > (1 << 20) ||
        s.out_dim > (1 << 20))
      return SALT_ERR_INVALID_ARG;
    // x and y of a full batch are each addressed with 32-bit byte offsets
    const int64_t esz = cfg->dtype == SALT_F32 ? 4 : 2;
    if ((int64_t)cfg->max_tokens * std::max(s.in_dim, s.out_dim) * esz >= salt::kMaxBufferBytes) {
      g_create_err = "max_tokens x max(in_dim, out_dim) x element size must stay below 2 GiB";
      return SALT_ERR_OUT_OF_RANGE;
    }
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
  c->table_ready.assign(cfg->n_tables, C == 0 ? 1 : 0);
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
  size_t max_dim = 8;
  for (const salt_shape& s : c->tables) max_dim = std::max<size_t>(max_dim, std::max(s.in_dim, s.out_dim));
  const size_t zero_bytes = round_up(max_dim * c->esize, kAlign);
  if (hipMalloc((void**)&c->zeros, zero_bytes) != hipSuccess) {
    (void)hipGetLastError();
    return bail(SALT_ERR_OUT_OF_MEMORY, hipSuccess, "");
  }
  e = hipMemset(c->zeros, 0, zero_bytes);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) return bail(SALT_ERR_HIP, e, "zero page");
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
  for (salt_plan* p : ctx->plans) free_plan(p);
  destroy_ctx_memory(ctx);
  delete ctx;
}

salt_status salt_pin_centroids(salt_ctx* ctx, int32_t table, int32_t c0, int32_t n, const void* At_host,
                               const void* B_host) {
  SALT_LIVE(ctx);
  if (table < 0 || table >= ctx->cfg.n_tables)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "table %d not in [0, %d)", table, ctx->cfg.n_tables);
  if (n < 0 || c0 < 0 || c0 + n > ctx->cfg.n_centroids)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "centroids [%d, %d) not in [0, %d)", c0, c0 + n, ctx->cfg.n_centroids);
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
  const int C = ctx->cfg.n_centroids;
  for (int i = c0; i < c0 + n; ++i) ctx->cent_pinned[(size_t)table * C + i] = 1;
  bool all = true;
  for (int i = 0; i < C; ++i) all = all && ctx->cent_pinned[(size_t)table * C + i];
  ctx->table_ready[table] = all ? 1 : 0;
  return SALT_OK;
}

salt_status salt_load_residual(salt_ctx* ctx, int32_t slot, int32_t r_u, const void* blob, size_t bytes) {
  return load_impl(ctx, 1, &slot, &r_u, &blob, &bytes);
}

salt_status salt_load_residuals(salt_ctx* ctx, int32_t n, const int32_t* slots, const int32_t* ranks,
                                const void* const* blobs, const size_t* bytes) {
  return load_impl(ctx, n, slots, ranks, blobs, bytes);
}

salt_status salt_wait_loads(salt_ctx* ctx) {
  SALT_LIVE(ctx);
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  SALT_HIP(ctx, hipStreamSynchronize(ctx->side));
  ctx->loaders.done = ctx->loaders.next - 1;
  return SALT_OK;
}

salt_status salt_plan_create(salt_ctx* ctx, salt_plan** out) {
  if (!out) return SALT_ERR_INVALID_ARG;
  *out = nullptr;
  SALT_LIVE(ctx);
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  return plan_create(ctx, out);
}

void salt_plan_destroy(salt_ctx* ctx, salt_plan* plan) {
  if (!ctx || !plan) return;
  auto it = std::find(ctx->plans.begin(), ctx->plans.end(), plan);
  if (it == ctx->plans.end()) return;
  (void)hipSetDevice(ctx->device);
  (void)hipDeviceSynchronize();
  ctx->plans.erase(it);
  if (ctx->map_plan == plan) ctx->map_plan = nullptr;
  free_plan(plan);
}

salt_status salt_plan_set_maps(salt_ctx* ctx, salt_plan* plan, int32_t T, const int32_t* tok_c, const int32_t* tok_u,
                               const float* tok_gamma, void* stream) {
  SALT_LIVE(ctx);
  if (!plan) return SALT_ERR_INVALID_ARG;
  return set_maps_impl(ctx, plan, T, tok_c, tok_u, tok_gamma, (hipStream_t)stream);
}

salt_status salt_plan_build(salt_ctx* ctx, salt_plan* plan, void* stream) {
  SALT_LIVE(ctx);
  if (!plan) return SALT_ERR_INVALID_ARG;
  return build_impl(ctx, plan, (hipStream_t)stream);
}

salt_status salt_plan_tiling(salt_ctx* ctx, const salt_plan* plan, int32_t* tile_tokens, int32_t* n_tiles,
                             int32_t* launches) {
  if (!ctx || !plan) return SALT_ERR_INVALID_ARG;
  if (plan->T < 0) return fail(ctx, SALT_ERR_BAD_STATE, "no maps were set on the plan");
  if (tile_tokens) *tile_tokens = plan->M;
  if (n_tiles) *n_tiles = plan->n_tiles;
  if (launches) *launches = plan->T > 0 ? 2 : 0;
  return SALT_OK;
}

salt_status salt_plan_errors(salt_ctx* ctx, const salt_plan* plan_c, void* stream, int32_t* n_errors) {
  SALT_LIVE(ctx);
  if (!plan_c || !n_errors) return SALT_ERR_INVALID_ARG;
  salt_plan* plan = const_cast<salt_plan*>(plan_c);
  *n_errors = 0;
  if (!plan->built || plan->T <= 0) return SALT_OK;
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  hipStream_t s = (hipStream_t)stream;
  SALT_HIP(ctx, use_stream(ctx, plan, s));
  SALT_HIP(ctx, hipStreamSynchronize(s));
  int32_t meta[salt::kMetaWords];
  SALT_HIP(ctx, hipMemcpy(meta, plan->meta, sizeof meta, hipMemcpyDeviceToHost));
  *n_errors = meta[salt::kMetaErr];
  if (meta[salt::kMetaNTiles] != plan->n_tiles + plan->n_stiles || meta[salt::kMetaT] != plan->T) {
    *n_errors += 1;
    return fail(ctx, SALT_ERR_BAD_STATE, "device plan has %d tiles of %d tokens, host staged %d of %d",
                meta[salt::kMetaNTiles], meta[salt::kMetaT], plan->n_tiles + plan->n_stiles, plan->T);
  }
  return SALT_OK;
}

salt_status salt_plan_download(salt_ctx* ctx, const salt_plan* plan_c, void* stream, int32_t* perm, int32_t* seg_off,
                               int32_t* seg_c, int32_t* seg_u, int32_t* grp_off, int32_t* n_seg, int32_t* n_grp) {
  SALT_LIVE(ctx);
  if (!plan_c) return SALT_ERR_INVALID_ARG;
  salt_plan* plan = const_cast<salt_plan*>(plan_c);
  if (!plan->built) return fail(ctx, SALT_ERR_BAD_STATE, "plan was not built");
  SALT_HIP(ctx, hipSetDevice(ctx->device));
  hipStream_t s = (hipStream_t)stream;
  const int T = plan->T;
  int32_t meta[3] = {0, 0, 0};
  if (T > 0) {
    SALT_HIP(ctx, use_stream(ctx, plan, s));
    SALT_HIP(ctx, hipStreamSynchronize(s));
    SALT_HIP(ctx, hipMemcpy(meta, plan->meta, sizeof meta, hipMemcpyDeviceToHost));
  }
  const int ns = std::min(std::max(meta[0], 0), std::max(T, 0)), ng = std::min(std::max(meta[1], 0), ns);
  if (n_seg) *n_seg = ns;
  if (n_grp) *n_grp = ng;
  if (T == 0) {
    if (seg_off) seg_off[0] = 0;
    if (grp_off) grp_off[0] = 0;
    return SALT_OK;
  }
  if (perm) SALT_HIP(ctx, hipMemcpy(perm, plan->perm(), (size_t)T * 4, hipMemcpyDeviceToHost));
  if (seg_off) SALT_HIP(ctx, hipMemcpy(seg_off, plan->seg_off(), (size_t)(ns + 1) * 4, hipMemcpyDeviceToHost));
  if (seg_c) SALT_HIP(ctx, hipMemcpy(seg_c, plan->seg_c(), (size_t)ns * 4, hipMemcpyDeviceToHost));
  if (seg_u) SALT_HIP(ctx, hipMemcpy(seg_u, plan->seg_u(), (size_t)ns * 4, hipMemcpyDeviceToHost));
  if (grp_off) SALT_HIP(ctx, hipMemcpy(grp_off, plan->grp_off(), (size_t)(ng + 1) * 4, hipMemcpyDeviceToHost));
  return SALT_OK;
}

salt_status salt_apply(salt_ctx* ctx, int32_t table, salt_plan* plan, const void* x, void* y, void* stream) {
  return apply_impl(ctx, 1, &table, plan, &x, &y, (hipStream_t)stream, nullptr);
}

salt_status salt_apply_batch(salt_ctx* ctx, int32_t n, const int32_t* tables, salt_plan* plan, const void* const* xs,
                             void* const* ys, void* stream) {
  return apply_impl(ctx, n, tables, plan, xs, ys, (hipStream_t)stream, nullptr);
}

salt_status salt_apply_batch_noalloc(salt_ctx* ctx, int32_t n, const int32_t* tables, salt_plan* plan,
                                     const void* const* xs, void* const* ys, void* stream) {
  return apply_impl(ctx, n, tables, plan, xs, ys, (hipStream_t)stream, nullptr, true);
}

salt_status salt_apply_batch_timed(salt_ctx* ctx, int32_t n, const int32_t* tables, salt_plan* plan,
                                   const void* const* xs, void* const* ys, void* stream, void* const* events) {
  if (!events || !events[0] || !events[1] || !events[2] || !events[3])
    return fail(ctx, SALT_ERR_INVALID_ARG, "null event");
  hipEvent_t ev[4] = {(hipEvent_t)events[0], (hipEvent_t)events[1], (hipEvent_t)events[2], (hipEvent_t)events[3]};
  return apply_impl(ctx, n, tables, plan, xs, ys, (hipStream_t)stream, ev);
}

salt_status salt_apply_map(salt_ctx* ctx, int32_t table, int32_t T, const int32_t* tok_c, const int32_t* tok_u,
                           const float* tok_gamma, const void* x, void* y, void* stream) {
  SALT_LIVE(ctx);
  if (table < 0 || table >= ctx->cfg.n_tables)
    return fail(ctx, SALT_ERR_OUT_OF_RANGE, "table %d not in [0, %d)", table, ctx->cfg.n_tables);
  if (!ctx->map_plan) {
    salt_plan* p = nullptr;
    SALT_HIP(ctx, hipSetDevice(ctx->device));
    const salt_status st = plan_create(ctx, &p);
    if (st != SALT_OK) return st;
    ctx->map_plan = p;
  }
  const hipStream_t s = (hipStream_t)stream;
  salt_status st = set_maps_impl(ctx, ctx->map_plan, T, tok_c, tok_u, tok_gamma, s);
  if (st != SALT_OK) return st;
  st = build_impl(ctx, ctx->map_plan, s);
  if (st != SALT_OK) return st;
  return apply_impl(ctx, 1, &table, ctx->map_plan, &x, &y, s, nullptr);
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

salt_status salt_route(int32_t K, const double* n_k, const double* mu_n, const double* sigma_n, const double* mu_r,
                       const double* sigma_r, double tau_n, double tau_r, double* z_n, double* z_r,
                       salt_route_result* out) {
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
  SALT_LIVE(ctx);
  if (!out) return SALT_ERR_INVALID_ARG;
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
  // one scratch buffer per context: table records, then the Grams, then the
  // results (each region 256-byte aligned); it grows to the largest call so far
  auto up = [](size_t n) { return (n + 255) / 256 * 256; };
  const size_t tabs_bytes = up(sizeof(salt::GramTable) * nt), g_bytes = up(sizeof(float) * a.g_table * nt);
  const size_t need = tabs_bytes + g_bytes + sizeof(double) * 3 * nt;
  if (need > ctx->gram_bytes) {
    // (the previous buffer is idle: every earlier call synchronised its stream)
    if (ctx->gram) (void)hipFree(ctx->gram);
    ctx->gram = nullptr;
    ctx->gram_bytes = 0;
    if (hipMalloc((void**)&ctx->gram, need) != hipSuccess) {
      (void)hipGetLastError();
      ctx->gram = nullptr;
      return fail(ctx, SALT_ERR_OUT_OF_MEMORY, "adapter Gram scratch (%zu bytes)", need);
    }
    ctx->gram_bytes = need;
  }
  char* tabs_d = ctx->gram;
  a.tabs = reinterpret_cast<const salt::GramTable*>(tabs_d);
  a.g = reinterpret_cast<float*>(tabs_d + tabs_bytes);
  a.out = reinterpret_cast<double*>(tabs_d + tabs_bytes + g_bytes);
  SALT_HIP(ctx, hipMemcpyAsync(tabs_d, tabs.data(), sizeof(salt::GramTable) * nt, hipMemcpyHostToDevice, s));
  SALT_HIP(ctx, hipMemsetAsync(a.g, 0, sizeof(float) * a.g_table * nt, s));
  SALT_HIP(ctx, salt::launch_gram(a, max_in, max_out, ctx->cfg.dtype == SALT_BF16, s));
  SALT_HIP(ctx, hipMemcpyAsync(out, a.out, sizeof(double) * 3 * nt, hipMemcpyDeviceToHost, s));
  SALT_HIP(ctx, hipStreamSynchronize(s));
  return SALT_OK;
}

}  // extern "C"
