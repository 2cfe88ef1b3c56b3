// Drives a host build of libsalt through its C ABI (include/salt.h) on the
// inputs in argv[1] and writes what it returns to argv[2].
//
// Input (little-endian int32 unless stated):
//   magic 0x53414c54, dtype, n_tables, C, r_c, n_slots, r_u_max, max_tokens, n_cu
//   shapes [n_tables][2]
//   per table (C > 0): At bytes [C][r_c][in], B bytes [C][r_c][out]
//   n_loads, then per load: slot, rank, blob bytes (rank * sum(in + out) * esize)
//   n_batches, then per batch:
//     mode (0: set_maps + build + apply_batch on the context's plan 0 .. n_plans-1;
//           1: salt_apply_map, one table; 2: as 0 with salt_apply_batch_noalloc),
//     plan index,
//     T, has_gamma, tok_c [T], tok_u [T], gamma (float32) [T] if has_gamma,
//     n_jobs, tables [n_jobs], then per job x bytes [T][in], y0 bytes [T][out]
// Output per batch: status of set_maps, build, apply, plan_errors; n_errors,
//   n_seg, n_grp, tile tokens, n_tiles; perm [T], seg_off [n_seg + 1],
//   seg_c [n_seg], seg_u [n_seg], grp_off [n_grp + 1]; per job y bytes.
// Test infrastructure only.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "salt.h"

namespace {
FILE* in_f;
FILE* out_f;
int32_t rd() {
  int32_t v;
  if (fread(&v, 4, 1, in_f) != 1) {
    fprintf(stderr, "harness: truncated input\n");
    exit(2);
  }
  return v;
}
void rd_bytes(void* p, size_t n) {
  if (n && fread(p, 1, n, in_f) != n) {
    fprintf(stderr, "harness: truncated input\n");
    exit(2);
  }
}
void wr(int32_t v) { fwrite(&v, 4, 1, out_f); }
void wr_bytes(const void* p, size_t n) { fwrite(p, 1, n, out_f); }
}  // namespace

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: harness in out\n");
    return 2;
  }
  in_f = fopen(argv[1], "rb");
  out_f = fopen(argv[2], "wb");
  if (!in_f || !out_f) return 2;
  if (rd() != 0x53414c54) return 3;
  salt_config cfg{};
  cfg.dtype = (salt_dtype)rd();
  cfg.n_tables = rd();
  cfg.n_centroids = rd();
  cfg.r_c = rd();
  cfg.n_slots = rd();
  cfg.r_u_max = rd();
  cfg.max_tokens = rd();
  const int n_cu = rd();
  (void)n_cu;
  std::vector<salt_shape> shapes(cfg.n_tables);
  for (auto& s : shapes) {
    s.in_dim = rd();
    s.out_dim = rd();
  }
  cfg.tables = shapes.data();
  const size_t es = cfg.dtype == SALT_F32 ? 4 : 2;
  salt_ctx* ctx = nullptr;
  salt_status st = salt_create(&cfg, &ctx);
  if (st != SALT_OK) {
    fprintf(stderr, "harness: salt_create %d: %s\n", st, salt_last_error(nullptr));
    return 4;
  }
  if (cfg.n_centroids > 0) {
    for (int t = 0; t < cfg.n_tables; ++t) {
      std::vector<char> at((size_t)cfg.n_centroids * cfg.r_c * shapes[t].in_dim * es);
      std::vector<char> b((size_t)cfg.n_centroids * cfg.r_c * shapes[t].out_dim * es);
      rd_bytes(at.data(), at.size());
      rd_bytes(b.data(), b.size());
      st = salt_pin_centroids(ctx, t, 0, cfg.n_centroids, at.data(), b.data());
      if (st != SALT_OK) {
        fprintf(stderr, "harness: pin %d: %s\n", st, salt_last_error(ctx));
        return 4;
      }
    }
  }
  const int n_loads = rd();
  std::vector<void*> blobs;
  std::vector<int32_t> slots, ranks;
  std::vector<size_t> sizes;
  for (int i = 0; i < n_loads; ++i) {
    const int slot = rd(), rank = rd();
    const size_t n = salt_residual_bytes(ctx, rank);
    void* p = nullptr;
    if (n) {
      if (salt_host_alloc(n, &p) != SALT_OK) return 4;
      rd_bytes(p, n);
    }
    blobs.push_back(p);
    slots.push_back(slot);
    ranks.push_back(rank);
    sizes.push_back(n);
  }
  st = salt_load_residuals(ctx, n_loads, slots.data(), ranks.data(), blobs.data(), sizes.data());
  if (st != SALT_OK) {
    fprintf(stderr, "harness: load %d: %s\n", st, salt_last_error(ctx));
    return 4;
  }
  if (salt_wait_loads(ctx) != SALT_OK) return 4;
  std::vector<salt_plan*> plans;
  const int n_batches = rd();
  for (int bi = 0; bi < n_batches; ++bi) {
    const int mode = rd(), pi = rd();
    const int T = rd(), has_gamma = rd();
    std::vector<int32_t> tc(T), tu(T);
    std::vector<float> gm(T);
    rd_bytes(tc.data(), 4 * (size_t)T);
    rd_bytes(tu.data(), 4 * (size_t)T);
    if (has_gamma) rd_bytes(gm.data(), 4 * (size_t)T);
    const int nj = rd();
    std::vector<int32_t> tabs(nj);
    rd_bytes(tabs.data(), 4 * (size_t)nj);
    std::vector<void*> xs(nj), ys(nj);
    std::vector<size_t> ybytes(nj);
    for (int j = 0; j < nj; ++j) {
      const salt_shape s = shapes[tabs[j]];
      const size_t xb = (size_t)T * s.in_dim * es, yb = (size_t)T * s.out_dim * es;
      // device buffers: exact sizes (a host build maps them to plain allocations)
      xs[j] = malloc(xb ? xb : 16);
      ys[j] = malloc(yb ? yb : 16);
      rd_bytes(xs[j], xb);
      rd_bytes(ys[j], yb);
      ybytes[j] = yb;
    }
    salt_status s_set = SALT_OK, s_build = SALT_OK, s_apply = SALT_OK, s_err = SALT_OK;
    int32_t n_err = 0, n_seg = 0, n_grp = 0, tile_m = 0, n_tiles = 0;
    std::vector<int32_t> perm(T + 1), seg_off(T + 1), seg_c(T + 1), seg_u(T + 1), grp_off(T + 1);
    if (mode == 1) {
      s_apply = salt_apply_map(ctx, tabs[0], T, tc.data(), tu.data(), has_gamma ? gm.data() : nullptr, xs[0], ys[0],
                               nullptr);
    } else {
      while ((int)plans.size() <= pi) {
        salt_plan* p = nullptr;
        if (salt_plan_create(ctx, &p) != SALT_OK) return 4;
        plans.push_back(p);
      }
      salt_plan* p = plans[pi];
      s_set = salt_plan_set_maps(ctx, p, T, tc.data(), tu.data(), has_gamma ? gm.data() : nullptr, nullptr);
      if (s_set == SALT_OK) s_build = salt_plan_build(ctx, p, nullptr);
      if (s_set == SALT_OK && s_build == SALT_OK) {
        s_apply = mode == 2 ? salt_apply_batch_noalloc(ctx, nj, tabs.data(), p, xs.data(), ys.data(), nullptr)
                            : salt_apply_batch(ctx, nj, tabs.data(), p, xs.data(), ys.data(), nullptr);
        s_err = salt_plan_errors(ctx, p, nullptr, &n_err);
        (void)salt_plan_tiling(ctx, p, &tile_m, &n_tiles, nullptr);
        (void)salt_plan_download(ctx, p, nullptr, perm.data(), seg_off.data(), seg_c.data(), seg_u.data(),
                                 grp_off.data(), &n_seg, &n_grp);
      }
    }
    if (s_set || s_build || s_apply || s_err)
      fprintf(stderr, "harness: batch %d: %s\n", bi, salt_last_error(ctx));
    wr(s_set);
    wr(s_build);
    wr(s_apply);
    wr(s_err);
    wr(n_err);
    wr(n_seg);
    wr(n_grp);
    wr(tile_m);
    wr(n_tiles);
    wr_bytes(perm.data(), 4 * (size_t)T);
    wr_bytes(seg_off.data(), 4 * (size_t)(n_seg + 1));
    wr_bytes(seg_c.data(), 4 * (size_t)n_seg);
    wr_bytes(seg_u.data(), 4 * (size_t)n_seg);
    wr_bytes(grp_off.data(), 4 * (size_t)(n_grp + 1));
    for (int j = 0; j < nj; ++j) {
      wr_bytes(ys[j], ybytes[j]);
      free(xs[j]);
      free(ys[j]);
    }
  }
  for (salt_plan* p : plans) salt_plan_destroy(ctx, p);
  salt_destroy(ctx);
  for (void* p : blobs)
    if (p) salt_host_free(p);
  fclose(out_f);
  return 0;
}
