// Two analysis / start-up paths of libsalt on gfx950 (MI355X), beside the apply:
//   k_fuse:  a pinned centroid folded into a base weight, W <- rne(W + gamma A_c B_c)
//            (Sec. 3.3: a node serving a high-frequency domain fuses its centroid
//            at start-up and then applies residuals only).
//   k_gram:  the r x r Gram products of two low-rank updates, from which Eq. 2's
//            alignment penalty (the matrix cosine of Sec. 3.1 / Sec. 4.5) follows
//            without forming the in x out updates.
#include <hip/hip_ext.h>

#include <algorithm>

#include "salt_device.h"
#include "salt_internal.h"

namespace salt {
namespace {

// A launch; with events, they record the kernel's own start and end.
template <typename K, typename Args>
void launch_k(K kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s, const Args& a, hipEvent_t e0,
              hipEvent_t e1) {
  if (e0 || e1) hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, s, e0, e1, 0u, a);
  else hipLaunchKernelGGL(kernel, grid, block, lds, s, a);
}
// ---------------------------------------------------------------------------
// centroid fused into a base weight
// ---------------------------------------------------------------------------
// Raw elements of an operand vector (8 per lane).
__device__ __forceinline__ void vec_elems(const uint4& v, uint16_t (&e)[8]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int k = 0; k < 8; ++k) e[k] = (uint16_t)(w[k >> 1] >> (16 * (k & 1)));
}
__device__ __forceinline__ void vec_elems(const Ops<float>::Vec& v, float (&e)[8]) {
  e[0] = v.lo.x; e[1] = v.lo.y; e[2] = v.lo.z; e[3] = v.lo.w;
  e[4] = v.hi.x; e[5] = v.hi.y; e[6] = v.hi.z; e[7] = v.hi.w;
}

constexpr int kFuseTI = 64, kFuseTO = 128, kFuseDS = kFuseTO + 4;
// Row stride (elements) of the transposed A_c tile: 32 * KS ranks + 8 of padding.
__host__ __device__ constexpr int fuse_rp(int ks) { return 32 * ks + 8; }
size_t fuse_lds(int ks, int esize) {
  return std::max((size_t)kFuseTI * fuse_rp(ks) * esize, sizeof(float) * kFuseTI * kFuseDS);
}

// W[i][o] <- rne(W[i][o] + gamma * sum_r A_c[i][r] B_c[r][o]) over a 64 x 128
// tile of W (in rows i, out columns o).  The rank-r_c product is an MFMA
// contraction over the ranks: D[o][i] = sum_r Bt_c[o][r] At_c[r][i], with the
// rows of Bt_c (8 consecutive ranks per lane) read straight from the pinned
// transposed B and At_c's columns taken from an LDS copy of the tile transposed
// to [i][r].  The fp32 delta goes through LDS so that W is read and written in
// whole rows, once, with one rounding.
template <typename E, int KS>
__global__ void __launch_bounds__(256) k_fuse(FuseArgs f) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  constexpr int TI = kFuseTI, TO = kFuseTO, DS = kFuseDS, RP = fuse_rp(KS);
  extern __shared__ __attribute__((aligned(16))) char lds[];
  E* s_a = reinterpret_cast<E*>(lds);            // [TI][RP]: A_c[i][r], ranks past r_c zero
  float* s_d = reinterpret_cast<float*>(lds);    // [TI][DS] delta, after s_a is consumed
  const int i0 = blockIdx.x * TI, o0 = blockIdx.y * TO;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4;
  const int in = f.in_dim, out = f.out_dim, rc = f.r_c;
  const E* at = reinterpret_cast<const E*>(f.at);   // [r_c][in] of the centroid
  const E* bt = reinterpret_cast<const E*>(f.bt);   // [out][r_c]

  for (int k = tid; k < 32 * KS * (TI / 8); k += 256) {
    const int r = k / (TI / 8), i8 = (k % (TI / 8)) * 8;
    E e[8];
    if (r < rc && i0 + i8 < in) {
      vec_elems(O::load(at + (size_t)r * in + i0 + i8), e);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) e[q] = E(0);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) s_a[(i8 + q) * RP + r] = e[q];
  }
  __syncthreads();

  f32x4 acc[2][4];
#pragma unroll
  for (int ob = 0; ob < 2; ++ob)
#pragma unroll
    for (int ib = 0; ib < 4; ++ib) acc[ob][ib] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int r8 = 32 * ks + 8 * g;               // this lane's 8 ranks (r_c is a multiple of 8)
    Vec bfr[2];
#pragma unroll
    for (int ob = 0; ob < 2; ++ob) {
      const int o = o0 + 32 * wave + 16 * ob + (lane & 15);
      bfr[ob] = (o < out && r8 < rc) ? O::load(bt + (size_t)o * rc + r8) : O::zero();
    }
#pragma unroll
    for (int ib = 0; ib < 4; ++ib) {
      const Vec afr = *reinterpret_cast<const Vec*>(s_a + (16 * ib + (lane & 15)) * RP + r8);
#pragma unroll
      for (int ob = 0; ob < 2; ++ob) acc[ob][ib] = O::mma(bfr[ob], afr, acc[ob][ib]);
    }
  }
  __syncthreads();                                // s_a consumed; s_d reuses it
  // D[o][i]: lane holds o = 4g + e (of its 16-row block), i = lane & 15
#pragma unroll
  for (int ob = 0; ob < 2; ++ob)
#pragma unroll
    for (int ib = 0; ib < 4; ++ib)
      *reinterpret_cast<float4*>(s_d + (16 * ib + (lane & 15)) * DS + 32 * wave + 16 * ob + 4 * g) =
          make_float4(acc[ob][ib][0], acc[ob][ib][1], acc[ob][ib][2], acc[ob][ib][3]);
  __syncthreads();

  for (int k = tid; k < TI * (TO / 8); k += 256) {
    const int i = k / (TO / 8), o8 = (k % (TO / 8)) * 8;
    if (i0 + i >= in || o0 + o8 >= out) continue;
    E* w = reinterpret_cast<E*>(f.w) + (size_t)(i0 + i) * f.ldw + o0 + o8;
    float v[8];
    O::to_f32(O::load(w), v);
    const float4 d0 = *reinterpret_cast<const float4*>(s_d + i * DS + o8);
    const float4 d1 = *reinterpret_cast<const float4*>(s_d + i * DS + o8 + 4);
    v[0] += f.gamma * d0.x; v[1] += f.gamma * d0.y; v[2] += f.gamma * d0.z; v[3] += f.gamma * d0.w;
    v[4] += f.gamma * d1.x; v[5] += f.gamma * d1.y; v[6] += f.gamma * d1.z; v[7] += f.gamma * d1.w;
    O::store(w, v);
  }
}

// ---------------------------------------------------------------------------
// adapter Gram products (matrix cosine in factor space)
// ---------------------------------------------------------------------------
// One block per work item: table t = blockIdx.y, factor side (0: the At
// factors, contracted over in; 1: the B factors, contracted over out), K chunk
// q of kGramKC elements (blockIdx.x over both sides; blocks past the table's
// chunks return at once).  The block adds the chunk's part of the three Gram
// matrices X1 X2^T, X1 X1^T and X2 X2^T (X = the side's [r][K] factors, rows
// padded to 16 with zeros) into g with fp32 atomics.  Each 16 x 16 tile is an
// MFMA contraction over K: both operands are 16 rank rows with 8 consecutive k
// per lane.  With both ranks <= 16 * NB (NB = 1, 2) every wave takes a quarter
// of the chunk's 32-wide steps for all tiles, loading each rank block's
// fragment once per step, and the four waves' tiles are summed in LDS before
// the atomics; otherwise (NB = 0) the waves split the tiles.
constexpr int kGramKC = 2048;

template <int NB>
__host__ __device__ constexpr int gram_lds() { return NB > 0 ? 4 * 3 * NB * NB * 256 * 4 : 0; }

template <typename E, int NB>
__global__ void __launch_bounds__(256) k_gram(GramArgs a) {
  using O = Ops<E>;
  using Vec = typename O::Vec;
  const int t = blockIdx.y, local = blockIdx.x;
  const GramTable tab = a.tabs[t];
  const int nq_in = (tab.in_dim + kGramKC - 1) / kGramKC, nq_out = (tab.out_dim + kGramKC - 1) / kGramKC;
  if (local >= nq_in + nq_out) return;
  const int side = local < nq_in ? 0 : 1;
  const int q = side == 0 ? local : local - nq_in;
  const int K = side == 0 ? tab.in_dim : tab.out_dim;
  const int k0 = q * kGramKC, kend = min(K, k0 + kGramKC);
  const E* x1 = reinterpret_cast<const E*>(side == 0 ? tab.at1 : tab.b1);
  const E* x2 = reinterpret_cast<const E*>(side == 0 ? tab.at2 : tab.b2);
  const int r1 = a.r1, r2 = a.r2, nb1 = (r1 + 15) / 16, nb2 = (r2 + 15) / 16;
  float* g = a.g + (size_t)t * a.g_table + (size_t)side * a.g_side;
  // tiles: [0, nb1 * nb2) of G12, then nb1 * nb1 of G11, then nb2 * nb2 of G22
  const int n12 = nb1 * nb2, n11 = nb1 * nb1, ntile = n12 + n11 + nb2 * nb2;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g8 = lane >> 4;
  // where tile `tile` goes: its Gram, its rank blocks, the Gram's row length
  auto place = [&](int tile, float*& gt, int& ba, int& bb, int& ldg) {
    if (tile < n12) {
      ba = tile / nb2; bb = tile % nb2; ldg = nb2 * 16; gt = g;
    } else if (tile < n12 + n11) {
      const int u = tile - n12;
      ba = u / nb1; bb = u % nb1; ldg = nb1 * 16; gt = g + a.g_12;
    } else {
      const int u = tile - n12 - n11;
      ba = u / nb2; bb = u % nb2; ldg = nb2 * 16; gt = g + a.g_12 + a.g_11;
    }
  };
  if constexpr (NB > 0) {
    constexpr int NT = 3 * NB * NB;
    extern __shared__ __attribute__((aligned(16))) char lds[];
    float* s_red = reinterpret_cast<float*>(lds);   // [4 waves][NT][256]
    f32x4 acc[NT];
#pragma unroll
    for (int u = 0; u < NT; ++u) acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int k = k0 + 32 * wave; k < kend; k += 128) {
      const int kk = k + 8 * g8;                     // K is a multiple of 8: a lane's 8 are all in or all out
      const bool kin = kk < kend;
      Vec f1[NB], f2[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int i1 = b * 16 + (lane & 15);
        f1[b] = (kin && i1 < r1) ? O::load(x1 + (size_t)i1 * K + kk) : O::zero();
        f2[b] = (kin && i1 < r2) ? O::load(x2 + (size_t)i1 * K + kk) : O::zero();
      }
#pragma unroll
      for (int b1 = 0; b1 < NB; ++b1)
#pragma unroll
        for (int b2 = 0; b2 < NB; ++b2) {
          acc[b1 * NB + b2] = O::mma(f1[b1], f2[b2], acc[b1 * NB + b2]);
          acc[NB * NB + b1 * NB + b2] = O::mma(f1[b1], f1[b2], acc[NB * NB + b1 * NB + b2]);
          acc[2 * NB * NB + b1 * NB + b2] = O::mma(f2[b1], f2[b2], acc[2 * NB * NB + b1 * NB + b2]);
        }
    }
    // lane holds rows 4 g8 + e, column lane & 15 of each tile
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) s_red[((size_t)wave * NT + u) * 256 + (4 * g8 + e) * 16 + (lane & 15)] = acc[u][e];
    __syncthreads();
    for (int i = threadIdx.x; i < NT * 256; i += 256) {
      const int u = i / 256, rc16 = i % 256;
      const int gram = u / (NB * NB), b1 = (u % (NB * NB)) / NB, b2 = u % NB;
      const int na = gram == 2 ? nb2 : nb1, nbb = gram == 0 ? nb2 : (gram == 1 ? nb1 : nb2);
      if (b1 >= na || b2 >= nbb) continue;                 // rank blocks this call does not have
      const int tile = gram == 0 ? b1 * nb2 + b2 : (gram == 1 ? n12 + b1 * nb1 + b2 : n12 + n11 + b1 * nb2 + b2);
      float* gt;
      int ba, bb, ldg;
      place(tile, gt, ba, bb, ldg);
      const float v = s_red[(size_t)u * 256 + rc16] + s_red[((size_t)NT + u) * 256 + rc16] +
                      s_red[((size_t)2 * NT + u) * 256 + rc16] + s_red[((size_t)3 * NT + u) * 256 + rc16];
      atomicAdd(gt + (size_t)(ba * 16 + rc16 / 16) * ldg + bb * 16 + rc16 % 16, v);
    }
  } else {
    for (int tile = wave; tile < ntile; tile += 4) {
      float* gt;
      int ba, bb, ldg;
      place(tile, gt, ba, bb, ldg);
      const E* xa = tile < n12 + n11 ? x1 : x2;
      const E* xb = tile < n12 ? x2 : (tile < n12 + n11 ? x1 : x2);
      const int ra = tile < n12 + n11 ? r1 : r2;
      const int rb = tile < n12 ? r2 : (tile < n12 + n11 ? r1 : r2);
      const int ia = ba * 16 + (lane & 15), ib = bb * 16 + (lane & 15);
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int k = k0; k < kend; k += 32) {
        const int kk = k + 8 * g8;
        const bool kin = kk < kend;
        const Vec va = (kin && ia < ra) ? O::load(xa + (size_t)ia * K + kk) : O::zero();
        const Vec vb = (kin && ib < rb) ? O::load(xb + (size_t)ib * K + kk) : O::zero();
        acc = O::mma(va, vb, acc);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) atomicAdd(gt + (size_t)(ba * 16 + 4 * g8 + e) * ldg + ib, acc[e]);
    }
  }
}

// Per table: sum of the elementwise products of the At-side and B-side Grams,
// in float64: Tr(dW1^T dW2), ||dW1||_F^2, ||dW2||_F^2.
__global__ void __launch_bounds__(256) k_gram_finish(GramArgs a) {
  const int t = blockIdx.x;
  const float* gA = a.g + (size_t)t * a.g_table;
  const float* gB = gA + a.g_side;
  const int sizes[3] = {a.g_12, a.g_11, a.g_22};
  const int offs[3] = {0, a.g_12, a.g_12 + a.g_11};
  __shared__ double s_red[3][4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int m = 0; m < 3; ++m) {
    double acc = 0.0;
    for (int i = threadIdx.x; i < sizes[m]; i += 256) acc += (double)gA[offs[m] + i] * (double)gB[offs[m] + i];
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_down(acc, off);
    if (lane == 0) s_red[m][wave] = acc;
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    const int m = threadIdx.x;
    a.out[3 * t + m] = s_red[m][0] + s_red[m][1] + s_red[m][2] + s_red[m][3];
  }
}

template <typename E>
hipError_t launch_gram_t(const GramArgs& a, int max_items, hipStream_t s) {
  const dim3 grid(max_items, a.n_tables), block(256);
  const int r = a.r1 > a.r2 ? a.r1 : a.r2;
  if (r <= 16) hipLaunchKernelGGL((k_gram<E, 1>), grid, block, gram_lds<1>(), s, a);
  else if (r <= 32) hipLaunchKernelGGL((k_gram<E, 2>), grid, block, gram_lds<2>(), s, a);
  else hipLaunchKernelGGL((k_gram<E, 0>), grid, block, 0, s, a);
  hipLaunchKernelGGL(k_gram_finish, dim3(a.n_tables), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename E>
hipError_t launch_fuse_t(const FuseArgs& f, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid((f.in_dim + kFuseTI - 1) / kFuseTI, (f.out_dim + kFuseTO - 1) / kFuseTO), block(256);
  const int ks = (f.r_c + 31) / 32;
  const size_t lds = fuse_lds(ks, (int)sizeof(E));
  switch (ks) {
    case 1: launch_k(k_fuse<E, 1>, grid, block, lds, s, f, e0, e1); break;
    case 2: launch_k(k_fuse<E, 2>, grid, block, lds, s, f, e0, e1); break;
    case 3: launch_k(k_fuse<E, 3>, grid, block, lds, s, f, e0, e1); break;
    case 4: launch_k(k_fuse<E, 4>, grid, block, lds, s, f, e0, e1); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_fuse(const FuseArgs& f, int bf16, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (f.r_c < 8 || f.r_c > kMaxRc || f.r_c % 8 || f.in_dim <= 0 || f.out_dim <= 0) return hipErrorInvalidValue;
  return bf16 ? launch_fuse_t<uint16_t>(f, s, e0, e1) : launch_fuse_t<float>(f, s, e0, e1);
}

hipError_t launch_gram(const GramArgs& a, int max_in, int max_out, int bf16, hipStream_t s) {
  if (a.n_tables < 1 || a.n_tables > 65535 || a.r1 < 1 || a.r2 < 1 || max_in < 8 || max_out < 8)
    return hipErrorInvalidValue;
  const int items = (max_in + kGramKC - 1) / kGramKC + (max_out + kGramKC - 1) / kGramKC;
  return bf16 ? launch_gram_t<uint16_t>(a, items, s) : launch_gram_t<float>(a, items, s);
}

}  // namespace salt
