// Gram form of the estimator (SN_FLAG_GRAM): the Gram sweep on the matrix
// cores and the d_h-space iteration, for MI355X (gfx950, wave64).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "sweep_device.h"

namespace sn {
namespace {

// ---------------------------------------------------------------------------
// Gram form (SN_FLAG_GRAM).  With G_Q = Q_h Q_h^T and G_K = K_j K_j^T
// (d_h x d_h), one step of the iteration is
//     w = G_Q z,  sigma^2 = z^T w,  y = w / sigma,
//     t = G_K y,  ||v'||^2 = y^T t,  z_next = t / ||v'||,
// because u' = Q_h^T z has ||u'||^2 = z^T G_Q z and Q_h u' = G_Q z, and
// likewise for v' = K_j^T y.  These are the iterates of the sweeps above,
// computed in d_h-space.
//
// gram_kernel forms G = R R^T for every d_h x d row block R (query heads
// first, then key heads) on the matrix cores: an output block (bi, bj) of
// 16 x 16 is one MFMA chain whose A operand is rows 16 bi.. of R and whose B
// operand is rows 16 bj.. of R, both in the rows' native layout (lane l
// holds row l % 16 and 16 bytes of consecutive columns; the contraction
// index may be permuted freely as long as both operands share it).  Only the
// upper triangle of blocks is formed.  A wave streams its rows through LDS in
// tiles of 128-byte row segments (coalesced loads; see stage_issue) and reads
// the operands back in the MFMA layout.


template <int RB>
__host__ __device__ constexpr int tri_index(int bi, int bj) {  // bj >= bi
  return bi * RB - bi * (bi - 1) / 2 + (bj - bi);
}

template <typename T, int DH>
__global__ void __launch_bounds__(64 * kGWaves) __attribute__((amdgpu_waves_per_eu(DH >= 128 ? 2 : 4)))
gram_kernel(GramArgs args) {
  GramArgs a = args;
  if (a.ctl) {  // tail: the listed units, with the count and strips chosen on the device
    a.s_g = uni(a.ctl[TC_GRAM + 1]);
    a.tps = uni(a.ctl[TC_GRAM + 2]);
    a.n_items = uni(a.ctl[TC_GRAM]) * a.s_g;
  }
  constexpr int ES = sizeof(T);
  constexpr int RB = DH / 16;
  constexpr int NB = RB * (RB + 1) / 2;
  constexpr int TC = 128 / ES;  // columns per tile
  __shared__ __attribute__((aligned(16))) uint8_t stage[kGWaves][DH * 128];
  const int lane = threadIdx.x & 63;
  const int wv = uni((int)(threadIdx.x >> 6));
  const int q = lane >> 4, s = lane & 15;
  const int item = blockIdx.x * kGWaves + wv;
  if (item >= a.n_items) return;
  const int unit = a.list ? uni(a.list[item / a.s_g]) : item / a.s_g, strip = item % a.s_g;
  int layer, row0, tab;
  if (unit < a.H) {
    layer = unit / a.n_q;
    row0 = (unit % a.n_q) * DH;
    tab = layer;
  } else {
    layer = (unit - a.H) / a.n_kv;
    row0 = ((unit - a.H) % a.n_kv) * DH;
    tab = a.L + layer;
  }
  const char* blk = uni(a.mats[tab]) + (int64_t)row0 * a.ld * ES;
  const uint32_t nrec = (uint32_t)((((int64_t)(DH - 1) * a.ld + a.d) * ES + 15) & ~int64_t(15));
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(blk), (short)0, (int)nrec, kRsrcWord3);
  const uint32_t row_bytes = (uint32_t)(a.ld * ES);
  uint8_t* tile = stage[wv];

  f32x4 acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int n_full = a.d / TC;
  const int t0 = strip * a.tps;
  const int t1 = min(t0 + a.tps, a.n_tiles);

  // one LDS tile per wave: the next tile streams in while this one is
  // multiplied from registers.  Each wave starts at its own pseudo-random
  // tile of the strip and wraps around, so that side-by-side waves read
  // different column offsets of their strided rows.
  const int n_mine = t1 - t0;
  const int rot = n_mine > 1 ? (int)((((uint32_t)item * 2654435761u) >> 16) % (uint32_t)n_mine) : 0;
  auto tile_at = [&](int i) { const int u = rot + i; return t0 + (u >= n_mine ? u - n_mine : u); };
  if (n_mine > 0) stage_issue<DH, kStreamPolicy>(rsrc, tile, (uint32_t)(tile_at(0) * 128), row_bytes, lane);
#pragma unroll 1
  for (int i = 0; i < n_mine; ++i) {
    const int t = tile_at(i);
    __builtin_amdgcn_s_waitcnt(0);  // the tile is in LDS
    u32x4 fr[RB][2];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) fr[rb][kc] = stage_chunk(tile, 16 * rb + s, 4 * kc + q);
    __builtin_amdgcn_s_waitcnt(0);  // read out before the next tile overwrites it
    if (i + 1 < n_mine) stage_issue<DH, kStreamPolicy>(rsrc, tile, (uint32_t)(tile_at(i + 1) * 128), row_bytes, lane);
    if (t >= n_full) {  // the ragged last tile: zero columns >= d
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) {
        const int nval = a.d - (t * TC + (64 * kc + 16 * q) / ES);
        u32x4 m;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (ES == 2)
            m[e] = (2 * e < nval ? 0x0000ffffu : 0u) | (2 * e + 1 < nval ? 0xffff0000u : 0u);
          else
            m[e] = e < nval ? 0xffffffffu : 0u;
        }
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) fr[rb][kc] &= m;
      }
    }
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int bi = 0; bi < RB; ++bi)
#pragma unroll
        for (int bj = bi; bj < RB; ++bj) {
          f32x4& c = acc[tri_index<RB>(bi, bj)];
          if constexpr (ES == 2) {
            c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, fr[bi][kc]),
                                                        __builtin_bit_cast(bf16x8, fr[bj][kc]), c, 0, 0, 0);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(fr[bi][kc][e]),
                                                       __uint_as_float(fr[bj][kc][e]), c, 0, 0, 0);
          }
        }
  }
  f32x4* out = reinterpret_cast<f32x4*>(a.gp) + ((size_t)item * NB) * 64 + lane;
#pragma unroll
  for (int b = 0; b < NB; ++b) out[(size_t)b * 64] = acc[b];
}

// d_h-space iteration of the Gram form: one workgroup of NT threads per query
// head.  Thread t = 16 R + C owns rows RPT R .. RPT R + RPT - 1 and columns
// CPT C .. CPT C + CPT - 1 (CPT = d_h / 16) of G_Q and of G_K in registers.
// A product G x reads CPT entries of x from LDS and sums the partial rows
// over the 16 lanes C = 0..15 of a DPP row with a butterfly (quad xor 1,
// xor 2, half-row mirror, row mirror) that leaves the same bits in every
// lane.  Norms are summed in a fixed order, and every thread takes the same
// per-head decisions from the same values.

template <int DH>
struct IterShape {
  static constexpr int RPT = DH >= 32 ? DH / 32 : 1;  // rows per thread
  static constexpr int CPT = DH / 16;                 // columns per thread
  static constexpr int NT = 16 * DH / RPT;            // threads per workgroup
  static constexpr int NW = NT / 64;                  // waves per workgroup
  static constexpr int RB = DH / 16, NB = RB * (RB + 1) / 2;
};

template <int CTRL>
__device__ __forceinline__ float dpp_add(float x) {
  return x + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over the 16 lanes of a DPP row; every lane of the row gets the same bits.
__device__ __forceinline__ float row16_sum(float x) {
  x = dpp_add<0xB1>(x);   // quad_perm [1, 0, 3, 2]
  x = dpp_add<0x4E>(x);   // quad_perm [2, 3, 0, 1]
  x = dpp_add<0x141>(x);  // row_half_mirror: quad 0 <-> 1, 2 <-> 3
  x = dpp_add<0x140>(x);  // row_mirror: half 0 <-> half 1
  return x;
}

// Sum of the values of lanes 0, 16, 32, 48 (the C == 0 lanes), in that order.
__device__ __forceinline__ float c0_lanes_sum(float x) {
  const int b = __builtin_bit_cast(int, x);
  return (__builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 0)) +
          __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 16))) +
         (__builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 32)) +
          __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 48)));
}


// Sums the strips of one Gram matrix (upper-triangle 16 x 16 blocks in the
// MFMA output layout), writes the whole symmetric matrix to LDS and hands
// each thread its RPT x CPT sub-block.
template <int DH>
__device__ __forceinline__ void gram_to_regs(const float* src, int s_g, float* gl,
                                             float (&reg)[IterShape<DH>::RPT][IterShape<DH>::CPT]) {
  using S = IterShape<DH>;
  constexpr int P = DH + 1, NE = S::NB * 256, NL = (NE + S::NT - 1) / S::NT;
  const int t = threadIdx.x;
  float x[NL];  // flat elements t, t + NT, ... of the blocks, summed over the strips
#pragma unroll
  for (int m = 0; m < NL; ++m) x[m] = (m * S::NT + t < NE) ? src[m * S::NT + t] : 0.f;
  for (int st = 1; st < s_g; ++st) {
#pragma unroll
    for (int m = 0; m < NL; ++m)
      if (m * S::NT + t < NE) x[m] += src[(size_t)st * NE + m * S::NT + t];
  }
#pragma unroll
  for (int m = 0; m < NL; ++m) {
    const int f = m * S::NT + t;
    if (f >= NE) continue;
    const int b = f >> 8, ln = (f & 255) >> 2, e = f & 3;  // block, lane and element in the MFMA layout
    int bi = 0, start = 0;
    while (b >= start + (S::RB - bi)) {  // upper-triangle block b -> (bi, bj)
      start += S::RB - bi;
      ++bi;
    }
    const int bj = bi + (b - start);
    const int r = 16 * bi + 4 * (ln >> 4) + e, c = 16 * bj + (ln & 15);
    gl[r * P + c] = x[m];
    if (bi != bj) gl[c * P + r] = x[m];
  }
  __syncthreads();
  const int R = t >> 4, C = t & 15;
#pragma unroll
  for (int i = 0; i < S::RPT; ++i)
#pragma unroll
    for (int j = 0; j < S::CPT; ++j) reg[i][j] = gl[(S::RPT * R + i) * P + S::CPT * C + j];
  __syncthreads();
}

// out[i] = sum_c G[RPT R + i][c] x[c], complete in every lane of the row.
template <int RPT, int CPT>
__device__ __forceinline__ void gram_matvec(const float (&g)[RPT][CPT], const float* x, int C, float (&out)[RPT]) {
  float xv[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) xv[j] = x[CPT * C + j];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < CPT; ++j) acc = fmaf(g[i][j], xv[j], acc);
    out[i] = row16_sum(acc);
  }
}

template <int DH>
__global__ void __launch_bounds__(IterShape<DH>::NT) gram_iterate_kernel(IterArgs a) {
  using S = IterShape<DH>;
  constexpr int RPT = S::RPT, CPT = S::CPT, NW = S::NW;
  __shared__ float gl[DH * (DH + 1)];
  __shared__ float wb[DH], tb[DH];
  __shared__ float red_a[NW], red_b[NW];
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int R = t >> 4, C = t & 15;
  // the head, and the Gram items of its query and key matrices
  int h = blockIdx.x, s_g = a.s_g;
  if (a.list) {
    const int nq = uni(a.ctl[TC_NQ]);
    if ((int)blockIdx.x >= nq) return;
    h = uni(a.list[blockIdx.x]);
    s_g = uni(a.ctl[TC_GRAM + 1]);
  }
  const int layer = h / a.n_q;
  const int j = layer * a.n_kv + (h % a.n_q) / a.g;
  const int item_q = a.list ? (int)blockIdx.x : h;
  const int item_k = a.list ? uni(a.ctl[TC_NQ]) + uni(a.kvpos[j]) : a.H + j;

  // z of step k0 + 1: K_j v' / ||v'|| from the partials of the W_K sweep of
  // step k0 (slot k0 & 1; at k0 = 0 the first sweep, v' = the start vector)
  const int slot = a.k0 & 1;
  float nv2 = 0.f;
  for (int st = 0; st < a.s_k; ++st) nv2 += a.w.zn[((size_t)slot * a.H + h) * a.s_k + st];
  if (a.k0 == 0) {
    if (t == 0) a.w.vnorm0[h] = sqrtf(nv2);
    if (!(nv2 > 0.f) || !isfinite(nv2)) {
      if (t == 0) {
        a.sigma[h] = __builtin_nanf("");
        a.iters[h] = -1;
      }
      return;
    }
  }
  const float inv0 = 1.0f / sqrtf(nv2);
  if (t < DH) {
    float z = 0.f;
    for (int st = 0; st < a.s_k; ++st) z += a.w.zp[(((size_t)slot * a.H + h) * a.s_k + st) * DH + t];
    tb[t] = z * inv0;
  }
  float gq[RPT][CPT], gk[RPT][CPT];
  gram_to_regs<DH>(a.gp + (size_t)item_q * s_g * S::NB * 256, s_g, gl, gq);
  gram_to_regs<DH>(a.gp + (size_t)item_k * s_g * S::NB * 256, s_g, gl, gk);

  float zscale = 1.f, prev = a.k0 > 0 ? a.w.sig[(size_t)slot * a.H + h] : 0.f;
  float out[RPT];
#pragma unroll 1
  for (int k = a.k0 + 1;; ++k) {
    // w = G_Q z with z = zscale * tb; lane C == 0 of row band R owns rows RPT R ..
    gram_matvec<RPT, CPT>(gq, tb, C, out);
    float part = 0.f;
    if (C == 0) {
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        const float wr = out[i] * zscale;
        part = fmaf(tb[RPT * R + i] * zscale, wr, part);
        wb[RPT * R + i] = wr;
      }
    }
    part = c0_lanes_sum(part);
    if (lane == 0) red_a[wv] = part;
    __syncthreads();
    const float s2 = sum_waves<NW>(red_a);
    const float sig = sqrtf(s2);
    if (s2 == 0.f) {  // M v = 0
      if (t == 0) {
        a.sigma[h] = 0.f;
        a.iters[h] = -2;
      }
      return;
    }
    const bool last = (k >= a.n_iter) || (a.tol > 0.f && k >= 2 && fabsf(sig - prev) <= a.tol * sig);
    const float inv = 1.0f / sig;
    if (last) {
      if (t < DH) {
        a.w.fin[(size_t)h * 2 * DH + t] = tb[t] * zscale;     // z of the last step
        a.w.fin[(size_t)h * 2 * DH + DH + t] = wb[t] * inv;   // y = Q_h u
      }
      if (t == 0) {
        a.sigma[h] = sig;
        a.iters[h] = k;
      }
      return;
    }
    // t = G_K y with y = w / sigma
    gram_matvec<RPT, CPT>(gk, wb, C, out);
    float part2 = 0.f;
    if (C == 0) {
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        const float tr = out[i] * inv;
        part2 = fmaf(wb[RPT * R + i] * inv, tr, part2);
        tb[RPT * R + i] = tr;
      }
    }
    part2 = c0_lanes_sum(part2);
    if (lane == 0) red_b[wv] = part2;
    __syncthreads();
    const float n2 = sum_waves<NW>(red_b);
    zscale = 1.0f / sqrtf(n2);
    prev = sig;
  }
}

template <typename T>
void gram_dispatch(int dh, dim3 grid, hipStream_t st, const GramArgs& g) {
  switch (dh) {
    case 16: gram_kernel<T, 16><<<grid, 64 * kGWaves, 0, st>>>(g); break;
    case 32: gram_kernel<T, 32><<<grid, 64 * kGWaves, 0, st>>>(g); break;
    case 64: gram_kernel<T, 64><<<grid, 64 * kGWaves, 0, st>>>(g); break;
    default: gram_kernel<T, 128><<<grid, 64 * kGWaves, 0, st>>>(g); break;
  }
}

}  // namespace

void launch_gram(bool bf16, int head_dim, int n_items, hipStream_t st, const GramArgs& g) {
  const dim3 grid((n_items + kGWaves - 1) / kGWaves);
  if (bf16)
    gram_dispatch<uint16_t>(head_dim, grid, st, g);
  else
    gram_dispatch<float>(head_dim, grid, st, g);
}

void launch_gram_iterate(int head_dim, int heads, hipStream_t st, const IterArgs& it) {
  switch (head_dim) {
    case 16: gram_iterate_kernel<16><<<dim3(heads), IterShape<16>::NT, 0, st>>>(it); break;
    case 32: gram_iterate_kernel<32><<<dim3(heads), IterShape<32>::NT, 0, st>>>(it); break;
    case 64: gram_iterate_kernel<64><<<dim3(heads), IterShape<64>::NT, 0, st>>>(it); break;
    default: gram_iterate_kernel<128><<<dim3(heads), IterShape<128>::NT, 0, st>>>(it); break;
  }
}

}  // namespace sn
