// Layer-level form of the estimator (spectral_step_layer), for MI355X
// (gfx950, wave64).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "sweep_device.h"

namespace sn {
namespace {

// ---------------------------------------------------------------------------
// Layer-level form (spectral_step_layer): the estimator as printed in App. E,
// one pair u, v in R^d per layer for the concatenated W^Q = [W^Q_1 .. W^Q_nq]
// and the key blocks repeated per group (RepeatBlocks) on the way in and
// summed per group (SumGroups) on the way back.  One step is:
//   rows(W_K, v):  z_j = K_j v                       (row sums, per key head)
//   vin:           z_j(h) for every query head h     (RepeatBlocks)
//   cols(W_Q, z):  u' = sum_h Q_h^T z_j(h)           (column sums over all rows)
//   sigma = ||u'||                                   (layer_colsum / layer_norm)
//   rows(W_Q, u):  y_h = Q_h u'/sigma
//   vin:           sum_{h in group j} y_h            (SumGroups)
//   cols(W_K, y):  v' = sum_j K_j^T (sum_{h in j} y_h)
//   ||v'||                                           (layer_colsum / layer_norm)
// A column-sweep wave owns one column tile of a layer and streams it down the
// layer's row blocks (16 KB of 128-byte row segments per block, as in the
// W_Q sweep), so its column sums are final for those rows: only one d-vector
// per layer (per row split, on small shapes) is written, not one per head.
// Per-layer status: 0 running, -1 start vector zero or not finite, -2 M v = 0.


template <typename T, int DH, int MODE>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4)))
layer_sweep_kernel(LayerArgs a) {
  constexpr int VEC = Traits<T>::VEC;
  constexpr int CPL = kCPL;
  constexpr int RPL = DH / kRG;
  constexpr int TILE_C = CPL * VEC;
  constexpr int ES = sizeof(T);
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int chunk = lane % CPL, rg = lane / CPL;
  const int item = blockIdx.x * kWaves + wv;
  const bool in_range = item < a.n_items;
  // rows: (layer, unit, strip of tiles); cols: (layer, row split, tile)
  int layer, ul = 0, strip = 0, rs = 0, tile_c = 0;
  if (MODE == LM_ROWS) {
    const int unit = in_range ? item / a.s_out : 0;
    strip = in_range ? item % a.s_out : 0;
    layer = unit / a.units;
    ul = unit % a.units;
  } else {
    tile_c = in_range ? item % a.n_tiles : 0;
    const int rest = in_range ? item / a.n_tiles : 0;
    rs = rest % a.n_rsplit;
    layer = rest / a.n_rsplit;
  }
  const bool valid = in_range && uni(a.lstat[layer]) == 0;
  if (!valid) return;

  const char* base = uni(a.mats[layer]);
  const uint32_t nrec = (uint32_t)((((int64_t)(DH - 1) * a.ld + a.d) * ES + 15) & ~int64_t(15));
  auto rsrc_of = [&](int rb) {  // the d_h x ld row block rb of this layer's matrix
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base + (int64_t)rb * DH * a.ld * ES), (short)0,
                                             (int)nrec, kRsrcWord3);
  };
  const uint32_t lane_off = (uint32_t)(((int64_t)rg * RPL * a.ld + chunk * VEC) * ES);
  const uint32_t row_bytes = (uint32_t)(a.ld * ES);
  auto load_tile = [&](u32x4 (&tile)[RPL], __amdgpu_buffer_rsrc_t rsrc, int t) {
    const uint32_t voff = lane_off + (uint32_t)(t * TILE_C * ES);
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr)
      tile[rr] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff, rr * row_bytes, kStreamPolicy);
  };
  const int n_full = a.d / TILE_C;
  // zero the elements at columns >= d of the ragged last tile
  auto mask_tail = [&](u32x4 (&tile)[RPL], int t) {
    if (t < n_full) return;
    const int nval = a.d - (t * TILE_C + chunk * VEC);
    u32x4 m;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (VEC == 8)
        m[q] = (2 * q < nval ? 0x0000ffffu : 0u) | (2 * q + 1 < nval ? 0xffff0000u : 0u);
      else
        m[q] = q < nval ? 0xffffffffu : 0u;
    }
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr) tile[rr] &= m;
  };

  if (MODE == LM_ROWS) {
    const __amdgpu_buffer_rsrc_t rsrc = rsrc_of(ul);
    const float* xrow = a.xvec + (size_t)layer * a.d;
    float acc[RPL];
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr) acc[rr] = 0.f;
    const int t0 = strip * a.tps;
    const int t1 = min(t0 + a.tps, a.n_tiles);
    // staggered start tile and loads ahead of arithmetic, as in the W_Q sweep
    const int n_mine = t1 - t0;
    int t = t0;
    if (n_mine > 1) t += (int)(((uint32_t)item * 2654435761u) >> 16) % n_mine;
#pragma unroll 1
    for (int i = 0; i < n_mine; ++i, t = (t + 1 == t1) ? t0 : t + 1) {
      u32x4 tile[RPL];
      load_tile(tile, rsrc, t);
      __builtin_amdgcn_sched_barrier(0);
      mask_tail(tile, t);
      const int col = t * TILE_C + chunk * VEC;
      const int nval = a.d - col;  // >= VEC on full tiles
      float xv[VEC];
#pragma unroll
      for (int c = 0; c < VEC; ++c) xv[c] = c < nval ? xrow[min(col + c, a.d - 1)] : 0.f;
#pragma unroll
      for (int rr = 0; rr < RPL; ++rr) {
        float s = acc[rr];
#pragma unroll
        for (int c = 0; c < VEC; ++c) s = fmaf(elem<T>(tile[rr], c), xv[c], s);
        acc[rr] = s;
      }
    }
    const float xs_inv = 1.0f / sqrtf(a.xn2[layer]);
    float* op = a.rowpart + (((size_t)layer * a.units + ul) * a.s_out + strip) * DH + rg * RPL;
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr) {
      float s = acc[rr];
#pragma unroll
      for (int m = 1; m < CPL; m <<= 1) s = xor_sum(s, m);
      if ((rr % CPL) == chunk) op[rr] = s * xs_inv;
    }
  } else {
    // one column tile down row blocks rb0 .. rb1 - 1, starting at a staggered
    // block so that the waves of neighbouring tiles read different rows
    const int rb0 = rs * a.rb_per, rb1 = min(a.nrb, rb0 + a.rb_per);
    const int n_mine = rb1 - rb0;
    int rb = rb0;
    if (n_mine > 1) rb += (int)(((uint32_t)item * 2654435761u) >> 16) % n_mine;
    const float* vl = a.vin + (size_t)layer * a.nrb * DH + rg * RPL;
    float w[VEC];
#pragma unroll
    for (int c = 0; c < VEC; ++c) w[c] = 0.f;
#pragma unroll 1
    for (int i = 0; i < n_mine; ++i, rb = (rb + 1 == rb1) ? rb0 : rb + 1) {
      u32x4 tile[RPL];
      load_tile(tile, rsrc_of(rb), tile_c);
      float z[RPL];
#pragma unroll
      for (int rr = 0; rr < RPL; ++rr) z[rr] = vl[(size_t)rb * DH + rr];
      __builtin_amdgcn_sched_barrier(0);
      mask_tail(tile, tile_c);
#pragma unroll
      for (int rr = 0; rr < RPL; ++rr)
#pragma unroll
        for (int c = 0; c < VEC; ++c) w[c] = fmaf(elem<T>(tile[rr], c), z[rr], w[c]);
    }
#pragma unroll
    for (int c = 0; c < VEC; ++c) w[c] = group_sum(w[c]);
    if (rg == 0) {  // columns past d are zero (masked) and land in the row's padding
      float* out = a.colout + ((size_t)layer * a.n_rsplit + rs) * a.cstride + tile_c * TILE_C + chunk * VEC;
#pragma unroll
      for (int c = 0; c < VEC; ++c) out[c] = w[c];
    }
  }
}

// vin of a column sweep (see LayerVinArgs): block (b, l), one thread per row.
__global__ void __launch_bounds__(64) layer_vin_kernel(LayerVinArgs v) {
  const int b = blockIdx.x, l = blockIdx.y;
  if (v.lstat[l] != 0) return;
  const float* src = v.part + ((size_t)l * v.src_units + (size_t)(b / v.div) * v.cnt) * v.strips * v.dh;
  const int n = v.cnt * v.strips;  // the cnt units' partials lie back to back
  for (int r = threadIdx.x; r < v.dh; r += 64) {
    float s = 0.f;
    for (int k = 0; k < n; ++k) s += src[(size_t)k * v.dh + r];
    v.vin[((size_t)l * v.nrb + b) * v.dh + r] = s;
  }
}


// Column sums: block (b, l) owns columns b * kRedThreads .. of layer l, one
// per thread; the units are summed in order, their loads issued eight at a
// time.
__global__ void __launch_bounds__(kRedThreads) layer_colsum_kernel(LayerReduceArgs r) {
  const int b = blockIdx.x, l = blockIdx.y, t = threadIdx.x;
  __shared__ float red[kRedThreads / 64];
  if (r.mode != 0 && r.lstat[l] != 0) return;
  const int c = b * kRedThreads + t;
  float sq = 0.f;
  if (c < r.d) {
    const float* p = r.col + (size_t)l * r.units * r.cstride + c;
    float s = 0.f;
#pragma unroll 8
    for (int u = 0; u < r.units; ++u) s += p[(size_t)u * r.cstride];
    r.vec[(size_t)l * r.d + c] = s;
    sq = s * s;
  }
  sq = wave_sum(sq);
  if ((t & 63) == 0) red[t >> 6] = sq;
  __syncthreads();
  if (t == 0) r.n2part[(size_t)l * r.nb + b] = sum_waves<kRedThreads / 64>(red);
}

// n2 of each layer from its column blocks, in block order, and the status.
__global__ void __launch_bounds__(64) layer_norm_kernel(LayerReduceArgs r) {
  const int l = blockIdx.x;
  if (threadIdx.x != 0 || (r.mode != 0 && r.lstat[l] != 0)) return;
  float n2 = 0.f;
  for (int b = 0; b < r.nb; ++b) n2 += r.n2part[(size_t)l * r.nb + b];
  r.n2[l] = n2;
  if (r.mode == 0) {
    r.n2_start[l] = n2;
    r.lstat[l] = (n2 > 0.f && isfinite(n2)) ? 0 : -1;
  } else if (r.mode == 1 && n2 == 0.f) {
    r.lstat[l] = -2;
  }
}


__global__ void __launch_bounds__(kThreads) layer_finalize_kernel(LayerFinArgs f) {
  const int l = blockIdx.x;
  const int st = f.lstat[l];
  const float sig = st == -1 ? __builtin_nanf("") : st == -2 ? 0.f : sqrtf(f.n2_u[l]);
  if (threadIdx.x == 0) {
    f.sigma[l] = sig;
    f.scale[l] = f.coef * sig;
  }
  float* vp = f.v + (size_t)l * f.d;
  float* up = f.u ? f.u + (size_t)l * f.d : nullptr;
  const float vs = st == 0 ? 1.0f / sqrtf(f.n2_v[l]) : st == -2 ? 1.0f / sqrtf(f.n2_start[l]) : 1.f;
  const float us = st == 0 ? 1.0f / sig : 0.f;
  for (int c = threadIdx.x; c < f.d; c += blockDim.x) {
    if (st == 0) vp[c] = f.lv[(size_t)l * f.d + c] * vs;
    else if (st == -2) vp[c] *= vs;
    if (up) up[c] = st == 0 ? f.lu[(size_t)l * f.d + c] * us : 0.f;
  }
}

template <typename T, int MODE>
void layer_dispatch(int dh, dim3 grid, hipStream_t st, const LayerArgs& a) {
  switch (dh) {
    case 8: layer_sweep_kernel<T, 8, MODE><<<grid, kThreads, 0, st>>>(a); break;
    case 16: layer_sweep_kernel<T, 16, MODE><<<grid, kThreads, 0, st>>>(a); break;
    case 32: layer_sweep_kernel<T, 32, MODE><<<grid, kThreads, 0, st>>>(a); break;
    case 64: layer_sweep_kernel<T, 64, MODE><<<grid, kThreads, 0, st>>>(a); break;
    default: layer_sweep_kernel<T, 128, MODE><<<grid, kThreads, 0, st>>>(a); break;
  }
}

}  // namespace

void launch_layer_sweep(bool bf16, int head_dim, int mode, int n_items, hipStream_t st, const LayerArgs& a) {
  const dim3 grid((n_items + kWaves - 1) / kWaves);
  if (bf16) {
    if (mode == LM_ROWS) layer_dispatch<uint16_t, LM_ROWS>(head_dim, grid, st, a);
    else layer_dispatch<uint16_t, LM_COLS>(head_dim, grid, st, a);
  } else {
    if (mode == LM_ROWS) layer_dispatch<float, LM_ROWS>(head_dim, grid, st, a);
    else layer_dispatch<float, LM_COLS>(head_dim, grid, st, a);
  }
}

void launch_layer_vin(int layers, hipStream_t st, const LayerVinArgs& v) {
  layer_vin_kernel<<<dim3(v.nrb, layers), 64, 0, st>>>(v);
}

void launch_layer_reduce(int layers, hipStream_t st, const LayerReduceArgs& r) {
  layer_colsum_kernel<<<dim3(r.nb, layers), kRedThreads, 0, st>>>(r);
  layer_norm_kernel<<<dim3(layers), 64, 0, st>>>(r);
}

void launch_layer_finalize(int layers, hipStream_t st, const LayerFinArgs& f) {
  layer_finalize_kernel<<<dim3(layers), kThreads, 0, st>>>(f);
}

}  // namespace sn
