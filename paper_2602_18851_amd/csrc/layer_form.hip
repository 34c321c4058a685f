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
// summed per group (SumGroups) on the way back.  One step is four sweeps:
//   rows(W_K, v):  z_j = K_j v                     (row sums, per key head)
//   cols(W_Q, z):  c_h = Q_h^T z_{j(h)}            (column sums, per query head)
//   u' = sum_h c_h, sigma = ||u'||                 (layer_reduce_kernel)
//   rows(W_Q, u):  y_h = Q_h u'/sigma
//   cols(W_K, y):  c_j = K_j^T sum_{h in group j} y_h
//   v' = sum_j c_j                                 (layer_reduce_kernel)
// A column sweep item owns whole columns of its unit, so it writes its part
// of c without partials; the per-layer sum over units runs in a fixed order.
// Per-layer status: 0 running, -1 start vector zero or not finite, -2 M v = 0.


template <typename T, int DH, int MODE>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4)))
layer_sweep_kernel(LayerArgs a) {
  constexpr int VEC = Traits<T>::VEC;
  constexpr int CPL = kCPL;
  constexpr int RPL = DH / kRG;
  constexpr int TILE_C = CPL * VEC;
  constexpr int ES = sizeof(T);
  __shared__ float xs[kWaves][DH];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int chunk = lane % CPL, rg = lane / CPL;
  const int item = blockIdx.x * kWaves + wv;
  const bool in_range = item < a.n_items;
  const int unit = in_range ? item / a.s_out : 0;
  const int strip = in_range ? item % a.s_out : 0;
  const int layer = unit / a.units, ul = unit % a.units;
  const bool valid = in_range && uni(a.lstat[layer]) == 0;
  if (MODE == LM_COLS && valid) {
    const int src0 = layer * a.y_units + (ul / a.y_div) * a.y_cnt;
    for (int r = lane; r < DH; r += 64) {
      float s = 0.f;
      for (int i = 0; i < a.y_cnt; ++i)
        for (int st = 0; st < a.y_strips; ++st) s += a.ypart[((size_t)(src0 + i) * a.y_strips + st) * DH + r];
      xs[wv][r] = s;
    }
  }
  __syncthreads();
  if (!valid) return;

  const char* blk = uni(a.mats[layer]) + (int64_t)ul * DH * a.ld * ES;
  const uint32_t nrec = (uint32_t)((((int64_t)(DH - 1) * a.ld + a.d) * ES + 15) & ~int64_t(15));
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(blk), (short)0, (int)nrec, kRsrcWord3);
  const uint32_t lane_off = (uint32_t)(((int64_t)rg * RPL * a.ld + chunk * VEC) * ES);
  const uint32_t row_bytes = (uint32_t)(a.ld * ES);

  float yr[MODE == LM_COLS ? RPL : 1];
  if (MODE == LM_COLS) {
#pragma unroll
    for (int rr = 0; rr < (MODE == LM_COLS ? RPL : 1); ++rr) yr[rr] = xs[wv][rg * RPL + rr];
  }
  const float* xrow = a.xvec + (size_t)layer * a.d;
  float acc[RPL];
#pragma unroll
  for (int rr = 0; rr < RPL; ++rr) acc[rr] = 0.f;

  const int n_full = a.d / TILE_C;
  const int t0 = strip * a.tps;
  const int t1 = min(t0 + a.tps, a.n_tiles);
  // staggered start tile and loads ahead of arithmetic, as in the W_Q sweep
  const int n_mine = t1 - t0;
  int t = t0;
  if (n_mine > 1) t += (int)(((uint32_t)item * 2654435761u) >> 16) % n_mine;
#pragma unroll 1
  for (int i = 0; i < n_mine; ++i, t = (t + 1 == t1) ? t0 : t + 1) {
    u32x4 tile[RPL];
    const uint32_t voff = lane_off + (uint32_t)(t * TILE_C * ES);
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr)
      tile[rr] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff, rr * row_bytes, kStreamPolicy);
    __builtin_amdgcn_sched_barrier(0);
    const int col = t * TILE_C + chunk * VEC;
    const int nval = a.d - col;  // >= VEC on full tiles
    if (t >= n_full) {
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
    }
    if (MODE == LM_ROWS) {
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
    } else {
      float w[VEC];
#pragma unroll
      for (int c = 0; c < VEC; ++c) w[c] = 0.f;
#pragma unroll
      for (int rr = 0; rr < RPL; ++rr)
#pragma unroll
        for (int c = 0; c < VEC; ++c) w[c] = fmaf(elem<T>(tile[rr], c), yr[MODE == LM_COLS ? rr : 0], w[c]);
#pragma unroll
      for (int c = 0; c < VEC; ++c) w[c] = group_sum(w[c]);
      if (rg == 0) {
        float* out = a.colout + (size_t)unit * a.d + col;
#pragma unroll
        for (int c = 0; c < VEC; ++c)
          if (c < nval) out[c] = w[c];
      }
    }
  }
  if (MODE == LM_ROWS) {
    const float xs_inv = 1.0f / sqrtf(a.xn2[layer]);
    float* op = a.rowpart + ((size_t)unit * a.s_out + strip) * DH + rg * RPL;
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr) {
      float s = acc[rr];
#pragma unroll
      for (int m = 1; m < CPL; m <<= 1) s = xor_sum(s, m);
      if ((rr % CPL) == chunk) op[rr] = s * xs_inv;
    }
  }
}



__global__ void __launch_bounds__(kRedThreads) layer_reduce_kernel(LayerReduceArgs r) {
  const int l = blockIdx.x, t = threadIdx.x;
  __shared__ float red[kRedThreads / 64];
  if (r.mode != 0 && r.lstat[l] != 0) return;
  float acc = 0.f;
  const float* base = r.col + (size_t)l * r.units * r.d;
  for (int c = t; c < r.d; c += kRedThreads) {
    float s = 0.f;
    for (int u = 0; u < r.units; ++u) s += base[(size_t)u * r.d + c];
    r.vec[(size_t)l * r.d + c] = s;
    acc = fmaf(s, s, acc);
  }
  acc = wave_sum(acc);
  if ((t & 63) == 0) red[t >> 6] = acc;
  __syncthreads();
  if (t == 0) {
    const float n2 = sum_waves<kRedThreads / 64>(red);
    r.n2[l] = n2;
    if (r.mode == 0) {
      r.n2_start[l] = n2;
      r.lstat[l] = (n2 > 0.f && isfinite(n2)) ? 0 : -1;
    } else if (r.mode == 1 && n2 == 0.f) {
      r.lstat[l] = -2;
    }
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

void launch_layer_reduce(int layers, hipStream_t st, const LayerReduceArgs& r) {
  layer_reduce_kernel<<<dim3(layers), kRedThreads, 0, st>>>(r);
}

void launch_layer_finalize(int layers, hipStream_t st, const LayerFinArgs& f) {
  layer_finalize_kernel<<<dim3(layers), kThreads, 0, st>>>(f);
}

}  // namespace sn
