// FP8 E4M3 consumer of the per-layer scale: the attention logits of
// stage 3 of the geometry-aware forward pass (Sec. 3.4, Algorithm
// "Geometry-Aware Attention Forward Pass"), scaled and quantised, with the
// overflow statistics the paper reports (Sec. 1 "Problem formulation":
// overflow when |S| > scale * R_max; Table "pretrained": largest scaled
// logit; App. "FP8 Utilization Statistics").
//
// For one layer with tokens X (seq x d, bf16):
//   Q = X W_Q^T, K = X W_K^T                 (projection GEMMs, fp32 accumulation)
//   S_h = Q_h K_{j(h)}^T / sqrt(d_h)        (j(h) = floor(h / g), no key expansion)
//   S~_h = S_h / scale                       -> OCP E4M3FN code, round to nearest even;
//                                               |S~| > 464 is NaN (no saturation)
//   per head: max |S~| and #{|S~| > 448}.
// The projections keep their fp32 sums as two bf16 planes (hi + lo, |x - hi -
// lo| <= 2^-16 |x|), and the logits use three bf16 matrix-core products
// (hi.hi + hi.lo + lo.hi), so S~ carries ~2^-15 relative error instead of the
// 2^-8 a bf16 Q and K would give.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "device_util.h"
#include "logits_fp8.h"

namespace {

using namespace sn_dev;

constexpr int kWaves = 4;      // 2 x 2 waves of 64 x 64 per 128 x 128 workgroup tile
constexpr int kTile = 128;
constexpr int kLdsPitch = 68;  // bytes per row of a wave's 64 x 64 code tile in LDS

__device__ __forceinline__ f32x4 mfma(const u32x4& a, const u32x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

// Zeroes the bytes of a 16-byte chunk at element positions >= nval (bf16).
__device__ __forceinline__ void mask_bf16(u32x4& q, int nval) {
#pragma unroll
  for (int e = 0; e < 4; ++e)
    q[e] &= (2 * e < nval ? 0x0000ffffu : 0u) | (2 * e + 1 < nval ? 0xffff0000u : 0u);
}

__device__ __forceinline__ uint16_t bf16_bits(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

// Q and K projections of one layer.  Tiles of 128 tokens x 128 output
// features, Q features first, then K; a wave covers 64 x 64 (4 x 4 blocks of
// 16 x 16).  Operands come straight from memory in the MFMA layout (lane l:
// row l % 16, 16 bytes of consecutive k at 8 (l / 16)); two loads per 16-row
// block cover one 128-byte segment of each row.  Workgroups are numbered so
// that the consecutive token tiles of one feature tile run on one XCD (the
// hardware deals workgroups round-robin over the 8 XCDs) and share its L2.
__global__ void __launch_bounds__(64 * kWaves) proj_kernel(ProjArgs a) {
  const int lane = threadIdx.x & 63;
  const int wv = uni((int)(threadIdx.x >> 6));
  const int q = lane >> 4, s = lane & 15;
  const int per_xcd = gridDim.x / 8;
  const int t = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  const int tiles_q = a.tiles_m * a.tiles_nq;
  if (t >= tiles_q + a.tiles_m * a.tiles_nk) return;
  const bool isq = t < tiles_q;
  const int tt = isq ? t : t - tiles_q;
  const int bm = tt % a.tiles_m, bn = tt / a.tiles_m;
  const int ncols = isq ? a.nq_cols : a.nk_cols;
  const int m0 = bm * kTile + (wv >> 1) * 64, n0 = bn * kTile + (wv & 1) * 64;
  if (m0 >= a.seq || n0 >= ncols) return;

  const char* abase = reinterpret_cast<const char*>(a.x) + (int64_t)m0 * a.ld_x * 2;
  const char* bbase = reinterpret_cast<const char*>(isq ? a.wq : a.wk) + (int64_t)n0 * a.ld_w * 2;
  const __amdgpu_buffer_rsrc_t ra =
      make_rsrc(abase, (uint32_t)((((int64_t)(a.seq - 1 - m0) * a.ld_x + a.d) * 2 + 15) & ~int64_t(15)));
  const __amdgpu_buffer_rsrc_t rb_ =
      make_rsrc(bbase, (uint32_t)((((int64_t)(ncols - 1 - n0) * a.ld_w + a.d) * 2 + 15) & ~int64_t(15)));
  const uint32_t a_off = (uint32_t)(s * a.ld_x * 2 + 16 * q), b_off = (uint32_t)(s * a.ld_w * 2 + 16 * q);
  const uint32_t a_row16 = (uint32_t)(16 * a.ld_x * 2), b_row16 = (uint32_t)(16 * a.ld_w * 2);

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int n_kt = (a.d + 63) / 64, n_full = a.d / 64;
#pragma unroll 1
  for (int kt = 0; kt < n_kt; ++kt) {
    u32x4 fa[4][2], fb[4][2];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) {
        fa[r][kc] = __builtin_amdgcn_raw_buffer_load_b128(ra, a_off + kt * 128 + 64 * kc, r * a_row16, 0);
        fb[r][kc] = __builtin_amdgcn_raw_buffer_load_b128(rb_, b_off + kt * 128 + 64 * kc, r * b_row16, 0);
      }
    if (kt >= n_full) {  // the ragged last k tile: zero columns >= d
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) {
        const int nval = a.d - (kt * 64 + 32 * kc + 8 * q);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          mask_bf16(fa[r][kc], nval);
          mask_bf16(fb[r][kc], nval);
        }
      }
    }
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma(fa[i][kc], fb[j][kc], acc[i][j]);
  }

  uint16_t* hi = isq ? a.qh : a.kh;
  uint16_t* lo = isq ? a.ql : a.kl;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + 16 * i + 4 * q + e, n = n0 + 16 * j + s;
        if (m < a.seq && n < ncols) {
          const float x = acc[i][j][e];
          const __bf16 h = (__bf16)x;
          hi[(size_t)m * ncols + n] = __builtin_bit_cast(uint16_t, h);
          lo[(size_t)m * ncols + n] = bf16_bits(x - (float)h);
        }
      }
}

// OCP E4M3FN code of an fp32 value, round to nearest even: magnitudes in
// [448, 464] give 448 (464 is the tie between 448 and the absent 480, and
// 448's mantissa is even), larger ones and NaN give the NaN code 0x7F.
__device__ __forceinline__ uint32_t e4m3_code(float x) {
  const uint32_t b = __float_as_uint(x);
  const uint32_t sign = (b >> 24) & 0x80u;
  const float ax = fabsf(x);
  if (!(ax <= 464.f)) return sign | 0x7Fu;
  if (ax >= 448.f) return sign | 0x7Eu;
  if (ax < 0.015625f) return sign | (uint32_t)__builtin_rintf(ax * 512.f);  // m * 2^-9, m = 0..8
  const uint32_t ab = b & 0x7FFFFFFFu;
  int e = (int)(ab >> 23) - 127;  // -6 .. 8
  uint32_t man = (ab >> 20) & 7u;
  const uint32_t rem = ab & 0xFFFFFu;
  if (rem > 0x80000u || (rem == 0x80000u && (man & 1u))) ++man;
  if (man == 8u) {
    man = 0u;
    ++e;
  }
  return sign | ((uint32_t)(e + 7) << 3) | man;
}

// Logits of one layer: one 128 x 128 tile of S for one query head per
// workgroup, 64 x 64 per wave, K-dimension d_h in steps of 32.
template <int DH>
__global__ void __launch_bounds__(64 * kWaves) logits_kernel(LogitArgs a) {
  constexpr int KC = (DH + 31) / 32;
  __shared__ __attribute__((aligned(16))) uint8_t lds[kWaves][64 * kLdsPitch];
  const int lane = threadIdx.x & 63;
  const int wv = uni((int)(threadIdx.x >> 6));
  const int q = lane >> 4, s = lane & 15;
  const int per_head = a.tiles * a.tiles;
  const int h = blockIdx.x / per_head;
  const int ti = (blockIdx.x % per_head) / a.tiles, tj = blockIdx.x % a.tiles;
  const int i0 = ti * kTile + (wv >> 1) * 64, j0 = tj * kTile + (wv & 1) * 64;
  if (i0 >= a.seq || j0 >= a.seq) return;
  const int kvh = h / a.g;

  const int64_t qrow = (int64_t)a.nq_cols * 2, krow = (int64_t)a.nk_cols * 2;
  const uint32_t q_bytes = (uint32_t)((((int64_t)(a.seq - 1 - i0) * a.nq_cols + DH) * 2 + 15) & ~int64_t(15));
  const uint32_t k_bytes = (uint32_t)((((int64_t)(a.seq - 1 - j0) * a.nk_cols + DH) * 2 + 15) & ~int64_t(15));
  const size_t qo = (size_t)i0 * a.nq_cols + (size_t)h * DH, ko = (size_t)j0 * a.nk_cols + (size_t)kvh * DH;
  const __amdgpu_buffer_rsrc_t rqh = make_rsrc(a.qh + qo, q_bytes), rql = make_rsrc(a.ql + qo, q_bytes);
  const __amdgpu_buffer_rsrc_t rkh = make_rsrc(a.kh + ko, k_bytes), rkl = make_rsrc(a.kl + ko, k_bytes);
  const uint32_t q_off = (uint32_t)(s * qrow + 16 * q), k_off = (uint32_t)(s * krow + 16 * q);
  const uint32_t q16 = (uint32_t)(16 * qrow), k16 = (uint32_t)(16 * krow);

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    const bool kval = 32 * kc + 8 * q < DH;  // chunks past d_h belong to the next head
    u32x4 ah[4], al[4], bh[4], bl[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      ah[r] = __builtin_amdgcn_raw_buffer_load_b128(rqh, q_off + 64 * kc, r * q16, 0);
      al[r] = __builtin_amdgcn_raw_buffer_load_b128(rql, q_off + 64 * kc, r * q16, 0);
      bh[r] = __builtin_amdgcn_raw_buffer_load_b128(rkh, k_off + 64 * kc, r * k16, 0);
      bl[r] = __builtin_amdgcn_raw_buffer_load_b128(rkl, k_off + 64 * kc, r * k16, 0);
      if (!kval) ah[r] = al[r] = bh[r] = bl[r] = u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc[i][j] = mfma(ah[i], bh[j], acc[i][j]);
        acc[i][j] = mfma(ah[i], bl[j], acc[i][j]);
        acc[i][j] = mfma(al[i], bh[j], acc[i][j]);
      }
  }

  // S~ = (q . k) / (sqrt(d_h) scale), the factor formed in double
  const float c = (float)(1.0 / (std::sqrt((double)DH) * (double)a.scale[a.layer]));
  uint8_t* tile = lds[wv];
  int n_over = 0;
  float mx = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * i + 4 * q + e, col = 16 * j + s;
        const bool in = (i0 + r < a.seq) && (j0 + col < a.seq);
        const float v = acc[i][j][e] * c;
        const float av = fabsf(v);
        n_over += (in && av > 448.f) ? 1 : 0;
        mx = in ? fmaxf(mx, av) : mx;
        tile[r * kLdsPitch + col] = (uint8_t)e4m3_code(v);
      }
  if (a.codes) {
    // lane = row of the tile: 64 bytes out, whole 16-byte stores where the
    // row lies inside the matrix
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int row = i0 + lane;
    if (row < a.seq) {
      uint8_t* out = a.codes + ((size_t)h * a.seq + row) * a.seq + j0;
      const uint8_t* src = tile + lane * kLdsPitch;
      const int ncol = min(64, a.seq - j0);
      if (ncol == 64 && (a.seq & 15) == 0) {
#pragma unroll
        for (int c16 = 0; c16 < 4; ++c16) {
          u32x4 w;
#pragma unroll
          for (int b = 0; b < 4; ++b) w[b] = *reinterpret_cast<const uint32_t*>(src + 16 * c16 + 4 * b);
          *reinterpret_cast<u32x4*>(out + 16 * c16) = w;
        }
      } else {
        for (int cc = 0; cc < ncol; ++cc) out[cc] = src[cc];
      }
    }
  }
  // per-head statistics: integer sum and maximum of non-negative floats are
  // independent of the order of the atomics
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    n_over += __shfl_xor(n_over, m);
    mx = fmaxf(mx, __shfl_xor(mx, m));
  }
  if (lane == 0) {
    if (n_over) atomicAdd(a.n_over + h, n_over);
    atomicMax(reinterpret_cast<int32_t*>(a.max_abs) + h, __float_as_int(mx));
  }
}

__global__ void zero_stats_kernel(float* max_abs, int32_t* n_over, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    max_abs[i] = 0.f;
    n_over[i] = 0;
  }
}

}  // namespace

int64_t sn_logits_workspace_bytes(int64_t seq, int64_t nq_cols, int64_t nk_cols) {
  return seq * (nq_cols + nk_cols) * 4;  // hi and lo bf16 planes of Q and K
}

void sn_launch_zero_stats(float* max_abs, int32_t* n_over, int n, hipStream_t st) {
  zero_stats_kernel<<<dim3((n + 255) / 256), 256, 0, st>>>(max_abs, n_over, n);
}

void sn_launch_proj(const ProjArgs& a, hipStream_t st) {
  const int tiles = a.tiles_m * (a.tiles_nq + a.tiles_nk);
  proj_kernel<<<dim3(((tiles + 7) / 8) * 8), 64 * kWaves, 0, st>>>(a);
}

void sn_launch_logits(const LogitArgs& a, int head_dim, int n_q, hipStream_t st) {
  const dim3 grid(n_q * a.tiles * a.tiles);
  switch (head_dim) {
    case 16: logits_kernel<16><<<grid, 64 * kWaves, 0, st>>>(a); break;
    case 32: logits_kernel<32><<<grid, 64 * kWaves, 0, st>>>(a); break;
    case 64: logits_kernel<64><<<grid, 64 * kWaves, 0, st>>>(a); break;
    default: logits_kernel<128><<<grid, 64 * kWaves, 0, st>>>(a); break;
  }
}
