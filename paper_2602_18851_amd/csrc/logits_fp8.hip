// FP8 E4M3 consumer of the per-layer scale: the attention logits of
// stage 3 of the geometry-aware forward pass (Sec. 3.4, Algorithm
// "Geometry-Aware Attention Forward Pass"), scaled and quantised, with the
// overflow statistics the paper reports (Sec. 1 "Problem formulation":
// overflow when |S| > scale * R_max; Table "pretrained": largest scaled
// logit; App. "FP8 Utilization Statistics").
//
// For each layer, with that layer's tokens X (seq x d, bf16); one launch of
// each kernel covers every layer:
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

constexpr int kWaves = 4;      // logit kernel: 2 x 2 waves of 64 x 64 per 128 x 128 tile
constexpr int kTile = 128;

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

// Q and K projections of all layers in one launch.  Workgroup tiles of
// 256 tokens x 256 output features (per layer Q features first, then K) and
// 8 waves, two per SIMD, each covering 128 x 64 as 8 x 4 blocks of 16 x 16:
// while one wave of a SIMD waits for LDS or the barrier, the other keeps the
// matrix core busy.  The workgroup streams its 256 token rows and 256 weight
// rows through LDS in steps of 64 columns (128-byte row segments, coalesced
// loads straight to LDS, two stages of 64 KB; see stage_issue).  Workgroups
// are numbered so that the consecutive token tiles of one feature tile run on
// one XCD (the hardware deals workgroups round-robin over the 8 XCDs) and
// share its L2.
constexpr int kPT = 256;                    // projection workgroup tile
constexpr int kPWaves = 8;
constexpr int kPStageBytes = 2 * kPT * 128;  // A and B rows of one 64-column step

__global__ void __launch_bounds__(64 * kPWaves) __attribute__((amdgpu_waves_per_eu(2, 2))) proj_kernel(ProjArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t stage[2][kPStageBytes];
  const int lane = threadIdx.x & 63;
  const int wv = uni((int)(threadIdx.x >> 6));
  const int q = lane >> 4, s = lane & 15;
  const int per_xcd = gridDim.x / 8;
  const int tq = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  const int tiles_q = a.tiles_m * a.tiles_nq, per_layer = tiles_q + a.tiles_m * a.tiles_nk;
  if (tq >= a.layers * per_layer) return;  // whole workgroup
  const int layer = tq / per_layer, t = tq % per_layer;
  const bool isq = t < tiles_q;
  const int tt = isq ? t : t - tiles_q;
  const int bm = tt % a.tiles_m, bn = tt / a.tiles_m;
  const int ncols = isq ? a.nq_cols : a.nk_cols;

  // this wave stages rows 32 wv .. 32 wv + 31 of the A (token) and B (weight) tiles
  const int am = bm * kPT + 32 * wv, bnr = bn * kPT + 32 * wv;
  const char* abase = uni(a.x[layer]) + (int64_t)am * a.ld_x * 2;
  const char* bbase = uni(isq ? a.wq[layer] : a.wk[layer]) + (int64_t)bnr * a.ld_w * 2;
  const int64_t a_len = am < a.seq ? (((int64_t)(a.seq - 1 - am) * a.ld_x + a.d) * 2 + 15) & ~int64_t(15) : 0;
  const int64_t b_len = bnr < ncols ? (((int64_t)(ncols - 1 - bnr) * a.ld_w + a.d) * 2 + 15) & ~int64_t(15) : 0;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(abase, (uint32_t)a_len);
  const __amdgpu_buffer_rsrc_t rb_ = make_rsrc(bbase, (uint32_t)b_len);
  const uint32_t a_rb = (uint32_t)(a.ld_x * 2), b_rb = (uint32_t)(a.ld_w * 2);
  auto issue = [&](int k, int st) {
    stage_issue<32, 0>(ra, stage[st] + 4096 * wv, (uint32_t)(k * 128), a_rb, lane);
    stage_issue<32, 0>(rb_, stage[st] + kPT * 128 + 4096 * wv, (uint32_t)(k * 128), b_rb, lane);
  };

  const int wm = wv >> 2, wn = wv & 3;  // 2 x 4 waves of 128 x 64
  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int n_k = (a.d + 63) / 64, n_full = a.d / 64;
  issue(0, 0);
#pragma unroll 1
  for (int k = 0; k < n_k; ++k) {
    __builtin_amdgcn_s_waitcnt(0);  // this wave's part of step k is in LDS
    __syncthreads();                // every part, and step k - 1 fully read
    if (k + 1 < n_k) issue(k + 1, (k + 1) & 1);
    const uint8_t* sa = stage[k & 1];
    const uint8_t* sb = sa + kPT * 128;
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      u32x4 fa[8], fb[4];
#pragma unroll
      for (int r = 0; r < 8; ++r) fa[r] = stage_chunk(sa, 128 * wm + 16 * r + s, 4 * kc + q);
#pragma unroll
      for (int r = 0; r < 4; ++r) fb[r] = stage_chunk(sb, 64 * wn + 16 * r + s, 4 * kc + q);
      if (k >= n_full) {  // the ragged last step: zero columns >= d
        const int nval = a.d - (k * 64 + 32 * kc + 8 * q);
#pragma unroll
        for (int r = 0; r < 8; ++r) mask_bf16(fa[r], nval);
#pragma unroll
        for (int r = 0; r < 4; ++r) mask_bf16(fb[r], nval);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma(fa[i], fb[j], acc[i][j]);
    }
  }

  const int m0 = bm * kPT + 128 * wm, n0 = bn * kPT + 64 * wn;
  const size_t plane = (size_t)layer * a.seq * ncols;
  uint16_t* hi = (isq ? a.qh : a.kh) + plane;
  uint16_t* lo = (isq ? a.ql : a.kl) + plane;
#pragma unroll
  for (int i = 0; i < 8; ++i)
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

// Logits of all layers in one launch: one 128 x 128 tile of S of one query
// head of one layer per workgroup, 64 x 64 per wave.  The workgroup stages the hi and lo planes of
// its 128 query rows and 128 key rows through LDS, 64 columns of d_h at a
// time (coalesced loads; see stage_issue), and every wave reads its operands
// back in the MFMA layout.  The products are formed transposed (A = key
// rows, B = query rows), so a lane holds 4 consecutive columns of one row of
// S: one 32-bit word of E4M3 codes.  v_cvt_pk_fp8_f32 (no clamp) rounds to
// nearest even and gives the NaN code past 464, the OCP E4M3FN conversion the
// oracle defines; a bit-by-bit comparison with an integer encoder over every
// rounding point and 400k random values in [-600, 600] found no difference
// for non-NaN inputs.
constexpr int kPlaneBytes = kTile * 128;  // 128 rows x 64 columns of one bf16 plane

template <int DH>
__global__ void __launch_bounds__(64 * kWaves) logits_kernel(LogitArgs a) {
  constexpr int NSTEP = (DH + 63) / 64;  // 64-column steps over d_h
  __shared__ __attribute__((aligned(16))) uint8_t stage[4 * kPlaneBytes];  // Q hi, Q lo, K hi, K lo
  const int lane = threadIdx.x & 63;
  const int wv = uni((int)(threadIdx.x >> 6));
  const int q = lane >> 4, s = lane & 15;
  // consecutive tiles (one head after another, the heads of a key group in
  // turn) run on one XCD and share its L2
  const int per_head = a.tiles * a.tiles;
  const int per_xcd = gridDim.x / 8;
  const int bl = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (bl >= a.layers * a.n_heads * per_head) return;  // whole workgroup
  const int layer = bl / (a.n_heads * per_head), b = bl % (a.n_heads * per_head);
  const int h = b / per_head;
  const int ti = (b % per_head) / a.tiles, tj = b % a.tiles;
  const int kvh = h / a.g;
  const int wm = wv >> 1, wn = wv & 1;
  const int i0 = ti * kTile + 64 * wm, j0 = tj * kTile + 64 * wn;  // this wave's rows of S

  // this wave stages rows 32 wv .. 32 wv + 31 of the four planes
  const int qr = ti * kTile + 32 * wv, kr = tj * kTile + 32 * wv;
  const int64_t q_len = qr < a.seq ? (((int64_t)(a.seq - 1 - qr) * a.nq_cols + DH) * 2 + 15) & ~int64_t(15) : 0;
  const int64_t k_len = kr < a.seq ? (((int64_t)(a.seq - 1 - kr) * a.nk_cols + DH) * 2 + 15) & ~int64_t(15) : 0;
  const size_t qo = ((size_t)layer * a.seq + qr) * a.nq_cols + (size_t)h * DH;
  const size_t ko = ((size_t)layer * a.seq + kr) * a.nk_cols + (size_t)kvh * DH;
  const __amdgpu_buffer_rsrc_t rqh = make_rsrc(a.qh + qo, (uint32_t)q_len), rql = make_rsrc(a.ql + qo, (uint32_t)q_len);
  const __amdgpu_buffer_rsrc_t rkh = make_rsrc(a.kh + ko, (uint32_t)k_len), rkl = make_rsrc(a.kl + ko, (uint32_t)k_len);
  const uint32_t q_rb = (uint32_t)(a.nq_cols * 2), k_rb = (uint32_t)(a.nk_cols * 2);
  auto issue = [&](int st) {
    const uint32_t col = (uint32_t)(st * 128);
    stage_issue<32, 0>(rqh, stage + 0 * kPlaneBytes + 4096 * wv, col, q_rb, lane);
    stage_issue<32, 0>(rql, stage + 1 * kPlaneBytes + 4096 * wv, col, q_rb, lane);
    stage_issue<32, 0>(rkh, stage + 2 * kPlaneBytes + 4096 * wv, col, k_rb, lane);
    stage_issue<32, 0>(rkl, stage + 3 * kPlaneBytes + 4096 * wv, col, k_rb, lane);
  };

  f32x4 acc[4][4];  // acc[i][j][e] = S[i0 + 16 i + s][j0 + 16 j + 4 q + e]
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  issue(0);
#pragma unroll
  for (int st = 0; st < NSTEP; ++st) {
    __builtin_amdgcn_s_waitcnt(0);  // this wave's part of step st is in LDS
    __syncthreads();                // every part
    u32x4 ah[2][4], al[2][4], bh[2][4], bl[2][4];
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      const bool kval = st * 64 + 32 * kc + 8 * q < DH;  // chunks past d_h belong to the next head
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        ah[kc][r] = stage_chunk(stage + 0 * kPlaneBytes, 64 * wm + 16 * r + s, 4 * kc + q);
        al[kc][r] = stage_chunk(stage + 1 * kPlaneBytes, 64 * wm + 16 * r + s, 4 * kc + q);
        bh[kc][r] = stage_chunk(stage + 2 * kPlaneBytes, 64 * wn + 16 * r + s, 4 * kc + q);
        bl[kc][r] = stage_chunk(stage + 3 * kPlaneBytes, 64 * wn + 16 * r + s, 4 * kc + q);
        if (!kval) ah[kc][r] = al[kc][r] = bh[kc][r] = bl[kc][r] = u32x4{0u, 0u, 0u, 0u};
      }
    }
    if (st + 1 < NSTEP) {
      __builtin_amdgcn_s_waitcnt(0);  // read out
      __syncthreads();                // by every wave, before the next step overwrites
      issue(st + 1);
    }
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[i][j] = mfma(bh[kc][j], ah[kc][i], acc[i][j]);
          acc[i][j] = mfma(bl[kc][j], ah[kc][i], acc[i][j]);
          acc[i][j] = mfma(bh[kc][j], al[kc][i], acc[i][j]);
        }
  }
  if (i0 >= a.seq || j0 >= a.seq) return;

  // S~ = (q . k) / (sqrt(d_h) scale), the factor formed in double
  const float c = (float)(1.0 / (std::sqrt((double)DH) * (double)a.scale[layer]));
  const bool words = (a.seq & 3) == 0;  // rows start 4-byte aligned
  // A scaled logit that is not finite (a NaN or zero scale, an inf product)
  // cannot be represented either: it counts as an overflow, and the maximum
  // is kept on the bit patterns of |S~| (ordered as integers, +inf and NaN
  // above every finite value), so a NaN or inf reaches max_abs.
  int n_over = 0;
  int mx = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = i0 + 16 * i + s;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = j0 + 16 * j + 4 * q;
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = acc[i][j][e] * c;
        const bool in = row < a.seq && col + e < a.seq;
        const float av = fabsf(v[e]);
        n_over += (in && !(av <= 448.f)) ? 1 : 0;
        mx = in ? max(mx, __float_as_int(av)) : mx;
      }
      if (a.codes && row < a.seq) {
        int w = __builtin_amdgcn_cvt_pk_fp8_f32(v[0], v[1], 0, false);
        w = __builtin_amdgcn_cvt_pk_fp8_f32(v[2], v[3], w, true);
        uint8_t* out = a.codes + (((size_t)layer * a.n_heads + h) * a.seq + row) * a.seq + col;
        if (words && col + 3 < a.seq) {
          *reinterpret_cast<int*>(out) = w;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (col + e < a.seq) out[e] = (uint8_t)(w >> (8 * e));
        }
      }
    }
  }
  // per-head statistics: integer sum and integer maximum of the bit patterns
  // of non-negative floats are independent of the order of the atomics
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    n_over += __shfl_xor(n_over, m);
    mx = max(mx, __shfl_xor(mx, m));
  }
  if (lane == 0) {
    const int hl = layer * a.n_heads + h;
    if (n_over) atomicAdd(a.n_over + hl, n_over);
    atomicMax(reinterpret_cast<int32_t*>(a.max_abs) + hl, mx);
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

int64_t sn_logits_workspace_bytes(int64_t layers, int64_t seq, int64_t nq_cols, int64_t nk_cols) {
  // device pointer tables (tokens, wq, wk of every layer), then the hi and lo
  // bf16 planes of Q and K of every layer
  return ((3 * layers * 8 + 255) & ~int64_t(255)) + layers * seq * (nq_cols + nk_cols) * 4;
}

void sn_launch_zero_stats(float* max_abs, int32_t* n_over, int n, hipStream_t st) {
  zero_stats_kernel<<<dim3((n + 255) / 256), 256, 0, st>>>(max_abs, n_over, n);
}

void sn_launch_proj(const ProjArgs& args, hipStream_t st) {
  ProjArgs a = args;
  a.tiles_m = (a.seq + kPT - 1) / kPT;
  a.tiles_nq = (a.nq_cols + kPT - 1) / kPT;
  a.tiles_nk = (a.nk_cols + kPT - 1) / kPT;
  const int tiles = a.layers * a.tiles_m * (a.tiles_nq + a.tiles_nk);
  proj_kernel<<<dim3(((tiles + 7) / 8) * 8), 64 * kPWaves, 0, st>>>(a);
}

void sn_launch_logits(const LogitArgs& a, int head_dim, hipStream_t st) {
  const dim3 grid(((a.layers * a.n_heads * a.tiles * a.tiles + 7) / 8) * 8);
  switch (head_dim) {
    case 16: logits_kernel<16><<<grid, 64 * kWaves, 0, st>>>(a); break;
    case 32: logits_kernel<32><<<grid, 64 * kWaves, 0, st>>>(a); break;
    case 64: logits_kernel<64><<<grid, 64 * kWaves, 0, st>>>(a); break;
    default: logits_kernel<128><<<grid, 64 * kWaves, 0, st>>>(a); break;
  }
}
