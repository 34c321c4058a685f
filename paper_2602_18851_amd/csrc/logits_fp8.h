// Internal interface between the C ABI (spectral.hip) and the FP8 logit
// consumer kernels (logits_fp8.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

struct ProjArgs {
  const uint16_t* x;   // [seq][ld_x] bf16 tokens of the layer
  int64_t ld_x;
  const uint16_t* wq;  // [n_q d_h][ld_w] bf16
  const uint16_t* wk;  // [n_kv d_h][ld_w] bf16
  int64_t ld_w;
  int32_t seq, d, nq_cols, nk_cols;  // nq_cols = n_q d_h, nk_cols = n_kv d_h
  int32_t tiles_m, tiles_nq, tiles_nk;
  uint16_t* qh;  // [seq][nq_cols] bf16 planes: Q = hi + lo
  uint16_t* ql;
  uint16_t* kh;  // [seq][nk_cols]
  uint16_t* kl;
};

struct LogitArgs {
  const uint16_t* qh;
  const uint16_t* ql;
  const uint16_t* kh;
  const uint16_t* kl;
  int32_t seq, g, nq_cols, nk_cols, tiles, n_heads;
  const float* scale;  // device [L]
  int32_t layer;
  uint8_t* codes;      // [n_q][seq][seq] of this layer, or nullptr
  float* max_abs;      // [n_q] of this layer
  int32_t* n_over;     // [n_q] of this layer
};

int64_t sn_logits_workspace_bytes(int64_t seq, int64_t nq_cols, int64_t nk_cols);
void sn_launch_zero_stats(float* max_abs, int32_t* n_over, int n, hipStream_t st);
void sn_launch_proj(const ProjArgs& a, hipStream_t st);
void sn_launch_logits(const LogitArgs& a, int head_dim, hipStream_t st);
