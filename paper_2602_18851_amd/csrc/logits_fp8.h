// Internal interface between the C ABI (spectral.hip) and the FP8 logit
// consumer kernels (logits_fp8.hip).  One launch of each kernel covers every
// layer.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

struct ProjArgs {
  const void* const* x;   // device table [L]: tokens of layer l, bf16 [seq][ld_x]
  int64_t ld_x;
  const void* const* wq;  // device table [L]: [n_q d_h][ld_w] bf16
  const void* const* wk;  // device table [L]: [n_kv d_h][ld_w] bf16
  int64_t ld_w;
  int32_t layers, seq, d, nq_cols, nk_cols;  // nq_cols = n_q d_h, nk_cols = n_kv d_h
  int32_t tiles_m, tiles_nq, tiles_nk;       // per layer (set by sn_launch_proj)
  uint16_t* qh;  // [L][seq][nq_cols] bf16 planes: Q = hi + lo
  uint16_t* ql;
  uint16_t* kh;  // [L][seq][nk_cols]
  uint16_t* kl;
};

struct LogitArgs {
  const uint16_t* qh;
  const uint16_t* ql;
  const uint16_t* kh;
  const uint16_t* kl;
  int32_t layers, seq, g, nq_cols, nk_cols, tiles, n_heads;
  const float* scale;  // device [L]
  uint8_t* codes;      // [L][n_q][seq][seq], or nullptr
  float* max_abs;      // [L][n_q]
  int32_t* n_over;     // [L][n_q]
};

int64_t sn_logits_workspace_bytes(int64_t layers, int64_t seq, int64_t nq_cols, int64_t nk_cols);
void sn_launch_zero_stats(float* max_abs, int32_t* n_over, int n, hipStream_t st);
void sn_launch_proj(const ProjArgs& a, hipStream_t st);
void sn_launch_logits(const LogitArgs& a, int head_dim, hipStream_t st);
