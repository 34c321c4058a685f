// Sweep kernels of the per-head spectral-norm estimator (the default form)
// and its finalize, for MI355X (gfx950, wave64).
//
// Method (arXiv 2602.18851, Sec. 4.1-4.2, App. E): for query head h with key
// head j = floor(h / g), one step is
//     z = K_j v,  u' = Q_h^T z (= M v),  sigma = ||u'||,
//     y = Q_h u' / sigma,  v' = K_j^T y (= M^T u),  v = v' / ||v'||,
// where Q_h, K_j are the d_h x d row blocks of the PyTorch-layout weights
// (the transposes of the paper's W^Q_h, W^K_j) and M = Q_h^T K_j is never
// formed.
//
// Schedule.  Each step is two fused sweeps over the weights:
//   W_Q sweep (one wave per (head, column strip)): reads every Q_h element
//     once, computes u'[c] = sum_r Q[r,c] z[r] for the strip's columns, its
//     squared norm, and the d_h-vector partial y[r] = sum_c Q[r,c] u'[c].
//   W_K sweep (one wave per (KV head, chunk of <= 8 query heads, strip)):
//     reads every K_j element once and applies it to all query heads of the
//     chunk from registers (the implicit-GQA form of Sec. 4.2 without key
//     expansion): v'[c] = sum_r K[r,c] y_h[r], ||v'||^2, z_h[r] partials.
//     With bf16 weights and 3..8 query heads per KV head, ksweep_mfma_kernel
//     does this on the matrix cores from a tile staged once in LDS.
// In tolerance mode the heads still running after the first steps are
// finished in d_h-space (gram.hip); the final sweeps that map their last
// vectors back to d-space are launched over lists of those heads and of the
// W_K units holding one (tail_lists_kernel), item r decoding to list entry r
// instead of r itself, with the count and strips read from the device.
// Partials (one d_h vector and one squared norm per strip) go to a small
// workspace and are summed, in a fixed order, by the consumer of the next
// sweep, which also normalises (y /= sigma, z /= ||v'||).  Every reduction
// has a fixed order, so results are bitwise reproducible run to run.
//
// Wave tile.  A wave covers d_h rows x (8 chunks of 16 bytes) columns:
// lane = 8 * rg + chunk, rows rg*RPL .. rg*RPL+RPL-1 (RPL = d_h / 8),
// columns chunk*VEC .. +VEC-1 (VEC = 8 bf16 or 4 fp32).  Each load
// instruction reads eight full 128-byte row segments.  The column sums of the
// first product are reduced over the 8 row groups with lane shuffles
// (xor 8, 16, 32), the row sums of the second product accumulate in registers
// across the whole strip and are reduced over the 8 chunks once at its end.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <type_traits>

#include "sweep_device.h"

namespace sn {
namespace {

// Work item of a sweep: which layer, which d_h-row block of that layer's
// matrix, and which query heads (head0 .. head0 + nvalid - 1).
struct Item {
  int layer, row0, head0, nvalid, strip;
};

template <int DH, int GC, int PH>
__device__ __forceinline__ Item decode_item(const SweepArgs& a, int item) {
  Item it;
  bool valid_item = item < a.n_items;
  it.strip = valid_item ? item % a.s_out : 0;
  int rest = valid_item ? item / a.s_out : 0;
  if (a.list && valid_item) rest = uni(a.list[rest]);  // tail launch: only the listed heads / units
  if (PH == PH_Q || PH == PH_EQ) {  // one query head per item
    it.layer = rest / a.n_q;
    it.row0 = (rest % a.n_q) * DH;
    it.head0 = rest;
    it.nvalid = 1;
  } else {
    const int grp = rest / a.nch, ch = rest % a.nch;
    it.layer = grp / a.n_kv;
    const int j = grp % a.n_kv;
    it.row0 = j * DH;
    const int hin = ch * GC;
    it.head0 = it.layer * a.n_q + j * a.g + hin;
    it.nvalid = min(GC, a.g - hin);
  }
  if (!valid_item) it.nvalid = 0;
  return it;
}

// Per-head bookkeeping at the start of a sweep (wave-uniform): which heads of
// the item still iterate, which of them take their last step here (W_K
// sweeps decide convergence, since sigma of the step is complete only after
// the W_Q sweep), status / sigma / iteration outputs (written once, by the
// strip-0 wave), and the normalised input vector of every active head, summed
// over the producer's strips in a fixed order, into xs[i][0 .. d_h).
// The per-head scalars are gathered by lanes 0 .. nvalid - 1 in one round of
// loads and the partial vectors of all heads in s_in rounds, instead of a
// chain of dependent loads per head.
__device__ __forceinline__ float lane_f(float x, int i) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), i));
}

template <int DH, int GC, int PH>
__device__ __forceinline__ void head_setup(const SweepArgs& a, const Item& itm, int lane, float (*xs)[DH],
                                           bool (&act)[GC], bool (&last)[GC]) {
  const int strip = itm.strip, head0 = itm.head0, nvalid = itm.nvalid;
  const int slot_prev = (a.k + 1) & 1;  // parity of step k-1
  const int slot_cur = a.k & 1;
  constexpr bool ITER = PH == PH_Q || PH == PH_K;
  // ---- per-head scalars: lane i reads head head0 + i
  int l_alive = 0;
  float l_nv2 = 0.f, l_n2 = 0.f, l_s2 = 0.f, l_prev = 0.f;
  if (ITER && lane < nvalid) {
    const int hh = head0 + lane;
    l_alive = a.w.alive[slot_prev * a.H + hh];
    if (a.k == 1)
      for (int s = 0; s < a.s_k; ++s) l_nv2 += a.w.zn[hh * a.s_k + s];
    if (PH == PH_Q) {
      for (int s = 0; s < a.s_k; ++s) l_n2 += a.w.zn[(slot_prev * a.H + hh) * a.s_k + s];
    } else {
      for (int s = 0; s < a.s_q; ++s) l_s2 += a.w.yn[hh * a.s_q + s];
      l_prev = a.w.sig[slot_prev * a.H + hh];
    }
  }
  // ---- per-head decisions (wave-uniform)
  float inv[GC];
  const float* part[GC];
#pragma unroll
  for (int i = 0; i < GC; ++i) {
    act[i] = false;
    last[i] = false;
    inv[i] = 0.f;
    part[i] = nullptr;
    if (i >= nvalid) continue;
    const int hh = head0 + i;
    if (PH == PH_INIT) {
      act[i] = true;
      if (strip == 0 && lane == 0) a.w.alive[hh] = 1;  // slot 0
      continue;
    }
    if (PH == PH_EK || PH == PH_EQ) {  // final sweeps of the Gram form / the tail: heads that ran
      act[i] = uni(a.iters[hh]) > 0 && (!a.only || uni(a.only[hh]) != 0);
      last[i] = act[i];
      if (act[i]) {
        const float* src = a.w.fin + (size_t)hh * 2 * DH + (PH == PH_EK ? DH : 0);
        for (int r = lane; r < DH; r += 64) xs[i][r] = src[r];
        if (PH == PH_EK && a.only && a.w.zs && strip == 0 && lane == 0) a.w.zs[hh] = a.s_out;
      }
      continue;
    }
    bool alive = __builtin_amdgcn_readlane(l_alive, i) != 0;
    bool dead_v = false, dead_m = false;
    float nv2 = 0.f;
    if (a.k == 1) {
      nv2 = lane_f(l_nv2, i);
      if (!(nv2 > 0.f) || !isfinite(nv2)) {
        alive = false;
        dead_v = true;
      }
    }
    if (PH == PH_Q) {
      if (alive) {
        inv[i] = 1.0f / sqrtf(lane_f(l_n2, i));
        part[i] = a.w.zp + ((size_t)slot_prev * a.H + hh) * a.s_k * DH;
        act[i] = true;
      }
    } else {  // PH_K: sigma of this step is now complete
      float sigma = 0.f;
      if (alive) {
        const float s2 = lane_f(l_s2, i);
        sigma = sqrtf(s2);
        if (s2 == 0.f) {
          dead_m = true;
        } else {
          act[i] = true;
          const float prev = lane_f(l_prev, i);
          last[i] = (a.k >= a.n_iter) ||
                    (a.tol > 0.f && a.k >= 2 && fabsf(sigma - prev) <= a.tol * sigma);
          inv[i] = 1.0f / sigma;
          part[i] = a.w.yp + (size_t)hh * a.s_q * DH;
        }
      }
      if (strip == 0 && lane == 0) {
        if (a.k == 1) a.w.vnorm0[hh] = sqrtf(nv2);
        if (dead_v) {
          a.sigma[hh] = __builtin_nanf("");
          a.iters[hh] = -1;
        }
        if (dead_m) {
          a.sigma[hh] = 0.f;
          a.iters[hh] = -2;
        }
        if (act[i]) {
          a.w.sig[slot_cur * a.H + hh] = sigma;
          if (last[i]) {
            a.sigma[hh] = sigma;
            a.iters[hh] = a.k;
            if (a.w.zs) a.w.zs[hh] = a.s_out;  // the strips of this sweep's ||v'||^2 partials
          }
        }
        a.w.alive[slot_cur * a.H + hh] = (act[i] && !last[i]) ? 1 : 0;
      }
    }
    if (PH == PH_Q && dead_v) act[i] = false;
  }
  if (!ITER) return;

  // ---- normalised input vectors: partial t of every active head, t = 0, 1, ...
  constexpr int NR = (DH + 63) / 64;
  const int s_in = PH == PH_Q ? a.s_k : a.s_q;
  float xv[GC][NR];
#pragma unroll
  for (int i = 0; i < GC; ++i)
#pragma unroll
    for (int rr = 0; rr < NR; ++rr) xv[i][rr] = 0.f;
#pragma unroll kSetupUnroll
  for (int t = 0; t < s_in; ++t) {
#pragma unroll
    for (int i = 0; i < GC; ++i) {
      if (!act[i]) continue;
#pragma unroll
      for (int rr = 0; rr < NR; ++rr) {
        const int r = lane + 64 * rr;
        if (r < DH) xv[i][rr] += part[i][t * DH + r];
      }
    }
  }
#pragma unroll
  for (int i = 0; i < GC; ++i) {
    if (!act[i]) continue;
#pragma unroll
    for (int rr = 0; rr < NR; ++rr) {
      const int r = lane + 64 * rr;
      if (r < DH) xs[i][r] = xv[i][rr] * inv[i];
    }
  }
}

// Final sweeps of the tolerance-mode tail: the count of listed entries and
// the strips chosen for it come from the device control block.
template <int PH>
__device__ __forceinline__ void apply_tail_ctl(SweepArgs& a) {
  if constexpr (PH == PH_EK || PH == PH_EQ) {
    if (a.ctl) {
      a.s_out = uni(a.ctl[1]);
      a.tps = uni(a.ctl[2]);
      a.n_items = uni(a.ctl[0]) * a.s_out;
    }
  }
}

template <typename T, int DH, int GC, int PH>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(waves_hint<DH, GC>())))
sweep_kernel(SweepArgs args) {
  SweepArgs a = args;
  apply_tail_ctl<PH>(a);
  constexpr int VEC = Traits<T>::VEC;
  constexpr int CPL = kCPL;  // 16-byte column chunks per wave row: 128-byte row segments
  constexpr int RPL = DH / kRG;
  constexpr int TILE_C = CPL * VEC;
  static_assert(DH % kRG == 0, "head_dim must be a multiple of 8");
  __shared__ float xs[kWaves][GC][DH];

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int chunk = lane % CPL;
  const int rg = lane / CPL;
  const Item itm = decode_item<DH, GC, PH>(a, blockIdx.x * kWaves + wv);
  const int layer = itm.layer, row0 = itm.row0, head0 = itm.head0, strip = itm.strip;
  const int slot_cur = a.k & 1;

  // Buffer resource over this head's (or KV head's) d_h x ld row block; the
  // hardware range check returns zeros past the last valid element, and the
  // per-row offsets ride in scalar registers.
  constexpr int ES = sizeof(T);
  const char* blk = uni(a.mats[layer]) + (int64_t)row0 * a.ld * ES;
  // The range ends at the block's last valid element, rounded up to whole 16-byte
  // chunks: the hardware drops a chunk that crosses the range end, and an aligned
  // chunk that starts inside the matrix never leaves its memory page.
  const uint32_t nrec = (uint32_t)((((int64_t)(DH - 1) * a.ld + a.d) * ES + 15) & ~int64_t(15));
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(blk), (short)0, (int)nrec, kRsrcWord3);
  const uint32_t lane_off = (uint32_t)(((int64_t)rg * RPL * a.ld + chunk * VEC) * ES);
  const uint32_t row_bytes = (uint32_t)(a.ld * ES);
  auto load_tile = [&](u32x4 (&tile)[RPL], int t) {
    const uint32_t voff = lane_off + (uint32_t)(t * TILE_C * ES);
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr)
      tile[rr] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff, rr * row_bytes, kStreamPolicy);
  };

  const int n_full = a.d / TILE_C;  // tiles whose columns are all inside d
  const int t_first = strip * a.tps;
  const int t_last = min(t_first + a.tps, a.n_tiles);  // exclusive
  const int t_full_end = min(t_last, n_full);
  const bool has_tail = t_last > n_full;               // the ragged last tile is ours
  // Each wave starts at its own pseudo-random tile of the strip and wraps
  // around, so the waves that run side by side read different column
  // offsets of their 16 KB-strided rows rather than the same ones in
  // lockstep; and all loads of a tile are issued before any of its
  // arithmetic.  Together with two strips per head this took the 70B W_Q
  // sweep from 6.56 to 6.78 TB/s.  The first tile is requested before the
  // per-head set-up below, whose loads it does not depend on, so the two
  // latencies overlap.
  const int n_mine = itm.nvalid > 0 ? t_full_end - t_first : 0;
  int t = t_first;
  if (n_mine > 1) t += (int)(((uint32_t)(blockIdx.x * kWaves + wv) * 2654435761u) >> 16) % n_mine;
  u32x4 first[RPL];
  if (n_mine > 0) load_tile(first, t);

  bool act[GC], last[GC];
  head_setup<DH, GC, PH>(a, itm, lane, xs[wv], act, last);
  __syncthreads();

  bool any = false;
#pragma unroll
  for (int i = 0; i < GC; ++i) any |= act[i];
  if (!any) return;

  float xr1[GC == 1 ? RPL : 1];
  if (GC == 1 && PH != PH_INIT) {
#pragma unroll
    for (int rr = 0; rr < (GC == 1 ? RPL : 1); ++rr) xr1[rr] = xs[wv][0][rg * RPL + rr];
  }

  float acc[GC][RPL];
  float nrm[GC];
#pragma unroll
  for (int i = 0; i < GC; ++i) {
    nrm[i] = 0.f;
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr) acc[i][rr] = 0.f;
  }

  auto tile_step = [&](auto full_tag, int t, u32x4 (&tile)[RPL]) {
    constexpr bool FULL = decltype(full_tag)::value;
    const int col = t * TILE_C + chunk * VEC;
    const int nval = FULL ? VEC : a.d - col;
    if (!FULL) {
      // the ragged tail: zero the elements at columns >= d (they belong to
      // the row's padding, to the next row, or read as 0 past the range)
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

#pragma unroll
    for (int i = 0; i < GC; ++i) {
      if (!act[i]) continue;
      const int hh = head0 + i;
      float w[VEC];
      if (PH == PH_INIT) {
        const float* vrow = a.v + (size_t)hh * a.d;
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
          const float x = vrow[FULL ? col + c : min(col + c, a.d - 1)];
          w[c] = (FULL || c < nval) ? x : 0.f;
        }
      } else {
#pragma unroll
        for (int c = 0; c < VEC; ++c) w[c] = 0.f;
#pragma unroll
        for (int rr = 0; rr < RPL; ++rr) {
          const float x = (GC == 1) ? xr1[GC == 1 ? rr : 0] : xs[wv][i][rg * RPL + rr];
#pragma unroll
          for (int c = 0; c < VEC; ++c) w[c] = fmaf(elem<T>(tile[rr], c), x, w[c]);
        }
#pragma unroll
        for (int rr = 0; rr < RPL; ++rr) reuse_fence(tile[rr]);
#pragma unroll
        for (int c = 0; c < VEC; ++c) w[c] = group_sum(w[c]);
      }
#pragma unroll
      for (int c = 0; c < VEC; ++c) nrm[i] = fmaf(w[c], w[c], nrm[i]);

      // full d-space vector of the final step: v' (W_K sweep) or u' (W_Q sweep)
      constexpr bool V_OUT = PH == PH_K || PH == PH_EK;
      const bool write_vec = V_OUT ? last[i] : (PH == PH_EQ || (PH == PH_Q && a.want_vec));
      if (write_vec && rg == 0) {
        float* out = (V_OUT ? a.v : a.u) + (size_t)hh * a.d + col;
#pragma unroll
        for (int c = 0; c < VEC; ++c)
          if (FULL || c < nval) out[c] = w[c];
      }
      // z of a finished head is not needed; the final sweeps produce no z or y
      if ((PH == PH_K && last[i]) || PH == PH_EK || PH == PH_EQ) continue;
#pragma unroll
      for (int rr = 0; rr < RPL; ++rr) {
        float s = acc[i][rr];
#pragma unroll
        for (int c = 0; c < VEC; ++c) s = fmaf(elem<T>(tile[rr], c), w[c], s);
        acc[i][rr] = s;
      }
    }
  };

  if (n_mine > 0) {
    tile_step(std::true_type{}, t, first);
    if (++t == t_full_end) t = t_first;
  }
#pragma unroll 1
  for (int i = 1; i < n_mine; ++i) {
    u32x4 cur[RPL];
    load_tile(cur, t);
    __builtin_amdgcn_sched_barrier(0);
    tile_step(std::true_type{}, t, cur);
    if (++t == t_full_end) t = t_first;
  }
  if (has_tail) {  // the ragged last tile
    u32x4 cur[RPL];
    load_tile(cur, n_full);
    tile_step(std::false_type{}, n_full, cur);
  }

  if (PH == PH_EQ) return;  // u' is the only output
  // ---- reduce over the 8 column chunks and write this strip's partials
  float* outp = (PH == PH_Q) ? a.w.yp : a.w.zp + (size_t)slot_cur * a.H * a.s_k * DH;
  float* outn = (PH == PH_Q) ? a.w.yn : a.w.zn + (size_t)slot_cur * a.H * a.s_k;
#pragma unroll
  for (int i = 0; i < GC; ++i) {
    if (!act[i]) continue;
    const int hh = head0 + i;
    float n = nrm[i];  // row group 0's copy of the column sums
#pragma unroll
    for (int m = 1; m < CPL; m <<= 1) n = xor_sum(n, m);
    if (lane == 0) outn[(size_t)hh * a.s_out + strip] = n;
    if ((PH == PH_K && last[i]) || PH == PH_EK) continue;
    float* op = outp + ((size_t)hh * a.s_out + strip) * DH + rg * RPL;
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr) {
      float s = acc[i][rr];
#pragma unroll
      for (int m = 1; m < CPL; m <<= 1) s = xor_sum(s, m);
      if ((rr % CPL) == chunk) op[rr] = s;
    }
  }
}

// ---------------------------------------------------------------------------
// W_K sweep on the matrix cores (bf16 weights, d_h in {64, 128}, groups of
// 4..8 query heads).  With g heads sharing K_j, the sweep is a skinny dense
// contraction: V' = K_j^T Y (d x g) and Z = K_j V' (d_h x g).  Both products
// run as v_mfma_f32_16x16x32_bf16 with 16 "slots" = 8 heads x {hi, lo}: every
// fp32 vector is split as x = hi + lo into two bf16 values (|x - hi - lo| <=
// 2^-16 |x|) so the products keep ~16 significant bits while K stays in its
// native bf16.
//   Each tile (d_h rows x 64 columns of K_j) is staged once in LDS by
//   coalesced loads (stage_issue) and read twice from there:
//   Product 1 (contraction over rows) needs column fragments, read with
//   ds_read_b64_tr_b16, which within each 16-lane group hands lane t element
//   (t % 4) of source lane 4j + t / 4 for j = 0..3; pointing source lane s at
//   row k0 + s / 4, column 4 (s % 4) gives lane t rows k0 .. k0 + 3 of
//   column t.
//   Product 2 (contraction over columns) reads the A-operand layout: lane
//   16 g + s holds row s of a 16-row block and 8 consecutive columns.
//   v' (16 slots x 64 columns) goes back through LDS to reach the B-operand
//   layout of product 2.
// The loads of tile t + 1 are in flight while tile t is multiplied.  The
// first sweep (v' = the start vector) has no product 1: its vector values
// are requested together with their tile.
constexpr int kMVPitch = kMTileC + 8;      // LDS row pitch of the split v'

typedef short s16x4 __attribute__((ext_vector_type(4)));

// Rows r and r + 4 of a staged tile, columns col .. col + 3, transposed over
// each 16-lane group (see the comment above).
__device__ __forceinline__ bf16x8 tr_read_staged(const uint8_t* tile, int r, int col) {
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const uint8_t* p0 = tile + 128 * r + 16 * ((col >> 3) ^ stage_swz(r)) + 2 * (col & 7);
  const uint8_t* p1 = tile + 128 * (r + 4) + 16 * ((col >> 3) ^ stage_swz(r + 4)) + 2 * (col & 7);
  const s16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p0));
  const s16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p1));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7));
}

template <int GC>
__device__ __forceinline__ bool pick(const bool (&f)[GC], int i) {
  bool r = false;
#pragma unroll
  for (int k = 0; k < GC; ++k) r |= (k == i) && f[k];
  return r;
}

template <int DH, int PH>
__global__ void __launch_bounds__(64 * kMWaves) __attribute__((amdgpu_waves_per_eu(2)))
ksweep_mfma_kernel(SweepArgs args) {
  SweepArgs a = args;
  apply_tail_ctl<PH>(a);
  constexpr int GC = 8;
  constexpr int RB = DH / 16;          // 16-row blocks (product-2 M blocks)
  constexpr int KB = DH / 32;          // 32-row blocks (product-1 K blocks)
  constexpr int CB = kMTileC / 16;     // 16-column blocks (product-1 N blocks)
  constexpr int KC = kMTileC / 32;     // 32-column blocks (product-2 K blocks)
  constexpr int ES = 2;
  static_assert(DH * 128 >= GC * DH * 4, "input vectors alias the tile buffer");
  __shared__ __attribute__((aligned(16))) uint8_t lds_tile[kMWaves][DH * 128];
  __shared__ __attribute__((aligned(16))) uint16_t lds_v[kMWaves][16 * kMVPitch];

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4, s = lane & 15;
  const Item itm = decode_item<DH, GC, PH>(a, blockIdx.x * kMWaves + wv);
  const int head0 = itm.head0, strip = itm.strip;
  const int slot_cur = a.k & 1;
  uint8_t* tl = &lds_tile[wv][0];
  float (*xs)[DH] = reinterpret_cast<float (*)[DH]>(tl);  // only until the first tile is staged
  bool act[GC], last[GC];
  head_setup<DH, GC, PH>(a, itm, lane, xs, act, last);
  __syncthreads();
  bool any = false;
#pragma unroll
  for (int i = 0; i < GC; ++i) any |= act[i];
  if (!any) return;

  // heads of this lane: product-1 outputs (columns) for heads 2g, 2g+1;
  // B-operand / partial-sum slot s = head s/2, part s%2
  const bool act0 = pick(act, 2 * g), act1 = pick(act, 2 * g + 1);
  const bool last0 = pick(last, 2 * g), last1 = pick(last, 2 * g + 1);
  const bool act_s = pick(act, s >> 1), last_s = pick(last, s >> 1);
  const bool lo_part = (s & 1) != 0;

  constexpr bool PROD1 = PH == PH_K || PH == PH_EK;  // v' = K^T y
  constexpr bool PROD2 = PH != PH_EK;                // z = K v'
  bf16x8 a1[KB];  // Y^T fragments: slot s, rows 32 kb + 8 g + t
  if (PROD1) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float y = act_s ? xs[s >> 1][32 * kb + 8 * g + t] : 0.f;
        const __bf16 h = (__bf16)y;
        a1[kb][t] = lo_part ? (__bf16)(y - (float)h) : h;
      }
  }

  const char* blk = uni(a.mats[itm.layer]) + (int64_t)itm.row0 * a.ld * ES;
  const uint32_t nrec = (uint32_t)((((int64_t)(DH - 1) * a.ld + a.d) * ES + 15) & ~int64_t(15));
  const __amdgpu_buffer_rsrc_t rsrc = make_rsrc(blk, nrec);
  const uint32_t row_bytes = (uint32_t)(a.ld * ES);

  f32x4 zacc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) zacc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float nrm0 = 0.f, nrm1 = 0.f;
  const int n_full = a.d / kMTileC;
  const int t0 = strip * a.tps;
  const int t1 = min(t0 + a.tps, a.n_tiles);  // exclusive
  uint16_t* vl = &lds_v[wv][0];

  // staggered start tile, as in the W_Q sweep
  const int n_mine = t1 - t0;
  const int rot = n_mine > 1
                      ? (int)((((uint32_t)(blockIdx.x * kMWaves + wv) * 2654435761u) >> 16) % (uint32_t)n_mine)
                      : 0;
  auto tile_at = [&](int i) { const int u = rot + i; return t0 + (u >= n_mine ? u - n_mine : u); };
  // First sweep: the start-vector values of a tile's columns (lane: head
  // s / 2, columns 32 kc + 8 g .. + 7) are requested with the tile, as two
  // 16-byte loads per kc where v allows, and become the bf16 operand before
  // the next tile is requested.
  float vx[PROD1 ? 1 : KC][8];
  const float* vrow = a.v + (size_t)(head0 + (s >> 1)) * a.d;
  const bool v_vec = (a.d & 3) == 0 && (reinterpret_cast<uintptr_t>(a.v) & 15) == 0;
  auto load_v = [&](int t) {
    if constexpr (!PROD1) {
      const int c0 = t * kMTileC;
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        const int cb = c0 + 32 * kc + 8 * g;
        if (v_vec && c0 + kMTileC <= a.d) {
          float4 p0 = make_float4(0.f, 0.f, 0.f, 0.f), p1 = p0;
          if (act_s) {
            p0 = *reinterpret_cast<const float4*>(vrow + cb);
            p1 = *reinterpret_cast<const float4*>(vrow + cb + 4);
          }
          vx[kc][0] = p0.x; vx[kc][1] = p0.y; vx[kc][2] = p0.z; vx[kc][3] = p0.w;
          vx[kc][4] = p1.x; vx[kc][5] = p1.y; vx[kc][6] = p1.z; vx[kc][7] = p1.w;
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int col = cb + e;
            vx[kc][e] = (act_s && col < a.d) ? vrow[min(col, a.d - 1)] : 0.f;
          }
        }
      }
    }
  };

  __builtin_amdgcn_s_waitcnt(0);  // xs is read out before the first tile overwrites it
  if (n_mine > 0) {
    stage_issue<DH, kStreamPolicy>(rsrc, tl, (uint32_t)(tile_at(0) * 128), row_bytes, lane);
    load_v(tile_at(0));
  }
#pragma unroll 1
  for (int i = 0; i < n_mine; ++i) {
    const int t = tile_at(i);
    const int c0 = t * kMTileC;
    __builtin_amdgcn_s_waitcnt(0);  // tile t is in LDS
    bf16x8 b2[KC];
    if (!PROD1) {  // first sweep: v' is the start vector itself
#pragma unroll
      for (int kc = 0; kc < KC; ++kc)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = vx[kc][e];
          if (!lo_part) nrm0 = fmaf(x, x, nrm0);
          const __bf16 h = (__bf16)x;
          b2[kc][e] = lo_part ? (__bf16)(x - (float)h) : h;
        }
    }
    f32x4 d1[CB];
    if (PROD1) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        d1[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
          d1[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              a1[kb], tr_read_staged(tl, 32 * kb + 8 * g + (s >> 2), 16 * cb + 4 * (s & 3)), d1[cb], 0, 0, 0);
      }
    }
    u32x4 cur[RB][KC];
    if (PROD2) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) cur[rb][kc] = stage_chunk(tl, 16 * rb + s, 4 * kc + g);
    }
    __builtin_amdgcn_s_waitcnt(0);  // the tile is read out: stage the next one
    if (i + 1 < n_mine) {
      stage_issue<DH, kStreamPolicy>(rsrc, tl, (uint32_t)(tile_at(i + 1) * 128), row_bytes, lane);
      load_v(tile_at(i + 1));
    }
    if (PROD2 && t >= n_full) {  // the ragged last tile: zero columns >= d
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        const int nval = a.d - (c0 + 32 * kc + 8 * g);
        u32x4 m;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          m[q] = (2 * q < nval ? 0x0000ffffu : 0u) | (2 * q + 1 < nval ? 0xffff0000u : 0u);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) cur[rb][kc] &= m;
      }
    }

    if (PROD1) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        // lane: column 16 cb + s; slots 4g .. 4g+3 = heads 2g (hi, lo), 2g+1 (hi, lo)
        const int col = c0 + 16 * cb + s;
        const bool inside = col < a.d;  // columns past d read the row's padding or the next row
        const float v0 = inside ? d1[cb][0] + d1[cb][1] : 0.f;
        const float v1 = inside ? d1[cb][2] + d1[cb][3] : 0.f;
        nrm0 = fmaf(v0, v0, nrm0);
        nrm1 = fmaf(v1, v1, nrm1);
        if (inside) {
          if (last0) a.v[(size_t)(head0 + 2 * g) * a.d + col] = v0;
          if (last1) a.v[(size_t)(head0 + 2 * g + 1) * a.d + col] = v1;
        }
        if (!PROD2) continue;
        const __bf16 h0 = (__bf16)v0, h1 = (__bf16)v1;
        const __bf16 l0 = (__bf16)(v0 - (float)h0), l1 = (__bf16)(v1 - (float)h1);
        const int c = 16 * cb + s;
        vl[(4 * g + 0) * kMVPitch + c] = __builtin_bit_cast(uint16_t, h0);
        vl[(4 * g + 1) * kMVPitch + c] = __builtin_bit_cast(uint16_t, l0);
        vl[(4 * g + 2) * kMVPitch + c] = __builtin_bit_cast(uint16_t, h1);
        vl[(4 * g + 3) * kMVPitch + c] = __builtin_bit_cast(uint16_t, l1);
      }
      if (PROD2) {
#pragma unroll
        for (int kc = 0; kc < KC; ++kc)
          b2[kc] = *reinterpret_cast<const bf16x8*>(vl + s * kMVPitch + 32 * kc + 8 * g);
      }
    }

    if (PROD2) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int kc = 0; kc < KC; ++kc)
          zacc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, cur[rb][kc]), b2[kc],
                                                             zacc[rb], 0, 0, 0);
    }
  }

  // ---- partials of this strip
  float* zp_out = a.w.zp + (size_t)slot_cur * a.H * a.s_k * DH;
  float* zn_out = a.w.zn + (size_t)slot_cur * a.H * a.s_k;
  // z = hi-slot + lo-slot (lanes s, s ^ 1); even lanes own head s / 2
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int j = 0; j < 4; ++j) zacc[rb][j] += __shfl_xor(zacc[rb][j], 1);
  if (PROD2 && !lo_part && act_s && !last_s) {
    float* op = zp_out + ((size_t)(head0 + (s >> 1)) * a.s_out + strip) * DH + 4 * g;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) *reinterpret_cast<f32x4*>(op + 16 * rb) = zacc[rb];
  }
  if (PROD1) {  // lane (g, s) summed columns of heads 2g, 2g+1: reduce over s
#pragma unroll
    for (int m = 1; m < 16; m <<= 1) {
      nrm0 += __shfl_xor(nrm0, m);
      nrm1 += __shfl_xor(nrm1, m);
    }
    if (s == 0) {
      if (act0) zn_out[(size_t)(head0 + 2 * g) * a.s_out + strip] = nrm0;
      if (act1) zn_out[(size_t)(head0 + 2 * g + 1) * a.s_out + strip] = nrm1;
    }
  } else {  // part-0 lanes of head s/2 summed disjoint columns: reduce over g
    nrm0 += __shfl_xor(nrm0, 16);
    nrm0 += __shfl_xor(nrm0, 32);
    if (g == 0 && !lo_part && act_s) zn_out[(size_t)(head0 + (s >> 1)) * a.s_out + strip] = nrm0;
  }
}

// Normalises the final vectors and computes the per-layer scale.
// Blocks [0, H): one head each; blocks [H, H + L): one layer each.
__global__ void __launch_bounds__(kThreads) finalize_kernel(FinArgs f) {
  const int b = blockIdx.x;
  if (b < f.H) {
    const int it = f.iters[b];
    float vs = 1.f, us = 0.f;
    bool touch_v = false;
    if (it > 0) {
      float n2 = 0.f;
      const int sk = f.zs ? f.zs[b] : f.s_k;
      if (f.tail && f.tail[b] != 0) {  // finished by the tail: the final W_K sweep's own buffer
        for (int s = 0; s < sk; ++s) n2 += f.zt[(size_t)b * sk + s];
      } else {
        const int slot = f.slot_fixed >= 0 ? f.slot_fixed : (it & 1);
        for (int s = 0; s < sk; ++s) n2 += f.w.zn[((size_t)slot * f.H + b) * sk + s];
      }
      vs = 1.0f / sqrtf(n2);
      us = 1.0f / f.sigma[b];
      touch_v = true;
    } else if (it == -2) {
      vs = 1.0f / f.w.vnorm0[b];
      touch_v = true;
    }
    float* vp = f.v + (size_t)b * f.d;
    float* up = f.u ? f.u + (size_t)b * f.d : nullptr;
    for (int c = threadIdx.x; c < f.d; c += blockDim.x) {
      if (touch_v) vp[c] *= vs;
      if (up) up[c] = (it > 0) ? up[c] * us : 0.f;
    }
  } else {
    const int l = b - f.H;
    __shared__ float red[kThreads];
    __shared__ int nan_seen;
    if (threadIdx.x == 0) nan_seen = 0;
    __syncthreads();
    float m = 0.f;
    for (int h = threadIdx.x; h < f.n_q; h += blockDim.x) {
      const float s = f.sigma[(size_t)l * f.n_q + h];
      if (isnan(s)) nan_seen = 1;
      m = fmaxf(m, s);
    }
    red[threadIdx.x] = m;
    __syncthreads();
    for (int off = kThreads / 2; off > 0; off >>= 1) {
      if ((int)threadIdx.x < off) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + off]);
      __syncthreads();
    }
    if (threadIdx.x == 0) f.scale[l] = nan_seen ? __builtin_nanf("") : f.coef * red[0];
  }
}

// Lists of the tolerance-mode tail, built by one workgroup from the running
// flags after step k of the chain: thread t owns a contiguous range of
// entries and counts the running ones, and an exclusive scan of the counts in
// LDS gives each thread its first place in the list, so every list comes out
// in ascending order.  Thread 0 then writes the counts, and the strips of
// each compacted launch for its count, to the control block (TC_*).
constexpr int kTailThreads = 1024;

__device__ __forceinline__ int block_exclusive_scan(int x, int* buf, int* total) {
  const int t = threadIdx.x;
  buf[t] = x;
  __syncthreads();
  for (int off = 1; off < kTailThreads; off <<= 1) {
    const int y = t >= off ? buf[t - off] : 0;
    __syncthreads();
    buf[t] += y;
    __syncthreads();
  }
  const int incl = buf[t];
  *total = buf[kTailThreads - 1];
  __syncthreads();
  return incl - x;
}

// Strips for a compacted launch over `count` entries: about target / count
// (rounded down, so count * strips <= max(count, target)), at least
// kTailMinTiles tiles each.
__device__ __forceinline__ void tail_strips(int count, int n_tiles, int target, int32_t* out) {
  int s = count > 0 ? max(1, target / count) : 1;
  s = max(1, min(s, max(1, n_tiles / kTailMinTiles)));
  const int tps = (n_tiles + s - 1) / s;
  out[0] = count;
  out[1] = (n_tiles + tps - 1) / tps;
  out[2] = tps;
}

__global__ void __launch_bounds__(kTailThreads)
tail_lists_kernel(SweepArgs a, int slot, int gc, int n_units, TailPlan tp) {
  __shared__ int buf[kTailThreads];
  const int t = threadIdx.x;
  const int32_t* cur = a.w.alive + (size_t)slot * a.H;
  int32_t* list_g = a.w.list_g;

  // running query heads: list_g[0 .. nq)
  int nq = 0;
  const int per_h = (a.H + kTailThreads - 1) / kTailThreads;
  const int h0 = min(a.H, t * per_h), h1 = min(a.H, h0 + per_h);
  int n = 0;
  for (int hh = h0; hh < h1; ++hh) n += cur[hh] != 0 ? 1 : 0;
  int pos = block_exclusive_scan(n, buf, &nq);
  for (int hh = h0; hh < h1; ++hh)
    if (cur[hh] != 0) list_g[pos++] = hh;

  // key heads x = layer * n_kv + j serving a running head: list_g[nq ..) = H + x
  const int n_kvh = (a.H / a.n_q) * a.n_kv;
  auto kv_running = [&](int x) {
    const int head0 = (x / a.n_kv) * a.n_q + (x % a.n_kv) * a.g;
    bool r = false;
    for (int i = 0; i < a.g; ++i) r = r || cur[head0 + i] != 0;
    return r;
  };
  int nk = 0;
  const int per_x = (n_kvh + kTailThreads - 1) / kTailThreads;
  const int x0 = min(n_kvh, t * per_x), x1 = min(n_kvh, x0 + per_x);
  int m = 0;
  for (int x = x0; x < x1; ++x) m += kv_running(x) ? 1 : 0;
  pos = block_exclusive_scan(m, buf, &nk);
  for (int x = x0; x < x1; ++x) {
    if (kv_running(x)) {
      a.w.kvpos[x] = pos;
      list_g[nq + pos++] = a.H + x;
    } else {
      a.w.kvpos[x] = -1;
    }
  }

  // W_K units u = (layer * n_kv + j) * nch + ch holding a running head: query heads
  // layer * n_q + j * g + ch * gc + (0 .. min(gc, g - ch * gc) - 1)
  auto unit_running = [&](int un) {
    const int grp = un / a.nch, ch = un % a.nch;
    const int head0 = (grp / a.n_kv) * a.n_q + (grp % a.n_kv) * a.g + ch * gc;
    const int nv = min(gc, a.g - ch * gc);
    bool r = false;
    for (int i = 0; i < nv; ++i) r = r || cur[head0 + i] != 0;
    return r;
  };
  int nu = 0;
  const int per_u = (n_units + kTailThreads - 1) / kTailThreads;
  const int u0 = min(n_units, t * per_u), u1 = min(n_units, u0 + per_u);
  m = 0;
  for (int un = u0; un < u1; ++un) m += unit_running(un) ? 1 : 0;
  pos = block_exclusive_scan(m, buf, &nu);
  for (int un = u0; un < u1; ++un)
    if (unit_running(un)) a.w.list_k[pos++] = un;

  if (t == 0) {
    int32_t* c = a.w.ctl;
    tail_strips(nq + nk, tp.n_tiles_g, tp.target_g, c + TC_GRAM);
    tail_strips(nu, tp.n_tiles_k, tp.target_k, c + TC_EK);
    tail_strips(nq, tp.n_tiles_q, tp.target_q, c + TC_EQ);
    c[TC_NQ] = nq;
  }
}

template <typename T, int DH, int GC>
void launch_k(int ph, dim3 grid, hipStream_t st, const SweepArgs& a) {
  if (ph == PH_INIT)
    sweep_kernel<T, DH, GC, PH_INIT><<<grid, kThreads, 0, st>>>(a);
  else if (ph == PH_K)
    sweep_kernel<T, DH, GC, PH_K><<<grid, kThreads, 0, st>>>(a);
  else if constexpr (DH >= 16)
    sweep_kernel<T, DH, GC, PH_EK><<<grid, kThreads, 0, st>>>(a);
}

template <typename T, int DH>
void launch_dh(int ph, int gc, bool mfma, dim3 grid, hipStream_t st, const SweepArgs& a) {
  if (ph == PH_Q) {
    sweep_kernel<T, DH, 1, PH_Q><<<grid, kThreads, 0, st>>>(a);
    return;
  }
  if (ph == PH_EQ) {
    if constexpr (DH >= 16) sweep_kernel<T, DH, 1, PH_EQ><<<grid, kThreads, 0, st>>>(a);
    return;
  }
  if constexpr (std::is_same<T, uint16_t>::value && (DH == 64 || DH == 128)) {
    if (mfma) {
      const dim3 mgrid((a.n_items + kMWaves - 1) / kMWaves);
      if (ph == PH_INIT)
        ksweep_mfma_kernel<DH, PH_INIT><<<mgrid, 64 * kMWaves, 0, st>>>(a);
      else if (ph == PH_K)
        ksweep_mfma_kernel<DH, PH_K><<<mgrid, 64 * kMWaves, 0, st>>>(a);
      else
        ksweep_mfma_kernel<DH, PH_EK><<<mgrid, 64 * kMWaves, 0, st>>>(a);
      return;
    }
  }
  switch (gc) {
    case 1: launch_k<T, DH, 1>(ph, grid, st, a); break;
    case 2: launch_k<T, DH, 2>(ph, grid, st, a); break;
    case 4: launch_k<T, DH, 4>(ph, grid, st, a); break;
    default: launch_k<T, DH, 8>(ph, grid, st, a); break;
  }
}

template <typename T>
void launch_t(int dh, int ph, int gc, bool mfma, dim3 grid, hipStream_t st, const SweepArgs& a) {
  switch (dh) {
    case 8: launch_dh<T, 8>(ph, gc, mfma, grid, st, a); break;
    case 16: launch_dh<T, 16>(ph, gc, mfma, grid, st, a); break;
    case 32: launch_dh<T, 32>(ph, gc, mfma, grid, st, a); break;
    case 64: launch_dh<T, 64>(ph, gc, mfma, grid, st, a); break;
    default: launch_dh<T, 128>(ph, gc, mfma, grid, st, a); break;
  }
}

}  // namespace

void launch_sweep(bool bf16, int head_dim, int ph, int gc, bool mfma, int n_items, hipStream_t st,
                  const SweepArgs& a) {
  const dim3 grid((n_items + kWaves - 1) / kWaves);
  if (bf16)
    launch_t<uint16_t>(head_dim, ph, gc, mfma, grid, st, a);
  else
    launch_t<float>(head_dim, ph, gc, mfma, grid, st, a);
}

void launch_finalize(int blocks, hipStream_t st, const FinArgs& f) {
  finalize_kernel<<<dim3(blocks), kThreads, 0, st>>>(f);
}

void launch_tail_lists(const SweepArgs& a, int slot, int gc, int n_units, const TailPlan& tp, hipStream_t st) {
  tail_lists_kernel<<<dim3(1), kTailThreads, 0, st>>>(a, slot, gc, n_units, tp);
}

}  // namespace sn
