// Per-head spectral norms of the query-key interaction matrices of every
// attention layer by implicit power iteration, and the per-layer FP8 E4M3
// scale factor, for MI355X (gfx950, wave64).
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

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <string>
#include <type_traits>
#include <vector>

#include "device_util.h"
#include "logits_fp8.h"
#include "spectral.h"

namespace {

using namespace sn_dev;

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define SN_HIP(expr)                                                                  \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess)                                                             \
      return fail(SN_EHIP, std::string(#expr) + " failed: " + hipGetErrorString(e_)); \
  } while (0)

constexpr int kWaves = 4;             // waves per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kRG = 8;                // row groups per wave (lane >> 3)
constexpr int kCPL = 8;               // 16-byte column chunks per wave row (lane & 7)
constexpr int kMaxGC = 8;             // query heads per W_K work item
constexpr int kQTargetItems = 16384;  // wave work items aimed for in a W_Q sweep
constexpr int kKTargetItems = 4096;   // ... and in a W_K sweep (register-heavier waves)
constexpr int kKMfmaResident = 2048;  // waves of the matrix-core W_K sweep resident at once (256 CUs x 8)
constexpr int kStreamPolicy = 2;       // cache policy of the weight loads: non-temporal (read once per sweep)

// Sweep phases: the first W_K sweep from v, the W_Q and W_K sweeps of a step,
// and the two final sweeps of the Gram form (v' = K_j^T y and u' = Q_h^T z
// from the d_h-vectors the Gram iteration leaves behind).
enum { PH_INIT = 0, PH_Q = 1, PH_K = 2, PH_EK = 3, PH_EQ = 4 };
enum {
  KIND_INIT = 0, KIND_Q = 1, KIND_K = 2, KIND_FIN = 3, KIND_GRAM = 4, KIND_ITER = 5, KIND_EMIT = 6,
  KIND_LROWS = 7, KIND_LCOLS = 8, KIND_LRED = 9, KIND_PROJ = 10, KIND_LOGITS = 11, KIND_N = 12
};
static_assert(KIND_N == SN_PROFILE_KINDS, "profile kinds");

struct Work {
  float* zp;         // [2][H][Sk][DH]  W_K-sweep partials of z, by step parity
  float* zn;         // [2][H][Sk]      ... and of ||v'||^2 (||v||^2 for the first sweep)
  float* yp;         // [H][Sq][DH]     W_Q-sweep partials of y
  float* yn;         // [H][Sq]         ... and of ||u'||^2 = sigma^2
  float* sig;        // [2][H]          sigma of the last two steps
  float* vnorm0;     // [H]             ||v|| of the start vector
  int32_t* alive;    // [2][H]          head continues after the step of that parity
  int32_t* n_alive;  // [2]             heads still running after a W_K sweep
  int32_t* iters;    // [H]             used when the caller passes no iters array
  float* fin;        // [H][2][DH]      Gram form: z and y of each head's last step
};

struct SweepArgs {
  const void* const* mats;  // device table: per-layer wq or wk
  int64_t ld;
  int32_t d, n_q, n_kv, g, H;
  int32_t s_q, s_k;         // strips of the W_Q and W_K sweeps
  int32_t s_out, tps, n_tiles, nch, n_items;
  int32_t k, n_iter, want_vec;
  float tol;
  Work w;
  float* v;
  float* u;
  float* sigma;
  int32_t* iters;
};

struct FinArgs {
  int32_t H, L, n_q, d, s_k;
  int32_t slot_fixed;  // workspace slot of the ||v'||^2 partials; -1: parity of the last step
  float coef;
  Work w;
  float* v;
  float* u;
  float* sigma;
  float* scale;
  int32_t* iters;
};

template <typename T>
struct Traits;
template <>
struct Traits<float> {
  static constexpr int VEC = 4;
};
template <>
struct Traits<uint16_t> {  // bf16 bit patterns
  static constexpr int VEC = 8;
};


template <typename T>
__device__ __forceinline__ float elem(const u32x4& q, int c);
template <>
__device__ __forceinline__ float elem<float>(const u32x4& q, int c) {
  return __uint_as_float(q[c]);
}
template <>
__device__ __forceinline__ float elem<uint16_t>(const u32x4& q, int c) {
  const uint32_t w = q[c >> 1];
  return __uint_as_float((c & 1) ? (w & 0xffff0000u) : (w << 16));
}

// Marks a chunk as redefined so the compiler re-derives its float values for
// the second product instead of keeping all of them live across the lane
// shuffles (that would double the register footprint of a tile).
__device__ __forceinline__ void reuse_fence(u32x4& q) { asm volatile("" : "+v"(q)); }

__device__ __forceinline__ float xor_sum(float x, int m) { return x + __shfl_xor(x, m); }

// Sum over the 64 lanes of a wave (butterfly: every lane gets the same bits).
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

// Occupancy floor per SIMD: the accumulators grow with GC * DH / 8 floats.
template <int DH, int GC>
constexpr int waves_hint() {
  return GC * DH / kRG >= 128 ? 2 : GC * DH / kRG >= 64 ? 3 : 4;
}

// Sum over the 8 row groups of a wave tile (lanes that share lane mod 8):
// the step inside a 16-lane row is a DPP row rotation by 8 fused into the
// add; the steps across rows are lane shuffles.  Every lane ends with the
// same total for its column.
__device__ __forceinline__ float group_sum(float x) {
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x128, 0xF, 0xF, false));
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

// Work item of a sweep: which layer, which d_h-row block of that layer's
// matrix, and which query heads (head0 .. head0 + nvalid - 1).
struct Item {
  int layer, row0, head0, nvalid, strip;
};

template <int DH, int GC, int PH>
__device__ __forceinline__ Item decode_item(const SweepArgs& a, int item) {
  Item it;
  const bool valid_item = item < a.n_items;
  it.strip = valid_item ? item % a.s_out : 0;
  const int rest = valid_item ? item / a.s_out : 0;
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
template <int DH, int GC, int PH>
__device__ __forceinline__ void head_setup(const SweepArgs& a, const Item& itm, int lane, float (*xs)[DH],
                                           bool (&act)[GC], bool (&last)[GC]) {
  const int strip = itm.strip, head0 = itm.head0, nvalid = itm.nvalid;
  const int slot_prev = (a.k + 1) & 1;  // parity of step k-1
  const int slot_cur = a.k & 1;
  // ---- per-head decisions (wave-uniform) and normalised input vectors
  int n_cont = 0;
#pragma unroll
  for (int i = 0; i < GC; ++i) {
    act[i] = false;
    last[i] = false;
    if (i >= nvalid) continue;
    const int hh = head0 + i;
    if (PH == PH_INIT) {
      act[i] = true;
      if (strip == 0 && lane == 0) a.w.alive[hh] = 1;  // slot 0
      continue;
    }
    if (PH == PH_EK || PH == PH_EQ) {  // final sweeps of the Gram form: heads that ran
      act[i] = uni(a.iters[hh]) > 0;
      last[i] = act[i];
      if (act[i]) {
        const float* src = a.w.fin + (size_t)hh * 2 * DH + (PH == PH_EK ? DH : 0);
        for (int r = lane; r < DH; r += 64) xs[i][r] = src[r];
      }
      continue;
    }
    bool alive = uni(a.w.alive[slot_prev * a.H + hh]) != 0;
    bool dead_v = false, dead_m = false;
    float nv2 = 0.f;
    if (a.k == 1) {
      for (int s = 0; s < a.s_k; ++s) nv2 += a.w.zn[hh * a.s_k + s];
      nv2 = uni(nv2);
      if (!(nv2 > 0.f) || !isfinite(nv2)) {
        alive = false;
        dead_v = true;
      }
    }
    float inv = 0.f;
    const float* part = nullptr;
    int s_in = 0;
    if (PH == PH_Q) {
      if (alive) {
        float n2 = 0.f;
        for (int s = 0; s < a.s_k; ++s) n2 += a.w.zn[(slot_prev * a.H + hh) * a.s_k + s];
        inv = 1.0f / sqrtf(uni(n2));
        part = a.w.zp + ((size_t)slot_prev * a.H + hh) * a.s_k * DH;
        s_in = a.s_k;
        act[i] = true;
      }
    } else {  // PH_K: sigma of this step is now complete
      float sigma = 0.f;
      if (alive) {
        float s2 = 0.f;
        for (int s = 0; s < a.s_q; ++s) s2 += a.w.yn[hh * a.s_q + s];
        s2 = uni(s2);
        sigma = sqrtf(s2);
        if (s2 == 0.f) {
          dead_m = true;
        } else {
          act[i] = true;
          const float prev = uni(a.w.sig[slot_prev * a.H + hh]);
          last[i] = (a.k >= a.n_iter) ||
                    (a.tol > 0.f && a.k >= 2 && fabsf(sigma - prev) <= a.tol * sigma);
          inv = 1.0f / sigma;
          part = a.w.yp + (size_t)hh * a.s_q * DH;
          s_in = a.s_q;
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
          }
        }
        a.w.alive[slot_cur * a.H + hh] = (act[i] && !last[i]) ? 1 : 0;
      }
      n_cont += (act[i] && !last[i]) ? 1 : 0;
    }
    if (PH == PH_Q && dead_v) act[i] = false;
    if (act[i]) {
      for (int r = lane; r < DH; r += 64) {
        float s = 0.f;
        for (int t = 0; t < s_in; ++t) s += part[t * DH + r];
        xs[i][r] = s * inv;
      }
    }
  }
  if (PH == PH_K && strip == 0 && lane == 0 && n_cont > 0) atomicAdd(&a.w.n_alive[slot_cur], n_cont);
}

template <typename T, int DH, int GC, int PH>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(waves_hint<DH, GC>())))
sweep_kernel(SweepArgs a) {
  constexpr int VEC = Traits<T>::VEC;
  constexpr int CPL = kCPL;  // 16-byte column chunks per wave row: 128-byte row segments
  constexpr int RPL = DH / kRG;
  constexpr int TILE_C = CPL * VEC;
  static_assert(DH % kRG == 0, "head_dim must be a multiple of 8");
  __shared__ float xs[kWaves][GC][DH];

  if (PH == PH_Q && blockIdx.x == 0 && threadIdx.x == 0) a.w.n_alive[a.k & 1] = 0;

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int chunk = lane % CPL;
  const int rg = lane / CPL;
  const Item itm = decode_item<DH, GC, PH>(a, blockIdx.x * kWaves + wv);
  const int layer = itm.layer, row0 = itm.row0, head0 = itm.head0, strip = itm.strip;
  const int slot_cur = a.k & 1;
  bool act[GC], last[GC];
  head_setup<DH, GC, PH>(a, itm, lane, xs[wv], act, last);
  __syncthreads();

  bool any = false;
#pragma unroll
  for (int i = 0; i < GC; ++i) any |= act[i];
  if (!any) return;

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

  const int n_full = a.d / TILE_C;  // tiles whose columns are all inside d
  const int t_first = strip * a.tps;
  const int t_last = min(t_first + a.tps, a.n_tiles);  // exclusive
  const int t_full_end = min(t_last, n_full);
  const bool has_tail = t_last > n_full;               // the ragged last tile is ours

  auto load_tile = [&](u32x4 (&tile)[RPL], int t) {
    const uint32_t voff = lane_off + (uint32_t)(t * TILE_C * ES);
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr)
      tile[rr] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff, rr * row_bytes, kStreamPolicy);
  };
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

#pragma unroll 1
  for (int t = t_first; t < t_full_end; ++t) {
    u32x4 cur[RPL];
    load_tile(cur, t);
    tile_step(std::true_type{}, t, cur);
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
// The loads of tile t + 1 are in flight while tile t is multiplied.
constexpr int kMWaves = 2;                 // waves per workgroup
constexpr int kMTileC = 64;                // columns per tile: 128-byte row segments
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
ksweep_mfma_kernel(SweepArgs a) {
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

  __builtin_amdgcn_s_waitcnt(0);  // xs is read out before the first tile overwrites it
  if (t0 < t1) stage_issue<DH, kStreamPolicy>(rsrc, tl, (uint32_t)(t0 * 128), row_bytes, lane);
#pragma unroll 1
  for (int t = t0; t < t1; ++t) {
    const int c0 = t * kMTileC;
    __builtin_amdgcn_s_waitcnt(0);  // tile t is in LDS
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
    if (t + 1 < t1) stage_issue<DH, kStreamPolicy>(rsrc, tl, (uint32_t)((t + 1) * 128), row_bytes, lane);
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

    bf16x8 b2[KC];
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
    } else {  // first sweep: v' is the start vector itself
      const float* vrow = a.v + (size_t)(head0 + (s >> 1)) * a.d;
#pragma unroll
      for (int kc = 0; kc < KC; ++kc)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int col = c0 + 32 * kc + 8 * g + e;
          const float x = (act_s && col < a.d) ? vrow[min(col, a.d - 1)] : 0.f;
          if (!lo_part) nrm0 = fmaf(x, x, nrm0);
          const __bf16 h = (__bf16)x;
          b2[kc][e] = lo_part ? (__bf16)(x - (float)h) : h;
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
constexpr int kGWaves = 4;                 // waves per workgroup of the Gram sweep
constexpr int kGTargetItems = 4096;        // Gram work items aimed for (about two waves per SIMD)

struct GramArgs {
  const void* const* mats;  // device table: wq pointers of all layers, then wk pointers
  int64_t ld;
  int32_t d, L, n_q, n_kv, H;
  int32_t s_g, tps, n_tiles, n_items;
  float* gp;  // [units][s_g][NB][64 lanes][4]: partial Gram blocks in the MFMA output layout
};

template <int RB>
__host__ __device__ constexpr int tri_index(int bi, int bj) {  // bj >= bi
  return bi * RB - bi * (bi - 1) / 2 + (bj - bi);
}

template <typename T, int DH>
__global__ void __launch_bounds__(64 * kGWaves) __attribute__((amdgpu_waves_per_eu(DH >= 128 ? 2 : 4)))
gram_kernel(GramArgs a) {
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
  const int unit = item / a.s_g, strip = item % a.s_g;
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

  // one LDS tile per wave: tile t + 1 streams in while tile t is multiplied
  // from registers
  if (t0 < t1) stage_issue<DH, kStreamPolicy>(rsrc, tile, (uint32_t)(t0 * 128), row_bytes, lane);
#pragma unroll 1
  for (int t = t0; t < t1; ++t) {
    __builtin_amdgcn_s_waitcnt(0);  // the tile is in LDS
    u32x4 fr[RB][2];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) fr[rb][kc] = stage_chunk(tile, 16 * rb + s, 4 * kc + q);
    __builtin_amdgcn_s_waitcnt(0);  // read out before the next tile overwrites it
    if (t + 1 < t1) stage_issue<DH, kStreamPolicy>(rsrc, tile, (uint32_t)((t + 1) * 128), row_bytes, lane);
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
struct IterArgs {
  int32_t H, n_q, n_kv, g, s_k, s_g, n_iter;
  float tol;
  const float* gp;
  Work w;
  float* sigma;
  int32_t* iters;
};

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

template <int NW>
__device__ __forceinline__ float sum_waves(const float* red) {
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) s += red[w];
  return s;
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
  const int h = blockIdx.x, t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int R = t >> 4, C = t & 15;
  const int layer = h / a.n_q;
  const int j = layer * a.n_kv + (h % a.n_q) / a.g;

  // start vector: ||v||^2 and z = K_j v from the first W_K sweep (slot 0)
  float nv2 = 0.f;
  for (int st = 0; st < a.s_k; ++st) nv2 += a.w.zn[(size_t)h * a.s_k + st];
  if (t == 0) a.w.vnorm0[h] = sqrtf(nv2);
  if (!(nv2 > 0.f) || !isfinite(nv2)) {
    if (t == 0) {
      a.sigma[h] = __builtin_nanf("");
      a.iters[h] = -1;
    }
    return;
  }
  const float inv0 = 1.0f / sqrtf(nv2);
  if (t < DH) {
    float z = 0.f;
    for (int st = 0; st < a.s_k; ++st) z += a.w.zp[((size_t)h * a.s_k + st) * DH + t];
    tb[t] = z * inv0;
  }
  float gq[RPT][CPT], gk[RPT][CPT];
  gram_to_regs<DH>(a.gp + (size_t)h * a.s_g * S::NB * 256, a.s_g, gl, gq);
  gram_to_regs<DH>(a.gp + (size_t)(a.H + j) * a.s_g * S::NB * 256, a.s_g, gl, gk);

  float zscale = 1.f, prev = 0.f;
  float out[RPT];
#pragma unroll 1
  for (int k = 1;; ++k) {
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
enum { LM_ROWS = 0, LM_COLS = 1 };

struct LayerArgs {
  const void* const* mats;  // device table of this matrix's per-layer pointers
  int64_t ld;
  int32_t d, units, n_items, s_out, tps, n_tiles;
  const int32_t* lstat;     // [L]
  // rows sweep: x = xvec[layer] / sqrt(xn2[layer]) -> rowpart [L*units][s_out][DH]
  const float* xvec;
  const float* xn2;
  float* rowpart;
  // cols sweep: y = sum over y_cnt source units starting at (ul / y_div) * y_cnt
  // of the source rows sweep's partials (y_units per layer, y_strips strips)
  const float* ypart;
  int32_t y_units, y_strips, y_div, y_cnt;
  float* colout;            // [L*units][d]
};

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
#pragma unroll 1
  for (int t = t0; t < t1; ++t) {
    u32x4 tile[RPL];
    const uint32_t voff = lane_off + (uint32_t)(t * TILE_C * ES);
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr)
      tile[rr] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff, rr * row_bytes, kStreamPolicy);
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

// Per layer: vec[c] = sum over the layer's units of col[unit][c] (fixed order)
// and n2 = ||vec||^2; mode 0 copies the caller's start vector instead and
// (re)initialises the layer status; mode 1 marks M v = 0.
struct LayerReduceArgs {
  const float* col;
  int32_t units, d, mode;
  float* vec;
  float* n2;
  float* n2_start;  // mode 0: ||v||^2 of the start vector
  int32_t* lstat;
};

constexpr int kRedThreads = 512;

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

// Outputs of the layer-level form: sigma, scale, v = v'/||v'||, u = u'/sigma.
struct LayerFinArgs {
  int32_t d, L;
  float coef;
  const int32_t* lstat;
  const float* lu;
  const float* lv;
  const float* n2_u;
  const float* n2_v;
  const float* n2_start;
  float* v;
  float* u;
  float* sigma;
  float* scale;
};

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
      const int slot = f.slot_fixed >= 0 ? f.slot_fixed : (it & 1);
      for (int s = 0; s < f.s_k; ++s) n2 += f.w.zn[((size_t)slot * f.H + b) * f.s_k + s];
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

// ------------------------------------------------------------------ host side

struct Plan {
  int H, g, gc, nch, vec, tile_c, n_tiles;   // W_K sweeps
  int tile_cq, n_tiles_q;                    // W_Q sweep
  bool mfma_k;  // W_K sweeps on the matrix cores
  int s_q, tps_q, s_k, tps_k;
  bool gram;    // Gram form
  int units_g, s_g, tps_g, n_tiles_g, nb_g;
  bool layer;   // layer-level form
  int s_lq, tps_lq, s_lk, tps_lk;  // row / column strips of the layer-form sweeps over W_Q and W_K
  size_t off_zp, off_zn, off_yp, off_yn, off_sig, off_vn, off_alive, off_nalive, off_iters, off_fin, off_gp;
  size_t off_lz, off_ly, off_lcol, off_lu, off_lv, off_ln2, off_lstat;
  size_t bytes;
};

int esize(int dtype) { return dtype == SN_F32 ? 4 : 2; }

bool supported_dh(int dh) { return dh == 8 || dh == 16 || dh == 32 || dh == 64 || dh == 128; }

int validate(const sn_shape* s, const sn_params* p) {
  if (!s || !p) return fail(SN_ENULL, "shape and params must not be NULL");
  if (s->dtype != SN_F32 && s->dtype != SN_BF16) return fail(SN_EDTYPE, "dtype must be SN_F32 or SN_BF16");
  if (s->n_layers < 1 || s->d_model < 1 || s->n_q_heads < 1 || s->n_kv_heads < 1 || s->head_dim < 1)
    return fail(SN_EINVAL, "n_layers, d_model, n_q_heads, n_kv_heads and head_dim must be >= 1");
  if (s->n_q_heads % s->n_kv_heads != 0) return fail(SN_EINVAL, "n_kv_heads must divide n_q_heads");
  if (!supported_dh(s->head_dim)) return fail(SN_EINVAL, "head_dim must be one of 8, 16, 32, 64, 128");
  const int64_t ld = s->ld == 0 ? s->d_model : s->ld;
  if (ld < s->d_model) return fail(SN_EINVAL, "ld must be >= d_model");
  if ((ld * esize(s->dtype)) % 16 != 0) return fail(SN_EINVAL, "ld * element size must be a multiple of 16 bytes");
  const int64_t H = (int64_t)s->n_layers * s->n_q_heads;
  if (H * (int64_t)s->d_model > (int64_t(1) << 40) || H > (1 << 26))
    return fail(SN_EINVAL, "shape too large");
  if (!(p->alpha > 0.f) || !(p->eta_fp8 > 0.f) || !(p->r_max > 0.f) || !std::isfinite(p->alpha) ||
      !std::isfinite(p->eta_fp8) || !std::isfinite(p->r_max))
    return fail(SN_EINVAL, "alpha, eta_fp8 and r_max must be finite and > 0");
  if (!(p->tol >= 0.f) || !std::isfinite(p->tol)) return fail(SN_EINVAL, "tol must be finite and >= 0");
  if (p->q_strips < 0 || p->k_strips < 0) return fail(SN_EINVAL, "strip counts must be >= 0");
  if (p->flags & ~(SN_FLAG_VALU_K_SWEEP | SN_FLAG_GRAM | SN_FLAG_LAYER)) return fail(SN_EINVAL, "unknown flag bits");
  if ((p->flags & SN_FLAG_GRAM) && s->head_dim < 16) return fail(SN_EINVAL, "the Gram form needs head_dim >= 16");
  if ((int64_t)s->head_dim * ld * esize(s->dtype) >= (int64_t(1) << 31))
    return fail(SN_EINVAL, "head_dim * ld * element size must be below 2^31 bytes");
  return SN_OK;
}

int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// Column strips per unit (head or KV head): the request if given, else about
// target / units (rounded up, or down when all waves should be resident at once).
void strips(int n_tiles, int64_t units, int requested, int target, bool round_down, int* s_out, int* tps_out) {
  const int64_t u = std::max<int64_t>(units, 1);
  int s = requested > 0 ? requested : round_down ? (int)std::max<int64_t>(1, target / u) : ceil_div(target, u);
  s = std::max(1, std::min(s, n_tiles));
  const int tps = ceil_div(n_tiles, s);
  *tps_out = tps;
  *s_out = ceil_div(n_tiles, tps);
}

Plan make_plan(const sn_shape* s, const sn_params* p) {
  Plan pl{};
  const int dh = s->head_dim;
  pl.H = s->n_layers * s->n_q_heads;
  pl.g = s->n_q_heads / s->n_kv_heads;
  pl.gc = 1;
  while (pl.gc < pl.g && pl.gc < kMaxGC) pl.gc *= 2;
  pl.nch = ceil_div(pl.g, pl.gc);
  pl.vec = 16 / esize(s->dtype);
  pl.mfma_k = s->dtype == SN_BF16 && (dh == 64 || dh == 128) && pl.gc >= 4 &&
              !(p->flags & SN_FLAG_VALU_K_SWEEP);
  // the MFMA W_K sweep tiles 64 columns, the vector sweeps 8 chunks of 16 bytes;
  // both sweeps of a plan share one tile width (so one strip split)
  pl.tile_c = pl.mfma_k ? kMTileC : kCPL * pl.vec;
  pl.n_tiles = ceil_div(s->d_model, pl.tile_c);
  pl.tile_cq = kCPL * pl.vec;
  pl.n_tiles_q = ceil_div(s->d_model, pl.tile_cq);
  strips(pl.n_tiles_q, pl.H, p->q_strips, kQTargetItems, false, &pl.s_q, &pl.tps_q);
  strips(pl.n_tiles, (int64_t)s->n_layers * s->n_kv_heads * pl.nch, p->k_strips,
         pl.mfma_k ? kKMfmaResident : kKTargetItems, pl.mfma_k, &pl.s_k, &pl.tps_k);
  pl.gram = (p->flags & SN_FLAG_GRAM) != 0;
  if (pl.gram) {
    const int rb = dh / 16;
    pl.nb_g = rb * (rb + 1) / 2;
    pl.units_g = pl.H + s->n_layers * s->n_kv_heads;
    pl.n_tiles_g = ceil_div((int64_t)s->d_model * esize(s->dtype), 128);
    strips(pl.n_tiles_g, pl.units_g, 0, kGTargetItems, true, &pl.s_g, &pl.tps_g);
  }
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += (bytes + 255) & ~size_t(255);
    return o;
  };
  const size_t H = pl.H;
  pl.off_zp = take(2 * H * pl.s_k * dh * 4);
  pl.off_zn = take(2 * H * pl.s_k * 4);
  pl.off_yp = take(H * pl.s_q * dh * 4);
  pl.off_yn = take(H * pl.s_q * 4);
  pl.off_sig = take(2 * H * 4);
  pl.off_vn = take(H * 4);
  pl.off_alive = take(2 * H * 4);
  pl.off_nalive = take(2 * 4);
  pl.off_iters = take(H * 4);
  if (pl.gram) {
    pl.off_fin = take(H * 2 * dh * 4);
    pl.off_gp = take((size_t)pl.units_g * pl.s_g * pl.nb_g * 256 * 4);
  }
  pl.layer = (p->flags & SN_FLAG_LAYER) != 0;
  if (pl.layer) {
    const size_t L = s->n_layers, Hk = L * s->n_kv_heads, d = s->d_model;
    strips(pl.n_tiles_q, pl.H, 0, kQTargetItems, false, &pl.s_lq, &pl.tps_lq);
    strips(pl.n_tiles_q, (int64_t)Hk, 0, kQTargetItems, false, &pl.s_lk, &pl.tps_lk);
    pl.off_lz = take(Hk * pl.s_lk * dh * 4);
    pl.off_ly = take(H * pl.s_lq * dh * 4);
    pl.off_lcol = take(H * d * 4);
    pl.off_lu = take(L * d * 4);
    pl.off_lv = take(L * d * 4);
    pl.off_ln2 = take(3 * L * 4);
    pl.off_lstat = take(L * 4);
  }
  pl.bytes = off;
  return pl;
}

struct ProfRec {
  int kind;
  hipEvent_t a, b;
};

}  // namespace

// Shared with the host-side calibration helpers (calibration.cpp).
void sn_set_last_error(const char* msg) { g_err = msg; }

struct sn_ctx {
  sn_shape shape;
  sn_params params;
  Plan plan;
  hipStream_t stream = nullptr;
  int device = 0;
  char* ws = nullptr;
  Work w{};
  const void** d_tab = nullptr;  // device [2L]: wq pointers then wk pointers
  const void** h_tab = nullptr;  // pinned staging for the table copy
  std::vector<const void*> cached;
  hipEvent_t tab_event = nullptr;
  int32_t* h_alive = nullptr;    // pinned readback of n_alive
  bool prof = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> pool;
};

namespace {

hipEvent_t take_event(sn_ctx* c) {
  if (!c->pool.empty()) {
    hipEvent_t e = c->pool.back();
    c->pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
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
      const dim3 mgrid(ceil_div(a.n_items, kMWaves));
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

// Brackets one launch with profiling events when profiling is on.
template <typename F>
int timed(sn_ctx* c, int kind, F&& launch) {
  ProfRec rec{kind, nullptr, nullptr};
  if (c->prof) {
    rec.a = take_event(c);
    rec.b = take_event(c);
    if (!rec.a || !rec.b) return fail(SN_EHIP, "hipEventCreate failed");
    SN_HIP(hipEventRecord(rec.a, c->stream));
  }
  launch();
  SN_HIP(hipGetLastError());
  if (c->prof) {
    SN_HIP(hipEventRecord(rec.b, c->stream));
    c->recs.push_back(rec);
  }
  return SN_OK;
}

int launch_sweep(sn_ctx* c, int ph, SweepArgs a) {
  const Plan& pl = c->plan;
  if (ph == PH_Q || ph == PH_EQ) {
    a.mats = c->d_tab;
    a.s_out = pl.s_q;
    a.tps = pl.tps_q;
    a.n_tiles = pl.n_tiles_q;
    a.n_items = pl.H * pl.s_q;
  } else {
    a.mats = c->d_tab + c->shape.n_layers;
    a.s_out = pl.s_k;
    a.tps = pl.tps_k;
    a.n_tiles = pl.n_tiles;
    a.n_items = c->shape.n_layers * c->shape.n_kv_heads * pl.nch * pl.s_k;
  }
  const dim3 grid(ceil_div(a.n_items, kWaves));
  const int kind = ph == PH_INIT ? KIND_INIT : ph == PH_Q ? KIND_Q : ph == PH_K ? KIND_K : KIND_EMIT;
  return timed(c, kind, [&] {
    if (c->shape.dtype == SN_BF16)
      launch_t<uint16_t>(c->shape.head_dim, ph, pl.gc, pl.mfma_k, grid, c->stream, a);
    else
      launch_t<float>(c->shape.head_dim, ph, pl.gc, pl.mfma_k, grid, c->stream, a);
  });
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

// Eq. "scale" per unit of sigma: alpha * d / sqrt(d_h) / (eta_fp8 * r_max), in double.
float scale_coef(const sn_ctx* c) {
  return (float)((double)c->params.alpha * (double)c->shape.d_model /
                 (std::sqrt((double)c->shape.head_dim) * (double)c->params.eta_fp8 * (double)c->params.r_max));
}

// Checks the layer pointers and the device, and refreshes the device copy of
// the per-layer pointer table when the pointers changed.
int update_table(sn_ctx* c, const void* const* wq_layers, const void* const* wk_layers) {
  const int L = c->shape.n_layers;
  for (int l = 0; l < L; ++l) {
    if (!wq_layers[l] || !wk_layers[l]) return fail(SN_ENULL, "a layer weight pointer is NULL");
    if ((reinterpret_cast<uintptr_t>(wq_layers[l]) | reinterpret_cast<uintptr_t>(wk_layers[l])) & 15)
      return fail(SN_EINVAL, "layer weight pointers must be 16-byte aligned");
  }
  int cur_dev = 0;
  SN_HIP(hipGetDevice(&cur_dev));
  if (cur_dev != c->device) return fail(SN_ESTATE, "the current HIP device is not the context's device");
  bool same = c->cached.size() == (size_t)(2 * L);
  for (int l = 0; same && l < L; ++l)
    same = c->cached[l] == wq_layers[l] && c->cached[L + l] == wk_layers[l];
  if (!same) {
    SN_HIP(hipEventSynchronize(c->tab_event));  // the staging buffer's previous copy has been read
    c->cached.assign(2 * L, nullptr);
    for (int l = 0; l < L; ++l) {
      c->h_tab[l] = c->cached[l] = wq_layers[l];
      c->h_tab[L + l] = c->cached[L + l] = wk_layers[l];
    }
    SN_HIP(hipMemcpyAsync(c->d_tab, c->h_tab, 2 * L * sizeof(void*), hipMemcpyHostToDevice, c->stream));
    SN_HIP(hipEventRecord(c->tab_event, c->stream));
  }
  return SN_OK;
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

// One layer-form sweep over W_Q (q = true) or W_K.
int layer_sweep(sn_ctx* c, bool q, int mode, LayerArgs a) {
  const Plan& pl = c->plan;
  const int L = c->shape.n_layers;
  a.mats = c->d_tab + (q ? 0 : L);
  a.ld = c->shape.ld;
  a.d = c->shape.d_model;
  a.units = q ? c->shape.n_q_heads : c->shape.n_kv_heads;
  a.s_out = q ? pl.s_lq : pl.s_lk;
  a.tps = q ? pl.tps_lq : pl.tps_lk;
  a.n_tiles = pl.n_tiles_q;
  a.n_items = L * a.units * a.s_out;
  a.lstat = reinterpret_cast<const int32_t*>(c->ws + pl.off_lstat);
  const dim3 grid(ceil_div(a.n_items, kWaves));
  const int dh = c->shape.head_dim;
  return timed(c, mode == LM_ROWS ? KIND_LROWS : KIND_LCOLS, [&] {
    if (c->shape.dtype == SN_BF16) {
      if (mode == LM_ROWS) layer_dispatch<uint16_t, LM_ROWS>(dh, grid, c->stream, a);
      else layer_dispatch<uint16_t, LM_COLS>(dh, grid, c->stream, a);
    } else {
      if (mode == LM_ROWS) layer_dispatch<float, LM_ROWS>(dh, grid, c->stream, a);
      else layer_dispatch<float, LM_COLS>(dh, grid, c->stream, a);
    }
  });
}

int layer_reduce(sn_ctx* c, const float* col, int units, int mode, float* vec, float* n2) {
  const Plan& pl = c->plan;
  LayerReduceArgs r{};
  r.col = col;
  r.units = units;
  r.d = c->shape.d_model;
  r.mode = mode;
  r.vec = vec;
  r.n2 = n2;
  r.n2_start = reinterpret_cast<float*>(c->ws + pl.off_ln2) + 2 * c->shape.n_layers;
  r.lstat = reinterpret_cast<int32_t*>(c->ws + pl.off_lstat);
  return timed(c, KIND_LRED,
               [&] { layer_reduce_kernel<<<dim3(c->shape.n_layers), kRedThreads, 0, c->stream>>>(r); });
}

// The sweeps of the default form: first W_K sweep, then n_iter x (W_Q sweep,
// W_K sweep).  In tolerance mode the host polls the count of running heads at
// iterations 2, 3, 4, 6, 9, ... and stops queueing once it is zero.
int run_chain(sn_ctx* c, SweepArgs a, float* u) {
  int rc;
  a.k = 0;
  if ((rc = launch_sweep(c, PH_INIT, a)) != SN_OK) return rc;
  int next_check = 2;
  for (int k = 1; k <= a.n_iter; ++k) {
    a.k = k;
    a.want_vec = (u != nullptr) && (c->params.tol > 0.f || k == a.n_iter);
    if ((rc = launch_sweep(c, PH_Q, a)) != SN_OK) return rc;
    a.want_vec = 0;
    if ((rc = launch_sweep(c, PH_K, a)) != SN_OK) return rc;
    if (c->params.tol > 0.f && k == next_check && k < a.n_iter) {
      SN_HIP(hipMemcpyAsync(c->h_alive, c->w.n_alive + (k & 1), sizeof(int32_t), hipMemcpyDeviceToHost,
                            c->stream));
      SN_HIP(hipStreamSynchronize(c->stream));
      if (c->h_alive[0] == 0) break;
      next_check = k < 4 ? k + 1 : k + k / 2;
    }
  }
  return SN_OK;
}

// The Gram form of one call: first W_K sweep, Gram sweep, d_h-space
// iteration, final W_K sweep (and W_Q sweep for u).
int run_gram(sn_ctx* c, SweepArgs a, float* u) {
  const Plan& pl = c->plan;
  int rc;
  a.k = 0;
  if ((rc = launch_sweep(c, PH_INIT, a)) != SN_OK) return rc;

  GramArgs g{};
  g.mats = c->d_tab;
  g.ld = c->shape.ld;
  g.d = c->shape.d_model;
  g.L = c->shape.n_layers;
  g.n_q = c->shape.n_q_heads;
  g.n_kv = c->shape.n_kv_heads;
  g.H = pl.H;
  g.s_g = pl.s_g;
  g.tps = pl.tps_g;
  g.n_tiles = pl.n_tiles_g;
  g.n_items = pl.units_g * pl.s_g;
  g.gp = reinterpret_cast<float*>(c->ws + pl.off_gp);
  const dim3 ggrid(ceil_div(g.n_items, kGWaves));
  const int dh = c->shape.head_dim;
  rc = timed(c, KIND_GRAM, [&] {
    if (c->shape.dtype == SN_BF16)
      gram_dispatch<uint16_t>(dh, ggrid, c->stream, g);
    else
      gram_dispatch<float>(dh, ggrid, c->stream, g);
  });
  if (rc != SN_OK) return rc;

  IterArgs it{};
  it.H = pl.H;
  it.n_q = c->shape.n_q_heads;
  it.n_kv = c->shape.n_kv_heads;
  it.g = pl.g;
  it.s_k = pl.s_k;
  it.s_g = pl.s_g;
  it.n_iter = a.n_iter;
  it.tol = a.tol;
  it.gp = g.gp;
  it.w = c->w;
  it.sigma = a.sigma;
  it.iters = a.iters;
  rc = timed(c, KIND_ITER, [&] {
    switch (dh) {
      case 16: gram_iterate_kernel<16><<<dim3(pl.H), IterShape<16>::NT, 0, c->stream>>>(it); break;
      case 32: gram_iterate_kernel<32><<<dim3(pl.H), IterShape<32>::NT, 0, c->stream>>>(it); break;
      case 64: gram_iterate_kernel<64><<<dim3(pl.H), IterShape<64>::NT, 0, c->stream>>>(it); break;
      default: gram_iterate_kernel<128><<<dim3(pl.H), IterShape<128>::NT, 0, c->stream>>>(it); break;
    }
  });
  if (rc != SN_OK) return rc;

  a.k = 0;  // the final sweeps write their ||v'||^2 partials to slot 0
  if ((rc = launch_sweep(c, PH_EK, a)) != SN_OK) return rc;
  if (u && (rc = launch_sweep(c, PH_EQ, a)) != SN_OK) return rc;
  return SN_OK;
}

}  // namespace

extern "C" {

SN_API const char* spectral_last_error(void) { return g_err.c_str(); }

SN_API int spectral_workspace_bytes(const sn_shape* shape, const sn_params* params, int64_t* bytes) {
  if (!bytes) return fail(SN_ENULL, "bytes must not be NULL");
  const int rc = validate(shape, params);
  if (rc != SN_OK) return rc;
  *bytes = (int64_t)make_plan(shape, params).bytes;
  return SN_OK;
}

SN_API int spectral_init(sn_ctx** ctx, const sn_shape* shape, const sn_params* params, void* hip_stream) {
  if (!ctx) return fail(SN_ENULL, "ctx must not be NULL");
  *ctx = nullptr;
  const int rc = validate(shape, params);
  if (rc != SN_OK) return rc;
  sn_ctx* c = new sn_ctx();
  c->shape = *shape;
  if (c->shape.ld == 0) c->shape.ld = shape->d_model;
  c->params = *params;
  c->plan = make_plan(&c->shape, params);
  c->stream = reinterpret_cast<hipStream_t>(hip_stream);
  auto cleanup = [&](int code) {
    spectral_destroy(c);
    return code;
  };
  if (hipGetDevice(&c->device) != hipSuccess) return cleanup(fail(SN_ESTATE, "no HIP device"));
  const size_t L = c->shape.n_layers;
  if (hipMalloc(&c->ws, c->plan.bytes) != hipSuccess) return cleanup(fail(SN_EHIP, "hipMalloc(workspace) failed"));
  if (hipMalloc(&c->d_tab, 2 * L * sizeof(void*)) != hipSuccess)
    return cleanup(fail(SN_EHIP, "hipMalloc(pointer table) failed"));
  if (hipHostMalloc(&c->h_tab, 2 * L * sizeof(void*), hipHostMallocDefault) != hipSuccess)
    return cleanup(fail(SN_EHIP, "hipHostMalloc(pointer table) failed"));
  if (hipHostMalloc(&c->h_alive, 2 * sizeof(int32_t), hipHostMallocDefault) != hipSuccess)
    return cleanup(fail(SN_EHIP, "hipHostMalloc failed"));
  if (hipEventCreateWithFlags(&c->tab_event, hipEventDisableTiming) != hipSuccess)
    return cleanup(fail(SN_EHIP, "hipEventCreate failed"));
  const Plan& pl = c->plan;
  c->w.zp = reinterpret_cast<float*>(c->ws + pl.off_zp);
  c->w.zn = reinterpret_cast<float*>(c->ws + pl.off_zn);
  c->w.yp = reinterpret_cast<float*>(c->ws + pl.off_yp);
  c->w.yn = reinterpret_cast<float*>(c->ws + pl.off_yn);
  c->w.sig = reinterpret_cast<float*>(c->ws + pl.off_sig);
  c->w.vnorm0 = reinterpret_cast<float*>(c->ws + pl.off_vn);
  c->w.alive = reinterpret_cast<int32_t*>(c->ws + pl.off_alive);
  c->w.n_alive = reinterpret_cast<int32_t*>(c->ws + pl.off_nalive);
  c->w.iters = reinterpret_cast<int32_t*>(c->ws + pl.off_iters);
  c->w.fin = pl.gram ? reinterpret_cast<float*>(c->ws + pl.off_fin) : nullptr;
  *ctx = c;
  return SN_OK;
}

SN_API int spectral_set_stream(sn_ctx* c, void* hip_stream) {
  if (!c) return fail(SN_ENULL, "ctx must not be NULL");
  c->stream = reinterpret_cast<hipStream_t>(hip_stream);
  return SN_OK;
}

SN_API void spectral_destroy(sn_ctx* c) {
  if (!c) return;
  if (c->stream || c->ws) (void)hipStreamSynchronize(c->stream);
  for (auto& r : c->recs) {
    if (r.a) (void)hipEventDestroy(r.a);
    if (r.b) (void)hipEventDestroy(r.b);
  }
  for (auto e : c->pool) (void)hipEventDestroy(e);
  if (c->tab_event) (void)hipEventDestroy(c->tab_event);
  if (c->h_alive) (void)hipHostFree(c->h_alive);
  if (c->h_tab) (void)hipHostFree(c->h_tab);
  if (c->d_tab) (void)hipFree(c->d_tab);
  if (c->ws) (void)hipFree(c->ws);
  delete c;
}

SN_API int spectral_profile(sn_ctx* c, int32_t enable) {
  if (!c) return fail(SN_ENULL, "ctx must not be NULL");
  c->prof = enable != 0;
  return SN_OK;
}

SN_API int spectral_profile_read(sn_ctx* c, double* ms, int64_t* launches) {
  if (!c || !ms || !launches) return fail(SN_ENULL, "ctx, ms and launches must not be NULL");
  for (int k = 0; k < KIND_N; ++k) {
    ms[k] = 0.0;
    launches[k] = 0;
  }
  SN_HIP(hipStreamSynchronize(c->stream));
  for (auto& r : c->recs) {
    float t = 0.f;
    SN_HIP(hipEventElapsedTime(&t, r.a, r.b));
    ms[r.kind] += t;
    launches[r.kind] += 1;
    c->pool.push_back(r.a);
    c->pool.push_back(r.b);
  }
  c->recs.clear();
  return SN_OK;
}

SN_API int spectral_step(sn_ctx* c, const void* const* wq_layers, const void* const* wk_layers, float* v,
                         float* u, int32_t n_iter, float* sigma, float* scale, int32_t* iters) {
  if (!c) return fail(SN_ENULL, "ctx must not be NULL");
  if (!wq_layers || !wk_layers || !v || !sigma || !scale)
    return fail(SN_ENULL, "wq_layers, wk_layers, v, sigma and scale must not be NULL");
  if (n_iter < 1) return fail(SN_EINVAL, "n_iter must be >= 1");
  const int L = c->shape.n_layers;
  int rc = update_table(c, wq_layers, wk_layers);
  if (rc != SN_OK) return rc;

  const Plan& pl = c->plan;
  SweepArgs a{};
  a.ld = c->shape.ld;
  a.d = c->shape.d_model;
  a.n_q = c->shape.n_q_heads;
  a.n_kv = c->shape.n_kv_heads;
  a.g = pl.g;
  a.H = pl.H;
  a.s_q = pl.s_q;
  a.s_k = pl.s_k;
  a.n_tiles = pl.n_tiles;
  a.nch = pl.nch;
  a.n_iter = n_iter;
  a.tol = c->params.tol;
  a.w = c->w;
  a.v = v;
  a.u = u;
  a.sigma = sigma;
  a.iters = iters ? iters : c->w.iters;

  rc = pl.gram ? run_gram(c, a, u) : run_chain(c, a, u);
  if (rc != SN_OK) return rc;

  FinArgs f{};
  f.H = pl.H;
  f.L = L;
  f.n_q = c->shape.n_q_heads;
  f.d = c->shape.d_model;
  f.s_k = pl.s_k;
  f.slot_fixed = pl.gram ? 0 : -1;
  f.coef = scale_coef(c);
  f.w = c->w;
  f.v = v;
  f.u = u;
  f.sigma = sigma;
  f.scale = scale;
  f.iters = a.iters;
  return timed(c, KIND_FIN, [&] { finalize_kernel<<<dim3(pl.H + L), kThreads, 0, c->stream>>>(f); });
}

SN_API int spectral_step_layer(sn_ctx* c, const void* const* wq_layers, const void* const* wk_layers, float* v,
                               float* u, int32_t n_iter, float* sigma, float* scale) {
  if (!c) return fail(SN_ENULL, "ctx must not be NULL");
  if (!wq_layers || !wk_layers || !v || !sigma || !scale)
    return fail(SN_ENULL, "wq_layers, wk_layers, v, sigma and scale must not be NULL");
  if (!c->plan.layer) return fail(SN_ESTATE, "the context was created without SN_FLAG_LAYER");
  if (n_iter < 1) return fail(SN_EINVAL, "n_iter must be >= 1");
  int rc = update_table(c, wq_layers, wk_layers);
  if (rc != SN_OK) return rc;
  const Plan& pl = c->plan;
  const int L = c->shape.n_layers;
  float* lz = reinterpret_cast<float*>(c->ws + pl.off_lz);
  float* ly = reinterpret_cast<float*>(c->ws + pl.off_ly);
  float* lcol = reinterpret_cast<float*>(c->ws + pl.off_lcol);
  float* lu = reinterpret_cast<float*>(c->ws + pl.off_lu);
  float* lv = reinterpret_cast<float*>(c->ws + pl.off_lv);
  float* n2_u = reinterpret_cast<float*>(c->ws + pl.off_ln2);
  float* n2_v = n2_u + L;
  // start vectors: copy, squared norms, layer status
  if ((rc = layer_reduce(c, v, 1, 0, lv, n2_v)) != SN_OK) return rc;
  for (int k = 1; k <= n_iter; ++k) {
    LayerArgs a{};
    a.xvec = lv;  // z_j = K_j v
    a.xn2 = n2_v;
    a.rowpart = lz;
    if ((rc = layer_sweep(c, false, LM_ROWS, a)) != SN_OK) return rc;
    a = LayerArgs{};  // c_h = Q_h^T z_{j(h)}: RepeatBlocks
    a.ypart = lz;
    a.y_units = c->shape.n_kv_heads;
    a.y_strips = pl.s_lk;
    a.y_div = pl.g;
    a.y_cnt = 1;
    a.colout = lcol;
    if ((rc = layer_sweep(c, true, LM_COLS, a)) != SN_OK) return rc;
    if ((rc = layer_reduce(c, lcol, c->shape.n_q_heads, 1, lu, n2_u)) != SN_OK) return rc;
    a = LayerArgs{};  // y_h = Q_h u
    a.xvec = lu;
    a.xn2 = n2_u;
    a.rowpart = ly;
    if ((rc = layer_sweep(c, true, LM_ROWS, a)) != SN_OK) return rc;
    a = LayerArgs{};  // c_j = K_j^T sum_{h in j} y_h: SumGroups
    a.ypart = ly;
    a.y_units = c->shape.n_q_heads;
    a.y_strips = pl.s_lq;
    a.y_div = 1;
    a.y_cnt = pl.g;
    a.colout = lcol;
    if ((rc = layer_sweep(c, false, LM_COLS, a)) != SN_OK) return rc;
    if ((rc = layer_reduce(c, lcol, c->shape.n_kv_heads, 2, lv, n2_v)) != SN_OK) return rc;
  }
  LayerFinArgs f{};
  f.d = c->shape.d_model;
  f.L = L;
  f.coef = scale_coef(c);
  f.lstat = reinterpret_cast<const int32_t*>(c->ws + pl.off_lstat);
  f.lu = lu;
  f.lv = lv;
  f.n2_u = n2_u;
  f.n2_v = n2_v;
  f.n2_start = n2_u + 2 * L;
  f.v = v;
  f.u = u;
  f.sigma = sigma;
  f.scale = scale;
  return timed(c, KIND_LRED, [&] { layer_finalize_kernel<<<dim3(L), kThreads, 0, c->stream>>>(f); });
}

SN_API int spectral_logits_workspace_bytes(const sn_shape* shape, int32_t seq_len, int64_t* bytes) {
  if (!shape || !bytes) return fail(SN_ENULL, "shape and bytes must not be NULL");
  if (seq_len < 1) return fail(SN_EINVAL, "seq_len must be >= 1");
  *bytes = sn_logits_workspace_bytes(seq_len, (int64_t)shape->n_q_heads * shape->head_dim,
                                     (int64_t)shape->n_kv_heads * shape->head_dim);
  return SN_OK;
}

SN_API int spectral_logits_fp8(sn_ctx* c, const void* const* x_layers, int64_t ld_x, int32_t seq_len,
                               const void* const* wq_layers, const void* const* wk_layers, const float* scale,
                               void* workspace, int64_t workspace_bytes, uint8_t* codes, float* max_abs,
                               int32_t* n_over) {
  if (!c) return fail(SN_ENULL, "ctx must not be NULL");
  if (!x_layers || !wq_layers || !wk_layers || !scale || !workspace || !max_abs || !n_over)
    return fail(SN_ENULL, "x_layers, wq_layers, wk_layers, scale, workspace, max_abs and n_over must not be NULL");
  const sn_shape& sh = c->shape;
  if (sh.dtype != SN_BF16) return fail(SN_EDTYPE, "the logit consumer needs bf16 weights and tokens");
  const int dh = sh.head_dim;
  if (dh != 16 && dh != 32 && dh != 64 && dh != 128)
    return fail(SN_EINVAL, "the logit consumer needs head_dim 16, 32, 64 or 128");
  if (seq_len < 1 || seq_len > 46340) return fail(SN_EINVAL, "seq_len must be in [1, 46340]");
  if (ld_x == 0) ld_x = sh.d_model;
  if (ld_x < sh.d_model || (ld_x * 2) % 16 != 0) return fail(SN_EINVAL, "ld_x must be >= d_model, 8-element aligned");
  const int64_t nq_cols = (int64_t)sh.n_q_heads * dh, nk_cols = (int64_t)sh.n_kv_heads * dh;
  if ((int64_t)seq_len * ld_x * 2 >= (int64_t(1) << 31) || (int64_t)seq_len * nq_cols * 2 >= (int64_t(1) << 31))
    return fail(SN_EINVAL, "seq_len x row bytes must stay below 2^31");
  const int64_t need = sn_logits_workspace_bytes(seq_len, nq_cols, nk_cols);
  if (workspace_bytes < need) return fail(SN_EINVAL, "workspace too small (spectral_logits_workspace_bytes)");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) || (reinterpret_cast<uintptr_t>(codes) & 15))
    return fail(SN_EINVAL, "workspace must be 256-byte and codes 16-byte aligned");
  const int L = sh.n_layers;
  for (int l = 0; l < L; ++l) {
    if (!x_layers[l] || !wq_layers[l] || !wk_layers[l]) return fail(SN_ENULL, "a layer pointer is NULL");
    if ((reinterpret_cast<uintptr_t>(x_layers[l]) | reinterpret_cast<uintptr_t>(wq_layers[l]) |
         reinterpret_cast<uintptr_t>(wk_layers[l])) & 15)
      return fail(SN_EINVAL, "layer pointers must be 16-byte aligned");
  }
  int cur_dev = 0;
  SN_HIP(hipGetDevice(&cur_dev));
  if (cur_dev != c->device) return fail(SN_ESTATE, "the current HIP device is not the context's device");

  uint16_t* ws = reinterpret_cast<uint16_t*>(workspace);
  ProjArgs p{};
  p.ld_x = ld_x;
  p.ld_w = sh.ld;
  p.seq = seq_len;
  p.d = sh.d_model;
  p.nq_cols = (int32_t)nq_cols;
  p.nk_cols = (int32_t)nk_cols;
  p.tiles_m = ceil_div(seq_len, 128);
  p.tiles_nq = ceil_div(nq_cols, 128);
  p.tiles_nk = ceil_div(nk_cols, 128);
  p.qh = ws;
  p.ql = ws + (size_t)seq_len * nq_cols;
  p.kh = ws + (size_t)2 * seq_len * nq_cols;
  p.kl = p.kh + (size_t)seq_len * nk_cols;
  LogitArgs g{};
  g.qh = p.qh;
  g.ql = p.ql;
  g.kh = p.kh;
  g.kl = p.kl;
  g.seq = seq_len;
  g.g = c->plan.g;
  g.nq_cols = (int32_t)nq_cols;
  g.nk_cols = (int32_t)nk_cols;
  g.tiles = ceil_div(seq_len, 128);
  g.scale = scale;
  int rc = timed(c, KIND_LOGITS, [&] { sn_launch_zero_stats(max_abs, n_over, L * sh.n_q_heads, c->stream); });
  if (rc != SN_OK) return rc;
  for (int l = 0; l < L; ++l) {
    p.x = reinterpret_cast<const uint16_t*>(x_layers[l]);
    p.wq = reinterpret_cast<const uint16_t*>(wq_layers[l]);
    p.wk = reinterpret_cast<const uint16_t*>(wk_layers[l]);
    if ((rc = timed(c, KIND_PROJ, [&] { sn_launch_proj(p, c->stream); })) != SN_OK) return rc;
    g.layer = l;
    g.codes = codes ? codes + (size_t)l * sh.n_q_heads * seq_len * seq_len : nullptr;
    g.max_abs = max_abs + (size_t)l * sh.n_q_heads;
    g.n_over = n_over + (size_t)l * sh.n_q_heads;
    if ((rc = timed(c, KIND_LOGITS, [&] { sn_launch_logits(g, dh, sh.n_q_heads, c->stream); })) != SN_OK)
      return rc;
  }
  return SN_OK;
}

}  // extern "C"
