// C ABI of the per-head spectral-norm estimator and the per-layer FP8 E4M3
// scale factor for MI355X (gfx950): validation, workspace plan, context and
// the entry points of include/spectral.h.  The kernels live in sweeps.hip
// (the default form), gram.hip (SN_FLAG_GRAM), layer_form.hip
// (spectral_step_layer) and logits_fp8.hip (spectral_logits_fp8).
//
// Method (arXiv 2602.18851, Sec. 4.1-4.2, App. E): for query head h with key
// head j = floor(h / g), one step is
//     z = K_j v,  u' = Q_h^T z (= M v),  sigma = ||u'||,
//     y = Q_h u' / sigma,  v' = K_j^T y (= M^T u),  v = v' / ||v'||,
// where Q_h, K_j are the d_h x d row blocks of the PyTorch-layout weights
// (the transposes of the paper's W^Q_h, W^K_j) and M = Q_h^T K_j is never
// formed.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "logits_fp8.h"
#include "spectral.h"

namespace {

using namespace sn;

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

enum {
  KIND_INIT = 0, KIND_Q = 1, KIND_K = 2, KIND_FIN = 3, KIND_GRAM = 4, KIND_ITER = 5, KIND_EMIT = 6,
  KIND_LROWS = 7, KIND_LCOLS = 8, KIND_LRED = 9, KIND_PROJ = 10, KIND_LOGITS = 11, KIND_TAIL = 12, KIND_N = 13
};
static_assert(KIND_N == SN_PROFILE_KINDS, "profile kinds");

// ------------------------------------------------------------------ host side

struct Plan {
  int H, g, gc, nch, vec, tile_c, n_tiles;   // W_K sweeps
  int tile_cq, n_tiles_q;                    // W_Q sweep
  bool mfma_k;  // W_K sweeps on the matrix cores
  int s_q, tps_q, s_k, tps_k;
  bool tail;    // tolerance mode of the default form: the heads still running after the first
                // steps are finished in d_h-space (needs d_h >= 16)
  int s_tmax;   // most strips of the tail's final W_K sweep
  bool gram;    // Gram form
  int units_g, s_g, tps_g, n_tiles_g, nb_g;
  int g_items;  // Gram partial items the workspace holds
  bool layer;   // layer-level form
  int s_lq, tps_lq, s_lk, tps_lk;  // strips of the layer-form row sweeps over W_Q and W_K
  int rs_q, rbp_q, rs_k, rbp_k;    // row splits (and row blocks per split) of its column sweeps
  size_t off_zp, off_zn, off_yp, off_yn, off_sig, off_vn, off_alive, off_iters, off_fin, off_gp;
  size_t off_lz, off_ly, off_lvin, off_lcol, off_lu, off_lv, off_ln2, off_ln2p, off_lstat;
  size_t off_zs, off_lg, off_lk, off_kvpos, off_ctl, off_zt;
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

// Row stride of the layer form's per-unit column sums: whole 64-column tiles.
int col_stride(int d) { return ceil_div(d, 64) * 64; }

// Column strips per unit (head or KV head): the request if given, else about
// target / units (rounded up, or down when all waves should be resident at
// once), with at least kMinTilesPerStrip tiles per strip so that a wave's
// stream outweighs its prologue (which sums one partial per producer strip).
void strips(int n_tiles, int64_t units, int requested, int target, bool round_down, int* s_out, int* tps_out,
            int min_tiles = kMinTilesPerStrip) {
  const int64_t u = std::max<int64_t>(units, 1);
  int s = requested > 0 ? requested : round_down ? (int)std::max<int64_t>(1, target / u) : ceil_div(target, u);
  if (requested <= 0) s = std::min(s, std::max(1, n_tiles / min_tiles));
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
  // Tolerance mode: after the first kTailSteps steps, the heads still running
  // are listed on the device and finished in d_h-space through their Gram
  // matrices, formed for the listed heads only; strips of those launches are
  // chosen on the device for the listed count (at most max(count, target)
  // items each).
  pl.tail = p->tol > 0.f && !pl.gram && dh >= 16;
  pl.s_tmax = std::max(1, pl.n_tiles / kTailMinTiles);
  if (pl.gram || pl.tail) {
    const int rb = dh / 16;
    pl.nb_g = rb * (rb + 1) / 2;
    pl.units_g = pl.H + s->n_layers * s->n_kv_heads;
    pl.n_tiles_g = ceil_div((int64_t)s->d_model * esize(s->dtype), 128);
    strips(pl.n_tiles_g, pl.units_g, 0, kGTargetItems, true, &pl.s_g, &pl.tps_g);
    pl.g_items = pl.gram ? pl.units_g * pl.s_g : std::max(pl.units_g, kGTargetItems);
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
  pl.off_iters = take(H * 4);
  if (pl.tail) {
    const size_t nkvh = (size_t)s->n_layers * s->n_kv_heads;
    pl.off_zs = take(H * 4);
    pl.off_lg = take((H + nkvh) * 4);
    pl.off_lk = take(nkvh * pl.nch * 4);
    pl.off_kvpos = take(nkvh * 4);
    pl.off_ctl = take(TC_WORDS * 4);
    pl.off_zt = take(H * pl.s_tmax * 4);
  }
  if (pl.gram || pl.tail) {
    pl.off_fin = take(H * 2 * dh * 4);
    pl.off_gp = take((size_t)pl.g_items * pl.nb_g * 256 * 4);
  }
  pl.layer = (p->flags & SN_FLAG_LAYER) != 0;
  if (pl.layer) {
    const size_t L = s->n_layers, Hk = L * s->n_kv_heads, d = s->d_model;
    strips(pl.n_tiles_q, pl.H, 0, kQTargetItems, false, &pl.s_lq, &pl.tps_lq);
    strips(pl.n_tiles_q, (int64_t)Hk, 0, kQTargetItems, false, &pl.s_lk, &pl.tps_lk);
    pl.off_lz = take(Hk * pl.s_lk * dh * 4);
    pl.off_ly = take(H * pl.s_lq * dh * 4);
    // column sweeps: one wave per column tile and row split; rows are split
    // only as far as needed for about kQTargetItems waves
    auto rsplit = [&](int nrb, int* n_split, int* per) {
      const int64_t base = (int64_t)L * pl.n_tiles_q;
      const int want = (int)std::min<int64_t>(nrb, std::max<int64_t>(1, (kQTargetItems + base - 1) / base));
      *per = ceil_div(nrb, want);
      *n_split = ceil_div(nrb, *per);
    };
    rsplit(s->n_q_heads, &pl.rs_q, &pl.rbp_q);
    rsplit(s->n_kv_heads, &pl.rs_k, &pl.rbp_k);
    pl.off_lvin = take(H * dh * 4);
    pl.off_lcol = take(L * (size_t)std::max(pl.rs_q, pl.rs_k) * col_stride(s->d_model) * 4);
    pl.off_lu = take(L * d * 4);
    pl.off_lv = take(L * d * 4);
    pl.off_ln2 = take(3 * L * 4);
    pl.off_ln2p = take(L * (size_t)ceil_div(d, kRedThreads) * 4);
    pl.off_lstat = take(L * 4);
  }
  pl.bytes = off;
  return pl;
}

struct ProfRec {
  int kind;
  hipEvent_t a, b;
};

// Device pointer tables are written by a kernel whose arguments carry the
// pointers: the values are taken when the launch is queued (or captured),
// with no host buffer that must outlive the call.
constexpr int kTabChunk = 256;
struct TabFill {
  const void* p[kTabChunk];
  const void** dst;
  int32_t n;
};

__global__ void table_fill_kernel(TabFill f) {
  const int i = threadIdx.x;
  if (i < f.n) f.dst[i] = f.p[i];
}

// dst[0 .. n) = src(0 .. n), in launches of up to kTabChunk pointers.
template <typename Src>
int fill_table(const void** dst, int n, Src src, hipStream_t st) {
  for (int i0 = 0; i0 < n; i0 += kTabChunk) {
    TabFill f{};
    f.dst = dst + i0;
    f.n = std::min(kTabChunk, n - i0);
    for (int i = 0; i < f.n; ++i) f.p[i] = src(i0 + i);
    table_fill_kernel<<<dim3(1), kTabChunk, 0, st>>>(f);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(SN_EHIP, std::string("table fill launch failed: ") + hipGetErrorString(e));
  }
  return SN_OK;
}

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
  bool owns_ws = true;
  Work w{};
  const void** d_tab = nullptr;  // device [2][2L]: the eager table, then the table of captured calls
  const void** tab = nullptr;    // the table the current call's launches read
  bool cache_table = true;       // eager calls skip the table write when the pointers did not change
  std::vector<const void*> cached;  // pointers in the eager table
  hipEvent_t tab_event = nullptr;
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

// Compacted launch of the tolerance-mode tail over the entries of `list`
// (query heads for a W_Q sweep, W_K units otherwise); the count and strips
// are read from `ctl` on the device, and the grid holds max_items items.
struct TailLaunch {
  const int32_t* list = nullptr;
  const int32_t* ctl = nullptr;
  int max_items = 0;
};

int run_sweep(sn_ctx* c, int ph, SweepArgs a, const TailLaunch& tl = TailLaunch{}) {
  a.ctl = tl.ctl;
  const Plan& pl = c->plan;
  const int n_units = c->shape.n_layers * c->shape.n_kv_heads * pl.nch;
  if (ph == PH_Q || ph == PH_EQ) {
    a.mats = c->tab;
    a.s_out = pl.s_q;
    a.tps = pl.tps_q;
    a.n_tiles = pl.n_tiles_q;
    a.n_items = pl.H * pl.s_q;
  } else {
    a.mats = c->tab + c->shape.n_layers;
    a.s_out = pl.s_k;
    a.tps = pl.tps_k;
    a.n_tiles = pl.n_tiles;
    a.n_items = n_units * pl.s_k;
  }
  if (tl.list) {
    a.list = tl.list;
    a.n_items = tl.max_items;
  }
  const int kind = ph == PH_INIT ? KIND_INIT : ph == PH_Q ? KIND_Q : ph == PH_K ? KIND_K : KIND_EMIT;
  return timed(c, kind, [&] {
    launch_sweep(c->shape.dtype == SN_BF16, c->shape.head_dim, ph, pl.gc, pl.mfma_k, a.n_items, c->stream, a);
  });
}


// Eq. "scale" per unit of sigma: alpha * d / sqrt(d_h) / (eta_fp8 * r_max), in double.
float scale_coef(const sn_ctx* c) {
  return (float)((double)c->params.alpha * (double)c->shape.d_model /
                 (std::sqrt((double)c->shape.head_dim) * (double)c->params.eta_fp8 * (double)c->params.r_max));
}

bool capturing(hipStream_t st) {
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  return hipStreamIsCapturing(st, &cap) == hipSuccess && cap != hipStreamCaptureStatusNone;
}

// Checks the layer pointers and the device, and points the call's launches
// at a device table of the per-layer pointers.  Eager calls share one table,
// rewritten only when the pointers change.  A call being captured into a
// graph always writes its pointers into a second table, so that every replay
// restores its own pointers whatever eager calls ran in between (graphs
// captured from one context must therefore not replay concurrently).
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
  auto src = [&](int i) { return i < L ? wq_layers[i] : wk_layers[i - L]; };
  if (capturing(c->stream)) {
    c->tab = c->d_tab + 2 * L;
    return fill_table(c->tab, 2 * L, src, c->stream);
  }
  c->tab = c->d_tab;
  if (!c->cache_table) return fill_table(c->tab, 2 * L, src, c->stream);
  bool same = c->cached.size() == (size_t)(2 * L);
  for (int l = 0; same && l < L; ++l)
    same = c->cached[l] == wq_layers[l] && c->cached[L + l] == wk_layers[l];
  if (!same) {
    int rc = fill_table(c->tab, 2 * L, src, c->stream);
    if (rc != SN_OK) return rc;
    c->cached.assign(wq_layers, wq_layers + L);
    c->cached.insert(c->cached.end(), wk_layers, wk_layers + L);
    if (c->tab_event) SN_HIP(hipEventRecord(c->tab_event, c->stream));
  }
  return SN_OK;
}


// One layer-form sweep over W_Q (q = true) or W_K.
int layer_sweep(sn_ctx* c, bool q, int mode, LayerArgs a) {
  const Plan& pl = c->plan;
  const int L = c->shape.n_layers;
  a.mats = c->tab + (q ? 0 : L);
  a.ld = c->shape.ld;
  a.d = c->shape.d_model;
  a.n_tiles = pl.n_tiles_q;
  a.lstat = reinterpret_cast<const int32_t*>(c->ws + pl.off_lstat);
  if (mode == LM_ROWS) {
    a.units = q ? c->shape.n_q_heads : c->shape.n_kv_heads;
    a.s_out = q ? pl.s_lq : pl.s_lk;
    a.tps = q ? pl.tps_lq : pl.tps_lk;
    a.n_items = L * a.units * a.s_out;
  } else {
    a.nrb = q ? c->shape.n_q_heads : c->shape.n_kv_heads;
    a.n_rsplit = q ? pl.rs_q : pl.rs_k;
    a.rb_per = q ? pl.rbp_q : pl.rbp_k;
    a.cstride = col_stride(c->shape.d_model);
    a.n_items = L * a.n_rsplit * a.n_tiles;
  }
  return timed(c, mode == LM_ROWS ? KIND_LROWS : KIND_LCOLS, [&] {
    launch_layer_sweep(c->shape.dtype == SN_BF16, c->shape.head_dim, mode, a.n_items, c->stream, a);
  });
}

// vin of a column sweep from the previous row sweep's partials.
int layer_vin(sn_ctx* c, const float* part, int src_units, int strips, int div, int cnt, int nrb) {
  const Plan& pl = c->plan;
  LayerVinArgs v{};
  v.part = part;
  v.src_units = src_units;
  v.strips = strips;
  v.div = div;
  v.cnt = cnt;
  v.nrb = nrb;
  v.dh = c->shape.head_dim;
  v.lstat = reinterpret_cast<const int32_t*>(c->ws + pl.off_lstat);
  v.vin = reinterpret_cast<float*>(c->ws + pl.off_lvin);
  return timed(c, KIND_LRED, [&] { launch_layer_vin(c->shape.n_layers, c->stream, v); });
}

int layer_reduce(sn_ctx* c, const float* col, int units, int cstride, int mode, float* vec, float* n2) {
  const Plan& pl = c->plan;
  LayerReduceArgs r{};
  r.col = col;
  r.units = units;
  r.d = c->shape.d_model;
  r.cstride = cstride;
  r.mode = mode;
  r.vec = vec;
  r.n2 = n2;
  r.nb = ceil_div(c->shape.d_model, kRedThreads);
  r.n2part = reinterpret_cast<float*>(c->ws + pl.off_ln2p);
  r.n2_start = reinterpret_cast<float*>(c->ws + pl.off_ln2) + 2 * c->shape.n_layers;
  r.lstat = reinterpret_cast<int32_t*>(c->ws + pl.off_lstat);
  return timed(c, KIND_LRED,
               [&] { launch_layer_reduce(c->shape.n_layers, c->stream, r); });
}

GramArgs gram_args(const sn_ctx* c) {
  const Plan& pl = c->plan;
  GramArgs g{};
  g.mats = c->tab;
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
  return g;
}

IterArgs iter_args(const sn_ctx* c, const SweepArgs& a) {
  const Plan& pl = c->plan;
  IterArgs it{};
  it.H = pl.H;
  it.n_q = c->shape.n_q_heads;
  it.n_kv = c->shape.n_kv_heads;
  it.g = pl.g;
  it.s_k = pl.s_k;
  it.s_g = pl.s_g;
  it.n_iter = a.n_iter;
  it.tol = a.tol;
  it.gp = reinterpret_cast<const float*>(c->ws + pl.off_gp);
  it.w = c->w;
  it.sigma = a.sigma;
  it.iters = a.iters;
  return it;
}

// Tolerance-mode tail after step k0 of the chain, as a fixed sequence of
// launches whatever the heads do: list the heads still running (and their
// key heads and W_K units), form the Gram matrices of the listed heads only,
// iterate each listed head in d_h-space to the tolerance or the cap, then map
// its last vectors back to v (and u) with final sweeps over the lists.  The
// iterates are those the sweep chain would compute (see gram.hip); nothing is
// read back to the host.
int run_tail(sn_ctx* c, SweepArgs a, float* u, int k0) {
  const Plan& pl = c->plan;
  const int n_units = c->shape.n_layers * c->shape.n_kv_heads * pl.nch;
  const int target_k = pl.mfma_k ? kKMfmaResident : kKTargetItems;
  TailPlan tp{pl.n_tiles_g, pl.n_tiles, pl.n_tiles_q, kGTargetItems, target_k, kQTargetItems};
  int rc = timed(c, KIND_TAIL, [&] { launch_tail_lists(a, k0 & 1, pl.gc, n_units, tp, c->stream); });
  if (rc != SN_OK) return rc;

  GramArgs g = gram_args(c);
  g.list = c->w.list_g;
  g.ctl = c->w.ctl;
  g.n_items = pl.g_items;  // grid: at most max(listed units, target) items
  const int dh = c->shape.head_dim;
  rc = timed(c, KIND_GRAM, [&] { launch_gram(c->shape.dtype == SN_BF16, dh, g.n_items, c->stream, g); });
  if (rc != SN_OK) return rc;

  IterArgs it = iter_args(c, a);
  it.k0 = k0;
  it.list = c->w.list_g;
  it.ctl = c->w.ctl;
  it.kvpos = c->w.kvpos;
  rc = timed(c, KIND_ITER, [&] { launch_gram_iterate(dh, pl.H, c->stream, it); });
  if (rc != SN_OK) return rc;

  SweepArgs e = a;
  e.k = 0;
  e.only = c->w.alive + (size_t)(k0 & 1) * pl.H;  // the heads running after step k0
  e.w.zn = c->w.zt;
  TailLaunch tk{c->w.list_k, c->w.ctl + TC_EK, std::max(n_units, target_k)};
  if ((rc = run_sweep(c, PH_EK, e, tk)) != SN_OK) return rc;
  if (u) {
    TailLaunch tq{c->w.list_g, c->w.ctl + TC_EQ, std::max(pl.H, kQTargetItems)};
    if ((rc = run_sweep(c, PH_EQ, e, tq)) != SN_OK) return rc;
  }
  return SN_OK;
}

// The sweeps of the default form: first W_K sweep, then n_iter x (W_Q sweep,
// W_K sweep).  In tolerance mode every W_K sweep decides, per head, whether
// the step's sigma meets the rule; a stopped head's waves leave at set-up in
// the later sweeps.  With d_h >= 16 only the first kTailSteps steps run as
// full sweeps and the tail finishes the rest (run_tail).  Nothing waits on
// the host.
int run_chain(sn_ctx* c, SweepArgs a, float* u) {
  const Plan& pl = c->plan;
  int rc;
  a.k = 0;
  if ((rc = run_sweep(c, PH_INIT, a)) != SN_OK) return rc;
  const int k_full = pl.tail ? std::min(a.n_iter, kTailSteps) : a.n_iter;
  for (int k = 1; k <= k_full; ++k) {
    a.k = k;
    a.want_vec = (u != nullptr) && (c->params.tol > 0.f || k == a.n_iter);
    if ((rc = run_sweep(c, PH_Q, a)) != SN_OK) return rc;
    a.want_vec = 0;
    if ((rc = run_sweep(c, PH_K, a)) != SN_OK) return rc;
  }
  if (pl.tail && a.n_iter > k_full) return run_tail(c, a, u, k_full);
  return SN_OK;
}

// The Gram form of one call: first W_K sweep, Gram sweep, d_h-space
// iteration, final W_K sweep (and W_Q sweep for u).
int run_gram(sn_ctx* c, SweepArgs a, float* u) {
  const Plan& pl = c->plan;
  int rc;
  a.k = 0;
  if ((rc = run_sweep(c, PH_INIT, a)) != SN_OK) return rc;
  GramArgs g = gram_args(c);
  const int dh = c->shape.head_dim;
  rc = timed(c, KIND_GRAM, [&] { launch_gram(c->shape.dtype == SN_BF16, dh, g.n_items, c->stream, g); });
  if (rc != SN_OK) return rc;
  IterArgs it = iter_args(c, a);
  rc = timed(c, KIND_ITER, [&] { launch_gram_iterate(dh, pl.H, c->stream, it); });
  if (rc != SN_OK) return rc;
  a.k = 0;  // the final sweeps write their ||v'||^2 partials to slot 0
  if ((rc = run_sweep(c, PH_EK, a)) != SN_OK) return rc;
  if (u && (rc = run_sweep(c, PH_EQ, a)) != SN_OK) return rc;
  return SN_OK;
}

// Views of the workspace of a plan.
void bind_workspace(sn_ctx* c) {
  const Plan& pl = c->plan;
  char* ws = c->ws;
  c->w = Work{};
  c->w.zp = reinterpret_cast<float*>(ws + pl.off_zp);
  c->w.zn = reinterpret_cast<float*>(ws + pl.off_zn);
  c->w.yp = reinterpret_cast<float*>(ws + pl.off_yp);
  c->w.yn = reinterpret_cast<float*>(ws + pl.off_yn);
  c->w.sig = reinterpret_cast<float*>(ws + pl.off_sig);
  c->w.vnorm0 = reinterpret_cast<float*>(ws + pl.off_vn);
  c->w.alive = reinterpret_cast<int32_t*>(ws + pl.off_alive);
  c->w.iters = reinterpret_cast<int32_t*>(ws + pl.off_iters);
  if (pl.gram || pl.tail) c->w.fin = reinterpret_cast<float*>(ws + pl.off_fin);
  if (pl.tail) {
    c->w.zs = reinterpret_cast<int32_t*>(ws + pl.off_zs);
    c->w.list_g = reinterpret_cast<int32_t*>(ws + pl.off_lg);
    c->w.list_k = reinterpret_cast<int32_t*>(ws + pl.off_lk);
    c->w.kvpos = reinterpret_cast<int32_t*>(ws + pl.off_kvpos);
    c->w.ctl = reinterpret_cast<int32_t*>(ws + pl.off_ctl);
    c->w.zt = reinterpret_cast<float*>(ws + pl.off_zt);
  }
}

// One spectral_step call on a bound context (table already in place).
int step_body(sn_ctx* c, float* v, float* u, int32_t n_iter, float* sigma, float* scale, int32_t* iters) {
  const Plan& pl = c->plan;
  const int L = c->shape.n_layers;
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

  int rc = pl.gram ? run_gram(c, a, u) : run_chain(c, a, u);
  if (rc != SN_OK) return rc;

  const bool tail_ran = pl.tail && n_iter > kTailSteps;
  FinArgs f{};
  f.H = pl.H;
  f.L = L;
  f.n_q = c->shape.n_q_heads;
  f.d = c->shape.d_model;
  f.s_k = pl.s_k;
  f.slot_fixed = pl.gram ? 0 : -1;
  f.zs = pl.tail ? c->w.zs : nullptr;
  f.tail = tail_ran ? c->w.alive + (size_t)(kTailSteps & 1) * pl.H : nullptr;
  f.zt = c->w.zt;
  f.coef = scale_coef(c);
  f.w = c->w;
  f.v = v;
  f.u = u;
  f.sigma = sigma;
  f.scale = scale;
  f.iters = a.iters;
  return timed(c, KIND_FIN, [&] { launch_finalize(pl.H + L, c->stream, f); });
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
  if (hipMalloc(&c->d_tab, 4 * L * sizeof(void*)) != hipSuccess)
    return cleanup(fail(SN_EHIP, "hipMalloc(pointer table) failed"));
  if (hipEventCreateWithFlags(&c->tab_event, hipEventDisableTiming) != hipSuccess)
    return cleanup(fail(SN_EHIP, "hipEventCreate failed"));
  c->tab = c->d_tab;
  bind_workspace(c);
  *ctx = c;
  return SN_OK;
}

SN_API int spectral_set_stream(sn_ctx* c, void* hip_stream) {
  if (!c) return fail(SN_ENULL, "ctx must not be NULL");
  hipStream_t st = reinterpret_cast<hipStream_t>(hip_stream);
  // later launches share the workspace and the eager pointer table with the
  // work queued on the previous stream: order the new stream after all of it
  // (a stream being captured into a graph cannot wait on an outside event;
  // its launches run at replay)
  if (st != c->stream && !capturing(st) && !capturing(c->stream)) {
    SN_HIP(hipEventRecord(c->tab_event, c->stream));
    SN_HIP(hipStreamWaitEvent(st, c->tab_event, 0));
  }
  c->stream = st;
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
  if (c->owns_ws && c->d_tab) (void)hipFree(c->d_tab);
  if (c->owns_ws && c->ws) (void)hipFree(c->ws);
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
  const int rc = update_table(c, wq_layers, wk_layers);
  if (rc != SN_OK) return rc;
  return step_body(c, v, u, n_iter, sigma, scale, iters);
}

}  // extern "C"

// ---- the allocation-free variant of spectral_step
//
// Its workspace and pointer table live in `scratch`, a static device array of
// kScratchBytes that each device holds from the library's first use on it
// until the process ends.  Host code reaches a device's copy only through the
// address hipGetSymbolAddress returns on that device (the array's name in
// host code is a host-side stand-in), kept per device here.  Nothing in the
// workspace must start at zero: every buffer a kernel reads was written
// earlier in the same call (the running flags by the first sweep, partials
// by their producer sweep, the tail's lists and control block by its list
// kernel).
namespace {

constexpr size_t kScratchBytes = size_t(32) << 20;
constexpr int kMaxDevices = 64;

static __device__ __attribute__((aligned(256))) uint8_t scratch[kScratchBytes];

std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's scratch (the current device), looked up
// once per device.
int scratch_on_device(int dev, char** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(SN_ESTATE, "device ordinal beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    SN_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(SN_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return SN_OK;
}

}  // namespace

extern "C" {

SN_API int spectral_step_noalloc(const sn_shape* shape, const sn_params* params, const void* const* wq_layers,
                                 const void* const* wk_layers, float* v, float* u, int32_t n_iter, float* sigma,
                                 float* scale, int32_t* iters, void* hip_stream) {
  if (!wq_layers || !wk_layers || !v || !sigma || !scale)
    return fail(SN_ENULL, "wq_layers, wk_layers, v, sigma and scale must not be NULL");
  int rc = validate(shape, params);
  if (rc != SN_OK) return rc;
  if (n_iter < 1) return fail(SN_EINVAL, "n_iter must be >= 1");
  sn_ctx c;
  c.shape = *shape;
  if (c.shape.ld == 0) c.shape.ld = shape->d_model;
  c.params = *params;
  c.params.flags &= ~SN_FLAG_LAYER;  // only reserves space for spectral_step_layer
  c.plan = make_plan(&c.shape, &c.params);
  const int L = c.shape.n_layers;
  const size_t tab_bytes = ((size_t)4 * L * sizeof(void*) + 255) & ~size_t(255);
  const size_t need = tab_bytes + c.plan.bytes;
  if (need > kScratchBytes)
    return fail(SN_EINVAL, "this shape needs " + std::to_string(need) + " bytes of scratch; spectral_step_noalloc " +
                               "holds at most " + std::to_string(kScratchBytes) + " (use spectral_init / spectral_step)");
  SN_HIP(hipGetDevice(&c.device));
  char* base = nullptr;
  if ((rc = scratch_on_device(c.device, &base)) != SN_OK) return rc;
  c.stream = reinterpret_cast<hipStream_t>(hip_stream);
  c.owns_ws = false;
  c.cache_table = false;
  c.d_tab = reinterpret_cast<const void**>(base);
  c.ws = base + tab_bytes;
  bind_workspace(&c);
  if ((rc = update_table(&c, wq_layers, wk_layers)) != SN_OK) return rc;
  return step_body(&c, v, u, n_iter, sigma, scale, iters);
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
  float* lvin = reinterpret_cast<float*>(c->ws + pl.off_lvin);
  float* lu = reinterpret_cast<float*>(c->ws + pl.off_lu);
  float* lv = reinterpret_cast<float*>(c->ws + pl.off_lv);
  float* n2_u = reinterpret_cast<float*>(c->ws + pl.off_ln2);
  float* n2_v = n2_u + L;
  // start vectors: copy, squared norms, layer status
  if ((rc = layer_reduce(c, v, 1, c->shape.d_model, 0, lv, n2_v)) != SN_OK) return rc;
  for (int k = 1; k <= n_iter; ++k) {
    LayerArgs a{};
    a.xvec = lv;  // z_j = K_j v
    a.xn2 = n2_v;
    a.rowpart = lz;
    if ((rc = layer_sweep(c, false, LM_ROWS, a)) != SN_OK) return rc;
    // u' = sum_h Q_h^T z_j(h): RepeatBlocks, then one column sweep over W_Q
    if ((rc = layer_vin(c, lz, c->shape.n_kv_heads, pl.s_lk, pl.g, 1, c->shape.n_q_heads)) != SN_OK) return rc;
    a = LayerArgs{};
    a.vin = lvin;
    a.colout = lcol;
    if ((rc = layer_sweep(c, true, LM_COLS, a)) != SN_OK) return rc;
    if ((rc = layer_reduce(c, lcol, pl.rs_q, col_stride(c->shape.d_model), 1, lu, n2_u)) != SN_OK) return rc;
    a = LayerArgs{};  // y_h = Q_h u
    a.xvec = lu;
    a.xn2 = n2_u;
    a.rowpart = ly;
    if ((rc = layer_sweep(c, true, LM_ROWS, a)) != SN_OK) return rc;
    // v' = sum_j K_j^T sum_{h in j} y_h: SumGroups, then one column sweep over W_K
    if ((rc = layer_vin(c, ly, c->shape.n_q_heads, pl.s_lq, 1, pl.g, c->shape.n_kv_heads)) != SN_OK) return rc;
    a = LayerArgs{};
    a.vin = lvin;
    a.colout = lcol;
    if ((rc = layer_sweep(c, false, LM_COLS, a)) != SN_OK) return rc;
    if ((rc = layer_reduce(c, lcol, pl.rs_k, col_stride(c->shape.d_model), 2, lv, n2_v)) != SN_OK) return rc;
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
  return timed(c, KIND_LRED, [&] { launch_layer_finalize(L, c->stream, f); });
}

SN_API int spectral_logits_workspace_bytes(const sn_shape* shape, int32_t seq_len, int64_t* bytes) {
  if (!shape || !bytes) return fail(SN_ENULL, "shape and bytes must not be NULL");
  if (seq_len < 1) return fail(SN_EINVAL, "seq_len must be >= 1");
  if (shape->n_layers < 1) return fail(SN_EINVAL, "n_layers must be >= 1");
  *bytes = sn_logits_workspace_bytes(shape->n_layers, seq_len, (int64_t)shape->n_q_heads * shape->head_dim,
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
  const int L = sh.n_layers;
  const int64_t nq_cols = (int64_t)sh.n_q_heads * dh, nk_cols = (int64_t)sh.n_kv_heads * dh;
  if ((int64_t)seq_len * ld_x * 2 >= (int64_t(1) << 31) || (int64_t)seq_len * nq_cols * 2 >= (int64_t(1) << 31))
    return fail(SN_EINVAL, "seq_len x row bytes must stay below 2^31");
  // the projection reads a layer's weight rows through one buffer range
  if (nq_cols * sh.ld * 2 >= (int64_t(1) << 32))
    return fail(SN_EINVAL, "n_q_heads x head_dim x ld x 2 bytes (one layer's W_Q) must stay below 2^32");
  const int64_t tiles = ceil_div(seq_len, 128);
  if ((int64_t)L * sh.n_q_heads * tiles * tiles >= (int64_t(1) << 31) ||
      (int64_t)L * tiles * ceil_div(nq_cols + nk_cols, 128) >= (int64_t(1) << 31))
    return fail(SN_EINVAL, "n_layers x n_q x (seq_len / 128)^2 must stay below 2^31");
  const int64_t need = sn_logits_workspace_bytes(L, seq_len, nq_cols, nk_cols);
  if (workspace_bytes < need) return fail(SN_EINVAL, "workspace too small (spectral_logits_workspace_bytes)");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) || (reinterpret_cast<uintptr_t>(codes) & 15))
    return fail(SN_EINVAL, "workspace must be 256-byte and codes 16-byte aligned");
  for (int l = 0; l < L; ++l) {
    if (!x_layers[l] || !wq_layers[l] || !wk_layers[l]) return fail(SN_ENULL, "a layer pointer is NULL");
    if ((reinterpret_cast<uintptr_t>(x_layers[l]) | reinterpret_cast<uintptr_t>(wq_layers[l]) |
         reinterpret_cast<uintptr_t>(wk_layers[l])) & 15)
      return fail(SN_EINVAL, "layer pointers must be 16-byte aligned");
  }
  int cur_dev = 0;
  SN_HIP(hipGetDevice(&cur_dev));
  if (cur_dev != c->device) return fail(SN_ESTATE, "the current HIP device is not the context's device");

  // pointer tables at the start of the workspace, written by a kernel whose
  // arguments carry the pointers (so the call can be captured into a graph)
  const void** d_tab = reinterpret_cast<const void**>(workspace);
  int rc = fill_table(d_tab, 3 * L,
                      [&](int i) { return i < L ? x_layers[i] : i < 2 * L ? wq_layers[i - L] : wk_layers[i - 2 * L]; },
                      c->stream);
  if (rc != SN_OK) return rc;
  uint16_t* planes = reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(workspace) + ((3 * L * 8 + 255) & ~255));
  const size_t qn = (size_t)L * seq_len * nq_cols, kn = (size_t)L * seq_len * nk_cols;
  ProjArgs p{};
  p.x = d_tab;
  p.wq = d_tab + L;
  p.wk = d_tab + 2 * L;
  p.ld_x = ld_x;
  p.ld_w = sh.ld;
  p.layers = L;
  p.seq = seq_len;
  p.d = sh.d_model;
  p.nq_cols = (int32_t)nq_cols;
  p.nk_cols = (int32_t)nk_cols;
  p.qh = planes;
  p.ql = planes + qn;
  p.kh = planes + 2 * qn;
  p.kl = planes + 2 * qn + kn;
  LogitArgs g{};
  g.qh = p.qh;
  g.ql = p.ql;
  g.kh = p.kh;
  g.kl = p.kl;
  g.layers = L;
  g.seq = seq_len;
  g.g = c->plan.g;
  g.nq_cols = (int32_t)nq_cols;
  g.nk_cols = (int32_t)nk_cols;
  g.tiles = ceil_div(seq_len, 128);
  g.n_heads = sh.n_q_heads;
  g.scale = scale;
  g.codes = codes;
  g.max_abs = max_abs;
  g.n_over = n_over;
  rc = timed(c, KIND_LOGITS, [&] { sn_launch_zero_stats(max_abs, n_over, L * sh.n_q_heads, c->stream); });
  if (rc != SN_OK) return rc;
  if ((rc = timed(c, KIND_PROJ, [&] { sn_launch_proj(p, c->stream); })) != SN_OK) return rc;
  return timed(c, KIND_LOGITS, [&] { sn_launch_logits(g, dh, c->stream); });
}
}  // extern "C"
