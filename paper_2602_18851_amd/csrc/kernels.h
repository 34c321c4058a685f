// Internal interface between the C ABI (spectral.hip) and the kernel sources
// of the estimator (sweeps.hip, gram.hip, layer_form.hip): launch arguments,
// workspace views, launch-shape constants and the launchers.  Not part of
// the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace sn {

constexpr int kWaves = 4;             // waves per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kRG = 8;                // row groups per wave (lane >> 3)
constexpr int kCPL = 8;               // 16-byte column chunks per wave row (lane & 7)
constexpr int kMaxGC = 8;             // query heads per W_K work item
constexpr int kQTargetItems = 10240;  // wave work items aimed for in a W_Q sweep
constexpr int kMinTilesPerStrip = 4;  // automatic strips: at least this many tiles per wave
constexpr int kTailMinTiles = 4;      // ... in the compacted launches of the tolerance-mode tail
constexpr int kTailSteps = 2;         // tolerance mode: full sweep steps before the tail (the rule's minimum)
constexpr int kSetupUnroll = 4;       // producer partials summed per round in a sweep's set-up
constexpr int kKTargetItems = 4096;   // ... and in a W_K sweep (register-heavier waves)
constexpr int kKMfmaResident = 2048;  // waves of the matrix-core W_K sweep resident at once (256 CUs x 8)
constexpr int kStreamPolicy = 2;       // cache policy of the weight loads: non-temporal (read once per sweep)

constexpr int kMWaves = 2;                 // waves per workgroup
constexpr int kMTileC = 64;                // columns per tile: 128-byte row segments
constexpr int kGWaves = 4;                 // waves per workgroup of the Gram sweep
constexpr int kGTargetItems = 4096;        // Gram work items aimed for (about two waves per SIMD)
constexpr int kRedThreads = 512;

// Sweep phases: the first W_K sweep from v, the W_Q and W_K sweeps of a step,
// and the two final sweeps of the Gram form (v' = K_j^T y and u' = Q_h^T z
// from the d_h-vectors the Gram iteration leaves behind).
enum { PH_INIT = 0, PH_Q = 1, PH_K = 2, PH_EK = 3, PH_EQ = 4 };
enum { LM_ROWS = 0, LM_COLS = 1 };

// Control block of the tolerance-mode tail, written on the device by the
// list kernel: for each compacted launch the number of listed entries and
// the strips (and tiles per strip) chosen for that count.
enum {
  TC_GRAM = 0,   // Gram sweep over the running query heads, then their key heads
  TC_EK = 3,     // final W_K sweep over the W_K units holding a running head
  TC_EQ = 6,     // final W_Q sweep over the running query heads
  TC_NQ = 9,     // running query heads (the first entries of the Gram list)
  TC_WORDS = 10
};

struct Work {
  // S below is the strip count of the sweep that wrote the partials (its
  // s_out): fixed, except in the final sweeps of the tolerance-mode tail; the
  // buffers hold the largest count the plan can use.
  float* zp;         // [2][H][S][DH]   W_K-sweep partials of z, by step parity
  float* zn;         // [2][H][S]       ... and of ||v'||^2 (||v||^2 for the first sweep)
  float* yp;         // [H][S][DH]      W_Q-sweep partials of y
  float* yn;         // [H][S]          ... and of ||u'||^2 = sigma^2
  float* sig;        // [2][H]          sigma of the last two steps
  float* vnorm0;     // [H]             ||v|| of the start vector
  int32_t* alive;    // [2][H]          head continues after the step of that parity
  int32_t* iters;    // [H]             used when the caller passes no iters array
  float* fin;        // [H][2][DH]      Gram form and tail: z and y of each head's last step
  int32_t* zs;       // [H]             tolerance mode: strips of each head's last ||v'||^2 partials
  int32_t* list_g;   // [H + L n_kv]    tail: running query heads, then their key heads (H + index)
  int32_t* list_k;   // [U]             tail: W_K units holding a running head
  int32_t* kvpos;    // [L n_kv]        tail: place of a key head among the listed key heads, or -1
  int32_t* ctl;      // [TC_WORDS]      tail control block
  float* zt;         // [H][S_t]        tail: ||v'||^2 partials of the final W_K sweep
};

struct SweepArgs {
  const void* const* mats;  // device table: per-layer wq or wk
  int64_t ld;
  int32_t d, n_q, n_kv, g, H;
  int32_t s_q, s_k;         // strips of the W_Q and W_K sweeps
  int32_t s_out, tps, n_tiles, nch, n_items;
  int32_t k, n_iter, want_vec;
  float tol;
  const int32_t* list;      // tail launches: the decoded unit of item index r is list[r]
  const int32_t* ctl;       // tail launches: count, strips, tiles per strip at ctl[0..2] (else nullptr)
  const int32_t* only;      // final sweeps of the tail: a head takes part only if only[head] != 0
  Work w;
  float* v;
  float* u;
  float* sigma;
  int32_t* iters;
};

struct FinArgs {
  int32_t H, L, n_q, d, s_k;
  int32_t slot_fixed;  // workspace slot of the ||v'||^2 partials; -1: parity of the last step
  const int32_t* zs;   // per-head strips of those partials, or nullptr: s_k for every head
  const int32_t* tail; // tolerance mode: flags of the heads the tail finished (else nullptr) ...
  const float* zt;     // ... whose ||v'||^2 partials are zt[head][zs[head]]
  float coef;
  Work w;
  float* v;
  float* u;
  float* sigma;
  float* scale;
  int32_t* iters;
};


struct GramArgs {
  const void* const* mats;  // device table: wq pointers of all layers, then wk pointers
  int64_t ld;
  int32_t d, L, n_q, n_kv, H;
  int32_t s_g, tps, n_tiles, n_items;
  const int32_t* list;      // tail: unit of list entry r is list[r]; count and strips in ctl (else nullptr)
  const int32_t* ctl;
  float* gp;  // [items][NB][64 lanes][4]: partial Gram blocks in the MFMA output layout, item = entry * s_g + strip
};

// The d_h-space iteration.  The Gram form starts at step 1 from the first W_K
// sweep's z partials (slot 0); the tolerance-mode tail continues the heads
// still running after step k0 of the sweep chain from that step's partials
// (slot k0 & 1) and sigma_{k0}, one workgroup per listed head.
struct IterArgs {
  int32_t H, n_q, n_kv, g, s_k, s_g, n_iter;
  int32_t k0;               // steps already taken
  float tol;
  const float* gp;
  const int32_t* list;      // tail: Gram list, its count of query heads in ctl (else nullptr)
  const int32_t* ctl;
  const int32_t* kvpos;
  Work w;
  float* sigma;
  int32_t* iters;
};

struct LayerArgs {
  const void* const* mats;  // device table of this matrix's per-layer pointers
  int64_t ld;
  int32_t d, n_tiles, n_items;
  const int32_t* lstat;     // [L]
  // rows sweep, item = (layer * units + unit) * s_out + strip:
  // x = xvec[layer] / sqrt(xn2[layer]) -> rowpart [L*units][s_out][DH]
  int32_t units, s_out, tps;
  const float* xvec;
  const float* xn2;
  float* rowpart;
  // cols sweep, item = (layer * n_rsplit + rs) * n_tiles + tile: one column
  // tile of the layer over row blocks rs * rb_per .. (of nrb), each block b
  // weighted by vin[layer][b] -> colout [L * n_rsplit][cstride]
  int32_t nrb, n_rsplit, rb_per;
  const float* vin;         // [L][nrb][DH]
  float* colout;            // columns 0 .. d - 1 of each row are written
  int32_t cstride;          // multiple of 64 and >= d
};

// Inputs of a column sweep, one d_h-vector per row block of the swept matrix:
// vin[l][b] = sum over the cnt source units starting at (b / div) * cnt of
// their strip partials (src_units units per layer, strips strips each), in
// unit then strip order.
struct LayerVinArgs {
  const float* part;
  int32_t src_units, strips, div, cnt, nrb, dh;
  const int32_t* lstat;
  float* vin;
};

// Per layer: vec[c] = sum over the layer's units of col[unit][c] (fixed order)
// and n2 = ||vec||^2; mode 0 copies the caller's start vector instead and
// (re)initialises the layer status; mode 1 marks M v = 0.  Two launches: the
// column sums over nb blocks of kRedThreads columns per layer, each leaving
// its part of n2 in n2part[layer][block], then one block per layer that adds
// the parts in block order.
struct LayerReduceArgs {
  const float* col;         // [L*units][cstride]
  int32_t units, d, cstride, mode, nb;
  float* vec;
  float* n2;
  float* n2part;    // [L][nb]
  float* n2_start;  // mode 0: ||v||^2 of the start vector
  int32_t* lstat;
};

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

// ---- launchers (one per kernel family; each picks the template instance)
void launch_sweep(bool bf16, int head_dim, int ph, int gc, bool mfma, int n_items, hipStream_t st,
                  const SweepArgs& a);
void launch_finalize(int blocks, hipStream_t st, const FinArgs& f);
// Tail of tolerance mode after step k of the chain (running flags of parity
// k & 1): lists the running query heads, then the key heads serving one of
// them (Gram list), and the W_K units holding one, all ascending; the place
// of each listed key head; and the counts and strips of the tail's launches
// (TailPlan) in the control block.  One workgroup.
struct TailPlan {
  int32_t n_tiles_g, n_tiles_k, n_tiles_q;   // column tiles of the Gram, W_K and W_Q sweeps
  int32_t target_g, target_k, target_q;      // wave items aimed for in each
};
void launch_tail_lists(const SweepArgs& a, int slot, int gc, int n_units, const TailPlan& tp, hipStream_t st);
void launch_gram(bool bf16, int head_dim, int n_items, hipStream_t st, const GramArgs& g);
void launch_gram_iterate(int head_dim, int heads, hipStream_t st, const IterArgs& a);
void launch_layer_sweep(bool bf16, int head_dim, int mode, int n_items, hipStream_t st, const LayerArgs& a);
void launch_layer_vin(int layers, hipStream_t st, const LayerVinArgs& v);
void launch_layer_reduce(int layers, hipStream_t st, const LayerReduceArgs& r);
void launch_layer_finalize(int layers, hipStream_t st, const LayerFinArgs& f);

}  // namespace sn
