// C ABI of the CurvaDion step (include/curvadion.h): argument checks, layer and
// group lifetimes, workspace, launch planning and the per-step schedule.
//
// One group step (Algorithm 2 of the paper):
//   1. B = M + G with per-block partial sums of B^2, up to MAXS layers of
//      any shapes per launch
//   2. gate kernel: fixed-order norms, RMMC_l, prev_norm update, max, flag
//   3. one device-to-host copy of {max, flag, RMMC_l}: the decision point that
//      stands in for the max all-reduce at one worker
//   4. sync branch, per unit (up to MAXB layers of one shape), each unit's
//      whole pipeline on one stream and up to four units at a time: P~ = B Q;
//      CholQR twice (fp64 Gram, Cholesky + inverse, apply); R = B^T P;
//      ColumnNormalize; M/X update.  The latency-bound factorisation of one
//      unit overlaps the GEMMs of the others.
//      local branch: X -= eta_local G (M already holds B).
// The streaming passes take up to MAXS layers of any shapes per launch; the
// sync branch's kernels take layers of equal (m, n) (up to MAXB per launch).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/curvadion.h"
#include "common.hpp"
#include "form_bq.hpp"
#include "plan.hpp"

namespace {

thread_local std::string g_err;

cd_status fail(cd_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define CD_HIP(call)                                                                         \
  do {                                                                                       \
    hipError_t e_ = (call);                                                                  \
    if (e_ != hipSuccess)                                                                    \
      return fail(CD_EHIP, "%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), __FILE__, \
                  __LINE__);                                                                 \
  } while (0)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Restores the caller's current device on scope exit.
struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) { ok = false; return; }
    if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

// K-splitting so that one launch has >= ~1024 working blocks, each slice >=
// 256 deep.  pieces > 0 selects the tile shape of the bf16-split kernels, else
// the fp32 / fp64 MFMA kernels; `upper` counts only the tiles an upper-only
// product computes (the others exit at once).
int plan_splits(int M, int N, int K, int nl, bool fp64, int* kchunk, int pieces = 0, bool upper = false) {
  const long long bm = pieces > 0 ? cd::gemm_bf_bm(N) : cd::gemm_bm(N, fp64);
  const long long bn = pieces > 0 ? cd::gemm_bf_bn(N, pieces) : cd::gemm_bn(N, fp64);
  const long long tiles_m = (M + bm - 1) / bm, tiles_n = (N + bn - 1) / bn;
  long long per_layer = tiles_m * tiles_n;
  if (upper) {
    per_layer = 0;
    for (long long i = 0; i < tiles_m; ++i) per_layer += std::max(0LL, tiles_n - i);
  }
  const long long tiles = per_layer * nl;
  int s = 1;
  while (tiles * s < 1024 && K / (2 * s) >= 256 && s < 32) s *= 2;
  int kc = (K + s - 1) / s;
  kc = (kc + cd::GBK - 1) / cd::GBK * cd::GBK;
  *kchunk = kc;
  return (K + kc - 1) / kc;
}

// ---- optional per-kernel timing (HIP events on the launch stream) ----------
enum Kind { K_FORM, K_FORM_X, K_GATE, K_LOCAL, K_PBQ, K_PBQ_BF, K_GRAM, K_GRAM_BF, K_CHOL, K_TRSM, K_TRTRI,
            K_APPLY_BF, K_PBTP, K_PBTP3, K_REDUCE, K_COLNORM, K_UPDATE, K_UPDATE_BF1, K_UPDATE_F32,
            K_SMALL_QR, K_SMALL_UPD, K_GRAM_X, K_FORM_BQ, K_NKINDS };
const char* const kKindName[K_NKINDS] = {
    "form_buffer", "form_buffer_local", "gate", "local_update", "power_bq_f64", "power_bq_bf16x3", "gram_f64",
    "gram_bf16x6", "cholesky_f64", "trsm_f64", "trtri_f64", "apply_bf16x6", "power_btp_f64",
    "power_btp_bf16x3", "reduce_splits", "colnorm", "update_bf16x6", "update_bf16", "update_f32",
    "small_cholqr", "small_update", "gram_bf16x9", "form_power_bq_bf16x3"};
static_assert(K_NKINDS <= 32, "the timing mask holds one bit per kind");

// Timing events only measure: recording them without the system-scope fence
// (cache write-back and invalidate) keeps them from stretching the gaps
// between the kernels they bracket.
constexpr unsigned kTimingEventFlags = hipEventDisableSystemFence;

struct Timer {
  struct Rec { int kind; hipEvent_t a, b; double bytes, flops; };
  bool on = false;
  unsigned mask = ~0u;   // kinds that get events while on
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  hipEvent_t get() {
    hipEvent_t e = nullptr;
    if (!pool.empty()) { e = pool.back(); pool.pop_back(); return e; }
    if (hipEventCreateWithFlags(&e, kTimingEventFlags) != hipSuccess) return nullptr;
    return e;
  }
  void release() {
    for (auto& r : recs) { pool.push_back(r.a); pool.push_back(r.b); }
    recs.clear();
  }
  // create events ahead of time so that a timed region creates none
  hipError_t reserve(size_t n) {
    while (pool.size() < n) {
      hipEvent_t e = nullptr;
      const hipError_t err = hipEventCreateWithFlags(&e, kTimingEventFlags);
      if (err != hipSuccess) return err;
      pool.push_back(e);
    }
    return hipSuccess;
  }
  ~Timer() {
    release();
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
  }
};

}  // namespace

struct cd_layer {
  cd_layer_desc d{};
  int device = 0;
  long long step = 0;
  void* ws = nullptr;           // the one device allocation the pointers below are carved from
  double* prev = nullptr;       // device, 1 double
  int* rankdef = nullptr;       // device, 1 int
  int* nid_ok = nullptr;        // device, 1 int: the second CholQR pass took the near-identity path
  int* rowok = nullptr;         // device, r_max ints: rows of T whose pivot was not floored
  double* pa = nullptr;         // m x r_max fp64: P~ (bf16-gradient layers: the slice planes
                                // and exponents of the exact pass-0 Gram matrix)
  float* pb = nullptr;          // m x r_max: P~ after the first CholQR pass
  float* Uf = nullptr;          // r_max^2: inverse Cholesky factor (fp32) for the bf16 apply
  float* P = nullptr;           // m x r_max fp32: the orthonormal P
  float* R = nullptr;           // n x r_max
  double* W = nullptr;          // r_max^2 Gram matrix, then its Cholesky factor
  double* Dinv = nullptr;       // inverses of the 64 x 64 diagonal blocks of the factor
  double* floor_ = nullptr;     // pivot floor of the current factorisation
  double* gram_part = nullptr;  // split-K partials of the Gram matrix; between the second Gram
                                // matrix and the step's end, the near-identity factor's buffers
  void* split_part = nullptr;   // split-K partials of the skinny GEMMs (fp32 or fp64)
  size_t split_cap = 0;         // bytes of split_part
  size_t gram_cap = 0;          // doubles of gram_part
  double* colsq = nullptr;      // column sum-of-squares partials
  __bf16* planes = nullptr;     // bf16 split planes of P, R, Q for the update
  float* colnrm = nullptr;      // r_max column norms
  cd_group* self = nullptr;     // one-layer group used by cd_step
  int last_r = 0;
  bool prev_zero = true;        // prev_norm is known to be 0 (new layer, or set so)
  // the group that stepped the layer last (its completion event and pinned
  // rank-deficiency mirror answer cd_layer_rank_deficient), the layer's
  // index there, and the mirror's last value once that group is destroyed
  cd_group* last_group = nullptr;
  int last_index = 0;
  int rankdef_cached = 0;
};

struct ShapeClass {
  int m, n;
  std::vector<int> idx;  // positions in the group
};

// A batch of at most MAXB layers of one shape: the sync branch enqueues a
// unit's whole pipeline on one stream.  Its layers occupy the contiguous
// range [off, off + sel.size()) of the group's factor tables, and its tile
// lists index the layers relative to `off`.
struct Unit {
  int sc;                // shape class
  std::vector<int> sel;  // positions in the group
  int fbq_splits = 1, fbq_kchunk = 0;   // K slices of the fused buffer pass + P~ = B Q
  int off;               // first factor-table entry
  int toff, nt;          // its (layer, 64-row tile of m) pairs in trsm_tiles
  int rtoff, nrt;        // its (layer, 64-row tile of r_max) pairs in trtri_tiles
};

struct cd_group {
  void* tables = nullptr;       // the one device allocation the tables below are carved from
  std::vector<cd_layer*> layers;
  std::vector<ShapeClass> shapes;
  int device = 0;
  int L = 0;
  bool g_bf16 = false;
  double tau = 0, eps = 0;
  cd_policy policy = CD_POLICY_RMMC;
  int H = 1;
  int nparts_stride = 0;
  double* parts = nullptr;      // [L][nparts_stride]
  int* nparts = nullptr;        // [L]: partials of the buffer pass
  int* nparts_fx = nullptr;     // [L]: partials of the fused buffer pass + P~ = B Q
  std::vector<int> np_fx;       // the same on the host; empty: no fused pass planned
  double** prev = nullptr;      // [L] device pointers to each layer's prev_norm
  double* norms = nullptr;      // [L] gate workspace
  unsigned* counter = nullptr;  // gate completion counter (returns to zero)
  cd::StepCtl* ctl = nullptr;   // the step's decision on the device (see cd::StepCtl)
  // RMMC policy: the branch predicted for the next step, when the host knows
  // the last decision (after a step that read it, or a last-result call);
  // otherwise the buffer pass takes the device's prediction
  bool predict_skip = false;
  bool pred_known = true;
  hipEvent_t done_ev = nullptr; // recorded after each step's last kernel
  bool stepped = false;
  cd::GateOut* out_dev = nullptr;
  // pinned, coherent, mapped: GateOut, L doubles, the sequence number the
  // gate stores last, then L ints mirroring each layer's rank-deficiency
  // flag; out_host_dev is the device view of the same memory
  void* out_host = nullptr;
  void* out_host_dev = nullptr;
  unsigned long long seq = 0;
  hipEvent_t ev = nullptr;
  std::vector<Unit> units;
  // the streaming passes (buffer formation, local update): batches of up to
  // MAXS layers of any shapes, in group order, each at most MAX_STREAM_BLOCKS
  // blocks
  std::vector<std::vector<int>> sbatches;
  cd::CholTab* chol_tab = nullptr;      // [L] static workspace pointers, in unit order
  cd::TrsmTab* trsm_tab[3] = {nullptr, nullptr, nullptr};  // P1 = P~ T^-1; U = T^-1; P = P1 T^-1
  int2* trsm_tiles = nullptr;           // per unit: (layer in the unit, 64-row tile of m) pairs
  int2* trtri_tiles = nullptr;          // per unit: (layer in the unit, 64-row tile of r_max) pairs
  // groups of several units: the sync branch runs unit u on stream
  // stream_of(u) (the caller's stream or one of these, default priority),
  // forked from and joined back to the caller's stream
  static constexpr int NSIDE = 3;
  int nside = 0;
  hipStream_t side[NSIDE] = {nullptr, nullptr, nullptr};
  hipEvent_t fork_ev = nullptr;
  hipEvent_t join_ev[NSIDE] = {nullptr, nullptr, nullptr};
  Timer timer;
};

namespace {

// Offsets inside a group's pinned host block.
size_t host_seq_off(int L) { return sizeof(cd::GateOut) + sizeof(double) * L; }
size_t host_rankdef_off(int L) { return host_seq_off(L) + sizeof(unsigned long long); }
size_t host_bytes(int L) { return host_rankdef_off(L) + sizeof(int) * L; }

void free_layer(cd_layer* L) {
  if (!L) return;
  if (L->ws) (void)hipFree(L->ws);
  delete L;
}

void free_group(cd_group* g) {
  if (!g) return;
  // layers whose last step this group took keep its rank-deficiency flags
  for (int i = 0; i < static_cast<int>(g->layers.size()); ++i) {
    cd_layer* L = g->layers[i];
    if (L && L->last_group == g) {
      if (g->done_ev) (void)hipEventSynchronize(g->done_ev);
      L->rankdef_cached = g->out_host ? static_cast<const int*>(static_cast<const void*>(
                                            static_cast<const char*>(g->out_host) + host_rankdef_off(g->L)))[i]
                                      : 0;
      L->last_group = nullptr;
    }
  }
  if (g->tables) (void)hipFree(g->tables);
  if (g->done_ev) (void)hipEventDestroy(g->done_ev);
  if (g->out_host) (void)hipHostFree(g->out_host);
  if (g->ev) (void)hipEventDestroy(g->ev);
  for (int i = 0; i < cd_group::NSIDE; ++i) {
    if (g->side[i]) (void)hipStreamDestroy(g->side[i]);
    if (g->join_ev[i]) (void)hipEventDestroy(g->join_ev[i]);
  }
  if (g->fork_ev) (void)hipEventDestroy(g->fork_ev);
  delete g;
}

long long blocks_for(long long numel) { return (numel + cd::FORM_CHUNK - 1) / cd::FORM_CHUNK; }

// Workspace of one layer for ranks up to rm, as byte offsets into one block
// (every piece 256-byte aligned).  cd_layer_create allocates the block; the
// allocation-free step carves it from the static scratch array.
struct LayerLayout {
  size_t prev, rankdef, nid_ok, rowok, pa, pb, Uf, P, R, W, Dinv, floor_, gram_part, split_part, colsq, planes, colnrm;
  size_t split_cap;   // bytes of split_part
  size_t gram_cap;    // doubles of gram_part
  size_t total;
};

struct Carver {
  size_t off = 0;
  size_t put(size_t bytes) {
    const size_t o = off;
    off += (std::max<size_t>(bytes, 1) + 255) / 256 * 256;
    return o;
  }
};

LayerLayout layer_layout(int m, int n, int rm) {
  // split-K capacity: the largest partial product any rank r <= rm needs,
  // for one layer per launch (the most splits) and every piece count (the
  // tile width, hence the split count, depends on it)
  size_t split_bytes = 8, gram_cap = 1;
  for (int r = 1; r <= rm; ++r) {
    int kc;
    const size_t mr = static_cast<size_t>(m) * r, nr = static_cast<size_t>(n) * r;
    split_bytes = std::max(split_bytes, plan_splits(m, r, n, 1, true, &kc) * mr * sizeof(double));
    split_bytes = std::max(split_bytes, plan_splits(n, r, m, 1, true, &kc) * nr * sizeof(double));
    for (int pieces = 1; pieces <= 3; ++pieces) {
      split_bytes = std::max(split_bytes, plan_splits(m, r, n, 1, false, &kc, pieces) * mr * sizeof(float));
      split_bytes = std::max(split_bytes, plan_splits(n, r, m, 1, false, &kc, pieces) * nr * sizeof(float));
      split_bytes = std::max(split_bytes, plan_splits(m, r, r, 1, false, &kc, pieces) * mr * sizeof(float));
      split_bytes = std::max(split_bytes, plan_splits(r, r, m, 1, false, &kc, pieces) * r * r * sizeof(float));
    }
    gram_cap = std::max(gram_cap, static_cast<size_t>(plan_splits(r, r, m, 1, true, &kc, 0, true)) * r * r);
  }
  // the second pass's near-identity factor (fp32-gradient layers) borrows it
  gram_cap = std::max(gram_cap, 2 * static_cast<size_t>(rm) * rm + cd::nearid_parts(rm));
  const size_t M = m, N = n, R = rm;
  const size_t nchunks = (N + cd::COLNORM_ROWS - 1) / cd::COLNORM_ROWS;
  const size_t nblk = (R + cd::CHOL_BLOCK - 1) / cd::CHOL_BLOCK;
  const size_t rpm = (R + 31) / 32 * 32;
  LayerLayout lo{};
  Carver c;
  lo.prev = c.put(sizeof(double));
  lo.rankdef = c.put(sizeof(int));
  lo.nid_ok = c.put(sizeof(int));
  lo.rowok = c.put(sizeof(int) * R);
  lo.pa = c.put(std::max(sizeof(double) * M * R, cd::gram_x_bytes(m, rm)));
  lo.pb = c.put(sizeof(float) * M * R);
  lo.Uf = c.put(sizeof(float) * R * R);
  lo.P = c.put(sizeof(float) * M * R);
  lo.R = c.put(sizeof(float) * N * R);
  lo.W = c.put(sizeof(double) * R * R);
  lo.Dinv = c.put(sizeof(double) * nblk * cd::CHOL_BLOCK * cd::CHOL_BLOCK);
  lo.floor_ = c.put(sizeof(double));
  lo.gram_part = c.put(sizeof(double) * gram_cap);
  lo.split_part = c.put(split_bytes);
  lo.colsq = c.put(sizeof(double) * nchunks * R);
  lo.planes = c.put(sizeof(__bf16) * 3 * (M + 2 * N) * rpm);
  lo.colnrm = c.put(sizeof(float) * R);
  lo.split_cap = split_bytes;
  lo.gram_cap = gram_cap;
  lo.total = c.off;
  return lo;
}

void carve_layer(cd_layer* L, char* base, const LayerLayout& lo) {
  L->prev = reinterpret_cast<double*>(base + lo.prev);
  L->rankdef = reinterpret_cast<int*>(base + lo.rankdef);
  L->nid_ok = reinterpret_cast<int*>(base + lo.nid_ok);
  L->rowok = reinterpret_cast<int*>(base + lo.rowok);
  L->pa = reinterpret_cast<double*>(base + lo.pa);
  L->pb = reinterpret_cast<float*>(base + lo.pb);
  L->Uf = reinterpret_cast<float*>(base + lo.Uf);
  L->P = reinterpret_cast<float*>(base + lo.P);
  L->R = reinterpret_cast<float*>(base + lo.R);
  L->W = reinterpret_cast<double*>(base + lo.W);
  L->Dinv = reinterpret_cast<double*>(base + lo.Dinv);
  L->floor_ = reinterpret_cast<double*>(base + lo.floor_);
  L->gram_part = reinterpret_cast<double*>(base + lo.gram_part);
  L->split_part = base + lo.split_part;
  L->colsq = reinterpret_cast<double*>(base + lo.colsq);
  L->planes = reinterpret_cast<__bf16*>(base + lo.planes);
  L->colnrm = reinterpret_cast<float*>(base + lo.colnrm);
  L->split_cap = lo.split_cap;
  L->gram_cap = lo.gram_cap;
}

// The device tables of a group of L layers, as byte offsets into one block.
struct GroupLayout {
  size_t parts, nparts, nparts_fx, prev, norms, counter, ctl, out_dev, chol_tab, trsm_tab[3], trsm_tiles, trtri_tiles;
  size_t total;
};

GroupLayout group_layout(int L, int nparts_stride, size_t ntiles, size_t nrtiles) {
  GroupLayout lo{};
  Carver c;
  lo.parts = c.put(sizeof(double) * L * nparts_stride);
  lo.nparts = c.put(sizeof(int) * L);
  lo.nparts_fx = c.put(sizeof(int) * L);
  lo.prev = c.put(sizeof(double*) * L);
  lo.norms = c.put(sizeof(double) * L);
  lo.counter = c.put(sizeof(unsigned));
  lo.ctl = c.put(sizeof(cd::StepCtl));
  lo.out_dev = c.put(sizeof(cd::GateOut) + sizeof(double) * L);
  lo.chol_tab = c.put(sizeof(cd::CholTab) * L);
  for (int k = 0; k < 3; ++k) lo.trsm_tab[k] = c.put(sizeof(cd::TrsmTab) * L);
  lo.trsm_tiles = c.put(sizeof(int2) * ntiles);
  lo.trtri_tiles = c.put(sizeof(int2) * nrtiles);
  lo.total = c.off;
  return lo;
}

void carve_group(cd_group* g, char* base, const GroupLayout& lo) {
  g->parts = reinterpret_cast<double*>(base + lo.parts);
  g->nparts = reinterpret_cast<int*>(base + lo.nparts);
  g->nparts_fx = reinterpret_cast<int*>(base + lo.nparts_fx);
  g->prev = reinterpret_cast<double**>(base + lo.prev);
  g->norms = reinterpret_cast<double*>(base + lo.norms);
  g->counter = reinterpret_cast<unsigned*>(base + lo.counter);
  g->ctl = reinterpret_cast<cd::StepCtl*>(base + lo.ctl);
  g->out_dev = reinterpret_cast<cd::GateOut*>(base + lo.out_dev);
  g->chol_tab = reinterpret_cast<cd::CholTab*>(base + lo.chol_tab);
  for (int k = 0; k < 3; ++k) g->trsm_tab[k] = reinterpret_cast<cd::TrsmTab*>(base + lo.trsm_tab[k]);
  g->trsm_tiles = reinterpret_cast<int2*>(base + lo.trsm_tiles);
  g->trtri_tiles = reinterpret_cast<int2*>(base + lo.trtri_tiles);
}

// The triangular-solve tables of one layer.  fp32-gradient layers solve
// both CholQR passes in place in the fp64 panel pa (P~ -> P1 -> P), so that
// every block column is formed from fp64 values of the earlier ones; P is
// rounded to fp32 afterwards.  bf16-gradient layers apply explicit inverses
// (t1: U = T^-1) and use t0 only to complete P1 (fp32, pb) past the rank.
void factor_tabs(const cd_layer* L, cd::TrsmTab& t0, cd::TrsmTab& t1, cd::TrsmTab& t2) {
  if (L->d.grad_dtype == CD_BF16) {
    t0 = cd::TrsmTab{L->pa, L->pb, L->W, L->Dinv, L->d.m};
    t2 = cd::TrsmTab{L->pb, L->P, L->W, L->Dinv, L->d.m};
  } else {
    t0 = cd::TrsmTab{L->pa, L->pa, L->W, L->Dinv, L->d.m};
    t2 = cd::TrsmTab{L->pa, L->pa, L->W, L->Dinv, L->d.m};
  }
  t1 = cd::TrsmTab{nullptr, L->Uf, L->W, L->Dinv, L->d.r_max};
}

// Host side of a group: shape classes, units (chunks of at most MAXB layers
// of one shape) with their rows of the factor tables, and the streaming
// launches; the table contents go to ct, t0..t2 and the tile lists.
// rankdef_host: the device view of the group's L-int rank-deficiency mirror.
void plan_group(cd_group* g, cd_layer* const* layers, int n, std::vector<int>& np, std::vector<double*>& pv,
                std::vector<cd::CholTab>& ct, std::vector<cd::TrsmTab>& t0, std::vector<cd::TrsmTab>& t1,
                std::vector<cd::TrsmTab>& t2, std::vector<int2>& tiles, std::vector<int2>& rtiles,
                int* rankdef_host) {
  g->layers.assign(layers, layers + n);
  g->L = n;
  g->device = layers[0]->device;
  g->g_bf16 = layers[0]->d.grad_dtype == CD_BF16;
  g->tau = layers[0]->d.tau;
  g->eps = layers[0]->d.eps;
  g->policy = layers[0]->d.policy;
  g->H = layers[0]->d.H;
  g->shapes.clear();
  g->units.clear();
  g->nparts_stride = 0;
  for (int i = 0; i < n; ++i) {
    const cd_layer* L = layers[i];
    auto it = std::find_if(g->shapes.begin(), g->shapes.end(), [&](const ShapeClass& s) {
      return s.m == L->d.m && s.n == L->d.n;
    });
    if (it == g->shapes.end()) g->shapes.push_back(ShapeClass{L->d.m, L->d.n, {i}});
    else it->idx.push_back(i);
    g->nparts_stride = std::max<int>(g->nparts_stride,
                                     static_cast<int>(blocks_for(1LL * L->d.m * L->d.n)));
  }
  np.assign(n, 0);
  pv.assign(n, nullptr);
  ct.assign(n, cd::CholTab{});
  t0.assign(n, cd::TrsmTab{});
  t1.assign(n, cd::TrsmTab{});
  t2.assign(n, cd::TrsmTab{});
  tiles.clear();
  rtiles.clear();
  for (int i = 0; i < n; ++i) {
    np[i] = static_cast<int>(blocks_for(1LL * layers[i]->d.m * layers[i]->d.n));
    pv[i] = layers[i]->prev;
  }
  int off = 0;
  for (int c = 0; c < static_cast<int>(g->shapes.size()); ++c) {
    const ShapeClass& sc = g->shapes[c];
    for (size_t c0 = 0; c0 < sc.idx.size(); c0 += cd::MAXB) {
      Unit u;
      u.sc = c;
      u.sel.assign(sc.idx.begin() + c0, sc.idx.begin() + std::min(sc.idx.size(), c0 + cd::MAXB));
      u.off = off;
      u.toff = static_cast<int>(tiles.size());
      u.rtoff = static_cast<int>(rtiles.size());
      for (int j = 0; j < static_cast<int>(u.sel.size()); ++j) {
        cd_layer* L = layers[u.sel[j]];
        const int k = off + j;
        ct[k] = cd::CholTab{L->W, L->Dinv, L->floor_, L->rankdef, L->rowok,
                            rankdef_host ? rankdef_host + u.sel[j] : nullptr, L->gram_part, L->nid_ok};
        factor_tabs(L, t0[k], t1[k], t2[k]);
        for (int rt = 0; rt < (L->d.m + cd::CHOL_BLOCK - 1) / cd::CHOL_BLOCK; ++rt) tiles.push_back(int2{j, rt});
        for (int rt = 0; rt < (L->d.r_max + cd::CHOL_BLOCK - 1) / cd::CHOL_BLOCK; ++rt)
          rtiles.push_back(int2{j, rt});
      }
      u.nt = static_cast<int>(tiles.size()) - u.toff;
      u.nrt = static_cast<int>(rtiles.size()) - u.rtoff;
      off += static_cast<int>(u.sel.size());
      g->units.push_back(std::move(u));
    }
  }
  // the fused buffer pass + P~ = B Q of bf16-gradient layers: K slices per
  // unit, so that a launch has about three workgroups per CU (one fits) and
  // a slice keeps at least 512 k
  g->np_fx.clear();
  if (g->g_bf16) {
    g->np_fx.assign(n, 0);
    for (Unit& u : g->units) {
      const int m = g->shapes[u.sc].m, nn = g->shapes[u.sc].n;
      const long long tiles = 1LL * ((m + cd::FBQ_BM - 1) / cd::FBQ_BM) * static_cast<long long>(u.sel.size());
      int sp = 1;
      while (tiles * sp < 768 && nn / (2 * sp) >= 512 && sp < 16) sp *= 2;
      int kc = (nn + sp - 1) / sp;
      kc = (kc + cd::GBK - 1) / cd::GBK * cd::GBK;
      u.fbq_kchunk = kc;
      u.fbq_splits = (nn + kc - 1) / kc;
      for (int li : u.sel) {
        g->np_fx[li] = cd::form_bq_nparts(m, u.fbq_splits);
        g->nparts_stride = std::max(g->nparts_stride, g->np_fx[li]);
      }
    }
  }
  std::vector<long long> numel(n);
  for (int i = 0; i < n; ++i) numel[i] = 1LL * layers[i]->d.m * layers[i]->d.n;
  g->sbatches = cd::plan_stream_batches(numel, cd::MAXS, cd::MAX_STREAM_BLOCKS, cd::FORM_CHUNK);
}

cd_status build_group(cd_layer* const* layers, int n, cd_group** out) {
  cd_group* g = new (std::nothrow) cd_group();
  if (!g) return fail(CD_ENOMEM, "host allocation failed");
  std::vector<int> np;
  std::vector<double*> pv;
  std::vector<cd::CholTab> ct;
  std::vector<cd::TrsmTab> t0, t1, t2;
  std::vector<int2> tiles, rtiles;
  g->device = layers[0]->device;
  DeviceGuard dg(g->device);
  if (!dg.ok) { free_group(g); return fail(CD_EHIP, "cannot select device %d", g->device); }
  hipError_t e = hipHostMalloc(&g->out_host, host_bytes(n), hipHostMallocMapped | hipHostMallocCoherent);
  if (e == hipSuccess) std::memset(g->out_host, 0, host_bytes(n));
  if (e == hipSuccess) e = hipHostGetDevicePointer(&g->out_host_dev, g->out_host, 0);
  if (e != hipSuccess) {
    free_group(g);
    return fail(e == hipErrorOutOfMemory ? CD_ENOMEM : CD_EHIP, "group setup: %s", hipGetErrorString(e));
  }
  plan_group(g, layers, n, np, pv, ct, t0, t1, t2, tiles, rtiles,
             reinterpret_cast<int*>(static_cast<char*>(g->out_host_dev) + host_rankdef_off(n)));
  const GroupLayout lo = group_layout(n, g->nparts_stride, tiles.size(), rtiles.size());
  e = hipMalloc(&g->tables, lo.total);
  if (e == hipSuccess) {
    carve_group(g, static_cast<char*>(g->tables), lo);
    e = hipMemset(g->counter, 0, sizeof(unsigned));
  }
  if (e == hipSuccess) e = hipMemset(g->ctl, 0, sizeof(cd::StepCtl));
  if (e == hipSuccess) e = hipEventCreateWithFlags(&g->ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&g->done_ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipMemcpy(g->nparts, np.data(), sizeof(int) * n, hipMemcpyHostToDevice);
  if (e == hipSuccess && !g->np_fx.empty())
    e = hipMemcpy(g->nparts_fx, g->np_fx.data(), sizeof(int) * n, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(g->prev, pv.data(), sizeof(double*) * n, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(g->chol_tab, ct.data(), sizeof(cd::CholTab) * n, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(g->trsm_tab[0], t0.data(), sizeof(cd::TrsmTab) * n, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(g->trsm_tab[1], t1.data(), sizeof(cd::TrsmTab) * n, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(g->trsm_tab[2], t2.data(), sizeof(cd::TrsmTab) * n, hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = hipMemcpy(g->trtri_tiles, rtiles.data(), sizeof(int2) * rtiles.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = hipMemcpy(g->trsm_tiles, tiles.data(), sizeof(int2) * tiles.size(), hipMemcpyHostToDevice);
  if (g->units.size() > 1) {
    g->nside = std::min(static_cast<int>(g->units.size()) - 1, cd_group::NSIDE);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&g->fork_ev, hipEventDisableTiming);
    for (int i = 0; i < g->nside && e == hipSuccess; ++i) {
      e = hipStreamCreateWithFlags(&g->side[i], hipStreamNonBlocking);
      if (e == hipSuccess) e = hipEventCreateWithFlags(&g->join_ev[i], hipEventDisableTiming);
    }
  }
  if (e != hipSuccess) {
    free_group(g);
    return fail(e == hipErrorOutOfMemory ? CD_ENOMEM : CD_EHIP, "group setup: %s",
                hipGetErrorString(e));
  }
  *out = g;
  return CD_OK;
}

cd_status check_desc(const cd_layer_desc* d) {
  if (!d) return fail(CD_EINVAL, "desc is NULL");
  if (d->m < 1 || d->n < 1) return fail(CD_EINVAL, "m and n must be >= 1 (got %d, %d)", d->m, d->n);
  if (d->r_max < 1 || d->r_max > std::min(d->m, d->n))
    return fail(CD_EINVAL, "r_max must be in [1, min(m, n)] (got %d)", d->r_max);
  if (d->r_max > 1024) return fail(CD_EINVAL, "r_max above 1024 is not supported (got %d)", d->r_max);
  if (d->grad_dtype != CD_F32 && d->grad_dtype != CD_BF16) return fail(CD_EINVAL, "unknown grad dtype");
  if (d->policy < CD_POLICY_RMMC || d->policy > CD_POLICY_EVERY_H) return fail(CD_EINVAL, "unknown policy");
  if (std::isnan(d->tau)) return fail(CD_EINVAL, "tau is NaN");
  if (!(d->eps >= 0.0) || !std::isfinite(d->eps)) return fail(CD_EINVAL, "eps must be finite and >= 0");
  if (!(d->eta_local_scale >= 0.0) || !std::isfinite(d->eta_local_scale))
    return fail(CD_EINVAL, "eta_local_scale must be finite and >= 0");
  if (d->policy == CD_POLICY_EVERY_H && d->H < 1) return fail(CD_EINVAL, "H must be >= 1");
  if (!(d->weight_decay >= 0.0) || !std::isfinite(d->weight_decay))
    return fail(CD_EINVAL, "weight_decay must be finite and >= 0");
  return CD_OK;
}

// Launch through `launch`, bracketed by timing events when timing is on.
template <typename F>
cd_status run(cd_group* g, int kind, double bytes, double flops, hipStream_t s, F&& launch) {
  if (!g->timer.on || !((g->timer.mask >> kind) & 1u)) {
    CD_HIP(launch());
    return CD_OK;
  }
  hipEvent_t a = g->timer.get(), b = g->timer.get();
  if (!a || !b) return fail(CD_EHIP, "hipEventCreate failed");
  CD_HIP(hipEventRecord(a, s));
  CD_HIP(launch());
  CD_HIP(hipEventRecord(b, s));
  g->timer.recs.push_back(Timer::Rec{kind, a, b, bytes, flops});
  return CD_OK;
}

// One stage of the sync branch for the layers `sel` (all of one shape):
//   0: P~ = B Q          1: Gram matrix of CholQR pass 0 (fp64)
//   2: pass-0 apply, bf16-gradient layers: P1 = P~ U (bf16 x 6, U = T^-1 in fp32)
//   3: Gram matrix of pass 1 (fp64 for fp32 layers; bf16 x 6 for bf16-gradient
//      layers, whose P1 is well conditioned)
//   4: pass-1 apply, bf16-gradient layers: P = P1 U
//   5: R = B^T P, ColumnNormalize, the M / X update
// Cholesky factorisations, triangular solves and inverses run between the
// stages over all layers at once (enqueue_factor); fp32 layers apply T^-1 by
// fp64 triangular solves there.
// spec: whether this step's buffer pass applied the skip branch's X update
// (the branch was predicted to be local), which the update stage takes back:
// 0, 1, or 2 = as the control word says.  run_if: NULL, or &ctl->flag when
// the branch is enqueued before the decision is known (every kernel then
// returns at once on a local step).
cd_status enqueue_sync(cd_group* g, const ShapeClass& sc, const std::vector<int>& sel,
                       const void* const* G, int spec,
                       float* const* M, float* const* X, float* const* Q, float mu, float eta,
                       int r, int stage, hipStream_t s, const int* run_if) {
  const int m = sc.m, n = sc.n, nl = static_cast<int>(sel.size());
  auto lay = [&](int j) { return g->layers[sel[j]]; };
  // small layers: four launches (see below), their products without split-K
  const bool small = cd::small_sync_fits(m, n, r);

  // skinny GEMM C = A.B with optional split-K and fixed-order reduction
  // pieces > 0: fp32 operands on the bf16 MFMA with `pieces`-way splits
  auto gemm = [&](int tkind, double flops, double bytes, cd::GemmKind kind, int Mr, int Nr, int K,
                  bool a_kc, int lda, bool b_kc, int ldb, bool upper, auto Aof, auto Bof, auto Cof,
                  auto Pof, int pieces = 0, bool bf_out64 = false, bool b_upper = false) -> cd_status {
    const bool acc64 = pieces == 0 && cd::gemm_acc64(kind);
    cd::GemmArgs ga{};
    ga.M = Mr; ga.N = Nr; ga.K = K; ga.lda = lda; ga.ldb = ldb; ga.ldc = Nr;
    ga.a_kc = a_kc; ga.b_kc = b_kc; ga.upper_only = upper; ga.out64 = bf_out64; ga.b_upper = b_upper;
    ga.run_if = run_if;
    if (small) {
      ga.splits = 1;
      ga.kchunk = (K + cd::GBK - 1) / cd::GBK * cd::GBK;
    } else {
      ga.splits = plan_splits(Mr, Nr, K, nl, acc64, &ga.kchunk, pieces, upper);
    }
    ga.split_stride = 1LL * Mr * Nr;
    if (ga.splits > 1) {
      // the partials must fit the workspace sized at create time
      const size_t need = static_cast<size_t>(ga.splits) * Mr * Nr * (acc64 ? 8 : 4);
      for (int j = 0; j < nl; ++j) {
        const bool gram = Pof(j) == static_cast<void*>(lay(j)->gram_part);
        const size_t cap = gram ? lay(j)->gram_cap * sizeof(double) : lay(j)->split_cap;
        if (need > cap)
          return fail(CD_ENOMEM, "split-K workspace too small (%zu > %zu bytes) for a %d x %d x %d product",
                      need, cap, Mr, Nr, K);
      }
    }
    for (int j = 0; j < nl; ++j) {
      ga.A[j] = Aof(j);
      ga.B[j] = Bof(j);
      ga.C[j] = ga.splits > 1 ? Pof(j) : Cof(j);
    }
    cd_status st2 = run(g, tkind, bytes * nl, flops * nl, s, [&] {
      if (pieces > 0) return cd::launch_gemm_bf(ga, nl, pieces, s);
      // P~ = B Q of small layers: every operand straight into registers
      if (small && kind == cd::GemmKind::F64_FROM_F32 && a_kc && cd::small_gemm_fits(Nr, K))
        return cd::launch_small_gemm(ga, nl, kind, s);
      return cd::launch_gemm(ga, nl, kind, s);
    });
    if (st2 != CD_OK) return st2;
    if (ga.splits > 1) {
      cd::ReduceArgs ra{};
      ra.count = 1LL * Mr * Nr; ra.stride = ga.split_stride; ra.splits = ga.splits; ra.run_if = run_if;
      for (int j = 0; j < nl; ++j) { ra.part[j] = Pof(j); ra.out[j] = Cof(j); }
      const bool out64 = pieces == 0 ? (kind == cd::GemmKind::F64 || kind == cd::GemmKind::F64_FROM_F32)
                                     : bf_out64;
      const double rb = static_cast<double>(ra.count) * nl * (acc64 ? 8.0 : 4.0) * (ga.splits + 1);
      st2 = run(g, K_REDUCE, rb, 0.0, s, [&] { return cd::launch_reduce_splits(ra, nl, acc64, out64, s); });
      if (st2 != CD_OK) return st2;
    }
    return CD_OK;
  };
  auto part = [&](int j) { return lay(j)->split_part; };
  const double mn = 1.0 * m * n, mr = 1.0 * m * r, nr = 1.0 * n * r, rr = 1.0 * r * r;
  // eta_local of each layer: what a speculative skip update subtracted
  auto eta_local = [&](int j) {
    return static_cast<float>(lay(j)->d.eta_local_scale * static_cast<double>(eta));
  };
  if (small) {
    // P~ = B Q (fp64) -> CholQR2 in one workgroup per layer -> R = B^T P
    // (fp64 products) -> column norms, Q and the M / X update in one launch
    if (stage == 0)
      return gemm(K_PBQ, 2.0 * mn * r, 4.0 * mn + 4.0 * nr + 8.0 * mr, cd::GemmKind::F64_FROM_F32, m, r,
                  n, true, n, false, r, false,
                  [&](int j) { return static_cast<const void*>(M[sel[j]]); },
                  [&](int j) { return static_cast<const void*>(Q[sel[j]]); },
                  [&](int j) { return static_cast<void*>(lay(j)->pa); }, part);
    if (stage == 1) {
      cd::SmallQrArgs qa{};
      qa.m = m; qa.r = r; qa.run_if = run_if;
      int* mirror = g->out_host_dev ? reinterpret_cast<int*>(static_cast<char*>(g->out_host_dev) +
                                                             host_rankdef_off(g->L))
                                    : nullptr;
      for (int j = 0; j < nl; ++j) {
        qa.Pt[j] = lay(j)->pa; qa.P64[j] = lay(j)->pa; qa.P32[j] = lay(j)->P;
        qa.rankdef[j] = lay(j)->rankdef;
        qa.rankdef_host[j] = mirror ? mirror + sel[j] : nullptr;
      }
      return run(g, K_SMALL_QR, (16.0 * mr + 4.0 * mr) * nl, 4.0 * (2.0 * mr * r + rr * r / 3.0) * nl, s,
                 [&] { return cd::launch_small_cholqr(qa, nl, s); });
    }
    if (stage != 5) return CD_OK;
    cd_status st = gemm(K_PBTP, 2.0 * mn * r, 4.0 * mn + 8.0 * mr + 4.0 * nr, cd::GemmKind::F32_F64_TO_F32, n,
                        r, m, false, n, false, r, false,
                        [&](int j) { return static_cast<const void*>(M[sel[j]]); },
                        [&](int j) { return static_cast<const void*>(lay(j)->pa); },
                        [&](int j) { return static_cast<void*>(lay(j)->R); }, part);
    if (st != CD_OK) return st;
    cd::SmallUpdArgs ua{};
    ua.m = m; ua.n = n; ua.r = r;
    ua.one_minus_mu = static_cast<float>(1.0 - static_cast<double>(mu));
    ua.c = static_cast<float>(static_cast<double>(eta) * std::sqrt(static_cast<double>(m) / n));
    ua.g_bf16 = g->g_bf16 ? 1 : 0;
    ua.spec = spec;
    ua.ctl = run_if ? g->ctl : nullptr;
    bool reads_g = false;
    for (int j = 0; j < nl; ++j) {
      ua.M[j] = M[sel[j]]; ua.X[j] = X[sel[j]]; ua.P[j] = lay(j)->P; ua.R[j] = lay(j)->R; ua.Q[j] = Q[sel[j]];
      ua.G[j] = G[sel[j]];
      ua.gc[j] = spec != 0 ? eta_local(j) : 0.0f;
      ua.xdecay[j] = static_cast<float>(1.0 - static_cast<double>(eta) * lay(j)->d.weight_decay);
      reads_g = reads_g || (spec != 0 && eta_local(j) != 0.0f);
    }
    const double ub = (16.0 + (reads_g ? (g->g_bf16 ? 2.0 : 4.0) : 0.0)) * mn * nl + 8.0 * nr * nl;
    return run(g, K_SMALL_UPD, ub, 4.0 * mn * r * nl, s, [&] { return cd::launch_small_update(ua, nl, s); });
  }
  // bf16-gradient layers: the power-iteration products P~ = B Q and R = B^T P
  // use two-piece splits (three bf16 products, relative error about 2^-16,
  // an order below what the plain-bf16 rank-r update of M contributes);
  // fp32 layers keep fp64 (P~) and six-product (R) arithmetic.
  const bool fast = g->g_bf16;
  if (stage == 0) {
    // P~ = B Q (B lives in M): fp64 for fp32 layers, into pa; bf16 x 3 for
    // bf16-gradient layers, into the fp32 panel P
    if (fast)
      return gemm(K_PBQ_BF, 2.0 * mn * r, 4.0 * mn + 4.0 * nr + 4.0 * mr, cd::GemmKind::F32, m, r, n,
                  true, n, false, r, false,
                  [&](int j) { return static_cast<const void*>(M[sel[j]]); },
                  [&](int j) { return static_cast<const void*>(Q[sel[j]]); },
                  [&](int j) { return static_cast<void*>(lay(j)->P); }, part, 2);
    return gemm(K_PBQ, 2.0 * mn * r, 4.0 * mn + 4.0 * nr + 8.0 * mr, cd::GemmKind::F64_FROM_F32, m, r,
                n, true, n, false, r, false,
                [&](int j) { return static_cast<const void*>(M[sel[j]]); },
                [&](int j) { return static_cast<const void*>(Q[sel[j]]); },
                [&](int j) { return static_cast<void*>(lay(j)->pa); }, part);
  }
  if (stage == 1) {
    // the pass-0 Gram matrix to fp64 accuracy: kappa(P~) reaches 1e5-1e6 in
    // these streams.  bf16-gradient layers (fp32 P~): exact slice products on
    // the bf16 MFMA (k_gram.hip), 64 x 64 upper tiles split over K as the fp64
    // kernel's
    if (fast) {
      cd::GramXArgs xa{};
      xa.m = m; xa.r = r; xa.run_if = run_if;
      xa.mp = (m + cd::GX_CHUNK - 1) / cd::GX_CHUNK * cd::GX_CHUNK;
      plan_splits(r, r, m, nl, true, &xa.kchunk, 0, true);
      xa.kchunk = (xa.kchunk + cd::GX_CHUNK - 1) / cd::GX_CHUNK * cd::GX_CHUNK;
      xa.splits = (xa.mp + xa.kchunk - 1) / xa.kchunk;
      xa.split_stride = 1LL * r * r;
      if (xa.splits > 1) {
        const size_t need = static_cast<size_t>(xa.splits) * r * r;
        for (int j = 0; j < nl; ++j)
          if (need > lay(j)->gram_cap)
            return fail(CD_ENOMEM, "Gram workspace too small (%zu > %zu doubles)", need, lay(j)->gram_cap);
      }
      for (int j = 0; j < nl; ++j) {
        xa.P[j] = lay(j)->P;
        xa.S[j] = reinterpret_cast<__bf16*>(lay(j)->pa);
        xa.E[j] = reinterpret_cast<int*>(reinterpret_cast<char*>(lay(j)->pa) + 6LL * r * xa.mp);
        xa.C[j] = xa.splits > 1 ? static_cast<void*>(lay(j)->gram_part) : static_cast<void*>(lay(j)->W);
      }
      cd_status st = run(g, K_GRAM_X, (10.0 * mr + 8.0 * rr * xa.splits) * nl, mr * (r + 1) * nl, s,
                         [&] { return cd::launch_gram_x(xa, nl, s); });
      if (st != CD_OK || xa.splits == 1) return st;
      cd::ReduceArgs ra{};
      ra.count = 1LL * r * r; ra.stride = xa.split_stride; ra.splits = xa.splits; ra.run_if = run_if;
      for (int j = 0; j < nl; ++j) { ra.part[j] = lay(j)->gram_part; ra.out[j] = lay(j)->W; }
      return run(g, K_REDUCE, static_cast<double>(ra.count) * nl * 8.0 * (xa.splits + 1), 0.0, s,
                 [&] { return cd::launch_reduce_splits(ra, nl, true, true, s); });
    }
    return gemm(K_GRAM, mr * (r + 1), 8.0 * mr + 8.0 * rr, cd::GemmKind::F64, r, r, m, false, r, false,
                r, true, [&](int j) { return static_cast<const void*>(lay(j)->pa); },
                [&](int j) { return static_cast<const void*>(lay(j)->pa); },
                [&](int j) { return static_cast<void*>(lay(j)->W); },
                [&](int j) { return static_cast<void*>(lay(j)->gram_part); });
  }
  if (stage == 2 || stage == 4) {
    // apply an inverse factor: out = in U, U upper triangular (fp32-accurate).
    // Any error in U keeps span(out) and leaves the final Q-factor unchanged;
    // it only changes how close to orthonormal `out` is.
    if (!fast) return CD_OK;   // fp32 layers: fp64 triangular solves in enqueue_factor
    auto In = [&](int j) { return static_cast<const void*>(stage == 2 ? lay(j)->P : lay(j)->pb); };
    auto Out = [&](int j) { return static_cast<void*>(stage == 2 ? lay(j)->pb : lay(j)->P); };
    // U is upper triangular: output column j takes k <= j only
    return gemm(K_APPLY_BF, mr * r, 12.0 * mr + 4.0 * rr, cd::GemmKind::F32, m, r, r, true, r, false, r,
                false, In, [&](int j) { return static_cast<const void*>(lay(j)->Uf); }, Out, part, 3,
                false, true);
  }
  if (stage == 3) {
    if (!fast) {
      // fp32 layers: P1 is fp64, in pa
      auto In64 = [&](int j) { return static_cast<const void*>(lay(j)->pa); };
      return gemm(K_GRAM, mr * (r + 1), 8.0 * mr + 8.0 * rr, cd::GemmKind::F64, r, r, m, false, r, false,
                  r, true, In64, In64, [&](int j) { return static_cast<void*>(lay(j)->W); },
                  [&](int j) { return static_cast<void*>(lay(j)->gram_part); });
    }
    auto In = [&](int j) { return static_cast<const void*>(lay(j)->pb); };
    // pass-1 Gram matrix of the nearly orthonormal P1, fp32-accurate, into
    // fp64 W (all tiles: with upper tiles only the launch takes more K-splits
    // and their reduction costs more than the skipped tiles save)
    return gemm(K_GRAM_BF, 2.0 * mr * r, 4.0 * mr + 8.0 * rr, cd::GemmKind::F32, r, r, m, false, r, false,
                r, false, In, In, [&](int j) { return static_cast<void*>(lay(j)->W); }, part, 3, true);
  }
  // R = B^T P: bf16-gradient layers from the fp32 P with two-piece splits;
  // fp32 layers from the fp64 P on the fp64 MFMA (R_j = B^T P_j cancels for
  // the weak directions, by up to ||B||_2 / ||R_j||, which fp32 products and
  // sums would pass on to Q)
  cd_status st = fast
      ? gemm(K_PBTP3, 2.0 * mn * r, 4.0 * mn + 4.0 * mr + 4.0 * nr, cd::GemmKind::F32, n, r, m, false, n,
             false, r, false, [&](int j) { return static_cast<const void*>(M[sel[j]]); },
             [&](int j) { return static_cast<const void*>(lay(j)->P); },
             [&](int j) { return static_cast<void*>(lay(j)->R); }, part, 2)
      : gemm(K_PBTP, 2.0 * mn * r, 4.0 * mn + 8.0 * mr + 4.0 * nr, cd::GemmKind::F32_F64_TO_F32, n, r, m,
             false, n, false, r, false, [&](int j) { return static_cast<const void*>(M[sel[j]]); },
             [&](int j) { return static_cast<const void*>(lay(j)->pa); },
             [&](int j) { return static_cast<void*>(lay(j)->R); }, part);
  if (st != CD_OK) return st;
  // M = B - (1 - mu) P R^T;  X -= eta sqrt(m/n) P Q^T.  The rank-r
  // corrections are fp32-accurate (6 bf16 piece products) for fp32 layers and
  // plain bf16 products for bf16-gradient layers; P, R, Q are split into bf16
  // planes once, then streamed by the update.
  const int up = fast ? 1 : 3;
  const int rp = (r + 31) / 32 * 32;
  // fp32 layers at r <= 32: the update runs on the fp32 vector units and
  // reads P, R, Q as they are (no bf16 planes)
  const bool vec_update = !fast && cd::update_vec_fits(r);
  // Q = ColumnNormalize(R), with the planes of R and Q in the same pass
  cd::ColnormArgs cn{};
  cn.n = n; cn.r = r; cn.nchunks = (n + cd::COLNORM_ROWS - 1) / cd::COLNORM_ROWS;
  cn.S = vec_update ? 0 : up; cn.rp = rp;
  cn.run_if = run_if;
  for (int j = 0; j < nl; ++j) {
    cn.R[j] = lay(j)->R; cn.part[j] = lay(j)->colsq; cn.nrm[j] = lay(j)->colnrm; cn.Q[j] = Q[sel[j]];
    cn.Rpl[j] = lay(j)->planes + 3LL * m * rp;
    cn.Qpl[j] = lay(j)->planes + 3LL * m * rp + 3LL * n * rp;
  }
  st = run(g, K_COLNORM, (12.0 + 4.0 * cn.S) * nr * nl, 3.0 * nr * nl, s,
           [&] { return cd::launch_colnorm(cn, nl, s); });
  if (st != CD_OK) return st;
  bool reads_g = false;
  for (int j = 0; j < nl && spec != 0; ++j) reads_g = reads_g || eta_local(j) != 0.0f;
  cd::StepCtl* const uctl = run_if ? g->ctl : nullptr;
  const double ub = (16.0 + (reads_g ? (g->g_bf16 ? 2.0 : 4.0) : 0.0)) * mn * nl;
  if (vec_update) {
    cd::UpdateVecArgs va{};
    va.m = m; va.n = n; va.r = r;
    va.one_minus_mu = static_cast<float>(1.0 - static_cast<double>(mu));
    va.c = static_cast<float>(static_cast<double>(eta) * std::sqrt(static_cast<double>(m) / n));
    va.g_bf16 = g->g_bf16 ? 1 : 0;
    va.spec = spec;
    va.ctl = uctl;
    for (int j = 0; j < nl; ++j) {
      va.G[j] = G[sel[j]];
      va.gc[j] = spec != 0 ? eta_local(j) : 0.0f;
      va.xdecay[j] = static_cast<float>(1.0 - static_cast<double>(eta) * lay(j)->d.weight_decay);
      va.M[j] = M[sel[j]]; va.X[j] = X[sel[j]];
      va.P[j] = lay(j)->P; va.R[j] = lay(j)->R; va.Q[j] = Q[sel[j]];
    }
    return run(g, K_UPDATE_F32, ub, 4.0 * mn * r * nl, s, [&] { return cd::launch_update_vec(va, nl, s); });
  }
  {
    cd::PlaneArgs pa{};
    pa.r = r; pa.rp = rp; pa.S = up;
    pa.run_if = run_if;
    pa.rows = m;
    for (int j = 0; j < nl; ++j) { pa.src[j] = lay(j)->P; pa.dst[j] = lay(j)->planes; }
    st = run(g, K_COLNORM, (4.0 + 2.0 * up) * mr * nl, 0.0, s, [&] { return cd::launch_split_planes(pa, nl, s); });
    if (st != CD_OK) return st;
  }
  cd::UpdatePlArgs ua{};
  ua.m = m; ua.n = n; ua.r = r; ua.rp = rp;
  ua.one_minus_mu = static_cast<float>(1.0 - static_cast<double>(mu));
  ua.c = static_cast<float>(static_cast<double>(eta) * std::sqrt(static_cast<double>(m) / n));
  ua.g_bf16 = g->g_bf16 ? 1 : 0;
  ua.spec = spec;
  ua.ctl = uctl;
  for (int j = 0; j < nl; ++j) {
    ua.G[j] = G[sel[j]];
    ua.gc[j] = spec != 0 ? eta_local(j) : 0.0f;
    ua.xdecay[j] = static_cast<float>(1.0 - static_cast<double>(eta) * lay(j)->d.weight_decay);
    ua.M[j] = M[sel[j]]; ua.X[j] = X[sel[j]];
    ua.P[j] = lay(j)->planes;
    ua.R[j] = lay(j)->planes + 3LL * m * rp;
    ua.Q[j] = lay(j)->planes + 3LL * m * rp + 3LL * n * rp;
  }
  return run(g, fast ? K_UPDATE_BF1 : K_UPDATE, ub, 4.0 * mn * r * nl, s,
             [&] { return cd::launch_update_planes(ua, nl, up, s); });
}

// Between the stages of CholQR pass `pass`, over every layer: Cholesky of each
// W, then either the fp64 triangular solve (fp32 layers: P1 = P~ T^-1, then
// P = P1 T^-1) or the inverse U = T^-1 in fp32 for the bf16 x 6 apply.  The
// second pass of fp32 layers, whose W = P1^T P1 is the identity to about
// kappa^2 u_fp64, factors W by the near-identity iteration; the blocked
// factorisation then runs only for layers where W is too far from I.
cd_status enqueue_factor(cd_group* g, const Unit& u, int r, int pass, hipStream_t s, const int* run_if) {
  const int nl = static_cast<int>(u.sel.size());
  const double L = nl, rr = 1.0 * r * r;
  const cd::CholTab* ct = g->chol_tab + u.off;
  const bool nearid = pass == 1 && !g->g_bf16;
  cd_status st = run(g, K_CHOL, 16.0 * rr * L, (1.0 / 3.0) * rr * r * L, s, [&] {
    if (nearid) {
      const hipError_t e = cd::launch_nearid(ct, nl, r, s, run_if);
      if (e != hipSuccess) return e;
    }
    return cd::launch_cholesky(ct, nl, r, pass, s, run_if, nearid);
  });
  if (st != CD_OK) return st;
  if (!g->g_bf16) {
    // in place in the fp64 panel: P1 = P~ T^-1 (pass 0), P = P1 T1^-1 (pass 1)
    double flops = 0, bytes = 0;
    for (int li : u.sel) {
      const double mr = 1.0 * g->layers[li]->d.m * r;
      flops += mr * r;
      bytes += 16.0 * mr + 8.0 * rr;
    }
    st = run(g, K_TRSM, bytes, flops, s, [&] {
      return cd::launch_trsm_rl(g->trsm_tab[pass == 0 ? 0 : 2] + u.off, g->trsm_tiles + u.toff, u.nt, r, s,
                                run_if);
    });
    if (st != CD_OK || pass == 0) return st;
    // P rounded to fp32 (the update's operand planes and cd_layer_last_factors)
    cd::ReduceArgs ra{};
    ra.count = 1LL * g->shapes[u.sc].m * r;
    ra.stride = ra.count;
    ra.splits = 1;
    ra.run_if = run_if;
    for (int j = 0; j < nl; ++j) {
      ra.part[j] = g->layers[u.sel[j]]->pa;
      ra.out[j] = g->layers[u.sel[j]]->P;
    }
    return run(g, K_REDUCE, 12.0 * ra.count * nl, 0.0, s,
               [&] { return cd::launch_reduce_splits(ra, nl, true, false, s); });
  }
  return run(g, K_TRTRI, 12.0 * rr * L, rr * r / 3.0 * L, s, [&] {
    return cd::launch_trsm(g->trsm_tab[1] + u.off, g->trtri_tiles + u.rtoff, u.nrt, r, true, false, s, true, r,
                           run_if);
  });
}

// Argument checks shared by every step entry point (nothing is enqueued yet).
cd_status check_step_args(const cd_group* g, const void* const* G, float* const* M, float* const* X,
                          float* const* Q, float mu, float eta, int r) {
  if (!G || !M || !X || !Q) return fail(CD_EINVAL, "pointer array is NULL");
  if (!(mu >= 0.0f && mu <= 1.0f)) return fail(CD_EINVAL, "mu must be in [0, 1] (got %g)", mu);
  if (!std::isfinite(eta) || eta < 0.0f) return fail(CD_EINVAL, "eta must be finite and >= 0 (got %g)", eta);
  if (r < 1) return fail(CD_EINVAL, "r must be >= 1 (got %d)", r);
  for (int i = 0; i < g->L; ++i) {
    const cd_layer* L = g->layers[i];
    if (r > L->d.r_max) return fail(CD_EINVAL, "r = %d exceeds r_max = %d of layer %d", r, L->d.r_max, i);
    if (!G[i] || !M[i] || !X[i] || !Q[i]) return fail(CD_EINVAL, "NULL matrix pointer for layer %d", i);
    if (!aligned16(G[i]) || !aligned16(M[i]) || !aligned16(X[i]) || !aligned16(Q[i]))
      return fail(CD_EINVAL, "matrix pointers of layer %d must be 16-byte aligned", i);
  }
  return CD_OK;
}

// 1. B = M + G, partial sums of B^2 and, by spec_mode, the skip branch's X
// update in the same pass (0: no, 1: yes, 2: as the control word predicts).
cd_status enqueue_form(cd_group* g, const void* const* G, float* const* M, float* const* X, float eta,
                       int spec_mode, hipStream_t s) {
  const bool with_x = spec_mode == 1 || (spec_mode == 2 && g->predict_skip);   // for the byte count
  for (const std::vector<int>& batch : g->sbatches) {
    const int nl = static_cast<int>(batch.size());
    cd::FormArgs fa{};
    fa.nl = nl;
    fa.ctl = g->ctl;
    long long total = 0, blocks = 0;
    for (int j = 0; j < nl; ++j) {
      const int li = batch[j];
      const cd_layer* Ly = g->layers[li];
      fa.numel[j] = 1LL * Ly->d.m * Ly->d.n;
      fa.block0[j] = static_cast<int>(blocks);
      blocks += blocks_for(fa.numel[j]);
      total += fa.numel[j];
      fa.M[j] = M[li]; fa.G[j] = G[li]; fa.part[j] = g->parts + 1LL * li * g->nparts_stride;
      fa.X[j] = X[li];
      fa.coef[j] = static_cast<float>(Ly->d.eta_local_scale * static_cast<double>(eta));
      fa.xdecay[j] = static_cast<float>(1.0 - static_cast<double>(eta) * Ly->d.weight_decay);
    }
    fa.block0[nl] = static_cast<int>(blocks);
    const double fb = static_cast<double>(total) * ((with_x ? 16.0 : 8.0) + (g->g_bf16 ? 2.0 : 4.0));
    cd_status st = run(g, with_x ? K_FORM_X : K_FORM, fb, (with_x ? 5.0 : 3.0) * total, s,
                       [&] { return cd::launch_form_buffer(fa, g->g_bf16, spec_mode, s); });
    if (st != CD_OK) return st;
  }
  return CD_OK;
}

// Whether a step at rank r can take the fused buffer pass + P~ = B Q:
// bf16-gradient layers with r in (256, 512] whose split partials fit.
bool fused_fits(const cd_group* g, int r) {
  if (g->np_fx.empty() || r < cd::FBQ_RMIN || r > cd::FBQ_RMAX) return false;
  for (const Unit& u : g->units) {
    const int m = g->shapes[u.sc].m;
    if (u.fbq_splits > 1)
      for (int li : u.sel)
        if (static_cast<size_t>(u.fbq_splits) * m * r * sizeof(float) > g->layers[li]->split_cap) return false;
  }
  return true;
}

// 1'. B = M + G fused into P~ = B Q (k_form_bq.hip), per unit on the unit's
// stream of the sync branch (forked from s and joined back to it here), then
// the split partials of P~ added in split order into P.
cd_status enqueue_form_bq(cd_group* g, const void* const* G, float* const* M, float* const* Q, int r,
                          hipStream_t s) {
  const int nu = static_cast<int>(g->units.size());
  const int nside = (g->timer.on && g->timer.mask == ~0u) ? 0 : g->nside;
  auto stream_of = [&](int u) -> hipStream_t {
    const int k = u % (nside + 1);
    return k == 0 ? s : g->side[k - 1];
  };
  if (nside > 0) {
    CD_HIP(hipEventRecord(g->fork_ev, s));
    for (int i = 0; i < nside; ++i) CD_HIP(hipStreamWaitEvent(g->side[i], g->fork_ev, 0));
  }
  for (int ui = 0; ui < nu; ++ui) {
    const Unit& u = g->units[ui];
    const hipStream_t su = stream_of(ui);
    const int m = g->shapes[u.sc].m, n = g->shapes[u.sc].n, nl = static_cast<int>(u.sel.size());
    cd::FormBqArgs fa{};
    fa.m = m; fa.n = n; fa.r = r;
    fa.splits = u.fbq_splits; fa.kchunk = u.fbq_kchunk;
    fa.split_stride = 1LL * m * r;
    for (int j = 0; j < nl; ++j) {
      cd_layer* Ly = g->layers[u.sel[j]];
      fa.M[j] = M[u.sel[j]];
      fa.G[j] = static_cast<const __bf16*>(G[u.sel[j]]);
      fa.Q[j] = Q[u.sel[j]];
      fa.C[j] = fa.splits > 1 ? static_cast<float*>(Ly->split_part) : Ly->P;
      fa.part[j] = g->parts + 1LL * u.sel[j] * g->nparts_stride;
    }
    const double mn = 1.0 * m * n, mr = 1.0 * m * r, nr = 1.0 * n * r;
    cd_status st = run(g, K_FORM_BQ, (10.0 * mn + 4.0 * nr + 4.0 * mr) * nl, 2.0 * mn * r * nl, su,
                       [&] { return cd::launch_form_bq(fa, nl, su); });
    if (st != CD_OK) return st;
    if (fa.splits > 1) {
      cd::ReduceArgs ra{};
      ra.count = 1LL * m * r; ra.stride = fa.split_stride; ra.splits = fa.splits; ra.run_if = nullptr;
      for (int j = 0; j < nl; ++j) {
        ra.part[j] = g->layers[u.sel[j]]->split_part;
        ra.out[j] = g->layers[u.sel[j]]->P;
      }
      st = run(g, K_REDUCE, static_cast<double>(ra.count) * nl * 4.0 * (fa.splits + 1), 0.0, su,
               [&] { return cd::launch_reduce_splits(ra, nl, false, false, su); });
      if (st != CD_OK) return st;
    }
  }
  for (int i = 0; i < nside; ++i) {
    CD_HIP(hipEventRecord(g->join_ev[i], g->side[i]));
    CD_HIP(hipStreamWaitEvent(s, g->join_ev[i], 0));
  }
  return CD_OK;
}

// 2. the gate: norms, RMMC, prev_norm, max, the branch (g > tau, or
// fixed_flag >= 0 for a fixed policy) into g->out_dev and the control word;
// with to_host also into the pinned block, followed by the step's sequence
// number.
// fused: the partials come from the fused buffer pass + P~ = B Q.
cd_status enqueue_gate(cd_group* g, hipStream_t s, bool to_host, int spec_mode, int fixed_flag,
                       bool fused = false) {
  cd::GateArgs ga{};
  ga.L = g->L; ga.nparts_stride = g->nparts_stride; ga.parts = g->parts;
  ga.nparts = fused ? g->nparts_fx : g->nparts;
  ga.prev = g->prev; ga.eps = g->eps; ga.tau = g->tau; ga.out = g->out_dev;
  ga.norms = g->norms; ga.counter = g->counter;
  ga.ctl = g->ctl; ga.spec_mode = spec_mode; ga.fixed_flag = fixed_flag;
  if (to_host) {
    ga.host_out = static_cast<cd::GateOut*>(g->out_host_dev);
    ga.host_seq = reinterpret_cast<unsigned long long*>(static_cast<char*>(g->out_host_dev) + host_seq_off(g->L));
    ga.seq = ++g->seq;
  }
  return run(g, K_GATE, 8.0 * g->L * g->nparts_stride, 0.0, s, [&] { return cd::launch_gate(ga, s); });
}

// 4. the branch.  BR_SYNC: the sync branch per unit (each unit's pipeline
// on its own stream, forked from and joined back to s).  BR_LOCAL: the
// stand-alone local update, unless spec already applied it in the buffer
// pass.  BR_BOTH (the decision is not known on the host): both, every kernel
// predicated on the control word, spec taken from it.
enum Branch { BR_LOCAL = 0, BR_SYNC = 1, BR_BOTH = 2 };

// fused: P~ = B Q of every unit already came out of the fused buffer pass.
cd_status enqueue_branch(cd_group* g, int branch, int spec, const void* const* G, float* const* M,
                         float* const* X, float* const* Q, float mu, float eta, int r, hipStream_t s,
                         bool fused = false) {
  if (branch == BR_LOCAL || branch == BR_BOTH) {
    for (const std::vector<int>& batch : g->sbatches) {
      if (branch == BR_LOCAL && spec != 0) break;
      const int nl = static_cast<int>(batch.size());
      cd::LocalArgs la{};
      la.nl = nl;
      la.ctl = branch == BR_BOTH ? g->ctl : nullptr;
      long long total = 0, blocks = 0;
      for (int j = 0; j < nl; ++j) {
        const int li = batch[j];
        const cd_layer* Ly = g->layers[li];
        la.numel[j] = 1LL * Ly->d.m * Ly->d.n;
        la.block0[j] = static_cast<int>(blocks);
        blocks += blocks_for(la.numel[j]);
        total += la.numel[j];
        la.X[j] = X[li]; la.G[j] = G[li];
        la.coef[j] = static_cast<float>(Ly->d.eta_local_scale * static_cast<double>(eta));
        la.xdecay[j] = static_cast<float>(1.0 - static_cast<double>(eta) * Ly->d.weight_decay);
      }
      la.block0[nl] = static_cast<int>(blocks);
      const double lb = static_cast<double>(total) * (8.0 + (g->g_bf16 ? 2.0 : 4.0));
      cd_status st = run(g, K_LOCAL, lb, 2.0 * total, s,
                         [&] { return cd::launch_local_update(la, g->g_bf16, s); });
      if (st != CD_OK) return st;
    }
  }
  if (branch == BR_SYNC || branch == BR_BOTH) {
    const int* run_if = branch == BR_BOTH ? &g->ctl->flag : nullptr;
    const int uspec = branch == BR_BOTH ? 2 : spec;
    // Each unit's pipeline in stage order on its own stream: the first unit
    // on the caller's stream, the others on the group's side streams, forked
    // from the caller's stream here and joined back to it below.  Units are
    // independent (no workspace is shared between layers), so the results do
    // not depend on how their kernels interleave.
    // While every kernel kind is bracketed by timing events, the units run
    // one after another on the caller's stream, so that each bracketed
    // launch times its kernel alone (not its wait for CUs that another
    // stream's kernels hold).
    const int nu = static_cast<int>(g->units.size());
    const int nside = (g->timer.on && g->timer.mask == ~0u) ? 0 : g->nside;
    auto stream_of = [&](int u) -> hipStream_t {
      const int k = u % (nside + 1);
      return k == 0 ? s : g->side[k - 1];
    };
    if (nside > 0) {
      CD_HIP(hipEventRecord(g->fork_ev, s));
      for (int i = 0; i < nside; ++i) CD_HIP(hipStreamWaitEvent(g->side[i], g->fork_ev, 0));
    }
    for (int stage = fused ? 1 : 0; stage < 6; ++stage) {
      for (int ui = 0; ui < nu; ++ui) {
        const Unit& u = g->units[ui];
        const hipStream_t su = stream_of(ui);
        cd_status st = enqueue_sync(g, g->shapes[u.sc], u.sel, G, uspec, M, X, Q, mu, eta, r, stage, su, run_if);
        if (st != CD_OK) return st;
        if (cd::small_sync_fits(g->shapes[u.sc].m, g->shapes[u.sc].n, r)) continue;
        if (stage == 1 || stage == 3) {
          st = enqueue_factor(g, u, r, stage == 1 ? 0 : 1, su, run_if);
          if (st != CD_OK) return st;
        }
        if (stage == 2) {
          // P1 is complete for the unit: new directions for the columns of
          // floored pass-0 pivots (layers without any return at once)
          const int nl = static_cast<int>(u.sel.size());
          const int mu_rows = g->shapes[u.sc].m;
          st = run(g, K_CHOL, 4.0 * nl, 0.0, su, [&] {
            return cd::launch_fill_dead(g->chol_tab + u.off, g->trsm_tab[0] + u.off, nl, mu_rows, r,
                                        !g->g_bf16, su, run_if);
          });
          if (st != CD_OK) return st;
        }
      }
    }
    for (int i = 0; i < nside; ++i) {
      CD_HIP(hipEventRecord(g->join_ev[i], g->side[i]));
      CD_HIP(hipStreamWaitEvent(s, g->join_ev[i], 0));
    }
    for (cd_layer* Ly : g->layers) Ly->last_r = r;
  }
  return CD_OK;
}

// The branch a fixed policy takes at step `step` (1-based); RMMC: unknown.
bool fixed_policy(const cd_group* g) { return g->policy != CD_POLICY_RMMC; }
bool fixed_sync(const cd_group* g, long long step) {
  return g->policy == CD_POLICY_ALWAYS_SYNC || (g->policy == CD_POLICY_EVERY_H && step % g->H == 0);
}

// Waits for the gate output of the group's last step in the pinned block
// (the event after the gate bounds the wait: once it has completed, the
// output is there or the step failed).
cd_status wait_gate(cd_group* g) {
  const volatile unsigned long long* hs = reinterpret_cast<const volatile unsigned long long*>(
      static_cast<const char*>(g->out_host) + host_seq_off(g->L));
  for (unsigned polls = 1; *hs != g->seq; ++polls) {
    if (polls % 4096 != 0) continue;
    const hipError_t q = hipEventQuery(g->ev);
    if (q == hipErrorNotReady) continue;
    if (q != hipSuccess) return fail(CD_EHIP, "gate: %s", hipGetErrorString(q));
    if (*hs != g->seq) return fail(CD_EHIP, "gate output did not reach host memory");
  }
  std::atomic_thread_fence(std::memory_order_acquire);
  return CD_OK;
}

// The step's results from the pinned block (after wait_gate).
const cd::GateOut* gate_out(const cd_group* g) { return static_cast<const cd::GateOut*>(g->out_host); }

cd_status group_step_impl(cd_group* g, const void* const* G, float* const* M, float* const* X,
                          float* const* Q, float mu, float eta, int r, void* stream,
                          double* rmmc_per_layer, cd_result* out) {
  if (!g) return fail(CD_EINVAL, "group is NULL");
  cd_status st = check_step_args(g, G, M, X, Q, mu, eta, r);
  if (st != CD_OK) return st;
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CD_EHIP, "cannot select device %d", g->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // a step with no host output is asynchronous: everything is enqueued and
  // nothing waits; cd_group_last_result reads the outcome later
  const bool blocking = out != nullptr || rmmc_per_layer != nullptr;

  // Skip-branch speculation: when the coming decision is known or predicted
  // to be "skip", X -= eta_local G rides along in the buffer pass, which saves
  // the second read of G; should the step sync after all, the sync update
  // first adds eta_local G back (in fp32, one rounding).  The RMMC policy
  // predicts the previous step's branch, except that a layer whose prev_norm
  // is 0 (its first step) has RMMC = ||B|| / eps: that step syncs unless B = 0.
  // When the host has not read the previous decision (after an asynchronous
  // step) the buffer pass takes the same prediction from the control word.
  const long long next_step = g->layers[0]->step + 1;
  bool any_prev_zero = false;
  for (const cd_layer* Ly : g->layers) any_prev_zero = any_prev_zero || Ly->prev_zero;
  const bool fixed = fixed_policy(g);
  const bool fsync = fixed && fixed_sync(g, next_step);
  int spec_mode;
  if (fixed) spec_mode = fsync ? 0 : 1;
  else if (any_prev_zero) spec_mode = 0;
  else if (g->pred_known) spec_mode = g->predict_skip ? 1 : 0;
  else spec_mode = 2;

  // A step that syncs for certain -- a fixed policy's sync step, or a layer's
  // first step (prev_norm = 0: RMMC = ||B|| / eps) -- forms B inside
  // P~ = B Q when the layers allow it (bf16 gradients, 256 < r <= 512): M and
  // G are streamed once, and P~ is ready when the gate decides.  A sync that
  // is only predicted (the previous step synced) takes the plain buffer pass:
  // the step after a sync usually skips, and a misprediction would waste the
  // whole product.  (Should a first step skip after all, B = 0, P~ is unused
  // workspace and the local branch finds M = B as after a plain buffer pass.)
  const bool fused = spec_mode == 0 && (fixed ? fsync : (blocking && any_prev_zero)) && fused_fits(g, r);
  st = fused ? enqueue_form_bq(g, G, M, Q, r, s) : enqueue_form(g, G, M, X, eta, spec_mode, s);
  if (st != CD_OK) return st;
  st = enqueue_gate(g, s, true, spec_mode, fixed ? (fsync ? 1 : 0) : -1, fused);
  if (st != CD_OK) return st;
  CD_HIP(hipEventRecord(g->ev, s));
  for (int i = 0; i < g->L; ++i) {
    cd_layer* L = g->layers[i];
    L->step += 1;
    L->prev_zero = false;
    L->last_group = g;
    L->last_index = i;
  }
  g->stepped = true;

  // ALWAYS, NEVER and EVERY_H fix the branch in advance, and an asynchronous
  // step enqueues both branches predicated on the control word: either way
  // the branch is enqueued before any wait for the gate's output, so the GPU
  // does not idle through the round trip.  A blocking RMMC step decides on
  // the output (3. the decision point, standing in for the max all-reduce).
  bool sync = fsync;
  if (fixed) {
    st = enqueue_branch(g, fsync ? BR_SYNC : BR_LOCAL, spec_mode, G, M, X, Q, mu, eta, r, s, fused);
    if (st != CD_OK) return st;
  } else if (!blocking) {
    st = enqueue_branch(g, BR_BOTH, 2, G, M, X, Q, mu, eta, r, s);
    if (st != CD_OK) return st;
  }
  if (blocking) {
    st = wait_gate(g);
    if (st != CD_OK) return st;
    const cd::GateOut* go = gate_out(g);
    if (!fixed) {
      sync = go->flag != 0;
      st = enqueue_branch(g, sync ? BR_SYNC : BR_LOCAL, go->spec, G, M, X, Q, mu, eta, r, s, fused);
      if (st != CD_OK) return st;
    }
    if (rmmc_per_layer) std::memcpy(rmmc_per_layer, go + 1, sizeof(double) * g->L);
    if (out) { out->rmmc = go->g; out->sync_flag = sync ? 1 : 0; }
  }
  CD_HIP(hipEventRecord(g->done_ev, s));
  if (fixed || blocking) {
    g->pred_known = true;
    g->predict_skip = !sync;
  } else {
    g->pred_known = false;
  }
  if (blocking && gate_out(g)->nonfinite != 0) return fail(CD_ENONFINITE, "a layer norm ||B|| was not finite");
  return CD_OK;
}

// The outcome of the group's last step: waits for that step's last kernel
// (its completion event, not the device), then reads the pinned block.
cd_status group_last_result(cd_group* g, double* rmmc_per_layer, cd_result* out) {
  if (!g) return fail(CD_EINVAL, "group is NULL");
  if (!g->stepped) return fail(CD_EINVAL, "the group has not been stepped");
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CD_EHIP, "cannot select device %d", g->device);
  CD_HIP(hipEventSynchronize(g->done_ev));
  cd_status st = wait_gate(g);
  if (st != CD_OK) return st;
  const cd::GateOut* go = gate_out(g);
  if (rmmc_per_layer) std::memcpy(rmmc_per_layer, go + 1, sizeof(double) * g->L);
  if (out) { out->rmmc = go->g; out->sync_flag = go->flag; }
  g->pred_known = true;
  g->predict_skip = go->flag == 0;
  if (go->nonfinite) return fail(CD_ENONFINITE, "a layer norm ||B|| was not finite");
  if (go->flag) {
    const int* rd = reinterpret_cast<const int*>(static_cast<const char*>(g->out_host) + host_rankdef_off(g->L));
    for (int i = 0; i < g->L; ++i)
      if (rd[i]) return fail(CD_ERANKDEF, "layer %d: P~ was numerically rank deficient", i);
  }
  return CD_OK;
}

// ---- the allocation-free step (cd_step_static) -------------------------------
// All workspace of one layer's step and the device tables of its one-layer
// group live in one fixed array per device.  Host code never uses the
// array's name as an address: its device address comes from
// hipGetSymbolAddress, once per device, and every kernel argument is carved
// from that address.
static __device__ __align__(256) unsigned char scratch[CD_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

// Per device: the array's device address and the host-side layer and group
// objects the step reuses (their vectors keep their one-element capacity, so
// a call after the first allocates nothing on the host either).
struct StaticSlot {
  std::mutex mu;
  void* base = nullptr;
  cd_layer layer;
  cd_group group;
};
StaticSlot g_static[kMaxDevices];

// Writes the one-layer group's device tables (a kernel instead of host-to-
// device copies, so that the step needs no staging memory).
struct StaticSetup {
  int* nparts;
  int np;
  double** prev_tab;
  double* prev;
  unsigned* counter;
  cd::CholTab* ct;
  cd::CholTab ctv;
  cd::TrsmTab* tt[3];
  cd::TrsmTab ttv[3];
  int2* tiles;
  int ntiles;
  int2* rtiles;
  int nrtiles;
};

__global__ __launch_bounds__(256) void k_static_setup(StaticSetup a) {
  const int t = threadIdx.x;
  if (t == 0) {
    *a.nparts = a.np;
    *a.prev_tab = a.prev;
    *a.counter = 0u;   // the gate's completion counter starts at zero
    *a.ct = a.ctv;
    for (int k = 0; k < 3; ++k) *a.tt[k] = a.ttv[k];
  }
  for (int i = t; i < a.ntiles; i += 256) a.tiles[i] = int2{0, i};
  for (int i = t; i < a.nrtiles; i += 256) a.rtiles[i] = int2{0, i};
}

// The one-layer group of a static step, planned in place.
void plan_static(cd_group* g, cd_layer* L, int r, int ntiles, int nrtiles) {
  g->layers.resize(1);
  g->layers[0] = L;
  g->L = 1;
  g->device = L->device;
  g->g_bf16 = L->d.grad_dtype == CD_BF16;
  g->tau = L->d.tau;
  g->eps = L->d.eps;
  g->policy = L->d.policy;
  g->H = L->d.H;
  g->nparts_stride = static_cast<int>(blocks_for(1LL * L->d.m * L->d.n));
  g->shapes.resize(1);
  g->shapes[0].m = L->d.m;
  g->shapes[0].n = L->d.n;
  g->shapes[0].idx.resize(1);
  g->shapes[0].idx[0] = 0;
  g->units.resize(1);
  Unit& u = g->units[0];
  u.sc = 0;
  u.sel.resize(1);
  u.sel[0] = 0;
  u.off = 0;
  u.toff = 0;
  u.nt = ntiles;
  u.rtoff = 0;
  u.nrt = nrtiles;
  g->sbatches.resize(1);
  g->sbatches[0].resize(1);
  g->sbatches[0][0] = 0;
  g->nside = 0;
  g->out_host = nullptr;
  g->out_host_dev = nullptr;
  g->ev = nullptr;
  g->timer.on = false;
  (void)r;
}

cd_status static_step_impl(const cd_layer_desc* desc, double* prev_norm, long long* step, const void* G,
                           float* M, float* X, float* Q, float mu, float eta, int r, void* stream,
                           cd_result* out) {
  cd_status st = check_desc(desc);
  if (st != CD_OK) return st;
  if (!prev_norm || !step) return fail(CD_EINVAL, "prev_norm and step must not be NULL");
  if ((reinterpret_cast<uintptr_t>(prev_norm) & 7u) != 0) return fail(CD_EINVAL, "prev_norm must be 8-byte aligned");
  if (*step < 0) return fail(CD_EINVAL, "step must be >= 0");
  if (r < 1 || r > desc->r_max) return fail(CD_EINVAL, "r must be in [1, r_max] (got %d)", r);
  const int m = desc->m, n = desc->n;
  const int ntiles = (m + cd::CHOL_BLOCK - 1) / cd::CHOL_BLOCK;
  const int nrtiles = (r + cd::CHOL_BLOCK - 1) / cd::CHOL_BLOCK;
  const LayerLayout lo = layer_layout(m, n, r);
  const GroupLayout glo = group_layout(1, static_cast<int>(blocks_for(1LL * m * n)), ntiles, nrtiles);
  const size_t need = lo.total + glo.total;
  if (need > CD_STATIC_SCRATCH_BYTES)
    return fail(CD_EINVAL,
                "a %d x %d layer at rank %d needs %zu bytes of workspace; the allocation-free step has "
                "%zu (CD_STATIC_SCRATCH_BYTES): use cd_step",
                m, n, r, need, static_cast<size_t>(CD_STATIC_SCRATCH_BYTES));
  int dev = -1;
  CD_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(CD_EINVAL, "device %d is beyond the %d supported", dev, kMaxDevices);
  StaticSlot& slot = g_static[dev];
  std::lock_guard<std::mutex> lock(slot.mu);
  if (!slot.base) {
    void* ptr = nullptr;
    CD_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    slot.base = ptr;
  }
  char* base = static_cast<char*>(slot.base);
  cd_layer* L = &slot.layer;
  L->d = *desc;
  L->d.r_max = r;   // the workspace is laid out for this rank
  L->device = dev;
  L->step = *step;
  carve_layer(L, base, lo);
  L->prev = prev_norm;
  L->prev_zero = false;
  cd_group* g = &slot.group;
  plan_static(g, L, r, ntiles, nrtiles);
  carve_group(g, base + lo.total, glo);
  const void* Ga[1] = {G};
  float* Ma[1] = {M};
  float* Xa[1] = {X};
  float* Qa[1] = {Q};
  st = check_step_args(g, Ga, Ma, Xa, Qa, mu, eta, r);
  if (st != CD_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);

  StaticSetup su{};
  su.nparts = g->nparts;
  su.np = g->nparts_stride;
  su.prev_tab = g->prev;
  su.prev = prev_norm;
  su.counter = g->counter;
  su.ct = g->chol_tab;
  su.ctv = cd::CholTab{L->W, L->Dinv, L->floor_, L->rankdef, L->rowok, nullptr, L->gram_part, L->nid_ok};
  su.tt[0] = g->trsm_tab[0];
  su.tt[1] = g->trsm_tab[1];
  su.tt[2] = g->trsm_tab[2];
  factor_tabs(L, su.ttv[0], su.ttv[1], su.ttv[2]);
  su.tiles = g->trsm_tiles;
  su.ntiles = ntiles;
  su.rtiles = g->trtri_tiles;
  su.nrtiles = nrtiles;
  hipLaunchKernelGGL(k_static_setup, dim3(1), dim3(256), 0, s, su);
  CD_HIP(hipGetLastError());

  // no branch prediction without state between calls: the buffer pass fuses
  // the skip update only when a fixed policy says the step is local
  const long long next_step = *step + 1;
  const bool fixed = fixed_policy(g);
  const bool spec = fixed && !fixed_sync(g, next_step);
  st = enqueue_form(g, Ga, Ma, Xa, eta, spec ? 1 : 0, s);
  if (st != CD_OK) return st;
  st = enqueue_gate(g, s, false, spec ? 1 : 0, fixed ? (fixed_sync(g, next_step) ? 1 : 0) : -1);
  if (st != CD_OK) return st;
  struct { cd::GateOut h; double rm; } hb;
  CD_HIP(hipMemcpyAsync(&hb, g->out_dev, sizeof(hb), hipMemcpyDeviceToHost, s));
  CD_HIP(hipStreamSynchronize(s));
  *step = next_step;
  const bool sync = hb.h.flag != 0;
  st = enqueue_branch(g, sync ? BR_SYNC : BR_LOCAL, spec ? 1 : 0, Ga, Ma, Xa, Qa, mu, eta, r, s);
  if (st != CD_OK) return st;
  if (out) { out->rmmc = hb.h.g; out->sync_flag = sync ? 1 : 0; }
  if (hb.h.nonfinite) return fail(CD_ENONFINITE, "the layer norm ||B|| was not finite");
  return CD_OK;
}

}  // namespace

extern "C" {

cd_status cd_layer_create(const cd_layer_desc* desc, cd_layer** out) {
  try {
    if (!out) return fail(CD_EINVAL, "out is NULL");
    *out = nullptr;
    cd_status st = check_desc(desc);
    if (st != CD_OK) return st;
    cd_layer* L = new (std::nothrow) cd_layer();
    if (!L) return fail(CD_ENOMEM, "host allocation failed");
    L->d = *desc;
    if (hipGetDevice(&L->device) != hipSuccess) { delete L; return fail(CD_EHIP, "hipGetDevice failed"); }
    const LayerLayout lo = layer_layout(desc->m, desc->n, desc->r_max);
    hipError_t e = hipMalloc(&L->ws, lo.total);
    if (e == hipSuccess) {
      carve_layer(L, static_cast<char*>(L->ws), lo);
      e = hipMemset(L->prev, 0, sizeof(double));
    }
    if (e == hipSuccess) e = hipMemset(L->rankdef, 0, sizeof(int));
    if (e != hipSuccess) {
      free_layer(L);
      return fail(e == hipErrorOutOfMemory ? CD_ENOMEM : CD_EHIP, "layer allocation: %s",
                  hipGetErrorString(e));
    }
    cd_layer* arr[1] = {L};
    st = build_group(arr, 1, &L->self);
    if (st != CD_OK) { free_layer(L); return st; }
    *out = L;
    return CD_OK;
  } catch (...) {
    return fail(CD_ENOMEM, "exception in cd_layer_create");
  }
}

cd_status cd_step(cd_layer* layer, const void* G, float* M, float* X, float* Q, float mu, float eta,
                  int r, void* stream, cd_result* out) {
  try {
    if (!layer) return fail(CD_EINVAL, "layer is NULL");
    const void* Ga[1] = {G};
    float* Ma[1] = {M};
    float* Xa[1] = {X};
    float* Qa[1] = {Q};
    return group_step_impl(layer->self, Ga, Ma, Xa, Qa, mu, eta, r, stream, nullptr, out);
  } catch (...) {
    return fail(CD_ENOMEM, "exception in cd_step");
  }
}

cd_status cd_step_static(const cd_layer_desc* desc, double* prev_norm, long long* step, const void* G,
                         float* M, float* X, float* Q, float mu, float eta, int r, void* stream,
                         cd_result* out) {
  try {
    return static_step_impl(desc, prev_norm, step, G, M, X, Q, mu, eta, r, stream, out);
  } catch (...) {
    return fail(CD_ENOMEM, "exception in cd_step_static");
  }
}

cd_status cd_destroy(cd_layer* layer) {
  if (!layer) return CD_OK;
  DeviceGuard dg(layer->device);
  free_group(layer->self);
  free_layer(layer);
  return CD_OK;
}

cd_status cd_group_create(cd_layer* const* layers, int n_layers, cd_group** out) {
  try {
    if (!out) return fail(CD_EINVAL, "out is NULL");
    *out = nullptr;
    if (!layers || n_layers < 1) return fail(CD_EINVAL, "need at least one layer");
    if (n_layers > 4096) return fail(CD_EINVAL, "at most 4096 layers per group");
    for (int i = 0; i < n_layers; ++i) {
      if (!layers[i]) return fail(CD_EINVAL, "layer %d is NULL", i);
      const cd_layer_desc& a = layers[0]->d;
      const cd_layer_desc& b = layers[i]->d;
      if (a.grad_dtype != b.grad_dtype || a.tau != b.tau || a.policy != b.policy ||
          (a.policy == CD_POLICY_EVERY_H && a.H != b.H) || a.eps != b.eps ||
          layers[i]->device != layers[0]->device)
        return fail(CD_EINVAL, "layer %d differs from layer 0 in dtype, tau, eps, policy, H or device", i);
      for (int j = 0; j < i; ++j)
        if (layers[j] == layers[i]) return fail(CD_EINVAL, "layer %d appears twice", i);
    }
    return build_group(layers, n_layers, out);
  } catch (...) {
    return fail(CD_ENOMEM, "exception in cd_group_create");
  }
}

cd_status cd_group_step(cd_group* group, const void* const* G, float* const* M, float* const* X,
                        float* const* Q, float mu, float eta, int r, void* stream,
                        double* rmmc_per_layer, cd_result* out) {
  try {
    return group_step_impl(group, G, M, X, Q, mu, eta, r, stream, rmmc_per_layer, out);
  } catch (...) {
    return fail(CD_ENOMEM, "exception in cd_group_step");
  }
}

cd_status cd_group_destroy(cd_group* group) {
  if (!group) return CD_OK;
  DeviceGuard dg(group->device);
  free_group(group);
  return CD_OK;
}

cd_status cd_group_set_timing(cd_group* group, int enable) {
  if (!group) return fail(CD_EINVAL, "group is NULL");
  DeviceGuard dg(group->device);
  for (const auto& r : group->timer.recs) CD_HIP(hipEventSynchronize(r.b));
  group->timer.release();
  if (enable) CD_HIP(group->timer.reserve(2048));
  group->timer.on = enable != 0;
  return CD_OK;
}

cd_status cd_group_set_timing_kinds(cd_group* group, const char* kinds) {
  if (!group) return fail(CD_EINVAL, "group is NULL");
  if (!kinds || !*kinds) {
    group->timer.mask = ~0u;
    return CD_OK;
  }
  unsigned mask = 0;
  const std::string list(kinds);
  size_t b = 0;
  while (b <= list.size()) {
    size_t e = list.find(',', b);
    if (e == std::string::npos) e = list.size();
    const std::string name = list.substr(b, e - b);
    int k = 0;
    while (k < K_NKINDS && name != kKindName[k]) ++k;
    if (k == K_NKINDS) return fail(CD_EINVAL, "unknown kernel kind '%s'", name.c_str());
    mask |= 1u << k;
    b = e + 1;
  }
  group->timer.mask = mask;
  return CD_OK;
}

cd_status cd_group_kernel_times(cd_group* group, cd_kernel_time* out, int max_kinds, int* count) {
  if (!group || !count || (max_kinds > 0 && !out)) return fail(CD_EINVAL, "NULL argument");
  DeviceGuard dg(group->device);
  Timer& t = group->timer;
  cd_kernel_time agg[K_NKINDS];
  for (int k = 0; k < K_NKINDS; ++k) {
    std::memset(&agg[k], 0, sizeof(agg[k]));
    std::snprintf(agg[k].name, sizeof(agg[k].name), "%s", kKindName[k]);
  }
  for (const auto& r : t.recs) CD_HIP(hipEventSynchronize(r.b));   // each launch's stream
  for (const auto& r : t.recs) {
    float ms = 0.f;
    CD_HIP(hipEventElapsedTime(&ms, r.a, r.b));
    agg[r.kind].launches += 1;
    agg[r.kind].total_ms += ms;
    agg[r.kind].bytes += r.bytes;
    agg[r.kind].flops += r.flops;
  }
  t.release();
  int n = 0;
  for (int k = 0; k < K_NKINDS; ++k) {
    if (agg[k].launches == 0) continue;
    if (n < max_kinds) out[n] = agg[k];
    ++n;
  }
  *count = n;
  return CD_OK;
}

cd_status cd_layer_get_state(const cd_layer* layer, double* prev_norm, long long* step) {
  if (!layer || !prev_norm || !step) return fail(CD_EINVAL, "NULL argument");
  DeviceGuard dg(layer->device);
  CD_HIP(hipDeviceSynchronize());
  CD_HIP(hipMemcpy(prev_norm, layer->prev, sizeof(double), hipMemcpyDeviceToHost));
  *step = layer->step;
  return CD_OK;
}

cd_status cd_layer_set_state(cd_layer* layer, double prev_norm, long long step) {
  if (!layer) return fail(CD_EINVAL, "layer is NULL");
  if (step < 0) return fail(CD_EINVAL, "step must be >= 0");
  DeviceGuard dg(layer->device);
  CD_HIP(hipDeviceSynchronize());
  CD_HIP(hipMemcpy(layer->prev, &prev_norm, sizeof(double), hipMemcpyHostToDevice));
  layer->step = step;
  layer->prev_zero = prev_norm == 0.0;
  return CD_OK;
}

cd_status cd_layer_last_factors(const cd_layer* layer, const float** P, const float** R) {
  if (!layer || !P || !R) return fail(CD_EINVAL, "NULL argument");
  *P = layer->P;
  *R = layer->R;
  return CD_OK;
}

cd_status cd_layer_rank_deficient(const cd_layer* layer, int* flag) {
  if (!layer || !flag) return fail(CD_EINVAL, "NULL argument");
  const cd_group* g = layer->last_group;
  if (!g) {
    *flag = layer->rankdef_cached;
    return CD_OK;
  }
  DeviceGuard dg(g->device);
  // the last step of that group only (its completion event), not the device
  CD_HIP(hipEventSynchronize(g->done_ev));
  const int* rd = reinterpret_cast<const int*>(static_cast<const char*>(g->out_host) + host_rankdef_off(g->L));
  *flag = rd[layer->last_index];
  return CD_OK;
}

cd_status cd_group_last_result(cd_group* group, double* rmmc_per_layer, cd_result* out) {
  try {
    return group_last_result(group, rmmc_per_layer, out);
  } catch (...) {
    return fail(CD_ENOMEM, "exception in cd_group_last_result");
  }
}

cd_status cd_layer_last_result(cd_layer* layer, cd_result* out) {
  if (!layer) return fail(CD_EINVAL, "layer is NULL");
  try {
    return group_last_result(layer->self, nullptr, out);
  } catch (...) {
    return fail(CD_ENOMEM, "exception in cd_layer_last_result");
  }
}

const char* cd_last_error(void) { return g_err.c_str(); }

int cd_abi_version(void) { return CD_ABI_VERSION; }

}  // extern "C"
