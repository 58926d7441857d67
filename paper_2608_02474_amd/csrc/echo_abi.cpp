// C ABI of libecho: argument validation, workspace carving and the launch
// sequence of each call.  Every check runs before the first HIP call, so a
// rejected call touches neither the device nor the stream.
#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include <cmath>
#include <mutex>
#include <vector>

#include "../../include/echo.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

// ---- per-thread error and timing state
static thread_local int g_last_hip_error = 0;

struct TimingRecord {
  const char* name;
  hipEvent_t start, stop;
};
static thread_local bool g_profile = false;
static thread_local std::vector<TimingRecord> g_records;
static thread_local std::vector<hipEvent_t> g_event_pool;

bool profile_enabled() { return g_profile; }
void profile_set(bool on) { g_profile = on; }

static hipEvent_t take_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

TimedLaunch::TimedLaunch(const char* name, hipStream_t s) : slot(-1), stream(s) {
  if (!g_profile) return;
  TimingRecord r{name, take_event(), take_event()};
  if (r.start == nullptr || r.stop == nullptr || hipEventRecord(r.start, s) != hipSuccess) {
    if (r.start) g_event_pool.push_back(r.start);
    if (r.stop) g_event_pool.push_back(r.stop);
    return;
  }
  g_records.push_back(r);
  slot = static_cast<int>(g_records.size()) - 1;
}
TimedLaunch::~TimedLaunch() {
  if (slot >= 0) (void)hipEventRecord(g_records[slot].stop, stream);
}

int device_cu_count() {
  static const int n = [] {
    int dev = 0, cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cu <= 0)
      cu = 256;
    return cu;
  }();
  return n;
}

size_t gemm_partial_bytes() { return sizeof(float) * 256 * 256 * 256; }

}  // namespace echo

using namespace echo;

namespace {

constexpr size_t kAlign = 256;
constexpr size_t align_up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline bool ok_ptr(const void* p) { return p != nullptr && aligned16(p); }
inline size_t esize(int dtype) { return dtype == ECHO_BF16 ? 2 : 4; }
inline bool ok_dtype(int dtype) { return dtype == ECHO_F32 || dtype == ECHO_BF16; }

int device_status(hipError_t e) {
  if (e == hipSuccess) return ECHO_OK;
  g_last_hip_error = static_cast<int>(e);
  return ECHO_EDEVICE;
}

// ---- energy
bool energy_cfg_ok(const echo_energy_cfg* c, int64_t n_samples) {
  return c != nullptr && c->T >= 1 && c->T <= 65535 && n_samples >= c->T && c->n_fft >= 16 &&
         c->n_fft <= 2048 && (c->n_fft % 2) == 0 && c->hop >= 1 && c->n_bands >= 1 &&
         c->n_bands <= 64 && c->sample_rate > 0;
}
size_t energy_ws(const echo_energy_cfg* c, int64_t n_samples) {
  const int mf = energy_max_frames(n_samples, c->T, c->n_fft, c->hop);
  // per-frame band energies, then per-segment energies and band sums
  return align_up(sizeof(double) * static_cast<size_t>(c->T) * mf * c->n_bands) +
         align_up(sizeof(double) * static_cast<size_t>(c->T) * (1 + c->n_bands));
}

// ---- select
bool select_cfg_ok(const echo_select_cfg* c) {
  if (c == nullptr || c->T < 1 || c->N < 1 || c->D < 8 || (c->D % 8) != 0 || !ok_dtype(c->dtype))
    return false;
  const int64_t L = static_cast<int64_t>(c->T) * c->N;
  if (L >= (int64_t(1) << 31)) return false;
  if (c->k > L) return false;
  if (!(c->xi >= 0.0) || isnan(c->threshold)) return false;
  return true;
}
size_t select_ws(const echo_select_cfg* c) {
  const size_t L = static_cast<size_t>(c->T) * c->N;
  return align_up(L * sizeof(float)) + 2 * align_up(L * sizeof(double));
}

int select_args_status(const echo_select_cfg* cfg, const void* x, const void* xref, const float* frame_weight,
                       const int32_t* idx, const uint8_t* mask, const int32_t* n_sel, const float* saliency,
                       const double* step_delta) {
  if (!select_cfg_ok(cfg)) return ECHO_EINVAL;
  if (!ok_ptr(x) || !ok_ptr(xref) || !ok_ptr(frame_weight) || !ok_ptr(idx) || !ok_ptr(mask) ||
      n_sel == nullptr)
    return ECHO_EINVAL;
  if ((saliency != nullptr && !aligned16(saliency)) ||
      (step_delta != nullptr && (reinterpret_cast<uintptr_t>(step_delta) & 7u)))
    return ECHO_EINVAL;
  return ECHO_OK;
}
int select_launch(const echo_select_cfg* cfg, const void* x, const void* xref, const float* frame_weight,
                  int32_t* idx, uint8_t* mask, int32_t* n_sel, float* saliency, double* step_delta,
                  void* workspace, void* stream);

// ---- allocation-free selection: the workspace of echo_select for up to
// ECHO_SELECT_NOALLOC_MAX_TOKENS tokens as a static device array.  Each GPU
// holds its own copy; its address is looked up once per device (with that
// device current) and kept, and only that address is handed to kernels: in
// host code the array's name is not a device address.
constexpr size_t kNoAllocScratchBytes =
    align_up(ECHO_SELECT_NOALLOC_MAX_TOKENS * sizeof(float)) + 2 * align_up(ECHO_SELECT_NOALLOC_MAX_TOKENS * sizeof(double));
__device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (ECHO_EDEVICE if the
// lookup fails).
int noalloc_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return device_status(e);
  if (dev < 0 || dev >= kMaxDevices) return ECHO_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return device_status(e);
    if (p == nullptr) return ECHO_EDEVICE;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ECHO_OK;
}

// ---- block
bool block_cfg_ok(const echo_block_cfg* c) {
  return c != nullptr && c->L >= 1 && c->D >= 8 && c->H >= 1 && c->F >= 8 && ok_dtype(c->dtype) &&
         c->D <= 16384 && c->F <= 65536 && (c->D % c->H) == 0 && (c->D % 8) == 0 &&
         (c->F % 8) == 0 && c->ln_eps >= 0.0f && (c->flags & ~ECHO_BLOCK_BATCH_INVARIANT) == 0;
}
bool block_supported(const echo_block_cfg* c) {
  const int dh = c->D / c->H;
  // bf16 GEMM tiles address their operands through 32-bit byte offsets
  if (c->dtype == ECHO_BF16)
    return dh == 128 && (c->D % 256) == 0 && (c->F % 256) == 0 &&
           int64_t(c->L) * c->D < (int64_t(1) << 30) && int64_t(c->F) * c->D < (int64_t(1) << 30);
  return dh <= 128;
}
struct BlockWs {
  void *a, *kv, *q, *o, *b, *h;
  float* x1;
  float* part;        // bf16 path: partial results of the GEMM and attention tails
  size_t part_bytes;  // its size: the larger of the two needs
  size_t bytes;
};
size_t max_size(size_t a, size_t b) { return a > b ? a : b; }
BlockWs block_ws_layout(const echo_block_cfg* c, int64_t n, char* base) {
  const size_t es = esize(c->dtype);
  const size_t L = c->L, D = c->D, F = c->F, m = static_cast<size_t>(n);
  BlockWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off += align_up(bytes);
    return p;
  };
  w.a = take(L * D * es);
  w.kv = take(L * 2 * D * es);
  w.q = take(m * D * es);
  w.o = take(m * D * es);
  w.x1 = reinterpret_cast<float*>(take(m * D * 4));
  w.b = take(m * D * es);
  w.h = take(m * F * es);
  if (c->dtype == ECHO_BF16) {
    w.part_bytes = max_size(gemm_partial_bytes(), attn_partial_bytes(static_cast<int>(n), c->L, c->H));
    w.part = reinterpret_cast<float*>(take(w.part_bytes));
  }
  w.bytes = off;
  return w;
}
bool weights_ok(const echo_block_weights* w) {
  return w != nullptr && ok_ptr(w->wq) && ok_ptr(w->wk) && ok_ptr(w->wv) && ok_ptr(w->wo) &&
         ok_ptr(w->w1) && ok_ptr(w->w2) && ok_ptr(w->bq) && ok_ptr(w->bk) && ok_ptr(w->bv) &&
         ok_ptr(w->bo) && ok_ptr(w->b1) && ok_ptr(w->b2) && ok_ptr(w->mod);
}

}  // namespace

namespace {
bool refcache_cfg_ok(const echo_refcache_cfg* c) {
  return c != nullptr && c->L >= 1 && c->D >= 8 && (c->D % 8) == 0 && c->D <= 16384 && ok_dtype(c->dtype) &&
         c->chain_len >= 1 && (c->L % c->chain_len) == 0 && std::isfinite(c->tau) &&
         static_cast<int64_t>(c->capacity) >= static_cast<int64_t>(c->L) + c->L / c->chain_len;
}
bool refcache_state_ok(const echo_refcache_state* s) {
  return s != nullptr && ok_ptr(s->pool) && ok_ptr(s->refcount) && ok_ptr(s->free_list) && ok_ptr(s->free_top) &&
         ok_ptr(s->chain_ref) && ok_ptr(s->ent_slot) && ok_ptr(s->ent_kind) && ok_ptr(s->codes) &&
         ok_ptr(s->scale);
}
}  // namespace

namespace {
bool wan_cfg_ok(const echo_wan_block_cfg* c) {
  return c != nullptr && c->B >= 1 && c->L >= 1 && c->D >= 8 && c->H >= 1 && c->F >= 8 && c->Lc >= 1 &&
         c->T >= 1 && c->gh >= 1 && c->gw >= 1 && int64_t(c->T) * c->gh * c->gw == c->L &&
         ok_dtype(c->dtype) && c->D <= 16384 && c->F <= 65536 && (c->D % c->H) == 0 && (c->D % 8) == 0 &&
         (c->F % 8) == 0 && c->ln_eps >= 0.0f && c->rms_eps >= 0.0f && std::isfinite(c->rope_base) &&
         c->rope_base > 0.0 && (c->flags & ~ECHO_BLOCK_BATCH_INVARIANT) == 0;
}
bool wan_supported(const echo_wan_block_cfg* c) {
  const int64_t lim = int64_t(1) << 30;
  return c->dtype == ECHO_BF16 && c->D / c->H == 128 && (c->D % 256) == 0 && (c->F % 256) == 0 &&
         int64_t(c->B) * c->L * c->D < lim && int64_t(c->B) * c->Lc * c->D < lim && int64_t(c->F) * c->D < lim;
}
struct WanWs {
  void *a, *kv, *kvc, *q, *o, *b, *h;
  float *x1, *x2, *part, *ones, *g3m1;
  float2* tab;
  size_t part_bytes;
  size_t bytes;
};
WanWs wan_ws_layout(const echo_wan_block_cfg* c, int64_t n, char* base) {
  const size_t es = esize(c->dtype);
  const size_t BL = size_t(c->B) * c->L, BLc = size_t(c->B) * c->Lc, D = c->D, F = c->F, m = size_t(n);
  WanWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off += align_up(bytes);
    return p;
  };
  w.a = take(BL * D * es);
  w.kv = take(BL * 2 * D * es);
  w.kvc = take(BLc * 2 * D * es);
  w.q = take(m * D * es);
  w.o = take(m * D * es);
  w.b = take(m * D * es);
  w.h = take(m * F * es);
  w.x1 = reinterpret_cast<float*>(take(m * D * 4));
  w.x2 = reinterpret_cast<float*>(take(m * D * 4));
  // the attention runs per batch element, with at most n selected rows
  w.part_bytes = max_size(gemm_partial_bytes(),
                          max_size(attn_partial_bytes(static_cast<int>(n), c->L, c->H),
                                   attn_partial_bytes(static_cast<int>(n), c->Lc, c->H)));
  w.part = reinterpret_cast<float*>(take(w.part_bytes));
  w.ones = reinterpret_cast<float*>(take(D * 4));
  w.g3m1 = reinterpret_cast<float*>(take(D * 4));
  w.tab = reinterpret_cast<float2*>(take(sizeof(float2) * size_t(rope_table_entries(c->T, c->gh, c->gw,
                                                                                     c->D / c->H))));
  w.bytes = off;
  return w;
}
bool wan_weights_ok(const echo_wan_block_weights* w) {
  return w != nullptr && weights_ok(&w->self) && ok_ptr(w->wqc) && ok_ptr(w->wkc) && ok_ptr(w->wvc) &&
         ok_ptr(w->woc) && ok_ptr(w->bqc) && ok_ptr(w->bkc) && ok_ptr(w->bvc) && ok_ptr(w->boc) &&
         ok_ptr(w->gq) && ok_ptr(w->gk) && ok_ptr(w->gqc) && ok_ptr(w->gkc) && ok_ptr(w->g3) && ok_ptr(w->b3);
}
}  // namespace

extern "C" {

const char* echo_status_str(int status) {
  switch (status) {
    case ECHO_OK: return "ok";
    case ECHO_EINVAL: return "invalid argument";
    case ECHO_EUNSUPPORTED: return "unsupported shape or dtype";
    case ECHO_EWORKSPACE: return "workspace missing or too small";
    case ECHO_EDEVICE: return "HIP device error";
    case ECHO_ELIMIT: return "size above the allocation-free limit";
    default: return "unknown status";
  }
}

int echo_last_hip_error(void) { return g_last_hip_error; }

const char* echo_version(void) { return "0.1.0"; }

size_t echo_energy_workspace(const echo_energy_cfg* cfg, int64_t n_samples) {
  if (!energy_cfg_ok(cfg, n_samples)) return 0;
  return energy_ws(cfg, n_samples);
}

int echo_energy(const echo_energy_cfg* cfg, const float* audio, int64_t n_samples, float* band_energy,
                float* frame_energy, float* frame_weight, void* workspace, size_t workspace_bytes,
                void* stream) {
  if (!energy_cfg_ok(cfg, n_samples)) return ECHO_EINVAL;
  if (!ok_ptr(audio) || !ok_ptr(band_energy) || !ok_ptr(frame_energy) || !ok_ptr(frame_weight))
    return ECHO_EINVAL;
  const size_t need = energy_ws(cfg, n_samples);
  if (!ok_ptr(workspace) || workspace_bytes < need) return ECHO_EWORKSPACE;
  const int mf = energy_max_frames(n_samples, cfg->T, cfg->n_fft, cfg->hop);
  double* part = static_cast<double*>(workspace);
  double* e_scr = reinterpret_cast<double*>(
      static_cast<char*>(workspace) +
      align_up(sizeof(double) * static_cast<size_t>(cfg->T) * mf * cfg->n_bands));
  return device_status(launch_energy(audio, n_samples, cfg->T, cfg->sample_rate, cfg->n_fft, cfg->hop,
                                     cfg->n_bands, band_energy, frame_energy, frame_weight, part,
                                     e_scr, static_cast<hipStream_t>(stream)));
}

size_t echo_select_workspace(const echo_select_cfg* cfg) {
  if (!select_cfg_ok(cfg)) return 0;
  return select_ws(cfg);
}

int echo_select(const echo_select_cfg* cfg, const void* x, const void* xref, const float* frame_weight,
                int32_t* idx, uint8_t* mask, int32_t* n_sel, float* saliency, double* step_delta,
                void* workspace, size_t workspace_bytes, void* stream) {
  const int bad = select_args_status(cfg, x, xref, frame_weight, idx, mask, n_sel, saliency, step_delta);
  if (bad != ECHO_OK) return bad;
  const size_t need = select_ws(cfg);
  if (!ok_ptr(workspace) || workspace_bytes < need) return ECHO_EWORKSPACE;
  return select_launch(cfg, x, xref, frame_weight, idx, mask, n_sel, saliency, step_delta, workspace, stream);
}

int echo_select_noalloc(const echo_select_cfg* cfg, const void* x, const void* xref, const float* frame_weight,
                        int32_t* idx, uint8_t* mask, int32_t* n_sel, float* saliency, double* step_delta,
                        void* stream) {
  const int bad = select_args_status(cfg, x, xref, frame_weight, idx, mask, n_sel, saliency, step_delta);
  if (bad != ECHO_OK) return bad;
  if (static_cast<int64_t>(cfg->T) * cfg->N > ECHO_SELECT_NOALLOC_MAX_TOKENS) return ECHO_ELIMIT;
  void* ws = nullptr;
  const int st = noalloc_scratch(&ws);
  if (st != ECHO_OK) return st;
  return select_launch(cfg, x, xref, frame_weight, idx, mask, n_sel, saliency, step_delta, ws, stream);
}

}  // extern "C"

namespace {
int select_launch(const echo_select_cfg* cfg, const void* x, const void* xref, const float* frame_weight,
                  int32_t* idx, uint8_t* mask, int32_t* n_sel, float* saliency, double* step_delta,
                  void* workspace, void* stream) {
  const int L = cfg->T * cfg->N;
  char* ws = static_cast<char*>(workspace);
  float* s_ws = reinterpret_cast<float*>(ws);
  double* num = reinterpret_cast<double*>(ws + align_up(L * sizeof(float)));
  double* den = reinterpret_cast<double*>(ws + align_up(L * sizeof(float)) + align_up(L * sizeof(double)));
  float* s = saliency ? saliency : s_ws;
  const int threshold_mode = cfg->k < 0 ? 1 : 0;
  return device_status(launch_select(cfg->dtype == ECHO_BF16, x, xref, frame_weight, L, cfg->N, cfg->D,
                                     cfg->xi, threshold_mode ? 0 : cfg->k, threshold_mode,
                                     cfg->threshold, s, num, den, idx, mask, n_sel, step_delta,
                                     static_cast<hipStream_t>(stream)));
}
}  // namespace

extern "C" {

size_t echo_saliency_workspace(const echo_select_cfg* cfg) {
  if (!select_cfg_ok(cfg)) return 0;
  const size_t L = static_cast<size_t>(cfg->T) * cfg->N;
  return 2 * align_up(L * sizeof(double));
}

int echo_saliency(const echo_select_cfg* cfg, const void* x, const void* xref, const float* frame_weight,
                  float* saliency, double* step_delta, void* workspace, size_t workspace_bytes, void* stream) {
  if (!select_cfg_ok(cfg)) return ECHO_EINVAL;
  if (!ok_ptr(x) || !ok_ptr(xref) || !ok_ptr(frame_weight) || !ok_ptr(saliency)) return ECHO_EINVAL;
  if (step_delta != nullptr && (reinterpret_cast<uintptr_t>(step_delta) & 7u)) return ECHO_EINVAL;
  const size_t need = echo_saliency_workspace(cfg);
  if (!ok_ptr(workspace) || workspace_bytes < need) return ECHO_EWORKSPACE;
  const int L = cfg->T * cfg->N;
  double* num = static_cast<double*>(workspace);
  double* den = reinterpret_cast<double*>(static_cast<char*>(workspace) + align_up(L * sizeof(double)));
  return device_status(launch_saliency(cfg->dtype == ECHO_BF16, x, xref, frame_weight, L, cfg->N, cfg->D,
                                       cfg->xi, saliency, num, den, step_delta,
                                       static_cast<hipStream_t>(stream)));
}

int echo_topk(const echo_select_cfg* cfg, const float* saliency, int32_t* idx, uint8_t* mask, int32_t* n_sel,
              void* stream) {
  if (!select_cfg_ok(cfg)) return ECHO_EINVAL;
  if (!ok_ptr(saliency) || !ok_ptr(idx) || !ok_ptr(mask) || n_sel == nullptr) return ECHO_EINVAL;
  const int L = cfg->T * cfg->N;
  const int threshold_mode = cfg->k < 0 ? 1 : 0;
  return device_status(launch_topk(saliency, L, threshold_mode ? 0 : cfg->k, threshold_mode, cfg->threshold,
                                   idx, mask, n_sel, static_cast<hipStream_t>(stream)));
}

int echo_anchors(const float* keys, int32_t T, int32_t k, int32_t mode, uint8_t* anchors, void* stream) {
  if (T < 1 || T > max_anchor_segments() || k < 0 || k > T) return ECHO_EINVAL;
  if (mode != ECHO_ANCHOR_TOPK && mode != ECHO_ANCHOR_UNIFORM) return ECHO_EINVAL;
  if (anchors == nullptr || (mode == ECHO_ANCHOR_TOPK && !ok_ptr(keys))) return ECHO_EINVAL;
  return device_status(launch_anchors(keys, T, k, mode, anchors, static_cast<hipStream_t>(stream)));
}

int echo_topk_segments(const float* saliency, const uint8_t* anchors, int32_t T, int32_t N, int32_t k,
                       int32_t* idx, uint8_t* mask, int32_t* n_sel, void* stream) {
  if (T < 1 || T > 65535 || N < 1 || k < 0) return ECHO_EINVAL;
  if (static_cast<int64_t>(T) * N >= (int64_t(1) << 31)) return ECHO_EINVAL;
  if (!ok_ptr(saliency) || anchors == nullptr || !ok_ptr(idx) || !ok_ptr(mask) || n_sel == nullptr)
    return ECHO_EINVAL;
  return device_status(
      launch_topk_segments(saliency, anchors, T, N, k, idx, mask, n_sel, static_cast<hipStream_t>(stream)));
}

int32_t echo_topk_count(double ratio, int32_t L) {
  if (L < 1 || !(ratio >= 0.0 && ratio <= 1.0)) return -ECHO_EINVAL;
  const double kk = std::ceil(ratio * L - 1e-9);
  return kk < 0.0 ? 0 : (kk > L ? L : static_cast<int32_t>(kk));
}

int32_t echo_segments_count(int32_t n_anchors, int32_t N, int32_t k) {
  if (n_anchors < 0 || N < 1 || k < 0) return -ECHO_EINVAL;
  const int64_t n = static_cast<int64_t>(n_anchors) * (k < N ? k : N);
  return n >= (int64_t(1) << 31) ? -ECHO_EINVAL : static_cast<int32_t>(n);
}

int32_t echo_schedule_next(const echo_schedule_cfg* cfg, echo_schedule_state* st, double delta_t, int32_t L,
                           int32_t* full) {
  if (cfg == nullptr || st == nullptr || full == nullptr || L < 1 || cfg->n_full < 0 ||
      !(cfg->r_min >= 0.0) || !(cfg->r_max <= 1.0) || !(cfg->r_min <= cfg->r_max) || !std::isfinite(cfg->alpha) ||
      std::isnan(cfg->refresh_delta) || std::isnan(delta_t))
    return -ECHO_EINVAL;
  const int32_t step = st->step++;
  if (step < cfg->n_full) {
    st->delta_acc = 0.0;
    *full = 1;
    return L;
  }
  st->delta_acc += delta_t;
  if (cfg->refresh_delta > 0.0 && st->delta_acc > cfg->refresh_delta) {
    st->delta_acc = 0.0;
    *full = 1;
    return L;
  }
  st->delta_max = delta_t > st->delta_max ? delta_t : st->delta_max;
  const double dhat = st->delta_max > 0.0 ? delta_t / st->delta_max : 0.0;
  double r = cfg->r_min + cfg->alpha * dhat;
  r = r < cfg->r_min ? cfg->r_min : (r > cfg->r_max ? cfg->r_max : r);
  *full = 0;
  return echo_topk_count(r, L);
}

size_t echo_block_workspace(const echo_block_cfg* cfg, int32_t n_sel_max) {
  if (!block_cfg_ok(cfg) || n_sel_max < 0) return 0;
  return block_ws_layout(cfg, n_sel_max, nullptr).bytes;
}

int echo_block_partial(const echo_block_cfg* cfg, const echo_block_weights* w, const void* x,
                       const int32_t* idx, int32_t n_sel, float* y_sel, void* workspace,
                       size_t workspace_bytes, void* stream) {
  if (!block_cfg_ok(cfg) || !weights_ok(w) || n_sel < 0) return ECHO_EINVAL;
  if (!block_supported(cfg)) return ECHO_EUNSUPPORTED;
  if (n_sel == 0) return ECHO_OK;
  if (cfg->dtype == ECHO_BF16 && int64_t(n_sel) * cfg->F >= (int64_t(1) << 30)) return ECHO_EUNSUPPORTED;
  if (!ok_ptr(x) || !ok_ptr(idx) || !ok_ptr(y_sel)) return ECHO_EINVAL;
  const size_t need = block_ws_layout(cfg, n_sel, nullptr).bytes;
  if (!ok_ptr(workspace) || workspace_bytes < need) return ECHO_EWORKSPACE;
  const BlockWs ws = block_ws_layout(cfg, n_sel, static_cast<char*>(workspace));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int L = cfg->L, D = cfg->D, H = cfg->H, F = cfg->F, n = n_sel;
  const float* mod = w->mod;
  const bool bf = cfg->dtype == ECHO_BF16;
  hipError_t e = launch_modln_input(bf, x, L, D, mod + 0 * D, mod + 1 * D, cfg->ln_eps, ws.a, st);
  if (e != hipSuccess) return device_status(e);
  if (bf) {
    typedef const bf16_t* P;
    GemmBf16Args g{};
    // partial results of the split tails (none when every row must be batch-invariant)
    float* part = (cfg->flags & ECHO_BLOCK_BATCH_INVARIANT) ? nullptr : ws.part;
    auto with_part = [&](GemmBf16Args a) {
      a.part = part;
      a.part_bytes = ws.part_bytes;
      return a;
    };
    // q = a[idx] Wq^T + bq
    g = GemmBf16Args{static_cast<P>(ws.a), D, idx, L, static_cast<P>(w->wq), static_cast<P>(w->wq), D, D,
                     static_cast<P>(w->bq), static_cast<P>(w->bq), n, D, D, ws.q, D,
                     nullptr, nullptr, 0, nullptr, 0};
    if ((e = launch_gemm_bf16("gemm_q_bf16", 0, with_part(g), st)) != hipSuccess) return device_status(e);
    // [k | v] = a [Wk; Wv]^T + [bk; bv], one N = 2D GEMM over all L rows
    g = GemmBf16Args{static_cast<P>(ws.a), D, nullptr, L, static_cast<P>(w->wk), static_cast<P>(w->wv), D,
                     D, static_cast<P>(w->bk), static_cast<P>(w->bv), L, 2 * D, D, ws.kv, 2 * D,
                     nullptr, nullptr, 0, nullptr, 0};
    if ((e = launch_gemm_bf16("gemm_kv_bf16", 0, with_part(g), st)) != hipSuccess) return device_status(e);
    const bf16_t* kvp = static_cast<const bf16_t*>(ws.kv);
    if ((e = launch_attn_bf16(static_cast<P>(ws.q), D, kvp, kvp + D, 2 * D, n, L, H,
                              static_cast<bf16_t*>(ws.o), D,
                              part, ws.part_bytes, st)) !=
        hipSuccess)
      return device_status(e);
    // x1 = x[idx] + gate1 * (o Wo^T + bo)
    g = GemmBf16Args{static_cast<P>(ws.o), D, nullptr, n, static_cast<P>(w->wo), static_cast<P>(w->wo), D,
                     D, static_cast<P>(w->bo), static_cast<P>(w->bo), n, D, D, ws.x1, D,
                     mod + 2 * D, x, D, idx, 1};
    if ((e = launch_gemm_bf16("gemm_o_bf16", 2, with_part(g), st)) != hipSuccess) return device_status(e);
    if ((e = launch_modln_x1(1, ws.x1, n, D, mod + 3 * D, mod + 4 * D, cfg->ln_eps, ws.b, st)) !=
        hipSuccess)
      return device_status(e);
    // h = GELU(b W1^T + b1)
    g = GemmBf16Args{static_cast<P>(ws.b), D, nullptr, n, static_cast<P>(w->w1), static_cast<P>(w->w1), F,
                     D, static_cast<P>(w->b1), static_cast<P>(w->b1), n, F, D, ws.h, F,
                     nullptr, nullptr, 0, nullptr, 0};
    if ((e = launch_gemm_bf16("gemm_ffn_up_bf16", 1, with_part(g), st)) != hipSuccess) return device_status(e);
    // y_sel = x1 + gate2 * (h W2^T + b2)
    g = GemmBf16Args{static_cast<P>(ws.h), F, nullptr, n, static_cast<P>(w->w2), static_cast<P>(w->w2), D,
                     F, static_cast<P>(w->b2), static_cast<P>(w->b2), n, D, F, y_sel, D,
                     mod + 5 * D, ws.x1, D, nullptr, 0};
    if ((e = launch_gemm_bf16("gemm_ffn_down_bf16", 2, with_part(g), st)) != hipSuccess) return device_status(e);
    return ECHO_OK;
  }
  typedef const float* P;
  const int dh = D / H;
  GemmF32Args g{};
  g = GemmF32Args{static_cast<P>(ws.a), D, idx, static_cast<P>(w->wq), static_cast<P>(w->wq), D, D,
                  static_cast<P>(w->bq), static_cast<P>(w->bq), n, D, D, static_cast<float*>(ws.q), D,
                  nullptr, nullptr, 0, nullptr};
  if ((e = launch_gemm_f32("gemm_q_f32", 0, g, st)) != hipSuccess) return device_status(e);
  g = GemmF32Args{static_cast<P>(ws.a), D, nullptr, static_cast<P>(w->wk), static_cast<P>(w->wv), D, D,
                  static_cast<P>(w->bk), static_cast<P>(w->bv), L, 2 * D, D,
                  static_cast<float*>(ws.kv), 2 * D, nullptr, nullptr, 0, nullptr};
  if ((e = launch_gemm_f32("gemm_kv_f32", 0, g, st)) != hipSuccess) return device_status(e);
  const float* kvp = static_cast<const float*>(ws.kv);
  if ((e = launch_attn_f32(static_cast<P>(ws.q), D, kvp, kvp + D, 2 * D, n, L, H, dh,
                           static_cast<float*>(ws.o), D, st)) != hipSuccess)
    return device_status(e);
  g = GemmF32Args{static_cast<P>(ws.o), D, nullptr, static_cast<P>(w->wo), static_cast<P>(w->wo), D, D,
                  static_cast<P>(w->bo), static_cast<P>(w->bo), n, D, D, ws.x1, D, mod + 2 * D,
                  static_cast<P>(x), D, idx};
  if ((e = launch_gemm_f32("gemm_o_f32", 2, g, st)) != hipSuccess) return device_status(e);
  if ((e = launch_modln_x1(0, ws.x1, n, D, mod + 3 * D, mod + 4 * D, cfg->ln_eps, ws.b, st)) !=
      hipSuccess)
    return device_status(e);
  g = GemmF32Args{static_cast<P>(ws.b), D, nullptr, static_cast<P>(w->w1), static_cast<P>(w->w1), F, D,
                  static_cast<P>(w->b1), static_cast<P>(w->b1), n, F, D, static_cast<float*>(ws.h), F,
                  nullptr, nullptr, 0, nullptr};
  if ((e = launch_gemm_f32("gemm_ffn_up_f32", 1, g, st)) != hipSuccess) return device_status(e);
  g = GemmF32Args{static_cast<P>(ws.h), F, nullptr, static_cast<P>(w->w2), static_cast<P>(w->w2), D, F,
                  static_cast<P>(w->b2), static_cast<P>(w->b2), n, D, F, y_sel, D, mod + 5 * D, ws.x1,
                  D, nullptr};
  if ((e = launch_gemm_f32("gemm_ffn_down_f32", 2, g, st)) != hipSuccess) return device_status(e);
  return ECHO_OK;
}


size_t echo_wan_block_workspace(const echo_wan_block_cfg* cfg, int32_t n_total_max) {
  if (!wan_cfg_ok(cfg) || n_total_max < 0) return 0;
  return wan_ws_layout(cfg, n_total_max, nullptr).bytes;
}

int echo_wan_block_partial(const echo_wan_block_cfg* cfg, const echo_wan_block_weights* w, const void* x,
                           const void* ctx, const int32_t* idx, const int32_t* n_sel, float* y_sel,
                           void* workspace, size_t workspace_bytes, void* stream) {
  if (!wan_cfg_ok(cfg) || !wan_weights_ok(w) || n_sel == nullptr) return ECHO_EINVAL;
  int64_t tot = 0;
  for (int b = 0; b < cfg->B; ++b) {
    if (n_sel[b] < 0 || n_sel[b] > cfg->L) return ECHO_EINVAL;
    tot += n_sel[b];
  }
  if (!wan_supported(cfg)) return ECHO_EUNSUPPORTED;
  if (tot == 0) return ECHO_OK;
  if (tot * cfg->F >= (int64_t(1) << 30)) return ECHO_EUNSUPPORTED;
  if (!ok_ptr(x) || !ok_ptr(ctx) || !ok_ptr(idx) || !ok_ptr(y_sel)) return ECHO_EINVAL;
  const size_t need = wan_ws_layout(cfg, tot, nullptr).bytes;
  if (!ok_ptr(workspace) || workspace_bytes < need) return ECHO_EWORKSPACE;
  const WanWs ws = wan_ws_layout(cfg, tot, static_cast<char*>(workspace));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int B = cfg->B, L = cfg->L, D = cfg->D, H = cfg->H, F = cfg->F, Lc = cfg->Lc, n = static_cast<int>(tot);
  const int BL = B * L, BLc = B * Lc, dh = D / H;
  const float* mod = w->self.mod;
  typedef const bf16_t* P;
  float* part = (cfg->flags & ECHO_BLOCK_BATCH_INVARIANT) ? nullptr : ws.part;
  auto with_part = [&](GemmBf16Args a) {
    a.part = part;
    a.part_bytes = ws.part_bytes;
    return a;
  };
  hipError_t e;
#define ECHO_TRY(call)                              \
  if ((e = (call)) != hipSuccess) return device_status(e);
  // constants: rotary table, the unit gate of the cross-attention output, g3 - 1
  ECHO_TRY(launch_rope_table(cfg->T, cfg->gh, cfg->gw, dh, cfg->rope_base, ws.tab, st));
  ECHO_TRY(launch_vec_shift(nullptr, 1.0f, ws.ones, D, st));
  ECHO_TRY(launch_vec_shift(w->g3, -1.0f, ws.g3m1, D, st));
  // self-attention
  ECHO_TRY(launch_modln_input(1, x, BL, D, mod + 0 * D, mod + 1 * D, cfg->ln_eps, ws.a, st));
  GemmBf16Args g{};
  g = GemmBf16Args{static_cast<P>(ws.a), D, idx, BL, static_cast<P>(w->self.wq), static_cast<P>(w->self.wq), D, D,
                   static_cast<P>(w->self.bq), static_cast<P>(w->self.bq), n, D, D, ws.q, D,
                   nullptr, nullptr, 0, nullptr, 0};
  ECHO_TRY(launch_gemm_bf16("gemm_q_bf16", 0, with_part(g), st));
  g = GemmBf16Args{static_cast<P>(ws.a), D, nullptr, BL, static_cast<P>(w->self.wk), static_cast<P>(w->self.wv), D,
                   D, static_cast<P>(w->self.bk), static_cast<P>(w->self.bv), BL, 2 * D, D, ws.kv, 2 * D,
                   nullptr, nullptr, 0, nullptr, 0};
  ECHO_TRY(launch_gemm_bf16("gemm_kv_bf16", 0, with_part(g), st));
  ECHO_TRY(launch_qk_norm_rope(static_cast<bf16_t*>(ws.q), D, n, D, w->gq, cfg->rms_eps, idx, ws.tab, L, cfg->T,
                               cfg->gh, cfg->gw, dh, st));
  ECHO_TRY(launch_qk_norm_rope(static_cast<bf16_t*>(ws.kv), 2 * D, BL, D, w->gk, cfg->rms_eps, nullptr, ws.tab, L,
                               cfg->T, cfg->gh, cfg->gw, dh, st));
  {
    const bf16_t* kvp = static_cast<const bf16_t*>(ws.kv);
    int64_t o = 0;
    for (int b = 0; b < B; ++b) {
      const bf16_t* kb = kvp + int64_t(b) * L * 2 * D;
      ECHO_TRY(launch_attn_bf16(static_cast<P>(ws.q) + o * D, D, kb, kb + D, 2 * D, n_sel[b], L, H,
                                static_cast<bf16_t*>(ws.o) + o * D, D, part, ws.part_bytes, st));
      o += n_sel[b];
    }
  }
  g = GemmBf16Args{static_cast<P>(ws.o), D, nullptr, n, static_cast<P>(w->self.wo), static_cast<P>(w->self.wo), D,
                   D, static_cast<P>(w->self.bo), static_cast<P>(w->self.bo), n, D, D, ws.x1, D,
                   mod + 2 * D, x, D, idx, 1};
  ECHO_TRY(launch_gemm_bf16("gemm_o_bf16", 2, with_part(g), st));
  // cross-attention: c = LN(x1) * g3 + b3 = LN(x1) * (1 + (g3 - 1)) + b3
  ECHO_TRY(launch_modln_x1(1, ws.x1, n, D, w->b3, ws.g3m1, cfg->ln_eps, ws.b, st));
  g = GemmBf16Args{static_cast<P>(ws.b), D, nullptr, n, static_cast<P>(w->wqc), static_cast<P>(w->wqc), D, D,
                   static_cast<P>(w->bqc), static_cast<P>(w->bqc), n, D, D, ws.q, D,
                   nullptr, nullptr, 0, nullptr, 0};
  ECHO_TRY(launch_gemm_bf16("gemm_qc_bf16", 0, with_part(g), st));
  g = GemmBf16Args{static_cast<P>(ctx), D, nullptr, BLc, static_cast<P>(w->wkc), static_cast<P>(w->wvc), D, D,
                   static_cast<P>(w->bkc), static_cast<P>(w->bvc), BLc, 2 * D, D, ws.kvc, 2 * D,
                   nullptr, nullptr, 0, nullptr, 0};
  ECHO_TRY(launch_gemm_bf16("gemm_kvc_bf16", 0, with_part(g), st));
  ECHO_TRY(launch_qk_norm_rope(static_cast<bf16_t*>(ws.q), D, n, D, w->gqc, cfg->rms_eps, nullptr, nullptr, L,
                               cfg->T, cfg->gh, cfg->gw, dh, st));
  ECHO_TRY(launch_qk_norm_rope(static_cast<bf16_t*>(ws.kvc), 2 * D, BLc, D, w->gkc, cfg->rms_eps, nullptr, nullptr,
                               L, cfg->T, cfg->gh, cfg->gw, dh, st));
  {
    const bf16_t* kvp = static_cast<const bf16_t*>(ws.kvc);
    int64_t o = 0;
    for (int b = 0; b < B; ++b) {
      const bf16_t* kb = kvp + int64_t(b) * Lc * 2 * D;
      ECHO_TRY(launch_attn_bf16(static_cast<P>(ws.q) + o * D, D, kb, kb + D, 2 * D, n_sel[b], Lc, H,
                                static_cast<bf16_t*>(ws.o) + o * D, D, part, ws.part_bytes, st,
                                "attn_cross_bf16"));
      o += n_sel[b];
    }
  }
  // x2 = x1 + 1 * (oc Woc^T + boc)
  g = GemmBf16Args{static_cast<P>(ws.o), D, nullptr, n, static_cast<P>(w->woc), static_cast<P>(w->woc), D, D,
                   static_cast<P>(w->boc), static_cast<P>(w->boc), n, D, D, ws.x2, D,
                   ws.ones, ws.x1, D, nullptr, 0};
  ECHO_TRY(launch_gemm_bf16("gemm_oc_bf16", 2, with_part(g), st));
  // FFN
  ECHO_TRY(launch_modln_x1(1, ws.x2, n, D, mod + 3 * D, mod + 4 * D, cfg->ln_eps, ws.b, st));
  g = GemmBf16Args{static_cast<P>(ws.b), D, nullptr, n, static_cast<P>(w->self.w1), static_cast<P>(w->self.w1), F,
                   D, static_cast<P>(w->self.b1), static_cast<P>(w->self.b1), n, F, D, ws.h, F,
                   nullptr, nullptr, 0, nullptr, 0};
  ECHO_TRY(launch_gemm_bf16("gemm_ffn_up_bf16", 1, with_part(g), st));
  g = GemmBf16Args{static_cast<P>(ws.h), F, nullptr, n, static_cast<P>(w->self.w2), static_cast<P>(w->self.w2), D,
                   F, static_cast<P>(w->self.b2), static_cast<P>(w->self.b2), n, D, F, y_sel, D,
                   mod + 5 * D, ws.x2, D, nullptr, 0};
  ECHO_TRY(launch_gemm_bf16("gemm_ffn_down_bf16", 2, with_part(g), st));
#undef ECHO_TRY
  return ECHO_OK;
}

int echo_cache_update(const echo_cache_cfg* cfg, const void* x, const int32_t* idx, const uint8_t* mask,
                      int32_t n_sel, const float* y_sel, void* xref, int8_t* codes, float* scale,
                      void* y, void* stream) {
  if (cfg == nullptr || cfg->L < 1 || cfg->D < 8 || (cfg->D % 8) != 0 || cfg->D > 16384 ||
      !ok_dtype(cfg->dtype))
    return ECHO_EINVAL;
  if (n_sel < 0 || n_sel > cfg->L) return ECHO_EINVAL;
  if (!ok_ptr(x) || !ok_ptr(mask) || !ok_ptr(xref) || !ok_ptr(codes) || !ok_ptr(scale) || !ok_ptr(y))
    return ECHO_EINVAL;
  if (n_sel > 0 && (!ok_ptr(idx) || !ok_ptr(y_sel))) return ECHO_EINVAL;
  return device_status(launch_cache_update(cfg->dtype == ECHO_BF16, x, idx, mask, n_sel, cfg->L, cfg->D,
                                           y_sel, xref, codes, scale, y,
                                           static_cast<hipStream_t>(stream)));
}

int echo_cache_update_codec(const echo_cache_cfg* cfg, int32_t codec, const void* x, const int32_t* idx,
                            const uint8_t* mask, int32_t n_sel, const float* y_sel, void* xref, void* store,
                            int8_t* codes, float* scale, void* y, void* stream) {
  if (cfg == nullptr || cfg->L < 1 || cfg->D < 8 || (cfg->D % 8) != 0 || cfg->D > 16384 ||
      !ok_dtype(cfg->dtype))
    return ECHO_EINVAL;
  if (codec != ECHO_CODEC_RESIDUAL_INT8 && codec != ECHO_CODEC_FULL && codec != ECHO_CODEC_NAIVE_INT8)
    return ECHO_EINVAL;
  if (n_sel < 0 || n_sel > cfg->L) return ECHO_EINVAL;
  if (!ok_ptr(x) || !ok_ptr(mask) || !ok_ptr(xref) || !ok_ptr(y)) return ECHO_EINVAL;
  if (codec == ECHO_CODEC_FULL ? !ok_ptr(store) : (!ok_ptr(codes) || !ok_ptr(scale))) return ECHO_EINVAL;
  if (n_sel > 0 && (!ok_ptr(idx) || !ok_ptr(y_sel))) return ECHO_EINVAL;
  return device_status(launch_cache_codec(cfg->dtype == ECHO_BF16, codec, x, idx, mask, n_sel, cfg->L, cfg->D,
                                          y_sel, xref, store, codes, scale, y, static_cast<hipStream_t>(stream)));
}


int echo_refcache_init(const echo_refcache_cfg* cfg, const echo_refcache_state* st, void* stream) {
  if (!refcache_cfg_ok(cfg) || !refcache_state_ok(st)) return ECHO_EINVAL;
  return device_status(launch_refcache_init(cfg->L, cfg->L / cfg->chain_len, cfg->capacity, st->refcount,
                                            st->free_list, st->free_top, st->chain_ref, st->ent_slot,
                                            st->ent_kind, st->scale, static_cast<hipStream_t>(stream)));
}

int echo_refcache_update(const echo_refcache_cfg* cfg, const echo_refcache_state* st, const void* x,
                         const int32_t* idx, const uint8_t* mask, int32_t n_sel, const float* y_sel,
                         void* xref, void* y, void* stream) {
  if (!refcache_cfg_ok(cfg) || !refcache_state_ok(st)) return ECHO_EINVAL;
  if (n_sel < 0 || n_sel > cfg->L) return ECHO_EINVAL;
  if (!ok_ptr(x) || !ok_ptr(mask) || !ok_ptr(xref) || !ok_ptr(y)) return ECHO_EINVAL;
  if (n_sel > 0 && (!ok_ptr(idx) || !ok_ptr(y_sel))) return ECHO_EINVAL;
  return device_status(launch_refcache_update(
      cfg->dtype == ECHO_BF16, x, idx, mask, n_sel, cfg->L, cfg->D, cfg->chain_len, cfg->tau, y_sel, st->pool,
      st->refcount, st->free_list, st->free_top, st->chain_ref, st->ent_slot, st->ent_kind, st->codes,
      st->scale, xref, y, static_cast<hipStream_t>(stream)));
}

int echo_mfma_ceiling(int32_t pattern, int32_t data, double seconds, double* tflops, void* stream) {
  if ((pattern != ECHO_MFMA_ATTENTION && pattern != ECHO_MFMA_GEMM) ||
      (data != ECHO_OPERANDS_CONSTANT && data != ECHO_OPERANDS_GAUSSIAN) || !(seconds > 0.0 && seconds <= 60.0) ||
      tflops == nullptr)
    return ECHO_EINVAL;
  const hipError_t e = run_mfma_ceiling(pattern, data == ECHO_OPERANDS_GAUSSIAN, seconds, tflops,
                                        static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ECHO_OK : device_status(e);
}

int echo_profile_enable(int on) {
  profile_set(on != 0);
  return ECHO_OK;
}

int echo_profile_read(echo_kernel_time* out, int32_t max) {
  if (max < 0 || (max > 0 && out == nullptr)) return -ECHO_EINVAL;
  int n = 0;
  int status = ECHO_OK;
  for (const TimingRecord& r : g_records) {
    float ms = 0.0f;
    hipError_t e = hipEventSynchronize(r.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess) {
      g_last_hip_error = static_cast<int>(e);
      status = ECHO_EDEVICE;
    }
    int slot = -1;
    for (int i = 0; i < n; ++i)
      if (strcmp(out[i].name, r.name) == 0) slot = i;
    if (slot < 0 && n < max) {
      slot = n++;
      out[slot].name = r.name;
      out[slot].launches = 0;
      out[slot].total_ms = 0.0;
    }
    if (slot >= 0) {
      out[slot].launches += 1;
      out[slot].total_ms += ms;
    }
    g_event_pool.push_back(r.start);
    g_event_pool.push_back(r.stop);
  }
  g_records.clear();
  return status == ECHO_OK ? n : -status;
}

}  // extern "C"
