// Host side of libbifattn: argument validation, work splitting, workspace
// ownership, launches and the C ABI declared in include/bifattn.h.
#include "bifattn.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <new>
#include <vector>

#include "bifattn_internal.h"

using namespace bifattn;

struct bifattn_plan_s {
  bifattn_dims_t dims{};
  float scale = 0.f;
  int p = 0, M = 0;  // query rows per (sample, group) unit (heads x tokens), rows per group
  int ntok = 1;
  int ctx_mode = kCtxNone;
  int dec_tiles = 1;
  int ctx_keys = 0, S_c = 0, ctx_row_blocks = 1, n_ctx_blocks = 0, n_ctx_small_blocks = 0;
  int ctx_wide = 0;  // many-row path: waves per work-group of the 32x32 kernel, or 0
  int dec_keys = 0, S_d = 0, n_dec_blocks = 0;
  int rep_keys = 0, S_r = 0, n_rep_blocks = 0;
  int fused = 1;
  int fork = 0;        // many-row path: decode launch on a side stream beside the context kernel
  // The plan's own stream (non-blocking, default priority): the workspace is
  // allocated and freed in its order (stream-ordered allocator, so that
  // freeing it does not synchronise the device) and, on many-row plans with
  // a large decode part, the decode launch runs on it beside the context
  // kernel.
  hipStream_t side = nullptr;
  bool ws_async = false;  // workspace from hipMallocAsync (else hipMalloc)
  hipEvent_t fork_ev = nullptr, join_ev = nullptr;
  // Recorded on the call's stream after the last launch of every call: what
  // destroy and set_timing wait for (the plan's own work, not the device's).
  hipEvent_t done_ev = nullptr;
  bool done_recorded = false;
  int path = BIFATTN_PATH_BIFURCATED;  // resolved: bifurcated or standard
  int device = 0;
  // workspace
  void* ws = nullptr;
  size_t ws_bytes = 0;
  float* ctx_acc = nullptr;
  float2* ctx_ml = nullptr;
  float* dec_acc = nullptr;
  float2* dec_ml = nullptr;
  int* status = nullptr;
  // timing
  int timed_kernel = -1;
  int timing_cap = 0;
  int timing_n = 0;
  std::vector<hipEvent_t> events;
};

namespace {

// Events that only order the plan's work on its device (the completion
// mark, the side-stream fork and join): no timing, and no system-scope fence
// when recorded (the host reads nothing through them; a recorded system
// fence writes back the L2 and costs ~3 us per call). Each kernel's own
// end-of-dispatch release still publishes its results to the device.
constexpr unsigned kOrderEventFlags = hipEventDisableTiming | hipEventDisableSystemFence;

constexpr int kCUs = 256;  // MI355X compute units; split heuristics aim at whole waves of them

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Tuning overrides from the environment: a positive integer, else `fallback`.
int env_int(const char* name, int fallback) {
  const char* v = std::getenv(name);
  if (!v || !*v) return fallback;
  char* end = nullptr;
  long x = std::strtol(v, &end, 10);
  return (end && *end == 0 && x > 0 && x < (1 << 30)) ? (int)x : fallback;
}

// A switch from the environment: -1 when unset or not an integer, else its value.
int env_switch(const char* name) {
  const char* v = std::getenv(name);
  if (!v || !*v) return -1;
  char* end = nullptr;
  long x = std::strtol(v, &end, 10);
  return (end && *end == 0 && x >= 0 && x < 16) ? (int)x : -1;
}

bool aligned(const void* ptr, uintptr_t a) { return ((uintptr_t)ptr & (a - 1)) == 0; }

// The plan's workspace lives on the device that was current at its creation:
// a call is accepted only on a stream of that device (the null stream: the
// current device), so that no kernel runs on one GPU against another GPU's
// workspace.
bool on_plan_device(const bifattn_plan_s* P, hipStream_t stream) {
  int dev = -1;
  if (stream) {
    hipDevice_t d = -1;
    if (hipStreamGetDevice(stream, &d) != hipSuccess) {
      (void)hipGetLastError();
      return false;
    }
    dev = d;
  } else if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return dev == P->device;
}

// Keys one decode work-group reads: the whole decode cache up to 1024 keys
// (each work-group writes partials for p rows per wave, so short chunks
// multiply that traffic, and ragged lengths leave short chunks nearly empty),
// halved (down to 128) only while fewer than half as many work-groups as
// CUs would exist.
int dec_chunk_keys(int64_t units, int64_t rows) {
  int keys = (int)std::min<int64_t>(1024, std::max<int64_t>(128, round_up(rows, 128)));
  while (keys > 128 && units * ceil_div(rows, keys) < kCUs / 2) keys /= 2;
  return keys;
}
// Rounding of the many-row context chunk: the wide kernel runs 128-key
// stages when its chunks are multiples of 128 keys, so chunks of at least
// 1024 keys are rounded to 128.
int ck_step(int key_step, int64_t m_c, int64_t splits) {
  return key_step == 64 && ceil_div(m_c, splits) >= 1024 ? 128 : key_step;
}

// Keys one replicated-ablation work-group reads: `start` by default, halved
// (down to 128) while fewer than two work-groups per CU would exist.
int seq_keys(int64_t units, int64_t rows, int start) {
  int keys = start;
  while (keys > 128 && units * ceil_div(rows, keys) < 2 * kCUs) keys /= 2;
  return keys;
}

// allow_fork: the many-row path may run the decode launch on the plan's own
// stream (off for the allocation-free entry point, which owns no stream).
bifattn_status_t plan_splits(bifattn_plan_s* P, bool allow_fork = true) {
  const bifattn_dims_t& d = P->dims;
  P->ntok = d.n > 0 ? d.n : 1;
  // The n tokens of a head are consecutive rows of q and out, so a unit's
  // query rows are its p heads times n tokens.
  P->p = d.h / d.g * P->ntok;
  P->M = d.b * P->p;
  P->dec_tiles = P->p <= 16 ? 1 : (P->p <= 32 ? 2 : 4);
  const int64_t M = P->M;
  const int64_t units = (int64_t)d.b * d.g;
  if (M <= 64) {
    // Few rows per group: S_c work-groups per group, interleaved over the
    // group's tiles; about four of them, each with 1024..2048 keys (2-4
    // decode work-groups' worth): fewer, longer context work-groups leave
    // fewer partials to merge, too few stop covering the decode part's time.
    P->ctx_mode = M <= 16 ? kCtxSmall1 : (M <= 32 ? kCtxSmall2 : kCtxSmall4);
    const int64_t quarter = round_up(ceil_div(d.m_c, 4), kWaves * kTileKeys);
    const int def_keys = (int)std::min<int64_t>(2048, std::max<int64_t>(1024, quarter));
    const int keys = (int)round_up(env_int("BIFATTN_CTX_KEYS", def_keys), kWaves * kTileKeys);
    P->ctx_keys = keys;
    P->ctx_row_blocks = 1;
  } else {
    // Many rows: eight-wave work-groups of 128 rows share each staged
    // K_c/V_c tile; about two work-groups per CU (four waves per SIMD).
    // With a large decode part (16 MiB of decode KV or more) the decode
    // launch runs on a side stream beside the context kernel, which then
    // takes about one work-group per CU and leaves the other slot to the
    // decode work-groups (the context part is bound by the matrix cores, the
    // decode part by HBM). BIFATTN_FORK=0/1 forces it off/on.
    P->ctx_mode = kCtxLarge;
    //
    // The decode launch goes to the plan's side stream, beside the context
    // kernel (eight 16-row waves per work-group, at two per CU, leaving room
    // for decode work-groups), when the decode part is large (16 MiB or more)
    // and comparable to the context part: its HBM time at ~5 TB/s above half
    // the context's matrix time at ~1 PFLOP/s. Otherwise both parts run one
    // after the other on the call's stream, and d = 128 takes the 32x32 MFMA
    // context kernel (work-groups of eight waves of 32 rows, one per CU, from
    // 256 rows per group, else of four, two per CU), which fills its CUs'
    // registers and LDS and so leaves no room for decode work beside it.
    // With the side stream, 256 or more rows per group still take the 32x32
    // kernel, on a grid of five eighths of the CUs: the decode work-groups
    // run on the rest (measured on the ragged GQA workload: 265 vs 276 us per
    // step with the 16x16 kernel beside the decode launch; 160 work-groups
    // 234-236 vs 240-241 us for 192, 243 for 144, 258 for 208: the two parts
    // take about as long either way, and fewer key splits leave the combine
    // fewer partials). 128 to 255 rows per group take its four-wave form on
    // about one work-group per CU, the other slot of each CU left to decode
    // work-groups (4 draft tokens: 89.8-89.9 vs 92.7-92.9 us for the 16x16
    // kernel; 128-192 or 320 work-groups 92-94 us); fewer rows keep the 16x16
    // kernel.
    // BIFATTN_FORK=0/1 and BIFATTN_CTX_WIDE=0/1 force either choice (d = 64
    // always takes the kernel of 16-row waves).
    const double dec_bytes = 2.0 * d.b * d.g * (double)d.m_d_max * kv_row_bytes(d.d, d.kv_type);
    const double ctx_flops = 4.0 * d.h * P->ntok * d.d * (double)d.b * d.m_c;
    const int fork_env = env_switch("BIFATTN_FORK");
    const bool big_decode = dec_bytes >= 16.0 * (1 << 20) && dec_bytes / 5e12 > 0.5 * ctx_flops / 1e15;
    P->fork = allow_fork && d.m_d_max > 0 && (fork_env == -1 ? big_decode : fork_env == 1);
    const int wide_env = env_switch("BIFATTN_CTX_WIDE");
    const bool wide = d.d == 128 && (wide_env == -1 ? (!P->fork || M >= 128) : wide_env == 1);
    P->ctx_wide = wide ? (M >= 256 ? 8 : 4) : 0;
    const int block_rows = wide ? 32 * P->ctx_wide : kLargeRowsPerBlock;
    const int key_step = wide ? 64 : kTileKeys;  // keys per stage of the kernel's loop
    P->ctx_row_blocks = (int)ceil_div(M, block_rows);
    // About one work-group per CU for eight-wave work-groups, two for
    // four-wave ones; with the side stream, one per CU for the 16x16 kernel
    // (the decode work-groups take the other slot of each CU) and for the
    // four-wave 32x32 kernel, and five eighths of the CUs for the eight-wave
    // 32x32 kernel (the decode work-groups take the rest).
    const int per_cu = P->ctx_wide == 8 ? 1 : 2;
    const int target = P->fork ? (P->ctx_wide == 8 ? kCUs * 5 / 8 : kCUs) : per_cu * kCUs;
    int64_t splits = ceil_div(env_int("BIFATTN_CTX_WGS", target), (int64_t)d.g * P->ctx_row_blocks);
    if (splits < 1) splits = 1;
    const int64_t ck = round_up(ceil_div(d.m_c, splits), ck_step(key_step, d.m_c, splits));
    P->ctx_keys = (int)round_up(env_int("BIFATTN_CTX_KEYS", (int)ck), key_step);
  }
  P->S_c = (int)ceil_div(d.m_c, P->ctx_keys);
  P->n_ctx_blocks = P->ctx_mode == kCtxLarge ? d.g * P->S_c * P->ctx_row_blocks : 0;
  P->n_ctx_small_blocks = P->ctx_mode == kCtxLarge ? 0 : d.g * P->S_c;
  if (d.m_d_max > 0) {
    P->dec_keys = (int)round_up(env_int("BIFATTN_DEC_KEYS", dec_chunk_keys(units, d.m_d_max)),
                                kTileKeys);
    P->S_d = (int)ceil_div(d.m_d_max, P->dec_keys);
  } else {
    P->dec_keys = kTileKeys;
    P->S_d = 0;
  }
  P->n_dec_blocks = (int)(units * P->S_d);
  const int64_t rep_rows = (int64_t)d.m_c + d.m_d_max;
  P->rep_keys = (int)round_up(env_int("BIFATTN_REP_KEYS", seq_keys(units, rep_rows, 1024)),
                              kTileKeys);
  P->S_r = (int)ceil_div(rep_rows, P->rep_keys);
  P->n_rep_blocks = (int)(units * P->S_r);
  // Few-row context and decode work-groups share one launch (the context
  // part then overlaps the decode part's streaming); BIFATTN_LAUNCH=2 splits
  // them into two launches. The many-row context path has a kernel of its
  // own (eight-wave work-groups), launched before the decode work-groups.
  const int launch = env_int("BIFATTN_LAUNCH", 1);
  P->fused = launch == 1 && P->ctx_mode != kCtxLarge ? 1 : 0;
  // The workload-based switch: the standard path reads the context once per
  // sample but needs one launch and no partials. It wins while every unit is
  // resident in one round of work-groups (b*g <= 512), has at most two query
  // tiles, and holds few keys: up to ~1100 (~600 once units share CUs), or
  // ~2200 when the bifurcated context part has 64 or more rows per group
  // (its four-tile and many-row work-groups are the costly ones). These are
  // the crossovers measured on MI355X over 38 MHA/GQA/MQA shapes.
  if (d.path == BIFATTN_PATH_AUTO) {
    const int64_t keys = (int64_t)d.m_c + d.m_d_max;
    const int64_t lmax = M >= 64 ? 2200 : (units > kCUs ? 600 : 1100);
    const bool small = units <= 2 * kCUs && P->p <= 32 && keys <= lmax;
    P->path = small ? BIFATTN_PATH_STANDARD : BIFATTN_PATH_BIFURCATED;
  } else {
    P->path = d.path;
  }
  if ((int64_t)P->n_ctx_blocks + P->n_ctx_small_blocks + P->n_dec_blocks > INT32_MAX / 2 ||
      units * P->S_r > INT32_MAX / 2)
    return BIFATTN_EINVAL;
  return BIFATTN_OK;
}

// Byte offsets of the workspace parts (256-byte aligned) and its size: the
// context partials, the decode partials (sized for the replicated ablation's
// splits too when `replicated`), and the status word.
struct WorkspaceLayout {
  size_t ctx_acc = 0, ctx_ml = 0, dec_acc = 0, dec_ml = 0, status = 0, bytes = 0;
};
WorkspaceLayout workspace_layout(const bifattn_plan_s* P, bool replicated) {
  const bifattn_dims_t& d = P->dims;
  const size_t D = (size_t)d.d;
  const size_t ctx_rows = (size_t)d.g * P->S_c * P->M;
  const int s_dec = replicated && P->S_r > P->S_d ? P->S_r : P->S_d;
  const size_t dec_rows = (size_t)d.b * d.g * (size_t)s_dec * kWaves * P->p;
  WorkspaceLayout L;
  size_t off = 0;
  L.ctx_acc = off;
  off = align256(off + ctx_rows * D * 4);
  L.ctx_ml = off;
  off = align256(off + ctx_rows * 8);
  L.dec_acc = off;
  off = align256(off + dec_rows * D * 4);
  L.dec_ml = off;
  off = align256(off + dec_rows * 8);
  L.status = off;
  L.bytes = align256(off + 4);
  return L;
}

void set_workspace(bifattn_plan_s* P, void* base_ptr, const WorkspaceLayout& L) {
  char* base = static_cast<char*>(base_ptr);
  P->ws = base_ptr;
  P->ws_bytes = L.bytes;
  P->ctx_acc = reinterpret_cast<float*>(base + L.ctx_acc);
  P->ctx_ml = reinterpret_cast<float2*>(base + L.ctx_ml);
  P->dec_acc = reinterpret_cast<float*>(base + L.dec_acc);
  P->dec_ml = reinterpret_cast<float2*>(base + L.dec_ml);
  P->status = reinterpret_cast<int*>(base + L.status);
}

bifattn_status_t check_dims(const bifattn_dims_t* d) {
  if (!d) return BIFATTN_EINVAL;
  if (d->b < 1 || d->h < 1 || d->g < 1 || d->m_c < 1 || d->m_d_max < 0 || d->n < 0)
    return BIFATTN_EINVAL;
  if (d->h % d->g) return BIFATTN_EINVAL;
  if (!(std::isfinite(d->scale))) return BIFATTN_EINVAL;
  if (d->kv_type != BIFATTN_KV_BF16 && d->kv_type != BIFATTN_KV_FP8_E4M3 &&
      d->kv_type != BIFATTN_KV_INT8 && d->kv_type != BIFATTN_KV_INT4)
    return BIFATTN_EINVAL;
  if (d->path != BIFATTN_PATH_AUTO && d->path != BIFATTN_PATH_BIFURCATED &&
      d->path != BIFATTN_PATH_STANDARD)
    return BIFATTN_EINVAL;
  if (d->d != 64 && d->d != 128) return BIFATTN_EUNSUPPORTED;
  const double ntok = d->n > 0 ? d->n : 1;
  if ((double)(d->h / d->g) * ntok > kMaxP) return BIFATTN_EUNSUPPORTED;
  // element counts of the largest tensors must stay far from 2^62
  const double lim = 4.0e18;
  const double dd = d->d;
  if ((double)d->b * d->h * ntok * dd > lim || (double)d->g * d->m_c * dd > lim ||
      (double)d->b * d->g * ((double)d->m_c + d->m_d_max) * dd > lim)
    return BIFATTN_EINVAL;
  if ((double)d->b * d->h * ntok > INT32_MAX / 2 || (double)d->b * d->g > INT32_MAX / 2)
    return BIFATTN_EINVAL;
  // Kernels address one cache (a group's context, a sample's decode rows, or
  // both in the replicated ablation) with 32-bit byte offsets.
  if (((double)d->m_c + d->m_d_max) * kv_row_bytes(d->d, d->kv_type) > INT32_MAX)
    return BIFATTN_EUNSUPPORTED;
  return BIFATTN_OK;
}

// Mark the end of a call's work on its stream.
void mark_done(bifattn_plan_s* P, hipStream_t stream) {
  if (!P->done_ev) return;
  if (hipEventRecord(P->done_ev, stream) == hipSuccess)
    P->done_recorded = true;
  else
    (void)hipGetLastError();
}

// The events of a call's last launch with the completion mark added: the
// launch records the plan's done event itself at the kernel's end (no
// separate marker on the stream), unless it already records a timing stop.
LaunchEvents last_launch(bifattn_plan_s* P, LaunchEvents ev) {
  if (!ev.stop && P->done_ev) {
    ev.stop = P->done_ev;
    P->done_recorded = true;
  }
  return ev;
}

// Wait for the plan's own enqueued work: the last call's end (every earlier
// call of the plan ran on a stream its successor was ordered after, or is
// covered by the caller's one-stream-at-a-time contract) and the side stream.
bool wait_done(bifattn_plan_s* P) {
  bool ok = true;
  if (P->done_recorded && hipEventSynchronize(P->done_ev) != hipSuccess) ok = false;
  if (P->side && hipStreamSynchronize(P->side) != hipSuccess) ok = false;
  return ok;
}

void free_events(bifattn_plan_s* P);

// Free everything the plan owns and the plan itself. The workspace is freed
// in the order of the plan's own stream (a stream-ordered free waits for
// that stream only; hipFree would synchronise the whole device), so the
// caller must have waited for the plan's work first.
bool release_plan(bifattn_plan_s* P) {
  bool ok = true;
  free_events(P);
  if (P->done_ev) (void)hipEventDestroy(P->done_ev);
  if (P->fork_ev) (void)hipEventDestroy(P->fork_ev);
  if (P->join_ev) (void)hipEventDestroy(P->join_ev);
  if (P->ws) {
    if (P->ws_async)
      ok = hipFreeAsync(P->ws, P->side) == hipSuccess && hipStreamSynchronize(P->side) == hipSuccess;
    else
      ok = hipFree(P->ws) == hipSuccess;
  }
  if (P->side) (void)hipStreamDestroy(P->side);
  if (!ok) (void)hipGetLastError();
  delete P;
  return ok;
}

void free_events(bifattn_plan_s* P) {
  for (hipEvent_t e : P->events) (void)hipEventDestroy(e);
  P->events.clear();
  P->timing_cap = P->timing_n = 0;
  P->timed_kernel = -1;
}

// Event pair of one timed section of this call, if that section is being
// timed. With `in_kernel`, the section's launches record the pair
// themselves (the first launch's kernel start, the last launch's kernel
// end: first() / last() / both()), so the time is the kernels' own, as a
// kernel trace shows it; otherwise the pair is recorded on the stream around
// the section.
struct TimedSection {
  bifattn_plan_s* P;
  hipStream_t stream;
  bool on = false;
  bool in_kernel = false;
  TimedSection(bifattn_plan_s* P_, int kernel, hipStream_t s, bool in_kernel_ = false)
      : P(P_), stream(s), in_kernel(in_kernel_) {
    on = P->timed_kernel == kernel && P->timing_n < P->timing_cap;
    if (on && !in_kernel) (void)hipEventRecord(P->events[2 * P->timing_n], stream);
  }
  hipEvent_t ev(int k) const { return on && in_kernel ? P->events[2 * P->timing_n + k] : nullptr; }
  LaunchEvents first() const { return LaunchEvents{ev(0), nullptr}; }
  LaunchEvents last() const { return LaunchEvents{nullptr, ev(1)}; }
  LaunchEvents both() const { return LaunchEvents{ev(0), ev(1)}; }
  // This section's events where they are set, else the other's (sections of
  // one call may share a launch; at most one of them is being timed).
  static LaunchEvents either(const LaunchEvents& a, const LaunchEvents& b) {
    return LaunchEvents{a.start ? a.start : b.start, a.stop ? a.stop : b.stop};
  }
  // For sections that span streams: the pair recorded on the call's stream.
  void record_start() {
    if (on && in_kernel) (void)hipEventRecord(P->events[2 * P->timing_n], stream);
  }
  void record_stop() {
    if (on && in_kernel) (void)hipEventRecord(P->events[2 * P->timing_n + 1], stream);
  }
  void end() {
    if (on) {
      if (!in_kernel) (void)hipEventRecord(P->events[2 * P->timing_n + 1], stream);
      ++P->timing_n;
      on = false;
    }
  }
};

PartialsParams base_params(const bifattn_plan_s* P, const void* q, const int32_t* lens,
                           const float* k_scale) {
  PartialsParams K{};
  K.q = static_cast<const uint16_t*>(q);
  K.lens = lens;
  K.k_scale = k_scale;
  K.ctx_acc = P->ctx_acc;
  K.ctx_ml = P->ctx_ml;
  K.dec_acc = P->dec_acc;
  K.dec_ml = P->dec_ml;
  K.status = P->status;
  K.b = P->dims.b;
  K.h = P->dims.h * P->ntok;
  K.g = P->dims.g;
  K.p = P->p;
  K.M = P->M;
  K.ntok = P->ntok;
  K.m_c = P->dims.m_c;
  K.m_d_max = P->dims.m_d_max;
  // scale * (q . k) = |scale| * ((-q) . k): a negative scale negates q, which
  // is exact in bf16, so the kernels only ever see a positive scale.
  K.scale_log2 = std::fabs(P->scale) * 1.4426950408889634f;
  K.q_sign = P->scale < 0.f ? 0x80008000u : 0u;
  return K;
}

CombineParams combine_params(const bifattn_plan_s* P, const int32_t* lens, const float* k_scale,
                             const float* v_scale, float* out) {
  CombineParams C{};
  C.k_scale = k_scale;
  C.v_scale = v_scale;
  C.ctx_acc = P->ctx_acc;
  C.ctx_ml = P->ctx_ml;
  C.dec_acc = P->dec_acc;
  C.dec_ml = P->dec_ml;
  C.lens = lens;
  C.out = out;
  C.status = P->status;
  C.b = P->dims.b;
  C.h = P->dims.h * P->ntok;
  C.g = P->dims.g;
  C.p = P->p;
  C.M = P->M;
  C.m_d_max = P->dims.m_d_max;
  return C;
}

}  // namespace

extern "C" {

const char* bifattn_status_string(bifattn_status_t s) {
  switch (s) {
    case BIFATTN_OK: return "ok";
    case BIFATTN_EINVAL: return "invalid argument";
    case BIFATTN_EUNSUPPORTED:
      return "unsupported shape (d must be 64 or 128, (h/g)*n at most 64, one sample's cache "
             "rows under 2^31 bytes)";
    case BIFATTN_EALIGN: return "tensor pointer not 16-byte aligned (decode_lens: 4-byte)";
    case BIFATTN_ENOMEM: return "device memory allocation failed";
    case BIFATTN_EHIP: return "HIP runtime error";
    case BIFATTN_ELENS: return "a decode length was outside [0, m_d_max] and was clamped";
    case BIFATTN_ESCALE: return "a key or value scale was not a positive normal float";
    case BIFATTN_ESCRATCH:
      return "the workspace of this problem exceeds the fixed scratch buffer of "
             "bifattn_decode_noalloc (64 MiB)";
  }
  return "unknown status";
}

int32_t bifattn_version(void) { return BIFATTN_VERSION; }

bifattn_status_t bifattn_plan_create(const bifattn_dims_t* dims, bifattn_plan_t* plan) {
  if (!plan) return BIFATTN_EINVAL;
  *plan = nullptr;
  bifattn_status_t st = check_dims(dims);
  if (st != BIFATTN_OK) return st;
  bifattn_plan_s* P = new (std::nothrow) bifattn_plan_s();
  if (!P) return BIFATTN_ENOMEM;
  P->dims = *dims;
  P->scale = dims->scale != 0.f ? dims->scale : 1.0f / std::sqrt((float)dims->d);
  st = plan_splits(P);
  if (st != BIFATTN_OK) {
    delete P;
    return st;
  }
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1 || hipGetDevice(&P->device) != hipSuccess) {
    delete P;
    return BIFATTN_EHIP;
  }
  const WorkspaceLayout L = workspace_layout(P, true);
  const size_t off = L.bytes;
  if (hipStreamCreateWithFlags(&P->side, hipStreamNonBlocking) != hipSuccess) {
    (void)hipGetLastError();
    delete P;
    return BIFATTN_EHIP;
  }
  if (hipMallocAsync(&P->ws, off, P->side) == hipSuccess) {
    P->ws_async = true;
  } else {
    (void)hipGetLastError();
    P->ws = nullptr;
    if (hipMalloc(&P->ws, off) != hipSuccess) {
      (void)hipGetLastError();
      P->ws = nullptr;
      release_plan(P);
      return BIFATTN_ENOMEM;
    }
  }
  set_workspace(P, P->ws, L);
  if (hipMemsetAsync(P->status, 0, 4, P->side) != hipSuccess ||
      hipStreamSynchronize(P->side) != hipSuccess ||
      hipEventCreateWithFlags(&P->done_ev, kOrderEventFlags) != hipSuccess) {
    (void)hipGetLastError();
    release_plan(P);
    return BIFATTN_EHIP;
  }
  if (P->fork) {
    if (hipEventCreateWithFlags(&P->fork_ev, kOrderEventFlags) != hipSuccess ||
        hipEventCreateWithFlags(&P->join_ev, kOrderEventFlags) != hipSuccess) {
      (void)hipGetLastError();
      P->fork = 0;
    }
  }
  *plan = P;
  return BIFATTN_OK;
}

bifattn_status_t bifattn_plan_destroy(bifattn_plan_t P) {
  if (!P) return BIFATTN_OK;
  bifattn_status_t st = BIFATTN_OK;
  if (!wait_done(P)) st = BIFATTN_EHIP;
  if (!release_plan(P)) st = BIFATTN_EHIP;
  return st;
}

bifattn_status_t bifattn_plan_get_info(bifattn_plan_t P, bifattn_plan_info_t* info) {
  if (!P || !info) return BIFATTN_EINVAL;
  info->ctx_keys_per_block = P->ctx_keys;
  info->ctx_splits = P->S_c;
  info->ctx_row_blocks = P->ctx_row_blocks;
  info->ctx_blocks = P->n_ctx_blocks + P->n_ctx_small_blocks;
  info->dec_keys_per_block = P->dec_keys;
  info->dec_splits = P->S_d * kWaves;
  info->dec_blocks = P->n_dec_blocks;
  info->fused = P->fused;
  info->path = P->path;
  info->workspace_bytes = P->ws_bytes;
  info->ctx_kernel = P->ctx_mode != kCtxLarge ? 0 : (P->ctx_wide ? 2 : 1);
  info->side_stream = P->fork;
  return BIFATTN_OK;
}

namespace {

// One decode step of plan P (a created plan, or the allocation-free entry
// point's plan on the stack, whose workspace is the fixed scratch buffer).
bifattn_status_t decode_impl(bifattn_plan_s* P, const void* q, const void* Kc, const void* Vc,
                             const void* Kd, const void* Vd, const int32_t* decode_lens,
                             const float* k_scale, const float* v_scale, float* out,
                             hipStream_t stream) {
  if (!P || !q || !Kc || !Vc || !out || !on_plan_device(P, stream)) return BIFATTN_EINVAL;
  if (!aligned(k_scale, 4) || !aligned(v_scale, 4)) return BIFATTN_EALIGN;
  const bool has_dec = P->dims.m_d_max > 0;
  if (has_dec && (!Kd || !Vd || !decode_lens)) return BIFATTN_EINVAL;
  if (!aligned(q, 16) || !aligned(Kc, 16) || !aligned(Vc, 16) || !aligned(out, 16))
    return BIFATTN_EALIGN;
  if (has_dec && (!aligned(Kd, 16) || !aligned(Vd, 16) || !aligned(decode_lens, 4)))
    return BIFATTN_EALIGN;
  const int kv = P->dims.kv_type;
  PartialsParams K = base_params(P, q, has_dec ? decode_lens : nullptr, k_scale);
  K.Kc = static_cast<const uint8_t*>(Kc);
  K.Vc = static_cast<const uint8_t*>(Vc);
  K.Kd = static_cast<const uint8_t*>(Kd);
  K.Vd = static_cast<const uint8_t*>(Vd);
  K.dec_rows = P->dims.m_d_max;
  K.len_offset = 0;
  K.ctx_keys = P->ctx_keys;
  K.S_c = P->S_c;
  K.ctx_row_blocks = P->ctx_row_blocks;
  K.ctx_wide = P->ctx_wide;
  K.dec_keys = P->dec_keys;
  K.S_d = P->S_d;
  TimedSection whole(P, BIFATTN_KERNEL_CALL, stream);
  TimedSection part(P, BIFATTN_KERNEL_PARTIALS, stream, true);
  TimedSection ctxs(P, BIFATTN_KERNEL_CONTEXT, stream, true);
  TimedSection decs(P, BIFATTN_KERNEL_DECODE, stream, true);
  auto ev = [](const LaunchEvents& a, const LaunchEvents& b) { return TimedSection::either(a, b); };
  hipError_t e = hipSuccess;
  if (P->path == BIFATTN_PATH_STANDARD) {
    K.out = out;
    K.v_scale = v_scale;
    const LaunchEvents lev = part.both();
    e = launch_standard(K, P->dims.d, kv, P->dec_tiles, stream, last_launch(P, lev));
    part.end();
    whole.end();
    if (lev.stop) mark_done(P, stream);
    return e == hipSuccess ? BIFATTN_OK : BIFATTN_EHIP;
  }
  K.n_ctx_blocks = 0;
  K.n_ctx_small_blocks = 0;
  K.n_dec_blocks = 0;
  // Two launches: the first carries the start event and the second the end
  // event, unless there are no decode work-groups (then the first carries both).
  const bool two = P->n_dec_blocks > 0;
  if (P->ctx_mode == kCtxLarge && P->fork && two) {
    // The decode work-groups on the side stream, beside the many-row context
    // kernel; the call's stream waits for them before the combine. The timed
    // section is the call's stream from before the fork to after the join.
    PartialsParams Kd = K;
    Kd.n_dec_blocks = P->n_dec_blocks;
    part.record_start();
    if (hipEventRecord(P->fork_ev, stream) != hipSuccess ||
        hipStreamWaitEvent(P->side, P->fork_ev, 0) != hipSuccess)
      return BIFATTN_EHIP;
    e = launch_partials(Kd, P->dims.d, kv, kCtxNone, P->dec_tiles, P->side, decs.both());
    K.n_ctx_blocks = P->n_ctx_blocks;
    if (e == hipSuccess) e = launch_ctx_large(K, P->dims.d, kv, stream, ctxs.both());
    if (e == hipSuccess && (hipEventRecord(P->join_ev, P->side) != hipSuccess ||
                            hipStreamWaitEvent(stream, P->join_ev, 0) != hipSuccess))
      e = hipErrorUnknown;
    part.record_stop();
    K.n_ctx_blocks = 0;
  } else if (P->ctx_mode == kCtxLarge) {
    // The many-row context kernel, then the decode work-groups.
    K.n_ctx_blocks = P->n_ctx_blocks;
    e = launch_ctx_large(K, P->dims.d, kv, stream,
                         ev(two ? part.first() : part.both(), ctxs.both()));
    K.n_ctx_blocks = 0;
    K.n_dec_blocks = P->n_dec_blocks;
    if (e == hipSuccess && two)
      e = launch_partials(K, P->dims.d, kv, kCtxNone, P->dec_tiles, stream,
                          ev(part.last(), decs.both()));
  } else if (P->fused) {
    // One launch holds the context and the decode work-groups: each section
    // times it.
    K.n_ctx_small_blocks = P->n_ctx_small_blocks;
    K.n_dec_blocks = P->n_dec_blocks;
    e = launch_partials(K, P->dims.d, kv, P->ctx_mode, P->dec_tiles, stream,
                        ev(ev(part.both(), ctxs.both()), decs.both()));
  } else {
    K.n_ctx_small_blocks = P->n_ctx_small_blocks;
    e = launch_partials(K, P->dims.d, kv, P->ctx_mode, P->dec_tiles, stream,
                        ev(two ? part.first() : part.both(), ctxs.both()));
    K.n_ctx_small_blocks = 0;
    K.n_dec_blocks = P->n_dec_blocks;
    if (e == hipSuccess && two)
      e = launch_partials(K, P->dims.d, kv, kCtxNone, P->dec_tiles, stream,
                          ev(part.last(), decs.both()));
  }
  part.end();
  ctxs.end();
  decs.end();
  if (e != hipSuccess) {
    mark_done(P, stream);
    return BIFATTN_EHIP;
  }
  TimedSection comb(P, BIFATTN_KERNEL_COMBINE, stream, true);
  CombineParams C = combine_params(P, has_dec ? decode_lens : nullptr, k_scale, v_scale, out);
  C.S_c = P->S_c;
  C.S_d = P->S_d * kWaves;
  const LaunchEvents cev = comb.both();
  e = launch_combine(C, P->dims.d, stream, last_launch(P, cev));
  comb.end();
  whole.end();
  if (cev.stop) mark_done(P, stream);
  return e == hipSuccess ? BIFATTN_OK : BIFATTN_EHIP;
}

}  // namespace

bifattn_status_t bifattn_decode_scaled(bifattn_plan_t P, const void* q, const void* Kc,
                                       const void* Vc, const void* Kd, const void* Vd,
                                       const int32_t* decode_lens, const float* k_scale,
                                       const float* v_scale, float* out, hipStream_t stream) {
  return decode_impl(P, q, Kc, Vc, Kd, Vd, decode_lens, k_scale, v_scale, out, stream);
}

bifattn_status_t bifattn_decode_noalloc(const bifattn_dims_t* dims, const void* q, const void* Kc,
                                        const void* Vc, const void* Kd, const void* Vd,
                                        const int32_t* decode_lens, const float* k_scale,
                                        const float* v_scale, float* out, hipStream_t stream) {
  bifattn_status_t st = check_dims(dims);
  if (st != BIFATTN_OK) return st;
  // A plan on the stack: the same splits as bifattn_plan_create's (the
  // decode launch always on the call's stream), no events, no streams, no
  // device allocation.
  bifattn_plan_s P;
  P.dims = *dims;
  P.scale = dims->scale != 0.f ? dims->scale : 1.0f / std::sqrt((float)dims->d);
  st = plan_splits(&P, false);
  if (st != BIFATTN_OK) return st;
  const WorkspaceLayout L = workspace_layout(&P, false);
  if (L.bytes > kScratchBytes) return BIFATTN_ESCRATCH;
  if (hipGetDevice(&P.device) != hipSuccess) {
    (void)hipGetLastError();
    return BIFATTN_EHIP;
  }
  void* scratch = nullptr;
  if (scratch_address(P.device, &scratch) != hipSuccess) {
    (void)hipGetLastError();
    return BIFATTN_EHIP;
  }
  set_workspace(&P, scratch, L);
  st = decode_impl(&P, q, Kc, Vc, Kd, Vd, decode_lens, k_scale, v_scale, out, stream);
  P.ws = nullptr;  // the scratch buffer is not the plan's to free
  return st;
}

bifattn_status_t bifattn_decode(bifattn_plan_t P, const void* q, const void* Kc, const void* Vc,
                                const void* Kd, const void* Vd, const int32_t* decode_lens,
                                float* out, hipStream_t stream) {
  return bifattn_decode_scaled(P, q, Kc, Vc, Kd, Vd, decode_lens, nullptr, nullptr, out, stream);
}

bifattn_status_t bifattn_decode_replicated_scaled(bifattn_plan_t P, const void* q, const void* K_,
                                                  const void* V_, const int32_t* decode_lens,
                                                  const float* k_scale, const float* v_scale,
                                                  float* out, hipStream_t stream) {
  if (!P || !q || !K_ || !V_ || !out || !on_plan_device(P, stream)) return BIFATTN_EINVAL;
  if (!aligned(k_scale, 4) || !aligned(v_scale, 4)) return BIFATTN_EALIGN;
  const bool has_dec = P->dims.m_d_max > 0;
  if (has_dec && !decode_lens) return BIFATTN_EINVAL;
  if (!aligned(q, 16) || !aligned(K_, 16) || !aligned(V_, 16) || !aligned(out, 16))
    return BIFATTN_EALIGN;
  if (has_dec && !aligned(decode_lens, 4)) return BIFATTN_EALIGN;
  PartialsParams K = base_params(P, q, has_dec ? decode_lens : nullptr, k_scale);
  K.Kd = static_cast<const uint8_t*>(K_);
  K.Vd = static_cast<const uint8_t*>(V_);
  K.dec_rows = P->dims.m_c + P->dims.m_d_max;
  K.len_offset = P->dims.m_c;
  K.dec_keys = P->rep_keys;
  K.S_d = P->S_r;
  K.S_c = 0;
  K.n_ctx_blocks = 0;
  K.n_ctx_small_blocks = 0;
  K.n_dec_blocks = P->n_rep_blocks;
  TimedSection whole(P, BIFATTN_KERNEL_CALL, stream);
  TimedSection part(P, BIFATTN_KERNEL_PARTIALS, stream, true);
  hipError_t e = launch_partials(K, P->dims.d, P->dims.kv_type, kCtxNone, P->dec_tiles, stream,
                                 part.both());
  part.end();
  if (e != hipSuccess) {
    mark_done(P, stream);
    return BIFATTN_EHIP;
  }
  TimedSection comb(P, BIFATTN_KERNEL_COMBINE, stream, true);
  CombineParams C = combine_params(P, has_dec ? decode_lens : nullptr, k_scale, v_scale, out);
  C.S_c = 0;
  C.S_d = P->S_r * kWaves;
  const LaunchEvents cev = comb.both();
  e = launch_combine(C, P->dims.d, stream, last_launch(P, cev));
  comb.end();
  whole.end();
  if (cev.stop) mark_done(P, stream);
  return e == hipSuccess ? BIFATTN_OK : BIFATTN_EHIP;
}

bifattn_status_t bifattn_decode_replicated(bifattn_plan_t P, const void* q, const void* K_,
                                           const void* V_, const int32_t* decode_lens, float* out,
                                           hipStream_t stream) {
  return bifattn_decode_replicated_scaled(P, q, K_, V_, decode_lens, nullptr, nullptr, out,
                                          stream);
}

bifattn_status_t bifattn_append_kv(bifattn_plan_t P, const void* k_new, const void* v_new,
                                   void* Kd, void* Vd, int32_t* decode_lens, hipStream_t stream) {
  if (!P || !k_new || !v_new || !Kd || !Vd || !decode_lens || P->dims.m_d_max < 1 ||
      !on_plan_device(P, stream))
    return BIFATTN_EINVAL;
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(Kd, 16) || !aligned(Vd, 16) ||
      !aligned(decode_lens, 4))
    return BIFATTN_EALIGN;
  AppendParams A{};
  A.k_new = static_cast<const uint8_t*>(k_new);
  A.v_new = static_cast<const uint8_t*>(v_new);
  A.Kd = static_cast<uint8_t*>(Kd);
  A.Vd = static_cast<uint8_t*>(Vd);
  A.lens = decode_lens;
  A.status = P->status;
  A.b = P->dims.b;
  A.g = P->dims.g;
  A.n = P->ntok;
  A.m_d_max = P->dims.m_d_max;
  const hipError_t e = launch_append(A, P->dims.d, P->dims.kv_type, stream,
                                     last_launch(P, LaunchEvents{}));
  return e == hipSuccess ? BIFATTN_OK : BIFATTN_EHIP;
}

bifattn_status_t bifattn_plan_status(bifattn_plan_t P, hipStream_t stream) {
  if (!P) return BIFATTN_EINVAL;
  if (hipStreamSynchronize(stream) != hipSuccess) return BIFATTN_EHIP;
  int flag = 0;
  if (hipMemcpy(&flag, P->status, sizeof flag, hipMemcpyDeviceToHost) != hipSuccess)
    return BIFATTN_EHIP;
  if (flag) {
    if (hipMemset(P->status, 0, sizeof flag) != hipSuccess) return BIFATTN_EHIP;
    return (flag & kStatusScale) ? BIFATTN_ESCALE : BIFATTN_ELENS;
  }
  return BIFATTN_OK;
}

bifattn_status_t bifattn_plan_set_timing(bifattn_plan_t P, bifattn_kernel_t kernel,
                                         int32_t capacity) {
  if (!P || capacity < 0 || (int)kernel < 0 || (int)kernel > BIFATTN_KERNEL_DECODE)
    return BIFATTN_EINVAL;
  if (!wait_done(P)) return BIFATTN_EHIP;  // the events to be freed may still be pending
  free_events(P);
  if (capacity == 0) return BIFATTN_OK;
  P->events.reserve(2 * (size_t)capacity);
  for (int i = 0; i < 2 * capacity; ++i) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) {
      free_events(P);
      return BIFATTN_ENOMEM;
    }
    P->events.push_back(e);
  }
  P->timed_kernel = (int)kernel;
  P->timing_cap = capacity;
  P->timing_n = 0;
  return BIFATTN_OK;
}

bifattn_status_t bifattn_plan_read_timing(bifattn_plan_t P, int32_t* calls, double* total_ms) {
  if (!P || !calls || !total_ms) return BIFATTN_EINVAL;
  double sum = 0.0;
  for (int k = 0; k < P->timing_n; ++k) {
    if (hipEventSynchronize(P->events[2 * k + 1]) != hipSuccess) return BIFATTN_EHIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, P->events[2 * k], P->events[2 * k + 1]) != hipSuccess)
      return BIFATTN_EHIP;
    sum += ms;
  }
  *calls = P->timing_n;
  *total_ms = sum;
  P->timing_n = 0;
  return BIFATTN_OK;
}

}  // extern "C"
