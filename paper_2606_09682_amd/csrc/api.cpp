// C ABI of the decode megakernel: handle lifecycle, launch, schedule
// introspection.  Host code only; the kernel lives in megakernel.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/amk.h"
#include "device.h"
#include "schedule.h"

using amk::DevLayer;
using amk::DevModel;
using amk::Schedule;
using amk::Shape;
using amk::amk_internal_attn_scratch;
using amk::amk_internal_launch;
using amk::amk_internal_occupancy;
using amk::amk_internal_prepare;
using amk::amk_internal_read_probe;
using amk::amk_internal_static_scratch;
using amk::amk_internal_threads;

constexpr int kVariants = 3;
bool valid_variant(int v) { return v >= 0 && v < kVariants; }

// One schedule variant as uploaded: device task table, queue offsets, trace.
// Each variant owns its counters and epoch: a counter's target is
// epoch * (its producers per launch), which holds only while every launch
// that touched the counter ran the same schedule.
struct DevSchedule {
  const amk_task_t* tasks = nullptr;
  const int32_t* queue_start = nullptr;
  uint64_t* trace = nullptr;
  uint32_t* counters = nullptr;
  size_t counter_bytes = 0;
  uint32_t epoch = 0;
};

struct amk_handle_s {
  Shape s;
  int device = 0;
  Schedule sch[kVariants];      // AMK_SCHEDULE_SHORT, _LONG, _TINY
  DevSchedule dsch[kVariants];
  int last_variant = -1;
  DevModel dm;
  void* d_block = nullptr;      // one device allocation for tables and scratch
  int32_t* h_status = nullptr;  // host-mapped
  int32_t* h_abort = nullptr;   // host-mapped
  // amk_create_static: the device block is the library's static scratch
  // array, and the status / abort / done words are device words in it
  bool is_static = false;
  int32_t* d_words = nullptr;   // static handles: status at [0], abort at [16]
  void* last_stream = nullptr;
  bool launched = false;
  uint64_t timeout_ticks = 0;
  // the last kv_cache / logits pointers found to be device memory of this
  // device with room for a step's accesses (the check is skipped while the
  // caller keeps passing them)
  const void* ok_kv = nullptr;
  const void* ok_logits = nullptr;
};

namespace {

// Restores the caller's current device on scope exit.
struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) return;
    ok = dev < 0 || dev == prev || hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int check_linear(const amk_linear_t& l, int fmt) {
  if (!l.w || !aligned16(l.w)) return AMK_ERR_INVALID_ARGUMENT;
  if (fmt == AMK_WEIGHTS_W8A16 && (!l.scale || ((uintptr_t)l.scale & 3u))) return AMK_ERR_INVALID_ARGUMENT;
  if (fmt == AMK_WEIGHTS_W4A16 && (!l.scale || ((uintptr_t)l.scale & 1u))) return AMK_ERR_INVALID_ARGUMENT;
  return AMK_OK;
}

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

size_t amk_kv_cache_bytes_of(const Shape& s) { return (size_t)s.L * 2 * s.nkv * (size_t)s.max_seq * s.hd * 2; }

// The live handle of each device whose device memory is the static scratch
// array (at most one: the array holds one handle's tables and scratch).
constexpr int kMaxDevices = 64;
std::mutex g_static_mu;
amk_handle_s* g_static_owner[kMaxDevices] = {};

bool claim_static(int device, amk_handle_s* h) {
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (device < 0 || device >= kMaxDevices || g_static_owner[device]) return false;
  g_static_owner[device] = h;
  return true;
}

void release_static(int device, amk_handle_s* h) {
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (device >= 0 && device < kMaxDevices && g_static_owner[device] == h) g_static_owner[device] = nullptr;
}

void free_handle(amk_handle_s* h) {
  if (!h) return;
  DeviceGuard g(h->device);
  if (h->launched) (void)hipDeviceSynchronize();
  if (h->is_static) release_static(h->device, h);
  else if (h->d_block) (void)hipFree(h->d_block);
  if (h->h_status) (void)hipHostFree(h->h_status);
  if (h->h_abort) (void)hipHostFree(h->h_abort);
  delete h;
}

// Whether [p, p + bytes) lies inside one allocation of device memory on
// `device` (not host, pinned host or another device's memory).
bool device_range(const void* p, size_t bytes, int device) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (a.type != hipMemoryTypeDevice || a.device != device) return false;
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  const uintptr_t b = (uintptr_t)base, q = (uintptr_t)p;
  return q >= b && bytes <= size && q - b <= size - bytes;
}

}  // namespace

extern "C" {

const char* amk_status_string(int status) {
  switch (status) {
    case AMK_OK: return "ok";
    case AMK_ERR_INVALID_ARGUMENT: return "invalid argument";
    case AMK_ERR_UNSUPPORTED: return "unsupported model shape or layout";
    case AMK_ERR_SCHEDULE_REJECTED: return "schedule rejected by the static check";
    case AMK_ERR_OUT_OF_MEMORY: return "out of device or host memory";
    case AMK_ERR_DEVICE: return "HIP runtime error";
    case AMK_ERR_COOPERATIVE_UNSUPPORTED: return "cooperative launch unavailable or too few co-resident workgroups";
    case AMK_ERR_TIMEOUT: return "device counter wait timed out";
    case AMK_ERR_BAD_STATE: return "handle in an error state";
    case AMK_ERR_ABORTED: return "launch aborted by the host abort flag";
    case AMK_ERR_NONFINITE: return "a logit was NaN";
    default: return "unknown status";
  }
}

size_t amk_kv_cache_bytes(const amk_config_t* cfg) {
  Shape s;
  if (amk::derive_shape(cfg, nullptr, 1, &s, nullptr) != AMK_OK) return 0;
  return amk_kv_cache_bytes_of(s);
}

int amk_schedule_size(const amk_config_t* cfg, const amk_tuning_t* tuning, int32_t n_cu, int32_t variant,
                      int32_t* n_tasks, int32_t* n_counters) {
  if (!valid_variant(variant)) return AMK_ERR_INVALID_ARGUMENT;
  try {
    Shape s;
    int st = amk::derive_shape(cfg, tuning, n_cu, &s, nullptr);
    if (st != AMK_OK) return st;
    Schedule sch = amk::build_schedule(s, n_cu, variant);
    if (n_tasks) *n_tasks = (int32_t)sch.tasks.size();
    if (n_counters) *n_counters = sch.n_counters;
    return AMK_OK;
  } catch (const std::bad_alloc&) {
    return AMK_ERR_OUT_OF_MEMORY;
  } catch (...) {
    return AMK_ERR_INVALID_ARGUMENT;
  }
}

int amk_schedule_export(const amk_config_t* cfg, const amk_tuning_t* tuning, int32_t n_cu, int32_t variant,
                        amk_task_t* tasks, int32_t cap, int32_t* n_tasks, int32_t* n_counters) {
  if (!valid_variant(variant)) return AMK_ERR_INVALID_ARGUMENT;
  try {
    Shape s;
    int st = amk::derive_shape(cfg, tuning, n_cu, &s, nullptr);
    if (st != AMK_OK) return st;
    Schedule sch = amk::build_schedule(s, n_cu, variant);
    if (n_tasks) *n_tasks = (int32_t)sch.tasks.size();
    if (n_counters) *n_counters = sch.n_counters;
    if (!tasks || cap < (int32_t)sch.tasks.size()) return AMK_ERR_INVALID_ARGUMENT;
    std::memcpy(tasks, sch.tasks.data(), sch.tasks.size() * sizeof(amk_task_t));
    return AMK_OK;
  } catch (const std::bad_alloc&) {
    return AMK_ERR_OUT_OF_MEMORY;
  } catch (...) {
    return AMK_ERR_INVALID_ARGUMENT;
  }
}

int amk_schedule_check(const amk_config_t* cfg, const amk_tuning_t* tuning, int32_t n_cu, const amk_task_t* tasks,
                       int32_t n_tasks, int32_t n_counters, amk_check_report_t* report) {
  if (!report) return AMK_ERR_INVALID_ARGUMENT;
  try {
    Shape s;
    int st = amk::derive_shape(cfg, tuning, n_cu, &s, nullptr);
    if (st != AMK_OK) return st;
    amk::check_schedule(s, n_cu, tasks, n_tasks, n_counters, report);
    return AMK_OK;
  } catch (const std::bad_alloc&) {
    return AMK_ERR_OUT_OF_MEMORY;
  } catch (...) {
    return AMK_ERR_INVALID_ARGUMENT;
  }
}

// Whether the kernel of a schedule runs all its tasks: the tiny-context
// kernel has no attention tasks, split merges or chained inline tasks, and
// computes the attention of every O task itself (aux 1); the other kernel
// computes it in none.
static bool kernel_runs(const Schedule& sch, bool tiny) {
  for (const amk_task_t& t : sch.tasks) {
    if (tiny && (t.op == AMK_OP_ATTN || t.op == AMK_OP_COMBINE || t.chain_counter >= 0)) return false;
    if (t.op == AMK_OP_O && (t.aux == 1) != tiny) return false;
  }
  return true;
}

int amk_check_config(const amk_config_t* cfg, int32_t n_cu) {
  try {
    Shape s;
    int st = amk::derive_shape(cfg, nullptr, n_cu, &s, nullptr);
    if (st != AMK_OK) return st;
    for (int v = 0; v < kVariants; ++v) {
      Schedule sch = amk::build_schedule(s, n_cu, v);
      amk_check_report_t rep;
      if (!amk::check_schedule(s, n_cu, sch.tasks.data(), (int)sch.tasks.size(), sch.n_counters, &rep) ||
          !kernel_runs(sch, v == AMK_SCHEDULE_TINY))
        return AMK_ERR_SCHEDULE_REJECTED;
    }
    return AMK_OK;
  } catch (const std::bad_alloc&) {
    return AMK_ERR_OUT_OF_MEMORY;
  } catch (...) {
    return AMK_ERR_INVALID_ARGUMENT;
  }
}

// amk_create and amk_create_static: `use_static` puts every byte of device
// memory the handle owns into the static scratch array (no allocation).
static int create_impl(const amk_config_t* cfg, const amk_weights_t* w, const amk_tuning_t* tuning,
                       amk_handle_t* out, bool use_static) {
  if (!out) return AMK_ERR_INVALID_ARGUMENT;
  *out = nullptr;
  if (!cfg || !w) return AMK_ERR_INVALID_ARGUMENT;
  amk_handle_s* h = nullptr;
  try {
    DeviceGuard guard(cfg->device);
    if (!guard.ok) return AMK_ERR_DEVICE;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return AMK_ERR_DEVICE;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return AMK_ERR_DEVICE;
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) return AMK_ERR_UNSUPPORTED;
    int coop = 0;
    if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess || !coop)
      return AMK_ERR_COOPERATIVE_UNSUPPORTED;
    const int n_cu = prop.multiProcessorCount;

    Shape s;
    std::string why;
    int st = amk::derive_shape(cfg, tuning, n_cu, &s, &why);
    if (st != AMK_OK) return st;

    // weights: presence, alignment, format
    if (!w->embed || !aligned16(w->embed) || !w->final_norm || !aligned16(w->final_norm) || !w->layers)
      return AMK_ERR_INVALID_ARGUMENT;
    if (s.tied) {
      if (w->lm_head.w) return AMK_ERR_INVALID_ARGUMENT;
    } else if (check_linear(w->lm_head, s.fmt) != AMK_OK) {
      return AMK_ERR_INVALID_ARGUMENT;
    }
    for (int l = 0; l < s.L; ++l) {
      const amk_layer_weights_t& lw = w->layers[l];
      if (!lw.attn_norm || !aligned16(lw.attn_norm) || !lw.mlp_norm || !aligned16(lw.mlp_norm))
        return AMK_ERR_INVALID_ARGUMENT;
      const amk_linear_t* ls[7] = {&lw.q, &lw.k, &lw.v, &lw.o, &lw.gate, &lw.up, &lw.down};
      for (auto* lp : ls)
        if (check_linear(*lp, s.fmt) != AMK_OK) return AMK_ERR_INVALID_ARGUMENT;
    }

    h = new amk_handle_s();
    h->s = s;
    h->device = dev;
    for (int v = 0; v < kVariants; ++v) {
      h->sch[v] = amk::build_schedule(s, n_cu, v);
      amk_check_report_t rep;
      if (!amk::check_schedule(s, n_cu, h->sch[v].tasks.data(), (int)h->sch[v].tasks.size(), h->sch[v].n_counters,
                               &rep)) {
        std::fprintf(stderr, "amk: schedule variant %d rejected (rule %d): %s\n", v, rep.rule, rep.message);
        free_handle(h);
        return AMK_ERR_SCHEDULE_REJECTED;
      }
    }
    const Schedule& sl = h->sch[AMK_SCHEDULE_LONG];
    if (sl.n_lm_slots != h->sch[AMK_SCHEDULE_SHORT].n_lm_slots ||
        sl.n_lm_slots != h->sch[AMK_SCHEDULE_TINY].n_lm_slots) {  // the argmax slots are shared
      free_handle(h);
      return AMK_ERR_SCHEDULE_REJECTED;
    }
    // each schedule runs on a kernel that carries only its own attention code
    for (int v = 0; v < kVariants; ++v) {
      if (!kernel_runs(h->sch[v], v == AMK_SCHEDULE_TINY)) {
        std::fprintf(stderr, "amk: schedule variant %d has tasks its kernel does not run\n", v);
        free_handle(h);
        return AMK_ERR_SCHEDULE_REJECTED;
      }
    }

    // LDS: activation vector (padded to a whole granule: 1 KiB of weights
    // covers 1024 int8 or 2048 int4 columns), static per-row data, residual
    // rows, partials / attention scratch, and under W4A16 the sums of each
    // 32 consecutive activations
    const int nsw = amk_internal_threads() / 64 - 1;
    const size_t act = round_up((size_t)std::max({s.H, s.nq * s.hd, s.I}), s.fmt == AMK_WEIGHTS_W4A16 ? 2048 : 1024);
    const size_t act_lds = act + act / 16;  // one float4 of padding per 64 floats (staggered LDS banks)
    const size_t xsum = s.fmt == AMK_WEIGHTS_W4A16 ? act / 32 : 0;
    // per-wave partial stride in whole float4s keeps every region 16-byte aligned
    const size_t pstride = round_up((size_t)s.max_jobs, 4);
    const size_t scr = std::max<size_t>((size_t)nsw * pstride, (size_t)amk_internal_attn_scratch(s.group, s.hd));
    const size_t lds_bytes = (act_lds + 3 * pstride + scr + xsum) * 4;
    int max_lds = 0;
    if (hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) {
      free_handle(h);
      return AMK_ERR_DEVICE;
    }
    if ((long)lds_bytes + 256 > (long)max_lds) {
      std::fprintf(stderr, "amk: needs %zu B of LDS per workgroup, device allows %d\n", lds_bytes, max_lds);
      free_handle(h);
      return AMK_ERR_UNSUPPORTED;
    }
    if (amk_internal_prepare(s.hd, s.group, s.fmt, (int)lds_bytes) != AMK_OK) {
      free_handle(h);
      return AMK_ERR_DEVICE;
    }
    int per_cu = 0;
    if (amk_internal_occupancy(s.hd, s.group, s.fmt, (int)lds_bytes, &per_cu) != AMK_OK || per_cu < 1) {
      free_handle(h);
      return AMK_ERR_COOPERATIVE_UNSUPPORTED;
    }

    // device block layout
    const int L = s.L;
    const int n_lm = sl.n_lm_slots;
    const int rec = s.group * (amk::kPartHead + s.hd);
    struct Region { size_t off, bytes; };
    size_t top = 0;
    auto take = [&](size_t bytes) { Region r{top, bytes}; top = round_up(top + bytes, 256); return r; };
    const Region r_layers = take(sizeof(DevLayer) * L);
    const Region r_rope = take(sizeof(float) * 2 * (size_t)s.max_seq * s.half);
    // vectors of the residual stream and per-layer activations on separate
    // 256-byte boundaries (64 floats)
    const int xs = (int)round_up(s.H, 64), qs = (int)round_up((size_t)s.nq * s.hd, 64);
    const int as = (int)round_up(s.I, 64), ps = (int)round_up((size_t)s.nkv * s.nsplit * rec, 64);
    const Region r_x = take(sizeof(float) * (size_t)(2 * L + 1) * xs);
    const Region r_q = take(sizeof(float) * (size_t)L * qs);
    const Region r_part = take(sizeof(float) * (size_t)L * ps);
    const Region r_o = take(sizeof(float) * (size_t)L * qs);
    const Region r_a = take(sizeof(float) * (size_t)L * as);
    const Region r_argp = take(sizeof(float) * 2 * n_lm);
    const Region r_next = take(sizeof(int32_t));
    const Region r_abort = take(sizeof(int32_t));
    // static handles: status and abort words, each on its own 64 bytes
    const Region r_words = take(use_static ? 2 * 64 : 0);
    const bool tracing = tuning && tuning->trace;
    Region r_tasks[kVariants], r_queue[kVariants], r_trace[kVariants], r_ctr[kVariants];
    for (int v = 0; v < kVariants; ++v) {
      r_ctr[v] = take(sizeof(uint32_t) * amk::kCounterStride * amk::kCounterReplicas * (size_t)h->sch[v].n_counters);
      r_tasks[v] = take(sizeof(amk_task_t) * h->sch[v].tasks.size());
      r_queue[v] = take(sizeof(int32_t) * h->sch[v].queue_start.size());
      r_trace[v] = take(tracing ? sizeof(uint64_t) * AMK_TRACE_FIELDS * h->sch[v].tasks.size() : 0);
    }
    if (use_static) {
      void* sp = nullptr;
      size_t cap = 0;
      if (amk::amk_internal_static_scratch(dev, &sp, &cap) != AMK_OK) {
        free_handle(h);
        return AMK_ERR_DEVICE;
      }
      if (top > cap) {
        std::fprintf(stderr, "amk: amk_create_static needs %zu bytes of device memory, the static scratch holds %zu\n",
                     top, cap);
        free_handle(h);
        return AMK_ERR_OUT_OF_MEMORY;
      }
      if (!claim_static(dev, h)) {
        std::fprintf(stderr, "amk: device %d already has a live amk_create_static handle\n", dev);
        free_handle(h);
        return AMK_ERR_BAD_STATE;
      }
      h->is_static = true;
      h->d_block = sp;
    } else if (hipMalloc(&h->d_block, top) != hipSuccess) {
      h->d_block = nullptr;
      free_handle(h);
      return AMK_ERR_OUT_OF_MEMORY;
    }
    char* base = (char*)h->d_block;
    // zeroes the counters, the scratch and (static handles) the status words:
    // the static array keeps whatever the previous handle left in it
    if (hipMemset(h->d_block, 0, top) != hipSuccess) {
      free_handle(h);
      return AMK_ERR_DEVICE;
    }
    int32_t* d_status = nullptr;
    int32_t* d_hab = nullptr;
    if (use_static) {
      h->d_words = (int32_t*)(base + r_words.off);
      d_status = h->d_words;
      d_hab = h->d_words + 16;
    } else {
      if (hipHostMalloc((void**)&h->h_status, sizeof(int32_t), hipHostMallocMapped | hipHostMallocCoherent) !=
              hipSuccess ||
          hipHostMalloc((void**)&h->h_abort, sizeof(int32_t), hipHostMallocMapped | hipHostMallocCoherent) !=
              hipSuccess) {
        free_handle(h);
        return AMK_ERR_OUT_OF_MEMORY;
      }
      *(volatile int32_t*)h->h_status = 0;
      *(volatile int32_t*)h->h_abort = 0;
      if (hipHostGetDevicePointer((void**)&d_status, h->h_status, 0) != hipSuccess ||
          hipHostGetDevicePointer((void**)&d_hab, h->h_abort, 0) != hipSuccess) {
        free_handle(h);
        return AMK_ERR_DEVICE;
      }
    }

    // host-built tables
    std::vector<DevLayer> layers(L);
    for (int l = 0; l < L; ++l) {
      const amk_layer_weights_t& lw = w->layers[l];
      const amk_linear_t* ls[7] = {&lw.q, &lw.k, &lw.v, &lw.o, &lw.gate, &lw.up, &lw.down};
      for (int i = 0; i < 7; ++i) {
        layers[l].w[i] = ls[i]->w;
        layers[l].s[i] = s.fmt != AMK_WEIGHTS_BF16 ? ls[i]->scale : nullptr;
      }
      layers[l].attn_norm = (const uint16_t*)lw.attn_norm;
      layers[l].mlp_norm = (const uint16_t*)lw.mlp_norm;
    }
    // RoPE table: angle p * theta^(-2i/d), cos and sin evaluated in float64, stored float32
    std::vector<float> rope(2 * (size_t)s.max_seq * s.half);
    for (int i = 0; i < s.half; ++i) {
      const double inv = std::pow((double)s.theta, -2.0 * i / (double)s.hd);
      for (int p = 0; p < s.max_seq; ++p) {
        const double a = (double)p * inv;
        rope[2 * ((size_t)p * s.half + i)] = (float)std::cos(a);
        rope[2 * ((size_t)p * s.half + i) + 1] = (float)std::sin(a);
      }
    }
    bool ok = hipMemcpy(base + r_layers.off, layers.data(), r_layers.bytes, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemcpy(base + r_rope.off, rope.data(), r_rope.bytes, hipMemcpyHostToDevice) == hipSuccess;
    for (int v = 0; v < kVariants && ok; ++v)
      ok = hipMemcpy(base + r_tasks[v].off, h->sch[v].tasks.data(), r_tasks[v].bytes, hipMemcpyHostToDevice) ==
               hipSuccess &&
           hipMemcpy(base + r_queue[v].off, h->sch[v].queue_start.data(), r_queue[v].bytes, hipMemcpyHostToDevice) ==
               hipSuccess;
    if (!ok) {
      free_handle(h);
      return AMK_ERR_DEVICE;
    }

    DevModel& m = h->dm;
    std::memset(&m, 0, sizeof(m));
    m.H = s.H; m.L = L; m.nq = s.nq; m.nkv = s.nkv; m.hd = s.hd; m.I = s.I; m.V = s.V; m.max_seq = s.max_seq;
    m.fmt = s.fmt;
    m.lm_fmt = s.tied ? AMK_WEIGHTS_BF16 : s.fmt;
    m.qglog2 = 0;
    while (s.qgroup && (1 << m.qglog2) < s.qgroup) ++m.qglog2;
    m.group = s.group; m.half = s.half;
    m.half_log2 = 0;
    while ((1 << m.half_log2) < s.half) ++m.half_log2;
    m.units = s.units; m.q_units = s.q_units; m.nsplit = s.nsplit; m.n_lm = n_lm;
    m.gq2 = s.group + 2;
    m.npg = s.npg;
    m.n_cu = n_cu;
    m.eps = s.eps;
    m.attn_scale = (float)(1.0 / std::sqrt((double)s.hd));
    m.embed = (const uint16_t*)w->embed;
    m.final_norm = (const uint16_t*)w->final_norm;
    m.lm_w = s.tied ? w->embed : w->lm_head.w;
    m.lm_s = m.lm_fmt != AMK_WEIGHTS_BF16 ? w->lm_head.scale : nullptr;
    m.layers = (const DevLayer*)(base + r_layers.off);
    m.rope = (const float2*)(base + r_rope.off);
    m.x = (float*)(base + r_x.off);
    m.q = (float*)(base + r_q.off);
    m.part = (float*)(base + r_part.off);
    m.o = (float*)(base + r_o.off);
    m.a = (float*)(base + r_a.off);
    m.xs = xs; m.qs = qs; m.as = as; m.ps = ps;
    m.argp = (float*)(base + r_argp.off);
    m.next_token = (int32_t*)(base + r_next.off);
    m.counters = nullptr;  // per launch: the variant's counters
    m.dev_abort = (int32_t*)(base + r_abort.off);
    m.host_status = d_status;
    m.host_abort = d_hab;
    for (int v = 0; v < kVariants; ++v) {
      h->dsch[v].tasks = (const amk_task_t*)(base + r_tasks[v].off);
      h->dsch[v].queue_start = (const int32_t*)(base + r_queue[v].off);
      h->dsch[v].trace = tracing ? (uint64_t*)(base + r_trace[v].off) : nullptr;
      h->dsch[v].counters = (uint32_t*)(base + r_ctr[v].off);
      h->dsch[v].counter_bytes = r_ctr[v].bytes;
    }
    m.lds_act = (int32_t)act_lds;
    m.part_stride = (int32_t)pstride;
    m.lds_scr = (int32_t)scr;
    m.lds_bytes = (int32_t)lds_bytes;

    const int timeout_us = tuning && tuning->timeout_us > 0 ? tuning->timeout_us : 2000000;
    h->timeout_ticks = (uint64_t)timeout_us * 100ull;  // the device wall clock runs at 100 MHz
    *out = h;
    return AMK_OK;
  } catch (const std::bad_alloc&) {
    free_handle(h);
    return AMK_ERR_OUT_OF_MEMORY;
  } catch (...) {
    free_handle(h);
    return AMK_ERR_INVALID_ARGUMENT;
  }
}

int amk_create(const amk_config_t* cfg, const amk_weights_t* w, const amk_tuning_t* tuning, amk_handle_t* out) {
  return create_impl(cfg, w, tuning, out, false);
}

int amk_create_static(const amk_config_t* cfg, const amk_weights_t* w, const amk_tuning_t* tuning,
                      amk_handle_t* out) {
  return create_impl(cfg, w, tuning, out, true);
}

int amk_decode_step(amk_handle_t h, int32_t token, int32_t pos, void* kv_cache, float* logits, void* stream) {
  if (!h || !kv_cache || !logits) return AMK_ERR_INVALID_ARGUMENT;
  if (token < 0 || token >= h->s.V || pos < 0 || pos >= h->s.max_seq) return AMK_ERR_INVALID_ARGUMENT;
  if (((uintptr_t)kv_cache & 255u) != 0 || !aligned16(logits)) return AMK_ERR_INVALID_ARGUMENT;
  // (a static handle's status word is device memory: reading it would wait
  // for the device, so the sticky check is not made for it)
  if (!h->is_static) {
    const int sticky = *(volatile int32_t*)h->h_status;
    if (sticky != 0) return sticky;
  }
  DeviceGuard guard(h->device);
  if (!guard.ok) return AMK_ERR_DEVICE;
  // another stream while the previous one still has work queued (which may
  // be this handle's last step): two steps would share the handle's
  // counters and scratch.  A stream that no longer exists reports an error
  // here, not pending work.
  if (h->launched && stream != h->last_stream) {
    const hipError_t q = hipStreamQuery((hipStream_t)h->last_stream);
    if (q != hipSuccess) (void)hipGetLastError();
    if (q == hipErrorNotReady) return AMK_ERR_BAD_STATE;
  }
  if (kv_cache != h->ok_kv) {
    if (!device_range(kv_cache, amk_kv_cache_bytes_of(h->s), h->device)) return AMK_ERR_INVALID_ARGUMENT;
    h->ok_kv = kv_cache;
  }
  if (logits != h->ok_logits) {
    if (!device_range(logits, sizeof(float) * (size_t)h->s.V, h->device)) return AMK_ERR_INVALID_ARGUMENT;
    h->ok_logits = logits;
  }
  const int variant = pos + 1 <= h->s.tiny_context    ? AMK_SCHEDULE_TINY
                      : pos + 1 <= h->s.short_context ? AMK_SCHEDULE_SHORT
                                                      : AMK_SCHEDULE_LONG;
  DevSchedule& ds = h->dsch[variant];
  DevModel m = h->dm;
  m.tasks = ds.tasks;
  m.queue_start = ds.queue_start;
  m.trace = ds.trace;
  m.counters = ds.counters;
  const uint32_t epoch = ds.epoch + 1;  // counter targets are epoch * producers, mod 2^32
  const int st = amk_internal_launch(&m, variant == AMK_SCHEDULE_TINY, token, pos, epoch, (uint16_t*)kv_cache, logits,
                                     h->timeout_ticks, stream);
  if (st != AMK_OK) return st;
  h->last_variant = variant;
  ds.epoch = epoch;
  h->last_stream = stream;
  h->launched = true;
  return AMK_OK;
}

const int32_t* amk_next_token_ptr(amk_handle_t h) { return h ? h->dm.next_token : nullptr; }

int amk_copy_next_token(amk_handle_t h, int32_t* dst, void* stream) {
  if (!h || !dst) return AMK_ERR_INVALID_ARGUMENT;
  DeviceGuard guard(h->device);
  if (hipMemcpyAsync(dst, h->dm.next_token, sizeof(int32_t), hipMemcpyDeviceToHost, (hipStream_t)stream) !=
          hipSuccess ||
      hipStreamSynchronize((hipStream_t)stream) != hipSuccess)
    return AMK_ERR_DEVICE;
  return AMK_OK;
}

int amk_read_probe(const void* buf, int64_t bytes, int32_t blocks, uint32_t* sink, void* stream) {
  if (!buf || !sink || bytes <= 0 || bytes % 16 || !aligned16(buf) || blocks < 1 || blocks > 65536)
    return AMK_ERR_INVALID_ARGUMENT;
  return amk_internal_read_probe(buf, bytes, blocks, sink, stream);
}

int amk_get_status(amk_handle_t h) {
  if (!h) return AMK_ERR_INVALID_ARGUMENT;
  DeviceGuard guard(h->device);
  if (h->launched && hipStreamSynchronize((hipStream_t)h->last_stream) != hipSuccess) return AMK_ERR_DEVICE;
  if (h->is_static) {
    int32_t v = 0;
    if (hipMemcpy(&v, h->d_words, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess) return AMK_ERR_DEVICE;
    return v;
  }
  return *(volatile int32_t*)h->h_status;
}

int amk_reset(amk_handle_t h) {
  if (!h) return AMK_ERR_INVALID_ARGUMENT;
  DeviceGuard guard(h->device);
  if (hipDeviceSynchronize() != hipSuccess) return AMK_ERR_DEVICE;
  for (auto& ds : h->dsch) {
    if (hipMemset(ds.counters, 0, ds.counter_bytes) != hipSuccess) return AMK_ERR_DEVICE;
    ds.epoch = 0;
  }
  if (hipMemset(h->dm.dev_abort, 0, sizeof(int32_t)) != hipSuccess) return AMK_ERR_DEVICE;
  if (h->is_static && hipMemset(h->d_words, 0, sizeof(int32_t)) != hipSuccess) return AMK_ERR_DEVICE;
  if (hipDeviceSynchronize() != hipSuccess) return AMK_ERR_DEVICE;
  if (!h->is_static) {
    *(volatile int32_t*)h->h_status = 0;
  }
  return AMK_OK;
}

int amk_trace_copy(amk_handle_t h, uint64_t* dst, int64_t capacity, int32_t* n_tasks, int32_t* variant) {
  if (!h || !dst) return AMK_ERR_INVALID_ARGUMENT;
  if (h->last_variant < 0 || !h->dsch[h->last_variant].trace) return AMK_ERR_BAD_STATE;
  const int v = h->last_variant;
  const size_t n = h->sch[v].tasks.size();
  if (n_tasks) *n_tasks = (int32_t)n;
  if (variant) *variant = v;
  if (capacity < (int64_t)(n * AMK_TRACE_FIELDS)) return AMK_ERR_INVALID_ARGUMENT;
  DeviceGuard guard(h->device);
  if (h->launched && hipStreamSynchronize((hipStream_t)h->last_stream) != hipSuccess) return AMK_ERR_DEVICE;
  if (hipMemcpy(dst, h->dsch[v].trace, n * AMK_TRACE_FIELDS * sizeof(uint64_t), hipMemcpyDeviceToHost) != hipSuccess)
    return AMK_ERR_DEVICE;
  return AMK_OK;
}

int amk_set_abort(amk_handle_t h, int32_t value) {
  if (!h) return AMK_ERR_INVALID_ARGUMENT;
  if (h->is_static) return AMK_ERR_UNSUPPORTED;  // its abort word is device memory
  __atomic_store_n(h->h_abort, value ? 1 : 0, __ATOMIC_SEQ_CST);
  return AMK_OK;
}

int amk_destroy(amk_handle_t h) {
  free_handle(h);
  return AMK_OK;
}

}  // extern "C"
