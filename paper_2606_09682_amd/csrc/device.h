// Device-side view of one handle: shape, borrowed weight pointers, handle-owned
// scratch and the uploaded schedule.  Passed BY VALUE as the megakernel's
// argument, so every field is a wave-uniform kernel-argument load.
#pragma once

#include <cstddef>
#include <cstdint>

#include "../../include/amk.h"

namespace amk {

enum { W_Q = 0, W_K, W_V, W_O, W_G, W_U, W_D, W_COUNT };

struct DevLayer {
  const void* w[W_COUNT];      // bf16 / int8 [out, in], or packed int4 [out, in / 2]
  const void* s[W_COUNT];      // fp32 [out] for int8, fp16 [out, in / group] for int4, else null
  const uint16_t* attn_norm;   // bf16 [H]
  const uint16_t* mlp_norm;    // bf16 [H]
};

// Counters live on separate 128-byte lines, each in kCounterReplicas copies
// (counter c, copy r at element (c * kCounterReplicas + r) * kCounterStride):
// a producer increments every copy, and workgroup b polls copy b % 16, so a
// line has 16 pollers (half an XCD) instead of the whole grid's 256.  With
// one line per counter the polls queue at that line's memory channel and
// delay the producers' increments (8B bf16: 160 us per step).
constexpr int kCounterStride = 32;  // uint32 elements
constexpr int kCounterReplicas = 16;

// Layout of one attention partial record for a (layer, kv head, split):
// for each of the `group` query heads: [m, l, pad, pad, acc[head_dim]].
constexpr int kPartHead = 4;  // floats before acc

struct DevModel {
  // shape
  int32_t H, L, nq, nkv, hd, I, V, max_seq;
  int32_t fmt;        // AMK_WEIGHTS_*
  int32_t lm_fmt;     // format of the LM head: fmt if untied, AMK_WEIGHTS_BF16 if tied
  int32_t qglog2;     // W4A16: log2 of the input columns per scale
  int32_t group, half, half_log2, units, q_units, nsplit, n_lm;
  int32_t gq2;        // group + 2: head slots of one KV group in QKV unit order
  int32_t npg;        // QKV tasks per KV group (producers of a group's QKV counter)
  int32_t n_cu;
  float eps;
  float attn_scale;   // 1 / sqrt(head_dim)
  // weights (borrowed)
  const uint16_t* embed;
  const uint16_t* final_norm;
  const void* lm_w;
  const void* lm_s;
  const DevLayer* layers;    // device array [L]
  // handle-owned tables and scratch
  const float2* rope;        // [max_seq][half] (cos, sin), computed in fp64 on the host
  // Every vector below is written at most once per launch and read only after
  // its producers' counter; each starts on its own 256-byte boundary (the
  // strides xs, qs, as, ps, in floats), so no cache line holds values of two
  // vectors, which the acquire without a cache invalidation relies on.
  float* x;                  // residual stream [2L + 1][xs]; slot 0 unused (embedding row is read directly)
  float* q;                  // [L][qs] roped queries (nq * hd used)
  float* part;               // [L][ps] records [nkv][nsplit][group][kPartHead + hd]
  float* o;                  // [L][qs] attention output (nq * hd used)
  float* a;                  // [L][as] SwiGLU output (I used)
  int32_t xs, qs, as, ps;
  float* argp;               // [n_lm][2] (max logit, index as float bits)
  int32_t* next_token;       // [1]
  uint32_t* counters;        // [n_counters * kCounterReplicas * kCounterStride]
  int32_t* dev_abort;        // device word: nonzero stops every workgroup at its next wait
  int32_t* host_status;      // host-mapped: first device error code
  const int32_t* host_abort; // host-mapped: raised by amk_set_abort
  // schedule of this launch (one of the handle's variants)
  uint64_t* trace;           // [n_tasks][AMK_TRACE_FIELDS] timestamps, or null
  const amk_task_t* tasks;   // sorted by (cu, seq)
  const int32_t* queue_start;// [n_cu + 1]
  // LDS layout (floats): act[lds_act] stat[2 * part_stride]
  // res[part_stride] part[lds_scr] xsum[lds_act / 32 under W4A16]
  int32_t lds_act;           // activation vector region in floats: a whole number of granules'
                             // elements plus one float4 of padding per 64 floats
  int32_t part_stride;       // rows of one GEMV task at most (partials per streaming wave)
  int32_t lds_scr;           // GEMV partials of all streaming waves, or attention scratch
  int32_t lds_bytes;         // dynamic LDS bytes of one workgroup
};

// Launch the decode-step megakernel (defined in megakernel.hip): `tiny` selects
// the kernel of the tiny-context schedule, which must be the schedule in m.
extern "C" int amk_internal_launch(const DevModel* m, int32_t tiny, int32_t token, int32_t pos, uint32_t epoch,
                                   uint16_t* kv, float* logits, uint64_t timeout_ticks, void* stream);
// Threads per workgroup and LDS the kernel needs beyond the model-dependent regions.
extern "C" int amk_internal_threads(void);
extern "C" int amk_internal_attn_scratch(int group, int head_dim);
extern "C" int amk_internal_prepare(int head_dim, int group, int fmt, int lds_bytes);
extern "C" int amk_internal_occupancy(int head_dim, int group, int fmt, int lds_bytes, int* blocks_per_cu);
extern "C" int amk_internal_read_probe(const void* buf, int64_t bytes, int32_t blocks, uint32_t* sink, void* stream);
// Device address and size of the static scratch array on `device`, which the
// caller has made current (looked up once per device, then cached).
extern "C" int amk_internal_static_scratch(int device, void** ptr, size_t* bytes);

}  // namespace amk
