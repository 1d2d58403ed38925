// One batch-1 Llama decode step as ONE persistent cooperative kernel for
// gfx950 (MI355X): one workgroup per CU walks its host-built task queue
// (paper §3 Algorithm alg:sm) and orders itself against other CUs only
// through monotonic counters (paper §4 "Synchronization model").
//
// Workgroup layout (512 threads = 8 wave64s):
//   wave 0      "sync wave": waits on counters (agent-scope acquire), reduces
//               the streaming waves' partial row sums, applies the fused
//               epilogue (RMSNorm scale, RoPE + KV append, SwiGLU, residual,
//               int8 row scale, argmax), writes every result other CUs read,
//               then releases and signals.
//   waves 1..7  "streaming waves": stream the task's weight rows from HBM in
//               16-byte-per-lane vectors through a double-buffered register
//               pipeline and reduce them against the LDS activation (int4
//               weights: with their fp16 group scales, dequantised in the
//               dot product).
//   all waves   load the task's input activation into LDS after the wait (one
//               round trip), run attention, and run inline continuations.
//
// Per task the workgroup passes four barriers:
//   B1a  the sync wave's counter wait is satisfied (or the launch aborts)
//   B1b  the input activation is in LDS (GEMV tasks)
//   B2   the task's compute is done (partials in LDS / attention stored)
//   B3   the sync wave has stored, released and signalled the task's results
// A task with a chain counter whose signal completed its counter (it is the
// last producer of this launch) then runs that counter's inline task with
// every wave: a KV group's whole attention after its QKV tasks, or the merge
// of a KV group's attention splits.  Each wave drains its own stores, the
// workgroup meets at B4, the sync wave releases and signals the chain
// counter, and B5 keeps the next task's weight loads behind that signal.
// The streaming waves issue the weight loads of their NEXT task right after
// B3 (int4 weights in the tiny-context kernel: right after B2).  Memory
// requests of one CU are served roughly in order, so loads issued before the
// result stores, the release or the counter increment would delay every
// consumer on other CUs; issued after them, the loads stream while the
// counters propagate and the next input is fetched.  The pipeline is kept
// shallow (two halves of Pipe<FMT>::N granules per wave): measured on the
// Llama-3-8B shape, deeper pipelines both delay the sync wave's polls and
// input loads and stream no faster.
//
// Every result another workgroup reads is stored coherent at agent scope
// (write-through past the XCD's L2), so releasing it takes only a drain of
// the storing wave's own stores before the counter increment: no L2
// writeback.  Only the sync wave waits on counters (acquire: agent-scope
// polls, then plain loads with no cache invalidation, see
// acquire_after_poll) and increments them; streaming waves never drain while
// their weight loads are in flight.
// Lane reductions use DPP (VALU latency) rather than LDS permutes.
//
// No MFMA: a batch-1 GEMV is a matrix-vector product, bound by HBM bandwidth.
#include <hip/hip_runtime.h>

#include <cmath>
#include <mutex>

#include "device.h"
#include "schedule.h"

namespace amk {

constexpr int NT = 512;       // threads per workgroup
constexpr int NW = NT / 64;   // waves
constexpr int NSW = NW - 1;   // streaming waves
constexpr int GRAN = 1024;    // bytes per wave-wide 16-B-per-lane load
// Granules per pipeline half, per wave: 4 for bf16 weights, 2 for int8 and
// int4 (their granules hold two and four times the multiply-adds).  Measured
// on the Llama-3-8B shape, deeper pipelines at a task switch delay the sync
// wave's polls and input loads and stream no faster.  EXTRA blocks of N
// granules more are issued once the task's input is in LDS, deepening only
// the steady state: int8 weights stream faster with two (four blocks in
// flight); bf16 and int4 weights, bound by VGPRs and by VALU issue, slower.
template <int FMT> struct Pipe {
  static constexpr int N = FMT == AMK_WEIGHTS_BF16 ? 4 : 2;
  static constexpr int EXTRA = FMT == AMK_WEIGHTS_W8A16 ? 2 : 0;
};
// int4 columns per granule, and per lane (one 16-byte load of 32 nibbles)
constexpr int GRAN4 = 2 * GRAN;
constexpr int LANE4 = 32;

struct Ctl {
  int abort;
  int cont;                     // this task runs its chain counter's inline task
  int res_buf, res_lo, res_hi;  // residual rows cached in LDS: x buffer index and row range
  float ssq[NW];                // per-wave sum of squares of the task input
};

// ---------------------------------------------------------------- memory helpers
// Pointers read out of the model record are generic; casting them to the
// global (1) or constant (4) address space makes the compiler emit global_*
// vector accesses and scalar s_load reads instead of flat accesses, which
// would also count against the LDS wait counter.
#define AMK_GLOBAL __attribute__((address_space(1)))
#define AMK_CONST __attribute__((address_space(4)))
// Raw storage of the same size as T (native vector types copy through any
// address space; HIP's vector structs do not).
template <int N> struct Bits;
template <> struct Bits<2> { typedef unsigned short T; };
template <> struct Bits<4> { typedef unsigned int T; };
template <> struct Bits<8> { typedef unsigned int T __attribute__((ext_vector_type(2))); };
template <> struct Bits<16> { typedef unsigned int T __attribute__((ext_vector_type(4))); };
template <> struct Bits<64> { typedef unsigned int T __attribute__((ext_vector_type(16))); };

template <typename T>
__device__ __forceinline__ T ldg(const void* p) {
  using B = typename Bits<sizeof(T)>::T;
  return __builtin_bit_cast(T, *(const AMK_GLOBAL B*)p);
}
template <typename T>
__device__ __forceinline__ void stg(void* p, const T& v) {
  using B = typename Bits<sizeof(T)>::T;
  *(AMK_GLOBAL B*)p = __builtin_bit_cast(B, v);
}
// Store of a published result: coherent at agent scope (written through the
// XCD's L2), so a producer releases its results by draining its stores
// (s_waitcnt vmcnt(0)) before the counter increment, with no L2 writeback.
__device__ __forceinline__ void stc(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void stc(uint16_t* p, uint16_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void stc(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void stc(float2* p, float2 v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), __builtin_bit_cast(uint64_t, v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

template <typename T>
__device__ __forceinline__ T ldc(const void* p) {
  using B = typename Bits<sizeof(T)>::T;
  return __builtin_bit_cast(T, *(const AMK_CONST B*)p);
}

// ---------------------------------------------------------------- numeric helpers
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) {  // round to nearest even
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float i8f(uint32_t w, int k) { return (float)(int8_t)(w >> (8 * k)); }
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
// Wait until every global load and store this wave issued has completed
// (s_waitcnt vmcnt(0)).  A barrier does not wait for them, so waves that
// store results another CU reads drain before the barrier that precedes the
// sync wave's agent-scope release.
__device__ __forceinline__ void drain_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// DPP lane moves.  Control codes: quad_perm [1,0,3,2] = 0xb1, [2,3,0,1] = 0x4e,
// row_mirror = 0x140, row_half_mirror = 0x141, row_bcast15 = 0x142,
// row_bcast31 = 0x143.  Lanes outside row_mask receive 0.
template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROWS, 0xf, false));
}

// Exchanges with lane ^ 16 and lane ^ 32 through the gfx950 row swaps: with
// both operands v, v_permlane16_swap returns (v[l], v[l ^ 16]) in even rows
// of 16 lanes and (v[l ^ 16], v[l]) in odd rows (v_permlane32_swap likewise
// for halves of 32), so one swap and one VALU op combine the two lanes.
__device__ __forceinline__ float xor16_add(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor16_max(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_add(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor32_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Sum over groups of N consecutive lanes (N in 2, 4, 8, 16, 32); every lane of
// a group receives its group's sum.
template <int N>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(N == 2 || N == 4 || N == 8 || N == 16 || N == 32, "group size");
  v += dpp<0xb1>(v);
  if constexpr (N >= 4) v += dpp<0x4e>(v);
  if constexpr (N >= 8) v += dpp<0x141>(v);
  if constexpr (N >= 16) v += dpp<0x140>(v);
  if constexpr (N >= 32) v = xor16_add(v);
  return v;
}
template <int N>
__device__ __forceinline__ float group_max(float v) {
  v = fmaxf(v, dpp<0xb1>(v));
  if constexpr (N >= 4) v = fmaxf(v, dpp<0x4e>(v));
  if constexpr (N >= 8) v = fmaxf(v, dpp<0x141>(v));
  if constexpr (N >= 16) v = fmaxf(v, dpp<0x140>(v));
  if constexpr (N >= 32) v = xor16_max(v);
  return v;
}

// Sum / max over the lanes l ^ k*G of a wave (G = 8, 16 or 32: the lanes that
// share l mod G), returned to every lane.
template <int G>
__device__ __forceinline__ float across_sum(float v) {
  static_assert(G == 8 || G == 16 || G == 32 || G == 64, "group stride");
  if constexpr (G == 8) v += dpp<0x128>(v);  // row_ror:8 = lane ^ 8 within a row of 16
  if constexpr (G <= 16) v = xor16_add(v);
  if constexpr (G <= 32) v = xor32_add(v);
  return v;
}
template <int G>
__device__ __forceinline__ float across_max(float v) {
  static_assert(G == 8 || G == 16 || G == 32 || G == 64, "group stride");
  if constexpr (G == 8) v = fmaxf(v, dpp<0x128>(v));
  if constexpr (G <= 16) v = xor16_max(v);
  if constexpr (G <= 32) v = xor32_max(v);
  return v;
}

// Full-wave sum / max, returned to every lane.
__device__ __forceinline__ float wave_sum(float v) {
  v = group_sum<16>(v);
  v += dpp<0x142, 0xa>(v);  // rows 1, 3 += last lane of rows 0, 2
  v += dpp<0x143, 0xc>(v);  // rows 2, 3 += lane 31
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
__device__ __forceinline__ float wave_max(float v) {
  v = group_max<16>(v);
  v = xor16_max(v);
  v = xor32_max(v);
  return v;
}

__device__ __forceinline__ bool is_gemv(int op) {
  return op == AMK_OP_QKV || op == AMK_OP_O || op == AMK_OP_GATEUP || op == AMK_OP_DOWN ||
         op == AMK_OP_LMHEAD;
}
__device__ __forceinline__ bool is_normed(int op) {
  return op == AMK_OP_QKV || op == AMK_OP_GATEUP || op == AMK_OP_LMHEAD;
}

// ---------------------------------------------------------------- LDS regions
// The task's input activation act[] is padded: element i sits at
// act_at(i) = i + 4 (i / 64), one unused float4 after every 64 floats.  A
// lane of a GEMV granule reads 8, 16 or 32 consecutive elements (bf16, int8,
// int4 weights) with float4 loads, so lanes start 32, 64 or 128 bytes apart
// and, unpadded, many lanes of one LDS access start in the same bank group
// (measured on the Llama-3-8B shape: int4 weights decode 1.3x slower
// unpadded); the padding staggers them.  A lane's elements stay inside one
// 64-float block, so its loads keep immediate offsets, and a granule's start
// c * E (E a multiple of 64) moves to c * E * 17 / 16.
// After act[]:
//   stat[2 * max_rows]      int8 row scales (rows [0, nj)), then for QKV the
//                           RoPE (cos, sin) of unit u at [nj + 2u, nj + 2u + 1]
//   res[max_rows]           residual rows of the last O / down task (or the
//                           layer-0 embedding rows)
//   part[...]               per-streaming-wave row partials / attention scratch
//   xsum[...]               W4A16: xsum[i] = sum of act[32 i .. 32 i + 31]
__device__ __forceinline__ int act_at(int i) { return i + ((i >> 6) << 2); }
// act_at(c * E + j) for a granule of E elements (a multiple of 64), j < E
template <int E>
__device__ __forceinline__ int act_gran(int c, int j) { return c * (E + E / 16) + act_at(j); }

struct Lds {
  float* act;
  float* stat;
  float* res;
  float* part;
  float* xsum;
};

// ---------------------------------------------------------------- GEMV task geometry
struct Gemv {
  int nj = 0;          // rows (jobs)
  int row_bytes = 0;
  int gpr = 1;         // granules per row
  int int8 = 0;        // int8 weights, fp32 row scales applied in the epilogue
  int q4 = 0;          // int4 weights, fp16 group scales applied per granule
  int tail = 0;        // row_bytes not a multiple of GRAN
  int G = 0;           // total granules = nj * gpr
  int srow = 0;        // int4: scale bytes per row
};

// QKV unit u: head slot u / (d/2) counts KV group by KV group, each group
// holding its query heads, then its K head, then its V head.
__device__ __forceinline__ void unit_head(const DevModel& m, int u, int* mat, int* head) {
  const int slot = u >> m.half_log2;
  const int g = slot / m.gq2;
  const int r = slot - g * m.gq2;
  if (r < m.group) { *mat = W_Q; *head = g * m.group + r; }
  else { *mat = r == m.group ? W_K : W_V; *head = g; }
}

// Which matrix and row job j of task t reads.  mat < 0 means the LM head.
__device__ __forceinline__ void job_row(const DevModel& m, const amk_task_t& t, int j, int* mat, int* row) {
  switch (t.op) {
    case AMK_OP_QKV: {
      const int u = t.begin + (j >> 1);
      int head;
      unit_head(m, u, mat, &head);
      *row = head * m.hd + (u & (m.half - 1)) + (j & 1) * m.half;
      break;
    }
    case AMK_OP_GATEUP: *mat = (j & 1) ? W_U : W_G; *row = t.begin + (j >> 1); break;
    case AMK_OP_O: *mat = W_O; *row = t.begin + j; break;
    case AMK_OP_DOWN: *mat = W_D; *row = t.begin + j; break;
    default: *mat = -1; *row = t.begin + j; break;
  }
}

__device__ __forceinline__ const uint8_t* mat_base(const DevModel& m, const amk_task_t& t, int mat) {
  if (mat < 0) return (const uint8_t*)m.lm_w;
  return (const uint8_t*)ldc<const void*>(&m.layers[t.layer].w[mat]);
}
__device__ __forceinline__ const uint8_t* mat_scale(const DevModel& m, const amk_task_t& t, int mat) {
  if (mat < 0) return (const uint8_t*)m.lm_s;
  return (const uint8_t*)ldc<const void*>(&m.layers[t.layer].s[mat]);
}

__device__ __forceinline__ int task_jobs_dev(const amk_task_t& t) {
  const int n = t.end - t.begin;
  return (t.op == AMK_OP_QKV || t.op == AMK_OP_GATEUP) ? 2 * n : n;
}

__device__ __forceinline__ int task_k(const DevModel& m, const amk_task_t& t) {
  switch (t.op) {
    case AMK_OP_O: return m.nq * m.hd;
    case AMK_OP_DOWN: return m.I;
    default: return m.H;
  }
}

__device__ __forceinline__ Gemv gemv_geom(const DevModel& m, const amk_task_t& t) {
  Gemv g;
  const int K = task_k(m, t);
  const int wf = (t.op == AMK_OP_LMHEAD) ? m.lm_fmt : m.fmt;
  g.int8 = wf == AMK_WEIGHTS_W8A16;
  g.q4 = wf == AMK_WEIGHTS_W4A16;
  g.row_bytes = g.q4 ? K / 2 : g.int8 ? K : 2 * K;
  g.srow = g.q4 ? (K >> m.qglog2) * 2 : 0;
  g.gpr = (g.row_bytes + GRAN - 1) / GRAN;
  g.tail = (g.row_bytes % GRAN) != 0;
  g.nj = task_jobs_dev(t);
  g.G = g.nj * g.gpr;
  return g;
}

// Granule range of streaming wave sw: [sw*G/NSW, (sw+1)*G/NSW).  G * NSW
// stays far below 2^31 (rows per task <= 1024, granules per row <= 64).
__device__ __forceinline__ int wave_gbegin(int G, int sw) { return (G * sw) / NSW; }

struct Cursor {
  int j, c;
  const uint8_t* p;
  const uint8_t* ps;  // W4A16: the row's fp16 group scales (int4 rows), else p
};

template <int FMT>
__device__ __forceinline__ void row_ptr(Cursor& cu, const DevModel& m, const amk_task_t& t, const Gemv& g, int j) {
  int mat, row;
  job_row(m, t, j, &mat, &row);
  cu.p = mat_base(m, t, mat) + (size_t)row * g.row_bytes;
  if constexpr (FMT == AMK_WEIGHTS_W4A16) cu.ps = g.q4 ? mat_scale(m, t, mat) + (size_t)row * g.srow : cu.p;
}

template <int FMT>
__device__ __forceinline__ void cursor_init(Cursor& cu, const DevModel& m, const amk_task_t& t, const Gemv& g,
                                            int gidx) {
  cu.j = gidx / g.gpr;
  cu.c = gidx - cu.j * g.gpr;
  row_ptr<FMT>(cu, m, t, g, cu.j < g.nj ? cu.j : g.nj - 1);
}

template <int FMT>
__device__ __forceinline__ void cursor_next(Cursor& cu, const DevModel& m, const amk_task_t& t, const Gemv& g) {
  if (++cu.c == g.gpr) {
    cu.c = 0;
    ++cu.j;
    if (cu.j < g.nj) row_ptr<FMT>(cu, m, t, g, cu.j);
  }
}

// The weight pipeline issues every load unconditionally, so the compiler can
// count outstanding loads exactly and wait for just the oldest one (a load
// under a branch forces it to drain the whole pipeline).  Lanes past the end
// of a short row, and granules past the end of the wave's range, re-read a
// valid address of the current row; consume_block() never uses them (rows)
// or zeroes them (tail lanes).
__device__ __forceinline__ uint4 load_gran(const Cursor& cu, const Gemv& g, int lane) {
  int off = cu.c * GRAN + lane * 16;
  if (g.tail && off >= g.row_bytes) off = 0;
  return ldg<uint4>(cu.p + off);
}

// The fp16 scale of the lane's 32 int4 columns (one group holds whole
// lanes); tail lanes and rows of other formats re-read a valid address.
__device__ __forceinline__ uint32_t load_scale4(const Cursor& cu, const DevModel& m, const Gemv& g, int lane) {
  int idx = (cu.c * GRAN4 + lane * LANE4) >> m.qglog2;
  if (!g.q4 || (g.tail && cu.c * GRAN + lane * 16 >= g.row_bytes)) idx = 0;
  return ldg<uint16_t>(cu.ps + 2 * idx);
}

// Issue N granules starting at global granule index gi (clipped to g1); under
// W4A16 also each granule's per-lane group scale.
template <int FMT, int N>
__device__ __forceinline__ void issue_block(uint4 (&buf)[N], uint32_t (&sc)[N], Cursor& cu, int& gi, int g1,
                                            const DevModel& m, const amk_task_t& t, const Gemv& g, int lane) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    buf[i] = load_gran(cu, g, lane);
    if constexpr (FMT == AMK_WEIGHTS_W4A16) sc[i] = load_scale4(cu, m, g, lane);
    if (gi < g1) cursor_next<FMT>(cu, m, t, g);
    ++gi;
  }
}

__device__ __forceinline__ float dot_gran(const uint4 v, const float* __restrict__ act, int c, int lane, int int8,
                                          float acc) {
  if (!int8) {
    const float* x = act + act_gran<GRAN / 2>(c, lane * 8);
    const float4 a = *reinterpret_cast<const float4*>(x);
    const float4 b = *reinterpret_cast<const float4*>(x + 4);
    acc = fmaf(bf_lo(v.x), a.x, acc); acc = fmaf(bf_hi(v.x), a.y, acc);
    acc = fmaf(bf_lo(v.y), a.z, acc); acc = fmaf(bf_hi(v.y), a.w, acc);
    acc = fmaf(bf_lo(v.z), b.x, acc); acc = fmaf(bf_hi(v.z), b.y, acc);
    acc = fmaf(bf_lo(v.w), b.z, acc); acc = fmaf(bf_hi(v.w), b.w, acc);
  } else {
    const float* x = act + act_gran<GRAN>(c, lane * 16);
    const float4 a = *reinterpret_cast<const float4*>(x);
    const float4 b = *reinterpret_cast<const float4*>(x + 4);
    const float4 d = *reinterpret_cast<const float4*>(x + 8);
    const float4 e = *reinterpret_cast<const float4*>(x + 12);
    acc = fmaf(i8f(v.x, 0), a.x, acc); acc = fmaf(i8f(v.x, 1), a.y, acc);
    acc = fmaf(i8f(v.x, 2), a.z, acc); acc = fmaf(i8f(v.x, 3), a.w, acc);
    acc = fmaf(i8f(v.y, 0), b.x, acc); acc = fmaf(i8f(v.y, 1), b.y, acc);
    acc = fmaf(i8f(v.y, 2), b.z, acc); acc = fmaf(i8f(v.y, 3), b.w, acc);
    acc = fmaf(i8f(v.z, 0), d.x, acc); acc = fmaf(i8f(v.z, 1), d.y, acc);
    acc = fmaf(i8f(v.z, 2), d.z, acc); acc = fmaf(i8f(v.z, 3), d.w, acc);
    acc = fmaf(i8f(v.w, 0), e.x, acc); acc = fmaf(i8f(v.w, 1), e.y, acc);
    acc = fmaf(i8f(v.w, 2), e.z, acc); acc = fmaf(i8f(v.w, 3), e.w, acc);
  }
  return acc;
}

// One int4 granule: the lane's 32 columns [c * 2048 + 32 lane, + 32) of one
// row, times their group scale s.  Word d of the lane's 16 bytes holds
// columns 8d .. 8d + 3 in its low nibbles and 8d + 4 .. 8d + 7 in its high
// nibbles, as unsigned code + 8.  Masked (and the high ones shifted down)
// into the low nibble of each byte, a byte n read as an FP8 E4M3 value
// (exponent field 0 or 1, bias 7) is exactly n * 2^-9, so one
// v_cvt_pk_f32_fp8 turns two nibbles into floats.  Every product and partial
// sum then carries the exact factor 2^-9, which rounding commutes with, so
// the sum equals the plain fp32 one bit for bit once the factor is taken
// out.  The zero point leaves sum (code + 8) x - 8 sum x, with sum x over the
// 32 columns precomputed.
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot_gran4(const uint4 v, uint32_t sbits, const float* __restrict__ act,
                                           const float* __restrict__ xsum, int c, int lane, bool valid, float acc) {
  const float* x = act + act_gran<GRAN4>(c, lane * LANE4);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  // all 32 activations and their sum are read before any product, so the
  // LDS latency is paid once per granule
  float4 xv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) xv[i] = *reinterpret_cast<const float4*>(x + 4 * i);
  const float xs = xsum[c * (GRAN4 / LANE4) + lane];
  float lo = 0.f, hi = 0.f;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const float4 a = xv[2 * d], b = xv[2 * d + 1];
    const int l = (int)(w[d] & 0x0f0f0f0fu), h = (int)((w[d] >> 4) & 0x0f0f0f0fu);
    const f32x2 l01 = __builtin_amdgcn_cvt_pk_f32_fp8(l, false), l23 = __builtin_amdgcn_cvt_pk_f32_fp8(l, true);
    const f32x2 h01 = __builtin_amdgcn_cvt_pk_f32_fp8(h, false), h23 = __builtin_amdgcn_cvt_pk_f32_fp8(h, true);
    lo = fmaf(l01.x, a.x, lo); lo = fmaf(l01.y, a.y, lo);
    lo = fmaf(l23.x, a.z, lo); lo = fmaf(l23.y, a.w, lo);
    hi = fmaf(h01.x, b.x, hi); hi = fmaf(h01.y, b.y, hi);
    hi = fmaf(h23.x, b.z, hi); hi = fmaf(h23.y, b.w, hi);
  }
  const float u = (lo + hi) * 512.f;                             // sum of (code + 8) x
  const float p = fmaf(-8.f, xs, u);                             // sum of code x
  const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)sbits);
  return valid ? fmaf(s, p, acc) : acc;
}

// Consume N granules; a finished row's wave-reduced partial goes to part[j].
template <int FMT, int N>
__device__ __forceinline__ void consume_block(const uint4 (&buf)[N], const uint32_t (&sc)[N], int& j, int& c, int& gi,
                                              int g1, float& acc, const Lds& L, float* __restrict__ part,
                                              const Gemv& g, int lane) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if (gi < g1) {
      if (FMT == AMK_WEIGHTS_W4A16 && g.q4) {
        const bool valid = !g.tail || c * GRAN + lane * 16 < g.row_bytes;
        acc = dot_gran4(buf[i], sc[i], L.act, L.xsum, c, lane, valid, acc);
      } else {
        uint4 v = buf[i];
        if (g.tail && c * GRAN + lane * 16 >= g.row_bytes) v = make_uint4(0, 0, 0, 0);
        acc = dot_gran(v, L.act, c, lane, g.int8, acc);
      }
      if (++c == g.gpr) {
        const float s = wave_sum(acc);
        if (lane == 0) part[j] = s;
        acc = 0.f;
        c = 0;
        ++j;
      }
    }
    ++gi;
  }
}

// ---------------------------------------------------------------- sync wave: counters
// Acquire after a counter poll.  The polls are agent-coherent loads; what they
// order is then read with plain loads, with no cache invalidation:
//  - every vector another workgroup reads (residual stream, q, attention
//    records and output, SwiGLU output, argmax partials, the KV row at pos) is
//    written at most once per launch, and read only after all its producers
//    signalled;
//  - the launch's own acquire has invalidated every cached copy of earlier
//    launches' data;
//  - no cache line holds parts of two such vectors (256-byte strides).
// Producers' row ranges are not line-aligned: several producers, often on
// different XCDs, write parts of one 128-byte line.  This relies on the L2
// keeping written-through bytes with a byte mask: a store does not make the
// rest of its line valid, so a later read of the line by a CU of that XCD
// fetches the other producers' bytes from memory.  (The SmolLM2-shaped
// decoder, whose residual tasks own 2 or 3 rows, puts up to 16 producers in
// one line and decodes 32 greedy steps in agreement with the oracle.)
// So a line a workgroup finds in its L1 or its XCD's L2 was fetched after the
// producers had released all of it, and the XCD's L2 serves one fetch of an
// input vector to all its CUs instead of one per CU.  The fence only keeps
// the compiler from moving those loads above the poll; the hardware issues
// them after it, since leaving the poll loop depends on the loaded value.
__device__ __forceinline__ void acquire_after_poll() { __atomic_signal_fence(__ATOMIC_SEQ_CST); }

// How a wait polls.  bf16 weights: two polls in flight (the older one is
// checked while the newer travels, which halves the time from an increment
// to its observation), the abort words every 8 spins.  W8A16: one poll and
// one abort-word load per spin, which measured faster there (its shorter,
// latency-bound streaming phases suffer from the extra poll traffic).
template <int FMT> struct Polls { static constexpr bool TWO = FMT == AMK_WEIGHTS_BF16; };

template <int FMT>
__device__ __forceinline__ bool wait_deps(const DevModel& m, const amk_task_t& t, const amk_task_t* tp, uint32_t epoch,
                                          uint64_t deadline, int lane, uint64_t* tr) {
  const int nw = t.n_wait;
  if (nw == 0) return __hip_atomic_load(m.dev_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0;
  // lanes past n_wait poll the first counter too and never block: the loads
  // are unconditional, so the compiler counts them exactly
  const int wl = lane < nw ? lane : 0;
  const uint32_t* p = m.counters + ((size_t)ldg<int32_t>(&tp->wait_counter[wl]) * kCounterReplicas +
                                    blockIdx.x % kCounterReplicas) * kCounterStride;
  const uint32_t target = epoch * (uint32_t)ldg<int32_t>(&tp->wait_count[wl]);
  uint32_t spins = 0;
  uint32_t v_old = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (;;) {
    uint32_t v_new = 0;
    if constexpr (Polls<FMT>::TWO) {
      __builtin_amdgcn_s_sleep(1);
      v_new = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const uint64_t now = wall_clock64();
    if (__all(lane >= nw || (int32_t)(v_old - target) >= 0)) break;
    ++spins;
    int code = 0;
    if (Polls<FMT>::TWO ? (spins & 7u) == 0 : true) {
      if (__hip_atomic_load(m.dev_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return false;
    }
    // host-mapped flag: read over the bus, so only every 64 spins
    if ((spins & 63u) == 0 && __hip_atomic_load(m.host_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM))
      code = AMK_ERR_ABORTED;
    else if (now > deadline)
      code = AMK_ERR_TIMEOUT;
    if (code) {
      if (lane == 0) {
        // plain stores (no read-modify-write over the bus); if two
        // workgroups stop at once, either code is a valid report
        __hip_atomic_store(m.host_status, code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        __hip_atomic_store(m.dev_abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      return false;
    }
    if constexpr (Polls<FMT>::TWO) {
      v_old = v_new;
    } else {
      __builtin_amdgcn_s_sleep(1);
      v_old = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if (tr && lane == 0) stg<uint64_t>(tr + AMK_TRACE_SATISFIED, (uint64_t)wall_clock64());
  acquire_after_poll();
  return true;
}

__device__ __forceinline__ void release_signal(const DevModel& m, int counter, int lane) {
  drain_vmem();  // every published store of this wave is coherent at agent scope
  if (lane < kCounterReplicas && counter >= 0)
    __hip_atomic_fetch_add(m.counters + ((size_t)counter * kCounterReplicas + lane) * kCounterStride, 1u,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Release, increment `counter`, and report whether this increment brought it
// to `target` (the last producer of this launch).  The caller that gets true
// acquires before reading what the other producers released.
__device__ __forceinline__ bool release_signal_last(const DevModel& m, int counter, uint32_t target, int lane) {
  drain_vmem();
  uint32_t old = 0;
  // copy 0's return value orders the producers
  if (lane < kCounterReplicas)
    old = __hip_atomic_fetch_add(m.counters + ((size_t)counter * kCounterReplicas + lane) * kCounterStride, 1u,
                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  old = (uint32_t)__builtin_amdgcn_readfirstlane((int)old);
  return (int32_t)(old + 1u - target) == 0;
}

// ---------------------------------------------------------------- per-row static data
// Data of a GEMV task that does not depend on this launch's results and is
// needed only in its epilogue (int8 row scales, RoPE factors, the layer-0
// embedding rows of the residual) is fetched by the sync wave while the
// streaming waves compute.

__device__ __forceinline__ void load_rowdata(const DevModel& m, const amk_task_t& t, int token, int pos,
                                             const Lds& L, Ctl& ctl, int lane) {
  const int op = t.op;
  const Gemv g = gemv_geom(m, t);
  if (g.int8) {
    for (int j = lane; j < g.nj; j += 64) {
      int mat, row;
      job_row(m, t, j, &mat, &row);
      L.stat[j] = ldg<float>(mat_scale(m, t, mat) + 4 * (size_t)row);
    }
  }
  if (op == AMK_OP_QKV) {
    const int nu = t.end - t.begin;
    for (int u = lane; u < nu; u += 64) {
      const int i = (t.begin + u) & (m.half - 1);
      const float2 cs = ldg<float2>(m.rope + (size_t)pos * m.half + i);
      L.stat[g.nj + 2 * u] = cs.x;
      L.stat[g.nj + 2 * u + 1] = cs.y;
    }
  }
  if (op == AMK_OP_O && t.layer == 0) {
    const uint16_t* e = m.embed + (size_t)token * m.H;
    for (int r = t.begin + lane; r < t.end; r += 64) L.res[r - t.begin] = bf16f(ldg<uint16_t>(e + r));
    if (lane == 0) {
      ctl.res_buf = 0;
      ctl.res_lo = t.begin;
      ctl.res_hi = t.end;
    }
  }
}

// ---------------------------------------------------------------- input activation (all waves)
// The task input moves into LDS in one round trip: wave w copies a 1/8 slice.
// Normed inputs load the RMSNorm gain in the same round trip, store x * gain
// and leave each wave's sum of x^2 in ctl.ssq; the GEMV result is scaled by
// 1/sqrt(mean(x^2) + eps) in the epilogue (RMSNorm folded into the consumer).
// Under W4A16 the slices are whole 32-column blocks and each block's sum of
// the stored values goes to xsum (8 lanes hold one block).
template <int FMT>
__device__ __forceinline__ void load_input(const DevModel& m, const amk_task_t& t, int token, const Lds& L, Ctl& ctl,
                                           int wave, int lane) {
  const int op = t.op;
  const float* src = nullptr;
  const uint16_t* src_bf = nullptr;
  const uint16_t* gain = nullptr;
  switch (op) {
    case AMK_OP_QKV:
      if (t.layer == 0) src_bf = m.embed + (size_t)token * m.H;
      else src = m.x + (size_t)(2 * t.layer) * m.xs;
      gain = ldc<const uint16_t*>(&m.layers[t.layer].attn_norm);
      break;
    case AMK_OP_GATEUP:
      src = m.x + (size_t)(2 * t.layer + 1) * m.xs;
      gain = ldc<const uint16_t*>(&m.layers[t.layer].mlp_norm);
      break;
    case AMK_OP_LMHEAD: src = m.x + (size_t)(2 * m.L) * m.xs; gain = m.final_norm; break;
    case AMK_OP_O: src = m.o + (size_t)t.layer * m.qs; break;
    case AMK_OP_DOWN: src = m.a + (size_t)t.layer * m.as; break;
    default: return;
  }
  const int K = task_k(m, t);
  const int n4 = K >> 2;  // float4 vectors (K is a multiple of 16; of 32 under W4A16)
  constexpr int AL = FMT == AMK_WEIGHTS_W4A16 ? 8 : 1;
  const int v0 = (n4 / AL * wave) / NW * AL, v1 = (n4 / AL * (wave + 1)) / NW * AL;
  float ss = 0.f;
  constexpr int NB = 8;
  for (int b = v0; b < v1; b += NB * 64) {
    float4 xv[NB];
    uint2 gv[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int v = b + i * 64 + lane;
      if (v < v1) {
        if (src_bf) {
          const uint2 r = ldg<uint2>(src_bf + (size_t)v * 4);
          xv[i] = make_float4(bf_lo(r.x), bf_hi(r.x), bf_lo(r.y), bf_hi(r.y));
        } else {
          xv[i] = ldg<float4>(src + (size_t)v * 4);
        }
        if (gain) gv[i] = ldg<uint2>(gain + (size_t)v * 4);
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int v = b + i * 64 + lane;
      float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
      if (v < v1) {
        x = xv[i];
        if (gain) {
          ss = fmaf(x.x, x.x, ss); ss = fmaf(x.y, x.y, ss); ss = fmaf(x.z, x.z, ss); ss = fmaf(x.w, x.w, ss);
          x = make_float4(x.x * bf_lo(gv[i].x), x.y * bf_hi(gv[i].x), x.z * bf_lo(gv[i].y), x.w * bf_hi(gv[i].y));
        }
        *reinterpret_cast<float4*>(L.act + act_at(v * 4)) = x;
      }
      if constexpr (FMT == AMK_WEIGHTS_W4A16) {
        // v0 and b are multiples of 8: lanes 8k .. 8k + 7 hold one block,
        // all in range or all out
        const float blk = group_sum<8>((x.x + x.y) + (x.z + x.w));
        if (v < v1 && (lane & 7) == 0) L.xsum[v >> 3] = blk;
      }
    }
  }
  if (gain) {
    ss = wave_sum(ss);
    if (lane == 0) ctl.ssq[wave] = ss;
  }
}

__device__ __forceinline__ float input_rs(const DevModel& m, const Ctl& ctl) {
  float ss = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) ss += ctl.ssq[w];
  return 1.0f / sqrtf(ss / (float)m.H + m.eps);
}

// ---------------------------------------------------------------- row sums of a GEMV task
// Granule boundaries of the streaming waves, computed once per epilogue.
struct Ranges {
  int b[NSW + 1];
};
__device__ __forceinline__ Ranges wave_ranges(const Gemv& g) {
  Ranges r;
#pragma unroll
  for (int sw = 0; sw <= NSW; ++sw) r.b[sw] = wave_gbegin(g.G, sw);
  return r;
}

__device__ __forceinline__ float row_sum(const float* part, int stride, const Gemv& g, const Ranges& wr, int j) {
  const int lo = j * g.gpr, hi = lo + g.gpr;
  // every wave's slot is read (all reads in flight at once), the ones of
  // waves that wrote nothing for row j are dropped: a wave with an empty
  // range wrote nothing, even if its start lies inside the row
  float v[NSW];
#pragma unroll
  for (int sw = 0; sw < NSW; ++sw) v[sw] = part[sw * stride + j];
  float s = 0.f;
#pragma unroll
  for (int sw = 0; sw < NSW; ++sw) {
    const int gb = wr.b[sw], ge = wr.b[sw + 1];
    s += (gb < ge && gb < hi && ge > lo) ? v[sw] : 0.f;
  }
  return s;
}

// ---------------------------------------------------------------- sync wave: epilogues
__device__ __forceinline__ void epi_qkv(const DevModel& m, const amk_task_t& t, const Gemv& g, const Lds& L, int pos,
                                        uint16_t* kv, float rs, int lane) {
  const int l = t.layer;
  const Ranges wr = wave_ranges(g);
  for (int u = t.begin + lane; u < t.end; u += 64) {
    const int j0 = 2 * (u - t.begin);
    float y0 = row_sum(L.part, m.part_stride, g, wr, j0) * rs;
    float y1 = row_sum(L.part, m.part_stride, g, wr, j0 + 1) * rs;
    if (g.int8) {
      y0 *= L.stat[j0];
      y1 *= L.stat[j0 + 1];
    }
    int mat, head;
    unit_head(m, u, &mat, &head);
    const int i = u & (m.half - 1);
    if (mat != W_V) {
      const float c = L.stat[g.nj + 2 * (u - t.begin)], s = L.stat[g.nj + 2 * (u - t.begin) + 1];
      const float a = y0 * c - y1 * s;
      const float b = y1 * c + y0 * s;
      y0 = a;
      y1 = b;
    }
    if (mat == W_Q) {
      float* qd = m.q + (size_t)l * m.qs + (size_t)head * m.hd;
      stc(qd + i, y0);
      stc(qd + i + m.half, y1);
    } else {
      const int which = (mat == W_K) ? 0 : 1;
      uint16_t* dst = kv + (((size_t)(l * 2 + which) * m.nkv + head) * m.max_seq + pos) * m.hd;
      stc(dst + i, f2bf(y0));
      stc(dst + i + m.half, f2bf(y1));
    }
  }
}

// O and down projections: x_out = x_in + W y, with x_in rows taken from LDS
// when this workgroup's previous residual task produced exactly those rows.
__device__ __forceinline__ void epi_residual(const DevModel& m, const amk_task_t& t, const Gemv& g, const Lds& L,
                                             Ctl& ctl, int lane) {
  const int xin = t.op == AMK_OP_O ? 2 * t.layer : 2 * t.layer + 1;
  const bool cached = ctl.res_buf == xin && ctl.res_lo == t.begin && ctl.res_hi == t.end;
  const Ranges wr = wave_ranges(g);
  for (int r = t.begin + lane; r < t.end; r += 64) {
    float y = row_sum(L.part, m.part_stride, g, wr, r - t.begin);
    if (g.int8) y *= L.stat[r - t.begin];
    const float x = cached ? L.res[r - t.begin] : ldg<float>(m.x + (size_t)xin * m.xs + r);
    const float o = x + y;
    stc(m.x + (size_t)(xin + 1) * m.xs + r, o);
    L.res[r - t.begin] = o;
  }
  if (lane == 0) {
    ctl.res_buf = xin + 1;
    ctl.res_lo = t.begin;
    ctl.res_hi = t.end;
  }
}

__device__ __forceinline__ void epi_gateup(const DevModel& m, const amk_task_t& t, const Gemv& g, const Lds& L,
                                           float rs, int lane) {
  const Ranges wr = wave_ranges(g);
  for (int r = t.begin + lane; r < t.end; r += 64) {
    const int j = 2 * (r - t.begin);
    float gv = row_sum(L.part, m.part_stride, g, wr, j) * rs;
    float uv = row_sum(L.part, m.part_stride, g, wr, j + 1) * rs;
    if (g.int8) {
      gv *= L.stat[j];
      uv *= L.stat[j + 1];
    }
    const float silu = gv / (1.0f + __expf(-gv));
    stc(m.a + (size_t)t.layer * m.as + r, silu * uv);
  }
}

// LM head: logits + per-task argmax partial (lowest index on ties).  A NaN
// logit never wins a comparison; it records the sticky status
// AMK_ERR_NONFINITE, so the step's next token is reported as meaningless
// instead of silently skipping it.
__device__ __forceinline__ void epi_lmhead(const DevModel& m, const amk_task_t& t, const Gemv& g, const Lds& L,
                                           float rs, float* logits, int lane) {
  float best = -INFINITY;
  int besti = 0x7fffffff;
  bool nan = false;
  const Ranges wr = wave_ranges(g);
  for (int r = t.begin + lane; r < t.end; r += 64) {
    float y = row_sum(L.part, m.part_stride, g, wr, r - t.begin) * rs;
    if (g.int8) y *= L.stat[r - t.begin];
    stc(logits + r, y);
    nan |= y != y;
    if (y > best || (y == best && r < besti)) { best = y; besti = r; }
  }
  if (__any(nan) && lane == 0)
    __hip_atomic_store(m.host_status, (int32_t)AMK_ERR_NONFINITE, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o);
    const int oi = __shfl_xor(besti, o);
    if (ob > best || (ob == best && oi < besti)) { best = ob; besti = oi; }
  }
  if (lane == 0) stc(reinterpret_cast<float2*>(m.argp + 2 * t.aux), make_float2(best, __int_as_float(besti)));
}

__device__ __forceinline__ void argmax_final(const DevModel& m, const amk_task_t& t, int lane) {
  float best = -INFINITY;
  int besti = 0x7fffffff;
  for (int s = t.begin + lane; s < t.end; s += 64) {
    const float2 vi = ldg<float2>(m.argp + 2 * s);
    const int i = __float_as_int(vi.y);
    if (vi.x > best || (vi.x == best && i < besti)) { best = vi.x; besti = i; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o);
    const int oi = __shfl_xor(besti, o);
    if (ob > best || (ob == best && oi < besti)) { best = ob; besti = oi; }
  }
  if (lane == 0) stc(m.next_token, besti);
}

// ---------------------------------------------------------------- attention (all 8 waves)
// Geometry of the attention of one KV group, shared with the host's LDS
// sizing.  HD: head dim; GM: largest query group handled; EPL: head dims per
// lane (8 for groups <= 4, 4 for groups <= 8 to halve the accumulators); LPR
// lanes cover one K/V row, RPW rows per wave-wide load; each lane holds KB K
// rows and KB V rows per pass, so a pass of the workgroup covers RP rows with
// all its loads in flight at once.
template <int HD, int GM>
struct AttnGeom {
  static constexpr int EPL = GM <= 4 ? 8 : 4;
  static constexpr int LPR = HD / EPL;
  static constexpr int RPW = 64 / LPR;
  static constexpr int KB = 9;
  static constexpr int SB = 3;  // most rows per lane per softmax update
  static constexpr int RP = NW * RPW * KB;
  // LDS scratch (floats): per-wave accumulators red[NW][GM][HD] and running
  // (max, sum) stat[NW][GM][2]; the split merge reuses the region
  static constexpr int SCRATCH = NW * GM * HD + 2 * NW * GM;
  static constexpr int MERGE = GM * 64 + 4 * NT;
  static constexpr int LDS = SCRATCH > MERGE ? SCRATCH : MERGE;
  static_assert(LPR >= 2 && LPR <= 32, "lanes per row");
};

template <int EPL> struct RowVec;
template <> struct RowVec<8> { uint4 v; };
template <> struct RowVec<4> { uint2 v; };

template <int EPL>
__device__ __forceinline__ RowVec<EPL> load_row(const uint16_t* p) {
  RowVec<EPL> r;
  if constexpr (EPL == 8) r.v = ldg<uint4>(p); else r.v = ldg<uint2>(p);
  return r;
}
template <int EPL>
__device__ __forceinline__ float row_elem(const RowVec<EPL>& r, int e) {
  uint32_t w;
  if constexpr (EPL == 8) w = (e < 2) ? r.v.x : (e < 4) ? r.v.y : (e < 6) ? r.v.z : r.v.w;
  else w = (e < 2) ? r.v.x : r.v.y;
  return (e & 1) ? bf_hi(w) : bf_lo(w);
}

// Attention of the query heads of KV group g over positions [j0, j1) of
// layer `layer` (j1 > j0), scores q.k / sqrt(d), max-subtracted softmax,
// V-weighted sum (paper §2 "Kernel authoring and attention" names the
// flash-decoding family this follows).  Every wave keeps its own running
// max / sum / accumulators over the rows it loads (online softmax, no
// barrier inside the position loop); the waves merge through LDS at the end.
// The queries are stored pre-multiplied by log2(e) / sqrt(d), so scores and
// maxima are in log2 units and each softmax weight is one exp2: the same
// weights as exp(q.k / sqrt(d) - max), up to fp32 rounding.
// `record`: store per head (m, l, unnormalised acc) at dst[h * (kPartHead +
// d)], else the normalised output at dst[h * d].  Stores are issued by every
// wave; the caller drains them.
template <int HD, int GM>
__device__ __forceinline__ void attention(const DevModel& m, int layer, int g, int j0, int j1,
                                          const uint16_t* __restrict__ kv, float* __restrict__ qs,
                                          float* __restrict__ scr, float* __restrict__ dst, bool record, int wave,
                                          int lane) {
  using A = AttnGeom<HD, GM>;
  constexpr int EPL = A::EPL, LPR = A::LPR, RPW = A::RPW, KB = A::KB, SB = A::SB, RP = A::RP;
  static_assert(KB == 9 && SB == 3, "sub-batches of 3, 3, 2 and 1 row slots");
  const int G = m.group;
  const int n = j1 - j0;
  const int sub = lane / LPR, c = lane % LPR;
  const size_t hs = (size_t)m.max_seq * HD;
  const uint16_t* Kp = kv + ((size_t)(layer * 2 + 0) * m.nkv + g) * hs + (size_t)j0 * HD + c * EPL;
  const uint16_t* Vp = kv + ((size_t)(layer * 2 + 1) * m.nkv + g) * hs + (size_t)j0 * HD + c * EPL;

  float m_run[GM], l_run[GM], acc[GM][EPL];
#pragma unroll
  for (int h = 0; h < GM; ++h) {
    m_run[h] = -INFINITY;
    l_run[h] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[h][e] = 0.f;
  }

  // the group's roped queries (G * HD / 4 <= NT float4s) into LDS first: the
  // threads that move them do so before issuing their rows, so the queries
  // do not wait behind the K / V stream
  static_assert(GM * HD / 4 <= NT, "one query vector per thread");
  if ((int)threadIdx.x < G * HD / 4) {
    const float* qsrc = m.q + (size_t)layer * m.qs + (size_t)g * G * HD;
    const float c = m.attn_scale * 1.4426950408889634f;  // log2(e) / sqrt(d)
    float4 qv = ldg<float4>(qsrc + 4 * threadIdx.x);
    qv.x *= c; qv.y *= c; qv.z *= c; qv.w *= c;
    *reinterpret_cast<float4*>(qs + 4 * threadIdx.x) = qv;
  }
  for (int p0 = 0; p0 < n; p0 += RP) {
    // rows of this lane: r_k = p0 + (k * NW + wave) * RPW + sub.  Every load
    // is issued (rows past the range re-read its first row, whose score is
    // masked to -inf, so it weighs 0): the compiler then waits for each row
    // alone instead of the whole batch.
    RowVec<EPL> kr[KB], vr[KB];
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      const int r = p0 + (k * NW + wave) * RPW + sub;
      if (r < n) {
        kr[k] = load_row<EPL>(Kp + (size_t)r * HD);
        vr[k] = load_row<EPL>(Vp + (size_t)r * HD);
      } else {
        kr[k] = load_row<EPL>(Kp);
        vr[k] = load_row<EPL>(Vp);
      }
    }
    if (p0 == 0) __syncthreads();
    // rows in sub-batches of 3, 3, 2 and 1 slots: scores for every query
    // head, then one online-softmax update per head and sub-batch.  A wave
    // whose range ends after 8 slots skips the last one instead of scoring a
    // fully masked slot.  The running max / sum
    // belong to the lane's row group (LPR lanes sharing its rows), so no
    // cross-lane maximum is needed inside the loop.
#pragma unroll
    for (int sb = 0; sb < 4; ++sb) {
      const int kb = sb == 0 ? 0 : sb == 1 ? 3 : sb == 2 ? 6 : 8;
      const int NB = sb < 2 ? 3 : sb == 2 ? 2 : 1;
      if (p0 + (kb * NW + wave) * RPW >= n) break;  // no row of this wave from here on
      float sc[GM][SB];
      // per query head: its LDS values once, then the scores of the SB rows
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        if (h < G) {
          float q[EPL];
#pragma unroll
          for (int e = 0; e < EPL; e += 4) {
            const float4 q4 = *reinterpret_cast<const float4*>(qs + h * HD + c * EPL + e);
            q[e] = q4.x; q[e + 1] = q4.y; q[e + 2] = q4.z; q[e + 3] = q4.w;
          }
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            const int k = kb + j;
            const int r = p0 + (k * NW + wave) * RPW + sub;
            float d = 0.f;
#pragma unroll
            for (int e = 0; e < EPL; ++e) d = fmaf(row_elem<EPL>(kr[k], e), q[e], d);
            d = group_sum<LPR>(d);
            sc[h][j] = r < n ? d : -INFINITY;
          }
        }
      }
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        if (h < G) {
          float mx = sc[h][0];
#pragma unroll
          for (int j = 1; j < NB; ++j) mx = fmaxf(mx, sc[h][j]);
          const float m_new = fmaxf(m_run[h], mx);
          // a row group that has seen no row keeps (-inf, 0, 0)
          const float mref = m_new == -INFINITY ? 0.f : m_new;
          const float alpha = __builtin_amdgcn_exp2f(m_run[h] - mref);
          float ls = 0.f;
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            sc[h][j] = __builtin_amdgcn_exp2f(sc[h][j] - mref);
            ls += sc[h][j];
          }
          l_run[h] = l_run[h] * alpha + ls;
          m_run[h] = m_new;
#pragma unroll
          for (int e = 0; e < EPL; ++e) acc[h][e] *= alpha;
        }
      }
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        float vf[EPL];
#pragma unroll
        for (int e = 0; e < EPL; ++e) vf[e] = row_elem<EPL>(vr[kb + j], e);
#pragma unroll
        for (int h = 0; h < GM; ++h) {
          if (h < G) {
#pragma unroll
            for (int e = 0; e < EPL; ++e) acc[h][e] = fmaf(sc[h][j], vf[e], acc[h][e]);
          }
        }
      }
    }
  }

  // per wave: sum the accumulators of its row groups; then merge the waves
  float* red = scr;                   // [NW][GM][HD]
  float* stat = scr + NW * GM * HD;   // [NW][GM][2]
#pragma unroll
  for (int h = 0; h < GM; ++h) {
    if (h < G) {
      // merge the row groups of the wave: rescale each to the wave's max
      const float M = across_max<LPR>(m_run[h]);
      const float f = m_run[h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run[h] - M);
      const float l = across_sum<LPR>(l_run[h] * f);
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const float v = across_sum<LPR>(acc[h][e] * f);
        if (sub == 0) red[(wave * GM + h) * HD + c * EPL + e] = v;
      }
      if (lane == 0) {
        stat[(wave * GM + h) * 2] = M;
        stat[(wave * GM + h) * 2 + 1] = l;
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < G * HD; i += NT) {
    const int h = i / HD, d = i - h * HD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, stat[(w * GM + h) * 2]);
    float l = 0.f, o = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = stat[(w * GM + h) * 2];
      if (mw != -INFINITY) {
        const float f = __builtin_amdgcn_exp2f(mw - M);
        l = fmaf(f, stat[(w * GM + h) * 2 + 1], l);
        o = fmaf(f, red[(w * GM + h) * HD + d], o);
      }
    }
    if (record) {
      float* rec = dst + h * (kPartHead + HD);
      stc(rec + kPartHead + d, o);
      // the record's maximum in natural-log units, as the split merge reads it
      if (d == 0) stc(reinterpret_cast<float2*>(rec), make_float2(M * 0.6931471805599453f, l));
    } else {
      stc(dst + h * HD + d, o / l);
    }
  }
}

// Attention of every query head over positions [0, pos] (pos < AMK_TINY_MAX)
// into act[h * HD + d]: the input of an O task of the tiny schedule, which
// computes it itself instead of waiting for an attention stage.  Each wave
// takes HR heads per round; lane owns head dims [lane * DPL, (lane + 1) * DPL).
// All q / K / V loads of a round go out before any arithmetic, once per KV
// group; positions past pos re-read row pos (clamped, unused).
template <int HD, int FMT>
__device__ __forceinline__ void attention_all(const DevModel& m, int layer, int pos, const uint16_t* __restrict__ kv,
                                              float* __restrict__ act, float* __restrict__ xsum, int wave,
                                              int lane) {
  constexpr int DPL = HD / 64;
  constexpr int HR = 4;
  constexpr int T = AMK_TINY_MAX;
  const int n = pos + 1;
  const size_t hs = (size_t)m.max_seq * HD;
  // the HR heads of a round share one KV group when the group size is a
  // multiple of HR (heads h0.. h0 + HR - 1 with h0 a multiple of HR)
  const bool one_group = m.group % HR == 0;
  for (int h0 = wave * HR; h0 < m.nq; h0 += NW * HR) {
    float qv[HR][DPL];
    uint32_t kr[HR][T], vr[HR][T];  // DPL bf16 values per row (the low half only when DPL == 1)
#pragma unroll
    for (int i = 0; i < HR; ++i) {
      const int h = min(h0 + i, m.nq - 1);
      const int g = h / m.group;
      const float* qh = m.q + (size_t)layer * m.qs + (size_t)h * HD + lane * DPL;
      const uint16_t* Kp = kv + ((size_t)(layer * 2) * m.nkv + g) * hs + lane * DPL;
      const uint16_t* Vp = kv + ((size_t)(layer * 2 + 1) * m.nkv + g) * hs + lane * DPL;
      if constexpr (DPL == 2) {
        const float2 q2 = ldg<float2>(qh);
        qv[i][0] = q2.x;
        qv[i][1] = q2.y;
      } else {
        qv[i][0] = ldg<float>(qh);
      }
      // one load per KV group (the other heads of the group copy it below);
      // positions past pos re-read row pos (clamped, unused)
      if (i > 0 && one_group) continue;
#pragma unroll
      for (int p = 0; p < T; ++p) {
        const size_t off = (size_t)min(p, n - 1) * HD;
        if constexpr (DPL == 2) {
          kr[i][p] = ldg<uint32_t>(Kp + off);
          vr[i][p] = ldg<uint32_t>(Vp + off);
        } else {
          kr[i][p] = ldg<uint16_t>(Kp + off);
          vr[i][p] = ldg<uint16_t>(Vp + off);
        }
      }
    }
    if (one_group) {
#pragma unroll
      for (int i = 1; i < HR; ++i)
#pragma unroll
        for (int p = 0; p < T; ++p) {
          kr[i][p] = kr[0][p];
          vr[i][p] = vr[0][p];
        }
    }
#pragma unroll
    for (int i = 0; i < HR; ++i) {
      float mrun = -INFINITY, l = 0.f, acc[DPL];
#pragma unroll
      for (int j = 0; j < DPL; ++j) acc[j] = 0.f;
#pragma unroll
      for (int p = 0; p < T; ++p) {
        if (p < n) {
          float d = qv[i][0] * bf_lo(kr[i][p]);
          if constexpr (DPL == 2) d = fmaf(qv[i][1], bf_hi(kr[i][p]), d);
          d = wave_sum(d) * m.attn_scale;
          const float mn = fmaxf(mrun, d);
          const float alpha = __expf(mrun - mn), e = __expf(d - mn);
          l = l * alpha + e;
          acc[0] = fmaf(e, bf_lo(vr[i][p]), acc[0] * alpha);
          if constexpr (DPL == 2) acc[1] = fmaf(e, bf_hi(vr[i][p]), acc[1] * alpha);
          mrun = mn;
        }
      }
      const int h = h0 + i;
      if (h < m.nq) {
        const float inv = 1.0f / l;
        float blk = 0.f;
#pragma unroll
        for (int j = 0; j < DPL; ++j) {
          const float o = acc[j] * inv;
          act[act_at(h * HD + lane * DPL + j)] = o;
          blk += o;
        }
        if constexpr (FMT == AMK_WEIGHTS_W4A16) {
          // W4A16 block sums: 32 / DPL lanes hold one 32-column block
          blk = group_sum<32 / DPL>(blk);
          if ((lane & (32 / DPL - 1)) == 0) xsum[(h * HD + lane * DPL) >> 5] = blk;
        }
      }
    }
  }
}

// Number of position splits with work at `pos` (split s covers positions
// [s * chunk, (s + 1) * chunk) of 0..pos).
__device__ __forceinline__ int active_splits(const DevModel& m, int pos, int* chunk_out) {
  const int n_pos = pos + 1;
  const int chunk = (n_pos + m.nsplit - 1) / m.nsplit;
  if (chunk_out) *chunk_out = chunk;
  return (n_pos + chunk - 1) / chunk;
}

// Merge the S (> 1) split records of KV group g into the normalised output of
// its query heads: o_h = sum_s exp(m_s - M) acc_s / sum_s exp(m_s - M) l_s.
// All waves: first the per-(head, split) weights, then every thread sums a
// float4 of the output over a share of the splits with all its loads in
// flight, then the shares are added through LDS.
template <int HD, int GM>
__device__ __forceinline__ void merge_splits(const DevModel& m, int layer, int g, int S, float* scr, int wave,
                                             int lane) {
  const int G = m.group;
  const int rec = G * (kPartHead + HD);
  const float* base = m.part + (size_t)layer * m.ps + (size_t)g * m.nsplit * rec;
  float* wts = scr;                                        // [GM][64]
  float4* red = reinterpret_cast<float4*>(scr + GM * 64);  // [SP][E4]
  if (wave < G) {
    const int h = wave;
    float ms = -INFINITY, ls = 0.f;
    if (lane < S) {
      const float2 ml = ldg<float2>(base + (size_t)lane * rec + h * (kPartHead + HD));
      ms = ml.x;
      ls = ml.y;
    }
    const float M = wave_max(ms);
    const float w = lane < S ? __expf(ms - M) : 0.f;
    const float inv = 1.0f / wave_sum(w * ls);
    wts[h * 64 + lane] = w * inv;
  }
  __syncthreads();
  const int E4 = G * HD / 4;         // float4s of output
  const int SP = max(1, NT / E4);    // split shares
  const int t = threadIdx.x;
  const int o4 = t % E4, sp = t / E4;
  const int h = (4 * o4) / HD, d = 4 * o4 - h * HD;
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
  if (sp < SP) {
    const float* src = base + h * (kPartHead + HD) + kPartHead + d;
    for (int s0 = sp; s0 < S; s0 += 8 * SP) {
      float4 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int s = s0 + k * SP;
        v[k] = s < S ? ldg<float4>(src + (size_t)s * rec) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int s = s0 + k * SP;
        const float w = s < S ? wts[h * 64 + s] : 0.f;
        a.x = fmaf(w, v[k].x, a.x); a.y = fmaf(w, v[k].y, a.y);
        a.z = fmaf(w, v[k].z, a.z); a.w = fmaf(w, v[k].w, a.w);
      }
    }
    red[sp * E4 + o4] = a;
  }
  __syncthreads();
  if (t < E4) {
    float4 o = red[t];
    for (int k = 1; k < SP; ++k) {
      const float4 v = red[k * E4 + t];
      o.x += v.x; o.y += v.y; o.z += v.z; o.w += v.w;
    }
    float* od = m.o + (size_t)layer * m.qs + (size_t)g * G * HD + 4 * t;
    stc(od, o.x); stc(od + 1, o.y); stc(od + 2, o.z); stc(od + 3, o.w);
  }
}

// ---------------------------------------------------------------- the kernel
// TINY: the kernel of the tiny-context schedule, whose O tasks compute the
// attention themselves; the other kernel runs the short and long schedules
// (attention tasks, the inline attention or split merge of a chain counter).
// Each carries only its own attention code, so the tiny one stays within
// 64 KiB of code: the instruction cache then holds it whole, where a larger
// kernel's lines evict each other depending on where the code lies
// (identical machine code measured 20-50 us apart per 8B step at different
// offsets, with instruction-cache misses rising from 6 to 100 thousand per
// step).  Each instantiation starts on a 64 KiB boundary, so its placement
// does not depend on the code size of the others.
template <int HD, int GM, int FMT, bool TINY>
__global__ void __launch_bounds__(NT, 1) __attribute__((aligned(65536)))
amk_decode_kernel(DevModel m, int32_t token, int32_t pos, uint32_t epoch, uint16_t* __restrict__ kv,
                  float* __restrict__ logits, uint64_t timeout_ticks) {
  constexpr int PIPE = Pipe<FMT>::N;
  extern __shared__ float4 lds4[];
  __shared__ Ctl ctl;
  Lds L;
  L.act = reinterpret_cast<float*>(lds4);
  L.stat = L.act + m.lds_act;
  L.res = L.stat + 2 * m.part_stride;
  L.part = L.res + m.part_stride;
  L.xsum = L.part + m.lds_scr;

  const int wave = uni(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int pstride = m.part_stride;

  for (int i = threadIdx.x; i < m.lds_act; i += NT) L.act[i] = 0.f;
  if (threadIdx.x == 0) {
    ctl.abort = 0;
    ctl.cont = 0;
    ctl.res_buf = -1;
    ctl.res_lo = ctl.res_hi = 0;
  }

  const int qb = ldc<int32_t>(m.queue_start + blockIdx.x), qe = ldc<int32_t>(m.queue_start + blockIdx.x + 1);
  // streaming state carried from one task to the next (the weight loads of
  // task idx are issued at the end of task idx - 1)
  uint4 bufA[PIPE], bufB[PIPE];
  uint32_t scA[PIPE], scB[PIPE];  // W4A16 group scales (unused otherwise)
  Cursor ic;
  int gi = 0, g0 = 0, g1 = 0;

  auto prefetch = [&](int idx) {
    g0 = g1 = gi = 0;
    // redefined on every path, so the buffers are dead between a consumer
    // and the next prefetch (attention and inline tasks reuse the registers)
#pragma unroll
    for (int i = 0; i < PIPE; ++i) {
      bufA[i] = bufB[i] = make_uint4(0, 0, 0, 0);
      scA[i] = scB[i] = 0;
    }
    if (idx >= qe) return;
    const amk_task_t tn = ldc<amk_task_t>(m.tasks + idx);
    if (!is_gemv(tn.op)) return;
    const Gemv gn = gemv_geom(m, tn);
    const int sw = wave - 1;
    g0 = wave_gbegin(gn.G, sw);
    g1 = wave_gbegin(gn.G, sw + 1);
    gi = g0;
    if (g0 < g1) {
      cursor_init<FMT>(ic, m, tn, gn, g0);
      issue_block<FMT>(bufA, scA, ic, gi, g1, m, tn, gn, lane);
      issue_block<FMT>(bufB, scB, ic, gi, g1, m, tn, gn, lane);
    }
  };

  // the step's deadline, on this workgroup's clock from its start
  const uint64_t deadline = wall_clock64() + timeout_ticks;
  if (qb < qe && wave != 0) prefetch(qb);
  __syncthreads();

  for (int idx = qb; idx < qe; ++idx) {
    const amk_task_t t = ldc<amk_task_t>(m.tasks + idx);
    const bool gemv = is_gemv(t.op);
    Gemv g;
    if (gemv) g = gemv_geom(m, t);
    uint64_t* tr = m.trace ? m.trace + (size_t)idx * AMK_TRACE_FIELDS : nullptr;

    // ---- B1a: the sync wave's counter wait
    if (wave == 0) {
      if (tr && lane == 0) stg<uint64_t>(tr + AMK_TRACE_WAIT_BEGIN, (uint64_t)wall_clock64());
      const bool ok = wait_deps<FMT>(m, t, m.tasks + idx, epoch, deadline, lane, tr);
      if (!ok && lane == 0) ctl.abort = 1;
      if (tr && lane == 0) stg<uint64_t>(tr + AMK_TRACE_WAIT_END, (uint64_t)wall_clock64());
    }
    __syncthreads();
    if (ctl.abort) return;

    // an attention split with no positions at `pos` has no work
    const bool attn = t.op == AMK_OP_ATTN;
    int chunk = 0;
    const int active = attn ? active_splits(m, pos, &chunk) : 0;
    const bool idle = attn && t.begin >= active;

    // ---- B1b: every wave moves its slice of the input activation
    if (gemv) {
      if constexpr (TINY) {
        if (t.op == AMK_OP_O && t.aux == 1) attention_all<HD, FMT>(m, t.layer, pos, kv, L.act, L.xsum, wave, lane);
        else load_input<FMT>(m, t, token, L, ctl, wave, lane);
      } else {
        load_input<FMT>(m, t, token, L, ctl, wave, lane);
      }
      __syncthreads();
    }
    if (tr && wave == 0 && lane == 0) stg<uint64_t>(tr + AMK_TRACE_INPUT_READY, (uint64_t)wall_clock64());

    // ---- compute (the sync wave meanwhile fetches the epilogue's row data)
    if (gemv && wave == 0) load_rowdata(m, t, token, pos, L, ctl, lane);
    if (gemv && wave != 0 && g0 < g1) {
      const int sw = wave - 1;
      float* mypart = L.part + sw * pstride;
      int cj = g0 / g.gpr, cc = g0 - cj * g.gpr, cg = g0;
      float acc = 0.f;
      constexpr int EX = Pipe<FMT>::EXTRA;
      if constexpr (EX > 0) {
        // blocks are consumed in the order they were issued: A, B, X[0], ...
        uint4 bufX[EX][PIPE];
        uint32_t scX[EX][PIPE];
#pragma unroll
        for (int b = 0; b < EX; ++b) issue_block<FMT>(bufX[b], scX[b], ic, gi, g1, m, t, g, lane);
        while (cg < g1) {
          consume_block<FMT>(bufA, scA, cj, cc, cg, g1, acc, L, mypart, g, lane);
          issue_block<FMT>(bufA, scA, ic, gi, g1, m, t, g, lane);
          consume_block<FMT>(bufB, scB, cj, cc, cg, g1, acc, L, mypart, g, lane);
          issue_block<FMT>(bufB, scB, ic, gi, g1, m, t, g, lane);
#pragma unroll
          for (int b = 0; b < EX; ++b) {
            consume_block<FMT>(bufX[b], scX[b], cj, cc, cg, g1, acc, L, mypart, g, lane);
            issue_block<FMT>(bufX[b], scX[b], ic, gi, g1, m, t, g, lane);
          }
        }
      } else {
        while (cg < g1) {
          consume_block<FMT>(bufA, scA, cj, cc, cg, g1, acc, L, mypart, g, lane);
          issue_block<FMT>(bufA, scA, ic, gi, g1, m, t, g, lane);
          consume_block<FMT>(bufB, scB, cj, cc, cg, g1, acc, L, mypart, g, lane);
          issue_block<FMT>(bufB, scB, ic, gi, g1, m, t, g, lane);
        }
      }
      if (cc != 0) {
        const float s = wave_sum(acc);
        if (lane == 0) mypart[cj] = s;
      }
    } else if constexpr (!TINY) {
      if (attn && !idle) {
        // one split: the normalised output directly; several: a partial record
        const int j0 = t.begin * chunk, j1 = min(pos + 1, j0 + chunk);
        const int rec = m.group * (kPartHead + HD);
        float* dst = active == 1 ? m.o + (size_t)t.layer * m.qs + (size_t)t.aux * m.group * HD
                                 : m.part + (size_t)t.layer * m.ps + ((size_t)t.aux * m.nsplit + t.begin) * rec;
        attention<HD, GM>(m, t.layer, t.aux, j0, j1, kv, L.act, L.part, dst, active > 1, wave, lane);
        drain_vmem();
      }
    }
    __syncthreads();  // B2: GEMV partials in LDS, attention results stored
    // W4A16 in the tiny-context kernel: the next task's weight loads go out now,
    // while the sync wave publishes.  They delay this task's result stores in
    // the CU's request queue, which measured slower for bf16 and int8 weights
    // (+23 us per 8B step each) and faster for int4 (-34 us), whose tasks carry
    // a quarter of bf16's bytes per row.
    constexpr bool EARLY = TINY && FMT == AMK_WEIGHTS_W4A16;
    if constexpr (EARLY) {
      if (wave != 0) prefetch(idx + 1);
    }

    // ---- publish (sync wave)
    if (wave == 0) {
      if (tr && lane == 0) stg<uint64_t>(tr + AMK_TRACE_COMPUTE_END, (uint64_t)wall_clock64());
      switch (t.op) {
        case AMK_OP_QKV: epi_qkv(m, t, g, L, pos, kv, input_rs(m, ctl), lane); break;
        case AMK_OP_O: case AMK_OP_DOWN: epi_residual(m, t, g, L, ctl, lane); break;
        case AMK_OP_GATEUP: epi_gateup(m, t, g, L, input_rs(m, ctl), lane); break;
        case AMK_OP_LMHEAD: epi_lmhead(m, t, g, L, input_rs(m, ctl), logits, lane); break;
        case AMK_OP_ARGMAX: argmax_final(m, t, lane); break;
        default: break;
      }
      if (tr && lane == 0) stg<uint64_t>(tr + AMK_TRACE_PUBLISHED, (uint64_t)wall_clock64());
      bool cont = false;
      if (t.chain_counter >= 0) {
        // the producer that completes the counter runs its inline task: a QKV
        // task's group has npg producers, an attention split's nsplit
        const uint32_t producers = t.op == AMK_OP_QKV ? (uint32_t)m.npg : (uint32_t)m.nsplit;
        cont = release_signal_last(m, t.signal_counter, epoch * producers, lane);
        if (cont) acquire_after_poll();
      } else {
        release_signal(m, t.signal_counter, lane);
      }
      if (lane == 0) ctl.cont = cont;
      if (tr && lane == 0) stg<uint64_t>(tr + AMK_TRACE_SIGNALLED, (uint64_t)wall_clock64());
    }
    __syncthreads();  // B3: results released and signalled

    // ---- inline task of the chain counter (all waves; never in the tiny schedule)
    if constexpr (!TINY) {
      if (ctl.cont) {
        if (t.op == AMK_OP_QKV) {
          float* dst = m.o + (size_t)t.layer * m.qs + (size_t)t.aux * m.group * HD;
          attention<HD, GM>(m, t.layer, t.aux, 0, pos + 1, kv, L.act, L.part, dst, false, wave, lane);
        } else if (active > 1) {
          merge_splits<HD, GM>(m, t.layer, t.aux, active, L.part, wave, lane);
        }
        drain_vmem();
        __syncthreads();  // B4: inline results stored
        if (wave == 0) {
          release_signal(m, t.chain_counter, lane);
          if (tr && lane == 0) stg<uint64_t>(tr + AMK_TRACE_CHAINED, (uint64_t)wall_clock64());
        }
        __syncthreads();  // B5: the next task's loads go out after the chain signal
      } else if (tr && wave == 0 && lane == 0) {
        stg<uint64_t>(tr + AMK_TRACE_CHAINED, 0ull);
      }
    } else if (tr && wave == 0 && lane == 0) {
      stg<uint64_t>(tr + AMK_TRACE_CHAINED, 0ull);
    }

    // ---- the next task's weight stream (streaming waves)
    if constexpr (!EARLY) {
      if (wave != 0) prefetch(idx + 1);
    }
  }
}

// ---------------------------------------------------------------- read probe
// Grid-stride streaming read, four 16-byte loads in flight per thread.
__global__ void __launch_bounds__(NT) amk_read_kernel(const uint4* __restrict__ p, int64_t n16,
                                                      uint32_t* __restrict__ sink) {
  const int64_t stride = (int64_t)gridDim.x * NT;
  int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = ldg<uint4>(p + i), b = ldg<uint4>(p + i + stride);
    const uint4 c = ldg<uint4>(p + i + 2 * stride), d = ldg<uint4>(p + i + 3 * stride);
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n16; i += stride) {
    const uint4 a = ldg<uint4>(p + i);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  sink[(size_t)blockIdx.x * NT + threadIdx.x] = acc;
}

extern "C" int amk_internal_read_probe(const void* buf, int64_t bytes, int32_t blocks, uint32_t* sink,
                                       void* stream) {
  hipLaunchKernelGGL(amk_read_kernel, dim3(blocks), dim3(NT), 0, (hipStream_t)stream, (const uint4*)buf, bytes / 16,
                     sink);
  return hipGetLastError() == hipSuccess ? AMK_OK : AMK_ERR_DEVICE;
}

// ---------------------------------------------------------------- static scratch
// Device memory of a handle made by amk_create_static (its task tables,
// counters, activations, RoPE table and status words): one array per device,
// held from the library's first use on that device until the process ends.
// In host code `scratch` only names the array; its device address on each
// device comes from hipGetSymbolAddress and is used everywhere instead.
static __device__ __align__(256) unsigned char scratch[AMK_STATIC_SCRATCH_BYTES];

extern "C" int amk_internal_static_scratch(int device, void** ptr, size_t* bytes) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  if (!ptr || !bytes || device < 0 || device >= kMaxDevices) return AMK_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[device]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return AMK_ERR_DEVICE;
    }
    addr[device] = p;
  }
  *ptr = addr[device];
  *bytes = sizeof(scratch);
  return AMK_OK;
}

// ---------------------------------------------------------------- host side
template <int HD, int GM, bool TINY>
static const void* kernel_ptr(int fmt) {
  if (fmt == AMK_WEIGHTS_W4A16) return (const void*)amk_decode_kernel<HD, GM, AMK_WEIGHTS_W4A16, TINY>;
  return fmt == AMK_WEIGHTS_W8A16 ? (const void*)amk_decode_kernel<HD, GM, AMK_WEIGHTS_W8A16, TINY>
                                  : (const void*)amk_decode_kernel<HD, GM, AMK_WEIGHTS_BF16, TINY>;
}

template <int HD, int GM>
static const void* kernel_ptr(int fmt, bool tiny) {
  return tiny ? kernel_ptr<HD, GM, true>(fmt) : kernel_ptr<HD, GM, false>(fmt);
}

static const void* kernel_for(int head_dim, int group, int fmt, bool tiny) {
  const bool small = group <= 4;
  if (head_dim == 64) return small ? kernel_ptr<64, 4>(fmt, tiny) : kernel_ptr<64, 8>(fmt, tiny);
  return small ? kernel_ptr<128, 4>(fmt, tiny) : kernel_ptr<128, 8>(fmt, tiny);
}

extern "C" int amk_internal_threads(void) { return NT; }

// Floats of LDS scratch the attention and split merge of one task need (in
// the partials region).
extern "C" int amk_internal_attn_scratch(int group, int head_dim) {
  const bool small = group <= 4;
  if (head_dim == 64) return small ? AttnGeom<64, 4>::LDS : AttnGeom<64, 8>::LDS;
  return small ? AttnGeom<128, 4>::LDS : AttnGeom<128, 8>::LDS;
}

// Both kernels of the shape and format (tiny schedule and the others).
extern "C" int amk_internal_prepare(int head_dim, int group, int fmt, int lds_bytes) {
  for (const bool tiny : {true, false}) {
    const hipError_t e = hipFuncSetAttribute(kernel_for(head_dim, group, fmt, tiny),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    if (e != hipSuccess) return AMK_ERR_DEVICE;
  }
  return AMK_OK;
}

// Largest number of co-resident workgroups per CU for this LDS size that
// both kernels of the shape and format reach.
extern "C" int amk_internal_occupancy(int head_dim, int group, int fmt, int lds_bytes, int* blocks_per_cu) {
  int least = 0;
  for (const bool tiny : {true, false}) {
    int n = 0;
    const hipError_t e =
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel_for(head_dim, group, fmt, tiny), NT, lds_bytes);
    if (e != hipSuccess) return AMK_ERR_DEVICE;
    least = tiny ? n : (n < least ? n : least);
  }
  *blocks_per_cu = least;
  return AMK_OK;
}

extern "C" int amk_internal_launch(const DevModel* m, int32_t tiny, int32_t token, int32_t pos, uint32_t epoch,
                                   uint16_t* kv, float* logits, uint64_t timeout_ticks, void* stream) {
  DevModel mm = *m;
  void* args[] = {&mm, &token, &pos, &epoch, &kv, &logits, &timeout_ticks};
  hipError_t e = hipLaunchCooperativeKernel(kernel_for(m->hd, m->group, m->fmt, tiny != 0), dim3(m->n_cu), dim3(NT), args,
                                            (unsigned)m->lds_bytes, (hipStream_t)stream);
  return e == hipSuccess ? AMK_OK : AMK_ERR_DEVICE;
}

}  // namespace amk
