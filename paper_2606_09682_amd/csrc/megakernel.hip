// One batch-1 Llama decode step as ONE persistent cooperative kernel for
// gfx950 (MI355X): one workgroup per CU walks its host-built task queue
// (paper §3 Algorithm alg:sm) and orders itself against other CUs only
// through monotonic counters (paper §4 "Synchronization model").
//
// Workgroup layout (512 threads = 8 wave64s):
//   wave 0      "sync wave": waits on counters (agent-scope acquire), moves the
//               task's input activation into LDS (RMSNorm folded in), writes
//               every result other CUs read, then releases and signals.
//   waves 1..7  "streaming waves": stream the task's weight rows from HBM in
//               16-byte-per-lane vectors through a double-buffered register
//               pipeline and reduce them against the LDS activation.
// The streaming waves issue the first weight loads of a task BEFORE the
// workgroup barrier that publishes the task's input, so HBM keeps streaming
// while the sync wave waits for producers on other CUs.  Only the sync wave
// executes agent-scope acquire/release sequences, whose vmcnt(0) drains would
// otherwise stall the streaming waves' in-flight loads.
//
// No MFMA: a batch-1 GEMV is a matrix-vector product, bound by HBM bandwidth.
#include <hip/hip_runtime.h>

#include <cmath>

#include "device.h"
#include "schedule.h"

namespace amk {

constexpr int NT = 512;       // threads per workgroup
constexpr int NW = NT / 64;   // waves
constexpr int NSW = NW - 1;   // streaming waves
constexpr int PIPE = 8;       // 1-KiB granules per pipeline half, per wave
constexpr int GRAN = 1024;    // bytes per wave-wide 16-B-per-lane load

struct Ctl {
  float rs;          // 1 / sqrt(mean(x^2) + eps) of the task input
  int abort;
  float m_run[8], l_run[8], alpha[8];
};

// ---------------------------------------------------------------- helpers
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
template <typename T>
__device__ __forceinline__ T ldc(const void* p) {
  using B = typename Bits<sizeof(T)>::T;
  return __builtin_bit_cast(T, *(const AMK_CONST B*)p);
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) {  // round to nearest even
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float i8f(uint32_t w, int k) { return (float)(int8_t)(w >> (8 * k)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ bool is_gemv(int op) {
  return op == AMK_OP_QKV || op == AMK_OP_O || op == AMK_OP_GATEUP || op == AMK_OP_DOWN ||
         op == AMK_OP_LMHEAD;
}

// ---------------------------------------------------------------- GEMV task geometry
struct Gemv {
  int nj;          // rows (jobs)
  int row_bytes;
  int gpr;         // granules per row
  int int8;
  int tail;        // row_bytes not a multiple of GRAN
  int G;           // total granules = nj * gpr
};

// Which matrix and row job j of task t reads.  mat < 0 means the LM head.
__device__ __forceinline__ void job_row(const DevModel& m, const amk_task_t& t, int j, int* mat, int* row) {
  switch (t.op) {
    case AMK_OP_QKV: {
      const int u = t.begin + (j >> 1);
      const int hh = u >> m.half_log2;
      const int r = (u & (m.half - 1)) + (j & 1) * m.half;
      if (hh < m.nq) { *mat = W_Q; *row = hh * m.hd + r; }
      else if (hh < m.nq + m.nkv) { *mat = W_K; *row = (hh - m.nq) * m.hd + r; }
      else { *mat = W_V; *row = (hh - m.nq - m.nkv) * m.hd + r; }
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
__device__ __forceinline__ const float* mat_scale(const DevModel& m, const amk_task_t& t, int mat) {
  if (mat < 0) return m.lm_s;
  return ldc<const float*>(&m.layers[t.layer].s[mat]);
}
__device__ __forceinline__ float scale_of(const DevModel& m, const amk_task_t& t, int mat, int row) {
  return ldg<float>(mat_scale(m, t, mat) + row);
}

__device__ __forceinline__ int task_jobs_dev(const amk_task_t& t) {
  const int n = t.end - t.begin;
  return (t.op == AMK_OP_QKV || t.op == AMK_OP_GATEUP) ? 2 * n : n;
}

__device__ __forceinline__ Gemv gemv_geom(const DevModel& m, const amk_task_t& t) {
  Gemv g;
  int K;
  switch (t.op) {
    case AMK_OP_O: K = m.nq * m.hd; break;
    case AMK_OP_DOWN: K = m.I; break;
    default: K = m.H; break;
  }
  g.int8 = (t.op == AMK_OP_LMHEAD) ? m.lm_int8 : (m.fmt == AMK_WEIGHTS_W8A16);
  g.row_bytes = g.int8 ? K : 2 * K;
  g.gpr = (g.row_bytes + GRAN - 1) / GRAN;
  g.tail = (g.row_bytes % GRAN) != 0;
  g.nj = task_jobs_dev(t);
  g.G = g.nj * g.gpr;
  return g;
}

// Granule range of streaming wave sw: [sw*G/NSW, (sw+1)*G/NSW).
__device__ __forceinline__ int wave_gbegin(int G, int sw) { return (int)(((long)G * sw) / NSW); }

struct Cursor {
  int j, c;
  const uint8_t* p;
};

__device__ __forceinline__ const uint8_t* row_ptr(const DevModel& m, const amk_task_t& t, const Gemv& g, int j) {
  int mat, row;
  job_row(m, t, j, &mat, &row);
  return mat_base(m, t, mat) + (size_t)row * g.row_bytes;
}

__device__ __forceinline__ void cursor_init(Cursor& cu, const DevModel& m, const amk_task_t& t, const Gemv& g,
                                            int gidx) {
  cu.j = gidx / g.gpr;
  cu.c = gidx - cu.j * g.gpr;
  cu.p = row_ptr(m, t, g, cu.j < g.nj ? cu.j : g.nj - 1);
}

__device__ __forceinline__ void cursor_next(Cursor& cu, const DevModel& m, const amk_task_t& t, const Gemv& g) {
  if (++cu.c == g.gpr) {
    cu.c = 0;
    ++cu.j;
    if (cu.j < g.nj) cu.p = row_ptr(m, t, g, cu.j);
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

// Issue PIPE granules starting at global granule index gi (clipped to g1).
__device__ __forceinline__ void issue_block(uint4 (&buf)[PIPE], Cursor& cu, int& gi, int g1, const DevModel& m,
                                            const amk_task_t& t, const Gemv& g, int lane) {
#pragma unroll
  for (int i = 0; i < PIPE; ++i) {
    buf[i] = load_gran(cu, g, lane);
    if (gi < g1) cursor_next(cu, m, t, g);
    ++gi;
  }
}

__device__ __forceinline__ float dot_gran(const uint4 v, const float* __restrict__ act, int c, int lane, int int8,
                                          float acc) {
  if (!int8) {
    const float* x = act + c * (GRAN / 2) + lane * 8;
    const float4 a = *reinterpret_cast<const float4*>(x);
    const float4 b = *reinterpret_cast<const float4*>(x + 4);
    acc = fmaf(bf_lo(v.x), a.x, acc); acc = fmaf(bf_hi(v.x), a.y, acc);
    acc = fmaf(bf_lo(v.y), a.z, acc); acc = fmaf(bf_hi(v.y), a.w, acc);
    acc = fmaf(bf_lo(v.z), b.x, acc); acc = fmaf(bf_hi(v.z), b.y, acc);
    acc = fmaf(bf_lo(v.w), b.z, acc); acc = fmaf(bf_hi(v.w), b.w, acc);
  } else {
    const float* x = act + c * GRAN + lane * 16;
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

// Consume PIPE granules; a finished row's wave-reduced partial goes to part[j].
__device__ __forceinline__ void consume_block(const uint4 (&buf)[PIPE], int& j, int& c, int& gi, int g1, float& acc,
                                              const float* __restrict__ act, float* __restrict__ part,
                                              const Gemv& g, int lane) {
#pragma unroll
  for (int i = 0; i < PIPE; ++i) {
    if (gi < g1) {
      uint4 v = buf[i];
      if (g.tail && c * GRAN + lane * 16 >= g.row_bytes) v = make_uint4(0, 0, 0, 0);
      acc = dot_gran(v, act, c, lane, g.int8, acc);
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

// ---------------------------------------------------------------- sync wave: waits
__device__ __forceinline__ bool wait_deps(const DevModel& m, const amk_task_t& t, const amk_task_t* tp, uint32_t epoch,
                          uint64_t timeout_ticks, int lane) {
  const int nw = t.n_wait;
  if (nw == 0) return __hip_atomic_load(m.dev_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0;
  uint32_t* p = nullptr;
  uint32_t target = 0;
  if (lane < nw) {
    p = m.counters + (size_t)ldg<int32_t>(&tp->wait_counter[lane]) * kCounterStride;
    target = epoch * (uint32_t)ldg<int32_t>(&tp->wait_count[lane]);
  }
  const uint64_t t0 = wall_clock64();
  uint32_t spins = 0;
  for (;;) {
    bool ok = true;
    if (lane < nw) ok = (int32_t)(__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) - target) >= 0;
    if (__all(ok)) break;
    if (__hip_atomic_load(m.dev_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return false;
    ++spins;
    if ((spins & 7u) == 0) {
      // host-mapped flag: read over the bus, so only every 64 spins
      int code = 0;
      if ((spins & 63u) == 0 && __hip_atomic_load(m.host_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM))
        code = AMK_ERR_ABORTED;
      else if (wall_clock64() - t0 > timeout_ticks)
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
    }
    __builtin_amdgcn_s_sleep(2);
  }
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  return true;
}

__device__ __forceinline__ void signal_done(const DevModel& m, const amk_task_t& t, int lane) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  if (lane == 0 && t.signal_counter >= 0)
    __hip_atomic_fetch_add(m.counters + (size_t)t.signal_counter * kCounterStride, 1u, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------- sync wave: prologues
// act[k] = x[k] * g[k] and ctl.rs = 1/sqrt(mean(x^2) + eps); the GEMV result
// is scaled by rs in the epilogue (RMSNorm folded into the consumer).
template <bool SRC_BF16>
__device__ __forceinline__ void load_normed(const void* src, const uint16_t* g, int K, float eps, float* act, Ctl& ctl, int lane) {
  constexpr int NB = 8;
  float ss = 0.f;
  for (int b = 0; b < K; b += NB * 256) {
    float4 xv[NB];
    uint2 gv[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int e = b + (i * 64 + lane) * 4;
      if (e < K) {
        if (SRC_BF16) {
          const uint2 r = ldg<uint2>((const uint16_t*)src + e);
          xv[i] = make_float4(bf_lo(r.x), bf_hi(r.x), bf_lo(r.y), bf_hi(r.y));
        } else {
          xv[i] = ldg<float4>((const float*)src + e);
        }
        gv[i] = ldg<uint2>(g + e);
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int e = b + (i * 64 + lane) * 4;
      if (e < K) {
        const float4 x = xv[i];
        ss = fmaf(x.x, x.x, ss); ss = fmaf(x.y, x.y, ss); ss = fmaf(x.z, x.z, ss); ss = fmaf(x.w, x.w, ss);
        const float4 o = make_float4(x.x * bf_lo(gv[i].x), x.y * bf_hi(gv[i].x), x.z * bf_lo(gv[i].y),
                                     x.w * bf_hi(gv[i].y));
        *reinterpret_cast<float4*>(act + e) = o;
      }
    }
  }
  ss = wave_sum(ss);
  if (lane == 0) ctl.rs = 1.0f / sqrtf(ss / (float)K + eps);
}

// Plain fp32 copy global -> LDS, 16 vectors of 16 B in flight per lane.
__device__ __forceinline__ void load_plain(const float* src, int K, float* act, int lane) {
  constexpr int NB = 16;
  const int n16 = K / 4;  // 16-byte vectors; K is a multiple of 4
  for (int b = 0; b < n16; b += NB * 64) {
    float4 v[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int e = b + i * 64 + lane;
      if (e < n16) v[i] = ldg<float4>(src + (size_t)e * 4);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int e = b + i * 64 + lane;
      if (e < n16) *reinterpret_cast<float4*>(act + (size_t)e * 4) = v[i];
    }
  }
}

// ---------------------------------------------------------------- row sums of a GEMV task
__device__ __forceinline__ float row_sum(const float* part, int stride, const Gemv& g, int j) {
  float s = 0.f;
  const int lo = j * g.gpr, hi = lo + g.gpr;
#pragma unroll
  for (int sw = 0; sw < NSW; ++sw) {
    const int gb = wave_gbegin(g.G, sw), ge = wave_gbegin(g.G, sw + 1);
    // a wave with an empty range wrote nothing, even if gb lies inside the row
    if (gb < ge && gb < hi && ge > lo) s += part[sw * stride + j];
  }
  return s;
}

// ---------------------------------------------------------------- sync wave: epilogues
__device__ __forceinline__ void epi_qkv(const DevModel& m, const amk_task_t& t, const Gemv& g, const float* part, int pos,
                        uint16_t* kv, float rs, int lane) {
  const int l = t.layer;
  for (int u = t.begin + lane; u < t.end; u += 64) {
    const int j0 = 2 * (u - t.begin);
    float y0 = row_sum(part, m.part_stride, g, j0) * rs;
    float y1 = row_sum(part, m.part_stride, g, j0 + 1) * rs;
    int mat, r0, r1;
    job_row(m, t, j0, &mat, &r0);
    job_row(m, t, j0 + 1, &mat, &r1);
    if (g.int8) {
      y0 *= scale_of(m, t, mat, r0);
      y1 *= scale_of(m, t, mat, r1);
    }
    const int hh = u >> m.half_log2;
    const int i = u & (m.half - 1);
    if (mat != W_V) {
      const float2 cs = ldg<float2>(m.rope + (size_t)pos * m.half + i);
      const float a = y0 * cs.x - y1 * cs.y;
      const float b = y1 * cs.x + y0 * cs.y;
      y0 = a;
      y1 = b;
    }
    if (mat == W_Q) {
      float* qd = m.q + (size_t)l * m.nq * m.hd + (size_t)hh * m.hd;
      stg<float>(qd + i, y0);
      stg<float>(qd + i + m.half, y1);
    } else {
      const int kvh = (mat == W_K) ? hh - m.nq : hh - m.nq - m.nkv;
      const int which = (mat == W_K) ? 0 : 1;
      uint16_t* dst = kv + (((size_t)(l * 2 + which) * m.nkv + kvh) * m.max_seq + pos) * m.hd;
      stg<uint16_t>(dst + i, f2bf(y0));
      stg<uint16_t>(dst + i + m.half, f2bf(y1));
    }
  }
}

__device__ __forceinline__ void epi_rows(const DevModel& m, const amk_task_t& t, const Gemv& g, const float* part, float rs,
                         float* logits, int lane) {
  const int l = t.layer;
  const int stride = m.part_stride;
  if (t.op == AMK_OP_GATEUP) {
    for (int r = t.begin + lane; r < t.end; r += 64) {
      const int j = 2 * (r - t.begin);
      float gv = row_sum(part, stride, g, j) * rs;
      float uv = row_sum(part, stride, g, j + 1) * rs;
      if (g.int8) {
        gv *= scale_of(m, t, W_G, r);
        uv *= scale_of(m, t, W_U, r);
      }
      const float silu = gv / (1.0f + __expf(-gv));
      stg<float>(m.a + (size_t)l * m.I + r, silu * uv);
    }
    return;
  }
  if (t.op == AMK_OP_O || t.op == AMK_OP_DOWN) {
    const int mat = t.op == AMK_OP_O ? W_O : W_D;
    const int xin = t.op == AMK_OP_O ? 2 * l : 2 * l + 1;
    for (int r = t.begin + lane; r < t.end; r += 64) {
      float y = row_sum(part, stride, g, r - t.begin);
      if (g.int8) y *= scale_of(m, t, mat, r);
      stg<float>(m.x + (size_t)(xin + 1) * m.H + r, ldg<float>(m.x + (size_t)xin * m.H + r) + y);
    }
    return;
  }
  // LM head: logits + per-task argmax partial (lowest index on ties)
  float best = -INFINITY;
  int besti = 0x7fffffff;
  for (int r = t.begin + lane; r < t.end; r += 64) {
    float y = row_sum(part, stride, g, r - t.begin) * rs;
    if (g.int8) y *= ldg<float>(m.lm_s + r);
    stg<float>(logits + r, y);
    if (y > best || (y == best && r < besti)) { best = y; besti = r; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o);
    const int oi = __shfl_xor(besti, o);
    if (ob > best || (ob == best && oi < besti)) { best = ob; besti = oi; }
  }
  if (lane == 0) stg<float2>(m.argp + 2 * t.aux, make_float2(best, __int_as_float(besti)));
}

// x1 = x0 + Wo o at layer 0 needs the gathered embedding row as x0.
__device__ __forceinline__ void epi_o_layer0(const DevModel& m, const amk_task_t& t, const Gemv& g, const float* part, int token,
                             int lane) {
  const int stride = m.part_stride;
  const uint16_t* e = m.embed + (size_t)token * m.H;
  for (int r = t.begin + lane; r < t.end; r += 64) {
    float y = row_sum(part, stride, g, r - t.begin);
    if (g.int8) y *= scale_of(m, t, W_O, r);
    stg<float>(m.x + (size_t)1 * m.H + r, bf16f(ldg<uint16_t>(e + r)) + y);
  }
}

// Merge the position splits of query heads [begin, end) (flash-decoding style).
__device__ __forceinline__ void combine(const DevModel& m, const amk_task_t& t, int pos, int lane) {
  const int l = t.layer;
  const int n_pos = pos + 1;
  const int chunk = (n_pos + m.nsplit - 1) / m.nsplit;
  const int active = (n_pos + chunk - 1) / chunk;
  const int rec = m.group * (kPartHead + m.hd);
  for (int h = t.begin; h < t.end; ++h) {
    const int g = h / m.group, hg = h - g * m.group;
    const float* base = m.part + ((size_t)(l * m.nkv + g) * m.nsplit) * rec + hg * (kPartHead + m.hd);
    float ms = -INFINITY, ls = 0.f;
    if (lane < active) {
      const float2 ml = ldg<float2>(base + (size_t)lane * rec);
      ms = ml.x;
      ls = ml.y;
    }
    const float M = wave_max(ms);
    const float w = lane < active ? __expf(ms - M) : 0.f;
    const float Ls = wave_sum(w * ls);
    const float inv = 1.0f / Ls;
    float* dst = m.o + (size_t)l * m.nq * m.hd + (size_t)h * m.hd;
    for (int d = lane; d < m.hd; d += 64) {
      float acc = 0.f;
      for (int s = 0; s < active; ++s) {
        const float ws = __shfl(w, s);
        acc = fmaf(ws, ldg<float>(base + (size_t)s * rec + kPartHead + d), acc);
      }
      stg<float>(dst + d, acc * inv);
    }
  }
}

__device__ __forceinline__ void argmax_final(const DevModel& m, const amk_task_t& t, int lane) {
  float best = -INFINITY;
  int besti = 0x7fffffff;
  for (int s = t.begin + lane; s < t.end; s += 64) {
    const float2 vi = ldg<float2>(m.argp + 2 * s);
    const float v = vi.x;
    const int i = __float_as_int(vi.y);
    if (v > best || (v == best && i < besti)) { best = v; besti = i; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o);
    const int oi = __shfl_xor(besti, o);
    if (ob > best || (ob == best && oi < besti)) { best = ob; besti = oi; }
  }
  if (lane == 0) stg<int32_t>(m.next_token, besti);
}

// ---------------------------------------------------------------- attention (all 8 waves)
// Partial attention of query group `t.aux` over position split t.begin of
// t.end: scores, running max / sum (online softmax) and the V-weighted sum.
// One K or V row slice of EPL bf16 values per lane.
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
__device__ __forceinline__ void zero_row(RowVec<EPL>& r) {
  if constexpr (EPL == 8) r.v = make_uint4(0, 0, 0, 0); else r.v = make_uint2(0, 0);
}
template <int EPL>
__device__ __forceinline__ float row_elem(const RowVec<EPL>& r, int e) {
  uint32_t w;
  if constexpr (EPL == 8) w = (e < 2) ? r.v.x : (e < 4) ? r.v.y : (e < 6) ? r.v.z : r.v.w;
  else w = (e < 2) ? r.v.x : r.v.y;
  return (e & 1) ? bf_hi(w) : bf_lo(w);
}

// Geometry of the attention work split (shared with the host LDS sizing).
// GM: largest query group handled; KB: K/V rows per lane per sub-chunk;
// EPL: head dims per lane (8 for groups <= 4, 4 for groups <= 8 to halve
// the per-lane accumulators).
template <int GM, int KB, int EPL>
struct AttnGeom {
  int LPR, RPW, RP, SC;
  __device__ __forceinline__ explicit AttnGeom(int hd) {
    LPR = hd / EPL;
    RPW = 64 / LPR;
    RP = NW * RPW;
    SC = RP * KB;
  }
};

// Partial attention of query group `t.aux` over position split t.begin of
// t.end: scores, running max / sum (online softmax) and the V-weighted sum.
template <int GM, int KB, int EPL>
__device__ __forceinline__ void attention(const DevModel& m, const amk_task_t& t, int pos,
                                          const uint16_t* __restrict__ kv, const float* __restrict__ q,
                                          float* __restrict__ scr, Ctl& ctl, int wave, int lane) {
  const int G = m.group, hd = m.hd;
  const int n_pos = pos + 1;
  const int chunk = (n_pos + m.nsplit - 1) / m.nsplit;
  const int j0 = t.begin * chunk;
  const int j1 = min(n_pos, j0 + chunk);
  const AttnGeom<GM, KB, EPL> ag(hd);
  const int LPR = ag.LPR, RPW = ag.RPW, RP = ag.RP, SC = ag.SC;
  const int sub = lane / LPR, c = lane - sub * LPR;
  const size_t hs = (size_t)m.max_seq * hd;
  const uint16_t* Kp = kv + ((size_t)(t.layer * 2 + 0) * m.nkv + t.aux) * hs + c * EPL;
  const uint16_t* Vp = kv + ((size_t)(t.layer * 2 + 1) * m.nkv + t.aux) * hs + c * EPL;
  float* sc = scr;                        // [GM][SC]
  float* red = scr + GM * SC;             // [NW][G][hd]
  float* out = red + NW * G * hd;         // [G][hd]

  if (threadIdx.x < 8) {
    ctl.m_run[threadIdx.x] = -INFINITY;
    ctl.l_run[threadIdx.x] = 0.f;
  }
  float acc[GM][EPL];
#pragma unroll
  for (int h = 0; h < GM; ++h)
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[h][e] = 0.f;
  __syncthreads();

  for (int t0 = j0; t0 < j1; t0 += SC) {
    const int n = min(SC, j1 - t0);
    RowVec<EPL> kr[KB], vr[KB];
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      const int r = wave * RPW + sub + k * RP;
      zero_row<EPL>(kr[k]);
      if (r < n) kr[k] = load_row<EPL>(Kp + (size_t)(t0 + r) * hd);
    }
    // scores s_j = q_h . k_j / sqrt(d) for the group's query heads
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      const int r = wave * RPW + sub + k * RP;
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        if (h < G) {
          const float* qh = q + h * hd + c * EPL;
          float d = 0.f;
#pragma unroll
          for (int e = 0; e < EPL; ++e) d = fmaf(row_elem<EPL>(kr[k], e), qh[e], d);
          for (int o = 1; o < LPR; o <<= 1) d += __shfl_xor(d, o);
          if (c == 0 && r < n) sc[h * SC + r] = d * m.attn_scale;
        }
      }
    }
    // V rows do not depend on the scores: their loads overlap the softmax statistics below
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      const int r = wave * RPW + sub + k * RP;
      zero_row<EPL>(vr[k]);
      if (r < n) vr[k] = load_row<EPL>(Vp + (size_t)(t0 + r) * hd);
    }
    __syncthreads();
    // running max / sum per head (wave h handles head h)
    if (wave < G) {
      const int h = wave;
      float mx = -INFINITY;
      for (int r = lane; r < n; r += 64) mx = fmaxf(mx, sc[h * SC + r]);
      mx = wave_max(mx);
      const float m_old = ctl.m_run[h];
      const float m_new = fmaxf(m_old, mx);
      float sum = 0.f;
      for (int r = lane; r < n; r += 64) {
        const float p = __expf(sc[h * SC + r] - m_new);
        sc[h * SC + r] = p;
        sum += p;
      }
      sum = wave_sum(sum);
      if (lane == 0) {
        const float alpha = __expf(m_old - m_new);
        ctl.alpha[h] = alpha;
        ctl.l_run[h] = ctl.l_run[h] * alpha + sum;
        ctl.m_run[h] = m_new;
      }
    }
    __syncthreads();
    // V accumulation with the rescaled running sums
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      if (h < G) {
        const float al = ctl.alpha[h];
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[h][e] *= al;
      }
    }
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      const int r = wave * RPW + sub + k * RP;
      if (r < n) {
#pragma unroll
        for (int h = 0; h < GM; ++h) {
          if (h < G) {
            const float p = sc[h * SC + r];
#pragma unroll
            for (int e = 0; e < EPL; ++e) acc[h][e] = fmaf(p, row_elem<EPL>(vr[k], e), acc[h][e]);
          }
        }
      }
    }
    __syncthreads();
  }
  // reduce over the rows a wave covers (lanes with equal c), then over waves
#pragma unroll
  for (int h = 0; h < GM; ++h) {
    if (h < G) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        float v = acc[h][e];
        for (int o = LPR; o < 64; o <<= 1) v += __shfl_xor(v, o);
        if (sub == 0) red[(wave * G + h) * hd + c * EPL + e] = v;
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < G * hd; i += NT) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) s += red[w * G * hd + i];
    out[i] = s;
  }
}

template <int GM, int KB, int EPL>
__device__ __forceinline__ void epi_attn(const DevModel& m, const amk_task_t& t, const float* scr, const Ctl& ctl,
                                         int pos, int lane) {
  const int G = m.group, hd = m.hd;
  const int n_pos = pos + 1;
  const int chunk = (n_pos + m.nsplit - 1) / m.nsplit;
  if (t.begin * chunk >= n_pos) return;  // empty split: the combine ignores it
  const AttnGeom<GM, KB, EPL> ag(hd);
  const float* out = scr + GM * ag.SC + NW * G * hd;
  const int rec = G * (kPartHead + hd);
  float* dst = m.part + ((size_t)(t.layer * m.nkv + t.aux) * m.nsplit + t.begin) * rec;
  for (int h = 0; h < G; ++h) {
    float* d = dst + h * (kPartHead + hd);
    if (lane == 0) stg<float2>(d, make_float2(ctl.m_run[h], ctl.l_run[h]));
    for (int e = lane; e < hd; e += 64) stg<float>(d + kPartHead + e, out[h * hd + e]);
  }
}

// ---------------------------------------------------------------- the kernel
// GM / KB / EPL: attention geometry (see attention()); one instantiation per
// query-group class keeps each kernel's register allocation independent.
template <int GM, int KB, int EPL>
__global__ void __launch_bounds__(NT, 1)
amk_decode_kernel(DevModel m, int32_t token, int32_t pos, uint32_t epoch, uint16_t* __restrict__ kv,
                  float* __restrict__ logits, uint64_t timeout_ticks) {
  extern __shared__ float4 lds4[];
  float* act = reinterpret_cast<float*>(lds4);
  float* part = act + m.lds_act;
  __shared__ Ctl ctl;

  const int wave = uni(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int pstride = m.part_stride;

  for (int i = threadIdx.x; i < m.lds_act; i += NT) act[i] = 0.f;
  if (threadIdx.x == 0) {
    ctl.abort = 0;
    ctl.rs = 1.f;
  }
  __syncthreads();

  const int qb = ldc<int32_t>(m.queue_start + blockIdx.x), qe = ldc<int32_t>(m.queue_start + blockIdx.x + 1);
  for (int idx = qb; idx < qe; ++idx) {
    const amk_task_t t = ldc<amk_task_t>(m.tasks + idx);
    const bool gemv = is_gemv(t.op);
    Gemv g = {0, 0, 1, 0, 0, 0};
    if (gemv) g = gemv_geom(m, t);

    // ---- phase 1: sync wave waits + loads the input; streaming waves prefetch weights
    uint4 bufA[PIPE], bufB[PIPE];
    Cursor ic;
    int gi = 0, g0 = 0, g1 = 0;
    if (wave == 0) {
      const bool ok = wait_deps(m, t, m.tasks + idx, epoch, timeout_ticks, lane);
      if (!ok) {
        if (lane == 0) ctl.abort = 1;
      } else {
        switch (t.op) {
          case AMK_OP_QKV:
            if (t.layer == 0)
              load_normed<true>(m.embed + (size_t)token * m.H, ldc<const uint16_t*>(&m.layers[0].attn_norm), m.H, m.eps, act, ctl, lane);
            else
              load_normed<false>(m.x + (size_t)(2 * t.layer) * m.H, ldc<const uint16_t*>(&m.layers[t.layer].attn_norm), m.H, m.eps, act,
                                 ctl, lane);
            break;
          case AMK_OP_GATEUP:
            load_normed<false>(m.x + (size_t)(2 * t.layer + 1) * m.H, ldc<const uint16_t*>(&m.layers[t.layer].mlp_norm), m.H, m.eps, act,
                               ctl, lane);
            break;
          case AMK_OP_LMHEAD:
            load_normed<false>(m.x + (size_t)(2 * m.L) * m.H, m.final_norm, m.H, m.eps, act, ctl, lane);
            break;
          case AMK_OP_O: load_plain(m.o + (size_t)t.layer * m.nq * m.hd, m.nq * m.hd, act, lane); break;
          case AMK_OP_DOWN: load_plain(m.a + (size_t)t.layer * m.I, m.I, act, lane); break;
          case AMK_OP_ATTN:
            load_plain(m.q + (size_t)t.layer * m.nq * m.hd + (size_t)t.aux * m.group * m.hd, m.group * m.hd, act,
                       lane);
            break;
          default: break;
        }
      }
    } else if (gemv) {
      const int sw = wave - 1;
      g0 = wave_gbegin(g.G, sw);
      g1 = wave_gbegin(g.G, sw + 1);
      gi = g0;
      if (g0 < g1) {
        cursor_init(ic, m, t, g, g0);
        issue_block(bufA, ic, gi, g1, m, t, g, lane);
        issue_block(bufB, ic, gi, g1, m, t, g, lane);
      }
    }
    __syncthreads();  // B1: input activation in LDS
    if (ctl.abort) return;

    // ---- phase 2: compute
    if (gemv && wave != 0 && g0 < g1) {
      const int sw = wave - 1;
      float* mypart = part + sw * pstride;
      int cj = g0 / g.gpr, cc = g0 - cj * g.gpr, cg = g0;
      float acc = 0.f;
      while (cg < g1) {
        consume_block(bufA, cj, cc, cg, g1, acc, act, mypart, g, lane);
        issue_block(bufA, ic, gi, g1, m, t, g, lane);
        consume_block(bufB, cj, cc, cg, g1, acc, act, mypart, g, lane);
        issue_block(bufB, ic, gi, g1, m, t, g, lane);
      }
      if (cc != 0) {
        const float s = wave_sum(acc);
        if (lane == 0) mypart[cj] = s;
      }
    } else if (t.op == AMK_OP_ATTN) {
      attention<GM, KB, EPL>(m, t, pos, kv, act, part, ctl, wave, lane);
    }
    __syncthreads();  // B2: results in LDS

    // ---- phase 3: sync wave publishes results, releases, signals
    if (wave == 0) {
      switch (t.op) {
        case AMK_OP_QKV: epi_qkv(m, t, g, part, pos, kv, ctl.rs, lane); break;
        case AMK_OP_ATTN:
          epi_attn<GM, KB, EPL>(m, t, part, ctl, pos, lane);
          break;
        case AMK_OP_COMBINE: combine(m, t, pos, lane); break;
        case AMK_OP_O:
          if (t.layer == 0) epi_o_layer0(m, t, g, part, token, lane);
          else epi_rows(m, t, g, part, ctl.rs, logits, lane);
          break;
        case AMK_OP_GATEUP: case AMK_OP_DOWN: case AMK_OP_LMHEAD:
          epi_rows(m, t, g, part, ctl.rs, logits, lane);
          break;
        case AMK_OP_ARGMAX: argmax_final(m, t, lane); break;
        default: break;
      }
      signal_done(m, t, lane);
    }
  }
}

// ---------------------------------------------------------------- host side
// Query groups up to 4 heads: 8 head dims per lane, 8 rows in flight per lane.
// Groups of 5..8 heads: 4 head dims per lane, 4 rows in flight per lane.
#define AMK_SMALL_GROUP 4, 8, 8
#define AMK_LARGE_GROUP 8, 4, 4

static const void* kernel_for(int group) {
  return group <= 4 ? (const void*)amk_decode_kernel<AMK_SMALL_GROUP> : (const void*)amk_decode_kernel<AMK_LARGE_GROUP>;
}

extern "C" int amk_internal_threads(void) { return NT; }

// Floats of LDS scratch the attention of one task needs (after the activation region).
extern "C" int amk_internal_attn_scratch(int group, int head_dim) {
  const int GM = group <= 4 ? 4 : 8, KB = group <= 4 ? 8 : 4, EPL = group <= 4 ? 8 : 4;
  const int RP = NW * (64 / (head_dim / EPL));
  return GM * RP * KB + NW * group * head_dim + group * head_dim;
}

extern "C" int amk_internal_prepare(int group, int lds_bytes) {
  hipError_t e = hipFuncSetAttribute(kernel_for(group), hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
  return e == hipSuccess ? AMK_OK : AMK_ERR_DEVICE;
}

// Largest number of co-resident workgroups of the kernel per CU for this LDS size.
extern "C" int amk_internal_occupancy(int group, int lds_bytes, int* blocks_per_cu) {
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, kernel_for(group), NT, lds_bytes);
  return e == hipSuccess ? AMK_OK : AMK_ERR_DEVICE;
}

extern "C" int amk_internal_launch(const DevModel* m, int32_t token, int32_t pos, uint32_t epoch, uint16_t* kv,
                                   float* logits, uint64_t timeout_ticks, void* stream) {
  DevModel mm = *m;
  void* args[] = {&mm, &token, &pos, &epoch, &kv, &logits, &timeout_ticks};
  hipError_t e = hipLaunchCooperativeKernel(kernel_for(m->group), dim3(m->n_cu), dim3(NT), args,
                                            (unsigned)m->lds_bytes, (hipStream_t)stream);
  return e == hipSuccess ? AMK_OK : AMK_ERR_DEVICE;
}

}  // namespace amk
