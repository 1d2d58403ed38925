// Lowering of one batch-1 decode step into per-CU task queues and the static
// schedule check (paper §4 "The invariants validate() proves", Table
// tab:checks; paper §3 Algorithm alg:sm for the queue walk it protects).
#include "schedule.h"

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <queue>

namespace amk {

namespace {

void set_msg(std::string* why, const char* fmt, long a = 0, long b = 0) {
  if (!why) return;
  char buf[256];
  std::snprintf(buf, sizeof(buf), fmt, a, b);
  *why = buf;
}

}  // namespace

int derive_shape(const amk_config_t* cfg, const amk_tuning_t* tuning, int n_cu, Shape* s,
                 std::string* why) {
  if (!cfg || !s) { set_msg(why, "null config"); return AMK_ERR_INVALID_ARGUMENT; }
  if (cfg->abi_version != AMK_ABI_VERSION) {
    set_msg(why, "abi_version %ld, library speaks %ld", cfg->abi_version, AMK_ABI_VERSION);
    return AMK_ERR_INVALID_ARGUMENT;
  }
  if (n_cu < 1) { set_msg(why, "n_cu %ld < 1", n_cu); return AMK_ERR_INVALID_ARGUMENT; }
  const int H = cfg->hidden, L = cfg->n_layers, nq = cfg->n_heads, nkv = cfg->n_kv_heads;
  const int hd = cfg->head_dim, I = cfg->intermediate, V = cfg->vocab, S = cfg->max_seq;
  if (H <= 0 || L <= 0 || nq <= 0 || nkv <= 0 || hd <= 0 || I <= 0 || V <= 0 || S <= 0) {
    set_msg(why, "all dimensions must be positive");
    return AMK_ERR_INVALID_ARGUMENT;
  }
  if (L > 65535) { set_msg(why, "n_layers %ld > 65535", L); return AMK_ERR_UNSUPPORTED; }
  if (cfg->weight_format != AMK_WEIGHTS_BF16 && cfg->weight_format != AMK_WEIGHTS_W8A16 &&
      cfg->weight_format != AMK_WEIGHTS_W4A16) {
    set_msg(why, "unknown weight_format %ld", cfg->weight_format);
    return AMK_ERR_INVALID_ARGUMENT;
  }
  if (cfg->tied_embeddings != 0 && cfg->tied_embeddings != 1) {
    set_msg(why, "tied_embeddings must be 0 or 1");
    return AMK_ERR_INVALID_ARGUMENT;
  }
  if (!(cfg->rope_theta > 0.f) || !(cfg->rms_eps >= 0.f)) {
    set_msg(why, "rope_theta must be > 0 and rms_eps >= 0");
    return AMK_ERR_INVALID_ARGUMENT;
  }
  if (nq % nkv) { set_msg(why, "n_heads %ld not a multiple of n_kv_heads %ld", nq, nkv); return AMK_ERR_UNSUPPORTED; }
  if (nq / nkv > 8) { set_msg(why, "query group %ld > 8", nq / nkv); return AMK_ERR_UNSUPPORTED; }
  if (hd != 64 && hd != 128) {
    set_msg(why, "head_dim %ld must be 64 or 128", hd);
    return AMK_ERR_UNSUPPORTED;
  }
  // every weight row must be a whole number of 16-byte vectors in both formats
  if (H % 16 || I % 16 || (nq * hd) % 16) {
    set_msg(why, "hidden, intermediate and n_heads*head_dim must be multiples of 16");
    return AMK_ERR_UNSUPPORTED;
  }
  // W4A16: a 16-byte vector holds 32 columns and one scale covers whole
  // vectors, so rows are whole vectors and every group a whole number of them
  int qgroup = 0;
  if (cfg->weight_format == AMK_WEIGHTS_W4A16) {
    qgroup = cfg->group_size ? cfg->group_size : 128;
    if (qgroup < 32 || qgroup > 1024 || (qgroup & (qgroup - 1))) {
      set_msg(why, "group_size %ld must be a power of two in [32, 1024]", qgroup);
      return AMK_ERR_INVALID_ARGUMENT;
    }
    if (H % qgroup || I % qgroup || (nq * hd) % qgroup) {
      set_msg(why, "hidden, intermediate and n_heads*head_dim must be multiples of group_size %ld", qgroup);
      return AMK_ERR_UNSUPPORTED;
    }
  }
  int nsplit = tuning && tuning->attn_splits ? tuning->attn_splits : n_cu / nkv;
  nsplit = std::max(1, std::min(nsplit, kMaxAttnSplits));
  if (tuning && tuning->attn_splits && (tuning->attn_splits < 1 || tuning->attn_splits > kMaxAttnSplits)) {
    set_msg(why, "attn_splits %ld outside [1, %ld]", tuning->attn_splits, kMaxAttnSplits);
    return AMK_ERR_INVALID_ARGUMENT;
  }
  int max_jobs = tuning && tuning->max_rows_per_task ? tuning->max_rows_per_task : kMaxJobsPerTask;
  if (max_jobs < 2 || max_jobs > kMaxJobsPerTask) {
    set_msg(why, "max_rows_per_task %ld outside [2, %ld]", max_jobs, kMaxJobsPerTask);
    return AMK_ERR_INVALID_ARGUMENT;
  }
  s->H = H; s->L = L; s->nq = nq; s->nkv = nkv; s->hd = hd; s->I = I; s->V = V; s->max_seq = S;
  s->fmt = cfg->weight_format; s->tied = cfg->tied_embeddings; s->qgroup = qgroup;
  s->group = nq / nkv; s->half = hd / 2;
  s->units = (nq + 2 * nkv) * s->half; s->q_units = nq * s->half;
  s->gunits = (s->group + 2) * s->half;
  s->nsplit = nsplit; s->max_jobs = max_jobs;
  s->theta = cfg->rope_theta; s->eps = cfg->rms_eps;
  // QKV tasks per KV group: the grid's share of the whole QKV stage, at least
  // one task per group and few enough units per task for the row cap
  {
    const int n_qkv = stage_tasks(s->units, 2, n_cu, max_jobs);
    int npg = std::max(1, std::min(n_qkv / nkv, s->gunits));
    while (((s->gunits + npg - 1) / npg) * 2 > max_jobs) ++npg;
    s->npg = npg;
  }
  const int sc = tuning ? tuning->short_context : 0;
  s->short_context = sc == 0 ? kDefaultShortContext : sc < 0 ? 0 : sc;
  const int tc = tuning ? tuning->tiny_context : 0;
  if (tc > AMK_TINY_MAX) {
    set_msg(why, "tiny_context %ld above %ld", tc, AMK_TINY_MAX);
    return AMK_ERR_INVALID_ARGUMENT;
  }
  s->tiny_context = tc == 0 ? kDefaultTinyContext : tc < 0 ? 0 : tc;
  const int qa = tuning ? tuning->queue_assign : AMK_ASSIGN_ROUND_ROBIN;
  if (qa != AMK_ASSIGN_ROUND_ROBIN && qa != AMK_ASSIGN_LPT) {
    set_msg(why, "queue_assign %ld unknown", qa);
    return AMK_ERR_INVALID_ARGUMENT;
  }
  s->assign = qa;
  return AMK_OK;
}

int stage_tasks(int items, int jobs_per_item, int n_cu, int max_jobs) {
  int n = std::min(n_cu, items);
  const int need = (int)(((long)items * jobs_per_item + max_jobs - 1) / max_jobs);
  // each task must also hold whole items: ceil(items / n) * jobs_per_item <= max_jobs
  n = std::max(n, need);
  while (((items + n - 1) / n) * jobs_per_item > max_jobs) ++n;
  return std::min(n, items);
}

UnitHead unit_head(const Shape& s, int u) {
  const int slot = u / s.half;
  const int g = slot / (s.group + 2), r = slot % (s.group + 2);
  UnitHead h;
  h.i = u % s.half;
  if (r < s.group) { h.kind = 0; h.head = g * s.group + r; }
  else { h.kind = r == s.group ? 1 : 2; h.head = g; }
  return h;
}

int task_jobs(const Shape& s, const amk_task_t& t) {
  const int n = t.end - t.begin;
  switch (t.op) {
    case AMK_OP_QKV: return 2 * n;
    case AMK_OP_GATEUP: return 2 * n;
    case AMK_OP_O: case AMK_OP_DOWN: case AMK_OP_LMHEAD: return n;
    default: return 0;
  }
}

// ---------------------------------------------------------------------------
// lowering
// ---------------------------------------------------------------------------
Schedule build_schedule(const Shape& s, int n_cu, int variant) {
  Schedule sch;
  std::vector<int> qlen(n_cu, 0);
  int n_ctr = 0;
  int rot = 0;  // rotating start CU for stages narrower than the grid

  auto add = [&](int op, int layer, int cu, int b, int e, int aux,
                 std::vector<std::pair<int, int>> waits, int sig, int chain = -1) {
    amk_task_t t;
    std::memset(&t, 0, sizeof(t));
    t.op = (uint16_t)op; t.layer = (uint16_t)layer; t.cu = cu;
    t.seq = cu == AMK_CU_INLINE ? 0 : qlen[cu]++;
    t.begin = b; t.end = e; t.aux = (int16_t)aux;
    t.n_wait = (int16_t)waits.size();
    t.chain_counter = chain;
    for (int i = 0; i < AMK_MAX_WAITS; ++i) { t.wait_counter[i] = -1; t.wait_count[i] = 0; }
    for (size_t i = 0; i < waits.size(); ++i) {
      t.wait_counter[i] = waits[i].first; t.wait_count[i] = waits[i].second;
    }
    t.signal_counter = sig;
    sch.tasks.push_back(t);
  };
  // number of tasks for a stage of `items` work items of `jobs_per_item` rows
  auto n_tasks = [&](int items, int jobs_per_item) { return stage_tasks(items, jobs_per_item, n_cu, s.max_jobs); };
  auto cu_of = [&](int i, int n) { return n >= n_cu ? i % n_cu : (rot + i) % n_cu; };
  auto bump = [&](int n) { if (n < n_cu) rot = (rot + n) % n_cu; };
  // LPT: estimated work per queue so far, in bytes streamed; a task costs
  // the bytes of its weight rows (or K/V rows) plus a fixed per-task cost
  // for its wait, input load and epilogue (about 2.5 us of streaming)
  const bool lpt = s.assign == AMK_ASSIGN_LPT;
  std::vector<double> load(n_cu, 0.0);
  constexpr double kTaskFixedBytes = 64.0 * 1024;
  const double wbytes = s.fmt == AMK_WEIGHTS_BF16 ? 2.0 : s.fmt == AMK_WEIGHTS_W8A16 ? 1.0 : 0.5;
  // queues for the n tasks of one stage with per-task costs `cost`
  auto place = [&](const std::vector<double>& cost) {
    const int n = (int)cost.size();
    std::vector<int> cu(n);
    if (!lpt) {
      for (int i = 0; i < n; ++i) cu[i] = cu_of(i, n);
      bump(n);
      return cu;
    }
    std::vector<int> idx(n);
    std::iota(idx.begin(), idx.end(), 0);
    std::stable_sort(idx.begin(), idx.end(), [&](int a, int b) { return cost[a] > cost[b]; });
    // least-loaded queue first, lowest index on ties
    using Item = std::pair<double, int>;
    std::priority_queue<Item, std::vector<Item>, std::greater<Item>> heap;
    for (int c = 0; c < n_cu; ++c) heap.push({load[c], c});
    for (int i : idx) {
      const Item it = heap.top();
      heap.pop();
      cu[i] = it.second;
      load[it.second] = it.first + cost[i] + kTaskFixedBytes;
      heap.push({load[it.second], it.second});
    }
    return cu;
  };
  auto gemv_cost = [&](int rows, int in) { return rows * (double)in * wbytes; };
  auto lo = [](int total, int parts, int i) { return (int)((long)total * i / parts); };
  // A stage's n producers signal kStageCounters counters (task i counter i mod
  // k), and its consumers wait on each with that counter's producer count:
  // fewer increments per counter line than one counter for the whole stage.
  using Waits = std::vector<std::pair<int, int>>;
  auto stage_counters = [&](int n, int* first) {
    const int k = std::min(kStageCounters, n);
    *first = n_ctr;
    n_ctr += k;
    Waits w;
    for (int j = 0; j < k; ++j) w.push_back({*first + j, (n - j + k - 1) / k});
    return w;
  };
  auto sig_of = [&](int first, int n, int i) { return first + i % std::min(kStageCounters, n); };
  // a stage of n tasks over `items` items, all waiting on `w`; returns its consumers' waits
  auto stage = [&](int op, int layer, int items, int jobs_per_item, const Waits& w) {
    const int n = n_tasks(items, jobs_per_item);
    int first = 0;
    const Waits out = stage_counters(n, &first);
    const int in = op == AMK_OP_O ? s.nq * s.hd : op == AMK_OP_DOWN ? s.I : s.H;
    std::vector<double> cost(n);
    for (int i = 0; i < n; ++i) cost[i] = gemv_cost((lo(items, n, i + 1) - lo(items, n, i)) * jobs_per_item, in);
    const std::vector<int> cu = place(cost);
    for (int i = 0; i < n; ++i)
      add(op, layer, cu[i], lo(items, n, i), lo(items, n, i + 1), 0, w, sig_of(first, n, i));
    return out;
  };

  const bool shortv = variant == AMK_SCHEDULE_SHORT, tinyv = variant == AMK_SCHEDULE_TINY;
  Waits prev;  // waits on the stage producing the layer input (none for layer 0)
  for (int l = 0; l < s.L; ++l) {
    // QKV: npg tasks per KV group over that group's units; each group's tasks
    // signal the group's counter (tiny schedule: the stage's counters).
    const int n_qkv = s.nkv * s.npg;
    int c_qkv0 = 0;
    Waits qkv_out;
    if (tinyv) {
      qkv_out = stage_counters(n_qkv, &c_qkv0);
    } else {
      c_qkv0 = n_ctr;
      n_ctr += s.nkv;
    }
    const int c_done = tinyv ? -1 : n_ctr++;  // every KV group's attention output is written
    std::vector<double> qcost(n_qkv);
    for (int k = 0; k < n_qkv; ++k)
      qcost[k] = gemv_cost(2 * (lo(s.gunits, s.npg, k % s.npg + 1) - lo(s.gunits, s.npg, k % s.npg)), s.H);
    const std::vector<int> qcu = place(qcost);
    for (int g = 0; g < s.nkv; ++g) {
      for (int i = 0; i < s.npg; ++i) {
        const int b = g * s.gunits + lo(s.gunits, s.npg, i), e = g * s.gunits + lo(s.gunits, s.npg, i + 1);
        add(AMK_OP_QKV, l, qcu[g * s.npg + i], b, e, g, prev,
            tinyv ? sig_of(c_qkv0, n_qkv, g * s.npg + i) : c_qkv0 + g, shortv ? c_done : -1);
      }
    }
    if (tinyv) {
      // O tasks compute the attention themselves from q and the KV cache
      const int n = n_tasks(s.H, 1);
      int first = 0;
      const Waits o_out = stage_counters(n, &first);
      std::vector<double> ocost(n);
      for (int i = 0; i < n; ++i) ocost[i] = gemv_cost(lo(s.H, n, i + 1) - lo(s.H, n, i), s.nq * s.hd);
      const std::vector<int> ocu = place(ocost);
      for (int i = 0; i < n; ++i)
        add(AMK_OP_O, l, ocu[i], lo(s.H, n, i), lo(s.H, n, i + 1), 1, qkv_out, sig_of(first, n, i));
      const Waits gu = stage(AMK_OP_GATEUP, l, s.I, 2, o_out);
      prev = stage(AMK_OP_DOWN, l, s.H, 1, gu);
      continue;
    }
    if (shortv) {
      // the QKV task of group g that finishes last runs the group's attention
      for (int g = 0; g < s.nkv; ++g)
        add(AMK_OP_ATTN, l, AMK_CU_INLINE, 0, 1, g, {{c_qkv0 + g, s.npg}}, c_done);
    } else {
      // one task per (KV group, position split); the splits of a group signal
      // the group's counter, and the split that increments it last runs the
      // group's inline COMBINE, which signals c_done
      const int c_grp0 = n_ctr;
      n_ctr += s.nkv;
      const int n_attn = s.nkv * s.nsplit;
      // a split's K/V rows are not known when the schedule is built (they
      // grow with the position): equal nominal costs
      const std::vector<int> acu = place(std::vector<double>(n_attn, 2.0 * s.hd * 2 * 256));
      for (int i = 0; i < n_attn; ++i) {
        const int g = i / s.nsplit;
        add(AMK_OP_ATTN, l, acu[i], i % s.nsplit, s.nsplit, g, {{c_qkv0 + g, s.npg}}, c_grp0 + g, c_done);
      }
      for (int g = 0; g < s.nkv; ++g)
        add(AMK_OP_COMBINE, l, AMK_CU_INLINE, g * s.group, (g + 1) * s.group, g, {{c_grp0 + g, s.nsplit}}, c_done);
    }
    const Waits o = stage(AMK_OP_O, l, s.H, 1, {{c_done, s.nkv}});
    const Waits gu = stage(AMK_OP_GATEUP, l, s.I, 2, o);
    prev = stage(AMK_OP_DOWN, l, s.H, 1, gu);
  }
  // LM head: one argmax partial slot per task
  {
    const int n = n_tasks(s.V, 1);
    int first = 0;
    const Waits lm_out = stage_counters(n, &first);
    const double lm_bytes = s.tied ? 2.0 : wbytes;
    std::vector<double> lcost(n);
    for (int i = 0; i < n; ++i) lcost[i] = (lo(s.V, n, i + 1) - lo(s.V, n, i)) * (double)s.H * lm_bytes;
    const std::vector<int> lcu = place(lcost);
    for (int i = 0; i < n; ++i)
      add(AMK_OP_LMHEAD, 0, lcu[i], lo(s.V, n, i), lo(s.V, n, i + 1), i, prev, sig_of(first, n, i));
    add(AMK_OP_ARGMAX, 0, place({0.0})[0], 0, n, 0, lm_out, -1);
    sch.n_lm_slots = n;
  }
  sch.n_counters = n_ctr;
  finalize_queues(&sch.tasks, n_cu, &sch.queue_start);
  return sch;
}

void finalize_queues(std::vector<amk_task_t>* tasks, int n_cu, std::vector<int32_t>* queue_start) {
  // queued tasks by (cu, seq); inline tasks (no queue) after all of them
  auto key = [n_cu](const amk_task_t& t) { return t.cu == AMK_CU_INLINE ? n_cu : t.cu; };
  std::stable_sort(tasks->begin(), tasks->end(), [&](const amk_task_t& a, const amk_task_t& b) {
    return key(a) != key(b) ? key(a) < key(b) : a.seq < b.seq;
  });
  queue_start->assign(n_cu + 1, 0);
  for (const auto& t : *tasks)
    if (t.cu != AMK_CU_INLINE) (*queue_start)[t.cu + 1]++;
  for (int c = 0; c < n_cu; ++c) (*queue_start)[c + 1] += (*queue_start)[c];
}

// ---------------------------------------------------------------------------
// static check
// ---------------------------------------------------------------------------
namespace {

// Buffers a task reads or writes within one launch.  Index spaces:
//   X(i)   i in [0, 2L]: residual stream, H elements; X(0) is the gathered
//          embedding row (an input, written by nobody)
//   Q(l)   q/RoPE units: n_heads * d/2
//   KV(l)  appended K and V row-pair units: 2 * n_kv * d/2 (K first)
//   PART(l) attention partial slots: n_kv * nsplit
//   O(l)   attention output: n_heads * d
//   A(l)   SwiGLU output: I
//   LOGITS V;  ARGP n_lm_slots;  NEXT 1
enum BufKind { B_X = 0, B_Q, B_KV, B_PART, B_O, B_A, B_LOGITS, B_ARGP, B_NEXT };

struct Access {
  int buf;  // dense buffer id
  int lo, hi;
};

struct BufIds {
  int L;
  int x(int i) const { return i; }
  int q(int l) const { return 2 * L + 1 + l; }
  int kv(int l) const { return 3 * L + 1 + l; }
  int part(int l) const { return 4 * L + 1 + l; }
  int o(int l) const { return 5 * L + 1 + l; }
  int a(int l) const { return 6 * L + 1 + l; }
  int logits() const { return 7 * L + 1; }
  int argp() const { return 7 * L + 2; }
  int next() const { return 7 * L + 3; }
  int count() const { return 7 * L + 4; }
  bool is_kv(int b) const { return b >= 3 * L + 1 && b < 4 * L + 1; }
  bool is_part(int b) const { return b >= 4 * L + 1 && b < 5 * L + 1; }
  bool is_o(int b) const { return b >= 5 * L + 1 && b < 6 * L + 1; }
};

void accesses(const Shape& s, const BufIds& ids, const amk_task_t& t, std::vector<Access>* rd,
              std::vector<Access>* wr) {
  rd->clear(); wr->clear();
  const int l = t.layer;
  switch (t.op) {
    case AMK_OP_QKV: {
      rd->push_back({ids.x(2 * l), 0, s.H});
      // group-major units -> query units (head-major) and K/V units (K heads, then V heads)
      for (int g = t.begin / s.gunits; g * s.gunits < t.end; ++g) {
        const int b = std::max(t.begin, g * s.gunits) - g * s.gunits;
        const int e = std::min(t.end, (g + 1) * s.gunits) - g * s.gunits;
        const int qn = s.group * s.half;
        if (b < qn) wr->push_back({ids.q(l), g * qn + b, g * qn + std::min(e, qn)});
        const int kb = std::max(b, qn), ke = std::min(e, qn + s.half);
        if (kb < ke) wr->push_back({ids.kv(l), g * s.half + kb - qn, g * s.half + ke - qn});
        const int vb = std::max(b, qn + s.half), ve = e;
        if (vb < ve)
          wr->push_back({ids.kv(l), (s.nkv + g) * s.half + vb - qn - s.half, (s.nkv + g) * s.half + ve - qn - s.half});
      }
      break;
    }
    case AMK_OP_ATTN: {
      const int g = t.aux;
      rd->push_back({ids.kv(l), g * s.half, (g + 1) * s.half});                         // K head g
      rd->push_back({ids.kv(l), (s.nkv + g) * s.half, (s.nkv + g + 1) * s.half});       // V head g
      rd->push_back({ids.q(l), g * s.group * s.half, (g + 1) * s.group * s.half});
      if (t.cu == AMK_CU_INLINE)  // the whole position range: writes the group's output
        wr->push_back({ids.o(l), g * s.group * s.hd, (g + 1) * s.group * s.hd});
      else
        wr->push_back({ids.part(l), g * s.nsplit + t.begin, g * s.nsplit + t.begin + 1});
      break;
    }
    case AMK_OP_COMBINE: {
      const int g0 = t.begin / s.group, g1 = (t.end - 1) / s.group + 1;
      rd->push_back({ids.part(l), g0 * s.nsplit, g1 * s.nsplit});
      wr->push_back({ids.o(l), t.begin * s.hd, t.end * s.hd});
      break;
    }
    case AMK_OP_O:
      if (t.aux == 1) {  // attention computed in the task from q and the whole KV stage of the layer
        rd->push_back({ids.q(l), 0, s.q_units});
        rd->push_back({ids.kv(l), 0, 2 * s.nkv * s.half});
      } else {
        rd->push_back({ids.o(l), 0, s.nq * s.hd});
      }
      rd->push_back({ids.x(2 * l), t.begin, t.end});
      wr->push_back({ids.x(2 * l + 1), t.begin, t.end});
      break;
    case AMK_OP_GATEUP:
      rd->push_back({ids.x(2 * l + 1), 0, s.H});
      wr->push_back({ids.a(l), t.begin, t.end});
      break;
    case AMK_OP_DOWN:
      rd->push_back({ids.a(l), 0, s.I});
      rd->push_back({ids.x(2 * l + 1), t.begin, t.end});
      wr->push_back({ids.x(2 * l + 2), t.begin, t.end});
      break;
    case AMK_OP_LMHEAD:
      rd->push_back({ids.x(2 * s.L), 0, s.H});
      wr->push_back({ids.logits(), t.begin, t.end});
      wr->push_back({ids.argp(), t.aux, t.aux + 1});
      break;
    case AMK_OP_ARGMAX:
      rd->push_back({ids.argp(), t.begin, t.end});
      wr->push_back({ids.next(), 0, 1});
      break;
    default: break;
  }
}

struct Reporter {
  amk_check_report_t* r;
  bool fail(int rule, int task, int other, const char* fmt, long a = 0, long b = 0, long c = 0) {
    r->ok = 0; r->rule = rule; r->task = task; r->other = other;
    std::snprintf(r->message, sizeof(r->message), fmt, a, b, c);
    return false;
  }
};

}  // namespace

bool check_schedule(const Shape& s, int n_cu, const amk_task_t* tasks, int n, int n_counters,
                    amk_check_report_t* rep) {
  std::memset(rep, 0, sizeof(*rep));
  rep->ok = 1; rep->rule = AMK_CHECK_OK; rep->task = -1; rep->other = -1;
  rep->n_tasks = n; rep->n_counters = n_counters;
  Reporter R{rep};
  if (n <= 0 || !tasks) return R.fail(AMK_CHECK_WELL_FORMED, -1, -1, "empty schedule");
  if (n_counters < 0) return R.fail(AMK_CHECK_WELL_FORMED, -1, -1, "negative counter count");

  // ---- 1. well-formedness and capacity -----------------------------------
  int n_lm = 0;
  for (int i = 0; i < n; ++i)
    if (tasks[i].op == AMK_OP_LMHEAD) ++n_lm;
  std::vector<int> qlen(n_cu, 0);
  for (int i = 0; i < n; ++i) {
    const amk_task_t& t = tasks[i];
    if (t.op < AMK_OP_QKV || t.op > AMK_OP_ARGMAX)
      return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: unknown op %ld", i, t.op);
    const bool inl = t.cu == AMK_CU_INLINE;
    if (!inl && (t.cu < 0 || t.cu >= n_cu))
      return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: queue %ld out of range", i, t.cu);
    if (inl && ((t.op != AMK_OP_COMBINE && t.op != AMK_OP_ATTN) || t.seq != 0))
      return R.fail(AMK_CHECK_INLINE, i, -1, "task %ld: only an ATTN or COMBINE (seq 0) may run inline", i);
    if (t.chain_counter < -1 || t.chain_counter >= n_counters)
      return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: chain counter %ld out of range", i, t.chain_counter);
    const bool layered = t.op <= AMK_OP_DOWN;
    if (layered && t.layer >= s.L)
      return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: layer %ld out of range", i, t.layer);
    if (t.n_wait < 0 || t.n_wait > AMK_MAX_WAITS)
      return R.fail(AMK_CHECK_CAPACITY, i, -1, "task %ld: %ld waits (cap 4)", i, t.n_wait);
    for (int w = 0; w < t.n_wait; ++w)
      if (t.wait_counter[w] < 0 || t.wait_counter[w] >= n_counters)
        return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: wait on counter %ld out of range", i,
                      t.wait_counter[w]);
    if (t.signal_counter < -1 || t.signal_counter >= n_counters)
      return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: signal counter %ld out of range", i,
                    t.signal_counter);
    int lim = 0;
    switch (t.op) {
      case AMK_OP_QKV: lim = s.units; break;
      case AMK_OP_ATTN: lim = s.nsplit; break;
      case AMK_OP_COMBINE: lim = s.nq; break;
      case AMK_OP_O: case AMK_OP_DOWN: lim = s.H; break;
      case AMK_OP_GATEUP: lim = s.I; break;
      case AMK_OP_LMHEAD: lim = s.V; break;
      case AMK_OP_ARGMAX: lim = n_lm; break;
    }
    if (t.op == AMK_OP_ATTN) {
      const bool split_ok = inl ? (t.begin == 0 && t.end == 1) : (t.end == s.nsplit && t.begin >= 0 && t.begin < s.nsplit);
      if (!split_ok || t.aux < 0 || t.aux >= s.nkv)
        return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: bad attention split/head", i);
    } else if (t.begin < 0 || t.end > lim || t.begin >= t.end) {
      return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: range [%ld, ...) out of bounds", i, t.begin);
    }
    if (t.op == AMK_OP_QKV && (t.aux < 0 || t.aux >= s.nkv || t.begin / s.gunits != t.aux ||
                               (t.end - 1) / s.gunits != t.aux))
      return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: QKV units must lie in KV group aux %ld", i, t.aux);
    if (t.op == AMK_OP_O && (t.aux < 0 || t.aux > 1))
      return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: O aux %ld must be 0 or 1", i, t.aux);
    if (t.op == AMK_OP_ARGMAX && (t.begin != 0 || t.end != n_lm))
      return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: argmax must reduce all %ld partial slots", i, n_lm);
    if (t.op == AMK_OP_LMHEAD && (t.aux < 0 || t.aux >= n_lm))
      return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: argmax slot %ld out of range", i, t.aux);
    if (task_jobs(s, t) > s.max_jobs)
      return R.fail(AMK_CHECK_CAPACITY, i, -1, "task %ld: %ld rows exceed the per-task cap", i, task_jobs(s, t));
    if (t.op == AMK_OP_COMBINE && t.end - t.begin > 64)
      return R.fail(AMK_CHECK_CAPACITY, i, -1, "task %ld: combine of more than 64 heads", i);
    if (!inl) qlen[t.cu]++;
  }
  // queue positions must be 0..len-1, each exactly once
  {
    std::vector<std::vector<int>> at(n_cu);
    for (int c = 0; c < n_cu; ++c) at[c].assign(qlen[c], -1);
    for (int i = 0; i < n; ++i) {
      const amk_task_t& t = tasks[i];
      if (t.cu == AMK_CU_INLINE) continue;
      if (t.seq < 0 || t.seq >= qlen[t.cu] || at[t.cu][t.seq] != -1)
        return R.fail(AMK_CHECK_WELL_FORMED, i, -1, "task %ld: queue position %ld invalid or repeated", i, t.seq);
      at[t.cu][t.seq] = i;
    }
  }

  // ---- 2. wait satisfiability and all-join ----------------------------------
  std::vector<std::vector<int>> producers(n_counters), waiters(n_counters);
  for (int i = 0; i < n; ++i) {
    if (tasks[i].signal_counter >= 0) producers[tasks[i].signal_counter].push_back(i);
    for (int w = 0; w < tasks[i].n_wait; ++w) waiters[tasks[i].wait_counter[w]].push_back(i);
  }
  for (int i = 0; i < n; ++i) {
    const amk_task_t& t = tasks[i];
    for (int w = 0; w < t.n_wait; ++w) {
      const int c = t.wait_counter[w], need = t.wait_count[w];
      const int np = (int)producers[c].size();
      if (need < 1) return R.fail(AMK_CHECK_WAIT_SATISFIABLE, i, c, "task %ld waits for %ld < 1 signals", i, need);
      if (np == 0) return R.fail(AMK_CHECK_WAIT_SATISFIABLE, i, c, "task %ld waits on counter %ld that nobody signals", i, c);
      if (need > np)
        return R.fail(AMK_CHECK_WAIT_SATISFIABLE, i, c, "task %ld needs %ld signals, counter has %ld producers", i, need, np);
      if (need != np)
        return R.fail(AMK_CHECK_ALL_JOIN, i, c, "task %ld waits for %ld of %ld producers (which-producer race)", i, need, np);
    }
  }

  // ---- 2b. inline tasks: one wait; every producer of that counter chains to
  //          the inline task's signal; every chaining task feeds exactly one
  //          inline task ------------------------------------------------------
  std::vector<int> inline_of(n_counters, -1);  // counter -> inline task waiting on it
  for (int i = 0; i < n; ++i) {
    const amk_task_t& t = tasks[i];
    if (t.cu != AMK_CU_INLINE) continue;
    if (t.n_wait != 1 || t.signal_counter < 0)
      return R.fail(AMK_CHECK_INLINE, i, -1, "inline task %ld needs exactly one wait and a signal", i);
    const int c = t.wait_counter[0];
    if (inline_of[c] != -1)
      return R.fail(AMK_CHECK_INLINE, i, inline_of[c], "counter %ld feeds two inline tasks", c);
    inline_of[c] = i;
    for (int p : producers[c])
      if (tasks[p].chain_counter != t.signal_counter || tasks[p].cu == AMK_CU_INLINE)
        return R.fail(AMK_CHECK_INLINE, i, p, "producer %ld of inline task %ld does not chain to its signal", p, i);
  }
  for (int i = 0; i < n; ++i) {
    const amk_task_t& t = tasks[i];
    if (t.chain_counter < 0) continue;
    const int k = t.signal_counter >= 0 ? inline_of[t.signal_counter] : -1;
    if (k < 0 || tasks[k].signal_counter != t.chain_counter)
      return R.fail(AMK_CHECK_INLINE, i, k, "task %ld chains to counter %ld without a matching inline task", i,
                    t.chain_counter);
    // the device runs the continuation from the chaining task alone: a QKV
    // task runs its group's attention, an attention split its group's
    // combine, and it counts npg resp. nsplit producers on the way
    const amk_task_t& it = tasks[k];
    const bool pair_ok = (t.op == AMK_OP_QKV && it.op == AMK_OP_ATTN) ||
                         (t.op == AMK_OP_ATTN && t.cu != AMK_CU_INLINE && it.op == AMK_OP_COMBINE);
    if (!pair_ok || it.aux != t.aux || (it.op == AMK_OP_COMBINE && (it.begin != t.aux * s.group ||
                                                                    it.end != (t.aux + 1) * s.group)))
      return R.fail(AMK_CHECK_INLINE, i, k, "task %ld (op %ld) cannot run inline task %ld", i, t.op, k);
    const int expect = t.op == AMK_OP_QKV ? s.npg : s.nsplit;
    if ((int)producers[t.signal_counter].size() != expect)
      return R.fail(AMK_CHECK_INLINE, i, t.signal_counter, "chained counter %ld has %ld producers, device counts %ld",
                    t.signal_counter, (long)producers[t.signal_counter].size(), expect);
  }

  // ---- 3. queue order: a producer on the same CU must be queued earlier ------
  long n_edges = 0;
  for (int i = 0; i < n; ++i) {
    const amk_task_t& t = tasks[i];
    for (int w = 0; w < t.n_wait; ++w) {
      for (int p : producers[t.wait_counter[w]]) {
        ++n_edges;
        if (t.cu != AMK_CU_INLINE && tasks[p].cu == t.cu && tasks[p].seq >= t.seq)
          return R.fail(AMK_CHECK_QUEUE_ORDER, i, p, "task %ld on queue %ld waits on task %ld queued at or after it", i,
                        t.cu, p);
      }
    }
  }
  rep->n_edges = (int)std::min<long>(n_edges, 0x7fffffff);

  // ---- 4. acyclicity of (counter edges + queue-order edges): Kahn ------------
  // A task is ready when its queue predecessor has run and every counter it
  // waits on has all its producers run.  The order found is also a valid
  // global order for the happens-before pass below.
  std::vector<std::vector<int>> queue(n_cu);
  for (int c = 0; c < n_cu; ++c) queue[c].assign(qlen[c], -1);
  for (int i = 0; i < n; ++i)
    if (tasks[i].cu != AMK_CU_INLINE) queue[tasks[i].cu][tasks[i].seq] = i;
  std::vector<int> indeg(n, 0), remaining(n_counters);
  for (int c = 0; c < n_counters; ++c) remaining[c] = (int)producers[c].size();
  for (int i = 0; i < n; ++i)
    indeg[i] = (tasks[i].cu != AMK_CU_INLINE && tasks[i].seq > 0 ? 1 : 0) + tasks[i].n_wait;
  std::vector<int> order;
  order.reserve(n);
  std::vector<int> stack;
  for (int i = 0; i < n; ++i)
    if (indeg[i] == 0) stack.push_back(i);
  while (!stack.empty()) {
    const int i = stack.back();
    stack.pop_back();
    order.push_back(i);
    const amk_task_t& t = tasks[i];
    if (t.cu != AMK_CU_INLINE && t.seq + 1 < qlen[t.cu]) {
      const int nx = queue[t.cu][t.seq + 1];
      if (--indeg[nx] == 0) stack.push_back(nx);
    }
    if (t.signal_counter >= 0 && --remaining[t.signal_counter] == 0) {
      for (int wt : waiters[t.signal_counter])
        if (--indeg[wt] == 0) stack.push_back(wt);
    }
  }
  if ((int)order.size() != n) {
    // witness: walk "blocked by" edges from an unscheduled task until a repeat
    std::vector<char> done(n, 0);
    for (int i : order) done[i] = 1;
    int cur = -1;
    for (int i = 0; i < n; ++i)
      if (!done[i]) { cur = i; break; }
    std::vector<int> seen(n, -1);
    int step = 0;
    while (cur >= 0 && seen[cur] < 0) {
      seen[cur] = step++;
      const amk_task_t& t = tasks[cur];
      int nxt = -1;
      if (t.cu != AMK_CU_INLINE && t.seq > 0 && !done[queue[t.cu][t.seq - 1]]) nxt = queue[t.cu][t.seq - 1];
      for (int w = 0; nxt < 0 && w < t.n_wait; ++w)
        for (int p : producers[t.wait_counter[w]])
          if (!done[p]) { nxt = p; break; }
      cur = nxt;
    }
    return R.fail(AMK_CHECK_ACYCLIC, cur, -1,
                  "deadlock: %ld tasks can never run; cycle through task %ld (cycle length %ld)",
                  n - (long)order.size(), cur, cur >= 0 ? step - seen[cur] : 0);
  }

  // ---- 5. happens-before (vector clocks over queues): every read of a region
  //         written in this launch must be ordered after all its writers -------
  BufIds ids{s.L};
  const int nb = ids.count();
  std::vector<int> buf_size(nb, 0);
  for (int i = 0; i <= 2 * s.L; ++i) buf_size[ids.x(i)] = s.H;
  for (int l = 0; l < s.L; ++l) {
    buf_size[ids.q(l)] = s.q_units;
    buf_size[ids.kv(l)] = 2 * s.nkv * s.half;
    buf_size[ids.part(l)] = s.nkv * s.nsplit;
    buf_size[ids.o(l)] = s.nq * s.hd;
    buf_size[ids.a(l)] = s.I;
  }
  buf_size[ids.logits()] = s.V;
  buf_size[ids.argp()] = n_lm;
  buf_size[ids.next()] = 1;

  struct W { int lo, hi, task; };
  std::vector<std::vector<W>> writers(nb);
  std::vector<Access> rd, wr;
  for (int i = 0; i < n; ++i) {
    accesses(s, ids, tasks[i], &rd, &wr);
    for (auto& a : wr) writers[a.buf].push_back({a.lo, a.hi, i});
  }
  // exactly-once outputs: writer intervals of each written buffer tile it.
  // Attention partials are scratch of the split schedule: required only
  // where some task reads them.
  std::vector<char> read_any(nb, 0);
  for (int i = 0; i < n; ++i) {
    accesses(s, ids, tasks[i], &rd, &wr);
    for (auto& a : rd) read_any[a.buf] = 1;
  }
  for (int b = 0; b < nb; ++b) {
    auto& v = writers[b];
    if (b == ids.x(0)) {
      if (!v.empty()) return R.fail(AMK_CHECK_OUTPUT, v[0].task, -1, "task %ld writes the embedding input", v[0].task);
      continue;
    }
    if ((ids.is_part(b) || ids.is_o(b)) && v.empty() && !read_any[b]) continue;
    std::sort(v.begin(), v.end(), [](const W& a, const W& c) { return a.lo < c.lo; });
    int at = 0;
    for (auto& w : v) {
      if (w.lo < at) return R.fail(AMK_CHECK_OUTPUT, w.task, -1, "task %ld rewrites a region of buffer %ld", w.task, b);
      if (w.lo > at) return R.fail(AMK_CHECK_OUTPUT, w.task, -1, "buffer %ld region [%ld, ...) is never written", b, at);
      at = w.hi;
    }
    if (at != buf_size[b])
      return R.fail(AMK_CHECK_OUTPUT, -1, -1, "buffer %ld written up to %ld only", b, at);
  }

  // vector clocks: vc[c] = highest queue position on queue c that happened
  // before; each inline task gets a virtual queue n_cu + k of its own
  std::vector<int> vq(n, -1);
  int n_inline = 0;
  for (int i = 0; i < n; ++i)
    if (tasks[i].cu == AMK_CU_INLINE) vq[i] = n_cu + n_inline++;
  const int W = n_cu + n_inline;
  auto qof = [&](int i) { return tasks[i].cu == AMK_CU_INLINE ? vq[i] : tasks[i].cu; };
  std::vector<int32_t> q_vc((size_t)n_cu * W, -1);          // clock of each queue's last task
  std::vector<int32_t> ctr_vc((size_t)n_counters * W, -1);  // join of each counter's producers
  std::vector<int32_t> vc(W);
  for (int i : order) {
    const amk_task_t& t = tasks[i];
    if (t.cu == AMK_CU_INLINE) std::fill(vc.begin(), vc.end(), -1);
    else std::copy(q_vc.begin() + (size_t)t.cu * W, q_vc.begin() + (size_t)(t.cu + 1) * W, vc.begin());
    for (int w = 0; w < t.n_wait; ++w) {
      const int32_t* cv = &ctr_vc[(size_t)t.wait_counter[w] * W];
      for (int c = 0; c < W; ++c) vc[c] = std::max(vc[c], cv[c]);
    }
    vc[qof(i)] = t.seq;
    // reads
    accesses(s, ids, t, &rd, &wr);
    for (auto& a : rd) {
      for (auto& w : writers[a.buf]) {
        if (w.hi <= a.lo || w.lo >= a.hi) continue;
        if (w.task == i) continue;
        const amk_task_t& wt = tasks[w.task];
        if (vc[qof(w.task)] < wt.seq) {
          const int rule = ids.is_kv(a.buf) ? AMK_CHECK_KV_ORDER : AMK_CHECK_RACE;
          return R.fail(rule, i, w.task, "task %ld reads buffer %ld before writer task %ld is ordered", i, a.buf,
                        w.task);
        }
      }
    }
    if (t.cu != AMK_CU_INLINE) std::copy(vc.begin(), vc.end(), q_vc.begin() + (size_t)t.cu * W);
    if (t.signal_counter >= 0) {
      int32_t* cv = &ctr_vc[(size_t)t.signal_counter * W];
      for (int c = 0; c < W; ++c) cv[c] = std::max(cv[c], vc[c]);
    }
  }
  return true;
}

}  // namespace amk
