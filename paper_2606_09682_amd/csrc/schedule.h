// Host-side lowering of one decode step into per-CU task queues, and the
// static check that must accept a schedule before it is launched.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/amk.h"

namespace amk {

// Largest number of GEMV output rows one task may own: the kernel keeps one
// fp32 partial per row and streaming wave in LDS.
constexpr int kMaxJobsPerTask = 1024;
// Largest number of position splits per KV head (one combine lane per split).
constexpr int kMaxAttnSplits = 64;
// Counters a wide stage signals (task i counter i mod k); its consumers wait
// on all of them, so the producers' increments spread over k counter lines.
constexpr int kStageCounters = 4;

// Derived shape of a validated config.
struct Shape {
  int H = 0, L = 0, nq = 0, nkv = 0, hd = 0, I = 0, V = 0, max_seq = 0;
  int fmt = 0, tied = 0;
  int qgroup = 0;        // W4A16: input columns per scale (0 for the other formats)
  int group = 0;         // query heads per KV head
  int half = 0;          // hd / 2: RoPE row pairs per head
  int units = 0;         // (nq + 2 nkv) * half: q/k/v row-pair units
  int gunits = 0;        // (group + 2) * half: units of one KV group
  int q_units = 0;       // nq * half
  int npg = 0;           // QKV tasks per KV group
  int nsplit = 0;        // attention position splits per KV head (long schedule)
  int max_jobs = 0;      // GEMV rows per task cap
  int short_context = 0; // steps with pos + 1 <= short_context use the short schedule
  int tiny_context = 0;  // steps with pos + 1 <= tiny_context use the tiny schedule
  int assign = 0;        // AMK_ASSIGN_ROUND_ROBIN or AMK_ASSIGN_LPT
  float theta = 0.f, eps = 0.f;
};

// Number of tasks of a GEMV stage over `items` items of `jobs_per_item` rows:
// one per CU (at most one per item), more if the row cap requires.
int stage_tasks(int items, int jobs_per_item, int n_cu, int max_jobs);

// Validates the config (shape family, divisibility, 16-byte row alignment)
// and fills *s.  Returns AMK_OK or AMK_ERR_INVALID_ARGUMENT / _UNSUPPORTED
// with a message.
int derive_shape(const amk_config_t* cfg, const amk_tuning_t* tuning, int n_cu, Shape* s,
                 std::string* why);

struct Schedule {
  std::vector<amk_task_t> tasks;   // sorted by (cu, seq)
  std::vector<int32_t> queue_start;// n_cu + 1 offsets into tasks
  int n_counters = 0;
  int n_lm_slots = 0;              // argmax partial slots (one per LM-head task)
};

// Defaults of amk_tuning_t.short_context and .tiny_context (measured crossovers
// on the 8B shape: the tiny schedule gains about 140 us at pos 0 and breaks
// even near pos 6, where its per-task attention catches up with the saved
// stage).
constexpr int kDefaultShortContext = 256;
constexpr int kDefaultTinyContext = 6;

// Deterministic lowering of one decode step onto n_cu queues, schedule
// variant AMK_SCHEDULE_SHORT or AMK_SCHEDULE_LONG.
Schedule build_schedule(const Shape& s, int n_cu, int variant);

// Which head a QKV unit belongs to: kind 0 = query head `head`, 1 = K head,
// 2 = V head (head = KV group); i = row-pair index within the head.
struct UnitHead {
  int kind, head, i;
};
UnitHead unit_head(const Shape& s, int u);

// Static check (never throws).  Fills *rep; returns true iff accepted.
bool check_schedule(const Shape& s, int n_cu, const amk_task_t* tasks, int n_tasks,
                    int n_counters, amk_check_report_t* rep);

// Sorts tasks by (cu, seq) and computes queue offsets (tasks must be checked).
void finalize_queues(std::vector<amk_task_t>* tasks, int n_cu, std::vector<int32_t>* queue_start);

// Number of rows (jobs) a GEMV task computes; 0 for non-GEMV ops.
int task_jobs(const Shape& s, const amk_task_t& t);

}  // namespace amk
