/*
 * amk.h -- C ABI of the batch-1 Llama decode megakernel for MI355X (gfx950).
 *
 * One call of amk_decode_step() runs one forward pass of a Llama-family
 * decoder for one token as ONE persistent cooperative kernel launch, and
 * leaves the greedy next token on the device (paper §3, Figure fig:pipeline:
 * one launch = one forward pass = one token).  Work is split into tasks that
 * the host lowers into per-CU queues (paper §3 Layer 0 and Algorithm alg:sm);
 * tasks on different CUs order themselves only through monotonic counters
 * that producers increment with release semantics and consumers wait on with
 * acquire semantics (paper §4 "Synchronization model").  Before anything is
 * launched the host checks the schedule (paper §4 "The invariants validate()
 * proves", Table tab:checks); a rejected schedule is never launched.
 *
 * Model family (paper §6 "Architecture coverage"): bias-free projections,
 * full-rotary RoPE (rotate-half pairs i, i + head_dim/2), SiLU-SwiGLU MLP,
 * RMSNorm, grouped-query attention.  Weight formats (paper §5 "Quantized
 * generation"; dequantisation folded into the GEMV): bf16; W8A16 = int8
 * weights with one fp32 scale per output row (symmetric); W4A16 = int4
 * weights with one fp16 scale per output row and group of group_size input
 * columns (symmetric, round to nearest; layout under amk_linear_t).
 * Activations are fp32 throughout; the KV cache is bf16.
 *
 * Conventions for every function:
 *   - returns an int status (AMK_OK or a negative AMK_ERR_*), never throws or
 *     aborts across the ABI;
 *   - "device pointer" means memory of the device the handle was created on
 *     (hipMalloc or torch allocations); "host pointer" means ordinary memory;
 *   - nothing here frees or copies caller memory.
 *
 * Plain C; callers need no HIP headers.  The stream argument is a hipStream_t
 * passed as void* (NULL = the null stream).
 */
#ifndef AMK_H_
#define AMK_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AMK_ABI_VERSION 5

/* ---- status codes ------------------------------------------------------ */
enum {
  AMK_OK = 0,
  AMK_ERR_INVALID_ARGUMENT = -1,      /* NULL pointer, out-of-range token / pos, bad enum */
  AMK_ERR_UNSUPPORTED = -2,           /* shape or alignment outside the supported family */
  AMK_ERR_SCHEDULE_REJECTED = -3,     /* the static schedule check failed: nothing launched */
  AMK_ERR_OUT_OF_MEMORY = -4,
  AMK_ERR_DEVICE = -5,                /* a HIP runtime call failed */
  AMK_ERR_COOPERATIVE_UNSUPPORTED = -6, /* no cooperative launch, or too few co-resident workgroups */
  AMK_ERR_TIMEOUT = -7,               /* a device-side counter wait exceeded its deadline (sticky) */
  AMK_ERR_BAD_STATE = -8,             /* handle in an error state; call amk_reset() */
  AMK_ERR_ABORTED = -9,               /* the host abort flag stopped a launch (sticky) */
  AMK_ERR_NONFINITE = -10             /* a logit of the step was NaN: its next token is meaningless
                                         (sticky, like AMK_ERR_TIMEOUT) */
};

enum { AMK_WEIGHTS_BF16 = 0, AMK_WEIGHTS_W8A16 = 1, AMK_WEIGHTS_W4A16 = 2 };

/* ---- model description ------------------------------------------------- */
typedef struct {
  uint32_t abi_version;     /* must be AMK_ABI_VERSION */
  int32_t hidden;           /* H; H, intermediate and n_heads * head_dim are multiples of 16
                               (of 32 and of group_size under W4A16) */
  int32_t n_layers;         /* L */
  int32_t n_heads;          /* query heads */
  int32_t n_kv_heads;       /* KV heads; n_heads % n_kv_heads == 0, n_heads / n_kv_heads <= 8 */
  int32_t head_dim;         /* d; 64 or 128 */
  int32_t intermediate;     /* SwiGLU width I */
  int32_t vocab;            /* V */
  int32_t max_seq;          /* KV cache capacity in positions */
  float rope_theta;
  float rms_eps;
  int32_t tied_embeddings;  /* 1: the LM head is the embedding table (stays bf16) */
  int32_t weight_format;    /* AMK_WEIGHTS_BF16, _W8A16 or _W4A16 */
  int32_t device;           /* HIP device ordinal; -1 = current device */
  int32_t group_size;       /* W4A16: input columns per scale, a power of two in [32, 1024];
                               0 = 128.  Ignored by the other formats. */
} amk_config_t;

/* One projection y = W x, W row-major [out, in] (nn.Linear layout).  w and
 * scale are device pointers; w is 16-byte aligned.
 *   bf16:  w = bf16 [out][in]; scale = NULL.
 *   W8A16: w = int8 [out][in]; scale = fp32 [out] (4-byte aligned);
 *          W[r][k] = w[r][k] * scale[r].
 *   W4A16: w = uint8 [out][in / 2]: byte 4d + b of a row (b = 0..3) holds
 *          column 8d + b in its low nibble and column 8d + 4 + b in its high
 *          nibble, each nibble the code c in [-8, 7] stored as c + 8;
 *          scale = fp16 [out][in / group_size] (2-byte aligned);
 *          W[r][k] = c[r][k] * scale[r][k / group_size].
 *          (Word d of a row thus carries columns 8d .. 8d + 7, low nibbles
 *          first: two masks give four byte-sized codes each.) */
typedef struct {
  const void* w;
  const void* scale;
} amk_linear_t;

typedef struct {
  const void* attn_norm;  /* bf16 [H] */
  const void* mlp_norm;   /* bf16 [H] */
  amk_linear_t q;         /* [n_heads * d, H] */
  amk_linear_t k;         /* [n_kv_heads * d, H] */
  amk_linear_t v;         /* [n_kv_heads * d, H] */
  amk_linear_t o;         /* [H, n_heads * d] */
  amk_linear_t gate;      /* [I, H] */
  amk_linear_t up;        /* [I, H] */
  amk_linear_t down;      /* [H, I] */
} amk_layer_weights_t;

typedef struct {
  const void* embed;                 /* bf16 [V, H] device pointer */
  const void* final_norm;            /* bf16 [H] */
  amk_linear_t lm_head;              /* untied: [V, H] in the weight format; tied: w = NULL */
  const amk_layer_weights_t* layers; /* HOST array [n_layers] of device pointers; read during amk_create only */
} amk_weights_t;

/* Optional tuning; zero fields take defaults. */
typedef struct {
  int32_t attn_splits;      /* attention tasks per KV head (1..64); 0 = derived from the CU count */
  int32_t timeout_us;       /* deadline of one decode step in microseconds, on each workgroup's
                               clock from its start: a counter wait still unsatisfied past it
                               stops the launch with AMK_ERR_TIMEOUT; 0 = 2 s */
  int32_t max_rows_per_task;/* cap on rows of one GEMV task; 0 = 1024 */
  int32_t trace;            /* 1: record per-task timestamps (see amk_trace_copy) */
  int32_t short_context;    /* steps with pos + 1 <= short_context run the short-context schedule
                               (AMK_SCHEDULE_SHORT); 0 = 256; negative = never */
  int32_t tiny_context;     /* steps with pos + 1 <= tiny_context (at most AMK_TINY_MAX) run the
                               tiny-context schedule (AMK_SCHEDULE_TINY); 0 = 6; negative = never */
  int32_t queue_assign;     /* how the tasks of a stage are placed on the CU queues (paper §4,
                               ScheduleConfig sm_assignment): AMK_ASSIGN_ROUND_ROBIN (0) or
                               AMK_ASSIGN_LPT (1) */
} amk_tuning_t;

/* amk_tuning_t.queue_assign.  ROUND_ROBIN: task i of a stage of n tasks goes to
 * queue i mod n_cu (stages narrower than the grid start where the previous
 * narrow stage stopped).  LPT (longest processing time first): the tasks of a
 * stage, largest estimated cost first (bytes streamed plus a fixed per-task
 * cost), each go to the queue with the least estimated work so far. */
enum { AMK_ASSIGN_ROUND_ROBIN = 0, AMK_ASSIGN_LPT = 1 };

/* Largest tiny_context: the tiny schedule's attention keeps every position in registers. */
#define AMK_TINY_MAX 8

typedef struct amk_handle_s* amk_handle_t;

/* ---- lifecycle ----------------------------------------------------------- */

/* Validate the config and weight pointers, build the per-CU task schedule for
 * the device, check it (acyclic, wait-satisfiable, deadlock-free queue order,
 * race-free reads and writes, every output produced exactly once), and upload
 * the schedule tables, counters, scratch activations and the RoPE table.
 * Weight pointers are BORROWED: they must stay valid and unchanged until
 * amk_destroy(); nothing is copied or repacked.  tuning may be NULL.
 * All three schedule variants (AMK_SCHEDULE_TINY, _SHORT and _LONG) are built
 * and checked; each step runs the one its position selects
 * (amk_tuning_t.tiny_context and .short_context).
 * On failure *out is set to NULL and nothing stays allocated. */
int amk_create(const amk_config_t* cfg, const amk_weights_t* w, const amk_tuning_t* tuning,
               amk_handle_t* out);

/* Enqueue one decode step on `stream` (asynchronous: returns before the GPU
 * finishes).  Reads token `token` at position `pos`, reads KV positions
 * 0..pos-1 and appends position pos (all layers), writes all `vocab` logits
 * and the greedy next token (lowest index among equal maxima) into the
 * handle's device slot (amk_next_token_ptr).
 *   kv_cache: device pointer, 256-byte aligned, bf16
 *             [n_layers][2 (K, V)][n_kv_heads][max_seq][head_dim]
 *             (every row then fills whole cache lines: rows appended by this
 *             step never share a line with rows another workgroup reads)
 *   logits:   device pointer, 16-byte aligned, fp32 [vocab]
 * Errors: AMK_ERR_INVALID_ARGUMENT for token outside [0, vocab), pos outside
 * [0, max_seq), a misaligned pointer, or a kv_cache / logits pointer that is
 * not device memory of the handle's device (host, pinned or another
 * device's memory is refused before any launch); a sticky device error of an
 * earlier step (AMK_ERR_TIMEOUT / AMK_ERR_ABORTED / AMK_ERR_NONFINITE,
 * visible once that step finished) is returned and nothing is launched until
 * amk_reset().  One handle must not be driven from two streams at once: a
 * step enqueued on a different stream than the previous step's while that
 * stream still has work queued (the previous step, or anything after it)
 * returns AMK_ERR_BAD_STATE and launches nothing (synchronise the old stream
 * before switching). */
int amk_decode_step(amk_handle_t h, int32_t token, int32_t pos, void* kv_cache, float* logits,
                    void* stream);

/* Synchronise the device, free everything the handle owns.  NULL is a no-op. */
int amk_destroy(amk_handle_t h);

/* ---- no-allocation variant --------------------------------------------------- */

/* Bytes of the library's static device array that amk_create_static uses. */
#define AMK_STATIC_SCRATCH_BYTES (64u << 20)

/* For callers that cannot allocate device memory (code running under HIP
 * graph capture, serving loops and harnesses that forbid hipMalloc): the same
 * handle as amk_create, with the same checks, schedules and kernels, but all
 * the device memory the handle owns (task tables, counters, activations, the
 * RoPE table and the status words) lives in one static device array of
 * AMK_STATIC_SCRATCH_BYTES per device, which every process that uses the
 * library on a device holds until it ends.  Calls no hipMalloc, hipHostMalloc
 * or hipFree (the schedule is built in ordinary host memory and copied in with
 * hipMemcpy; the array is cleared with hipMemset).
 * Limits: a model whose tables and scratch need more than
 * AMK_STATIC_SCRATCH_BYTES (the Llama-3-8B shape with an 8194-position cache
 * needs about 35 MiB) fails with AMK_ERR_OUT_OF_MEMORY and a message on stderr.  One
 * array per device holds one handle: while a static handle lives, another
 * amk_create_static on that device fails with AMK_ERR_BAD_STATE; destroy the
 * first one before creating the next (the new handle clears what it uses;
 * two handles would race on the same counters and scratch).  Because the
 * status words are device memory, amk_decode_step on a static handle does not
 * return an earlier step's sticky error (amk_get_status, which waits for the
 * stream, does) and amk_set_abort returns AMK_ERR_UNSUPPORTED; every counter
 * wait is still bounded by the deadline.  amk_destroy and every other function work as for amk_create. */
int amk_create_static(const amk_config_t* cfg, const amk_weights_t* w, const amk_tuning_t* tuning,
                      amk_handle_t* out);

/* ---- helpers --------------------------------------------------------------- */

/* Bytes of the KV cache amk_decode_step expects for cfg (0 for an invalid cfg). */
size_t amk_kv_cache_bytes(const amk_config_t* cfg);

/* Device pointer to the int32 next-token slot written by every step. */
const int32_t* amk_next_token_ptr(amk_handle_t h);

/* Copy the next token written by the last enqueued step into *dst (host
 * memory): enqueues the copy on `stream` and waits for it. */
int amk_copy_next_token(amk_handle_t h, int32_t* dst, void* stream);

/* Synchronise the handle's last stream and return its sticky device status
 * (AMK_OK, AMK_ERR_TIMEOUT, AMK_ERR_ABORTED, AMK_ERR_NONFINITE). */
int amk_get_status(amk_handle_t h);

/* Clear a sticky error: waits for the device, zeroes the counters and
 * restarts the epoch.  The KV cache content is the caller's business. */
int amk_reset(amk_handle_t h);

/* Raise (value 1) or clear (value 0) the host abort flag.  A launch whose
 * workgroup is spinning on a counter polls the flag about every hundred spins
 * and, once it sees it, stops every workgroup and records AMK_ERR_ABORTED
 * (sticky).  The flag lives in host-mapped memory, so it can be raised while
 * a step runs. */
int amk_set_abort(amk_handle_t h, int32_t value);

const char* amk_status_string(int status);

/* Number of uint64 timestamps per task in a trace record. */
#define AMK_TRACE_FIELDS 8
enum {
  AMK_TRACE_WAIT_BEGIN = 0, /* sync wave starts waiting on the task's counters */
  AMK_TRACE_WAIT_END = 1,   /* counters satisfied (after the acquire) */
  AMK_TRACE_INPUT_READY = 2,/* input activation in LDS, streaming waves released */
  AMK_TRACE_COMPUTE_END = 3,/* every wave finished the task's compute */
  AMK_TRACE_SIGNALLED = 4,  /* results published, counter incremented */
  AMK_TRACE_PUBLISHED = 5,  /* result stores issued, before the release fence */
  AMK_TRACE_CHAINED = 6,    /* inline task run by this task finished and signalled (0: none ran) */
  AMK_TRACE_SATISFIED = 7   /* counters observed satisfied, before the acquire fence */
};

/* Copy the per-task timestamps of the last finished step of a handle created
 * with tuning.trace = 1 into dst[capacity] (host memory), AMK_TRACE_FIELDS
 * uint64 per task, tasks in amk_schedule_export() order of the schedule
 * variant that step ran (*variant, may be NULL).  Timestamps are the device's
 * constant 100 MHz wall clock.  Synchronises the handle's stream.  *n_tasks
 * receives the task count.  AMK_ERR_BAD_STATE if tracing is off or nothing
 * was launched. */
int amk_trace_copy(amk_handle_t h, uint64_t* dst, int64_t capacity, int32_t* n_tasks, int32_t* variant);

/* ---- measurement --------------------------------------------------------- */

/* Streaming-read reference: enqueue on `stream` one read of `bytes` of device
 * memory at `buf` by `blocks` workgroups of 512 threads (16 bytes per thread
 * and load, grid-stride, a few loads in flight per thread), each thread
 * leaving an XOR of what it read in sink[thread] (a device buffer of
 * blocks * 512 uint32, owned by the caller, so the reads are not optimised
 * away).  Asynchronous; time it with events on the same stream.  The read
 * rate of a large buffer is this device's practical HBM peak, which the
 * decode step's achieved bandwidth is compared with.
 * Errors: AMK_ERR_INVALID_ARGUMENT for NULL pointers, bytes not a positive
 * multiple of 16, buf not 16-byte aligned or blocks outside [1, 65536];
 * AMK_ERR_DEVICE for a launch failure. */
int amk_read_probe(const void* buf, int64_t bytes, int32_t blocks, uint32_t* sink, void* stream);

/* ---- schedule introspection (CPU only, no device needed) -------------------- */

/* Schedule variants.  All compute the same step; they differ in where the
 * attention runs.  SHORT: the last QKV task of each KV group to finish runs
 * that group's whole attention inline (no attention stage).  LONG: the
 * attention of each KV group is split over `attn_splits` position ranges on
 * as many queues (flash-decoding style), and the last split of a group to
 * finish merges the splits inline.  TINY (at most AMK_TINY_MAX positions):
 * every O task computes the attention of all query heads itself, straight
 * from q and the KV cache, and waits only for the QKV stage. */
enum { AMK_SCHEDULE_SHORT = 0, AMK_SCHEDULE_LONG = 1, AMK_SCHEDULE_TINY = 2 };

/* Operations of the task graph, in the order of one layer.
 * QKV units: unit u is the RoPE row pair (i, i + d/2), i = u % (d/2), of head
 * slot u / (d/2); head slots are numbered KV group by KV group, each group g
 * holding its `group` query heads g*group .. g*group+group-1, then K head g,
 * then V head g.  A QKV task's units lie in one KV group, `aux`. */
enum {
  AMK_OP_QKV = 1,      /* RMSNorm + q/k/v GEMV of units [begin, end) of KV group `aux` + RoPE + KV append */
  AMK_OP_ATTN = 2,     /* attention of KV group `aux` over position split `begin` of `end` splits; queued
                          splits leave partial results, the inline task (begin 0, end 1) the output */
  AMK_OP_COMBINE = 3,  /* merge the position splits of query heads [begin, end) (inline, see below) */
  AMK_OP_O = 4,        /* rows [begin, end) of x1 = x + Wo o; aux 1: o is first computed by the task
                          itself from q and the KV cache (tiny schedule) */
  AMK_OP_GATEUP = 5,   /* rows [begin, end) of a = silu(Wg h2) * (Wu h2), h2 = RMSNorm(x1) */
  AMK_OP_DOWN = 6,     /* rows [begin, end) of x2 = x1 + Wd a */
  AMK_OP_LMHEAD = 7,   /* rows [begin, end) of logits = W_lm RMSNorm(x); argmax partial slot `aux` */
  AMK_OP_ARGMAX = 8    /* reduce argmax partial slots [begin, end) into the next token */
};

#define AMK_MAX_WAITS 4
/* Queue value of an inline task: it runs on no queue of its own but at the
 * end of whichever producer of its single wait counter increments that
 * counter last (that producer's chain_counter names the inline task's
 * signal counter).  Used for the ATTN of a KV group after its QKV tasks
 * (short schedule) and for the COMBINE of its attention splits (long). */
#define AMK_CU_INLINE (-1)

/* Fixed-size task descriptor (64 bytes), the unit the device walks.  A task
 * waits until, for every i < n_wait, counter wait_counter[i] has been
 * incremented wait_count[i] times in this launch, then runs, then increments
 * signal_counter (if >= 0) once.  If chain_counter >= 0 and this task's
 * increment of signal_counter is the last of the launch, it then runs the
 * inline task waiting on signal_counter, which increments chain_counter. */
typedef struct {
  uint16_t op;
  uint16_t layer;
  int32_t cu;          /* queue (workgroup index) that runs the task, or AMK_CU_INLINE */
  int32_t seq;         /* position inside that queue, 0-based, contiguous (0 for inline tasks) */
  int32_t begin, end;  /* op-specific range, see AMK_OP_* */
  int16_t aux;         /* op-specific */
  int16_t n_wait;
  int32_t wait_counter[AMK_MAX_WAITS];
  int32_t wait_count[AMK_MAX_WAITS];
  int32_t signal_counter;
  int32_t chain_counter;
} amk_task_t;

typedef struct {
  int32_t ok;            /* 1 accepted, 0 rejected */
  int32_t rule;          /* first failed rule, AMK_CHECK_* */
  int32_t task;          /* offending task index (or -1) */
  int32_t other;         /* second task / counter involved (or -1) */
  int32_t n_tasks, n_counters, n_edges;
  char message[256];
} amk_check_report_t;

enum {
  AMK_CHECK_OK = 0,
  AMK_CHECK_WELL_FORMED = 1,   /* bad op, counter index, queue index, range or arity */
  AMK_CHECK_CAPACITY = 2,      /* more waits than AMK_MAX_WAITS, rows over the LDS budget */
  AMK_CHECK_WAIT_SATISFIABLE = 3, /* count < 1, counter without producer, count > producers */
  AMK_CHECK_ALL_JOIN = 4,      /* a multi-producer counter waited on with count != producers */
  AMK_CHECK_ACYCLIC = 5,       /* cycle in producer->consumer edges plus per-queue order edges */
  AMK_CHECK_QUEUE_ORDER = 6,   /* a consumer queued before its producer on the same CU */
  AMK_CHECK_RACE = 7,          /* a read not ordered after every writer of the region it reads */
  AMK_CHECK_KV_ORDER = 8,      /* a KV-cache read not ordered after this pass's append */
  AMK_CHECK_OUTPUT = 9,        /* an output region written twice or never */
  AMK_CHECK_INLINE = 10        /* an inline task or a chain counter that does not pair up */
};

/* Number of tasks / counters schedule `variant` (AMK_SCHEDULE_*) of cfg has
 * on n_cu queues (after validating cfg; tuning may be NULL).  Returns a
 * status. */
int amk_schedule_size(const amk_config_t* cfg, const amk_tuning_t* tuning, int32_t n_cu, int32_t variant,
                      int32_t* n_tasks, int32_t* n_counters);

/* Lower cfg onto n_cu queues into tasks[cap] (cap >= n_tasks). */
int amk_schedule_export(const amk_config_t* cfg, const amk_tuning_t* tuning, int32_t n_cu, int32_t variant,
                        amk_task_t* tasks, int32_t cap, int32_t* n_tasks, int32_t* n_counters);

/* Check an arbitrary task array for cfg on n_cu queues with n_counters
 * counters.  Never fails for a bad schedule: the verdict is in *report
 * (report->ok); the return value is AMK_OK unless the arguments themselves
 * are unusable.  Accepted iff amk_create would launch it.  The rules do not
 * depend on the variant. */
int amk_schedule_check(const amk_config_t* cfg, const amk_tuning_t* tuning, int32_t n_cu,
                       const amk_task_t* tasks, int32_t n_tasks, int32_t n_counters,
                       amk_check_report_t* report);

/* Validate cfg and build + check both schedule variants for n_cu queues (no
 * device). */
int amk_check_config(const amk_config_t* cfg, int32_t n_cu);

#ifdef __cplusplus
}
#endif
#endif /* AMK_H_ */
