/*
 * dstack.h -- C ABI of an MI355X-native implementation of the D-STACK hot
 * path (Dhakal, Kulkarni, Ramakrishnan, "D-STACK: High Throughput DNN
 * Inference by Effective Multiplexing and Spatio-Temporal Scheduling of
 * GPUs", arxiv 2304.13541).
 *
 * The paper's problem (Sec. 1, Sec. 5, Sec. 6): give each DNN only the GPU
 * share beyond which its latency stops improving (its "Knee"), choose the
 * batch that maximises efficacy under its SLO, and run several models at
 * once without over-subscribing the GPU.  Here a GPU share is a CU-masked
 * HIP stream ("partition") whose CUs are counted in slots: slot j is the
 * j-th CU of every one of the 8 XCDs, so a partition of s slots owns 8*s of
 * the 256 CUs, spread evenly over the XCDs.
 *
 * Conventions
 *  - Every call returns dstack_status; results go through out-parameters.
 *    No C++ exception crosses this boundary.
 *  - DSTACK_E_INVALID: a NULL pointer, a fraction <= 0, > 1 or NaN, a batch
 *    < 1 or above the model's maximum, a slot range outside 0..32, a size
 *    that does not match.  DSTACK_E_UNSUPPORTED: unknown architecture or a
 *    shape a kernel does not handle.  DSTACK_E_HIP: a HIP runtime error
 *    (its text is in dstack_last_error()).  DSTACK_E_STATE: a second
 *    concurrent call on the same (model, partition) pair.
 *  - Handles are created and destroyed by the caller.  The library owns
 *    weights, workspaces and the masked streams.  Device pointers passed in
 *    (inputs, outputs) stay owned by the caller.
 *  - dstack_last_error() is thread-local text for the last non-OK status.
 */
#ifndef DSTACK_H
#define DSTACK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DSTACK_OK = 0,
  DSTACK_E_INVALID = -1,
  DSTACK_E_UNSUPPORTED = -2,
  DSTACK_E_HIP = -3,
  DSTACK_E_OOM = -4,
  DSTACK_E_INFEASIBLE = -5,
  DSTACK_E_STATE = -6
} dstack_status;

#define DSTACK_TOTAL_SLOTS 32
#define DSTACK_CUS_PER_SLOT 8
#define DSTACK_MAX_SWEEP 32
#define DSTACK_MAX_BATCHES 8
#define DSTACK_MAX_MODELS 16
#define DSTACK_MAX_JOBS 512

typedef struct dstack_partition_s* dstack_partition;
typedef struct dstack_model_s* dstack_model;

/* Text of the last non-OK status on the calling thread ("" if none). */
const char* dstack_last_error(void);

/* ------------------------------------------------------------------ */
/* Partitions (CU-masked streams)                                      */
/* ------------------------------------------------------------------ */
/* The paper confines each model to a share of the SMs with MPS
 * (Sec. 3.1); here the share is a CU mask on a HIP stream.
 *
 * dstack_fraction_to_slots: slots = clamp(floor(32*f + 1/2), 1, 32).
 *   Host only.  E_INVALID for f <= 0, f > 1 or NaN.
 * dstack_partition_create: a partition of that many slots starting at slot 0.
 * dstack_partition_create_at: slots [slot_offset, slot_offset + n_slots).
 * dstack_partition_create_mask: any non-empty set of slots (bit j = slot j),
 *   as produced by dstack_schedule's per-job slot masks.
 * The partition owns one new HIP stream (default priority) whose CU mask
 * has bits 8j..8j+7 set for every slot j (mask bit i selects CU i/8 of XCD
 * i%8).  Several partitions may overlap; keeping concurrent ones disjoint
 * is the scheduler's job.
 * At most 4 partitions may be live at once in a process (a CU-masked stream
 * has a hardware queue of its own; a run with five live masked streams stopped
 * making progress on MI355X, runs with four completed).  A fifth create call
 * returns E_UNSUPPORTED before any stream is made.  The library's own calls
 * count too: a knee sweep or search needs 1 free, dstack_switch_probe 2,
 * dstack_serve one per model.
 * dstack_partition_query: n_cu, the 8 CU-mask words and the hipStream_t (as
 *   void*, usable with torch.cuda.ExternalStream).  Any out pointer may be
 *   NULL.
 * dstack_partition_count: live partitions and the limit (either may be NULL).
 * dstack_partition_destroy waits for the partition's stream, frees the
 *   workspaces that models hold for it (activations, split-K slices,
 *   captured graphs) and destroys the stream. */
dstack_status dstack_fraction_to_slots(double cu_fraction, int* slots);
dstack_status dstack_partition_create(double cu_fraction, dstack_partition* out);
dstack_status dstack_partition_create_at(int slot_offset, int n_slots, dstack_partition* out);
dstack_status dstack_partition_create_mask(uint32_t slot_mask, dstack_partition* out);
dstack_status dstack_partition_query(dstack_partition p, int* n_cu, uint32_t mask_words[8], void** hip_stream);
dstack_status dstack_synchronize(dstack_partition p);
dstack_status dstack_partition_count(int* live, int* max_live);
void dstack_partition_destroy(dstack_partition p);

/* Probe (verification of the slot -> CU mapping): launches n_blocks
 * one-wave workgroups on the partition's stream; each records its hardware
 * XCC id and HW_ID register into host_out[2*i], host_out[2*i+1].  With
 * via_graph != 0 the launch is captured into a HIP graph and the graph is
 * launched on the partition's stream (forward passes run that way).  Blocks
 * until done.  n_blocks in 1..65536; host_out holds 2*n_blocks words. */
dstack_status dstack_probe_cu_ids(dstack_partition p, int n_blocks, int via_graph, uint32_t* host_out);

/* ------------------------------------------------------------------ */
/* Models                                                              */
/* ------------------------------------------------------------------ */
/* arch: "tinycnn", "resnet50", "mobilenetv2", "vgg19", "lstm2".
 * Weights are drawn from `seed` (Sec. 3 uses trained models; here
 * random-weight models of the same architecture):
 *   tensor t uses the splitmix64 stream whose state starts at
 *   seed ^ (0x9E3779B97F4A7C15 * (t + 1)); u = (next >> 11) * 2^-53, with
 *   u = 0 replaced by 1; conv/FC weights are He-normal (std sqrt(2/fan_in),
 *   Box-Muller pairs in order, 2*pi as its fp64 value); LSTM tensors are
 *   (2u - 1)/32; conv/FC biases are 0; every value is rounded to bf16 RNE
 *   from fp64.  Tensor order is layer order, weight before bias
 *   (ResNet block: conv1, conv2, conv3, downsample).  Logical layouts:
 *   conv [K][R][S][C], depthwise [C][3][3], FC [out][in], LSTM [4H][in]
 *   with gate order i, f, g, o.  BN layers have gamma 1, beta 0, mean 0,
 *   var 1, eps 1e-5 (folded into per-channel fp32 scale/shift).
 *   "bert" / "bert_long": BERT-base encoders (Sec. 4.4's transformer) on 20
 *   / 40 tokens, 2 classes: word [30522][768], position [512][768] and
 *   type [2][768] embeddings, then per layer q|k|v [2304][768] + bias,
 *   output [768][768] + bias, feed-forward [3072][768] + bias and
 *   [768][3072] + bias, then pooler [768][768] + bias and classifier
 *   [2][768] + bias; all N(0, 0.02^2) (the normal rule with fan-in 5000);
 *   layer norms gain 1, bias 0, eps 1e-12. */
typedef struct {
  char arch[16];
  int is_lstm;              /* 0: image classifier or transformer, 1: LSTM */
  int max_batch;            /* largest batch dstack_infer accepts */
  int in_h, in_w, in_c;     /* CNN: per-item input [H][W][C] bf16 NHWC */
  int seq_len, in_features; /* LSTM: input [T][batch][in_features] bf16 */
  int out_features;         /* CNN, transformer: classes (fp32 logits); LSTM: hidden (fp32 h) */
  int num_tensors;
  int64_t num_params;
  int num_kernels;          /* kernel launches per forward */
  double flops_per_item;    /* algorithmic FLOPs (2 per MAC) per inference */
  double mfma_flops_per_item; /* of which in MFMA convolution/GEMM kernels */
  double weight_bytes;      /* bf16 weights read per forward */
  int input_tokens;         /* 1: transformer, input int32 token ids [batch][seq_len]
                               (ids outside the vocabulary read its last row) */
} dstack_model_info;

dstack_status dstack_model_load(const char* arch, uint64_t seed, dstack_model* out);
dstack_status dstack_model_query(dstack_model m, dstack_model_info* out);
/* Copy tensor `tensor_index` (bf16 bits, logical layout) to host memory;
 * `bytes` must equal 2 * numel. */
dstack_status dstack_model_export_params(dstack_model m, int tensor_index, void* host_dst, size_t bytes);
void dstack_model_destroy(dstack_model m);

/* Host-only generation of one tensor of an architecture (same bits as
 * dstack_model_load), without a device.  With host_dst == NULL only
 * *numel is filled. */
dstack_status dstack_generate_params(const char* arch, uint64_t seed, int tensor_index, void* host_dst,
                                     size_t bytes, int64_t* numel);

/* ------------------------------------------------------------------ */
/* Inference                                                           */
/* ------------------------------------------------------------------ */
/* Batched forward pass, asynchronous on the partition's stream.
 *   CNN:  d_in = [batch][H][W][3] bf16 NHWC, d_out = [batch][classes] fp32.
 *   LSTM: d_in = [50][batch][512] bf16,       d_out = [50][batch][1024] fp32
 *         (the second layer's h for every step).
 * Activations between layers are bf16 (fp32 accumulation; LSTM cell state
 * and h in fp32).  Workspace is per (model, partition) and is allocated on
 * the first call for that pair. */
dstack_status dstack_infer(dstack_model m, int batch, const void* d_in, void* d_out, dstack_partition p);

/* Transformer models only (Sec. 4.4's BERT): the forward up to the end of
 * encoder layer `layer` (0: the embeddings and their layer norm; 1..12: the
 * output of that encoder layer, after its second layer norm; < 0: the
 * last), run eagerly on the partition's stream, and that hidden state, bf16
 * [batch][T][768], copied to the caller's d_hidden.  E_UNSUPPORTED for the
 * other architectures, E_INVALID for a layer past the last.  Asynchronous;
 * same workspace rules as dstack_infer. */
dstack_status dstack_infer_hidden(dstack_model m, int batch, const void* d_in, int layer, void* d_hidden,
                                  dstack_partition p);

/* Per-kernel timing of one forward: fills up to max_layers entries with
 * the elapsed device time (ms, HIP events around each kernel on the
 * partition's stream), the kernel class (0 MFMA conv/GEMM, 1 depthwise,
 * 2 FC, 3 LSTM step, 4 pool/glue, 5 direct RGB stem conv, 6 fused expand
 * + depthwise) and its algorithmic FLOPs and bytes.
 * Synchronises the partition. */
typedef struct {
  int kind;
  float ms;
  double flops;
  double bytes;
  int gemm_m, gemm_n, gemm_k;  /* GEMM view of MFMA kernels (pixels, out channels, depth); else 0 */
} dstack_layer_time;
dstack_status dstack_profile_layers(dstack_model m, int batch, const void* d_in, void* d_out, dstack_partition p,
                                    dstack_layer_time* out, int max_layers, int* n_layers);

/* Launch shapes of one forward (the per-kernel parallelism N_i of Sec.
 * 4.3's analytical model, taken from this library's own kernels): one entry
 * per timed unit of dstack_profile_layers, in the same order, with the
 * unit's kernel class, its number of kernel launches, the workgroups of its
 * largest launch and how many of those workgroups one CU holds at once
 * (occupancy from the kernel's registers and LDS), plus its algorithmic
 * FLOPs and bytes.  Nothing is launched and d_in / d_out (the buffers a
 * forward would use, as in dstack_infer) are neither read nor written: the
 * forward's host logic runs with kernel launches recorded instead (launch
 * plans use the partition's CU count).  Needs a GPU (occupancy queries);
 * fills at most max_units entries. */
typedef struct {
  int kind;
  int launches;
  int64_t workgroups;
  int blocks_per_cu;
  int pad;
  double flops;
  double bytes;
} dstack_kernel_shape;
dstack_status dstack_kernel_shapes(dstack_model m, int batch, const void* d_in, void* d_out, dstack_partition p,
                                   dstack_kernel_shape* out, int max_units, int* n_units);

/* ------------------------------------------------------------------ */
/* Knee sweep (Sec. 3.2 measurement; Sec. 4.3 Eq. first_order_derivative;  */
/* Sec. 5 Eq. efficiencySquareLatency)                                 */
/* ------------------------------------------------------------------ */
/* For each fraction: a partition of dstack_fraction_to_slots(f) slots,
 * `warmup` untimed forwards, then `reps` forwards each timed with HIP
 * events; latency = median, rounded half-up to whole microseconds.
 * Efficacy eta = batch / (L^2 * slots); knee = argmax eta (exact integer
 * comparison, ties to fewer slots); deployed = min(32, knee + 2 slots),
 * the paper's 5-10% over-provisioning.  reps >= 1, n in 1..32. */
typedef struct {
  int n;
  int batch;
  int slots[DSTACK_MAX_SWEEP];
  int n_cu[DSTACK_MAX_SWEEP];
  int64_t latency_us[DSTACK_MAX_SWEEP];  /* median, whole us */
  double latency_us_exact[DSTACK_MAX_SWEEP];
  double p99_us[DSTACK_MAX_SWEEP];
  int knee_index;
  int knee_slots;
  int deployed_slots;
} dstack_knee_result;

dstack_status dstack_knee_sweep(dstack_model m, int batch, const double* fractions, int n, int warmup, int reps,
                                dstack_knee_result* out);

/* Knee search for a model without a profile (Sec. 3.6: it starts at a
 * nominal 30% and the knee is found from its latency by a binary search).
 * Reading: the search runs over the same ascending GPU% grid as the sweep
 * (candidate slot counts c[0..n)), with eta(s) = b / (L(s)^2 s) taken as
 * unimodal over it (at single-slot steps latency falls in steps and eta has
 * local maxima).  It keeps an index interval [lo, hi] = [0, n - 1], probes
 * c[mid] and c[mid + 1] (mid = the last candidate <= start_slots first, then
 * (lo + hi) / 2, clamped into [lo, hi - 1]) and moves lo = mid + 1 when
 * eta(c[mid + 1]) > eta(c[mid]) (exact 128-bit compare), else hi = mid,
 * until lo == hi; c[lo] is the knee.  Each candidate is measured at most
 * once; probe_slots/probe_latency_us list the measurements in order.
 *  - _table: latency_us[i] (> 0) stands in for the measurement at slots[i]
 *    (ascending, in 1..total); pure host; deployed = min(total, knee +
 *    overprov_slots).
 *  - live: candidates from `fractions` (ascending) as dstack_knee_sweep;
 *    each probe measures the median latency (integer us, rounded half up)
 *    of `reps` forwards after `warmup` on a fresh partition of the first s
 *    slots; total 32, over-provision 2; seconds = wall time of the search.
 *    start_slots 10 = 30%. */
#define DSTACK_MAX_PROBES 64
typedef struct {
  int batch;
  int knee_slots;
  int deployed_slots;
  int n_probes;
  int probe_slots[DSTACK_MAX_PROBES];
  int64_t probe_latency_us[DSTACK_MAX_PROBES];
  double seconds;
} dstack_knee_search_result;

dstack_status dstack_knee_search_table(int batch, const int* slots, const int64_t* latency_us, int n,
                                       int start_slots, int total, int overprov_slots,
                                       dstack_knee_search_result* out);
dstack_status dstack_knee_search(dstack_model m, int batch, const double* fractions, int n, int start_slots,
                                 int warmup, int reps, dstack_knee_search_result* out);

/* ------------------------------------------------------------------ */
/* Analytical DNN model (Sec. 4.3, Eqs. layer_num_ops,                  */
/* execution_time_per_layer, memory_latency,                           */
/* total_non_paralleizable_time, total_time_shrinking_kernel;          */
/* Eq. first_order_derivative), host only                              */
/* ------------------------------------------------------------------ */
/* A DNN of n_kernels kernels: kernel i has n_par[i] (N_i >= 0) parallel
 * operations of t_p[i] each, repeats reps[i] times (NULL: 1) and moves
 * data[i] bytes (NULL: no memory term).  On S CUs
 *   E_i  = N_i t_p / max(1, min(S, N_i)),
 *   E_m  = d_i / (M S)   (M = mem_bw_per_sm, bandwidth per CU; <= 0: none;
 *                         the printed d_i S / M is read as d_i / (M S), the
 *                         total bandwidth growing with S as the text says),
 *   W_se = batch_serial * sum_i R_i (t_np + E_m),
 *   E_t  = W_se + sum_i R_i E_i,
 * sums in kernel order, fp64.  dstack_knee_model_eval writes E_t for each of
 * the n_s candidates s_values[j] >= 1 into et_out and the index of the
 * knee, the first candidate with the least E_t^2 S (the largest
 * 1 / (E_t^2 S)).  Negative or non-finite N_i, t_p, R_i, d_i, t_np or
 * batch_serial -> E_INVALID.  Times are in any one unit. */
typedef struct {
  int n_kernels;
  int pad;
  const double* n_par;
  const double* t_p;
  const double* reps;
  const double* data;
  double t_np;
  double mem_bw_per_sm;
  double batch_serial;
} dstack_knee_model;
dstack_status dstack_knee_model_eval(const dstack_knee_model* m, const int* s_values, int n_s, double* et_out,
                                     int* knee_index);
/* The paper's synthetic kernel sequence (Eq. layer_num_ops): N_1 = p*b,
 * N_i = max(0, floor(N_{i-1} - p*b/kmax)) for i = 2..kmax (clamped at 0
 * once the work is used up), into n_out[kmax].  p >= 0, b >= 1,
 * kmax >= 1. */
dstack_status dstack_knee_model_sequence(int p, int b, int kmax, double* n_out);

/* GPU% change of a running model (Sec. 3.5).  A GPU% is a CU-masked stream
 * here, so a change creates a stream (no model reload: weights are shared).
 * The model runs at batch on the first from_slots slots (warmed up); then
 *  - cold: a partition of the first to_slots slots is created and its first
 *    forward (workspace allocation, graph capture) is run: create_us is the
 *    stream creation, cold_us creation through the first result (host clock);
 *  - active-standby: with that partition ready, `reps` times the active
 *    runs a batch and the host, on its completion, hands the next batch to
 *    the standby; standby_gap_us is the median (max: _max_us) device-clock
 *    time between the active's end and the standby's start;
 *  - from/to_latency_us: median of 5 forwards on each size.
 * Uses profiling buffers of the model (fixed input pattern). */
typedef struct {
  double create_us, cold_us, standby_gap_us, standby_gap_max_us, from_latency_us, to_latency_us;
} dstack_switch_result;

dstack_status dstack_switch_probe(dstack_model m, int batch, int from_slots, int to_slots, int reps,
                                  dstack_switch_result* out);

/* ------------------------------------------------------------------ */
/* Scheduling (pure host, deterministic, integer microseconds)          */
/* ------------------------------------------------------------------ */
/* Per model (Sec. 5.1, Eqs. max_batch_size, meet_slo, meet_half_slo):
 * choose (b, s) on the measured grid maximising eta = b/(L^2 s) subject to
 * b <= max_batch, L + C(b) <= SLO, L <= floor(SLO/2), where C(b) =
 * ceil(b*1e6/rate) if rate > 0 else 482*b us; ties: higher eta, fewer
 * slots, larger b.  None feasible: b = 1 (else the smallest batch), its
 * lowest-latency s (ties fewer), feasible = 0.  Deployed slots =
 * min(total, s + overprov).
 * Session plan (Sec. 6.1, 6.1.1): model i has jobs k = 0..ceil(T/SLO)-1 in
 * windows [k*SLO, min((k+1)*SLO, T)); EDF order (deadline, SLO, model, k);
 * even k earliest feasible start, odd k latest; candidate starts are the
 * window ends and every placed job's end and start - L; a start is
 * feasible if the slots of all overlapping jobs plus its own never exceed
 * the total; otherwise retry at the knee, then each smaller swept slot
 * count ("below the knee"); otherwise missed = 1 (slots 0, duration 0,
 * start = release).  Latency at an unswept slot count = that of the
 * largest swept count below it.  Slot ids: jobs in (start, placement
 * order) take the lowest free ids.  utilisation_ppm =
 * floor(1e6 * sum(s*L) / (total*T)).
 * Returns DSTACK_E_INFEASIBLE (with the full best-effort plan filled) if
 * any model had no feasible (b, s) or any job was missed. */
typedef struct {
  int64_t slo_us;
  int max_batch;
  int rate_per_s;                       /* 0: no rate, C(b) = 482*b */
  int n_batches;                        /* rows of the timing table */
  int batches[DSTACK_MAX_BATCHES];
  int n_slots;                          /* columns (ascending slot counts) */
  int slots[DSTACK_MAX_SWEEP];
  int64_t latency_us[DSTACK_MAX_BATCHES][DSTACK_MAX_SWEEP]; /* <= 0: not measured */
} dstack_sched_model;

typedef struct {
  int64_t period_us;
  int total_slots;      /* 1..64; 32 = the whole MI355X */
  int overprov_slots;   /* 2 by default */
  int placement;        /* 0: each job takes the lowest free slot ids;
                           1: home ranges -- each model owns one contiguous
                           range of its deployed size (models by decreasing
                           size, then index, take the offset of least summed
                           overlap with the ranges placed before, lowest on
                           ties); a job uses its whole home range (no
                           below-knee fallback) and starts only when no
                           overlapping job uses a slot of it */
} dstack_sched_params;

typedef struct {
  int model, k;
  int64_t release_us, deadline_us, start_us, duration_us;
  int slots;
  int missed;
  uint64_t slot_mask;
} dstack_job;

typedef struct {
  int n_models;
  int batch[DSTACK_MAX_MODELS];
  int knee_slots[DSTACK_MAX_MODELS];
  int deployed_slots[DSTACK_MAX_MODELS];
  int64_t latency_us[DSTACK_MAX_MODELS];
  int feasible[DSTACK_MAX_MODELS];
  int n_jobs;                           /* in placement (EDF) order */
  dstack_job jobs[DSTACK_MAX_JOBS];
  int64_t utilisation_ppm;
  int home_offset[DSTACK_MAX_MODELS];   /* placement 1: first slot of each home range */
} dstack_schedule_out;

dstack_status dstack_schedule(const dstack_sched_model* models, int n_models, const dstack_sched_params* params,
                              dstack_schedule_out* out);

/* ------------------------------------------------------------------ */
/* Launcher simulation (Sec. 6.1.2: fair, opportunistic, dynamic fill)  */
/* ------------------------------------------------------------------ */
/* Runs the dstack_schedule plan every period for duration_us against a
 * virtual integer-us clock whose job durations come from the timing table,
 * with per-model request queues fed by the arrival traces.
 *  - A planned job takes up to the model's batch of the oldest queued
 *    requests (none queued: it does not run) and lasts its planned time.
 *  - With fod != 0, every arrival and every completion triggers one FOD
 *    pass: candidates are models with no running job and a non-empty queue,
 *    ordered by runs in the last sessions_window sessions (session = t /
 *    period), then cumulative busy us, then index; the first that fits
 *    starts on the lowest-numbered free slots (its deployed count) with the
 *    largest batch of {1,2,4,8,16,32} that is <= max_batch, <= queued and
 *    whose latency ends before the next planned start (at or after now) that
 *    touches those slots or its own next planned start.  At most one FOD
 *    start per pass.
 *  - Same-instant events: completions, then planned starts, then arrivals
 *    (each by model index, then issue order).
 *  - No job starts at or after duration_us.  Served requests with
 *    completion - arrival > SLO and requests still queued when the last
 *    started job ends both count as violations.
 * arrivals_us[i] must be sorted and inside [0, duration_us).  job_hash is
 * FNV-1a (64-bit) over (start, model, batch, slot mask, duration, kind) of
 * every started job, kind 0 planned / 1 FOD, each as 8 little-endian bytes.
 *
 * policy selects the scheduler (Sec. 6.3's comparators; dstack_serve takes
 * 0 only): 0 D-STACK (the plan plus the FOD fill above); 1 max-throughput
 * and 2 max-min fair run no plan, only the fill on every trigger (fod is
 * ignored) with no planned start to respect and the candidates in another
 * order: 1 by the model's SLO-optimal latency at its knee (least runtime
 * first), then index; 2 by deployed slots (smallest GPU% demand first),
 * then busy time, then index.
 * 3 temporal sharing (the time-sliced full-GPU baseline of Sec. 6.1 and the
 * "T" arm of Sec. 7): one model at a time holds all total_slots during its
 * time slice; slices are proportional to the SLOs and repeat every
 * slice_cycle_us (0: the smallest SLO, so every model gets a turn inside
 * each of its SLO intervals): model i's slice is [off_i, off_i + len_i) of
 * each cycle, len_i = floor(cycle * SLO_i / sum of SLOs), offsets in model
 * order, the remainder of the cycle idle.  At every slice start, completion
 * and arrival, if no job runs and the instant lies in the slice of a model
 * with queued requests, that model starts a job (kind 0) on all the slots
 * with the largest grid batch (<= max_batch, <= queued) whose table latency
 * at total_slots ends by its slice's end; none fits: it waits.  No plan, no
 * FOD (fod is ignored).  Other values -> E_INVALID.
 *
 * resize_violations > 0 (policy 0 with placement 1 only, else E_INVALID): a
 * GPU% change triggered by SLO violations (Sec. 3.5's dynamic GPU resource
 * reconfiguration; the trigger count is a parameter).  A request of model i
 * that arrived at or after the model's last change (earlier ones waited
 * through the previous size) counts once: when its job starts, if it has
 * waited more than half its SLO by then (the share Eq. meet_half_slo leaves
 * to waiting), else when its job completes past its SLO.  At the completion
 * that brings the count to the trigger, the model moves to the next larger
 * slot count of its table's columns that has a latency at its plan batch,
 * keeping its home offset if the larger range fits, else ending at the last
 * slot; it stays (and the count restarts) when there is none, or when the
 * larger range would meet the range of another model that its current range
 * does not meet (a change never adds contention).  From then on its planned
 * jobs and FOD jobs use that range and the table latency there; a planned
 * start runs only if its slots are free.  The live launcher moves the model
 * at that moment (between its batches) to the stream of its new range (see
 * dstack_serve); if that stream is not ready yet the model starts no job
 * until it is, and its count restarts from that time. */
typedef struct {
  int64_t duration_us;
  int fod;
  int sessions_window;                          /* 10 */
  const int64_t* arrivals_us[DSTACK_MAX_MODELS];
  int n_arrivals[DSTACK_MAX_MODELS];
  int policy;                                   /* 0 D-STACK, 1 max-throughput, 2 max-min fair, 3 temporal */
  int resize_violations;                        /* 0: off; else late requests that trigger a GPU% change */
  int64_t slice_cycle_us;                       /* policy 3: slice cycle (0: the smallest SLO); >= 0 */
} dstack_sim_params;

typedef struct {
  int64_t served, violations, unserved, planned_runs, fod_runs, busy_us, p50_us, p99_us;
  int64_t plan_skips;   /* planned starts that did not run (empty queue, model still running,
                           or its slots still held: an overrunning job, a GPU% change) */
  int64_t resizes;      /* GPU% changes on SLO violations */
  int64_t final_slots;  /* the model's slots at the end (temporal: all) */
} dstack_model_stats;

typedef struct {
  int n_models;
  dstack_model_stats models[DSTACK_MAX_MODELS];
  int64_t utilisation_ppm;                      /* floor(1e6 * slot-us inside [0, duration) / (total * duration)) */
  uint64_t job_hash;
  int64_t last_end_us;
} dstack_run_out;

dstack_status dstack_simulate(const dstack_sched_model* models, int n_models, const dstack_sched_params* params,
                              const dstack_sim_params* sim, dstack_run_out* out);

/* The ideal spatio-temporal schedule of Sec. 6.2 (Eqs. maximization and
 * constraints): time slots of slot_us, kernel granularity, preemption.
 * Model i runs forwards of n_kernels kernels in order, kernel k at its own
 * knee share slots[k] (1..total) for dur_us[k] >= 1 us, batch items each;
 * closed loop: the next forward is released when one ends, due release +
 * slo_us.  In every slot the eligible kernels are each model's current
 * kernel; of all model subsets whose shares sum to at most total_slots the
 * one with the largest sum runs (exhaustive), ties to the subset whose
 * inclusion bits, taken in (deadline, index) order with the earliest first,
 * form the largest number.  A running kernel's remaining time drops by
 * slot_us; at or below 0 the model moves to its next kernel from the next
 * slot on, and after its last kernel the forward ends at the slot's end
 * (late if past its deadline).  Slots start at 0 while < horizon_us.
 * utilisation_ppm = floor(1e6 * sum of used shares over slots / (total *
 * slots)); hash = FNV-1a over (slot start, chosen subset bits) of every slot.
 * n_models 1..8, horizon_us >= 1, slot_us >= 1, else E_INVALID. */
typedef struct {
  int n_kernels;
  int batch;
  const int* slots;
  const int64_t* dur_us;
  int64_t slo_us;
} dstack_ideal_model;
typedef struct {
  int n_models;
  int64_t items[DSTACK_MAX_MODELS];
  int64_t forwards[DSTACK_MAX_MODELS];
  int64_t late[DSTACK_MAX_MODELS];
  int64_t busy_slot_us[DSTACK_MAX_MODELS];   /* share x slot length of every slot it ran in */
  int64_t utilisation_ppm;
  uint64_t hash;
} dstack_ideal_out;
dstack_status dstack_simulate_ideal(const dstack_ideal_model* models, int n_models, int64_t horizon_us, int64_t slot_us,
                                    int total_slots, dstack_ideal_out* out);

/* ------------------------------------------------------------------ */
/* Live launcher (Sec. 6.1.2 on the GPU)                                */
/* ------------------------------------------------------------------ */
/* Runs the same plan and the same FOD decisions as dstack_simulate, on the
 * host's monotonic clock (us since the call's start, after a warm-up) with
 * real batches: model i runs on a partition over its home range (placement
 * must be 1; models with identical ranges share one, as their jobs never
 * overlap) and every job of model i runs as dstack_infer(models[i], b,
 * d_in[i], d_out[i], that partition) would, with a workspace (activations,
 * split-K buffers, captured graphs) the model keeps for the launcher across
 * partitions and calls.  Requests arrive when the clock passes their
 * trace time; a job's requests complete when its end event is seen by the
 * polling host thread (latency = that time - arrival).  Decisions use the
 * timing table only (busy time is charged with the table latency); a planned
 * start finds its home range still held by an overrunning job, or the model
 * still running, and is skipped (plan_skips).  busy_us, the percentiles and
 * utilisation_ppm use measured GPU time (device events around each job).
 * Not reproducible run to run: job_hash covers the decisions taken.
 *  - n_models in 1..4 (at most one CU-masked stream per model);
 *  - GPU% changes (sim->resize_violations > 0, the rule of dstack_simulate):
 *    a model's next range runs on the stream of that range if one is live,
 *    else on a new one created on a helper thread while the other models
 *    keep running (the model starts no job until it is ready); while the
 *    partition limit leaves room, a model at risk of its next change (a
 *    request late since its last change, or one that waited more than half
 *    its SLO before its job started) gets that stream ahead of the change (a
 *    standby), so that the change takes effect when it is decided (kind 3
 *    below at that time);
 *  - d_in[i], d_out[i]: caller-owned device buffers holding the model's
 *    input and output at tables[i].max_batch (shapes of dstack_model_query);
 *    a job of batch b reads its input from the start of d_in[i] and writes
 *    its output to the start of d_out[i], in the layouts of dstack_infer at
 *    batch b (the trace's requests carry no data of their own);
 *  - tables[i]: the timing table of models[i] (max_batch <= the model's);
 *  - the call blocks for about duration_us plus the last job, then waits for
 *    the device; log (may be NULL) receives up to log_capacity job records,
 *    *n_log the number of jobs started.
 *  - sim->policy 0 (D-STACK) or 3 (temporal sharing, see dstack_simulate):
 *    with 3 every model runs on one partition of all total_slots (<= 32),
 *    one job at a time, in the slices dstack_simulate describes, with slice
 *    starts in place of planned starts;
 *  - events (may be NULL) receives up to event_capacity triggers in the order
 *    the launcher handled them, *n_events the number handled: kind 0 a
 *    completion seen (model), kind 1 a planned start due (model, value_us =
 *    its planned time, slot_mask = its slots; temporal: a slice start, mask
 *    all slots), kind 2 an arrival admitted (model, value_us = its trace
 *    time), kind 3 a GPU% change took effect (model, slot_mask = its new
 *    range); t_us is the clock value the decision taken at that trigger used
 *    (a job started there has start_us == t_us), so that the decisions can be
 *    replayed from the table and this list alone.
 * Errors: E_INVALID (bad arguments, D-STACK without placement 1, a policy
 * other than 0 or 3), E_UNSUPPORTED (more than 4 models), E_HIP; the plan's
 * E_INFEASIBLE is not an error here (the filled plan runs, as in
 * dstack_simulate). */
typedef struct {
  int64_t start_us;     /* host clock at launch */
  int64_t end_us;       /* host clock when completion was seen */
  int64_t gpu_us;       /* device time between the job's start and end events */
  int64_t table_us;     /* latency the decision assumed */
  int model, batch, kind;  /* kind 0 planned, 1 FOD */
  uint64_t slot_mask;
} dstack_job_record;

typedef struct {
  int64_t t_us;        /* clock value of the decision at this trigger */
  int64_t value_us;    /* arrival: trace time; planned / slice start: its planned time; else 0 */
  uint64_t slot_mask;  /* planned / slice start: its slots; else 0 */
  int kind;            /* 0 completion seen, 1 planned or slice start due, 2 arrival admitted, 3 GPU% change ready */
  int model;
} dstack_serve_event;

dstack_status dstack_serve(const dstack_model* models, int n_models, const void* const* d_in, void* const* d_out,
                           const dstack_sched_model* tables, const dstack_sched_params* params,
                           const dstack_sim_params* sim, dstack_run_out* out, dstack_job_record* log,
                           int log_capacity, int* n_log, dstack_serve_event* events, int event_capacity,
                           int* n_events);

/* ------------------------------------------------------------------ */
/* Kernel-level entry points (the layers of Sec. 4.1's A.int table)     */
/* ------------------------------------------------------------------ */
/* All pointers are device pointers; `stream` is a hipStream_t (NULL = the
 * null stream).  Asynchronous.  Layouts are NHWC / KRSC bf16 with fp32
 * per-channel scale and shift; act: 0 none, 1 ReLU, 2 ReLU6.
 *
 * conv2d: y = act(scale[k] * sum_{r,s,c} x[n, ho*st-pad+r, wo*st-pad+s, c]
 *   * w[k,r,s,c] + shift[k] (+ res[n,ho,wo,k])), zero outside the image;
 *   act 0 none, 1 ReLU, 2 ReLU6, 3 GELU (erf form), 4 tanh;
 *   C % 8 == 0 and K % 4 == 0 (else E_UNSUPPORTED); res may be NULL;
 *   out_fp32 selects an fp32 instead of bf16 output.  The tile plan is
 *   chosen for the CUs the stream's CU mask enables (the whole device for
 *   the null stream); no split-K workspace is used here (dstack_op_conv2d_ws
 *   takes one).
 * dwconv3x3: per-channel 3x3, pad 1, stride 1 or 2, w [3][3][C] (device
 *   layout), then scale/shift and act; C % 8 == 0.
 * fc: y[b][o] = act(sum_i x[b][i] * w[o][i] + bias[o]); batch 1..32,
 *   I % 8 == 0; out_fp32 selects fp32 output.  workspace (device, may be
 *   NULL) holds fp32 partial sums when the depth I is split over several
 *   blocks: fc_workspace_bytes(B, I, O) bytes give the split chosen for the
 *   whole GPU; NULL or fewer bytes run fewer splits (same result up to fp32
 *   summation order).
 * maxpool: k x k window, stride, pad (padding never wins); C % 8 == 0.
 * avgpool: global mean over H x W, fp32 accumulate, bf16 out; C % 8 == 0.
 * lstm_layer: one LSTM layer over T steps (gate order i, f, g, o; h0 = c0
 *   = 0); x [T][B][I] bf16; w_ih [4H][I], w_hh [4H][H] bf16; bias [4H]
 *   fp32 (= b_ih + b_hh); h_bf16 [T][B][H] receives h rounded to bf16;
 *   h_f32 [T][B][H] (may be NULL) receives h in fp32; B in 1..32,
 *   H % 32 == 0 and H <= 2048, I % 8 == 0; workspace (device, 256-byte
 *   aligned, caller owned) needs lstm_workspace_bytes(T, B, H) bytes: the
 *   input projections, the cell state, and copies of W_hh and of h(t-1) in
 *   the recurrent product's fragment order (W_hh is repacked on each call).
 *   The recurrent step's launch (hidden units per workgroup) is chosen for
 *   the CUs of the stream's CU mask; the result does not depend on it. */
dstack_status dstack_op_conv2d(const void* x, int N, int H, int W, int C, const void* w, int K, int R, int S,
                               int stride, int pad, const float* scale, const float* shift, const void* res, int act,
                               void* y, int out_fp32, void* stream);
/* conv2d_ws: conv2d with the library's depth split (split-K): the depth
 *   R*S*C is cut into `splits` slices run by separate workgroups, each writes
 *   fp32 partial sums, and the last workgroup of each output tile (counted
 *   by a per-tile arrival counter) sums the slices in slice order and applies
 *   the epilogue, all in one kernel launch.  The plan (tile, splits, LDS ring)
 *   is chosen for n_cu CUs (n_cu <= 0: the CUs of the stream's CU mask), as
 *   dstack_conv2d_plan reports.  workspace (device, 256-byte aligned, caller
 *   owned, may be NULL) = 16 KiB of arrival counters followed by the slices;
 *   the counters must be zero before the first call that uses the workspace
 *   and every call leaves them zero.  A workspace smaller than the plan's
 *   workspace_bytes (or NULL) runs fewer splits (same result up to fp32
 *   summation order).  out_fp32 never splits.  Calls sharing a workspace must
 *   not overlap in time.
 * conv2d_plan (host only): the launch dstack_op_conv2d_ws takes for a shape
 *   on n_cu CUs (<= 0: 256) with a workspace of `workspace_bytes` bytes
 *   (SIZE_MAX: unlimited), and the workspace that plan needs (0 without a
 *   split).  Same shape checks as conv2d.
 * arch_convs (host only): the implicit-GEMM convolutions of one forward of
 *   an architecture at `batch`, in launch order, as conv2d arguments (the
 *   LSTM's input projections as 1x1 convolutions over T*batch pixels with an
 *   fp32 output); fills at most max_convs, *n_convs = the total. */
typedef struct {
  int kernel;          /* 0: tiled implicit GEMM; 1: streaming 1x1 (C <= 32) */
  int mode;            /* activation addressing: 0 1x1 strided, 1 C % 64 == 0, 2 general, 3 1x1 stride 1 */
  int tile_n, tile_m;  /* output channels x output pixels per workgroup (kernel 1: channels per wave, 0) */
  int splits;          /* depth slices (1: no split) */
  int tiles_per_split; /* 64-deep depth tiles per slice */
  int stages;          /* LDS ring depth (kernel 0) */
  int pad;
  size_t workspace_bytes;
} dstack_conv_plan;
typedef struct {
  int N, H, W, C, K, R, S, stride, pad, act, has_residual, out_fp32;
} dstack_conv_shape;
dstack_status dstack_op_conv2d_ws(const void* x, int N, int H, int W, int C, const void* w, int K, int R, int S,
                                  int stride, int pad, const float* scale, const float* shift, const void* res,
                                  int act, void* y, int out_fp32, int n_cu, void* workspace, size_t workspace_bytes,
                                  void* stream);
dstack_status dstack_conv2d_plan(int N, int H, int W, int C, int K, int R, int S, int stride, int pad, int act,
                                 int out_fp32, int n_cu, size_t workspace_bytes, dstack_conv_plan* out);
/* conv2d_noalloc: dstack_op_conv2d_ws for callers that cannot allocate
 *   device memory (code under HIP graph capture, tight serving loops,
 *   harnesses that forbid hipMalloc).  The split-K slices and arrival
 *   counters live in a fixed scratch array inside the library, of
 *   dstack_conv2d_noalloc_scratch_bytes() bytes (32 MiB + 16 KiB) on every
 *   device the library runs on, held until the process ends; the call
 *   allocates nothing.  The plan is the one dstack_op_conv2d_ws takes with a
 *   workspace as large as that plan needs (dstack_conv2d_plan with
 *   workspace_bytes = SIZE_MAX), so both give the same result; a shape whose
 *   plan needs more scratch than the array holds returns E_UNSUPPORTED
 *   before anything is launched.  The first call on a device looks up the
 *   array's address and clears its counters with a small kernel on
 *   `stream`; every call leaves them zero.  All calls on one device share
 *   the array: calls that overlap in time on one device race (serialise
 *   them, e.g. on one stream).  Other arguments and errors as conv2d_ws. */
dstack_status dstack_op_conv2d_noalloc(const void* x, int N, int H, int W, int C, const void* w, int K, int R, int S,
                                       int stride, int pad, const float* scale, const float* shift, const void* res,
                                       int act, void* y, int out_fp32, int n_cu, void* stream);
size_t dstack_conv2d_noalloc_scratch_bytes(void);
dstack_status dstack_arch_convs(const char* arch, int batch, dstack_conv_shape* out, int max_convs, int* n_convs);
/* conv2d_rgb: the conv2d above for a 3-channel image x [N][H][W][3] read as
 *   it is (the stems of Sec. 3's CNNs; no packing to 8 channels), with
 *   weights w4 [K][R][R][4] bf16 (channel 3 zero: the stem layout the
 *   models store), no residual and bf16 output.  (R, K) one of (3, 16),
 *   (3, 32), (3, 64), (7, 64) (else E_UNSUPPORTED); stride >= 1,
 *   0 <= pad < R; scale and shift are required; image rows too wide for a
 *   64 KB LDS tile of the input rows that 256 output pixels touch give
 *   E_UNSUPPORTED. */
dstack_status dstack_op_conv2d_rgb(const void* x, int N, int H, int W, const void* w4, int K, int R, int stride,
                                   int pad, const float* scale, const float* shift, int act, void* y, void* stream);
/* expand_dw: the expand half of an inverted residual block (Sec. 3's
 *   MobileNet) in one kernel: e = act_e(se[c] * sum_i x[n,h,w,i] * we[c,i]
 *   + he[c]) rounded to bf16, then y = act_d(sd[c] * dwconv3x3(e) + hd[c])
 *   with pad 1 and stride 1 or 2 (zero e outside the image); x [N][H][W][Cin],
 *   we [Ce][Cin], wd [3][3][Ce] (device layout), y [N][Ho][Wo][Ce] bf16; the
 *   expanded tensor e is never written to memory.  Cin % 8 == 0 and <= 160,
 *   Ce a multiple of 48 or 64 (else E_UNSUPPORTED); all pointers required. */
dstack_status dstack_op_expand_dw(const void* x, int N, int H, int W, int Cin, const void* we, int Ce,
                                  const float* se, const float* he, int act_e, const void* wd, int stride,
                                  const float* sd, const float* hd, int act_d, void* y, void* stream);
dstack_status dstack_op_dwconv3x3(const void* x, int N, int H, int W, int C, const void* w, int stride,
                                  const float* scale, const float* shift, int act, void* y, void* stream);
size_t dstack_fc_workspace_bytes(int B, int I, int O);
dstack_status dstack_op_fc(const void* x, int B, int I, const void* w, const float* bias, int O, int act, void* y,
                           int out_fp32, void* workspace, size_t workspace_bytes, void* stream);
dstack_status dstack_op_maxpool(const void* x, int N, int H, int W, int C, int k, int stride, int pad, void* y,
                                void* stream);
dstack_status dstack_op_avgpool(const void* x, int N, int H, int W, int C, void* y, void* stream);
size_t dstack_lstm_workspace_bytes(int T, int B, int H);
dstack_status dstack_op_lstm_layer(const void* x, int T, int B, int I, int H, const void* w_ih, const void* w_hh,
                                   const float* bias, void* h_bf16, float* h_f32, void* workspace, void* stream);
/* Transformer kernels (the BERT encoder of Sec. 4.4's transformer workload).
 * embed_ln: for each of `rows` tokens (ids int32 [rows], position = row %
 *   T, token type 0): e = we[id] + pe[row % T] + te[0] (tables bf16
 *   [vocab][H], [>= T][H], [>= 1][H]), then layer norm y = (e - mean) /
 *   sqrt(var + eps) * gamma + beta over the H values (biased variance; gamma
 *   / beta fp32 [H] or NULL for 1 / 0), y bf16 [rows][H].  Ids outside
 *   [0, vocab) read row vocab - 1.  H <= 2048 (else E_UNSUPPORTED).
 * layernorm: the same normalisation of x bf16 [rows][H] into y bf16.
 * attention: qkv bf16 [B][T][3 * heads * dh] (queries, keys, values, head h
 *   at columns h*dh of each) -> out bf16 [B][T][heads * dh] with, per
 *   sequence and head, out_i = sum_j softmax_j(q_i . k_j / sqrt(dh)) v_j
 *   (no mask, fp32 arithmetic).  dh == 64 and T <= 48 (else
 *   E_UNSUPPORTED). */
dstack_status dstack_op_embed_ln(const int32_t* ids, int rows, int T, int vocab, const void* we, const void* pe,
                                 const void* te, int H, const float* gamma, const float* beta, float eps, void* y,
                                 void* stream);
dstack_status dstack_op_layernorm(const void* x, int rows, int H, const float* gamma, const float* beta, float eps,
                                  void* y, void* stream);
dstack_status dstack_op_attention(const void* qkv, int B, int T, int heads, int dh, void* out, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* DSTACK_H */
